// Device twin of the seeded input generator in synth.c (inputs only; none of
// the layer's arithmetic). Same definition, bit-identical values:
//   h(i) = splitmix64 output of key + (i + 1) * 0x9E3779B97F4A7C15,
//   S(i) = sum of the eight bytes of h(i),
//   value = fp32(fp32((float)(S - 1020) * c) + bias), rounded to bfloat16
// with one correctly rounded multiply and one correctly rounded add (no
// contraction), so the host can regenerate any slice the GPU holds.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

__host__ __device__ inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

__device__ inline int byte_sum(uint64_t h) {
  uint64_t a = (h & 0x00FF00FF00FF00FFULL) + ((h >> 8) & 0x00FF00FF00FF00FFULL);
  a = (a & 0x0000FFFF0000FFFFULL) + ((a >> 16) & 0x0000FFFF0000FFFFULL);
  a = (a & 0x00000000FFFFFFFFULL) + (a >> 32);
  return (int)a;
}

__device__ inline uint16_t to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)((u >> 16) | ((u & 0xFFFFu) ? 0x40u : 0u));
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ inline float draw(uint64_t key, uint64_t i, float c, float bias) {
  const uint64_t h = mix64(key + (i + 1) * 0x9E3779B97F4A7C15ULL);
  return __fadd_rn(__fmul_rn((float)(byte_sum(h) - 1020), c), bias);
}

// 8 consecutive values per thread, one 16-byte store
__global__ void fill_bf16_kernel(uint64_t key, uint64_t offset, int64_t n, float c, float bias, uint16_t* out) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x * 8;
  for (int64_t j = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 8; j < n; j += stride) {
    if (j + 8 <= n) {
      uint32_t w[4];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        w[q] = (uint32_t)to_bf16_rne(draw(key, offset + j + 2 * q, c, bias)) |
               ((uint32_t)to_bf16_rne(draw(key, offset + j + 2 * q + 1, c, bias)) << 16);
      *reinterpret_cast<uint4*>(out + j) = make_uint4(w[0], w[1], w[2], w[3]);
    } else {
      for (int64_t q = j; q < n; ++q) out[q] = to_bf16_rne(draw(key, offset + q, c, bias));
    }
  }
}

// bulk variant (synth.c: synth_fill_fast_bf16): murmur3 finaliser, Irwin-Hall(4)
__device__ inline uint32_t fmix32(uint32_t h) {
  h ^= h >> 16;
  h *= 0x85EBCA6Bu;
  h ^= h >> 13;
  h *= 0xC2B2AE35u;
  h ^= h >> 16;
  return h;
}

__device__ inline float draw_fast(uint32_t key, uint32_t i, float c, float bias) {
  const uint32_t g = fmix32(key + i * 0x9E3779B9u);
  const int s = (int)(g & 0xFF) + (int)((g >> 8) & 0xFF) + (int)((g >> 16) & 0xFF) + (int)(g >> 24);
  return __fadd_rn(__fmul_rn((float)(s - 510), c), bias);
}

__global__ void fill_fast_bf16_kernel(uint32_t key, uint32_t offset, int64_t n, float c, float bias, uint16_t* out) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x * 8;
  for (int64_t j = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 8; j < n; j += stride) {
    if (j + 8 <= n) {
      uint32_t w[4];
#pragma unroll
      for (int q = 0; q < 4; ++q)
        w[q] = (uint32_t)to_bf16_rne(draw_fast(key, offset + (uint32_t)(j + 2 * q), c, bias)) |
               ((uint32_t)to_bf16_rne(draw_fast(key, offset + (uint32_t)(j + 2 * q + 1), c, bias)) << 16);
      *reinterpret_cast<uint4*>(out + j) = make_uint4(w[0], w[1], w[2], w[3]);
    } else {
      for (int64_t q = j; q < n; ++q) out[q] = to_bf16_rne(draw_fast(key, offset + (uint32_t)q, c, bias));
    }
  }
}

__global__ void fill_u8_kernel(uint64_t key, uint64_t offset, int64_t n, uint8_t* out) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j < n; j += stride)
    out[j] = (uint8_t)(mix64(key + (offset + j + 1) * 0x9E3779B97F4A7C15ULL) & 0xFF);
}

}  // namespace

extern "C" {

// out: device array of n bfloat16 (16-byte aligned when n >= 8). Returns a hipError_t.
int synth_fill_device_bf16(uint64_t seed, uint64_t tensor_id, uint64_t offset, int64_t n, float c, float bias,
                           void* out, void* stream) {
  if (n <= 0) return 0;
  const uint64_t key = mix64(mix64(seed) ^ tensor_id);
  const int64_t groups = (n + 7) / 8;
  const int blocks = (int)((groups + 255) / 256 < 65536 ? (groups + 255) / 256 : 65536);
  hipLaunchKernelGGL(fill_bf16_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream, key,
                     offset, n, c, bias, (uint16_t*)out);
  return (int)hipGetLastError();
}

int synth_fill_device_fast_bf16(uint64_t seed, uint64_t tensor_id, uint32_t offset, int64_t n, float c, float bias,
                                void* out, void* stream) {
  if (n <= 0) return 0;
  const uint32_t key = (uint32_t)mix64(mix64(seed) ^ tensor_id);
  const int64_t groups = (n + 7) / 8;
  const int blocks = (int)((groups + 255) / 256 < 65536 ? (groups + 255) / 256 : 65536);
  hipLaunchKernelGGL(fill_fast_bf16_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream, key, offset, n, c,
                     bias, (uint16_t*)out);
  return (int)hipGetLastError();
}

int synth_fill_device_u8(uint64_t seed, uint64_t tensor_id, uint64_t offset, int64_t n, void* out, void* stream) {
  if (n <= 0) return 0;
  const uint64_t key = mix64(mix64(seed) ^ tensor_id);
  const int64_t b = (n + 255) / 256;
  const int blocks = (int)(b < 16384 ? b : 16384);
  hipLaunchKernelGGL(fill_u8_kernel, dim3(blocks), dim3(256), 0, (hipStream_t)stream, key, offset, n,
                     (uint8_t*)out);
  return (int)hipGetLastError();
}

}  // extern "C"
