// Device-side helpers shared by the gfx950 kernels: storage types, bfloat16
// conversion, wavefront reductions and the matrix-core (MFMA) fragment
// operations the kernels are built on.
//
// Fragment convention. Every matrix-core product here is D[16][16] += A[16][K] * B[K][16]
// with K a multiple of 32. A wavefront lane l (0..63) supplies row (or column)
// l % 16 and the 8 consecutive reduction indices 8 * (l / 16) .. +7 of each
// 32-wide reduction chunk, for both A and B. The accumulator lane l holds
// D[4 * (l / 16) + r][l % 16], r = 0..3.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mcpu {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));

// Streaming loads for data that one workgroup reads once (KV pages, weight
// slabs no other workgroup shares): the non-temporal cache policy. On MI355X
// a cold 1 GiB read runs at 6.8-6.9 TB/s with it against 5.9-6.3 TB/s with
// plain loads; lines it brings in do not stay in L2, so data that other
// workgroups re-read from L2 keeps plain loads.
typedef uint32_t stream_u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t stream_u32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ stream_u32x4 ld_stream16(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const stream_u32x4*>(p));
}
__device__ __forceinline__ stream_u32x2 ld_stream8(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const stream_u32x2*>(p));
}

struct bf16 {  // storage-only bfloat16 (raw bits)
  uint16_t bits;
};

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// round to nearest, ties to even; NaN stays NaN
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7F800000u) == 0x7F800000u) return (uint16_t)((u >> 16) | ((u & 0xFFFFu) ? 0x40u : 0u));
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <typename T> struct Elem;
template <> struct Elem<float> {
  static __device__ __forceinline__ float load(const float* p, int64_t i) { return p[i]; }
  static __device__ __forceinline__ void store(float* p, int64_t i, float v) { p[i] = v; }
};
template <> struct Elem<bf16> {
  static __device__ __forceinline__ float load(const bf16* p, int64_t i) { return bf16_to_f32(p[i].bits); }
  static __device__ __forceinline__ void store(bf16* p, int64_t i, float v) { p[i].bits = f32_to_bf16(v); }
};

// four consecutive elements from fp32 (p 16- or 8-byte aligned)
__device__ __forceinline__ void store4(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
__device__ __forceinline__ void store4(bf16* p, float4 v) {
  *reinterpret_cast<uint2*>(p) = make_uint2((uint32_t)f32_to_bf16(v.x) | ((uint32_t)f32_to_bf16(v.y) << 16),
                                            (uint32_t)f32_to_bf16(v.z) | ((uint32_t)f32_to_bf16(v.w) << 16));
}

// ---------------------------------------------------------------------------
// wavefront helpers (64 lanes)
// ---------------------------------------------------------------------------

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Load of a wave-uniform element of memory the kernel only reads (a page
// table), through the constant address space so that it becomes a scalar load:
// its wait counter is separate from the vector loads a kernel keeps in flight.
__device__ __forceinline__ int32_t load_uniform(const int32_t* p, int64_t i) {
  typedef __attribute__((address_space(4))) const int32_t cint32;
  return reinterpret_cast<cint32*>(reinterpret_cast<uintptr_t>(p))[i];
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
// inclusive prefix sum over the 64 lanes
__device__ __forceinline__ int wave_incl_scan(int v) {
  const int l = lane_id();
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int t = __shfl_up(v, o, 64);
    if (l >= o) v += t;
  }
  return v;
}

// ---------------------------------------------------------------------------
// 8-element fragments: one lane's 8 consecutive reduction indices
// ---------------------------------------------------------------------------

template <typename T> struct Frag;

template <> struct Frag<bf16> {
  uint4 v;  // 8 x bf16
  __device__ __forceinline__ void load(const bf16* p) { v = *reinterpret_cast<const uint4*>(p); }
  __device__ __forceinline__ void load_stream(const bf16* p) {
    const stream_u32x4 r = ld_stream16(p);
    v = make_uint4(r[0], r[1], r[2], r[3]);
  }
  __device__ __forceinline__ void zero() { v = make_uint4(0, 0, 0, 0); }
  __device__ __forceinline__ void keep_if(bool k) {  // zero unless k, without a branch
    v.x = k ? v.x : 0u; v.y = k ? v.y : 0u; v.z = k ? v.z : 0u; v.w = k ? v.w : 0u;
  }
};
template <> struct Frag<float> {
  float4 a, b;  // 8 x fp32
  __device__ __forceinline__ void load(const float* p) {
    a = reinterpret_cast<const float4*>(p)[0];
    b = reinterpret_cast<const float4*>(p)[1];
  }
  __device__ __forceinline__ void load_stream(const float* p) {
    const stream_u32x4 r0 = ld_stream16(p), r1 = ld_stream16(p + 4);
    a = make_float4(__uint_as_float(r0[0]), __uint_as_float(r0[1]), __uint_as_float(r0[2]), __uint_as_float(r0[3]));
    b = make_float4(__uint_as_float(r1[0]), __uint_as_float(r1[1]), __uint_as_float(r1[2]), __uint_as_float(r1[3]));
  }
  __device__ __forceinline__ void zero() { a = b = make_float4(0.f, 0.f, 0.f, 0.f); }
  __device__ __forceinline__ void keep_if(bool k) {
    a.x = k ? a.x : 0.f; a.y = k ? a.y : 0.f; a.z = k ? a.z : 0.f; a.w = k ? a.w : 0.f;
    b.x = k ? b.x : 0.f; b.y = k ? b.y : 0.f; b.z = k ? b.z : 0.f; b.w = k ? b.w : 0.f;
  }
};

// acc += A-fragment x B-fragment over one 32-wide reduction chunk
__device__ __forceinline__ f32x4 mma32(const Frag<bf16>& A, const Frag<bf16>& B, f32x4 acc) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, A.v),
                                                  __builtin_bit_cast(bf16x8_t, B.v), acc, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma32(const Frag<float>& A, const Frag<float>& B, f32x4 acc) {
  // eight K=4 products; product e pairs element e of every lane group
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(A.a.x, B.a.x, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(A.a.y, B.a.y, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(A.a.z, B.a.z, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(A.a.w, B.a.w, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(A.b.x, B.b.x, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(A.b.y, B.b.y, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(A.b.z, B.b.z, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(A.b.w, B.b.w, acc, 0, 0, 0);
  return acc;
}

// ---------------------------------------------------------------------------
// 4-element fragments for the value product: lane l supplies reduction
// indices 4 * (l / 16) .. +3 of a 16-wide chunk (one 16-token page).
// ---------------------------------------------------------------------------

template <typename T> struct Frag4;
template <> struct Frag4<bf16> {
  uint2 v;
  __device__ __forceinline__ void load(const bf16* p) { v = *reinterpret_cast<const uint2*>(p); }
  __device__ __forceinline__ void load_stream(const bf16* p) {
    const stream_u32x2 r = ld_stream8(p);
    v = make_uint2(r[0], r[1]);
  }
};
template <> struct Frag4<float> {
  float4 v;
  __device__ __forceinline__ void load(const float* p) { v = *reinterpret_cast<const float4*>(p); }
  __device__ __forceinline__ void load_stream(const float* p) {
    const stream_u32x4 r = ld_stream16(p);
    v = make_float4(__uint_as_float(r[0]), __uint_as_float(r[1]), __uint_as_float(r[2]), __uint_as_float(r[3]));
  }
};

// acc += A(16 x 16 chunk) * B(16 x 16) where B's lane values are 4 fp32 p[r]
// (converted to the operand type here).
__device__ __forceinline__ f32x4 mma16_p(const Frag4<bf16>& A, const float p[4], f32x4 acc, float* psum) {
  uint16_t b0 = f32_to_bf16(p[0]), b1 = f32_to_bf16(p[1]), b2 = f32_to_bf16(p[2]), b3 = f32_to_bf16(p[3]);
  if (psum) *psum += bf16_to_f32(b0) + bf16_to_f32(b1) + bf16_to_f32(b2) + bf16_to_f32(b3);
  uint2 bv = make_uint2((uint32_t)b0 | ((uint32_t)b1 << 16), (uint32_t)b2 | ((uint32_t)b3 << 16));
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(i16x4_t, A.v),
                                                    __builtin_bit_cast(i16x4_t, bv), acc, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma16_p(const Frag4<float>& A, const float p[4], f32x4 acc, float* psum) {
  if (psum) *psum += p[0] + p[1] + p[2] + p[3];
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(A.v.x, p[0], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(A.v.y, p[1], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(A.v.z, p[2], acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(A.v.w, p[3], acc, 0, 0, 0);
  return acc;
}

// acc += A * B over 32 keys taken from two 16-key pages: the reduction slots
// of lane l are keys 4 (l / 16) .. +3 of page a, then the same keys of page b,
// in both operands, so the score tiles of two pages feed one 16x16x32 product.
// Lane values pa[r], pb[r] are rounded to the operand type; their rounded sum
// is added to *psum.
__device__ __forceinline__ f32x4 mma32_p(const Frag4<bf16>& Va, const Frag4<bf16>& Vb, const float pa[4],
                                         const float pb[4], f32x4 acc, float* psum) {
  uint16_t b[8];
  float s = 0.f;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    b[r] = f32_to_bf16(pa[r]);
    b[4 + r] = f32_to_bf16(pb[r]);
  }
#pragma unroll
  for (int r = 0; r < 8; ++r) s += bf16_to_f32(b[r]);
  *psum += s;
  const uint4 bv = make_uint4((uint32_t)b[0] | ((uint32_t)b[1] << 16), (uint32_t)b[2] | ((uint32_t)b[3] << 16),
                              (uint32_t)b[4] | ((uint32_t)b[5] << 16), (uint32_t)b[6] | ((uint32_t)b[7] << 16));
  const uint4 av = make_uint4(Va.v.x, Va.v.y, Vb.v.x, Vb.v.y);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, av), __builtin_bit_cast(bf16x8_t, bv),
                                                  acc, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma32_p(const Frag4<float>& Va, const Frag4<float>& Vb, const float pa[4],
                                         const float pb[4], f32x4 acc, float* psum) {
  acc = mma16_p(Va, pa, acc, psum);
  return mma16_p(Vb, pb, acc, psum);
}

// Maximum over the four lanes l, l ^ 16, l ^ 32, l ^ 48 (the four 16-lane rows
// holding one accumulator column), with the gfx950 row-swap permutes.
// Maximum that propagates NaN (IEEE 754-2019 maximum). Unlike fmaxf it needs
// no quieting of its operands, so a max over products is one v_maximum3_f32
// per two or three values instead of a canonicalising v_max per operand.
__device__ __forceinline__ float vmax(float a, float b) { return __builtin_elementwise_maximum(a, b); }

__device__ __forceinline__ float max_over_rows(float v) {
  uint32_t u = __float_as_uint(v);
  auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);  // rows {0,1} vs {2,3}
  v = vmax(__uint_as_float(a[0]), __uint_as_float(a[1]));
  u = __float_as_uint(v);
  auto b = __builtin_amdgcn_permlane16_swap(u, u, false, false);  // rows {0,2} vs {1,3}
  return vmax(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
// two floats to packed bfloat16 (round to nearest even, in hardware)
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{lo, hi}), bf16x2_t));
}

// As mma32_p, without the running sum (the caller gets it from a product
// against a fragment of ones).
__device__ __forceinline__ f32x4 mma32_pv(const Frag4<bf16>& Va, const Frag4<bf16>& Vb, const float pa[4],
                                          const float pb[4], f32x4 acc) {
  const uint4 bv = make_uint4(pack_bf16(pa[0], pa[1]), pack_bf16(pa[2], pa[3]), pack_bf16(pb[0], pb[1]),
                              pack_bf16(pb[2], pb[3]));
  const uint4 av = make_uint4(Va.v.x, Va.v.y, Vb.v.x, Vb.v.y);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, av), __builtin_bit_cast(bf16x8_t, bv),
                                                  acc, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma32_pv(const Frag4<float>& Va, const Frag4<float>& Vb, const float pa[4],
                                          const float pb[4], f32x4 acc) {
  acc = mma16_p(Va, pa, acc, nullptr);
  return mma16_p(Vb, pb, acc, nullptr);
}
// V operand of a two-page PV product: the lane's 4 values of page a, then
// the same slots of page b, loaded straight into one register quadruple.
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
template <typename T> struct PVFrag;
template <> struct PVFrag<bf16> {
  u32x4_t v;
  __device__ __forceinline__ void load(const bf16* a, const bf16* b) {
    const u32x2_t x = *reinterpret_cast<const u32x2_t*>(a), y = *reinterpret_cast<const u32x2_t*>(b);
    v = __builtin_shufflevector(x, y, 0, 1, 2, 3);
  }
};
template <> struct PVFrag<float> {
  Frag4<float> a, b;
  __device__ __forceinline__ void load(const float* pa, const float* pb) {
    a.load(pa);
    b.load(pb);
  }
};
__device__ __forceinline__ f32x4 mma32_pv(const PVFrag<bf16>& V, const float pa[4], const float pb[4], f32x4 acc) {
  const uint4 bv = make_uint4(pack_bf16(pa[0], pa[1]), pack_bf16(pa[2], pa[3]), pack_bf16(pb[0], pb[1]),
                              pack_bf16(pb[2], pb[3]));
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, V.v), __builtin_bit_cast(bf16x8_t, bv),
                                                  acc, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma32_pv(const PVFrag<float>& V, const float pa[4], const float pb[4], f32x4 acc) {
  acc = mma16_p(V.a, pa, acc, nullptr);
  return mma16_p(V.b, pb, acc, nullptr);
}
__device__ __forceinline__ void ones(Frag4<bf16>& f) { f.v = make_uint2(0x3F803F80u, 0x3F803F80u); }
__device__ __forceinline__ void ones(Frag4<float>& f) { f.v = make_float4(1.f, 1.f, 1.f, 1.f); }

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as
// easy as 1, 2, 3", SC 2011): ten rounds of two 32 x 32 -> 64-bit products
// with the multipliers 0xD2511F53 and 0xCD9E8D57, the key bumped by the Weyl
// constants 0x9E3779B9 and 0xBB67AE85 between rounds.
struct U32x4 {
  uint32_t x, y, z, w;
};
__device__ __forceinline__ U32x4 philox4x32_10(U32x4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint32_t hi0 = __umulhi(0xD2511F53u, c.x), lo0 = 0xD2511F53u * c.x;
    const uint32_t hi1 = __umulhi(0xCD9E8D57u, c.z), lo1 = 0xCD9E8D57u * c.z;
    c = U32x4{hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0};
  }
  return c;
}

// Gumbel noise from a 32-bit draw: u = (top 23 bits + 1/2) / 2^23, strictly
// inside (0, 1) and exact in binary32, then g = -log(-log u). t = -ln u needs
// relative accuracy down to 2^-24 (u next to 1: the largest noise). For
// e = 1 - u < 1/16 (exact: u >= 1/2) it comes from the series
// e + e^2/2 + ... + e^6/6 (truncation below e^7/7, relative 2^-24 / 7); further
// from 1 the hardware log2 is accurate relative to the result. The outer
// logarithm only needs absolute accuracy (its value is the noise), which the
// hardware log2 gives.
__device__ __forceinline__ float gumbel_of(uint32_t w) {
  const float u = ((float)(w >> 9) + 0.5f) * 0x1p-23f;
  const float e = 1.0f - u;
  const float ts = e * (1.0f + e * (0.5f + e * (0.333333343f + e * (0.25f + e * (0.200000003f + e * 0.166666672f)))));
  const float tl = -__builtin_amdgcn_logf(u) * 0.693147180559945309f;
  const float t = e < 0.0625f ? ts : tl;
  return -__builtin_amdgcn_logf(t) * 0.693147180559945309f;
}

// page format (see include/mcpu.h)
// ---------------------------------------------------------------------------

constexpr int PAGE = 16;

__device__ __forceinline__ int k_off(int s, int i) { return ((i >> 3) * PAGE + s) * 8 + (i & 7); }
__device__ __forceinline__ int v_off(int s, int i) {
  return (((i >> 4) * (PAGE / 4) + (s >> 2)) * 16 + (i & 15)) * 4 + (s & 3);
}

__device__ __forceinline__ void set_error(int32_t* err, int bit) {
  if (err) atomicOr(err, bit);
}

}  // namespace mcpu
