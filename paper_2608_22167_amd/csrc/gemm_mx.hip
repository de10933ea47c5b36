// Grouped GEMM on gfx950's scaled matrix cores: MXFP8 (E4M3) activations
// times MXFP4 (E2M1) weights, both with E8M0 scales per 32 elements along the
// reduction, accumulated in fp32 (v_mfma_scale_f32_32x32x64_f8f6f4). Used
// for the native-MXFP4 experts of prefill-sized steps, where the bf16 path
// (weights decoded to bf16 before bf16 products) is bound by the matrix cores.
//
// Operand layout of one 32 x 32 x 64 product (lane l, g = l / 32; measured):
//   A (fp8, 32 bytes): row l % 32; bytes 0-15 hold k = 16 g .. 16 g + 15,
//     bytes 16-31 hold k = 32 + 16 g .. 32 + 16 g + 15;
//   B (fp4, 16 bytes, low nibble first): column l % 32, k = 32 g .. 32 g + 31;
//   scales: lane l supplies A's scale of (row l % 32, block g) and B's of
//     (column l % 32, block g), in byte 0;
//   C: element j of lane l is (row 8 (j / 4) + 4 g + j % 4, column l % 32).
// So each lane's A bytes are two 16-byte halves of a staged 64-byte row
// slice and its B bytes one 16-byte quarter of a 32-byte slice.
//
// Tile 256 token rows x 256 weight rows, eight wavefronts (4 x 2), each
// owning 64 x 128 = 2 x 4 products of 32 x 32. The reduction runs in slices
// of 64 (one product deep) through a ring of six LDS stages that 16-byte
// buffer loads fill straight from global memory (a wavefront's load fills
// 1 KB of LDS, lane l at byte 16 l), so staging costs neither registers nor
// LDS write instructions. Every operand is in slice order (kernels.h), so a
// slice of the tile is four contiguous runs: 16 KB of activation codes, 8 KB
// of weight codes and 1 KB of scale dwords each, read as whole cache lines.
// While slice i is multiplied, the fragments of slice i + 1 are read, and
// slice i + 5 is requested into the stage slice i - 1 left; before each
// barrier a wavefront waits for its own loads of slice i + 2, which the
// barrier then publishes (three slices stay in flight across it).
//   Stage layout: token rows 64 B (chunk q of row r in slot q ^ ((r >> 1) & 3)),
// weight rows 32 B (chunk q in slot q ^ (((r >> 2) ^ (r >> 3)) & 1)), which
// keeps the fragment reads free of bank conflicts, then the token rows' and
// the weight rows' scale dwords (1 KB each: wavefronts 0-3 load the former,
// 4-7 the latter, so every wavefront issues the same four loads per slice).
// The finished fp32 tile goes through LDS to the fused epilogue
// (gemm_epilogue.h), 16 rows at a time.
#include <type_traits>

#include "device.h"
#include "gemm_epilogue.h"
#include "kernels.h"

namespace mcpu {
namespace {

typedef int32_t v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;

constexpr int XM = 256, XN = 256, XK = 64;  // output tile, reduction per slice
constexpr int XTH = 512;
constexpr int XS_A = XM * XK, XS_B = XN * XK / 2, XS_S = 4 * (XM + XN);
constexpr int XSTAGE = XS_A + XS_B + XS_S;  // 26 KB
constexpr int XEP = 16, XCLD = XN + 4;      // epilogue pass rows, fp32 row stride
static_assert(XEP * XCLD * 4 <= XSTAGE, "an epilogue pass fits one stage");
static_assert(6 * XSTAGE + 4 * (TILE_MAXG + 1) <= 160 * 1024, "LDS");
constexpr int XGM = 2;                      // m-tiles per band
constexpr int XBUF_DWORD3 = 0x00020000;     // raw buffer descriptor word 3 (gfx9 family)

__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }
__device__ __forceinline__ int swz_a(int r) { return (r >> 1) & 3; }
__device__ __forceinline__ int swz_b(int r) { return ((r >> 2) ^ (r >> 3)) & 1; }
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const uint8_t* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(base), 0, 0x7FFFFFFF, XBUF_DWORD3);
}

// MXFP8 quantization of bf16 rows (OCP MX v1.0): the block's scale is
// 2^(floor(log2 amax) - 8) as E8M0, the elements v / scale rounded to
// nearest-even E4M3 with saturation at +-448; an all-zero block gets scale
// byte 0. v / scale is exact (a power-of-two scaling of a bf16 value), and
// the hardware's packed conversion rounds it to nearest even; it gives NaN
// above 448, so values are clamped to +-448 first, and it keeps the sign of a
// negative value that rounds to zero (0x80), which becomes code 0. (Checked
// against a bit-arithmetic encoder over every bf16 value times 2^-24 .. 2^12.)
__device__ __forceinline__ float sat448(float x) { return fminf(fmaxf(x, -448.f), 448.f); }
__device__ __forceinline__ uint32_t e4m3x4(float a0, float a1, float a2, float a3) {
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(sat448(a0), sat448(a1), 0, false);  // bytes 0, 1
  w = __builtin_amdgcn_cvt_pk_fp8_f32(sat448(a2), sat448(a3), w, true);       // bytes 2, 3
  const uint32_t u = (uint32_t)w, t = u ^ 0x80808080u;
  const uint32_t z = ~(((t & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | t) & 0x80808080u;  // bytes that are 0x80
  return u & ~z;
}

// The gate/up product's epilogue with MXFP8 output: 16 rows x 128 SwiGLU
// columns per pass, four consecutive columns per thread; eight threads hold a
// 32-column block, whose maximum they reduce by shuffles. Each value is the
// bf16-rounded SwiGLU output (the value the unfused path stores), quantized
// exactly as mx_quant_kernel does, and written in slice order.
// A thread's eight gate/up biases, the same in every pass: loaded once per tile.
struct MxBias {
  float4 b0, b1;
};
__device__ __forceinline__ MxBias swiglu_mx_bias(const Gemm& P, int n0, int nrows, int grp) {
  MxBias b{make_float4(0.f, 0.f, 0.f, 0.f), make_float4(0.f, 0.f, 0.f, 0.f)};
  const int q = threadIdx.x & 31;
  if (8 * q < nrows) {
    const float* bias = P.bias + (int64_t)grp * P.bias_group_stride + n0 + 8 * q;
    b.b0 = *reinterpret_cast<const float4*>(bias);
    b.b1 = *reinterpret_cast<const float4*>(bias + 4);
  }
  return b;
}

__device__ __forceinline__ void swiglu_mx_pass(const Gemm& P, const float* cr, int ld, int row0, int mrows, int n0,
                                               int nrows, const MxBias& bb) {
  const int tid = threadIdx.x;
  const int m = tid >> 5, q = tid & 31;  // row of the pass, 4-column group
  // all eight threads of a block agree (n is a multiple of 64)
  const bool valid = m < mrows && 8 * q < nrows;
  const float4 b0 = bb.b0, b1 = bb.b1;
  const float* c = cr + m * ld + 8 * q;
  float a[4];
  a[0] = swiglu(c[0] + b0.x, c[1] + b0.y, P.swiglu_alpha, P.swiglu_limit, P.swiglu_beta);
  a[1] = swiglu(c[2] + b0.z, c[3] + b0.w, P.swiglu_alpha, P.swiglu_limit, P.swiglu_beta);
  a[2] = swiglu(c[4] + b1.x, c[5] + b1.y, P.swiglu_alpha, P.swiglu_limit, P.swiglu_beta);
  a[3] = swiglu(c[6] + b1.z, c[7] + b1.w, P.swiglu_alpha, P.swiglu_limit, P.swiglu_beta);
  float amax = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    a[i] = bf16_to_f32(f32_to_bf16(a[i]));
    amax = fmaxf(amax, fabsf(a[i]));
  }
  // the block's maximum over its eight threads (lanes 8 r .. 8 r + 7)
#pragma unroll
  for (int d = 1; d < 8; d <<= 1) amax = fmaxf(amax, __shfl_xor(amax, d, 64));
  int e = -127;
  if (amax > 0.f) {
    e = (int)((__float_as_uint(amax) >> 23) & 0xFF) - 127 - 8;
    e = max(-127, min(127, e));
  }
  const float inv = __uint_as_float((uint32_t)(127 - e) << 23);
  const uint32_t w = e4m3x4(a[0] * inv, a[1] * inv, a[2] * inv, a[3] * inv);
  if (!valid) return;
  const int64_t R = P.n_rows, row = row0 + m;
  const int k = n0 / 2 + 4 * q;  // SwiGLU column
  *reinterpret_cast<uint32_t*>(reinterpret_cast<uint8_t*>(P.out) + ((int64_t)(k / 64) * R + row) * 64 + k % 64) = w;
  if ((q & 7) == 0) P.out_scales[((int64_t)(k / 128) * R + row) * 4 + (k / 32) % 4] = (uint8_t)(e + 127);
}

template <int EPI>
__global__ __launch_bounds__(XTH) void gemm_mx_kernel(Gemm P) {
  __shared__ __align__(1024) uint8_t d0[XSTAGE];
  __shared__ __align__(1024) uint8_t d1[XSTAGE];
  __shared__ __align__(1024) uint8_t d2[XSTAGE];
  __shared__ __align__(1024) uint8_t d3[XSTAGE];
  __shared__ __align__(1024) uint8_t d4[XSTAGE];
  __shared__ __align__(1024) uint8_t d5[XSTAGE];
  __shared__ int mt_start[TILE_MAXG + 1];
  const int tid = threadIdx.x, lane = tid & 63, wave = uniform(tid >> 6);

  int grp, mt, tn;
  if (!tile_of_block<XM, XN, XGM>(P, mt_start, grp, mt, tn)) return;
  const int gr0 = P.group_off ? P.group_off[grp] : 0;
  const int gr1 = P.group_off ? P.group_off[grp + 1] : P.n_rows;
  const int m0 = uniform(gr0 + mt * XM);
  const int mrows = min(XM, gr1 - m0);
  const int n0 = uniform(tn * XN), nrows = min(XN, P.n - n0);
  const int K = P.k, N = P.n, nk = K / XK;
  const int xrows = P.x_rows > 0 ? P.x_rows : P.n_rows;

  // Loads of a slice: wavefront w fills token rows 32 w + 16 j + [0, 16)
  // (j = 0, 1; lane l lands in row + l / 4, slot l % 4), weight rows
  // 32 w + [0, 32) (lane l in row l / 2, slot l % 2), and the scale dwords of
  // token rows 64 w + [0, 64) (w < 4) or of weight rows 64 (w - 4) + [0, 64);
  // each lane loads the global chunk its slot holds. Token rows past the tile's end read the next x rows
  // (the last one at the end of x), weight rows past n repeat the last one;
  // their results are dropped. Buffer loads: per-slice bases, 32-bit per-lane
  // row offsets.
  const uint8_t* xq = reinterpret_cast<const uint8_t*>(P.x);
  const uint8_t* wq = reinterpret_cast<const uint8_t*>(P.w) + grp * P.w_group_stride;
  const uint8_t* ws = P.w_scales + grp * mx_scale_bytes(N, K);
  uint32_t avo[2], bvo, svo;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int r = 32 * wave + 16 * j + (lane >> 2);
    avo[j] = (uint32_t)min(m0 + r, xrows - 1) * 64u + 16u * ((lane & 3) ^ swz_a(r));
  }
  {
    const int r = 32 * wave + (lane >> 1);
    bvo = (uint32_t)(n0 + min(r, nrows - 1)) * 32u + 16u * ((lane & 1) ^ swz_b(r));
    const int q = 64 * (wave & 3) + lane;
    svo = wave < 4 ? (uint32_t)min(m0 + q, xrows - 1) * 4u : (uint32_t)(n0 + min(q, nrows - 1)) * 4u;
  }

  auto stage_of = [&](int s) __attribute__((always_inline)) {
    return s == 0 ? d0 : s == 1 ? d1 : s == 2 ? d2 : s == 3 ? d3 : s == 4 ? d4 : d5;
  };
  // the loads of slice ks into a stage (4 per wavefront); slices past the
  // end re-read the last one (never multiplied), so every slice issues the
  // same loads and the waits below count whole slices
  auto dma = [&](uint8_t* stg, int ks) __attribute__((always_inline)) {
    ks = uniform(min(ks, nk - 1));
    const __amdgpu_buffer_rsrc_t xr = rsrc(xq + (size_t)ks * xrows * 64);
    const __amdgpu_buffer_rsrc_t wr = rsrc(wq + (size_t)ks * N * 32);
    const __amdgpu_buffer_rsrc_t sr = wave < 4 ? rsrc(P.x_scales + (size_t)(ks >> 1) * xrows * 4)
                                               : rsrc(ws + (size_t)(ks >> 1) * N * 4);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_ptr_t)(stg + 32 * wave * 64), 16, avo[0], 0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_ptr_t)(stg + (32 * wave + 16) * 64), 16, avo[1], 0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (lds_ptr_t)(stg + XS_A + 32 * wave * 32), 16, bvo, 0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(sr, (lds_ptr_t)(stg + XS_A + XS_B + 256 * wave), 4, svo, 0, 0, 0);
  };
  // wait until at most this wavefront's three newest slices are in flight
  // (and its LDS reads are done), then the barrier that publishes everyone's
  // older slices
  auto publish = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(12 | (7 << 4));  // vmcnt(12) expcnt(7) lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
  };

  // wavefront (wm, wn): token rows wm * 64 + [0, 64), weight rows wn * 128 + [0, 128)
  const int wm = wave >> 1, wn = wave & 1;
  const int fr = lane & 31, fg = lane >> 5;
  // per-lane fragment offsets within a stage: token-row halves h = 0, 1 of
  // product 0 (product 1 is 32 rows = 2 KB further), weight rows of product 0
  // (product ct is 1 KB further), the scale bytes (the next 32 rows' dwords
  // are 128 B further)
  uint32_t a0, a1, b0, q0, p0;
  {
    const int r = wm * 64 + fr;
    a0 = r * 64 + 16 * (fg ^ swz_a(r));
    a1 = r * 64 + 16 * ((2 + fg) ^ swz_a(r));
    q0 = XS_A + XS_B + 4 * r + fg;
    const int rb = wn * 128 + fr;
    b0 = XS_A + rb * 32 + 16 * (fg ^ swz_b(rb));
    p0 = XS_A + XS_B + 4 * XM + 4 * rb + fg;
  }
  struct Frag {
    u32x4 a[2][2], b[4];
    int sa[2], sb[4];
  };
  // fragments of a slice of parity PAR from a stage; the offsets pass through
  // an empty asm statement so that the stage addresses are formed per slice
  // rather than kept in registers for all five stages
  auto read = [&](Frag& f, const uint8_t* stg, auto PAR_) __attribute__((always_inline)) {
    constexpr int PAR = decltype(PAR_)::value;
    asm volatile("" : "+v"(a0), "+v"(a1), "+v"(b0), "+v"(q0), "+v"(p0));
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      f.a[rt][0] = ld16(stg + a0 + 2048 * rt);
      f.a[rt][1] = ld16(stg + a1 + 2048 * rt);
      f.sa[rt] = stg[q0 + 128 * rt + 2 * PAR];
    }
#pragma unroll
    for (int ct = 0; ct < 4; ++ct) {
      f.b[ct] = ld16(stg + b0 + 1024 * ct);
      f.sb[ct] = stg[p0 + 128 * ct + 2 * PAR];
    }
  };
  v16f acc[2][4];
#pragma unroll
  for (int rt = 0; rt < 2; ++rt)
#pragma unroll
    for (int ct = 0; ct < 4; ++ct)
#pragma unroll
      for (int j = 0; j < 16; ++j) acc[rt][ct][j] = 0.f;
  auto mfma = [&](const Frag& f) __attribute__((always_inline)) {
#pragma unroll
    for (int rt = 0; rt < 2; ++rt) {
      union {
        v8i v;
        u32x4 h[2];
      } a;
      a.h[0] = f.a[rt][0];
      a.h[1] = f.a[rt][1];
#pragma unroll
      for (int ct = 0; ct < 4; ++ct) {
        union {
          v8i v;
          u32x4 h[2];
        } b;
        b.h[0] = f.b[ct];
        b.h[1] = u32x4{0u, 0u, 0u, 0u};
        acc[rt][ct] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a.v, b.v, acc[rt][ct], 0, 4, 0, f.sa[rt], 0,
                                                                      f.sb[ct]);
      }
    }
  };

  // prologue: slices 0 .. 4 requested, 0 and 1 published, slice 0 read
#pragma unroll
  for (int s = 0; s < 5; ++s) dma(stage_of(s), s);
  publish();
  Frag fa[2];
  read(fa[0], d0, std::integral_constant<int, 0>{});

  // slice i uses stage i % 6 and fragment set i % 2 (the loop is unrolled
  // six times); the fragments read past the last slice are never used
  auto slice = [&](auto S_, auto H_, int i) __attribute__((always_inline)) {
    constexpr int S = decltype(S_)::value, H = decltype(H_)::value;
    __builtin_amdgcn_sched_barrier(0);  // nothing moves between slices
    dma(stage_of((S + 5) % 6), i + 5);
    read(fa[H ^ 1], stage_of((S + 1) % 6), std::integral_constant<int, H ^ 1>{});
    mfma(fa[H]);
    publish();
  };
  using C0 = std::integral_constant<int, 0>;
  using C1 = std::integral_constant<int, 1>;
  using C2 = std::integral_constant<int, 2>;
  using C3 = std::integral_constant<int, 3>;
  using C4 = std::integral_constant<int, 4>;
  using C5 = std::integral_constant<int, 5>;
  int i = 0;
  for (; i + 6 <= nk; i += 6) {
    slice(C0{}, C0{}, i);
    slice(C1{}, C1{}, i + 1);
    slice(C2{}, C0{}, i + 2);
    slice(C3{}, C1{}, i + 3);
    slice(C4{}, C0{}, i + 4);
    slice(C5{}, C1{}, i + 5);
  }
  if (i < nk) slice(C0{}, C0{}, i);
  if (i + 1 < nk) slice(C1{}, C1{}, i + 1);
  if (i + 2 < nk) slice(C2{}, C0{}, i + 2);
  if (i + 3 < nk) slice(C3{}, C1{}, i + 3);
  if (i + 4 < nk) slice(C4{}, C0{}, i + 4);
  __builtin_amdgcn_s_waitcnt(0);  // every load landed and every read done before stage 0 holds the fp32 tile
  __syncthreads();

  // acc[rt][ct][j] = C[m = wm*64 + 32 rt + 8 (j/4) + 4 fg + j%4][n = wn*128 + 32 ct + fr]
  float* cr = reinterpret_cast<float*>(d0);
  EpiBias eb{};
  MxBias mb{};
  if constexpr (EPI == EPI_SWIGLU_MX) mb = swiglu_mx_bias(P, n0, nrows, grp);
  else eb = epilogue_bias<EPI>(P, n0 >> 4, nrows >> 4, grp);
  for (int e0 = 0; e0 < XM; e0 += XEP) {
    if (e0 >= mrows) break;  // uniform
    if (wm == e0 / 64) {
      const int q = (e0 % 64) / 16;  // product rt = q / 2, its rows 16 (q % 2) + [0, 16)
#pragma unroll
      for (int qq = 0; qq < 4; ++qq)
        if (qq == q) {
#pragma unroll
          for (int ct = 0; ct < 4; ++ct)
#pragma unroll
            for (int j = 8 * (qq & 1); j < 8 * (qq & 1) + 8; ++j)
              cr[(8 * (j >> 2) + 4 * fg + (j & 3) - 16 * (qq & 1)) * XCLD + wn * 128 + ct * 32 + fr] = acc[qq >> 1][ct][j];
        }
    }
    __syncthreads();
    if constexpr (EPI == EPI_SWIGLU_MX) swiglu_mx_pass(P, cr, XCLD, m0 + e0, min(XEP, mrows - e0), n0, nrows, mb);
    else epilogue<bf16, EPI>(P, cr, XCLD, m0 + e0, min(XEP, mrows - e0), n0 >> 4, nrows >> 4, grp, &eb);
    __syncthreads();
  }
}

// bf16 rows to MXFP8: a thread per block of 32 consecutive elements (16-byte
// loads), the block maximum, the E8M0 exponent from the binary32 exponent
// field, four codes per conversion; the codes and the scale go to each of the
// row's output copies.
__global__ __launch_bounds__(256) void mx_quant_kernel(MxQuant P) {
  const int64_t blk = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int per_row = P.cols / 32;
  if (blk >= (int64_t)P.rows * per_row) return;
  const int64_t row = blk / per_row;
  const int c0 = (int)(blk - row * per_row) * 32;
  const bf16* src = reinterpret_cast<const bf16*>(P.in) + row * P.cols + c0;
  float v[32];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const u32x4 w = ld16(src + 8 * q);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[8 * q + 2 * i] = __uint_as_float(w[i] << 16);
      v[8 * q + 2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
  float amax = 0.f;
#pragma unroll
  for (int i = 0; i < 32; ++i) amax = fmaxf(amax, fabsf(v[i]));
  int e = -127;
  if (amax > 0.f) {
    // floor(log2 amax): the binary32 exponent field (bf16 values are normal here)
    e = (int)((__float_as_uint(amax) >> 23) & 0xFF) - 127 - 8;
    e = max(-127, min(127, e));
  }
  const float inv = __uint_as_float((uint32_t)(127 - e) << 23);  // 2^-e, a normal power of two for e in [-127, 119]
  uint32_t out[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) out[q] = e4m3x4(v[4 * q] * inv, v[4 * q + 1] * inv, v[4 * q + 2] * inv, v[4 * q + 3] * inv);
  // the GEMM operand layout: 64-column slices of all rows in turn, the four
  // scale bytes of a row's 128 columns in one dword
  for (int c = 0; c < P.copies; ++c) {
    const int64_t dst_row = P.row_dst ? P.row_dst[row * P.copies + c] : row;
    const int64_t sidx = P.gemm_layout ? ((int64_t)(c0 / 128) * P.out_rows + dst_row) * 4 + (c0 / 32) % 4
                                       : dst_row * per_row + c0 / 32;
    P.scales[sidx] = (uint8_t)(e + 127);
    uint8_t* dst = P.codes + (P.gemm_layout ? ((int64_t)(c0 / 64) * P.out_rows + dst_row) * 64 + c0 % 64
                                            : dst_row * P.cols + c0);
    st16(dst, u32x4{out[0], out[1], out[2], out[3]});
    st16(dst + 16, u32x4{out[4], out[5], out[6], out[7]});
  }
}

// MXFP4 weights into slice order: a thread per (group, row, block of 32):
// 16 code bytes to their 64-column slice, the scale byte to its dword; the
// unused bytes of a last, partial dword get 127 (scale 1)
__global__ __launch_bounds__(256) void mx_pack_kernel(MxPack P) {
  const int kb = P.cols / 32, kq = (kb + 3) / 4;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)P.groups * P.rows * kq * 4) return;
  const int b = (int)(t % (kq * 4));
  const int64_t gr = t / (kq * 4);  // group * rows + row
  const int g = (int)(gr / P.rows), r = (int)(gr - (int64_t)g * P.rows);
  uint8_t* ds = P.dst + mx_packed_codes_bytes(P.groups, P.rows, P.cols) +
                ((int64_t)g * kq + b / 4) * P.rows * 4 + (int64_t)r * 4 + b % 4;
  if (b >= kb) {
    *ds = 127;
    return;
  }
  *ds = P.scales[gr * kb + b];
  const u32x4 c = ld16(P.codes + gr * (P.cols / 2) + 16 * b);
  st16(P.dst + (((int64_t)g * (P.cols / 64) + b / 2) * P.rows + r) * 32 + 16 * (b % 2), c);
}

}  // namespace

bool mx_gemm_applies(const Gemm& g) {
  // buffer loads address a slice's rows with 32-bit offsets below 2^31
  const int64_t xr = g.x_rows > 0 ? g.x_rows : g.n_rows;
  return g.k > 0 && g.k % 64 == 0 && g.n % 16 == 0 && g.n_groups <= TILE_MAXG && g.x_scales && g.w_scales &&
         !g.row_src && (uintptr_t)g.x % 16 == 0 && (uintptr_t)g.w % 16 == 0 && (uintptr_t)g.x_scales % 4 == 0 &&
         (uintptr_t)g.w_scales % 4 == 0 && xr * 64 < (1LL << 31) && g.w_group_stride == (int64_t)g.n * g.k / 2;
}

hipError_t launch_gemm_mx(const Gemm& g, hipStream_t s) {
  if (!mx_gemm_applies(g)) return hipErrorInvalidValue;
  const int64_t grid = tile_grid(g, XM, XN);
  if (grid > 0x7FFFFFFF) return hipErrorInvalidValue;
  dim3 gd((unsigned)grid), bd(XTH);
  switch (g.epi) {
    case EPI_SWIGLU: hipLaunchKernelGGL((gemm_mx_kernel<EPI_SWIGLU>), gd, bd, 0, s, g); break;
    case EPI_BIAS: hipLaunchKernelGGL((gemm_mx_kernel<EPI_BIAS>), gd, bd, 0, s, g); break;
    case EPI_SWIGLU_MX:
      // whole 32-column blocks of SwiGLU output in every tile
      if (g.n % 64 || !g.out_scales || g.n_rows <= 0) return hipErrorInvalidValue;
      hipLaunchKernelGGL((gemm_mx_kernel<EPI_SWIGLU_MX>), gd, bd, 0, s, g);
      break;
    default: return hipErrorNotSupported;
  }
  return hipGetLastError();
}

hipError_t launch_mx_pack(const MxPack& p, hipStream_t s) {
  if (p.groups <= 0 || p.rows <= 0 || p.cols <= 0 || p.cols % 64) return hipErrorInvalidValue;
  const int64_t n = (int64_t)p.groups * p.rows * ((p.cols / 32 + 3) / 4) * 4;
  hipLaunchKernelGGL(mx_pack_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p);
  return hipGetLastError();
}

hipError_t launch_mx_quant(const MxQuant& p, hipStream_t s) {
  if (p.rows == 0) return hipSuccess;
  if (p.cols % 32) return hipErrorInvalidValue;
  const int64_t blocks = (int64_t)p.rows * (p.cols / 32);
  hipLaunchKernelGGL(mx_quant_kernel, dim3((unsigned)((blocks + 255) / 256)), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace mcpu
