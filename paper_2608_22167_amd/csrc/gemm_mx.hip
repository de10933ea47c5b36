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
// Tile 256 token rows x 256 weight rows, eight wavefronts (2 x 4), each
// owning 128 x 64 = 4 x 2 products of 32 x 32; the reduction runs in stages
// of 128 (two products deep) through two LDS buffers, one barrier per stage.
// LDS rows are 160 B (A, 128 B of data) and 96 B (B, 64 B) apart, which keeps
// the 16-byte fragment reads free of bank conflicts. Scales: the activation
// rows' four scale bytes of a stage are one dword (the operand layout groups
// them so), staged with the codes; the tile's weight scales, a contiguous run
// of 256 rows, are copied to LDS once and read from there for the whole
// reduction, so no scale byte costs a separate memory request. The finished
// fp32 tile goes through LDS to the fused epilogue (gemm_epilogue.h), 32 rows
// at a time.
#include <type_traits>

#include "device.h"
#include "gemm_epilogue.h"
#include "kernels.h"

namespace mcpu {
namespace {

typedef int32_t v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int XM = 256, XN = 256, XK = 128;  // output tile, reduction per stage
constexpr int XTH = 512;
constexpr int XA_LD = 160, XB_LD = 96;       // staged row strides (bytes)
constexpr int XA_BYTES = XM * XA_LD, XB_BYTES = XN * XB_LD;
constexpr int XSTAGE = XA_BYTES + XB_BYTES + 4 * XM;  // + the token rows' scale dwords
constexpr int XBS_BYTES = XN * (MX_MAX_K / 32);       // the tile's weight scales
constexpr int XEP = 32, XCLD = XN + 4;       // epilogue pass rows, fp32 row stride
static_assert(XEP * XCLD * 4 <= XSTAGE, "an epilogue pass fits one stage");
static_assert(2 * XSTAGE + XBS_BYTES + 4 * (TILE_MAXG + 1) <= 160 * 1024, "LDS");
constexpr int XGM = 2;                       // m-tiles per band

__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }

template <int EPI>
__global__ __launch_bounds__(XTH) void gemm_mx_kernel(Gemm P) {
  __shared__ __align__(16) uint8_t lds[2 * XSTAGE + XBS_BYTES];
  __shared__ int mt_start[TILE_MAXG + 1];
  const int tid = threadIdx.x, lane = tid & 63, wave = uniform(tid >> 6);

  int grp, mt, tn;
  if (!tile_of_block<XM, XN, XGM>(P, mt_start, grp, mt, tn)) return;
  const int gr0 = P.group_off ? P.group_off[grp] : 0;
  const int gr1 = P.group_off ? P.group_off[grp + 1] : P.n_rows;
  const int m0 = uniform(gr0 + mt * XM);
  const int mrows = min(XM, gr1 - m0);
  const int n0 = uniform(tn * XN), nrows = min(XN, P.n - n0);
  const int K = P.k, kb32 = K / 32, lda = mx_code_stride(K);
  const uint32_t xrows = (uint32_t)(P.x_rows > 0 ? P.x_rows : P.n_rows);

  // staging: A chunk c = tid + 512 j (j < 4) is row c / 8, 16-byte piece c % 8;
  // B chunk c = tid + 512 j (j < 2) is row c / 4, piece c % 4; threads 0-255
  // stage the scale dword of token row tid. Rows past the tile's end repeat
  // its last row (results dropped). Token rows, one expert's weights and the
  // scale rows are addressed by 32-bit offsets from uniform bases (the host
  // checks that they fit).
  const uint8_t* xq = reinterpret_cast<const uint8_t*>(P.x);
  const uint8_t* wq = reinterpret_cast<const uint8_t*>(P.w) + grp * P.w_group_stride;
  const uint8_t* ws = P.w_scales + grp * (P.w_group_stride / 16) + (uint32_t)n0 * (uint32_t)kb32;
  const uint32_t a_piece = 16u * (tid & 7), b_piece = 16u * (tid & 3);
  uint32_t a_off[4], b_off[2], s_row;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int r = (tid + XTH * j) >> 3;
    const int row = m0 + min(r, mrows - 1);
    const int src = P.row_src ? P.row_src[row] : row;
    a_off[j] = (uint32_t)src * (uint32_t)lda;
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int r = (tid + XTH * j) >> 2;
    b_off[j] = (uint32_t)(n0 + min(r, nrows - 1)) * (uint32_t)(K / 2);
  }
  {
    const int row = m0 + min(tid & 255, mrows - 1);
    s_row = (uint32_t)(P.row_src ? P.row_src[row] : row);
  }

  // the tile's weight scales [256 rows][kb32] into LDS (rows past the end
  // get scale 1; the run is a multiple of 16 bytes since n is of 16)
  uint8_t* bsc = lds + 2 * XSTAGE;
  {
    const int span = nrows * kb32;
    const u32x4 one = {0x7F7F7F7Fu, 0x7F7F7F7Fu, 0x7F7F7F7Fu, 0x7F7F7F7Fu};
    for (int c = 16 * tid; c < XN * kb32; c += 16 * XTH) st16(bsc + c, c < span ? ld16(ws + c) : one);
  }

  struct Regs {
    u32x4 a[4], b[2];
    uint32_t s;
  };
  // Past the end of the reduction (a last stage of 64) the pieces are zero:
  // the load address is clamped into the row and the value replaced, so no
  // load is conditional and none leaves the row; scale bytes past the end
  // become 1.
  auto fetch = [&](Regs& g, int st) __attribute__((always_inline)) {
    const int k0 = st * XK;
    const u32x4 z = {0u, 0u, 0u, 0u};
    const int ka = k0 + (int)a_piece, kb = k0 / 2 + (int)b_piece;  // byte offsets in a row
    const uint32_t ka_c = (uint32_t)min(ka, K - 16), kb_c = (uint32_t)min(kb, K / 2 - 16);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const u32x4 v = ld16(xq + (a_off[j] + ka_c));
      g.a[j] = ka < K ? v : z;
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const u32x4 v = ld16(wq + (b_off[j] + kb_c));
      g.b[j] = kb < K / 2 ? v : z;
    }
    if (tid < 256) {
      uint32_t s = *reinterpret_cast<const uint32_t*>(P.x_scales + ((uint32_t)st * xrows + s_row) * 4u);
      const int valid = kb32 - 4 * st;  // uniform
      if (valid < 4) {
        const uint32_t keep = (1u << (8 * valid)) - 1u;
        s = (s & keep) | (0x7F7F7F7Fu & ~keep);
      }
      g.s = s;
    }
  };
  auto store = [&](const Regs& g, uint8_t* stage) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < 4; ++j) st16(stage + ((tid + XTH * j) >> 3) * XA_LD + a_piece, g.a[j]);
#pragma unroll
    for (int j = 0; j < 2; ++j) st16(stage + XA_BYTES + ((tid + XTH * j) >> 2) * XB_LD + b_piece, g.b[j]);
    if (tid < 256) *reinterpret_cast<uint32_t*>(stage + XA_BYTES + XB_BYTES + 4 * tid) = g.s;
  };

  // wavefront (wm, wn): token rows wm * 128 + [0, 128), weight rows wn * 64 + [0, 64)
  const int wm = wave >> 2, wn = wave & 3;
  const int fr = lane & 31, fg = lane >> 5;
  v16f acc[4][2];
#pragma unroll
  for (int rt = 0; rt < 4; ++rt)
#pragma unroll
    for (int ct = 0; ct < 2; ++ct)
#pragma unroll
      for (int j = 0; j < 16; ++j) acc[rt][ct][j] = 0.f;

  // the two product depths of stage st, one at a time (the next depth's
  // fragments are not read ahead: their registers would spill the accumulators)
  auto compute = [&](const uint8_t* stage, int st) __attribute__((always_inline)) {
    const uint8_t* sa = stage + XA_BYTES + XB_BYTES;
#pragma unroll 1
    for (int ks = 0; ks < 2; ++ks) {
      union Op {
        v8i v;
        u32x4 h[2];
      };
      Op a[4], b[2];
      int sca[4], scb[2];
      const int blk = min(4 * st + 2 * ks + fg, kb32 - 1);
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) {
        const int row = wm * 128 + rt * 32 + fr;
        const uint8_t* p = stage + row * XA_LD + 64 * ks + 16 * fg;
        a[rt].h[0] = ld16(p);
        a[rt].h[1] = ld16(p + 32);
        sca[rt] = sa[row * 4 + 2 * ks + fg];
      }
#pragma unroll
      for (int ct = 0; ct < 2; ++ct) {
        const int row = wn * 64 + ct * 32 + fr;
        b[ct].h[0] = ld16(stage + XA_BYTES + row * XB_LD + 32 * ks + 16 * fg);
        b[ct].h[1] = u32x4{0u, 0u, 0u, 0u};
        scb[ct] = bsc[row * kb32 + blk];
      }
#pragma unroll
      for (int rt = 0; rt < 4; ++rt)
#pragma unroll
        for (int ct = 0; ct < 2; ++ct)
          acc[rt][ct] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a[rt].v, b[ct].v, acc[rt][ct], 0, 4, 0,
                                                                        sca[rt], 0, scb[ct]);
    }
  };

  // Stage s is multiplied out of LDS buffer s % 2 while stage s + 1 is
  // loaded into registers and then written to the other buffer; one barrier
  // per stage.
  const int ns = (K + XK - 1) / XK;
  {
    Regs r;
    fetch(r, 0);
    store(r, lds);
  }
  __syncthreads();
  for (int s = 0; s < ns; ++s) {
    uint8_t* cur = lds + (s & 1) * XSTAGE;
    uint8_t* nxt = lds + ((s + 1) & 1) * XSTAGE;
    Regs r;
    const bool more = s + 1 < ns;  // uniform
    if (more) fetch(r, s + 1);
    // a last stage of 64 (k % 128 == 64) has its second half zero-filled: its
    // products add zero, and one code path keeps the accumulators in place
    compute(cur, s);
    if (more) store(r, nxt);
    __syncthreads();
  }

  // acc[rt][ct][j] = C[m = wm*128 + 32 rt + 8 (j/4) + 4 fg + j%4][n = wn*64 + 32 ct + fr];
  // the fp32 tile goes through LDS (buffer 0, free after the last barrier)
  float* cr = reinterpret_cast<float*>(lds);
  const EpiBias eb = epilogue_bias<EPI>(P, n0 >> 4, nrows >> 4, grp);
  for (int e0 = 0; e0 < XM; e0 += XEP) {
    if (e0 >= mrows) break;  // uniform
    if (wm == e0 / 128) {
      const int rt = (e0 % 128) / 32;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (q == rt) {
#pragma unroll
          for (int ct = 0; ct < 2; ++ct)
#pragma unroll
            for (int j = 0; j < 16; ++j)
              cr[(8 * (j >> 2) + 4 * fg + (j & 3)) * XCLD + wn * 64 + ct * 32 + fr] = acc[q][ct][j];
        }
    }
    __syncthreads();
    epilogue<bf16, EPI>(P, cr, XCLD, m0 + e0, min(XEP, mrows - e0), n0 >> 4, nrows >> 4, grp, &eb);
    __syncthreads();
  }
}

// MXFP8 quantization of bf16 rows (OCP MX v1.0): thread = one block of 32
// consecutive elements; scale 2^(floor(log2 amax) - 8) as E8M0, elements
// v / scale rounded to nearest-even E4M3 with saturation at +-448 (by bit
// arithmetic on the binary32 value, exact: v / scale has at most 8
// significant bits); an all-zero block gets scale byte 0.
__device__ __forceinline__ uint32_t e4m3_of(float y) {
  const uint32_t u = __float_as_uint(y), sign = (u >> 24) & 0x80u;
  const float a = fabsf(y);
  if (a >= 448.f) return sign | 0x7Eu;
  uint32_t code;
  if (a < 0x1p-6f) {
    // subnormal: multiples of 2^-9, nearest-even (a * 2^9 is exact)
    const float m = rintf(a * 512.f);
    code = (uint32_t)m;  // 8 is the smallest normal, 2^-6
  } else {
    const uint32_t b = __float_as_uint(a);
    int e = (int)(b >> 23) - 127;
    uint32_t man = b & 0x7FFFFFu, r = man >> 20, rem = man & 0xFFFFFu;
    if (rem > 0x80000u || (rem == 0x80000u && (r & 1u))) ++r;
    if (r == 8u) { r = 0; ++e; }
    code = ((uint32_t)(e + 7) << 3) | r;
    if (code > 0x7Eu) code = 0x7Eu;
  }
  return code == 0 ? 0u : (sign | code);
}

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
  // the GEMM operand layout: code rows padded to whole 128-byte lines, the
  // four scale bytes of a row's 128 columns in one dword
  const int64_t sidx = P.gemm_layout ? ((int64_t)(c0 / 128) * P.rows + row) * 4 + (c0 / 32) % 4
                                     : row * per_row + c0 / 32;
  P.scales[sidx] = (uint8_t)(e + 127);
  const float inv = __uint_as_float((uint32_t)(127 - e) << 23);  // 2^-e, a normal power of two for e in [-127, 119]
  uint32_t out[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    uint32_t w = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) w |= e4m3_of(v[4 * q + i] * inv) << (8 * i);
    out[q] = w;
  }
  uint8_t* dst = P.codes + row * (P.gemm_layout ? mx_code_stride(P.cols) : P.cols) + c0;
  st16(dst, u32x4{out[0], out[1], out[2], out[3]});
  st16(dst + 16, u32x4{out[4], out[5], out[6], out[7]});
}

}  // namespace

bool mx_gemm_applies(const Gemm& g) {
  // 32-bit offsets: token rows and their scales from x itself, one group's
  // codes and scales
  const int64_t xr = g.x_rows > 0 ? g.x_rows : g.n_rows;
  return g.k > 0 && g.k % 64 == 0 && g.k <= MX_MAX_K && g.n % 16 == 0 && g.n_groups <= TILE_MAXG && g.x_scales &&
         g.w_scales && (uintptr_t)g.w_scales % 16 == 0 && (uintptr_t)g.x % 16 == 0 &&
         (uintptr_t)g.x_scales % 4 == 0 && xr * mx_code_stride(g.k) < (1LL << 32) &&
         mx_scale_bytes(xr, g.k) < (1LL << 32) && (int64_t)g.n * g.k / 2 < (1LL << 32);
}

hipError_t launch_gemm_mx(const Gemm& g, hipStream_t s) {
  if (!mx_gemm_applies(g)) return hipErrorInvalidValue;
  const int64_t grid = tile_grid(g, XM, XN);
  if (grid > 0x7FFFFFFF) return hipErrorInvalidValue;
  dim3 gd((unsigned)grid), bd(XTH);
  switch (g.epi) {
    case EPI_SWIGLU: hipLaunchKernelGGL((gemm_mx_kernel<EPI_SWIGLU>), gd, bd, 0, s, g); break;
    case EPI_BIAS: hipLaunchKernelGGL((gemm_mx_kernel<EPI_BIAS>), gd, bd, 0, s, g); break;
    default: return hipErrorNotSupported;
  }
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
