// Software-pipelined 256 x 256 grouped GEMM (gfx950, bf16 activations, bf16
// or MXFP4 weights) for launches with hundreds of token rows per weight
// matrix: the expert projections of a prefill-sized step and the dense
// projections of tens of thousands of tokens.
//
// On gfx950 the LDS, not the matrix cores, bounds an LDS-tiled GEMM: a
// 16x16x32 product takes 16 cycles, while the 16-byte fragment reads that
// feed it run at about 128 B per clock per CU and the staging writes at about
// 85. Per multiply-accumulate the LDS traffic falls with the tile a wavefront
// owns, so eight wavefronts (two per SIMD) each own a 128 x 64 piece of a
// 256 x 256 output tile: 12 fragment reads per 32 products, against 8 per 16
// for 64 x 64 pieces.
//
// The reduction runs in 32-wide slices through three LDS stages, each a
// separate array so the compiler can order accesses to different stages
// freely. While slice i is multiplied out of its stage, slice i + 2 is
// written from one of two register sets into the stage slice i - 1 used,
// slice i + 4 is loaded from global memory into that set, and the first
// fragments of slice i + 1 are read, all interleaved with the products
// (scheduling groups pin the interleave). Slice i + 1 was written before the previous barrier,
// so the one barrier per slice never waits for a fragment read.
//
// LDS layout: rows 96 B apart (64 B of data). The 16-byte fragment reads of
// 16 rows then fall in distinct banks, and each 8-lane group of a staging
// write (rows r and r + 2) covers all eight 16-byte bank groups of a 128-byte
// bank row; with rows 80 or 144 B apart both take twice the LDS cycles.
//
// MXFP4 weights are decoded while they are staged (the packed e2m1 -> bf16
// conversion with the block scale; exact). The finished fp32 tile goes through
// LDS to the fused epilogue, 32 rows at a time.
#include <type_traits>

#include "device.h"
#include "gemm_epilogue.h"
#include "kernels.h"

namespace mcpu {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int PM = 256, PN = 256, PK = 32;   // output tile, reduction slice
constexpr int PTH = 512;                     // eight wavefronts
constexpr int PLD = PK + 16;                 // LDS row stride in bf16 (96 B, see below)
constexpr int PSTAGE = (PM + PN) * PLD;      // bf16 elements per stage
constexpr int PWN = PN / 4;                  // weight rows per wavefront (wavefronts in 2 x 4)
constexpr int PMF = PM / 2 / 16, PNF = PWN / 16;  // 8 token-row and 4 weight-row fragments
constexpr int PEP = 32, PCLD = PN + 4;       // epilogue pass rows, fp32 row stride
static_assert(PEP * PCLD * 4 <= PSTAGE * 2, "an epilogue pass fits one stage");
constexpr int PGM = 2;                       // m-tiles per band
constexpr int NR = 2;                        // register sets of staged slices in flight

__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(void* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }
__device__ __forceinline__ f32x4 mfma(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b), c,
                                                  0, 0, 0);
}

// Staged weights of one slice, in two parts that are written to LDS and
// refilled from global memory in turn: two 16-byte chunks of bf16 rows per
// thread ...
// Staging assignment: thread t stages 16-byte chunk t % 4 of rows
// stage_row(t) and stage_row(t) + 128 of both operands (parts 0 and 1). The
// four lanes of a row read its 64 bytes of the slice with one access, and
// each 8-lane group writes rows r and r + 2, whose 96-byte-strided chunks
// fill all eight 16-byte bank groups.
__device__ __forceinline__ int stage_row(int t) {
  const int g = t >> 3;
  return 4 * (g >> 1) + (g & 1) + 2 * ((t & 7) >> 2);
}

// Staged weights of one slice, in two parts (rows r and r + 128) that are
// written to LDS and refilled from global memory in turn: bf16 rows ...
template <int WF>
struct PipeW {
  struct Regs {
    u32x4 r[2];
  };
  const bf16* src[2];
  int dst;  // LDS offset (bf16) of part 0 within a stage
  __device__ __forceinline__ void init(const Gemm& P, int grp, int n0, int nrows, int tid, int epi_qkv) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int rr = stage_row(tid) + 128 * j, rc = min(rr, nrows - 1);
      const int blk = (n0 + rc) >> 4, nl = rc & 15;
      const int wrow = epi_qkv ? block_row<EPI_QKV>(P, blk, nl) : blk * 16 + nl;
      src[j] = reinterpret_cast<const bf16*>(P.w) + grp * P.w_group_stride + (int64_t)wrow * P.k + (tid & 3) * 8;
    }
    dst = (PM + stage_row(tid)) * PLD + (tid & 3) * 8;
  }
  __device__ __forceinline__ void fetch(Regs& g, int p, int ks) const { g.r[p] = ld16(src[p] + ks * PK); }
  __device__ __forceinline__ void store(const Regs& g, int p, bf16* stage, bool&) const {
    st16(stage + dst + 128 * PLD * p, g.r[p]);
  }
};

// ... or MXFP4: per part the 8 weights of the chunk (4 code bytes) and the
// E8M0 scale of the row's 32-weight block, decoded into 16 bytes.
template <>
struct PipeW<1> {
  struct Regs {
    uint32_t c[2];
    uint32_t s[2];
  };
  // one expert's codes and scales stay below 4 GiB: a uniform base and 32-bit offsets
  const uint8_t* cbase;
  const uint8_t* sbase;
  uint32_t coff[2], soff[2];
  int dst;
  __device__ __forceinline__ void init(const Gemm& P, int grp, int n0, int nrows, int tid, int) {
    cbase = reinterpret_cast<const uint8_t*>(P.w) + grp * P.w_group_stride;
    sbase = P.w_scales + grp * (P.w_group_stride / 16);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int rr = stage_row(tid) + 128 * j, rc = min(rr, nrows - 1);
      const uint32_t wrow = n0 + rc;
      coff[j] = wrow * (uint32_t)(P.k / 2) + 4 * (tid & 3);
      soff[j] = wrow * (uint32_t)(P.k / 32);
    }
    dst = (PM + stage_row(tid)) * PLD + (tid & 3) * 8;
  }
  __device__ __forceinline__ void fetch(Regs& g, int p, int ks) const {
    g.c[p] = *reinterpret_cast<const uint32_t*>(cbase + (coff[p] + ks * (PK / 2)));
    g.s[p] = sbase[soff[p] + ks];
  }
  __device__ __forceinline__ void store(const Regs& g, int p, bf16* stage, bool& bad) const {
    const bool ok = g.s[p] >= 2u && g.s[p] <= 252u;
    bad = bad || !ok;
    const float scale = __uint_as_float(ok ? g.s[p] << 23 : 127u << 23);
    // byte b of the word holds weights 2b (low nibble) and 2b + 1 of the chunk
    const uint32_t w = ok ? g.c[p] : 0u;
    const u32x4 o = {__builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, scale, 0)),
                     __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, scale, 1)),
                     __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, scale, 2)),
                     __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(w, scale, 3))};
    st16(stage + dst + 128 * PLD * p, o);
  }
};

template <int EPI, int WF>
__global__ __launch_bounds__(PTH) void gemm_pipe_kernel(Gemm P) {
  __shared__ __align__(16) bf16 st0[PSTAGE];
  __shared__ __align__(16) bf16 st1[PSTAGE];
  __shared__ __align__(16) bf16 st2[PSTAGE];
  __shared__ int mt_start[TILE_MAXG + 1];
  const int tid = threadIdx.x, lane = tid & 63, wave = uniform(tid >> 6);

  int grp, mt, tn;
  if (!tile_of_block<PM, PN, PGM>(P, mt_start, grp, mt, tn)) return;
  const int gr0 = P.group_off ? P.group_off[grp] : 0;
  const int gr1 = P.group_off ? P.group_off[grp + 1] : P.n_rows;
  const int m0 = uniform(gr0 + mt * PM);
  const int mrows = min(PM, gr1 - m0);
  const int n0 = uniform(tn * PN), nrows = min(PN, P.n - n0);

  // staging (stage_row): rows past the tile's end repeat its last row (their
  // results are dropped)
  const bf16* xsrc[2];
  const int xdst = stage_row(tid) * PLD + (tid & 3) * 8;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int row = m0 + min(stage_row(tid) + 128 * j, mrows - 1);
    const int src = P.row_src ? P.row_src[row] : row;
    xsrc[j] = reinterpret_cast<const bf16*>(P.x) + (int64_t)src * P.k + (tid & 3) * 8;
  }
  PipeW<WF> wl;
  wl.init(P, grp, n0, nrows, tid, EPI == EPI_QKV);
  struct Regs {
    u32x4 x[2];
    typename PipeW<WF>::Regs w;
  };
  const int nk = P.k / PK;
  bool bad_scale = false;

  // fragments: wavefront (wm, wn) multiplies token rows wm * 128 + [0, 128)
  // by weight rows wn * 64 + [0, 64); lane l supplies row l % 16, k-chunk 8 (l / 16)
  const int wm = wave & 1, wn = wave >> 1;
  const int fr = lane & 15, fk = 8 * (lane >> 4);
  const int xoff = (wm * (PM / 2) + fr) * PLD + fk;
  const int woff = (PM + wn * PWN + fr) * PLD + fk;
  f32x4 acc[PNF][PMF];
#pragma unroll
  for (int nb = 0; nb < PNF; ++nb)
#pragma unroll
    for (int mb = 0; mb < PMF; ++mb) acc[nb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto stage_of = [&](int s) __attribute__((always_inline)) { return s == 0 ? st0 : s == 1 ? st1 : st2; };
  // slices past the end re-read the last one (never multiplied); part p < 2
  // of a register set is token-row part p, part 2 + q weight part q
  auto fetch = [&](Regs& g, int p, int ks) __attribute__((always_inline)) {
    ks = min(ks, nk - 1);
    if (p < 2) g.x[p] = ld16(xsrc[p] + ks * PK);
    else wl.fetch(g.w, p - 2, ks);
  };
  auto store = [&](const Regs& g, int p, bf16* stage) __attribute__((always_inline)) {
    if (p < 2) st16(stage + xdst + 128 * PLD * p, g.x[p]);
    else wl.store(g.w, p - 2, stage, bad_scale);
  };

  // prologue: slices 0 and 1 staged, slices 2 .. 1 + NR in flight in the
  // register sets, the head of slice 0 read
  Regs rs[NR];
  {
    Regs r0, r1;
#pragma unroll
    for (int p = 0; p < 4; ++p) fetch(r0, p, 0);
#pragma unroll
    for (int p = 0; p < 4; ++p) fetch(r1, p, 1);
#pragma unroll
    for (int r = 0; r < NR; ++r)
#pragma unroll
      for (int p = 0; p < 4; ++p) fetch(rs[r], p, 2 + r);
#pragma unroll
    for (int p = 0; p < 4; ++p) store(r0, p, st0);
#pragma unroll
    for (int p = 0; p < 4; ++p) store(r1, p, st1);
  }
  __syncthreads();
  // head fragments of a slice (its weight fragments and first two token-row
  // fragments) in two sets by slice parity: slice i reads set i % 2 and
  // fills set (i + 1) % 2, so the unrolled loop needs no register copies
  u32x4 ah[2][PNF], bh[2][2];
#pragma unroll
  for (int nb = 0; nb < PNF; ++nb) ah[0][nb] = ld16(st0 + woff + nb * 16 * PLD);
  bh[0][0] = ld16(st0 + xoff);
  bh[0][1] = ld16(st0 + xoff + 16 * PLD);

  // Slice i (stage S = i % 3, register set R = i % 2): eight steps of four
  // products (token-row fragment s against the four weight-row fragments)
  // with the reads two steps ahead. Steps 0-3 each write one part of set R
  // (slice i + 2) to stage (S + 2) % 3 and refill it with slice i + 4; steps
  // 4-7 read the head of slice i + 1.
  auto slice = [&](auto S_, auto R_, int i) __attribute__((always_inline)) {
    constexpr int S = decltype(S_)::value, R = decltype(R_)::value;
    bf16* cur = stage_of(S);
    bf16* nxt = stage_of((S + 1) % 3);
    bf16* wr = stage_of((S + 2) % 3);
    constexpr int H = R;  // slice parity (the register set alternates with it)
    u32x4* a = ah[H];
    u32x4 b[PMF];
    b[0] = bh[H][0];
    b[1] = bh[H][1];
#pragma unroll
    for (int s = 0; s < PMF; ++s) {
      if (s + 2 < PMF) b[s + 2] = ld16(cur + xoff + (s + 2) * 16 * PLD);
      else bh[H ^ 1][s + 2 - PMF] = ld16(nxt + xoff + (s + 2 - PMF) * 16 * PLD);
      if (s >= 4) ah[H ^ 1][s - 4] = ld16(nxt + woff + (s - 4) * 16 * PLD);
      if (s < 4) {
        store(rs[R], s, wr);
        fetch(rs[R], s, i + 2 + NR);
      }
#pragma unroll
      for (int nb = 0; nb < PNF; ++nb) acc[nb][s] = mfma(a[nb], b[s], acc[nb][s]);
    }
    // interleave: per step the LDS reads (0x100), the LDS write (0x200) and
    // global load (0x020) of steps 0-3, then four products (0x008)
#define PIPE_STEP(NR, NM)                              \
  __builtin_amdgcn_sched_group_barrier(0x100, NR, 0);  \
  __builtin_amdgcn_sched_group_barrier(0x200, NM, 0);  \
  __builtin_amdgcn_sched_group_barrier(0x020, NM, 0);  \
  __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
    PIPE_STEP(1, 1) PIPE_STEP(1, 1) PIPE_STEP(1, 1) PIPE_STEP(1, 1)
    PIPE_STEP(2, 0) PIPE_STEP(2, 0) PIPE_STEP(2, 0) PIPE_STEP(2, 0)
#undef PIPE_STEP
    __syncthreads();
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;

  int i = 0;
  for (; i + 6 <= nk; i += 6) {
    slice(I0{}, I0{}, i);
    slice(I1{}, I1{}, i + 1);
    slice(I2{}, I0{}, i + 2);
    slice(I0{}, I1{}, i + 3);
    slice(I1{}, I0{}, i + 4);
    slice(I2{}, I1{}, i + 5);
  }
  if (i < nk) slice(I0{}, I0{}, i);
  if (i + 1 < nk) slice(I1{}, I1{}, i + 1);
  if (i + 2 < nk) slice(I2{}, I0{}, i + 2);
  if (i + 3 < nk) slice(I0{}, I1{}, i + 3);
  if (i + 4 < nk) slice(I1{}, I0{}, i + 4);
  if (bad_scale) set_error(P.err, 16);

  // acc[nb][mb][r] = C[m = wm*128 + 16 mb + fr][n = wn*64 + 16 nb + 4 (lane/16) + r];
  // the fp32 tile goes through LDS (stage 0, free after the last barrier)
  float* cr = reinterpret_cast<float*>(st0);
  const EpiBias eb = epilogue_bias<EPI>(P, n0 >> 4, nrows >> 4, grp);
#pragma unroll
  for (int e0 = 0; e0 < PM; e0 += PEP) {
    if (e0 >= mrows) break;  // uniform
    if (wm == e0 / (PM / 2)) {
#pragma unroll
      for (int mb = 0; mb < PMF; ++mb) {
        const int m = wm * (PM / 2) + mb * 16;
        if (m >= e0 && m < e0 + PEP) {
#pragma unroll
          for (int nb = 0; nb < PNF; ++nb) {
            const int n = wn * PWN + nb * 16 + 4 * (lane >> 4);
            *reinterpret_cast<float4*>(cr + (m + fr - e0) * PCLD + n) =
                make_float4(acc[nb][mb][0], acc[nb][mb][1], acc[nb][mb][2], acc[nb][mb][3]);
          }
        }
      }
    }
    __syncthreads();
    epilogue<bf16, EPI>(P, cr, PCLD, m0 + e0, min(PEP, mrows - e0), n0 >> 4, nrows >> 4, grp, &eb);
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// bf16 weights: the same tile and wavefront split, with every slice loaded
// straight from global memory into LDS by 16-byte direct loads (a
// wavefront's load fills 1 KB of LDS, lane l at byte 16 l), so staging costs
// neither registers nor LDS write instructions. Five stages (all of the
// LDS): while slice i is multiplied, the head of slice i + 1 is read, slices
// i + 2 and i + 3 land and slice i + 4 is requested; before each barrier a
// wavefront waits for its own loads of slice i + 2 (the barrier then
// publishes them to all wavefronts). Rows
// are 64 bytes with no padding; chunk q of row r sits in 16-byte slot
// q ^ ((r >> 1) & 3) of its row, which keeps the fragment reads free of bank
// conflicts, and each lane loads the global chunk its slot holds. With the
// weights' streaming-order copy (WP), a 16-row block's slice is one
// contiguous KiB already in fragment order (lane l's 16 bytes at 16 l), so
// the weight loads are whole contiguous lines and land as they are.
// ---------------------------------------------------------------------------
constexpr int DROW = PK * 2;              // bytes per staged row
constexpr int DSTAGE = (PM + PN) * DROW;  // bytes per stage (32 KB)
constexpr int DEP = 16;                   // epilogue rows per pass
constexpr int DNS = 5;                    // stages
static_assert(DEP * PCLD * 4 <= DSTAGE, "an epilogue pass fits one stage");
__device__ __forceinline__ int dswz(int r) { return (r >> 1) & 3; }
constexpr int BUF_DWORD3 = 0x00020000;  // raw buffer descriptor word 3 (gfx9 family)
typedef __attribute__((address_space(3))) void* lds_void_t;

template <int EPI, bool WP>
__global__ __launch_bounds__(PTH) void gemm_dma_kernel(Gemm P) {
  static_assert(!(WP && EPI == EPI_QKV), "the projection's row order is not the copy's");
  __shared__ __align__(1024) uint8_t d0[DSTAGE];
  __shared__ __align__(1024) uint8_t d1[DSTAGE];
  __shared__ __align__(1024) uint8_t d2[DSTAGE];
  __shared__ __align__(1024) uint8_t d3[DSTAGE];
  __shared__ __align__(1024) uint8_t d4[DSTAGE];
  const int tid = threadIdx.x, lane = tid & 63, wave = uniform(tid >> 6);

  // the m-tile prefix lives in stage 4 until the first barrier after it is
  // read (stage 4 first receives slice 4, requested after that barrier)
  static_assert((TILE_MAXG + 1) * 4 <= DSTAGE, "the m-tile prefix fits a stage");
  int grp, mt, tn;
  if (!tile_of_block<PM, PN, PGM>(P, reinterpret_cast<int*>(d4), grp, mt, tn)) return;
  const int gr0 = P.group_off ? P.group_off[grp] : 0;
  const int gr1 = P.group_off ? P.group_off[grp + 1] : P.n_rows;
  const int m0 = uniform(gr0 + mt * PM);
  const int mrows = min(PM, gr1 - m0);
  const int n0 = uniform(tn * PN), nrows = min(PN, P.n - n0);

  // wavefront w loads rows 32 w + 16 j + [0, 16) of both operands (j = 0, 1);
  // lane l lands in row + l / 4, slot l % 4, the home of chunk (l % 4) ^ swz.
  // Rows past the tile's end repeat its last row (their results are dropped).
  // Buffer loads: a uniform base (the tile's first row, or x itself when rows
  // are gathered; the group's weights), a 32-bit per-lane row offset and the
  // slice offset in a scalar register.
  const int lr = lane >> 2, chunk = (lane & 3) ^ dswz(lr);
  const uint8_t* xb = reinterpret_cast<const uint8_t*>(P.x) + (P.row_src ? 0 : (int64_t)m0 * P.k * 2);
  // streaming-order copy: per group rows / 16 blocks of ceil(k / 128) 4 KiB
  // chunks; slice ks of block b at (b * chunks) * 4 KiB + ks KiB
  const int wchunks = (P.k + 127) / 128;
  const uint8_t* wb = WP ? reinterpret_cast<const uint8_t*>(P.w_packed) + (int64_t)grp * (P.n / 16) * wchunks * 4096
                         : reinterpret_cast<const uint8_t*>(P.w) + (int64_t)grp * P.w_group_stride * 2;
  const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(xb), 0, 0x7FFFFFFF, BUF_DWORD3);
  const __amdgpu_buffer_rsrc_t wr = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(wb), 0, 0x7FFFFFFF, BUF_DWORD3);
  uint32_t xvo[2], wvo[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int rr = 32 * wave + 16 * j + lr;
    const int rm = min(rr, mrows - 1);
    xvo[j] = P.row_src ? (uint32_t)P.row_src[m0 + rm] * (uint32_t)(P.k * 2) + chunk * 16
                       : (uint32_t)rm * (uint32_t)(P.k * 2) + chunk * 16;
    const int rc = min(rr, nrows - 1);
    const int blk = (n0 + rc) >> 4, nl = rc & 15;
    const int wrow = EPI == EPI_QKV ? block_row<EPI_QKV>(P, blk, nl) : blk * 16 + nl;
    if (WP) {
      const int b = min(n0 / 16 + 2 * wave + j, P.n / 16 - 1);  // the wavefront's 16-row block
      wvo[j] = (uint32_t)b * (uint32_t)(wchunks * 4096) + 16u * lane;
    } else {
      wvo[j] = (uint32_t)wrow * (uint32_t)(P.k * 2) + chunk * 16;
    }
  }
  const int ldst = 32 * wave * DROW;  // this wavefront's rows within an operand
  const int nk = P.k / PK;

  const int wm = wave & 1, wn = wave >> 1;
  const int fr = lane & 15, slot = ((lane >> 4) ^ dswz(fr)) * 16;
  const int xoff = (wm * (PM / 2) + fr) * DROW + slot;
  const int woff = WP ? PM * DROW + wn * PWN * DROW + 16 * lane : (PM + wn * PWN + fr) * DROW + slot;
  f32x4 acc[PNF][PMF];
#pragma unroll
  for (int nb = 0; nb < PNF; ++nb)
#pragma unroll
    for (int mb = 0; mb < PMF; ++mb) acc[nb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto stage_of = [&](int s) __attribute__((always_inline)) {
    return s == 0 ? d0 : s == 1 ? d1 : s == 2 ? d2 : s == 3 ? d3 : d4;
  };
  // load p of a slice (0, 1: token rows, 2, 3: weight rows); slices past the
  // end re-read the last one (never multiplied)
  auto dma = [&](uint8_t* stg, int p, int ks) __attribute__((always_inline)) {
    const int soff = uniform(min(ks, nk - 1) * (PK * 2));
    uint8_t* dst = stg + (p < 2 ? 0 : PM * DROW) + ldst + 16 * (p & 1) * DROW;
    if (p < 2) __builtin_amdgcn_raw_ptr_buffer_load_lds(xr, (lds_void_t)(dst), 16, xvo[p], soff, 0, 0);
    else __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (lds_void_t)(dst), 16, wvo[p - 2], WP ? soff * 16 : soff, 0, 0);
  };
  // each wavefront's own loads of all but the two latest slices done (4
  // loads per slice), LDS reads done, then the barrier that publishes them
  auto publish = [&]() __attribute__((always_inline)) {
    __builtin_amdgcn_s_waitcnt(8 | (7 << 4) | (0 << 8));  // vmcnt(8) expcnt(7) lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
  };

  // prologue: slices 0 .. 3 requested, 0 and 1 published, head of slice 0 read
#pragma unroll
  for (int s = 0; s < DNS - 1; ++s)
#pragma unroll
    for (int p = 0; p < 4; ++p) dma(stage_of(s), p, s);
  publish();
  u32x4 ah[2][PNF], bh[2][2];
#pragma unroll
  for (int nb = 0; nb < PNF; ++nb) ah[0][nb] = ld16(d0 + woff + nb * 16 * DROW);
  bh[0][0] = ld16(d0 + xoff);
  bh[0][1] = ld16(d0 + xoff + 16 * DROW);

  // slice i uses stage i % 5 and head set i % 2: the loop is unrolled ten times
  auto slice = [&](auto S_, auto H_, int i) __attribute__((always_inline)) {
    constexpr int S = decltype(S_)::value, H = decltype(H_)::value;
    uint8_t* cur = stage_of(S);
    uint8_t* nxt = stage_of((S + 1) % DNS);
    uint8_t* req = stage_of((S + DNS - 1) % DNS);
    u32x4* a = ah[H];
    u32x4 b[PMF];
    b[0] = bh[H][0];
    b[1] = bh[H][1];
#pragma unroll
    for (int s = 0; s < PMF; ++s) {
      if (s + 2 < PMF) b[s + 2] = ld16(cur + xoff + (s + 2) * 16 * DROW);
      else bh[H ^ 1][s + 2 - PMF] = ld16(nxt + xoff + (s + 2 - PMF) * 16 * DROW);
      if (s >= 4) ah[H ^ 1][s - 4] = ld16(nxt + woff + (s - 4) * 16 * DROW);
      if (s < 4) dma(req, s, i + DNS - 1);
#pragma unroll
      for (int nb = 0; nb < PNF; ++nb) acc[nb][s] = mfma(a[nb], b[s], acc[nb][s]);
    }
#define DMA_STEP(NR, NM)                               \
  __builtin_amdgcn_sched_group_barrier(0x100, NR, 0);  \
  __builtin_amdgcn_sched_group_barrier(0x020, NM, 0);  \
  __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
    DMA_STEP(1, 1) DMA_STEP(1, 1) DMA_STEP(1, 1) DMA_STEP(1, 1)
    DMA_STEP(2, 0) DMA_STEP(2, 0) DMA_STEP(2, 0) DMA_STEP(2, 0)
#undef DMA_STEP
    publish();
  };
  using C0 = std::integral_constant<int, 0>;
  using C1 = std::integral_constant<int, 1>;
  using C2 = std::integral_constant<int, 2>;
  using C3 = std::integral_constant<int, 3>;
  using C4 = std::integral_constant<int, 4>;
  int i = 0;
  for (; i + 10 <= nk; i += 10) {
    slice(C0{}, C0{}, i);
    slice(C1{}, C1{}, i + 1);
    slice(C2{}, C0{}, i + 2);
    slice(C3{}, C1{}, i + 3);
    slice(C4{}, C0{}, i + 4);
    slice(C0{}, C1{}, i + 5);
    slice(C1{}, C0{}, i + 6);
    slice(C2{}, C1{}, i + 7);
    slice(C3{}, C0{}, i + 8);
    slice(C4{}, C1{}, i + 9);
  }
  if (i < nk) slice(C0{}, C0{}, i);
  if (i + 1 < nk) slice(C1{}, C1{}, i + 1);
  if (i + 2 < nk) slice(C2{}, C0{}, i + 2);
  if (i + 3 < nk) slice(C3{}, C1{}, i + 3);
  if (i + 4 < nk) slice(C4{}, C0{}, i + 4);
  if (i + 5 < nk) slice(C0{}, C1{}, i + 5);
  if (i + 6 < nk) slice(C1{}, C0{}, i + 6);
  if (i + 7 < nk) slice(C2{}, C1{}, i + 7);
  if (i + 8 < nk) slice(C3{}, C0{}, i + 8);
  __syncthreads();  // every load landed before stage 0 holds the fp32 tile

  // acc[nb][mb][r] = C[m = wm*128 + 16 mb + fr][n = wn*64 + 16 nb + 4 (lane/16) + r]
  float* cr = reinterpret_cast<float*>(d0);
  const EpiBias eb = epilogue_bias<EPI>(P, n0 >> 4, nrows >> 4, grp);
  for (int e0 = 0; e0 < PM; e0 += DEP) {
    if (e0 >= mrows) break;  // uniform
    if (wm == e0 / (PM / 2)) {
#pragma unroll
      for (int mb = 0; mb < PMF; ++mb) {
        if (wm * (PM / 2) + mb * 16 == e0) {
#pragma unroll
          for (int nb = 0; nb < PNF; ++nb) {
            const int n = wn * PWN + nb * 16 + 4 * (lane >> 4);
            *reinterpret_cast<float4*>(cr + fr * PCLD + n) =
                make_float4(acc[nb][mb][0], acc[nb][mb][1], acc[nb][mb][2], acc[nb][mb][3]);
          }
        }
      }
    }
    __syncthreads();
    epilogue<bf16, EPI>(P, cr, PCLD, m0 + e0, min(DEP, mrows - e0), n0 >> 4, nrows >> 4, grp, &eb);
    __syncthreads();
  }
}

}  // namespace

bool pipe_gemm_applies(int dtype, const Gemm& g) {
  if (dtype != 1 || g.k <= 0 || g.k % PK || g.n % 16 || g.n_groups > TILE_MAXG) return false;
  const int64_t groups = g.group_off ? g.n_groups : 1;
  // rows per group of a full tile on average, and at least two tiles per CU;
  // the vocabulary head (one matrix, every tile streaming its own weights from
  // HBM once) only from 1024 rows: below, 128 x 128 tiles keep more loads in
  // flight per compute unit (256 rows: 569 against 714 us)
  if (g.epi == EPI_LOGITS && g.n_rows < 1024) return false;
  return (int64_t)g.n_rows >= (int64_t)PM * groups && tile_grid(g, PM, PN) >= 512;
}

hipError_t launch_gemm_pipe(int expert_fmt, const Gemm& g, hipStream_t s) {
  const int64_t grid = tile_grid(g, PM, PN);
  if (grid > 0x7FFFFFFF) return hipErrorInvalidValue;
  if (expert_fmt != 0 && !g.w_scales) return hipErrorInvalidValue;
  dim3 gd((unsigned)grid), bd(PTH);
  // direct loads address rows with 32-bit offsets: from the tile's first row,
  // or from x itself when rows are gathered, and within one group's weights
  const int64_t xr = g.row_src ? (g.x_rows > 0 ? g.x_rows : g.n_rows) : PM;
  const bool dma = xr * g.k * 2 < (1LL << 31) && (int64_t)g.n * g.k * 2 < (1LL << 31);
  // the streaming-order weight copy, when given, for every epilogue but the
  // projection's (whose row order is its own)
  const bool wp = g.w_packed && g.k % PK == 0 && (int64_t)(g.n / 16) * ((g.k + 127) / 128) * 4096 < (1LL << 31);
#define PIPE_LAUNCH(E)                                                                          \
  do {                                                                                          \
    if (expert_fmt != 0) hipLaunchKernelGGL((gemm_pipe_kernel<E, 1>), gd, bd, 0, s, g);        \
    else if (dma && wp) hipLaunchKernelGGL((gemm_dma_kernel<E, true>), gd, bd, 0, s, g);        \
    else if (dma) hipLaunchKernelGGL((gemm_dma_kernel<E, false>), gd, bd, 0, s, g);             \
    else hipLaunchKernelGGL((gemm_pipe_kernel<E, 0>), gd, bd, 0, s, g);                         \
  } while (0)
  switch (g.epi) {
    case EPI_QKV:
      if (dma) hipLaunchKernelGGL((gemm_dma_kernel<EPI_QKV, false>), gd, bd, 0, s, g);
      else hipLaunchKernelGGL((gemm_pipe_kernel<EPI_QKV, 0>), gd, bd, 0, s, g);
      break;
    case EPI_RESIDUAL: PIPE_LAUNCH(EPI_RESIDUAL); break;
    case EPI_SWIGLU: PIPE_LAUNCH(EPI_SWIGLU); break;
    case EPI_LOGITS:  // vocabulary logits: bf16 weights only
      if (expert_fmt != 0) return hipErrorNotSupported;
      if (dma && wp) hipLaunchKernelGGL((gemm_dma_kernel<EPI_LOGITS, true>), gd, bd, 0, s, g);
      else if (dma) hipLaunchKernelGGL((gemm_dma_kernel<EPI_LOGITS, false>), gd, bd, 0, s, g);
      else hipLaunchKernelGGL((gemm_pipe_kernel<EPI_LOGITS, 0>), gd, bd, 0, s, g);
      break;
    default: PIPE_LAUNCH(EPI_BIAS); break;
  }
#undef PIPE_LAUNCH
  return hipGetLastError();
}

}  // namespace mcpu
