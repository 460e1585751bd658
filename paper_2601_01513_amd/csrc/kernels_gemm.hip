// MFMA GEMMs of the verifier scoring pass with fused epilogues.
//
// Every GEMM here is C = A . B^T with A [rows][K] and B [N][K] both
// K-contiguous (activations and nn.Linear weights), fp32 accumulation on the
// gfx950 v_mfma_f32_32x32x16_f16 matrix cores. Activations are fp16. Weights
// are 16-bit: fp16 (loaded straight into LDS) or bf16, converted to fp16 in
// registers on their way into LDS (exact: a bf16 value's 8 significant bits
// fit fp16's 11). The two forms cost the same HBM bytes; the fp16 form saves
// the register path and its conversion (about 6% of the GEMM time).
//
// Block: 512 threads = 8 waves (two per SIMD) on a 256 x 256 tile; the waves
// form a 4 x 2 grid, each owning 64 x 128 outputs (2 x 4 MFMA 32x32 blocks).
// K advances in panels of 64 through a two-stage LDS ring (2 x 64 KB): while
// the MFMAs consume panel k, panel k+1 is in flight -- fp16 operands straight
// from global memory into LDS (global_load_lds, no registers), bf16 operands
// through registers and the converter. One barrier per panel. LDS rows are
// eight 16-byte chunks; gfx950 LDS serves 256 bytes (64 banks) per cycle, so
// two consecutive 128-byte rows share a bank window: chunk c of row r sits at
// c ^ ((r / 2) % 8), which gives the 16 lanes of a 16-byte fragment load
// (rows r..r+15, one chunk) 16 distinct bank groups. For the direct loads the
// swizzle is applied to the global addresses (a direct load writes lane l's
// 16 bytes at base + 16 l).
//
// Blocks are numbered so that the ones resident on one XCD at the same time
// share A and B panels in that XCD's L2 (the hardware deals block b to XCD
// b % 8). Optional split-K: blocks of one tile take disjoint K ranges and
// write fp32 partials that a reduction kernel sums in a fixed order.
//
// MFMA 32x32x16 lane layout (lane l, element e, accumulator register r):
//   A operand: A[i = l % 32][k = 8 (l / 32) + e]
//   B operand: B[k = 8 (l / 32) + e][j = l % 32]
//   result   : C[i = 8 (r / 4) + 4 (l / 32) + r % 4][j = l % 32]
// so each lane holds one output column and sixteen output rows; epilogues
// work directly on the registers.
#include <algorithm>

#include "common.h"

namespace vsr {

namespace {

constexpr int BK = 64;        // K elements per panel (8 chunks of 16 bytes per row)
constexpr int NT = 512;       // threads per block
constexpr int NWAVES = NT / 64;

template <int BM_, int BN_, int WM_, int WN_>
struct Tile {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_;
  static constexpr int TM = BM / WM, TN = BN / WN;  // wave sub-tile
  static constexpr int FM = TM / 32, FN = TN / 32;  // MFMA blocks per wave
  static constexpr int STAGE = (BM + BN) * 8;       // 16-byte chunks per LDS stage
  static_assert(WM * WN == NWAVES, "eight waves");
  static_assert(TM % 32 == 0 && TN % 32 == 0, "32x32 MFMA blocks");
  static_assert(BM % 64 == 0 && BN % 64 == 0, "operand loads cover 64-row groups");
};

// 256 x 256 tile, waves 4 x 2 of 64 x 128: a wave's 128 columns hold a whole
// attention head (QKV) or 64 gate + 64 up columns (SwiGLU), so the rotary
// pairs and the gate/up pairs sit in the same lane and register.
typedef Tile<256, 256, 4, 2> TileStd;

__device__ __forceinline__ int swz(int row, int c) { return row * 8 + (c ^ ((row >> 1) & 7)); }
__device__ __forceinline__ f16x8 as_f16x8(u32x4 v) { return __builtin_bit_cast(f16x8, v); }

// Eight bf16 values -> eight fp16 values (exact for |v| in [2^-17, 65504];
// smaller magnitudes truncate below 2^-24).
__device__ __forceinline__ u32x4 bf16x8_to_f16x8(u32x4 v) {
  u32x4 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float lo = __uint_as_float(v[i] << 16);
    const float hi = __uint_as_float(v[i] & 0xFFFF0000u);
    r[i] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(lo, hi));
  }
  return r;
}

// One operand (ROWS rows of a panel). CVT: stored as bf16, staged through
// registers and converted; otherwise fp16, loaded straight into LDS.
template <int ROWS, bool CVT>
struct Operand {
  static constexpr int PER_THREAD = ROWS * 8 / NT;  // 16-byte chunks per thread
  const uint16_t *g[PER_THREAD];                     // row base + chunk, K-tile 0
  int slot[PER_THREAD];                              // LDS chunk (register path)
  u32x4 r[CVT ? PER_THREAD : 1];

  template <class RowFn>
  __device__ __forceinline__ void init(const void *base, long ld, RowFn row_of) {
    const uint16_t *p = static_cast<const uint16_t *>(base);
    const int t = threadIdx.x;
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      int row, c;
      if constexpr (CVT) {
        const int id = i * NT + t;
        row = id >> 3;
        c = id & 7;
        slot[i] = swz(row, c);
      } else {
        // Direct load i of wave w fills LDS rows 8 (i * NWAVES + w) .. +7;
        // lane l lands in physical chunk l % 8 of row l / 8.
        const int w = t >> 6, l = t & 63;
        row = (i * NWAVES + w) * 8 + (l >> 3);
        c = (l & 7) ^ ((row >> 1) & 7);
        slot[i] = 0;
      }
      g[i] = p + (long)row_of(row) * ld + c * 8;
    }
  }
  // Starts loading K-panel kt into LDS stage `dst` (direct) or registers.
  __device__ __forceinline__ void issue(int kt, u32x4 *dst) {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      if constexpr (CVT) {
        r[i] = *reinterpret_cast<const u32x4 *>(g[i] + kt * BK);
      } else {
        const int w = threadIdx.x >> 6;
        __builtin_amdgcn_global_load_lds(g[i] + kt * BK, dst + (i * NWAVES + w) * 64, 16, 0, 0);
      }
    }
  }
  // Register path: convert and store the panel into LDS stage `dst`.
  __device__ __forceinline__ void commit(u32x4 *dst) {
    if constexpr (CVT) {
#pragma unroll
      for (int i = 0; i < PER_THREAD; ++i) dst[slot[i]] = bf16x8_to_f16x8(r[i]);
    }
  }
};

// Fragment loads of one 16-wide k-step and the MFMAs that consume them.
template <class TL>
struct Frags {
  f16x8 a[TL::FM], b[TL::FN];
  __device__ __forceinline__ void load(const u32x4 *stage, const int (&fa)[TL::FM],
                                       const int (&fb)[TL::FN], int c) {
#pragma unroll
    for (int fm = 0; fm < TL::FM; ++fm) a[fm] = as_f16x8(stage[swz(fa[fm], c)]);
#pragma unroll
    for (int fn = 0; fn < TL::FN; ++fn) b[fn] = as_f16x8(stage[swz(fb[fn], c)]);
  }
  __device__ __forceinline__ void mma(f32x16 (&acc)[TL::FM][TL::FN]) const {
#pragma unroll
    for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < TL::FN; ++fn)
        acc[fm][fn] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[fm], b[fn], acc[fm][fn], 0, 0, 0);
  }
};

// Scheduling hints: interleave the next k-step's LDS reads (and the
// register-path panel conversion) with the current k-step's MFMAs.
__device__ __forceinline__ void interleave_reads(int nreads, int nmfma) {
  for (int i = 0; i < nmfma; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // 1 MFMA
    if (i < nreads) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // 1 LDS read
  }
}

// acc += A[rows arow(0..BM)] . B[rows brow(0..BN)]^T over K-panels [kt0, kt1).
// The row functions must return in-range rows (results of clamped rows are
// never stored). CVT_A / CVT_B mark an operand stored as bf16. Fragments are
// double-buffered in registers: the LDS reads of k-step s+1 are in flight
// while the MFMAs of k-step s run.
// Split operands: with asplit = 2 each A row holds [hi | lo], the fp16 value
// and its fp16 remainder (K each), and B (K per row) is walked twice, so the
// product is B.hi + B.lo -- an operand carried to about 22 significant bits.
template <class TL, bool CVT_A, bool CVT_B, class ARow, class BRow>
__device__ __forceinline__ void mainloop(const void *A, ARow arow, const void *B, BRow brow,
                                         int K, int asplit, int kt0, int kt1, u32x4 *lds,
                                         f32x16 (&acc)[TL::FM][TL::FN]) {
  const int nkb = K / BK;  // K panels of B
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int wm = w / TL::WN, wn = w % TL::WN;
  Operand<TL::BM, CVT_A> oa;
  Operand<TL::BN, CVT_B> ob;
  oa.init(A, (long)K * asplit, arow);
  ob.init(B, K, brow);
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < TL::FN; ++fn) acc[fm][fn] = f32x16{};
  if (kt1 <= kt0) return;

  int fa[TL::FM], fb[TL::FN];
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm) fa[fm] = wm * TL::TM + fm * 32 + (lane & 31);
#pragma unroll
  for (int fn = 0; fn < TL::FN; ++fn) fb[fn] = TL::BM + wn * TL::TN + fn * 32 + (lane & 31);
  const int hc = lane >> 5;
  constexpr int NR = TL::FM + TL::FN, NM = TL::FM * TL::FN;

  oa.issue(kt0, lds);
  ob.issue(kt0 >= nkb ? kt0 - nkb : kt0, lds + TL::BM * 8);
  oa.commit(lds);
  ob.commit(lds + TL::BM * 8);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  Frags<TL> f0, f1;
  f0.load(lds, fa, fb, hc);
  for (int kt = kt0; kt < kt1; ++kt) {
    u32x4 *cur = lds + ((kt - kt0) & 1) * TL::STAGE;
    u32x4 *nxt = lds + (((kt - kt0) & 1) ^ 1) * TL::STAGE;
    const bool more = kt + 1 < kt1;
    if (more) {
      oa.issue(kt + 1, nxt);
      ob.issue(kt + 1 >= nkb ? kt + 1 - nkb : kt + 1, nxt + TL::BM * 8);
    }
    f1.load(cur, fa, fb, 2 + hc);
    f0.mma(acc);
    interleave_reads(NR, NM);
    f0.load(cur, fa, fb, 4 + hc);
    f1.mma(acc);
    interleave_reads(NR, NM);
    f1.load(cur, fa, fb, 6 + hc);
    f0.mma(acc);
    interleave_reads(NR, NM);
    if (more) {
      oa.commit(nxt);
      ob.commit(nxt + TL::BM * 8);
    }
    f1.mma(acc);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (more) f0.load(nxt, fa, fb, hc);
  }
}

// Output row / column (within the block tile) of accumulator register r of
// MFMA block (fm, fn) for this lane.
template <class TL>
__device__ __forceinline__ int acc_row(int wm, int fm, int r, int lane) {
  return wm * TL::TM + fm * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
}
template <class TL>
__device__ __forceinline__ int acc_col(int wn, int fn, int lane) {
  return wn * TL::TN + fn * 32 + (lane & 31);
}

// Work of one launch: ntiles = nm x nn output tiles. The first ndp tiles
// (whole rounds of the 256 CUs) run one block per tile; the remaining ntail
// tiles run nsplit blocks each over disjoint K ranges, writing fp32 partial
// tiles that a reduction kernel sums in a fixed order. Tiles are numbered GM
// m-tiles fastest, then n-tiles, so neighbouring tiles share operand panels.
struct Launch {
  int nm, nn, gm;
  int ndp, ntail, nsplit;
  unsigned blocks() const { return (unsigned)(ndp + ntail * nsplit); }
};

struct Work {
  int tm, tn, split;
  int tail;  // index among the tail tiles, -1 for a whole-K tile
};

__device__ __forceinline__ void tile_coords(int L, int nm, int nn, int gm, int &tm, int &tn) {
  const int g = min(gm, nm);
  const int grp = L / (g * nn);
  const int gsz = min(g, nm - grp * g);
  const int in = L - grp * g * nn;
  tm = grp * g + in % gsz;
  tn = in / gsz;
}

// The hardware deals block b to XCD b % 8; each XCD is given a contiguous
// range of whole-K tiles, so the blocks it runs together share panels in
// its L2.
__device__ __forceinline__ Work block_work(const Launch &ln) {
  const int b = blockIdx.x;
  Work w;
  int L;
  if (b < ln.ndp) {
    const int q = ln.ndp / 8, rem = ln.ndp % 8, x = b % 8, k = b / 8;
    L = (x < rem ? x * (q + 1) : rem * (q + 1) + (x - rem) * q) + k;
    w.split = 0;
    w.tail = -1;
  } else {
    const int bt = b - ln.ndp;
    w.tail = bt / ln.nsplit;
    w.split = bt % ln.nsplit;
    L = ln.ndp + w.tail;
  }
  tile_coords(L, ln.nm, ln.nn, ln.gm, w.tm, w.tn);
  return w;
}

constexpr int kMaxSplit = 8;
constexpr int kTileElems = 256 * 256;

// Whole rounds data-parallel, the tail split so that it fills one round.
Launch plan_launch(int nm, int nn, int gm, int nk) {
  Launch ln{nm, nn, gm, 0, 0, 1};
  const int tiles = nm * nn;
  const int tail = tiles % 256;
  ln.ndp = tiles - tail;
  ln.ntail = tail;
  if (tail > 0) {
    int s = std::min(256 / tail, std::min(kMaxSplit, std::max(1, nk / 4)));
    ln.nsplit = std::max(1, s);
    if (ln.nsplit == 1) {  // nothing to split: all tiles whole-K
      ln.ndp = tiles;
      ln.ntail = 0;
    }
  }
  return ln;
}

// K-panel range of split s of nsplit over nk panels.
__device__ __forceinline__ void split_range(int nk, int nsplit, int s, int &k0, int &k1) {
  k0 = (int)((long)nk * s / nsplit);
  k1 = (int)((long)nk * (s + 1) / nsplit);
}

// Raw fp32 partial tile: part[(tail * nsplit + split)][256][256], local
// coordinates (rows / columns past the matrix edge hold unused values).
template <class TL>
__device__ __forceinline__ void store_partial(const f32x16 (&acc)[TL::FM][TL::FN], float *part,
                                              const Launch &ln, const Work &wk) {
  static_assert(TL::BM == 256 && TL::BN == 256, "partial tiles are 256 x 256");
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w / TL::WN, wn = w % TL::WN;
  float *p = part + ((long)wk.tail * ln.nsplit + wk.split) * kTileElems;
#pragma unroll
  for (int fn = 0; fn < TL::FN; ++fn) {
    const int col = acc_col<TL>(wn, fn, lane);
#pragma unroll
    for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
      for (int r = 0; r < 16; ++r) p[acc_row<TL>(wm, fm, r, lane) * 256 + col] = acc[fm][fn][r];
  }
}

// Sum of the partials of local element e (row * 256 + col) of tail tile i,
// in split order. The reduce kernels are instantiated per split count NS
// (= ln.nsplit), so exactly NS loads are issued, all before the first add
// (the latencies overlap instead of adding up).
template <int NS>
__device__ __forceinline__ float sum_partials(const float *part, int i, int e) {
  const float *p = part + (long)i * NS * kTileElems + e;
  float v[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) v[s] = p[(long)s * kTileElems];
  float sum = 0.f;
#pragma unroll
  for (int s = 0; s < NS; ++s) sum += v[s];
  return sum;
}

// Launch of reduce kernel `kern<NS>` for the launch's split count (2 .. 8).
#define VSR_REDUCE_LAUNCH(ns, kern, grid, block, ...)                              \
  do {                                                                            \
    switch (ns) {                                                                 \
      case 2: kern<2><<<grid, block, 0, s>>>(__VA_ARGS__); break;                 \
      case 3: kern<3><<<grid, block, 0, s>>>(__VA_ARGS__); break;                 \
      case 4: kern<4><<<grid, block, 0, s>>>(__VA_ARGS__); break;                 \
      case 5: kern<5><<<grid, block, 0, s>>>(__VA_ARGS__); break;                 \
      case 6: kern<6><<<grid, block, 0, s>>>(__VA_ARGS__); break;                 \
      case 7: kern<7><<<grid, block, 0, s>>>(__VA_ARGS__); break;                 \
      default: kern<kMaxSplit><<<grid, block, 0, s>>>(__VA_ARGS__); break;        \
    }                                                                             \
  } while (0)

// silu(g) * u with the hardware reciprocal (about 1 ulp; the result is
// rounded to fp16 next): an IEEE division here cost ten instructions per
// output of the gate/up epilogue. Large negative g: exp(-g) = inf, rcp = 0.
__device__ __forceinline__ float silu_mul(float g, float u) {
  return g * __builtin_amdgcn_rcpf(1.f + __expf(-g)) * u;
}

// Activation store: fp16 value at base + col; with split = 2 also its fp16
// remainder at base + n + col (row layout [hi | lo]).
__device__ __forceinline__ void store_act(f16 *p, long base, int col, int n, int split, float v) {
  const f16 hi = static_cast<f16>(v);
  p[base + col] = hi;
  if (split == 2) p[base + n + col] = static_cast<f16>(v - static_cast<float>(hi));
}

// ------------------------------------------------------- residual (O, down)
// x += acc for one wave's NI x 4 MFMA blocks: this lane holds rows r0 + dr
// (dr = 32 i + 8 (r / 4) + r % 4 for block row i, register r) of columns
// c0 + 32 j (block column j). Buffer loads and stores over x (rows * N * 4
// bytes < 2 GiB, checked at launch): the lane offset carries the row, so
// rows past the matrix fail the buffer's range check (which covers the lane
// offset, not the scalar one) -- their loads read 0 and their stores are
// dropped -- and a lane whose column is past N starts beyond the buffer.
// Branch-free: masking each element made the compiler branch per element;
// per-element 64-bit addresses spilled registers. Batches of 8 rows x 4
// column blocks (32 values) are loaded before any of them is stored (the
// compiler cannot move a load of x above a store to x).
template <int NI>
__device__ __forceinline__ void residual_epilogue(const f32x16 (&acc)[NI][4], int r0, int c0,
                                                  int rows, int N, float *x) {
  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc(x, (short)0, (int)((size_t)rows * N * 4), 0x00020000);
  uint32_t bx[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int col = c0 + 32 * j;
    bx[j] = col < N ? (uint32_t)(r0 * N + col) * 4u : 0x80000000u;
  }
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int rh = 0; rh < 2; ++rh) {
      float xv[8][4];
      // (the b32 buffer builtins move raw bits: bit-cast, not convert)
#pragma unroll
      for (int rr = 0; rr < 8; ++rr)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint32_t dr = 32 * i + 16 * rh + 8 * (rr >> 2) + (rr & 3);
          xv[rr][j] = __uint_as_float(
              __builtin_amdgcn_raw_buffer_load_b32(xr, bx[j] + dr * (uint32_t)N * 4u, 0, 0));
        }
#pragma unroll
      for (int rr = 0; rr < 8; ++rr) {
        const uint32_t dr = 32 * i + 16 * rh + 8 * (rr >> 2) + (rr & 3);
#pragma unroll
        for (int j = 0; j < 4; ++j)
          __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(xv[rr][j] + acc[i][j][8 * rh + rr]),
                                                xr, bx[j] + dr * (uint32_t)N * 4u, 0, 0);
      }
    }
}

template <class TL, bool WCVT>
__global__ __launch_bounds__(NT) void k_gemm_residual(const f16 *__restrict__ A,
                                                      const uint16_t *__restrict__ W, int rows,
                                                      int N, int K, int asplit, Launch ln,
                                                      float *__restrict__ x,
                                                      float *__restrict__ part) {
  __shared__ u32x4 lds[2 * TL::STAGE];
  const Work wk = block_work(ln);
  const int m0 = wk.tm * TL::BM, n0 = wk.tn * TL::BN;
  const bool split = wk.tail >= 0;
  int k0 = 0, k1 = K / BK * asplit;
  if (split) split_range(k1, ln.nsplit, wk.split, k0, k1);
  f32x16 acc[TL::FM][TL::FN];
  mainloop<TL, false, WCVT>(
      A, [=](int r) { return min(m0 + r, rows - 1); }, W,
      [=](int r) { return min(n0 + r, N - 1); }, K, asplit, k0, k1, lds, acc);
  if (split) {
    store_partial<TL>(acc, part, ln, wk);
    return;
  }
  static_assert(TL::FN == 4 && TL::TN == 128, "four 32-column blocks per wave");
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w / TL::WN, wn = w % TL::WN;
  residual_epilogue<TL::FM>(acc, m0 + wm * TL::TM + 4 * (lane >> 5), n0 + wn * TL::TN + (lane & 31),
                            rows, N, x);
}

// Tail tiles: x += sum of the partials. Block (tail tile, 256-element slab).
template <int NS>
__global__ __launch_bounds__(256) void k_reduce_residual(const float *__restrict__ part,
                                                         Launch ln, int rows, int N,
                                                         float *__restrict__ x) {
  const int i = blockIdx.x / 256, e = (blockIdx.x % 256) * 256 + threadIdx.x;
  int tm, tn;
  tile_coords(ln.ndp + i, ln.nm, ln.nn, ln.gm, tm, tn);
  const int row = tm * 256 + e / 256, col = tn * 256 + e % 256;
  if (row >= rows || col >= N) return;
  x[(long)row * N + col] += sum_partials<NS>(part, i, e);
}

// ------------------------------------------------------------------- SwiGLU
// Output column tile o0 .. o0+128 of the FFN hidden. Its 256 B rows are laid
// out per wave column: wave column wn takes gate rows o0+64wn .. +63 then the
// matching up rows, so MFMA blocks fn and fn+2 hold gate and up of the same
// output columns (partial tiles keep that column order).
template <class TL, bool WCVT>
__global__ __launch_bounds__(NT) void k_gemm_swiglu(const f16 *__restrict__ A,
                                                    const uint16_t *__restrict__ W, int rows,
                                                    int F, int K, int asplit, Launch ln,
                                                    f16 *__restrict__ h, float *__restrict__ part) {
  static_assert(TL::WN == 2 && TL::TN == 128 && TL::BN == 256, "gate/up pairing");
  __shared__ u32x4 lds[2 * TL::STAGE];
  const Work wk = block_work(ln);
  const int m0 = wk.tm * TL::BM, o0 = wk.tn * 128;
  const bool split = wk.tail >= 0;
  int k0 = 0, k1 = K / BK * asplit;
  if (split) split_range(k1, ln.nsplit, wk.split, k0, k1);
  f32x16 acc[TL::FM][TL::FN];
  mainloop<TL, false, WCVT>(
      A, [=](int r) { return min(m0 + r, rows - 1); }, W,
      [=](int r) {
        const int q = r & 127;
        const int oc = min(o0 + (r >> 7) * 64 + (q & 63), F - 1);
        return q < 64 ? oc : F + oc;
      },
      K, asplit, k0, k1, lds, acc);
  if (split) {
    store_partial<TL>(acc, part, ln, wk);
    return;
  }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w / TL::WN, wn = w % TL::WN;
  if (m0 + TL::BM <= rows && o0 + 128 <= F && (F & 1) == 0) {
    // Whole tile (4-byte aligned pairs): adjacent lanes (columns c, c + 1) trade values so that each
    // writes two adjacent columns of one row with one 4-byte store, the even
    // lane rows 2k and the odd lane rows 2k + 1 (half the store instructions
    // of one fp16 value per store; measured 1% faster per launch).
    const bool odd = lane & 1;
#pragma unroll
    for (int fn = 0; fn < 2; ++fn) {
      const int c0 = o0 + wn * 64 + fn * 32 + (lane & 30);
#pragma unroll
      for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const float a = silu_mul(acc[fm][fn][2 * k], acc[fm][fn + 2][2 * k]);
          const float b = silu_mul(acc[fm][fn][2 * k + 1], acc[fm][fn + 2][2 * k + 1]);
          // quad_perm [1, 0, 3, 2]: the value of lane l ^ 1.
          const float got = __int_as_float(
              __builtin_amdgcn_update_dpp(0, __float_as_int(odd ? a : b), 0xB1, 0xF, 0xF, false));
          const float v0 = odd ? got : a, v1 = odd ? b : got;
          const int row = m0 + acc_row<TL>(wm, fm, 2 * k + (odd ? 1 : 0), lane);
          const long base = (long)row * F * asplit + c0;
          const f16 h0 = static_cast<f16>(v0), h1 = static_cast<f16>(v1);
          *reinterpret_cast<f16x2 *>(h + base) = f16x2{h0, h1};
          if (asplit == 2)
            *reinterpret_cast<f16x2 *>(h + base + F) =
                f16x2{static_cast<f16>(v0 - static_cast<float>(h0)),
                      static_cast<f16>(v1 - static_cast<float>(h1))};
        }
    }
    return;
  }
#pragma unroll
  for (int fn = 0; fn < 2; ++fn) {
    const int col = o0 + wn * 64 + fn * 32 + (lane & 31);
    if (col >= F) continue;
#pragma unroll
    for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + acc_row<TL>(wm, fm, r, lane);
        if (row < rows) store_act(h, (long)row * F * asplit, col, F, asplit,
                                  silu_mul(acc[fm][fn][r], acc[fm][fn + 2][r]));
      }
  }
}

// ------------------------------------ four-wave tile with an ordered K loop
// 256 threads = 4 waves, one per SIMD, on a 256 x 256 tile: wave w owns
// rows 128 (w / 2) .. + 127 and columns 128 (w % 2) .. + 127 as 4 x 4 MFMA
// blocks (256 accumulation registers). With one wave per SIMD every stall of
// the wave idles the matrix core, so the K loop is one inline-assembly block
// (gemm_loop_4w.inc, written and checked by gen_gemm_loop.py) that places
// each LDS read, LDS-direct load, wait and barrier between the MFMAs; a
// compiler-scheduled form of the same tile lost 5-14% to the 8-wave kernel,
// waiting on whole groups of reads mid-stream. Same LDS row layout and
// swizzle as the 8-wave tile, with the operands apart and all 160 KB of LDS
// in use: A (activations, mostly cache hits) in two stages of 32 KB at 0,
// loaded one panel ahead; B (weights, streamed from HBM) in three at 64 KB,
// loaded two panels ahead (the load waits at the panel hand-off fell from
// 5.8% to 2.4% of the loop, gate/up 2% faster). fp16 operands only, K a
// multiple of 64, and every byte offset into A and B below 4 GiB (the loads
// take 32-bit offsets from 64-bit bases).
template <class ARow, class BRow>
__device__ __forceinline__ void mainloop_4w(const void *A, ARow arow, const void *B, BRow brow,
                                            int K, int kt0, int kt1, u32x4 *lds,
                                            f32x16 (&acc)[4][4]) {
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int wm = w >> 1, wn = w & 1;
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};
  const int n = kt1 - kt0;
  if (n <= 0) return;
  // The LDS byte address is the low half of the array's generic address.
  const uint32_t lb = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(lds));
  // LDS-direct load i of wave w fills tile rows (4 i + w) * 8 .. + 7; lane l
  // lands in physical chunk l % 8 of row l / 8 (so the four waves' load i
  // fill rows 32 i .. + 31, the rows of fragment i).
  uint32_t dA[8], dB[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int row = (i * 4 + w) * 8 + (lane >> 3);
    const int c = (lane & 7) ^ ((row >> 1) & 7);
    dA[i] = static_cast<uint32_t>(((size_t)arow(row) * K + c * 8) * 2 + (size_t)kt0 * 128);
    dB[i] = static_cast<uint32_t>(((size_t)brow(row) * K + c * 8) * 2 + (size_t)kt0 * 128);
  }
  // Fragment reads of k-step s: row (lane % 32) of the wave's first 32-row
  // block, chunk 2 s + lane / 32, swizzled; blocks 1..3 and the other
  // stages are immediate offsets (4 KB per block, 32 KB per stage), except
  // B's third stage, read from rdC = rdB + 64 KB (past the 16-bit offset).
  const int x = ((lane & 31) >> 1) & 7, hc = lane >> 5;
  uint32_t rdA[4], rdB[4], rdC[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    const uint32_t cp = (((2 * s + hc) ^ x) * 16);
    rdA[s] = lb + (wm * 128 + (lane & 31)) * 128 + cp;
    rdB[s] = lb + 65536 + (wn * 128 + (lane & 31)) * 128 + cp;
    rdC[s] = rdB[s] + 65536;
  }
  const uint32_t mw = __builtin_amdgcn_readfirstlane(lb + w * 1024);
  int np = __builtin_amdgcn_readfirstlane(n);
  u32x4 fa00, fa01, fa02, fa03, fb00, fb01, fb02, fb03;
  u32x4 fa10, fa11, fa12, fa13, fb10, fb11, fb12, fb13;
  // M0 is a reserved register, so its clobber draws a note that the
  // compiler may not preserve it: nothing in these kernels keeps a value in
  // M0 across the block (the loads set it before each use).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
  asm volatile(
#include "gemm_loop_4w.inc"
      : [c00] "+a"(acc[0][0]), [c01] "+a"(acc[0][1]), [c02] "+a"(acc[0][2]), [c03] "+a"(acc[0][3]),
        [c10] "+a"(acc[1][0]), [c11] "+a"(acc[1][1]), [c12] "+a"(acc[1][2]), [c13] "+a"(acc[1][3]),
        [c20] "+a"(acc[2][0]), [c21] "+a"(acc[2][1]), [c22] "+a"(acc[2][2]), [c23] "+a"(acc[2][3]),
        [c30] "+a"(acc[3][0]), [c31] "+a"(acc[3][1]), [c32] "+a"(acc[3][2]), [c33] "+a"(acc[3][3]),
        [fa00] "=&v"(fa00), [fa01] "=&v"(fa01), [fa02] "=&v"(fa02), [fa03] "=&v"(fa03),
        [fb00] "=&v"(fb00), [fb01] "=&v"(fb01), [fb02] "=&v"(fb02), [fb03] "=&v"(fb03),
        [fa10] "=&v"(fa10), [fa11] "=&v"(fa11), [fa12] "=&v"(fa12), [fa13] "=&v"(fa13),
        [fb10] "=&v"(fb10), [fb11] "=&v"(fb11), [fb12] "=&v"(fb12), [fb13] "=&v"(fb13),
        [dA0] "+v"(dA[0]), [dA1] "+v"(dA[1]), [dA2] "+v"(dA[2]), [dA3] "+v"(dA[3]),
        [dA4] "+v"(dA[4]), [dA5] "+v"(dA[5]), [dA6] "+v"(dA[6]), [dA7] "+v"(dA[7]),
        [dB0] "+v"(dB[0]), [dB1] "+v"(dB[1]), [dB2] "+v"(dB[2]), [dB3] "+v"(dB[3]),
        [dB4] "+v"(dB[4]), [dB5] "+v"(dB[5]), [dB6] "+v"(dB[6]), [dB7] "+v"(dB[7]),
        [n] "+s"(np)
      : [rdA0] "v"(rdA[0]), [rdA1] "v"(rdA[1]), [rdA2] "v"(rdA[2]), [rdA3] "v"(rdA[3]),
        [rdB0] "v"(rdB[0]), [rdB1] "v"(rdB[1]), [rdB2] "v"(rdB[2]), [rdB3] "v"(rdB[3]),
        [rdC0] "v"(rdC[0]), [rdC1] "v"(rdC[1]), [rdC2] "v"(rdC[2]), [rdC3] "v"(rdC[3]),
        [pa] "s"(A), [pb] "s"(B), [mw] "s"(mw)
      : "memory", "m0", "scc");
#pragma clang diagnostic pop
}

// Tile row of accumulator register r of block row i (four-wave tile).
__device__ __forceinline__ int row_4w(int wm, int i, int r, int lane) {
  return wm * 128 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
}

// Raw fp32 partial tile of a split block, the 8-wave tile's layout.
__device__ __forceinline__ void store_partial_4w(const f32x16 (&acc)[4][4], float *part,
                                                 const Launch &ln, const Work &wk) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, wm = w >> 1, wn = w & 1;
  float *p = part + ((long)wk.tail * ln.nsplit + wk.split) * kTileElems;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int col = wn * 128 + j * 32 + (lane & 31);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) p[row_4w(wm, i, r, lane) * 256 + col] = acc[i][j][r];
  }
}

// x += A . W^T on the four-wave tile (fp16 weights, unsplit activations).
// The residual values of two block rows (32 per lane) are loaded before any
// of them is stored back: the compiler cannot move a load of x above a
// store to x, and 64 at a time spilled registers.
__global__ __launch_bounds__(256) void k_gemm_residual_4w(const f16 *__restrict__ A,
                                                          const uint16_t *__restrict__ W,
                                                          int rows, int N, int K, Launch ln,
                                                          float *__restrict__ x,
                                                          float *__restrict__ part) {
  __shared__ u32x4 lds[10240];  // A: 2 stages, B: 3 stages of 32 KB
  const Work wk = block_work(ln);
  const int m0 = wk.tm * 256, n0 = wk.tn * 256;
  const bool split = wk.tail >= 0;
  int k0 = 0, k1 = K / BK;
  if (split) split_range(k1, ln.nsplit, wk.split, k0, k1);
  f32x16 acc[4][4];
  mainloop_4w(
      A, [=](int r) { return min(m0 + r, rows - 1); }, W,
      [=](int r) { return min(n0 + r, N - 1); }, K, k0, k1, lds, acc);
  if (split) {
    store_partial_4w(acc, part, ln, wk);
    return;
  }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, wm = w >> 1, wn = w & 1;
  residual_epilogue<4>(acc, m0 + wm * 128 + 4 * (lane >> 5), n0 + wn * 128 + (lane & 31), rows, N,
                       x);
}

// Gate/up projection + SwiGLU on the four-wave tile (fp16 weights, unsplit
// activations). A wave's 128 B rows are 64 gate + 64 up rows, as in the
// 8-wave kernel, so block columns j and j + 2 pair up in one lane.
__global__ __launch_bounds__(256) void k_gemm_swiglu_4w(const f16 *__restrict__ A,
                                                        const uint16_t *__restrict__ W, int rows,
                                                        int F, int K, Launch ln,
                                                        f16 *__restrict__ h,
                                                        float *__restrict__ part) {
  __shared__ u32x4 lds[10240];  // A: 2 stages, B: 3 stages of 32 KB
  const Work wk = block_work(ln);
  const int m0 = wk.tm * 256, o0 = wk.tn * 128;
  const bool split = wk.tail >= 0;
  int k0 = 0, k1 = K / BK;
  if (split) split_range(k1, ln.nsplit, wk.split, k0, k1);
  f32x16 acc[4][4];
  mainloop_4w(
      A, [=](int r) { return min(m0 + r, rows - 1); }, W,
      [=](int r) {
        const int q = r & 127;
        const int oc = min(o0 + (r >> 7) * 64 + (q & 63), F - 1);
        return q < 64 ? oc : F + oc;
      },
      K, k0, k1, lds, acc);
  if (split) {
    store_partial_4w(acc, part, ln, wk);
    return;
  }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, wm = w >> 1, wn = w & 1;
  if (m0 + 256 <= rows && o0 + 128 <= F && (F & 1) == 0) {
    // Adjacent lanes trade values so each writes two adjacent columns of one
    // row with one 4-byte store (as in the 8-wave kernel).
    const bool odd = lane & 1;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int c0 = o0 + wn * 64 + j * 32 + (lane & 30);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          const float a = silu_mul(acc[i][j][2 * k], acc[i][j + 2][2 * k]);
          const float b = silu_mul(acc[i][j][2 * k + 1], acc[i][j + 2][2 * k + 1]);
          const float got = __int_as_float(
              __builtin_amdgcn_update_dpp(0, __float_as_int(odd ? a : b), 0xB1, 0xF, 0xF, false));
          const float v0 = odd ? got : a, v1 = odd ? b : got;
          const int row = m0 + row_4w(wm, i, 2 * k + (odd ? 1 : 0), lane);
          *reinterpret_cast<f16x2 *>(h + (long)row * F + c0) =
              f16x2{static_cast<f16>(v0), static_cast<f16>(v1)};
        }
    }
    return;
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int col = o0 + wn * 64 + j * 32 + (lane & 31);
    if (col >= F) continue;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + row_4w(wm, i, r, lane);
        if (row < rows) h[(long)row * F + col] = static_cast<f16>(silu_mul(acc[i][j][r], acc[i][j + 2][r]));
      }
  }
}

// Tail tiles: h = silu(gate) * up from the summed partials. Block (tail tile,
// half of its 256 rows); thread -> (row, output column oc < 128).
template <int NS>
__global__ __launch_bounds__(256) void k_reduce_swiglu(const float *__restrict__ part,
                                                       Launch ln, int rows, int F, int hsplit,
                                                       f16 *__restrict__ h) {
  const int i = blockIdx.x / 128, e = (blockIdx.x % 128) * 256 + threadIdx.x;
  int tm, tn;
  tile_coords(ln.ndp + i, ln.nm, ln.nn, ln.gm, tm, tn);
  const int lr = e / 128, oc = e % 128;
  const int row = tm * 256 + lr, o = tn * 128 + oc;
  if (row >= rows || o >= F) return;
  const int cg = (oc / 64) * 128 + oc % 64;
  const float g = sum_partials<NS>(part, i, lr * 256 + cg);
  const float u = sum_partials<NS>(part, i, lr * 256 + cg + 64);
  store_act(h, (long)row * F * hsplit, o, F, hsplit, silu_mul(g, u));
}

// ------------------------------------------------- QKV + rotary + KV caches
// Staged stores. A 64-row block of one head slot (a wave's outputs, or a
// quarter of a summed tail tile) passes through 16 KB of LDS and leaves in
// 16-byte stores, each store instruction covering whole 128-byte lines.
// Stored straight from the accumulators, a lane wrote 2 bytes: a value tile,
// transposed into the Vt cache, touched 64 lines per store instruction.
//
// Row form (queries, keys): [64 rows][128 dims], 256 B a row; chunk c of row
// s sits at c ^ 4 ((s / 4) % 2), so the rows s and s + 4 written by the two
// half-waves of one accumulator register fall in different banks.
__device__ __forceinline__ int stg_row(int s, int d) {
  return s * 128 + (((d >> 3) ^ (((s >> 2) & 1) << 2)) << 3) + (d & 7);
}
// Transposed form (values): [128 dims][64 cache positions], 128 B a dim;
// chunk C of dim e sits at C ^ ((e / 2) % 8).
__device__ __forceinline__ int stg_vt(int e, int p) {
  return e * 64 + (((p >> 3) ^ ((e >> 1) & 7)) << 3) + (p & 7);
}
// Position (within its aligned group of 16) that the Vt interleave gives
// position p: quarters 1 and 2 swap. Groups of 4 stay contiguous.
__device__ __forceinline__ int vt_interleave(int p) {
  return (p & ~12) | ((p & 4) << 1) | ((p & 8) >> 1);
}

__device__ __forceinline__ bool aligned16(const void *p) {
  return (reinterpret_cast<uintptr_t>(p) & 15) == 0;
}

// Destination of a staged 64-row block of a value slot: Vt cache rows at
// positions crow0 .. crow0 + 63. Only blocks whose rows are all valid, lie
// in one cache and start at a multiple of 16 there (the interleave then maps
// the block onto itself) are staged; the rest are stored element by element.
struct VtBlock {
  f16 *vt;
  int npos, crow0;
};
__device__ __forceinline__ bool vt_block(const QKVOut<f16> &o, int n_heads, int n_kv, int slot,
                                         int r0, int rows, VtBlock &b) {
  if (o.cache_row || r0 + 64 > rows) return false;
  const bool first = r0 + 64 <= o.split;
  const bool second = r0 >= o.split && (o.split & 15) == 0;
  if (!first && !second) return false;
  b.npos = second ? o.kv_npos2 : o.kv_npos;
  f16 *vt = second ? o.vt2 : o.vt;
  b.vt = vt + (long)(slot - n_heads - n_kv) * 128 * b.npos;
  b.crow0 = second ? r0 - o.split : r0;
  return (b.npos & 7) == 0 && aligned16(vt);
}

// Query and key destinations 16-byte aligned (their rows are 256 B).
__device__ __forceinline__ bool qk_staged_ok(const QKVOut<f16> &o) {
  return aligned16(o.q) && aligned16(o.k) && aligned16(o.k2);
}

// Destination of row `row` of query / key slot `slot`; NULL past the rows.
__device__ __forceinline__ f16 *qk_row_dst(const QKVOut<f16> &o, int n_heads, int slot, int row,
                                           int rows) {
  if (row >= rows) return nullptr;
  if (slot < n_heads) return o.q + ((long)row * n_heads + slot) * 128;
  const bool second = row >= o.split;
  f16 *k = second ? o.k2 : o.k;
  const int crow = second ? row - o.split : o.cache_row ? o.cache_row[row] : row;
  const int npos = second ? o.kv_npos2 : o.kv_npos;
  return k + ((long)(slot - n_heads) * npos + crow) * 128;
}

// Copy-out of a staged block by one wave: store rounds it0 .. it0 + NIT - 1
// of 16 (a round: 64 lanes x 16 B, 4 rows or 8 dims).
template <int NIT>
__device__ __forceinline__ void qk_copy_out(const f16 *stg, const QKVOut<f16> &o, int n_heads,
                                            int slot, int r0, int rows, int it0) {
  const int lane = threadIdx.x & 63;
#pragma unroll 2
  for (int it = it0; it < it0 + NIT; ++it) {
    const int s = it * 4 + (lane >> 4), c = lane & 15;
    const u32x4 v = *reinterpret_cast<const u32x4 *>(stg + stg_row(s, c * 8));
    f16 *p = qk_row_dst(o, n_heads, slot, r0 + s, rows);
    if (p) *reinterpret_cast<u32x4 *>(p + c * 8) = v;
  }
}
template <int NIT>
__device__ __forceinline__ void vt_copy_out(const f16 *stg, f16 *dst, int npos, int crow0, int it0) {
  const int lane = threadIdx.x & 63;
#pragma unroll 2
  for (int it = it0; it < it0 + NIT; ++it) {
    const int e = it * 8 + (lane >> 3), c = lane & 7;
    const u32x4 v = *reinterpret_cast<const u32x4 *>(stg + stg_vt(e, c * 8));
    *reinterpret_cast<u32x4 *>(dst + (long)e * npos + crow0 + c * 8) = v;
  }
}

// Column tile = two heads of the stacked q|k|v projection; wave column wn owns
// head slot 2 tn + wn. MFMA blocks fn and fn+2 hold head dims d and d + 64,
// the rotate-half pair.
template <class TL, bool WCVT>
__global__ __launch_bounds__(NT) void k_gemm_qkv(const f16 *__restrict__ A,
                                                 const uint16_t *__restrict__ W, int rows,
                                                 int K, int asplit, int n_heads, int n_kv,
                                                 Launch ln,
                                                 QKVOut<f16> o, float *__restrict__ part) {
  static_assert(TL::WN == 2 && TL::TN == 128 && TL::BN == 256, "one head per wave column");
  static_assert(TL::TM == 64 && TL::STAGE * 2 >= NWAVES * 1024, "a 16 KB staging block per wave");
  __shared__ u32x4 lds[2 * TL::STAGE];
  const Work wk = block_work(ln);
  const int nslots = n_heads + 2 * n_kv, nrows = nslots * 128;
  const int m0 = wk.tm * TL::BM, n0 = wk.tn * 256;
  const bool split = wk.tail >= 0;
  int k0 = 0, k1 = K / BK * asplit;
  if (split) split_range(k1, ln.nsplit, wk.split, k0, k1);
  f32x16 acc[TL::FM][TL::FN];
  mainloop<TL, false, WCVT>(
      A, [=](int r) { return min(m0 + r, rows - 1); }, W,
      [=](int r) { return min(n0 + r, nrows - 1); }, K, asplit, k0, k1, lds, acc);
  if (split) {
    store_partial<TL>(acc, part, ln, wk);
    return;
  }
  // The main loop ends on a barrier after its last LDS reads, so each wave
  // may now use its own 16 KB of the ring as a staging block. Precise layers
  // (remainder planes too) store element by element.
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w / TL::WN, wn = w % TL::WN;
  const int slot = wk.tn * 2 + wn;
  if (slot >= nslots) return;
  const int r0 = m0 + wm * TL::TM;
  const bool precise = o.q_lo || o.k_lo || o.vt_lo;
  f16 *stg = reinterpret_cast<f16 *>(lds + w * 1024);
  if (slot >= n_heads + n_kv) {  // values: no rotary
    VtBlock vb;
    if (!precise && vt_block(o, n_heads, n_kv, slot, r0, rows, vb)) {
      // Lane rows 8 q + 4 (lane / 32) + j (j < 4) of MFMA row block fm go to
      // interleaved positions 32 fm + 16 (q / 2) + 8 (lane / 32) + 4 (q % 2) + j.
#pragma unroll
      for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < TL::FN; ++fn)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            f16x4 h;
#pragma unroll
            for (int j = 0; j < 4; ++j) h[j] = static_cast<f16>(acc[fm][fn][4 * q + j]);
            const int p = 32 * fm + 16 * (q >> 1) + 8 * (lane >> 5) + 4 * (q & 1);
            *reinterpret_cast<f16x4 *>(stg + stg_vt(fn * 32 + (lane & 31), p)) = h;
          }
      vt_copy_out<16>(stg, vb.vt, vb.npos, vb.crow0, 0);
      return;
    }
#pragma unroll
    for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + acc_row<TL>(wm, fm, r, lane);
        if (row >= rows) continue;
#pragma unroll
        for (int fn = 0; fn < 2; ++fn)
          qkv_store_rotated(o, n_heads, n_kv, slot, row, fn * 32 + (lane & 31), acc[fm][fn][r],
                            acc[fm][fn + 2][r]);
      }
    return;
  }
  // Queries and keys: the positions and rotary-table entries of a block's 16
  // rows are all loaded before any of them is used. (Loaded row by row
  // between stores, they waited out two memory round trips per row: the
  // compiler cannot move a load above a store that may alias it.)
  const bool staged = !precise && qk_staged_ok(o);
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm) {
    int pos[16];
#pragma unroll
    for (int r = 0; r < 16; ++r)
      pos[r] = qkv_row_pos(o, min(m0 + acc_row<TL>(wm, fm, r, lane), rows - 1));
    float2 cs[16][2];
#pragma unroll
    for (int r = 0; r < 16; ++r)
#pragma unroll
      for (int fn = 0; fn < 2; ++fn) cs[r][fn] = o.rope[(long)pos[r] * 64 + fn * 32 + (lane & 31)];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = m0 + acc_row<TL>(wm, fm, r, lane);
#pragma unroll
      for (int fn = 0; fn < 2; ++fn) {
        const int d = fn * 32 + (lane & 31);
        if (staged) {
          float x1 = acc[fm][fn][r], x2 = acc[fm][fn + 2][r];
          qk_turn(o, n_heads, n_kv, slot, x1, x2, cs[r][fn]);
          const int sr = acc_row<TL>(0, fm, r, lane);
          stg[stg_row(sr, d)] = static_cast<f16>(x1);
          stg[stg_row(sr, d + 64)] = static_cast<f16>(x2);
        } else if (row < rows) {
          qkv_store_cs(o, n_heads, n_kv, slot, row, d, acc[fm][fn][r], acc[fm][fn + 2][r],
                       cs[r][fn]);
        }
      }
    }
  }
  if (staged) qk_copy_out<16>(stg, o, n_heads, slot, r0, rows, 0);
}

// Tail tiles: the partials summed in split order, then the rotary and the
// staged stores as above. Block (tail tile, 64-row quarter), 4 waves: wave w
// sums head h = w % 2 of the pair for the 4-row groups g = 2 it + w / 2
// (it < 8), then stores its half of that head's staging block.
template <int NS>
__global__ __launch_bounds__(256) void k_reduce_qkv(const float *__restrict__ part, Launch ln,
                                                    int rows, int n_heads, int n_kv,
                                                    QKVOut<f16> o) {
  __shared__ u32x4 lds[2 * 1024];  // a 16 KB staging block per head
  const int i = blockIdx.x >> 2, quarter = blockIdx.x & 3;
  int tm, tn;
  tile_coords(ln.ndp + i, ln.nm, ln.nn, ln.gm, tm, tn);
  const int w = threadIdx.x >> 6, h = w & 1, d = threadIdx.x & 63;
  const int slot = tn * 2 + h, nslots = n_heads + 2 * n_kv;
  const bool live = slot < nslots, value = slot >= n_heads + n_kv;
  const int r0 = tm * 256 + quarter * 64;
  f16 *stg = reinterpret_cast<f16 *>(lds + h * 1024);
  const bool precise = o.q_lo || o.k_lo || o.vt_lo;
  VtBlock vb;
  const bool staged = live && !precise &&
                      (value ? vt_block(o, n_heads, n_kv, slot, r0, rows, vb) : qk_staged_ok(o));
  // The rotary entries of the thread's 32 rows, loaded before the loop (in
  // it they waited out two memory round trips per row group: the position,
  // then the entry).
  float2 cs[8][4];
  if (live && !value) {
    int pos[8][4];
#pragma unroll
    for (int it = 0; it < 8; ++it)
#pragma unroll
      for (int j = 0; j < 4; ++j)
        pos[it][j] = qkv_row_pos(o, min(r0 + 4 * (2 * it + (w >> 1)) + j, rows - 1));
#pragma unroll
    for (int it = 0; it < 8; ++it)
#pragma unroll
      for (int j = 0; j < 4; ++j) cs[it][j] = o.rope[(long)pos[it][j] * 64 + d];
  }
#pragma unroll
  for (int it = 0; it < 8; ++it) {
    const int g = 2 * it + (w >> 1);
    float x1[4], x2[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = (quarter * 64 + 4 * g + j) * 256 + h * 128 + d;
      x1[j] = sum_partials<NS>(part, i, e);
      x2[j] = sum_partials<NS>(part, i, e + 64);
    }
    if (!live) continue;
    if (!value) {
#pragma unroll
      for (int j = 0; j < 4; ++j) qk_turn(o, n_heads, n_kv, slot, x1[j], x2[j], cs[it][j]);
    }
    if (!staged) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (r0 + 4 * g + j < rows)
          qkv_store_rotated(o, n_heads, n_kv, slot, r0 + 4 * g + j, d, x1[j], x2[j]);
    } else if (value) {
      f16x4 a, b;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        a[j] = static_cast<f16>(x1[j]);
        b[j] = static_cast<f16>(x2[j]);
      }
      const int p = vt_interleave(4 * g);
      *reinterpret_cast<f16x4 *>(stg + stg_vt(d, p)) = a;
      *reinterpret_cast<f16x4 *>(stg + stg_vt(d + 64, p)) = b;
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        stg[stg_row(4 * g + j, d)] = static_cast<f16>(x1[j]);
        stg[stg_row(4 * g + j, d + 64)] = static_cast<f16>(x2[j]);
      }
    }
  }
  __syncthreads();
  if (!staged) return;
  if (value)
    vt_copy_out<8>(stg, vb.vt, vb.npos, vb.crow0, 8 * (w >> 1));
  else
    qk_copy_out<8>(stg, o, n_heads, slot, r0, rows, 8 * (w >> 1));
}

// ------------------------------------------------------ LM head + chunk LSE
// Transposed product: the MFMA rows are vocabulary entries (A = W_lm) and the
// columns are scored tokens (B = normed hidden rows), so a token's reduction
// over the vocabulary runs down a lane's registers, across the two lane
// halves and across the WM waves of a column. Block (vocab tile c, token
// tile) writes, for each token t, part[c][t] = (max_v l, sum_v exp(l - max))
// over its BM vocabulary rows, and the target logit when the target falls in
// the tile. The [tokens x vocab] logits never leave registers.
template <class TL, bool WCVT>
__global__ __launch_bounds__(NT) void k_gemm_lmhead(const f16 *__restrict__ Hn,
                                                    const uint16_t *__restrict__ Wlm, int T,
                                                    int vocab, int K, Launch ln,
                                                    const int32_t *__restrict__ lm_tgt,
                                                    float2 *__restrict__ part,
                                                    float *__restrict__ tgt_logit) {
  __shared__ u32x4 lds[2 * TL::STAGE];
  __shared__ float red[TL::WM][TL::BN];
  const Work wk = block_work(ln);
  const int m0 = wk.tm * TL::BM, n0 = wk.tn * TL::BN;
  f32x16 acc[TL::FM][TL::FN];
  mainloop<TL, WCVT, false>(
      Wlm, [=](int r) { return min(m0 + r, vocab - 1); }, Hn,
      [=](int r) { return min(n0 + r, T - 1); }, K, 1, 0, K / BK, lds, acc);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w / TL::WN, wn = w % TL::WN;

  float mx[TL::FN];
#pragma unroll
  for (int fn = 0; fn < TL::FN; ++fn) {
    float v = -INFINITY;
#pragma unroll
    for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (m0 + acc_row<TL>(wm, fm, r, lane) < vocab) v = fmaxf(v, acc[fm][fn][r]);
    v = fmaxf(v, __shfl_xor(v, 32, 64));
    if (lane < 32) red[wm][acc_col<TL>(wn, fn, lane)] = v;
  }
  __syncthreads();
#pragma unroll
  for (int fn = 0; fn < TL::FN; ++fn) {
    const int c = acc_col<TL>(wn, fn, lane);
    float v = red[0][c];
#pragma unroll
    for (int i = 1; i < TL::WM; ++i) v = fmaxf(v, red[i][c]);
    mx[fn] = v;
  }
  __syncthreads();
#pragma unroll
  for (int fn = 0; fn < TL::FN; ++fn) {
    float s = 0.f;
#pragma unroll
    for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (m0 + acc_row<TL>(wm, fm, r, lane) < vocab) s += __expf(acc[fm][fn][r] - mx[fn]);
    s += __shfl_xor(s, 32, 64);
    if (lane < 32) red[wm][acc_col<TL>(wn, fn, lane)] = s;
  }
  __syncthreads();
#pragma unroll
  for (int fn = 0; fn < TL::FN; ++fn) {
    const int c = acc_col<TL>(wn, fn, lane);
    const int t = n0 + c;
    if (t >= T) continue;
    if (wm == 0 && lane < 32) {
      float s = red[0][c];
#pragma unroll
      for (int i = 1; i < TL::WM; ++i) s += red[i][c];
      part[(long)wk.tm * T + t] = make_float2(mx[fn], s);
    }
    // Target logit: row tr of this wave's sub-tile, held by lane half
    // (tr / 4) % 2 in register 4 (tr % 32 / 8) + tr % 4 of block tr / 32.
    const int tr = lm_tgt[t] - m0 - wm * TL::TM;
    if (tr >= 0 && tr < TL::TM && ((tr >> 2) & 1) == (lane >> 5)) {
      const int fm_t = tr >> 5, w32 = tr & 31, rr = (w32 >> 3) * 4 + (w32 & 3);
      float v = 0.f;
#pragma unroll
      for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (fm == fm_t && r == rr) v = acc[fm][fn][r];
      tgt_logit[t] = v;
    }
  }
}

// The LM head on the four-wave tile (fp16 weights): the same transposed
// product and partials, 128 vocabulary rows x 128 tokens per wave, so a
// token's reduction runs down a lane's registers, across the lane halves and
// across the two waves of a token column. The main loop fills all of LDS;
// after a barrier its first 4 KB hold the cross-wave values.
__global__ __launch_bounds__(256) void k_gemm_lmhead_4w(const f16 *__restrict__ Hn,
                                                        const uint16_t *__restrict__ Wlm, int T,
                                                        int vocab, int K, Launch ln,
                                                        const int32_t *__restrict__ lm_tgt,
                                                        float2 *__restrict__ part,
                                                        float *__restrict__ tgt_logit) {
  __shared__ u32x4 lds[10240];  // A: 2 stages, B: 3 stages of 32 KB
  const Work wk = block_work(ln);
  const int m0 = wk.tm * 256, n0 = wk.tn * 256;
  f32x16 acc[4][4];
  mainloop_4w(
      Wlm, [=](int r) { return min(m0 + r, vocab - 1); }, Hn,
      [=](int r) { return min(n0 + r, T - 1); }, K, 0, K / BK, lds, acc);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, wm = w >> 1, wn = w & 1;
  float (*red)[256] = reinterpret_cast<float (*)[256]>(lds);  // [4][256]
  __syncthreads();  // every wave is past its last LDS fragment reads
  float mx[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    float v = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (m0 + row_4w(wm, i, r, lane) < vocab) v = fmaxf(v, acc[i][j][r]);
    v = fmaxf(v, __shfl_xor(v, 32, 64));
    if (lane < 32) red[wm][wn * 128 + j * 32 + lane] = v;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int c = wn * 128 + j * 32 + (lane & 31);
    mx[j] = fmaxf(red[0][c], red[1][c]);
  }
  __syncthreads();
  // Sums of exp(l - max) per 64-row half of the wave, added in row order
  // across the halves: the order of the 8-wave kernel (four waves of 64
  // rows), so that fp16 and bf16 weight storage give bitwise equal scores.
#pragma unroll
  for (int j = 0; j < 4; ++j) {
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      float sum = 0.f;
#pragma unroll
      for (int i = 2 * hh; i < 2 * hh + 2; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (m0 + row_4w(wm, i, r, lane) < vocab) sum += __expf(acc[i][j][r] - mx[j]);
      sum += __shfl_xor(sum, 32, 64);
      if (lane < 32) red[2 * wm + hh][wn * 128 + j * 32 + lane] = sum;
    }
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int c = wn * 128 + j * 32 + (lane & 31);
    const int t = n0 + c;
    if (t >= T) continue;
    if (wm == 0 && lane < 32) {
      float sum = red[0][c];
#pragma unroll
      for (int q = 1; q < 4; ++q) sum += red[q][c];
      part[(long)wk.tm * T + t] = make_float2(mx[j], sum);
    }
    // Target logit: row tr of this wave's 128 rows, held by lane half
    // (tr / 4) % 2 in register 4 (tr % 32 / 8) + tr % 4 of block row tr / 32.
    const int tr = lm_tgt[t] - m0 - wm * 128;
    if (tr >= 0 && tr < 128 && ((tr >> 2) & 1) == (lane >> 5)) {
      const int it = tr >> 5, w32 = tr & 31, rr = (w32 >> 3) * 4 + (w32 & 3);
      float v = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (i == it && r == rr) v = acc[i][j][r];
      tgt_logit[t] = v;
    }
  }
}

// Greedy variant of the LM head: per (vocab tile, token) the largest logit and
// its vocabulary index (the lowest on ties), part[c][t] = (max, index bits).
template <class TL, bool WCVT>
__global__ __launch_bounds__(NT) void k_gemm_lmargmax(const f16 *__restrict__ Hn,
                                                      const uint16_t *__restrict__ Wlm, int T,
                                                      int vocab, int K, Launch ln,
                                                      float2 *__restrict__ part) {
  __shared__ u32x4 lds[2 * TL::STAGE];
  __shared__ float redv[TL::WM][TL::BN];
  __shared__ int redi[TL::WM][TL::BN];
  const Work wk = block_work(ln);
  const int m0 = wk.tm * TL::BM, n0 = wk.tn * TL::BN;
  f32x16 acc[TL::FM][TL::FN];
  mainloop<TL, WCVT, false>(
      Wlm, [=](int r) { return min(m0 + r, vocab - 1); }, Hn,
      [=](int r) { return min(n0 + r, T - 1); }, K, 1, 0, K / BK, lds, acc);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w / TL::WN, wn = w % TL::WN;
#pragma unroll
  for (int fn = 0; fn < TL::FN; ++fn) {
    float v = -INFINITY;
    int vi = -1;
    // Rows increase with (fm, r) in a lane, so a strict > keeps the lowest.
#pragma unroll
    for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + acc_row<TL>(wm, fm, r, lane);
        if (row < vocab && (vi < 0 || acc[fm][fn][r] > v)) {
          v = acc[fm][fn][r];
          vi = row;
        }
      }
    const float v2 = __shfl_xor(v, 32, 64);
    const int i2 = __shfl_xor(vi, 32, 64);
    if (i2 >= 0 && (vi < 0 || v2 > v || (v2 == v && i2 < vi))) {
      v = v2;
      vi = i2;
    }
    if (lane < 32) {
      redv[wm][acc_col<TL>(wn, fn, lane)] = v;
      redi[wm][acc_col<TL>(wn, fn, lane)] = vi;
    }
  }
  __syncthreads();
  if (wm == 0 && lane < 32) {
#pragma unroll
    for (int fn = 0; fn < TL::FN; ++fn) {
      const int c = acc_col<TL>(wn, fn, lane);
      const int t = n0 + c;
      if (t >= T) continue;
      float v = redv[0][c];
      int vi = redi[0][c];
#pragma unroll
      for (int i = 1; i < TL::WM; ++i) {
        const float v2 = redv[i][c];
        const int i2 = redi[i][c];
        if (i2 >= 0 && (vi < 0 || v2 > v || (v2 == v && i2 < vi))) {
          v = v2;
          vi = i2;
        }
      }
      part[(long)wk.tm * T + t] = make_float2(v, __int_as_float(vi));
    }
  }
}

}  // namespace

size_t gemm_split_floats(int rows, int N, int K) {
  const Launch ln = plan_launch((rows + 255) / 256, (N + 255) / 256, 8, K / BK);  // K: A width
  return (size_t)ln.ntail * ln.nsplit * kTileElems;
}

// Where the four-wave kernels run: bit 0 the gate/up projection, bit 1 the
// residual projections with K >= kFourWaveMinK, bit 2 those with smaller K,
// bit 3 the LM head. Building with VSR_FOUR_WAVE=<mask> changes it (for
// comparisons).
#ifdef VSR_FOUR_WAVE
constexpr int kFourWave = VSR_FOUR_WAVE;
#else
constexpr int kFourWave = 3 | 8;
#endif
constexpr int kFourWaveMinK = 8192;

// The four-wave kernels' conditions: fp16 weights, unsplit activations, and
// 32-bit byte offsets reaching every operand row.
inline bool four_wave_ok(bool w_f16, int asplit, int rows, int nrows_w, int K) {
  return w_f16 && asplit == 1 && K % BK == 0 && (size_t)rows * K * 2 <= UINT32_MAX &&
         (size_t)nrows_w * K * 2 <= UINT32_MAX;
}

// Weight-format dispatch of a GEMM kernel launch.
#define VSR_WLAUNCH(kern, grid, ...)                                              \
  do {                                                                           \
    const uint16_t *W16 = static_cast<const uint16_t *>(W);                      \
    if (w_f16)                                                                   \
      kern<TL, false><<<grid, NT, 0, s>>>(__VA_ARGS__);                           \
    else                                                                         \
      kern<TL, true><<<grid, NT, 0, s>>>(__VA_ARGS__);                            \
  } while (0)

hipError_t gemm_residual(const f16 *A, const void *W, bool w_f16, int rows, int N, int K,
                         int asplit, float *x, float *part, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  typedef TileStd TL;
  // Both residual epilogues address x through buffer descriptors of 32-bit
  // byte ranges.
  if ((size_t)rows * N * 4 > INT32_MAX) return hipErrorInvalidValue;
  const Launch ln = plan_launch((rows + TL::BM - 1) / TL::BM, (N + TL::BN - 1) / TL::BN, 8,
                                K / BK * asplit);
  const int fw = K >= kFourWaveMinK ? 2 : 4;
  if ((kFourWave & fw) && four_wave_ok(w_f16, asplit, rows, N, K))
    k_gemm_residual_4w<<<ln.blocks(), 256, 0, s>>>(A, static_cast<const uint16_t *>(W), rows, N, K,
                                                     ln, x, part);
  else
    VSR_WLAUNCH(k_gemm_residual, ln.blocks(), A, W16, rows, N, K, asplit, ln, x, part);
  if (ln.ntail > 0)
    VSR_REDUCE_LAUNCH(ln.nsplit, k_reduce_residual, ln.ntail * 256, 256, part, ln, rows, N, x);
  return hipGetLastError();
}

hipError_t gemm_swiglu(const f16 *A, const void *W, bool w_f16, int rows, int F, int K,
                       int asplit, f16 *h, float *part, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  typedef TileStd TL;
  // Row-tile groups of at most 9, evenly sized (16 row tiles: 2 x 8; 18: 2 x
  // 9): measured 1.6% faster than groups of 8 on 4608 rows, where the last
  // group of 2 row tiles shares its operand panels poorly.
  const int nm = (rows + TL::BM - 1) / TL::BM;
  const int ng = (nm + 8) / 9;
  const Launch ln = plan_launch(nm, (F + 127) / 128, (nm + ng - 1) / ng, K / BK * asplit);
  // The four-wave tile with the ordered K loop where it applies (same
  // tiles, same partial layout).
  if ((kFourWave & 1) && four_wave_ok(w_f16, asplit, rows, 2 * F, K))
    k_gemm_swiglu_4w<<<ln.blocks(), 256, 0, s>>>(A, static_cast<const uint16_t *>(W), rows, F, K,
                                                   ln, h, part);
  else
    VSR_WLAUNCH(k_gemm_swiglu, ln.blocks(), A, W16, rows, F, K, asplit, ln, h, part);
  if (ln.ntail > 0)
    VSR_REDUCE_LAUNCH(ln.nsplit, k_reduce_swiglu, ln.ntail * 128, 256, part, ln, rows, F, asplit,
                      h);
  return hipGetLastError();
}

hipError_t gemm_qkv_rope(const f16 *A, const void *W, bool w_f16, int rows, int K, int asplit,
                         int n_heads, int n_kv, const QKVOut<f16> &out, float *part,
                         hipStream_t s) {
  if (rows == 0) return hipSuccess;
  typedef TileStd TL;
  const int nslots = n_heads + 2 * n_kv;
  const Launch ln = plan_launch((rows + TL::BM - 1) / TL::BM, (nslots + 1) / 2, 8,
                                K / BK * asplit);
  VSR_WLAUNCH(k_gemm_qkv, ln.blocks(), A, W16, rows, K, asplit, n_heads, n_kv, ln, out, part);
  if (ln.ntail > 0)
    VSR_REDUCE_LAUNCH(ln.nsplit, k_reduce_qkv, ln.ntail * 4, 256, part, ln, rows, n_heads, n_kv,
                      out);
  return hipGetLastError();
}

int lmhead_chunks(int vocab) { return (vocab + TileStd::BM - 1) / TileStd::BM; }

hipError_t gemm_lmhead(const f16 *A, const void *W, bool w_f16, int rows, int vocab, int K,
                       const int32_t *lm_tgt, float2 *part, float *tgt_logit, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  typedef TileStd TL;
  // Token tiles fastest (GM = 1): the blocks sharing a vocabulary tile run
  // together. No K split (every block writes whole-vocabulary-tile LSE
  // partials).
  const int nm = lmhead_chunks(vocab), nn = (rows + TL::BN - 1) / TL::BN;
  const Launch ln{nm, nn, 1, nm * nn, 0, 1};
  if ((kFourWave & 8) && four_wave_ok(w_f16, 1, vocab, rows, K))
    k_gemm_lmhead_4w<<<ln.blocks(), 256, 0, s>>>(A, static_cast<const uint16_t *>(W), rows, vocab,
                                                   K, ln, lm_tgt, part, tgt_logit);
  else
    VSR_WLAUNCH(k_gemm_lmhead, ln.blocks(), A, W16, rows, vocab, K, ln, lm_tgt, part, tgt_logit);
  return hipGetLastError();
}

hipError_t gemm_lmargmax(const f16 *A, const void *W, bool w_f16, int rows, int vocab, int K,
                         float2 *part, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  typedef TileStd TL;
  const int nm = lmhead_chunks(vocab), nn = (rows + TL::BN - 1) / TL::BN;
  const Launch ln{nm, nn, 1, nm * nn, 0, 1};
  VSR_WLAUNCH(k_gemm_lmargmax, ln.blocks(), A, W16, rows, vocab, K, ln, part);
  return hipGetLastError();
}

#undef VSR_WLAUNCH
#undef VSR_REDUCE_LAUNCH

namespace {
// Eight values per thread (16-byte loads and stores); the tail one by one.
__global__ __launch_bounds__(256) void k_bf16_to_f16(const u32x4 *src, u32x4 *dst, size_t n8,
                                                     const uint16_t *tsrc, uint16_t *tdst,
                                                     int ntail) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n8) dst[i] = bf16x8_to_f16x8(src[i]);
  if (i < (size_t)ntail) {
    const float v = __uint_as_float((uint32_t)tsrc[i] << 16);
    tdst[i] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(v, 0.f)) & 0xFFFFu;
  }
}
}  // namespace

hipError_t convert_bf16_to_f16(const uint16_t *src, uint16_t *dst, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const size_t n8 = n / 8, work = n8 > 8 ? n8 : 8;
  const int ntail = (int)(n % 8);
  k_bf16_to_f16<<<(unsigned)((work + 255) / 256), 256, 0, s>>>(
      reinterpret_cast<const u32x4 *>(src), reinterpret_cast<u32x4 *>(dst), n8, src + n8 * 8,
      dst + n8 * 8, ntail);
  return hipGetLastError();
}

}  // namespace vsr
