// Attention of the verifier scoring pass on the gfx950 matrix cores.
//
// One kernel serves the prefix prefill (causal) and the candidate pass
// (cascade: the shared prefix keys, then each candidate's own causal block).
// For KV head h the query rows of all G = n_heads / n_kv query heads that read
// it are stacked, row r = (token t0 + r / G, head h G + r % G), so every key
// tile staged in LDS is used by all of them -- and, in the candidate pass, by
// all M candidates at once: the prefix keys are read once per query tile, not
// once per candidate.
//
// A 512-thread block owns 256 stacked query rows (32 per wave, two waves per
// SIMD; each lane holds its query's operand chunks in registers) and walks
// 64-key tiles through a two-stage LDS ring filled by direct global->LDS
// loads. Each wave computes S^T = K . Q^T on MFMA 32x32x16 (keys
// as MFMA rows, queries as columns), so a lane owns one query's scores and
// every per-query softmax quantity is a per-lane scalar. The probabilities
// feed O^T += V^T . P^T straight from registers: the MFMA k-index of that
// product is permuted to the key order the S^T accumulator leaves in each
// lane, and the Vt cache stores positions in the matching order (within each
// aligned group of 16 positions the middle two quarters are swapped), so a
// lane's V^T operand is one 16-byte LDS read. Softmax runs online in fp32
// with c = log2(e) / sqrt(hd): the fast kernels take queries already
// multiplied by c (the QKV epilogue does it), start the S^T products from -m
// so each probability is one exp2, and add the row sums with v_dot2 over the
// fp16 probabilities; the precise kernels keep the reference on the raw
// scores, exp2(s * c - m * c). Either way the reference moves (and the
// output is rescaled) only when a tile's maximum exceeds it by a factor 2^8
// after scaling. A query's 64 keys of a tile sit in two lanes (l, l ^ 32),
// combined by v_permlane32_swap; operands (queries, keys, values,
// probabilities) are fp16.
//
// The candidate and draft passes may split a block's keys (prefix tiles, then
// branch tiles) into chunks (more blocks on the chip); each chunk writes (max,
// sum, unnormalised output) partials and attn_merge combines them. Decode
// steps (at most 32 stacked query rows per KV head) run one-wave blocks.
//
// Precise variant (the leading layers of a deep model, where rounding is
// amplified most): queries, keys and values arrive as fp16 value + fp16
// remainder planes and the probabilities are split the same way; each product
// takes three MFMAs (hi.hi + hi.lo + lo.hi), which leaves an error of the
// order of fp32 rounding. Its blocks hold 128 query rows on 4 waves, whose
// query remainders also sit in registers.
#include <algorithm>

#include "common.h"

namespace vsr {

namespace {

constexpr int HD = 128;   // head dim of the MFMA path
constexpr int KT = 64;    // keys per tile
constexpr int KCH = KT * 16;   // 16-byte chunks of a K tile  [64 keys][128 dims]
constexpr int VCH = HD * 8;    // 16-byte chunks of a V^T tile [128 dims][64 keys]

// Block shape of the fast (PREC = false), precise (PREC = true) and decode
// (DEC: one wave, the draft pass's decode steps with at most 32 stacked query
// rows per KV head, where a wider block would mostly compute padding rows)
// variants. An LDS stage holds [K | V^T] tiles, precise: [K | V^T | K lo |
// V^T lo].
template <bool PREC, bool DEC = false>
struct Shape {
  static constexpr int NW = PREC ? 4 : (DEC ? 1 : 8);  // waves per block
  static constexpr int NT = NW * 64;
  static constexpr int QT = NW * 32;       // stacked query rows per block
  static constexpr int STAGE = (PREC ? 2 : 1) * (KCH + VCH);
};
constexpr int QT_FAST = Shape<false>::QT;

__device__ __forceinline__ f16x8 as_f16x8(u32x4 v) { return __builtin_bit_cast(f16x8, v); }

// LDS serves 256 bytes (64 banks) per cycle; the 16 lanes of a 16-byte load
// served together must hit distinct bank groups.
// K tile: a key row is 256 bytes (16 chunks); chunk c of key k at c ^ (k % 16).
__device__ __forceinline__ int ks_idx(int key, int c) { return key * 16 + (c ^ (key & 15)); }
// V^T tile: a row is 128 bytes (8 chunks), two rows per bank window; chunk c
// of row d at c ^ ((d / 2) % 8).
__device__ __forceinline__ int vs_idx(int d, int c) { return d * 8 + (c ^ ((d >> 1) & 7)); }

// Key visibility of one key segment.
enum SegMode { SEG_ALL = 0, SEG_CAUSAL = 1, SEG_BRANCH = 2 };

struct Seg {
  const f16 *k;    // [npos][HD] of this KV head
  const f16 *vt;   // [HD][npos] of this KV head (interleaved positions)
  const f16 *k_lo, *vt_lo;  // their remainder planes (precise variant)
  int npos;        // position stride of vt
  int kvalid;      // keys >= kvalid hold no data (never visible)
  int kbeg, kend;  // key range walked by the block: [kbeg, kend), kbeg % 64 == 0
  int mode;
  int tok_min;     // smallest query token of the block (mask-free tile test)
};

struct Lane {
  int tok;   // SEG_CAUSAL: the row's query token (its last visible key);
             // SEG_BRANCH: its last visible branch key (its own cache position)
  int lo;    // SEG_BRANCH: first visible key
  float m;   // reference of the exponents (raw score units): the running
             // maximum, moved only when a score exceeds it by more than thr
  float l;   // running sum of exp2(s * c - m * c) over this lane's half of
             // the keys (the halves are added once, after the walk)
  float thr; // 8 / c: probabilities stay below 2^8 between moves
  f32x16 o[HD / 32];
  f32x16 negm;  // fast kernels: -m in every element (the S^T products start from it)
  bool seen;    // fast kernels: a key of this query was visible (in either lane half)
  f16x8 qh[HD / 16], ql[HD / 16];  // chunks 2kk + h of the row (precise: hi / lo)
};

// Direct loads of key tile kb into an LDS stage. Load i of wave w fills K
// rows 4 (i NW + w) .. +3 and V^T rows 8 (i NW + w) .. +7; lane l lands in
// 16-byte slot l of that 1 KB, i.e. physical chunk l % 16 of K row l / 16, or
// l % 8 of V^T row l / 8; the global address carries the logical chunk.
// Addresses are a uniform tile base plus a 32-bit per-lane element offset
// (d * npos + c < 2^32: cache capacities are below 2^25 positions), which
// keeps the per-lane part of the addressing small.
template <int NW>
__device__ __forceinline__ void load_kv(const f16 *k, const f16 *vt, int npos, int kb,
                                        u32x4 *stage) {
  const int t = threadIdx.x, w = t >> 6, l = t & 63;
  const f16 *kt = k + (long)kb * HD, *vtt = vt + kb;
#pragma unroll
  for (int i = 0; i < KCH / (NW * 64); ++i) {
    const int j = i * NW + w, key = j * 4 + (l >> 4), c = (l & 15) ^ (key & 15);
    const unsigned off = (unsigned)(key * HD + c * 8);
    __builtin_amdgcn_global_load_lds(kt + off, stage + j * 64, 16, 0, 0);
  }
#pragma unroll
  for (int i = 0; i < VCH / (NW * 64); ++i) {
    const int j = i * NW + w, d = j * 8 + (l >> 3), c = (l & 7) ^ ((d >> 1) & 7);
    const unsigned off = (unsigned)d * (unsigned)npos + (unsigned)(c * 8);
    __builtin_amdgcn_global_load_lds(vtt + off, stage + KCH + j * 64, 16, 0, 0);
  }
}

template <bool PREC, bool DEC>
__device__ __forceinline__ void load_tile(const Seg &sg, int kb, u32x4 *stage) {
  constexpr int NW = Shape<PREC, DEC>::NW;
  load_kv<NW>(sg.k, sg.vt, sg.npos, kb, stage);
  if constexpr (PREC) load_kv<NW>(sg.k_lo, sg.vt_lo, sg.npos, kb, stage + KCH + VCH);
}

// Lane pairs (l, l ^ 32) hold the two halves of a query's keys; these
// combine a value over the pair through v_permlane32_swap (no LDS trip). The
// swap of x with itself leaves (x[l], x[l ^ 32]) in some order in every lane.
__device__ __forceinline__ float max_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  // r[0] is the lower-half lane's value in both halves: the same order in both.
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ f32x16 mfma(f16x8 a, f16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

// One 64-key tile against this wave's 32 query rows.
template <bool MASK, bool PREC>
__device__ __forceinline__ void tile_step(const Seg &sg, int kb, const u32x4 *st, Lane &L,
                                          float scale_log2) {
  const int lane = threadIdx.x & 63, h = lane >> 5;
  const u32x4 *Ks = st, *Vs = st + KCH;
  const u32x4 *Kl = st + KCH + VCH, *Vl = Kl + KCH;  // remainder planes (precise)
  f32x16 s[2] = {f32x16{}, f32x16{}};
#pragma unroll
  for (int kk = 0; kk < HD / 16; ++kk) {
    const f16x8 qf = L.qh[kk];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int ki = ks_idx(b * 32 + (lane & 31), 2 * kk + h);
      const f16x8 kf = as_f16x8(Ks[ki]);
      if constexpr (PREC) {
        s[b] = mfma(as_f16x8(Kl[ki]), qf, s[b]);
        s[b] = mfma(kf, L.ql[kk], s[b]);
      }
      s[b] = mfma(kf, qf, s[b]);
    }
  }
  // Mask; key of register r of block b: kb + 32b + 8(r/4) + 4h + r%4.
  float mloc = -INFINITY;
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      if constexpr (MASK) {
        const int key = kb + b * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
        bool vis = key < sg.kvalid;
        if (sg.mode == SEG_CAUSAL) vis = vis && key <= L.tok;
        if (sg.mode == SEG_BRANCH) vis = vis && key >= L.lo && key <= L.tok;
        s[b][r] = vis ? s[b][r] : -INFINITY;
      }
      mloc = fmaxf(mloc, s[b][r]);
    }
  mloc = max_halves(mloc);
  // Lazy reference: moving it costs a rescale of the 64 output accumulators,
  // so it moves only when this tile's maximum exceeds it by more than thr
  // (exp2 values below 2^8 stay exact to fp16's relative precision; l and o
  // share the reference, so the normalised output is unchanged).
  const float mnew = mloc > L.m + L.thr ? mloc : L.m;
  const float mref = mnew == -INFINITY ? 0.f : -mnew * scale_log2;  // exponent offset
  float psum = 0.f;
  f16x8 p[4], pl[4];
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float e = __builtin_amdgcn_exp2f(fmaf(s[b][r], scale_log2, mref));
      psum += e;
      const f16 eh = static_cast<f16>(e);
      p[b * 2 + (r >> 3)][r & 7] = eh;
      if constexpr (PREC) pl[b * 2 + (r >> 3)][r & 7] = static_cast<f16>(e - static_cast<float>(eh));
    }
  // Rescale when the reference of any lane of the wave moved (a wave-uniform
  // branch: the 64 multiplies are skipped in the common case, not predicated).
  const bool moved = mnew != L.m;
  if (__builtin_amdgcn_ballot_w64(moved)) {
    const float alpha = moved ? __builtin_amdgcn_exp2f(fmaf(L.m, scale_log2, mref)) : 1.f;
    L.l *= alpha;
#pragma unroll
    for (int db = 0; db < HD / 32; ++db) L.o[db] *= alpha;
  }
  L.l += psum;
  L.m = mnew;
  // O^T[d][q] += V^T[d][key] P^T[key][q]; for 16-key chunk c the MFMA k-index
  // 8h' + e of lane half h' is key 16c + 8(e/4) + 4h' + e%4, which the Vt
  // position interleave places at chunk 2c + h' of the row.
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int db = 0; db < HD / 32; ++db) {
      const int vi = vs_idx(db * 32 + (lane & 31), 2 * c + h);
      const f16x8 vf = as_f16x8(Vs[vi]);
      if constexpr (PREC) {
        L.o[db] = mfma(as_f16x8(Vl[vi]), p[c], L.o[db]);
        L.o[db] = mfma(vf, pl[c], L.o[db]);
      }
      L.o[db] = mfma(vf, p[c], L.o[db]);
    }
}

// Largest of the 32 scores a lane holds for one tile, as a tree of 3-input
// maxima (depth 4 instead of a chain of 16). All but one step take three
// inputs: the compiler turns those into v_max3 as they are, but precedes a
// two-input maximum with canonicalizing moves of both inputs (the two left
// over from 32 inputs join a[9]).
__device__ __forceinline__ float tile_max(const f32x16 (&s)[2]) {
  float a[10];
#pragma unroll
  for (int i = 0; i < 10; ++i) {
    const int j = 3 * i;
    a[i] = fmaxf(fmaxf(s[j >> 4][j & 15], s[(j + 1) >> 4][(j + 1) & 15]),
                 s[(j + 2) >> 4][(j + 2) & 15]);
  }
  const float b0 = fmaxf(fmaxf(a[0], a[1]), a[2]), b1 = fmaxf(fmaxf(a[3], a[4]), a[5]);
  const float b2 = fmaxf(fmaxf(a[6], a[7]), a[8]), b3 = fmaxf(fmaxf(a[9], s[1][14]), s[1][15]);
  return fmaxf(fmaxf(fmaxf(b0, b1), b2), b3);
}

// Fast kernels: one 64-key tile against this wave's 32 query rows: the
// scores, the probabilities and the PV products. The queries
// arrive multiplied by log2(e) / sqrt(hd), so S^T is in log2 units, and the
// products start from -m (L.negm), so the accumulators hold s - m and each
// probability is one exp2. The reference m moves (the output is rescaled)
// only when a tile's largest s - m exceeds 8, or at the first visible key of
// a row. The row sum adds the fp16 probabilities that the PV products use
// (v_dot2_f32_f16 against ones, fp32 accumulation).
__device__ __forceinline__ void scores_fast(const u32x4 *Ks, const Lane &L, f32x16 (&s)[2]) {
  const int lane = threadIdx.x & 63, h = lane >> 5;
#pragma unroll
  for (int kk = 0; kk < HD / 16; ++kk) {
    const f16x8 qf = L.qh[kk];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const f16x8 kf = as_f16x8(Ks[ks_idx(b * 32 + (lane & 31), 2 * kk + h)]);
      s[b] = mfma(kf, qf, kk == 0 ? L.negm : s[b]);
    }
  }
}

__device__ __forceinline__ void probs_fast(f32x16 (&s)[2], Lane &L, f16x8 (&p)[4]) {
  // t and seen are the same in both lane halves of a query, so the two halves
  // move together and keep one reference.
  const float t = max_halves(tile_max(s));
  const bool move = t > 8.f || (!L.seen && t != -INFINITY);
  if (__builtin_amdgcn_ballot_w64(move)) {
    // Rare: new reference m + d for the lanes that move (alpha rescales what
    // was summed against the old one; nothing was before the first visible key).
    const float d = move ? t : 0.f;
    const float alpha = L.seen ? __builtin_amdgcn_exp2f(-d) : 0.f;
    L.seen = L.seen || move;
    L.m += d;
    L.l *= alpha;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      L.negm[r] = -L.m;
      s[0][r] -= d;
      s[1][r] -= d;
    }
#pragma unroll
    for (int db = 0; db < HD / 32; ++db) L.o[db] *= alpha;
  }
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r)
      p[b * 2 + (r >> 3)][r & 7] = static_cast<f16>(__builtin_amdgcn_exp2f(s[b][r]));
  const f16x2 one = {static_cast<f16>(1.f), static_cast<f16>(1.f)};
  float ps[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    ps[c] = 0.f;
#pragma unroll
    for (int e = 0; e < 4; ++e)
      ps[c] = __builtin_amdgcn_fdot2(f16x2{p[c][2 * e], p[c][2 * e + 1]}, one, ps[c], false);
  }
  L.l += (ps[0] + ps[1]) + (ps[2] + ps[3]);
}

__device__ __forceinline__ void pv_fast(const u32x4 *Vs, const f16x8 (&p)[4], Lane &L) {
  const int lane = threadIdx.x & 63, h = lane >> 5;
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int db = 0; db < HD / 32; ++db) {
      const f16x8 vf = as_f16x8(Vs[vs_idx(db * 32 + (lane & 31), 2 * c + h)]);
      L.o[db] = mfma(vf, p[c], L.o[db]);
    }
}

// Scheduling order of a run of NSTEP steps of two LDS fragment reads and the
// two matrix products that use them: each step's reads are issued before the
// previous step's products, so a wave's LDS latency overlaps its own
// products (left to itself, the scheduler issues each pair of reads right
// before its products and waits for them).
template <int NSTEP>
__device__ __forceinline__ void order_reads_ahead() {
  __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);  // LDS reads
#pragma unroll
  for (int i = 1; i < NSTEP; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // matrix products
  }
  __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
}

template <bool MASK>
__device__ __forceinline__ void tile_step_fast(const Seg &sg, int kb, const u32x4 *st, Lane &L) {
  const int h = (threadIdx.x & 63) >> 5;
  f32x16 s[2];
  scores_fast(st, L, s);
  order_reads_ahead<8>();
  if constexpr (MASK) {
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = kb + b * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
        bool vis = key < sg.kvalid;
        if (sg.mode == SEG_CAUSAL) vis = vis && key <= L.tok;
        if (sg.mode == SEG_BRANCH) vis = vis && key >= L.lo && key <= L.tok;
        s[b][r] = vis ? s[b][r] : -INFINITY;
      }
  }
  f16x8 p[4];
  probs_fast(s, L, p);
  pv_fast(st + KCH, p, L);
  order_reads_ahead<8>();
}

// One tile of either variant.
template <bool MASK, bool PREC>
__device__ __forceinline__ void tile_any(const Seg &sg, int kb, const u32x4 *st, Lane &L,
                                         float scale_log2) {
  if constexpr (PREC)
    tile_step<MASK, true>(sg, kb, st, L, scale_log2);
  else
    tile_step_fast<MASK>(sg, kb, st, L);
}

// Whether tile kb can skip the per-key mask for every row of the block.
__device__ __forceinline__ bool tile_clear(const Seg &sg, int kb) {
  if (kb + KT > sg.kvalid) return false;
  if (sg.mode == SEG_CAUSAL) return kb + KT - 1 <= sg.tok_min;
  return sg.mode == SEG_ALL;
}

template <bool PREC, bool DEC>
__device__ __forceinline__ void walk_segment(const Seg &sg, u32x4 *lds, Lane &L,
                                             float scale_log2) {
  constexpr int STAGE = Shape<PREC, DEC>::STAGE;
  if (sg.kend <= sg.kbeg) return;
  load_tile<PREC, DEC>(sg, sg.kbeg, lds);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  // The mask-free tiles come first (tile_clear holds for a prefix of the
  // walk), so the two variants run in two loops: with one loop around both,
  // the fast kernels spilled about 20 registers inside it.
  // The mask-free loop is unrolled by two, one copy per stage, so that the
  // stage offset is an immediate of the LDS reads and their per-lane
  // addresses stay in registers across tiles.
  int stage = 0;
  int kb = sg.kbeg;
  while (kb < sg.kend && tile_clear(sg, kb)) {
    if (kb + KT < sg.kend) load_tile<PREC, DEC>(sg, kb + KT, lds + STAGE);
    tile_any<false, PREC>(sg, kb, lds, L, scale_log2);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    kb += KT;
    if (!(kb < sg.kend && tile_clear(sg, kb))) {
      stage = 1;
      break;
    }
    if (kb + KT < sg.kend) load_tile<PREC, DEC>(sg, kb + KT, lds);
    tile_any<false, PREC>(sg, kb, lds + STAGE, L, scale_log2);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    kb += KT;
  }
  for (; kb < sg.kend; kb += KT) {
    u32x4 *cur = lds + stage * STAGE;
    if (kb + KT < sg.kend) load_tile<PREC, DEC>(sg, kb + KT, lds + (stage ^ 1) * STAGE);
    tile_any<true, PREC>(sg, kb, cur, L, scale_log2);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    stage ^= 1;
  }
}

// Tiles v0 .. v1-1 of the concatenation [prefix tiles 0 .. pre_t-1 | branch
// tiles from key bbeg on]: one pipeline for both sources (the tile's source
// is chosen per tile), so that one set of load offsets is live.
template <bool PREC, bool DEC>
__device__ __forceinline__ void walk_concat(const Seg &sp, const Seg &sb, int pre_t, int bbeg,
                                            int v0, int v1, u32x4 *lds, Lane &L,
                                            float scale_log2) {
  constexpr int STAGE = Shape<PREC, DEC>::STAGE;
  if (v1 <= v0) return;
  auto src = [&](int v) -> const Seg & { return v < pre_t ? sp : sb; };
  auto key0 = [&](int v) { return v < pre_t ? v * KT : bbeg + (v - pre_t) * KT; };
  load_tile<PREC, DEC>(src(v0), key0(v0), lds);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  // Mask-free tiles first (whole prefix tiles), then the masked ones (a
  // short last prefix tile, the branch tiles), as in walk_segment.
  int stage = 0;
  int v = v0;
  for (; v < v1 && tile_clear(src(v), key0(v)); ++v) {
    u32x4 *cur = lds + stage * STAGE;
    if (v + 1 < v1) load_tile<PREC, DEC>(src(v + 1), key0(v + 1), lds + (stage ^ 1) * STAGE);
    tile_any<false, PREC>(src(v), key0(v), cur, L, scale_log2);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    stage ^= 1;
  }
  for (; v < v1; ++v) {
    u32x4 *cur = lds + stage * STAGE;
    if (v + 1 < v1) load_tile<PREC, DEC>(src(v + 1), key0(v + 1), lds + (stage ^ 1) * STAGE);
    tile_any<true, PREC>(src(v), key0(v), cur, L, scale_log2);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    stage ^= 1;
  }
}

// mode 0: prefill (causal over the prefix cache, one chunk, direct output);
// mode 1: candidate pass (chunk blockIdx.z of [prefix tiles | the
//         candidates' own tiles]);
// mode 2: draft pass (chunk blockIdx.z of the prefix + branch-cache tiles).
template <int MODE, bool PREC, bool DEC = false>
__global__ __launch_bounds__((Shape<PREC, DEC>::NT)) void k_attn(AttnArgs a) {
  constexpr int QT = Shape<PREC, DEC>::QT;
  __shared__ u32x4 lds[2 * Shape<PREC, DEC>::STAGE];
  const int G = a.n_heads / a.n_kv, TG = (a.T - a.t0) * G;
  // Prefill: one block index over (query tile, KV head), tiles with more keys
  // first across all heads, so that the longest blocks start in the first
  // round and the short ones fill in behind them.
  const int nqt = MODE == 0 ? (int)gridDim.x / a.n_kv : (int)gridDim.x;
  const int kvh = MODE == 0 ? (int)blockIdx.x % a.n_kv : (int)blockIdx.y;
  const int qt = MODE == 0 ? nqt - 1 - (int)blockIdx.x / a.n_kv : (int)blockIdx.x;
  const int q0 = qt * QT;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int row = q0 + w * 32 + (lane & 31);
  const int rowc = min(row, TG - 1);

  Lane L;
  const int tok = a.t0 + rowc / G;
  const int head = kvh * G + rowc % G;
  L.lo = MODE >= 1 ? a.row_lo[tok] : 0;
  L.tok = MODE == 2 ? a.q_pos[tok] : tok;
  // Precise kernels: raw reference, none yet; fast kernels: log2 units, 0.
  L.m = PREC ? -INFINITY : 0.f;
  L.l = 0.f;
  L.negm = f32x16{};
  L.seen = false;
#pragma unroll
  for (int db = 0; db < HD / 32; ++db) L.o[db] = f32x16{};
  {
    // Queries -> registers: the chunks this lane feeds to the S^T products
    // (no per-tile LDS reads of the query tile).
    const long qoff = ((long)tok * a.n_heads + head) * HD + 8 * (lane >> 5);
#pragma unroll
    for (int kk = 0; kk < HD / 16; ++kk) {
      L.qh[kk] = *reinterpret_cast<const f16x8 *>(a.q + qoff + 16 * kk);
      if constexpr (PREC) L.ql[kk] = *reinterpret_cast<const f16x8 *>(a.q_lo + qoff + 16 * kk);
    }
  }
  const float scale_log2 = 1.4426950408889634f * rsqrtf((float)HD);
  L.thr = 8.f / scale_log2;
  const int tok_first = a.t0 + q0 / G;
  const int tok_last = a.t0 + min(q0 + QT - 1, TG - 1) / G;

  const int chunk = blockIdx.z;
  const long koff = (long)kvh * a.kv_npos * HD, boff = (long)kvh * a.bk_npos * HD;
  if (MODE == 0) {
    // Causal keys 0 .. tok_last; with nchunks > 1 (few blocks on the chip)
    // chunk `chunk` takes an even share of the block's key tiles.
    const int nt = (tok_last + KT) / KT;
    const int kb = (int)((long)nt * chunk / a.nchunks) * KT;
    const int ke = min(tok_last + 1, (int)((long)nt * (chunk + 1) / a.nchunks) * KT);
    Seg sg{a.k + koff, a.vt + koff, PREC ? a.k_lo + koff : nullptr,
           PREC ? a.vt_lo + koff : nullptr, a.kv_npos, a.T, kb, ke, SEG_CAUSAL, tok_first};
    walk_segment<PREC, DEC>(sg, lds, L, scale_log2);
  } else if (MODE == 1) {
    // Candidate pass: chunk `chunk` walks an even share of the block's tiles
    // [prefix tiles | branch tiles], the branch tiles running from the
    // block's first query's segment start to its last query (both
    // non-decreasing in token order). (With the branch tiles all on the last
    // chunk on top of an even share of the prefix, that chunk bounded the
    // launch.)
    const int pre_t = (a.P + KT - 1) / KT;
    const int lo = a.row_lo[tok_first] & ~(KT - 1);
    const int tot = pre_t + (tok_last + 1 - lo + KT - 1) / KT;
    const int c0 = (int)((long)tot * chunk / a.nchunks);
    const int c1 = (int)((long)tot * (chunk + 1) / a.nchunks);
    Seg sp{a.k + koff, a.vt + koff, PREC ? a.k_lo + koff : nullptr,
           PREC ? a.vt_lo + koff : nullptr, a.kv_npos, a.P, min(a.P, c0 * KT),
           min(a.P, min(c1, pre_t) * KT), SEG_ALL, tok_first};
    walk_segment<PREC, DEC>(sp, lds, L, scale_log2);
    if (c1 > pre_t) {
      const int b0 = max(c0, pre_t) - pre_t;
      Seg sb{a.bk + boff, a.bvt + boff, PREC ? a.bk_lo + boff : nullptr,
             PREC ? a.bvt_lo + boff : nullptr, a.bk_npos, a.T, lo + b0 * KT,
             min(tok_last + 1, lo + (c1 - pre_t) * KT), SEG_BRANCH, tok_first};
      walk_segment<PREC, DEC>(sb, lds, L, scale_log2);
    }
  } else {
    // Draft pass (cache positions given): one query tile may hold rows of
    // several branches, whose cache segments lie between the block's first
    // query's segment start and its last query's position, so the branch
    // tiles are many: every chunk walks an even share of [prefix tiles |
    // branch tiles].
    const int pre_t = (a.P + KT - 1) / KT;
    const int lo = a.row_lo[tok_first] & ~(KT - 1);
    const int hi = a.q_pos[tok_last];
    const int tot = pre_t + (hi - lo) / KT + 1;
    const int c0 = (int)((long)tot * chunk / a.nchunks);
    const int c1 = (int)((long)tot * (chunk + 1) / a.nchunks);
    const Seg sp{a.k + koff, a.vt + koff, PREC ? a.k_lo + koff : nullptr,
                 PREC ? a.vt_lo + koff : nullptr, a.kv_npos, a.P, 0, 0, SEG_ALL, tok_first};
    const Seg sb{a.bk + boff, a.bvt + boff, PREC ? a.bk_lo + boff : nullptr,
                 PREC ? a.bvt_lo + boff : nullptr, a.bk_npos, a.bk_valid, 0, 0, SEG_BRANCH,
                 tok_first};
    walk_concat<PREC, DEC>(sp, sb, pre_t, lo, c0, c1, lds, L, scale_log2);
  }

  L.l = sum_halves(L.l);
  if (row >= TG) return;
  const int h = lane >> 5;
  if (a.nchunks == 1) {
    const float inv = 1.f / L.l;
    f16 *op = a.out + ((long)(a.t0 + rowc / G) * a.out_split * a.n_heads + head) * HD;
    f16 *olo = op + (long)a.n_heads * HD;  // remainder half of a split row
#pragma unroll
    for (int db = 0; db < HD / 32; ++db)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        f16x4 v, vl;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float x = L.o[db][g4 * 4 + j] * inv;
          v[j] = static_cast<f16>(x);
          vl[j] = static_cast<f16>(x - static_cast<float>(v[j]));
        }
        *reinterpret_cast<f16x4 *>(op + db * 32 + 8 * g4 + 4 * h) = v;
        if (a.out_split == 2) *reinterpret_cast<f16x4 *>(olo + db * 32 + 8 * g4 + 4 * h) = vl;
      }
  } else {
    const long prow = ((long)chunk * a.n_kv + kvh) * TG + row;
    float *pa = a.part_acc + prow * HD;
#pragma unroll
    for (int db = 0; db < HD / 32; ++db)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        f32x4 v;
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = L.o[db][g4 * 4 + j];
        *reinterpret_cast<f32x4 *>(pa + db * 32 + 8 * g4 + 4 * h) = v;
      }
    // The merge works in the scaled log2 domain.
    if (h == 0) {
      // A chunk with no visible key of this row reports m = -inf (no weight).
      const float m = PREC ? L.m * scale_log2 : L.l == 0.f ? -INFINITY : L.m;
      a.part_ml[prow] = make_float2(m, L.l);
    }
  }
}

// Block of NW waves per (token, query head): combine the chunk partials
// (nchunks <= 64). Lane c of every wave reads chunk c's (max, sum); wave w
// sums the outputs of chunks w, w + NW, ... in order, eight chunks' loads in
// flight at a time; with NW > 1, wave 0 then adds the waves' sums in order.
template <int NW>
__global__ __launch_bounds__(64 * NW) void k_attn_merge(AttnArgs a) {
  __shared__ float po[NW][HD];
  const int t = blockIdx.x, head = blockIdx.y;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int G = a.n_heads / a.n_kv, TG = a.T * G;
  const int kvh = head / G, row = t * G + head % G;
  const long r0 = (long)kvh * TG + row, cstride = (long)a.n_kv * TG;
  // The first eight chunks' outputs are loaded together with the (max, sum)
  // pairs: they do not depend on the weights.
  float v0[8], v1[8];
  const auto load8 = [&](int i0) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const long prow = min(w + NW * (i0 + j), a.nchunks - 1) * cstride + r0;
      v0[j] = a.part_acc[prow * HD + lane];
      v1[j] = a.part_acc[prow * HD + 64 + lane];
    }
  };
  load8(0);
  const float2 ml = lane < a.nchunks ? a.part_ml[lane * cstride + r0]
                                     : make_float2(-INFINITY, 0.f);
  const float M = wave_max(ml.x);
  const float wl = ml.x == -INFINITY ? 0.f : exp2f(ml.x - M);
  const float Lsum = wave_sum(ml.y * wl);
  float o0 = 0.f, o1 = 0.f;
  for (int i0 = 0; w + NW * i0 < a.nchunks; i0 += 8) {
    if (i0 > 0) load8(i0);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int c = w + NW * (i0 + j);
      const float wgt = __shfl(wl, min(c, 63), 64);
      if (c < a.nchunks) {
        o0 += v0[j] * wgt;
        o1 += v1[j] * wgt;
      }
    }
  }
  if constexpr (NW > 1) {
    po[w][lane] = o0;
    po[w][64 + lane] = o1;
    __syncthreads();
    if (w) return;
    o0 = po[0][lane];
    o1 = po[0][64 + lane];
#pragma unroll
    for (int i = 1; i < NW; ++i) {
      o0 += po[i][lane];
      o1 += po[i][64 + lane];
    }
  }
  const float inv = 1.f / Lsum;
  f16 *op = a.out + ((long)t * a.out_split * a.n_heads + head) * HD;
  const float x0 = o0 * inv, x1 = o1 * inv;
  const f16 h0 = static_cast<f16>(x0), h1 = static_cast<f16>(x1);
  op[lane] = h0;
  op[64 + lane] = h1;
  if (a.out_split == 2) {
    f16 *olo = op + (long)a.n_heads * HD;
    olo[lane] = static_cast<f16>(x0 - static_cast<float>(h0));
    olo[64 + lane] = static_cast<f16>(x1 - static_cast<float>(h1));
  }
}

template <int MODE, bool PREC, bool DEC = false>
hipError_t launch_attn(const AttnArgs &a, hipStream_t s) {
  using S = Shape<PREC, DEC>;
  const int G = a.n_heads / a.n_kv;
  const int nqt = ((a.T - a.t0) * G + S::QT - 1) / S::QT;
  const dim3 grid = MODE == 0 ? dim3(nqt * a.n_kv, 1, a.nchunks) : dim3(nqt, a.n_kv, a.nchunks);
  k_attn<MODE, PREC, DEC><<<grid, S::NT, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace

int attn_query_tile() { return QT_FAST; }

int prefill_chunks(int T, int n_heads, int n_kv) {
  // Fewer than ~1.5 rounds of blocks (few KV heads, short prefixes): split
  // each block's causal keys into up to 4 chunks, merged by attn_merge.
  const int blocks = (T * (n_heads / n_kv) + QT_FAST - 1) / QT_FAST * n_kv;
  return std::max(1, std::min(4, (384 + blocks - 1) / blocks));
}

hipError_t attn_prefill(const AttnArgs &a, bool precise, hipStream_t s) {
  if (a.T <= a.t0) return hipSuccess;
  if (a.nchunks < 1 || a.nchunks > 64 || (a.nchunks > 1 && a.t0 != 0))
    return hipErrorInvalidValue;
  if (precise && (!a.q_lo || !a.k_lo || !a.vt_lo)) return hipErrorInvalidValue;
  return precise ? launch_attn<0, true>(a, s) : launch_attn<0, false>(a, s);
}

hipError_t attn_cascade(const AttnArgs &a, bool precise, hipStream_t s) {
  if (a.T == 0 || a.t0 != 0) return a.T == 0 ? hipSuccess : hipErrorInvalidValue;
  if (precise && (!a.q_lo || !a.k_lo || !a.vt_lo || !a.bk_lo || !a.bvt_lo))
    return hipErrorInvalidValue;
  if (a.q_pos) {  // draft pass
    if (a.bk_valid <= 0) return hipErrorInvalidValue;
    if (precise) return launch_attn<2, true>(a, s);
    // Decode steps: all stacked query rows of a KV head in one wave.
    if ((a.T - a.t0) * (a.n_heads / a.n_kv) <= Shape<false, true>::QT)
      return launch_attn<2, false, true>(a, s);
    return launch_attn<2, false>(a, s);
  }
  return precise ? launch_attn<1, true>(a, s) : launch_attn<1, false>(a, s);
}

hipError_t attn_merge(const AttnArgs &a, hipStream_t s) {
  if (a.T == 0 || a.nchunks == 1) return hipSuccess;
  if (a.nchunks > 64) return hipErrorInvalidValue;
  // Many chunks (decode steps: few rows, single-tile chunks): four waves.
  if (a.nchunks > 16)
    k_attn_merge<4><<<dim3(a.T, a.n_heads), 256, 0, s>>>(a);
  else
    k_attn_merge<1><<<dim3(a.T, a.n_heads), 64, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace vsr
