// Internal declarations shared by the HIP kernels and the host orchestrator of
// the verifier scoring pass. Not part of the C ABI (include/vsr.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace vsr {

typedef __bf16 bf16;
typedef _Float16 f16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return static_cast<float>(x); }
__device__ __forceinline__ float to_f32(f16 x) { return static_cast<float>(x); }
template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return static_cast<bf16>(x); }
template <> __device__ __forceinline__ f16 from_f32<f16>(float x) { return static_cast<f16>(x); }

// Arithmetic types of the two paths. A VSR_BF16 context keeps its weights in
// bf16 and its activations (GEMM / attention operands) in fp16: every bf16
// weight converts exactly to fp16 (8 significant bits fit in 11), and the
// fp16 operands carry 3 more mantissa bits than bf16 at the same MFMA rate.
// A VSR_F32 context is fp32 throughout.

// Largest number of candidates one score call may carry.
constexpr int kMaxCands = 256;

// Packed candidate rows: candidate m owns rows [cu[m], cu[m+1]).
// Sum / maximum over the 64 lanes of a wave (butterfly, fixed order), the
// result in every lane.
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

struct Branches {
  int M;
  int cmax;
  int cu[kMaxCands + 1];
};

// ---------------------------------------------------------------- launchers
// Every launcher enqueues on `s` and returns the hipError_t of the launch.

// Rotary table: cs[p][i] = (cos, sin)(p * base^(-2i/hd)), i < hd/2, p < npos.
hipError_t launch_rope_table(float2 *cs, int npos, int hd, float base, hipStream_t s);

// Status word of a checked call (vsr_set_checks): kernels that read an id
// outside [0, vocab) (and use id 0 instead) set kFlagBadId; the finiteness
// check of a call's outputs sets kFlagNonFinite.
constexpr int32_t kFlagBadId = 1;
constexpr int32_t kFlagNonFinite = 2;
hipError_t launch_flags_clear(int32_t *flags, hipStream_t s);
// Sets kFlagNonFinite in *flags if any of x[0 .. n) is NaN or infinite.
hipError_t launch_check_finite(const float *x, long n, int32_t *flags, hipStream_t s);

// Row tables of one score call: for packed row t of candidate m at offset j,
// row_lo[t] = cu[m] (first row of its candidate), row_pos[t] = P + j,
// lm_tgt[t] = cand_ids[m][j] (clamped into [0, vocab); a clamped id sets
// kFlagBadId in *flags).
hipError_t launch_row_tables(const Branches &br, int P, const int32_t *cand_ids, int vocab,
                             int32_t *flags, int32_t *row_lo, int32_t *row_pos,
                             int32_t *lm_tgt, hipStream_t s);

// x[p] = visual[p] for p < n_visual, else embed[ids[p - n_visual]] (fp32 out;
// an id outside [0, vocab) reads row 0 and sets kFlagBadId in *flags).
template <typename T>
hipError_t launch_embed_prefix(const T *visual, int n_visual, const int32_t *ids, int n_text,
                               const T *embed, int vocab, int d, float *x, int32_t *flags,
                               hipStream_t s);
// x[t] = embed[ids[t]] for t < rows (ids already in [0, vocab)).
template <typename T>
hipError_t launch_embed_rows(const int32_t *ids, int rows, const T *embed, int d, float *x,
                             hipStream_t s);

// y[r] = TA(x[r] / sqrt(mean(x[r]^2) + eps) * g) for rows r < rows; with
// split = 2 the rows of y are [hi | lo] (2d wide).
template <typename TW, typename TA>
hipError_t launch_rmsnorm(const float *x, const TW *g, int rows, int d, float eps, TA *y,
                          int split, hipStream_t s);
// LM-head inputs of a score call: y[t] = norm(h_last) if t is the first row
// of its candidate, else norm(x[t - 1]).
template <typename TW, typename TA>
hipError_t launch_lm_inputs(const float *x, const float *h_last, const int32_t *row_lo,
                            const TW *g, int T_rows, int d, float eps, TA *y, hipStream_t s);

// Draft calls (decode cache with a fixed stride S per branch): prompt row
// tables, per-step tables, the last prompt row's norm per branch and the
// greedy pick from the LM-head argmax partials.
hipError_t launch_draft_rows(const Branches &br, int P, int S, const int32_t *ids, int vocab,
                             int32_t *flags, int32_t *row_lo, int32_t *row_pos,
                             int32_t *cache_row, int32_t *lm_tgt, hipStream_t s);
hipError_t launch_draft_step(const Branches &br, int P, int S, int step, int32_t *row_lo,
                             int32_t *row_pos, int32_t *cache_row, hipStream_t s);
template <typename TW, typename TA>
hipError_t launch_branch_last_norm(const float *x, const Branches &br, const TW *g, int d,
                                   float eps, TA *y, hipStream_t s);
hipError_t launch_argmax_merge(const float2 *part, int nchunks, int M, int n_new, int step,
                               int32_t *tokens, int32_t *next_ids, hipStream_t s);

// LM-head inputs of a reliability call (2M rows): y[b] = norm(x[last row of
// branch b % M]); lm_tgt[b] = yes_id for b < M, no_id for b >= M.
template <typename TW, typename TA>
hipError_t launch_last_inputs(const float *x, const Branches &br, const TW *g, int d, float eps,
                              int yes_id, int no_id, TA *y, int32_t *lm_tgt, hipStream_t s);
// Reliability from the LM-head partials of those 2M rows (Eq. 11-13):
// lp_yes_no[m] = (tgt[m] - lse[m], tgt[M + m] - lse[M + m]),
// rel[m] = 1 / (1 + exp(lp_no - lp_yes)), keep[m] = rel[m] >= max rel - delta.
hipError_t launch_reliability_finish(int M, const float2 *part, int nchunks,
                                     const float *tgt_logit, float delta, float *lp_yes_no,
                                     float *rel, int32_t *keep, hipStream_t s);
// Entity alignment and final choice (Eq. 14-15, Algorithm 1, Table 3).
hipError_t launch_align_select(const float *ent, const float *frames, int M, int NF, int D,
                               const float *rel, float delta, int strategy, float *align,
                               int32_t *choice, hipStream_t s);

// Retrieval stage (Eq. 1-3): histograms + keyframes, then per-keyframe top-k
// and the merged top-K (kernels_retrieval.hip).
hipError_t launch_keyframes(const uint8_t *frames, int NF, int H, int W, float theta,
                            int32_t *hist, int32_t *inter, int32_t *key_idx, int32_t *n_keys,
                            hipStream_t s);
size_t retrieve_workspace_bytes(int NF, int ND, int k);
hipError_t launch_retrieve(const float *frame_emb, const int32_t *key_idx, const int32_t *n_keys,
                           int NF, const float *docs, int ND, int D, int k, int K, void *ws,
                           int32_t *top_idx, float *top_sim, int32_t *sel_idx, float *sel_sim,
                           int32_t *n_sel, hipStream_t s);

// Retrieval with library-owned scratch (vsr_retrieve_static): the size of
// the file-scope device array, and its device address on the current device
// (looked up once per device; the largest device index it serves is
// kMaxDevices - 1).
constexpr size_t kRetrieveStaticBytes = size_t(32) << 20;
constexpr int kMaxDevices = 64;
hipError_t retrieve_static_scratch(void **ptr);

// Per-row merge of the LM-head partials: lse over the vocabulary chunks,
// lp = target logit - lse, scattered to logprobs[m][j] (zeros elsewhere).
hipError_t launch_lse_gather(const Branches &br, const float2 *part, int nchunks,
                             const float *tgt_logit, float *logprobs, hipStream_t s);
// scores[m] = sum_j logprobs[m][j] (fixed order), argmax = lowest best m.
hipError_t launch_reduce_select(const Branches &br, const float *logprobs, float *scores,
                                int32_t *argmax, hipStream_t s);

// ----- layouts of the caches -----------------------------------------------
// K cache  : [n_kv][npos][hd]  (rotated keys, position-major)
// Vt cache : [n_kv][hd][npos]  (values, transposed: position-contiguous). On
//            the MFMA path position p is stored at (p & ~12) | ((p & 4) << 1)
//            | ((p & 8) >> 1) (quarters 1 and 2 of each 16-group swapped),
//            the key order of the attention kernel's PV operand.

// Destinations of the QKV projection epilogue.
template <typename T>
struct QKVOut {
  T *q;            // [rows][n_heads][hd] rotated queries
  T *k;            // K cache base (this layer)
  T *vt;           // Vt cache base (this layer)
  int kv_npos;     // position stride of the caches (their capacity)
  const int32_t *row_pos;  // rotary position of each row (NULL: position = row)
  const float2 *rope;      // rotary table [npos][hd/2]
  // Precise layers (MFMA path): the fp16 remainders x - fp16(x) of q, k, v in
  // planes laid out like q, k, vt (NULL: not written).
  T *q_lo = nullptr, *k_lo = nullptr, *vt_lo = nullptr;
  // Cache position of each row's key / value (NULL: the row index).
  const int32_t *cache_row = nullptr;
  // Prefix and candidate rows in one projection: rows >= split go to a second
  // pair of caches (k2 / vt2 and their remainder planes, capacity kv_npos2) at
  // cache position row - split, rotated at position row_pos2[row - split];
  // rows below split as above. split = INT32_MAX: one destination.
  int split = 0x7fffffff;
  T *k2 = nullptr, *vt2 = nullptr, *k2_lo = nullptr, *vt2_lo = nullptr;
  int kv_npos2 = 0;
  const int32_t *row_pos2 = nullptr;
  // Queries are stored multiplied by q_scale (after the rotary): the fast
  // attention kernels take them pre-scaled by log2(e) / sqrt(hd).
  float q_scale = 1.f;
};

// Rotary position of row `row`.
__device__ __forceinline__ int qkv_row_pos(const QKVOut<f16> &o, int row) {
  // One load through a selected pointer (two loads into one register in
  // different branches would make the second wait for the first).
  const int32_t *p = row >= o.split ? o.row_pos2 + (row - o.split)
                                    : o.row_pos ? o.row_pos + row : nullptr;
  return p ? *p : row;
}

// qkv_store without the rotary: x1, x2 are the pair as stored (queries and
// keys already rotated).
__device__ __forceinline__ void qkv_store_rotated(const QKVOut<f16> &o, int n_heads, int n_kv,
                                                  int slot, int row, int d, float x1, float x2) {
  const bool second = row >= o.split;  // a candidate row of a fused pass
  const int row2 = row - o.split;
  const f16 h1 = static_cast<f16>(x1), h2 = static_cast<f16>(x2);
  const f16 l1 = static_cast<f16>(x1 - static_cast<float>(h1));
  const f16 l2 = static_cast<f16>(x2 - static_cast<float>(h2));
  if (slot < n_heads) {
    const long off = ((long)row * n_heads + slot) * 128;
    o.q[off + d] = h1;
    o.q[off + d + 64] = h2;
    if (o.q_lo) {
      o.q_lo[off + d] = l1;
      o.q_lo[off + d + 64] = l2;
    }
  } else {
    const int crow = second ? row2 : o.cache_row ? o.cache_row[row] : row;
    const int npos = second ? o.kv_npos2 : o.kv_npos;
    if (slot < n_heads + n_kv) {
      f16 *k = second ? o.k2 : o.k, *k_lo = second ? o.k2_lo : o.k_lo;
      const long off = ((long)(slot - n_heads) * npos + crow) * 128;
      k[off + d] = h1;
      k[off + d + 64] = h2;
      if (k_lo) {
        k_lo[off + d] = l1;
        k_lo[off + d + 64] = l2;
      }
    } else {
      // Values go to the Vt cache at the attention kernel's interleaved
      // position: within each aligned group of 16, quarters 1 and 2 swap.
      f16 *vt = second ? o.vt2 : o.vt, *vt_lo = second ? o.vt2_lo : o.vt_lo;
      const long base = (long)(slot - n_heads - n_kv) * 128 * npos;
      const int pp = (crow & ~12) | ((crow & 4) << 1) | ((crow & 8) >> 1);
      const long o1 = base + (long)d * npos + pp, o2 = base + (long)(d + 64) * npos + pp;
      vt[o1] = h1;
      vt[o2] = h2;
      if (vt_lo) {
        vt_lo[o1] = l1;
        vt_lo[o2] = l2;
      }
    }
  }
}

// The rotate-half pair of query / key slots turned by the rotary-table entry
// cs of (row's position, d).
__device__ __forceinline__ void rope_pair(float &x1, float &x2, float2 cs) {
  const float y1 = x1 * cs.x - x2 * cs.y, y2 = x2 * cs.x + x1 * cs.y;
  x1 = y1;
  x2 = y2;
}

// Rotary of a query / key pair (entry cs), then the query scale.
__device__ __forceinline__ void qk_turn(const QKVOut<f16> &o, int n_heads, int n_kv, int slot,
                                        float &x1, float &x2, float2 cs) {
  if (slot < n_heads + n_kv) rope_pair(x1, x2, cs);
  if (slot < n_heads) {
    x1 *= o.q_scale;
    x2 *= o.q_scale;
  }
}

// qkv_store with the rotary-table entry given as cs (unused for value slots),
// so that a caller can load the entries of many rows before it stores any of
// them.
__device__ __forceinline__ void qkv_store_cs(const QKVOut<f16> &o, int n_heads, int n_kv,
                                             int slot, int row, int d, float x1, float x2,
                                             float2 cs) {
  qk_turn(o, n_heads, n_kv, slot, x1, x2, cs);
  qkv_store_rotated(o, n_heads, n_kv, slot, row, d, x1, x2);
}

// Stores one rotate-half pair (dims d and d + 64 of head slot `slot` of the
// stacked q | k | v projection) of row `row`: rotary on q and k at the row's
// position, then q to its rows, k to the key cache and v to the Vt cache (at
// the attention kernel's interleaved position), each with its fp16 remainder
// where the remainder planes are given. head_dim 128.
__device__ __forceinline__ void qkv_store(const QKVOut<f16> &o, int n_heads, int n_kv, int slot,
                                          int row, int d, float x1, float x2) {
  const float2 cs = slot < n_heads + n_kv ? o.rope[(long)qkv_row_pos(o, row) * 64 + d]
                                          : make_float2(1.f, 0.f);
  qkv_store_cs(o, n_heads, n_kv, slot, row, d, x1, x2, cs);
}


// ------------------------------------------------------------ MFMA path
// C = A[rows][K] . W[N][K]^T with fused epilogues; A fp16 activations, W
// 16-bit weights: bf16 (w_f16 = false: converted to fp16 on their way into
// LDS) or fp16 (w_f16 = true: loaded straight into LDS); fp32 accumulation.
// Shapes with few output tiles split K; `part` is fp32 scratch of
// gemm_split_floats(rows, N, K) floats (N = B rows) for the partials.
// asplit = 2: each A row is [hi | lo] (2K wide), an fp16 value and its fp16
// remainder, multiplied by the same W (about 22-bit operands); outputs that
// feed a split GEMM are written the same way.
size_t gemm_split_floats(int rows, int N, int K);
hipError_t gemm_qkv_rope(const f16 *A, const void *W, bool w_f16, int rows, int K, int asplit,
                         int n_heads, int n_kv, const QKVOut<f16> &out, float *part,
                         hipStream_t s);
// x[rows][N] += A . W^T (residual stream, fp32).
hipError_t gemm_residual(const f16 *A, const void *W, bool w_f16, int rows, int N, int K,
                         int asplit, float *x, float *part, hipStream_t s);
// h[rows][F] = silu(A . Wg^T) * (A . Wu^T), W = [Wg; Wu] ([2F][K]); h rows are
// [hi | lo] (2F wide) when asplit == 2.
hipError_t gemm_swiglu(const f16 *A, const void *W, bool w_f16, int rows, int F, int K,
                       int asplit, f16 *h, float *part, hipStream_t s);
// LM head: per (vocab chunk c, row t): part[c][t] = (max, sum exp(l - max)) over
// the chunk's logits l = W[v] . A[t]; tgt_logit[t] = logit of lm_tgt[t].
int lmhead_chunks(int vocab);
// Greedy LM head: part[c][t] = (largest logit of vocab chunk c for row t,
// its vocabulary index as int bits; the lowest index on ties).
hipError_t gemm_lmargmax(const f16 *A, const void *W, bool w_f16, int rows, int vocab, int K,
                         float2 *part, hipStream_t s);
// Few-row products (rows <= kSkinnyMaxRows; N a multiple of 64, K of 32): the
// same operands and epilogues as the GEMMs above, computed as a weight stream
// (K split over up to kSkinnyMaxSplit slices, fp32 partials of
// skinny_part_floats(rows, N, K) floats in `part`, summed in slice order).
// skinny_residual also writes the RMSNorm (gain g, NULL: none) of the updated
// rows to y, [hi | lo] when ysplit == 2.
constexpr int kSkinnyMaxRows = 32;
constexpr int kSkinnyMaxSplit = 16;
int skinny_split(int N, int K);
size_t skinny_part_floats(int rows, int N, int K);
hipError_t skinny_residual(const f16 *A, int rows, int asplit, const void *W, bool w_f16, int N,
                           int K, float *x, const bf16 *g, float eps, f16 *y, int ysplit,
                           float *part, hipStream_t s);
hipError_t skinny_swiglu(const f16 *A, int rows, int asplit, const void *W, bool w_f16, int F,
                         int K, f16 *h, float *part, hipStream_t s);
hipError_t skinny_qkv_rope(const f16 *A, int rows, int asplit, const void *W, bool w_f16, int K,
                           int n_heads, int n_kv, const QKVOut<f16> &out, float *part,
                           hipStream_t s);
// Greedy LM head of few rows: part[c][t] = (largest logit among vocabulary
// entries 64c .. 64c+63 for row t, its lowest index as int bits), c <
// skinny_lm_chunks(vocab) (0: vocab not a multiple of 64, not supported).
int skinny_lm_chunks(int vocab);
hipError_t skinny_lmargmax(const f16 *A, int rows, const void *W, bool w_f16, int vocab, int K,
                           float2 *part, hipStream_t s);
// dst[i] = fp16 of the bf16 src[i], the GEMMs' in-register conversion.
hipError_t convert_bf16_to_f16(const uint16_t *src, uint16_t *dst, size_t n, hipStream_t s);
hipError_t gemm_lmhead(const f16 *A, const void *W, bool w_f16, int rows, int vocab, int K,
                       const int32_t *lm_tgt, float2 *part, float *tgt_logit, hipStream_t s);

// Attention of query rows against one key source. Query row r of KV head h is
// (token r / G, head h*G + r % G). Keys of a token t are the positions
// [lo(t), hi(t)] of the key source:
//   mode 0 (prefill)  : lo = 0, hi = t (causal);
//   mode 1 (cascade)  : prefix keys [0, P) all visible, then the branch keys
//                       [row_lo[t], t] of the token's own candidate.
struct AttnArgs {
  const f16 *q;         // [T][n_heads][hd]
  const f16 *k;         // prefix / own K cache of this layer
  const f16 *vt;        // prefix / own Vt cache
  int kv_npos;          // position stride of k / vt
  const f16 *bk;        // mode 1: branch K  [n_kv][bk_npos][hd]
  const f16 *bvt;       // mode 1: branch Vt [n_kv][hd][bk_npos]
  int bk_npos;
  const int32_t *row_lo;  // mode 1
  int T;                // tokens (queries are tokens t0 .. T-1; keys up to T-1)
  int t0;               // first query token
  int P;                // mode 1: prefix length
  int n_heads, n_kv;
  int nchunks;          // key split of each block (partials when > 1; the
                        // prefill only with t0 = 0)
  f16 *out;             // [T][out_split][n_heads][hd] when nchunks == 1 (or merged)
  int out_split;        // 2: [hi | lo] rows for a split output projection
  float *part_acc;      // [nchunks][n_kv][T*G][hd]
  float2 *part_ml;      // [nchunks][n_kv][T*G]
  // Precise layers: remainder planes of q, k, vt (and bk, bvt), same layouts.
  const f16 *q_lo, *k_lo, *vt_lo, *bk_lo, *bvt_lo;
  // Mode 1: branch-cache position of each query token (its key limit; NULL:
  // the token index, keys packed by token) and the number of branch-cache
  // positions that hold data or zeros (0: T). q_pos and row_lo must be
  // non-decreasing in token order.
  const int32_t *q_pos;
  int bk_valid;
};
int attn_query_tile();  // stacked query rows per attention block
// precise = true: q/k/v and the probabilities are carried as fp16 value +
// remainder (three MFMAs per product); needs the *_lo planes of AttnArgs.
// Prefill: with a.nchunks > 1 (only for t0 = 0) the keys of each block are
// split into chunks that write partials, and attn_merge(a) writes the output;
// prefill_chunks gives the split for T query tokens.
int prefill_chunks(int T, int n_heads, int n_kv);
hipError_t attn_prefill(const AttnArgs &a, bool precise, hipStream_t s);
hipError_t attn_cascade(const AttnArgs &a, bool precise, hipStream_t s);
hipError_t attn_merge(const AttnArgs &a, hipStream_t s);

// ------------------------------------------------------ simple (fp32) path
// Plain kernels, one output element per thread; the path of VSR_F32 contexts.
template <typename T>
hipError_t simple_qkv_rope(const T *A, const T *W, int rows, int K, int n_heads, int n_kv,
                           int hd, const QKVOut<T> &out, hipStream_t s);
template <typename T>
hipError_t simple_residual(const T *A, const T *W, int rows, int N, int K, float *x,
                           hipStream_t s);
template <typename T>
hipError_t simple_swiglu(const T *A, const T *W, int rows, int F, int K, T *h, hipStream_t s);
template <typename T>
hipError_t simple_lmhead(const T *A, const T *W, int rows, int vocab, int K,
                         const int32_t *lm_tgt, float2 *part, float *tgt_logit,
                         hipStream_t s);
// Attention with the same key rules as AttnArgs (mode 0: causal over the
// prefix cache; mode 1: prefix + own candidate), one block per (token, head).
struct SimpleAttnArgs {
  const void *q, *k, *vt, *bk, *bvt;
  int kv_npos, bk_npos;
  const int32_t *row_lo;
  const int32_t *q_pos;  // mode 1: branch-cache position of each query (NULL: token)
  int T, t0, P, n_heads, n_kv, hd;  // query tokens t0 .. T-1
  int mode;
  void *out;
};
template <typename T>
hipError_t simple_attn(const SimpleAttnArgs &a, hipStream_t s);
// Greedy LM head of the plain path: part[t] = (largest logit, index bits).
template <typename T>
hipError_t simple_lmargmax(const T *A, const T *W, int rows, int vocab, int K, float2 *part,
                           hipStream_t s);

}  // namespace vsr
