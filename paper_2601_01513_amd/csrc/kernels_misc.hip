// Memory-bound helper kernels of the verifier scoring pass: rotary table,
// per-row tables, embedding gathers, RMSNorm, LM-head inputs, the log-sum-exp
// merge with the target gather, and the per-candidate sum and argmax
// (Eq. 6-7). All of them read and write rows with consecutive lanes on
// consecutive elements; reductions run in a fixed order (no atomics).
#include <algorithm>

#include "common.h"

namespace vsr {

// Sum over a 256-thread block, same value returned to every thread.
__device__ __forceinline__ float block_sum256(float v, float *red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}

// ------------------------------------------------------------- rotary table
__global__ void k_rope_table(float2 *cs, int npos, int hd, double base) {
  const int half = hd / 2;
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)npos * half) return;
  const int p = (int)(idx / half), i = (int)(idx % half);
  const double inv = pow(base, -2.0 * i / hd);
  const double ang = (double)p * inv;
  cs[idx] = make_float2((float)cos(ang), (float)sin(ang));
}

hipError_t launch_rope_table(float2 *cs, int npos, int hd, float base, hipStream_t s) {
  const long n = (long)npos * (hd / 2);
  k_rope_table<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(cs, npos, hd, (double)base);
  return hipGetLastError();
}

// --------------------------------------------------------------- row tables
__global__ void k_row_tables(Branches br, int P, const int32_t *cand_ids, int vocab,
                             int32_t *flags, int32_t *row_lo, int32_t *row_pos,
                             int32_t *lm_tgt) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= br.cu[br.M]) return;
  int m = 0;
  while (br.cu[m + 1] <= t) ++m;
  const int j = t - br.cu[m];
  int id = cand_ids[(long)m * br.cmax + j];
  if (id < 0 || id >= vocab) {
    atomicOr(flags, kFlagBadId);
    id = 0;
  }
  row_lo[t] = br.cu[m];
  row_pos[t] = P + j;
  lm_tgt[t] = id;
}

hipError_t launch_row_tables(const Branches &br, int P, const int32_t *cand_ids, int vocab,
                             int32_t *flags, int32_t *row_lo, int32_t *row_pos,
                             int32_t *lm_tgt, hipStream_t s) {
  const int T = br.cu[br.M];
  if (T == 0) return hipSuccess;
  k_row_tables<<<(T + 255) / 256, 256, 0, s>>>(br, P, cand_ids, vocab, flags, row_lo, row_pos,
                                               lm_tgt);
  return hipGetLastError();
}

// Row tables of a draft call. Prompt row t of branch m at offset j sits at
// decode-cache position m S + j (a fixed stride S per branch, room for the
// prompt and the new tokens): row_lo = m S, row_pos = P + j (rotary),
// cache_row = m S + j, lm_tgt = the prompt id (clamped).
__global__ void k_draft_rows(Branches br, int P, int S, const int32_t *ids, int vocab,
                             int32_t *flags, int32_t *row_lo, int32_t *row_pos,
                             int32_t *cache_row, int32_t *lm_tgt) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= br.cu[br.M]) return;
  int m = 0;
  while (br.cu[m + 1] <= t) ++m;
  const int j = t - br.cu[m];
  int id = ids[(long)m * br.cmax + j];
  if (id < 0 || id >= vocab) {
    atomicOr(flags, kFlagBadId);
    id = 0;
  }
  row_lo[t] = m * S;
  row_pos[t] = P + j;
  cache_row[t] = m * S + j;
  lm_tgt[t] = id;
}

hipError_t launch_draft_rows(const Branches &br, int P, int S, const int32_t *ids, int vocab,
                             int32_t *flags, int32_t *row_lo, int32_t *row_pos,
                             int32_t *cache_row, int32_t *lm_tgt, hipStream_t s) {
  const int T = br.cu[br.M];
  k_draft_rows<<<(T + 255) / 256, 256, 0, s>>>(br, P, S, ids, vocab, flags, row_lo, row_pos,
                                               cache_row, lm_tgt);
  return hipGetLastError();
}

// Decode step s >= 1: row m is new token s - 1 of branch m, at branch offset
// n_m + s - 1.
__global__ void k_draft_step(Branches br, int P, int S, int step, int32_t *row_lo,
                             int32_t *row_pos, int32_t *cache_row) {
  const int m = blockIdx.x * blockDim.x + threadIdx.x;
  if (m >= br.M) return;
  const int j = br.cu[m + 1] - br.cu[m] + step - 1;
  row_lo[m] = m * S;
  row_pos[m] = P + j;
  cache_row[m] = m * S + j;
}

hipError_t launch_draft_step(const Branches &br, int P, int S, int step, int32_t *row_lo,
                             int32_t *row_pos, int32_t *cache_row, hipStream_t s) {
  k_draft_step<<<(br.M + 63) / 64, 64, 0, s>>>(br, P, S, step, row_lo, row_pos, cache_row);
  return hipGetLastError();
}

// Greedy pick per row from the LM-head partials (chunks in vocabulary order,
// each holding its lowest best index): tokens[m][step] and the next inputs.
// Block per row: threads stride over the chunks, then waves and blocks keep
// the largest value and, among equal values, the lowest index.
__device__ __forceinline__ void keep_best(float &v, int &i, float v2, int i2) {
  if (i2 >= 0 && (i < 0 || v2 > v || (v2 == v && i2 < i))) {
    v = v2;
    i = i2;
  }
}

__global__ __launch_bounds__(1024) void k_argmax_merge(const float2 *part, int nchunks, int M,
                                                       int n_new, int step, int32_t *tokens,
                                                       int32_t *next_ids) {
  __shared__ float sv[16];
  __shared__ int si[16];
  const int m = blockIdx.x, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  float best = -INFINITY;
  int bi = -1;
  for (int c = threadIdx.x; c < nchunks; c += 1024) {
    const float2 p = part[(long)c * M + m];
    keep_best(best, bi, p.x, __float_as_int(p.y));
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1)
    keep_best(best, bi, __shfl_xor(best, o, 64), __shfl_xor(bi, o, 64));
  if (lane == 0) {
    sv[w] = best;
    si[w] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int i = 1; i < 16; ++i) keep_best(best, bi, sv[i], si[i]);
    tokens[(long)m * n_new + step] = bi;
    next_ids[m] = bi;
  }
}

hipError_t launch_argmax_merge(const float2 *part, int nchunks, int M, int n_new, int step,
                               int32_t *tokens, int32_t *next_ids, hipStream_t s) {
  k_argmax_merge<<<M, 1024, 0, s>>>(part, nchunks, M, n_new, step, tokens, next_ids);
  return hipGetLastError();
}

// ---------------------------------------------------------- call validator
// The status word of a checked call: cleared at its start, bits set by the
// kernels that meet a bad id or a non-finite result, read once at its end.
__global__ void k_flags_clear(int32_t *flags) {
  if (threadIdx.x == 0) flags[0] = 0;
}

hipError_t launch_flags_clear(int32_t *flags, hipStream_t s) {
  k_flags_clear<<<1, 64, 0, s>>>(flags);
  return hipGetLastError();
}

// Sets kFlagNonFinite if any of x[0 .. n) is NaN or infinite.
__global__ __launch_bounds__(256) void k_check_finite(const float *x, long n, int32_t *flags) {
  bool bad = false;
  for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < n; i += (long)gridDim.x * 256)
    bad |= !isfinite(x[i]);
  if (__any(bad) && (threadIdx.x & 63) == 0) atomicOr(flags, kFlagNonFinite);
}

hipError_t launch_check_finite(const float *x, long n, int32_t *flags, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const long blocks = std::min<long>((n + 255) / 256, 1024);
  k_check_finite<<<(unsigned)blocks, 256, 0, s>>>(x, n, flags);
  return hipGetLastError();
}

// ---------------------------------------------------------------- embedding
template <typename T>
__global__ void k_embed_prefix(const T *visual, int n_visual, const int32_t *ids,
                               const T *embed, int vocab, int d, float *x, int32_t *flags) {
  const int p = blockIdx.x;
  const T *src;
  if (p < n_visual) {
    src = visual + (long)p * d;
  } else {
    int id = ids[p - n_visual];
    if (id < 0 || id >= vocab) {
      if (threadIdx.x == 0) atomicOr(flags, kFlagBadId);
      id = 0;
    }
    src = embed + (long)id * d;
  }
  float *dst = x + (long)p * d;
  for (int c = threadIdx.x; c < d; c += blockDim.x) dst[c] = to_f32(src[c]);
}

template <typename T>
hipError_t launch_embed_prefix(const T *visual, int n_visual, const int32_t *ids, int n_text,
                               const T *embed, int vocab, int d, float *x, int32_t *flags,
                               hipStream_t s) {
  const int P = n_visual + n_text;
  k_embed_prefix<T><<<P, 256, 0, s>>>(visual, n_visual, ids, embed, vocab, d, x, flags);
  return hipGetLastError();
}

template <typename T>
__global__ void k_embed_rows(const int32_t *ids, const T *embed, int d, float *x) {
  const int t = blockIdx.x;
  const T *src = embed + (long)ids[t] * d;
  float *dst = x + (long)t * d;
  for (int c = threadIdx.x; c < d; c += blockDim.x) dst[c] = to_f32(src[c]);
}

// Candidate rows use the row table's clamped ids (lm_tgt holds cand_ids[m][j]).
template <typename T>
hipError_t launch_embed_rows(const int32_t *ids, int rows, const T *embed, int d, float *x,
                             hipStream_t s) {
  if (rows == 0) return hipSuccess;
  k_embed_rows<T><<<rows, 256, 0, s>>>(ids, embed, d, x);
  return hipGetLastError();
}

// ------------------------------------------------------------------ RMSNorm
// One row by a 256-thread block: y = x / sqrt(mean(x^2) + eps) * g (+ the
// remainder half when split == 2). Rows of d % 4 == 0, d <= 8192 are read once
// as float4 and kept in registers; others take the scalar two-pass path.
template <typename TW, typename TA>
__device__ __forceinline__ void norm_row(const float *src, const TW *g, int d, float eps,
                                         TA *dst, float *red, int split = 1) {
  constexpr int NV = 8;  // float4 per thread: d <= 256 * 4 * NV
  if (d % 4 == 0 && d <= 256 * 4 * NV) {
    const int n4 = d / 4;
    float4 v[NV];
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int c4 = threadIdx.x + 256 * i;
      v[i] = c4 < n4 ? reinterpret_cast<const float4 *>(src)[c4] : make_float4(0.f, 0.f, 0.f, 0.f);
      ss += v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w;
    }
    ss = block_sum256(ss, red);
    const float r = rsqrtf(ss / (float)d + eps);
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int c4 = threadIdx.x + 256 * i;
      if (c4 >= n4) break;
      const float x[4] = {v[i].x, v[i].y, v[i].z, v[i].w};
      TA hi[4], lo[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float y = x[e] * r * to_f32(g[4 * c4 + e]);
        hi[e] = from_f32<TA>(y);
        lo[e] = from_f32<TA>(y - to_f32(hi[e]));
      }
      // Four outputs per store.
      struct alignas(4 * sizeof(TA)) Q4 { TA v[4]; };
      *reinterpret_cast<Q4 *>(dst + 4 * c4) = Q4{{hi[0], hi[1], hi[2], hi[3]}};
      if (split == 2) *reinterpret_cast<Q4 *>(dst + d + 4 * c4) = Q4{{lo[0], lo[1], lo[2], lo[3]}};
    }
    return;
  }
  float ss = 0.f;
  for (int c = threadIdx.x; c < d; c += 256) {
    const float v = src[c];
    ss += v * v;
  }
  ss = block_sum256(ss, red);
  const float r = rsqrtf(ss / (float)d + eps);
  for (int c = threadIdx.x; c < d; c += 256) {
    const float v = src[c] * r * to_f32(g[c]);
    const TA hi = from_f32<TA>(v);
    dst[c] = hi;
    if (split == 2) dst[d + c] = from_f32<TA>(v - to_f32(hi));
  }
}

template <typename TW, typename TA>
__global__ __launch_bounds__(256) void k_rmsnorm(const float *x, const TW *g, int d, float eps,
                                                 TA *y, int split) {
  __shared__ float red[4];
  const long r = blockIdx.x;
  norm_row(x + r * d, g, d, eps, y + r * d * split, red, split);
}

template <typename TW, typename TA>
hipError_t launch_rmsnorm(const float *x, const TW *g, int rows, int d, float eps, TA *y,
                          int split, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  k_rmsnorm<TW, TA><<<rows, 256, 0, s>>>(x, g, d, eps, y, split);
  return hipGetLastError();
}

template <typename TW, typename TA>
__global__ __launch_bounds__(256) void k_lm_inputs(const float *x, const float *h_last,
                                                   const int32_t *row_lo, const TW *g, int d,
                                                   float eps, TA *y) {
  __shared__ float red[4];
  const int t = blockIdx.x;
  const float *src = (row_lo[t] == t) ? h_last : x + (long)(t - 1) * d;
  norm_row(src, g, d, eps, y + (long)t * d, red);
}

template <typename TW, typename TA>
hipError_t launch_lm_inputs(const float *x, const float *h_last, const int32_t *row_lo,
                            const TW *g, int T_rows, int d, float eps, TA *y, hipStream_t s) {
  if (T_rows == 0) return hipSuccess;
  k_lm_inputs<TW, TA><<<T_rows, 256, 0, s>>>(x, h_last, row_lo, g, d, eps, y);
  return hipGetLastError();
}

// Draft prompt stage: block m normalises the last prompt row of branch m.
template <typename TW, typename TA>
__global__ __launch_bounds__(256) void k_branch_last_norm(const float *x, Branches br,
                                                          const TW *g, int d, float eps,
                                                          TA *y) {
  __shared__ float red[4];
  const int m = blockIdx.x;
  norm_row(x + (long)(br.cu[m + 1] - 1) * d, g, d, eps, y + (long)m * d, red);
}

template <typename TW, typename TA>
hipError_t launch_branch_last_norm(const float *x, const Branches &br, const TW *g, int d,
                                   float eps, TA *y, hipStream_t s) {
  k_branch_last_norm<TW, TA><<<br.M, 256, 0, s>>>(x, br, g, d, eps, y);
  return hipGetLastError();
}

// Reliability rows: block b normalises the last row of branch b % M.
template <typename TW, typename TA>
__global__ __launch_bounds__(256) void k_last_inputs(const float *x, Branches br, const TW *g,
                                                     int d, float eps, int yes_id, int no_id,
                                                     TA *y, int32_t *lm_tgt) {
  __shared__ float red[4];
  const int b = blockIdx.x, m = b % br.M;
  const int t = br.cu[m + 1] - 1;  // every branch has at least one row
  norm_row(x + (long)t * d, g, d, eps, y + (long)b * d, red);
  if (threadIdx.x == 0) lm_tgt[b] = b < br.M ? yes_id : no_id;
}

template <typename TW, typename TA>
hipError_t launch_last_inputs(const float *x, const Branches &br, const TW *g, int d, float eps,
                              int yes_id, int no_id, TA *y, int32_t *lm_tgt, hipStream_t s) {
  k_last_inputs<TW, TA><<<2 * br.M, 256, 0, s>>>(x, br, g, d, eps, yes_id, no_id, y, lm_tgt);
  return hipGetLastError();
}

// ----------------------------------------------------- LSE merge and gather
// Log-sum-exp of LM-head row t (T rows) over its vocabulary chunks, by one
// wave (fixed order).
__device__ __forceinline__ float wave_lse(const float2 *part, int nchunks, int T, int t) {
  const int lane = threadIdx.x & 63;
  float mx = -INFINITY;
  for (int c = lane; c < nchunks; c += 64) mx = fmaxf(mx, part[(long)c * T + t].x);
  mx = wave_max(mx);
  float sum = 0.f;
  for (int c = lane; c < nchunks; c += 64) {
    const float2 p = part[(long)c * T + t];
    sum += p.y * __expf(p.x - mx);
  }
  return mx + __logf(wave_sum(sum));
}

// One block: wave w handles branches w, w+4, ...; then thread 0 takes the
// maximum reliability and every thread marks its branches (Eq. 13).
__global__ __launch_bounds__(256) void k_reliability_finish(int M, const float2 *part,
                                                            int nchunks, const float *tgt,
                                                            float delta, float *lp_yes_no,
                                                            float *rel, int32_t *keep) {
  __shared__ float r[kMaxCands];
  __shared__ float best;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int m = w; m < M; m += 4) {
    const float ly = tgt[m] - wave_lse(part, nchunks, 2 * M, m);
    const float ln = tgt[M + m] - wave_lse(part, nchunks, 2 * M, M + m);
    if (lane == 0) {
      const float v = 1.f / (1.f + expf(ln - ly));
      lp_yes_no[2 * m] = ly;
      lp_yes_no[2 * m + 1] = ln;
      rel[m] = v;
      r[m] = v;
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float b = r[0];
    for (int m = 1; m < M; ++m) b = fmaxf(b, r[m]);
    best = b;
  }
  __syncthreads();
  for (int m = threadIdx.x; m < M; m += 256) keep[m] = r[m] >= best - delta ? 1 : 0;
}

hipError_t launch_reliability_finish(int M, const float2 *part, int nchunks,
                                     const float *tgt_logit, float delta, float *lp_yes_no,
                                     float *rel, int32_t *keep, hipStream_t s) {
  k_reliability_finish<<<1, 256, 0, s>>>(M, part, nchunks, tgt_logit, delta, lp_yes_no, rel,
                                         keep);
  return hipGetLastError();
}

// --------------------------------------------- entity alignment and choice
// Block m (16 waves): wave w takes frames w, w+16, ...; lanes stride over the
// D coordinates. cos = (e . f) / (|e| |f|), 0 if either norm is 0.
__global__ __launch_bounds__(1024) void k_align(const float *ent, const float *frames, int NF,
                                                int D, float *align) {
  __shared__ float red[16];
  const int m = blockIdx.x, w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const float *e = ent + (long)m * D;
  float ee = 0.f;
  for (int c = lane; c < D; c += 64) ee += e[c] * e[c];
  ee = wave_sum(ee);
  float best = -INFINITY;
  for (int f = w; f < NF; f += 16) {
    const float *fr = frames + (long)f * D;
    float ef = 0.f, ff = 0.f;
    for (int c = lane; c < D; c += 64) {
      const float v = fr[c];
      ef += e[c] * v;
      ff += v * v;
    }
    ef = wave_sum(ef);
    ff = wave_sum(ff);
    const float den = sqrtf(ee) * sqrtf(ff);
    best = fmaxf(best, den > 0.f ? ef / den : 0.f);
  }
  if (lane == 0) red[w] = best;
  __syncthreads();
  if (threadIdx.x == 0) {
    float b = red[0];
    for (int i = 1; i < 16; ++i) b = fmaxf(b, red[i]);
    align[m] = b;
  }
}

// First index of the largest value among the allowed ones (-1 if none).
__device__ __forceinline__ int argmax_where(const float *v, const bool *ok, int n) {
  int best = -1;
  for (int i = 0; i < n; ++i)
    if (ok[i] && (best < 0 || v[i] > v[best])) best = i;
  return best;
}

__global__ __launch_bounds__(64) void k_choose(const float *rel, const float *align, int M,
                                               float delta, int strategy, int32_t *choice) {
  __shared__ float r[kMaxCands], a[kMaxCands], sum[kMaxCands];
  __shared__ bool ok[kMaxCands];
  for (int m = threadIdx.x; m < M; m += 64) {
    r[m] = rel[m];
    a[m] = align[m];
    sum[m] = r[m] + a[m];
  }
  __syncthreads();
  if (threadIdx.x != 0) return;
  int best;
  if (strategy == 1) {  // addition
    for (int m = 0; m < M; ++m) ok[m] = true;
    best = argmax_where(sum, ok, M);
  } else {
    const float *filt = strategy == 0 ? r : a, *rank = strategy == 0 ? a : r;
    float mx = filt[0];
    for (int m = 1; m < M; ++m) mx = fmaxf(mx, filt[m]);
    for (int m = 0; m < M; ++m) ok[m] = filt[m] >= mx - delta;
    best = argmax_where(rank, ok, M);
  }
  *choice = best;
}

hipError_t launch_align_select(const float *ent, const float *frames, int M, int NF, int D,
                               const float *rel, float delta, int strategy, float *align,
                               int32_t *choice, hipStream_t s) {
  k_align<<<M, 1024, 0, s>>>(ent, frames, NF, D, align);
  k_choose<<<1, 64, 0, s>>>(rel, align, M, delta, strategy, choice);
  return hipGetLastError();
}


// One wave per output slot (m, j); lanes stride over the vocabulary chunks.
__global__ __launch_bounds__(256) void k_lse_gather(Branches br, const float2 *part,
                                                    int nchunks, const float *tgt_logit,
                                                    float *logprobs) {
  const int slot = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (slot >= br.M * br.cmax) return;
  const int m = slot / br.cmax, j = slot % br.cmax;
  const int n = br.cu[m + 1] - br.cu[m];
  if (j >= n) {
    if (lane == 0) logprobs[slot] = 0.f;
    return;
  }
  const int t = br.cu[m] + j;
  const float lse = wave_lse(part, nchunks, br.cu[br.M], t);
  if (lane == 0) logprobs[slot] = tgt_logit[t] - lse;
}

hipError_t launch_lse_gather(const Branches &br, const float2 *part, int nchunks,
                             const float *tgt_logit, float *logprobs, hipStream_t s) {
  const int slots = br.M * br.cmax;
  k_lse_gather<<<(slots + 3) / 4, 256, 0, s>>>(br, part, nchunks, tgt_logit, logprobs);
  return hipGetLastError();
}

// ------------------------------------------------- per-candidate sum, argmax
// One block; wave w sums candidates w, w+4, ... with a fixed lane order, then
// thread 0 takes the first index of the largest score (Eq. 7).
__global__ __launch_bounds__(256) void k_reduce_select(Branches br, const float *logprobs,
                                                       float *scores, int32_t *argmax) {
  __shared__ float sc[kMaxCands];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int m = w; m < br.M; m += 4) {
    const int n = br.cu[m + 1] - br.cu[m];
    float v = 0.f;
    for (int j = lane; j < n; j += 64) v += logprobs[(long)m * br.cmax + j];
    v = wave_sum(v);
    if (lane == 0) {
      sc[m] = v;
      scores[m] = v;
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int best = 0;
    for (int m = 1; m < br.M; ++m)
      if (sc[m] > sc[best]) best = m;
    *argmax = best;
  }
}

hipError_t launch_reduce_select(const Branches &br, const float *logprobs, float *scores,
                                int32_t *argmax, hipStream_t s) {
  k_reduce_select<<<1, 256, 0, s>>>(br, logprobs, scores, argmax);
  return hipGetLastError();
}

#define VSR_INST(T)                                                                          \
  template hipError_t launch_embed_prefix<T>(const T *, int, const int32_t *, int, const T *, \
                                             int, int, float *, int32_t *, hipStream_t);    \
  template hipError_t launch_embed_rows<T>(const int32_t *, int, const T *, int, float *,     \
                                           hipStream_t);
VSR_INST(float)
VSR_INST(bf16)
#undef VSR_INST
#define VSR_INST2(TW, TA)                                                                     \
  template hipError_t launch_rmsnorm<TW, TA>(const float *, const TW *, int, int, float,      \
                                             TA *, int, hipStream_t);                         \
  template hipError_t launch_lm_inputs<TW, TA>(const float *, const float *, const int32_t *, \
                                               const TW *, int, int, float, TA *, hipStream_t); \
  template hipError_t launch_last_inputs<TW, TA>(const float *, const Branches &, const TW *, \
                                                 int, float, int, int, TA *, int32_t *,       \
                                                 hipStream_t);                                \
  template hipError_t launch_branch_last_norm<TW, TA>(const float *, const Branches &,        \
                                                      const TW *, int, float, TA *,           \
                                                      hipStream_t);
VSR_INST2(float, float)
VSR_INST2(bf16, f16)
#undef VSR_INST2

}  // namespace vsr
