// Retrieval stage of VideoSpeculateRAG (Section 3.1, Eq. 1-3): keyframes by
// colour-histogram intersection of neighbouring frames, then per-keyframe
// top-k documents by the cosine of CLIP embeddings and the merged top-K.
//
// Every decision is integer or uses one fixed reduction order, so repeated
// calls give identical results: histogram counts are integer LDS atomics;
// the keyframe test compares an integer sum with theta * 3HW in float64;
// rankings break ties by the lower document index.
#include <mutex>

#include "common.h"

namespace vsr {

namespace {

constexpr int BINS = 64;            // per channel, bin = value >> 2
constexpr int HB = 3 * BINS;        // bins of one frame
constexpr int HIST_T = 1024;        // threads of the histogram block
constexpr int HIST_W = HIST_T / 64;

constexpr int HIST_SPLIT = 4;       // blocks per frame

__global__ void k_zero_i32(int32_t *p, long n) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

// Block (f, part): the histogram of part `part` of HIST_SPLIT of frame f's
// 16-byte chunks (and, for the last part, its trailing bytes), added into
// hist[f] (zeroed before) with integer atomics: exact, so the counts do not
// depend on the order. Each wave counts into its own LDS copy, then the
// copies are summed.
__global__ __launch_bounds__(HIST_T) void k_hist(const uint8_t *frames, long frame_bytes,
                                                 int32_t *hist) {
  __shared__ int32_t h[HIST_W][HB];
  const int t = threadIdx.x, w = t >> 6;
  const int f = blockIdx.x / HIST_SPLIT, part = blockIdx.x % HIST_SPLIT;
  for (int i = t; i < HIST_W * HB; i += HIST_T) (&h[0][0])[i] = 0;
  __syncthreads();
  const uint8_t *src = frames + (long)f * frame_bytes;
  // 16-byte loads need every frame 16-byte aligned (the base is, by contract).
  const long n16 = frame_bytes % 16 == 0 ? frame_bytes / 16 : 0;
  const long i0 = n16 * part / HIST_SPLIT, i1 = n16 * (part + 1) / HIST_SPLIT;
  // Byte b of the frame belongs to channel b % 3; a 16-byte chunk at byte
  // 16 i starts at channel (16 i) % 3 = i % 3.
  // Batches of HIST_B chunks per thread, all loads issued before counting.
  constexpr int HIST_B = 8;
  for (long i = i0 + t; i < i1; i += (long)HIST_B * HIST_T) {
    u32x4 v[HIST_B];
#pragma unroll
    for (int b = 0; b < HIST_B; ++b) {
      const long ib = i + (long)b * HIST_T;
      v[b] = ib < i1 ? reinterpret_cast<const u32x4 *>(src)[ib] : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int b = 0; b < HIST_B; ++b) {
      const long ib = i + (long)b * HIST_T;
      if (ib >= i1) break;
      int c = (int)(ib % 3);
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const uint32_t byte = (v[b][j >> 2] >> (8 * (j & 3))) & 0xFFu;
        atomicAdd(&h[w][c * BINS + (byte >> 2)], 1);
        c = c == 2 ? 0 : c + 1;
      }
    }
  }
  if (part == HIST_SPLIT - 1)
    for (long b = n16 * 16 + t; b < frame_bytes; b += HIST_T)
      atomicAdd(&h[w][(int)(b % 3) * BINS + (src[b] >> 2)], 1);
  __syncthreads();
  for (int i = t; i < HB; i += HIST_T) {
    int32_t s = 0;
    for (int k = 0; k < HIST_W; ++k) s += h[k][i];
    if (s) atomicAdd(&hist[(long)f * HB + i], s);
  }
}

// One block: inter[i] = sum_b min(hist[i][b], hist[i-1][b]) (inter[0] = -1),
// keyframe flags (frame 0, and inter[i] < theta * 3HW), then the ordered
// list of keyframe indices.
__global__ __launch_bounds__(1024) void k_keyframes(const int32_t *hist, int NF, double thr,
                                                    int32_t *inter, int32_t *key_idx,
                                                    int32_t *n_keys) {
  __shared__ int32_t cnt[1024];
  const int t = threadIdx.x;
  // Frames are handled in contiguous runs per thread so that the compaction
  // keeps their order.
  const int per = (NF + 1023) / 1024, f0 = t * per, f1 = min(NF, f0 + per);
  int mine = 0;
  for (int f = f0; f < f1; ++f) {
    bool key = f == 0;
    if (f > 0) {
      const int32_t *a = hist + (long)f * HB, *b = a - HB;
      int32_t s = 0;
      for (int i = 0; i < HB; ++i) s += min(a[i], b[i]);
      inter[f] = s;
      key = (double)s < thr;
    } else {
      inter[0] = -1;
    }
    mine += key;
  }
  cnt[t] = mine;
  __syncthreads();
  // Exclusive prefix sum of the per-thread counts (Hillis-Steele in LDS).
  for (int off = 1; off < 1024; off <<= 1) {
    const int v = t >= off ? cnt[t - off] : 0;
    __syncthreads();
    cnt[t] += v;
    __syncthreads();
  }
  int pos = cnt[t] - mine;
  for (int f = f0; f < f1; ++f) {
    const bool key = f == 0 || (double)inter[f] < thr;
    if (key) key_idx[pos++] = f;
  }
  if (t == 1023) *n_keys = cnt[1023];
}

constexpr int RG = 16;       // keyframes per retrieval block
constexpr int RT = 256;      // threads of a retrieval block = documents per block
constexpr int RW = RT / 64;

struct SimIdx {
  float s;
  int32_t i;
};

// a ranks before b: higher similarity, then lower document index.
__device__ __forceinline__ bool before(float sa, int ia, float sb, int ib) {
  return sa > sb || (sa == sb && ia < ib);
}

// The better of two (similarity, index) candidates; index -1 is no candidate.
__device__ __forceinline__ void keep_better(float &s, int &i, float s2, int i2) {
  if (i2 >= 0 && (i < 0 || before(s2, i2, s, i))) {
    s = s2;
    i = i2;
  }
}

// Best candidate of the wave (fixed butterfly order), in every lane.
__device__ __forceinline__ void wave_best(float &s, int &i) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float s2 = __shfl_xor(s, o, 64);
    const int i2 = __shfl_xor(i, o, 64);
    keep_better(s, i, s2, i2);
  }
}

// The per-chunk top-k of keyframes g0 .. g0+ng-1 from sims [RG][RT] in LDS:
// wave w of NWV takes keyframes w, w + NWV, ..., k passes of a wave-wide best.
template <int NWV>
__device__ __forceinline__ void chunk_topk(const float (*sims)[RT], int g0, int ng, int d0,
                                           int nvalid, int k, int nchunks, SimIdx *part) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int r = w; r < ng; r += NWV) {
    SimIdx *out = part + ((long)(g0 + r) * nchunks + blockIdx.x) * k;
    float last_s = INFINITY;
    int last_i = -1;
    for (int p = 0; p < k; ++p) {
      float bs = -INFINITY;
      int bi = -1;
      for (int j = lane; j < nvalid; j += 64) {
        const float sj = sims[r][j];
        if (before(last_s, last_i, sj, d0 + j)) keep_better(bs, bi, sj, d0 + j);
      }
      wave_best(bs, bi);
      if (lane == 0) out[p] = SimIdx{bs, bi};  // -1: fewer than k documents left
      last_s = bi < 0 ? -INFINITY : bs;
      last_i = bi;
    }
  }
}

// Block (document chunk, keyframe group): thread t scores document
// d0 + t against up to RG keyframes held in LDS (every lane reads the same
// keyframe value: an LDS broadcast), then wave w picks the top-k of the chunk
// for keyframes w, w + RW, ... -> part[key][chunk][k].
__global__ __launch_bounds__(RT) void k_retrieve_chunk(const float *frame_emb,
                                                       const int32_t *key_idx,
                                                       const int32_t *n_keys,
                                                       const float *docs, int ND, int D, int k,
                                                       int nchunks, SimIdx *part) {
  __shared__ __align__(16) float q[RG][1024];
  __shared__ float qn[RG];
  __shared__ float sims[RG][RT];
  const int nk = *n_keys;
  const int g0 = blockIdx.y * RG;
  if (g0 >= nk) return;  // uniform per block
  const int ng = min(RG, nk - g0);
  const int t = threadIdx.x, w = t >> 6, lane = t & 63;
  for (int r = 0; r < ng; ++r) {
    const float *src = frame_emb + (long)key_idx[g0 + r] * D;
    for (int c = t; c < D; c += RT) q[r][c] = src[c];
  }
  __syncthreads();
  for (int r = w; r < ng; r += RW) {
    float s = 0.f;
    for (int c = lane; c < D; c += 64) s += q[r][c] * q[r][c];
    s = wave_sum(s);
    if (lane == 0) qn[r] = sqrtf(s);
  }
  __syncthreads();
  const int d0 = blockIdx.x * RT, doc = d0 + t;
  float dot[RG], dd = 0.f;
#pragma unroll
  for (int r = 0; r < RG; ++r) dot[r] = 0.f;
  if (doc < ND) {
    const float *src = docs + (long)doc * D;
    if ((D & 3) == 0) {  // rows 16-byte aligned (the base is, by contract)
      for (int c = 0; c < D; c += 4) {
        const float4 v = *reinterpret_cast<const float4 *>(src + c);
        dd += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
#pragma unroll
        for (int r = 0; r < RG; ++r) {
          const float4 e = *reinterpret_cast<const float4 *>(&q[r][c]);
          dot[r] += e.x * v.x + e.y * v.y + e.z * v.z + e.w * v.w;
        }
      }
    } else {
      for (int c = 0; c < D; ++c) {
        const float v = src[c];
        dd += v * v;
#pragma unroll
        for (int r = 0; r < RG; ++r) dot[r] += q[r][c] * v;
      }
    }
  }
  const float dn = sqrtf(dd);
#pragma unroll
  for (int r = 0; r < RG; ++r) {
    if (r < ng) {
      const float den = qn[r] * dn;
      sims[r][t] = den > 0.f ? dot[r] / den : 0.f;
    }
  }
  __syncthreads();
  chunk_topk<RW>(sims, g0, ng, d0, min(RT, ND - d0), k, nchunks, part);
}

// Matrix-core scan for D % 16 == 0: the dot products of a chunk's 256
// documents with up to 16 keyframes are a [256 x D] . [D x 16] product in
// fp32 (v_mfma_f32_16x16x4_f32). Eight waves; wave w owns documents
// 32 w .. 32 w + 31 as two 16-row tiles. Per 16 dimensions lane l loads 4
// consecutive values of document (l % 16) of each tile (16 rows x 64
// contiguous bytes per load) and the matching 4 values of keyframe (l % 16)
// from LDS, and runs 4 products per tile (product j takes dimension
// 4 (l / 16) + j of each lane group, the same for both operands). The
// documents' squared norms come from the same loads. Steps of 64 dimensions;
// the next step's loads are issued before the current step's products.
constexpr int RM_T = 512;
__global__ __launch_bounds__(RM_T) void k_retrieve_mfma(const float *frame_emb,
                                                        const int32_t *key_idx,
                                                        const int32_t *n_keys, const float *docs,
                                                        int ND, int D, int k, int nchunks,
                                                        SimIdx *part) {
  constexpr int NG = RT / (RM_T / 64) / 16;  // 16-row tiles per wave
  // The keyframes, [RG][D] (dynamic: D floats a row, so that two blocks fit
  // a CU at D = 768).
  extern __shared__ __align__(16) float q[];
  __shared__ float qn[RG];
  __shared__ float dn[RT];
  __shared__ float sims[RG][RT];
  const int nk = *n_keys;
  const int g0 = blockIdx.y * RG;
  if (g0 >= nk) return;  // uniform per block
  const int ng = min(RG, nk - g0);
  const int t = threadIdx.x, w = t >> 6, lane = t & 63;
  for (int r = 0; r < RG; ++r) {  // rows past ng: zeros (their columns are unused)
    const float *src = frame_emb + (long)key_idx[g0 + min(r, ng - 1)] * D;
    for (int c = t; c < D; c += RM_T) q[r * D + c] = r < ng ? src[c] : 0.f;
  }
  __syncthreads();
  for (int r = w; r < ng; r += RM_T / 64) {
    float s = 0.f;
    for (int c = lane; c < D; c += 64) s += q[r * D + c] * q[r * D + c];
    s = wave_sum(s);
    if (lane == 0) qn[r] = sqrtf(s);
  }
  const int d0 = blockIdx.x * RT;
  const int sub = 4 * (lane >> 4);
  const float *dp[NG];
#pragma unroll
  for (int g = 0; g < NG; ++g)
    dp[g] = docs + (long)min(d0 + 16 * NG * w + 16 * g + (lane & 15), ND - 1) * D + sub;
  const float *qp = q + (lane & 15) * D + sub;
  f32x4 acc[NG];
  float dd[NG];
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    acc[g] = f32x4{0.f, 0.f, 0.f, 0.f};
    dd[g] = 0.f;
  }
  // Loads of the step at dimension c (pieces past D repeat the last one).
  auto load = [&](int c, float4 (&v)[4][NG]) {
    const int cnt = min(4, (D - c) / 16);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int cc = c + 16 * min(u, cnt - 1);
#pragma unroll
      for (int g = 0; g < NG; ++g) v[u][g] = *reinterpret_cast<const float4 *>(dp[g] + cc);
    }
  };
  auto step = [&](int c, const float4 (&v)[4][NG]) {
    const int cnt = min(4, (D - c) / 16);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (u >= cnt) break;
      const float4 e = *reinterpret_cast<const float4 *>(qp + c + 16 * u);
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        const float4 x = v[u][g];
        dd[g] += x.x * x.x + x.y * x.y + x.z * x.z + x.w * x.w;
        acc[g] = __builtin_amdgcn_mfma_f32_16x16x4f32(x.x, e.x, acc[g], 0, 0, 0);
        acc[g] = __builtin_amdgcn_mfma_f32_16x16x4f32(x.y, e.y, acc[g], 0, 0, 0);
        acc[g] = __builtin_amdgcn_mfma_f32_16x16x4f32(x.z, e.z, acc[g], 0, 0, 0);
        acc[g] = __builtin_amdgcn_mfma_f32_16x16x4f32(x.w, e.w, acc[g], 0, 0, 0);
      }
    }
  };
  float4 va[4][NG], vb[4][NG];
  load(0, va);
  for (int c = 0; c < D; c += 128) {
    if (c + 64 < D) load(c + 64, vb);
    __builtin_amdgcn_sched_barrier(0);
    step(c, va);
    if (c + 64 >= D) break;
    if (c + 128 < D) load(c + 128, va);
    __builtin_amdgcn_sched_barrier(0);
    step(c + 64, vb);
  }
  // Squared norm of document 16 NG w + 16 g + l % 16: the four lane groups'
  // partial sums (fixed order).
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    float s = dd[g];
    s += __shfl_xor(s, 16, 64);
    s += __shfl_xor(s, 32, 64);
    if (lane < 16) dn[16 * NG * w + 16 * g + lane] = sqrtf(s);
  }
  __syncthreads();
  // Lane l holds document 16 NG w + 16 g + 4 (l / 16) + i against keyframe l % 16.
  const int r = lane & 15;
  if (r < ng) {
#pragma unroll
    for (int g = 0; g < NG; ++g)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = 16 * NG * w + 16 * g + 4 * (lane >> 4) + i;
        const float den = qn[r] * dn[j];
        sims[r][j] = den > 0.f ? acc[g][i] / den : 0.f;
      }
  }
  __syncthreads();
  chunk_topk<RM_T / 64>(sims, g0, ng, d0, min(RT, ND - d0), k, nchunks, part);
}

// Block r < n_keys: the top-k of keyframe r over every chunk's top-k. Each
// thread holds its first MERGE_PER candidates in registers (loaded once; a
// larger bank's further candidates are re-read on each pass); k passes of a
// block-wide best (wave butterflies, then the waves in order).
constexpr int MERGE_T = 1024;
constexpr int MERGE_PER = 8;
__global__ __launch_bounds__(MERGE_T) void k_retrieve_merge(const SimIdx *part,
                                                            const int32_t *n_keys, int nchunks,
                                                            int k, int32_t *top_idx,
                                                            float *top_sim) {
  __shared__ float ws[MERGE_T / 64];
  __shared__ int wi[MERGE_T / 64];
  const int r = blockIdx.x, t = threadIdx.x, lane = t & 63, w = t >> 6;
  if (r >= *n_keys) return;  // uniform per block
  const SimIdx *p = part + (long)r * nchunks * k;
  const int n = nchunks * k;
  float cs[MERGE_PER];
  int ci[MERGE_PER];
#pragma unroll
  for (int e = 0; e < MERGE_PER; ++e) {
    const int j = t + e * MERGE_T;
    const SimIdx c = j < n ? p[j] : SimIdx{-INFINITY, -1};
    cs[e] = c.s;
    ci[e] = c.i;
  }
  float last_s = INFINITY;
  int last_i = -1;
  for (int q = 0; q < k; ++q) {
    float bs = -INFINITY;
    int bi = -1;
#pragma unroll
    for (int e = 0; e < MERGE_PER; ++e)
      if (ci[e] >= 0 && before(last_s, last_i, cs[e], ci[e])) keep_better(bs, bi, cs[e], ci[e]);
    for (int j = t + MERGE_PER * MERGE_T; j < n; j += MERGE_T) {
      const SimIdx c = p[j];
      if (c.i >= 0 && before(last_s, last_i, c.s, c.i)) keep_better(bs, bi, c.s, c.i);
    }
    wave_best(bs, bi);
    if (lane == 0) {
      ws[w] = bs;
      wi[w] = bi;
    }
    __syncthreads();
    bs = ws[0];
    bi = wi[0];
    for (int i = 1; i < MERGE_T / 64; ++i) keep_better(bs, bi, ws[i], wi[i]);
    __syncthreads();
    if (t == 0) {
      top_idx[(long)r * k + q] = bi;
      top_sim[(long)r * k + q] = bi < 0 ? 0.f : bs;
    }
    last_s = bi < 0 ? -INFINITY : bs;
    last_i = bi;
  }
}

// One block: T* = the K best documents of the union of the top-k lists, a
// document scored by the best similarity it was retrieved with (Eq. 3).
__global__ __launch_bounds__(1024) void k_select_docs(const int32_t *top_idx,
                                                      const float *top_sim,
                                                      const int32_t *n_keys, int k, int K,
                                                      int32_t *sel_idx, float *sel_sim,
                                                      int32_t *n_sel) {
  __shared__ float bs[1024];
  __shared__ int bi[1024];
  __shared__ int chosen[64];
  const int t = threadIdx.x, n = *n_keys * k;
  int got = 0;
  for (int q = 0; q < K; ++q) {
    // Thread-local best among entries not yet chosen.
    float s = -INFINITY;
    int i = -1;
    for (int e = t; e < n; e += 1024) {
      const int d = top_idx[e];
      if (d < 0) continue;
      bool taken = false;
      for (int c = 0; c < got; ++c) taken = taken || chosen[c] == d;
      if (taken) continue;
      const float v = top_sim[e];
      if (i < 0 || before(v, d, s, i)) {
        s = v;
        i = d;
      }
    }
    bs[t] = s;
    bi[t] = i;
    __syncthreads();
    for (int off = 512; off > 0; off >>= 1) {
      if (t < off) {
        const int j = bi[t + off];
        if (j >= 0 && (bi[t] < 0 || before(bs[t + off], j, bs[t], bi[t]))) {
          bs[t] = bs[t + off];
          bi[t] = j;
        }
      }
      __syncthreads();
    }
    const int best = bi[0];
    const float bsim = bs[0];
    __syncthreads();
    if (best < 0) break;  // uniform: every thread read the same bi[0]
    if (t == 0) {
      sel_idx[got] = best;
      sel_sim[got] = bsim;
      chosen[got] = best;
    }
    ++got;
    __syncthreads();
  }
  if (t == 0) *n_sel = got;
}

}  // namespace

hipError_t launch_keyframes(const uint8_t *frames, int NF, int H, int W, float theta,
                            int32_t *hist, int32_t *inter, int32_t *key_idx, int32_t *n_keys,
                            hipStream_t s) {
  const long fb = (long)H * W * 3;
  const long nh = (long)NF * HB;
  k_zero_i32<<<(unsigned)((nh + 255) / 256), 256, 0, s>>>(hist, nh);
  k_hist<<<NF * HIST_SPLIT, HIST_T, 0, s>>>(frames, fb, hist);
  const double thr = (double)theta * 3.0 * (double)((long)H * W);  // (theta 3) (H W)
  k_keyframes<<<1, 1024, 0, s>>>(hist, NF, thr, inter, key_idx, n_keys);
  return hipGetLastError();
}

size_t retrieve_workspace_bytes(int NF, int ND, int k) {
  const size_t nchunks = ((size_t)ND + RT - 1) / RT;
  return (size_t)NF * nchunks * (size_t)k * sizeof(SimIdx);
}

hipError_t launch_retrieve(const float *frame_emb, const int32_t *key_idx, const int32_t *n_keys,
                           int NF, const float *docs, int ND, int D, int k, int K, void *ws,
                           int32_t *top_idx, float *top_sim, int32_t *sel_idx, float *sel_sim,
                           int32_t *n_sel, hipStream_t s) {
  const int nchunks = (ND + RT - 1) / RT;
  SimIdx *part = static_cast<SimIdx *>(ws);
  const dim3 grid(nchunks, (NF + RG - 1) / RG);
  if (D % 16 == 0)
    k_retrieve_mfma<<<grid, RM_T, RG * D * sizeof(float), s>>>(frame_emb, key_idx, n_keys, docs,
                                                               ND, D, k, nchunks, part);
  else
    k_retrieve_chunk<<<grid, RT, 0, s>>>(frame_emb, key_idx, n_keys, docs, ND, D, k, nchunks,
                                         part);
  k_retrieve_merge<<<NF, MERGE_T, 0, s>>>(part, n_keys, nchunks, k, top_idx, top_sim);
  k_select_docs<<<1, 1024, 0, s>>>(top_idx, top_sim, n_keys, k, K, sel_idx, sel_sim, n_sel);
  return hipGetLastError();
}

// ---- the same retrieval with library-owned scratch ------------------------
// For callers that cannot allocate device memory: the per-chunk partial lists
// live in this file-scope array (one copy per GPU, held until the process
// ends). Host code never passes the array's name to a kernel: it is a
// host-side stand-in there. The device address comes from
// hipGetSymbolAddress, looked up once per device with that device current.
static __device__ __align__(256) unsigned char scratch[kRetrieveStaticBytes];

namespace {
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t retrieve_static_scratch(void **ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace vsr
