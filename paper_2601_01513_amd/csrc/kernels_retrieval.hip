// Retrieval stage of VideoSpeculateRAG (Section 3.1, Eq. 1-3): keyframes by
// colour-histogram intersection of neighbouring frames, then per-keyframe
// top-k documents by the cosine of CLIP embeddings and the merged top-K.
//
// Every decision is integer or uses one fixed reduction order, so repeated
// calls give identical results: histogram counts are integer LDS atomics;
// the keyframe test compares an integer sum with theta * 3HW in float64;
// rankings break ties by the lower document index.
#include "common.h"

namespace vsr {

namespace {

constexpr int BINS = 64;            // per channel, bin = value >> 2
constexpr int HB = 3 * BINS;        // bins of one frame
constexpr int HIST_T = 1024;        // threads of the histogram block
constexpr int HIST_W = HIST_T / 64;

// Block f: the histogram of frame f. Each wave counts into its own LDS copy
// (less contention on flat scenes), then the copies are summed.
__global__ __launch_bounds__(HIST_T) void k_hist(const uint8_t *frames, long frame_bytes,
                                                 int32_t *hist) {
  __shared__ int32_t h[HIST_W][HB];
  const int t = threadIdx.x, w = t >> 6;
  for (int i = t; i < HIST_W * HB; i += HIST_T) (&h[0][0])[i] = 0;
  __syncthreads();
  const uint8_t *src = frames + (long)blockIdx.x * frame_bytes;
  // 16-byte loads need every frame 16-byte aligned (the base is, by contract).
  const long n16 = frame_bytes % 16 == 0 ? frame_bytes / 16 : 0;
  // Byte b of the frame belongs to channel b % 3; a 16-byte chunk at byte
  // 16 i starts at channel (16 i) % 3 = i % 3.
  for (long i = t; i < n16; i += HIST_T) {
    const u32x4 v = reinterpret_cast<const u32x4 *>(src)[i];
    int c = (int)(i % 3);
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const uint32_t byte = (v[j >> 2] >> (8 * (j & 3))) & 0xFFu;
      atomicAdd(&h[w][c * BINS + (byte >> 2)], 1);
      c = c == 2 ? 0 : c + 1;
    }
  }
  for (long b = n16 * 16 + t; b < frame_bytes; b += HIST_T)
    atomicAdd(&h[w][(int)(b % 3) * BINS + (src[b] >> 2)], 1);
  __syncthreads();
  for (int i = t; i < HB; i += HIST_T) {
    int32_t s = 0;
    for (int k = 0; k < HIST_W; ++k) s += h[k][i];
    hist[(long)blockIdx.x * HB + i] = s;
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
  const int nvalid = min(RT, ND - d0);
  for (int r = w; r < ng; r += RW) {
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

// Block r < n_keys (one wave): the top-k of keyframe r over every chunk's
// top-k, k passes of a wave-wide best.
__global__ __launch_bounds__(64) void k_retrieve_merge(const SimIdx *part, const int32_t *n_keys,
                                                       int nchunks, int k, int32_t *top_idx,
                                                       float *top_sim) {
  const int r = blockIdx.x, lane = threadIdx.x;
  if (r >= *n_keys) return;
  const SimIdx *p = part + (long)r * nchunks * k;
  const int n = nchunks * k;
  float last_s = INFINITY;
  int last_i = -1;
  for (int q = 0; q < k; ++q) {
    float bs = -INFINITY;
    int bi = -1;
    for (int e = lane; e < n; e += 64) {
      const SimIdx c = p[e];
      if (c.i >= 0 && before(last_s, last_i, c.s, c.i)) keep_better(bs, bi, c.s, c.i);
    }
    wave_best(bs, bi);
    if (lane == 0) {
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
  k_hist<<<NF, HIST_T, 0, s>>>(frames, fb, hist);
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
  k_retrieve_chunk<<<dim3(nchunks, (NF + RG - 1) / RG), RT, 0, s>>>(
      frame_emb, key_idx, n_keys, docs, ND, D, k, nchunks, part);
  k_retrieve_merge<<<NF, 64, 0, s>>>(part, n_keys, nchunks, k, top_idx, top_sim);
  k_select_docs<<<1, 1024, 0, s>>>(top_idx, top_sim, n_keys, k, K, sel_idx, sel_sim, n_sel);
  return hipGetLastError();
}

}  // namespace vsr
