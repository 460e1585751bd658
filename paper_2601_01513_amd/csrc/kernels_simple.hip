// Plain kernels of the verifier scoring pass: one output element (or one
// rotary pair) per thread, dot products read straight from memory. They serve
// the fp32 contexts, whose shapes are small, and use the same buffers and
// layouts as the MFMA path so that either can fill a given stage.
#include "common.h"

namespace vsr {

template <typename T>
__device__ __forceinline__ float dot_row(const T *a, const T *b, int K) {
  float s = 0.f;
  for (int k = 0; k < K; ++k) s = fmaf(to_f32(a[k]), to_f32(b[k]), s);
  return s;
}

__device__ __forceinline__ float silu_f(float g) { return g / (1.f + __expf(-g)); }

// ------------------------------------------------------- QKV + rotary + cache
// grid (rows, n_heads + 2 n_kv), block hd/2: thread i owns the pair (i, i+hd/2).
template <typename T>
__global__ void k_simple_qkv(const T *A, const T *W, int K, int n_heads, int n_kv, int hd,
                             QKVOut<T> o) {
  const int row = blockIdx.x, slot = blockIdx.y, i = threadIdx.x, half = hd / 2;
  const T *a = A + (long)row * K;
  const T *w = W + (long)slot * hd * K;
  float x1 = dot_row(a, w + (long)i * K, K);
  float x2 = dot_row(a, w + (long)(i + half) * K, K);
  const int pos = o.row_pos ? o.row_pos[row] : row;
  if (slot < n_heads + n_kv) {
    const float2 cs = o.rope[(long)pos * half + i];
    const float y1 = x1 * cs.x - x2 * cs.y, y2 = x2 * cs.x + x1 * cs.y;
    x1 = y1;
    x2 = y2;
  }
  if (slot < n_heads) {
    T *q = o.q + ((long)row * n_heads + slot) * hd;
    q[i] = from_f32<T>(x1);
    q[i + half] = from_f32<T>(x2);
  } else if (slot < n_heads + n_kv) {
    const int crow = o.cache_row ? o.cache_row[row] : row;
    T *k = o.k + ((long)(slot - n_heads) * o.kv_npos + crow) * hd;
    k[i] = from_f32<T>(x1);
    k[i + half] = from_f32<T>(x2);
  } else {
    const int crow = o.cache_row ? o.cache_row[row] : row;
    T *vt = o.vt + (long)(slot - n_heads - n_kv) * hd * o.kv_npos;
    vt[(long)i * o.kv_npos + crow] = from_f32<T>(x1);
    vt[(long)(i + half) * o.kv_npos + crow] = from_f32<T>(x2);
  }
}

template <typename T>
hipError_t simple_qkv_rope(const T *A, const T *W, int rows, int K, int n_heads, int n_kv,
                           int hd, const QKVOut<T> &out, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  k_simple_qkv<T><<<dim3(rows, n_heads + 2 * n_kv), hd / 2, 0, s>>>(A, W, K, n_heads, n_kv,
                                                                     hd, out);
  return hipGetLastError();
}

// ------------------------------------------------------------ residual GEMM
template <typename T>
__global__ void k_simple_residual(const T *A, const T *W, int N, int K, float *x) {
  const int row = blockIdx.x, c = blockIdx.y * blockDim.x + threadIdx.x;
  if (c >= N) return;
  x[(long)row * N + c] += dot_row(A + (long)row * K, W + (long)c * K, K);
}

template <typename T>
hipError_t simple_residual(const T *A, const T *W, int rows, int N, int K, float *x,
                           hipStream_t s) {
  if (rows == 0) return hipSuccess;
  k_simple_residual<T><<<dim3(rows, (N + 127) / 128), 128, 0, s>>>(A, W, N, K, x);
  return hipGetLastError();
}

// --------------------------------------------------------------- SwiGLU FFN
template <typename T>
__global__ void k_simple_swiglu(const T *A, const T *W, int F, int K, T *h) {
  const int row = blockIdx.x, c = blockIdx.y * blockDim.x + threadIdx.x;
  if (c >= F) return;
  const T *a = A + (long)row * K;
  const float g = dot_row(a, W + (long)c * K, K);
  const float u = dot_row(a, W + (long)(F + c) * K, K);
  h[(long)row * F + c] = from_f32<T>(silu_f(g) * u);
}

template <typename T>
hipError_t simple_swiglu(const T *A, const T *W, int rows, int F, int K, T *h, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  k_simple_swiglu<T><<<dim3(rows, (F + 127) / 128), 128, 0, s>>>(A, W, F, K, h);
  return hipGetLastError();
}

// ------------------------------------------------------------------ LM head
// One block per row, one vocabulary chunk: online (max, sum exp) per thread,
// merged across the block in a fixed order.
template <typename T>
__global__ __launch_bounds__(256) void k_simple_lmhead(const T *A, const T *W, int vocab,
                                                       int K, const int32_t *lm_tgt,
                                                       float2 *part, float *tgt_logit) {
  __shared__ float sm[256], ss[256];
  const int t = blockIdx.x;
  const T *a = A + (long)t * K;
  const int tgt = lm_tgt[t];
  float m = -INFINITY, s = 0.f;
  for (int v = threadIdx.x; v < vocab; v += 256) {
    const float l = dot_row(a, W + (long)v * K, K);
    if (v == tgt) tgt_logit[t] = l;
    if (l > m) {
      s = s * __expf(m - l) + 1.f;
      m = l;
    } else {
      s += __expf(l - m);
    }
  }
  sm[threadIdx.x] = m;
  ss[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) {
      const float m1 = sm[threadIdx.x], m2 = sm[threadIdx.x + w];
      const float mm = fmaxf(m1, m2);
      const float s1 = m1 == -INFINITY ? 0.f : ss[threadIdx.x] * __expf(m1 - mm);
      const float s2 = m2 == -INFINITY ? 0.f : ss[threadIdx.x + w] * __expf(m2 - mm);
      sm[threadIdx.x] = mm;
      ss[threadIdx.x] = s1 + s2;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) part[t] = make_float2(sm[0], ss[0]);
}

template <typename T>
hipError_t simple_lmhead(const T *A, const T *W, int rows, int vocab, int K,
                         const int32_t *lm_tgt, float2 *part, float *tgt_logit,
                         hipStream_t s) {
  if (rows == 0) return hipSuccess;
  k_simple_lmhead<T><<<rows, 256, 0, s>>>(A, W, vocab, K, lm_tgt, part, tgt_logit);
  return hipGetLastError();
}

// Greedy variant: one block per row; each thread keeps the first best of its
// strided vocabulary subset, then a tree reduction prefers the lower index.
template <typename T>
__global__ __launch_bounds__(256) void k_simple_lmargmax(const T *A, const T *W, int vocab,
                                                         int K, float2 *part) {
  __shared__ float sv[256];
  __shared__ int si[256];
  const int t = blockIdx.x;
  const T *a = A + (long)t * K;
  float best = -INFINITY;
  int bi = -1;
  for (int v = threadIdx.x; v < vocab; v += 256) {
    const float l = dot_row(a, W + (long)v * K, K);
    if (bi < 0 || l > best) {
      best = l;
      bi = v;
    }
  }
  sv[threadIdx.x] = best;
  si[threadIdx.x] = bi;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) {
      const float v2 = sv[threadIdx.x + w];
      const int i2 = si[threadIdx.x + w];
      if (i2 >= 0 && (si[threadIdx.x] < 0 || v2 > sv[threadIdx.x] ||
                      (v2 == sv[threadIdx.x] && i2 < si[threadIdx.x]))) {
        sv[threadIdx.x] = v2;
        si[threadIdx.x] = i2;
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) part[t] = make_float2(sv[0], __int_as_float(si[0]));
}

template <typename T>
hipError_t simple_lmargmax(const T *A, const T *W, int rows, int vocab, int K, float2 *part,
                           hipStream_t s) {
  if (rows == 0) return hipSuccess;
  k_simple_lmargmax<T><<<rows, 256, 0, s>>>(A, W, vocab, K, part);
  return hipGetLastError();
}

// ---------------------------------------------------------------- attention
// One wave per (token, query head); online softmax over the visible keys in
// position order. Lane l owns dims l, l+64, ... of the head.
template <typename T>
__device__ __forceinline__ void attend_keys(const T *kc, const T *vtc, int npos, int lo, int hi,
                                            int hd, const float *q, float &m, float &l,
                                            float *acc) {
  const int lane = threadIdx.x;
  const float scale = rsqrtf((float)hd);
  for (int kp = lo; kp <= hi; ++kp) {
    float s = 0.f;
    for (int d = lane, i = 0; d < hd; d += 64, ++i) s += q[i] * to_f32(kc[(long)kp * hd + d]);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
    s *= scale;
    const float mn = fmaxf(m, s);
    const float alpha = __expf(m - mn), p = __expf(s - mn);
    l = l * alpha + p;
    for (int d = lane, i = 0; d < hd; d += 64, ++i)
      acc[i] = acc[i] * alpha + p * to_f32(vtc[(long)d * npos + kp]);
    m = mn;
  }
}

template <typename T>
__global__ __launch_bounds__(64) void k_simple_attn(SimpleAttnArgs a) {
  const int t = a.t0 + blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
  const int G = a.n_heads / a.n_kv, kv = h / G, hd = a.hd;
  const T *q = (const T *)a.q + ((long)t * a.n_heads + h) * hd;
  float qr[4], acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int d = lane, i = 0; d < hd; d += 64, ++i) qr[i] = to_f32(q[d]);
  float m = -INFINITY, l = 0.f;
  const T *kc = (const T *)a.k + (long)kv * a.kv_npos * hd;
  const T *vtc = (const T *)a.vt + (long)kv * hd * a.kv_npos;
  if (a.mode == 0) {
    attend_keys(kc, vtc, a.kv_npos, 0, t, hd, qr, m, l, acc);
  } else {
    attend_keys(kc, vtc, a.kv_npos, 0, a.P - 1, hd, qr, m, l, acc);
    const T *bk = (const T *)a.bk + (long)kv * a.bk_npos * hd;
    const T *bvt = (const T *)a.bvt + (long)kv * hd * a.bk_npos;
    attend_keys(bk, bvt, a.bk_npos, a.row_lo[t], a.q_pos ? a.q_pos[t] : t, hd, qr, m, l, acc);
  }
  T *o = (T *)a.out + ((long)t * a.n_heads + h) * hd;
  const float inv = 1.f / l;
  for (int d = lane, i = 0; d < hd; d += 64, ++i) o[d] = from_f32<T>(acc[i] * inv);
}

template <typename T>
hipError_t simple_attn(const SimpleAttnArgs &a, hipStream_t s) {
  if (a.T <= a.t0) return hipSuccess;
  k_simple_attn<T><<<dim3(a.T - a.t0, a.n_heads), 64, 0, s>>>(a);
  return hipGetLastError();
}

#define VSR_INST(T)                                                                           \
  template hipError_t simple_qkv_rope<T>(const T *, const T *, int, int, int, int, int,       \
                                         const QKVOut<T> &, hipStream_t);                     \
  template hipError_t simple_residual<T>(const T *, const T *, int, int, int, float *,        \
                                         hipStream_t);                                        \
  template hipError_t simple_swiglu<T>(const T *, const T *, int, int, int, T *, hipStream_t); \
  template hipError_t simple_lmhead<T>(const T *, const T *, int, int, int, const int32_t *,  \
                                       float2 *, float *, hipStream_t);                       \
  template hipError_t simple_attn<T>(const SimpleAttnArgs &, hipStream_t);                    \
  template hipError_t simple_lmargmax<T>(const T *, const T *, int, int, int, float2 *,       \
                                         hipStream_t);
VSR_INST(float)
VSR_INST(bf16)
#undef VSR_INST

}  // namespace vsr
