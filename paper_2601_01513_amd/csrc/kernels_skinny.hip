// Projections of a few rows (decode steps of the drafter, the prefix pass's
// last-row layer): Y = A W^T with A [rows <= 32][K] fp16 activations and W
// [N][K] weights. With so few rows the product is a stream over the weights,
// bound by HBM bandwidth, not by the matrix cores: the kernel's job is to keep
// enough weight bytes in flight on every CU, in as few launches as possible.
//
// Layout of the work: a wave owns 16 weight rows and one K slice; it streams
// its rows in 256-wide K steps (eight 16-byte weight loads per lane and the
// matching activation loads, all issued before the first use), each 32-wide
// piece feeding one v_mfma_f32_16x16x32_f16 with the weights as the 16-row
// operand and up to 16 activation rows as the 16-column operand (a second
// product per row group for the fp16 remainder half of precise-layer rows, a
// second row group for 17..32 rows). A block is four waves over one group of
// 64 weight rows and the same K slice, so their activation loads hit the same
// cache lines.
//
// The K slices write fp32 partials part[s][row][n]; a small reduce kernel
// sums them in slice order (deterministic) and applies the epilogue: residual
// add (+ the RMSNorm that follows), SwiGLU, or rotary + cache scatter. (A
// reduction by the last-arriving block of each group would save that launch,
// but its cross-block release is an L2 writeback per block on this chip,
// which costs more than the launch.)
#include <algorithm>

#include "common.h"

namespace vsr {

namespace {

constexpr int SK_ROWS = 64;   // weight rows per block (16 per wave)
constexpr int SK_STEP = 256;  // K per unrolled step
constexpr int SK_U = SK_STEP / 32;

__device__ __forceinline__ f16x8 as_h8(u32x4 v) { return __builtin_bit_cast(f16x8, v); }

// Eight bf16 weights -> fp16 with the tile GEMMs' rounding (exact for
// magnitudes in [2^-17, 65504]).
__device__ __forceinline__ u32x4 sk_bf16_to_f16(u32x4 v) {
  u32x4 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float lo = __uint_as_float(v[i] << 16);
    const float hi = __uint_as_float(v[i] & 0xFFFF0000u);
    r[i] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pkrtz(lo, hi));
  }
  return r;
}

__device__ __forceinline__ u32x4 ld16(const void *p) {
  return *reinterpret_cast<const u32x4 *>(p);
}

// Sum of the ksplit slices of element i in slice order. All loads are issued
// before the first add (slices past ksplit re-load the last one and add 0).
__device__ __forceinline__ float sum_slices(const float *part, int ksplit, long stride,
                                            long i) {
  float v[kSkinnyMaxSplit];
#pragma unroll
  for (int s = 0; s < kSkinnyMaxSplit; ++s) v[s] = part[min(s, ksplit - 1) * stride + i];
  float acc = v[0];
#pragma unroll
  for (int s = 1; s < kSkinnyMaxSplit; ++s) acc += s < ksplit ? v[s] : 0.f;
  return acc;
}

// RG row groups of 16 activation rows; AS = 2: rows are [hi | lo] of width 2K.
// ARGMAX (one K slice): instead of the products, each block writes, per row,
// the largest of its 64 outputs and the lowest index holding it,
// part[blockIdx.x][row] = (value, index bits).
template <int RG, int AS, bool WCVT, bool ARGMAX>
__global__ __launch_bounds__(256) void k_skinny(const f16 *__restrict__ A, int rows,
                                                const uint16_t *__restrict__ W, int N, int K,
                                                int ksplit, float *__restrict__ part) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int b = blockIdx.x, s = blockIdx.y;
  const int n0 = SK_ROWS * b + 16 * w;
  // Slices are whole 256-wide steps (only the last one may end short).
  const int nsteps = (K + SK_STEP - 1) / SK_STEP;
  const int k0 = (int)((long)nsteps * s / ksplit) * SK_STEP;
  const int k1 = min(K, (int)((long)nsteps * (s + 1) / ksplit) * SK_STEP);
  const int sub = 8 * (lane >> 4);  // this lane's 8 of each 32-wide K piece
  const uint16_t *wp = W + (long)(n0 + (lane & 15)) * K + sub;
  const f16 *ap[RG];
#pragma unroll
  for (int g = 0; g < RG; ++g)
    ap[g] = A + (long)min(g * 16 + (lane & 15), rows - 1) * K * AS + sub;
  f32x4 acc[RG];
#pragma unroll
  for (int g = 0; g < RG; ++g) acc[g] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int k = k0; k < k1; k += SK_STEP) {
    // Every load of the step is issued before the first product; pieces past
    // the slice end (a short last step) re-load its last piece and multiply
    // zero activations (cnt is the same for the whole wave).
    const int cnt = min(SK_U, (k1 - k) / 32);
    u32x4 wv[SK_U], av[SK_U][RG][AS];
#pragma unroll
    for (int u = 0; u < SK_U; ++u) {
      const int kk = k + 32 * min(u, cnt - 1);
      wv[u] = ld16(wp + kk);
#pragma unroll
      for (int g = 0; g < RG; ++g)
#pragma unroll
        for (int h = 0; h < AS; ++h) av[u][g][h] = ld16(ap[g] + h * K + kk);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < SK_U; ++u) {
      const f16x8 wf = as_h8(WCVT ? sk_bf16_to_f16(wv[u]) : wv[u]);
      const u32x4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int g = 0; g < RG; ++g)
#pragma unroll
        for (int h = 0; h < AS; ++h)
          acc[g] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
              wf, as_h8(u < cnt ? av[u][g][h] : zero), acc[g], 0, 0, 0);
    }
  }
  // Lane l holds activation row l % 16 of each group and weight rows
  // n0 + 4 (l / 16) + i, i < 4.
  if constexpr (ARGMAX) {
    __shared__ float bv[4][16 * RG];
    __shared__ int bi[4][16 * RG];
#pragma unroll
    for (int g = 0; g < RG; ++g) {
      float v = acc[g][0];
      int vi = n0 + 4 * (lane >> 4);
#pragma unroll
      for (int i = 1; i < 4; ++i)
        if (acc[g][i] > v) {  // ascending indices: a strict > keeps the lowest
          v = acc[g][i];
          vi = n0 + 4 * (lane >> 4) + i;
        }
#pragma unroll
      for (int o = 16; o < 64; o <<= 1) {
        const float v2 = __shfl_xor(v, o, 64);
        const int i2 = __shfl_xor(vi, o, 64);
        if (v2 > v || (v2 == v && i2 < vi)) {
          v = v2;
          vi = i2;
        }
      }
      if (lane < 16) {
        bv[w][g * 16 + lane] = v;
        bi[w][g * 16 + lane] = vi;
      }
    }
    __syncthreads();
    const int r = threadIdx.x;
    if (r < 16 * RG && r < rows) {
      float v = bv[0][r];
      int vi = bi[0][r];
#pragma unroll
      for (int i = 1; i < 4; ++i)
        if (bv[i][r] > v) {  // waves hold ascending index ranges
          v = bv[i][r];
          vi = bi[i][r];
        }
      reinterpret_cast<float2 *>(part)[(long)b * rows + r] = make_float2(v, __int_as_float(vi));
    }
  } else {
#pragma unroll
    for (int g = 0; g < RG; ++g) {
      const int r = g * 16 + (lane & 15);
      if (r < rows)
        *reinterpret_cast<f32x4 *>(part + ((long)s * rows + r) * N + n0 + 4 * (lane >> 4)) =
            acc[g];
    }
  }
}

// Block per row: x += sum of the slices; then, if g is given, the RMSNorm of
// the new row into y (fp16, with its remainder half when split == 2).
__global__ __launch_bounds__(1024) void k_skinny_residual(const float *__restrict__ part,
                                                          int ksplit, int rows, int d,
                                                          float *__restrict__ x, const bf16 *g,
                                                          float eps, f16 *__restrict__ y,
                                                          int split) {
  __shared__ float red[16];
  const int r = blockIdx.x, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  float *xr = x + (long)r * d;
  const long stride = (long)rows * d;
  float ss = 0.f;
  for (int c = threadIdx.x; c < d; c += 1024) {
    const float v = xr[c] + sum_slices(part, ksplit, stride, (long)r * d + c);
    xr[c] = v;
    ss += v * v;
  }
  if (!g) return;
  ss = wave_sum(ss);
  if (lane == 0) red[w] = ss;
  __syncthreads();
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < 16; ++i) t += red[i];
  const float rs = rsqrtf(t / (float)d + eps);
  f16 *yr = y + (long)r * d * split;
  for (int c = threadIdx.x; c < d; c += 1024) {
    const float v = xr[c] * rs * static_cast<float>(g[c]);
    const f16 hi = static_cast<f16>(v);
    yr[c] = hi;
    if (split == 2) yr[d + c] = static_cast<f16>(v - static_cast<float>(hi));
  }
}

// Thread per (row, f): h = silu(gate) * up from the summed slices (gate rows
// 0..F-1, up rows F..2F-1 of the product), fp16 with its remainder half when
// hsplit == 2.
__global__ __launch_bounds__(256) void k_skinny_swiglu(const float *__restrict__ part,
                                                       int ksplit, int rows, int F, int hsplit,
                                                       f16 *__restrict__ h) {
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= (long)rows * F) return;
  const int r = (int)(i / F), f = (int)(i % F);
  const long stride = (long)rows * 2 * F, base = (long)r * 2 * F;
  const float gt = sum_slices(part, ksplit, stride, base + f);
  const float up = sum_slices(part, ksplit, stride, base + F + f);
  const float v = gt / (1.f + __expf(-gt)) * up;
  const f16 hi = static_cast<f16>(v);
  const long o = (long)r * F * hsplit + f;
  h[o] = hi;
  if (hsplit == 2) h[o + F] = static_cast<f16>(v - static_cast<float>(hi));
}

// Thread per (row, head slot, d < 64): rotary + stores of the pair (d, d + 64).
__global__ __launch_bounds__(256) void k_skinny_qkv(const float *__restrict__ part, int ksplit,
                                                    int rows, int n_heads, int n_kv,
                                                    QKVOut<f16> o) {
  const int nslots = n_heads + 2 * n_kv, N = nslots * 128;
  const long i = (long)blockIdx.x * 256 + threadIdx.x;
  if (i >= (long)rows * nslots * 64) return;
  const int r = (int)(i / (nslots * 64)), rem = (int)(i % (nslots * 64));
  const int slot = rem / 64, d = rem % 64;
  const long stride = (long)rows * N, base = (long)r * N + slot * 128 + d;
  const float x1 = sum_slices(part, ksplit, stride, base);
  const float x2 = sum_slices(part, ksplit, stride, base + 64);
  qkv_store(o, n_heads, n_kv, slot, r, d, x1, x2);
}

template <bool ARGMAX, int RG, int AS>
hipError_t launch_rg(const f16 *A, int rows, const void *W, bool w_f16, int N, int K, int ks,
                     float *part, hipStream_t s) {
  const dim3 grid(N / SK_ROWS, ks);
  const uint16_t *W16 = static_cast<const uint16_t *>(W);
  if (w_f16)
    k_skinny<RG, AS, false, ARGMAX><<<grid, 256, 0, s>>>(A, rows, W16, N, K, ks, part);
  else
    k_skinny<RG, AS, true, ARGMAX><<<grid, 256, 0, s>>>(A, rows, W16, N, K, ks, part);
  return hipGetLastError();
}

template <bool ARGMAX = false>
hipError_t launch(const f16 *A, int rows, int asplit, const void *W, bool w_f16, int N, int K,
                  int ks, float *part, hipStream_t s) {
  if (rows <= 16)
    return asplit == 2 ? launch_rg<ARGMAX, 1, 2>(A, rows, W, w_f16, N, K, ks, part, s)
                       : launch_rg<ARGMAX, 1, 1>(A, rows, W, w_f16, N, K, ks, part, s);
  return asplit == 2 ? launch_rg<ARGMAX, 2, 2>(A, rows, W, w_f16, N, K, ks, part, s)
                     : launch_rg<ARGMAX, 2, 1>(A, rows, W, w_f16, N, K, ks, part, s);
}

bool skinny_args_ok(int rows, int N, int K, int asplit) {
  return rows >= 1 && rows <= kSkinnyMaxRows && N % SK_ROWS == 0 && K % 32 == 0 && K > 0 &&
         (asplit == 1 || asplit == 2);
}

}  // namespace

int skinny_split(int N, int K) {
  const int blocks = std::max(1, N / SK_ROWS);
  const int by_k = (K + SK_STEP - 1) / SK_STEP;
  return std::min({by_k, std::max(1, (1024 + blocks - 1) / blocks), kSkinnyMaxSplit});
}

size_t skinny_part_floats(int rows, int N, int K) {
  return (size_t)skinny_split(N, K) * rows * N;
}

hipError_t skinny_residual(const f16 *A, int rows, int asplit, const void *W, bool w_f16, int N,
                           int K, float *x, const bf16 *g, float eps, f16 *y, int ysplit,
                           float *part, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  if (!skinny_args_ok(rows, N, K, asplit)) return hipErrorInvalidValue;
  const int ks = skinny_split(N, K);
  hipError_t e = launch(A, rows, asplit, W, w_f16, N, K, ks, part, s);
  if (e != hipSuccess) return e;
  k_skinny_residual<<<rows, 1024, 0, s>>>(part, ks, rows, N, x, g, eps, y, ysplit);
  return hipGetLastError();
}

hipError_t skinny_swiglu(const f16 *A, int rows, int asplit, const void *W, bool w_f16, int F,
                         int K, f16 *h, float *part, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  if (!skinny_args_ok(rows, 2 * F, K, asplit)) return hipErrorInvalidValue;
  const int ks = skinny_split(2 * F, K);
  hipError_t e = launch(A, rows, asplit, W, w_f16, 2 * F, K, ks, part, s);
  if (e != hipSuccess) return e;
  const long n = (long)rows * F;
  k_skinny_swiglu<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(part, ks, rows, F, asplit, h);
  return hipGetLastError();
}

hipError_t skinny_qkv_rope(const f16 *A, int rows, int asplit, const void *W, bool w_f16, int K,
                           int n_heads, int n_kv, const QKVOut<f16> &out, float *part,
                           hipStream_t s) {
  if (rows == 0) return hipSuccess;
  const int N = (n_heads + 2 * n_kv) * 128;
  if (!skinny_args_ok(rows, N, K, asplit)) return hipErrorInvalidValue;
  const int ks = skinny_split(N, K);
  hipError_t e = launch(A, rows, asplit, W, w_f16, N, K, ks, part, s);
  if (e != hipSuccess) return e;
  const long n = (long)rows * (n_heads + 2 * n_kv) * 64;
  k_skinny_qkv<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(part, ks, rows, n_heads, n_kv, out);
  return hipGetLastError();
}

int skinny_lm_chunks(int vocab) { return vocab % SK_ROWS ? 0 : vocab / SK_ROWS; }

hipError_t skinny_lmargmax(const f16 *A, int rows, const void *W, bool w_f16, int vocab, int K,
                           float2 *part, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  if (rows < 1 || rows > kSkinnyMaxRows || vocab % SK_ROWS || K % 32 || K <= 0)
    return hipErrorInvalidValue;
  return launch<true>(A, rows, 1, W, w_f16, vocab, K, 1, reinterpret_cast<float *>(part), s);
}

}  // namespace vsr
