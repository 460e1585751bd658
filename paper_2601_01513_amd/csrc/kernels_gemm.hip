// bf16 MFMA GEMMs of the verifier scoring pass with fused epilogues.
//
// Every GEMM here is C = A . B^T with A [rows][K] and B [N][K] both
// K-contiguous (activations and nn.Linear weights), fp32 accumulation on the
// gfx950 v_mfma_f32_32x32x16_f16 matrix cores. Activations are fp16; the bf16
// weight operand is converted to fp16 in registers on its way into LDS (exact:
// a bf16 value's 8 significant bits fit fp16's 11). A 256-thread block owns a
// BM x BN tile; its four waves form a WM x WN grid and each wave owns a
// (BM/WM) x (BN/WN) sub-tile of 32x32 MFMA blocks. K advances in steps of 64:
// the next A/B panels are fetched into registers while the MFMAs consume the
// current panels from LDS (16-byte chunks, XOR-swizzled by row so that both
// the panel stores and the fragment loads are free of bank conflicts).
//
// MFMA 32x32x16 (f16 and bf16 alike) lane layout (lane l, element e, accumulator register r):
//   A operand: A[i = l % 32][k = 8 (l / 32) + e]
//   B operand: B[k = 8 (l / 32) + e][j = l % 32]
//   result   : C[i = 8 (r / 4) + 4 (l / 32) + r % 4][j = l % 32]
// so each lane holds one output column and sixteen output rows; epilogues
// work directly on the registers.
#include "common.h"

namespace vsr {

constexpr int BK = 64;  // K elements per panel (8 chunks of 16 bytes per row)

template <int BM_, int BN_, int WM_, int WN_>
struct Tile {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_;
  static constexpr int TM = BM / WM, TN = BN / WN;  // wave sub-tile
  static constexpr int FM = TM / 32, FN = TN / 32;  // MFMA blocks per wave
  static constexpr int A_LOADS = BM * 8 / 256, B_LOADS = BN * 8 / 256;
  static constexpr int LDS_CHUNKS = (BM + BN) * 8;
  static_assert(WM * WN == 4, "four waves");
  static_assert(TM % 32 == 0 && TN % 32 == 0, "32x32 MFMA blocks");
};

__device__ __forceinline__ int swz(int row, int c) { return row * 8 + (c ^ (row & 7)); }

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
template <bool CVT>
__device__ __forceinline__ u32x4 stage(u32x4 v) {
  if constexpr (CVT) return bf16x8_to_f16x8(v);
  return v;
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

// Main loop: acc += A[m0 .. m0+BM) . B[rows given by brow(lr)]^T over all of K.
// A rows past `rows` are clamped to the last row (their results are never
// stored); brow must return an in-range B row for every lr < BN. CVT_A / CVT_B
// mark an operand stored as bf16 in memory (converted to fp16 when staged).
template <class TL, bool CVT_A, bool CVT_B, class BRow>
__device__ __forceinline__ void mainloop(const void *__restrict__ Av, int rows, int m0,
                                         const void *__restrict__ Bv, BRow brow, int K,
                                         u32x4 *lds, f32x16 (&acc)[TL::FM][TL::FN]) {
  const uint16_t *A = static_cast<const uint16_t *>(Av);
  const uint16_t *B = static_cast<const uint16_t *>(Bv);
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int wm = w / TL::WN, wn = w % TL::WN;
  u32x4 *As = lds;
  u32x4 *Bs = lds + TL::BM * 8;

  const u32x4 *ga[TL::A_LOADS];
  int la[TL::A_LOADS];
#pragma unroll
  for (int i = 0; i < TL::A_LOADS; ++i) {
    const int id = i * 256 + t, r = id >> 3, c = id & 7;
    const int gr = min(m0 + r, rows - 1);
    ga[i] = reinterpret_cast<const u32x4 *>(A + (long)gr * K) + c;
    la[i] = swz(r, c);
  }
  const u32x4 *gb[TL::B_LOADS];
  int lb[TL::B_LOADS];
#pragma unroll
  for (int i = 0; i < TL::B_LOADS; ++i) {
    const int id = i * 256 + t, r = id >> 3, c = id & 7;
    gb[i] = reinterpret_cast<const u32x4 *>(B + (long)brow(r) * K) + c;
    lb[i] = swz(r, c);
  }

#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < TL::FN; ++fn) acc[fm][fn] = f32x16{};

  u32x4 ra[TL::A_LOADS], rb[TL::B_LOADS];
  const int nk = K / BK;
#pragma unroll
  for (int i = 0; i < TL::A_LOADS; ++i) ra[i] = ga[i][0];
#pragma unroll
  for (int i = 0; i < TL::B_LOADS; ++i) rb[i] = gb[i][0];
#pragma unroll
  for (int i = 0; i < TL::A_LOADS; ++i) As[la[i]] = stage<CVT_A>(ra[i]);
#pragma unroll
  for (int i = 0; i < TL::B_LOADS; ++i) Bs[lb[i]] = stage<CVT_B>(rb[i]);
  __syncthreads();

  // Fragment rows of this lane.
  int fa[TL::FM], fb[TL::FN];
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm) fa[fm] = wm * TL::TM + fm * 32 + (lane & 31);
#pragma unroll
  for (int fn = 0; fn < TL::FN; ++fn) fb[fn] = wn * TL::TN + fn * 32 + (lane & 31);
  const int hc = lane >> 5;

  for (int kt = 0; kt < nk; ++kt) {
    const bool more = kt + 1 < nk;
    if (more) {
      const int off = (kt + 1) * (BK / 8);
#pragma unroll
      for (int i = 0; i < TL::A_LOADS; ++i) ra[i] = ga[i][off];
#pragma unroll
      for (int i = 0; i < TL::B_LOADS; ++i) rb[i] = gb[i][off];
    }
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int c = ks * 2 + hc;
      f16x8 af[TL::FM], bfr[TL::FN];
#pragma unroll
      for (int fm = 0; fm < TL::FM; ++fm) af[fm] = as_f16x8(As[swz(fa[fm], c)]);
#pragma unroll
      for (int fn = 0; fn < TL::FN; ++fn) bfr[fn] = as_f16x8(Bs[swz(fb[fn], c)]);
#pragma unroll
      for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < TL::FN; ++fn)
          acc[fm][fn] =
              __builtin_amdgcn_mfma_f32_32x32x16_f16(af[fm], bfr[fn], acc[fm][fn], 0, 0, 0);
    }
    __syncthreads();
    if (more) {
#pragma unroll
      for (int i = 0; i < TL::A_LOADS; ++i) As[la[i]] = stage<CVT_A>(ra[i]);
#pragma unroll
      for (int i = 0; i < TL::B_LOADS; ++i) Bs[lb[i]] = stage<CVT_B>(rb[i]);
      __syncthreads();
    }
  }
}

// The tile used by every GEMM of the pass: 128 x 256, waves 2 x 2 (64 x 128).
// A wave's 128 columns hold a whole attention head (QKV) or 64 gate + 64 up
// columns (SwiGLU), so the rotary pairs and the gate/up pairs sit in the same
// lane and register.
typedef Tile<128, 256, 2, 2> TileStd;

// ------------------------------------------------------- residual (O, down)
template <class TL>
__global__ __launch_bounds__(256) void k_gemm_residual(const f16 *__restrict__ A,
                                                       const bf16 *__restrict__ W, int rows,
                                                       int N, int K, float *__restrict__ x) {
  __shared__ u32x4 lds[TL::LDS_CHUNKS];
  const int n0 = blockIdx.x * TL::BN, m0 = blockIdx.y * TL::BM;
  f32x16 acc[TL::FM][TL::FN];
  mainloop<TL, false, true>(A, rows, m0, W, [=](int r) { return min(n0 + r, N - 1); }, K, lds,
                            acc);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w / TL::WN, wn = w % TL::WN;
#pragma unroll
  for (int fn = 0; fn < TL::FN; ++fn) {
    const int col = n0 + acc_col<TL>(wn, fn, lane);
    if (col >= N) continue;
#pragma unroll
    for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + acc_row<TL>(wm, fm, r, lane);
        if (row < rows) x[(long)row * N + col] += acc[fm][fn][r];
      }
  }
}

hipError_t gemm_residual(const f16 *A, const bf16 *W, int rows, int N, int K, float *x,
                         hipStream_t s) {
  if (rows == 0) return hipSuccess;
  typedef TileStd TL;
  dim3 grid((N + TL::BN - 1) / TL::BN, (rows + TL::BM - 1) / TL::BM);
  k_gemm_residual<TL><<<grid, 256, 0, s>>>(A, W, rows, N, K, x);
  return hipGetLastError();
}

// ------------------------------------------------------------------- SwiGLU
// Block column tile o0 .. o0+128 of the FFN hidden. Its 256 B rows are laid
// out per wave: wave wn takes gate rows o0+64wn .. +63 then the matching up
// rows, so MFMA blocks fn and fn+2 of a wave hold gate and up of the same
// output columns.
template <class TL>
__global__ __launch_bounds__(256) void k_gemm_swiglu(const f16 *__restrict__ A,
                                                     const bf16 *__restrict__ W, int rows,
                                                     int F, int K, f16 *__restrict__ h) {
  static_assert(TL::WN == 2 && TL::TN == 128, "gate/up pairing needs 128-column waves");
  __shared__ u32x4 lds[TL::LDS_CHUNKS];
  const int o0 = blockIdx.x * 128, m0 = blockIdx.y * TL::BM;
  f32x16 acc[TL::FM][TL::FN];
  mainloop<TL, false, true>(A, rows, m0, W,
               [=](int r) {
                 const int q = r & 127;
                 const int oc = min(o0 + (r >> 7) * 64 + (q & 63), F - 1);
                 return q < 64 ? oc : F + oc;
               },
               K, lds, acc);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w / TL::WN, wn = w % TL::WN;
#pragma unroll
  for (int fn = 0; fn < 2; ++fn) {
    const int col = o0 + wn * 64 + fn * 32 + (lane & 31);
    if (col >= F) continue;
#pragma unroll
    for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = m0 + acc_row<TL>(wm, fm, r, lane);
        if (row >= rows) continue;
        const float g = acc[fm][fn][r], u = acc[fm][fn + 2][r];
        h[(long)row * F + col] = static_cast<f16>(g / (1.f + __expf(-g)) * u);
      }
  }
}

hipError_t gemm_swiglu(const f16 *A, const bf16 *W, int rows, int F, int K, f16 *h,
                       hipStream_t s) {
  if (rows == 0) return hipSuccess;
  typedef TileStd TL;
  dim3 grid((F + 127) / 128, (rows + TL::BM - 1) / TL::BM);
  k_gemm_swiglu<TL><<<grid, 256, 0, s>>>(A, W, rows, F, K, h);
  return hipGetLastError();
}

// ------------------------------------------------- QKV + rotary + KV caches
// Block column tile = two heads of the stacked q|k|v projection; wave wn owns
// head slot 2 blockIdx.x + wn. MFMA blocks fn and fn+2 hold head dims d and
// d + 64, the rotate-half pair.
template <class TL>
__global__ __launch_bounds__(256) void k_gemm_qkv(const f16 *__restrict__ A,
                                                  const bf16 *__restrict__ W, int rows, int K,
                                                  int n_heads, int n_kv, QKVOut<f16> o) {
  static_assert(TL::WN == 2 && TL::TN == 128, "one head per wave");
  __shared__ u32x4 lds[TL::LDS_CHUNKS];
  const int nslots = n_heads + 2 * n_kv;
  const int n0 = blockIdx.x * 256, m0 = blockIdx.y * TL::BM;
  const int nrows = nslots * 128;
  f32x16 acc[TL::FM][TL::FN];
  mainloop<TL, false, true>(A, rows, m0, W, [=](int r) { return min(n0 + r, nrows - 1); }, K,
                            lds, acc);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w / TL::WN, wn = w % TL::WN;
  const int slot = blockIdx.x * 2 + wn;
  if (slot >= nslots) return;
  const bool rot = slot < n_heads + n_kv;
#pragma unroll
  for (int fm = 0; fm < TL::FM; ++fm)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = m0 + acc_row<TL>(wm, fm, r, lane);
      if (row >= rows) continue;
      const int pos = o.row_pos ? o.row_pos[row] : row;
#pragma unroll
      for (int fn = 0; fn < 2; ++fn) {
        const int d = fn * 32 + (lane & 31);
        float x1 = acc[fm][fn][r], x2 = acc[fm][fn + 2][r];
        if (rot) {
          const float2 cs = o.rope[(long)pos * 64 + d];
          const float y1 = x1 * cs.x - x2 * cs.y, y2 = x2 * cs.x + x1 * cs.y;
          x1 = y1;
          x2 = y2;
        }
        if (slot < n_heads) {
          f16 *q = o.q + ((long)row * n_heads + slot) * 128;
          q[d] = static_cast<f16>(x1);
          q[d + 64] = static_cast<f16>(x2);
        } else if (rot) {
          f16 *k = o.k + ((long)(slot - n_heads) * o.kv_npos + row) * 128;
          k[d] = static_cast<f16>(x1);
          k[d + 64] = static_cast<f16>(x2);
        } else {
          f16 *vt = o.vt + (long)(slot - n_heads - n_kv) * 128 * o.kv_npos;
          vt[(long)d * o.kv_npos + row] = static_cast<f16>(x1);
          vt[(long)(d + 64) * o.kv_npos + row] = static_cast<f16>(x2);
        }
      }
    }
}

hipError_t gemm_qkv_rope(const f16 *A, const bf16 *W, int rows, int K, int n_heads, int n_kv,
                         const QKVOut<f16> &out, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  typedef TileStd TL;
  const int nslots = n_heads + 2 * n_kv;
  dim3 grid((nslots + 1) / 2, (rows + TL::BM - 1) / TL::BM);
  k_gemm_qkv<TL><<<grid, 256, 0, s>>>(A, W, rows, K, n_heads, n_kv, out);
  return hipGetLastError();
}

// ------------------------------------------------------ LM head + chunk LSE
// Transposed product: the MFMA rows are vocabulary entries (A = W_lm) and the
// columns are scored tokens (B = normed hidden rows), so a token's reduction
// over the vocabulary runs down a lane's registers, across the two lane
// halves and across the WM waves. Block (vocab tile c, token tile) writes, for
// each token t, part[c][t] = (max_v l, sum_v exp(l - max)) over its BM
// vocabulary rows, and the target logit when the target falls in the tile.
// The [tokens x vocab] logits never leave registers.
template <class TL>
__global__ __launch_bounds__(256) void k_gemm_lmhead(const f16 *__restrict__ Hn,
                                                     const bf16 *__restrict__ Wlm, int T,
                                                     int vocab, int K,
                                                     const int32_t *__restrict__ lm_tgt,
                                                     float2 *__restrict__ part,
                                                     float *__restrict__ tgt_logit) {
  __shared__ u32x4 lds[TL::LDS_CHUNKS];
  __shared__ float red[TL::WM][TL::BN];
  const int n0 = blockIdx.x * TL::BN, m0 = blockIdx.y * TL::BM;
  f32x16 acc[TL::FM][TL::FN];
  mainloop<TL, true, false>(Wlm, vocab, m0, Hn, [=](int r) { return min(n0 + r, T - 1); }, K,
                            lds, acc);
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
      part[(long)blockIdx.y * T + t] = make_float2(mx[fn], s);
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

int lmhead_chunks(int vocab) { return (vocab + TileStd::BM - 1) / TileStd::BM; }

hipError_t gemm_lmhead(const f16 *A, const bf16 *W, int rows, int vocab, int K,
                       const int32_t *lm_tgt, float2 *part, float *tgt_logit, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  typedef TileStd TL;
  dim3 grid((rows + TL::BN - 1) / TL::BN, lmhead_chunks(vocab));
  k_gemm_lmhead<TL><<<grid, 256, 0, s>>>(A, W, rows, vocab, K, lm_tgt, part, tgt_logit);
  return hipGetLastError();
}

}  // namespace vsr
