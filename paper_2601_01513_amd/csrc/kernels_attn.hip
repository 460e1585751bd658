// Attention of the verifier scoring pass on the gfx950 matrix cores.
//
// One kernel serves the prefix prefill (causal) and the candidate pass
// (cascade: the shared prefix keys, then each candidate's own causal block).
// For KV head h the query rows of all G = n_heads / n_kv query heads that read
// it are stacked, row r = (token r / G, head h G + r % G), so every key tile
// staged in LDS is used by all of them -- and, in the candidate pass, by all
// M candidates at once: the prefix keys are read once per query tile, not
// once per candidate.
//
// A 256-thread block owns 128 stacked query rows (32 per wave) and walks 64-key
// tiles. Each wave computes S^T = K . Q^T on MFMA 32x32x16 (keys as MFMA rows,
// queries as columns), so a lane owns one query's scores and every per-query
// softmax quantity is a per-lane scalar. The probabilities feed O^T += V^T . P^T
// straight from registers: the k-index of that product is permuted to match
// the key order the S^T accumulator leaves in each lane, and V^T is staged
// with the same permutation (the Vt cache stores values position-contiguous).
// Softmax runs online in the log2 domain in fp32; P is rounded to fp16 for the
// PV product.
//
// The candidate pass may split the prefix keys into chunks (more blocks on the
// chip); each chunk writes (max, sum, unnormalised output) partials and
// attn_merge combines them.
#include "common.h"

namespace vsr {

namespace {

constexpr int HD = 128;   // head dim of the MFMA path
constexpr int QT = 128;   // stacked query rows per block
constexpr int KT = 64;    // keys per tile

__device__ __forceinline__ f16x8 as_f16x8(u32x4 v) { return __builtin_bit_cast(f16x8, v); }

// K tile [64 keys][128 dims]: 16 chunks per key, XOR-swizzled by key.
__device__ __forceinline__ int ks_idx(int key, int c) { return key * 16 + (c ^ (key & 7)); }
// V^T tile [128 dims][64 keys]: 8 chunks per dim row, XOR-swizzled by row;
// rows with bit 3 set store their two 8-byte halves swapped so that the
// 8-byte fragment reads of 16 consecutive rows hit distinct banks.
__device__ __forceinline__ int vs_idx(int d, int c) { return d * 8 + (c ^ (d & 7)); }

// Key visibility of one key segment.
enum SegMode { SEG_ALL = 0, SEG_CAUSAL = 1, SEG_BRANCH = 2 };

struct Seg {
  const f16 *k;    // [npos][HD] of this KV head
  const f16 *vt;   // [HD][npos] of this KV head
  int npos;        // position stride of vt
  int kvalid;      // keys >= kvalid hold no data (never visible)
  int kbeg, kend;  // key range walked by the block: [kbeg, kend), kbeg % 64 == 0
  int mode;
};

struct Lane {
  int tok;   // query token of this lane's row
  int lo;    // SEG_BRANCH: first visible key
  float m, l;
  f32x16 o[HD / 32];
  f16x8 q[HD / 16];
};

__device__ __forceinline__ void load_tile(const Seg &sg, int kb, u32x4 (&rk)[4], u32x4 (&rv)[4]) {
  const int t = threadIdx.x;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int id = i * 256 + t;
    const int key = id >> 4, c = id & 15;
    rk[i] = reinterpret_cast<const u32x4 *>(sg.k + (long)(kb + key) * HD)[c];
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int id = i * 256 + t;
    const int d = id >> 3, c = id & 7;
    const int k0 = kb + c * 8;
    u32x4 v = reinterpret_cast<const u32x4 *>(sg.vt + (long)d * sg.npos + k0)[0];
    if (k0 + 8 > sg.kvalid) {  // zero values past the written keys (P = 0 there)
      uint32_t *e = reinterpret_cast<uint32_t *>(&v);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t lo = (k0 + 2 * j < sg.kvalid) ? 0x0000FFFFu : 0u;
        const uint32_t hi = (k0 + 2 * j + 1 < sg.kvalid) ? 0xFFFF0000u : 0u;
        e[j] &= (lo | hi);
      }
    }
    rv[i] = v;
  }
}

__device__ __forceinline__ void store_tile(u32x4 *Ks, u32x4 *Vs, const u32x4 (&rk)[4],
                                           const u32x4 (&rv)[4]) {
  const int t = threadIdx.x;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int id = i * 256 + t;
    Ks[ks_idx(id >> 4, id & 15)] = rk[i];
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int id = i * 256 + t;
    const int d = id >> 3;
    u32x4 v = rv[i];
    if (d & 8) v = u32x4{v.z, v.w, v.x, v.y};
    Vs[vs_idx(d, id & 7)] = v;
  }
}

// One 64-key tile against this wave's 32 query rows.
__device__ __forceinline__ void tile_step(const Seg &sg, int kb, const u32x4 *Ks,
                                          const u32x4 *Vs, Lane &L, float scale_log2) {
  const int lane = threadIdx.x & 63, h = lane >> 5;
  f32x16 s[2];
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    s[b] = f32x16{};
    const int key = b * 32 + (lane & 31);
#pragma unroll
    for (int kk = 0; kk < HD / 16; ++kk)
      s[b] = __builtin_amdgcn_mfma_f32_32x32x16_f16(as_f16x8(Ks[ks_idx(key, 2 * kk + h)]),
                                                     L.q[kk], s[b], 0, 0, 0);
  }
  // Mask and scale; key of register r of block b: kb + 32b + 8(r/4) + 4h + r%4.
  float mloc = -INFINITY;
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = kb + b * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
      bool vis = key < sg.kvalid;
      if (sg.mode == SEG_CAUSAL) vis = vis && key <= L.tok;
      if (sg.mode == SEG_BRANCH) vis = vis && key >= L.lo && key <= L.tok;
      const float v = vis ? s[b][r] * scale_log2 : -INFINITY;
      s[b][r] = v;
      mloc = fmaxf(mloc, v);
    }
  mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
  const float mnew = fmaxf(L.m, mloc);
  const float mref = mnew == -INFINITY ? 0.f : mnew;
  const float alpha = exp2f(L.m - mref);
  float psum = 0.f;
  f16x8 p[4];
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float e = exp2f(s[b][r] - mref);
      psum += e;
      p[b * 2 + (r >> 3)][r & 7] = static_cast<f16>(e);
    }
  psum += __shfl_xor(psum, 32, 64);
  L.l = L.l * alpha + psum;
  L.m = mnew;
#pragma unroll
  for (int db = 0; db < HD / 32; ++db) L.o[db] *= alpha;
  // O^T[d][q] += V^T[d][key] P^T[key][q]; for 16-key chunk c the MFMA k-index
  // 8h' + e of lane half h' is key 16c + 8(e/4) + 4h' + e%4.
#pragma unroll
  for (int c = 0; c < 4; ++c) {
#pragma unroll
    for (int db = 0; db < HD / 32; ++db) {
      const int d = db * 32 + (lane & 31);
      const int sw = (d >> 3) & 1;  // halves swapped on this row
      const uint64_t *r0 =
          reinterpret_cast<const uint64_t *>(&Vs[vs_idx(d, 2 * c)]) + (h ^ sw);
      const uint64_t *r1 =
          reinterpret_cast<const uint64_t *>(&Vs[vs_idx(d, 2 * c + 1)]) + (h ^ sw);
      uint64_t v2[2] = {*r0, *r1};
      const f16x8 va = __builtin_bit_cast(f16x8, v2);
      L.o[db] = __builtin_amdgcn_mfma_f32_32x32x16_f16(va, p[c], L.o[db], 0, 0, 0);
    }
  }
}

__device__ __forceinline__ void walk_segment(const Seg &sg, u32x4 *Ks, u32x4 *Vs, Lane &L, float scale_log2) {
  if (sg.kend <= sg.kbeg) return;
  u32x4 rk[4], rv[4];
  load_tile(sg, sg.kbeg, rk, rv);
  store_tile(Ks, Vs, rk, rv);
  __syncthreads();
  for (int kb = sg.kbeg; kb < sg.kend; kb += KT) {
    const bool more = kb + KT < sg.kend;
    if (more) load_tile(sg, kb + KT, rk, rv);
    tile_step(sg, kb, Ks, Vs, L, scale_log2);
    __syncthreads();
    if (more) {
      store_tile(Ks, Vs, rk, rv);
      __syncthreads();
    }
  }
}

// mode 0: prefill (causal over the prefix cache, one chunk, direct output);
// mode 1: candidate pass (prefix chunk blockIdx.z; the last chunk also walks
//         the candidate's own keys).
template <int MODE>
__global__ __launch_bounds__(256) void k_attn(AttnArgs a) {
  __shared__ u32x4 Ks[KT * 16];
  __shared__ u32x4 Vs[HD * 8];
  const int G = a.n_heads / a.n_kv, TG = a.T * G;
  const int kvh = blockIdx.y;
  // Prefill tiles with more keys first.
  const int qt = MODE == 0 ? gridDim.x - 1 - blockIdx.x : blockIdx.x;
  const int q0 = qt * QT;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int row = q0 + w * 32 + (lane & 31);
  const int rowc = min(row, TG - 1);

  Lane L;
  L.tok = rowc / G;
  const int head = kvh * G + rowc % G;
  L.lo = MODE == 1 ? a.row_lo[L.tok] : 0;
  L.m = -INFINITY;
  L.l = 0.f;
#pragma unroll
  for (int db = 0; db < HD / 32; ++db) L.o[db] = f32x16{};
  {
    const u32x4 *qp = reinterpret_cast<const u32x4 *>(a.q + ((long)L.tok * a.n_heads + head) * HD);
#pragma unroll
    for (int kk = 0; kk < HD / 16; ++kk) L.q[kk] = as_f16x8(qp[2 * kk + (lane >> 5)]);
  }
  const float scale_log2 = 1.4426950408889634f * rsqrtf((float)HD);
  const int tok_last = min(q0 + QT - 1, TG - 1) / G;

  const int chunk = blockIdx.z;
  if (MODE == 0) {
    Seg sg{a.k + (long)kvh * a.kv_npos * HD, a.vt + (long)kvh * HD * a.kv_npos, a.kv_npos,
           a.T, 0, tok_last + 1, SEG_CAUSAL};
    walk_segment(sg, Ks, Vs, L, scale_log2);
  } else {
    const int kb = chunk * a.chunk, ke = min(a.P, kb + a.chunk);
    Seg sp{a.k + (long)kvh * a.kv_npos * HD, a.vt + (long)kvh * HD * a.kv_npos, a.kv_npos,
           a.P, kb, ke, SEG_ALL};
    walk_segment(sp, Ks, Vs, L, scale_log2);
    if (chunk == a.nchunks - 1) {
      const int tok_first = q0 / G;
      const int lo = a.row_lo[tok_first] & ~(KT - 1);
      Seg sb{a.bk + (long)kvh * a.bk_npos * HD, a.bvt + (long)kvh * HD * a.bk_npos, a.bk_npos,
             a.T, lo, tok_last + 1, SEG_BRANCH};
      walk_segment(sb, Ks, Vs, L, scale_log2);
    }
  }

  if (row >= TG) return;
  const int h = lane >> 5;
  if (MODE == 0 || a.nchunks == 1) {
    const float inv = 1.f / L.l;
    f16 *op = a.out + ((long)L.tok * a.n_heads + head) * HD;
#pragma unroll
    for (int db = 0; db < HD / 32; ++db)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        f16x4 v;
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = static_cast<f16>(L.o[db][g4 * 4 + j] * inv);
        *reinterpret_cast<f16x4 *>(op + db * 32 + 8 * g4 + 4 * h) = v;
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
    if (h == 0) a.part_ml[prow] = make_float2(L.m, L.l);
  }
}

// One wave per (token, query head): combine the chunk partials.
__global__ __launch_bounds__(64) void k_attn_merge(AttnArgs a) {
  const int t = blockIdx.x, head = blockIdx.y, lane = threadIdx.x;
  const int G = a.n_heads / a.n_kv, TG = a.T * G;
  const int kvh = head / G, row = t * G + head % G;
  float M = -INFINITY;
  for (int c = 0; c < a.nchunks; ++c)
    M = fmaxf(M, a.part_ml[((long)c * a.n_kv + kvh) * TG + row].x);
  float Lsum = 0.f, o0 = 0.f, o1 = 0.f;
  for (int c = 0; c < a.nchunks; ++c) {
    const long prow = ((long)c * a.n_kv + kvh) * TG + row;
    const float2 ml = a.part_ml[prow];
    const float wgt = ml.x == -INFINITY ? 0.f : exp2f(ml.x - M);
    Lsum += ml.y * wgt;
    o0 += a.part_acc[prow * HD + lane] * wgt;
    o1 += a.part_acc[prow * HD + 64 + lane] * wgt;
  }
  const float inv = 1.f / Lsum;
  f16 *op = a.out + ((long)t * a.n_heads + head) * HD;
  op[lane] = static_cast<f16>(o0 * inv);
  op[64 + lane] = static_cast<f16>(o1 * inv);
}

}  // namespace

hipError_t attn_prefill(const AttnArgs &a, hipStream_t s) {
  if (a.T == 0) return hipSuccess;
  const int G = a.n_heads / a.n_kv;
  dim3 grid((a.T * G + QT - 1) / QT, a.n_kv, 1);
  k_attn<0><<<grid, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t attn_cascade(const AttnArgs &a, hipStream_t s) {
  if (a.T == 0) return hipSuccess;
  const int G = a.n_heads / a.n_kv;
  dim3 grid((a.T * G + QT - 1) / QT, a.n_kv, a.nchunks);
  k_attn<1><<<grid, 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t attn_merge(const AttnArgs &a, hipStream_t s) {
  if (a.T == 0 || a.nchunks == 1) return hipSuccess;
  k_attn_merge<<<dim3(a.T, a.n_heads), 64, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace vsr
