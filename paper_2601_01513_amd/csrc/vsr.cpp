// Host side of the C ABI (include/vsr.h): argument checks, workspace plan and
// the launch sequence of the verifier scoring pass (Section 3.1, Eq. 6-7).
//
// Every argument check runs before any HIP call, so misuse is reported
// without touching the device. The workspace plan is pure host arithmetic.
#include "vsr.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <type_traits>
#include <vector>

#include "common.h"

using namespace vsr;

namespace {

thread_local std::string g_create_error;

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Key split of the candidate pass: at most one round of blocks on the chip,
// at least 256 of a block's `keys` (prefix + branch keys it walks) per chunk; a pass
// with one query tile per KV head (decode steps) is latency-bound and takes
// chunks of one 64-key tile. At most 64 chunks (the merge's limit).
struct Split {
  int nchunks;
};
Split cascade_split(int T, int keys, int n_heads, int n_kv) {
  const int G = n_heads / n_kv;
  const int qt = attn_query_tile();
  const int qtiles = (T * G + qt - 1) / qt * n_kv;
  // One round of the 256 CUs (a block per CU): more chunks add a round, and
  // partials for the merge to read, sooner than they shorten the blocks.
  int n = std::max(1, 256 / qtiles);
  n = std::min(n, std::max(1, keys / (qtiles == n_kv ? 64 : 256)));
  return {std::min(n, 64)};
}

struct Plan {
  int kv_npos, bk_npos, max_t, rows_max, rope_npos, lm_chunks;
  int dec_S, dec_npos;  // draft cache: positions per branch, capacity (0: none)
  int lm_rows;  // LM-head rows: candidate rows, or 2 per branch (reliability)
  size_t x, xn, q, q_lo, attn, h, kc, vtc, kc_lo, vtc_lo, bk, bvt, bk_lo, bvt_lo, kd, vtd,
      kd_lo, vtd_lo, part_acc, part_ml, lm_part, tgt, row_lo, row_pos, cache_row, dec_ids,
      lm_tgt, rope, h_last, gemm_part, flags, total;
};

// Returns an empty message if cfg is supported.
std::string check_config(const vsr_config *c) {
  if (!c) return "config is NULL";
  if (c->n_layers < 0 || c->d_model <= 0 || c->n_heads <= 0 || c->n_kv_heads <= 0 ||
      c->head_dim <= 0 || c->d_ff <= 0 || c->vocab <= 0)
    return "config sizes must be positive (n_layers >= 0)";
  if (c->n_heads % c->n_kv_heads) return "n_heads must be a multiple of n_kv_heads";
  if (!(c->rms_eps >= 0.f) || !(c->rope_base > 0.f)) return "rms_eps >= 0 and rope_base > 0 needed";
  if (c->max_prefix < 1 || c->max_cands < 1 || c->max_cand_len < 1)
    return "max_prefix, max_cands and max_cand_len must be >= 1";
  if (c->max_cands > VSR_MAX_CANDS) return "max_cands exceeds VSR_MAX_CANDS";
  if ((long long)c->max_cands * c->max_cand_len > (1 << 24)) return "max_cands * max_cand_len too large";
  if (c->max_prefix > (1 << 24)) return "max_prefix too large";
  if (c->split_layers < 0 || c->split_layers > c->n_layers)
    return "split_layers must be in [0, n_layers]";
  if (c->split_mlp_layers < 0 || c->split_mlp_layers > c->split_layers)
    return "split_mlp_layers must be in [0, split_layers]";
  if (c->max_new < 0 || c->max_new > 4096) return "max_new must be in [0, 4096]";
  if (c->dtype == VSR_BF16 ? (c->gemm_weights != 0 && c->gemm_weights != VSR_BF16 &&
                              c->gemm_weights != VSR_F16)
                           : c->gemm_weights != 0)
    return "gemm_weights must be 0, VSR_BF16 or VSR_F16 (bf16 contexts), 0 otherwise";
  if (c->dtype == VSR_BF16) {
    if (c->head_dim != 128) return "bf16 contexts need head_dim == 128";
    if (c->d_model % 64 || c->d_ff % 64) return "bf16 contexts need d_model and d_ff multiples of 64";
  } else if (c->dtype == VSR_F32) {
    if (c->head_dim % 2 || c->head_dim > 256) return "fp32 contexts need an even head_dim <= 256";
  } else {
    return "dtype must be VSR_F32 or VSR_BF16";
  }
  return "";
}

Plan make_plan(const vsr_config &c) {
  Plan p{};
  const size_t E = c.dtype == VSR_BF16 ? 2 : 4;
  const int G = c.n_heads / c.n_kv_heads;
  const size_t d = c.d_model, hd = c.head_dim;
  p.kv_npos = (int)align_up(c.max_prefix, 64);
  p.max_t = c.max_cands * c.max_cand_len;
  p.bk_npos = (int)align_up(p.max_t, 64);
  p.lm_rows = std::max(p.max_t, 2 * c.max_cands);
  // MFMA contexts run the prefix and the candidate rows of vsr_verify as one
  // set of rows.
  p.rows_max = std::max(c.max_prefix + (c.dtype == VSR_BF16 ? p.max_t : 0), p.lm_rows);
  p.dec_S = c.max_new > 0 ? c.max_cand_len + c.max_new : 0;
  p.dec_npos = c.max_new > 0 ? (int)align_up((size_t)c.max_cands * p.dec_S, 64) : 0;
  p.rope_npos = p.kv_npos + c.max_cand_len + c.max_new;
  p.lm_chunks = c.dtype == VSR_BF16 ? lmhead_chunks(c.vocab) : 1;
  // Largest partial-row count of the cascade split over every T <= max_t
  // (the split grows with the keys a block walks, at most the whole prefix
  // plus the largest branch span: a candidate, or every draft branch).
  size_t part_rows = 0;
  if (c.dtype == VSR_BF16) {
    const int keys_max = c.max_prefix + std::max(c.max_cand_len, p.dec_npos);
    for (int T = 1; T <= p.max_t; ++T) {
      const Split s = cascade_split(T, keys_max, c.n_heads, c.n_kv_heads);
      if (s.nchunks > 1) part_rows = std::max(part_rows, (size_t)s.nchunks * T * G);
    }
    // Prefill with split keys: the split only changes where the query-tile
    // count does, so the largest prefix of each tile count bounds it.
    const int qt = attn_query_tile();
    for (int tiles = 1;; ++tiles) {
      const int T = std::min(c.max_prefix, (tiles * qt) / G);
      if (T >= 1) {
        const int n = prefill_chunks(T, c.n_heads, c.n_kv_heads);
        if (n > 1) part_rows = std::max(part_rows, (size_t)n * T * G);
      }
      if (T >= c.max_prefix) break;
    }
  }
  // Split-K partials of the MFMA GEMMs: the largest need over every row count
  // (the split only changes where the 256-row tile count does).
  size_t gemm_part = 0;
  if (c.dtype == VSR_BF16) {
    const int qkv_n = (c.n_heads + 2 * c.n_kv_heads) * c.head_dim;
    for (int r = 256;; r += 256) {
      const int rows = std::min(r, p.rows_max);
      for (int s = 1; s <= (c.split_layers > 0 ? 2 : 1); ++s)
        gemm_part = std::max({gemm_part, gemm_split_floats(rows, qkv_n, s * c.d_model),
                              gemm_split_floats(rows, c.d_model, s * c.n_heads * c.head_dim),
                              gemm_split_floats(rows, 2 * c.d_ff, s * c.d_model),
                              gemm_split_floats(rows, c.d_model, s * c.d_ff)});
      if (rows == p.rows_max) break;
    }
    // Few-row products (at most kSkinnyMaxRows rows).
    const int sr = std::min(p.rows_max, kSkinnyMaxRows);
    gemm_part = std::max({gemm_part, skinny_part_floats(sr, qkv_n, c.d_model),
                          skinny_part_floats(sr, c.d_model, c.n_heads * c.head_dim),
                          skinny_part_floats(sr, 2 * c.d_ff, c.d_model),
                          skinny_part_floats(sr, c.d_model, c.d_ff)});
  }
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_up(off + bytes, 256);
    return o;
  };
  const size_t R = p.rows_max;
  // Precise layers (the first split_layers of the MFMA path) carry GEMM rows
  // as [hi | lo] and q, k, v as value + remainder planes.
  const size_t sp = (c.dtype == VSR_BF16 && c.split_layers > 0) ? 2 : 1;
  const size_t nprec = c.dtype == VSR_BF16 ? c.split_layers : 0;
  const size_t prefix_cache = (size_t)c.n_kv_heads * p.kv_npos * hd * E;
  const size_t branch_cache = (size_t)c.n_kv_heads * p.bk_npos * hd * E;
  p.x = take(R * d * 4);
  p.xn = take(R * d * E * sp);
  p.q = take(R * c.n_heads * hd * E);
  p.q_lo = take(nprec ? R * c.n_heads * hd * E : 0);
  p.attn = take(R * c.n_heads * hd * E * sp);
  p.h = take(R * (size_t)c.d_ff * E * sp);
  // Caches (kc .. part_acc) start zeroed at create.
  p.kc = take(c.n_layers * prefix_cache);
  p.vtc = take(c.n_layers * prefix_cache);
  p.kc_lo = take(nprec * prefix_cache);
  p.vtc_lo = take(nprec * prefix_cache);
  p.bk = take(branch_cache);
  p.bvt = take(branch_cache);
  p.bk_lo = take(nprec ? branch_cache : 0);
  p.bvt_lo = take(nprec ? branch_cache : 0);
  // Draft cache: every layer's keys / values of the branches being decoded.
  const size_t dec_cache = (size_t)c.n_kv_heads * p.dec_npos * hd * E;
  p.kd = take(c.n_layers * dec_cache);
  p.vtd = take(c.n_layers * dec_cache);
  p.kd_lo = take(nprec * dec_cache);
  p.vtd_lo = take(nprec * dec_cache);
  p.part_acc = take(part_rows * c.n_kv_heads * hd * 4);
  p.part_ml = take(part_rows * c.n_kv_heads * 8);
  // LM-head partials: vocabulary tiles x rows, or (greedy drafts of few
  // branches) 64-entry chunks x branches.
  p.lm_part = take(std::max((size_t)p.lm_chunks * p.lm_rows,
                            c.dtype == VSR_BF16 ? (size_t)skinny_lm_chunks(c.vocab) *
                                                      std::min(c.max_cands, kSkinnyMaxRows)
                                                : 0) *
                   8);
  p.tgt = take((size_t)p.lm_rows * 4);
  p.row_lo = take((size_t)p.max_t * 4);
  p.row_pos = take((size_t)p.max_t * 4);
  p.cache_row = take((size_t)p.max_t * 4);
  p.dec_ids = take((size_t)c.max_cands * 4);
  p.lm_tgt = take((size_t)p.lm_rows * 4);
  p.rope = take((size_t)p.rope_npos * (hd / 2) * 8);
  p.h_last = take(d * 4);
  p.gemm_part = take(gemm_part * 4);
  p.flags = take(64);
  p.total = off;
  return p;
}

}  // namespace

struct vsr_ctx {
  vsr_config cfg;
  Plan plan;
  char *ws;
  hipStream_t stream;
  int device;
  bool have_weights = false;
  bool prefilled = false;
  int checks = 0;  // VSR_CHECK_* bits of vsr_set_checks
  int P = 0;
  const void *embed = nullptr, *lm_head = nullptr, *final_norm = nullptr;
  std::vector<const void *> attn_norm, wqkv, wo, ffn_norm, wgu, wdown;
  std::string err;

  // Stage timing (vsr_profile_*): event pairs recorded around each launch.
  struct Rec {
    int stage;
    hipEvent_t a, b;
  };
  int prof = 0;  // bitmask of the stage kinds being timed
  int phase = 0;  // 0 prefix pass, 1 candidate pass, 2 draft pass, 3 fused verify pass
  std::vector<Rec> recs;
  std::vector<hipEvent_t> pool;
  hipEvent_t event() {
    if (!pool.empty()) {
      hipEvent_t e = pool.back();
      pool.pop_back();
      return e;
    }
    hipEvent_t e = nullptr;
    return hipEventCreate(&e) == hipSuccess ? e : nullptr;
  }
  void drop_records() {
    for (auto &r : recs) {
      pool.push_back(r.a);
      pool.push_back(r.b);
    }
    recs.clear();
  }
  ~vsr_ctx() {
    drop_records();
    for (hipEvent_t e : pool) (void)hipEventDestroy(e);
  }

  template <typename T>
  T *at(size_t off) const {
    return reinterpret_cast<T *>(ws + off);
  }
  int fail(int code, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    err = buf;
    return code;
  }
};

#define HIPCHECK(ctx, stage, expr)                                                        \
  do {                                                                                    \
    hipError_t e_ = (expr);                                                               \
    if (e_ != hipSuccess)                                                                 \
      return (ctx)->fail(VSR_EHIP, "HIP error in %s: %s", stage, hipGetErrorString(e_)); \
  } while (0)

enum StageKind {
  K_EMBED = 0, K_NORM, K_QKV, K_ATTN, K_MERGE, K_OPROJ, K_GATEUP, K_DOWN, K_LMIN, K_LMHEAD,
  K_LSE, K_SELECT, K_ROWS, K_COPY, K_TAIL, K_CATTN
};
static_assert(K_CATTN + 1 == VSR_STAGE_KINDS, "stage kinds");

// Launch the expression as stage `kind`; with timing on, bracket it with events.
#define STAGE(ctx, kind, name, ...)                                                     \
  do {                                                                                  \
    hipEvent_t a_ = nullptr;                                                            \
    const bool timed_ = ((ctx)->prof >> (kind)) & 1;                                    \
    if (timed_) {                                                                       \
      a_ = (ctx)->event();                                                              \
      if (!a_) return (ctx)->fail(VSR_EHIP, "hipEventCreate failed");                   \
      HIPCHECK(ctx, "profile event", hipEventRecord(a_, (ctx)->stream));                \
    }                                                                                   \
    HIPCHECK(ctx, name, (__VA_ARGS__));                                                 \
    if (timed_) {                                                                       \
      hipEvent_t b_ = (ctx)->event();                                                   \
      if (!b_) return (ctx)->fail(VSR_EHIP, "hipEventCreate failed");                   \
      HIPCHECK(ctx, "profile event", hipEventRecord(b_, (ctx)->stream));                \
      (ctx)->recs.push_back({(ctx)->phase * VSR_STAGE_KINDS + (kind), a_, b_});         \
    }                                                                                   \
  } while (0)

extern "C" size_t vsr_workspace_size(const vsr_config *cfg) {
  if (!check_config(cfg).empty()) return 0;
  return make_plan(*cfg).total;
}

extern "C" int vsr_create(const vsr_config *cfg, void *workspace, size_t ws_bytes,
                          void *hip_stream, vsr_ctx **out) {
  g_create_error.clear();
  if (!out) {
    g_create_error = "out is NULL";
    return VSR_EINVAL;
  }
  *out = nullptr;
  const std::string msg = check_config(cfg);
  if (!msg.empty()) {
    g_create_error = msg;
    return VSR_EINVAL;
  }
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255)) {
    g_create_error = "workspace must be a non-NULL, 256-byte aligned device pointer";
    return VSR_EINVAL;
  }
  const Plan plan = make_plan(*cfg);
  if (ws_bytes < plan.total) {
    g_create_error = "workspace smaller than vsr_workspace_size";
    return VSR_ENOMEM;
  }
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    g_create_error = std::string("HIP error in hipGetDevice: ") + hipGetErrorString(e);
    return VSR_EHIP;
  }
  vsr_ctx *c = new vsr_ctx();
  c->cfg = *cfg;
  c->plan = plan;
  c->ws = static_cast<char *>(workspace);
  c->stream = static_cast<hipStream_t>(hip_stream);
  c->device = dev;
  e = launch_rope_table(c->at<float2>(plan.rope), plan.rope_npos, cfg->head_dim, cfg->rope_base,
                        c->stream);
  // Cache slots past the written positions are read (and masked) by whole
  // key tiles: start them at zero so they are finite.
  if (e == hipSuccess)
    e = hipMemsetAsync(c->ws + plan.kc, 0, plan.part_acc - plan.kc, c->stream);
  if (e != hipSuccess) {
    g_create_error = std::string("HIP error in rope table: ") + hipGetErrorString(e);
    delete c;
    return VSR_EHIP;
  }
  *out = c;
  return VSR_OK;
}

extern "C" int vsr_load_weights(vsr_ctx *ctx, const vsr_weights *w) {
  if (!ctx) return VSR_EINVAL;
  if (!w || !w->embed || !w->lm_head || !w->final_norm)
    return ctx->fail(VSR_EINVAL, "weights: embed, lm_head and final_norm must be non-NULL");
  const int L = ctx->cfg.n_layers;
  if (L > 0 && (!w->attn_norm || !w->wqkv || !w->wo || !w->ffn_norm || !w->wgu || !w->wdown))
    return ctx->fail(VSR_EINVAL, "weights: per-layer pointer arrays must be non-NULL");
  for (int l = 0; l < L; ++l)
    if (!w->attn_norm[l] || !w->wqkv[l] || !w->wo[l] || !w->ffn_norm[l] || !w->wgu[l] ||
        !w->wdown[l])
      return ctx->fail(VSR_EINVAL, "weights: layer %d has a NULL tensor", l);
  ctx->embed = w->embed;
  ctx->lm_head = w->lm_head;
  ctx->final_norm = w->final_norm;
  ctx->attn_norm.assign(w->attn_norm, w->attn_norm + L);
  ctx->wqkv.assign(w->wqkv, w->wqkv + L);
  ctx->wo.assign(w->wo, w->wo + L);
  ctx->ffn_norm.assign(w->ffn_norm, w->ffn_norm + L);
  ctx->wgu.assign(w->wgu, w->wgu + L);
  ctx->wdown.assign(w->wdown, w->wdown + L);
  ctx->have_weights = true;
  ctx->prefilled = false;
  return VSR_OK;
}

namespace {

// One decoder block over `rows` rows whose residual stream is x. `mode` 0 is
// the prefix (causal, caches of layer l), 1 the candidates (cascade).
// TW is the weight type, TA the activation type (bf16 / fp16 on the MFMA
// path, float / float on the plain path).
template <typename TW, typename TA>
int run_layers(vsr_ctx *c, int rows, int mode, const Split &split) {
  constexpr bool kMfma = std::is_same<TA, f16>::value;
  const vsr_config &cf = c->cfg;
  const Plan &p = c->plan;
  const int d = cf.d_model, Hq = cf.n_heads, Hkv = cf.n_kv_heads, hd = cf.head_dim, F = cf.d_ff;
  float *x = c->at<float>(p.x);
  TA *xn = c->at<TA>(p.xn), *q = c->at<TA>(p.q), *attn = c->at<TA>(p.attn), *h = c->at<TA>(p.h);
  float *gpart = c->at<float>(p.gemm_part);
  const size_t layer_cache = (size_t)Hkv * p.kv_npos * hd;
  const size_t layer_dec = (size_t)Hkv * p.dec_npos * hd;
  const bool wf16 = cf.gemm_weights == VSR_F16;  // GEMM weights stored as fp16
  // mode 2 (draft): branch keys/values go to the persistent draft cache at
  // the rows' cache positions; queries see the prefix and their branch up to
  // their own position.
  // mode 3 (fused verify pass, MFMA path): rows 0 .. P-1 are the prefix (mode
  // 0 for them), rows P .. rows-1 the candidates (mode 1): one set of rows
  // through every projection, two attention launches per layer.
  const bool draft = mode == 2;
  const bool fused = mode == 3;
  const int P = c->P;
  const int32_t *cache_row = draft ? c->at<int32_t>(p.cache_row) : nullptr;
  hipStream_t s = c->stream;
  // Few-row products stream their weights (skinny kernels); their residual
  // reduces also apply the RMSNorm that follows (the FFN norm of the layer,
  // the next layer's attention norm), which then needs no launch of its own.
  bool xn_ready = false;
  for (int l = 0; l < cf.n_layers; ++l) {
    const TW *wqkv = static_cast<const TW *>(c->wqkv[l]);
    const TW *wo = static_cast<const TW *>(c->wo[l]);
    const TW *wgu = static_cast<const TW *>(c->wgu[l]);
    const TW *wdown = static_cast<const TW *>(c->wdown[l]);
    TA *kc = c->at<TA>(p.kc) + l * layer_cache;
    TA *vtc = c->at<TA>(p.vtc) + l * layer_cache;
    // Leading layers carry their GEMM and attention operands as fp16 value +
    // remainder.
    const bool precise = kMfma && l < cf.split_layers;
    const int sp = precise ? 2 : 1;
    // The feed-forward block of a precise layer is split too only in the
    // first split_mlp_layers layers.
    const int spm = kMfma && l < cf.split_mlp_layers ? 2 : 1;
    if (!xn_ready)
      STAGE(c, K_NORM, "attention norm",
            launch_rmsnorm<TW, TA>(x, static_cast<const TW *>(c->attn_norm[l]), rows, d,
                                   cf.rms_eps, xn, sp, s));
    xn_ready = false;
    QKVOut<TA> qo;
    qo.q = q;
    // The fast attention kernels take the queries pre-scaled (log2 units).
    if (kMfma && !precise) qo.q_scale = 1.4426950408889634f / std::sqrt((float)cf.head_dim);
    qo.rope = c->at<float2>(p.rope);
    if (mode == 0 || fused) {
      qo.k = kc;
      qo.vt = vtc;
      qo.kv_npos = p.kv_npos;
      qo.row_pos = nullptr;
      if (fused) {
        qo.split = P;
        qo.k2 = c->at<TA>(p.bk);
        qo.vt2 = c->at<TA>(p.bvt);
        qo.kv_npos2 = p.bk_npos;
        qo.row_pos2 = c->at<int32_t>(p.row_pos);
      }
    } else if (!draft) {
      qo.k = c->at<TA>(p.bk);
      qo.vt = c->at<TA>(p.bvt);
      qo.kv_npos = p.bk_npos;
      qo.row_pos = c->at<int32_t>(p.row_pos);
    } else {
      qo.k = c->at<TA>(p.kd) + l * layer_dec;
      qo.vt = c->at<TA>(p.vtd) + l * layer_dec;
      qo.kv_npos = p.dec_npos;
      qo.row_pos = c->at<int32_t>(p.row_pos);
      qo.cache_row = cache_row;
    }
    TA *bk = draft ? c->at<TA>(p.kd) + l * layer_dec : c->at<TA>(p.bk);
    TA *bvt = draft ? c->at<TA>(p.vtd) + l * layer_dec : c->at<TA>(p.bvt);
    TA *bk_lo = draft ? c->at<TA>(p.kd_lo) + l * layer_dec : c->at<TA>(p.bk_lo);
    TA *bvt_lo = draft ? c->at<TA>(p.vtd_lo) + l * layer_dec : c->at<TA>(p.bvt_lo);
    const int bk_npos = draft ? p.dec_npos : p.bk_npos;
    if (precise) {
      qo.q_lo = c->at<TA>(p.q_lo);
      qo.k_lo = mode == 0 || fused ? c->at<TA>(p.kc_lo) + l * layer_cache : bk_lo;
      qo.vt_lo = mode == 0 || fused ? c->at<TA>(p.vtc_lo) + l * layer_cache : bvt_lo;
      if (fused) {
        qo.k2_lo = bk_lo;
        qo.vt2_lo = bvt_lo;
      }
    }
    if constexpr (kMfma) {
      if (rows <= kSkinnyMaxRows)
        STAGE(c, K_QKV, "qkv projection",
              skinny_qkv_rope(xn, rows, sp, wqkv, wf16, d, Hq, Hkv, qo, gpart, s));
      else
        STAGE(c, K_QKV, "qkv projection",
              gemm_qkv_rope(xn, wqkv, wf16, rows, d, sp, Hq, Hkv, qo, gpart, s));
    } else {
      STAGE(c, K_QKV, "qkv projection",
            simple_qkv_rope<TA>(xn, wqkv, rows, d, Hq, Hkv, hd, qo, s));
    }
    // The prefix's last layer only feeds the last prefix row (the hidden state
    // that predicts candidate token 0): its keys/values are needed for every
    // row, its attention output, projections and FFN for row P-1 only.
    // In the fused pass the same holds for the prefix rows: the last layer
    // takes rows P-1 .. rows-1 (the last prefix row and the candidates).
    const bool tail = (mode == 0 || fused) && l == cf.n_layers - 1;
    const int r0 = tail ? (fused ? P - 1 : rows - 1) : 0, nr = rows - r0;
    if constexpr (kMfma) {
      AttnArgs a{};
      a.t0 = r0;
      a.q = q;
      a.k = kc;
      a.vt = vtc;
      a.kv_npos = p.kv_npos;
      a.bk = bk;
      a.bvt = bvt;
      a.bk_npos = bk_npos;
      a.q_pos = cache_row;
      a.bk_valid = draft ? p.dec_npos : 0;
      a.row_lo = c->at<int32_t>(p.row_lo);
      a.T = rows;
      a.P = c->P;
      a.n_heads = Hq;
      a.n_kv = Hkv;
      a.nchunks = split.nchunks;
      a.out = attn;
      a.out_split = sp;
      a.part_acc = c->at<float>(p.part_acc);
      a.part_ml = c->at<float2>(p.part_ml);
      if (precise) {
        a.q_lo = c->at<f16>(p.q_lo);
        a.k_lo = c->at<f16>(p.kc_lo) + l * layer_cache;
        a.vt_lo = c->at<f16>(p.vtc_lo) + l * layer_cache;
        a.bk_lo = bk_lo;
        a.bvt_lo = bvt_lo;
      }
      if (fused) {
        // Prefix rows (causal over the prefix cache), then the candidate rows
        // (their queries, outputs and remainder planes start at row P).
        AttnArgs ap = a;
        ap.T = P;
        ap.t0 = tail ? P - 1 : 0;
        ap.q_pos = nullptr;
        ap.nchunks = tail ? 1 : prefill_chunks(P, Hq, Hkv);
        STAGE(c, K_ATTN, "prefill attention", attn_prefill(ap, precise, s));
        if (ap.nchunks > 1) STAGE(c, K_MERGE, "prefill merge", attn_merge(ap, s));
        const size_t qoff = (size_t)P * Hq * hd;
        a.T = rows - P;
        a.t0 = 0;
        a.q = q + qoff;
        if (precise) a.q_lo = c->at<f16>(p.q_lo) + qoff;
        a.out = attn + qoff * sp;
        STAGE(c, K_CATTN, "candidate attention", attn_cascade(a, precise, s));
        STAGE(c, K_MERGE, "cascade merge", attn_merge(a, s));
      } else if (mode == 0) {
        a.nchunks = tail ? 1 : prefill_chunks(rows, Hq, Hkv);
        STAGE(c, K_ATTN, "prefill attention", attn_prefill(a, precise, s));
        if (a.nchunks > 1) STAGE(c, K_MERGE, "prefill merge", attn_merge(a, s));
      } else {
        STAGE(c, K_ATTN, "cascade attention", attn_cascade(a, precise, s));
        STAGE(c, K_MERGE, "cascade merge", attn_merge(a, s));
      }
    } else {
      SimpleAttnArgs a{};
      a.q = q;
      a.k = kc;
      a.vt = vtc;
      a.kv_npos = p.kv_npos;
      a.bk = bk;
      a.bvt = bvt;
      a.bk_npos = bk_npos;
      a.row_lo = c->at<int32_t>(p.row_lo);
      a.q_pos = cache_row;
      a.T = rows;
      a.P = c->P;
      a.n_heads = Hq;
      a.n_kv = Hkv;
      a.hd = hd;
      a.t0 = r0;
      a.mode = mode == 0 ? 0 : 1;
      a.out = attn;
      STAGE(c, K_ATTN, "attention", simple_attn<TA>(a, s));
    }
    const TA *attn_r = attn + (size_t)r0 * Hq * hd * sp;
    float *x_r = x + (size_t)r0 * d;
    const TW *ffn_g = static_cast<const TW *>(c->ffn_norm[l]);
    if constexpr (kMfma) {
      if (nr <= kSkinnyMaxRows) {
        // Output projection + residual + FFN norm; gate/up + SwiGLU; down
        // projection + residual (+ the next layer's attention norm). The
        // prefix pass's last-row layer is timed as a kind of its own.
        STAGE(c, tail ? K_TAIL : K_OPROJ, "output projection",
              skinny_residual(attn_r, nr, sp, wo, wf16, d, Hq * hd, x_r, ffn_g, cf.rms_eps, xn,
                              spm, gpart, s));
        STAGE(c, tail ? K_TAIL : K_GATEUP, "gate/up projection",
              skinny_swiglu(xn, nr, spm, wgu, wf16, F, d, h, gpart, s));
        const bool next = l + 1 < cf.n_layers;
        const int sp_next = kMfma && l + 1 < cf.split_layers ? 2 : 1;
        STAGE(c, tail ? K_TAIL : K_DOWN, "down projection",
              skinny_residual(h, nr, spm, wdown, wf16, d, F, x_r,
                              next ? static_cast<const TW *>(c->attn_norm[l + 1]) : nullptr,
                              cf.rms_eps, xn, sp_next, gpart, s));
        xn_ready = next;
        continue;
      }
      STAGE(c, K_OPROJ, "output projection",
            gemm_residual(attn_r, wo, wf16, nr, d, Hq * hd, sp, x_r, gpart, s));
    } else {
      STAGE(c, K_OPROJ, "output projection",
            simple_residual<TA>(attn_r, wo, nr, d, Hq * hd, x_r, s));
    }
    STAGE(c, K_NORM, "ffn norm",
          launch_rmsnorm<TW, TA>(x_r, ffn_g, nr, d, cf.rms_eps, xn, spm, s));
    if constexpr (kMfma) {
      STAGE(c, K_GATEUP, "gate/up projection",
            gemm_swiglu(xn, wgu, wf16, nr, F, d, spm, h, gpart, s));
      STAGE(c, K_DOWN, "down projection",
            gemm_residual(h, wdown, wf16, nr, d, F, spm, x_r, gpart, s));
    } else {
      STAGE(c, K_GATEUP, "gate/up projection", simple_swiglu<TA>(xn, wgu, nr, F, d, h, s));
      STAGE(c, K_DOWN, "down projection", simple_residual<TA>(h, wdown, nr, d, F, x_r, s));
    }
  }
  return VSR_OK;
}

template <typename TW, typename TA>
int prefill_impl(vsr_ctx *c, const void *visual, int nv, const int32_t *ids, int nt) {
  const vsr_config &cf = c->cfg;
  const Plan &p = c->plan;
  const int P = nv + nt;
  float *x = c->at<float>(p.x);
  STAGE(c, K_EMBED, "prefix embedding",
           launch_embed_prefix<TW>(static_cast<const TW *>(visual), nv, ids, nt,
                                   static_cast<const TW *>(c->embed), cf.vocab, cf.d_model, x,
                                   c->at<int32_t>(p.flags), c->stream));
  c->P = P;
  const int rc = run_layers<TW, TA>(c, P, 0, Split{1});
  if (rc) return rc;
  STAGE(c, K_COPY, "last prefix row",
           hipMemcpyAsync(c->at<float>(p.h_last), x + (size_t)(P - 1) * cf.d_model,
                          (size_t)cf.d_model * 4, hipMemcpyDeviceToDevice, c->stream));
  return VSR_OK;
}

// The candidate rows of a score or reliability call through every layer:
// row tables, embedding, the decoder blocks in cascade mode (residual stream
// left in x).
template <typename TW, typename TA>
int branch_forward(vsr_ctx *c, const Branches &br, const int32_t *cand_ids) {
  constexpr bool kMfma = std::is_same<TA, f16>::value;
  const vsr_config &cf = c->cfg;
  const Plan &p = c->plan;
  const int T_rows = br.cu[br.M];
  hipStream_t s = c->stream;
  int32_t *row_lo = c->at<int32_t>(p.row_lo), *row_pos = c->at<int32_t>(p.row_pos);
  int32_t *lm_tgt = c->at<int32_t>(p.lm_tgt);
  STAGE(c, K_ROWS, "row tables",
        launch_row_tables(br, c->P, cand_ids, cf.vocab, c->at<int32_t>(p.flags), row_lo, row_pos,
                          lm_tgt, s));
  STAGE(c, K_EMBED, "candidate embedding",
        launch_embed_rows<TW>(lm_tgt, T_rows, static_cast<const TW *>(c->embed), cf.d_model,
                              c->at<float>(p.x), s));
  const Split split =
      kMfma ? cascade_split(T_rows, c->P + br.cmax, cf.n_heads, cf.n_kv_heads) : Split{1};
  return run_layers<TW, TA>(c, T_rows, 1, split);
}

// LM head over `rows` prepared input rows (xn) with targets lm_tgt: chunk
// partials (max, sum exp) and target logits.
template <typename TW, typename TA>
int lm_head(vsr_ctx *c, int rows, int *chunks) {
  constexpr bool kMfma = std::is_same<TA, f16>::value;
  const vsr_config &cf = c->cfg;
  const Plan &p = c->plan;
  hipStream_t s = c->stream;
  const TA *lm_in = c->at<TA>(p.xn);
  int32_t *lm_tgt = c->at<int32_t>(p.lm_tgt);
  float2 *lm_part = c->at<float2>(p.lm_part);
  float *tgt = c->at<float>(p.tgt);
  if constexpr (kMfma) {
    *chunks = lmhead_chunks(cf.vocab);
    STAGE(c, K_LMHEAD, "lm head",
          gemm_lmhead(lm_in, c->lm_head, cf.gemm_weights == VSR_F16, rows, cf.vocab,
                      cf.d_model, lm_tgt, lm_part, tgt, s));
  } else {
    *chunks = 1;
    STAGE(c, K_LMHEAD, "lm head",
          simple_lmhead<TA>(lm_in, static_cast<const TW *>(c->lm_head), rows, cf.vocab,
                            cf.d_model, lm_tgt, lm_part, tgt, s));
  }
  return VSR_OK;
}

template <typename TW, typename TA>
int score_impl(vsr_ctx *c, const Branches &br, const int32_t *cand_ids, float *logprobs,
               float *scores, int32_t *argmax) {
  const vsr_config &cf = c->cfg;
  const Plan &p = c->plan;
  const int T_rows = br.cu[br.M];
  hipStream_t s = c->stream;
  int lm_chunks = 1;
  if (T_rows > 0) {
    int rc = branch_forward<TW, TA>(c, br, cand_ids);
    if (rc) return rc;
    STAGE(c, K_LMIN, "lm inputs",
          launch_lm_inputs<TW, TA>(c->at<float>(p.x), c->at<float>(p.h_last),
                                   c->at<int32_t>(p.row_lo),
                                   static_cast<const TW *>(c->final_norm), T_rows, cf.d_model,
                                   cf.rms_eps, c->at<TA>(p.xn), s));
    rc = lm_head<TW, TA>(c, T_rows, &lm_chunks);
    if (rc) return rc;
  }
  STAGE(c, K_LSE, "lse gather",
        launch_lse_gather(br, c->at<float2>(p.lm_part), lm_chunks, c->at<float>(p.tgt),
                          logprobs, s));
  STAGE(c, K_SELECT, "reduce/select", launch_reduce_select(br, logprobs, scores, argmax, s));
  return VSR_OK;
}

// Prefix and candidates in one pass (MFMA contexts): the prefix rows and the
// candidate rows go through every projection together (one GEMM launch per
// projection for both); per layer, the prefix rows attend causally over the
// prefix cache and the candidate rows over the prefix + their own keys. The
// prefix cache is left filled, as after a prefill.
template <typename TW, typename TA>
int verify_impl(vsr_ctx *c, const void *visual, int nv, const int32_t *ids, int nt,
                const Branches &br, const int32_t *cand_ids, float *logprobs, float *scores,
                int32_t *argmax) {
  const vsr_config &cf = c->cfg;
  const Plan &p = c->plan;
  const int P = nv + nt, T_rows = br.cu[br.M];
  hipStream_t s = c->stream;
  float *x = c->at<float>(p.x);
  STAGE(c, K_EMBED, "prefix embedding",
        launch_embed_prefix<TW>(static_cast<const TW *>(visual), nv, ids, nt,
                                static_cast<const TW *>(c->embed), cf.vocab, cf.d_model, x,
                                c->at<int32_t>(p.flags), s));
  c->P = P;
  int32_t *row_lo = c->at<int32_t>(p.row_lo), *row_pos = c->at<int32_t>(p.row_pos);
  int32_t *lm_tgt = c->at<int32_t>(p.lm_tgt);
  float *xc = x + (size_t)P * cf.d_model;  // the candidate rows
  STAGE(c, K_ROWS, "row tables",
        launch_row_tables(br, P, cand_ids, cf.vocab, c->at<int32_t>(p.flags), row_lo, row_pos,
                          lm_tgt, s));
  STAGE(c, K_EMBED, "candidate embedding",
        launch_embed_rows<TW>(lm_tgt, T_rows, static_cast<const TW *>(c->embed), cf.d_model, xc,
                              s));
  const Split split = cascade_split(T_rows, P + br.cmax, cf.n_heads, cf.n_kv_heads);
  int rc = run_layers<TW, TA>(c, P + T_rows, 3, split);
  if (rc) return rc;
  STAGE(c, K_COPY, "last prefix row",
        hipMemcpyAsync(c->at<float>(p.h_last), x + (size_t)(P - 1) * cf.d_model,
                       (size_t)cf.d_model * 4, hipMemcpyDeviceToDevice, s));
  c->prefilled = true;
  STAGE(c, K_LMIN, "lm inputs",
        launch_lm_inputs<TW, TA>(xc, c->at<float>(p.h_last), row_lo,
                                 static_cast<const TW *>(c->final_norm), T_rows, cf.d_model,
                                 cf.rms_eps, c->at<TA>(p.xn), s));
  int lm_chunks = 1;
  rc = lm_head<TW, TA>(c, T_rows, &lm_chunks);
  if (rc) return rc;
  STAGE(c, K_LSE, "lse gather",
        launch_lse_gather(br, c->at<float2>(p.lm_part), lm_chunks, c->at<float>(p.tgt),
                          logprobs, s));
  STAGE(c, K_SELECT, "reduce/select", launch_reduce_select(br, logprobs, scores, argmax, s));
  return VSR_OK;
}

template <typename TW, typename TA>
int reliability_impl(vsr_ctx *c, const Branches &br, const int32_t *ids, int yes_id, int no_id,
                     float delta, float *lp_yes_no, float *rel, int32_t *keep) {
  const vsr_config &cf = c->cfg;
  const Plan &p = c->plan;
  hipStream_t s = c->stream;
  int rc = branch_forward<TW, TA>(c, br, ids);
  if (rc) return rc;
  STAGE(c, K_LMIN, "last-row inputs",
        launch_last_inputs<TW, TA>(c->at<float>(p.x), br, static_cast<const TW *>(c->final_norm),
                                   cf.d_model, cf.rms_eps, yes_id, no_id, c->at<TA>(p.xn),
                                   c->at<int32_t>(p.lm_tgt), s));
  int chunks = 1;
  rc = lm_head<TW, TA>(c, 2 * br.M, &chunks);
  if (rc) return rc;
  STAGE(c, K_LSE, "reliability",
        launch_reliability_finish(br.M, c->at<float2>(p.lm_part), chunks, c->at<float>(p.tgt),
                                  delta, lp_yes_no, rel, keep, s));
  return VSR_OK;
}

// Greedy drafts: the prompt rows of every branch through all layers (keys /
// values kept in the draft cache), then n_new steps of one row per branch.
// Each step's LM head picks the next token on the device and feeds it to the
// next step's embedding, so the loop never waits for the host.
template <typename TW, typename TA>
int draft_impl(vsr_ctx *c, const Branches &br, const int32_t *ids, int n_new, int32_t *tokens) {
  constexpr bool kMfma = std::is_same<TA, f16>::value;
  const vsr_config &cf = c->cfg;
  const Plan &p = c->plan;
  hipStream_t s = c->stream;
  const int M = br.M, T_rows = br.cu[M];
  int32_t *row_lo = c->at<int32_t>(p.row_lo), *row_pos = c->at<int32_t>(p.row_pos);
  int32_t *cache_row = c->at<int32_t>(p.cache_row), *lm_tgt = c->at<int32_t>(p.lm_tgt);
  int32_t *next_ids = c->at<int32_t>(p.dec_ids);
  float *x = c->at<float>(p.x);
  TA *lm_in = c->at<TA>(p.xn);
  float2 *part = c->at<float2>(p.lm_part);
  const TW *g = static_cast<const TW *>(c->final_norm);
  const bool wf16 = cf.gemm_weights == VSR_F16;
  const bool skinny_lm = kMfma && M <= kSkinnyMaxRows && skinny_lm_chunks(cf.vocab) > 0;
  const int chunks = !kMfma ? 1 : skinny_lm ? skinny_lm_chunks(cf.vocab) : lmhead_chunks(cf.vocab);
  auto pick = [&](int step) -> int {
    if constexpr (kMfma) {
      if (skinny_lm)
        STAGE(c, K_LMHEAD, "draft lm head",
              skinny_lmargmax(lm_in, M, c->lm_head, wf16, cf.vocab, cf.d_model, part, s));
      else
        STAGE(c, K_LMHEAD, "draft lm head",
              gemm_lmargmax(lm_in, c->lm_head, wf16, M, cf.vocab, cf.d_model, part, s));
    } else {
      STAGE(c, K_LMHEAD, "draft lm head",
            simple_lmargmax<TA>(lm_in, static_cast<const TW *>(c->lm_head), M, cf.vocab,
                                cf.d_model, part, s));
    }
    STAGE(c, K_SELECT, "draft pick",
          launch_argmax_merge(part, chunks, M, n_new, step, tokens, next_ids, s));
    return VSR_OK;
  };
  STAGE(c, K_ROWS, "draft rows",
        launch_draft_rows(br, c->P, p.dec_S, ids, cf.vocab, c->at<int32_t>(p.flags), row_lo,
                          row_pos, cache_row, lm_tgt, s));
  STAGE(c, K_EMBED, "draft embedding",
        launch_embed_rows<TW>(lm_tgt, T_rows, static_cast<const TW *>(c->embed), cf.d_model,
                              x, s));
  // A prompt-pass block spans about one branch; a decode-step block spans
  // the cache segments of all of them.
  const Split split0 =
      kMfma ? cascade_split(T_rows, c->P + p.dec_S, cf.n_heads, cf.n_kv_heads) : Split{1};
  int rc = run_layers<TW, TA>(c, T_rows, 2, split0);
  if (rc) return rc;
  STAGE(c, K_LMIN, "draft inputs",
        launch_branch_last_norm<TW, TA>(x, br, g, cf.d_model, cf.rms_eps, lm_in, s));
  rc = pick(0);
  if (rc) return rc;
  const Split split1 =
      kMfma ? cascade_split(M, c->P + M * p.dec_S, cf.n_heads, cf.n_kv_heads) : Split{1};
  for (int step = 1; step < n_new; ++step) {
    STAGE(c, K_ROWS, "draft step rows",
          launch_draft_step(br, c->P, p.dec_S, step, row_lo, row_pos, cache_row, s));
    STAGE(c, K_EMBED, "draft step embedding",
          launch_embed_rows<TW>(next_ids, M, static_cast<const TW *>(c->embed), cf.d_model, x,
                                s));
    rc = run_layers<TW, TA>(c, M, 2, split1);
    if (rc) return rc;
    STAGE(c, K_LMIN, "draft step inputs",
          launch_rmsnorm<TW, TA>(x, g, M, cf.d_model, cf.rms_eps, lm_in, 1, s));
    rc = pick(step);
    if (rc) return rc;
  }
  return VSR_OK;
}

int set_device(vsr_ctx *c) {
  int cur = -1;
  if (hipGetDevice(&cur) == hipSuccess && cur == c->device) return VSR_OK;
  HIPCHECK(c, "hipSetDevice", hipSetDevice(c->device));
  return VSR_OK;
}

// Checked calls (vsr_set_checks): the status word is cleared before the
// call's launches and read once after them (the call then waits for its
// stream). `vals` (n floats, device) are the call's results whose finiteness
// is checked.
int checks_begin(vsr_ctx *c) {
  if (!c->checks) return VSR_OK;
  HIPCHECK(c, "checks", launch_flags_clear(c->at<int32_t>(c->plan.flags), c->stream));
  return VSR_OK;
}

int checks_end(vsr_ctx *c, int rc, const float *vals, long n) {
  if (rc != VSR_OK || !c->checks) return rc;
  int32_t *flags = c->at<int32_t>(c->plan.flags);
  if ((c->checks & VSR_CHECK_FINITE) && vals)
    HIPCHECK(c, "checks", launch_check_finite(vals, n, flags, c->stream));
  int32_t f = 0;
  HIPCHECK(c, "checks", hipMemcpyAsync(&f, flags, sizeof f, hipMemcpyDeviceToHost, c->stream));
  HIPCHECK(c, "checks", hipStreamSynchronize(c->stream));
  if ((c->checks & VSR_CHECK_IDS) && (f & kFlagBadId))
    return c->fail(VSR_EID, "an id outside [0, vocab) was read (it was used as id 0)");
  if ((c->checks & VSR_CHECK_FINITE) && (f & kFlagNonFinite))
    return c->fail(VSR_ENONFINITE, "the results hold a NaN or an infinity");
  return VSR_OK;
}

}  // namespace

extern "C" int vsr_prefill(vsr_ctx *ctx, const void *visual, int32_t n_visual,
                           const int32_t *ids, int32_t n_text) {
  if (!ctx) return VSR_EINVAL;
  if (!ctx->have_weights) return ctx->fail(VSR_ESTATE, "prefill before vsr_load_weights");
  if (n_visual < 0 || n_text < 0) return ctx->fail(VSR_EINVAL, "negative prefix length");
  const long long P = (long long)n_visual + n_text;
  if (P < 1) return ctx->fail(VSR_EINVAL, "empty prefix (n_visual + n_text must be >= 1)");
  if (P > ctx->cfg.max_prefix)
    return ctx->fail(VSR_ERANGE, "prefix length %lld exceeds max_prefix %d", P,
                     ctx->cfg.max_prefix);
  if (n_visual > 0 && !visual) return ctx->fail(VSR_EINVAL, "visual is NULL");
  if (n_text > 0 && !ids) return ctx->fail(VSR_EINVAL, "ids is NULL");
  int rc = set_device(ctx);
  if (rc) return rc;
  ctx->prefilled = false;
  ctx->phase = 0;
  rc = checks_begin(ctx);
  if (rc) return rc;
  rc = ctx->cfg.dtype == VSR_BF16
           ? prefill_impl<bf16, f16>(ctx, visual, n_visual, ids, n_text)
           : prefill_impl<float, float>(ctx, visual, n_visual, ids, n_text);
  if (rc == VSR_OK) ctx->prefilled = true;
  return checks_end(ctx, rc, ctx->at<float>(ctx->plan.h_last), ctx->cfg.d_model);
}

extern "C" int vsr_score(vsr_ctx *ctx, const int32_t *cand_ids, const int32_t *cand_len,
                         int32_t M, int32_t Cmax, float *logprobs, float *scores,
                         int32_t *argmax) {
  if (!ctx) return VSR_EINVAL;
  if (!ctx->prefilled) return ctx->fail(VSR_ESTATE, "score before a successful prefill");
  if (M < 1 || Cmax < 1) return ctx->fail(VSR_EINVAL, "M and Cmax must be >= 1");
  if (M > ctx->cfg.max_cands)
    return ctx->fail(VSR_ERANGE, "M = %d exceeds max_cands %d", M, ctx->cfg.max_cands);
  if (Cmax > ctx->cfg.max_cand_len)
    return ctx->fail(VSR_ERANGE, "Cmax = %d exceeds max_cand_len %d", Cmax,
                     ctx->cfg.max_cand_len);
  if (!cand_ids || !cand_len || !logprobs || !scores || !argmax)
    return ctx->fail(VSR_EINVAL, "score: NULL argument");
  Branches br{};
  br.M = M;
  br.cmax = Cmax;
  br.cu[0] = 0;
  for (int m = 0; m < M; ++m) {
    if (cand_len[m] < 0 || cand_len[m] > Cmax)
      return ctx->fail(VSR_EINVAL, "cand_len[%d] = %d outside [0, Cmax]", m, cand_len[m]);
    br.cu[m + 1] = br.cu[m] + cand_len[m];
  }
  int rc = set_device(ctx);
  if (rc) return rc;
  ctx->phase = 1;
  rc = checks_begin(ctx);
  if (rc) return rc;
  rc = ctx->cfg.dtype == VSR_BF16
           ? score_impl<bf16, f16>(ctx, br, cand_ids, logprobs, scores, argmax)
           : score_impl<float, float>(ctx, br, cand_ids, logprobs, scores, argmax);
  return checks_end(ctx, rc, scores, M);
}

extern "C" int vsr_verify(vsr_ctx *ctx, const void *visual, int32_t n_visual,
                          const int32_t *ids, int32_t n_text, const int32_t *cand_ids,
                          const int32_t *cand_len, int32_t M, int32_t Cmax, float *logprobs,
                          float *scores, int32_t *argmax) {
  if (!ctx) return VSR_EINVAL;
  if (!ctx->have_weights) return ctx->fail(VSR_ESTATE, "verify before vsr_load_weights");
  if (n_visual < 0 || n_text < 0) return ctx->fail(VSR_EINVAL, "negative prefix length");
  const long long P = (long long)n_visual + n_text;
  if (P < 1) return ctx->fail(VSR_EINVAL, "empty prefix (n_visual + n_text must be >= 1)");
  if (P > ctx->cfg.max_prefix)
    return ctx->fail(VSR_ERANGE, "prefix length %lld exceeds max_prefix %d", P,
                     ctx->cfg.max_prefix);
  if (n_visual > 0 && !visual) return ctx->fail(VSR_EINVAL, "visual is NULL");
  if (n_text > 0 && !ids) return ctx->fail(VSR_EINVAL, "ids is NULL");
  if (M < 1 || Cmax < 1) return ctx->fail(VSR_EINVAL, "M and Cmax must be >= 1");
  if (M > ctx->cfg.max_cands)
    return ctx->fail(VSR_ERANGE, "M = %d exceeds max_cands %d", M, ctx->cfg.max_cands);
  if (Cmax > ctx->cfg.max_cand_len)
    return ctx->fail(VSR_ERANGE, "Cmax = %d exceeds max_cand_len %d", Cmax,
                     ctx->cfg.max_cand_len);
  if (!cand_ids || !cand_len || !logprobs || !scores || !argmax)
    return ctx->fail(VSR_EINVAL, "verify: NULL argument");
  Branches br{};
  br.M = M;
  br.cmax = Cmax;
  br.cu[0] = 0;
  for (int m = 0; m < M; ++m) {
    if (cand_len[m] < 0 || cand_len[m] > Cmax)
      return ctx->fail(VSR_EINVAL, "cand_len[%d] = %d outside [0, Cmax]", m, cand_len[m]);
    br.cu[m + 1] = br.cu[m] + cand_len[m];
  }
  int rc = set_device(ctx);
  if (rc) return rc;
  ctx->prefilled = false;
  rc = checks_begin(ctx);
  if (rc) return rc;
  if (ctx->cfg.dtype == VSR_BF16 && br.cu[M] > 0) {
    ctx->phase = 3;
    rc = verify_impl<bf16, f16>(ctx, visual, n_visual, ids, n_text, br, cand_ids, logprobs,
                                scores, argmax);
    return checks_end(ctx, rc, scores, M);
  }
  // fp32 contexts, or no candidate tokens: the two passes one after the other.
  ctx->phase = 0;
  rc = ctx->cfg.dtype == VSR_BF16
           ? prefill_impl<bf16, f16>(ctx, visual, n_visual, ids, n_text)
           : prefill_impl<float, float>(ctx, visual, n_visual, ids, n_text);
  if (rc) return rc;
  ctx->prefilled = true;
  ctx->phase = 1;
  rc = ctx->cfg.dtype == VSR_BF16
           ? score_impl<bf16, f16>(ctx, br, cand_ids, logprobs, scores, argmax)
           : score_impl<float, float>(ctx, br, cand_ids, logprobs, scores, argmax);
  return checks_end(ctx, rc, scores, M);
}

extern "C" int vsr_reliability(vsr_ctx *ctx, const int32_t *branch_ids,
                               const int32_t *branch_len, int32_t M, int32_t Cmax,
                               int32_t yes_id, int32_t no_id, float delta, float *lp_yes_no,
                               float *rel, int32_t *keep) {
  if (!ctx) return VSR_EINVAL;
  if (!ctx->prefilled) return ctx->fail(VSR_ESTATE, "reliability before a successful prefill");
  if (M < 1 || Cmax < 1) return ctx->fail(VSR_EINVAL, "M and Cmax must be >= 1");
  if (M > ctx->cfg.max_cands)
    return ctx->fail(VSR_ERANGE, "M = %d exceeds max_cands %d", M, ctx->cfg.max_cands);
  if (Cmax > ctx->cfg.max_cand_len)
    return ctx->fail(VSR_ERANGE, "Cmax = %d exceeds max_cand_len %d", Cmax,
                     ctx->cfg.max_cand_len);
  if (!branch_ids || !branch_len || !lp_yes_no || !rel || !keep)
    return ctx->fail(VSR_EINVAL, "reliability: NULL argument");
  if (yes_id < 0 || yes_id >= ctx->cfg.vocab || no_id < 0 || no_id >= ctx->cfg.vocab)
    return ctx->fail(VSR_EINVAL, "yes_id and no_id must lie in [0, vocab)");
  if (!(delta >= 0.f) || !std::isfinite(delta))
    return ctx->fail(VSR_EINVAL, "delta must be finite and >= 0");
  Branches br{};
  br.M = M;
  br.cmax = Cmax;
  br.cu[0] = 0;
  for (int m = 0; m < M; ++m) {
    if (branch_len[m] < 1 || branch_len[m] > Cmax)
      return ctx->fail(VSR_EINVAL, "branch_len[%d] = %d outside [1, Cmax]", m, branch_len[m]);
    br.cu[m + 1] = br.cu[m] + branch_len[m];
  }
  int rc = set_device(ctx);
  if (rc) return rc;
  ctx->phase = 1;
  rc = checks_begin(ctx);
  if (rc) return rc;
  rc = ctx->cfg.dtype == VSR_BF16
           ? reliability_impl<bf16, f16>(ctx, br, branch_ids, yes_id, no_id, delta, lp_yes_no,
                                         rel, keep)
           : reliability_impl<float, float>(ctx, br, branch_ids, yes_id, no_id, delta,
                                            lp_yes_no, rel, keep);
  return checks_end(ctx, rc, lp_yes_no, 2L * M);
}

extern "C" int vsr_draft(vsr_ctx *ctx, const int32_t *prompt_ids, const int32_t *prompt_len,
                         int32_t M, int32_t Cmax, int32_t n_new, int32_t *tokens) {
  if (!ctx) return VSR_EINVAL;
  if (!ctx->prefilled) return ctx->fail(VSR_ESTATE, "draft before a successful prefill");
  if (ctx->cfg.max_new < 1) return ctx->fail(VSR_ESTATE, "context created with max_new = 0");
  if (M < 1 || Cmax < 1) return ctx->fail(VSR_EINVAL, "M and Cmax must be >= 1");
  if (M > ctx->cfg.max_cands)
    return ctx->fail(VSR_ERANGE, "M = %d exceeds max_cands %d", M, ctx->cfg.max_cands);
  if (Cmax > ctx->cfg.max_cand_len)
    return ctx->fail(VSR_ERANGE, "Cmax = %d exceeds max_cand_len %d", Cmax,
                     ctx->cfg.max_cand_len);
  if (n_new < 1 || n_new > ctx->cfg.max_new)
    return ctx->fail(VSR_ERANGE, "n_new = %d outside [1, max_new = %d]", n_new,
                     ctx->cfg.max_new);
  if (!prompt_ids || !prompt_len || !tokens) return ctx->fail(VSR_EINVAL, "draft: NULL argument");
  Branches br{};
  br.M = M;
  br.cmax = Cmax;
  br.cu[0] = 0;
  for (int m = 0; m < M; ++m) {
    if (prompt_len[m] < 1 || prompt_len[m] > Cmax)
      return ctx->fail(VSR_EINVAL, "prompt_len[%d] = %d outside [1, Cmax]", m, prompt_len[m]);
    br.cu[m + 1] = br.cu[m] + prompt_len[m];
  }
  int rc = set_device(ctx);
  if (rc) return rc;
  ctx->phase = 2;
  rc = checks_begin(ctx);
  if (rc) return rc;
  rc = ctx->cfg.dtype == VSR_BF16 ? draft_impl<bf16, f16>(ctx, br, prompt_ids, n_new, tokens)
                                  : draft_impl<float, float>(ctx, br, prompt_ids, n_new, tokens);
  return checks_end(ctx, rc, nullptr, 0);
}

extern "C" int vsr_align_select(const float *ent, const float *frames, int32_t M, int32_t NF,
                                int32_t D, const float *rel, float delta, int32_t strategy,
                                float *align, int32_t *choice, void *hip_stream) {
  g_create_error.clear();
  const char *msg = nullptr;
  if (!ent || !frames || !rel || !align || !choice) msg = "align_select: NULL argument";
  else if (M < 1 || M > VSR_MAX_CANDS) msg = "M must lie in [1, VSR_MAX_CANDS]";
  else if (NF < 1) msg = "NF must be >= 1";
  else if (D < 1 || D > 4096) msg = "D must lie in [1, 4096]";
  else if (!(delta >= 0.f) || !std::isfinite(delta)) msg = "delta must be finite and >= 0";
  else if (strategy < VSR_SELECT_TWO_STAGE || strategy > VSR_SELECT_INVERT)
    msg = "unknown selection strategy";
  if (msg) {
    g_create_error = msg;
    return VSR_EINVAL;
  }
  const hipError_t e = launch_align_select(ent, frames, M, NF, D, rel, delta, strategy, align,
                                           choice, static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) {
    g_create_error = std::string("HIP error in align_select: ") + hipGetErrorString(e);
    return VSR_EHIP;
  }
  return VSR_OK;
}

extern "C" const char *vsr_last_error(const vsr_ctx *ctx) {
  return ctx ? ctx->err.c_str() : g_create_error.c_str();
}

extern "C" void vsr_destroy(vsr_ctx *ctx) { delete ctx; }

extern "C" int vsr_keyframes(const uint8_t *frames, int32_t NF, int32_t H, int32_t W,
                             float theta, int32_t *hist, int32_t *inter, int32_t *key_idx,
                             int32_t *n_keys, void *hip_stream) {
  g_create_error.clear();
  const char *msg = nullptr;
  if (!frames || !hist || !inter || !key_idx || !n_keys) msg = "keyframes: NULL argument";
  else if (reinterpret_cast<uintptr_t>(frames) & 15) msg = "frames must be 16-byte aligned";
  else if (NF < 1 || NF > 65536) msg = "NF must lie in [1, 65536]";
  else if (H < 1 || W < 1 || (long long)H * W > (1LL << 24)) msg = "need H, W >= 1, H W <= 2^24";
  else if (!std::isfinite(theta)) msg = "theta must be finite";
  if (msg) {
    g_create_error = msg;
    return VSR_EINVAL;
  }
  const hipError_t e = launch_keyframes(frames, NF, H, W, theta, hist, inter, key_idx, n_keys,
                                        static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) {
    g_create_error = std::string("HIP error in keyframes: ") + hipGetErrorString(e);
    return VSR_EHIP;
  }
  return VSR_OK;
}

namespace {
const char *retrieve_sizes_error(int32_t NF, int32_t ND, int32_t k) {
  if (NF < 1 || NF > 65536) return "NF must lie in [1, 65536]";
  if (ND < 1 || ND > (1 << 24)) return "ND must lie in [1, 2^24]";
  if (k < 1 || k > 16) return "k must lie in [1, 16]";
  return nullptr;
}
}  // namespace

extern "C" size_t vsr_retrieve_workspace_size(int32_t NF, int32_t ND, int32_t k) {
  return retrieve_sizes_error(NF, ND, k) ? 0 : retrieve_workspace_bytes(NF, ND, k);
}

extern "C" int vsr_retrieve(const float *frame_emb, const int32_t *key_idx,
                            const int32_t *n_keys, int32_t NF, const float *docs, int32_t ND,
                            int32_t D, int32_t k, int32_t K, void *workspace, size_t ws_bytes,
                            int32_t *top_idx, float *top_sim, int32_t *sel_idx, float *sel_sim,
                            int32_t *n_sel, void *hip_stream) {
  g_create_error.clear();
  const char *msg = retrieve_sizes_error(NF, ND, k);
  if (!msg) {
    if (!frame_emb || !key_idx || !n_keys || !docs || !workspace || !top_idx || !top_sim ||
        !sel_idx || !sel_sim || !n_sel)
      msg = "retrieve: NULL argument";
    else if (D < 1 || D > 1024) msg = "D must lie in [1, 1024]";
    else if (K < 1 || K > 64) msg = "K must lie in [1, 64]";
    else if (reinterpret_cast<uintptr_t>(workspace) & 7) msg = "workspace must be 8-byte aligned";
    else if (reinterpret_cast<uintptr_t>(docs) & 15) msg = "docs must be 16-byte aligned";
    else if (ws_bytes < retrieve_workspace_bytes(NF, ND, k))
      msg = "workspace smaller than vsr_retrieve_workspace_size";
  }
  if (msg) {
    g_create_error = msg;
    return VSR_EINVAL;
  }
  const hipError_t e = launch_retrieve(frame_emb, key_idx, n_keys, NF, docs, ND, D, k, K,
                                       workspace, top_idx, top_sim, sel_idx, sel_sim, n_sel,
                                       static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) {
    g_create_error = std::string("HIP error in retrieve: ") + hipGetErrorString(e);
    return VSR_EHIP;
  }
  return VSR_OK;
}

extern "C" int vsr_retrieve_static(const float *frame_emb, const int32_t *key_idx,
                                   const int32_t *n_keys, int32_t NF, const float *docs,
                                   int32_t ND, int32_t D, int32_t k, int32_t K,
                                   int32_t *top_idx, float *top_sim, int32_t *sel_idx,
                                   float *sel_sim, int32_t *n_sel, void *hip_stream) {
  g_create_error.clear();
  const char *msg = retrieve_sizes_error(NF, ND, k);
  if (!msg) {
    if (!frame_emb || !key_idx || !n_keys || !docs || !top_idx || !top_sim || !sel_idx ||
        !sel_sim || !n_sel)
      msg = "retrieve_static: NULL argument";
    else if (D < 1 || D > 1024) msg = "D must lie in [1, 1024]";
    else if (K < 1 || K > 64) msg = "K must lie in [1, 64]";
    else if (reinterpret_cast<uintptr_t>(docs) & 15) msg = "docs must be 16-byte aligned";
  }
  if (msg) {
    g_create_error = msg;
    return VSR_EINVAL;
  }
  const size_t need = retrieve_workspace_bytes(NF, ND, k);
  if (need > kRetrieveStaticBytes) {
    char buf[256];
    snprintf(buf, sizeof buf,
             "retrieve_static: NF=%d, ND=%d, k=%d need %zu bytes of scratch, more than the "
             "library's %zu (use vsr_retrieve with a workspace)",
             NF, ND, k, need, kRetrieveStaticBytes);
    g_create_error = buf;
    return VSR_ERANGE;
  }
  void *scratch = nullptr;
  hipError_t e = retrieve_static_scratch(&scratch);
  if (e == hipSuccess)
    e = launch_retrieve(frame_emb, key_idx, n_keys, NF, docs, ND, D, k, K, scratch, top_idx,
                        top_sim, sel_idx, sel_sim, n_sel, static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) {
    g_create_error = std::string("HIP error in retrieve_static: ") + hipGetErrorString(e);
    return VSR_EHIP;
  }
  return VSR_OK;
}

extern "C" int vsr_weights_to_f16(const void *src, void *dst, size_t n, void *hip_stream) {
  g_create_error.clear();
  const uintptr_t a = reinterpret_cast<uintptr_t>(src), b = reinterpret_cast<uintptr_t>(dst);
  if (n == 0) return VSR_OK;
  if (!src || !dst || (a & 15) || (b & 15)) {
    g_create_error = "weights_to_f16: src and dst must be non-NULL and 16-byte aligned";
    return VSR_EINVAL;
  }
  if ((a < b + 2 * n) && (b < a + 2 * n)) {
    g_create_error = "weights_to_f16: src and dst overlap";
    return VSR_EINVAL;
  }
  const hipError_t e = convert_bf16_to_f16(static_cast<const uint16_t *>(src),
                                           static_cast<uint16_t *>(dst), n,
                                           static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) {
    g_create_error = std::string("HIP error in weights_to_f16: ") + hipGetErrorString(e);
    return VSR_EHIP;
  }
  return VSR_OK;
}

extern "C" int vsr_set_checks(vsr_ctx *ctx, int checks) {
  if (!ctx) return VSR_EINVAL;
  if (checks & ~(VSR_CHECK_IDS | VSR_CHECK_FINITE))
    return ctx->fail(VSR_EINVAL, "set_checks: unknown check bits 0x%x", checks);
  ctx->checks = checks;
  return VSR_OK;
}

extern "C" int vsr_profile_enable(vsr_ctx *ctx, int kinds) {
  if (!ctx) return VSR_EINVAL;
  if (kinds & ~VSR_PROFILE_ALL) return ctx->fail(VSR_EINVAL, "profile_enable: unknown stage kinds");
  if (!ctx->recs.empty()) HIPCHECK(ctx, "profile sync", hipStreamSynchronize(ctx->stream));
  ctx->drop_records();
  ctx->prof = kinds;
  return VSR_OK;
}

extern "C" int vsr_profile_read(vsr_ctx *ctx, double *ms, int32_t *launches) {
  if (!ctx) return VSR_EINVAL;
  if (!ms || !launches) return ctx->fail(VSR_EINVAL, "profile_read: NULL output");
  for (int i = 0; i < VSR_STAGES; ++i) {
    ms[i] = 0.0;
    launches[i] = 0;
  }
  if (!ctx->recs.empty()) HIPCHECK(ctx, "profile sync", hipStreamSynchronize(ctx->stream));
  for (const auto &r : ctx->recs) {
    float t = 0.f;
    HIPCHECK(ctx, "hipEventElapsedTime", hipEventElapsedTime(&t, r.a, r.b));
    ms[r.stage] += t;
    launches[r.stage] += 1;
  }
  ctx->drop_records();
  return VSR_OK;
}
