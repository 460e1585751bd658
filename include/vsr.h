/*
 * vsr.h -- C ABI of the MI355X (gfx950) verifier scoring pass of
 * VideoSpeculateRAG (arxiv 2601.01513).
 *
 * The paper's verification stage (Section 3.1, Eq. 6-7) scores every drafted
 * answer a_i with the heavyweight verifier conditioned on the question and the
 * video, score_i = Verifier(Q, V, a_i), and selects a* = argmax_i score_i.
 * This library computes that pass for a decoder-only verifier:
 *
 *   vsr_prefill  runs the verifier once over the shared conditioning prefix
 *                [visual-frame rows ; text ids (retrieved passages + question)]
 *                and keeps every layer's rotated keys/values (the prefix cache);
 *   vsr_score    teacher-forces M candidates against that cache and returns
 *                lp[m][j] = log P(c_mj | prefix, c_m<j)   (j < n_m, else 0),
 *                score[m] = sum_j lp[m][j]                 (Eq. 6),
 *                argmax   = lowest m with the largest score (Eq. 7);
 *   vsr_verify   both in one pass (the prefix rows and the candidate rows
 *                share every projection launch), leaving the prefix cache
 *                as vsr_prefill does.
 *
 * Each candidate sees the prefix plus its own earlier tokens only (the drafts
 * are scored independently, Eq. 6); candidate token j sits at position P + j.
 *
 * Conventions shared by every call:
 *   - Device pointers are HIP device addresses on the device that was current
 *     at vsr_create. Host pointers are plain host memory. Each argument below
 *     says which it is.
 *   - Floating-point tensors are in the context's dtype (VSR_F32: float,
 *     VSR_BF16: bfloat16; the GEMM weights may instead be fp16, see
 *     gemm_weights); ids are int32; outputs are float / int32.
 *   - Matrices use the torch nn.Linear layout [out][in], rows contiguous.
 *   - Calls are asynchronous and ordered on the stream given to vsr_create:
 *     device outputs are valid once that stream has been synchronised.
 *   - Every call returns VSR_OK (0) or a negative code; vsr_last_error gives
 *     the message of the last failure. No call throws or aborts.
 *   - The library allocates no device memory: everything it keeps (prefix
 *     cache, activations, partial results) lives in the caller's workspace.
 *   - A context is not thread-safe; use one context per stream.
 */
#ifndef VSR_H
#define VSR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define VSR_OK 0
#define VSR_EINVAL (-1)  /* null pointer, bad shape, unsupported config   */
#define VSR_ESTATE (-2)  /* call out of order (e.g. score before prefill) */
#define VSR_ERANGE (-3)  /* a size exceeds the maxima given at create     */
#define VSR_ENOMEM (-4)  /* workspace smaller than vsr_workspace_size     */
#define VSR_EHIP (-5)    /* a HIP runtime call failed (message has text)  */
#define VSR_EID (-6)     /* checked call: an id outside [0, vocab) was read */
#define VSR_ENONFINITE (-7) /* checked call: a NaN or infinity in the results */

/* Arithmetic types of weights, visual rows and activations. */
#define VSR_F32 0
#define VSR_BF16 1
#define VSR_F16 2

/* Verifier architecture and the maxima the workspace is sized for.
 * Decoder: pre-RMSNorm blocks with rotary grouped-query attention (query head
 * h reads KV head h / (n_heads / n_kv_heads); rotate-half pairs (i, i+hd/2),
 * inverse frequency rope_base^(-2i/hd)) and a SwiGLU FFN, final RMSNorm and an
 * untied LM head; no biases.
 * Supported: n_heads % n_kv_heads == 0; VSR_BF16 needs head_dim == 128 and
 * d_model, d_ff multiples of 64; VSR_F32 needs head_dim even and <= 256. */
typedef struct vsr_config {
  int32_t n_layers, d_model, n_heads, n_kv_heads, head_dim, d_ff, vocab;
  float rms_eps, rope_base;
  int32_t dtype;        /* VSR_F32 or VSR_BF16 */
  int32_t max_prefix;   /* largest P = n_visual + n_text passed to prefill */
  int32_t max_cands;    /* largest M passed to score (<= VSR_MAX_CANDS)    */
  int32_t max_cand_len; /* largest Cmax passed to score                    */
  /* VSR_BF16 arithmetic: weights stay bf16 and are converted exactly to fp16
   * operands; activations are fp16 with fp32 accumulation. The first
   * split_layers decoder layers (0 <= split_layers <= n_layers) are precise
   * layers: every GEMM activation operand is carried as an fp16 value plus
   * its fp16 remainder (about 22 significant bits, twice the matrix-core
   * work), and attention carries queries, keys, values and probabilities the
   * same way (three products each, plus remainder caches of those layers in
   * the workspace): the earliest layers set the rounding that a deep decoder
   * amplifies. Ignored by VSR_F32 contexts (fp32 throughout). */
  int32_t split_layers;
  /* Storage type of the GEMM weights (wqkv, wo, wgu, wdown, lm_head) of a
   * VSR_BF16 context: 0 or VSR_BF16 (converted to fp16 inside the GEMMs) or
   * VSR_F16 (the bf16 values stored as fp16 by the caller, exact for
   * magnitudes >= 2^-17; loaded without conversion, about 6% faster GEMMs).
   * Embedding, norm gains and visual rows stay bf16. VSR_F32 contexts: 0. */
  int32_t gemm_weights;
  /* Largest number of tokens vsr_draft may generate per branch (0: no draft
   * cache in the workspace; vsr_draft then fails with VSR_ESTATE). The draft
   * cache holds every layer's keys/values of max_cands branches of
   * max_cand_len + max_new positions. 0 <= max_new <= 4096. */
  int32_t max_new;
  /* How many of the precise layers also carry their feed-forward block that
   * way (FFN RMSNorm output, gate/up products, SwiGLU output, down product;
   * 0 <= split_mlp_layers <= split_layers); the rest of the precise layers
   * split only their attention and its projections. Shallower decoders
   * amplify the FFN's fp16 rounding less: measured against the float32
   * oracle, a 28-layer 7B-class verifier with a plain FFN in its precise
   * layer stays at 8.4e-3 per token (limit 2e-2) and saves the FFN's doubled
   * matrix-core work, while a 64-layer one reaches 1.8e-2 and needs it split. */
  int32_t split_mlp_layers;
} vsr_config;

#define VSR_MAX_CANDS 256

/* Borrowed device pointers to the verifier weights (no copy is made; they
 * must outlive the context). The per-layer members are HOST arrays of
 * n_layers device pointers; they are copied at vsr_load_weights.
 *   embed, lm_head [vocab][d_model]; final_norm [d_model];
 *   attn_norm, ffn_norm [d_model];
 *   wqkv  [(n_heads + 2 n_kv_heads) head_dim][d_model]: q rows, then k rows,
 *         then v rows, each head-major;
 *   wo    [d_model][n_heads head_dim];
 *   wgu   [2 d_ff][d_model]: gate rows, then up rows;
 *   wdown [d_model][d_ff]. */
typedef struct vsr_weights {
  const void *embed, *lm_head, *final_norm;
  const void *const *attn_norm;
  const void *const *wqkv;
  const void *const *wo;
  const void *const *ffn_norm;
  const void *const *wgu;
  const void *const *wdown;
} vsr_weights;

typedef struct vsr_ctx vsr_ctx;

/* Bytes of device workspace a context with this config needs (0 if the
 * config is invalid). Pure host computation. */
size_t vsr_workspace_size(const vsr_config *cfg);

/* Creates a context. `workspace` is a device buffer of at least
 * vsr_workspace_size(cfg) bytes, 256-byte aligned, owned by the caller and
 * kept alive until vsr_destroy. `hip_stream` is a hipStream_t (NULL = the
 * default stream). On success *out receives the context. Enqueues the rotary
 * table construction on the stream. */
int vsr_create(const vsr_config *cfg, void *workspace, size_t ws_bytes,
               void *hip_stream, vsr_ctx **out);

/* Binds the weights (borrowed device pointers, layout above). */
int vsr_load_weights(vsr_ctx *ctx, const vsr_weights *w);

/* Prefill over the conditioning prefix (Eq. 6 conditions on (Q, V)).
 *   visual : device [n_visual][d_model] rows fed directly as layer-0 inputs
 *            (may be NULL when n_visual == 0);
 *   ids    : device [n_text] int32 text ids in [0, vocab) (may be NULL when
 *            n_text == 0); out-of-range ids are read as id 0 (VSR_EID
 *            under vsr_set_checks).
 * P = n_visual + n_text must satisfy 1 <= P <= max_prefix. Replaces any
 * earlier prefix. */
int vsr_prefill(vsr_ctx *ctx, const void *visual, int32_t n_visual,
                const int32_t *ids, int32_t n_text);

/* Teacher-forced scoring of M candidates against the current prefix
 * (Eq. 6-7). May be called any number of times after one prefill.
 *   cand_ids : device [M][Cmax] int32, row m holds candidate m's tokens in
 *              positions 0..cand_len[m]-1 (the rest is ignored);
 *              out-of-range ids are read as id 0 (VSR_EID under
 *              vsr_set_checks);
 *   cand_len : HOST [M] int32, each in [0, Cmax];
 *   logprobs : device [M][Cmax] float out; 0 past each candidate's length;
 *   scores   : device [M] float out, sum of each candidate's log-probs;
 *   argmax   : device [1] int32 out, lowest index among the largest scores.
 * 1 <= M <= max_cands, 1 <= Cmax <= max_cand_len. */
int vsr_score(vsr_ctx *ctx, const int32_t *cand_ids, const int32_t *cand_len,
              int32_t M, int32_t Cmax, float *logprobs, float *scores,
              int32_t *argmax);

/* vsr_prefill followed by vsr_score, computed as one pass (Section 3.1,
 * Eq. 6-7): the prefix rows and the candidate rows go through each
 * projection of each layer as one set of rows, so the candidates add rows to
 * the prefix's matrix products instead of running products of their own;
 * per layer the prefix rows attend causally over the prefix and each
 * candidate row over the prefix and its own earlier tokens, as in the two
 * calls. Arguments as vsr_prefill (visual, n_visual, ids, n_text) and
 * vsr_score (cand_ids .. argmax), with the same checks and errors; the
 * outputs agree with the two calls' to rounding (products of other row
 * groupings). On success the context holds the prefix cache, as after
 * vsr_prefill, for later vsr_score / vsr_reliability / vsr_draft calls. A
 * call rejected by its argument checks changes nothing; one that fails later
 * leaves no prefix current (like vsr_prefill). */
int vsr_verify(vsr_ctx *ctx, const void *visual, int32_t n_visual, const int32_t *ids,
               int32_t n_text, const int32_t *cand_ids, const int32_t *cand_len, int32_t M,
               int32_t Cmax, float *logprobs, float *scores, int32_t *argmax);

/* Stage 1 of the two-stage verification (Section 3.2, Eq. 11-13): the
 * reliability of M drafts against the current prefix. Branch m (the draft's
 * answer, entity and reasoning tokens followed by the verification prompt)
 * runs after the prefix at positions P.. exactly like a scored candidate;
 * at its last token the verifier's next-token distribution gives
 *   lp_yes_no[m] = (log p(yes_id), log p(no_id))            (Eq. 11)
 *   rel[m]       = p_yes / (p_yes + p_no)                   (Eq. 12)
 *   keep[m]      = rel[m] >= max_j rel[j] - delta ? 1 : 0   (Eq. 13, A_H)
 *   branch_ids : device [M][Cmax] int32 (out-of-range ids read as id 0);
 *   branch_len : HOST [M] int32, each in [1, Cmax] (a branch needs a last token);
 *   yes_id, no_id in [0, vocab); delta finite and >= 0;
 *   lp_yes_no  : device [M][2] float out; rel : device [M] float out;
 *   keep       : device [M] int32 out.
 * 1 <= M <= max_cands, 1 <= Cmax <= max_cand_len. Uses the same workspace
 * buffers as vsr_score (the two calls may be interleaved freely). */
int vsr_reliability(vsr_ctx *ctx, const int32_t *branch_ids, const int32_t *branch_len,
                    int32_t M, int32_t Cmax, int32_t yes_id, int32_t no_id, float delta,
                    float *lp_yes_no, float *rel, int32_t *keep);

/* Parallel draft generation over the shared prefix (Section 3.1, Eq. 5;
 * Section 3.2, Eq. 8-10): the context's model, used as the drafter, extends
 * every branch greedily. Branch m is the prefix followed by its prompt
 * (the retrieved document and the generation prompt, prompt_len[m] tokens at
 * positions P..); step s appends
 *   tokens[m][s] = argmax_v logits(last row of branch m)[v]
 * (lowest id among equal maxima) at the next position. Branches see the
 * prefix and their own tokens only; all of them advance together, one batched
 * pass per step, and the next step's inputs never leave the device.
 *   prompt_ids : device [M][Cmax] int32 (out-of-range ids read as id 0);
 *   prompt_len : HOST [M] int32, each in [1, Cmax];
 *   tokens     : device [M][n_new] int32 out.
 * 1 <= M <= max_cands, 1 <= Cmax <= max_cand_len, 1 <= n_new <= max_new;
 * needs a prefill. Keeps the branches' keys/values in the draft cache of the
 * workspace (overwritten by the next vsr_draft); vsr_score and
 * vsr_reliability may be called before or after it against the same prefix. */
int vsr_draft(vsr_ctx *ctx, const int32_t *prompt_ids, const int32_t *prompt_len, int32_t M,
              int32_t Cmax, int32_t n_new, int32_t *tokens);

/* Stage 2 and the final choice (Section 3.2, Eq. 14-15; Algorithm 1; the
 * strategies compared in Table 3). No context: the inputs are CLIP
 * embeddings, not verifier state.
 *   ent    : device [M][D] float, one entity embedding per draft;
 *   frames : device [NF][D] float, one embedding per keyframe;
 *   rel    : device [M] float, the drafts' reliability (Eq. 12);
 *   align  : device [M] float out, max_f cos(ent[m], frames[f]) (Eq. 14-15);
 *            a zero-norm row has similarity 0 with every row;
 *   choice : device [1] int32 out, the selected draft:
 *     VSR_SELECT_TWO_STAGE  argmax of align over A_H = {rel >= max rel - delta}
 *     VSR_SELECT_ADDITION   argmax of rel + align over all drafts
 *     VSR_SELECT_INVERT     argmax of rel over {align >= max align - delta}
 *   every argmax takes the lowest index among equal maxima.
 * 1 <= M <= VSR_MAX_CANDS, NF >= 1, 1 <= D <= 4096, delta finite and >= 0.
 * Enqueued on hip_stream (NULL = default stream). Errors are reported by
 * vsr_last_error(NULL). */
#define VSR_SELECT_TWO_STAGE 0
#define VSR_SELECT_ADDITION 1
#define VSR_SELECT_INVERT 2
int vsr_align_select(const float *ent, const float *frames, int32_t M, int32_t NF, int32_t D,
                     const float *rel, float delta, int32_t strategy, float *align,
                     int32_t *choice, void *hip_stream);

/* Message of the last failed call on this context ("" if none). With
 * ctx == NULL: message of the last failed context-free call on this thread
 * (vsr_create, vsr_align_select, vsr_weights_to_f16, vsr_keyframes,
 * vsr_retrieve, vsr_retrieve_static). */
const char *vsr_last_error(const vsr_ctx *ctx);

/* Keyframes of a video (Section 3.1, Eq. 1). Each frame is compared with the
 * frame before it through colour histograms (64 bins per RGB channel, bin =
 * value >> 2); the similarity is the histogram intersection
 * S[i] = sum over channels and bins of min(count_i, count_{i-1}), divided by
 * 3 H W. Frame 0 and every frame with S[i] < theta * 3 H W (decided in
 * float64) are keyframes.
 *   frames  : device uint8 [NF][H][W][3], 16-byte aligned;
 *   hist    : device int32 [NF][3][64] out, the per-frame counts;
 *   inter   : device int32 [NF] out, S[i] (S[0] = -1);
 *   key_idx : device int32 [NF] out, the keyframe indices in order;
 *   n_keys  : device int32 [1] out, their number (stays on the device).
 * 1 <= NF <= 65536, H, W >= 1, H W <= 2^24, theta finite. Enqueued on
 * hip_stream; errors via vsr_last_error(NULL). */
int vsr_keyframes(const uint8_t *frames, int32_t NF, int32_t H, int32_t W, float theta,
                  int32_t *hist, int32_t *inter, int32_t *key_idx, int32_t *n_keys,
                  void *hip_stream);

/* Bytes of device workspace vsr_retrieve needs (0 for invalid sizes). */
size_t vsr_retrieve_workspace_size(int32_t NF, int32_t ND, int32_t k);

/* Document retrieval for the keyframes (Section 3.1, Eq. 2-3). For keyframe
 * r (frame key_idx[r], r < n_keys) the k documents with the largest cosine
 * similarity of embeddings (Eq. 2), then T*: the K best documents of the
 * union of those lists, each scored by the best similarity it was retrieved
 * with (Eq. 3). Rankings break ties by the lower document index; a zero-norm
 * embedding has similarity 0 with everything.
 *   frame_emb : device float [NF][D] (embeddings of every frame);
 *   key_idx, n_keys : device, as written by vsr_keyframes;
 *   docs      : device float [ND][D], 16-byte aligned;
 *   workspace : device, >= vsr_retrieve_workspace_size(NF, ND, k) bytes,
 *               8-byte aligned, caller-owned;
 *   top_idx, top_sim : device [NF][k] out (rows r < n_keys written);
 *   sel_idx, sel_sim : device [K] out (the first n_sel entries written);
 *   n_sel     : device int32 [1] out, min(K, |T|).
 * 1 <= NF <= 65536, 1 <= ND <= 2^24, 1 <= D <= 1024, 1 <= k <= 16,
 * 1 <= K <= 64. Enqueued on hip_stream; errors via vsr_last_error(NULL). */
int vsr_retrieve(const float *frame_emb, const int32_t *key_idx, const int32_t *n_keys,
                 int32_t NF, const float *docs, int32_t ND, int32_t D, int32_t k, int32_t K,
                 void *workspace, size_t ws_bytes, int32_t *top_idx, float *top_sim,
                 int32_t *sel_idx, float *sel_sim, int32_t *n_sel, void *hip_stream);

/* vsr_retrieve for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same computation, arguments, outputs and errors as vsr_retrieve minus
 * the workspace. The per-chunk partial lists live in a library-owned static
 * device array of VSR_RETRIEVE_STATIC_BYTES (32 MiB) on each GPU the call runs
 * on (the current device), allocated with the library's code on that GPU and
 * held until the process ends; the call itself allocates nothing. Sizes whose
 * vsr_retrieve_workspace_size(NF, ND, k) exceeds it (e.g. more than 1M
 * documents at 220 keyframes and k = 3) fail with VSR_ERANGE. Every call on a
 * GPU shares that GPU's array: calls that overlap in time on one GPU (two
 * streams, or two host threads) race and must be serialised by the caller.
 * Device indices up to 63. */
#define VSR_RETRIEVE_STATIC_BYTES (32u << 20)
int vsr_retrieve_static(const float *frame_emb, const int32_t *key_idx, const int32_t *n_keys,
                        int32_t NF, const float *docs, int32_t ND, int32_t D, int32_t k,
                        int32_t K, int32_t *top_idx, float *top_sim, int32_t *sel_idx,
                        float *sel_sim, int32_t *n_sel, void *hip_stream);

/* Weight preparation for gemm_weights = VSR_F16: writes the n bf16 values of
 * src (device) to dst (device, n fp16 values, not overlapping src) with the
 * rounding the GEMMs apply to bf16 weights (exact for magnitudes in
 * [2^-17, 65504]; smaller ones truncate toward zero), so both weight forms
 * give bit-identical results. src and dst 16-byte aligned. Enqueued on
 * hip_stream (NULL = default); errors via vsr_last_error(NULL). */
int vsr_weights_to_f16(const void *src, void *dst, size_t n, void *hip_stream);

/* Call validator, off by default. With checks set, every later vsr_prefill,
 * vsr_score, vsr_verify, vsr_reliability and vsr_draft call on the context
 * clears a status word in the workspace before its launches, then waits for
 * its stream and reads the word once after them (the call becomes
 * synchronous), and returns
 *   VSR_EID        (VSR_CHECK_IDS) if a text, candidate, branch or prompt id
 *                  outside [0, vocab) was read; such ids are used as id 0,
 *                  checked or not, so the results are those of id 0;
 *   VSR_ENONFINITE (VSR_CHECK_FINITE) if a result is NaN or infinite: the
 *                  scores (vsr_score, vsr_verify), the Yes/No log-probs
 *                  (vsr_reliability) or the last prefix row's hidden state
 *                  (vsr_prefill). A NaN or infinite visual row, or an fp16
 *                  activation that overflows (|x| > 65504) on the bf16 path,
 *                  propagates to them.
 * VSR_EID is reported before VSR_ENONFINITE. Either way the outputs are
 * written as in an unchecked call and the prefix state changes as it would
 * on success. checks: an OR of the bits below (0 turns checking off). */
#define VSR_CHECK_IDS 1
#define VSR_CHECK_FINITE 2
int vsr_set_checks(vsr_ctx *ctx, int checks);

/* Releases the context (not the workspace or the weights). NULL is a no-op. */
void vsr_destroy(vsr_ctx *ctx);

/* ---- measurement (not part of the method) ----------------------------------
 * Per-stage kernel timing for benchmarks: while enabled, every stage launch of
 * vsr_prefill / vsr_score / vsr_reliability / vsr_draft / vsr_verify is
 * bracketed by HIP events on the context's stream. Stage s of the prefix pass
 * is s, of the candidate pass (score, reliability) VSR_STAGE_KINDS + s, of the
 * draft pass 2 VSR_STAGE_KINDS + s (there kind 9 is the LM head + chunk argmax
 * and kind 11 the greedy pick), of the fused pass of vsr_verify on bf16
 * contexts 3 VSR_STAGE_KINDS + s (there kind 3 is the prefix rows' attention,
 * kind 15 the candidate rows'; on fp32 contexts vsr_verify records prefix and
 * candidate passes);
 * kinds: 0 embedding, 1 RMSNorm, 2 QKV projection + rotary + cache write,
 * 3 attention, 4 attention merge, 5 output projection, 6 gate/up + SwiGLU,
 * 7 down projection, 8 LM-head inputs, 9 LM head + chunk LSE,
 * 10 LSE merge + target gather, 11 sum + argmax, 12 row tables, 13 copy,
 * 14 the prefix pass's last-row layer projections (O, gate/up, down),
 * 15 the candidate rows' attention of the fused pass. */
#define VSR_STAGE_KINDS 16
#define VSR_STAGES (4 * VSR_STAGE_KINDS)

/* Times the stage kinds whose bits are set in kinds (bit k: kind k, in all
 * passes; VSR_PROFILE_ALL: every kind; 0: timing off) and clears what was
 * recorded. Each timed launch adds two event records to the stream, so a
 * benchmark that times few kinds perturbs the pass least. */
#define VSR_PROFILE_ALL ((1 << VSR_STAGE_KINDS) - 1)
int vsr_profile_enable(vsr_ctx *ctx, int kinds);

/* Waits for the recorded launches, then writes, for every stage, the summed
 * kernel time in milliseconds (ms, HOST [VSR_STAGES]) and the number of
 * launches (launches, HOST [VSR_STAGES]) since the last read, and clears them. */
int vsr_profile_read(vsr_ctx *ctx, double *ms, int32_t *launches);

#ifdef __cplusplus
}
#endif
#endif /* VSR_H */
