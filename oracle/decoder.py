"""Plain CPU oracle of the verifier scoring pass of VideoSpeculateRAG.

TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the benchmark's
CPU-baseline leg import this module; the product path (the HIP library and its
binding) never does, and this module imports nothing from it.

What is computed (Section 3.1, Eq. 6-7; Algorithm 1 final selection):
  the verifier scores every drafted answer a_i against the shared conditioning
  (Q, V) and the highest-scoring draft is selected. The score is read as the
  verifier's teacher-forced sequence log-likelihood of the draft (the
  "self-consistent" strategy of Section 4.6, Table 3, which ranks drafts by
  the verifier's own likelihood and is sensitive to draft length, i.e. an
  unnormalised sum):

      lp[i][j]  = log softmax(W_lm . norm_f(h[P + j - 1]))[c_ij],  j < n_i
      score[i]  = sum_{j < n_i} lp[i][j]
      a*        = argmax_i score[i]   (lowest index among equal maxima)

  where h are the hidden states of a plain causal decoder run over the
  sequence  prefix (+) c_i,  prefix = [visual rows ; E[text ids]].

The decoder is the verifier architecture the workloads are shaped after
(Qwen2-style: pre-RMSNorm, rotary GQA attention, SwiGLU FFN, untied LM head).

Readings where the paper is silent (each is shared with the HIP path; the ones
marked "unpinned" are fixed by nothing but this reading):
  * score = sum of token log-probs, ties to the lowest index (Table 3
    discussion) -- sum vs mean: parity unpinned;
  * prefix order [visual rows][text ids], visual rows fed directly as layer-0
    inputs with no projector;
  * 1-D rotary positions: prefix 0..P-1, every candidate P..P+n_i-1;
    rotate-half pairing (i, i + hd/2), inverse frequency base^(-2i/hd);
  * query head h reads KV head floor(h / G);
  * q, k, v rows stacked head-major in one projection; gate rows then up rows
    (row order: parity unpinned);
  * no biases; untied LM head; RMSNorm eps 1e-6 (parity unpinned).

Arithmetic is float64 by default (the paper fixes no precision); pass
dtype=np.float32 for the plain-fp32 variant. Inputs may be float32 arrays
holding exact bf16 values. Weights are visited one layer at a time, so a
lazily fetched layer list streams them.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, List, Optional, Sequence

import numpy as np
from threadpoolctl import threadpool_limits

ROW_BLOCK = 1024  # query rows per attention block (bounds memory, not maths)
# Host threads for independent heads: the CPUs this process may use, at most
# the OpenMP thread count when one is set (a share of a larger machine).
THREADS = max(1, min(len(os.sched_getaffinity(0)),
                     int(os.environ.get("OMP_NUM_THREADS") or 1 << 30)))


def _c(a, dtype):
    return np.asarray(a, dtype=dtype)


def rms_norm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm of each row: x / sqrt(mean(x^2) + eps) * gain."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * gain


def rope_angles(positions: np.ndarray, head_dim: int, base: float) -> np.ndarray:
    """Rotation angle theta[p][i] = p * base^(-2i/hd) for i < hd/2 (float64)."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    inv_freq = base ** (-2.0 * i / head_dim)
    return np.outer(np.asarray(positions, dtype=np.float64), inv_freq)


def apply_rope(x: np.ndarray, positions: np.ndarray, base: float) -> np.ndarray:
    """Rotate each pair (x[i], x[i + hd/2]) of every head by theta[p][i].

    x is [n][H][hd]; positions is [n].
    """
    hd = x.shape[-1]
    half = hd // 2
    ang = rope_angles(positions, hd, base)
    cos = np.cos(ang).astype(x.dtype)[:, None, :]
    sin = np.sin(ang).astype(x.dtype)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def causal_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                     q_pos: np.ndarray, k_pos: np.ndarray) -> np.ndarray:
    """Scaled dot-product attention of one sequence with a causal mask.

    q [nq][Hq][hd]; k, v [nk][Hkv][hd]; a query at position p sees the keys
    whose position is <= p. Query head h reads KV head floor(h / G),
    G = Hq / Hkv. Softmax of q.k / sqrt(hd) over the visible keys.

    Queries are taken ROW_BLOCK rows at a time (memory only). A block's
    products are formed with the keys that at least one of its queries sees;
    a key hidden from every query of the block would get probability exactly
    0, so leaving it out changes nothing. Heads are independent and run on a
    pool of host threads (BLAS single-threaded inside it); each head's
    arithmetic is the same as in a loop over heads.
    """
    nq, hq, hd = q.shape
    hkv = k.shape[1]
    g = hq // hkv
    scale = 1.0 / math.sqrt(hd)
    out = np.empty_like(q)
    q_pos, k_pos = np.asarray(q_pos), np.asarray(k_pos)
    for r0 in range(0, nq, ROW_BLOCK):
        r1 = min(nq, r0 + ROW_BLOCK)
        seen = k_pos <= q_pos[r0:r1].max()
        kb, vb = k[seen], v[seen]
        hidden = k_pos[seen][None, :] > q_pos[r0:r1, None]

        def one_head(h):
            kh = h // g
            s = q[r0:r1, h, :] @ kb[:, kh, :].T
            s *= scale
            np.putmask(s, hidden, -np.inf)
            s -= s.max(axis=1, keepdims=True)
            np.exp(s, out=s)
            s /= s.sum(axis=1, keepdims=True)
            out[r0:r1, h, :] = s @ vb[:, kh, :]
        with threadpool_limits(1, user_api="blas"), ThreadPoolExecutor(min(hq, THREADS)) as ex:
            list(ex.map(one_head, range(hq)))
    return out


def silu(x: np.ndarray) -> np.ndarray:
    """x * sigmoid(x)."""
    with np.errstate(over="ignore"):
        return x / (1.0 + np.exp(-x))


def decoder_layer(x, lw: Dict, positions, cfg, dtype,
                  past_k=None, past_v=None, past_pos=None):
    """One pre-norm decoder block over the rows `x` ([n][d]).

    Keys of this call are its own rows plus, if given, `past_*` (the cached
    keys/values of earlier positions of the same sequence, already rotated).
    Returns (new x, this call's rotated keys, values).
    """
    n = x.shape[0]
    hq, hkv, hd, f = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_ff
    h = rms_norm(x, _c(lw["attn_norm"], dtype), cfg.rms_eps)
    qkv = h @ _c(lw["wqkv"], dtype).T
    q = qkv[:, :hq * hd].reshape(n, hq, hd)
    k = qkv[:, hq * hd:(hq + hkv) * hd].reshape(n, hkv, hd)
    v = qkv[:, (hq + hkv) * hd:].reshape(n, hkv, hd)
    q = apply_rope(q, positions, cfg.rope_base)
    k = apply_rope(k, positions, cfg.rope_base)
    if past_k is not None:
        keys = np.concatenate([past_k, k], axis=0)
        vals = np.concatenate([past_v, v], axis=0)
        kpos = np.concatenate([past_pos, positions])
    else:
        keys, vals, kpos = k, v, positions
    a = causal_attention(q, keys, vals, positions, kpos)
    x = x + a.reshape(n, hq * hd) @ _c(lw["wo"], dtype).T
    h = rms_norm(x, _c(lw["ffn_norm"], dtype), cfg.rms_eps)
    gu = h @ _c(lw["wgu"], dtype).T
    x = x + (silu(gu[:, :f]) * gu[:, f:]) @ _c(lw["wdown"], dtype).T
    return x, k, v


def embed_prefix(weights: Dict, visual, prefix_ids, dtype) -> np.ndarray:
    """Layer-0 inputs of the prefix: the visual rows, then E[text ids]."""
    e = _c(weights["embed"], dtype)
    return np.concatenate([_c(visual, dtype), e[np.asarray(prefix_ids)]], axis=0)


def forward_hidden(x: np.ndarray, weights: Dict, positions, cfg, dtype):
    """Final hidden states (before the final norm) of one causal sequence."""
    for lw in weights["layers"]:
        x, _, _ = decoder_layer(x, lw, positions, cfg, dtype)
    return x


def token_log_probs(h: np.ndarray, weights: Dict, cfg, dtype) -> np.ndarray:
    """Full log-softmax rows over the vocabulary for hidden rows h [n][d]."""
    hn = rms_norm(h, _c(weights["final_norm"], dtype), cfg.rms_eps)
    logits = hn @ _c(weights["lm_head"], dtype).T
    mx = logits.max(axis=1, keepdims=True)
    lse = mx + np.log(np.exp(logits - mx).sum(axis=1, keepdims=True))
    return logits - lse


def select(scores: Sequence[float]) -> int:
    """Eq. 7: index of the highest score; the lowest index among equal maxima."""
    best = 0
    for i in range(1, len(scores)):
        if scores[i] > scores[best]:
            best = i
    return best


def _gather_lp(h_rows, weights, cfg, dtype, ids):
    lp = token_log_probs(h_rows, weights, cfg, dtype)
    return lp[np.arange(len(ids)), np.asarray(ids)]


def score_bruteforce(cfg, weights: Dict, visual, prefix_ids, cand_ids, cand_len,
                     dtype=np.float64):
    """Definition mode: each candidate runs as its own full sequence.

    Returns (lp [M][Cmax] with zeros past each length, score [M], argmax).
    """
    P = cfg.n_visual + len(prefix_ids)
    M, cmax = np.asarray(cand_ids).shape
    x_pre = embed_prefix(weights, visual, prefix_ids, dtype)
    e = _c(weights["embed"], dtype)
    lp = np.zeros((M, cmax), dtype=dtype)
    for m in range(M):
        n = int(cand_len[m])
        ids = np.asarray(cand_ids[m, :n])
        x = np.concatenate([x_pre, e[ids]], axis=0)
        h = forward_hidden(x, weights, np.arange(P + n), cfg, dtype)
        # Row P-1+j predicts candidate token j (row P-1 is the last prefix row).
        lp[m, :n] = _gather_lp(h[P - 1:P - 1 + n], weights, cfg, dtype, ids)
    scores = lp.sum(axis=1)
    return lp, scores, select(scores)


def score_shared_prefix(cfg, weights: Dict, visual, prefix_ids, cand_ids, cand_len,
                        dtype=np.float64, cands: Optional[List[int]] = None,
                        progress=None):
    """Shared-prefix mode: the prefix is run once, each layer's rotated prefix
    keys/values are reused by every candidate. Exactly the definition above
    re-associated (a candidate token's visible keys are the prefix keys plus
    its own earlier tokens, as in one full causal sequence).

    `cands` restricts the work to some candidates (the others get lp = 0 and
    score = nan); `progress(layer)` is called after each layer.
    Returns (lp, score, argmax or -1 if restricted).
    """
    P = cfg.n_visual + len(prefix_ids)
    M, cmax = np.asarray(cand_ids).shape
    todo = list(range(M)) if cands is None else list(cands)
    e = _c(weights["embed"], dtype)
    x_pre = embed_prefix(weights, visual, prefix_ids, dtype)
    pos_pre = np.arange(P)
    xs = {m: e[np.asarray(cand_ids[m, :int(cand_len[m])])] for m in todo}
    for li, lw in enumerate(weights["layers"]):
        x_next, kp, vp = decoder_layer(x_pre, lw, pos_pre, cfg, dtype)
        for m in todo:
            n = xs[m].shape[0]
            if n:
                xs[m], _, _ = decoder_layer(xs[m], lw, P + np.arange(n), cfg, dtype,
                                            kp, vp, pos_pre)
        x_pre = x_next
        if progress is not None:
            progress(li)
    lp = np.zeros((M, cmax), dtype=dtype)
    scores = np.full(M, np.nan, dtype=dtype)
    for m in todo:
        n = int(cand_len[m])
        if n:
            rows = np.concatenate([x_pre[P - 1:P], xs[m][:n - 1]], axis=0)
            lp[m, :n] = _gather_lp(rows, weights, cfg, dtype, cand_ids[m, :n])
        scores[m] = lp[m].sum()
    best = select(scores) if cands is None else -1
    return lp, scores, best
