"""Plain CPU oracle of the two-stage verification of VideoSpeculateRAG
(Section 3.2, two-stage verification, Eq. 11-15; Algorithm 1 final selection;
Table 3 strategies of Section 4.6).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.

Stage 1, reliability (Eq. 11-13). The verifier reads the shared conditioning
(Q, V) followed by one branch per draft: the draft's answer, entity and
reasoning and a fixed verification prompt (all given here as token ids). The
distribution of the first token it would generate is the softmax at the
branch's last row; with p_yes and p_no the probabilities of the "Yes" and
"No" tokens there,

    rel[i]  = p_yes[i] / (p_yes[i] + p_no[i])                      (Eq. 12)
    A_H     = { i : rel[i] >= max_j rel[j] - delta }                (Eq. 13)

Stage 2, entity alignment (Eq. 14-15). With CLIP embeddings of each draft's
entity ent[i] and of the keyframes frames[f] (inputs here; CLIP itself is
not part of this work),

    sim[i][f] = cos(ent[i], frames[f])                              (Eq. 14)
    align[i]  = max_f sim[i][f]                                     (Eq. 15)
    a*        = argmax_{i in A_H} align[i]                          (Algorithm 1)

Table 3 compares selection strategies: "addition" ranks all drafts by
rel + align, "invert" swaps the stages (filter by alignment with the same
margin, then rank by reliability); "self-consistent" is the sequence
log-likelihood of Eq. 6-7 (decoder.score_*). Every argmax takes the lowest
index among equal maxima.

Readings (shared with the HIP path): the branch's own tokens follow the
prefix at positions P.. like a scored candidate; a branch has at least one
token; delta >= 0; "invert" uses the same delta as its margin (parity of that
reading unpinned: the paper gives no threshold for it); a zero-norm embedding
has cosine similarity 0 with everything (the paper's cosine is undefined there).
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence

import numpy as np

from .decoder import (_c, decoder_layer, embed_prefix, forward_hidden, rms_norm, select)

TWO_STAGE = "two_stage"
ADDITION = "addition"
INVERT = "invert"


def yes_no_log_probs(h_last: np.ndarray, weights: Dict, cfg, yes_id: int, no_id: int,
                     dtype) -> np.ndarray:
    """log p(yes), log p(no) of the next token after hidden rows h_last [M][d]
    (Eq. 11: the full softmax over the vocabulary)."""
    hn = rms_norm(h_last, _c(weights["final_norm"], dtype), cfg.rms_eps)
    logits = hn @ _c(weights["lm_head"], dtype).T
    mx = logits.max(axis=1, keepdims=True)
    lse = mx + np.log(np.exp(logits - mx).sum(axis=1, keepdims=True))
    lp = logits - lse
    return np.stack([lp[:, yes_id], lp[:, no_id]], axis=1)


def branch_last_hidden(cfg, weights: Dict, visual, prefix_ids, branch_ids, branch_len,
                       dtype=np.float64, mode: str = "shared", progress=None) -> np.ndarray:
    """Final hidden state (before the final norm) of each branch's last token.

    mode "brute": every branch runs as its own full causal sequence
    prefix (+) branch; mode "shared": the prefix runs once and each layer's
    rotated prefix keys/values serve every branch (the same result
    re-associated)."""
    P = cfg.n_visual + len(prefix_ids)
    M = len(branch_len)
    e = _c(weights["embed"], dtype)
    x_pre = embed_prefix(weights, visual, prefix_ids, dtype)
    out = np.zeros((M, cfg.d_model), dtype=dtype)
    lens = [int(n) for n in branch_len]
    if min(lens) < 1:
        raise ValueError("every branch needs at least one token")
    if mode == "brute":
        for m in range(M):
            x = np.concatenate([x_pre, e[np.asarray(branch_ids[m, :lens[m]])]], axis=0)
            h = forward_hidden(x, weights, np.arange(P + lens[m]), cfg, dtype)
            out[m] = h[-1]
        return out
    xs = [e[np.asarray(branch_ids[m, :lens[m]])] for m in range(M)]
    pos_pre = np.arange(P)
    for li, lw in enumerate(weights["layers"]):
        x_next, kp, vp = decoder_layer(x_pre, lw, pos_pre, cfg, dtype)
        for m in range(M):
            xs[m], _, _ = decoder_layer(xs[m], lw, P + np.arange(lens[m]), cfg, dtype,
                                        kp, vp, pos_pre)
        x_pre = x_next
        if progress is not None:
            progress(li)
    for m in range(M):
        out[m] = xs[m][-1]
    return out


def reliability_from_log_probs(lp_yes_no: np.ndarray, delta: float):
    """Eq. 12 and Eq. 13 from per-branch (log p_yes, log p_no)."""
    if not delta >= 0.0:
        raise ValueError("delta must be >= 0")
    p_yes = np.exp(lp_yes_no[:, 0])
    p_no = np.exp(lp_yes_no[:, 1])
    rel = p_yes / (p_yes + p_no)
    keep = rel >= rel.max() - delta
    return rel, keep


def reliability(cfg, weights: Dict, visual, prefix_ids, branch_ids, branch_len, yes_id: int,
                no_id: int, delta: float, dtype=np.float64, mode: str = "shared",
                progress=None):
    """Stage 1 (Eq. 11-13). Returns (lp_yes_no [M][2], rel [M], keep [M] bool)."""
    h = branch_last_hidden(cfg, weights, visual, prefix_ids, branch_ids, branch_len, dtype,
                           mode, progress)
    lp = yes_no_log_probs(h, weights, cfg, yes_id, no_id, dtype)
    rel, keep = reliability_from_log_probs(lp, delta)
    return lp, rel, keep


def entity_alignment(ent, frames) -> np.ndarray:
    """Eq. 14-15: for each entity row, the largest cosine similarity with any
    frame row (float64). A zero-norm row has similarity 0 with every row."""
    e = np.asarray(ent, dtype=np.float64)
    f = np.asarray(frames, dtype=np.float64)
    num = e @ f.T
    den = np.outer(np.linalg.norm(e, axis=1), np.linalg.norm(f, axis=1))
    sim = np.divide(num, den, out=np.zeros_like(num), where=den > 0)
    return sim.max(axis=1)


def _argmax_within(values: Sequence[float], allowed: Sequence[bool]) -> int:
    best = -1
    for i, (v, ok) in enumerate(zip(values, allowed)):
        if ok and (best < 0 or v > values[best]):
            best = i
    return best


def select_final(rel, align, delta: float, strategy: str = TWO_STAGE) -> int:
    """Final answer index under one of the Table 3 strategies (lowest index
    among equal maxima)."""
    rel = np.asarray(rel, dtype=np.float64)
    align = np.asarray(align, dtype=np.float64)
    if strategy == TWO_STAGE:
        keep = rel >= rel.max() - delta
        return _argmax_within(align, keep)
    if strategy == ADDITION:
        return select(rel + align)
    if strategy == INVERT:
        keep = align >= align.max() - delta
        return _argmax_within(rel, keep)
    raise ValueError(f"unknown strategy {strategy!r}")
