"""Plain CPU oracle of the parallel draft generation of VideoSpeculateRAG
(Section 3.1, "Speculate Generation", Eq. 5; Section 3.2, Eq. 8-10).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.

Each retrieved document t_i starts its own branch after the shared
conditioning (Q, V); a light drafter model continues every branch greedily
and in parallel, so that one set of drafts A_draft comes out of one batched
decode (Eq. 5). Eq. 8-10 chain three such generations (entity, reasoning,
answer) through text prompts; at the level of the model each is the same
operation: extend a branch of given tokens by n new tokens.

    branch m = prefix (+) prompt_m (+) g_m[0] (+) ... (+) g_m[n-1]
    g_m[s]   = argmax_v logits(h at the position before g_m[s])[v]

Readings (shared with the HIP path): greedy decoding (the paper names no
sampling); ties take the lowest token id; positions continue the branch
(prefix 0..P-1, prompt P..P+n_m-1, new tokens after it); every prompt has at
least one token; generation runs a fixed number of steps (random weights have
no end-of-sequence behaviour worth modelling).
"""
from __future__ import annotations

from typing import Dict, List, Optional

import numpy as np

from .decoder import _c, decoder_layer, embed_prefix, forward_hidden, rms_norm


def next_token_logits(h: np.ndarray, weights: Dict, cfg, dtype) -> np.ndarray:
    """Logits over the vocabulary for hidden rows h [n][d]."""
    hn = rms_norm(h, _c(weights["final_norm"], dtype), cfg.rms_eps)
    return hn @ _c(weights["lm_head"], dtype).T


def greedy(logits: np.ndarray) -> int:
    """argmax with ties to the lowest id."""
    return int(np.argmax(logits))


def decode_bruteforce(cfg, weights: Dict, visual, prefix_ids, prompt_ids, prompt_len,
                      n_new: int, dtype=np.float64) -> np.ndarray:
    """Definition mode: every step reruns the whole sequence."""
    P = cfg.n_visual + len(prefix_ids)
    M = len(prompt_len)
    e = _c(weights["embed"], dtype)
    x_pre = embed_prefix(weights, visual, prefix_ids, dtype)
    out = np.zeros((M, n_new), dtype=np.int64)
    for m in range(M):
        toks = [int(t) for t in np.asarray(prompt_ids[m, :int(prompt_len[m])])]
        if not toks:
            raise ValueError("every prompt needs at least one token")
        for s in range(n_new):
            x = np.concatenate([x_pre, e[np.asarray(toks)]], axis=0)
            h = forward_hidden(x, weights, np.arange(P + len(toks)), cfg, dtype)
            nxt = greedy(next_token_logits(h[-1:], weights, cfg, dtype)[0])
            out[m, s] = nxt
            toks.append(nxt)
    return out


def decode_shared(cfg, weights: Dict, visual, prefix_ids, prompt_ids, prompt_len, n_new: int,
                  dtype=np.float64, progress=None) -> np.ndarray:
    """Incremental mode: the prefix runs once; each branch keeps every layer's
    rotated keys/values of its prompt and generated tokens and extends them
    one token per step (the same result re-associated)."""
    P = cfg.n_visual + len(prefix_ids)
    M = len(prompt_len)
    L = len(weights["layers"])
    e = _c(weights["embed"], dtype)
    x_pre = embed_prefix(weights, visual, prefix_ids, dtype)
    pos_pre = np.arange(P)
    lens = [int(n) for n in prompt_len]
    if min(lens) < 1:
        raise ValueError("every prompt needs at least one token")
    # Prefix keys/values per layer.
    pk, pv = [], []
    for lw in weights["layers"]:
        x_pre, k, v = decoder_layer(x_pre, lw, pos_pre, cfg, dtype)
        pk.append(k)
        pv.append(v)
    out = np.zeros((M, n_new), dtype=np.int64)
    for m in range(M):
        bk, bv = [None] * L, [None] * L
        x = e[np.asarray(prompt_ids[m, :lens[m]])]
        pos = P + np.arange(lens[m])
        for s in range(n_new):
            # The rows of this step (the prompt, then the last new token)
            # through every layer, keeping their keys/values.
            for li, lw in enumerate(weights["layers"]):
                past_k = pk[li] if bk[li] is None else np.concatenate([pk[li], bk[li]])
                past_v = pv[li] if bv[li] is None else np.concatenate([pv[li], bv[li]])
                past_p = np.arange(P + (0 if bk[li] is None else bk[li].shape[0]))
                x, k, v = decoder_layer(x, lw, pos, cfg, dtype, past_k, past_v, past_p)
                bk[li] = k if bk[li] is None else np.concatenate([bk[li], k])
                bv[li] = v if bv[li] is None else np.concatenate([bv[li], v])
            nxt = greedy(next_token_logits(x[-1:], weights, cfg, dtype)[0])
            out[m, s] = nxt
            x = e[np.asarray([nxt])]
            pos = np.asarray([P + lens[m] + s])
        if progress is not None:
            progress(m)
    return out


def teacher_forced(cfg, weights: Dict, visual, prefix_ids, prompt_ids, prompt_len, tokens,
                   dtype=np.float64):
    """Given generated tokens [M][n], the logits that predicted each of them
    (prefix (+) prompt (+) tokens run as one sequence). Returns, per (m, s):
    the logit of tokens[m][s], the largest logit, the argmax and the gap
    between the largest and second-largest logits."""
    P = cfg.n_visual + len(prefix_ids)
    M, n = np.asarray(tokens).shape
    e = _c(weights["embed"], dtype)
    x_pre = embed_prefix(weights, visual, prefix_ids, dtype)
    got = np.zeros((M, n), dtype=dtype)
    top = np.zeros((M, n), dtype=dtype)
    arg = np.zeros((M, n), dtype=np.int64)
    gap = np.zeros((M, n), dtype=dtype)
    for m in range(M):
        pl = int(prompt_len[m])
        toks = np.concatenate([np.asarray(prompt_ids[m, :pl]), np.asarray(tokens[m])])
        x = np.concatenate([x_pre, e[toks]], axis=0)
        h = forward_hidden(x, weights, np.arange(P + len(toks)), cfg, dtype)
        lg = next_token_logits(h[P + pl - 1:P + pl - 1 + n], weights, cfg, dtype)
        got[m], top[m], arg[m], gap[m] = _report(lg, tokens[m], dtype)
    return got, top, arg, gap


def _report(lg: np.ndarray, tokens, dtype):
    """Per row of logits lg [n][V] and the chosen tokens [n]: (logit of the
    token, largest logit, argmax, gap between the two largest logits)."""
    n = lg.shape[0]
    got, top, gap = (np.zeros(n, dtype=dtype) for _ in range(3))
    arg = np.zeros(n, dtype=np.int64)
    for s in range(n):
        row = lg[s]
        a = greedy(row)
        srt = np.partition(row, -2)[-2:]
        got[s], top[s], arg[s], gap[s] = row[int(tokens[s])], row[a], a, srt[1] - srt[0]
    return got, top, arg, gap


def teacher_forced_shared(cfg, weights: Dict, visual, prefix_ids, prompt_ids, prompt_len,
                          tokens, dtype=np.float64, branches: Optional[List[int]] = None,
                          progress=None):
    """teacher_forced with the prefix run once per layer and its keys/values
    reused by every branch (the same result re-associated), restricted to
    `branches` (the other rows are nan / -1); progress(layer) after each
    layer. Branch m runs prompt_m (+) tokens[m][:n-1]: the rows that predict
    tokens[m][0..n-1]."""
    P = cfg.n_visual + len(prefix_ids)
    tokens = np.asarray(tokens)
    M, n = tokens.shape
    todo = list(range(M)) if branches is None else list(branches)
    e = _c(weights["embed"], dtype)
    x_pre = embed_prefix(weights, visual, prefix_ids, dtype)
    pos_pre = np.arange(P)
    xs = {}
    for m in todo:
        pl = int(prompt_len[m])
        xs[m] = e[np.concatenate([np.asarray(prompt_ids[m, :pl]), tokens[m, :n - 1]])]
    for li, lw in enumerate(weights["layers"]):
        x_next, kp, vp = decoder_layer(x_pre, lw, pos_pre, cfg, dtype)
        for m in todo:
            xs[m], _, _ = decoder_layer(xs[m], lw, P + np.arange(xs[m].shape[0]), cfg, dtype,
                                        kp, vp, pos_pre)
        x_pre = x_next
        if progress is not None:
            progress(li)
    got, top, gap = (np.full((M, n), np.nan, dtype=dtype) for _ in range(3))
    arg = np.full((M, n), -1, dtype=np.int64)
    for m in todo:
        pl = int(prompt_len[m])
        lg = next_token_logits(xs[m][pl - 1:pl - 1 + n], weights, cfg, dtype)
        got[m], top[m], arg[m], gap[m] = _report(lg, tokens[m], dtype)
    return got, top, arg, gap
