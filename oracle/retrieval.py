"""Plain CPU oracle of the multimodal retrieval stage of VideoSpeculateRAG
(Section 3.1, "Multimodal Retrieval", Eq. 1-3).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.

Keyframes (Eq. 1). Every frame is compared with the frame before it through
colour histograms; a frame whose similarity falls below theta joins the
keyframe set F.

Retrieval (Eq. 2-3). Each keyframe retrieves its top-k documents by the
cosine similarity of CLIP embeddings; the retrieved documents form T, and
the top-K of T by similarity is T*, the knowledge passed to the drafters.

Readings where the paper is silent (shared with the HIP path):
  * histogram: 64 bins per RGB channel (value >> 2) of the uint8 frame;
    similarity = histogram intersection, sum over channels and bins of
    min(count_a, count_b), divided by 3 * H * W (1 for equal histograms,
    0 for disjoint ones); integer counts, so the test sum < theta * 3HW is
    decided exactly (compared in float64 on both sides);
  * frame 0 has no predecessor and is always a keyframe; frame i > 0 is
    compared with frame i - 1 (not with the last keyframe), as Eq. 1 states;
  * CLIP is out of scope: frame and document embeddings are inputs;
  * a zero-norm embedding has cosine 0 with everything;
  * a document's score in T is the best similarity it was retrieved with
    (the maximum over the keyframes whose top-k contain it); T* lists the K
    best of T by that score, fewer if |T| < K;
  * every ranking breaks ties by the lower document index.
Parity of the binning, the intersection measure and the T scoring is
unpinned by the paper (readings).
"""
from __future__ import annotations

from typing import List, Tuple

import numpy as np

BINS = 64  # per channel


def frame_histograms(frames: np.ndarray) -> np.ndarray:
    """Per-frame colour histograms: frames uint8 [NF][H][W][3] -> int64
    counts [NF][3][BINS] (bin = value >> 2)."""
    f = np.asarray(frames, dtype=np.uint8)
    nf = f.shape[0]
    out = np.zeros((nf, 3, BINS), dtype=np.int64)
    for i in range(nf):
        for c in range(3):
            out[i, c] = np.bincount((f[i, :, :, c] >> 2).ravel(), minlength=BINS)
    return out


def histogram_similarity(ha: np.ndarray, hb: np.ndarray, pixels: int) -> float:
    """Histogram intersection of two frames' [3][BINS] counts, in [0, 1]."""
    return float(np.minimum(ha, hb).sum()) / (3.0 * pixels)


def keyframes(frames: np.ndarray, theta: float) -> Tuple[np.ndarray, np.ndarray]:
    """Eq. 1. Returns (indices of the keyframes in order, intersection sums
    S[i] = sum min(h_i, h_{i-1}) for i >= 1 with S[0] = -1)."""
    h = frame_histograms(frames)
    nf = h.shape[0]
    hw = int(np.asarray(frames).shape[1]) * int(np.asarray(frames).shape[2])
    s = np.full(nf, -1, dtype=np.int64)
    keys: List[int] = [0] if nf else []
    for i in range(1, nf):
        s[i] = int(np.minimum(h[i], h[i - 1]).sum())
        if float(s[i]) < float(theta) * 3.0 * hw:   # sim(f_i, f_{i-1}) < theta
            keys.append(i)
    return np.asarray(keys, dtype=np.int64), s


def cosine_matrix(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """cos(a_i, b_j) for all rows (float64; 0 where a norm is 0) -- Eq. 2."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    num = a @ b.T
    den = np.outer(np.linalg.norm(a, axis=1), np.linalg.norm(b, axis=1))
    return np.divide(num, den, out=np.zeros_like(num), where=den > 0)


def top_indices(scores: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k largest scores, descending, ties to the lower index."""
    order = sorted(range(len(scores)), key=lambda j: (-scores[j], j))
    return np.asarray(order[:k], dtype=np.int64)


def retrieve(frame_emb: np.ndarray, key_idx: np.ndarray, doc_emb: np.ndarray, k: int,
             K: int):
    """Eq. 2-3 for the keyframes key_idx. Returns (per-keyframe top-k document
    indices [NK][k], their similarities [NK][k], T* indices [<=K], T* scores)."""
    sims = cosine_matrix(np.asarray(frame_emb)[np.asarray(key_idx, dtype=np.int64)], doc_emb)
    nk = sims.shape[0]
    kk = min(k, sims.shape[1])
    top = np.zeros((nk, kk), dtype=np.int64)
    top_s = np.zeros((nk, kk), dtype=np.float64)
    best = {}
    for r in range(nk):
        top[r] = top_indices(sims[r], kk)
        top_s[r] = sims[r, top[r]]
        for j, v in zip(top[r], top_s[r]):
            best[int(j)] = max(best.get(int(j), -np.inf), float(v))
    docs = sorted(best, key=lambda j: (-best[j], j))[:K]
    return top, top_s, np.asarray(docs, dtype=np.int64), np.asarray([best[j] for j in docs])
