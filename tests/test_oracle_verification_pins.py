"""Pins of the two-stage verification oracle (Section 3.2, Eq. 11-15;
Algorithm 1; Table 3 strategies) against things other than itself (CPU only).

* the sequence-scoring path (Eq. 6), itself pinned against an independent
  library decoder: the Yes/No log-probs at a branch's last row equal the
  log-prob that scoring the branch extended by that token assigns to it;
* library routines (torch log_softmax, sigmoid, cosine_similarity);
* closed forms: a zero LM head gives 1/2; a one-layer-free decoder with a
  single non-zero LM-head row gives a logistic of one normed coordinate;
  collinear, orthogonal and basis-aligned embeddings; delta limits;
* small hand-worked selections for each strategy;
* planted mistakes, each of which must break one of these pins.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import verification as ov
from tests.pin_cases import PIN, sharp_inputs

YES, NO = 5, 11


def _branches(seed=0, lens=(4, 1, 6)):
    w, vis, pre, ids, lens = sharp_inputs(PIN, seed, lens=list(lens))
    return w, vis, pre, ids, lens


@pytest.mark.parametrize("seed", [0, 1])
def test_bruteforce_equals_shared_prefix(seed):
    w, vis, pre, ids, lens = _branches(seed)
    hb = ov.branch_last_hidden(PIN, w, vis, pre, ids, lens, mode="brute")
    hs = ov.branch_last_hidden(PIN, w, vis, pre, ids, lens, mode="shared")
    np.testing.assert_allclose(hs, hb, rtol=1e-10, atol=1e-10)


def test_yes_no_log_probs_agree_with_sequence_scoring():
    """Scoring branch (+) yes with Eq. 6 gives lp(yes | branch) as its last
    token log-prob; the same for no."""
    w, vis, pre, ids, lens = _branches(2)
    lp, _, _ = ov.reliability(PIN, w, vis, pre, ids, lens, YES, NO, 0.05)
    M, cmax = ids.shape
    for col, tok in ((0, YES), (1, NO)):
        ext = np.zeros((M, cmax + 1), dtype=ids.dtype)
        ext[:, :cmax] = ids
        for m in range(M):
            ext[m, lens[m]] = tok
        lp_seq, _, _ = oracle.score_bruteforce(PIN, w, vis, pre, ext, np.asarray(lens) + 1)
        got = [lp_seq[m, lens[m]] for m in range(M)]
        np.testing.assert_allclose(lp[:, col], got, rtol=1e-10, atol=1e-10)


def test_log_probs_match_torch_log_softmax():
    w, vis, pre, ids, lens = _branches(3)
    h = ov.branch_last_hidden(PIN, w, vis, pre, ids, lens)
    hn = torch.nn.functional.rms_norm(torch.tensor(h), (PIN.d_model,),
                                      torch.tensor(w["final_norm"]), PIN.rms_eps)
    ref = torch.log_softmax(hn @ torch.tensor(w["lm_head"]).T, dim=1).numpy()
    lp = ov.yes_no_log_probs(h, w, PIN, YES, NO, np.float64)
    np.testing.assert_allclose(lp, ref[:, [YES, NO]], rtol=1e-12, atol=1e-12)


def test_reliability_is_logistic_of_log_odds():
    rng = np.random.default_rng(4)
    lp = -rng.uniform(0.0, 30.0, size=(9, 2))
    rel, _ = ov.reliability_from_log_probs(lp, 0.05)
    ref = torch.sigmoid(torch.tensor(lp[:, 0] - lp[:, 1])).numpy()
    np.testing.assert_allclose(rel, ref, rtol=1e-12, atol=1e-14)


def test_zero_lm_head_gives_one_half():
    w, vis, pre, ids, lens = _branches(5)
    w = dict(w, lm_head=np.zeros_like(w["lm_head"]))
    lp, rel, keep = ov.reliability(PIN, w, vis, pre, ids, lens, YES, NO, 0.0)
    np.testing.assert_allclose(lp, -np.log(PIN.vocab), rtol=0, atol=1e-12)
    assert np.all(rel == 0.5) and np.all(keep)


def test_single_lm_head_row_closed_form():
    """No layers: the last row's hidden state is the embedding of the branch's
    last token; with only the yes row of W_lm non-zero (alpha e_k), the log-odds
    are alpha * norm(E[last])_k."""
    cfg = PIN.replace(n_layers=0)
    w, vis, pre, ids, lens = sharp_inputs(cfg, 6, lens=[3, 2, 5])
    k, alpha = 7, 2.5
    lm = np.zeros_like(w["lm_head"])
    lm[YES, k] = alpha
    w = dict(w, lm_head=lm)
    _, rel, _ = ov.reliability(cfg, w, vis, pre, ids, lens, YES, NO, 0.05)
    for m in range(cfg.n_cands):
        e = w["embed"][ids[m, lens[m] - 1]]
        normed = e / np.sqrt(np.mean(e * e) + cfg.rms_eps) * w["final_norm"]
        assert rel[m] == pytest.approx(1.0 / (1.0 + np.exp(-alpha * normed[k])), abs=1e-13)


def test_delta_limits():
    rel_lp = np.log(np.array([[0.2, 0.8], [0.7, 0.3], [0.7, 0.3], [0.65, 0.35]]))
    rel, keep = ov.reliability_from_log_probs(rel_lp, 0.0)
    np.testing.assert_allclose(rel, [0.2, 0.7, 0.7, 0.65], rtol=1e-12)
    assert keep.tolist() == [False, True, True, False]
    _, keep = ov.reliability_from_log_probs(rel_lp, 0.05)
    assert keep.tolist() == [False, True, True, True]
    _, keep = ov.reliability_from_log_probs(rel_lp, 1.0)
    assert keep.all()
    with pytest.raises(ValueError):
        ov.reliability_from_log_probs(rel_lp, -0.01)


def test_alignment_closed_forms():
    frames = np.eye(4)[:3] * np.array([[2.0], [0.5], [3.0]])  # basis rows, scaled
    ent = np.array([[3.0, 4.0, 0.0, 0.0],      # cos with f0 = 0.6, f1 = 0.8
                    [0.0, 0.0, 0.0, 1.0],      # orthogonal to every frame
                    [-1.0, 0.0, 0.0, 0.0],     # anti-parallel to f0
                    [0.0, 0.0, 7.0, 0.0]])     # parallel to f2
    a = ov.entity_alignment(ent, frames)
    np.testing.assert_allclose(a, [0.8, 0.0, 0.0, 1.0], rtol=0, atol=1e-15)


def test_zero_norm_rows_have_zero_similarity():
    frames = np.array([[0.0, 0.0, 0.0], [-1.0, 0.0, 0.0]])
    ent = np.array([[0.0, 0.0, 0.0], [1.0, 0.0, 0.0], [0.0, 2.0, 0.0]])
    # row 0: zero entity -> 0 with both; row 1: 0 (zero frame) vs -1 -> 0;
    # row 2: orthogonal to f1 -> 0.
    np.testing.assert_array_equal(ov.entity_alignment(ent, frames), [0.0, 0.0, 0.0])


def test_alignment_matches_torch_and_is_scale_invariant():
    rng = np.random.default_rng(7)
    ent, frames = rng.normal(size=(6, 32)), rng.normal(size=(10, 32))
    ref = torch.nn.functional.cosine_similarity(torch.tensor(ent)[:, None, :],
                                                torch.tensor(frames)[None, :, :], dim=2)
    a = ov.entity_alignment(ent, frames)
    np.testing.assert_allclose(a, ref.max(dim=1).values.numpy(), rtol=1e-12, atol=1e-12)
    scaled = ov.entity_alignment(ent * 3.0, frames * rng.uniform(0.1, 5.0, size=(10, 1)))
    np.testing.assert_allclose(scaled, a, rtol=1e-12, atol=1e-12)


def test_selection_strategies_hand_worked():
    rel = [0.90, 0.93, 0.50, 0.91]
    align = [0.80, 0.30, 0.99, 0.85]
    # A_H (delta 0.05): 0.90, 0.93, 0.91 >= 0.88 -> {0, 1, 3}; best alignment 3.
    assert ov.select_final(rel, align, 0.05, ov.TWO_STAGE) == 3
    # delta 0: only the most reliable draft remains.
    assert ov.select_final(rel, align, 0.0, ov.TWO_STAGE) == 1
    # large delta: plain argmax of the alignment.
    assert ov.select_final(rel, align, 1.0, ov.TWO_STAGE) == 2
    # addition: 1.70, 1.23, 1.49, 1.76 -> 3.
    assert ov.select_final(rel, align, 0.05, ov.ADDITION) == 3
    # invert: alignment filter >= 0.94 keeps {2}; then reliability -> 2.
    assert ov.select_final(rel, align, 0.05, ov.INVERT) == 2
    # invert with a wide margin: all kept, most reliable is 1.
    assert ov.select_final(rel, align, 1.0, ov.INVERT) == 1


def test_selection_ties_take_lowest_index():
    assert ov.select_final([0.5, 0.5, 0.5], [0.2, 0.7, 0.7], 0.0, ov.TWO_STAGE) == 1
    assert ov.select_final([0.4, 0.6], [0.6, 0.4], 0.0, ov.ADDITION) == 0
    assert ov.select_final([0.3, 0.3], [0.9, 0.9], 0.0, ov.INVERT) == 0


# --- planted mistakes -------------------------------------------------------------

def test_planted_ratio_mistakes_break_logistic_pin():
    rng = np.random.default_rng(8)
    lp = -rng.uniform(0.0, 10.0, size=(5, 2))
    ref = torch.sigmoid(torch.tensor(lp[:, 0] - lp[:, 1])).numpy()
    for fake in (lambda py, pn: py / (py + py),          # dropped term
                 lambda py, pn: pn / (py + pn),          # swapped yes / no
                 lambda py, pn: py / (1.0 + pn)):        # wrong denominator
        p_yes, p_no = np.exp(lp[:, 0]), np.exp(lp[:, 1])
        assert not np.allclose(fake(p_yes, p_no), ref, atol=1e-6)


def test_planted_wrong_row_breaks_sequence_pin(monkeypatch):
    """Reading the second-to-last branch row instead of the last one."""
    w, vis, pre, ids, lens = _branches(9, lens=(4, 3, 6))
    good, _, _ = ov.reliability(PIN, w, vis, pre, ids, lens, YES, NO, 0.05)
    real = ov.branch_last_hidden

    def shifted(cfg, weights, visual, prefix_ids, branch_ids, branch_len, dtype=np.float64,
                mode="shared", progress=None):
        lens2 = np.maximum(np.asarray(branch_len) - 1, 1)
        return real(cfg, weights, visual, prefix_ids, branch_ids, lens2, dtype, mode, progress)
    monkeypatch.setattr(ov, "branch_last_hidden", shifted)
    bad, _, _ = ov.reliability(PIN, w, vis, pre, ids, lens, YES, NO, 0.05)
    assert np.abs(bad - good).max() > 1e-3


def test_planted_missing_norm_breaks_alignment_pin():
    frames = np.eye(4)[:3] * np.array([[2.0], [0.5], [3.0]])
    ent = np.array([[3.0, 4.0, 0.0, 0.0]])
    unnormalised = (ent @ frames.T).max(axis=1)          # forgets the norms
    assert not np.allclose(unnormalised, [0.8])
    assert ov.entity_alignment(ent, frames)[0] == pytest.approx(0.8, abs=1e-15)
