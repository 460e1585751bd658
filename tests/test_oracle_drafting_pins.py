"""Pins of the draft-generation oracle (Section 3.1, Eq. 5; Section 3.2,
Eq. 8-10) against things other than itself (CPU only):

* an independent library decoder: transformers' Qwen2 greedy generation
  (`generate`, do_sample=False) from the same embedded prompt;
* the scoring path (Eq. 6), itself pinned to that decoder: under teacher
  forcing every greedy token has the largest log-prob of its step;
* incremental decoding equals full recomputation at every step;
* a closed form: with no layers the next token is argmax of the LM head on
  the normed embedding of the previous token;
* planted mistakes, which must break these pins.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import drafting as D
from tests.pin_cases import PIN, sharp_inputs
from tests.test_oracle_pins import _hf_model


def _prompt(seed=0, lens=(4, 1, 6)):
    return sharp_inputs(PIN, seed, lens=list(lens))


@pytest.mark.parametrize("seed", [0, 1])
def test_incremental_equals_recompute(seed):
    w, vis, pre, ids, lens = _prompt(seed)
    a = D.decode_shared(PIN, w, vis, pre, ids, lens, 6)
    b = D.decode_bruteforce(PIN, w, vis, pre, ids, lens, 6)
    np.testing.assert_array_equal(a, b)


def test_matches_transformers_greedy_generate():
    w, vis, pre, ids, lens = _prompt(2)
    model = _hf_model(PIN, w)
    e = np.asarray(w["embed"])
    n_new = 5
    ours = D.decode_shared(PIN, w, vis, pre, ids, lens, n_new)
    for m in range(PIN.n_cands):
        x = np.concatenate([vis, e[pre], e[ids[m, :lens[m]]]], axis=0)
        with torch.no_grad():
            gen = model.generate(inputs_embeds=torch.tensor(x)[None], max_new_tokens=n_new,
                                 do_sample=False, min_new_tokens=n_new, eos_token_id=None,
                                 pad_token_id=0)
        ref = gen[0, -n_new:].numpy()
        np.testing.assert_array_equal(ours[m], ref)


def test_greedy_tokens_have_the_largest_log_prob():
    """Teacher forcing through the Eq. 6 path: lp of each generated token is
    the maximum over the vocabulary at its step."""
    w, vis, pre, ids, lens = _prompt(3)
    n_new = 4
    toks = D.decode_shared(PIN, w, vis, pre, ids, lens, n_new)
    M, cmax = ids.shape
    ext = np.zeros((M, cmax + n_new), dtype=ids.dtype)
    for m in range(M):
        ext[m, :lens[m]] = ids[m, :lens[m]]
        ext[m, lens[m]:lens[m] + n_new] = toks[m]
    lp, _, _ = oracle.score_bruteforce(PIN, w, vis, pre, ext, np.asarray(lens) + n_new)
    for m in range(M):
        P = PIN.n_visual + len(pre)
        x = np.concatenate([vis, np.asarray(w["embed"])[pre],
                            np.asarray(w["embed"])[ext[m, :lens[m] + n_new]]], axis=0)
        h = oracle.forward_hidden(x, w, np.arange(len(x)), PIN, np.float64)
        full = oracle.token_log_probs(h, w, PIN, np.float64)
        for s in range(n_new):
            row = full[P + lens[m] - 1 + s]
            assert lp[m, lens[m] + s] == pytest.approx(row.max(), abs=1e-10)


def test_teacher_forced_report_is_consistent():
    w, vis, pre, ids, lens = _prompt(4)
    toks = D.decode_shared(PIN, w, vis, pre, ids, lens, 3)
    got, top, arg, gap = D.teacher_forced(PIN, w, vis, pre, ids, lens, toks)
    np.testing.assert_array_equal(arg, toks)
    np.testing.assert_allclose(got, top, rtol=0, atol=1e-12)
    assert np.all(gap >= 0)
    # a perturbed token is reported as such
    bad = toks.copy()
    bad[0, 1] = (bad[0, 1] + 1) % PIN.vocab
    got2, top2, _, _ = D.teacher_forced(PIN, w, vis, pre, ids, lens, bad)
    assert got2[0, 1] < top2[0, 1]


def test_shared_teacher_forcing_equals_per_branch_sequences():
    w, vis, pre, ids, lens = _prompt(8, lens=(3, 6, 1))
    toks = D.decode_bruteforce(PIN, w, vis, pre, ids, lens, 4)
    toks[1, 2] = (toks[1, 2] + 5) % PIN.vocab       # not the greedy path: still reported
    full = D.teacher_forced(PIN, w, vis, pre, ids, lens, toks)
    shared = D.teacher_forced_shared(PIN, w, vis, pre, ids, lens, toks)
    for a, b in zip(full, shared):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-10)
    part = D.teacher_forced_shared(PIN, w, vis, pre, ids, lens, toks, branches=[2])
    np.testing.assert_allclose(part[1][2], full[1][2], rtol=0, atol=1e-10)
    assert np.all(np.isnan(part[1][:2])) and np.all(part[2][:2] == -1)
    assert full[0][1, 2] < full[1][1, 2]


def test_no_layers_closed_form():
    cfg = PIN.replace(n_layers=0)
    w, vis, pre, ids, lens = sharp_inputs(cfg, 5, lens=[2, 3, 1])
    toks = D.decode_shared(cfg, w, vis, pre, ids, lens, 4)
    e, g, lm = np.asarray(w["embed"]), np.asarray(w["final_norm"]), np.asarray(w["lm_head"])

    def step(t):
        x = e[t]
        return int(np.argmax(lm @ (x / np.sqrt(np.mean(x * x) + cfg.rms_eps) * g)))
    for m in range(cfg.n_cands):
        t = int(ids[m, lens[m] - 1])
        for s in range(4):
            t = step(t)
            assert toks[m, s] == t


def test_ties_take_the_lowest_id():
    assert D.greedy(np.array([0.1, 0.7, 0.7, -1.0])) == 1


# --- planted mistakes ------------------------------------------------------------

def test_planted_position_reset_breaks_recompute_pin(monkeypatch):
    """New tokens placed at position P (instead of continuing the branch)."""
    w, vis, pre, ids, lens = _prompt(6)
    good = D.decode_bruteforce(PIN, w, vis, pre, ids, lens, 4)
    real = D.decoder_layer

    def shifted(x, lw, positions, cfg, dtype, past_k=None, past_v=None, past_pos=None):
        if past_k is not None and len(positions) == 1:
            positions = np.asarray([cfg.n_visual + len(pre)])
        return real(x, lw, positions, cfg, dtype, past_k, past_v, past_pos)
    monkeypatch.setattr(D, "decoder_layer", shifted)
    bad = D.decode_shared(PIN, w, vis, pre, ids, lens, 4)
    assert not np.array_equal(bad, good)


def test_planted_dropped_branch_cache_breaks_recompute_pin(monkeypatch):
    """Each step attending to the prefix only (the branch's own keys lost)."""
    w, vis, pre, ids, lens = _prompt(7, lens=(5, 4, 6))
    good = D.decode_bruteforce(PIN, w, vis, pre, ids, lens, 4)
    real = D.decoder_layer
    P = PIN.n_visual + len(pre)

    def forgetful(x, lw, positions, cfg, dtype, past_k=None, past_v=None, past_pos=None):
        if past_k is not None and len(positions) == 1:
            past_k, past_v, past_pos = past_k[:P], past_v[:P], past_pos[:P]
        return real(x, lw, positions, cfg, dtype, past_k, past_v, past_pos)
    monkeypatch.setattr(D, "decoder_layer", forgetful)
    bad = D.decode_shared(PIN, w, vis, pre, ids, lens, 4)
    assert not np.array_equal(bad, good)
