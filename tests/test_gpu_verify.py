"""GPU parity of vsr_verify, the prefix pass and the candidate pass fused
into one set of rows per projection (Section 3.1, Eq. 6-7), against the CPU
oracle on the same seeded inputs, with the tolerances of the scoring pass
(per-token log-prob 2e-2 for bf16, 1e-4 for fp32; score 1e-2 relative;
argmax where the oracle's top-2 margin exceeds 0.1).

Cases: small bf16 shapes with ragged and empty candidates and none, some or
all layers precise; seven query heads per KV head; a pass small enough
(prefix + candidate rows <= 32) for the few-row kernels; a one-row prefix
with one one-token candidate, and with candidates inside one row tile; the fp32 and
no-candidate-token fallbacks; the prefix state it leaves for later calls;
argument errors; candidate tokens at the end of the vocabulary (the LM head's
partial last tile). The full-size 7B-class pass (the benchmark's) is checked in
test_gpu_parity.py next to the two-call pass.
"""
import sys

import numpy as np
import pytest

from paper_2601_01513_amd import workload as W
from test_gpu_parity import (GQA7_BF16, SMALL_BF16, _case, _torch, check, run_gpu,
                             run_gpu_verify, run_oracle)

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, file=sys.stderr, flush=True)


@pytest.mark.parametrize("seed,split", [(0, 0), (1, 1), (2, 2)])
def test_verify_small_bf16_ragged(seed, split):
    wl = _case(SMALL_BF16, seed, lens=[40, 1, 0, 23, 37], split=split)
    fused = run_gpu_verify(wl, split_layers=split)
    check(wl.cfg, fused, run_oracle(wl), wl.cand_len)


@pytest.mark.parametrize("seed,split", [(0, 0), (1, 1)])
def test_verify_gqa7(seed, split):
    wl = _case(GQA7_BF16, seed, split=split)
    check(wl.cfg, run_gpu_verify(wl, split_layers=split), run_oracle(wl), wl.cand_len)


def test_verify_targets_at_the_vocabulary_end():
    """Candidate tokens among the last 300 vocabulary entries (vocab 1000: the
    LM head's last 256-entry tile is partial), so the target logits come
    from the partial tile and the full one before it, at every row offset."""
    wl = _case(SMALL_BF16, 4, lens=[40, 17, 33, 40, 9])
    vocab = wl.cfg.vocab
    k = np.arange(wl.cand_ids.size).reshape(wl.cand_ids.shape)
    wl.cand_ids = (vocab - 1 - (k * 7) % 300).astype(wl.cand_ids.dtype)
    for m, n in enumerate(wl.cand_len):
        wl.cand_ids[m, n:] = 0
    check(wl.cfg, run_gpu_verify(wl), run_oracle(wl), wl.cand_len)


def test_verify_agrees_with_prefill_and_score():
    """Same kernels, other row groupings in the products: the two paths agree
    to rounding, and both with the oracle."""
    wl = _case(SMALL_BF16, 3, lens=[40, 12, 5, 33, 1], split=1)
    two = run_gpu(wl, split_layers=1)
    fused = run_gpu_verify(wl, verifier=two[3])
    ora = run_oracle(wl)
    check(wl.cfg, two, ora, wl.cand_len)
    check(wl.cfg, fused, ora, wl.cand_len)
    valid = np.arange(two[0].shape[1])[None, :] < np.asarray(wl.cand_len)[:, None]
    d = np.abs(two[0] - fused[0])[valid].max()
    _say(f"  max |dlp| between the two paths: {d:.3e}")
    assert d <= 2e-2


def test_verify_is_deterministic():
    """Fixed-order reductions everywhere: two passes on the same inputs are
    bitwise equal (GQA-7, 8 x 64 ragged candidates, one precise layer)."""
    wl = _case(GQA7_BF16, 2, split=1)
    a = run_gpu_verify(wl, split_layers=1)
    b = run_gpu_verify(wl, verifier=a[3])
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]) and a[2] == b[2]


def test_verify_few_rows():
    """Prefix + candidate rows <= 32: every projection on the few-row kernels,
    which route the candidate rows' keys and values to the branch cache."""
    cfg = SMALL_BF16.replace(name="small bf16 P12 M4x5", n_prefix=12, n_visual=4, n_cands=4,
                             cand_len=5)
    wl = _case(cfg, 4, lens=[5, 3, 0, 4])
    assert cfg.n_prefix + int(np.sum(wl.cand_len)) <= 32
    check(cfg, run_gpu_verify(wl), run_oracle(wl), wl.cand_len)


@pytest.mark.parametrize("split", [0, 1])
def test_verify_degenerate_sizes(split):
    """A one-token prefix (P = 1: the last layer's prefix row is row 0), one
    candidate of one token, and a single 256-row tile holding both."""
    cfg = SMALL_BF16.replace(name="small bf16 P1 M1x1", n_prefix=1, n_visual=0, n_cands=1,
                             cand_len=1)
    wl = _case(cfg, 11, split=split)
    check(cfg, run_gpu_verify(wl, split_layers=split), run_oracle(wl), wl.cand_len)
    cfg = SMALL_BF16.replace(name="small bf16 P1 M3x70", n_prefix=1, n_visual=1, n_cands=3,
                             cand_len=70)
    wl = _case(cfg, 12, lens=[70, 1, 33], split=split)
    check(cfg, run_gpu_verify(wl, split_layers=split), run_oracle(wl), wl.cand_len)


def test_verify_fp32_and_no_candidate_tokens():
    """fp32 contexts and candidates of no tokens take the two passes in turn."""
    wl = _case(W.TINY_F32, 5)
    check(wl.cfg, run_gpu_verify(wl), run_oracle(wl), wl.cand_len)
    wl = _case(SMALL_BF16, 6, lens=[0, 0, 0, 0, 0])
    lp, sc, am, _ = run_gpu_verify(wl)
    assert np.all(lp == 0.0) and np.all(sc == 0.0) and am == 0


def test_verify_leaves_the_prefix_for_later_calls():
    """After vsr_verify the prefix cache is current: vsr_score on it matches the
    oracle, and so does a second vsr_verify on a new prefix."""
    torch = _torch()
    wl = _case(SMALL_BF16, 7, lens=[40, 2, 7, 23, 37], split=1)
    fused = run_gpu_verify(wl, split_layers=1)
    v = fused[3]
    ora = run_oracle(wl)
    check(wl.cfg, fused, ora, wl.cand_len)
    lp, sc, am = v.score(torch.tensor(wl.cand_ids, dtype=torch.int32, device="cuda"),
                         wl.cand_len)
    torch.cuda.synchronize()
    check(wl.cfg, (lp.cpu().numpy(), sc.cpu().numpy(), int(am.cpu()[0])), ora, wl.cand_len)
    wl2 = _case(SMALL_BF16.replace(n_prefix=130, n_visual=64), 8, lens=[1, 2, 3, 4, 40])
    wl2.weights = wl.weights
    check(wl2.cfg, run_gpu_verify(wl2, verifier=v), run_oracle(wl2), wl2.cand_len)


def test_verify_errors():
    torch = _torch()
    from paper_2601_01513_amd.binding import (VSR_EINVAL, VSR_ERANGE, VSR_ESTATE, Verifier,
                                              VsrError)
    wl = _case(SMALL_BF16, 9)
    v = Verifier(wl.cfg, wl.weights, device="cuda")
    ids = torch.tensor(wl.prefix_ids, dtype=torch.int32, device="cuda")
    cids = torch.tensor(wl.cand_ids, dtype=torch.int32, device="cuda")
    lens = list(wl.cand_len)
    cases = [
        ((wl.visual, ids, cids, [lens[0] + 100] + lens[1:]), VSR_EINVAL),  # > Cmax
        ((wl.visual, ids, cids[:, :0], [0] * len(lens)), VSR_EINVAL),      # Cmax = 0
        ((None, None, cids, lens), VSR_EINVAL),                              # empty prefix
    ]
    for args, code in cases:
        with pytest.raises(VsrError) as e:
            v.verify(*args)
        assert e.value.code == code
    big = torch.zeros((wl.cfg.n_cands + 1, cids.shape[1]), dtype=torch.int32, device="cuda")
    with pytest.raises(VsrError) as e:
        v.verify(wl.visual, ids, big, [1] * (wl.cfg.n_cands + 1))
    assert e.value.code == VSR_ERANGE
    # A failed call leaves no prefix current.
    with pytest.raises(VsrError) as e:
        v.score(cids, lens)
    assert e.value.code == VSR_ESTATE
    check(wl.cfg, run_gpu_verify(wl, verifier=v), run_oracle(wl), wl.cand_len)
