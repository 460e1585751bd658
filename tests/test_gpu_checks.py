"""The call validator (vsr_set_checks) through the C ABI: bad ids give
VSR_EID, non-finite results VSR_ENONFINITE; the outputs are those of the
unchecked call (an out-of-range id is read as id 0), and valid inputs pass
unchanged. The oracle, given the same NaN visual row, also yields non-finite
scores (a NaN key reaches every later query through the softmax)."""
import sys

import numpy as np
import pytest

import oracle
from paper_2601_01513_amd import workload as W

pytestmark = pytest.mark.gpu

SMALL = W.VerifierConfig(
    name="checks bf16 L2 d256 G2 F320 V1000", n_layers=2, d_model=256, n_heads=4,
    n_kv_heads=2, head_dim=128, d_ff=320, vocab=1000, rope_base=1e6, dtype=W.BF16,
    n_prefix=300, n_visual=100, n_cands=5, cand_len=40)


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _say(msg):
    print(msg, file=sys.stderr, flush=True)


def _run(v, wl, cids, visual=None, prefix_ids=None):
    torch = _torch()
    ids = torch.tensor(wl.prefix_ids if prefix_ids is None else prefix_ids, dtype=torch.int32,
                       device="cuda")
    lp, sc, am = v.verify(wl.visual if visual is None else visual, ids,
                          torch.tensor(cids, dtype=torch.int32, device="cuda"), wl.cand_len)
    torch.cuda.synchronize()
    return lp.cpu().numpy(), sc.cpu().numpy(), int(am.cpu()[0])


def _expect(code, fn):
    from paper_2601_01513_amd.binding import VsrError
    with pytest.raises(VsrError) as e:
        fn()
    assert e.value.code == code, str(e.value)
    _say(f"  status {e.value.code}: {e.value}")


@pytest.mark.parametrize("cfg", [SMALL, W.TINY_F32], ids=["bf16", "fp32"])
def test_valid_inputs_pass_and_match_unchecked(cfg):
    torch = _torch()
    from paper_2601_01513_amd.binding import Verifier
    _say(f"case: {cfg.name} checks on, valid inputs")
    wl = W.make_workload(cfg, 0, device="cuda")
    v = Verifier(cfg, wl.weights, device="cuda")
    ref = _run(v, wl, wl.cand_ids)
    v.set_checks(ids=True, finite=True)
    got = _run(v, wl, wl.cand_ids)
    assert np.array_equal(ref[0], got[0]) and np.array_equal(ref[1], got[1])
    assert ref[2] == got[2]
    v.prefill(wl.visual, torch.tensor(wl.prefix_ids, dtype=torch.int32, device="cuda"))
    v.score(torch.tensor(wl.cand_ids, dtype=torch.int32, device="cuda"), wl.cand_len)
    torch.cuda.synchronize()


@pytest.mark.parametrize("cfg", [SMALL, W.TINY_F32], ids=["bf16", "fp32"])
def test_out_of_range_ids_report_eid(cfg):
    torch = _torch()
    from paper_2601_01513_amd.binding import VSR_EID, Verifier
    _say(f"case: {cfg.name} out-of-range ids")
    wl = W.make_workload(cfg, 1, device="cuda")
    v = Verifier(cfg, wl.weights, device="cuda")
    bad = wl.cand_ids.copy()
    bad[1, 3] = cfg.vocab + 5
    bad[2, 0] = -1
    zero = wl.cand_ids.copy()
    zero[1, 3] = 0
    zero[2, 0] = 0
    ref = _run(v, wl, zero)
    unchecked = _run(v, wl, bad)          # default: no check, id read as 0
    assert np.array_equal(ref[0], unchecked[0])
    # The two-call pass (it agrees with vsr_verify to rounding only).
    v.prefill(wl.visual, torch.tensor(wl.prefix_ids, dtype=torch.int32, device="cuda"))
    ref2 = v.score(torch.tensor(zero, dtype=torch.int32, device="cuda"), wl.cand_len)[0]
    torch.cuda.synchronize()
    ref2 = ref2.cpu().numpy()
    v.set_checks(ids=True, finite=False)
    _expect(VSR_EID, lambda: _run(v, wl, bad))
    pid = wl.prefix_ids.copy()
    pid[7] = 1 << 30
    _expect(VSR_EID, lambda: v.prefill(wl.visual, torch.tensor(pid, dtype=torch.int32,
                                                               device="cuda")))
    v.prefill(wl.visual, torch.tensor(wl.prefix_ids, dtype=torch.int32, device="cuda"))
    lens = [max(1, int(n)) for n in wl.cand_len]
    _expect(VSR_EID, lambda: v.reliability(torch.tensor(bad, dtype=torch.int32, device="cuda"),
                                           lens, 1, 2, 0.05))
    lp, sc, am = v.score(torch.tensor(zero, dtype=torch.int32, device="cuda"), wl.cand_len)
    torch.cuda.synchronize()
    assert np.array_equal(lp.cpu().numpy(), ref2)


@pytest.mark.parametrize("cfg", [SMALL, W.TINY_F32], ids=["bf16", "fp32"])
def test_nan_visual_row_reports_enonfinite(cfg):
    torch = _torch()
    from paper_2601_01513_amd.binding import VSR_ENONFINITE, Verifier
    _say(f"case: {cfg.name} NaN visual row")
    wl = W.make_workload(cfg, 2, device="cuda")
    vis = wl.visual.clone()
    vis[17, :] = float("nan")
    v = Verifier(cfg, wl.weights, device="cuda")
    v.set_checks(ids=True, finite=True)
    _expect(VSR_ENONFINITE, lambda: _run(v, wl, wl.cand_ids, visual=vis))
    _expect(VSR_ENONFINITE, lambda: v.prefill(vis, torch.tensor(
        wl.prefix_ids, dtype=torch.int32, device="cuda")))
    # The oracle on the same inputs: no finite score either.
    with np.errstate(invalid="ignore", over="ignore"):
        lp_o, sc_o, _ = oracle.score_shared_prefix(cfg, W.host_weights(wl.weights),
                                                   W.to_host_f32(vis), wl.prefix_ids,
                                                   wl.cand_ids, wl.cand_len, dtype=np.float32)
    assert not np.any(np.isfinite(sc_o))
    # Finite inputs again: the context recovers.
    _run(v, wl, wl.cand_ids)


def test_unknown_check_bits_are_rejected():
    _torch()
    from paper_2601_01513_amd.binding import VSR_EINVAL, Verifier
    wl = W.make_workload(W.TINY_F32, 0, device="cuda")
    v = Verifier(W.TINY_F32, wl.weights, device="cuda")
    assert v.lib.vsr_set_checks(v.h, 4) == VSR_EINVAL
    assert b"unknown" in v.lib.vsr_last_error(v.h)
