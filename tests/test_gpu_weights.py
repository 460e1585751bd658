"""GPU checks of the fp16 GEMM-weight form (vsr_config.gemm_weights): the
conversion kernel against an independent host rounding, and bit-identical
scoring with bf16 and fp16 weight storage (the GEMMs apply the same
conversion either way)."""
import sys

import numpy as np
import pytest

from paper_2601_01513_amd import workload as W

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _say(msg):
    print(msg, file=sys.stderr, flush=True)


def _f16_toward_zero(x32: np.ndarray) -> np.ndarray:
    """float32 -> float16 rounding toward zero (host reference): round to
    nearest, then step one ulp toward zero wherever that moved away from
    zero."""
    h = x32.astype(np.float16)
    away = np.abs(h.astype(np.float32)) > np.abs(x32)
    fix = np.nextafter(h, np.float16(0))
    return np.where(away, fix, h)


@pytest.mark.parametrize("n", [1, 7, 8, 9, 4096 + 5, 1 << 20])
def test_conversion_matches_host_rounding(n):
    torch = _torch()
    from paper_2601_01513_amd.binding import weights_to_f16
    g = torch.Generator(device="cuda").manual_seed(n)
    x = torch.randn(n, generator=g, device="cuda") * 0.02
    # include tiny magnitudes (fp16 subnormals), exact zero and large values
    x[: n // 4] *= 1e-4
    x[0] = 0.0
    if n > 3:
        x[1], x[2] = -3.0e4, 2.0 ** -20
    b = x.to(torch.bfloat16)
    y = weights_to_f16(b)
    torch.cuda.synchronize()
    ref = _f16_toward_zero(b.float().cpu().numpy())
    got = y.cpu().numpy()
    np.testing.assert_array_equal(got.view(np.uint16), ref.view(np.uint16))


@pytest.mark.parametrize("cfg", [
    W.VerifierConfig(name="small bf16 L2 d256 G2 F320 V1000", n_layers=2, d_model=256,
                     n_heads=4, n_kv_heads=2, head_dim=128, d_ff=320, vocab=1000,
                     rope_base=1e6, dtype=W.BF16, n_prefix=300, n_visual=100, n_cands=5,
                     cand_len=40),
    W.B7.replace(name="7B-class bf16 P4096 M8x64 (2 layers)", n_layers=2)],
    ids=["small", "7B-2layers"])
def test_fp16_and_bf16_weight_storage_score_identically(cfg):
    torch = _torch()
    from paper_2601_01513_amd.binding import Verifier
    _say(f"case: {cfg.name}")
    wl = W.make_workload(cfg, 0, device="cuda")
    ids = torch.tensor(wl.prefix_ids, dtype=torch.int32, device="cuda")
    cids = torch.tensor(wl.cand_ids, dtype=torch.int32, device="cuda")
    res = {}
    for form in ("bf16", "f16"):
        v = Verifier(cfg, wl.weights, device="cuda", gemm_weights=form)
        v.prefill(wl.visual, ids)
        lp, sc, am = v.score(cids, wl.cand_len)
        torch.cuda.synchronize()
        res[form] = (lp.cpu().numpy(), sc.cpu().numpy(), int(am.cpu()[0]))
        del v
    np.testing.assert_array_equal(res["bf16"][0], res["f16"][0])
    np.testing.assert_array_equal(res["bf16"][1], res["f16"][1])
    assert res["bf16"][2] == res["f16"][2]
