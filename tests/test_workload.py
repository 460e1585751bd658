"""The seeded input generator: shapes, determinism, padding, ragged lengths."""
import numpy as np
import torch

from paper_2601_01513_amd import workload as W


def test_configs_match_their_stated_sizes():
    c = W.B7
    assert (c.n_layers, c.d_model, c.n_heads, c.n_kv_heads, c.head_dim, c.d_ff, c.vocab) == \
        (28, 3584, 28, 4, 128, 18944, 152064)
    assert (c.n_prefix, c.n_visual, c.n_cands, c.cand_len) == (4096, 2048, 8, 64)
    assert abs(c.n_params() / 1e9 - 7.62) < 0.01
    assert abs(W.B32.n_params() / 1e9 - 32.8) < 0.1
    assert abs(W.B1_5.n_params() / 1e9 - 1.78) < 0.01
    assert W.B7_LONG.ragged == (32, 128) and W.B7_LONG.n_prefix == 16384
    assert W.TINY_F32.dtype == W.F32 and all(c.dtype == W.BF16 for c in W.CONFIGS[1:])


def test_ids_are_seeded_padded_and_in_range():
    cfg = W.B7_LONG.replace(n_prefix=64, n_visual=16)
    a = W.make_ids(cfg, 3)
    b = W.make_ids(cfg, 3)
    c = W.make_ids(cfg, 4)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    assert not np.array_equal(a[1], c[1])
    pids, cids, lens = a
    assert pids.shape == (48,) and cids.shape == (16, 128)
    assert lens.min() >= 32 and lens.max() <= 128
    for m in range(16):
        assert np.all(cids[m, lens[m]:] == 0)
    assert cids.min() >= 0 and cids.max() < cfg.vocab and pids.max() < cfg.vocab


def test_weights_are_seeded_and_rounded():
    cfg = W.TINY_F32.replace(n_layers=1, dtype=W.BF16)
    w1 = W.make_weights(cfg, 0)
    w2 = W.make_weights(cfg, 0)
    assert torch.equal(w1["embed"], w2["embed"]) and w1["embed"].dtype == torch.bfloat16
    assert not torch.equal(w1["embed"], w1["lm_head"])
    assert torch.all(w1["final_norm"] == 1)
    std = w1["layers"][0]["wgu"].float().std().item()
    assert abs(std - 0.02) < 0.001
    h = W.host_weights(w1)
    assert h["embed"].dtype == np.float32
    assert np.array_equal(h["embed"], w1["embed"].float().numpy())
