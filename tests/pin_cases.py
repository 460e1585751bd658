"""Small, sharp decoders for pinning the oracle on the CPU.

Weights are drawn with a large standard deviation and random norm gains so
that attention is peaked and every term of the decoder moves the result: a
dropped term, a wrong sign or index or a transposed operand changes the
log-probs by far more than rounding.
"""
import numpy as np

from paper_2601_01513_amd.workload import F32, VerifierConfig

PIN = VerifierConfig(name="pin L2 d64 GQA2", n_layers=2, d_model=64, n_heads=4,
                     n_kv_heads=2, head_dim=16, d_ff=96, vocab=97,
                     rope_base=10000.0, dtype=F32, n_prefix=11, n_visual=4,
                     n_cands=3, cand_len=6)


def sharp_inputs(cfg, seed=0, std=0.3, lens=None):
    rng = np.random.default_rng(seed)
    d = cfg.d_model
    n = lambda *s: rng.normal(0.0, std, size=s)  # noqa: E731
    gain = lambda: rng.uniform(0.5, 1.5, size=d)  # noqa: E731
    w = {"embed": rng.normal(0.0, 1.0, size=(cfg.vocab, d)),
         "lm_head": n(cfg.vocab, d), "final_norm": gain(), "layers": []}
    for _ in range(cfg.n_layers):
        w["layers"].append({
            "attn_norm": gain(), "wqkv": n(cfg.qkv_rows, d),
            "wo": n(d, cfg.n_heads * cfg.head_dim), "ffn_norm": gain(),
            "wgu": n(2 * cfg.d_ff, d), "wdown": n(d, cfg.d_ff)})
    visual = rng.normal(0.0, 1.0, size=(cfg.n_visual, d))
    prefix_ids = rng.integers(0, cfg.vocab, size=cfg.n_text)
    cand_ids = rng.integers(0, cfg.vocab, size=(cfg.n_cands, cfg.cand_len))
    if lens is None:
        lens = rng.integers(1, cfg.cand_len + 1, size=cfg.n_cands)
    lens = np.asarray(lens)
    for m in range(cfg.n_cands):
        cand_ids[m, lens[m]:] = 0
    return w, visual, prefix_ids, cand_ids, lens
