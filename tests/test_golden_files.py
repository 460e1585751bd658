"""The stored oracle outputs (tests/golden/) are consistent and current: they
were written by the oracle source that is in the tree, every score is the sum
of its log-probs, padded slots are 0, and a stored argmax is the lowest index
of the largest score (Eq. 7)."""
import os

import numpy as np
import pytest

from tests.golden_util import golden_files, load, oracle_sha256
from paper_2601_01513_amd import workload as W

FILES = golden_files()


@pytest.mark.parametrize("path", FILES, ids=[os.path.basename(p) for p in FILES])
def test_golden_file_is_current_and_consistent(path):
    rec = load(path)
    assert rec["oracle_sha256"] == oracle_sha256(), \
        "oracle/decoder.py changed since this file was written: rerun tests/golden/make_golden.py"
    cfg = W.CONFIGS[rec["workload_index"]]
    assert cfg.name == rec["workload"]
    assert [int(x) for x in W.cand_lengths(cfg, rec["seed"])] == rec["cand_len"]
    lp, sc = rec["lp_array"], rec["score_array"]
    for m in rec["cands"]:
        n = rec["cand_len"][m]
        assert np.all(lp[m, n:] == 0.0) and np.all(lp[m, :n] < 0.0)
        assert abs(sc[m] - lp[m].sum()) <= 1e-3 * abs(sc[m])
    if rec["argmax"] is not None:
        assert sorted(rec["cands"]) == list(range(cfg.n_cands))
        best = int(np.argmax(sc))
        assert rec["argmax"] == best


def test_golden_set_covers_the_full_size_workloads():
    have = {(load(p)["workload_index"], load(p)["seed"]) for p in FILES}
    for w in (1, 2, 3, 4):
        assert any(k[0] == w for k in have), f"no stored oracle output for workload {w}"
