"""Loading and checking of the stored oracle outputs under tests/golden/
(written by tests/golden/make_golden.py, which calls only the oracle)."""
import glob
import hashlib
import json
import os

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLDEN_DIR = os.path.join(ROOT, "tests", "golden")
ORACLE_SRC = os.path.join(ROOT, "oracle", "decoder.py")


def golden_files():
    return sorted(glob.glob(os.path.join(GOLDEN_DIR, "w*_s*_*.json")))


def load(path):
    rec = json.load(open(path))
    M, cmax = rec["config"]["n_cands"], rec["config"]["cand_len"]
    lp = np.zeros((M, cmax), dtype=np.float64)
    score = np.full(M, np.nan)
    for m in rec["cands"]:
        lp[m] = rec["lp"][str(m)]
        score[m] = rec["score"][str(m)]
    rec["lp_array"], rec["score_array"] = lp, score
    return rec


def oracle_sha256():
    return hashlib.sha256(open(ORACLE_SRC, "rb").read()).hexdigest()
