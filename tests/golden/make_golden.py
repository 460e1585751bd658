"""Writes the oracle's log-probabilities for a full-size scoring workload.

The expected values of the full-depth parity tests (tests/test_gpu_golden.py)
come from here. This script calls only the CPU oracle (oracle/, float32,
shared-prefix mode: Section 3.1, Eq. 6-7 as the definition restated there)
and the seeded input generator; it never loads the HIP library. The weights
are drawn by the generator on a GPU (torch's device generator, the inputs
the tests and the benchmark use), copied to the host layer by layer, and the
oracle runs on the host cores.

    python tests/golden/make_golden.py --workload 3 --seed 0 --cands all \
        --out tests/golden

writes <out>/<key>.json (key: workload index, seed, candidate set) holding
the candidates' log-probs (zeros past each length), their scores, the
oracle's argmax when every candidate is scored, the SHA-256 of
oracle/decoder.py and of the workload module, and the fingerprint of the
generated inputs (the tests regenerate the inputs and compare it first).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2601_01513_amd import workload as W  # noqa: E402

ORACLE_SRC = os.path.join(ROOT, "oracle", "decoder.py")
WORKLOAD_SRC = os.path.join(ROOT, "paper_2601_01513_amd", "workload.py")


def sha256_file(path: str) -> str:
    return hashlib.sha256(open(path, "rb").read()).hexdigest()


def golden_key(workload: int, seed: int, cands) -> str:
    tag = "all" if cands is None else "c" + "-".join(str(c) for c in cands)
    return f"w{workload}_s{seed}_{tag}"


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", type=int, required=True, help="index into workload.CONFIGS")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cands", default="all", help="'all' or comma-separated candidate indices")
    ap.add_argument("--out", default=os.path.join(ROOT, "tests", "golden"))
    args = ap.parse_args()

    import torch
    cfg = W.CONFIGS[args.workload]
    cands = None if args.cands == "all" else [int(c) for c in args.cands.split(",")]
    t_start = time.time()
    print(f"golden: {cfg.name} seed {args.seed} candidates {args.cands}", flush=True)
    wl = W.make_workload(cfg, args.seed, device="cuda")
    torch.cuda.synchronize()
    fp = W.input_fingerprint(wl)
    print(f"  inputs generated ({time.time() - t_start:.0f}s), fingerprint {fp[:16]}",
          flush=True)
    hw = W.host_weights(wl.weights, lazy=True)
    vis = W.to_host_f32(wl.visual)
    t0 = time.time()

    def progress(layer):
        print(f"  oracle layer {layer + 1}/{cfg.n_layers} at {time.time() - t0:.0f}s", flush=True)
    lp, sc, am = oracle.score_shared_prefix(cfg, hw, vis, wl.prefix_ids, wl.cand_ids, wl.cand_len,
                                            dtype=np.float32, cands=cands, progress=progress)
    secs = time.time() - t0
    scored = list(range(cfg.n_cands)) if cands is None else cands
    rec = {
        "workload": cfg.name, "workload_index": args.workload, "seed": args.seed,
        "config": {k: v for k, v in cfg.__dict__.items()},
        "oracle": "oracle.score_shared_prefix, float32",
        "oracle_sha256": sha256_file(ORACLE_SRC), "workload_sha256": sha256_file(WORKLOAD_SRC),
        "input_fingerprint": fp, "torch": torch.__version__,
        "device": torch.cuda.get_device_name(0),
        "cands": scored, "cand_len": [int(x) for x in wl.cand_len],
        "lp": {str(m): [float(x) for x in lp[m]] for m in scored},
        "score": {str(m): float(sc[m]) for m in scored},
        "argmax": None if cands is not None else int(am),
        "oracle_seconds": round(secs, 1), "host_threads": oracle.decoder.THREADS,
        "host_cpu": cpu_model(),
    }
    os.makedirs(args.out, exist_ok=True)
    path = os.path.join(args.out, golden_key(args.workload, args.seed, cands) + ".json")
    with open(path, "w") as f:
        json.dump(rec, f, indent=1)
    print(f"  wrote {path}: oracle {secs:.0f}s, scores {np.round(sc[scored], 3)}, "
          f"argmax {rec['argmax']}", flush=True)


if __name__ == "__main__":
    main()
