"""Summaries of rocprofv3 CSV output for the scoring-pass kernels.

    python -m paper_2601_01513_amd.profsummary stats KERNEL_STATS_CSV
        markdown table of the kernel-trace statistics
    python -m paper_2601_01513_amd.profsummary counters COUNTER_CSV [REGEX]
        mean counter value per dispatch, per kernel name and grid size
    python -m paper_2601_01513_amd.profsummary traffic KERNEL_REGEX FETCH_CSV WRITE_CSV \\
            COPY_FETCH_CSV COPY_WRITE_CSV COPY_BYTES SOURCE OUT_JSON
        HBM bytes per launch of the kernel: FETCH_SIZE / WRITE_SIZE (KiB per
        dispatch) scaled by what the same counters read for a plain copy of
        COPY_BYTES bytes (read COPY_BYTES, write COPY_BYTES); records the
        SHA-256 of SOURCE so that a later change of the kernel voids the numbers.
"""
from __future__ import annotations

import collections
import csv
import hashlib
import json
import re
import statistics
import sys


def _rows(path):
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def _short(name: str) -> str:
    m = re.search(r"(k_[a-z_0-9]+)", name)
    base = m.group(1) if m else name[:40]
    # k_attn<mode, precise, ...>: the first bool is the precise variant.
    ma = re.search(r"k_attnILi\dELb(\d)", name) or re.search(r"k_attn<\d, (true|false)", name)
    precise = bool(ma) and ma.group(1) in ("1", "true")
    if "k_attnILi0" in name or "k_attn<0" in name:
        base = "k_attn<0> (prefill" + (", precise)" if precise else ")")
    elif "k_attnILi1" in name or "k_attn<1" in name:
        base = "k_attn<1> (cascade" + (", precise)" if precise else ")")
    elif "k_attnILi2" in name or "k_attn<2" in name:
        dec = "k_attnILi2ELb0ELb1E" in name or "k_attn<2, false, true>" in name
        base = "k_attn<2> (draft" + (", precise)" if precise else
                                     ", decode blocks)" if dec else ")")
    elif base == "k_skinny":
        # k_skinny<rows per group, A split, bf16 weights, greedy LM head>
        m = re.search(r"k_skinnyILi(\d+)ELi(\d+)ELb(\d)ELb(\d)E", name)
        if m:
            base = "k_skinny (" + ("greedy LM head" if m.group(4) == "1" else "product") + \
                (", split A" if m.group(2) == "2" else "") + ")"
    return base


def stats(path):
    rows = _rows(path)
    out = ["| kernel | calls | avg us | total ms | % |", "|---|---|---|---|---|"]
    for r in rows:
        out.append(f"| {_short(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                   f"{float(r['TotalDurationNs']) / 1e6:.2f} | {float(r['Percentage']):.2f} |")
    return "\n".join(out)


def counters(path, regex="."):
    agg = collections.defaultdict(lambda: collections.defaultdict(list))
    for r in _rows(path):
        if not re.search(regex, r["Kernel_Name"]):
            continue
        key = (_short(r["Kernel_Name"]), r["Grid_Size"])
        agg[key][r["Counter_Name"]].append(float(r["Counter_Value"]))
    return {k: {c: statistics.mean(v) for c, v in d.items()} for k, d in agg.items()}


def _per_dispatch(path, regex, counter):
    rows = [r for r in _rows(path)
            if re.search(regex, r["Kernel_Name"]) and r["Counter_Name"] == counter]
    if not rows:
        raise SystemExit(f"no {counter} rows for /{regex}/ in {path}")
    return (statistics.mean(float(r["Counter_Value"]) for r in rows), len(rows),
            _short(rows[0]["Kernel_Name"]))


def traffic(kregex, fetch_csv, write_csv, cfetch_csv, cwrite_csv, copy_bytes, source, out):
    fetch, n, kname = _per_dispatch(fetch_csv, kregex, "FETCH_SIZE")
    write, _, _ = _per_dispatch(write_csv, kregex, "WRITE_SIZE")
    cregex = r"copy|elementwise|Copy"
    cf = max(float(r["Counter_Value"]) for r in _rows(cfetch_csv)
             if re.search(cregex, r["Kernel_Name"]) and r["Counter_Name"] == "FETCH_SIZE")
    cw = max(float(r["Counter_Value"]) for r in _rows(cwrite_csv)
             if re.search(cregex, r["Kernel_Name"]) and r["Counter_Name"] == "WRITE_SIZE")
    f_scale = copy_bytes / (cf * 1024.0)
    w_scale = copy_bytes / (cw * 1024.0)
    with open(source, "rb") as f:
        digest = hashlib.sha256(f.read()).hexdigest()
    rec = {"kernel": kname, "kernel_regex": kregex, "dispatches": n,
           "fetch_kib_per_dispatch": fetch, "write_kib_per_dispatch": write,
           "copy_bytes": copy_bytes, "copy_fetch_kib": cf, "copy_write_kib": cw,
           "fetch_scale": f_scale, "write_scale": w_scale,
           "hbm_bytes_per_launch": fetch * 1024.0 * f_scale + write * 1024.0 * w_scale,
           "source": source, "source_sha256": digest}
    with open(out, "w") as f:
        json.dump(rec, f, indent=1)
    return rec


if __name__ == "__main__":
    cmd = sys.argv[1]
    if cmd == "stats":
        print(stats(sys.argv[2]))
    elif cmd == "counters":
        res = counters(sys.argv[2], sys.argv[3] if len(sys.argv) > 3 else ".")
        for (k, g), d in sorted(res.items()):
            print(f"{k} grid={g}")
            for c, v in sorted(d.items()):
                print(f"    {c:28s} {v:18.1f}")
    elif cmd == "traffic":
        a = sys.argv[2:]
        print(json.dumps(traffic(a[0], a[1], a[2], a[3], a[4], float(a[5]), a[6], a[7]), indent=1))
    else:
        raise SystemExit(__doc__)
