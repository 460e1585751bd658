"""Benchmark of the verifier scoring pass on one GPU.

A step is one verify pass: vsr_verify, the prefill over the shared prefix
and the scoring of all candidates as one fused pass (the prefix KV is rebuilt
every step). Inputs are seeded synthetic tensors resident in HBM before the
timed region.

Prints one JSON line: candidate tokens scored per second over the timed steps,
the roofline position of the dominant kernel (from per-launch HIP-event
timings inside the library, on its stream, over the same timed region) and
the CPU oracle timed on a bounded sample on the host cores.

An untimed profiled pass first times every stage (the breakdown, and which
kernel dominates); the timed steps then bracket only that kernel's launches
with events, so the timing perturbs the pass as little as possible.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2601_01513_amd import workload as W  # noqa: E402

METRIC = ("candidate tokens scored/sec and ms per verify pass "
          "(7B-class, 4k prefix, 8×64)")
PEAK_BF16_TFLOPS = 2500.0  # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0

# Kernels as the profiler sees them (fp16 GEMM weights, the default), and
# the stages each one serves.
KERNELS = {
    "k_gemm_swiglu_4w": ["verify.gate_up_swiglu"],
    "k_gemm_residual_4w": ["verify.down_proj"],
    "k_gemm_residual": ["verify.o_proj"],
    "k_gemm_qkv": ["verify.qkv_rope"],
    "k_attn<0> (prefill)": ["verify.attention"],
    "k_attn<1> (cascade)": ["verify.cand_attention"],
    "k_attn_merge": ["verify.attn_merge"],
    "k_gemm_lmhead": ["verify.lm_head_lse"],
    "k_rmsnorm": ["verify.rmsnorm"],
}


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def stage_flops(cfg, P, lens):
    """Algorithmic FLOPs of one fused verify pass per stage (multiply-add = 2).

    The prefix rows and the candidate rows share every projection. The last
    layer needs keys/values for every row but attention, projections and FFN
    only for the last prefix row (the one predicting candidate token 0) and
    the candidate rows, which is all the library computes there.
    """
    d, hq, hd, F, V = cfg.d_model, cfg.n_heads, cfg.head_dim, cfg.d_ff, cfg.vocab
    L = cfg.n_layers
    T = int(sum(lens))
    rows = P + T
    body = rows * max(L - 1, 0) + (T + 1 if L else 0)
    f = {"verify.qkv_rope": 2.0 * rows * cfg.qkv_rows * d * L,
         "verify.o_proj": 2.0 * body * d * hq * hd,
         "verify.gate_up_swiglu": 2.0 * body * 2 * F * d,
         "verify.down_proj": 2.0 * body * d * F}
    # QK^T and PV over the visible keys of every query (causal / cascade).
    f["verify.attention"] = 4.0 * hd * hq * ((P * (P + 1) / 2) * (L - 1) + P) if L else 0.0
    f["verify.cand_attention"] = 4.0 * hd * hq * sum(n * P + n * (n + 1) / 2 for n in lens) * L
    f["verify.lm_head_lse"] = 2.0 * T * V * d
    return f


def stage_bytes(cfg, P, lens):
    """Algorithmic HBM bytes of one fused verify pass per stage: every operand
    read once and every output written once, in the storage types of the
    path (fp16 GEMM weights and activations, fp16 K/V caches, fp32 residual
    stream and partials). Precise-layer remainder planes are left out (an
    implementation choice, not the method's work)."""
    d, hq, hkv, hd, F, V = (cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_ff,
                            cfg.vocab)
    L = cfg.n_layers
    T = int(sum(lens))
    rows = P + T
    body = rows * max(L - 1, 0) + (T + 1 if L else 0)   # rows past attention
    qd = hq * hd
    kv = 2 * hkv * hd * 2                                # K + V bytes per position
    b = {"verify.qkv_rope": L * cfg.qkv_rows * d * 2 + rows * L * (d * 2 + qd * 2 + kv),
         "verify.o_proj": L * d * qd * 2 + body * (qd * 2 + d * 8),
         "verify.gate_up_swiglu": L * 2 * F * d * 2 + body * (d * 2 + F * 2),
         "verify.down_proj": L * d * F * 2 + body * (F * 2 + d * 8),
         # prefix keys/values once per layer, queries in, outputs out
         "verify.attention": L * P * kv + (P * max(L - 1, 0) + 1) * qd * 4,
         # the prefix keys/values once for all candidates, their own keys, q, out
         "verify.cand_attention": L * (P * kv + T * kv + T * qd * 4),
         # LM head once, inputs, per-chunk partials and target logits
         "verify.lm_head_lse": V * d * 2 + T * d * 2 + (V // 256 + 1) * T * 8 + T * 4,
         # two norms per layer (attention: every row; FFN: the rows past
         # attention): fp32 rows in, fp16 rows out
         "verify.rmsnorm": (rows * L + body) * d * 6,
         "verify.embed": rows * d * 6}
    return b


def stage_row(fl, nb, ms):
    """One breakdown row: achieved rates and the roofline position."""
    sec = ms * 1e-3
    row = {"ms": round(ms, 3)}
    t_mfma = fl / (PEAK_BF16_TFLOPS * 1e12)
    t_hbm = (nb or 0) / (PEAK_HBM_GBS * 1e9)
    if fl:
        row["tflops"] = round(fl / sec / 1e12, 1)
        row["mfma_frac"] = round(fl / sec / 1e12 / PEAK_BF16_TFLOPS, 4)
    if nb:
        row["GBs"] = round(nb / sec / 1e9, 1)
        row["hbm_frac"] = round(nb / sec / 1e9 / PEAK_HBM_GBS, 4)
        row["flop_per_byte"] = round(fl / nb, 1) if fl else 0.0
    row["bound"] = "mfma" if t_mfma >= t_hbm else "hbm"
    row["frac"] = round(max(t_mfma, t_hbm) / sec, 4)
    return row


def measured_traffic(kname):
    """HBM bytes per launch of `kname` from the committed counter runs
    (profiles/traffic.json), or None if absent or if the kernel source has
    changed since they were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        rec = json.load(open(path))
        src = os.path.join(ROOT, rec["source"])
        if rec.get("kernel") != kname:
            return None
        if hashlib.sha256(open(src, "rb").read()).hexdigest() != rec["source_sha256"]:
            return None
        return round(rec["hbm_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def time_next_rows(v, cids, lens, dev, reps, log_fn):
    """The two-stage verification on the same workload, after the timed
    region: vsr_reliability over the same branches (against the current
    prefix) and vsr_align_select at M drafts x 64 keyframes x 768 (CLIP
    ViT-L/14 embedding width), timed with events on the stream."""
    import numpy as np
    import torch
    from paper_2601_01513_amd.binding import align_select
    M = len(lens)
    st = torch.cuda.current_stream(dev)

    def timed(fn, n):
        for _ in range(2):
            fn()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(st)
        for _ in range(n):
            fn()
        b.record(st)
        b.synchronize()
        return a.elapsed_time(b) / n
    blens = [max(1, n) for n in lens]
    rel_ms = timed(lambda: v.reliability(cids, blens, 17, 29, 0.05), reps)
    rng = np.random.default_rng(0)
    ent = torch.tensor(rng.normal(size=(M, 768)).astype(np.float32), device=dev)
    frames = torch.tensor(rng.normal(size=(64, 768)).astype(np.float32), device=dev)
    rel = torch.rand(M, device=dev)
    sel_ms = timed(lambda: align_select(ent, frames, rel, 0.05, "two_stage"), 100)
    log_fn(f"reliability {rel_ms:.3f} ms/call, align_select {sel_ms * 1e3:.1f} us/call")
    out = {"reliability_ms": round(rel_ms, 3),
           "reliability_tok_s": round(sum(blens) / (rel_ms * 1e-3), 1),
           "align_select_us": round(sel_ms * 1e3, 2),
           "align_select_shape": f"M={M} frames=64 D=768"}
    # Retrieval stage: keyframes of a 22 s video (220 frames of 336 x 336) and
    # top-k over a 100k-document bank.
    from paper_2601_01513_amd.binding import Retriever
    rc = W.VIDEO_22S_BANK
    frames, femb, demb = W.make_retrieval(rc, 0)
    r = Retriever(rc.n_frames, rc.height, rc.width, rc.n_docs, rc.dim, rc.k, rc.K, device=dev)
    fr, fe, de = (torch.tensor(a, device=dev) for a in (frames, femb, demb))
    kf_us = timed(lambda: r.keyframes(fr, rc.theta), 20) * 1e3
    rt_us = timed(lambda: r.retrieve(fe, de), 20) * 1e3
    nk = int(r.n_keys.cpu()[0])
    log_fn(f"keyframes {kf_us:.1f} us/call, retrieve {rt_us:.1f} us/call ({nk} keyframes)")
    frame_bytes = frames.nbytes
    bank_bytes = demb.nbytes * ((nk + 15) // 16)   # the bank is read once per 16 keyframes
    out.update({"keyframes_us": round(kf_us, 1),
                "keyframes_GBs": round(frame_bytes / (kf_us * 1e-6) / 1e9, 1),
                "retrieve_us": round(rt_us, 1),
                "retrieve_GBs": round(bank_bytes / (rt_us * 1e-6) / 1e9, 1),
                "retrieval_shape": f"{rc.n_frames} frames {rc.height}x{rc.width}, "
                                   f"{nk} keyframes, {rc.n_docs} docs x {rc.dim}, k={rc.k}"})
    return out


def time_draft(dev, log_fn, reps=3):
    """Parallel drafting (Eq. 5, 8-10) with the 3B-class drafter: one
    vsr_draft call = the branch prompts through every layer, then 64 decode
    steps of one row per branch. A decode step streams every GEMM weight
    (fp16) and the LM head once: its HBM roofline."""
    import torch
    from paper_2601_01513_amd.binding import Verifier
    cfg, n_new = W.DRAFT_3B, W.DRAFT_NEW
    wl = W.make_workload(cfg, 0, device=dev)
    v = Verifier(cfg, wl.weights, device=dev, max_new=n_new)
    ids = torch.tensor(wl.prefix_ids, dtype=torch.int32, device=dev)
    v.prefill(wl.visual, ids)
    pids = torch.tensor(wl.cand_ids, dtype=torch.int32, device=dev)
    lens = [int(x) for x in wl.cand_len]
    M = len(lens)
    st = torch.cuda.current_stream(dev)

    def timed(n):
        out = torch.empty((M, n), dtype=torch.int32, device=dev)
        v.draft(pids, lens, n, out=out)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(st)
        for _ in range(reps):
            v.draft(pids, lens, n, out=out)
        b.record(st)
        b.synchronize()
        return a.elapsed_time(b) / reps
    one = timed(1)
    full = timed(n_new)
    step_ms = (full - one) / (n_new - 1)
    d, F, L = cfg.d_model, cfg.d_ff, cfg.n_layers
    weight_bytes = 2 * (L * d * (cfg.qkv_rows + cfg.n_heads * cfg.head_dim + 3 * F)
                        + cfg.vocab * d)
    gbs = weight_bytes / (step_ms * 1e-3) / 1e9
    log_fn(f"draft: {full:.2f} ms per call ({M} branches x {n_new} new tokens), prompt pass "
           f"{one:.2f} ms, decode step {step_ms:.3f} ms = {gbs:.0f} GB/s of weights")
    res = {"draft_ms": round(full, 2), "draft_tok_s": round(M * n_new / (full * 1e-3), 1),
           "draft_prompt_pass_ms": round(one, 2), "draft_step_ms": round(step_ms, 3),
           "draft_step_weight_GBs": round(gbs, 1),
           "draft_step_hbm_frac": round(gbs / PEAK_HBM_GBS, 4),
           "draft_shape": f"{cfg.name}: prefix {cfg.n_prefix}, {M} branches x "
                          f"{cfg.cand_len} prompt tokens, {n_new} new"}
    v.close()
    del v, wl
    torch.cuda.empty_cache()
    return res


def blas_info():
    """(threads, vendor string) of the BLAS numpy uses."""
    try:
        from threadpoolctl import threadpool_info
        for i in threadpool_info():
            if i.get("user_api") == "blas":
                return (int(i.get("num_threads", 1)),
                        f"{i.get('internal_api')} {i.get('version')} "
                        f"({i.get('threading_layer')}, {i.get('architecture')})")
    except Exception:
        pass
    return 1, "unknown"


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, log_fn, sample_layers=3):
    """The plain fp32 oracle (oracle.score_shared_prefix, float32) on this
    workload's own inputs, with its first `sample_layers` layers: one bounded
    run, timed per part (embedding + host copies, each layer, LM head), and
    the per-layer time scaled to the full depth."""
    import numpy as np
    import oracle
    threads, vendor = blas_info()
    cfg = wl.cfg
    nl = min(sample_layers, cfg.n_layers)
    t0 = time.perf_counter()
    hw = {"embed": W.to_host_f32(wl.weights["embed"]),
          "lm_head": W.to_host_f32(wl.weights["lm_head"]),
          "final_norm": W.to_host_f32(wl.weights["final_norm"]),
          "layers": W.HostLayers(wl.weights["layers"][:nl])}
    vis = W.to_host_f32(wl.visual)
    marks = []
    c = cfg.replace(n_layers=nl)
    t1 = time.perf_counter()
    oracle.score_shared_prefix(c, hw, vis, wl.prefix_ids, wl.cand_ids, wl.cand_len,
                               dtype=np.float32, progress=lambda l: marks.append(time.perf_counter()))
    t2 = time.perf_counter()
    layer_s = [b - a for a, b in zip([t1] + marks[:-1], marks)]
    per_layer = sum(layer_s) / len(layer_s)
    tail = t2 - marks[-1]
    full = (t1 - t0) + per_layer * cfg.n_layers + tail
    log_fn(f"cpu oracle (fp32): setup {t1 - t0:.1f}s, layers "
           f"{', '.join(f'{x:.1f}' for x in layer_s)}s, LM head {tail:.1f}s")
    tokens = int(sum(wl.cand_len))
    return {"value": tokens / full, "unit": "candidate tokens/s",
            "cores": max(threads, oracle.decoder.THREADS), "kind": "oracle",
            "sample": (f"plain fp32 oracle (oracle.score_shared_prefix, float32, shared-prefix "
                       f"mode) on this workload's inputs with its first {nl} of {cfg.n_layers} "
                       f"layers in one run ({t2 - t0:.1f}s: host copies + embedding "
                       f"{t1 - t0:.1f}s, {per_layer:.2f}s per layer, LM head {tail:.1f}s); "
                       f"the per-layer time scaled to {cfg.n_layers} layers gives "
                       f"{full:.1f}s per verify pass (extrapolated). Host: {cpu_model()}; "
                       f"BLAS {vendor}, {threads} threads; attention heads on "
                       f"{oracle.decoder.THREADS} threads")}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=2,
                    help="index into the workload list (default: the 7B-class 4k prefix 8x64)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-next-rows", action="store_true",
                    help="skip the two-stage verification timings (counter runs)")
    ap.add_argument("--stages", action="store_true", help="print per-stage times to stderr")
    ap.add_argument("--only-draft", action="store_true",
                    help="only time the drafter (vsr_draft, 3B-class) and print its figures")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="only copy MIB MiB device-to-device (counter calibration) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}): the scoring pass is "
              "not sharded across GPUs", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2601_01513_amd.binding import Verifier

    if args.copy_probe:
        # A plain elementwise kernel that reads n bytes and writes n bytes:
        # the scale for the HBM byte counters.
        n = args.copy_probe << 20
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n, "copies": 3}))
        return

    if args.only_draft:
        dev = torch.device("cuda:0")
        torch.cuda.set_device(dev)
        print(json.dumps(time_draft(dev, log)), flush=True)
        return

    cfg = W.CONFIGS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log(f"workload: {cfg.name}; generating inputs on the GPU")
    wl = W.make_workload(cfg, args.seed, device=dev)
    ids = torch.tensor(wl.prefix_ids, dtype=torch.int32, device=dev) if cfg.n_text else None
    vis = wl.visual if cfg.n_visual else None
    cids = torch.tensor(wl.cand_ids, dtype=torch.int32, device=dev)
    lens = [int(x) for x in wl.cand_len]
    v = Verifier(cfg, wl.weights, device=dev)
    M, cmax = cids.shape
    out = (torch.empty((M, cmax), dtype=torch.float32, device=dev),
           torch.empty(M, dtype=torch.float32, device=dev),
           torch.empty(1, dtype=torch.int32, device=dev))

    def step():
        v.verify(vis, ids, cids, lens, out=out)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps); timing {args.steps} steps")

    # Untimed profiled steps: every stage, for the breakdown and to find the
    # dominant kernel.
    nprof = 2
    v.profile(True)
    for _ in range(nprof):
        step()
    stages = v.profile_read()
    v.profile(False)
    flops = stage_flops(cfg, cfg.n_prefix, lens)
    nbytes = stage_bytes(cfg, cfg.n_prefix, lens)
    per_step = {k: ms / nprof for k, (ms, n) in stages.items()}
    if args.stages:
        for k, ms in sorted(per_step.items(), key=lambda kv: -kv[1]):
            tf = flops.get(k, 0.0) / (ms * 1e-3) / 1e12 if ms > 0 else 0.0
            log(f"  {k:28s} {ms:8.3f} ms/step  {stages[k][1] // nprof:4d} launches"
                + (f"  {tf:7.1f} TFLOP/s" if k in flops else ""))
    ktime = {k: sum(stages.get(s, (0.0, 0))[0] for s in ss) for k, ss in KERNELS.items()}
    kname = max(ktime, key=ktime.get)
    kst = KERNELS[kname]

    # Timed steps: events around the dominant kernel's launches only.
    v.profile(True, kinds=sorted({s.split(".", 1)[1] for s in kst}))
    st = torch.cuda.current_stream(dev)
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    marks[0].record(st)
    for i in range(args.steps):
        step()
        marks[i + 1].record(st)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    timed = v.profile_read()
    v.profile(False)
    step_ms = sorted(a.elapsed_time(b) for a, b in zip(marks[:-1], marks[1:]))

    def pct(q):
        return round(step_ms[min(len(step_ms) - 1, int(round(q * (len(step_ms) - 1))))], 3)

    ms_step = (t1 - t0) * 1e3 / args.steps
    tokens = sum(lens)
    value = tokens / (ms_step / 1e3)
    launches = sum(timed.get(s, (0.0, 0))[1] for s in kst)
    kflops = sum(flops.get(s, 0.0) for s in kst) * args.steps
    avg_ms = sum(timed.get(s, (0.0, 0))[0] for s in kst) / max(launches, 1)
    achieved = kflops / launches / (avg_ms * 1e-3) / 1e12
    roofline = {"kernel": kname, "bound": "mfma", "achieved": round(achieved, 1),
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": measured_traffic(kname),
                "launches": launches, "avg_launch_ms": round(avg_ms, 4),
                "flop_per_launch": kflops / launches}

    total = sum(per_step.values())
    gemm = sum(per_step.get(f"verify.{k}", 0.0)
               for k in ("qkv_rope", "o_proj", "gate_up_swiglu", "down_proj", "lm_head_lse"))
    attn = sum(per_step.get(f"verify.{k}", 0.0)
               for k in ("attention", "cand_attention", "attn_merge"))
    result = {
        "metric": METRIC if args.workload == 2 else "candidate tokens scored/sec and ms per verify pass",
        "value": round(value, 1), "unit": "candidate tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "ms_per_step_p10_p50_p90": [pct(0.1), pct(0.5), pct(0.9)],
        "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None,
        "dtype": (f"bf16 weights, fp16 MFMA operands, fp32 accumulation; "
                  f"{v.c.split_layers} precise layer(s) with fp16 value+remainder operands"
                  if cfg.dtype == W.BF16 else "f32"),
        "data": "synthetic (seeded, random-init weights)",
        "config": {"workload": cfg.name, "layers": cfg.n_layers, "d_model": cfg.d_model,
                   "heads": f"{cfg.n_heads}/{cfg.n_kv_heads}", "d_ff": cfg.d_ff,
                   "vocab": cfg.vocab, "prefix": cfg.n_prefix, "visual_rows": cfg.n_visual,
                   "candidates": M, "cand_len": cmax, "tokens_scored": tokens},
        "breakdown": {"kernel_ms": round(total, 3), "gemm_ms": round(gemm, 3),
                      "attention_ms": round(attn, 3),
                      # every stage of the untimed profiled pass with its
                      # algorithmic work: ms per pass, TF/s and GB/s, the
                      # fractions of the bf16 MFMA peak and of HBM peak, the
                      # bound its arithmetic intensity selects (ridge 312.5
                      # FLOP/B) and the roofline fraction against that bound
                      "stages": {k.split(".", 1)[1]: stage_row(flops.get(k, 0.0), nbytes.get(k),
                                                               per_step[k])
                                 for k in sorted(set(flops) | set(nbytes))
                                 if per_step.get(k, 0.0) > 0}},
        "roofline": roofline,
    }
    if not args.no_next_rows:
        result["next_rows"] = time_next_rows(v, cids, lens, dev, max(3, args.steps // 2), log)
        result["next_rows"].update(time_draft(dev, log))
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, log)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
