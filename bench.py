#!/usr/bin/env python3
"""Fastmax forward throughput on one MI355X (tokens*heads/s) with its
roofline fraction and the fp64 CPU oracle timed beside it.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

One step = one full forward (standardisation, moments, query contraction,
divide) over the whole workload, inputs already resident in HBM.  Prints ONE
JSON line.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "Fastmax fwd tokens·heads/s on 1 GPU (D=64,p=2,causal); % MFMA peak"
PEAK = {  # MI355X published dense peaks
    ("mfma", "bf16"): 2500.0,   # TFLOP/s
    ("mfma", "f16"): 2500.0,
    ("mfma", "f32"): 157.3,
    # fp32 vector peak as published (packed FMA: 256 CU x 4 SIMD x 16 lanes x
    # 2 x 2 x 2.4 GHz); the float32 kernels are built without packed fp32 math,
    # so they can reach at most half of it
    ("alu", "f32"): 157.3,
    ("hbm", None): 8000.0,      # GB/s
}


def n_features(D, p):
    return 1 + D + (D * (D + 1) // 2 if p == 2 else 0)


def fwd_flops(B, H, N, D, p):
    """Algorithmic forward flops: moment build + query contraction, each
    2*P*(D+1) per token per head (symmetric packing of the quadratic term)."""
    return 4.0 * n_features(D, p) * (D + 1) * B * H * N


def bwd_flops(B, H, N, D, p):
    """Algorithmic backward flops (moment form of the custom gradient), per
    token per head 2 x [P(D+1) forward state + D^2(D+1) dq contraction
    + P(D+1) reverse state (symmetric in q (x) q) + D^2(D+1) dk contraction
    + P D reverse dv state + P D dv contraction]; p = 2 only."""
    if p != 2:
        return None
    P = n_features(D, p)
    per = 2 * (2 * P * (D + 1) + 2 * D * D * (D + 1) + 2 * P * D)
    return float(per) * B * H * N


def source_hash():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2402_07901_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode())
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(kernel, workload):
    """Measured HBM bytes per launch from profiles/traffic.json, if it was
    taken on the current kernel sources; otherwise None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    ent = data.get(f"{kernel}@{workload}")
    if not ent or ent.get("source_hash") != source_hash():
        return None
    return ent.get("bytes_per_launch")


def cpu_baseline(w, inp_bits, scale=1.0, budget_s=12.0, dropout=None):
    """The fp64 oracle (factorised form) on a bounded sample of the workload:
    the workload's own heads, in groups of one head per host thread (the
    oracle runs one head per thread), until the whole workload is done or
    about budget_s seconds have passed.  With ``dropout`` the oracle's masked
    factorised forward, its keep bits drawn (untimed) by the oracle."""
    import numpy as np

    import oracle
    from paper_2402_07901_amd.inputs import bf16_bits_to_f64
    threads = oracle.num_threads()
    total = w.B * w.H
    group = max(1, min(total, threads))

    def cut(x, sel):
        a = np.stack([x[b, h] for b, h in sel])[None]
        return bf16_bits_to_f64(a) if w.dtype == "bf16" else a.astype(np.float64)
    done, dt, first = 0, 0.0, None
    while done < total and dt < budget_s:
        sel = [(i // w.H, i % w.H) for i in range(done, min(total, done + group))]
        q, k, v = (cut(inp_bits[n], sel) for n in ("q", "k", "v"))
        if first is None:
            first = (q, k, v)
        if dropout is None:
            t0 = time.perf_counter()
            oracle.fwd_fact(q, k, v, w.p, w.causal, scale=scale)
        else:
            bits = oracle.dropout_mask(1, len(sel), w.N, w.D, float(np.float32(dropout)), done)
            t0 = time.perf_counter()
            oracle.fwd_drop_fact(q, k, v, bits, float(np.float32(dropout)), w.causal, scale=scale)
        dt += time.perf_counter() - t0
        done += len(sel)
    sample = (f"all {total} heads of the workload" if done == total
              else f"first {done} of the workload's {total} heads") + f" at full N={w.N}"
    rec = {"value": done * w.N / dt, "unit": "tokens*heads/s", "cores": group,
           "kind": "oracle",
           "sample": sample + (f" (fwd_fact, {dt:.1f} s)" if dropout is None
                               else f" (fwd_drop_fact, {dt:.1f} s)"),
           "cpu_model": cpu_model()}
    if w.N <= 4096 and dropout is None:
        # the explicit N x N definition as well, on the first group
        t0 = time.perf_counter()
        oracle.fwd_brute(*first, w.p, w.causal, scale=scale)
        rec["brute_force_value"] = first[0].shape[1] * w.N / (time.perf_counter() - t0)
    return rec


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="gpt_causal_bf16")
    ap.add_argument("--mode", choices=["fwd", "fwdbwd"], default="fwd",
                    help="fwd: one forward per step (the headline); fwdbwd: forward + "
                         "backward per step")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--timed-only", action="store_true",
                    help="no cold calls and no N = 8192 comparison run (for profiling: "
                         "every dispatch of the kernels is then a timed-region call)")
    ap.add_argument("--qk-scale", type=float, default=None, metavar="TAU",
                    help="time the score-scaled entry points with weights f_p(TAU q^.k^) "
                         "(e.g. 1/D, the unit-norm variant); default: the plain entry points")
    ap.add_argument("--dropout", type=float, default=None, metavar="RATE",
                    help="time the quadratic-term dropout entry points: each step draws "
                         "fresh keep bits (fastmax_dropout_mask) and runs the masked "
                         "forward (and backward in --mode fwdbwd)")
    ap.add_argument("--cold", type=int, default=None, metavar="ITERS",
                    help="after the timed region, time ITERS calls each preceded by a "
                         "512 MiB write that flushes the caches (default 10 for the bf16 "
                         "MFMA workloads, 0 otherwise)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MiB",
                    help="only run a plain device-to-device copy of this many MiB "
                         "(for scaling rocprofv3 FETCH_SIZE/WRITE_SIZE) and exit")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the Fastmax kernels here run on a single "
              "MI355X and no multi-GPU path is built (heads would shard with no "
              "communication). Use --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2402_07901_amd import fastmax as fm
    from paper_2402_07901_amd.inputs import WORKLOADS, make_inputs, workload_inputs

    dev = torch.device("cuda:0")
    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        for _ in range(max(1, args.steps)):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n, "steps": max(1, args.steps)}))
        return

    w = WORKLOADS[args.workload]
    fm.lib()
    # dO (when timed) is drawn on the host by the same seeded recipe, after q, k, v
    inp = make_inputs(w.B, w.H, w.N, w.D, w.key, w.dtype, w.mask_frac, w.mask_scale,
                      with_dout=(args.mode == "fwdbwd"), want64=False)

    def to_dev(x):
        if w.dtype == "bf16":
            return torch.from_numpy(x.view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(x).to(dev)

    q, k, v = (to_dev(inp[n]) for n in ("q", "k", "v"))
    dout = to_dev(inp["dout"]) if args.mode == "fwdbwd" else None
    out = torch.empty_like(q)
    g = torch.empty((w.B, w.H, w.N), dtype=torch.float32, device=dev)
    dt = fm.BF16 if w.dtype == "bf16" else fm.F32
    drop = args.dropout
    if drop is not None and w.p != 2:
        print("--dropout needs a p = 2 workload (it masks the quadratic features)",
              file=sys.stderr)
        sys.exit(2)
    if drop is None:
        need = fm.workspace_bytes(w.B, w.H, w.N, w.D, w.p, w.causal, dt, False)
    else:
        need = fm.dropout_workspace_bytes(w.B, w.H, w.N, w.D, w.causal, dt, False)
        bits = torch.empty((w.B, w.H, w.N, fm.mask_words(w.D)), dtype=torch.int32, device=dev)
    ws = torch.empty(max(need, 1), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    scale = 1.0 if args.qk_scale is None else args.qk_scale

    if args.mode == "fwdbwd":
        if drop is None:
            need_b = fm.workspace_bytes(w.B, w.H, w.N, w.D, w.p, w.causal, dt, True)
        else:
            need_b = fm.dropout_workspace_bytes(w.B, w.H, w.N, w.D, w.causal, dt, True)
        ws_b = torch.empty(max(need_b, 1), dtype=torch.uint8, device=dev)
        dq, dk, dv = (torch.empty_like(q) for _ in range(3))
    bwd_start = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    fwd_start = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]

    def step(i=None):
        if drop is not None:
            # a training step draws fresh keep bits, then runs the masked calls
            rc = fm.fastmax_dropout_mask_raw(bits, w.B, w.H, w.N, w.D, drop,
                                             0x5EED0000 + (i or 0), stream)
            if rc != fm.OK:
                raise fm.FastmaxError(rc, "fastmax_dropout_mask")
            if i is not None:
                fwd_start[i].record(stream)
            rc = fm.fastmax_fwd_dropout_raw(q, k, v, out, g, bits, drop, w.B, w.H, w.N, w.D,
                                            w.causal, scale, dt, ws, need, stream)
        else:
            rc = fm.fastmax_fwd_raw(q, k, v, out, g, w.B, w.H, w.N, w.D, w.p, w.causal, dt, ws,
                                    need, stream, args.qk_scale)
        if rc != fm.OK:
            raise fm.FastmaxError(rc, "fastmax_fwd")
        if args.mode == "fwdbwd":
            if i is not None:
                bwd_start[i].record(stream)
            if drop is not None:
                rc = fm.fastmax_bwd_dropout_raw(q, k, v, out, dout, g, bits, drop, dq, dk, dv,
                                                w.B, w.H, w.N, w.D, w.causal, scale, dt, ws_b,
                                                need_b, stream)
            else:
                rc = fm.fastmax_bwd_raw(q, k, v, out, dout, g, dq, dk, dv, w.B, w.H, w.N, w.D,
                                        w.p, w.causal, dt, ws_b, need_b, stream, args.qk_scale)
            if rc != fm.OK:
                raise fm.FastmaxError(rc, "fastmax_bwd")

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    stops = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        starts[i].record(stream)
        step(i)
        stops[i].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    fstarts = fwd_start if drop is not None else starts
    if drop is not None:
        mask_ms = [s.elapsed_time(e) for s, e in zip(starts, fwd_start)]
    if args.mode == "fwdbwd":
        fwd_ms = [s.elapsed_time(e) for s, e in zip(fstarts, bwd_start)]
        bwd_ms = [s.elapsed_time(e) for s, e in zip(bwd_start, stops)]
        launch_ms = fwd_ms
    else:
        launch_ms = [s.elapsed_time(e) for s, e in zip(fstarts, stops)]
    avg_launch_s = sum(launch_ms) / len(launch_ms) / 1e3
    ms_per_step = wall / args.steps * 1e3

    tokens_heads = w.B * w.H * w.N
    value = tokens_heads / (ms_per_step / 1e3)
    flops = fwd_flops(w.B, w.H, w.N, w.D, w.p)
    kernel = "fastmax_fwd"
    if w.p == 2 and w.dtype == "bf16" and w.D == 64 and drop is None:
        bound, unit, peak = "mfma", "TFLOP/s", PEAK[("mfma", "bf16")]
        achieved = flops / avg_launch_s / 1e12
    elif w.p == 2 and drop is None:
        # every other p = 2 case runs on the float32 MFMA kernels
        bound, unit, peak = "mfma", "TFLOP/s", PEAK[("mfma", "f32")]
        achieved = flops / avg_launch_s / 1e12
    elif w.p == 2:
        # quadratic dropout: the float32 kernels on the vector ALU
        bound, unit, peak = "alu", "TFLOP/s", PEAK[("alu", "f32")]
        achieved = flops / avg_launch_s / 1e12
    else:
        bound, unit, peak = "hbm", "GB/s", PEAK[("hbm", None)]
        elt = 2 if w.dtype == "bf16" else 4
        achieved = tokens_heads * (4 * w.D * elt + 4) / avg_launch_s / 1e9

    rec = {
        "metric": METRIC if (w.name == "gpt_causal_bf16" and args.mode == "fwd" and drop is None)
                  else f"Fastmax {args.mode} tokens·heads/s on 1 GPU ({w.name}"
                       + ("" if drop is None else f", quadratic dropout {drop}") + ")",
        "value": value,
        "unit": "tokens*heads/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "mode": args.mode, "B": w.B, "H": w.H, "N": w.N,
                   "D": w.D, "p": w.p, "causal": w.causal, "io_dtype": w.dtype,
                   "global_batch": w.B, "seq_len": w.N, "parallelism": "none (1 GPU)",
                   "qk_scale": 1.0 if args.qk_scale is None else args.qk_scale,
                   "dropout": drop},
        "roofline": {"bound": bound, "achieved": achieved, "peak": peak, "unit": unit,
                     "frac": achieved / peak, "traffic": load_traffic(kernel, w.name),
                     "kernel": kernel, "avg_launch_ms": avg_launch_s * 1e3,
                     "algorithmic_flops_per_launch": flops},
    }
    if args.mode == "fwdbwd":
        bms = sum(bwd_ms) / len(bwd_ms)
        bf = bwd_flops(w.B, w.H, w.N, w.D, w.p)
        rec["backward"] = {"avg_ms": bms,
                           "note": "fastmax_bwd call (all its kernels), HIP events on the stream"}
        if bf is not None and drop is not None:
            ach = bf / (bms / 1e3) / 1e12
            rec["backward"].update({"algorithmic_flops_per_call": bf, "achieved": ach,
                                    "unit": "TFLOP/s", "bound": "alu",
                                    "peak": PEAK[("alu", "f32")],
                                    "frac": ach / PEAK[("alu", "f32")], "traffic": None})
        elif bf is not None:
            # bf16 D = 64: the fp16 MFMA kernels; every other p = 2 case the
            # float32 MFMA kernels
            ach = bf / (bms / 1e3) / 1e12
            pk = PEAK[("mfma", "bf16" if w.dtype == "bf16" and w.D == 64 else "f32")]
            rec["backward"].update({"algorithmic_flops_per_call": bf, "achieved": ach,
                                    "unit": "TFLOP/s", "bound": "mfma", "peak": pk,
                                    "frac": ach / pk,
                                    "traffic": load_traffic("fastmax_bwd", w.name)})
    rec["roofline"]["median_launch_ms"] = float(np.median(launch_ms))
    if drop is not None:
        # the generator's cost per step (its own kernel), beside the forward
        mw = fm.mask_words(w.D)
        mms = sum(mask_ms) / len(mask_ms)
        rec["dropout_mask"] = {"avg_ms": mms, "words": w.B * w.H * w.N * mw,
                               "written_GBps": w.B * w.H * w.N * mw * 4 / (mms / 1e3) / 1e9}
        rec["roofline"]["traffic"] = None
    if args.mode == "fwdbwd":
        rec["backward"]["median_ms"] = float(np.median(bwd_ms))

    # cold calls: caches flushed by a 512 MiB write before each one
    cold = args.cold if args.cold is not None else (
        10 if w.dtype == "bf16" and w.p == 2 and drop is None else 0)
    if args.timed_only:
        cold = 0
    if cold > 0:
        flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * cold)]

        def cold_median(call):
            for i in range(cold):
                flush.fill_(i & 255)
                ev[2 * i].record(stream)
                call()
                ev[2 * i + 1].record(stream)
            torch.cuda.synchronize()
            return float(np.median([ev[2 * i].elapsed_time(ev[2 * i + 1]) for i in range(cold)]))

        def fwd_call():
            rc = fm.fastmax_fwd_raw(q, k, v, out, g, w.B, w.H, w.N, w.D, w.p, w.causal, dt, ws,
                                    need, stream, args.qk_scale)
            if rc != fm.OK:
                raise fm.FastmaxError(rc, "fastmax_fwd")

        def bwd_call():
            rc = fm.fastmax_bwd_raw(q, k, v, out, dout, g, dq, dk, dv, w.B, w.H, w.N, w.D, w.p,
                                    w.causal, dt, ws_b, need_b, stream, args.qk_scale)
            if rc != fm.OK:
                raise fm.FastmaxError(rc, "fastmax_bwd")

        rec["cold"] = {"iters": cold, "flush_bytes": 512 << 20,
                       "fwd_median_ms": cold_median(fwd_call)}
        if args.mode == "fwdbwd":
            rec["cold"]["bwd_median_ms"] = cold_median(bwd_call)
        del flush

    # linear in N (long non-causal workload): the same recipe at N = 8192
    if (not w.causal and w.N > 8192 and w.dtype == "bf16" and w.p == 2 and args.mode == "fwd"
            and not args.timed_only and drop is None):
        n_s = 8192
        inp_s = workload_inputs(w, want64=False, N=n_s)
        qs, ks, vs = (to_dev(inp_s[n]) for n in ("q", "k", "v"))
        outs = torch.empty_like(qs)
        need_s = fm.workspace_bytes(w.B, w.H, n_s, w.D, w.p, w.causal, dt, False)
        ws_s = torch.empty(max(need_s, 1), dtype=torch.uint8, device=dev)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * max(args.steps, 1))]
        for i in range(args.warmup + max(args.steps, 1)):
            j = i - args.warmup
            if j >= 0:
                ev[2 * j].record(stream)
            rc = fm.fastmax_fwd_raw(qs, ks, vs, outs, None, w.B, w.H, n_s, w.D, w.p, w.causal,
                                    dt, ws_s, need_s, stream, args.qk_scale)
            if rc != fm.OK:
                raise fm.FastmaxError(rc, "fastmax_fwd")
            if j >= 0:
                ev[2 * j + 1].record(stream)
        torch.cuda.synchronize()
        t_s = float(np.median([ev[2 * j].elapsed_time(ev[2 * j + 1])
                               for j in range(max(args.steps, 1))]))
        t_f = rec["roofline"]["median_launch_ms"]
        rec["linear_in_n"] = {"n_small": n_s, "n_full": w.N, "small_median_ms": t_s,
                              "full_median_ms": t_f, "ratio": t_f / t_s,
                              "ideal": w.N / n_s}
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(w, inp, 1.0 if args.qk_scale is None else args.qk_scale,
                                           dropout=drop)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
