"""Throughput of the fused quantized state update on one MI355X.

One step = one decode token through every SSM layer of the workload: for each
layer, ssmq_state_update reads the stored state, applies the recurrence, writes
y and re-quantizes the state in place. Inputs are synthetic (seeded, shaped like
the paper's hybrid Mamba-2 models) and resident in HBM before timing starts;
each layer keeps one input set across steps while the step counter t advances.

Prints one JSON line. `value` is the state read+write bandwidth (GB/s) of the
headline variant (bf16 state, Weyl dither); the other formats and rules are
reported under "variants".
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

PEAK_HBM_GBPS = 8000.0  # MI355X HBM3E, vendor figure
METRIC = "quantized state-update HBM GB/s (state R+W) & % of peak; decode steps/s"


def parse_args():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="hybrid_m2_stack")
    ap.add_argument("--variants", default="bf16:weyl,bf16:sr,bf16:rtn,e4m3:weyl,e4m3:sr,e4m3:rtn",
                    help="comma-separated format:rule list; the first is the headline")
    ap.add_argument("--layers", type=int, default=0, help="override the layer count (0 = workload's)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU time of the oracle baseline sample (0 disables it)")
    ap.add_argument("--no-copy", action="store_true", help="skip the copy-bandwidth ceiling")
    return ap.parse_args()


def state_bytes_per_entry(fmt: str) -> float:
    return {"bf16": 2, "fp16": 2, "e4m3": 1, "fp32": 4}[fmt]


def main() -> int:
    args = parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this build measures one GPU only; the state update shards "
                                   "by batch or head with no communication, so --gpus must be 1"}))
        return 2

    import torch

    import paper_2609_39185_amd as ssmq
    from paper_2609_39185_amd import workloads as wl

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = wl.WORKLOADS[args.workload]
    L = args.layers or w.layers
    b, H, P, N, G = w.batch, w.nheads, w.headdim, w.dstate, w.ngroups
    n_entries = w.entries_per_layer
    variants = [tuple(v.split(":")) for v in args.variants.split(",") if v]
    fmts = sorted({f for f, _ in variants})

    # ---- resident inputs and states -------------------------------------------------
    layers = []
    for ell in range(L):
        A, D = wl.layer_params(w.family, H, N, seed=1000 + ell, device=dev)
        x, dt, B, C = wl.step_inputs(b, H, P, N, G, seed=2000 + ell, device=dev)
        y = torch.empty((b, H, P), dtype=torch.float32, device=dev)
        states = {}
        for f in fmts:
            states[f] = wl.initial_state(f, b, H, P, N, seed=3000 + ell, group=w.scale_group,
                                         device=dev)
        layers.append(dict(A=A, D=D, x=x, dt=dt, B=B, C=C, y=y, states=states))
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)

    def one_step(fmt, rule, t, events=None):
        for ell, lay in enumerate(layers):
            st, sc = lay["states"][fmt]
            if events is not None:
                events[ell][0].record(stream)
            ssmq.state_update(st, sc, lay["x"], lay["dt"], lay["A"], lay["B"], lay["C"], lay["D"],
                              lay["y"], rule=rule, fmt=fmt, dither_block=w.dither_block,
                              scale_group=w.scale_group, layer=ell, step=t, seed=0,
                              stream=stream)
            if events is not None:
                events[ell][1].record(stream)

    results = {}
    t_global = 1
    for fmt, rule in variants:
        for _ in range(args.warmup):
            one_step(fmt, rule, t_global)
            t_global += 1
        torch.cuda.synchronize()
        ev = [[[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(L)]
              for _ in range(args.steps)]
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record(stream)
        for k in range(args.steps):
            one_step(fmt, rule, t_global, ev[k])
            t_global += 1
        stop.record(stream)
        torch.cuda.synchronize()
        total_ms = start.elapsed_time(stop)
        launch_ms = [e[0].elapsed_time(e[1]) for step_ev in ev for e in step_ev]
        ms_step = total_ms / args.steps
        sbytes = n_entries * state_bytes_per_entry(fmt) * 2
        if fmt == "e4m3":
            sbytes += (n_entries // (w.scale_group or P * N)) * 8
        avg_launch_ms = sum(launch_ms) / len(launch_ms)
        results[f"{fmt}:{rule}"] = {
            "ms_per_step": ms_step,
            "steps_per_s": 1000.0 / ms_step,
            "state_GBps": sbytes * L / (ms_step * 1e6),
            "pct_of_peak": 100.0 * sbytes * L / (ms_step * 1e6) / PEAK_HBM_GBPS,
            "kernel_avg_us": avg_launch_ms * 1e3,
            "kernel_state_GBps": sbytes / (avg_launch_ms * 1e6),
            "state_bytes_per_launch": sbytes,
        }

    # ---- copy ceiling: read + write the same bytes as one bf16 layer -----------------
    copy = None
    if not args.no_copy:
        nbytes = n_entries * 2
        src = torch.empty(nbytes // 4, dtype=torch.int32, device=dev).random_()
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        reps = 20
        e0.record(stream)
        for _ in range(reps):
            dst.copy_(src)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        copy = {"bytes_read_plus_written": 2 * nbytes, "us": ms * 1e3,
                "GBps": 2 * nbytes / (ms * 1e6)}
        del src, dst

    # ---- CPU baseline: the oracle on a bounded sample of one layer -------------------
    cpu = None
    if args.cpu_seconds > 0:
        cpu = cpu_baseline(w, variants[0], args.cpu_seconds)

    head_fmt, head_rule = variants[0]
    head = results[f"{head_fmt}:{head_rule}"]
    roof = {
        "bound": "hbm",
        "achieved": head["kernel_state_GBps"],
        "peak": PEAK_HBM_GBPS,
        "unit": "GB/s",
        "frac": head["kernel_state_GBps"] / PEAK_HBM_GBPS,
        "traffic": None,
        "kernel": "k_update_head",
        "algorithmic_bytes_per_launch": head["state_bytes_per_launch"],
        "avg_launch_us": head["kernel_avg_us"],
    }
    line = {
        "metric": METRIC,
        "value": head["state_GBps"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": head_fmt,
        "data": "synthetic",
        "config": {"workload": w.name, "family": w.family, "batch": b, "layers": L, "nheads": H,
                   "headdim": P, "dstate": N, "ngroups": G, "format": head_fmt,
                   "rule": head_rule, "dither_block": w.dither_block,
                   "scale_group": w.scale_group or P * N},
        "pct_of_peak": head["pct_of_peak"],
        "steps_per_s": head["steps_per_s"],
        "roofline": roof,
        "cpu_baseline": cpu,
        "copy_ceiling": copy,
        "variants": results,
    }
    print(json.dumps(line), flush=True)
    return 0


def cpu_baseline(w, variant, target_s):
    """Time the oracle on whole head tiles of one layer until ~target_s of CPU work."""
    import numpy as np
    import torch

    import oracle
    from paper_2609_39185_amd import workloads as wl

    fmt, rule = variant
    P, N = w.headdim, w.dstate
    A, D = wl.layer_params(w.family, w.nheads, N, seed=1000)
    x, dt, B, C = wl.step_inputs(1, w.nheads, P, N, w.ngroups, seed=2000)
    codes, scale = wl.initial_state(fmt, 1, w.nheads, P, N, seed=3000, group=w.scale_group)
    codes_np = wl.to_numpy_codes(fmt, codes)
    args = (None if scale is None else scale.numpy(), x.numpy(), dt.numpy(), A.numpy(),
            B.numpy(), C.numpy(), D.numpy())

    def run(nh):
        c = codes_np[:, :nh]
        sc = None if args[0] is None else args[0][:nh]
        t0 = time.perf_counter()
        oracle.state_update(fmt, rule, c, sc, args[1][:, :nh], args[2][:, :nh], args[3][:nh],
                            args[4][:, :1], args[5][:, :1], args[6][:nh], block=w.dither_block,
                            group=w.scale_group, step=1)
        return time.perf_counter() - t0

    probe_heads = w.nheads // w.ngroups   # the heads of one B/C group
    t_probe = run(probe_heads)
    per_head = t_probe / probe_heads
    reps = max(1, int(target_s / max(t_probe, 1e-6)))
    total = 0.0
    for _ in range(reps):
        total += run(probe_heads)
    entries = reps * probe_heads * P * N
    bytes_rw = entries * state_bytes_per_entry(fmt) * 2
    return {
        "value": bytes_rw / total / 1e9,
        "unit": "GB/s",
        "cores": 1,
        "kind": "oracle",
        "sample": f"{reps} x {probe_heads} head tiles ({P}x{N}) of one layer of {w.name}, "
                  f"{fmt} {rule}, single-threaded C oracle, {total:.1f} s",
        "us_per_head_tile": per_head * 1e6,
    }


if __name__ == "__main__":
    sys.exit(main())
