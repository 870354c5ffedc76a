"""Throughput of the fused quantized state update on one MI355X.

One step = one decode token through every SSM layer of the workload: for each
layer, ssmq_state_update reads the stored state, applies the recurrence, writes
y and re-quantizes the state in place. Inputs are synthetic (seeded, shaped like
the paper's hybrid Mamba-2 models) and resident in HBM before timing starts;
each layer keeps one input set across steps while the step counter t advances.

Prints one JSON line. `value` is the state read+write bandwidth (GB/s) of the
headline variant (bf16 state, Weyl dither); the other formats and rules are
reported under "variants". Each variant's timed region is exactly --steps steps
between two events on the launch stream; since that stream carries only the
update launches, the region's time over their number is the average launch
duration behind roofline.achieved. With --rounds R the variants are timed in R
interleaved rounds and each reports its median round; --graph replays the timed
steps from one HIP graph. cpu_baseline times the CPU oracle on one thread and on
every usable core (at most 16).

Other modes print their own JSON line instead: --entry-points (ssmq_requantize
and ssmq_dither_fill alone), --state-error (quantized states against an FP32
twin in lockstep), --replay (open-loop replay of synthetic recorded traces); the
--summarize-* options turn rocprofv3 CSV output into the summaries under
profiles/.
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
CAL_ELEMS = 1 << 28      # calibration kernel: fp32 elements in and out
CAL_BYTES = CAL_ELEMS * 4
KERNEL_SOURCES = ("ssmq_kernels.hip", "ssmq_device.hpp", "ssmq_launch.hpp", "ssmq_abi.cpp")
PROFILE_DIR = os.path.join(ROOT, "profiles")
METRIC = "quantized state-update HBM GB/s (state R+W) & % of peak; decode steps/s"


def parse_args():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps (default 20; with --state-error the workload's steps)")
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=None,
                    help="default hybrid_m2_stack (m1_long with --state-error)")
    ap.add_argument("--state-error", action="store_true",
                    help="instead of throughput: quantized states vs an FP32 twin in lockstep")
    ap.add_argument("--block", type=int, default=512, help="--state-error: steps per reported block")
    ap.add_argument("--se-format", default="fp16", help="--state-error: storage format")
    ap.add_argument("--se-group", type=int, default=16, help="--state-error: entries per scale")
    ap.add_argument("--se-memory", default="short", choices=("short", "trained"),
                    help="--state-error: decay-rate recipe")
    ap.add_argument("--se-cc", type=int, default=0,
                    help="--state-error: also run checkpointed rules, rounding every k-th write")
    ap.add_argument("--entry-points", action="store_true",
                    help="instead of the fused step: ssmq_requantize and ssmq_dither_fill on one "
                         "layer's entries (GB/s of their own reads and writes)")
    ap.add_argument("--replay", action="store_true",
                    help="instead of throughput: open-loop replay of synthetic recorded traces")
    ap.add_argument("--rp-batch", type=int, default=0,
                    help="--replay: sequences in the traced layer (0 = the workload's batch)")
    ap.add_argument("--rp-memory", default="trained", choices=("short", "trained"),
                    help="--replay: decay-rate recipe")
    ap.add_argument("--variants", default="bf16:weyl,bf16:sr,bf16:rtn,bf16:philox,"
                                          "e4m3:weyl,e4m3:sr,e4m3:rtn,e4m3:philox,"
                                          "int8:weyl,int8:sr,int8:rtn,int8:philox,"
                                          "int4:weyl,int4:sr,int4:rtn",
                    help="comma-separated format[/group]:rule list (group: entries per scale, 0 = one per head); the first is the headline")
    ap.add_argument("--layers", type=int, default=0, help="override the layer count (0 = workload's)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="seconds of each oracle baseline leg, one thread and all cores (0 disables it)")
    ap.add_argument("--rounds", type=int, default=1,
                    help="timed regions per variant, interleaved across variants; the median is reported")
    ap.add_argument("--graph", action="store_true",
                    help="replay the timed steps from one HIP graph (removes host launch gaps)")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the other workloads (HIP-graph timing, oracle timing, config-3 "
                         "state error) in the default line")
    ap.add_argument("--config-steps", type=int, default=20,
                    help="timed steps per rule for each of the other workloads")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the streaming-kernel bandwidth ceiling")
    ap.add_argument("--summarize-profiles", nargs=3, metavar=("TRACE_DIR", "FETCH_DIR", "WRITE_DIR"),
                    help="turn rocprofv3 CSV output (kernel trace with --stats, then --pmc "
                         "FETCH_SIZE, then --pmc WRITE_SIZE) into the summaries under profiles/")
    ap.add_argument("--summarize-entry-trace", metavar="TRACE_DIR",
                    help="write the entry-point kernel trace summary under profiles/")
    ap.add_argument("--summarize-trace", nargs=2, metavar=("TRACE_DIR", "NAME"),
                    help="turn a rocprofv3 --kernel-trace --stats run of --replay into "
                         "profiles/NAME.kernel_trace.md")
    ap.add_argument("--summarize-valu", metavar="PMC_DIR",
                    help="turn a rocprofv3 --pmc run of SQ_WAVES, SQ_INSTS_VALU, "
                         "SQ_ACTIVE_INST_VALU and GRBM_GUI_ACTIVE into profiles/...valu.md")
    ap.add_argument("--summarize-mix", nargs=2, metavar=("PMC_DIR_A", "PMC_DIR_B"),
                    help="turn the two --pmc runs of the instruction-mix counters into "
                         "profiles/...valu_mix.md")
    return ap.parse_args()


def state_bytes_per_entry(fmt: str) -> float:
    return {"bf16": 2, "fp16": 2, "e4m3": 1, "fp32": 4, "int8": 1, "int4": 0.5}[fmt]


def state_bytes_per_launch(w, fmt: str, group=None) -> int:
    """Algorithmic bytes of one layer's update: codes read and written, plus each
    group scale read and written (4 B each way). group: entries per scale (0 = one
    head; None = the workload's own)."""
    from paper_2609_39185_amd import workloads as wl

    n = w.entries_per_layer
    total = int(n * state_bytes_per_entry(fmt) * 2)
    if fmt in ("e4m3", "int8", "int4"):
        if group is None:
            group = wl.scale_group_of(w, fmt)
        total += (n // (group or w.headdim * w.dstate)) * 8
    return total


def parse_variant(spec: str, w):
    """'fmt:rule' or 'fmt/group:rule' (group: entries per scale of a scaled format,
    0 = one per head) -> dict(key, fmt, rule, group)."""
    from paper_2609_39185_amd import workloads as wl

    head, rule = spec.split(":")
    fmt, _, g = head.partition("/")
    if g and fmt not in ("e4m3", "int8", "int4"):
        raise SystemExit(f"variant {spec}: only e4m3, int8 and int4 take a scale group")
    group = int(g) if g else wl.scale_group_of(w, fmt)
    return {"key": spec, "fmt": fmt, "rule": rule, "group": group}


def main() -> int:
    args = parse_args()
    if args.workload is None:
        args.workload = "m1_long" if (args.state_error or args.replay) else "hybrid_m2_stack"
    if args.summarize_profiles:
        return summarize_profiles(args.workload, *args.summarize_profiles)
    if args.summarize_valu:
        return summarize_valu(args.workload, args.summarize_valu)
    if args.summarize_mix:
        return summarize_mix(args.workload, *args.summarize_mix)
    if args.summarize_trace:
        return summarize_replay_trace(*args.summarize_trace)
    if args.summarize_entry_trace:
        return summarize_entry_points_trace(args.summarize_entry_trace)
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this benchmark measures one GPU only; the state update shards "
                                   "by batch or head with no communication, so --gpus must be 1"}))
        return 2
    if args.rounds < 1:
        print(json.dumps({"error": "--rounds must be at least 1"}))
        return 2

    import torch

    import paper_2609_39185_amd as ssmq
    from paper_2609_39185_amd import workloads as wl

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = wl.WORKLOADS[args.workload]
    if args.replay:
        res = replay_study(w, steps=args.steps or 2048, batch=args.rp_batch or w.batch,
                           block=args.block, memory=args.rp_memory, device=dev)
        print(json.dumps(res), flush=True)
        return 0
    if args.entry_points:
        res = entry_point_rates(w, steps=args.steps or 10, warmup=args.warmup, device=dev)
        print(json.dumps(res), flush=True)
        return 0
    if args.state_error:
        res = state_error_study(w, steps=args.steps or w.steps, layers=args.layers or w.layers,
                                block=args.block, device=dev, fmt=args.se_format,
                                group=args.se_group, memory=args.se_memory, cc=args.se_cc)
        print(json.dumps(res), flush=True)
        return 0
    if args.steps is None:
        args.steps = 20
    L = args.layers or w.layers
    b, H, P, N, G = w.batch, w.nheads, w.headdim, w.dstate, w.ngroups
    n_entries = w.entries_per_layer
    variants = [parse_variant(v, w) for v in args.variants.split(",") if v]
    stored = sorted({(v["fmt"], v["group"]) for v in variants})

    # ---- resident inputs and states -------------------------------------------------
    layers = []
    for ell in range(L):
        A, D = wl.layer_params(w.family, H, N, seed=1000 + ell, device=dev)
        x, dt, B, C = wl.step_inputs(b, H, P, N, G, seed=2000 + ell, device=dev)
        y = torch.empty((b, H, P), dtype=torch.float32, device=dev)
        states = {}
        for f, g in stored:
            states[(f, g)] = wl.initial_state(f, b, H, P, N, seed=3000 + ell, group=g, device=dev)
        layers.append(dict(A=A, D=D, x=x, dt=dt, B=B, C=C, y=y, states=states))
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)

    def one_step(var, t, events=None, on=None):
        for ell, lay in enumerate(layers):
            st, sc = lay["states"][(var["fmt"], var["group"])]
            if events is not None:
                events[ell][0].record(stream)
            ssmq.state_update(st, sc, lay["x"], lay["dt"], lay["A"], lay["B"], lay["C"], lay["D"],
                              lay["y"], rule=var["rule"], fmt=var["fmt"],
                              dither_block=w.dither_block, scale_group=var["group"], layer=ell,
                              step=t, seed=0, stream=on or stream)
            if events is not None:
                events[ell][1].record(stream)

    results = {}
    t_global = 1
    launches = args.steps * L
    round_ms = {v["key"]: [] for v in variants}

    def timed_region(var):
        """Warm-up steps, then exactly --steps timed steps; returns the region's ms."""
        nonlocal t_global
        for _ in range(args.warmup):
            one_step(var, t_global)
            t_global += 1
        torch.cuda.synchronize()
        # Timed region: exactly --steps steps between two events on the launch stream.
        # The stream holds only the update launches, so the region's time divided by
        # their number is the average launch duration (gaps included).
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        if args.graph:
            # All launches of the timed steps (each with its own step t) are captured
            # into one HIP graph beforehand; the timed region replays it once.
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                cap = torch.cuda.current_stream(dev)
                for k in range(args.steps):
                    one_step(var, t_global + k, on=cap)
            torch.cuda.synchronize()
            start.record(stream)
            graph.replay()
            stop.record(stream)
            t_global += args.steps
        else:
            start.record(stream)
            for k in range(args.steps):
                one_step(var, t_global)
                t_global += 1
            stop.record(stream)
        torch.cuda.synchronize()
        return start.elapsed_time(stop)

    # --rounds R > 1 interleaves the variants round by round and keeps each
    # variant's median round (the paper's kernel table takes the median of seven
    # interleaved rounds); one round is one timed region per variant.
    for _ in range(args.rounds):
        for var in variants:
            round_ms[var["key"]].append(timed_region(var))
    for var in variants:
        key = var["key"]
        rounds = sorted(round_ms[key])
        total_ms = rounds[len(rounds) // 2]
        ms_step = total_ms / args.steps
        avg_launch_ms = total_ms / launches
        # Diagnostic only: one more step with events around every launch (each pair
        # adds a few microseconds, so these durations run long).
        ev = [[[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(L)]]
        one_step(var, t_global, ev[0])
        t_global += 1
        torch.cuda.synchronize()
        per_launch = [e[0].elapsed_time(e[1]) for e in ev[0]]
        sbytes = state_bytes_per_launch(w, var["fmt"], var["group"])
        results[key] = {
            "ms_per_step": ms_step,
            "steps_per_s": 1000.0 / ms_step,
            "state_GBps": sbytes * L / (ms_step * 1e6),
            "pct_of_peak": 100.0 * sbytes * L / (ms_step * 1e6) / PEAK_HBM_GBPS,
            "kernel_avg_us": avg_launch_ms * 1e3,
            "kernel_state_GBps": sbytes / (avg_launch_ms * 1e6),
            "state_bytes_per_launch": sbytes,
            "event_bracketed_launch_us": {"avg": 1e3 * sum(per_launch) / len(per_launch),
                                          "min": 1e3 * min(per_launch),
                                          "max": 1e3 * max(per_launch)},
        }
        if args.rounds > 1:
            results[key]["rounds_kernel_avg_us"] = [1e3 * r / launches for r in round_ms[key]]

    # ---- streaming ceiling: a plain elementwise kernel of known size ----------------
    # torch.neg over 1 GiB of fp32 reads 1 GiB and writes 1 GiB; it is also the
    # kernel that calibrates the FETCH_SIZE / WRITE_SIZE counters.
    ceiling = None
    if not args.no_ceiling:
        src = torch.empty(CAL_ELEMS, dtype=torch.float32, device=dev).uniform_()
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        reps = 20
        e0.record(stream)
        for _ in range(reps):
            torch.neg(src, out=dst)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        ceiling = {"kernel": "torch.neg fp32 (1 GiB read, 1 GiB written)",
                   "bytes_read_plus_written": 2 * CAL_BYTES, "us": ms * 1e3,
                   "GBps": 2 * CAL_BYTES / (ms * 1e6)}
        del src, dst

    # ---- CPU baseline: the oracle on a bounded sample of one layer -------------------
    cpu = None
    if args.cpu_seconds > 0:
        cpu = cpu_baseline(w, variants[0], args.cpu_seconds)

    # ---- the other workloads: device time per launch, oracle time, state error ------
    configs = None
    if not args.no_configs:
        del layers
        torch.cuda.empty_cache()
        configs = config_sweep(dev, steps=args.config_steps, warmup=args.warmup,
                               cpu_seconds=min(args.cpu_seconds, 2.0))

    head_var = variants[0]
    head_fmt, head_rule = head_var["fmt"], head_var["rule"]
    head = results[head_var["key"]]
    measured = load_traffic(w.name)
    for key, r in results.items():
        t = measured.get(key) if measured else None
        r["hbm_traffic_bytes_per_launch"] = t["traffic_bytes"] if t else None
        r["kernel"] = t["kernel"] if t else "k_update_slab"
    roof = {
        "bound": "hbm",
        "achieved": head["kernel_state_GBps"],
        "peak": PEAK_HBM_GBPS,
        "unit": "GB/s",
        "frac": head["kernel_state_GBps"] / PEAK_HBM_GBPS,
        "traffic": head["hbm_traffic_bytes_per_launch"],
        "kernel": head["kernel"],
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
        "dtype": "f32",  # the arithmetic of the step; the stored format is config["format"]
        "data": "synthetic",
        "config": {"workload": w.name, "family": w.family, "batch": b, "layers": L, "nheads": H,
                   "headdim": P, "dstate": N, "ngroups": G, "format": head_fmt,
                   "rule": head_rule, "dither_block": w.dither_block,
                   "scale_group": (head_var["group"] or P * N)
                   if head_fmt in ("e4m3", "int8", "int4") else None,
                   "launch": "hip_graph" if args.graph else "stream"},
        "pct_of_peak": head["pct_of_peak"],
        "steps_per_s": head["steps_per_s"],
        "roofline": roof,
        "cpu_baseline": cpu,
        "stream_ceiling": ceiling,
        "variants": results,
        "targets": targets_summary(results),
        "configs": configs,
    }
    print(json.dumps(line), flush=True)
    return 0


SE_RULES = (("rtn", 0), ("sr", 0), ("sr", 1), ("weyl", 0))  # (rule, seed sigma)
TAU_EDGES = (10.0, 100.0, 1000.0)  # memory bins: tau < 10, 10-100, 100-1000, >= 1000 steps


def mean_step_size() -> float:
    """E[softplus(z - 4)], z ~ N(0, 1): the mean of the synthetic step sizes."""
    import numpy as np

    z = np.linspace(-12.0, 12.0, 240001)
    pdf = np.exp(-0.5 * z * z) / np.sqrt(2.0 * np.pi)
    return float(np.trapezoid(np.logaddexp(0.0, z - 4.0) * pdf, z))


def decode_state(fmt: str, codes, scale, group: int):
    """fp32 values of a stored state on the GPU (torch), for the error metric only:
    fp16/bf16 reinterpret, E4M3 and INT8/INT4 times their group scale."""
    import torch

    if fmt == "fp32":
        return codes.view(torch.float32)
    if fmt in ("fp16", "bf16"):
        return codes.view({"fp16": torch.float16, "bf16": torch.bfloat16}[fmt]).float()
    if fmt == "e4m3":
        v = codes.view(torch.float8_e4m3fn).float()
    elif fmt == "int8":
        v = codes.view(torch.int8).float()
    else:  # int4: even entry in the low nibble
        lo = (codes & 0xF).to(torch.int16)
        hi = (codes >> 4).to(torch.int16)
        v = torch.stack(((lo ^ 8) - 8, (hi ^ 8) - 8), dim=-1).flatten(-2).float()
    flat = v.reshape(-1, group) * scale.reshape(-1, 1)
    return flat.reshape(v.shape)


REPLAY_FORMATS = (("fp16", 0), ("bf16", 0), ("int8", 16), ("int4", 16), ("e4m3", 16))
REPLAY_RULES = (("rtn", 0), ("sr", 0), ("sr", 1), ("weyl", 0), ("philox", 0))
TAU_LABELS = ("<10", "10-100", "100-1000", ">=1000")


def replay_study(w, *, steps: int, batch: int, block: int, memory: str, device, warmup: int = 128,
                 formats=REPLAY_FORMATS, rules=REPLAY_RULES) -> dict:
    """Open-loop replay (Appendix B "Open-loop replay"; Section 6.2): the rounding
    error of the state recurrence alone, on recorded per-entry decays and writes.

    One Mamba-1 layer of workload w ([batch][d_inner][N] entries, dither block 16)
    is run in FP32 for `warmup` steps (the prefill, from a zero state); the state
    then is h0, and the next `steps` steps are recorded as traces a_t = exp(dt A)
    and w_t = dt x B ([steps][n] each, resident in HBM). Step t draws dt, x and B
    from a generator seeded with splitmix64(5000, t). ssmq_replay then replays the
    traces for every (format, rule), starting from the quantized h0 (step 0), and
    the error sum (hq_t - h_t)^2 / sum h_t^2 is reported over the whole replay,
    per block of `block` steps, and per memory bin tau = 1 / (1 - exp(A dt_bar)),
    dt_bar the channel's mean step size over the recorded steps and sequences.
    Each replay launch is timed with events: trace bytes (8 per entry and step)
    over its duration.
    """
    import torch

    import paper_2609_39185_amd as ssmq
    from paper_2609_39185_amd import workloads as wl

    if w.family != "mamba1":
        raise ValueError("the replay study is defined on the Mamba-1 shapes")
    b, d, N = batch, w.nheads, w.dstate
    n = b * d * N
    params = wl.layer_params if memory == "short" else wl.layer_params_trained_memory
    A, _ = params(w.family, d, N, seed=1000, device=device)              # [d, N]
    a_tr = torch.empty((steps, n), dtype=torch.float32, device=device)
    w_tr = torch.empty((steps, n), dtype=torch.float32, device=device)
    h = torch.zeros((b, d, N), dtype=torch.float32, device=device)
    dt_sum = torch.zeros(d, dtype=torch.float64, device=device)
    t0 = time.perf_counter()
    for t in range(1 - warmup, steps + 1):
        gen = torch.Generator(device=device)
        gen.manual_seed(wl.splitmix64(5000, t + warmup))
        dt = torch.nn.functional.softplus(torch.randn((b, d), generator=gen, device=device) - 4.0)
        x = torch.randn((b, d), generator=gen, device=device)
        B = torch.randn((b, N), generator=gen, device=device)
        at = torch.exp(dt[:, :, None] * A[None])                           # [b, d, N]
        wt = (dt * x)[:, :, None] * B[:, None, :]
        if t <= 0:
            h = torch.addcmul(wt, at, h)
        else:
            a_tr[t - 1].copy_(at.reshape(-1))
            w_tr[t - 1].copy_(wt.reshape(-1))
            dt_sum += dt.double().sum(0)
    h0 = h.reshape(-1).contiguous()
    torch.cuda.synchronize()
    gen_s = time.perf_counter() - t0
    dt_bar = (dt_sum / (b * max(steps, 1))).float()
    tau = 1.0 / (1.0 - torch.exp(A * dt_bar[:, None]))                     # [d, N]
    bins = torch.bucketize(tau, torch.tensor(TAU_EDGES, device=device))
    n_bins = len(TAU_EDGES) + 1
    onehot = torch.nn.functional.one_hot(bins, n_bins).to(torch.float64)   # [d, N, bins]
    share = torch.bincount(bins.flatten(), minlength=n_bins).double() / bins.numel()
    nb = (steps + block - 1) // block
    stream = torch.cuda.current_stream(device)
    # one small untimed replay per format loads the kernels before the timed launches
    for fmt, g in formats:
        tiny = torch.empty((1, 256), dtype=torch.float64, device=device)
        ssmq.replay(h0[:256], a_tr[:1, :256].contiguous(), w_tr[:1, :256].contiguous(), tiny,
                    rule="rtn", fmt=fmt, scale_group=g, stream=stream)
    torch.cuda.synchronize()
    out, timing = {}, {}
    den_bins = None
    for fmt, g in formats:
        res = {}
        for rule, seed in rules:
            err = torch.empty((nb, n), dtype=torch.float64, device=device)
            ref = torch.empty((nb, n), dtype=torch.float64, device=device)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            ssmq.replay(h0, a_tr, w_tr, err, rule=rule, fmt=fmt, ref=ref, block_steps=block,
                        scale_group=g, dither_block=w.dither_block, seed=seed, layer=0, step=0,
                        stream=stream)
            e1.record(stream)
            e1.synchronize()
            ms = e0.elapsed_time(e1)
            name = rule if rule != "sr" else f"sr_seed{seed}"
            timing[f"{fmt}:{name}"] = ms
            num = torch.einsum("kdn,dnj->kj", err.view(nb, b, d, N).sum(1), onehot)   # [blocks, bins]
            den = torch.einsum("kdn,dnj->kj", ref.view(nb, b, d, N).sum(1), onehot)
            den_bins = den
            res[name] = {
                "error": float(num.sum() / den.sum()),
                "error_per_block": [float(v) for v in num.sum(1) / den.sum(1)],
                "error_by_tau_bin": {TAU_LABELS[j]: float(num[:, j].sum() / den[:, j].sum())
                                     for j in range(n_bins) if float(den[:, j].sum()) > 0},
            }
            print(f"replay: {fmt} {name} {ms:.2f} ms", file=sys.stderr, flush=True)
        sr = res["sr_seed0"]
        for name, r in res.items():
            r["over_sr_seed0"] = r["error"] / sr["error"]
            r["over_sr_seed0_by_tau_bin"] = {k: v / sr["error_by_tau_bin"][k]
                                             for k, v in r["error_by_tau_bin"].items()}
        out[fmt + (f"_block{g}" if g else "")] = res
    trace_bytes = 8 * n * steps
    best = min(timing.values())
    return {
        "study": "open_loop_replay",
        "metric": "relative state error sum((hq-h)^2)/sum(h^2) of the replayed recurrence",
        "workload": w.name, "batch": b, "d_inner": d, "dstate": N, "entries": n, "steps": steps,
        "warmup_steps": warmup, "block": block, "dither_block": w.dither_block, "memory": memory,
        "data": "synthetic traces", "tau_bin_share": dict(zip(TAU_LABELS, [float(v) for v in share])),
        "results": out,
        "replay_ms": timing,
        "replay_trace_GBps_best": trace_bytes / (best * 1e-3) / 1e9,
        "replay_entry_steps_per_s_best": n * steps / (best * 1e-3),
        "trace_generation_s": gen_s,
    }


def state_error_study(w, *, steps: int, layers: int, block: int, device, fmt: str = "fp16",
                      group: int = 16, memory: str = "short", cc: int = 0, rules=SE_RULES,
                      on_step=None, init=None) -> dict:
    """Quantized states against an unrounded FP32 twin, decoded in lockstep on the
    same teacher-forced inputs (Appendix B, "Open-loop replay" and "Decode regime").

    Every (layer, step) runs the fused update once per rule and once in the FP32
    format (the twin). Both start from the same stored state. Per block of `block`
    steps and per layer the error is sum((h_hat - h)^2) / sum(h^2) over entries,
    batch and steps; the model-level figure is the mean over layers. Errors are also
    split into memory bins by tau = 1 / (1 - exp(A * E[dt])).

    fmt: fp16, bf16, e4m3, int8 or int4 (the scaled ones with `group` entries per
    scale). memory: "short" (the throughput bench's decay rates) or "trained" (a
    trained model's spread, workloads.layer_params_trained_memory). cc > 0 adds,
    for RTN, SR (seed 0) and Weyl, a periodically checkpointed run: an fp32 state
    rounded onto the format's grid at every cc-th write only (Section 6.5 "Periodic
    checkpointing").

    Inputs: A, D per layer; x, dt, B, C for all layers of step t from one generator
    seeded with splitmix64(4000, t). on_step(t, x, dt, B, C) is called with each
    step's inputs, and init = {"A", "D", "codes0"} replaces the generated layer
    parameters and initial codes (both for cross-checks on small sizes).
    """
    import numpy as np
    import torch

    import paper_2609_39185_amd as ssmq
    from paper_2609_39185_amd import workloads as wl

    if w.family != "mamba1":
        raise ValueError("the state-error study is defined on the Mamba-1 shapes")
    b, d, N = w.batch, w.nheads, w.dstate
    L = layers
    scaled = fmt in ("e4m3", "int8", "int4")
    g_ = group if scaled else 0
    n_blocks = (steps + block - 1) // block
    code_dt = wl.CODE_TORCH_DTYPE[fmt]
    per = 2 if fmt == "int4" else 1
    params = wl.layer_params if memory == "short" else wl.layer_params_trained_memory
    A, D = [], []
    for ell in range(L):
        if init is not None:
            a, dd = init["A"][ell].to(device), init["D"][ell].to(device)
        else:
            a, dd = params(w.family, d, N, seed=1000 + ell, device=device)
        A.append(a.contiguous())
        D.append(dd.contiguous())
    runs = list(rules) + ([(r, sd, cc) for r, sd in (("rtn", 0), ("sr", 0), ("weyl", 0))]
                          if cc > 0 else [])
    codes, scales = {}, {}
    for r in runs:
        if len(r) == 3:
            codes[r] = torch.empty((L, b, d, 1, N), dtype=torch.float32, device=device)
        else:
            codes[r] = torch.empty((L, b, d, 1, N // per), dtype=code_dt, device=device)
            scales[r] = (torch.empty((L, b * d * N // g_), dtype=torch.float32, device=device)
                         if scaled else None)
    twin = torch.empty((L, b, d, 1, N), dtype=torch.float32, device=device)
    for ell in range(L):
        if init is not None:
            c0, s0 = init["codes0"][ell].to(device), None
            if scaled:
                s0 = init["scale0"][ell].to(device)
        else:
            c0, s0 = wl.initial_state(fmt, b, d, 1, N, seed=3000 + ell, group=g_, device=device)
        h0 = decode_state(fmt, c0, s0, g_ or 1)
        for r in runs:
            if len(r) == 3:
                codes[r][ell].copy_(h0)
            else:
                codes[r][ell].copy_(c0)
                if scaled:
                    scales[r][ell].copy_(s0)
        twin[ell].copy_(h0)
    twin_codes = twin.view(torch.int32)
    y = torch.empty((b, d, 1), dtype=torch.float32, device=device)

    # memory bins of each (layer, channel, n)
    dt_mean = mean_step_size()
    abar = torch.exp(torch.stack(A) * dt_mean)                       # [L, d, N]
    tau = 1.0 / (1.0 - abar)
    bins = torch.bucketize(tau, torch.tensor(TAU_EDGES, device=device))  # [L, d, N] in 0..3
    n_bins = len(TAU_EDGES) + 1
    onehot = torch.nn.functional.one_hot(bins, n_bins).to(torch.float64)  # [L, d, N, n_bins]

    num = {r: torch.zeros((n_blocks, L, n_bins), dtype=torch.float64, device=device) for r in runs}
    den = torch.zeros((n_blocks, L, n_bins), dtype=torch.float64, device=device)
    # per-entry sums over batch and the steps of the current block
    acc = {r: torch.zeros((L, d, N), dtype=torch.float64, device=device) for r in runs}
    acc_h = torch.zeros((L, d, N), dtype=torch.float64, device=device)
    stream = torch.cuda.current_stream(device)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for t in range(1, steps + 1):
        gen = torch.Generator(device=device)
        gen.manual_seed(wl.splitmix64(4000, t))
        x = torch.randn((L, b, d, 1), generator=gen, device=device)
        dt = torch.nn.functional.softplus(torch.randn((L, b, d), generator=gen, device=device) - 4.0)
        B = torch.randn((L, b, 1, N), generator=gen, device=device)
        C = torch.randn((L, b, 1, N), generator=gen, device=device)
        if on_step is not None:
            on_step(t, x, dt, B, C)
        for ell in range(L):
            args = (x[ell], dt[ell], A[ell], B[ell], C[ell], D[ell], y)
            ssmq.state_update(twin_codes[ell], None, *args, rule="rtn", fmt="fp32",
                              dither_block=w.dither_block, layer=ell, step=t, stream=stream)
            for r in runs:
                if len(r) == 3:
                    if t % r[2] == 0:
                        ssmq.state_update(codes[r][ell], None, *args, rule=r[0], fmt=fmt,
                                          seed=r[1], scale_group=g_, dither_block=w.dither_block,
                                          layer=ell, step=t, fp32_state=True, stream=stream)
                    else:
                        ssmq.state_update(codes[r][ell].view(torch.int32), None, *args,
                                          rule="rtn", fmt="fp32", dither_block=w.dither_block,
                                          layer=ell, step=t, stream=stream)
                else:
                    ssmq.state_update(codes[r][ell], None if scales[r] is None else scales[r][ell],
                                      *args, rule=r[0], fmt=fmt, seed=r[1], scale_group=g_,
                                      dither_block=w.dither_block, layer=ell, step=t,
                                      stream=stream)
        acc_h += twin.square().sum(dim=(1, 3))
        for r in runs:
            if len(r) == 3:
                e = codes[r] - twin
            else:
                e = decode_state(fmt, codes[r], scales[r], g_ or 1).sub_(twin)
            acc[r] += e.square_().sum(dim=(1, 3))
        if t % block == 0 or t == steps:
            k = (t - 1) // block
            den[k] = torch.einsum("ldn,ldnk->lk", acc_h, onehot)
            acc_h.zero_()
            for r in runs:
                num[r][k] = torch.einsum("ldn,ldnk->lk", acc[r], onehot)
                acc[r].zero_()
            print(f"state-error study: {t} of {steps} steps, "
                  f"{time.perf_counter() - t_start:.1f} s", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start

    def name(r):
        base = r[0] if r[0] != "sr" else f"sr_seed{r[1]}"
        return base if len(r) == 2 else f"{base}_cc{r[2]}"

    out_rules, out_bins = {}, {}
    for r in runs:
        tot = num[r].sum(-1) / den.sum(-1)                                   # [blocks, L]
        out_rules[name(r)] = [float(v) for v in tot.mean(-1)]
        per_bin = num[r] / den                                               # [blocks, L, bins]
        out_bins[name(r)] = {}
        for j in range(n_bins):
            if float(den[..., j].sum()) > 0:
                lab = ("<10", "10-100", "100-1000", ">=1000")[j]
                out_bins[name(r)][lab] = [float(v) for v in per_bin[..., j].nanmean(-1)]
    ref = name(("sr", 0))
    share = [float(v) for v in torch.bincount(bins.flatten(), minlength=n_bins).double() / bins.numel()]
    return {
        "study": "state_error",
        "metric": "relative state error sum((h_hat-h)^2)/sum(h^2) per block, mean over layers",
        "workload": w.name, "format": fmt, "scale_group": g_ or None, "memory": memory,
        "checkpoint_every": cc or None, "batch": b, "d_inner": d, "dstate": N, "layers": L,
        "steps": steps, "block": block, "dither_block": w.dither_block, "data": "synthetic",
        "mean_dt": dt_mean, "tau_bin_share": dict(zip(("<10", "10-100", "100-1000", ">=1000"), share)),
        "error": out_rules,
        "error_over_sr_seed0": {k: [a / c for a, c in zip(v, out_rules[ref])]
                                for k, v in out_rules.items()},
        "error_by_tau_bin": out_bins,
        "wall_s": elapsed,
        "ms_per_step": 1e3 * elapsed / steps,
        "launches_per_step": L * (1 + len(runs)),
    }


SWEEP_WORKLOADS = ("m1_small", "m2_ssd_b8", "m2_b64_fp8", "m1_long")
TARGET_FRACTION = 0.80  # of peak HBM bandwidth, on the largest workload, per stored format


def targets_summary(results: dict) -> dict:
    """Each format's Weyl variant against the 80 % target, with what bounds it:
    bf16 (4 B per entry) is bound by HBM; E4M3, INT8 and INT4 (2, 2 and 1 B per
    entry) need two to four times the entries per second for the same bytes and
    are bound by vector issue (the dithered conversion, threshold and sign per
    entry)."""
    out = {}
    for key, r in results.items():
        stored, rule = key.split(":", 1)
        if rule != "weyl":
            continue
        fmt = stored.split("/")[0]
        frac = r["pct_of_peak"] / 100.0
        out[key] = {"pct_of_peak": r["pct_of_peak"], "target_pct": 100.0 * TARGET_FRACTION,
                    "meets_target": frac >= TARGET_FRACTION,
                    "bound": "hbm" if fmt in ("bf16", "fp16") else "vector issue"}
    return out


def graph_launch_us(w, fmt, rule, group, L, steps, warmup, device, t0=1):
    """Average device time per ssmq_state_update launch on workload w: all layers
    resident, `steps` steps (each with its own step t) captured into one HIP graph
    and replayed between two events on the launch stream. Returns (us per launch,
    ms per step)."""
    import torch

    import paper_2609_39185_amd as ssmq
    from paper_2609_39185_amd import workloads as wl

    b, H, P, N, G = w.batch, w.nheads, w.headdim, w.dstate, w.ngroups
    layers = []
    for ell in range(L):
        A, D = wl.layer_params(w.family, H, N, seed=1000 + ell, device=device)
        x, dt, B, C = wl.step_inputs(b, H, P, N, G, seed=2000 + ell, device=device)
        st, sc = wl.initial_state(fmt, b, H, P, N, seed=3000 + ell, group=group, device=device)
        layers.append((st, sc, x, dt, A, B, C, D, torch.empty((b, H, P), device=device)))
    stream = torch.cuda.current_stream(device)

    def step(t, on):
        for ell, (st, sc, x, dt, A, B, C, D, y) in enumerate(layers):
            ssmq.state_update(st, sc, x, dt, A, B, C, D, y, rule=rule, fmt=fmt,
                              dither_block=w.dither_block, scale_group=group, layer=ell, step=t,
                              stream=on)

    for k in range(warmup):
        step(t0 + k, stream)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        cap = torch.cuda.current_stream(device)
        for k in range(steps):
            step(t0 + warmup + k, cap)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    graph.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    del graph, layers
    torch.cuda.empty_cache()
    return 1e3 * ms / (steps * L), ms / steps


def oracle_layer_rate(w, fmt, rule, group, target_s, threads):
    """The C oracle on a slice of one layer of workload w (Mamba-2: the heads of one
    B/C group of one sequence; Mamba-1: one sequence's channels), repeated for about
    target_s seconds on `threads` threads; returns (entries per second, sample text)."""
    from concurrent.futures import ThreadPoolExecutor

    import oracle
    from paper_2609_39185_amd import workloads as wl

    H, P, N, G = w.nheads, w.headdim, w.dstate, w.ngroups
    nh = H // G if w.family == "mamba2" else H
    A, D = wl.layer_params(w.family, H, N, seed=1000)
    x, dt, B, C = wl.step_inputs(1, H, P, N, G, seed=2000)
    codes, scale = wl.initial_state(fmt, 1, H, P, N, seed=3000, group=group)
    c = wl.to_numpy_codes(fmt, codes)[:, :nh]
    per_head = P * N // (group or P * N) if scale is not None else 0
    sc = None if scale is None else scale.numpy()[:nh * per_head]
    args = (x.numpy()[:, :nh], dt.numpy()[:, :nh], A.numpy()[:nh], B.numpy()[:, :1],
            C.numpy()[:, :1], D.numpy()[:nh])

    def run():
        oracle.state_update(fmt, rule, c, sc, *args, block=w.dither_block, group=group, step=1)

    run()
    def worker(deadline):
        n = 0
        while time.perf_counter() < deadline:
            run()
            n += 1
        return n

    t0 = time.perf_counter()
    with ThreadPoolExecutor(max_workers=threads) as pool:
        calls = sum(pool.map(worker, [t0 + target_s] * threads))
    wall = time.perf_counter() - t0
    sample_entries = nh * P * N
    return calls * sample_entries / wall, f"{calls} calls of {sample_entries} entries, {wall:.1f} s"


def config_sweep(device, *, steps: int, warmup: int, cpu_seconds: float) -> dict:
    """The measurement plan's other workloads, each in its own storage format and
    under RTN, hash SR and Weyl: device time per launch (HIP graph, all layers
    resident), the oracle's time for the same layer-step (extrapolated from a slice,
    one thread and every usable core), and for the long-horizon Mamba-1 shape a short
    state-error run against the FP32 twin (per rule, per block of steps)."""
    from paper_2609_39185_amd import workloads as wl

    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    cores = max(1, min(cores, int(os.environ.get("OMP_NUM_THREADS") or 16), 16))
    out = {}
    for name in SWEEP_WORKLOADS:
        w = wl.WORKLOADS[name]
        fmt = w.formats[0]
        group = wl.scale_group_of(w, fmt)
        L = w.layers
        sbytes = state_bytes_per_launch(w, fmt, group)
        entry = {"workload": w.name, "notes": w.notes, "format": fmt, "layers": L,
                 "dither_block": w.dither_block, "entries_per_layer": w.entries_per_layer,
                 "state_bytes_per_launch": sbytes, "launch": "hip_graph", "rules": {}}
        for rule in ("rtn", "sr", "weyl"):
            print(f"bench: {name} {fmt} {rule}: {steps} steps x {L} layers (HIP graph)",
                  file=sys.stderr, flush=True)
            us, ms_step = graph_launch_us(w, fmt, rule, group, L, steps, warmup, device)
            r = {"us_per_launch": us, "ms_per_step": ms_step, "steps_per_s": 1e3 / ms_step,
                 "state_GBps": sbytes / (us * 1e3), "pct_of_peak": 100.0 * sbytes / (us * 1e3) / PEAK_HBM_GBPS}
            if cpu_seconds > 0:
                e1, s1 = oracle_layer_rate(w, fmt, rule, group, cpu_seconds / 2, 1)
                ea, sa = oracle_layer_rate(w, fmt, rule, group, cpu_seconds / 2, cores)
                bpe = sbytes / w.entries_per_layer
                r["oracle"] = {"us_per_layer_step_1_thread": 1e6 * w.entries_per_layer / e1,
                               "us_per_layer_step_all_cores": 1e6 * w.entries_per_layer / ea,
                               "GBps_1_thread": e1 * bpe / 1e9, "GBps_all_cores": ea * bpe / 1e9,
                               "cores": cores, "sample_1_thread": s1, "sample_all_cores": sa}
            entry["rules"][rule] = r
        out[name] = entry
    w = wl.WORKLOADS["m1_long"]
    print("bench: m1_long state error against the FP32 twin, 512 steps x 64 layers",
          file=sys.stderr, flush=True)
    se = state_error_study(w, steps=512, layers=w.layers, block=128, device=device)
    out["m1_long"]["state_error"] = {k: se[k] for k in ("metric", "steps", "block", "layers",
                                                        "error", "error_over_sr_seed0",
                                                        "tau_bin_share", "wall_s")}
    return out


def kernel_sources_digest() -> str:
    """sha256 over the sources that decide which kernel runs and what it does."""
    import hashlib

    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_39185_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def traffic_path(workload: str) -> str:
    return os.path.join(PROFILE_DIR, f"k_update_slab.{workload}.traffic.json")


def load_traffic(workload: str):
    """Measured HBM bytes per launch for each variant, if the counters were taken
    on the kernels as they are now (else None)."""
    try:
        with open(traffic_path(workload)) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_sources_sha256") != kernel_sources_digest():
        return None
    return rec.get("variants")


# rocprofv3 names the update kernels k_update_slab<F, R, NT, CPT> with these codes
_FMT_CODE = {"fp16": 0, "bf16": 1, "e4m3": 2, "fp32": 3, "int8": 4, "int4": 5}
_RULE_CODE = {"rtn": 0, "sr": 1, "weyl": 2, "philox": 3}


def _csv_rows(d: str, suffix: str):
    import csv
    import glob

    hits = sorted(glob.glob(os.path.join(d, "**", "*" + suffix), recursive=True))
    if not hits:
        raise SystemExit(f"no *{suffix} under {d}")
    with open(hits[0], newline="") as f:
        return list(csv.DictReader(f))


def _grid(row) -> int:
    """Threads of a dispatch: the counter CSV has Grid_Size, the kernel trace CSV
    Grid_Size_X, _Y and _Z."""
    if row.get("Grid_Size") not in (None, ""):
        return int(row["Grid_Size"])
    return int(row["Grid_Size_X"]) * int(row["Grid_Size_Y"]) * int(row["Grid_Size_Z"])


def _variant_of(kernel_name: str):
    import re

    m = re.search(r"k_update_(?:slab|rows)<(\d+), (\d+)", kernel_name)
    if not m:
        return None
    f = {v: k for k, v in _FMT_CODE.items()}[int(m.group(1))]
    r = {v: k for k, v in _RULE_CODE.items()}[int(m.group(2))]
    return f"{f}:{r}"


def _short_kernel(name: str) -> str:
    return name.replace("void ", "").replace("(ssmq::UpdateArgs)", "").replace("ssmq::", "")


def summarize_profiles(workload: str, trace_dir: str, fetch_dir: str, write_dir: str) -> int:
    """Write profiles/k_update_slab.<workload>.{kernel_trace.md,traffic.md,traffic.json}.

    FETCH_SIZE and WRITE_SIZE (KiB per dispatch) are scaled by what they read for
    the calibration kernel (torch.neg over CAL_BYTES in, CAL_BYTES out).
    """
    import statistics
    from collections import defaultdict

    from paper_2609_39185_amd import workloads as wl

    w = wl.WORKLOADS[workload]
    os.makedirs(PROFILE_DIR, exist_ok=True)
    trace = _csv_rows(trace_dir, "kernel_trace.csv")
    dur = defaultdict(list)
    for r in trace:
        dur[(r["Kernel_Name"], _grid(r))].append(
            int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))

    def counter(d, name):
        vals = defaultdict(list)
        for r in _csv_rows(d, "counter_collection.csv"):
            if r["Counter_Name"] == name:
                vals[(r["Kernel_Name"], _grid(r))].append(float(r["Counter_Value"]))
        return vals

    fetch, write = counter(fetch_dir, "FETCH_SIZE"), counter(write_dir, "WRITE_SIZE")

    def calib(vals):
        c = [statistics.mean(v) for (k, g), v in vals.items() if "neg_kernel" in k]
        if not c:
            raise SystemExit("no calibration kernel dispatch in the counter output")
        return CAL_BYTES / (max(c) * 1024.0)

    f_fetch, f_write = calib(fetch), calib(write)
    n_entries = w.entries_per_layer
    variants = {}
    for (k, g), v in fetch.items():
        key = _variant_of(k)
        if key is None:
            continue
        fmt = key.split(":")[0]
        algo = state_bytes_per_launch(w, fmt)
        fk = statistics.mean(v)
        wk = statistics.mean(write.get((k, g), [float("nan")]))
        traffic = fk * 1024.0 * f_fetch + wk * 1024.0 * f_write
        variants[key] = {
            "kernel": _short_kernel(k),
            "dispatches": len(v), "fetch_KiB": fk, "write_KiB": wk,
            "traffic_bytes": traffic, "algorithmic_bytes": algo,
            "traffic_over_algorithmic": traffic / algo,
            "trace_avg_us": statistics.mean(dur[(k, g)]) / 1e3 if (k, g) in dur else None,
        }
    rec = {
        "workload": workload,
        "kernel_sources_sha256": kernel_sources_digest(),
        "calibration": {"kernel": "torch.neg fp32", "bytes_in": CAL_BYTES, "bytes_out": CAL_BYTES,
                        "fetch_scale": f_fetch, "write_scale": f_write},
        "commands": PROFILE_COMMANDS,
        "variants": dict(sorted(variants.items())),
    }
    with open(traffic_path(workload), "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")

    lines = [f"# k_update_slab on {workload}: HBM traffic per launch", "",
             "Commands (repository root as $R, an output directory as $OUT, run from /tmp with TMPDIR=/tmp):", ""]
    lines += [f"    {PROFILE_COMMANDS[k]}" for k in ("trace", "fetch", "write", "summary")]
    lines += ["", f"Calibration: torch.neg over {CAL_BYTES} B in and out reads "
                  f"FETCH_SIZE x {f_fetch:.4f}, WRITE_SIZE x {f_write:.4f} of the true bytes.", "",
              "| variant | kernel | FETCH KiB | WRITE KiB | traffic B | algorithmic B | ratio |",
              "|---|---|---|---|---|---|---|"]
    for key, r in rec["variants"].items():
        lines.append(f"| {key} | `{r['kernel']}` | {r['fetch_KiB']:.0f} | {r['write_KiB']:.0f} | "
                     f"{r['traffic_bytes']:.4g} | {r['algorithmic_bytes']} | "
                     f"{r['traffic_over_algorithmic']:.4f} |")
    with open(os.path.join(PROFILE_DIR, f"k_update_slab.{workload}.traffic.md"), "w") as f:
        f.write("\n".join(lines) + "\n")

    # Per (kernel, grid size): the default run also launches the same kernel
    # instances on the smaller workloads of its configs block, whose launches
    # must not be averaged with the hybrid stack's.
    by_grid = defaultdict(list)
    for r in trace:
        by_grid[(r["Kernel_Name"], _grid(r))].append(
            int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    lines = [f"# Kernel trace of the default bench run on {workload}", "",
             "Command (repository root as $R, an output directory as $OUT, run from /tmp with TMPDIR=/tmp):", "",
             f"    {PROFILE_COMMANDS['trace']}", "",
             "Launches grouped by kernel and grid size (threads); the largest grids are the "
             f"{workload} layers, the smaller ones the configs block's workloads. The 16 kernels "
             "with the most total time:", "",
             "| kernel | grid | calls | avg us | min us | max us | total ms |",
             "|---|---|---|---|---|---|---|"]
    for (name, grid), v in sorted(by_grid.items(), key=lambda kv: -sum(kv[1]))[:16]:
        if len(name) > 80:
            name = name[:77] + "..."
        lines.append(f"| `{name}` | {grid} | {len(v)} | {statistics.mean(v) / 1e3:.1f} | "
                     f"{min(v) / 1e3:.1f} | {max(v) / 1e3:.1f} | {sum(v) / 1e6:.2f} |")
    with open(os.path.join(PROFILE_DIR, f"k_update_slab.{workload}.kernel_trace.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print(json.dumps({k: round(v["traffic_over_algorithmic"], 4) for k, v in variants.items()}))
    return 0


def summarize_replay_trace(trace_dir: str, name: str) -> int:
    """Write profiles/<name>.kernel_trace.md from a kernel trace of the replay study
    (PROFILE_COMMANDS["replay_trace"]): per k_replay instance, calls and durations,
    and the trace rate 8 B x entries x steps / average duration."""
    import re

    stats = _csv_rows(trace_dir, "kernel_stats.csv")
    m = re.search(r"--steps (\d+)", PROFILE_COMMANDS["replay_trace"])
    steps = int(m.group(1))
    from paper_2609_39185_amd import workloads as wl
    w = wl.WORKLOADS["m1_long"]
    n = w.batch * w.nheads * w.dstate
    fmts = {v: k for k, v in _FMT_CODE.items()}
    rules = {v: k for k, v in _RULE_CODE.items()}
    lines = [f"# Kernel trace of the replay study ({n} entries x {steps} steps per launch)", "",
             "Command (repository root as $R, an output directory as $OUT, run from /tmp with TMPDIR=/tmp):", "",
             f"    {PROFILE_COMMANDS['replay_trace']}",
             f"    {PROFILE_COMMANDS['replay_trace_summary']}", "",
             "The longest call of each instance is a full-size launch: the RTN instances also run "
             "one untimed 256-entry, one-step launch, the hash-SR instances run twice at full size "
             "(seeds 0 and 1). Trace rate = 8 B x entries x steps / the full-size duration.", "",
             "| kernel | format:rule | calls | full-size launch us | trace GB/s |",
             "|---|---|---|---|---|"]
    for r in sorted(stats, key=lambda r: r["Name"]):
        km = re.search(r"k_replay<(\d+), (\d+)>", r["Name"])
        if not km:
            continue
        key = f"{fmts[int(km.group(1))]}:{rules[int(km.group(2))]}"
        mx = float(r["MaxNs"]) / 1e3
        lines.append(f"| `{_short_kernel(r['Name'])}` | {key} | {r['Calls']} | {mx:.1f} | "
                     f"{8 * n * steps / (mx * 1e3):.0f} |")
    os.makedirs(PROFILE_DIR, exist_ok=True)
    with open(os.path.join(PROFILE_DIR, f"{name}.kernel_trace.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))
    return 0


def summarize_entry_points_trace(trace_dir: str) -> int:
    """Write profiles/entry_points.hybrid_m2_stack.kernel_trace.md from a kernel
    trace of `bench.py --entry-points` (PROFILE_COMMANDS["entry_trace"]): per
    requantize and threshold-fill kernel instance, calls and durations."""
    import re

    stats = _csv_rows(trace_dir, "kernel_stats.csv")
    lines = ["# Kernel trace of the requantize and threshold-fill calls (268,435,456 entries per launch)", "",
             "Command (repository root as $R, an output directory as $OUT, run from /tmp with TMPDIR=/tmp):", "",
             f"    {PROFILE_COMMANDS['entry_trace']}",
             f"    {PROFILE_COMMANDS['entry_trace_summary']}", "",
             "Template arguments: format code (0 fp16, 1 bf16, 2 E4M3, 4 INT8, 5 INT4), rule code "
             "(0 RTN, 1 hash SR, 2 Weyl, 3 Philox), and for the per-group kernel the chunks per thread.", "",
             "| kernel | calls | avg us | min us | max us |", "|---|---|---|---|---|"]
    for r in sorted(stats, key=lambda r: r["Name"]):
        if not re.search(r"k_requant|k_dither_fill", r["Name"]):
            continue
        lines.append(f"| `{_short_kernel(r['Name'])}` "
                     f"| {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | {float(r['MinNs']) / 1e3:.1f} | "
                     f"{float(r['MaxNs']) / 1e3:.1f} |")
    os.makedirs(PROFILE_DIR, exist_ok=True)
    with open(os.path.join(PROFILE_DIR, "entry_points.hybrid_m2_stack.kernel_trace.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))
    return 0


def summarize_valu(workload: str, pmc_dir: str) -> int:
    """Write profiles/k_update_slab.<workload>.valu.md: per variant, VALU
    instructions per wave and per entry (lane operations), and the VALU busy
    fraction SQ_ACTIVE_INST_VALU * 4 / SIMDs / (GRBM_GUI_ACTIVE / XCDs)."""
    import statistics
    from collections import defaultdict

    from paper_2609_39185_amd import workloads as wl

    w = wl.WORKLOADS[workload]
    agent = [r for r in _csv_rows(pmc_dir, "agent_info.csv") if r.get("Agent_Type") == "GPU"][0]
    simds, xcc = int(agent["Simd_Count"]), int(agent["Num_Xcc"])
    vals = defaultdict(lambda: defaultdict(list))
    for r in _csv_rows(pmc_dir, "counter_collection.csv"):
        if _variant_of(r["Kernel_Name"]) is not None:
            vals[r["Kernel_Name"]][r["Counter_Name"]].append(float(r["Counter_Value"]))
    rows = []
    for k, c in vals.items():
        m = {n: statistics.mean(v) for n, v in c.items()}
        busy = m["SQ_ACTIVE_INST_VALU"] * 4 / simds / (m["GRBM_GUI_ACTIVE"] / xcc)
        rows.append((_variant_of(k), _short_kernel(k), m["SQ_INSTS_VALU"] / m["SQ_WAVES"],
                     m["SQ_INSTS_VALU"] * 64 / w.entries_per_layer, busy, len(c["SQ_WAVES"])))
    lines = [f"# k_update_slab on {workload}: vector-instruction budget per launch", "",
             "Command (repository root as $R, an output directory as $OUT, run from /tmp with TMPDIR=/tmp):", "",
             f"    {PROFILE_COMMANDS['valu']}", f"    {PROFILE_COMMANDS['valu_summary']}", "",
             f"Lane operations per entry = SQ_INSTS_VALU x 64 / {w.entries_per_layer} entries; "
             f"VALU busy = SQ_ACTIVE_INST_VALU x 4 / {simds} SIMDs / (GRBM_GUI_ACTIVE / {xcc} XCDs).",
             "", "| variant | kernel | VALU instr per wave | lane ops per entry | VALU busy | dispatches |",
             "|---|---|---|---|---|---|"]
    for v, k, per_wave, per_entry, busy, n in sorted(rows):
        lines.append(f"| {v} | `{k}` | {per_wave:.0f} | {per_entry:.1f} | {100 * busy:.0f} % | {n} |")
    os.makedirs(PROFILE_DIR, exist_ok=True)
    with open(os.path.join(PROFILE_DIR, f"k_update_slab.{workload}.valu.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))
    return 0


MIX_COUNTERS_A = ("SQ_INSTS_VALU_FMA_F32", "SQ_INSTS_VALU_MUL_F32", "SQ_INSTS_VALU_ADD_F32",
                  "SQ_INSTS_VALU_CVT", "SQ_INSTS_VALU_INT32", "SQ_INSTS_VALU_INT64")
MIX_COUNTERS_B = ("SQ_INSTS_VALU_FMA_F64", "SQ_INSTS_VALU_ADD_F64", "SQ_INSTS_VALU_MUL_F64",
                  "SQ_INSTS_VALU_TRANS_F32", "SQ_INSTS_SALU", "SQ_INSTS_LDS", "SQ_INSTS_BRANCH")


def summarize_mix(workload: str, dir_a: str, dir_b: str) -> int:
    """Write profiles/k_update_slab.<workload>.valu_mix.md: per variant, the VALU
    instructions per wave by kind (fp32 FMA, multiply and add, conversions, 32- and
    64-bit integer, fp64, transcendental), the rest of the VALU count (bitwise,
    min/max/med3, moves, selects, compares, DPP and byte permutes), and the scalar,
    LDS and branch instructions per wave. Two --pmc passes, each with SQ_WAVES."""
    import statistics
    from collections import defaultdict

    vals = defaultdict(lambda: defaultdict(list))
    for d in (dir_a, dir_b):
        for r in _csv_rows(d, "counter_collection.csv"):
            if _variant_of(r["Kernel_Name"]) is not None:
                key = (r["Kernel_Name"], d)
                vals[key][r["Counter_Name"]].append(float(r["Counter_Value"]))
    per_wave = defaultdict(dict)
    for (k, d), c in vals.items():
        waves = statistics.mean(c["SQ_WAVES"])
        for n, v in c.items():
            if n != "SQ_WAVES":
                per_wave[k][n] = statistics.mean(v) / waves
    fp64 = ("SQ_INSTS_VALU_FMA_F64", "SQ_INSTS_VALU_ADD_F64", "SQ_INSTS_VALU_MUL_F64")
    head = ["FMA f32", "MUL f32", "ADD f32", "CVT", "INT32", "INT64", "f64", "TRANS f32", "rest",
            "VALU", "SALU", "LDS", "branch"]
    lines = [f"# k_update_slab on {workload}: VALU instructions per wave by kind", "",
             "Commands (repository root as $R, an output directory as $OUT, run from /tmp with TMPDIR=/tmp):",
             "", f"    {PROFILE_COMMANDS['mix_a']}", f"    {PROFILE_COMMANDS['mix_b']}",
             f"    {PROFILE_COMMANDS['mix_summary']}", "",
             "Per wave (counter / SQ_WAVES of its pass). \"rest\" is SQ_INSTS_VALU minus the kinds "
             "counted: bitwise operations, min / max / med3, moves, selects, compares, DPP moves and "
             "byte permutes.", "",
             "| variant | kernel | " + " | ".join(head) + " |", "|---|---|" + "---|" * len(head)]
    rows = []
    for k, c in per_wave.items():
        if "SQ_INSTS_VALU" not in c or "SQ_INSTS_SALU" not in c:
            continue
        kinds = [c[n] for n in MIX_COUNTERS_A] + [sum(c[n] for n in fp64), c["SQ_INSTS_VALU_TRANS_F32"]]
        rest = c["SQ_INSTS_VALU"] - sum(kinds)
        rows.append((_variant_of(k), _short_kernel(k),
                     kinds + [rest, c["SQ_INSTS_VALU"], c["SQ_INSTS_SALU"], c["SQ_INSTS_LDS"],
                              c["SQ_INSTS_BRANCH"]]))
    for v, k, nums in sorted(rows):
        lines.append(f"| {v} | `{k}` | " + " | ".join(f"{x:.1f}" for x in nums) + " |")
    os.makedirs(PROFILE_DIR, exist_ok=True)
    with open(os.path.join(PROFILE_DIR, f"k_update_slab.{workload}.valu_mix.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))
    return 0


PROFILE_COMMANDS = {
    "trace": "rocprofv3 --kernel-trace --stats --output-format csv -d $OUT/prof_trace "
             "-o run -- python3 $R/bench.py",
    "fetch": "timeout -s KILL 120 rocprofv3 --pmc FETCH_SIZE --output-format csv "
             "-d $OUT/prof_fetch -o run -- python3 $R/bench.py --steps 2 --warmup 1 "
             "--cpu-seconds 0 --no-configs",
    "write": "timeout -s KILL 120 rocprofv3 --pmc WRITE_SIZE --output-format csv "
             "-d $OUT/prof_write -o run -- python3 $R/bench.py --steps 2 --warmup 1 "
             "--cpu-seconds 0 --no-configs",
    "summary": "python3 $R/bench.py --summarize-profiles $OUT/prof_trace "
               "$OUT/prof_fetch $OUT/prof_write",
    "valu": "timeout -s KILL 120 rocprofv3 --pmc SQ_WAVES SQ_ACTIVE_INST_VALU SQ_WAVE_CYCLES "
            "SQ_BUSY_CYCLES SQ_INSTS_VALU GRBM_GUI_ACTIVE --output-format csv "
            "-d $OUT/pmc_busy -o run -- python3 $R/bench.py --steps 2 --warmup 0 "
            "--layers 4 --cpu-seconds 0 --no-ceiling --no-configs",
    "valu_summary": "python3 $R/bench.py --summarize-valu $OUT/pmc_busy",
    "mix_a": "timeout -s KILL 120 rocprofv3 --pmc SQ_WAVES SQ_INSTS_VALU "
             + " ".join(MIX_COUNTERS_A) + " --output-format csv -d $OUT/pmc_mix_a -o run -- "
             "python3 $R/bench.py --steps 2 --warmup 0 --layers 4 --cpu-seconds 0 --no-ceiling "
             "--no-configs",
    "mix_b": "timeout -s KILL 120 rocprofv3 --pmc SQ_WAVES " + " ".join(MIX_COUNTERS_B)
             + " --output-format csv -d $OUT/pmc_mix_b -o run -- python3 $R/bench.py --steps 2 "
             "--warmup 0 --layers 4 --cpu-seconds 0 --no-ceiling --no-configs",
    "mix_summary": "python3 $R/bench.py --summarize-mix $OUT/pmc_mix_a $OUT/pmc_mix_b",
    "replay_trace": "rocprofv3 --kernel-trace --stats --output-format csv -d $OUT/prof_replay "
                    "-o run -- python3 $R/bench.py --replay --steps 4096",
    "entry_trace": "rocprofv3 --kernel-trace --stats --output-format csv -d $OUT/prof_entry "
                   "-o run -- python3 $R/bench.py --entry-points",
    "entry_trace_summary": "python3 $R/bench.py --summarize-entry-trace $OUT/prof_entry",
    "replay_trace_summary": "python3 $R/bench.py --summarize-trace $OUT/prof_replay "
                            "k_replay.m1_long",
}


def entry_point_rates(w, steps, warmup, device):
    """Rates of the boundary's other two calls on one layer's worth of entries: the
    rounding step alone (fp32 values in, codes and group scales out) and the
    threshold words alone (32-bit words out). Each is timed over `steps` launches
    between two events on the launch stream; bytes are the call's own reads and
    writes (fp32 in 4 B, codes, 4 B per scale, 4 B per threshold word)."""
    import torch

    import paper_2609_39185_amd as ssmq
    from paper_2609_39185_amd import workloads as wl

    n = w.entries_per_layer
    head = w.headdim * w.dstate
    stream = torch.cuda.current_stream(device)
    g = torch.Generator(device=device).manual_seed(7)
    h = torch.randn(n, generator=g, device=device) * 0.3
    code_dtype = {"bf16": torch.int16, "fp16": torch.int16, "e4m3": torch.uint8,
                  "int8": torch.uint8, "int4": torch.uint8}

    def timed(fn):
        for k in range(warmup):
            fn(k)
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record(stream)
        for k in range(steps):
            fn(warmup + k)
        stop.record(stream)
        torch.cuda.synchronize()
        return start.elapsed_time(stop) * 1e3 / steps

    out = {"workload": w.name, "entries": n, "launches_timed": steps, "requantize": {}, "dither_fill": {}}
    for fmt, rule, group in (("bf16", "rtn", 0), ("bf16", "weyl", 0), ("bf16", "sr", 0),
                             ("bf16", "philox", 0), ("e4m3", "weyl", head), ("e4m3", "weyl", 128),
                             ("int8", "weyl", 128), ("int4", "weyl", 128)):
        codes = torch.empty(n // (2 if fmt == "int4" else 1), dtype=code_dtype[fmt], device=device)
        scale = torch.empty(n // group, device=device) if fmt in ("e4m3", "int8", "int4") else None
        us = timed(lambda k: ssmq.requantize(h, codes, scale, rule=rule, fmt=fmt, head_size=head,
                                             dither_block=w.dither_block, scale_group=group,
                                             step=k, stream=stream))
        nbytes = n * 4 + int(n * state_bytes_per_entry(fmt)) + (4 * (n // group) if scale is not None else 0)
        out["requantize"][f"{fmt}/{group}:{rule}" if scale is not None else f"{fmt}:{rule}"] = {
            "us": us, "GBps": nbytes / (us * 1e3), "bytes": nbytes}
        del codes, scale
    words = torch.empty(n, dtype=torch.int32, device=device)
    for rule in ("weyl", "sr", "philox"):
        us = timed(lambda k: ssmq.dither_fill(words, rule=rule, step=k, dither_block=w.dither_block,
                                              stream=stream))
        out["dither_fill"][rule] = {"us": us, "GBps": 4 * n / (us * 1e3), "bytes": 4 * n}
    return out


def cpu_baseline(w, variant, target_s):
    """Time the oracle on whole head tiles of one layer until ~target_s of CPU work."""
    import numpy as np
    import torch

    import oracle
    from paper_2609_39185_amd import workloads as wl

    fmt, rule, group = variant["fmt"], variant["rule"], variant["group"]
    P, N = w.headdim, w.dstate
    A, D = wl.layer_params(w.family, w.nheads, N, seed=1000)
    x, dt, B, C = wl.step_inputs(1, w.nheads, P, N, w.ngroups, seed=2000)
    codes, scale = wl.initial_state(fmt, 1, w.nheads, P, N, seed=3000, group=group)
    codes_np = wl.to_numpy_codes(fmt, codes)
    args = (None if scale is None else scale.numpy(), x.numpy(), dt.numpy(), A.numpy(),
            B.numpy(), C.numpy(), D.numpy())

    def run(nh):
        c = codes_np[:, :nh]
        sc = None if args[0] is None else args[0][:nh]
        t0 = time.perf_counter()
        oracle.state_update(fmt, rule, c, sc, args[1][:, :nh], args[2][:, :nh], args[3][:nh],
                            args[4][:, :1], args[5][:, :1], args[6][:nh], block=w.dither_block,
                            group=group, step=1)
        return time.perf_counter() - t0

    probe_heads = w.nheads // w.ngroups   # the heads of one B/C group
    tile_bytes = probe_heads * P * N * state_bytes_per_entry(fmt) * 2
    run(probe_heads)                       # first call: loading and first-touch costs
    # one thread
    reps, total = 0, 0.0
    while total < target_s:
        total += run(probe_heads)
        reps += 1
    single = {"value": reps * tile_bytes / total / 1e9,
              "sample": f"{reps} calls, {total:.1f} s",
              "us_per_head_tile": total / (reps * probe_heads) * 1e6}
    # every core the process may use (at most 16, the host share of one GPU):
    # independent calls on separate threads (the C oracle runs without the GIL)
    from concurrent.futures import ThreadPoolExecutor

    cores = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else (os.cpu_count() or 1)
    cores = max(1, min(cores, int(os.environ.get("OMP_NUM_THREADS") or 16), 16))

    def worker(deadline):
        n = 0
        while time.perf_counter() < deadline:
            run(probe_heads)
            n += 1
        return n

    t0 = time.perf_counter()
    with ThreadPoolExecutor(max_workers=cores) as pool:
        calls = sum(pool.map(worker, [t0 + target_s] * cores))
    wall = time.perf_counter() - t0
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), None)
    except OSError:
        pass
    host = {"cpu_model": model, "cpu_count": os.cpu_count(),
            "usable_cpus": len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else None}
    return {
        "value": calls * tile_bytes / wall / 1e9,
        "unit": "GB/s",
        "cores": cores,
        "kind": "oracle",
        "sample": f"{calls} calls on {cores} threads, each a {probe_heads}-head tile group "
                  f"({P}x{N} per head) of one layer of {w.name}, {fmt} {rule}, the C oracle, "
                  f"{wall:.1f} s wall",
        "single_thread": single,
        "host": host,
    }


if __name__ == "__main__":
    sys.exit(main())
