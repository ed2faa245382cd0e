#!/usr/bin/env python3
"""Benchmark of the beam-search decode step on one MI355X.

One step = the whole hot path on one batch, in one launch
(fs_beam_decode_step): the cross-attention in which the k beams of every
source read its one de-duplicated K/V copy, with the no-repeat-n-gram scan of
the step's hypotheses done by extra workgroups of the same grid.  The same
step as two launches (fs_beam_cross_attn, then fs_ngram_block) is timed
beside it.  Inputs are
seeded synthetic BART-large-shaped tensors (workloads.py), resident in HBM
before timing starts.  Each step reads a different K/V set, rotating over at
least 1 GiB of sets so that the 256 MB last-level cache cannot hold them.

Prints ONE JSON line:
  value        algorithmic bytes of the step / step time (GB/s)
  ms_per_step  mean step time over exactly K timed steps (HIP events at the
               two ends of the region, on the stream the kernels run on)
  roofline     the cross-attention kernel's algorithmic GB/s against 8 TB/s:
               its bytes per launch / its average launch duration, timed
               with HIP events around K back-to-back launches on the same
               stream (per-launch event records would add several us each)
  cpu_baseline the CPU oracle on the host cores, on the same inputs
"""
from __future__ import annotations

import argparse
import json
import math
import os
import pathlib
import sys
import time

ROOT = pathlib.Path(__file__).resolve().parent
sys.path.insert(0, str(ROOT))

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E
# The oracle is timed over repeated whole steps until about this much host
# time is spent (or this many repetitions), and the median is reported.
ORACLE_BUDGET_S = 10.0
ORACLE_MAX_REPS = 2000


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=500,
                    help="untimed steps first (about 12 ms at the BART shape, enough for the clocks to settle)")
    ap.add_argument("--config", default="bart",
                    help="decode step: tiny | bart | t5 | prophetnet | large; "
                         "split-cache self-attention step: gpt2 | tiny_prefix")
    ap.add_argument("--part", default="step", choices=("step", "select", "reorder", "indirect", "sweep"),
                    help="step: the decode step (cross-attention + n-gram blocking); "
                         "select: the beam-selection step on the same config's logits")
    ap.add_argument("--rounds", type=int, default=5,
                    help="alternating (steps, cross-attention only) region pairs for the per-kernel split")
    ap.add_argument("--rotate-gib", type=float, default=1.0,
                    help="minimum total size of the rotated K/V sets")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-reps", type=int, default=0,
                    help="oracle repetitions for the CPU baseline (0: until ~10 s)")
    ap.add_argument("--copy-calibrate", type=float, default=0.0, metavar="GIB",
                    help="instead of the step, run a plain device copy of this many GiB "
                         "(reference for the FETCH_SIZE/WRITE_SIZE counters)")
    ap.add_argument("--summarize-trace", default="", metavar="CSV",
                    help="instead of running, print the kernel durations of a rocprofv3 kernel-trace CSV "
                         "grouped by kernel and grid size (a fused step and the attention alone differ in grid)")
    ap.add_argument("--traffic", default=str(ROOT / "profiles" / "traffic.json"),
                    help="HBM traffic per launch measured with rocprofv3 counters")
    return ap.parse_args()


def attn_bytes(cfg, lens) -> int:
    """Algorithmic bytes of one cross-attention call: valid K and V rows,
    q and out, and src_len.  Padding rows are never read."""
    e = cfg.esize
    kv = 2 * int(sum(int(x) for x in lens)) * cfg.H * cfg.D * e
    qo = 2 * cfg.B * cfg.k * cfg.H * cfg.D * e
    return kv + qo + 4 * cfg.B


def ngram_bytes(rows: int, t: int, bans: int) -> int:
    """Algorithmic bytes of one n-gram call: the token history is read once;
    each banned logit is one 4-byte store (the logits are never read)."""
    return rows * t * 4 + 4 * bans


def prefix_bytes(cfg, lens, t: int) -> int:
    """Algorithmic bytes of one split-cache self-attention call: the valid
    prefix rows of K and V once per sample, the t generated rows of every
    beam, q and out, and prefix_len."""
    e = cfg.esize
    kv = 2 * int(sum(int(x) for x in lens)) * cfg.H * cfg.D * e
    gen = 2 * cfg.B * cfg.k * cfg.H * t * cfg.D * e
    qo = 2 * cfg.B * cfg.k * cfg.H * cfg.D * e
    return kv + gen + qo + 4 * cfg.B


SETTLE_MS = 20.0        # back-to-back steps before the warm-up, so that the clocks are up
SPREAD_MIN_CALLS = 20   # calls per sub-region of the spread, whatever --steps is


def settle(stream, fn, ms: float = SETTLE_MS) -> int:
    """Run ``fn(i)`` back to back for about ``ms`` of GPU time (untimed);
    returns the number of calls."""
    import torch
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    calls, batch = 0, 50
    torch.cuda.synchronize()
    a.record(stream)
    while True:
        for i in range(batch):
            fn(calls + i)
        calls += batch
        b.record(stream)
        b.synchronize()
        if a.elapsed_time(b) >= ms or calls >= 100000:
            return calls


def launch_spread(stream, fn, K: int, parts: int = 10) -> dict:
    """Median, p10 and p90 of the mean per-call time of ``fn(i)`` over
    ``parts`` equal sub-regions of back-to-back calls (events only at the
    sub-region ends), each of at least SPREAD_MIN_CALLS calls.  Timed in a
    pass of its own, so that its extra events never enter the headline
    means."""
    import numpy as np
    import torch
    per = max(SPREAD_MIN_CALLS, K // parts)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(parts + 1)]
    torch.cuda.synchronize()
    i = 0
    ev[0].record(stream)
    for p in range(parts):
        for _ in range(per):
            fn(i)
            i += 1
        ev[p + 1].record(stream)
    torch.cuda.synchronize()
    us = np.array([ev[p].elapsed_time(ev[p + 1]) * 1e3 / per for p in range(parts)])
    return {"median": round(float(np.median(us)), 3), "p10": round(float(np.percentile(us, 10)), 3),
            "p90": round(float(np.percentile(us, 90)), 3), "subregions": parts, "calls_each": per}


def graph_step_us(dev, step, n_steps: int, replays: int = 10):
    """Per-step time when n_steps steps (the K/V rotation included) are
    captured into one HIP graph and the graph is replayed: the same kernels
    without the host's launch calls between them.  None if a call refuses
    capture."""
    import torch
    try:
        cur = torch.cuda.current_stream(dev)
        side = torch.cuda.Stream(dev)
        side.wait_stream(cur)
        with torch.cuda.stream(side):
            for i in range(n_steps):
                step(i)
        cur.wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for i in range(n_steps):
                step(i)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(cur)
        for _ in range(replays):
            g.replay()
        b.record(cur)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / (replays * n_steps)
    except Exception:  # noqa: BLE001 - a decomposition that cannot be captured
        return None


def load_traffic(path: str, name: str):
    """HBM bytes per launch from the counter summary, if it was taken on the
    current kernel sources."""
    tp = pathlib.Path(path)
    if not tp.exists():
        return None
    try:
        rec = json.loads(tp.read_text()).get(name)
    except (ValueError, OSError):
        return None
    if rec and rec.get("kernel_source_sha") == kernel_source_sha():
        return rec.get("bytes_per_launch")
    return None


def copy_bandwidth(dev, gib: float = 1.0, reps: int = 5) -> float:
    """Read+write GB/s of a plain 1 GiB device copy: the achievable-bandwidth reference."""
    import torch
    n = int(gib * (1 << 30)) // 4
    src = torch.ones(n, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record()
    for _ in range(reps):
        dst.copy_(src)
    b.record()
    torch.cuda.synchronize()
    gbps = 2 * n * 4 * reps / (a.elapsed_time(b) * 1e-3) / 1e9
    del src, dst
    return gbps


def copy_calibrate(gib: float) -> None:
    import torch
    n = int(gib * (1 << 30)) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "launches": 5}))


def summarize_trace(path: str) -> int:
    """Kernel durations of a rocprofv3 --kernel-trace CSV, grouped by
    (kernel, workgroups): device begin/end timestamps, in microseconds."""
    import csv
    import statistics
    groups: dict = {}
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            wg = int(r["Grid_Size_X"]) // max(1, int(r["Workgroup_Size_X"]))
            us = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3
            groups.setdefault((r["Kernel_Name"], wg, int(r["Workgroup_Size_X"])), []).append(us)
    print(f"{'kernel':70s} {'workgroups':>10s} {'threads':>7s} {'calls':>6s} {'avg us':>8s} "
          f"{'median':>8s} {'min us':>8s} {'max us':>8s}")
    for (name, wg, th), v in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        print(f"{name[:70]:70s} {wg:10d} {th:7d} {len(v):6d} {statistics.fmean(v):8.2f} "
              f"{statistics.median(v):8.2f} {min(v):8.2f} {max(v):8.2f}")
    return 0


def main() -> int:
    args = parse()
    if args.summarize_trace:
        return summarize_trace(args.summarize_trace)
    if args.gpus != 1:
        print(f"bench.py: the benchmark runs on one GPU; --gpus {args.gpus} is not supported "
              "(the decode step would shard by source with no exchange between GPUs)",
              file=sys.stderr)
        return 2
    import numpy as np
    import torch

    from paper_2106_04718_amd import api, workloads

    if args.copy_calibrate > 0:
        copy_calibrate(args.copy_calibrate)
        return 0

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    if args.config in workloads.PREFIX_CONFIGS:
        if args.part == "indirect":
            return bench_indirect(args, workloads.PREFIX_CONFIGS[args.config], dev)
        return bench_prefix(args, workloads.PREFIX_CONFIGS[args.config], dev)
    if args.part == "indirect":
        print("bench.py: --part indirect runs on a split-cache config (gpt2, tiny_prefix)", file=sys.stderr)
        return 2
    if args.part == "select":
        return bench_select(args, workloads.get(args.config), dev)
    if args.part == "reorder":
        return bench_reorder(args, workloads.get(args.config), dev)
    if args.part == "sweep":
        return bench_sweep(args, workloads.get(args.config), dev)
    cfg = workloads.get(args.config)
    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32

    def dev_tensor(a):
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    # ---- inputs, resident in HBM -----------------------------------------
    t0 = time.perf_counter()
    base = workloads.attn_inputs(cfg)
    lens = base["src_len"]
    set_bytes = 2 * cfg.B * cfg.H * cfg.S * cfg.D * cfg.esize
    R = max(1, math.ceil(args.rotate_gib * (1 << 30) / set_bytes))
    q = dev_tensor(base["q"])
    lens_d = dev_tensor(lens)
    Ks, Vs = [dev_tensor(base["K"])], [dev_tensor(base["V"])]
    for r in range(1, R):
        d = workloads.attn_inputs(cfg, rep=r)
        Ks.append(dev_tensor(d["K"]))
        Vs.append(dev_tensor(d["V"]))
        del d
    g = workloads.ngram_inputs(cfg)
    tokens_d = dev_tensor(g["tokens"])
    logits_d = dev_tensor(g["logits"])
    out = torch.empty_like(q)
    ws = api.new_workspace(api.beam_cross_attn_workspace_bytes(cfg.B, cfg.k, cfg.H, cfg.S, cfg.D, tdt), dev)
    torch.cuda.synchronize()
    log(f"config={cfg.name} K/V sets={R} ({R * set_bytes / 2**30:.2f} GiB) inputs ready in "
        f"{time.perf_counter() - t0:.1f}s")

    def step(i: int):
        # the whole step in one launch: the n-gram rows ride in the attention grid
        api.beam_decode_step(q, Ks[i % R], Vs[i % R], lens_d, tokens_d, cfg.n, logits_d, out=out, workspace=ws)

    def step_separate(i: int):
        api.beam_cross_attn(q, Ks[i % R], Vs[i % R], lens_d, out=out, workspace=ws)
        api.ngram_block(tokens_d, cfg.n, logits_d)

    def ca_only(i: int):
        api.beam_cross_attn(q, Ks[i % R], Vs[i % R], lens_d, out=out, workspace=ws)

    # ---- first step: outputs kept for the CPU-baseline comparison ---------
    step(0)
    torch.cuda.synchronize()
    out0 = out.float().cpu().numpy().astype(np.float64)
    logits0 = logits_d.cpu().numpy()
    bans = int(np.isneginf(logits0).sum())

    # ---- settle, warm-up and timed regions ---------------------------------
    # The clocks are settled first by SETTLE_MS of back-to-back steps, so
    # that a short warm-up (--warmup) still times a GPU at its working
    # clocks; then W warm-up steps and region A, which times exactly K steps
    # with events only at its two ends (event records between kernels would
    # themselves add microseconds per step).  Region A gives the headline.
    # Then `rounds` triples of regions alternate on the same stream with the
    # same K/V rotation: K steps (A_r), K cross-attention launches alone
    # (B_r) and K steps as two launches (C_r).  The cross-attention's average
    # launch duration is the median of B_r; the n-gram scan's cost in the
    # fused step is the median of A_r - B_r (pairing cancels clock drift),
    # and in the two-launch step the median of C_r - B_r.
    stream = torch.cuda.current_stream(dev)
    settle_calls = settle(stream, step)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    K_ = args.steps

    def region_us(fn) -> float:
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for i in range(K_):
            fn(i)
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / K_

    w0 = time.perf_counter()
    step_us = region_us(step)
    wall = time.perf_counter() - w0
    trips = [(region_us(step), region_us(ca_only), region_us(step_separate)) for _ in range(max(1, args.rounds))]
    ca_us = float(np.median([b for _, b, _ in trips]))
    ng_us = max(float(np.median([a - b for a, b, _ in trips])), 0.0)
    sep_us = float(np.median([c for _, _, c in trips]))
    ng_sep_us = max(float(np.median([c - b for _, b, c in trips])), 0.0)
    step_spread = launch_spread(stream, step, K_)
    ca_spread = launch_spread(stream, ca_only, K_)
    g_us = graph_step_us(dev, step, 3 * R)
    ms_per_step = step_us * 1e-3
    b_ca = attn_bytes(cfg, lens)
    b_ng = ngram_bytes(cfg.rows, cfg.t, bans)
    b_step = b_ca + b_ng
    value = b_step / (ms_per_step * 1e-3) / 1e9
    ca_gbps = b_ca / (ca_us * 1e-6) / 1e9
    copy_gbps = copy_bandwidth(dev)
    log(f"step {step_us:.2f} us (one launch; wall {wall / K_ * 1e6:.2f} us) = {value:.0f} GB/s; cross-attn "
        f"{ca_us:.2f} us = {ca_gbps:.0f} GB/s ({100 * ca_gbps / HBM_PEAK_GBPS:.1f}% of 8 TB/s, "
        f"{100 * ca_gbps / copy_gbps:.1f}% of the measured copy bandwidth {copy_gbps:.0f} GB/s); "
        f"n-gram adds {ng_us:.2f} us = {100 * ng_us / step_us:.1f}% of the step; as two launches the step takes "
        f"{sep_us:.2f} us (n-gram {100 * ng_sep_us / sep_us:.1f}%)")
    if g_us is not None:
        log(f"the same step replayed from a HIP graph of {3 * R} steps: {g_us:.2f} us per step")

    traffic = load_traffic(args.traffic, cfg.name)

    line = {
        "metric": "decode-step µs and achieved HBM GB/s (cross-attn + n-gram block), BART-large shape",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K_,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 6),
        "step_us": round(ms_per_step * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded; BART-large-shaped K/V, Zipf(1.1) token prefixes)",
        "config": {"workload": workload_name(cfg), "B": cfg.B, "k": cfg.k, "H": cfg.H, "D": cfg.D,
                   "S": cfg.S, "t": cfg.t, "V": cfg.V, "n": cfg.n, "kv_sets_rotated": R,
                   "bytes_per_step": b_step},
        "step_us_spread": step_spread,
        "step_launches": 1,
        "settle_calls": settle_calls,
        "cross_attn_us": round(ca_us, 3),
        "cross_attn_us_spread": ca_spread,
        "ngram_us": round(ng_us, 3),
        "ngram_share_of_step": round(ng_us / step_us, 4),
        "step_two_launches_us": round(sep_us, 3),
        "ngram_share_two_launches": round(ng_sep_us / sep_us, 4),
        "step_us_graph": None if g_us is None else round(g_us, 3),
        "timing_rounds": max(1, args.rounds),
        "copy_gbps": round(copy_gbps, 1),
        "roofline": {"bound": "hbm", "kernel": "fs_beam_cross_attn", "achieved": round(ca_gbps, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(ca_gbps / HBM_PEAK_GBPS, 4),
                     "algorithmic_bytes_per_launch": b_ca, "traffic": traffic},
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"], line["parity"] = cpu_baseline(cfg, base, g, out0, logits0, b_step,
                                                             args.cpu_reps)
    print(json.dumps(line), flush=True)
    return 0


def bench_sweep(args, cfg, dev) -> int:
    """The decode step over the prefix lengths t = 1 .. cfg.t of one token
    buffer (ld = cfg.t; step t reads its first t columns), at the config's
    full batch.  The cross-attention does not depend on t; at every t the
    step (cross-attention then n-gram) is timed against the cross-attention
    alone, in alternating regions of K steps."""
    import numpy as np
    import torch

    from paper_2106_04718_amd import api, workloads

    def dev_tensor(a):
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    t0 = time.perf_counter()
    base = workloads.attn_inputs(cfg)
    lens = base["src_len"]
    set_bytes = 2 * cfg.B * cfg.H * cfg.S * cfg.D * cfg.esize
    R = max(1, math.ceil(args.rotate_gib * (1 << 30) / set_bytes))
    q, lens_d = dev_tensor(base["q"]), dev_tensor(lens)
    Ks, Vs = [dev_tensor(base["K"])], [dev_tensor(base["V"])]
    for r in range(1, R):
        d = workloads.attn_inputs(cfg, rep=r)
        Ks.append(dev_tensor(d["K"]))
        Vs.append(dev_tensor(d["V"]))
        del d
    del base
    g = workloads.ngram_inputs(cfg)
    tokens_d, logits0 = dev_tensor(g["tokens"]), dev_tensor(g["logits"])
    del g
    logits_d = torch.empty_like(logits0)
    out = torch.empty_like(q)
    ws = api.new_workspace(api.beam_cross_attn_workspace_bytes(cfg.B, cfg.k, cfg.H, cfg.S, cfg.D, tdt), dev)
    torch.cuda.synchronize()
    log(f"config={cfg.name} sweep: K/V sets={R} ({R * set_bytes / 2**30:.2f} GiB), t = 1..{cfg.t}, "
        f"inputs ready in {time.perf_counter() - t0:.1f}s")
    stream = torch.cuda.current_stream(dev)
    K_ = args.steps

    def region_us(fn) -> float:
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record(stream)
        for i in range(K_):
            fn(i)
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / K_

    def ca_only(i: int):
        api.beam_cross_attn(q, Ks[i % R], Vs[i % R], lens_d, out=out, workspace=ws)

    logits_d.copy_(logits0)
    for i in range(args.warmup):
        ca_only(i)
        api.ngram_block(tokens_d, cfg.n, logits_d)
    b_ca = attn_bytes(cfg, lens)
    rows = []
    for t in range(1, cfg.t + 1):
        logits_d.copy_(logits0)
        tok_t = tokens_d[:, :t]
        api.ngram_block(tok_t, cfg.n, logits_d)
        bans = int(torch.isneginf(logits_d).sum().item())

        def step(i: int, tok_t=tok_t):
            api.beam_decode_step(q, Ks[i % R], Vs[i % R], lens_d, tok_t, cfg.n, logits_d, out=out, workspace=ws)

        a_us, b_us = region_us(step), region_us(ca_only)
        b_step = b_ca + ngram_bytes(cfg.rows, t, bans)
        rows.append({"t": t, "step_us": round(a_us, 3), "cross_attn_us": round(b_us, 3),
                     "ngram_us": round(max(a_us - b_us, 0.0), 3), "bans": bans,
                     "step_gbps": round(b_step / (a_us * 1e-6) / 1e9, 1)})
        if t in (1, 2, 4, 8, 16, 32, 64, 96, 128, cfg.t):
            r = rows[-1]
            log(f"t={t:3d}: step {r['step_us']:.2f} us = {r['step_gbps']:.0f} GB/s; cross-attn {r['cross_attn_us']:.2f} us; "
                f"n-gram {r['ngram_us']:.2f} us ({bans} bans)")
    ca = float(np.median([r["cross_attn_us"] for r in rows]))
    ca_gbps = b_ca / (ca * 1e-6) / 1e9
    last = rows[-1]
    line = {
        "metric": "decode-step µs and achieved HBM GB/s (cross-attn + n-gram block) over the prefix-length sweep",
        "value": last["step_gbps"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K_,
        "warmup": args.warmup,
        "ms_per_step": round(last["step_us"] * 1e-3, 6),
        "step_us": last["step_us"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded; BART-large-shaped K/V, Zipf(1.1) token prefixes)",
        "config": {"workload": workload_name(cfg) + f", prefix length swept t = 1..{cfg.t}", "B": cfg.B,
                   "k": cfg.k, "H": cfg.H, "D": cfg.D, "S": cfg.S, "V": cfg.V, "n": cfg.n,
                   "kv_sets_rotated": R},
        "cross_attn_us_median": round(ca, 3),
        "roofline": {"bound": "hbm", "kernel": "fs_beam_cross_attn", "achieved": round(ca_gbps, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(ca_gbps / HBM_PEAK_GBPS, 4),
                     "algorithmic_bytes_per_launch": b_ca, "traffic": None},
        "sweep": rows,
        "cpu_baseline": None,
    }
    print(json.dumps(line), flush=True)
    return 0


def bench_prefix(args, cfg, dev) -> int:
    """Split-cache self-attention step (decoder-only beam search): each
    sample's prefix K/V read once for its k beams, plus each beam's own
    generated K/V, one softmax.  A step is one fs_beam_prefix_attn call."""
    import numpy as np
    import torch

    from paper_2106_04718_amd import api, workloads

    def dev_tensor(a):
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    t0 = time.perf_counter()
    base = workloads.prefix_inputs(cfg)
    lens, t = base["prefix_len"], base["t"]
    set_bytes = sum(base[x].nbytes for x in ("Kp", "Vp", "Kt", "Vt"))
    R = max(1, math.ceil(args.rotate_gib * (1 << 30) / set_bytes))
    q, lens_d = dev_tensor(base["q"]), dev_tensor(lens)
    sets = [tuple(dev_tensor(base[x]) for x in ("Kp", "Vp", "Kt", "Vt"))]
    for r in range(1, R):
        d = workloads.prefix_inputs(cfg, rep=r)
        sets.append(tuple(dev_tensor(d[x]) for x in ("Kp", "Vp", "Kt", "Vt")))
        del d
    out = torch.empty_like(q)
    ws = api.new_workspace(api.beam_prefix_attn_workspace_bytes(cfg.B, cfg.k, cfg.H, cfg.N, cfg.T, cfg.D, tdt),
                           dev)
    torch.cuda.synchronize()
    log(f"config={cfg.name} K/V sets={R} ({R * set_bytes / 2**30:.2f} GiB) inputs ready in "
        f"{time.perf_counter() - t0:.1f}s")

    def step(i: int):
        Kp, Vp, Kt, Vt = sets[i % R]
        api.beam_prefix_attn(q, Kp, Vp, lens_d, Kt, Vt, t, out=out, workspace=ws)

    step(0)
    torch.cuda.synchronize()
    out0 = out.float().cpu().numpy().astype(np.float64)
    for i in range(args.warmup):
        step(i)
    K_ = args.steps
    stream = torch.cuda.current_stream(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for i in range(K_):
        step(i)
    e1.record(stream)
    torch.cuda.synchronize()
    step_us = e0.elapsed_time(e1) * 1e3 / K_
    spread = launch_spread(stream, step, K_)
    b = prefix_bytes(cfg, lens, t)
    gbps = b / (step_us * 1e-6) / 1e9
    copy_gbps = copy_bandwidth(dev)
    log(f"prefix step {step_us:.2f} us = {gbps:.0f} GB/s ({100 * gbps / HBM_PEAK_GBPS:.1f}% of 8 TB/s, "
        f"{100 * gbps / copy_gbps:.1f}% of the measured copy bandwidth {copy_gbps:.0f} GB/s)")
    line = {
        "metric": "self-attention step µs and achieved HBM GB/s (split-cache prefix attention), GPT2 shape",
        "value": round(gbps, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K_,
        "warmup": args.warmup,
        "ms_per_step": round(step_us * 1e-3, 6),
        "step_us": round(step_us, 3),
        "step_us_spread": spread,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded; shared prefix K/V per sample, per-beam generated K/V)",
        "config": {"workload": (f"{cfg.name}-shaped split-cache self-attention step: B={cfg.B} k={cfg.k} "
                                f"H={cfg.H} D={cfg.D}, shared prefix N={cfg.N} (lengths U{{{cfg.len_lo}.."
                                f"{cfg.len_hi}}}), {t} generated tokens per beam (capacity {cfg.T}), "
                                f"{cfg.dtype}"),
                   "B": cfg.B, "k": cfg.k, "H": cfg.H, "D": cfg.D, "N": cfg.N, "T": cfg.T, "t": t,
                   "kv_sets_rotated": R, "bytes_per_step": b},
        "copy_gbps": round(copy_gbps, 1),
        "roofline": {"bound": "hbm", "kernel": "fs_beam_prefix_attn", "achieved": round(gbps, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(gbps / HBM_PEAK_GBPS, 4),
                     "algorithmic_bytes_per_launch": b, "traffic": load_traffic(args.traffic, cfg.name)},
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        import oracle
        qd, Kpd, Vpd, Ktd, Vtd = (np.ascontiguousarray(oracle.widen(base[x]))
                                  for x in ("q", "Kp", "Vp", "Kt", "Vt"))
        times, ref = [], None
        while True:
            c0 = time.perf_counter()
            ref = oracle.prefix_attn(qd, Kpd, Vpd, lens, Ktd, Vtd, t)
            times.append(time.perf_counter() - c0)
            if (args.cpu_reps and len(times) >= args.cpu_reps) or \
                    (not args.cpu_reps and (sum(times) > ORACLE_BUDGET_S or len(times) >= ORACLE_MAX_REPS)):
                break
        sec = float(np.median(times))
        err = float(np.max(np.abs(out0 - ref)))
        tol = 2e-2 if cfg.dtype == "bf16" else 1e-5 * float(np.max(np.abs(ref)))
        log(f"oracle: {sec * 1e3:.1f} ms per step on {oracle.num_threads()} threads; attn max abs err {err:.3e}")
        line["cpu_baseline"] = {"value": round(b / sec / 1e9, 4), "unit": "GB/s", "cores": oracle.num_threads(),
                                "kind": "oracle",
                                "sample": f"whole {cfg.name}-shaped step, K/V set 0, median of {len(times)} reps, "
                                          f"{sec * 1e3:.1f} ms per step"}
        line["parity"] = {"attn_max_abs_err": err, "attn_tol": tol, "attn_ok": err <= tol}
    print(json.dumps(line), flush=True)
    return 0


def bench_indirect(args, cfg, dev) -> int:
    """Split-cache self-attention with the generated rows read through an
    ancestry table (the reorder-free cache maintenance).  A step is one
    fs_beam_prefix_attn_indirect call; the same run times the direct call on
    the same inputs, the fs_cache_reorder of that layer's generated K/V that
    the table replaces, and one fs_beam_ancestry_step (once per decode step,
    shared by the layers)."""
    import numpy as np
    import torch

    from paper_2106_04718_amd import api, workloads

    def dev_tensor(a):
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(a).to(dev)

    tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    t0 = time.perf_counter()
    base = workloads.prefix_inputs(cfg)
    am = workloads.ancestry_inputs(cfg)
    lens, t = base["prefix_len"], base["t"]
    set_bytes = sum(base[x].nbytes for x in ("Kp", "Vp", "Kt", "Vt"))
    R = max(1, math.ceil(args.rotate_gib * (1 << 30) / set_bytes))
    q, lens_d = dev_tensor(base["q"]), dev_tensor(lens)
    anc_d, par_d = dev_tensor(am["anc"]), dev_tensor(am["parent"])
    anc_scratch = anc_d.clone()
    sets = [tuple(dev_tensor(base[x]) for x in ("Kp", "Vp", "Kt", "Vt"))]
    for r in range(1, R):
        d = workloads.prefix_inputs(cfg, rep=r)
        sets.append(tuple(dev_tensor(d[x]) for x in ("Kp", "Vp", "Kt", "Vt")))
        del d
    out = torch.empty_like(q)
    ws = api.new_workspace(api.beam_prefix_attn_workspace_bytes(cfg.B, cfg.k, cfg.H, cfg.N, cfg.T, cfg.D, tdt),
                           dev)
    torch.cuda.synchronize()
    log(f"config={cfg.name} indirect: K/V sets={R} ({R * set_bytes / 2**30:.2f} GiB) inputs ready in "
        f"{time.perf_counter() - t0:.1f}s")
    stream = torch.cuda.current_stream(dev)

    def timed(fn, K):
        for i in range(args.warmup):
            fn(i)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for i in range(K):
            fn(i)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / K

    def step(i: int):
        Kp, Vp, Kt, Vt = sets[i % R]
        api.beam_prefix_attn(q, Kp, Vp, lens_d, Kt, Vt, t, out=out, workspace=ws, anc=anc_d)

    def direct(i: int):
        Kp, Vp, Kt, Vt = sets[i % R]
        api.beam_prefix_attn(q, Kp, Vp, lens_d, Kt, Vt, t, out=out, workspace=ws)

    def reorder(i: int):
        _, _, Kt, Vt = sets[i % R]
        api.cache_reorder(Kt, Vt, par_d, cfg.k, t)

    def anc_step(i: int):
        api.ancestry_step(anc_scratch, par_d, cfg.k, min(t, cfg.T - 1))

    step(0)
    torch.cuda.synchronize()
    out0 = out.float().cpu().numpy().astype(np.float64)
    K_ = args.steps
    step_us = timed(step, K_)
    spread = launch_spread(stream, step, K_)
    direct_us = timed(direct, K_)
    reorder_us = timed(reorder, K_)
    anc_us = timed(anc_step, K_)
    b = prefix_bytes(cfg, lens, t) + cfg.B * cfg.k * t * 4
    gbps = b / (step_us * 1e-6) / 1e9
    copy_gbps = copy_bandwidth(dev)
    log(f"indirect step {step_us:.2f} us = {gbps:.0f} GB/s ({100 * gbps / HBM_PEAK_GBPS:.1f}% of 8 TB/s); direct "
        f"{direct_us:.2f} us; the layer's reorder it replaces {reorder_us:.2f} us; ancestry step {anc_us:.2f} us "
        f"per decode step (rate of back-to-back single launches)")
    line = {
        "metric": "split-cache self-attention step through an ancestry table, µs and achieved HBM GB/s, GPT2 shape",
        "value": round(gbps, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K_,
        "warmup": args.warmup,
        "ms_per_step": round(step_us * 1e-3, 6),
        "step_us": round(step_us, 3),
        "step_us_spread": spread,
        "direct_step_us": round(direct_us, 3),
        "reorder_us": round(reorder_us, 3),
        "ancestry_step_us": round(anc_us, 3),
        "per_layer_saving_us": round(direct_us + reorder_us - step_us, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded; shared prefix K/V per sample, per-beam generated K/V, ancestry floor(k*u^2))",
        "config": {"workload": (f"{cfg.name}-shaped split-cache self-attention step through an ancestry table: "
                                f"B={cfg.B} k={cfg.k} H={cfg.H} D={cfg.D}, shared prefix N={cfg.N}, {t} generated "
                                f"tokens per beam (capacity {cfg.T}), {cfg.dtype}"),
                   "B": cfg.B, "k": cfg.k, "H": cfg.H, "D": cfg.D, "N": cfg.N, "T": cfg.T, "t": t,
                   "kv_sets_rotated": R, "bytes_per_step": b},
        "copy_gbps": round(copy_gbps, 1),
        "roofline": {"bound": "hbm", "kernel": "fs_beam_prefix_attn_indirect", "achieved": round(gbps, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(gbps / HBM_PEAK_GBPS, 4),
                     "algorithmic_bytes_per_launch": b,
                     "traffic": load_traffic(args.traffic, cfg.name + "-indirect")},
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        import oracle
        times, ref = [], None
        while True:
            c0 = time.perf_counter()
            ref = oracle.prefix_attn_indirect(base["q"], base["Kp"], base["Vp"], lens, base["Kt"], base["Vt"],
                                              am["anc"], t)
            times.append(time.perf_counter() - c0)
            if (args.cpu_reps and len(times) >= args.cpu_reps) or \
                    (not args.cpu_reps and (sum(times) > ORACLE_BUDGET_S or len(times) >= ORACLE_MAX_REPS)):
                break
        sec = float(np.median(times))
        err = float(np.max(np.abs(out0 - ref)))
        tol = 2e-2 if cfg.dtype == "bf16" else 1e-5 * float(np.max(np.abs(ref)))
        log(f"oracle: {sec * 1e3:.1f} ms per step on {oracle.num_threads()} threads; attn max abs err {err:.3e}")
        line["cpu_baseline"] = {"value": round(b / sec / 1e9, 4), "unit": "GB/s", "cores": oracle.num_threads(),
                                "kind": "oracle",
                                "sample": f"whole {cfg.name}-shaped step, K/V set 0, median of {len(times)} reps, "
                                          f"{sec * 1e3:.1f} ms per step"}
        line["parity"] = {"attn_max_abs_err": err, "attn_tol": tol, "attn_ok": err <= tol}
    print(json.dumps(line), flush=True)
    return 0


def select_bytes(rows: int, V: int, t: int, B: int, c: int) -> int:
    """Algorithmic bytes of one beam-selection call: every logit once, the
    token history, the beam scores, and the three outputs."""
    return rows * V * 4 + rows * t * 4 + rows * 4 + B * c * 12


def bench_select(args, cfg, dev) -> int:
    """Beam-selection step (log-softmax, n-gram bans and each source's 2k best
    candidates) over the decode-step config's logits.  A step is one
    fs_beam_select call; each reads a different logits set, rotating over at
    least 1 GiB."""
    import numpy as np
    import torch

    from paper_2106_04718_amd import api, workloads

    t0 = time.perf_counter()
    d = workloads.select_inputs(cfg)
    rows, V, k, c, B = cfg.rows, cfg.V, d["k"], d["c"], d["B"]
    set_bytes = rows * V * 4
    R = max(1, math.ceil(args.rotate_gib * (1 << 30) / set_bytes))
    lg0 = torch.from_numpy(d["logits"]).to(dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(210604718 + cfg.index)
    sets = [lg0] + [torch.randn(rows, V, generator=gen, device=dev, dtype=torch.float32) for _ in range(R - 1)]
    bs = torch.from_numpy(d["beam_scores"]).to(dev)
    tok = torch.from_numpy(d["tokens"]).to(dev)
    outs = (torch.empty((B, c), dtype=torch.float32, device=dev), torch.empty((B, c), dtype=torch.int32, device=dev),
            torch.empty((B, c), dtype=torch.int32, device=dev))
    ws = api.new_workspace(api.beam_select_workspace_bytes(B, k, V, c), dev)
    torch.cuda.synchronize()
    log(f"config={cfg.name} select: logits sets={R} ({R * set_bytes / 2**30:.2f} GiB) inputs ready in "
        f"{time.perf_counter() - t0:.1f}s")

    def step(i: int):
        api.beam_select(sets[i % R], bs, k, c, tokens=tok, n=cfg.n, out=outs, workspace=ws)

    step(0)
    torch.cuda.synchronize()
    first = tuple(o.cpu().numpy().copy() for o in outs)
    for i in range(args.warmup):
        step(i)
    K_ = args.steps
    stream = torch.cuda.current_stream(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for i in range(K_):
        step(i)
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / K_
    spread = launch_spread(stream, step, K_)
    b = select_bytes(rows, V, cfg.t, B, c)
    gbps = b / (us * 1e-6) / 1e9
    copy_gbps = copy_bandwidth(dev)
    log(f"select step {us:.2f} us = {gbps:.0f} GB/s ({100 * gbps / HBM_PEAK_GBPS:.1f}% of 8 TB/s, "
        f"{100 * gbps / copy_gbps:.1f}% of the measured copy bandwidth {copy_gbps:.0f} GB/s)")
    line = {
        "metric": "beam-selection step µs and achieved HBM GB/s (log-softmax + n-gram ban + per-source top-2k)",
        "value": round(gbps, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K_,
        "warmup": args.warmup,
        "ms_per_step": round(us * 1e-3, 6),
        "step_us": round(us, 3),
        "step_us_spread": spread,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded; N(0,1) logits, Zipf token prefixes with one planted repeat per row)",
        "config": {"workload": (f"{cfg.name}-shaped beam-selection step: {rows} hypotheses (B={B}, k={k}) x "
                                f"V={V} fp32 logits, no-repeat-{cfg.n}-gram on t={cfg.t} tokens, c={c} "
                                f"candidates per source"),
                   "B": B, "k": k, "V": V, "t": cfg.t, "n": cfg.n, "c": c, "logits_sets_rotated": R,
                   "bytes_per_step": b},
        "copy_gbps": round(copy_gbps, 1),
        "roofline": {"bound": "hbm", "kernel": "fs_beam_select", "achieved": round(gbps, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(gbps / HBM_PEAK_GBPS, 4),
                     "algorithmic_bytes_per_launch": b,
                     "traffic": load_traffic(args.traffic, cfg.name + "-select")},
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        import oracle
        times, ref = [], None
        while True:
            c0 = time.perf_counter()
            ref = oracle.beam_select(d["logits"], d["beam_scores"], d["tokens"], cfg.t, cfg.n, k, c)
            times.append(time.perf_counter() - c0)
            if (args.cpu_reps and len(times) >= args.cpu_reps) or \
                    (not args.cpu_reps and (sum(times) > ORACLE_BUDGET_S or len(times) >= ORACLE_MAX_REPS)):
                break
        sec = float(np.median(times))
        same = bool(np.array_equal(first[1], ref[1]) and np.array_equal(first[2], ref[2]))
        err = float(np.max(np.abs(first[0].astype(np.float64) - ref[0])))
        log(f"oracle: {sec * 1e3:.1f} ms per step on {oracle.num_threads()} threads; same picks {same}, "
            f"max score err {err:.2e}")
        line["cpu_baseline"] = {"value": round(b / sec / 1e9, 4), "unit": "GB/s", "cores": oracle.num_threads(),
                                "kind": "oracle",
                                "sample": f"whole {cfg.name}-shaped selection step, logits set 0, median of "
                                          f"{len(times)} reps, {sec * 1e3:.1f} ms per step"}
        line["parity"] = {"same_picks": same, "max_score_err": err}
    print(json.dumps(line), flush=True)
    return 0


def workload_name(cfg) -> str:
    return (f"{cfg.name}-shaped decode step: cross-attn B={cfg.B} k={cfg.k} H={cfg.H} D={cfg.D} "
            f"S={cfg.S} (lengths U{{{cfg.len_lo}..{cfg.len_hi}}}) {cfg.dtype} + no-repeat-{cfg.n}-gram "
            f"on [{cfg.rows}, {cfg.t}] tokens, V={cfg.V}")


def reorder_bytes(parent, k: int, row_bytes: int, tensors: int = 2) -> int:
    """Algorithmic bytes of one cache reorder: each beam some other beam of
    its source continues is read once, each beam whose parent is another
    beam is written once; row_bytes = H*t*D*esize per beam and tensor."""
    import numpy as np
    p = np.asarray(parent).reshape(-1, k)
    reads = writes = 0
    for row in p:
        moved = [j for j in range(k) if 0 <= row[j] < k and row[j] != j]
        writes += len(moved)
        reads += len({int(row[j]) for j in moved})
    return (reads + writes) * row_bytes * tensors


def bench_reorder(args, cfg, dev) -> int:
    """Per-beam cache reorder of one decoder layer's K and V on the
    decode-step config.  A step is one fs_cache_reorder call; each reorders a
    different cache set, rotating over at least 1 GiB."""
    import numpy as np
    import torch

    from paper_2106_04718_amd import api, workloads

    t0 = time.perf_counter()
    d = workloads.reorder_inputs(cfg)
    B, k, H, T, t, D = d["B"], d["k"], d["H"], d["T"], d["t"], d["D"]
    dt = torch.bfloat16 if d["dtype"] == "bf16" else torch.float32
    esize = 2 if dt == torch.bfloat16 else 4
    set_bytes = 2 * B * k * H * T * D * esize
    R = max(1, math.ceil(args.rotate_gib * (1 << 30) / set_bytes))
    gen = torch.Generator(device=dev)
    gen.manual_seed(210604718 + cfg.index)
    sets = [(torch.randn((B * k, H, T, D), generator=gen, device=dev).to(dt),
             torch.randn((B * k, H, T, D), generator=gen, device=dev).to(dt)) for _ in range(R)]
    parent = torch.from_numpy(d["parent"]).to(dev)
    b = reorder_bytes(d["parent"], k, H * t * D * esize)
    torch.cuda.synchronize()
    log(f"config={cfg.name} reorder: cache sets={R} ({R * set_bytes / 2**30:.2f} GiB), "
        f"{b / 1e6:.1f} MB moved per call, inputs ready in {time.perf_counter() - t0:.1f}s")

    def step(i: int):
        Kc, Vc = sets[i % R]
        api.cache_reorder(Kc, Vc, parent, k, t)

    for i in range(args.warmup):
        step(i)
    K_ = args.steps
    stream = torch.cuda.current_stream(dev)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for i in range(K_):
        step(i)
    e1.record(stream)
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / K_
    spread = launch_spread(stream, step, K_)
    gbps = b / (us * 1e-6) / 1e9
    copy_gbps = copy_bandwidth(dev)
    log(f"reorder step {us:.2f} us = {gbps:.0f} GB/s ({100 * gbps / HBM_PEAK_GBPS:.1f}% of 8 TB/s, "
        f"{100 * gbps / copy_gbps:.1f}% of the measured copy bandwidth {copy_gbps:.0f} GB/s)")
    line = {
        "metric": "per-beam cache reorder µs and achieved HBM GB/s (one decoder layer's K and V, in place)",
        "value": round(gbps, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K_,
        "warmup": args.warmup,
        "ms_per_step": round(us * 1e-3, 6),
        "step_us": round(us, 3),
        "step_us_spread": spread,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": d["dtype"],
        "data": "synthetic (seeded; N(0,1) cache values, parents floor(k*u^2))",
        "config": {"workload": (f"{cfg.name}-shaped per-beam cache reorder: K and V [{B * k}, {H}, {T}, {D}] "
                                f"{d['dtype']} (B={B}, k={k}), t={t} positions, seeded parents"),
                   "B": B, "k": k, "H": H, "T": T, "t": t, "D": D, "cache_sets_rotated": R,
                   "bytes_per_step": b},
        "copy_gbps": round(copy_gbps, 1),
        "roofline": {"bound": "hbm", "kernel": "fs_cache_reorder", "achieved": round(gbps, 1),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(gbps / HBM_PEAK_GBPS, 4),
                     "algorithmic_bytes_per_launch": b,
                     "traffic": load_traffic(args.traffic, cfg.name + "-reorder")},
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        import oracle
        Kc, Vc = sets[0]
        view = torch.int16 if dt == torch.bfloat16 else torch.int32
        kh, vh = Kc.view(view).cpu().numpy(), Vc.view(view).cpu().numpy()
        par = d["parent"]
        times = []
        while True:
            c0 = time.perf_counter()
            rk = oracle.cache_reorder(kh, par, k, t)
            rv = oracle.cache_reorder(vh, par, k, t)
            times.append(time.perf_counter() - c0)
            if (args.cpu_reps and len(times) >= args.cpu_reps) or \
                    (not args.cpu_reps and (sum(times) > ORACLE_BUDGET_S or len(times) >= ORACLE_MAX_REPS)):
                break
        sec = float(np.median(times))
        api.cache_reorder(Kc, Vc, parent, k, t)
        torch.cuda.synchronize()
        same = bool(np.array_equal(Kc.view(view).cpu().numpy(), rk) and np.array_equal(Vc.view(view).cpu().numpy(), rv))
        log(f"oracle: {sec * 1e3:.1f} ms per step on {oracle.num_threads()} threads; GPU bit-exact {same}")
        line["cpu_baseline"] = {"value": round(b / sec / 1e9, 4), "unit": "GB/s", "cores": oracle.num_threads(),
                                "kind": "oracle",
                                "sample": f"whole {cfg.name}-shaped reorder step (K and V), cache set 0, median of "
                                          f"{len(times)} reps, {sec * 1e3:.1f} ms per step"}
        line["parity"] = {"bit_exact": same}
    print(json.dumps(line), flush=True)
    return 0


def kernel_source_sha() -> str:
    """Hash of what the kernels and their launches are built from: the HIP
    sources, the launch declarations and the build flags (a stored traffic
    figure is only used while it matches; host-side argument checks do not
    enter it)."""
    import hashlib
    h = hashlib.sha256()
    pkg = ROOT / "paper_2106_04718_amd"
    for p in [*sorted((pkg / "csrc").glob("*.hip")), pkg / "csrc" / "launch.h", pkg / "build.py"]:
        h.update(p.read_bytes())
    return h.hexdigest()[:16]


def cpu_baseline(cfg, base, g, out0, logits0, step_bytes, reps):
    """The oracle, as it is, on the host cores: the same step on the same
    inputs (K/V set 0).  Its outputs are also compared with the GPU's first step."""
    import numpy as np

    import oracle

    qd, Kd, Vd = (np.ascontiguousarray(oracle.widen(base[x])) for x in ("q", "K", "V"))
    tokens = np.ascontiguousarray(g["tokens"])
    cores = oracle.num_threads()
    times, t_attn, t_ng = [], [], []
    ref = None
    while True:
        lg = np.array(g["logits"], copy=True)
        t0 = time.perf_counter()
        ref = oracle.cross_attn_f64(qd, Kd, Vd, base["src_len"])
        t1 = time.perf_counter()
        oracle.ngram_block_inplace(tokens, cfg.n, lg, cfg.t)
        t2 = time.perf_counter()
        times.append(t2 - t0)
        t_attn.append(t1 - t0)
        t_ng.append(t2 - t1)
        if (reps and len(times) >= reps) or (not reps and (sum(times) > ORACLE_BUDGET_S or len(times) >= ORACLE_MAX_REPS)):
            break
    sec = float(np.median(times))
    # One more pass on a single thread, for the per-core figure.
    oracle.set_num_threads(1)
    try:
        lg1 = np.array(g["logits"], copy=True)
        s0 = time.perf_counter()
        oracle.cross_attn_f64(qd, Kd, Vd, base["src_len"])
        s1 = time.perf_counter()
        oracle.ngram_block_inplace(tokens, cfg.n, lg1, cfg.t)
        s2 = time.perf_counter()
    finally:
        oracle.set_num_threads(cores)
    err = float(np.max(np.abs(out0 - ref)))
    tol = 2e-2 if cfg.dtype == "bf16" else 1e-5 * float(np.max(np.abs(ref)))
    ng_ok = bool(np.array_equal(lg.view(np.uint32), logits0.view(np.uint32)))
    log(f"oracle: {sec * 1e3:.1f} ms per step on {cores} threads ({len(times)} reps); "
        f"attn max abs err {err:.3e} (tol {tol:.1e}); n-gram bit-exact {ng_ok}")
    cpu = {"value": round(step_bytes / sec / 1e9, 4), "unit": "GB/s", "cores": cores, "kind": "oracle",
           "sample": f"whole {cfg.name}-shaped step (all {cfg.B} sources x {cfg.k} beams x {cfg.H} heads, "
                     f"{cfg.rows} token rows), K/V set 0, median of {len(times)} reps, "
                     f"{sec * 1e3:.1f} ms per step",
           "attn_ms": round(float(np.median(t_attn)) * 1e3, 3), "ngram_ms": round(float(np.median(t_ng)) * 1e3, 3),
           "attn_ms_1thread": round((s1 - s0) * 1e3, 3), "ngram_ms_1thread": round((s2 - s1) * 1e3, 3)}
    parity = {"attn_max_abs_err": err, "attn_tol": tol, "attn_ok": err <= tol, "ngram_bitexact": ng_ok}
    return cpu, parity


if __name__ == "__main__":
    sys.exit(main())
