"""Benchmark of the cold exact full-vocabulary mask on one MI355X.

One step = the whole hot path over one batch of 32 configurations of the
read-only DML SQL workload (V = 151,936): prologue (allowed terminals, EOS
gate, first-shift summaries), class verdicts, the id-ordered mask stream, the
residue walk, row finalize, and the -inf fill of bf16 logits [32, V].  Steps
cycle through distinct, device-resident config batches; the mask cache is not
used (every step is a cold mask).

The throughput comes from K whole steps back to back with nothing recorded
between them; per-step latency (p50/p99 per mask) from a second pass with an
event pair around each step, and the phase split and the stream kernel's
launch time (roofline) from a third pass with events between the phases, all
on the launch stream.  Prints one JSON line: masks/s, p50/p99 microseconds per
mask, the stream kernel's roofline numbers, the CPU oracle's throughput on a
bounded sample of the same workload, and, beside the cold figure, the mask
cache's miss-and-insert and hit throughputs on the same batches.
"""

import argparse
import json
import os
import sys
import time
from pathlib import Path

import numpy as np

ROOT = Path(__file__).resolve().parent
sys.path.insert(0, str(ROOT))

HBM_PEAK_GBS = 8000.0
TRAFFIC_PROFILE = ROOT / "profiles" / "stream_kernel_traffic_dml_b32.md"
KERNEL_SOURCE = ROOT / "paper_2607_11951_amd" / "csrc" / "kernels.hip"


def stream_traffic_bytes():
    """HBM bytes per stream-kernel launch from the committed counter summary
    (FETCH_SIZE and WRITE_SIZE per dispatch, each scaled by its plain-copy
    calibration factor), or None when the kernels changed since it was taken."""
    import hashlib
    if not TRAFFIC_PROFILE.exists():
        return None
    kv = {}
    for line in TRAFFIC_PROFILE.read_text().splitlines():
        if line.startswith("- ") and ": " in line:
            k, v = line[2:].split(": ", 1)
            kv[k.strip()] = v.strip().strip("`")
    sha = hashlib.sha256(KERNEL_SOURCE.read_bytes()).hexdigest()
    try:
        if kv.get("kernels.hip sha256") != sha:
            return None
        fetch = float(kv["FETCH_SIZE KiB per stream dispatch"]) * float(kv["FETCH_SIZE copy factor"])
        write = float(kv["WRITE_SIZE KiB per stream dispatch"]) * float(kv["WRITE_SIZE copy factor"])
    except (KeyError, ValueError):
        return None
    return (fetch + write) * 1024.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--batches", type=int, default=8, help="distinct config batches cycled through")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="CPU oracle sample budget")
    ap.add_argument("--copy-calib", action="store_true",
                    help="also run a plain 1 GiB device copy (counter calibration runs)")
    ap.add_argument("--flatness", action="store_true",
                    help="instead: per-mask cost against position n and nesting depth on the "
                         "16,000-token workload (one JSON line)")
    return ap.parse_args()


def flatness(args):
    """Cost per mask at positions n = 1k / 4k / 16k tokens and nesting depths
    1 / 8 / 32 / 128 (32 configurations per cell, one batch each), and per depth
    the least-squares slope of the per-mask cost against n with a 95% interval
    (t quantile for the degrees of freedom); flat when |slope| x 15,000 stays
    under 5 % of the cost at n = 1,000."""
    import torch
    import paper_2607_11951_amd as G
    from workloads import make_workload
    from scipy import stats
    dev = torch.device("cuda:0")
    t0 = time.time()
    wl = make_workload(4)
    grid, slots = G.from_workload(wl)
    grid.to_device(dev)
    B = wl.batch
    print(f"16,000-token workload ready in {time.time() - t0:.0f}s", file=sys.stderr, flush=True)
    stream = torch.cuda.current_stream()
    ws = grid.new_workspace(B, dev)
    mask = torch.empty((B, grid.W), dtype=torch.int32, device=dev)
    eos = torch.empty(B, dtype=torch.uint8, device=dev)
    status = torch.empty(B, dtype=torch.int32, device=dev)
    cells, samples = [], {}
    for idx in wl.batches():
        n_pos, depth, _ = wl.meta["cells"][idx[0]]
        cfgs, pool = grid.configs([wl.prefixes[j] for j in idx], [slots[wl.slots[j]] for j in idx])
        c, p = grid.configs_to_device(cfgs, pool, dev)
        for _ in range(args.warmup):
            grid.mask(c, p, B, mask, eos, status, ws, stream)
        torch.cuda.synchronize()
        assert (status.cpu() == 0).all()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(args.steps)]
        for e0, e1 in evs:
            e0.record(stream)
            grid.mask(c, p, B, mask, eos, status, ws, stream)
            e1.record(stream)
        torch.cuda.synchronize()
        us = np.array([e0.elapsed_time(e1) * 1000.0 / B for e0, e1 in evs])
        samples[(n_pos, depth)] = us
        cells.append({"n": n_pos, "depth": depth, "us_per_mask_median": float(np.median(us)),
                      "us_per_mask_p99": float(np.percentile(us, 99)),
                      "max_stack_depth": int(cfgs["stk_depth"].max())})
        print(f"n={n_pos:6d} depth={depth:4d}: {np.median(us):.2f} us/mask "
              f"(stack <= {int(cfgs['stk_depth'].max())})", file=sys.stderr, flush=True)
    slopes = []
    for depth in sorted({d for _, d in samples}):
        xs, ys = [], []
        for (n_pos, d), us in samples.items():
            if d == depth:
                xs += [n_pos] * len(us)
                ys += list(us)
        fit = stats.linregress(xs, ys)
        dof = len(xs) - 2
        half = stats.t.ppf(0.975, dof) * fit.stderr
        base = float(np.median(samples[(1000, depth)]))
        slopes.append({"depth": depth, "slope_us_per_token": float(fit.slope),
                       "ci95": [float(fit.slope - half), float(fit.slope + half)],
                       "cost_at_1k_us": base, "change_over_15k_tokens_pct": float(100.0 * fit.slope * 15000 / base),
                       "flat": bool(abs(fit.slope) * 15000 < 0.05 * base)})
    print(json.dumps({"metric": "per-mask cost vs position n and nesting depth (flatness)",
                      "unit": "us/mask", "steps_per_cell": args.steps, "batch": B, "vocab": wl.V,
                      "workload": "read-only DML SQL, 16,000-token sentences, 32 configs per cell",
                      "cells": cells, "slopes": slopes}), flush=True)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}); "
              "rows are independent, so a multi-GPU run is batch sharding with no exchange and is "
              "not part of this build.", file=sys.stderr, flush=True)
        sys.exit(2)

    import torch
    import paper_2607_11951_amd as G
    from workloads import make_workload

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.flatness:
        flatness(args)
        return
    dev = torch.device("cuda:0")
    t0 = time.time()
    wl = make_workload(3, n_batches=args.batches)
    grid, slots = G.from_workload(wl)
    grid.to_device(dev)
    B = wl.batch
    batches = []
    for idx in wl.batches():
        cfgs, pool = grid.configs([wl.prefixes[j] for j in idx], [slots[wl.slots[j]] for j in idx])
        batches.append(grid.configs_to_device(cfgs, pool, dev))
    info = grid.info()
    mask = torch.empty((B, grid.W), dtype=torch.int32, device=dev)
    eos = torch.empty(B, dtype=torch.uint8, device=dev)
    status = torch.empty(B, dtype=torch.int32, device=dev)
    ws = grid.new_workspace(B, dev)
    gen = torch.Generator(device="cpu").manual_seed(3999)
    logits = (torch.randn(B, wl.V, generator=gen) * 2.0).to(torch.bfloat16).to(dev)
    print(f"setup {time.time() - t0:.1f}s: {info}", file=sys.stderr, flush=True)

    stream = torch.cuda.current_stream()

    def step(i):
        c, p = batches[i % len(batches)]
        grid.mask(c, p, B, mask, eos, status, ws, stream)
        G.apply(mask, logits, stream)

    def step_phases(i, ev):
        c, p = batches[i % len(batches)]
        ev[0].record(stream)
        for k, ph in enumerate((G.grid.PHASE_PROLOGUE, G.grid.PHASE_WALK, G.grid.PHASE_RESIDUE)):
            grid.mask(c, p, B, mask, eos, status, ws, stream, phases=ph)
            ev[k + 1].record(stream)
        grid.mask(c, p, B, mask, eos, status, ws, stream, phases=G.grid.PHASE_FINALIZE)
        G.apply(mask, logits, stream)
        ev[4].record(stream)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    st = status.cpu()
    assert (st == 0).all(), f"row status {st.tolist()}"

    # timed region: K whole steps back to back, nothing recorded between them
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start

    # per-step latency: the same K steps, an event pair around each (the
    # events themselves add a few microseconds per step)
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
             for _ in range(args.steps)]
    for i, (e0, e1) in enumerate(pairs):
        e0.record(stream)
        step(i)
        e1.record(stream)
    torch.cuda.synchronize()
    per_mask_us = np.array([e0.elapsed_time(e1) for e0, e1 in pairs]) * 1000.0 / B

    # phase times on the launch stream, events between the phases
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    for i in range(args.steps):
        step_phases(i, evs[i])
    torch.cuda.synchronize()
    pro_ms = np.array([e[0].elapsed_time(e[1]) for e in evs])
    walk_ms = np.array([e[1].elapsed_time(e[2]) for e in evs])
    res_ms = np.array([e[2].elapsed_time(e[3]) for e in evs])
    tail_ms = np.array([e[3].elapsed_time(e[4]) for e in evs])

    # device incremental advance beside the mask: every row takes one token its
    # mask allows (grid_accept), timed over the same batches
    acc_inputs = []
    for i in range(len(batches)):
        c, p = batches[i]
        grid.mask(c, p, B, mask, eos, status, ws, stream)
        torch.cuda.synchronize()
        bits = np.unpackbits(mask.cpu().numpy().view(np.uint8), axis=1, bitorder="little")[:, :wl.V]
        rng = np.random.default_rng(5000 + i)
        toks = []
        for r in range(B):
            allowed = np.flatnonzero(bits[r])
            allowed = allowed[allowed != wl.eos_id]
            toks.append(int(rng.choice(allowed)) if len(allowed) else wl.eos_id)
        acc_inputs.append(torch.tensor(toks, dtype=torch.int32, device=dev))
    acc_cap = 1024
    acc_out = (torch.empty(B * 32, dtype=torch.uint8, device=dev),
               torch.empty(B * acc_cap, dtype=torch.int16, device=dev),
               torch.empty(B, dtype=torch.int32, device=dev))
    for i in range(len(batches)):
        c, p = batches[i]
        grid.accept(c, p, acc_inputs[i], B, acc_cap, *acc_out, stream=stream)
    torch.cuda.synchronize()
    assert (acc_out[2].cpu() == 0).all()
    a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a0.record(stream)
    for i in range(args.steps):
        c, p = batches[i % len(batches)]
        grid.accept(c, p, acc_inputs[i % len(batches)], B, acc_cap, *acc_out, stream=stream)
    a1.record(stream)
    torch.cuda.synchronize()
    accept_us = a0.elapsed_time(a1) * 1000.0 / args.steps

    # algorithmic bytes of one stream launch per row: the class of every token
    # id for the row's lexer state (u16) and the row's W mask words; the
    # verdict table (2 bits per class) is not counted
    bytes_per_mask = 2 * wl.V + 4 * grid.W
    walk_s = float(walk_ms.mean()) / 1000.0
    achieved = B * bytes_per_mask / walk_s / 1e9

    # mask cache beside the cold figure: every row missing and inserting (the
    # cache cleared before each step), then every row hitting
    n_entries = 1
    while n_entries < 2 * B * len(batches):
        n_entries *= 2
    cache = grid.new_cache(n_entries, dev)
    cache_steps = max(10, args.steps // 4)

    def cached_step(i, clear):
        c, p = batches[i % len(batches)]
        if clear:
            grid.clear_cache(cache, stream)
        grid.mask(c, p, B, mask, eos, status, ws, stream, cache=cache)
        G.apply(mask, logits, stream)

    cache_out = {"entries": n_entries}
    for label, clear in (("miss_insert", True), ("hit", False)):
        for i in range(len(batches)):
            cached_step(i, clear)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for i in range(cache_steps):
            cached_step(i, clear)
        e1.record(stream)
        torch.cuda.synchronize()
        cache_out[f"{label}_masks_per_s"] = B * cache_steps / (e0.elapsed_time(e1) / 1000.0)
    assert (status.cpu() == 0).all()

    if args.copy_calib:
        a = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()

    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        if not oracle.LIB.exists():
            oracle.build()
        o = oracle.from_workload(wl)
        threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
        threads = max(1, min(threads, os.cpu_count() or 1))
        n = 0
        t1 = time.perf_counter()
        while time.perf_counter() - t1 < args.cpu_seconds:  # rows cycled until the budget is spent
            o.mask(wl.prefixes[n % len(wl.prefixes)], mode=1, nthreads=threads)
            n += 1
        dt = time.perf_counter() - t1
        cpu = {"value": n / dt, "unit": "masks/s", "cores": threads, "kind": "oracle",
               "sample": f"{n} full-vocabulary masks (V={wl.V}) over the {len(wl.prefixes)} rows of "
                         f"the read-only DML workload, cycled; oracle checkpoint mode (prefix parsed "
                         f"once per row, pending lexeme + token re-lexed per token), {dt:.1f}s"}

    out = {
        "metric": "cold next-token masks/s at B=32, V=151,936; p50/p99 us per mask",
        "value": B * args.steps / wall,
        "unit": "masks/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall * 1000.0 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32",
        "data": "synthetic",
        "config": {"workload": "read-only DML SQL (183-production grammar, 200x30 schema lexicon), "
                               "B=32 rows per step, V=151936 byte-level vocabulary, "
                               f"{len(batches)} distinct config batches cycled, cache off, "
                               "+ bf16 -inf apply [32, 151936]",
                   "global_batch": B, "vocab": wl.V, "parallelism": "none (1 GPU)"},
        "p50_us_per_mask": float(np.percentile(per_mask_us, 50)),
        "p99_us_per_mask": float(np.percentile(per_mask_us, 99)),
        "phase_ms": {"prologue+verdicts": float(pro_ms.mean()), "stream": float(walk_ms.mean()),
                     "residue": float(res_ms.mean()), "finalize+apply": float(tail_ms.mean()),
                     "note": "separate pass, an event between phases"},
        "roofline": {"bound": "hbm", "kernel": "stream_kernel", "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": stream_traffic_bytes(), "bytes_per_mask": bytes_per_mask,
                     "stream_us_per_launch": walk_s * 1e6},
        "cpu_baseline": cpu,
        "cache": cache_out,
        "accept": {"us_per_step": accept_us, "rows": B,
                   "note": "grid_accept of one allowed token per row, back to back over the same batches"},
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
