"""Benchmark of the cold exact full-vocabulary mask on one MI355X.

One step = the whole hot path over one batch of 32 configurations of the
read-only DML SQL workload (V = 151,936): prologue (allowed terminals, EOS
gate, first-shift summaries), class verdicts, the id-ordered mask stream, the
residue walk, row finalize, and the -inf fill of bf16 logits [32, V].  Steps
cycle through distinct, device-resident config batches; the mask cache is not
used (every step is a cold mask).

The throughput comes from K whole steps back to back with nothing recorded
between them; the per-step latency from a second pass with an event pair
around each step (p50/p99 per mask are that step latency divided by B, i.e.
amortized over the batch); the phase split from a third pass with events
between the launches, all on the launch stream.  The roofline is the whole
mask call's: the algorithmic bytes of B masks over the summed mask-phase
time, with each phase's own figure beside it.

Beside the headline line: the 256-schema workload (B = 256, one lexicon per
row) with its fused bf16 apply in GB/s, the small workloads' throughputs, the
device incremental advance, the mask cache, and the CPU oracle (multi-thread
and single-thread, checkpoint and from-scratch modes, per workload) on
bounded samples.  Prints one JSON line.
"""

import argparse
import hashlib
import json
import os
import platform
import sys
import time
from pathlib import Path

import numpy as np

ROOT = Path(__file__).resolve().parent
sys.path.insert(0, str(ROOT))

HBM_PEAK_GBS = 8000.0
TRAFFIC_PROFILE = ROOT / "profiles" / "mask_traffic_dml_b32.md"
KERNEL_SOURCE = ROOT / "paper_2607_11951_amd" / "csrc" / "kernels.hip"
MASK_KERNELS = ("prologue_kernel", "verdict_kernel", "stream_kernel", "residue_kernel", "finalize_kernel")


def mask_traffic_bytes():
    """HBM bytes of one grid_mask call at B = 32 from the committed counter
    summary (FETCH_SIZE and WRITE_SIZE per dispatch of each mask kernel, each
    scaled by its plain-copy calibration factor), or None when the kernels
    changed since the counters were taken."""
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
        ff, wf = float(kv["FETCH_SIZE copy factor"]), float(kv["WRITE_SIZE copy factor"])
        total = 0.0
        for k in MASK_KERNELS:
            total += float(kv[f"{k} FETCH_SIZE KiB"]) * ff + float(kv[f"{k} WRITE_SIZE KiB"]) * wf
    except (KeyError, ValueError):
        return None
    return total * 1024.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--batches", type=int, default=8, help="distinct config batches cycled through")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true",
                    help="only the headline workload (no 256-schema, small-workload, cache or advance figures)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0, help="CPU oracle budget of the main sample")
    ap.add_argument("--copy-calib", action="store_true",
                    help="also run a plain 1 GiB device copy (counter calibration runs)")
    ap.add_argument("--flatness", action="store_true",
                    help="instead: per-mask cost against position n and nesting depth on the "
                         "16,000-token workload (one JSON line)")
    return ap.parse_args()


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def flatness_one(args, k):
    """Cost per mask at positions n = 1k / 4k / 16k tokens and nesting depths
    1 / 8 / 32 / 128 (32 configurations per cell, one batch each) on workload
    k, and per depth the least-squares slope of the per-mask cost against n
    with a 95% interval (t quantile for the degrees of freedom); flat when
    |slope| x 15,000 stays under 5 % of the cost at n = 1,000."""
    import torch
    import paper_2607_11951_amd as G
    from workloads import make_workload
    from scipy import stats
    dev = torch.device("cuda:0")
    t0 = time.time()
    wl = make_workload(k)
    grid, slots = G.from_workload(wl)
    grid.to_device(dev)
    B = wl.batch
    log(f"workload {wl.name} ready in {time.time() - t0:.0f}s")
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
        toks = [wl.meta["cells"][j][2] for j in idx]
        cells.append({"n": n_pos, "depth": depth, "us_per_mask_median": float(np.median(us)),
                      "us_per_mask_p99": float(np.percentile(us, 99)),
                      "tokens_min": int(min(toks)), "tokens_max": int(max(toks)),
                      "max_stack_depth": int(cfgs["stk_depth"].max())})
        log(f"{wl.name} n={n_pos:6d} depth={depth:4d}: {np.median(us):.2f} us/mask "
            f"(stack <= {int(cfgs['stk_depth'].max())})")
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
    return {"workload": wl.name, "vocab": wl.V, "batch": B, "cells": cells, "slopes": slopes}


def flatness(args):
    """Flatness on the 16,000-token workload (every configuration its own
    content) and on its position-isolated variant (the same local contexts
    at the three positions, so a slope there is position alone); one JSON
    line."""
    out = {"metric": "per-mask cost vs position n and nesting depth (flatness)", "unit": "us/mask",
           "steps_per_cell": args.steps,
           "content_varies": flatness_one(args, 4),
           "position_isolated": flatness_one(args, 6)}
    print(json.dumps(out), flush=True)


def device_batches(G, grid, wl, slots, dev):
    out, depths = [], []
    for idx in wl.batches():
        cfgs, pool = grid.configs([wl.prefixes[j] for j in idx], [slots[wl.slots[j]] for j in idx])
        out.append(grid.configs_to_device(cfgs, pool, dev))
        depths.append(cfgs["stk_depth"].astype(np.int64))
    return out, depths


def mask_bytes(V, W, depths):
    """Algorithmic bytes of the masks of one batch: per row the class of every
    token id for the row's lexer state (u16), its W mask words, its stack
    (u16 per entry) and its 32-byte configuration record."""
    return int(len(depths) * (2 * V + 4 * W + 32) + 2 * int(np.sum(depths)))


def timed_steps(torch, stream, step, n):
    """Wall time of n steps back to back (nothing recorded between them)."""
    torch.cuda.synchronize()
    t = time.perf_counter()
    for i in range(n):
        step(i)
    torch.cuda.synchronize()
    return time.perf_counter() - t


def small_workload(torch, G, k, dev, steps, warmup):
    """Throughput and per-call latency of workload k (1: V = 1,024, one row per
    call; 2: V = 32,000, B = 32), cache off."""
    from workloads import make_workload
    wl = make_workload(k, n_batches=4) if k == 2 else make_workload(k)
    grid, slots = G.from_workload(wl)
    grid.to_device(dev)
    batches, _ = device_batches(G, grid, wl, slots, dev)
    B = wl.batch
    stream = torch.cuda.current_stream()
    mask = torch.empty((B, grid.W), dtype=torch.int32, device=dev)
    eos = torch.empty(B, dtype=torch.uint8, device=dev)
    status = torch.empty(B, dtype=torch.int32, device=dev)
    ws = grid.new_workspace(B, dev)

    def step(i):
        c, p = batches[i % len(batches)]
        grid.mask(c, p, B, mask, eos, status, ws, stream)

    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    assert (status.cpu() == 0).all()
    wall = timed_steps(torch, stream, step, steps)
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for i, (e0, e1) in enumerate(pairs):
        e0.record(stream)
        step(i)
        e1.record(stream)
    torch.cuda.synchronize()
    call_us = np.array([e0.elapsed_time(e1) * 1000.0 for e0, e1 in pairs])
    return {"workload": wl.name, "vocab": wl.V, "batch": B, "masks_per_s": B * steps / wall,
            "p50_call_us": float(np.percentile(call_us, 50)), "p99_call_us": float(np.percentile(call_us, 99))}


def cold_schema(torch, G, dev, steps, warmup):
    """The 256-schema workload: B = 256 rows, each on its own freshly compiled
    schema lexicon, cache off, each mask followed by the fused -inf fill of
    bf16 logits [256, 151,936] ~ N(0, 4); the apply's own time and GB/s."""
    from workloads import make_workload, grammar_text
    t0 = time.time()
    wl = make_workload(5)
    grid = G.Grid(grammar_text(wl.grammar), wl.drop, wl.vocab, wl.specials, wl.eos_id)
    t1 = time.perf_counter()
    slots = [grid.add_lexicon(lex) for lex in wl.lexicons]
    lex_ms = (time.perf_counter() - t1) * 1000.0 / len(wl.lexicons)
    grid.to_device(dev)
    batches, depths = device_batches(G, grid, wl, slots, dev)
    c, p = batches[0]
    B = wl.batch
    log(f"256-schema workload ready in {time.time() - t0:.0f}s")
    stream = torch.cuda.current_stream()
    mask = torch.empty((B, grid.W), dtype=torch.int32, device=dev)
    eos = torch.empty(B, dtype=torch.uint8, device=dev)
    status = torch.empty(B, dtype=torch.int32, device=dev)
    ws = grid.new_workspace(B, dev)
    gen = torch.Generator(device="cpu").manual_seed(wl.meta["logits_seed"])
    base = (torch.randn(B, wl.V, generator=gen) * wl.meta["logits_std"]).to(torch.bfloat16).to(dev)
    logits = base.clone()
    for _ in range(warmup):
        grid.mask(c, p, B, mask, eos, status, ws, stream)
        G.apply(mask, logits, stream)
    torch.cuda.synchronize()
    assert (status.cpu() == 0).all()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    for i in range(steps):
        logits.copy_(base)  # every apply masks fresh logits (outside the timed events)
        evs[i][0].record(stream)
        grid.mask(c, p, B, mask, eos, status, ws, stream)
        evs[i][1].record(stream)
        G.apply(mask, logits, stream)
        evs[i][2].record(stream)
    torch.cuda.synchronize()
    mask_ms = np.array([e[0].elapsed_time(e[1]) for e in evs])
    apply_ms = np.array([e[1].elapsed_time(e[2]) for e in evs])
    bits = np.unpackbits(mask.cpu().numpy().view(np.uint8), axis=1, bitorder="little")[:, :wl.V]
    disallowed = int(bits.size - bits.sum())
    apply_bytes = B * 4 * grid.W + 2 * disallowed
    apply_gbs = apply_bytes / (float(np.median(apply_ms)) / 1000.0) / 1e9
    mb = mask_bytes(wl.V, grid.W, depths[0])
    mask_gbs = mb / (float(np.median(mask_ms)) / 1000.0) / 1e9
    return {"workload": "read-only DML SQL, 256 fresh schemas (50..500 tables x 5..60 columns), one per row, "
                        "B=256, V=151936, cache off, + bf16 -inf apply [256, 151936]",
            "masks_per_s": B / (float(np.median(mask_ms + apply_ms)) / 1000.0),
            "mask_ms_median": float(np.median(mask_ms)), "apply_ms_median": float(np.median(apply_ms)),
            "mask_roofline": {"achieved_gbs": mask_gbs, "frac": mask_gbs / HBM_PEAK_GBS, "bytes": mb},
            "apply_roofline": {"bound": "hbm", "achieved_gbs": apply_gbs, "peak_gbs": HBM_PEAK_GBS,
                               "frac": apply_gbs / HBM_PEAK_GBS, "bytes": apply_bytes,
                               "note": "mask words read + one bf16 store per disallowed logit"},
            "add_lexicon_ms_per_schema": lex_ms}


def warm_decode(torch, G, grid, wl, slots, dev, n_steps):
    """Decode loops over the headline batches: each row's stack in its own
    region of a pool, every step the row's mask, the bf16 -inf fill and an
    in-place advance by a token its mask allows (grid_accept_inplace, rolling
    hashes kept).  The token trajectories are drawn once from the masks
    (untimed), then replayed from the same starting configurations three
    ways: cold masks (grid_mask), warm masks with an empty cache of
    context-independent words at the start of the replay, and warm masks
    with the cache the previous replay left (steady state).  Rows served by
    cached words = rows - entries published."""
    B, cap = wl.batch, 1024
    stride = 96 + (4 * grid.W + 15) // 16 * 16
    starts = []
    for idx in wl.batches():
        cfgs, pool = grid.configs([wl.prefixes[j] for j in idx], [slots[wl.slots[j]] for j in idx])
        region = np.zeros(B * cap, dtype=np.uint16)
        for b in range(B):
            off, d = int(cfgs["stk_off"][b]), int(cfgs["stk_depth"][b])
            region[b * cap:b * cap + d] = pool[off:off + d]
            cfgs["stk_off"][b] = b * cap
        starts.append(grid.configs_to_device(cfgs, region, dev))
    stream = torch.cuda.current_stream()
    c = torch.empty_like(starts[0][0])
    p = torch.empty_like(starts[0][1])
    h = torch.zeros(B * cap, dtype=torch.int64, device=dev)
    mask = torch.empty((B, grid.W), dtype=torch.int32, device=dev)
    eos = torch.empty(B, dtype=torch.uint8, device=dev)
    status = torch.empty(B, dtype=torch.int32, device=dev)
    acc_st = torch.empty(B, dtype=torch.int32, device=dev)
    ws = grid.new_workspace(B, dev)
    logits = torch.zeros((B, wl.V), dtype=torch.bfloat16, device=dev)
    rng = np.random.default_rng(6100)
    traj = []
    for c0, p0 in starts:  # token trajectories from the exact masks
        c.copy_(c0)
        p.copy_(p0)
        toks = []
        for _ in range(n_steps):
            grid.mask(c, p, B, mask, eos, status, ws, stream)
            torch.cuda.synchronize()
            bits = np.unpackbits(mask.cpu().numpy().view(np.uint8), axis=1, bitorder="little")[:, :wl.V]
            t = []
            for r in range(B):
                allowed = np.flatnonzero(bits[r])
                allowed = allowed[allowed != wl.eos_id]
                t.append(int(rng.choice(allowed)) if len(allowed) else wl.eos_id)
            tt = torch.tensor(t, dtype=torch.int32, device=dev)
            toks.append(tt)
            grid.accept_inplace(c, p, tt, B, cap, status=acc_st, stream=stream)
        traj.append(toks)
    cache = grid.new_ci_cache(8192, dev)
    flags = G.grid.CI_LOOKUP | G.grid.CI_INSERT

    def published():
        st = cache.view(-1, stride)[:, :4].contiguous().view(torch.int32)[:, 0]
        return int((st == 2).sum().item())

    def replay(kind):
        total = 0.0
        for bi, (c0, p0) in enumerate(starts):
            c.copy_(c0)
            p.copy_(p0)
            grid.stack_hash(c, p, B, out=h, stream=stream)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for tt in traj[bi]:
                if kind == "cold":
                    grid.mask(c, p, B, mask, eos, status, ws, stream)
                else:
                    grid.mask_warm(c, p, B, cache, flags, mask, eos, status, ws, stream)
                G.apply(mask, logits, stream)
                grid.accept_inplace(c, p, tt, B, cap, stack_hash=h, status=acc_st, stream=stream)
            e1.record(stream)
            torch.cuda.synchronize()
            assert (status.cpu() == 0).all() and (acc_st.cpu() == 0).all()
            total += e0.elapsed_time(e1) / 1000.0
        return total

    rows = B * n_steps * len(starts)
    replay("cold")
    t_cold = replay("cold")
    grid.clear_ci_cache(cache, stream)
    n0 = published()
    t_first = replay("warm")
    n1 = published()
    t_steady = replay("warm")
    n2 = published()
    # the in-place advance alone, same trajectories
    t_acc = 0.0
    for bi, (c0, p0) in enumerate(starts):
        c.copy_(c0)
        p.copy_(p0)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for tt in traj[bi]:
            grid.accept_inplace(c, p, tt, B, cap, stack_hash=h, status=acc_st, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        t_acc += e0.elapsed_time(e1) / 1000.0
    return {"workload": f"read-only DML SQL, {len(starts)} batches x B={B} rows x {n_steps} decode steps, "
                        "tokens sampled from the exact masks, replayed",
            "cold_masks_per_s": rows / t_cold, "cold_step_us": t_cold * 1e6 / (n_steps * len(starts)),
            "warm_first_pass_masks_per_s": rows / t_first, "warm_first_pass_rows_cached": 1.0 - (n1 - n0) / rows,
            "warm_steady_masks_per_s": rows / t_steady, "warm_steady_rows_cached": 1.0 - (n2 - n1) / rows,
            "warm_steady_step_us": t_steady * 1e6 / (n_steps * len(starts)),
            "accept_inplace_step_us": t_acc * 1e6 / (n_steps * len(starts)),
            "note": "each step = mask (+ warm cache) + bf16 -inf fill [B, V] + in-place advance with rolling "
                    "hashes; rows cached = 1 - entries published / rows"}


def completion_cost(G, grid, wl, slots, n_rows):
    """Host cost of the mode-1 reserve: grid_complete on rows of the workload."""
    lens, t = [], time.perf_counter()
    for j in range(n_rows):
        lens.append(len(grid.complete(wl.prefixes[j], slots[wl.slots[j]])))
    dt = time.perf_counter() - t
    return {"rows": n_rows, "ms_per_completion": dt * 1000.0 / n_rows,
            "reserve_tokens_median": float(np.median(lens)), "reserve_tokens_max": int(max(lens))}


def cpu_baselines(wl_main, seconds):
    """The oracle on the host cores: checkpoint mode with every thread (the
    reported value) and with one thread, from-scratch mode (every token
    re-lexes and re-parses the whole extended prefix) on a token sample, and
    checkpoint mode on the other workloads."""
    import oracle
    from workloads import make_workload
    if not oracle.LIB.exists():
        oracle.build()
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    threads = max(1, min(threads, os.cpu_count() or 1))

    def run(o, wl, budget, nthreads, mode=1, tokens=None):
        n = 0
        t1 = time.perf_counter()
        while time.perf_counter() - t1 < budget:  # rows cycled until the budget is spent
            lexicon = None
            o.mask(wl.prefixes[n % len(wl.prefixes)], mode=mode, nthreads=nthreads, tokens=tokens, lexicon=lexicon)
            n += 1
        return n, time.perf_counter() - t1

    o = oracle.from_workload(wl_main)
    n, dt = run(o, wl_main, seconds, threads)
    n1, dt1 = run(o, wl_main, seconds / 2, 1)
    toks = np.random.default_rng(77).choice(wl_main.V, 2000, replace=False).astype(np.int32)
    n0, dt0 = run(o, wl_main, seconds / 2, threads, mode=0, tokens=toks)
    cpu_model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                cpu_model = line.split(":", 1)[1].strip()
                break
    except OSError:
        cpu_model = platform.processor()
    out = {"value": n / dt, "unit": "masks/s", "cores": threads, "kind": "oracle",
           "sample": f"{n} full-vocabulary masks (V={wl_main.V}) over the {len(wl_main.prefixes)} rows of the "
                     f"read-only DML workload, cycled; oracle checkpoint mode (prefix parsed once per row, "
                     f"pending lexeme + token re-lexed per token), {threads} threads, {dt:.1f}s",
           "host_cpu": cpu_model, "host_threads_available": os.cpu_count(),
           "single_thread_masks_per_s": n1 / dt1,
           "from_scratch_masks_per_s": (n0 / dt0) * len(toks) / wl_main.V,
           "from_scratch_note": f"from-scratch mode on {len(toks)} seeded token ids per row ({n0} rows, "
                                f"{dt0:.1f}s, {threads} threads), scaled to a full-vocabulary mask",
           "per_workload": {}}
    for k in (1, 2):
        wl = make_workload(k, n_batches=2) if k == 2 else make_workload(k)
        ok = oracle.from_workload(wl)
        nk, dtk = run(ok, wl, 2.0, threads)
        out["per_workload"][wl.name] = {"masks_per_s": nk / dtk, "mode": "checkpoint", "threads": threads}
    return out


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
    batches, depths = device_batches(G, grid, wl, slots, dev)
    info = grid.info()
    mask = torch.empty((B, grid.W), dtype=torch.int32, device=dev)
    eos = torch.empty(B, dtype=torch.uint8, device=dev)
    status = torch.empty(B, dtype=torch.int32, device=dev)
    ws = grid.new_workspace(B, dev)
    gen = torch.Generator(device="cpu").manual_seed(3999)
    logits = (torch.randn(B, wl.V, generator=gen) * 2.0).to(torch.bfloat16).to(dev)
    log(f"setup {time.time() - t0:.1f}s: {info}")

    stream = torch.cuda.current_stream()

    def step(i):
        c, p = batches[i % len(batches)]
        grid.mask(c, p, B, mask, eos, status, ws, stream)
        G.apply(mask, logits, stream)

    phases = (G.grid.PHASE_PROLOGUE, G.grid.PHASE_WALK, G.grid.PHASE_RESIDUE, G.grid.PHASE_FINALIZE)

    def step_phases(i, ev):
        c, p = batches[i % len(batches)]
        ev[0].record(stream)
        for k, ph in enumerate(phases):
            grid.mask(c, p, B, mask, eos, status, ws, stream, phases=ph)
            ev[k + 1].record(stream)
        G.apply(mask, logits, stream)
        ev[5].record(stream)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    st = status.cpu()
    assert (st == 0).all(), f"row status {st.tolist()}"

    # timed region: K whole steps back to back, nothing recorded between them
    wall = timed_steps(torch, stream, step, args.steps)
    log(f"timed region: {args.steps} steps in {wall * 1000:.1f} ms")

    # per-step latency: the same K steps, an event pair around each (the
    # events themselves add a few microseconds per step)
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
             for _ in range(args.steps)]
    for i, (e0, e1) in enumerate(pairs):
        e0.record(stream)
        step(i)
        e1.record(stream)
    torch.cuda.synchronize()
    step_us = np.array([e0.elapsed_time(e1) for e0, e1 in pairs]) * 1000.0

    # phase times on the launch stream, events between the launches
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(args.steps)]
    for i in range(args.steps):
        step_phases(i, evs[i])
    torch.cuda.synchronize()
    ph_ms = np.array([[e[k].elapsed_time(e[k + 1]) for k in range(5)] for e in evs])  # [steps, 5]
    ph_mean_s = ph_ms.mean(axis=0) / 1000.0
    mask_s = float(ph_mean_s[:4].sum())

    # roofline of the whole mask call: the algorithmic bytes of the B masks
    # of a step (mean over the batches cycled) over the summed phase time;
    # each phase's own time and, for the stream, its own bytes
    bytes_step = float(np.mean([mask_bytes(wl.V, grid.W, d) for d in depths]))
    achieved = bytes_step / mask_s / 1e9
    stream_bytes = B * (2 * wl.V + 4 * grid.W)
    per_phase = {
        "prologue+verdicts": {"us": ph_mean_s[0] * 1e6},
        "stream": {"us": ph_mean_s[1] * 1e6, "bytes": stream_bytes,
                   "achieved_gbs": stream_bytes / ph_mean_s[1] / 1e9,
                   "frac": stream_bytes / ph_mean_s[1] / 1e9 / HBM_PEAK_GBS},
        "residue": {"us": ph_mean_s[2] * 1e6},
        "finalize": {"us": ph_mean_s[3] * 1e6},
        "apply": {"us": ph_mean_s[4] * 1e6},
    }
    dominant = max(("prologue+verdicts", "stream", "residue", "finalize"), key=lambda k: per_phase[k]["us"])

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
        "p50_us_per_mask": float(np.percentile(step_us, 50)) / B,
        "p99_us_per_mask": float(np.percentile(step_us, 99)) / B,
        "per_mask_note": "amortized: per-step latency (event pair around each step) divided by B",
        "p50_step_us": float(np.percentile(step_us, 50)),
        "p99_step_us": float(np.percentile(step_us, 99)),
        "phase_us": {k: v["us"] for k, v in per_phase.items()},
        "roofline": {"bound": "hbm", "kernel": "grid_mask (prologue, verdict, stream, residue, finalize kernels)",
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": mask_traffic_bytes(), "bytes_per_launch": bytes_step,
                     "mask_us_per_launch": mask_s * 1e6, "dominant_phase": dominant,
                     "per_phase": per_phase,
                     "note": "bytes = B x (2V class map + 4W mask words + 32 config) + 2 x stack entries; "
                             "time = summed phase times of one grid_mask call on the launch stream"},
    }

    extra = {}
    if not args.no_extra:
        # device incremental advance beside the mask: every row takes one token
        # its mask allows (grid_accept), timed over the same batches
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
        extra["accept"] = {"us_per_step": a0.elapsed_time(a1) * 1000.0 / args.steps, "rows": B,
                           "note": "grid_accept of one allowed token per row, back to back over the same batches"}

        # mask cache beside the cold figure: every row missing and inserting
        # (the cache cleared before each step), then every row hitting
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
        extra["cache"] = cache_out
        extra["decode"] = warm_decode(torch, G, grid, wl, slots, dev, 16)
        extra["completion"] = completion_cost(G, grid, wl, slots, 64)
        extra["cold_schema"] = cold_schema(torch, G, dev, max(20, args.steps // 4), 3)
        extra["small_workloads"] = [small_workload(torch, G, 2, dev, args.steps, args.warmup),
                                    small_workload(torch, G, 1, dev, args.steps, args.warmup)]

    if args.copy_calib:
        a = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()

    out["cpu_baseline"] = None if args.no_cpu_baseline else cpu_baselines(wl, args.cpu_seconds)
    out.update(extra)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
