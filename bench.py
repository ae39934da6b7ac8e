#!/usr/bin/env python3
"""Decode-step benchmark of the dynamic sparse mixed-precision FFN stack.

One step = one decode token through every FFN layer of the stack: for each
layer, predictor scores -> top-k and tiers -> cache plan -> cache fill from
the pinned host store -> gather-dequant sparse FFN, all through the C ABI.
The default workload is the 70B-shaped stack (80 layers, d 8192, d_ff 28672,
k 2867 with tiers 286/860/1721, C = k), the configuration the roofline target
is quoted on.

Streams (paper_2410_14740_amd.pipeline): predict + plan on an aux stream,
fills on a copy stream, the FFN on the main stream; layer l's predict may
start once the FFN of layer l-2 is done, so the fill of layer l overlaps the
FFN of layer l-1 (Sec. 1: asynchronous loading overlapped with computation;
Sec. 6.1: dedicated streams).

Prints one JSON line (the benchmark contract), including the HBM roofline of
the sparse FFN on the workload's layer shape and the oracle timed on the host
cores at one thread and at every core this process may use.
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import json
import os
import sys
import time

import numpy as np
from fractions import Fraction as F

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "sparse MP-FFN µs/layer-step + tokens/s; achieved HBM GB/s vs MI355X peak"
PEAK_HBM_GBPS = 8000.0  # MI355X HBM3E, vendor figure
PEAK_HOST_LINK_GBPS = 64.0  # PCIe Gen5 x16, one direction, before protocol overhead


def parse_args():
    p = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=120, help="timed decode steps")
    p.add_argument("--warmup", type=int, default=8, help="untimed decode steps first")
    p.add_argument("--workload", default="llama2-70b")
    p.add_argument("--weight-sets", type=int, default=-1,
                   help="draw only this many distinct weight sets and let layers share their "
                        "pinned neuron stores (0 = every layer its own weights; -1 = 8 for the "
                        "70B stack, whose 80 stores would take 199 GB of pinned host memory, "
                        "else 0). Every layer keeps its own predictor, inputs and slot cache.")
    p.add_argument("--policy", choices=("exact", "dominance"), default="dominance",
                   help="cache hits: a resident tier at or above the requested one (default; "
                        "with the per-tier arena, a neuron missing from its tier's pool is served "
                        "by the lowest higher-precision pool that holds it) or the exact tier")
    p.add_argument("--arena", choices=("pools", "single"), default="pools",
                   help="pools (default): the HBM of the workload's C FP16-sized slots split into "
                        "one pool per tier, each the same multiple of its tier's per-step demand; "
                        "single: C FP16-sized slots shared by every tier")
    p.add_argument("--no-variants", action="store_true",
                   help="skip the other policy and arena stacks (per-tier arena with the other "
                        "policy, single arena with exact-tier and dominance hits) reported beside "
                        "the headline")
    p.add_argument("--policy-sweep", action="store_true",
                   help="only the cache-policy measurement: hit rates of exact-tier and "
                        "dominance hits, LRU at C = 30%% and at C = k (the ATU regime), against "
                        "the AR(1) correlation rho of the inputs, plus the 7B stack's tokens/s "
                        "under both policies")
    p.add_argument("--cpu-seconds", type=float, default=15.0,
                   help="target CPU time of the oracle baseline sample (0 = skip)")
    p.add_argument("--layers", type=int, default=0, help="override the layer count (0 = workload's)")
    p.add_argument("--ffn-layers", type=int, default=8,
                   help="layers cycled by the isolated sparse-FFN measurement on the workload's "
                        "layer shape (their active records exceed the 256 MB Infinity Cache)")
    p.add_argument("--ffn-reps", type=int, default=10, help="passes over those layers")
    p.add_argument("--extra-workload", default="llama2-7b",
                   help="second isolated sparse-FFN measurement on this layer shape ('' = skip)")
    p.add_argument("--extra-layers", type=int, default=16)
    p.add_argument("--overlap-steps", type=int, default=4,
                   help="untimed steps after the timed ones with events around every stage, "
                        "to measure how much of the fill time overlaps compute")
    p.add_argument("--stage-events", action="store_true",
                   help="record HIP events around every fill and FFN of the timed steps (their "
                        "markers add latency to the cross-stream waits; off for the headline)")
    p.add_argument("--deterministic-ffn", action="store_true",
                   help="use the three-kernel sparse FFN whose output repeats bit for bit")
    p.add_argument("--only-ffn", default="", metavar="WORKLOAD",
                   help="run only the isolated sparse-FFN measurement on this layer shape "
                        "(for profiling)")
    p.add_argument("--only-predict", default="", metavar="WORKLOAD",
                   help="run only the isolated predictor + top-k measurement on this layer shape")
    p.add_argument("--fill-sweep", action="store_true",
                   help="only the host-to-HBM transfer sweep: gather kernel vs per-record "
                        "hipMemcpyAsync vs one bulk copy, against the number of records")
    p.add_argument("--ssd-tier", action="store_true",
                   help="only the SSD -> DRAM tier measurement on the 7B-shaped stack")
    p.add_argument("--ssd-dir", default=os.environ.get("TMPDIR", "/tmp"),
                   help="directory of the layer store file")
    p.add_argument("--ssd-sets", type=int, default=4)
    p.add_argument("--ssd-fixed", type=int, default=4)
    p.add_argument("--ssd-slots", type=int, default=8)
    p.add_argument("--ssd-lookahead", type=int, default=2)
    p.add_argument("--ratio-search", action="store_true",
                   help="only the offline neuron-ratio search (Algorithm 1) on the 7B-shaped layer")
    p.add_argument("--batch-sweep", action="store_true",
                   help="only the batched-decode workload (7B-shaped layer, batch 8): LRU capacity "
                        "10/30/60%% x tiers 10/40/50 or all FP16, one JSON line")
    p.add_argument("--sweep-point", default="", metavar="CAP:MIX",
                   help="with --batch-sweep: only this point, e.g. 0.3:10/40/50 or 0.1:fp16 (for "
                        "counter runs that need one configuration)")
    p.add_argument("--calibrate-copy", type=int, default=0, metavar="MB",
                   help="only copy a buffer of this many MB device to device, 5 times "
                        "(a plain copy kernel of known size, to scale HBM counters)")
    return p.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def build_stack(wl, n_layers, steps_total, weight_sets, torch, m2c, W, flags=0, tier_slots=None):
    """Create every layer (weights drawn in a thread pool, layers created in
    order) and stage every layer's decode inputs on the device."""
    k, n16, n8 = wl.counts()
    C = wl.cache_slots()
    B = wl.batch
    desc = m2c.make_desc(wl.d_model, wl.d_ff, wl.pred_rank, k, C, max_batch=B, flags=flags,
                         tier_slots=tier_slots)
    x_dev = torch.empty((n_layers, steps_total, B, wl.d_model), dtype=torch.float16, device="cuda")
    layers, first = [], None

    def draw(l):
        wsrc = None if weight_sets <= 0 else l % weight_sets
        return W.workload_layer(wl, l, steps=steps_total, weight_layer=wsrc,
                                draw_weights=weight_sets <= 0 or l < weight_sets)

    keep = None
    with cf.ThreadPoolExecutor(4) as ex:
        futs = [ex.submit(draw, l) for l in range(n_layers)]
        for l, fu in enumerate(futs):
            ld = fu.result()
            futs[l] = None
            x_dev[l].copy_(torch.from_numpy(ld.x[:, :B].view(np.uint16)).view(torch.float16))
            owner = None
            if weight_sets > 0 and l >= weight_sets:
                owner = layers[l % weight_sets]
            layers.append(m2c.Layer(desc, ld, weights_of=owner))
            if l == 0:
                keep = ld
            if l % 8 == 7 or l == n_layers - 1:
                log(f"created {l + 1}/{n_layers} layers")
    return layers, x_dev, keep


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(wl, ld, n_layers, budget_s, oracle, policy, tier_slots=None):
    """The oracle on a bounded sample of the same work: layer 0 of the stack,
    consecutive decode steps of predict + select + LRU plan + fp64 sparse FFN
    until about `budget_s` seconds have run, timed twice: at one thread (the
    paper's one-core setting) and at every core this process may use (OpenMP
    over independent sums; the results are the same bits). Building the
    records of the neurons the sample touches is set-up, not timed. Returns
    the contract's cpu_baseline object (the all-core leg) with the one-thread
    leg inside."""
    k, n16, n8 = wl.counts()
    C = wl.cache_slots()
    B = wl.batch
    cap = min(wl.d_ff, B * k)
    n_cores = len(os.sched_getaffinity(0))
    oracle.set_threads(n_cores)

    def tier_maps(t):  # [B][d_ff] (rows of step t)
        return np.stack([oracle.select_tiers(oracle.predict(ld.pred_a, ld.pred_b, ld.bias,
                                                            ld.x[t, b])[1], k, n16, n8)[0]
                         for b in range(B)])

    # records for the neurons the sample can touch (found by a first pass)
    steps_avail = ld.x.shape[0]
    tiers_by_step = [tier_maps(t) for t in range(steps_avail)]
    used = np.nonzero(np.any(np.concatenate(tiers_by_step) > 0, axis=0))[0]
    row = np.full(wl.d_ff, -1, np.int64)
    row[used] = np.arange(used.size)
    recs = {q: oracle.build_records(ld.w_gate[used], ld.w_up[used],
                                    np.ascontiguousarray(ld.w_down[:, used]), q) for q in (1, 2, 3)}

    def leg(threads, budget):
        oracle.set_threads(threads)
        if tier_slots is None:
            cache = oracle.LRUCache(wl.d_ff, C, max(0, cap - C), policy)
        else:
            cache = oracle.TierPoolCache(wl.d_ff, tier_slots,
                                         {t: max(0, cap - tier_slots[t]) for t in (1, 2, 3)}, policy)
        t_start = time.perf_counter()
        done = 0
        for t in range(steps_avail):
            tm = tier_maps(t)
            plan = cache.plan(tm if B > 1 else tm[0], t)
            ids = row[plan["req_ids"]].astype(np.int32)
            oracle.sparse_ffn(ld.x[t], ids, plan["req_tier"], recs,
                              plan["req_mask"] if B > 1 else None)
            done += 1
            if time.perf_counter() - t_start > budget:
                break
        per = (time.perf_counter() - t_start) / done
        return per, done, oracle.get_threads()

    per1, done1, _ = leg(1, budget_s / 2)
    perN, doneN, used_threads = leg(n_cores, budget_s / 2)
    oracle.set_threads(1)
    rows = f" of {B} rows" if B > 1 else ""
    return {"value": B / (perN * n_layers), "unit": "tokens/s", "cores": used_threads,
            "kind": "oracle",
            "sample": f"layer 0 of the {wl.name} stack, {doneN} consecutive decode steps{rows} of "
                      f"predict + select + LRU plan + fp64 sparse FFN on {used_threads} threads "
                      f"(OpenMP over independent sums); {perN * 1e3:.1f} ms per layer-step, "
                      f"scaled to {n_layers} layers",
            "ms_per_layer_step": perN * 1e3,
            "cpu_model": _cpu_model(), "sched_getaffinity": n_cores,
            "one_thread": {"value": B / (per1 * n_layers), "unit": "tokens/s", "cores": 1,
                           "ms_per_layer_step": per1 * 1e3, "steps": done1}}


def hold_stream(torch, s, host_seconds):
    """Enqueue a spin kernel on `s` that lasts longer than `host_seconds` of
    host work, so that everything the host enqueues behind it runs back to
    back on the GPU (measured launches are then not spaced out by the host's
    own enqueue time). Returns the event recorded before the spin."""
    probe = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(s):
        probe[0].record(s)
        torch.cuda._sleep(1 << 20)
        probe[1].record(s)
        torch.cuda.synchronize()
        ms_per_cycle = max(probe[0].elapsed_time(probe[1]), 1e-3) / float(1 << 20)
        # twice the host time, at most two seconds
        ms = min(2.0 * host_seconds * 1e3, 2000.0)
        cycles = int(ms / ms_per_cycle) + (1 << 20)
        start = torch.cuda.Event(enable_timing=True)
        start.record(s)
        torch.cuda._sleep(cycles)
    return start


def _union(iv):
    """Sorted, merged list of (start, end) intervals."""
    out = []
    for a, b in sorted(iv):
        if out and a <= out[-1][1]:
            out[-1] = (out[-1][0], max(out[-1][1], b))
        else:
            out.append((a, b))
    return out


def _measure(iv):
    return sum(b - a for a, b in iv)


def _intersect(u, v):
    """Measure of the intersection of two merged interval lists."""
    i = j = 0
    tot = 0.0
    while i < len(u) and j < len(v):
        a, b = max(u[i][0], v[j][0]), min(u[i][1], v[j][1])
        tot += max(0.0, b - a)
        if u[i][1] < v[j][1]:
            i += 1
        else:
            j += 1
    return tot


def stage_overlap(spans):
    """From per layer-step events (aux start/end, fill start/end, FFN
    start/end, all on one clock): the fraction of the fills' busy time during
    which predict / plan or the FFN was also running, and the fraction of the
    compute's busy time that ran under a fill."""
    base = spans[0][0]
    t = [[base.elapsed_time(e) for e in sp] for sp in spans]
    fill = _union([(r[2], r[3]) for r in t])
    comp = _union([(r[0], r[1]) for r in t] + [(r[4], r[5]) for r in t])
    both = _intersect(fill, comp)
    return {"fill_time_overlapped_with_compute": both / max(_measure(fill), 1e-12),
            "compute_time_under_fills": both / max(_measure(comp), 1e-12),
            "fill_busy_frac_of_span": _measure(fill) / max(t[-1][5] - t[0][0], 1e-12),
            "layer_steps": len(spans)}


def timed_back_to_back(torch, s, calls, host_seconds):
    """Run `calls` (zero-argument launchers) back to back on stream `s`
    behind a spin kernel, between one pair of HIP events. Returns the average
    time per call in ms and whether the spin outlasted the host's enqueue
    (if not, the GPU waited on the host and the average is too high)."""
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start = hold_stream(torch, s, host_seconds)
    t0 = time.perf_counter()
    e0.record(s)
    for fn in calls:
        fn()
    e1.record(s)
    enq_ms = (time.perf_counter() - t0) * 1e3
    torch.cuda.synchronize()
    covered = start.elapsed_time(e0) > enq_ms
    return e0.elapsed_time(e1) / len(calls), covered


def ffn_isolated(wl, n_layers, reps, torch, m2c, W, flags=0):
    """The sparse FFN alone on `n_layers` layers of workload `wl`'s shape that
    share one neuron store: a few decode steps fill every layer's cache, then
    the FFN of each layer is launched `reps` times, cycling through the layers
    (their active records exceed the 256 MB Infinity Cache for the 70B shape,
    so the data comes from HBM), back to back on one stream. Returns the HBM
    roofline of the FFN call (algorithmic bytes: every active record at its
    tier, x and y; with a batch, the union of the rows' active records at
    the union tier, averaged over the layers)."""
    k, n16, n8 = wl.counts()
    n4 = k - n16 - n8
    C = wl.cache_slots()
    B = wl.batch
    desc = m2c.make_desc(wl.d_model, wl.d_ff, wl.pred_rank, k, C, max_batch=B, flags=flags)
    steps = 4
    layers = []
    for l in range(n_layers):
        ld = W.workload_layer(wl, l, steps=steps, draw_weights=(l == 0))
        layers.append((m2c.Layer(desc, ld, weights_of=layers[0][0] if l else None),
                       torch.from_numpy(ld.x[:, :B].view(np.uint16)).view(torch.float16).cuda()))
    d, d_ff = wl.d_model, wl.d_ff
    tiers = torch.empty((B, d_ff), dtype=torch.uint8, device="cuda")
    y = torch.zeros((B, d), dtype=torch.float32, device="cuda")
    s = torch.cuda.current_stream()
    for t in range(steps):
        for L, x in layers:
            L.predict_rank(x[t], B, k, n16, n8, None, tiers, stream=s)
            L.cache_plan(tiers, B, t, stream=s)
            L.cache_fill(stream=s)
            L.sparse_ffn(x[t], B, y, stream=s)
    torch.cuda.synchronize()
    calls = [(lambda L=L, x=x: L.sparse_ffn(x[steps - 1], B, y, stream=s))
             for _ in range(reps) for L, x in layers]
    t0 = time.perf_counter()
    for fn in calls[:n_layers]:
        fn()
    torch.cuda.synchronize()
    per_call = (time.perf_counter() - t0) / n_layers
    ms, covered = timed_back_to_back(torch, s, calls, per_call * len(calls) * 10 + 0.05)
    rb = layers[0][0].info.record_bytes
    if B == 1:
        nbytes = n16 * rb[3] + n8 * rb[2] + n4 * rb[1] + 2 * d + 4 * d
    else:
        per = [L.read_plan()["counts"] for L, _ in layers]
        nbytes = int(round(sum(c[m2c.CNT_REQ_FP16] * rb[3] + c[m2c.CNT_REQ_INT8] * rb[2] +
                               c[m2c.CNT_REQ_INT4] * rb[1] for c in per) / len(per))) + B * 6 * d
    avg = ms * 1e-3
    for L, _ in layers:
        L.close()
    if not covered:
        log("warning: the host enqueue outlasted the stream hold; FFN time is overstated")
    return {"workload": wl.name, "layers_cycled": n_layers, "launches": len(calls),
            "us_avg": avg * 1e6, "bytes_per_launch": nbytes, "achieved_GBps": nbytes / avg / 1e9,
            "frac_of_peak": nbytes / avg / 1e9 / PEAK_HBM_GBPS, "host_hidden": bool(covered)}


def predict_isolated(wl, n_layers, reps, torch, m2c, W):
    """m2c_predict_rank (predictor z and s kernels, then the top-k select)
    alone on `n_layers` layers of workload `wl`'s shape (their predictors
    exceed the Infinity Cache for the 70B shape), back to back on one stream.
    Algorithmic bytes per call: 2 (r d + d_ff r) of predictor weights, 2 d of x,
    4 d_ff of scores written and read by the select, d_ff of tier map."""
    k, n16, n8 = wl.counts()
    d, d_ff, r = wl.d_model, wl.d_ff, wl.pred_rank
    desc = m2c.make_desc(d, d_ff, r, k, 0)
    layers = []
    for l in range(n_layers):
        ld = W.workload_layer(wl, l, steps=1, draw_weights=(l == 0))
        layers.append((m2c.Layer(desc, ld, weights_of=layers[0][0] if l else None),
                       torch.from_numpy(ld.x[:, 0].view(np.uint16)).view(torch.float16).cuda()))
    tiers = torch.empty((1, d_ff), dtype=torch.uint8, device="cuda")
    s = torch.cuda.current_stream()
    calls = [(lambda L=L, x=x: L.predict_rank(x[0], 1, k, n16, n8, None, tiers, stream=s))
             for _ in range(reps) for L, x in layers]
    for fn in calls[:n_layers]:
        fn()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for fn in calls[:n_layers]:
        fn()
    torch.cuda.synchronize()
    per_call = (time.perf_counter() - t0) / n_layers
    ms, covered = timed_back_to_back(torch, s, calls, per_call * len(calls) * 10 + 0.05)
    nbytes = 2 * (r * d + d_ff * r) + 2 * d + 4 * d_ff * 2 + d_ff
    for L, _ in layers:
        L.close()
    return {"workload": wl.name, "layers_cycled": n_layers, "launches": len(calls),
            "us_avg": ms * 1e3, "bytes_per_call": nbytes,
            "achieved_GBps": nbytes / (ms * 1e-3) / 1e9, "host_hidden": bool(covered)}


def fill_sweep(torch, m2c, W):
    """Host-to-HBM transfer rate against the size of a transfer (the analog of
    the paper's Fig. 5, transfer time and bandwidth against tensor size), on
    the 70B record sizes: for n records of one tier, n in 1 .. 2048,
      gather  m2c_cache_fill of a plan with n NEW neurons (one launch of the
              device gather kernel over the pinned host store);
      memcpy  n hipMemcpyAsync calls of one record each, pinned host to
              scattered slots of a device arena (the neuron-level copies the
              paper issues on its streams);
      bulk    one hipMemcpyAsync of the same n records' bytes, contiguous
              (the copy engine's rate on large transfers).
    Each is timed with HIP events on one stream, averaged over repetitions."""
    wl = W.WORKLOADS["llama2-70b"]
    d, d_ff, r = wl.d_model, 4096, 8
    ld = W.make_layer(wl.seed + 7, 0, d, d_ff, r, 1, sigma_w=wl.sigma_w)
    desc = m2c.make_desc(d, d_ff, r, 2048, 2048)
    L = m2c.Layer(desc, ld)
    s = torch.cuda.current_stream()
    rows = []
    host = torch.empty(2048 * 6 * d, dtype=torch.uint8, pin_memory=True)
    arena = torch.empty(4096 * 6 * d, dtype=torch.uint8, device="cuda")
    perm = np.random.default_rng(3).permutation(4096)
    for tier in (3, 2, 1):
        rb = L.info.record_bytes[tier]
        for n in (1, 4, 16, 64, 256, 1024, 2048):
            reps = max(2, min(50, 4096 // n))
            tm = np.zeros((1, d_ff), np.uint8)
            tm[0, :n] = tier
            tmd = torch.from_numpy(tm).cuda()
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            tot = 0.0
            for q in range(reps):
                L.reset_cache(stream=s)
                L.cache_plan(tmd, 1, 0, stream=s)
                ev[0].record(s)
                L.cache_fill(stream=s)
                ev[1].record(s)
                torch.cuda.synchronize()
                tot += ev[0].elapsed_time(ev[1])
            g_ms = tot / reps
            # per-record copies into scattered slots of the arena
            tot = 0.0
            for q in range(reps):
                ev[0].record(s)
                for j in range(n):
                    dst = int(perm[j]) * 6 * d
                    arena[dst:dst + rb].copy_(host[j * rb:(j + 1) * rb], non_blocking=True)
                ev[1].record(s)
                torch.cuda.synchronize()
                tot += ev[0].elapsed_time(ev[1])
            m_ms = tot / reps
            tot = 0.0
            for q in range(reps):
                ev[0].record(s)
                arena[:n * rb].copy_(host[:n * rb], non_blocking=True)
                ev[1].record(s)
                torch.cuda.synchronize()
                tot += ev[0].elapsed_time(ev[1])
            b_ms = tot / reps
            nb = n * rb
            rows.append({"tier": tier, "record_bytes": rb, "records": n, "bytes": nb,
                         "gather_us": g_ms * 1e3, "gather_GBps": nb / g_ms / 1e6,
                         "memcpy_us": m_ms * 1e3, "memcpy_GBps": nb / m_ms / 1e6,
                         "bulk_us": b_ms * 1e3, "bulk_GBps": nb / b_ms / 1e6})
            log(f"fill sweep tier {tier} n {n}: gather {rows[-1]['gather_GBps']:.1f} GB/s, "
                f"memcpy {rows[-1]['memcpy_GBps']:.1f}, bulk {rows[-1]['bulk_GBps']:.1f}")
    L.close()
    return {"d_model": d, "rows": rows}


def batched_sweep(steps, warmup, torch, m2c, W, only=None):
    """The batched-decode workload: one 7B-shaped layer, batch 8 (rows with
    rho 0.5 and 0.95, log-Zipf neuron popularity), predict -> plan -> fill ->
    batched FFN per step on one stream, for LRU capacity 10 / 30 / 60 % of
    d_ff and tiers 10/40/50 or all FP16. Per point: step time, tokens/s
    (batch rows per second), the union's size and hit rate, fill traffic and
    the FFN's algorithmic bytes over its time. `only` = (capacity fraction,
    tier mix) restricts the sweep to that point."""
    wl = W.WORKLOADS["llama2-7b-b8"]
    B = wl.batch
    k, n16_m, n8_m = wl.counts()
    ld = W.workload_layer(wl, 0, steps=warmup + steps)
    x = torch.from_numpy(ld.x.view(np.uint16)).view(torch.float16).cuda()  # [steps][B][d]
    d, d_ff = wl.d_model, wl.d_ff
    tiers = torch.empty((B, d_ff), dtype=torch.uint8, device="cuda")
    y = torch.zeros((B, d), dtype=torch.float32, device="cuda")
    s = torch.cuda.current_stream()
    owner, points = None, []
    for cap in (F(1, 10), F(3, 10), F(3, 5)):
        for mix in ("10/40/50", "fp16"):
            if only is not None and (cap, mix) != only:
                continue
            n16, n8 = (n16_m, n8_m) if mix != "fp16" else (k, 0)
            C = int(d_ff * cap // 1)
            desc = m2c.make_desc(d, d_ff, wl.pred_rank, k, C, max_batch=B)
            L = m2c.Layer(desc, ld, weights_of=owner)
            if owner is None:
                owner = L
            ev = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(steps)]
            for t in range(warmup + steps):
                e = ev[t - warmup] if t >= warmup else None
                y.zero_()
                if e:
                    e[0].record(s)
                L.predict_rank(x[t], B, k, n16, n8, None, tiers, stream=s)
                if e:
                    e[1].record(s)
                L.cache_plan(tiers, B, t, stream=s)
                if e:
                    e[2].record(s)
                L.cache_fill(stream=s)
                if e:
                    e[3].record(s)
                L.sparse_ffn(x[t], B, y, stream=s)
                if e:
                    e[4].record(s)
                if t == warmup - 1:
                    torch.cuda.synchronize()
                    st0 = L.stats()
            torch.cuda.synchronize()
            st1 = L.stats()
            ms = np.array([[e[i].elapsed_time(e[i + 1]) for i in range(4)] for e in ev])
            step_ms = np.array([e[0].elapsed_time(e[4]) for e in ev])
            req = st1.req - st0.req
            ffn_bytes = (st1.req_bytes - st0.req_bytes) / steps + B * (2 * d + 4 * d)
            ffn_s = float(ms[:, 3].mean()) * 1e-3
            points.append({
                "cache_frac": float(cap), "cache_slots": C, "tiers": mix,
                "us_per_step": float(step_ms.mean()) * 1e3,
                "tokens_per_s": B / (float(step_ms.mean()) * 1e-3),
                "us_predict_plan_fill_ffn": [round(float(v) * 1e3, 2) for v in ms.mean(axis=0)],
                "union_neurons": req / steps, "hit_rate": (st1.hit - st0.hit) / max(req, 1),
                "bypass_rate": (st1.bypass - st0.bypass) / max(req, 1),
                "fill_MB_per_step": (st1.host_bytes - st0.host_bytes) / steps / 1e6,
                "derived_MB_per_step": ((st1.fill_bytes - st0.fill_bytes)
                                        - (st1.host_bytes - st0.host_bytes)) / steps / 1e6,
                "ffn_bytes_per_step": ffn_bytes, "ffn_GBps": ffn_bytes / ffn_s / 1e9})
            log(f"batched sweep: cache {float(cap):.0%} tiers {mix}: "
                f"{points[-1]['us_per_step']:.1f} us/step")
            if L is not owner:
                L.close()
    owner.close()
    return {"workload": wl.name, "batch": B, "steps": steps, "warmup": warmup, "points": points}


class _StageEvents:
    """Hooks of the schedule that record HIP events around the stages:
    `timed` keeps (FFN start, FFN end, fill start, fill end) per layer-step,
    `spans` keeps (aux start, aux end, fill start, fill end, FFN start, FFN
    end) for the overlap measurement."""

    def __init__(self, torch, timed, spans):
        self.torch = torch
        self.timed, self.spans = timed, spans
        self.cur = None

    def _ev(self, s, i):
        self.cur[i].record(s)

    def before_predict(self, l, t, s):
        self.cur = [self.torch.cuda.Event(enable_timing=True) for _ in range(6)]
        self._ev(s, 0)

    def after_plan(self, l, t, s):
        self._ev(s, 1)

    def before_fill(self, l, t, s):
        self._ev(s, 2)

    def after_fill(self, l, t, s):
        self._ev(s, 3)

    def before_ffn(self, l, t, s):
        self._ev(s, 4)

    def after_ffn(self, l, t, s):
        self._ev(s, 5)
        (self.spans if self.spans is not None else self.timed).append(self.cur)


def run_stack(wl, n_layers, steps, warmup, weight_sets, flags, overlap_steps, stage_events,
              torch, m2c, W, tier_slots=None):
    """The decode pipeline over the whole stack: `warmup` untimed steps,
    `steps` timed ones between a synchronization on each side, then
    `overlap_steps` untimed steps with events around every stage."""
    from paper_2410_14740_amd import pipeline
    k, n16, n8 = wl.counts()
    steps_total = warmup + steps
    t_setup = time.perf_counter()
    layers, x_dev, ld0 = build_stack(wl, n_layers, steps_total + overlap_steps, weight_sets, torch,
                                     m2c, W, flags=flags, tier_slots=tier_slots)
    log(f"setup {time.perf_counter() - t_setup:.1f} s")
    d, d_ff, B = wl.d_model, wl.d_ff, wl.batch
    tiers = torch.empty((n_layers, B, d_ff), dtype=torch.uint8, device="cuda")
    # m2c_sparse_ffn adds into y (a residual stream): zeroed rows per
    # layer-step, so every output is the plain FFN of its token
    y = torch.zeros((steps_total + overlap_steps, n_layers, B, d), dtype=torch.float32,
                    device="cuda")
    sched = pipeline.StackSchedule(torch, layers, k, n16, n8, tiers, lag=2, batch=B)
    timing = []
    ev_hooks = _StageEvents(torch, timing, None) if stage_events else None

    def step(t, hooks=None):
        sched.step(t, lambda l: x_dev[l, t], lambda l: y[t, l], hooks=hooks)

    for t in range(warmup):
        step(t)
    torch.cuda.synchronize()
    st0 = [L.stats() for L in layers]
    t0 = time.perf_counter()
    for t in range(warmup, steps_total):
        step(t, ev_hooks)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    st1 = [L.stats() for L in layers]
    # A few more steps, untimed, with events around every stage: how much of
    # the fills' time runs while predict / plan or the FFN runs on another
    # stream (the events themselves delay the cross-stream waits a little, so
    # they stay out of the timed steps). The aux stream (and through the
    # events the other two) is held by a spin kernel while the host enqueues,
    # so the extra calls do not space the stages out.
    spans = []
    if overlap_steps:
        hold_stream(torch, sched.aux, 0.002 * n_layers * overlap_steps)
        sp_hooks = _StageEvents(torch, None, spans)
        for t in range(steps_total, steps_total + overlap_steps):
            step(t, sp_hooks)
    torch.cuda.synchronize()
    overlap = stage_overlap(spans) if spans else None
    ffn_ms = np.array([e[4].elapsed_time(e[5]) for e in timing]) if timing else None
    fill_ms = np.array([e[2].elapsed_time(e[3]) for e in timing]) if timing else None
    diff = lambda f: sum(getattr(b, f) - getattr(a, f) for a, b in zip(st0, st1))
    reqs = diff("req")
    # bytes the fills read over the host link (fills derived on the GPU from a
    # resident FP16 record read none)
    fill_bytes = diff("host_bytes")
    derived_bytes = diff("fill_bytes") - fill_bytes
    n_ls = steps * n_layers
    # host-link rate of the fills: from the stage events if recorded, else the
    # fill bytes over the wall time (a lower bound: fills run back to back only
    # when nothing else is on the critical path)
    fill_avg_s = float(fill_ms.mean()) * 1e-3 if fill_ms is not None else wall / n_ls
    info = layers[0].info
    for L in layers:
        L.close()
    return {
        "wall": wall, "n_layer_steps": n_ls, "ld0": ld0, "info": info,
        "tokens_per_s": steps * B / wall, "us_per_layer_step": wall / n_ls * 1e6,
        "pipeline": {
            "stage_events": bool(stage_events),
            "ffn_us_avg": float(ffn_ms.mean()) * 1e3 if ffn_ms is not None else None,
            "fill_us_avg": fill_avg_s * 1e6 if fill_ms is not None else None,
            "fill_MB_per_layer_step": fill_bytes / n_ls / 1e6,
            "derived_MB_per_layer_step": derived_bytes / n_ls / 1e6,
            "ffn_MB_per_layer_step": diff("req_bytes") / n_ls / 1e6,
            "cache": {"hit_rate": diff("hit") / max(reqs, 1),
                      "refill_rate": diff("refill") / max(reqs, 1),
                      "new_rate": diff("new_") / max(reqs, 1),
                      "bypass_rate": diff("bypass") / max(reqs, 1)},
            "overlap": overlap,
        },
        "host_link": {"kernel": "fill_kernel (device gather from pinned host memory)",
                      "achieved": fill_bytes / n_ls / fill_avg_s / 1e9,
                      "peak": PEAK_HOST_LINK_GBPS, "unit": "GB/s",
                      "frac": fill_bytes / n_ls / fill_avg_s / 1e9 / PEAK_HOST_LINK_GBPS,
                      "measured_over": "fill kernels" if fill_ms is not None else "wall time"},
    }


def policy_sweep(steps, torch, m2c, W):
    """Cache behaviour against the inter-token correlation of the inputs (the
    paper's Fig. 6 reports about 80% overlap between consecutive tokens' active
    sets): on two 7B-shaped layers, for rho in {0.5, 0.7, 0.8, 0.9, 0.95},
    the consecutive-step overlap |S_t & S_t-1| / k measured from the plans and
    the hit rates of exact-tier and dominance hits with LRU at C = 30% of d_ff
    and at C = k (where LRU is the paper's Adjacent Token Update policy);
    then the 7B stack's tokens/s and host-link bytes under both policies."""
    wl0 = W.WORKLOADS["llama2-7b"]
    k, n16, n8 = wl0.counts()
    d, d_ff = wl0.d_model, wl0.d_ff
    rows = []
    owner = None
    tiers = torch.empty((1, d_ff), dtype=torch.uint8, device="cuda")
    s = torch.cuda.current_stream()
    for rho in (0.5, 0.7, 0.8, 0.9, 0.95):
        for C, cname in ((wl0.cache_slots(), "lru_30pct"), (k, "atu_c_eq_k")):
            for pol, flag in (("exact", 0), ("dominance", m2c.FLAG_DOMINANT_HITS)):
                hits = reqs = host = ovl = 0
                for l in range(2):
                    ld = W.make_layer(wl0.seed + 100, l, d, d_ff, wl0.pred_rank, steps, (rho,),
                                      wl0.sigma_w, wl0.sigma_p, draw_weights=owner is None)
                    L = m2c.Layer(m2c.make_desc(d, d_ff, wl0.pred_rank, k, C, flags=flag), ld,
                                  weights_of=owner)
                    if owner is None:
                        owner = L
                    x = torch.from_numpy(ld.x[:, 0].view(np.uint16)).view(torch.float16).cuda()
                    prev = None
                    for t in range(steps):
                        L.predict_rank(x[t], 1, k, n16, n8, None, tiers, stream=s)
                        L.cache_plan(tiers, 1, t, stream=s)
                        L.cache_fill(stream=s)
                        if t >= 4:  # steady state: the cache has warmed up
                            if t == 4:
                                torch.cuda.synchronize()
                                st0 = L.stats()
                        cur = set(L.read_plan()["req_ids"].tolist())
                        if prev is not None and t >= 4:
                            ovl += len(cur & prev)
                        prev = cur
                    torch.cuda.synchronize()
                    st1 = L.stats()
                    hits += st1.hit - st0.hit
                    reqs += st1.req - st0.req
                    host += st1.host_bytes - st0.host_bytes
                    if L is not owner:
                        L.close()
                n = 2 * (steps - 4)
                rows.append({"rho": rho, "cache": cname, "cache_slots": C, "policy": pol,
                             "overlap": ovl / (n * k), "hit_rate": hits / max(reqs, 1),
                             "host_MB_per_layer_step": host / n / 1e6})
                log(f"policy sweep rho {rho} {cname} {pol}: hit {rows[-1]['hit_rate']:.3f}")
    owner.close()
    stacks = {}
    for pol, flag in (("exact", 0), ("dominance", m2c.FLAG_DOMINANT_HITS)):
        r = run_stack(wl0, wl0.n_layers, 24, 8, 0, flag, 0, False, torch, m2c, W)
        stacks[pol] = {"tokens_per_s": r["tokens_per_s"], "us_per_layer_step": r["us_per_layer_step"],
                       "host_MB_per_layer_step": r["pipeline"]["fill_MB_per_layer_step"],
                       "cache": r["pipeline"]["cache"]}
        log(f"7B stack, {pol}: {r['tokens_per_s']:.1f} tokens/s")
    return {"workload": wl0.name, "steps_per_point": steps, "points": rows, "stack_7b": stacks}


def ssd_tier(args, torch, m2c, W):
    """The SSD -> DRAM tier (Sec. 5.4) on the 7B-shaped stack: the layers'
    neuron stores in a file (`--ssd-sets` distinct weight sets, layer l reads
    set l mod sets, so every load is a real read of a whole layer), a pinned
    two-level DRAM cache (`--ssd-fixed` layers in the fixed area,
    `--ssd-slots` dynamic slots, look-ahead `--ssd-lookahead`, direct I/O),
    and the decode pipeline reading every fill through the cache. Reports
    tokens/s, the file read rate, how long fills waited for their layer, and
    the DRAM the cache holds against all layers in DRAM."""
    from paper_2410_14740_amd import pipeline
    wl = W.WORKLOADS["llama2-7b"]
    n_layers = args.layers or wl.n_layers
    k, n16, n8 = wl.counts()
    C = wl.cache_slots()
    desc = m2c.make_desc(wl.d_model, wl.d_ff, wl.pred_rank, k, C)
    sets = args.ssd_sets
    steps = args.warmup + args.steps
    path = os.path.join(args.ssd_dir, f"m2c_stores_{os.getpid()}.bin")
    offs, off = [], 0
    t0 = time.perf_counter()
    for q in range(sets):
        ld = W.workload_layer(wl, q, steps=1)
        o = m2c.Layer(desc, ld)
        offs.append(off)
        off += m2c.m2c_layer_write_store(o.handle, path, off)
        o.close()
        log(f"wrote store {q + 1}/{sets} ({off / 1e9:.2f} GB)")
    os.sync()
    log(f"store file {off / 1e9:.2f} GB in {time.perf_counter() - t0:.1f} s")
    layer_bytes = sum(wl.d_ff * ((m2c.m2c_record_bytes(wl.d_model, t) + 15) // 16 * 16)
                      for t in (1, 2, 3))
    dd = m2c.DramDesc(n_layers, args.ssd_fixed, args.ssd_slots, args.ssd_lookahead, layer_bytes,
                      m2c.DRAM_DIRECT_IO, 0)
    dram = m2c.m2c_dram_create(dd, path, [offs[l % sets] for l in range(n_layers)])
    layers = []
    x_dev = torch.empty((n_layers, steps, wl.d_model), dtype=torch.float16, device="cuda")
    for l in range(n_layers):
        ld = W.workload_layer(wl, l, steps=steps, draw_weights=False)
        x_dev[l].copy_(torch.from_numpy(ld.x[:, 0].view(np.uint16)).view(torch.float16))
        layers.append(m2c.Layer(desc, ld, dram=dram, dram_index=l))
    tiers = torch.empty((n_layers, wl.d_ff), dtype=torch.uint8, device="cuda")
    y = torch.zeros((steps, n_layers, wl.d_model), dtype=torch.float32, device="cuda")
    sched = pipeline.StackSchedule(torch, layers, k, n16, n8, tiers, lag=2)
    for t in range(args.warmup):
        sched.step(t, lambda l: x_dev[l, t], lambda l: y[t, l])
        log(f"ssd tier: warm-up token {t}")
    torch.cuda.synchronize()
    s0 = m2c.m2c_dram_get_stats(dram)
    t0 = time.perf_counter()
    for t in range(args.warmup, steps):
        sched.step(t, lambda l: x_dev[l, t], lambda l: y[t, l])
        log(f"ssd tier: token {t}")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    s1 = m2c.m2c_dram_get_stats(dram)
    for L in layers:
        L.close()
    m2c.m2c_dram_destroy(dram)
    os.remove(path)
    loads = s1.loads - s0.loads
    rd = s1.bytes_read - s0.bytes_read
    return {"workload": wl.name, "layers": n_layers, "tokens": args.steps, "tokens_per_s":
            args.steps / wall, "ms_per_token": wall / args.steps * 1e3,
            "fixed_layers": args.ssd_fixed, "dynamic_slots": args.ssd_slots,
            "lookahead": args.ssd_lookahead, "distinct_weight_sets_in_file": sets,
            "layer_MB": layer_bytes / 1e6, "loads_per_token": loads / args.steps,
            "file_read_GBps": rd / max(s1.read_seconds - s0.read_seconds, 1e-9) / 1e9,
            "file_GB_per_token": rd / args.steps / 1e9,
            "fill_wait_s_per_token": (s1.wait_seconds - s0.wait_seconds) / args.steps,
            "direct_io": bool(s1.direct_io),
            "dram_GB_cache": (args.ssd_fixed + args.ssd_slots) * layer_bytes / 1e9,
            "dram_GB_all_layers": n_layers * layer_bytes / 1e9}


def ratio_search(torch, m2c, W):
    """Algorithm 1 (offline neuron-ratio search) on the 7B-shaped layer with
    16 calibration tokens of its AR(1) input stream: starting from k = 20%
    of d_ff at the low tier, FP16 vs INT4 (bit ratio 4) and FP16 vs INT8
    (bit ratio 2); reports every candidate's proxy score, the chosen ratio
    and the search's wall time."""
    wl = W.WORKLOADS["llama2-7b"]
    k, _, _ = wl.counts()
    T = 16
    ld = W.workload_layer(wl, 0, steps=T)
    L = m2c.Layer(m2c.make_desc(wl.d_model, wl.d_ff, wl.pred_rank, wl.d_ff, wl.cache_slots()), ld)
    x = torch.from_numpy(np.ascontiguousarray(ld.x[:, 0].view(np.uint16))).cuda()
    out = {"workload": wl.name, "calibration_tokens": T, "n_low0": k, "searches": []}
    for step, n in ((32, 4), (64, 2)):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        cands, uqs, best = m2c.m2c_ratio_search(L.handle, x, T, k, step, n)
        el = time.perf_counter() - t0
        out["searches"].append({"bit_ratio": n, "step": step, "candidates": cands, "uq": uqs,
                                "best": cands[best], "best_uq": uqs[best], "seconds": el})
        log(f"ratio search n={n}: best {cands[best]} uq {uqs[best]:.4e} in {el:.2f} s")
    L.close()
    return out


def main():
    args = parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}): the hot path is "
              "built and measured on a single MI355X.", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2410_14740_amd import m2c
    from paper_2410_14740_amd import workloads as W

    if not os.path.exists(m2c.LIB_PATH):
        from paper_2410_14740_amd import build as hip_build
        hip_build.build()
    m2c.load()
    torch.cuda.set_device(0)
    if args.calibrate_copy:
        n = args.calibrate_copy << 20
        a = torch.ones(n, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        for _ in range(5):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n, "launches": 5}), flush=True)
        return
    ffn_flags = m2c.FLAG_DETERMINISTIC_FFN if args.deterministic_ffn else 0
    if args.batch_sweep:
        only = None
        if args.sweep_point:
            cap_s, mix = args.sweep_point.split(":")
            only = (F(cap_s), mix)
        print(json.dumps({"batched_sweep": batched_sweep(min(args.steps, 56), args.warmup, torch,
                                                          m2c, W, only)}), flush=True)
        return
    if args.policy_sweep:
        print(json.dumps({"policy_sweep": policy_sweep(min(args.steps, 36), torch, m2c, W)}),
              flush=True)
        return
    if args.only_predict:
        wl_p = W.WORKLOADS[args.only_predict]
        print(json.dumps({"predict_isolated": predict_isolated(wl_p, 8, args.ffn_reps, torch, m2c,
                                                               W)}), flush=True)
        return
    if args.ratio_search:
        print(json.dumps({"ratio_search": ratio_search(torch, m2c, W)}), flush=True)
        return
    if args.ssd_tier:
        print(json.dumps({"ssd_tier": ssd_tier(args, torch, m2c, W)}), flush=True)
        return
    if args.fill_sweep:
        print(json.dumps({"fill_sweep": fill_sweep(torch, m2c, W)}), flush=True)
        return
    if args.only_ffn:
        wl_f = W.WORKLOADS[args.only_ffn]
        g = ffn_isolated(wl_f, args.ffn_layers if args.only_ffn == args.workload
                         else args.extra_layers, args.ffn_reps, torch, m2c, W, flags=ffn_flags)
        print(json.dumps({"ffn_isolated": g}), flush=True)
        return
    wl = W.WORKLOADS[args.workload]
    n_layers = args.layers or wl.n_layers
    k, n16, n8 = wl.counts()
    n4 = k - n16 - n8
    weight_sets = args.weight_sets if args.weight_sets >= 0 else (
        8 if wl.name == "llama2-70b" else 0)
    flags = ffn_flags | (m2c.FLAG_DOMINANT_HITS if args.policy == "dominance" else 0)
    tier_slots = None
    if wl.batch > 1:
        log(f"batch {wl.batch}: one arena (the per-tier arena serves batch 1)")
    elif args.arena == "pools":
        tier_slots = m2c.pool_slots_for_budget(wl.d_model, {3: n16, 2: n8, 1: n4},
                                               wl.cache_slots() * 6 * wl.d_model)
        log(f"per-tier arena: {tier_slots} resident slots (FP16, INT8, INT4 pools)")
    r = run_stack(wl, n_layers, args.steps, args.warmup, weight_sets, flags, args.overlap_steps,
                  args.stage_events, torch, m2c, W, tier_slots=tier_slots)
    log(f"stack: {r['tokens_per_s']:.2f} tokens/s")
    variants = {}
    if not args.no_variants and tier_slots is not None:
        # the other cache policies and arenas at the same HBM budget
        others = [("single_arena_exact_tier", ffn_flags, None),
                  ("single_arena_dominance", ffn_flags | m2c.FLAG_DOMINANT_HITS, None)]
        if args.policy == "dominance":
            others.insert(0, ("pools_exact_tier", ffn_flags, tier_slots))
        else:
            others.insert(0, ("pools_dominance", ffn_flags | m2c.FLAG_DOMINANT_HITS, tier_slots))
        for name, fl, ts in others:
            rv = run_stack(wl, n_layers, args.steps, args.warmup, weight_sets, fl, 0, False, torch,
                           m2c, W, tier_slots=ts)
            variants[name] = {"tokens_per_s": rv["tokens_per_s"],
                              "us_per_layer_step": rv["us_per_layer_step"],
                              "host_MB_per_layer_step": rv["pipeline"]["fill_MB_per_layer_step"],
                              "cache": rv["pipeline"]["cache"]}
            log(f"variant {name}: {rv['tokens_per_s']:.2f} tokens/s")
    log(f"isolated sparse FFN on {args.ffn_layers} {wl.name}-shaped layers")
    iso = ffn_isolated(wl, args.ffn_layers, args.ffn_reps, torch, m2c, W, flags=ffn_flags)
    extra = None
    if args.extra_workload and args.extra_workload != wl.name:
        log(f"isolated sparse FFN on {args.extra_layers} {args.extra_workload}-shaped layers")
        extra = ffn_isolated(W.WORKLOADS[args.extra_workload], args.extra_layers, args.ffn_reps,
                             torch, m2c, W, flags=ffn_flags)

    cpu = None
    if args.cpu_seconds > 0:
        import oracle
        log("timing the oracle on the host")
        cpu = cpu_baseline(wl, r["ld0"], n_layers, args.cpu_seconds, oracle,
                           oracle.POLICY_DOMINANCE if args.policy == "dominance"
                           else oracle.POLICY_EXACT, tier_slots)

    # HBM bytes per call from the committed counter summary of this layer
    # shape, or None when the FFN kernels have changed since it was taken
    from paper_2410_14740_amd import rocprof_summary

    def traffic(name):
        return None if args.deterministic_ffn else rocprof_summary.read_ffn_traffic(
            os.path.join(ROOT, "profiles", f"sparse_ffn_{name}_layer.md"))

    ffn_kind = ("three kernels (up, down, ordered reduce), deterministic" if args.deterministic_ffn
                else "batched: gate/up and down on the matrix cores" if wl.batch > 1
                else "one launch (h tasks, then down tasks that wait on the h words)")
    d, d_ff = wl.d_model, wl.d_ff

    def roof(g, name, layers_cycled):
        return {"bound": "hbm", "achieved": g["achieved_GBps"], "peak": PEAK_HBM_GBPS,
                "unit": "GB/s", "frac": g["achieved_GBps"] / PEAK_HBM_GBPS,
                "traffic": traffic(name) if W.WORKLOADS[name].batch == 1 else None,
                "kernel": ("m2c_sparse_ffn (ffn_bh_kernel + ffn_bdm_kernel)"
                           if W.WORKLOADS[name].batch > 1 else "m2c_sparse_ffn (ffn_fused_kernel)"),
                "workload": f"{name} layer shape, {layers_cycled} layers cycled",
                "bytes_per_launch": g["bytes_per_launch"], "us_per_launch": g["us_avg"]}

    out = {
        "metric": METRIC,
        "value": r["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": r["wall"] / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": wl.name, "layers": n_layers, "d_model": d, "d_ff": d_ff,
            "pred_rank": wl.pred_rank, "k": k, "tiers_fp16_int8_int4": [n16, n8, n4],
            "cache_slots": wl.cache_slots(), "batch": wl.batch,
            "decode_steps": args.warmup + args.steps,
            "weights": "fp16 records with int8/int4 copies (group 128, fp16 scales), "
                       "pinned host store",
            "distinct_weight_sets": weight_sets or n_layers,
            "cache_policy": "LRU, " + ("dominance hits" if args.policy == "dominance"
                                       else "exact-tier hits") + (
                ", per-tier arena {FP16, INT8, INT4} = " + str([tier_slots[3], tier_slots[2],
                                                                tier_slots[1]])
                if tier_slots else ""),
            "ffn": ffn_kind,
        },
        "us_per_layer_step": r["us_per_layer_step"],
        "pipeline": r["pipeline"],
        # the step's gather-GEMV (m2c_sparse_ffn: ffn_fused_kernel) on this
        # workload's layer shape: algorithmic bytes per call over the per-call
        # time of back-to-back calls between one pair of HIP events
        "roofline": roof(iso, wl.name, args.ffn_layers),
        "roofline_extra_layer": None if extra is None else roof(extra, extra["workload"],
                                                                 args.extra_layers),
        # the fills are bound by the host link, not by HBM
        "host_link": r["host_link"],
        "cpu_baseline": cpu,
        "variants": variants or None,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
