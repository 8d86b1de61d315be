#!/usr/bin/env python3
"""Benchmark of the error-feedback sparsification hot path on one MI355X.

One step = every simulated worker (W of them) runs one fused worker step
(accumulate, compress, residual update) with each compressor variant, and the
W messages of each variant are aggregated into a dense averaged gradient.
Default workload: ResNet-50-shaped fp32 gradients (161 tensors, d = 25,557,032,
Laplace values with per-tensor scales), density 0.1 %, W = 16, compressors
top-k, random-k and block-random-k with start alignments 256 / 4096 / 65536,
global (flat) scope.  Inputs are resident in HBM before the timed region.

Prints ONE JSON line on stdout (progress goes to stderr).  `value` is compressed
gradient elements per second over the whole step: n_variants * W * d elements
per step.  `roofline` is for the kernel with the largest total time, timed
per launch with HIP events the library records on the launch's stream.
`cpu_baseline` times the CPU oracle on a bounded sample of the same workload.
"""

from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

import numpy as np

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, 8 TB/s
METRIC = "compressed gradient elements/s per compressor at 1 GPU; % of MI355X HBM BW"


def _note(msg):
    """A progress line on stderr (the JSON result goes to stdout)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def gen_gradients(wl, W, t=0):
    """The W workers' gradients of step t.  Drawn on host threads (NumPy's generators release the
    interpreter lock while they fill an array), not in forked processes: a process forked under a
    profiler carries the profiler's state with it."""
    from concurrent.futures import ThreadPoolExecutor
    from workloads import gradient
    n = max(1, min(8, os.cpu_count() or 1, W))
    if n == 1:
        return [gradient(wl, w, t) for w in range(W)]
    with ThreadPoolExecutor(n) as ex:
        return list(ex.map(lambda w: gradient(wl, w, t), range(W)))


def variant_list(spec, blocks):
    out = []
    for v in spec.split(","):
        v = v.strip()
        if v == "randblock":
            out += [("randblock", b) for b in blocks]
        elif v.startswith("randblock"):
            out.append(("randblock", int(v[len("randblock"):])))
        else:
            out.append((v, 1))
    return out


def vname(v):
    return v[0] if v[0] != "randblock" else f"randblock{v[1]}"


def alg_bytes_op(kind, d, K, L, W):
    """Algorithmic HBM bytes of one fused worker step (fp32 g) and of one aggregate."""
    if kind in ("topk", "randk"):
        step = 12 * d + 8 * K
        agg = 4 * d + W * 8 * K
    else:
        step = 12 * d + 4 * K + 4 * L
        agg = 4 * d + W * (4 * K + 4 * L)
    return step, agg


def kernel_alg_bytes(name, d, K, L, W):
    """Algorithmic bytes per launch of the streaming kernels (None for the small helpers)."""
    if name.startswith("k_randblock_step"):
        return 12 * d + 4 * K + 4 * L
    if "k_stream_sel" in name and "true>" in name:  # fused: read g, read e, write e
        return 12 * d
    if name.startswith("k_agg_sparse"):
        return 4 * d + W * 8 * K
    if name.startswith("k_agg_block"):
        return 4 * d + W * (4 * K + 4 * L)
    return None


def measure_next(E, torch, dev, wl, lay0, layouts, msg, variants, W, d, K, L, args, reps=20):
    """Average duration and HBM fraction of: the shared-coordinate aggregates (allReduce mode, the
    coordinates of worker 0's last message shared by all), the block aggregate fused with a
    momentum update of the parameters, and the dense average of W uncompressed gradients."""
    res = {}

    def timed(name, fn, alg_bytes):
        for _ in range(3):
            fn()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        us = a.elapsed_time(b) * 1e3 / reps
        res[name] = {"us": round(us, 3), "alg_bytes": int(alg_bytes),
                     "frac_of_hbm_peak": round(alg_bytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}

    out = torch.empty(d, dtype=torch.float32, device=dev)
    ws_sh = lay0.workspace(E.EF_OP_AGG_SHARED, W, dev)
    kinds = {vname(v): v for v in variants}
    if "randk" in kinds:
        mi, mv = msg["randk"]
        timed("shared_sparse_aggregate",
              lambda: E.decompress_aggregate_shared(lay0, E.EF_MSG_SPARSE, W, mi[0], mv, out, ws_sh),
              4 * d + W * 4 * K + 4 * K)
    blk = [v for v in variants if v[0] == "randblock"]
    if blk:
        v = blk[0]
        lay = layouts[v[1]]
        mi, mv = msg[vname(v)]
        timed(f"shared_block_aggregate_{vname(v)}",
              lambda: E.decompress_aggregate_shared(lay, E.EF_MSG_BLOCK, W, mi[0], mv, out, ws_sh),
              4 * d + W * 4 * K + 4 * L)
        x = torch.zeros(d, dtype=torch.float32, device=dev)
        m = torch.zeros(d, dtype=torch.float32, device=dev)
        timed(f"aggregate_apply_momentum_{vname(v)}",
              lambda: E.decompress_aggregate_apply(lay, E.EF_MSG_BLOCK, W, mi, mv, x, m, 0.9, 1e-5),
              16 * d + W * (4 * K + 4 * L))
        del x, m
    G = torch.randn((W, d), dtype=torch.float32, device=dev)
    timed("dense_average", lambda: E.ef_dense_average(lay0, W, G, out), (W + 1) * 4 * d)
    del G
    return res


def measure_prepared(E, torch, dev, timed, entry, lay, g, e, seeds, mv, step_b, d):
    """Random-k with the selection prepared ahead: the prepare call alone (it needs no gradient, so
    it can run any time before the step) and the prepared step alone, with its kernel split."""
    res = {}
    wsp = [lay.workspace(E.EF_OP_RANDK_PREP, 1, dev)]
    idx = [torch.empty(lay.K, dtype=torch.int32, device=dev)]
    def split(fn):  # per-kernel averages of fn's launches (library events, a separate pass)
        E.timing_collect(reset=True)
        E.timing_enable(True)
        timed(fn)
        E.timing_enable(False)
        return {name: round(tot * 1e3 / nl, 3) for name, (tot, nl) in E.timing_collect(reset=True).items()}

    prep = lambda: E.ef_randk_prepare(lay, seeds[0], 0, idx[0], wsp[0])  # noqa: E731
    res["prepare"] = {"us": round(timed(prep), 3), "kernels_us": split(prep)}
    step = lambda: E.ef_step_randk_prepared(lay, g[0], e, idx[0], mv[0], wsp[0])  # noqa: E731
    res["prepared_step"] = entry(timed(step), step_b, d)
    res["prepared_step"]["kernels_us"] = split(step)
    return res


def measure_single(E, torch, dev, offs, density, variants, W, g, seeds, reps=20, g_bf16=None):
    """Each compressor at the given scope: one worker's step alone (the fused entry point, and the
    composed calls accumulate + compress + update), and the aggregate of the W workers' messages
    alone; back-to-back repetitions on one stream, timed with events on that stream.  Also the
    library's plain copy kernel over d floats, as a measured streaming ceiling.  With g_bf16 (a
    bf16 copy of worker 0's gradient), the fused steps on it too."""
    d = offs[-1]
    st = torch.cuda.Stream(dev)

    def timed(fn):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        with torch.cuda.stream(st):
            for _ in range(3):
                fn()
            a.record(st)
            for _ in range(reps):
                fn()
            b.record(st)
        torch.cuda.synchronize()
        return a.elapsed_time(b) * 1e3 / reps

    def entry(us, alg_bytes, elements):
        return {"us": round(us, 3), "elements_per_s": elements / (us * 1e-6), "alg_bytes": int(alg_bytes),
                "frac_of_hbm_peak": round(alg_bytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}

    acc = torch.empty(d, dtype=torch.float32, device=dev)
    e = torch.zeros(d, dtype=torch.float32, device=dev)
    out = torch.empty(d, dtype=torch.float32, device=dev)
    res = {}
    for kind, b in variants:
        lay = E.Layout(d, offs, density, b if kind == "randblock" else 1).bind(dev)
        K, L = lay.K, lay.n_seg
        block = kind == "randblock"
        mi = torch.empty((W, L if block else K), dtype=torch.int32, device=dev)
        mv = torch.empty((W, K), dtype=torch.float32, device=dev)
        ws = None if block else lay.workspace(E.EF_OP_TOPK if kind == "topk" else E.EF_OP_RANDK, 1, dev)
        ws_agg = None if block else lay.workspace(E.EF_OP_AGG_SPARSE, W, dev)
        kindm = E.EF_MSG_BLOCK if block else E.EF_MSG_SPARSE

        def fused(w=0):
            if kind == "topk":
                E.ef_step_topk(lay, g[w], e, mi[w], mv[w], ws)
            elif kind == "randk":
                E.ef_step_randk(lay, g[w], e, seeds[w], 0, mi[w], mv[w], ws)
            else:
                E.ef_step_randblock(lay, g[w], e, seeds[w], 0, mi[w], mv[w])

        def composed():
            E.ef_accumulate(lay, g[0], e, acc)
            if kind == "topk":
                E.compress_topk(lay, acc, mi[0], mv[0], ws)
            elif kind == "randk":
                E.compress_randk(lay, acc, seeds[0], 0, mi[0], mv[0], ws)
            else:
                E.compress_randblock(lay, acc, seeds[0], 0, mi[0], mv[0])
            E.ef_update(lay, acc, kindm, mi[0], e)

        step_b, agg_b = alg_bytes_op(kind, d, K, L, W)
        r = {"fused_step": entry(timed(fused), step_b, d)}
        if g_bf16 is not None:  # the same step on a bf16 gradient: 2 bytes fewer per element
            gb = g_bf16

            def fused_bf16():
                if kind == "topk":
                    E.ef_step_topk(lay, gb, e, mi[0], mv[0], ws)
                elif kind == "randk":
                    E.ef_step_randk(lay, gb, e, seeds[0], 0, mi[0], mv[0], ws)
                else:
                    E.ef_step_randblock(lay, gb, e, seeds[0], 0, mi[0], mv[0])

            r["fused_step_bf16_gradient"] = entry(timed(fused_bf16), step_b - 2 * d, d)
        # the step's kernels (library events per launch, a separate pass)
        E.timing_collect(reset=True)
        E.timing_enable(True)
        timed(fused)
        E.timing_enable(False)
        r["fused_step"]["kernels_us"] = {name: round(tot * 1e3 / nl, 3)
                                         for name, (tot, nl) in E.timing_collect(reset=True).items()}
        if ws is not None:  # the diagnostics word over every run of this step so far
            r["fused_step"]["diag"] = lay.diag(ws, E.EF_OP_TOPK if kind == "topk" else E.EF_OP_RANDK)
        # composed: the same algorithmic bytes (the intermediate acc costs 8d more by construction)
        r["composed_step"] = entry(timed(composed), step_b, d)
        if kind == "randk":
            r.update(measure_prepared(E, torch, dev, timed, entry, lay, g, e, seeds, mv, step_b, d))
        with torch.cuda.stream(st):
            for w in range(W):
                fused(w)
        r["aggregate"] = entry(timed(lambda: E.decompress_aggregate(lay, kindm, W, mi, mv, out, ws_agg)), agg_b, d)
        res[vname((kind, b))] = r
    none = torch.full((1,), d, dtype=torch.int32, device=dev)
    lay = E.Layout(d, [0, d], 1.0 / d, 1).bind(dev)  # k = 1: a one-entry message past the end zeroes nothing
    E.timing_collect(reset=True)
    E.timing_enable(True)
    timed(lambda: E.ef_update(lay, acc, E.EF_MSG_SPARSE, none, out))
    E.timing_enable(False)
    tot_ms, n = E.timing_collect(reset=True)["k_copy"]
    res["copy_ceiling"] = entry(tot_ms * 1e3 / n, 8 * d, d)
    res["copy_ceiling"]["kernel"] = "k_copy: read d floats, write d floats (per-launch events)"
    return res


def host_description():
    """The host the oracle runs on: logical CPUs, this process's affinity set and the CPU model."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    aff = sorted(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else None
    return {"os_cpu_count": os.cpu_count(), "affinity": aff, "cpu_model": model}


def cpu_baseline(wl, offs, ks, variants, W, grads, budget_note, min_s=10.0):
    """Time the CPU oracle on a bounded sample of worker steps plus one aggregate per variant,
    and scale to the GPU step's work (W steps + 1 aggregate per variant).  The oracle runs on one
    core: its process is pinned to one CPU of its affinity set and BLAS / OpenMP pools to one
    thread; the affinity is restored afterwards."""
    from oracle import efsparse_oracle as O
    from threadpoolctl import threadpool_limits
    host = host_description()
    old = set(host["affinity"]) if host["affinity"] else None
    pinned = None
    if old and hasattr(os, "sched_setaffinity"):
        pinned = min(old)
        os.sched_setaffinity(0, {pinned})
    try:
        with threadpool_limits(1):
            r = _cpu_baseline(O, wl, offs, ks, variants, W, grads, budget_note, min_s=min_s)
    finally:
        if pinned is not None:
            os.sched_setaffinity(0, old)
    r["host"] = dict(host, pinned_cpu=pinned)
    return r


def _cpu_baseline(O, wl, offs, ks, variants, W, grads, budget_note, min_s=10.0):
    """Workers 0, 1, ... (as many as it takes to pass min_s seconds, at most W) each run one
    fused step per variant; each variant also aggregates W copies of worker 0's message."""
    from workloads import worker_seed
    d = offs[-1]
    e0 = np.zeros(d, np.float32)
    t_steps = {v: [] for v in variants}
    t_aggs, parts, spent = {}, [], 0.0
    nw = 0
    while nw < W and (nw == 0 or spent < min_s):
        for kind, b in variants:
            t0 = time.perf_counter()
            (m, val), _ = O.ef_step(kind, grads[nw], e0, offs, ks, seed=worker_seed(wl, nw), step=0, block=b)
            t1 = time.perf_counter()
            t_steps[(kind, b)].append(t1 - t0)
            spent += t1 - t0
            if nw == 0:
                if kind == "randblock":
                    O.decompress_aggregate_block(d, offs, ks, [m] * W, [val] * W)
                else:
                    O.decompress_aggregate_sparse(d, [m] * W, [val] * W)
                t_aggs[(kind, b)] = time.perf_counter() - t1
                spent += t_aggs[(kind, b)]
        nw += 1
    est_step_s = 0.0
    for v in variants:
        mean = sum(t_steps[v]) / len(t_steps[v])
        est_step_s += W * mean + t_aggs[v]
        parts.append(f"{vname(v)} step {mean:.2f}s + aggregate {t_aggs[v]:.2f}s")
    value = len(variants) * W * d / est_step_s
    return {
        "value": value,
        "unit": "elements/s",
        "cores": 1,
        "kind": "oracle",
        "sample": (f"step 0 of workers 0..{nw - 1} of the same workload: one fused step per worker and "
                   f"variant, and one aggregate of W={W} messages per variant (means: {'; '.join(parts)}); "
                   f"scaled to the GPU step as W x step + aggregate per variant; NumPy, 1 thread{budget_note}"),
        "measured_s": round(spent, 2),
    }


def flat1g_gradient(torch, wl, w, out, gen, chunk=1 << 27):
    """Worker w's 1e9-element gradient drawn on the device (the host would need 4 GB and tens of
    seconds per worker): per element N(0, 1e-4) with probability 0.99, else N(0, 1e-1) (variances),
    from a torch generator seeded with (cfg_id << 32) | w.  Timing input only: parity tests use the
    host generator."""
    gen.manual_seed((wl.cfg_id << 32) | w)
    for a in range(0, out.numel(), chunk):
        part = out[a:a + chunk]
        part.normal_(generator=gen)
        wide = torch.empty_like(part).uniform_(generator=gen) < 0.01
        part.mul_(torch.where(wide, 0.1 ** 0.5, 1e-4 ** 0.5))


def measure_flat1g(args, E, torch, dev, reps=20):
    """The 1e9-element flat workload: for every density of the workload, one worker's fused step
    of each compressor (fp32 and bf16 gradient) and the aggregate of W = 32 workers' messages; for
    the block sizes 2^8 ... 2^20 at 1 %, the block-random-k step and its aggregate.  Messages come
    from 32 workers' own gradients (drawn on the device one after another); the timed steps use
    worker 0's gradient.  Back-to-back repetitions on one stream, each timed with events; the
    median repetition is reported."""
    from workloads import WORKLOADS, worker_seed
    wl = WORKLOADS["flat1g"]
    d, W = wl.d, args.workers or wl.W
    st = torch.cuda.Stream(dev)
    gen = torch.Generator(device=dev)

    def timed(fn):
        # the median of the repetitions' own durations (an event between each two): a one-off
        # stall of several ms inside one repetition moved a mean of 20 by 0.5 ms
        torch.cuda.synchronize()  # work enqueued on other streams first
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
        with torch.cuda.stream(st):
            for _ in range(3):
                fn()
            ev[0].record(st)
            for r in range(reps):
                fn()
                ev[r + 1].record(st)
        torch.cuda.synchronize()
        return statistics.median(ev[r].elapsed_time(ev[r + 1]) for r in range(reps)) * 1e3

    def split(fn):
        torch.cuda.synchronize()
        E.timing_collect(reset=True)
        E.timing_enable(True)
        with torch.cuda.stream(st):
            fn()
        torch.cuda.synchronize()
        E.timing_enable(False)
        return {n: round(t * 1e3 / c, 3) for n, (t, c) in E.timing_collect(reset=True).items()}

    def entry(us, alg):
        return {"us": round(us, 3), "elements_per_s": d / (us * 1e-6), "alg_bytes": int(alg),
                "frac_of_hbm_peak": round(alg / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}

    g0 = torch.empty(d, dtype=torch.float32, device=dev)
    flat1g_gradient(torch, wl, 0, g0, gen)
    gb = g0.to(torch.bfloat16)
    gw = torch.empty(d, dtype=torch.float32, device=dev)
    e = torch.zeros(d, dtype=torch.float32, device=dev)
    out = torch.empty(d, dtype=torch.float32, device=dev)
    seeds = [worker_seed(wl, w) for w in range(W)]

    def run_variant(kind, density, block):
        lay = E.Layout(d, [0, d], density, block).bind(dev)
        K, L = lay.K, lay.n_seg
        blk = kind == "randblock"
        op = E.EF_OP_TOPK if kind == "topk" else E.EF_OP_RANDK
        ws = None if blk else lay.workspace(op, 1, dev)
        mi = torch.empty((W, L if blk else K), dtype=torch.int32, device=dev)
        mv = torch.empty((W, K), dtype=torch.float32, device=dev)

        def step(g, w=0):
            if kind == "topk":
                E.ef_step_topk(lay, g, e, mi[w], mv[w], ws)
            elif kind == "randk":
                E.ef_step_randk(lay, g, e, seeds[w], 0, mi[w], mv[w], ws)
            else:
                E.ef_step_randblock(lay, g, e, seeds[w], 0, mi[w], mv[w])

        for w in range(W):  # the workers' messages, each from its own gradient and a zero residual
            flat1g_gradient(torch, wl, w, gw, gen)  # all on the current stream, in order
            e.zero_()
            step(gw, w)
        torch.cuda.synchronize()
        step_b, agg_b = alg_bytes_op(kind, d, K, L, W)
        ws_a = None if blk else lay.workspace(E.EF_OP_AGG_SPARSE, W, dev)
        kindm = E.EF_MSG_BLOCK if blk else E.EF_MSG_SPARSE
        agg = lambda: E.decompress_aggregate(lay, kindm, W, mi, mv, out, ws_a)  # noqa: E731
        r = {"K": K, "aggregate": entry(timed(agg), agg_b)}
        r["aggregate"]["kernels_us"] = split(agg)
        e.zero_()
        r["fused_step"] = entry(timed(lambda: step(g0)), step_b)
        r["fused_step"]["kernels_us"] = split(lambda: step(g0))
        e.zero_()
        r["fused_step_bf16_gradient"] = entry(timed(lambda: step(gb)), step_b - 2 * d)
        if ws is not None:
            r["fused_step"]["diag"] = lay.diag(ws, op)
        del ws, ws_a, mi, mv
        return r

    res = {"densities": {}, "blocks_at_1pct": {}}
    for density in wl.densities:
        _note(f"flat1g: density {density}")
        res["densities"][str(density)] = {f"{k}{b if k == 'randblock' else ''}": run_variant(k, density, b)
                                          for k, b in (("topk", 1), ("randk", 1), ("randblock", 4096))}
    for s in range(8, 21, 2):
        _note(f"flat1g: block 2^{s}")
        res["blocks_at_1pct"][f"2^{s}"] = run_variant("randblock", 0.01, 1 << s)
    cpu = None
    if not args.no_cpu_baseline:
        _note("CPU oracle sample (1e7 elements of the same distribution)")
        cpu = flat1g_cpu_sample(wl)
    line = {"metric": METRIC, "n_gpus": 1, "unit": "elements/s", "higher_is_better": True, "dtype": "f32",
            "data": "synthetic (drawn on the device)",
            "config": {"workload": f"flat1g: flat 1e9-element fp32 / bf16 gradients, densities "
                                   f"{list(wl.densities)}, block sizes 2^8..2^20, W={W} messages aggregated",
                       "d": d, "W": W},
            "flat1g": res, "cpu_baseline": cpu}
    print(json.dumps(line), flush=True)


def flat1g_cpu_sample(wl, n=10_000_000, density=0.01):
    """The oracle's worker step per compressor on a 1e7-element slice of the same distribution, one
    core (the full 1e9-element sort would take minutes per step)."""
    from oracle import efsparse_oracle as O
    from threadpoolctl import threadpool_limits
    from workloads import worker_seed
    rng = np.random.default_rng([wl.cfg_id, 0, 0])
    g = (rng.standard_normal(n) * np.where(rng.random(n) < 0.01, 0.1 ** 0.5, 1e-4 ** 0.5)).astype(np.float32)
    e0 = np.zeros(n, np.float32)
    offs = [0, n]
    ks = O.segment_ks(offs, density)
    out = {}
    with threadpool_limits(1):
        for kind, b in (("topk", 1), ("randk", 1), ("randblock", 4096)):
            t0 = time.perf_counter()
            O.ef_step(kind, g, e0, offs, ks, seed=worker_seed(wl, 0), step=0, block=b)
            out[kind] = {"s": round(time.perf_counter() - t0, 3), "elements_per_s": n / (time.perf_counter() - t0)}
    return {"kind": "oracle", "cores": 1, "sample": f"one worker step per compressor on {n} elements at "
            f"density {density}, NumPy, 1 thread", "per_compressor": out, "host": host_description()}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="resnet50")
    ap.add_argument("--scope", default="flat", choices=["flat", "layer"])
    ap.add_argument("--density", type=float, default=None)
    ap.add_argument("--workers", type=int, default=None)
    ap.add_argument("--variants", default="topk,randk,randblock")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kernel-timing", action="store_true")
    ap.add_argument("--no-single", action="store_true", help="skip the one-worker step and aggregate "
                    "measurements per compressor at flat and per-layer scope")
    ap.add_argument("--no-next", action="store_true", help="skip the shared-coordinate, fused-update and "
                    "dense-average measurements")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="N",
                    help="first launch the library's plain copy kernel N times on d floats (a known "
                         "4d-byte read + 4d-byte write per launch) to calibrate HBM byte counters")
    ap.add_argument("--schedule", default="batch", choices=["batch", "fused", "pipelined"],
                    help="batch: each variant's W top-k / random-k steps in one ef_step_*_batch call; "
                         "fused: each top-k / random-k worker step on one of --worker-streams streams; "
                         "pipelined: its phases split over a streaming stream and two selection streams")
    ap.add_argument("--worker-streams", type=int, default=3)
    ap.add_argument("--streams", type=int, default=3,
                    help="workspace slots: top-k / random-k worker steps in flight at once (pipelined: at "
                         "least 4)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU only: --gpus {args.gpus} is not supported "
              "(the library has no multi-GPU path; the value is one GPU's share of the data-parallel step).",
              file=sys.stderr)
        sys.exit(2)

    if args.workload == "flat1g":  # 4 GB per array: a sweep of one-worker steps and 32-worker aggregates
        import torch
        import paper_2009_09271_amd as E
        dev = torch.device("cuda", 0)
        torch.cuda.set_device(dev)
        return measure_flat1g(args, E, torch, dev)

    from workloads import WORKLOADS, worker_seed
    wl = WORKLOADS[args.workload]
    W = args.workers or wl.W
    density = args.density or wl.densities[0]
    variants = variant_list(args.variants, wl.blocks)
    offs = wl.seg_offsets(args.scope)
    d = offs[-1]

    _note(f"generating {W} gradients of {d} elements")
    t_gen = time.perf_counter()
    grads = gen_gradients(wl, W)
    t_gen = time.perf_counter() - t_gen

    import torch
    import paper_2009_09271_amd as E

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    layouts = {}
    for kind, b in variants:
        key = b if kind == "randblock" else 1
        if key not in layouts:
            layouts[key] = E.Layout(d, offs, density, key).bind(dev)
    lay0 = next(iter(layouts.values()))
    K, L = lay0.K, lay0.n_seg

    # one allocation per worker: streaming over rows of one [W][d] stack of 1.6 GB measured slower
    # (53 against 47 us per pass) whatever the row padding
    g = [torch.from_numpy(x).to(dev) for x in grads]
    if args.calibrate_copy:
        src_c = torch.randn(d, device=dev)
        dst_c = torch.empty(d, device=dev)
        none = torch.full((K,), d, dtype=torch.int32, device=dev)  # out-of-range: nothing zeroed
        for _ in range(args.calibrate_copy):
            E.ef_update(lay0, src_c, E.EF_MSG_SPARSE, none, dst_c)
        torch.cuda.synchronize()
        del src_c, dst_c, none
    e = {vname(v): [torch.zeros(d, dtype=torch.float32, device=dev) for _ in range(W)] for v in variants}
    # two message buffers per variant, alternating by step, so that a step's aggregate can run while
    # the next step's workers write their messages
    msg_bufs = {}
    for v in variants:
        n_m = L if v[0] == "randblock" else K
        msg_bufs[vname(v)] = [(torch.empty((W, n_m), dtype=torch.int32, device=dev),
                               torch.empty((W, K), dtype=torch.float32, device=dev)) for _ in range(2)]
    msg = {k: b[0] for k, b in msg_bufs.items()}  # the current step's buffers (set by run_step)
    out = {vname(v): torch.empty(d, dtype=torch.float32, device=dev) for v in variants}
    # workspace slots of the top-k / random-k steps in flight
    S = max(4, args.streams) if args.schedule == "pipelined" else max(1, args.streams)
    kinds = {k for k, _ in variants}
    ws_topk = [lay0.workspace(E.EF_OP_TOPK, 1, dev) for _ in range(S)] if "topk" in kinds else None
    ws_randk = [lay0.workspace(E.EF_OP_RANDK, 1, dev) for _ in range(S)] if "randk" in kinds else None
    ws_agg = lay0.workspace(E.EF_OP_AGG_SPARSE, W, dev)
    wsb = {}
    if args.schedule == "batch":
        for k, op in (("topk", E.EF_OP_TOPK), ("randk", E.EF_OP_RANDK)):
            if k in kinds:
                wsb[k] = E.batch_workspace(lay0, op, W, dev)
    # stream A: the streaming passes; streams B0 / B1: the selection phases of even / odd workers;
    # one stream for the aggregates (all at the default priority)
    sA, astream = torch.cuda.Stream(dev), torch.cuda.Stream(dev)
    sB = [torch.cuda.Stream(dev), torch.cuda.Stream(dev)]

    # events reused every step (a wait takes the event's latest record at the time it is enqueued)
    evs = {vname(v): [[torch.cuda.Event() for _ in range(W)] for _ in range(3)] for v in variants}

    def phase(v, w, t, p, st):
        kind, _ = v
        mi, mv = msg[vname(v)]
        ev = e[vname(v)]
        if kind == "topk":
            E.ef_step_topk_phases(lay0, p, g[w], ev[w], mi[w], mv[w], ws_topk[w % S], stream=st)
        else:
            E.ef_step_randk_phases(lay0, p, g[w], ev[w], worker_seed(wl, w), t, mi[w], mv[w], ws_randk[w % S],
                                   stream=st)

    def aggregate(v, st):
        kind, b = v
        lay = layouts[b if kind == "randblock" else 1]
        mi, mv = msg[vname(v)]
        kindm = E.EF_MSG_BLOCK if kind == "randblock" else E.EF_MSG_SPARSE
        E.decompress_aggregate(lay, kindm, W, mi, mv, out[vname(v)], ws_agg if kindm == E.EF_MSG_SPARSE else None,
                               stream=st)

    wstreams = [torch.cuda.Stream(dev) for _ in range(args.worker_streams)]

    def run_step_fused(t, vs):
        """Top-k / random-k workers run their fused step, worker w on worker stream w % n; each
        variant's aggregate waits for all of them on its own stream."""
        cur = torch.cuda.current_stream(dev)
        for st in wstreams + [sA, astream]:
            st.wait_stream(cur)
        for v in vs:
            kind, b = v
            mi, mv = msg[vname(v)]
            ev = e[vname(v)]
            if kind == "randblock":
                for w in range(W):
                    E.ef_step_randblock(layouts[b], g[w], ev[w], worker_seed(wl, w), t, mi[w], mv[w], stream=sA)
                astream.wait_stream(sA)
                aggregate(v, astream)
                continue
            n = len(wstreams)
            for w in range(W):
                st = wstreams[w % n]
                ws = ws_topk[w % S] if kind == "topk" else ws_randk[w % S]
                if w >= S and S % n:  # the workspace slot of worker w - S (same stream when n divides S)
                    st.wait_event(evs[vname(v)][2][w - S])
                if kind == "topk":
                    E.ef_step_topk_phases(lay0, E.EF_PHASE_ALL, g[w], ev[w], mi[w], mv[w], ws, stream=st)
                else:
                    E.ef_step_randk_phases(lay0, E.EF_PHASE_ALL, g[w], ev[w], worker_seed(wl, w), t, mi[w], mv[w],
                                           ws, stream=st)
                if w + S < W and (S % n):
                    evs[vname(v)][2][w].record(st)
            for st in wstreams:
                astream.wait_stream(st)
            aggregate(v, astream)
        for st in wstreams + [sA, astream]:
            cur.wait_stream(st)

    def run_step_serial(t, vs):
        """Every worker step and aggregate one after another on stream A (per-kernel durations
        without concurrency)."""
        cur = torch.cuda.current_stream(dev)
        sA.wait_stream(cur)
        for v in vs:
            kind, b = v
            mi, mv = msg[vname(v)]
            ev = e[vname(v)]
            for w in range(W):
                if kind == "randblock":
                    E.ef_step_randblock(layouts[b], g[w], ev[w], worker_seed(wl, w), t, mi[w], mv[w], stream=sA)
                elif kind == "topk":
                    E.ef_step_topk_phases(lay0, E.EF_PHASE_ALL, g[w], ev[w], mi[w], mv[w], ws_topk[0], stream=sA)
                else:
                    E.ef_step_randk_phases(lay0, E.EF_PHASE_ALL, g[w], ev[w], worker_seed(wl, w), t, mi[w], mv[w],
                                           ws_randk[0], stream=sA)
            aggregate(v, sA)
        cur.wait_stream(sA)

    seeds = [worker_seed(wl, w) for w in range(W)]

    agg_done = [torch.cuda.Event(), torch.cuda.Event()]

    def run_step_batch(t, vs):
        """Each variant's W worker steps on stream A, one after another (block-random-k: W one-kernel
        steps; top-k / random-k: one ef_step_*_batch call, whose streaming passes run back to back and
        whose selection kernels run once for all W workers).  Each variant's aggregate runs on a
        second stream, overlapping the next variant's workers; message buffers alternate by step, and
        a step's workers only wait for the aggregates of two steps before."""
        sA.wait_event(agg_done[t % 2])
        for v in vs:
            kind, b = v
            mi, mv = msg[vname(v)]
            ev = e[vname(v)]
            if kind == "randblock":
                for w in range(W):
                    E.ef_step_randblock(layouts[b], g[w], ev[w], seeds[w], t, mi[w], mv[w], stream=sA)
            elif kind == "topk":
                E.ef_step_topk_batch(lay0, g, ev, mi, mv, wsb["topk"][0], wsb["topk"][1], stream=sA)
            else:
                E.ef_step_randk_batch(lay0, g, ev, seeds, t, mi, mv, wsb["randk"][0], wsb["randk"][1], stream=sA)
            astream.wait_stream(sA)
            aggregate(v, astream)
        agg_done[t % 2].record(astream)

    def run_variant_alone(t, v):
        """One variant by itself: its W worker steps and its aggregate, all on stream A."""
        kind, b = v
        mi, mv = msg[vname(v)]
        ev = e[vname(v)]
        if kind == "randblock":
            for w in range(W):
                E.ef_step_randblock(layouts[b], g[w], ev[w], seeds[w], t, mi[w], mv[w], stream=sA)
        elif kind == "topk":
            E.ef_step_topk_batch(lay0, g, ev, mi, mv, wsb["topk"][0], wsb["topk"][1], stream=sA)
        else:
            E.ef_step_randk_batch(lay0, g, ev, seeds, t, mi, mv, wsb["randk"][0], wsb["randk"][1], stream=sA)
        aggregate(v, sA)

    def run_step(t, vs=None):
        vs = vs or variants
        schedule = args.schedule
        for k, bufs in msg_bufs.items():
            msg[k] = bufs[t % 2]
        if schedule == "batch":
            return run_step_batch(t, vs)
        if schedule == "fused":
            return run_step_fused(t, vs)
        return run_step_pipelined(t, vs)

    def run_step_pipelined(t, vs):
        """Top-k / random-k workers run their fused step in three phases (ef_step_*_phases): the
        streaming passes follow each other on stream A, while streams B0 / B1 (even / odd workers)
        run the selection phases around them, each worker's prepare two workers ahead of its
        stream pass.  Block-random-k workers are one streaming kernel each on stream A."""
        cur = torch.cuda.current_stream(dev)
        for st in [sA, astream] + sB:
            st.wait_stream(cur)
        for v in vs:
            kind, b = v
            if kind == "randblock":
                mi, mv = msg[vname(v)]
                ev = e[vname(v)]
                for w in range(W):
                    E.ef_step_randblock(layouts[b], g[w], ev[w], worker_seed(wl, w), t, mi[w], mv[w], stream=sA)
                astream.wait_stream(sA)
                aggregate(v, astream)
                continue
            prep = kind == "topk"  # random-k has nothing to prepare
            ready, done, fin = evs[vname(v)]

            def prepare(w):
                if prep and w < W:
                    phase(v, w, t, E.EF_PHASE_PREPARE, sB[w % 2])
                    ready[w].record(sB[w % 2])

            prepare(0)
            prepare(1)
            for w in range(W):
                sb = sB[w % 2]
                prepare(w + 2)  # its slot was last used by worker w - 2, finished earlier on sb
                if prep:
                    sA.wait_event(ready[w])
                elif w >= S:  # the workspace slot is free once the step that used it finished
                    sA.wait_event(fin[w - S])
                phase(v, w, t, E.EF_PHASE_STREAM, sA)
                done[w].record(sA)
                sb.wait_event(done[w])
                phase(v, w, t, E.EF_PHASE_FINISH, sb)
                fin[w].record(sb)
            for sb in sB:
                astream.wait_stream(sb)
            aggregate(v, astream)
        for st in [sA, astream] + sB:
            cur.wait_stream(st)

    _note(f"warm-up ({args.warmup} steps), then {args.steps} timed steps")
    step_no = 0
    with torch.cuda.stream(sA):
        for _ in range(args.warmup):
            run_step(step_no)
            step_no += 1
    torch.cuda.synchronize()

    # ---- timed region: exactly `steps` steps --------------------------------------------------
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    with torch.cuda.stream(sA):
        for _ in range(args.steps):
            run_step(step_no)
            step_no += 1
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_per_step = elapsed * 1e3 / args.steps
    elems_per_step = len(variants) * W * d
    value = elems_per_step / (ms_per_step / 1e3)

    # diagnostics words of the top-k / random-k workspaces, OR-ed over every worker and every step
    # so far (warm-up and timed): bit 1 = a segment took the exact whole-segment path, bit 3 = a top-k
    # segment collected its candidates again at a lower threshold, bit 2 = a row-count mismatch
    # (never expected)
    diagnostics = {}
    for k, op in (("topk", E.EF_OP_TOPK), ("randk", E.EF_OP_RANDK)):
        if k not in kinds:
            continue
        rows = [wsb[k][0][w] for w in range(W)] if args.schedule == "batch" else \
            (ws_topk if k == "topk" else ws_randk)
        word = 0
        for r in rows:
            word |= lay0.diag(r, op)
        diagnostics[k] = {"word": word, "exact_path_taken": bool(word & E.DIAG_SLOW_PATH),
                          "candidate_retry": bool(word & E.DIAG_RETRY),
                          "count_mismatch": bool(word & E.DIAG_COUNT_MISMATCH)}

    # ---- per-variant breakdown: each variant alone (batch schedule: its W steps and aggregate on
    # one stream; other schedules: their own schedule with one variant) -------------------------
    _note("each variant alone")
    per = {}
    for v in variants:
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        with torch.cuda.stream(sA):
            for _ in range(args.steps):
                if args.schedule == "batch":
                    for k, bufs in msg_bufs.items():
                        msg[k] = bufs[step_no % 2]
                    run_variant_alone(step_no, v)
                else:
                    run_step(step_no, [v])
                step_no += 1
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t1) * 1e3 / args.steps
        step_b, agg_b = alg_bytes_op(v[0], d, K, L, W)
        per[vname(v)] = {
            "ms_per_step": round(ms, 4),
            "elements_per_s": W * d / (ms / 1e3),
            "alg_GB_per_step": round((W * step_b + agg_b) / 1e9, 4),
            "alg_GBps": round((W * step_b + agg_b) / (ms / 1e3) / 1e9, 1),
            "frac_of_hbm_peak": round((W * step_b + agg_b) / (ms / 1e3) / 1e9 / HBM_PEAK_GBS, 4),
        }

    # ---- per-kernel durations from library-recorded HIP events ---------------------------------
    # (1) the same schedule as the timed steps (the roofline kernel's launches); (2) per variant,
    # its W steps and aggregate alone on one stream (each kernel's duration without concurrency)
    def kernel_table(run_one):
        E.timing_collect(reset=True)
        E.timing_enable(True)
        with torch.cuda.stream(sA):
            for _ in range(args.steps):
                t = nonlocal_step[0]
                for k, bufs in msg_bufs.items():
                    msg[k] = bufs[t % 2]
                run_one(t)
                nonlocal_step[0] = t + 1
        torch.cuda.synchronize()
        E.timing_enable(False)
        tm = E.timing_collect(reset=True)
        table = {}
        for name, (tot_ms, n) in sorted(tm.items(), key=lambda kv: -kv[1][0]):
            avg_us = tot_ms * 1e3 / n
            ab = kernel_alg_bytes(name, d, K, L, W)
            table[name] = {"avg_us": round(avg_us, 3), "launches": n, "total_ms": round(tot_ms, 3)}
            if ab is not None:
                table[name]["alg_bytes"] = ab
                table[name]["alg_GBps"] = round(ab / (avg_us * 1e-6) / 1e9, 1)
                table[name]["frac"] = round(ab / (avg_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)
        return table

    def alone(v):
        if args.schedule == "batch":
            return lambda t: run_variant_alone(t, v)
        return lambda t: run_step_serial(t, [v])

    nonlocal_step = [step_no]
    kernels, kernels_serial, roofline = {}, {}, None
    if not args.no_kernel_timing:
        _note("per-kernel timing")
        kernels = kernel_table(lambda t: run_step(t))
        kernels_serial = {vname(v): kernel_table(alone(v)) for v in variants}
        dom = next(iter(kernels))
        ab = kernel_alg_bytes(dom, d, K, L, W)
        if ab is not None:
            from paper_2009_09271_amd.rocprof_summary import read_traffic
            achieved = ab / (kernels[dom]["avg_us"] * 1e-6) / 1e9
            base = dom.strip("(").split("<")[0]
            tfile = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles",
                                 f"{base}_{wl.name}_{args.scope}_traffic.md")
            traffic = read_traffic(tfile, base)
            roofline = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                        "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                        "traffic": round(traffic) if traffic is not None else None,
                        "alg_bytes_per_launch": ab, "avg_launch_us": kernels[dom]["avg_us"],
                        "traffic_source": os.path.relpath(tfile, os.path.dirname(os.path.abspath(__file__)))
                        if traffic is not None else None}

    # ---- each compressor alone, one worker's step and one aggregate, at both scopes ---------------
    single = {}
    if not args.no_single:
        g_bf16 = g[0].to(torch.bfloat16)
        for scope in ("flat", "layer"):
            _note(f"one worker's step and the aggregate alone, {scope} scope")
            single[scope] = measure_single(E, torch, dev, wl.seg_offsets(scope), density, variants, W, g,
                                           seeds, g_bf16=g_bf16 if scope == "flat" else None)
        del g_bf16

    # ---- the paths next to the hot path, on the same workload (each alone, events on one stream) --
    if not args.no_next:
        _note("next rows")
    nxt = {} if args.no_next else measure_next(E, torch, dev, wl, lay0, layouts, msg, variants, W, d, K, L, args)

    # each compressor's own fraction of the HBM roofline, next to the dominant kernel's: its W
    # batched steps plus aggregate, one worker's lone fused step and the aggregate alone
    per_roof = {}
    for v in variants:
        n = vname(v)
        ent = {"batched_steps_and_aggregate": per[n]["frac_of_hbm_peak"]}
        for scope, sres in single.items():
            ent[f"lone_step_{scope}"] = sres[n]["fused_step"]["frac_of_hbm_peak"]
            ent[f"aggregate_{scope}"] = sres[n]["aggregate"]["frac_of_hbm_peak"]
        per_roof[n] = ent

    cpu = None
    if not args.no_cpu_baseline:
        _note("CPU oracle sample")
        ks = [int(k) for k in lay0.segment_k()]
        cpu = cpu_baseline(wl, offs, ks, variants, W, grads, "")

    line = {
        "metric": METRIC,
        "value": value,
        "unit": "elements/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": (f"{wl.name}-shaped fp32 gradients ({len(wl.seg_offsets('layer')) - 1} tensors), "
                         f"{args.scope} scope, d={d}, density {density}, W={W}, variants "
                         f"{'/'.join(vname(v) for v in variants)}, one fused step per worker per variant "
                         f"+ one aggregate per variant per step"),
            "d": d, "segments": L, "K": K, "W": W, "density": density,
            "variants": [vname(v) for v in variants], "scope": args.scope,
            "schedule": {"batch": "each variant's W steps on one stream (top-k / random-k: one ef_step_*_batch "
                                  "call); aggregates on a second stream",
                         "fused": f"top-k / random-k worker steps on {args.worker_streams} streams; aggregates "
                                  "on another",
                         "pipelined": "streaming phases on one stream, selection phases on two more, aggregates "
                                      "on another"}[args.schedule],
        },
        "roofline": roofline,
        "per_compressor_roofline": per_roof,
        "diagnostics": diagnostics,
        "cpu_baseline": cpu,
        "per_compressor": per,
        "kernels": kernels,
        "kernels_serial": kernels_serial,
        "single": single,
        "next_rows": nxt,
        "input_generation_s": round(t_gen, 2),
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
