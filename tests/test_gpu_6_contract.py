"""GPU contract tests of the C ABI on a bound layout: the entry points enqueue and return without
waiting for the device (no host synchronisation), and bad workspaces or misaligned pointers are
rejected with their status codes before anything is enqueued."""

import time

import numpy as np
import pytest

from efs_gpu import Case, announce, dev, host

pytestmark = pytest.mark.gpu


def _busy_queue(a, n=8):
    """Enqueue about 0.1 s of matrix products on the current stream."""
    for _ in range(n):
        a = a @ a * 1e-4
    return a


def test_entry_points_do_not_synchronise():
    """Each call returns while a long product enqueued before it is still running."""
    import paper_2009_09271_amd as E
    import torch
    announce("no host synchronisation")
    c = Case([0, 100000, 250001], 0.01, 256)
    cs = Case([0, 100000, 250001], 0.01)
    d, K, L, W = c.d, c.K, len(c.ks), 4
    rng = np.random.default_rng(1)
    g = dev((rng.standard_normal(d) * 0.01).astype(np.float32))
    e = torch.zeros(d, dtype=torch.float32, device="cuda")
    acc = torch.empty_like(e)
    out = torch.empty_like(e)
    x = torch.zeros_like(e)
    idx = torch.empty((W, K), dtype=torch.int32, device="cuda")
    val = torch.empty((W, K), dtype=torch.float32, device="cuda")
    start = torch.zeros((W, L), dtype=torch.int32, device="cuda")
    ws_t, ws_r = cs.ws(E.EF_OP_TOPK), cs.ws(E.EF_OP_RANDK)
    ws_p, ws_p2 = cs.ws(E.EF_OP_RANDK_PREP), cs.ws(E.EF_OP_RANDK_PREP)
    idx_p, idx_p2 = (torch.empty(K, dtype=torch.int32, device="cuda") for _ in range(2))
    idx_pb = torch.empty((W, K), dtype=torch.int32, device="cuda")
    ws_a = cs.ws(E.EF_OP_AGG_SPARSE, W)
    ws_s = cs.ws(E.EF_OP_AGG_SHARED, W)
    wsb, stride = E.batch_workspace(cs.L, E.EF_OP_RANDK, W)
    wsbp, stridep = E.batch_workspace(cs.L, E.EF_OP_RANDK_PREP, W)
    gl = [g] * W
    el = [torch.zeros_like(e) for _ in range(W)]
    G = torch.zeros((W, d), dtype=torch.float32, device="cuda")
    E.ef_randk_prepare(cs.L, 5, 0, idx_p, ws_p)  # the selection the prepared step below uses
    calls = {
        "ef_accumulate": lambda: E.ef_accumulate(c.L, g, e, acc),
        "compress_topk": lambda: E.compress_topk(cs.L, acc, idx[0], val[0], ws_t),
        "compress_randk": lambda: E.compress_randk(cs.L, acc, 5, 0, idx[0], val[0], ws_r),
        "compress_randblock": lambda: E.compress_randblock(c.L, acc, 5, 0, start[0], val[0]),
        "ef_update": lambda: E.ef_update(cs.L, acc, E.EF_MSG_SPARSE, idx[0], e),
        "ef_step_topk": lambda: E.ef_step_topk(cs.L, g, e, idx[0], val[0], ws_t),
        "ef_step_randk": lambda: E.ef_step_randk(cs.L, g, e, 5, 0, idx[0], val[0], ws_r),
        "ef_step_randblock": lambda: E.ef_step_randblock(c.L, g, e, 5, 0, start[0], val[0]),
        "ef_step_randk_batch": lambda: E.ef_step_randk_batch(cs.L, gl, el, [1, 2, 3, 4], 0, idx, val, wsb, stride),
        "ef_randk_prepare": lambda: E.ef_randk_prepare(cs.L, 5, 1, idx_p2, ws_p2),
        "ef_randk_prepare_batch": lambda: E.ef_randk_prepare_batch(cs.L, [1, 2, 3, 4], 0, idx_pb, wsbp, stridep),
        "ef_step_randk_prepared": lambda: E.ef_step_randk_prepared(cs.L, g, e, idx_p, val[0], ws_p),
        "decompress_aggregate sparse": lambda: E.decompress_aggregate(cs.L, E.EF_MSG_SPARSE, W, idx, val, out,
                                                                      ws_a),
        "decompress_aggregate block": lambda: E.decompress_aggregate(c.L, E.EF_MSG_BLOCK, W, start, val, out),
        "decompress_aggregate_apply": lambda: E.decompress_aggregate_apply(c.L, E.EF_MSG_BLOCK, W, start, val, x),
        "decompress_aggregate_shared": lambda: E.decompress_aggregate_shared(cs.L, E.EF_MSG_SPARSE, W, idx[0],
                                                                             val, out, ws_s),
        "ef_dense_average": lambda: E.ef_dense_average(c.L, W, G, out),
    }
    for fn in calls.values():  # first calls (library and module set-up) outside the check
        fn()
    torch.cuda.synchronize()
    a = torch.randn(4096, 4096, device="cuda")
    stream = torch.cuda.current_stream()
    for name, fn in calls.items():
        torch.cuda.synchronize()
        _busy_queue(a)
        t0 = time.perf_counter()
        fn()
        dt = time.perf_counter() - t0
        busy = not stream.query()
        torch.cuda.synchronize()
        assert busy, f"{name}: the stream had drained when the call returned ({dt * 1e3:.1f} ms)"


def test_bad_workspaces_and_pointers_are_rejected_before_launch():
    import paper_2009_09271_amd as E
    import torch
    announce("status codes on a bound layout")
    c = Case([0, 5000, 20001], 0.01)
    d, K, W = c.d, c.K, 3
    g = torch.zeros(d, dtype=torch.float32, device="cuda")
    e = torch.zeros(d + 4, dtype=torch.float32, device="cuda")
    idx = torch.full((W, K), 7, dtype=torch.int32, device="cuda")
    val = torch.full((W, K), 3.0, dtype=torch.float32, device="cuda")
    out = torch.full((d,), 5.0, dtype=torch.float32, device="cuda")

    def code(fn):
        with pytest.raises(E.EfError) as ex:
            fn()
        return ex.value.code

    for op, call in ((E.EF_OP_TOPK, lambda ws: E.ef_step_topk(c.L, g, e[:d], idx[0], val[0], ws)),
                     (E.EF_OP_RANDK, lambda ws: E.ef_step_randk(c.L, g, e[:d], 1, 0, idx[0], val[0], ws)),
                     (E.EF_OP_RANDK_PREP, lambda ws: E.ef_randk_prepare(c.L, 1, 0, idx[0], ws)),
                     (E.EF_OP_RANDK_PREP, lambda ws: E.ef_step_randk_prepared(c.L, g, e[:d], idx[0], val[0], ws))):
        n = c.L.workspace_bytes(op, 1)
        full = torch.zeros(n + 256, dtype=torch.uint8, device="cuda")
        assert code(lambda: call(full[:n - 4])) == E.EF_EWORKSPACE
        assert code(lambda: call(full[1:n + 1])) == E.EF_EINVAL  # base not 256-byte aligned
    ws = c.ws(E.EF_OP_TOPK)
    assert code(lambda: E.ef_step_topk(c.L, g, e[1:d + 1], idx[0], val[0], ws)) == E.EF_EINVAL  # e not 16-aligned
    assert code(lambda: E.ef_step_topk(c.L, g[1:], e[:d - 1], idx[0], val[0], ws)) == E.EF_EINVAL
    n = c.L.workspace_bytes(E.EF_OP_AGG_SPARSE, W)
    wa = torch.zeros(n, dtype=torch.uint8, device="cuda")
    assert code(lambda: E.decompress_aggregate(c.L, E.EF_MSG_SPARSE, W, idx, val, out, None)) == E.EF_EINVAL
    assert code(lambda: E.decompress_aggregate(c.L, E.EF_MSG_SPARSE, W, idx, val, out, wa[:n - 4])) == \
        E.EF_EWORKSPACE
    assert code(lambda: E.decompress_aggregate(c.L, 9, W, idx, val, out, wa)) == E.EF_EINVAL
    assert code(lambda: E.ef_randk_prepare_batch(c.L, [], 0, idx, wa, 256)) == E.EF_ERANGE
    torch.cuda.synchronize()
    # nothing was enqueued: the outputs still hold their fill values
    assert torch.all(out == 5.0) and torch.all(val == 3.0) and torch.all(idx == 7)


@pytest.mark.parametrize("kind", ["topk", "randk"])
def test_same_step_in_every_launch_configuration(kind):
    """One worker's step gives the same bits alone (one row per wavefront), as the first worker of
    batches of 3 and of 12 (the batch forms for 8 or more workers: four rows per wavefront, the
    worker in the grid's second dimension), split into phases, and for random-k prepared ahead."""
    import paper_2009_09271_amd as E
    import torch
    announce("launch configurations", kind)
    c = Case([0, 5, 70000, 70004, 300000], 0.01)
    rng = np.random.default_rng(3)
    g = dev((rng.standard_normal(c.d) * 10.0 ** rng.integers(-3, 1, c.d)).astype(np.float32))
    e0 = dev((rng.standard_normal(c.d) * 1e-3).astype(np.float32))
    op = E.EF_OP_TOPK if kind == "topk" else E.EF_OP_RANDK
    seed = 41

    def single(phased):
        e = e0.clone()
        idx = torch.empty(c.K, dtype=torch.int32, device="cuda")
        val = torch.empty(c.K, dtype=torch.float32, device="cuda")
        ws = c.ws(op)
        phases = [E.EF_PHASE_PREPARE, E.EF_PHASE_STREAM, E.EF_PHASE_FINISH] if phased else [E.EF_PHASE_ALL]
        for p in phases:
            if kind == "topk":
                E.ef_step_topk_phases(c.L, p, g, e, idx, val, ws)
            else:
                E.ef_step_randk_phases(c.L, p, g, e, seed, 0, idx, val, ws)
        return idx, val, e

    def batch(W):
        es = [e0.clone() for _ in range(W)]
        idx = torch.empty((W, c.K), dtype=torch.int32, device="cuda")
        val = torch.empty((W, c.K), dtype=torch.float32, device="cuda")
        ws, stride = E.batch_workspace(c.L, op, W)
        if kind == "topk":
            E.ef_step_topk_batch(c.L, [g] * W, es, idx, val, ws, stride)
        else:
            E.ef_step_randk_batch(c.L, [g] * W, es, [seed] * W, 0, idx, val, ws, stride)
        return idx[0], val[0], es[0]

    runs = {"alone": single(False), "phases": single(True), "batch of 3": batch(3), "batch of 12": batch(12)}
    if kind == "randk":
        e = e0.clone()
        idx = torch.empty(c.K, dtype=torch.int32, device="cuda")
        val = torch.empty(c.K, dtype=torch.float32, device="cuda")
        ws = c.ws(E.EF_OP_RANDK_PREP)
        E.ef_randk_prepare(c.L, seed, 0, idx, ws)
        E.ef_step_randk_prepared(c.L, g, e, idx, val, ws)
        runs["prepared"] = (idx, val, e)
    ref = [host(t).view(np.uint32) for t in runs["alone"]]
    for name, r in runs.items():
        for got, want, what in zip(r, ref, ("indices", "values", "residual")):
            assert np.array_equal(host(got).view(np.uint32), want), f"{kind} {name}: {what} differ"
