"""GPU parity on seeded random configurations: random segment layouts (1 to 40 segments, sizes
from 1 element up), densities, block sizes, worker counts and gradient dtypes.  For each, the
fused steps of every compressor over two steps (residual carried), the batched steps, random-k
prepared ahead, and the sparse and block aggregates of the workers' messages (plain, fused with a
parameter update, and with shared coordinates), bit for bit against the CPU oracle."""

import numpy as np
import pytest

from efs_gpu import Case, announce, assert_f32_equal, assert_msg_equal, dev, host
from oracle import efsparse_oracle as O

pytestmark = pytest.mark.gpu


def _config(i):
    rng = np.random.default_rng([2009, 9271, i])
    n_seg = int(rng.integers(1, 41))
    sizes = np.where(rng.random(n_seg) < 0.3, rng.integers(1, 64, n_seg), rng.integers(64, 40000, n_seg))
    offs = [0] + np.cumsum(sizes).tolist()
    density = float(rng.choice([0.001, 0.01, 0.05, 0.3, 1.0]))
    block = int(rng.choice([1, 2, 7, 256, 4096]))
    W = int(rng.integers(1, 13))
    bf16 = bool(rng.random() < 0.3)
    scales = 10.0 ** rng.uniform(-4, 0, n_seg)
    return rng, offs, density, block, W, bf16, scales


def _gradients(rng, offs, scales, W, bf16):
    from workloads import to_bf16_bits
    d = offs[-1]
    G = np.empty((W, d), np.float32)
    for w in range(W):
        x = rng.laplace(0.0, 1.0, d)
        for l in range(len(offs) - 1):
            x[offs[l]:offs[l + 1]] *= scales[l]
        x[rng.random(d) < 0.05] = 0.0  # exact zeros: ties at the threshold
        G[w] = x.astype(np.float32)
    if bf16:
        G = np.stack([to_bf16_bits(x) for x in G])
    return G


def _dev_g(x):
    import torch
    t = dev(x)
    return t.view(torch.bfloat16) if x.dtype == np.uint16 else t


@pytest.mark.parametrize("i", range(64))
def test_random_configuration(i):
    import paper_2009_09271_amd as E
    import torch
    rng, offs, density, block, W, bf16, scales = _config(i)
    announce("random configuration", i, len(offs) - 1, offs[-1], density, block, W, bf16)
    G = _gradients(rng, offs, scales, W, bf16)
    seeds = [(int(rng.integers(0, 2**31)) << 32) | w for w in range(W)]
    for kind in ("topk", "randk", "randblock"):
        c = Case(offs, density, block if kind == "randblock" else 1)
        e = np.zeros((W, c.d), np.float32)
        msgs = []
        for step in range(2):
            msgs = []
            for w in range(W):
                ed = dev(e[w])
                m, val, _ = c.step(kind, G[w], ed, seeds[w], step)
                (wm, wv), we = c.oracle_step(kind, G[w], e[w], seeds[w], step)
                assert_msg_equal(kind, (m, val), (wm, wv), f"cfg {i} {kind} w{w} step {step}")
                assert_f32_equal(ed, we, f"cfg {i} {kind} e' w{w} step {step}")
                e[w] = we
                msgs.append((wm, wv))
        # the aggregate of the last step's messages
        out = torch.empty(c.d, dtype=torch.float32, device="cuda")
        mi = dev(np.stack([m for m, _ in msgs]).astype(np.uint32).view(np.int32))
        mv = dev(np.stack([v for _, v in msgs]))
        if kind == "randblock":
            E.decompress_aggregate(c.L, E.EF_MSG_BLOCK, W, mi, mv, out, None)
            want = O.decompress_aggregate_block(c.d, c.offs, c.ks, [m for m, _ in msgs], [v for _, v in msgs])
        else:
            E.decompress_aggregate(c.L, E.EF_MSG_SPARSE, W, mi, mv, out, c.ws(E.EF_OP_AGG_SPARSE, W))
            want = O.decompress_aggregate_sparse(c.d, [m for m, _ in msgs], [v for _, v in msgs])
        assert_f32_equal(out, want, f"cfg {i} {kind} aggregate W={W}")
        kindm = E.EF_MSG_BLOCK if kind == "randblock" else E.EF_MSG_SPARSE
        ws_a = None if kind == "randblock" else c.ws(E.EF_OP_AGG_SPARSE, W)
        # the same aggregate fused with an update of random parameters (momentum, weight decay)
        beta, wd = float(rng.choice([0.0, 0.9])), float(rng.choice([0.0, 1e-4]))
        use_m = beta != 0.0 or bool(rng.random() < 0.5)
        x0 = rng.standard_normal(c.d).astype(np.float32)
        m0 = (rng.standard_normal(c.d) * 0.1).astype(np.float32)
        xd, md = dev(x0), dev(m0)
        E.decompress_aggregate_apply(c.L, kindm, W, mi, mv, xd, md if use_m else None, beta, wd, None, ws_a)
        wx, wmom = O.apply_update(x0, want, m0 if use_m else None, beta, wd)
        assert_f32_equal(xd, wx, f"cfg {i} {kind} apply x")
        if use_m:
            assert_f32_equal(md, wmom, f"cfg {i} {kind} apply momentum")
        # shared coordinates: worker 0's indices (or starts) for every worker's values
        wss = c.ws(E.EF_OP_AGG_SHARED, W)
        E.decompress_aggregate_shared(c.L, kindm, W, mi[0], mv, out, wss)
        vals = [v for _, v in msgs]
        if kind == "randblock":
            want_s = O.decompress_aggregate_shared_block(c.d, c.offs, c.ks, msgs[0][0], vals)
        else:
            want_s = O.decompress_aggregate_shared_sparse(c.d, msgs[0][0], vals)
        assert_f32_equal(out, want_s, f"cfg {i} {kind} shared aggregate")
        if kind == "randblock":
            continue
        # the same two steps batched, from zero residuals, against the per-worker results above
        eb = [torch.zeros(c.d, dtype=torch.float32, device="cuda") for _ in range(W)]
        gb = [_dev_g(x) for x in G]
        op = E.EF_OP_TOPK if kind == "topk" else E.EF_OP_RANDK
        ws, stride = E.batch_workspace(c.L, op, W)
        for step in range(2):
            idx = torch.empty((W, c.K), dtype=torch.int32, device="cuda")
            val = torch.empty((W, c.K), dtype=torch.float32, device="cuda")
            if kind == "topk":
                E.ef_step_topk_batch(c.L, gb, eb, idx, val, ws, stride)
            else:
                E.ef_step_randk_batch(c.L, gb, eb, seeds, step, idx, val, ws, stride)
        hi, hv = host(idx).view(np.uint32), host(val)
        for w in range(W):
            assert_msg_equal(kind, (hi[w], hv[w]), msgs[w], f"cfg {i} {kind} batch w{w}")
            assert_f32_equal(eb[w], e[w], f"cfg {i} {kind} batch e' w{w}")
        if kind == "randk":  # prepared ahead: the first worker's two steps
            ep = torch.zeros(c.d, dtype=torch.float32, device="cuda")
            wsp = c.ws(E.EF_OP_RANDK_PREP)
            for step in range(2):
                idx = torch.empty(c.K, dtype=torch.int32, device="cuda")
                val = torch.empty(c.K, dtype=torch.float32, device="cuda")
                E.ef_randk_prepare(c.L, seeds[0], step, idx, wsp)
                E.ef_step_randk_prepared(c.L, gb[0], ep, idx, val, wsp)
            assert_msg_equal(kind, (idx, val), msgs[0], f"cfg {i} prepared")
            assert_f32_equal(ep, e[0], f"cfg {i} prepared e'")
