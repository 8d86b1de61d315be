"""GPU parity for the paths next to the hot path: the shared-coordinate aggregate (the allReduce
mode), the aggregate fused with the parameter update, and the dense average of uncompressed
gradients (standard SGD's exchange).  Bit-exact against the CPU oracle, through the C ABI."""

import numpy as np
import pytest

from efs_gpu import Case, announce, assert_f32_equal, bits, dev, host
from oracle import efsparse_oracle as O

pytestmark = pytest.mark.gpu

LAYOUTS = [
    [0, 1001],
    [0, 8193],
    [0, 100000],
    [0, 1, 5, 64, 65, 300, 301, 10007, 10008, 40000],
    [0, 3, 8190, 8195, 16384, 16385, 16386, 30000],
]


def _values(W, K, seed):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((W, K)) * 10.0 ** rng.integers(-3, 3, (W, 1))).astype(np.float32)


@pytest.mark.parametrize("offs", LAYOUTS, ids=lambda o: f"d{o[-1]}_L{len(o) - 1}")
@pytest.mark.parametrize("W", [1, 3, 16, 70])
def test_shared_coordinates_sparse(offs, W):
    """One random-k index list for every worker: the shared path equals the oracle and, bit for
    bit, the general aggregate given the repeated list."""
    import paper_2009_09271_amd as E
    import torch
    announce("shared sparse", offs[-1], len(offs) - 1, W)
    c = Case(offs, 0.05)
    acc = np.random.default_rng(W).standard_normal(c.d).astype(np.float32)
    idx, _ = O.compress_randk(acc, c.offs, c.ks, 4242, 1)
    V = _values(W, c.K, W + 1)
    out = torch.empty(c.d, dtype=torch.float32, device="cuda")
    ws = c.L.workspace(E.EF_OP_AGG_SHARED, W)
    for average in (True, False):
        E.decompress_aggregate_shared(c.L, E.EF_MSG_SPARSE, W, dev(idx.view(np.int32)), dev(V), out, ws, average)
        want = O.decompress_aggregate_shared_sparse(c.d, idx, V, average)
        assert_f32_equal(out, want, f"shared sparse avg={average}")
        gen = torch.empty_like(out)
        stack = np.repeat(idx[None, :], W, axis=0)
        E.decompress_aggregate(c.L, E.EF_MSG_SPARSE, W, dev(stack.view(np.int32)), dev(V), gen,
                               c.L.workspace(E.EF_OP_AGG_SPARSE, W), average)
        assert np.array_equal(bits(host(out)), bits(host(gen)))


@pytest.mark.parametrize("offs", LAYOUTS, ids=lambda o: f"d{o[-1]}_L{len(o) - 1}")
@pytest.mark.parametrize("W,block", [(1, 1), (5, 256), (16, 1024)])
def test_shared_coordinates_block(offs, W, block):
    import paper_2009_09271_amd as E
    import torch
    announce("shared block", offs[-1], len(offs) - 1, W, block)
    c = Case(offs, 0.3, block)
    acc = np.random.default_rng(W).standard_normal(c.d).astype(np.float32)
    start, _ = O.compress_randblock(acc, c.offs, c.ks, block, 777, 2)
    V = _values(W, c.K, W + 2)
    out = torch.empty(c.d, dtype=torch.float32, device="cuda")
    ws = c.L.workspace(E.EF_OP_AGG_SHARED, W)
    for average in (True, False):
        E.decompress_aggregate_shared(c.L, E.EF_MSG_BLOCK, W, dev(start.view(np.int32)), dev(V), out, ws, average)
        want = O.decompress_aggregate_shared_block(c.d, c.offs, c.ks, start, V, average)
        assert_f32_equal(out, want, f"shared block avg={average}")


@pytest.mark.parametrize("offs", LAYOUTS, ids=lambda o: f"d{o[-1]}_L{len(o) - 1}")
@pytest.mark.parametrize("kind", ["sparse", "block"])
@pytest.mark.parametrize("W,beta,wd,momentum,with_out", [(1, 0.0, 0.0, False, False), (3, 0.9, 1e-4, True, True),
                                                        (16, 0.9, 0.0, True, False), (4, 0.0, 0.01, False, True)],
                         ids=["plain", "momentum-wd-out", "momentum", "wd-out"])
def test_aggregate_apply(offs, kind, W, beta, wd, momentum, with_out):
    """The aggregate fused with x = x - d (d = q + wd x; with momentum m = beta m + d, d = m), over
    two steps with the momentum buffer carried."""
    import paper_2009_09271_amd as E
    import torch
    announce("apply", offs[-1], len(offs) - 1, kind, W, beta, wd, momentum, with_out)
    c = Case(offs, 0.05, 64)
    rng = np.random.default_rng(W + 31)
    x = rng.standard_normal(c.d).astype(np.float32)
    m = (rng.standard_normal(c.d) * 0.01).astype(np.float32) if momentum else None
    xd, md = dev(x), (dev(m) if momentum else None)
    out = torch.empty(c.d, dtype=torch.float32, device="cuda") if with_out else None
    for step in range(2):
        msgs = []
        for w in range(W):
            acc = (rng.standard_normal(c.d) * 10.0 ** rng.integers(-3, 1)).astype(np.float32)
            msgs.append(O.compress_randk(acc, c.offs, c.ks, 100 + w, step) if kind == "sparse"
                        else O.compress_randblock(acc, c.offs, c.ks, 64, 100 + w, step))
        mi = np.stack([q[0] for q in msgs]).astype(np.uint32)
        mv = np.stack([q[1] for q in msgs]).astype(np.float32)
        if kind == "sparse":
            q = O.decompress_aggregate_sparse(c.d, mi, mv)
            E.decompress_aggregate_apply(c.L, E.EF_MSG_SPARSE, W, dev(mi.view(np.int32)), dev(mv), xd, md, beta, wd,
                                         out, c.L.workspace(E.EF_OP_AGG_SPARSE, W))
        else:
            q = O.decompress_aggregate_block(c.d, c.offs, c.ks, mi, mv)
            E.decompress_aggregate_apply(c.L, E.EF_MSG_BLOCK, W, dev(mi.view(np.int32)), dev(mv), xd, md, beta, wd,
                                         out, None)
        x, m = O.apply_update(x, q, m, beta=beta, wd=wd)
        assert_f32_equal(xd, x, f"x step {step}")
        if momentum:
            assert_f32_equal(md, m, f"m step {step}")
        if with_out:
            assert_f32_equal(out, q, f"q step {step}")


def test_aggregate_apply_rejects_aliases():
    import paper_2009_09271_amd as E
    import torch
    c = Case([0, 1000], 0.1)
    x = torch.zeros(1000, device="cuda")
    idx = torch.zeros((2, c.K), dtype=torch.int32, device="cuda")
    val = torch.zeros((2, c.K), device="cuda")
    ws = c.L.workspace(E.EF_OP_AGG_SPARSE, 2)
    for mom, out in ((x, None), (None, x)):
        with pytest.raises(E.EfError):
            E.decompress_aggregate_apply(c.L, E.EF_MSG_SPARSE, 2, idx, val, x, mom, 0.9, 0.0, out, ws)


@pytest.mark.parametrize("d", [1, 5, 1001, 8192, 100003])
@pytest.mark.parametrize("W", [1, 3, 8, 17])
def test_dense_average(d, W):
    import paper_2009_09271_amd as E
    import torch
    announce("dense average", d, W)
    c = Case([0, d], 0.5)
    G = _values(W, d, d + W)
    G[:, ::7] = -0.0
    out = torch.empty(d, dtype=torch.float32, device="cuda")
    for average in (True, False):
        E.ef_dense_average(c.L, W, dev(G), out, average)
        assert_f32_equal(out, O.dense_average(G, average), f"dense avg={average}")
