"""GPU parity: accumulate, random-block and the aggregate against the CPU oracle
(bit-exact), through the C ABI via the Python binding."""

import numpy as np
import pytest

from efs_gpu import Case, announce, assert_f32_equal, assert_msg_equal, bits, dev, host
from oracle import efsparse_oracle as O

pytestmark = pytest.mark.gpu

LAYOUTS = [
    [0, 1],
    [0, 5],
    [0, 1001],
    [0, 8192],
    [0, 8193],
    [0, 100000],
    [0, 1, 5, 64, 65, 300, 301, 10007, 10008, 40000],
    [0, 3, 8190, 8195, 16384, 16385, 16386, 30000],
]


def _inputs(d, seed):
    rng = np.random.default_rng(seed)
    g = (rng.standard_normal(d) * 0.01).astype(np.float32)
    e = (rng.standard_normal(d) * 0.003).astype(np.float32)
    g[::97] = 0.0
    e[::89] = -0.0
    return g, e


@pytest.mark.parametrize("offs", LAYOUTS, ids=lambda o: f"d{o[-1]}_L{len(o) - 1}")
def test_accumulate(offs):
    import paper_2009_09271_amd as E
    import torch
    announce("accumulate", offs[-1], len(offs) - 1)
    c = Case(offs, 0.1)
    g, e = _inputs(c.d, 1)
    acc = torch.empty(c.d, dtype=torch.float32, device="cuda")
    E.ef_accumulate(c.L, dev(g), dev(e), acc)
    assert_f32_equal(acc, O.ef_accumulate(g, e), "acc")
    # bf16 gradient, in place
    from workloads import to_bf16_bits
    gb = to_bf16_bits(g)
    ed = dev(e)
    E.ef_accumulate(c.L, dev(gb).view(torch.bfloat16), ed, ed)
    assert_f32_equal(ed, O.ef_accumulate(gb, e), "acc bf16 in place")


@pytest.mark.parametrize("offs", LAYOUTS, ids=lambda o: f"d{o[-1]}_L{len(o) - 1}")
@pytest.mark.parametrize("block", [1, 2, 256, 1024])
@pytest.mark.parametrize("rho", [0.01, 0.3, 1.0])
def test_randblock_fused_and_composed(offs, block, rho):
    announce("randblock", offs[-1], len(offs) - 1, block, rho)
    c = Case(offs, rho, block)
    g, e = _inputs(c.d, 2)
    seed = (7 << 32) | 3
    for step in range(3):
        ed = dev(e)
        st, val, _ = c.step("randblock", g, ed, seed, step)
        (wst, wval), we = c.oracle_step("randblock", g, e, seed, step)
        assert_msg_equal("randblock", (st, val), (wst, wval), f"step {step}")
        assert_f32_equal(ed, we, f"e' step {step}")
        ed2 = dev(e)
        m2, val2 = c.step_composed("randblock", g, ed2, seed, step)
        assert_msg_equal("randblock", (m2, val2), (wst, wval), f"composed step {step}")
        assert_f32_equal(ed2, we, f"composed e' step {step}")
        e = we


def _agg_check(c, kind, msgs, W, average):
    import paper_2009_09271_amd as E
    import torch
    out = torch.empty(c.d, dtype=torch.float32, device="cuda")
    if kind == "sparse":
        idx = np.stack([m[0] for m in msgs]).astype(np.uint32)
        val = np.stack([m[1] for m in msgs]).astype(np.float32)
        ws = c.L.workspace(E.EF_OP_AGG_SPARSE, W)
        E.decompress_aggregate(c.L, E.EF_MSG_SPARSE, W, dev(idx.view(np.int32)), dev(val), out, ws, average)
        want = O.decompress_aggregate_sparse(c.d, idx, val, average)
    else:
        st = np.stack([m[0] for m in msgs]).astype(np.uint32)
        val = np.stack([m[1] for m in msgs]).astype(np.float32)
        E.decompress_aggregate(c.L, E.EF_MSG_BLOCK, W, dev(st.view(np.int32)), dev(val), out, None, average)
        want = O.decompress_aggregate_block(c.d, c.offs, c.ks, st, val, average)
    assert_f32_equal(out, want, f"aggregate {kind} W={W} avg={average}")


@pytest.mark.parametrize("offs", LAYOUTS[2:], ids=lambda o: f"d{o[-1]}_L{len(o) - 1}")
@pytest.mark.parametrize("W", [1, 3, 16])
def test_aggregate_sparse_and_block(offs, W):
    announce("aggregate", offs[-1], len(offs) - 1, W)
    c = Case(offs, 0.05, 64)
    rng = np.random.default_rng(W)
    sparse, block = [], []
    for w in range(W):
        acc = (rng.standard_normal(c.d) * 10.0 ** rng.integers(-3, 3)).astype(np.float32)
        sparse.append(O.compress_randk(acc, c.offs, c.ks, 100 + w, 0))
        block.append(O.compress_randblock(acc, c.offs, c.ks, 64, 100 + w, 0))
    for average in (True, False):
        _agg_check(c, "sparse", sparse, W, average)
        _agg_check(c, "block", block, W, average)


def test_aggregate_order_and_signed_zero():
    """Worker order matters in float32 ((1 + 1e8) - 1e8 = 0); the sum starts at +0."""
    announce("aggregate order")
    c = Case([0, 8], 1.0)  # k = d = 8
    msgs = []
    vals = [[1.0] * 8, [1e8] * 8, [-1e8] * 8, [-0.0] * 8]
    for v in vals:
        msgs.append((np.arange(8, dtype=np.uint32), np.array(v, np.float32)))
    _agg_check(c, "sparse", msgs, 4, False)
    _agg_check(c, "sparse", msgs[3:], 1, True)


def test_randblock_deterministic_and_shared_seed():
    announce("randblock determinism")
    c = Case([0, 50000, 123457], 0.01, 256)
    g, e = _inputs(c.d, 5)
    a = c.step("randblock", g, dev(e), 11, 4)
    b = c.step("randblock", g, dev(e), 11, 4)
    assert np.array_equal(host(a[0]), host(b[0])) and np.array_equal(bits(host(a[1])), bits(host(b[1])))


@pytest.mark.parametrize("W,rho", [(70, 0.002), (70, 0.05), (4, 0.5)], ids=["regs-2groups", "lds-2groups", "lds-dense"])
def test_aggregate_sparse_modes(W, rho):
    """Tiles summed in registers (few entries) and in LDS (many), more than one worker group of
    ranges, and several staging passes per group."""
    announce("aggregate modes", W, rho)
    c = Case([0, 3, 9000, 9001, 20000], rho)
    rng = np.random.default_rng(int(W * 1000 * rho))
    msgs = []
    for w in range(W):
        acc = (rng.standard_normal(c.d) * 10.0 ** rng.integers(-3, 3)).astype(np.float32)
        msgs.append(O.compress_randk(acc, c.offs, c.ks, 7 + w, 1))
    for average in (True, False):
        _agg_check(c, "sparse", msgs, W, average)


@pytest.mark.parametrize("W", [3, 20, 70])
def test_aggregate_block_many_segments_per_tile(W):
    """150 segments of 7 elements share the first tile (more than one pass of segments and, with
    many workers, more than one group of block starts)."""
    announce("aggregate block segments", W)
    offs = list(range(0, 7 * 151, 7)) + [30000]
    c = Case(offs, 0.3, 4)
    rng = np.random.default_rng(W)
    msgs = []
    for w in range(W):
        acc = rng.standard_normal(c.d).astype(np.float32)
        msgs.append(O.compress_randblock(acc, c.offs, c.ks, 4, 50 + w, 2))
    for average in (True, False):
        _agg_check(c, "block", msgs, W, average)


@pytest.mark.parametrize("W,rho,block", [(70, 0.6, 16), (130, 0.02, 1), (5, 1.0, 1)],
                         ids=["wrapping-2groups", "3groups", "k=d"])
def test_aggregate_block_single_segment(W, rho, block):
    """One segment (flat scope): more than one wavefront's worth of workers, runs that wrap around
    the end of the vector, and k = d (every worker covers everything)."""
    announce("aggregate block single segment", W, rho, block)
    c = Case([0, 10007], rho, block)
    rng = np.random.default_rng(W + 7)
    msgs = []
    for w in range(W):
        acc = rng.standard_normal(c.d).astype(np.float32)
        msgs.append(O.compress_randblock(acc, c.offs, c.ks, block, 60 + w, 3))
    for average in (True, False):
        _agg_check(c, "block", msgs, W, average)


@pytest.mark.parametrize("W,rho", [(4, 0.002), (16, 0.05)], ids=["few-shared", "many-shared"])
def test_aggregate_sparse_shared_coordinates(W, rho):
    """Random-k with one seed for all workers (every position is hit by every worker): the shared
    positions are summed in worker order, by walking (few) or worker by worker (many)."""
    announce("aggregate shared", W, rho)
    c = Case([0, 3, 9000, 9001, 20000], rho)
    rng = np.random.default_rng(W)
    msgs = []
    for w in range(W):
        acc = (rng.standard_normal(c.d) * 10.0 ** rng.integers(-3, 3)).astype(np.float32)
        msgs.append(O.compress_randk(acc, c.offs, c.ks, 1234, 3))
    for average in (True, False):
        _agg_check(c, "sparse", msgs, W, average)


@pytest.mark.parametrize("W", [2, 16, 70])
def test_aggregate_sparse_concentrated(W):
    """Messages that crowd into a few tiles with long empty gaps (top-k on layers of very
    different scales): tile boundaries far from every entry (more than one strided pass of the
    ranges kernel), tiles no message enters, and tiles with thousands of entries."""
    announce("aggregate concentrated", W)
    d = 4096 * 700 + 123
    offs = [0, d]
    rng = np.random.default_rng(W + 11)
    msgs = []
    for w in range(W):
        hot = rng.choice(np.arange(4096 * 300, 4096 * 303), size=3000, replace=False)
        far = np.array([5, d - 1], dtype=np.int64)
        i = np.unique(np.concatenate([hot, far])).astype(np.uint32)
        v = (rng.standard_normal(i.size) * 10.0 ** rng.integers(-3, 3)).astype(np.float32)
        msgs.append((i, v))
    K = msgs[0][0].size
    assert all(m[0].size == K for m in msgs)
    c = Case(offs, K / d)
    assert c.K == K
    for average in (True, False):
        _agg_check(c, "sparse", msgs, W, average)


@pytest.mark.parametrize("offs", LAYOUTS, ids=lambda o: f"d{o[-1]}_L{len(o) - 1}")
@pytest.mark.parametrize("aligned16", [True, False], ids=["g16", "g8"])
def test_randblock_bf16_gradient(offs, aligned16):
    """The fused block-random-k step on a bf16 gradient, 16-byte aligned and only 8-byte aligned
    (the entry point's requirement for bf16)."""
    import paper_2009_09271_amd as E
    import torch
    from workloads import to_bf16_bits
    announce("randblock bf16", offs[-1], len(offs) - 1, aligned16)
    c = Case(offs, 0.05, 256)
    g, e = _inputs(c.d, 4)
    gb = to_bf16_bits(g)
    off = 0 if aligned16 else 4  # 4 bf16 values = 8 bytes past a 256-byte aligned allocation
    buf = np.zeros(c.d + 8, np.uint16)
    buf[off:off + c.d] = gb
    gd = dev(buf)[off:off + c.d].view(torch.bfloat16)
    assert (gd.data_ptr() % 16 == 0) == aligned16
    seed = (9 << 32) | 2
    for step in range(2):
        ed = dev(e)
        start = torch.empty(len(c.ks), dtype=torch.int32, device="cuda")
        val = torch.empty(c.K, dtype=torch.float32, device="cuda")
        E.ef_step_randblock(c.L, gd, ed, seed, step, start, val)
        (wst, wval), we = c.oracle_step("randblock", gb, e, seed, step)
        assert_msg_equal("randblock", (start, val), (wst, wval), f"bf16 step {step}")
        assert_f32_equal(ed, we, f"bf16 e' step {step}")
        e = we
