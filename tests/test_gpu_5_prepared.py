"""GPU parity of random-k with the selection prepared ahead (ef_randk_prepare +
ef_step_randk_prepared, and their batch forms): the prepared indices equal the
oracle's support, and the prepared step equals the oracle's step and the fused
step bit for bit (indices, values, residual), on ragged layouts, bf16 gradients,
the exact slow path, layouts without direct lists and k_l above 2^20."""

import numpy as np
import pytest

from efs_gpu import Case, announce, assert_f32_equal, assert_msg_equal, dev, host
from oracle import efsparse_oracle as O

pytestmark = pytest.mark.gpu


def _inputs(d, seed):
    rng = np.random.default_rng(seed)
    g = (rng.standard_normal(d) * 0.01).astype(np.float32)
    e = (rng.standard_normal(d) * 0.003).astype(np.float32)
    g[::97] = 0.0
    e[::89] = -0.0
    return g, e


def _prepared_steps(c, g_list, e, seed, bf16=False):
    """Prepared steps over consecutive steps with the residual carried, each against the oracle
    and against the fused step; returns the last prepare's diagnostics word."""
    import paper_2009_09271_amd as E
    import torch
    from workloads import to_bf16_bits
    ws = c.L.workspace(E.EF_OP_RANDK_PREP)
    for step, g in enumerate(g_list):
        gh = to_bf16_bits(g) if bf16 else g
        gd = dev(gh)
        if bf16:
            gd = gd.view(torch.bfloat16)
        idx = torch.empty(c.K, dtype=torch.int32, device="cuda")
        val = torch.empty(c.K, dtype=torch.float32, device="cuda")
        E.ef_randk_prepare(c.L, seed, step, idx, ws)
        want_idx = O.randk_support(c.offs, c.ks, seed, step)
        got_idx = host(idx).view(np.uint32)
        assert np.array_equal(got_idx, want_idx), f"prepared indices step {step}"
        ed = dev(e)
        E.ef_step_randk_prepared(c.L, gd, ed, idx, val, ws)
        (wm, wval), we = c.oracle_step("randk", gh, e, seed, step)
        assert_msg_equal("randk", (idx, val), (wm, wval), f"prepared step {step}")
        assert_f32_equal(ed, we, f"prepared e' step {step}")
        ef = dev(e)
        mf, vf, _ = c.step("randk", gh, ef, seed, step)
        assert_msg_equal("randk", (mf, vf), (got_idx, host(val)), f"fused vs prepared step {step}")
        e = we
    return c.L.diag(ws, E.EF_OP_RANDK)


LAYOUTS = [
    [0, 1],
    [0, 1001],
    [0, 8193],
    [0, 100000],
    [0, 1, 5, 64, 65, 300, 301, 10007, 10008, 40000],
    [0, 3, 8190, 8195, 16384, 16385, 16386, 30000],
    [0, 4095, 4096, 4097, 8191, 12289, 20000],
]


@pytest.mark.parametrize("offs", LAYOUTS, ids=lambda o: f"d{o[-1]}_L{len(o) - 1}")
@pytest.mark.parametrize("rho", [0.001, 0.05, 1.0])
def test_prepared_matches_oracle_and_fused(offs, rho):
    announce("prepared randk", offs[-1], len(offs) - 1, rho)
    c = Case(offs, rho)
    g, e = _inputs(c.d, 3)
    _prepared_steps(c, [g, g * np.float32(0.5)], e, seed=(5 << 32) | 1)


def test_prepared_bf16_gradient():
    announce("prepared randk bf16")
    c = Case([0, 5, 50000, 120000], 0.01)
    g, e = _inputs(c.d, 4)
    _prepared_steps(c, [g], e, seed=9, bf16=True)


def test_prepared_forced_slow_path():
    """A window of zero width makes every segment take the exact path, which runs without data."""
    import paper_2009_09271_amd as E
    announce("prepared randk slow")
    c = Case([0, 1, 5, 64, 65, 300, 301, 10007, 10008, 40000, 100000], 0.01, tune={E.EF_TUNE_RANDK_SIGMA: -1e9})
    g, e = _inputs(c.d, 5)
    diag = _prepared_steps(c, [g], e, seed=77)
    assert diag & E.DIAG_SLOW_PATH, "the slow path did not run"


def test_prepared_without_direct_lists():
    """k_l = d / 2 = 10^6 on one segment: the expected window (about 12 sqrt(k_l) keys) exceeds
    the select kernel's LDS list, so the candidates are collected by k_collect (no direct lists)."""
    announce("prepared randk collect")
    c = Case([0, 2000000], 0.5)
    g, e = _inputs(c.d, 6)
    _prepared_steps(c, [g], e, seed=21)


@pytest.mark.parametrize("offs", [[0, 3000000], [0, 5, 1234567, 1234570, 3000000]], ids=["flat", "ragged"])
def test_prepared_large_k(offs):
    """k_l above 2^20: the row winners are counted and scanned by the many-workgroup kernels."""
    announce("prepared randk large k", offs[-1])
    c = Case(offs, 0.6)
    g, e = _inputs(c.d, 7)
    _prepared_steps(c, [g], e, seed=17)


@pytest.mark.parametrize("offs,rho,W", [
    ([0, 3, 8192, 8196, 16384, 16388, 16392, 30000, 100000], 0.02, 3),
    ([0, 1, 5, 64, 68, 300, 304, 10008, 10012, 40000], 0.1, 70),
], ids=["ragged-W3", "small-segments-W70"])
def test_prepared_batch(offs, rho, W):
    """The batch forms: W workers' selections prepared in one call (more than 64 workers: two
    selection launches) and their steps, worker by worker against the oracle over two steps."""
    import paper_2009_09271_amd as E
    import torch
    announce("prepared randk batch", offs[-1], W)
    c = Case(offs, rho)
    rng = np.random.default_rng(W)
    G = (rng.standard_normal((W, c.d)) * 10.0 ** rng.integers(-3, 1, (W, 1))).astype(np.float32)
    gd = [dev(x) for x in G]
    e = np.zeros((W, c.d), np.float32)
    ed = [dev(x) for x in e]
    ws, stride = E.batch_workspace(c.L, E.EF_OP_RANDK_PREP, W)
    seeds = [(13 << 32) | w for w in range(W)]
    for step in range(2):
        idx = torch.empty((W, c.K), dtype=torch.int32, device="cuda")
        val = torch.empty((W, c.K), dtype=torch.float32, device="cuda")
        E.ef_randk_prepare_batch(c.L, seeds, step, idx, ws, stride)
        E.ef_step_randk_prepared_batch(c.L, gd, ed, idx, val, ws, stride)
        hi, hv, he = host(idx).view(np.uint32), host(val), np.stack([host(x) for x in ed])
        for w in range(W):
            (wm, wv), we = c.oracle_step("randk", G[w], e[w], seeds[w], step)
            assert_msg_equal("randk", (hi[w], hv[w]), (wm, wv), f"batch worker {w} step {step}")
            assert_f32_equal(he[w], we, f"batch worker {w} e' step {step}")
            e[w] = we


def test_prepared_two_streams():
    """The production order: the selection of step t + 1 prepared on a side stream while step t
    runs, each step waiting for its own selection only."""
    import paper_2009_09271_amd as E
    import torch
    announce("prepared randk two streams")
    c = Case([0, 7, 70000, 70003, 250000], 0.01)
    g, e = _inputs(c.d, 8)
    seed = 99
    side, main = torch.cuda.Stream(), torch.cuda.current_stream()
    ws = [c.L.workspace(E.EF_OP_RANDK_PREP) for _ in range(2)]
    idx = [torch.empty(c.K, dtype=torch.int32, device="cuda") for _ in range(2)]
    ready = [torch.cuda.Event() for _ in range(2)]
    done = [torch.cuda.Event() for _ in range(2)]
    E.ef_randk_prepare(c.L, seed, 0, idx[0], ws[0], stream=side)
    ready[0].record(side)
    ed = dev(e)
    for t in range(4):
        b, nb = t % 2, (t + 1) % 2
        if t >= 1:
            side.wait_event(done[nb])  # buffers nb last used by step t - 1
        E.ef_randk_prepare(c.L, seed, t + 1, idx[nb], ws[nb], stream=side)
        ready[nb].record(side)
        main.wait_event(ready[b])
        val = torch.empty(c.K, dtype=torch.float32, device="cuda")
        E.ef_step_randk_prepared(c.L, dev(g), ed, idx[b], val, ws[b])
        done[b].record(main)
        torch.cuda.synchronize()
        (wm, wv), we = c.oracle_step("randk", g, e, seed, t)
        assert_msg_equal("randk", (idx[b], val), (wm, wv), f"two streams step {t}")
        assert_f32_equal(ed, we, f"two streams e' step {t}")
        e = we
