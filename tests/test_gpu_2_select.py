"""GPU parity: fused and composed top-k / random-k worker steps against the CPU
oracle, bit-exact (indices, values, residual), on ragged layouts, ties, signed
zeros, bf16 gradients and the forced exact slow paths."""

import numpy as np
import pytest

from efs_gpu import Case, announce, assert_f32_equal, assert_msg_equal, bits, dev, host

pytestmark = pytest.mark.gpu

LAYOUTS = [
    [0, 1],
    [0, 7],
    [0, 1001],
    [0, 8192],
    [0, 8193],
    [0, 100000],
    [0, 1, 5, 64, 65, 300, 301, 10007, 10008, 40000],
    [0, 3, 8190, 8195, 16384, 16385, 16386, 30000],
    [0, 2, 6, 10, 14, 8200, 8204, 8300, 70000],
    [0, 4095, 4096, 4097, 8191, 12289, 20000],
]


def _inputs(d, seed, ties=False):
    rng = np.random.default_rng(seed)
    if ties:  # few distinct magnitudes: many equal keys, both zeros
        g = rng.choice(np.array([0.0, -0.0, 0.5, -0.5, 0.25, 1.0, -1.0, 2.0 ** -130], np.float32), size=d)
        e = np.zeros(d, np.float32)
        e[::3] = -0.0
    else:
        g = (rng.standard_normal(d) * 0.01).astype(np.float32)
        e = (rng.standard_normal(d) * 0.003).astype(np.float32)
        g[::97] = 0.0
    return g, e


def _run_steps(c, kind, g_list, e, seed=0, composed=True):
    for step, g in enumerate(g_list):
        ed = dev(e)
        m, val, ws = c.step(kind, g, ed, seed, step)
        (wm, wval), we = c.oracle_step(kind, g, e, seed, step)
        assert_msg_equal(kind, (m, val), (wm, wval), f"{kind} step {step}")
        assert_f32_equal(ed, we, f"{kind} e' step {step}")
        diag = c.L.diag(ws, c.E.EF_OP_TOPK if kind == "topk" else c.E.EF_OP_RANDK)
        assert not diag & c.E.DIAG_COUNT_MISMATCH, f"{kind} row counts inconsistent at step {step}"
        if composed:
            ed2 = dev(e)
            m2, val2 = c.step_composed(kind, g, ed2, seed, step)
            assert_msg_equal(kind, (m2, val2), (wm, wval), f"{kind} composed step {step}")
            assert_f32_equal(ed2, we, f"{kind} composed e' step {step}")
        e = we
    return diag


@pytest.mark.parametrize("offs", LAYOUTS, ids=lambda o: f"d{o[-1]}_L{len(o) - 1}")
@pytest.mark.parametrize("rho", [0.001, 0.01, 0.3, 1.0])
@pytest.mark.parametrize("kind", ["topk", "randk"])
def test_select_parity(kind, rho, offs):
    announce(kind, offs[-1], len(offs) - 1, rho)
    c = Case(offs, rho)
    g0, e = _inputs(c.d, 3)
    g1, _ = _inputs(c.d, 4)
    _run_steps(c, kind, [g0, g1], e, seed=(5 << 32) | 9)


@pytest.mark.parametrize("offs", LAYOUTS[2:], ids=lambda o: f"d{o[-1]}_L{len(o) - 1}")
@pytest.mark.parametrize("rho", [0.01, 0.5])
def test_topk_ties_and_signed_zeros(rho, offs):
    announce("topk ties", offs[-1], rho)
    c = Case(offs, rho)
    g, e = _inputs(c.d, 6, ties=True)
    _run_steps(c, "topk", [g, g], e)


# Segments sampled whole are ranked directly when they hold at most 256 keys, with 16, 8 or 4
# threads per key (up to 64, 128 and 256 keys) over a list padded to a multiple of 64 words; the
# sizes fall on both sides of each width and of the largest segment sampled whole (4096).
RANK_SIZES = [1, 63, 64, 65, 127, 128, 129, 255, 256, 257, 4096, 4097]


@pytest.mark.parametrize("rho", [0.02, 0.5, 1.0])
@pytest.mark.parametrize("ties", [False, True], ids=["smooth", "ties"])
def test_topk_segments_at_the_ranking_widths(rho, ties):
    offs = np.concatenate([[0], np.cumsum(RANK_SIZES)]).tolist()
    announce("topk ranking widths", offs[-1], rho, ties)
    c = Case(offs, rho)
    g, e = _inputs(c.d, 11, ties=ties)
    _run_steps(c, "topk", [g, g], e)


@pytest.mark.parametrize("kind", ["topk", "randk"])
def test_bf16_gradient(kind):
    from workloads import to_bf16_bits
    announce(kind, "bf16")
    c = Case([0, 1, 5, 64, 65, 300, 301, 10007, 10008, 40000], 0.02)
    g, e = _inputs(c.d, 7)
    _run_steps(c, kind, [to_bf16_bits(g), to_bf16_bits(g * 3)], e, seed=42, composed=False)


@pytest.mark.parametrize("offs", [[0, 100000], [0, 5, 50000, 120000], [0, 3, 40000, 40001, 90001]],
                         ids=["flat", "two-large", "mixed"])
def test_topk_forced_slow_path(offs):
    """A threshold margin of -1e9 standard deviations puts the sampled threshold at the sample's
    largest key, so every sampled segment has fewer candidates than k; with the retry switched
    off, the exact whole-segment path must give the same result."""
    import paper_2009_09271_amd as E
    announce("topk slow", offs[-1])
    c = Case(offs, 0.01, tune={E.EF_TUNE_TOPK_SIGMA: -1e9, E.EF_TUNE_TOPK_RETRY: 0})
    g, e = _inputs(c.d, 8)
    diag = _run_steps(c, "topk", [g, g], e)
    assert diag & E.DIAG_SLOW_PATH, "the slow path did not run"


@pytest.mark.parametrize("offs", [[0, 100000], [0, 5, 50000, 120000], [0, 3, 40000, 40001, 90001],
                                  [0, 1 << 21]],
                         ids=["flat", "two-large", "mixed", "many-rows"])
@pytest.mark.parametrize("scale", [1.0, 0.0], ids=["spread", "equal"])
def test_topk_forced_retry(offs, scale):
    """The same forced shortfall with the retry on: the sampled segments collect their candidates
    again at a lower threshold over the whole device and must give the same result, without the
    exact whole-segment path.  'equal' gives every element of a segment the same magnitude outside
    a few large values, so the retry's list is all ties, ranked by index."""
    import paper_2009_09271_amd as E
    announce("topk retry", offs[-1], scale)
    c = Case(offs, 0.01, tune={E.EF_TUNE_TOPK_SIGMA: -1e9})
    rng = np.random.default_rng(12)
    if scale:
        g = (rng.standard_normal(c.d) * 10.0 ** rng.integers(-2, 1, c.d)).astype(np.float32)
    else:
        g = np.full(c.d, 0.75, np.float32)
        g[rng.choice(c.d, size=c.d // 1000, replace=False)] = 1.0  # fewer than k: the rest are ties
    e = np.zeros(c.d, np.float32)
    diag = _run_steps(c, "topk", [g], e)
    assert diag & E.DIAG_RETRY and not diag & E.DIAG_SLOW_PATH, f"diagnostics {diag:#x}"


def test_randk_forced_slow_path():
    import paper_2009_09271_amd as E
    announce("randk slow")
    c = Case([0, 1, 5, 64, 65, 300, 301, 10007, 10008, 40000, 100000], 0.01, tune={E.EF_TUNE_RANDK_SIGMA: -1e9})
    g, e = _inputs(c.d, 9)
    diag = _run_steps(c, "randk", [g, g], e, seed=77)
    assert diag & E.DIAG_SLOW_PATH, "the slow path did not run"


@pytest.mark.parametrize("offs", [[0, 4096], [0, 3, 4099, 9000]], ids=["one-row", "ragged"])
def test_randk_rows_wholly_undecided(offs):
    """A window margin of 2000 around k_l = d_l / 2 makes nearly every element of a 4096-element
    segment undecided: each row lists all of them from its own candidate entries, and the
    selection over that list must be exact without the whole-segment path."""
    import paper_2009_09271_amd as E
    announce("randk rows wholly undecided", offs)
    c = Case(offs, 0.5, tune={E.EF_TUNE_RANDK_EXTRA: 2000.0})
    g, e = _inputs(c.d, 12)
    diag = _run_steps(c, "randk", [g, g], e, seed=79)
    assert not diag & E.DIAG_SLOW_PATH, f"diagnostics {diag:#x}"


def _front_loaded(d, seed):
    """Magnitudes 100x larger in the first quarter: its rows hold all of top-k's candidates."""
    rng = np.random.default_rng(seed)
    g = rng.standard_normal(d).astype(np.float32)
    g[: d // 4] *= np.float32(100.0)
    return g


@pytest.mark.parametrize("kind,offs,rho,tune", [
    ("topk", [0, 100000], 0.05, {}),
    ("topk", [0, 5, 50000, 120000], 0.05, {}),
    ("topk", [0, 3, 40000, 40001, 90001], 0.01, {"TOPK_SIGMA": -1e9}),
    ("randk", [0, 1000000], 0.3, {"RANDK_EXTRA": 5000.0}),
], ids=["topk-flat", "topk-two-large", "topk-retry", "randk-lists"])
def test_pool_overflow_takes_exact_path(kind, offs, rho, tune):
    """With the candidate pool and lists tuned to nothing, a row with more candidates than its
    static slot (top-k: the pass or the retry) or any listed candidate (random-k, wide windows)
    does not fit the workspace: its segment takes the exact whole-segment path, same result."""
    import paper_2009_09271_amd as E
    announce("pool overflow", kind, offs[-1], rho, tune)
    t = {getattr(E, "EF_TUNE_" + k): v for k, v in tune.items()}
    t[E.EF_TUNE_POOL] = 0.0
    c = Case(offs, rho, tune=t)
    assert c.L.workspace_bytes(E.EF_OP_TOPK if kind == "topk" else E.EF_OP_RANDK) < 12 * c.d
    g = _front_loaded(c.d, 13)
    diag = _run_steps(c, kind, [g, g * np.float32(0.5)], np.zeros(c.d, np.float32), seed=81)
    assert diag & E.DIAG_SLOW_PATH, f"diagnostics {diag:#x}"


@pytest.mark.parametrize("rho,scales,must_retry", [
    (0.001, (0.006, 0.01, 0.015, 0.02), True),
    (0.01, (0.04, 0.06, 0.08, 0.1), False),
], ids=["sparse", "dense"])
def test_topk_pool_overflow_retries(rho, scales, must_retry):
    """Candidates crowded into a few rows overflow a small pool in the streaming pass; the
    histogram still counted them all, so the rows collect again only the keys of the threshold bin
    and above.  Each pool size must give the oracle's result.  At 0.1 % (the residual is +0 at the
    winners) the pool starts again from empty and at least one size must take that retry without
    the exact path (which costs ~0.3 s at 1e8); at 1 % the pass stored +0 at the candidates, whose
    rows put them back first, so the pool keeps them and a retry that does not fit ends on the
    exact path."""
    import paper_2009_09271_amd as E
    d = 1 << 20
    rng = np.random.default_rng(14)
    g = rng.standard_normal(d).astype(np.float32)
    g[: d // 16] *= np.float32(100.0)  # the winners lie in the first 16 rows
    retried = []
    for scale in scales:
        announce("topk pool overflow retry", rho, scale)
        c = Case([0, d], rho, tune={E.EF_TUNE_POOL: scale})
        diag = _run_steps(c, "topk", [g], np.zeros(d, np.float32))
        retried.append((scale, diag))
    if must_retry:
        assert any(dg & E.DIAG_RETRY and not dg & E.DIAG_SLOW_PATH for _, dg in retried), retried


def test_randk_every_element_a_candidate():
    import paper_2009_09271_amd as E
    announce("randk all candidates")
    c = Case([0, 1, 5, 64, 65, 300, 301, 10007, 10008, 40000, 100000], 0.01, tune={E.EF_TUNE_RANDK_EXTRA: 1e9})
    g, e = _inputs(c.d, 10)
    diag = _run_steps(c, "randk", [g, g], e, seed=78)
    assert not diag & E.DIAG_SLOW_PATH


@pytest.mark.parametrize("kind", ["topk", "randk"])
def test_deterministic_repeat(kind):
    announce(kind, "repeat")
    c = Case([0, 300000], 0.01)
    g, e = _inputs(c.d, 10)
    a = c.step(kind, g, dev(e), 3, 1)
    b = c.step(kind, g, dev(e), 3, 1)
    assert np.array_equal(host(a[0]), host(b[0])) and np.array_equal(bits(host(a[1])), bits(host(b[1])))


def test_randk_shared_seed_same_coordinates():
    announce("randk shared seed")
    c = Case([0, 50000], 0.01)
    g1, e = _inputs(c.d, 11)
    g2, _ = _inputs(c.d, 12)
    a = c.step("randk", g1, dev(e), 1 << 32, 5)
    b = c.step("randk", g2, dev(e), 1 << 32, 5)
    d_ = c.step("randk", g2, dev(e), (1 << 32) | 1, 5)
    assert np.array_equal(host(a[0]), host(b[0]))
    assert not np.array_equal(host(a[0]), host(d_[0]))


@pytest.mark.parametrize("kind", ["topk", "randk"])
def test_sparse_candidates_across_many_chunks(kind):
    """Few candidates per chunk (often 0 or 1) over hundreds of chunks, plus long runs of chunks
    without candidates (layer scales spanning three orders of magnitude)."""
    announce(kind, "sparse candidates")
    offs = [0, 8192 * 100 + 7, 8192 * 100 + 11, 8192 * 300]
    c = Case(offs, 0.0001)
    rng = np.random.default_rng(21)
    d = c.d
    scale = np.where(np.arange(d) < offs[1], 1e-3, np.where(np.arange(d) < offs[2], 1.0, 1e-5))
    g = (rng.standard_normal(d) * scale).astype(np.float32)
    e = np.zeros(d, np.float32)
    _run_steps(c, kind, [g, g], e, seed=99)


def test_topk_flat_layered_scales():
    """Flat scope over layers of very different scale: the candidates sit in a few chunks."""
    announce("topk layered")
    rng = np.random.default_rng(22)
    sizes = [40000, 300000, 5000, 800000, 64, 150000]
    scales = [1e-4, 1e-2, 1.0, 1e-5, 3.0, 1e-3]
    g = np.concatenate([rng.laplace(0, s, n) for n, s in zip(sizes, scales)]).astype(np.float32)
    c = Case([0, len(g)], 0.001)
    _run_steps(c, "topk", [g, g * 0.5], np.zeros(len(g), np.float32))


@pytest.mark.parametrize("kind", ["topk", "randk"])
def test_workspace_reused_with_stale_contents(kind):
    """One workspace, filled with stale bytes, serves several calls (and the other selection op):
    nothing may depend on its previous contents."""
    import torch
    announce(kind, "stale workspace")
    offs = [0, 3, 40000, 40001, 90001, 200000]
    c = Case(offs, 0.01)
    n = max(c.L.workspace_bytes(c.E.EF_OP_TOPK), c.L.workspace_bytes(c.E.EF_OP_RANDK))
    ws = torch.full((n,), 0xA5, dtype=torch.uint8, device="cuda")
    g, e = _inputs(c.d, 31)
    for step in range(3):
        ed = dev(e)
        other = "randk" if kind == "topk" else "topk"
        c.step(other, g, dev(e), 5, step, ws=ws)  # leaves its own state behind
        m, val, _ = c.step(kind, g, ed, 5, step, ws=ws)
        (wm, wval), we = c.oracle_step(kind, g, e, 5, step)
        assert_msg_equal(kind, (m, val), (wm, wval), f"{kind} step {step}")
        assert_f32_equal(ed, we, f"{kind} e' step {step}")
        e = we
        g = g * np.float32(0.5)


def test_topk_concentrated_magnitudes():
    """A sampled segment whose keys all share their top 11 bits: the candidate threshold is refined
    inside that bin (otherwise every element would become a candidate)."""
    announce("topk concentrated")
    rng = np.random.default_rng(23)
    d = 200000
    g = ((1.0 + 0.1 * rng.random(d)) * rng.choice([-1.0, 1.0], d)).astype(np.float32)
    c = Case([0, d], 0.01)
    _run_steps(c, "topk", [g, g], np.zeros(d, np.float32))


@pytest.mark.parametrize("zero_frac,rho", [(0.9, 0.2), (0.9, 0.05), (0.5, 0.6)], ids=["k>nonzeros", "k<nonzeros", "half-zero"])
@pytest.mark.parametrize("layered", [False, True], ids=["flat", "layers"])
def test_topk_threshold_on_a_massive_tie(zero_frac, rho, layered):
    """Most elements exactly zero (embedding rows without tokens): when k exceeds the nonzeros the
    threshold is the key 0 itself and the zeros are taken by index; the threshold bin is then a
    pure tie, resolved from per-row tie counts."""
    announce("topk massive tie", zero_frac, rho, layered)
    rng = np.random.default_rng(24)
    d = 300000
    offs = [0, 123457, 123461, d] if layered else [0, d]
    c = Case(offs, rho)
    g = (rng.standard_normal(d) * 1e-3).astype(np.float32)
    g[rng.random(d) < zero_frac] = 0.0
    g[::7] = np.where(g[::7] == 0.0, np.float32(-0.0), g[::7])
    _run_steps(c, "topk", [g, g * np.float32(0.5)], np.zeros(d, np.float32))


def test_topk_threshold_on_a_repeated_value():
    """A value repeated many times right at the threshold (quantised gradients)."""
    announce("topk repeated value")
    rng = np.random.default_rng(25)
    d = 250000
    g = rng.choice(np.array([0.5, -0.5, 0.25, 0.125, 1.0], np.float32), size=d, p=[0.3, 0.3, 0.2, 0.15, 0.05])
    c = Case([0, d], 0.2)
    _run_steps(c, "topk", [g, g], np.zeros(d, np.float32))


@pytest.mark.parametrize("d,rho,big_frac,tie_frac", [(1_000_000, 0.08, 0.07, 0.02), (1 << 22, 0.26, 0.25, 0.02)],
                         ids=["k-below-2^20", "k-above-2^20"])
def test_topk_list_of_equal_keys_beyond_lds(d, rho, big_frac, tie_frac):
    """A magnitude repeated tens of thousands of times strictly inside a histogram bin, right at the
    threshold (quantised or bf16 gradients): the listed candidates outgrow the select kernel's LDS
    list (8192 entries) and are swept from the sub-lists in global memory; the second step, with
    the residual carried, puts the threshold on another such value.  Without the exact path."""
    announce("topk list beyond LDS", d, rho)
    rng = np.random.default_rng(26)
    u = rng.random(d)
    sign = np.where(rng.random(d) < 0.5, np.float32(-1.0), np.float32(1.0))
    g = (0.01 * rng.standard_normal(d)).astype(np.float32)
    g[u < big_frac] = 1.5
    g[(u >= big_frac) & (u < big_frac + tie_frac)] = 0.7
    g = np.where(u < big_frac + tie_frac, g * sign, g).astype(np.float32)
    c = Case([0, d], rho)
    assert c.K > (d * big_frac) and c.K < d * (big_frac + tie_frac)  # the threshold is the tie value
    diag = _run_steps(c, "topk", [g, g], np.zeros(d, np.float32), composed=False)
    assert not diag & c.E.DIAG_SLOW_PATH, "exact whole-segment path taken"


@pytest.mark.parametrize("offs", [[0, 3000000], [0, 5, 1234567, 1234570, 3000000]], ids=["flat", "ragged"])
@pytest.mark.parametrize("kind", ["topk", "randk"])
@pytest.mark.parametrize("ties", [False, True], ids=["smooth", "ties"])
def test_large_k_row_counting(offs, kind, ties):
    """k_l above 2^20: the row winners are counted and scanned by the many-workgroup kernels."""
    announce(kind, "large k", offs[-1], ties)
    c = Case(offs, 0.6)
    g, e = _inputs(c.d, 31, ties=ties)
    _run_steps(c, kind, [g, g * np.float32(0.5)], e, seed=17, composed=False)


@pytest.mark.parametrize("kind", ["topk", "randk"])
@pytest.mark.parametrize("two_streams", [False, True], ids=["one-stream", "two-streams"])
def test_phased_step_matches_oracle(kind, two_streams):
    """ef_step_*_phases: PREPARE, STREAM and FINISH as separate calls (the stream pass on a second
    stream, ordered by events, when two_streams) give the fused step's result bit for bit, over
    three steps with the residual carried; invalid phase masks are rejected."""
    import paper_2009_09271_amd as E
    import torch
    announce("phased step", kind, two_streams)
    offs = [0, 3, 8190, 8195, 16384, 16385, 16386, 30000, 100000]
    c = Case(offs, 0.02)
    rng = np.random.default_rng(5)
    g = (rng.standard_normal(c.d) * 0.01).astype(np.float32)
    e = np.zeros(c.d, np.float32)
    ws = c.ws(E.EF_OP_TOPK if kind == "topk" else E.EF_OP_RANDK)
    seed = (9 << 32) | 4
    side = torch.cuda.Stream() if two_streams else torch.cuda.current_stream()
    main = torch.cuda.current_stream()
    gd = dev(g)
    for step in range(3):
        ed = dev(e)
        idx = torch.empty(c.K, dtype=torch.int32, device="cuda")
        val = torch.empty(c.K, dtype=torch.float32, device="cuda")

        def phase(p):
            if kind == "topk":
                E.ef_step_topk_phases(c.L, p, gd, ed, idx, val, ws)
            else:
                E.ef_step_randk_phases(c.L, p, gd, ed, seed, step, idx, val, ws)

        phase(E.EF_PHASE_PREPARE)
        side.wait_stream(main)
        with torch.cuda.stream(side):
            phase(E.EF_PHASE_STREAM)
        main.wait_stream(side)
        phase(E.EF_PHASE_FINISH)
        (wm, wv), we = c.oracle_step(kind, g, e, seed, step)
        assert_msg_equal(kind, (idx, val), (wm, wv), f"step {step}")
        assert_f32_equal(ed, we, f"e' step {step}")
        e = we
    for bad in (0, 8, 15):
        with pytest.raises(E.EfError):
            if kind == "topk":
                E.ef_step_topk_phases(c.L, bad, gd, ed, idx, val, ws)
            else:
                E.ef_step_randk_phases(c.L, bad, gd, ed, seed, 0, idx, val, ws)


@pytest.mark.parametrize("kind", ["topk", "randk"])
@pytest.mark.parametrize("offs,rho,W,bf16", [
    ([0, 3, 8192, 8196, 16384, 16388, 16392, 30000, 100000], 0.02, 3, False),
    ([0, 1, 5, 64, 68, 300, 304, 10008, 10012, 40000], 0.1, 70, False),
    ([0, 100000], 0.01, 1, True),
    ([0, 2200000], 0.5, 2, False),
], ids=["ragged-W3", "small-segments-W70", "flat-W1-bf16", "big-k-W2"])
@pytest.mark.parametrize("split", [False, True], ids=["fused", "split-phases"])
def test_batched_steps_match_oracle(kind, offs, rho, W, bf16, split):
    """ef_step_*_batch: W workers' fused steps in one call (selection kernels with the worker in
    the grid, in chunks of 64) equal the oracle's steps worker by worker, over two steps with the
    residual carried."""
    import paper_2009_09271_amd as E
    import torch
    from workloads import to_bf16_bits
    announce("batched steps", kind, offs[-1], len(offs) - 1, W, bf16)
    c = Case(offs, rho)
    rng = np.random.default_rng(W + len(offs))
    G = (rng.standard_normal((W, c.d)) * 10.0 ** rng.integers(-3, 1, (W, 1))).astype(np.float32)
    if bf16:
        G = np.stack([to_bf16_bits(x) for x in G])
    gd = [dev(x) for x in G]
    if bf16:
        gd = [x.view(torch.bfloat16) for x in gd]
    e = np.zeros((W, c.d), np.float32)
    ed = [dev(x) for x in e]
    ws, stride = E.batch_workspace(c.L, E.EF_OP_TOPK if kind == "topk" else E.EF_OP_RANDK, W)
    seeds = [(11 << 32) | w for w in range(W)]
    for step in range(2):
        idx = torch.empty((W, c.K), dtype=torch.int32, device="cuda")
        val = torch.empty((W, c.K), dtype=torch.float32, device="cuda")
        def call(p, st=None):
            if kind == "topk":
                E.ef_step_topk_batch(c.L, gd, ed, idx, val, ws, stride, phases=p, stream=st)
            else:
                E.ef_step_randk_batch(c.L, gd, ed, seeds, step, idx, val, ws, stride, phases=p, stream=st)

        if split:  # prepare + stream on one stream, finish on another after an event
            side = torch.cuda.Stream()
            call(E.EF_PHASE_PREPARE | E.EF_PHASE_STREAM)
            side.wait_stream(torch.cuda.current_stream())
            call(E.EF_PHASE_FINISH, side)
            torch.cuda.current_stream().wait_stream(side)
        else:
            call(E.EF_PHASE_ALL)
        hi, hv, he = host(idx).view(np.uint32), host(val), np.stack([host(x) for x in ed])
        for w in range(W):
            (wm, wv), we = c.oracle_step(kind, G[w], e[w], seeds[w], step)
            assert_msg_equal(kind, (hi[w], hv[w]), (wm, wv), f"step {step} worker {w}")
            assert np.array_equal(bits(he[w]), bits(we)), f"e' step {step} worker {w}"
            e[w] = we
        op = E.EF_OP_TOPK if kind == "topk" else E.EF_OP_RANDK
        for w in range(min(W, 3)):
            assert not (c.L.diag(ws[w], op) & E.DIAG_COUNT_MISMATCH), f"worker {w}: row counts do not add up"
