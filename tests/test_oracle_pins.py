"""Pins for the CPU oracle: each check ties it to something other than itself
(brute force over subsets, library routines on special cases, an independent
Philox implementation, closed forms, invariants and hand-worked vectors under
tests/golden/).  CPU only."""

import itertools
import os
import shutil
import subprocess
import tempfile

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from conftest import golden
from oracle import efsparse_oracle as O
from oracle.philox import philox4x32_10


def f32_from_hex(hs):
    return np.array([int(h, 16) for h in hs], dtype=np.uint32).view(np.float32)


def bits(x):
    return np.asarray(x, dtype=np.float32).view(np.uint32)


# ----------------------------------------------------------------------------- k per segment
def test_k_rule_examples_and_workload_sizes():
    g = golden("k_sizes.json")
    for ex in g["examples"]:
        assert O.k_rule(ex["d"], ex["density"]) == ex["k"]
    from workloads import WORKLOADS
    for w in g["workloads"]:
        wl = WORKLOADS[w["name"]]
        assert wl.d == w["d"]
        assert len(wl.seg_offsets("layer")) - 1 == w["segments"]
        assert sum(O.segment_ks(wl.seg_offsets("flat"), w["density"])) == w["K_flat"]
        assert sum(O.segment_ks(wl.seg_offsets("layer"), w["density"])) == w["K_layer"]


@given(st.integers(1, 10**9), st.floats(1e-9, 1.0))
def test_k_rule_bounds(d, rho):
    k = O.k_rule(d, rho)
    assert 1 <= k <= d
    # within half an element of rho*d unless clamped
    if 1 < k < d:
        assert abs(k - rho * d) <= 0.5 + 1e-9 * d


# ----------------------------------------------------------------------------- accumulate
def test_accumulate_matches_torch_float32_add():
    import torch
    rng = np.random.default_rng(1)
    g = (rng.standard_normal(4096) * 10.0 ** rng.integers(-30, 30, 4096)).astype(np.float32)
    e = (rng.standard_normal(4096) * 10.0 ** rng.integers(-30, 30, 4096)).astype(np.float32)
    g[:4] = [1.0, -0.0, 0.0, 1.0]
    e[:4] = [2.0 ** -24, -0.0, -0.0, 2.0 ** -23]  # tie to even, signed zeros
    want = (torch.from_numpy(g) + torch.from_numpy(e)).numpy()
    assert np.array_equal(bits(O.ef_accumulate(g, e)), bits(want))
    assert bits(O.ef_accumulate(g, e))[0] == bits(np.float32(1.0))
    assert bits(O.ef_accumulate(g, e))[1] == 0x80000000
    assert bits(O.ef_accumulate(g, e))[2] == 0


def test_bf16_widening_matches_torch():
    import torch
    b = np.arange(0, 1 << 16, 7, dtype=np.uint32).astype(np.uint16)
    b = b[(b & 0x7F80) != 0x7F80]  # skip Inf/NaN patterns
    want = torch.from_numpy(b.view(np.int16)).view(torch.bfloat16).float().numpy()
    assert np.array_equal(bits(O.bf16_to_f32(b)), bits(want))


def test_bf16_rounding_of_generator_matches_torch():
    import torch
    from workloads import to_bf16_bits
    x = (np.random.default_rng(3).standard_normal(100000) * 1e-3).astype(np.float32)
    want = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(to_bf16_bits(x), want)


# ----------------------------------------------------------------------------- top-k
def test_topk_hand_vector_x1():
    g = golden("x1_topk_ties.json")
    acc = f32_from_hex(g["acc_hex"])
    for case in g["cases"]:
        idx, val = O.compress_topk(acc, [0, len(acc)], [case["k"]])
        assert idx.tolist() == case["idx"]
        if "val_hex" in case:
            assert np.array_equal(bits(val), bits(f32_from_hex(case["val_hex"])))
        if "e_hex" in case:
            assert np.array_equal(bits(O.ef_update(acc, idx)), bits(f32_from_hex(case["e_hex"])))


def test_ef_three_steps_x2():
    g = golden("x2_ef_three_steps.json")
    e = np.zeros(g["d"], np.float32)
    for s in g["steps"]:
        (idx, val), e = O.ef_step("topk", np.array(s["g"], np.float32), e, [0, g["d"]], [g["k"]])
        assert idx.tolist() == s["idx"] and val.tolist() == s["val"] and e.tolist() == s["e"]


def _dominance_ok(key, sel):
    """Every sent entry beats every unsent one: larger magnitude key, or equal
    key and lower index.  (Pairwise characterisation of top-k with ties.)"""
    n = len(key)
    for i in sel:
        for j in range(n):
            if j in sel:
                continue
            if not (key[i] > key[j] or (key[i] == key[j] and i < j)):
                return False
    return True


def test_topk_brute_force_all_subsets():
    rng = np.random.default_rng(7)
    pool = np.array([0.0, -0.0, 0.5, -0.5, 0.25, -0.25, 1.0, 3e-39, -3e-39, np.inf, -np.inf], np.float32)
    for trial in range(300):
        n = int(rng.integers(1, 9))
        acc = rng.choice(pool, size=n)
        key = O.magnitude_key(acc).astype(np.int64)
        k = int(rng.integers(1, n + 1))
        winners = [set(c) for c in itertools.combinations(range(n), k) if _dominance_ok(key, set(c))]
        assert len(winners) == 1
        idx, val = O.compress_topk(acc, [0, n], [k])
        assert set(idx.tolist()) == winners[0]
        assert np.all(np.diff(idx.astype(np.int64)) > 0)
        assert np.array_equal(bits(val), bits(acc[idx]))


def test_topk_special_cases_library_routines():
    rng = np.random.default_rng(11)
    for _ in range(50):
        n = int(rng.integers(2, 3000))
        acc = np.round(rng.standard_normal(n) * 4).astype(np.float32) / 4  # many ties
        # k = 1: first occurrence of the largest magnitude (numpy argmax)
        idx, _ = O.compress_topk(acc, [0, n], [1])
        assert idx.tolist() == [int(np.argmax(np.abs(acc)))]
        # k = n: everything
        idx, _ = O.compress_topk(acc, [0, n], [n])
        assert idx.tolist() == list(range(n))
        # distinct magnitudes: same set as numpy argpartition
        x = rng.permutation(n).astype(np.float32) * np.where(rng.random(n) < 0.5, -1, 1).astype(np.float32)
        k = int(rng.integers(1, n))
        idx, _ = O.compress_topk(x, [0, n], [k])
        want = np.sort(np.argpartition(-np.abs(x), k - 1)[:k])
        assert idx.tolist() == want.tolist()


def test_topk_layerwise_is_per_segment():
    rng = np.random.default_rng(5)
    offs = [0, 1, 5, 64, 65, 300, 301]
    acc = rng.standard_normal(offs[-1]).astype(np.float32)
    ks = O.segment_ks(offs, 0.1)
    idx, _ = O.compress_topk(acc, offs, ks)
    P = O.message_offsets(ks)
    for l in range(len(ks)):
        seg = idx[P[l]:P[l + 1]].astype(np.int64)
        assert len(seg) == ks[l] and np.all((seg >= offs[l]) & (seg < offs[l + 1]))
        n = offs[l + 1] - offs[l]
        key = O.magnitude_key(acc[offs[l]:offs[l + 1]])
        sel = set((seg - offs[l]).tolist())
        if n <= 12:
            assert _dominance_ok(key.astype(np.int64), sel)
        else:  # O(n) certificate: min sent (key desc, idx asc) beats max unsent
            uns = np.array(sorted(set(range(n)) - sel))
            s = np.array(sorted(sel))
            worst_sent = min(zip(key[s].astype(np.int64), -s))
            best_unsent = max(zip(key[uns].astype(np.int64), -uns))
            assert worst_sent > best_unsent


# ----------------------------------------------------------------------------- Philox
def _aten_helper():
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    import torch
    inc = os.path.join(os.path.dirname(torch.__file__), "include")
    out = os.path.join(tempfile.gettempdir(), "efsparse_philox_aten_ref")
    src = os.path.join(os.path.dirname(__file__), "philox_aten_ref.cpp")
    if not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(src):
        subprocess.check_call([gxx, "-O1", "-std=c++17", "-I" + inc, src, "-o", out])
    return out


def _aten(triples):
    exe = _aten_helper()
    inp = "".join(f"{s} {u} {o}\n" for s, u, o in triples)
    res = subprocess.run([exe], input=inp, capture_output=True, text=True, check=True).stdout.split("\n")
    return [tuple(int(w, 16) for w in line.split()) for line in res if line.strip()]


def test_philox_matches_independent_implementation():
    rng = np.random.default_rng(2024)
    triples = [(0, 0, 0), (2**64 - 1, 2**64 - 1, 2**64 - 1), (1, 2, 3)]
    triples += [tuple(int(v) for v in rng.integers(0, 2**63, 3, dtype=np.uint64) * 2 + rng.integers(0, 2, 3, dtype=np.uint64))
                for _ in range(200)]
    want = _aten(triples)
    for (seed, sub, off), w in zip(triples, want):
        got = philox4x32_10(off & 0xFFFFFFFF, off >> 32, sub & 0xFFFFFFFF, sub >> 32, seed & 0xFFFFFFFF, seed >> 32)
        assert tuple(int(v) for v in got) == w


def test_randk_key_mapping_matches_independent_philox():
    seed, step = (3 << 32) | 17, 9
    for l, n in ((0, 1000), (5, 37)):
        u = O.randk_keys(n, l, seed, step)
        js = list(range(0, n, 7)) + [n - 1]
        sub = step | ((O.RANDK_TAG | l) << 32)
        want = _aten([(seed, sub, j >> 2) for j in js])
        for j, w in zip(js, want):
            assert int(u[j]) == w[j & 3]


def test_randk_key_ranges_match_independent_philox():
    """Keys of a position range (the form the certificates of 1e9-element segments use) at offsets
    far into a segment, including ranges that start and end inside a Philox block, against ATen;
    and every range of a small segment equals the same slice of the whole-segment call."""
    seed, step, n = (4 << 32) | 5, 3, 1_000_000_000
    for l, j0, m in ((0, 999_999_963, 37), (0, 123_456_789, 11), (2, 536_870_910, 9)):
        u = O.randk_keys(n, l, seed, step, j0, j0 + m)
        assert u.shape == (m,)
        sub = step | ((O.RANDK_TAG | l) << 32)
        want = _aten([(seed, sub, j >> 2) for j in range(j0, j0 + m)])
        for t, w in enumerate(want):
            assert int(u[t]) == w[(j0 + t) & 3]
    full = O.randk_keys(1001, 6, seed, step)
    rng = np.random.default_rng(11)
    for _ in range(50):
        a, b = sorted(int(v) for v in rng.integers(0, 1002, 2))
        assert np.array_equal(O.randk_keys(1001, 6, seed, step, a, b), full[a:b])


def test_randblock_start_matches_independent_philox():
    seed = (2 << 32) | 3
    for l, n, b in ((0, 25557032, 4096), (7, 1000, 256), (3, 64, 256), (1, 10, 2)):
        for step in range(5):
            (w,) = _aten([(seed, step | ((O.RANDBLOCK_TAG | l) << 32), 0)])
            r = w[0] | (w[1] << 32)
            bl = b if n > b else 1
            nb = -(-n // bl)
            assert O.randblock_start(n, l, b, seed, step) == bl * ((r * nb) >> 64)


def test_philox_output_is_uniform():
    c = np.arange(1 << 16, dtype=np.uint64)
    x = np.concatenate(philox4x32_10(c, 0, 1, 2, 3, 4))
    counts = np.bincount(x >> np.uint32(24), minlength=256)
    from scipy.stats import chisquare
    assert chisquare(counts).pvalue > 1e-4


# ----------------------------------------------------------------------------- random-k
def test_randk_certificates():
    rng = np.random.default_rng(8)
    for trial in range(40):
        offs = np.concatenate([[0], np.cumsum(rng.integers(1, 400, size=int(rng.integers(1, 6))))]).tolist()
        ks = O.segment_ks(offs, float(rng.uniform(0.001, 1.0)))
        seed, step = int(rng.integers(0, 2**63)), int(rng.integers(0, 2**32))
        idx = O.randk_support(offs, ks, seed, step)
        P = O.message_offsets(ks)
        for l, k in enumerate(ks):
            n = offs[l + 1] - offs[l]
            seg = idx[P[l]:P[l + 1]].astype(np.int64) - offs[l]
            assert len(seg) == k and np.all(np.diff(seg) > 0) and seg.min() >= 0 and seg.max() < n
            u = O.randk_keys(n, l, seed, step).astype(np.int64)
            sel = np.zeros(n, bool)
            sel[seg] = True
            if 0 < k < n:  # the k sent keys are the k smallest (ties: lower index)
                worst_sent = max(zip(u[sel], np.nonzero(sel)[0]))
                best_unsent = min(zip(u[~sel], np.nonzero(~sel)[0]))
                assert worst_sent < best_unsent
        assert np.array_equal(idx, O.randk_support(offs, ks, seed, step))


def test_randk_seed_and_step_change_the_choice():
    offs, ks = [0, 100000], [100]
    a = O.randk_support(offs, ks, 1, 0)
    assert not np.array_equal(a, O.randk_support(offs, ks, 2, 0))
    assert not np.array_equal(a, O.randk_support(offs, ks, 1, 1))


def test_randk_inclusion_frequency_is_k_over_d():
    n, k, steps = 200, 10, 4000
    counts = np.zeros(n)
    for t in range(steps):
        counts[O.randk_support([0, n], [k], 99, t).astype(np.int64)] += 1
    p = k / n
    sd = np.sqrt(steps * p * (1 - p))
    assert np.all(np.abs(counts - steps * p) < 5.5 * sd)


# ----------------------------------------------------------------------------- random-block
def test_randblock_wrap_x3():
    g = golden("x3_randblock_wrap.json")
    s = g["b"] * g["start_block"]
    assert s == g["start"]
    assert O.randblock_positions(g["d"], g["k"], s).tolist() == g["positions"]


def test_randblock_support_is_one_wrapped_run():
    rng = np.random.default_rng(4)
    for _ in range(100):
        offs = np.concatenate([[0], np.cumsum(rng.integers(1, 3000, size=int(rng.integers(1, 5))))]).tolist()
        b = int(rng.choice([1, 2, 16, 256, 4096]))
        ks = O.segment_ks(offs, float(rng.uniform(0.001, 1.0)))
        seed, step = int(rng.integers(0, 2**63)), int(rng.integers(0, 1000))
        acc = rng.standard_normal(offs[-1]).astype(np.float32)
        start, val = O.compress_randblock(acc, offs, ks, b, seed, step)
        P = O.message_offsets(ks)
        for l, k in enumerate(ks):
            n = offs[l + 1] - offs[l]
            bl = b if n > b else 1
            s = int(start[l])
            assert 0 <= s < n and s % bl == 0
            pos = [(s + t) % n for t in range(k)]
            assert len(set(pos)) == k
            assert np.array_equal(bits(val[P[l]:P[l + 1]]), bits(acc[offs[l] + np.array(pos)]))


def test_randblock_start_uniform():
    from scipy.stats import chisquare
    n, b = 64 * 100, 64
    starts = [O.randblock_start(n, 0, b, 12345, t) // b for t in range(20000)]
    assert chisquare(np.bincount(starts, minlength=100)).pvalue > 1e-4


def test_randblock_full_density_is_rotation():
    acc = np.arange(1, 11, dtype=np.float32)
    start, val = O.compress_randblock(acc, [0, 10], [10], 1, 77, 3)
    assert np.array_equal(val, np.roll(acc, -int(start[0])))


# ----------------------------------------------------------------------------- residual identity
@pytest.mark.parametrize("kind", ["topk", "randk", "randblock"])
def test_residual_identity(kind):
    rng = np.random.default_rng(12)
    offs = [0, 3, 700, 701, 5000]
    ks = O.segment_ks(offs, 0.05)
    g = rng.standard_normal(offs[-1]).astype(np.float32)
    e = (rng.standard_normal(offs[-1]) * 0.1).astype(np.float32)
    g[10] = -0.0
    e[10] = -0.0
    acc = O.ef_accumulate(g, e)
    (m0, val), e2 = O.ef_step(kind, g, e, offs, ks, seed=5, step=1, block=64)
    sup = O.block_support(offs, ks, m0) if kind == "randblock" else m0.astype(np.int64)
    assert len(set(sup.tolist())) == sum(ks)
    sent = np.zeros_like(acc)
    sent[sup] = val
    assert np.array_equal(acc, sent + e2)  # value equality (-0 == +0)
    on = np.zeros(len(acc), bool)
    on[sup] = True
    assert np.all(bits(e2[on]) == 0)
    assert np.array_equal(bits(e2[~on]), bits(acc[~on]))


# ----------------------------------------------------------------------------- aggregate
def test_aggregate_order_x4():
    g = golden("x4_aggregate_order.json")
    sup = [w["idx"] for w in g["workers"]]
    val = [np.array(w["val"], np.float32) for w in g["workers"]]
    assert O.decompress_aggregate(g["d"], sup, val, average=False).tolist() == [g["sum"]]
    assert O.decompress_aggregate(g["d"], sup, val).tolist() == [g["mean"]]


def test_aggregate_signed_zero_x5():
    g = golden("x5_aggregate_signed_zero.json")
    sup = [w["idx"] for w in g["workers"]]
    val = [f32_from_hex(w["val_hex"]) for w in g["workers"]]
    out = O.decompress_aggregate(g["d"], sup, val)
    assert bits(out)[0] == int(g["mean_hex"], 16)


def test_aggregate_exact_dyadic_matches_float64():
    rng = np.random.default_rng(9)
    d, W = 5000, 8
    sups, vals = [], []
    for w in range(W):
        s = np.sort(rng.choice(d, size=500, replace=False))
        sups.append(s)
        vals.append((rng.integers(-1000, 1000, size=500) / 64.0).astype(np.float32))
    ref = np.zeros(d)
    for s, v in zip(sups, vals):
        np.add.at(ref, s, v.astype(np.float64))
    assert np.array_equal(O.decompress_aggregate(d, sups, vals, average=False), ref.astype(np.float32))
    assert np.array_equal(O.decompress_aggregate(d, sups, vals), (ref / W).astype(np.float32))


def test_aggregate_single_worker_is_scatter():
    rng = np.random.default_rng(10)
    d = 1000
    s = np.sort(rng.choice(d, 50, replace=False))
    v = rng.standard_normal(50).astype(np.float32)
    want = np.zeros(d, np.float32)
    want[s] = v
    assert np.array_equal(bits(O.decompress_aggregate(d, [s], [v])), bits(want))


def test_randblock_segment_not_longer_than_block_uses_unit_alignment():
    # A segment of d_l <= b elements cannot hold two aligned starts, so its
    # start is unaligned (b_l = 1) and spreads over all d_l positions.
    for n in (256, 100):
        starts = {O.randblock_start(n, 3, 256, 4242, t) for t in range(3000)}
        assert starts == set(range(n))
    # one element more than b: aligned starts 0 and b only
    starts = {O.randblock_start(257, 3, 256, 4242, t) for t in range(200)}
    assert starts == {0, 256}


# ----------------------------------------------------------------------------- shared coordinates
def test_shared_sparse_aggregate_is_dense_sum_of_aligned_values():
    """With one index list for every worker, the aggregate at idx[j] is the ordered float32 sum of
    the workers' j-th values (a plain column sum of the [W][K] value matrix, worker by worker),
    divided by W; zero elsewhere."""
    rng = np.random.default_rng(3)
    d, W, K = 500, 5, 37
    idx = np.sort(rng.choice(d, K, replace=False)).astype(np.uint32)
    V = (rng.standard_normal((W, K)) * 10.0 ** rng.integers(-3, 3, (W, 1))).astype(np.float32)
    col = np.zeros(K, np.float32)
    for w in range(W):
        col = col + V[w]
    want = np.zeros(d, np.float32)
    want[idx.astype(np.int64)] = col / np.float32(W)
    got = O.decompress_aggregate_shared_sparse(d, idx, V)
    assert np.array_equal(bits(got), bits(want))


def test_shared_block_aggregate_matches_general_with_repeated_starts():
    offs = [0, 7, 100, 1000]
    ks = O.segment_ks(offs, 0.1)
    rng = np.random.default_rng(4)
    start = np.array([3, 40, 512], dtype=np.uint32)
    V = rng.standard_normal((3, sum(ks))).astype(np.float32)
    a = O.decompress_aggregate_shared_block(1000, offs, ks, start, V)
    b = O.decompress_aggregate_block(1000, offs, ks, [start] * 3, list(V))
    assert np.array_equal(bits(a), bits(b))


# ----------------------------------------------------------------------------- parameter update
def test_apply_update_plain_is_subtraction():
    """Algorithm 1's update without momentum or weight decay: x - q (NumPy's float32 subtract)."""
    rng = np.random.default_rng(5)
    x = rng.standard_normal(1000).astype(np.float32)
    q = (rng.standard_normal(1000) * 1e-3).astype(np.float32)
    x2, m2 = O.apply_update(x, q)
    assert m2 is None
    assert np.array_equal(bits(x2), bits(np.subtract(x, q, dtype=np.float32)))


def test_apply_update_exact_dyadic():
    """Small dyadic values with beta = 1/2 and wd = 1/4: every operation is exact, so the result
    equals the formula evaluated in float64."""
    rng = np.random.default_rng(6)
    x = rng.integers(-64, 64, 200).astype(np.float32) / 8
    q = rng.integers(-64, 64, 200).astype(np.float32) / 16
    m = rng.integers(-64, 64, 200).astype(np.float32) / 4
    x2, m2 = O.apply_update(x, q, m, beta=0.5, wd=0.25)
    d = q.astype(np.float64) + 0.25 * x.astype(np.float64)
    mm = 0.5 * m.astype(np.float64) + d
    assert np.array_equal(m2.astype(np.float64), mm)
    assert np.array_equal(x2.astype(np.float64), x.astype(np.float64) - mm)


def test_apply_update_matches_torch_sgd():
    """Three steps with the buffer carried, against torch.optim.SGD on the CPU (lr = 1, momentum,
    weight decay, no dampening): the same order of operations, within one float32 rounding of
    each value (torch may fuse the weight-decay multiply-add)."""
    import torch
    rng = np.random.default_rng(7)
    x = rng.standard_normal(4096).astype(np.float32)
    p = torch.nn.Parameter(torch.from_numpy(x.copy()))
    opt = torch.optim.SGD([p], lr=1.0, momentum=0.9, weight_decay=1e-4, dampening=0.0, nesterov=False)
    m = np.zeros_like(x)
    for t in range(3):
        q = (rng.standard_normal(4096) * 1e-2).astype(np.float32)
        p.grad = torch.from_numpy(q.copy())
        opt.step()
        x, m = O.apply_update(x, q, m, beta=0.9, wd=1e-4)
        ref = p.detach().numpy()
        assert np.allclose(x, ref, rtol=2 ** -22, atol=1e-7), f"step {t}"


# ----------------------------------------------------------------------------- dense average
def test_dense_average_exact_integers_match_numpy_sum():
    """Integer-valued gradients: every partial sum is exact, so the ordered sum equals NumPy's sum
    (any order) and the average its float32 division."""
    rng = np.random.default_rng(8)
    G = rng.integers(-1000, 1000, (6, 999)).astype(np.float32)
    want = (G.astype(np.float64).sum(axis=0).astype(np.float32)) / np.float32(6)
    assert np.array_equal(bits(O.dense_average(G)), bits(want))
    assert np.array_equal(bits(O.dense_average(G, average=False)), bits(G.astype(np.float64).sum(axis=0).astype(np.float32)))


def test_dense_average_worker_order_and_single_worker():
    """(1 + 1e8) - 1e8 = 0 in float32 (the spacing at 1e8 is 8), while 1 + (1e8 - 1e8) = 1: the
    sum runs in worker order.  One worker: the gradient itself (division by 1)."""
    G = np.array([[1.0], [1e8], [-1e8]], np.float32)
    assert O.dense_average(G, average=False)[0] == 0.0
    g = np.random.default_rng(9).standard_normal((1, 50)).astype(np.float32)
    assert np.array_equal(bits(O.dense_average(g)), bits(g[0]))


def test_dense_average_close_to_float64_mean():
    rng = np.random.default_rng(10)
    G = rng.standard_normal((16, 5000)).astype(np.float32)
    ref = G.astype(np.float64).mean(axis=0)
    assert np.max(np.abs(O.dense_average(G) - ref)) < 16 * 2 ** -23 * np.max(np.abs(G).sum(axis=0))
