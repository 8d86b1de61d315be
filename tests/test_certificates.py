"""CPU checks of the piecewise certificates the largest GPU parity cases rely on: they accept the
oracle's answer for every piece size and reject answers with a planted mistake (a beaten member,
a tie given to the higher index, a wrong value or residual)."""

import numpy as np
import pytest

from efs_gpu import certify_randk_chunked, certify_topk_chunked, topk_shaped_messages
from oracle import efsparse_oracle as O


def _layout(rng):
    offs = np.concatenate([[0], np.cumsum(rng.integers(1, 500, size=int(rng.integers(1, 5))))]).tolist()
    ks = O.segment_ks(offs, float(rng.choice([0.01, 0.1, 0.5, 1.0])))
    return offs, ks


def _acc(rng, d):
    a = (rng.standard_normal(d) * 10.0 ** rng.integers(-3, 1, d)).astype(np.float32)
    a[rng.random(d) < 0.2] = 0.0  # ties on zeros
    a[rng.random(d) < 0.1] = np.float32(0.5)  # ties on a repeated value
    return a


@pytest.mark.parametrize("chunk", [1, 7, 64, 1 << 20])
def test_certificates_accept_the_oracle_answer(chunk):
    rng = np.random.default_rng(chunk)
    for _ in range(20):
        offs, ks = _layout(rng)
        acc = _acc(rng, offs[-1])
        idx, val = O.compress_topk(acc, offs, ks)
        certify_topk_chunked(acc, offs, ks, idx, val, O.ef_update(acc, idx), chunk=chunk)
        seed, step = int(rng.integers(0, 2**63)), int(rng.integers(0, 100))
        idx, val = O.compress_randk(acc, offs, ks, seed, step)
        certify_randk_chunked(acc, offs, ks, idx, val, O.ef_update(acc, idx), seed, step, chunk=chunk)


def test_certificates_reject_planted_mistakes():
    rng = np.random.default_rng(4)
    offs = [0, 300, 301, 900]
    ks = O.segment_ks(offs, 0.1)
    acc = _acc(rng, offs[-1])
    idx, val = O.compress_topk(acc, offs, ks)
    e = O.ef_update(acc, idx)
    key = acc.view(np.uint32) & np.uint32(0x7FFFFFFF)
    # a sent position replaced by a strictly smaller unsent one in the same segment
    bad = idx.copy()
    seg0 = np.setdiff1d(np.arange(300), idx[:ks[0]])
    j = seg0[np.argmin(key[seg0])]
    if key[j] < key[idx[:ks[0]]].min():
        bad[0] = j
        bad[:ks[0]] = np.sort(bad[:ks[0]])
        with pytest.raises(AssertionError):
            certify_topk_chunked(acc, offs, ks, bad, acc[bad.astype(np.int64)], O.ef_update(acc, bad), chunk=13)
    # a wrong value, a wrong residual
    with pytest.raises(AssertionError):
        v = val.copy()
        v[1] = -v[1] if v[1] != 0 else 1.0
        certify_topk_chunked(acc, offs, ks, idx, v, e)
    with pytest.raises(AssertionError):
        e2 = e.copy()
        e2[int(idx[2])] = 1.0
        certify_topk_chunked(acc, offs, ks, idx, val, e2)
    # ties: all-equal keys, the sent set must be the lowest indices
    flat = np.full(64, 0.5, dtype=np.float32)
    kk = [5]
    good = np.arange(5, dtype=np.uint32)
    certify_topk_chunked(flat, [0, 64], kk, good, flat[:5], O.ef_update(flat, good), chunk=3)
    late = np.array([0, 1, 2, 3, 40], dtype=np.uint32)
    with pytest.raises(AssertionError):
        certify_topk_chunked(flat, [0, 64], kk, late, flat[late.astype(np.int64)], O.ef_update(flat, late), chunk=3)
    # random-k: a set chosen with another seed is rejected
    seed = 77
    ridx, rval = O.compress_randk(acc, offs, ks, seed + 1, 0)
    with pytest.raises(AssertionError):
        certify_randk_chunked(acc, offs, ks, ridx, rval, O.ef_update(acc, ridx), seed, 0, chunk=50)


def test_topk_shaped_messages_are_the_largest_per_segment():
    rng = np.random.default_rng(9)
    offs = [0, 1000, 1001, 5000]
    ks = O.segment_ks(offs, 0.05)
    grads = [rng.standard_normal(offs[-1]).astype(np.float32) for _ in range(3)]  # distinct magnitudes
    idx, val = topk_shaped_messages(grads, offs, ks)
    for w, g in enumerate(grads):
        want, wv = O.compress_topk(g, offs, ks)
        assert np.array_equal(idx[w], want) and np.array_equal(val[w].view(np.uint32), wv.view(np.uint32))
