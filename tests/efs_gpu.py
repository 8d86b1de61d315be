"""Helpers for the GPU parity tests: run the library through its Python binding
on seeded inputs and compare with the CPU oracle bit for bit."""

import sys

import numpy as np

from oracle import efsparse_oracle as O


def announce(*what):
    print("[case]", *what, file=sys.stderr, flush=True)


def bits(x):
    return np.asarray(x, dtype=np.float32).view(np.uint32)


def dev(x):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x))
    return t.to("cuda")


def host(t):
    return t.detach().cpu().numpy()


class Case:
    """One layout on the GPU plus its oracle parameters."""

    def __init__(self, offs, density, block=1, tune=None):
        import paper_2009_09271_amd as E
        self.E = E
        self.offs = [int(o) for o in offs]
        self.d = self.offs[-1]
        self.density = density
        self.block = block
        self.ks = O.segment_ks(self.offs, density)
        self.K = sum(self.ks)
        self.L = E.Layout(self.d, self.offs, density, block, tune=tune).bind("cuda")
        assert self.L.K == self.K

    def ws(self, op, W=1):
        return self.L.workspace(op, W)

    # ---- one worker step through the fused entry points -------------------------------------
    def step(self, kind, g_host, e_dev, seed=0, step=0, ws=None):
        import torch
        E = self.E
        g = dev(g_host)
        if g_host.dtype == np.uint16:
            g = g.view(torch.bfloat16)
        val = torch.empty(self.K, dtype=torch.float32, device="cuda")
        if kind == "topk":
            idx = torch.empty(self.K, dtype=torch.int32, device="cuda")
            ws = self.ws(E.EF_OP_TOPK) if ws is None else ws
            E.ef_step_topk(self.L, g, e_dev, idx, val, ws)
            return idx, val, ws
        if kind == "randk":
            idx = torch.empty(self.K, dtype=torch.int32, device="cuda")
            ws = self.ws(E.EF_OP_RANDK) if ws is None else ws
            E.ef_step_randk(self.L, g, e_dev, seed, step, idx, val, ws)
            return idx, val, ws
        if kind == "randblock":
            start = torch.empty(len(self.ks), dtype=torch.int32, device="cuda")
            E.ef_step_randblock(self.L, g, e_dev, seed, step, start, val)
            return start, val, None
        raise ValueError(kind)

    # ---- the same step through the separate entry points -------------------------------------
    def step_composed(self, kind, g_host, e_dev, seed=0, step=0):
        import torch
        E = self.E
        g = dev(g_host)
        if g_host.dtype == np.uint16:
            g = g.view(torch.bfloat16)
        acc = torch.empty(self.d, dtype=torch.float32, device="cuda")
        E.ef_accumulate(self.L, g, e_dev, acc)
        val = torch.empty(self.K, dtype=torch.float32, device="cuda")
        m = torch.empty(self.K if kind != "randblock" else len(self.ks), dtype=torch.int32, device="cuda")
        if kind == "topk":
            E.compress_topk(self.L, acc, m, val, self.ws(E.EF_OP_TOPK))
            kindm = E.EF_MSG_SPARSE
        elif kind == "randk":
            E.compress_randk(self.L, acc, seed, step, m, val, self.ws(E.EF_OP_RANDK))
            kindm = E.EF_MSG_SPARSE
        else:
            E.compress_randblock(self.L, acc, seed, step, m, val)
            kindm = E.EF_MSG_BLOCK
        E.ef_update(self.L, acc, kindm, m, e_dev)
        return m, val

    def oracle_step(self, kind, g_host, e_host, seed=0, step=0):
        return O.ef_step(kind, g_host, e_host, self.offs, self.ks, seed=seed, step=step, block=self.block)


def assert_msg_equal(kind, got, want, where=""):
    m, val = got
    wm, wval = want
    m = host(m).view(np.uint32) if not isinstance(m, np.ndarray) else m
    val = host(val) if not isinstance(val, np.ndarray) else val
    assert m.shape == wm.shape, where
    bad = np.nonzero(m != wm)[0]
    assert bad.size == 0, f"{where}: {bad.size} {kind} index/start mismatches, first at {bad[:5]}: {m[bad[:5]]} vs {wm[bad[:5]]}"
    badv = np.nonzero(bits(val) != bits(wval))[0]
    assert badv.size == 0, f"{where}: {badv.size} value mismatches, first at {badv[:5]}"


def assert_f32_equal(got, want, where=""):
    got = host(got) if not isinstance(got, np.ndarray) else got
    bad = np.nonzero(bits(got) != bits(want))[0]
    assert bad.size == 0, f"{where}: {bad.size} mismatching elements, first {bad[:5]}: {got[bad[:5]]} vs {want[bad[:5]]}"


# ---- exact certificates for sizes where the full oracle sort is too slow ------------------------
# Each checks the definition directly: the sent set is unique given (key order, index order), so
# these properties hold for the oracle's answer and for no other set.

def _check_message_and_residual(acc, idx, val, e_new, where):
    idx = np.asarray(idx).view(np.uint32).astype(np.int64)
    assert np.array_equal(bits(val), bits(acc[idx])), f"{where}: values differ from acc at the indices"
    want = acc.copy()
    want[idx] = 0.0
    assert_f32_equal(e_new, want, f"{where}: residual")
    return idx


def certify_topk(acc, offs, ks, idx, val, e_new, where="topk"):
    """Per segment: k sorted distinct indices inside it; every unsent key <= the smallest sent key
    T; among keys equal to T the sent ones have the lower indices."""
    idx = _check_message_and_residual(acc, idx, val, e_new, where)
    key = acc.view(np.uint32) & np.uint32(0x7FFFFFFF)
    P = 0
    for l, k in enumerate(ks):
        o, n = offs[l], offs[l + 1] - offs[l]
        S = idx[P:P + k] - o
        P += k
        assert S.size == k and S.min() >= 0 and S.max() < n and np.all(np.diff(S) > 0), f"{where} seg {l}: support"
        seg = key[o:o + n]
        T = seg[S].min()
        sel = np.zeros(n, dtype=bool)
        sel[S] = True
        assert np.where(sel, np.uint32(0), seg).max() <= T, f"{where} seg {l}: an unsent key beats a sent one"
        tie_sent = S[seg[S] == T]
        tie_unsent = np.nonzero(~sel & (seg == T))[0]
        if tie_unsent.size:
            assert tie_sent.max() < tie_unsent.min(), f"{where} seg {l}: ties must go to lower indices"


def certify_randk(acc, offs, ks, idx, val, e_new, seed, step, where="randk"):
    """Per segment, with the oracle's Philox keys u: every unsent u >= the largest sent u T; among
    keys equal to T the sent ones have the lower indices."""
    idx = _check_message_and_residual(acc, idx, val, e_new, where)
    P = 0
    for l, k in enumerate(ks):
        o, n = offs[l], offs[l + 1] - offs[l]
        S = idx[P:P + k] - o
        P += k
        assert S.size == k and S.min() >= 0 and S.max() < n and np.all(np.diff(S) > 0), f"{where} seg {l}: support"
        u = O.randk_keys(n, l, seed, step)
        T = u[S].max()
        sel = np.zeros(n, dtype=bool)
        sel[S] = True
        assert np.where(sel, np.uint32(0xFFFFFFFF), u).min() >= T, f"{where} seg {l}: an unsent key beats a sent one"
        tie_sent = S[u[S] == T]
        tie_unsent = np.nonzero(~sel & (u == T))[0]
        if tie_unsent.size:
            assert tie_sent.max() < tie_unsent.min(), f"{where} seg {l}: ties must go to lower indices"


# ---- the same certificates, piece by piece (for segments of up to 1e9 elements) -----------------
# A segment's sent set S (k sorted distinct positions) is the definition's answer exactly when its
# worst member beats the best position outside it under the selection order (score descending,
# then index ascending).  Each piece of positions gives its worst sent and best unsent (score,
# -index) pair; the pieces run on host threads (NumPy releases the interpreter lock in its loops).

def _piece(S, a, b, score):
    sc = score(a, b)
    sel = np.zeros(b - a, dtype=bool)
    lo, hi = np.searchsorted(S, [a, b])
    sel[S[lo:hi] - a] = True
    worst = best = None
    if hi > lo:
        m = sc[sel].min()
        worst = (int(m), -int(np.nonzero(sel & (sc == m))[0].max() + a))
    uns = ~sel
    if uns.any():
        M = sc[uns].max()
        best = (int(M), -int(np.nonzero(uns & (sc == M))[0].min() + a))
    return worst, best


def order_certificate(S, n, k, score, where, chunk=1 << 24, threads=8):
    """S: sent local positions of a segment of n elements; score(a, b): uint32 scores of positions
    a..b-1 (larger is better).  Asserts |S| = k, S sorted, distinct and inside the segment, and that
    every sent position beats every unsent one (equal scores: the lower index wins)."""
    from concurrent.futures import ThreadPoolExecutor
    S = np.asarray(S, dtype=np.int64)
    assert S.size == k and S.min() >= 0 and S.max() < n and np.all(np.diff(S) > 0), f"{where}: support"
    bounds = [(a, min(n, a + chunk)) for a in range(0, n, chunk)]
    with ThreadPoolExecutor(max(1, min(threads, len(bounds)))) as ex:
        parts = list(ex.map(lambda ab: _piece(S, ab[0], ab[1], score), bounds))
    worst = min(p[0] for p in parts if p[0] is not None)
    bests = [p[1] for p in parts if p[1] is not None]
    if bests:
        best = max(bests)
        assert worst > best, f"{where}: an unsent position {-best[1]} (score {best[0]}) beats the sent " \
                             f"position {-worst[1]} (score {worst[0]})"


def certify_topk_chunked(acc, offs, ks, idx, val, e_new, where="topk", chunk=1 << 24):
    """certify_topk piece by piece: score = magnitude key."""
    idx = _check_message_and_residual(acc, idx, val, e_new, where)
    P = 0
    for l, k in enumerate(ks):
        o, n = offs[l], offs[l + 1] - offs[l]
        S = idx[P:P + k] - o
        P += k
        order_certificate(S, n, k, lambda a, b: acc[o + a:o + b].view(np.uint32) & np.uint32(0x7FFFFFFF),
                          f"{where} seg {l}", chunk)


def certify_randk_chunked(acc, offs, ks, idx, val, e_new, seed, step, where="randk", chunk=1 << 24):
    """certify_randk piece by piece, the oracle's keys computed per range: score = complement of
    the Philox key (smaller keys are better)."""
    idx = _check_message_and_residual(acc, idx, val, e_new, where)
    P = 0
    for l, k in enumerate(ks):
        o, n = offs[l], offs[l + 1] - offs[l]
        S = idx[P:P + k] - o
        P += k
        order_certificate(S, n, k, lambda a, b: ~O.randk_keys(n, l, seed, step, a, b), f"{where} seg {l}", chunk)


def topk_shaped_messages(grads, offs, ks):
    """Sparse messages with top-k's shape (each worker's largest magnitudes per segment, ascending
    indices; ties in any order), from the workers' gradients.  Test inputs only."""
    idx, val = [], []
    for g in grads:
        key = g.view(np.uint32) & np.uint32(0x7FFFFFFF)
        sup = []
        for l, k in enumerate(ks):
            o, n = offs[l], offs[l + 1] - offs[l]
            part = np.argpartition(key[o:o + n], n - k)[n - k:] if k < n else np.arange(n)
            sup.append(np.sort(part) + o)
        s = np.concatenate(sup).astype(np.uint32)
        idx.append(s)
        val.append(g[s.astype(np.int64)])
    return np.stack(idx), np.stack(val).astype(np.float32)


def synthetic_sparse_messages(d, K, W, seed):
    """W messages of K ascending distinct indices with random values (seeded; message shape only)."""
    rng = np.random.default_rng(seed)
    idx = np.stack([np.sort(rng.choice(d, size=K, replace=False)) for _ in range(W)]).astype(np.uint32)
    val = rng.standard_normal((W, K)).astype(np.float32)
    return idx, val
