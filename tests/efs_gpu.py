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


def synthetic_sparse_messages(d, K, W, seed):
    """W messages of K ascending distinct indices with random values (seeded; message shape only)."""
    rng = np.random.default_rng(seed)
    idx = np.stack([np.sort(rng.choice(d, size=K, replace=False)) for _ in range(W)]).astype(np.uint32)
    val = rng.standard_normal((W, K)).astype(np.float32)
    return idx, val
