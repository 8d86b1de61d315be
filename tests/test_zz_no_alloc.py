"""GPU test of decompress_aggregate_noalloc, the aggregate for callers that cannot allocate: called
through the C ABI, it must give bitwise the result of decompress_aggregate (and of the oracle) on
consecutive calls that share the library's static scratch, the second with a smaller input, and it
must refuse a tile table larger than that scratch before anything is enqueued."""

import ctypes

import numpy as np
import pytest

from efs_gpu import Case, announce, assert_f32_equal, dev, host, synthetic_sparse_messages
from oracle import efsparse_oracle as O

pytestmark = pytest.mark.gpu


def _noalloc(E, c, kind, W, m, v, out):
    import torch
    st = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    return E.lib().decompress_aggregate_noalloc(c.L.handle, kind, W, ctypes.c_void_p(m.data_ptr()),
                                                ctypes.c_void_p(v.data_ptr()), 1, ctypes.c_void_p(out.data_ptr()),
                                                st)


def _sparse_case(E, offs, density, W, seed):
    import torch
    c = Case(offs, density)
    idx, val = synthetic_sparse_messages(c.d, c.K, W, seed)
    m, v = dev(idx.view(np.int32)), dev(val)
    out = torch.full((c.d,), 7.0, dtype=torch.float32, device="cuda")
    assert _noalloc(E, c, E.EF_MSG_SPARSE, W, m, v, out) == E.EF_OK
    ref = torch.empty(c.d, dtype=torch.float32, device="cuda")
    E.decompress_aggregate(c.L, E.EF_MSG_SPARSE, W, m, v, ref, c.L.workspace(E.EF_OP_AGG_SPARSE, W))
    torch.cuda.synchronize()
    assert_f32_equal(out, host(ref), f"noalloc vs decompress_aggregate d={c.d} W={W}")
    assert_f32_equal(out, O.decompress_aggregate_sparse(c.d, idx, val), f"noalloc vs oracle d={c.d} W={W}")


def test_noalloc_aggregate_matches_the_workspace_form_on_consecutive_calls():
    import paper_2009_09271_amd as E
    announce("decompress_aggregate_noalloc: two calls, the second smaller")
    # first call: 5 ragged segments, 12 workers; second: a smaller layout and 3 workers, so the
    # scratch still holds the first call's larger table when the second runs
    _sparse_case(E, [0, 3, 70001, 70002, 250000, 300000], 0.01, 12, 91)
    _sparse_case(E, [0, 50000], 0.02, 3, 92)


def test_noalloc_block_aggregate_and_the_size_limit():
    import torch
    import paper_2009_09271_amd as E
    announce("decompress_aggregate_noalloc: block messages, size limit")
    c = Case([0, 4000, 4001, 100000], 0.05, 512)
    W = 5
    starts, vals = [], []
    rng = np.random.default_rng(93)
    for w in range(W):
        g = rng.standard_normal(c.d).astype(np.float32)
        s, v = O.compress_randblock(g, c.offs, c.ks, 512, 1000 + w, 0)
        starts.append(s)
        vals.append(v)
    st, va = np.stack(starts), np.stack(vals)
    out = torch.empty(c.d, dtype=torch.float32, device="cuda")
    assert _noalloc(E, c, E.EF_MSG_BLOCK, W, dev(st.view(np.int32)), dev(va), out) == E.EF_OK
    assert_f32_equal(out, O.decompress_aggregate_block(c.d, c.offs, c.ks, st, va), "noalloc block vs oracle")
    # a tile table beyond the static scratch is refused before anything is enqueued
    cap = int(E.lib().ef_noalloc_scratch_bytes())
    big = Case([0, 1 << 24], 1e-4)
    Wb = cap // (4 * ((1 << 24) // 1024 + 1)) + 1
    assert big.L.workspace_bytes(E.EF_OP_AGG_SPARSE, Wb) > cap
    m = torch.zeros(Wb * big.K, dtype=torch.int32, device="cuda")
    v = torch.zeros(Wb * big.K, dtype=torch.float32, device="cuda")
    ob = torch.full((big.d,), 3.0, dtype=torch.float32, device="cuda")
    assert _noalloc(E, big, E.EF_MSG_SPARSE, Wb, m, v, ob) == E.EF_EWORKSPACE
    torch.cuda.synchronize()
    assert bool(torch.all(ob == 3.0))
