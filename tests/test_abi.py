"""C-ABI contract tests that need no GPU: the library loads, exports every
function include/efsparse.h declares, and its host-side logic (layout
validation, k per segment, workspace sizing, status codes) behaves as the
header states.  No kernel is launched here."""

import ctypes
import os
import re

import numpy as np
import pytest

from conftest import ROOT

E = pytest.importorskip("paper_2009_09271_amd")
from oracle import efsparse_oracle as O  # noqa: E402


def header_functions():
    text = open(os.path.join(ROOT, "include", "efsparse.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[a-z0-9_]+\s*\*?\s*([a-z_][a-z0-9_]*)\s*\(", text, flags=re.M)))


def test_header_declares_the_entry_points():
    names = header_functions()
    for n in ("ef_accumulate", "compress_topk", "compress_randk", "compress_randblock", "ef_update",
              "decompress_aggregate", "ef_step_topk", "ef_step_randk", "ef_step_randblock"):
        assert n in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(E.LIB_PATH)
    for n in header_functions():
        assert hasattr(lib, n), n
    assert set(header_functions()) == set(E.EXPORTED)


def test_binding_names_match_c_names():
    for n in ("ef_accumulate", "compress_topk", "compress_randk", "compress_randblock", "ef_update",
              "decompress_aggregate", "ef_step_topk", "ef_step_randk", "ef_step_randblock"):
        assert callable(getattr(E, n))


@pytest.mark.parametrize("offs,rho", [([0, 1 << 20], 0.01), ([0, 1, 5, 64, 65, 300, 301, 10007], 0.29),
                                      ([0, 100], 0.29), ([0, 7], 1.0), ([0, 3, 4], 1e-9)])
def test_segment_k_matches_oracle_rule(offs, rho):
    L = E.Layout(offs[-1], offs, rho, 16)
    assert L.segment_k().tolist() == O.segment_ks(offs, rho)
    assert L.K == sum(O.segment_ks(offs, rho))


def test_workload_sizes():
    from workloads import RESNET18, RESNET50, BERT
    for wl, rho in ((RESNET18, 0.01), (RESNET50, 0.001), (BERT, 0.1)):
        for scope in ("flat", "layer"):
            offs = wl.seg_offsets(scope)
            assert E.Layout(offs[-1], offs, rho, 4096).K == sum(O.segment_ks(offs, rho))


def _create(d, offs, rho=0.1, block=1):
    arr = np.asarray(offs, dtype=np.int64)
    h = ctypes.c_void_p()
    rc = E.lib().ef_layout_create(d, arr.ctypes.data, len(offs) - 1, rho, block, ctypes.byref(h))
    if rc == 0:
        E.lib().ef_layout_destroy(h)
    return rc


def test_layout_create_status_codes():
    assert _create(10, [0, 10]) == E.EF_OK
    assert _create(0, [0, 0]) == E.EF_ERANGE
    assert _create(1 << 31, [0, 1 << 31]) == E.EF_ERANGE
    assert _create((1 << 31) - 1, [0, (1 << 31) - 1]) == E.EF_OK
    assert _create(10, [0, 5, 5, 10]) == E.EF_EINVAL      # empty segment
    assert _create(10, [0, 6, 5, 10]) == E.EF_EINVAL      # not increasing
    assert _create(10, [1, 10]) == E.EF_EINVAL            # does not start at 0
    assert _create(10, [0, 9]) == E.EF_EINVAL             # does not end at d
    assert _create(10, [0, 10], rho=0.0) == E.EF_EINVAL
    assert _create(10, [0, 10], rho=1.5) == E.EF_EINVAL
    assert _create(10, [0, 10], rho=float("nan")) == E.EF_EINVAL
    assert _create(10, [0, 10], block=0) == E.EF_EINVAL
    h = ctypes.c_void_p()
    assert E.lib().ef_layout_create(10, None, 1, 0.1, 1, ctypes.byref(h)) == E.EF_EINVAL
    assert E.lib().ef_layout_create(10, np.array([0, 10], np.int64).ctypes.data, 0, 0.1, 1,
                                    ctypes.byref(h)) == E.EF_ERANGE


def test_calls_on_unbound_layout_fail_before_any_launch():
    L = E.Layout(1000, None, 0.1)
    lib = E.lib()
    P = ctypes.c_void_p
    fake = P(256 * 1024)  # never dereferenced: validation fails first
    assert lib.ef_accumulate(L.handle, fake, 0, fake, fake, None) == E.EF_EINVAL
    assert lib.compress_topk(L.handle, fake, fake, fake, fake, 1 << 30, None) == E.EF_EINVAL
    assert lib.ef_step_randblock(L.handle, fake, 0, fake, 1, 2, fake, fake, None) == E.EF_EINVAL
    assert lib.decompress_aggregate(L.handle, 0, 4, fake, fake, 1, fake, fake, 1 << 30, None) == E.EF_EINVAL
    assert lib.ef_accumulate(None, fake, 0, fake, fake, None) == E.EF_EINVAL


def test_workspace_sizes():
    L = E.Layout(1 << 20, None, 0.01, 1024)
    assert L.workspace_bytes(E.EF_OP_TOPK) > 0
    assert L.workspace_bytes(E.EF_OP_RANDK) > 0
    assert L.workspace_bytes(E.EF_OP_RANDBLOCK) == 0
    assert L.workspace_bytes(E.EF_OP_AGG_BLOCK, 4) == 0
    assert L.workspace_bytes(E.EF_OP_AGG_SPARSE, 8) >= 8 * (L.d // 8192 + 1) * 4
    assert L.workspace_bytes(E.EF_OP_AGG_SPARSE, 0) == 0
    assert L.workspace_bytes(99) == 0
    # candidate pools sized by k and the rows, not by d: well under 2 bytes per element at 0.1 %
    big = E.Layout(1 << 26, None, 0.001)
    assert 0 < big.workspace_bytes(E.EF_OP_TOPK) < 2 * big.d
    assert 0 < big.workspace_bytes(E.EF_OP_RANDK) < 2 * big.d
    assert E.lib().ef_workspace_diag_offset(L.handle, E.EF_OP_TOPK) == 0
    assert E.lib().ef_workspace_diag_offset(L.handle, E.EF_OP_RANDBLOCK) == ctypes.c_size_t(-1).value


def test_tune_rejects_bad_knobs():
    L = E.Layout(100, None, 0.1)
    assert E.lib().ef_layout_tune(L.handle, 99, 1.0) == E.EF_EINVAL
    assert E.lib().ef_layout_tune(L.handle, 0, float("inf")) == E.EF_EINVAL
    assert E.lib().ef_layout_tune(L.handle, 0, 5.0) == E.EF_OK
    assert E.lib().ef_layout_tune(L.handle, E.EF_TUNE_TOPK_RETRY, 0.0) == E.EF_OK
    assert E.lib().ef_layout_tune(L.handle, E.EF_TUNE_POOL, -1.0) == E.EF_EINVAL


def test_pool_knob_scales_the_workspace():
    """The candidate pool and lists follow the pool knob; 0 leaves the rows' static slots."""
    sizes = []
    for scale in (0.0, 1.0, 2.0):
        L = E.Layout(1 << 24, [0, 1 << 20, 1 << 24], 0.01, tune={E.EF_TUNE_POOL: scale})
        sizes.append((L.workspace_bytes(E.EF_OP_TOPK), L.workspace_bytes(E.EF_OP_RANDK)))
    for op in range(2):
        assert sizes[0][op] < sizes[1][op] < sizes[2][op]
    assert sizes[0][0] < 2 * (1 << 24)  # static slots of 128 entries per 4096-element row, 12 B each


def test_status_strings():
    for c in range(6):
        assert E.lib().ef_status_string(c).decode().startswith("EF_")
    assert "memory" in E.lib().ef_status_string(E.EF_ENOMEM).decode()


def test_binding_refuses_tensors_that_do_not_fit_before_calling_the_library():
    """The binding checks every tensor argument (device, contiguity, dtype, size) before its
    pointer crosses the ABI; host tensors and short or mistyped ones raise EF_EINVAL."""
    import torch
    L = E.Layout(1000, None, 0.1)
    g = torch.zeros(1000)
    idx = torch.zeros(L.K, dtype=torch.int32)
    with pytest.raises(E.EfError) as ex:
        E.ef_step_topk(L, g, g, idx, torch.zeros(L.K), torch.zeros(256, dtype=torch.uint8))
    assert ex.value.code == E.EF_EINVAL and "not on a GPU" in str(ex.value)
    with pytest.raises(E.EfError) as ex:
        E.ef_step_randblock(L, None, g, 1, 0, idx, torch.zeros(L.K))
    assert ex.value.code == E.EF_EINVAL and "g is None" in str(ex.value)


def test_tune_unbinds_and_keeps_the_layout_usable():
    L = E.Layout(100, None, 0.1)
    K = L.K
    assert E.lib().ef_layout_tune(L.handle, E.EF_TUNE_TOPK_SIGMA, 3.0) == E.EF_OK
    assert L.K == K and L.device_bytes() > 0
