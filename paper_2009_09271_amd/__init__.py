"""Python binding of libefsparse (error-feedback gradient sparsification on MI355X).

Argument marshalling only: every step of the hot path runs in the HIP kernels of
``libefsparse.so``; this module passes device pointers (``tensor.data_ptr()``),
sizes and the current HIP stream across the C ABI declared in
``include/efsparse.h``.  Function names match the C entry points.

If the shared library has not been built, importing this package raises
ImportError: there is no fallback implementation.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("EFSPARSE_LIB") or os.path.join(_HERE, "libefsparse.so")

EF_OK, EF_EINVAL, EF_ERANGE, EF_EWORKSPACE, EF_EHIP, EF_ENOMEM = range(6)
EF_F32, EF_BF16 = 0, 1
EF_OP_TOPK, EF_OP_RANDK, EF_OP_RANDBLOCK, EF_OP_AGG_SPARSE, EF_OP_AGG_BLOCK, EF_OP_AGG_SHARED, EF_OP_RANDK_PREP = range(7)
EF_MSG_SPARSE, EF_MSG_BLOCK = 0, 1
EF_TUNE_RANDK_SIGMA, EF_TUNE_RANDK_EXTRA, EF_TUNE_TOPK_SIGMA, EF_TUNE_TOPK_EXTRA, EF_TUNE_TOPK_RETRY, EF_TUNE_POOL = range(6)
EF_PHASE_PREPARE, EF_PHASE_STREAM, EF_PHASE_FINISH, EF_PHASE_ALL = 1, 2, 4, 7
DIAG_SLOW_PATH = 2
DIAG_COUNT_MISMATCH = 4
DIAG_RETRY = 8

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built: run `python paper_2009_09271_amd/build.py` "
                      "(or __graft_entry__.build()) first")

# Load PyTorch first so that the library binds to the same HIP runtime that
# allocates the tensors and owns the streams passed across the ABI.
try:
    import torch as _torch  # noqa: F401
except ImportError:  # host-only use (layout queries) works without it
    _torch = None

_lib = ctypes.CDLL(LIB_PATH)

_c = ctypes
_P = _c.c_void_p
_SIGS = {
    "ef_status_string": (_c.c_char_p, [_c.c_int]),
    "ef_last_hip_error": (_c.c_int, []),
    "ef_last_hip_error_string": (_c.c_char_p, []),
    "ef_layout_create": (_c.c_int, [_c.c_int64, _P, _c.c_int32, _c.c_double, _c.c_int64, _c.POINTER(_P)]),
    "ef_layout_destroy": (_c.c_int, [_P]),
    "ef_layout_total_k": (_c.c_int64, [_P]),
    "ef_layout_num_segments": (_c.c_int32, [_P]),
    "ef_layout_segment_k": (_c.c_int, [_P, _P]),
    "ef_layout_tune": (_c.c_int, [_P, _c.c_int, _c.c_double]),
    "ef_layout_device_bytes": (_c.c_size_t, [_P]),
    "ef_layout_bind": (_c.c_int, [_P, _P, _c.c_size_t, _P]),
    "ef_workspace_bytes": (_c.c_size_t, [_P, _c.c_int, _c.c_int32]),
    "ef_workspace_diag_offset": (_c.c_size_t, [_P, _c.c_int]),
    "ef_accumulate": (_c.c_int, [_P, _P, _c.c_int, _P, _P, _P]),
    "compress_topk": (_c.c_int, [_P, _P, _P, _P, _P, _c.c_size_t, _P]),
    "compress_randk": (_c.c_int, [_P, _P, _c.c_uint64, _c.c_uint32, _P, _P, _P, _c.c_size_t, _P]),
    "compress_randblock": (_c.c_int, [_P, _P, _c.c_uint64, _c.c_uint32, _P, _P, _P]),
    "ef_update": (_c.c_int, [_P, _P, _c.c_int, _P, _P, _P]),
    "decompress_aggregate": (_c.c_int, [_P, _c.c_int, _c.c_int32, _P, _P, _c.c_int, _P, _P, _c.c_size_t, _P]),
    "decompress_aggregate_apply": (_c.c_int, [_P, _c.c_int, _c.c_int32, _P, _P, _c.c_int, _P, _P, _c.c_float,
                                              _c.c_float, _P, _P, _c.c_size_t, _P]),
    "decompress_aggregate_noalloc": (_c.c_int, [_P, _c.c_int, _c.c_int32, _P, _P, _c.c_int, _P, _P]),
    "ef_noalloc_scratch_bytes": (_c.c_size_t, []),
    "decompress_aggregate_shared": (_c.c_int, [_P, _c.c_int, _c.c_int32, _P, _P, _c.c_int, _P, _P, _c.c_size_t,
                                               _P]),
    "ef_dense_average": (_c.c_int, [_P, _c.c_int32, _P, _c.c_int, _P, _P]),
    "ef_step_topk": (_c.c_int, [_P, _P, _c.c_int, _P, _P, _P, _P, _c.c_size_t, _P]),
    "ef_step_randk": (_c.c_int, [_P, _P, _c.c_int, _P, _c.c_uint64, _c.c_uint32, _P, _P, _P, _c.c_size_t, _P]),
    "ef_step_randblock": (_c.c_int, [_P, _P, _c.c_int, _P, _c.c_uint64, _c.c_uint32, _P, _P, _P]),
    "ef_step_topk_batch": (_c.c_int, [_P, _c.c_uint, _c.c_int32, _P, _c.c_int, _P, _P, _P, _P, _c.c_size_t, _P]),
    "ef_step_randk_batch": (_c.c_int, [_P, _c.c_uint, _c.c_int32, _P, _c.c_int, _P, _P, _c.c_uint32, _P, _P, _P,
                                       _c.c_size_t, _P]),
    "ef_randk_prepare": (_c.c_int, [_P, _c.c_uint64, _c.c_uint32, _P, _P, _c.c_size_t, _P]),
    "ef_randk_prepare_batch": (_c.c_int, [_P, _c.c_int32, _P, _c.c_uint32, _P, _P, _c.c_size_t, _P]),
    "ef_step_randk_prepared": (_c.c_int, [_P, _P, _c.c_int, _P, _P, _P, _P, _c.c_size_t, _P]),
    "ef_step_randk_prepared_batch": (_c.c_int, [_P, _c.c_int32, _P, _c.c_int, _P, _P, _P, _P, _c.c_size_t, _P]),
    "ef_step_topk_phases": (_c.c_int, [_P, _c.c_uint, _P, _c.c_int, _P, _P, _P, _P, _c.c_size_t, _P]),
    "ef_step_randk_phases": (_c.c_int, [_P, _c.c_uint, _P, _c.c_int, _P, _c.c_uint64, _c.c_uint32, _P, _P, _P,
                                        _c.c_size_t, _P]),
    "ef_timing_enable": (_c.c_int, [_c.c_int]),
    "ef_timing_collect": (_c.c_int, []),
    "ef_timing_count": (_c.c_int, []),
    "ef_timing_get": (_c.c_int, [_c.c_int, _c.POINTER(_c.c_char_p), _c.POINTER(_c.c_double),
                                 _c.POINTER(_c.c_int64)]),
    "ef_timing_reset": (_c.c_int, []),
}
for _name, (_res, _args) in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.restype, _f.argtypes = _res, _args

EXPORTED = tuple(_SIGS)


class EfError(RuntimeError):
    def __init__(self, code, where, detail=None):
        self.code = code
        msg = f"{where}: {_lib.ef_status_string(code).decode()}"
        if code == EF_EHIP:
            msg += f" ({_lib.ef_last_hip_error()}: {_lib.ef_last_hip_error_string().decode()})"
        if detail:
            msg += f" ({detail})"
        super().__init__(msg)


def _check(code, where):
    if code != EF_OK:
        raise EfError(code, where)


def _stream(t, stream=None):
    """The HIP stream handle to enqueue on: `stream` (a torch.cuda.Stream) when given, else the
    current stream of t's device."""
    if stream is not None:
        return ctypes.c_void_p(stream.cuda_stream)
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _nbytes(t):
    """Byte size of a workspace tensor (0 for None)."""
    return t.numel() * t.element_size() if t is not None else 0


_F32, _IDX, _GRAD, _ANY = "f32", "idx", "grad", "any"


def _need(layout, t, n, kind, name, where, optional=False):
    """Checks a tensor argument before its pointer crosses the ABI: on the layout's device,
    contiguous, of the expected dtype and holding at least n elements, so that no kernel can write
    past its end.  Raises EfError(EF_EINVAL) otherwise."""
    import torch
    if t is None:
        if optional:
            return
        raise EfError(EF_EINVAL, where, f"{name} is None")
    ok = {_F32: (torch.float32,), _GRAD: (torch.float32, torch.bfloat16),
          _IDX: tuple(x for x in (torch.int32, getattr(torch, "uint32", None)) if x is not None)}.get(kind)
    if not isinstance(t, torch.Tensor):
        raise EfError(EF_EINVAL, where, f"{name} is not a tensor")
    if not t.is_cuda:
        raise EfError(EF_EINVAL, where, f"{name} is not on a GPU")
    dev = layout.tables.device if getattr(layout, "tables", None) is not None else None
    if dev is not None and t.device != dev:
        raise EfError(EF_EINVAL, where, f"{name} is on {t.device}, the layout on {dev}")
    if not t.is_contiguous():
        raise EfError(EF_EINVAL, where, f"{name} is not contiguous")
    if ok is not None and t.dtype not in ok:
        raise EfError(EF_EINVAL, where, f"{name} has dtype {t.dtype}")
    if t.numel() < n:
        raise EfError(EF_EINVAL, where, f"{name} holds {t.numel()} elements, {n} needed")


def _gdt(g):
    import torch
    if g.dtype == torch.float32:
        return EF_F32
    if g.dtype == torch.bfloat16:
        return EF_BF16
    raise TypeError(f"gradient dtype {g.dtype} not supported (float32 or bfloat16)")


class Layout:
    """Segment table, density and block size of one gradient layout (host object).

    ``seg_offsets``: [0, o_1, ..., d] (one segment per layer, or [0, d] for global scope).
    ``bind(device)`` uploads its tables to device memory; compute calls need a bound layout.
    """

    def __init__(self, d, seg_offsets=None, density=0.01, block=1, tune=None):
        offs = np.asarray([0, d] if seg_offsets is None else seg_offsets, dtype=np.int64)
        self._offs = np.ascontiguousarray(offs)
        h = ctypes.c_void_p()
        _check(_lib.ef_layout_create(int(d), self._offs.ctypes.data, len(offs) - 1, float(density),
                                     int(block), ctypes.byref(h)), "ef_layout_create")
        self._h = h
        self.d = int(d)
        self.density = float(density)
        self.block = int(block)
        self.tables = None
        for knob, value in (tune or {}).items():
            _check(_lib.ef_layout_tune(self._h, int(knob), float(value)), "ef_layout_tune")

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value and _lib is not None:
            _lib.ef_layout_destroy(h)
            self._h = None

    @property
    def handle(self):
        return self._h

    @property
    def K(self) -> int:
        return int(_lib.ef_layout_total_k(self._h))

    @property
    def n_seg(self) -> int:
        return int(_lib.ef_layout_num_segments(self._h))

    @property
    def seg_offsets(self):
        return self._offs.copy()

    def segment_k(self):
        out = np.zeros(self.n_seg, dtype=np.int64)
        _check(_lib.ef_layout_segment_k(self._h, out.ctypes.data), "ef_layout_segment_k")
        return out

    def device_bytes(self) -> int:
        return int(_lib.ef_layout_device_bytes(self._h))

    def workspace_bytes(self, op, W=1) -> int:
        return int(_lib.ef_workspace_bytes(self._h, int(op), int(W)))

    def bind(self, device="cuda"):
        import torch
        n = max(self.device_bytes(), 256)
        self.tables = torch.empty(n, dtype=torch.uint8, device=device)
        _check(_lib.ef_layout_bind(self._h, _ptr(self.tables), n, _stream(self.tables)), "ef_layout_bind")
        return self

    def workspace(self, op, W=1, device="cuda"):
        """A zero-filled workspace (zeroed so that the diagnostics word starts clear)."""
        import torch
        n = max(self.workspace_bytes(op, W), 256)
        return torch.zeros(n, dtype=torch.uint8, device=device)

    def diag(self, ws, op) -> int:
        """Diagnostics word of a top-k / random-k workspace (synchronises)."""
        off = int(_lib.ef_workspace_diag_offset(self._h, int(op)))
        return int(ws[off:off + 4].cpu().numpy().view(np.uint32)[0])


def _msg_len(layout, msg_kind):
    """Entries of one message's index (sparse) or start (block) array."""
    return layout.n_seg if msg_kind == EF_MSG_BLOCK else layout.K


def ef_accumulate(layout, g, e, acc):
    w, d = "ef_accumulate", layout.d
    _need(layout, g, d, _GRAD, "g", w)
    _need(layout, e, d, _F32, "e", w)
    _need(layout, acc, d, _F32, "acc", w)
    _check(_lib.ef_accumulate(layout.handle, _ptr(g), _gdt(g), _ptr(e), _ptr(acc), _stream(e)), w)


def compress_topk(layout, acc, idx, val, ws):
    w = "compress_topk"
    _need(layout, acc, layout.d, _F32, "acc", w)
    _need(layout, idx, layout.K, _IDX, "idx", w)
    _need(layout, val, layout.K, _F32, "val", w)
    _need(layout, ws, 0, _ANY, "ws", w)
    _check(_lib.compress_topk(layout.handle, _ptr(acc), _ptr(idx), _ptr(val), _ptr(ws), _nbytes(ws), _stream(acc)),
           w)


def compress_randk(layout, acc, seed, step, idx, val, ws):
    w = "compress_randk"
    _need(layout, acc, layout.d, _F32, "acc", w)
    _need(layout, idx, layout.K, _IDX, "idx", w)
    _need(layout, val, layout.K, _F32, "val", w)
    _need(layout, ws, 0, _ANY, "ws", w)
    _check(_lib.compress_randk(layout.handle, _ptr(acc), int(seed), int(step), _ptr(idx), _ptr(val), _ptr(ws),
                               _nbytes(ws), _stream(acc)), w)


def compress_randblock(layout, acc, seed, step, start, val):
    w = "compress_randblock"
    _need(layout, acc, layout.d, _F32, "acc", w)
    _need(layout, start, layout.n_seg, _IDX, "start", w)
    _need(layout, val, layout.K, _F32, "val", w)
    _check(_lib.compress_randblock(layout.handle, _ptr(acc), int(seed), int(step), _ptr(start), _ptr(val),
                                   _stream(acc)), w)


def ef_update(layout, acc, msg_kind, idx_or_start, e):
    w = "ef_update"
    _need(layout, acc, layout.d, _F32, "acc", w)
    _need(layout, e, layout.d, _F32, "e", w)
    _need(layout, idx_or_start, _msg_len(layout, msg_kind), _IDX, "idx_or_start", w)
    _check(_lib.ef_update(layout.handle, _ptr(acc), int(msg_kind), _ptr(idx_or_start), _ptr(e), _stream(e)), w)


def _agg_args(layout, msg_kind, W, idx_or_start, val, w):
    _need(layout, idx_or_start, int(W) * _msg_len(layout, msg_kind), _IDX, "idx_or_start", w)
    _need(layout, val, int(W) * layout.K, _F32, "val", w)


def decompress_aggregate(layout, msg_kind, W, idx_or_start, val, out, ws=None, average=True, stream=None):
    w = "decompress_aggregate"
    _agg_args(layout, msg_kind, W, idx_or_start, val, w)
    _need(layout, out, layout.d, _F32, "out", w)
    _need(layout, ws, 0, _ANY, "ws", w, optional=True)
    _check(_lib.decompress_aggregate(layout.handle, int(msg_kind), int(W), _ptr(idx_or_start), _ptr(val),
                                     1 if average else 0, _ptr(out), _ptr(ws), _nbytes(ws), _stream(out, stream)), w)


def decompress_aggregate_noalloc(layout, msg_kind, W, idx_or_start, val, out, average=True, stream=None):
    """decompress_aggregate with its scratch in the library's static device array (no workspace)."""
    w = "decompress_aggregate_noalloc"
    _agg_args(layout, msg_kind, W, idx_or_start, val, w)
    _need(layout, out, layout.d, _F32, "out", w)
    _check(_lib.decompress_aggregate_noalloc(layout.handle, int(msg_kind), int(W), _ptr(idx_or_start), _ptr(val),
                                             1 if average else 0, _ptr(out), _stream(out, stream)), w)


def decompress_aggregate_apply(layout, msg_kind, W, idx_or_start, val, x, mom=None, beta=0.0, wd=0.0, out=None,
                               ws=None, average=True, stream=None):
    w = "decompress_aggregate_apply"
    _agg_args(layout, msg_kind, W, idx_or_start, val, w)
    _need(layout, x, layout.d, _F32, "x", w)
    _need(layout, mom, layout.d, _F32, "mom", w, optional=True)
    _need(layout, out, layout.d, _F32, "out", w, optional=True)
    _need(layout, ws, 0, _ANY, "ws", w, optional=True)
    _check(_lib.decompress_aggregate_apply(layout.handle, int(msg_kind), int(W), _ptr(idx_or_start), _ptr(val),
                                           1 if average else 0, _ptr(x), _ptr(mom), float(beta), float(wd),
                                           _ptr(out), _ptr(ws), _nbytes(ws), _stream(x, stream)), w)


def decompress_aggregate_shared(layout, msg_kind, W, idx_or_start, val, out, ws, average=True, stream=None):
    w = "decompress_aggregate_shared"
    _need(layout, idx_or_start, _msg_len(layout, msg_kind), _IDX, "idx_or_start", w)
    _need(layout, val, int(W) * layout.K, _F32, "val", w)
    _need(layout, out, layout.d, _F32, "out", w)
    _need(layout, ws, 0, _ANY, "ws", w)
    _check(_lib.decompress_aggregate_shared(layout.handle, int(msg_kind), int(W), _ptr(idx_or_start), _ptr(val),
                                            1 if average else 0, _ptr(out), _ptr(ws), _nbytes(ws),
                                            _stream(out, stream)), w)


def ef_dense_average(layout, W, g, out, average=True, stream=None):
    w = "ef_dense_average"
    _need(layout, g, int(W) * layout.d, _F32, "g", w)
    _need(layout, out, layout.d, _F32, "out", w)
    _check(_lib.ef_dense_average(layout.handle, int(W), _ptr(g), 1 if average else 0, _ptr(out),
                                 _stream(out, stream)), w)


def _step_args(layout, g, e, idx, val, ws, w, idx_len=None):
    _need(layout, g, layout.d, _GRAD, "g", w)
    _need(layout, e, layout.d, _F32, "e", w)
    _need(layout, idx, layout.K if idx_len is None else idx_len, _IDX, "idx", w)
    _need(layout, val, layout.K, _F32, "val", w)
    if ws is not False:
        _need(layout, ws, 0, _ANY, "ws", w)


def ef_step_topk(layout, g, e, idx, val, ws):
    w = "ef_step_topk"
    _step_args(layout, g, e, idx, val, ws, w)
    _check(_lib.ef_step_topk(layout.handle, _ptr(g), _gdt(g), _ptr(e), _ptr(idx), _ptr(val), _ptr(ws), _nbytes(ws),
                             _stream(e)), w)


def ef_step_randk(layout, g, e, seed, step, idx, val, ws):
    w = "ef_step_randk"
    _step_args(layout, g, e, idx, val, ws, w)
    _check(_lib.ef_step_randk(layout.handle, _ptr(g), _gdt(g), _ptr(e), int(seed), int(step), _ptr(idx), _ptr(val),
                              _ptr(ws), _nbytes(ws), _stream(e)), w)


def ef_step_topk_phases(layout, phases, g, e, idx, val, ws, stream=None):
    w = "ef_step_topk_phases"
    _step_args(layout, g, e, idx, val, ws, w)
    _check(_lib.ef_step_topk_phases(layout.handle, int(phases), _ptr(g), _gdt(g), _ptr(e), _ptr(idx), _ptr(val),
                                    _ptr(ws), _nbytes(ws), _stream(e, stream)), w)


def ef_step_randk_phases(layout, phases, g, e, seed, step, idx, val, ws, stream=None):
    w = "ef_step_randk_phases"
    _step_args(layout, g, e, idx, val, ws, w)
    _check(_lib.ef_step_randk_phases(layout.handle, int(phases), _ptr(g), _gdt(g), _ptr(e), int(seed), int(step),
                                     _ptr(idx), _ptr(val), _ptr(ws), _nbytes(ws), _stream(e, stream)), w)


def batch_workspace(layout, op, W, device="cuda"):
    """W zero-filled workspaces for ef_step_*_batch, one row of `stride` bytes each: (tensor, stride)."""
    import torch
    stride = (max(layout.workspace_bytes(op, 1), 256) + 255) // 256 * 256
    return torch.zeros((W, stride), dtype=torch.uint8, device=device), stride


def _ptr_table(tensors):
    return (ctypes.c_void_p * len(tensors))(*[t.data_ptr() for t in tensors])


def _batch_args(layout, g, e, idx, val, ws, ws_stride, w):
    """Per-worker gradients and residuals, [W][K] messages and W workspace rows of ws_stride bytes."""
    if g is not None and len(g) != len(e):
        raise ValueError("one gradient and one residual per worker")
    W = len(e)
    if W == 0:
        raise EfError(EF_ERANGE, w, "no workers")
    for i in range(W):
        if g is not None:
            _need(layout, g[i], layout.d, _GRAD, f"g[{i}]", w)
        _need(layout, e[i], layout.d, _F32, f"e[{i}]", w)
    if g is not None and any(x.dtype != g[0].dtype for x in g):
        raise EfError(EF_EINVAL, w, "the gradients differ in dtype")
    _need(layout, idx, W * layout.K, _IDX, "idx", w)
    if val is not None:
        _need(layout, val, W * layout.K, _F32, "val", w)
    _need(layout, ws, 0, _ANY, "ws", w)
    if _nbytes(ws) < W * int(ws_stride):
        raise EfError(EF_EWORKSPACE, w, f"ws holds {_nbytes(ws)} bytes, {W} rows of {int(ws_stride)} needed")


def ef_step_topk_batch(layout, g, e, idx, val, ws, ws_stride, phases=EF_PHASE_ALL, stream=None):
    """W workers' fused top-k steps: g, e lists of W tensors; idx, val [W][K] (rows of the batch); ws rows
    from batch_workspace."""
    w = "ef_step_topk_batch"
    _batch_args(layout, g, e, idx, val, ws, ws_stride, w)
    _check(_lib.ef_step_topk_batch(layout.handle, int(phases), len(e), _ptr_table(g), _gdt(g[0]), _ptr_table(e),
                                   _ptr(idx), _ptr(val), _ptr(ws), int(ws_stride), _stream(e[0], stream)), w)


def ef_step_randk_batch(layout, g, e, seeds, step, idx, val, ws, ws_stride, phases=EF_PHASE_ALL, stream=None):
    """W workers' fused random-k steps; seeds: W integers (host)."""
    w = "ef_step_randk_batch"
    sd = np.ascontiguousarray(np.asarray(seeds, dtype=np.uint64))
    if len(g) != len(e) or sd.shape != (len(e),):
        raise ValueError("one gradient, one residual and one seed per worker")
    _batch_args(layout, g, e, idx, val, ws, ws_stride, w)
    _check(_lib.ef_step_randk_batch(layout.handle, int(phases), len(e), _ptr_table(g), _gdt(g[0]), _ptr_table(e),
                                    sd.ctypes.data, int(step), _ptr(idx), _ptr(val), _ptr(ws), int(ws_stride),
                                    _stream(e[0], stream)), w)


def ef_randk_prepare(layout, seed, step, idx, ws, stream=None):
    """The random-k message indices of (seed, step) and their tile table in ws (EF_OP_RANDK_PREP)."""
    w = "ef_randk_prepare"
    _need(layout, idx, layout.K, _IDX, "idx", w)
    _need(layout, ws, 0, _ANY, "ws", w)
    _check(_lib.ef_randk_prepare(layout.handle, int(seed), int(step), _ptr(idx), _ptr(ws), _nbytes(ws),
                                 _stream(idx, stream)), w)


def ef_randk_prepare_batch(layout, seeds, step, idx, ws, ws_stride, stream=None):
    """W workers' prepared selections: seeds W integers (host); idx [W][K]; ws rows from batch_workspace
    (EF_OP_RANDK_PREP)."""
    w = "ef_randk_prepare_batch"
    sd = np.ascontiguousarray(np.asarray(seeds, dtype=np.uint64))
    W = sd.shape[0]
    _need(layout, idx, W * layout.K, _IDX, "idx", w)
    _need(layout, ws, 0, _ANY, "ws", w)
    if W and _nbytes(ws) < W * int(ws_stride):
        raise EfError(EF_EWORKSPACE, w, f"ws holds {_nbytes(ws)} bytes, {W} rows of {int(ws_stride)} needed")
    _check(_lib.ef_randk_prepare_batch(layout.handle, W, sd.ctypes.data, int(step), _ptr(idx), _ptr(ws),
                                       int(ws_stride), _stream(idx, stream)), w)


def ef_step_randk_prepared(layout, g, e, idx, val, ws, stream=None):
    """The random-k step given prepared indices and workspace."""
    w = "ef_step_randk_prepared"
    _step_args(layout, g, e, idx, val, ws, w)
    _check(_lib.ef_step_randk_prepared(layout.handle, _ptr(g), _gdt(g), _ptr(e), _ptr(idx), _ptr(val), _ptr(ws),
                                       _nbytes(ws), _stream(e, stream)), w)


def ef_step_randk_prepared_batch(layout, g, e, idx, val, ws, ws_stride, stream=None):
    """W workers' random-k steps given their prepared indices (rows of idx) and workspaces (rows of ws)."""
    w = "ef_step_randk_prepared_batch"
    _batch_args(layout, g, e, idx, val, ws, ws_stride, w)
    _check(_lib.ef_step_randk_prepared_batch(layout.handle, len(e), _ptr_table(g), _gdt(g[0]), _ptr_table(e),
                                             _ptr(idx), _ptr(val), _ptr(ws), int(ws_stride), _stream(e[0], stream)),
           w)


def ef_step_randblock(layout, g, e, seed, step, start, val, stream=None):
    w = "ef_step_randblock"
    _step_args(layout, g, e, start, val, False, w, idx_len=layout.n_seg)
    _check(_lib.ef_step_randblock(layout.handle, _ptr(g), _gdt(g), _ptr(e), int(seed), int(step), _ptr(start),
                                  _ptr(val), _stream(e, stream)), w)


def lib():
    """The loaded ctypes library (for contract tests)."""
    return _lib


def timing_enable(on=True):
    """Time every library kernel launch with dispatch-bound HIP events (see ef_timing_enable)."""
    _check(_lib.ef_timing_enable(1 if on else 0), "ef_timing_enable")


def timing_collect(reset=True):
    """Wait for recorded launches; return {kernel: (total_ms, launches)} and optionally reset."""
    _check(_lib.ef_timing_collect(), "ef_timing_collect")
    out = {}
    for i in range(_lib.ef_timing_count()):
        name, ms, n = ctypes.c_char_p(), ctypes.c_double(), ctypes.c_int64()
        _check(_lib.ef_timing_get(i, ctypes.byref(name), ctypes.byref(ms), ctypes.byref(n)), "ef_timing_get")
        out[name.value.decode()] = (ms.value, n.value)
    if reset:
        _lib.ef_timing_reset()
    return out
