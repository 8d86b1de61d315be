"""CPU oracle for the error-feedback sparsified-gradient hot path.

TEST INFRASTRUCTURE.  This is the plain, slow, obviously-correct reference that
the GPU library is checked against.  Only ``tests/``, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py`` may import it; the product path never
does, and it shares no code with the HIP library.

What the paper fixes (Algorithm 1 and Section 3):

* each worker adds its carried residual to its new gradient (p = g + e,
  Algorithm 1, the accumulate step; the learning rate is folded into g by the
  caller, so no gamma appears here);
* compresses p with a compressor C (Section 3: top-k, random-k or
  block-random-k), optionally per layer (Section 3, sparsification scope);
* the workers' messages are summed (Algorithm 1, the aggregate step);
* the worker keeps what it did not send as its new residual (Section 3, the
  worker steps; Algorithm 1's residual update).

Readings where the paper is silent or leaves a choice open:

* k per segment: k = clamp(floor(rho * d_l + 0.5), 1, d_l) in IEEE double.
* top-k orders by magnitude; ties go to the lower index.  The magnitude key is
  the float's bit pattern with the sign bit cleared (uint32), which orders
  |x| for every non-NaN x and makes -0 and +0 equal.
* random-k: key u_j of local position j is word (j mod 4) of Philox4x32-10
  with counter (j div 4, 0, step, 0x01000000 | l) and key (seed lo, seed hi);
  the k positions with the smallest (u_j, j) are sent.
* random-block: b_l = b if d_l > b else 1, n_l = ceil(d_l / b_l); with
  (x0, x1, ...) = Philox(counter (0, 0, step, 0x02000000 | l), same key) and
  r = x0 + 2**32 x1, the start is s_l = b_l * floor(r * n_l / 2**64); the
  support is positions (s_l + t) mod d_l for t = 0..k_l-1 (wrapping).
* residual: e' = +0.0 on the support and acc elsewhere (bits unchanged), so
  acc == sent + e' as values.
* aggregate: out_i = (sum over workers w = 0..W-1, in that order, of the
  entries present at i, starting from +0.0, in float32) / W, with IEEE
  float32 division; ``average=False`` gives the plain sum of Algorithm 1.
  With shared coordinates (equal seeds) it is the same sum.
* parameter update: x' = x - d with d = q (+ wd x) and, with momentum,
  m' = beta m + d, d = m' (the order of a plain SGD step; the learning rate is
  inside q), each float32 operation rounded on its own.
* dense average (the uncompressed baseline): the same ordered sum over dense
  gradients.

Message formats: sparse messages are (idx uint32[K], val float32[K]) with
segment l's entries at positions [P_l, P_l + k_l), P_l = sum of earlier k,
indices global and ascending.  Block messages are (start uint32[L] segment-local,
val float32[K]) with values in run order t = 0..k_l-1.

Parity status: every function here is pinned by ``tests/test_oracle_pins.py``
(brute force, special cases, invariants, hand-worked vectors under
``tests/golden/`` and an independent Philox implementation).
"""

from __future__ import annotations

import math

import numpy as np

from .philox import philox4x32_10

RANDK_TAG = 0x01000000
RANDBLOCK_TAG = 0x02000000


# ----------------------------------------------------------------------------
# k per segment (Section 4.1 sets k to a fraction of the vector size; the
# rounding is a reading).
# ----------------------------------------------------------------------------
def k_rule(d_l: int, density: float) -> int:
    k = math.floor(float(density) * float(d_l) + 0.5)
    return int(min(max(k, 1), d_l))


def segment_ks(seg_offsets, density: float):
    return [k_rule(seg_offsets[i + 1] - seg_offsets[i], density) for i in range(len(seg_offsets) - 1)]


def message_offsets(ks):
    """P_l: where segment l's entries start in a message."""
    return np.concatenate([[0], np.cumsum(np.asarray(ks, dtype=np.int64))]).astype(np.int64)


# ----------------------------------------------------------------------------
# Algorithm 1, the accumulate step: p = g + e (one float32 add per element).
# ----------------------------------------------------------------------------
def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) widened exactly to float32."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def ef_accumulate(g: np.ndarray, e: np.ndarray) -> np.ndarray:
    if g.dtype == np.uint16:
        g = bf16_to_f32(g)
    assert g.dtype == np.float32 and e.dtype == np.float32
    return np.add(g, e, dtype=np.float32)


def magnitude_key(x: np.ndarray) -> np.ndarray:
    return x.astype(np.float32).view(np.uint32) & np.uint32(0x7FFFFFFF)


# ----------------------------------------------------------------------------
# Section 3, top-k sparsification: keep the k entries of largest magnitude.
# ----------------------------------------------------------------------------
def topk_support(acc: np.ndarray, seg_offsets, ks):
    """Global indices chosen by top-k, ascending, segment by segment."""
    out = []
    for l, k in enumerate(ks):
        o, n = seg_offsets[l], seg_offsets[l + 1] - seg_offsets[l]
        key = magnitude_key(acc[o:o + n]).astype(np.int64)
        pos = np.arange(n, dtype=np.int64)
        order = np.lexsort((pos, -key))  # key descending, then index ascending
        out.append(np.sort(order[:k]) + o)
    return np.concatenate(out).astype(np.uint32)


def compress_topk(acc, seg_offsets, ks):
    idx = topk_support(acc, seg_offsets, ks)
    return idx, acc[idx.astype(np.int64)].copy()


# ----------------------------------------------------------------------------
# Section 3, random-k sparsification: keep k entries chosen at random.
# ----------------------------------------------------------------------------
def randk_keys(n: int, l: int, seed: int, step: int, j0: int = 0, j1=None) -> np.ndarray:
    """Random keys u_j of segment l (n elements) for the local positions j = j0..j1-1 (default: the
    whole segment).  A range evaluates the same definition on part of the segment, so that a very
    large segment can be checked piece by piece."""
    j1 = n if j1 is None else int(j1)
    assert 0 <= j0 <= j1 <= n
    b0 = j0 // 4
    c = np.arange(b0, (j1 + 3) // 4, dtype=np.uint64)
    x = philox4x32_10(c & np.uint64(0xFFFFFFFF), c >> np.uint64(32), np.uint64(step & 0xFFFFFFFF),
                      np.uint64(RANDK_TAG | l), seed & 0xFFFFFFFF, seed >> 32)
    return np.stack(x, axis=1).reshape(-1)[j0 - 4 * b0:j1 - 4 * b0]


def randk_support(seg_offsets, ks, seed: int, step: int):
    out = []
    for l, k in enumerate(ks):
        o, n = seg_offsets[l], seg_offsets[l + 1] - seg_offsets[l]
        u = randk_keys(n, l, seed, step).astype(np.int64)
        pos = np.arange(n, dtype=np.int64)
        order = np.lexsort((pos, u))  # key ascending, then index ascending
        out.append(np.sort(order[:k]) + o)
    return np.concatenate(out).astype(np.uint32)


def compress_randk(acc, seg_offsets, ks, seed: int, step: int):
    idx = randk_support(seg_offsets, ks, seed, step)
    return idx, acc[idx.astype(np.int64)].copy()


# ----------------------------------------------------------------------------
# Section 3, block-random-k: one random start, then the following k-1 values.
# ----------------------------------------------------------------------------
def block_params(n: int, block: int):
    b = block if n > block else 1
    return b, -(-n // b)


def randblock_start(n: int, l: int, block: int, seed: int, step: int) -> int:
    b, nb = block_params(n, block)
    x0, x1, _, _ = philox4x32_10(0, 0, step & 0xFFFFFFFF, RANDBLOCK_TAG | l, seed & 0xFFFFFFFF, seed >> 32)
    r = int(x0) | (int(x1) << 32)
    return b * ((r * nb) >> 64)


def randblock_positions(n: int, k: int, s: int) -> np.ndarray:
    """Segment-local positions of a run of k values starting at s, wrapping."""
    return (s + np.arange(k, dtype=np.int64)) % n


def compress_randblock(acc, seg_offsets, ks, block: int, seed: int, step: int):
    starts, vals = [], []
    for l, k in enumerate(ks):
        o, n = seg_offsets[l], seg_offsets[l + 1] - seg_offsets[l]
        s = randblock_start(n, l, block, seed, step)
        starts.append(s)
        vals.append(acc[o + randblock_positions(n, k, s)])
    return np.asarray(starts, dtype=np.uint32), np.concatenate(vals).astype(np.float32)


def block_support(seg_offsets, ks, starts):
    out = []
    for l, k in enumerate(ks):
        o, n = seg_offsets[l], seg_offsets[l + 1] - seg_offsets[l]
        out.append(o + randblock_positions(n, k, int(starts[l])))
    return np.concatenate(out)


# ----------------------------------------------------------------------------
# Residual update (Section 3 worker steps / Algorithm 1): keep what was not sent.
# ----------------------------------------------------------------------------
def ef_update(acc: np.ndarray, support: np.ndarray) -> np.ndarray:
    e = acc.copy()
    e[np.asarray(support, dtype=np.int64)] = np.float32(0.0)
    return e


# ----------------------------------------------------------------------------
# Algorithm 1, the aggregate step: sum the workers' messages (then average).
# ----------------------------------------------------------------------------
def decompress_aggregate(d: int, supports, values, average: bool = True) -> np.ndarray:
    """``supports[w]`` / ``values[w]``: global positions and values of worker
    w's message (positions distinct within a worker).  Dense float32 sum in
    worker order from +0.0, then division by W."""
    out = np.zeros(d, dtype=np.float32)
    for pos, val in zip(supports, values):
        out[np.asarray(pos, dtype=np.int64)] += np.asarray(val, dtype=np.float32)
    if average:
        out = out / np.float32(len(supports))
    return out


def decompress_aggregate_sparse(d, idx_stack, val_stack, average=True):
    return decompress_aggregate(d, list(idx_stack), list(val_stack), average)


def decompress_aggregate_block(d, seg_offsets, ks, start_stack, val_stack, average=True):
    sup = [block_support(seg_offsets, ks, st) for st in start_stack]
    return decompress_aggregate(d, sup, list(val_stack), average)


def decompress_aggregate_shared_sparse(d, idx, val_stack, average=True):
    """Shared coordinates (Section 3, the allReduce mode: every worker uses the
    same seed, so every message has the same indices ``idx``): the aggregate is
    the general one with that index list repeated for each worker."""
    return decompress_aggregate(d, [idx] * len(val_stack), list(val_stack), average)


def decompress_aggregate_shared_block(d, seg_offsets, ks, start, val_stack, average=True):
    """Shared block starts (the allReduce mode of block-random-k)."""
    sup = block_support(seg_offsets, ks, start)
    return decompress_aggregate(d, [sup] * len(val_stack), list(val_stack), average)


# ----------------------------------------------------------------------------
# Algorithm 1, the parameter update x_{t+1} = x_t - q_t, with the momentum and
# weight decay of the paper's training setup (Section 4, experimental setup) as
# options.
# ----------------------------------------------------------------------------
def apply_update(x, q, m=None, beta=0.0, wd=0.0):
    """One update of the parameters x by the aggregated step q, in float32 with
    every operation rounded on its own (no fused multiply-add):

        d = q + (wd * x)              when wd != 0
        m' = (beta * m) + d, d = m'   when a momentum buffer m is given
        x' = x - d

    The learning rate is already inside q (the accumulate step scales g), so wd
    is the learning rate times the weight-decay factor.  Returns (x', m')."""
    f = np.float32
    x = np.asarray(x, dtype=f)
    d = np.asarray(q, dtype=f).copy()
    if wd != 0.0:
        d = d + (f(wd) * x).astype(f)
    m_new = None
    if m is not None:
        m_new = (f(beta) * np.asarray(m, dtype=f)).astype(f) + d
        d = m_new
    return (x - d).astype(f), m_new


# ----------------------------------------------------------------------------
# Standard SGD's exchange (no compression), the paper's baseline (Section 4,
# results): the dense average of the W workers' gradients.
# ----------------------------------------------------------------------------
def dense_average(G, average=True):
    """out = (sum over workers w = 0..W-1, in that order, of the dense
    gradients, from +0.0, in float32) / W."""
    G = np.asarray(G, dtype=np.float32)
    out = np.zeros(G.shape[1], dtype=np.float32)
    for g in G:
        out = out + g
    if average:
        out = out / np.float32(G.shape[0])
    return out


# ----------------------------------------------------------------------------
# One worker step: accumulate, compress, residual update.
# ----------------------------------------------------------------------------
def ef_step(kind: str, g, e, seg_offsets, ks, seed=0, step=0, block=1):
    acc = ef_accumulate(g, e)
    if kind == "topk":
        idx, val = compress_topk(acc, seg_offsets, ks)
        return (idx, val), ef_update(acc, idx)
    if kind == "randk":
        idx, val = compress_randk(acc, seg_offsets, ks, seed, step)
        return (idx, val), ef_update(acc, idx)
    if kind == "randblock":
        start, val = compress_randblock(acc, seg_offsets, ks, block, seed, step)
        return (start, val), ef_update(acc, block_support(seg_offsets, ks, start))
    raise ValueError(kind)
