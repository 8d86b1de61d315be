"""Seeded synthetic gradients shaped like the paper's workloads.

The paper measures on ResNet-18 / CIFAR-10 gradients (Section 4.1).  Neither
the dataset nor trained models are used here: every input is drawn from a
seeded NumPy generator with the layer structure and value distribution listed
per workload below.  The same arrays feed the GPU path and the CPU oracle.

This module generates inputs only; it contains none of the compressor or
aggregation arithmetic.

Recipe (each draw in float64, rounded to float32 by NumPy's round-to-nearest):

* ``flat1m``   d = 2**20, N(0, 0.01**2); worker w, step t uses
  ``default_rng([0, w, t])`` (worker 0 / step 0 is seed vector [0, 0, 0]).
* ``resnet18`` 62 tensors, Student-t(nu=3) / sqrt(fan_in) per tensor.
  fan_in = prod(shape[1:]) for a tensor of rank >= 2; a 1-D tensor takes the
  fan_in of the nearest preceding tensor of rank >= 2.
* ``resnet50`` 161 tensors, Laplace(0, b_l) with b_l = 10**U(-5, -2) drawn
  once per tensor from ``default_rng([2, 999])``.
* ``bert``     199 tensors, every entry N(0, 1e-3) (1e-3 read as the
  variance), except that 90 % of the word-embedding rows (chosen once, without
  replacement, from ``default_rng([3, 999])``) are exactly zero.
* ``flat1g``   d = 1e9, per element N(0, 1e-4) with probability 0.99 else
  N(0, 1e-1) (variances).  Too large for host generation in tests; drawn in
  blocks.

Worker w at step t of workload c always draws from ``default_rng([c, w, t])``.
The compressor seed for worker w is ``(c << 32) | w`` (distinct coordinates);
``shared_seed(c)`` gives every worker the same seed (shared coordinates).
"""

from __future__ import annotations

from dataclasses import dataclass, field
from math import prod, sqrt

import numpy as np

from . import shapes as S


@dataclass(frozen=True)
class Workload:
    name: str
    cfg_id: int
    kind: str                     # value distribution family
    tensor_shapes: tuple = ()     # ((name, shape), ...); empty for flat workloads
    flat_d: int = 0
    densities: tuple = (0.01,)
    blocks: tuple = (1024,)
    W: int = 4
    steps: int = 3
    scopes: tuple = ("flat",)
    dtypes: tuple = ("f32",)

    @property
    def d(self) -> int:
        return self.flat_d if not self.tensor_shapes else S.numel(self.tensor_shapes)

    def seg_offsets(self, scope: str):
        """Segment boundaries for a scope: one segment per tensor (layer-wise)
        or a single segment covering everything (global/flat)."""
        if scope == "flat" or not self.tensor_shapes:
            return [0, self.d]
        return S.segment_offsets(self.tensor_shapes)

    def scaled(self, div: int) -> "Workload":
        """A smaller copy with the same structure (tensor count and order)."""
        if self.tensor_shapes:
            return Workload(self.name + f"/{div}", self.cfg_id, self.kind,
                            tuple(S.scaled(self.tensor_shapes, div)), 0, self.densities,
                            self.blocks, self.W, self.steps, self.scopes, self.dtypes)
        return Workload(self.name + f"/{div}", self.cfg_id, self.kind, (), max(1, self.flat_d // div),
                        self.densities, self.blocks, self.W, self.steps, self.scopes, self.dtypes)


FLAT1M = Workload("flat1m", 0, "normal", flat_d=1 << 20, densities=(0.01,), blocks=(1024,),
                  W=4, steps=3, scopes=("flat",))
RESNET18 = Workload("resnet18", 1, "student_t", tuple(S.resnet18_shapes()), densities=(0.01,),
                    blocks=(1, 1024), W=8, steps=10, scopes=("layer", "flat"))
RESNET50 = Workload("resnet50", 2, "laplace", tuple(S.resnet50_shapes()), densities=(0.001,),
                    blocks=(256, 4096, 65536), W=16, steps=10, scopes=("flat", "layer"))
BERT = Workload("bert", 3, "bert", tuple(S.bert_base_shapes()), densities=(0.001, 0.01, 0.1),
                blocks=(4096,), W=16, steps=3, scopes=("layer", "flat"))
FLAT1G = Workload("flat1g", 4, "mixture", flat_d=1_000_000_000,
                  densities=(0.0001, 0.001, 0.01, 0.1), blocks=tuple(1 << s for s in range(8, 21)),
                  W=32, steps=2, scopes=("flat",), dtypes=("f32", "bf16"))

WORKLOADS = {w.name: w for w in (FLAT1M, RESNET18, RESNET50, BERT, FLAT1G)}


def worker_seed(wl: Workload, w: int) -> int:
    return (wl.cfg_id << 32) | w


def shared_seed(wl: Workload) -> int:
    return wl.cfg_id << 32


def _fan_ins(tensor_shapes):
    fans, last = [], 1
    for _, s in tensor_shapes:
        if len(s) >= 2:
            last = prod(s[1:])
        fans.append(last)
    return fans


def _structure(wl: Workload):
    """Per-tensor parameters drawn once per workload (not per worker/step)."""
    rng = np.random.default_rng([wl.cfg_id, 999])
    if wl.kind == "laplace":
        return {"b": 10.0 ** rng.uniform(-5.0, -2.0, size=len(wl.tensor_shapes))}
    if wl.kind == "bert":
        vocab = wl.tensor_shapes[0][1][0]
        nzero = int(round(0.9 * vocab))
        return {"zero_rows": np.sort(rng.choice(vocab, size=nzero, replace=False))}
    return {}


def gradient(wl: Workload, w: int, t: int) -> np.ndarray:
    """Float32 gradient of worker ``w`` at step ``t`` (flattened, length wl.d)."""
    rng = np.random.default_rng([wl.cfg_id, w, t])
    d = wl.d
    if wl.kind == "normal":
        return (rng.standard_normal(d) * 0.01).astype(np.float32)
    if wl.kind == "mixture":
        out = np.empty(d, dtype=np.float32)
        step = 1 << 24
        for a in range(0, d, step):
            n = min(step, d - a)
            wide = rng.random(n) < 0.01
            z = rng.standard_normal(n)
            out[a:a + n] = (z * np.where(wide, sqrt(1e-1), sqrt(1e-4))).astype(np.float32)
        return out
    st = _structure(wl)
    parts = []
    for i, ((_, shp), fan) in enumerate(zip(wl.tensor_shapes, _fan_ins(wl.tensor_shapes))):
        n = prod(shp)
        if wl.kind == "student_t":
            parts.append(rng.standard_t(3.0, size=n) / sqrt(fan))
        elif wl.kind == "laplace":
            parts.append(rng.laplace(0.0, st["b"][i], size=n))
        elif wl.kind == "bert":
            v = rng.standard_normal(n) * sqrt(1e-3)
            if i == 0:
                rows, cols = shp
                v = v.reshape(rows, cols)
                v[st["zero_rows"][st["zero_rows"] < rows]] = 0.0
                v = v.reshape(-1)
            parts.append(v)
        else:
            raise ValueError(wl.kind)
    return np.concatenate(parts).astype(np.float32)


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even) and return the
    16-bit patterns as uint16.  Used to make bf16 gradient inputs."""
    u = x.astype(np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)
