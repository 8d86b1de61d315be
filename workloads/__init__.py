"""Seeded synthetic inputs shared by the tests, the benchmark and the CPU
oracle's timing.  Input generation only: no compressor arithmetic lives here."""

from .generate import (BERT, FLAT1G, FLAT1M, RESNET18, RESNET50, WORKLOADS, Workload,
                       gradient, shared_seed, to_bf16_bits, worker_seed)
from . import shapes

__all__ = ["BERT", "FLAT1G", "FLAT1M", "RESNET18", "RESNET50", "WORKLOADS", "Workload",
           "gradient", "shared_seed", "to_bf16_bits", "worker_seed", "shapes"]
