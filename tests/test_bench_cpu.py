"""CPU checks of bench.py's host side: the one-GPU contract, the variant list, the algorithmic byte
counts its roofline fractions divide by, and the CPU-baseline record (on a small sample)."""

import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


@pytest.mark.parametrize("n", [0, 2, 8])
def test_more_than_one_gpu_is_refused_with_a_message(n):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", str(n)],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr and r.stdout == ""


def test_variant_list():
    assert bench.variant_list("topk,randk,randblock", (256, 4096)) == \
        [("topk", 1), ("randk", 1), ("randblock", 256), ("randblock", 4096)]
    assert bench.variant_list("randblock64, topk", (256,)) == [("randblock", 64), ("topk", 1)]
    assert [bench.vname(v) for v in bench.variant_list("randk,randblock", (256,))] == ["randk", "randblock256"]


@pytest.mark.parametrize("d,K,L,W", [(25_557_032, 25_557, 1, 16), (1000, 10, 7, 3)])
def test_kernel_bytes_add_up_to_the_step_bytes(d, K, L, W):
    """A fused step reads g and e and writes e (4 bytes each per element) plus its message; the
    per-kernel figures of the streaming kernels add up to the per-operation figures."""
    for kind in ("topk", "randk"):
        step, agg = bench.alg_bytes_op(kind, d, K, L, W)
        assert step == bench.kernel_alg_bytes("k_stream_sel<1, true>", d, K, L, W) + 8 * K
        assert agg == bench.kernel_alg_bytes("k_agg_sparse", d, K, L, W)
        assert step == 3 * 4 * d + K * (4 + 4)  # index and value per sent element
    step, agg = bench.alg_bytes_op("randblock", d, K, L, W)
    assert step == bench.kernel_alg_bytes("k_randblock_step<0>", d, K, L, W) == 12 * d + 4 * K + 4 * L
    assert agg == bench.kernel_alg_bytes("k_agg_block", d, K, L, W)
    assert bench.kernel_alg_bytes("k_resolve", d, K, L, W) is None


def test_cpu_baseline_record():
    from oracle import efsparse_oracle as O
    from workloads import WORKLOADS
    wl = WORKLOADS["flat1m"]
    offs = [0, 30000, 50001]
    ks = O.segment_ks(offs, 0.01)
    rng = np.random.default_rng(5)
    W = 3
    grads = [rng.standard_normal(offs[-1]).astype(np.float32) for _ in range(W)]
    variants = [("topk", 1), ("randk", 1), ("randblock", 256)]
    r = bench._cpu_baseline(O, wl, offs, ks, variants, W, grads, "", min_s=0.0)
    assert r["kind"] == "oracle" and r["cores"] == 1 and r["unit"] == "elements/s"
    assert r["value"] > 0 and r["measured_s"] >= 0
    assert "workers 0..0" in r["sample"] and "randblock256" in r["sample"]


def test_cpu_baseline_pins_one_core_and_describes_the_host():
    from oracle import efsparse_oracle as O
    from workloads import WORKLOADS
    wl = WORKLOADS["flat1m"]
    offs = [0, 20000]
    ks = O.segment_ks(offs, 0.01)
    grads = [np.random.default_rng(6).standard_normal(offs[-1]).astype(np.float32)]
    before = os.sched_getaffinity(0)
    r = bench.cpu_baseline(wl, offs, ks, [("topk", 1)], 1, grads, "", min_s=0.0)
    assert os.sched_getaffinity(0) == before  # restored
    h = r["host"]
    assert h["os_cpu_count"] == os.cpu_count() and h["affinity"] == sorted(before)
    assert h["pinned_cpu"] in before and r["cores"] == 1
    assert h["cpu_model"] is None or isinstance(h["cpu_model"], str)
