"""GPU parity on the workload shapes.

* the 2^20-element flat case in full: every worker and step, every compressor and the aggregate,
  bit-exact against the oracle;
* the ResNet-18 and ResNet-50 shapes at full size (per-layer and flat): the first workers over
  consecutive steps with the residual carried, bit-exact against the oracle, and the aggregate of
  16 full-size messages;
* the BERT shape (1.1e8 elements) and the 1e9-element flat case: exact certificates of the top-k
  and random-k definitions (the sent set is unique, and the certificate accepts it and no other)
  over the densities of the workloads, the block-random-k step against the oracle, and the
  aggregates of 32 messages;
* the ResNet-50 flat case over all 10 steps with the residual carried, and aggregates of 16
  messages of top-k's shape taken from the workers' own gradients.
"""

import numpy as np
import pytest

from efs_gpu import (Case, announce, assert_f32_equal, assert_msg_equal, certify_randk, certify_randk_chunked,
                     certify_topk, certify_topk_chunked, dev, host, synthetic_sparse_messages, topk_shaped_messages)
from oracle import efsparse_oracle as O
from workloads import WORKLOADS, gradient, to_bf16_bits, worker_seed

pytestmark = pytest.mark.gpu


def _steps(c, wl, kind, workers, steps, block=1, check=True):
    """Fused GPU steps against the oracle, residual carried; returns the oracle messages of the
    last step (one per worker)."""
    msgs = []
    for w in workers:
        e = np.zeros(c.d, np.float32)
        for t in steps:
            g = gradient(wl, w, t)
            ed = dev(e)
            m, val, _ = c.step(kind, g, ed, worker_seed(wl, w), t)
            (wm, wval), we = c.oracle_step(kind, g, e, worker_seed(wl, w), t)
            assert_msg_equal(kind, (m, val), (wm, wval), f"{wl.name} {kind} w{w} t{t}")
            assert_f32_equal(ed, we, f"{wl.name} {kind} e' w{w} t{t}")
            e = we
        msgs.append((wm, wval))
    return msgs


def _agg(c, kind, msgs, W):
    import torch
    import paper_2009_09271_amd as E
    out = torch.empty(c.d, dtype=torch.float32, device="cuda")
    a = np.stack([m[0] for m in msgs]).astype(np.uint32)
    v = np.stack([m[1] for m in msgs]).astype(np.float32)
    if kind == "sparse":
        E.decompress_aggregate(c.L, E.EF_MSG_SPARSE, W, dev(a.view(np.int32)), dev(v), out,
                               c.L.workspace(E.EF_OP_AGG_SPARSE, W))
        want = O.decompress_aggregate_sparse(c.d, a, v)
    else:
        E.decompress_aggregate(c.L, E.EF_MSG_BLOCK, W, dev(a.view(np.int32)), dev(v), out, None)
        want = O.decompress_aggregate_block(c.d, c.offs, c.ks, a, v)
    assert_f32_equal(out, want, f"aggregate {kind} W={W}")


@pytest.mark.parametrize("kind", ["topk", "randk", "randblock"])
def test_flat1m_every_worker_and_step(kind):
    wl = WORKLOADS["flat1m"]
    announce("flat1m", kind)
    block = wl.blocks[0] if kind == "randblock" else 1
    c = Case(wl.seg_offsets("flat"), wl.densities[0], block)
    es = [np.zeros(c.d, np.float32) for _ in range(wl.W)]
    for t in range(wl.steps):
        msgs = []
        for w in range(wl.W):
            g = gradient(wl, w, t)
            ed = dev(es[w])
            m, val, _ = c.step(kind, g, ed, worker_seed(wl, w), t)
            (wm, wval), we = c.oracle_step(kind, g, es[w], worker_seed(wl, w), t)
            assert_msg_equal(kind, (m, val), (wm, wval), f"flat1m {kind} w{w} t{t}")
            assert_f32_equal(ed, we, f"flat1m {kind} e' w{w} t{t}")
            es[w] = we
            msgs.append((wm, wval))
        _agg(c, "block" if kind == "randblock" else "sparse", msgs, wl.W)


@pytest.mark.parametrize("scope", ["layer", "flat"])
@pytest.mark.parametrize("kind,block", [("topk", 1), ("randk", 1), ("randblock", 1), ("randblock", 1024)])
def test_resnet18_full_size(scope, kind, block):
    wl = WORKLOADS["resnet18"]
    announce("resnet18", scope, kind, block)
    c = Case(wl.seg_offsets(scope), wl.densities[0], block)
    _steps(c, wl, kind, workers=[0, 1], steps=[0, 1], block=block)


@pytest.mark.parametrize("scope", ["flat", "layer"])
@pytest.mark.parametrize("kind,block", [("topk", 1), ("randk", 1), ("randblock", 256), ("randblock", 4096),
                                        ("randblock", 65536)])
def test_resnet50_full_size(scope, kind, block):
    wl = WORKLOADS["resnet50"]
    announce("resnet50", scope, kind, block)
    c = Case(wl.seg_offsets(scope), wl.densities[0], block)
    _steps(c, wl, kind, workers=[0], steps=[0, 1], block=block)


@pytest.mark.parametrize("scope", ["flat", "layer"])
def test_resnet50_aggregate_16_workers(scope):
    """Block messages of the 16 workers from the oracle, sparse messages synthetic (same shape)."""
    wl = WORKLOADS["resnet50"]
    announce("resnet50 aggregate", scope)
    c = Case(wl.seg_offsets(scope), wl.densities[0], 4096)
    blocks = []
    for w in range(wl.W):
        g = gradient(wl, w, 0)
        blocks.append(O.compress_randblock(g, c.offs, c.ks, 4096, worker_seed(wl, w), 0))
    _agg(c, "block", blocks, wl.W)
    idx, val = synthetic_sparse_messages(c.d, c.K, wl.W, 77)
    _agg(c, "sparse", list(zip(idx, val)), wl.W)


def _dominated(case):
    """Worker 0's ResNet-50 gradient with parts of much larger magnitude than the rest: the cases
    where a threshold sample that misses a small part would leave fewer than k candidates."""
    from workloads import shapes
    wl = WORKLOADS["resnet50"]
    g = gradient(wl, 0, 0).astype(np.float64)
    offs = wl.seg_offsets("layer")
    names = [n for n, _ in wl.tensor_shapes]
    rng = np.random.default_rng(2020)

    def fill(name, scale):
        i = names.index(name)
        g[offs[i]:offs[i + 1]] = rng.laplace(0.0, scale, offs[i + 1] - offs[i])

    if case in ("fc.bias", "both"):
        fill("fc.bias", 0.05)
    if case in ("conv1", "both"):
        fill("conv1.weight", 0.03)
    if case == "both":
        fill("bn1.bias", 1.0)  # 64 elements
    if case == "periodic":
        g[::781] *= 100.0  # a stride close to the sample's strata
    return g.astype(np.float32)


@pytest.mark.parametrize("case", ["fc.bias", "conv1", "both", "periodic"])
def test_topk_flat_with_a_dominant_small_tensor(case):
    """Top-k over the flat ResNet-50 gradient when one small tensor (the 1000-element fc.bias at
    Laplace scale 0.05, the stem convolution at 0.03, a 64-element bias at 1.0) or a periodic set of
    elements holds values far above the rest: bit-exact against the oracle, and the candidates of
    the threshold sample always contain the answer (the exact whole-segment path is not taken)."""
    import paper_2009_09271_amd as E
    wl = WORKLOADS["resnet50"]
    announce("resnet50 flat top-k, dominated by", case)
    c = Case(wl.seg_offsets("flat"), wl.densities[0])
    g = _dominated(case)
    e = np.zeros(c.d, np.float32)
    ed = dev(e)
    m, val, ws = c.step("topk", g, ed)
    (wm, wval), we = c.oracle_step("topk", g, e)
    assert_msg_equal("topk", (m, val), (wm, wval), f"dominated {case}")
    assert_f32_equal(ed, we, f"dominated {case} e'")
    assert c.L.diag(ws, E.EF_OP_TOPK) & E.DIAG_SLOW_PATH == 0, f"{case}: the exact whole-segment path ran"


@pytest.fixture(scope="module")
def bert_g():
    return gradient(WORKLOADS["bert"], 0, 0)


@pytest.mark.parametrize("scope,density,kind", [("layer", 0.01, "topk"), ("layer", 0.1, "topk"),
                                                ("flat", 0.1, "topk"), ("flat", 0.001, "topk"),
                                                ("layer", 0.01, "randk"), ("flat", 0.001, "randk"),
                                                ("layer", 0.01, "randblock"), ("flat", 0.1, "randblock")])
def test_bert_full_size(bert_g, scope, density, kind):
    """Per layer at 10 % the word embedding's k exceeds its nonzeros: zeros are chosen by index."""
    wl = WORKLOADS["bert"]
    announce("bert", scope, density, kind)
    block = wl.blocks[0] if kind == "randblock" else 1
    c = Case(wl.seg_offsets(scope), density, block)
    g = bert_g
    e = np.zeros(c.d, np.float32)
    ed = dev(e)
    seed = worker_seed(wl, 0)
    m, val, _ = c.step(kind, g, ed, seed, 0)
    if kind == "randblock":
        (wm, wval), we = c.oracle_step(kind, g, e, seed, 0)
        assert_msg_equal(kind, (m, val), (wm, wval), "bert randblock")
        assert_f32_equal(ed, we, "bert randblock e'")
        return
    acc = O.ef_accumulate(g, e)
    if kind == "topk":
        certify_topk(acc, c.offs, c.ks, host(m), host(val), host(ed), f"bert {scope} {density}")
    else:
        certify_randk(acc, c.offs, c.ks, host(m), host(val), host(ed), seed, 0, f"bert {scope} {density}")


@pytest.mark.parametrize("scope", ["layer", "flat"])
def test_bert_randk_10_percent(bert_g, scope):
    """Random-k at the densest BERT setting (K = 10.9 M): the exact certificate of the definition."""
    wl = WORKLOADS["bert"]
    announce("bert randk 10%", scope)
    c = Case(wl.seg_offsets(scope), 0.1)
    e = np.zeros(c.d, np.float32)
    ed = dev(e)
    seed = worker_seed(wl, 0)
    m, val, _ = c.step("randk", bert_g, ed, seed, 0)
    acc = O.ef_accumulate(bert_g, e)
    certify_randk_chunked(acc, c.offs, c.ks, host(m), host(val), host(ed), seed, 0, f"bert {scope} 10%")


def _grads(wl, W, t=0):
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(8) as ex:
        return list(ex.map(lambda w: gradient(wl, w, t), range(W)))


@pytest.mark.parametrize("wname,scope,density", [("resnet50", "flat", 0.001), ("resnet50", "layer", 0.001),
                                                 ("bert", "flat", 0.01)])
def test_aggregate_16_topk_shaped_messages(wname, scope, density):
    """The aggregate of the 16 workers' messages of top-k's shape (crowded into the layers of largest
    magnitude), taken from the workers' own gradients, against the oracle."""
    wl = WORKLOADS[wname]
    announce("aggregate of 16 top-k-shaped messages", wname, scope, density)
    c = Case(wl.seg_offsets(scope), density)
    idx, val = topk_shaped_messages(_grads(wl, 16), c.offs, c.ks)
    _agg(c, "sparse", list(zip(idx, val)), 16)


@pytest.mark.parametrize("kind,block", [("topk", 1), ("randk", 1), ("randblock", 4096)])
def test_resnet50_flat_ef_carried_ten_steps(kind, block):
    """Worker 0 over the workload's 10 steps, the residual carried from step to step."""
    wl = WORKLOADS["resnet50"]
    announce("resnet50 flat, 10 steps", kind, block)
    c = Case(wl.seg_offsets("flat"), wl.densities[0], block)
    _steps(c, wl, kind, workers=[0], steps=list(range(wl.steps)), block=block)


@pytest.fixture(scope="module")
def flat1g_g():
    return gradient(WORKLOADS["flat1g"], 0, 0)


FLAT1G_CASES = ["topk-f32-0.01%", "topk-f32-0.1%", "topk-f32-10%", "topk-bf16-1%",
                "randk-f32-0.01%", "randk-f32-1%", "randk-bf16-1%",
                "randblock-f32-1%-b2^20", "randblock-bf16-1%-b2^8",
                "aggregate-W32-0.01%", "block-aggregate-W32-0.1%-b2^12"]


@pytest.mark.parametrize("case", FLAT1G_CASES)
def test_flat1g(flat1g_g, case):
    """1e9 elements: top-k and random-k by exact certificates checked piece by piece (fp32 and bf16
    gradients), block-random-k against the oracle, and the sparse and block aggregates of 32
    messages against the oracle."""
    wl = WORKLOADS["flat1g"]
    announce("flat1g", case)
    offs = wl.seg_offsets("flat")
    g = flat1g_g
    parts = case.split("-")
    pct = {"0.01%": 1e-4, "0.1%": 1e-3, "1%": 1e-2, "10%": 1e-1}
    density = pct.get(parts[2]) if len(parts) > 2 else None
    if parts[0] in ("topk", "randk"):
        kind = parts[0]
        c = Case(offs, density)
        gi = to_bf16_bits(g) if parts[1] == "bf16" else g
        e = np.zeros(c.d, np.float32)
        ed = dev(e)
        seed = worker_seed(wl, 0)
        m, val, _ = c.step(kind, gi, ed, seed, 0)
        acc = O.ef_accumulate(gi, e)
        del e
        if kind == "topk":
            certify_topk_chunked(acc, c.offs, c.ks, host(m), host(val), host(ed), f"flat1g {case}")
        else:
            certify_randk_chunked(acc, c.offs, c.ks, host(m), host(val), host(ed), seed, 0, f"flat1g {case}")
    elif parts[0] == "randblock":
        b = 1 << int(parts[3][3:])
        c = Case(offs, density, b)
        gi = to_bf16_bits(g) if parts[1] == "bf16" else g
        e = np.zeros(c.d, np.float32)
        ed = dev(e)
        st, val, _ = c.step("randblock", gi, ed, worker_seed(wl, 0), 0)
        (wst, wval), we = c.oracle_step("randblock", gi, e, worker_seed(wl, 0), 0)
        assert_msg_equal("randblock", (st, val), (wst, wval), f"flat1g {case}")
        assert_f32_equal(ed, we, f"flat1g {case} e'")
    elif parts[0] == "aggregate":
        c = Case(offs, 0.0001)
        idx, val = synthetic_sparse_messages(c.d, c.K, wl.W, 78)
        _agg(c, "sparse", list(zip(idx, val)), wl.W)
    else:  # the block aggregate of 32 workers' messages: their own random starts, synthetic values
        b = 1 << 12
        c = Case(offs, 0.001, b)
        rng = np.random.default_rng(79)
        msgs = [(np.array([O.randblock_start(c.d, 0, b, worker_seed(wl, w), 0)], dtype=np.uint32),
                 rng.standard_normal(c.K).astype(np.float32)) for w in range(wl.W)]
        _agg(c, "block", msgs, wl.W)
