"""Parameter-tensor shape lists for the synthetic gradient workloads.

The paper trains ResNet-18 (Section 4.1, experimental setup) and sparsifies
either each layer's gradient separately or the concatenation of all layers
(Section 3, sparsification scope).  Real gradients are not available here, so
the workloads use synthetic values laid out like the parameter tensors of
three standard architectures, in the order a framework would flatten them:

* ResNet-18 (ImageNet form: 7x7 stem, fc 512 -> 1000): 62 tensors, 11,689,512
* ResNet-50 (bottleneck blocks, fc 2048 -> 1000):      161 tensors, 25,557,032
* BERT-base encoder (vocab 30522, hidden 768, FFN 3072, 12 layers, pooler):
  199 tensors, 109,482,240

Each entry is ``(name, shape)``.  Weights and biases are separate tensors, so a
"layer" in layer-wise scope is one parameter tensor.  This module holds only
architecture shapes; it performs none of the compression arithmetic.
"""

from __future__ import annotations

from math import prod


def resnet18_shapes():
    out = [("conv1.weight", (64, 3, 7, 7)), ("bn1.weight", (64,)), ("bn1.bias", (64,))]
    inplanes = 64
    for stage, planes in enumerate((64, 128, 256, 512), start=1):
        for blk in range(2):
            stride_change = blk == 0 and planes != inplanes
            p = f"layer{stage}.{blk}."
            cin = inplanes if blk == 0 else planes
            out += [
                (p + "conv1.weight", (planes, cin, 3, 3)),
                (p + "bn1.weight", (planes,)),
                (p + "bn1.bias", (planes,)),
                (p + "conv2.weight", (planes, planes, 3, 3)),
                (p + "bn2.weight", (planes,)),
                (p + "bn2.bias", (planes,)),
            ]
            if stride_change:
                out += [
                    (p + "downsample.0.weight", (planes, cin, 1, 1)),
                    (p + "downsample.1.weight", (planes,)),
                    (p + "downsample.1.bias", (planes,)),
                ]
        inplanes = planes
    out += [("fc.weight", (1000, 512)), ("fc.bias", (1000,))]
    return out


def resnet50_shapes():
    out = [("conv1.weight", (64, 3, 7, 7)), ("bn1.weight", (64,)), ("bn1.bias", (64,))]
    inplanes = 64
    for stage, (planes, nblocks) in enumerate(((64, 3), (128, 4), (256, 6), (512, 3)), start=1):
        for blk in range(nblocks):
            p = f"layer{stage}.{blk}."
            cin = inplanes if blk == 0 else planes * 4
            out += [
                (p + "conv1.weight", (planes, cin, 1, 1)),
                (p + "bn1.weight", (planes,)),
                (p + "bn1.bias", (planes,)),
                (p + "conv2.weight", (planes, planes, 3, 3)),
                (p + "bn2.weight", (planes,)),
                (p + "bn2.bias", (planes,)),
                (p + "conv3.weight", (planes * 4, planes, 1, 1)),
                (p + "bn3.weight", (planes * 4,)),
                (p + "bn3.bias", (planes * 4,)),
            ]
            if blk == 0:
                out += [
                    (p + "downsample.0.weight", (planes * 4, cin, 1, 1)),
                    (p + "downsample.1.weight", (planes * 4,)),
                    (p + "downsample.1.bias", (planes * 4,)),
                ]
        inplanes = planes * 4
    out += [("fc.weight", (1000, 2048)), ("fc.bias", (1000,))]
    return out


def bert_base_shapes(vocab=30522, hidden=768, ffn=3072, layers=12, max_pos=512, types=2):
    h = hidden
    out = [
        ("embeddings.word_embeddings.weight", (vocab, h)),
        ("embeddings.position_embeddings.weight", (max_pos, h)),
        ("embeddings.token_type_embeddings.weight", (types, h)),
        ("embeddings.LayerNorm.weight", (h,)),
        ("embeddings.LayerNorm.bias", (h,)),
    ]
    for i in range(layers):
        p = f"encoder.layer.{i}."
        for m in ("query", "key", "value"):
            out += [(p + f"attention.self.{m}.weight", (h, h)), (p + f"attention.self.{m}.bias", (h,))]
        out += [
            (p + "attention.output.dense.weight", (h, h)),
            (p + "attention.output.dense.bias", (h,)),
            (p + "attention.output.LayerNorm.weight", (h,)),
            (p + "attention.output.LayerNorm.bias", (h,)),
            (p + "intermediate.dense.weight", (ffn, h)),
            (p + "intermediate.dense.bias", (ffn,)),
            (p + "output.dense.weight", (h, ffn)),
            (p + "output.dense.bias", (h,)),
            (p + "output.LayerNorm.weight", (h,)),
            (p + "output.LayerNorm.bias", (h,)),
        ]
    out += [("pooler.dense.weight", (h, h)), ("pooler.dense.bias", (h,))]
    return out


def numel(shapes):
    return sum(prod(s) for _, s in shapes)


def segment_offsets(shapes):
    """Offsets [0, n_0, n_0+n_1, ..., d] of each tensor in the flattened vector."""
    offs = [0]
    for _, s in shapes:
        offs.append(offs[-1] + prod(s))
    return offs


def scaled(shapes, div):
    """The same architecture with every dimension except kernel sizes divided by
    ``div`` (at least 1): keeps the tensor count, ordering and the mix of 1-D /
    conv / matrix tensors, at a size the CPU oracle handles in seconds."""
    out = []
    for name, s in shapes:
        if len(s) == 4:
            ns = (max(1, s[0] // div), max(1, s[1] // div), s[2], s[3])
        else:
            ns = tuple(max(1, x // div) for x in s)
        out.append((name, ns))
    return out
