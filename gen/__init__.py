"""Seeded synthetic inputs shaped like the paper's workloads.

This module only draws random numbers and lays them out. It holds none of the
method's arithmetic (no residual add, no selection, no aggregation, no update),
so both the CPU oracle and the HIP path can be fed from it without sharing any
part of the computation.

Every draw comes from ``numpy.random.default_rng(SeedSequence([ROOT, config,
step, tensor, stream]))``. Values are drawn in float64 and rounded to float32
(round-to-nearest-even, numpy's ``astype``).

Workload shapes:

* ResNet-50 gradient set: the torchvision ResNet-50 parameter list, 161
  tensors, 25,557,032 elements. The paper's layer-wise LR discussion counts 161
  layers for this model (Sec. 4.2, "PTO for LARS") and its HiTopKComm breakdown
  uses 25 M parameters for it (Sec. 5.3).
* Transformer gradient set: a 6+6-layer, d_model 512 Transformer with four
  32,000 x 512 vocabulary matrices, 109,708,544 elements, standing in for the
  "110 million parameters" model of Sec. 5.3.
* Flat buffers: the 256 K .. 128 M single-vector sweep of Sec. 5.2, and a
  340 M BERT-large-sized buffer with planted magnitude ties.
"""
from __future__ import annotations

import math
from typing import List, Sequence, Tuple

import numpy as np

ROOT_SEED = 201010458

# stream ids inside one (config, step, tensor) seed
S_VALUES = 0
S_OUTLIER = 1
S_PARAMS = 2
S_LIST_IDX = 3
S_LIST_VAL = 4
S_TIES = 5


def rng(config: int, step: int, tensor: int, stream: int) -> np.random.Generator:
    return np.random.default_rng(
        np.random.SeedSequence([ROOT_SEED, config, step, tensor, stream]))


# --------------------------------------------------------------------------
# shape recipes
# --------------------------------------------------------------------------

def resnet50_shapes() -> List[Tuple[str, Tuple[int, ...]]]:
    """torchvision ResNet-50 parameters in module order (161 tensors)."""
    out: List[Tuple[str, Tuple[int, ...]]] = [
        ("conv1.weight", (64, 3, 7, 7)), ("bn1.weight", (64,)), ("bn1.bias", (64,))]
    inplanes = 64
    for si, (width, blocks) in enumerate(zip([64, 128, 256, 512], [3, 4, 6, 3])):
        for b in range(blocks):
            p = f"layer{si + 1}.{b}."
            out += [(p + "conv1.weight", (width, inplanes, 1, 1)),
                    (p + "bn1.weight", (width,)), (p + "bn1.bias", (width,)),
                    (p + "conv2.weight", (width, width, 3, 3)),
                    (p + "bn2.weight", (width,)), (p + "bn2.bias", (width,)),
                    (p + "conv3.weight", (4 * width, width, 1, 1)),
                    (p + "bn3.weight", (4 * width,)), (p + "bn3.bias", (4 * width,))]
            if b == 0:
                out += [(p + "downsample.0.weight", (4 * width, inplanes, 1, 1)),
                        (p + "downsample.1.weight", (4 * width,)),
                        (p + "downsample.1.bias", (4 * width,))]
            inplanes = 4 * width
    out += [("fc.weight", (1000, 2048)), ("fc.bias", (1000,))]
    return out


def transformer_shapes(vocab: int = 32000, d_model: int = 512, d_ff: int = 2048,
                       layers: int = 6) -> List[Tuple[str, Tuple[int, ...]]]:
    """Transformer-base-like parameter list, 109,708,544 elements.

    Separate Q/K/V/O projections with biases, a two-matrix FFN, LayerNorm gain
    and bias (two per encoder layer, three per decoder layer, one final norm on
    each side), source and target embeddings, an output projection with bias,
    and a fourth vocabulary-sized matrix that brings the total to the size the
    paper quotes for its Transformer.
    """
    out: List[Tuple[str, Tuple[int, ...]]] = []

    def attn(p):
        for m in ("q", "k", "v", "o"):
            out.append((p + m + ".weight", (d_model, d_model)))
            out.append((p + m + ".bias", (d_model,)))

    def ffn(p):
        out.extend([(p + "w1.weight", (d_ff, d_model)), (p + "w1.bias", (d_ff,)),
                    (p + "w2.weight", (d_model, d_ff)), (p + "w2.bias", (d_model,))])

    def ln(p):
        out.extend([(p + ".weight", (d_model,)), (p + ".bias", (d_model,))])

    out.append(("src_embed.weight", (vocab, d_model)))
    for i in range(layers):
        p = f"encoder.{i}."
        attn(p + "self_attn.")
        ln(p + "norm1")
        ffn(p + "ffn.")
        ln(p + "norm2")
    ln("encoder.norm")
    out.append(("tgt_embed.weight", (vocab, d_model)))
    for i in range(layers):
        p = f"decoder.{i}."
        attn(p + "self_attn.")
        ln(p + "norm1")
        attn(p + "cross_attn.")
        ln(p + "norm2")
        ffn(p + "ffn.")
        ln(p + "norm3")
    ln("decoder.norm")
    out.append(("generator.weight", (vocab, d_model)))
    out.append(("generator.bias", (vocab,)))
    out.append(("aux_vocab.weight", (vocab, d_model)))
    return out


def numels(shapes: Sequence[Tuple[str, Tuple[int, ...]]]) -> List[int]:
    return [int(np.prod(s)) for _, s in shapes]


# --------------------------------------------------------------------------
# value distributions
# --------------------------------------------------------------------------

def normal_f32(g: np.random.Generator, n: int, std: float) -> np.ndarray:
    return (g.standard_normal(n) * std).astype(np.float32)


def resnet_grads(step: int, config: int = 2, std: float = 1e-2,
                 outlier_p: float = 0.01, outlier_scale: float = 100.0,
                 sizes: Sequence[int] | None = None) -> List[np.ndarray]:
    """N(0, std) per element, a Bernoulli(outlier_p) subset scaled by
    outlier_scale, one array per tensor."""
    sizes = numels(resnet50_shapes()) if sizes is None else sizes
    out = []
    for t, n in enumerate(sizes):
        v = rng(config, step, t, S_VALUES).standard_normal(n) * std
        m = rng(config, step, t, S_OUTLIER).random(n) < outlier_p
        v[m] *= outlier_scale
        out.append(v.astype(np.float32))
    return out


def laplace_grads(step: int, sizes: Sequence[int], scale: float = 1e-3,
                  config: int = 3) -> List[np.ndarray]:
    return [rng(config, step, t, S_VALUES).laplace(0.0, scale, n).astype(np.float32)
            for t, n in enumerate(sizes)]


def flat_normal(n: int, config: int, step: int = 0, std: float = 1.0,
                chunk: int = 1 << 24) -> np.ndarray:
    """One flat N(0, std) float32 buffer, drawn chunk by chunk (bounded host
    memory for the 340 M case)."""
    out = np.empty(n, dtype=np.float32)
    for c, s in enumerate(range(0, n, chunk)):
        e = min(n, s + chunk)
        out[s:e] = (rng(config, step, c, S_VALUES).standard_normal(e - s) * std)
    return out


def params_like(sizes: Sequence[int], config: int, std: float = 0.1) -> List[np.ndarray]:
    return [normal_f32(rng(config, 0, t, S_PARAMS), n, std) for t, n in enumerate(sizes)]


# Inverse normal CDF at 1 - 0.0005 (two-sided 0.1 % tail of N(0, 1)).
NORMAL_TAIL_0P001 = 3.2905267314919255


def tie_stressed(n: int, config: int = 4, tie_frac: float = 0.1,
                 band: float = 5e-3, anchor: float = NORMAL_TAIL_0P001) -> np.ndarray:
    """Flat N(0, 1) buffer with exact-duplicate magnitudes.

    A Bernoulli(tie_frac) subset is truncated to bfloat16 precision (low 16
    bits cleared, sign kept), which creates exact-duplicate magnitude classes
    at every scale. Subset members whose magnitude lies within a relative
    ``band`` of ``anchor`` (the expected 0.1 % two-sided tail point of
    N(0, 1)) are then set to exactly +-anchor, so that a large tie class sits
    where a rho = 0.001 selection boundary falls.
    """
    x = flat_normal(n, config)
    chunk = 1 << 24
    a32 = np.float32(anchor)
    for c, s in enumerate(range(0, n, chunk)):
        e = min(n, s + chunk)
        sub = rng(config, 0, c, S_TIES).random(e - s) < tie_frac
        seg = x[s:e]
        bits = seg.view(np.uint32)
        bits[sub] &= np.uint32(0xFFFF0000)
        mag = np.abs(seg)
        snap = sub & (np.abs(mag - a32) <= band * a32)
        seg[snap] = np.copysign(a32, seg[snap])
    return x


def sparse_lists(d: int, P: int, k: int, config: int = 5, step: int = 0,
                 std: float = 1e-2) -> Tuple[np.ndarray, np.ndarray]:
    """P workers' sparse gradients in the gathered layout of Alg. 2: worker p's
    k indices (distinct, ascending, uniform over [0, d)) at rows p of a
    (P, k) int32 array, and its N(0, std) values at the same place."""
    idx = np.empty((P, k), dtype=np.int32)
    val = np.empty((P, k), dtype=np.float32)
    for p in range(P):
        idx[p] = np.sort(rng(config, step, p, S_LIST_IDX).choice(d, size=k, replace=False))
        val[p] = normal_f32(rng(config, step, p, S_LIST_VAL), k, std)
    return idx, val


# --------------------------------------------------------------------------
# named workloads
# --------------------------------------------------------------------------

RESNET50_D = 25_557_032
TRANSFORMER_D = 109_708_544
BERT_LARGE_D = 340_000_000
C1_D = 1 << 20


def concat(arrs: Sequence[np.ndarray]) -> np.ndarray:
    return np.concatenate([np.asarray(a, dtype=np.float32).ravel() for a in arrs])
