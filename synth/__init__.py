"""Seeded synthetic inputs shaped like SparseProp's workloads.

This module only draws random numbers: masks, weights, activations and
output gradients, returned as dense numpy arrays.  It holds none of the
method's arithmetic (no encoding, no products), so it can feed both the
HIP path and the CPU oracle.

Recipe (one ``numpy.random.default_rng(seed)`` per layer, fixed draw order):
  1. mask: ``k = floor((1 - sparsity) * numel + 0.5)`` positions drawn
     without replacement, i.e. an exact-count uniform unstructured mask;
  2. W: ``standard_normal(numel) * sigma`` cast to float32, then masked;
  3. X: ``standard_normal`` float32;
  4. dY: ``standard_normal`` float32.
sigma is 0.02 for linear layers and 0.05 for convolutions.  The seeds of
the named workloads are 1000 * (workload number - 1) + layer index.

The paper's datasets and pretrained sparse checkpoints are not used: these
draws stand in for them with the paper's layer shapes (the BERT-base FFN
768<->3072 of Sec. 4.1, ResNet 3x3 convolutions, and ResNet-18).
"""
from __future__ import annotations

import math

import numpy as np


def exact_count(numel: int, sparsity: float) -> int:
    """Number of stored entries of an exact-count mask."""
    return int(math.floor((1.0 - sparsity) * numel + 0.5))


def _mask(rng, shape, sparsity):
    numel = int(np.prod(shape))
    k = exact_count(numel, sparsity)
    pos = np.sort(rng.choice(numel, k, replace=False)) if k > 0 else np.zeros(0, np.int64)
    m = np.zeros(numel, np.uint8)
    m[pos] = 1
    return m.reshape(shape)


def linear_layer(seed: int, out_f: int, in_f: int, B: int, sparsity: float,
                 sigma: float = 0.02):
    """Dense mask/W (out_f x in_f), X (B x in_f), dY (B x out_f)."""
    rng = np.random.default_rng(seed)
    mask = _mask(rng, (out_f, in_f), sparsity)
    W = (rng.standard_normal(out_f * in_f) * sigma).astype(np.float32)
    W = W.reshape(out_f, in_f) * mask
    X = rng.standard_normal((B, in_f)).astype(np.float32)
    dY = rng.standard_normal((B, out_f)).astype(np.float32)
    return {"mask": mask, "W": W.astype(np.float32), "X": X, "dY": dY}


def conv_layer(seed: int, B: int, IC: int, H: int, W: int, OC: int, KH: int,
               KW: int, out_hw, sparsity: float, sigma: float = 0.05):
    """Dense mask/W [OC][IC][KH][KW], X [B][IC][H][W], dY [B][OC][OH][OW].

    ``out_hw`` is the output size (OH, OW) of the convolution, supplied by
    the caller so that this module does no convolution arithmetic."""
    rng = np.random.default_rng(seed)
    shape = (OC, IC, KH, KW)
    mask = _mask(rng, shape, sparsity)
    numel = int(np.prod(shape))
    Wt = (rng.standard_normal(numel) * sigma).astype(np.float32).reshape(shape) * mask
    X = rng.standard_normal((B, IC, H, W)).astype(np.float32)
    OH, OW = out_hw
    dY = rng.standard_normal((B, OC, OH, OW)).astype(np.float32)
    return {"mask": mask, "W": Wt.astype(np.float32), "X": X, "dY": dY}


# ----------------------------------------------------------------------
# Named workloads.  Linear entries: (name, out_f, in_f, B, sparsity).
# Conv entries: (name, B, IC, H, W, OC, KH, KW, stride, pad, sparsity).

LINEAR_SMALL = [("linear 256x256 @90% B16", 256, 256, 16, 0.90)]

FFN_PAIR = [
    ("ffn W1 768->3072 @95% B8192", 3072, 768, 8192, 0.95),
    ("ffn W2 3072->768 @95% B8192", 768, 3072, 8192, 0.95),
]

CONV_3X3_56 = [("conv3x3 64->64 56x56 s1p1 @90% B32", 32, 64, 56, 56, 64, 3, 3, 1, 1, 0.90)]


def conv_sweep():
    out = []
    for s in (0.80, 0.90, 0.95, 0.98):
        out.append(("conv3x3 128->128 28x28 @%d%% B32" % round(s * 100), 32, 128, 28, 28, 128, 3, 3, 1, 1, s))
        out.append(("conv3x3 256->256 14x14 @%d%% B32" % round(s * 100), 32, 256, 14, 14, 256, 3, 3, 1, 1, s))
        out.append(("conv1x1 256->1024 14x14 @%d%% B32" % round(s * 100), 32, 256, 14, 14, 1024, 1, 1, 1, 0, s))
    return out


def resnet18_convs(B: int = 64, sparsity: float = 0.95):
    """The 20 convolutions of a ResNet-18 at 224x224 (torchvision layout)."""
    L = [("conv1 7x7 s2", B, 3, 224, 224, 64, 7, 7, 2, 3, sparsity)]
    for blk in range(2):
        for c in range(2):
            L.append(("layer1.%d.conv%d" % (blk, c + 1), B, 64, 56, 56, 64, 3, 3, 1, 1, sparsity))
    for stage, (cin, cout, hw) in enumerate([(64, 128, 56), (128, 256, 28), (256, 512, 14)], start=2):
        oh = hw // 2
        L.append(("layer%d.0.conv1" % stage, B, cin, hw, hw, cout, 3, 3, 2, 1, sparsity))
        L.append(("layer%d.0.conv2" % stage, B, cout, oh, oh, cout, 3, 3, 1, 1, sparsity))
        L.append(("layer%d.0.downsample" % stage, B, cin, hw, hw, cout, 1, 1, 2, 0, sparsity))
        L.append(("layer%d.1.conv1" % stage, B, cout, oh, oh, cout, 3, 3, 1, 1, sparsity))
        L.append(("layer%d.1.conv2" % stage, B, cout, oh, oh, cout, 3, 3, 1, 1, sparsity))
    return L


RESNET18_FC = ("fc 512->1000", 1000, 512, 64, 0.95)


def seed_for(workload: int, layer: int) -> int:
    return 1000 * (workload - 1) + layer
