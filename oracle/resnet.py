"""ResNet-50-shaped forward on the CPU oracle -- TEST INFRASTRUCTURE ONLY.

Composes the oracle's convolution (Sec. 3.2, direct from the definition, in
double precision) with the masked weights of the magnitude projection
(Sec. 5.1: top-K per group of G output channels), batch norm folded into a
per-channel scale and bias, ReLU, the bottleneck's residual add before its
last ReLU, exact max pooling, average pooling and the classifier, rounding to
bf16 at the points a bf16-activation network rounds: after every conv's
epilogue and after the average pool.  Logits stay in double precision.

Rounding detail: a double-precision result is rounded to fp32 and then to
bf16 (round to nearest even both times).  This differs from a single
rounding only when the fp32 value lands exactly on a bf16 tie, i.e. by at
most one bf16 ulp in rare elements, which the parity tolerance covers.

Parity pin: ``tests/test_oracle_resnet.py`` checks this composition against
torch's float64 functional convolution / pooling on a reduced network.
"""
from __future__ import annotations

import numpy as np

from . import (bf16_bits_to_f32, bf16_rne, conv2d_nhwc, dense_rows, global_avgpool_nhwc,
               maxpool2d_nhwc, pack, unpack)


def round_bf16(y) -> np.ndarray:
    """Values rounded to bf16, returned as exact fp32."""
    return bf16_bits_to_f32(bf16_rne(np.asarray(y, np.float32)))


def masked_weight(W: np.ndarray, G: int, K: int) -> np.ndarray:
    """Dense [O, C] matrix holding the K kept bf16 weights of every group
    (the projection of Sec. 5.1 applied to the fp32 master weights)."""
    v32, ix = pack(W, G, K)
    return unpack(round_bf16(v32), ix, G)


def conv_layer(x, L, W, G, scale, bias, residual=None, pixels=None, want_abs=False):
    """One conv + folded batch norm (+ residual) (+ ReLU), before rounding.
    x fp32 NHWC; returns float64 [npix, Cout] (and the sum of |terms|)."""
    Wm = masked_weight(W, G, L.K).reshape(L.Cout, L.k, L.k, L.Cin)
    return conv2d_nhwc(x, Wm, (L.stride, L.stride), (L.pad, L.pad), scale=scale, bias=bias,
                       residual=residual, relu=L.relu, pixels=pixels, want_abs=want_abs)


def resnet50_forward(X, layers, conv_weights, fc_weight, G, scales, biases):
    """X fp32 NHWC images (bf16 values); returns float64 logits [B, classes].

    ``layers`` lists the convs in network order (stem, then per bottleneck
    c1, c2, c3 and, in the first block of a stage, the downsample conv);
    ``scales`` / ``biases`` are the folded batch-norm vectors per conv."""
    def run(i, x, residual=None):
        L = layers[i]
        y = conv_layer(x, L, conv_weights[i], G, scales[i], biases[i], residual)
        B = x.shape[0]
        Ho = (x.shape[1] + 2 * L.pad - L.k) // L.stride + 1
        Wo = (x.shape[2] + 2 * L.pad - L.k) // L.stride + 1
        return round_bf16(y).reshape(B, Ho, Wo, L.Cout)

    x = run(0, np.asarray(X, np.float32))
    x = maxpool2d_nhwc(x, 3, 2, 1)
    i = 1
    while i < len(layers):
        ds = i + 3 < len(layers) and layers[i + 3].name.endswith(".ds")
        y = run(i, x)
        y = run(i + 1, y)
        ident = run(i + 3, x) if ds else x
        x = run(i + 2, y, residual=ident.reshape(-1, ident.shape[-1]))
        i += 4 if ds else 3
    pooled = round_bf16(global_avgpool_nhwc(x))
    Wfc = masked_weight(fc_weight, G, G)  # K = G: the dense classifier
    return dense_rows(pooled, Wfc)
