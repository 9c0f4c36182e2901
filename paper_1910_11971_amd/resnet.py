"""ResNet-50-shaped forward pass on the CCI kernels (bf16 activations).

Every convolution, the first one and the classifier included, runs through
``cci_conv_im2col`` / ``cci_spmm``: the first conv and the FC layer carry
K = G (dense) packed weights, the other 52 convs K < G.  Batch norm at its
initial state is folded into each conv's epilogue scale and bias; the
bottleneck's residual add is fused into its last 1x1 conv, before the ReLU.
Pooling runs on the library's NHWC max-pool (exact) and global average pool
(fp32 accumulation, one rounding to bf16 before the FC).  Every conv output
is rounded to bf16 once, after its fused epilogue; the logits are fp32.

The first conv (7x7, stride 2, 3 channels) runs with its images copied into
a 4-channel buffer whose fourth channel stays zero and its weights
zero-padded to 7x8 taps of 4 channels: the sums are unchanged (every added
term is an exact zero), and the layer takes the matrix-core kernels' short
reduction path (a lane's 8 reduction columns are two adjacent taps' 4
channels, one 16-byte span of the image) instead of the vector-ALU path.
"""
from __future__ import annotations

import numpy as np
import torch

from . import cci
from .workloads import ResNet50, bn_fold


STEM_CIN, STEM_KW = 4, 8  # the first conv's channels and tap columns after zero padding


class ResNet50CCI:
    """Packs the weights once (``cci_pack`` per layer) and runs forwards."""

    def __init__(self, net: ResNet50, conv_weights, fc_weight, device="cuda"):
        self.net = net
        self.layers = net.layers
        self.device = torch.device(device)
        self.packed = []
        self._stem_in = None  # the zero-padded image buffer (one per input shape)
        for i, (L, w) in enumerate(zip(self.layers, conv_weights)):
            if i == 0:  # [Cout, k*k*Cin] -> [Cout, k*STEM_KW*STEM_CIN], zeros in the added taps / channels
                wp = np.zeros((L.Cout, L.k, STEM_KW, STEM_CIN), np.float32)
                wp[:, :, :L.k, :L.Cin] = np.asarray(w, np.float32).reshape(L.Cout, L.k, L.k, L.Cin)
                w = wp.reshape(L.Cout, -1)
            W = torch.from_numpy(np.ascontiguousarray(w)).to(self.device)
            vals, idx = cci.pack(W, net.G, L.K, torch.bfloat16)
            sc, bi = bn_fold(L.Cout)
            self.packed.append((vals, idx, torch.from_numpy(sc).to(self.device), torch.from_numpy(bi).to(self.device)))
        Wf = torch.from_numpy(np.ascontiguousarray(fc_weight)).to(self.device)
        self.fc = cci.pack(Wf, net.G, net.G, torch.bfloat16)

    def conv(self, i, x, residual=None):
        L = self.layers[i]
        vals, idx, sc, bi = self.packed[i]
        kw = STEM_KW if i == 0 else L.k
        return cci.conv_im2col(x, vals, idx, self.net.G, L.k, kw, (L.stride, L.stride), (L.pad, L.pad),
                               scale=sc, bias=bi, residual=residual, relu=L.relu, out_dtype=torch.bfloat16)

    def stem_input(self, X: torch.Tensor) -> torch.Tensor:
        """X [B, H, W, 3] copied into channels 0..2 of a [B, H, W', STEM_CIN]
        buffer whose other entries are zeroed when the buffer is allocated.
        W' = W rounded up to even: with 8 tap columns (the eighth all-zero)
        at stride 2 the output width (W' + 2*3 - 8)/2 + 1 then equals the
        7-tap width (W + 2*3 - 7)/2 + 1 for odd W too, and the extra input
        column is the zero padding the 7x7 conv would read there."""
        B, H, W, C = X.shape
        shape = (B, H, W + (W & 1), STEM_CIN)
        if self._stem_in is None or tuple(self._stem_in.shape) != shape:
            self._stem_in = torch.zeros(shape, dtype=X.dtype, device=X.device)
        self._stem_in[:, :, :W, :C].copy_(X)
        return self._stem_in

    def forward(self, X: torch.Tensor, record: list | None = None) -> torch.Tensor:
        """X bf16 NHWC [B, HW, HW, 3] on the device -> fp32 logits [B, classes].

        ``record``, if given, receives (kind, layer index or name, input, output)
        for every operation, with the residual of a fused add where there is one.
        """
        def rec(kind, key, inp, out, res=None):
            if record is not None:
                record.append((kind, key, inp, out, res))

        x = self.conv(0, self.stem_input(X))
        rec("conv", 0, X, x)
        y = cci.maxpool2d_nhwc(x, 3, 2, 1)
        rec("maxpool", "maxpool", x, y)
        x = y
        i = 1
        while i < len(self.layers):
            L = self.layers[i]
            assert L.name.endswith(".c1")
            has_ds = i + 3 < len(self.layers) and self.layers[i + 3].name.endswith(".ds")
            y1 = self.conv(i, x)
            rec("conv", i, x, y1)
            y2 = self.conv(i + 1, y1)
            rec("conv", i + 1, y1, y2)
            if has_ds:
                ident = self.conv(i + 3, x)
                rec("conv", i + 3, x, ident)
            else:
                ident = x
            y3 = self.conv(i + 2, y2, residual=ident)
            rec("conv", i + 2, y2, y3, ident)
            x = y3
            i += 4 if has_ds else 3
        pooled = cci.global_avgpool_nhwc(x, out_dtype=torch.bfloat16)
        rec("avgpool", "avgpool", x, pooled)
        vals, idx = self.fc
        logits = cci.spmm(pooled, vals, idx, self.net.G, out_dtype=torch.float32)
        rec("fc", "fc", pooled, logits)
        return logits
