"""A chain of sparse-sparse layers run through the C ABI.

Each layer description needs the attributes kind ("conv"/"linear"), c_in,
c_out, n, kh, kw, stride, pad, pool, k (or None), shift (or None).  Weights
are packed once on the host (cs_pack), uploaded, and every buffer the chain
needs (workspaces, per-layer sums and k-WTA outputs) is allocated up front for
a fixed batch, so forward() only enqueues kernels.

Per layer: compaction + multiply/route/sum (+ bias, + 2x2 max-pool), then
k-WTA (+ int8 requantisation of the winners in int8 chains).  A conv output
feeding a linear layer is read as [batch][h*w*c] (NHWC flatten, no copy).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch

from . import ops
from .ops import conv_out


@dataclass
class PackedLayer:
    spec: object
    val: torch.Tensor        # [r][G] device
    kid: torch.Tensor        # [r][G] uint8 device
    bias: torch.Tensor | None
    holes: int


class Network:
    def __init__(self, layers, weights, biases, in_shape, batch: int, device="cuda"):
        self.layers = list(layers)
        self.device = torch.device(device)
        self.batch = batch
        self.in_shape = tuple(in_shape)
        self.packed = []
        for spec, W, b in zip(self.layers, weights, biases):
            W2 = np.asarray(W).reshape(spec.c_out, -1)
            val, kid, holes = ops.pack(W2, spec.n)
            bias = None if b is None else torch.from_numpy(np.asarray(b)).to(self.device)
            self.packed.append(PackedLayer(spec, torch.from_numpy(val).to(self.device),
                                           torch.from_numpy(kid).to(self.device), bias, holes))
        self._plan()

    # shapes and buffers ----------------------------------------------------
    def _plan(self):
        shape = (self.batch,) + self.in_shape
        self.in_shapes, self.acc, self.out, self.ws = [], [], [], []
        for p in self.packed:
            s = p.spec
            dt = torch.int8 if p.val.dtype == torch.int8 else torch.float32
            acc_dt = torch.int32 if dt == torch.int8 else torch.float32
            if s.kind == "conv":
                if len(shape) != 4:
                    raise ValueError(f"{s} needs an NHWC input, got {shape}")
                b, h, w, c = shape
                if c != s.c_in:
                    raise ValueError("channel mismatch")
                ho, wo = conv_out(h, s.kh, s.stride, s.pad), conv_out(w, s.kw, s.stride, s.pad)
                oshape = (b, ho // s.pool, wo // s.pool, s.c_out)
                ws = ops.workspace(1, dt, b * h * w, c, self.device)
            else:
                b = shape[0]
                d_in = int(np.prod(shape[1:]))
                if d_in != s.c_in:
                    raise ValueError("input length mismatch")
                oshape = (b, s.c_out)
                ws = ops.workspace(0, dt, b, d_in, self.device)
            self.in_shapes.append(shape)
            self.ws.append(ws)
            acc = torch.empty(oshape, dtype=acc_dt, device=self.device)
            self.acc.append(acc)
            if s.k is None:
                self.out.append(acc)
            else:
                odt = torch.int8 if s.shift is not None else acc_dt
                self.out.append(torch.empty(oshape, dtype=odt, device=self.device))
            shape = oshape
        self.out_shape = shape

    # execution -------------------------------------------------------------
    def forward_layer(self, li: int, x: torch.Tensor) -> torch.Tensor:
        p = self.packed[li]
        s = p.spec
        if s.kind == "conv":
            ops.conv2d(x, p.val, p.kid, s.kh, s.kw, s.n, s.stride, s.pad, p.bias, s.pool,
                       ws=self.ws[li], out=self.acc[li])
        else:
            ops.linear(x.reshape(x.shape[0], -1), p.val, p.kid, s.n, p.bias, ws=self.ws[li],
                       out=self.acc[li])
        if s.k is not None:
            if s.shift is not None:
                ops.kwta(self.acc[li], s.k, torch.int8, s.shift, out=self.out[li])
            else:
                ops.kwta(self.acc[li], s.k, out=self.out[li])
        return self.out[li]

    def forward(self, x: torch.Tensor) -> torch.Tensor:
        if tuple(x.shape) != tuple(self.in_shapes[0]):
            raise ValueError(f"input shape {tuple(x.shape)} != planned {self.in_shapes[0]}")
        cur = x
        for li in range(len(self.packed)):
            cur = self.forward_layer(li, cur)
        return cur
