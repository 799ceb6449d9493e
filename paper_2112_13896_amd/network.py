"""A chain of sparse-sparse layers run through the C ABI.

Each layer description needs the attributes kind ("conv"/"linear"), c_in,
c_out, n, kh, kw, stride, pad, pool, k (or None), shift (or None).  Weights
are packed once on the host (cs_pack) and uploaded.  Buffers (compaction
lists, per-layer sums, k-WTA outputs) live in a Buffers object allocated up
front for a fixed batch; several Buffers can share one Network, so a caller
can rotate among them.  forward() only enqueues kernels, on torch's current
stream.

Per layer: cs_compact (Select's (index, value) lists), cs_mrs_conv2d
(multiply/route/sum + bias + optional 2x2 max-pool), then cs_kwta (+ int8
requantisation of the winners in int8 chains).  A conv output feeding a
linear layer is read as [batch][h*w*c] (NHWC flatten, no copy).
"""
from __future__ import annotations

from dataclasses import dataclass, field

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


@dataclass
class Buffers:
    idx: list = field(default_factory=list)    # per layer: [rows][c_in] uint16 (as int16)
    lval: list = field(default_factory=list)   # per layer: [rows][c_in] list values
    cnt: list = field(default_factory=list)    # per layer: [rows] int32
    acc: list = field(default_factory=list)    # per layer: sums after pool
    out: list = field(default_factory=list)    # per layer: k-WTA / requantised output

    def nbytes(self) -> int:
        return sum(t.numel() * t.element_size() for lst in
                   (self.idx, self.lval, self.cnt, self.acc, self.out) for t in lst)


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
        self._shapes()
        self.bufs = self.make_buffers()

    @property
    def acc(self):
        return self.bufs.acc

    @property
    def out(self):
        return self.bufs.out

    # shapes and buffers ----------------------------------------------------
    def _shapes(self):
        shape = (self.batch,) + self.in_shape
        self.in_shapes, self.out_shapes, self.list_rows = [], [], []
        for p in self.packed:
            s = p.spec
            if s.kind == "conv":
                if len(shape) != 4:
                    raise ValueError(f"{s} needs an NHWC input, got {shape}")
                b, h, w, c = shape
                if c != s.c_in:
                    raise ValueError("channel mismatch")
                ho, wo = conv_out(h, s.kh, s.stride, s.pad), conv_out(w, s.kw, s.stride, s.pad)
                oshape = (b, ho // s.pool, wo // s.pool, s.c_out)
                rows = b * h * w
            else:
                b = shape[0]
                d_in = int(np.prod(shape[1:]))
                if d_in != s.c_in:
                    raise ValueError("input length mismatch")
                oshape = (b, s.c_out)
                rows = b
            self.in_shapes.append(shape)
            self.out_shapes.append(oshape)
            self.list_rows.append(rows)
            shape = oshape
        self.out_shape = shape

    def make_buffers(self) -> Buffers:
        B = Buffers()
        for p, oshape, rows in zip(self.packed, self.out_shapes, self.list_rows):
            s = p.spec
            dt = p.val.dtype
            acc_dt = torch.int32 if dt == torch.int8 else torch.float32
            lr = 0 if getattr(s, "dense_input", False) else rows
            B.idx.append(torch.empty((lr, s.c_in), dtype=torch.int16, device=self.device))
            B.lval.append(torch.empty((lr, s.c_in), dtype=dt, device=self.device))
            B.cnt.append(torch.empty((lr,), dtype=torch.int32, device=self.device))
            acc = torch.empty(oshape, dtype=acc_dt, device=self.device)
            B.acc.append(acc)
            if s.k is None:
                B.out.append(acc)
            else:
                odt = torch.int8 if s.shift is not None else acc_dt
                B.out.append(torch.empty(oshape, dtype=odt, device=self.device))
        return B

    # execution -------------------------------------------------------------
    def forward_layer(self, li: int, x: torch.Tensor, bufs: Buffers | None = None,
                      timer=None) -> torch.Tensor:
        B = self.bufs if bufs is None else bufs
        p = self.packed[li]
        s = p.spec
        rows = self.list_rows[li]
        t = timer or _NoTimer()
        if getattr(s, "dense_input", False):
            # sparse-dense variant: dense activations, no compaction
            t.start(f"{s.name}.mrs")
            ops.conv2d_dense(x, p.val, p.kid, s.kh, s.kw, s.n, s.stride, s.pad, p.bias, s.pool,
                             out=B.acc[li])
            t.stop(f"{s.name}.mrs")
            return self._select(li, s, B, t)
        xin = x.reshape(rows, s.c_in)
        t.start(f"{s.name}.compact")
        ops.compact_into(xin, B.idx[li], B.lval[li], B.cnt[li])
        t.stop(f"{s.name}.compact")
        if s.kind == "conv":
            geo = self.in_shapes[li]
            kh, kw, stride, pad, pool = s.kh, s.kw, s.stride, s.pad, s.pool
        else:
            geo = (rows, 1, 1, s.c_in)
            kh = kw = stride = pool = 1
            pad = 0
        acc = B.acc[li]
        t.start(f"{s.name}.mrs")
        ops.mrs_conv2d(B.idx[li], B.lval[li], B.cnt[li], geo, p.val, p.kid, kh, kw, s.n,
                       stride, pad, p.bias, pool, out=acc.reshape(
                           (geo[0], (conv_out(geo[1], kh, stride, pad)) // pool,
                            (conv_out(geo[2], kw, stride, pad)) // pool, s.c_out)))
        t.stop(f"{s.name}.mrs")
        return self._select(li, s, B, t)

    def _select(self, li, s, B, t):
        acc = B.acc[li]
        if s.k is not None:
            t.start(f"{s.name}.kwta")
            if s.shift is not None:
                ops.kwta(acc, s.k, torch.int8, s.shift, out=B.out[li])
            else:
                ops.kwta(acc, s.k, out=B.out[li])
            t.stop(f"{s.name}.kwta")
        return B.out[li]

    def forward(self, x: torch.Tensor, bufs: Buffers | None = None, timer=None) -> torch.Tensor:
        if tuple(x.shape) != tuple(self.in_shapes[0]):
            raise ValueError(f"input shape {tuple(x.shape)} != planned {self.in_shapes[0]}")
        cur = x
        for li in range(len(self.packed)):
            cur = self.forward_layer(li, cur, bufs, timer)
        return cur

    def kernel_names(self) -> list:
        names = []
        for p in self.packed:
            s = p.spec
            if not getattr(s, "dense_input", False):
                names.append(f"{s.name}.compact")
            names.append(f"{s.name}.mrs")
            if s.k is not None:
                names.append(f"{s.name}.kwta")
        return names


class _NoTimer:
    def start(self, name):
        pass

    def stop(self, name):
        pass


class EventTimer:
    """HIP events around selected launches, recorded on torch's current stream
    (the stream every launch of this package goes to)."""

    def __init__(self, names=None):
        self.names = None if names is None else set(names)
        self.pairs = {}
        self._open = {}

    def start(self, name):
        if self.names is None or name in self.names:
            e = torch.cuda.Event(enable_timing=True)
            e.record()
            self._open[name] = e

    def stop(self, name):
        if name in self._open:
            e = torch.cuda.Event(enable_timing=True)
            e.record()
            self.pairs.setdefault(name, []).append((self._open.pop(name), e))

    def mean_ms(self) -> dict:
        torch.cuda.synchronize()
        return {k: sum(a.elapsed_time(b) for a, b in v) / len(v) for k, v in self.pairs.items()}
