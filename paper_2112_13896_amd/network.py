"""A chain of sparse-sparse layers run through the C ABI.

Each layer description needs the attributes name, kind ("conv"/"linear"),
c_in, c_out, n, kh, kw, stride, pad, pool, k (or None), shift (or None) and
optionally dense_input.  Weights are packed once on the host (cs_pack) and
uploaded.  Buffers live in a Buffers object allocated up front for a fixed
batch; several Buffers can share one Network so a caller can rotate among
them.  forward() only enqueues kernels, on torch's current stream.

Data flow (Section 3.2; Figure 10 sends the k-WTA winners on "along with
their indices"):
  * the first layer's dense input is compacted into (index, value) lists
    (cs_compact), or read densely by the sparse-dense kernel when the layer
    is marked dense_input (cs_conv2d_dense);
  * multiply/route/sum + bias + optional 2x2 max-pool + k-WTA run as one
    call (cs_mrs_kwta_conv2d) that reads the lists and emits the next layer's
    lists directly (capacity k rounded up to 4, winners requantised to int8
    in int8 chains), or a dense masked output for the last layer; the sums
    reach HBM only when keep_sums is set (tests) - a layer whose packed table
    is too large for one workgroup falls back inside the library to separate
    sum and k-WTA kernels;
  * a dense first layer runs as the sparse-dense variant (dense input, dense
    weights), with k-WTA in the same call (cs_conv2d_dense_kwta);
  * a layer without k-WTA writes its sums (cs_mrs_conv2d / cs_conv2d_dense);
  * the last layer, a linear layer without k-WTA on the int8 winners of a
    layer with one output vector per sample, runs in that layer's call
    (cs_mrs_kwta_chain2: the winners feed it on chip) unless fuse_tail is off;
    when that pair reads a conv layer's lists as a window over its whole
    pooled map, the three run in the conv layer's call (cs_mrs_kwta_chain3),
    and when that conv layer reads a dense-input first layer's lists, all
    four run in the first layer's call (cs_conv2d_dense_kwta_chain3).
A linear layer that follows a conv layer reads the conv output's per-pixel
lists as a convolution whose window is the whole h x w map: its slots
(h, w, c) in NHWC flatten order are exactly the window's taps-major slots.
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
    aug: torch.Tensor        # augmented packed tensor [r][G] on the device
    bias: torch.Tensor | None
    holes: int


@dataclass
class Plan:
    """How one layer runs: list geometry and kernel parameters."""
    in_lists: bool           # input arrives as the previous layer's k-WTA lists
    dense_kernel: bool       # sparse-dense kernel on a dense input
    geo: tuple               # (b, h, w, c_in) of the list rows / dense input
    kh: int
    kw: int
    stride: int
    pad: int
    pool: int
    out_shape: tuple         # sums after pool
    emit_lists: bool         # k-WTA writes lists for the next layer
    cap_out: int             # capacity of the emitted lists
    fuse_next: bool = False  # the next (last) layer runs in this layer's call
    fuse_next2: bool = False  # the next two (last) layers run in this layer's call
    fuse_next3: bool = False  # the next three (last) layers run in this layer's call


@dataclass
class Buffers:
    idx: list = field(default_factory=list)     # per layer: compaction lists (dense input only)
    lval: list = field(default_factory=list)
    cnt: list = field(default_factory=list)
    acc: list = field(default_factory=list)     # per layer: sums after pool
    out: list = field(default_factory=list)     # per layer: dense k-WTA output, or None
    lists: list = field(default_factory=list)   # per layer: (idx, val, cnt) emitted, or None

    def nbytes(self) -> int:
        ts = [t for lst in (self.idx, self.lval, self.cnt, self.acc, self.out) for t in lst
              if t is not None]
        ts += [t for trip in self.lists if trip is not None for t in trip]
        return sum(t.numel() * t.element_size() for t in ts)


class Network:
    def __init__(self, layers, weights, biases, in_shape, batch: int, device="cuda",
                 keep_sums: bool = True, fuse_tail: bool = True):
        self.layers = list(layers)
        self.keep_sums = keep_sums
        self.fuse_tail = fuse_tail
        self.device = torch.device(device)
        self.batch = batch
        self.in_shape = tuple(in_shape)
        self.packed = []
        for spec, W, b in zip(self.layers, weights, biases):
            W2 = np.asarray(W).reshape(spec.c_out, -1)
            aug, holes = ops.pack(W2, spec.n)
            bias = None if b is None else torch.from_numpy(np.asarray(b)).to(self.device)
            self.packed.append(PackedLayer(spec, ops.aug_to_device(aug, self.device), bias, holes))
        self._plan()
        self.bufs = self.make_buffers()

    @property
    def acc(self):
        return self.bufs.acc

    @property
    def out(self):
        return self.bufs.out

    # plan ------------------------------------------------------------------
    def _plan(self):
        shape = (self.batch,) + self.in_shape
        self.plans = []
        self.in_shapes = []
        nl = len(self.packed)
        prev_k = None
        for li, p in enumerate(self.packed):
            s = p.spec
            in_lists = prev_k is not None
            if s.kind == "conv":
                if len(shape) != 4 or shape[3] != s.c_in:
                    raise ValueError(f"layer {s.name}: NHWC input with {s.c_in} channels expected")
                b, h, w, c = shape
                geo = (b, h, w, c)
                kh, kw, st, pad, pool = s.kh, s.kw, s.stride, s.pad, s.pool
                ho, wo = conv_out(h, kh, st, pad), conv_out(w, kw, st, pad)
                oshape = (b, ho // pool, wo // pool, s.c_out)
            else:
                b = shape[0]
                if int(np.prod(shape[1:])) != s.c_in:
                    raise ValueError(f"layer {s.name}: input length {s.c_in} expected")
                if len(shape) == 4:
                    # linear after conv: a convolution whose window is the whole map
                    geo = shape
                    kh, kw = shape[1], shape[2]
                else:
                    geo = (b, 1, 1, s.c_in)
                    kh = kw = 1
                st, pad, pool = 1, 0, 1
                oshape = (b, s.c_out)
            dense_kernel = bool(getattr(s, "dense_input", False)) and not in_lists
            emit = s.k is not None and li + 1 < nl
            self.plans.append(Plan(in_lists, dense_kernel, geo, kh, kw, st, pad, pool, oshape,
                                   emit, ops.list_capacity(s.k) if emit else 0))
            self.in_shapes.append(shape)
            prev_k = s.k
            shape = oshape
        self.out_shape = shape
        # the tail: a last linear layer without k-WTA on the int8 winners of a
        # layer whose output is one vector per sample
        if self.fuse_tail and nl >= 2:
            a, z = self.plans[nl - 2], self.plans[nl - 1]
            sa, sz = self.packed[nl - 2].spec, self.packed[nl - 1].spec
            int8 = self.packed[nl - 2].aug.dtype == torch.int16 and self.packed[nl - 1].aug.dtype == torch.int16
            if (int8 and sa.k is not None and sa.shift is not None and a.emit_lists and
                    not a.dense_kernel and len(a.out_shape) == 2 and sz.kind == "linear" and
                    sz.k is None and z.in_lists):
                a.fuse_next = True
        # a conv layer whose lists feed that pair as a window over its whole
        # pooled map: the three run in one call (cs_mrs_kwta_chain3)
        if self.fuse_tail and nl >= 3 and self.plans[nl - 2].fuse_next:
            c, a = self.plans[nl - 3], self.plans[nl - 2]
            sc = self.packed[nl - 3].spec
            int8 = self.packed[nl - 3].aug.dtype == torch.int16
            if (int8 and sc.k is not None and sc.shift is not None and c.emit_lists and
                    not c.dense_kernel and len(c.out_shape) == 4 and a.in_lists and
                    tuple(a.geo) == tuple(c.out_shape) and a.kh == c.out_shape[1] and
                    a.kw == c.out_shape[2] and a.stride == 1 and a.pad == 0 and a.pool == 1):
                c.fuse_next2 = True
        # a dense-input first layer whose lists feed those three: all four in
        # one call (cs_conv2d_dense_kwta_chain3)
        if self.fuse_tail and nl == 4 and self.plans[1].fuse_next2:
            d = self.plans[0]
            sd = self.packed[0].spec
            int8 = self.packed[0].aug.dtype == torch.int16
            if (int8 and d.dense_kernel and sd.k is not None and sd.shift is not None and
                    d.emit_lists and self.plans[1].in_lists):
                d.fuse_next3 = True

    def make_buffers(self) -> Buffers:
        B = Buffers()
        for p, pl in zip(self.packed, self.plans):
            s = p.spec
            dt = torch.int8 if p.aug.dtype == torch.int16 else torch.float32
            acc_dt = torch.int32 if dt == torch.int8 else torch.float32
            b, h, w, c = pl.geo
            rows = b * h * w
            if not pl.in_lists and not pl.dense_kernel:
                B.idx.append(torch.empty((rows, c), dtype=torch.int16, device=self.device))
                B.lval.append(torch.empty((rows, c), dtype=dt, device=self.device))
                B.cnt.append(torch.empty((rows,), dtype=torch.int32, device=self.device))
            else:
                B.idx.append(None)
                B.lval.append(None)
                B.cnt.append(None)
            acc = torch.empty(pl.out_shape, dtype=acc_dt, device=self.device)
            B.acc.append(acc)
            if s.k is None:
                B.out.append(acc)
                B.lists.append(None)
            elif pl.emit_lists:
                orow = int(np.prod(pl.out_shape[:-1]))
                odt = torch.int8 if s.shift is not None else acc_dt
                B.out.append(None)
                B.lists.append((torch.empty((orow, pl.cap_out), dtype=torch.int16, device=self.device),
                                torch.empty((orow, pl.cap_out), dtype=odt, device=self.device),
                                torch.empty((orow,), dtype=torch.int32, device=self.device)))
            else:
                odt = torch.int8 if s.shift is not None else acc_dt
                B.out.append(torch.empty(pl.out_shape, dtype=odt, device=self.device))
                B.lists.append(None)
        return B

    # execution -------------------------------------------------------------
    def launches(self, li: int, x, bufs: Buffers | None = None) -> list:
        """The kernel launches of layer li as (name, call) pairs in order; each
        call enqueues one library call on torch's current stream, reading and
        writing only preallocated buffers, so a call can be replayed alone or
        recorded into a HIP graph.  x: the dense input (first layer) or None
        (the lists of layer li-1)."""
        B = self.bufs if bufs is None else bufs
        p = self.packed[li]
        s = p.spec
        pl = self.plans[li]
        b, h, w, c = pl.geo
        acc = B.acc[li]
        acc4 = acc.reshape(b, -1, 1, s.c_out) if acc.dim() == 2 else acc
        odt = torch.int8 if s.shift is not None else None
        shift = s.shift if s.shift is not None else 0
        lists_out = B.lists[li] if pl.emit_lists else None
        out = None if pl.emit_lists else B.out[li]
        calls = []
        if pl.dense_kernel and pl.fuse_next3:
            # one call: this layer and the three after it on its lists
            q, r, t = self.packed[li + 1], self.packed[li + 2], self.packed[li + 3]
            pq = self.plans[li + 1]
            bq = pq.geo[0]
            calls.append((f"{s.name}.dense_kwta+{q.spec.name}.mrs_kwta+{r.spec.name}.mrs_kwta+"
                          f"{t.spec.name}.mrs", lambda: ops.conv2d_dense_kwta_chain3(
                x, p.aug, pl.kh, pl.kw, s.n, pl.stride, pl.pad, p.bias, pl.pool, k=s.k,
                shift=shift, aug2=q.aug, kh2=pq.kh, kw2=pq.kw, n2=q.spec.n, stride2=pq.stride,
                pad2=pq.pad, bias2=q.bias, pool2=pq.pool, k2=q.spec.k, shift2=q.spec.shift,
                aug3=r.aug, n3=r.spec.n, bias3=r.bias, k3=r.spec.k, shift3=r.spec.shift,
                aug4=t.aug, n4=t.spec.n, bias4=t.bias, keep_sums=self.keep_sums, y=acc,
                lists=lists_out, y2=B.acc[li + 1], lists2=B.lists[li + 1],
                y3=B.acc[li + 2].reshape(bq, -1), lists3=B.lists[li + 2], y4=B.acc[li + 3])))
            return calls
        if pl.dense_kernel:
            if s.k is not None:
                # sparse-dense variant with k-WTA: dense activations, no
                # compaction, one call (on the matrix cores where it applies)
                calls.append((f"{s.name}.dense_kwta", lambda: ops.conv2d_dense_kwta(
                    x, p.aug, pl.kh, pl.kw, s.n, pl.stride, pl.pad, p.bias, pl.pool, k=s.k,
                    out_dtype=odt, shift=shift, y=acc, keep_sums=self.keep_sums,
                    lists=lists_out, out=out)))
            else:
                calls.append((f"{s.name}.mrs", lambda: ops.conv2d_dense(
                    x, p.aug, pl.kh, pl.kw, s.n, pl.stride, pl.pad, p.bias, pl.pool, out=acc)))
            return calls
        if ((li > 0 and (self.plans[li - 1].fuse_next or self.plans[li - 1].fuse_next2 or
                         self.plans[li - 1].fuse_next3)) or
                (li > 1 and self.plans[li - 2].fuse_next2)):
            return []                                   # run by an earlier layer's call
        if pl.in_lists:
            idx, lval, cnt = B.lists[li - 1]
        else:
            idx, lval, cnt = B.idx[li], B.lval[li], B.cnt[li]
            calls.append((f"{s.name}.compact", lambda: ops.compact_into(
                x.reshape(b * h * w, c), idx, lval, cnt)))
        if pl.fuse_next2:
            # one call: this layer with its k-WTA and lists, the next layer over
            # them with its k-WTA, and the last layer on its winners
            q, r = self.packed[li + 1], self.packed[li + 2]
            sq = q.spec
            calls.append((f"{s.name}.mrs_kwta+{sq.name}.mrs_kwta+{r.spec.name}.mrs",
                          lambda: ops.mrs_kwta_chain3(
                idx, lval, cnt, pl.geo, p.aug, pl.kh, pl.kw, s.n, pl.stride, pl.pad, p.bias,
                pl.pool, k=s.k, shift=shift, aug2=q.aug, n2=sq.n, bias2=q.bias, k2=sq.k,
                shift2=sq.shift, aug3=r.aug, n3=r.spec.n, bias3=r.bias,
                keep_sums=self.keep_sums, y=acc4, lists=lists_out,
                y2=B.acc[li + 1].reshape(b, -1), lists2=B.lists[li + 1], y3=B.acc[li + 2])))
        elif pl.fuse_next:
            # one call: this layer with its k-WTA, then the last layer on its winners
            q = self.packed[li + 1]
            acc2 = B.acc[li + 1]
            calls.append((f"{s.name}.mrs_kwta+{q.spec.name}.mrs", lambda: ops.mrs_kwta_chain2(
                idx, lval, cnt, pl.geo, p.aug, pl.kh, pl.kw, s.n, pl.stride, pl.pad, p.bias,
                pl.pool, k=s.k, shift=shift, aug2=q.aug, n2=q.spec.n, bias2=q.bias, y=acc4,
                keep_sums=self.keep_sums, lists=lists_out, y2=acc2)))
        elif s.k is not None:
            # one call: sums, pool, k-WTA, requantisation, lists or dense output
            calls.append((f"{s.name}.mrs_kwta", lambda: ops.mrs_kwta_conv2d(
                idx, lval, cnt, pl.geo, p.aug, pl.kh, pl.kw, s.n, pl.stride, pl.pad, p.bias,
                pl.pool, k=s.k, out_dtype=odt, shift=shift, y=acc4, keep_sums=self.keep_sums,
                lists=lists_out, out=out)))
        else:
            calls.append((f"{s.name}.mrs", lambda: ops.mrs_conv2d(
                idx, lval, cnt, pl.geo, p.aug, pl.kh, pl.kw, s.n, pl.stride, pl.pad, p.bias,
                pl.pool, out=acc4)))
        return calls

    def forward_layer(self, li: int, x, bufs: Buffers | None = None, timer=None):
        """x: the dense input tensor (first layer) or None (lists of layer li-1)."""
        B = self.bufs if bufs is None else bufs
        t = timer or _NoTimer()
        for name, call in self.launches(li, x, B):
            t.start(name)
            call()
            t.stop(name)
        return B.out[li]

    def forward(self, x: torch.Tensor, bufs: Buffers | None = None, timer=None):
        if tuple(x.shape) != tuple(self.in_shapes[0]):
            raise ValueError(f"input shape {tuple(x.shape)} != planned {self.in_shapes[0]}")
        out = None
        for li in range(len(self.packed)):
            out = self.forward_layer(li, x if li == 0 else None, bufs, timer)
        return out

    def capture(self, x: torch.Tensor, bufs: Buffers | None = None) -> torch.cuda.CUDAGraph:
        """Record one forward pass over x into a HIP graph: replaying it runs
        every layer's kernels on the same buffers with no per-launch host
        work (no library call inside allocates, synchronises or clears memory
        with a memset node)."""
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            self.forward(x, bufs)
        return g

    def dense_output(self, li: int, bufs: Buffers | None = None) -> torch.Tensor:
        """Layer li's k-WTA output as a dense tensor (scattered back from its
        lists when the layer emits lists).  For checks, not the timed path."""
        B = self.bufs if bufs is None else bufs
        if B.lists[li] is None:
            return B.out[li]
        idx, val, cnt = B.lists[li]
        pl = self.plans[li]
        rows, cap = idx.shape
        dense = torch.zeros((rows, pl.out_shape[-1]), dtype=val.dtype, device=val.device)
        pos = torch.arange(cap, device=val.device)[None, :]
        keep = pos < cnt[:, None].to(torch.int64)
        r = torch.arange(rows, device=val.device)[:, None].expand(rows, cap)
        ii = idx.to(torch.int64) & 0xFFFF
        dense[r[keep], ii[keep]] = val[keep]
        return dense.reshape(pl.out_shape)

    def kernel_names(self) -> list:
        return [name for li in range(len(self.packed)) for name, _ in self.launches(li, None)]


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
