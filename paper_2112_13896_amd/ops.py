"""Torch-facing wrappers of the C ABI (argument marshalling only).

Every step of the layer runs in the HIP kernels of libcs.so; these functions
check tensor placement/dtype/shape, allocate outputs with torch and pass raw
device pointers plus torch's current HIP stream.  They never compute on the
host and have no fallback.
"""
from __future__ import annotations

import ctypes

import numpy as np
import torch

from . import _lib
from ._lib import CS_F32, CS_I8, CS_I32, check, lib

_TORCH_DT = {torch.int8: CS_I8, torch.int32: CS_I32, torch.float32: CS_F32}
_NP_DT = {np.dtype(np.int8): CS_I8, np.dtype(np.float32): CS_F32}


def _dt(t: torch.Tensor) -> int:
    try:
        return _TORCH_DT[t.dtype]
    except KeyError:
        raise TypeError(f"unsupported dtype {t.dtype}") from None


def _dev(t: torch.Tensor, name: str) -> int:
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _opt(t: torch.Tensor | None, name: str):
    return None if t is None else _dev(t, name)


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


# ------------------------------------------------------------------ pack (host)
def pack(W: np.ndarray, n: int):
    """Combine on the host: W [d_out][r] (int8 or float32) -> (aug, holes).

    aug is the augmented packed tensor [r][G] (G = d_out / n): for int8
    weights a uint16 array, entry = uint8(value) | kid << 8; for float32
    weights a uint32 array [r][G][2] holding (value bits, kid).  Raises
    CSError(CS_ERR_COLLISION) with .bad = (g, i) when two kernels of a set
    share a slot."""
    W = np.ascontiguousarray(W)
    if W.ndim != 2:
        raise ValueError("W must be [d_out][r]")
    d_out, r = W.shape
    wt = _NP_DT.get(W.dtype)
    if wt is None:
        raise TypeError(f"unsupported weight dtype {W.dtype}")
    G = d_out // n if n > 0 else 0
    if wt == CS_I8:
        aug = np.zeros((r, max(G, 1)), dtype=np.uint16)
    else:
        aug = np.zeros((r, max(G, 1), 2), dtype=np.uint32)
    holes = ctypes.c_int64(0)
    bg, bi = ctypes.c_int(0), ctypes.c_int(0)
    st = lib().cs_pack(wt, W.ctypes.data, d_out, r, n, aug.ctypes.data,
                       ctypes.byref(holes), ctypes.byref(bg), ctypes.byref(bi))
    if st != _lib.CS_OK:
        err = _lib.CSError("cs_pack", st)
        err.bad = (bg.value, bi.value)
        raise err
    return aug, int(holes.value)


def unpack_aug(aug: np.ndarray):
    """Split a host augmented tensor into (values [r][G], kernel IDs [r][G])."""
    if aug.dtype == np.uint16:
        return (aug & 0xFF).astype(np.uint8).view(np.int8), (aug >> 8).astype(np.int64)
    if aug.dtype == np.uint32 and aug.ndim == 3 and aug.shape[2] == 2:
        return aug[..., 0].copy().view(np.float32), aug[..., 1].astype(np.int64)
    raise TypeError("not an augmented tensor")


def aug_to_device(aug: np.ndarray, device="cuda") -> torch.Tensor:
    """Upload an augmented tensor: int16 [r][G] (int8 weights) or int32
    [r][G][2] (float32 weights), bit patterns unchanged."""
    if aug.dtype == np.uint16:
        return torch.from_numpy(aug.view(np.int16)).to(device)
    if aug.dtype == np.uint32:
        return torch.from_numpy(aug.view(np.int32)).to(device)
    raise TypeError("not an augmented tensor")


def _aug(aug: torch.Tensor, xdt: torch.dtype, n: int):
    """Device pointer and c_out of an augmented tensor that matches activations of dtype xdt."""
    ok = (xdt == torch.int8 and aug.dtype == torch.int16 and aug.dim() == 2) or \
         (xdt == torch.float32 and aug.dtype == torch.int32 and aug.dim() == 3 and
          aug.shape[2] == 2)
    if not ok:
        raise TypeError(f"augmented tensor {aug.dtype}{tuple(aug.shape)} does not match {xdt}")
    return _dev(aug, "aug"), aug.shape[1] * n


# ------------------------------------------------------------------ device ops
def compact(x: torch.Tensor):
    """x [rows][c] (int8/float32) -> (idx uint16-as-int16 [rows][c], val, cnt int32).
    Only idx[r, :cnt[r]] and val[r, :cnt[r]] are defined."""
    if x.dim() != 2:
        raise ValueError("x must be [rows][c]")
    rows, c = x.shape
    idx = torch.empty((rows, c), dtype=torch.int16, device=x.device)
    val = torch.empty_like(x)
    cnt = torch.empty((rows,), dtype=torch.int32, device=x.device)
    check("cs_compact", lib().cs_compact(_dt(x), _dev(x, "x"), rows, c, _dev(idx, "idx"),
                                         _dev(val, "val"), _dev(cnt, "cnt"), _stream()))
    return idx, val, cnt


def compact_into(x: torch.Tensor, idx: torch.Tensor, val: torch.Tensor, cnt: torch.Tensor) -> None:
    """cs_compact into caller-provided buffers (idx int16 [rows][c], val like x, cnt int32)."""
    rows, c = x.shape
    if idx.shape != (rows, c) or val.shape != (rows, c) or cnt.shape != (rows,):
        raise ValueError("buffer shapes do not match x")
    if idx.dtype != torch.int16 or val.dtype != x.dtype or cnt.dtype != torch.int32:
        raise TypeError("buffer dtypes do not match")
    check("cs_compact", lib().cs_compact(_dt(x), _dev(x, "x"), rows, c, _dev(idx, "idx"),
                                         _dev(val, "val"), _dev(cnt, "cnt"), _stream()))


def conv_out(h: int, k: int, stride: int, pad: int) -> int:
    return (h + 2 * pad - k) // stride + 1


def mrs_conv2d(idx: torch.Tensor, lval: torch.Tensor, cnt: torch.Tensor, in_shape, aug,
               kh: int, kw: int, n: int, stride: int = 1, pad: int = 0, bias=None, pool: int = 1,
               out: torch.Tensor | None = None) -> torch.Tensor:
    """Multiply/route/sum on compacted lists of the b*h*w input pixels."""
    b, h, w, c_in = in_shape
    pa, c_out = _aug(aug, lval.dtype, n)
    ho, wo = conv_out(h, kh, stride, pad), conv_out(w, kw, stride, pad)
    ydt = torch.int32 if lval.dtype == torch.int8 else torch.float32
    if out is None:
        out = torch.empty((b, ho // pool, wo // pool, c_out), dtype=ydt, device=lval.device)
    check("cs_mrs_conv2d", lib().cs_mrs_conv2d(
        _dt(lval), _dev(idx, "idx"), _dev(lval, "lval"), _dev(cnt, "cnt"), idx.shape[-1],
        b, h, w, c_in, kh, kw, stride, pad, pa, c_out, n,
        _opt(bias, "bias"), pool, _dev(out, "out"), _stream()))
    return out


def mrs_kwta_conv2d(idx: torch.Tensor, lval: torch.Tensor, cnt: torch.Tensor, in_shape, aug,
                    kh: int, kw: int, n: int, stride: int = 1, pad: int = 0, bias=None,
                    pool: int = 1, *, k: int, out_dtype: torch.dtype | None = None,
                    shift: int = 0, y: torch.Tensor | None = None, keep_sums: bool = True,
                    cap: int | None = None, lists=None, out: torch.Tensor | None = None):
    """One layer: multiply/route/sum (+ bias, pool) and k-WTA over each output
    pixel's channels.  Returns (y, result) where y holds the sums (when
    keep_sums) and result is the dense masked output, or the (idx, val, cnt)
    lists when `cap` or `lists` is given."""
    b, h, w, c_in = in_shape
    pa, c_out = _aug(aug, lval.dtype, n)
    ho, wo = conv_out(h, kh, stride, pad), conv_out(w, kw, stride, pad)
    acc_dt = torch.int32 if lval.dtype == torch.int8 else torch.float32
    odt = acc_dt if out_dtype is None else out_dtype
    oshape = (b, max(ho, 0) // pool, max(wo, 0) // pool, c_out)
    rows = oshape[0] * oshape[1] * oshape[2]
    if y is None:
        y = torch.empty(oshape, dtype=acc_dt, device=lval.device)
    if lists is None and cap is not None:
        lists = (torch.empty((rows, cap), dtype=torch.int16, device=lval.device),
                 torch.empty((rows, cap), dtype=odt, device=lval.device),
                 torch.empty((rows,), dtype=torch.int32, device=lval.device))
    if lists is not None:
        oi, ov, oc = lists
        if oi.dtype != torch.int16 or ov.dtype != odt or oc.dtype != torch.int32:
            raise TypeError("list buffer dtypes do not match")
        if oi.shape != ov.shape or oi.dim() != 2 or oi.shape[0] != rows or oc.shape != (rows,):
            raise ValueError("list buffer shapes do not match the output")
        args = (None, _dev(oi, "oidx"), _dev(ov, "oval"), _dev(oc, "ocnt"), oi.shape[1])
        result = lists
    else:
        if out is None:
            out = torch.empty(oshape, dtype=odt, device=lval.device)
        if out.dtype != odt or out.numel() != rows * c_out:
            raise ValueError("out does not match the output")
        args = (_dev(out, "out"), None, None, None, 0)
        result = out
    check("cs_mrs_kwta_conv2d", lib().cs_mrs_kwta_conv2d(
        _dt(lval), _dev(idx, "idx"), _dev(lval, "lval"), _dev(cnt, "cnt"), idx.shape[-1],
        b, h, w, c_in, kh, kw, stride, pad, pa, c_out, n, _opt(bias, "bias"), pool,
        _dev(y, "y"), 1 if keep_sums else 0, k, _TORCH_DT[odt], shift, *args, _stream()))
    return y, result


def mrs_kwta_units_conv2d(idx: torch.Tensor, lval: torch.Tensor, cnt: torch.Tensor, in_shape,
                          aug, kh: int, kw: int, n: int, stride: int = 1, pad: int = 0,
                          bias=None, pool: int = 1, *, k: int, unit: int,
                          y: torch.Tensor | None = None, keep_sums: bool = True,
                          cap: int | None = None, lists=None, out: torch.Tensor | None = None):
    """One fp32 layer with k-WTA in units (cs_mrs_kwta_units_conv2d): every
    `unit` consecutive channels of an output pixel keep their own k winners.
    Returns (y, result) as mrs_kwta_conv2d."""
    b, h, w, c_in = in_shape
    pa, c_out = _aug(aug, lval.dtype, n)
    ho, wo = conv_out(h, kh, stride, pad), conv_out(w, kw, stride, pad)
    acc_dt = torch.int32 if lval.dtype == torch.int8 else torch.float32
    oshape = (b, max(ho, 0) // pool, max(wo, 0) // pool, c_out)
    rows = oshape[0] * oshape[1] * oshape[2]
    if y is None:
        y = torch.empty(oshape, dtype=acc_dt, device=lval.device)
    if lists is None and cap is not None:
        lists = (torch.empty((rows, cap), dtype=torch.int16, device=lval.device),
                 torch.empty((rows, cap), dtype=acc_dt, device=lval.device),
                 torch.empty((rows,), dtype=torch.int32, device=lval.device))
    if lists is not None:
        oi, ov, oc = lists
        if oi.dtype != torch.int16 or ov.dtype != acc_dt or oc.dtype != torch.int32:
            raise TypeError("list buffer dtypes do not match")
        if oi.shape != ov.shape or oi.dim() != 2 or oi.shape[0] != rows or oc.shape != (rows,):
            raise ValueError("list buffer shapes do not match the output")
        args = (None, _dev(oi, "oidx"), _dev(ov, "oval"), _dev(oc, "ocnt"), oi.shape[1])
        result = lists
    else:
        if out is None:
            out = torch.empty(oshape, dtype=acc_dt, device=lval.device)
        if out.dtype != acc_dt or out.numel() != rows * c_out:
            raise ValueError("out does not match the output")
        args = (_dev(out, "out"), None, None, None, 0)
        result = out
    check("cs_mrs_kwta_units_conv2d", lib().cs_mrs_kwta_units_conv2d(
        _dt(lval), _dev(idx, "idx"), _dev(lval, "lval"), _dev(cnt, "cnt"), idx.shape[-1],
        b, h, w, c_in, kh, kw, stride, pad, pa, c_out, n, _opt(bias, "bias"), pool,
        _dev(y, "y"), 1 if keep_sums else 0, k, unit, *args, _stream()))
    return y, result


def mrs_kwta_chain2(idx: torch.Tensor, lval: torch.Tensor, cnt: torch.Tensor, in_shape, aug,
                    kh: int, kw: int, n: int, stride: int = 1, pad: int = 0, bias=None,
                    pool: int = 1, *, k: int, shift: int, aug2, n2: int, bias2=None,
                    y: torch.Tensor | None = None, keep_sums: bool = True, cap: int | None = None,
                    lists=None, y2: torch.Tensor | None = None):
    """An int8 layer with k-WTA (one output vector per sample) and the linear
    layer on its requantised winners (cs_mrs_kwta_chain2).  Returns
    (y, lists, y2): the first layer's sums (when keep_sums), its winners'
    lists and the second layer's int32 sums [b][c_out2]."""
    if lval.dtype != torch.int8:
        raise TypeError("mrs_kwta_chain2 takes int8 lists")
    b, h, w, c_in = in_shape
    pa, c_out = _aug(aug, lval.dtype, n)
    pa2, c_out2 = _aug(aug2, torch.int8, n2)
    ho, wo = conv_out(h, kh, stride, pad), conv_out(w, kw, stride, pad)
    oshape = (b, max(ho, 0) // pool, max(wo, 0) // pool, c_out)
    rows = oshape[0] * oshape[1] * oshape[2]
    if y is None:
        y = torch.empty(oshape, dtype=torch.int32, device=lval.device)
    if lists is None:
        cap = list_capacity(k) if cap is None else cap
        lists = (torch.empty((rows, cap), dtype=torch.int16, device=lval.device),
                 torch.empty((rows, cap), dtype=torch.int8, device=lval.device),
                 torch.empty((rows,), dtype=torch.int32, device=lval.device))
    oi, ov, oc = lists
    if oi.dtype != torch.int16 or ov.dtype != torch.int8 or oc.dtype != torch.int32:
        raise TypeError("list buffer dtypes do not match")
    if oi.shape != ov.shape or oi.dim() != 2 or oi.shape[0] != rows or oc.shape != (rows,):
        raise ValueError("list buffer shapes do not match the output")
    if y2 is None:
        y2 = torch.empty((b, c_out2), dtype=torch.int32, device=lval.device)
    if y2.dtype != torch.int32 or y2.numel() != b * c_out2:
        raise ValueError("y2 does not match the second layer's output")
    check("cs_mrs_kwta_chain2", lib().cs_mrs_kwta_chain2(
        CS_I8, _dev(idx, "idx"), _dev(lval, "lval"), _dev(cnt, "cnt"), idx.shape[-1],
        b, h, w, c_in, kh, kw, stride, pad, pa, c_out, n, _opt(bias, "bias"), pool,
        _dev(y, "y"), 1 if keep_sums else 0, k, CS_I8, shift, _dev(oi, "oidx"), _dev(ov, "oval"),
        _dev(oc, "ocnt"), oi.shape[1], pa2, c_out2, n2, _opt(bias2, "bias2"), _dev(y2, "y2"),
        _stream()))
    return y, lists, y2


def _list_buffers(rows: int, cap: int, device, lists=None):
    if lists is None:
        lists = (torch.empty((rows, cap), dtype=torch.int16, device=device),
                 torch.empty((rows, cap), dtype=torch.int8, device=device),
                 torch.empty((rows,), dtype=torch.int32, device=device))
    oi, ov, oc = lists
    if oi.dtype != torch.int16 or ov.dtype != torch.int8 or oc.dtype != torch.int32:
        raise TypeError("list buffer dtypes do not match")
    if oi.shape != ov.shape or oi.dim() != 2 or oi.shape[0] != rows or oc.shape != (rows,):
        raise ValueError("list buffer shapes do not match the output")
    return lists


def mrs_kwta_chain3(idx: torch.Tensor, lval: torch.Tensor, cnt: torch.Tensor, in_shape, aug,
                    kh: int, kw: int, n: int, stride: int = 1, pad: int = 0, bias=None,
                    pool: int = 1, *, k: int, shift: int, aug2, n2: int, bias2=None, k2: int,
                    shift2: int, aug3, n3: int, bias3=None, keep_sums: bool = True,
                    y: torch.Tensor | None = None, cap: int | None = None, lists=None,
                    y2: torch.Tensor | None = None, cap2: int | None = None, lists2=None,
                    y3: torch.Tensor | None = None):
    """An int8 conv layer with k-WTA and lists, a layer with k-WTA over its
    whole pooled map, and a linear layer on the second one's winners
    (cs_mrs_kwta_chain3).  aug2 packs [c_out2][hp*wp*c_out] weights in the
    (y, x, channel) slot order of the first layer's NHWC output.  Returns
    (y, lists, y2, lists2, y3)."""
    if lval.dtype != torch.int8:
        raise TypeError("mrs_kwta_chain3 takes int8 lists")
    b, h, w, c_in = in_shape
    pa, c_out = _aug(aug, lval.dtype, n)
    pa2, c_out2 = _aug(aug2, torch.int8, n2)
    pa3, c_out3 = _aug(aug3, torch.int8, n3)
    ho, wo = conv_out(h, kh, stride, pad), conv_out(w, kw, stride, pad)
    oshape = (b, max(ho, 0) // pool, max(wo, 0) // pool, c_out)
    rows = oshape[0] * oshape[1] * oshape[2]
    dev = lval.device
    if y is None:
        y = torch.empty(oshape, dtype=torch.int32, device=dev)
    lists = _list_buffers(rows, list_capacity(k) if cap is None else cap, dev, lists)
    if y2 is None:
        y2 = torch.empty((b, c_out2), dtype=torch.int32, device=dev)
    lists2 = _list_buffers(b, list_capacity(k2) if cap2 is None else cap2, dev, lists2)
    if y3 is None:
        y3 = torch.empty((b, c_out3), dtype=torch.int32, device=dev)
    for t, nm, m in ((y2, "y2", c_out2), (y3, "y3", c_out3)):
        if t.dtype != torch.int32 or t.numel() != b * m:
            raise ValueError(f"{nm} does not match its layer's output")
    oi, ov, oc = lists
    oi2, ov2, oc2 = lists2
    check("cs_mrs_kwta_chain3", lib().cs_mrs_kwta_chain3(
        CS_I8, _dev(idx, "idx"), _dev(lval, "lval"), _dev(cnt, "cnt"), idx.shape[-1],
        b, h, w, c_in, kh, kw, stride, pad, pa, c_out, n, _opt(bias, "bias"), pool,
        _dev(y, "y"), 1 if keep_sums else 0, k, CS_I8, shift, _dev(oi, "oidx"), _dev(ov, "oval"),
        _dev(oc, "ocnt"), oi.shape[1], pa2, c_out2, n2, _opt(bias2, "bias2"), _dev(y2, "y2"),
        k2, shift2, _dev(oi2, "oidx2"), _dev(ov2, "oval2"), _dev(oc2, "ocnt2"), oi2.shape[1],
        pa3, c_out3, n3, _opt(bias3, "bias3"), _dev(y3, "y3"), _stream()))
    return y, lists, y2, lists2, y3


def conv2d_dense_kwta_chain3(x: torch.Tensor, aug, kh: int, kw: int, n: int, stride: int = 1,
                             pad: int = 0, bias=None, pool: int = 1, *, k: int, shift: int,
                             aug2, kh2: int, kw2: int, n2: int, stride2: int = 1, pad2: int = 0,
                             bias2=None, pool2: int = 1, k2: int, shift2: int, aug3, n3: int,
                             bias3=None, k3: int, shift3: int, aug4, n4: int, bias4=None,
                             keep_sums: bool = True, y=None, lists=None, y2=None, lists2=None,
                             y3=None, lists3=None, y4=None):
    """The dense-input int8 first layer with k-WTA lists, then the three layers
    of mrs_kwta_chain3 on them (cs_conv2d_dense_kwta_chain3).  Returns
    (y, lists, y2, lists2, y3, lists3, y4)."""
    if x.dim() != 4 or x.dtype != torch.int8:
        raise ValueError("x must be int8 NHWC")
    b, h, w, c_in = x.shape
    dev = x.device
    pa, c_out = _aug(aug, torch.int8, n)
    pa2, c_out2 = _aug(aug2, torch.int8, n2)
    pa3, c_out3 = _aug(aug3, torch.int8, n3)
    pa4, c_out4 = _aug(aug4, torch.int8, n4)
    ho, wo = conv_out(h, kh, stride, pad), conv_out(w, kw, stride, pad)
    s1 = (b, max(ho, 0) // pool, max(wo, 0) // pool, c_out)
    ho2, wo2 = conv_out(s1[1], kh2, stride2, pad2), conv_out(s1[2], kw2, stride2, pad2)
    s2 = (b, max(ho2, 0) // pool2, max(wo2, 0) // pool2, c_out2)
    r1, r2 = s1[0] * s1[1] * s1[2], s2[0] * s2[1] * s2[2]
    y = torch.empty(s1, dtype=torch.int32, device=dev) if y is None else y
    y2 = torch.empty(s2, dtype=torch.int32, device=dev) if y2 is None else y2
    y3 = torch.empty((b, c_out3), dtype=torch.int32, device=dev) if y3 is None else y3
    y4 = torch.empty((b, c_out4), dtype=torch.int32, device=dev) if y4 is None else y4
    for t, nm, m in ((y, "y", r1 * c_out), (y2, "y2", r2 * c_out2), (y3, "y3", b * c_out3),
                     (y4, "y4", b * c_out4)):
        if t.dtype != torch.int32 or t.numel() != m:
            raise ValueError(f"{nm} does not match its layer's output")
    lists = _list_buffers(r1, list_capacity(k), dev, lists)
    lists2 = _list_buffers(r2, list_capacity(k2), dev, lists2)
    lists3 = _list_buffers(b, list_capacity(k3), dev, lists3)
    (oi, ov, oc), (oi2, ov2, oc2), (oi3, ov3, oc3) = lists, lists2, lists3
    check("cs_conv2d_dense_kwta_chain3", lib().cs_conv2d_dense_kwta_chain3(
        CS_I8, _dev(x, "x"), b, h, w, c_in, kh, kw, stride, pad, pa, c_out, n, _opt(bias, "bias"),
        pool, _dev(y, "y"), 1 if keep_sums else 0, k, CS_I8, shift, _dev(oi, "oidx"),
        _dev(ov, "oval"), _dev(oc, "ocnt"), oi.shape[1],
        kh2, kw2, stride2, pad2, pa2, c_out2, n2, _opt(bias2, "bias2"), pool2, _dev(y2, "y2"),
        k2, shift2, _dev(oi2, "oidx2"), _dev(ov2, "oval2"), _dev(oc2, "ocnt2"), oi2.shape[1],
        pa3, c_out3, n3, _opt(bias3, "bias3"), _dev(y3, "y3"), k3, shift3, _dev(oi3, "oidx3"),
        _dev(ov3, "oval3"), _dev(oc3, "ocnt3"), oi3.shape[1],
        pa4, c_out4, n4, _opt(bias4, "bias4"), _dev(y4, "y4"), _stream()))
    return y, lists, y2, lists2, y3, lists3, y4


def mrs_plan(dtype: torch.dtype, cap: int, in_shape, kh: int, kw: int, stride: int, pad: int,
             c_out: int, n: int, pool: int = 1, k: int = -1) -> dict:
    """The launch plan the library picks for a layer (host only)."""
    b, h, w, c_in = in_shape
    info = (ctypes.c_int64 * 11)()
    check("cs_mrs_plan", lib().cs_mrs_plan(_TORCH_DT[dtype], cap, b, h, w, c_in, kh, kw, stride,
                                           pad, c_out, n, pool, k, info))
    path = ("simple", "tiled", "fused", "sample", "scatter", "rows", "blocks")[info[0]]
    kwta = None if k < 0 else ("separate" if info[10] else "fused")
    if path == "blocks":
        return {"path": path, "kwta": kwta, "select": info[1], "rows_per_block": info[2],
                "table_blocks": info[3], "blocks": info[6], "lds": info[7],
                "sets_per_lane": info[8]}
    if path == "rows":
        return {"path": path, "kwta": kwta, "blocks": info[6], "lds": info[7],
                "channels_per_lane": info[8]}
    if path == "scatter":
        return {"path": path, "kwta": kwta, "band_rows": info[2], "blocks": info[6],
                "lds": info[7], "sets_per_lane": info[8]}
    if path == "sample":
        return {"path": path, "kwta": kwta, "blocks": info[6], "lds": info[7],
                "slices": info[8]}
    if path != "fused":
        return {"path": path, "kwta": kwta}
    return {"path": path, "tile_mode": info[1], "tile": info[2], "tile_cols": info[3],
            "list_cap": info[4], "npix_cap": info[5], "blocks": info[6], "lds": info[7],
            "log2_slices": info[8], "select": info[9], "kwta": kwta}


def workspace_bytes(op: int, dtype: torch.dtype, rows: int, c_in: int) -> int:
    return int(lib().cs_workspace_bytes(op, _TORCH_DT[dtype], rows, c_in))


def workspace(op: int, dtype: torch.dtype, rows: int, c_in: int, device) -> torch.Tensor:
    nbytes = workspace_bytes(op, dtype, rows, c_in)
    if nbytes == 0:
        raise ValueError("invalid workspace request")
    return torch.empty((nbytes,), dtype=torch.uint8, device=device)


def conv2d_noalloc(x: torch.Tensor, aug: torch.Tensor, kh: int, kw: int, n: int,
                   stride: int = 1, pad: int = 0, bias: torch.Tensor | None = None,
                   pool: int = 1, out: torch.Tensor | None = None) -> torch.Tensor:
    """conv2d without a workspace argument: the library's own scratch holds the
    compaction lists (cs_conv2d_noalloc; nothing is allocated when `out` is
    given).  Calls that overlap on one GPU race on that scratch."""
    if x.dim() != 4:
        raise ValueError("x must be NHWC")
    b, h, w, c_in = x.shape
    pa, c_out = _aug(aug, x.dtype, n)
    ho, wo = conv_out(h, kh, stride, pad), conv_out(w, kw, stride, pad)
    ydt = torch.int32 if x.dtype == torch.int8 else torch.float32
    if out is None:
        out = torch.empty((b, max(ho, 0) // pool, max(wo, 0) // pool, c_out), dtype=ydt,
                          device=x.device)
    check("cs_conv2d_noalloc", lib().cs_conv2d_noalloc(
        _dt(x), _dev(x, "x"), b, h, w, c_in, kh, kw, stride, pad, pa, c_out, n,
        _opt(bias, "bias"), pool, _dev(out, "out"), _stream()))
    return out


def conv2d(x: torch.Tensor, aug: torch.Tensor, kh: int, kw: int, n: int,
           stride: int = 1, pad: int = 0, bias: torch.Tensor | None = None, pool: int = 1,
           ws: torch.Tensor | None = None, out: torch.Tensor | None = None) -> torch.Tensor:
    """Sparse-sparse conv of NHWC x with packed OHWI kernels (aug [kh*kw*c_in][G])."""
    if x.dim() != 4:
        raise ValueError("x must be NHWC")
    b, h, w, c_in = x.shape
    pa, c_out = _aug(aug, x.dtype, n)
    ho, wo = conv_out(h, kh, stride, pad), conv_out(w, kw, stride, pad)
    ydt = torch.int32 if x.dtype == torch.int8 else torch.float32
    if out is None:
        out = torch.empty((b, max(ho, 0) // pool, max(wo, 0) // pool, c_out), dtype=ydt,
                          device=x.device)
    if ws is None:
        ws = workspace(1, x.dtype, b * h * w, c_in, x.device)
    check("cs_conv2d", lib().cs_conv2d(
        _dt(x), _dev(x, "x"), b, h, w, c_in, kh, kw, stride, pad, pa, c_out, n,
        _opt(bias, "bias"), pool, _dev(out, "out"), _dev(ws, "ws"), ws.numel(), _stream()))
    return out


def conv2d_dense_blocks(x: torch.Tensor, aug: torch.Tensor, kidb: torch.Tensor, kh: int,
                        kw: int, n: int, stride: int = 1, pad: int = 0,
                        bias: torch.Tensor | None = None,
                        out: torch.Tensor | None = None) -> torch.Tensor:
    """Sparse-dense int8 conv with block CS, a block being one pixel's c_in <= 4
    channels (cs_conv2d_dense_blocks); aug and kidb as ops.pack_blocks gives
    them with b = c_in (on the device)."""
    if x.dim() != 4 or x.dtype != torch.int8:
        raise ValueError("x must be int8 NHWC")
    b, h, w, c_in = x.shape
    pa, c_out = _aug(aug, x.dtype, n)
    if kidb.dtype != torch.uint8 or tuple(kidb.shape) != (kh * kw, c_out // n):
        raise ValueError("kidb must be uint8 [kh*kw][c_out/n]")
    ho, wo = conv_out(h, kh, stride, pad), conv_out(w, kw, stride, pad)
    if out is None:
        out = torch.empty((b, max(ho, 0), max(wo, 0), c_out), dtype=torch.int32,
                          device=x.device)
    check("cs_conv2d_dense_blocks", lib().cs_conv2d_dense_blocks(
        _dev(x, "x"), b, h, w, c_in, kh, kw, stride, pad, pa, _dev(kidb, "kidb"), c_out, n,
        _opt(bias, "bias"), _dev(out, "out"), _stream()))
    return out


def conv2d_dense(x: torch.Tensor, aug: torch.Tensor, kh: int, kw: int, n: int,
                 stride: int = 1, pad: int = 0, bias: torch.Tensor | None = None, pool: int = 1,
                 out: torch.Tensor | None = None) -> torch.Tensor:
    """Sparse-dense conv (dense NHWC input, no compaction); see cs_conv2d_dense for the
    supported shapes."""
    if x.dim() != 4:
        raise ValueError("x must be NHWC")
    b, h, w, c_in = x.shape
    pa, c_out = _aug(aug, x.dtype, n)
    ho, wo = conv_out(h, kh, stride, pad), conv_out(w, kw, stride, pad)
    ydt = torch.int32 if x.dtype == torch.int8 else torch.float32
    if out is None:
        out = torch.empty((b, max(ho, 0) // pool, max(wo, 0) // pool, c_out), dtype=ydt,
                          device=x.device)
    check("cs_conv2d_dense", lib().cs_conv2d_dense(
        _dt(x), _dev(x, "x"), b, h, w, c_in, kh, kw, stride, pad, pa, c_out, n,
        _opt(bias, "bias"), pool, _dev(out, "out"), _stream()))
    return out


def conv2d_dense_kwta(x: torch.Tensor, aug: torch.Tensor, kh: int, kw: int, n: int,
                      stride: int = 1, pad: int = 0, bias: torch.Tensor | None = None,
                      pool: int = 1, *, k: int, out_dtype: torch.dtype | None = None,
                      shift: int = 0, y: torch.Tensor | None = None, keep_sums: bool = True,
                      cap: int | None = None, lists=None, out: torch.Tensor | None = None):
    """The dense-input first layer with k-WTA (cs_conv2d_dense_kwta).  Returns
    (y, result) as mrs_kwta_conv2d does."""
    if x.dim() != 4:
        raise ValueError("x must be NHWC")
    b, h, w, c_in = x.shape
    pa, c_out = _aug(aug, x.dtype, n)
    ho, wo = conv_out(h, kh, stride, pad), conv_out(w, kw, stride, pad)
    acc_dt = torch.int32 if x.dtype == torch.int8 else torch.float32
    odt = acc_dt if out_dtype is None else out_dtype
    oshape = (b, max(ho, 0) // pool, max(wo, 0) // pool, c_out)
    rows = oshape[0] * oshape[1] * oshape[2]
    if y is None:
        y = torch.empty(oshape, dtype=acc_dt, device=x.device)
    if lists is None and cap is not None:
        lists = (torch.empty((rows, cap), dtype=torch.int16, device=x.device),
                 torch.empty((rows, cap), dtype=odt, device=x.device),
                 torch.empty((rows,), dtype=torch.int32, device=x.device))
    if lists is not None:
        oi, ov, oc = lists
        if oi.dtype != torch.int16 or ov.dtype != odt or oc.dtype != torch.int32:
            raise TypeError("list buffer dtypes do not match")
        if oi.shape != ov.shape or oi.dim() != 2 or oi.shape[0] != rows or oc.shape != (rows,):
            raise ValueError("list buffer shapes do not match the output")
        args = (None, _dev(oi, "oidx"), _dev(ov, "oval"), _dev(oc, "ocnt"), oi.shape[1])
        result = lists
    else:
        if out is None:
            out = torch.empty(oshape, dtype=odt, device=x.device)
        if out.dtype != odt or out.numel() != rows * c_out:
            raise ValueError("out does not match the output")
        args = (_dev(out, "out"), None, None, None, 0)
        result = out
    check("cs_conv2d_dense_kwta", lib().cs_conv2d_dense_kwta(
        _dt(x), _dev(x, "x"), b, h, w, c_in, kh, kw, stride, pad, pa, c_out, n,
        _opt(bias, "bias"), pool, _dev(y, "y"), 1 if keep_sums else 0, k, _TORCH_DT[odt], shift,
        *args, _stream()))
    return y, result


def reorder_table(aug: np.ndarray, kh: int, kw: int, c_in: int, c_out: int, n: int) -> np.ndarray:
    """cs_reorder_table: the fp32 packed kernel (host, from pack) in Kernel-ID
    order, int32 [c_out][smax][2] (tile byte offset, value bits), smax the
    longest support rounded up to a multiple of 8."""
    if not (aug.dtype == np.uint32 and aug.ndim == 3 and aug.shape[2] == 2):
        raise TypeError("reorder_table takes an fp32 packed kernel (uint32 [r][G][2])")
    aug = np.ascontiguousarray(aug)
    smax = ctypes.c_int(0)
    check("cs_reorder_table", lib().cs_reorder_table(aug.ctypes.data, kh, kw, c_in, c_out, n,
                                                     ctypes.byref(smax), None))
    smax.value = (smax.value + 7) // 8 * 8           # the kernel reads 8 entries at a time
    table = np.zeros((c_out, smax.value, 2), dtype=np.int32)
    check("cs_reorder_table", lib().cs_reorder_table(aug.ctypes.data, kh, kw, c_in, c_out, n,
                                                     ctypes.byref(smax), table.ctypes.data))
    return table


def pack_blocks(W: np.ndarray, n: int, b: int):
    """Combine with blocks of b slots on the host (cs_pack_blocks): W [d_out][r]
    int8/float32 -> (aug as pack gives it, kidb uint8 [r/b][G], holes).
    Raises CSError with .bad = (kernel or set, block) when a support splits a
    block (CS_ERR_SHAPE) or two kernels of a set share one (CS_ERR_COLLISION)."""
    W = np.ascontiguousarray(W)
    if W.ndim != 2:
        raise ValueError("W must be [d_out][r]")
    d_out, r = W.shape
    wt = _NP_DT.get(W.dtype)
    if wt is None:
        raise TypeError(f"unsupported weight dtype {W.dtype}")
    G = d_out // n if n > 0 else 0
    aug = (np.zeros((r, max(G, 1)), dtype=np.uint16) if wt == CS_I8
           else np.zeros((r, max(G, 1), 2), dtype=np.uint32))
    kidb = np.zeros((max(r // b, 1) if b > 0 else 1, max(G, 1)), dtype=np.uint8)
    holes = ctypes.c_int64(0)
    bg, bi = ctypes.c_int(0), ctypes.c_int(0)
    st = lib().cs_pack_blocks(wt, W.ctypes.data, d_out, r, n, b, aug.ctypes.data,
                              kidb.ctypes.data, ctypes.byref(holes), ctypes.byref(bg),
                              ctypes.byref(bi))
    if st != _lib.CS_OK:
        err = _lib.CSError("cs_pack_blocks", st)
        err.bad = (bg.value, bi.value)
        raise err
    return aug, kidb, int(holes.value)


def pack_channels(W4: np.ndarray, n: int):
    """Combine along the channel dimension on the host (cs_pack_channels):
    W4 [c_out][kh][kw][c_in] fp32 -> (packed uint32 [c_out][c_in/n][kh][kw][2]
    holding (value bits, channel ID), holes); int8 -> packed uint16
    [c_out][c_in/n][kh][kw] (value byte | channel ID << 8).  Raises CSError
    (CS_ERR_COLLISION) with .bad = (o, slot) on a collision."""
    i8 = np.asarray(W4).dtype == np.int8
    W4 = np.ascontiguousarray(W4, dtype=np.int8 if i8 else np.float32)
    if W4.ndim != 4:
        raise ValueError("W4 must be [c_out][kh][kw][c_in]")
    c_out, kh, kw, c_in = W4.shape
    q = c_in // n if n > 0 else 0
    if i8:
        packed = np.zeros((c_out, max(q, 1), kh, kw), dtype=np.uint16)
    else:
        packed = np.zeros((c_out, max(q, 1), kh, kw, 2), dtype=np.uint32)
    holes = ctypes.c_int64(0)
    bo, bi = ctypes.c_int(0), ctypes.c_int(0)
    st = lib().cs_pack_channels(CS_I8 if i8 else CS_F32, W4.ctypes.data, c_out, kh, kw, c_in, n,
                                packed.ctypes.data, ctypes.byref(holes), ctypes.byref(bo),
                                ctypes.byref(bi))
    if st != _lib.CS_OK:
        err = _lib.CSError("cs_pack_channels", st)
        err.bad = (bo.value, bi.value)
        raise err
    return packed, int(holes.value)


def channel_table(packed: np.ndarray, kh: int, kw: int, c_in: int, c_out: int, n: int,
                  stride: int = 1) -> np.ndarray:
    """cs_channel_table: an int8 channel-overlaid layer's table for
    conv2d_channels at this stride, int32 [c_out][5 * ceil((c_in/n)*kh*kw / 4)]."""
    packed = np.ascontiguousarray(packed, dtype=np.uint16)
    s4 = ((c_in // n) * kh * kw + 3) // 4
    table = np.zeros((c_out, 5 * s4), dtype=np.int32)
    check("cs_channel_table", lib().cs_channel_table(packed.ctypes.data, kh, kw, c_in, c_out, n,
                                                      stride, table.ctypes.data))
    return table


def conv2d_channels(x: torch.Tensor, table: torch.Tensor, kh: int, kw: int, c_out: int, n: int,
                    stride: int = 1, pad: int = 0, bias: torch.Tensor | None = None,
                    out: torch.Tensor | None = None) -> torch.Tensor:
    """int8 dense-input conv with the channel-dimension overlay (cs_conv2d_channels);
    table: device copy of channel_table(...) for this stride."""
    if x.dim() != 4 or x.dtype != torch.int8:
        raise ValueError("x must be int8 NHWC")
    b, h, w, c_in = x.shape
    ho, wo = conv_out(h, kh, stride, pad), conv_out(w, kw, stride, pad)
    if out is None:
        out = torch.empty((b, max(ho, 0), max(wo, 0), c_out), dtype=torch.int32, device=x.device)
    check("cs_conv2d_channels", lib().cs_conv2d_channels(
        _dev(x, "x"), b, h, w, c_in, kh, kw, stride, pad, _dev(table, "table"), c_out, n,
        _opt(bias, "bias"), _dev(out, "out"), _stream()))
    return out


def reorder_table_channels(packed: np.ndarray, kh: int, kw: int, c_in: int, c_out: int,
                           n: int) -> np.ndarray:
    """cs_reorder_table_channels: a channel-overlaid layer's table for
    conv2d_reorder_kwta, int32 [c_out][smax][2] (smax a multiple of 8)."""
    packed = np.ascontiguousarray(packed)
    smax = ctypes.c_int(0)
    check("cs_reorder_table_channels", lib().cs_reorder_table_channels(
        packed.ctypes.data, kh, kw, c_in, c_out, n, ctypes.byref(smax), None))
    smax.value = (smax.value + 7) // 8 * 8
    table = np.zeros((c_out, smax.value, 2), dtype=np.int32)
    check("cs_reorder_table_channels", lib().cs_reorder_table_channels(
        packed.ctypes.data, kh, kw, c_in, c_out, n, ctypes.byref(smax), table.ctypes.data))
    return table


def conv2d_reorder_kwta(x: torch.Tensor, table: torch.Tensor, kh: int, kw: int, pad: int = 0,
                        bias: torch.Tensor | None = None, *, k: int,
                        y: torch.Tensor | None = None, keep_sums: bool = True,
                        cap: int | None = None, lists=None, out: torch.Tensor | None = None):
    """A dense-input fp32 conv layer by reordering (cs_conv2d_reorder_kwta);
    table is reorder_table's result on the device.  Returns (y, result) as
    mrs_kwta_conv2d does."""
    if x.dim() != 4:
        raise ValueError("x must be NHWC")
    if table.dim() != 3 or table.dtype != torch.int32 or table.shape[2] != 2:
        raise ValueError("table must be int32 [c_out][smax][2]")
    b, h, w, c_in = x.shape
    c_out, smax = table.shape[0], table.shape[1]
    ho, wo = conv_out(h, kh, 1, pad), conv_out(w, kw, 1, pad)
    oshape = (b, max(ho, 0), max(wo, 0), c_out)
    rows = oshape[0] * oshape[1] * oshape[2]
    if y is None:
        y = torch.empty(oshape, dtype=torch.float32, device=x.device)
    if lists is None and cap is not None:
        lists = (torch.empty((rows, cap), dtype=torch.int16, device=x.device),
                 torch.empty((rows, cap), dtype=torch.float32, device=x.device),
                 torch.empty((rows,), dtype=torch.int32, device=x.device))
    if lists is not None:
        oi, ov, oc = lists
        if oi.dtype != torch.int16 or ov.dtype != torch.float32 or oc.dtype != torch.int32:
            raise TypeError("list buffer dtypes do not match")
        if oi.shape != ov.shape or oi.dim() != 2 or oi.shape[0] != rows or oc.shape != (rows,):
            raise ValueError("list buffer shapes do not match the output")
        args = (None, _dev(oi, "oidx"), _dev(ov, "oval"), _dev(oc, "ocnt"), oi.shape[1])
        result = lists
    else:
        if out is None:
            out = torch.empty(oshape, dtype=torch.float32, device=x.device)
        if out.dtype != torch.float32 or out.numel() != rows * c_out:
            raise ValueError("out does not match the output")
        args = (_dev(out, "out"), None, None, None, 0)
        result = out
    check("cs_conv2d_reorder_kwta", lib().cs_conv2d_reorder_kwta(
        _dt(x), _dev(x, "x"), b, h, w, c_in, kh, kw, pad, _dev(table, "table"), smax, c_out,
        _opt(bias, "bias"), _dev(y, "y"), 1 if keep_sums else 0, k, CS_F32, *args, _stream()))
    return y, result


def linear(x: torch.Tensor, aug: torch.Tensor, n: int,
           bias: torch.Tensor | None = None, ws: torch.Tensor | None = None,
           out: torch.Tensor | None = None) -> torch.Tensor:
    """Sparse-sparse linear layer: x [batch][d_in], packed aug [d_in][G]."""
    if x.dim() != 2:
        raise ValueError("x must be [batch][d_in]")
    batch, d_in = x.shape
    pa, d_out = _aug(aug, x.dtype, n)
    ydt = torch.int32 if x.dtype == torch.int8 else torch.float32
    if out is None:
        out = torch.empty((batch, d_out), dtype=ydt, device=x.device)
    if ws is None:
        ws = workspace(0, x.dtype, batch, d_in, x.device)
    check("cs_linear", lib().cs_linear(
        _dt(x), _dev(x, "x"), batch, d_in, pa, d_out, n,
        _opt(bias, "bias"), _dev(out, "out"), _dev(ws, "ws"), ws.numel(), _stream()))
    return out


def kwta(x: torch.Tensor, k: int, out_dtype: torch.dtype | None = None, shift: int = 0,
         out: torch.Tensor | None = None) -> torch.Tensor:
    """k-WTA along the last axis.  out_dtype=torch.int8 on int32 input
    requantises the winners with `shift`."""
    c = x.shape[-1]
    rows = x.numel() // c if c else 0
    odt = x.dtype if out_dtype is None else out_dtype
    if out is None:
        out = torch.empty(x.shape, dtype=odt, device=x.device)
    check("cs_kwta", lib().cs_kwta(_dt(x), _dev(x, "x"), rows, c, k, _TORCH_DT[odt], shift,
                                   _dev(out, "out"), _stream()))
    return out


def list_capacity(k: int) -> int:
    """Row stride for k-entry lists: k rounded up to a multiple of 4 (vector reads)."""
    return max(4, (k + 3) // 4 * 4)


def kwta_lists(x: torch.Tensor, k: int, out_dtype: torch.dtype | None = None, shift: int = 0,
               cap: int | None = None, out=None):
    """k-WTA along the last axis, winners emitted as (idx, val, cnt) lists of
    capacity `cap` (default: list_capacity(k)).  Rows are all leading axes."""
    c = x.shape[-1]
    rows = x.numel() // c if c else 0
    odt = x.dtype if out_dtype is None else out_dtype
    cap = list_capacity(k) if cap is None else cap
    if out is None:
        idx = torch.empty((rows, cap), dtype=torch.int16, device=x.device)
        val = torch.empty((rows, cap), dtype=odt, device=x.device)
        cnt = torch.empty((rows,), dtype=torch.int32, device=x.device)
    else:
        idx, val, cnt = out
    check("cs_kwta_lists", lib().cs_kwta_lists(
        _dt(x), _dev(x, "x"), rows, c, k, _TORCH_DT[odt], shift, _dev(idx, "idx"),
        _dev(val, "val"), _dev(cnt, "cnt"), cap, _stream()))
    return idx, val, cnt
