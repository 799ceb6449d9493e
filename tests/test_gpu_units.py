"""GPU parity of the k-WTA in units (cs_mrs_kwta_units_conv2d; Section 5:
channels partitioned into modules of 64, each with its own k-WTA).

Each case runs the fp32 layer through the C ABI and checks it against the
oracle: the sums within 1e-5 * sum|products| of the dense convolution, and in
every unit the winners are the exact top-k of the kernel's own sums (ties to
the lower index), differing from the oracle's `kwta_units_winners` only at
near-ties.  Lists hold every unit's winners of a pixel in ascending channel
order.  The launch path is asserted: one kernel (the table-block kernel with
the selection on the lanes' own accumulators) where it applies, else the sums
and a k-WTA on the unit view.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import cs_oracle as o
from paper_2112_13896_amd import _lib, ops
from tests.gpu_util import assert_f32_close, check_kwta_f32, dev, host
from tests.test_gpu_fused import dense_from_lists, sparse_input, weights

pytestmark = pytest.mark.gpu

# (b, h, w, c_in), nnz, kh, kw, pad, c_out, n, k, unit, out, fused
CASES = [
    # the ResNet-50 stage-3 3x3 shape with 64-channel modules: one kernel, lists
    ((2, 7, 7, 256), 26, 3, 3, 1, 256, 16, 7, 64, "lists", True),
    ((2, 7, 7, 256), 26, 3, 3, 1, 256, 16, 7, 64, "dense", True),
    # units of 32 on a 1x1 layer (the table streamed in channel blocks), ragged tiles
    ((2, 9, 5, 1024), 102, 1, 1, 0, 256, 16, 3, 32, "lists", True),
    # 128 channels, 8 per set: units of 64 = four lanes of sixteen channels
    ((3, 6, 6, 64), 7, 3, 3, 1, 128, 8, 5, 64, "dense", True),
    # k = 0, k = unit, one lane per unit
    ((2, 5, 6, 64), 7, 3, 3, 1, 64, 8, 0, 16, "lists", True),
    ((2, 5, 6, 64), 7, 3, 3, 1, 64, 8, 16, 16, "dense", True),
    # 48 outputs (sets not a power of two): two kernels, dense output
    ((2, 6, 7, 32), 5, 3, 3, 1, 48, 8, 4, 16, "dense", False),
]


@pytest.mark.parametrize("case", CASES, ids=[str(i) for i in range(len(CASES))])
def test_units_match_oracle(case):
    shape, nnz, kh, kw, pad, c_out, n, k, unit, outk, fused = case
    r = np.random.default_rng(2112 + len(str(case)))
    x = sparse_input(r, shape, nnz, "f32")
    W = weights(r, c_out, kh, kw, shape[3], n, "f32")
    bias = r.normal(size=c_out).astype(np.float32)
    b, h, w, c_in = shape
    rows_in = b * h * w
    idx, val, cnt = ops.compact(dev(x.reshape(rows_in, c_in)))
    aug = ops.aug_to_device(ops.pack(W.reshape(c_out, -1), n)[0])
    ref = o.conv2d_nhwc(x, W, 1, pad, bias)
    # the bias is one more term of every sum (the tolerance scale counts it)
    S = o.abs_sum_conv(x, W, 1, pad) + np.abs(bias.astype(np.float64))
    ho, wo = ref.shape[1], ref.shape[2]
    rows = b * ho * wo
    cap = ops.list_capacity(k * (c_out // unit)) if outk == "lists" else None
    got = {}
    for keep in (True, False):
        y, res = ops.mrs_kwta_units_conv2d(idx, val, cnt, shape, aug, kh, kw, n, 1, pad,
                                           dev(bias), 1, k=k, unit=unit, keep_sums=keep, cap=cap)
        torch.cuda.synchronize()
        if outk == "lists":
            gi, gv, gc = (host(t) for t in res)
            got[keep] = dense_from_lists(gi, gv, gc, c_out)
        else:
            got[keep] = host(res).reshape(rows, c_out)
        if keep:
            acc = host(y).reshape(rows, c_out)
    assert np.array_equal(got[True].view(np.uint32), got[False].view(np.uint32))
    assert_f32_close(acc, ref.reshape(rows, c_out), S.reshape(rows, c_out), "sums")
    # per unit: the exact top-k of the kernel's own sums; near-ties only against the oracle
    outd = got[True]
    if outk == "lists":
        # a list leaves out winners whose value is exactly 0: restore them from the sums
        win = o.kwta_units_winners(acc, k, unit)
        assert np.array_equal(outd != 0, win & (acc != 0))
        outd = np.where(win, acc, np.float32(0))
    check_kwta_f32(acc.reshape(-1, unit), outd.reshape(-1, unit), ref.reshape(-1, unit),
                   S.reshape(-1, unit), k)
    # the launch path: lists are only written by the one-kernel path, so a
    # list call that succeeds shows it applies (the dense fallback cannot)
    ocap = ops.list_capacity(k * (c_out // unit))
    if fused:
        ops.mrs_kwta_units_conv2d(idx, val, cnt, shape, aug, kh, kw, n, 1, pad, dev(bias), 1,
                                  k=k, unit=unit, keep_sums=False, cap=ocap)
    else:
        with pytest.raises(_lib.CSError):
            ops.mrs_kwta_units_conv2d(idx, val, cnt, shape, aug, kh, kw, n, 1, pad, dev(bias),
                                      1, k=k, unit=unit, keep_sums=False, cap=ocap)
    torch.cuda.synchronize()


def test_unit_equal_to_row_is_the_plain_layer():
    shape, nnz, c_out, n, k = (2, 6, 6, 64), 7, 64, 8, 8
    r = np.random.default_rng(5)
    x = sparse_input(r, shape, nnz, "f32")
    W = weights(r, c_out, 3, 3, shape[3], n, "f32")
    idx, val, cnt = ops.compact(dev(x.reshape(-1, shape[3])))
    aug = ops.aug_to_device(ops.pack(W.reshape(c_out, -1), n)[0])
    _, a = ops.mrs_kwta_units_conv2d(idx, val, cnt, shape, aug, 3, 3, n, 1, 1, None, 1, k=k,
                                     unit=c_out)
    _, p = ops.mrs_kwta_conv2d(idx, val, cnt, shape, aug, 3, 3, n, 1, 1, None, 1, k=k)
    assert np.array_equal(host(a).view(np.uint32), host(p).view(np.uint32))
