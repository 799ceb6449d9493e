"""GPU parity of the reordering layer (cs_conv2d_reorder_kwta): every output
reads the dense activations at its kernel's support (cs_reorder_table) and
sums in a register; then k-WTA as the routed layer kernels.  Checked against
the oracle (dense convolution of the unpacked weights, full-sort k-WTA): fp32
sums within 1e-5 * sum|products|, the winners the exact top-k of the kernel's
own sums (differing from the oracle's only at near-ties), lists in channel
order holding exactly the non-zero winners; the same layer through the routed
path (compaction + cs_mrs_kwta_conv2d) gives the same winners."""
from __future__ import annotations

import zlib

import numpy as np
import pytest
import torch

from oracle import cs_oracle as o
from paper_2112_13896_amd import ops
from tests.gpu_util import assert_f32_close, check_kwta_f32, dev, host
from tests.test_gpu_fused import dense_from_lists, sparse_input, weights

pytestmark = pytest.mark.gpu

# (b, h, w, c_in), nnz, kh, kw, pad, n, k, bias, out
CASES = [
    ((2, 56, 56, 64), 7, 3, 3, 1, 8, 8, True, "lists"),      # config 3's layer, batch 2
    ((3, 13, 19, 64), 7, 3, 3, 1, 8, 8, False, "dense"),     # ragged tiles
    ((2, 16, 16, 30), 6, 3, 3, 1, 2, 16, True, "lists"),     # c_in not a multiple of 4
    ((2, 12, 12, 64), 10, 1, 1, 0, 16, 26, True, "lists"),   # 1x1, k in (16, 32]
    ((1, 10, 10, 16), 4, 5, 5, 2, 2, 0, False, "lists"),     # k = 0: empty lists
    ((1, 10, 10, 16), 4, 5, 5, 2, 2, 64, True, "dense"),     # k = c_out
    ((2, 9, 9, 64), 64, 3, 3, 0, 8, 32, True, "lists"),      # dense activations, no padding
]


@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}-{c[2]}x{c[3]}-n{c[5]}-k{c[6]}-{c[8]}"
                                             for c in CASES])
def test_reorder_layer(case):
    shape, nnz, kh, kw, pad, n, k, has_bias, mode = case
    r = np.random.default_rng(zlib.crc32(repr(case).encode()))
    b, h, w, c_in = shape
    c_out = 64
    x = sparse_input(r, shape, nnz, "f32")
    W = weights(r, c_out, kh, kw, c_in, n, "f32")
    bias = r.normal(size=c_out).astype(np.float32) if has_bias else None
    aug, _ = ops.pack(W.reshape(c_out, -1), n)
    table = dev(ops.reorder_table(aug, kh, kw, c_in, c_out, n))
    xd, bd = dev(x), None if bias is None else dev(bias)
    cap = ops.list_capacity(k) if mode == "lists" else None
    y, res = ops.conv2d_reorder_kwta(xd, table, kh, kw, pad, bd, k=k, cap=cap)
    y2, res2 = ops.conv2d_reorder_kwta(xd, table, kh, kw, pad, bd, k=k, cap=cap, keep_sums=False)
    y = host(y)
    if mode == "lists":
        res, res2 = tuple(host(t) for t in res), tuple(host(t) for t in res2)
        assert np.array_equal(res[2], res2[2])
        out = dense_from_lists(*res, c_out)
        assert np.array_equal(out, dense_from_lists(*res2, c_out))
    else:
        out, out2 = host(res).reshape(-1, c_out), host(res2).reshape(-1, c_out)
        assert np.array_equal(out, out2)
    ref = o.conv2d_nhwc(x, W, 1, pad, bias)
    S = o.abs_sum_conv(x, W, 1, pad)
    if bias is not None:
        S = S + np.abs(bias.astype(np.float64))
    assert y.shape == ref.shape
    assert_f32_close(y, ref, S, "reorder sums")
    near = check_kwta_f32(y, out, ref, S, k)
    assert near <= max(1, out.shape[0] // 100)
    if mode == "lists":
        assert np.array_equal(res[2], (out != 0).sum(axis=1))
        assert (res[2] <= k).all()


def test_reorder_matches_routed_path():
    """The same layer routed (compaction + cs_mrs_kwta_conv2d) and reordered:
    equal winners wherever the two sums' k-th and (k+1)-th values are apart."""
    r = np.random.default_rng(77)
    shape, kh, n, k = (2, 20, 20, 64), 3, 8, 8
    x = sparse_input(r, shape, 7, "f32")
    W = weights(r, 64, kh, kh, 64, n, "f32")
    aug, _ = ops.pack(W.reshape(64, -1), n)
    xd = dev(x)
    yr, lr = ops.conv2d_reorder_kwta(xd, dev(ops.reorder_table(aug, kh, kh, 64, 64, n)), kh, kh, 1,
                                     None, k=k, cap=8)
    idx, lv, cnt = ops.compact(xd.reshape(-1, 64))
    ym, lm = ops.mrs_kwta_conv2d(idx, lv, cnt, shape, ops.aug_to_device(aug), kh, kh, n, 1, 1,
                                 None, 1, k=k, cap=8)
    a = dense_from_lists(*(host(t) for t in lr), 64)
    m = dense_from_lists(*(host(t) for t in lm), 64)
    ys = np.sort(host(ym).reshape(-1, 64), axis=1)
    gap = ys[:, 64 - k] - ys[:, 63 - k]
    clear = gap > 1e-4 * (np.abs(ys).max(axis=1) + 1)
    assert clear.mean() > 0.95
    assert np.array_equal(a[clear] != 0, m[clear] != 0)
    np.testing.assert_allclose(a[clear], m[clear], rtol=1e-5, atol=1e-5)


def test_reorder_rejects():
    r = np.random.default_rng(3)
    W = weights(r, 64, 3, 3, 64, 8, "f32")
    aug, _ = ops.pack(W.reshape(64, -1), 8)
    t = dev(ops.reorder_table(aug, 3, 3, 64, 64, 8))
    x = dev(np.zeros((1, 8, 8, 64), np.float32))
    with pytest.raises(ops._lib.CSError):
        ops.conv2d_reorder_kwta(x, t, 3, 3, 1, None, k=40, cap=40)     # 32 < k < c_out
    with pytest.raises(ops._lib.CSError):
        ops.conv2d_reorder_kwta(x, t, 3, 3, 1, None, k=8, cap=6)      # cap not a multiple of 4


@pytest.mark.parametrize("shape,kh,pad,n,k", [((2, 20, 20, 48), 3, 1, 3, 8),
                                              ((1, 12, 13, 40), 5, 2, 5, 16)])
def test_channel_overlay_layer(shape, kh, pad, n, k):
    """Complementary Sparsity in the channel dimension (cs_pack_channels): the
    layer runs by reordering (cs_reorder_table_channels + the reordering
    kernel) and matches the oracle's convolution of the dense filters."""
    from workloads import channel_complementary_weights
    r = np.random.default_rng(zlib.crc32(repr((shape, kh, n)).encode()))
    c_in = shape[3]
    x = sparse_input(r, shape, c_in // 6, "f32")
    W4 = channel_complementary_weights(r, r, 64, kh, kh, c_in, n)
    bias = r.normal(size=64).astype(np.float32)
    packed, holes = ops.pack_channels(W4, n)
    assert holes == 0
    table = dev(ops.reorder_table_channels(packed, kh, kh, c_in, 64, n))
    y, lists = ops.conv2d_reorder_kwta(dev(x), table, kh, kh, pad, dev(bias), k=k,
                                       cap=ops.list_capacity(k))
    y = host(y)
    out = dense_from_lists(*(host(t) for t in lists), 64)
    ref = o.conv2d_nhwc(x, W4, 1, pad, bias)
    S = o.abs_sum_conv(x, W4, 1, pad) + np.abs(bias.astype(np.float64))
    assert_f32_close(y, ref, S, "channel-overlay sums")
    near = check_kwta_f32(y, out, ref, S, k)
    assert near <= max(1, out.shape[0] // 100)


def test_block_cs_stem_layer():
    """Block Complementary Sparsity on a 7 x 7 stem over RGB input (the 3
    values of a pixel form one block, Section 5): cs_pack_blocks, then the
    layer routed (dense input compacted, stride 2) and reordered (stride 1),
    both against the oracle's convolution of the dense filters."""
    from workloads import block_complementary_weights
    r = np.random.default_rng(91)
    b, h, w, c, n, kh = 2, 32, 32, 3, 4, 7
    x = np.abs(r.normal(size=(b, h, w, c))).astype(np.float32)      # dense image
    W = block_complementary_weights(r, r, 64, kh * kh * c, n, 3).reshape(64, kh, kh, c)
    aug, kidb, holes = ops.pack_blocks(W.reshape(64, -1), n, 3)
    assert holes == 0 and kidb.shape == (kh * kh, 64 // n)
    y = host(ops.conv2d(dev(x), ops.aug_to_device(aug), kh, kh, n, 2, 3))
    ref = o.conv2d_nhwc(x, W, 2, 3, None)
    assert_f32_close(y, ref, o.abs_sum_conv(x, W, 2, 3), "block-CS stem, routed")
    table = dev(ops.reorder_table(aug, kh, kh, c, 64, n))
    y1, out1 = ops.conv2d_reorder_kwta(dev(x), table, kh, kh, 3, None, k=64)
    ref1 = o.conv2d_nhwc(x, W, 1, 3, None)
    S1 = o.abs_sum_conv(x, W, 1, 3)
    assert_f32_close(host(y1), ref1, S1, "block-CS stem, reordered")
    assert np.array_equal(host(out1), host(y1))                      # k = c_out: all win
