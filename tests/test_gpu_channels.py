"""GPU parity of the int8 layer with Complementary Sparsity overlaid in the
channel dimension (cs_conv2d_channels; Section 3.1).

Each filter's channel groups hold complementary kh x kw slices; the layer is
packed with cs_pack_channels (int8) and cs_channel_table, and its int32 sums
must equal the oracle's dense convolution of the unpacked filters bit for bit:
stride 1 and 2, padding, rows wider than one 64-pixel tile, every supported
filter count, a bias.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import cs_oracle as o
from paper_2112_13896_amd import ops
from tests.gpu_util import dev, host
from workloads import channel_complementary_weights

pytestmark = pytest.mark.gpu


def int8_channel_weights(r, c_out, kh, kw, c, n):
    mask = channel_complementary_weights(r, r, c_out, kh, kw, c, n) != 0
    vals = r.integers(1, 128, size=mask.shape) * r.choice([-1, 1], size=mask.shape)
    return np.where(mask, vals, 0).astype(np.int8)


# (b, h, w, c_in), kh, stride, pad, c_out, n, bias
CASES = [
    ((2, 10, 12, 12), 3, 1, 1, 16, 3, False),
    ((2, 9, 9, 24), 3, 2, 1, 32, 3, True),
    ((1, 8, 70, 8), 1, 1, 0, 16, 1, False),      # 70 columns: two tiles per row, the second ragged
    ((2, 7, 7, 48), 3, 1, 1, 64, 3, True),
    ((1, 6, 131, 36), 3, 1, 0, 128, 9, True),    # n = 9: every tap of a 3x3 slice a different channel
]


@pytest.mark.parametrize("case", CASES, ids=[str(i) for i in range(len(CASES))])
def test_channels_match_oracle(case):
    shape, kh, stride, pad, c_out, n, has_bias = case
    r = np.random.default_rng(31 + sum(shape) + c_out)
    x = r.integers(-127, 128, size=shape).astype(np.int8)
    W4 = int8_channel_weights(r, c_out, kh, kh, shape[3], n)
    bias = r.integers(-5000, 5001, size=c_out).astype(np.int32) if has_bias else None
    packed, holes = ops.pack_channels(W4, n)
    assert holes == 0
    table = dev(ops.channel_table(packed, kh, kh, shape[3], c_out, n, stride))
    y = host(ops.conv2d_channels(dev(x), table, kh, kh, c_out, n, stride, pad,
                                 None if bias is None else dev(bias)))
    ref = o.conv2d_nhwc(x, W4, stride, pad, bias)
    assert np.array_equal(y.astype(np.int64), ref)
