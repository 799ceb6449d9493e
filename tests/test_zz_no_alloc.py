"""cs_conv2d_noalloc (the entry point for callers that cannot allocate: its
compaction lists live in the library's own device scratch) against cs_conv2d
with a caller workspace: the same kernels, so the same bits, on two calls in
a row, the second on a smaller input, plus the oracle on both."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import cs_oracle as o
from paper_2112_13896_amd import _lib, ops
from tests.gpu_util import assert_f32_close, dev, host
from workloads import complementary_weights

pytestmark = pytest.mark.gpu


def _case(seed, dtype, shape, nnz, kh, pad, c_out, n, pool, bias):
    r = np.random.default_rng(seed)
    b, h, w, c_in = shape
    rows = b * h * w
    x = np.zeros((rows, c_in), dtype=np.int8 if dtype == "i8" else np.float32)
    for i in range(rows):
        pos = r.choice(c_in, size=nnz, replace=False)
        x[i, pos] = (r.integers(1, 128, size=nnz) if dtype == "i8"
                     else np.abs(r.normal(size=nnz)).astype(np.float32))
    x = x.reshape(shape)
    W = complementary_weights(r, r, c_out, kh * kh * c_in, n,
                              "int8" if dtype == "i8" else "normal").reshape(c_out, kh, kh, c_in)
    bv = None
    if bias:
        bv = (r.integers(-1000, 1001, size=c_out).astype(np.int32) if dtype == "i8"
              else r.normal(size=c_out).astype(np.float32))
    return x, W, bv


CASES = [
    # a 3x3 fp32 layer (several tiles, ragged image), then a smaller int8 1x1 layer
    ("f32", (3, 23, 19, 64), 7, 3, 1, 64, 8, 1, False),
    ("i8", (2, 7, 9, 96), 12, 1, 0, 576, 8, 1, True),
    # and a larger one again after the small one, pooled
    ("i8", (2, 14, 14, 64), 8, 5, 0, 64, 16, 2, False),
]


def test_noalloc_matches_workspace_entry_point():
    torch.cuda.set_device(0)
    for ci, (dtype, shape, nnz, kh, pad, c_out, n, pool, bias) in enumerate(CASES):
        print(f"no_alloc case {ci}: {dtype} {shape} {kh}x{kh} pad {pad} -> {c_out} n={n}",
              flush=True)
        x, W, bv = _case(100 + ci, dtype, shape, nnz, kh, pad, c_out, n, pool, bias)
        aug = ops.aug_to_device(ops.pack(W.reshape(c_out, -1), n)[0])
        xd = dev(x)
        bd = dev(bv) if bv is not None else None
        want = ops.conv2d(xd, aug, kh, kh, n, 1, pad, bd, pool)
        got = ops.conv2d_noalloc(xd, aug, kh, kh, n, 1, pad, bd, pool)
        torch.cuda.synchronize()
        g, e = host(got), host(want)
        assert np.array_equal(g.view(np.uint8), e.view(np.uint8)), f"case {ci}: differs"
        ref = o.conv2d_nhwc(x, W, 1, pad, bv)
        if pool == 2:
            ref = o.maxpool2x2_nhwc(ref)
        if dtype == "i8":
            assert np.array_equal(g.astype(np.int64), ref), f"case {ci}: oracle"
        else:
            S = o.abs_sum_conv(x, W, 1, pad)
            assert_f32_close(g, ref, S, f"case {ci}: oracle")


def test_noalloc_rejects_inputs_beyond_the_scratch():
    """Lists larger than the scratch are refused before any launch."""
    rows = _lib.CS_NOALLOC_SCRATCH_BYTES // (64 * 6) + 1024
    need = ops.workspace_bytes(1, torch.float32, rows, 64)
    assert need > _lib.CS_NOALLOC_SCRATCH_BYTES
    x = torch.zeros((1, rows, 1, 64), dtype=torch.float32, device="cuda")
    W = complementary_weights(np.random.default_rng(1), np.random.default_rng(2), 64, 64, 8,
                              "normal")
    aug = ops.aug_to_device(ops.pack(W, 8)[0])
    with pytest.raises(_lib.CSError) as ei:
        ops.conv2d_noalloc(x, aug, 1, 1, 8)
    assert ei.value.status == _lib.CS_ERR_WORKSPACE
