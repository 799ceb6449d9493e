"""GPU parity of each kernel against the CPU oracle, through the C ABI.

Small and odd sizes that span several wavefronts/blocks and end in ragged
tails; empty rows, fully dense rows, heavy ties, +-0, n = 1 .. 32, pad,
stride, pool, bias / no bias.  Integer results are bit-exact; fp32 results
are within 1e-5 * sum|products| per output.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import cs_oracle as o
from paper_2112_13896_amd import ops
from tests.gpu_util import assert_f32_close, dev, host, pool_S
from workloads import complementary_weights, sparse_rows

pytestmark = pytest.mark.gpu


def rng(seed):
    return np.random.default_rng(seed)


def random_rows(r, rows, c, density, dtype):
    if dtype == "i8":
        v = r.integers(-127, 128, size=(rows, c)).astype(np.int8)
    else:
        v = r.normal(size=(rows, c)).astype(np.float32)
    mask = r.random((rows, c)) < density
    v = np.where(mask, v, np.zeros_like(v))
    if rows > 2:
        v[0] = 0                           # an empty row
        v[1] = np.where(v[1] == 0, 1, v[1]) if dtype == "i8" else np.where(v[1] == 0, 1.5, v[1])
    if dtype == "f32":
        z = (v == 0) & (r.random((rows, c)) < 0.5)
        v[z] = -0.0                        # signed zeros are zeros
    return v


# ------------------------------------------------------------------ compaction
@pytest.mark.parametrize("dtype", ["i8", "f32"])
@pytest.mark.parametrize("c", [1, 2, 3, 7, 31, 33, 63, 64, 65, 96, 200, 1500, 1600])
def test_compact(dtype, c):
    r = rng(c)
    for rows, dens in [(1, 0.5), (5, 0.0), (130, 0.1), (1001, 0.7)]:
        x = random_rows(r, rows, c, dens, dtype)
        idx, val, cnt = ops.compact(dev(x))
        idx_h = host(idx).view(np.uint16)
        val_h, cnt_h = host(val), host(cnt)
        for ri, (ii, vv) in enumerate(o.compact_rows(x)):
            n = cnt_h[ri]
            assert n == len(ii), (ri, n, len(ii))
            assert np.array_equal(idx_h[ri, :n], ii)
            assert np.array_equal(val_h[ri, :n], vv)


@pytest.mark.parametrize("dtype", ["i8", "f32"])
@pytest.mark.parametrize("c", [4096, 65532, 65535])
def test_compact_widest_rows(dtype, c):
    """Rows up to the widest the 16-bit list indices allow (CS_MAX_ROW): the
    vector path (width a multiple of the vector) and the chunked one."""
    r = rng(c + 3)
    for rows, dens in [(1, 0.3), (3, 0.02), (9, 0.9)]:
        x = random_rows(r, rows, c, dens, dtype)
        idx, val, cnt = ops.compact(dev(x))
        idx_h = host(idx).view(np.uint16)
        val_h, cnt_h = host(val), host(cnt)
        for ri, (ii, vv) in enumerate(o.compact_rows(x)):
            n = cnt_h[ri]
            assert n == len(ii), (ri, n, len(ii))
            assert np.array_equal(idx_h[ri, :n], ii)
            assert np.array_equal(val_h[ri, :n], vv)


def test_compact_empty():
    x = torch.zeros((0, 64), dtype=torch.int8, device="cuda")
    idx, val, cnt = ops.compact(x)
    torch.cuda.synchronize()
    assert cnt.numel() == 0


# ------------------------------------------------------------------ k-WTA
def kwta_cases():
    for c, ks in [(1, [0, 1]), (5, [0, 2, 5]), (64, [1, 8, 16, 32, 33, 64]), (65, [1, 7, 65]),
                  (96, [12]), (256, [26, 255]), (576, [72]), (1500, [75, 225]), (2048, [1, 300])]:
        for k in ks:
            yield c, k


@pytest.mark.parametrize("dtype", ["i32", "f32"])
@pytest.mark.parametrize("c,k", list(kwta_cases()))
def test_kwta(dtype, c, k):
    r = rng(1000 + c * 7 + k)
    for rows in (1, 127, 129, 517):
        if dtype == "i32":
            spread = [3, 1000, 2 ** 30][rows % 3]
            v = r.integers(-spread, spread + 1, size=(rows, c)).astype(np.int32)
            if rows > 1:
                v[1] = 7                                     # all equal
        else:
            v = np.round(r.normal(size=(rows, c)), 1 if rows % 2 else 4).astype(np.float32)
            v[v == 0] = -0.0 if rows % 2 else 0.0
            if rows > 1:
                v[1] = np.where(np.arange(c) % 2, 0.0, -0.0)  # +-0 ties
        out = host(ops.kwta(dev(v), k))
        exp = o.kwta(v, k)
        assert np.array_equal(out, exp)
        assert (out != 0).sum() <= k * rows


@pytest.mark.parametrize("c,k", [(64, 8), (64, 16), (576, 72), (1500, 75), (7, 3)])
@pytest.mark.parametrize("shift", [0, 3, 9, 11, 31])
def test_kwta_requant(c, k, shift):
    r = rng(c + k + shift)
    v = r.integers(-400000, 400001, size=(333, c)).astype(np.int32)
    v[2] = -5
    out = host(ops.kwta(dev(v), k, torch.int8, shift))
    exp = o.requant(v, shift, o.kwta_winners(v, k))
    assert out.dtype == np.int8 and np.array_equal(out, exp)


@pytest.mark.parametrize("c,k", [(64, 8), (64, 16), (64, 32), (256, 26), (576, 72), (1500, 75), (7, 3), (1, 1), (2048, 300)])
@pytest.mark.parametrize("mode", ["i32", "i32->i8", "f32"])
def test_kwta_lists(c, k, mode):
    """k-WTA emitting (index, value) lists: exactly the non-zero entries of the
    dense k-WTA (or requantised) row, in index order."""
    r = rng(c * 3 + k + len(mode))
    rows = 301
    if mode == "f32":
        v = np.round(r.normal(size=(rows, c)), 2).astype(np.float32)
        v[:, ::5] = 0.0
    else:
        v = r.integers(-3000, 3001, size=(rows, c)).astype(np.int32)
        v[::7] = 5
    shift = 4 if mode == "i32->i8" else 0
    odt = torch.int8 if mode == "i32->i8" else None
    from paper_2112_13896_amd.ops import list_capacity
    cap = list_capacity(k) + (4 if c == 64 else 0)
    idx, val, cnt = (host(t) for t in ops.kwta_lists(dev(v), k, odt, shift, cap))
    win = o.kwta_winners(v, k)
    dense = o.requant(v, shift, win) if mode == "i32->i8" else np.where(win, v, np.zeros_like(v))
    for row in range(rows):
        nz = np.flatnonzero(dense[row])
        assert cnt[row] == len(nz) and cnt[row] <= k
        assert np.array_equal(idx[row, :cnt[row]].view(np.uint16), nz)
        assert np.array_equal(val[row, :cnt[row]], dense[row, nz])


# ------------------------------------------------------------------ linear
LINEAR_CASES = [
    # batch, d_in, d_out, n, nnz per row
    (16, 512, 64, 8, 64),
    (3, 40, 60, 20, 7),
    (67, 96, 576, 8, 12),
    (5, 1600, 1500, 20, 200),
    (2, 1500, 12, 1, 75),
    (9, 64, 64, 32, 64),       # dense input rows
    (4, 33, 6, 3, 0),          # all-zero input: output = bias
    (130, 256, 256, 16, 26),
    (2, 8192, 16, 2, 300),     # packed table too large for one workgroup's LDS
]


@pytest.mark.parametrize("case", LINEAR_CASES)
@pytest.mark.parametrize("dtype", ["i8", "f32"])
@pytest.mark.parametrize("with_bias", [True, False])
def test_linear(case, dtype, with_bias):
    batch, d_in, d_out, n, nnz = case
    r = rng(sum(case) + (dtype == "f32") * 7 + with_bias)
    if d_in % n:
        pytest.skip("n must divide d_in for the generator")
    W = complementary_weights(r, r, d_out, d_in, n, "int8" if dtype == "i8" else "normal")
    x = sparse_rows(r, batch, d_in, nnz if nnz < d_in else None,
                    "u_m127_127" if dtype == "i8" else "absnormal") if nnz else \
        np.zeros((batch, d_in), dtype=np.int8 if dtype == "i8" else np.float32)
    if dtype == "f32" and nnz:
        x = x * np.where(r.random(x.shape) < 0.5, -1, 1).astype(np.float32)
    b = None
    if with_bias:
        b = r.integers(-1000, 1001, size=d_out).astype(np.int32) if dtype == "i8" else \
            r.normal(size=d_out).astype(np.float32)
    aug, _ = ops.pack(W, n)
    y = host(ops.linear(dev(x), ops.aug_to_device(aug), n, None if b is None else dev(b)))
    ref = o.linear(x, W, b)
    if dtype == "i8":
        assert y.dtype == np.int32 and np.array_equal(y.astype(np.int64), ref)
    else:
        S = o.abs_sum_linear(x, W) + (0 if b is None else np.abs(b.astype(np.float64)))
        assert_f32_close(y, ref, S, f"linear {case}")


# ------------------------------------------------------------------ conv
CONV_CASES = [
    # b, h, w, c_in, c_out, n, kh, kw, stride, pad, pool, nnz per pixel
    (2, 9, 11, 64, 64, 8, 3, 3, 1, 1, 1, 7),
    (3, 14, 14, 96, 576, 8, 1, 1, 1, 0, 1, 12),
    (2, 14, 14, 64, 64, 16, 5, 5, 1, 0, 2, 8),
    (2, 32, 32, 1, 64, 1, 5, 5, 1, 0, 2, None),
    (1, 7, 5, 256, 256, 16, 3, 3, 1, 1, 1, 26),
    (2, 9, 9, 24, 12, 4, 3, 3, 2, 1, 1, 5),
    (1, 6, 8, 32, 32, 32, 1, 1, 1, 0, 2, 32),
    (3, 5, 5, 12, 8, 2, 2, 3, 1, 1, 1, 0),
]


@pytest.mark.parametrize("case", CONV_CASES)
@pytest.mark.parametrize("dtype", ["i8", "f32"])
def test_conv2d(case, dtype):
    b, h, w, c_in, c_out, n, kh, kw, stride, pad, pool, nnz = case
    r = rng(sum(x or 0 for x in case) + (dtype == "f32"))
    R = kh * kw * c_in
    W = complementary_weights(r, r, c_out, R, n, "int8" if dtype == "i8" else "normal")
    W = W.reshape(c_out, kh, kw, c_in)
    if nnz == 0:
        x = np.zeros((b, h, w, c_in), dtype=np.int8 if dtype == "i8" else np.float32)
    else:
        x = sparse_rows(r, b * h * w, c_in, nnz if (nnz or c_in) < c_in else None,
                        "u_m127_127" if dtype == "i8" else "absnormal").reshape(b, h, w, c_in)
    bias = (r.integers(-1000, 1001, size=c_out).astype(np.int32) if dtype == "i8"
            else r.normal(size=c_out).astype(np.float32)) if b % 2 else None
    aug, _ = ops.pack(W.reshape(c_out, -1), n)
    y = host(ops.conv2d(dev(x), ops.aug_to_device(aug), kh, kw, n, stride, pad,
                        None if bias is None else dev(bias), pool))
    ref = o.conv2d_nhwc(x, W, stride, pad, bias)
    if pool == 2:
        ref = o.maxpool2x2_nhwc(ref)
    assert y.shape == ref.shape
    if dtype == "i8":
        assert np.array_equal(y.astype(np.int64), ref)
    else:
        S = o.abs_sum_conv(x, W, stride, pad) + (0 if bias is None else np.abs(bias.astype(np.float64)))
        if pool == 2:
            S = pool_S(S)
        assert_f32_close(y, ref, S, f"conv {case}")


DENSE_CASES = [
    # b, h, w, c_in, kh, kw, stride, pad, pool
    (3, 32, 32, 1, 5, 5, 1, 0, 2),
    (2, 9, 11, 3, 3, 3, 1, 1, 1),
    (2, 12, 12, 2, 3, 3, 2, 1, 2),
    (1, 7, 6, 8, 2, 2, 1, 0, 1),
]


@pytest.mark.parametrize("case", DENSE_CASES)
@pytest.mark.parametrize("dtype", ["i8", "f32"])
def test_conv2d_dense(case, dtype):
    """Sparse-dense variant (dense input, dense kernels) against the oracle."""
    b, h, w, c_in, kh, kw, stride, pad, pool = case
    r = rng(sum(case) + (dtype == "f32"))
    R = kh * kw * c_in
    W = complementary_weights(r, r, 64, R, 1, "int8" if dtype == "i8" else "normal")
    W = W.reshape(64, kh, kw, c_in)
    x = sparse_rows(r, b * h * w, c_in, None,
                    "u_m127_127" if dtype == "i8" else "absnormal").reshape(b, h, w, c_in)
    bias = (r.integers(-1000, 1001, size=64).astype(np.int32) if dtype == "i8"
            else r.normal(size=64).astype(np.float32)) if b != 2 else None
    aug, _ = ops.pack(W.reshape(64, -1), 1)
    y = host(ops.conv2d_dense(dev(x), ops.aug_to_device(aug), kh, kw, 1, stride, pad,
                              None if bias is None else dev(bias), pool))
    ref = o.conv2d_nhwc(x, W, stride, pad, bias)
    if pool == 2:
        ref = o.maxpool2x2_nhwc(ref)
    assert y.shape == ref.shape
    if dtype == "i8":
        assert np.array_equal(y.astype(np.int64), ref)
    else:
        S = o.abs_sum_conv(x, W, stride, pad) + (0 if bias is None else np.abs(bias.astype(np.float64)))
        if pool == 2:
            S = pool_S(S)
        assert_f32_close(y, ref, S, f"dense conv {case}")


def test_mrs_on_compacted_lists_matches_conv2d():
    r = rng(5)
    W = complementary_weights(r, r, 64, 576, 8, "normal").reshape(64, 3, 3, 64)
    x = sparse_rows(r, 2 * 10 * 12, 64, 7, "absnormal").reshape(2, 10, 12, 64)
    aug, _ = ops.pack(W.reshape(64, -1), 8)
    xd, ad = dev(x), ops.aug_to_device(aug)
    y1 = ops.conv2d(xd, ad, 3, 3, 8, 1, 1)
    idx, lv, cnt = ops.compact(xd.reshape(-1, 64))
    y2 = ops.mrs_conv2d(idx, lv, cnt, x.shape, ad, 3, 3, 8, 1, 1)
    assert torch.equal(y1, y2)


@pytest.mark.parametrize("dtype", ["i8", "f32"])
def test_mrs_reads_kwta_lists(dtype):
    """A conv whose input is the previous k-WTA's capacity-k lists, and a
    linear layer over a whole conv map read as a window-sized conv."""
    r = rng(33 + (dtype == "f32"))
    b, h, w, c = 3, 6, 7, 64
    k = 9
    acc_prev = (r.integers(-500, 500, size=(b, h, w, c)).astype(np.int32) if dtype == "i8"
                else r.normal(size=(b, h, w, c)).astype(np.float32))
    shift = 2
    odt = torch.int8 if dtype == "i8" else None
    lists = ops.kwta_lists(dev(acc_prev), k, odt, shift if dtype == "i8" else 0)
    win = o.kwta_winners(acc_prev, k)
    x_ref = o.requant(acc_prev, shift, win) if dtype == "i8" else np.where(win, acc_prev, np.float32(0))
    wd = "int8" if dtype == "i8" else "normal"
    for (kh, kw, pad, n, c_out) in [(3, 3, 1, 8, 64), (h, w, 0, 16, 48)]:
        W = complementary_weights(r, r, c_out, kh * kw * c, n, wd).reshape(c_out, kh, kw, c)
        aug, _ = ops.pack(W.reshape(c_out, -1), n)
        y = host(ops.mrs_conv2d(*lists, (b, h, w, c), ops.aug_to_device(aug), kh, kw, n, 1, pad))
        ref = o.conv2d_nhwc(x_ref, W, 1, pad)
        if dtype == "i8":
            assert np.array_equal(y.astype(np.int64), ref)
        else:
            assert_f32_close(y, ref, o.abs_sum_conv(x_ref, W, 1, pad), "mrs on k-WTA lists")


def test_fp32_bitwise_reproducible():
    r = rng(6)
    W = complementary_weights(r, r, 256, 2304, 16, "normal").reshape(256, 3, 3, 256)
    x = sparse_rows(r, 2 * 14 * 14, 256, 26, "absnormal").reshape(2, 14, 14, 256)
    aug, _ = ops.pack(W.reshape(256, -1), 16)
    xd, ad = dev(x), ops.aug_to_device(aug)
    a = host(ops.conv2d(xd, ad, 3, 3, 16, 1, 1))
    b = host(ops.conv2d(xd, ad, 3, 3, 16, 1, 1))
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_kwta_in_units_of_64():
    """k-WTA in units of 64 channels (wide layers as [64:64] modules): cs_kwta
    on the [rows * c/64][64] view of a [rows][c] tensor keeps each unit's own
    k winners, as the oracle's unit k-WTA does; lists per unit likewise."""
    r = rng(4242)
    v = r.integers(-3000, 3000, size=(333, 256)).astype(np.int32)
    k = 6
    out = host(ops.kwta(dev(v).reshape(-1, 64), k)).reshape(333, 256)
    win = o.kwta_units_winners(v, k)
    assert np.array_equal(out, np.where(win, v, 0))
    idx, val, cnt = (host(t) for t in ops.kwta_lists(dev(v).reshape(-1, 64), k))
    units = np.where(win, v, 0).reshape(-1, 64)
    for ri in range(units.shape[0]):
        nz = np.flatnonzero(units[ri])
        assert cnt[ri] == len(nz)
        assert np.array_equal(idx[ri, :cnt[ri]].view(np.uint16), nz)

