"""GPU parity of the one-kernel layer (cs_mrs_kwta_conv2d): multiply, route,
sum, bias, 2x2 max-pool, k-WTA, requantisation, list or dense output.

Every case is checked against the oracle (dense convolution of the unpacked
weights, full-sort k-WTA): int8 bit for bit (sums, winners, requantised
values, list order and counts); fp32 sums within 1e-5 * sum|products| and the
winners as the exact top-k of the kernel's own sums, differing from the
oracle's only at near-ties.  Each case runs twice, keeping the sums (checked)
and not keeping them (the benchmark's setting), and both outputs must be
identical.  The launch plan is asserted so that every tiling path (rows of
items, full-width image rows, column tiles, partial LDS staging with global
reads, one workgroup per sample for linear layers, input-stationary int8
convolutions, one wavefront per item for 1x1 layers, the two-kernel fallback)
is known to run.
"""
from __future__ import annotations

import zlib

import numpy as np
import pytest
import torch

from oracle import cs_oracle as o
from oracle import networks
from paper_2112_13896_amd import ops
from tests.gpu_util import assert_f32_close, check_kwta_f32, dev, host, pool_S
from workloads import LayerSpec, complementary_weights

pytestmark = pytest.mark.gpu


def sparse_input(r, shape, nnz, dtype, low_range=False):
    """NHWC input with exactly `nnz` non-zero channels per pixel."""
    b, h, w, c = shape
    rows = b * h * w
    x = np.zeros((rows, c), dtype=np.int8 if dtype == "i8" else np.float32)
    for i in range(rows):
        pos = r.choice(c, size=min(nnz, c), replace=False)
        if dtype == "i8":
            x[i, pos] = 1 if low_range else r.integers(1, 128, size=len(pos))
        else:
            x[i, pos] = np.abs(r.normal(size=len(pos))).astype(np.float32)
    if rows > 3:
        x[2] = 0                                   # an empty pixel
    return x.reshape(shape)


def weights(r, c_out, kh, kw, c_in, n, dtype, low_range=False):
    W = complementary_weights(r, r, c_out, kh * kw * c_in, n,
                              "int8" if dtype == "i8" else "normal")
    if low_range and dtype == "i8":
        W = np.sign(W).astype(np.int8)             # +-1: many equal sums (ties)
    return W.reshape(c_out, kh, kw, c_in)


def dense_from_lists(idx, val, cnt, c):
    rows, cap = idx.shape
    out = np.zeros((rows, c), dtype=val.dtype)
    for row in range(rows):
        m = cnt[row]
        ii = idx[row, :m].view(np.uint16).astype(np.int64)
        assert (np.diff(ii) > 0).all(), f"row {row}: list indices not ascending"
        out[row, ii] = val[row, :m]
    return out


def check_chain_against_oracle(layers, x, Ws, bs, sums, lists):
    """Every layer of a fused int8 chain against networks.run_chain (the
    oracle's dense layers in Table 1's order): the sums after pool bit for bit,
    and each k-WTA layer's list (counts, ascending indices, requantised values)
    equal to the oracle's requantised winners with zero values left out.
    `sums[l]` is the GPU's sums tensor of layer l, `lists[l]` its (idx, val,
    cnt) or None for a layer without k-WTA."""
    ref = networks.run_chain(layers, x, Ws, bs)
    for li, (spec, r) in enumerate(zip(layers, ref)):
        acc = r["acc"].reshape(-1, spec.c_out)
        got = host(sums[li]).reshape(acc.shape).astype(np.int64)
        assert np.array_equal(got, acc), f"layer {li} ({spec.name}): sums differ from the oracle"
        if lists[li] is None:
            continue
        gi, gv, gc = (host(t) for t in lists[li])
        want = np.asarray(r["out"], dtype=np.int64).reshape(-1, spec.c_out)
        assert np.array_equal(gc, (want != 0).sum(axis=1)), f"layer {li}: list counts"
        dense = dense_from_lists(gi, gv, gc, spec.c_out).astype(np.int64)
        assert np.array_equal(dense, want), f"layer {li} ({spec.name}): lists differ from the oracle"


# dtype, (b, h, w, c_in), nnz, kh, kw, stride, pad, c_out, n, pool, k, bias, shift,
# out ("lists"/"dense"), expected plan (path, tile mode or None)
CASES = [
    # keyword-spotting conv2 shape: 5x5, 2x2 pool, int8: input-stationary, whole image
    ("i8", (3, 14, 14, 64), 8, 5, 5, 1, 0, 64, 16, 2, 8, False, 9, "lists", ("scatter", None)),
    # the same layer with stride 2: the gather kernel (rectangle tiles)
    ("i8", (2, 17, 17, 64), 8, 5, 5, 2, 2, 64, 16, 1, 8, False, 9, "lists", ("fused", 1)),
    # 3x3 pad 1, ragged image against the tiles, fp32 dense output: the
    # table-block kernel (one block), the last tile part-full
    ("f32", (2, 19, 13, 64), 7, 3, 3, 1, 1, 64, 8, 1, 8, False, None, "dense", ("blocks", None)),
    # wide image, 6 sets (not a power of two): the gather kernel, column tiles
    ("f32", (1, 9, 150, 64), 7, 3, 3, 1, 1, 48, 8, 1, 8, False, None, "lists", ("fused", 1)),
    # 1x1 expand: rows of items, bias, requantised lists, ragged last tile
    ("i8", (2, 7, 9, 96), 12, 1, 1, 1, 0, 576, 8, 1, 72, True, 9, "lists", ("fused", 0)),
    # linear, int32 dense output, bias: one workgroup per sample
    ("i8", (37, 1, 1, 512), 64, 1, 1, 1, 0, 64, 8, 1, 16, True, None, "dense", ("sample", None)),
    ("i8", (29, 1, 1, 300), 40, 1, 1, 1, 0, 12, 1, 1, 3, False, None, "lists", ("sample", None)),
    # dense kernels (n = 1), one accumulator per set in registers
    ("i8", (3, 4, 5, 300), 40, 1, 1, 1, 0, 12, 1, 1, 3, False, None, "lists", ("fused", 0)),
    ("f32", (3, 6, 5, 40), 9, 3, 3, 1, 1, 16, 1, 1, 5, True, None, "dense", ("blocks", None)),
    ("f32", (3, 6, 5, 40), 9, 3, 3, 1, 1, 12, 1, 1, 5, True, None, "dense", ("fused", 1)),
    # stride 2, odd input
    ("f32", (2, 17, 17, 32), 5, 3, 3, 2, 1, 32, 4, 1, 4, False, None, "lists", ("blocks", None)),
    ("f32", (2, 17, 17, 32), 5, 3, 3, 2, 1, 24, 4, 1, 4, False, None, "lists", ("fused", 1)),
    # 5x5 pad 2 with pool, odd number of sets (one set per lane)
    ("f32", (2, 12, 10, 16), 4, 5, 5, 1, 2, 24, 8, 2, 6, True, None, "dense", ("fused", 1)),
    # k = 0 and k = c_out
    ("i8", (2, 8, 8, 32), 6, 3, 3, 1, 1, 32, 4, 1, 0, False, 3, "lists", ("scatter", None)),
    ("i8", (2, 8, 8, 32), 6, 3, 3, 1, 1, 32, 4, 1, 32, True, None, "dense", ("scatter", None)),
    # ties everywhere: +-1 weights, all-one inputs
    ("i8", (4, 9, 9, 64), 8, 3, 3, 1, 1, 64, 16, 1, 8, False, 0, "lists", ("scatter", None)),
    # lists that do not fit the LDS budget: some pixels are read from global memory
    ("f32", (2, 24, 24, 128), 100, 3, 3, 1, 1, 12, 4, 1, 4, False, None, "lists", ("fused", 1)),
    # c_out not a multiple of 4, odd set count (one set per lane): input-stationary
    ("i8", (3, 6, 6, 24), 5, 3, 3, 1, 1, 6, 2, 1, 2, True, 2, "lists", ("scatter", None)),
    # the same with stride 2: two kernels (sums, then k-WTA)
    ("i8", (3, 7, 7, 24), 5, 3, 3, 2, 1, 6, 2, 1, 2, True, 2, "lists", ("tiled", None)),
    # input-stationary: 7x7 pad 3 with pool; 128 channels (two keys per lane);
    # a map wider than one band (several bands per image); a map too wide
    # for the byte-sized column field (the gather kernel)
    ("i8", (2, 12, 12, 16), 5, 7, 7, 1, 3, 32, 4, 2, 6, True, 8, "lists", ("scatter", None)),
    ("i8", (2, 9, 9, 32), 6, 3, 3, 1, 1, 128, 16, 1, 20, True, None, "dense", ("scatter", None)),
    ("i8", (2, 9, 9, 32), 6, 3, 3, 1, 1, 128, 16, 1, 20, False, 10, "lists", ("scatter", None)),
    ("i8", (1, 40, 40, 32), 6, 3, 3, 1, 1, 64, 8, 2, 8, True, 9, "lists", ("scatter", None)),
    # k-WTA by merged top lists (k <= 8): 8 channels per lane with ties, and
    # 96 channels (lanes past the row) with pooling
    ("i8", (2, 9, 9, 32), 6, 3, 3, 1, 1, 128, 16, 1, 7, False, 0, "lists", ("scatter", None)),
    ("i8", (2, 10, 10, 32), 6, 3, 3, 1, 1, 96, 16, 2, 5, True, 0, "lists", ("scatter", None)),
    ("i8", (1, 6, 300, 16), 4, 3, 3, 1, 1, 16, 4, 1, 4, False, 5, "lists", ("fused", 1)),
    # int8 1x1 layers with many items and a k-WTA over long rows: one
    # wavefront per item (config 5's expand shape; more sets than lanes; ties
    # with fewer sets than lanes; lists longer than one 64-entry chunk with
    # int32 dense output; eight sets with k = 0 and k = c_out)
    ("i8", (8, 24, 24, 96), 12, 1, 1, 1, 0, 576, 8, 1, 72, True, 9, "lists", ("rows", None)),
    ("i8", (1, 64, 64, 32), 4, 1, 1, 1, 0, 1600, 8, 1, 100, True, 6, "lists", ("rows", None)),
    ("i8", (2, 48, 48, 64), 8, 1, 1, 1, 0, 192, 16, 1, 40, False, 0, "lists", ("rows", None)),
    ("i8", (2, 48, 48, 128), 100, 1, 1, 1, 0, 1000, 8, 1, 120, True, None, "dense", ("rows", None)),
    ("i8", (1, 70, 70, 64), 3, 1, 1, 1, 0, 256, 32, 1, 0, False, 9, "lists", ("rows", None)),
    ("i8", (1, 70, 70, 64), 3, 1, 1, 1, 0, 256, 32, 1, 256, True, None, "dense", ("rows", None)),
    # the same shape in fp32: the table-block kernel, k-WTA over 256 channels
    ("f32", (4, 32, 32, 64), 7, 1, 1, 1, 0, 256, 16, 1, 26, True, None, "dense", ("blocks", None)),
    # fp32 table-block kernel: a 3x3 layer whose taps are split into channel
    # blocks (the stage-3 3x3 shape), a 1x1 layer over 1024 channels in 8
    # channel blocks (lists continue from block to block), k = 0, k = c_out,
    # 64 channels in 4 sets, 128 channels with two keys per lane
    ("f32", (2, 9, 9, 256), 26, 3, 3, 1, 1, 256, 16, 1, 26, False, None, "lists", ("blocks", None)),
    ("f32", (2, 7, 5, 1024), 102, 1, 1, 1, 0, 256, 16, 1, 26, True, None, "lists", ("blocks", None)),
    ("f32", (2, 7, 5, 1024), 102, 1, 1, 1, 0, 256, 16, 1, 0, False, None, "lists", ("blocks", None)),
    ("f32", (2, 6, 6, 256), 26, 3, 3, 1, 1, 256, 16, 1, 256, True, None, "dense", ("blocks", None)),
    ("f32", (3, 10, 10, 64), 7, 3, 3, 1, 1, 64, 16, 1, 8, True, None, "lists", ("blocks", None)),
    ("f32", (2, 8, 9, 96), 9, 3, 3, 1, 1, 128, 4, 1, 20, False, None, "lists", ("blocks", None)),
    ("f32", (2, 7, 7, 64), 7, 3, 3, 1, 1, 128, 4, 1, 16, True, None, "dense", ("blocks", None)),
    # 256 sets of one kernel (64 lanes per pixel): k-WTA on a copied tile, 16 lanes per row
    ("f32", (2, 5, 6, 32), 5, 3, 3, 1, 1, 256, 1, 1, 40, True, None, "lists", ("blocks", None)),
    ("f32", (2, 5, 6, 32), 5, 3, 3, 1, 1, 256, 1, 1, 40, False, None, "dense", ("blocks", None)),
    # a table too large for LDS, one output vector per sample: one workgroup
    # per sample (keyword-spotting linear1: the 5x5x64 map as a whole-map conv)
    ("i8", (8, 5, 5, 64), 8, 5, 5, 1, 0, 1500, 20, 1, 75, False, 8, "lists", ("sample", None)),
    # plain linear layers: fp32 with bias, int32 dense output at the 2048 row limit
    ("f32", (6, 1, 1, 2000), 200, 1, 1, 1, 0, 1024, 8, 1, 50, True, None, "dense", ("sample", None)),
    ("i8", (5, 1, 1, 1600), 150, 1, 1, 1, 0, 2048, 16, 1, 200, True, None, "dense", ("sample", None)),
    # odd set count (G = 167), k not a multiple of 4, requantised lists
    ("i8", (3, 1, 1, 1200), 90, 1, 1, 1, 0, 1002, 6, 1, 33, True, 10, "lists", ("sample", None)),
    # k = 0 and k = c_out
    ("i8", (3, 1, 1, 1200), 100, 1, 1, 1, 0, 1536, 12, 1, 0, False, 9, "lists", ("sample", None)),
    ("f32", (3, 1, 1, 1200), 100, 1, 1, 1, 0, 1536, 12, 1, 1536, False, None, "lists", ("sample", None)),
    # ties everywhere: +-1 weights, all-one inputs, whole-map 3x3 window
    ("i8", (4, 3, 3, 256), 20, 3, 3, 1, 0, 1000, 8, 1, 60, False, 0, "lists", ("sample", None)),
    # 256 taps per sample (16x16 map), fp32 whole-map window
    ("f32", (2, 16, 16, 32), 4, 16, 16, 1, 0, 512, 8, 1, 20, False, None, "lists", ("sample", None)),
]


@pytest.mark.parametrize("case", CASES, ids=[f"{c[0]}-{c[1]}-{c[3]}x{c[4]}-n{c[8]}-k{c[10]}-{c[13]}"
                                             for c in CASES])
def test_fused_layer(case):
    (dtype, shape, nnz, kh, kw, stride, pad, c_out, n, pool, k, has_bias, shift, mode,
     want) = case
    r = np.random.default_rng(zlib.crc32(repr(case[:13]).encode()))
    b, h, w, c_in = shape
    ties = shift == 0
    x = sparse_input(r, shape, nnz, dtype, low_range=ties)
    W = weights(r, c_out, kh, kw, c_in, n, dtype, low_range=ties)
    bias = None
    if has_bias:
        bias = (r.integers(-1000, 1001, size=c_out).astype(np.int32) if dtype == "i8"
                else r.normal(size=c_out).astype(np.float32))
    aug, _ = ops.pack(W.reshape(c_out, -1), n)
    ad = ops.aug_to_device(aug)
    xd = dev(x)
    idx, lv, cnt = ops.compact(xd.reshape(-1, c_in))
    tdt = torch.int8 if dtype == "i8" else torch.float32
    plan = ops.mrs_plan(tdt, c_in, shape, kh, kw, stride, pad, c_out, n, pool, k)
    assert plan["path"] == want[0], plan
    if want[1] is not None:
        assert plan["tile_mode"] == want[1], plan
    odt = torch.int8 if shift is not None and dtype == "i8" else None
    cap = ops.list_capacity(k) if mode == "lists" else None
    bd = None if bias is None else dev(bias)

    def run(keep):
        y, res = ops.mrs_kwta_conv2d(idx, lv, cnt, shape, ad, kh, kw, n, stride, pad, bd, pool,
                                     k=k, out_dtype=odt, shift=shift or 0, keep_sums=keep,
                                     cap=cap)
        if mode == "lists":
            res = tuple(host(t) for t in res)
        else:
            res = host(res)
        return host(y), res

    y, res = run(True)
    _, res2 = run(False)
    if mode == "lists":
        # entries past a row's count are unspecified; the rest must agree
        assert np.array_equal(res[2], res2[2]), "keep_sums changed the counts"
        live = np.arange(res[0].shape[1])[None, :] < res[2][:, None]
        for a, b2 in zip(res[:2], res2[:2]):
            assert np.array_equal(a[live], b2[live]), "keep_sums changed the output"
        out = dense_from_lists(*res, c_out)
    else:
        assert np.array_equal(res, res2), "keep_sums changed the output"
        out = res.reshape(-1, c_out)

    ref = o.conv2d_nhwc(x, W, stride, pad, bias)
    if pool == 2:
        ref = o.maxpool2x2_nhwc(ref)
    assert y.shape == ref.shape
    win = o.kwta_winners(ref, k)
    if dtype == "i8":
        assert np.array_equal(y.astype(np.int64), ref), "sums"
        if odt == torch.int8:
            want_out = o.requant(ref, shift, win).reshape(-1, c_out)
        else:
            want_out = np.where(win, ref, 0).reshape(-1, c_out)
        assert np.array_equal(out.astype(np.int64), want_out.astype(np.int64)), "k-WTA output"
        if mode == "lists":
            # the lists hold exactly the non-zero outputs
            assert np.array_equal(res[2], (want_out != 0).sum(axis=1))
    else:
        S = o.abs_sum_conv(x, W, stride, pad)
        if pool == 2:
            S = pool_S(S)
        if bias is not None:
            S = S + np.abs(bias.astype(np.float64))
        assert_f32_close(y, ref, S, "fused sums")
        near = check_kwta_f32(y, out, ref, S, k)
        assert near <= max(1, out.shape[0] // 100)


@pytest.mark.parametrize("mode", ["lists", "dense"])
@pytest.mark.parametrize("shape,kh", [((2, 6, 6, 256), 3), ((2, 7, 5, 1024), 1)])
def test_blocks_f32_exact_ties(shape, kh, mode):
    """The fp32 table-block layer with 32 channels per lane when many sums are
    equal: integer-valued inputs, +-1 weights and an integer bias make every
    sum an exact integer, with ties at the k-th largest in most pixels, so the
    threshold search runs to its last bit and the tied channels are taken in
    index order.  The sums and the k-WTA must equal the oracle's exactly."""
    c_in = shape[3]
    c_out, n, k, nnz = 256, 16, 26, 26 if kh == 3 else 102
    pad = 1 if kh == 3 else 0
    r = np.random.default_rng(4242 + kh)
    rows = int(np.prod(shape[:3]))
    x = np.zeros((rows, c_in), dtype=np.float32)
    for i in range(rows):
        pos = r.choice(c_in, size=nnz, replace=False)
        x[i, pos] = r.integers(1, 3, size=nnz).astype(np.float32)
    x = x.reshape(shape)
    W = np.sign(weights(r, c_out, kh, kh, c_in, n, "f32")).astype(np.float32)
    bias = r.integers(-2, 3, size=c_out).astype(np.float32)
    aug, _ = ops.pack(W.reshape(c_out, -1), n)
    xd = dev(x)
    idx, lv, cnt = ops.compact(xd.reshape(-1, c_in))
    plan = ops.mrs_plan(torch.float32, c_in, shape, kh, kh, 1, pad, c_out, n, 1, k)
    assert plan["path"] == "blocks", plan
    cap = ops.list_capacity(k) if mode == "lists" else None
    y, res = ops.mrs_kwta_conv2d(idx, lv, cnt, shape, ops.aug_to_device(aug), kh, kh, n, 1, pad,
                                 dev(bias), 1, k=k, keep_sums=True, cap=cap)
    torch.cuda.synchronize()
    ref = o.conv2d_nhwc(x, W, 1, pad, bias).reshape(-1, c_out)
    assert np.array_equal(host(y).reshape(-1, c_out).astype(np.float64), ref), "sums"
    srt = -np.sort(-ref, axis=1)
    assert (srt[:, k - 1] == srt[:, k]).mean() > 0.5, "too few ties at the threshold"
    want = np.where(o.kwta_winners(ref, k), ref, 0.0)
    out = (dense_from_lists(*(host(t) for t in res), c_out) if mode == "lists"
           else host(res).reshape(-1, c_out))
    assert np.array_equal(out.astype(np.float64), want), "k-WTA output"


@pytest.mark.parametrize("dtype", ["i8", "f32"])
def test_sample_sums_only(dtype):
    """cs_mrs_conv2d (no k-WTA) of a large-table linear layer takes the
    one-workgroup-per-sample kernel; the sums match the oracle."""
    r = np.random.default_rng(4242 if dtype == "i8" else 4243)
    shape, c_out, n = (7, 1, 1, 1600), 1500, 20
    x = sparse_input(r, shape, 160, dtype)
    W = weights(r, c_out, 1, 1, 1600, n, dtype)
    bias = (r.integers(-1000, 1001, size=c_out).astype(np.int32) if dtype == "i8"
            else r.normal(size=c_out).astype(np.float32))
    tdt = torch.int8 if dtype == "i8" else torch.float32
    assert ops.mrs_plan(tdt, 1600, shape, 1, 1, 1, 0, c_out, n, 1, -1)["path"] == "sample"
    aug, _ = ops.pack(W.reshape(c_out, -1), n)
    idx, lv, cnt = ops.compact(dev(x).reshape(-1, 1600))
    y = host(ops.mrs_conv2d(idx, lv, cnt, shape, ops.aug_to_device(aug), 1, 1, n, 1, 0,
                            dev(bias), 1))
    ref = o.conv2d_nhwc(x, W, 1, 0, bias)
    if dtype == "i8":
        assert np.array_equal(y.astype(np.int64), ref)
    else:
        S = o.abs_sum_conv(x, W, 1, 0) + np.abs(bias.astype(np.float64))
        assert_f32_close(y, ref, S, "sample sums")


# (b, h, w, c_in), nnz, c_out, n, bias: int8 1x1 sums only, one wavefront per
# item (config 5's project shape: G = 12, slices of sets; G = 72, one set per
# lane; c_out not a multiple of 4; lists longer than 64 entries)
ROWS_SUMS_CASES = [
    ((4, 32, 32, 576), 72, 96, 8, True),
    ((2, 48, 48, 96), 12, 576, 8, False),
    ((1, 70, 70, 120), 15, 150, 10, True),
    ((2, 48, 48, 256), 100, 200, 8, True),
]


@pytest.mark.parametrize("case", ROWS_SUMS_CASES, ids=[str(c[0]) + f"-{c[2]}" for c in ROWS_SUMS_CASES])
def test_rows_sums_only(case):
    """cs_mrs_conv2d (no k-WTA) of an int8 1x1 layer with many items takes
    the one-wavefront-per-item kernel; the sums match the oracle exactly."""
    shape, nnz, c_out, n, has_bias = case
    r = np.random.default_rng(zlib.crc32(repr(case).encode()))
    c_in = shape[3]
    x = sparse_input(r, shape, nnz, "i8")
    W = weights(r, c_out, 1, 1, c_in, n, "i8")
    bias = r.integers(-1000, 1001, size=c_out).astype(np.int32) if has_bias else None
    assert ops.mrs_plan(torch.int8, c_in, shape, 1, 1, 1, 0, c_out, n, 1, -1)["path"] == "rows"
    aug, _ = ops.pack(W.reshape(c_out, -1), n)
    idx, lv, cnt = ops.compact(dev(x).reshape(-1, c_in))
    y = host(ops.mrs_conv2d(idx, lv, cnt, shape, ops.aug_to_device(aug), 1, 1, n, 1, 0,
                            None if bias is None else dev(bias), 1))
    assert np.array_equal(y.astype(np.int64), o.conv2d_nhwc(x, W, 1, 0, bias))


def test_fused_partial_staging_plan():
    """The budget case above really leaves pixels unstaged: its lists need
    more chunks than the LDS list budget of a tile."""
    plan = ops.mrs_plan(torch.float32, 128, (2, 24, 24, 128), 3, 3, 1, 1, 12, 4, 1, 4)
    assert plan["path"] == "fused"
    need = plan["npix_cap"] * 25                 # 100 entries per pixel = 25 chunks
    assert plan["list_cap"] < need, plan


def test_fused_column_tiles_plan():
    plan = ops.mrs_plan(torch.float32, 64, (1, 9, 150, 64), 3, 3, 1, 1, 48, 8, 1, 8)
    assert plan["path"] == "fused" and plan["tile_mode"] == 1
    assert 0 < plan["tile_cols"] < 150, plan


def test_fused_repeatable_and_overwrites():
    """Two calls give identical bits, and stale data in the outputs is
    overwritten (lists beyond the count are not read)."""
    r = np.random.default_rng(77)
    shape = (2, 11, 11, 64)
    x = sparse_input(r, shape, 7, "f32")
    W = weights(r, 64, 3, 3, 64, 8, "f32")
    aug, _ = ops.pack(W.reshape(64, -1), 8)
    ad = ops.aug_to_device(aug)
    idx, lv, cnt = ops.compact(dev(x).reshape(-1, 64))
    cap = ops.list_capacity(8)
    rows = 2 * 11 * 11
    lists = (torch.full((rows, cap), -1, dtype=torch.int16, device="cuda"),
             torch.full((rows, cap), 7.0, dtype=torch.float32, device="cuda"),
             torch.full((rows,), 99, dtype=torch.int32, device="cuda"))
    y = torch.full((2, 11, 11, 64), 3.0, device="cuda")
    ops.mrs_kwta_conv2d(idx, lv, cnt, shape, ad, 3, 3, 8, 1, 1, k=8, y=y, lists=lists)
    a = [host(t).copy() for t in lists] + [host(y).copy()]
    ops.mrs_kwta_conv2d(idx, lv, cnt, shape, ad, 3, 3, 8, 1, 1, k=8, y=y, lists=lists)
    b = [host(t).copy() for t in lists] + [host(y).copy()]
    assert (a[2] <= 8).all() and (a[2] >= 0).all()
    assert np.array_equal(a[2], b[2]) and np.array_equal(a[3].view(np.uint32), b[3].view(np.uint32))
    live = np.arange(cap)[None, :] < a[2][:, None]
    assert np.array_equal(a[0][live], b[0][live])
    assert np.array_equal(a[1][live].view(np.uint32), b[1][live].view(np.uint32))


# ------------------------------------------------------------------ dense first layer
# dtype, (b, h, w, c_in), kh, kw, stride, pad, pool, k, bias, shift, out
DENSE_KWTA_CASES = [
    ("i8", (5, 32, 32, 1), 5, 5, 1, 0, 2, 8, False, 11, "lists"),     # keyword-spotting conv1
    ("i8", (3, 20, 18, 1), 5, 5, 1, 0, 2, 8, True, 7, "dense"),
    ("i8", (2, 13, 11, 2), 3, 3, 1, 1, 1, 12, True, None, "lists"),   # no pool, pad, 2 channels
    ("i8", (2, 16, 16, 3), 3, 3, 2, 1, 2, 5, False, 4, "lists"),      # stride 2
    ("i8", (2, 12, 12, 1), 5, 5, 1, 2, 2, 0, False, 3, "lists"),      # k = 0
    ("i8", (4, 12, 12, 1), 3, 3, 1, 1, 2, 8, False, 0, "lists"),      # ties: +-1 weights, 0/1 input
    ("i8", (2, 12, 12, 1), 5, 5, 1, 0, 2, 40, False, 6, "lists"),     # k > 32: two kernels
    ("i8", (3, 10, 12, 1), 3, 3, 1, 1, 1, 20, True, 5, "lists"),      # top-32 networks, no pool
    ("i8", (520, 36, 36, 1), 5, 5, 1, 0, 2, 3, True, 9, "lists"),     # 256 items per workgroup
    ("f32", (2, 14, 14, 1), 5, 5, 1, 0, 2, 8, True, None, "dense"),   # fp32: two kernels
]


@pytest.mark.parametrize("case", DENSE_KWTA_CASES,
                         ids=[f"{c[0]}-{c[1]}-{c[2]}x{c[3]}-p{c[6]}-k{c[7]}-{c[10]}"
                              for c in DENSE_KWTA_CASES])
def test_dense_kwta_layer(case):
    dtype, shape, kh, kw, stride, pad, pool, k, has_bias, shift, mode = case
    r = np.random.default_rng(zlib.crc32(repr(case).encode()))
    b, h, w, c_in = shape
    ties = shift == 0
    if dtype == "i8":
        x = (r.integers(0, 2, size=shape) if ties else r.integers(-127, 128, size=shape)).astype(np.int8)
        W = r.integers(-127, 128, size=(64, kh, kw, c_in)).astype(np.int8)
        W[W == 0] = 1
        if ties:
            W = np.sign(W).astype(np.int8)
    else:
        x = r.normal(size=shape).astype(np.float32)
        W = r.normal(size=(64, kh, kw, c_in)).astype(np.float32)
    bias = None
    if has_bias:
        bias = (r.integers(-1000, 1001, size=64).astype(np.int32) if dtype == "i8"
                else r.normal(size=64).astype(np.float32))
    aug, _ = ops.pack(W.reshape(64, -1), 1)
    ad = ops.aug_to_device(aug)
    odt = torch.int8 if shift is not None and dtype == "i8" else None
    cap = ops.list_capacity(k) if mode == "lists" else None
    bd = None if bias is None else dev(bias)

    def run(keep):
        y, res = ops.conv2d_dense_kwta(dev(x), ad, kh, kw, 1, stride, pad, bd, pool, k=k,
                                       out_dtype=odt, shift=shift or 0, keep_sums=keep, cap=cap)
        res = tuple(host(t) for t in res) if mode == "lists" else host(res)
        return host(y), res

    y, res = run(True)
    _, res2 = run(False)
    if mode == "lists":
        assert np.array_equal(res[2], res2[2])
        live = np.arange(res[0].shape[1])[None, :] < res[2][:, None]
        for a, b2 in zip(res[:2], res2[:2]):
            assert np.array_equal(a[live], b2[live]), "keep_sums changed the output"
        out = dense_from_lists(*res, 64)
    else:
        assert np.array_equal(res, res2)
        out = res.reshape(-1, 64)
    ref = o.conv2d_nhwc(x, W, stride, pad, bias)
    if pool == 2:
        ref = o.maxpool2x2_nhwc(ref)
    win = o.kwta_winners(ref, k)
    if dtype == "i8":
        assert np.array_equal(y.astype(np.int64), ref), "sums"
        want = (o.requant(ref, shift, win) if odt == torch.int8
                else np.where(win, ref, 0)).reshape(-1, 64)
        assert np.array_equal(out.astype(np.int64), want.astype(np.int64)), "k-WTA output"
        if mode == "lists":
            assert np.array_equal(res[2], (want != 0).sum(axis=1))
    else:
        S = o.abs_sum_conv(x, W, stride, pad)
        if pool == 2:
            S = pool_S(S)
        if bias is not None:
            S = S + np.abs(bias.astype(np.float64))
        assert_f32_close(y, ref, S, "dense sums")
        check_kwta_f32(y, out, ref, S, k)


# ------------------------------------------------------------- three-layer tail
# (b, h, w, c_in), nnz, kh, kw, pad, c_out, n, pool, k, shift, c_out2, n2, k2, shift2,
# c_out3, n3, ties
CHAIN3_CASES = [
    # keyword-spotting shape at a small batch: one kernel
    ((6, 14, 14, 64), 8, 5, 5, 0, 64, 16, 2, 8, 9, 1500, 20, 75, 8, 12, 1, False),
    # 3x3 pad 1 without pool, 96 channels, ties everywhere: one kernel
    ((3, 6, 7, 32), 5, 3, 3, 1, 96, 8, 1, 7, 0, 200, 8, 20, 0, 10, 2, True),
    # an image wider than one band: the two-call fallback
    ((2, 64, 64, 16), 3, 3, 3, 1, 32, 4, 2, 4, 6, 64, 4, 10, 4, 8, 1, False),
    # k = 0 in the first layer: empty lists into the second (its sums are its bias)
    ((2, 10, 10, 16), 4, 3, 3, 1, 32, 4, 2, 0, 6, 64, 8, 10, 4, 8, 1, False),
]


@pytest.mark.parametrize("case", CHAIN3_CASES, ids=[f"{c[0]}-{c[1]}x{c[2]}-to{c[10]}" for c in CHAIN3_CASES])
def test_chain3_matches_separate_calls(case):
    """cs_mrs_kwta_chain3 against the oracle at every layer (sums, lists), and
    against cs_mrs_kwta_conv2d followed by cs_mrs_kwta_chain2 on its lists:
    the same bits in every output."""
    (shape, nnz, kh, kw, pad, c_out, n, pool, k, shift, c_out2, n2, k2, shift2, c_out3, n3,
     ties) = case
    r = np.random.default_rng(zlib.crc32(repr(case).encode()))
    b, h, w, c_in = shape
    x = sparse_input(r, shape, nnz, "i8", low_range=ties)
    ho, wo = h + 2 * pad - kh + 1, w + 2 * pad - kw + 1
    hp, wp = ho // pool, wo // pool
    W1 = weights(r, c_out, kh, kw, c_in, n, "i8", low_range=ties)
    W2 = weights(r, c_out2, hp, wp, c_out, n2, "i8", low_range=ties)
    W3 = weights(r, c_out3, 1, 1, c_out2, n3, "i8")
    b1, b2, b3 = (dev(r.integers(-1000, 1001, size=m).astype(np.int32)) for m in (c_out, c_out2, c_out3))
    a1, a2, a3 = (ops.aug_to_device(ops.pack(Wx.reshape(Wx.shape[0], -1), nx)[0])
                  for Wx, nx in ((W1, n), (W2, n2), (W3, n3)))
    idx, lv, cnt = ops.compact(dev(x).reshape(-1, c_in))
    cap1, cap2 = ops.list_capacity(k), ops.list_capacity(k2)
    got = ops.mrs_kwta_chain3(idx, lv, cnt, shape, a1, kh, kw, n, 1, pad, b1, pool, k=k,
                              shift=shift, aug2=a2, n2=n2, bias2=b2, k2=k2, shift2=shift2,
                              aug3=a3, n3=n3, bias3=b3, keep_sums=True, cap=cap1, cap2=cap2)
    y, lists = ops.mrs_kwta_conv2d(idx, lv, cnt, shape, a1, kh, kw, n, 1, pad, b1, pool, k=k,
                                   out_dtype=torch.int8, shift=shift, keep_sums=True, cap=cap1)
    y2, lists2, y3 = ops.mrs_kwta_chain2(*lists, (b, hp, wp, c_out), a2, hp, wp, n2, 1, 0, b2, 1,
                                         k=k2, shift=shift2, aug2=a3, n2=n3, bias2=b3,
                                         keep_sums=True, cap=cap2)
    torch.cuda.synchronize()
    for nm, g, e in (("y", got[0], y), ("y2", got[2], y2), ("y3", got[4], y3)):
        assert np.array_equal(host(g).reshape(-1), host(e).reshape(-1)), nm
    for nm, g, e in (("lists", got[1], lists), ("lists2", got[3], lists2)):
        gi, gv, gc = (host(t) for t in g)
        ei, ev, ec = (host(t) for t in e)
        assert np.array_equal(gc, ec), nm + " counts"
        live = np.arange(gi.shape[1])[None, :] < ec[:, None]
        assert np.array_equal(gi[live], ei[live]) and np.array_equal(gv[live], ev[live]), nm
    # every layer against the oracle: conv (pool, k-WTA, requant) -> a window
    # over the whole pooled map (the NHWC flatten of a linear layer) -> linear
    layers = (
        LayerSpec("conv", "conv", c_in, c_out, n=n, kh=kh, kw=kw, pad=pad, pool=pool, k=k,
                  shift=shift, bias=True),
        LayerSpec("map", "linear", hp * wp * c_out, c_out2, n=n2, k=k2, shift=shift2, bias=True),
        LayerSpec("last", "linear", c_out2, c_out3, n=n3, bias=True),
    )
    check_chain_against_oracle(layers, x, [W1, W2.reshape(c_out2, -1), W3.reshape(c_out3, -1)],
                               [host(b1), host(b2), host(b3)], [got[0], got[2], got[4]],
                               [got[1], got[3], None])


# ------------------------------------------------------------- four-layer chain
# (b, h, w, c_in), kh, kw, pad, pool, k, shift | kh2, pad2, c_out2, n2, pool2, k2, shift2 |
# c_out3, n3, k3, shift3 | c_out4, n4 | ties
DENSE_CHAIN_CASES = [
    # keyword-spotting shape at a small batch: one kernel (second layer output-stationary)
    ((5, 32, 32, 1), 5, 5, 0, 2, 8, 11, 5, 0, 64, 16, 2, 8, 9, 1500, 20, 75, 8, 12, 1, False),
    # output-stationary second layer with padding, no second pool, one 64-pixel
    # block, ties in the first layer
    ((3, 16, 16, 1), 3, 3, 1, 2, 8, 0, 3, 1, 64, 16, 1, 8, 3, 100, 4, 10, 5, 10, 2, True),
    # output-stationary with 48 outputs (four sets of 12) and three pixel blocks
    ((2, 28, 28, 1), 5, 5, 2, 2, 8, 10, 3, 1, 48, 12, 2, 6, 8, 60, 6, 12, 6, 12, 1, False),
    # no first pool, 3x3 pad 1 twice, ties in the first layer: one kernel
    ((3, 12, 12, 2), 3, 3, 1, 1, 8, 0, 3, 1, 64, 8, 2, 6, 5, 100, 4, 10, 5, 10, 2, True),
    # 128 channels in the second layer: the two-call fallback
    ((2, 16, 16, 1), 5, 5, 0, 2, 8, 11, 3, 1, 128, 16, 1, 12, 7, 200, 8, 20, 6, 8, 1, False),
    # every output of the third layer wins (k3 = c_out3); no pool in the second
    ((2, 12, 12, 1), 3, 3, 1, 2, 4, 6, 3, 1, 64, 8, 1, 8, 5, 16, 4, 16, 5, 4, 1, False),
]


@pytest.mark.parametrize("case", DENSE_CHAIN_CASES,
                         ids=[f"{c[0]}-{c[1]}x{c[2]}-p{c[4]}-to{c[9]}" for c in DENSE_CHAIN_CASES])
def test_dense_chain3_matches_separate_calls(case):
    """cs_conv2d_dense_kwta_chain3 against the oracle at every layer (sums,
    lists), and against cs_conv2d_dense_kwta followed by cs_mrs_kwta_chain3 on
    its lists: the same bits in every output."""
    (shape, kh, kw, pad, pool, k, shift, kh2, pad2, c_out2, n2, pool2, k2, shift2, c_out3, n3,
     k3, shift3, c_out4, n4, ties) = case
    r = np.random.default_rng(zlib.crc32(repr(case).encode()))
    b, h, w, c_in = shape
    if ties:
        x = r.integers(0, 2, size=shape).astype(np.int8)
        W1 = np.sign(r.integers(-127, 128, size=(64, kh, kw, c_in))).astype(np.int8)
        W1[W1 == 0] = 1
    else:
        x = r.integers(-127, 128, size=shape).astype(np.int8)
        W1 = r.integers(-127, 128, size=(64, kh, kw, c_in)).astype(np.int8)
        W1[W1 == 0] = 1
    ho1, wo1 = (h + 2 * pad - kh + 1) // pool, (w + 2 * pad - kw + 1) // pool
    ho2, wo2 = (ho1 + 2 * pad2 - kh2 + 1) // pool2, (wo1 + 2 * pad2 - kh2 + 1) // pool2
    W2 = weights(r, c_out2, kh2, kh2, 64, n2, "i8")
    W3 = weights(r, c_out3, ho2, wo2, c_out2, n3, "i8")
    W4 = weights(r, c_out4, 1, 1, c_out3, n4, "i8")
    b1, b2, b3, b4 = (dev(r.integers(-1000, 1001, size=m).astype(np.int32))
                      for m in (64, c_out2, c_out3, c_out4))
    a1, a2, a3, a4 = (ops.aug_to_device(ops.pack(Wx.reshape(Wx.shape[0], -1), nx)[0])
                      for Wx, nx in ((W1, 1), (W2, n2), (W3, n3), (W4, n4)))
    xd = dev(x)
    got = ops.conv2d_dense_kwta_chain3(
        xd, a1, kh, kw, 1, 1, pad, b1, pool, k=k, shift=shift, aug2=a2, kh2=kh2, kw2=kh2, n2=n2,
        pad2=pad2, bias2=b2, pool2=pool2, k2=k2, shift2=shift2, aug3=a3, n3=n3, bias3=b3, k3=k3,
        shift3=shift3, aug4=a4, n4=n4, bias4=b4, keep_sums=True)
    y, lists = ops.conv2d_dense_kwta(xd, a1, kh, kw, 1, 1, pad, b1, pool, k=k,
                                     out_dtype=torch.int8, shift=shift, keep_sums=True,
                                     cap=ops.list_capacity(k))
    rest = ops.mrs_kwta_chain3(*lists, (b, ho1, wo1, 64), a2, kh2, kh2, n2, 1, pad2, b2, pool2,
                               k=k2, shift=shift2, aug2=a3, n2=n3, bias2=b3, k2=k3,
                               shift2=shift3, aug3=a4, n3=n4, bias3=b4, keep_sums=True)
    torch.cuda.synchronize()
    want = (y, lists) + tuple(rest)
    for i, nm in ((0, "y"), (2, "y2"), (4, "y3"), (6, "y4")):
        assert np.array_equal(host(got[i]).reshape(-1), host(want[i]).reshape(-1)), nm
    for i, nm in ((1, "lists"), (3, "lists2"), (5, "lists3")):
        gi, gv, gc = (host(t) for t in got[i])
        ei, ev, ec = (host(t) for t in want[i])
        assert np.array_equal(gc, ec), nm + " counts"
        live = np.arange(gi.shape[1])[None, :] < ec[:, None]
        assert np.array_equal(gi[live], ei[live]) and np.array_equal(gv[live], ev[live]), nm
    # every layer against the oracle: dense conv (pool, k-WTA, requant) -> conv
    # (pool, k-WTA, requant) -> a window over the whole map -> linear
    layers = (
        LayerSpec("conv1", "conv", c_in, 64, n=1, kh=kh, kw=kw, pad=pad, pool=pool, k=k,
                  shift=shift, bias=True),
        LayerSpec("conv2", "conv", 64, c_out2, n=n2, kh=kh2, kw=kh2, pad=pad2, pool=pool2, k=k2,
                  shift=shift2, bias=True),
        LayerSpec("map", "linear", ho2 * wo2 * c_out2, c_out3, n=n3, k=k3, shift=shift3,
                  bias=True),
        LayerSpec("last", "linear", c_out3, c_out4, n=n4, bias=True),
    )
    check_chain_against_oracle(
        layers, x, [W1, W2, W3.reshape(c_out3, -1), W4.reshape(c_out4, -1)],
        [host(b1), host(b2), host(b3), host(b4)], [got[0], got[2], got[4], got[6]],
        [got[1], got[3], got[5], None])
