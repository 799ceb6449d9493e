"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each check is independent of the oracle's own formula: a pure-Python brute
force, a library routine (torch float64 conv/linear/max-pool), the paper's
printed counts, the paper's own k-WTA hardware procedures (sorting network +
FIFOs, 8-bit histogram), closed forms and special cases.
"""
from __future__ import annotations

import dataclasses
import itertools
import json
import os

import numpy as np
import pytest
import torch

from oracle import cs_oracle as o
from oracle import networks
from tests import paper_kwta
from workloads import CONFIGS, complementary_weights, generate, sparse_rows, tensor_digest

GOLD = os.path.join(os.path.dirname(__file__), "golden")
PAPER = json.load(open(os.path.join(GOLD, "paper_values.json")))

pytestmark = pytest.mark.filterwarnings("ignore::DeprecationWarning")


def rng(seed=0):
    return np.random.default_rng(seed)


# ---------------------------------------------------------------- linear / conv
def brute_linear(x, W, b):
    B, D = x.shape
    O = W.shape[0]
    y = [[0] * O for _ in range(B)]
    for bi in range(B):
        for oi in range(O):
            s = 0 if b is None else int(b[oi]) if np.issubdtype(b.dtype, np.integer) else float(b[oi])
            for i in range(D):
                s += x[bi, i].item() * W[oi, i].item()
            y[bi][oi] = s
    return np.array(y)


def brute_conv(x, W, stride, pad, b):
    B, H, Wd, C = x.shape
    O, KH, KW, _ = W.shape
    Ho = (H + 2 * pad - KH) // stride + 1
    Wo = (Wd + 2 * pad - KW) // stride + 1
    y = np.zeros((B, Ho, Wo, O), dtype=object)
    for bi, ho, wo, oi in itertools.product(range(B), range(Ho), range(Wo), range(O)):
        s = 0 if b is None else b[oi].item()
        for ky, kx, c in itertools.product(range(KH), range(KW), range(C)):
            hy, wx = ho * stride + ky - pad, wo * stride + kx - pad
            if 0 <= hy < H and 0 <= wx < Wd:
                s += x[bi, hy, wx, c].item() * W[oi, ky, kx, c].item()
        y[bi, ho, wo, oi] = s
    return y


@pytest.mark.parametrize("dtype", ["i8", "f32"])
def test_linear_brute_force(dtype):
    r = rng(1)
    if dtype == "i8":
        x = r.integers(-127, 128, size=(3, 17)).astype(np.int8)
        x[x % 3 == 0] = 0
        W = r.integers(-127, 128, size=(6, 17)).astype(np.int8)
        b = r.integers(-1000, 1001, size=6).astype(np.int32)
        y = o.linear(x, W, b)
        assert y.dtype == np.int64
        assert np.array_equal(y, brute_linear(x, W, b).astype(np.int64))
    else:
        x = r.normal(size=(3, 17)).astype(np.float32)
        W = r.normal(size=(6, 17)).astype(np.float32)
        y = o.linear(x, W, None)
        np.testing.assert_allclose(y, brute_linear(x, W, None).astype(np.float64), rtol=1e-13, atol=1e-13)


def test_linear_matches_torch_float64():
    r = rng(2)
    x = r.normal(size=(5, 40))
    W = r.normal(size=(9, 40))
    b = r.normal(size=9)
    ref = torch.nn.functional.linear(torch.from_numpy(x), torch.from_numpy(W), torch.from_numpy(b)).numpy()
    np.testing.assert_allclose(o.linear(x, W, b), ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("kh,kw,stride,pad", [(1, 1, 1, 0), (3, 3, 1, 1), (5, 5, 1, 0), (3, 3, 2, 1), (3, 2, 1, 1)])
def test_conv_brute_force_int(kh, kw, stride, pad):
    r = rng(3 + kh + stride)
    x = r.integers(-127, 128, size=(2, 6, 7, 3)).astype(np.int8)
    x[r.random(x.shape) < 0.5] = 0
    W = r.integers(-127, 128, size=(4, kh, kw, 3)).astype(np.int8)
    b = r.integers(-1000, 1001, size=4).astype(np.int32)
    y = o.conv2d_nhwc(x, W, stride, pad, b)
    assert np.array_equal(y, brute_conv(x, W, stride, pad, b).astype(np.int64))


@pytest.mark.parametrize("kh,kw,stride,pad", [(1, 1, 1, 0), (3, 3, 1, 1), (5, 5, 1, 0), (3, 3, 2, 1), (2, 3, 2, 0)])
def test_conv_matches_torch_float64(kh, kw, stride, pad):
    """Cross-correlation in NHWC with OHWI weights equals torch's NCHW/OIHW conv2d."""
    r = rng(7)
    x = r.normal(size=(2, 9, 8, 5))
    W = r.normal(size=(6, kh, kw, 5))
    b = r.normal(size=6)
    ref = torch.nn.functional.conv2d(
        torch.from_numpy(x).permute(0, 3, 1, 2), torch.from_numpy(W).permute(0, 3, 1, 2),
        torch.from_numpy(b), stride=stride, padding=pad).permute(0, 2, 3, 1).numpy()
    np.testing.assert_allclose(o.conv2d_nhwc(x, W, stride, pad, b), ref, rtol=1e-12, atol=1e-12)


def test_conv3x3_is_nine_1x1():
    """Section 5.1: a 3x3 conv is computed as nine 1x1 convs."""
    r = rng(8)
    x = r.integers(-127, 128, size=(2, 7, 6, 4)).astype(np.int8)
    W = r.integers(-127, 128, size=(5, 3, 3, 4)).astype(np.int8)
    xp = np.zeros((2, 9, 8, 4), dtype=np.int8)
    xp[:, 1:8, 1:7, :] = x
    total = np.zeros((2, 7, 6, 5), dtype=np.int64)
    for ky in range(3):
        for kx in range(3):
            total += o.conv2d_nhwc(xp[:, ky:ky + 7, kx:kx + 6, :], W[:, ky:ky + 1, kx:kx + 1, :])
    assert np.array_equal(o.conv2d_nhwc(x, W, 1, 1), total)


def test_maxpool_matches_torch():
    r = rng(9)
    y = r.integers(-10 ** 6, 10 ** 6, size=(3, 8, 6, 5)).astype(np.int64)
    ref = torch.nn.functional.max_pool2d(torch.from_numpy(y.astype(np.float64)).permute(0, 3, 1, 2), 2, 2)
    ref = ref.permute(0, 2, 3, 1).numpy().astype(np.int64)
    assert np.array_equal(o.maxpool2x2_nhwc(y), ref)


def test_integer_results_exact_and_int32():
    """Integer configurations stay exact (|partial sums| far below 2^53) and
    fit in int32, the accumulator type of the int8 path."""
    bound = 1600 * 127 * 127 + 1000
    assert bound < 2 ** 31 - 1 and bound < 2 ** 53


# ---------------------------------------------------------------- k-WTA
def test_kwta_local_sorting_network_shape():
    """Section 3.3.3: the 8-input sorting network has 19 comparators in 6 layers."""
    p = PAPER["local_kwta_sorter"]
    comps = paper_kwta.batcher_network(p["inputs"])
    assert len(comps) == p["comparators"]
    assert paper_kwta.network_depth(comps, p["inputs"]) == p["depth"]
    # 0-1 principle: it sorts every binary input, so it sorts everything
    for bits in range(256):
        v = [((bits >> j) & 1, j) for j in range(8)]
        s = paper_kwta.sort_desc(v, comps)
        vals = [t[0] for t in s]
        assert vals == sorted(vals, reverse=True)


@pytest.mark.parametrize("k", [1, 8, 16, 63, 64])
def test_kwta_matches_paper_local_fifo_structure(k):
    """Oracle winners == the paper's local k-WTA (8 sorted FIFOs + tree), rows
    with many ties and with floats including +-0."""
    r = rng(10 + k)
    rows = [r.integers(-3, 4, size=64), r.integers(-1000, 1000, size=64),
            np.round(r.normal(size=64), 1).astype(np.float32),
            np.array([0.0, -0.0] * 32, dtype=np.float32), np.zeros(64, dtype=np.int32)]
    for row in rows:
        ref = paper_kwta.local_kwta_fifo(row, k)
        got = o.kwta_winners(row[None, :], k)[0]
        assert np.array_equal(got, ref)


def test_kwta_matches_paper_global_histogram():
    """Figure 10's shape: 1500 8-bit activations, 5-way histogram, 85% sparse
    (K = 225).  Without ties at the threshold the winner sets are equal; with
    ties, the histogram passes a superset whose extra members equal the
    threshold, and the oracle keeps the lowest-index ties."""
    p = PAPER["global_kwta_histogram"]
    K = round(p["row"] * (1 - p["sparsity"]))
    assert K == 225 and p["blocks"] * p["ways"] == p["row"]
    r = rng(11)
    # distinct values near the top so the threshold is unique
    row = np.concatenate([np.arange(256 - 240, 256), r.integers(0, 10, size=p["row"] - 240)])
    r.shuffle(row)
    thresh, passed = paper_kwta.global_kwta_histogram(row, K, p["ways"])
    win = o.kwta_winners(row[None, :].astype(np.int64), K)[0]
    assert passed.sum() == K and np.array_equal(win, passed)
    # heavy ties
    row = r.integers(0, 256, size=p["row"])
    thresh, passed = paper_kwta.global_kwta_histogram(row, K, p["ways"])
    win = o.kwta_winners(row[None, :].astype(np.int64), K)[0]
    assert win.sum() == K and passed.sum() >= K
    assert np.all(passed[win])
    assert np.all(row[passed & ~win] == thresh)
    tied = np.nonzero(row == thresh)[0]
    kept = tied[win[tied]]
    assert np.array_equal(kept, tied[:len(kept)])


def test_kwta_special_cases():
    r = rng(12)
    v = r.integers(-50, 50, size=(7, 33))
    assert o.kwta_winners(v, 33).all()
    assert not o.kwta_winners(v, 0).any()
    eq = np.full((3, 20), 5)
    m = o.kwta_winners(eq, 6)
    assert np.array_equal(m, np.tile(np.arange(20) < 6, (3, 1)))
    # winners keep their value even when negative (exactly K propagate)
    neg = -np.arange(1, 11)[None, :]
    assert np.array_equal(o.kwta(neg, 3), np.array([[-1, -2, -3] + [0] * 7]))


def test_kwta_invariants_random():
    r = rng(13)
    for c, k in [(64, 8), (256, 26), (576, 72), (1500, 75)]:
        v = r.integers(-20, 20, size=(5, c))
        m = o.kwta_winners(v, k)
        assert (m.sum(axis=1) == k).all()
        for row, mr in zip(v, m):
            assert row[mr].min() >= row[~mr].max()
            t = row[mr].min()
            tied = np.nonzero(row == t)[0]
            assert np.array_equal(tied[mr[tied]], tied[:mr[tied].sum()])


# ---------------------------------------------------------------- requantisation
def test_kwta_units_brute_force():
    """k-WTA in units of 64: each unit of a 256-wide row keeps exactly its own
    k largest (brute force over the unit by repeated maximum, ties to the
    lower index); k = 64 keeps everything."""
    r = rng(21)
    v = r.integers(-5, 6, size=(7, 256)).astype(np.int32)
    m = o.kwta_units_winners(v, 3)
    for row in range(7):
        for u in range(4):
            seg = v[row, 64 * u:64 * (u + 1)].astype(np.int64).tolist()
            want = set()
            for _ in range(3):
                best = max(i for i in range(64) if i not in want and
                           all(seg[i] > seg[j] or (seg[i] == seg[j] and i < j)
                               for j in range(64) if j not in want and j != i))
                want.add(best)
            assert set(np.flatnonzero(m[row, 64 * u:64 * (u + 1)]).tolist()) == want
    assert o.kwta_units_winners(v, 64).all()
    assert (o.kwta_units_winners(v, 5).reshape(7, 4, 64).sum(axis=2) == 5).all()


def test_requant_values():
    a = np.array([0, 1, -1, 255, 256, 257, -256, -257, 10 ** 6, -10 ** 6, 127, -128, 32767])
    got = o.requant(a, 1)
    exp = np.array([0, 0, -1, 127, 127, 127, -127, -127, 127, -127, 63, -64, 127], dtype=np.int8)
    assert np.array_equal(got, exp)
    assert np.array_equal(o.requant(np.array([-5, 5, -3]), 0), np.array([-5, 5, -3], dtype=np.int8))
    assert np.array_equal(o.requant(np.array([-5, 6]), 2), np.array([-2, 1], dtype=np.int8))
    w = np.array([True, False, True])
    assert np.array_equal(o.requant(np.array([1000, 1000, -1000]), 3, w), np.array([125, 0, -125], dtype=np.int8))


# ---------------------------------------------------------------- pack
def test_pack_roundtrip_and_invariants():
    r = rng(14)
    for d_out, R, n, dist in [(64, 512, 8, "int8"), (12, 36, 3, "normal"), (20, 25, 5, "int8"), (6, 10, 1, "int8")]:
        W = complementary_weights(r, r, d_out, R, n, dist)
        Wn = W != 0
        for g in range(d_out // n):
            cnt = Wn[g * n:(g + 1) * n].sum(axis=0)
            assert (cnt == 1).all()            # disjoint and covering
        assert (Wn.sum(axis=1) == R // n).all()
        val, kid, holes = o.pack(W, n)
        assert holes == 0 and (val != 0).all() and kid.max() < n
        assert np.array_equal(o.unpack(val, kid, n), W)


def test_pack_collision_and_holes():
    W = np.zeros((4, 6), dtype=np.int8)
    W[0, [0, 1]] = 3
    W[1, [2]] = -2
    W[2, [0, 5]] = 1
    val, kid, holes = o.pack(W, 2)
    assert holes == 3 + 4     # group 0 misses slots 3,4,5; group 1 misses 1,2,3,4
    assert np.array_equal(o.unpack(val, kid, 2), W)
    W[1, 1] = 7              # collides with kernel 0 at slot 1
    with pytest.raises(o.PackCollision) as e:
        o.pack(W, 2)
    assert (e.value.g, e.value.i) == (0, 1)


def test_pack_channels_hand_example():
    """One 1 x 2 filter over 2 channels, n = 2: channel 0 holds the left tap,
    channel 1 the right one; the overlay is one dense 1 x 2 slice."""
    W4 = np.zeros((1, 1, 2, 2), dtype=np.float32)
    W4[0, 0, 0, 0] = 1.5
    W4[0, 0, 1, 1] = -2.0
    val, cid, holes = o.pack_channels(W4, 2)
    assert val.shape == (1, 1, 1, 2) and holes == 0
    assert val[0, 0, 0].tolist() == [1.5, -2.0] and cid[0, 0, 0].tolist() == [0, 1]


def test_pack_channels_roundtrip_collision_holes():
    from workloads import channel_complementary_weights
    r = rng(19)
    for c_out, kh, kw, c, n in [(4, 3, 3, 6, 3), (3, 5, 5, 10, 5), (2, 1, 1, 4, 1)]:
        W4 = channel_complementary_weights(r, r, c_out, kh, kw, c, n)
        nz = (W4 != 0).reshape(c_out, kh * kw, c // n, n)
        assert (nz.sum(axis=3) == 1).all()            # each tap: exactly one channel per group
        val, cid, holes = o.pack_channels(W4, n)
        assert holes == 0 and (val != 0).all() and cid.max() < n
        assert np.array_equal(o.unpack_channels(val, cid, n), W4)
    # holes: brute-force count of the (filter, group, tap) with no channel
    W4 = np.zeros((2, 2, 2, 4), dtype=np.float32)
    W4[0, 0, 0, 1] = 1.0
    W4[1, 1, 1, 2] = 2.0
    W4[1, 0, 1, 3] = 3.0
    val, cid, holes = o.pack_channels(W4, 2)
    assert holes == 2 * 2 * 4 - 3
    assert np.array_equal(o.unpack_channels(val, cid, 2), W4)
    W4[1, 1, 1, 3] = 4.0                      # channels 2 and 3 of filter 1 at tap (1, 1)
    with pytest.raises(o.PackCollision) as e:
        o.pack_channels(W4, 2)
    assert (e.value.g, e.value.i) == (1, (1 * 2 + 1) * 2 + 1)


def test_pack_blocks_hand_example_and_invariants():
    """Two kernels over two blocks of 2 slots: kernel 0 owns block 0, kernel 1
    block 1; one Kernel ID per block.  Random block-complementary weights:
    the per-slot Kernel IDs are the block IDs repeated, the supports are whole
    blocks; a support splitting a block is refused."""
    from workloads import block_complementary_weights
    W = np.array([[1, 2, 0, 0], [0, 0, 3, 4]], dtype=np.int8)
    val, kidb, holes = o.pack_blocks(W, 2, 2)
    assert kidb[:, 0].tolist() == [0, 1] and holes == 0
    assert val[:, 0].tolist() == [1, 2, 3, 4]
    r = rng(20)
    for d_out, R, n, b in [(64, 147, 4, 3), (12, 40, 3, 4), (8, 6, 2, 3)]:
        W = block_complementary_weights(r, r, d_out, R, n, b)
        val, kidb, holes = o.pack_blocks(W, n, b)
        v2, kid, h2 = o.pack(W, n)
        assert np.array_equal(val, v2) and np.array_equal(np.repeat(kidb, b, axis=0), kid)
        assert holes == 0 and h2 == 0
        nzb = (W != 0).reshape(d_out, R // b, b)
        assert (nzb.all(axis=2) | ~nzb.any(axis=2)).all()
    W = np.array([[1, 0, 0, 0], [0, 0, 3, 4]], dtype=np.int8)
    with pytest.raises(o.BlockViolation) as e:
        o.pack_blocks(W, 2, 2)
    assert (e.value.o, e.value.blk) == (0, 0)


def test_pack_factors_from_paper():
    """Section 3 / Figure 7: 80% sparse kernels pack 5 to one dense kernel and
    20 channels give 4 sets; 66% sparse 3x3 kernels pack 3 to one."""
    p = PAPER["pack_factor_80"]
    n = round(1 / (1 - p["sparsity"]))
    assert n == p["kernels_per_set"]
    W = complementary_weights(rng(15), rng(16), p["channels"], 25, n, "int8")
    val, kid, holes = o.pack(W, n)
    assert val.shape[1] == p["sets"] and holes == 0
    q = PAPER["pack_factor_66"]
    W = complementary_weights(rng(17), rng(18), 3, q["kh"] * q["kw"], q["kernels_per_set"], "int8")
    assert ((W != 0).sum(axis=1) == q["nnz_per_kernel"]).all()
    val, kid, holes = o.pack(W, q["kernels_per_set"])
    assert val.shape == (9, 1) and holes == 0 and (val != 0).all()


# ---------------------------------------------------------------- product counts
def test_pair_count_closed_form_linear():
    """With complementary, covering sets, each non-zero input meets exactly one
    non-zero weight per set: products = sum_b nnz(x_b) * G."""
    r = rng(19)
    W = complementary_weights(r, r, 64, 512, 8, "int8")
    x = sparse_rows(r, 16, 512, 64, "u1_127")
    assert o.pair_count_linear(x, W) == int((x != 0).sum()) * 8


def test_pair_count_closed_form_conv():
    r = rng(20)
    W = complementary_weights(r, r, 16, 3 * 3 * 8, 4, "int8").reshape(16, 3, 3, 8)
    x = sparse_rows(r, 2 * 5 * 6, 8, 3, "u1_127").reshape(2, 5, 6, 8)
    cols = o.im2col_nhwc((x != 0).astype(np.int64), 3, 3, 1, 1)
    assert o.pair_count_conv(x, W, 1, 1) == int(cols.sum()) * 4


def test_paper_conv1x1_64_64_product_count():
    """Section 5.1: 4096 dense multiplies become 32 with 4 non-zeros per kernel
    and 8 non-zero inputs (complement factor 16)."""
    p = PAPER["conv1x1_64_64"]
    n = p["c_in"] // p["nnz_per_kernel"]
    W = complementary_weights(rng(21), rng(22), p["c_out"], p["c_in"], n, "int8").reshape(64, 1, 1, 64)
    x = sparse_rows(rng(23), 1, 64, p["nnz_inputs"], "u1_127").reshape(1, 1, 1, 64)
    assert o.dense_macs_conv(1, 1, 1, 64, 64, 1, 1) == p["dense_products"]
    assert o.pair_count_conv(x, W) == p["sparse_products"]


def test_paper_multiplicative_savings():
    """Figure 1: 90%/90% leaves 1% of the products; Section 2.3.2: 96% gives
    25x sparse-dense and 625x sparse-sparse."""
    p = PAPER["fig1_multiplicative"]
    n = round(1 / (1 - p["weight_sparsity"]))
    D, O, B = 1000, 40, 6
    W = complementary_weights(rng(24), rng(25), O, D, n, "int8")
    x = sparse_rows(rng(26), B, D, round(D * (1 - p["activation_sparsity"])), "u1_127")
    assert o.pair_count_linear(x, W) / o.dense_macs_linear(B, D, O) == pytest.approx(p["product_fraction"], rel=1e-12)
    q = PAPER["oneapi_theoretical"]
    n = round(1 / (1 - q["sparsity"]))
    W = complementary_weights(rng(27), rng(28), 50, 1000, n, "int8")
    xd = sparse_rows(rng(29), 4, 1000, None, "u1_127")
    xs = sparse_rows(rng(30), 4, 1000, round(1000 * (1 - q["sparsity"])), "u1_127")
    dense = o.dense_macs_linear(4, 1000, 50)
    assert dense / o.pair_count_linear(xd, W) == pytest.approx(q["sparse_dense_factor"])
    assert dense / o.pair_count_linear(xs, W) == pytest.approx(q["sparse_sparse_factor"])


def test_packed_product_equals_dense():
    """The multiply/route/sum of Section 3.2 done literally on the packed
    form (loop over non-zero activations, route each product by kernel id)
    reaches the oracle's dense result exactly."""
    r = rng(31)
    W = complementary_weights(r, r, 24, 60, 4, "int8")
    x = sparse_rows(r, 5, 60, 9, "u1_127")
    b = r.integers(-1000, 1001, size=24).astype(np.int32)
    val, kid, _ = o.pack(W, 4)
    y = np.tile(b.astype(np.int64), (5, 1))
    products = 0
    for bi in range(5):
        for i in np.nonzero(x[bi])[0]:
            for g in range(6):
                y[bi, g * 4 + kid[i, g]] += int(x[bi, i]) * int(val[i, g])
                products += 1
    assert np.array_equal(o.linear(x, W, b), y)
    # Figure 1 / Section 3.2: one product per (non-zero activation, non-zero
    # weight) pair and no other; with covering sets that is nnz(x) * G
    assert products == o.pair_count_linear(x, W) == int((x != 0).sum()) * 6


@pytest.mark.parametrize("cid", [1, 3, 5])
def test_config_product_counts_match_closed_form(cid):
    """The products a sparse-sparse layer needs (the oracle's pair count) equal
    the closed form: sum over rows of nnz(x) * G (covering sets), summed over
    the output pixels' windows for a convolution."""
    cfg = CONFIGS[cid]
    inp = generate(cfg, batch=2)
    spec = cfg.layers[0]
    x = inp["x"]
    W = inp["W"][0]
    if spec.kind == "linear":
        assert o.pair_count_linear(x, W.reshape(spec.c_out, -1)) == \
            int((x != 0).sum()) * spec.groups
    else:
        B, H, Wd, C = x.shape
        nnz = (x != 0).sum(axis=3)
        Ho = (H + 2 * spec.pad - spec.kh) // spec.stride + 1
        Wo = (Wd + 2 * spec.pad - spec.kw) // spec.stride + 1
        win = 0
        for ho in range(Ho):
            for wo in range(Wo):
                for ky in range(spec.kh):
                    for kx in range(spec.kw):
                        hy, wx = ho * spec.stride + ky - spec.pad, wo * spec.stride + kx - spec.pad
                        if 0 <= hy < H and 0 <= wx < Wd:
                            win += int(nnz[:, hy, wx].sum())
        assert o.pair_count_conv(x, W, spec.stride, spec.pad) == win * spec.groups


# ---------------------------------------------------------------- configs
def test_gsc_shapes_and_parameter_count():
    """Section 4 / Table 1: shapes of the keyword-spotting CNN and its
    2,522,128 dense parameters (weights of all four layers + conv biases)."""
    p = PAPER["gsc_parameters"]
    cfg = CONFIGS[2]
    L = cfg.layers
    weights = sum(l.c_out * l.r for l in L)
    conv_bias = sum(l.c_out for l in L if l.kind == "conv")
    assert weights + conv_bias == p["parameters"]
    x = np.zeros((1,) + cfg.in_shape, dtype=np.int8)
    assert list(x.shape[1:]) == p["shapes"]["input"]
    y1 = o.conv2d_nhwc(x, np.zeros((64, 5, 5, 1), np.int8))
    assert list(y1.shape[1:]) == p["shapes"]["conv1"]
    y1p = o.maxpool2x2_nhwc(y1)
    assert list(y1p.shape[1:]) == p["shapes"]["pool1"]
    y2 = o.conv2d_nhwc(y1p, np.zeros((64, 5, 5, 64), np.int8))
    assert list(y2.shape[1:]) == p["shapes"]["conv2"]
    y2p = o.maxpool2x2_nhwc(y2)
    assert list(y2p.shape[1:]) == p["shapes"]["pool2"]
    assert y2p.size == p["shapes"]["flatten"] == L[2].c_in
    assert L[2].c_out == p["shapes"]["linear1"] and L[3].c_out == p["shapes"]["output"]


def test_requant_shifts_frozen():
    """The frozen shifts equal what the oracle derives from the seeded batch."""
    import importlib.util
    spec = importlib.util.spec_from_file_location("mk", os.path.join(GOLD, "make_requant_shifts.py"))
    mk = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mk)
    stored = json.load(open(os.path.join(GOLD, "requant_shifts.json")))
    for cid, shifts in stored.items():
        assert mk.derive(int(cid)) == shifts
        for l in CONFIGS[int(cid)].layers:
            if l.shift is not None:
                assert shifts[l.name] == l.shift


def test_generator_properties_and_determinism():
    for cid in (1, 3, 5):
        cfg = CONFIGS[cid]
        a = generate(cfg)
        b = generate(cfg)
        assert tensor_digest(a["x"]) == tensor_digest(b["x"])
        x = a["x"].reshape(-1, cfg.in_shape[-1])
        assert ((x != 0).sum(axis=1) == cfg.in_nnz).all()
        for spec, W in zip(cfg.layers, a["W"]):
            W2 = W.reshape(spec.c_out, -1)
            assert ((W2 != 0).sum(axis=1) == spec.nnz_k).all()
            _, _, holes = o.pack(W2, spec.n)
            assert holes == 0
    x2 = generate(CONFIGS[2])["x"]
    assert x2.min() >= -127 and x2.max() <= 127


def test_chain_runner_int_config1():
    cfg = CONFIGS[1]
    inp = generate(cfg)
    res = networks.run_chain(cfg.layers, inp["x"], inp["W"], inp["b"])
    acc = o.linear(inp["x"], inp["W"][0], inp["b"][0])
    assert np.array_equal(res[0]["acc"], acc)
    assert (res[0]["win"].sum(axis=1) == 16).all()
    assert np.abs(acc).max() < 2 ** 31


def test_requant_shift_rule():
    assert networks.requant_shift(np.array([127, -127])) == 0
    assert networks.requant_shift(np.array([128])) == 1
    assert networks.requant_shift(np.array([-255, 3])) == 1
    assert networks.requant_shift(np.array([256])) == 2


def test_compact_rows_brute_force():
    r = rng(32)
    x = r.integers(-3, 4, size=(9, 13)).astype(np.int8)
    xf = np.where(r.random((4, 7)) < 0.5, 0.0, r.normal(size=(4, 7))).astype(np.float32)
    xf[0, 0] = -0.0
    for arr in (x, xf):
        res = o.compact_rows(arr)
        for row, (ii, vv) in zip(arr, res):
            exp_i = [j for j in range(len(row)) if row[j] != 0]
            assert list(ii) == exp_i
            assert [row[j] for j in exp_i] == list(vv)
