"""C ABI checks that need no GPU: exports, host pack, argument validation.

There is no GPU in the build container, so any HIP call made by an entry
point would come back as CS_ERR_DEVICE.  Getting the specific validation code
instead shows that every check runs on the host before the first HIP call.
"""
from __future__ import annotations

import ctypes
import os
import re

import numpy as np
import pytest

from oracle import cs_oracle as o
from paper_2112_13896_amd import _lib, ops
from paper_2112_13896_amd._lib import (CS_ERR_ARG, CS_ERR_COLLISION, CS_ERR_DTYPE, CS_ERR_SHAPE,
                                       CS_ERR_WORKSPACE, CS_F32, CS_I8, CS_I32, CS_OK)
from workloads import complementary_weights

HEADER = os.path.join(os.path.dirname(__file__), "..", "include", "cs.h")
FAKE = 0x10000          # a non-null address that must never be dereferenced
FAKE_WS = 0x100000      # 256-aligned fake workspace


@pytest.fixture(scope="module")
def L():
    return _lib.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:int|size_t|const char\*)\s+(cs_\w+)\s*\(", text, flags=re.M)))


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert set(names) == set(_lib.SIGNATURES), names
    for nm in names:
        assert hasattr(L, nm)


def test_status_strings(L):
    for code in range(0, -8, -1):
        s = _lib.status_str(code)
        assert s and s != "unknown status"
    assert _lib.status_str(5) == "unknown status"


def test_counting_build_exports_every_declared_symbol():
    """The counting build (libcs_count.so) is the same ABI; in the product
    build the counter is absent and says so without touching a device."""
    C = _lib._load(_lib.COUNT_LIB_PATH)
    for nm in declared_functions():
        assert hasattr(C, nm)
    v = ctypes.c_ulonglong(7)
    assert _lib.lib().cs_product_count(ctypes.byref(v), 1) == _lib.CS_ERR_UNSUPPORTED
    assert v.value == 0
    with pytest.raises(_lib.CSError):
        _lib.product_count()


def test_stamping_build_exports_every_declared_symbol():
    """The stamping build (libcs_stamps.so) is the same ABI; the other builds
    have no phase stamps and say so without touching a device, and the
    argument check comes first in the stamping build."""
    S = _lib._load(_lib.STAMP_LIB_PATH)
    for nm in declared_functions():
        assert hasattr(S, nm)
    acc = (ctypes.c_ulonglong * 32)()
    khz = ctypes.c_int(5)
    assert _lib.lib().cs_phase_stamps(acc, 32, 0, ctypes.byref(khz)) == _lib.CS_ERR_UNSUPPORTED
    assert khz.value == 0
    C = _lib._load(_lib.COUNT_LIB_PATH)
    assert C.cs_phase_stamps(acc, 32, 0, None) == _lib.CS_ERR_UNSUPPORTED
    assert S.cs_phase_stamps(acc, 33, 0, None) == _lib.CS_ERR_ARG
    assert S.cs_phase_stamps(None, 4, 0, None) == _lib.CS_ERR_ARG
    with pytest.raises(_lib.CSError):
        _lib.phase_stamps()


@pytest.mark.parametrize("dtype", ["int8", "float32"])
def test_pack_matches_oracle(dtype):
    r = np.random.default_rng(3)
    for d_out, R, n in [(64, 512, 8), (1500, 1600, 20), (12, 1500, 1), (64, 1600, 16), (9, 7, 3)]:
        if R % n:
            W = r.integers(-5, 6, size=(d_out, R)).astype(dtype)
            W[:, :] = 0
            for g in range(d_out // n):          # disjoint but not covering: holes
                for i in range(R):
                    j = r.integers(0, n + 1)
                    if j < n:
                        W[g * n + j, i] = r.integers(1, 100)
        else:
            W = complementary_weights(r, r, d_out, R, n, "int8" if dtype == "int8" else "normal")
        aug, holes = ops.pack(W, n)
        v2, k2, h2 = o.pack(W, n)
        assert holes == h2
        # augmented entry layout: int8 -> uint8(value) | kid << 8; fp32 -> (value bits, kid)
        if W.dtype == np.int8:
            assert aug.dtype == np.uint16
            want = v2.view(np.uint8).astype(np.uint16) | (k2.astype(np.uint16) << 8)
            assert np.array_equal(aug, want)
        else:
            assert aug.dtype == np.uint32 and aug.shape == v2.shape + (2,)
            assert np.array_equal(aug[..., 0], v2.astype(np.float32).view(np.uint32))
            assert np.array_equal(aug[..., 1], k2.astype(np.uint32))
        val, kid = ops.unpack_aug(aug)
        assert np.array_equal(val, v2) and np.array_equal(kid, k2)


def test_pack_collision_reports_first_offender():
    W = np.zeros((6, 10), dtype=np.int8)
    W[3, 4] = 1
    W[5, 4] = 2      # group 1 collides at slot 4
    W[4, 9] = 1
    W[3, 9] = 1      # group 1 collides at slot 9 too (later)
    with pytest.raises(_lib.CSError) as e:
        ops.pack(W, 3)
    assert e.value.status == CS_ERR_COLLISION and e.value.bad == (1, 4)
    with pytest.raises(o.PackCollision) as e2:
        o.pack(W, 3)
    assert (e2.value.g, e2.value.i) == (1, 4)


def test_pack_argument_errors(L):
    w = np.ones((4, 4), dtype=np.int8)
    out = np.zeros(64, dtype=np.uint16)
    p = lambda *a: L.cs_pack(*a)  # noqa: E731
    assert p(CS_I8, None, 4, 4, 2, out.ctypes.data, None, None, None) == CS_ERR_ARG
    assert p(CS_I8, w.ctypes.data, 4, 4, 2, None, None, None, None) == CS_ERR_ARG
    assert p(CS_I8, w.ctypes.data, 4, 4, 3, out.ctypes.data, None, None, None) == CS_ERR_SHAPE
    assert p(CS_I8, w.ctypes.data, 4, 4, 0, out.ctypes.data, None, None, None) == CS_ERR_ARG
    assert p(CS_I32, w.ctypes.data, 4, 4, 2, out.ctypes.data, None, None, None) == CS_ERR_DTYPE
    assert p(CS_I8, w.ctypes.data, 64, 4, 64, out.ctypes.data, None, None, None) == CS_ERR_SHAPE
    assert p(CS_I8, w.ctypes.data, 4, 0, 2, out.ctypes.data, None, None, None) == CS_ERR_ARG


def test_compact_validation(L):
    c = L.cs_compact
    assert c(CS_I32, FAKE, 4, 8, FAKE, FAKE, FAKE, None) == CS_ERR_DTYPE
    assert c(CS_I8, FAKE, -1, 8, FAKE, FAKE, FAKE, None) == CS_ERR_ARG
    assert c(CS_I8, FAKE, 4, 0, FAKE, FAKE, FAKE, None) == CS_ERR_ARG
    assert c(CS_I8, FAKE, 4, 70000, FAKE, FAKE, FAKE, None) == CS_ERR_SHAPE
    assert c(CS_F32, None, 4, 8, FAKE, FAKE, FAKE, None) == CS_ERR_ARG
    assert c(CS_F32, FAKE, 4, 8, FAKE, FAKE, None, None) == CS_ERR_ARG
    assert c(CS_F32, None, 0, 8, None, None, None, None) == CS_OK       # empty: nothing launched


def conv_args(**kw):
    a = dict(xt=CS_I8, x=FAKE, b=2, h=8, w=8, c_in=4, kh=3, kw=3, stride=1, pad=1, aug=FAKE,
             c_out=8, n=4, bias=None, pool=1, y=FAKE, ws=FAKE_WS, ws_bytes=1 << 30,
             stream=None)
    a.update(kw)
    return list(a.values())


def test_conv2d_validation(L):
    f = L.cs_conv2d
    assert f(*conv_args(xt=CS_I32)) == CS_ERR_DTYPE
    assert f(*conv_args(b=0)) == CS_ERR_ARG
    assert f(*conv_args(stride=0)) == CS_ERR_ARG
    assert f(*conv_args(pad=-1)) == CS_ERR_ARG
    assert f(*conv_args(n=3)) == CS_ERR_SHAPE                  # 3 does not divide 8
    assert f(*conv_args(n=40, c_out=80)) == CS_ERR_SHAPE       # n > CS_MAX_N
    assert f(*conv_args(c_in=70000)) == CS_ERR_SHAPE
    assert f(*conv_args(kh=11, pad=1)) == CS_ERR_SHAPE         # window larger than padded input
    assert f(*conv_args(pool=3)) == CS_ERR_ARG
    assert f(*conv_args(pool=2, h=7, w=7)) == CS_ERR_SHAPE     # odd conv output
    assert f(*conv_args(x=None)) == CS_ERR_ARG
    assert f(*conv_args(aug=None)) == CS_ERR_ARG
    assert f(*conv_args(y=None)) == CS_ERR_ARG
    need = L.cs_workspace_bytes(1, CS_I8, 2 * 8 * 8, 4)
    assert f(*conv_args(ws_bytes=need - 1)) == CS_ERR_WORKSPACE
    assert f(*conv_args(ws=None)) == CS_ERR_WORKSPACE
    assert f(*conv_args(ws=FAKE_WS + 8)) == CS_ERR_WORKSPACE   # misaligned


def test_conv2d_noalloc_validation(L):
    """Host checks of the entry point without a workspace, including the
    scratch limit; all are refused before any HIP call."""
    f = L.cs_conv2d_noalloc

    def args(**kw):
        a = conv_args(**kw)
        del a[17:19]                                  # no ws, ws_bytes
        return a
    assert f(*args(xt=CS_I32)) == CS_ERR_DTYPE
    assert f(*args(b=0)) == CS_ERR_ARG
    assert f(*args(n=3)) == CS_ERR_SHAPE
    assert f(*args(pool=2, h=7, w=7)) == CS_ERR_SHAPE
    assert f(*args(x=None)) == CS_ERR_ARG
    assert f(*args(y=None)) == CS_ERR_ARG
    # lists of more rows than the scratch holds
    per_row = 64 * (2 + 4) + 4
    rows = _lib.CS_NOALLOC_SCRATCH_BYTES // per_row + 4096
    assert L.cs_workspace_bytes(1, CS_F32, rows, 64) > _lib.CS_NOALLOC_SCRATCH_BYTES
    assert f(*args(xt=CS_F32, b=1, h=rows, w=1, c_in=64, kh=1, kw=1, pad=0, c_out=64,
                   n=8)) == CS_ERR_WORKSPACE


def test_conv2d_dense_validation(L):
    f = L.cs_conv2d_dense
    ok = dict(xt=CS_I8, x=FAKE, b=2, h=32, w=32, c_in=1, kh=5, kw=5, stride=1, pad=0, aug=FAKE,
              c_out=64, n=1, bias=None, pool=2, y=FAKE, stream=None)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return f(*a.values())
    assert call(xt=CS_I32) == CS_ERR_DTYPE
    assert call(n=2) == CS_ERR_SHAPE              # only dense kernels (n == 1)
    assert call(c_out=32) == CS_ERR_SHAPE         # one wavefront of 64 channels
    assert call(c_in=2) == CS_ERR_SHAPE           # 50 weights per channel > 32
    assert call(kh=7, kw=7) == CS_ERR_SHAPE
    assert call(x=None) == CS_ERR_ARG
    assert call(aug=None) == CS_ERR_ARG
    assert call(pool=2, h=33, w=33) == CS_ERR_SHAPE


def _reorder_eval(x, table, kh, kw, pad, bias):
    """The reordering kernel's sums, evaluated on the CPU in float64 from the
    table: each output tile's zero-padded input halo laid out as the kernel
    stages it (rows of tile + kw - 1 pixels of c_in + 1 words), every output
    the sum of halo[pixel offset + table offset] * value over its entries."""
    T = 8
    b, h, w, c = x.shape
    ho, wo = h + 2 * pad - kh + 1, w + 2 * pad - kw + 1
    hw, hh, cp = T + kw - 1, T + kh - 1, c + 1
    off = table[..., 0] // 4
    val = table[..., 1].copy().view(np.float32).astype(np.float64)
    y = np.zeros((b, ho, wo, table.shape[0]))
    for bi in range(b):
        for ty in range(0, ho, T):
            for tx in range(0, wo, T):
                halo = np.zeros((hh, hw, cp))
                for yy in range(hh):
                    for xx in range(hw):
                        iy, ix = ty + yy - pad, tx + xx - pad
                        if 0 <= iy < h and 0 <= ix < w:
                            halo[yy, xx, :c] = x[bi, iy, ix]
                flat = halo.reshape(-1)
                for py in range(min(T, ho - ty)):
                    for px in range(min(T, wo - tx)):
                        base = (py * hw + px) * cp
                        y[bi, ty + py, tx + px] = (flat[base + off] * val).sum(axis=1)
    if bias is not None:
        y += bias
    return y


def test_reorder_table_lists_each_support():
    """Every output's table entries are exactly its kernel's non-zero weights,
    each once, with the slot's (ky, kx, c) recoverable from the offset."""
    r = np.random.default_rng(11)
    for c_out, kh, kw, c_in, n in [(64, 3, 3, 64, 8), (64, 1, 1, 30, 2), (64, 5, 5, 16, 2)]:
        W = complementary_weights(r, r, c_out, kh * kw * c_in, n, "normal")
        aug, _ = ops.pack(W, n)
        t = ops.reorder_table(aug, kh, kw, c_in, c_out, n)
        hw, cp = 8 + kw - 1, c_in + 1
        longest = max(np.count_nonzero(W, axis=1).max(), 1)
        assert t.shape[0] == c_out and t.shape[1] == (longest + 7) // 8 * 8
        for oi in range(c_out):
            got = {}
            for off, vb in t[oi]:
                v = np.array([vb], np.int32).view(np.float32)[0]
                if v == 0:
                    assert off == 0                    # padding
                    continue
                wrd = off // 4
                pix, ch = divmod(wrd, cp)
                ky, kx = divmod(pix, hw)
                slot = (ky * kw + kx) * c_in + ch
                assert slot not in got
                got[slot] = v
            want = {i: W[oi, i] for i in np.flatnonzero(W[oi])}
            assert got == want


def test_reorder_table_sums_match_oracle():
    """The table evaluated the way the kernel reads it (tile halos in its LDS
    layout) gives the oracle's convolution, including ragged edge tiles."""
    r = np.random.default_rng(12)
    for shape, kh, pad, n in [((1, 11, 13, 16), 3, 1, 4), ((2, 9, 10, 8), 5, 2, 2)]:
        b, h, w, c = shape
        x = np.where(r.random(shape) < 0.2, np.abs(r.normal(size=shape)), 0).astype(np.float32)
        W = complementary_weights(r, r, 64, kh * kh * c, n, "normal").reshape(64, kh, kh, c)
        bias = r.normal(size=64).astype(np.float32)
        aug, _ = ops.pack(W.reshape(64, -1), n)
        t = ops.reorder_table(aug, kh, kh, c, 64, n)
        np.testing.assert_allclose(_reorder_eval(x, t, kh, kh, pad, bias),
                                   o.conv2d_nhwc(x, W, 1, pad, bias), rtol=1e-12, atol=1e-12)


def test_pack_blocks_matches_oracle():
    from workloads import block_complementary_weights
    r = np.random.default_rng(15)
    for d_out, R, n, b, dt in [(64, 147, 4, 3, np.float32), (12, 40, 3, 4, np.int8)]:
        W = block_complementary_weights(r, r, d_out, R, n, b)
        if dt == np.int8:
            W = (np.sign(W) * r.integers(1, 128, size=W.shape)).astype(np.int8)
        W[:n, :b] = 0                                     # a hole: block 0 of set 0
        aug, kidb, holes = ops.pack_blocks(W, n, b)
        val, okidb, oholes = o.pack_blocks(W, n, b)
        assert holes == oholes == 1
        assert np.array_equal(kidb, okidb)
        v, kid = ops.unpack_aug(aug)
        assert np.array_equal(v, val)
    W = block_complementary_weights(r, r, 8, 12, 2, 3)
    W[1, 4] = 0                                           # kernel 1 splits block 1
    if not (W[1, 3:6] != 0).any():
        W[1, 3] = 1.0
    with pytest.raises(_lib.CSError) as e:
        ops.pack_blocks(W, 2, 3)
    assert e.value.status == CS_ERR_SHAPE
    W = block_complementary_weights(r, r, 8, 12, 2, 3)
    owner = int(np.nonzero(W[:2, 0])[0][0])
    W[1 - owner, 0:3] = 2.0                               # both kernels of set 0 own block 0
    with pytest.raises(_lib.CSError) as e:
        ops.pack_blocks(W, 2, 3)
    assert e.value.status == CS_ERR_COLLISION and e.value.bad == (0, 0)


def test_pack_channels_matches_oracle():
    from workloads import channel_complementary_weights
    r = np.random.default_rng(13)
    for c_out, kh, kw, c, n in [(8, 3, 3, 12, 3), (4, 5, 5, 10, 5), (3, 1, 2, 6, 2)]:
        W4 = channel_complementary_weights(r, r, c_out, kh, kw, c, n)
        W4[0, 0, 0, :] = 0                                # a few holes
        packed, holes = ops.pack_channels(W4, n)
        val, cid, oh = o.pack_channels(W4, n)
        assert holes == oh
        assert np.array_equal(packed[..., 0].view(np.float32), val)
        assert np.array_equal(packed[..., 1], cid.astype(np.uint32))
    W4 = channel_complementary_weights(r, r, 2, 3, 3, 6, 3)
    W4[1, 2, 0, 4] = 1.0                                  # a second channel of group 1 at tap (2, 0)
    if W4[1, 2, 0, 3] == 0 and W4[1, 2, 0, 5] == 0:
        W4[1, 2, 0, 5] = 2.0
    with pytest.raises(_lib.CSError) as e:
        ops.pack_channels(W4, 3)
    assert e.value.status == CS_ERR_COLLISION and e.value.bad == (1, (1 * 3 + 2) * 3 + 0)


def test_reorder_table_channels_sums_match_oracle():
    """A channel-overlaid layer's table, evaluated the way the reordering
    kernel reads it, gives the oracle's convolution of the dense filters."""
    from workloads import channel_complementary_weights
    r = np.random.default_rng(14)
    for shape, kh, pad, n in [((1, 9, 11, 12), 3, 1, 3), ((1, 8, 7, 10), 5, 2, 5)]:
        b, h, w, c = shape
        x = np.where(r.random(shape) < 0.3, np.abs(r.normal(size=shape)), 0).astype(np.float32)
        W4 = channel_complementary_weights(r, r, 64, kh, kh, c, n)
        packed, _ = ops.pack_channels(W4, n)
        t = ops.reorder_table_channels(packed, kh, kh, c, 64, n)
        assert t.shape[1] == (kh * kh * c // n + 7) // 8 * 8
        np.testing.assert_allclose(_reorder_eval(x, t, kh, kh, pad, None),
                                   o.conv2d_nhwc(x, W4, 1, pad, None), rtol=1e-12, atol=1e-12)


def _int8_channel_weights(r, c_out, kh, kw, c, n):
    from workloads import channel_complementary_weights
    mask = channel_complementary_weights(r, r, c_out, kh, kw, c, n) != 0
    vals = r.integers(1, 128, size=mask.shape) * r.choice([-1, 1], size=mask.shape)
    return np.where(mask, vals, 0).astype(np.int8)


def _channel_eval(x, table, kh, kw, stride, pad, c_out):
    """The int8 channel kernel's indexing on the CPU: per 64-pixel segment of
    an output row, the staged tile [kh][63*stride + kw][cp] bytes (zero
    outside the image); output pixel p of the segment reads byte
    p*stride*cp + off of it for every slot offset of its filter's row and
    multiplies it by the slot's weight byte (little-endian in the weight
    words after the offsets)."""
    b, h, w, c = x.shape
    ho, wo = (h + 2 * pad - kh) // stride + 1, (w + 2 * pad - kw) // stride + 1
    sw = 63 * stride + kw
    cp = c if (c // 4) % 2 == 1 else c + 4
    s4 = table.shape[1] // 5
    off = table[:, :4 * s4].astype(np.int64)
    wt = np.ascontiguousarray(table[:, 4 * s4:]).view(np.uint8).reshape(c_out, 4 * s4)
    wt = wt.view(np.int8).astype(np.int64)
    y = np.zeros((b, ho, wo, c_out), dtype=np.int64)
    for bi in range(b):
        for oy in range(ho):
            for ox0 in range(0, wo, 64):
                tile = np.zeros((kh, sw, cp), dtype=np.int64)
                for ky in range(kh):
                    iy = oy * stride - pad + ky
                    for px in range(sw):
                        ix = ox0 * stride - pad + px
                        if 0 <= iy < h and 0 <= ix < w:
                            tile[ky, px, :c] = x[bi, iy, ix]
                flat = tile.reshape(-1)
                for p_ in range(min(64, wo - ox0)):
                    g = flat[p_ * stride * cp + off]          # [c_out][S]
                    y[bi, oy, ox0 + p_] = (g * wt).sum(axis=1)
    return y


def test_channel_table_int8_matches_oracle():
    """int8 channel-dimension overlay: cs_pack_channels (CS_I8) matches the
    oracle's pack, and its cs_channel_table, read the way cs_conv2d_channels
    reads it, gives the oracle's convolution of the dense filters exactly."""
    r = np.random.default_rng(17)
    for shape, kh, stride, pad, n, c_out in [((1, 9, 11, 12), 3, 1, 1, 3, 16),
                                             ((2, 10, 9, 24), 3, 2, 1, 3, 32),
                                             ((1, 8, 70, 8), 1, 1, 0, 1, 16)]:
        W4 = _int8_channel_weights(r, c_out, kh, kh, shape[3], n)
        packed, holes = ops.pack_channels(W4, n)
        val, cid, oh = o.pack_channels(W4, n)
        assert packed.dtype == np.uint16 and holes == oh
        assert np.array_equal((packed & 0xFF).astype(np.uint8).view(np.int8), val)
        assert np.array_equal(packed >> 8, cid.astype(np.uint16))
        t = ops.channel_table(packed, kh, kh, shape[3], c_out, n, stride)
        x = r.integers(-127, 128, size=shape).astype(np.int8)
        assert np.array_equal(_channel_eval(x, t, kh, kh, stride, pad, c_out),
                              o.conv2d_nhwc(x, W4, stride, pad, None))


def test_channels_validation(L):
    f = L.cs_conv2d_channels
    #       x     b  h   w   c   kh kw s  p  table c_out n  bias  y     stream
    base = [FAKE, 2, 16, 16, 48, 3, 3, 1, 1, FAKE, 64, 3, None, FAKE, None]

    def call(i, v):
        a = list(base)
        a[i] = v
        return f(*a)
    assert call(4, 50) == CS_ERR_SHAPE                          # c_in not a multiple of 4
    assert call(11, 5) == CS_ERR_SHAPE                          # n does not divide c_in
    assert call(10, 48) == CS_ERR_SHAPE                         # c_out not 16/32/64/128
    assert call(0, None) == CS_ERR_ARG
    assert call(9, None) == CS_ERR_ARG
    assert call(13, FAKE + 4) == CS_ERR_ARG                     # y not 16-byte aligned
    t = L.cs_channel_table
    assert t(None, 3, 3, 48, 64, 3, 1, FAKE) == CS_ERR_ARG
    bad = np.zeros((64, 16, 3, 3), dtype=np.uint16)
    bad[0, 0, 0, 0] = 3 << 8                                    # channel ID 3 with n = 3
    out = np.zeros((64, 5 * 36), dtype=np.int32)
    assert t(bad.ctypes.data, 3, 3, 48, 64, 3, 1, out.ctypes.data) == CS_ERR_ARG


def test_reorder_validation(L):
    f = L.cs_reorder_table
    sm = ctypes.c_int(0)
    assert f(None, 3, 3, 64, 64, 8, ctypes.byref(sm), None) == CS_ERR_ARG
    assert f(FAKE, 3, 3, 64, 64, 7, ctypes.byref(sm), None) == CS_ERR_SHAPE   # 7 does not divide 64
    assert f(FAKE, 3, 3, 64, 64, 40, ctypes.byref(sm), None) == CS_ERR_SHAPE  # n > CS_MAX_N
    pc = L.cs_pack_channels
    hz = ctypes.c_int64(0)
    assert pc(CS_I32, FAKE, 4, 3, 3, 6, 3, FAKE, ctypes.byref(hz), None, None) == CS_ERR_DTYPE
    assert pc(CS_F32, None, 4, 3, 3, 6, 3, FAKE, None, None, None) == CS_ERR_ARG
    assert pc(CS_F32, FAKE, 4, 3, 3, 6, 4, FAKE, None, None, None) == CS_ERR_SHAPE   # 4 does not divide 6
    tc = L.cs_reorder_table_channels
    assert tc(None, 3, 3, 6, 4, 3, ctypes.byref(sm), None) == CS_ERR_ARG
    assert tc(FAKE, 3, 3, 6, 4, 4, ctypes.byref(sm), None) == CS_ERR_SHAPE
    g = L.cs_conv2d_reorder_kwta
    ok = dict(xt=CS_F32, x=FAKE, b=1, h=8, w=8, c_in=64, kh=3, kw=3, pad=1, table=FAKE, smax=72,
              c_out=64, bias=None, y=FAKE, keep_sums=0, k=8, ot=CS_F32, out=None, oidx=FAKE,
              oval=FAKE, ocnt=FAKE, ocap=8, stream=None)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return g(*a.values())
    assert call(xt=CS_I8) == CS_ERR_DTYPE
    assert call(c_out=32) == CS_ERR_SHAPE
    assert call(c_in=65) == CS_ERR_SHAPE
    assert call(k=40, ocap=40) == CS_ERR_SHAPE      # 32 < k < c_out
    assert call(ocap=6) == CS_ERR_SHAPE             # not a multiple of 4
    assert call(ocap=4) == CS_ERR_SHAPE             # < k
    assert call(table=None) == CS_ERR_ARG
    assert call(smax=70) == CS_ERR_SHAPE            # not a multiple of 8
    assert call(out=FAKE) == CS_ERR_ARG             # both output forms
    assert call(oidx=None, oval=None, ocnt=None, ocap=0) == CS_ERR_ARG   # neither
    assert call(y=FAKE + 4) == CS_ERR_ARG           # y not 16-byte aligned


def test_chain2_validation(L):
    f = L.cs_mrs_kwta_chain2
    ok = dict(xt=CS_I8, idx=FAKE, lval=FAKE, cnt=FAKE, cap=8, b=4, h=5, w=5, c_in=64, kh=5, kw=5,
              stride=1, pad=0, aug=FAKE, c_out=1500, n=20, bias=None, pool=1, y=FAKE, keep_sums=0,
              k=75, ot=CS_I8, shift=8, oidx=FAKE, oval=FAKE, ocnt=FAKE, ocap=76, aug2=FAKE,
              c_out2=12, n2=1, bias2=None, y2=FAKE, stream=None)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return f(*a.values())
    assert call(xt=CS_F32) == CS_ERR_DTYPE
    assert call(ot=CS_I32) == CS_ERR_DTYPE
    assert call(aug2=None) == CS_ERR_ARG
    assert call(y2=None) == CS_ERR_ARG
    assert call(oidx=None) == CS_ERR_ARG            # list output only
    assert call(n2=5) == CS_ERR_SHAPE               # 5 does not divide 12
    assert call(kh=3, kw=3) == CS_ERR_SHAPE         # a 3 x 3 output map: not one vector per sample
    assert call(k=80) == CS_ERR_SHAPE               # more winners than the list holds
    assert call(shift=40) == CS_ERR_ARG


def test_chain3_validation(L):
    f = L.cs_mrs_kwta_chain3
    ok = dict(xt=CS_I8, idx=FAKE, lval=FAKE, cnt=FAKE, cap=8, b=4, h=14, w=14, c_in=64, kh=5,
              kw=5, stride=1, pad=0, aug=FAKE, c_out=64, n=16, bias=None, pool=2, y=FAKE,
              keep_sums=0, k=8, ot=CS_I8, shift=9, oidx=FAKE, oval=FAKE, ocnt=FAKE, ocap=8,
              aug2=FAKE, c_out2=1500, n2=20, bias2=None, y2=FAKE, k2=75, shift2=8, oidx2=FAKE,
              oval2=FAKE, ocnt2=FAKE, ocap2=76, aug3=FAKE, c_out3=12, n3=1, bias3=None, y3=FAKE,
              stream=None)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return f(*a.values())
    assert call(xt=CS_F32) == CS_ERR_DTYPE
    assert call(ot=CS_I32) == CS_ERR_DTYPE
    for name in ("idx", "aug", "oidx", "aug2", "y2", "oidx2", "ocnt2", "aug3", "y3"):
        assert call(**{name: None}) == CS_ERR_ARG, name
    assert call(k=-1) == CS_ERR_ARG
    assert call(shift2=32) == CS_ERR_ARG
    assert call(keep_sums=2) == CS_ERR_ARG
    assert call(k=9) == CS_ERR_SHAPE                # more winners than the first list holds
    assert call(k2=80) == CS_ERR_SHAPE              # more winners than the second list holds
    assert call(n2=7) == CS_ERR_SHAPE               # 7 does not divide 1500
    assert call(n3=5) == CS_ERR_SHAPE               # 5 does not divide 12
    assert call(ocap2=0) == CS_ERR_SHAPE


def test_dense_chain3_validation(L):
    f = L.cs_conv2d_dense_kwta_chain3
    ok = dict(xt=CS_I8, x=FAKE, b=4, h=32, w=32, c_in=1, kh=5, kw=5, stride=1, pad=0, aug=FAKE,
              c_out=64, n=1, bias=None, pool=2, y=FAKE, keep_sums=0, k=8, ot=CS_I8, shift=11,
              oidx=FAKE, oval=FAKE, ocnt=FAKE, ocap=8, kh2=5, kw2=5, stride2=1, pad2=0, aug2=FAKE,
              c_out2=64, n2=16, bias2=None, pool2=2, y2=FAKE, k2=8, shift2=9, oidx2=FAKE,
              oval2=FAKE, ocnt2=FAKE, ocap2=8, aug3=FAKE, c_out3=1500, n3=20, bias3=None, y3=FAKE,
              k3=75, shift3=8, oidx3=FAKE, oval3=FAKE, ocnt3=FAKE, ocap3=76, aug4=FAKE, c_out4=12,
              n4=1, bias4=None, y4=FAKE, stream=None)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return f(*a.values())
    assert call(xt=CS_F32) == CS_ERR_DTYPE
    assert call(ot=CS_I32) == CS_ERR_DTYPE
    for name in ("x", "aug", "oidx", "aug2", "oidx2", "y3", "ocnt3", "aug4", "y4"):
        assert call(**{name: None}) == CS_ERR_ARG, name
    assert call(k3=-1) == CS_ERR_ARG
    assert call(shift3=32) == CS_ERR_ARG
    assert call(n=2) == CS_ERR_SHAPE                # the first layer is dense (n == 1)
    assert call(c_out=32, c_out2=32) == CS_ERR_SHAPE   # the first layer has 64 outputs
    assert call(kh=7, kw=7) == CS_ERR_SHAPE         # 49 slots > 32
    assert call(k=9) == CS_ERR_SHAPE                # more winners than the first list holds
    assert call(k3=80) == CS_ERR_SHAPE
    assert call(n4=5) == CS_ERR_SHAPE               # 5 does not divide 12


def test_mrs_and_linear_validation(L):
    m = L.cs_mrs_conv2d
    base = [CS_F32, FAKE, FAKE, FAKE, 4, 2, 8, 8, 4, 3, 3, 1, 1, FAKE, 8, 4, None, 1, FAKE, None]
    assert m(*base[:4], 0, *base[5:]) == CS_ERR_SHAPE          # list capacity 0
    bad = list(base)
    bad[1] = None
    assert m(*bad) == CS_ERR_ARG
    bad = list(base)
    bad[13] = None                                              # no augmented tensor
    assert m(*bad) == CS_ERR_ARG
    bad = list(base)
    bad[0] = CS_I32
    assert m(*bad) == CS_ERR_DTYPE
    lin = L.cs_linear
    assert lin(CS_I8, FAKE, 16, 512, FAKE, 64, 7, None, FAKE, FAKE_WS, 1 << 30, None) == CS_ERR_SHAPE
    assert lin(CS_I8, FAKE, 0, 512, FAKE, 64, 8, None, FAKE, FAKE_WS, 1 << 30, None) == CS_ERR_ARG
    assert lin(CS_I8, FAKE, 16, 512, FAKE, 64, 8, None, FAKE, FAKE_WS, 10, None) == CS_ERR_WORKSPACE
    assert lin(CS_F32, FAKE, 16, 512, None, 64, 8, None, FAKE, FAKE_WS, 1 << 30, None) == CS_ERR_ARG


def test_units_validation(L):
    """cs_mrs_kwta_units_conv2d rejects bad arguments on the host, before any
    device call."""
    u = L.cs_mrs_kwta_units_conv2d
    #      xt      idx   lval  cnt  cap b  h  w  cin kh kw s  p  aug   c_out n  bias pool y
    base = [CS_F32, FAKE, FAKE, FAKE, 8, 2, 8, 8, 16, 3, 3, 1, 1, FAKE, 64, 8, None, 1, FAKE,
            1, 4, 16, None, FAKE, FAKE, FAKE, 16, None]
    #       keep k unit out  oidx oval  ocnt  ocap stream

    def call(**kw):
        a = list(base)
        pos = {"xt": 0, "idx": 1, "cap": 4, "c_out": 14, "k": 20, "unit": 21, "out": 22,
               "oidx": 23, "ocap": 26}
        for key, v in kw.items():
            a[pos[key]] = v
        return u(*a)
    assert call(unit=24) == CS_ERR_SHAPE                        # does not divide c_out
    assert call(k=17) == CS_ERR_SHAPE                           # k > unit
    assert call(ocap=15) == CS_ERR_SHAPE                        # 4 units x 4 winners
    assert call(xt=CS_I8) == CS_ERR_DTYPE                       # units: fp32 only
    assert call(idx=None) == CS_ERR_ARG
    assert call(out=FAKE) == CS_ERR_ARG                         # both output forms
    assert call(oidx=None) == CS_ERR_ARG                        # neither output form
    assert call(cap=0) == CS_ERR_SHAPE
    assert call(unit=0) == CS_ERR_SHAPE


def test_dense_blocks_validation(L):
    """cs_conv2d_dense_blocks rejects bad arguments on the host."""
    f = L.cs_conv2d_dense_blocks
    #       x     b  h   w   c  kh kw s  p  aug   kidb  c_out n bias y     stream
    base = [FAKE, 2, 32, 32, 3, 7, 7, 2, 3, FAKE, FAKE, 64, 4, None, FAKE, None]

    def call(i, v):
        a = list(base)
        a[i] = v
        return f(*a)
    assert call(4, 5) == CS_ERR_SHAPE                           # a block is at most 4 channels
    assert call(12, 3) == CS_ERR_SHAPE                          # n does not divide c_out
    assert call(0, None) == CS_ERR_ARG
    assert call(10, None) == CS_ERR_ARG                         # no block Kernel IDs
    assert call(14, None) == CS_ERR_ARG
    assert call(2, 0) == CS_ERR_ARG
    assert call(5, 40) == CS_ERR_SHAPE                          # window larger than the map
    # a 31 x 31 window with 32 sets: its table does not fit a workgroup's LDS
    assert f(FAKE, 2, 64, 64, 3, 31, 31, 1, 3, FAKE, FAKE, 64, 2, None, FAKE, None) == CS_ERR_SHAPE


def test_kwta_validation(L):
    k = L.cs_kwta
    assert k(CS_I8, FAKE, 4, 64, 8, CS_I8, 0, FAKE, None) == CS_ERR_DTYPE
    assert k(CS_F32, FAKE, 4, 64, 8, CS_I8, 0, FAKE, None) == CS_ERR_DTYPE
    assert k(CS_I32, FAKE, 4, 64, 8, CS_F32, 0, FAKE, None) == CS_ERR_DTYPE
    assert k(CS_I32, FAKE, 4, 64, 65, CS_I32, 0, FAKE, None) == CS_ERR_SHAPE
    assert k(CS_I32, FAKE, 4, 3000, 8, CS_I32, 0, FAKE, None) == CS_ERR_SHAPE
    assert k(CS_I32, FAKE, 4, 64, -1, CS_I32, 0, FAKE, None) == CS_ERR_ARG
    assert k(CS_I32, FAKE, 4, 0, 0, CS_I32, 0, FAKE, None) == CS_ERR_ARG
    assert k(CS_I32, FAKE, 4, 64, 8, CS_I8, 32, FAKE, None) == CS_ERR_ARG
    assert k(CS_I32, None, 4, 64, 8, CS_I8, 3, FAKE, None) == CS_ERR_ARG
    assert k(CS_I32, None, 0, 64, 8, CS_I8, 3, None, None) == CS_OK     # empty: nothing launched


def test_kwta_lists_validation(L):
    k = L.cs_kwta_lists
    ok = [CS_I32, FAKE, 4, 64, 8, CS_I8, 3, FAKE, FAKE, FAKE, 8, None]

    def call(**kw):
        a = list(ok)
        for i, v in kw.items():
            a[int(i[1:])] = v
        return k(*a)
    assert call(a0=CS_I8) == CS_ERR_DTYPE
    assert call(a0=CS_F32) == CS_ERR_DTYPE              # f32 input cannot requantise
    assert call(a10=7) == CS_ERR_SHAPE                  # capacity below k
    assert call(a10=0) == CS_ERR_ARG
    assert call(a4=65) == CS_ERR_SHAPE
    assert call(a7=None) == CS_ERR_ARG
    assert call(a6=40) == CS_ERR_ARG
    assert call(a2=0, a1=None, a7=None, a8=None, a9=None) == CS_OK


def test_workspace_bytes(L):
    def al(v):
        return (v + 255) // 256 * 256
    for op, xt, rows, c in [(0, CS_I8, 16, 512), (1, CS_F32, 100352, 64), (1, CS_I8, 262144, 1)]:
        es = 1 if xt == CS_I8 else 4
        exp = al(rows * c * 2) + al(rows * c * es) + al(rows * 4)
        assert L.cs_workspace_bytes(op, xt, rows, c) == exp
    assert L.cs_workspace_bytes(2, CS_I8, 4, 4) == 0
    assert L.cs_workspace_bytes(0, CS_I32, 4, 4) == 0
    assert L.cs_workspace_bytes(0, CS_I8, 4, 0) == 0
    assert L.cs_workspace_bytes(0, CS_I8, -1, 4) == 0


def test_product_path_has_no_fallback(monkeypatch, tmp_path):
    """With the library absent the binding raises instead of computing."""
    monkeypatch.setattr(_lib, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(_lib, "_LIB", None)
    with pytest.raises(RuntimeError):
        _lib.lib()
    with pytest.raises(RuntimeError):
        ops.pack(np.ones((2, 2), dtype=np.int8), 1)


def test_ctypes_signatures_match_header():
    """Each binding signature has as many arguments as the header declares."""
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    for name, (_, args) in _lib.SIGNATURES.items():
        m = re.search(name + r"\s*\(([^;]*)\)\s*;", text, flags=re.S)
        assert m, name
        nargs = len([a for a in m.group(1).split(",") if a.strip()])
        assert nargs == len(args), (name, nargs, len(args))
        assert ctypes  # silence unused import warnings in some linters


def test_fast_division_formula():
    """The kernels divide by launch-time constants with the round-up
    reciprocal m = floor(2^32 (2^s - d) / d) + 1, s = ceil(log2 d):
    floor(n / d) == (mulhi(n, m) + n) >> s for every 32-bit n."""
    rng = np.random.default_rng(5)
    for d in list(range(1, 3000)) + [65535, 65536, 100352, 2 ** 31 - 1, 2 ** 32 - 1]:
        s = (d - 1).bit_length() if d > 1 else 0
        m = (((1 << 32) * ((1 << s) - d)) // d + 1) if d > 1 else 0
        ns = [0, 1, d - 1, d, d + 1, 2 ** 32 - 1] + [int(v) for v in rng.integers(0, 2 ** 32, 50)]
        for n in ns:
            if 0 <= n < 2 ** 32:
                assert (((n * m) >> 32) + n) >> s == n // d
