"""CPU oracle for the Complementary Sparsity sparse-sparse layer.

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or
execute this module; only the tests, the smoke check and the CPU-baseline leg
of the benchmark use it.

The method (Hunter, Spracklen and Ahmad, "Two Sparsities Are Better Than One",
Section 3) reorganises the non-zero weights of N sparse kernels into one packed
kernel and then visits only non-zero activations.  Zero weights and zero
activations contribute nothing to a weighted sum (Section 2.3.1, Figure 3), and
packing only moves the non-zero weights (Section 3), so every layer reaches
exactly the dense result.  The oracle is therefore the plain dense definition,
computed from the UNPACKED weights:

* linear layer  : y = x W^T + b                      (Section 2.2)
* convolution   : cross-correlation, NHWC, zero pad   (Section 5.1: a 3x3 conv
                  is nine 1x1 convs; Table 1 for the 5x5 GSC layers)
* 2x2 max-pool  : stride 2                            (Table 1)
* k-WTA         : keep exactly the k largest values   (Section 2.2.2, 3.3.3)
* requantisation: arithmetic shift + clamp to int8    (reading of Section 4:
                  "activations and weights are quantized to 8 bits")

Everything is computed in float64 (exact for the integer configurations, whose
partial sums stay far below 2**53) or in int64.  The packing definition is here
too, because the product's pack routine is checked against it.

Readings taken where the paper is silent (listed in the design notes as well):
  * the N kernels overlaid into one packed kernel are the N contiguous output
    channels [g*N, (g+1)*N);
  * a kernel id is the local position o - g*N in [0, N);
  * a conv receptive-field slot is i = (ky*KW + kx)*C_in + c (taps major);
  * k-WTA keeps exactly k values, ties going to the lower index, and a winner
    keeps its value even when it is <= 0;
  * requantisation of an int32 winner a is clamp(a >> s, -127, 127) with an
    arithmetic (floor) shift; losers become 0.
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "PackCollision",
    "pack",
    "unpack",
    "compact_rows",
    "linear",
    "conv2d_nhwc",
    "im2col_nhwc",
    "maxpool2x2_nhwc",
    "kwta_winners",
    "kwta",
    "requant",
    "pair_count_linear",
    "pair_count_conv",
    "abs_sum_linear",
    "abs_sum_conv",
    "dense_macs_linear",
    "dense_macs_conv",
]

_EXACT = float(2 ** 53)


class PackCollision(ValueError):
    """Two kernels of one packed set have a non-zero weight at the same slot."""

    def __init__(self, g: int, i: int):
        super().__init__(f"kernels of group {g} collide at slot {i}")
        self.g = g
        self.i = i


# ---------------------------------------------------------------------------
# Combine (Section 3.1 step 1, Section 3.2 step 1; Figure 7; Section 3.3.1 for
# the Kernel ID attached to each packed weight, Section 3.3.2 for the id only
# needing to identify the position inside the partition).
# ---------------------------------------------------------------------------
def pack(W: np.ndarray, n: int):
    """Overlay each set of n kernels into one packed kernel.

    W : [d_out][r] dense weights (zero = absent connection).
    Returns (val[r][G], kid[r][G] uint8, holes) with G = d_out // n, where
    val[i][g] = W[g*n + kid][i] for the unique kernel of group g that is
    non-zero at slot i.  A slot no kernel of the group uses ("hole") holds
    val = 0, kid = 0.  Raises PackCollision at the first (g, i) in group-major,
    slot-minor order where two kernels of one group are both non-zero.
    """
    W = np.asarray(W)
    d_out, r = W.shape
    if n <= 0 or d_out % n != 0:
        raise ValueError("n must divide d_out")
    G = d_out // n
    val = np.zeros((r, G), dtype=W.dtype)
    kid = np.zeros((r, G), dtype=np.uint8)
    holes = 0
    for g in range(G):
        block = W[g * n:(g + 1) * n]              # the n kernels of this set
        nz = block != 0                             # [n][r]
        count = nz.sum(axis=0)                      # kernels present per slot
        bad = np.nonzero(count > 1)[0]
        if bad.size:
            raise PackCollision(g, int(bad[0]))
        holes += int((count == 0).sum())
        owner = nz.argmax(axis=0)                   # the present kernel (0 if none)
        kid[:, g] = owner.astype(np.uint8)
        val[:, g] = block[owner, np.arange(r)]      # 0 for holes (block is 0 there)
    return val, kid, holes


def unpack(val: np.ndarray, kid: np.ndarray, n: int) -> np.ndarray:
    """Inverse of pack: rebuild the dense [G*n][r] weights."""
    r, G = val.shape
    W = np.zeros((G * n, r), dtype=val.dtype)
    for g in range(G):
        for i in range(r):
            if val[i, g] != 0:
                W[g * n + int(kid[i, g]), i] = val[i, g]
    return W


# ---------------------------------------------------------------------------
# Combine along the channel dimension (Section 3.1: sets of kernels can be
# overlaid in the filter or in the channel dimension).  For one filter
# W[o] (kh x kw x C), the n channel slices of a group q (channels q*n ..
# q*n+n-1) have disjoint kh x kw supports and are overlaid into one dense
# kh x kw slice whose every slot keeps its weight and the channel ID (the
# slice it came from) - the channel-dimension counterpart of the Kernel ID.
# ---------------------------------------------------------------------------
def pack_channels(W4: np.ndarray, n: int):
    """W4 : [c_out][kh][kw][C] dense weights (zero = absent).
    Returns (val[c_out][C/n][kh][kw], cid[..] uint8, holes): val[o][q][y][x] =
    W4[o][y][x][q*n + cid] for the unique channel of group q non-zero at
    (y, x) in filter o; holes hold 0, 0.  Raises PackCollision(o, slot) with
    slot = (q*kh + y)*kw + x at the first collision in (o, q, y, x) order."""
    W4 = np.asarray(W4)
    c_out, kh, kw, C = W4.shape
    if n <= 0 or C % n != 0:
        raise ValueError("n must divide the channels")
    Q = C // n
    val = np.zeros((c_out, Q, kh, kw), dtype=W4.dtype)
    cid = np.zeros((c_out, Q, kh, kw), dtype=np.uint8)
    holes = 0
    for o in range(c_out):
        for q in range(Q):
            block = W4[o, :, :, q * n:(q + 1) * n]       # [kh][kw][n]
            nz = block != 0
            count = nz.sum(axis=2)
            bad = np.argwhere(count > 1)
            if bad.size:
                y, x = bad[0]
                raise PackCollision(o, int((q * kh + y) * kw + x))
            holes += int((count == 0).sum())
            owner = nz.argmax(axis=2)
            cid[o, q] = owner.astype(np.uint8)
            val[o, q] = np.take_along_axis(block, owner[..., None], axis=2)[..., 0]
    return val, cid, holes


def unpack_channels(val: np.ndarray, cid: np.ndarray, n: int) -> np.ndarray:
    """Inverse of pack_channels: the dense [c_out][kh][kw][C] weights."""
    c_out, Q, kh, kw = val.shape
    W4 = np.zeros((c_out, kh, kw, Q * n), dtype=val.dtype)
    for o in range(c_out):
        for q in range(Q):
            for y in range(kh):
                for x in range(kw):
                    if val[o, q, y, x] != 0:
                        W4[o, y, x, q * n + int(cid[o, q, y, x])] = val[o, q, y, x]
    return W4


# ---------------------------------------------------------------------------
# Complementary Sparsity with blocks of non-zeros (Section 3.1: complementary
# patterns whose non-zero elements come in blocks; the stem of Section 5 treats
# a pixel's 3 RGB values as one block, all non-zero or all zero).  Slots
# i*b .. i*b+b-1 form block i; every kernel's support is a union of whole
# blocks, and the kernels of a set are complementary block by block, so one
# Kernel ID per block routes all b of its products.
# ---------------------------------------------------------------------------
class BlockViolation(ValueError):
    """A kernel's support covers part of a block."""

    def __init__(self, o: int, blk: int):
        super().__init__(f"kernel {o} covers part of block {blk}")
        self.o = o
        self.blk = blk


def pack_blocks(W: np.ndarray, n: int, b: int):
    """W : [d_out][r] dense weights, r a multiple of b.  Returns
    (val[r][G], kidb[r/b][G] uint8, holes) - val as pack() gives it, kidb the
    Kernel ID of each block (0 for a block no kernel of the set uses), holes
    the number of such (block, set) pairs.  Raises BlockViolation(o, block)
    for the first kernel (in output order) whose support splits a block, or
    PackCollision(g, block) at the first block two kernels of a set share."""
    W = np.asarray(W)
    d_out, r = W.shape
    if b <= 0 or r % b != 0:
        raise ValueError("b must divide the slots")
    if n <= 0 or d_out % n != 0:
        raise ValueError("n must divide d_out")
    nb = r // b
    nzb = (W != 0).reshape(d_out, nb, b)
    part = nzb.any(axis=2) & ~nzb.all(axis=2)
    for o_ in range(d_out):
        bad = np.nonzero(part[o_])[0]
        if bad.size:
            raise BlockViolation(o_, int(bad[0]))
    G = d_out // n
    kidb = np.zeros((nb, G), dtype=np.uint8)
    holes = 0
    for g in range(G):
        present = nzb[g * n:(g + 1) * n].any(axis=2)   # [n][nb]
        count = present.sum(axis=0)
        bad = np.nonzero(count > 1)[0]
        if bad.size:
            raise PackCollision(g, int(bad[0]))
        holes += int((count == 0).sum())
        kidb[:, g] = present.argmax(axis=0).astype(np.uint8)
    val, _, _ = pack(W, n)
    return val, kidb, holes


# ---------------------------------------------------------------------------
# Select's sparse representation (Section 3.2 step 2; Figure 10 sends the
# winners on "along with their indices").
# ---------------------------------------------------------------------------
def compact_rows(x: np.ndarray):
    """Per row of x [rows][c]: (indices of the non-zero elements in ascending
    order, their values).  A float -0.0 is a zero."""
    x = np.asarray(x)
    out = []
    for row in x.reshape(-1, x.shape[-1]):
        nz = np.flatnonzero(row != 0)
        out.append((nz, row[nz]))
    return out


# ---------------------------------------------------------------------------
# Multiply / route / sum, written as the dense definition it equals.
# ---------------------------------------------------------------------------
def _to_result(acc: np.ndarray, integer: bool) -> np.ndarray:
    if not integer:
        return acc
    if acc.size and np.abs(acc).max() >= _EXACT:
        raise OverflowError("integer accumulation left the exact float64 range")
    out = np.rint(acc).astype(np.int64)
    assert np.array_equal(out.astype(np.float64), acc)
    return out


def _is_int(*arrays) -> bool:
    return all(a is None or np.issubdtype(np.asarray(a).dtype, np.integer) for a in arrays)


def linear(x: np.ndarray, W: np.ndarray, bias: np.ndarray | None = None) -> np.ndarray:
    """y[b][o] = bias[o] + sum_i W[o][i] * x[b][i]  (Section 2.2: a layer is a
    matrix product of the weights with the activations).

    Integer inputs give an int64 result (exact); float inputs a float64 result.
    """
    integer = _is_int(x, W, bias)
    acc = np.asarray(x, dtype=np.float64) @ np.asarray(W, dtype=np.float64).T
    if bias is not None:
        acc = acc + np.asarray(bias, dtype=np.float64)[None, :]
    return _to_result(acc, integer)


def conv_out_size(h: int, k: int, stride: int, pad: int) -> int:
    return (h + 2 * pad - k) // stride + 1


def im2col_nhwc(x: np.ndarray, kh: int, kw: int, stride: int, pad: int) -> np.ndarray:
    """cols[b, ho, wo, (ky*kw + kx)*c + ch] = x[b, ho*s + ky - p, wo*s + kx - p, ch]
    (zero outside the image).  Slot order is taps major, channels inner."""
    x = np.asarray(x)
    b, h, w, c = x.shape
    ho = conv_out_size(h, kh, stride, pad)
    wo = conv_out_size(w, kw, stride, pad)
    xp = np.zeros((b, h + 2 * pad, w + 2 * pad, c), dtype=np.float64)
    xp[:, pad:pad + h, pad:pad + w, :] = x
    cols = np.empty((b, ho, wo, kh, kw, c), dtype=np.float64)
    for ky in range(kh):
        for kx in range(kw):
            cols[:, :, :, ky, kx, :] = xp[:, ky:ky + stride * (ho - 1) + 1:stride,
                                          kx:kx + stride * (wo - 1) + 1:stride, :]
    return cols.reshape(b, ho, wo, kh * kw * c)


def conv2d_nhwc(x: np.ndarray, W: np.ndarray, stride: int = 1, pad: int = 0,
                bias: np.ndarray | None = None) -> np.ndarray:
    """Convolution (cross-correlation, no kernel flip) of NHWC x with OHWI W.

    y[b, ho, wo, o] = bias[o] + sum_{ky,kx,c} W[o, ky, kx, c] *
                      x[b, ho*s + ky - p, wo*s + kx - p, c]
    Section 5.1 describes a 3x3 conv as nine 1x1 convs; this is that sum.
    """
    W = np.asarray(W)
    o, kh, kw, c = W.shape
    assert x.shape[3] == c
    integer = _is_int(x, W, bias)
    cols = im2col_nhwc(x, kh, kw, stride, pad)
    acc = cols @ W.reshape(o, kh * kw * c).astype(np.float64).T
    if bias is not None:
        acc = acc + np.asarray(bias, dtype=np.float64)
    return _to_result(acc, integer)


def maxpool2x2_nhwc(y: np.ndarray) -> np.ndarray:
    """2x2 max-pool with stride 2 (Table 1, MaxPool-1/2)."""
    b, h, w, c = y.shape
    assert h % 2 == 0 and w % 2 == 0
    return y.reshape(b, h // 2, 2, w // 2, 2, c).max(axis=(2, 4))


# ---------------------------------------------------------------------------
# k-WTA (Section 2.2.2: exactly the top K activations propagate; Section 3.3.3
# global/local variants select the K largest of a vector or of a channel row).
# ---------------------------------------------------------------------------
def kwta_winners(v: np.ndarray, k: int) -> np.ndarray:
    """Boolean mask of the k winners of each row of v (last axis).

    Rows are ordered by decreasing value with ties kept in index order (a
    stable sort), and the first k of that order win.  Values compare
    numerically, so -0.0 and +0.0 tie.
    """
    v = np.asarray(v)
    c = v.shape[-1]
    if not 0 <= k <= c:
        raise ValueError("need 0 <= k <= row length")
    flat = v.reshape(-1, c)
    key = flat.astype(np.float64) + 0.0 if not np.issubdtype(flat.dtype, np.integer) \
        else flat.astype(np.int64)
    order = np.argsort(-key, axis=1, kind="stable")
    mask = np.zeros(flat.shape, dtype=bool)
    rows = np.arange(flat.shape[0])[:, None]
    mask[rows, order[:, :k]] = True
    return mask.reshape(v.shape)


def kwta(v: np.ndarray, k: int) -> np.ndarray:
    """Winners keep their value, every other element becomes zero."""
    v = np.asarray(v)
    return np.where(kwta_winners(v, k), v, np.zeros_like(v))


def kwta_units_winners(v: np.ndarray, k: int, unit: int = 64) -> np.ndarray:
    """k-WTA in units (Section 5: the k-WTA operator takes a convolution's
    output in units of 64 elements, so that wide layers are built from [64:64]
    modules): the last axis is cut into consecutive units of `unit` elements
    and each unit keeps its own k winners (ties to the lower index)."""
    v = np.asarray(v)
    c = v.shape[-1]
    if unit <= 0 or c % unit != 0:
        raise ValueError("unit must divide the row length")
    units = v.reshape(v.shape[:-1] + (c // unit, unit))
    return kwta_winners(units, k).reshape(v.shape)


def requant(a: np.ndarray, shift: int, winners: np.ndarray | None = None) -> np.ndarray:
    """int32 accumulator -> int8: clamp(a >> shift, -127, 127), arithmetic shift.

    Elements outside `winners` (when given) become 0.
    """
    a = np.asarray(a, dtype=np.int64)
    if shift < 0:
        raise ValueError("shift must be >= 0")
    q = np.clip(np.right_shift(a, shift), -127, 127).astype(np.int8)
    if winners is not None:
        q = np.where(winners, q, np.int8(0)).astype(np.int8)
    return q


# ---------------------------------------------------------------------------
# Side outputs: counts and magnitudes used by the checks.
# ---------------------------------------------------------------------------
def pair_count_linear(x: np.ndarray, W: np.ndarray) -> int:
    """Number of (w != 0, x != 0) pairs = products a sparse-sparse layer needs
    (Figure 1 / Figure 3: a product is needed only when both are non-zero)."""
    xm = (np.asarray(x) != 0).astype(np.int64)
    wm = (np.asarray(W) != 0).astype(np.int64)
    return int((xm @ wm.T).sum())


def pair_count_conv(x: np.ndarray, W: np.ndarray, stride: int = 1, pad: int = 0) -> int:
    o, kh, kw, c = W.shape
    xm = (np.asarray(x) != 0).astype(np.float64)
    cols = im2col_nhwc(xm, kh, kw, stride, pad)
    wm = (np.asarray(W).reshape(o, -1) != 0).astype(np.float64)
    return int(round((cols @ wm.T).sum()))


def abs_sum_linear(x: np.ndarray, W: np.ndarray) -> np.ndarray:
    """S[b][o] = sum_i |W[o][i] * x[b][i]| (float64): sets the fp32 tolerance."""
    return np.abs(np.asarray(x, dtype=np.float64)) @ np.abs(np.asarray(W, dtype=np.float64)).T


def abs_sum_conv(x: np.ndarray, W: np.ndarray, stride: int = 1, pad: int = 0) -> np.ndarray:
    o, kh, kw, c = W.shape
    cols = np.abs(im2col_nhwc(x, kh, kw, stride, pad))
    return cols @ np.abs(np.asarray(W, dtype=np.float64)).reshape(o, -1).T


def dense_macs_linear(batch: int, d_in: int, d_out: int) -> int:
    return batch * d_in * d_out


def dense_macs_conv(b: int, ho: int, wo: int, c_in: int, c_out: int, kh: int, kw: int) -> int:
    return b * ho * wo * c_out * kh * kw * c_in
