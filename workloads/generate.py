"""Seeded synthetic inputs for the five configurations.

Random streams: numpy PCG64 seeded with SeedSequence(2112_13896 + config id),
spawned into, per layer, a partition stream, a weight-value stream and a bias
stream, followed by one activation stream.  Everything is drawn on the host
once; the GPU path and the CPU oracle receive the same arrays.

Nothing here computes any part of the layer: it draws supports, values and
activations only.
"""
from __future__ import annotations

import hashlib

import numpy as np

from .configs import Config, LayerSpec


def tensor_digest(a: np.ndarray) -> str:
    """SHA-256 of an array's dtype, shape and bytes (records what was generated)."""
    a = np.ascontiguousarray(a)
    h = hashlib.sha256()
    h.update(str(a.dtype).encode())
    h.update(str(a.shape).encode())
    h.update(a.tobytes())
    return h.hexdigest()


def _nonzero_int8(rng: np.random.Generator, shape) -> np.ndarray:
    """Uniform over {-127..-1, 1..127}."""
    u = rng.integers(0, 254, size=shape)
    return np.where(u < 127, u - 127, u - 126).astype(np.int8)


def complementary_weights(rng_part: np.random.Generator, rng_val: np.random.Generator,
                          d_out: int, r: int, n: int, dist: str) -> np.ndarray:
    """Dense [d_out][r] weights whose kernels form complementary sets.

    For every set g (outputs g*n .. g*n+n-1) a random permutation of the r
    slots is cut into n disjoint pieces of r/n slots, one per kernel, so the
    supports of a set are disjoint and together cover every slot.  Values are
    non-zero on the support and zero elsewhere.
    dist: "int8"   -> uniform over the non-zero int8 values in [-127, 127]
          "normal" -> N(0, 2/nnz_k) drawn in float64, rounded once to float32
    """
    if d_out % n or r % n:
        raise ValueError("n must divide d_out and r")
    nnz_k = r // n
    mask = np.zeros((d_out, r), dtype=bool)
    for g in range(d_out // n):
        perm = rng_part.permutation(r)
        for j in range(n):
            mask[g * n + j, perm[j * nnz_k:(j + 1) * nnz_k]] = True
    if dist == "int8":
        vals = _nonzero_int8(rng_val, (d_out, r))
        W = np.where(mask, vals, np.int8(0)).astype(np.int8)
    elif dist == "normal":
        sigma = np.sqrt(2.0 / nnz_k)
        vals = rng_val.normal(0.0, sigma, size=(d_out, r)).astype(np.float32)
        if np.any(vals[mask] == 0):
            raise RuntimeError("a support weight rounded to zero")
        W = np.where(mask, vals, np.float32(0)).astype(np.float32)
    else:
        raise ValueError(dist)
    return W


def channel_complementary_weights(rng_part: np.random.Generator, rng_val: np.random.Generator,
                                  c_out: int, kh: int, kw: int, c: int, n: int) -> np.ndarray:
    """Dense fp32 [c_out][kh][kw][c] filters whose channel slices form
    complementary sets: for every filter and every group of n consecutive
    channels, a random permutation of the kh*kw positions is cut into n
    pieces, one per channel of the group.  Values N(0, 2/nnz) per filter,
    drawn in float64 and rounded once to float32."""
    t = kh * kw
    if c % n or t % n:
        raise ValueError("n must divide the channels and kh*kw")
    per = t // n
    mask = np.zeros((c_out, t, c), dtype=bool)
    for o in range(c_out):
        for q in range(c // n):
            perm = rng_part.permutation(t)
            for j in range(n):
                mask[o, perm[j * per:(j + 1) * per], q * n + j] = True
    nnz = t * c // n
    vals = rng_val.normal(0.0, np.sqrt(2.0 / nnz), size=mask.shape).astype(np.float32)
    if np.any(vals[mask] == 0):
        raise RuntimeError("a support weight rounded to zero")
    return np.where(mask, vals, np.float32(0)).astype(np.float32).reshape(c_out, kh, kw, c)


def block_complementary_weights(rng_part: np.random.Generator, rng_val: np.random.Generator,
                                d_out: int, r: int, n: int, b: int) -> np.ndarray:
    """Dense fp32 [d_out][r] weights, complementary in blocks of b slots: for
    every set, a random permutation of the r/b blocks is split into n nearly
    equal pieces, one per kernel; a kernel is non-zero on all slots of its
    blocks.  Values N(0, 2/nnz) per kernel, float64 rounded once to float32."""
    if r % b or d_out % n:
        raise ValueError("b must divide r and n must divide d_out")
    nb = r // b
    mask = np.zeros((d_out, nb), dtype=bool)
    for g in range(d_out // n):
        for j, piece in enumerate(np.array_split(rng_part.permutation(nb), n)):
            mask[g * n + j, piece] = True
    mask = np.repeat(mask, b, axis=1)
    nnz = np.maximum(mask.sum(axis=1, keepdims=True), 1)
    vals = (rng_val.normal(size=mask.shape) * np.sqrt(2.0 / nnz)).astype(np.float32)
    if np.any(vals[mask] == 0):
        raise RuntimeError("a support weight rounded to zero")
    return np.where(mask, vals, np.float32(0)).astype(np.float32)


def sparse_rows(rng: np.random.Generator, rows: int, c: int, nnz: int | None, dist: str):
    """[rows][c] activations with exactly `nnz` non-zeros per row at uniform
    positions (without replacement); nnz=None gives a dense draw.

    dist: "u1_127"     -> int8 uniform in [1, 127]
          "u_m127_127" -> int8 uniform in [-127, 127] (zeros possible)
          "absnormal"  -> float32 |N(0, 1)|
    """
    if dist == "u1_127":
        vals = rng.integers(1, 128, size=(rows, c)).astype(np.int8)
    elif dist == "u_m127_127":
        vals = rng.integers(-127, 128, size=(rows, c)).astype(np.int8)
    elif dist == "absnormal":
        vals = np.abs(rng.normal(0.0, 1.0, size=(rows, c))).astype(np.float32)
        vals[vals == 0] = np.float32(1.0)
    else:
        raise ValueError(dist)
    if nnz is None:
        return vals
    keys = rng.random((rows, c))
    pos = np.argpartition(keys, nnz - 1, axis=1)[:, :nnz] if nnz < c else None
    if pos is None:
        return vals
    mask = np.zeros((rows, c), dtype=bool)
    np.put_along_axis(mask, pos, True, axis=1)
    return np.where(mask, vals, np.zeros_like(vals))


def layer_weight_shape(spec: LayerSpec) -> tuple:
    if spec.kind == "conv":
        return (spec.c_out, spec.kh, spec.kw, spec.c_in)   # OHWI
    return (spec.c_out, spec.c_in)


def generate(cfg: Config, batch: int | None = None) -> dict:
    """Inputs of a configuration: x, per-layer dense weights W and biases.

    `batch` below cfg.batch returns the first `batch` samples of the full draw
    (the activation stream is always drawn for the full batch).
    """
    ss = np.random.SeedSequence(cfg.seed)
    kids = ss.spawn(3 * len(cfg.layers) + 1)
    Ws, bs = [], []
    for li, spec in enumerate(cfg.layers):
        rng_part = np.random.Generator(np.random.PCG64(kids[3 * li]))
        rng_val = np.random.Generator(np.random.PCG64(kids[3 * li + 1]))
        rng_bias = np.random.Generator(np.random.PCG64(kids[3 * li + 2]))
        W2 = complementary_weights(rng_part, rng_val, spec.c_out, spec.r, spec.n, spec.weight_dist)
        Ws.append(W2.reshape(layer_weight_shape(spec)))
        if spec.bias:
            bs.append(rng_bias.integers(-1000, 1001, size=spec.c_out).astype(np.int32))
        else:
            bs.append(None)
    rng_x = np.random.Generator(np.random.PCG64(kids[-1]))
    shape = (cfg.batch,) + tuple(cfg.in_shape)
    rows = int(np.prod(shape[:-1]))
    x = sparse_rows(rng_x, rows, shape[-1], cfg.in_nnz, cfg.in_dist).reshape(shape)
    if batch is not None:
        if not 0 < batch <= cfg.batch:
            raise ValueError("batch out of range")
        x = x[:batch].copy()
    return {"x": x, "W": Ws, "b": bs}
