"""Pins of the oracle's tolerance scale, layer-chain composition and
requantisation shift, each against a pure-Python loop written from the
definitions (no numpy algebra shared with the oracle), plus a mutation check:
every plausible mistake planted in the oracle (on the CPU) fails a pin.

* S[o] = sum |w * x| over the receptive field (padding and stride included)
  sets the fp32 tolerance of every fp32 layer (1e-5 * S per output).
* A layer of the keyword-spotting CNN runs in Table 1's order: conv, 2x2
  max-pool on the int32 sums, k-WTA (Section 2.2.2: exactly k winners), then
  the requantisation of the winners to int8; a conv map feeding a linear layer
  is flattened in (h, w, c) order, the slot order of the packed kernels.
* The requantisation shift is the smallest s with max|winner| >> s <= 127,
  i.e. max(0, bit_length(max|winner|) - 7).
"""
from __future__ import annotations

import itertools

import numpy as np
import pytest

from oracle import cs_oracle as o
from oracle import networks
from workloads import LayerSpec


def _rng(seed):
    return np.random.default_rng(seed)


# ------------------------------------------------------------ brute force
def bf_abs_sum_linear(x, W):
    B, D = x.shape
    O = W.shape[0]
    S = np.zeros((B, O))
    for b, oi in itertools.product(range(B), range(O)):
        s = 0.0
        for i in range(D):
            s += abs(float(W[oi, i]) * float(x[b, i]))
        S[b, oi] = s
    return S


def bf_conv_terms(x, W, stride, pad):
    """Yields (b, ho, wo, o, w*x) for every in-image term of the convolution."""
    B, H, Wd, C = x.shape
    O, KH, KW, _ = W.shape
    Ho = (H + 2 * pad - KH) // stride + 1
    Wo = (Wd + 2 * pad - KW) // stride + 1
    for b, ho, wo, oi in itertools.product(range(B), range(Ho), range(Wo), range(O)):
        for ky, kx, c in itertools.product(range(KH), range(KW), range(C)):
            hy, wx = ho * stride + ky - pad, wo * stride + kx - pad
            if 0 <= hy < H and 0 <= wx < Wd:
                yield b, ho, wo, oi, W[oi, ky, kx, c].item() * x[b, hy, wx, c].item()


def bf_conv_shape(x, W, stride, pad):
    B, H, Wd, _ = x.shape
    O, KH, KW, _ = W.shape
    return (B, (H + 2 * pad - KH) // stride + 1, (Wd + 2 * pad - KW) // stride + 1, O)


def bf_abs_sum_conv(x, W, stride, pad):
    S = np.zeros(bf_conv_shape(x, W, stride, pad))
    for b, ho, wo, oi, t in bf_conv_terms(x, W, stride, pad):
        S[b, ho, wo, oi] += abs(float(t))
    return S


def bf_conv(x, W, stride, pad, bias):
    shape = bf_conv_shape(x, W, stride, pad)
    y = {}
    for b, ho, wo, oi in itertools.product(*map(range, shape)):
        y[b, ho, wo, oi] = 0 if bias is None else int(bias[oi])
    for b, ho, wo, oi, t in bf_conv_terms(x, W, stride, pad):
        y[b, ho, wo, oi] += int(t)
    return shape, y


def bf_pool(shape, y):
    B, H, Wd, O = shape
    ps = (B, H // 2, Wd // 2, O)
    p = {}
    for b, hp, wp, oi in itertools.product(*map(range, ps)):
        p[b, hp, wp, oi] = max(y[b, 2 * hp + dy, 2 * wp + dx, oi] for dy in (0, 1) for dx in (0, 1))
    return ps, p


def bf_winners(values, k):
    """Indices of the k largest values, ties to the lower index."""
    order = sorted(range(len(values)), key=lambda i: (-values[i], i))
    return set(order[:k])


def bf_requant(a, s):
    q = a >> s                     # Python's >> on int is a floor shift
    return max(-127, min(127, q))


def bf_shift(m):
    return max(0, int(m).bit_length() - 7)


def bf_chain(x, layers, Ws, bs):
    """The keyword-spotting layer order of Table 1 on dictionaries of Python
    ints.  Returns, per layer, (sums after pool, winner mask, output)."""
    cur = x.astype(np.int64)
    out = []
    for spec, W, bias in zip(layers, Ws, bs):
        if spec.kind == "conv":
            shape, y = bf_conv(cur, W, spec.stride, spec.pad, bias)
            if spec.pool == 2:
                shape, y = bf_pool(shape, y)
            acc = np.zeros(shape, dtype=np.int64)
            for key, v in y.items():
                acc[key] = v
        else:
            B = cur.shape[0]
            if cur.ndim == 4:      # flatten in (h, w, c) order
                _, H, Wd, C = cur.shape
                flat = np.zeros((B, H * Wd * C), dtype=np.int64)
                for b, h, w_, c in itertools.product(range(B), range(H), range(Wd), range(C)):
                    flat[b, (h * Wd + w_) * C + c] = cur[b, h, w_, c]
                cur = flat
            D = cur.shape[1]
            acc = np.zeros((B, W.shape[0]), dtype=np.int64)
            for b, oi in itertools.product(range(B), range(W.shape[0])):
                s = 0 if bias is None else int(bias[oi])
                for i in range(D):
                    s += int(W[oi, i]) * int(cur[b, i])
                acc[b, oi] = s
        rows = acc.reshape(-1, acc.shape[-1])
        if spec.k is None:
            out.append((acc, None, acc))
            cur = acc
            continue
        win = np.zeros(rows.shape, dtype=bool)
        q = np.zeros(rows.shape, dtype=np.int64)
        for r, row in enumerate(rows):
            vals = [int(v) for v in row]
            for j in bf_winners(vals, spec.k):
                win[r, j] = True
                q[r, j] = bf_requant(vals[j], spec.shift)
        win = win.reshape(acc.shape)
        q = q.reshape(acc.shape)
        out.append((acc, win, q))
        cur = q
    return out


# ------------------------------------------------------------ the checks
def check_abs_sum_linear():
    r = _rng(101)
    x = r.normal(size=(3, 11)).astype(np.float32)
    x[r.random(x.shape) < 0.4] = 0
    W = r.normal(size=(5, 11)).astype(np.float32)
    got = o.abs_sum_linear(x, W)
    assert got.shape == (3, 5)
    assert np.allclose(got, bf_abs_sum_linear(x, W), rtol=1e-12, atol=0)


def check_abs_sum_conv():
    r = _rng(102)
    x = r.normal(size=(2, 7, 6, 3)).astype(np.float32)
    x[r.random(x.shape) < 0.5] = 0
    W = r.normal(size=(4, 3, 3, 3)).astype(np.float32)
    for stride, pad in ((1, 1), (2, 1), (1, 0), (2, 2)):
        got = o.abs_sum_conv(x, W, stride, pad)
        exp = bf_abs_sum_conv(x, W, stride, pad)
        assert got.shape == exp.shape
        assert np.allclose(got, exp, rtol=1e-12, atol=0)


def tiny_chain():
    """A four-layer int8 chain in the keyword-spotting CNN's layer order:
    conv 3x3 (pool, k-WTA, requant) -> conv 3x3 pad 1 (pool, k-WTA, requant)
    -> flatten -> linear (k-WTA, requant) -> linear."""
    layers = (
        LayerSpec("c1", "conv", 2, 6, n=1, kh=3, kw=3, pool=2, k=3, shift=9, bias=True),
        LayerSpec("c2", "conv", 6, 4, n=1, kh=3, kw=3, pad=1, pool=2, k=2, shift=8),
        LayerSpec("l1", "linear", 16, 10, n=1, k=4, shift=8),
        LayerSpec("l2", "linear", 10, 3, n=1, bias=True),
    )
    r = _rng(103)
    x = r.integers(-127, 128, size=(2, 10, 10, 2)).astype(np.int8)
    Ws = [r.integers(-127, 128, size=(6, 3, 3, 2)).astype(np.int8),
          r.integers(-127, 128, size=(4, 3, 3, 6)).astype(np.int8),
          r.integers(-127, 128, size=(10, 16)).astype(np.int8),
          r.integers(-127, 128, size=(3, 10)).astype(np.int8)]
    bs = [r.integers(-1000, 1001, size=6).astype(np.int32), None, None,
          r.integers(-1000, 1001, size=3).astype(np.int32)]
    return layers, x, Ws, bs


def check_chain():
    layers, x, Ws, bs = tiny_chain()
    exp = bf_chain(x, layers, Ws, bs)
    got = networks.run_chain(layers, x, Ws, bs)
    assert len(got) == len(exp)
    # the chain is not trivial: every requantised layer keeps some unsaturated
    # winners and its k-WTA drops something
    for li, ((acc, win, out), g) in enumerate(zip(exp, got)):
        assert g["acc"].shape == acc.shape, li
        assert np.array_equal(np.asarray(g["acc"], dtype=np.int64), acc), li
        if win is None:
            assert g["win"] is None
        else:
            assert np.array_equal(g["win"], win), li
            assert (np.abs(out[win]) < 127).any() and (~win).any()
        assert np.array_equal(np.asarray(g["out"], dtype=np.int64), out), li


def check_requant_shift():
    for m in list(range(0, 1100)) + [2 ** 20 - 1, 2 ** 20, 2 ** 30 + 5]:
        for sign in (1, -1):
            vals = np.array([sign * m, 1, -1], dtype=np.int64)
            assert networks.requant_shift(vals) == bf_shift(m), (sign, m)
    # the boundary the rule turns on
    assert networks.requant_shift(np.array([255])) == 1
    assert networks.requant_shift(np.array([-255, 17])) == 1
    assert networks.requant_shift(np.array([-256])) == 2
    assert networks.requant_shift(np.array([12, -127])) == 0


def test_abs_sum_linear_brute_force():
    check_abs_sum_linear()


def test_abs_sum_conv_brute_force():
    check_abs_sum_conv()


def test_chain_matches_table1_order_brute_force():
    check_chain()


def test_requant_shift_rule_brute_force():
    check_requant_shift()


def test_config2_chain_order_on_a_sample():
    """The oracle's keyword-spotting chain on one sample of the seeded config-2
    batch equals the brute-force chain at the real shapes for the first conv
    and the pooled map it feeds (conv1 -> pool -> k-WTA -> requant)."""
    from workloads import CONFIGS, generate
    cfg = CONFIGS[2]
    inp = generate(cfg, batch=1)
    l1 = cfg.layers[0]
    exp = bf_chain(inp["x"], (l1,), inp["W"][:1], inp["b"][:1])
    got = networks.run_chain((l1,), inp["x"], inp["W"][:1], inp["b"][:1])
    assert np.array_equal(np.asarray(got[0]["acc"], np.int64), exp[0][0])
    assert np.array_equal(got[0]["win"], exp[0][1])
    assert np.array_equal(np.asarray(got[0]["out"], np.int64), exp[0][2])


# ------------------------------------------------------------ mutations
def _abs_linear_no_abs(x, W):
    return np.asarray(x, dtype=np.float64) @ np.asarray(W, dtype=np.float64).T


def _abs_conv_no_abs(x, W, stride=1, pad=0):
    oc = W.shape[0]
    cols = o.im2col_nhwc(x, W.shape[1], W.shape[2], stride, pad)
    return cols @ np.asarray(W, dtype=np.float64).reshape(oc, -1).T


def _abs_conv_no_pad(x, W, stride=1, pad=0):
    return _ORIG["abs_sum_conv"](x, W, stride, 0)


def _layer_kwta_before_pool(spec, x, W, bias):
    if spec.kind != "conv" or spec.pool != 2:
        return _ORIG["layer_forward"](spec, x, W, bias)
    acc = o.conv2d_nhwc(x, W, spec.stride, spec.pad, bias)
    win = o.kwta_winners(acc, spec.k)
    masked = np.where(win, acc, 0)
    pooled = o.maxpool2x2_nhwc(masked)
    win2 = pooled != 0
    out = o.requant(pooled, spec.shift, win2) if spec.shift is not None else pooled
    return {"acc": pooled, "win": win2, "out": out}


def _layer_nchw_flatten(spec, x, W, bias):
    if spec.kind == "linear" and x.ndim == 4:
        x = np.ascontiguousarray(np.transpose(x, (0, 3, 1, 2))).reshape(x.shape[0], -1)
    return _ORIG["layer_forward"](spec, x, W, bias)


def _layer_requant_all(spec, x, W, bias):
    r = _ORIG["layer_forward"](spec, x, W, bias)
    if spec.shift is not None:
        r["out"] = o.requant(r["acc"], spec.shift)        # losers not zeroed
    return r


def _shift_log_rule(v):
    m = int(np.abs(np.asarray(v, dtype=np.int64)).max()) if np.size(v) else 0
    return 0 if m <= 127 else int(np.ceil(np.log2(m / 127.0)))


_ORIG = {"abs_sum_conv": o.abs_sum_conv, "layer_forward": networks.layer_forward}

MUTATIONS = {
    "abs_sum_linear without abs": (o, "abs_sum_linear", _abs_linear_no_abs, check_abs_sum_linear),
    "abs_sum_conv without abs": (o, "abs_sum_conv", _abs_conv_no_abs, check_abs_sum_conv),
    "abs_sum_conv without padding": (o, "abs_sum_conv", _abs_conv_no_pad, check_abs_sum_conv),
    "k-WTA before the pool": (networks, "layer_forward", _layer_kwta_before_pool, check_chain),
    "NCHW flatten": (networks, "layer_forward", _layer_nchw_flatten, check_chain),
    "losers requantised": (networks, "layer_forward", _layer_requant_all, check_chain),
    "ceil(log2(m/127)) shift": (networks, "requant_shift", _shift_log_rule, check_requant_shift),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_fails_a_pin(monkeypatch, name):
    module, attr, fn, check = MUTATIONS[name]
    check()                                   # passes on the oracle as it is
    monkeypatch.setattr(module, attr, fn)
    with pytest.raises(AssertionError):
        check()
