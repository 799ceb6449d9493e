"""Oracle for whole layer chains (TEST INFRASTRUCTURE ONLY).

A chain is a sequence of layer descriptions (any object with the attributes
kind, kh, kw, stride, pad, pool, k, shift); the oracle applies, per layer, the
dense definition of Section 3.2's steps in the paper's order:
multiply/route/sum (here: the dense product), the optional 2x2 max-pool of
Table 1, then Select (k-WTA) for the next layer and, for int8 chains, the
requantisation of the winners to int8.

Order inside a layer follows Table 1 for the keyword-spotting CNN: conv, then
max-pool on the int32 sums, then k-WTA, then requantisation.  A conv output
feeding a linear layer is flattened in NHWC order (h, w, c).
"""
from __future__ import annotations

import numpy as np

from . import cs_oracle as o


def layer_forward(spec, x: np.ndarray, W: np.ndarray, bias: np.ndarray | None) -> dict:
    """One layer.  Returns {"acc": sums after pool, "win": k-WTA mask or None,
    "out": what the next layer consumes}."""
    if spec.kind == "conv":
        if x.ndim != 4:
            raise ValueError("conv input must be NHWC")
        acc = o.conv2d_nhwc(x, W, spec.stride, spec.pad, bias)
        if spec.pool == 2:
            acc = o.maxpool2x2_nhwc(acc)
    else:
        xin = x.reshape(x.shape[0], -1)
        acc = o.linear(xin, W, bias)
    win = None
    out = acc
    if spec.k is not None:
        win = o.kwta_winners(acc, spec.k)
        if spec.shift is not None:
            out = o.requant(acc, spec.shift, win)
        else:
            out = np.where(win, acc, np.zeros_like(acc))
    return {"acc": acc, "win": win, "out": out}


def run_chain(layers, x: np.ndarray, Ws, bs, inputs=None) -> list:
    """Run every layer.  `inputs[l]`, when given and not None, replaces the
    input of layer l (used to check fp32 chains layer by layer)."""
    res = []
    cur = x
    for li, spec in enumerate(layers):
        if inputs is not None and li < len(inputs) and inputs[li] is not None:
            cur = inputs[li]
        r = layer_forward(spec, cur, Ws[li], bs[li])
        res.append(r)
        cur = r["out"]
    return res


def requant_shift(winner_values: np.ndarray) -> int:
    """The smallest s >= 0 with max|winner| >> s <= 127: the smallest
    arithmetic shift that brings every winner into the int8 range [-127, 127]
    (equal to max(0, bit_length(max|winner|) - 7); at max|winner| = 255 it is
    1, where ceil(log2(255 / 127)) would give 2)."""
    m = int(np.abs(np.asarray(winner_values, dtype=np.int64)).max()) if np.size(winner_values) else 0
    s = 0
    while (m >> s) > 127:
        s += 1
    return s
