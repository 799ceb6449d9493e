"""The sparse work, counted in the kernels (Section 3.2, Figure 1).

The counting build of the library (libcs_count.so: the same sources compiled
with CS_COUNT_PRODUCTS) makes every multiply-route-sum kernel add the number of
weight x activation products it forms to a device counter.  Each configuration
runs through the C ABI exactly as the benchmark launches it (full batch, sums
not kept), and the count must equal the oracle's number of (w != 0, x != 0)
pairs of every routed layer, computed on the dense, unpacked weights and the
oracle's own layer inputs.  A kernel that multiplied whole rows, or entries past
a list's count, would count more; one that skipped entries would count less
and also fail the parity tests.  The first layer of the keyword-spotting
network is a dense contraction on the matrix cores (dense input, one kernel
per set) and is left out of both sides.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from oracle import cs_oracle as o
from oracle import networks
from paper_2112_13896_amd import _lib
from paper_2112_13896_amd.network import Network
from tests.gpu_util import dev
from workloads import CONFIGS, generate

pytestmark = pytest.mark.gpu


def oracle_pairs(cfg, inp) -> int:
    """Sum over the routed layers of the (w != 0, x != 0) pairs, each layer's
    input being the oracle's output of the layer before (for fp32 chains the
    number of non-zeros a pixel passes on is k either way)."""
    ref = networks.run_chain(cfg.layers, inp["x"], inp["W"], inp["b"])
    total = 0
    for li, spec in enumerate(cfg.layers):
        if spec.dense_input:
            continue
        x = inp["x"] if li == 0 else ref[li - 1]["out"]
        W = inp["W"][li]
        if spec.kind == "conv":
            total += o.pair_count_conv(x, W, spec.stride, spec.pad)
        else:
            total += o.pair_count_linear(x.reshape(x.shape[0], -1), W.reshape(W.shape[0], -1))
    return total


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_kernels_form_exactly_the_nonzero_pairs(cid):
    cfg = CONFIGS[cid]
    inp = generate(cfg)
    expect = oracle_pairs(cfg, inp)
    print(f"config {cid} ({cfg.name}): expecting {expect} products", flush=True)
    with _lib.counting_library():
        net = Network(cfg.layers, inp["W"], inp["b"], cfg.in_shape, cfg.batch, keep_sums=False)
        x = dev(inp["x"])
        _lib.product_count(reset=True)
        net.forward(x)
        torch.cuda.synchronize()
        got = _lib.product_count(reset=True)
        # a second pass counts the same again (the counter is not stale)
        net.forward(x)
        torch.cuda.synchronize()
        again = _lib.product_count(reset=True)
    assert got == expect, f"config {cid}: kernels formed {got} products, oracle pairs {expect}"
    assert again == expect
