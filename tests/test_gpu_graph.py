"""A whole forward pass recorded into a HIP graph (Network.capture, what the
benchmark replays) gives the eager pass's bits on every replay.

The graph is replayed several times with the program's own eager work and
synchronisations in between (another buffer set run eagerly on a different
input, torch kernels on unrelated memory); after every replay the sums and
the k-WTA outputs of every layer must equal those of the eager pass over the
same input, bit for bit, for int8 and fp32 chains alike (the kernels'
summation order does not depend on timing).
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

from paper_2112_13896_amd.network import Network
from tests.gpu_util import dev, host
from workloads import CONFIGS, generate

pytestmark = pytest.mark.gpu


def snapshot(net, bufs):
    torch.cuda.synchronize()
    outs = [host(net.dense_output(li, bufs)).view(np.uint8).copy()
            for li in range(len(net.packed))]
    sums = [host(a).view(np.uint8).copy() for a in bufs.acc]
    return outs, sums


@pytest.mark.parametrize("cid", [1, 2, 3, 5])
def test_graph_replay_matches_eager(cid):
    cfg = CONFIGS[cid]
    inp = generate(cfg)
    net = Network(cfg.layers, inp["W"], inp["b"], cfg.in_shape, cfg.batch)
    x = dev(inp["x"])
    net.forward(x)
    want_outs, want_sums = snapshot(net, net.bufs)

    bufs = net.make_buffers()
    g = net.capture(x, bufs)
    side = net.make_buffers()
    x2 = torch.flip(x, dims=[0]).contiguous()      # the same samples in reverse order
    scratch = torch.arange(1 << 20, dtype=torch.float32, device="cuda")
    for rep in range(3):
        g.replay()
        outs, sums = snapshot(net, bufs)
        for li in range(len(cfg.layers)):
            assert np.array_equal(outs[li], want_outs[li]), f"replay {rep}: layer {li} output"
            assert np.array_equal(sums[li], want_sums[li]), f"replay {rep}: layer {li} sums"
        # eager work between replays: the chain on other buffers and input,
        # and unrelated torch kernels
        net.forward(x2, side)
        scratch.mul_(1.0001).add_(rep)
        torch.cuda.synchronize()
