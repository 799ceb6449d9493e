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


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
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


@pytest.mark.parametrize("cid,mode", [(2, "sequential"), (2, "alternate"), (3, "overlapped"),
                                      (3, "alternate"), (4, "alternate"), (5, "overlapped")])
def test_multi_pass_graph_matches_eager(cid, mode):
    """The benchmark's graph of several passes over rotating buffer sets (seven
    passes over three sets, so sets are written again inside one replay), in
    each of the three schedules: after each replay every set
    holds the eager pass's bits for its own input."""
    from bench import capture_passes
    cfg = CONFIGS[cid]
    batch = min(cfg.batch, 16)
    inp = generate(cfg, batch=batch)
    net = Network(cfg.layers, inp["W"], inp["b"], cfg.in_shape, batch, keep_sums=False)
    nsets = 3
    sets = [net.bufs] + [net.make_buffers() for _ in range(nsets - 1)]
    # a different input per set: the first one and two scaled/rolled copies
    xs = []
    for j in range(nsets):
        xj = np.roll(inp["x"], j, axis=0).copy()
        xs.append(dev(xj))
    want = []
    for j in range(nsets):
        net.forward(xs[j], sets[j])
        want.append(snapshot(net, sets[j])[0])
    for j in range(nsets):                               # scribble over every output
        for a in sets[j].acc:
            a.zero_()
        for o in sets[j].out:
            if o is not None:
                o.zero_()
        for lst in sets[j].lists:
            if lst is not None:
                for t in lst:
                    t.fill_(-1)
    g = capture_passes(net, xs, sets, 7, mode)
    for rep in range(3):
        g.replay()
        torch.cuda.synchronize()
        for j in range(nsets):
            got = snapshot(net, sets[j])[0]
            for li in range(len(net.packed)):
                assert np.array_equal(got[li], want[j][li]), f"replay {rep} set {j} layer {li}"
        torch.zeros(1 << 20, device="cuda").add_(1)      # unrelated eager work between replays


@pytest.mark.parametrize("cid", [3, 4])
def test_repeated_forward_identical_full_size(cid):
    """fp32 chains at their full batch: two eager passes over the same input
    give the same bits in every layer (no summation order depends on timing)."""
    cfg = CONFIGS[cid]
    inp = generate(cfg)
    net = Network(cfg.layers, inp["W"], inp["b"], cfg.in_shape, cfg.batch)
    x = dev(inp["x"])
    net.forward(x)
    a_outs, a_sums = snapshot(net, net.bufs)
    net.forward(x)
    b_outs, b_sums = snapshot(net, net.bufs)
    for li in range(len(cfg.layers)):
        assert np.array_equal(a_outs[li], b_outs[li]), f"layer {li} output"
        assert np.array_equal(a_sums[li], b_sums[li]), f"layer {li} sums"
