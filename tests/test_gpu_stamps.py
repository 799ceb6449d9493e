"""The stamping build's phase report (libcs_stamps.so, cs_phase_stamps): the
one-kernel keyword-spotting chain stamps every workgroup once per phase, so
after P passes the count slot holds P x (workgroups), every phase has a
non-negative mean and a workgroup's time is plausible; the
table-block kernel counts its tiles.  The stamping build computes the same
layer outputs as the product build (the stamps only add clock reads)."""
from __future__ import annotations

import numpy as np
import pytest
import torch

from paper_2112_13896_amd import _lib
from paper_2112_13896_amd.network import Network
from tests.gpu_util import dev, host
from workloads import CONFIGS, generate

pytestmark = pytest.mark.gpu


def _forward(cfg, inp, passes):
    net = Network(cfg.layers, inp["W"], inp["b"], cfg.in_shape, cfg.batch, keep_sums=False)
    x = dev(inp["x"])
    net.forward(x)
    torch.cuda.synchronize()
    _lib.phase_stamps(reset=True)
    for _ in range(passes):
        out = net.forward(x)
    torch.cuda.synchronize()
    acc, khz = _lib.phase_stamps(reset=True)
    return out, acc, khz


def test_chain_phases_add_up():
    cfg = CONFIGS[2]
    inp = generate(cfg)
    with _lib.stamping_library():
        out, acc, khz = _forward(cfg, inp, 3)
    assert khz > 0
    assert acc[15] == 3 * cfg.batch                        # one workgroup per image and pass
    # each workgroup passes the stamps in phase order: every mean is >= 0, and
    # a workgroup's whole time is above 0 and below a millisecond
    means = [(acc[i + 1] - acc[i]) / acc[15] for i in range(13)]
    assert all(m >= 0 for m in means)
    assert 0 < (acc[13] - acc[0]) / acc[15] / khz * 1e3 < 1000
    ref = Network(cfg.layers, inp["W"], inp["b"], cfg.in_shape, cfg.batch,
                  keep_sums=False).forward(dev(inp["x"]))
    torch.cuda.synchronize()
    assert np.array_equal(host(out), host(ref))


def test_table_block_tiles_counted():
    cfg = CONFIGS[3]
    inp = generate(cfg)
    with _lib.stamping_library():
        _, acc, khz = _forward(cfg, inp, 2)
    b, h, w, _ = (cfg.batch,) + tuple(cfg.in_shape)
    tiles = -(-b * h * w // 64)                            # 64 pixels a tile
    assert acc[31] == 2 * tiles
    assert acc[18] >= acc[17] >= acc[16] > 0
