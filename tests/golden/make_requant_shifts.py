"""Derive the frozen requantisation shifts of the int8 chains.

Calls only the CPU oracle and the seeded generators.  For each layer that
requantises, the shift is the smallest s with |winner| >> s <= 127 over all
k-WTA winners of the seeded batch, the layer's input being the previous
layer's requantised output.  Writes requant_shifts.json next to this file.

    python tests/golden/make_requant_shifts.py
"""
from __future__ import annotations

import dataclasses
import json
import os
import sys

ROOT = os.path.abspath(os.path.join(os.path.dirname(__file__), "..", ".."))
sys.path.insert(0, ROOT)

from oracle import cs_oracle, networks  # noqa: E402
from workloads import CONFIGS, generate  # noqa: E402


def derive(cid: int) -> dict:
    cfg = CONFIGS[cid]
    inp = generate(cfg)
    cur = inp["x"]
    shifts = {}
    for li, spec in enumerate(cfg.layers):
        plain = dataclasses.replace(spec, shift=None)
        r = networks.layer_forward(plain, cur, inp["W"][li], inp["b"][li])
        if spec.shift is not None:
            s = networks.requant_shift(r["acc"][r["win"]])
            shifts[spec.name] = s
            cur = cs_oracle.requant(r["acc"], s, r["win"])
        else:
            cur = r["out"]
    return shifts


def main() -> None:
    out = {str(cid): derive(cid) for cid in sorted(CONFIGS)
           if any(l.shift is not None for l in CONFIGS[cid].layers)}
    path = os.path.join(os.path.dirname(__file__), "requant_shifts.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1, sort_keys=True)
        f.write("\n")
    print(json.dumps(out))


if __name__ == "__main__":
    main()
