"""Complementary Sparsity sparse-sparse layer for AMD Instinct MI355X (gfx950).

Pack (host), compaction, multiply-route-sum and k-WTA run as hand-written HIP
kernels behind the C ABI of include/cs.h (libcs.so, built in-tree by
`python -m paper_2112_13896_amd.build`).  The Python side only marshals
arguments: `ops` wraps each entry point, `network.Network` chains layers.
"""
__all__ = ["ops", "network", "build"]
