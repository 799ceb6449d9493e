"""Independent k-WTA procedures taken from the paper's hardware description.

These are used only to pin the oracle's sort-based k-WTA: they follow the
structures of Section 3.3.3 rather than a sort.

* local k-WTA: a row is split into sub-vectors of 8, each sub-vector goes
  through an 8-input sorting network (19 comparators, depth 6), the sorted
  sub-vectors sit in FIFOs with the largest at the front, and K times a
  comparator tree finds the largest front element, which is popped;
* global k-WTA on 8-bit data: a 256-bin histogram (built as several partial
  histograms, one per parallel lane) is read from the largest value down until
  the running count reaches K; everything >= that threshold passes.

The sorting network is Batcher's odd-even merge sort, built recursively.
"""
from __future__ import annotations

import numpy as np


def _merge(lo: int, n: int, r: int, out: list) -> None:
    """Odd-even merge of the two sorted halves of positions lo..lo+n-1 taken
    with stride r."""
    step = 2 * r
    if step < n:
        _merge(lo, n, step, out)          # even subsequence
        _merge(lo + r, n, step, out)      # odd subsequence
        for i in range(lo + r, lo + n - r, step):
            out.append((i, i + r))
    else:
        out.append((lo, lo + r))


def _sort(lo: int, n: int, out: list) -> None:
    if n > 1:
        half = n // 2
        _sort(lo, half, out)
        _sort(lo + half, half, out)
        _merge(lo, n, 1, out)


def batcher_network(n: int) -> list:
    """Comparator list (a, b), a < b, of Batcher's odd-even merge sort on n = 2^m inputs."""
    assert n & (n - 1) == 0
    out: list = []
    _sort(0, n, out)
    return out


def network_depth(comps: list, n: int) -> int:
    """Number of parallel layers when each comparator runs as early as possible."""
    ready = [0] * n
    depth = 0
    for a, b in comps:
        t = max(ready[a], ready[b]) + 1
        ready[a] = ready[b] = t
        depth = max(depth, t)
    return depth


def _greater(x, y) -> bool:
    """Order used for winners: larger value first, then lower index first.
    x and y are (value, index)."""
    return x[0] > y[0] or (x[0] == y[0] and x[1] < y[1])


def sort_desc(items: list, comps: list) -> list:
    """Run the network so position 0 ends with the largest item."""
    v = list(items)
    for a, b in comps:
        if _greater(v[b], v[a]):
            v[a], v[b] = v[b], v[a]
    return v


def local_kwta_fifo(row: np.ndarray, k: int, sub: int = 8) -> np.ndarray:
    """Winner mask of one row via sorted sub-vector FIFOs and a comparator tree."""
    c = len(row)
    assert c % sub == 0
    comps = batcher_network(sub)
    fifos = []
    for s in range(c // sub):
        items = [(row[s * sub + j].item(), s * sub + j) for j in range(sub)]
        fifos.append(sort_desc(items, comps))
    mask = np.zeros(c, dtype=bool)
    for _ in range(k):
        # comparator tree over the FIFO fronts
        fronts = [(f[0], i) for i, f in enumerate(fifos) if f]
        while len(fronts) > 1:
            nxt = []
            for j in range(0, len(fronts), 2):
                if j + 1 == len(fronts):
                    nxt.append(fronts[j])
                else:
                    a, b = fronts[j], fronts[j + 1]
                    nxt.append(a if _greater(a[0], b[0]) else b)
            fronts = nxt
        item, fi = fronts[0]
        mask[item[1]] = True
        fifos[fi].pop(0)
    return mask


def global_kwta_histogram(row_u8: np.ndarray, k: int, ways: int = 5):
    """Threshold and pass mask of the histogram method on unsigned 8-bit data.

    The row is read as blocks of `ways` elements; element j of a block
    increments histogram j.  The histograms are summed, then read from bin 255
    down until the running count reaches k; values >= that bin pass.
    """
    row = np.asarray(row_u8, dtype=np.int64)
    assert row.min() >= 0 and row.max() <= 255 and len(row) % ways == 0
    hists = np.zeros((ways, 256), dtype=np.int64)
    for blk in range(len(row) // ways):
        for j in range(ways):
            hists[j, row[blk * ways + j]] += 1
    hist = hists.sum(axis=0)
    accum = 0
    thresh = 0
    for v in range(255, -1, -1):
        accum += hist[v]
        if accum >= k:
            thresh = v
            break
    return thresh, row >= thresh
