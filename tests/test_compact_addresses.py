"""A CPU model of the vectorised compaction kernel's index arithmetic
(compact_vec: 16-byte loads, rows packed 64 / L to a wavefront in groups of L
lanes, or one row per wavefront): every element address it loads lies inside
the input, every list position it writes lies inside its row, and the lists
and counts it produces equal the non-zeros of each row in index order.  The
model follows the kernel statement by statement for the grid the host picks,
including the last wavefront's partial group of rows and the lanes past a
row's last vector."""
from __future__ import annotations

import numpy as np
import pytest


def host_lg(c, E):
    """compact_vec_lg: log2 lanes per row group, or -1."""
    if c % E:
        return -1
    nl = c // E
    if nl > 16:
        return 6
    lg = 0
    while (1 << lg) < nl:
        lg += 1
    return lg


UN = 1            # vector rounds per wavefront round


def put(nl_of, q, lanes_ld, vi_of, run, lg, rows_of, idx, val, c, E):
    """compact_put for all 64 lanes: writes the lists, returns each lane's
    group total."""
    L = 1 << lg
    tot = np.zeros(64, dtype=np.int64)
    for lane in range(64):
        p = lane & (L - 1)
        g0 = lane - p
        incl = int(nl_of[g0:lane + 1].sum())
        pos = run[lane] + incl - nl_of[lane]
        if lane in lanes_ld:
            row = rows_of[lane]
            for e in np.flatnonzero(q[lane] != 0):
                assert 0 <= pos < c                      # inside the row's list
                idx[row, pos] = vi_of[lane] * E + e
                val[row, pos] = q[lane][e]
                pos += 1
        tot[lane] = int(nl_of[g0:g0 + L].sum())
    return tot


def model(x, E, cus=256):
    rows, c = x.shape
    lg = host_lg(c, E)
    assert lg >= 0
    rpw = 1 if lg == 6 else (64 >> lg) * UN            # rows per wavefront round (host)
    waves = -(-rows // rpw)
    blocks = min(-(-waves // 4), cus * 16)
    nwaves = blocks * 4
    NL = c // E
    L = 1 << lg
    idx = np.full((rows, c), -1, dtype=np.int64)
    val = np.zeros((rows, c), dtype=x.dtype)
    cnt = np.full(rows, -1, dtype=np.int64)
    flat = x.reshape(-1)
    loads = []

    def load(row, vi):
        a = row * c + vi * E                            # element address of the 16-byte load
        assert 0 <= a and a + E <= rows * c
        loads.append(a)
        return flat[a:a + E]

    for w in range(nwaves):
        if lg <= 4:
            g = 64 >> lg
            for r0 in range(w * g * UN, rows, nwaves * g * UN):
                for u in range(UN):
                    q, nl, rows_of, vi_of = {}, np.zeros(64, dtype=np.int64), {}, {}
                    for lane in range(64):
                        sub, p = lane >> lg, lane & (L - 1)
                        row = r0 + u * g + sub
                        if row < rows and p < NL:
                            q[lane] = load(row, p)
                            nl[lane] = int((q[lane] != 0).sum())
                            rows_of[lane], vi_of[lane] = row, p
                    tot = put(nl, q, q, vi_of, np.zeros(64, dtype=np.int64), lg, rows_of, idx,
                              val, c, E)
                    for lane in range(64):
                        sub, p = lane >> lg, lane & (L - 1)
                        row = r0 + u * g + sub
                        if row < rows and p == 0:
                            cnt[row] = tot[lane]
        else:
            for row in range(w, rows, nwaves):
                run = np.zeros(64, dtype=np.int64)
                for v0 in range(0, NL, 64 * UN):
                    for u in range(UN):
                        q, nl, rows_of, vi_of = {}, np.zeros(64, dtype=np.int64), {}, {}
                        for lane in range(64):
                            vi = v0 + u * 64 + lane
                            if vi < NL:
                                q[lane] = load(row, vi)
                                nl[lane] = int((q[lane] != 0).sum())
                                rows_of[lane], vi_of[lane] = row, vi
                        run = run + put(nl, q, q, vi_of, run, 6, rows_of, idx, val, c, E)
                cnt[row] = run[0]
    return idx, val, cnt, loads


@pytest.mark.parametrize("rows,c,dtype,nnz", [
    (37, 96, np.int8, 12),        # 6 vectors per row, groups of 8 lanes, 8 rows per wavefront
    (29, 64, np.float32, 7),      # 16 lanes per row, 4 rows per wavefront, partial last wavefront
    (5, 1024, np.float32, 102),   # one row per wavefront, 4 rounds of 64 vectors
    (3, 2048, np.float32, 300),   # one row per wavefront, 8 rounds (two batches of 4)
    (300, 64, np.float32, 7),     # several row groups per wavefront round
    (7, 512, np.int8, 64),        # 32 vectors: one row per wavefront, lanes past the row idle
    (11, 16, np.int8, 16),        # one vector per row (a full row), 64 rows per wavefront
    (3, 4, np.float32, 2),        # one vector per row
    (9, 96, np.float32, 30),      # 24 vectors: one row per wavefront
    (3, 65532, np.float32, 2000), # the widest fp32 row that is whole vectors: 16383 of them
    (2, 4096, np.int8, 300),      # 256 vectors of 16 int8
])
def test_compact_vec_model(rows, c, dtype, nnz):
    r = np.random.default_rng(rows * 1000 + c)
    x = np.zeros((rows, c), dtype=dtype)
    for i in range(rows):
        k = 0 if i % 5 == 2 else nnz            # some empty rows
        pos = r.choice(c, size=k, replace=False)
        x[i, pos] = r.integers(1, 100, size=k) if dtype == np.int8 else r.normal(size=k)
    E = 16 // np.dtype(dtype).itemsize
    idx, val, cnt, loads = model(x, E)
    # every vector of every row loaded exactly once
    assert sorted(loads) == list(range(0, rows * c, E))
    for i in range(rows):
        nz = np.flatnonzero(x[i])
        assert cnt[i] == len(nz)
        assert np.array_equal(idx[i, :cnt[i]], nz)
        assert np.array_equal(val[i, :cnt[i]], x[i, nz])


def test_compact_vec_refuses_ragged_rows():
    assert host_lg(100, 16) == -1 and host_lg(6, 4) == -1
    assert host_lg(96, 16) == 3 and host_lg(64, 4) == 4 and host_lg(1024, 4) == 6
