"""A CPU model of the output-stationary chain layer's index arithmetic
(gather_body, the second layer of the keyword-spotting chain): for each shape
the host plan accepts, every global address the kernel forms lies inside its
buffer, every LDS access inside its region of the planned allocation, every
routed add inside the accumulator blocks, and the sums the model's adds build
equal the convolution of the lists with the weights the packed table encodes
(each packed slot of set g belongs to kernel g*n + kid).  The model follows
the kernel's statements for every thread of the workgroup: the staging loads
(clamped in range), the table pieces' split by set pairs, the wavefronts'
(tap row, 64-pixel block) jobs with their padding checks, and the pooled
transpose."""
from __future__ import annotations

import numpy as np
import pytest

BD = 1024          # threads per workgroup
GC = 64            # input channels
CAP = 8            # list slots per input pixel
BLK_B = 64 * 64 * 4


def r16(v):
    return (v + 15) // 16 * 16


def plan(H, W, KW, P, c_out, n, pool):
    """The host plan's layout (None where it declines the shape)."""
    G = c_out // n
    Ho, Wo = H + 2 * P - KW + 1, W + 2 * P - KW + 1
    if KW not in (3, 5) or G != 4 or c_out > 64 or pool not in (1, 2):
        return None
    npix, nout = H * W, Ho * Wo
    if npix < 1 or npix > BD or nout < 1:
        return None
    NH = (nout + 63) // 64
    if KW * NH > BD // 64:
        return None
    nitems = (Ho // pool) * (Wo // pool)
    if nitems < 1:
        return None
    o_tab = NH * BLK_B
    o_ent = o_tab + (G // 2) * KW * KW * GC * 4
    o_cnt = o_ent + npix * CAP * 2
    o_bias = o_cnt + r16(npix * 4)
    o_pt = o_bias + r16(c_out * 4)
    total = o_pt + r16(nitems * (c_out + 1) * 4)
    if total > 160 * 1024:
        return None
    return dict(G=G, Ho=Ho, Wo=Wo, NH=NH, nitems=nitems, npix=npix, o_tab=o_tab, o_ent=o_ent,
                o_cnt=o_cnt, o_bias=o_bias, o_pt=o_pt, total=total)


class Lds:
    """Byte-addressed LDS with region checks."""

    def __init__(self, pl):
        self.pl = pl
        self.regions = {
            "acc": (0, pl["o_tab"]),
            "tab": (pl["o_tab"], pl["o_ent"]),
            "ent": (pl["o_ent"], pl["o_cnt"]),
            "cnt": (pl["o_cnt"], pl["o_bias"]),
            "bias": (pl["o_bias"], pl["o_pt"]),
            "pt": (pl["o_pt"], pl["total"]),
        }

    def check(self, region, addr, nbytes):
        lo, hi = self.regions[region]
        a = np.asarray(addr)
        assert (a >= lo).all() and (a + nbytes <= hi).all(), (region, a.min(), a.max(), lo, hi)
        assert (a % min(nbytes, 16) == 0).all(), (region, "alignment")


def model_image(H, W, KW, P, c_out, n, pool, cnt, li, lv, aug16, B, blk):
    """Runs one workgroup (image blk) of the model; returns the accumulator
    sums [c_out][Ho*Wo] its routed adds build."""
    pl = plan(H, W, KW, P, c_out, n, pool)
    G, NH, npix = pl["G"], pl["NH"], pl["npix"]
    Ho, Wo = pl["Ho"], pl["Wo"]
    T, NPR = KW * KW, G // 2
    lds = Lds(pl)
    tid = np.arange(BD)
    prow0 = blk * npix
    # ---- staging loads (global indices in elements of the buffers)
    m = tid[tid < npix]
    assert (prow0 + m < B * npix).all()
    npairs = npix * CAP // 2
    PRE = 4
    assert npairs <= PRE * BD
    for u in range(PRE):
        mm = u * BD + tid
        mc = np.minimum(mm, npairs - 1)
        # u32 pairs of lidx and u16 pairs of lval from element prow0*CAP
        assert ((prow0 * CAP + 2 * mc + 1) < B * npix * CAP).all()
    N16 = T * GC * NPR // 4
    TPRE = (N16 + BD - 1) // BD
    aug_bytes = aug16.size * 2
    for u in range(TPRE):
        mm = u * BD + tid
        assert (16 * np.minimum(mm, N16 - 1) + 16 <= aug_bytes).all()
    # ---- staging stores
    words = aug16.reshape(-1).view(np.uint32)            # the packed tensor as 32-bit words
    tab = np.zeros(NPR * T * GC, dtype=np.uint32)

    def chan(w, pr):
        k0, k1 = (w >> 8) & 0xFF, w >> 24
        c0 = 2 * pr * n + min(int(k0), n - 1)
        c1 = (2 * pr + 1) * n + min(int(k1), n - 1)
        return (int(w) & 0x00FF00FF) | c0 << 8 | c1 << 24

    for u in range(TPRE):
        for t in range(BD):
            mp = u * BD + t
            if mp >= N16:
                continue
            v = words[4 * mp:4 * mp + 4]
            if NPR == 2:
                lds.check("tab", pl["o_tab"] + 4 * (2 * mp), 8)
                lds.check("tab", pl["o_tab"] + 4 * (T * GC + 2 * mp), 8)
                tab[2 * mp], tab[2 * mp + 1] = chan(v[0], 0), chan(v[2], 0)
                tab[T * GC + 2 * mp], tab[T * GC + 2 * mp + 1] = chan(v[1], 1), chan(v[3], 1)
    lds.check("acc", 16 * np.arange(NH * (BLK_B // 16)), 16)
    lds.check("bias", pl["o_bias"] + 4 * np.arange(c_out), 4)
    lds.check("cnt", pl["o_cnt"] + 4 * np.arange(npix), 4)
    lds.check("ent", pl["o_ent"] + 4 * np.arange(npairs), 4)
    cnt_s = np.clip(cnt[prow0:prow0 + npix], 0, CAP)
    ent = np.zeros((npix, CAP), dtype=np.uint32)       # channel | value << 8
    for q in range(npix):
        for j in range(CAP):
            e = (prow0 + q) * CAP + j
            ent[q, j] = (int(li[e]) & 0x3F) | (int(lv[e]) & 0xFF) << 8
    # ---- products: wavefront wv < KW*NH, lanes = 64 output pixels
    acc = np.zeros(NH * 64 * 64, dtype=np.int64)       # int32 words of [block][channel][pixel]
    lane = np.arange(64)
    for wv in range(KW * NH):
        ky, hb = wv // NH, wv % NH
        p = hb * 64 + lane
        live = p < Ho * Wo
        oy, ox = p // Wo, p % Wo
        iy = oy + ky - P
        rok = live & (iy >= 0) & (iy < H)
        abase = hb * BLK_B + lane * 4
        tabb = pl["o_tab"] + ky * KW * GC * 4
        for kx in range(KW):
            ix = ox + kx - P
            ok = rok & (ix >= 0) & (ix < W)
            q = np.where(ok, iy * W + ix, 0)
            lds.check("cnt", pl["o_cnt"] + 4 * q, 4)
            lds.check("ent", pl["o_ent"] + 16 * q, 16)
            cq = np.where(ok, cnt_s[q], 0)
            for j in range(CAP):
                e = ent[q, j]
                ch = e & 0x3F
                x = ((e >> 8) & 0xFF).astype(np.int64)
                x = np.where(x >= 128, x - 256, x)
                for pr in range(NPR):
                    ta = tabb + kx * GC * 4 + ch * 4 + pr * T * GC * 4
                    lds.check("tab", ta, 4)
                    tw = tab[(ta - pl["o_tab"]) // 4]
                    for hf in range(2):
                        wk = tw >> (16 * hf)
                        och = (wk >> 8) & 0xFF
                        w = (wk & 0xFF).astype(np.int64)
                        w = np.where(w >= 128, w - 256, w)
                        assert (och < c_out).all()
                        addr = abase + och * 256
                        lds.check("acc", addr, 4)
                        on = j < cq
                        np.add.at(acc, (addr[on] // 4), (x * w)[on])
    # ---- epilogue reads: the pooled transpose and the k-WTA tile
    nitems, Wp = pl["nitems"], Wo // pool
    t = np.arange(nitems * c_out)
    ch, it = t // nitems, t % nitems
    pr_, pc = it // Wp, it % Wp
    px = pr_ * pool * Wo + pc * pool
    for d in ([0] if pool == 1 else [0, 1, Wo, Wo + 1]):
        pp = px + d
        assert (pp < Ho * Wo).all()
        lds.check("acc", (pp >> 6) * BLK_B + ch * 256 + (pp & 63) * 4, 4)
    lds.check("pt", pl["o_pt"] + 4 * (it * (c_out + 1) + ch), 4)
    # sums as [channel][pixel]
    out = np.zeros((c_out, Ho * Wo), dtype=np.int64)
    for pp in range(Ho * Wo):
        out[:, pp] = acc.reshape(NH, 64, 64)[pp // 64, :c_out, pp % 64]
    return out


def reference(H, W, KW, P, c_out, n, cnt, li, lv, aug16, blk):
    """The convolution of image blk's lists with the weights the table
    encodes (slot r = (ky*KW + kx)*C + c of set g belongs to kernel g*n + kid)."""
    G = c_out // n
    R = KW * KW * GC
    Wd = np.zeros((c_out, R), dtype=np.int64)
    a = aug16.reshape(R, G)
    for r in range(R):
        for g in range(G):
            w = int(a[r, g] & 0xFF)
            w = w - 256 if w >= 128 else w
            Wd[g * n + int(a[r, g] >> 8), r] = w
    xd = np.zeros((H, W, GC), dtype=np.int64)
    for q in range(H * W):
        for j in range(min(max(int(cnt[blk * H * W + q]), 0), CAP)):
            e = (blk * H * W + q) * CAP + j
            v = int(lv[e])
            xd[q // W, q % W, int(li[e])] += v - 256 if v >= 128 else v
    Ho, Wo = H + 2 * P - KW + 1, W + 2 * P - KW + 1
    out = np.zeros((c_out, Ho * Wo), dtype=np.int64)
    for oy in range(Ho):
        for ox in range(Wo):
            for ky in range(KW):
                for kx in range(KW):
                    iy, ix = oy + ky - P, ox + kx - P
                    if 0 <= iy < H and 0 <= ix < W:
                        r0 = (ky * KW + kx) * GC
                        out[:, oy * Wo + ox] += Wd[:, r0:r0 + GC] @ xd[iy, ix]
    return out


# (H, W, KW, P, c_out, n, pool): the keyword-spotting shape, the GPU test shapes,
# a map whose output fills whole 64-pixel blocks, and the plan's largest block count
SHAPES = [
    (14, 14, 5, 0, 64, 16, 2),
    (8, 8, 3, 1, 64, 16, 1),
    (14, 14, 3, 1, 48, 12, 2),
    (8, 16, 5, 2, 64, 16, 2),
    (16, 16, 3, 0, 32, 8, 1),
]


@pytest.mark.parametrize("shape", SHAPES, ids=[str(s) for s in SHAPES])
def test_gather_addresses_and_sums(shape):
    H, W, KW, P, c_out, n, pool = shape
    pl = plan(H, W, KW, P, c_out, n, pool)
    assert pl is not None
    B = 2
    r = np.random.default_rng(13 + H * W + KW)
    npix = H * W
    # lists: counts 0..8 (some rows empty, some full), distinct channels, non-zero values;
    # slots past a count hold stale entries (any channel, any value)
    cnt = r.integers(0, CAP + 1, size=B * npix).astype(np.int32)
    cnt[::7] = CAP
    cnt[3::11] = 0
    li = r.integers(0, 256, size=B * npix * CAP).astype(np.uint16)
    lv = r.integers(0, 256, size=B * npix * CAP).astype(np.uint8)
    for q in range(B * npix):
        ch = r.choice(GC, size=CAP, replace=False)
        li[q * CAP:q * CAP + cnt[q]] = ch[:cnt[q]]
        vals = r.integers(1, 128, size=CAP) * r.choice([-1, 1], size=CAP)
        lv[q * CAP:q * CAP + cnt[q]] = (vals[:cnt[q]] & 0xFF).astype(np.uint8)
    G = c_out // n
    R = KW * KW * GC
    w = r.integers(1, 128, size=(R, G)) * r.choice([-1, 1], size=(R, G))
    kid = r.integers(0, n, size=(R, G))
    aug16 = ((w & 0xFF) | (kid << 8)).astype(np.uint16)
    for blk in range(B):
        got = model_image(H, W, KW, P, c_out, n, pool, cnt, li, lv, aug16, B, blk)
        want = reference(H, W, KW, P, c_out, n, cnt, li, lv, aug16, blk)
        assert np.array_equal(got, want)


def test_plan_declines_what_the_kernel_cannot_hold():
    assert plan(14, 14, 7, 0, 64, 16, 2) is None        # 7x7 window
    assert plan(14, 14, 5, 0, 64, 8, 2) is None         # eight sets
    assert plan(40, 40, 3, 1, 64, 16, 2) is None        # more than 1024 input pixels
    assert plan(30, 30, 5, 2, 64, 16, 2) is None        # 15 blocks x 5 tap rows > 16 wavefronts
