#!/usr/bin/env python3
"""Throughput of the Complementary Sparsity sparse-sparse layer chain on one GPU.

    python bench.py [--steps K] [--warmup W] [--config C] [--also 1,3,4,5]

A step is one pass of the whole chain over one batch: per layer, compaction
of the activations into (index, value) lists (dense inputs only),
multiply-route-sum (+ bias, + 2x2 max-pool), k-WTA (+ int8 requantisation)
emitting the next layer's lists; where a layer's packed table fits one
workgroup the last three are one kernel and the sums never reach HBM.  Inputs
are resident in HBM when the timed region starts.

Cache-cold protocol: the chain rotates among buffer sets (input + every
intermediate), as many as make the bytes one pass touches (the sum of its
launches' algorithmic bytes) times the number of sets exceed 512 MiB, so a set
comes round again only after twice the 256 MiB Infinity Cache of other data;
and a 512 MiB buffer is read before every timed region.  The K timed passes
(K <= 256; else one pass per buffer set) are recorded once into a HIP graph (a
serving loop's batches in one launch), pass i on buffer set i mod sets, in
three schedules: one after another; each pass's first kernel on one stream and
the rest on a second, so the next batch's first kernel runs beside the current
batch's later ones; or whole passes on the two streams in turn.  The fastest
in a few warm-up replays is timed (`schedule`); the same K passes with one
graph launch each are timed after and reported beside it.  Per-kernel
durations (and the roofline of the dominant kernel) come from graphs holding
one launch of that kernel per buffer set, each replay after the scrub, timed
with HIP events on the replaying stream.

Default workload: the keyword-spotting CNN of Table 1 (config 2, int8, batch
256), then the other workloads (`--also`), each reported under "workloads"
with its step time and every kernel's duration and HBM fraction.  Prints ONE
JSON line on stdout; progress goes to stderr.  `--eager-passes N` only runs N
eager passes (for profiler runs); `--calibrate-copy MIB` times a device copy.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "sparse-sparse layer samples/s + dense-equiv GMAC/s; achieved HBM GB/s (1 GPU)"
HBM_PEAK_GBS = 8000.0               # MI355X HBM3E, published
KREP = 20                           # launches per graph when timing one kernel
INT_VALU_PEAK_TOPS = 78.6           # 256 CU x 64 lanes x 2.4 GHz x (mul+add) int32 VALU
FP32_VALU_PEAK_TFLOPS = 157.3       # published fp32 vector peak


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def conv_products(cnt_map: np.ndarray, pl, groups: int) -> int:
    """Products the multiply-route-sum kernel performs: for every conv output
    pixel (before pooling), the non-zeros under its window, times G."""
    b, h, w = cnt_map.shape
    ho = (h + 2 * pl.pad - pl.kh) // pl.stride + 1
    wo = (w + 2 * pl.pad - pl.kw) // pl.stride + 1
    pad = np.zeros((b, h + 2 * pl.pad, w + 2 * pl.pad), dtype=np.int64)
    pad[:, pl.pad:pl.pad + h, pl.pad:pl.pad + w] = cnt_map
    tot = 0
    for ky in range(pl.kh):
        for kx in range(pl.kw):
            tot += int(pad[:, ky:ky + pl.stride * (ho - 1) + 1:pl.stride,
                           kx:kx + pl.stride * (wo - 1) + 1:pl.stride].sum())
    return tot * groups


def layer_costs(net, bufs, cfg) -> dict:
    """Algorithmic bytes (and products) per launch of every kernel, from the
    actual non-zero counts of this batch.  "bytes" is what the launch must move
    (its inputs, the packed table, the bias and what it writes: lists or dense
    outputs); "bytes_dense_out" counts a layer as if it wrote its dense sums
    after pooling instead (lists or dense input in + table + bias + 4 B per
    output), the per-layer form of the multiply-route-sum byte count."""
    import torch
    costs = {}
    dense8 = {}
    for li, (p, pl) in enumerate(zip(net.packed, net.plans)):
        s = p.spec
        is_int = p.aug.dtype == torch.int16          # int8 weights/activations
        es = 1 if is_int else 4
        b, h, w, c = pl.geo
        rows = b * h * w
        out_elems = int(np.prod(pl.out_shape))
        table = p.aug.numel() * p.aug.element_size()   # the augmented tensor
        bias = 0 if p.bias is None else s.c_out * 4
        if pl.dense_kernel:
            # sparse-dense: every input element is read and multiplied
            cnt = np.full(rows, c, dtype=np.int64)
            mrs_bytes = rows * c * es + table + bias + out_elems * 4
        else:
            src = bufs.lists[li - 1][2] if pl.in_lists else bufs.cnt[li]
            cnt = src.cpu().numpy().astype(np.int64)
            nnz = int(cnt.sum())
            lists = nnz * (2 + es) + rows * 4
            if not pl.in_lists:
                costs[f"{s.name}.compact"] = {"bytes": rows * c * es + lists}
            mrs_bytes = lists + table + bias + out_elems * 4
        dense8[s.name] = mrs_bytes
        prods = conv_products(cnt.reshape(b, h, w), pl, s.c_out // s.n)
        if s.k is not None and pl.dense_kernel:
            # one launch: dense input, weights, the k-WTA output (lists or dense)
            ob = 1 if s.shift is not None else 4
            if pl.emit_lists:
                lc = bufs.lists[li][2].cpu().numpy().astype(np.int64)
                obytes = int(lc.sum()) * (2 + ob) + len(lc) * 4
            else:
                obytes = out_elems * ob
            sums = out_elems * 4 if net.keep_sums else 0
            costs[f"{s.name}.dense_kwta"] = {"bytes": rows * c * es + table + bias + sums + obytes,
                                             "products": prods, "int": is_int,
                                             "bytes_dense_out": mrs_bytes}
            continue
        if s.k is not None and not pl.dense_kernel:
            # one launch: lists in, table, bias, the k-WTA output (lists or
            # dense); the sums are written only when the network keeps them
            ob = 1 if s.shift is not None else 4
            if pl.emit_lists:
                lc = bufs.lists[li][2].cpu().numpy().astype(np.int64)
                obytes = int(lc.sum()) * (2 + ob) + len(lc) * 4
            else:
                obytes = out_elems * ob
            sums = out_elems * 4 if net.keep_sums else 0
            costs[f"{s.name}.mrs_kwta"] = {"bytes": mrs_bytes - out_elems * 4 + sums + obytes,
                                           "products": prods, "int": is_int,
                                           "bytes_dense_out": mrs_bytes}
            continue
        costs[f"{s.name}.mrs"] = {"bytes": mrs_bytes, "products": prods, "bytes_dense_out": mrs_bytes,
                                  "int": is_int, "lists_in": 0 if pl.dense_kernel else lists}
        if s.k is not None:
            if pl.emit_lists:
                lc = bufs.lists[li][2].cpu().numpy().astype(np.int64)
                ob = 1 if s.shift is not None else 4
                costs[f"{s.name}.kwta"] = {"bytes": out_elems * 4 + int(lc.sum()) * (2 + ob) + len(lc) * 4}
            else:
                ob = 1 if s.shift is not None else 4
                costs[f"{s.name}.kwta"] = {"bytes": out_elems * (4 + ob)}
    # a call that runs several layers: all their bytes, less the later layers'
    # reads of lists that stay on chip
    names = [p.spec.name for p in net.packed]
    for li, pl in enumerate(net.plans):
        if pl.fuse_next2:
            c = costs[f"{names[li]}.mrs_kwta"]
            a = costs[f"{names[li + 1]}.mrs_kwta"]
            z = costs[f"{names[li + 2]}.mrs"]
            costs[f"{names[li]}.mrs_kwta+{names[li + 1]}.mrs_kwta+{names[li + 2]}.mrs"] = {
                "bytes": c["bytes"] + a["bytes"] + z["bytes"] - z["lists_in"],
                "products": c["products"] + a["products"] + z["products"], "int": c["int"],
                "bytes_dense_out": sum(dense8[names[li + i]] for i in range(3))}
    for li, pl in enumerate(net.plans):
        if pl.fuse_next3:
            # the dense first layer and the three-layer tail: bytes of both;
            # the products counted are the routed ones (VALU work), the first
            # layer's dense multiply-adds run on the matrix cores
            d = costs[f"{names[li]}.dense_kwta"]
            t = costs[f"{names[li + 1]}.mrs_kwta+{names[li + 2]}.mrs_kwta+{names[li + 3]}.mrs"]
            costs[f"{names[li]}.dense_kwta+{names[li + 1]}.mrs_kwta+{names[li + 2]}.mrs_kwta+"
                  f"{names[li + 3]}.mrs"] = {
                "bytes": d["bytes"] + t["bytes"], "products": t["products"], "int": t["int"],
                "mfma_macs": d["products"],
                "bytes_dense_out": sum(dense8[names[li + i]] for i in range(4))}
    for li, pl in enumerate(net.plans):
        if pl.fuse_next:
            a = costs[f"{names[li]}.mrs_kwta"]
            z = costs[f"{names[li + 1]}.mrs"]
            costs[f"{names[li]}.mrs_kwta+{names[li + 1]}.mrs"] = {
                "bytes": a["bytes"] + z["bytes"] - z["lists_in"],
                "products": a["products"] + z["products"], "int": a["int"],
                "bytes_dense_out": dense8[names[li]] + dense8[names[li + 1]]}
    return costs


def capture_passes(net, xs, sets, steps: int, mode: str):
    """One graph of `steps` passes, pass i on buffer set i % len(sets), in one
    of three schedules: "sequential" (one stream), "overlapped" (a pass's
    first launch on the capture stream, the rest after it on a second stream)
    or "alternate" (whole passes on the two streams in turn).  Two passes in
    flight at once always use different buffer sets: at each wrap of the sets
    the two streams wait for each other."""
    import torch
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()                      # default priority
    nsets = len(sets)
    with torch.cuda.graph(g):
        main = torch.cuda.current_stream()
        side.wait_stream(main)
        for i in range(steps):
            j = i % nsets
            calls = [c for li in range(len(net.packed))
                     for _, c in net.launches(li, xs[j] if li == 0 else None, sets[j])]
            if mode == "sequential":
                for c in calls:
                    c()
                continue
            if i > 0 and j == 0:                    # set 0 .. are written again
                main.wait_stream(side)
                side.wait_stream(main)
            if mode == "alternate":
                with torch.cuda.stream(main if i % 2 == 0 else side):
                    for c in calls:
                        c()
                continue
            calls[0]()
            if len(calls) > 1:
                side.wait_stream(main)
                with torch.cuda.stream(side):
                    for c in calls[1:]:
                        c()
        main.wait_stream(side)
    return g


def dense_macs(cfg) -> int:
    shape = (cfg.batch,) + tuple(cfg.in_shape)
    tot = 0
    for s in cfg.layers:
        if s.kind == "conv":
            b, h, w, c = shape
            ho = (h + 2 * s.pad - s.kh) // s.stride + 1
            wo = (w + 2 * s.pad - s.kw) // s.stride + 1
            tot += b * ho * wo * s.c_out * s.kh * s.kw * c
            shape = (b, ho // s.pool, wo // s.pool, s.c_out)
        else:
            b = shape[0]
            tot += b * int(np.prod(shape[1:])) * s.c_out
            shape = (b, s.c_out)
    return tot


def roofline_for(name: str, cost: dict, ms: float) -> dict:
    sec = ms * 1e-3
    gbs = cost["bytes"] / sec / 1e9
    extra = {}
    if "bytes_dense_out" in cost:
        extra["hbm_frac_dense_out"] = round(cost["bytes_dense_out"] / sec / 1e9 / HBM_PEAK_GBS, 4)
    if "products" in cost:
        # ridge: products per byte above which the VALU roof is the lower one
        if cost["int"]:
            peak_ops = INT_VALU_PEAK_TOPS
        else:
            peak_ops = FP32_VALU_PEAK_TFLOPS
        ops = 2.0 * cost["products"]
        intensity = ops / cost["bytes"]
        ridge = peak_ops * 1e12 / (HBM_PEAK_GBS * 1e9)
        if intensity > ridge:
            ach = ops / sec / 1e12
            return {"bound": "alu", "achieved": round(ach, 3), "peak": peak_ops,
                    "unit": "TOP/s" if cost["int"] else "TFLOP/s", "frac": round(ach / peak_ops, 4),
                    "traffic": None, "kernel": name, "us": round(ms * 1e3, 2),
                    "algorithmic_bytes": cost["bytes"], "products": cost["products"],
                    "hbm_gbs": round(gbs, 1), "hbm_frac": round(gbs / HBM_PEAK_GBS, 4), **extra,
                    **({"mfma_macs": cost["mfma_macs"]} if "mfma_macs" in cost else {})}
    return {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None, "kernel": name,
            "us": round(ms * 1e3, 2), "algorithmic_bytes": cost["bytes"], **extra,
            **({"products": cost["products"]} if "products" in cost else {})}


def load_traffic(kernel: str, workload: str):
    """HBM bytes per launch measured with rocprofv3 counters (FETCH_SIZE and
    WRITE_SIZE scaled by a copy-kernel calibration), if a record for exactly
    this kernel source is committed; else None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
        from paper_2112_13896_amd import build as b
        if rec.get("source_digest") != b.source_digest():
            return None
        return rec.get("kernels", {}).get(workload, {}).get(kernel)
    except Exception:
        return None


def cpu_model() -> str:
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_rate(cfg, inp, seconds: float):
    from oracle import networks
    reps, t0 = 0, time.perf_counter()
    while True:
        networks.run_chain(cfg.layers, inp["x"], inp["W"], inp["b"])
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds or reps >= 50:
            break
    return reps, el


def cpu_baseline(cfg, inp, seconds: float) -> dict:
    """The CPU oracle (as it stands) on whole batches of the workload, repeated
    for about `seconds`: once with the BLAS threads numpy starts with (all
    host cores), once on one core (one BLAS thread, the process pinned to
    one CPU).  samples/s over all repetitions."""
    from threadpoolctl import threadpool_info, threadpool_limits
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    reps, el = _oracle_rate(cfg, inp, seconds)
    res = {"value": round(reps * cfg.batch / el, 2), "unit": "samples/s", "cores": int(threads),
           "kind": "oracle", "cpu_model": cpu_model(), "host_cpus": os.cpu_count(),
           "sample": f"{reps} x full batch of {cfg.batch} ({cfg.name}), float64 numpy oracle, "
                     f"{el:.1f} s, BLAS threads {threads}"}
    aff = os.sched_getaffinity(0)
    try:
        os.sched_setaffinity(0, {min(aff)})
        with threadpool_limits(limits=1):
            reps1, el1 = _oracle_rate(cfg, inp, seconds)
    finally:
        os.sched_setaffinity(0, aff)
    res["one_core"] = {"value": round(reps1 * cfg.batch / el1, 2), "unit": "samples/s",
                       "cores": 1, "sample": f"{reps1} x full batch of {cfg.batch}, {el1:.1f} s, "
                                             "one BLAS thread, pinned to one CPU"}
    return res


def ab_reorder(cfg, inp, x, kernel_ms, breakdown) -> dict:
    """The first layer by reordering (cs_conv2d_reorder_kwta, the support of
    every output gathered from the dense input) against the routed launches
    of the same layer (compaction + multiply-route-sum with k-WTA)."""
    import torch
    from paper_2112_13896_amd import ops

    spec = cfg.layers[0]
    if not (cfg.dtype == "f32" and spec.kind == "conv" and spec.c_out == 64 and spec.stride == 1
            and spec.pool == 1 and spec.k is not None and spec.k <= 32):
        return {"layer": spec.name, "supported": False}
    W = inp["W"][0]
    aug, _ = ops.pack(W.reshape(spec.c_out, -1), spec.n)
    table = torch.from_numpy(ops.reorder_table(aug, spec.kh, spec.kw, spec.c_in, spec.c_out,
                                               spec.n)).cuda()
    bias = None if inp["b"][0] is None else torch.from_numpy(inp["b"][0]).cuda()
    rows = x.shape[0] * x.shape[1] * x.shape[2]
    cap = ops.list_capacity(spec.k)
    lists = (torch.empty((rows, cap), dtype=torch.int16, device="cuda"),
             torch.empty((rows, cap), dtype=torch.float32, device="cuda"),
             torch.empty((rows,), dtype=torch.int32, device="cuda"))
    y = torch.empty(x.shape[:3] + (spec.c_out,), dtype=torch.float32, device="cuda")

    def call():
        ops.conv2d_reorder_kwta(x, table, spec.kh, spec.kw, spec.pad, bias, k=spec.k, y=y,
                                keep_sums=False, lists=lists)
    call()
    routed = sum(v for k, v in breakdown.items() if k.startswith(spec.name + "."))
    return {"layer": spec.name, "supported": True, "reorder_us": round(kernel_ms(call) * 1e3, 2),
            "routed_us": round(routed * 1e3, 2), "table_entries_per_output": int(table.shape[1])}


def ab_units(net, cfg, unit: int) -> list:
    """k-WTA in units of `unit` channels (Section 5's [64:64] modules) on every
    fp32 layer that reads lists: the one-kernel layer
    (cs_mrs_kwta_units_conv2d, lists out) against the same result from
    separate launches (sums, k-WTA on the unit view, compaction of the masked
    output into lists).  Warm timings (20-launch graphs)."""
    import torch
    from paper_2112_13896_amd import ops

    out = []
    for li, (p, pl) in enumerate(zip(net.packed, net.plans)):
        s = p.spec
        if (net.packed[0].aug.dtype == torch.int16 or not pl.in_lists or s.k is None
                or s.kind != "conv" or s.c_out % unit or pl.pool != 1):
            continue
        ku = -(-s.k * unit // s.c_out)                    # winners per unit, rounded up
        idx, lval, cnt = net.bufs.lists[li - 1]
        b, h, w, c = pl.geo
        bias = p.bias
        y = torch.empty_like(net.bufs.acc[li])
        y4 = y.reshape(b, -1, 1, s.c_out) if y.dim() == 2 else y
        rows = y.numel() // s.c_out
        dense = torch.empty_like(y)
        cap = ops.list_capacity(ku * (s.c_out // unit))
        lists = (torch.empty((rows, cap), dtype=torch.int16, device="cuda"),
                 torch.empty((rows, cap), dtype=torch.float32, device="cuda"),
                 torch.empty((rows,), dtype=torch.int32, device="cuda"))
        clists = (torch.empty((rows, s.c_out), dtype=torch.int16, device="cuda"),
                  torch.empty((rows, s.c_out), dtype=torch.float32, device="cuda"),
                  torch.empty((rows,), dtype=torch.int32, device="cuda"))

        def fused():
            ops.mrs_kwta_units_conv2d(idx, lval, cnt, pl.geo, p.aug, pl.kh, pl.kw, s.n,
                                      pl.stride, pl.pad, bias, 1, k=ku, unit=unit, y=y4,
                                      keep_sums=False, lists=lists)

        def sums():
            ops.mrs_conv2d(idx, lval, cnt, pl.geo, p.aug, pl.kh, pl.kw, s.n, pl.stride, pl.pad,
                           bias, 1, out=y4)

        def kw():
            ops.kwta(y.reshape(-1, unit), ku, out=dense.reshape(-1, unit))

        def comp():
            ops.compact_into(dense.reshape(rows, s.c_out), *clists)
        fused()
        sums(); kw(); comp()
        torch.cuda.synchronize()
        t = {nm: _time_call(f) * 1e3 for nm, f in
             (("fused", fused), ("sums", sums), ("kwta", kw), ("compact", comp))}
        out.append({"layer": s.name, "unit": unit, "k_per_unit": ku,
                    "one_kernel_us": round(t["fused"], 2),
                    "separate_us": {"sums": round(t["sums"], 2), "kwta_units": round(t["kwta"], 2),
                                    "compact": round(t["compact"], 2),
                                    "total": round(t["sums"] + t["kwta"] + t["compact"], 2)}})
    return out


def ab_stem(batch: int = 32) -> dict:
    """A ResNet-50 stem with block Complementary Sparsity (Section 5: a pixel's
    RGB values one block; 7x7, stride 2, pad 3, 64 outputs, n = 4: 75 % of
    the weights zero) on a dense int8 224x224x3 batch: the sparse-dense block
    kernel (cs_conv2d_dense_blocks, one dot product and one routed add per
    tap and set) against the routed path on the compacted input (cs_conv2d).
    Synthetic seeded data; warm timings (20-launch graphs); the two sums must
    be equal."""
    import torch
    from paper_2112_13896_amd import ops
    from workloads import block_complementary_weights

    r = np.random.default_rng(2112_13896 + 50)
    h = w = 224
    c, kh, n, c_out = 3, 7, 4, 64
    mask = block_complementary_weights(r, r, c_out, kh * kh * c, n, c) != 0
    W = np.where(mask, r.integers(1, 128, size=mask.shape) * r.choice([-1, 1], size=mask.shape),
                 0).astype(np.int8)
    aug, kidb, _ = ops.pack_blocks(W, n, c)
    ad, kd = ops.aug_to_device(aug), torch.from_numpy(kidb).cuda()
    x = torch.from_numpy(r.integers(-127, 128, size=(batch, h, w, c)).astype(np.int8)).cuda()
    ho = (h + 6 - kh) // 2 + 1
    y1 = torch.empty((batch, ho, ho, c_out), dtype=torch.int32, device="cuda")
    y2 = torch.empty_like(y1)
    rows = batch * h * w
    ws = torch.empty(ops.workspace_bytes(1, torch.int8, rows, c), dtype=torch.uint8, device="cuda")

    def blocks():
        ops.conv2d_dense_blocks(x, ad, kd, kh, kh, n, 2, 3, None, out=y1)

    def routed():
        ops.conv2d(x, ad, kh, kh, n, 2, 3, None, ws=ws, out=y2)
    blocks()
    routed()
    torch.cuda.synchronize()
    same = bool(torch.equal(y1, y2))
    tb, tr = _time_call(blocks) * 1e3, _time_call(routed) * 1e3
    nbytes = x.numel() + y1.numel() * 4 + aug.nbytes + kidb.nbytes
    return {"layer": "stem 7x7/2, 3 -> 64, n = 4, blocks of 3 (RGB)", "batch": batch,
            "input": [h, w, c], "equal_sums": same, "dense_blocks_us": round(tb, 2),
            "routed_us": round(tr, 2), "dense_blocks_hbm_frac": round(
                nbytes / (tb * 1e-6) / 1e9 / HBM_PEAK_GBS, 4), "algorithmic_bytes": nbytes}


def ab_channels(batch: int = 32) -> dict:
    """Complementary Sparsity overlaid in the channel dimension (Section 3.1)
    on a ResNet-50 stage-1-shaped layer (56x56, 3x3 pad 1, 48 -> 64 channels,
    n = 3: every filter's three-channel groups overlaid, 1/3 of its weights
    non-zero; dense input): the int8 kernel (cs_conv2d_channels) against the
    fp32 reordering kernel the overlay ran on before (cs_conv2d_reorder_kwta,
    every output winning so that both give the sums).  Synthetic seeded data;
    warm timings (20-launch graphs)."""
    import torch
    from paper_2112_13896_amd import ops
    from workloads import channel_complementary_weights

    r = np.random.default_rng(2112_13896 + 60)
    h = w = 56
    c, kh, n, c_out = 48, 3, 3, 64
    Wf = channel_complementary_weights(r, r, c_out, kh, kh, c, n)
    mask = Wf != 0
    W8 = np.where(mask, r.integers(1, 128, size=mask.shape) * r.choice([-1, 1], size=mask.shape),
                  0).astype(np.int8)
    p8, _ = ops.pack_channels(W8, n)
    t8 = torch.from_numpy(ops.channel_table(p8, kh, kh, c, c_out, n, 1)).cuda()
    pf, _ = ops.pack_channels(Wf, n)
    tf = torch.from_numpy(ops.reorder_table_channels(pf, kh, kh, c, c_out, n)).cuda()
    x8 = torch.from_numpy(r.integers(-127, 128, size=(batch, h, w, c)).astype(np.int8)).cuda()
    xf = torch.from_numpy(np.abs(r.normal(size=(batch, h, w, c))).astype(np.float32)).cuda()
    y8 = torch.empty((batch, h, w, c_out), dtype=torch.int32, device="cuda")
    yf = torch.empty((batch, h, w, c_out), dtype=torch.float32, device="cuda")
    of = torch.empty_like(yf)

    def i8():
        ops.conv2d_channels(x8, t8, kh, kh, c_out, n, 1, 1, None, out=y8)

    def f32():
        ops.conv2d_reorder_kwta(xf, tf, kh, kh, 1, None, k=c_out, y=yf, keep_sums=False, out=of)
    i8()
    f32()
    torch.cuda.synchronize()
    t8us, tfus = _time_call(i8) * 1e3, _time_call(f32) * 1e3
    nbytes = x8.numel() + y8.numel() * 4 + t8.numel() * 4
    return {"layer": "3x3 pad 1, 48 -> 64, n = 3 channel overlay, 56x56", "batch": batch,
            "int8_channels_us": round(t8us, 2), "fp32_reorder_us": round(tfus, 2),
            "int8_hbm_frac": round(nbytes / (t8us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
            "slots_per_filter": int(kh * kh * c // n)}


MALL_MIB = 256.0                    # MI355X Infinity Cache (last-level cache)
SET_MEM_CAP = 24 << 30              # most device memory the rotating buffer sets may take


def scrub(buf) -> None:
    """Read a buffer twice the size of the last-level cache, so that no
    earlier launch's data is still cached (outside every timed region).  A
    read leaves clean lines behind: a write would leave the caches full of
    dirty lines whose write-back the next kernel would pay for."""
    buf.sum()


def measure(cfg, steps: int, warmup: int, rotate_mib: float, eager_only: int = 0,
            ab: bool = False, ab_unit: int = 0) -> dict:
    """One workload: the whole chain, K timed passes, per-kernel durations.

    Buffer sets (input + every intermediate) rotate; their number is chosen
    from the bytes one pass actually touches (the sum of its launches'
    algorithmic bytes) so that a set is reused only after more than
    `rotate_mib` of other data, and a 512 MiB read (the scrub) precedes every
    timed region, so no pass finds its data in the 256 MiB Infinity Cache or
    in L2."""
    import torch

    from paper_2112_13896_amd.network import Network
    from workloads import generate

    log(f"bench: workload {cfg.name}, batch {cfg.batch}")
    inp = generate(cfg)
    net = Network(cfg.layers, inp["W"], inp["b"], cfg.in_shape, cfg.batch, keep_sums=False)
    x0 = torch.from_numpy(inp["x"]).cuda()
    net.forward(x0, net.bufs)
    torch.cuda.synchronize()
    costs = layer_costs(net, net.bufs, cfg)
    names0 = [nm for li in range(len(net.packed)) for nm, _ in net.launches(
        li, x0 if li == 0 else None, net.bufs)]
    touched = sum(costs[nm]["bytes"] for nm in names0 if nm in costs)
    alloc = net.bufs.nbytes() + inp["x"].nbytes
    nsets = max(8, math.ceil(rotate_mib * 2 ** 20 / max(touched, 1)))
    nsets = max(2, min(nsets, 512, SET_MEM_CAP // max(alloc, 1)))
    sets = [net.bufs] + [net.make_buffers() for _ in range(nsets - 1)]
    # a different input per set: the batch rolled by j samples (same work)
    xs = [x0] + [torch.from_numpy(np.roll(inp["x"], j, axis=0)).cuda() for j in range(1, nsets)]
    log(f"bench: {nsets} rotating buffer sets, {touched / 2 ** 20:.2f} MiB touched per pass "
        f"({alloc / 2 ** 20:.1f} MiB allocated per set)")
    for j in range(nsets):                           # every set holds a whole pass's data
        net.forward(xs[j], sets[j])
    torch.cuda.synchronize()
    scrub_buf = torch.ones(int(2 * MALL_MIB * 2 ** 20) // 4, dtype=torch.int32, device="cuda")
    if eager_only:
        # profiler mode: eager passes only (every launch a plain dispatch)
        t0 = time.perf_counter()
        for i in range(eager_only):
            net.forward(xs[i % nsets], sets[i % nsets])
        torch.cuda.synchronize()
        return {"workload": cfg.name, "eager_passes": eager_only,
                "ms_per_pass_eager": round((time.perf_counter() - t0) * 1e3 / eager_only, 4)}
    for i in range(warmup):
        net.forward(xs[i % nsets], sets[i % nsets])
    torch.cuda.synchronize()
    # one HIP graph per buffer set: one pass per replay
    graphs = [net.capture(xs[j], sets[j]) for j in range(nsets)]
    # the timed steps: one graph of all the passes, pass i on set i % nsets,
    # in the fastest of three schedules
    gsteps = steps if steps <= 256 else nsets
    g_mode = {m: capture_passes(net, xs, sets, gsteps, m)
              for m in ("sequential", "overlapped", "alternate")}
    sched = {}
    for name, g in g_mode.items():
        g.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(3):
            g.replay()
        torch.cuda.synchronize()
        sched[name] = time.perf_counter() - t0
    schedule = min(sched, key=sched.get)
    g_all = g_mode[schedule]
    log(f"bench: schedule {schedule} ("
        + ", ".join(f"{k} {v * 1e6 / (3 * gsteps):.1f} us" for k, v in sched.items())
        + " per step, cache-warm)")

    scrub(scrub_buf)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps // gsteps):
        g_all.replay()
    for i in range(steps % gsteps):
        graphs[i % nsets].replay()
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / steps
    # the same steps with one graph launch each
    scrub(scrub_buf)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        graphs[i % nsets].replay()
    torch.cuda.synchronize()
    ms_step_1 = (time.perf_counter() - t0) * 1e3 / steps

    # per-kernel durations, cache-cold: a graph of one launch of the kernel per
    # buffer set (min(nsets, 32) sets), timed with HIP events on the replaying
    # stream, each replay after a scrub
    per_set = [dict(nc for li in range(len(net.packed)) for nc in net.launches(
        li, xs[j] if li == 0 else None, sets[j])) for j in range(nsets)]
    nk = min(nsets, 32)

    def kernel_ms(name, reps=4):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for j in range(nk):
                per_set[j][name]()
        g.replay()
        tot = 0.0
        for _ in range(reps):
            scrub(scrub_buf)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            g.replay()
            e1.record()
            torch.cuda.synchronize()
            tot += e0.elapsed_time(e1)
        return tot / (reps * nk)

    breakdown = {name: kernel_ms(name) for name in names0}
    dominant = max(breakdown, key=breakdown.get)
    log("bench: per-kernel ms (cold) " + ", ".join(f"{k}={v:.4f}" for k, v in breakdown.items()))
    dom_ms = kernel_ms(dominant, reps=max(4, steps // 4))
    roof = roofline_for(dominant, costs[dominant], dom_ms)
    roof["traffic"] = load_traffic(dominant, cfg.name)
    kernels = {}
    for k, ms in breakdown.items():
        c = costs.get(k, {})
        e = {"us": round(ms * 1e3, 2)}
        if "bytes" in c:
            e["bytes"] = c["bytes"]
            e["hbm_frac"] = round(c["bytes"] / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
        if "bytes_dense_out" in c:
            e["bytes_dense_out"] = c["bytes_dense_out"]
            e["hbm_frac_dense_out"] = round(c["bytes_dense_out"] / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)
        if "products" in c:
            e["Gproducts/s"] = round(c["products"] / (ms * 1e-3) / 1e9, 1)
        kernels[k] = e
    rec = {"workload": cfg.name, "batch": cfg.batch, "steps": steps,
           "ms_per_step": round(ms_step, 4), "samples_per_s": round(cfg.batch / (ms_step * 1e-3), 1),
           "dense_equiv_gmac_per_s": round(dense_macs(cfg) / (ms_step * 1e-3) / 1e9, 1),
           "ms_per_step_one_launch_per_step": round(ms_step_1, 4), "schedule": schedule,
           "buffer_sets": nsets, "touched_bytes_per_pass": int(touched),
           "roofline": roof, "kernels": kernels}
    if ab:
        rec["ab_reorder"] = ab_reorder(cfg, inp, xs[0], lambda call: _time_call(call),
                                       breakdown)
    if ab_unit:
        rec["ab_units"] = ab_units(net, cfg, ab_unit)
    rec["_inp"] = inp
    return rec


def _time_call(call, reps=4) -> float:
    import torch
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(KREP):
            call()
    g.replay()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / (reps * KREP)


CHAIN_PHASES = ("conv1 staging", "conv1 products (MFMA)", "conv1 k-WTA", "conv1 lists out",
                "conv2 staging", "conv2 products (routed adds)", "conv2 pool + k-WTA + lists",
                "linear1 staging", "linear1 products", "linear1 sums", "linear1 threshold",
                "linear1 winners + lists", "output layer")


def phase_report(cids) -> dict:
    """Per-phase times from the stamping build (libcs_stamps.so): for the
    one-kernel keyword-spotting chain, the mean time of each phase per
    workgroup, with one pass at a time on one stream and with passes
    alternating on two streams (two images per CU, as the benchmark's graph
    runs them); for the table-block layers, the mean time per tile of its
    set-up + products and of its epilogue.  Eager launches, warm caches."""
    import torch
    from paper_2112_13896_amd import _lib
    from paper_2112_13896_amd.network import Network
    from workloads import CONFIGS, generate

    out = {}
    with _lib.stamping_library():
        for cid in cids:
            cfg = CONFIGS[cid]
            inp = generate(cfg)
            nets = [Network(cfg.layers, inp["W"], inp["b"], cfg.in_shape, cfg.batch,
                            keep_sums=False) for _ in range(2)]
            x = torch.from_numpy(inp["x"]).cuda()
            for n in nets:
                n.forward(x)
            torch.cuda.synchronize()
            rec = {}
            for li in range(len(cfg.layers)):
                for name, call in nets[0].launches(li, x if li == 0 else None):
                    if "mrs" not in name:
                        continue
                    _lib.phase_stamps(reset=True)
                    for _ in range(20):
                        call()
                    acc, khz = _lib.phase_stamps(reset=True)
                    us = lambda a, b, c: round((acc[b] - acc[a]) / max(acc[c], 1) / khz * 1e3, 2)
                    if acc[15]:
                        rec[name] = {"workgroups": acc[15] // 20, "one stream": {
                            "workgroup us": us(0, 13, 15),
                            **{CHAIN_PHASES[i]: us(i, i + 1, 15) for i in range(13)}}}
                        # two passes at a time, on two streams (separate buffers)
                        side = torch.cuda.Stream()
                        calls = [c for nm2, c in nets[1].launches(li, x if li == 0 else None)
                                 if nm2 == name]
                        torch.cuda.synchronize()
                        for i in range(20):
                            if i % 2:
                                with torch.cuda.stream(side):
                                    calls[0]()
                            else:
                                call()
                        acc, khz = _lib.phase_stamps(reset=True)
                        rec[name]["two streams"] = {
                            "workgroup us": us(0, 13, 15),
                            **{CHAIN_PHASES[i]: us(i, i + 1, 15) for i in range(13)}}
                    elif acc[31]:
                        rec[name] = {"tiles": acc[31] // 20,
                                     "tile set-up + products us": us(16, 17, 31),
                                     "of it: products (table blocks in LDS) us":
                                         round(acc[21] / max(acc[31], 1) / khz * 1e3, 2),
                                     "epilogue us": us(17, 18, 31)}
                        if acc[19] and acc[20]:
                            # the selection on the lanes' own columns, in parts
                            rec[name].update({"epilogue: threshold search us": us(17, 19, 31),
                                              "epilogue: threshold, ties, masks us": us(19, 20, 31),
                                              "epilogue: output us": us(20, 18, 31)})
            out[cfg.name] = rec
            torch.cuda.synchronize()
    return out


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=2, help="workload id (default 2: keyword-spotting CNN)")
    ap.add_argument("--also", default="1,3,4,5",
                    help="other workloads measured after the headline one and reported in "
                         "\"workloads\" (comma-separated ids; empty for none)")
    ap.add_argument("--rotate-mib", type=float, default=512.0)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--eager-passes", type=int, default=0, metavar="N",
                    help="profiler mode: only N eager passes of the workload (no graphs, no timing)")
    ap.add_argument("--ab-reorder", action="store_true",
                    help="also time the first layer by reordering the activations instead of "
                         "routing the products (fp32 dense-input 64-channel layers)")
    ap.add_argument("--ab-units", type=int, default=0, metavar="UNIT",
                    help="also time k-WTA in units of UNIT channels on the fp32 layers that "
                         "read lists: one kernel against sums + unit k-WTA + compaction")
    ap.add_argument("--ab-stem", action="store_true",
                    help="also time a block-CS ResNet-50 stem (dense int8 224x224x3, batch 32): "
                         "the sparse-dense block kernel against the routed path")
    ap.add_argument("--ab-channels", action="store_true",
                    help="also time a channel-overlaid layer (56x56, 3x3, 48 -> 64, n = 3, batch "
                         "32): the int8 channel kernel against the fp32 reordering kernel")
    ap.add_argument("--phase-stamps", default="", metavar="IDS",
                    help="only report per-phase times of the given workloads (comma-separated "
                         "ids) from the stamping build libcs_stamps.so")
    ap.add_argument("--calibrate-copy", type=float, default=0.0, metavar="MIB",
                    help="only copy a MIB-sized device buffer --steps times (reference kernel "
                         "for scaling the HBM byte counters, and the copy ceiling)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for {args.gpus} GPUs, WORLD_SIZE={world}); "
              "the sparse-sparse path shards over samples with no exchange, so N GPUs run N "
              "independent copies of this measurement.", file=sys.stderr)
        return 2

    import torch

    from workloads import CONFIGS

    if not torch.cuda.is_available():
        log("bench.py needs a GPU")
        return 1
    if args.calibrate_copy > 0:
        nbytes = int(args.calibrate_copy * 2 ** 20) // 16 * 16
        src = torch.ones(nbytes // 4, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        sec = e0.elapsed_time(e1) * 1e-3
        print(json.dumps({"copy_bytes_read": nbytes, "copy_bytes_written": nbytes,
                          "launches": args.steps,
                          "GB/s": round(2 * nbytes * args.steps / sec / 1e9, 1)}), flush=True)
        return 0
    if args.phase_stamps:
        ids = [int(c) for c in args.phase_stamps.split(",") if c.strip()]
        print(json.dumps({"phase_stamps": phase_report(ids)}), flush=True)
        return 0
    cfg = CONFIGS[args.config]
    if args.eager_passes:
        print(json.dumps(measure(cfg, args.steps, args.warmup, args.rotate_mib,
                                 eager_only=args.eager_passes)), flush=True)
        return 0
    head = measure(cfg, args.steps, args.warmup, args.rotate_mib, ab=args.ab_reorder,
                   ab_unit=args.ab_units)
    inp = head.pop("_inp")
    res = {
        "metric": METRIC, "value": head["samples_per_s"], "unit": "samples/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": head["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "i8*i8->i32" if cfg.dtype == "i8" else "f32",
        "data": "synthetic (seeded; stands in for the paper's dataset)",
        "config": {"workload": cfg.name, "batch": cfg.batch, "layers": [s.name for s in cfg.layers]},
        "dense_equiv_gmac_per_s": head["dense_equiv_gmac_per_s"],
        "ms_per_step_one_launch_per_step": head["ms_per_step_one_launch_per_step"],
        "schedule": head["schedule"],
        "buffer_sets": head["buffer_sets"],
        "touched_bytes_per_pass": head["touched_bytes_per_pass"],
        "roofline": head["roofline"],
        "kernels": head["kernels"],
    }
    for key in ("ab_reorder", "ab_units"):
        if key in head:
            res[key] = head[key]
    if args.ab_stem:
        res["ab_stem"] = ab_stem()
    if args.ab_channels:
        res["ab_channels"] = ab_channels()
    others = [int(c) for c in args.also.split(",") if c.strip() and int(c) != args.config]
    if others:
        res["workloads"] = {}
        for cid in others:
            sub = measure(CONFIGS[cid], min(args.steps, 20), min(args.warmup, 5), args.rotate_mib)
            sub.pop("_inp")
            res["workloads"][sub.pop("workload")] = sub
            torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        log("bench: timing the CPU oracle")
        res["cpu_baseline"] = cpu_baseline(cfg, inp, args.cpu_seconds)
    print(json.dumps(res), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
