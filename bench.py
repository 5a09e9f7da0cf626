#!/usr/bin/env python3
"""Benchmark of the Sherry 1.25-bit ternary hot path on one MI355X.

Workload (the metric's headline configuration): one decode step (M = 1) of the
linear layers of LLaMA-3.2-1B -- 16 layers x {q 2048x2048, k/v 512x2048,
o 2048x2048, gate/up 8192x2048, down 2048x8192} -- as 3:4 ternary weights
packed at 1.25 bits, per-tensor scales U(0.01, 0.05), a fresh fp32 N(0,1)
activation vector per projection.  A step is the whole hot path on device in
one launch: per-token int8 quantization of each of the 112 activation vectors
fused with its product, on lane-interleaved weights (sherry_pack_il,
sherry_gemv_f32_il_batched).  Weights and activations are rotated over 16
copies (2.4 GB, about 10x the 256 MB Infinity Cache, so cache hits cannot
inflate the figures).

Prints one JSON line.  `value` = algorithmic bytes of a step / step time
(GB/s), timed with HIP events around back-to-back steps on the stream the
kernel runs on, after a heat-up; `roofline` is that same fused kernel;
`fused_tiled` times the same step on the tiled layout; `unfused` times it as
separate quantize and int8 product launches;
`cpu_baseline` is the CPU oracle on the host cores over full steps;
`parity` checks the timed step against the oracle.  Unless --no-extra, the
M = 2048 prefill GEMM on the LLaMA-3.2-3B and -1B shapes is timed too
(dense-equivalent TOPS), with context lines: streaming reads of 2 GiB and of
the step's own bytes per launch (`hbm_read_same_bytes`), the 3B and 8B-scale
decode steps, grouped small-M steps, the 1.25 / 1.67 / 2-bit layouts of one
8B-scale step, GPU ternarize + pack and a single q-projection GEMV.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402

HBM_PEAK_GBS = 8000.0
KERNEL_NAMES = {1: "gemv", 2: "mfma", 3: "skinny"}  # SHERRY_KERNEL_* values
INT8_PEAK_TOPS = 5000.0
COPIES = 16  # rotated copies of the weights: 16 x 152 MB = 2.4 GB, ~10x the Infinity Cache


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def kernel_source_hash(files) -> str:
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2601_07892_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


# ---------------------------------------------------------------------------
# decode step (M = 1)
# ---------------------------------------------------------------------------

class DecodeStep:
    """Device buffers of COPIES rotated copies of one decode step."""

    def __init__(self, sh, torch, dev, spec, seed, copies=COPIES, keep_host=True):
        self.sh, self.torch, self.dev = sh, torch, dev
        self.lins = synth.model_linears(spec)
        self.count = len(self.lins)
        t0 = time.time()
        self.t = []        # host ternary matrices (for the CPU baseline)
        self.packed = []   # device packed weights, [copy][i]
        self.scales = []
        host_packed = []
        host_il = []       # the same matrices, lane-interleaved (sherry_pack_il)
        for i, (layer, lin) in enumerate(self.lins):
            t = synth.ternary_34(lin.n, lin.k, seed, "w", layer, lin.name)
            if keep_host:
                self.t.append(t)
            host_packed.append(sh.sherry_pack(t))
            host_il.append(sh.sherry_pack_il(t))
            self.scales.append(synth.weight_scale(seed, "s", layer, lin.name))
        log("generated+packed %d weights in %.1fs" % (sum(l.n * l.k for _, l in self.lins),
                                                       time.time() - t0))
        self.ks = sorted({lin.k for _, lin in self.lins})
        self.x_host = {kk: synth.activations(sum(1 for _, l in self.lins if l.k == kk), kk, seed,
                                             "x", kk) for kk in self.ks}
        self.channel_scales = [
            torch.from_numpy((np.random.default_rng([seed, i]).random(lin.n) * 0.04 + 0.01)
                             .astype(np.float32)).to(dev) for i, (_, lin) in enumerate(self.lins)]
        self.copies = []
        for c in range(copies):
            w = [torch.from_numpy(p).to(dev) for p in host_packed]
            xs = {kk: torch.from_numpy(self.x_host[kk]).to(dev) for kk in self.ks}
            qs = {kk: torch.empty(xs[kk].shape, dtype=torch.int8, device=dev) for kk in self.ks}
            sxs = {kk: torch.empty(xs[kk].shape[0], dtype=torch.float32, device=dev)
                   for kk in self.ks}
            ys = [torch.empty(lin.n, dtype=torch.float32, device=dev) for _, lin in self.lins]
            descs = (sh.sherry_gemv_desc * self.count)()
            row = {kk: 0 for kk in self.ks}
            for i, (_, lin) in enumerate(self.lins):
                r = row[lin.k]
                row[lin.k] += 1
                d = descs[i]
                d.w = w[i].data_ptr()
                d.x = qs[lin.k][r].data_ptr()
                d.x_scale = sxs[lin.k][r:r + 1].data_ptr()
                d.y = ys[i].data_ptr()
                d.acc = None
                d.n, d.k, d.w_scale = lin.n, lin.k, self.scales[i]
            total = sh.sherry_gemv_batched_prepare(descs)
            ddev = torch.from_numpy(sh.descs_to_bytes(descs)).to(dev)
            # fused descriptors: fp32 activations in, scales written back
            fdescs = (sh.sherry_gemv_f32_desc * self.count)()
            for i in range(self.count):
                f, d = fdescs[i], descs[i]
                lin = self.lins[i][1]
                f.w, f.y, f.acc, f.x_scale = d.w, d.y, None, d.x_scale
                f.x = xs[lin.k].data_ptr() + (d.x - qs[lin.k].data_ptr()) * 4
                f.n, f.k, f.w_scale = d.n, d.k, d.w_scale
            ftotal = sh.sherry_gemv_f32_batched_prepare(fdescs)
            fdev = torch.from_numpy(sh.descs_to_bytes(fdescs)).to(dev)
            # the same fused step on lane-interleaved weights (same buffers
            # otherwise): the timed headline step
            w_il = [torch.from_numpy(p).to(dev) for p in host_il]
            for i in range(self.count):
                fdescs[i].w = w_il[i].data_ptr()
            ftotal_il = sh.sherry_gemv_f32_il_batched_prepare(fdescs)
            fdev_il = torch.from_numpy(sh.descs_to_bytes(fdescs)).to(dev)
            # the same step with one weight scale per output channel (Eq. 5)
            for i in range(self.count):
                fdescs[i].w_scales = self.channel_scales[i].data_ptr()
            fdev_ch_il = torch.from_numpy(sh.descs_to_bytes(fdescs)).to(dev)
            for i in range(self.count):
                fdescs[i].w = w[i].data_ptr()
            fdev_ch = torch.from_numpy(sh.descs_to_bytes(fdescs)).to(dev)
            # every activation matrix of the step in one quantize launch
            qdescs = (sh.sherry_quant_desc * len(self.ks))()
            for j, kk in enumerate(self.ks):
                qd = qdescs[j]
                qd.x, qd.q, qd.x_scale = (xs[kk].data_ptr(), qs[kk].data_ptr(),
                                          sxs[kk].data_ptr())
                qd.m, qd.k = xs[kk].shape[0], kk
            qrows, qmaxk = sh.sherry_quantize_act_batched_prepare(qdescs)
            qdev = torch.from_numpy(sh.descs_to_bytes(qdescs)).to(dev)
            cp = dict(w=w, w_il=w_il, xs=xs, qs=qs, sxs=sxs, ys=ys, descs=ddev, total=total,
                      fdescs=fdev, ftotal=ftotal, fdescs_ch=fdev_ch, fdescs_il=fdev_il,
                      ftotal_il=ftotal_il, fdescs_ch_il=fdev_ch_il, qdescs=qdev,
                      qrows=qrows, qmaxk=qmaxk)
            if c == 0:
                # the same fused step with int32 outputs as well (parity check)
                accs = [torch.empty(lin.n, dtype=torch.int32, device=dev)
                        for _, lin in self.lins]
                for i in range(self.count):
                    fdescs[i].w_scales = None
                    fdescs[i].acc = accs[i].data_ptr()
                    fdescs[i].w = w_il[i].data_ptr()
                cp["accs"] = accs
                cp["fdescs_acc_il"] = torch.from_numpy(sh.descs_to_bytes(fdescs)).to(dev)
            self.copies.append(cp)
        torch.cuda.synchronize()
        self.total_blocks = self.copies[0]["total"]
        self.weight_bytes = sum(sh.sherry_packed_bytes(l.n, l.k) for _, l in self.lins)
        # algorithmic bytes of one grouped product launch: packed weights,
        # int8 x, its fp32 scale, fp32 y
        self.gemv_bytes = sum(sh.sherry_packed_bytes(l.n, l.k) + l.k + 4 + 4 * l.n
                              for _, l in self.lins)
        # quantization: fp32 x read, int8 q written, fp32 scale written
        self.quant_bytes = sum(5 * l.k + 4 for _, l in self.lins)
        # fused step: packed weights, fp32 x, its scale written, fp32 y
        self.fused_bytes = sum(sh.sherry_packed_bytes(l.n, l.k) + 4 * l.k + 4 + 4 * l.n
                               for _, l in self.lins)
        self.ops = sum(2 * l.n * l.k for _, l in self.lins)
        log("working set: %.1f MB of packed weights per copy x %d copies" %
            (self.weight_bytes / 1e6, copies))

    def quantize(self, c):
        cp = self.copies[c]
        for kk in self.ks:
            self.sh.sherry_quantize_act(cp["xs"][kk], cp["qs"][kk], cp["sxs"][kk])

    def quantize_grouped(self, c):
        cp = self.copies[c]
        self.sh.sherry_quantize_act_batched(cp["qdescs"], len(self.ks), cp["qrows"], cp["qmaxk"])

    def gemv(self, c):
        cp = self.copies[c]
        self.sh.sherry_gemv_batched(cp["descs"], self.count, cp["total"])

    def fused(self, c):
        # the headline step: fused quantization + products, lane-interleaved
        cp = self.copies[c]
        self.sh.sherry_gemv_f32_il_batched(cp["fdescs_il"], self.count, cp["ftotal_il"])

    def fused_channel(self, c):
        cp = self.copies[c]
        self.sh.sherry_gemv_f32_il_batched(cp["fdescs_ch_il"], self.count, cp["ftotal_il"])

    def fused_tiled(self, c):
        # the same step on the tiled layout
        cp = self.copies[c]
        self.sh.sherry_gemv_f32_batched(cp["fdescs"], self.count, cp["ftotal"])


def _events(torch):
    return torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)


def settle(run, torch, seconds=0.02):
    """Untimed back-to-back launches of the timed loop's own work for about
    `seconds`: the first few milliseconds over a cold working set run slower
    than the steady state that the timed loop reports."""
    torch.cuda.synchronize()
    t0, i = time.perf_counter(), 0
    while time.perf_counter() - t0 < seconds:
        for _ in range(32):
            run(i)
            i += 1
        torch.cuda.synchronize()


def bench_fused(step: DecodeStep, torch, steps, warmup, channel=False, tiled=False):
    """ms per decode step (one fused launch), back to back after a heat-up;
    channel=True runs the step with per-channel weight scales, tiled=True on
    the tiled layout instead of the lane-interleaved one."""
    ncp = len(step.copies)
    run = step.fused_tiled if tiled else (step.fused_channel if channel else step.fused)
    heat(step.sh, torch, step.dev)
    settle(lambda i: run(i % ncp), torch)
    for i in range(warmup):
        run(i % ncp)
    start, stop = _events(torch)
    torch.cuda.synchronize()
    start.record()
    for i in range(steps):
        run(i % ncp)
    stop.record()
    torch.cuda.synchronize()
    return start.elapsed_time(stop) / steps


def bench_ternarize(sh, torch, dev, seed, shapes=(("llama-3.2-3b gate", 8192, 3072),
                                                  ("stress-8b down", 4096, 14336)), reps=10):
    """GB/s of the GPU Sparse-AbsMean ternarize + pack (fp32 W read, packed
    layout and per-channel alpha written), over rotated weight copies."""
    rows = []
    for name, n, k in shapes:
        w0 = torch.from_numpy(synth.dense_weights(n, k, seed, "tp", name)).to(dev)
        ncp = max(2, -(-600_000_000 // (4 * n * k)))  # > 600 MB, past the Infinity Cache
        ws = [w0.clone() for _ in range(ncp)]
        packed = torch.empty(sh.sherry_packed_bytes(n, k), dtype=torch.uint8, device=dev)
        alpha = torch.empty(n, dtype=torch.float32, device=dev)
        for i in range(2):
            sh.sherry_ternarize_pack(ws[i % ncp], n, k, packed, alpha)
        start, stop = _events(torch)
        torch.cuda.synchronize()
        start.record()
        for i in range(reps):
            sh.sherry_ternarize_pack(ws[i % ncp], n, k, packed, alpha)
        stop.record()
        torch.cuda.synchronize()
        us = start.elapsed_time(stop) / reps * 1e3
        nbytes = 4 * n * k + sh.sherry_packed_bytes(n, k) + 4 * n
        rows.append({"shape": name, "n": n, "k": k, "us": round(us, 2), "bytes": nbytes,
                     "gbs": round(nbytes / us / 1e3, 1),
                     "frac": round(nbytes / us / 1e3 / HBM_PEAK_GBS, 4)})
        del ws, w0, packed, alpha
        torch.cuda.empty_cache()
    return rows


def bench_unfused(step: DecodeStep, torch, steps, warmup):
    """ms per step as separate launches (2 quantize + grouped int8 product)."""
    ncp = len(step.copies)

    def unfused(i):
        step.quantize(i % ncp)
        step.gemv(i % ncp)
    settle(unfused, torch)
    for i in range(warmup):
        step.quantize(i % ncp)
        step.gemv(i % ncp)
    start, stop = _events(torch)
    torch.cuda.synchronize()
    start.record()
    for i in range(steps):
        step.quantize(i % ncp)
        step.gemv(i % ncp)
    stop.record()
    torch.cuda.synchronize()
    return start.elapsed_time(stop) / steps


def bench_two_launch(step: DecodeStep, torch, steps, warmup):
    """ms per step as two launches: every activation row quantized in one
    launch (sherry_quantize_act_batched), then the grouped int8 product."""
    ncp = len(step.copies)

    def run(i):
        step.quantize_grouped(i % ncp)
        step.gemv(i % ncp)
    settle(run, torch)
    for i in range(warmup):
        run(i)
    start, stop = _events(torch)
    torch.cuda.synchronize()
    start.record()
    for i in range(steps):
        run(i)
    stop.record()
    torch.cuda.synchronize()
    return start.elapsed_time(stop) / steps


def heat(sh, torch, dev, seconds=0.03):
    """Brings the GPU to its steady loaded state before a timed loop (the
    first few milliseconds of sustained HBM load run slower): repeated
    streaming reads of 1 GiB, a different kernel from the ones timed."""
    nbytes = 1 << 30
    src = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    sink = torch.empty(sh.sherry_stream_read_groups(nbytes), dtype=torch.int32, device=dev)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(20):
            sh.sherry_stream_read(src, nbytes, sink)
        torch.cuda.synchronize()
    del src, sink


def bench_product_only(step: DecodeStep, torch, launches):
    """Average duration of the grouped product kernel alone: back-to-back
    launches over the rotated copies, one event pair around the whole run, so
    that per-launch event overhead does not enter the figure."""
    ncp = len(step.copies)
    settle(lambda i: step.gemv(i % ncp), torch)
    start, stop = _events(torch)
    torch.cuda.synchronize()
    start.record()
    for i in range(launches):
        step.gemv(i % ncp)
    stop.record()
    torch.cuda.synchronize()
    return start.elapsed_time(stop) / launches


def bench_stream_ceiling(sh, torch, dev, nbytes=2 << 30, reps=20):
    """Practical HBM read ceiling: a streaming read of 2 GiB with the loads the
    products use for their weights (128-bit buffer loads, non-temporal)."""
    src = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    sink = torch.empty(sh.sherry_stream_read_groups(nbytes), dtype=torch.int32, device=dev)
    for _ in range(3):
        sh.sherry_stream_read(src, nbytes, sink)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record()
    for _ in range(reps):
        sh.sherry_stream_read(src, nbytes, sink)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    del src
    return nbytes / (ms * 1e-3) / 1e9


def bench_stream_same_bytes(sh, torch, dev, nbytes, copies=16, launches=400):
    """The same streaming read over as many bytes per launch as the decode
    step moves, rotated over copies like its weights and launched back to
    back: the read ceiling at this transfer size, launch and ramp included."""
    stride = (nbytes + 255) // 256 * 256
    src = torch.empty(stride * copies, dtype=torch.uint8, device=dev)
    sink = torch.empty(sh.sherry_stream_read_groups(nbytes), dtype=torch.int32, device=dev)
    run = lambda i: sh.sherry_stream_read(src[(i % copies) * stride:], nbytes, sink)
    settle(run, torch)
    a, b = _events(torch)
    torch.cuda.synchronize()
    a.record()
    for i in range(launches):
        run(i)
    b.record()
    torch.cuda.synchronize()
    us = a.elapsed_time(b) / launches * 1e3
    del src, sink
    return {"bytes": nbytes, "copies": copies, "us": round(us, 2),
            "gbs": round(nbytes / (us * 1e-6) / 1e9, 1)}


# ---------------------------------------------------------------------------
# prefill GEMM (M = 2048)
# ---------------------------------------------------------------------------

def bench_prefill(sh, torch, dev, spec, m, seed, reps=10):
    blk = synth.llama_block(spec["hidden"], spec["kv"], spec["inter"])
    rows = []
    tot_ops, tot_ms, tot_ref = 0.0, 0.0, 0.0
    for lin in blk:
        t = synth.ternary_34(lin.n, lin.k, seed, "pw", lin.name, lin.k)
        w = torch.from_numpy(sh.sherry_pack(t)).to(dev)
        x = torch.from_numpy(synth.activations(m, lin.k, seed, "px", lin.name,
                                               outlier_frac=0.01)).to(dev)
        q = torch.empty((m, lin.k), dtype=torch.int8, device=dev)
        sx = torch.empty(m, dtype=torch.float32, device=dev)
        y = torch.empty((m, lin.n), dtype=torch.float32, device=dev)
        sh.sherry_quantize_act(x, q, sx)
        sw = synth.weight_scale(seed, "ps", lin.name)
        for _ in range(2):
            sh.sherry_gemm(w, q, sx, sw, y, None, m, lin.n, lin.k)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        for _ in range(reps):
            sh.sherry_gemm(w, q, sx, sw, y, None, m, lin.n, lin.k)
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / reps
        ops = 2.0 * m * lin.n * lin.k
        tot_ops += ops
        tot_ms += ms
        # context: the vendor's dense int8 GEMM (torch._int_mm, hipBLASLt) on
        # the same shape with unpacked int8 weights (no decode, 1 byte per
        # weight), the practical ceiling of a plain int8 MFMA GEMM here
        wd = torch.from_numpy(t).to(dev).t()  # [k][n] view of the [n][k] matrix
        for _ in range(2):
            torch._int_mm(q, wd)
        a.record()
        for _ in range(reps):
            torch._int_mm(q, wd)
        b.record()
        torch.cuda.synchronize()
        ms_ref = a.elapsed_time(b) / reps
        tot_ref += ms_ref
        rows.append({"proj": lin.name, "n": lin.n, "k": lin.k, "us": round(ms * 1e3, 2),
                     "tops": round(ops / (ms * 1e-3) / 1e12, 1),
                     "kernel": KERNEL_NAMES[sh.sherry_gemm_kernel_for(m, lin.n, lin.k)],
                     "dense_int8_ref_us": round(ms_ref * 1e3, 2)})
        del w, x, q, y, wd
    return {"m": m, "per_layer_us": round(tot_ms * 1e3, 2),
            "tops": round(tot_ops / (tot_ms * 1e-3) / 1e12, 1),
            "mfma_frac": round(tot_ops / (tot_ms * 1e-3) / 1e12 / INT8_PEAK_TOPS, 4),
            "dense_int8_ref": {"per_layer_us": round(tot_ref * 1e3, 2),
                               "tops": round(tot_ops / (tot_ref * 1e-3) / 1e12, 1),
                               "what": "torch._int_mm (hipBLASLt) on unpacked int8 weights, "
                                       "same shapes: the plain int8 MFMA GEMM, no decode"},
            "shapes": rows}


def bench_prefill_grouped(sh, torch, dev, spec, m, seed, reps=10):
    """One layer at M tokens in the four launches its data dependences allow:
    q, k and v grouped in one launch (they read the same activations), o
    alone, gate and up grouped, down alone (lone launches: automatic kernel
    choice).  Dense-equivalent 2MNK ops over the layer's time."""
    blk = {lin.name: lin for lin in synth.llama_block(spec["hidden"], spec["kv"], spec["inter"])}
    bufs = {}
    for name, lin in blk.items():
        t = synth.ternary_34(lin.n, lin.k, seed, "pw", lin.name, lin.k)
        bufs[name] = (torch.from_numpy(sh.sherry_pack(t)).to(dev),
                      torch.empty((m, lin.n), dtype=torch.float32, device=dev))
    acts = {}
    for src in ("qkv", "o", "gateup", "down"):
        k = blk["down"].k if src == "down" else blk["q"].k
        x = torch.from_numpy(synth.activations(m, k, seed, "pgx", src, outlier_frac=0.01)).to(dev)
        q = torch.empty((m, k), dtype=torch.int8, device=dev)
        sx = torch.empty(m, dtype=torch.float32, device=dev)
        sh.sherry_quantize_act(x, q, sx)
        acts[src] = (q, sx)

    def group(names, src):
        descs = (sh.sherry_gemm_desc * len(names))()
        q, sx = acts[src]
        for i, name in enumerate(names):
            lin, (w, y) = blk[name], bufs[name]
            d = descs[i]
            d.w, d.x, d.x_scale, d.y, d.acc = (w.data_ptr(), q.data_ptr(), sx.data_ptr(),
                                               y.data_ptr(), None)
            d.n, d.k, d.m, d.w_scale = lin.n, lin.k, m, 0.02
        total, max_m = sh.sherry_gemm_batched_prepare(descs)
        return torch.from_numpy(sh.descs_to_bytes(descs)).to(dev), len(names), total, max_m

    g_qkv, g_gu = group(["q", "k", "v"], "qkv"), group(["gate", "up"], "gateup")

    def layer():
        sh.sherry_gemm_batched(*g_qkv)
        q, sx = acts["o"]
        sh.sherry_gemm(bufs["o"][0], q, sx, 0.02, bufs["o"][1], None, m, blk["o"].n, blk["o"].k)
        sh.sherry_gemm_batched(*g_gu)
        q, sx = acts["down"]
        sh.sherry_gemm(bufs["down"][0], q, sx, 0.02, bufs["down"][1], None, m, blk["down"].n,
                       blk["down"].k)

    for _ in range(2):
        layer()
    a, b = _events(torch)
    torch.cuda.synchronize()
    a.record()
    for _ in range(reps):
        layer()
    b.record()
    torch.cuda.synchronize()
    us = a.elapsed_time(b) / reps * 1e3
    ops = sum(2.0 * m * lin.n * lin.k for lin in blk.values())
    return {"m": m, "launches": ["qkv grouped", "o", "gate+up grouped", "down"],
            "per_layer_us": round(us, 2), "tops": round(ops / (us * 1e-6) / 1e12, 1),
            "mfma_frac": round(ops / (us * 1e-6) / 1e12 / INT8_PEAK_TOPS, 4)}


# ---------------------------------------------------------------------------
# other decode configurations: LLaMA-3.2-3B and the 8B-scale stress model
# ---------------------------------------------------------------------------

def time_graph(run, count, torch, replays=5):
    """us per launch of run(0..count-1), captured once in a HIP graph and
    replayed (no host launch cost between the kernels)."""
    for i in range(count):
        run(i)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            for i in range(count):
                run(i)
    torch.cuda.synchronize()
    for _ in range(2):
        g.replay()
    torch.cuda.synchronize()
    a, b = _events(torch)
    a.record()
    for _ in range(replays):
        g.replay()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / (replays * count) * 1e3


def bench_model_step(sh, torch, dev, spec, seed, copies, steps=100):
    """One fused decode step (all linears of the model, M = 1) in one launch."""
    step = DecodeStep(sh, torch, dev, spec, seed, copies=copies, keep_host=False)
    ms = bench_fused(step, torch, steps, 10)
    out = {"products": step.count, "copies": copies,
           "working_set_mb": round(step.weight_bytes * copies / 1e6, 1),
           "step_us": round(ms * 1e3, 2), "bytes_per_step": step.fused_bytes,
           "gbs": round(step.fused_bytes / (ms * 1e-3) / 1e9, 1)}
    out["frac"] = round(out["gbs"] / HBM_PEAK_GBS, 4)
    del step
    torch.cuda.empty_cache()
    return out


def bench_model_step_m(sh, torch, dev, spec, seed, m, copies, reps=20, group_scales=False,
                       il=False):
    """All linears of the model at M tokens in one grouped launch
    (sherry_gemm_batched, small-M MFMA kernel), int8 activations ready; with
    group_scales every product carries per-group (128 along K) scales; with
    il the weights are lane-interleaved (sherry_gemm_il_batched, M <= 16)."""
    lins = synth.model_linears(spec)
    pack = sh.sherry_pack_il if il else sh.sherry_pack
    host = [pack(synth.ternary_34(l.n, l.k, seed, "w", layer, l.name)) for layer, l in lins]
    sets = []
    for c in range(copies):
        w = [torch.from_numpy(p).to(dev) for p in host]
        ks = sorted({l.k for _, l in lins})
        q = {kk: torch.randint(-127, 128, (m, kk), dtype=torch.int8, device=dev) for kk in ks}
        sx = torch.full((m,), 0.01, dtype=torch.float32, device=dev)
        ys = [torch.empty((m, l.n), dtype=torch.float32, device=dev) for _, l in lins]
        gsc = ([torch.full((l.n, (l.k + 127) // 128), 0.02, dtype=torch.float32, device=dev)
                for _, l in lins] if group_scales else None)
        descs = (sh.sherry_gemm_desc * len(lins))()
        for i, (_, l) in enumerate(lins):
            d = descs[i]
            d.w, d.x, d.x_scale, d.y, d.acc = (w[i].data_ptr(), q[l.k].data_ptr(),
                                               sx.data_ptr(), ys[i].data_ptr(), None)
            d.n, d.k, d.m, d.w_scale = l.n, l.k, m, 0.02
            if group_scales:
                d.w_group_scales = gsc[i].data_ptr()
        prep = sh.sherry_gemm_il_batched_prepare if il else sh.sherry_gemm_batched_prepare
        total, max_m = prep(descs)
        dd = torch.from_numpy(sh.descs_to_bytes(descs)).to(dev)
        sets.append((w, q, sx, ys, dd, total, max_m, gsc))
    launch = sh.sherry_gemm_il_batched if il else sh.sherry_gemm_batched
    run = lambda i: launch(sets[i % copies][4], len(lins), sets[i % copies][5],
                           sets[i % copies][6])
    settle(run, torch, 0.02)
    a, b = _events(torch)
    a.record()
    for i in range(reps):
        run(i)
    b.record()
    torch.cuda.synchronize()
    us = a.elapsed_time(b) / reps * 1e3
    wbytes = sum(int(p.size) for p in host)
    byts = wbytes + sum(m * l.k + 4 * m + 4 * m * l.n for _, l in lins)
    if group_scales:
        byts += sum(4 * l.n * ((l.k + 127) // 128) for _, l in lins)
    del sets
    torch.cuda.empty_cache()
    return {"m": m, "products": len(lins), "group_scales": group_scales,
            "weights": "lane-interleaved" if il else "tiled",
            "step_us": round(us, 2), "bytes_per_step": byts,
            "gbs": round(byts / (us * 1e-6) / 1e9, 1),
            "tops": round(sum(2.0 * m * l.n * l.k for _, l in lins) / (us * 1e-6) / 1e12, 1)}


def _rotation(nbytes, floor=512 << 20):
    """Copies of a buffer of nbytes that together exceed floor (rotated so
    that the 256 MB Infinity Cache cannot serve them)."""
    return max(2, -(-floor // nbytes))


def bench_shapes(sh, torch, dev, spec, seed, ms, shapes=("q", "gate", "down"), reps=3):
    """Per-projection products at M tokens (sherry_gemm, automatic kernel
    choice), each timed over rotated copies of its weights, launched from a
    captured graph."""
    blk = {lin.name: lin for lin in synth.llama_block(spec["hidden"], spec["kv"], spec["inter"])}
    rows = []
    for name in shapes:
        lin = blk[name]
        t = synth.ternary_34(lin.n, lin.k, seed, "sk", name)
        packed = torch.from_numpy(sh.sherry_pack(t)).to(dev)
        nb = packed.numel()
        ws = [packed.clone() for _ in range(_rotation(nb))]
        for m in ms:
            x = torch.from_numpy(synth.activations(m, lin.k, seed, "skx", name, m)).to(dev)
            q = torch.empty((m, lin.k), dtype=torch.int8, device=dev)
            sx = torch.empty(m, dtype=torch.float32, device=dev)
            sh.sherry_quantize_act(x, q, sx)
            y = torch.empty((m, lin.n), dtype=torch.float32, device=dev)
            run = lambda i: sh.sherry_gemm(ws[i % len(ws)], q, sx, 0.02, y, None, m, lin.n, lin.k)
            us = time_graph(run, reps * len(ws), torch)
            byts = nb + m * lin.k + 4 * m + 4 * m * lin.n
            rows.append({"proj": name, "n": lin.n, "k": lin.k, "m": m, "us": round(us, 3),
                         "gbs": round(byts / (us * 1e-6) / 1e9, 1),
                         "tops": round(2.0 * m * lin.n * lin.k / (us * 1e-6) / 1e12, 2),
                         "kernel": KERNEL_NAMES[sh.sherry_gemm_kernel_for(m, lin.n, lin.k)]})
            del x, q, sx, y
        del ws, packed
        torch.cuda.empty_cache()
    return rows


def bench_scale_granularity(sh, torch, dev, spec, seed, ms=(1, 16), shapes=("q", "gate", "down"),
                            reps=3):
    """The same products with one weight scale, one per output channel and
    one per 128-weight group (M = 1 on the VALU kernel, M = 16 on the
    register-decoded one), each timed over rotated weight copies from a
    captured graph.  Bytes count the scale vectors (4N, 4N*K/128)."""
    blk = {lin.name: lin for lin in synth.llama_block(spec["hidden"], spec["kv"], spec["inter"])}
    rows = []
    for name in shapes:
        lin = blk[name]
        n, k = lin.n, lin.k
        t = synth.ternary_34(n, k, seed, "gsk", name)
        packed = torch.from_numpy(sh.sherry_pack(t)).to(dev)
        nb = packed.numel()
        ws = [packed.clone() for _ in range(_rotation(nb))]
        g = (k + 127) // 128
        rng = np.random.default_rng([seed, n, k])
        sw_rows = torch.from_numpy((rng.random(n) * 0.04 + 0.01).astype(np.float32)).to(dev)
        sw_groups = torch.from_numpy((rng.random((n, g)) * 0.04 + 0.01).astype(np.float32)).to(dev)
        for m in ms:
            q = torch.from_numpy(synth.int8_any(m, k, seed, "gskx", name, m)).to(dev)
            sx = torch.full((m,), 0.01, dtype=torch.float32, device=dev)
            y = torch.empty((m, n), dtype=torch.float32, device=dev)
            kern = sh.SHERRY_KERNEL_GEMV if m <= 4 else sh.SHERRY_KERNEL_SKINNY
            base = nb + m * k + 4 * m + 4 * m * n
            runs = {
                "tensor": (lambda i: sh.sherry_gemm_ex(ws[i % len(ws)], q, sx, 0.02, y, None,
                                                       m, n, k, kern), base),
                "channel": (lambda i: sh.sherry_gemm_channel(ws[i % len(ws)], q, sx, sw_rows, y,
                                                             None, m, n, k, kern), base + 4 * n),
                "group128": (lambda i: sh.sherry_gemm_group(ws[i % len(ws)], q, sx, sw_groups, y,
                                                            None, m, n, k, kern),
                             base + 4 * n * g),
            }
            row = {"proj": name, "n": n, "k": k, "m": m, "kernel": KERNEL_NAMES[kern]}
            for key, (run, byts) in runs.items():
                us = time_graph(run, reps * len(ws), torch)
                row[key + "_us"] = round(us, 3)
                row[key + "_gbs"] = round(byts / (us * 1e-6) / 1e9, 1)
            rows.append(row)
            del q, sx, y
        del ws, packed
        torch.cuda.empty_cache()
    return rows


def bench_activation_tables(sh, torch, dev, spec, seed, shapes=("q", "gate", "down"), reps=3):
    """M = 1 products on the weight-table kernel (the library's GEMV) and on
    the activation-table kernel (the paper's LUT direction), same packed
    weights rotated over copies, launched from a captured graph."""
    blk = {lin.name: lin for lin in synth.llama_block(spec["hidden"], spec["kv"], spec["inter"])}
    rows = []
    for name in shapes:
        lin = blk[name]
        n, k = lin.n, lin.k
        t = synth.ternary_34(n, k, seed, "atk", name)
        packed = torch.from_numpy(sh.sherry_pack(t)).to(dev)
        nb = packed.numel()
        ws = [packed.clone() for _ in range(_rotation(nb))]
        q = torch.from_numpy(synth.int8_any(1, k, seed, "atkx", name)).to(dev)
        sx = torch.full((1,), 0.01, dtype=torch.float32, device=dev)
        y = torch.empty((n,), dtype=torch.float32, device=dev)
        byts = nb + k + 4 + 4 * n
        row = {"proj": name, "n": n, "k": k}
        for key, kern in (("weight_table", sh.SHERRY_KERNEL_GEMV),
                          ("activation_table", sh.SHERRY_KERNEL_ALUT)):
            us = time_graph(lambda i: sh.sherry_gemm_ex(ws[i % len(ws)], q, sx, 0.02, y, None,
                                                        1, n, k, kern), reps * len(ws), torch)
            row[key + "_us"] = round(us, 3)
            row[key + "_gbs"] = round(byts / (us * 1e-6) / 1e9, 1)
        rows.append(row)
        del ws, packed, q, sx, y
        torch.cuda.empty_cache()
    return rows


def bench_layouts_8b(sh, torch, dev, seed, reps=30):
    """One M = 1 decode step of the 8B-scale stress model (32 layers x 7
    linears, int8 activations and scales ready) in each of the three layouts
    of Sec. 2.3, each as one grouped launch: the 1.25-bit 3:4 codes
    (sherry_gemv_batched), three weights per 5-bit code (1.67 bits,
    sherry_gemv3_batched) and 2 bits per weight (sherry_gemv2_batched).  The
    same ternary 3:4 weights feed all three.  One layer's seven matrices are
    generated and packed on the host; each of the 32 layers streams its own
    device copy of them, so every step reads its whole weight set from HBM
    (1.09 to 1.74 GB, beyond the Infinity Cache)."""
    spec = synth.STRESS_8B
    blk = synth.llama_block(spec["hidden"], spec["kv"], spec["inter"])
    ts = [synth.ternary_34(lin.n, lin.k, seed, "lay", lin.name) for lin in blk]
    ks = sorted({lin.k for lin in blk})
    q = {kk: torch.from_numpy(synth.int8_any(1, kk, seed, "layx", kk)).to(dev) for kk in ks}
    sx = torch.full((1,), 0.01, dtype=torch.float32, device=dev)
    layouts = (("sherry_1.25bit", sh.sherry_pack, sh.sherry_gemv_batched_prepare,
                sh.sherry_gemv_batched),
               ("three_in_5bit_1.67bit", sh.sherry_pack3, sh.sherry_gemv3_batched_prepare,
                sh.sherry_gemv3_batched),
               ("two_bit", sh.sherry_pack2, sh.sherry_gemv2_batched_prepare,
                sh.sherry_gemv2_batched))
    rows = {}
    for name, pack, prep, run in layouts:
        host = [pack(t) for t in ts]
        w = [[torch.from_numpy(h).to(dev) for h in host] for _ in range(spec["layers"])]
        ys = [[torch.empty(lin.n, dtype=torch.float32, device=dev) for lin in blk]
              for _ in range(spec["layers"])]
        count = spec["layers"] * len(blk)
        descs = (sh.sherry_gemv_desc * count)()
        for layer in range(spec["layers"]):
            for j, lin in enumerate(blk):
                d = descs[layer * len(blk) + j]
                d.w, d.x, d.x_scale, d.y, d.acc = (w[layer][j].data_ptr(), q[lin.k].data_ptr(),
                                                   sx.data_ptr(), ys[layer][j].data_ptr(), None)
                d.n, d.k, d.w_scale = lin.n, lin.k, 0.02
        total = prep(descs)
        dd = torch.from_numpy(sh.descs_to_bytes(descs)).to(dev)
        go = lambda i: run(dd, count, total)
        settle(go, torch, 0.03)
        a, b = _events(torch)
        a.record()
        for i in range(reps):
            go(i)
        b.record()
        torch.cuda.synchronize()
        us = a.elapsed_time(b) / reps * 1e3
        wbytes = spec["layers"] * sum(int(h.size) for h in host)
        byts = wbytes + spec["layers"] * sum(lin.k + 4 + 4 * lin.n for lin in blk)
        rows[name] = {"weight_bytes": wbytes, "bytes_per_step": byts, "step_us": round(us, 2),
                      "gbs": round(byts / (us * 1e-6) / 1e9, 1),
                      "frac": round(byts / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}
        del w, ys, dd, host
        torch.cuda.empty_cache()
    ref = rows["sherry_1.25bit"]
    for name in ("three_in_5bit_1.67bit", "two_bit"):
        rows[name]["sherry_bytes_ratio"] = round(ref["weight_bytes"] / rows[name]["weight_bytes"], 4)
        rows[name]["sherry_time_ratio"] = round(ref["step_us"] / rows[name]["step_us"], 4)
    return {"workload": "8B-scale stress decode step, M=1, 32 layers x 7 linears (224 products), "
                        "int8 activations, one grouped launch per layout",
            "products": spec["layers"] * len(blk), "layouts": rows}


# ---------------------------------------------------------------------------
# CPU baseline: the oracle on the host cores
# ---------------------------------------------------------------------------

def oracle_step(step: DecodeStep, threads: int):
    """One full decode step on the CPU oracle: per product, the activation
    quantization, the int32 product on the unpacked ternary matrix and the
    fp64 epilogue.  Returns [(x_scale, acc, y)] in product order."""
    import oracle
    out = []
    row = {kk: 0 for kk in step.ks}
    for i, (_, lin) in enumerate(step.lins):
        q, sx = oracle.quantize_act(step.x_host[lin.k][row[lin.k]:row[lin.k] + 1])
        row[lin.k] += 1
        acc = oracle.gemm_i32(q, step.t[i], threads=threads)
        out.append((sx, acc, oracle.epilogue(acc, sx, step.scales[i])))
    return out


def host_cpu():
    """Core counts and model of the host CPU the oracle runs on."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    avail = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    return {"nproc": os.cpu_count(), "available": avail, "model": model}


def _time_oracle(step, threads, min_seconds, max_reps=2000):
    reps, t_total, last = 0, 0.0, None
    while (t_total < min_seconds or reps == 0) and reps < max_reps:
        t0 = time.perf_counter()
        last = oracle_step(step, threads)
        t_total += time.perf_counter() - t0
        reps += 1
    return reps, t_total / reps, last


def cpu_baseline(step: DecodeStep, min_seconds=10.0, single_seconds=5.0):
    """The oracle as it stands, timed on the host over full decode steps of
    the benchmark's workload: with one thread per core of this process's
    share (at most 16, the host share of one GPU) and with one thread.
    Returns the JSON record and the last step's results."""
    cpu = host_cpu()
    threads = max(1, min(16, cpu["available"] or 1))
    reps, per_step, last = _time_oracle(step, threads, min_seconds)
    reps1, per_step1, _ = _time_oracle(step, 1, single_seconds)
    rec = {"value": round(step.fused_bytes / per_step / 1e9, 3),
           "unit": "GB/s", "cores": threads, "kind": "oracle",
           "sample": "%d full decode step(s) of the same workload (112 products of the "
                     "16-layer LLaMA-3.2-1B linears, quantize + int32 product + fp64 "
                     "epilogue), %d threads over output rows; algorithmic bytes as the GPU "
                     "line, the oracle reads T unpacked at 1 byte/weight; %.3f s per step"
                     % (reps, threads, per_step),
           "single_thread": {"value": round(step.fused_bytes / per_step1 / 1e9, 4),
                             "unit": "GB/s", "cores": 1, "steps": reps1,
                             "s_per_step": round(per_step1, 3)},
           "host": cpu}
    return rec, last


def step_parity(sh, step: DecodeStep, torch, ref):
    """Checks the decode step against the oracle's results for the same
    inputs: every fp32 output of the last timed launch of copy 0 (saved right
    after the timed loop), then an untimed launch of the same descriptors
    with int32 outputs (bit-exact) and the activation scales it writes
    (bit-exact)."""
    cp = step.copies[0]
    ys = step.timed_y
    torch.cuda.synchronize()
    sh.sherry_gemv_f32_il_batched(cp["fdescs_acc_il"], step.count, cp["ftotal_il"])
    torch.cuda.synchronize()
    accs = [a.cpu().numpy() for a in cp["accs"]]
    sxs = {kk: cp["sxs"][kk].cpu().numpy() for kk in step.ks}
    row = {kk: 0 for kk in step.ks}
    acc_ok = sx_ok = True
    worst, outputs = 0.0, 0
    for i, (_, lin) in enumerate(step.lins):
        sx_ref, acc_ref, y_ref = ref[i]
        acc_ok &= bool(np.array_equal(accs[i], acc_ref[0]))
        sx_ok &= bool(sxs[lin.k][row[lin.k]] == sx_ref[0])
        row[lin.k] += 1
        yr = y_ref[0]
        err = np.abs(ys[i].astype(np.float64) - yr)
        nz = yr != 0
        if (~nz & (err != 0)).any():
            worst = float("inf")
        elif nz.any():
            worst = max(worst, float(np.max(err[nz] / np.abs(yr[nz]))))
        outputs += lin.n
    ok = acc_ok and sx_ok and worst <= 1e-5
    return {"products": step.count, "outputs": outputs, "acc_bit_exact": acc_ok,
            "x_scale_bit_exact": sx_ok, "y_max_rel_err": worst, "tolerance": 1e-5, "ok": ok,
            "checked": "every y of the timed step (copy 0), every int32 accumulator and "
                       "activation scale of one more launch of the same descriptors, "
                       "against the CPU oracle on the same inputs"}


def bench_config0(sh, torch, dev, seed, reps=3):
    """The single-GEMV case: LLaMA-3.2-1B q_proj shape, M = 1, K = N = 2048,
    per-tensor scale 0.02, fp32 N(0,1) activations quantized in the same
    launch (sherry_gemv_f32); weights rotated over copies totalling more than
    600 MB, launched from a captured graph."""
    n = k = 2048
    t = synth.ternary_34(n, k, seed, "c0", "q")
    packed = torch.from_numpy(sh.sherry_pack(t)).to(dev)
    nb = packed.numel()
    ncp = -(-600_000_000 // nb) + 24
    ws = [packed.clone() for _ in range(ncp)]
    x = torch.from_numpy(synth.activations(1, k, seed, "c0x")[0]).to(dev)
    sx = torch.empty(1, dtype=torch.float32, device=dev)
    y = torch.empty(n, dtype=torch.float32, device=dev)
    us = time_graph(lambda i: sh.sherry_gemv_f32(ws[i % ncp], x, sx, 0.02, y, None, n, k),
                    reps * ncp, torch)
    byts = nb + 4 * k + 4 + 4 * n
    del ws, packed
    torch.cuda.empty_cache()
    return {"workload": "single GEMV, M=1, K=N=2048 (LLaMA-3.2-1B q_proj), sw=0.02, "
                        "fused int8 quantization", "copies": ncp,
            "working_set_mb": round(nb * ncp / 1e6, 1), "us": round(us, 3),
            "bytes": byts, "gbs": round(byts / (us * 1e-6) / 1e9, 1),
            "frac": round(byts / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
            "note": "one launch per GEMV; 665 KB per call, so launch latency dominates"}


# the kernel of the headline step (the fused product on lane-interleaved units)
DECODE_KERNEL = "gemv_f32_batched_kernel<true>"


def load_traffic(src_hash: str, kernel: str):
    path = os.path.join(ROOT, "profiles", "traffic_gemv_f32_batched.json")
    try:
        with open(path) as f:
            d = json.load(f)
    except (OSError, ValueError):
        return None
    if d.get("kernel_source_hash") != src_hash or d.get("kernel") != kernel:
        return None
    return d.get("bytes_per_launch")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--seed", type=int, default=synth.DEFAULT_SEED)
    ap.add_argument("--copies", type=int, default=COPIES,
                    help="rotated weight copies (working set = copies x 152 MB)")
    ap.add_argument("--no-extra", action="store_true", help="skip the M=2048 GEMM and ceiling")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--only", choices=["decode", "product", "prefill", "grouped", "ternarize",
                                       "tables", "layouts", "read"],
                    default=None,
                    help="run only one part (for profiler runs): the timed decode steps, the "
                         "back-to-back product launches, the M=2048 LLaMA-3.2-3B layer, the "
                         "grouped small-M steps, ternarize + pack, or the streaming read of "
                         "the decode step's bytes per launch")
    ap.add_argument("--product-launches", type=int, default=1000,
                    help="back-to-back grouped product launches timed for the roofline")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="run 10 plain device copies of BYTES and exit (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(see DESIGN.md for how the product would shard); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2601_07892_amd as sh
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log(sh.sherry_version(), torch.cuda.get_device_name(dev))

    if args.copy_probe:
        n = args.copy_probe // 4 * 4
        src = torch.ones(n // 4, dtype=torch.int32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(10):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_probe_bytes": n, "launches": 10}), flush=True)
        return
    if args.only:
        args.no_extra = args.no_cpu = True
    if args.only == "prefill":
        r = bench_prefill(sh, torch, dev, synth.LLAMA_3B, 2048, args.seed)
        g = bench_prefill_grouped(sh, torch, dev, synth.LLAMA_3B, 2048, args.seed)
        log("prefill llama-3.2-3b M=2048: %.1f TOPS per projection launch, %.1f TOPS "
            "with grouped launches" % (r["tops"], g["tops"]))
        print(json.dumps({"prefill_m2048_llama-3.2-3b": r,
                          "prefill_m2048_grouped_llama-3.2-3b": g}), flush=True)
        return
    if args.only == "grouped":
        rows = [bench_model_step_m(sh, torch, dev, synth.LLAMA_3B, args.seed, mm, 2)
                for mm in (4, 16)]
        rows += [bench_model_step_m(sh, torch, dev, synth.LLAMA_3B, args.seed, mm, 2, il=True)
                 for mm in (4, 8, 16)]
        rows.append(bench_model_step_m(sh, torch, dev, synth.STRESS_8B, args.seed, 64, 1))
        rows += [bench_model_step_m(sh, torch, dev, synth.LLAMA_3B, args.seed, mm, 2,
                                    group_scales=True) for mm in (4, 16)]
        print(json.dumps({"decode_small_m_grouped": rows}), flush=True)
        return
    if args.only == "read":
        nbytes = sum(sh.sherry_packed_bytes(l.n, l.k) + 4 * l.k + 4 + 4 * l.n
                     for _, l in synth.model_linears(synth.LLAMA_1B))
        print(json.dumps({"hbm_read_same_bytes": bench_stream_same_bytes(sh, torch, dev, nbytes)}),
              flush=True)
        return
    if args.only == "tables":
        print(json.dumps({"activation_vs_weight_tables_3b": bench_activation_tables(
            sh, torch, dev, synth.LLAMA_3B, args.seed)}), flush=True)
        return
    if args.only == "layouts":
        print(json.dumps({"layouts_8b_step": bench_layouts_8b(sh, torch, dev, args.seed)}),
              flush=True)
        return
    if args.only == "ternarize":
        print(json.dumps({"ternarize_pack": bench_ternarize(sh, torch, dev, args.seed)}),
              flush=True)
        return

    step = DecodeStep(sh, torch, dev, synth.LLAMA_1B, args.seed, copies=args.copies)
    if args.only == "product":
        heat(sh, torch, dev)
        kern_ms = bench_product_only(step, torch, args.product_launches)
        log("int8 grouped product %.2f us back to back over %d launches" %
            (kern_ms * 1e3, args.product_launches))
        print(json.dumps({"kernel": "gemv_batched_kernel", "launches": args.product_launches,
                          "avg_launch_us": round(kern_ms * 1e3, 3),
                          "bytes_per_launch": step.gemv_bytes}), flush=True)
        return
    ms_step = bench_fused(step, torch, args.steps, args.warmup)
    # the outputs of the timed steps (copy 0's last launch), before any other
    # run writes the same buffers
    step.timed_y = [y.cpu().numpy() for y in step.copies[0]["ys"]]
    value = step.fused_bytes / (ms_step * 1e-3) / 1e9
    log("decode step (fused quantize + product, one launch) %.2f us, %.0f GB/s" %
        (ms_step * 1e3, value))
    if args.only == "decode":
        print(json.dumps({"kernel": "gemv_f32_batched_kernel<true>", "launches": args.steps,
                          "avg_launch_us": round(ms_step * 1e3, 3),
                          "bytes_per_launch": step.fused_bytes}), flush=True)
        return
    ms_tiled = bench_fused(step, torch, args.steps, args.warmup, tiled=True)
    log("the same step on the tiled layout %.2f us" % (ms_tiled * 1e3))
    ms_unfused = bench_unfused(step, torch, args.steps, args.warmup)
    ms_two = bench_two_launch(step, torch, args.steps, args.warmup)
    kern_ms = bench_product_only(step, torch, args.product_launches)
    log("unfused step %.2f us; grouped quantize + product %.2f us; int8 grouped product alone "
        "%.2f us (%.0f GB/s)" % (ms_unfused * 1e3, ms_two * 1e3, kern_ms * 1e3,
                                 step.gemv_bytes / (kern_ms * 1e-3) / 1e9))
    src_hash = kernel_source_hash(["gemv.hip", "sherry_internal.h"])
    out = {
        "metric": "ternary GEMV GB/s & % HBM peak at M=1; GEMM TOPS at M=2048 (LLaMA-1B shapes)",
        "value": round(value, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "int8xternary->int32",
        "data": "synthetic",
        "config": {"workload": "llama-3.2-1b decode step, M=1, 16 layers x 7 projections "
                               "(112 GEMVs), 1.25-bit 3:4 ternary, %d rotated copies" % args.copies,
                   "weights_mb_per_copy": round(step.weight_bytes / 1e6, 2),
                   "working_set_mb": round(step.weight_bytes * args.copies / 1e6, 1),
                   "step": "1 launch: per-token int8 quantization fused with the 112 products",
                   "weights": "lane-interleaved units (sherry_pack_il)",
                   "seed": args.seed},
        "roofline": {"bound": "hbm", "achieved": round(value, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(value / HBM_PEAK_GBS, 4),
                     "traffic": load_traffic(src_hash, DECODE_KERNEL),
                     "kernel": DECODE_KERNEL,
                     "bytes_per_launch": step.fused_bytes,
                     "avg_launch_us": round(ms_step * 1e3, 3),
                     "kernel_source_hash": src_hash},
        "fused_tiled": {"step_us": round(ms_tiled * 1e3, 2),
                        "gbs": round(step.fused_bytes / (ms_tiled * 1e-3) / 1e9, 1),
                        "what": "the same fused step on the tiled layout (sherry_gemv_f32_batched)"},
        "two_launch": {"step_us": round(ms_two * 1e3, 2),
                       "gbs": round(step.fused_bytes / (ms_two * 1e-3) / 1e9, 1),
                       "launches": "sherry_quantize_act_batched (112 rows) + "
                                   "sherry_gemv_batched (112 products)"},
        "unfused": {"step_us": round(ms_unfused * 1e3, 2),
                    "int8_product_us": round(kern_ms * 1e3, 3),
                    "int8_product_gbs": round(step.gemv_bytes / (kern_ms * 1e-3) / 1e9, 1),
                    "int8_product_bytes": step.gemv_bytes},
    }
    if not args.no_extra:
        ms_ch = bench_fused(step, torch, args.steps, args.warmup, channel=True)
        ch_bytes = step.fused_bytes + sum(4 * lin.n for _, lin in step.lins)
        out["per_channel_decode_step"] = {
            "step_us": round(ms_ch * 1e3, 2), "bytes_per_step": ch_bytes,
            "gbs": round(ch_bytes / (ms_ch * 1e-3) / 1e9, 1),
            "time_vs_per_tensor": round(ms_ch / ms_step, 4)}
        log("decode step, per-channel scales: %.2f us" % (ms_ch * 1e3))
        out["scale_granularity_3b"] = bench_scale_granularity(sh, torch, dev, synth.LLAMA_3B,
                                                              args.seed)
        for r in out["scale_granularity_3b"]:
            log("3b %s M=%d: tensor %.2f us, channel %.2f us, group-128 %.2f us" %
                (r["proj"], r["m"], r["tensor_us"], r["channel_us"], r["group128_us"]))
        out["ternarize_pack"] = bench_ternarize(sh, torch, dev, args.seed)
        for r in out["ternarize_pack"]:
            log("ternarize+pack %s: %.1f us, %.0f GB/s" % (r["shape"], r["us"], r["gbs"]))
        out["hbm_read_ceiling_gbs"] = round(bench_stream_ceiling(sh, torch, dev), 1)
        same = bench_stream_same_bytes(sh, torch, dev, step.fused_bytes)
        same["decode_step_over_read"] = round(same["us"] / (ms_step * 1e3), 4)
        out["hbm_read_same_bytes"] = same
        log("streaming read of the step's %d bytes: %.2f us, %.0f GB/s" %
            (same["bytes"], same["us"], same["gbs"]))
        out["config0_single_gemv"] = bench_config0(sh, torch, dev, args.seed)
        log("config 0 single GEMV: %.2f us, %.0f GB/s" % (out["config0_single_gemv"]["us"],
                                                       out["config0_single_gemv"]["gbs"]))
        pre = {}
        for name, spec in (("llama-3.2-3b", synth.LLAMA_3B), ("llama-3.2-1b", synth.LLAMA_1B)):
            pre[name] = bench_prefill(sh, torch, dev, spec, 2048, args.seed)
            log("prefill %s M=2048: %.1f TOPS (dense int8 GEMM on unpacked weights: %.1f TOPS)" %
                (name, pre[name]["tops"], pre[name]["dense_int8_ref"]["tops"]))
        out["prefill_m2048"] = pre
        grp = {}
        for name, spec in (("llama-3.2-3b", synth.LLAMA_3B), ("llama-3.2-1b", synth.LLAMA_1B)):
            grp[name] = bench_prefill_grouped(sh, torch, dev, spec, 2048, args.seed)
            log("prefill %s M=2048, grouped launches: %.1f TOPS" % (name, grp[name]["tops"]))
        out["prefill_m2048_grouped"] = grp
        other = {}
        for name, spec, copies in (("llama-3.2-3b", synth.LLAMA_3B, 2),
                                   ("stress-8b", synth.STRESS_8B, 1)):
            other[name] = bench_model_step(sh, torch, dev, spec, args.seed, copies)
            log("decode step %s (%d products): %.2f us, %.0f GB/s" %
                (name, other[name]["products"], other[name]["step_us"], other[name]["gbs"]))
        out["decode_other_models"] = other
        grouped = {"llama-3.2-3b": [bench_model_step_m(sh, torch, dev, synth.LLAMA_3B, args.seed,
                                                       mm, 2) for mm in (4, 16)],
                   "stress-8b": [bench_model_step_m(sh, torch, dev, synth.STRESS_8B, args.seed,
                                                    64, 1)],
                   "llama-3.2-3b-group128": [bench_model_step_m(sh, torch, dev, synth.LLAMA_3B,
                                                                args.seed, mm, 2,
                                                                group_scales=True)
                                             for mm in (4, 16)],
                   "llama-3.2-3b-interleaved": [bench_model_step_m(sh, torch, dev,
                                                                   synth.LLAMA_3B, args.seed,
                                                                   mm, 2, il=True)
                                                for mm in (4, 8, 16)]}
        for name, rows in grouped.items():
            for r in rows:
                log("grouped step %s M=%d: %.2f us, %.0f GB/s, %.1f TOPS" %
                    (name, r["m"], r["step_us"], r["gbs"], r["tops"]))
        out["decode_small_m_grouped"] = grouped
        out["projections_by_m"] = {
            "llama-3.2-3b": bench_shapes(sh, torch, dev, synth.LLAMA_3B, args.seed, (1, 4, 16)),
            "stress-8b": bench_shapes(sh, torch, dev, synth.STRESS_8B, args.seed, (1, 64)),
        }
        out["layouts_8b_step"] = bench_layouts_8b(sh, torch, dev, args.seed)
        out["activation_vs_weight_tables_3b"] = bench_activation_tables(sh, torch, dev,
                                                                        synth.LLAMA_3B, args.seed)
        for r in out["activation_vs_weight_tables_3b"]:
            log("3b %s M=1: weight tables %.2f us, activation tables %.2f us" %
                (r["proj"], r["weight_table_us"], r["activation_table_us"]))
        for name, r in out["layouts_8b_step"]["layouts"].items():
            log("8b step, %s: %.2f us, %.0f GB/s (%d weight bytes)" %
                (name, r["step_us"], r["gbs"], r["weight_bytes"]))
    t0 = time.time()
    if not args.no_cpu:
        out["cpu_baseline"], ref = cpu_baseline(step)
        log("cpu baseline %.1f s" % (time.time() - t0))
    else:
        ref = oracle_step(step, max(1, min(16, host_cpu()["available"] or 1)))
    out["parity"] = step_parity(sh, step, torch, ref)
    log("parity of the timed step against the oracle: %s (max rel err %.3g)" %
        ("ok" if out["parity"]["ok"] else "FAILED", out["parity"]["y_max_rel_err"]))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
