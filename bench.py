#!/usr/bin/env python3
"""Benchmark of the sparse-input convolution on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--all --out FILE]

A step is one pass of the whole hot path over one batch of synthetic input
already resident in HBM: isc_conv2d on the AUTO path, i.e. the nonzero count
of the input and the device-side sparse/dense decision, then the
zero-skipping convolution (ISC steps 1-3: compaction on the fly, the
multiply-adds over nonzeros only, the write-out to NCHW); the dense kernel is
launched too and exits on the decision.

Workload: AlexNet conv2 (96 -> 256 maps, 27 x 27, 5 x 5, pad 2) at batch 128,
input sparsity 0.9 (i.i.d. zeros, |N(0,1)| nonzeros, N(0, 0.01) weights): the
largest single-GPU configuration at the sparsity the metric is quoted at.

Timing protocol: each timed step (and each rep of every other figure) runs
after a 512 MiB write that evicts the caches (twice the 256 MB last-level
cache), outside the interval timed by HIP events on the launch stream; a
step is replayed from a HIP graph whose launches are queued behind that
write, so host-side enqueue time never enters the interval.  `value` is the
dense-equivalent rate at the median of the K cold steps (p10 / p90 beside
it); the warm figures (back-to-back replays, caches hot) come alongside.
Paths compared with each other (AUTO, sparse, dense, the compaction and the
sparse kernel alone; the chain's three forms) take their cold reps
interleaved, rep i of each before rep i + 1 of any.

Prints ONE JSON line: value = dense-equivalent TFLOP/s of the step
(2*N*K*C*R*S*Ho*Wo per step), speedup against the same GPU's dense path
(fp32-MFMA GEMM with the im2col gather inside) and against the vendor
library's fp32 convolution, nonzero-MAC/s, the LeNet conv2 sparsity sweep
0.5 .. 0.99 with roofline fractions per point, the roofline of the dominant
kernel (HIP events on the launch stream), and the CPU oracle timed on a
bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workloads  # noqa: E402

METRIC = "sparse-input conv: dense-equiv TFLOP/s & speedup vs dense at sparsity 0.9"
HBM_PEAK_GBS = 8000.0
# fp32 FMA on the vector ALUs without packed instructions (disabled in this
# build): 256 CUs x 4 SIMDs x 16 lanes x 2 flop x 2.4 GHz
VALU_F32_PEAK_TFLOPS = 78.6
VALU_F32_PACKED_PEAK_TFLOPS = 157.3
MFMA_F32_PEAK_TFLOPS = 157.3


def dense_flops(layer, Ho, Wo) -> float:
    return 2.0 * layer.N * layer.K * layer.C * layer.R * layer.S * Ho * Wo


def taps_per_coord(n_in, k, pad, stride, n_out) -> np.ndarray:
    """For each input coordinate u, how many filter offsets q put it on a
    valid output ((u + pad - q) divisible by stride, quotient in range)."""
    u = np.arange(n_in)[:, None]
    q = np.arange(k)[None, :]
    num = u + pad - q
    ok = (num >= 0) & (num % stride == 0) & (num // stride < n_out)
    return ok.sum(axis=1)


def nonzero_macs(x, layer, Ho, Wo) -> int:
    """Multiply-adds the zero-skipping convolution performs on x (bookkeeping
    for the nonzero-MAC/s figure)."""
    nzmask = (x.view(np.uint32) & np.uint32(0x7FFFFFFF)) != 0
    per_pos = nzmask.sum(axis=(0, 1)).astype(np.int64)          # H x W counts
    ty = taps_per_coord(layer.H, layer.R, layer.P, layer.T, Ho)
    tx = taps_per_coord(layer.W, layer.S, layer.P, layer.T, Wo)
    return int(layer.K * (per_pos * ty[:, None] * tx[None, :]).sum())


FLUSH_BYTES = 512 << 20   # twice the 256 MB last-level cache (MALL)


class ColdTimer:
    """Per-rep HIP-event times with the caches evicted before every rep: a
    512 MiB write, then the start event, the work, the end event, all on the
    current stream with no host synchronisation in between (so the work's
    launches wait queued behind the write)."""

    def __init__(self, torch):
        self.torch = torch
        self.buf = torch.empty(FLUSH_BYTES // 4, dtype=torch.float32, device="cuda")
        self.count = 0

    def flush(self):
        self.count += 1
        self.buf.fill_(float(self.count & 0xFFFF))

    def times(self, fn, reps: int, warm: int = 2):
        torch = self.torch
        evs = []
        for i in range(warm + reps):
            self.flush()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            evs.append((a, b))
        torch.cuda.synchronize()
        return [a.elapsed_time(b) for a, b in evs[warm:]]

    def times_interleaved(self, fns: dict, reps: int, warm: int = 2) -> dict:
        """times() of several functions with their reps interleaved (rep i of
        every function before rep i + 1 of any), so that clock and cache
        drift over the run falls on all of them alike."""
        torch = self.torch
        evs = {name: [] for name in fns}
        for i in range(warm + reps):
            for name, fn in fns.items():
                self.flush()
                a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record()
                fn()
                b.record()
                evs[name].append((a, b))
        torch.cuda.synchronize()
        return {name: [a.elapsed_time(b) for a, b in ev[warm:]] for name, ev in evs.items()}


def stats(ms) -> dict:
    """Median, p10, p90 and mean of per-rep milliseconds."""
    a = np.asarray(ms, dtype=np.float64)
    return {"median": round(float(np.median(a)), 6), "p10": round(float(np.percentile(a, 10)), 6),
            "p90": round(float(np.percentile(a, 90)), 6), "mean": round(float(a.mean()), 6), "reps": int(a.size)}


def event_time_ms(torch, fn, reps: int, warm: int = 3) -> float:
    """Average ms per call of fn, by HIP events on the current stream around
    `reps` back-to-back calls."""
    for _ in range(warm):
        fn()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    s.record()
    for _ in range(reps):
        fn()
    e.record()
    e.synchronize()
    return s.elapsed_time(e) / reps


def graph_of(torch, fn, inner: int = 1):
    """Capture `inner` back-to-back calls of fn (which launches on the
    current stream) into one HIP graph."""
    fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(inner):
            fn()
    torch.cuda.synchronize()
    return g


def kernel_time_ms(torch, fn, reps: int, graphs: bool = True, inner: int = 20) -> float:
    """Average device time per launch of fn: `inner` launches captured in one
    graph and replayed, HIP events around the replays on the launch stream,
    so that host-side argument marshalling does not enter the figure."""
    if not graphs:
        return event_time_ms(torch, fn, reps)
    g = graph_of(torch, fn, inner)
    return event_time_ms(torch, g.replay, max(2, reps // inner + 1)) / inner


class LayerRun:
    """Device buffers and callables for one layer."""

    def __init__(self, torch, isc, layer):
        self.torch, self.isc, self.layer = torch, isc, layer
        x, w = workloads.make_inputs(layer)
        self.x_host = x
        self.x = torch.from_numpy(x).cuda()
        self.w = torch.from_numpy(w).cuda()
        L = layer
        self.desc = isc.make_desc(L.N, L.C, L.H, L.W, L.K, L.R, L.S, L.T, L.P)
        self.Ho, self.Wo = isc.isc_out_shape(self.desc)
        self.y = torch.empty((L.N, L.K, self.Ho, self.Wo), device="cuda")
        self.ws = {p: isc.workspace(self.desc, p) for p in ("auto", "sparse", "dense")}
        self.kernel = isc.isc_sparse_kernel(self.desc)  # the sparse path's main kernel
        self.lists = isc.isc_compact(self.x)
        self.wt = isc.isc_repack_filter(self.w)
        self.col = None  # im2col matrix, allocated by im2col() when first used
        torch.cuda.synchronize()
        self.nnz = int(self.lists[2].item())
        self.sparsity = 1.0 - self.nnz / x.size
        self.flops = dense_flops(L, self.Ho, self.Wo)
        self.nz_macs = nonzero_macs(x, L, self.Ho, self.Wo)

    def conv(self, path, threshold=None):
        L = self.layer
        return lambda: self.isc.isc_conv2d(self.x, self.w, L.T, L.P, path=path, threshold=threshold,
                                           out=self.y, ws=self.ws[path])

    def compact(self):
        return lambda: self.isc.isc_compact(self.x, out=self.lists)

    def sparse_kernel(self):
        """The sparse path's main kernel alone, through its own entry point:
        on-the-fly compaction (isc_sparse_conv_fused) or the kernel over
        compacted lists (isc_sparse_conv)."""
        L = self.layer
        if self.kernel in ("fused", "fused_ring", "fused_reg"):
            return lambda: self.isc.isc_sparse_conv_fused(self.x, self.wt, L.T, L.P, out=self.y)
        return lambda: self.isc.isc_sparse_conv(self.x.shape, self.lists, self.wt, L.T, L.P,
                                                out=self.y)

    def im2col(self):
        """The stand-alone im2col entry point (not on the dense path, which
        gathers inside its GEMM); kept for the counter runs."""
        L = self.layer
        if self.col is None:
            self.col = self.torch.empty((L.C * L.R * L.S, L.N * self.Ho * self.Wo), device="cuda")
        return lambda: self.isc.isc_im2col(self.x, L.R, L.S, L.T, L.P, out=self.col)

    def measure(self, cold, reps, graphs=True):
        """Cold medians (t_*_ms, with p10/p90 in t_*) and warm averages
        (warm_*_ms) of the three paths, the stand-alone compaction and the
        sparse path's main kernel alone."""
        torch = self.torch
        res = {}
        fns = {"auto": self.conv("auto"), "sparse": self.conv("sparse"), "dense": self.conv("dense"),
               "compact": self.compact(), "sparse_kernel": self.sparse_kernel()}
        if graphs:
            fns = {name: graph_of(torch, fn).replay for name, fn in fns.items()}
        for name, ms in cold.times_interleaved(fns, reps).items():
            st = stats(ms)
            res["t_%s_ms" % name] = st["median"]
            res["t_%s" % name] = st
        for name, fn in fns.items():
            res["warm_%s_ms" % name] = round(event_time_ms(torch, fn, max(20, reps)), 6)
        return res

    def measure_dw(self, cold, reps, graphs=True):
        """The weight gradient (training) on this layer's input with a random
        output gradient: the zero-skipping kernel (isc_conv2d_dw, graph
        replayed) against torch's GPU weight gradient of the same
        convolution (the vendor library, eager), when the kernel takes the
        shape."""
        torch, isc, L = self.torch, self.isc, self.layer
        try:
            nbytes = isc.isc_conv2d_dw_workspace_size(self.desc)
        except isc.IscError:
            return {}
        gen = torch.Generator(device="cuda")
        gen.manual_seed(self.layer.seed)
        dy = torch.randn((L.N, L.K, self.Ho, self.Wo), device="cuda", generator=gen)
        ws = torch.empty(max(nbytes, 1), dtype=torch.uint8, device="cuda")
        dw = torch.empty((L.K, L.C, L.R, L.S), device="cuda")
        fn = lambda: isc.isc_conv2d_dw(self.x, dy, L.R, L.S, L.T, L.P, out=dw, ws=ws)
        if graphs:
            fn = graph_of(torch, fn).replay
        res = {"t_dw_sparse_ms": stats(cold.times(fn, reps))["median"]}
        ref = lambda: torch.nn.grad.conv2d_weight(self.x, (L.K, L.C, L.R, L.S), dy, stride=L.T, padding=L.P)
        ref()
        res["t_dw_library_ms"] = stats(cold.times(ref, reps))["median"]
        res["speedup_dw_vs_library"] = round(res["t_dw_library_ms"] / res["t_dw_sparse_ms"], 3)
        res["dw_tflops_nonzero"] = round(2 * self.nz_macs / (res["t_dw_sparse_ms"] * 1e-3) / 1e12, 3)
        res["dw_tflops_dense_equiv"] = round(self.flops / (res["t_dw_sparse_ms"] * 1e-3) / 1e12, 3)
        del dy, ws, dw
        return res

    def measure_library(self, cold, reps, t_sparse_ms):
        """The vendor library's forward convolution of the same layer (torch's
        GPU conv2d in fp32, TF32 off, eager), a second dense reference beside
        this library's own dense path: cold median and warm average."""
        torch, L = self.torch, self.layer
        torch.backends.cudnn.allow_tf32 = False
        torch.backends.cuda.matmul.allow_tf32 = False
        fn = lambda: torch.nn.functional.conv2d(self.x, self.w, stride=L.T, padding=L.P)
        fn()  # the library's algorithm search, outside every timing
        st = stats(cold.times(fn, reps))
        return {"t_library_ms": st["median"], "t_library": st,
                "warm_library_ms": round(event_time_ms(torch, fn, max(20, reps)), 6),
                "speedup_sparse_vs_library": round(st["median"] / t_sparse_ms, 3)}

    def summary(self, res):
        f, nzm = self.flops, self.nz_macs
        L = self.layer
        out = {
            "workload": L.name, "N": L.N, "C": L.C, "H": L.H, "W": L.W, "K": L.K, "R": L.R,
            "S": L.S, "stride": L.T, "pad": L.P, "target_sparsity": L.sparsity,
            "measured_sparsity": round(self.sparsity, 6), "clustered": L.clustered,
            "dense_gflop": round(f / 1e9, 4), "nonzero_macs": nzm,
        }
        for k, v in res.items():
            out[k] = round(v, 6) if isinstance(v, float) else v
        for path in ("auto", "sparse", "dense"):
            out["tflops_%s" % path] = round(f / (res["t_%s_ms" % path] * 1e-3) / 1e12, 3)
        out["nonzero_mac_per_s_auto"] = nzm / (res["t_auto_ms"] * 1e-3)
        out["speedup_auto_vs_dense"] = round(res["t_dense_ms"] / res["t_auto_ms"], 3)
        # AUTO's time over the faster of the two forced paths (1.0: the
        # dispatcher chose the faster path at no cost)
        out["auto_vs_best"] = round(res["t_auto_ms"] / min(res["t_sparse_ms"], res["t_dense_ms"]), 3)
        out["speedup_sparse_vs_dense"] = round(res["t_dense_ms"] / res["t_sparse_ms"], 3)
        out["sparse_kernel_tflops_nonzero"] = round(2 * nzm / (res["t_sparse_kernel_ms"] * 1e-3) / 1e12, 3)
        out["sparse_kernel_frac_valu_peak"] = round(out["sparse_kernel_tflops_nonzero"] / VALU_F32_PEAK_TFLOPS, 4)
        out["dense_frac_mfma_peak"] = round(f / (res["t_dense_ms"] * 1e-3) / 1e12 / MFMA_F32_PEAK_TFLOPS, 4)
        return out


class ChainRun:
    """conv3 -> ReLU -> conv4 -> ReLU -> conv5 (the layer-chain workload):
    the rectifier fused into each layer's epilogue, each layer deciding from
    the census its predecessor wrote, filters repacked once (as an inference
    engine holds them); against the same chain with separate launches
    (isc_conv2d, which counts its input and repacks its filter, then a ReLU
    pass) and against the dense path with the fused rectifier."""

    def __init__(self, torch, isc, workload):
        self.torch, self.isc, self.workload = torch, isc, workload
        x0, ws = workloads.make_chain(workload)
        self.x0 = torch.from_numpy(x0).cuda()
        self.w = [torch.from_numpy(w).cuda() for w in ws]
        self.wt = [isc.isc_repack_filter(w) for w in self.w]
        self.layers = workload.layers
        self.descs, self.ys, self.census, self.ws = [], [], [], []
        x_shape = x0.shape
        for L in self.layers:
            d = isc.make_desc(*x_shape, L.K, L.R, L.S, L.T, L.P)
            ho, wo = isc.isc_out_shape(d)
            self.descs.append(d)
            self.ys.append(torch.empty((x_shape[0], L.K, ho, wo), device="cuda"))
            self.census.append(isc.census(d))
            self.ws.append({p: isc.workspace(d, p) for p in ("auto", "dense")})
            x_shape = (x_shape[0], L.K, ho, wo)
        torch.cuda.synchronize()

    def fused(self):
        isc, L = self.isc, self.layers

        def run():
            x, xc = self.x0, None
            for i in range(len(L)):
                isc.isc_conv2d_relu(x, self.w[i], L[i].T, L[i].P, path="auto", x_census=xc, wt=self.wt[i],
                                    y_census=self.census[i], out=self.ys[i], ws=self.ws[i]["auto"])
                x, xc = self.ys[i], self.census[i]
        return run

    def separate(self):
        isc, L, torch = self.isc, self.layers, self.torch

        def run():
            x = self.x0
            for i in range(len(L)):
                isc.isc_conv2d(x, self.w[i], L[i].T, L[i].P, path="auto", out=self.ys[i], ws=self.ws[i]["auto"])
                torch.relu_(self.ys[i])
                x = self.ys[i]
        return run

    def dense(self):
        isc, L = self.isc, self.layers

        def run():
            x = self.x0
            for i in range(len(L)):
                isc.isc_conv2d_relu(x, self.w[i], L[i].T, L[i].P, path="dense", out=self.ys[i],
                                    ws=self.ws[i]["dense"])
                x = self.ys[i]
        return run

    def measure(self, cold, reps, graphs=True):
        torch = self.torch
        res = {}
        fns = {name: getattr(self, name)() for name in ("fused", "separate", "dense")}
        if graphs:
            fns = {name: graph_of(torch, fn).replay for name, fn in fns.items()}
        for name, ms in cold.times_interleaved(fns, reps).items():
            st = stats(ms)
            res["t_chain_%s_ms" % name] = st["median"]
            res["t_chain_%s" % name] = st
        for name, fn in fns.items():
            res["warm_chain_%s_ms" % name] = round(event_time_ms(torch, fn, max(20, reps)), 6)
        # the activations of the fused run (the last one timed wrote the
        # dense run's outputs, equal up to rounding): run it once more
        self.fused()()
        torch.cuda.synchronize()
        xs = [self.x0] + self.ys[:-1]
        res["input_sparsity"] = [round(1.0 - int(torch.count_nonzero(x).item()) / x.numel(), 6) for x in xs]
        res["paths"] = []
        for i, d in enumerate(self.descs):
            _, path = self.isc.isc_decision(d, self.ws[i]["auto"])
            res["paths"].append(path)
        flops = 0.0
        x_shape = tuple(self.x0.shape)
        for L in self.layers:
            d = self.isc.make_desc(*x_shape, L.K, L.R, L.S, L.T, L.P)
            ho, wo = self.isc.isc_out_shape(d)
            flops += dense_flops(L.with_(N=x_shape[0]), ho, wo)
            x_shape = (x_shape[0], L.K, ho, wo)
        res["dense_gflop"] = round(flops / 1e9, 4)
        res["tflops_chain_fused"] = round(flops / (res["t_chain_fused_ms"] * 1e-3) / 1e12, 3)
        res["speedup_fused_vs_separate"] = round(res["t_chain_separate_ms"] / res["t_chain_fused_ms"], 3)
        res["speedup_fused_vs_dense"] = round(res["t_chain_dense_ms"] / res["t_chain_fused_ms"], 3)
        return res


# Tab. 3 of the paper: one image on one core of a Xeon E5-2630 v4 at 2.2 GHz,
# ms for Caffe's GEMM convolution (MKL) and for ISC, and the speedup printed,
# per Tab. 2 layer.
PAPER_TAB3_MS = {
    "tab2_lenet_conv2_n1": (0.854, 0.123, 6.96), "tab2_alexnetc_conv3_n1": (0.329, 0.122, 2.69),
    "tab2_alexneti_conv4_n1": (4.874, 1.660, 2.94), "tab2_inception4a_1_n1": (1.795, 1.292, 1.39),
    "tab2_inception4a_2_n1": (0.943, 0.558, 1.69), "tab2_inception4e_3_n1": (7.602, 4.782, 1.59),
    "tab2_inception5a_1_n1": (1.912, 0.645, 2.97), "tab2_inception5a_2_n1": (0.742, 0.258, 2.87),
    "tab2_inception5b_3_n1": (4.410, 0.931, 4.74), "tab2_inception5b_5_n1": (1.560, 0.220, 7.11),
}


def host_cpu_rows(budget_s: float = 1.0) -> list:
    """The paper's CPU comparison on this machine's host: for every Tab. 2
    layer at one image, ISC on one core (the host library: steps 1-3,
    AVX2 FMAs over K, filter repacked beforehand as an inference engine holds
    it) against the GEMM convolution on one core (im2col, then a BLAS sgemm
    limited to one thread), and the oracle (fp64 direct convolution) on one
    thread; medians over repeats filling about budget_s per method."""
    import oracle
    from paper_1704_07724_amd import host
    from threadpoolctl import threadpool_limits

    def med_ms(fn):
        fn()
        times, t_end = [], time.perf_counter() + budget_s
        while time.perf_counter() < t_end or len(times) < 3:
            t0 = time.perf_counter()
            fn()
            times.append((time.perf_counter() - t0) * 1e3)
        return float(np.median(times)), len(times)

    rows = []
    saved = oracle.threads()
    oracle.set_threads(1)
    try:
        with threadpool_limits(1):
            for layer in workloads.WORKLOADS["paper_tab2_n1"].layers:
                x, w = workloads.make_inputs(layer)
                T, P = layer.T, layer.P
                Ho, Wo = host.out_shape(layer.H, layer.W, layer.R, layer.S, T, P)
                wt = host.repack(w)
                wm = np.ascontiguousarray(w.reshape(layer.K, -1))
                y = np.empty((1, layer.K, Ho, Wo), np.float32)
                yg = np.empty((layer.K, Ho * Wo), np.float32)

                def gemm():
                    np.matmul(wm, host.im2col(x[0], layer.R, layer.S, T, P), out=yg)

                t_isc, n_isc = med_ms(lambda: host.conv2d(x, wt, T, P, threads=1, out=y))
                t_gemm, n_gemm = med_ms(gemm)
                t_oracle, _ = med_ms(lambda: oracle.conv2d_f64(x, w, T, P))
                err = float(np.max(np.abs(yg.reshape(y.shape) - y)))
                paper = PAPER_TAB3_MS.get(layer.name)
                rows.append({"layer": layer.name, "sparsity": round(float(1.0 - np.count_nonzero(x) / x.size), 4),
                             "t_isc_ms": round(t_isc, 4), "t_gemm_ms": round(t_gemm, 4),
                             "t_oracle_ms": round(t_oracle, 4), "speedup_isc_vs_gemm": round(t_gemm / t_isc, 3),
                             "max_abs_isc_minus_gemm": err, "reps": [n_isc, n_gemm],
                             "paper_gemm_ms": paper[0] if paper else None, "paper_isc_ms": paper[1] if paper else None,
                             "paper_speedup": paper[2] if paper else None})
                r = rows[-1]
                print("# host %s: ISC %.3f ms, GEMM %.3f ms (%.2fx; paper %.2fx), oracle %.3f ms" % (
                    layer.name, t_isc, t_gemm, r["speedup_isc_vs_gemm"], r["paper_speedup"] or 0, t_oracle),
                    file=sys.stderr, flush=True)
    finally:
        oracle.set_threads(saved)
    return rows


def cpu_baseline(layer, budget_s=10.0):
    """The oracle (fp64 direct convolution) on the headline workload, timed on
    this host: with all its threads, repeated over the whole batch (or the
    first n images when one pass is longer than budget_s) until about budget_s
    seconds have passed; and with one thread on a few images."""
    import oracle
    x, w = workloads.make_inputs(layer)
    all_threads = oracle.threads()

    def rate(n, min_s):
        oracle.conv2d_f64(x[:1], w, layer.T, layer.P)  # warm
        reps, t0 = 0, time.perf_counter()
        while True:
            out = oracle.conv2d_f64(x[:n], w, layer.T, layer.P)
            reps += 1
            dt = time.perf_counter() - t0
            if dt >= min_s:
                break
        Ho, Wo = out.shape[2], out.shape[3]
        flops = 2.0 * n * layer.K * layer.C * layer.R * layer.S * Ho * Wo
        return flops * reps / dt / 1e12, reps, dt

    t0 = time.perf_counter()
    oracle.conv2d_f64(x[:1], w, layer.T, layer.P)
    t1 = time.perf_counter() - t0
    n = int(max(1, min(layer.N, budget_s / max(t1, 1e-6))))
    value, reps, dt = rate(n, budget_s)
    oracle.set_threads(1)
    try:
        n1 = int(max(1, min(layer.N, 1.0 / max(t1 * all_threads, 1e-6))))
        value1, reps1, dt1 = rate(n1, 1.0)
    finally:
        oracle.set_threads(all_threads)
    return {"value": round(value, 6), "unit": "TFLOP/s", "cores": all_threads, "kind": "oracle",
            "sample": "%d x images 0..%d of %s (N=%d, sparsity %g), fp64 direct convolution over "
                      "%d threads, %.2f s; dense-equivalent flops" % (
                          reps, n - 1, layer.name, layer.N, layer.sparsity, all_threads, dt),
            "one_thread": {"value": round(value1, 6), "unit": "TFLOP/s", "cores": 1,
                           "sample": "%d x images 0..%d, %.2f s" % (reps1, n1 - 1, dt1)},
            "cpu_model": _cpu_model()}


CSRC = os.path.join(ROOT, "paper_1704_07724_amd", "csrc")
# the sources of each sparse kernel (a counter summary holds only while they hash the same)
KERNEL_SOURCES = {
    "fused": ("sparse_fused.hpp", "sparse_fused.hip", "sparse_tile.hpp", "isc_internal.hpp"),
    "fused_reg": ("sparse_fused.hpp", "sparse_fused.hip", "sparse_tile.hpp", "isc_internal.hpp"),
    "fused_ring": ("sparse_fring.hpp", "sparse_fring.hip", "sparse_tile.hpp", "isc_internal.hpp"),
}


def counters_file(workload: str) -> str:
    return os.path.join(ROOT, "profiles", "%s_hbm_counters.md" % workload)


def sparse_source_hash(kernel: str) -> str:
    """First 16 hex digits of the SHA-256 of a sparse kernel's sources,
    concatenated in KERNEL_SOURCES order."""
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES.get(kernel, ()):
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def kernel_symbol(isc, desc, R: int) -> str:
    """The sparse path's main kernel as the kernel trace names it, with its
    tile (the on-the-fly kernels; the plan's kernel name otherwise)."""
    p = isc.isc_sparse_plan(desc)
    k = p["kernel"]
    if k == "fused_ring":
        return "sparse_conv_fring_kernel<%d, %d, %d, %d, %d>" % (R, p["maps_per_lane"], p["rows"], p["cols"],
                                                                p["waves"])
    if k == "fused_reg":
        return "sparse_conv_fused_reg_kernel<%d, %d, %d, ...>" % (R, p["rows"], p["cols"])
    if k == "fused":
        return "sparse_conv_fused_kernel<%d, %d, %d, ...>" % (R, p["rows"], p["cols"])
    return "sparse kernel %s" % k


def counted_traffic(workload: str, kernel: str):
    """HBM bytes per launch of the sparse kernel from the committed counter
    summary of the workload (FETCH_SIZE and WRITE_SIZE scaled by a copy
    kernel), or None when the kernel's sources have changed since the
    counters were taken."""
    import re
    path = counters_file(workload)
    try:
        text = open(path).read()
    except OSError:
        return None
    m = re.search(r"^traffic_bytes_per_launch (\S+): read=(\d+) write=(\d+) source_sha256=([0-9a-f]+)",
                  text, re.M)
    if not m or m.group(4) != sparse_source_hash(kernel):
        return None
    return {"kernel": m.group(1), "read_bytes": int(m.group(2)), "write_bytes": int(m.group(3)),
            "bytes": int(m.group(2)) + int(m.group(3)), "source": os.path.relpath(path, ROOT)}


def algorithmic_bytes(run) -> dict:
    """Bytes each kernel of the path must move at least once, per launch:
    the AUTO step's count-and-repack kernel reads the input and the filter and
    writes the repacked filter (and, on shapes the on-the-fly kernels do not
    take, the compaction writes the lists); the sparse kernel reads the input
    and the repacked filter and writes the output (over lists: lists, row
    offsets and repacked filter); the dense GEMM reads the input and the
    filter and writes the output."""
    L = run.layer
    planes = L.N * L.C
    row_ptr = planes * (L.H + 1) * 4
    x_bytes = run.x_host.size * 4
    y_bytes = L.N * L.K * run.Ho * run.Wo * 4
    w_bytes = L.K * L.C * L.R * L.S * 4
    kp = (L.K + 63) // 64 * 64
    wt_bytes = L.C * L.R * L.S * kp * 4
    if run.kernel in ("fused", "fused_reg", "fused_ring"):   # reads x and the repacked filter once, writes y
        sparse = x_bytes + wt_bytes + y_bytes
        prep = x_bytes + w_bytes + wt_bytes
    else:                                        # lists, row offsets, repacked filter; writes y
        sparse = run.nnz * 8 + row_ptr + wt_bytes + y_bytes
        prep = x_bytes + run.nnz * 8 + row_ptr + w_bytes + wt_bytes
    return {
        "count_repack": prep,
        "compact": x_bytes + run.nnz * 8 + row_ptr,
        "sparse_kernel": sparse,
        "dense_gemm": x_bytes + w_bytes + y_bytes,
    }


def probe(torch, isc, layer, n):
    """Short eager program for counter runs: a copy kernel moving a known
    number of bytes (the scale of the HBM counters), then n launches each of
    the sparse kernel alone, the stand-alone compaction, the whole AUTO step
    (count and repack, sparse kernel, the dense kernel that exits on the
    decision) and the dense path, each launch after the 512 MiB cache-evicting
    write (so the counters see cold traffic)."""
    run = LayerRun(torch, isc, layer)
    cold = ColdTimer(torch)
    src = torch.ones(64 << 20, dtype=torch.float32, device="cuda")  # 256 MiB
    dst = torch.empty_like(src)
    steps = [("copy", lambda: torch.mul(src, 1.0, out=dst)), ("sparse_kernel", run.sparse_kernel()),
             ("compact", run.compact()), ("auto", run.conv("auto")), ("dense", run.conv("dense"))]
    for name, fn in steps:
        for _ in range(n):
            cold.flush()
            fn()
        torch.cuda.synchronize()
        print("# probe %s x%d done" % (name, n), file=sys.stderr, flush=True)
    alg = algorithmic_bytes(run)
    alg["copy"] = {"read": src.numel() * 4, "write": dst.numel() * 4}
    print(json.dumps({"probe": layer.name, "kernel": run.kernel, "launches_each": n, "nnz": run.nnz,
                      "nonzero_macs": run.nz_macs, "algorithmic_bytes": alg,
                      "source_sha256": sparse_source_hash(run.kernel)}), flush=True)


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def sweep_point(torch, isc, cold, layer, reps, graphs, run=None):
    """One point of a sparsity sweep: cold medians of the three paths and of
    the sparse kernel alone, rates and roofline fractions."""
    run = run or LayerRun(torch, isc, layer)
    sm = run.summary(run.measure(cold, reps, graphs))
    keep = ("target_sparsity", "measured_sparsity", "t_auto_ms", "t_sparse_ms", "t_dense_ms",
            "t_compact_ms", "t_sparse_kernel_ms", "warm_auto_ms", "warm_sparse_kernel_ms", "tflops_auto",
            "tflops_sparse", "tflops_dense", "nonzero_mac_per_s_auto", "speedup_auto_vs_dense", "auto_vs_best",
            "speedup_sparse_vs_dense", "sparse_kernel_tflops_nonzero", "sparse_kernel_frac_valu_peak",
            "dense_frac_mfma_peak")
    out = {k: sm[k] for k in keep}
    _, out["auto_path"] = isc.isc_decision(run.desc, run.ws["auto"])
    out["sparse_kernel"] = run.kernel
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[1])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-graph", action="store_true", help="launch eagerly instead of graph replay")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--all", action="store_true", help="also measure every workload layer")
    ap.add_argument("--out", default=None, help="JSONL file for --all rows")
    ap.add_argument("--workload", default="alexnet_conv2", help="headline workload (a workloads.py layer name)")
    ap.add_argument("--host-cpu", action="store_true",
                    help="only the paper's CPU comparison on the host: ISC against im2col + BLAS "
                         "on one core for every Tab. 2 layer at one image (no GPU needed)")
    ap.add_argument("--probe", type=int, default=0, metavar="N",
                    help="only launch each kernel of the headline layer N times, eagerly, after "
                         "a copy kernel of known size, and print their algorithmic bytes "
                         "(a short program for hardware-counter runs)")
    args = ap.parse_args()

    if args.host_cpu:
        rows = host_cpu_rows()
        cpu = _cpu_model()
        for r in rows:
            r["cpu"] = cpu
        if args.out:
            with open(args.out, "a") as fh:
                for r in rows:
                    fh.write(json.dumps(r) + "\n")
        print(json.dumps({"host_cpu": rows}))
        return

    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(the convolution would shard by batch; see the design notes).", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_1704_07724_amd as isc
    isc.lib()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)

    layers = {l.name: l for wl in workloads.WORKLOADS.values() for l in wl.layers}
    head_layer = layers[args.workload]
    if args.probe:
        probe(torch, isc, head_layer, args.probe)
        return
    graphs = not args.no_graph
    cold = ColdTimer(torch)

    # headline: whole hot path, AUTO with the library's default threshold,
    # K cold steps bracketed by synchronize; each timed by HIP events
    head = LayerRun(torch, isc, head_layer)
    step_fn = head.conv("auto")
    if graphs:
        step_fn = graph_of(torch, step_fn).replay
    cold.times(step_fn, args.warmup, warm=0)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    step_ms = cold.times(step_fn, args.steps, warm=0)
    wall_s = time.perf_counter() - t0
    st = stats(step_ms)
    ms_per_step = st["median"]
    value = head.flops / (ms_per_step * 1e-3) / 1e12
    _, head_path = isc.isc_decision(head.desc, head.ws["auto"])
    print("# headline %s: AUTO (%s) cold median %.4f ms (p10 %.4f, p90 %.4f)" % (
        head_layer.name, head_path, st["median"], st["p10"], st["p90"]), file=sys.stderr, flush=True)

    reps = max(10, args.steps)
    res = head.measure(cold, reps, graphs)
    hs = head.summary(res)
    lib = head.measure_library(cold, reps, ms_per_step)
    print("# paths: sparse %.4f dense %.4f library %.4f ms; sparse kernel %.4f ms" % (
        res["t_sparse_ms"], res["t_dense_ms"], lib["t_library_ms"], res["t_sparse_kernel_ms"]),
        file=sys.stderr, flush=True)

    # the dominant kernel: the sparse kernel alone, average of its cold launches
    t_kernel = res["t_sparse_kernel"]["mean"]
    achieved = 2.0 * head.nz_macs / (t_kernel * 1e-3) / 1e12
    traffic = counted_traffic(head_layer.name, head.kernel)
    roofline = {"bound": "alu", "kernel": kernel_symbol(isc, head.desc, head_layer.R),
                "achieved": round(achieved, 3), "peak": VALU_F32_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / VALU_F32_PEAK_TFLOPS, 4),
                "traffic": traffic["bytes"] if traffic else None, "traffic_detail": traffic,
                "per_launch": {"nonzero_macs": head.nz_macs, "flops": 2 * head.nz_macs,
                               "avg_duration_ms": round(t_kernel, 6),
                               "median_duration_ms": res["t_sparse_kernel"]["median"],
                               "warm_avg_duration_ms": res["warm_sparse_kernel_ms"]},
                "frac_vs_packed_peak": round(achieved / VALU_F32_PACKED_PEAK_TFLOPS, 4)}

    alg = algorithmic_bytes(head)
    hbm = {}
    for kern, t_key in (("compact", "t_compact_ms"), ("sparse_kernel", "t_sparse_kernel_ms")):
        gbs = alg[kern] / (res[t_key] * 1e-3) / 1e9
        hbm[kern] = {"algorithmic_bytes": alg[kern], "ms": round(res[t_key], 6),
                     "GB/s": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4)}

    sweep = []
    if not args.no_sweep:
        for layer in workloads.WORKLOADS["lenet_conv2_batch"].layers:
            pt = sweep_point(torch, isc, cold, layer, max(10, args.steps // 2), graphs)
            sweep.append(pt)
            print("# sweep %s: auto %.4f sparse %.4f dense %.4f ms (%s)" % (
                layer.name, pt["t_auto_ms"], pt["t_sparse_ms"], pt["t_dense_ms"], pt["auto_path"]),
                file=sys.stderr, flush=True)
            torch.cuda.empty_cache()

    line = {
        "metric": METRIC, "value": round(value, 4), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": head_layer.name, "N": head_layer.N, "C": head_layer.C,
                   "H": head_layer.H, "W": head_layer.W, "K": head_layer.K, "R": head_layer.R,
                   "S": head_layer.S, "stride": head_layer.T, "pad": head_layer.P,
                   "sparsity": head_layer.sparsity, "path": "auto",
                   "threshold": "per-shape crossover" if isc.default_threshold() < 0 else isc.default_threshold(),
                   "launch": "eager" if not graphs else "hip_graph", "caches": "cold (512 MiB flush per step)"},
        "step_ms": st,
        "wall_s_timed_steps": round(wall_s, 4),
        "auto_path": head_path,
        "speedup_vs_dense": round(res["t_dense_ms"] / ms_per_step, 3),
        "speedup_vs_library": round(lib["t_library_ms"] / ms_per_step, 3),
        "nonzero_mac_per_s": head.nz_macs / (ms_per_step * 1e-3),
        "measured_sparsity": hs["measured_sparsity"],
        "dense_path_tflops": hs["tflops_dense"],
        "dense_frac_mfma_peak": hs["dense_frac_mfma_peak"],
        "library_conv2d_ms": lib["t_library_ms"],
        "warm": {"auto_ms": res["warm_auto_ms"], "sparse_ms": res["warm_sparse_ms"],
                 "dense_ms": res["warm_dense_ms"], "library_ms": lib["warm_library_ms"],
                 "tflops_auto": round(head.flops / (res["warm_auto_ms"] * 1e-3) / 1e12, 3)},
        "roofline": roofline,
        "hbm": hbm,
        "timings_ms": {k: hs[k] for k in hs if k.startswith("t_") and isinstance(hs[k], float)},
        "sweep": sweep,
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(head_layer)

    if args.all:
        rows = []
        for wl in workloads.WORKLOADS.values():
            if wl.name == "alexnet_chain345":
                chain = ChainRun(torch, isc, wl)
                r = chain.measure(cold, max(10, args.steps // 2), graphs)
                r["workload"] = wl.name
                rows.append(r)
                print("# %s: fused %.4f ms separate %.4f dense %.4f (fused vs separate %.2fx, vs dense %.2fx) "
                      "input sparsity %s paths %s" % (
                          wl.name, r["t_chain_fused_ms"], r["t_chain_separate_ms"], r["t_chain_dense_ms"],
                          r["speedup_fused_vs_separate"], r["speedup_fused_vs_dense"], r["input_sparsity"],
                          r["paths"]), file=sys.stderr, flush=True)
                del chain
                torch.cuda.empty_cache()
                continue
            for layer in wl.layers:
                if wl.name == "lenet_conv2_batch":
                    continue
                run = LayerRun(torch, isc, layer)
                s = run.summary(run.measure(cold, max(10, args.steps // 2), graphs))
                _, s["auto_path"] = isc.isc_decision(run.desc, run.ws["auto"])
                s.update(run.measure_dw(cold, max(10, args.steps // 2), graphs))
                s.update(run.measure_library(cold, max(10, args.steps // 2), s["t_sparse_ms"]))
                rows.append(s)
                dws = (" | dw sparse %.4f ms library %.4f (%.2fx)" % (
                    s["t_dw_sparse_ms"], s["t_dw_library_ms"], s["speedup_dw_vs_library"])
                       if "t_dw_sparse_ms" in s else "")
                print("# %s: auto %.4f ms (%s, %.3f of best) sparse %.4f dense %.4f speedup %.2fx library %.4f (%.2fx)%s" % (
                    layer.name, s["t_auto_ms"], s["auto_path"], s["auto_vs_best"], s["t_sparse_ms"], s["t_dense_ms"],
                    s["speedup_sparse_vs_dense"], s["t_library_ms"], s["speedup_sparse_vs_library"], dws),
                      file=sys.stderr, flush=True)
                del run
                torch.cuda.empty_cache()
        if args.out:
            with open(args.out, "w") as f:
                for r in rows:
                    f.write(json.dumps(r) + "\n")
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
