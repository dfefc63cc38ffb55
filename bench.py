#!/usr/bin/env python3
"""Benchmark of the fused dequantize x matrix-vector product on one MI355X.

A step is one decode token's pass over every weight matrix of a workload: one
lw_matvec per matrix, except that a layer's gate and up projections (same
input, independent outputs) share one lw_matvec_multi call, as a decode step
issues them (--no-fuse: one call each). Each matrix has its own HBM buffer (the 8B Q4_K-style set
is 4.2 GB, far above the 256 MB Infinity Cache, so every step streams the
weights from HBM). Inputs are synthetic and seeded (paper_2605_20706_amd.synth)
and resident in HBM before the timed region starts.

Printed (one JSON line): HBM GB/s from algorithmic bytes (packed W + x + y),
its fraction of the 8 TB/s peak, the equivalent decode tokens/s, a roofline
object for the kernel that takes most of a step (from HIP events around
back-to-back launches of each matrix shape; lw_kernel_name says which kernel
each shape runs), and the CPU oracle timed on a bounded sample of the same
workload on this host.

Usage: python bench.py [--workload q4_k_llama8b] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

from paper_2605_20706_amd import binding, layout, synth  # noqa: E402

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFS = 2500.0  # dense bf16 matrix-core peak of MI355X
MFMA_FP4_PEAK_TFS = 10100.0  # dense fp4 / fp6 matrix-core peak of MI355X
# the fp4 matrix-core path's per-output bound (mxfp4 prefill through lw_matvec_ws)
FP4_SPLIT, FP4_MFMA = 2.0 ** -16, 2.0 ** -11
CSRC = os.path.join(ROOT, "paper_2605_20706_amd", "csrc")
# Kernel nodes one captured HIP graph may hold. A 1-bit benchmark process
# once ended in a segmentation fault while its graphs held 90 k and 180 k
# kernel nodes (512 tokens at 128 launches per call); the cause was not
# isolated, so captures stay far below that: the timed steps are split over
# several graphs (replayed back to back inside the timed region), and a step
# that alone exceeds the budget runs eagerly.
MAX_GRAPH_NODES = 16384
# Rounding bound of the factored evaluations (see lw.h): 2^-17 per unit of
# the term mass F on top of 1e-4 per unit of A.
C_FACTORED = 2.0 ** -17
F32_BOUND = 1e-4
MFMA_KERNELS = ("fewtok_kernel", "multitok_kernel", "multitok_pk_kernel", "skinny_kernel", "gemm_kernel",
                "gemm32_kernel")
METRIC_ATTN = "decode attention over a quantized KV cache, HBM GB/s of K and V read per decode step"
# Llama-3-8B attention: 32 layers, 32 query heads over 8 key/value heads of 128
ATTN_MODEL = {"n_layers": 32, "n_heads": 32, "n_kv": 8, "head_dim": 128}
METRIC = "dequant-GEMV HBM GB/s (% of peak) and equiv. decode tok/s, Llama-1B/8B shapes"
METRIC_DEQUANT = "standalone dequant HBM GB/s (packed read + float32 write), Llama-1B/8B shapes"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class Workset:
    """All matrices of a workload on the GPU, their x and y buffers (or, for
    op "dequant", one float32 output per matrix), and the raw argument tuples
    of one lw_matvec (lw_dequant) per matrix."""

    def __init__(self, wl, n_tok, keep_host=0, op="matvec", rotate_bytes=2e9, fuse=True):
        import torch

        self.wl, self.n_tok, self.op = wl, n_tok, op
        self.lib = binding.library()
        mats = list(wl.matrices)
        t0 = time.time()
        self.host = {}
        self.W, self.y = [], []

        def gen(i):
            return i, synth.gen_matrix(wl, mats[i])

        with ThreadPoolExecutor(8) as ex:
            for i, Wh in ex.map(gen, range(len(mats))):
                self.W.append(torch.from_numpy(Wh).to("cuda"))
                if i < keep_host:
                    self.host[i] = Wh
        self.x = {K: torch.from_numpy(synth.gen_x(wl, K, n_tok)).to("cuda")
                  for K in sorted({m.K for m in mats})}
        self.xh = {K: v.cpu().numpy() for K, v in self.x.items()}
        self.y = [torch.empty((n_tok, m.M), dtype=torch.float32, device="cuda") for m in mats]
        # A workload smaller than rotate_bytes gets identical copies of its
        # weights, and consecutive steps (and the per-shape phase) rotate
        # through them, so no launch finds its weights in the 256 MB
        # Infinity Cache or L2 from a previous launch.
        packed = sum(w.numel() for w in self.W)
        self.reps = max(1, int(-(-rotate_bytes // packed)))
        for _ in range(1, self.reps):
            self.W.extend(w.clone() for w in self.W[:len(mats)])
        torch.cuda.synchronize()
        log("workload %s: %d matrices, %.3f GB packed (%d copies), generated+uploaded in %.1fs"
            % (wl.key, len(mats), packed / 1e9, self.reps, time.time() - t0))
        self.mats = mats
        n = len(mats)
        if op == "dequant":
            self.out = [torch.empty(m.M * m.K, dtype=torch.float32, device="cuda") for m in mats]
            self.args = [(wl.fmt, self.W[r * n + i].data_ptr(), self.out[i].data_ptr(), m.M * m.K)
                         for r in range(self.reps) for i, m in enumerate(mats)]
            # packed read + float32 write
            self.alg_bytes = [layout.BYTES_PER_WEIGHT[wl.fmt] * m.M * m.K + 4.0 * m.M * m.K for m in mats]
            self.flops = [0.0 for _ in mats]
        else:
            self.args = [(wl.fmt, self.W[r * n + i].data_ptr(), self.x[m.K].data_ptr(), self.y[i].data_ptr(),
                          m.M, m.K, n_tok) for r in range(self.reps) for i, m in enumerate(mats)]
            self.alg_bytes = [synth.algorithmic_bytes(wl.fmt, m.M, m.K, n_tok) for m in mats]
            self.flops = [2.0 * m.M * m.K * n_tok for m in mats]
        # Calls whose fastest path needs a workspace (lw_matvec_workspace_bytes
        # > 0: mxfp4 prefill on the fp4 matrix cores) go through lw_matvec_ws
        # with one workspace shared by the step's calls (they run in order on
        # one stream), one call per matrix.
        need = [binding.matvec_workspace_bytes(wl.fmt, m.M, m.K, n_tok) for m in mats] if op == "matvec" else [0]
        self.use_ws = max(need) > 0
        self.wsbuf = torch.empty(max(need), dtype=torch.uint8, device="cuda") if self.use_ws else None
        if self.use_ws:
            fuse = False
        # Calls of a step: one per matrix, except that a layer's gate and up
        # projections (same input, independent outputs) are one
        # lw_matvec_multi call when fuse is set (op "matvec" only).
        self.groups = []
        for i, m in enumerate(mats):
            prev = self.groups[-1] if self.groups else None
            if (fuse and op == "matvec" and m.name == "up" and prev and len(prev) == 1
                    and mats[prev[0]].name == "gate" and mats[prev[0]].layer == m.layer and mats[prev[0]].K == m.K):
                self.groups[-1] = (prev[0], i)
            else:
                self.groups.append((i,))
        self._keep = []
        self.calls = []  # (kind "one" / "multi" / "ws", args) per weight copy and group
        for r in range(self.reps):
            for grp in self.groups:
                if self.use_ws:
                    self.calls.append(("ws", self.args[r * n + grp[0]]
                                       + (self.wsbuf.data_ptr(), self.wsbuf.numel())))
                elif len(grp) == 1 or op != "matvec":
                    self.calls.append(("one", self.args[r * n + grp[0]]))
                else:
                    K = mats[grp[0]].K
                    arr = binding.multi_args([self.W[r * n + i].data_ptr() for i in grp],
                                             [self.y[i].data_ptr() for i in grp], [mats[i].M for i in grp])
                    self._keep.append(arr)
                    self.calls.append(("multi", (wl.fmt, len(grp)) + arr + (self.x[K].data_ptr(), K, n_tok)))
        self.fuse_used = any(len(g) > 1 for g in self.groups)
        # kernel launches per call: a multi call is one launch where the
        # library fuses it (lw_kernel_name_multi then names another kernel
        # than the first matrix's lw_matvec), else one launch per matrix
        self.call_launches = []
        for grp in self.groups:
            fused = False
            if len(grp) > 1:
                Ms = [mats[i].M for i in grp]
                K = mats[grp[0]].K
                fused = (binding.kernel_name_multi(wl.fmt, Ms, K, n_tok)
                         != binding.kernel_name(wl.fmt, Ms[0], K, n_tok))
            self.call_launches.append(1 if fused or len(grp) == 1 else len(grp))
        # kernel launches (graph nodes) per call, from the library's own count
        self.call_nodes = []
        for grp in self.groups:
            ms = [mats[i] for i in grp]
            if op == "dequant":
                self.call_nodes.append(1)
            elif self.use_ws:
                self.call_nodes.append(binding.launch_count_ws(wl.fmt, ms[0].M, ms[0].K, n_tok))
            elif len(grp) == 1:
                self.call_nodes.append(binding.launch_count(wl.fmt, ms[0].M, ms[0].K, n_tok))
            else:
                self.call_nodes.append(binding.launch_count_multi(wl.fmt, [m.M for m in ms], ms[0].K, n_tok))
        self.step_nodes = sum(self.call_nodes)
        self.call_bytes = [sum(self.alg_bytes[i] for i in grp) for grp in self.groups]
        self.call_flops = [sum(self.flops[i] for i in grp) for grp in self.groups]

    def step(self, stream, idx=None, rep=0):
        """The calls of weight copy `rep`, or the calls `idx` (indices over all
        copies). lw_dequant runs on the null stream: op "dequant" is timed
        eagerly on it."""
        ng = len(self.groups)
        calls = range(rep * ng, rep * ng + ng) if idx is None else idx
        if self.op == "dequant":
            f = self.lib.lw_dequant
            for i in calls:
                rc = f(*self.calls[i][1])
                if rc != 0:
                    raise binding.LwError(rc, "lw_dequant")
            return
        fns = {"one": self.lib.lw_matvec, "multi": self.lib.lw_matvec_multi, "ws": self.lib.lw_matvec_ws}
        for i in calls:
            kind, a = self.calls[i]
            rc = fns[kind](*a, stream)
            if rc != 0:
                raise binding.LwError(rc, "lw_matvec_" + kind)

    def kernel_names(self):
        """The kernel each call of a step launches (lw_kernel_name /
        lw_kernel_name_multi for op matvec)."""
        if self.op == "dequant":
            return ["dequant_kernel<%d>" % self.wl.fmt for _ in self.groups]
        out = []
        for grp in self.groups:
            ms = [self.mats[i] for i in grp]
            if self.use_ws:
                out.append(binding.kernel_name_ws(self.wl.fmt, ms[0].M, ms[0].K, self.n_tok))
            elif len(grp) == 1:
                out.append(binding.kernel_name(self.wl.fmt, ms[0].M, ms[0].K, self.n_tok))
            else:
                out.append(binding.kernel_name_multi(self.wl.fmt, [m.M for m in ms], ms[0].K, self.n_tok))
        return out

    def call_label(self, j):
        ms = [self.mats[i] for i in self.groups[j]]
        return "+".join(m.name for m in ms) + " " + "+".join("%dx%d" % (m.M, m.K) for m in ms)

    def shapes(self):
        """Call indices (over all weight copies) grouped by 'names MxK', in
        first-seen order."""
        groups = {}
        ng = len(self.groups)
        for r in range(self.reps):
            for j in range(ng):
                groups.setdefault(self.call_label(j), []).append(r * ng + j)
        return groups


def graph_chunks(first, count, nodes_per_step, budget=MAX_GRAPH_NODES):
    """Steps [first, first + count) as consecutive (first, count) pieces of
    at most `budget` kernel nodes each, or None when one step alone exceeds
    the budget (then the steps run eagerly)."""
    if count <= 0:
        return []
    if nodes_per_step > budget:
        return None
    per = max(1, budget // max(1, nodes_per_step))
    return [(f, min(per, first + count - f)) for f in range(first, first + count, per)]


def run_gpu(ws, steps, warmup, mode):
    import ctypes

    import torch

    # ---- whole-step throughput (timed region) ----
    # Step i runs on weight copy i mod ws.reps. In graph mode the warm-up
    # steps are one graph and the timed steps another, so that a step of a
    # few short launches is not paced by the host's graph launches.
    def steps_on(stream, first, count):
        for i in range(first, first + count):
            ws.step(ctypes.c_void_p(stream), rep=i % ws.reps)

    if mode == "graph" and (graph_chunks(0, 1, ws.step_nodes) is None):
        log("a step of %d kernel launches exceeds the graph budget of %d nodes: eager mode"
            % (ws.step_nodes, MAX_GRAPH_NODES))
        mode = "eager"
    if mode == "graph":
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            ws.step(ctypes.c_void_p(side.cuda_stream))
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        runs = []
        for first, count in ((0, warmup), (warmup, steps)):
            gs = []
            for f, c in graph_chunks(first, count, ws.step_nodes):
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g):
                    steps_on(torch.cuda.current_stream().cuda_stream, f, c)
                gs.append(g)

            def replay(gs=gs):
                for g in gs:
                    g.replay()
            runs.append(replay)
        warm, timed = runs
    else:
        def warm():
            steps_on(torch.cuda.current_stream().cuda_stream, 0, warmup)

        def timed():
            steps_on(torch.cuda.current_stream().cuda_stream, warmup, steps)
    if warmup:
        warm()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    timed()  # exactly `steps` steps, continuing the rotation after the warm-up
    end.record()
    torch.cuda.synchronize()
    ms_per_step = start.elapsed_time(end) / steps
    # the outputs of the last timed step, for the parity check against the oracle
    y_timed = [v.cpu().numpy() for v in ws.y] if ws.op == "matvec" else None

    # ---- per-shape launch durations: 192 launches of one matrix shape back
    # to back (cycling over that shape's matrices; one graph in graph mode),
    # queued behind a short device-side sleep so that host launch latency stays
    # out of the timed span; events on the launch stream ----
    stream = torch.cuda.current_stream()
    per_shape = {}
    for key, idx in ws.shapes().items():
        # 192 launches of the shape, fewer where its calls launch several kernels
        n_seq = max(1, min(192, MAX_GRAPH_NODES // ws.call_nodes[idx[0] % len(ws.groups)]))
        seq = (idx * ((n_seq + len(idx) - 1) // len(idx)))[:max(n_seq, len(idx))]

        def sub():
            ws.step(ctypes.c_void_p(torch.cuda.current_stream().cuda_stream), seq)

        if mode == "graph":
            g2 = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g2):
                sub()
            sub_run = g2.replay
        else:
            sub_run = sub
        sub_run()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(int(2.4e6 * 5))  # ~5 ms at 2.4 GHz
        e0.record(stream)
        sub_run()
        e1.record(stream)
        torch.cuda.synchronize()
        per_shape[key] = (e0.elapsed_time(e1) / len(seq), idx)
    return ms_per_step, per_shape, y_timed, mode


KERNEL_SOURCES = {"gemv_kernel": "gemv.hip", "gemv1_kernel": "gemv.hip", "gemv1r_kernel": "gemv.hip",
                  "multitok_kernel": "multitok.hip", "multitok_pk_kernel": "multitok.hip",
                  "fewtok_kernel": "fewtok.hip", "skinny_kernel": "skinny.hip", "gemm_kernel": "prefill.hip",
                  "gemm32_kernel": "prefill.hip", "fp4mm_kernel": "fp4mm.hip",
                  "dequant_kernel": "dequant.hip"}


def source_hash(kernels):
    """sha256 over the sources of the given kernels (names as lw_kernel_name
    gives them), the shared device and host headers and the C header: a stored
    HBM traffic figure is valid only for the sources it was measured on."""
    import hashlib

    files = sorted({KERNEL_SOURCES[k.split("<")[0]] for k in kernels})
    files = [os.path.join(CSRC, f) for f in files + ["lw_device.hpp", "lw_internal.hpp"]]
    files.append(os.path.join(ROOT, "include", "lw.h"))
    h = hashlib.sha256()
    for f in files:
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def stored_traffic(workload, n_tok, kernel):
    """HBM bytes per launch of `kernel` from the calibrated rocprofv3 FETCH_SIZE
    and WRITE_SIZE summary in profiles/, or None when there is none for these
    sources (the hash covers the sources of every kernel the summary lists)."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic_%s_nt%d.txt" % (workload, n_tok))
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as fh:
        for line in fh:
            if "=" in line and not line.startswith((" ", "#", "|")):
                k, v = line.strip().split("=", 1)
                vals[k.strip()] = v.strip()
    kernels = [k[len("hbm_bytes_per_launch["):-1] for k in vals if k.startswith("hbm_bytes_per_launch[")]
    if not kernels or vals.get("source_sha256") != source_hash(kernels):
        return None
    try:
        return float(vals["hbm_bytes_per_launch[%s]" % kernel])
    except (KeyError, ValueError):
        return None


def traffic_method(workload, n_tok):
    """How the stored traffic figure was taken: the counters and the
    calibration factors (a plain 1 GiB elementwise copy, confirmed by a 1 GiB
    read of the 128-bit non-temporal read kernel)."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic_%s_nt%d.txt" % (workload, n_tok))
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        for line in fh:
            if "bytes = FETCH_SIZE" in line:
                return ("rocprofv3 --pmc, one counter per run; " + line.strip("# \n")
                        + "; factors from a 1 GiB elementwise copy, confirmed by a 1 GiB 128-bit read (%s)"
                        % os.path.relpath(path, ROOT))
    return None


def ceilings(write, launch_bytes, mode, extra_bytes=()):
    """Streaming ceilings from libceiling.so in this process: GB/s of a plain
    128-bit read (write: non-temporal write, the dequantization's store form)
    over a 1 GiB buffer (one launch), and at `launch_bytes` per launch timed as
    the per-shape launches are (192 back to back at rotating offsets of that
    buffer, so no launch finds the previous one's bytes in the 256 MB Infinity
    Cache; one graph in graph mode; behind a device-side sleep; HIP events on
    the launch stream). Also returns {b: GB/s} at each size in `extra_bytes`,
    timed the same way."""
    import ctypes
    import torch

    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2605_20706_amd", "libceiling.so"))
    lib.lw_ceiling_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
    lib.lw_ceiling_write.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
    total = 1 << 30
    buf = torch.empty(total, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")

    def launches(offs, nbytes):
        s = torch.cuda.current_stream().cuda_stream
        for off in offs:
            ptr = buf.data_ptr() + off
            rc = lib.lw_ceiling_write(ptr, nbytes, s) if write else lib.lw_ceiling_read(ptr, nbytes, sink.data_ptr(), s)
            if rc != 0:
                raise RuntimeError("libceiling: code %d" % rc)

    def rate(nbytes, n, graph):
        step = (nbytes + 255) // 256 * 256
        offs = [(i * step) % (total - step + 1) // 256 * 256 for i in range(n)]
        run = lambda: launches(offs, nbytes)  # noqa: E731
        if graph:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                run()
            run = g.replay
        run()
        torch.cuda.synchronize()
        stream = torch.cuda.current_stream()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(int(2.4e6 * 5))  # ~5 ms at 2.4 GHz
        e0.record(stream)
        run()
        e1.record(stream)
        torch.cuda.synchronize()
        return nbytes * n / (e0.elapsed_time(e1) * 1e-3) / 1e9

    def clamp(b):
        return max(16, min(int(b), total) // 16 * 16)

    lb = clamp(launch_bytes)
    out = {"kind": "write" if write else "read", "GB/s_1GiB": round(rate(total, 3, False), 1),
           "launch_bytes": lb, "GB/s_at_launch_bytes": round(rate(lb, 192, mode == "graph"), 1)}
    at = {}
    for b in extra_bytes:
        cb = clamp(b)
        if cb not in at:
            at[cb] = out["GB/s_at_launch_bytes"] if cb == lb else rate(cb, 192, mode == "graph")
    return out, {b: at[clamp(b)] for b in extra_bytes}


def kernel_groups(ws, per_shape):
    """Launches of a step grouped by the kernel the library selects for them
    (lw_kernel_name / lw_kernel_name_multi), with each group's time per step
    from the per-shape launch durations: {kernel: {launches, us, bytes, flop}}."""
    names = ws.kernel_names()
    ng = len(ws.groups)
    groups = {}
    for _, (ms, idx) in per_shape.items():
        one = [i for i in idx if i < ng]  # this shape's calls in one step
        g = groups.setdefault(names[one[0]], {"launches": 0, "us": 0.0, "bytes": 0.0, "flop": 0.0})
        g["launches"] += sum(ws.call_launches[i] for i in one)
        g["us"] += ms * 1e3 * len(one)
        g["bytes"] += sum(ws.call_bytes[i] for i in one)
        g["flop"] += sum(ws.call_flops[i] for i in one)
    return names, groups


def cpu_baseline(ws, budget_s, y_timed=None):
    """The oracle on the host's cores over the first matrices of the workload
    until budget_s is used (timed: its y and A), and, for op matvec, the
    outputs of the last timed GPU step compared with the oracle on those
    matrices (untimed: y, A and the term mass F of the kernel's form)."""
    import oracle

    wl = ws.wl
    host_cpus = os.cpu_count() or 1
    # the host share of one GPU: OMP_NUM_THREADS when set, else at most 16 threads
    n_threads = int(os.environ.get("OMP_NUM_THREADS", "0")) or min(16, host_cpus)
    t_used, nbytes, nweights, done = 0.0, 0, 0, []
    threads = 0
    refs = {}
    for i, m in enumerate(ws.mats):
        if i not in ws.host:
            break
        t0 = time.perf_counter()
        if ws.op == "dequant":
            oracle.dequant(wl.fmt, ws.host[i], m.M * m.K)  # one thread
            threads = 1
        else:
            refs[i] = oracle.matvec(wl.fmt, ws.host[i], ws.xh[m.K], m.M, m.K, n_threads=n_threads)
            threads = refs[i][2]
        t_used += time.perf_counter() - t0
        nbytes += ws.alg_bytes[i]
        nweights += m.M * m.K
        done.append("%s[%d]" % (m.name, m.layer))
        if t_used >= budget_s:
            break
    gbs = nbytes / t_used / 1e9
    tok_s = ws.n_tok * gbs * 1e9 / sum(ws.alg_bytes)
    out = {"value": round(gbs, 4), "unit": "GB/s", "cores": int(threads), "host_cpus": int(host_cpus),
           "kind": "oracle", "equiv_decode_tok_s": round(tok_s, 4), "seconds": round(t_used, 2),
           "sample": "%d of %d matrices (%s), %.3g weights, same inputs; oracle = plain C, "
                     "double accumulation, one thread per row block; %d threads of %d host CPUs"
                     % (len(done), len(ws.mats), ", ".join(done[:6]) + (" ..." if len(done) > 6 else ""),
                        nweights, threads, host_cpus)}
    parity = None
    if y_timed is not None and refs:
        parity = timed_parity(ws, refs, y_timed, n_threads)
    return out, parity


def block_max_mass(oracle, fmt, W, x, M, K, rows=4096):
    """Bm[t][r] = sum_k |w_rk| * (largest |x_t| of k's 32-block), from the
    oracle's exact dequantization: the activation-split term of the fp4
    matrix-core path's bound."""
    x = np.atleast_2d(np.asarray(x, np.float64))
    xm = np.abs(x).reshape(x.shape[0], K // 32, 32).max(axis=2)
    Bm = np.empty((x.shape[0], M))
    Wd = oracle.dequant(fmt, W, M * K).reshape(M, K)
    for r0 in range(0, M, rows):
        S = np.abs(Wd[r0:r0 + rows].astype(np.float64)).reshape(-1, K // 32, 32).sum(axis=2)
        Bm[:, r0:r0 + rows] = xm @ S.T
    return Bm


def timed_parity(ws, refs, y_timed, n_threads):
    """Every output of the last timed step, for the matrices the CPU baseline
    covered, against the oracle: the float32 bound |dy| <= 1e-4 A + 2^-17 F
    per output (F the term mass of the form the call's kernel evaluates; f16
    and Q8_0 are plain sums, F = 0), the 2e-3 gate, the normwise error and
    the NMSE."""
    import oracle

    wl = ws.wl
    names = ws.kernel_names()
    kern_of = {}
    for j, grp in enumerate(ws.groups):
        for i in grp:
            kern_of[i] = names[j]
    worst = {"scaled": 0.0, "normwise": 0.0, "nmse": 0.0, "f32_bound_ratio": 0.0}
    n_out, ok, fp4 = 0, True, False
    for i, (y_ref, A, _) in refs.items():
        m = ws.mats[i]
        y = y_timed[i].astype(np.float64).reshape(y_ref.shape)
        if wl.fmt in (layout.F16, layout.Q8_0, layout.MXFP4):
            F = np.zeros_like(A)
        else:
            beta = 128 if kern_of[i].split("<")[0] in MFMA_KERNELS else 0
            _, _, F, _ = oracle.matvec_f(wl.fmt, ws.host[i], ws.xh[m.K], m.M, m.K, beta, n_threads=n_threads)
        d = np.abs(y - y_ref)
        bound = F32_BOUND * A + C_FACTORED * F
        if kern_of[i].split("<")[0] == "fp4mm_kernel":
            fp4 = True
            Bm = block_max_mass(oracle, wl.fmt, ws.host[i], ws.xh[m.K], m.M, m.K)
            bound = FP4_SPLIT * Bm + FP4_MFMA * (A + Bm / 4)
        with np.errstate(divide="ignore", invalid="ignore"):
            r = np.where(bound > 0, d / bound, np.where(d > 0, np.inf, 0.0))
            sc = np.where(A > 0, d / A, 0.0)
        den = np.abs(y_ref).max(axis=1)
        den[den == 0] = 1.0
        worst["scaled"] = max(worst["scaled"], float(sc.max()))
        worst["normwise"] = max(worst["normwise"], float((d.max(axis=1) / den).max()))
        worst["nmse"] = max(worst["nmse"], float((d ** 2).sum() / max((y_ref ** 2).sum(), 1e-300)))
        worst["f32_bound_ratio"] = max(worst["f32_bound_ratio"], float(r.max()))
        ok = ok and bool(np.isfinite(y).all()) and float(r.max()) <= 1.0 and float((d.max(axis=1) / den).max()) <= 2e-3
        n_out += d.size
    return {"outputs_checked": int(n_out), "matrices": len(refs), "of_matrices": len(ws.mats),
            "what": "the last timed step's outputs vs the oracle",
            "bound": ("|dy| <= 2^-16*Bm + 2^-11*(A + Bm/4) per output (fp4 matrix cores: activations in four "
                      "e2m3 pieces; Bm = sum |w| * block max |x|); normwise <= 2e-3" if fp4 else
                      "|dy| <= 1e-4*A + 2^-17*F per output; normwise <= 2e-3"),
            "scaled_max": float("%.4g" % worst["scaled"]), "normwise_max": float("%.4g" % worst["normwise"]),
            "nmse_max": float("%.4g" % worst["nmse"]), "f32_bound_ratio_max": float("%.4g" % worst["f32_bound_ratio"]),
            "pass": ok}


# Shapes of the selection sweep: (format, n_tok, K, M or (M1, M2) for a
# fused pair): the Llama-3.2-1B and Llama-3-8B decode shapes (q/k/v, o,
# gate+up fused, down, lm_head), their tensor-parallel shards over eight GPUs
# (8B q/k/v 768 x 4096, gate 1792 x 4096, down 4096 x 1792), and the 8B
# projections at 2 to 32 tokens.
SWEEP_REG = {1: {2048: (10, 11, 12), 4096: (13, 14, 15, 16, 17), 14336: (18, 19, 20)},
             2: {2048: (21,), 4096: (22, 25), 8192: (23,), 14336: (24,)}}


def sweep_shapes():
    out = []
    for fmt in (layout.Q4_0, layout.Q4_K):
        for K, M in [(2048, 3072), (2048, 2048), (2048, (8192, 8192)), (2048, 8192), (2048, 128256),
                     (4096, 768), (4096, 1792), (4096, 4096), (4096, 6144), (4096, (14336, 14336)),
                     (4096, 14336), (4096, 128256), (14336, 4096), (1792, 4096)]:
            out.append((fmt, 1, K, M))
        for K, M in [(2048, 8192), (4096, 4096), (4096, 6144), (4096, 14336), (4096, 128256), (14336, 4096)]:
            for nt in (2, 3, 4, 8, 12, 16, 24, 32):
                out.append((fmt, nt, K, M))
    return out


def sweep_cands(n_tok, K):
    if n_tok == 1:
        return (1,) + SWEEP_REG[1].get(K, ())
    if n_tok == 2:
        return SWEEP_REG[2].get(K, ()) + (30, 31)
    if n_tok <= 8:
        return (30, 31)
    if n_tok <= 16:
        return (31, 32)
    return (32,)


def run_sweep(out_path, n_seq=192, min_bytes=6e8):
    """Times every candidate of the selection table at each sweep shape (HIP
    events around n_seq back-to-back launches in one graph, rotating over
    copies of the weights that together exceed the 256 MB Infinity Cache,
    behind a device-side sleep) and writes the results as JSON."""
    import ctypes

    import torch

    lib = binding.library()
    shapes = []
    for fmt, nt, K, Mspec in sweep_shapes():
        Ms = list(Mspec) if isinstance(Mspec, tuple) else [Mspec]
        Mtot = sum(Ms)
        x = torch.from_numpy(synth.gen_x_seeded([5, K, nt], K, nt)).to("cuda")
        base = [torch.from_numpy(synth.gen_packed(fmt, m * K, np.random.default_rng([6, fmt, m, K]))).to("cuda")
                for m in Ms]
        nbytes = sum(w.numel() for w in base)
        reps = max(2, int(-(-min_bytes // nbytes)))
        Ws = [base] + [[w.clone() for w in base] for _ in range(reps - 1)]
        ys = [torch.empty((nt, m), dtype=torch.float32, device="cuda") for m in Ms]
        keep = []
        calls = []
        for ws in Ws:
            if len(Ms) > 1:
                arr = binding.multi_args([w.data_ptr() for w in ws], [v.data_ptr() for v in ys], Ms)
                keep.append(arr)
                calls.append((True, (fmt, len(Ms)) + arr + (x.data_ptr(), K, nt)))
            else:
                calls.append((False, (fmt, ws[0].data_ptr(), x.data_ptr(), ys[0].data_ptr(), Ms[0], K, nt)))
        results, names = [], {}
        for cand in sweep_cands(nt, K):
            os.environ["LW_FORCE_CFG"] = str(cand)
            try:
                name = (binding.kernel_name_multi(fmt, Ms, K, nt) if len(Ms) > 1
                        else binding.kernel_name(fmt, Ms[0], K, nt))
                if name in names:  # the candidate does not take the shape: the same kernel as another
                    continue
                stream = torch.cuda.current_stream()

                def run():
                    s_ = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
                    for i in range(n_seq):
                        multi, a = calls[i % len(calls)]
                        rc = lib.lw_matvec_multi(*a, s_) if multi else lib.lw_matvec(*a, s_)
                        if rc != 0:
                            raise binding.LwError(rc, "sweep")
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g):
                    run()
                g.replay()
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                torch.cuda._sleep(int(2.4e6 * 5))
                e0.record(stream)
                g.replay()
                e1.record(stream)
                torch.cuda.synchronize()
                us = e0.elapsed_time(e1) * 1e3 / n_seq
            finally:
                del os.environ["LW_FORCE_CFG"]
            names[name] = cand
            gbs = (sum(synth.algorithmic_bytes(fmt, m, K, nt) for m in Ms)) / (us * 1e-6) / 1e9
            results.append({"cand": cand, "kernel": name, "us": round(us, 3), "GB/s": round(gbs, 1)})
        best = min(results, key=lambda r: r["us"])
        log("sweep fmt=%d n_tok=%d K=%d M=%s: %s" % (fmt, nt, K, Ms, ", ".join(
            "%d:%.2fus" % (r["cand"], r["us"]) for r in results)))
        shapes.append({"fmt": fmt, "n_tok": nt, "K": K, "M": Mtot, "Ms": Ms, "results": results,
                       "best": best["cand"]})
        del Ws, base, ys, calls, keep
        torch.cuda.empty_cache()
    doc = {"what": "launch duration of every kernel-selection candidate per shape (HIP events, %d back-to-back "
                   "launches in one graph, weights rotated over copies above 600 MB)" % n_seq,
           "command": "python bench.py --sweep " + os.path.relpath(out_path, ROOT),
           "device": torch.cuda.get_device_name(0), "shapes": shapes}
    with open(out_path, "w") as fh:
        json.dump(doc, fh, indent=1)
    print(json.dumps({"sweep": out_path, "shapes": len(shapes)}))


def run_attn(args):
    """A decode step's attention: one lw_attn_decode per layer of a
    Llama-3-8B-shaped model over a KV cache of --kv-len positions in the
    --kv-fmt format (every layer its own K and V buffers, rotated over copies
    above 1 GB), timed as the matrix-vector steps are. Prints one JSON line."""
    import ctypes

    import torch

    lib = binding.library()
    fmt = layout.FORMATS[args.kv_fmt]
    Lkv = args.kv_len
    nl, H, nkv, D = (ATTN_MODEL[k] for k in ("n_layers", "n_heads", "n_kv", "head_dim"))
    n = nkv * Lkv * D
    t0 = time.time()
    host = []
    Ks, Vs, qs, outs = [], [], [], []
    for layer in range(nl):
        rk = np.random.default_rng(np.random.SeedSequence([0, 20, layer, 0]))
        rv = np.random.default_rng(np.random.SeedSequence([0, 20, layer, 1]))
        Kh, Vh = synth.gen_packed(fmt, n, rk), synth.gen_packed(fmt, n, rv)
        q = synth.gen_x_seeded([0, 20, layer, 2], D, H)
        host.append((Kh, Vh, q))
        Ks.append(torch.from_numpy(Kh).to("cuda"))
        Vs.append(torch.from_numpy(Vh).to("cuda"))
        qs.append(torch.from_numpy(q).to("cuda"))
        outs.append(torch.empty((H, D), dtype=torch.float32, device="cuda"))
    packed = sum(k.numel() + v.numel() for k, v in zip(Ks, Vs))
    reps = max(1, int(-(-1e9 // packed)))
    Kall = [Ks] + [[k.clone() for k in Ks] for _ in range(reps - 1)]
    Vall = [Vs] + [[v.clone() for v in Vs] for _ in range(reps - 1)]
    wsb = binding.attn_workspace_bytes(fmt, H, nkv, D, Lkv)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    torch.cuda.synchronize()
    log("attention: %d layers, %s cache of %d positions, %.3f GB (%d copies), generated in %.1fs"
        % (nl, args.kv_fmt, Lkv, packed / 1e9, reps, time.time() - t0))
    scale = ctypes.c_float(1.0 / np.sqrt(D))

    def step(rep, s_):
        for layer in range(nl):
            rc = lib.lw_attn_decode(fmt, qs[layer].data_ptr(), Kall[rep][layer].data_ptr(),
                                    Vall[rep][layer].data_ptr(), outs[layer].data_ptr(), H, nkv, D, Lkv, scale,
                                    ws.data_ptr(), wsb, s_)
            if rc != 0:
                raise binding.LwError(rc, "lw_attn_decode")

    def steps_on(first, count):
        s_ = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        for i in range(first, first + count):
            step(i % reps, s_)
    nodes = 2 * nl
    graphs = []
    for first, count in ((0, args.warmup), (args.warmup, args.steps)):
        gs = []
        for f, c in graph_chunks(first, count, nodes) or []:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                steps_on(f, c)
            gs.append(g)
        graphs.append(gs)
    for g in graphs[0]:
        g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for g in graphs[1]:
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    y_timed = [o.cpu().numpy() for o in outs]
    kv_bytes = packed  # one copy of every layer's K and V
    alg = kv_bytes + nl * 2 * H * D * 4  # K, V, q, out
    gbs = alg / (ms * 1e-3) / 1e9
    # per call: the two kernels of one layer, 192 back to back, behind a device-side sleep
    g2 = torch.cuda.CUDAGraph()
    seq = 192

    def sub():
        s_ = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        for i in range(seq):
            rep, layer = (i // nl) % reps, i % nl
            rc = lib.lw_attn_decode(fmt, qs[layer].data_ptr(), Kall[rep][layer].data_ptr(),
                                    Vall[rep][layer].data_ptr(), outs[layer].data_ptr(), H, nkv, D, Lkv, scale,
                                    ws.data_ptr(), wsb, s_)
            if rc != 0:
                raise binding.LwError(rc, "lw_attn_decode")
    with torch.cuda.graph(g2):
        sub()
    g2.replay()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    torch.cuda._sleep(int(2.4e6 * 5))
    e0.record(stream)
    g2.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    call_us = e0.elapsed_time(e1) * 1e3 / seq
    call_bytes = alg / nl
    kname = binding.attn_kernel_name(fmt, H, nkv, D, Lkv)
    roof = {"bound": "hbm", "achieved": round(call_bytes / (call_us * 1e-6) / 1e9, 1), "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": round(call_bytes / (call_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4), "traffic": None,
            "kernel": kname + " + attn_combine_kernel<%d>" % D, "launches_per_step": 2 * nl,
            "avg_call_us": round(call_us, 3), "alg_bytes_per_call": round(call_bytes),
            "note": "achieved = one call's algorithmic bytes (K, V, q, out) over the call's duration (both kernels)"}
    ceil, _ = ceilings(False, call_bytes, "graph")
    out = {"metric": METRIC_ATTN, "value": round(gbs, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "f32",
           "data": "synthetic (seeded; cache codes and scales drawn as for the weight formats, query N(0,1))",
           "config": {"workload": "attn_llama8b_%s_kv%d" % (args.kv_fmt, Lkv),
                      "description": "decode attention of a Llama-3-8B-shaped model (32 layers, 32 query heads over "
                                     "8 key/value heads of 128) over a %s KV cache of %d positions" % (args.kv_fmt, Lkv),
                      "format": args.kv_fmt, "kv_len": Lkv, "layers": nl, "bytes_per_step": round(alg),
                      "mode": "graph", "op": "attn", "copies": reps},
           "pct_of_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2), "roofline": roof, "stream_ceiling": ceil}
    if not args.no_cpu_baseline:
        import oracle
        t_used, done, nb_ = 0.0, 0, 0
        worst, ok, n_out = 0.0, True, 0
        for layer in range(nl):
            Kh, Vh, q = host[layer]
            t1 = time.perf_counter()
            ref, A, T = oracle.attn_decode(fmt, q, Kh, Vh, H, nkv, D, Lkv, 1.0 / np.sqrt(D))
            t_used += time.perf_counter() - t1
            done += 1
            nb_ += alg / nl
            err = np.abs(y_timed[layer].astype(np.float64) - ref)
            bound = 2.0 ** -12 * (1 + T)[:, None] * A
            with np.errstate(divide="ignore", invalid="ignore"):
                worst = max(worst, float(np.where(bound > 0, err / bound, np.where(err > 0, np.inf, 0)).max()))
            n_out += err.size
            if t_used >= args.cpu_seconds:
                break
        ok = worst <= 1.0
        out["cpu_baseline"] = {"value": round(nb_ / t_used / 1e9, 4), "unit": "GB/s", "cores": 1,
                               "host_cpus": os.cpu_count() or 1, "kind": "oracle", "seconds": round(t_used, 2),
                               "sample": "%d of %d layers, same inputs; oracle = plain C, double, one thread"
                                         % (done, nl)}
        out["parity"] = {"outputs_checked": n_out, "layers": done, "of_layers": nl,
                         "what": "the last timed step's outputs vs the oracle",
                         "bound": "|dout| <= 2^-12 (1 + T) sum_j p_j |v_j| per output",
                         "bound_ratio_max": float("%.4g" % worst), "pass": ok}
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="q4_k_llama8b", choices=sorted(synth.WORKLOADS))
    ap.add_argument("--n-tok", type=int, default=1)
    ap.add_argument("--mode", choices=["graph", "eager"], default="graph")
    ap.add_argument("--kv-len", type=int, default=8192, help="--op attn: cached positions")
    ap.add_argument("--kv-fmt", default="q8_0", choices=["f16", "q8_0", "q4_0", "q4_1", "q5_0", "q5_1", "mxfp4"],
                    help="--op attn: KV cache format")
    ap.add_argument("--op", choices=["matvec", "dequant", "attn"], default="matvec",
                    help="matvec: one lw_matvec per matrix (the decode step); dequant: one lw_dequant per "
                         "matrix into float32 (eager, on the null stream); attn: one lw_attn_decode per layer")
    ap.add_argument("--no-fuse", action="store_true",
                    help="one lw_matvec per matrix (default: a layer's gate and up share one lw_matvec_multi call)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sweep", metavar="OUT_JSON", default=None,
                    help="time every kernel-selection candidate at the sweep shapes and write OUT_JSON "
                         "(the committed copy is profiles/sweep_select.json, which generates the table)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain copy kernel over MIB MiB 20 times (HBM counter calibration)")
    ap.add_argument("--calibrate-read", type=int, default=0, metavar="MIB",
                    help="only run libceiling's 128-bit non-temporal read kernel over MIB MiB 20 times "
                         "(a second, read-only HBM counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (use --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import torch

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    binding.library()  # fails loudly if the HIP library is missing

    if args.sweep:
        os.environ.pop("LW_FORCE_CFG", None)
        run_sweep(args.sweep)
        return

    if args.calibrate_copy:
        n = args.calibrate_copy * (1 << 20)
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(20):
            torch.neg(src, out=dst)  # a plain elementwise kernel: reads n bytes, writes n bytes
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n, "copies": 20}))
        return

    if args.calibrate_read:
        # reads exactly n bytes per launch and writes nothing (the sink word
        # is stored only if the folded value hits a fixed constant)
        import ctypes
        n = args.calibrate_read * (1 << 20)
        lib = ctypes.CDLL(os.path.join(ROOT, "paper_2605_20706_amd", "libceiling.so"))
        lib.lw_ceiling_read.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        sink = torch.zeros(1, dtype=torch.int32, device="cuda")
        torch.cuda.synchronize()
        s = torch.cuda.current_stream().cuda_stream
        for _ in range(20):
            rc = lib.lw_ceiling_read(src.data_ptr(), n, sink.data_ptr(), s)
            if rc != 0:
                raise RuntimeError("libceiling: code %d" % rc)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_read_bytes": n, "reads": 20}))
        return

    if args.op == "attn":
        run_attn(args)
        return

    wl = synth.WORKLOADS[args.workload]
    keep = 0 if args.no_cpu_baseline else len(wl.matrices)
    if args.op == "dequant":
        args.mode = "eager"  # lw_dequant is on the null stream, which a graph capture cannot record
    ws = Workset(wl, args.n_tok, keep_host=keep, op=args.op, fuse=not args.no_fuse)
    ms_per_step, per_shape, y_timed, mode_used = run_gpu(ws, args.steps, args.warmup, args.mode)

    n_launch = len(ws.groups)
    step_bytes = sum(ws.alg_bytes)
    gbs = step_bytes / (ms_per_step * 1e-3) / 1e9
    tok_s = args.n_tok / (ms_per_step * 1e-3)
    fmt_name = layout.FORMAT_NAMES[wl.fmt]
    # the roofline of the kernel that takes most of a step: its algorithmic
    # bytes (or flops) per launch over its average launch duration, both from
    # the per-shape phase (HIP events around back-to-back launches of one
    # shape on the launch stream)
    names, groups = kernel_groups(ws, per_shape)
    kname = max(groups, key=lambda k: groups[k]["us"])
    g = groups[kname]
    # the bound follows the arithmetic intensity, not the unit: matrix-core
    # kernels at a few tokens are still memory-bound
    ridge = MFMA_BF16_PEAK_TFS * 1e12 / (HBM_PEAK_GBS * 1e9)  # flop per byte
    mfma = g["flop"] / g["bytes"] > ridge
    avg_launch_s = g["us"] * 1e-6 / g["launches"]
    if mfma:
        # the contraction's own operand types: e2m1 x e2m3 on the fp4 path
        # (four activation pieces, so its algorithmic flops are a quarter of
        # the matrix-core flops it issues), else bf16
        fp4 = kname.split("<")[0] == "fp4mm_kernel"
        peak = MFMA_FP4_PEAK_TFS if fp4 else MFMA_BF16_PEAK_TFS
        kern_tfs = g["flop"] / (g["us"] * 1e-6) / 1e12
        roof = {"bound": "mfma", "achieved": round(kern_tfs, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(kern_tfs / peak, 4), "mfma_operands": "fp4 x fp6" if fp4 else "bf16 x bf16"}
    else:
        kern_gbs = g["bytes"] / (g["us"] * 1e-6) / 1e9
        roof = {"bound": "hbm", "achieved": round(kern_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(kern_gbs / HBM_PEAK_GBS, 4)}
    roof.update({"traffic": stored_traffic(wl.key, args.n_tok, kname),
                 "traffic_method": traffic_method(wl.key, args.n_tok), "kernel": kname,
                 "launches_per_step": g["launches"], "avg_launch_us": round(avg_launch_s * 1e6, 3),
                 "alg_bytes_per_launch": round(g["bytes"] / g["launches"]),
                 "alg_flop_per_launch": round(g["flop"] / g["launches"]),
                 "share_of_step": round(g["us"] / sum(v["us"] for v in groups.values()), 4)})
    kernels_out = {k: {"launches": v["launches"], "us_per_step": round(v["us"], 1),
                       "GB/s": round(v["bytes"] / (v["us"] * 1e-6) / 1e9, 1)} for k, v in groups.items()}
    shape_out = {}
    ng = len(ws.groups)
    for k, (ms, idx) in per_shape.items():
        j = idx[0] % ng
        b = ws.call_bytes[j]
        shape_out[k] = {"us": round(ms * 1e3, 2), "GB/s": round(b / (ms * 1e-3) / 1e9, 1), "kernel": names[j]}
        if mfma:
            shape_out[k]["TFLOP/s"] = round(ws.call_flops[j] / (ms * 1e-3) / 1e12, 1)
    out = {
        "metric": METRIC if args.op == "matvec" else METRIC_DEQUANT, "value": round(gbs, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "fp4*fp6->f32" if ws.use_ws else "f32",
        "data": "synthetic (seeded; shapes and value distributions of the workload)",
        "config": {"workload": wl.key, "description": wl.description, "format": fmt_name,
                   "matrices": len(ws.mats), "calls_per_step": n_launch,
                   "fused": "a layer's gate and up in one lw_matvec_multi call" if ws.fuse_used else "none",
                   "weights": wl.weights, "n_tok": args.n_tok,
                   "bytes_per_step": round(step_bytes), "mode": mode_used, "op": args.op,
                   "launches_per_step": ws.step_nodes,
                   "weight_copies": ws.reps},
        "pct_of_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
        "equiv_decode_tok_s": round(tok_s, 1) if args.op == "matvec" else None,
        "roofline": roof,
        "kernels": kernels_out,
        "per_shape": shape_out,
    }
    # the value against a plain streaming kernel's rate in the same process
    # (read, or write for the dequantization), and the dominant kernel against
    # that kernel at the dominant kernel's bytes per launch
    # Per call shape (memory-bound paths): the streaming kernel at the call's
    # bytes per launch; and the step as a whole if every call ran at that
    # rate (the launch sequence's own ceiling, launch gaps and ramp included).
    shape_b = {k: ws.call_bytes[idx[0] % ng] for k, (_, idx) in per_shape.items()}
    ceil, at = ceilings(args.op == "dequant", roof["alg_bytes_per_launch"], args.mode,
                        () if mfma else tuple(shape_b.values()))
    ceil["value_over_1GiB_ceiling"] = round(gbs / ceil["GB/s_1GiB"], 4)
    if roof["bound"] == "hbm":
        ceil["dominant_kernel_over_launch_ceiling"] = round(roof["achieved"] / ceil["GB/s_at_launch_bytes"], 4)
    if at:
        step_s = 0.0
        for k, (_, idx) in per_shape.items():
            c = at[shape_b[k]]
            shape_out[k]["ceiling_GB/s"] = round(c, 1)
            shape_out[k]["over_ceiling"] = round(shape_out[k]["GB/s"] / c, 4)
            step_s += sum(1 for i in idx if i < ng) * shape_b[k] / (c * 1e9)
        ceil["step_GB/s_at_shape_ceilings"] = round(step_bytes / step_s / 1e9, 1)
        ceil["value_over_step_ceiling"] = round(gbs * 1e9 * step_s / step_bytes, 4)
    out["stream_ceiling"] = ceil
    if not args.no_cpu_baseline:
        out["cpu_baseline"], parity = cpu_baseline(ws, args.cpu_seconds, y_timed)
        if parity is not None:
            out["parity"] = parity
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
