#!/usr/bin/env python3
"""Benchmark: one GPU's TP-aware MLP shard (Alg. 3 without its AllReduce).

Default workload: the Llama-70B MLP problem size (hidden 8192, intermediate
28672, up_proj then down_proj) at TP = 8, rank 0: W1 shard 8192 x 3584,
W2 shard 3584 x 8192, int4 weights with G = 128, fp16 activations, decode
batch M = 16 (M = 1 and 4 are reported alongside).

A step is one pass of the hot path: gather X[:, P1] -> ordered W4A16 GEMM1 ->
ordered W4A16 GEMM2 (tpdq_mlp_shard). Weights are resident in HBM and rotate
over replicas whose total exceeds twice the 256 MB Infinity Cache, so every
step streams its weights from HBM. The timed steps are replayed from one HIP
graph (the library launches on torch's current stream, which torch captures),
timed with events on that stream.

Prints ONE JSON line on stdout.
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
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "W4A16 MLP-shard latency (us) + achieved HBM GB/s vs peak, Llama-70B shapes"
HBM_PEAK_GBS = 8000.0
MFMA_F16_PEAK_TFLOPS = 2500.0
MALL_BYTES = 256 << 20
ROTATE_MIN_BYTES = 640 << 20


def eprint(*a):
    print(*a, file=sys.stderr, flush=True)


def shard_bytes(K, N, G, ng=None):
    """Algorithmic bytes of one W4 layer shard: packed weights, fp16 scales,
    packed zeros (ng metadata rows)."""
    ng = K // G if ng is None else ng
    return K * N // 2 + ng * N * 2 + ng * N // 2


def gemm_bytes(M, K, N, G, ng=None, gidx=False, xperm=False):
    b = shard_bytes(K, N, G, ng) + M * K * 2 + M * N * 2
    if gidx:
        b += K * 4
    if xperm:
        b += K * 4
    return b


def kernel_source_hash():
    h = hashlib.sha256()
    for f in ("decode_kernels.h", "gemm_decode.hip", "kernels_common.h", "tpdq_internal.h"):
        with open(os.path.join(ROOT, "paper_2402_04925_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def read_traffic(workload, M):
    """HBM traffic (FETCH_SIZE + WRITE_SIZE per launch of the ordered decode
    kernel) from a committed counter summary, if one exists for the current
    kernel source; None otherwise."""
    path = os.path.join(ROOT, "profiles", f"traffic_decode_ordered_{workload}_M{M}.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if "=" in line and not line.startswith("#"):
                k, v = line.split("=", 1)
                vals[k.strip()] = v.strip()
    if vals.get("kernel_source_hash") != kernel_source_hash():
        return None
    try:
        return float(vals["bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def read_mfma_util():
    """MFMA utilisation of the prefill GEMMs from the committed counter
    summary: SQ_VALU_MFMA_BUSY_CYCLES over (GRBM_GUI_ACTIVE / 8) x 1024 SIMDs,
    and the clock the part ran at, averaged per GEMM (by grid); None when the
    summary is absent."""
    path = os.path.join(ROOT, "profiles", "prefill_llama70b_tp2_M2048.md")
    if not os.path.exists(path):
        return None
    rows = {}
    in_util = False
    with open(path) as f:
        for line in f:
            if line.startswith("## MFMA utilisation"):
                in_util = True
            elif in_util and line.startswith("| ") and "`k_prefill" in line:
                c = [x.strip() for x in line.strip().strip("|").split("|")]
                try:
                    grid, ghz, util = int(c[2]), float(c[7]), float(c[8])
                except (IndexError, ValueError):
                    continue
                rows.setdefault(grid, []).append((util, ghz))
    if not rows:
        return None
    out = {}
    for grid, name in ((448, "gemm1"), (256, "gemm2")):
        v = rows.get(grid)
        if v:
            out[name] = dict(mfma_busy_of_clocks=round(sum(u for u, _ in v) / len(v), 3),
                             clock_ghz=round(sum(g for _, g in v) / len(v), 2))
    out["denominator"] = "GRBM_GUI_ACTIVE / 8 (the dispatch's clocks) x 1024 SIMDs"
    out["source"] = "profiles/prefill_llama70b_tp2_M2048.md"
    return out


class Setup:
    """Device-resident shards (rank 0) of one workload, replicated for rotation.
    bf16: bfloat16 scales (and activations, in Calls)."""

    def __init__(self, wl, dev, min_bytes=ROTATE_MIN_BYTES, bf16=False):
        import torch
        import paper_2402_04925_amd as tpdq
        from paper_2402_04925_amd import inputs

        self.wl = wl
        self.bf16 = bf16
        t0 = time.time()
        L1, L2 = inputs.make_workload(wl, scale_dtype=inputs.BF16 if bf16 else np.float16)
        self.L1, self.L2 = L1, L2
        eprint(f"[bench] generated {wl.name} layers{' (bf16 scales)' if bf16 else ''} in {time.time() - t0:.1f}s")

        def dev_layer(L):
            sc = torch.from_numpy(L.scales)
            if bf16:
                sc = sc.to(torch.bfloat16)
            return tpdq.QuantWeight.from_tensors(
                torch.from_numpy(L.qweight).to(dev), sc.to(dev),
                torch.from_numpy(L.qzeros).to(dev), torch.from_numpy(L.g_idx.astype(np.int32)).to(dev),
                L.G)

        d1, d2 = dev_layer(L1), dev_layer(L2)
        P1, _, P2, _, w1o, w2o = tpdq.reorder(d1, d2)
        # Alg. 2's local data flow at TP = 1 needs W1[P1] with its columns in place
        w1u = tpdq.reorder(d1)[4] if wl.tp == 1 else None
        torch.cuda.synchronize()
        tp = wl.tp
        self.P1 = P1
        self.P2 = P2
        # rank-0 shards, materialised densely (what a deployment would ship)
        ord1 = w1o.column_shard(0, tp)
        ord2 = w2o.row_shard(0, tp, sorted_rows=True)
        act1 = d1.column_shard(0, tp)
        act2 = d2.row_shard(0, tp, sorted_rows=False)

        def dense(q, with_g):
            return tpdq.QuantWeight(q.qweight.contiguous(), q.scales.contiguous(), q.qzeros.contiguous(),
                                    q.g_idx.contiguous() if with_g and q.g_idx is not None else None,
                                    q.K, q.N, q.G, q.num_groups, q.layout)

        a1, a2 = dense(act1, True), dense(act2, True)
        base = [dense(ord1, False), dense(ord2, False), a1, a2, tpdq.pack_tiled(a1), tpdq.pack_tiled(a2)]
        if w1u is not None:
            base.append(dense(w1u, False))   # index 6: W1[P1] (Alg. 2 at TP = 1)
        per = sum(t.qweight.numel() * 4 + t.scales.numel() * 2 + t.qzeros.numel() * 4 for t in base[:2])
        self.R = max(2, -(-min_bytes // per))
        self.reps = [base]
        for _ in range(self.R - 1):
            self.reps.append([tpdq.QuantWeight(q.qweight.clone(), q.scales.clone(), q.qzeros.clone(),
                                               q.g_idx.clone() if q.g_idx is not None else None,
                                               q.K, q.N, q.G, q.num_groups, q.layout) for q in base])
        torch.cuda.synchronize()
        del d1, d2, w1o, w2o, w1u
        eprint(f"[bench] {self.R} weight replicas of {per / 1e6:.1f} MB (ordered pair)")


def capture_and_time(fn_list, steps, warmup, dev):
    """Replay the calls fn_list[i % len] for `steps` iterations from a HIP
    graph; return ms per iteration (events on the capture stream)."""
    import torch
    s = torch.cuda.Stream(device=dev)
    s.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(s):
        for i in range(min(3, len(fn_list))):   # eager warm-up on the capture stream
            fn_list[i % len(fn_list)]()
    torch.cuda.current_stream(dev).wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        for i in range(steps):
            fn_list[i % len(fn_list)]()
    torch.cuda.synchronize()
    for _ in range(max(1, warmup // max(1, steps) + 1)):
        g.replay()
    torch.cuda.synchronize()
    times = []
    cur = torch.cuda.current_stream(dev)
    for _ in range(5):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(cur)
        g.replay()
        e1.record(cur)
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1) / steps)
    del g
    return float(np.median(times)), times


def cpu_baseline(wl, M, L1, L2, budget_s=20.0):
    """The oracle's rank-0 Alg. 3 partial, timed on the host on a bounded
    sample of runs. Reported only."""
    from oracle import tpdq_oracle as o
    X = None
    from paper_2402_04925_amd import inputs
    X = inputs.make_x(wl, M)
    P2, _ = o.reorder(L2.g_idx)
    l1 = (L1.qweight, L1.scales, L1.qzeros, L1.g_idx)
    l2 = (L2.qweight, L2.scales, L2.qzeros, L2.g_idx)
    # one thread: the oracle's dequantization is single-threaded numpy, which
    # is most of its time, so its BLAS pool is held to one thread as well and
    # the core count reported is the one it used
    from threadpoolctl import threadpool_limits
    runs = []
    t_start = time.time()
    with threadpool_limits(limits=1):
        while not runs or (time.time() - t_start < budget_s and len(runs) < 20):
            t0 = time.perf_counter()
            o.mlp_rank_from_global(X, l1, l2, 0, wl.tp, True, P2=P2)
            runs.append(time.perf_counter() - t0)
    return dict(value=float(np.median(runs)) * 1e6, unit="us", cores=1, kind="oracle",
                sample=f"{len(runs)} runs of the oracle's rank-0 MLP shard ({wl.name}, M={M}, "
                       f"ordered, float64 dequant + GEMM, one thread), median")


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_detail():
    """The oracle on the host beyond the headline sample (reported only):
    Alg. 1 (the stable argsort of both g_idx) and the rank-0 MLP shard of
    every decode workload at its largest decode M, with the BLAS thread pool
    at its default size and at one thread, and the tiny single GEMM on both
    paths. One run per item except the tiny GEMM (median of 20); the
    unsharded Llama-70B shard computes 512 of the 8192 GEMM2 columns. The
    TP=2 prefill shard (M = 2048) runs once, with the default pool, on 1024
    of its GEMM2 columns."""
    from threadpoolctl import threadpool_info, threadpool_limits
    from oracle import tpdq_oracle as o
    from paper_2402_04925_amd import inputs

    def timed(fn, runs=1):
        ts = []
        for _ in range(runs):
            t0 = time.perf_counter()
            fn()
            ts.append(time.perf_counter() - t0)
        return float(np.median(ts)) * 1e6

    pool = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    out = dict(cpu_model=cpu_model(), logical_cpus=os.cpu_count(), blas_threads=int(pool),
               unit="us", kind="oracle", items={})
    w = inputs.WORKLOADS["tiny_gemm"]
    L, _ = inputs.make_workload(w)
    X = inputs.make_x(w, 4)
    P, g = o.reorder(L.g_idx)
    l_act = (L.qweight, L.scales, L.qzeros, L.g_idx)
    qo = o.permute_rows(dict(qweight=L.qweight, scales=L.scales, qzeros=L.qzeros), P)["qweight"]
    out["items"]["tiny_gemm"] = dict(
        M=4, reorder_us=round(timed(lambda: o.reorder(L.g_idx), 20), 1),
        actorder_gemm_us=round(timed(lambda: o.w4a16_gemm(X, *l_act), 20), 1),
        ordered_gemm_us=round(timed(lambda: o.w4a16_gemm(X, qo, L.scales, L.qzeros, g, x_perm=P), 20), 1))
    for name, M, sample in (("llama70b_tp8", 16, None), ("granite20b_tp4", 16, None),
                            ("llama70b_tp1", 64, 512)):
        w = inputs.WORKLOADS[name]
        L1, L2 = inputs.make_workload(w)
        X = inputs.make_x(w, M)
        P2, _ = o.reorder(L2.g_idx)
        l1 = (L1.qweight, L1.scales, L1.qzeros, L1.g_idx)
        l2 = (L2.qweight, L2.scales, L2.qzeros, L2.g_idx)
        cols = None if sample is None else np.arange(0, w.N2, w.N2 // sample)
        mlp = lambda: o.mlp_rank_from_global(X, l1, l2, 0, w.tp, True, P2=P2, cols2=cols)
        it = dict(M=M, reorder_us=round(timed(lambda: (o.reorder(L1.g_idx), o.reorder(L2.g_idx))), 1),
                  mlp_shard_us=round(timed(mlp), 1))
        with threadpool_limits(limits=1):
            it["mlp_shard_us_1thread"] = round(timed(mlp), 1)
        if sample is not None:
            it["gemm2_columns"] = f"{sample} of {w.N2}"
        out["items"][name] = it
        eprint(f"[bench] oracle on the host, {name} M={M}: {it}")
        del L1, L2
    # the TP=2 prefill shard once (M = 2048; about 240 GFLOP of float64 GEMM1),
    # the default pool only, GEMM2 on 1024 of its 8192 columns
    w = inputs.WORKLOADS["llama70b_tp2_prefill"]
    L1, L2 = inputs.make_workload(w)
    M = w.Ms[0]
    X = inputs.make_x(w, M)
    P2, _ = o.reorder(L2.g_idx)
    l1 = (L1.qweight, L1.scales, L1.qzeros, L1.g_idx)
    l2 = (L2.qweight, L2.scales, L2.qzeros, L2.g_idx)
    cols = np.arange(0, w.N2, w.N2 // 1024)
    it = dict(M=M, reorder_us=round(timed(lambda: (o.reorder(L1.g_idx), o.reorder(L2.g_idx))), 1),
              mlp_shard_us=round(timed(lambda: o.mlp_rank_from_global(X, l1, l2, 0, w.tp, True, P2=P2,
                                                                      cols2=cols)), 1),
              gemm2_columns=f"1024 of {w.N2}")
    out["items"][w.name] = it
    eprint(f"[bench] oracle on the host, {w.name} M={M}: {it}")
    return out


class Calls:
    """Library calls of one batch size M on the rank-0 shards: the MLP shard
    and each GEMM on its own, for every path, one closure per weight replica."""

    PAIRS = {"ordered": (0, 1), "actorder": (2, 3), "actorder_global": (2, 3), "actorder_tiled": (4, 5)}

    def __init__(self, st, M, dev):
        import torch
        import paper_2402_04925_amd as tpdq
        from paper_2402_04925_amd import inputs
        wl = st.wl
        self.st, self.M, self.dev = st, M, dev
        self.tpdq = tpdq
        self.lib = tpdq._abi.lib()
        if st.bf16:
            self.X = torch.from_numpy(inputs.make_x(wl, M, dtype=inputs.BF16)).to(torch.bfloat16).to(dev)
        else:
            self.X = torch.from_numpy(inputs.make_x(wl, M)).to(dev)
        self.dt = tpdq.BF16 if st.bf16 else tpdq.FP16
        self.y1 = torch.empty(M, wl.N1 // wl.tp, dtype=self.X.dtype, device=dev)
        self.y2 = torch.empty(M, wl.N2, dtype=self.X.dtype, device=dev)
        self.xg = self.X[:, st.P1.long()].contiguous()   # X[:, P1] for the single-GEMM timings
        self.ws = tpdq.Workspace(dev)
        self.paths = {"ordered": tpdq.PATH_ORDERED, "actorder": tpdq.PATH_ACTORDER,
                      "actorder_global": tpdq.PATH_ACTORDER_GLOBAL,
                      "actorder_tiled": tpdq.PATH_ACTORDER}

    def _stream(self):
        import torch
        return torch.cuda.current_stream(self.dev).cuda_stream

    def mlp(self, rep, pname):
        import ctypes
        tpdq, lib, M = self.tpdq, self.lib, self.M
        path = self.paths[pname]
        i1, i2 = self.PAIRS[pname]
        c1, c2 = rep[i1].c_struct(), rep[i2].c_struct()
        nb = lib.tpdq_workspace_bytes(tpdq.OP_MLP, M, ctypes.byref(c1), ctypes.byref(c2))
        buf = self.ws.get(nb)
        P1 = self.st.P1.data_ptr() if path == tpdq.PATH_ORDERED else None
        X, y1, y2 = self.X, self.y1, self.y2

        def call():
            tpdq._abi.check(lib.tpdq_mlp_shard(
                X.data_ptr(), X.stride(0), M, P1, ctypes.byref(c1), ctypes.byref(c2), path,
                self.dt, y1.data_ptr(), y2.data_ptr(), buf.data_ptr(), buf.numel(), self._stream()))
        return call

    def alg2_mlp(self, rep):
        """Alg. 2's local data flow at TP = 1: Y1 = X[:, P1] @ W1[P1] (columns in
        place), then Y2 = Y1[:, P2] @ W2[P2], the gather inside GEMM2 (x_perm)."""
        import ctypes
        tpdq, lib, M = self.tpdq, self.lib, self.M
        c1, c2 = rep[6].c_struct(), rep[1].c_struct()
        nb = max(lib.tpdq_workspace_bytes(tpdq.OP_GEMM, M, ctypes.byref(c1), None),
                 lib.tpdq_workspace_bytes(tpdq.OP_GEMM, M, ctypes.byref(c2), None))
        buf = self.ws.get(nb)
        X, y1, y2 = self.X, self.y1, self.y2
        P1, P2 = self.st.P1.data_ptr(), self.st.P2.data_ptr()

        def call():
            tpdq._abi.check(lib.tpdq_w4a16_gemm(
                X.data_ptr(), X.stride(0), M, P1, ctypes.byref(c1), tpdq.PATH_ORDERED, self.dt,
                y1.data_ptr(), y1.stride(0), buf.data_ptr(), buf.numel(), self._stream()))
            tpdq._abi.check(lib.tpdq_w4a16_gemm(
                y1.data_ptr(), y1.stride(0), M, P2, ctypes.byref(c2), tpdq.PATH_ORDERED, self.dt,
                y2.data_ptr(), y2.stride(0), buf.data_ptr(), buf.numel(), self._stream()))
        return call

    def gemm1_gather(self, rep):
        """The ordered GEMM1 as the MLP runs it: X[:, P1] gathered in the call."""
        import ctypes
        tpdq, lib, M = self.tpdq, self.lib, self.M
        c = rep[0].c_struct()
        nb = lib.tpdq_workspace_bytes(tpdq.OP_GEMM, M, ctypes.byref(c), None)
        buf = self.ws.get(nb)
        X, P1, out = self.X, self.st.P1.data_ptr(), self.y1

        def call():
            tpdq._abi.check(lib.tpdq_w4a16_gemm(
                X.data_ptr(), X.stride(0), M, P1, ctypes.byref(c), tpdq.PATH_ORDERED, self.dt,
                out.data_ptr(), out.stride(0), buf.data_ptr(), buf.numel(), self._stream()))
        return call

    def gemm(self, rep, which, pname):
        import ctypes
        tpdq, lib, M = self.tpdq, self.lib, self.M
        path = self.paths[pname]
        c = rep[self.PAIRS[pname][which]].c_struct()
        nb = lib.tpdq_workspace_bytes(tpdq.OP_GEMM, M, ctypes.byref(c), None)
        buf = self.ws.get(nb)
        xin = (self.xg if path == tpdq.PATH_ORDERED else self.X) if which == 0 else self.y1
        out = self.y1 if which == 0 else self.y2

        def call():
            tpdq._abi.check(lib.tpdq_w4a16_gemm(
                xin.data_ptr(), xin.stride(0), M, None, ctypes.byref(c), path, self.dt,
                out.data_ptr(), out.stride(0), buf.data_ptr(), buf.numel(), self._stream()))
        return call


COPY_BYTES = 1 << 30


def copy_ceiling(dev, reps=10):
    """Plain device copy (torch's copy kernel) of 1 GiB: read + write GB/s.
    Context for the roofline fraction; also the calibration kernel of the HBM
    traffic counters."""
    import torch
    src = torch.empty(COPY_BYTES // 2, dtype=torch.float16, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    cur = torch.cuda.current_stream(dev)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(cur)
    for _ in range(reps):
        dst.copy_(src)
    e1.record(cur)
    torch.cuda.synchronize()
    sec = e0.elapsed_time(e1) / 1e3 / reps
    del src, dst
    return 2 * COPY_BYTES / sec / 1e9


def copy_shard(dev, nbytes, steps, warmup):
    """Graph-timed device copy of one buffer the size of a weight shard
    (torch's copy kernel, one launch per step, rotating over enough buffers
    that every step reads HBM): what one launch that moves this many bytes
    costs on the part, for comparison with the GEMMs of the same size."""
    import torch
    n = nbytes // 2
    reps = max(2, -(-ROTATE_MIN_BYTES // nbytes))
    pairs = [(torch.ones(n, dtype=torch.float16, device=dev), torch.empty(n, dtype=torch.float16, device=dev))
             for _ in range(reps)]
    fns = [(lambda s=s_, d=d_: d.copy_(s)) for s_, d_ in pairs]
    ms, _ = capture_and_time(fns, steps, warmup, dev)
    del pairs, fns
    torch.cuda.synchronize()
    return ms * 1e3


def profile_run(st, Ms, launches, dev):
    """Eager launches for rocprofv3 (kernel trace or counters): every path's
    GEMM1 and GEMM2 and the ordered MLP shard at each M (and Alg. 2's local
    flow at TP = 1), `launches` times each over the rotating replicas, then
    the 1 GiB copy kernel."""
    import torch
    for M in Ms:
        c = Calls(st, M, dev)
        for pname in ("ordered", "actorder", "actorder_global", "actorder_tiled"):
            for which in (0, 1):
                fns = [c.gemm(rep, which, pname) for rep in st.reps]
                for i in range(launches):
                    fns[i % len(fns)]()
                torch.cuda.synchronize()
                eprint(f"[profile] M={M} {pname} gemm{which + 1}: {launches} launches")
        fns = [c.mlp(rep, "ordered") for rep in st.reps]
        for i in range(launches):
            fns[i % len(fns)]()
        torch.cuda.synchronize()
        eprint(f"[profile] M={M} ordered mlp: {launches} launches")
        if st.wl.tp == 1:   # Alg. 2's local data flow (W1[P1] with its columns in place)
            fns = [c.alg2_mlp(rep) for rep in st.reps]
            for i in range(launches):
                fns[i % len(fns)]()
            torch.cuda.synchronize()
            eprint(f"[profile] M={M} alg2 mlp: {launches} launches")
    src = torch.empty(COPY_BYTES // 2, dtype=torch.float16, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    for _ in range(launches):
        dst.copy_(src)
    torch.cuda.synchronize()
    eprint(f"[profile] copy of {COPY_BYTES} bytes: {launches} launches")


MFMA_F16_PEAK_TFLOPS = 2500.0   # MI355X dense fp16 MFMA


def config_lines(dev, steps, warmup):
    """The other decode configurations, timed like the headline one: the
    Granite-20B TP = 4 shard and the unsharded Llama-70B MLP (TP = 1, whose
    117 MB GEMMs are large enough to stream near the HBM roofline), with the
    ordered and act-order MLPs, the ordered GEMMs' achieved GB/s, and at TP = 1
    an fp16 dense reference of the same shapes (torch.matmul on random fp16
    weights, hipBLASLt)."""
    import torch
    from paper_2402_04925_amd import inputs
    out = {}
    # these lines are reported, not the headline: at least 100 steps per timing,
    # since at TP = 1 a replay of 20 steps is a few hundred microseconds
    steps = max(steps, 100)
    for name in ("granite20b_tp4", "llama70b_tp1"):
        wl = inputs.WORKLOADS[name]
        st = Setup(wl, dev)
        N1 = wl.N1 // wl.tp
        K2 = wl.K2 // wl.tp
        dense = None
        if wl.tp == 1:
            g = torch.Generator(device=dev).manual_seed(5)
            dense = (torch.randn(wl.K1, N1, device=dev, generator=g).half() * 0.02,
                     torch.randn(K2, wl.N2, device=dev, generator=g).half() * 0.02)
        res = {}
        for M in wl.Ms:
            c = Calls(st, M, dev)
            mo, _ = capture_and_time([c.mlp(rep, "ordered") for rep in st.reps], steps, warmup, dev)
            ma, _ = capture_and_time([c.mlp(rep, "actorder") for rep in st.reps], steps, warmup, dev)
            g1, _ = capture_and_time([c.gemm(rep, 0, "ordered") for rep in st.reps], steps, warmup, dev)
            g2, _ = capture_and_time([c.gemm(rep, 1, "ordered") for rep in st.reps], steps, warmup, dev)
            g1g, _ = capture_and_time([c.gemm1_gather(rep) for rep in st.reps], steps, warmup, dev)
            b1 = gemm_bytes(M, wl.K1, N1, wl.G)
            b2 = gemm_bytes(M, K2, wl.N2, wl.G)
            gbs = (b1 + b2) / ((g1 + g2) * 1e-3) / 1e9
            flops = 2 * M * (wl.K1 * N1 + K2 * wl.N2)
            r = dict(ordered_mlp_us=round(mo * 1e3, 3), actorder_mlp_us=round(ma * 1e3, 3),
                     speedup_ordered_vs_actorder=round(ma / mo, 3),
                     ordered_gemm_us=[round(g1 * 1e3, 3), round(g2 * 1e3, 3)],
                     # GEMM1 as the MLP calls it (X[:, P1] gathered in the call), and
                     # what the MLP takes beyond that GEMM1 and GEMM2
                     ordered_gemm1_with_gather_us=round(g1g * 1e3, 3),
                     mlp_over_gathered_gemms_us=round((mo - g1g - g2) * 1e3, 3),
                     ordered_gemm_gbs=round(gbs, 1), ordered_gemm_hbm_frac=round(gbs / HBM_PEAK_GBS, 4),
                     ordered_mlp_tflops=round(flops / (mo * 1e-3) / 1e12, 2))
            if wl.tp == 1:
                m2, _ = capture_and_time([c.alg2_mlp(rep) for rep in st.reps], steps, warmup, dev)
                r["alg2_local_mlp_us"] = round(m2 * 1e3, 3)
                r["alg2_local_over_alg3"] = round(m2 / mo, 4)
                eprint(f"[bench] {name} M={M}: Alg. 2 local data flow {m2*1e3:.2f} us "
                       f"(Alg. 3 {mo*1e3:.2f} us, ratio {m2 / mo:.3f})")
            if dense is not None:
                X = c.X
                y1 = torch.empty(M, N1, dtype=torch.float16, device=dev)
                y2 = torch.empty(M, wl.N2, dtype=torch.float16, device=dev)

                def dense_mlp():
                    torch.matmul(X, dense[0], out=y1)
                    torch.matmul(y1, dense[1], out=y2)
                md, _ = capture_and_time([dense_mlp], steps, warmup, dev)
                r["fp16_dense_mlp_us"] = round(md * 1e3, 3)
                r["speedup_ordered_vs_fp16_dense"] = round(md / mo, 3)
            eprint(f"[bench] {name} M={M}: ordered mlp {mo*1e3:.2f} us (gemms {g1*1e3:.2f} + {g2*1e3:.2f} us, "
                   f"{gbs:.0f} GB/s), actorder mlp {ma*1e3:.2f} us"
                   + (f", fp16 dense mlp {r['fp16_dense_mlp_us']:.2f} us" if dense is not None else ""))
            res[str(M)] = r
            del c
        out[name] = dict(
            workload=f"{wl.name}: rank-0 TP-aware MLP shard, W1 {wl.K1}x{N1}, W2 {K2}x{wl.N2}, int4 G={wl.G}, fp16 X",
            weight_replicas=st.R, by_M=res)
        del st, dense
        torch.cuda.synchronize()
    return out


def bf16_line(dev, steps, warmup):
    """The headline workload (Llama-70B TP = 8 rank-0 shard) with bfloat16
    activations, scales and outputs: ordered and act-order MLPs and the
    ordered GEMMs' achieved GB/s at each M, timed like the fp16 line."""
    import torch
    from paper_2402_04925_amd import inputs
    wl = inputs.WORKLOADS["llama70b_tp8"]
    st = Setup(wl, dev, bf16=True)
    N1, K2 = wl.N1 // wl.tp, wl.K2 // wl.tp
    res = {}
    for M in wl.Ms:
        c = Calls(st, M, dev)
        mo, _ = capture_and_time([c.mlp(rep, "ordered") for rep in st.reps], steps, warmup, dev)
        ma, _ = capture_and_time([c.mlp(rep, "actorder") for rep in st.reps], steps, warmup, dev)
        g1, _ = capture_and_time([c.gemm(rep, 0, "ordered") for rep in st.reps], steps, warmup, dev)
        g2, _ = capture_and_time([c.gemm(rep, 1, "ordered") for rep in st.reps], steps, warmup, dev)
        gbs = (gemm_bytes(M, wl.K1, N1, wl.G) + gemm_bytes(M, K2, wl.N2, wl.G)) / ((g1 + g2) * 1e-3) / 1e9
        res[str(M)] = dict(ordered_mlp_us=round(mo * 1e3, 3), actorder_mlp_us=round(ma * 1e3, 3),
                           speedup_ordered_vs_actorder=round(ma / mo, 3),
                           ordered_gemm_us=[round(g1 * 1e3, 3), round(g2 * 1e3, 3)],
                           ordered_gemm_gbs=round(gbs, 1), ordered_gemm_hbm_frac=round(gbs / HBM_PEAK_GBS, 4))
        eprint(f"[bench] bf16 {wl.name} M={M}: ordered mlp {mo*1e3:.2f} us (gemms {g1*1e3:.2f} + {g2*1e3:.2f} us, "
               f"{gbs:.0f} GB/s), actorder mlp {ma*1e3:.2f} us")
        del c
    del st
    torch.cuda.synchronize()
    return dict(workload=f"{wl.name}: rank-0 TP-aware MLP shard, W1 {wl.K1}x{N1}, W2 {K2}x{wl.N2}, int4 G={wl.G}, "
                         f"bf16 X, scales and outputs", by_M=res)


def gated_line(dev, steps, warmup):
    """The gated form of the headline workload (Llama-70B TP = 8 rank 0:
    gate and up 8192 x 3584 each, down 3584 x 8192): tpdq_gated_mlp_shard on
    the ordered path (P2 folded into gate and up) and the act-order path, at
    each M, weights rotating over replicas of at least ROTATE_MIN_BYTES."""
    import ctypes
    import torch
    import paper_2402_04925_amd as tpdq
    from paper_2402_04925_amd import inputs
    wl = inputs.WORKLOADS["llama70b_tp8"]
    gate, up, down = inputs.make_gated_workload(wl)

    def dl(L):
        return tpdq.QuantWeight.from_tensors(
            torch.from_numpy(L.qweight).to(dev), torch.from_numpy(L.scales).to(dev),
            torch.from_numpy(L.qzeros).to(dev), torch.from_numpy(L.g_idx.astype(np.int32)).to(dev), L.G)

    dg, du, dd = dl(gate), dl(up), dl(down)
    P1, _, _, _, gf, do = tpdq.reorder(dg, dd)
    _, _, _, _, uf, _ = tpdq.reorder(du, dd)
    tp = wl.tp

    def dense(q, with_g):
        return tpdq.QuantWeight(q.qweight.contiguous(), q.scales.contiguous(), q.qzeros.contiguous(),
                                q.g_idx.contiguous() if with_g and q.g_idx is not None else None,
                                q.K, q.N, q.G, q.num_groups, q.layout)

    base = [dense(gf.column_shard(0, tp), False), dense(uf.column_shard(0, tp), False),
            dense(do.row_shard(0, tp, True), False), dense(dg.column_shard(0, tp), True),
            dense(du.column_shard(0, tp), True), dense(dd.row_shard(0, tp, False), True)]
    per = sum(t.qweight.numel() * 4 + t.scales.numel() * 2 + t.qzeros.numel() * 4 for t in base[:3])
    R = max(2, -(-ROTATE_MIN_BYTES // per))
    reps = [base] + [[tpdq.QuantWeight(q.qweight.clone(), q.scales.clone(), q.qzeros.clone(),
                                       q.g_idx.clone() if q.g_idx is not None else None,
                                       q.K, q.N, q.G, q.num_groups, q.layout) for q in base]
                     for _ in range(R - 1)]
    del dg, du, dd, gf, uf, do
    torch.cuda.synchronize()
    eprint(f"[bench] gated {wl.name}: {R} weight replicas of {per / 1e6:.1f} MB (ordered triple)")
    lib = tpdq._abi.lib()
    ws = tpdq.Workspace(dev)
    N1, K2 = wl.N1 // tp, wl.K2 // tp
    res = {}
    for M in wl.Ms:
        X = torch.from_numpy(inputs.make_x(wl, M)).to(dev)
        y1 = torch.empty(M, N1, dtype=torch.float16, device=dev)
        y2 = torch.empty(M, wl.N2, dtype=torch.float16, device=dev)

        def mk(rep, ordered):
            g, u, d = (rep[0], rep[1], rep[2]) if ordered else (rep[3], rep[4], rep[5])
            cg, cu, cd = g.c_struct(), u.c_struct(), d.c_struct()
            nb = lib.tpdq_workspace_bytes(tpdq.OP_GATED_MLP, M, ctypes.byref(cg), ctypes.byref(cd))
            buf = ws.get(nb)
            path = tpdq.PATH_ORDERED if ordered else tpdq.PATH_ACTORDER
            p1 = P1.data_ptr() if ordered else None

            def call():
                tpdq._abi.check(lib.tpdq_gated_mlp_shard(
                    X.data_ptr(), X.stride(0), M, p1, ctypes.byref(cg), ctypes.byref(cu), ctypes.byref(cd),
                    path, tpdq.FP16, y1.data_ptr(), y2.data_ptr(), buf.data_ptr(), buf.numel(),
                    torch.cuda.current_stream(dev).cuda_stream))
            return call

        mo, _ = capture_and_time([mk(rep, True) for rep in reps], steps, warmup, dev)
        ma, _ = capture_and_time([mk(rep, False) for rep in reps], steps, warmup, dev)
        b = 2 * shard_bytes(wl.K1, N1, wl.G) + M * wl.K1 * 2 + M * N1 * 2 + gemm_bytes(M, K2, wl.N2, wl.G)
        res[str(M)] = dict(ordered_mlp_us=round(mo * 1e3, 3), actorder_mlp_us=round(ma * 1e3, 3),
                           speedup_ordered_vs_actorder=round(ma / mo, 3),
                           ordered_mlp_gbs=round(b / (mo * 1e-3) / 1e9, 1))
        eprint(f"[bench] gated {wl.name} M={M}: ordered mlp {mo*1e3:.2f} us ({b / (mo * 1e-3) / 1e9:.0f} GB/s), "
               f"actorder mlp {ma*1e3:.2f} us")
    del reps, base
    torch.cuda.synchronize()
    return dict(workload=f"{wl.name} gated: rank-0 shard, gate and up {wl.K1}x{N1}, down {K2}x{wl.N2}, "
                         f"int4 G={wl.G}, fp16 X, Y1 = silu(X W_gate) * (X W_up)", weight_replicas=R, by_M=res)


def prefill_line(dev, steps=10):
    """The Llama-70B TP = 2 prefill shard (M = 2048): the ordered MLP shard
    and its two GEMMs (graph replay), TFLOP/s against the dense fp16 MFMA
    peak, and the act-order MLP for the speedup. Weights are not rotated:
    at this size the MFMA pipe, not HBM, bounds the GEMMs."""
    import torch
    from paper_2402_04925_amd import inputs
    wl = inputs.WORKLOADS["llama70b_tp2_prefill"]
    st = Setup(wl, dev, min_bytes=0)
    M = wl.Ms[0]
    c = Calls(st, M, dev)
    reps = st.reps[:1]
    ms, _ = capture_and_time([c.mlp(rep, "ordered") for rep in reps], steps, 2, dev)
    g1, _ = capture_and_time([c.gemm(rep, 0, "ordered") for rep in reps], steps, 2, dev)
    g2, _ = capture_and_time([c.gemm(rep, 1, "ordered") for rep in reps], steps, 2, dev)
    ma, _ = capture_and_time([c.mlp(rep, "actorder") for rep in reps], 2, 1, dev)
    N1 = wl.N1 // wl.tp
    K2 = wl.K2 // wl.tp
    flops = 2 * M * (wl.K1 * N1 + K2 * wl.N2)
    tf = flops / (ms * 1e-3) / 1e12
    tf_g = [2 * M * wl.K1 * N1 / (g1 * 1e-3) / 1e12, 2 * M * K2 * wl.N2 / (g2 * 1e-3) / 1e12]
    eprint(f"[bench] prefill M={M}: ordered mlp {ms*1e3:.1f} us ({tf:.0f} TFLOP/s), gemm1 {g1*1e3:.1f} us, "
           f"gemm2 {g2*1e3:.1f} us; actorder mlp {ma*1e3:.1f} us")
    del c, st
    torch.cuda.synchronize()
    # context: the same MLP as two dense fp16 GEMMs (torch.matmul, i.e. the
    # vendor GEMM library) on random fp16 weights of the shard's shapes, the
    # MFMA throughput a dense GEMM reaches on this part at these sizes
    gen = torch.Generator(device=dev)
    gen.manual_seed(1)
    Xd = torch.randn(M, wl.K1, generator=gen, device=dev).to(torch.float16)
    Wd1 = (torch.randn(wl.K1, N1, generator=gen, device=dev) * 0.01).to(torch.float16)
    Wd2 = (torch.randn(K2, wl.N2, generator=gen, device=dev) * 0.01).to(torch.float16)
    yd1 = torch.empty(M, N1, dtype=torch.float16, device=dev)
    yd2 = torch.empty(M, wl.N2, dtype=torch.float16, device=dev)

    def dense_mlp():
        torch.matmul(Xd, Wd1, out=yd1)
        torch.matmul(yd1, Wd2, out=yd2)
    md, _ = capture_and_time([dense_mlp], steps, 2, dev)
    tfd = flops / (md * 1e-3) / 1e12
    eprint(f"[bench] prefill M={M}: fp16 dense mlp (torch.matmul) {md*1e3:.1f} us ({tfd:.0f} TFLOP/s)")
    del Xd, Wd1, Wd2, yd1, yd2
    torch.cuda.synchronize()
    # the same ordered MLP with bf16 activations and scales (bf16 MFMA; the
    # weights are dequantized in fp32 and rounded to bf16)
    st = Setup(wl, dev, min_bytes=0, bf16=True)
    c = Calls(st, M, dev)
    mb, _ = capture_and_time([c.mlp(rep, "ordered") for rep in st.reps[:1]], steps, 2, dev)
    tfb = flops / (mb * 1e-3) / 1e12
    eprint(f"[bench] prefill M={M} bf16: ordered mlp {mb*1e3:.1f} us ({tfb:.0f} TFLOP/s)")
    del c, st
    torch.cuda.synchronize()
    return dict(
        workload=f"{wl.name}: rank-0 TP-aware MLP shard, W1 {wl.K1}x{N1}, W2 {K2}x{wl.N2}, "
                 f"int4 G={wl.G}, fp16 X, M={M}",
        bound="mfma", ordered_mlp_us=round(ms * 1e3, 1),
        ordered_gemm_us=[round(g1 * 1e3, 1), round(g2 * 1e3, 1)],
        tflops=round(tf, 1), gemm_tflops=[round(t, 1) for t in tf_g],
        peak_tflops=MFMA_F16_PEAK_TFLOPS, frac=round(tf / MFMA_F16_PEAK_TFLOPS, 4),
        actorder_mlp_us=round(ma * 1e3, 1), speedup_vs_actorder=round(ma / ms, 2),
        bf16_ordered_mlp_us=round(mb * 1e3, 1), bf16_tflops=round(tfb, 1),
        bf16_frac=round(tfb / MFMA_F16_PEAK_TFLOPS, 4),
        fp16_dense_mlp_us=round(md * 1e3, 1), fp16_dense_tflops=round(tfd, 1),
        ordered_over_fp16_dense_tflops=round(tf / tfd, 3),
        mfma_counters=read_mfma_util(),
        timing="HIP graph replay, events, median of 5")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="llama70b_tp8")
    ap.add_argument("--M", type=int, default=16)
    ap.add_argument("--sweep", default=None,
                    help="batch sizes reported alongside (default 1,2,4,8,16,32,64; with "
                         "--profile-run 1,4,16, the workload's own M set)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the Granite-20B TP=4 and Llama-70B TP=1 decode lines")
    ap.add_argument("--no-prefill", action="store_true",
                    help="skip the Llama-70B TP=2 prefill shard (M=2048, MFMA-bound) line")
    ap.add_argument("--no-bf16", action="store_true",
                    help="skip the bf16 line (the headline shard with bf16 activations and scales)")
    ap.add_argument("--no-gated", action="store_true",
                    help="skip the gated-MLP line (the headline shard with a gate projection)")
    ap.add_argument("--profile-run", action="store_true",
                    help="eager launches for rocprofv3 (kernel trace or counters); no JSON")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs one GPU's TP share only (the MLP shard of one rank); "
              f"--gpus {args.gpus} is not supported: collectives are outside this build.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2402_04925_amd import inputs

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    wl = inputs.WORKLOADS[args.workload]
    st = Setup(wl, dev)
    sweep = args.sweep if args.sweep is not None else ("1,4,16" if args.profile_run else "1,2,4,8,16,32,64")
    Ms = sorted(set([args.M] + [int(m) for m in sweep.split(",") if m]))
    if args.profile_run:
        profile_run(st, Ms, args.steps, dev)
        return

    results = {}
    for M in Ms:
        c = Calls(st, M, dev)
        r = {}
        for pname in ("ordered", "actorder", "actorder_global", "actorder_tiled"):
            ms, _ = capture_and_time([c.mlp(rep, pname) for rep in st.reps], args.steps,
                                     args.warmup, dev)
            g1, _ = capture_and_time([c.gemm(rep, 0, pname) for rep in st.reps], args.steps,
                                     args.warmup, dev)
            g2, _ = capture_and_time([c.gemm(rep, 1, pname) for rep in st.reps], args.steps,
                                     args.warmup, dev)
            r[pname] = dict(mlp_us=ms * 1e3, gemm1_us=g1 * 1e3, gemm2_us=g2 * 1e3)
            eprint(f"[bench] M={M} {pname}: mlp {ms*1e3:.2f} us, gemm1 {g1*1e3:.2f} us, gemm2 {g2*1e3:.2f} us")
        N1 = wl.N1 // wl.tp
        K2 = wl.K2 // wl.tp
        ng2_act = wl.K2 // wl.G
        b1 = gemm_bytes(M, wl.K1, N1, wl.G)
        b2 = gemm_bytes(M, K2, wl.N2, wl.G)
        b_mlp = b1 + b2 + wl.K1 * 4   # + P1 for the gather
        b1a = gemm_bytes(M, wl.K1, N1, wl.G, gidx=True)
        b2a = gemm_bytes(M, K2, wl.N2, wl.G, ng=ng2_act, gidx=True)
        flops = 2 * M * (wl.K1 * N1 + K2 * wl.N2)
        r["bytes"] = dict(gemm1=b1, gemm2=b2, mlp=b_mlp, gemm1_actorder=b1a, gemm2_actorder=b2a)
        r["flops"] = flops
        results[M] = r
        del c
        torch.cuda.synchronize()
    copy_gbs = copy_ceiling(dev)
    eprint(f"[bench] 1 GiB device copy: {copy_gbs:.0f} GB/s (read + write)")
    shard_bytes_w1 = wl.K1 * (wl.N1 // wl.tp) // 2
    copy_shard_us = copy_shard(dev, shard_bytes_w1, args.steps, args.warmup)
    eprint(f"[bench] device copy of {shard_bytes_w1 / 1e6:.1f} MB (one launch): {copy_shard_us:.2f} us")
    configs = None if args.no_configs else config_lines(dev, args.steps, args.warmup)
    prefill = None if args.no_prefill else prefill_line(dev)
    bf16 = None if args.no_bf16 else bf16_line(dev, args.steps, args.warmup)
    gated = None if args.no_gated else gated_line(dev, args.steps, args.warmup)

    M = args.M
    r = results[M]
    o_ = r["ordered"]
    b = r["bytes"]
    mlp_us = o_["mlp_us"]
    kern_us = o_["gemm1_us"] + o_["gemm2_us"]
    achieved = (b["gemm1"] + b["gemm2"]) / (kern_us * 1e-6) / 1e9
    traffic = read_traffic(wl.name, M)
    roof = dict(bound="hbm", achieved=round(achieved, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                frac=round(achieved / HBM_PEAK_GBS, 4), traffic=traffic,
                kernel="k_ordered (its GEMM1 and GEMM2 launches averaged)")
    cpu = cpu_host = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, M, st.L1, st.L2)
        cpu_host = cpu_detail()

    sweep = {}
    for m, rr in results.items():
        bb = rr["bytes"]
        sweep[str(m)] = dict(
            ordered_mlp_us=round(rr["ordered"]["mlp_us"], 3),
            actorder_mlp_us=round(rr["actorder"]["mlp_us"], 3),
            speedup_ordered_vs_actorder=round(rr["actorder"]["mlp_us"] / rr["ordered"]["mlp_us"], 3),
            actorder_global_mlp_us=round(rr["actorder_global"]["mlp_us"], 3),
            speedup_ordered_vs_actorder_global=round(rr["actorder_global"]["mlp_us"] / rr["ordered"]["mlp_us"], 3),
            actorder_global_gemm_us=[round(rr["actorder_global"]["gemm1_us"], 3),
                                     round(rr["actorder_global"]["gemm2_us"], 3)],
            actorder_tiled_mlp_us=round(rr["actorder_tiled"]["mlp_us"], 3),
            speedup_ordered_vs_actorder_tiled=round(rr["actorder_tiled"]["mlp_us"] / rr["ordered"]["mlp_us"], 3),
            actorder_tiled_gemm_us=[round(rr["actorder_tiled"]["gemm1_us"], 3),
                                    round(rr["actorder_tiled"]["gemm2_us"], 3)],
            ordered_gemm_us=[round(rr["ordered"]["gemm1_us"], 3), round(rr["ordered"]["gemm2_us"], 3)],
            actorder_gemm_us=[round(rr["actorder"]["gemm1_us"], 3), round(rr["actorder"]["gemm2_us"], 3)],
            ordered_mlp_gbs=round(bb["mlp"] / (rr["ordered"]["mlp_us"] * 1e-6) / 1e9, 1),
            ordered_gemm_gbs=round((bb["gemm1"] + bb["gemm2"]) /
                                   ((rr["ordered"]["gemm1_us"] + rr["ordered"]["gemm2_us"]) * 1e-6) / 1e9, 1),
            actorder_gemm_gbs=round((bb["gemm1_actorder"] + bb["gemm2_actorder"]) /
                                    ((rr["actorder"]["gemm1_us"] + rr["actorder"]["gemm2_us"]) * 1e-6) / 1e9, 1),
            ordered_tflops=round(rr["flops"] / (rr["ordered"]["mlp_us"] * 1e-6) / 1e12, 2),
        )
    out = dict(
        metric=METRIC, value=round(mlp_us, 3), unit="us", n_gpus=1, steps=args.steps,
        warmup=args.warmup, ms_per_step=round(mlp_us / 1e3, 6), higher_is_better=False,
        scaling="weak", vs_baseline=None, dtype="f16", data="synthetic",
        config=dict(workload=f"{wl.name}: rank-0 TP-aware MLP shard, W1 {wl.K1}x{wl.N1 // wl.tp}, "
                             f"W2 {wl.K2 // wl.tp}x{wl.N2}, int4 G={wl.G}, fp16 X, M={M}",
                    M=M, tp=wl.tp, path="ordered (Alg. 3)", weight_replicas=st.R,
                    timing="HIP graph replay, events, median of 5"),
        hbm_gbs=round(b["mlp"] / (mlp_us * 1e-6) / 1e9, 1),
        hbm_frac=round(b["mlp"] / (mlp_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
        tflops=round(r["flops"] / (mlp_us * 1e-6) / 1e12, 3),
        speedup_vs_actorder=round(r["actorder"]["mlp_us"] / mlp_us, 3),
        roofline=roof, cpu_baseline=cpu, cpu_detail=cpu_host, configs=configs, prefill=prefill, bf16=bf16, gated=gated,
        copy_1gib_gbs=round(copy_gbs, 1),
        copy_w1_shard=dict(bytes=shard_bytes_w1, us=round(copy_shard_us, 3),
                           gbs=round(2 * shard_bytes_w1 / (copy_shard_us * 1e-6) / 1e9, 1),
                           what="one device-copy launch of a buffer the size of the packed W1 shard "
                                "(read + write), graph-timed like the GEMMs"),
        roofline_frac_of_copy=round(achieved / copy_gbs, 4),
        sweep=sweep,
        paper_context="paper: up to 1.81x (Llama-70B) / 1.78x (Granite-20B) Alg. 3 vs Alg. 2 on "
                      "A100/H100 DGX, multi-GPU, communication included; not comparable",
    )
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
