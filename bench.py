#!/usr/bin/env python3
"""Benchmark of the propagate hot path on one MI355X.

Workload: the large power-law graph (Chung-Lu degree exponent 2.1, N=232,965,
~114.6M directed edges plus N self-loops, mean in-degree ~493), F=128 fp32
features. One step is one pass of the whole path on that graph, inputs
already resident in HBM:

    coo_to_csr -> degree (from the CSR row bounds) -> gcn_norm (CSR slot
    order, formed and written inside the propagate) + propagate
    (gcn_norm-weighted sum, CSR segment kernel) -> global mean pool

`value` is E*F of the step's propagate divided by the step time
(edges*features/s). The `roofline` object covers the dominant call, the
fused gcn_norm + propagate (its launches together), timed with HIP events on
the launch stream inside the timed steps: its bytes past L2 (rocprofv3
counters recorded below) against the gather ceiling the bandwidth probes
measure in the same run.
`cpu_baseline` times the oracle (single-threaded plain C loop) on a bounded
sample of the same workload, and (`all_cores`) the same sample split over the
host's cores, one unchanged oracle call per core. `detail` adds per-call times and the COO-vs-CSR,
fp32-vs-bf16 and sum-vs-mean comparison.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published peak

# Byte counters of the step's propagate call (pyg_gcn_propagate_blocked, fp32,
# two source blocks, no per-edge norms, on the large power-law graph) from
# rocprofv3 --pmc runs of this script (FETCH_SIZE, then WRITE_SIZE, then
# TCC_HIT_sum + TCC_MISS_sum; KiB / counts per call, summed over the call's
# five launches: d^-1/2, the row pre-scaling, the four windows, the long-row
# fix-up and the block fold; the first three calls of each run, the timed
# steps, before the detail calls), with FETCH_SIZE and WRITE_SIZE on a plain
# 1024 MiB device copy for scale; see profiles/propagate_c5_counters.md.
# They describe the sources with the recorded hash only: after any change to
# those sources the traffic field is reported as null.
COUNTERS = {
    "source_hash": "a2d2b7630495b08d",
    "fetch_kib": 12901985.6, "write_kib": 502042.8, "tcc_hit": 300259659.0, "tcc_miss": 210657761.3,
    "copy_mib": 1024, "copy_fetch_kib": 524320.3, "copy_write_kib": 1048576.0,
}
# everything that decides which kernels a propagate call launches and how
KERNEL_SOURCES = ["paper_1903_02428_amd/csrc/segment.hip", "paper_1903_02428_amd/csrc/common.hpp",
                  "paper_1903_02428_amd/csrc/api.hip", "paper_1903_02428_amd/csrc/gcn_norm.hip",
                  "paper_1903_02428_amd/binding.py"]


def source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic():
    """Bytes past L2 (fetched plus written) per propagate call from the
    recorded counters, scaled by the copy calibration; None if the sources
    changed since they were taken."""
    if COUNTERS["source_hash"] is None or source_hash() != COUNTERS["source_hash"]:
        return None
    ref_kib = COUNTERS["copy_mib"] * 1024.0
    fetch = COUNTERS["fetch_kib"] * ref_kib / COUNTERS["copy_fetch_kib"]
    write = COUNTERS["write_kib"] * ref_kib / COUNTERS["copy_write_kib"]
    return (fetch + write) * 1024.0


def measured_l2_hit():
    if COUNTERS["source_hash"] is None or source_hash() != COUNTERS["source_hash"] or not COUNTERS["tcc_hit"]:
        return None
    return COUNTERS["tcc_hit"] / (COUNTERS["tcc_hit"] + COUNTERS["tcc_miss"])


class Probe:
    """The bandwidth probes (libpyg_probe.so): a >= 1 GiB flush that evicts
    every L2 and the Infinity Cache, random 128-byte-line gathers with exactly
    known byte counts, and a streaming read."""

    def __init__(self, torch, dev, flush_bytes=1 << 30):
        import ctypes
        from paper_1903_02428_amd import build
        if not os.path.exists(build.PROBE_PATH):
            build.build_probe()
        lib = ctypes.CDLL(build.PROBE_PATH)
        u64, i32, u32, p = ctypes.c_uint64, ctypes.c_int, ctypes.c_uint32, ctypes.c_void_p
        lib.pyg_probe_sink_elems.argtypes, lib.pyg_probe_sink_elems.restype = [], ctypes.c_int64
        lib.pyg_probe_flush.argtypes, lib.pyg_probe_flush.restype = [p, u64, u32, p], i32
        lib.pyg_probe_gather.argtypes, lib.pyg_probe_gather.restype = [p, u64, i32, i32, i32, u64, u32, i32, i32, p,
                                                                        p], i32
        lib.pyg_probe_stream_read.argtypes, lib.pyg_probe_stream_read.restype = [p, u64, p, p], i32
        lib.pyg_probe_atomic.argtypes, lib.pyg_probe_atomic.restype = [p, u64, u64, u32, p], i32
        self.lib, self.torch, self.dev = lib, torch, dev
        self.flush_buf = torch.empty(flush_bytes, dtype=torch.uint8, device=dev)
        self.sink = torch.empty(int(lib.pyg_probe_sink_elems()), dtype=torch.int32, device=dev)
        self.salt = 0

    def _stream(self):
        import ctypes
        return ctypes.c_void_p(self.torch.cuda.current_stream(self.dev).cuda_stream)

    def flush(self):
        import ctypes
        self.salt += 1
        rc = self.lib.pyg_probe_flush(ctypes.c_void_p(self.flush_buf.data_ptr()), self.flush_buf.numel(),
                                      self.salt, self._stream())
        assert rc == 0, f"pyg_probe_flush: {rc}"

    def gather(self, buf, nbytes, line, parts, n, seed=1, in_flight=8, groups=2048, stride=1):
        import ctypes
        rc = self.lib.pyg_probe_gather(ctypes.c_void_p(buf.data_ptr()), nbytes, line, parts, stride, n, seed,
                                       in_flight, groups, ctypes.c_void_p(self.sink.data_ptr()), self._stream())
        assert rc == 0, f"pyg_probe_gather: {rc}"

    def atomic(self, buf, nbytes, n_ops, seed=1):
        import ctypes
        rc = self.lib.pyg_probe_atomic(ctypes.c_void_p(buf.data_ptr()), nbytes, n_ops, seed, self._stream())
        assert rc == 0, f"pyg_probe_atomic: {rc}"

    def stream_read(self, buf, nbytes):
        import ctypes
        rc = self.lib.pyg_probe_stream_read(ctypes.c_void_p(buf.data_ptr()), nbytes,
                                            ctypes.c_void_p(self.sink.data_ptr()), self._stream())
        assert rc == 0, f"pyg_probe_stream_read: {rc}"


def probe_ladder(probe, torch, dev, x_bytes):
    """Gather and stream rates of this GPU (GB/s of requested bytes, median
    of 5 launches). Random 128-byte lines from buffers of growing size, warm
    (each buffer touched once before timing): a buffer of x's size stays in
    the 256 MB Infinity Cache, so nearly every gather misses L2 and is served
    over the fabric from there; that rate is the ceiling of the propagate's
    traffic past L2. With parts = 8 each XCD draws from its own eighth (a 32
    MiB buffer then fits the eight 4 MB L2s). Streams: a cold 4 GiB read
    (HBM)."""
    res = {"unit": "GB/s", "line_bytes": 128, "gathers_per_launch": 1 << 26}
    n = 1 << 26
    sizes = [("16MiB", 16 << 20), ("32MiB", 32 << 20), ("64MiB", 64 << 20), ("x", x_bytes),
             ("256MiB", 256 << 20), ("1GiB", 1 << 30), ("4GiB", 4 << 30)]
    for name, nbytes in sizes:
        nbytes = nbytes // 128 * 128
        buf = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        buf.zero_()
        if name == "64MiB":  # 4 MiB of distinct lines per XCD: every 2nd / 4th line of an 8 / 16 MiB part
            for stride, big in ((2, 64 << 20), (4, 128 << 20)):
                b2 = torch.zeros(big, dtype=torch.uint8, device=dev)
                ms = timed(torch, lambda: probe.gather(b2, big, 128, 8, n, stride=stride), reps=5, warm=1)
                res[f"gather_4MiB_per_xcd_stride{stride}"] = n * 128 / (ms * 1e-3) / 1e9
                del b2
        for parts in ((1, 8) if nbytes <= (64 << 20) else (1,)):
            ms = timed(torch, lambda: probe.gather(buf, nbytes, 128, parts, n), reps=5, warm=1)
            res[f"gather_{name}" + ("_xcd_local" if parts == 8 else "")] = n * 128 / (ms * 1e-3) / 1e9
        if name == "x":
            ms = timed(torch, lambda: probe.gather(buf, nbytes, 64, 1, n), reps=5, warm=1)
            res["gather64_x"] = n * 64 / (ms * 1e-3) / 1e9
            # launch shapes: gathers in flight per lane x workgroups; the
            # best of them is the ceiling
            best = res["gather_x"]
            for u in (4, 8, 16):
                for groups in (1024, 2048, 4096, 8192):
                    ms = timed(torch, lambda: probe.gather(buf, nbytes, 128, 1, n, in_flight=u, groups=groups),
                               reps=5, warm=1)
                    r = n * 128 / (ms * 1e-3) / 1e9
                    res[f"gather_x_u{u}_g{groups}"] = r
                    best = max(best, r)
            res["gather_x_best"] = best
            # one 128-byte window of 512-byte rows: every 4th line; per XCD
            # an eighth of the rows (the pattern of an XCD-affine propagate)
            for parts in (1, 8):
                ms = timed(torch, lambda: probe.gather(buf, nbytes, 128, parts, n, stride=4), reps=5, warm=1)
                res["gather_x_stride4" + ("_xcd_local" if parts == 8 else "")] = n * 128 / (ms * 1e-3) / 1e9
            # float atomics (the COO kernel's scatter): 64-byte atomic requests per second
            ops = 1 << 24
            ms = timed(torch, lambda: probe.atomic(buf, nbytes, ops), reps=5, warm=1)
            res["atomic_x_requests_per_s"] = ops * 4 / (ms * 1e-3)
            res["atomic_x_float_adds_per_s"] = ops * 64 / (ms * 1e-3)
        if name == "4GiB":
            ms = timed(torch, lambda: probe.stream_read(buf, nbytes), reps=5, warm=1, flush=probe.flush)
            res["stream_read_4GiB_cold"] = nbytes / (ms * 1e-3) / 1e9
        del buf
        torch.cuda.empty_cache()
    res["x_bytes"] = x_bytes
    return res


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--chunk", type=int, default=0, help="edges per CSR work chunk (0 = library default)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-detail", action="store_true")
    ap.add_argument("--cpu-sample-rows", type=float, default=0.3, help="fraction of target rows in the CPU sample")
    ap.add_argument("--fig2", action="store_true",
                    help="run the degree sweep of the paper's Fig. 2 (gather/scatter vs CSR, forward and backward) "
                         "instead of the headline step; prints one JSON line per point")
    ap.add_argument("--backward-only", action="store_true",
                    help="only the gradient of the propagate on the large graph (one JSON object)")
    ap.add_argument("--configs-only", action="store_true",
                    help="only the throughput of the four smaller synthetic graphs (one JSON object)")
    ap.add_argument("--attention-only", action="store_true",
                    help="time only the attention calls (GAT softmax, attention sum) on the large graph")
    ap.add_argument("--gcn-layer-only", action="store_true",
                    help="time only the GCN layer (matrix-core X Theta, then propagate) on the large graph")
    ap.add_argument("--edge-features-only", action="store_true",
                    help="time only the edge-feature propagate (max(x_j + e, 0), F-dimensional e) on the large graph")
    ap.add_argument("--coo-only", action="store_true",
                    help="only the COO atomic kernel on the large graph (gcn-weighted sum and mean, fp32; one JSON "
                         "object), e.g. under rocprofv3 counters")
    ap.add_argument("--fig2-degrees", type=str, default="1,2,4,8,16,32,64,128,256,512",
                    help="average degrees of the Fig. 2 sweep (comma-separated)")
    ap.add_argument("--fig2-features", type=int, default=64)
    ap.add_argument("--fig2-runs", type=int, default=1000)
    ap.add_argument("--probe-only", action="store_true",
                    help="only the bandwidth probes (gather ladder, stream read; one JSON object)")
    ap.add_argument("--warm-detail", action="store_true",
                    help="time the large-graph detail calls back to back instead of after a 1 GiB flush each")
    ap.add_argument("--blocks", type=int, default=2,
                    help="source blocks of the step's propagate (pyg_csr_blocks_build + pyg_gcn_propagate_blocked); "
                         "0 = the unblocked CSR propagate (pyg_gcn_propagate)")
    ap.add_argument("--step-norms", action="store_true",
                    help="the blocked step's propagate also forms and writes every edge's gcn norm (by default it "
                         "applies d^-1/2 to the rows before and after the sum and forms no per-edge norm)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run one plain device copy of this size (for scaling rocprofv3 byte counters)")
    return ap.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def b_alg_csr(N, E, F, s_x, weighted=True, s_out=None):
    """Algorithmic bytes of one CSR propagate: row pointers, int32 columns,
    weights, one source-row gather per edge, one output write."""
    s_out = s_x if s_out is None else s_out
    return 8 * (N + 1) + 4 * E + (4 * E if weighted else 0) + E * F * s_x + N * F * s_out


def b_uniq_csr(N, E, F, s_x, weighted=True, s_out=None):
    """Compulsory bytes of one CSR propagate: every distinct byte once (x read
    once however often its rows are gathered)."""
    s_out = s_x if s_out is None else s_out
    return 8 * (N + 1) + 4 * E + (4 * E if weighted else 0) + N * F * s_x + N * F * s_out


def b_alg_coo(N, E, F, s_x, weighted=True):
    """Algorithmic bytes of one COO propagate: int64 source and target, weights,
    one gather per edge, one output write."""
    return 16 * E + (4 * E if weighted else 0) + E * F * s_x + N * F * s_x


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the multi-GPU design is described but not built)", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_1903_02428_amd as pyg
    import synth

    if not os.path.exists(pyg.library_path()):
        from paper_1903_02428_amd import build
        build.build()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.probe_only:
        probe = Probe(torch, dev)
        print(json.dumps({"workload": "bandwidth probes", "probe": probe_ladder(probe, torch, dev, 232965 * 128 * 4)}),
              flush=True)
        return
    if args.fig2:
        fig2_sweep(pyg, torch, synth, dev, args)
        return
    if args.configs_only:
        print(json.dumps({"workload": "the four smaller synthetic graphs", "configs": small_configs(pyg, torch, dev,
                                                                                                  args.seed),
                          "step_graph_small": step_graph_small(pyg, torch, dev, args.seed)}), flush=True)
        return

    t0 = time.time()
    c = synth.make_config(5, seed=args.seed)
    N, F = c["N"], c["F"]
    ei_np, x_np = c["edge_index_gcn"], c["x"]
    E = ei_np.shape[1]
    log(f"generated {c['name']}: N={N} E={E} F={F} in {time.time() - t0:.1f}s")

    global FLUSH
    probe = Probe(torch, dev)  # allocated first: the 1 GiB flush buffer
    if not args.warm_detail:
        FLUSH = probe.flush
    ei = torch.from_numpy(ei_np).to(dev)
    x = torch.from_numpy(x_np).to(dev)
    batch = torch.zeros(N, dtype=torch.int64, device=dev)  # one graph: whole-graph readout

    # all outputs and workspaces allocated once, outside the timed region
    deg = torch.empty(N, dtype=torch.int64, device=dev)
    norm = torch.empty(E, dtype=torch.float32, device=dev)
    csr = pyg.CSR(torch.empty(N + 1, dtype=torch.int64, device=dev), torch.empty(E, dtype=torch.int32, device=dev),
                  torch.empty(E, dtype=torch.int64, device=dev), None, N, E, args.chunk)
    csr_w = pyg.CSR(csr.rowptr, csr.col, csr.perm, norm, N, E, args.chunk)  # same CSR, weighted by the norms
    out = torch.empty_like(x)
    pooled = torch.empty(1, F, dtype=torch.float32, device=dev)
    lib = pyg.library()
    import ctypes
    sz = ctypes.c_size_t()
    lib.pyg_coo_to_csr_workspace(E, N, ctypes.byref(sz))
    ws_csr = torch.empty(sz.value, dtype=torch.uint8, device=dev)
    lib.pyg_gcn_norm_csr_workspace(N, ctypes.byref(sz))
    ws_norm = torch.empty(sz.value, dtype=torch.uint8, device=dev)
    lib.pyg_degree_workspace(E, N, ctypes.byref(sz))
    ws_deg = torch.empty(sz.value, dtype=torch.uint8, device=dev)
    ws_prop = torch.empty(pyg.propagate_workspace_bytes(x, E, "sum", "csr", args.chunk), dtype=torch.uint8, device=dev)
    lib.pyg_global_pool_workspace(0, N, F, 1, 1, ctypes.byref(sz))
    ws_pool = torch.empty(sz.value, dtype=torch.uint8, device=dev)

    if args.attention_only:
        pyg.coo_to_csr(ei, N, None, chunk=args.chunk, out=csr, workspace=ws_csr)
        print(json.dumps({"workload": "large power-law graph, GAT attention", "N": N, "E": E, "F": F,
                          "attention": attention(pyg, torch, x, ei, csr, N, E, F, dev)}), flush=True)
        return

    if args.gcn_layer_only:
        pyg.coo_to_csr(ei, N, None, chunk=args.chunk, out=csr, workspace=ws_csr)
        pyg.gcn_norm_csr(csr, out=norm, workspace=ws_norm)
        print(json.dumps({"workload": "large power-law graph, GCN layer", "N": N, "E": E, "F": F,
                          "gcn_layer": gcn_layer(pyg, torch, x, csr_w, N, E, F, dev)}), flush=True)
        return

    if args.backward_only:
        pyg.coo_to_csr(ei, N, None, chunk=args.chunk, out=csr, workspace=ws_csr)
        pyg.gcn_norm_csr(csr, out=norm, workspace=ws_norm)
        print(json.dumps({"workload": "large power-law graph, gradient of the propagate", "N": N, "E": E, "F": F,
                          "backward": backward_calls(pyg, torch, x, ei, csr_w, N, E, F, dev)}), flush=True)
        return

    if args.coo_only:
        w_coo = pyg.gcn_norm(ei, N)
        res = {}
        for aggr in ("sum", "mean"):
            ws = torch.empty(pyg.propagate_workspace_bytes(x, E, aggr, "coo"), dtype=torch.uint8, device=dev)
            ms = cold(torch, lambda: pyg.propagate(x, ei, w_coo, aggr=aggr, kernel="coo", out=out, workspace=ws),
                      reps=3)
            b = b_alg_coo(N, E, F, 4)
            res[f"coo-{aggr}-f32"] = {"ms": ms, "alg_GBps": b / (ms * 1e-3) / 1e9, "bytes": b,
                                      "atomics": E * F, "atomics_per_s": E * F / (ms * 1e-3)}
        print(json.dumps({"workload": "large power-law graph, COO atomic kernel", "N": N, "E": E, "F": F,
                          "coo": res}), flush=True)
        return

    if args.edge_features_only:
        pyg.coo_to_csr(ei, N, None, chunk=args.chunk, out=csr, workspace=ws_csr)
        print(json.dumps({"workload": "large power-law graph, edge-feature messages", "N": N, "E": E, "F": F,
                          "edge_features": edge_features(pyg, torch, x, ei, csr, N, E, F, dev)}), flush=True)
        return

    ws_gcn = torch.empty(pyg.gcn_propagate_workspace_bytes(x, csr), dtype=torch.uint8, device=dev)
    B = args.blocks
    if B:
        # the source-blocked CSR (virtual row b*N + i: the slots of target i
        # whose source lies in block b), built straight from the COO every step
        bcsr = pyg.CSRBlocks(torch.empty(B * N + 1, dtype=torch.int64, device=dev),
                             torch.empty(E, dtype=torch.int32, device=dev), None, None, N, E, B, args.chunk)
        ws_blk = torch.empty(pyg.coo_to_csr_blocked_workspace_bytes(E, N, B), dtype=torch.uint8, device=dev)
        ws_gcnb = torch.empty(pyg.gcn_propagate_blocked_workspace_bytes(x, bcsr), dtype=torch.uint8, device=dev)
        # the plain CSR of the detail calls, built once
        pyg.coo_to_csr(ei, N, None, chunk=args.chunk, out=csr, workspace=ws_csr)
    names = ["coo_to_csr", "degree", "gcn_norm+propagate", "global_pool"]
    ev = {n: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for n in names}
    times = {n: [] for n in names}

    def step(record):
        def mark(n, i):
            if record:
                ev[n][i].record()
        if B:
            mark("coo_to_csr", 0)  # stable sort by (source block, target, edge id)
            pyg.coo_to_csr_blocked(ei, N, B, None, chunk=args.chunk, out=bcsr, workspace=ws_blk)
            mark("coo_to_csr", 1)
            mark("degree", 0)  # the in-degree, read off the virtual rows' boundaries
            pyg.degree_csr_blocks(bcsr, out=deg)
            mark("degree", 1)
            # gcn_norm inside the propagate (pyg_gcn_propagate_blocked): d from
            # the blocked CSR, the rows scaled by d_j^-1/2 before the sum and by
            # d_i^-1/2 after it (with --step-norms: every edge's norm formed,
            # written to `norm` in blocked slot order and used by window 0),
            # one source block after another
            mark("gcn_norm+propagate", 0)
            pyg.gcn_propagate_blocked(x, None, bcsr, norm_out=norm if args.step_norms else None, out=out,
                                      workspace=ws_gcnb)
            mark("gcn_norm+propagate", 1)
        else:
            mark("coo_to_csr", 0)
            pyg.coo_to_csr(ei, N, None, chunk=args.chunk, out=csr, workspace=ws_csr)
            mark("coo_to_csr", 1)
            mark("degree", 0)  # the in-degree, read off the row boundaries the sort produced
            pyg.degree_csr(csr, out=deg)
            mark("degree", 1)
            # gcn_norm formed inside the propagate (pyg_gcn_propagate): the norms are
            # written to `norm` (CSR slot order) and summed with the gathered rows
            mark("gcn_norm+propagate", 0)
            pyg.gcn_propagate(x, csr, norm_out=norm, out=out, workspace=ws_gcn)
            mark("gcn_norm+propagate", 1)
        mark("global_pool", 0)
        pyg.global_pool(out, batch, 1, "mean", out=pooled, workspace=ws_pool)
        mark("global_pool", 1)

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    log(f"warmup {args.warmup} steps done")
    if args.copy_calibration_mib:
        n = args.copy_calibration_mib * (1 << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)  # reads and writes exactly copy_calibration_mib MiB
        torch.cuda.synchronize()
        del a, b
        log(f"calibration copy of {args.copy_calibration_mib} MiB done")

    wall = 0.0
    for k in range(args.steps):
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        step(True)
        torch.cuda.synchronize()
        wall += time.perf_counter() - t1
        for n in names:
            times[n].append(ev[n][0].elapsed_time(ev[n][1]))
    ms_per_step = wall / args.steps * 1e3
    log(f"timed {args.steps} steps: {ms_per_step:.3f} ms/step")
    out_step = out.clone()  # the step's output, for the sampled parity check after the detail calls

    t_prop = float(np.mean(times["gcn_norm+propagate"])) * 1e-3
    # the fused call: columns once per window, x rows gathered, the norms
    # formed (rowptr, dinv per node and per slot) and written, the output
    balg = b_alg_csr(N, E, F, 4, weighted=False) + 8 * N + 8 * E + 4 * E
    buniq = b_uniq_csr(N, E, F, 4, weighted=False) + 8 * N + 4 * E
    if B:  # B row pointers per target, and the fp32 partial rows written and folded
        balg += 8 * (B - 1) * N + 2 * B * N * F * 4
        buniq += 8 * (B - 1) * N
        if not args.step_norms:
            # no per-edge norm: no d^-1/2 gather per edge and no norm written,
            # the rows pre-scaled (read and written once) instead
            balg += -8 * E - 4 * E + 2 * N * F * 4
            buniq += -4 * E + N * F * 4
    value = E * F / (ms_per_step * 1e-3)
    ladder = probe_ladder(probe, torch, dev, N * F * 4)
    log("probe ladder done")
    traffic = measured_traffic()
    peak = ladder["gather_x_best"]
    achieved = traffic / t_prop / 1e9 if traffic is not None else None

    result = {
        "metric": "propagate throughput: edges·features/s and achieved HBM GB/s (% of peak)",
        "value": value,
        "unit": "edges·features/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "large power-law graph (Chung-Lu gamma=2.1), gcn_norm-weighted sum, CSR segment kernel"
                               + (f" over {B} source blocks" if B else ""),
                   "N": N, "E": E, "F": F, "seed": args.seed, "chunk": args.chunk or "default",
                   "source_blocks": B or None,
                   "step": ("coo_to_csr_blocked(B=%d: stable sort by source block, target, edge id)+degree(blocked "
                            "row bounds)+[gcn_norm inside the propagate: %s (sum, blocked csr, partials folded)]"
                            "+global_pool(mean)" % (B, "every edge's norm formed and written, window 0 weighted by "
                                                       "them, the other windows by pre-scaled rows"
                                                    if args.step_norms else
                                                    "d^-1/2 from the row bounds, rows scaled by d_j^-1/2 before "
                                                    "and d_i^-1/2 after the sum, no per-edge norm"))
                           if B else
                           "coo_to_csr+degree(csr row bounds)+[gcn_norm(csr order) formed and written inside the "
                           "propagate (sum, csr)]+global_pool(mean)"},
        "roofline": {"bound": "fabric", "achieved": achieved, "peak": peak, "unit": "GB/s",
                     "frac": achieved / peak if achieved is not None else None, "traffic": traffic,
                     "peak_source": "measured in this run: random 128-byte lines gathered from a buffer the size "
                                    "of x (%.1f MB), resident in the Infinity Cache (pyg_probe_gather)" %
                                    (N * F * 4 / 1e6),
                     "achieved_source": "bytes past L2 per call (FETCH_SIZE + WRITE_SIZE counters, copy-calibrated) "
                                        "/ the call's event time in the timed steps",
                     "l2_hit": measured_l2_hit(),
                     "kernel": ("pyg_gcn_propagate_blocked, fp32, B=%d: %s (virtual rows b*N+i, fp32 partial "
                                "rows), k_segment_fixup, k_block_fold (times d_i^-1/2)" %
                                (B, "k_segment over feature window 0 forming and writing the gcn norms, "
                                    "k_prescale_rows, k_segment over windows 1-3"
                                 if args.step_norms else "k_prescale_rows (d_j^-1/2 x), one k_segment over the four "
                                                         "windows")) if B else
                               "pyg_gcn_propagate, fp32: k_segment over feature window 0 forming and writing the "
                               "gcn norms, k_segment over windows 1-3 reading them, k_segment_fixup",
                     "unit_of_work": "one gcn_norm+propagate call over the whole graph",
                     "avg_call_ms": t_prop * 1e3,
                     "algorithmic": {"bytes_per_call": balg, "GBps": balg / t_prop / 1e9, "hbm_peak": HBM_PEAK_GBS,
                                     "frac_of_hbm": balg / t_prop / 1e9 / HBM_PEAK_GBS,
                                     "convention": ("every edge gathers its source row once (cache reuse counted "
                                                    "as traffic), plus rowptr, columns, d^-1/2 per node, the rows "
                                                    "pre-scaled, the fp32 partial rows written and read by the fold "
                                                    "and one output write")
                                                   if B and not args.step_norms else
                                                   ("every edge gathers its source row and its source's d^-1/2 once "
                                                    "(cache reuse counted as traffic), plus rowptr, columns, d^-1/2 "
                                                    "per node, the norms written and one output write"
                                                    + (", and the fp32 partial rows written and read by the fold"
                                                       if B else ""))},
                     "compulsory": {"bytes_per_call": buniq, "GBps": buniq / t_prop / 1e9,
                                    "frac_of_hbm": buniq / t_prop / 1e9 / HBM_PEAK_GBS,
                                    "convention": "every distinct byte once: rowptr, columns, d^-1/2, x, "
                                                  + ("the pre-scaled rows, " if B and not args.step_norms else
                                                     "norms written, ") + "output"}},
        "probe": ladder,
        "detail": {"per_call_ms": {n: float(np.mean(times[n])) for n in names},
                   "per_call_cache": "in-step: each call follows the previous call of the same step",
                   "detail_cache": "warm (back to back)" if args.warm_detail else
                                   "cold: a 1 GiB write before every timed call evicts L2 and the Infinity Cache",
                   "propagate_edges_features_per_s": E * F / t_prop,
                   "degree_from_coo_ms": cold(torch, lambda: pyg.degree(ei, N, out=deg, workspace=ws_deg)),
                   # the same two rows as separate calls (gcn_norm pass, then the weighted propagate)
                   "gcn_norm_csr_ms": cold(torch, lambda: pyg.gcn_norm_csr(csr, out=norm, workspace=ws_norm)),
                   "propagate_weighted_ms": cold(torch, lambda: pyg.propagate(x, csr=csr_w, aggr="sum", out=out,
                                                                              workspace=ws_prop)),
                   # the step's call forming and writing every edge's norm
                   "gcn_propagate_blocked_with_norms_ms": cold(torch, lambda: pyg.gcn_propagate_blocked(
                       x, None, bcsr, norm_out=norm, out=out, workspace=ws_gcnb)) if B else None,
                   # the step's calls without source blocks: the plain CSR build and
                   # pyg_gcn_propagate over it
                   "coo_to_csr_unblocked_ms": cold(torch, lambda: pyg.coo_to_csr(ei, N, None, chunk=args.chunk,
                                                                                 out=csr, workspace=ws_csr)),
                   "gcn_propagate_unblocked_ms": cold(torch, lambda: pyg.gcn_propagate(x, csr, norm_out=norm, out=out,
                                                                                       workspace=ws_gcn))},
    }

    if not args.no_detail:
        result["detail"]["variants"] = variants(pyg, torch, x, ei, csr_w, N, E, F, dev)
        result["detail"]["backward"] = backward_calls(pyg, torch, x, ei, csr_w, N, E, F, dev)
        result["detail"]["attention"] = attention(pyg, torch, x, ei, csr, N, E, F, dev)
        result["detail"]["gcn_layer"] = gcn_layer(pyg, torch, x, csr_w, N, E, F, dev)
        result["detail"]["edge_features"] = edge_features(pyg, torch, x, ei, csr, N, E, F, dev)
        result["detail"]["configs"] = small_configs(pyg, torch, dev, args.seed)
        result["detail"]["step_graph_small"] = step_graph_small(pyg, torch, dev, args.seed)
    if not (args.no_detail and args.no_cpu_baseline):
        import oracle
        w_ref = oracle.gcn_norm(ei_np, N).astype(np.float32)  # the oracle's own weights
    if not args.no_detail:
        result["detail"]["parity_sampled"] = sampled_parity(x_np, ei_np, w_ref, out_step, N)
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(x_np, ei_np, w_ref, N, F, args.cpu_sample_rows, args.seed)
    print(json.dumps(result), flush=True)


def fig2_sweep(pyg, torch, synth, dev, args):
    """The paper's Fig. 2 on this GPU: Erdos-Renyi graphs with 10,000 nodes and
    a swept average degree, edges in target order ("coalesced") or shuffled.
    Forward = sum propagate; backward = its gradient with respect to x, the
    propagate of grad_out over the transposed graph.
      gs   : the COO atomic kernel, straight from the given edge order, both ways;
      csr  : the CSR segment kernel; its forward uses a CSR built beforehand
             (preprocessing, timed separately as csr_build); its backward must
             first build the CSR of the transposed graph, which is timed inside.
    Times are totals of `runs` back-to-back runs (HIP events), in ms."""
    N, F, runs = 10_000, args.fig2_features, args.fig2_runs
    rng = np.random.default_rng([args.seed, 2])
    x = torch.randn(N, F, device=dev)
    g = torch.randn(N, F, device=dev)
    out = torch.empty_like(x)

    def total_ms(fn):
        fn()
        torch.cuda.synchronize()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for _ in range(runs):
            fn()
        e.record()
        e.synchronize()
        return s.elapsed_time(e)

    for deg in [int(d) for d in args.fig2_degrees.split(",")]:
        for coalesced in (True, False):
            ei_np = synth.erdos_renyi(N, deg, rng, coalesced)
            E = ei_np.shape[1]
            ei = torch.from_numpy(ei_np).to(dev)
            eit = torch.from_numpy(np.ascontiguousarray(ei_np[::-1])).to(dev)  # transposed graph
            csr = pyg.coo_to_csr(ei, N)
            csr_t = pyg.coo_to_csr(eit, N)
            ws_c = torch.empty(pyg.propagate_workspace_bytes(x, E, "sum", "coo"), dtype=torch.uint8, device=dev)
            ws_s = torch.empty(pyg.propagate_workspace_bytes(x, E, "sum", "csr"), dtype=torch.uint8, device=dev)
            import ctypes
            sz = ctypes.c_size_t()
            pyg.library().pyg_coo_to_csr_workspace(E, N, ctypes.byref(sz))
            ws_b = torch.empty(sz.value, dtype=torch.uint8, device=dev)
            rec = {
                "metric": "fig2_gs_vs_csr", "n_nodes": N, "avg_degree": deg, "E": E, "F": F, "runs": runs,
                "layout": "coalesced" if coalesced else "shuffled",
                "gs_fwd_ms": total_ms(lambda: pyg.propagate(x, ei, kernel="coo", out=out, workspace=ws_c)),
                "gs_bwd_ms": total_ms(lambda: pyg.propagate(g, eit, kernel="coo", out=out, workspace=ws_c)),
                "csr_fwd_ms": total_ms(lambda: pyg.propagate(x, csr=csr, kernel="csr", out=out, workspace=ws_s)),
                "csr_bwd_ms": total_ms(lambda: (pyg.coo_to_csr(eit, N, out=csr_t, workspace=ws_b),
                                                pyg.propagate(g, csr=csr_t, kernel="csr", out=out, workspace=ws_s))),
                "csr_build_ms": total_ms(lambda: pyg.coo_to_csr(ei, N, out=csr, workspace=ws_b)),
            }
            print(json.dumps(rec), flush=True)


FLUSH = None  # set to a Probe's flush: the large-graph detail calls are then timed cold


def timed(torch, fn, reps=10, warm=1, flush=None):
    """Median of `reps` calls, each bracketed by HIP events on the current
    stream. With `flush`, every timed call starts cold: the flush runs before
    it, outside the events."""
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for _ in range(warm):
        fn()
    ts = []
    for _ in range(reps):
        if flush is not None:
            flush()
        s.record()
        fn()
        e.record()
        e.synchronize()
        ts.append(s.elapsed_time(e))
    return float(np.median(ts))


def cold(torch, fn, reps=10, warm=1):
    """timed() with the 1 GiB flush before every call when a probe is loaded."""
    return timed(torch, fn, reps=reps, warm=warm, flush=FLUSH)


def step_graph_small(pyg, torch, dev, seed):
    """The whole step (coo_to_csr, degree, gcn_norm, propagate, mean pool) on
    the Cora-shaped graph and the mini-batch, run eagerly (one Python call
    per entry point) and as one captured HIP graph replayed: at these sizes
    the step is launch-bound, and the graph removes the host side of every
    call. Median of 20 after warm-up."""
    import ctypes
    import synth
    res = {}
    c1, c3 = synth.make_config(1, seed=seed), synth.make_config(3, seed=seed)
    for name, ei_np, N, x_np, batch_np, B in (("C1", c1["edge_index_gcn"], c1["N"], c1["x"],
                                               np.zeros(c1["N"], np.int64), 1),
                                              ("C3", c3["edge_index"], c3["N"], c3["x"], c3["batch"], c3["B"])):
        lib = pyg.library()
        E = ei_np.shape[1]
        ei, x, batch = (torch.from_numpy(np.ascontiguousarray(a)).to(dev) for a in (ei_np, x_np, batch_np))
        F = x.shape[1]
        csr = pyg.CSR(torch.empty(N + 1, dtype=torch.int64, device=dev), torch.empty(E, dtype=torch.int32, device=dev),
                      torch.empty(E, dtype=torch.int64, device=dev), None, N, E, 0)
        norm = torch.empty(E, dtype=torch.float32, device=dev)
        csr_w = pyg.CSR(csr.rowptr, csr.col, csr.perm, norm, N, E, 0)
        deg = torch.empty(N, dtype=torch.int64, device=dev)
        out = torch.empty_like(x)
        pooled = torch.empty(B, F, dtype=torch.float32, device=dev)
        sz = ctypes.c_size_t()

        def ws(fn, *a):
            fn(*a, ctypes.byref(sz))
            return torch.empty(max(sz.value, 1), dtype=torch.uint8, device=dev)
        ws_csr, ws_norm = ws(lib.pyg_coo_to_csr_workspace, E, N), ws(lib.pyg_gcn_norm_csr_workspace, N)
        ws_pool = ws(lib.pyg_global_pool_workspace, 0, N, F, B, 1)
        ws_prop = torch.empty(pyg.propagate_workspace_bytes(x, E, "sum", "csr", 0), dtype=torch.uint8, device=dev)

        def step():
            pyg.coo_to_csr(ei, N, None, out=csr, workspace=ws_csr)
            pyg.degree_csr(csr, out=deg)
            pyg.gcn_norm_csr(csr, out=norm, workspace=ws_norm)
            pyg.propagate(x, csr=csr_w, aggr="sum", out=out, workspace=ws_prop)
            pyg.global_pool(out, batch, B, "mean", out=pooled, workspace=ws_pool)
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            step()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()
        eager = timed(torch, step, reps=20, warm=50)
        replay = timed(torch, graph.replay, reps=20, warm=50)
        res[name] = {"N": N, "E": E, "F": F, "graphs": B, "eager_ms": eager, "graph_replay_ms": replay,
                     "speedup": eager / replay}
        del graph
    return res


def small_configs(pyg, torch, dev, seed):
    """Throughput on the four smaller synthetic graphs, for the runs each one
    names: the Cora-shaped and PubMed-shaped graphs (gcn_norm-weighted sum,
    mean, max; F = 64 and 500 for the latter), the mini-batch (unweighted
    sum, mean, max, then global sum/mean/max pooling of the sum), the kNN
    clouds (x_j - x_i with max and mean). Both kernels, each call timed alone
    (median of 10, after 50 warm-up calls that bring the clocks up) against its
    algorithmic bytes. At these sizes (0.2 to
    55 MB per call) launch latency and the chip's fill dominate."""
    import synth
    res = {}

    def rec(ms, b, E, F):
        return {"ms": ms, "edges_features_per_s": E * F / (ms * 1e-3), "alg_GBps": b / (ms * 1e-3) / 1e9,
                "hbm_frac": b / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS}

    runs = [(1, {}), (2, {"F": 64}), (2, {"F": 500}), (3, {}), (4, {})]
    for ci, kw in runs:
        c = synth.make_config(ci, seed=seed, **kw)
        N, F = c["N"], c["F"]
        name = f"C{ci}" + (f"-F{F}" if ci == 2 else "")
        ei_np = c["edge_index_gcn"] if ci in (1, 2) else c["edge_index"]
        E = ei_np.shape[1]
        ei = torch.from_numpy(ei_np).to(dev)
        x = torch.from_numpy(c["x"]).to(dev)
        weighted = ci in (1, 2)
        w = pyg.gcn_norm(ei, N) if weighted else None
        csr = pyg.coo_to_csr(ei, N, w)
        msg = "diff" if ci == 4 else "src"
        aggrs = ("max", "mean") if ci == 4 else ("sum", "mean", "max")
        out = torch.empty_like(x)
        am = torch.empty((N, F), dtype=torch.int64, device=dev)
        entry = {"N": N, "E": E, "F": F, "msg": msg, "weighted": weighted}
        for aggr in aggrs:
            for kernel in ("csr", "coo"):
                ws = torch.empty(pyg.propagate_workspace_bytes(x, E, aggr, kernel, csr.chunk), dtype=torch.uint8,
                                 device=dev)
                ms = timed(torch, lambda: pyg.propagate(x, ei, w, csr=csr if kernel == "csr" else None, aggr=aggr,
                                                        msg=msg, kernel=kernel, out=out,
                                                        argmax=am if aggr == "max" else None, workspace=ws),
                           warm=50)
                b = b_alg_csr(N, E, F, 4, weighted) if kernel == "csr" else b_alg_coo(N, E, F, 4, weighted)
                if msg == "diff":  # x_i: once per row (CSR), once per edge (COO)
                    b += N * F * 4 if kernel == "csr" else E * F * 4
                if aggr == "max":
                    b += N * F * 8  # argmax
                entry[f"{kernel}-{aggr}"] = rec(ms, b, E, F)
        if ci == 3:
            B = c["B"]
            batch = torch.from_numpy(c["batch"]).to(dev)
            h = pyg.propagate(x, csr=csr, aggr="sum")[0]
            pooled = torch.empty((B, F), device=dev)
            pam = torch.empty((B, F), dtype=torch.int64, device=dev)
            for aggr in ("sum", "mean", "max"):
                ms = timed(torch, lambda: pyg.global_pool(h, batch, B, aggr, out=pooled,
                                                          argmax=pam if aggr == "max" else None), warm=50)
                b = 8 * N + N * F * 4 + B * F * 4 + (B * F * 8 if aggr == "max" else 0)
                entry[f"pool-{aggr}"] = {"ms": ms, "alg_GBps": b / (ms * 1e-3) / 1e9,
                                         "hbm_frac": b / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS}
        res[name] = entry
    return res


def backward_calls(pyg, torch, x, ei, csr_w, N, E, F, dev):
    """The gradient of the propagate on the same graph (fp32): gcn-weighted
    sum with the weight gradient (in COO edge order, and in CSR slot order),
    mean, and max routed through the forward's argmax. The reversed CSR (with the weights) is preprocessing,
    built once. Algorithmic bytes: grad_x as the propagate over the reversed
    graph; grad_w one g row per target row, one x gather per edge, columns,
    the slot -> edge permutation and the weight written; max: argmax, g and
    one source id, x read and grad_x added per output element."""
    w_coo = torch.empty_like(csr_w.weight)  # the weights in COO order
    w_coo[csr_w.perm] = csr_w.weight
    csr_t = pyg.coo_to_csr(pyg.reverse_edges(ei), N, w_coo, chunk=csr_w.chunk)
    plain = pyg.CSR(csr_w.rowptr, csr_w.col, csr_w.perm, None, N, E, csr_w.chunk)
    plain_t = pyg.CSR(csr_t.rowptr, csr_t.col, csr_t.perm, None, N, E, csr_t.chunk)
    gen = torch.Generator(device=dev)
    gen.manual_seed(17)
    g = torch.randn(N, F, device=dev, generator=gen)
    rp = 8 * (N + 1)
    res = {}

    def rec(ms, b):
        return {"ms": ms, "alg_GBps": b / (ms * 1e-3) / 1e9, "hbm_frac": b / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                "bytes": b, "edges_features_per_s": E * F / (ms * 1e-3)}

    ms = cold(torch, lambda: pyg.propagate_backward(g, x, ei, w_coo, csr=csr_w, csr_t=csr_t, aggr="sum",
                                                     need_grad_w=True), reps=5)
    res["sum-weighted-grad_x+grad_w"] = rec(ms, b_alg_csr(N, E, F, 4) + rp + 4 * E + 8 * E + N * F * 4 + E * F * 4
                                           + 4 * E)
    # grad_w in CSR slot order (the order of the CSR's weights): no scatter through perm
    ms = cold(torch, lambda: pyg.propagate_backward(g, x, ei, w_coo, csr=csr_w, csr_t=csr_t, aggr="sum",
                                                     need_grad_w=True, w_order="csr"), reps=5)
    res["sum-weighted-grad_x+grad_w-csr-order"] = rec(ms, b_alg_csr(N, E, F, 4) + rp + 4 * E + N * F * 4
                                                     + E * F * 4 + 4 * E)
    ms = cold(torch, lambda: pyg.propagate_backward(g, x, ei, None, csr=plain, csr_t=plain_t, aggr="mean"), reps=5)
    res["mean-grad_x"] = rec(ms, b_alg_csr(N, E, F, 4, weighted=False) + rp + 2 * N * F * 4)
    _, am = pyg.propagate(x, csr=plain, aggr="max")
    ms = cold(torch, lambda: pyg.propagate_backward(g, x, ei, None, csr=plain, csr_t=plain_t, aggr="max",
                                                     argmax=am), reps=5)
    res["max-grad_x"] = rec(ms, N * F * (8 + 4 + 8 + 4) + N * F * 4)
    del csr_t, plain_t, g, am, w_coo
    torch.cuda.empty_cache()
    return res


def variants(pyg, torch, x, ei, csr, N, E, F, dev):
    """Propagate-only times: CSR vs COO, fp32 vs bf16 storage, sum vs mean."""
    xb = x.to(torch.bfloat16)
    norm = pyg.gcn_norm(ei, N)  # the same norms in COO order (equal bit for bit), for the COO kernel
    res = {}
    for dtname, xx, s in (("f32", x, 4), ("bf16", xb, 2)):
        o = torch.empty_like(xx)
        for aggr in ("sum", "mean"):
            for kernel in ("csr", "coo"):
                ws = torch.empty(pyg.propagate_workspace_bytes(xx, E, aggr, kernel, csr.chunk), dtype=torch.uint8,
                                 device=dev)
                ms = cold(torch, lambda: pyg.propagate(xx, ei, norm, csr=csr if kernel == "csr" else None, aggr=aggr,
                                                        kernel=kernel, out=o, workspace=ws))
                b = b_alg_csr(N, E, F, s) if kernel == "csr" else b_alg_coo(N, E, F, s)
                res[f"{kernel}-{aggr}-{dtname}"] = {"ms": ms, "edges_features_per_s": E * F / (ms * 1e-3),
                                                   "alg_GBps": b / (ms * 1e-3) / 1e9,
                                                   "hbm_frac": b / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS}
    # the source-blocked form (block-major virtual rows, fp32 partial rows
    # folded): regrouping a built CSR, building it straight from the COO,
    # and the gcn-weighted sum over it
    for B in (2, 4, 8):
        bc = pyg.csr_blocks(csr, B)
        res[f"csr_blocks_build-B{B}"] = {"ms": cold(torch, lambda: pyg.csr_blocks(csr, B, out=bc))}
        bd = pyg.coo_to_csr_blocked(ei, N, B)
        res[f"coo_to_csr_blocked-B{B}"] = {"ms": cold(torch, lambda: pyg.coo_to_csr_blocked(ei, N, B, out=bd))}
        del bd
        for dtname, xx, s in (("f32", x, 4), ("bf16", xb, 2)):
            o = torch.empty_like(xx)
            ws = torch.empty(pyg.propagate_blocked_workspace_bytes(xx, bc, "sum"), dtype=torch.uint8, device=dev)
            ms = cold(torch, lambda: pyg.propagate_blocked(xx, bc, "sum", out=o, workspace=ws))
            b = b_alg_csr(N, E, F, s) + 8 * B * N
            res[f"blocked-B{B}-sum-{dtname}"] = {"ms": ms, "edges_features_per_s": E * F / (ms * 1e-3),
                                                 "alg_GBps": b / (ms * 1e-3) / 1e9,
                                                 "hbm_frac": b / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS}
            del ws
        del bc
        torch.cuda.empty_cache()
    return res


def attention(pyg, torch, x, ei, csr, N, E, F, dev, H=8):
    """GAT-style attention on the same graph: H heads of C = F / H columns.
    Times the fused score+softmax call, the attention-weighted sum (fp32 and
    bf16 rows), the softmax forward from stored scores and its backward, and
    the backward of the attention sum and of the scores, each with its
    algorithmic bytes (unique bytes read and written once; gathered rows
    counted once per edge, as for the propagate)."""
    gen = torch.Generator(device=dev)
    gen.manual_seed(7)
    a_src = torch.randn(N, H, device=dev, generator=gen)
    a_dst = torch.randn(N, H, device=dev, generator=gen)
    alpha = torch.empty(E, H, device=dev)
    scores = torch.randn(E, H, device=dev, generator=gen)
    grad = torch.randn(E, H, device=dev, generator=gen)
    gs = torch.empty(E, H, device=dev)
    ws_sm = pyg.binding._softmax_ws(csr, H, None)
    rp = 8 * (N + 1)

    def rec(ms, b):
        return {"ms": ms, "alg_GBps": b / (ms * 1e-3) / 1e9, "hbm_frac": b / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                "bytes": b}

    res = {"heads": H, "channels_per_head": F // H}
    ms = cold(torch, lambda: pyg.gat_softmax(a_src, a_dst, csr, 0.2, "csr", out=alpha, workspace=ws_sm))
    res["gat_softmax"] = rec(ms, rp + 4 * E + 4 * E * H + 8 * N * H)
    ms = cold(torch, lambda: pyg.segment_softmax(scores, csr, "csr", out=gs, workspace=ws_sm))
    res["segment_softmax"] = rec(ms, rp + 8 * E * H)
    ms = cold(torch, lambda: pyg.segment_softmax_backward(alpha, grad, csr, "csr", out=gs, workspace=ws_sm))
    res["segment_softmax_backward"] = rec(ms, rp + 12 * E * H)
    for dtname, xx, sz in (("f32", x, 4), ("bf16", x.to(torch.bfloat16), 2)):
        o = torch.empty_like(xx)
        ws = torch.empty(pyg.binding._size(pyg.library().pyg_propagate_heads_workspace, pyg.binding.DTYPE[xx.dtype],
                                           N, H, F // H, E, csr.chunk), dtype=torch.uint8, device=dev)
        ms = cold(torch, lambda: pyg.propagate_heads(xx, csr, alpha, H, out=o, workspace=ws))
        r = rec(ms, rp + 4 * E + 4 * E * H + E * F * sz + N * F * sz)
        r["edges_features_per_s"] = E * F / (ms * 1e-3)
        res[f"propagate_heads_{dtname}"] = r
    layer = res["gat_softmax"]["ms"] + res["propagate_heads_f32"]["ms"]
    res["attention_layer_f32"] = {"ms": layer, "edges_features_per_s": E * F / (layer * 1e-3)}

    # Backward. The reversed CSR is part of the graph preprocessing (built
    # once per graph), not of the timed calls.
    csr_t = pyg.coo_to_csr(pyg.reverse_edges(ei), N, chunk=csr.chunk)
    map_t = pyg.csr_transpose_map(csr, csr_t)
    ws_map = torch.empty(pyg.binding._size(pyg.library().pyg_csr_transpose_map_workspace, E), dtype=torch.uint8,
                         device=dev)
    ms = cold(torch, lambda: pyg.csr_transpose_map(csr, csr_t, out=map_t, workspace=ws_map))
    res["csr_transpose_map"] = rec(ms, 16 * E + 4 * E)  # both permutations in, the map out
    tmap = 4 * E  # the transpose map (slot of csr for each slot of csr_t)
    g_alpha = torch.empty(E, H, device=dev)
    for dtname, xx, sz in (("f32", x, 4), ("bf16", x.to(torch.bfloat16), 2)):
        g = torch.randn(N, F, device=dev, generator=gen).to(xx.dtype)
        gx = torch.empty_like(g)
        wsb = torch.empty(pyg.binding._size(pyg.library().pyg_propagate_heads_backward_workspace,
                                            pyg.binding.DTYPE[xx.dtype], N, H, F // H, E, csr_t.chunk),
                          dtype=torch.uint8, device=dev)
        ms = cold(torch, lambda: pyg.propagate_heads_backward(g, xx, csr, csr_t, alpha, H, workspace=wsb,
                                                               out=(gx, g_alpha), map_t=map_t))
        # grad_x: the attention sum over the reversed graph; grad_alpha: per
        # edge and head a dot product of a gathered x row block with g's row.
        b = 2 * rp + 8 * E + tmap + 4 * E * H + 4 * E * H + E * F * sz + N * F * sz \
            + E * F * sz + N * F * sz
        r = rec(ms, b)
        r["edges_features_per_s"] = E * F / (ms * 1e-3)
        res[f"propagate_heads_backward_{dtname}"] = r
    outs = (torch.empty(N, H, device=dev), torch.empty(N, H, device=dev))
    wsg = torch.empty(pyg.binding._size(pyg.library().pyg_gat_scores_backward_workspace, N, H, E, csr_t.chunk),
                      dtype=torch.uint8, device=dev)
    ms = cold(torch, lambda: pyg.gat_scores_backward(a_src, a_dst, csr, csr_t, grad, 0.2, workspace=wsg, out=outs,
                                                      map_t=map_t))
    res["gat_scores_backward"] = rec(ms, 2 * rp + 4 * E + tmap + 4 * E * H + 4 * E * H + 8 * N * H + 8 * N * H)
    back = res["segment_softmax_backward"]["ms"] + res["propagate_heads_backward_f32"]["ms"] \
        + res["gat_scores_backward"]["ms"]
    res["attention_layer_backward_f32"] = {"ms": back, "edges_features_per_s": E * F / (back * 1e-3)}
    return res


def gcn_layer(pyg, torch, x, csr_w, N, E, F, dev, Fo=128):
    """One GCN layer on the same graph in bf16 storage: X Theta on the matrix
    cores (bf16 operands, fp32 accumulation, bf16 out), then the
    gcn_norm-weighted CSR propagate of the result. Theta ~ N(0, 1/F). The
    same layer in fp32 (fp32 operands and output) beside it."""
    gen = torch.Generator(device=dev)
    gen.manual_seed(11)
    xb = x.to(torch.bfloat16)
    theta = (torch.randn(F, Fo, device=dev, generator=gen) / F ** 0.5).to(torch.bfloat16)
    h = torch.empty(N, Fo, dtype=torch.bfloat16, device=dev)
    o = torch.empty_like(h)
    ws_d = torch.empty(pyg.binding._size(pyg.library().pyg_dense_transform_workspace, F, Fo), dtype=torch.uint8,
                       device=dev)
    ws_p = torch.empty(pyg.propagate_workspace_bytes(h, E, "sum", "csr", csr_w.chunk), dtype=torch.uint8, device=dev)
    t_d = cold(torch, lambda: pyg.dense_transform(xb, theta, torch.bfloat16, out=h, workspace=ws_d))
    t_p = cold(torch, lambda: pyg.propagate(h, csr=csr_w, aggr="sum", out=o, workspace=ws_p))

    def layer():
        pyg.dense_transform(xb, theta, torch.bfloat16, out=h, workspace=ws_d)
        pyg.propagate(h, csr=csr_w, aggr="sum", out=o, workspace=ws_p)
    t_l = cold(torch, layer)
    bytes_d = N * F * 2 + F * Fo * 2 + N * Fo * 2
    flops = 2.0 * N * F * Fo
    # the same layer in fp32 (fp32 operands on the fp32 matrix-core path, the same Theta values)
    theta32 = theta.float()
    h32 = torch.empty(N, Fo, dtype=torch.float32, device=dev)
    o32 = torch.empty_like(h32)
    ws_p32 = torch.empty(pyg.propagate_workspace_bytes(h32, E, "sum", "csr", csr_w.chunk), dtype=torch.uint8,
                         device=dev)
    t_d32 = cold(torch, lambda: pyg.dense_transform(x, theta32, torch.float32, out=h32, workspace=ws_d))

    def layer32():
        pyg.dense_transform(x, theta32, torch.float32, out=h32, workspace=ws_d)
        pyg.propagate(h32, csr=csr_w, aggr="sum", out=o32, workspace=ws_p32)
    t_l32 = cold(torch, layer32)
    bytes_d32 = N * F * 4 + F * Fo * 4 + N * Fo * 4
    return {"F_in": F, "F_out": Fo, "dtype": "bf16 storage, fp32 accumulation",
            "dense_transform": {"ms": t_d, "alg_GBps": bytes_d / (t_d * 1e-3) / 1e9,
                                "hbm_frac": bytes_d / (t_d * 1e-3) / 1e9 / HBM_PEAK_GBS,
                                "TFLOPs": flops / (t_d * 1e-3) / 1e12, "mfma_bf16_frac": flops / (t_d * 1e-3) / 2.5e15,
                                "bytes": bytes_d},
            "propagate_bf16": {"ms": t_p, "alg_GBps": b_alg_csr(N, E, Fo, 2) / (t_p * 1e-3) / 1e9},
            "layer": {"ms": t_l, "edges_features_per_s": E * Fo / (t_l * 1e-3)},
            "dense_transform_f32": {"ms": t_d32, "alg_GBps": bytes_d32 / (t_d32 * 1e-3) / 1e9,
                                    "hbm_frac": bytes_d32 / (t_d32 * 1e-3) / 1e9 / HBM_PEAK_GBS,
                                    "TFLOPs": flops / (t_d32 * 1e-3) / 1e12,
                                    "mfma_f32_frac": flops / (t_d32 * 1e-3) / 157.3e12, "bytes": bytes_d32},
            "layer_f32": {"ms": t_l32, "edges_features_per_s": E * Fo / (t_l32 * 1e-3)}}


def edge_features(pyg, torch, x, ei, csr, N, E, F, dev):
    """Propagate with an F-dimensional feature on every edge (GINE-style
    max(x_j + e, 0), sum): the CSR kernel with the features in CSR slot
    order (streamed once, coalesced) and the COO atomic kernel with them in
    COO order, and the backward of the CSR call in both dtypes. Algorithmic
    bytes: the plain propagate's plus E*F*s."""
    gen = torch.Generator(device=dev)
    gen.manual_seed(13)
    res = {"msg": "max(x_j + e, 0)", "aggr": "sum"}
    csr_t = pyg.coo_to_csr(pyg.reverse_edges(ei), N, chunk=csr.chunk)
    map_t = pyg.csr_transpose_map(csr, csr_t)
    for dtname, dt, sz in (("f32", torch.float32, 4), ("bf16", torch.bfloat16, 2)):
        xx = x.to(dt)
        ea = torch.randn(E, F, device=dev, generator=gen).to(dt)
        o = torch.empty_like(xx)
        kernels = (("csr", "csr"), ("coo", "coo")) if dt == torch.float32 else (("csr", "csr"),)
        for kernel, order in kernels:
            ws = torch.empty(pyg.propagate_workspace_bytes(xx, E, "sum", kernel, csr.chunk), dtype=torch.uint8,
                             device=dev)
            ms = cold(torch, lambda: pyg.propagate_edge(xx, ea, ei, csr if kernel == "csr" else None, "edge_relu",
                                                         "sum", kernel, order, out=o, workspace=ws), reps=5)
            b = (b_alg_csr(N, E, F, sz, weighted=False) if kernel == "csr" else b_alg_coo(N, E, F, sz, weighted=False))
            b += E * F * sz
            res[f"{kernel}-{dtname}"] = {"ms": ms, "alg_GBps": b / (ms * 1e-3) / 1e9,
                                         "hbm_frac": b / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, "bytes": b,
                                         "edges_features_per_s": E * F / (ms * 1e-3)}
        # the backward of the same call: grad_x over the reversed graph, edge
        # rows reached through the transpose map, and grad_e
        g = torch.randn(N, F, device=dev, generator=gen).to(dt)
        ws = torch.empty(pyg.binding._size(pyg.library().pyg_propagate_edge_backward_workspace,
                                           pyg.binding.DTYPE[dt], N, F, E, pyg.binding.MSG["edge_relu"],
                                           pyg.binding.AGGR["sum"], csr_t.chunk), dtype=torch.uint8, device=dev)
        ms = cold(torch, lambda: pyg.propagate_edge_backward(g, xx, ea, csr, "edge_relu", "sum", "csr",
                                                              csr_t=csr_t, map_t=map_t, workspace=ws), reps=5)
        rp = 8 * (N + 1)
        # grad_x: columns and map, one gathered g row, one edge row per
        # edge, the row's own x and the output; grad_e: columns, g per
        # row, one x gather, one edge row in and one out per edge
        b = (rp + 8 * E + 2 * E * F * sz + 2 * N * F * sz) + (rp + 4 * E + N * F * sz + 3 * E * F * sz)
        res[f"backward-csr-{dtname}"] = {"ms": ms, "alg_GBps": b / (ms * 1e-3) / 1e9,
                                         "hbm_frac": b / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, "bytes": b,
                                         "edges_features_per_s": E * F / (ms * 1e-3)}
        del g, ws
        del ea
        torch.cuda.empty_cache()
    del csr_t, map_t
    return res


def sampled_parity(x_np, ei_np, w_ref, out, N, rows=200):
    """The step's output (device gcn_norm -> CSR -> propagate) on a few sampled
    rows against the oracle chain (oracle gcn_norm -> oracle propagate)."""
    import oracle
    rng = np.random.default_rng(123)
    sample = rng.choice(N, rows, replace=False)
    keep = np.isin(ei_np[1], sample)
    sub = ei_np[:, keep]
    w = w_ref[keep]
    ref, _, sabs = oracle.propagate(x_np, sub, w, aggr="sum")
    got = out.cpu().numpy()[sample].astype(np.float64)
    bound = 1e-5 * sabs[sample] + 1e-6
    ratio = float((np.abs(got - ref[sample]) / bound).max())
    return {"rows": rows, "worst_error_over_bound": ratio, "ok": ratio <= 1.0}


def cpu_baseline(x_np, ei_np, w_ref, N, F, frac, seed):
    """The oracle (single-threaded plain C loop, fp64 accumulation) timed on a
    bounded sample: all edges into a random fraction of the target rows. Beside
    it, the same sample over all the host's cores: the sampled rows split into
    one group per core, the unchanged oracle run on every group at once (one
    thread each; the foreign call releases the interpreter lock)."""
    import oracle
    from concurrent.futures import ThreadPoolExecutor
    rng = np.random.default_rng([seed, 99])
    rows = rng.choice(N, int(N * frac), replace=False)
    keep = np.isin(ei_np[1], rows)
    sub = np.ascontiguousarray(ei_np[:, keep])
    w = w_ref[keep]
    Es = sub.shape[1]
    t = time.perf_counter()
    oracle.propagate(x_np, sub, w, aggr="sum")
    dt = time.perf_counter() - t
    cores = min(16, len(os.sched_getaffinity(0)))
    groups = np.array_split(np.sort(rows), cores)
    parts = []
    for g in groups:
        k = np.isin(sub[1], g)
        parts.append((np.ascontiguousarray(sub[:, k]), np.ascontiguousarray(w[k])))
    oracle.load()
    with ThreadPoolExecutor(cores) as ex:
        t = time.perf_counter()
        list(ex.map(lambda pw: oracle.propagate(x_np, pw[0], pw[1], aggr="sum")[0].shape, parts))
        dt_all = time.perf_counter() - t
    return {"value": Es * F / dt, "unit": "edges·features/s", "cores": 1, "kind": "oracle",
            "sample": f"gcn_norm-weighted sum over the {Es} edges into {len(rows)} random target rows "
                      f"({frac:.0%} of rows) of the same graph, F={F}, {dt:.1f}s",
            "host": platform.processor() or platform.machine(), "host_cpus": os.cpu_count(),
            "all_cores": {"value": Es * F / dt_all, "unit": "edges·features/s", "cores": cores,
                          "sample": f"the same edges, the target rows split into {cores} groups, one oracle "
                                    f"call per group on its own thread, {dt_all:.2f}s"}}


if __name__ == "__main__":
    main()
