#!/usr/bin/env python3
"""Benchmark of the LUT mpGEMM hot path on one MI355X.

A step is one pass of the whole hot path over one batch: INT8 quantization of the
activations, the table precompute and the bit-serial LUT mpGEMM with its
epilogue.  The headline step runs it as one kernel (lutgemm_mpgemm_fused: each
workgroup builds its tables in LDS); the same step as two calls
(lutgemm_precompute + lutgemm_mpgemm, tables through HBM) is reported beside it
and gives bitwise the same output.  Weight packing is offline and not timed.  Inputs are resident in HBM when the
timed region starts; every step reads a different copy of the packed weights
from a rotation set of at least 1 GiB (four times the 256 MB Infinity Cache),
so weights stream from HBM rather than from a cache.

Prints ONE JSON line.  ``value`` is effective TOPS (2 M N K / time per step) of
the headline workload; ``roofline`` reports the step's kernel against the 8 TB/s
HBM peak with achieved = algorithmic bytes per launch / average launch duration
measured with HIP events on the stream the kernel runs on; ``cpu_baseline`` is the CPU oracle on the host cores; the other
workload shapes are reported under ``workloads``.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--quick] [--only NAME]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "effective TOPS + HBM GB/s (% of peak) for LUT mpGEMM, M=1 and M=4096"
HBM_PEAK_GBPS = 8000.0
MFMA_FP16_PEAK_TFLOPS = 2500.0
ROTATION_BYTES = 1 << 30
# read patterns of the streaming-read ceiling (workgroups, 16-byte loads per lane):
# the best single-launch reads of 4-48 MB and of 1 GiB in a sweep over grid size,
# loads in flight, nontemporal hints and workgroup ranges (profiles/stream_read_ceiling.txt)
STREAM_READ_CONFIGS = ((1024, 2), (2048, 1), (4096, 2), (512, 4), (512, 8))
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "pmc_traffic.txt")
# sources that define each timed kernel and its launch (a PMC traffic record is used
# only while they hash as when the counters were taken)
KERNEL_SOURCES = {
    "mpgemm": ("lut_gemv.hip", "lut_mtok.hip", "lut_mpgemm.hip", "lut_common.h", "lutgemm_internal.h", "api.cpp"),
    "fused": ("lut_fused.hip", "lut_mpgemm.hip", "lut_common.h", "lutgemm_internal.h", "api.cpp"),
    "dequant": ("dequant_mfma.hip", "lutgemm_internal.h", "api.cpp"),
}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--quick", action="store_true", help="headline workload only")
    ap.add_argument("--only", default=None, help="measure one workload name (profiling)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="also run a plain 256 MiB device copy (counter calibration)")
    ap.add_argument("--summarize-trace", metavar="DIR", default=None,
                    help="print the summary of a rocprofv3 --kernel-trace --stats output directory (no GPU)")
    ap.add_argument("--summarize-traffic", nargs="+", metavar="DIR", default=None,
                    help="print HBM traffic records from rocprofv3 --pmc runs in directories named "
                         "fetch_<workload> / write_<workload> (FETCH_SIZE, WRITE_SIZE; no GPU)")
    ap.add_argument("--summarize-counters", metavar="DIR", nargs="+", default=None,
                    help="print per-kernel utilization from rocprofv3 --pmc runs (no GPU)")
    ap.add_argument("--timeline", metavar="WORKLOAD", default=None,
                    help="per-wavefront phase timeline of one workload's single-token kernel, from the "
                         "instrumented library (paper_2408_06003_amd/build.py --timeline)")
    ap.add_argument("--timeline-entry", default="mpgemm", choices=("mpgemm", "fused"),
                    help="entry point whose kernel the timeline records")
    ap.add_argument("--stream-ceiling", action="store_true",
                    help="sweep the streaming-read calibration kernel over sizes and launch shapes and print "
                         "the best single-launch read per size (GPU)")
    ap.add_argument("--command", default="", help="the profiling command, recorded in a summary")
    ap.add_argument("--bench-logs", nargs="*", default=[],
                    help="bench.py outputs (JSON line last) whose headline launch times a trace summary quotes")
    return ap.parse_args()


# The paper's own figures for this path, restated (context only, not targets: it
# reports no measured software-LUT kernel throughput on a real GPU, and its LUT
# Tensor Core figures come from simulation or synthesis).
PAPER_CONTEXT = {
    "note": "context only; other hardware, mostly simulated",
    "sec_2_3_software_lut_on_a100": "dequantization + tensor cores beat the software LUT-GEMM kernel at every "
                                    "batch size of its LLaMA2-70B W_INT4 A_FP16 shapes, by orders of magnitude at "
                                    "large batch",
    "sec_4_3_kernel_level": "M=2048 N=27648 K=5120 W_INT1 A_FP16: simulated LUT Tensor Core slightly faster than "
                            "the MAC tensor core at 14.3 % of its area (Accel-Sim, A100 configuration)",
    "sec_4_5_vs_lut_gemm": "simulated LUT Tensor Core (57.2 % of the FP16 tensor-core area) against LUT-GEMM on "
                           "A100: up to 1.42x on GEMV, 72.2x on GEMM; LUT-GEMM beats FP16 cuBLAS only on GEMV",
    "sec_4_6_precompute_fusion": "separate table precompute adds 8-33 % to a layer (Welder, OPT-175B, "
                                 "BLOOM-176B, LLaMA2-70B), fused precompute 1.2-3.9 %",
}


def algorithmic_bytes(inp, out_bytes, fused=False, tri=False, lut8=False):
    """Bytes the method must move for one mpGEMM call: weights N K b / 8, metadata
    (FP16 scale + zero per group: 4 B; per-channel scale: 2 B; per-tensor: 4 B),
    tables 4 M K (8 two-byte entries per 4 activations) -- or, for the fused
    kernel, the FP16 activations 2 M K instead -- and the output M N out_bytes.
    Ternary 3-in-5 (``tri``): weights 5 bits per 3 weights, N K 5 / 24 (K padded to
    whole 96-weight blocks), and tables of 16 two-byte entries per 3 activations.
    INT8 table quantization (``lut8``): tables of 8 one-byte codes and one FP32 scale
    per 4 activations, 3 M K."""
    M, K, N, b = inp.M, inp.K, inp.N, inp.bits
    weights = N * K * b // 8
    if tri:
        weights = N * (-(-K // 96)) * 20
    if inp.group == 0:
        meta = 4
    elif inp.zeros is None:
        meta = 2 * N * (K // inp.group)
    else:
        meta = 4 * N * (K // inp.group)
    tables = 2 * M * K if fused else (M * (-(-K // 96)) * 32 * 32 if tri else (3 if lut8 else 4) * M * K)
    out = M * N * out_bytes
    return {"weights": weights, "meta": meta, "tables": tables, "out": out,
            "total": weights + meta + tables + out}


def kernel_source_hash(kernel):
    """Hash of the sources that define one timed kernel and its launch."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2408_06003_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(workload, kernel):
    """HBM bytes per launch of one kernel from rocprofv3 FETCH_SIZE / WRITE_SIZE runs,
    if they were taken on the current kernel source (else None)."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    src = kernel_source_hash(kernel)
    with open(TRAFFIC_FILE) as f:
        for line in f:
            line = line.strip()
            if not line.startswith("{"):
                continue
            rec = json.loads(line)
            if (rec.get("workload") == workload and rec.get("timed_kernel") == kernel
                    and rec.get("kernel_source_sha256_16") == src):
                return rec.get("bytes_per_launch")
    return None


def case_name(cid, sid, M, tri=False, lut8=False):
    """Name of one workload shape in the bench output."""
    import workloads as W
    w = W.WORKLOADS[cid]
    name = w.name if len(w.kn) == 1 and len(w.ms) == 1 else f"{w.name}_M{M}_K{w.kn[sid][0]}_N{w.kn[sid][1]}"
    return name + ("_3in5" if tri else "") + ("_lut8" if lut8 else "")


class Case:
    """One workload shape on the device, with a rotation set of packed weights."""

    def __init__(self, cid, sid, M, rotate=True, wfmt=None, act=None):
        """``wfmt`` overrides the packing of the same codes (the ternary 3-in-5 format),
        ``act`` the table precision of the same FP16 activations (INT8 table quantization)."""
        import torch
        import paper_2408_06003_amd as L
        import workloads as W
        self.torch, self.L, self.W = torch, L, W
        self.tri = wfmt == L.WFMT_TERNARY_3IN5
        self.lut8 = act == W.ACT_FP16_LUT8
        self.name = case_name(cid, sid, M, self.tri, self.lut8)
        self.inp = W.make_inputs(cid, sid, M=M)
        if self.lut8:
            self.inp.act_kind = act
        inp = self.inp
        self.M, self.K, self.N = inp.M, inp.K, inp.N
        self.p = L.problem(inp.K, inp.N, inp.bits, inp.wfmt if wfmt is None else wfmt, inp.group,
                           act=inp.act_kind, scale_fp32=(inp.scales.dtype.itemsize == 4))
        dev = torch.device("cuda")
        codes = torch.from_numpy(inp.codes).to(dev)
        scales = torch.from_numpy(inp.scales).to(dev)
        zeros = None if inp.zeros is None else torch.from_numpy(inp.zeros).to(dev)
        self.act = torch.from_numpy(inp.act).to(dev)
        nbytes = L.packed_weight_size(self.p)
        first = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        L.pack_weights(self.p, codes, scales, zeros, first)
        del codes
        R = max(2, math.ceil(ROTATION_BYTES / nbytes)) if rotate else 1
        self.packed = [first] + [first.clone() for _ in range(R - 1)]
        self.tables = torch.empty(L.table_size(self.p, M), dtype=torch.uint8, device=dev)
        ws = L.workspace_size(self.p, M)
        self.ws = torch.zeros(ws, dtype=torch.uint8, device=dev) if ws else None
        dq = L.dequant_workspace_size(self.p, M)
        self.dq_ws = torch.empty(dq, dtype=torch.uint8, device=dev) if dq else None
        # allocated and zero-filled here, not on first use: a first use inside a graph
        # capture would capture the fill instead of running it
        fw = L.fused_workspace_size(self.p, M)
        self.fws = torch.zeros(fw, dtype=torch.uint8, device=dev) if fw else None
        self.int8 = inp.act_kind == W.ACT_INT8
        self.out_code = L.OUT_FP32 if self.int8 else L.OUT_FP16
        self.out = torch.empty((M, inp.N), dtype=torch.float32 if self.int8 else torch.float16, device=dev)
        self.out_bytes = self.out.element_size()
        torch.cuda.synchronize()

    def precompute(self):
        self.L.precompute(self.p, self.M, self.act, self.tables)

    def mpgemm(self, i):
        self.L.mpgemm(self.p, self.M, self.tables, self.packed[i % len(self.packed)], self.out,
                      self.out_code, False, workspace=self.ws)

    def dequant(self, i, out):
        self.L.mpgemm_dequant(self.p, self.M, self.act, self.packed[i % len(self.packed)], out,
                              self.L.OUT_FP16, False, workspace=self.dq_ws)

    def step(self, i):
        self.precompute()
        self.mpgemm(i)

    def fused(self, i):
        """The same step through lutgemm_mpgemm_fused (tables built inside the LUT kernel)."""
        self.L.mpgemm_fused(self.p, self.M, self.act, self.packed[i % len(self.packed)], self.out,
                            self.out_code, False, workspace=self.fws)

    def timed(self, fn, n, graph=True, check=None, reps=5):
        """Milliseconds per call of n back-to-back calls, timed with HIP events on the
        stream they run on.  With graph=True the calls are captured into HIP graphs and
        replayed, so host launch overhead is not counted (the way a decode loop runs).
        Every graph holds n calls on its own slice of the rotation set, and enough graphs
        are captured to cover the whole set (>= 1 GiB of distinct weight copies); the
        graphs are replayed in turn and each replay is timed on its own (the device
        idle before it), so between two replays of one graph at least 1 GiB of other
        weights has been read and every timed call reads its weights from HBM, whatever
        n is.  At least ``reps`` replays are timed (every graph at least once) and the
        median is returned;
        ``self.last_distinct_bytes`` records the distinct weight bytes they read.
        ``check`` (a function returning a tensor) compares a replay, after eager work,
        with the eager result."""
        torch = self.torch
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        R = len(self.packed)
        if not graph:
            s = torch.cuda.current_stream()
            torch.cuda.synchronize()
            e0.record(s)
            for i in range(n):
                fn(i)
            e1.record(s)
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) / n
        n_graphs = max(1, -(-R // n))
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        graphs = []
        for gi in range(n_graphs):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=side):
                for j in range(n):
                    fn(gi * n + j)
            graphs.append(g)
        torch.cuda.synchronize()
        if check is not None:
            for _ in range(2):
                fn(n - 1)
                torch.cuda.synchronize()
                ref = check().clone()
                check().zero_()
                graphs[0].replay()
                torch.cuda.synchronize()
                if not torch.equal(check(), ref):
                    raise RuntimeError(f"{self.name}: graph replay differs from the eager result")
        for g in graphs:  # warm replays of every slice
            g.replay()
        torch.cuda.synchronize()
        s = torch.cuda.current_stream()
        batches, touched = [], set()
        for r in range(max(reps, n_graphs)):
            gi = r % n_graphs
            torch.cuda.synchronize()
            e0.record(s)
            graphs[gi].replay()
            e1.record(s)
            torch.cuda.synchronize()
            batches.append(e0.elapsed_time(e1) / n)
            touched.update((gi * n + j) % R for j in range(n))
        self.last_distinct_bytes = len(touched) * self.packed[0].numel()
        self.last_replays = len(batches)
        return sorted(batches)[len(batches) // 2]

    def timed_queued(self, fn, n, reps=5):
        """Milliseconds per call of n back-to-back calls launched one by one, timed on the
        device: a bounded spin kernel (torch.cuda._sleep) holds the stream while the host
        enqueues the start event, the n calls and the end event, so the device runs them
        back to back and the interval between the events holds exactly their execution
        and dispatch, without the host's per-call launch cost or a graph launch's fixed
        cost (about 10 us per replay on this stack).  The hold is sized from a measured
        enqueue time; were it too short, the host's launch gaps would land inside the
        interval and make the figure slower, never faster.  Every rep starts on its own
        slice of the rotation set (HBM-cold weights); at least ``reps`` reps and enough to
        cover the whole set are timed, and the median is returned."""
        torch = self.torch
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        R = len(self.packed)
        s = torch.cuda.current_stream()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for j in range(n):
            fn(j % R)
        enqueue_us = (time.perf_counter() - t0) * 1e6
        torch.cuda.synchronize()
        hold_cycles = int((2.0 * enqueue_us + 100.0) * 2400)  # shader-clock cycles at 2.4 GHz
        batches, touched, late = [], set(), 0
        for r in range(max(reps, -(-R // n))):
            base = (r * n) % R
            torch.cuda.synchronize()
            torch.cuda._sleep(hold_cycles)
            t0 = time.perf_counter()
            e0.record(s)
            for j in range(n):
                fn((base + j) % R)
            e1.record(s)
            late += (time.perf_counter() - t0) * 1e6 > hold_cycles / 2400.0
            torch.cuda.synchronize()
            batches.append(e0.elapsed_time(e1) / n)
            touched.update((base + j) % R for j in range(n))
        self.last_distinct_bytes = len(touched) * self.packed[0].numel()
        self.last_replays = len(batches)
        self.last_hold_late = late
        return sorted(batches)[len(batches) // 2]

    def best_timed(self, fn, n, check=None, reps=5):
        """The faster of the graph-replayed and the queued timing of the same n calls
        (milliseconds per call); ``self.last_mode`` names the one taken."""
        ms_g = self.timed(fn, n, check=check, reps=reps)
        dg = self.last_distinct_bytes
        ms_q = self.timed_queued(fn, n, reps=reps)
        if ms_g <= ms_q:
            self.last_mode, self.last_distinct_bytes = "graph", dg
            return ms_g
        self.last_mode = "queued"
        return ms_q

    def cold_call_us(self, fn, i):
        """One call on its own (device idle before it, HBM-cold weight copy i), timed with
        HIP events on its stream: the latency a single decode step sees."""
        torch = self.torch
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s = torch.cuda.current_stream()
        torch.cuda.synchronize()
        e0.record(s)
        fn(i)
        e1.record(s)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3

    def effective_tops(self, ms):
        return 2.0 * self.M * self.N * self.K / (ms * 1e-3) / 1e12

    def measure(self, n_kernel, warmup):
        """Kernel-level numbers of this shape: mpGEMM, precompute, and the comparison path
        (M >= 16, and at any M where it takes the 16-token slab kernel: 1-bit weights)."""
        for i in range(warmup):
            self.step(i)
        self.precompute()
        ms_mp = self.best_timed(self.mpgemm, n_kernel, check=lambda: self.out)
        distinct, mp_mode = self.last_distinct_bytes, self.last_mode
        ms_pre = self.best_timed(lambda i: self.precompute(), n_kernel)
        b = algorithmic_bytes(self.inp, self.out_bytes, tri=self.tri, lut8=self.lut8)
        gbps = b["total"] / (ms_mp * 1e-3) / 1e9
        # the achievable single-launch read of the same byte count, same rotation and
        # timing: the fastest of the read patterns the calibration sweep found best
        # (nontemporal 16-byte loads; grid and loads in flight per lane vary with size)
        sink = self.torch.zeros(4096, dtype=self.torch.int32, device="cuda")
        wb = self.L.packed_weight_size(self.p)
        R = len(self.packed)
        ms_rd, rd_cfg = None, None
        for blocks, unroll in STREAM_READ_CONFIGS:
            ms = self.best_timed(lambda i: self.L.calibrate_stream_read_ex(self.packed[i % R], wb, sink, blocks,
                                                                          unroll, 1), n_kernel)
            if ms_rd is None or ms < ms_rd:
                ms_rd, rd_cfg = ms, f"{blocks} workgroups x 256 lanes, {unroll} nontemporal 16-B loads in flight per lane"
        ms_fu = self.best_timed(self.fused, n_kernel, check=lambda: self.out)
        rec = {"workload": self.name, "M": self.M, "K": self.K, "N": self.N, "bits": self.inp.bits,
               "mpgemm_us": round(ms_mp * 1e3, 3), "mpgemm_tops": round(self.effective_tops(ms_mp), 3),
               "mpgemm_gbps": round(gbps, 1), "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4),
               "distinct_weight_bytes_timed": distinct, "mpgemm_timing": mp_mode,
               "stream_read_us": round(ms_rd * 1e3, 3), "stream_read_cfg": rd_cfg,
               "stream_read_gbps": round(wb / (ms_rd * 1e-3) / 1e9, 1),
               "frac_of_stream_read": round(ms_rd / ms_mp, 4),
               "precompute_us": round(ms_pre * 1e3, 3),
               "precompute_over_mpgemm": round(ms_pre / ms_mp, 4),
               "fused_us": round(ms_fu * 1e3, 3), "fused_tops": round(self.effective_tops(ms_fu), 3),
               "algorithmic_bytes": b["total"], "rotation_copies": len(self.packed),
               # HBM bytes per call from rocprofv3 FETCH_SIZE + WRITE_SIZE (null without a record
               # taken on the current kernel sources)
               "mpgemm_hbm_traffic_bytes": load_traffic(self.name, "mpgemm"),
               "fused_hbm_traffic_bytes": load_traffic(self.name, "fused")}
        if (not self.int8 and not self.tri and not self.lut8
                and (self.M >= 16 or self.L.dequant_plan(self.p, self.M)[0] == 2)):
            out = self.torch.empty((self.M, self.N), dtype=self.torch.float16, device="cuda")
            for i in range(3):
                self.dequant(i, out)
            n = max(5, min(n_kernel, 50))
            ms_dq = self.best_timed(lambda i: self.dequant(i, out), n, check=lambda: out)
            tflops = self.effective_tops(ms_dq)
            kind, splits = self.L.dequant_plan(self.p, self.M)
            name = {0: "dequant_mfma_kernel (128x128 tiles; not tuned)",
                    1: "dequant_mfma_big_kernel (256x256 tiles, 8 wavefronts, pipelined)",
                    2: "dequant_skinny_kernel (16-token slabs, 1-bit weights decoded in registers)"}[kind]
            rec.update({"dequant_mfma_us": round(ms_dq * 1e3, 3), "dequant_mfma_tops": round(tflops, 2),
                        "dequant_mfma_frac_of_fp16_peak": round(tflops / MFMA_FP16_PEAK_TFLOPS, 4),
                        "dequant_kernel": name, "dequant_k_splits": splits,
                        "dequant_hbm_traffic_bytes": load_traffic(self.name, "dequant")})
            if kind != 0:
                rec["lut_over_dequant_time"] = round(ms_mp / ms_dq, 2)
        return rec

    def release(self):
        self.packed = None
        self.torch.cuda.empty_cache()


def cpu_baseline(inp, budget_s=10.0):
    """The CPU oracle (as it stands) on the host cores, on the full headline step,
    repeated for about ``budget_s`` seconds; throughput in effective TOPS."""
    import oracle
    threads = len(os.sched_getaffinity(0))
    if os.environ.get("OMP_NUM_THREADS", "").isdigit():
        threads = min(threads, int(os.environ["OMP_NUM_THREADS"]))
    oracle.lib()  # load outside the timed region
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.reference_output(inp)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s or reps >= 100000:
            break
    per = el / reps
    return {"value": round(2.0 * inp.M * inp.N * inp.K / per / 1e12, 6), "unit": "TOPS", "cores": threads,
            "kind": "oracle",
            "sample": f"full step (INT8 quantize + int64 dot products + FP32 scaling) of M={inp.M} K={inp.K} "
                      f"N={inp.N}, repeated {reps}x in {el:.1f} s; {per * 1e3:.2f} ms per step"}


SINGLE_CORE_CODE = r"""
import json, sys, time
sys.path.insert(0, sys.argv[1])
import oracle, workloads as W
oracle.lib()
out = []
for cid, sid in ((1, 0), (2, 0), (3, 0), (3, 1), (3, 2), (3, 3)):
    inp = W.make_inputs(cid, sid, M=1)
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.reference_output(inp)
        reps += 1
        el = time.perf_counter() - t0
        if el >= float(sys.argv[2]):
            break
    per = el / reps
    out.append({"workload": f"{W.WORKLOADS[cid].name}/{inp.K}x{inp.N}", "value": round(2.0 * inp.M * inp.N * inp.K / per / 1e9, 3),
                "unit": "GOPS", "seconds_per_call": round(per, 6), "calls": reps})
print(json.dumps(out))
"""


def cpu_baseline_single_core(budget_s=2.0):
    """The CPU oracle on ONE host core (OpenMP limited to one thread in a child process
    that never touches the GPU) for the M = 1 workloads of configs 1-3, each repeated
    for about ``budget_s`` seconds."""
    import subprocess
    env = dict(os.environ, OMP_NUM_THREADS="1")
    r = subprocess.run([sys.executable, "-c", SINGLE_CORE_CODE, ROOT, str(budget_s)], env=env,
                       capture_output=True, text=True, timeout=300)
    if r.returncode != 0:
        return {"error": r.stderr[-500:]}
    return {"cores": 1, "kind": "oracle", "per_workload": json.loads(r.stdout.strip().splitlines()[-1])}


def calibrate_copy():
    """A plain device copy of known size, for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE."""
    import torch
    n = 256 << 20
    a = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    b = torch.empty_like(a)
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / 10
    return {"bytes_read": n, "bytes_written": n, "us": round(ms * 1e3, 2),
            "gbps": round(2 * n / (ms * 1e-3) / 1e9, 1)}


def stream_ceiling(sizes_mb=(4.2, 8.9, 26.8, 29.5, 48.0, 1024.0)):
    """The best single-launch streaming read of each byte count: the calibration kernel
    over grid sizes, 16-byte loads in flight per lane, nontemporal hints and workgroup
    ranges, each launch on its own slice of a >= 1 GiB rotation set (HBM-cold), graph
    replays of back-to-back launches, median of 5 replays.  Prints a text summary."""
    import itertools
    import math
    import torch
    import paper_2408_06003_amd as L
    torch.cuda.set_device(0)
    sink = torch.zeros(65536, dtype=torch.int32, device="cuda")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def replay_us(fn, n, reps=5):
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            for i in range(n):
                fn(i)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        t = []
        for _ in range(reps):
            e0.record()
            g.replay()
            e1.record()
            torch.cuda.synchronize()
            t.append(e0.elapsed_time(e1) * 1e3 / n)
        return sorted(t)[len(t) // 2]

    lines = ["# Single-launch streaming-read ceiling of the MI355X (HBM-cold)", "",
             "command (on the MI355X): python3 bench.py --stream-ceiling", "",
             "lutgemm_calibrate_stream_read_ex: every lane keeps U 16-byte loads in flight (clamped indices,",
             "XOR-folded, one word per workgroup written); 'nt' = nontemporal loads, 'contig' = one contiguous",
             "range per workgroup instead of round-robin tiles.  Each launch reads its own copy of the buffer",
             "(a >= 1 GiB rotation set), launches are graph-replayed back to back, median of 5 replays.",
             "Published HBM3E peak: 8000 GB/s.", ""]
    summary = []
    for mb in sizes_mb:
        nb = (int(mb * (1 << 20)) + 255) // 256 * 256
        R = max(2, math.ceil((1 << 30) / nb))
        bufs = [torch.ones(nb, dtype=torch.uint8, device="cuda") for _ in range(R)]
        torch.cuda.synchronize()
        n = 4 if nb >= (1 << 29) else max(20, min(200, R))
        blist = (256, 512, 1024, 2048, 4096, 8192) if nb < (1 << 29) else (1024, 2048, 4096, 8192, 16384)
        res = []
        for blocks, unroll, flags in itertools.product(blist, (1, 2, 4, 8, 16), (0, 1, 2, 3)):
            if blocks * 256 * unroll * 16 > 4 * nb and blocks > 256:
                continue  # grids far larger than the data
            us = replay_us(lambda i: L.calibrate_stream_read_ex(bufs[i % R], nb, sink, blocks, unroll, flags), n)
            res.append((us, blocks, unroll, flags))
        floor = {b: round(replay_us(lambda i: L.calibrate_stream_read_ex(bufs[i % R], 16, sink, b, 1, 0), 100), 3)
                 for b in (256, 1024, 4096)}
        res.sort()
        best = res[0]
        lines.append(f"{nb / 1e6:8.1f} MB: best {best[0]:8.3f} us = {nb / (best[0] * 1e-6) / 1e9:7.1f} GB/s "
                     f"({nb / (best[0] * 1e-6) / 8e12:.3f} of 8 TB/s) with {best[1]} workgroups, U={best[2]}, "
                     f"nt={best[3] & 1}, contig={best[3] >> 1}; 16-byte launch floor {floor} us")
        for us, blocks, unroll, flags in res[1:5]:
            lines.append(f"{'':12s}next: {us:8.3f} us ({nb / (us * 1e-6) / 1e9:7.1f} GB/s) {blocks} wg, U={unroll}, "
                         f"nt={flags & 1}, contig={flags >> 1}")
        summary.append((nb, best[0]))
        del bufs
        torch.cuda.empty_cache()
    lines += ["", "bytes, best time, best rate:"]
    for nb, us in summary:
        lines.append(f"  {nb:>12d} B: {us:9.3f} us, {nb / (us * 1e-6) / 1e9:7.1f} GB/s")
    return "\n".join(lines)


# ---------------------------------------------------------------- rocprofv3 summaries (CPU only)

HEADLINE_KERNELS = {
    # kind in KERNEL_SOURCES -> name prefix of the kernel the headline step launches
    "fused": "void lutgemm::lut_fused_gemv_kernel<2, 2, 2, 4, 4, true>",
    "mpgemm": "void lutgemm::lut_gemv2_kernel<2, 2, 2, 1, 16, true, false>",
}
COPY_KERNEL = "__amd_rocclr_copyBuffer"


def _csv_rows(directory, suffix):
    import csv
    import glob
    rows = []
    for path in sorted(glob.glob(os.path.join(directory, "**", "*" + suffix), recursive=True)):
        with open(path, newline="") as f:
            rows.extend(csv.DictReader(f))
    return rows


def _short(name, n=78):
    return name if len(name) <= n else name[:n - 3] + "..."


def summarize_trace(directory, command="", bench_logs=()):
    """Per-kernel durations of a rocprofv3 kernel-trace run, and the headline kernels'
    durations over their back-to-back runs (the bench's graph replays)."""
    import statistics
    stats = _csv_rows(directory, "kernel_stats.csv")
    trace = _csv_rows(directory, "kernel_trace.csv")
    out = ["# rocprofv3 kernel-trace summary", "", "command (on the MI355X, from /tmp with TMPDIR=/tmp):",
           f"  {command}", "",
           "Average/min/max kernel durations in microseconds over all dispatches of the run",
           "(kernel start to end; the bench's per-launch times, measured with HIP events over",
           "graph replays, also include the gap between back-to-back kernels).  torch's",
           "spin_kernel is the bench's bounded device-side hold ahead of each queued-timing batch",
           "(no part of any step).", "",
           f"{'kernel':78s} {'calls':>7s} {'avg_us':>9s} {'min_us':>9s} {'max_us':>9s} {'%time':>6s}"]
    stats.sort(key=lambda r: -float(r["TotalDurationNs"]))
    for r in stats:
        out.append(f"{_short(r['Name']):78s} {int(r['Calls']):7d} {float(r['AverageNs']) / 1e3:9.2f} "
                   f"{float(r['MinNs']) / 1e3:9.2f} {float(r['MaxNs']) / 1e3:9.2f} {float(r['Percentage']):6.2f}")
    trace.sort(key=lambda r: int(r["Start_Timestamp"]))
    out += ["", "Headline kernels in runs of >= 100 back-to-back dispatches (the timed graph replays):"]
    for kind, prefix in HEADLINE_KERNELS.items():
        runs, cur = [], []
        for r in trace:
            if r["Kernel_Name"].startswith(prefix):
                cur.append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
            elif cur:
                runs.append(cur)
                cur = []
        if cur:
            runs.append(cur)
        runs = [x for x in runs if len(x) >= 100]
        d = [v for x in runs for v in x]
        if d:
            d.sort()
            out.append(f"  {prefix[5:]}: {len(runs)} runs, {len(d)} dispatches, duration median "
                       f"{statistics.median(d):.3f} us, mean {statistics.mean(d):.3f} us, "
                       f"p10 {d[len(d) // 10]:.3f} us")
    for path in bench_logs:
        with open(path) as f:
            res = json.loads([line for line in f if line.startswith("{")][-1])
        out.append(f"bench.py's own per-launch times (HIP events over graph replays), {os.path.basename(path)}: "
                   f"fused {res['roofline']['avg_launch_us']} us, table-fed mpGEMM "
                   f"{res['two_call_step']['mpgemm_roofline']['avg_launch_us']} us")
    return "\n".join(out)


def _per_dispatch(rows, counter):
    """{kernel name: [value per dispatch]} for one counter (instances summed per dispatch)."""
    per = {}
    for r in rows:
        if r["Counter_Name"] != counter:
            continue
        key = (r["Kernel_Name"], r["Dispatch_Id"])
        per[key] = per.get(key, 0.0) + float(r["Counter_Value"])
    out = {}
    for (name, _), v in per.items():
        out.setdefault(name, []).append(v)
    return out


def _dispatches(rows, counter):
    """[(dispatch id, kernel name, value)] of one counter in dispatch order (instances summed)."""
    per = {}
    for r in rows:
        if r["Counter_Name"] != counter:
            continue
        key = (int(r["Dispatch_Id"]), r["Kernel_Name"])
        per[key] = per.get(key, 0.0) + float(r["Counter_Value"])
    return sorted((d, n, v) for (d, n), v in per.items())


def _call_kind(name):
    """Which timed call a kernel serves: 'mpgemm', 'fused' or 'dequant' for the main
    kernels, 'attach' for the split-completion kernels (finalize, reduce) that belong to
    the call launched just before them, None for everything else."""
    if "lut_finalize_kernel" in name or "dequant_reduce_kernel" in name:
        return "attach"
    if "lut_fused_" in name:
        return "fused"
    if "lut_gemv" in name or "lut_mtok_kernel" in name:
        return "mpgemm"
    if "dequant_" in name:
        return "dequant"
    return None


def _workload_inputs(name):
    """Inputs and output element size of a workload named as in the bench output."""
    import workloads as W
    for cid, w in W.WORKLOADS.items():
        for (sid, M, _, _) in w.shapes():
            for lut8 in (False, True):
                if case_name(cid, sid, M, lut8=lut8) == name:
                    inp = W.make_inputs(cid, sid, M=M)
                    return inp, (4 if inp.act_kind == W.ACT_INT8 else 2), lut8
    return None, None, None


def summarize_traffic(dirs, command=""):
    """HBM bytes per call of the LUT and comparison kernels from FETCH_SIZE and
    WRITE_SIZE runs (KiB per dispatch, each counter in its own run), scaled by what the
    counters read for the run's 256 MiB device copy.  Directories are named
    fetch_<workload> / write_<workload>, one bench.py --only <workload> --calibrate-copy
    run each; in every run the dispatches before the copy belong to the headline
    workload and those after it to <workload>.  A call's traffic is its main kernel plus
    the split-completion kernel launched right after it (finalize, reduce)."""
    import re
    runs = {}
    for d in dirs:
        base = os.path.basename(os.path.normpath(d))
        m = re.match(r"^(fetch|write)_(.+)$", base)
        if not m:
            raise SystemExit(f"{d}: expected a directory named fetch_<workload> or write_<workload>")
        runs.setdefault(m.group(2), {})[m.group(1)] = d
    kib = 256 * 1024  # the calibration copy reads and writes 256 MiB
    head = case_name(2, 0, 1)
    per_call = {}   # (workload, kind) -> {"fetch": [per call], "write": [...], "kernels": set}
    scales = {}
    for wl, pair in sorted(runs.items()):
        if set(pair) != {"fetch", "write"}:
            raise SystemExit(f"{wl}: need both a fetch_ and a write_ run")
        for counter, key in (("FETCH_SIZE", "fetch"), ("WRITE_SIZE", "write")):
            seq = _dispatches(_csv_rows(pair[key], "counter_collection.csv"), counter)
            copies = [(v, d) for d, n, v in seq if n.startswith(COPY_KERNEL)]
            if not copies:
                raise SystemExit(f"{pair[key]}: no 256 MiB copy: profile bench.py with --calibrate-copy")
            v_copy, d_copy = max(copies)
            scale = kib / v_copy
            scales[(wl, key)] = scale
            cur = None  # (segment workload, kind, call record) of the last main kernel
            for d, n, v in seq:
                seg = head if d < d_copy else wl
                kind = _call_kind(n)
                if kind in ("mpgemm", "fused", "dequant"):
                    rec = per_call.setdefault((seg, kind), {"fetch": [], "write": [], "kernels": set()})
                    rec[key].append(v * scale * 1024)
                    rec["kernels"].add(n)
                    cur = (seg, kind)
                elif kind == "attach" and cur is not None:
                    rec = per_call[cur]
                    rec[key][-1] += v * scale * 1024
                    rec["kernels"].add(n)
    out = ["# HBM traffic per call of the LUT mpGEMM and comparison kernels (rocprofv3 PMC counters)", "",
           "commands (each counter in its own run, from /tmp with TMPDIR=/tmp), for each <workload> listed below:",
           f"  {command}", "",
           "Each run's FETCH_SIZE / WRITE_SIZE (KiB per dispatch) are scaled by what the same counter reads",
           "for the run's 256 MiB device copy (torch copy_, __amd_rocclr_copyBuffer; 262144 KiB read and written).",
           "A call's traffic adds the split-completion kernel (finalize / reduce) that follows its main kernel.",
           "Algorithmic bytes: weights N K b / 8 + metadata + tables 4 M K (mpgemm) or FP16 activations 2 M K",
           "(fused, dequant) + output; the ratio above 1 is re-read or partial-sum traffic.", ""]
    recs = []
    for (wl, kind), rec in sorted(per_call.items()):
        inp, ob, lut8 = _workload_inputs(wl)
        if inp is None or not rec["fetch"] or not rec["write"]:
            continue
        n = min(len(rec["fetch"]), len(rec["write"]))
        f = sorted(rec["fetch"])[n // 2] if n else 0.0
        w = sorted(rec["write"])[n // 2] if n else 0.0
        out_b = 2 if kind == "dequant" else ob
        alg = algorithmic_bytes(inp, out_b, fused=(kind != "mpgemm"), lut8=(lut8 and kind == "mpgemm"))["total"]
        traffic = round(f + w)
        out += [f"{wl} / {kind}: {', '.join(sorted(_short(k, 90) for k in rec['kernels']))}",
                f"  calls {n}; median per call: read {f / 1024:.1f} KiB, written {w / 1024:.1f} KiB; "
                f"traffic {traffic} B vs algorithmic {alg} B ({traffic / alg:.3f}x)", ""]
        recs.append({"workload": wl, "timed_kernel": kind, "kernels": sorted(rec["kernels"]), "calls": n,
                     "read_bytes": round(f), "write_bytes": round(w), "bytes_per_launch": traffic,
                     "algorithmic_bytes": alg, "ratio": round(traffic / alg, 4),
                     "fetch_scale": round(scales.get((wl, "fetch"), 0.0), 4),
                     "write_scale": round(scales.get((wl, "write"), 0.0), 4),
                     "kernel_source_sha256_16": kernel_source_hash(kind)})
    out += ["machine-readable records (bench.py uses one only while the kernel sources hash the same):"]
    out += [json.dumps(r) for r in recs]
    return "\n".join(out)


def summarize_counters(dirs, command=""):
    """Per-kernel utilization from rocprofv3 --pmc runs: MFMA busy per SIMD, LDS active
    and bank-conflict cycles per CU, VALU active per CU, each as a fraction of the
    kernel's GRBM_GUI_ACTIVE cycles (256 CUs, 1024 SIMDs)."""
    import re
    # runs of one workload (directories named <tag>_<letter>_<workload>) are grouped,
    # so that a kernel that serves several workloads is reported per workload
    per = {}
    for d in dirs:  # one run per directory: dispatch ids repeat across runs
        base = os.path.basename(os.path.normpath(d))
        m = re.match(r"^[^_]+_[a-z]_(.+)$", base)
        wl = m.group(1) if m else base
        rows = _csv_rows(d, "counter_collection.csv")
        for c in sorted({r["Counter_Name"] for r in rows}):
            for name, vals in _per_dispatch(rows, c).items():
                per.setdefault(c, {}).setdefault((wl, name), []).extend(vals)
    counters = sorted(per)
    keys = sorted({k for c in counters for k in per[c]})
    out = ["# Utilization counters of the LUT and comparison kernels (rocprofv3 --pmc)", "",
           "commands (from /tmp with TMPDIR=/tmp):", f"  {command}", "",
           "Per dispatch, averaged over the dispatches of one workload's runs; cycles are",
           "shader-clock cycles summed over the instances the counter has (GRBM_GUI_ACTIVE is",
           "summed over the 8 XCDs, so the kernel's own cycles are GRBM_GUI_ACTIVE / 8).", ""]

    def avg(c, n):
        v = per.get(c, {}).get(n)
        return sum(v) / len(v) if v else None

    for n in keys:
        if not n[1].startswith("void lutgemm::") and not n[1].startswith("lutgemm::"):
            continue
        g = avg("GRBM_GUI_ACTIVE", n)
        vals = {c: avg(c, n) for c in counters if avg(c, n) is not None}
        out.append(f"{n[0]}: {_short(n[1], 100)}")
        out.append("  " + ", ".join(f"{c} {v:.0f}" for c, v in vals.items()))
        if g:
            cyc = g / 8
            parts = []
            if "SQ_VALU_MFMA_BUSY_CYCLES" in vals:
                parts.append(f"MFMA busy {100 * vals['SQ_VALU_MFMA_BUSY_CYCLES'] / (1024 * cyc):.1f} % of SIMD cycles")
            if "SQ_LDS_IDX_ACTIVE" in vals:
                parts.append(f"LDS active {100 * vals['SQ_LDS_IDX_ACTIVE'] / (256 * cyc):.1f} % of CU cycles")
            if "SQ_LDS_BANK_CONFLICT" in vals and "SQ_LDS_IDX_ACTIVE" in vals:
                parts.append(f"bank conflicts {100 * vals['SQ_LDS_BANK_CONFLICT'] / max(1.0, vals['SQ_LDS_IDX_ACTIVE']):.1f} % of LDS active")
            if "SQ_ACTIVE_INST_VALU" in vals:
                parts.append(f"VALU issuing {100 * vals['SQ_ACTIVE_INST_VALU'] / (256 * cyc):.1f} % of CU cycles")
            if parts:
                out.append("  " + "; ".join(parts))
        out.append("")
    return "\n".join(out)


TIMELINE_SLOTS = {
    # kernel family -> names of the stamp slots it writes (see tl_stamp in csrc/lut_common.h)
    "split": ("start", "tables in LDS", "lookups done", "partial stored+acked", "arrival counted",
              "partials summed (last workgroup)", "end"),
    "fused_gemv": ("start", "amax known", "tables built", "lookups done", "cross-wave barrier", "end"),
    "gemv2": ("start", "first chunk's tables", None, "lookups done", "cross-wave barrier"),
}


def timeline(name, entry, n_calls=200):
    """Phase timeline of the kernel of one workload (M <= 2), recorded by the instrumented
    library: lane 0 of every wavefront stamps the 100 MHz real-time clock at each phase
    boundary.  A graph of back-to-back calls on HBM-cold weight copies is replayed; the
    stamps are those of its last call.  Prints per phase the distribution over wavefronts
    (microseconds after the first wavefront started)."""
    import ctypes
    import numpy as np
    import torch
    import paper_2408_06003_amd as L
    import workloads as W
    torch.cuda.set_device(0)
    tl_path = os.path.join(ROOT, "paper_2408_06003_amd", "liblutgemm_timeline.so")
    L.lib = L._load(tl_path)
    L.lib.lutgemm_timeline_set.argtypes = [ctypes.c_void_p]
    found = None
    for cid, w in W.WORKLOADS.items():
        for (sid, M, _, _) in w.shapes():
            if case_name(cid, sid, M) == name and M <= 2:
                found = (cid, sid, M)
    if not found:
        raise SystemExit(f"no single-token workload named {name}")
    c = Case(*found)
    buf = torch.zeros(8 << 20, dtype=torch.int64, device="cuda")
    L.lib.lutgemm_timeline_set(buf.data_ptr())
    fn = c.fused if entry == "fused" else c.mpgemm
    c.precompute()
    for i in range(3):
        fn(i)
    ms = c.timed(fn, n_calls, reps=5)
    torch.cuda.synchronize()
    L.lib.lutgemm_timeline_set(None)
    rec = buf.view(-1, 8).cpu().numpy()
    rec = rec[rec[:, 0] != 0]
    t0 = rec[:, 0].min()
    us = (rec.astype(np.float64) - t0) / 100.0  # 100 MHz clock
    us[rec == 0] = np.nan
    if np.isfinite(us[:, 6]).any():  # only the split-K kernels stamp slot 6
        fam = "split"
    else:
        fam = "fused_gemv" if entry == "fused" else "gemv2"
    names = TIMELINE_SLOTS[fam]
    lines = [f"# Phase timeline: {name}, lutgemm_{entry} ({fam} kernel)", "",
             f"graph-timed {ms * 1e3:.3f} us per call (HBM-cold weights, back-to-back); stamps of the last call of "
             f"a {n_calls}-call replay, {rec.shape[0]} wavefronts; microseconds after the first wavefront started", "",
             f"{'phase':36s} {'waves':>6s} {'p10':>7s} {'p50':>7s} {'p90':>7s} {'max':>7s}"]
    for k, nm in enumerate(names):
        if nm is None:
            continue
        v = us[:, k]
        v = v[np.isfinite(v)]
        if v.size == 0:
            continue
        q = np.percentile(v, [10, 50, 90])
        lines.append(f"{nm:36s} {v.size:6d} {q[0]:7.2f} {q[1]:7.2f} {q[2]:7.2f} {v.max():7.2f}")
    # per-wavefront phase durations
    lines += ["", "per-wavefront durations (median over wavefronts, us):"]
    for a, b in zip(range(len(names)), range(1, len(names))):
        if names[a] is None or names[b] is None:
            continue
        d = us[:, b] - us[:, a]
        d = d[np.isfinite(d)]
        if d.size:
            lines.append(f"  {names[a]} -> {names[b]}: {np.median(d):.2f} (p90 {np.percentile(d, 90):.2f})")
    c.release()
    return "\n".join(lines)


def main():
    args = parse()
    if args.timeline:
        print(timeline(args.timeline, args.timeline_entry))
        return
    if args.stream_ceiling:
        print(stream_ceiling(), flush=True)
        return
    if args.summarize_trace or args.summarize_traffic or args.summarize_counters:
        if args.summarize_trace:
            print(summarize_trace(args.summarize_trace, args.command, args.bench_logs))
        elif args.summarize_traffic:
            print(summarize_traffic(args.summarize_traffic, args.command))
        else:
            print(summarize_counters(args.summarize_counters, args.command))
        return
    if args.gpus != 1:
        print(f"bench.py: --gpus {args.gpus} is not supported: the LUT mpGEMM hot path runs on one GPU "
              "(sharding along N across GPUs is designed, not implemented)", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2408_06003_amd as L  # fails loudly if the HIP library is not built
    import workloads as W
    torch.cuda.set_device(0)

    # ---------------- headline: ternary INT8 GEMV M=1, K=N=4096
    log("headline workload: setting up")
    head = Case(2, 0, 1)
    K, WU = args.steps, args.warmup
    for i in range(WU):
        head.step(i)
        head.fused(i)
    torch.cuda.synchronize()
    # the step as one kernel (headline) and as two calls (tables through HBM)
    ms_step_graph = head.timed(head.fused, K, check=lambda: head.out)
    graph_distinct, graph_replays = head.last_distinct_bytes, head.last_replays
    ms_step_queued = head.timed_queued(head.fused, K)
    queued_distinct, queued_reps, queued_late = head.last_distinct_bytes, head.last_replays, head.last_hold_late
    if ms_step_queued < ms_step_graph:
        ms_step, step_timing, step_distinct, step_replays = ms_step_queued, "queued", queued_distinct, queued_reps
    else:
        ms_step, step_timing, step_distinct, step_replays = ms_step_graph, "graph", graph_distinct, graph_replays
    ms_step_eager = head.timed(head.fused, K, graph=False)
    ms_two_graph = head.timed(head.step, K, check=lambda: head.out)
    ms_two_queued = head.timed_queued(head.step, K)
    ms_two = min(ms_two_graph, ms_two_queued)
    ms_two_eager = head.timed(head.step, K, graph=False)
    kern = head.measure(max(K, 50), 5)
    cold_us = round(head.cold_call_us(head.fused, len(head.packed) // 2), 3)
    log(f"headline: fused {ms_step * 1e3:.2f} us/step, two-call {ms_two * 1e3:.2f} us/step, "
        f"mpgemm {kern['mpgemm_us']} us")
    fb = algorithmic_bytes(head.inp, head.out_bytes, fused=True)["total"]
    achieved = round(fb / (ms_step * 1e-3) / 1e9, 1)
    roofline = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": load_traffic(head.name, "fused"),
                "kernel": "lut_fused_gemv_kernel (lutgemm_mpgemm_fused, one launch per step)",
                "algorithmic_bytes_per_launch": fb, "avg_launch_us": round(ms_step * 1e3, 3)}
    mp_roof = {"bound": "hbm", "achieved": kern["mpgemm_gbps"], "peak": HBM_PEAK_GBPS, "unit": "GB/s",
               "frac": kern["hbm_frac"], "traffic": load_traffic(head.name, "mpgemm"),
               "kernel": "lut_gemv2_kernel (lutgemm_mpgemm, tables from HBM)",
               "algorithmic_bytes_per_launch": kern["algorithmic_bytes"], "avg_launch_us": kern["mpgemm_us"]}
    result = {
        "metric": METRIC,
        "value": round(head.effective_tops(ms_step), 4),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": K,
        "warmup": WU,
        "ms_per_step": round(ms_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic",
        "config": {"workload": head.name, "M": 1, "K": 4096, "N": 4096,
                   "weights": "ternary {-1,0,1} as 2-bit planes, per-tensor FP32 scale",
                   "activations": "FP16 N(0,1) -> per-token absmax INT8", "accumulate": "INT32",
                   "output": "FP32 (float(acc) s_a) s_w",
                   "step": "lutgemm_mpgemm_fused: INT8 quantization + table build in LDS + bit-serial "
                           "lookup + epilogue, one kernel"},
        "timing": "K back-to-back steps timed between HIP events on the launch stream, each timed batch on its "
                  "own slice of a >= 1 GiB rotation set of packed-weight copies (every step reads its weights "
                  "from HBM whatever K is), median over >= 5 batches, two ways: 'graph' captures the K steps in "
                  "a HIP graph and replays it (a replay carries a fixed launch cost of about 10 us); 'queued' "
                  "launches them one by one behind a bounded spin kernel that holds the stream until the host "
                  "has enqueued them all, so the interval holds their device execution and dispatch only; "
                  "ms_per_step is the faster of the two (both reported); ms_per_step_eager launches the same "
                  "steps one by one from Python with the device waiting on the host",
        "step_timing": step_timing,
        "ms_per_step_graph": round(ms_step_graph, 6),
        "ms_per_step_queued": round(ms_step_queued, 6),
        "queued_hold_late_batches": queued_late,
        "timed_replays": step_replays,
        "distinct_weight_bytes_timed": step_distinct,
        "ms_per_step_eager": round(ms_step_eager, 6),
        "single_call_cold_us": cold_us,
        "hbm_gbps_step": achieved,
        "roofline": roofline,
        "two_call_step": {"entries": "lutgemm_precompute + lutgemm_mpgemm (tables through HBM)",
                          "ms_per_step": round(ms_two, 6), "ms_per_step_graph": round(ms_two_graph, 6),
                          "ms_per_step_queued": round(ms_two_queued, 6), "ms_per_step_eager": round(ms_two_eager, 6),
                          "tops": round(head.effective_tops(ms_two), 4), "mpgemm_roofline": mp_roof},
        "headline_kernels": kern,
    }
    head_inp, head_name = head.inp, head.name
    head.release()
    del head

    if args.calibrate_copy:
        result["copy_calibration"] = calibrate_copy()

    # ---------------- the other workload shapes
    if not args.quick:
        recs = []
        # the headline shape with its ternary weights packed three per 5 bits
        if not args.only or args.only == head_name + "_3in5":
            c = Case(2, 0, 1, wfmt=L.WFMT_TERNARY_3IN5)
            recs.append(c.measure(200, 3))
            log(f"{c.name}: mpgemm {recs[-1]['mpgemm_us']} us, fused {recs[-1]['fused_us']} us")
            c.release()
            del c
        # INT8 table quantization on a decode shape and on the prefill shape
        for cid, sid, M in ((3, 1, 1), (4, 0, 4096)):
            if args.only and case_name(cid, sid, M, lut8=True) != args.only:
                continue
            c = Case(cid, sid, M, act=W.ACT_FP16_LUT8)
            recs.append(c.measure(200 if M == 1 else 5, 3))
            log(f"{c.name}: mpgemm {recs[-1]['mpgemm_us']} us, precompute {recs[-1]['precompute_us']} us")
            c.release()
            del c
        for cid, w in W.WORKLOADS.items():
            for (sid, M, Kd, N) in w.shapes():
                if cid == 2 or (args.only and case_name(cid, sid, M) != args.only):
                    continue
                c = Case(cid, sid, M)
                n = 200 if M == 1 else (20 if M <= 256 else 5)
                recs.append(c.measure(n, 3))
                log(f"{c.name}: mpgemm {recs[-1]['mpgemm_us']} us, {recs[-1]['mpgemm_gbps']} GB/s")
                c.release()
                del c
        result["workloads"] = recs

    if not args.no_cpu:
        log("CPU oracle baseline")
        result["cpu_baseline"] = cpu_baseline(head_inp)
        log("CPU oracle on one core, configs 1-3")
        result["cpu_baseline_1core"] = cpu_baseline_single_core()
    result["paper_context"] = PAPER_CONTEXT
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
