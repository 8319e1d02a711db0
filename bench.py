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
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "pmc_traffic.txt")
# sources that define each timed kernel and its launch (a PMC traffic record is used
# only while they hash as when the counters were taken)
KERNEL_SOURCES = {
    "mpgemm": ("lut_gemv.hip", "lut_common.h", "lutgemm_internal.h", "api.cpp"),
    "fused": ("lut_fused.hip", "lut_common.h", "lutgemm_internal.h", "api.cpp"),
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
    return ap.parse_args()


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


class Case:
    """One workload shape on the device, with a rotation set of packed weights."""

    def __init__(self, cid, sid, M, rotate=True, wfmt=None, act=None):
        """``wfmt`` overrides the packing of the same codes (the ternary 3-in-5 format),
        ``act`` the table precision of the same FP16 activations (INT8 table quantization)."""
        import torch
        import paper_2408_06003_amd as L
        import workloads as W
        self.torch, self.L, self.W = torch, L, W
        w = W.WORKLOADS[cid]
        self.name = w.name if len(w.kn) == 1 and len(w.ms) == 1 else f"{w.name}_M{M}_K{w.kn[sid][0]}_N{w.kn[sid][1]}"
        self.tri = wfmt == L.WFMT_TERNARY_3IN5
        if self.tri:
            self.name += "_3in5"
        self.inp = W.make_inputs(cid, sid, M=M)
        self.lut8 = act == W.ACT_FP16_LUT8
        if self.lut8:
            self.inp.act_kind = act
            self.name += "_lut8"
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
                              self.L.OUT_FP16, False)

    def step(self, i):
        self.precompute()
        self.mpgemm(i)

    def fused(self, i):
        """The same step through lutgemm_mpgemm_fused (tables built inside the LUT kernel)."""
        if not hasattr(self, "fws"):
            n = self.L.fused_workspace_size(self.p, self.M)
            self.fws = self.torch.empty(n, dtype=self.torch.uint8, device="cuda") if n else None
        self.L.mpgemm_fused(self.p, self.M, self.act, self.packed[i % len(self.packed)], self.out,
                            self.out_code, False, workspace=self.fws)

    def timed(self, fn, n, graph=True, check=None):
        """Average milliseconds per call over n back-to-back calls, timed with HIP events
        on the stream they run on.  With graph=True the n calls are captured once into a
        HIP graph and replayed, so host launch overhead is not counted (the way a decode
        loop runs); ``check`` (a function returning a tensor) compares two replays,
        separated by eager work, with the eager result."""
        torch = self.torch
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        if not graph:
            s = torch.cuda.current_stream()
            torch.cuda.synchronize()
            e0.record(s)
            for i in range(n):
                fn(i)
            e1.record(s)
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) / n
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            for i in range(n):
                fn(i)
        torch.cuda.synchronize()
        if check is not None:
            for _ in range(2):
                fn(n - 1)
                torch.cuda.synchronize()
                ref = check().clone()
                check().zero_()
                g.replay()
                torch.cuda.synchronize()
                if not torch.equal(check(), ref):
                    raise RuntimeError(f"{self.name}: graph replay differs from the eager result")
        g.replay()  # warm replay
        torch.cuda.synchronize()
        s = torch.cuda.current_stream()
        e0.record(s)
        g.replay()
        e1.record(s)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    def effective_tops(self, ms):
        return 2.0 * self.M * self.N * self.K / (ms * 1e-3) / 1e12

    def measure(self, n_kernel, warmup):
        """Kernel-level numbers of this shape: mpGEMM, precompute, and (M >= 16) the comparison path."""
        for i in range(warmup):
            self.step(i)
        self.precompute()
        ms_mp = self.timed(self.mpgemm, n_kernel, check=lambda: self.out)
        ms_pre = self.timed(lambda i: self.precompute(), n_kernel)
        b = algorithmic_bytes(self.inp, self.out_bytes, tri=self.tri, lut8=self.lut8)
        gbps = b["total"] / (ms_mp * 1e-3) / 1e9
        # achievable streaming read of the same byte count, same rotation and timing
        sink = self.torch.zeros(4096, dtype=self.torch.int32, device="cuda")
        wb = self.L.packed_weight_size(self.p)
        ms_rd = self.timed(lambda i: self.L.calibrate_stream_read(self.packed[i % len(self.packed)], wb, sink, 1024),
                           n_kernel)
        ms_fu = self.timed(self.fused, n_kernel, check=lambda: self.out)
        rec = {"workload": self.name, "M": self.M, "K": self.K, "N": self.N, "bits": self.inp.bits,
               "mpgemm_us": round(ms_mp * 1e3, 3), "mpgemm_tops": round(self.effective_tops(ms_mp), 3),
               "mpgemm_gbps": round(gbps, 1), "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4),
               "stream_read_us": round(ms_rd * 1e3, 3),
               "stream_read_gbps": round(wb / (ms_rd * 1e-3) / 1e9, 1),
               "frac_of_stream_read": round(ms_rd / ms_mp, 4),
               "precompute_us": round(ms_pre * 1e3, 3),
               "precompute_over_mpgemm": round(ms_pre / ms_mp, 4),
               "fused_us": round(ms_fu * 1e3, 3), "fused_tops": round(self.effective_tops(ms_fu), 3),
               "algorithmic_bytes": b["total"], "rotation_copies": len(self.packed)}
        if self.M >= 16 and not self.int8 and not self.tri and not self.lut8:
            out = self.torch.empty((self.M, self.N), dtype=self.torch.float16, device="cuda")
            for i in range(3):
                self.dequant(i, out)
            n = max(5, min(n_kernel, 50))
            ms_dq = self.timed(lambda i: self.dequant(i, out), n, check=lambda: out)
            tflops = self.effective_tops(ms_dq)
            rec.update({"dequant_mfma_us": round(ms_dq * 1e3, 3), "dequant_mfma_tops": round(tflops, 2),
                        "dequant_mfma_frac_of_fp16_peak": round(tflops / MFMA_FP16_PEAK_TFLOPS, 4),
                        "lut_over_dequant_time": round(ms_mp / ms_dq, 2)})
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


def main():
    args = parse()
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
    ms_step = head.timed(head.fused, K, check=lambda: head.out)
    ms_step_eager = head.timed(head.fused, K, graph=False)
    ms_two = head.timed(head.step, K, check=lambda: head.out)
    ms_two_eager = head.timed(head.step, K, graph=False)
    kern = head.measure(max(K, 50), 5)
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
        "timing": "HIP graph of the K steps replayed once between HIP events (host launch overhead "
                  "excluded); ms_per_step_eager launches the same steps one by one from Python",
        "ms_per_step_eager": round(ms_step_eager, 6),
        "hbm_gbps_step": achieved,
        "roofline": roofline,
        "two_call_step": {"entries": "lutgemm_precompute + lutgemm_mpgemm (tables through HBM)",
                          "ms_per_step": round(ms_two, 6), "ms_per_step_eager": round(ms_two_eager, 6),
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
            c = Case(cid, sid, M, act=W.ACT_FP16_LUT8)
            if args.only and c.name != args.only:
                c.release()
                continue
            recs.append(c.measure(200 if M == 1 else 5, 3))
            log(f"{c.name}: mpgemm {recs[-1]['mpgemm_us']} us, precompute {recs[-1]['precompute_us']} us")
            c.release()
            del c
        for cid, w in W.WORKLOADS.items():
            for (sid, M, Kd, N) in w.shapes():
                if cid == 2:
                    continue
                c = Case(cid, sid, M)
                if args.only and c.name != args.only:
                    c.release()
                    continue
                n = 200 if M == 1 else (20 if M <= 256 else 5)
                recs.append(c.measure(n, 3))
                log(f"{c.name}: mpgemm {recs[-1]['mpgemm_us']} us, {recs[-1]['mpgemm_gbps']} GB/s")
                c.release()
                del c
        result["workloads"] = recs

    if not args.no_cpu:
        log("CPU oracle baseline")
        result["cpu_baseline"] = cpu_baseline(head_inp)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
