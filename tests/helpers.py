"""Shared helpers for the GPU parity tests: run the HIP path, compare with the oracle."""
from __future__ import annotations

import numpy as np

import workloads as W

# Tolerances for FP16-activation / FP32-accumulate results: relative Frobenius
# error and max-abs error normalized by the RMS of the reference.  The paper gives
# no error bound; FP16 table entries (relative 2^-11 each) and FP16 outputs put the
# expected error at a few times 1e-4 for N(0,1) activations, well inside these.
REL_FRO_TOL = 2e-3
MAX_ABS_OVER_RMS_TOL = 1e-2


def problem_of(inp, wfmt=None):
    """The C-ABI problem of ``inp``; ``wfmt`` overrides the weight format (the
    ternary 3-in-5 packing of the same ternary codes)."""
    import paper_2408_06003_amd as L
    return L.problem(inp.K, inp.N, inp.bits, inp.wfmt if wfmt is None else wfmt, inp.group,
                     act=inp.act_kind, scale_fp32=(inp.scales.dtype == np.float32))


def to_dev(x):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


class GpuProblem:
    """Device copies of one workload plus its packed weights."""

    def __init__(self, inp, wfmt=None):
        import paper_2408_06003_amd as L
        self.inp = inp
        self.p = problem_of(inp, wfmt)
        assert L.validate(self.p, inp.M) == L.SUCCESS, L.status_string(L.validate(self.p, inp.M))
        self.codes = to_dev(inp.codes)
        self.scales = to_dev(inp.scales)
        self.zeros = None if inp.zeros is None else to_dev(inp.zeros)
        self.act = to_dev(inp.act)
        self.g = L.LutGemm(self.p, self.codes, self.scales, self.zeros)

    def lut(self, out_dtype=None, accumulate=False, out=None, act=None):
        import torch
        a = self.act if act is None else act
        od = out_dtype or (torch.int32 if self.inp.act_kind == W.ACT_INT8 else torch.float16)
        y = self.g(a, out=out, out_dtype=od, accumulate=accumulate)
        torch.cuda.synchronize()
        return y

    def fused(self, out_dtype=None, accumulate=False, out=None, act=None):
        import torch
        a = self.act if act is None else act
        od = out_dtype or (torch.int32 if self.inp.act_kind == W.ACT_INT8 else torch.float16)
        y = self.g.fused(a, out=out, out_dtype=od, accumulate=accumulate)
        torch.cuda.synchronize()
        return y

    def dequant(self, out_dtype=None, accumulate=False, out=None):
        import torch
        y = self.g.dequant(self.act, out=out, out_dtype=out_dtype or torch.float16, accumulate=accumulate)
        torch.cuda.synchronize()
        return y


class tuning:
    """Context manager: planner overrides (``paper_2408_06003_amd.TUNE`` names) for the
    duration of a block, restored to their previous values afterwards."""

    def __init__(self, **kw):
        self.kw = kw

    def __enter__(self):
        import paper_2408_06003_amd as L
        self.old = {k: L.get_tuning(k) for k in self.kw}
        for k, v in self.kw.items():
            L.set_tuning(k, v)
        return self

    def __exit__(self, *exc):
        import paper_2408_06003_amd as L
        for k, v in self.old.items():
            L.set_tuning(k, v)
        return False


def fp_errors(y, ref):
    y = np.asarray(y, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    diff = y - ref
    fro = np.linalg.norm(diff) / max(np.linalg.norm(ref), 1e-300)
    rms = np.sqrt(np.mean(ref * ref)) if ref.size else 0.0
    mx = np.abs(diff).max() / max(rms, 1e-300) if diff.size else 0.0
    return float(fro), float(mx)


def assert_fp_close(y, ref, what=""):
    fro, mx = fp_errors(y, ref)
    assert np.all(np.isfinite(np.asarray(y, dtype=np.float64))), f"{what}: non-finite output"
    assert fro <= REL_FRO_TOL, f"{what}: relative Frobenius error {fro:.3e} > {REL_FRO_TOL}"
    assert mx <= MAX_ABS_OVER_RMS_TOL, f"{what}: max-abs/rms {mx:.3e} > {MAX_ABS_OVER_RMS_TOL}"
    return fro, mx


def sample_indices(M, N, seed, n_rows=4, n_cols=384):
    rng = np.random.default_rng(seed)
    rows = sorted(set(rng.choice(M, size=min(M, n_rows), replace=False).tolist()) | {M - 1})
    cols = sorted(set(rng.choice(N, size=min(N, n_cols), replace=False).tolist()) | {0, N - 1})
    return np.array(rows, dtype=np.int64), np.array(cols, dtype=np.int64)
