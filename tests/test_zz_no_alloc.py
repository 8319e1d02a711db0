"""The allocation-free entry point (lutgemm_mpgemm_noalloc) against lutgemm_mpgemm.

Both run the same kernels; the no-alloc variant keeps the K-split partial sums in
the library's static scratch array instead of a caller workspace.  Two calls in a
row on different problems (the second smaller) must each give exactly what
lutgemm_mpgemm gives with its own workspace, and that output must meet the parity
bar against the oracle (bit-exact on the INT8 path, the FP tolerance otherwise).
A problem whose partial sums exceed the array is rejected before any launch.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from helpers import GpuProblem, assert_fp_close

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2408_06003_amd as L  # noqa: E402


def run_both(gp, out_dtype):
    """(lutgemm_mpgemm with a torch workspace, lutgemm_mpgemm_noalloc) outputs."""
    inp, p, M = gp.inp, gp.p, gp.inp.M
    tables = gp.g.tables(M)
    L.precompute(p, M, gp.act, tables)
    code = gp.g.out_dtype_code(out_dtype)
    ref = torch.full((M, inp.N), 7, dtype=out_dtype, device="cuda")
    ws = gp.g.workspace(M)
    L.mpgemm(p, M, tables, gp.g.packed, ref, code, False, workspace=ws)
    y = torch.full((M, inp.N), -3, dtype=out_dtype, device="cuda")
    L.mpgemm_noalloc(p, M, tables, gp.g.packed, y, code, False)
    torch.cuda.synchronize()
    return ref, y


CASES = [
    # first call: K split into many workgroups (large partial-sum buffer)
    ("binary 1x8192x28672", lambda: W.make_inputs(5, 0, M=1)),
    # second call: a smaller problem on the same scratch
    ("INT4 1x4096x4096 split", lambda: W.make_inputs(3, 1, M=1, N=1000)),
]


@pytest.mark.parametrize("exact", [0, 1])
def test_noalloc_matches_mpgemm_two_calls(exact):
    """Both K-split completions of the split-K kernel on the static scratch: partial
    sums and arrival counters (exact = 0), or only the exact split-sum words (1)."""
    L.set_tuning("GEMV_KIND", 2)  # the split-K kernel, so both calls use the scratch
    L.set_tuning("SPLIT_EXACT", exact)
    try:
        sizes = []
        for name, make in CASES:
            print(f"\n[case] noalloc {name} exact={exact}", flush=True)
            inp = make()
            gp = GpuProblem(inp)
            need = L.workspace_size(gp.p, inp.M)
            assert 0 < need <= (16 << 20)
            sizes.append(need)
            ref, y = run_both(gp, torch.float16)
            assert torch.equal(ref, y), f"{name}: no-alloc output differs from lutgemm_mpgemm"
            rows, cols = np.arange(inp.M), np.unique(np.linspace(0, inp.N - 1, 512).astype(np.int64))
            want = oracle.reference_output(inp, rows=rows, cols=cols)
            assert_fp_close(y.float().cpu().numpy()[np.ix_(rows, cols)], want, f"noalloc {name}")
        if exact:
            assert sizes[1] == sizes[0] == L.WORKSPACE_ZERO_BYTES
        else:
            assert sizes[1] < sizes[0]
    finally:
        L.set_tuning("GEMV_KIND", -1)
        L.set_tuning("SPLIT_EXACT", -1)


def test_noalloc_int8_path_bit_exact():
    print("\n[case] noalloc ternary INT8 1x4096x4096 split", flush=True)
    L.set_tuning("GEMV_KIND", 2)
    try:
        inp = W.make_inputs(2, 0, M=1)
        gp = GpuProblem(inp)
        ref, y = run_both(gp, torch.int32)
        assert torch.equal(ref, y)
        acc_ref, _ = oracle.reference_output(inp)
        assert np.array_equal(y.cpu().numpy().astype(np.int64), acc_ref)
    finally:
        L.set_tuning("GEMV_KIND", -1)


def test_noalloc_rejects_oversized_scratch():
    print("\n[case] noalloc oversized", flush=True)
    p = L.problem(28672, 8192, 1, L.WFMT_BINARY, 28672)
    need = L.workspace_size(p, 256)
    assert need > (16 << 20)
    out = torch.zeros((256, 8192), dtype=torch.float16, device="cuda")
    dummy = torch.zeros(256, dtype=torch.uint8, device="cuda")
    st = L.lib.lutgemm_mpgemm_noalloc(__import__("ctypes").byref(p), 256, dummy.data_ptr(), dummy.data_ptr(),
                                      out.data_ptr(), L.OUT_FP16, 0, torch.cuda.current_stream().cuda_stream)
    assert st == L.ERROR_NOT_SUPPORTED
    assert "scratch" in L.lib.lutgemm_last_error().decode()
    torch.cuda.synchronize()
    assert not out.any()
