"""GPU parity of lutgemm_mpgemm_fused (table precompute fused into the LUT kernel).

The fused path is compared with the CPU oracle (INT8 activations bit-exactly, FP16
activations within the FP tolerance) and, for INT8 activations, with the two-call
path (lutgemm_precompute + lutgemm_mpgemm) bitwise.  Cases cover one and two
tokens, a single K chunk, several K chunks (K = 11008), K split across
workgroups (few columns), ragged column tails, every weight format, accumulate,
determinism, the zero token, the split-K kernel that builds FP32 tables from the
activations (large layers; INT8 activations: every workgroup reads the whole token for
the absmax), and the two-call path behind the same entry point (INT8 activations with
M > 2).
"""
import numpy as np
import pytest

import oracle
import workloads as W
from helpers import GpuProblem, assert_fp_close, sample_indices

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2408_06003_amd as L  # noqa: E402


def banner(msg):
    print(f"\n[case] {msg}", flush=True)


def check_fused(gp, rows=None, cols=None, what=""):
    inp = gp.inp
    if inp.act_kind == W.ACT_INT8:
        acc_ref, y_ref = oracle.reference_output(inp, rows=rows, cols=cols)
        yi = gp.fused(out_dtype=torch.int32).cpu().numpy()
        yf = gp.fused(out_dtype=torch.float32).cpu().numpy()
        # the two-call path gives the same bits
        assert np.array_equal(yi, gp.lut(out_dtype=torch.int32).cpu().numpy()), f"{what}: fused INT32 != two-call"
        assert np.array_equal(yf, gp.lut(out_dtype=torch.float32).cpu().numpy()), f"{what}: fused FP32 != two-call"
        if rows is not None:
            yi, yf = yi[np.ix_(rows, cols)], yf[np.ix_(rows, cols)]
        assert np.array_equal(yi.astype(np.int64), acc_ref), f"{what}: INT32 accumulator differs from the oracle"
        assert np.array_equal(yf, y_ref), f"{what}: FP32 output differs from the oracle"
        return
    ref = oracle.reference_output(inp, rows=rows, cols=cols)
    for od in (torch.float16, torch.float32):
        y = gp.fused(out_dtype=od).float().cpu().numpy()
        if rows is not None:
            y = y[np.ix_(rows, cols)]
        fro, mx = assert_fp_close(y, ref, f"{what} fused {od}")
        print(f"[err] {what} fused {od}: relFro {fro:.3e} max/rms {mx:.3e}", flush=True)


CASES = [
    # (family, M, K, N): single chunk, several chunks, K split (few columns), ragged tails
    (1, 1, 1024, 1000),
    (1, 2, 1024, 300),
    (2, 1, 4096, 4096),
    (2, 1, 2560, 700),   # INT8, 4 wavefronts: 20 of the chunk's 32 blocks
    (2, 2, 3968, 300),   # INT8, 4 wavefronts, 31 blocks, two tokens
    (2, 1, 4096, 300),   # INT8, 4 wavefronts, K split (few column tiles)
    (2, 2, 2048, 777),
    (2, 1, 8192, 1000),
    (3, 1, 4096, 1000),
    (3, 1, 11008, 520),
    (3, 1, 11008, 1000),
    (3, 2, 2048, 33),
    (5, 1, 2048, 1000),
    (5, 2, 4096, 130),
]


@pytest.mark.parametrize("cid,M,K,N", CASES)
def test_fused_parity(cid, M, K, N):
    banner(f"fused parity config={cid} M={M} K={K} N={N}")
    gp = GpuProblem(W.make_inputs(cid, 0, M=M, K=K, N=N))
    print(f"[ws] fused workspace {L.fused_workspace_size(gp.p, M)} B", flush=True)
    check_fused(gp, what=f"config {cid} M={M} K={K} N={N}")


@pytest.mark.parametrize("wfmt,bits,G,act", [(W.WFMT_UINT, 1, 128, W.ACT_FP16), (W.WFMT_UINT, 2, 256, W.ACT_FP16),
                                             (W.WFMT_UINT, 4, 1024, W.ACT_FP16), (W.WFMT_TERNARY, 2, 128, W.ACT_FP16),
                                             (W.WFMT_BINARY, 1, 2048, W.ACT_INT8), (W.WFMT_TERNARY, 2, 0, W.ACT_INT8)])
def test_fused_formats_and_groups(wfmt, bits, G, act):
    banner(f"fused formats wfmt={wfmt} b={bits} G={G} act={act}")
    inp = W.make_custom(wfmt, bits, G, act, M=1, K=2048, N=640, seed=91, scale_fp32=(G == 0))
    check_fused(GpuProblem(inp), what=f"wfmt={wfmt} b={bits} G={G}")


def test_fused_fallback_paths():
    """M = 5 with FP16 activations takes the multi-token kernel with its own table
    build (tests/test_gpu_fused_mtok.py covers it in depth); INT8 activations with
    M > 2 run precompute + mpGEMM behind the same entry point."""
    banner("fused entry point: M = 5 FP16 (multi-token build), INT8 M = 6 (two-call path)")
    gp = GpuProblem(W.make_inputs(3, 0, M=5, K=2048, N=700))
    check_fused(gp, what="M=5")
    gpi = GpuProblem(W.make_custom(W.WFMT_TERNARY, 2, 0, W.ACT_INT8, M=6, K=2048, N=300, seed=93, scale_fp32=True))
    check_fused(gpi, what="INT8 M=6")


def test_fused_int8_large_weights_full_size():
    """Ternary INT8 at 1 x 8192 x 28672 (58 MB of weights: the planned split-K kernel),
    bitwise against the two-call path, sampled columns against the oracle."""
    inp = W.make_custom(W.WFMT_TERNARY, 2, 0, W.ACT_INT8, M=1, K=8192, N=28672, seed=141, scale_fp32=True)
    banner("fused INT8 split-K full size 1x8192x28672")
    gp = GpuProblem(inp)
    assert L.fused_workspace_size(gp.p, 1) < L.table_size(gp.p, 1) + L.workspace_size(gp.p, 1)
    rows, cols = sample_indices(1, inp.N, seed=141)
    check_fused(gp, rows=rows, cols=cols, what="INT8 1x8192x28672")


@pytest.mark.parametrize("cid,sid", [(1, 0), (2, 0), (3, 0), (3, 1), (3, 2), (3, 3), (5, 0), (5, 1)])
def test_fused_full_size(cid, sid):
    inp = W.make_inputs(cid, sid, M=1)
    banner(f"fused full size config={cid} shape={sid} K={inp.K} N={inp.N}")
    gp = GpuProblem(inp)
    if inp.act_kind == W.ACT_INT8:
        check_fused(gp, what=f"config {cid}/{sid}")
        return
    rows, cols = sample_indices(1, inp.N, seed=cid * 100 + sid)
    check_fused(gp, rows=rows, cols=cols, what=f"config {cid}/{sid}")


def test_fused_zero_token_accumulate_determinism():
    banner("fused: zero token, accumulate, determinism")
    inp = W.make_inputs(2, 0, M=2, K=4096, N=1000)
    inp.act[1] = 0
    gp = GpuProblem(inp)
    check_fused(gp, what="zero second token")
    y1 = gp.fused(out_dtype=torch.float32)
    y2 = gp.fused(out_dtype=torch.float32)
    assert torch.equal(y1, y2)
    bi = torch.randint(-1000, 1000, (2, 1000), device="cuda", dtype=torch.int32)
    acc = bi.clone()
    gp.fused(out=acc, accumulate=True)
    assert torch.equal(acc, bi + gp.fused(out_dtype=torch.int32))
    inpf = W.make_inputs(3, 0, M=1, K=4096, N=1000)
    gpf = GpuProblem(inpf)
    f1 = gpf.fused(out_dtype=torch.float32)
    assert torch.equal(f1, gpf.fused(out_dtype=torch.float32)), "fused FP path not deterministic"
    base = torch.randn(1, 1000, device="cuda")
    accf = base.clone()
    gpf.fused(out=accf, accumulate=True)
    assert torch.equal(accf, base + f1)


@pytest.mark.parametrize("cid,M,K,N", [(3, 1, 4096, 1000), (3, 2, 11008, 300), (5, 1, 8192, 700),
                                       (1, 1, 1024, 1000), (1, 2, 2048, 257)])
def test_fused_split_k_parity(cid, M, K, N, tune):
    """The split-K GEMV with its tables built from the activations (FP path: FP32 entries,
    no token scaling), forced at reduced sizes: ragged column tails, one and two tokens,
    K split into many workgroups, zero points per 128-block."""
    tune(GEMV_KIND=2)
    banner(f"fused split-K config={cid} M={M} K={K} N={N}")
    gp = GpuProblem(W.make_inputs(cid, 0, M=M, K=K, N=N))
    check_fused(gp, what=f"split-K config {cid} M={M} K={K} N={N}")


@pytest.mark.parametrize("wfmt,bits,G,sf,M,K,N,kbs", [
    (W.WFMT_TERNARY, 2, 0, True, 1, 4096, 1000, 0),     # ternary, per-tensor FP32 scale, planned K ranges
    (W.WFMT_TERNARY, 2, 0, True, 2, 8192, 300, 0),      # two tokens, ragged columns
    (W.WFMT_BINARY, 1, 0, True, 1, 4096, 777, 0),       # binary per-tensor
    (W.WFMT_BINARY, 1, 2048, False, 2, 2048, 520, 0),   # binary per-channel FP16 scale
    (W.WFMT_TERNARY, 2, 0, True, 1, 8192, 600, 1),      # 64 K ranges: the finalize kernel, token factor from the workspace
    (W.WFMT_TERNARY, 2, 0, True, 2, 4096, 300, 2),      # 16 K ranges, completed in the kernel
])
def test_fused_split_k_int8(wfmt, bits, G, sf, M, K, N, kbs, tune):
    """INT8 activations on the split-K kernel: every workgroup reads the whole token for
    the absmax and builds the exact INT16 entries of its K range; bitwise against the
    two-call path and the oracle (check_fused), including a zero token and a token
    whose absmax sits in another workgroup's K range."""
    tune(GEMV_KIND=2, KBS=kbs)
    banner(f"fused split-K INT8 wfmt={wfmt} b={bits} G={G} M={M} K={K} N={N} kbs={kbs or 'planned'}")
    inp = W.make_custom(wfmt, bits, G, W.ACT_INT8, M=M, K=K, N=N, seed=131 + bits + K // 1024, scale_fp32=sf)
    a = inp.act.astype(np.float32)
    a[0, K - 5] = 9.0  # the token's absmax in the last K range only
    if M > 1:
        a[1] = 0.0      # a zero token: factor 0, zero output
    inp.act = a.astype(np.float16)
    gp = GpuProblem(inp)
    check_fused(gp, what=f"split-K INT8 wfmt={wfmt} M={M} K={K}")
    if M > 1:
        assert not gp.fused(out_dtype=torch.int32)[1].any()


@pytest.mark.parametrize("wfmt,bits,G", [(W.WFMT_UINT, 1, 128), (W.WFMT_UINT, 2, 1024), (W.WFMT_UINT, 4, 512),
                                         (W.WFMT_TERNARY, 2, 128), (W.WFMT_BINARY, 1, 2048)])
def test_fused_split_k_formats(wfmt, bits, G, tune):
    tune(GEMV_KIND=2)
    banner(f"fused split-K formats wfmt={wfmt} b={bits} G={G}")
    inp = W.make_custom(wfmt, bits, G, W.ACT_FP16, M=1, K=2048, N=640, seed=97)
    inp.act[0] *= np.float16(300)  # large activations: the FP32 tables need no token scaling
    gp = GpuProblem(inp)
    check_fused(gp, what=f"split-K wfmt={wfmt} b={bits} G={G}")
    f1 = gp.fused(out_dtype=torch.float32)
    assert torch.equal(f1, gp.fused(out_dtype=torch.float32)), "fused split-K not deterministic"
    base = torch.randn(1, 640, device="cuda")
    acc = base.clone()
    gp.fused(out=acc, accumulate=True)
    assert torch.equal(acc, base + f1)
