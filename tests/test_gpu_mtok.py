"""Multi-token LUT kernel (M >= 3) across metadata layouts, group sizes, ragged chunks
and forced K splits: every output against the oracle (FP paths within the FP bar,
INT8 path bit-exact), FP16 and FP32 outputs, and run-to-run bitwise determinism.

The cases are chosen for the kernel's bookkeeping: the zero-point term of Eq. 3
enters once per quantization group (groups of 4 blocks split mid-group, per-tensor
groups that only the first split sees), chunks of two 128-blocks with an odd block
count, token tiles of 8 with 3 and 5 live rows, and K splits that leave a short last
range.
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import workloads as W
from helpers import GpuProblem, assert_fp_close

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2408_06003_amd as L  # noqa: E402,F401  (fails loudly when the HIP library is missing)

FP_CASES = [
    # (weight format, bits, group, FP32 per-tensor scale, M, K, N, forced K splits)
    (W.WFMT_TERNARY, 2, 0, True, 11, 2048, 300, 0),     # per-tensor FP32 s, z' = -1
    (W.WFMT_TERNARY, 2, 0, True, 11, 2048, 300, 3),     # ... zero-point term in the first split only
    (W.WFMT_UINT, 2, 512, False, 9, 2048, 520, 3),      # groups of 4 blocks, splits of 6 blocks
    (W.WFMT_UINT, 4, 1024, False, 20, 1024, 257, 2),    # per-channel, one block per chunk
    (W.WFMT_BINARY, 1, 256, False, 13, 1536, 300, 5),   # binary group scales (z' = 0)
    (W.WFMT_UINT, 1, 128, False, 8, 1152, 300, 0),      # 9 blocks: the last chunk holds one
    (W.WFMT_UINT, 2, 128, False, 3, 1152, 64, 2),       # 3 live rows of 8, a single column tile
    (W.WFMT_UINT, 4, 256, False, 45, 2048, 700, 0),     # 5 live rows in the last token tile
]


@pytest.mark.parametrize("mt16", [1, 0])
@pytest.mark.parametrize("wfmt,bits,G,fp32,M,K,N,splits", FP_CASES)
def test_multi_token_fp_layouts(wfmt, bits, G, fp32, M, K, N, splits, mt16, tune):
    """mt16 = 0 keeps 8-token workgroups where 16-token ones would be used (M >= 16)."""
    if splits:
        tune(MT_SPLITS=splits)
    tune(MT16=mt16)
    what = f"wfmt={wfmt} b={bits} G={G} M={M} K={K} N={N} splits={splits}"
    print(f"\n[case] multi-token FP {what}", flush=True)
    inp = W.make_custom(wfmt, bits, G, W.ACT_FP16, M=M, K=K, N=N, seed=M + K + N + splits, scale_fp32=fp32)
    gp = GpuProblem(inp)
    ref = oracle.reference_output(inp)
    y32 = gp.lut(out_dtype=torch.float32)
    fro, mx = assert_fp_close(y32.cpu().numpy(), ref, what)
    print(f"[err] {what}: relFro {fro:.3e} max/rms {mx:.3e}", flush=True)
    assert_fp_close(gp.lut(out_dtype=torch.float16).float().cpu().numpy(), ref, what + " fp16 out")
    assert torch.equal(gp.lut(out_dtype=torch.float32), y32), f"{what}: two runs differ bitwise"


INT_CASES = [
    # (weight format, bits, group, FP32 per-tensor scale, M, K, N, forced K splits)
    (W.WFMT_TERNARY, 2, 0, True, 10, 1152, 300, 3),
    (W.WFMT_TERNARY, 2, 0, True, 21, 2048, 513, 0),
    (W.WFMT_BINARY, 1, 1536, False, 9, 1536, 300, 2),
]


@pytest.mark.parametrize("wfmt,bits,G,fp32,M,K,N,splits", INT_CASES)
def test_multi_token_int8_layouts(wfmt, bits, G, fp32, M, K, N, splits, tune):
    if splits:
        tune(MT_SPLITS=splits)
    print(f"\n[case] multi-token INT8 wfmt={wfmt} b={bits} G={G} M={M} K={K} N={N} splits={splits}", flush=True)
    inp = W.make_custom(wfmt, bits, G, W.ACT_INT8, M=M, K=K, N=N, seed=M + K + N + splits, scale_fp32=fp32)
    gp = GpuProblem(inp)
    acc_ref, y_ref = oracle.reference_output(inp)
    yi = gp.lut(out_dtype=torch.int32).cpu().numpy()
    yf = gp.lut(out_dtype=torch.float32).cpu().numpy()
    assert np.array_equal(yi.astype(np.int64), acc_ref), "INT32 accumulator differs from the oracle"
    assert np.array_equal(yf, y_ref), "FP32 scaled output differs from the oracle"


FOUR_CASES = [
    # (weight format, bits, group, FP32 per-tensor scale, activations, M, K, N, forced K splits)
    (W.WFMT_UINT, 2, 128, False, W.ACT_FP16, 4, 2048, 520, 0),    # INT2 g128, 4 live rows
    (W.WFMT_UINT, 4, 512, False, W.ACT_FP16, 3, 2560, 300, 3),    # INT4, groups of 4 blocks split mid-group, 3 rows
    (W.WFMT_UINT, 1, 0, False, W.ACT_FP16, 4, 1152, 257, 0),      # UINT1 per-channel, 9 blocks
    (W.WFMT_BINARY, 1, 256, False, W.ACT_FP16, 3, 4096, 1000, 0),  # binary group scales
    (W.WFMT_TERNARY, 2, 0, True, W.ACT_FP16, 4, 2048, 300, 5),    # per-tensor FP32 scale, z' = -1
    (W.WFMT_TERNARY, 2, 0, True, W.ACT_INT8, 4, 2048, 513, 3),    # INT8: exact
    (W.WFMT_BINARY, 1, 1536, False, W.ACT_INT8, 3, 1536, 300, 0),
]


@pytest.mark.parametrize("wfmt,bits,G,fp32,act,M,K,N,splits", FOUR_CASES)
def test_multi_token_four_token_tiles(wfmt, bits, G, fp32, act, M, K, N, splits, tune):
    """M <= 4 takes 4-token tiles (half-filled rows, 8-byte reads): against the oracle,
    and against the 8-token tiles of the same call (bitwise on the INT8 path, within
    the FP bar on the FP path: the same entries summed in the same order per token)."""
    if splits:
        tune(MT_SPLITS=splits)
    what = f"4-token tiles wfmt={wfmt} b={bits} G={G} act={act} M={M} K={K} N={N} splits={splits}"
    print(f"\n[case] {what}", flush=True)
    inp = W.make_custom(wfmt, bits, G, act, M=M, K=K, N=N, seed=7 * M + K + N + splits, scale_fp32=fp32)
    gp = GpuProblem(inp)
    tune(MT4=1)
    if act == W.ACT_INT8:
        acc_ref, y_ref = oracle.reference_output(inp)
        yi = gp.lut(out_dtype=torch.int32)
        assert np.array_equal(yi.cpu().numpy().astype(np.int64), acc_ref), f"{what}: INT32 accumulator differs"
        assert np.array_equal(gp.lut(out_dtype=torch.float32).cpu().numpy(), y_ref), f"{what}: FP32 output differs"
        tune(MT4=0)
        assert torch.equal(gp.lut(out_dtype=torch.int32), yi), f"{what}: 4- and 8-token tiles differ"
        return
    ref = oracle.reference_output(inp)
    y4 = gp.lut(out_dtype=torch.float32)
    fro, mx = assert_fp_close(y4.cpu().numpy(), ref, what)
    print(f"[err] {what}: relFro {fro:.3e} max/rms {mx:.3e}", flush=True)
    assert torch.equal(gp.lut(out_dtype=torch.float32), y4), f"{what}: two runs differ bitwise"
    assert_fp_close(gp.fused(out_dtype=torch.float32).cpu().numpy(), ref, what + " fused")
    tune(MT4=0)
    y8 = gp.lut(out_dtype=torch.float32)
    assert torch.equal(y8, y4), f"{what}: 4- and 8-token tiles differ"


@pytest.mark.parametrize("M", [5, 17])
@pytest.mark.parametrize("splits", [5, 9, 17, 33, 65, 128])
def test_multi_token_many_splits(splits, M, tune):
    """K split into 5 .. 128 ranges: the finalize kernel's load batch (4 .. 64 partials,
    looping when there are more) at every size it takes, FP and INT8 paths, with 8-token
    (M = 5) and 16-token (M = 17: one full tile and one with a single live row) workgroups."""
    tune(MT_SPLITS=splits)
    print(f"\n[case] multi-token K splits={splits} (M={M}, K=16384, N=200)", flush=True)
    inp = W.make_custom(W.WFMT_BINARY, 1, 16384, W.ACT_FP16, M=M, K=16384, N=200, seed=300 + splits)
    gp = GpuProblem(inp)
    ref = oracle.reference_output(inp)
    y32 = gp.lut(out_dtype=torch.float32)
    assert_fp_close(y32.cpu().numpy(), ref, f"splits={splits}")
    assert torch.equal(gp.lut(out_dtype=torch.float32), y32), f"splits={splits}: two runs differ bitwise"
    inpi = W.make_custom(W.WFMT_TERNARY, 2, 0, W.ACT_INT8, M=M, K=16384, N=200, seed=400 + splits,
                         scale_fp32=True)
    gpi = GpuProblem(inpi)
    acc_ref, y_ref = oracle.reference_output(inpi)
    assert np.array_equal(gpi.lut(out_dtype=torch.int32).cpu().numpy().astype(np.int64), acc_ref)
    assert np.array_equal(gpi.lut(out_dtype=torch.float32).cpu().numpy(), y_ref)


@pytest.mark.parametrize("order", [1, 8, 16])
def test_multi_token_tile_orders(order, tune):
    """XCD-aware workgroup orders (token-fastest, bands of 8 or 16 token tiles) over a
    grid whose token tiles do not fill the last band, every output against the oracle."""
    tune(MT_ORDER=order)
    tune(MT_SPLITS=1)
    print(f"\n[case] multi-token tile order {order} (M=300, K=1024, N=520)", flush=True)
    inp = W.make_custom(W.WFMT_UINT, 2, 128, W.ACT_FP16, M=300, K=1024, N=520, seed=500 + order)
    gp = GpuProblem(inp)
    assert_fp_close(gp.lut(out_dtype=torch.float32).cpu().numpy(), oracle.reference_output(inp), f"order {order}")


@pytest.mark.parametrize("splits", [1, 3])
@pytest.mark.parametrize("M", [10, 20])
def test_multi_token_accumulate(M, splits, tune):
    """O += A W^T through the multi-token kernel's own epilogue (one split) and through the
    finalize kernel (three splits), FP32 and FP16 outputs, and the INT8 path's INT32 output."""
    tune(MT_SPLITS=splits)
    print(f"\n[case] multi-token accumulate M={M} splits={splits}", flush=True)
    inp = W.make_custom(W.WFMT_UINT, 2, 128, W.ACT_FP16, M=M, K=1024, N=300, seed=600 + M + splits)
    gp = GpuProblem(inp)
    y1 = gp.lut(out_dtype=torch.float32)
    base = torch.randn(M, 300, device="cuda", dtype=torch.float32)
    acc = base.clone()
    gp.lut(out=acc, accumulate=True)
    assert torch.equal(acc, base + y1), "FP32 accumulate is not O + A W^T"
    base16 = torch.randn(M, 300, device="cuda", dtype=torch.float32).half()
    acc16 = base16.clone()
    gp.lut(out=acc16, accumulate=True)
    assert torch.equal(acc16, (base16.float() + y1).half()), "FP16 accumulate is not round(O + A W^T)"
    inpi = W.make_custom(W.WFMT_TERNARY, 2, 0, W.ACT_INT8, M=M, K=1024, N=300, seed=700 + M + splits,
                         scale_fp32=True)
    gpi = GpuProblem(inpi)
    bi = torch.randint(-1000, 1000, (M, 300), device="cuda", dtype=torch.int32)
    acci = bi.clone()
    gpi.lut(out=acci, accumulate=True)
    assert torch.equal(acci, bi + gpi.lut(out_dtype=torch.int32)), "INT32 accumulate is not O + acc"


@pytest.mark.parametrize("M,K,N", [(33, 256, 1), (17, 128, 255), (16, 128, 1), (3, 128, 1), (40, 384, 257)])
def test_multi_token_tiny_shapes(M, K, N):
    """Degenerate multi-token shapes: a single output column, a single 128-block of K, a
    ragged column tile, token counts at and just past the 8/16-token tile sizes."""
    print(f"\n[case] multi-token tiny M={M} K={K} N={N}", flush=True)
    inp = W.make_custom(W.WFMT_UINT, 2, 128, W.ACT_FP16, M=M, K=K, N=N, seed=1000 + M + K + N)
    gp = GpuProblem(inp)
    assert_fp_close(gp.lut(out_dtype=torch.float32).cpu().numpy(), oracle.reference_output(inp), "tiny FP")
    inpi = W.make_custom(W.WFMT_TERNARY, 2, 0, W.ACT_INT8, M=M, K=K, N=N, seed=1100 + M + K + N, scale_fp32=True)
    gpi = GpuProblem(inpi)
    acc_ref, y_ref = oracle.reference_output(inpi)
    assert np.array_equal(gpi.lut(out_dtype=torch.int32).cpu().numpy().astype(np.int64), acc_ref)
    assert np.array_equal(gpi.lut(out_dtype=torch.float32).cpu().numpy(), y_ref)
