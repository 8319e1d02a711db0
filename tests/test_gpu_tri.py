"""GPU parity of the ternary 3-in-5 weight format (three ternary weights per 5-bit
code, one table lookup per 3 weights).

The same ternary codes drawn for the bit-serial ternary format are packed as
LUTGEMM_WFMT_TERNARY_3IN5 and run through lutgemm_precompute + lutgemm_mpgemm and
through lutgemm_mpgemm_fused; results are compared with the CPU oracle (which sees
only the ternary codes, never a packing): INT8 activations bit-exactly (INT32 and
FP32 outputs), FP16 activations within the FP tolerance.  The fused and two-call
paths must agree bitwise.  Cases: K below one 96-block, K not a multiple of 96
(ragged last block and a triple straddling K), several LDS chunks (K > 4608),
ragged column tails, several tokens, per-tensor FP32 / FP16 and per-channel scales,
accumulate, the zero token, the headline shape at full size.
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

T35 = L.WFMT_TERNARY_3IN5


def banner(msg):
    print(f"\n[case] {msg}", flush=True)


def check(gp, what):
    inp = gp.inp
    if inp.act_kind == W.ACT_INT8:
        acc_ref, y_ref = oracle.reference_output(inp)
        for od in (torch.int32, torch.float32):
            y2 = gp.lut(out_dtype=od).cpu().numpy()
            yf = gp.fused(out_dtype=od).cpu().numpy()
            assert np.array_equal(y2, yf), f"{what}: fused {od} differs from the two-call path"
            if od == torch.int32:
                assert np.array_equal(y2.astype(np.int64), acc_ref), f"{what}: INT32 accumulator differs"
            else:
                assert np.array_equal(y2, y_ref), f"{what}: FP32 output differs"
        return
    ref = oracle.reference_output(inp)
    for od in (torch.float16, torch.float32):
        y2 = gp.lut(out_dtype=od)
        yf = gp.fused(out_dtype=od)
        assert torch.equal(y2, yf), f"{what}: fused {od} differs from the two-call path"
        fro, mx = assert_fp_close(y2.float().cpu().numpy(), ref, f"{what} {od}")
        print(f"[err] {what} {od}: relFro {fro:.3e} max/rms {mx:.3e}", flush=True)


CASES = [
    # (act, group, scale_fp32, M, K, N)
    (W.ACT_INT8, 0, True, 1, 128, 300),       # one full and one partial 96-block
    (W.ACT_INT8, 0, True, 1, 4096, 1000),     # 43 blocks, the last with 64 weights
    (W.ACT_INT8, 0, True, 2, 1024, 17),       # two tokens, N below one workgroup
    (W.ACT_INT8, 0, True, 3, 11008, 520),     # 115 blocks: three LDS chunks; M > 2
    (W.ACT_INT8, None, False, 5, 2048, 777),  # per-channel FP16 scale
    (W.ACT_FP16, 0, True, 1, 4096, 1000),
    (W.ACT_FP16, 0, False, 2, 384, 300),      # per-tensor FP16 scale, K = 4 blocks exactly
    (W.ACT_FP16, None, False, 1, 11008, 640),
    (W.ACT_FP16, None, False, 7, 2048, 333),
]


@pytest.mark.parametrize("act,group,fp32,M,K,N", CASES)
def test_tri_parity(act, group, fp32, M, K, N):
    banner(f"3in5 act={act} group={group} fp32={fp32} M={M} K={K} N={N}")
    G = K if group is None else group
    inp = W.make_custom(W.WFMT_TERNARY, 2, G, act, M, K, N, seed=K + N + M, scale_fp32=fp32)
    check(GpuProblem(inp, wfmt=T35), f"3in5 M={M} K={K} N={N}")


def test_tri_headline_shape_full_size():
    banner("3in5 ternary INT8 1x4096x4096")
    inp = W.make_inputs(2, 0)
    check(GpuProblem(inp, wfmt=T35), "3in5 headline shape")


def test_tri_accumulate_zero_token_and_determinism():
    banner("3in5 accumulate / zero token / determinism")
    inp = W.make_custom(W.WFMT_TERNARY, 2, 0, W.ACT_INT8, 3, 1024, 300, seed=7, scale_fp32=True)
    inp.act[1, :] = 0  # an all-zero token: s_a = 0, output 0
    gp = GpuProblem(inp, wfmt=T35)
    acc_ref, _ = oracle.reference_output(inp)
    base = torch.from_numpy(np.arange(3 * 300, dtype=np.int32).reshape(3, 300)).cuda()
    out = base.clone()
    gp.lut(out_dtype=torch.int32, accumulate=True, out=out)
    assert np.array_equal(out.cpu().numpy().astype(np.int64), acc_ref + base.cpu().numpy()), "accumulate"
    out2 = base.clone()
    gp.fused(out_dtype=torch.int32, accumulate=True, out=out2)
    assert torch.equal(out, out2), "fused accumulate"
    y = gp.lut(out_dtype=torch.float32)
    assert torch.all(y[1] == 0), "zero token"
    for _ in range(3):
        assert torch.equal(gp.lut(out_dtype=torch.float32), y), "run-to-run determinism"

    inp = W.make_custom(W.WFMT_TERNARY, 2, 1024, W.ACT_FP16, 2, 1024, 260, seed=8)
    gp = GpuProblem(inp, wfmt=T35)
    ref = oracle.reference_output(inp)
    prev = torch.randn(2, 260, device="cuda", dtype=torch.float32)
    out = prev.clone()
    gp.lut(out_dtype=torch.float32, accumulate=True, out=out)
    assert_fp_close((out - prev).cpu().numpy(), ref, "3in5 FP accumulate")


def test_tri_dequant_not_supported():
    inp = W.make_custom(W.WFMT_TERNARY, 2, 0, W.ACT_FP16, 16, 1024, 64, seed=9)
    gp = GpuProblem(inp, wfmt=T35)
    with pytest.raises(L.LutGemmError):
        gp.dequant()
