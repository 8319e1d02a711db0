"""GPU parity of INT8 table quantization (Section 3.1.3; LUTGEMM_ACT_FP16_LUT8).

The approximation has its own reference, the table-quantized oracle
(``oracle.mpgemm_lut8``, pinned in test_oracle_pins.py):
* the precompute's INT8 codes and FP32 scales equal the oracle's bit for bit (both
  quantize the same FP32 half tables with the same FP32 operations);
* single-token kernels (whole-K and split-K GEMV): FP32 outputs within relFro 1e-5 of
  the table-quantized oracle (the tables are staged as FP32 products rounded to
  2^-20, summed exactly in INT32), FP16 outputs within the FP tolerance;
* multi-token kernel (entries staged as FP16, partial FP16 sums): the FP tolerance;
* against the exact product the error is the approximation's own, about 3e-3
  relative: checked to stay below 1e-2 (relFro) as a sanity bound.
The fused entry point runs the two calls for this mode and must agree bitwise.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from helpers import GpuProblem, assert_fp_close, fp_errors, sample_indices

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2408_06003_amd as L  # noqa: E402


def banner(msg):
    print(f"\n[case] {msg}", flush=True)


def lut8(inp):
    inp.act_kind = W.ACT_FP16_LUT8
    return inp


def check(gp, what, rows=None, cols=None, tight=True):
    inp = gp.inp
    ref8 = oracle.reference_output(inp, rows=rows, cols=cols)
    exact = oracle.mpgemm_fp(inp.act, inp.codes, inp.wfmt, inp.group, inp.scales, inp.zeros, rows=rows, cols=cols)
    y32 = gp.lut(out_dtype=torch.float32)
    y16 = gp.lut(out_dtype=torch.float16)
    assert torch.equal(gp.fused(out_dtype=torch.float32), y32), f"{what}: fused entry differs from the two calls"
    a32, a16 = y32.cpu().numpy().astype(np.float64), y16.float().cpu().numpy().astype(np.float64)
    if rows is not None:
        a32, a16 = a32[np.ix_(rows, cols)], a16[np.ix_(rows, cols)]
    fro, mx = fp_errors(a32, ref8)
    print(f"[err] {what} fp32 vs table-quantized oracle: relFro {fro:.3e} max/rms {mx:.3e}", flush=True)
    if tight:
        assert fro <= 1e-5 and mx <= 1e-4, f"{what}: FP32 output off the table-quantized oracle"
    else:
        assert_fp_close(a32, ref8, f"{what} fp32")
    assert_fp_close(a16, ref8, f"{what} fp16")
    fe, me = fp_errors(a32, exact)
    print(f"[err] {what} vs exact: relFro {fe:.3e} max/rms {me:.3e}", flush=True)
    assert fe <= 1e-2, f"{what}: approximation error {fe:.3e} above the sanity bound"


@pytest.mark.parametrize("wfmt,bits,group", [(W.WFMT_UINT, 2, 128), (W.WFMT_UINT, 4, 256),
                                             (W.WFMT_BINARY, 1, 2048), (W.WFMT_TERNARY, 2, 0)])
def test_lut8_precompute_matches_oracle_tables(wfmt, bits, group):
    banner(f"lut8 precompute wfmt={wfmt} b={bits} G={group}")
    M, K = 3, 2048
    inp = lut8(W.make_custom(wfmt, bits, group, W.ACT_FP16, M, K, 64, seed=11))
    # token 2: magnitudes from FP16 subnormals to 6e4 in one group (an FP32 sum of the
    # four terms would round) and groups whose 127 T / amax are half-integers (ties)
    rng = np.random.default_rng(44)
    mags = 2.0 ** rng.integers(-24, 15, size=K)
    inp.act[2] = np.clip(rng.standard_normal(K) * mags, -6e4, 6e4).astype(np.float16)
    inp.act[2, :8] = [-31.25, 31.25, 31.25, 33.25, 31.25, -31.25, -31.25, -33.25]
    gp = GpuProblem(inp)
    gp.lut()
    buf = gp.g.tables(M).cpu().numpy()
    J = K // 4
    sc_off = -(-(8 * M * J) // 256) * 256
    s_off, t_off = L.table_offsets(gp.p, M)
    q = buf[:8 * M * J].view(np.int8).reshape(M, J, 8)
    sc = buf[sc_off:sc_off + 4 * M * J].view(np.float32).reshape(M, J)
    tok = buf[t_off:t_off + 4 * M].view(np.float32)
    q_ref, sc_ref, mult = oracle.lut8_tables(inp.act)
    assert np.array_equal(q, q_ref), "INT8 table codes differ from the oracle"
    assert np.array_equal(sc, sc_ref), "table scales differ from the oracle"
    assert np.array_equal(tok.astype(np.float64), mult), "per-token factor differs"
    G = group or K
    S = buf[s_off:s_off + 4 * M * (K // G)].view(np.float32).reshape(M, K // G)
    S_ref = oracle.group_sums(inp.act.astype(np.float64) / mult[:, None], G)
    assert np.allclose(S, S_ref, rtol=1e-5, atol=1e-4)


CASES = [
    # (family, M, K, N): whole-K GEMV, split-K GEMV (large weights), multi-token
    (1, 1, 1024, 1000),
    (3, 1, 4096, 1000),
    (3, 2, 2048, 777),
    (5, 1, 2048, 1000),
    (2, 1, 4096, 300),  # ternary, per-tensor FP32 scale (FP16 activations here)
]


@pytest.mark.parametrize("cid,M,K,N", CASES)
def test_lut8_single_token_parity(cid, M, K, N):
    banner(f"lut8 config={cid} M={M} K={K} N={N}")
    inp = lut8(W.make_inputs(cid, 0, M=M, K=K, N=N))
    check(GpuProblem(inp), f"lut8 config {cid} M={M}")


@pytest.mark.parametrize("cid,M,K,N", [(4, 40, 1024, 520), (5, 16, 2048, 600), (5, 37, 1024, 300),
                                       (3, 9, 4096, 300)])
def test_lut8_multi_token_parity(cid, M, K, N):
    banner(f"lut8 multi-token config={cid} M={M} K={K} N={N}")
    inp = lut8(W.make_inputs(cid, 0, M=M, K=K, N=N))
    check(GpuProblem(inp), f"lut8 config {cid} M={M}", tight=False)


@pytest.mark.parametrize("cid,sid", [(3, 0), (3, 2), (5, 0)])
def test_lut8_full_size_sampled(cid, sid):
    w = W.WORKLOADS[cid]
    M = w.ms[0]
    K, N = w.kn[sid]
    banner(f"lut8 full size config={cid} shape={sid} M={M} K={K} N={N}")
    inp = lut8(W.make_inputs(cid, sid, M=M))
    rows, cols = sample_indices(M, N, seed=700 + cid * 10 + sid)
    check(GpuProblem(inp), f"lut8 full {cid}/{sid}", rows=rows, cols=cols, tight=(M <= 2))


@pytest.mark.parametrize("cid,M,K,N,kbs", [(3, 1, 4096, 1000, 1), (3, 2, 2048, 777, 2), (5, 2, 4096, 600, 4),
                                           (1, 1, 8192, 300, 1)])
def test_lut8_split_k_exact(cid, M, K, N, kbs, tune):
    """The split-K GEMV (forced) on INT8-quantized tables: staged as fixed-point entries
    like FP16 tables, so the K split is completed exactly (one atomic per output; two
    tokens per workgroup for 1-bit weights) -- within the tight bar of the single-token
    kernels."""
    tune(GEMV_KIND=2, KBS=kbs)
    banner(f"lut8 split-K exact config={cid} M={M} K={K} N={N} kbs={kbs}")
    inp = lut8(W.make_inputs(cid, 0, M=M, K=K, N=N))
    check(GpuProblem(inp), f"lut8 split-K config {cid} M={M}")
