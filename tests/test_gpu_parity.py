"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

* every workload family at reduced sizes that still span several column tiles,
  several K splits and a ragged column tail: all outputs compared;
* every workload shape at full size, in the launch configuration the benchmark
  times: sampled outputs (the INT8 family: all outputs, bit-exact);
* the precompute step against the table definition;
* one-hot activations (each output is one dequantized weight: checks packing and
  indexing element by element), zero activations, N tails, small K, several M,
  accumulate, INT32 / FP32 / FP16 outputs, run-to-run determinism;
* the dequantize + matrix-core comparison path.

FP16-activation results must satisfy relative Frobenius error <= 2e-3 and
max |error| / rms(reference) <= 1e-2; INT8-activation results are bit-exact.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from helpers import GpuProblem, assert_fp_close, fp_errors, sample_indices, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # collected on CPU hosts, skipped there
    pytest.skip("no GPU", allow_module_level=True)

import paper_2408_06003_amd as L  # noqa: E402  (fails loudly when the HIP library is missing)


def banner(msg):
    print(f"\n[case] {msg}", flush=True)


def check_int_path(gp, rows=None, cols=None):
    inp = gp.inp
    acc_ref, y_ref = oracle.reference_output(inp, rows=rows, cols=cols)
    yi = gp.lut(out_dtype=torch.int32).cpu().numpy()
    yf = gp.lut(out_dtype=torch.float32).cpu().numpy()
    if rows is not None:
        yi, yf = yi[np.ix_(rows, cols)], yf[np.ix_(rows, cols)]
    assert np.array_equal(yi.astype(np.int64), acc_ref), "INT32 accumulator differs from the oracle"
    assert np.array_equal(yf, y_ref), "FP32 scaled output differs from the oracle"


def check_fp_path(gp, rows=None, cols=None, dequant=False, out_dtype=None, what=""):
    inp = gp.inp
    ref = oracle.reference_output(inp, rows=rows, cols=cols)
    y = (gp.dequant(out_dtype=out_dtype) if dequant else gp.lut(out_dtype=out_dtype)).float().cpu().numpy()
    if rows is not None:
        y = y[np.ix_(rows, cols)]
    fro, mx = assert_fp_close(y, ref, what)
    print(f"[err] {what}: relFro {fro:.3e} max/rms {mx:.3e}", flush=True)
    return fro, mx


# ----------------------------------------------------------------- reduced sizes, all outputs

SMALL = [
    # (config family, M, K, N)
    (1, 1, 1024, 1000),
    (1, 2, 1024, 300),
    (2, 1, 4096, 1000),
    (2, 2, 2048, 777),
    (3, 1, 2048, 1000),
    (3, 1, 11008, 300),
    (4, 40, 1024, 520),
    (5, 1, 2048, 1000),
    (5, 16, 2048, 600),
    (5, 37, 1024, 300),
    (6, 45, 1024, 700),
]


@pytest.mark.parametrize("cid,M,K,N", SMALL)
def test_small_parity(cid, M, K, N):
    banner(f"small parity config={cid} M={M} K={K} N={N}")
    inp = W.make_inputs(cid, 0, M=M, K=K, N=N)
    gp = GpuProblem(inp)
    if inp.act_kind == W.ACT_INT8:
        check_int_path(gp)
    else:
        check_fp_path(gp, what=f"config {cid}")
        check_fp_path(gp, out_dtype=torch.float32, what=f"config {cid} fp32 out")


@pytest.mark.parametrize("cid,M,K,N", [(4, 40, 1024, 520), (5, 16, 2048, 600), (1, 3, 1024, 1000),
                                       (3, 130, 1024, 300)])
def test_small_dequant_parity(cid, M, K, N):
    banner(f"small dequant parity config={cid} M={M} K={K} N={N}")
    gp = GpuProblem(W.make_inputs(cid, 0, M=M, K=K, N=N))
    check_fp_path(gp, dequant=True, what=f"dequant config {cid}")


# ----------------------------------------------------------------- full sizes (bench launch configuration)

FULL = [(cid, sid, M, K, N) for cid, w in W.WORKLOADS.items() for (sid, M, K, N) in w.shapes()]


@pytest.mark.parametrize("cid,sid,M,K,N", FULL)
def test_full_size_sampled(cid, sid, M, K, N):
    banner(f"full size config={cid} shape={sid} M={M} K={K} N={N}")
    inp = W.make_inputs(cid, sid, M=M)
    gp = GpuProblem(inp)
    if inp.act_kind == W.ACT_INT8:
        check_int_path(gp)                            # all outputs, bit-exact
        return
    rows, cols = sample_indices(M, N, seed=cid * 100 + sid)
    check_fp_path(gp, rows=rows, cols=cols, what=f"config {cid}/{sid} LUT")
    if M >= 16:
        check_fp_path(gp, rows=rows, cols=cols, dequant=True, what=f"config {cid}/{sid} dequant")


# ----------------------------------------------------------------- precompute

@pytest.mark.parametrize("act_kind,M,K,G", [(W.ACT_FP16, 3, 1024, 128), (W.ACT_INT8, 3, 1024, 0),
                                             # several 1024-activation blocks per workgroup (large M),
                                             # group sums by lane butterflies and by whole workgroups
                                             (W.ACT_FP16, 300, 4096, 128), (W.ACT_FP16, 260, 8192, 2048),
                                             (W.ACT_INT8, 300, 4096, 0),
                                             # the longest tokens staged in LDS (K = 32768) and the
                                             # global-memory branch for longer ones
                                             (W.ACT_FP16, 3, 32768, 128), (W.ACT_INT8, 3, 32768, 0),
                                             (W.ACT_FP16, 3, 36864, 1024), (W.ACT_INT8, 3, 36864, 0),
                                             (W.ACT_FP16, 4, 65536, 128), (W.ACT_INT8, 4, 65536, 0)])
def test_precompute_matches_table_definition(act_kind, M, K, G):
    banner(f"precompute act={act_kind} M={M} K={K} G={G}")
    wfmt, bits = (W.WFMT_UINT, 2) if act_kind == W.ACT_FP16 else (W.WFMT_TERNARY, 2)
    inp = W.make_custom(wfmt, bits, G, act_kind, M=M, K=K, N=256, seed=21, scale_fp32=(G == 0))
    inp.act[1] *= np.float16(300)            # a large-magnitude token
    inp.act[2, :] = 0                        # an all-zero token
    inp.act[2, 5] = np.float16(-1e-3)
    p = L.problem(K, 256, bits, wfmt, G, act_kind, G == 0)
    t = torch.empty(L.table_size(p, M), dtype=torch.uint8, device="cuda")
    L.precompute(p, M, to_dev(inp.act), t)
    torch.cuda.synchronize()
    raw = t.cpu().numpy()
    s_off, t_off = L.table_offsets(p, M)
    J, Q = K // 4, (K // G if G else 1)
    tok = raw[t_off:t_off + 4 * M].view(np.float32)
    if act_kind == W.ACT_FP16:
        T = raw[:M * J * 16].view(np.float16).reshape(M, J, 8).astype(np.float64)
        mult = oracle.token_pow2(inp.act)
        assert np.array_equal(tok.astype(np.float64), mult)
        exact = oracle.half_tables(inp.act) / mult[:, None, None]
        ref16 = exact.astype(np.float16).astype(np.float64)
        ulp = np.spacing(np.abs(ref16).astype(np.float16)).astype(np.float64)
        assert np.all(np.abs(T - ref16) <= ulp), "table entry more than 1 FP16 ulp from the definition"
        S = raw[s_off:s_off + 4 * M * Q].view(np.float32).reshape(M, Q).astype(np.float64)
        S_ref = oracle.group_sums(inp.act, G) / mult[:, None]
        assert np.allclose(S, S_ref, rtol=1e-5, atol=1e-5)
    else:
        qa, sa = oracle.quantize_int8(inp.act)
        assert np.array_equal(tok, sa), "per-token absmax scale is not bit-exact"
        T = raw[:M * J * 16].view(np.int16).reshape(M, J, 8).astype(np.int64)
        assert np.array_equal(T, oracle.half_tables(qa))
        S = raw[s_off:s_off + 4 * M * Q].view(np.int32).reshape(M, Q).astype(np.int64)
        assert np.array_equal(S, oracle.group_sums(qa, 0))


# ----------------------------------------------------------------- element-exact checks and edges

@pytest.mark.parametrize("wfmt,bits,G", [(W.WFMT_UINT, 1, 128), (W.WFMT_UINT, 2, 256), (W.WFMT_UINT, 4, 128),
                                         (W.WFMT_BINARY, 1, 512), (W.WFMT_TERNARY, 2, 128)])
def test_one_hot_rows_extract_weights(wfmt, bits, G):
    """Activation rows e_k: output n is the dequantized weight r[n, k], for k across tables,
    plane words, quantization groups and K splits; checks packing and indexing exactly."""
    K, N = 1024, 300
    ks = [0, 1, 2, 3, 4, 127, 128, 300, 511, 640, 1023]
    banner(f"one-hot wfmt={wfmt} b={bits} G={G}")
    inp = W.make_custom(wfmt, bits, G, W.ACT_FP16, M=len(ks), K=K, N=N, seed=31)
    inp.act[:] = 0
    for i, k in enumerate(ks):
        inp.act[i, k] = 1.0
    gp = GpuProblem(inp)
    y = gp.lut(out_dtype=torch.float32).cpu().numpy().astype(np.float64)
    ref = oracle.reference_output(inp)
    assert np.allclose(y, ref, rtol=1e-6, atol=1e-7), np.abs(y - ref).max()


def test_zero_activations_and_small_k():
    banner("zero activations, K = G = 128, N = 1 / 7 / 257")
    for N in (1, 7, 257):
        inp = W.make_custom(W.WFMT_UINT, 2, 128, W.ACT_FP16, M=2, K=128, N=N, seed=41)
        gp = GpuProblem(inp)
        check_fp_path(gp, what=f"K=128 N={N}")
        inp0 = W.make_custom(W.WFMT_UINT, 2, 128, W.ACT_FP16, M=2, K=128, N=N, seed=41)
        inp0.act[:] = 0
        y0 = GpuProblem(inp0).lut(out_dtype=torch.float32).cpu().numpy()
        assert not np.any(y0), "zero activations must give zero output"


@pytest.mark.parametrize("M", [1, 2, 3, 5, 17])
def test_token_counts(M):
    banner(f"token count M={M}")
    inp = W.make_custom(W.WFMT_UINT, 4, 128, W.ACT_FP16, M=M, K=2048, N=513, seed=50 + M)
    check_fp_path(GpuProblem(inp), what=f"M={M}")
    inpi = W.make_custom(W.WFMT_TERNARY, 2, 0, W.ACT_INT8, M=M, K=2048, N=513, seed=60 + M, scale_fp32=True)
    check_int_path(GpuProblem(inpi))


def test_int8_binary_per_channel():
    banner("INT8 activations, binary per-channel weights")
    inp = W.make_custom(W.WFMT_BINARY, 1, 4096, W.ACT_INT8, M=3, K=4096, N=700, seed=71)
    check_int_path(GpuProblem(inp))


def test_accumulate_and_determinism():
    banner("accumulate flag and run-to-run determinism")
    inp = W.make_inputs(3, 0, K=4096, N=2000)
    gp = GpuProblem(inp)
    y1 = gp.lut(out_dtype=torch.float32)
    y2 = gp.lut(out_dtype=torch.float32)
    assert torch.equal(y1, y2), "two runs differ bitwise"
    base = torch.randn(1, 2000, device="cuda", dtype=torch.float32)
    acc = base.clone()
    gp.lut(out=acc, accumulate=True)
    assert torch.equal(acc, base + y1), "accumulate is not O + A W^T"
    inpi = W.make_inputs(2, 0, N=1500)
    gpi = GpuProblem(inpi)
    bi = torch.randint(-1000, 1000, (1, 1500), device="cuda", dtype=torch.int32)
    acci = bi.clone()
    gpi.lut(out=acci, accumulate=True)
    assert torch.equal(acci, bi + gpi.lut(out_dtype=torch.int32))


def test_extreme_scales():
    banner("extreme scales and activations")
    inp = W.make_custom(W.WFMT_UINT, 2, 128, W.ACT_FP16, M=2, K=1024, N=300, seed=81)
    inp.scales[:, 0] = np.float16(6e-5)
    inp.scales[:, 1] = np.float16(300.0)
    inp.act[1] = (inp.act[1].astype(np.float32) * 1000).astype(np.float16)
    ref = oracle.reference_output(inp)
    y = GpuProblem(inp).lut(out_dtype=torch.float32).cpu().numpy()
    assert_fp_close(y, ref, "extreme scales")


# ----------------------------------------------------------------- large-M comparison kernel

@pytest.mark.parametrize("cid,M,K,N", [(4, 300, 1024, 520), (3, 257, 2048, 300), (5, 280, 1024, 600),
                                       (6, 512, 1024, 256)])
def test_dequant_big_tile_parity(cid, M, K, N, tune):
    """The 256 x 256 pipelined dequantization + MFMA kernel (chosen for large M) on
    small shapes with ragged M and N tails, every output against the oracle."""
    tune(DEQUANT_KIND=1)
    banner(f"dequant 256x256 tile config={cid} M={M} K={K} N={N}")
    gp = GpuProblem(W.make_inputs(cid, 0, M=M, K=K, N=N))
    check_fp_path(gp, dequant=True, what=f"dequant big config {cid}")
    check_fp_path(gp, dequant=True, out_dtype=torch.float32, what=f"dequant big config {cid} fp32 out")


@pytest.mark.parametrize("kbs", [0, 1, 4])
def test_split_k_gemv_two_tokens(kbs, tune):
    """The table-fed split-K GEMV (forced) with two tokens and a ragged column tail, K
    split into 8-64 ranges summed by the finalize kernel: FP (all outputs within the FP
    bar) and INT8 (bit-exact) paths, and accumulation through the finalize epilogue."""
    tune(GEMV_KIND=2)
    if kbs:
        tune(KBS=kbs)
    banner(f"split-K GEMV M=2 kbs={kbs or 'planned'}")
    inp = W.make_custom(W.WFMT_UINT, 2, 128, W.ACT_FP16, M=2, K=8192, N=777, seed=800 + kbs)
    gp = GpuProblem(inp)
    y = check_fp_path(gp, out_dtype=torch.float32, what=f"split-K M=2 kbs={kbs}")
    y32 = gp.lut(out_dtype=torch.float32)
    base = torch.randn(2, 777, device="cuda", dtype=torch.float32)
    acc = base.clone()
    gp.lut(out=acc, accumulate=True)
    assert torch.equal(acc, base + y32), "accumulate through the finalize kernel"
    inpi = W.make_custom(W.WFMT_TERNARY, 2, 0, W.ACT_INT8, M=2, K=8192, N=777, seed=900 + kbs, scale_fp32=True)
    check_int_path(GpuProblem(inpi))


# ----------------------------------------------------------------- long tokens (K > 32768)

@pytest.mark.parametrize("wfmt,bits,G,act,K,N,M", [
    (W.WFMT_UINT, 4, 128, W.ACT_FP16, 36864, 300, 1),
    (W.WFMT_UINT, 2, 1024, W.ACT_FP16, 65536, 260, 2),
    (W.WFMT_TERNARY, 2, 0, W.ACT_INT8, 36864, 300, 1),
    (W.WFMT_BINARY, 1, 65536, W.ACT_INT8, 65536, 200, 1),
    (W.WFMT_UINT, 2, 128, W.ACT_FP16, 36864, 300, 5),      # multi-token kernel
    (W.WFMT_TERNARY, 2, 0, W.ACT_INT8, 65536, 130, 9),
])
def test_long_k_parity(wfmt, bits, G, act, K, N, M, tune):
    """Tokens longer than the 32768 activations the precompute stages in LDS (its
    global-memory branch), through the two-call path, the fused entry point and the
    split-K GEMV (long K splits: finalize kernel), against the oracle, all outputs."""
    banner(f"long K wfmt={wfmt} b={bits} G={G} act={act} K={K} N={N} M={M}")
    inp = W.make_custom(wfmt, bits, G, act, M=M, K=K, N=N, seed=71, scale_fp32=(G == 0))
    gp = GpuProblem(inp)
    paths = [("two-call", gp.lut), ("fused", gp.fused)]
    for name, run in paths:
        if act == W.ACT_INT8:
            acc_ref, y_ref = oracle.reference_output(inp)
            assert np.array_equal(run(out_dtype=torch.int32).cpu().numpy().astype(np.int64), acc_ref), name
            assert np.array_equal(run(out_dtype=torch.float32).cpu().numpy(), y_ref), name
        else:
            ref = oracle.reference_output(inp)
            fro, mx = assert_fp_close(run(out_dtype=torch.float32).cpu().numpy(), ref, f"long K {name}")
            print(f"[err] long K {name}: relFro {fro:.3e} max/rms {mx:.3e}", flush=True)
    if M <= 2:  # the split-K GEMV on the same problem
        tune(GEMV_KIND=2)
        gs = GpuProblem(inp)
        if act == W.ACT_INT8:
            acc_ref, _ = oracle.reference_output(inp)
            assert np.array_equal(gs.lut(out_dtype=torch.int32).cpu().numpy().astype(np.int64), acc_ref)
        else:
            assert_fp_close(gs.lut(out_dtype=torch.float32).cpu().numpy(), oracle.reference_output(inp),
                            "long K split-K")
            assert_fp_close(gs.fused(out_dtype=torch.float32).cpu().numpy(), oracle.reference_output(inp),
                            "long K fused split-K")
