"""GPU parity of the exact K-split completion of the single-token split-K GEMV.

Every K split turns its partial sum into an integer -- the INT32 sum of the INT8
path (Section 3.1.3 quantization, Eq. 3 epilogue); on the FP16 path with one scale
per column or per tensor the sum of the split's fixed-point table entries; otherwise
the FP32 partial sum in fixed point with a per-column exponent that the packer
derives from a bound on the column's partial sums -- and adds it with an arrival
count to one 64-bit word per output with a single atomic; the split that completes
the count applies the output epilogue.  The sum is exact, so the result does not
depend on the order in which splits arrive.

Checked here, all outputs against the CPU oracle: 1-bit weights with a scale per
column, 2- and 4-bit weights with a scale and zero point per column (the zero-point
term applied once, by the completing split) and per group of 128 (fixed point; up to
64 splits, beyond the arrival protocol's 32), ternary weights with one FP32 scale,
scales spread over 2^22 within a column, INT8 activations (bit for bit, and bit for
bit equal to the split-order protocol), the fused entry point (tables built from the
unscaled activations), one and two tokens, ragged column tails, accumulation into the
output, run-to-run determinism, and a layer too wide for the split-sum words (falls
back to the arrival protocol), and the planner's limits: 127 splits and exactly the
split-sum words of the zero region take the exact completion, one split or one column
tile more fall back, all equal to the oracle.  That the words are left zero for the next call, also
of another problem on the same workspace, is checked in test_gpu_workspace.py.
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


def banner(msg):
    print(f"\n[case] {msg}", flush=True)


CASES = [
    # (wfmt, bits, group (K: per column, 0: per tensor), act, FP32 scale, M, K, N, KBS forced)
    (W.WFMT_BINARY, 1, "K", W.ACT_FP16, False, 1, 8192, 777, 0),
    (W.WFMT_BINARY, 1, "K", W.ACT_FP16, False, 2, 8192, 300, 2),
    (W.WFMT_UINT, 2, "K", W.ACT_FP16, False, 1, 4096, 520, 2),
    (W.WFMT_UINT, 4, "K", W.ACT_FP16, False, 2, 6144, 260, 2),
    (W.WFMT_TERNARY, 2, 0, W.ACT_FP16, True, 2, 4096, 700, 4),
    (W.WFMT_TERNARY, 2, 0, W.ACT_INT8, True, 1, 8192, 777, 0),
    (W.WFMT_BINARY, 1, "K", W.ACT_INT8, False, 2, 8192, 300, 2),
    (W.WFMT_BINARY, 1, 0, W.ACT_INT8, True, 1, 4096, 1000, 8),
    (W.WFMT_UINT, 4, 128, W.ACT_FP16, False, 1, 11008, 300, 0),
    (W.WFMT_UINT, 2, 128, W.ACT_FP16, False, 2, 8192, 520, 1),
    (W.WFMT_UINT, 2, 1024, W.ACT_FP16, False, 1, 4096, 777, 2),
    (W.WFMT_TERNARY, 2, 128, W.ACT_FP16, False, 1, 4096, 260, 0),
]


@pytest.mark.parametrize("wfmt,bits,G,act,sf,M,K,N,kbs", CASES)
def test_exact_split_parity(wfmt, bits, G, act, sf, M, K, N, kbs, tune):
    tune(GEMV_KIND=2, SPLIT_EXACT=1)
    if kbs:
        tune(KBS=kbs)
    group = K if G == "K" else G
    banner(f"exact split wfmt={wfmt} b={bits} G={group} act={act} M={M} K={K} N={N} kbs={kbs or 'planned'}")
    inp = W.make_custom(wfmt, bits, group, act, M=M, K=K, N=N, seed=1200 + 17 * wfmt + bits + kbs, scale_fp32=sf)
    gp = GpuProblem(inp)
    base = torch.randn(M, N, device="cuda", dtype=torch.float32)
    if act == W.ACT_INT8:
        acc_ref, y_ref = oracle.reference_output(inp)
        yi = gp.lut(out_dtype=torch.int32)
        yf = gp.lut(out_dtype=torch.float32)
        assert np.array_equal(yi.cpu().numpy().astype(np.int64), acc_ref), "INT32 accumulator differs from the oracle"
        assert np.array_equal(yf.cpu().numpy(), y_ref), "FP32 output differs from the oracle"
        assert torch.equal(gp.lut(out_dtype=torch.int32), yi), "not deterministic"
        # the same integer sums as the split-order protocol
        L.set_tuning("SPLIT_EXACT", 0)
        assert torch.equal(gp.lut(out_dtype=torch.int32), yi), "differs from the arrival protocol"
        assert torch.equal(gp.lut(out_dtype=torch.float32), yf), "differs from the arrival protocol"
        L.set_tuning("SPLIT_EXACT", 1)
    else:
        ref = oracle.reference_output(inp)
        for od in (torch.float16, torch.float32):
            y = gp.lut(out_dtype=od)
            fro, mx = assert_fp_close(y.float().cpu().numpy(), ref, f"exact split {od}")
            print(f"[err] {od}: relFro {fro:.3e} max/rms {mx:.3e}", flush=True)
            assert torch.equal(gp.lut(out_dtype=od), y), "not deterministic"
        yf = gp.lut(out_dtype=torch.float32)
    acc = base.clone()
    gp.lut(out=acc, accumulate=True, out_dtype=torch.float32)
    assert torch.equal(acc, base + yf), "accumulation through the exact completion"


def test_exact_split_wide_layer_falls_back(tune):
    """Two tokens of 65 536 columns need more split-sum words than the workspace's zero
    region holds: the arrival protocol completes the split instead, same bar."""
    tune(GEMV_KIND=2, KBS=2)
    inp = W.make_custom(W.WFMT_BINARY, 1, 2048, W.ACT_FP16, M=2, K=2048, N=65536, seed=1301)
    banner("exact split: 2 x 2048 x 65536, beyond the split-sum words")
    gp = GpuProblem(inp)
    ref = oracle.reference_output(inp)
    fro, mx = assert_fp_close(gp.lut(out_dtype=torch.float32).cpu().numpy(), ref, "wide layer")
    print(f"[err] relFro {fro:.3e} max/rms {mx:.3e}", flush=True)



@pytest.mark.parametrize("wfmt,bits,G,act,sf,M,K,N,kbs", [c for c in CASES if c[3] == W.ACT_FP16])
def test_exact_split_fused_entry(wfmt, bits, G, act, sf, M, K, N, kbs, tune):
    """The fused entry point's split-K kernel (tables built from the activations of its
    K range, unscaled FP32 entries) with the fixed-point exact completion."""
    tune(GEMV_KIND=2, SPLIT_EXACT=1)
    if kbs:
        tune(KBS=kbs)
    group = K if G == "K" else G
    banner(f"exact split, fused entry: wfmt={wfmt} b={bits} G={group} M={M} K={K} N={N} kbs={kbs or 'planned'}")
    inp = W.make_custom(wfmt, bits, group, act, M=M, K=K, N=N, seed=1400 + 17 * wfmt + bits + kbs, scale_fp32=sf)
    gp = GpuProblem(inp)
    ref = oracle.reference_output(inp)
    for od in (torch.float16, torch.float32):
        y = gp.fused(out_dtype=od)
        fro, mx = assert_fp_close(y.float().cpu().numpy(), ref, f"fused exact split {od}")
        print(f"[err] {od}: relFro {fro:.3e} max/rms {mx:.3e}", flush=True)
        assert torch.equal(gp.fused(out_dtype=od), y), "not deterministic"


def test_exact_split_extreme_scales(tune):
    """Scales 6e-5 and 300 in the same columns (2^22 apart) and a token scaled by 1000:
    the fixed-point unit follows the largest scale of each column, the small groups
    keep their precision within the FP bar."""
    tune(GEMV_KIND=2, KBS=1, SPLIT_EXACT=1)
    inp = W.make_custom(W.WFMT_UINT, 2, 128, W.ACT_FP16, M=2, K=4096, N=300, seed=1381)
    inp.scales[:, 0::2] = np.float16(6e-5)
    inp.scales[:, 1] = np.float16(300.0)
    inp.act[1] = (inp.act[1].astype(np.float32) * 1000).astype(np.float16)
    banner("exact split: extreme scales")
    gp = GpuProblem(inp)
    ref = oracle.reference_output(inp)
    for run in (gp.lut, gp.fused):
        fro, mx = assert_fp_close(run(out_dtype=torch.float32).cpu().numpy(), ref, "extreme scales")
        print(f"[err] relFro {fro:.3e} max/rms {mx:.3e}", flush=True)


@pytest.mark.parametrize("sid", [0, 1])
def test_exact_split_two_tokens_full_size(sid):
    """Two tokens of the 1-bit 70B layers at full size (planned: both tokens in each
    workgroup of the split-K kernel), sampled outputs against the oracle, and the same
    outputs as one token at a time."""
    inp = W.make_inputs(5, sid, M=2)
    banner(f"exact split, two tokens per workgroup: 2 x {inp.K} x {inp.N}")
    gp = GpuProblem(inp)
    y = gp.lut(out_dtype=torch.float32)
    cols = np.unique(np.linspace(0, inp.N - 1, 512).astype(np.int64))
    rows = np.arange(2)
    ref = oracle.reference_output(inp, rows=rows, cols=cols)
    fro, mx = assert_fp_close(y.cpu().numpy()[np.ix_(rows, cols)], ref, "two tokens")
    print(f"[err] relFro {fro:.3e} max/rms {mx:.3e}", flush=True)
    for m in range(2):  # token m alone: same integer sums, same output bits
        one = W.make_inputs(5, sid, M=2)
        one.act = one.act[m:m + 1].copy()
        one.M = 1
        assert torch.equal(GpuProblem(one).lut(out_dtype=torch.float32)[0], y[m]), f"token {m} differs alone"


def _align256(x):
    return (x + 255) // 256 * 256


@pytest.mark.parametrize("wfmt,bits,group,sf", [(W.WFMT_UINT, 4, 128, False), (W.WFMT_UINT, 2, 1024, False),
                                                (W.WFMT_BINARY, 1, "K", False), (W.WFMT_TERNARY, 2, 0, True)])
def test_exact_split_column_exponents(wfmt, bits, group, sf):
    """The per-column fixed-point exponent the packer stores after the metadata (R27):
    E = floor(log2 B) + 1 - 54 with B = 1.0625 sum_q (kpg |s'_q| 128 (2^b - 1) +
    |s'_q z'_q| G), recomputed here in float64 from the problem's scales and zeros
    (s' = s, z' = 0 for 1-bit weights; s' = s/2, z' = -1 for ternary; s' = s/2,
    z' = 2 z + 1 - 2^b otherwise), with scales spread over 2^20 across columns."""
    K, N = 2048, 300
    G = K if group == "K" else group
    inp = W.make_custom(wfmt, bits, G, W.ACT_FP16, M=1, K=K, N=N, seed=1391, scale_fp32=sf)
    if not sf:  # columns whose scales differ by up to 2^20
        inp.scales = (inp.scales.astype(np.float64) * (2.0 ** (np.arange(N) % 21 - 10))[:, None]).astype(np.float16)
    gp = GpuProblem(inp)
    raw = gp.g.packed.cpu().numpy()
    n_pad = -(-N // 256) * 256
    kb = K // 128
    Q = 1 if G in (0, K) else K // G
    meta_off = _align256(kb * bits * n_pad * 16)
    meta_bytes = 256 if G == 0 else Q * n_pad * 4
    bnd = raw[meta_off + _align256(meta_bytes):][:n_pad * 4].view(np.int32)
    Gq = K if G == 0 else G
    kpg = Gq // 128
    if G == 0:  # one scale for the tensor
        s = np.full((N, 1), float(inp.scales.reshape(-1)[0]))
    else:
        s = inp.scales.astype(np.float64).reshape(N, -1)
    if wfmt == W.WFMT_BINARY:
        sp, zp = s, np.zeros_like(s)
    elif wfmt == W.WFMT_TERNARY:
        sp, zp = s * 0.5, -np.ones_like(s)
    else:
        sp, zp = s * 0.5, 2.0 * inp.zeros.astype(np.float64).reshape(N, -1) + (1.0 - 2 ** bits)
    terms = kpg * np.abs(sp) * 128.0 * (2 ** bits - 1) + np.abs(sp * zp) * Gq
    B = np.cumsum(terms, axis=1)[:, -1] * 1.0625  # in group order, as the packer sums
    want = np.frexp(B)[1].astype(np.int64) - 54  # ilogb(B) + 1 - 54
    assert np.array_equal(bnd[:N].astype(np.int64), want), "column exponents differ from the bound"
    assert not bnd[N:].any(), "padding columns keep exponent 0"


@pytest.mark.parametrize("cid,sid", [(3, 0), (5, 0)])
def test_split_prefetch_depth_same_bits(cid, sid, tune):
    """How many weight words a lane requests before its tables arrive (SPLIT_PRE: none,
    2, 4, all, or half by default) changes only when loads are issued: the outputs of
    the full decode layer are equal bit for bit, table-fed and fused."""
    inp = W.make_inputs(cid, sid, M=1)
    banner(f"split-K prefetch depth 1 x {inp.K} x {inp.N}")
    gp = GpuProblem(inp)
    ref = (gp.lut(out_dtype=torch.float32), gp.fused(out_dtype=torch.float32))
    for pre in (0, 2, 4, 8):
        tune(SPLIT_PRE=pre)
        assert torch.equal(gp.lut(out_dtype=torch.float32), ref[0]), f"SPLIT_PRE={pre}: table-fed output differs"
        assert torch.equal(gp.fused(out_dtype=torch.float32), ref[1]), f"SPLIT_PRE={pre}: fused output differs"


LIMITS = [
    # (what, M, K, N, exact completion expected)
    ("127 splits, the most one word counts", 1, 127 * 128, 300, True),
    ("128 splits: the finalize kernel", 1, 128 * 128, 300, False),
    ("two tokens, 127 splits", 2, 127 * 128, 260, True),
    ("122880 words, exactly the zero region", 1, 512, 122880, True),
    ("one column tile more: the arrival protocol", 1, 512, 122881, False),
]


@pytest.mark.parametrize("what,M,K,N,exact", LIMITS)
def test_exact_split_limits(what, M, K, N, exact, tune):
    """At the planner's limits of the exact completion (splits and split-sum words) and
    one step beyond, INT8 ternary layers (one K block per split) equal the oracle bit
    for bit.  Which completion ran is read from the workspace the plan asks for: the
    exact one needs only the zero region, the others add FP32 partial sums."""
    tune(GEMV_KIND=2, KBS=1, SPLIT_EXACT=1)
    banner(f"exact split limits: {what}: M={M} K={K} N={N}")
    inp = W.make_custom(W.WFMT_TERNARY, 2, 0, W.ACT_INT8, M=M, K=K, N=N, seed=1401 + K + N, scale_fp32=True)
    gp = GpuProblem(inp)
    ws = L.workspace_size(gp.p, M)
    assert (ws == L.WORKSPACE_ZERO_BYTES) == exact, f"workspace {ws} B: exact completion {'not ' if exact else ''}planned"
    acc_ref, y_ref = oracle.reference_output(inp)
    yi = gp.lut(out_dtype=torch.int32)
    assert np.array_equal(yi.cpu().numpy().astype(np.int64), acc_ref), "INT32 accumulator differs from the oracle"
    assert np.array_equal(gp.lut(out_dtype=torch.float32).cpu().numpy(), y_ref), "FP32 output differs from the oracle"


def test_exact_split_limit_fp16_fixed_point(tune):
    """127 splits of 1-bit weights with one scale per column on FP16 activations: the
    fixed-point form of the completion at its largest arrival count."""
    tune(GEMV_KIND=2, KBS=1, SPLIT_EXACT=1)
    banner("exact split limits: FP16 binary 1 x 16256 x 300, 127 splits")
    inp = W.make_custom(W.WFMT_BINARY, 1, 127 * 128, W.ACT_FP16, M=1, K=127 * 128, N=300, seed=1409)
    gp = GpuProblem(inp)
    assert L.workspace_size(gp.p, 1) == L.WORKSPACE_ZERO_BYTES
    ref = oracle.reference_output(inp)
    fro, mx = assert_fp_close(gp.lut(out_dtype=torch.float32).cpu().numpy(), ref, "127 splits")
    print(f"[err] relFro {fro:.3e} max/rms {mx:.3e}", flush=True)
