"""GPU parity of lutgemm_mpgemm_fused for several tokens (M > 2) with FP16
activations: the multi-token kernel reads the activations of its tokens and K range,
scales each token by a power of two from its absmax over that range, and builds its
LDS tables itself (the precompute fused into the consumer, Section 3.1.1).

Every output is compared with the CPU oracle at the FP bar.  Where every K range of
a token has the same absmax exponent as the whole token (one planted activation of
magnitude 3.5 per 128-block), the fused call uses the two-call path's scale, and its
output on weights without zero points is compared bit for bit with precompute +
mpGEMM.  Cases: 8- and 16-token tiles, ragged token and column tails, planned and
forced K splits, K ranges capped for the zero-point sums (K = 11008), every weight
format with zero points per 128-block, per group of 1024, per channel and per tensor,
a zero token, a token scaled by 300, accumulation and determinism.
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


@pytest.fixture(autouse=True)
def forced_fused(tune):
    """The in-kernel table build for every case here, whatever the planner would pick
    (it takes it for M <= 64 on layers of at most 64 column tiles)."""
    tune(MT_FUSED=1)


def banner(msg):
    print(f"\n[case] {msg}", flush=True)


def check(gp, what, rows=None, cols=None):
    ref = oracle.reference_output(gp.inp, rows=rows, cols=cols)
    for od in (torch.float16, torch.float32):
        y = gp.fused(out_dtype=od).float().cpu().numpy()
        if rows is not None:
            y = y[np.ix_(rows, cols)]
        fro, mx = assert_fp_close(y, ref, f"{what} {od}")
        print(f"[err] {what} {od}: relFro {fro:.3e} max/rms {mx:.3e}", flush=True)


def plant_block_maxima(inp, value=3.5):
    """One activation of magnitude `value` in every 128-block of every token, so that
    every K range has the absmax exponent of the whole token."""
    a = inp.act.astype(np.float32)
    np.clip(a, -3.0, 3.0, out=a)
    a[:, ::128] = value
    inp.act = a.astype(np.float16)
    return inp


@pytest.mark.parametrize("cid,M,K,N", [
    (5, 3, 1024, 300),     # one 8-token tile, ragged tokens and columns
    (5, 16, 2048, 600),    # one 16-token tile
    (5, 40, 4736, 1000),   # three 16-token tiles, ragged
    (5, 17, 8192, 520),    # planned K split
    (1, 5, 2048, 700),     # INT2 g128, zero point per block
    (1, 70, 4096, 300),    # INT2, 16-token tiles
    (3, 8, 2048, 600),     # INT4 g128
    (3, 33, 11008, 300),   # INT4, K range capped at 64 blocks for the block sums
])
def test_fused_mtok_parity(cid, M, K, N):
    banner(f"fused multi-token config={cid} M={M} K={K} N={N}")
    gp = GpuProblem(W.make_inputs(cid, 0, M=M, K=K, N=N))
    print(f"[ws] fused workspace {L.fused_workspace_size(gp.p, M)} B", flush=True)
    check(gp, f"config {cid} M={M} K={K} N={N}")


@pytest.mark.parametrize("wfmt,bits,G,sf", [(W.WFMT_UINT, 1, 128, False), (W.WFMT_UINT, 2, 1024, False),
                                            (W.WFMT_UINT, 4, 0, False), (W.WFMT_TERNARY, 2, 128, False),
                                            (W.WFMT_TERNARY, 2, 0, True), (W.WFMT_BINARY, 1, 0, True)])
@pytest.mark.parametrize("M", [6, 20])
def test_fused_mtok_formats(wfmt, bits, G, sf, M):
    banner(f"fused multi-token formats wfmt={wfmt} b={bits} G={G} per-tensor={sf} M={M}")
    inp = W.make_custom(wfmt, bits, G, W.ACT_FP16, M=M, K=3072, N=520, seed=301 + bits + 7 * wfmt, scale_fp32=sf)
    check(GpuProblem(inp), f"wfmt={wfmt} b={bits} G={G} M={M}")


@pytest.mark.parametrize("cid,splits", [(5, 3), (5, 7), (1, 2), (1, 5)])
def test_fused_mtok_forced_splits(cid, splits, tune):
    tune(MT_SPLITS=splits)
    banner(f"fused multi-token forced splits={splits} config={cid} M=24 K=4096 N=600")
    gp = GpuProblem(W.make_inputs(cid, 0, M=24, K=4096, N=600))
    check(gp, f"splits={splits} config {cid}")


@pytest.mark.parametrize("M,K,N,splits", [(16, 4096, 700, 0), (9, 2048, 300, 3), (40, 8192, 520, 0)])
def test_fused_mtok_bitwise_two_call(M, K, N, splits, tune):
    """Binary weights (no zero point) with every K range at the token's absmax exponent:
    the fused call equals precompute + mpGEMM bit for bit."""
    if splits:
        tune(MT_SPLITS=splits)
    banner(f"fused multi-token bitwise vs two-call M={M} K={K} N={N} splits={splits or 'planned'}")
    gp = GpuProblem(plant_block_maxima(W.make_inputs(5, 0, M=M, K=K, N=N)))
    for od in (torch.float16, torch.float32):
        a = gp.fused(out_dtype=od)
        b = gp.lut(out_dtype=od)
        assert torch.equal(a, b), f"fused != two-call ({od}): max diff {(a.float() - b.float()).abs().max().item()}"
    check(gp, "bitwise case")


def test_fused_mtok_tokens_zero_large_accumulate():
    banner("fused multi-token: zero token, token x 300, accumulate, determinism, tuning off")
    inp = W.make_inputs(1, 0, M=12, K=4096, N=700)
    a = inp.act.astype(np.float32)
    a[3] = 0.0
    a[7] *= 300.0
    inp.act = a.astype(np.float16)
    gp = GpuProblem(inp)
    check(gp, "zero and large tokens")
    y1 = gp.fused(out_dtype=torch.float32)
    assert torch.equal(y1, gp.fused(out_dtype=torch.float32)), "fused multi-token not deterministic"
    assert not y1[3].any(), "zero token gives nonzero output"
    base = torch.randn(12, 700, device="cuda")
    acc = base.clone()
    gp.fused(out=acc, accumulate=True, out_dtype=torch.float32)
    assert torch.equal(acc, base + y1)
    # the two-call path behind the same entry point (tuning key) stays within the bar
    L.set_tuning("MT_FUSED", 0)
    check(gp, "MT_FUSED=0")


@pytest.mark.parametrize("sid", [0, 1])
def test_fused_mtok_full_size(sid):
    """The 16-token layers of the 70B workload at full size, sampled outputs."""
    inp = W.make_inputs(5, sid, M=16)
    banner(f"fused multi-token full size M=16 K={inp.K} N={inp.N}")
    gp = GpuProblem(inp)
    rows, cols = sample_indices(16, inp.N, seed=500 + sid)
    check(gp, f"70B shape {sid}", rows=rows, cols=cols)
