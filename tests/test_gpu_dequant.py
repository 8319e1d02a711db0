"""GPU parity of the dequantize + matrix-core comparison path (Section 2.2) in each of
its launch forms, every output against the oracle:

* the 16-token-slab kernel of 1-bit weights (per-column and per-tensor scales): token
  tails, K ranges that end inside the activation chunk and inside the register ring
  of weight words, planned and forced K splits;
* the 256 x 256 and 128 x 128 tile kernels with and without a K split (FP32 partial
  sums added in split order by the reduce kernel);
* accumulation into an existing output, FP32 and FP16 outputs, run-to-run
  determinism.

Tolerance: the FP bar of the LUT path (relative Frobenius <= 2e-3, max |error| /
rms(reference) <= 1e-2).
"""
import numpy as np
import pytest

import oracle
import workloads as W
from helpers import GpuProblem, assert_fp_close

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # collected on CPU hosts, skipped there
    pytest.skip("no GPU", allow_module_level=True)

import paper_2408_06003_amd as L  # noqa: E402  (fails loudly when the HIP library is missing)


def banner(msg):
    print(f"\n[case] {msg}", flush=True)


def check(gp, what, out_dtype=torch.float16):
    ref = oracle.reference_output(gp.inp)
    y = gp.dequant(out_dtype=out_dtype).float().cpu().numpy()
    fro, mx = assert_fp_close(y, ref, what)
    print(f"[err] {what}: relFro {fro:.3e} max/rms {mx:.3e}", flush=True)
    return y


# ----------------------------------------------------------------- 16-token slabs (1-bit weights)

@pytest.mark.parametrize("M,K,N", [(1, 1024, 300), (5, 1664, 1000), (16, 2048, 600), (17, 4736, 1000),
                                   (40, 1024, 300), (64, 8192, 520)])
def test_slab_kernel_binary_per_column(M, K, N, tune):
    tune(DEQUANT_KIND=2)
    banner(f"dequant slab kernel, binary per-column, M={M} K={K} N={N}")
    gp = GpuProblem(W.make_inputs(5, 0, M=M, K=K, N=N))
    check(gp, f"slab M={M} K={K} N={N}")


@pytest.mark.parametrize("splits", [1, 2, 3, 37])
def test_slab_kernel_forced_splits(splits, tune):
    """K = 37 128-blocks: one split stages chunks of 16, 16 and 5 blocks (the last
    ends inside the ring of eight blocks of weight words); 3 splits give 13-block
    ranges; 37 splits one block each."""
    tune(DEQUANT_KIND=2, DEQUANT_SPLITS=splits)
    banner(f"dequant slab kernel, forced splits={splits}, M=20 K=4736 N=700")
    gp = GpuProblem(W.make_inputs(5, 0, M=20, K=4736, N=700))
    check(gp, f"slab splits={splits}")
    need = L.dequant_workspace_size(gp.p, 20)
    assert (need > 0) == (splits > 1)


def test_slab_kernel_binary_per_tensor(tune):
    tune(DEQUANT_KIND=2)
    banner("dequant slab kernel, binary per-tensor FP32 scale, M=16 K=2048 N=700")
    inp = W.make_custom(W.WFMT_BINARY, 1, 0, W.ACT_FP16, M=16, K=2048, N=700, seed=901, scale_fp32=True)
    check(GpuProblem(inp), "slab per-tensor")


def test_slab_kernel_planned_for_few_tokens():
    """Binary per-column weights at M <= 64 take the slab kernel by default and split
    K on a narrow layer (FP32 partials in the workspace)."""
    banner("dequant planned: binary M=16 K=8192 N=1000")
    gp = GpuProblem(W.make_inputs(5, 0, M=16, K=8192, N=1000))
    assert L.dequant_workspace_size(gp.p, 16) > 0
    check(gp, "slab planned")


# ----------------------------------------------------------------- tile kernels with K splits

@pytest.mark.parametrize("kind,splits,cid,M,K,N", [
    (1, 0, 4, 256, 2048, 520),    # 3 tiles: K split into 16 one-block ranges
    (1, 3, 4, 300, 2048, 1000),   # ragged M: two tile rows, 6-block ranges
    (1, 1, 5, 260, 1024, 300),    # no split
    (0, 0, 4, 100, 1024, 520),    # 128 x 128 tiles, planned split
    (0, 3, 3, 70, 2048, 300),     # INT4 groups of 128, 6-block ranges
    (0, 1, 1, 33, 1024, 1000),    # INT2 no split
])
def test_tile_kernels_with_k_split(kind, splits, cid, M, K, N, tune):
    tune(DEQUANT_KIND=kind, DEQUANT_SPLITS=splits)
    banner(f"dequant tile kernel kind={kind} splits={splits or 'planned'} config={cid} M={M} K={K} N={N}")
    gp = GpuProblem(W.make_inputs(cid, 0, M=M, K=K, N=N))
    check(gp, f"tile kind={kind} splits={splits}")
    check(gp, f"tile kind={kind} splits={splits} fp32 out", out_dtype=torch.float32)


# ----------------------------------------------------------------- epilogue and determinism

@pytest.mark.parametrize("kind,splits", [(2, 1), (2, 4), (1, 0), (0, 2)])
def test_accumulate_and_determinism(kind, splits, tune):
    tune(DEQUANT_KIND=kind, DEQUANT_SPLITS=splits)
    banner(f"dequant accumulate kind={kind} splits={splits}")
    M = 40 if kind == 2 else 200
    gp = GpuProblem(W.make_inputs(5, 0, M=M, K=2048, N=600))
    ref = oracle.reference_output(gp.inp)
    base = torch.from_numpy(np.random.default_rng(7).standard_normal((M, 600)).astype(np.float32)).cuda()
    out = base.clone()
    y = gp.dequant(out_dtype=torch.float32, accumulate=True, out=out)
    assert y.data_ptr() == out.data_ptr()
    assert_fp_close((out - base).cpu().numpy(), ref, "accumulate")
    a = gp.dequant(out_dtype=torch.float32)
    b = gp.dequant(out_dtype=torch.float32)
    assert torch.equal(a, b), "comparison path not bitwise reproducible"


@pytest.mark.parametrize("kind", [0, 1])
@pytest.mark.parametrize("wfmt,bits", [(W.WFMT_TERNARY, 2), (W.WFMT_UINT, 4), (W.WFMT_BINARY, 1)])
def test_tile_kernels_per_tensor_scale(kind, wfmt, bits, tune):
    """One FP32 scale (and zero) for the whole tensor: the 256 x 256 kernel reads them
    once per workgroup, the 128 x 128 kernel per K step."""
    tune(DEQUANT_KIND=kind)
    banner(f"dequant tile kernel kind={kind}, per-tensor scale, wfmt={wfmt} b={bits}, M=130 K=1024 N=300")
    inp = W.make_custom(wfmt, bits, 0, W.ACT_FP16, M=130, K=1024, N=300, seed=950 + 10 * kind + wfmt,
                        scale_fp32=(wfmt != W.WFMT_UINT))  # UINT: FP16 scale and zero
    check(GpuProblem(inp), f"tile kind={kind} per-tensor wfmt={wfmt}")
