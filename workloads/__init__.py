"""Seeded synthetic workloads for LUT-based mixed-precision GEMM.

This module only draws random inputs of the right shapes, dtypes and value
distributions. It holds none of the method's arithmetic (no dequantization, no
tables, no reinterpretation), so both the CPU oracle and the HIP path can use it
without sharing any computation.

The workload families are the synthetic stand-ins for the layer shapes the
paper evaluates on (LLaMA-2 7B/70B GEMV/GEMM shapes in the motivation figure of
Section 2.3, BitNet b1.58 ternary weights in Table 1, and the LLaMA-2-13B shape of
the kernel-level evaluation in Section 4.3).  No dataset or trained
weight is used anywhere.

Seeding: ``numpy.random.default_rng([2408, 6003, config_id, shape_id, M])``;
draw order is codes, scales, zeros, activations; real values are drawn in
float64 and rounded to their storage dtype (round-to-nearest-even).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np

# Weight formats (same integer values as the C ABI enum).
WFMT_UINT = 0      # codes q in [0, 2^b), real weight r = s * (q - z), s and z per group
WFMT_BINARY = 1    # codes q in {0, 1}, real weight r = s * (2q - 1)
WFMT_TERNARY = 2   # int8 w in {-1, 0, +1}, real weight r = s * w

ACT_FP16 = 0
ACT_INT8 = 1
ACT_FP16_LUT8 = 2   # FP16 activations, tables quantized to INT8 per table (same draws as ACT_FP16)


@dataclass(frozen=True)
class Workload:
    """One workload family: a weight format plus a list of (K, N) shapes and token counts."""
    config_id: int
    name: str
    wfmt: int
    bits: int
    group: Optional[int]          # quantization group along K; None = per-channel (G = K); 0 = per-tensor
    scale_fp32: bool
    zero_max: float               # zeros drawn U(0, zero_max) for the UINT format
    act: int
    kn: Tuple[Tuple[int, int], ...]
    ms: Tuple[int, ...]
    description: str = ""

    def group_size(self, K: int) -> int:
        if self.group is None:
            return K
        return self.group

    def shapes(self) -> List[Tuple[int, int, int, int]]:
        """All (shape_id, M, K, N) of the family."""
        out = []
        for sid, (K, N) in enumerate(self.kn):
            for M in self.ms:
                out.append((sid, M, K, N))
        return out


WORKLOADS: Dict[int, Workload] = {
    1: Workload(1, "int2_g128_gemv_1k", WFMT_UINT, 2, 128, False, 3.0, ACT_FP16,
                ((1024, 1024),), (1,),
                "mpGEMV M=1 K=N=1024, INT2 codes U{0..3}, group-128 FP16 scale U(0.01,0.1) and zero U(0,3), "
                "FP16 activations N(0,1), FP32 accumulate"),
    2: Workload(2, "ternary_int8_gemv_4k", WFMT_TERNARY, 2, 0, True, 0.0, ACT_INT8,
                ((4096, 4096),), (1,),
                "ternary mpGEMV M=1 K=N=4096, w in {-1,0,+1} p=1/3, per-tensor FP32 scale U(0.01,0.1), "
                "activations N(0,1) -> per-token absmax INT8, INT32 accumulate"),
    3: Workload(3, "int4_g128_llama7b_decode", WFMT_UINT, 4, 128, False, 15.0, ACT_FP16,
                ((4096, 12288), (4096, 4096), (4096, 22016), (11008, 4096)), (1,),
                "LLaMA-7B-shaped decode M=1, INT4 codes U{0..15}, group-128 FP16 scale U(0.01,0.1) and "
                "zero U(0,15), FP16 activations N(0,1), FP32 accumulate"),
    4: Workload(4, "int2_g128_prefill_4k", WFMT_UINT, 2, 128, False, 3.0, ACT_FP16,
                ((4096, 4096),), (4096,),
                "prefill mpGEMM M=4096 K=N=4096, INT2 group-128 as the 1k GEMV, FP16 activations"),
    5: Workload(5, "binary_llama70b", WFMT_BINARY, 1, None, False, 0.0, ACT_FP16,
                ((8192, 28672), (28672, 8192)), (1, 16, 256),
                "LLaMA-70B-shaped layers, binary {-1,+1} weights with per-channel FP16 scale "
                "U(0.01,0.1), FP16 activations N(0,1), M in {1,16,256}"),
    6: Workload(6, "binary_llama13b_kernel_eval", WFMT_BINARY, 1, None, False, 0.0, ACT_FP16,
                ((5120, 27648),), (2048,),
                "the LLaMA-2-13B mpGEMM shape of the paper's kernel-level evaluation (Section 4.3): "
                "M=2048 N=27648 K=5120, binary {-1,+1} weights (W_INT1 A_FP16) with per-channel FP16 "
                "scale U(0.01,0.1), FP16 activations N(0,1)"),
}


@dataclass
class Inputs:
    """Host arrays for one mpGEMM problem (all C-contiguous)."""
    M: int
    K: int
    N: int
    wfmt: int
    bits: int
    group: int                    # 0 = per-tensor, else divides K
    act_kind: int
    codes: np.ndarray             # [N, K] uint8 (UINT/BINARY) or int8 (TERNARY)
    scales: np.ndarray            # [N, K/G] float16, or [1] float32 (per-tensor)
    zeros: Optional[np.ndarray]   # [N, K/G] float16 (UINT) or None
    act: np.ndarray               # [M, K] float16
    meta: dict = field(default_factory=dict)


def rng_for(config_id: int, shape_id: int, M: int) -> np.random.Generator:
    return np.random.default_rng([2408, 6003, config_id, shape_id, M])


def draw(wfmt: int, bits: int, group: int, scale_fp32: bool, zero_max: float, act_kind: int,
         M: int, K: int, N: int, rng: np.random.Generator) -> Inputs:
    """Draw codes, scales, zeros and activations, in that order."""
    if group != 0 and K % group != 0:
        raise ValueError(f"group {group} does not divide K={K}")
    n_groups = 1 if group == 0 else K // group
    # codes
    if wfmt == WFMT_UINT:
        codes = rng.integers(0, 1 << bits, size=(N, K), dtype=np.uint8)
    elif wfmt == WFMT_BINARY:
        codes = rng.integers(0, 2, size=(N, K), dtype=np.uint8)
    elif wfmt == WFMT_TERNARY:
        codes = rng.integers(-1, 2, size=(N, K), dtype=np.int8)
    else:
        raise ValueError(f"unknown weight format {wfmt}")
    # scales
    if group == 0:
        s = rng.uniform(0.01, 0.1, size=(1,))
        scales = s.astype(np.float32) if scale_fp32 else s.astype(np.float16)
    else:
        s = rng.uniform(0.01, 0.1, size=(N, n_groups))
        scales = s.astype(np.float32) if scale_fp32 else s.astype(np.float16)
    # zeros
    zeros = None
    if wfmt == WFMT_UINT:
        zeros = rng.uniform(0.0, zero_max, size=scales.shape).astype(np.float16)
    # activations
    act = rng.standard_normal(size=(M, K)).astype(np.float16)
    return Inputs(M=M, K=K, N=N, wfmt=wfmt, bits=bits, group=group, act_kind=act_kind,
                  codes=np.ascontiguousarray(codes), scales=np.ascontiguousarray(scales),
                  zeros=None if zeros is None else np.ascontiguousarray(zeros),
                  act=np.ascontiguousarray(act))


def make_inputs(config_id: int, shape_id: int = 0, M: Optional[int] = None,
                K: Optional[int] = None, N: Optional[int] = None) -> Inputs:
    """Inputs of workload family ``config_id``.

    ``shape_id`` picks the (K, N) pair of the family; ``M``, ``K`` and ``N`` may be
    overridden to draw a smaller case with the same distributions (parity tests).
    """
    w = WORKLOADS[config_id]
    k0, n0 = w.kn[shape_id]
    M = w.ms[0] if M is None else M
    K = k0 if K is None else K
    N = n0 if N is None else N
    G = w.group_size(K)
    inp = draw(w.wfmt, w.bits, G, w.scale_fp32, w.zero_max, w.act, M, K, N,
               rng_for(config_id, shape_id, M))
    inp.meta = {"config_id": config_id, "shape_id": shape_id, "name": w.name}
    return inp


def make_custom(wfmt: int, bits: int, group: int, act_kind: int, M: int, K: int, N: int,
                seed: int, scale_fp32: bool = False, zero_max: Optional[float] = None) -> Inputs:
    """Inputs for an edge-case shape, seeded by ``seed``."""
    if zero_max is None:
        zero_max = float((1 << bits) - 1)
    rng = np.random.default_rng([2408, 6003, 99, seed, M, K, N])
    return draw(wfmt, bits, group, scale_fp32, zero_max, act_kind, M, K, N, rng)
