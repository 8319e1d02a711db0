"""CPU oracle for LUT-based mixed-precision GEMM -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's ``cpu_baseline``
leg may import this package.  The product path (``paper_2408_06003_amd``) never
imports it, and it never imports the product path: the two share no code, only
the seeded input generators in ``workloads``.

The heavy lifting is the plain C file ``mpgemm_oracle.c`` (float64 / int64
direct dot products of dequantized weights, Section 3.1.2 Eq. 1 and Eq. 3 of
the paper), compiled with gcc into ``liboracle.so``; this module marshals numpy
arrays into it.  ``lut_identities`` is an exact-rational model of the paper's
table method used to pin this oracle.

Functions and the passage each follows:
* ``mpgemm_fp``        -- y = A x dequant(W)^T (+Acc), Eq. 1 / Eq. 3, LMMA semantics (Section 3.3.1)
* ``quantize_int8``    -- per-token absmax INT8 activations (FP32 replica; quantizer not fixed by the paper)
* ``mpgemm_int``       -- integer accumulator of INT8 activations x BINARY/TERNARY weights
* ``int_output_f32``   -- y = (float(acc) * s_a) * s_w
* ``half_tables``      -- precompute output: symmetric half tables (Eq. 4-5)
* ``group_sums``       -- activation sums per quantization group (zero-point term of Eq. 3)
* ``token_pow2``       -- per-token power-of-two normalizer of the FP16 tables
* ``lut8_tables``      -- INT8 table quantization, per table (Section 3.1.3): codes, scales
* ``mpgemm_lut8``      -- FP mpGEMM through the INT8-quantized tables: the approximation
                          follows the method's steps (Section 3.1.3, Eq. 2-6, bit-serial
                          planes of Section 3.2.1); no closed form exists for it
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mpgemm_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

WFMT_UINT, WFMT_BINARY, WFMT_TERNARY = 0, 1, 2

_P = ctypes.c_void_p
_I64 = ctypes.c_int64


def build(force: bool = False) -> str:
    """Compile ``liboracle.so`` with gcc (plain C, OpenMP, no FP contraction)."""
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp"
        cmd = ["gcc", "-O2", "-std=c99", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
               "-shared", "-fPIC", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        L = ctypes.CDLL(_LIB_PATH)
        L.oracle_mpgemm_f64.restype = ctypes.c_int
        L.oracle_mpgemm_f64.argtypes = [_I64, _I64, _I64, _P, _P, ctypes.c_int, _I64, _P, _P,
                                        _P, _I64, _P, _I64, _P, _P]
        L.oracle_quantize_int8.restype = None
        L.oracle_quantize_int8.argtypes = [_I64, _I64, _P, _P, _P]
        L.oracle_mpgemm_i64.restype = ctypes.c_int
        L.oracle_mpgemm_i64.argtypes = [_I64, _I64, _I64, _P, _P, ctypes.c_int, _P, _I64, _P, _I64,
                                        _P, _P]
        L.oracle_int_output_f32.restype = None
        L.oracle_int_output_f32.argtypes = [_I64, _I64, _P, _P, _P, _P]
        L.oracle_half_tables_f64.restype = None
        L.oracle_half_tables_f64.argtypes = [_I64, _I64, _P, _P]
        L.oracle_half_tables_i64.restype = None
        L.oracle_half_tables_i64.argtypes = [_I64, _I64, _P, _P]
        L.oracle_group_sums_f64.restype = None
        L.oracle_group_sums_f64.argtypes = [_I64, _I64, _I64, _P, _P]
        L.oracle_group_sums_i64.restype = None
        L.oracle_group_sums_i64.argtypes = [_I64, _I64, _I64, _P, _P]
        L.oracle_token_pow2.restype = None
        L.oracle_token_pow2.argtypes = [_I64, _I64, _P, _P]
        L.oracle_lut8_tables.restype = None
        L.oracle_lut8_tables.argtypes = [_I64, _I64, _P, _P, _P, _P]
        L.oracle_mpgemm_lut8.restype = ctypes.c_int
        L.oracle_mpgemm_lut8.argtypes = [_I64, _I64, _I64, _P, _P, ctypes.c_int, ctypes.c_int, _I64, _P, _P,
                                         _P, _I64, _P, _I64, _P]
        _lib = L
    return _lib


def _ptr(x: Optional[np.ndarray]):
    return None if x is None else x.ctypes.data_as(ctypes.c_void_p)


def _f64(x) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(x, dtype=np.float64))


def _subset(idx: Optional[Sequence[int]]):
    if idx is None:
        return None, 0
    arr = np.ascontiguousarray(np.asarray(idx, dtype=np.int64))
    return arr, int(arr.size)


def mpgemm_fp(act: np.ndarray, codes: np.ndarray, wfmt: int, group: int, scales: np.ndarray,
              zeros: Optional[np.ndarray], rows=None, cols=None,
              acc: Optional[np.ndarray] = None) -> np.ndarray:
    """float64 y[rows][cols] = sum_k a[m,k] * r[n,k] (+ acc), r from Eq. 1 element by element."""
    a = _f64(act)
    M, K = a.shape
    N = codes.shape[0]
    if codes.shape[1] != K:
        raise ValueError("codes must be [N, K]")
    c = np.ascontiguousarray(codes)
    s = _f64(scales).reshape(-1)
    z = None if zeros is None else _f64(zeros).reshape(-1)
    r_arr, nr = _subset(rows)
    c_arr, nc = _subset(cols)
    out_r = nr if rows is not None else M
    out_c = nc if cols is not None else N
    y = np.empty((out_r, out_c), dtype=np.float64)
    acc64 = None if acc is None else _f64(acc).reshape(out_r, out_c)
    rc = lib().oracle_mpgemm_f64(M, N, K, _ptr(a), _ptr(c), wfmt, group, _ptr(s), _ptr(z),
                                 _ptr(r_arr), nr, _ptr(c_arr), nc, _ptr(acc64), _ptr(y))
    if rc != 0:
        raise ValueError("oracle_mpgemm_f64 rejected its arguments")
    return y


def quantize_int8(act: np.ndarray):
    """Per-token absmax INT8 quantization in FP32: returns (q int8 [M,K], s_a float32 [M])."""
    a = np.ascontiguousarray(np.asarray(act).astype(np.float32))
    M, K = a.shape
    q = np.empty((M, K), dtype=np.int8)
    s = np.empty((M,), dtype=np.float32)
    lib().oracle_quantize_int8(M, K, _ptr(a), _ptr(q), _ptr(s))
    return q, s


def mpgemm_int(qa: np.ndarray, codes: np.ndarray, wfmt: int, rows=None, cols=None,
               acc: Optional[np.ndarray] = None) -> np.ndarray:
    """int64 acc[rows][cols] = sum_k qa[m,k] * w[n,k] for BINARY (w = 2q-1) or TERNARY weights."""
    q = np.ascontiguousarray(qa.astype(np.int8))
    M, K = q.shape
    N = codes.shape[0]
    c = np.ascontiguousarray(codes)
    r_arr, nr = _subset(rows)
    c_arr, nc = _subset(cols)
    out_r = nr if rows is not None else M
    out_c = nc if cols is not None else N
    out = np.empty((out_r, out_c), dtype=np.int64)
    acc64 = None if acc is None else np.ascontiguousarray(acc.astype(np.int64)).reshape(out_r, out_c)
    rc = lib().oracle_mpgemm_i64(M, N, K, _ptr(q), _ptr(c), wfmt, _ptr(r_arr), nr, _ptr(c_arr), nc,
                                 _ptr(acc64), _ptr(out))
    if rc != 0:
        raise ValueError("oracle_mpgemm_i64 supports BINARY and TERNARY weights only")
    return out


def int_output_f32(acc: np.ndarray, s_a_rows: np.ndarray, s_w_cols: np.ndarray) -> np.ndarray:
    """y = (float(acc) * s_a[row]) * s_w[col] in FP32."""
    a = np.ascontiguousarray(acc.astype(np.int64))
    nr, nc = a.shape
    sa = np.ascontiguousarray(np.asarray(s_a_rows, dtype=np.float32).reshape(nr))
    sw = np.ascontiguousarray(np.asarray(s_w_cols, dtype=np.float32).reshape(nc))
    y = np.empty((nr, nc), dtype=np.float32)
    lib().oracle_int_output_f32(nr, nc, _ptr(a), _ptr(sa), _ptr(sw), _ptr(y))
    return y


def half_tables(act: np.ndarray) -> np.ndarray:
    """Half tables T[m][j][idx] (float64 for float inputs, int64 for int8 inputs)."""
    if act.dtype == np.int8:
        q = np.ascontiguousarray(act)
        M, K = q.shape
        T = np.empty((M, K // 4, 8), dtype=np.int64)
        lib().oracle_half_tables_i64(M, K, _ptr(q), _ptr(T))
        return T
    a = _f64(act)
    M, K = a.shape
    T = np.empty((M, K // 4, 8), dtype=np.float64)
    lib().oracle_half_tables_f64(M, K, _ptr(a), _ptr(T))
    return T


def group_sums(act: np.ndarray, group: int) -> np.ndarray:
    """S[m][q] = sum of the activations of quantization group q (group 0 = whole row)."""
    if act.dtype == np.int8:
        q = np.ascontiguousarray(act)
        M, K = q.shape
        Q = 1 if group == 0 else K // group
        S = np.empty((M, Q), dtype=np.int64)
        lib().oracle_group_sums_i64(M, K, group, _ptr(q), _ptr(S))
        return S
    a = _f64(act)
    M, K = a.shape
    Q = 1 if group == 0 else K // group
    S = np.empty((M, Q), dtype=np.float64)
    lib().oracle_group_sums_f64(M, K, group, _ptr(a), _ptr(S))
    return S


def token_pow2(act: np.ndarray) -> np.ndarray:
    """mult[m] = 2^e with max_k |a[m,k]| = f 2^e, f in [0.5, 1) (1 for an all-zero row)."""
    a = _f64(act)
    M, K = a.shape
    out = np.empty((M,), dtype=np.float64)
    lib().oracle_token_pow2(M, K, _ptr(a), _ptr(out))
    return out


def reference_output(inp, rows=None, cols=None, acc=None):
    """Oracle output for a ``workloads.Inputs`` problem.

    FP16 activations: float64 y.  INT8 activations: (int64 accumulator, float32 y) where
    y = (float(acc) * s_a) * s_w.  FP16 activations with INT8 table quantization
    (act_kind 2): float64 y through the quantized tables (``mpgemm_lut8``).
    """
    if inp.act_kind == 0:
        return mpgemm_fp(inp.act, inp.codes, inp.wfmt, inp.group, inp.scales, inp.zeros,
                         rows=rows, cols=cols, acc=acc)
    if inp.act_kind == 2:  # FP16 activations through INT8-quantized tables
        y = mpgemm_lut8(inp.act, inp.codes, inp.wfmt, inp.bits, inp.group, inp.scales, inp.zeros,
                        rows=rows, cols=cols)
        return y if acc is None else y + np.asarray(acc, dtype=np.float64)
    qa, sa = quantize_int8(inp.act)
    iacc = mpgemm_int(qa, inp.codes, inp.wfmt, rows=rows, cols=cols)
    r = np.arange(inp.M) if rows is None else np.asarray(rows)
    c = np.arange(inp.N) if cols is None else np.asarray(cols)
    if inp.group == 0:
        sw = np.full(c.shape, np.asarray(inp.scales, dtype=np.float32).reshape(-1)[0], dtype=np.float32)
    else:
        if inp.group != inp.K:
            raise ValueError("INT8 activations need a per-tensor or per-channel weight scale")
        sw = np.asarray(inp.scales, dtype=np.float32).reshape(inp.N)[c]
    y = int_output_f32(iacc, sa[r], sw)
    return iacc, y


def lut8_tables(act: np.ndarray):
    """INT8-quantized half tables: (q int8 [M, K/4, 8], scale float32 [M, K/4], mult float64 [M])."""
    a = np.ascontiguousarray(np.asarray(act).astype(np.float32))
    M, K = a.shape
    q = np.empty((M, K // 4, 8), dtype=np.int8)
    sc = np.empty((M, K // 4), dtype=np.float32)
    mult = np.empty((M,), dtype=np.float64)
    lib().oracle_lut8_tables(M, K, _ptr(a), _ptr(q), _ptr(sc), _ptr(mult))
    return q, sc, mult


def mpgemm_lut8(act: np.ndarray, codes: np.ndarray, wfmt: int, bits: int, group: int, scales: np.ndarray,
                zeros: Optional[np.ndarray], rows=None, cols=None) -> np.ndarray:
    """float64 y[rows][cols] through INT8-quantized tables (the approximation's own reference)."""
    a = np.ascontiguousarray(np.asarray(act).astype(np.float32))
    M, K = a.shape
    N = codes.shape[0]
    c = np.ascontiguousarray(codes)
    s = _f64(scales).reshape(-1)
    z = None if zeros is None else _f64(zeros).reshape(-1)
    r_arr, nr = _subset(rows)
    c_arr, nc = _subset(cols)
    y = np.empty((nr if rows is not None else M, nc if cols is not None else N), dtype=np.float64)
    rc = lib().oracle_mpgemm_lut8(M, N, K, _ptr(a), _ptr(c), wfmt, bits, group, _ptr(s), _ptr(z),
                                  _ptr(r_arr), nr, _ptr(c_arr), nc, _ptr(y))
    if rc != 0:
        raise ValueError("oracle_mpgemm_lut8 rejected its arguments")
    return y
