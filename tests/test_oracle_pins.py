"""Pins of the CPU oracle against what the paper and the mathematics fix.

Every test here runs without a GPU.  The oracle (float64/int64 dense definition,
``oracle/mpgemm_oracle.c``) is checked against:
* the paper's worked example (Section 3.1.2) and its Eq. 2 mapping example (golden fixtures),
* the LUT reformulation identities, Eq. 2-6, evaluated exactly in rationals and by
  brute force over every weight pattern of one table group,
* library routines it reduces to on small shapes (numpy float64 matmul, np.rint),
* invariants (one-hot activations, zero activations, T[0] = -sum of the group).
"""
import os
from fractions import Fraction
from itertools import product

import numpy as np
import pytest

import oracle
from oracle import lut_identities as L
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def read_fixture(name):
    out = {}
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            k, v = line.split("=", 1)
            out[k.strip()] = v.split()
    return out


def frac(x):
    return Fraction(x)


# --------------------------------------------------------------------------- worked example

def test_worked_example_dense_oracle():
    fx = read_fixture("worked_example_sec312.txt")
    bits = [int(b) for b in fx["bits"]]
    s = float(Fraction(fx["s"][0]))
    z = float(Fraction(fx["z"][0]))
    coef = [int(c) for c in fx["coefficients"]]
    codes = np.array([bits], dtype=np.uint8)                # N=1, K=4, W3 first
    scales = np.array([[s]], dtype=np.float16)
    zeros = np.array([[z]], dtype=np.float16)
    # one-hot activations read off the coefficient of each of A, B, C, D
    eye = np.eye(4, dtype=np.float16)
    y = oracle.mpgemm_fp(eye, codes, W.WFMT_UINT, 4, scales, zeros)
    assert y[:, 0].tolist() == coef
    # and the value for a concrete (A, B, C, D)
    act = np.array([[1.0, 2.0, 4.0, 8.0]], dtype=np.float16)
    y = oracle.mpgemm_fp(act, codes, W.WFMT_UINT, 4, scales, zeros)
    assert y[0, 0] == -1.0 + 2.0 - 4.0 - 8.0


def test_worked_example_reinterpretation():
    fx = read_fixture("worked_example_sec312.txt")
    bits = [int(b) for b in fx["bits"]]
    s, z = Fraction(fx["s"][0]), Fraction(fx["z"][0])
    qp = []
    for q in bits:
        q1, s1, z1 = L.reinterpret(q, s, z, 1)
        assert s1 == Fraction(fx["s_prime"][0]) and z1 == Fraction(fx["z_prime"][0])
        qp.append(q1)
    assert qp == [int(v) for v in fx["q_prime"]]
    acts = [Fraction(1), Fraction(2), Fraction(4), Fraction(8)]
    assert L.lut_group_dot(acts, bits, s, z, 1) == -1 + 2 - 4 - 8


def test_eq2_mapping_fixture():
    fx = read_fixture("eq2_uint4_mapping.txt")
    b = int(fx["bits"][0])
    got = [L.reinterpret(int(q), Fraction(1), Fraction(0), b)[0] for q in fx["q"]]
    assert got == [int(v) for v in fx["q_prime"]]


# --------------------------------------------------------------------------- identities

def rand_fracs(rng, n, den=64):
    return [Fraction(int(v), den) for v in rng.integers(-500, 500, size=n)]


@pytest.mark.parametrize("b", [1, 2, 3, 4])
def test_eq2_dequant_identity(b):
    rng = np.random.default_rng(1)
    for _ in range(20):
        s = Fraction(int(rng.integers(1, 1000)), 512)
        z = Fraction(int(rng.integers(0, 1000)), 97)
        for q in range(1 << b):
            q1, s1, z1 = L.reinterpret(q, s, z, b)
            assert s1 * (q1 - z1) == s * (q - z)


def test_eq4_symmetry_and_eq5_eq6_lookup():
    rng = np.random.default_rng(2)
    for _ in range(50):
        acts = rand_fracs(rng, 4)
        full = L.full_table(acts)
        half = L.half_table(acts)
        assert len(half) == 8
        for p in range(16):
            assert full[p] == -full[(~p) & 0xF]                  # Eq. 4
            assert L.lookup_eq5(half, p) == full[p]              # Eq. 5
            sign, idx = L.offline_negate(p)
            assert sign == (p >> 3) & 1 and 0 <= idx < 8
            assert L.lookup_eq6(half, sign, idx) == full[p]      # Eq. 6
        # T[0] is the all-(-1) pattern: minus the group sum
        assert half[0] == -sum(acts)


@pytest.mark.parametrize("b", [1, 2, 4])
def test_bit_serial_composes_with_reinterpretation(b):
    for q in range(1 << b):
        planes = L.bit_planes(q, b)
        assert sum((1 << t) * (2 * planes[t] - 1) for t in range(b)) == 2 * q - ((1 << b) - 1)


@pytest.mark.parametrize("b", [1, 2, 4])
def test_lut_bruteforce_equals_dense_oracle(b):
    """Every (2^b)^4 code combination of one table group: LUT evaluation (exact) == oracle."""
    rng = np.random.default_rng(10 + b)
    combos = np.array(list(product(range(1 << b), repeat=4)), dtype=np.uint8)   # [N, 4]
    N = combos.shape[0]
    M = 1 if b == 4 else 2
    act = rng.standard_normal((M, 4)).astype(np.float16)
    scales = rng.uniform(0.01, 0.1, size=(N, 1)).astype(np.float16)
    zeros = rng.uniform(0, (1 << b) - 1, size=(N, 1)).astype(np.float16)
    y = oracle.mpgemm_fp(act, combos, W.WFMT_UINT, 4, scales, zeros)
    sub = range(N) if b < 4 else rng.choice(N, size=4096, replace=False)
    for n in sub:
        for m in range(M):
            a4 = [frac(float(v)) for v in act[m]]
            exact = L.lut_group_dot(a4, [int(c) for c in combos[n]], frac(float(scales[n, 0])),
                                    frac(float(zeros[n, 0])), b)
            mag = sum(abs(x) for x in a4) * frac(float(scales[n, 0])) * (1 << b)
            assert abs(frac(y[m, n]) - exact) <= mag * Fraction(1, 2 ** 50)
    # the direct definition also holds column by column, exactly, on a rational rendering
    n = int(rng.integers(0, N))
    direct = sum(frac(float(act[0, k])) * L.dequant(int(combos[n, k]), frac(float(scales[n, 0])),
                                                    frac(float(zeros[n, 0]))) for k in range(4))
    assert abs(frac(y[0, n]) - direct) <= abs(direct) * Fraction(1, 2 ** 50) + Fraction(1, 2 ** 80)


def test_ternary_all_patterns_integer_lut():
    """All 3^4 ternary patterns: (sum_t 2^t L_t + S) is even and /2 equals the integer dot product."""
    rng = np.random.default_rng(5)
    pats = np.array(list(product([-1, 0, 1], repeat=4)), dtype=np.int8)
    for _ in range(4):
        qa = rng.integers(-127, 128, size=(1, 4)).astype(np.int8)
        acc = oracle.mpgemm_int(qa, pats, W.WFMT_TERNARY)
        for n in range(pats.shape[0]):
            numer, val = L.ternary_int_dot([int(v) for v in qa[0]], [int(v) for v in pats[n]])
            assert numer % 2 == 0
            assert val == int(acc[0, n]) == int(np.dot(qa[0].astype(np.int64), pats[n].astype(np.int64)))


def test_lut_mpgemm_small_uint_groups():
    """Whole small problem through the table model vs the oracle (several quant groups)."""
    inp = W.make_custom(W.WFMT_UINT, 2, 8, W.ACT_FP16, M=2, K=16, N=3, seed=7)
    y = oracle.mpgemm_fp(inp.act, inp.codes, inp.wfmt, inp.group, inp.scales, inp.zeros)
    A = [[frac(float(v)) for v in row] for row in inp.act]
    C = [[int(v) for v in row] for row in inp.codes]
    S = [[frac(float(v)) for v in row] for row in inp.scales]
    Z = [[frac(float(v)) for v in row] for row in inp.zeros]
    yl = L.lut_mpgemm(A, C, S, Z, 2, 8)
    for m in range(2):
        for n in range(3):
            assert abs(frac(y[m, n]) - yl[m][n]) <= Fraction(1, 2 ** 40)


# --------------------------------------------------------------------------- library reductions

def numpy_dense(inp):
    K = inp.K
    G = inp.group if inp.group else K
    s = np.repeat(np.asarray(inp.scales, np.float64).reshape(inp.N if inp.group else 1, -1), G, axis=1)
    if inp.group == 0:
        s = np.broadcast_to(s.reshape(1, -1)[:, :1], (inp.N, K))
    if inp.wfmt == W.WFMT_UINT:
        z = np.repeat(np.asarray(inp.zeros, np.float64), G, axis=1)
        R = s * (inp.codes.astype(np.float64) - z)
    elif inp.wfmt == W.WFMT_BINARY:
        R = s * (2.0 * inp.codes.astype(np.float64) - 1.0)
    else:
        R = s * inp.codes.astype(np.float64)
    return inp.act.astype(np.float64) @ R.T


@pytest.mark.parametrize("wfmt,bits,group", [(W.WFMT_UINT, 2, 128), (W.WFMT_UINT, 4, 64),
                                             (W.WFMT_BINARY, 1, 256), (W.WFMT_TERNARY, 2, 0),
                                             (W.WFMT_UINT, 1, 32)])
def test_oracle_matches_numpy_matmul(wfmt, bits, group):
    inp = W.make_custom(wfmt, bits, group, W.ACT_FP16, M=5, K=256, N=37, seed=3,
                        scale_fp32=(group == 0))
    y = oracle.mpgemm_fp(inp.act, inp.codes, inp.wfmt, inp.group, inp.scales, inp.zeros)
    ref = numpy_dense(inp)
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-12)
    # row / column subsets return the same entries
    rows, cols = [4, 0, 2], [36, 1, 5, 5]
    ys = oracle.mpgemm_fp(inp.act, inp.codes, inp.wfmt, inp.group, inp.scales, inp.zeros,
                          rows=rows, cols=cols)
    assert np.array_equal(ys, y[np.ix_(rows, cols)])
    # the +Acc term
    acc = np.arange(5 * 37, dtype=np.float64).reshape(5, 37)
    ya = oracle.mpgemm_fp(inp.act, inp.codes, inp.wfmt, inp.group, inp.scales, inp.zeros, acc=acc)
    assert np.allclose(ya, y + acc, rtol=1e-13, atol=1e-12)


def test_one_hot_and_zero_activations():
    inp = W.make_custom(W.WFMT_UINT, 4, 128, W.ACT_FP16, M=1, K=256, N=8, seed=4)
    for k in [0, 1, 127, 128, 255]:
        e = np.zeros((1, 256), dtype=np.float16)
        e[0, k] = 1.0
        y = oracle.mpgemm_fp(e, inp.codes, inp.wfmt, inp.group, inp.scales, inp.zeros)
        q = k // 128
        expect = inp.scales[:, q].astype(np.float64) * (inp.codes[:, k].astype(np.float64)
                                                       - inp.zeros[:, q].astype(np.float64))
        assert np.array_equal(y[0], expect)
    y0 = oracle.mpgemm_fp(np.zeros((2, 256), np.float16), inp.codes, inp.wfmt, inp.group,
                          inp.scales, inp.zeros)
    assert not y0.any()


def test_int_oracle_bruteforce():
    rng = np.random.default_rng(9)
    for wfmt in (W.WFMT_TERNARY, W.WFMT_BINARY):
        qa = rng.integers(-127, 128, size=(3, 12)).astype(np.int8)
        if wfmt == W.WFMT_TERNARY:
            codes = rng.integers(-1, 2, size=(5, 12)).astype(np.int8)
            w = [[int(v) for v in r] for r in codes]
        else:
            codes = rng.integers(0, 2, size=(5, 12)).astype(np.uint8)
            w = [[2 * int(v) - 1 for v in r] for r in codes]
        acc = oracle.mpgemm_int(qa, codes, wfmt)
        for m in range(3):
            for n in range(5):
                assert int(acc[m, n]) == sum(int(qa[m, k]) * w[n][k] for k in range(12))


def test_quantizer_reduces_to_rint_and_bounds():
    rng = np.random.default_rng(11)
    a = rng.standard_normal((4, 300)).astype(np.float16)
    a[0, 17] = 127.0                       # amax = 127 -> inv = 1 -> q = rint(a)
    a[0] = np.clip(a[0] * 30, -126, 126).astype(np.float16)
    a[0, 17] = 127.0
    a[0, :6] = np.array([2.5, -2.5, 3.5, 0.5, -0.5, 1.5], dtype=np.float16)   # ties to even
    a[3] = 0.0
    q, s = oracle.quantize_int8(a)
    assert np.array_equal(q[0], np.rint(a[0].astype(np.float32)).astype(np.int8))
    assert q[0, :6].tolist() == [2, -2, 4, 0, 0, 2]
    assert s[0] == np.float32(1.0)
    assert not q[3].any() and s[3] == 0.0
    for m in range(3):
        am = a[m].astype(np.float32)
        k = int(np.argmax(np.abs(am)))
        assert abs(int(q[m, k])) == 127
        assert np.abs(q[m].astype(np.int32)).max() <= 127
        err = np.abs(am - s[m] * q[m].astype(np.float32))
        assert err.max() <= s[m] * 0.5 * (1 + 1e-5)


def test_int_output_rounding_order():
    acc = np.array([[3, -7, 1 << 23]], dtype=np.int64)
    y = oracle.int_output_f32(acc, np.array([np.float32(0.1)]), np.array([0.3, 0.07, 0.001], np.float32))
    ref = (acc.astype(np.float32) * np.float32(0.1)) * np.array([0.3, 0.07, 0.001], np.float32)
    assert np.array_equal(y, ref.astype(np.float32))


# --------------------------------------------------------------------------- precompute definitions

def test_half_tables_match_rational_model():
    rng = np.random.default_rng(12)
    a = rng.standard_normal((2, 16)).astype(np.float16)
    T = oracle.half_tables(a)
    for m in range(2):
        for j in range(4):
            h = L.half_table([frac(float(v)) for v in a[m, 4 * j:4 * j + 4]])
            assert [frac(x) for x in T[m, j]] == h
    qa = rng.integers(-127, 128, size=(2, 16)).astype(np.int8)
    Ti = oracle.half_tables(qa)
    for m in range(2):
        for j in range(4):
            h = L.half_table([Fraction(int(v)) for v in qa[m, 4 * j:4 * j + 4]])
            assert [Fraction(int(x)) for x in Ti[m, j]] == h
            assert np.abs(Ti[m, j]).max() <= 4 * 127


def test_group_sums_equal_minus_T0():
    rng = np.random.default_rng(13)
    a = rng.standard_normal((3, 64)).astype(np.float16)
    T = oracle.half_tables(a)
    S4 = oracle.group_sums(a, 4)
    assert np.array_equal(S4, -T[:, :, 0])
    S = oracle.group_sums(a, 32)
    assert np.allclose(S, S4.reshape(3, 2, 8).sum(axis=2), rtol=0, atol=1e-12)
    qa = rng.integers(-127, 128, size=(3, 64)).astype(np.int8)
    assert np.array_equal(oracle.group_sums(qa, 4), -oracle.half_tables(qa)[:, :, 0])
    assert np.array_equal(oracle.group_sums(qa, 0)[:, 0], qa.astype(np.int64).sum(axis=1))


def test_token_pow2():
    rng = np.random.default_rng(14)
    a = np.clip(rng.standard_normal((5, 50)) * np.array([[1e-3], [1.0], [300.0], [2e4], [0.0]]),
                -6e4, 6e4).astype(np.float16)
    mult = oracle.token_pow2(a)
    amax = np.abs(a.astype(np.float64)).max(axis=1)
    for m in range(5):
        if amax[m] == 0:
            assert mult[m] == 1.0
            continue
        mant, _ = np.frexp(mult[m])
        assert mant == 0.5                                   # a power of two
        assert mult[m] / 2 <= amax[m] < mult[m]


# --------------------------------------------------------------------------- workloads

def test_workloads_shapes_and_determinism():
    for cid, w in W.WORKLOADS.items():
        sid, M, K, N = w.shapes()[0]
        inp = W.make_inputs(cid, sid, M=min(M, 2), K=min(K, 1024) if K % 1024 == 0 else K, N=64)
        assert inp.codes.shape == (64, inp.K)
        assert inp.act.dtype == np.float16 and inp.act.shape == (inp.M, inp.K)
        inp2 = W.make_inputs(cid, sid, M=min(M, 2), K=inp.K, N=64)
        assert np.array_equal(inp.codes, inp2.codes) and np.array_equal(inp.act, inp2.act)
        if w.wfmt == W.WFMT_UINT:
            assert inp.codes.max() < (1 << w.bits) and inp.zeros.shape == inp.scales.shape
        if w.wfmt == W.WFMT_TERNARY:
            assert set(np.unique(inp.codes).tolist()) <= {-1, 0, 1}
            assert inp.scales.dtype == np.float32 and inp.scales.size == 1


def test_reference_output_int8_path():
    inp = W.make_inputs(2, 0, K=256, N=16)
    acc, y = oracle.reference_output(inp)
    qa, sa = oracle.quantize_int8(inp.act)
    ref = qa.astype(np.int64) @ inp.codes.astype(np.int64).T
    assert np.array_equal(acc, ref)
    yy = (acc.astype(np.float32) * sa[0]) * inp.scales.astype(np.float32)[0]
    assert np.array_equal(y, yy.astype(np.float32))


# ----------------------------------------------------------------- INT8 table quantization (Section 3.1.4)

def _exact_table_activations(M, K, rng):
    """Integer activations whose groups of 4 have |a0| + |a1| + |a2| + |a3| = 127: the
    largest half-table entry of every group is then 127 times the token's power-of-two
    unit, so INT8 table quantization is lossless."""
    a = np.zeros((M, K))
    for m in range(M):
        for j in range(K // 4):
            cut = np.sort(rng.integers(0, 128, size=3))
            parts = np.diff(np.concatenate([[0], cut, [127]]))
            a[m, 4 * j:4 * j + 4] = parts * rng.choice([-1.0, 1.0], size=4)
    return a.astype(np.float16)


@pytest.mark.parametrize("wfmt,bits,group", [(W.WFMT_UINT, 2, 128), (W.WFMT_UINT, 4, 256),
                                             (W.WFMT_BINARY, 1, 512), (W.WFMT_TERNARY, 2, 0)])
def test_lut8_lossless_tables_reduce_to_the_exact_product(wfmt, bits, group):
    """When every table is exactly representable in INT8 the table-quantized oracle must
    give the dense result: this pins its lookup (Eq. 4-6 sign handling), bit-serial
    planes, reinterpretation and zero-point term against the plain definition."""
    rng = np.random.default_rng(31)
    inp = W.make_custom(wfmt, bits, group, W.ACT_FP16, 3, 512, 40, seed=5)
    inp.act = _exact_table_activations(3, 512, rng)
    y = oracle.reference_output(inp)
    y8 = oracle.mpgemm_lut8(inp.act, inp.codes, wfmt, bits, group, inp.scales, inp.zeros)
    assert np.allclose(y8, y, rtol=1e-12, atol=1e-9 * np.abs(y).max())
    q, sc, mult = oracle.lut8_tables(inp.act)
    assert np.all(np.abs(q).max(axis=2) == 127)  # every table uses the full INT8 range


def test_lut8_table_codes_within_half_a_step():
    """Each quantized entry is within half a quantization step of the table it
    approximates (the half tables of the precompute, Eq. 5, of the normalized token)."""
    inp = W.make_custom(W.WFMT_UINT, 2, 128, W.ACT_FP16, 4, 1024, 8, seed=6)
    q, sc, mult = oracle.lut8_tables(inp.act)
    x = inp.act.astype(np.float64) / mult[:, None]
    T = oracle.half_tables(x)
    err = np.abs(q.astype(np.float64) * sc[:, :, None] - T)
    assert np.all(err <= sc[:, :, None] * (0.5 + 1e-5) + 1e-6)
    assert np.all((np.abs(q) <= 127))
    assert np.all(np.abs(q).max(axis=2) == 127)


@pytest.mark.parametrize("wfmt,bits,group", [(W.WFMT_UINT, 2, 128), (W.WFMT_UINT, 4, 128),
                                             (W.WFMT_BINARY, 1, 2048), (W.WFMT_TERNARY, 2, 0)])
def test_lut8_error_bound_and_symmetry(wfmt, bits, group):
    """Against the exact product: within the bound implied by half a step per entry
    (|T| < 4 for the normalized token, so each table step is below 4/127), and a real
    approximation (not exact).  Negating the activations negates the result exactly."""
    inp = W.make_custom(wfmt, bits, group, W.ACT_FP16, 3, 2048, 96, seed=7)
    y = oracle.reference_output(inp)
    y8 = oracle.reference_output(_as_lut8(inp))
    G = group or 2048
    s = np.asarray(inp.scales, dtype=np.float64).reshape(-1)
    smax = np.abs(s).max() * (1.0 if wfmt == W.WFMT_BINARY else 0.5)
    mult = oracle.token_pow2(inp.act)
    bound = mult[:, None] * (2048 // G) * smax * (G // 4) * ((1 << bits) - 1) * (2.0 / 127.0)
    assert np.all(np.abs(y8 - y) <= bound)
    rel = np.linalg.norm(y8 - y) / np.linalg.norm(y)
    assert 1e-4 < rel < 1e-2
    neg = _as_lut8(inp)
    neg.act = (-inp.act.astype(np.float32)).astype(np.float16)
    assert np.array_equal(oracle.reference_output(neg), -y8)


def _as_lut8(inp):
    import copy
    out = copy.copy(inp)
    out.act_kind = W.ACT_FP16_LUT8
    return out
