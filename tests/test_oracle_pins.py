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


def rne_binary32(x: Fraction) -> Fraction:
    """Exact rational x rounded to the nearest IEEE binary32 value, ties to even
    (24-bit significand, subnormals below 2^-126): the rounding IEEE 754 defines,
    computed with integers only, independently of any hardware FP arithmetic."""
    if x == 0:
        return Fraction(0)
    sign = -1 if x < 0 else 1
    a = abs(x)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1                                   # now 2^e <= a < 2^(e+1)
    ulp = Fraction(2) ** (max(e, -126) - 23)
    q = a / ulp
    n = q.numerator // q.denominator
    r = q - n
    if r > Fraction(1, 2) or (r == Fraction(1, 2) and n % 2 == 1):
        n += 1
    return sign * n * ulp


def test_rne_binary32_helper_matches_numpy_casts():
    """The helper above is itself checked against numpy's float64 -> float32 cast on
    values exactly representable in float64 (a single rounding there)."""
    rng = np.random.default_rng(40)
    vals = np.concatenate([rng.standard_normal(2000) * 10.0 ** rng.integers(-40, 30, 2000),
                           [1 + 2.0 ** -24, 1 + 3 * 2.0 ** -24, -(1 + 2.0 ** -24), 2.0 ** -149 * 1.5]])
    for v in vals:
        assert rne_binary32(Fraction(float(v))) == Fraction(float(np.float32(v)))


def test_int_output_exact_with_power_of_two_scales():
    """Power-of-two scales and |acc| < 2^24: both FP32 multiplies are exact, so
    y[i][c] must equal acc[i][c] * s_a[i] * s_w[c] exactly.  Distinct scales per row
    and per column pin the indexing (a row/column mix-up changes every value)."""
    rng = np.random.default_rng(41)
    acc = rng.integers(-(1 << 23), 1 << 23, size=(3, 5)).astype(np.int64)
    s_a = np.array([2.0 ** -3, 2.0 ** -7, 4.0], np.float32)
    s_w = np.array([2.0 ** -5, 0.5, 1.0, 8.0, 2.0 ** -10], np.float32)
    y = oracle.int_output_f32(acc, s_a, s_w)
    assert y.shape == (3, 5) and y.dtype == np.float32
    for i in range(3):
        for c in range(5):
            assert Fraction(float(y[i, c])) == int(acc[i, c]) * Fraction(float(s_a[i])) * Fraction(float(s_w[c]))
    # transposing the scale roles would give other values
    assert not np.array_equal(y, oracle.int_output_f32(acc, s_a[::-1].copy(), s_w[::-1].copy()))


def test_int_output_large_accumulators_round_on_conversion():
    """|acc| >= 2^24 is not exact in FP32: the conversion rounds to nearest, ties to
    even (2^24 + 1 -> 2^24, 2^24 + 3 -> 2^24 + 4, -(2^25 + 2) -> -2^25, and
    2^25 + 6 -> 2^25 + 8); with unit scales y is that rounded value."""
    acc = np.array([[(1 << 24) + 1, (1 << 24) + 3, -((1 << 25) + 2), (1 << 25) + 6,
                     (1 << 31) - 1]], dtype=np.int64)
    y = oracle.int_output_f32(acc, np.array([1.0], np.float32), np.ones(5, np.float32))
    expect = [1 << 24, (1 << 24) + 4, -(1 << 25), (1 << 25) + 8, 1 << 31]
    assert [int(v) for v in y[0]] == expect


def test_int_output_two_roundings_in_order():
    """Random accumulators and scales: y equals RNE32(RNE32(RNE32(acc) s_a) s_w)
    evaluated with exact rationals (the definition: two FP32 multiplies, the token
    scale first); the result lies within two binary32 roundings of the exact product;
    and the sample contains cases where the other association would differ, so the
    order is really pinned."""
    rng = np.random.default_rng(42)
    R, C = 6, 40
    acc = rng.integers(-(1 << 30), 1 << 30, size=(R, C)).astype(np.int64)
    acc[:, :10] = rng.integers(-5000, 5000, size=(R, 10))
    s_a = (rng.uniform(0.5, 1.0, R) * 2.0 ** rng.integers(-12, 2, R)).astype(np.float32)
    s_w = rng.uniform(0.01, 0.1, C).astype(np.float32)
    y = oracle.int_output_f32(acc, s_a, s_w)
    other_order = 0
    for i in range(R):
        for c in range(C):
            a, sa, sw = int(acc[i, c]), Fraction(float(s_a[i])), Fraction(float(s_w[c]))
            want = rne_binary32(rne_binary32(rne_binary32(Fraction(a)) * sa) * sw)
            assert Fraction(float(y[i, c])) == want
            exact = a * sa * sw
            assert abs(Fraction(float(y[i, c])) - exact) <= abs(exact) * Fraction(3, 1 << 24)
            if rne_binary32(rne_binary32(Fraction(a)) * rne_binary32(sa * sw)) != want:
                other_order += 1
    assert other_order > 0


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


# ----------------------------------------------------------------- INT8 table quantization (Section 3.1.3)

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


def _exact_codes(act_row_f16):
    """Codes and FP32 scales of the INT8-quantized half tables of one token, from the
    definition in exact rational arithmetic: T exact, q = round(127 T / amax) with
    ties to even (Python's round on a Fraction), scale = amax / 127 rounded to binary32,
    in the unit of the token normalized by its power of two."""
    x = [Fraction(float(v)) for v in act_row_f16.astype(np.float32)]
    amax_a = max(abs(v) for v in x)
    unit = Fraction(1)
    if amax_a != 0:
        _, e = np.frexp(float(amax_a))
        unit = Fraction(2) ** int(e)
    codes, scales = [], []
    for j in range(len(x) // 4):
        h = L.half_table([v / unit for v in x[4 * j:4 * j + 4]])
        tmax = max(abs(t) for t in h)
        if tmax == 0:
            codes.append([0] * 8)
            scales.append(Fraction(0))
            continue
        codes.append([round(127 * t / tmax) for t in h])
        scales.append(rne_binary32(tmax / 127))
    return codes, scales


def test_lut8_codes_round_half_even_exactly():
    """The table-quantized oracle's codes and scales equal the exact-rational definition
    on activations that mix magnitudes from FP16 subnormals to 6e4 (where an FP32 sum of
    the four terms would round), and on groups built so that 127 T / amax is a
    half-integer: (-31.25, 31.25, 31.25, 33.25) gives T = (-64.5, 2, -2, 64.5, -2, 64.5,
    60.5, 127), so ties to even give (-64, 2, -2, 64, -2, 64, 60, 127) where rounding
    half away from zero would give -65, 65, 61."""
    rng = np.random.default_rng(43)
    mags = 2.0 ** rng.integers(-24, 15, size=(3, 64))
    act = np.clip(rng.standard_normal((3, 64)) * mags, -6e4, 6e4).astype(np.float16)
    act[2, :8] = [-31.25, 31.25, 31.25, 33.25, 31.25, -31.25, -31.25, -33.25]
    act[2, 8:12] = [2.0 ** -24, 1024.0, -3.0 * 2.0 ** -20, 7.0]
    q, sc, mult = oracle.lut8_tables(act)
    for m in range(3):
        codes, scales = _exact_codes(act[m])
        assert q[m].tolist() == codes
        assert [Fraction(float(v)) for v in sc[m]] == scales
    assert q[2, 0].tolist() == [-64, 2, -2, 64, -2, 64, 60, 127]
    assert q[2, 1].tolist() == [64, -2, 2, -64, 2, -64, -60, -127]  # negated group: negated codes
