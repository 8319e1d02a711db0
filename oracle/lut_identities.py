"""Exact-rational model of the paper's LUT reformulation -- TEST INFRASTRUCTURE ONLY.

Each function follows one step of LUT Tensor Core, Section 3.1 (software table
optimizations), in the paper's order and notation, on Python ``Fraction`` values
so every identity can be checked exactly.  Only the tests use it, to pin the
dense float64/int64 oracle: for tiny inputs, the LUT evaluation below must equal
the oracle's direct dot product exactly.

Conventions (readings of the paper):
* g = 4 activations per table (the paper's dot-product length "K = 4").
* Pattern bits are written MSB first, W_3 W_2 W_1 W_0, and W_3 belongs to the
  first activation of the group (as in the worked example of Section 3.1.2,
  where W_3 = 0 pairs with A).
* In the reinterpretation formula (Eq. 2) the exponent "K" is the weight bit
  width b.
"""
from __future__ import annotations

from fractions import Fraction
from typing import List, Sequence, Tuple

G4 = 4  # activations per table


def reinterpret(q: int, s: Fraction, z: Fraction, b: int) -> Tuple[int, Fraction, Fraction]:
    """Eq. 2: q' = 2q - (2^b - 1), s' = s / 2, z' = 2z + 1 - 2^b."""
    return 2 * q - ((1 << b) - 1), Fraction(s) / 2, 2 * Fraction(z) + 1 - (1 << b)


def dequant(q: int, s: Fraction, z: Fraction) -> Fraction:
    """Eq. 1: r = s (q - z)."""
    return Fraction(s) * (q - Fraction(z))


def pattern_sign(p: int, i: int) -> int:
    """Bit of activation i in pattern p (MSB = activation 0), read as -1 / +1."""
    return 1 if (p >> (G4 - 1 - i)) & 1 else -1


def full_table(acts: Sequence[Fraction]) -> List[Fraction]:
    """Table over all 2^4 one-bit patterns: LUT[p] = sum_i a_i * (+-1)  (Section 3.1, Fig. 3 with {0,1} -> {-1,+1})."""
    assert len(acts) == G4
    return [sum((Fraction(acts[i]) * pattern_sign(p, i) for i in range(G4)), Fraction(0))
            for p in range(1 << G4)]


def half_table(acts: Sequence[Fraction]) -> List[Fraction]:
    """Symmetrized table: the 2^(4-1) entries whose MSB is 0 (Eq. 5, W_3 = 0 branch)."""
    lut = full_table(acts)
    return [lut[idx] for idx in range(1 << (G4 - 1))]


def lookup_eq5(half: Sequence[Fraction], p: int) -> Fraction:
    """Eq. 5: LUT[p] = -T[~(W_2 W_1 W_0)] if W_3 = 1 else T[W_2 W_1 W_0]."""
    low = p & 0b111
    if (p >> 3) & 1:
        return -half[(~low) & 0b111]
    return half[low]


def offline_negate(p: int) -> Tuple[int, int]:
    """Eq. 6 storage form: keep the MSB as the sign and store the low bits inverted when it is set."""
    sign = (p >> 3) & 1
    idx = ((~p) & 0b111) if sign else (p & 0b111)
    return sign, idx


def lookup_eq6(half: Sequence[Fraction], sign: int, idx: int) -> Fraction:
    """Eq. 6: LUT[W_3' W_2' W_1' W_0'] = -T[W_2' W_1' W_0'] if W_3' = 1 else T[...]."""
    return -half[idx] if sign else half[idx]


def bit_planes(q: int, b: int) -> List[int]:
    """Bit-serial decomposition (Section 3.1): plane t holds bit t of the code."""
    return [(q >> t) & 1 for t in range(b)]


def plane_pattern(codes4: Sequence[int], t: int) -> int:
    """4-bit pattern of bit-plane t over one group of 4 codes, MSB = first code."""
    p = 0
    for i in range(G4):
        p = (p << 1) | ((codes4[i] >> t) & 1)
    return p


def lut_group_dot(acts: Sequence[Fraction], codes: Sequence[int], s: Fraction, z: Fraction,
                  b: int) -> Fraction:
    """Dot product of one quantization group by table lookup (Eq. 3 with Eq. 2, 5, 6).

    sum_k a_k s (q_k - z) = s' ( sum_t 2^t sum_j LUT_j[pattern_{t,j}] - z' sum_k a_k ),
    since sum_t 2^t (2 bit_t(q) - 1) = 2q - (2^b - 1) = q' for every code q.
    """
    assert len(acts) == len(codes) and len(acts) % G4 == 0
    _, s_p, z_p = reinterpret(0, s, z, b)
    acc = Fraction(0)
    for j in range(len(acts) // G4):
        a4 = [Fraction(x) for x in acts[G4 * j:G4 * j + G4]]
        half = half_table(a4)
        c4 = codes[G4 * j:G4 * j + G4]
        for t in range(b):
            sign, idx = offline_negate(plane_pattern(c4, t))
            acc += (1 << t) * lookup_eq6(half, sign, idx)
    S = sum((Fraction(x) for x in acts), Fraction(0))
    return s_p * (acc - z_p * S)


def lut_mpgemm(A: Sequence[Sequence[Fraction]], codes: Sequence[Sequence[int]],
               scales: Sequence[Sequence[Fraction]], zeros: Sequence[Sequence[Fraction]],
               b: int, group: int) -> List[List[Fraction]]:
    """Whole mpGEMM y = A x dequant(W)^T evaluated group by group through the tables."""
    M = len(A)
    N = len(codes)
    K = len(A[0])
    y = [[Fraction(0)] * N for _ in range(M)]
    for m in range(M):
        for n in range(N):
            tot = Fraction(0)
            for q in range(K // group):
                sl = slice(q * group, (q + 1) * group)
                tot += lut_group_dot(A[m][sl], codes[n][sl], scales[n][q], zeros[n][q], b)
            y[m][n] = tot
    return y


def ternary_int_dot(qa: Sequence[int], w: Sequence[int]) -> Tuple[int, int]:
    """Integer LUT evaluation for ternary weights w in {-1,0,1} stored as 2-bit codes q = w + 1.

    Returns (numerator, result) where numerator = sum_t 2^t L_t + S and result =
    numerator / 2; with z = 1, b = 2 the reinterpreted zero is z' = -1 (Eq. 2).
    """
    codes = [x + 1 for x in w]
    acc = 0
    for j in range(len(qa) // G4):
        a4 = [Fraction(x) for x in qa[G4 * j:G4 * j + G4]]
        half = half_table(a4)
        for t in range(2):
            sign, idx = offline_negate(plane_pattern(codes[G4 * j:G4 * j + G4], t))
            v = lookup_eq6(half, sign, idx)
            assert v.denominator == 1
            acc += (1 << t) * int(v)
    numer = acc + sum(qa)
    return numer, numer // 2
