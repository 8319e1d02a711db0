"""Host-only checks of the C ABI: the library loads, exports every declared symbol,
and validates arguments before launching anything.  No GPU is touched: every call
here returns from host-side validation (size queries, invalid or unsupported
arguments), so these run in the CPU suite."""
import ctypes
import os
import re

import pytest

from helpers import tuning

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lutgemm.h")

L = pytest.importorskip("paper_2408_06003_amd")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lutgemm_[a-z_0-9]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 11
    for name in names:
        assert hasattr(L.lib, name), f"{name} declared in lutgemm.h but not exported"
    assert sorted(L.EXPORTS) == names


def test_header_constants_match_binding():
    """The tuning keys and size constants of lutgemm.h equal the binding's."""
    text = open(HEADER).read()
    keys = dict(re.findall(r"LUTGEMM_TUNE_([A-Z_0-9]+)\s*=\s*(\d+)", text))
    count = int(keys.pop("COUNT"))
    assert {k: int(v) for k, v in keys.items()} == L.TUNE
    assert count == len(L.TUNE)
    m = re.search(r"#define LUTGEMM_WORKSPACE_ZERO_BYTES \(\(size_t\)(\d+) << (\d+)\)", text)
    assert m and (int(m.group(1)) << int(m.group(2))) == L.WORKSPACE_ZERO_BYTES


def test_version_and_status_strings():
    assert "gfx950" in L.version()
    for s in range(5):
        assert L.status_string(s).startswith("LUTGEMM_")
    assert L.status_string(99) == "LUTGEMM_UNKNOWN_STATUS"


def test_problem_struct_layout():
    assert ctypes.sizeof(L.Problem) == 40


@pytest.mark.parametrize("K,N,b,wfmt,G,act,fp32,expect", [
    (4096, 4096, 2, L.WFMT_TERNARY, 0, L.ACT_INT8, True, L.SUCCESS),
    (1024, 1024, 2, L.WFMT_UINT, 128, L.ACT_FP16, False, L.SUCCESS),
    (11008, 4096, 4, L.WFMT_UINT, 128, L.ACT_FP16, False, L.SUCCESS),
    (8192, 28672, 1, L.WFMT_BINARY, 8192, L.ACT_FP16, False, L.SUCCESS),
    (8192, 100, 1, L.WFMT_BINARY, 8192, L.ACT_INT8, False, L.SUCCESS),
    (1000, 64, 2, L.WFMT_UINT, 0, L.ACT_FP16, False, L.ERROR_NOT_SUPPORTED),      # K % 128
    (1024, 64, 2, L.WFMT_UINT, 64, L.ACT_FP16, False, L.ERROR_NOT_SUPPORTED),     # G % 128
    (1024, 64, 2, L.WFMT_UINT, 384, L.ACT_FP16, False, L.ERROR_NOT_SUPPORTED),    # K % G
    (1024, 64, 3, L.WFMT_UINT, 128, L.ACT_FP16, False, L.ERROR_NOT_SUPPORTED),    # b = 3
    (1024, 64, 2, L.WFMT_BINARY, 128, L.ACT_FP16, False, L.ERROR_NOT_SUPPORTED),  # binary is 1 bit
    (1024, 64, 1, L.WFMT_TERNARY, 128, L.ACT_FP16, False, L.ERROR_NOT_SUPPORTED), # ternary is 2 bits
    (1024, 64, 2, L.WFMT_UINT, 0, L.ACT_FP16, True, L.ERROR_NOT_SUPPORTED),       # fp32 scale needs no zero
    (1024, 64, 2, L.WFMT_TERNARY, 128, L.ACT_FP16, True, L.ERROR_NOT_SUPPORTED),  # fp32 scale per-tensor only
    (1024, 64, 2, L.WFMT_UINT, 128, L.ACT_INT8, False, L.ERROR_NOT_SUPPORTED),    # INT8 act needs int weights
    (1024, 64, 2, L.WFMT_TERNARY, 128, L.ACT_INT8, False, L.ERROR_NOT_SUPPORTED), # INT8 act: per-channel at most
    (4096, 4096, 2, L.WFMT_TERNARY_3IN5, 0, L.ACT_INT8, True, L.SUCCESS),
    (4096, 4096, 2, L.WFMT_TERNARY_3IN5, 0, L.ACT_FP16, False, L.SUCCESS),
    (11008, 300, 2, L.WFMT_TERNARY_3IN5, 11008, L.ACT_FP16, False, L.SUCCESS),
    (1024, 64, 2, L.WFMT_TERNARY_3IN5, 128, L.ACT_FP16, False, L.ERROR_NOT_SUPPORTED),  # 3-in-5: G = 0 or K
    (4096, 4096, 4, L.WFMT_UINT, 128, L.ACT_FP16_LUT8, False, L.SUCCESS),
    (8192, 1000, 1, L.WFMT_BINARY, 8192, L.ACT_FP16_LUT8, False, L.SUCCESS),
    (4096, 64, 2, L.WFMT_TERNARY, 0, L.ACT_FP16_LUT8, True, L.SUCCESS),
    (4096, 64, 2, L.WFMT_TERNARY_3IN5, 0, L.ACT_FP16_LUT8, True, L.ERROR_NOT_SUPPORTED),  # no 3-in-5 LUT8
    (1024, 64, 1, L.WFMT_TERNARY_3IN5, 0, L.ACT_FP16, False, L.ERROR_NOT_SUPPORTED),    # 3-in-5 is ternary
    (0, 64, 2, L.WFMT_UINT, 0, L.ACT_FP16, False, L.ERROR_INVALID_VALUE),
    (1024, 0, 2, L.WFMT_UINT, 0, L.ACT_FP16, False, L.ERROR_INVALID_VALUE),
    (1024, 64, 2, 7, 0, L.ACT_FP16, False, L.ERROR_INVALID_VALUE),
    (1024, 64, 2, L.WFMT_UINT, 0, 5, False, L.ERROR_INVALID_VALUE),
    (1024, 64, 0, L.WFMT_UINT, 0, L.ACT_FP16, False, L.ERROR_INVALID_VALUE),
    (1024, 64, 2, L.WFMT_UINT, -128, L.ACT_FP16, False, L.ERROR_INVALID_VALUE),
])
def test_validate(K, N, b, wfmt, G, act, fp32, expect):
    p = L.problem(K, N, b, wfmt, G, act, fp32)
    assert L.validate(p, 1) == expect
    if expect == L.SUCCESS:
        assert L.packed_weight_size(p) > 0 and L.table_size(p, 3) > 0
    else:
        assert L.packed_weight_size(p) == 0 and L.table_size(p, 1) == 0 and L.workspace_size(p, 1) == 0


def test_validate_m_and_reserved():
    p = L.problem(1024, 64, 2, L.WFMT_UINT, 128)
    assert L.validate(p, 0) == L.ERROR_INVALID_VALUE
    assert L.validate(p, -3) == L.ERROR_INVALID_VALUE
    assert L.validate(p, 1 << 20) == L.ERROR_NOT_SUPPORTED
    p.reserved = 1
    assert L.validate(p, 1) == L.ERROR_INVALID_VALUE
    assert L.lib.lutgemm_validate(None, 1) == L.ERROR_INVALID_VALUE


def test_size_formulas():
    """Eq. 7-8 read as storage sizes: tables are 2^(4-1) entries of 16 bits per 4 activations
    and token; grouped binary weights are K x N x b bits (plus alignment of N and metadata)."""
    M, K, N = 3, 4096, 1000
    p = L.problem(K, N, 4, L.WFMT_UINT, 128)
    s_off, t_off = L.table_offsets(p, M)
    assert s_off >= M * (K // 4) * 8 * 2 and s_off % 256 == 0
    assert t_off >= s_off + M * (K // 128) * 4 and t_off % 256 == 0
    assert L.table_size(p, M) >= t_off + 4 * M
    n_pad = 1024
    planes = K * n_pad * 4 // 8
    # planes, (s, z) per group and column, and one fixed-point exponent per column
    assert planes <= L.packed_weight_size(p) <= planes + (K // 128) * n_pad * 4 + n_pad * 4 + 512


def test_size_formulas_ternary_3in5():
    """3-in-5 ternary: 5 bits per 3 weights (16 index bytes + 4 sign bytes per 96 weights of a
    column, K padded to 96); tables of 16 two-byte entries per triple and token."""
    M, K, N = 2, 4096, 1000
    p = L.problem(K, N, 2, L.WFMT_TERNARY_3IN5, 0, L.ACT_INT8, True)
    kb3, n_pad = -(-K // 96), 1024
    body = kb3 * n_pad * 20
    assert body <= L.packed_weight_size(p) <= body + 3 * 256
    assert L.packed_weight_size(p) < K * n_pad * 2 // 8  # smaller than the 2-bit planes
    s_off, t_off = L.table_offsets(p, M)
    assert s_off >= M * kb3 * 32 * 16 * 2 and s_off % 256 == 0
    assert L.table_size(p, M) >= t_off + 4 * M
    assert L.workspace_size(p, M) == 0 and L.fused_workspace_size(p, M) == 0
    # grid limit: ceil(N / 16) * M workgroups below 2^24
    big = L.problem(1024, 1 << 16, 2, L.WFMT_TERNARY_3IN5, 0, L.ACT_FP16)
    assert L.validate(big, 4095) == L.SUCCESS
    assert L.validate(big, 4096) == L.ERROR_NOT_SUPPORTED


def test_size_formulas_int8_table_quantization():
    """INT8 table quantization (Section 3.1.3): 8 one-byte codes and one FP32 scale per 4
    activations and token, i.e. 12 bytes against 16 for FP16 tables."""
    M, K, N = 5, 4096, 300
    p = L.problem(K, N, 2, L.WFMT_UINT, 128, L.ACT_FP16_LUT8)
    q = L.problem(K, N, 2, L.WFMT_UINT, 128, L.ACT_FP16)
    s_off, t_off = L.table_offsets(p, M)
    assert s_off >= M * (K // 4) * 12 and s_off % 256 == 0
    assert s_off < L.table_offsets(q, M)[0]
    assert t_off >= s_off + M * (K // 128) * 4
    assert L.table_size(p, M) < L.table_size(q, M)
    assert L.packed_weight_size(p) == L.packed_weight_size(q)


def test_entry_points_reject_before_launch():
    """Invalid pointers / sizes are rejected on the host; nothing reaches the GPU."""
    p = L.problem(1024, 256, 2, L.WFMT_UINT, 128)
    ok = 1 << 20  # an aligned fake address, never dereferenced because validation fails first
    f = L.lib
    bp = ctypes.byref(p)
    big = 1 << 40
    # null pointers
    assert f.lutgemm_pack_weights(bp, None, ok, ok, ok, big, None) == L.ERROR_INVALID_VALUE
    assert f.lutgemm_pack_weights(bp, ok, ok, None, ok, big, None) == L.ERROR_INVALID_VALUE  # UINT needs zeros
    assert f.lutgemm_precompute(bp, 1, None, ok, big, None) == L.ERROR_INVALID_VALUE
    assert f.lutgemm_mpgemm(bp, 1, ok, ok, None, L.OUT_FP16, 0, ok, big, None) == L.ERROR_INVALID_VALUE
    # misaligned pointers
    assert f.lutgemm_pack_weights(bp, ok + 4, ok, ok, ok, big, None) == L.ERROR_INVALID_VALUE
    assert f.lutgemm_precompute(bp, 1, ok, ok + 8, big, None) == L.ERROR_INVALID_VALUE
    assert f.lutgemm_mpgemm_dequant(bp, 1, ok + 2, ok, ok, L.OUT_FP16, 0, None, 0, None) == L.ERROR_INVALID_VALUE
    # too-small buffers
    assert f.lutgemm_pack_weights(bp, ok, ok, ok, ok, 16, None) == L.ERROR_INSUFFICIENT_SIZE
    assert f.lutgemm_precompute(bp, 1, ok, ok, 16, None) == L.ERROR_INSUFFICIENT_SIZE
    # bad enums / unsupported output
    assert f.lutgemm_mpgemm(bp, 1, ok, ok, ok, 9, 0, ok, big, None) == L.ERROR_INVALID_VALUE
    assert f.lutgemm_mpgemm(bp, 1, ok, ok, ok, L.OUT_INT32, 0, ok, big, None) == L.ERROR_NOT_SUPPORTED
    assert f.lutgemm_mpgemm(bp, 1, ok, ok, ok, L.OUT_FP16, 2, ok, big, None) == L.ERROR_INVALID_VALUE
    assert f.lutgemm_mpgemm_dequant(bp, 1, ok, ok, ok, L.OUT_INT32, 0, None, 0, None) == L.ERROR_INVALID_VALUE
    pi = L.problem(1024, 256, 2, L.WFMT_TERNARY, 0, L.ACT_INT8, True)
    assert f.lutgemm_mpgemm_dequant(ctypes.byref(pi), 1, ok, ok, ok, L.OUT_FP16, 0, None, 0, None) == L.ERROR_NOT_SUPPORTED
    # workspace required but missing / too small
    pw = L.problem(8192, 1024, 2, L.WFMT_TERNARY, 0, L.ACT_INT8, True)  # too few columns: K is split
    need = L.workspace_size(pw, 1)
    assert need > 0
    assert f.lutgemm_mpgemm(ctypes.byref(pw), 1, ok, ok, ok, L.OUT_INT32, 0, None, need, None) == L.ERROR_INVALID_VALUE
    assert f.lutgemm_mpgemm(ctypes.byref(pw), 1, ok, ok, ok, L.OUT_INT32, 0, ok, need - 1, None) == L.ERROR_INSUFFICIENT_SIZE
    # comparison path: a few tokens on few columns split K (FP32 partials per split)
    pd = L.problem(8192, 1024, 1, L.WFMT_BINARY, 0)
    need = L.dequant_workspace_size(pd, 16)
    assert need > 0 and need % (16 * 1024 * 4) == 0
    assert f.lutgemm_mpgemm_dequant(ctypes.byref(pd), 16, ok, ok, ok, L.OUT_FP16, 0, None, need, None) == L.ERROR_INVALID_VALUE
    assert f.lutgemm_mpgemm_dequant(ctypes.byref(pd), 16, ok, ok, ok, L.OUT_FP16, 0, ok, need - 1, None) == L.ERROR_INSUFFICIENT_SIZE
    # large M on a wide layer: whole K per workgroup, no scratch; unsupported problems report 0
    assert L.dequant_workspace_size(L.problem(4096, 16384, 2, L.WFMT_UINT, 128), 4096) == 0
    assert L.dequant_workspace_size(pi, 16) == 0
    # launch plans: 16-token slabs for few tokens of 1-bit weights, 256 x 256 tiles at
    # large M (K split only while the grid stays within one round of 256 workgroups)
    assert L.dequant_plan(pd, 16)[0] == 2
    assert L.dequant_plan(L.problem(4096, 4096, 2, L.WFMT_UINT, 128), 4096) == (1, 1)
    assert L.dequant_plan(L.problem(8192, 28672, 1, L.WFMT_BINARY, 8192), 256) == (1, 2)
    assert L.dequant_plan(L.problem(28672, 8192, 1, L.WFMT_BINARY, 28672), 256) == (1, 8)
    assert f.lutgemm_dequant_plan(ctypes.byref(pi), 16, None, None) == L.ERROR_NOT_SUPPORTED


def test_fused_entry_point_rejects_before_launch():
    f = L.lib
    ok, big = 1 << 20, 1 << 40
    p = L.problem(4096, 4096, 2, L.WFMT_TERNARY, 0, L.ACT_INT8, True)
    bp = ctypes.byref(p)
    assert L.fused_workspace_size(p, 1) == 0           # one token, whole K per workgroup: no scratch
    assert f.lutgemm_mpgemm_fused(bp, 1, None, ok, ok, L.OUT_INT32, 0, None, 0, None) == L.ERROR_INVALID_VALUE
    assert f.lutgemm_mpgemm_fused(bp, 1, ok + 4, ok, ok, L.OUT_INT32, 0, None, 0, None) == L.ERROR_INVALID_VALUE
    assert f.lutgemm_mpgemm_fused(bp, 1, ok, ok, ok, 7, 0, None, 0, None) == L.ERROR_INVALID_VALUE
    assert f.lutgemm_mpgemm_fused(bp, 1, ok, ok, ok, L.OUT_INT32, 3, None, 0, None) == L.ERROR_INVALID_VALUE
    assert f.lutgemm_mpgemm_fused(bp, 0, ok, ok, ok, L.OUT_INT32, 0, None, 0, None) == L.ERROR_INVALID_VALUE
    pf = L.problem(1024, 256, 2, L.WFMT_UINT, 128)
    assert f.lutgemm_mpgemm_fused(ctypes.byref(pf), 1, ok, ok, ok, L.OUT_INT32, 0, None, 0, None) == L.ERROR_NOT_SUPPORTED
    # whole-K kernel with K split across workgroups (4 column tiles are too few for the
    # split-K kernel): the zero region, partial sums and per-token factors
    ps = L.problem(8192, 1000, 2, L.WFMT_TERNARY, 0, L.ACT_INT8, True)
    need = L.fused_workspace_size(ps, 1)
    assert need >= L.WORKSPACE_ZERO_BYTES + 2 * 1024 * 4 + 4
    assert f.lutgemm_mpgemm_fused(ctypes.byref(ps), 1, ok, ok, ok, L.OUT_FP32, 0, None, need, None) == L.ERROR_INVALID_VALUE
    assert f.lutgemm_mpgemm_fused(ctypes.byref(ps), 1, ok, ok, ok, L.OUT_FP32, 0, ok, need - 1, None) == L.ERROR_INSUFFICIENT_SIZE
    # several tokens: tables (lutgemm_table_size) plus the table-fed kernel's workspace
    M = 8
    assert L.fused_workspace_size(p, M) >= L.table_size(p, M) + L.workspace_size(p, M)
    assert L.fused_workspace_size(L.problem(1000, 64, 2, L.WFMT_UINT, 0), 1) == 0  # invalid problem


def test_fused_multi_token_plan():
    """lutgemm_mpgemm_fused with FP16 activations and M > 2: the multi-token kernel
    builds its own tables (scratch: the partial sums only) for M <= 64 on layers of at
    most 64 x 256 columns, else precompute + mpGEMM (scratch: tables too); the tuning
    key forces either; zero-point formats keep K ranges within 64 blocks."""
    def tables_in_scratch(p, M):  # the two-call layout: [workspace, 256-aligned][tables]
        ws = L.workspace_size(p, M)
        return L.fused_workspace_size(p, M) == (ws + 255) // 256 * 256 + L.table_size(p, M)
    small = L.problem(4096, 12288, 4, L.WFMT_UINT, 128)    # 48 column tiles
    wide = L.problem(8192, 28672, 1, L.WFMT_BINARY, 8192)   # 112 column tiles
    assert not tables_in_scratch(small, 8) and not tables_in_scratch(small, 64)
    assert tables_in_scratch(small, 65) and tables_in_scratch(wide, 16)
    assert L.fused_workspace_size(small, 8) == L.workspace_size(small, 8)
    old = L.get_tuning("MT_FUSED")
    try:
        L.set_tuning("MT_FUSED", 1)
        assert not tables_in_scratch(wide, 16) and not tables_in_scratch(small, 300)
        L.set_tuning("MT_FUSED", 0)
        assert tables_in_scratch(small, 8)
        # INT4 K = 11008 (86 blocks), no split planned for the table-fed kernel at M = 2048:
        # the fused build splits K so that every range holds at most 64 blocks
        L.set_tuning("MT_FUSED", 1)
        k = L.problem(11008, 4096, 4, L.WFMT_UINT, 128)
        assert L.fused_workspace_size(k, 2048) > 0 and L.workspace_size(k, 2048) == 0
    finally:
        L.set_tuning("MT_FUSED", old)
    # INT8 activations with several tokens always take the two-call path
    pi = L.problem(4096, 4096, 2, L.WFMT_TERNARY, 0, L.ACT_INT8, True)
    assert tables_in_scratch(pi, 8)


def test_tuning_overrides():
    """Planner overrides go through lutgemm_set_tuning (no entry point reads the
    environment per call): unknown keys and out-of-range values are rejected, -1
    restores the default, and a forced value changes the planned workspace."""
    assert L.lib.lutgemm_get_tuning(-1) == -2 and L.lib.lutgemm_get_tuning(99) == -2
    assert L.lib.lutgemm_set_tuning(99, 1) == L.ERROR_INVALID_VALUE
    assert L.lib.lutgemm_set_tuning(L.TUNE["KBS"], -2) == L.ERROR_INVALID_VALUE
    assert L.lib.lutgemm_set_tuning(L.TUNE["TARGET_BLOCKS"], 0) == L.ERROR_INVALID_VALUE
    old = L.get_tuning("GEMV_KIND")
    p = L.problem(4096, 4096, 2, L.WFMT_UINT, 128)
    ws = L.workspace_size(p, 1)
    assert ws == L.WORKSPACE_ZERO_BYTES  # planned: split-K GEMV, exact completion
    try:
        L.set_tuning("GEMV_KIND", 0)   # the whole-K kernel: 256 column tiles, no K split
        assert L.get_tuning("GEMV_KIND") == 0
        assert L.workspace_size(p, 1) == 0
        L.set_tuning("GEMV_KIND", -1)
        assert L.get_tuning("GEMV_KIND") == -1
        assert L.workspace_size(p, 1) == ws
        with tuning(SPLIT_EXACT=0):  # split-K GEMV with the arrival protocol: partial sums
            assert L.workspace_size(L.problem(8192, 28672, 1, L.WFMT_BINARY, 8192), 1) > ws
    finally:
        L.set_tuning("GEMV_KIND", old)
