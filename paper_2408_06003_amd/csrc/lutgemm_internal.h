// Internal definitions shared by the host library and the HIP kernels.
//
// Packed-weight layout (opaque to callers, owned by this library):
//   planes: [KB][b][N_pad] x 16 bytes, KB = K/128.  One 16-byte word holds the
//           32 four-bit table indices of one bit-plane of one column over 128
//           consecutive k (4-bit index i covers k = 128 kb + 4 i .. + 3, stored
//           at bits 4(i % 8) of 32-bit word i / 8).  An index is the pattern of
//           the plane's bits over those 4 weights, first weight as MSB, with the
//           low 3 bits inverted when the MSB is set (Eq. 6): bit 3 = sign,
//           bits 0-2 = half-table row.  Columns n >= N are zero words.
//   meta:   per-group scales: [Q][N_pad] x (FP16 s, FP16 z) pairs (z = 0 unless
//           UINT); per-tensor: two FP32 values (s, z).  Stored as given; the
//           reinterpretation of Eq. 2 is applied in FP32 where they are used.
// Consecutive columns are adjacent in memory so that a wavefront whose lanes are
// 64 consecutive columns reads 1 KiB contiguous with 128-bit loads.
//
// Ternary 3-in-5 layout (LUTGEMM_WFMT_TERNARY_3IN5): K is covered by KB3 =
// ceil(K/96) blocks of 32 triples of consecutive weights (weights past K are 0).
// A triple (w0, w1, w2) is the base-3 value v = 9(w0+1) + 3(w1+1) + (w2+1) in
// [0, 27); negation maps v to 26 - v and v = 13 is the zero triple, so the code
// is sign = (v < 13) and index i = |v - 13| in [0, 14): the entry of pattern
// 13 + i, negated when sign is set (the symmetry of Eq. 4 for three-valued
// weights: 5 bits per 3 weights).
//   index words: [KB3][N_pad] x 16 bytes, index of triple t at bits 4(t % 8) of
//                32-bit word t / 8 (the plane-word arrangement above);
//   sign words:  [KB3][N_pad] x 4 bytes, sign of triple t = 8d + 2k + h (d = word,
//                k = byte, h = nibble) at bit 8k + 2d + h;
//   meta:        as above, with G = K (per-channel) or per-tensor.
// 20 bytes per 96 weights of a column: 1.67 bits per weight.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "lutgemm.h"

namespace lutgemm {

constexpr int KBLK = 128;       // activations covered by one packed plane word
constexpr int GPB = 32;         // 4-activation table groups per plane word
constexpr int NTILE = 256;      // columns per workgroup (one column per lane)
constexpr int FIX_SHIFT = 20;   // fixed-point fraction bits of FP table entries staged in LDS
constexpr int FIN_BATCH = 64;   // split partial sums the finalize kernel requests at once per output
constexpr int TBLK = 96;        // activations per 3-in-5 block (32 triples)
constexpr int TPB = 32;         // triples per 3-in-5 block
constexpr int TENT = 16;        // stored entries per triple table (14 used, 2 zero)
// Every workspace that is needed at all starts with this many bytes that are zero
// between calls (touched only by the split-K GEMV, which re-arms what it uses): the
// 32-bit arrival counters in the first CNT_BYTES, then the 64-bit exact split-sum
// words; partial sums and staged tables always come after it, so no call can leave
// a nonzero value where a later call, of any problem, expects a zero.
constexpr size_t CNT_AREA = LUTGEMM_WORKSPACE_ZERO_BYTES;
constexpr size_t CNT_BYTES = 65536;
constexpr int64_t CNT_MAX = (int64_t)(CNT_BYTES / 4);
constexpr int64_t EXACT_MAX = (int64_t)((CNT_AREA - CNT_BYTES) / 8);  // exact split-sum words
// Exact split completion: a split-sum word holds (arrivals) 2^57 + V with |V| < 2^56,
// so at most 127 splits; FP partial sums are fixed point in units of 2^E with E
// chosen per column so that the column's partial sums stay below 2^BND_BITS.
constexpr int EXACT_MAX_SPLITS = 127;
constexpr int BND_BITS = 54;
// Largest K split the split-K GEMV completes inside the kernel (one batch of partial
// loads by the last workgroup); longer splits are summed by the finalize kernel.
constexpr int INKERNEL_MAX_SPLITS = 32;
// Multi-token kernel with the table build fused in, for formats with zero points: the
// per-128-block activation sums of a workgroup's K range stay in LDS, so a K range
// holds at most this many blocks (the planner splits K further when it would not).
constexpr int MTOK_FUSED_SMAX = 64;

struct Layout {
    int64_t K, N, N_pad, KB, J, Q, G;  // G = group size (K when per-tensor)
    int bits, wfmt, act;
    bool per_tensor;
    bool tri;                          // ternary 3-in-5: KB counts 96-blocks, J triples
    size_t planes_bytes, sgn_off, meta_off, meta_bytes, bnd_off, packed_bytes;
};

// Eq. 2 reinterpretation constants of a weight format: s' = cs s, z' = cz z + c0.
inline void format_consts(int wfmt, int bits, float &cs, float &cz, float &c0) {
    if (wfmt == LUTGEMM_WFMT_BINARY) {  // codes {0,1} read as {-1,+1}: s' = s, z' = 0
        cs = 1.f;
        cz = 0.f;
        c0 = 0.f;
    } else if (wfmt == LUTGEMM_WFMT_TERNARY) {  // q = w + 1, z = 1, b = 2: s' = s/2, z' = -1
        cs = 0.5f;
        cz = 0.f;
        c0 = -1.f;
    } else {  // Eq. 2: s' = s/2, z' = 2z + 1 - 2^b
        cs = 0.5f;
        cz = 2.f;
        c0 = 1.f - (float)(1 << bits);
    }
}

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

inline Layout make_layout(const lutgemm_problem_t &p) {
    Layout L{};
    L.K = p.K;
    L.N = p.N;
    L.N_pad = (p.N + NTILE - 1) / NTILE * NTILE;
    L.KB = p.K / KBLK;
    L.J = p.K / 4;
    L.per_tensor = p.group_size == 0;
    L.G = p.group_size ? p.group_size : p.K;
    L.Q = p.group_size ? p.K / p.group_size : 1;
    L.bits = p.w_bits;
    L.wfmt = p.wfmt;
    L.act = p.act;
    L.tri = p.wfmt == LUTGEMM_WFMT_TERNARY_3IN5;
    if (L.tri) {
        L.KB = (p.K + TBLK - 1) / TBLK;
        L.J = L.KB * TPB;
        L.planes_bytes = (size_t)L.KB * L.N_pad * 16;
        L.sgn_off = align256(L.planes_bytes);
        L.meta_off = align256(L.sgn_off + (size_t)L.KB * L.N_pad * 4);
    } else {
        L.planes_bytes = (size_t)L.KB * L.bits * L.N_pad * 16;
        L.sgn_off = 0;
        L.meta_off = align256(L.planes_bytes);
    }
    L.meta_bytes = L.per_tensor ? 256 : (size_t)L.Q * L.N_pad * 4;
    // per column: the fixed-point exponent of the exact K-split completion (INT32;
    // not kept for 3-in-5 weights, whose kernel never splits K)
    L.bnd_off = L.meta_off + align256(L.meta_bytes);
    L.packed_bytes = L.bnd_off + (L.tri ? 0 : align256((size_t)L.N_pad * 4));
    return L;
}

struct TableLayout {
    size_t t_bytes, sc_off, s_off, tok_off, total;  // sc_off: INT8-quantized tables' scales
};

inline TableLayout make_table_layout(const Layout &L, int64_t M) {
    TableLayout T{};
    if (L.act == LUTGEMM_ACT_FP16_LUT8) {  // [M][J] x 8 INT8 codes, then [M][J] FP32 scales
        T.t_bytes = (size_t)M * L.J * 8;
        T.sc_off = align256(T.t_bytes);
        T.s_off = align256(T.sc_off + (size_t)M * L.J * 4);
    } else {
        T.t_bytes = (size_t)M * L.J * (L.tri ? 2 * TENT : 16);
        T.sc_off = 0;
        T.s_off = align256(T.t_bytes);
    }
    T.tok_off = align256(T.s_off + (size_t)M * L.Q * 4);
    T.total = align256(T.tok_off + (size_t)M * 4);
    return T;
}

// Launch plan of the LUT mpGEMM for (problem, M).
struct LutPlan {
    int kind;        // 0: single-token whole-K GEMV, 1: multi-token kernel, 2: single-token split-K GEMV,
                     // 3: ternary 3-in-5 kernel (whole K, any M)
    int gemv_cfg;    // single-token kernel: lane decomposition (see lut_gemv.hip)
    int kbs;         // 128-blocks of K per split
    int pre;         // split-K GEMV: weight words per lane requested before the tables are waited for
    bool inkernel;   // split-K GEMV: the K split is completed in the kernel (else by the finalize kernel)
    bool exact;      // split-K GEMV: ... by one 64-bit atomic per output on exact integer partials
    int splits;      // K splits (1 = no workspace)
    int mt;          // tokens per workgroup (multi-token kernel)
    int64_t m_tiles; // token tiles
    int64_t n_tiles; // column tiles
    int order;       // multi-token kernel: workgroup order (0: columns fastest; 1: tokens fastest
                     // per XCD; g >= 2: per XCD, bands of g token tiles, tokens fastest in a band)
    size_t ws_bytes;
    size_t part_off;  // byte offset of the split partial sums in the workspace (counters at 0)
};

// fused: the plan of lutgemm_mpgemm_fused (the multi-token kernel that builds its tables
// from the activations keeps a K range within MTOK_FUSED_SMAX blocks for zero-point formats)
LutPlan plan_lut(const Layout &L, int64_t M, bool fused = false);

// Current value of planner override `key` (LUTGEMM_TUNE_*, see lutgemm_set_tuning).
int tuning(int key);

// Text returned by lutgemm_last_error for the calling thread.
void set_last_error(const char *msg);
// LUTGEMM_ERROR_HIP with the HIP error's text recorded for lutgemm_last_error.
lutgemm_status_t hip_error(int e);

// Kernel parameter blocks.
struct PackParams {
    const void *codes;
    const void *scales;
    const void *zeros;
    uint4 *planes;
    uint32_t *sgn;         // 3-in-5 sign words
    void *meta;
    int *bnd;              // per-column fixed-point exponent of the exact split completion
    int64_t K, N, N_pad, KB, Q, G;
    int bits, wfmt, per_tensor, scale_fp32;
};

struct PrecomputeParams {
    const uint16_t *act;   // FP16 bits [M][K]
    uint4 *T;              // [M][J] x 8 entries
    void *S;               // [M][Q]
    float *tok;            // [M]
    int64_t M, K, J, Q, G;
    int tri;               // ternary 3-in-5 tables: [M][J triples] x 16 entries, no S
    float *tsc;            // INT8 table quantization: per-table scales [M][J] (T holds [M][J] x 8 INT8)
    int vbs;               // blocks of 256 table groups per workgroup (set by the launcher)
};

struct LutParams {
    const uint4 *T;        // half tables (INT8 table quantization: [M][J] x 8 INT8 codes)
    const float *tsc;      // INT8 table quantization: per-table scales [M][J], else NULL
    const void *S;         // group sums
    const float *tok;      // per-token factor (NULL in the fused kernel, which computes it)
    const uint16_t *act;   // FP16 [M][K]: activations of the fused kernel
    float *tok_out;        // fused kernel with K split: per-token factor for the finalize kernel
    const uint4 *planes;
    const uint32_t *sgn;   // 3-in-5 sign words
    const void *meta;
    void *out;
    unsigned long long *tl; // instrumented builds: per-wavefront phase stamps (see lut_common.h), else NULL
    float *part;           // split partial sums [splits][rows][N_pad] (float or int bits)
    uint32_t *cnt;         // split-K GEMV: arrival counters [M][n_tiles], zero between calls
    unsigned long long *acc64;  // split-K GEMV, exact completion: words [M][N_pad], zero between calls
    const int *bnd;        // per-column fixed-point exponent E of FP partial sums (packed weights)
    int64_t M, N, N_pad, K, KB, J, Q, G;
    int splits, kbs, out_dtype, accumulate;
    int kpg;               // 128-blocks of K per quantization group (G / 128)
    int per_tensor;        // one (s, z) pair for the whole tensor, FP32
    float inv_kpg;         // 1 / kpg (group index of a 128-block by one multiply)
    // Eq. 2 for the weight format: s' = cs * s, z' = cz * z + c0
    float cs, cz, c0;
};

struct DequantParams {
    const uint16_t *act;   // FP16 [M][K]
    const uint4 *planes;
    const void *meta;
    void *out;
    float *part;           // K split: FP32 partial sums [splits][M][N_pad], else NULL
    int64_t M, N, N_pad, K, KB, Q, G;
    int out_dtype, accumulate;
    int splits, kbs;       // K splits and 128-blocks per split
};

// Launch plan of the comparison path: which kernel, and its K split.
struct DequantPlan {
    int kind;        // 0: 128 x 128 tiles, 1: pipelined 256 x 256 tiles, 2: 16-token slabs (binary weights)
    int splits, kbs;
    size_t ws_bytes; // FP32 partial sums when splits > 1
};
DequantPlan plan_dequant(const Layout &L, int64_t M);

// Launchers (return hipError_t as int).
int launch_pack(const PackParams &p, void *stream);
int launch_precompute(const PrecomputeParams &p, int act_int8, void *stream);
int launch_lut(const LutParams &p, const Layout &L, const LutPlan &plan, void *stream);
int launch_gemv(const LutParams &p, const Layout &L, const LutPlan &plan, void *stream);
int launch_fused_gemv(const LutParams &p, const Layout &L, const LutPlan &plan, void *stream);
int launch_fused_split(const LutParams &p, const Layout &L, const LutPlan &plan, void *stream);
int launch_finalize(const LutParams &p, const Layout &L, const LutPlan &plan, void *stream);
int launch_mtok(const LutParams &p, const Layout &L, const LutPlan &plan, void *stream);
// The multi-token kernel building its tables from the FP16 activations (p.act).
int launch_mtok_fused(const LutParams &p, const Layout &L, const LutPlan &plan, void *stream);
int launch_tri(const LutParams &p, const Layout &L, bool fused, void *stream);
int launch_dequant(const DequantParams &p, const Layout &L, const DequantPlan &plan, void *stream);

}  // namespace lutgemm
