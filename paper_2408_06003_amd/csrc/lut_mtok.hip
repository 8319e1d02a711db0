// Multi-token bit-serial LUT mpGEMM with token-interleaved tables (LUT Tensor
// Core, Section 3.1 with Eq. 3, 5-6; the elongated M dimension of the LUT tile
// of Section 3.2.2, where one index selects an entry from the tables of several
// tokens at once).
//
// gfx950 mapping.  A workgroup of 256 lanes owns 256 columns (one per lane) and
// 8 tokens.  For each 4-activation group the signed 16-entry tables of the 8
// tokens are stored interleaved in LDS, entry i of tokens 0..7 in one 16-byte
// row, as 16-bit values: the exact INT16 entries on the INT8 path, the FP16
// entries of the precompute on the FP path.  One lookup is then one SDWA byte
// extract (the Eq. 6 index times 16) and one ds_read_b128 that returns the 8
// tokens' entries: 2 LDS bytes per lookup instead of 4.  INT8 path: the entries
// of one 128-block and bit-plane are summed in packed INT16 pairs (|sum| <= 32 x
// 508 < 2^15, exact), then widened to INT32 with the plane weight 2^t.  FP path:
// the 8 entries selected by one weight word (8 consecutive groups of one plane)
// are summed in packed FP16 pairs (v_pk_add_f16, two tokens per instruction; the
// tables are normalized to |T| < 4, so these sums stay below 32), the sums of
// planes 2i and 2i + 1 are combined as h_2i + 2 h_2i+1 (v_pk_fma_f16), and each
// result is added into the per-token FP32 outputs with factor 4^i s' (one
// v_fma_mix_f32 per token).  The zero-point term s' z' S of Eq. 3 is applied by
// the first block of each quantization group, the 8 tokens' sums S broadcast
// from 8 lanes by readlane.
//
// K is walked in chunks of CH 128-blocks.  Everything a chunk needs from memory
// (the 8 tokens' half-table words it stages, the weight words, the blocks'
// metadata and zero-point sums) is loaded one chunk ahead into one of two
// register buffers (used alternately, no copies, every load unconditional with
// clamped indices so that waits count exactly), and the LDS tables are
// double-buffered, so each chunk costs one barrier.  The loads go through buffer
// resources: workgroup-uniform offsets in scalar registers, fixed 32-bit lane
// offsets, no 64-bit address arithmetic in the loop.  When the grid would not
// fill the GPU, K is split and lut_finalize_kernel sums the partials.
//
// Precompute fused into the kernel (FZ != 0, FP16 activations; Section 3.1.1 splits
// the precompute out so that it can be fused): the workgroup reads the FP16
// activations of its tokens instead of precomputed half tables.  A first pass over
// its K range gives each token's absmax (and, FZ = 2, the sum of every 128-block:
// the S of Eq. 3 per block) and the power-of-two scale 2^-e with amax = f 2^e; each
// staging lane then forms its two table entries per token as
// ((-x0 + (+-x1)) + (+-x2)) + (+-x3) in FP32 from the scaled activations (exact
// products, one rounding per addition) and rounds them to FP16, the operations of
// the precompute operator.  The scale is local to the workgroup's K range; the
// partial sums are multiplied back by 2^e before they are stored, and power-of-two
// scaling commutes with every rounding on the way, so the output equals that of the
// two-launch path whenever no entry or partial sum is subnormal.
#include <type_traits>

#include "lut_common.h"

namespace lutgemm {

constexpr int MTK = 8;  // token slots of a 16-byte table row (tokens per half)
constexpr int FZ_SMAX = MTOK_FUSED_SMAX;  // fused build with zero points: most 128-blocks per K range

// The 16-bit lanes of x selected by SEL (v_perm_b32 byte selector) from {hi, lo}.
__device__ __forceinline__ uint32_t perm(uint32_t hi, uint32_t lo, uint32_t sel) {
    return __builtin_amdgcn_perm(hi, lo, sel);
}

// Sum of v over each row of 16 lanes by DPP (quad_perm [1,0,3,2], [2,3,0,1], row half
// mirror, row mirror): every lane of the row ends with the same bits.
__device__ __forceinline__ float row_sum16(float v) {
    v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0xB1, 0xF, 0xF, false));
    v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x4E, 0xF, 0xF, false));
    v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x141, 0xF, 0xF, false));
    v += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x140, 0xF, 0xF, false));
    return v;
}

template <bool INT8>
__device__ __forceinline__ uint32_t neg16x2(uint32_t x) {
    if constexpr (INT8) return neg_i16x2(x);
    return x ^ 0x80008000u;  // FP16: flip both sign bits (exact)
}

// Raw buffer resource over `bytes` bytes at `base` (stride 0; a load at or past the
// extent returns 0).  Loads through it take a 32-bit lane offset and a
// workgroup-uniform scalar offset, so they need no 64-bit address arithmetic.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ uint32_t buf_u32(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, (int)soff, 0);
}
__device__ __forceinline__ uint32_t buf_u16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    return __builtin_amdgcn_raw_buffer_load_b16(r, (int)voff, (int)soff, 0);
}
__device__ __forceinline__ uint2 buf_u64(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
    const u32x2 v = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(r, (int)voff, (int)soff, 0));
    return make_uint2(v.x, v.y);
}
__device__ __forceinline__ uint4 buf_u128(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0);
    return make_uint4(v.x, v.y, v.z, v.w);
}

// (x >> 8 j) & 0xF0 for a compile-time byte j (after unrolling) in one SDWA
// instruction: the high nibble of byte j of x, times 16, i.e. the byte offset of
// that Eq. 6 index's row in a token-interleaved table.  (The compiler emits a
// shift and a mask for bytes 1 and 2.)
__device__ __forceinline__ uint32_t nib_off(uint32_t x, int j) {
    uint32_t r;
    const uint32_t m = 0xF0u;
    switch (j) {
        case 0:
            asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0 src1_sel:DWORD"
                : "=v"(r) : "v"(x), "s"(m));
            break;
        case 1:
            asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1 src1_sel:DWORD"
                : "=v"(r) : "v"(x), "s"(m));
            break;
        case 2:
            asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2 src1_sel:DWORD"
                : "=v"(r) : "v"(x), "s"(m));
            break;
        default:
            asm("v_and_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3 src1_sel:DWORD"
                : "=v"(r) : "v"(x), "s"(m));
            break;
    }
    return r;
}

// h = a + b as four packed FP16 pairs (8 tokens): the first two entries of a word
// are summed without copying either into the accumulator.
__device__ __forceinline__ uint4 pk_sum4(uint4 a, uint4 b) {
    uint4 h;
    asm("v_pk_add_f16 %0, %4, %8\n\t"
        "v_pk_add_f16 %1, %5, %9\n\t"
        "v_pk_add_f16 %2, %6, %10\n\t"
        "v_pk_add_f16 %3, %7, %11"
        : "=&v"(h.x), "=&v"(h.y), "=&v"(h.z), "=&v"(h.w)
        : "v"(a.x), "v"(a.y), "v"(a.z), "v"(a.w), "v"(b.x), "v"(b.y), "v"(b.z), "v"(b.w));
    return h;
}

// 2 a + b as four packed FP16 pairs (8 tokens): two bit-planes' word sums combined.
__device__ __forceinline__ uint4 pk_fma2x4(uint4 a, uint4 b) {
    uint4 h;
    const uint32_t two = 0x40004000u;  // FP16 2.0 in both halves
    asm("v_pk_fma_f16 %0, %4, %12, %8\n\t"
        "v_pk_fma_f16 %1, %5, %12, %9\n\t"
        "v_pk_fma_f16 %2, %6, %12, %10\n\t"
        "v_pk_fma_f16 %3, %7, %12, %11"
        : "=&v"(h.x), "=&v"(h.y), "=&v"(h.z), "=&v"(h.w)
        : "v"(a.x), "v"(a.y), "v"(a.z), "v"(a.w), "v"(b.x), "v"(b.y), "v"(b.z), "v"(b.w), "s"(two));
    return h;
}

// ha += ea and hb += eb (two token halves), one statement for both reads of an index
__device__ __forceinline__ void pk_add4x2(uint4 &ha, uint4 ea, uint4 &hb, uint4 eb) {
    asm("v_pk_add_f16 %0, %0, %8\n\t"
        "v_pk_add_f16 %1, %1, %9\n\t"
        "v_pk_add_f16 %2, %2, %10\n\t"
        "v_pk_add_f16 %3, %3, %11\n\t"
        "v_pk_add_f16 %4, %4, %12\n\t"
        "v_pk_add_f16 %5, %5, %13\n\t"
        "v_pk_add_f16 %6, %6, %14\n\t"
        "v_pk_add_f16 %7, %7, %15"
        : "+v"(ha.x), "+v"(ha.y), "+v"(ha.z), "+v"(ha.w), "+v"(hb.x), "+v"(hb.y), "+v"(hb.z), "+v"(hb.w)
        : "v"(ea.x), "v"(ea.y), "v"(ea.z), "v"(ea.w), "v"(eb.x), "v"(eb.y), "v"(eb.z), "v"(eb.w));
}

// h += e as four packed FP16 pairs (8 tokens), one statement per read for the same
// reason as fma_mix8 below.
__device__ __forceinline__ void pk_add4(uint4 &h, uint4 e) {
    asm("v_pk_add_f16 %0, %0, %4\n\t"
        "v_pk_add_f16 %1, %1, %5\n\t"
        "v_pk_add_f16 %2, %2, %6\n\t"
        "v_pk_add_f16 %3, %3, %7"
        : "+v"(h.x), "+v"(h.y), "+v"(h.z), "+v"(h.w)
        : "v"(e.x), "v"(e.y), "v"(e.z), "v"(e.w));
}

// Four-token rows (two packed FP16 pairs): the same operations on uint2.
__device__ __forceinline__ uint2 pk_sum4(uint2 a, uint2 b) {
    uint2 h;
    asm("v_pk_add_f16 %0, %2, %4\n\t"
        "v_pk_add_f16 %1, %3, %5"
        : "=&v"(h.x), "=&v"(h.y)
        : "v"(a.x), "v"(a.y), "v"(b.x), "v"(b.y));
    return h;
}
__device__ __forceinline__ void pk_add4(uint2 &h, uint2 e) {
    asm("v_pk_add_f16 %0, %0, %2\n\t"
        "v_pk_add_f16 %1, %1, %3"
        : "+v"(h.x), "+v"(h.y)
        : "v"(e.x), "v"(e.y));
}
__device__ __forceinline__ uint2 pk_fma2x4(uint2 a, uint2 b) {
    uint2 h;
    const uint32_t two = 0x40004000u;
    asm("v_pk_fma_f16 %0, %2, %6, %4\n\t"
        "v_pk_fma_f16 %1, %3, %6, %5"
        : "=&v"(h.x), "=&v"(h.y)
        : "v"(a.x), "v"(a.y), "v"(b.x), "v"(b.y), "s"(two));
    return h;
}
__device__ __forceinline__ void fma_mix8(float *af, uint2 e, float sc) {
    asm("v_fma_mix_f32 %0, %4, %6, %0 op_sel_hi:[1,0,0]\n\t"
        "v_fma_mix_f32 %1, %4, %6, %1 op_sel:[1,0,0] op_sel_hi:[1,0,0]\n\t"
        "v_fma_mix_f32 %2, %5, %6, %2 op_sel_hi:[1,0,0]\n\t"
        "v_fma_mix_f32 %3, %5, %6, %3 op_sel:[1,0,0] op_sel_hi:[1,0,0]"
        : "+v"(af[0]), "+v"(af[1]), "+v"(af[2]), "+v"(af[3])
        : "v"(e.x), "v"(e.y), "v"(sc));
}
__device__ __forceinline__ uint32_t row_word(const uint4 &e, int j) {
    return j == 0 ? e.x : j == 1 ? e.y : j == 2 ? e.z : e.w;
}
__device__ __forceinline__ uint32_t row_word(const uint2 &e, int j) { return j == 0 ? e.x : e.y; }

// af[t] += sc * (FP16 entry of token t in e), t = 0..7: eight v_fma_mix_f32 in one
// statement, so each LDS read is consumed as a whole (the compiler would otherwise
// regroup the accumulations by token and keep every read of a block live).
__device__ __forceinline__ void fma_mix8(float *af, uint4 e, float sc) {
    asm("v_fma_mix_f32 %0, %8, %12, %0 op_sel_hi:[1,0,0]\n\t"
        "v_fma_mix_f32 %1, %8, %12, %1 op_sel:[1,0,0] op_sel_hi:[1,0,0]\n\t"
        "v_fma_mix_f32 %2, %9, %12, %2 op_sel_hi:[1,0,0]\n\t"
        "v_fma_mix_f32 %3, %9, %12, %3 op_sel:[1,0,0] op_sel_hi:[1,0,0]\n\t"
        "v_fma_mix_f32 %4, %10, %12, %4 op_sel_hi:[1,0,0]\n\t"
        "v_fma_mix_f32 %5, %10, %12, %5 op_sel:[1,0,0] op_sel_hi:[1,0,0]\n\t"
        "v_fma_mix_f32 %6, %11, %12, %6 op_sel_hi:[1,0,0]\n\t"
        "v_fma_mix_f32 %7, %11, %12, %7 op_sel:[1,0,0] op_sel_hi:[1,0,0]"
        : "+v"(af[0]), "+v"(af[1]), "+v"(af[2]), "+v"(af[3]), "+v"(af[4]), "+v"(af[5]), "+v"(af[6]), "+v"(af[7])
        : "v"(e.x), "v"(e.y), "v"(e.z), "v"(e.w), "v"(sc));
}

// Tile of a workgroup from its linear index.  Workgroups are dealt round-robin to the
// 8 XCDs, each with its own L2; with order != 0 the linear index is first turned into
// a position in the dealing XCD's own contiguous share of the tile space, so that the
// workgroups one XCD runs at the same time share weight tiles (same columns) and
// table tiles (same tokens) in that XCD's L2.  Splits of K vary slowest.
struct Tile {
    int64_t nt, mt;
    int split;
};
// (all counts below 2^24: 32-bit arithmetic)
__device__ __forceinline__ Tile tile_of(uint32_t b, uint32_t n_tiles, uint32_t m_tiles, int order) {
    const uint32_t per_split = n_tiles * m_tiles;
    const uint32_t total = gridDim.x;  // per_split x splits
    if (order != 0) {
        const uint32_t q = total >> 3, r = total & 7, x = b & 7, i = b >> 3;
        b = x * q + (x < r ? x : r) + i;
    }
    Tile t;
    t.split = (int)(b / per_split);
    const uint32_t w = b - (uint32_t)t.split * per_split;
    if (order == 0) {
        t.nt = w % n_tiles;
        t.mt = w / n_tiles;
    } else if (order == 1) {
        t.mt = w % m_tiles;
        t.nt = w / m_tiles;
    } else {
        // bands of `order` token tiles; inside a band tokens vary fastest, then columns
        const uint32_t o = (uint32_t)order;
        const uint32_t band = w / (o * n_tiles);
        const uint32_t first = band * o;
        const uint32_t rows = (m_tiles - first) < o ? (m_tiles - first) : o;
        const uint32_t v = w - band * o * n_tiles;
        t.mt = first + v % rows;
        t.nt = v / rows;
    }
    return t;
}

// NH halves of TK tokens per workgroup (NH = 2: one decoded index serves two 16-byte
// reads, the second at a fixed +256-byte offset, so index decoding, weight loads and
// metadata are shared by 16 tokens).  TK = 4 (one half, M <= 4): only the first 8
// bytes of each table row are filled and read (ds_read_b64), so a lookup costs half
// the LDS bytes and half the packed adds of an 8-token row.
// FZ: 0 = tables from the precompute; 1 = tables built from the FP16 activations;
// 2 = the same with the per-block activation sums of the zero-point term.
template <int BITS, bool INT8, bool TQ, int NH, int FZ, int TK>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(TQ ? 1 : (BITS == 1 && NH == 1 ? 6 : 4)))) void lut_mtok_kernel(LutParams p, int wfmt, int64_t n_tiles, int64_t m_tiles,
                                                       int order) {
    static_assert(FZ == 0 || (!INT8 && !TQ), "the fused table build takes FP16 activations");
    static_assert(TK == MTK || (TK == 4 && NH == 1 && !TQ), "rows of 8 tokens, or 4 in a single half");
    constexpr int MT = TK * NH;                   // tokens per workgroup
    typedef std::conditional_t<TK == MTK, uint4, uint2> Row;  // the row part a lookup reads
    // 128-blocks per chunk (b = 1 and 16 tokens: 16 KB of LDS per buffer, more workgroups per CU)
    constexpr int CH = (BITS == 1 || NH == 2) ? 1 : 4 / BITS;
    // staging tasks per chunk: (block, group, index pair); with FZ (token slice, block,
    // group, index pair), a slice being the 8 tokens of a half.  1-bit weights (one plane
    // of lookups per chunk, so the build weighs most) take slices of 4 tokens where 8
    // would leave half the lanes idle, so every lane shares the build (measured at M = 4
    // and 8: 1.5 us faster for 1-bit weights, 2 us slower for 4-bit ones)
    constexpr int HT = CH * GPB * 4 * NH;         // FZ: (half, block, group, index pair) tasks
    constexpr int TOK = (FZ && BITS == 1 && HT < 256 && TK == MTK) ? MTK * HT / 256 : TK;  // FZ: tokens per task
    constexpr int TASKS = FZ ? HT * (TK / TOK) : CH * GPB * 4;
    constexpr int TPL = (TASKS + 255) / 256;      // staging tasks per lane
    static_assert(FZ == 0 || (TPL == 1 && (TOK == 4 || TOK == 8)), "one fused staging task per lane");
    constexpr int GST = 256 * NH;                 // LDS bytes of one group (16 entries x 8 tokens x 2 B per half)
    constexpr int BUF = CH * GPB * GST;           // LDS bytes of one table buffer
    // 16 KB (b = 1, 4, 8 tokens) or 32 KB, plus with FZ = 2 the block sums of the K range
    // (at most FZ_SMAX blocks).  Occupancy hints: b = 1 with 8 tokens keeps six
    // workgroups per CU; the others measured faster at four, where the scheduler keeps
    // more LDS reads in flight per wavefront
    __shared__ __attribute__((aligned(16))) char F[2 * BUF + (FZ == 2 ? FZ_SMAX * MT * 4 : 0)];

    const int tid = threadIdx.x;
    const Tile tl = tile_of(blockIdx.x, (uint32_t)n_tiles, (uint32_t)m_tiles, order);
    const uint32_t n = (uint32_t)(tl.nt * NTILE + tid);
    const int split = tl.split;
    const int64_t m0 = tl.mt * MT;
    // 128-block indices fit in 32 bits (K < 2^38)
    const int kbA = split * p.kbs;
    const int kbB = (kbA + p.kbs < (int)p.KB) ? kbA + p.kbs : (int)p.KB;
    const bool need_s = !INT8 && wfmt != LUTGEMM_WFMT_BINARY;
    // Token rows past M repeat row M - 1: their sums are computed but never stored.
    auto row_of = [&](int t) { return (m0 + t < p.M) ? m0 + t : p.M - 1; };
    // Loads go through buffer resources: the workgroup-uniform part of each address
    // (token row, chunk, block, quantization group) is a scalar offset, lanes add
    // 32-bit offsets, so the loads cost almost no vector instructions.  Extents: the
    // tile's live token rows (K < 2^20: under 2^25 bytes), one chunk of planes.
    const int64_t J = p.J;
    const uint32_t rows_live = (uint32_t)((p.M - m0) < MT ? (p.M - m0) : MT);
    constexpr uint32_t TB = TQ ? 8 : 16;  // bytes per stored half table
    // (FZ: the tile's activation rows instead of its tables)
    const __amdgpu_buffer_rsrc_t rT = FZ ? buf_rsrc(p.act + m0 * p.K, rows_live * (uint32_t)p.K * 2u)
                                         : buf_rsrc((const char *)p.T + m0 * J * TB, rows_live * (uint32_t)J * TB);
    const __amdgpu_buffer_rsrc_t rTs = buf_rsrc(TQ ? (const void *)(p.tsc + m0 * J) : (const void *)p.T,
                                                TQ ? rows_live * (uint32_t)J * 4u : 0u);
    const __amdgpu_buffer_rsrc_t rS = FZ ? buf_rsrc(nullptr, 0u)
                                         : buf_rsrc((const float *)p.S + m0 * p.Q, rows_live * (uint32_t)p.Q * 4u);
    const uint32_t n_meta = p.per_tensor ? 0u : n;  // metadata column (0: one pair per tensor)
    // quantization group of a 128-block (workgroup-uniform: moved to a scalar register,
    // so that what depends on it is scalar arithmetic)
    auto group_of = [&](int kb) {
        return __builtin_amdgcn_readfirstlane((int)(((float)kb + 0.5f) * p.inv_kpg));
    };
    // staged table words: entries 2ip, 2ip + 1 of a token's half table (FP16 / INT16
    // pair), or with INT8-quantized tables (TQ) their two codes and the table's scale;
    // FZ: the 4 FP16 activations of the task's group, for the TOK tokens of its slice
    typedef std::conditional_t<TQ || FZ, uint2, uint32_t> SDE;
    typedef SDE SD[TPL][FZ ? TOK : MT];
    typedef uint4 WW[CH][BITS];
    struct MW {
        uint2 w[CH];  // metadata words of each block's group
        int q[CH];    // each block's group
    };
    typedef float SV[1];
    auto load = [&](int kc, SD &sd, WW &w, MW &mw, SV &sv) {
        const int nkb = (kbB - kc) < CH ? (kbB - kc) : CH;
        if constexpr (FZ) {
            // task (token slice q, block kbl, group g, index pair ip), ip fastest; q and
            // kbl are uniform over a wavefront, so the row and block offsets are scalar
            // (lanes past the tasks load rows past the tile: clamped, or zero from the
            // buffer's extent, and never staged)
            const int q = __builtin_amdgcn_readfirstlane(tid / (CH * 128));
            const int kbl = __builtin_amdgcn_readfirstlane((tid / 128) % CH);
            const int kbc = kbl < nkb ? kbl : nkb - 1;
            const uint32_t g = (uint32_t)((tid >> 2) & 31);
#pragma unroll
            for (int t = 0; t < TOK; ++t) {
                const uint32_t so = (uint32_t)(row_of(TOK * q + t) - m0) * (uint32_t)p.K * 2u + (uint32_t)(kc + kbc) * 256u;
                sd[0][t] = buf_u64(rT, g * 8u, so);
            }
        } else {
#pragma unroll
        for (int r = 0; r < TPL; ++r) {
            const int task = tid + 256 * r;
            const int tk = task < TASKS ? task : TASKS - 1;
            const int kbl = tk >> 7, g = (tk >> 2) & 31, ip = tk & 3;
            const int kbc = kbl < nkb ? kbl : nkb - 1;
            const uint32_t tab = (uint32_t)(kbc * GPB + g);  // the lane's table within the chunk
#pragma unroll
            for (int t = 0; t < MT; ++t) {
                const uint32_t so = ((uint32_t)(row_of(t) - m0) * (uint32_t)J + (uint32_t)kc * GPB) * TB;
                if constexpr (TQ)
                    sd[r][t] = make_uint2(buf_u16(rT, tab * 8 + ip * 2, so), buf_u32(rTs, tab * 4, so / 2));
                else
                    sd[r][t] = buf_u32(rT, tab * 16 + ip * 4, so);
            }
        }
        }
        const __amdgpu_buffer_rsrc_t rW =
            buf_rsrc(p.planes + (int64_t)kc * BITS * p.N_pad, (uint32_t)(CH * BITS) * (uint32_t)p.N_pad * 16u);
#pragma unroll
        for (int kbl = 0; kbl < CH; ++kbl) {
            const int kbc = kbl < nkb ? kbl : nkb - 1;
#pragma unroll
            for (int t = 0; t < BITS; ++t)
                w[kbl][t] = buf_u128(rW, n * 16u, (uint32_t)(kbc * BITS + t) * (uint32_t)p.N_pad * 16u);
        }
        if constexpr (!INT8) {
#pragma unroll
            for (int kbl = 0; kbl < CH; ++kbl) {
                const int kbc = kbl < nkb ? kbl : nkb - 1;
                const int q = group_of(kc + kbc);
                const __amdgpu_buffer_rsrc_t rM =
                    buf_rsrc((const uint32_t *)p.meta + (p.per_tensor ? 0 : (int64_t)q * p.N_pad), (uint32_t)p.N_pad * 4u);
                mw.w[kbl] = make_uint2(buf_u32(rM, n_meta * 4u, 0), buf_u32(rM, n_meta * 4u, p.per_tensor ? 4u : 0u));
                mw.q[kbl] = q;
            }
            // one activation sum per (block, token): lanes 0 .. MT CH - 1 of every wavefront,
            // broadcast to the others by readlane (FZ: the block sums are in LDS)
            if constexpr (!FZ) {
                const int ln = tid & 63;
                const int t = ln % MT;
                const int q = (CH == 1 || ln < MT) ? mw.q[0] : mw.q[CH - 1];
                const uint32_t rt = (uint32_t)(row_of(t) - m0);
                sv[0] = __uint_as_float(buf_u32(rS, (rt * (uint32_t)p.Q + (uint32_t)q) * 4u, 0));
            }
        }
    };

    float yf[MT];
    int yi[MT];
#pragma unroll
    for (int t = 0; t < MT; ++t) {
        yf[t] = 0.f;
        yi[t] = 0;
    }
    // FZ: lane l holds the scale 2^-e and the output factor 2^e of token l % MT
    float escl = 1.f, etok = 1.f;

    auto process = [&](int kc, const SD &sd, const WW &w, const MW &mw, const SV &sv, int b) {
        const int nkb = (kbB - kc) < CH ? (kbB - kc) : CH;
        char *Fb = F + b * BUF;
        // stage: for each task, entries 2ip, 2ip + 1 and their negations for the 8 tokens
        if constexpr (FZ) {
            // the two entries formed here from the activations: T[2ip + s] =
            // ((-x0 + (+-x1)) + (+-x2)) + (+-x3), x1 added when bit 2 of 2ip is set, x2
            // when bit 1 is, x3 subtracted for s = 0 and added for s = 1; the signs of x1
            // and x2 are applied by flipping the FP16 sign bits, x_e = a_e 2^-e exactly
            const int q = __builtin_amdgcn_readfirstlane(tid / (CH * 128));
            const int kbl = (tid / 128) % CH, g = (tid >> 2) & 31, ip = tid & 3;
            if (tid < TASKS && kbl < nkb) {
                const uint32_t f1 = (ip & 2) ? 0u : 0x80000000u, f2 = (ip & 1) ? 0u : 0x8000u;
                uint32_t r0[TOK / 2], r1[TOK / 2];
#pragma unroll
                for (int t = 0; t < TOK; ++t) {
                    const float sc = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(escl), TOK * q + t));
                    const uint32_t ax = sd[0][t].x ^ f1, ay = sd[0][t].y ^ f2;
                    const float nx0 = fmaf(h2f(ax & 0xFFFFu), -sc, -0.0f);  // -x0, exact (and -0 for +0)
                    const float bb = fmaf(h2f(ax >> 16), sc, nx0);
                    const float u = fmaf(h2f(ay & 0xFFFFu), sc, bb);
                    const float x3 = h2f(ay >> 16);
                    float t0 = fmaf(-x3, sc, u), t1 = fmaf(x3, sc, u);
                    // rounded to FP32 first, then to FP16 (not one fused FMA-to-FP16 rounding)
                    asm volatile("" : "+v"(t0), "+v"(t1));
                    const uint32_t q0 = __half_as_ushort(__float2half_rn(t0));
                    const uint32_t q1 = __half_as_ushort(__float2half_rn(t1));
                    if (t & 1) {
                        r0[t / 2] |= q0 << 16;
                        r1[t / 2] |= q1 << 16;
                    } else {
                        r0[t / 2] = q0;
                        r1[t / 2] = q1;
                    }
                }
                // slice q: half (TOK q) / 8 of the row, at token (TOK q) % 8 within it
                char *row = Fb + (kbl * GPB + g) * GST + 256 * (TOK * q / TK) + 2 * (TOK * q % TK);
                if constexpr (TOK == MTK) {
                    const uint4 e0 = make_uint4(r0[0], r0[1], r0[2], r0[3]), e1 = make_uint4(r1[0], r1[1], r1[2], r1[3]);
                    *(uint4 *)(row + (2 * ip) * 16) = e0;
                    *(uint4 *)(row + (2 * ip + 1) * 16) = e1;
                    *(uint4 *)(row + (2 * ip + 8) * 16) =
                        make_uint4(neg16x2<false>(e0.x), neg16x2<false>(e0.y), neg16x2<false>(e0.z), neg16x2<false>(e0.w));
                    *(uint4 *)(row + (2 * ip + 9) * 16) =
                        make_uint4(neg16x2<false>(e1.x), neg16x2<false>(e1.y), neg16x2<false>(e1.z), neg16x2<false>(e1.w));
                } else {
                    *(uint2 *)(row + (2 * ip) * 16) = make_uint2(r0[0], r0[1]);
                    *(uint2 *)(row + (2 * ip + 1) * 16) = make_uint2(r1[0], r1[1]);
                    *(uint2 *)(row + (2 * ip + 8) * 16) = make_uint2(neg16x2<false>(r0[0]), neg16x2<false>(r0[1]));
                    *(uint2 *)(row + (2 * ip + 9) * 16) = make_uint2(neg16x2<false>(r1[0]), neg16x2<false>(r1[1]));
                }
            }
        } else {
#pragma unroll
        for (int r = 0; r < TPL; ++r) {
            const int task = tid + 256 * r;
            const int kbl = task >> 7, g = (task >> 2) & 31, ip = task & 3;
            if (task < TASKS && kbl < nkb) {
#pragma unroll
                for (int h = 0; h < NH; ++h) {
                    uint32_t v[MTK];
#pragma unroll
                    for (int t = 0; t < TK; ++t) {
                        if constexpr (TQ) {  // code x scale, rounded to FP16
                            const float sc = __uint_as_float(sd[r][MTK * h + t].y);
                            const float f0 = (float)(int8_t)(sd[r][MTK * h + t].x & 0xFFu) * sc;
                            const float f1 = (float)(int8_t)((sd[r][MTK * h + t].x >> 8) & 0xFFu) * sc;
                            v[t] = (uint32_t)__half_as_ushort(__float2half_rn(f0)) |
                                   ((uint32_t)__half_as_ushort(__float2half_rn(f1)) << 16);
                        } else {
                            v[t] = sd[r][TK * h + t];
                        }
                    }
                    char *row = Fb + (kbl * GPB + g) * GST + 256 * h;
                    if constexpr (TK == MTK) {
                        uint4 e0, e1;  // entries 2ip (low halves) and 2ip + 1 (high halves), tokens 8h .. 8h + 7
                        e0.x = perm(v[1], v[0], 0x05040100u);
                        e0.y = perm(v[3], v[2], 0x05040100u);
                        e0.z = perm(v[5], v[4], 0x05040100u);
                        e0.w = perm(v[7], v[6], 0x05040100u);
                        e1.x = perm(v[1], v[0], 0x07060302u);
                        e1.y = perm(v[3], v[2], 0x07060302u);
                        e1.z = perm(v[5], v[4], 0x07060302u);
                        e1.w = perm(v[7], v[6], 0x07060302u);
                        *(uint4 *)(row + (2 * ip) * 16) = e0;
                        *(uint4 *)(row + (2 * ip + 1) * 16) = e1;
                        *(uint4 *)(row + (2 * ip + 8) * 16) =
                            make_uint4(neg16x2<INT8>(e0.x), neg16x2<INT8>(e0.y), neg16x2<INT8>(e0.z), neg16x2<INT8>(e0.w));
                        *(uint4 *)(row + (2 * ip + 9) * 16) =
                            make_uint4(neg16x2<INT8>(e1.x), neg16x2<INT8>(e1.y), neg16x2<INT8>(e1.z), neg16x2<INT8>(e1.w));
                    } else {  // tokens 0 .. 3 in the first 8 bytes of each row
                        const uint2 e0 = make_uint2(perm(v[1], v[0], 0x05040100u), perm(v[3], v[2], 0x05040100u));
                        const uint2 e1 = make_uint2(perm(v[1], v[0], 0x07060302u), perm(v[3], v[2], 0x07060302u));
                        *(uint2 *)(row + (2 * ip) * 16) = e0;
                        *(uint2 *)(row + (2 * ip + 1) * 16) = e1;
                        *(uint2 *)(row + (2 * ip + 8) * 16) = make_uint2(neg16x2<INT8>(e0.x), neg16x2<INT8>(e0.y));
                        *(uint2 *)(row + (2 * ip + 9) * 16) = make_uint2(neg16x2<INT8>(e1.x), neg16x2<INT8>(e1.y));
                    }
                }
            }
        }
        }
        lds_barrier();
#pragma unroll
        for (int kbl = 0; kbl < CH; ++kbl) {
            if (kbl >= nkb) continue;
            if constexpr (INT8) {
                // INT8 path: per plane, the 32 entries of the block summed exactly in packed
                // INT16 (|sum| <= 32 x 508 < 2^15), then widened with the plane weight 2^pl
#pragma unroll
                for (int pl = 0; pl < BITS; ++pl) {
                    short2_v a16[NH][TK / 2];
#pragma unroll
                    for (int h = 0; h < NH; ++h)
#pragma unroll
                        for (int j = 0; j < TK / 2; ++j) a16[h][j] = short2_v{0, 0};
                    const uint32_t wd[4] = {w[kbl][pl].x, w[kbl][pl].y, w[kbl][pl].z, w[kbl][pl].w};
#pragma unroll
                    for (int d = 0; d < 4; ++d) {
                        const uint32_t lo = wd[d] << 4, hi = wd[d];
#pragma unroll
                        for (int k = 0; k < 8; ++k) {
                            const uint32_t off = nib_off((k & 1) ? hi : lo, k >> 1);
                            const int g = d * 8 + k;  // groups 2j (low nibble) and 2j + 1 (high nibble) of byte j
#pragma unroll
                            for (int h = 0; h < NH; ++h) {
                                const Row e = *(const Row *)(Fb + (kbl * GPB + g) * GST + 256 * h + off);
#pragma unroll
                                for (int j = 0; j < TK / 2; ++j) a16[h][j] += __builtin_bit_cast(short2_v, row_word(e, j));
                            }
                        }
                    }
#pragma unroll
                    for (int h = 0; h < NH; ++h)
#pragma unroll
                        for (int j = 0; j < TK / 2; ++j) {
                            yi[TK * h + 2 * j] += (int)a16[h][j].x << pl;
                            yi[TK * h + 2 * j + 1] += (int)a16[h][j].y << pl;
                        }
                }
            } else {
                // FP path, per weight word: the 8 entries one plane's word selects summed in
                // packed FP16, pairs of planes combined as h_2i + 2 h_2i+1 (v_pk_fma_f16),
                // and each result added into the FP32 outputs with factor 4^i s' (one
                // v_fma_mix_f32 per token)
                const SZ sz = decode_sz(p, mw.w[kbl]);
#pragma unroll
                for (int d = 0; d < 4; ++d) {
                    Row hp[NH][BITS];
#pragma unroll
                    for (int pl = 0; pl < BITS; ++pl) {
                        const uint32_t wv = d == 0 ? w[kbl][pl].x : d == 1 ? w[kbl][pl].y : d == 2 ? w[kbl][pl].z : w[kbl][pl].w;
                        const uint32_t lo = wv << 4, hi = wv;
                        Row e[8][NH];
#pragma unroll
                        for (int k = 0; k < 8; ++k) {
                            const uint32_t off = nib_off((k & 1) ? hi : lo, k >> 1);
                            const int g = d * 8 + k;  // groups 2j (low nibble) and 2j + 1 (high nibble) of byte j
#pragma unroll
                            for (int h = 0; h < NH; ++h) e[k][h] = *(const Row *)(Fb + (kbl * GPB + g) * GST + 256 * h + off);
                            if (k == 1) {
#pragma unroll
                                for (int h = 0; h < NH; ++h) hp[h][pl] = pk_sum4(e[0][h], e[1][h]);
                            } else if (k >= 2) {
                                if constexpr (NH == 2 && BITS > 1) {
                                    if (k & 1) {  // two indices, four reads in flight together
                                        pk_add4x2(hp[0][pl], e[k - 1][0], hp[1][pl], e[k - 1][1]);
                                        pk_add4x2(hp[0][pl], e[k][0], hp[1][pl], e[k][1]);
                                    }
                                } else {
#pragma unroll
                                    for (int h = 0; h < NH; ++h) pk_add4(hp[h][pl], e[k][h]);
                                }
                            }
                        }
                    }
#pragma unroll
                    for (int h = 0; h < NH; ++h) {
                        if constexpr (BITS == 1) {
                            fma_mix8(yf + TK * h, hp[h][0], sz.sp);
                        } else {
#pragma unroll
                            for (int i = 0; i < BITS / 2; ++i)
                                fma_mix8(yf + TK * h, pk_fma2x4(hp[h][2 * i + 1], hp[h][2 * i]), sz.sp * (float)(1 << (2 * i)));
                        }
                    }
                }
                if constexpr (FZ == 2) {  // the zero-point term of this block, from its sums in LDS
                    if (need_s) {
                        const float nspz = -(sz.sp * sz.zp);
                        const float *sb = (const float *)(F + 2 * BUF) + (kc + kbl - kbA) * MT;
#pragma unroll
                        for (int t = 0; t < MT; ++t) yf[t] = fmaf(nspz, sb[t], yf[t]);
                    }
                } else if (need_s && kc + kbl == mw.q[kbl] * p.kpg) {
                    // the zero-point term enters with the first block of each group only
                    const float nspz = -(sz.sp * sz.zp);
#pragma unroll
                    for (int t = 0; t < MT; ++t) {
                        const float st = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(sv[0]), kbl * MT + t));
                        yf[t] = fmaf(nspz, st, yf[t]);
                    }
                }
            }
        }
    };

    // INT8 ternary: the activation sums S[m][0], added once (first K split)
    if (INT8 && split == 0 && wfmt == LUTGEMM_WFMT_TERNARY) {
#pragma unroll
        for (int t = 0; t < MT; ++t) yi[t] = ((const int *)p.S)[lane_value(row_of(t) * p.Q)];
    }
    const int last = kbA + (kbB - 1 - kbA) / CH * CH;
    SD sdA, sdB;
    WW wA, wB;
    MW mwA, mwB;
    SV svA, svB;
    load(kbA, sdA, wA, mwA, svA);
    if constexpr (FZ) {
        // absmax of each token over this workgroup's K range (FZ = 2: and the sum of each
        // 128-block), LPT lanes per token and 16 bytes per lane and block, eight loads in
        // flight (issued after the first chunk's, whose latency they share)
        constexpr int LPT = 256 / MT;  // 16 or 32
        constexpr int BPS = LPT / 16;  // 128-blocks per step
        const int t = tid / LPT, sub = tid % LPT;
        const uint32_t rowoff = (uint32_t)(row_of(t) - m0) * (uint32_t)p.K * 2u + (uint32_t)(sub & 15) * 16u;
        float *sl = (float *)(F + 2 * BUF);
        uint32_t mx = 0u;  // two FP16 magnitudes (the bits of a finite |a| order like integers)
        for (int i0 = 0; i0 < kbB - kbA; i0 += 8 * BPS) {
            uint4 v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int kb = kbA + i0 + u * BPS + (sub >> 4);
                v[u] = buf_u128(rT, rowoff + (uint32_t)(kb < kbB ? kb : kbB - 1) * 256u, 0);
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                mx = max_u16x2(mx, max_u16x2(max_u16x2(v[u].x & 0x7FFF7FFFu, v[u].y & 0x7FFF7FFFu),
                                             max_u16x2(v[u].z & 0x7FFF7FFFu, v[u].w & 0x7FFF7FFFu)));
                if constexpr (FZ == 2) {
                    const uint32_t d[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
                    float sm = 0.f;
#pragma unroll
                    for (int i = 0; i < 4; ++i) sm = (sm + h2f(d[i] & 0xFFFFu)) + h2f(d[i] >> 16);
                    sm = row_sum16(sm);
                    const int kb = kbA + i0 + u * BPS + (sub >> 4);
                    if ((sub & 15) == 0 && kb < kbB && kb - kbA < FZ_SMAX) sl[(kb - kbA) * MT + t] = sm;
                }
            }
        }
        uint32_t m16 = (mx & 0xFFFFu) > (mx >> 16) ? (mx & 0xFFFFu) : (mx >> 16);
#pragma unroll
        for (int off = 1; off < LPT; off <<= 1) {
            const uint32_t o = (uint32_t)__shfl_xor((int)m16, off, 64);
            m16 = o > m16 ? o : m16;
        }
        float *xs = (float *)(F + BUF);  // scale and factor per token, in the second table buffer
        if (sub == 0) {
            const float amax = h2f(m16);
            float sc = 1.f, tk = 1.f;
            if (amax != 0.f) {
                int e2;
                (void)frexpf(amax, &e2);
                sc = ldexpf(1.f, -e2);
                tk = ldexpf(1.f, e2);
            }
            xs[t] = sc;
            xs[MT + t] = tk;
        }
        lds_barrier();
        if constexpr (FZ == 2) {  // the block sums of the scaled activations (exact rescaling)
            for (int i = tid; i < (kbB - kbA) * MT && i < FZ_SMAX * MT; i += 256) sl[i] *= xs[i % MT];
        }
        escl = xs[tid % MT];
        etok = xs[MT + tid % MT];
        if constexpr (FZ == 2) lds_barrier();
    }
    for (int kc = kbA; kc < kbB; kc += 2 * CH) {
        load(kc + CH < last ? kc + CH : last, sdB, wB, mwB, svB);
        process(kc, sdA, wA, mwA, svA, 0);
        if (kc + CH >= kbB) break;
        load(kc + 2 * CH < last ? kc + 2 * CH : last, sdA, wA, mwA, svA);
        process(kc + CH, sdB, wB, mwB, svB, 1);
    }

    const int rows = (int)((p.M - m0) < MT ? (p.M - m0) : MT);
    if (p.splits == 1) {
#pragma unroll
        for (int t = 0; t < MT; ++t)
            if (t < rows) {
                Epi ep = load_epi<INT8>(p, wfmt, m0 + t, n, false);
                if constexpr (FZ != 0) ep.tok = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(etok), t));
                store_out<INT8>(p, wfmt, m0 + t, n, yf[t], yi[t], ep);
            }
        return;
    }
    const int64_t m_alloc = m_tiles * MT;
#pragma unroll
    for (int t = 0; t < MT; ++t) {  // the finalize kernel reads rows below M only
        // FZ: the partial times this K range's 2^e (the finalize kernel applies no factor)
        const float v = FZ ? yf[t] * __int_as_float(__builtin_amdgcn_readlane(__float_as_int(etok), t)) : yf[t];
        if (t < rows) p.part[((int64_t)split * m_alloc + m0 + t) * p.N_pad + n] = INT8 ? __int_as_float(yi[t]) : v;
    }
}

template <int NH, int TK>
static void launch_mtok_nh(const LutParams &p, const Layout &L, const LutPlan &plan, hipStream_t s) {
    // one-dimensional grid (tile_of decodes it); the planner keeps it under 2^32 work-items
    const dim3 grid((unsigned)(plan.n_tiles * plan.m_tiles * plan.splits), 1, 1);
    const bool i8 = L.act == LUTGEMM_ACT_INT8;
    const int64_t nt = plan.n_tiles, mt = plan.m_tiles;
    const int o = plan.order;
    if (L.bits == 1) {
        if (i8) hipLaunchKernelGGL((lut_mtok_kernel<1, true, false, NH, 0, TK>), grid, dim3(256), 0, s, p, L.wfmt, nt, mt, o);
        else hipLaunchKernelGGL((lut_mtok_kernel<1, false, false, NH, 0, TK>), grid, dim3(256), 0, s, p, L.wfmt, nt, mt, o);
    } else if (L.bits == 2) {
        if (i8) hipLaunchKernelGGL((lut_mtok_kernel<2, true, false, NH, 0, TK>), grid, dim3(256), 0, s, p, L.wfmt, nt, mt, o);
        else hipLaunchKernelGGL((lut_mtok_kernel<2, false, false, NH, 0, TK>), grid, dim3(256), 0, s, p, L.wfmt, nt, mt, o);
    } else {
        hipLaunchKernelGGL((lut_mtok_kernel<4, false, false, NH, 0, TK>), grid, dim3(256), 0, s, p, L.wfmt, nt, mt, o);
    }
}

// Tables built in the kernel from FP16 activations: FZ = 2 when the format has zero
// points (the per-block activation sums are kept in LDS), else 1.
template <int NH, int FZ, int TK>
static void launch_mtok_fz(const LutParams &p, const Layout &L, const LutPlan &plan, hipStream_t s) {
    const dim3 grid((unsigned)(plan.n_tiles * plan.m_tiles * plan.splits), 1, 1);
    const int64_t nt = plan.n_tiles, mt = plan.m_tiles;
    const int o = plan.order;
    if (L.bits == 1) hipLaunchKernelGGL((lut_mtok_kernel<1, false, false, NH, FZ, TK>), grid, dim3(256), 0, s, p, L.wfmt, nt, mt, o);
    else if (L.bits == 2) hipLaunchKernelGGL((lut_mtok_kernel<2, false, false, NH, FZ, TK>), grid, dim3(256), 0, s, p, L.wfmt, nt, mt, o);
    else hipLaunchKernelGGL((lut_mtok_kernel<4, false, false, NH, FZ, TK>), grid, dim3(256), 0, s, p, L.wfmt, nt, mt, o);
}

int launch_mtok(const LutParams &p, const Layout &L, const LutPlan &plan, void *stream) {
    hipStream_t s = (hipStream_t)stream;
    if (L.act == LUTGEMM_ACT_FP16_LUT8) {  // INT8-quantized tables: 8 tokens per workgroup
        const dim3 grid((unsigned)(plan.n_tiles * plan.m_tiles * plan.splits), 1, 1);
        const int64_t nt = plan.n_tiles, mt = plan.m_tiles;
        const int o = plan.order;
        if (L.bits == 1) hipLaunchKernelGGL((lut_mtok_kernel<1, false, true, 1, 0, 8>), grid, dim3(256), 0, s, p, L.wfmt, nt, mt, o);
        else if (L.bits == 2) hipLaunchKernelGGL((lut_mtok_kernel<2, false, true, 1, 0, 8>), grid, dim3(256), 0, s, p, L.wfmt, nt, mt, o);
        else hipLaunchKernelGGL((lut_mtok_kernel<4, false, true, 1, 0, 8>), grid, dim3(256), 0, s, p, L.wfmt, nt, mt, o);
    } else if (plan.mt == 16) {
        launch_mtok_nh<2, 8>(p, L, plan, s);
    } else if (plan.mt == 4) {
        launch_mtok_nh<1, 4>(p, L, plan, s);
    } else {
        launch_mtok_nh<1, 8>(p, L, plan, s);
    }
    return (int)hipGetLastError();
}

int launch_mtok_fused(const LutParams &p, const Layout &L, const LutPlan &plan, void *stream) {
    hipStream_t s = (hipStream_t)stream;
    if (L.act != LUTGEMM_ACT_FP16 || !p.act) return (int)hipErrorInvalidValue;
    const bool zp = L.wfmt != LUTGEMM_WFMT_BINARY;
    if (zp && plan.kbs > MTOK_FUSED_SMAX) return (int)hipErrorInvalidValue;  // the planner caps it
    if (plan.mt == 16) {
        if (zp) launch_mtok_fz<2, 2, 8>(p, L, plan, s);
        else launch_mtok_fz<2, 1, 8>(p, L, plan, s);
    } else if (plan.mt == 4) {
        if (zp) launch_mtok_fz<1, 2, 4>(p, L, plan, s);
        else launch_mtok_fz<1, 1, 4>(p, L, plan, s);
    } else {
        if (zp) launch_mtok_fz<1, 2, 8>(p, L, plan, s);
        else launch_mtok_fz<1, 1, 8>(p, L, plan, s);
    }
    return (int)hipGetLastError();
}

}  // namespace lutgemm
