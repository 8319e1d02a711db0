// Device helpers shared by the LUT mpGEMM kernels (single-token GEMV and
// multi-token GEMM): table expansion, the Eq. 2 / Eq. 3 epilogue operands,
// output conversion and the fixed-order split-K sum.
#pragma once

#include <hip/hip_runtime.h>

#include <climits>
#include <hip/hip_fp16.h>

#include "lutgemm_internal.h"

namespace lutgemm {

// Phase timestamps of instrumented builds (-DLUTGEMM_TIMELINE, never the product
// library): lane 0 of each wavefront stores the 100 MHz real-time clock at a phase
// boundary into slot `slot` of its record, p.tl[(linear workgroup id x waves per
// workgroup + wave) x TL_SLOTS + slot].  Every use is a no-op in normal builds.
constexpr int TL_SLOTS = 8;
template <typename P>
__device__ __forceinline__ void tl_stamp(const P &p, int slot) {
#ifdef LUTGEMM_TIMELINE
    if (p.tl && (threadIdx.x & 63) == 0) {
        const uint64_t wg = ((uint64_t)blockIdx.z * gridDim.y + blockIdx.y) * gridDim.x + blockIdx.x;
        p.tl[(wg * (blockDim.x >> 6) + (threadIdx.x >> 6)) * TL_SLOTS + slot] = wall_clock64();
    }
#else
    (void)p;
    (void)slot;
#endif
}

template <typename P>
__device__ __forceinline__ void tl_clear(const P &p, int slot) {
#ifdef LUTGEMM_TIMELINE
    if (p.tl && (threadIdx.x & 63) == 0) {
        const uint64_t wg = ((uint64_t)blockIdx.z * gridDim.y + blockIdx.y) * gridDim.x + blockIdx.x;
        p.tl[(wg * (blockDim.x >> 6) + (threadIdx.x >> 6)) * TL_SLOTS + slot] = 0;
    }
#else
    (void)p;
    (void)slot;
#endif
}

// LDS-only barrier: waits for this wave's LDS writes (lgkmcnt) but not for its
// global loads, so prefetches issued before it stay in flight.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Keeps a value in a VGPR so that loads indexed by it stay vector loads (scalar
// loads share the LDS completion counter and would serialize the lookups).
__device__ __forceinline__ int64_t lane_value(int64_t x) {
    asm volatile("" : "+v"(x));
    return x;
}

__device__ __forceinline__ float h2f(uint32_t bits16) {
    return __half2float(__ushort_as_half((unsigned short)bits16));
}

// Activation value entering a table: the INT8 quantization of the activation
// quantizer, or the exact power-of-two token scaling of the FP path.
template <bool INT8>
__device__ __forceinline__ float act_value(uint32_t bits16, float scale) {
    // a * scale, one rounding, as a mixed-precision fma on the FP16 operand (adding -0
    // leaves every product, signed zeros included, unchanged)
    const float x = fmaf(h2f(bits16), scale, -0.0f);
    if (INT8) return __builtin_amdgcn_fmed3f(rintf(x), -127.f, 127.f);  // clamp to [-127, 127]
    return x;  // exact: scale is a power of two
}

__device__ __forceinline__ float absmax4(uint2 v) {
    return fmaxf(fmaxf(fabsf(h2f(v.x & 0xFFFFu)), fabsf(h2f(v.x >> 16))),
                 fmaxf(fabsf(h2f(v.y & 0xFFFFu)), fabsf(h2f(v.y >> 16))));
}

template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_f(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, ROW_MASK, 0xF, true));
}
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ int dpp_i(int v) {
    return __builtin_amdgcn_update_dpp(0, v, CTRL, ROW_MASK, 0xF, true);
}

// Sum over the 64 lanes of a wavefront in a fixed order (row shifts 1, 2, 4, 8,
// then row broadcasts 15 and 31); the total is in lane 63.
__device__ __forceinline__ float wave_sum_f(float v) {
    v += dpp_f<0x111, 0xF>(v);
    v += dpp_f<0x112, 0xF>(v);
    v += dpp_f<0x114, 0xF>(v);
    v += dpp_f<0x118, 0xF>(v);
    v += dpp_f<0x142, 0xA>(v);
    v += dpp_f<0x143, 0xC>(v);
    return v;
}
__device__ __forceinline__ int wave_sum_i(int v) {
    v += dpp_i<0x111, 0xF>(v);
    v += dpp_i<0x112, 0xF>(v);
    v += dpp_i<0x114, 0xF>(v);
    v += dpp_i<0x118, 0xF>(v);
    v += dpp_i<0x142, 0xA>(v);
    v += dpp_i<0x143, 0xC>(v);
    return v;
}
// v(l) + v(l ^ OFF) for OFF = 16 or 32 in every lane, by the gfx950 lane-swap
// instructions (v_permlane16_swap_b32 exchanges the odd 16-lane rows of one register
// with the even rows of another, v_permlane32_swap_b32 the two halves): vector ALU
// work, no LDS round trip as a shuffle through ds_bpermute has.  Both lanes of a pair
// add the lower lane's value and the upper lane's in that order (identical bits).
template <int OFF>
__device__ __forceinline__ uint32_t xor_swap_pair(uint32_t v, uint32_t *hi) {
    static_assert(OFF == 16 || OFF == 32, "lane-swap distance");
    if constexpr (OFF == 16) {
        const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
        *hi = r[1];
        return r[0];
    } else {
        const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
        *hi = r[1];
        return r[0];
    }
}
template <int OFF>
__device__ __forceinline__ int xor_sum_i(int v) {
    uint32_t hi;
    const uint32_t lo = xor_swap_pair<OFF>((uint32_t)v, &hi);
    return (int)lo + (int)hi;
}
template <int OFF>
__device__ __forceinline__ float xor_sum_f(float v) {
    uint32_t hi;
    const uint32_t lo = xor_swap_pair<OFF>(__float_as_uint(v), &hi);
    return __uint_as_float(lo) + __uint_as_float(hi);
}

// Lane-wise maximum of two packed unsigned 16-bit pairs (v_pk_max_u16); on the bits of
// FP16 magnitudes (sign cleared) it is the maximum magnitude of finite values.
__device__ __forceinline__ uint32_t max_u16x2(uint32_t a, uint32_t b) {
    typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t,
                              __builtin_elementwise_max(__builtin_bit_cast(u16x2, a), __builtin_bit_cast(u16x2, b)));
}

// Maximum over the 64 lanes of an unsigned value (FP16 magnitude bits compare as
// their values); in lane 63.
__device__ __forceinline__ uint32_t wave_max_u(uint32_t v) {
    v = max(v, (uint32_t)dpp_i<0x111, 0xF>((int)v));
    v = max(v, (uint32_t)dpp_i<0x112, 0xF>((int)v));
    v = max(v, (uint32_t)dpp_i<0x114, 0xF>((int)v));
    v = max(v, (uint32_t)dpp_i<0x118, 0xF>((int)v));
    v = max(v, (uint32_t)dpp_i<0x142, 0xA>((int)v));
    v = max(v, (uint32_t)dpp_i<0x143, 0xC>((int)v));
    return v;
}

// Largest FP16 magnitude bits of the 4 activations in v (as an unsigned value).
__device__ __forceinline__ uint32_t absmax4_bits(uint2 v) {
    const uint32_t m = max_u16x2(v.x & 0x7FFF7FFFu, v.y & 0x7FFF7FFFu);
    return max(m & 0xFFFFu, m >> 16);
}

// Maximum over the 64 lanes (any order gives the same result); in lane 63.
__device__ __forceinline__ float wave_max(float v) {
    v = fmaxf(v, dpp_f<0x111, 0xF>(v));
    v = fmaxf(v, dpp_f<0x112, 0xF>(v));
    v = fmaxf(v, dpp_f<0x114, 0xF>(v));
    v = fmaxf(v, dpp_f<0x118, 0xF>(v));
    v = fmaxf(v, dpp_f<0x142, 0xA>(v));
    v = fmaxf(v, dpp_f<0x143, 0xC>(v));
    return v;
}

// (byte B of w) & 0x3C: a 4-bit index pre-shifted left by 2 becomes an INT32
// table offset in one VALU op (SDWA byte select).
template <int B>
__device__ __forceinline__ uint32_t idx4(uint32_t w) {
    uint32_t r;
    if constexpr (B == 0)
        asm("v_and_b32_sdwa %0, 60, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_0"
            : "=v"(r) : "v"(w));
    else if constexpr (B == 1)
        asm("v_and_b32_sdwa %0, 60, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_1"
            : "=v"(r) : "v"(w));
    else if constexpr (B == 2)
        asm("v_and_b32_sdwa %0, 60, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_2"
            : "=v"(r) : "v"(w));
    else
        asm("v_and_b32_sdwa %0, 60, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_3"
            : "=v"(r) : "v"(w));
    return r;
}


// Signed 16-entry tables staged in LDS (entry s i = (s ? -1 : 1) T[i], Eq. 4-5)
// for the 32 four-activation groups of a 128-block: INT16 entries on the INT8 path
// (exact, |entry| <= 508), INT32 fixed point (FP16 entry x 2^20) on the FP path.
// Blocks are padded by one group table, so the tables of two consecutive blocks
// at the same group sit in different LDS banks.
template <bool INT8>
struct Tab {
    static constexpr int E = INT8 ? 2 : 4;       // bytes per entry
    // bytes per group table: the INT16 tables (32 bytes) are padded to 48 so that one
    // 16-byte store per lane of 16 consecutive groups covers 64 different LDS banks
    static constexpr int G = INT8 ? 48 : 16 * E;
    static constexpr int BLK = (GPB + 1) * G;    // bytes per 128-block
};

// (byte B of w) & MASK, one VALU op (SDWA byte select); with w pre-shifted so a
// 4-bit index lands at bit 1 (INT16 tables, MASK 30) or bit 2 (INT32, MASK 60)
// this is the byte offset of the entry.
template <int B, bool INT8>
__device__ __forceinline__ uint32_t idx_off(uint32_t w) {
    if constexpr (!INT8) return idx4<B>(w);
    uint32_t r;
    if constexpr (B == 0)
        asm("v_and_b32_sdwa %0, 30, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_0"
            : "=v"(r) : "v"(w));
    else if constexpr (B == 1)
        asm("v_and_b32_sdwa %0, 30, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_1"
            : "=v"(r) : "v"(w));
    else if constexpr (B == 2)
        asm("v_and_b32_sdwa %0, 30, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_2"
            : "=v"(r) : "v"(w));
    else
        asm("v_and_b32_sdwa %0, 30, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_3"
            : "=v"(r) : "v"(w));
    return r;
}

// One table entry: ds_read_i16 (sign-extended) or ds_read_b32.
template <bool INT8>
__device__ __forceinline__ int lds_entry(const char *base, uint32_t off) {
    if constexpr (INT8) return (int)*(const int16_t *)(base + off);
    return *(const int *)(base + off);
}

// base + (byte B of x), one VALU op (SDWA byte select).
template <int B>
__device__ __forceinline__ uint32_t add_byte(uint32_t base, uint32_t x) {
    uint32_t r;
    if constexpr (B == 0)
        asm("v_add_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_0"
            : "=v"(r) : "v"(base), "v"(x));
    else if constexpr (B == 1)
        asm("v_add_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_1"
            : "=v"(r) : "v"(base), "v"(x));
    else if constexpr (B == 2)
        asm("v_add_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_2"
            : "=v"(r) : "v"(base), "v"(x));
    else
        asm("v_add_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_3"
            : "=v"(r) : "v"(base), "v"(x));
    return r;
}

// Sum of the 32 entries addressed by one 16-byte plane word (the 4-bit indices of
// one 128-block, index i at bits 4 (i % 8) of 32-bit word i / 8) in the signed
// tables of that block (layout Tab<INT8>), which start at byte `base` of F.  A
// lookup is one SDWA byte-add, one LDS read and half a v_add3_u32.  On the FP path
// entries are below 2^22 in magnitude, so sum_t 2^t (word sum of plane t) stays
// below 15 * 32 * 2^22 < 2^31.
template <bool INT8>
__device__ __forceinline__ int lookup_word(const char *F, uint32_t base, uint4 w) {
    constexpr int GS = Tab<INT8>::G;
    constexpr uint32_t MASK = INT8 ? 0x1E1E1E1Eu : 0x3C3C3C3Cu;
    const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
    int acc = 0;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
        const uint32_t lo = (INT8 ? wd[d] << 1 : wd[d] << 2) & MASK, hi = (INT8 ? wd[d] >> 3 : wd[d] >> 2) & MASK;
        const char *Fg = F + d * 8 * GS;
        acc += lds_entry<INT8>(Fg + 0 * GS, add_byte<0>(base, lo)) + lds_entry<INT8>(Fg + 1 * GS, add_byte<0>(base, hi));
        acc += lds_entry<INT8>(Fg + 2 * GS, add_byte<1>(base, lo)) + lds_entry<INT8>(Fg + 3 * GS, add_byte<1>(base, hi));
        acc += lds_entry<INT8>(Fg + 4 * GS, add_byte<2>(base, lo)) + lds_entry<INT8>(Fg + 5 * GS, add_byte<2>(base, hi));
        acc += lds_entry<INT8>(Fg + 6 * GS, add_byte<3>(base, lo)) + lds_entry<INT8>(Fg + 7 * GS, add_byte<3>(base, hi));
    }
    return acc;
}

typedef short short2_v __attribute__((ext_vector_type(2)));

// Negation of two packed INT16 values (one v_pk_sub_i16).
__device__ __forceinline__ uint32_t neg_i16x2(uint32_t x) {
    short2_v v = __builtin_bit_cast(short2_v, x);
    v = -v;
    return __builtin_bit_cast(uint32_t, v);
}

// Stores quarter qr (entries 4 qr .. 4 qr + 3) of the signed table of group g of
// the staged block `blk`, from half (qr & 1) of its 8-entry half table (4 FP16 or
// INT16 values): quarters 0, 1 are T[0..3], T[4..7]; quarters 2, 3 their negation.
// INT8-quantized tables (TQ, FP path): h holds the 4 INT8 codes of that half and the
// table's FP32 scale; the staged entry is round(code x scale x 2^20).
template <bool INT8, bool TQ = false>
__device__ __forceinline__ void store_quarter(char *F, int blk, int g, int qr, uint2 h) {
    char *dst = F + blk * Tab<INT8>::BLK + g * Tab<INT8>::G + qr * 4 * Tab<INT8>::E;
    if constexpr (INT8) {
        if (qr >= 2) h = make_uint2(neg_i16x2(h.x), neg_i16x2(h.y));
        *(uint2 *)dst = h;
    } else if constexpr (TQ) {
        const float f = __uint_as_float(h.y) * (qr >= 2 ? -(float)(1 << FIX_SHIFT) : (float)(1 << FIX_SHIFT));
        *(int4 *)dst = make_int4((int)rintf((float)(int8_t)(h.x & 0xFFu) * f),
                                 (int)rintf((float)(int8_t)((h.x >> 8) & 0xFFu) * f),
                                 (int)rintf((float)(int8_t)((h.x >> 16) & 0xFFu) * f),
                                 (int)rintf((float)(int8_t)(h.x >> 24) * f));
    } else {
        const float f = qr >= 2 ? -(float)(1 << FIX_SHIFT) : (float)(1 << FIX_SHIFT);
        *(int4 *)dst = make_int4((int)rintf(h2f(h.x & 0xFFFFu) * f), (int)rintf(h2f(h.x >> 16) * f),
                                 (int)rintf(h2f(h.y & 0xFFFFu) * f), (int)rintf(h2f(h.y >> 16) * f));
    }
}

// Half `half` (entries 4 half .. + 3) of the half table of table group rg = m J + j:
// 4 FP16 / INT16 entries, or (TQ) the 4 INT8 codes and the table's scale bits.
template <bool TQ>
__device__ __forceinline__ uint2 load_quarter(const LutParams &p, int64_t rg, int half) {
    if constexpr (TQ) return make_uint2(((const uint32_t *)p.T)[2 * rg + half], __float_as_uint(p.tsc[rg]));
    return ((const uint2 *)(p.T + rg))[half];
}

// Reinterpreted scale and zero (Eq. 2) of quantization group q, column n.
struct SZ {
    float sp, zp;
};

// Raw metadata words of quantization group q, column n (FP16 s and z, or the two
// FP32 per-tensor values).  Branch-free, and every load is a vector load (the
// index is kept in a VGPR): scalar loads share the completion counter of LDS
// reads and would serialize them.
__device__ __forceinline__ uint2 load_meta_words(const LutParams &p, int q, int64_t n) {
    int64_t idx = p.per_tensor ? 0 : (int64_t)q * p.N_pad + n;
    asm volatile("" : "+v"(idx));
    const uint32_t *mw = (const uint32_t *)p.meta;
    return make_uint2(mw[idx], mw[idx + (p.per_tensor ? 1 : 0)]);
}

// Reinterpreted scale and zero (Eq. 2) from the raw metadata words.
__device__ __forceinline__ SZ decode_sz(const LutParams &p, uint2 mw) {
    const float s = p.per_tensor ? __uint_as_float(mw.x) : h2f(mw.x & 0xFFFFu);
    const float z = p.per_tensor ? __uint_as_float(mw.y) : h2f(mw.x >> 16);
    SZ r;
    r.sp = p.cs * s;
    r.zp = fmaf(p.cz, z, p.c0);
    return r;
}

// Epilogue operands of one 128-block kb and column n, as raw loads that can be
// issued long before they are used: the metadata word(s) of the block's
// quantization group and the group's activation sum S[m][q] (the zero-point term
// is applied by the group's first block only, see blk_epilogue).  Nothing here
// uses a loaded value, so no wait is placed until blk_epilogue.
struct BlkMeta {
    uint32_t m0, m1;
    float s;
};

__device__ __forceinline__ BlkMeta load_blk_meta(const LutParams &p, int64_t kb, int64_t m, int64_t n) {
    const int q = (int)(((float)kb + 0.5f) * p.inv_kpg);
    int64_t idx = p.per_tensor ? 0 : (int64_t)q * p.N_pad + n;
    asm volatile("" : "+v"(idx));
    const uint32_t *mw = (const uint32_t *)p.meta;
    BlkMeta b;
    b.m0 = mw[idx];
    b.m1 = mw[idx + (p.per_tensor ? 1 : 0)];
    b.s = ((const float *)p.S)[lane_value(m * p.Q + q)];
    return b;
}

// (s'/2^FIX_SHIFT, s' z' S or 0) of block kb from its raw operands (Eq. 2-3).
__device__ __forceinline__ float2 blk_epilogue(const LutParams &p, const BlkMeta &b, int64_t kb) {
    const int q = (int)(((float)kb + 0.5f) * p.inv_kpg);
    const float s = p.per_tensor ? __uint_as_float(b.m0) : h2f(b.m0 & 0xFFFFu);
    const float z = p.per_tensor ? __uint_as_float(b.m1) : h2f(b.m0 >> 16);
    const float sp = p.cs * s, zp = fmaf(p.cz, z, p.c0);
    return make_float2(sp * (1.0f / (float)(1 << FIX_SHIFT)), kb == (int64_t)q * p.kpg ? sp * zp * b.s : 0.f);
}

// Operands of the output epilogue of (m, n): the per-token factor t[m], the INT8
// path's weight scale, the previous output when accumulating, and the ternary
// group sum S[m][0] (added by the first K split only).  Loaded ahead of the main
// loop as raw words, so that their memory latency overlaps the lookups instead of
// following them, and decoded by store_out; every load is a vector load.
struct Epi {
    float tok;
    uint32_t sw;    // weight scale word: FP32 bits (per tensor) or FP16 s in the low half (per channel)
    uint32_t prev;  // previous output bits (INT32, FP32, or FP16 in the low half)
    int s0;
};

template <bool INT8>
__device__ __forceinline__ Epi load_epi(const LutParams &p, int wfmt, int64_t m, int64_t n, bool first_split) {
    Epi e{1.f, 0x3F800000u, 0u, 0};
    if (n >= p.N) return e;
    const int64_t mv = lane_value(m), nv = lane_value(n), o = mv * p.N + nv;
    if (p.tok) e.tok = p.tok[mv];
    if (INT8) {
        e.sw = ((const uint32_t *)p.meta)[p.per_tensor ? lane_value(0) : nv];
        if (first_split && wfmt == LUTGEMM_WFMT_TERNARY) e.s0 = ((const int *)p.S)[mv * p.Q];
    }
    if (p.accumulate) {
        if (p.out_dtype == LUTGEMM_OUT_FP16)
            e.prev = ((const uint16_t *)p.out)[o];
        else
            e.prev = ((const uint32_t *)p.out)[o];
    }
    return e;
}

// Final value of output (m, n): scale, optional accumulate, dtype conversion.
// yi already includes the ternary group sum (Epi::s0).
template <bool INT8>
__device__ __forceinline__ void store_out(const LutParams &p, int wfmt, int64_t m, int64_t n, float yf, int yi,
                                          const Epi &e) {
    if (n >= p.N) return;
    const int64_t o = m * p.N + n;
    float v;
    if (INT8) {
        const int y = (wfmt == LUTGEMM_WFMT_TERNARY) ? (yi >> 1) : yi;  // (A + S) / 2 is exact
        if (p.out_dtype == LUTGEMM_OUT_INT32) {
            ((int *)p.out)[o] = p.accumulate ? y + (int)e.prev : y;
            return;
        }
        const float sw = p.per_tensor ? __uint_as_float(e.sw) : h2f(e.sw & 0xFFFFu);
        v = ((float)y * e.tok) * sw;
    } else {
        v = e.tok * yf;
    }
    if (p.accumulate) v += p.out_dtype == LUTGEMM_OUT_FP16 ? h2f(e.prev) : __uint_as_float(e.prev);
    if (p.out_dtype == LUTGEMM_OUT_FP32)
        ((float *)p.out)[o] = v;
    else
        ((__half *)p.out)[o] = __float2half_rn(v);
}

// Partial sums of row m, column n for splits s0 .. s0 + PB - 1 (indices past the
// last split clamped to it).  Unconditional loads, so all PB are in flight before
// the first is used (a load under a condition makes the compiler wait for it
// before issuing the next one).
template <int PB>
__device__ __forceinline__ void load_partials(const LutParams &p, int64_t m_alloc, int64_t m, int64_t n, int s0,
                                              float (&v)[PB]) {
    const float *src = p.part + m * p.N_pad + n;
    const int64_t stride = m_alloc * p.N_pad;
#pragma unroll
    for (int j = 0; j < PB; ++j) {
        const int sp = (s0 + j < p.splits) ? s0 + j : p.splits - 1;
        v[j] = src[(int64_t)sp * stride];
    }
}

// Adds the loaded partials of splits s0 .. in split order.
template <bool INT8, int PB>
__device__ __forceinline__ void add_partials(const LutParams &p, int s0, const float (&v)[PB], float &sf, int &si) {
#pragma unroll
    for (int j = 0; j < PB; ++j) {
        const bool in = s0 + j < p.splits;
        if (INT8)
            si += in ? __float_as_int(v[j]) : 0;
        else
            sf += in ? v[j] : 0.f;
    }
}

// Nontemporal 16-byte load (a streaming read that should not displace cached data):
// used for the packed weights, which every call reads exactly once.
__device__ __forceinline__ uint4 ld_nt(const uint4 *p) {
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
    const u32x4 v = __builtin_nontemporal_load((const u32x4 *)p);
    return make_uint4(v.x, v.y, v.z, v.w);
}

// Completes a K split inside the LUT kernel itself, with no second launch.  Every
// workgroup publishes its partial sum of (m, n) with an agent-coherent store (written
// through to memory), waits until all of its stores are acknowledged, and one lane
// counts the workgroup on the arrival counter of its column tile.  The workgroup
// that arrives last reads the partial sums of all splits back with agent-coherent
// loads, adds them in split order (so the result does not depend on the order of
// arrival), applies the output epilogue and re-arms the counter to 0 for the next
// call.  No fence instruction is needed: the partial stores are complete before the
// counter is touched, and the last workgroup's loads are issued after it has seen
// the count.  The counter is re-armed by an atomic subtraction whose returned value
// the last workgroup waits for, so the re-arm has been performed before the kernel
// ends: a launch that follows directly (also one with no memory fence in between, as
// between the kernel nodes of a graph) never finds the counter still at `splits`.
// Returns only after the output is stored (or at once for the others).
// Partials of split s, row m at part[(s M + m) N_pad + n]; split 0 includes the
// ternary group sum.
template <bool INT8>
__device__ __forceinline__ void split_complete(const LutParams &p, int wfmt, int64_t m, int64_t n, int split,
                                               float yf, int yi, uint32_t *counter, float tok = -1.f) {
    __shared__ int is_last;
    float *part = p.part + m * p.N_pad + n;
    const int64_t stride = p.M * p.N_pad;
    __hip_atomic_store(part + split * stride, INT8 ? __int_as_float(yi) : yf, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
    __builtin_amdgcn_s_waitcnt(0);  // every outstanding memory operation of this wave acknowledged
    tl_stamp(p, 3);
    __syncthreads();
    if (threadIdx.x == 0)
        is_last = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                  (uint32_t)(p.splits - 1);
    __syncthreads();
    tl_stamp(p, 4);
    if (!is_last) {
        tl_clear(p, 5);
        return;
    }
    // re-arm the counter (all `splits` arrivals have been counted), issued before the
    // partial loads so that its round trip overlaps theirs
    uint32_t rearmed = 0u;
    if (threadIdx.x == 0)
        rearmed = __hip_atomic_fetch_add(counter, 0u - (uint32_t)p.splits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    // every split's partial in one batch of loads (splits <= INKERNEL_MAX_SPLITS, indices
    // past the last split clamped to it), then the fixed-order sum
    float v[INKERNEL_MAX_SPLITS];
#pragma unroll
    for (int j = 0; j < INKERNEL_MAX_SPLITS; ++j) {
        const int sp = j < p.splits ? j : p.splits - 1;
        v[j] = __hip_atomic_load(part + sp * stride, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    Epi ep = load_epi<INT8>(p, wfmt, m, n, false);
    if (tok >= 0.f) ep.tok = tok;  // a token factor the calling kernel formed itself
    float sf = 0.f;
    int si = 0;
#pragma unroll
    for (int j = 0; j < INKERNEL_MAX_SPLITS; ++j) {
        if (INT8)
            si += j < p.splits ? __float_as_int(v[j]) : 0;
        else
            sf += j < p.splits ? v[j] : 0.f;
    }
    tl_stamp(p, 5);
    store_out<INT8>(p, wfmt, m, n, sf, si, ep);
    // the re-arm's returned value is needed here: the wave waits until it is performed
    asm volatile("; counter re-armed from %0" ::"v"(rearmed));
}

// Completes a K split by one 64-bit atomic per output, summing exactly.  A split's
// partial sum v is an integer: the INT32 sum of the INT8 path; on the FP16 path with
// one scale per column or tensor the integer sum of the split's fixed-point table
// entries (every block shares s', so the output is s' 2^-FIX_SHIFT times the total
// minus the zero-point term: sx, sy); otherwise the FP32 partial sum in fixed point,
// v = rint(partial 2^-E) with the column's exponent E (|v| < 2^BND_BITS, see
// pack_bound_kernel), the output 2^E times the total.  The zeroed word of (m, n)
// accumulates c 2^57 + V (c arrivals, V the signed sum so far, |V| < 2^56): each split
// adds 2^57 + v with one agent-coherent atomic and gets the previous word back, and
// the split that sees c = splits - 1 holds the exact total, which integer addition
// gives whatever the order of arrival.  That split applies the epilogue (operands
// loaded before the atomic, so only the atomic's round trip precedes the store) and
// clears the word, waiting for the clear's return so that it is performed before the
// kernel ends.  E = INT_MIN selects the (sx, sy) form.
// The two halves of split_complete_exact, so that a kernel with several outputs per
// lane can have all its atomics in flight before it looks at any return: exact_add
// issues the atomic and returns the previous word; exact_finish decides, for the
// split that completed the count, the epilogue and the clear (returning the clear's
// result, which the caller must consume before the kernel ends; 0 for the others).
__device__ __forceinline__ unsigned long long exact_add(const LutParams &p, int64_t m, int64_t n, long long v) {
    return __hip_atomic_fetch_add(p.acc64 + m * p.N_pad + n, (1ull << 57) + (unsigned long long)v, __ATOMIC_RELAXED,
                                  __HIP_MEMORY_SCOPE_AGENT);
}

template <bool INT8>
__device__ __forceinline__ unsigned long long exact_finish(const LutParams &p, int wfmt, int64_t m, int64_t n,
                                                           unsigned long long old, long long v, float sx, float sy,
                                                           int E, const Epi &ep) {
    const unsigned long long c = (old + (1ull << 56)) >> 57;
    if (c != (unsigned long long)(p.splits - 1)) return 0ull;
    const unsigned long long cleared =
        __hip_atomic_exchange(p.acc64 + m * p.N_pad + n, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const long long tot = (long long)(old - (c << 57)) + v;
    float yf = 0.f;
    if constexpr (!INT8) yf = E == INT_MIN ? fmaf(sx, (float)tot, -sy) : ldexpf((float)tot, E);
    store_out<INT8>(p, wfmt, m, n, yf, (int)tot, ep);
    return cleared;
}

template <bool INT8>
__device__ __forceinline__ void split_complete_exact(const LutParams &p, int wfmt, int64_t m, int64_t n, long long v,
                                                     float sx, float sy, int E, const Epi &ep) {
    const unsigned long long cleared = exact_finish<INT8>(p, wfmt, m, n, exact_add(p, m, n, v), v, sx, sy, E, ep);
    asm volatile("; exact split word cleared: %0" ::"v"(cleared));
}

// The fixed-point value rint(x 2^-E) of an FP32 partial sum (|x 2^-E| < 2^BND_BITS).
__device__ __forceinline__ long long to_fixed(float x, int E) { return (long long)rintf(ldexpf(x, -E)); }

}  // namespace lutgemm
