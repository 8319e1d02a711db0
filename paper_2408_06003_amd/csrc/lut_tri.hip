// Ternary LUT mpGEMM with three weights per 5-bit code (LUT Tensor Core, Section 5:
// a LUT needs 5 bits for 3 ternary weights where a multiply-accumulate datapath
// needs 6; tables and their symmetry as in Section 3.1, Eq. 4-5, with
// three-valued instead of one-bit weights).
//
// Tables.  For 3 activations x0..x2 the 27 patterns w in {-1,0,1}^3 give the dot
// products sum_e w_e x_e.  Pattern v (base-3 digits w_e + 1, first activation
// most significant) and 26 - v are negations of each other and v = 13 is zero,
// so 14 entries T[i] (pattern 13 + i) are stored and a code is a sign bit plus a
// 4-bit index (packing in lutgemm_internal.h).  In LDS each triple gets a signed
// table of 32 two-byte slots, slot i = T[i] and slot 16 + i = -T[i]: exact INT16
// entries on the INT8 path (|T| <= 381, stored biased), FP16 entries on the FP
// path (the precompute's rounding), so a lookup is one SDWA byte-add (slot
// offset), one LDS read and 3/4 of an add (INT8: pairs of SDWA word adds) or one
// v_fma_mix_f32 (FP).  One lookup covers 3 weights, against 4 / (2 planes) = 2 for
// the bit-serial ternary format.
//
// gfx950 mapping.  A workgroup of NW wavefronts owns 16 columns and one token over
// the whole K; the 64 lanes of a wavefront are (column, K slice): 16 columns x 4
// slices, and K slice sigma of the workgroup takes 96-blocks sigma, sigma + S, ...
// (S = 4 NW slices).  Per chunk of S blocks every lane builds (fused) or expands
// (from precomputed tables) the signed tables of 2 triples, consecutive lanes
// taking consecutive triples.  Triple tables sit 80 bytes apart, so the 16-byte
// stores of 8 consecutive lanes cover all 8 16-byte bank groups of a 128-byte bank
// row (conflict-free), and blocks are 64 mod 128 bytes apart, so the 4 slices of a
// wavefront read their tables from two (32 banks) or four (64 banks) disjoint
// halves or quarters of the banks.  Slices are summed by a fixed butterfly, wavefronts in
// order, so results are bitwise reproducible.  Every workgroup of the fused
// variant reads its token (8 KiB at K = 4096, from L2) and performs the same FP32
// quantization / scaling as the precompute kernel, so both variants produce the
// same tables and the same result bits.
#include "lut_common.h"
#include "tri_table.h"

namespace lutgemm {

constexpr int TRI_SW = 4;                          // K slices per wavefront
constexpr int TRI_CW = 64 / TRI_SW;                // columns per workgroup
constexpr int TRI_TAB = 64;                        // bytes of one signed triple table (32 x 2 B)
constexpr int TRI_TS = 80;                         // LDS stride of the triple tables of a block
constexpr int TRI_BLK = TPB * TRI_TS + 64;         // LDS bytes per 96-block (= 64 mod 128)

template <bool INT8>
__device__ __forceinline__ uint32_t neg2(uint32_t x) {
    if constexpr (INT8) return neg_i16x2(x);
    return x ^ 0x80008000u;  // FP16: flip both signs (exact)
}

// Writes the signed table of one triple from its 16 stored entries (8 words).  INT8
// path: entries are kept biased by 2^15 (e + 32768 as an unsigned 16-bit value,
// the sign bit flipped), so lookups add zero-extended values and the bias is
// removed once at the end; negating a biased value is the plain 16-bit negation.
template <bool INT8>
__device__ __forceinline__ void store_tri(char *dst, uint4 lo, uint4 hi) {
    if constexpr (INT8) {
        lo = make_uint4(lo.x ^ 0x80008000u, lo.y ^ 0x80008000u, lo.z ^ 0x80008000u, lo.w ^ 0x80008000u);
        hi = make_uint4(hi.x ^ 0x80008000u, hi.y ^ 0x80008000u, hi.z ^ 0x80008000u, hi.w ^ 0x80008000u);
    }
    *(uint4 *)dst = lo;
    *(uint4 *)(dst + 16) = hi;
    *(uint4 *)(dst + 32) = make_uint4(neg2<INT8>(lo.x), neg2<INT8>(lo.y), neg2<INT8>(lo.z), neg2<INT8>(lo.w));
    *(uint4 *)(dst + 48) = make_uint4(neg2<INT8>(hi.x), neg2<INT8>(hi.y), neg2<INT8>(hi.z), neg2<INT8>(hi.w));
}

// The 16 stored entries of the triple x0..x2 (14 patterns and two zeros, formed
// by tri_table14), as 16-bit words: exact INT16 from the quantized integers, or
// FP16 (round to nearest even) from the FP32 sums.
template <bool INT8>
__device__ __forceinline__ void tri_entries(float x0, float x1, float x2, uint4 &lo, uint4 &hi) {
    uint32_t h[16];
    if constexpr (INT8) {
        int e[14];
        tri_table14<int>((int)x0, (int)x1, (int)x2, e);
#pragma unroll
        for (int i = 0; i < 14; ++i) h[i] = (uint32_t)e[i] & 0xFFFFu;
    } else {
        float e[14];
        tri_table14<float>(x0, x1, x2, e);
#pragma unroll
        for (int i = 0; i < 14; ++i) h[i] = (uint32_t)__half_as_ushort(__float2half_rn(e[i]));
    }
    h[14] = h[15] = 0u;
    uint32_t w[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) w[i] = h[2 * i] | (h[2 * i + 1] << 16);
    lo = make_uint4(w[0], w[1], w[2], w[3]);
    hi = make_uint4(w[4], w[5], w[6], w[7]);
}

// Slot byte offsets (2 x (16 sign + index)) of the 8 codes of index word d, as two
// words of 4 bytes: `lo` for the codes in the low nibbles (triples 8d + 2k), `hi`
// for the high nibbles (8d + 2k + 1).  The sign of triple 8d + 2k + h sits at bit
// 8k + 2d + h of the sign word and is moved to bit 5 of byte k.
template <int D>
__device__ __forceinline__ void slot_offsets(uint32_t wd, uint32_t sg, uint32_t &lo, uint32_t &hi) {
    constexpr int X0 = 2 * D, X1 = 2 * D + 1;
    const uint32_t s0 = X0 <= 5 ? sg << (5 - X0) : sg >> (X0 - 5);
    const uint32_t s1 = X1 <= 5 ? sg << (5 - X1) : sg >> (X1 - 5);
    lo = ((wd << 1) & 0x1E1E1E1Eu) | (s0 & 0x20202020u);
    hi = ((wd >> 3) & 0x1E1E1E1Eu) | (s1 & 0x20202020u);
}

// The 8 lookups of one index word d (triples 8d .. 8d + 7 of the block whose tables
// start at F + base).  INT8 path: the biased entries are zero-extended 16-bit
// reads summed in pairs (SDWA word adds); FP path: each FP16 entry is added into
// the FP32 sum with one v_fma_mix_f32 (entry x 1.0 + sum).
template <bool INT8>
__device__ __forceinline__ void tri_lookup8(uint32_t &ai, float &af, const char *Fd, uint32_t base, uint32_t lo,
                                            uint32_t hi) {
    uint16_t h[8];
    h[0] = *(const uint16_t *)(Fd + 0 * TRI_TS + add_byte<0>(base, lo));
    h[1] = *(const uint16_t *)(Fd + 1 * TRI_TS + add_byte<0>(base, hi));
    h[2] = *(const uint16_t *)(Fd + 2 * TRI_TS + add_byte<1>(base, lo));
    h[3] = *(const uint16_t *)(Fd + 3 * TRI_TS + add_byte<1>(base, hi));
    h[4] = *(const uint16_t *)(Fd + 4 * TRI_TS + add_byte<2>(base, lo));
    h[5] = *(const uint16_t *)(Fd + 5 * TRI_TS + add_byte<2>(base, hi));
    h[6] = *(const uint16_t *)(Fd + 6 * TRI_TS + add_byte<3>(base, lo));
    h[7] = *(const uint16_t *)(Fd + 7 * TRI_TS + add_byte<3>(base, hi));
    if constexpr (INT8) {
        uint32_t pr[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t x = h[2 * i], y = h[2 * i + 1];
            asm("v_add_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_0 src1_sel:WORD_0"
                : "=v"(pr[i]) : "v"(x), "v"(y));
        }
        ai += pr[0] + pr[1];
        ai += pr[2] + pr[3];
    } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const uint32_t x = h[i];
            asm("v_fma_mix_f32 %0, %1, 1.0, %0 op_sel_hi:[1,0,0]" : "+v"(af) : "v"(x));
        }
    }
}

template <bool INT8, bool FUSED, int NW>
__global__ __launch_bounds__(64 * NW) void lut_tri_kernel(LutParams p, int wfmt, uint32_t n_tiles) {
    constexpr int NT = 64 * NW;
    constexpr int S = NW * TRI_SW;    // 96-blocks per chunk
    constexpr int TPT = S * TPB / NT;  // triples built per thread and chunk
    static_assert(TPT == 2, "two triples (6 activations, 3 words) per thread and chunk");
    __shared__ __attribute__((aligned(16))) char F[S * TRI_BLK];
    __shared__ float redf[NW][TRI_CW];
    __shared__ int redi[NW][TRI_CW];
    __shared__ float wmax[NW];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int c = lane & (TRI_CW - 1), sl = lane >> 4;
    const int sigma = wave * TRI_SW + sl;
    const int64_t m = blockIdx.x / n_tiles;
    const int64_t n = (int64_t)(blockIdx.x % n_tiles) * TRI_CW + c;  // < N_pad
    // this thread's two triples of every chunk: g = tid and tid + NT, in block g / 32
    int tb[2], tj[2];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
        tb[r] = (tid + NT * r) / TPB;
        tj[r] = (tid + NT * r) % TPB;
    }

    // epilogue operands first (their latency overlaps everything below)
    const Epi ep = load_epi<INT8>(p, wfmt, m, n, false);
    const uint32_t swf = ((const uint32_t *)p.meta)[p.per_tensor ? lane_value(0) : lane_value(n)];

    // weights of the lane's block in chunk kc (clamped, unconditional)
    auto load_w = [&](int64_t kc, int nkb, uint4 &w, uint32_t &sg) {
        const int64_t kb = kc + (sigma < nkb ? sigma : nkb - 1);
        w = p.planes[kb * p.N_pad + n];
        sg = p.sgn[kb * p.N_pad + n];
    };

    const uint16_t *arow = FUSED ? p.act + m * p.K : nullptr;
    const uint32_t *a32 = (const uint32_t *)arow;
    const int64_t kw = p.K / 2;  // activation words of the token
    // the 2 activation words holding triple g of chunk kc (halves 3g .. 3g + 2 start
    // in the low half of the first word when g is even, in its high half when odd;
    // words past the token are 0)
    auto load_a = [&](int64_t kc, uint32_t (&aw)[2][2]) {
#pragma unroll
        for (int r = 0; r < 2; ++r) {
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int64_t q = kc * (TBLK / 2) + ((3 * (tid + NT * r)) >> 1) + i;
                const uint32_t v = a32[q < kw ? q : kw - 1];
                aw[r][i] = q < kw ? v : 0u;
            }
        }
    };
    // the table words of this thread's triples in chunk kc (table-fed)
    auto load_t = [&](int64_t kc, int nkb, uint4 (&tw)[2][2]) {
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int64_t j = (kc + (tb[r] < nkb ? tb[r] : nkb - 1)) * TPB + tj[r];
            const uint4 *src = p.T + 2 * (m * p.J + j);
            tw[r][0] = src[0];
            tw[r][1] = src[1];
        }
    };
    // activations e = 0..2 of triple r from its two words (tid odd shifts by a half)
    auto act3 = [&](const uint32_t (&aw)[2][2], int r, int e) -> uint32_t {
        const uint64_t v = ((uint64_t)aw[r][1] << 32) | aw[r][0];
        const int sh = 16 * (((tid + NT * r) & 1) + e);
        return (uint32_t)(v >> sh) & 0xFFFFu;
    };

    float scale = 0.f;
    uint32_t aw[2][2] = {{0u, 0u}, {0u, 0u}};
    uint4 tw[2][2];
    uint4 w;
    uint32_t sg;
    int nkb = (int)(p.KB < S ? p.KB : S);
    if constexpr (FUSED) {
        load_a(0, aw);
        load_w(0, nkb, w, sg);
        // amax of the whole token: the first chunk from registers, the rest from memory
        float amax = 0.f;
#pragma unroll
        for (int r = 0; r < 2; ++r)
#pragma unroll
            for (int i = 0; i < 2; ++i)
                amax = fmaxf(amax, fmaxf(fabsf(h2f(aw[r][i] & 0xFFFFu)), fabsf(h2f(aw[r][i] >> 16))));
        for (int64_t q = (int64_t)S * (TBLK / 2) + tid; q < kw; q += NT)
            amax = fmaxf(amax, fmaxf(fabsf(h2f(a32[q] & 0xFFFFu)), fabsf(h2f(a32[q] >> 16))));
        amax = wave_max(amax);
        if (lane == 63) wmax[wave] = amax;
        lds_barrier();
        amax = wmax[0];
#pragma unroll
        for (int v = 1; v < NW; ++v) amax = fmaxf(amax, wmax[v]);
        // same FP32 operations as the precompute kernel
        if (INT8) {
            scale = amax == 0.f ? 0.f : __fdiv_rn(127.0f, amax);
        } else if (amax == 0.f) {
            scale = 1.f;
        } else {
            int e;
            (void)frexpf(amax, &e);
            scale = ldexpf(1.f, -e);
        }
    } else {
        load_t(0, nkb, tw);
        load_w(0, nkb, w, sg);
    }

    uint32_t ai = 0u;  // INT8 path: biased sum (wraps mod 2^32, exact after the bias is removed)
    uint32_t nlook = 0u;
    float af = 0.f;
    for (int64_t kc = 0; kc < p.KB; kc += S) {
        nkb = (int)((p.KB - kc) < S ? (p.KB - kc) : S);
        if (kc > 0) {
            lds_barrier();  // every lookup of the previous chunk is done
            if constexpr (FUSED)
                load_a(kc, aw);
            else
                load_t(kc, nkb, tw);
            load_w(kc, nkb, w, sg);
        }
        // build or expand this thread's two triple tables
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            if (tb[r] < nkb) {
                char *dst = F + tb[r] * TRI_BLK + tj[r] * TRI_TS;
                if constexpr (FUSED) {
                    uint4 lo, hi;
                    tri_entries<INT8>(act_value<INT8>(act3(aw, r, 0), scale), act_value<INT8>(act3(aw, r, 1), scale),
                                      act_value<INT8>(act3(aw, r, 2), scale), lo, hi);
                    store_tri<INT8>(dst, lo, hi);
                } else {
                    store_tri<INT8>(dst, tw[r][0], tw[r][1]);
                }
            }
        }
        lds_barrier();
        if (sigma < nkb) {
            nlook += TPB;
            const uint32_t base = (uint32_t)(sigma * TRI_BLK);
            const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int d = 0; d < 4; ++d) {
                uint32_t lo, hi;
                if (d == 0) slot_offsets<0>(wd[0], sg, lo, hi);
                if (d == 1) slot_offsets<1>(wd[1], sg, lo, hi);
                if (d == 2) slot_offsets<2>(wd[2], sg, lo, hi);
                if (d == 3) slot_offsets<3>(wd[3], sg, lo, hi);
                tri_lookup8<INT8>(ai, af, F + (8 * d) * TRI_TS, base, lo, hi);
            }
        }
    }

    // slices of the wavefront (lanes c, c + 16, c + 32, c + 48), then wavefronts in order
    if (INT8) {
        int a = (int)(ai - 32768u * nlook);
        a = xor_sum_i<32>(xor_sum_i<16>(a));
        if (lane < TRI_CW) redi[wave][c] = a;
    } else {
        af = xor_sum_f<32>(xor_sum_f<16>(af));
        if (lane < TRI_CW) redf[wave][c] = af;
    }
    lds_barrier();
    if (wave == 0 && lane < TRI_CW) {
        int si = redi[0][c];
        float sf = redf[0][c];
#pragma unroll
        for (int v = 1; v < NW; ++v) {
            if (INT8)
                si += redi[v][c];
            else
                sf += redf[v][c];
        }
        Epi e = ep;
        if constexpr (FUSED) {
            // the per-token factor the precompute would have stored
            if (INT8) {
                // s_a = amax / 127, recomputed from the scale's inputs
                float amax = wmax[0];
#pragma unroll
                for (int v = 1; v < NW; ++v) amax = fmaxf(amax, wmax[v]);
                e.tok = amax == 0.f ? 0.f : __fdiv_rn(amax, 127.0f);
            } else {
                e.tok = 1.f / scale;  // 2^e, exact
            }
        }
        // FP path: the weight scale (per tensor FP32, per channel FP16), then t_m
        const float sw = p.per_tensor ? __uint_as_float(swf) : h2f(swf & 0xFFFFu);
        store_out<INT8>(p, wfmt, m, n, sf * sw, si, e);
    }
}

template <bool INT8, bool FUSED>
static void launch_tri_cfg(const LutParams &p, const Layout &L, hipStream_t s) {
    const uint32_t n_tiles = (uint32_t)((L.N + TRI_CW - 1) / TRI_CW);
    const dim3 grid((unsigned)(n_tiles * p.M));
    hipLaunchKernelGGL((lut_tri_kernel<INT8, FUSED, 12>), grid, dim3(64 * 12), 0, s, p, L.wfmt, n_tiles);
}

int launch_tri(const LutParams &p, const Layout &L, bool fused, void *stream) {
    hipStream_t s = (hipStream_t)stream;
    if (L.act == LUTGEMM_ACT_INT8) {
        if (fused) launch_tri_cfg<true, true>(p, L, s);
        else launch_tri_cfg<true, false>(p, L, s);
    } else {
        if (fused) launch_tri_cfg<false, true>(p, L, s);
        else launch_tri_cfg<false, false>(p, L, s);
    }
    return (int)hipGetLastError();
}

}  // namespace lutgemm
