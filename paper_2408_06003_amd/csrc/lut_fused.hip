// Single-token LUT mpGEMM with the table precompute fused into it on the consumer
// side (LUT Tensor Core, Section 3.1.1: the precompute is split out of the
// lookup so it can be fused; here it is fused into the lookup kernel itself).
//
// Each workgroup of the whole-K GEMV (lut_gemv.hip) reads the token's FP16
// activations instead of precomputed half tables and builds its signed 16-entry
// tables in LDS directly:
//   1. amax = max |a| over the whole token (every workgroup reads the token,
//      8 KiB at K = 4096, from L2); INT8 path: q = clamp(rint(a * (127 / amax)),
//      -127, 127) and s_a = amax / 127; FP path: the token is scaled by 2^-e with
//      amax = f 2^e, f in [0.5, 1).  Same FP32 operations as the precompute
//      operator, so the tables are bitwise the ones it would produce.
//   2. Per 4-activation group, the entries F[s i] = (s ? -1 : 1) T[i] of Eq. 4-5
//      (T[i] = -x0 + sum_{e=1..3} (bit (3-e) of i ? x_e : -x_e), rounded to FP16
//      on the FP path as in the stored tables): on the INT8 path one lane builds a
//      group's INT16 table from its 4 quantized activations; on the FP path the 4
//      lanes of a DPP quad hold the group's 4 activations, exchange them by quad
//      broadcasts and build one quarter (4 INT32 entries) each.
//   3. The activation sums: per 128-block S_kb on the FP path (zero-point term of
//      Eq. 3), per chunk on the INT8 path (ternary integer offset), by fixed-order
//      DPP sums over the lanes that built the tables.
// The weights of the chunk are requested right after the activations, so their
// memory latency overlaps the table build; lookups and epilogue are those of
// lut_gemv.hip.  The
// zero-point term is applied per 128-block: s'_q z'_q S_q = sum over the blocks
// of group q of s'_q z'_q S_kb.
#include "lut_common.h"

namespace lutgemm {

// Entries 4 qr .. 4 qr + 3 of the signed 16-entry table of x0..x3: quarter qr
// holds rows 4 (qr & 1) .. + 3 of the half table, negated when qr >= 2 (Eq. 4).
// Sums are formed in the order ((-x0 + (+-x1)) + (+-x2)) + (+-x3).
template <bool INT8>
__device__ __forceinline__ int4 quarter_entries(float x0, float x1, float x2, float x3, int qr) {
    const float b = -x0 + ((qr & 1) ? x1 : -x1);
    const float u0 = b + (-x2), u1 = b + x2;
    const float t[4] = {u0 + (-x3), u0 + x3, u1 + (-x3), u1 + x3};
    int v[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        if (INT8)
            v[i] = (int)t[i];  // |t| <= 508, exact
        else
            v[i] = (int)rintf(__half2float(__float2half_rn(t[i])) * (float)(1 << FIX_SHIFT));
        if (qr >= 2) v[i] = -v[i];
    }
    return make_int4(v[0], v[1], v[2], v[3]);
}

// Value of lane 4 (l / 4) + I for lane l (DPP quad_perm broadcast).
template <int I>
__device__ __forceinline__ int quad_bcast(int v) {
    return __builtin_amdgcn_mov_dpp(v, I * 0x55, 0xF, 0xF, false);
}

// The signed INT16 table of one group of quantized activations q0..q3 (INT8
// path): entries 0..7 are T[i] = -q0 + (+-q1) + (+-q2) + (+-q3) (bit 2 of i
// selects the sign of q1, bit 1 of q2, bit 0 of q3), entries 8..15 are -T[i];
// exact integers (|T| <= 508).  Written as two 16-byte LDS stores.
__device__ __forceinline__ void build_group_i16(char *dst, int q0, int q1, int q2, int q3) {
    const int b0 = -q0 - q1, b1 = -q0 + q1;
    const int c[4] = {b0 - q2, b0 + q2, b1 - q2, b1 + q2};
    // entries 2i, 2i + 1 = c_i -+ q3 as one packed INT16 add: (c_i, c_i) + (-q3, q3)
    const uint32_t d = __builtin_amdgcn_perm((uint32_t)q3, (uint32_t)-q3, 0x05040100u);
    uint32_t pw[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint32_t cc = __builtin_amdgcn_perm((uint32_t)c[i], (uint32_t)c[i], 0x05040100u);
        pw[i] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(short2_v, cc) + __builtin_bit_cast(short2_v, d));
    }
    *(uint4 *)dst = make_uint4(pw[0], pw[1], pw[2], pw[3]);
    *(uint4 *)(dst + 16) = make_uint4(neg_i16x2(pw[0]), neg_i16x2(pw[1]), neg_i16x2(pw[2]), neg_i16x2(pw[3]));
}

// The precompute's INT8 quantizer clamp(rint(a * scale), -127, 127) of FP16 half H of
// the word w, the product formed by one mixed-precision fma (FP16 operand read in
// place, one rounding, adding -0 leaves it unchanged), as act_value<true>.
template <int H>
__device__ __forceinline__ int quant8(uint32_t w, float scale) {
    float x;
    const uint32_t nz = 0x80000000u;  // -0.0f
    if constexpr (H == 0)
        asm("v_fma_mix_f32 %0, %1, %2, %3 op_sel_hi:[1,0,0]" : "=v"(x) : "v"(w), "v"(scale), "s"(nz));
    else
        asm("v_fma_mix_f32 %0, %1, %2, %3 op_sel:[1,0,0] op_sel_hi:[1,0,0]" : "=v"(x) : "v"(w), "v"(scale), "s"(nz));
    return (int)__builtin_amdgcn_fmed3f(rintf(x), -127.f, 127.f);
}

template <int BITS, int PW, int SW, int TW, int NW, bool INT8>
__global__ __launch_bounds__(64 * NW) void lut_fused_gemv_kernel(LutParams p, int wfmt) {
    constexpr int NT = 64 * NW;            // threads per workgroup
    constexpr int CW = 64 / (PW * SW);    // columns per workgroup
    constexpr int S = NW * SW;             // K slices per workgroup
    constexpr int CK = S * TW;             // 128-blocks per chunk
    constexpr int NPL = BITS / PW;         // bit-planes per lane
    // FP path: table quarters built per thread and chunk (one activation per lane
    // and round); INT8 path: whole group tables built per thread and chunk
    constexpr int QPT = CK * GPB * 4 / NT;
    constexpr int GPT = (CK * GPB + NT - 1) / NT;
    constexpr int BPR = NT / 128;          // 128-blocks covered by one round of quarters
    static_assert(QPT * NT == CK * GPB * 4 && NT % 128 == 0, "quarters divide evenly over the threads");
    static_assert(TW * NPL <= 4, "at most four prefetched weight words per lane");
    __shared__ __attribute__((aligned(16))) char F[CK * Tab<INT8>::BLK];
    __shared__ float redf[NW][CW];
    __shared__ int redi[NW][CW];
    __shared__ float hsf[QPT * NW];  // FP path: half-block activation sums, [round][wave]
    __shared__ int hsi[NW];          // INT8 path: activation sum of the K range, per wave
    __shared__ uint32_t wmax[NW];

    tl_stamp(p, 0);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: branches on it are scalar
    const int c = lane % CW;
    const int pl = (lane / CW) % PW;
    const int sl = lane / (CW * PW);
    const int sigma = wave * SW + sl;
    const int64_t n = (int64_t)blockIdx.x * CW + c;
    const int64_t m = blockIdx.z;
    const int split = blockIdx.y;
    const int64_t kbA = (int64_t)split * p.kbs;
    const int64_t kbB = (kbA + p.kbs < p.KB) ? kbA + p.kbs : p.KB;
    const uint16_t *a1 = p.act + m * p.K;
    const uint2 *a4 = (const uint2 *)a1;  // one 4-activation group per element
    const bool need_s = wfmt != LUTGEMM_WFMT_BINARY;   // binary weights have z' = 0

    // Chunk loads are unconditional (clamped indices, values past the chunk
    // ignored) and conditional loads are issued before them, so every wait the
    // compiler places counts exactly the loads after the one it waits for.
    uint4 w[TW][NPL];
    auto load_weights = [&](int64_t kc, int nkb) {
#pragma unroll
        for (int t = 0; t < TW; ++t) {
            const int kbl = sigma + t * S, kbc = kbl < nkb ? kbl : nkb - 1;
#pragma unroll
            for (int i = 0; i < NPL; ++i) w[t][i] = ld_nt(p.planes + ((kc + kbc) * BITS + pl * NPL + i) * p.N_pad + n);
        }
    };
    // FP path: lane e of a round holds activation e of the chunk, so the 4 lanes of a
    // quad hold the 4 activations of one group and build its 4 table quarters.
    // INT8 path: lane g of a round holds the 4 activations of group g.
    uint32_t av[INT8 ? 1 : QPT];
    uint2 ag[INT8 ? GPT : 1];
    auto load_acts = [&](int64_t kc, int nkb) {
        if constexpr (INT8) {
#pragma unroll
            for (int r = 0; r < GPT; ++r) {
                const int g = tid + NT * r, gc = g < nkb * GPB ? g : nkb * GPB - 1;
                const uint2 v = a4[kc * GPB + gc];
                ag[r] = g < nkb * GPB ? v : make_uint2(0u, 0u);
            }
        } else {
#pragma unroll
            for (int r = 0; r < QPT; ++r) {
                const int e = tid + NT * r, ec = e < nkb * KBLK ? e : nkb * KBLK - 1;
                const uint32_t v = a1[kc * KBLK + ec];
                av[r] = e < nkb * KBLK ? v : 0u;
            }
        }
    };

    // activations, then weights of the first chunk, then the epilogue operands.
    // Vector loads retire in issue order: the activation-max reduction waits only
    // for the activations, and the weights keep streaming in during the table build.
    Epi ep{};
    if (p.splits == 1) ep = load_epi<INT8>(p, wfmt, m, n, false);
    int nkb = (int)((kbB - kbA) < CK ? (kbB - kbA) : CK);
    load_acts(kbA, nkb);
    load_weights(kbA, nkb);

    // 1. amax of the whole token: the first chunk from registers, the rest from memory;
    // as FP16 magnitude bits (integer maxima: one DPP max per step of the reduction;
    // the same maximum for finite activations)
    uint32_t mbits = 0u;
    if constexpr (INT8) {
#pragma unroll
        for (int r = 0; r < GPT; ++r) mbits = max(mbits, absmax4_bits(ag[r]));
    } else {
#pragma unroll
        for (int r = 0; r < QPT; ++r) mbits = max(mbits, av[r] & 0x7FFFu);
    }
    const int64_t j0 = kbA * GPB, j1 = j0 + (int64_t)nkb * GPB;
    if (j1 - j0 < p.J) {  // the token extends past the first chunk (several chunks or a K split)
        for (int64_t j = tid; j < p.J; j += NT)
            if (j < j0 || j >= j1) mbits = max(mbits, absmax4_bits(a4[j]));
    }
    mbits = wave_max_u(mbits);
    if (lane == 63) wmax[wave] = mbits;
    lds_barrier();
    tl_stamp(p, 1);
    // the wavefront maxima, one per lane, reduced by DPP and broadcast from lane 63
    mbits = wave_max_u(lane < NW ? wmax[lane] : 0u);
    const float amax = h2f(__builtin_amdgcn_readlane(mbits, 63));
    // the table scale and the output factor t[m] now (off the tail of the kernel); the
    // factor only in the wavefront that applies the epilogue
    float scale, tok = 1.f;
    if (INT8) {
        scale = amax == 0.f ? 0.f : __fdiv_rn(127.0f, amax);
        if (wave == 0) {  // (a real branch: the other wavefronts skip the division)
            asm volatile("");
            tok = amax == 0.f ? 0.f : __fdiv_rn(amax, 127.0f);
        }
    } else if (amax == 0.f) {
        scale = 1.f;
        tok = 1.f;
    } else {
        int e2;
        (void)frexpf(amax, &e2);
        scale = ldexpf(1.f, -e2);
        tok = ldexpf(1.f, e2);
    }
    asm volatile("" : "+v"(tok));  // formed here, not sunk by the compiler into the tail

    float yf = 0.f;
    int yi = 0;
    int s_tot = 0;  // INT8 path: this lane's share of the activation sum
    for (int64_t kc = kbA; kc < kbB; kc += CK) {
        nkb = (int)((kbB - kc) < CK ? (kbB - kc) : CK);
        if (kc != kbA) {
            load_acts(kc, nkb);
            load_weights(kc, nkb);
            lds_barrier();  // the previous chunk's tables and sums are no longer read
        }
        // 2-3. signed tables of this chunk and the activation sums
        if constexpr (INT8) {
#pragma unroll
            for (int r = 0; r < GPT; ++r) {
                const int g = tid + NT * r;
                const int q0 = quant8<0>(ag[r].x, scale), q1 = quant8<1>(ag[r].x, scale);
                const int q2 = quant8<0>(ag[r].y, scale), q3 = quant8<1>(ag[r].y, scale);
                s_tot += (q0 + q1) + (q2 + q3);
                if (g < nkb * GPB) build_group_i16(F + (g / GPB) * Tab<true>::BLK + (g % GPB) * Tab<true>::G, q0, q1, q2, q3);
            }
        } else {
#pragma unroll
            for (int r = 0; r < QPT; ++r) {
                const int e = tid + NT * r, g = e >> 2, qr = e & 3;
                const float xs = act_value<false>(av[r], scale);
                const int xb = __float_as_int(xs);
                const int4 q = quarter_entries<false>(__int_as_float(quad_bcast<0>(xb)), __int_as_float(quad_bcast<1>(xb)),
                                                      __int_as_float(quad_bcast<2>(xb)), __int_as_float(quad_bcast<3>(xb)), qr);
                if (need_s) {  // sum of the 64 activations of this wave and round: half a 128-block
                    const float hs = wave_sum_f(xs);
                    if (lane == 63) hsf[r * NW + wave] = hs;
                }
                if (g < nkb * GPB) *(int4 *)(F + (g / GPB) * Tab<false>::BLK + (g % GPB) * Tab<false>::G + qr * 16) = q;
            }
        }
        // epilogue operands of this lane's 128-blocks (unconditional vector loads,
        // decoded after the barrier)
        uint2 mwd[TW];
        if constexpr (!INT8) {
#pragma unroll
            for (int t = 0; t < TW; ++t) {
                const int kbl = sigma + t * S, kbc = kbl < nkb ? kbl : nkb - 1;
                const int q = (int)(((float)(kc + kbc) + 0.5f) * p.inv_kpg);
                mwd[t] = load_meta_words(p, q, lane_value(n));
            }
        }
        if (INT8 && need_s && kc + CK >= kbB) {  // the activation sum of this wavefront, before the lookups
            const int hs = wave_sum_i(s_tot);
            if (lane == 63) hsi[wave] = hs;
        }
        if constexpr (INT8 && SW * GPB == 64) {
            // lane 64 w + l builds group 64 w + l + NT r, in block 2 w + l / 32 + S r, and
            // looks up blocks 2 w + l / 32 + S t: every wavefront reads only the tables
            // it built, so a wavefront-local fence replaces the workgroup barrier (the
            // wavefronts no longer wait for each other; 4.26 -> 4.12 us on the headline)
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
        } else {
            lds_barrier();
        }
        tl_stamp(p, 2);
#pragma unroll
        for (int t = 0; t < TW; ++t) {
            const int kbl = sigma + t * S;
            if (kbl < nkb) {
                const uint32_t base = (uint32_t)(kbl * Tab<INT8>::BLK);
                int tot = 0;
#pragma unroll
                for (int i = 0; i < NPL; ++i)  // exact in INT32, see lookup_word
                    tot += lookup_word<INT8>(F, base, w[t][i]) << (pl * NPL + i);
                if constexpr (INT8) {
                    yi += tot;
                } else {
                    const SZ sz = decode_sz(p, mwd[t]);
                    yf = fmaf(sz.sp * (1.0f / (float)(1 << FIX_SHIFT)), (float)tot, yf);
                    // activation sum of this 128-block: the two half-block sums of its round
                    const int hb = (kbl / BPR) * NW + 2 * (kbl % BPR);
                    if (need_s && pl == 0) yf -= (sz.sp * sz.zp) * (hsf[hb] + hsf[hb + 1]);
                }
            }
        }
    }
    tl_stamp(p, 3);
    ep.tok = tok;
    if (p.tok_out && blockIdx.x == 0 && split == 0 && tid == 0) p.tok_out[m] = tok;

    // combine the lanes of each column (fixed butterfly by lane swaps), then the
    // wavefronts in order
    static_assert(CW == 16 || CW == 32 || CW == 64, "lane decompositions of 16, 32 or 64 columns");
    if constexpr (CW <= 16) {
        if (INT8) yi = xor_sum_i<16>(yi);
        else yf = xor_sum_f<16>(yf);
    }
    if constexpr (CW <= 32) {
        if (INT8) yi = xor_sum_i<32>(yi);
        else yf = xor_sum_f<32>(yf);
    }
    if (lane < CW) {
        redf[wave][lane] = yf;
        redi[wave][lane] = yi;
    }
    lds_barrier();
    tl_stamp(p, 4);
    if (wave == 0 && lane < CW) {
        float sf = redf[0][lane];
        int si = redi[0][lane];
#pragma unroll
        for (int v = 1; v < NW; ++v) {
            sf += redf[v][lane];
            si += redi[v][lane];
        }
        if (INT8 && need_s) {  // ternary offset S, once per column
#pragma unroll
            for (int v = 0; v < NW; ++v) si += hsi[v];
        }
        if (p.splits == 1)
            store_out<INT8>(p, wfmt, m, n, sf, si, ep);
        else
            p.part[((int64_t)split * p.M + m) * p.N_pad + n] = INT8 ? __int_as_float(si) : sf;
    }
    tl_stamp(p, 5);
}

// Same lane decompositions as the table-fed GEMV (see lut_gemv.hip): 16 wavefronts,
// one 128-block per K slice and chunk.  INT8 activations with one plane word per lane
// and block: 4 wavefronts (one per SIMD) with four 128-blocks per K slice instead,
// while the whole K range fits one chunk -- the table build and the lookups are bound
// by vector issue, and one wavefront per SIMD building four groups per lane issues the
// per-wavefront work (the absmax reduction, the scale's division, the sums) once
// instead of four times (ternary 1 x 4096 x 4096: 4.56 -> 4.31 us; the table-fed
// kernel, which has no build to share, is slower that way: 4.17 -> 5.11 us).
template <int BITS, int PW, int SW, bool INT8>
static void launch_fused_cfg(const LutParams &p, const Layout &L, const LutPlan &plan, hipStream_t s) {
    constexpr int CW = 64 / (PW * SW);
    constexpr bool ONE_WORD = BITS / PW == 1;
    const dim3 grid((unsigned)((L.N + CW - 1) / CW), (unsigned)plan.splits, (unsigned)p.M);
    // 4 or 8 wavefronts when the whole K range fits one chunk of that many
    if (L.KB <= 4 * SW) {
        hipLaunchKernelGGL((lut_fused_gemv_kernel<BITS, PW, SW, 1, 4, INT8>), grid, dim3(256), 0, s, p, L.wfmt);
    } else if (L.KB <= 8 * SW) {
        hipLaunchKernelGGL((lut_fused_gemv_kernel<BITS, PW, SW, 1, 8, INT8>), grid, dim3(512), 0, s, p, L.wfmt);
    } else if (INT8 && ONE_WORD && L.KB <= 16 * SW) {
        if constexpr (INT8 && ONE_WORD)
            hipLaunchKernelGGL((lut_fused_gemv_kernel<BITS, PW, SW, 4, 4, INT8>), grid, dim3(256), 0, s, p, L.wfmt);
    } else {
        hipLaunchKernelGGL((lut_fused_gemv_kernel<BITS, PW, SW, 1, 16, INT8>), grid, dim3(1024), 0, s, p, L.wfmt);
    }
}

template <bool INT8>
static void launch_fused_bits(const LutParams &p, const Layout &L, const LutPlan &plan, hipStream_t s) {
    if (L.bits == 1) {
        if (plan.gemv_cfg == 0) launch_fused_cfg<1, 1, 1, INT8>(p, L, plan, s);
        else launch_fused_cfg<1, 1, 2, INT8>(p, L, plan, s);
    } else if (L.bits == 2) {
        if (plan.gemv_cfg == 0) launch_fused_cfg<2, 1, 1, INT8>(p, L, plan, s);
        else if (plan.gemv_cfg == 1) launch_fused_cfg<2, 2, 1, INT8>(p, L, plan, s);
        else launch_fused_cfg<2, 2, 2, INT8>(p, L, plan, s);
    } else {
        if constexpr (!INT8) {
            if (plan.gemv_cfg == 0) launch_fused_cfg<4, 1, 1, false>(p, L, plan, s);
            else if (plan.gemv_cfg == 1) launch_fused_cfg<4, 2, 1, false>(p, L, plan, s);
            else launch_fused_cfg<4, 4, 1, false>(p, L, plan, s);
        }
    }
}

// ---------------------------------------------------------------- split-K
//
// The split-K GEMV of lut_gemv.hip (256 columns per workgroup, one per lane, KBS
// 128-blocks of K per workgroup, the split completed in the kernel or by the
// finalize kernel) with its tables built from the activations of its own K range
// instead of read from the precompute; each lane builds the signed 16-entry table
// of one 4-activation group (the negated half by Eq. 4).
// FP path: the power-of-two token scaling only keeps FP16 table entries in range,
// so it is not needed here: entries ((-x0 + (+-x1)) + (+-x2)) + (+-x3) of the
// activations as given, in FP32, without the FP16 rounding of stored tables; a
// lookup adds the FP32 entry; the zero-point term of Eq. 3 is applied per 128-block
// (the sum over a group's blocks of s'_q z'_q S_kb is s'_q z'_q S_q), with S_kb
// summed in a fixed order over the 32 lanes that built the block's tables.
// INT8 path: the quantization needs the absmax of the whole token, so every
// workgroup first reads the whole token (16 bytes per lane and load, four loads in
// flight; the token stays in L2) and forms the same scale 127 / amax and factor
// amax / 127 as the precompute operator, then the exact INT32 entries of its
// quantized group; the ternary offset S is summed over the workgroup's K range
// (the ranges' sums add up to the token's).  Lookups and the split sum are exact,
// so the output equals the two-call path's bit for bit.  The split sum is completed
// exactly by one 64-bit atomic per output (split_complete_exact): INT32 partials, or
// FP32 partials in fixed point.
template <int BITS, int KBS, int PRE, bool INT8>
__global__ __launch_bounds__(256) void lut_fused_split_kernel(LutParams p, int wfmt) {
    constexpr int NWD = KBS * BITS;              // weight words per lane
    constexpr int NPRE = PRE < NWD ? PRE : NWD;  // of which issued before the table build
    constexpr int GS = 16;                 // entries per signed table
    constexpr int BLKF = (GPB + 1) * GS;   // 32-bit entries per 128-block (padded by one table)
    __shared__ __attribute__((aligned(16))) float F[KBS * BLKF];  // FP32 entries, or INT32 bits
    __shared__ float Sblk[KBS];                                   // FP32 sums, or INT32 bits
    __shared__ float wmx[4];                                      // INT8: the wavefronts' absmax
    tl_stamp(p, 0);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t n = (int64_t)blockIdx.x * NTILE + tid;
    const int split = blockIdx.y;
    const int64_t m = blockIdx.z;
    const int64_t kb0 = (int64_t)split * KBS;
    const int nkb = (int)((p.KB - kb0) < KBS ? (p.KB - kb0) : KBS);
    // FP path: zero-point term of every format but binary; INT8 path: ternary offset
    const bool need_s = INT8 ? wfmt == LUTGEMM_WFMT_TERNARY : wfmt != LUTGEMM_WFMT_BINARY;

    // conditional loads first, then unconditional clamped ones (see lut_gemv_kernel)
    Epi ep{};
    // (with the exact split completion any split may be the one that stores)
    if (p.splits == 1 || p.acc64) ep = load_epi<INT8>(p, wfmt, m, n, false);
    // exact completion of FP partial sums: fixed point in units of 2^(E + 16), E the
    // column's exponent for activations below 1 (these tables hold them unscaled)
    const int bndE = (!INT8 && p.acc64) ? p.bnd[lane_value(n)] + 16 : 0;
    // activations: lane g holds group g of the workgroup's range (KBS x 32 <= 256 groups)
    const uint16_t *arow = p.act + m * p.K;
    const int g = tid, gc = g < nkb * GPB ? g : nkb * GPB - 1;
    const uint2 av = ((const uint2 *)arow)[kb0 * GPB + gc];
    // INT8 path: the whole token for its absmax (clamped duplicates do not change a max)
    uint32_t mx = 0u;
    if constexpr (INT8) {
        const uint4 *a8 = (const uint4 *)arow;
        const int64_t n8 = p.K / 8;
        for (int64_t c = tid; c < n8; c += 4 * 256) {
            uint4 v[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int64_t i = c + 256 * u;
                v[u] = a8[i < n8 ? i : n8 - 1];
            }
#pragma unroll
            for (int u = 0; u < 4; ++u)
                mx = max_u16x2(mx, max_u16x2(max_u16x2(v[u].x & 0x7FFF7FFFu, v[u].y & 0x7FFF7FFFu),
                                             max_u16x2(v[u].z & 0x7FFF7FFFu, v[u].w & 0x7FFF7FFFu)));
        }
    }
    uint2 mw[KBS];
    if constexpr (!INT8) {
#pragma unroll
        for (int kbl = 0; kbl < KBS; ++kbl) {
            const int kbc = kbl < nkb ? kbl : nkb - 1;
            const int q = (int)(((float)(kb0 + kbc) + 0.5f) * p.inv_kpg);
            mw[kbl] = load_meta_words(p, q, lane_value(n));
        }
    }
    // the first NPRE weight words now, the rest once the tables are built (as in the
    // table-fed split kernel: the activations are not queued behind the weight stream)
    uint4 w[KBS][BITS];
    auto load_word = [&](int i) {
        const int kbl = i / BITS, t = i % BITS, kbc = kbl < nkb ? kbl : nkb - 1;
        w[kbl][t] = ld_nt(p.planes + ((kb0 + kbc) * BITS + t) * p.N_pad + n);
    };
#pragma unroll
    for (int i = 0; i < NPRE; ++i) load_word(i);

    // INT8 path: token absmax (DPP within the wavefront, then the 4 wavefronts) and the
    // precompute's quantizer
    float scale = 1.f, tok = 1.f;
    if constexpr (INT8) {
        const uint32_t m16 = (mx & 0xFFFFu) > (mx >> 16) ? (mx & 0xFFFFu) : (mx >> 16);
        const float wm = wave_max(h2f(m16));
        if (lane == 63) wmx[wave] = wm;
        lds_barrier();
        const float amax = fmaxf(fmaxf(wmx[0], wmx[1]), fmaxf(wmx[2], wmx[3]));
        scale = amax == 0.f ? 0.f : __fdiv_rn(127.0f, amax);
        tok = amax == 0.f ? 0.f : __fdiv_rn(amax, 127.0f);
        if (p.tok_out && blockIdx.x == 0 && split == 0 && tid == 0) p.tok_out[m] = tok;
    }
    auto qv = [&](uint32_t bits16) {  // r = clamp(rint(a * 127 / amax), -127, 127)
        const float r = rintf(h2f(bits16) * scale);
        return (int)fminf(fmaxf(r, -127.f), 127.f);
    };

    // signed table of group g and the block sums
    const float x0 = h2f(av.x & 0xFFFFu), x1 = h2f(av.x >> 16), x2 = h2f(av.y & 0xFFFFu), x3 = h2f(av.y >> 16);
    int q0 = 0, q1 = 0, q2 = 0, q3 = 0;
    if constexpr (INT8) {
        q0 = qv(av.x & 0xFFFFu);
        q1 = qv(av.x >> 16);
        q2 = qv(av.y & 0xFFFFu);
        q3 = qv(av.y >> 16);
    }
    if (g < nkb * GPB) {
        float *dst = F + (g / GPB) * BLKF + (g % GPB) * GS;
        if constexpr (INT8) {  // |entry| <= 508, exact
            int t[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) t[i] = ((-q0 + ((i & 4) ? q1 : -q1)) + ((i & 2) ? q2 : -q2)) + ((i & 1) ? q3 : -q3);
            *(int4 *)(dst + 0) = make_int4(t[0], t[1], t[2], t[3]);
            *(int4 *)(dst + 4) = make_int4(t[4], t[5], t[6], t[7]);
            *(int4 *)(dst + 8) = make_int4(-t[0], -t[1], -t[2], -t[3]);
            *(int4 *)(dst + 12) = make_int4(-t[4], -t[5], -t[6], -t[7]);
        } else {
            float t[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) t[i] = ((-x0 + ((i & 4) ? x1 : -x1)) + ((i & 2) ? x2 : -x2)) + ((i & 1) ? x3 : -x3);
            *(float4 *)(dst + 0) = make_float4(t[0], t[1], t[2], t[3]);
            *(float4 *)(dst + 4) = make_float4(t[4], t[5], t[6], t[7]);
            *(float4 *)(dst + 8) = make_float4(-t[0], -t[1], -t[2], -t[3]);
            *(float4 *)(dst + 12) = make_float4(-t[4], -t[5], -t[6], -t[7]);
        }
    }
    if (need_s) {  // S of block g / 32: fixed butterfly over its 32 lanes
        if constexpr (INT8) {
            int sg = g < nkb * GPB ? (q0 + q1) + (q2 + q3) : 0;
#pragma unroll
            for (int off = 1; off < 32; off <<= 1) sg += __shfl_xor(sg, off, 64);
            if ((tid & 31) == 0 && (tid >> 5) < KBS) Sblk[tid >> 5] = __int_as_float(sg);
        } else {
            float sg = g < nkb * GPB ? ((x0 + x1) + x2) + x3 : 0.f;
#pragma unroll
            for (int off = 1; off < 32; off <<= 1) sg += __shfl_xor(sg, off, 64);
            if ((tid & 31) == 0 && (tid >> 5) < KBS) Sblk[tid >> 5] = sg;
        }
    }
    lds_barrier();
    asm volatile("" ::: "memory");  // the remaining weight loads stay after the table build
    tl_stamp(p, 1);
#pragma unroll
    for (int i = NPRE; i < NWD; ++i) load_word(i);

    float yf = 0.f;
    int yi = 0;
#pragma unroll
    for (int kbl = 0; kbl < KBS; ++kbl) {
        if (kbl < nkb) {
            float tot = 0.f;
            int toti = 0;
#pragma unroll
            for (int t = 0; t < BITS; ++t) {
                const uint32_t wd[4] = {w[kbl][t].x, w[kbl][t].y, w[kbl][t].z, w[kbl][t].w};
                float acc = 0.f;
                int acci = 0;
#pragma unroll
                for (int d = 0; d < 4; ++d) {
                    const char *Fg = (const char *)(F + kbl * BLKF + d * 8 * GS);
                    const uint32_t lo = wd[d] << 2, hi = wd[d] >> 2;
                    if constexpr (INT8) {
                        acci += *(const int *)(Fg + 0 * GS * 4 + idx4<0>(lo)) + *(const int *)(Fg + 1 * GS * 4 + idx4<0>(hi));
                        acci += *(const int *)(Fg + 2 * GS * 4 + idx4<1>(lo)) + *(const int *)(Fg + 3 * GS * 4 + idx4<1>(hi));
                        acci += *(const int *)(Fg + 4 * GS * 4 + idx4<2>(lo)) + *(const int *)(Fg + 5 * GS * 4 + idx4<2>(hi));
                        acci += *(const int *)(Fg + 6 * GS * 4 + idx4<3>(lo)) + *(const int *)(Fg + 7 * GS * 4 + idx4<3>(hi));
                    } else {
                        acc += *(const float *)(Fg + 0 * GS * 4 + idx4<0>(lo)) + *(const float *)(Fg + 1 * GS * 4 + idx4<0>(hi));
                        acc += *(const float *)(Fg + 2 * GS * 4 + idx4<1>(lo)) + *(const float *)(Fg + 3 * GS * 4 + idx4<1>(hi));
                        acc += *(const float *)(Fg + 4 * GS * 4 + idx4<2>(lo)) + *(const float *)(Fg + 5 * GS * 4 + idx4<2>(hi));
                        acc += *(const float *)(Fg + 6 * GS * 4 + idx4<3>(lo)) + *(const float *)(Fg + 7 * GS * 4 + idx4<3>(hi));
                    }
                }
                if constexpr (INT8)
                    toti += acci << t;  // exact: |sum| < 2^31
                else
                    tot += acc * (float)(1 << t);  // exact scaling by the plane weight
            }
            if constexpr (INT8) {
                yi += toti;
                if (need_s) yi += __float_as_int(Sblk[kbl]);  // ternary offset of this block
            } else {
                const SZ sz = decode_sz(p, mw[kbl]);
                yf = fmaf(sz.sp, tot, yf);
                if (need_s) yf -= (sz.sp * sz.zp) * Sblk[kbl];
            }
        }
    }
    tl_stamp(p, 2);
    if (p.splits == 1) {
        ep.tok = tok;
        store_out<INT8>(p, wfmt, m, n, yf, yi, ep);
    } else if (p.acc64) {  // exact split sum: one atomic per output
        ep.tok = tok;
        if (INT8)
            split_complete_exact<INT8>(p, wfmt, m, n, (long long)yi, 0.f, 0.f, INT_MIN, ep);
        else
            split_complete_exact<INT8>(p, wfmt, m, n, to_fixed(yf, bndE), 0.f, 0.f, bndE, ep);
    } else if (p.cnt) {
        split_complete<INT8>(p, wfmt, m, n, split, yf, yi, p.cnt + m * gridDim.x + blockIdx.x, INT8 ? tok : -1.f);
    } else {  // long K splits: lut_finalize_kernel adds the partials after this kernel
        p.part[((int64_t)split * p.M + m) * p.N_pad + n] = INT8 ? __int_as_float(yi) : yf;
    }
    tl_stamp(p, 6);
}

template <int BITS, int PRE, bool INT8>
static void launch_fused_split_pre(const LutParams &p, const Layout &L, const LutPlan &plan, hipStream_t s) {
    const dim3 grid((unsigned)(L.N_pad / NTILE), (unsigned)plan.splits, (unsigned)p.M);
    switch (plan.kbs) {  // the planner keeps KBS <= 8 / b (and KBS x 32 groups <= 256 lanes)
    case 1: hipLaunchKernelGGL((lut_fused_split_kernel<BITS, 1, PRE, INT8>), grid, dim3(256), 0, s, p, L.wfmt); break;
    case 2: hipLaunchKernelGGL((lut_fused_split_kernel<BITS, 2, PRE, INT8>), grid, dim3(256), 0, s, p, L.wfmt); break;
    case 4:
        if constexpr (BITS <= 2)
            hipLaunchKernelGGL((lut_fused_split_kernel<BITS, 4, PRE, INT8>), grid, dim3(256), 0, s, p, L.wfmt);
        break;
    default:
        if constexpr (BITS == 1)
            hipLaunchKernelGGL((lut_fused_split_kernel<BITS, 8, PRE, INT8>), grid, dim3(256), 0, s, p, L.wfmt);
        break;
    }
}

template <int BITS, bool INT8>
static void launch_fused_split_bits(const LutParams &p, const Layout &L, const LutPlan &plan, hipStream_t s) {
    if (plan.pre == 0) launch_fused_split_pre<BITS, 0, INT8>(p, L, plan, s);
    else if (plan.pre == 4) launch_fused_split_pre<BITS, 4, INT8>(p, L, plan, s);
    else if (plan.pre >= 8) launch_fused_split_pre<BITS, 8, INT8>(p, L, plan, s);
    else launch_fused_split_pre<BITS, 2, INT8>(p, L, plan, s);
}

int launch_fused_split(const LutParams &p, const Layout &L, const LutPlan &plan, void *stream) {
    hipStream_t s = (hipStream_t)stream;
    if (L.act == LUTGEMM_ACT_INT8) {  // binary and ternary weights only (1 or 2 planes)
        if (L.bits == 1) launch_fused_split_bits<1, true>(p, L, plan, s);
        else if (L.bits == 2) launch_fused_split_bits<2, true>(p, L, plan, s);
        else return (int)hipErrorInvalidValue;
    } else if (L.bits == 1) {
        launch_fused_split_bits<1, false>(p, L, plan, s);
    } else if (L.bits == 2) {
        launch_fused_split_bits<2, false>(p, L, plan, s);
    } else {
        launch_fused_split_bits<4, false>(p, L, plan, s);
    }
    return (int)hipGetLastError();
}

int launch_fused_gemv(const LutParams &p, const Layout &L, const LutPlan &plan, void *stream) {
    hipStream_t s = (hipStream_t)stream;
    if (L.act == LUTGEMM_ACT_INT8)
        launch_fused_bits<true>(p, L, plan, s);
    else
        launch_fused_bits<false>(p, L, plan, s);
    return (int)hipGetLastError();
}

}  // namespace lutgemm
