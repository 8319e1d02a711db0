// Single-token bit-serial LUT mpGEMM (LUT Tensor Core, Section 3.1 bit-serial
// tables with Eq. 3, 5 and 6; LMMA semantics O = A x W^T + Acc, Section 3.3.1).
//
// gfx950 mapping.  A workgroup (NW wavefronts) owns CW output columns over its
// whole K range, so no other workgroup has to combine its results.  The 64 lanes
// of a wavefront are (column, bit-plane group, K slice): CW = 64 / (PW * SW)
// columns, PW lanes per column splitting the b bit-planes, SW K slices; the
// wavefronts add NW times more K slices.  At any LDS read every lane of a
// wavefront addresses the table of the same 4-activation group in at most SW = 2
// different 128-blocks of K, whose tables sit in different LDS banks (padded
// block stride), so reads are conflict-free; each table entry is reused by the
// CW x (b / PW) lookups of that group (table reuse across columns, the
// "elongated N" idea of Section 3.2.2, here across lanes and planes).
//
// K is processed in chunks of CK 128-blocks.  For every chunk the half tables of
// Eq. 5 (8 entries per 4 activations, the HBM format) are expanded into full
// signed 16-entry tables in LDS, F[s i] = (s ? -T[i] : T[i]), so the stored Eq. 6
// index addresses its entry directly (the inversion of Eq. 6 was done by the
// packer and the negation here, once per workgroup, instead of per lookup).
// Entries are INT16 on the INT8 path (exact) and INT32 on the FP path (the FP16
// entries times 2^20: exact for |T| >= 2^-10, otherwise within 2^-21; tables are
// normalized to |T| < 4 by the precompute).  Each chunk's half tables are loaded
// before its weight words, so the expansion overlaps the weight stream.
//
// A lookup is one SDWA byte-add (table base + entry offset), one LDS read and
// half of a v_add3_u32.  Per 128-block the plane sums are combined as
// sum_t 2^t acc_t (exact in INT32) and the Eq. 3 epilogue s' (A - z' S) is
// applied in FP32; lanes of one column are then combined by a fixed butterfly
// and the wavefronts in order, so results are bitwise reproducible.
#include "lut_common.h"

namespace lutgemm {

template <int BITS, int PW, int SW, int TW, int NW, bool INT8, bool TQ>
__global__ __launch_bounds__(64 * NW) void lut_gemv2_kernel(LutParams p, int wfmt) {
    constexpr int NT = 64 * NW;            // threads per workgroup
    constexpr int CW = 64 / (PW * SW);    // columns per workgroup
    constexpr int S = NW * SW;             // K slices per workgroup
    constexpr int CK = S * TW;             // 128-blocks per chunk
    constexpr int NPL = BITS / PW;         // bit-planes per lane
    constexpr int QPT = CK * GPB * 4 / NT; // table quarters staged per thread and chunk
    static_assert(QPT * NT == CK * GPB * 4, "table quarters divide evenly over the threads");
    static_assert(TW * NPL <= 4, "at most four prefetched weight words per lane");
    __shared__ __attribute__((aligned(16))) char F[CK * Tab<INT8>::BLK];
    __shared__ float redf[NW][CW];
    __shared__ int redi[NW][CW];

    tl_stamp(p, 0);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int c = lane % CW;
    const int pl = (lane / CW) % PW;       // plane group of this lane
    const int sl = lane / (CW * PW);       // in-wave K slice
    const int sigma = wave * SW + sl;      // K slice within a chunk
    const int64_t n = (int64_t)blockIdx.x * CW + c;
    const int64_t m = blockIdx.z;
    const int split = blockIdx.y;
    const int64_t kbA = (int64_t)split * p.kbs;
    const int64_t kbB = (kbA + p.kbs < p.KB) ? kbA + p.kbs : p.KB;

    // Loads of one chunk: table quarters first, then the lane's weight words.
    // Loads retire in issue order, so waiting for the tables never waits for the
    // weights, which keep streaming in while the tables are expanded.  The next
    // chunk's loads are issued before this chunk's lookups (software pipeline), so
    // with several chunks per workgroup only the first one waits a full latency.
    // Every chunk load is unconditional (indices past the chunk are clamped to its
    // last group / block and the values ignored), so the waits the compiler
    // places count exactly the loads issued after the ones they wait for;
    // conditional loads (the epilogue operands) are issued before them.
    uint2 tq[QPT], tqn[QPT];
    uint4 w[TW][NPL], wn[TW][NPL];
    auto load_chunk = [&](int64_t kc, uint2(&tq_)[QPT], uint4(&w_)[TW][NPL]) {
        const int nkb = (int)((kbB - kc) < CK ? (kbB - kc) : CK);
#pragma unroll
        for (int r = 0; r < QPT; ++r) {
            const int e = tid + NT * r, g = e >> 2, gc = g < nkb * GPB ? g : nkb * GPB - 1;
            tq_[r] = load_quarter<TQ>(p, m * p.J + kc * GPB + gc, e & 1);
        }
#pragma unroll
        for (int t = 0; t < TW; ++t) {
            const int kbl = sigma + t * S, kbc = kbl < nkb ? kbl : nkb - 1;
#pragma unroll
            for (int i = 0; i < NPL; ++i) w_[t][i] = ld_nt(p.planes + ((kc + kbc) * BITS + pl * NPL + i) * p.N_pad + n);
        }
    };

    float yf = 0.f;
    int yi = 0;
    Epi ep{};
    if (p.splits == 1) ep = load_epi<INT8>(p, wfmt, m, n, true);
    load_chunk(kbA, tq, w);
    for (int64_t kc = kbA; kc < kbB; kc += CK) {
        const int nkb = (int)((kbB - kc) < CK ? (kbB - kc) : CK);
        lds_barrier();  // the previous chunk's tables are no longer read
#pragma unroll
        for (int r = 0; r < QPT; ++r) {
            const int e = tid + NT * r, g = e >> 2;
            if (g < nkb * GPB) store_quarter<INT8, TQ>(F, g / GPB, g % GPB, e & 3, tq[r]);
        }
        // epilogue operands of this lane's 128-blocks (unconditional vector loads,
        // issued before the lookups)
        BlkMeta bm[TW];
        if constexpr (!INT8) {
#pragma unroll
            for (int t = 0; t < TW; ++t) {
                const int kbl = sigma + t * S, kbc = kbl < nkb ? kbl : nkb - 1;
                bm[t] = load_blk_meta(p, kc + kbc, m, lane_value(n));
            }
        }
        const bool more = kc + CK < kbB;
        if (more) load_chunk(kc + CK, tqn, wn);
        lds_barrier();
        if (kc == kbA) tl_stamp(p, 1);
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
                    const float2 e = blk_epilogue(p, bm[t], kc + kbl);
                    yf = fmaf(e.x, (float)tot, yf) - (pl == 0 ? e.y : 0.f);
                }
            }
        }
        if (more) {
#pragma unroll
            for (int r = 0; r < QPT; ++r) tq[r] = tqn[r];
#pragma unroll
            for (int t = 0; t < TW; ++t)
#pragma unroll
                for (int i = 0; i < NPL; ++i) w[t][i] = wn[t][i];
        }
    }

    tl_stamp(p, 3);
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
        if (p.splits == 1)
            store_out<INT8>(p, wfmt, m, n, sf, si + ep.s0, ep);
        else if (INT8 && split == 0 && wfmt == LUTGEMM_WFMT_TERNARY)
            p.part[((int64_t)split * p.M + m) * p.N_pad + n] = __int_as_float(si + ((const int *)p.S)[m * p.Q]);
        else
            p.part[((int64_t)split * p.M + m) * p.N_pad + n] = INT8 ? __int_as_float(si) : sf;
    }
}

// Split-K variant for large weights.  One lane per column and 256 columns per
// workgroup, so each staged table serves 256 columns (the widest reuse); each
// workgroup covers KBS 128-blocks of K.  Load order: the half tables and the
// epilogue operands, then the first PRE of the lane's KBS x b weight words
// (nontemporal), then -- once the tables are in LDS -- the remaining words.  The
// tables are tiny L2 hits, but requested behind a full load of weight misses they
// would wait about one loaded HBM latency and hold every lookup back until the
// weight stream is over; staged first, the lookups follow the weight words as they
// arrive, while the PRE early words keep HBM busy during the table latency.  The 4
// wavefronts read the same table at a time (no bank conflicts) and the
// compile-time table offsets leave one SDWA AND per lookup.  With more than one K
// split the workgroups of a column tile complete the sum themselves, so the call is
// one launch: by one exact 64-bit atomic per output (split_complete_exact), or with
// INT8-quantized tables by the arrival protocol (split_complete: the last one to
// finish adds the partials in split order).
// TPW tokens per workgroup (1, or 2 for two tokens with 1-bit weights: the weight
// words, their index decoding and the metadata then serve both tokens, whose tables
// sit side by side in LDS, so two tokens cost one pass over the weights instead of
// two; only with the exact completion, the finalize kernel or no K split).
template <int BITS, int KBS, bool INT8, bool TQ, int PRE, int TPW>
__global__ __launch_bounds__(256) void lut_gemv_split_kernel(LutParams p, int wfmt) {
    constexpr int QPT = (KBS * GPB * 4 + 255) / 256;  // table quantities per thread
    constexpr int NWD = KBS * BITS;                  // weight words per lane
    constexpr int NPRE = PRE < NWD ? PRE : NWD;      // of which issued before the table wait
    constexpr int FB = KBS * Tab<INT8>::BLK;         // LDS bytes of one token's tables
    __shared__ __attribute__((aligned(16))) char F[TPW * FB];
    tl_stamp(p, 0);
    const int tid = threadIdx.x;
    const int64_t n = (int64_t)blockIdx.x * NTILE + tid;
    const int split = blockIdx.y;
    const int64_t m0 = (int64_t)blockIdx.z * TPW;
    // the workgroup's tokens; a row past M repeats row M - 1 and is never stored
    int64_t mr[TPW];
#pragma unroll
    for (int u = 0; u < TPW; ++u) mr[u] = m0 + u < p.M ? m0 + u : p.M - 1;
    const int64_t kb0 = (int64_t)split * KBS;
    const int nkb = (int)((p.KB - kb0) < KBS ? (p.KB - kb0) : KBS);

    // conditional loads (epilogue operands) first, then the unconditional loads with
    // clamped indices (see lut_gemv2_kernel)
    Epi ep[TPW];
    int yi[TPW];
#pragma unroll
    for (int u = 0; u < TPW; ++u) {
        ep[u] = Epi{};
        if (p.splits == 1 || p.acc64)  // (exact completion: any split may be the one that stores)
            ep[u] = load_epi<INT8>(p, wfmt, mr[u], n, split == 0);
        else if (INT8 && split == 0 && wfmt == LUTGEMM_WFMT_TERNARY)
            ep[u].s0 = ((const int *)p.S)[lane_value(mr[u] * p.Q)];
        yi[u] = ep[u].s0;
    }
    // exact completion of FP partial sums in fixed point: the column's exponent
    const int bndE = (!INT8 && p.acc64 && p.Q != 1) ? p.bnd[lane_value(n)] : 0;
    uint2 tq[TPW][QPT];
#pragma unroll
    for (int u = 0; u < TPW; ++u)
#pragma unroll
        for (int r = 0; r < QPT; ++r) {
            const int e = tid + 256 * r, g = e >> 2, gc = g < nkb * GPB ? g : nkb * GPB - 1;
            tq[u][r] = load_quarter<TQ>(p, mr[u] * p.J + kb0 * GPB + gc, e & 1);
        }
    BlkMeta bm[TPW][KBS];
    if constexpr (!INT8) {
#pragma unroll
        for (int u = 0; u < TPW; ++u)
#pragma unroll
            for (int kbl = 0; kbl < KBS; ++kbl) {
                const int kbc = kbl < nkb ? kbl : nkb - 1;
                bm[u][kbl] = load_blk_meta(p, kb0 + kbc, mr[u], lane_value(n));
            }
    }
    uint4 w[KBS][BITS];
    auto load_word = [&](int i) {
        const int kbl = i / BITS, t = i % BITS, kbc = kbl < nkb ? kbl : nkb - 1;
        w[kbl][t] = ld_nt(p.planes + ((kb0 + kbc) * BITS + t) * p.N_pad + n);
    };
#pragma unroll
    for (int i = 0; i < NPRE; ++i) load_word(i);
#pragma unroll
    for (int u = 0; u < TPW; ++u)
#pragma unroll
        for (int r = 0; r < QPT; ++r) {
            const int e = tid + 256 * r, g = e >> 2;
            if (g < nkb * GPB)
                store_quarter<INT8, TQ>(F + u * FB, g / GPB, g % GPB, e & 3, tq[u][r]);
        }
    lds_barrier();
    asm volatile("" ::: "memory");  // the remaining weight loads stay after the table wait
    tl_stamp(p, 1);
#pragma unroll
    for (int i = NPRE; i < NWD; ++i) load_word(i);

    float yf[TPW];
    long long yx[TPW];  // FP path, exact completion: the integer sum of the split's entries
#pragma unroll
    for (int u = 0; u < TPW; ++u) {
        yf[u] = 0.f;
        yx[u] = 0;
    }
#pragma unroll
    for (int kbl = 0; kbl < KBS; ++kbl) {
        if (kbl < nkb) {
            int tot[TPW];
#pragma unroll
            for (int u = 0; u < TPW; ++u) tot[u] = 0;
#pragma unroll
            for (int t = 0; t < BITS; ++t) {
                const uint32_t wd[4] = {w[kbl][t].x, w[kbl][t].y, w[kbl][t].z, w[kbl][t].w};
                int acc[TPW];
#pragma unroll
                for (int u = 0; u < TPW; ++u) acc[u] = 0;
#pragma unroll
                for (int d = 0; d < 4; ++d) {
                    constexpr int GS = Tab<INT8>::G;
                    const uint32_t lo = INT8 ? wd[d] << 1 : wd[d] << 2, hi = INT8 ? wd[d] >> 3 : wd[d] >> 2;
                    const uint32_t o0 = idx_off<0, INT8>(lo), o1 = idx_off<0, INT8>(hi), o2 = idx_off<1, INT8>(lo),
                                   o3 = idx_off<1, INT8>(hi), o4 = idx_off<2, INT8>(lo), o5 = idx_off<2, INT8>(hi),
                                   o6 = idx_off<3, INT8>(lo), o7 = idx_off<3, INT8>(hi);
#pragma unroll
                    for (int u = 0; u < TPW; ++u) {
                        const char *Fg = F + u * FB + kbl * Tab<INT8>::BLK + d * 8 * GS;
                        acc[u] += lds_entry<INT8>(Fg + 0 * GS, o0) + lds_entry<INT8>(Fg + 1 * GS, o1);
                        acc[u] += lds_entry<INT8>(Fg + 2 * GS, o2) + lds_entry<INT8>(Fg + 3 * GS, o3);
                        acc[u] += lds_entry<INT8>(Fg + 4 * GS, o4) + lds_entry<INT8>(Fg + 5 * GS, o5);
                        acc[u] += lds_entry<INT8>(Fg + 6 * GS, o6) + lds_entry<INT8>(Fg + 7 * GS, o7);
                    }
                }
#pragma unroll
                for (int u = 0; u < TPW; ++u) tot[u] += acc[u] << t;  // exact in INT32, see the kernel above
            }
#pragma unroll
            for (int u = 0; u < TPW; ++u) {
                if constexpr (INT8) {
                    yi[u] += tot[u];
                } else {
                    const float2 e = blk_epilogue(p, bm[u][kbl], kb0 + kbl);
                    yf[u] = fmaf(e.x, (float)tot[u], yf[u]) - e.y;
                    yx[u] += tot[u];
                }
            }
        }
    }
    tl_stamp(p, 2);
    if (p.splits == 1) {
#pragma unroll
        for (int u = 0; u < TPW; ++u)
            if (m0 + u < p.M) store_out<INT8>(p, wfmt, m0 + u, n, yf[u], yi[u], ep[u]);
    } else if (p.acc64) {
        // every token's atomic in flight before any return is looked at
        long long v[TPW];
        float sx[TPW], sy[TPW];
        unsigned long long old[TPW];
#pragma unroll
        for (int u = 0; u < TPW; ++u) {
            sx[u] = 0.f;
            sy[u] = 0.f;
            if (INT8) {
                v[u] = (long long)yi[u];
            } else if (p.Q == 1) {  // integer entries, the column's one group applied at the end
                const float2 e = blk_epilogue(p, bm[u][0], 0);
                v[u] = yx[u];
                sx[u] = e.x;
                sy[u] = e.y;
            } else {
                v[u] = to_fixed(yf[u], bndE);
            }
            old[u] = m0 + u < p.M ? exact_add(p, m0 + u, n, v[u]) : 0ull;
        }
        const int E = (INT8 || p.Q == 1) ? INT_MIN : bndE;
        unsigned long long cleared = 0ull;
#pragma unroll
        for (int u = 0; u < TPW; ++u)
            if (m0 + u < p.M) cleared |= exact_finish<INT8>(p, wfmt, m0 + u, n, old[u], v[u], sx[u], sy[u], E, ep[u]);
        asm volatile("; exact split words cleared: %0" ::"v"(cleared));
    } else if (TPW == 1 && p.cnt) {
        split_complete<INT8>(p, wfmt, m0, n, split, yf[0], yi[0], p.cnt + m0 * gridDim.x + blockIdx.x);
    } else {  // long K splits: lut_finalize_kernel adds the partials after this kernel
#pragma unroll
        for (int u = 0; u < TPW; ++u)
            if (m0 + u < p.M)
                p.part[((int64_t)split * p.M + m0 + u) * p.N_pad + n] = INT8 ? __int_as_float(yi[u]) : yf[u];
    }
    tl_stamp(p, 6);
}

template <int BITS, bool INT8, bool TQ, int PRE, int TPW>
static void launch_split_tpw(const LutParams &p, const Layout &L, const LutPlan &plan, hipStream_t s) {
    const dim3 grid((unsigned)(L.N_pad / NTILE), (unsigned)plan.splits, (unsigned)((p.M + TPW - 1) / TPW));
    switch (plan.kbs) {  // at most 8 weight words per lane (the planner keeps KBS <= 8 / b)
    case 1: hipLaunchKernelGGL((lut_gemv_split_kernel<BITS, 1, INT8, TQ, PRE, TPW>), grid, dim3(256), 0, s, p, L.wfmt); break;
    case 2: hipLaunchKernelGGL((lut_gemv_split_kernel<BITS, 2, INT8, TQ, PRE, TPW>), grid, dim3(256), 0, s, p, L.wfmt); break;
    case 4:
        if constexpr (BITS <= 2)
            hipLaunchKernelGGL((lut_gemv_split_kernel<BITS, 4, INT8, TQ, PRE, TPW>), grid, dim3(256), 0, s, p, L.wfmt);
        break;
    default:
        if constexpr (BITS == 1)
            hipLaunchKernelGGL((lut_gemv_split_kernel<BITS, 8, INT8, TQ, PRE, TPW>), grid, dim3(256), 0, s, p, L.wfmt);
        break;
    }
}

template <int BITS, bool INT8, bool TQ, int PRE>
static void launch_split_pre(const LutParams &p, const Layout &L, const LutPlan &plan, hipStream_t s) {
    if constexpr (BITS == 1) {  // two tokens per workgroup: 1-bit weights only (planner)
        if (plan.mt == 2) {
            launch_split_tpw<BITS, INT8, TQ, PRE, 2>(p, L, plan, s);
            return;
        }
    }
    launch_split_tpw<BITS, INT8, TQ, PRE, 1>(p, L, plan, s);
}

// weight words issued before the table wait: plan.pre (half of the lane's words by
// default, at least one; 8 = all of them)
template <int BITS, bool INT8, bool TQ>
static void launch_split(const LutParams &p, const Layout &L, const LutPlan &plan, hipStream_t s) {
    if (plan.pre == 0) launch_split_pre<BITS, INT8, TQ, 0>(p, L, plan, s);
    else if (plan.pre == 4) launch_split_pre<BITS, INT8, TQ, 4>(p, L, plan, s);
    else if (plan.pre >= 8) launch_split_pre<BITS, INT8, TQ, 8>(p, L, plan, s);
    else launch_split_pre<BITS, INT8, TQ, 2>(p, L, plan, s);
}

// 16 wavefronts per workgroup, one 128-block per K slice and chunk; 4 or 8 when
// the whole K range fits one chunk of that many (short K: no idle wavefronts and a
// shorter cross-wavefront reduction).
template <int BITS, int PW, int SW, bool INT8, bool TQ>
static void launch_cfg(const LutParams &p, const Layout &L, const LutPlan &plan, hipStream_t s) {
    constexpr int CW = 64 / (PW * SW);
    const dim3 grid((unsigned)((L.N + CW - 1) / CW), (unsigned)plan.splits, (unsigned)p.M);
    if (L.KB <= 4 * SW)
        hipLaunchKernelGGL((lut_gemv2_kernel<BITS, PW, SW, 1, 4, INT8, TQ>), grid, dim3(256), 0, s, p, L.wfmt);
    else if (L.KB <= 8 * SW)
        hipLaunchKernelGGL((lut_gemv2_kernel<BITS, PW, SW, 1, 8, INT8, TQ>), grid, dim3(512), 0, s, p, L.wfmt);
    else
        hipLaunchKernelGGL((lut_gemv2_kernel<BITS, PW, SW, 1, 16, INT8, TQ>), grid, dim3(1024), 0, s, p, L.wfmt);
}

// Lane decompositions (PW, SW) offered per bit width, indexed by LutPlan::gemv_cfg
// (columns per workgroup CW = 64 / (PW SW), 128-blocks per chunk CK = 16 SW):
//   b = 1: 0 -> (1,1) CW=64 CK=16   1 -> (1,2) CW=32 CK=32
//   b = 2: 0 -> (1,1) CW=64 CK=16   1 -> (2,1) CW=32 CK=16   2 -> (2,2) CW=16 CK=32
//   b = 4: 0 -> (1,1) CW=64 CK=16   1 -> (2,1) CW=32 CK=16   2 -> (4,1) CW=16 CK=16
template <bool INT8, bool TQ>
static int launch_gemv_bits(const LutParams &p, const Layout &L, const LutPlan &plan, hipStream_t s) {
    if (L.bits == 1) {
        if (plan.gemv_cfg == 0) launch_cfg<1, 1, 1, INT8, TQ>(p, L, plan, s);
        else launch_cfg<1, 1, 2, INT8, TQ>(p, L, plan, s);
    } else if (L.bits == 2) {
        if (plan.gemv_cfg == 0) launch_cfg<2, 1, 1, INT8, TQ>(p, L, plan, s);
        else if (plan.gemv_cfg == 1) launch_cfg<2, 2, 1, INT8, TQ>(p, L, plan, s);
        else launch_cfg<2, 2, 2, INT8, TQ>(p, L, plan, s);
    } else {
        if constexpr (!INT8) {
            if (plan.gemv_cfg == 0) launch_cfg<4, 1, 1, false, TQ>(p, L, plan, s);
            else if (plan.gemv_cfg == 1) launch_cfg<4, 2, 1, false, TQ>(p, L, plan, s);
            else launch_cfg<4, 4, 1, false, TQ>(p, L, plan, s);
        }
    }
    return (int)hipGetLastError();
}

int launch_gemv(const LutParams &p, const Layout &L, const LutPlan &plan, void *stream) {
    hipStream_t s = (hipStream_t)stream;
    const bool i8 = L.act == LUTGEMM_ACT_INT8, tq = L.act == LUTGEMM_ACT_FP16_LUT8;
    if (plan.kind == 2) {
        if (L.bits == 1) {
            if (i8) launch_split<1, true, false>(p, L, plan, s);
            else if (tq) launch_split<1, false, true>(p, L, plan, s);
            else launch_split<1, false, false>(p, L, plan, s);
        } else if (L.bits == 2) {
            if (i8) launch_split<2, true, false>(p, L, plan, s);
            else if (tq) launch_split<2, false, true>(p, L, plan, s);
            else launch_split<2, false, false>(p, L, plan, s);
        } else {
            if (tq) launch_split<4, false, true>(p, L, plan, s);
            else launch_split<4, false, false>(p, L, plan, s);
        }
        return (int)hipGetLastError();
    }
    if (i8) return launch_gemv_bits<true, false>(p, L, plan, s);
    return tq ? launch_gemv_bits<false, true>(p, L, plan, s) : launch_gemv_bits<false, false>(p, L, plan, s);
}

}  // namespace lutgemm
