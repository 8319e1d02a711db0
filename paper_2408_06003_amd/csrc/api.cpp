// C ABI of the LUT mpGEMM library: argument validation, size queries, launch
// planning and dispatch.  Everything here runs on the host; the arithmetic of
// every step runs in the HIP kernels of pack.hip, precompute.hip, lut_gemv.hip,
// lut_mpgemm.hip, lut_fused.hip and dequant_mfma.hip.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "lutgemm_internal.h"

using namespace lutgemm;

namespace {

constexpr int64_t MAX_M = int64_t(1) << 19;
constexpr int64_t MAX_K = int64_t(1) << 20;
constexpr int64_t MAX_N = int64_t(1) << 24;
constexpr int64_t MAX_TILES = int64_t(1) << 24;

bool aligned16(const void *p) { return ((uintptr_t)p & 15u) == 0; }

lutgemm_status_t check_problem(const lutgemm_problem_t *p, int64_t M) {
    if (!p) return LUTGEMM_ERROR_INVALID_VALUE;
    if (p->K <= 0 || p->N <= 0 || M <= 0 || p->reserved != 0) return LUTGEMM_ERROR_INVALID_VALUE;
    if (p->wfmt < LUTGEMM_WFMT_UINT || p->wfmt > LUTGEMM_WFMT_TERNARY_3IN5) return LUTGEMM_ERROR_INVALID_VALUE;
    if (p->act != LUTGEMM_ACT_FP16 && p->act != LUTGEMM_ACT_INT8 && p->act != LUTGEMM_ACT_FP16_LUT8)
        return LUTGEMM_ERROR_INVALID_VALUE;
    if (p->scale_fp32 != 0 && p->scale_fp32 != 1) return LUTGEMM_ERROR_INVALID_VALUE;
    if (p->w_bits <= 0 || p->group_size < 0) return LUTGEMM_ERROR_INVALID_VALUE;
    if (p->K > MAX_K || p->N > MAX_N || M > MAX_M) return LUTGEMM_ERROR_NOT_SUPPORTED;
    // the multi-token kernel runs one workgroup per (8 tokens, 256 columns) tile, the
    // 3-in-5 kernel one per (token, 16 columns), in one-dimensional grids of at most
    // 2^24 workgroups
    if (p->wfmt == LUTGEMM_WFMT_TERNARY_3IN5) {
        if (((p->N + 15) / 16) * M >= MAX_TILES) return LUTGEMM_ERROR_NOT_SUPPORTED;
    } else if (M > 2 && ((M + 7) / 8) * ((p->N + 255) / 256) >= MAX_TILES) {
        return LUTGEMM_ERROR_NOT_SUPPORTED;
    }
    if (p->K % KBLK != 0) return LUTGEMM_ERROR_NOT_SUPPORTED;
    if (p->group_size != 0 && (p->group_size % KBLK != 0 || p->K % p->group_size != 0))
        return LUTGEMM_ERROR_NOT_SUPPORTED;
    switch (p->wfmt) {
    case LUTGEMM_WFMT_UINT:
        if (p->w_bits != 1 && p->w_bits != 2 && p->w_bits != 4) return LUTGEMM_ERROR_NOT_SUPPORTED;
        if (p->scale_fp32) return LUTGEMM_ERROR_NOT_SUPPORTED;
        break;
    case LUTGEMM_WFMT_BINARY:
        if (p->w_bits != 1) return LUTGEMM_ERROR_NOT_SUPPORTED;
        break;
    case LUTGEMM_WFMT_TERNARY_3IN5:  // triples never straddle a scale: per tensor or per channel only
        if (p->w_bits != 2) return LUTGEMM_ERROR_NOT_SUPPORTED;
        if (p->group_size != 0 && p->group_size != p->K) return LUTGEMM_ERROR_NOT_SUPPORTED;
        break;
    default:
        if (p->w_bits != 2) return LUTGEMM_ERROR_NOT_SUPPORTED;
        break;
    }
    if (p->scale_fp32 && p->group_size != 0) return LUTGEMM_ERROR_NOT_SUPPORTED;
    if (p->act == LUTGEMM_ACT_FP16_LUT8 && p->wfmt == LUTGEMM_WFMT_TERNARY_3IN5) return LUTGEMM_ERROR_NOT_SUPPORTED;
    if (p->act == LUTGEMM_ACT_INT8) {
        if (p->wfmt == LUTGEMM_WFMT_UINT) return LUTGEMM_ERROR_NOT_SUPPORTED;
        if (p->group_size != 0 && p->group_size != p->K) return LUTGEMM_ERROR_NOT_SUPPORTED;
    }
    return LUTGEMM_SUCCESS;
}

// Planner overrides: environment variables read once, when the library is loaded
// (a static initializer), then only changed through lutgemm_set_tuning.
const char *const kTuneEnv[LUTGEMM_TUNE_COUNT] = {
    "LUTGEMM_TARGET_BLOCKS", "LUTGEMM_WHOLEK_MAX_KB", "LUTGEMM_GEMV_KIND", "LUTGEMM_GEMV_CFG",
    "LUTGEMM_SPLITS",        "LUTGEMM_KBS",           "LUTGEMM_MT16",      "LUTGEMM_MT_TARGET",
    "LUTGEMM_MT_SPLITS",     "LUTGEMM_MT_ORDER",      "LUTGEMM_DEQUANT_KIND", "LUTGEMM_LOG",
    "LUTGEMM_SPLIT_PRE",     "LUTGEMM_DEQUANT_SPLITS", "LUTGEMM_MT_FUSED", "LUTGEMM_MT4",
    "LUTGEMM_SPLIT_EXACT"};
const int kTuneDefault[LUTGEMM_TUNE_COUNT] = {256, 10000, -1, -1, 0, 0, 1, 8, 0, -1, -1, 0, -1, 0, -1, 1, 1};
std::atomic<int> g_tune[LUTGEMM_TUNE_COUNT];

bool tune_value_ok(int key, int value) {
    if (value < -1 || value > (1 << 24)) return false;
    if (key == LUTGEMM_TUNE_TARGET_BLOCKS && value == 0) return false;
    return true;
}

struct TuneInit {
    TuneInit() {
        for (int k = 0; k < LUTGEMM_TUNE_COUNT; ++k) {
            int v = kTuneDefault[k];
            const char *e = std::getenv(kTuneEnv[k]);
            if (e && *e) {
                const int x = std::atoi(e);
                if (tune_value_ok(k, x) && x != -1) v = x;
            }
            g_tune[k].store(v, std::memory_order_relaxed);
        }
    }
};
const TuneInit g_tune_init;

thread_local char g_last_error[256] = "";

#ifdef LUTGEMM_TIMELINE
unsigned long long *g_timeline = nullptr;  // instrumented builds: phase-stamp buffer
#endif

lutgemm_status_t hip_status(int e) {
    if (e == 0) return LUTGEMM_SUCCESS;
    std::snprintf(g_last_error, sizeof(g_last_error), "%s (hipError_t %d)",
                  hipGetErrorString((hipError_t)e), e);
    return LUTGEMM_ERROR_HIP;
}

}  // namespace

namespace lutgemm {

int tuning(int key) { return g_tune[key].load(std::memory_order_relaxed); }

void set_last_error(const char *msg) { std::snprintf(g_last_error, sizeof(g_last_error), "%s", msg); }

lutgemm_status_t hip_error(int e) { return e == 0 ? LUTGEMM_SUCCESS : hip_status(e); }

// Work decomposition.
// Single token (M <= 2, one grid layer per token): the GEMV kernel of
// lut_gemv.hip; pick the widest lane decomposition (most columns per workgroup,
// i.e. most table reuse) that still gives at least `target` workgroups, and
// split K across workgroups only when even the narrowest one does not.
// Several tokens: 8 tokens per workgroup of 256 columns, K split only when the
// token x column grid is smaller than 8 x `target` workgroups (to twice that when the
// K ranges stay at least 32 blocks long).
// Whether lutgemm_mpgemm_fused runs the multi-token kernel with its own table build
// (FP16 activations, M > 2).  Every 256-column tile builds the tables of its tokens and
// K range again, work the precompute does once, and the build is vector work in a
// kernel bound by vector issue at large M; measured on MI355X it is faster than
// precompute + mpGEMM up to M = 64 on layers of at most 64 column tiles (INT4 4096 x
// 12288: 18 and 22 us against 22.5 and 25 at M = 4 and 8; binary 28672 x 8192: 21-28
// against 24-30; INT2 4096^2 at M = 64: 25 against 28) and slower beyond (binary 8192
// x 28672, 112 tiles: +1.5 us at M = 16; +17 % at M = 256, +10 % for INT2 at M = 4096).
static bool mtok_fused(const Layout &L, int64_t M) {
    if (L.act != LUTGEMM_ACT_FP16 || M <= 2 || L.tri) return false;
    const int f = tuning(LUTGEMM_TUNE_MT_FUSED);
    if (f >= 0) return f != 0;
    return M <= 64 && L.N_pad / NTILE <= 64;
}

LutPlan plan_lut(const Layout &L, int64_t M, bool fused) {
    LutPlan P{};
    const int64_t target = tuning(LUTGEMM_TUNE_TARGET_BLOCKS);
    const int64_t weight_bytes = L.KB * L.bits * L.N * 16;
    if (L.tri) {  // one token per grid layer, whole K, 16 columns per workgroup (lut_tri.hip)
        P.kind = 3;
        P.mt = 1;
        P.m_tiles = M;
        P.n_tiles = (L.N + 15) / 16;
        P.kbs = (int)L.KB;
        P.splits = 1;
        P.ws_bytes = 0;
        return P;
    }
    int kind = M > 2 ? 1 : (weight_bytes <= (int64_t)tuning(LUTGEMM_TUNE_WHOLEK_MAX_KB) * 1000 ? 0 : 2);
    // with FP16 activations the split-K GEMV and its exact completion also win on
    // smaller layers once one 128-block per workgroup gives 2 x `target` workgroups
    // (measured, table-fed / fused entry, us: INT4 1 x 4096 x 4096 5.3 / 5.5 against the
    // whole-K GEMV's 5.8 / 7.4; INT2 1 x 1024 x 1024, 32 such workgroups, stays whole-K:
    // 3.15 against 3.58); INT8 activations keep the whole-K GEMV (ternary 1 x 4096 x 4096:
    // 4.66 / 4.79 against 4.20 / 4.83).  (INT8-quantized tables are staged as fixed-point
    // entries like FP16 ones, so their partial sums complete exactly too.)
    const bool exact_fmt = M * L.N_pad <= EXACT_MAX && tuning(LUTGEMM_TUNE_SPLIT_EXACT) == 1;
    if (kind == 0 && exact_fmt && L.act != LUTGEMM_ACT_INT8 && (L.N_pad / NTILE) * M * L.KB >= 2 * target &&
        L.KB <= EXACT_MAX_SPLITS)
        kind = 2;
    const int forced_kind = tuning(LUTGEMM_TUNE_GEMV_KIND);
    if (M <= 2 && (forced_kind == 0 || forced_kind == 1 || forced_kind == 2)) kind = forced_kind;
    // the split-K GEMV keeps one arrival counter per (token, 256-column tile); layers with
    // more tiles than the counter area holds fill the GPU without a K split anyway
    if (kind == 2 && M * (L.N_pad / NTILE) > CNT_MAX) kind = 0;
    if (kind == 0) {
        P.kind = 0;
        P.mt = 1;
        P.m_tiles = M;
        // (columns per workgroup, 128-blocks per chunk) of each decomposition, widest first
        static const int b1[2][2] = {{64, 16}, {32, 32}};
        static const int b2[3][2] = {{64, 16}, {32, 16}, {16, 32}};
        static const int b4[3][2] = {{64, 16}, {32, 16}, {16, 16}};
        const int(*cfg)[2] = L.bits == 1 ? b1 : (L.bits == 2 ? b2 : b4);
        const int ncfg = L.bits == 1 ? 2 : 3;
        int pick = ncfg - 1;
        for (int i = 0; i < ncfg; ++i)
            if ((L.N + cfg[i][0] - 1) / cfg[i][0] * M >= target) {
                pick = i;
                break;
            }
        const int forced = tuning(LUTGEMM_TUNE_GEMV_CFG);
        if (forced >= 0 && forced < ncfg) pick = forced;
        P.gemv_cfg = pick;
        const int cw = cfg[pick][0], ck = cfg[pick][1];
        P.n_tiles = (L.N + cw - 1) / cw;
        const int64_t blocks = P.n_tiles * M;
        int64_t splits = 1;
        if (blocks < target) splits = (target + blocks - 1) / blocks;
        const int64_t max_splits = (L.KB + ck - 1) / ck;  // at least one chunk per split
        if (splits > max_splits) splits = max_splits;
        const int fs = tuning(LUTGEMM_TUNE_SPLITS);
        if (fs > 0) splits = fs;
        int64_t kbs = (L.KB + splits - 1) / splits;
        kbs = (kbs + ck - 1) / ck * ck;
        if (kbs > L.KB) kbs = L.KB;
        P.kbs = (int)kbs;
        P.splits = (int)((L.KB + kbs - 1) / kbs);
    } else if (kind == 2) {
        // split-K GEMV: 256 columns per workgroup (one per lane), KBS 128-blocks each, the
        // K split completed inside the kernel.  About eight weight words per lane (KBS =
        // 8 / b): few, long-lived workgroups that the GPU holds all at once, so the
        // end-of-workgroup arrival protocol never delays a waiting workgroup; KBS is
        // halved only while the grid would have fewer than 2 x `target` workgroups.
        // With the exact completion nothing waits: shorter workgroups pay until about
        // 6 x `target` of them, while at most 64 splits add into one output word
        // (measured, us, KBS chosen / the next: INT4 1 x 4096 x 12288 8.4 / 8.9, INT4
        // 1 x 11008 x 4096 8.5 / 9.6, 1-bit 1 x 8192 x 28672 9.7 / 10.7)
        // 1-bit weights, two tokens: both share each workgroup's pass over the weights
        // (with the exact completion; 2 x 8192 x 28672: 17.1 -> 15.0-16.4 us, 2 x 28672 x
        // 8192: 17.0 -> 15.2-15.7).  Wider weights keep a token per workgroup: their
        // two-token kernels hold every lookup of a block in registers (2 x 4096 x 12288
        // INT4: 23.6 against 16.5 us)
        P.kind = 2;
        P.mt = (M == 2 && exact_fmt && L.bits == 1) ? 2 : 1;
        P.m_tiles = (M + P.mt - 1) / P.mt;
        P.n_tiles = L.N_pad / NTILE;
        const int kmax = 8 / L.bits;
        auto n_splits = [&](int k) { return (L.KB + k - 1) / k; };
        int kbs = kmax;
        const int forced = tuning(LUTGEMM_TUNE_KBS);
        if (forced == 1 || forced == 2 || forced == 4 || forced == 8) {
            kbs = forced > kmax ? kmax : forced;
        } else if (exact_fmt) {
            while (kbs > 1 && P.n_tiles * P.m_tiles * n_splits(kbs) < 6 * target && n_splits(kbs >> 1) <= 64)
                kbs >>= 1;
        } else {
            while (kbs > 1 && P.n_tiles * M * n_splits(kbs) < 2 * target) kbs >>= 1;
            // 1-bit weights: four words per lane (twice the workgroups) while the split
            // stays short enough to complete in the kernel (1 x 8192 x 28672: 11.7 -> 10.9 us)
            if (L.bits == 1 && kbs == 8 && n_splits(4) <= INKERNEL_MAX_SPLITS) kbs = 4;
        }
        P.kbs = kbs;
        P.splits = (int)((L.KB + kbs - 1) / kbs);
        // weight words per lane requested before the tables arrive: half of them
        // (measured, table-fed / fused, us: INT4 1 x 4096 x 12288, 4 words: 8.6 / 8.4 at
        // 2 against 9.0 / 8.9 at 4; INT4 1 x 11008 x 4096, 8 words: 8.6 / 8.9 at 4
        // against 8.9 / 9.7 at 2; 1-bit 1 x 8192 x 28672, 4 words: 9.6 / 9.3 at 2
        // against 9.7 / 9.5 at 4)
        const int pre = tuning(LUTGEMM_TUNE_SPLIT_PRE);
        P.pre = pre >= 0 ? pre : ((kbs * L.bits) / 2 > 1 ? (kbs * L.bits) / 2 : 1);
        // Partial sums that are integers (INT8 activations; fixed-point FP16 table entries
        // on weights with one scale per column or tensor) or fixed point (FP16
        // activations, per-column exponent stored with the packed weights) are summed
        // exactly by one 64-bit atomic per output: one memory round trip instead of the
        // four of the arrival protocol, and no limit from a batch of partial loads
        P.exact = P.splits > 1 && P.splits <= EXACT_MAX_SPLITS && exact_fmt;
        P.inkernel = P.exact || (P.splits > 1 && P.splits <= INKERNEL_MAX_SPLITS);
        if (P.inkernel && !P.exact) {  // the arrival protocol takes one token per workgroup
            P.mt = 1;
            P.m_tiles = M;
        }
        // (else the arrival protocol: the last workgroup of a tile loads every split's
        // partial sum in one batch, up to INKERNEL_MAX_SPLITS; beyond that the finalize
        // kernel's wide batches are faster -- measured: 1 x 11008 x 4096 INT4, 43 splits:
        // 15.5 us in the kernel, 11.8 us with the finalize launch)
    } else {
        P.kind = 1;
        // tokens per workgroup of the multi-token kernel (lut_mtok.hip): 16 from M = 16 on
        // (one decoded index serves two token halves), 4 up to M = 4 (half-filled rows,
        // half the LDS bytes and packed adds per lookup), except with INT8-quantized tables
        const int mt16 = tuning(LUTGEMM_TUNE_MT16);
        const bool lut8 = L.act == LUTGEMM_ACT_FP16_LUT8;
        P.mt = (M >= 16 && !lut8 && mt16) ? 16 : ((M <= 4 && !lut8 && tuning(LUTGEMM_TUNE_MT4)) ? 4 : 8);
        P.m_tiles = (M + P.mt - 1) / P.mt;
        P.n_tiles = L.N_pad / NTILE;
        const int64_t base = P.n_tiles * P.m_tiles;
        const int64_t ch = L.bits == 1 ? 1 : 4 / L.bits;  // 128-blocks per chunk of the kernel
        const int64_t mt_target = tuning(LUTGEMM_TUNE_MT_TARGET) * target;
        int64_t splits = 1;
        if (base < mt_target) {
            splits = (mt_target + base - 1) / base;
            // long K ranges stay long enough at twice the grid: take it (1-bit
            // 256 x 28672 x 8192: 2 -> 4 splits, 383 -> 367 us); short ones (M = 16) do not
            const int64_t s2 = (2 * mt_target + base - 1) / base;
            if (L.KB / s2 >= 32) splits = s2;
            // but each split keeps about 6 or more block-planes of lookups: shorter K
            // ranges spend more on pipeline fill and partial sums than the extra
            // workgroups gain (M = 3-8 decode shapes: 8-15 % faster than 19-64 splits)
            const int64_t cap = L.KB * L.bits / 6 > 1 ? L.KB * L.bits / 6 : 1;
            if (splits > cap) splits = cap;
        }
        const int64_t max_splits = (L.KB + ch - 1) / ch;  // at least one chunk per split
        if (splits > max_splits) splits = max_splits;
        const int fs = tuning(LUTGEMM_TUNE_MT_SPLITS);
        if (fs > 0) splits = fs;
        if (splits * base >= MAX_TILES) splits = (MAX_TILES - 1) / base;
        if (splits < 1) splits = 1;
        // the fused table build with zero points keeps each K range's block sums in LDS
        const bool zp_fused = fused && mtok_fused(L, M) && L.wfmt != LUTGEMM_WFMT_BINARY;
        if (zp_fused && (L.KB + splits - 1) / splits > MTOK_FUSED_SMAX) splits = (L.KB + MTOK_FUSED_SMAX - 1) / MTOK_FUSED_SMAX;
        int64_t kbs = (L.KB + splits - 1) / splits;
        kbs = (kbs + ch - 1) / ch * ch;
        if (kbs > L.KB) kbs = L.KB;
        P.kbs = (int)kbs;
        P.splits = (int)((L.KB + kbs - 1) / kbs);
        // (the K split is summed by the finalize kernel: an exact completion with one
        // atomic per output and split measured slower from M = 8 on -- 1-bit 8 x 8192 x
        // 28672: 27-35 us against 23 us; 16 tokens: 48 against 36 us -- as the atomics
        // grow with the token count; equal at M = 4)
        // workgroup order: with 16 or more token tiles and no K split, each XCD walks its
        // own contiguous share of the tiles in bands of 8 token tiles, tokens fastest
        // (the LLaMA-2-13B shape 1616 -> 1579 us, the 4096^3 prefill 704 -> 701 us); else
        // columns fastest (the XCD-aware orders measured up to 18 % slower at M = 16)
        P.order = tuning(LUTGEMM_TUNE_MT_ORDER);
        if (P.order < 0) P.order = (P.m_tiles >= 16 && P.splits == 1) ? 8 : 0;
    }
    const int64_t rows = P.kind == 1 ? P.m_tiles * P.mt : M;
    // [arrival counters: CNT_AREA][partial sums]
    P.part_off = CNT_AREA;
    // (the exact completion needs only the zero region)
    P.ws_bytes = P.splits > 1 ? CNT_AREA + (P.exact ? 0 : align256((size_t)P.splits * rows * L.N_pad * 4)) : 0;
    return P;
}

}  // namespace lutgemm

namespace lutgemm {

// Kernel parameters of one LUT mpGEMM call (tables in the layout of lutgemm_table_size).
static LutParams lut_params(const Layout &L, const LutPlan &plan, int64_t M, const void *tables,
                            const void *packed, void *out, int32_t out_dtype, int32_t accumulate,
                            void *workspace) {
    TableLayout T = make_table_layout(L, M);
    LutParams lp{};
    lp.T = (const uint4 *)tables;
    lp.tsc = tables && L.act == LUTGEMM_ACT_FP16_LUT8 ? (const float *)((const char *)tables + T.sc_off) : nullptr;
    lp.S = tables ? (const char *)tables + T.s_off : nullptr;
    lp.tok = tables ? (const float *)((const char *)tables + T.tok_off) : nullptr;
    lp.planes = (const uint4 *)packed;
    lp.sgn = L.tri ? (const uint32_t *)((const char *)packed + L.sgn_off) : nullptr;
    lp.meta = (const char *)packed + L.meta_off;
    lp.out = out;
    lp.part = plan.splits > 1 && !plan.exact ? (float *)((char *)workspace + plan.part_off) : nullptr;
    lp.cnt = plan.kind == 2 && plan.inkernel ? (uint32_t *)workspace : nullptr;
    lp.acc64 = plan.kind == 2 && plan.exact ? (unsigned long long *)((char *)workspace + CNT_BYTES) : nullptr;
    lp.bnd = (const int *)((const char *)packed + L.bnd_off);
    lp.M = M;
    lp.N = L.N;
    lp.N_pad = L.N_pad;
    lp.K = L.K;
    lp.KB = L.KB;
    lp.J = L.J;
    lp.Q = L.Q;
    lp.G = L.G;
    lp.splits = plan.splits;
    lp.kbs = plan.kbs;
    lp.kpg = (int)(L.G / KBLK);
    lp.per_tensor = L.per_tensor ? 1 : 0;
    lp.inv_kpg = 1.0f / (float)lp.kpg;
    format_consts(L.wfmt, L.bits, lp.cs, lp.cz, lp.c0);
    lp.out_dtype = out_dtype;
    lp.accumulate = accumulate;
#ifdef LUTGEMM_TIMELINE
    lp.tl = g_timeline;
#endif
    return lp;
}

static void log_plan(const char *who, const Layout &L, const LutPlan &plan, int64_t M) {
    std::fprintf(stderr, "%s: M=%lld K=%lld N=%lld b=%d kind=%d cfg=%d kbs=%d splits=%d mt=%d grid=%lldx%dx%lld\n",
                 who, (long long)M, (long long)L.K, (long long)L.N, L.bits, plan.kind, plan.gemv_cfg,
                 plan.kbs, plan.splits, plan.mt, (long long)plan.n_tiles, plan.splits, (long long)plan.m_tiles);
}

// Scratch of lutgemm_mpgemm_fused: the plan's workspace (counters, partial sums) at
// offset 0 as for lutgemm_mpgemm, then the per-token factors when the fused GEMV
// splits K, or the staged tables when the call runs precompute + mpGEMM.  (The fused
// multi-token kernel stores its partial sums already multiplied by the token factors.)
struct FusedScratch {
    bool fused;
    size_t tables, tables_off, tok_off, total;
};

static FusedScratch fused_scratch(const Layout &L, const LutPlan &plan, int64_t M) {
    FusedScratch f{};
    // INT8 table quantization exists to shrink the tables that travel through HBM, so
    // that mode always takes the two-call path; with INT8 activations the split-K GEMV's
    // workgroups read the whole token for the quantizer's absmax, while the multi-token
    // kernel (several tokens, K split across workgroups) takes the two-call path
    f.fused = ((plan.kind == 0 || plan.kind == 2 || plan.kind == 3) && L.act != LUTGEMM_ACT_FP16_LUT8) ||
              (plan.kind == 1 && mtok_fused(L, M));
    if (f.fused && plan.kind == 1) {
        f.total = plan.ws_bytes;
    } else if (f.fused) {
        // (token factors for the finalize kernel; not with the exact completion)
        f.tok_off = plan.ws_bytes;
        f.total = plan.splits > 1 ? plan.ws_bytes + (plan.exact ? 0 : align256((size_t)M * 4)) : 0;
    } else {
        f.tables = make_table_layout(L, M).total;
        f.tables_off = align256(plan.ws_bytes);
        f.total = f.tables_off + f.tables;
    }
    return f;
}

}  // namespace lutgemm

extern "C" {

const char *lutgemm_status_string(lutgemm_status_t s) {
    switch (s) {
    case LUTGEMM_SUCCESS: return "LUTGEMM_SUCCESS";
    case LUTGEMM_ERROR_INVALID_VALUE: return "LUTGEMM_ERROR_INVALID_VALUE";
    case LUTGEMM_ERROR_NOT_SUPPORTED: return "LUTGEMM_ERROR_NOT_SUPPORTED";
    case LUTGEMM_ERROR_INSUFFICIENT_SIZE: return "LUTGEMM_ERROR_INSUFFICIENT_SIZE";
    case LUTGEMM_ERROR_HIP: return "LUTGEMM_ERROR_HIP";
    }
    return "LUTGEMM_UNKNOWN_STATUS";
}

const char *lutgemm_version(void) { return "lutgemm-gfx950 0.1.0"; }

const char *lutgemm_last_error(void) { return g_last_error; }

#ifdef LUTGEMM_TIMELINE
// Instrumented builds only (not declared in lutgemm.h): the device buffer that the
// single-token kernels write their per-wavefront phase stamps to (NULL: none).
void lutgemm_timeline_set(void *buf) { g_timeline = (unsigned long long *)buf; }
#endif

lutgemm_status_t lutgemm_set_tuning(int32_t key, int32_t value) {
    if (key < 0 || key >= LUTGEMM_TUNE_COUNT || !tune_value_ok(key, value)) return LUTGEMM_ERROR_INVALID_VALUE;
    g_tune[key].store(value == -1 ? kTuneDefault[key] : value, std::memory_order_relaxed);
    return LUTGEMM_SUCCESS;
}

int32_t lutgemm_get_tuning(int32_t key) {
    if (key < 0 || key >= LUTGEMM_TUNE_COUNT) return -2;
    return g_tune[key].load(std::memory_order_relaxed);
}

lutgemm_status_t lutgemm_validate(const lutgemm_problem_t *problem, int64_t M) {
    return check_problem(problem, M);
}

size_t lutgemm_packed_weight_size(const lutgemm_problem_t *problem) {
    if (check_problem(problem, 1) != LUTGEMM_SUCCESS) return 0;
    return make_layout(*problem).packed_bytes;
}

size_t lutgemm_table_size(const lutgemm_problem_t *problem, int64_t M) {
    if (check_problem(problem, M) != LUTGEMM_SUCCESS) return 0;
    return make_table_layout(make_layout(*problem), M).total;
}

lutgemm_status_t lutgemm_table_offsets(const lutgemm_problem_t *problem, int64_t M, size_t *s_offset,
                                       size_t *t_offset) {
    lutgemm_status_t st = check_problem(problem, M);
    if (st != LUTGEMM_SUCCESS) return st;
    if (!s_offset || !t_offset) return LUTGEMM_ERROR_INVALID_VALUE;
    TableLayout T = make_table_layout(make_layout(*problem), M);
    *s_offset = T.s_off;
    *t_offset = T.tok_off;
    return LUTGEMM_SUCCESS;
}

size_t lutgemm_workspace_size(const lutgemm_problem_t *problem, int64_t M) {
    if (check_problem(problem, M) != LUTGEMM_SUCCESS) return 0;
    Layout L = make_layout(*problem);
    return plan_lut(L, M).ws_bytes;
}

lutgemm_status_t lutgemm_pack_weights(const lutgemm_problem_t *problem, const void *codes,
                                      const void *scales, const void *zeros, void *packed,
                                      size_t packed_bytes, void *stream) {
    lutgemm_status_t st = check_problem(problem, 1);
    if (st != LUTGEMM_SUCCESS) return st;
    if (!codes || !scales || !packed) return LUTGEMM_ERROR_INVALID_VALUE;
    if (problem->wfmt == LUTGEMM_WFMT_UINT && !zeros) return LUTGEMM_ERROR_INVALID_VALUE;
    if (!aligned16(codes) || !aligned16(scales) || !aligned16(packed)) return LUTGEMM_ERROR_INVALID_VALUE;
    if (problem->wfmt == LUTGEMM_WFMT_UINT && !aligned16(zeros)) return LUTGEMM_ERROR_INVALID_VALUE;
    Layout L = make_layout(*problem);
    if (packed_bytes < L.packed_bytes) return LUTGEMM_ERROR_INSUFFICIENT_SIZE;
    PackParams pp{};
    pp.codes = codes;
    pp.scales = scales;
    pp.zeros = problem->wfmt == LUTGEMM_WFMT_UINT ? zeros : nullptr;
    pp.planes = (uint4 *)packed;
    pp.sgn = L.tri ? (uint32_t *)((char *)packed + L.sgn_off) : nullptr;
    pp.meta = (char *)packed + L.meta_off;
    pp.bnd = (int *)((char *)packed + L.bnd_off);
    pp.K = L.K;
    pp.N = L.N;
    pp.N_pad = L.N_pad;
    pp.KB = L.KB;
    pp.Q = L.Q;
    pp.G = L.G;
    pp.bits = L.bits;
    pp.wfmt = L.wfmt;
    pp.per_tensor = L.per_tensor ? 1 : 0;
    pp.scale_fp32 = problem->scale_fp32;
    return hip_status(launch_pack(pp, stream));
}

lutgemm_status_t lutgemm_precompute(const lutgemm_problem_t *problem, int64_t M, const void *act,
                                    void *tables, size_t table_bytes, void *stream) {
    lutgemm_status_t st = check_problem(problem, M);
    if (st != LUTGEMM_SUCCESS) return st;
    if (!act || !tables || !aligned16(act) || !aligned16(tables)) return LUTGEMM_ERROR_INVALID_VALUE;
    Layout L = make_layout(*problem);
    TableLayout T = make_table_layout(L, M);
    if (table_bytes < T.total) return LUTGEMM_ERROR_INSUFFICIENT_SIZE;
    PrecomputeParams pp{};
    pp.act = (const uint16_t *)act;
    pp.T = (uint4 *)tables;
    pp.S = (char *)tables + T.s_off;
    pp.tok = (float *)((char *)tables + T.tok_off);
    pp.M = M;
    pp.K = L.K;
    pp.J = L.J;
    pp.Q = L.Q;
    pp.G = L.G;
    pp.tri = L.tri ? 1 : 0;
    pp.tsc = L.act == LUTGEMM_ACT_FP16_LUT8 ? (float *)((char *)tables + T.sc_off) : nullptr;
    return hip_status(launch_precompute(pp, L.act == LUTGEMM_ACT_INT8, stream));
}

lutgemm_status_t lutgemm_mpgemm(const lutgemm_problem_t *problem, int64_t M, const void *tables,
                                const void *packed, void *out, int32_t out_dtype, int32_t accumulate,
                                void *workspace, size_t workspace_bytes, void *stream) {
    lutgemm_status_t st = check_problem(problem, M);
    if (st != LUTGEMM_SUCCESS) return st;
    if (!tables || !packed || !out) return LUTGEMM_ERROR_INVALID_VALUE;
    if (!aligned16(tables) || !aligned16(packed) || !aligned16(out)) return LUTGEMM_ERROR_INVALID_VALUE;
    if (out_dtype != LUTGEMM_OUT_FP16 && out_dtype != LUTGEMM_OUT_FP32 && out_dtype != LUTGEMM_OUT_INT32)
        return LUTGEMM_ERROR_INVALID_VALUE;
    if (out_dtype == LUTGEMM_OUT_INT32 && problem->act != LUTGEMM_ACT_INT8) return LUTGEMM_ERROR_NOT_SUPPORTED;
    if (accumulate != 0 && accumulate != 1) return LUTGEMM_ERROR_INVALID_VALUE;
    Layout L = make_layout(*problem);
    LutPlan plan = plan_lut(L, M);
    if (plan.ws_bytes > 0) {
        if (!workspace || !aligned16(workspace)) return LUTGEMM_ERROR_INVALID_VALUE;
        if (workspace_bytes < plan.ws_bytes) return LUTGEMM_ERROR_INSUFFICIENT_SIZE;
    }
    LutParams lp = lut_params(L, plan, M, tables, packed, out, out_dtype, accumulate, workspace);
    if (tuning(LUTGEMM_TUNE_LOG)) log_plan("lutgemm_mpgemm", L, plan, M);
    return hip_status(launch_lut(lp, L, plan, stream));
}

size_t lutgemm_fused_workspace_size(const lutgemm_problem_t *problem, int64_t M) {
    if (check_problem(problem, M) != LUTGEMM_SUCCESS) return 0;
    Layout L = make_layout(*problem);
    return fused_scratch(L, plan_lut(L, M, true), M).total;
}

lutgemm_status_t lutgemm_mpgemm_fused(const lutgemm_problem_t *problem, int64_t M, const void *act,
                                      const void *packed, void *out, int32_t out_dtype, int32_t accumulate,
                                      void *workspace, size_t workspace_bytes, void *stream) {
    lutgemm_status_t st = check_problem(problem, M);
    if (st != LUTGEMM_SUCCESS) return st;
    if (!act || !packed || !out) return LUTGEMM_ERROR_INVALID_VALUE;
    if (!aligned16(act) || !aligned16(packed) || !aligned16(out)) return LUTGEMM_ERROR_INVALID_VALUE;
    if (out_dtype != LUTGEMM_OUT_FP16 && out_dtype != LUTGEMM_OUT_FP32 && out_dtype != LUTGEMM_OUT_INT32)
        return LUTGEMM_ERROR_INVALID_VALUE;
    if (out_dtype == LUTGEMM_OUT_INT32 && problem->act != LUTGEMM_ACT_INT8) return LUTGEMM_ERROR_NOT_SUPPORTED;
    if (accumulate != 0 && accumulate != 1) return LUTGEMM_ERROR_INVALID_VALUE;
    Layout L = make_layout(*problem);
    LutPlan plan = plan_lut(L, M, true);
    FusedScratch fs = fused_scratch(L, plan, M);
    if (fs.total > 0) {
        if (!workspace || !aligned16(workspace)) return LUTGEMM_ERROR_INVALID_VALUE;
        if (workspace_bytes < fs.total) return LUTGEMM_ERROR_INSUFFICIENT_SIZE;
    }
    char *ws = (char *)workspace;
    if (tuning(LUTGEMM_TUNE_LOG)) log_plan(fs.fused ? "lutgemm_mpgemm_fused" : "lutgemm_mpgemm_fused(unfused)", L, plan, M);
    if (!fs.fused) {  // precompute into the workspace, then the table-fed kernels
        st = lutgemm_precompute(problem, M, act, ws + fs.tables_off, fs.tables, stream);
        if (st != LUTGEMM_SUCCESS) return st;
        LutParams lp = lut_params(L, plan, M, ws + fs.tables_off, packed, out, out_dtype, accumulate, ws);
        return hip_status(launch_lut(lp, L, plan, stream));
    }
    LutParams lp = lut_params(L, plan, M, nullptr, packed, out, out_dtype, accumulate, ws);
    lp.act = (const uint16_t *)act;
    if (plan.kind == 3) return hip_status(launch_tri(lp, L, true, stream));
    if (plan.kind == 1) {  // tables from the FP16 activations inside the multi-token kernel
        int e = launch_mtok_fused(lp, L, plan, stream);
        if (e == 0 && plan.splits > 1) e = launch_finalize(lp, L, plan, stream);
        return hip_status(e);
    }
    if (plan.kind == 2) {  // tables from the activations of each K range, then the split sum
        // INT8: the kernel forms the token factor itself; the finalize kernel (long K
        // splits) takes it from the workspace
        lp.tok_out = (L.act == LUTGEMM_ACT_INT8 && plan.splits > 1 && !plan.exact) ? (float *)(ws + fs.tok_off) : nullptr;
        int e = launch_fused_split(lp, L, plan, stream);
        if (e == 0 && plan.splits > 1 && !plan.inkernel) {
            lp.tok = lp.tok_out;
            e = launch_finalize(lp, L, plan, stream);
        }
        return hip_status(e);
    }
    lp.tok_out = plan.splits > 1 ? (float *)(ws + fs.tok_off) : nullptr;
    int e = launch_fused_gemv(lp, L, plan, stream);
    if (e == 0 && plan.splits > 1) {
        lp.tok = lp.tok_out;  // the finalize kernel scales with the factors the fused kernel wrote
        e = launch_finalize(lp, L, plan, stream);
    }
    return hip_status(e);
}

size_t lutgemm_dequant_workspace_size(const lutgemm_problem_t *problem, int64_t M) {
    if (check_problem(problem, M) != LUTGEMM_SUCCESS) return 0;
    if (problem->act == LUTGEMM_ACT_INT8 || problem->wfmt == LUTGEMM_WFMT_TERNARY_3IN5) return 0;
    return plan_dequant(make_layout(*problem), M).ws_bytes;
}

lutgemm_status_t lutgemm_dequant_plan(const lutgemm_problem_t *problem, int64_t M, int32_t *kernel,
                                      int32_t *splits) {
    lutgemm_status_t st = check_problem(problem, M);
    if (st != LUTGEMM_SUCCESS) return st;
    if (problem->act == LUTGEMM_ACT_INT8 || problem->wfmt == LUTGEMM_WFMT_TERNARY_3IN5)
        return LUTGEMM_ERROR_NOT_SUPPORTED;
    if (!kernel || !splits) return LUTGEMM_ERROR_INVALID_VALUE;
    const DequantPlan plan = plan_dequant(make_layout(*problem), M);
    *kernel = plan.kind;
    *splits = plan.splits;
    return LUTGEMM_SUCCESS;
}

lutgemm_status_t lutgemm_mpgemm_dequant(const lutgemm_problem_t *problem, int64_t M, const void *act,
                                        const void *packed, void *out, int32_t out_dtype,
                                        int32_t accumulate, void *workspace, size_t workspace_bytes,
                                        void *stream) {
    lutgemm_status_t st = check_problem(problem, M);
    if (st != LUTGEMM_SUCCESS) return st;
    if (problem->act == LUTGEMM_ACT_INT8 || problem->wfmt == LUTGEMM_WFMT_TERNARY_3IN5)
        return LUTGEMM_ERROR_NOT_SUPPORTED;
    if (!act || !packed || !out) return LUTGEMM_ERROR_INVALID_VALUE;
    if (!aligned16(act) || !aligned16(packed) || !aligned16(out)) return LUTGEMM_ERROR_INVALID_VALUE;
    if (out_dtype != LUTGEMM_OUT_FP16 && out_dtype != LUTGEMM_OUT_FP32) return LUTGEMM_ERROR_INVALID_VALUE;
    if (accumulate != 0 && accumulate != 1) return LUTGEMM_ERROR_INVALID_VALUE;
    Layout L = make_layout(*problem);
    DequantParams dp{};
    dp.act = (const uint16_t *)act;
    dp.planes = (const uint4 *)packed;
    dp.meta = (const char *)packed + L.meta_off;
    dp.out = out;
    dp.M = M;
    dp.N = L.N;
    dp.N_pad = L.N_pad;
    dp.K = L.K;
    dp.KB = L.KB;
    dp.Q = L.Q;
    dp.G = L.G;
    dp.out_dtype = out_dtype;
    dp.accumulate = accumulate;
    const DequantPlan plan = plan_dequant(L, M);
    if (plan.ws_bytes) {
        if (!workspace || !aligned16(workspace)) return LUTGEMM_ERROR_INVALID_VALUE;
        if (workspace_bytes < plan.ws_bytes) return LUTGEMM_ERROR_INSUFFICIENT_SIZE;
        dp.part = (float *)workspace;
    }
    dp.splits = plan.splits;
    dp.kbs = plan.kbs;
    if (tuning(LUTGEMM_TUNE_LOG) > 0)
        std::fprintf(stderr, "lutgemm_mpgemm_dequant: M=%lld K=%lld N=%lld kind=%d splits=%d kbs=%d ws=%zu\n",
                (long long)M, (long long)L.K, (long long)L.N, plan.kind, plan.splits, plan.kbs, plan.ws_bytes);
    return hip_status(launch_dequant(dp, L, plan, stream));
}

}  // extern "C"
