// Multi-token bit-serial LUT mpGEMM (LUT Tensor Core, Section 3.1 with Eq. 3,
// 5 and 6; LMMA semantics O = A x W^T + Acc, Section 3.3.1), the split-K
// finalize kernel, and the dispatch of lutgemm_mpgemm.
//
// gfx950 mapping of the multi-token kernel.  Each lane owns one output column for
// MT tokens and a workgroup covers 256 columns, so one table entry read from LDS
// serves every column of the workgroup, all lanes of a wavefront read the same
// 16-entry table at a time (no LDS bank conflicts), and a wavefront's weight
// loads are 1 KiB contiguous 128-bit loads.  The weight index of a lookup is
// decoded once and reused for the MT tokens' tables.  Tables are staged per chunk
// of CH 128-blocks as full signed INT32 tables (see lut_gemv.hip).  When the grid
// would not fill the GPU, K is split across workgroups and lut_finalize_kernel
// sums the partials in split order after the kernel ends.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>

#include "lut_common.h"

namespace lutgemm {

// ------------------------------------------------------------------ several tokens

constexpr int CH = 2;  // 128-blocks of K staged in LDS at a time

template <int BITS, int MT, bool INT8>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void lut_gemm_kernel(LutParams p, int wfmt, int per_tensor_i) {
    __shared__ __attribute__((aligned(16))) int F[MT * CH * GPB * 16];
    const bool per_tensor = per_tensor_i != 0;
    const int tid = threadIdx.x;
    const int64_t n = (int64_t)blockIdx.x * NTILE + tid;
    const int split = blockIdx.y;
    const int64_t m0 = (int64_t)blockIdx.z * MT;
    const int64_t kb_begin = (int64_t)split * p.kbs;
    const int64_t kb_end = (kb_begin + p.kbs < p.KB) ? kb_begin + p.kbs : p.KB;
    const char *Fb = (const char *)F;

    float yf[MT];
    int yi[MT];
#pragma unroll
    for (int r = 0; r < MT; ++r) {
        yf[r] = 0.f;
        yi[r] = 0;
    }

    if (INT8 && split == 0 && wfmt == LUTGEMM_WFMT_TERNARY) {
#pragma unroll
        for (int r = 0; r < MT; ++r)
            if (m0 + r < p.M) yi[r] = ((const int *)p.S)[(m0 + r) * p.Q];
    }
    int q = (int)(kb_begin / p.kpg);
    int phase = (int)(kb_begin - (int64_t)q * p.kpg);
    for (int64_t kc = kb_begin; kc < kb_end; kc += CH) {
        const int nkb = (int)((kb_end - kc) < CH ? (kb_end - kc) : CH);
        uint4 w[CH][BITS];
#pragma unroll
        for (int kbl = 0; kbl < CH; ++kbl) {
            if (kbl < nkb) {
#pragma unroll
                for (int t = 0; t < BITS; ++t) w[kbl][t] = p.planes[((kc + kbl) * BITS + t) * p.N_pad + n];
            }
        }
        // epilogue operands of this chunk, fetched before the lookups (see the GEMV kernel)
        float e_scale[CH], e_zero[CH][MT];
#pragma unroll
        for (int kbl = 0; kbl < CH; ++kbl) {
            e_scale[kbl] = 0.f;
#pragma unroll
            for (int r = 0; r < MT; ++r) e_zero[kbl][r] = 0.f;
            if (!INT8 && kbl < nkb) {
                const SZ sz = load_sz(p, q, n);
                e_scale[kbl] = sz.sp * (1.0f / (float)(1 << FIX_SHIFT));
                if (phase == 0) {
#pragma unroll
                    for (int r = 0; r < MT; ++r) {
                        const int64_t mr = (m0 + r < p.M) ? m0 + r : p.M - 1;  // rows past M are never stored
                        e_zero[kbl][r] = sz.sp * sz.zp * ((const float *)p.S)[mr * p.Q + q];
                    }
                }
            }
            if (kbl < nkb && ++phase == p.kpg) {
                phase = 0;
                ++q;
            }
        }
        __syncthreads();  // previous chunk's tables are no longer read
        for (int e = tid; e < MT * CH * GPB; e += 256) {
            const int r = e / (CH * GPB);
            const int jl = e % (CH * GPB);
            int *dst = F + e * 16;
            if (m0 + r < p.M && jl < nkb * GPB) {
                expand_table<INT8>(p.T[(m0 + r) * p.J + kc * GPB + jl], dst);
            } else {
                int4 *d4 = (int4 *)dst;
                d4[0] = d4[1] = d4[2] = d4[3] = make_int4(0, 0, 0, 0);
            }
        }
        __syncthreads();

#pragma unroll
        for (int kbl = 0; kbl < CH; ++kbl) {
            if (kbl < nkb) {
                int acc[MT][BITS];
#pragma unroll
                for (int t = 0; t < BITS; ++t) {
#pragma unroll
                    for (int r = 0; r < MT; ++r) acc[r][t] = 0;
                    const uint32_t wd[4] = {w[kbl][t].x, w[kbl][t].y, w[kbl][t].z, w[kbl][t].w};
#pragma unroll
                    for (int d = 0; d < 4; ++d) {
                        const uint32_t lo = wd[d] << 2, hi = wd[d] >> 2;
                        const uint32_t a[8] = {idx4<0>(lo), idx4<0>(hi), idx4<1>(lo), idx4<1>(hi),
                                               idx4<2>(lo), idx4<2>(hi), idx4<3>(lo), idx4<3>(hi)};
                        const uint32_t g = (uint32_t)((kbl * GPB + d * 8) * 64);
#pragma unroll
                        for (int r = 0; r < MT; ++r) {
                            const char *Fr = Fb + r * (CH * GPB * 64) + g;
#pragma unroll
                            for (int i = 0; i < 8; i += 2)
                                acc[r][t] += lds_i32(Fr + i * 64, a[i]) + lds_i32(Fr + (i + 1) * 64, a[i + 1]);
                        }
                    }
                }
                int tot[MT];
#pragma unroll
                for (int r = 0; r < MT; ++r) {
                    tot[r] = 0;
#pragma unroll
                    for (int t = 0; t < BITS; ++t) tot[r] += acc[r][t] << t;
                }
#pragma unroll
                for (int r = 0; r < MT; ++r) {
                    if (INT8)
                        yi[r] += tot[r];
                    else
                        yf[r] = fmaf(e_scale[kbl], (float)tot[r], yf[r]) - e_zero[kbl][r];
                }
            }
        }
    }
    const int rows = (int)((p.M - m0) < MT ? (p.M - m0) : MT);
    if (p.splits == 1) {
#pragma unroll
        for (int r = 0; r < MT; ++r)
            if (r < rows) store_out<INT8>(p, wfmt, m0 + r, n, yf[r], yi[r], load_epi<INT8>(p, wfmt, m0 + r, n, false));
        return;
    }
    float vals[MT];
#pragma unroll
    for (int r = 0; r < MT; ++r) vals[r] = INT8 ? __int_as_float(yi[r]) : yf[r];
    const int64_t m_alloc = (int64_t)gridDim.z * MT;
#pragma unroll
    for (int r = 0; r < MT; ++r) p.part[((int64_t)split * m_alloc + m0 + r) * p.N_pad + n] = vals[r];
}

// ------------------------------------------------------------------ split-K finalize

// Sums the split partials of output (m, n) in split order and applies the output
// epilogue.  Runs after the LUT kernel on the same stream, so the kernel boundary
// makes every partial visible without fences inside the LUT kernel.
template <bool INT8>
__global__ __launch_bounds__(64) void lut_finalize_kernel(LutParams p, int wfmt, int per_tensor_i,
                                                          int64_t m_alloc) {
    const int64_t n = (int64_t)blockIdx.x * 64 + threadIdx.x;
    const int64_t m = blockIdx.y;
    const Epi ep = load_epi<INT8>(p, wfmt, m, n, false);
    float sf;
    int si;
    sum_partials<INT8>(p, m_alloc, m, n, sf, si);
    store_out<INT8>(p, wfmt, m, n, sf, si, ep);
}

// ------------------------------------------------------------------ dispatch

template <int BITS, bool INT8>
static void launch_gemm_mt(const LutParams &p, const Layout &L, const LutPlan &plan, hipStream_t s) {
    dim3 grid((unsigned)plan.n_tiles, (unsigned)plan.splits, (unsigned)plan.m_tiles);
    const int pt = L.per_tensor ? 1 : 0;
    if (plan.mt == 4 || BITS == 4)  // the planner uses 4 tokens per workgroup for 4-bit weights
        hipLaunchKernelGGL((lut_gemm_kernel<BITS, 4, INT8>), grid, dim3(256), 0, s, p, L.wfmt, pt);
    else if constexpr (BITS != 4)
        hipLaunchKernelGGL((lut_gemm_kernel<BITS, 8, INT8>), grid, dim3(256), 0, s, p, L.wfmt, pt);
}

template <bool INT8>
static void launch_bits(const LutParams &p, const Layout &L, const LutPlan &plan, hipStream_t s) {
    if (L.bits == 1) launch_gemm_mt<1, INT8>(p, L, plan, s);
    else if (L.bits == 2) launch_gemm_mt<2, INT8>(p, L, plan, s);
    else launch_gemm_mt<4, INT8>(p, L, plan, s);
}

int launch_lut(const LutParams &p, const Layout &L, const LutPlan &plan, void *stream) {
    hipStream_t s = (hipStream_t)stream;
    if (plan.kind != 1) {
        const int e0 = launch_gemv(p, L, plan, stream);
        if (e0 != 0) return e0;
    } else if (L.act == LUTGEMM_ACT_INT8) {
        launch_bits<true>(p, L, plan, s);
    } else {
        launch_bits<false>(p, L, plan, s);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || plan.splits == 1) return (int)e;
    return launch_finalize(p, L, plan, stream);
}

// Sums the K-split partials of the LUT kernel (after it, on the same stream).
int launch_finalize(const LutParams &p, const Layout &L, const LutPlan &plan, void *stream) {
    hipStream_t s = (hipStream_t)stream;
    const int64_t m_alloc = plan.kind == 1 ? plan.m_tiles * plan.mt : p.M;
    const dim3 grid((unsigned)(L.N_pad / 64), (unsigned)p.M);  // one lane per padded column
    const int pt = L.per_tensor ? 1 : 0;
    if (L.act == LUTGEMM_ACT_INT8)
        hipLaunchKernelGGL(lut_finalize_kernel<true>, grid, dim3(64), 0, s, p, L.wfmt, pt, m_alloc);
    else
        hipLaunchKernelGGL(lut_finalize_kernel<false>, grid, dim3(64), 0, s, p, L.wfmt, pt, m_alloc);
    return (int)hipGetLastError();
}

}  // namespace lutgemm
