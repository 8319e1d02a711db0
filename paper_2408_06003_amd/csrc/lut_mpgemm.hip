// The split-K finalize kernel and the dispatch of lutgemm_mpgemm (LUT Tensor
// Core, Section 3.1 with Eq. 3, 5 and 6; LMMA semantics O = A x W^T + Acc,
// Section 3.3.1): single tokens go to the GEMV kernels of lut_gemv.hip, several
// tokens to the multi-token kernel of lut_mtok.hip, ternary 3-in-5 weights to
// lut_tri.hip.  When the grid would not fill
// the GPU, K is split across workgroups and lut_finalize_kernel sums the partials
// in split order after the LUT kernel ends.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>

#include "lut_common.h"

namespace lutgemm {

// ------------------------------------------------------------------ split-K finalize

// Sums the split partials of output (m, n) in split order and applies the output
// epilogue.  Runs after the LUT kernel on the same stream, so the kernel boundary
// makes every partial visible without fences inside the LUT kernel.  (Completing
// the sum inside the LUT kernel instead, by its last workgroup per column tile,
// needs a device-scope release per workgroup, i.e. an L2 write-back; measured on
// MI355X that costs far more than this launch.)  The first PB partials are
// requested before the epilogue operands, so the kernel waits about one memory
// latency for up to PB splits; PB is the smallest power of two covering the
// splits (at most FIN_BATCH), so few splits issue few loads.  NT lanes per
// workgroup, one per padded column.
template <bool INT8, int PB, int NT>
__global__ __launch_bounds__(NT) void lut_finalize_kernel(LutParams p, int wfmt, int per_tensor_i,
                                                          int64_t m_alloc) {
    const int64_t n = (int64_t)blockIdx.x * NT + threadIdx.x;
    const int64_t m = blockIdx.y;
    float v[PB];
    load_partials<PB>(p, m_alloc, m, n, 0, v);
    const Epi ep = load_epi<INT8>(p, wfmt, m, n, false);
    float sf = 0.f;
    int si = 0;
    add_partials<INT8, PB>(p, 0, v, sf, si);
    for (int s0 = PB; s0 < p.splits; s0 += PB) {
        load_partials<PB>(p, m_alloc, m, n, s0, v);
        add_partials<INT8, PB>(p, s0, v, sf, si);
    }
    store_out<INT8>(p, wfmt, m, n, sf, si, ep);
}

template <bool INT8, int NT>
static void launch_finalize_pb(const LutParams &p, const Layout &L, int pt, int64_t m_alloc, hipStream_t s) {
    const dim3 grid((unsigned)(L.N_pad / NT), (unsigned)p.M);
    const int sp = p.splits;
    if (sp <= 4)
        hipLaunchKernelGGL((lut_finalize_kernel<INT8, 4, NT>), grid, dim3(NT), 0, s, p, L.wfmt, pt, m_alloc);
    else if (sp <= 8)
        hipLaunchKernelGGL((lut_finalize_kernel<INT8, 8, NT>), grid, dim3(NT), 0, s, p, L.wfmt, pt, m_alloc);
    else if (sp <= 16)
        hipLaunchKernelGGL((lut_finalize_kernel<INT8, 16, NT>), grid, dim3(NT), 0, s, p, L.wfmt, pt, m_alloc);
    else if (sp <= 32)
        hipLaunchKernelGGL((lut_finalize_kernel<INT8, 32, NT>), grid, dim3(NT), 0, s, p, L.wfmt, pt, m_alloc);
    else
        hipLaunchKernelGGL((lut_finalize_kernel<INT8, FIN_BATCH, NT>), grid, dim3(NT), 0, s, p, L.wfmt, pt, m_alloc);
}

// ------------------------------------------------------------------ dispatch

int launch_lut(const LutParams &p, const Layout &L, const LutPlan &plan, void *stream) {
    hipStream_t s = (hipStream_t)stream;
    if (plan.kind == 3) return launch_tri(p, L, false, stream);
    if (plan.kind != 1) {
        const int e0 = launch_gemv(p, L, plan, stream);
        if (e0 != 0) return e0;
    } else {
        const int e0 = launch_mtok(p, L, plan, stream);
        if (e0 != 0) return e0;
    }
    hipError_t e = hipGetLastError();
    // the split-K GEMV (kind 2) completes short K splits itself
    if (e != hipSuccess || plan.splits == 1 || (plan.kind == 2 && plan.inkernel)) return (int)e;
    return launch_finalize(p, L, plan, stream);
}

// Sums the K-split partials of the LUT kernel (after it, on the same stream).
int launch_finalize(const LutParams &p, const Layout &L, const LutPlan &plan, void *stream) {
    hipStream_t s = (hipStream_t)stream;
    const int64_t m_alloc = plan.kind == 1 ? plan.m_tiles * plan.mt : p.M;
    const int pt = L.per_tensor ? 1 : 0;
    // single tokens: 64-lane workgroups spread the few columns over many CUs; several
    // tokens: 256 lanes, a quarter of the workgroups
    const bool wide = p.M > 2;
    if (L.act == LUTGEMM_ACT_INT8) {
        if (wide) launch_finalize_pb<true, 256>(p, L, pt, m_alloc, s);
        else launch_finalize_pb<true, 64>(p, L, pt, m_alloc, s);
    } else {
        if (wide) launch_finalize_pb<false, 256>(p, L, pt, m_alloc, s);
        else launch_finalize_pb<false, 64>(p, L, pt, m_alloc, s);
    }
    return (int)hipGetLastError();
}

}  // namespace lutgemm
