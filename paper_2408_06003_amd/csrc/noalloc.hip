// lutgemm_mpgemm_noalloc: the LUT mpGEMM of lutgemm_mpgemm for callers that cannot
// allocate device memory (code under HIP graph capture, tight serving loops,
// harnesses that forbid allocation).  The only scratch memory lutgemm_mpgemm
// needs is the workspace of K-split partial sums; here it is a file-scope static
// device array, one per GPU, held until the process ends.
//
// The array's name is a host-side stand-in in host code, not a device address:
// the device address of each GPU's copy is looked up once per device with
// hipGetSymbolAddress (on the first call made with that device current) and only
// that address is ever handed to kernels.  Every call on one GPU shares its
// array, so calls that overlap on one GPU (different streams, or different host
// threads) race on it.  The partial sums are written completely before they are
// read within a call; the arrival counters of the split-K GEMV must start at
// zero: a static device array is zero when the code object is loaded, and every
// call re-arms the counters it used, so the array stays a valid workspace.
#include <hip/hip_runtime.h>

#include <cstdio>
#include <mutex>

#include "lutgemm_internal.h"

namespace {

static __device__ __align__(256) char scratch[LUTGEMM_NOALLOC_SCRATCH_BYTES];

constexpr int MAX_DEVICES = 64;
std::once_flag g_once[MAX_DEVICES];
void *g_scratch_ptr[MAX_DEVICES];
hipError_t g_scratch_err[MAX_DEVICES];

}  // namespace

extern "C" lutgemm_status_t lutgemm_mpgemm_noalloc(const lutgemm_problem_t *problem, int64_t M,
                                                   const void *tables, const void *packed, void *out,
                                                   int32_t out_dtype, int32_t accumulate, void *stream) {
    lutgemm_status_t st = lutgemm_validate(problem, M);
    if (st != LUTGEMM_SUCCESS) return st;
    const size_t need = lutgemm_workspace_size(problem, M);
    if (need > LUTGEMM_NOALLOC_SCRATCH_BYTES) {
        char msg[160];
        std::snprintf(msg, sizeof(msg), "lutgemm_mpgemm_noalloc: needs %zu bytes of scratch, the static array holds %zu",
                      need, (size_t)LUTGEMM_NOALLOC_SCRATCH_BYTES);
        lutgemm::set_last_error(msg);
        return LUTGEMM_ERROR_NOT_SUPPORTED;
    }
    void *ws = nullptr;
    if (need > 0) {
        int dev = -1;
        hipError_t e = hipGetDevice(&dev);
        if (e != hipSuccess) return lutgemm::hip_error(e);
        if (dev < 0 || dev >= MAX_DEVICES) return LUTGEMM_ERROR_NOT_SUPPORTED;
        std::call_once(g_once[dev], [dev] {
            g_scratch_err[dev] = hipGetSymbolAddress(&g_scratch_ptr[dev], HIP_SYMBOL(scratch));
        });
        if (g_scratch_err[dev] != hipSuccess) return lutgemm::hip_error(g_scratch_err[dev]);
        ws = g_scratch_ptr[dev];
    }
    return lutgemm_mpgemm(problem, M, tables, packed, out, out_dtype, accumulate, ws,
                          LUTGEMM_NOALLOC_SCRATCH_BYTES, stream);
}
