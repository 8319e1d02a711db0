// Streaming-read calibration kernels: the achievable HBM read bandwidth for a given
// byte count, measured the same way as the LUT kernels (128-bit loads, one
// launch per buffer).  Used by the benchmark to express results as a fraction of
// measured, not only published, bandwidth.  The variants differ in how many
// 16-byte loads each lane keeps in flight (U), whether the loads carry the
// nontemporal hint, and how the words are spread over the grid, so that the best
// single-launch read of a byte count can be searched for.
#include <hip/hip_runtime.h>

#include "lutgemm_internal.h"

namespace lutgemm {

typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

template <bool NT>
__device__ __forceinline__ u32x4_t ld16(const u32x4_t *p) {
    if constexpr (NT) return __builtin_nontemporal_load(p);
    return *p;
}

// Each lane issues U 16-byte loads before it uses any (indices clamped to the last
// word, values past the end ignored, so every load is unconditional) and XOR-folds
// them; one word per workgroup is written so the loads cannot be removed.
// CONTIG = false: tiles of 256 U words are dealt to the workgroups round robin;
// CONTIG = true: workgroup b reads one contiguous range of about words / grid.
template <int U, bool NT, bool CONTIG>
__global__ __launch_bounds__(256) void stream_read_kernel(const u32x4_t *__restrict__ src, int64_t words,
                                                          uint32_t *__restrict__ sink) {
    constexpr int64_t TW = 256 * U;
    int64_t t0, t1, step;
    if (CONTIG) {
        const int64_t tiles = (words + TW - 1) / TW;
        const int64_t per = (tiles + gridDim.x - 1) / gridDim.x;
        t0 = (int64_t)blockIdx.x * per;
        t1 = t0 + per < tiles ? t0 + per : tiles;
        step = 1;
    } else {
        t0 = blockIdx.x;
        t1 = (words + TW - 1) / TW;
        step = gridDim.x;
    }
    uint32_t acc = 0;
    for (int64_t t = t0; t < t1; t += step) {
        const int64_t base = t * TW + threadIdx.x;
        u32x4_t v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t i = base + 256 * u;
            v[u] = ld16<NT>(src + (i < words ? i : words - 1));
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const uint32_t x = v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
            acc ^= (base + 256 * u < words) ? x : 0u;
        }
    }
    __shared__ uint32_t red[4];
    for (int off = 32; off > 0; off >>= 1) acc ^= __shfl_xor(acc, off, 64);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) sink[blockIdx.x] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

template <int U>
static void launch_stream_u(const void *src, int64_t words, uint32_t *sink, int blocks, int flags, hipStream_t s) {
    const bool nt = flags & 1, contig = flags & 2;
    const dim3 g((unsigned)blocks), b(256);
    const u32x4_t *p = (const u32x4_t *)src;
    if (nt && contig) hipLaunchKernelGGL((stream_read_kernel<U, true, true>), g, b, 0, s, p, words, sink);
    else if (nt) hipLaunchKernelGGL((stream_read_kernel<U, true, false>), g, b, 0, s, p, words, sink);
    else if (contig) hipLaunchKernelGGL((stream_read_kernel<U, false, true>), g, b, 0, s, p, words, sink);
    else hipLaunchKernelGGL((stream_read_kernel<U, false, false>), g, b, 0, s, p, words, sink);
}

}  // namespace lutgemm

extern "C" lutgemm_status_t lutgemm_calibrate_stream_read_ex(const void *src, size_t bytes, void *sink,
                                                             int32_t blocks, int32_t unroll, int32_t flags,
                                                             void *stream) {
    if (!src || !sink || ((uintptr_t)src & 15u) || bytes < 16 || blocks <= 0 || blocks > 65536)
        return LUTGEMM_ERROR_INVALID_VALUE;
    if (flags < 0 || flags > 3) return LUTGEMM_ERROR_INVALID_VALUE;
    const int64_t words = (int64_t)(bytes / 16);
    hipStream_t s = (hipStream_t)stream;
    uint32_t *k = (uint32_t *)sink;
    switch (unroll) {
    case 1: lutgemm::launch_stream_u<1>(src, words, k, blocks, flags, s); break;
    case 2: lutgemm::launch_stream_u<2>(src, words, k, blocks, flags, s); break;
    case 4: lutgemm::launch_stream_u<4>(src, words, k, blocks, flags, s); break;
    case 8: lutgemm::launch_stream_u<8>(src, words, k, blocks, flags, s); break;
    case 16: lutgemm::launch_stream_u<16>(src, words, k, blocks, flags, s); break;
    default: return LUTGEMM_ERROR_INVALID_VALUE;
    }
    return hipGetLastError() == hipSuccess ? LUTGEMM_SUCCESS : LUTGEMM_ERROR_HIP;
}

extern "C" lutgemm_status_t lutgemm_calibrate_stream_read(const void *src, size_t bytes, void *sink,
                                                          int32_t blocks, void *stream) {
    return lutgemm_calibrate_stream_read_ex(src, bytes, sink, blocks, 4, 0, stream);
}
