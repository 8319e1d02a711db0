// Streaming-read calibration kernel: the achievable HBM read bandwidth for a given
// byte count, measured the same way as the LUT kernels (128-bit loads, one
// launch per buffer).  Used by the benchmark to express results as a fraction of
// measured, not only published, bandwidth.
#include <hip/hip_runtime.h>

#include "lutgemm_internal.h"

namespace lutgemm {

// Each lane XOR-folds `per_lane` 16-byte words strided by the grid; one word per
// workgroup is written so the loads cannot be removed.
__global__ __launch_bounds__(256) void stream_read_kernel(const uint4 *__restrict__ src, int64_t words,
                                                          uint32_t *__restrict__ sink) {
    const int64_t stride = (int64_t)gridDim.x * 256;
    uint32_t acc = 0;
    int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    for (; i + 3 * stride < words; i += 4 * stride) {
        const uint4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
        acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w;
    }
    for (; i < words; i += stride) {
        const uint4 a = src[i];
        acc ^= a.x ^ a.y ^ a.z ^ a.w;
    }
    __shared__ uint32_t red[4];
    for (int off = 32; off > 0; off >>= 1) acc ^= __shfl_xor(acc, off, 64);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) sink[blockIdx.x] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

}  // namespace lutgemm

extern "C" lutgemm_status_t lutgemm_calibrate_stream_read(const void *src, size_t bytes, void *sink,
                                                          int32_t blocks, void *stream) {
    if (!src || !sink || ((uintptr_t)src & 15u) || bytes < 16 || blocks <= 0 || blocks > 65536)
        return LUTGEMM_ERROR_INVALID_VALUE;
    hipLaunchKernelGGL(lutgemm::stream_read_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream,
                       (const uint4 *)src, (int64_t)(bytes / 16), (uint32_t *)sink);
    return hipGetLastError() == hipSuccess ? LUTGEMM_SUCCESS : LUTGEMM_ERROR_HIP;
}
