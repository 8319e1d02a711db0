// Table precompute as an independent operator (LUT Tensor Core, Section 3.1.1),
// building the symmetric half tables of Eq. 4-5.
//
// One workgroup per token m:
//   1. amax = max_k |a[m,k]|.  FP16 tables: the token is scaled by 2^-e with
//      amax = f 2^e, f in [0.5, 1), so every entry lies in (-4, 4) and neither
//      overflows nor loses range in FP16 (the factor 2^e is returned in t[m]).
//      INT8 tables: q_a = clamp(rint(a * (127 / amax)), -127, 127), FP32 with
//      correctly rounded division, s_a = amax / 127.
//   2. For every group j of 4 activations x_0..x_3 and row i in [0, 8):
//      T[m][j][i] = -x_0 + sum_{e=1..3} (bit (3-e) of i ? x_e : -x_e), which is
//      the entry of pattern 0 i of the full 16-entry table (Eq. 5); the other
//      half is its negation (Eq. 4) and is never stored.
//   3. S[m][q] = sum of x over quantization group q (zero-point term of Eq. 3).
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>

#include "lutgemm_internal.h"

namespace lutgemm {

__device__ __forceinline__ float h2f(uint32_t bits16) {
    return __half2float(__ushort_as_half((unsigned short)bits16));
}

__device__ __forceinline__ float block_max(float v, float *red) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    if (lane == 0) red[wave] = v;
    __syncthreads();
    float r = red[0];
    for (int w = 1; w < (int)(blockDim.x >> 6); ++w) r = fmaxf(r, red[w]);
    __syncthreads();
    return r;
}

template <bool INT8>
__device__ __forceinline__ float token_value(float a, float scale) {
    if (INT8) {
        float r = rintf(a * scale);
        r = fminf(fmaxf(r, -127.f), 127.f);
        return r;
    }
    return a * scale;  // exact: scale is a power of two
}

template <bool INT8>
__global__ __launch_bounds__(256) void precompute_kernel(PrecomputeParams p) {
    __shared__ float red[4];
    const int64_t m = blockIdx.x;
    const uint16_t *a = p.act + m * p.K;
    const int tid = threadIdx.x;

    // 1. absmax of the token
    float amax = 0.f;
    for (int64_t k = (int64_t)tid * 4; k < p.K; k += 1024) {
        const uint2 v = *(const uint2 *)(a + k);
        amax = fmaxf(amax, fabsf(h2f(v.x & 0xFFFFu)));
        amax = fmaxf(amax, fabsf(h2f(v.x >> 16)));
        amax = fmaxf(amax, fabsf(h2f(v.y & 0xFFFFu)));
        amax = fmaxf(amax, fabsf(h2f(v.y >> 16)));
    }
    amax = block_max(amax, red);

    float scale, tok;
    if (INT8) {
        if (amax == 0.f) {
            scale = 0.f;
            tok = 0.f;
        } else {
            scale = __fdiv_rn(127.0f, amax);
            tok = __fdiv_rn(amax, 127.0f);
        }
    } else {
        if (amax == 0.f) {
            scale = 1.f;
            tok = 1.f;
        } else {
            int e;
            (void)frexpf(amax, &e);
            scale = ldexpf(1.f, -e);
            tok = ldexpf(1.f, e);
        }
    }
    if (tid == 0) p.tok[m] = tok;

    // 2. half tables, one group of 4 activations per thread and step
    for (int64_t j = tid; j < p.J; j += 256) {
        const uint2 v = *(const uint2 *)(a + 4 * j);
        const float x0 = token_value<INT8>(h2f(v.x & 0xFFFFu), scale);
        const float x1 = token_value<INT8>(h2f(v.x >> 16), scale);
        const float x2 = token_value<INT8>(h2f(v.y & 0xFFFFu), scale);
        const float x3 = token_value<INT8>(h2f(v.y >> 16), scale);
        uint32_t e[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const float t = ((-x0 + ((i & 4) ? x1 : -x1)) + ((i & 2) ? x2 : -x2)) + ((i & 1) ? x3 : -x3);
            if (INT8)
                e[i] = (uint32_t)(uint16_t)(int16_t)(int)t;  // |t| <= 508, exact
            else
                e[i] = (uint32_t)__half_as_ushort(__float2half_rn(t));
        }
        p.T[m * p.J + j] = make_uint4(e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16),
                                      e[6] | (e[7] << 16));
    }

    // 3. group sums, one wavefront per quantization group, fixed summation order
    const int wave = tid >> 6, lane = tid & 63;
    for (int64_t q = wave; q < p.Q; q += 4) {
        const uint16_t *aq = a + q * p.G;
        if (INT8) {
            int s = 0;
            for (int64_t k = lane; k < p.G; k += 64) s += (int)token_value<true>(h2f(aq[k]), scale);
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
            if (lane == 0) ((int *)p.S)[m * p.Q + q] = s;
        } else {
            float s = 0.f;
            for (int64_t k = lane; k < p.G; k += 64) s += token_value<false>(h2f(aq[k]), scale);
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
            if (lane == 0) ((float *)p.S)[m * p.Q + q] = s;
        }
    }
}

int launch_precompute(const PrecomputeParams &p, int act_int8, void *stream) {
    hipStream_t s = (hipStream_t)stream;
    if (p.M <= 0) return 0;
    if (act_int8)
        hipLaunchKernelGGL(precompute_kernel<true>, dim3((unsigned)p.M), dim3(256), 0, s, p);
    else
        hipLaunchKernelGGL(precompute_kernel<false>, dim3((unsigned)p.M), dim3(256), 0, s, p);
    return (int)hipGetLastError();
}

}  // namespace lutgemm
