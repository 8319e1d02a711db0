// Table precompute as an independent operator (LUT Tensor Core, Section 3.1.1),
// building the symmetric half tables of Eq. 4-5.
//
// Grid (ceil(J / (256 R)), M): workgroup b of token m owns table groups
// [256 R b, 256 R (b + 1)), one group of 4 activations per lane and step of R
// (R = 1, 2, 4 or 8: the largest that keeps the grid at >= 256 workgroups).
//   1. amax = max_k |a[m,k]| over the whole token (every workgroup reads the
//      token once, into LDS when K <= 32768, so steps 2-3 read no global memory;
//      the token is at most a few tens of KiB and stays in L2).  FP16 tables: the
//      token is scaled by 2^-e with amax = f 2^e, f in [0.5, 1), so every entry
//      lies in (-4, 4) and FP16 neither overflows nor loses range (the factor 2^e
//      is returned in t[m]).  INT8 tables: q_a = clamp(rint(a * (127 / amax)),
//      -127, 127), FP32 with correctly rounded division, s_a = amax / 127.
//   2. For its group j with activations x_0..x_3 and row i in [0, 8):
//      T[m][j][i] = -x_0 + sum_{e=1..3} (bit (3-e) of i ? x_e : -x_e), the entry of
//      pattern 0 i of the full 16-entry table (Eq. 5); the other half is its
//      negation (Eq. 4) and is never stored.
//      INT8 table quantization (Section 3.1.3, `tsc` set): each half table is
//      stored as 8 INT8 codes round(127 T / amax), ties to even, with amax = max |T|
//      of the exact entries (formed in FP64, where they are exact), and its scale
//      amax / 127 rounded to FP32.
//   3. S[m][q] = sum of x over quantization group q (zero-point term of Eq. 3):
//      groups of 128..1024 activations are reduced across the lanes that built
//      them; larger ones are summed by the workgroup that holds their first
//      activation.  All reductions have a fixed order.
// Ternary 3-in-5 weights (TRI): step 2 builds, per triple j of activations
// x_{3j..3j+2} (0 past K), the 14 entries T[i] = sum_e w_e(13 + i) x_{3j+e} of
// the stored half of the 27-pattern table (tri_table.h); there is no zero point,
// so step 3 is skipped.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>

#include "lutgemm_internal.h"
#include "tri_table.h"

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

__device__ __forceinline__ float block_sum_f(float v, float *red) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    __syncthreads();
    if (lane == 0) red[wave] = v;
    __syncthreads();
    return ((red[0] + red[1]) + red[2]) + red[3];
}

__device__ __forceinline__ int block_sum_i(int v, int *red) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    __syncthreads();
    if (lane == 0) red[wave] = v;
    __syncthreads();
    return red[0] + red[1] + red[2] + red[3];
}

constexpr int64_t ROW_LDS_MAX_K = 32768;  // tokens up to this length are staged in LDS once

template <bool INT8, bool TRI>
__device__ __forceinline__ void build_block(const PrecomputeParams &p, const uint16_t *a, int64_t vb, int64_t m,
                                            float scale, float *redf, int *redi, float *segf, int *segi);

template <bool INT8, bool ROW_LDS, bool TRI>
__global__ __launch_bounds__(256) void precompute_kernel(PrecomputeParams p) {
    extern __shared__ __attribute__((aligned(16))) uint16_t row[];  // K halves when ROW_LDS
    __shared__ float redf[4];
    __shared__ int redi[4];
    __shared__ float segf[4];
    __shared__ int segi[4];
    const int64_t m = blockIdx.y;
    const uint16_t *ag = p.act + m * p.K;
    const uint16_t *a = ROW_LDS ? row : ag;  // reads after step 1 come from the staged row
    const int tid = threadIdx.x;

    // 1. absmax of the token, 8 activations per load (unrolled: long tokens keep
    // several loads in flight per lane)
    float amax = 0.f;
#pragma unroll 8
    for (int64_t c = tid; c < p.K / 8; c += 256) {
        const uint4 v = ((const uint4 *)ag)[c];
        if (ROW_LDS) ((uint4 *)row)[c] = v;
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            amax = fmaxf(amax, fabsf(h2f(w[i] & 0xFFFFu)));
            amax = fmaxf(amax, fabsf(h2f(w[i] >> 16)));
        }
    }
    amax = block_max(amax, redf);  // its barrier also publishes the staged row

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
    if (blockIdx.x == 0 && tid == 0) p.tok[m] = tok;

    // steps 2-3 for the R virtual blocks of 256 table groups this workgroup owns
    if (p.vbs == 1) {
        build_block<INT8, TRI>(p, a, blockIdx.x, m, scale, redf, redi, segf, segi);
        return;
    }
    for (int r = 0; r < p.vbs; ++r) {
        const int64_t vb = (int64_t)blockIdx.x * p.vbs + r;
        if (vb * 256 >= p.J) break;  // uniform
        build_block<INT8, TRI>(p, a, vb, m, scale, redf, redi, segf, segi);
    }
}

// Steps 2-3 for virtual block vb (table groups [256 vb, 256 vb + 256)).
template <bool INT8, bool TRI>
__device__ __forceinline__ void build_block(const PrecomputeParams &p, const uint16_t *a, int64_t vb, int64_t m,
                                            float scale, float *redf, int *redi, float *segf, int *segi) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t j = vb * 256 + tid;
    if constexpr (TRI) {
        // 2'. triple table of this lane's triple
        if (j < p.J) {
            float x[3];
#pragma unroll
            for (int e = 0; e < 3; ++e) {
                const int64_t k = 3 * j + e;
                x[e] = k < p.K ? token_value<INT8>(h2f(a[k]), scale) : 0.f;
            }
            uint32_t h[16];
            if (INT8) {
                int e[14];  // |e| <= 381, exact
                tri_table14<int>((int)x[0], (int)x[1], (int)x[2], e);
#pragma unroll
                for (int i = 0; i < 14; ++i) h[i] = (uint32_t)e[i] & 0xFFFFu;
            } else {
                float e[14];
                tri_table14<float>(x[0], x[1], x[2], e);
#pragma unroll
                for (int i = 0; i < 14; ++i) h[i] = (uint32_t)__half_as_ushort(__float2half_rn(e[i]));
            }
            h[14] = h[15] = 0u;
            uint32_t w[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) w[i] = h[2 * i] | (h[2 * i + 1] << 16);
            uint4 *dst = p.T + 2 * (m * p.J + j);
            dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
            dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
        }
        return;
    }

    // 2. half table of this lane's group
    float g4f = 0.f;
    int g4i = 0;
    if (j < p.J) {
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
        if (!INT8 && p.tsc) {
            // INT8 table quantization (Section 3.1.3), one scale per table.  The table
            // is formed in FP64, where it is exact (the x are FP16 values times a power
            // of two: integer multiples of 2^(-24-e) below 1, so every sum is exact);
            // 127 T is exact too, and the rounding of the FP64 quotient cannot reach or
            // cross a half-integer the exact 127 T / amax does not lie on, so rint gives
            // round-half-to-even of the exact value.  Scale: amax / 127 to FP32.
            const double d0 = x0, d1 = x1, d2 = x2, d3 = x3;
            double td[8], tmax = 0.0;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                td[i] = ((-d0 + ((i & 4) ? d1 : -d1)) + ((i & 2) ? d2 : -d2)) + ((i & 1) ? d3 : -d3);
                tmax = fmax(tmax, fabs(td[i]));
            }
            uint32_t c[2] = {0u, 0u};
            if (tmax != 0.0) {
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const int r = (int)rint((127.0 * td[i]) / tmax);  // |r| <= 127
                    c[i >> 2] |= ((uint32_t)r & 0xFFu) << (8 * (i & 3));
                }
            }
            ((uint2 *)p.T)[m * p.J + j] = make_uint2(c[0], c[1]);
            p.tsc[m * p.J + j] = tmax == 0.0 ? 0.f : __double2float_rn(tmax / 127.0);
        } else {
            p.T[m * p.J + j] = make_uint4(e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16),
                                          e[6] | (e[7] << 16));
        }
        g4f = ((x0 + x1) + x2) + x3;
        g4i = (int)x0 + (int)x1 + (int)x2 + (int)x3;
    }

    // 3. group sums
    const int64_t seg = p.G / 4;  // table groups per quantization group
    if (seg <= 256 && 256 % seg == 0) {
        // reduce over `seg` consecutive lanes (butterfly within the wave, then waves in order)
        const int width = seg < 64 ? (int)seg : 64;
        float sf = g4f;
        int si = g4i;
        for (int off = width >> 1; off > 0; off >>= 1) {
            if (INT8)
                si += __shfl_xor(si, off, 64);
            else
                sf += __shfl_xor(sf, off, 64);
        }
        if (seg > 64) {
            __syncthreads();
            if (lane == 0) {
                segf[wave] = sf;
                segi[wave] = si;
            }
            __syncthreads();
            const int wpq = (int)(seg / 64), w0 = wave - wave % wpq;
            sf = segf[w0];
            si = segi[w0];
            for (int w = 1; w < wpq; ++w) {
                sf += segf[w0 + w];
                si += segi[w0 + w];
            }
        }
        if (j < p.J && (j % seg) == 0) {
            const int64_t q = j / seg;
            if (INT8)
                ((int *)p.S)[m * p.Q + q] = si;
            else
                ((float *)p.S)[m * p.Q + q] = sf;
        }
    } else {
        // quantization groups starting in this block's range, summed by the whole workgroup
        const int64_t k_lo = vb * 1024;
        const int64_t k_hi = (k_lo + 1024 < p.K) ? k_lo + 1024 : p.K;
        for (int64_t q = (k_lo + p.G - 1) / p.G; q * p.G < k_hi; ++q) {
            const uint16_t *aq = a + q * p.G;
            float sf = 0.f;
            int si = 0;
            for (int64_t c = tid; c < p.G / 8; c += 256) {
                const uint4 v = ((const uint4 *)aq)[c];
                const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float lo = token_value<INT8>(h2f(w[i] & 0xFFFFu), scale);
                    const float hi = token_value<INT8>(h2f(w[i] >> 16), scale);
                    if (INT8)
                        si += (int)lo + (int)hi;
                    else
                        sf += lo + hi;
                }
            }
            if (INT8) {
                const int tot = block_sum_i(si, redi);
                if (tid == 0) ((int *)p.S)[m * p.Q + q] = tot;
            } else {
                const float tot = block_sum_f(sf, redf);
                if (tid == 0) ((float *)p.S)[m * p.Q + q] = tot;
            }
            __syncthreads();
        }
    }
}

int launch_precompute(const PrecomputeParams &p_in, int act_int8, void *stream) {
    hipStream_t s = (hipStream_t)stream;
    if (p_in.M <= 0) return 0;
    // virtual blocks of 256 table groups per workgroup: more when the grid stays at
    // >= 512 workgroups, so fewer workgroups each read the whole token for its absmax
    // (M = 256: K = 8192 7.9 -> 6.7 us, K = 28672 19.9 -> 17.8 us against >= 256;
    // >= 1024 measured slower at K = 28672, 24.4 us)
    PrecomputeParams p = p_in;
    const int64_t nvb = (p.J + 255) / 256;
    p.vbs = 1;
    for (int r = 32; r > 1; r /= 2)
        if ((nvb + r - 1) / r * p.M >= 512) {
            p.vbs = r;
            break;
        }
    const dim3 grid((unsigned)((nvb + p.vbs - 1) / p.vbs), (unsigned)p.M);
    const bool lds = p.K <= ROW_LDS_MAX_K;
    const size_t shm = lds ? (size_t)p.K * 2 : 0;
    if (p.tri) {
        if (act_int8) {
            if (lds) hipLaunchKernelGGL((precompute_kernel<true, true, true>), grid, dim3(256), shm, s, p);
            else hipLaunchKernelGGL((precompute_kernel<true, false, true>), grid, dim3(256), 0, s, p);
        } else {
            if (lds) hipLaunchKernelGGL((precompute_kernel<false, true, true>), grid, dim3(256), shm, s, p);
            else hipLaunchKernelGGL((precompute_kernel<false, false, true>), grid, dim3(256), 0, s, p);
        }
    } else if (act_int8) {
        if (lds) hipLaunchKernelGGL((precompute_kernel<true, true, false>), grid, dim3(256), shm, s, p);
        else hipLaunchKernelGGL((precompute_kernel<true, false, false>), grid, dim3(256), 0, s, p);
    } else {
        if (lds) hipLaunchKernelGGL((precompute_kernel<false, true, false>), grid, dim3(256), shm, s, p);
        else hipLaunchKernelGGL((precompute_kernel<false, false, false>), grid, dim3(256), 0, s, p);
    }
    return (int)hipGetLastError();
}

}  // namespace lutgemm
