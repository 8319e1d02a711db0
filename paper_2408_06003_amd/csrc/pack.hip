// Offline weight packing: bit-serial planes of 4-bit table indices with the
// offline bit-level negation of Eq. 6, plus the scale / zero metadata.
//
// LUT Tensor Core, Section 3.1: a b-bit weight is processed as b one-bit planes
// sharing one table; Section 3.1.2, Eq. 2: the plane bits {0,1} are read as
// {-1,+1} (the reinterpreted code q' = 2q - (2^b - 1) = sum_t 2^t (2 bit_t - 1));
// Eq. 5-6: an index whose MSB is set addresses the negated half-table row of
// its inverted low bits, so the inversion is done here, once, offline.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>

#include "lutgemm_internal.h"

namespace lutgemm {

// 4-bit stored index of one plane over 4 codes (first code = MSB), Eq. 6.
__device__ __forceinline__ uint32_t plane_index(uint32_t q0, uint32_t q1, uint32_t q2, uint32_t q3,
                                                int t) {
    uint32_t pat = (((q0 >> t) & 1u) << 3) | (((q1 >> t) & 1u) << 2) | (((q2 >> t) & 1u) << 1) |
                   ((q3 >> t) & 1u);
    uint32_t sign = pat >> 3;
    uint32_t low = sign ? (~pat & 7u) : (pat & 7u);
    return (sign << 3) | low;
}

// Code q of byte e of a 32-bit load of 4 consecutive codes.
__device__ __forceinline__ uint32_t code_of(const PackParams &p, uint32_t word, int e) {
    uint32_t c = (word >> (8 * e)) & 0xFFu;
    if (p.wfmt == LUTGEMM_WFMT_TERNARY) {
        int v = (int)(int8_t)c;
        v = v < -1 ? -1 : (v > 1 ? 1 : v);
        return (uint32_t)(v + 1);
    }
    return c & ((1u << p.bits) - 1u);
}

// One thread per (column n, 128-block kb), kb fastest so that a wavefront reads
// consecutive 128-byte code segments of one row.
__global__ __launch_bounds__(256) void pack_planes_kernel(PackParams p) {
    const int64_t total = p.N_pad * p.KB;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int64_t kb = idx % p.KB;
        const int64_t n = idx / p.KB;
        uint32_t w[4][4];
#pragma unroll
        for (int t = 0; t < 4; ++t)
#pragma unroll
            for (int d = 0; d < 4; ++d) w[t][d] = 0u;
        if (n < p.N) {
            const int64_t base = n * p.K + kb * KBLK;
            const uint32_t *row = (const uint32_t *)((const uint8_t *)p.codes + base);
#pragma unroll
            for (int g = 0; g < GPB; ++g) {
                const uint32_t word = row[g];
                const uint32_t q0 = code_of(p, word, 0), q1 = code_of(p, word, 1);
                const uint32_t q2 = code_of(p, word, 2), q3 = code_of(p, word, 3);
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    if (t < p.bits) w[t][g >> 3] |= plane_index(q0, q1, q2, q3, t) << (4 * (g & 7));
                }
            }
        }
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            if (t < p.bits)
                p.planes[(kb * p.bits + t) * p.N_pad + n] = make_uint4(w[t][0], w[t][1], w[t][2], w[t][3]);
        }
    }
}

// Ternary 3-in-5 (Section 5, three ternary weights in 5 bits): one thread per
// (column n, 96-block kb), kb fastest.  Triple t of the block holds weights
// 96 kb + 3t .. + 2 (0 past K); its base-3 value v = 9(w0+1) + 3(w1+1) + (w2+1)
// becomes sign = (v < 13) and index |v - 13|: the index addresses the stored
// half of the 27-pattern table and the sign selects its negation (Eq. 4), the
// ternary counterpart of the offline negation of Eq. 6.
__global__ __launch_bounds__(256) void pack_tri_kernel(PackParams p) {
    const int64_t total = p.N_pad * p.KB;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int64_t kb = idx % p.KB;
        const int64_t n = idx / p.KB;
        uint32_t word[4] = {0u, 0u, 0u, 0u}, sgn = 0u;
        if (n < p.N) {
            const int64_t k0 = kb * TBLK;
            const int nwords = (int)((p.K - k0) < TBLK ? (p.K - k0) : TBLK) / 4;  // K % 32 == 0
            const uint32_t *row = (const uint32_t *)((const int8_t *)p.codes + n * p.K + k0);
            uint32_t c[TBLK / 4];
#pragma unroll
            for (int i = 0; i < TBLK / 4; ++i) c[i] = i < nwords ? row[i] : 0u;
#pragma unroll
            for (int t = 0; t < TPB; ++t) {
                int v = 0;
#pragma unroll
                for (int e = 0; e < 3; ++e) {
                    const int k = 3 * t + e;
                    int w = (int)(int8_t)((c[k >> 2] >> (8 * (k & 3))) & 0xFFu);
                    w = w < -1 ? -1 : (w > 1 ? 1 : w);
                    v = 3 * v + (w + 1);
                }
                const uint32_t s = v < 13 ? 1u : 0u;
                const uint32_t i4 = (uint32_t)(v < 13 ? 13 - v : v - 13);
                const int d = t >> 3, k = (t & 7) >> 1, h = t & 1;
                word[d] |= i4 << (4 * (t & 7));
                sgn |= s << (8 * k + 2 * d + h);
            }
        }
        p.planes[kb * p.N_pad + n] = make_uint4(word[0], word[1], word[2], word[3]);
        p.sgn[kb * p.N_pad + n] = sgn;
    }
}

// Per-group metadata: (s, z) FP16 pairs [Q][N_pad]; per-tensor: FP32 (s, z).
__global__ __launch_bounds__(256) void pack_meta_kernel(PackParams p) {
    if (p.per_tensor) {
        if (blockIdx.x == 0 && threadIdx.x == 0) {
            float s, z = 0.f;
            if (p.scale_fp32) {
                s = ((const float *)p.scales)[0];
            } else {
                s = __half2float(((const __half *)p.scales)[0]);
                if (p.wfmt == LUTGEMM_WFMT_UINT) z = __half2float(((const __half *)p.zeros)[0]);
            }
            float *m = (float *)p.meta;
            m[0] = s;
            m[1] = z;
        }
        return;
    }
    const int64_t total = p.Q * p.N_pad;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (int64_t)gridDim.x * blockDim.x) {
        const int64_t q = idx / p.N_pad;
        const int64_t n = idx % p.N_pad;
        uint32_t sbits = 0, zbits = 0;
        if (n < p.N) {
            sbits = ((const uint16_t *)p.scales)[n * p.Q + q];
            if (p.wfmt == LUTGEMM_WFMT_UINT) zbits = ((const uint16_t *)p.zeros)[n * p.Q + q];
        }
        ((uint32_t *)p.meta)[idx] = sbits | (zbits << 16);
    }
}

// Fixed-point exponent E of column n for the exact K-split completion of FP partial
// sums (split_complete_exact).  With the token scaled to |x| < 1 by the precompute, a
// table entry (a signed sum of 4 activations) is below 4 in magnitude, stored as at
// most 4 2^FIX_SHIFT, so one 128-block of bit-plane t adds at most |s'| 2^t 128 to a
// partial sum and the zero-point term of a group is at most |s' z'| G (|S| <= G).
// Their sum over the column's groups, B (with 1/16 added for the FP32 rounding of the
// partial sums), bounds every split's partial sum and their total; E is the smallest
// integer with B < 2^(BND_BITS + E).  (The fused split kernel, whose tables hold the
// unscaled FP16 activations, |x| <= 65504 < 2^16, uses E + 16.)  E = 0 for padding
// columns and all-zero scales; B is not finite only for non-finite scales, whose
// outputs are unspecified on this path.
__global__ __launch_bounds__(256) void pack_bound_kernel(PackParams p, float cs, float cz, float c0) {
    const int64_t n = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (n >= p.N_pad) return;
    int E = 0;
    if (n < p.N) {
        const double kpg = (double)(p.G / KBLK), planes = (double)((1 << p.bits) - 1), G = (double)p.G;
        double B = 0.0;
        for (int64_t q = 0; q < p.Q; ++q) {
            float s, z;
            if (p.per_tensor) {
                s = ((const float *)p.meta)[0];
                z = ((const float *)p.meta)[1];
            } else {
                const uint32_t w = ((const uint32_t *)p.meta)[q * p.N_pad + n];
                s = __half2float(__ushort_as_half((unsigned short)(w & 0xFFFFu)));
                z = __half2float(__ushort_as_half((unsigned short)(w >> 16)));
            }
            const double sp = (double)cs * (double)s, zp = (double)cz * (double)z + (double)c0;
            B += kpg * fabs(sp) * 128.0 * planes + fabs(sp * zp) * G;
        }
        B *= 1.0625;
        if (B > 0.0 && B <= 1e300) E = ilogb(B) + 1 - BND_BITS;
    }
    p.bnd[n] = E;
}

int launch_pack(const PackParams &p, void *stream) {
    hipStream_t s = (hipStream_t)stream;
    int64_t total = p.N_pad * p.KB;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 65535 * 16) blocks = 65535 * 16;
    if (p.wfmt == LUTGEMM_WFMT_TERNARY_3IN5)
        hipLaunchKernelGGL(pack_tri_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p);
    else
        hipLaunchKernelGGL(pack_planes_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return (int)e;
    int64_t mt = p.per_tensor ? 1 : p.Q * p.N_pad;
    int64_t mblocks = (mt + 255) / 256;
    if (mblocks > 65535 * 16) mblocks = 65535 * 16;
    hipLaunchKernelGGL(pack_meta_kernel, dim3((unsigned)mblocks), dim3(256), 0, s, p);
    e = hipGetLastError();
    if (e != hipSuccess) return (int)e;
    if (p.wfmt == LUTGEMM_WFMT_TERNARY_3IN5) return (int)hipSuccess;
    float cs, cz, c0;
    format_consts(p.wfmt, p.bits, cs, cz, c0);
    hipLaunchKernelGGL(pack_bound_kernel, dim3((unsigned)((p.N_pad + 255) / 256)), dim3(256), 0, s, p, cs, cz, c0);
    return (int)hipGetLastError();
}

}  // namespace lutgemm
