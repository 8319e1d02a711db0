// Comparison path: dequantization-based mpGEMM (LUT Tensor Core, Section 2.2,
// "indirect mpGEMM with dequantization"), fused into one gfx950 matrix-core
// kernel.  Weights are rebuilt from the same packed bit-planes as FP16
// r = s' (q' - z') = s (q - z) (Eq. 1-2) in LDS, then multiplied with FP16
// activations by v_mfma_f32_32x32x16_f16 with FP32 accumulation.
//
// Workgroup tile 128 (M) x 128 (N), K step 128 (one packed plane word per
// column and plane); 4 wavefronts, each owning a 64 x 64 sub-tile as 2 x 2
// MFMA 32x32 blocks.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>

#include "lutgemm_internal.h"

namespace lutgemm {

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float floatx16_t __attribute__((ext_vector_type(16)));

constexpr int DBM = 128, DBN = 128, DBK = 128;
constexpr int LDS_STRIDE = DBK + 8;  // halves per LDS row (padding against bank conflicts)

__device__ __forceinline__ float dq_h2f(uint32_t bits16) {
    return __half2float(__ushort_as_half((unsigned short)bits16));
}

template <int BITS>
__global__ __launch_bounds__(256) void dequant_mfma_kernel(DequantParams p, int wfmt, int per_tensor) {
    __shared__ __attribute__((aligned(16))) _Float16 As[DBM * LDS_STRIDE];
    __shared__ __attribute__((aligned(16))) _Float16 Bs[DBN * LDS_STRIDE];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int64_t m0 = (int64_t)blockIdx.y * DBM;
    const int64_t n0 = (int64_t)blockIdx.x * DBN;
    const int wm = (wave >> 1) * 64, wn = (wave & 1) * 64;

    floatx16_t acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    // dequantization role of this thread: column c, K half h
    const int c = tid & (DBN - 1);
    const int h = tid >> 7;
    const int64_t n = n0 + c;

    for (int64_t kb = 0; kb < p.KB; ++kb) {
        // ---- A tile: 128 rows x 128 halves, 16-byte chunks
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int chunk = tid + 256 * i;
            const int row = chunk >> 4, c16 = chunk & 15;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (m0 + row < p.M) v = *(const uint4 *)(p.act + (m0 + row) * p.K + kb * DBK + c16 * 8);
            *(uint4 *)(As + row * LDS_STRIDE + c16 * 8) = v;
        }
        // ---- B tile: rebuild 64 weights of column c
        {
            uint2 pw[BITS];
#pragma unroll
            for (int t = 0; t < BITS; ++t) {
                const uint4 w = p.planes[(kb * BITS + t) * p.N_pad + n];
                pw[t] = h ? make_uint2(w.z, w.w) : make_uint2(w.x, w.y);
            }
            float s, z;
            const int64_t q = (kb * DBK) / p.G;
            if (per_tensor) {
                s = ((const float *)p.meta)[0];
                z = ((const float *)p.meta)[1];
            } else {
                const uint32_t mz = ((const uint32_t *)p.meta)[q * p.N_pad + n];
                s = dq_h2f(mz & 0xFFFFu);
                z = dq_h2f(mz >> 16);
            }
            float sp, zp;
            if (wfmt == LUTGEMM_WFMT_BINARY) {
                sp = s;
                zp = 0.f;
            } else if (wfmt == LUTGEMM_WFMT_TERNARY) {
                sp = 0.5f * s;
                zp = -1.f;
            } else {
                sp = 0.5f * s;
                zp = 2.f * z + 1.f - (float)(1 << BITS);
            }
            const float off = -(float)((1 << BITS) - 1) - zp;  // r = s' (2q - (2^b - 1) - z')
            _Float16 *dst = Bs + c * LDS_STRIDE + h * 64;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                uint32_t qv[4] = {0u, 0u, 0u, 0u};
#pragma unroll
                for (int t = 0; t < BITS; ++t) {
                    const uint32_t word = (i < 8) ? pw[t].x : pw[t].y;
                    const uint32_t nib = (word >> (4 * (i & 7))) & 0xFu;
                    const uint32_t raw = (nib & 8u) ? (nib ^ 7u) : nib;  // undo Eq. 6 inversion
#pragma unroll
                    for (int e = 0; e < 4; ++e) qv[e] |= ((raw >> (3 - e)) & 1u) << t;
                }
                uint32_t packed[2];
#pragma unroll
                for (int e = 0; e < 4; e += 2) {
                    const float r0 = sp * (2.f * (float)qv[e] + off);
                    const float r1 = sp * (2.f * (float)qv[e + 1] + off);
                    const uint32_t b0 = __half_as_ushort(__float2half_rn(r0));
                    const uint32_t b1 = __half_as_ushort(__float2half_rn(r1));
                    packed[e >> 1] = b0 | (b1 << 16);
                }
                *(uint2 *)(dst + 4 * i) = make_uint2(packed[0], packed[1]);
            }
        }
        __syncthreads();
        // ---- MFMA over the 128-wide K step
#pragma unroll
        for (int ks = 0; ks < DBK / 16; ++ks) {
            const int kofs = ks * 16 + (lane >> 5) * 8;
            half8_t a[2], b[2];
#pragma unroll
            for (int i = 0; i < 2; ++i)
                a[i] = *(const half8_t *)(As + (wm + 32 * i + (lane & 31)) * LDS_STRIDE + kofs);
#pragma unroll
            for (int j = 0; j < 2; ++j)
                b[j] = *(const half8_t *)(Bs + (wn + 32 * j + (lane & 31)) * LDS_STRIDE + kofs);
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        __syncthreads();
    }

    // ---- epilogue: lane holds column (lane % 32), rows 8*(v/4) + 4*(lane/32) + v%4
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t col = n0 + wn + 32 * j + (lane & 31);
            if (col >= p.N) continue;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t row = m0 + wm + 32 * i + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
                if (row >= p.M) continue;
                const int64_t o = row * p.N + col;
                float y = acc[i][j][v];
                if (p.out_dtype == LUTGEMM_OUT_FP32) {
                    if (p.accumulate) y += ((const float *)p.out)[o];
                    ((float *)p.out)[o] = y;
                } else {
                    if (p.accumulate) y += __half2float(((const __half *)p.out)[o]);
                    ((__half *)p.out)[o] = __float2half_rn(y);
                }
            }
        }
}

int launch_dequant(const DequantParams &p, const Layout &L, void *stream) {
    hipStream_t s = (hipStream_t)stream;
    dim3 grid((unsigned)(L.N_pad / DBN), (unsigned)((p.M + DBM - 1) / DBM));
    const int pt = L.per_tensor ? 1 : 0;
    if (L.bits == 1)
        hipLaunchKernelGGL(dequant_mfma_kernel<1>, grid, dim3(256), 0, s, p, L.wfmt, pt);
    else if (L.bits == 2)
        hipLaunchKernelGGL(dequant_mfma_kernel<2>, grid, dim3(256), 0, s, p, L.wfmt, pt);
    else
        hipLaunchKernelGGL(dequant_mfma_kernel<4>, grid, dim3(256), 0, s, p, L.wfmt, pt);
    return (int)hipGetLastError();
}

}  // namespace lutgemm
