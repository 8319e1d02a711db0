// Comparison path: dequantization-based mpGEMM (LUT Tensor Core, Section 2.2,
// "indirect mpGEMM with dequantization"), fused into one gfx950 matrix-core
// kernel.  Weights are rebuilt from the same packed bit-planes as FP16
// r = s' (q' - z') = s (q - z) (Eq. 1-2) in LDS, then multiplied with FP16
// activations by v_mfma_f32_32x32x16_f16 with FP32 accumulation.
//
// Small grids: workgroup tile 128 (M) x 128 (N), K step 128 (one packed plane
// word per column and plane); 4 wavefronts, each owning a 64 x 64 sub-tile as
// 2 x 2 MFMA 32x32 blocks.  Large M: the pipelined 256 x 256 kernel below.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>

#include <cstdlib>

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

// ---------------------------------------------------------------- large M
//
// Workgroup tile 256 (M) x 256 (N), K step 64; 4 wavefronts, each owning a
// 128 x 128 sub-tile as 4 x 4 MFMA 32x32 blocks (256 FP32 accumulators per lane,
// one wavefront per SIMD).  LDS holds two K steps of activations and dequantized
// weights (2 x 68 KiB): while the matrix cores work on one, the next step's
// activations stream straight into the other buffer (global_load_lds_dwordx4, no
// registers) and the next step's packed weights are dequantized into it, so each
// K step costs one barrier.  Activation rows are 128 bytes with their 16-byte
// chunks XOR-swizzled by the row (chunk c of row r at slot c ^ (r & 7)), which
// keeps both the lane-contiguous direct loads and the 128-bit MFMA operand reads
// free of bank conflicts.  Each thread dequantizes one column's 64 weights of a
// step: the Eq. 6 inversion is undone on whole 32-bit words, the 4 weights of a
// 4-bit index are spread into the 4 bytes of a register (one multiply), the planes
// are combined there, and each byte is converted (v_cvt_f32_ubyte) and scaled as
// r = s q - s z in FP32 (exact) before rounding to FP16.
constexpr int QBM = 256, QBN = 256, QBK = 64;
constexpr int QST = QBK + 8;  // halves per dequantized-weight LDS row (16-byte padding)

// Low 3 bits of every 4-bit index inverted where its bit 3 is set: undoes the
// offline negation of Eq. 6 for 8 indices at once.
__device__ __forceinline__ uint32_t undo_eq6(uint32_t w) {
    return w ^ (((w >> 3) & 0x11111111u) * 7u);
}

// The 4 bits of nibble j of w in the 4 bytes of the result (bit e -> byte e).
__device__ __forceinline__ uint32_t spread_nibble(uint32_t w, int j) {
    return (((w >> (4 * j)) & 0xFu) * 0x00204081u) & 0x01010101u;
}

// Byte b of v as a float (one v_cvt_f32_ubyte<b>).
__device__ __forceinline__ float ubyte_f(uint32_t v, int b) {
    return (float)((v >> (8 * b)) & 0xFFu);
}

typedef __attribute__((address_space(3))) void lds_void;
typedef const __attribute__((address_space(1))) void glb_void;

template <int BITS>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(1, 1)))
void dequant_mfma_big_kernel(DequantParams p, int wfmt, int per_tensor) {
    // two buffers per operand as distinct objects, so the compiler can tell the
    // direct loads into one from the reads of the other
    __shared__ __attribute__((aligned(16))) _Float16 As0[QBM * QBK], As1[QBM * QBK];
    __shared__ __attribute__((aligned(16))) _Float16 Bs0[QBN * QST], Bs1[QBN * QST];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int64_t m0 = (int64_t)blockIdx.y * QBM;
    const int64_t n0 = (int64_t)blockIdx.x * QBN;
    const int wm = (wave >> 1) * 128, wn = (wave & 1) * 128;
    const int64_t n = n0 + tid;  // column this thread dequantizes (< N_pad)
    const int nk = (int)(p.K / QBK);

    floatx16_t acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    // Activations of step ks into buffer `buf`: 8 direct loads per wavefront, each
    // writing 1 KiB of LDS (8 rows); lane L of load i fills slot L % 8 of row
    // 64 wave + 8 i + L / 8 with the chunk that belongs there under the swizzle.
    auto load_act = [&](int ks, _Float16 *dst) {
        const int64_t k0 = (int64_t)ks * QBK;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int row = 64 * wave + 8 * i + (lane >> 3), slot = lane & 7;
            const int c = slot ^ (row & 7);
            const int64_t r = (m0 + row < p.M) ? m0 + row : p.M - 1;  // rows past M: clamped, never stored
            __builtin_amdgcn_global_load_lds((glb_void *)(p.act + r * p.K + k0 + 8 * c),
                                             (lds_void *)(dst + (64 * wave + 8 * i) * QBK), 16, 0, 0);
        }
    };
    // packed weights of a step: the 64 indices of each plane (two 32-bit words) and
    // the column's metadata word(s); two register sets, loaded two steps ahead
    struct WReg {
        uint2 br[BITS];
        uint2 mr;
    };
    auto load_w = [&](int ks, WReg &w) {
        const int64_t k0 = (int64_t)ks * QBK;
        const int64_t kb = k0 / KBLK;
        const int hw = (int)((k0 % KBLK) / QBK);  // which half of the 128-k plane word
#pragma unroll
        for (int t = 0; t < BITS; ++t) w.br[t] = ((const uint2 *)(p.planes + (kb * BITS + t) * p.N_pad + n))[hw];
        // branch-free (a load under a condition makes the compiler wait for every
        // load in flight, the direct activation loads included)
        const int64_t idx = per_tensor ? 0 : (k0 / p.G) * p.N_pad + n;
        const uint32_t *mw = (const uint32_t *)p.meta;
        w.mr = make_uint2(mw[idx], mw[idx + per_tensor]);
    };
    // r = A q + B with A = 2 s', B = s' (-(2^b - 1) - z') (Eq. 2): s q - s z for UINT
    auto affine = [&](const WReg &w) {
        float s, z;
        if (per_tensor) {
            s = __uint_as_float(w.mr.x);
            z = __uint_as_float(w.mr.y);
        } else {
            s = dq_h2f(w.mr.x & 0xFFFFu);
            z = dq_h2f(w.mr.x >> 16);
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
        return make_float2(2.f * sp, sp * (-(float)((1 << BITS) - 1) - zp));
    };
    // weights it*8 .. it*8 + 7 of the column (it in [0, 8)): one 16-byte LDS store
    auto dequant8 = [&](const WReg &w, float2 ab, _Float16 *dst, int it) {
        const int d = it >> 2, jj = 2 * (it & 3);
        uint32_t raw[BITS];
#pragma unroll
        for (int t = 0; t < BITS; ++t) raw[t] = undo_eq6(d ? w.br[t].y : w.br[t].x);
        uint32_t packed[4];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            uint32_t qb = 0;  // byte e: bit e of each plane's index, i.e. weight 3 - e
#pragma unroll
            for (int t = 0; t < BITS; ++t) qb |= spread_nibble(raw[t], jj + u) << t;
            const float r3 = fmaf(ab.x, ubyte_f(qb, 0), ab.y), r2 = fmaf(ab.x, ubyte_f(qb, 1), ab.y);
            const float r1 = fmaf(ab.x, ubyte_f(qb, 2), ab.y), r0 = fmaf(ab.x, ubyte_f(qb, 3), ab.y);
            packed[2 * u] = (uint32_t)__half_as_ushort(__float2half_rn(r0)) |
                            ((uint32_t)__half_as_ushort(__float2half_rn(r1)) << 16);
            packed[2 * u + 1] = (uint32_t)__half_as_ushort(__float2half_rn(r2)) |
                                ((uint32_t)__half_as_ushort(__float2half_rn(r3)) << 16);
        }
        *(uint4 *)(dst + tid * QST + 32 * d + 4 * jj) = make_uint4(packed[0], packed[1], packed[2], packed[3]);
    };

    // one K step: MFMAs on (as, bs) while the next step's activations stream into
    // as_n; then the next step's weights (wn_, requested one step earlier) are
    // dequantized into bs_n; the weights two steps ahead are requested into wl_
    auto step = [&](int ks, const _Float16 *as, const _Float16 *bs, _Float16 *as_n, _Float16 *bs_n,
                    const WReg &wn_, WReg &wl_) {
        const bool more = ks + 1 < nk;
        if (more) load_act(ks + 1, as_n);
        if (ks + 2 < nk) load_w(ks + 2, wl_);
        const float2 ab = affine(wn_);
        // operand fragments double-buffered across the four 16-deep sub-steps
        half8_t a[2][4], b[2][4];
        auto read_frags = [&](int kk, int f) {
            const int c = 2 * kk + (lane >> 5);  // 16-byte chunk of the K step this lane supplies
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = wm + 32 * i + (lane & 31);
                a[f][i] = *(const half8_t *)(as + row * QBK + 8 * (c ^ (row & 7)));
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) b[f][j] = *(const half8_t *)(bs + (wn + 32 * j + (lane & 31)) * QST + 8 * c);
        };
        read_frags(0, 0);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int kk = 0; kk < QBK / 16; ++kk) {
            const int f = kk & 1;
            if (kk + 1 < QBK / 16) read_frags(kk + 1, f ^ 1);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[f][i], b[f][j], acc[i][j], 0, 0, 0);
            // issue order: the next sub-step's 8 LDS reads between the first 8 MFMAs
            if (kk + 1 < QBK / 16) {
#pragma unroll
                for (int t = 0; t < 8; ++t) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
                }
                __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        if (more) {
#pragma unroll
            for (int it = 0; it < 8; ++it) dequant8(wn_, ab, bs_n, it);
            __builtin_amdgcn_s_waitcnt(0);  // this wavefront's direct LDS loads have landed
        }
        __syncthreads();
    };

    WReg wA, wB;
    load_act(0, As0);
    load_w(0, wA);
    if (nk > 1) load_w(1, wB);
    {
        const float2 ab = affine(wA);
#pragma unroll
        for (int it = 0; it < 8; ++it) dequant8(wA, ab, Bs0, it);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    for (int ks = 0; ks < nk; ks += 2) {  // nk is even (K is a multiple of 128)
        step(ks, As0, Bs0, As1, Bs1, wB, wA);      // dequantizes step ks + 1 from wB, loads ks + 2 into wA
        step(ks + 1, As1, Bs1, As0, Bs0, wA, wB);  // dequantizes step ks + 2 from wA, loads ks + 3 into wB
    }

    // epilogue: lane holds column (lane % 32), rows 8*(v/4) + 4*(lane/32) + v%4 of each block
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
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
    const int pt = L.per_tensor ? 1 : 0;
    // 256 x 256 tiles when they alone fill the GPU (one workgroup per CU); the
    // LUTGEMM_TUNE_DEQUANT_BIG override forces one kernel (tests, experiments)
    const dim3 big((unsigned)(L.N_pad / QBN), (unsigned)((p.M + QBM - 1) / QBM));
    const int force = tuning(LUTGEMM_TUNE_DEQUANT_BIG);
    const bool use_big = force >= 0 ? force != 0 : (int64_t)big.x * big.y >= 256;
    if (use_big) {
        if (L.bits == 1)
            hipLaunchKernelGGL(dequant_mfma_big_kernel<1>, big, dim3(256), 0, s, p, L.wfmt, pt);
        else if (L.bits == 2)
            hipLaunchKernelGGL(dequant_mfma_big_kernel<2>, big, dim3(256), 0, s, p, L.wfmt, pt);
        else
            hipLaunchKernelGGL(dequant_mfma_big_kernel<4>, big, dim3(256), 0, s, p, L.wfmt, pt);
        return (int)hipGetLastError();
    }
    dim3 grid((unsigned)(L.N_pad / DBN), (unsigned)((p.M + DBM - 1) / DBM));
    if (L.bits == 1)
        hipLaunchKernelGGL(dequant_mfma_kernel<1>, grid, dim3(256), 0, s, p, L.wfmt, pt);
    else if (L.bits == 2)
        hipLaunchKernelGGL(dequant_mfma_kernel<2>, grid, dim3(256), 0, s, p, L.wfmt, pt);
    else
        hipLaunchKernelGGL(dequant_mfma_kernel<4>, grid, dim3(256), 0, s, p, L.wfmt, pt);
    return (int)hipGetLastError();
}

}  // namespace lutgemm
