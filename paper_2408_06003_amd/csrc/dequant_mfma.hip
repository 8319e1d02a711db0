// Comparison path: dequantization-based mpGEMM (LUT Tensor Core, Section 2.2,
// "indirect mpGEMM with dequantization"), fused into gfx950 matrix-core kernels.
// Weights are rebuilt from the same packed bit-planes as FP16
// r = s' (q' - z') = s (q - z) (Eq. 1-2), in LDS or in registers, then multiplied
// with the FP16 activations on the matrix cores with FP32 accumulation.
//
// Three kernels, chosen by plan_dequant at the end of this file: 1-bit weights at
// a few tokens, 16-token slabs on v_mfma_f32_16x16x32_f16 with the weights decoded
// in registers; large M, the pipelined 256 x 256 kernel; other shapes, 128 x 128
// tiles with K step 128 (one packed plane word per column and plane), 4
// wavefronts each owning a 64 x 64 sub-tile as 2 x 2 MFMA 32x32 blocks.  Any of them
// can split K; the FP32 partial sums are then added in split order by
// dequant_reduce_kernel.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>

#include <cstdlib>

#include "lutgemm_internal.h"

namespace lutgemm {

typedef _Float16 half8_t __attribute__((ext_vector_type(8)));

// Keeps an index in a VGPR, so that the load it addresses stays a vector load.
__device__ __forceinline__ int64_t lane_value_dq(int64_t x) {
    asm volatile("" : "+v"(x));
    return x;
}
typedef float floatx16_t __attribute__((ext_vector_type(16)));

constexpr int DBM = 128, DBN = 128, DBK = 128;
constexpr int LDS_STRIDE = DBK + 8;  // halves per LDS row (padding against bank conflicts)

__device__ __forceinline__ float dq_h2f(uint32_t bits16) {
    return __half2float(__ushort_as_half((unsigned short)bits16));
}

// Result y of output (row, col): with a K split the FP32 partial of this workgroup's
// split (blockIdx.z), summed later by dequant_reduce_kernel; else the output itself
// (optional accumulate, dtype conversion).  Rows and columns past the problem are
// skipped.
__device__ __forceinline__ void dq_store(const DequantParams &p, int64_t row, int64_t col, float y) {
    if (row >= p.M || col >= p.N) return;
    if (p.part) {
        p.part[((int64_t)blockIdx.z * p.M + row) * p.N_pad + col] = y;
        return;
    }
    const int64_t o = row * p.N + col;
    if (p.out_dtype == LUTGEMM_OUT_FP32) {
        if (p.accumulate) y += ((const float *)p.out)[o];
        ((float *)p.out)[o] = y;
    } else {
        if (p.accumulate) y += __half2float(((const __half *)p.out)[o]);
        ((__half *)p.out)[o] = __float2half_rn(y);
    }
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

    const int64_t kbA = (int64_t)blockIdx.z * p.kbs;
    const int64_t kbB = kbA + p.kbs < p.KB ? kbA + p.kbs : p.KB;
    for (int64_t kb = kbA; kb < kbB; ++kb) {
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
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t row = m0 + wm + 32 * i + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
                dq_store(p, row, col, acc[i][j][v]);
            }
        }
}

// ---------------------------------------------------------------- large M
//
// Workgroup tile 256 (M) x 256 (N), K step 64, 8 wavefronts: two per SIMD, so that
// one can dequantize or wait while the other drives the matrix cores.  Wavefront w
// owns the 128 x 64 sub-tile at rows 128 (w / 4), columns 64 (w % 4) as 4 x 2 MFMA
// 32x32 blocks (128 FP32 accumulators per lane).  LDS holds two K steps of
// activations (2 x 32 KiB) and of dequantized weights (2 x 36 KiB): while the matrix
// cores work on one, the next step's activations stream straight into the other
// buffer (global_load_lds_dwordx4, no registers) and the next step's packed weights
// are dequantized into it, so each K step costs one barrier.  Activation rows are
// 128 bytes with their 16-byte chunks XOR-swizzled (chunk c of row r at slot
// c ^ ((r / 2) % 8)): the lane-contiguous direct loads and the 128-bit operand reads
// of 16 consecutive rows then touch distinct banks.  Dequantized-weight rows (one
// per column) are padded to 144 bytes, which spreads 16 consecutive columns over all
// banks.  Each thread dequantizes 32 weights of one column per step: the Eq. 6
// inversion is undone on whole 32-bit words, the 4 weights of a 4-bit index are
// spread into the 4 bytes of a register (one multiply), the planes are combined
// there, and each byte is converted (v_cvt_f32_ubyte) and scaled as r = s q - s z in
// FP32 (exact) before rounding to FP16, a quarter of it between the MFMAs of each
// 16-deep sub-step.  The packed words are loaded two K steps ahead.  Tiles are
// assigned so that each XCD works on a contiguous band of them (shared activation
// rows stay in that XCD's L2).
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

// r = A q + B for a b-bit index q, with A = 2 s', B = s' (-(2^b - 1) - z') (Eq. 2):
// s q - s z for UINT, s (2 q - 1) for BINARY, s (q - 1) for TERNARY codes.
template <int BITS>
__device__ __forceinline__ float2 dq_affine(int wfmt, float s, float z) {
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
}

typedef __attribute__((address_space(3))) void lds_void;
typedef const __attribute__((address_space(1))) void glb_void;

template <int BITS, bool PT>
__global__ __launch_bounds__(512) void dequant_mfma_big_kernel(DequantParams p, int wfmt) {
    // two buffers per operand as distinct objects, so the compiler can tell the
    // direct loads into one from the reads of the other
    __shared__ __attribute__((aligned(16))) _Float16 As0[QBM * QBK], As1[QBM * QBK];
    __shared__ __attribute__((aligned(16))) _Float16 Bs0[QBN * QST], Bs1[QBN * QST];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    // Tile of this workgroup.  Workgroups are dealt to the 8 XCDs round robin; when the
    // tile count allows, XCD x gets tiles x T/8 .. (x + 1) T/8 - 1 in row-major order,
    // so the workgroups sharing an XCD's L2 also share activation rows.
    const uint32_t nx = gridDim.x, tiles = gridDim.x * gridDim.y;
    uint32_t t = blockIdx.x + nx * blockIdx.y;
    if (tiles % 8 == 0) t = (t % 8) * (tiles / 8) + t / 8;
    const int64_t m0 = (int64_t)(t / nx) * QBM;
    const int64_t n0 = (int64_t)(t % nx) * QBN;
    const int wm = (wave >> 2) * 128, wn = (wave & 3) * 64;
    const int col = tid & (QBN - 1), hf = tid >> 8;  // dequantized column, which 32 k of a step
    const int64_t n = n0 + col;
    // K steps of this workgroup's split: two per 128-block
    const int64_t kb0 = (int64_t)blockIdx.z * p.kbs;
    const int nkb = (int)(p.KB - kb0 < p.kbs ? p.KB - kb0 : p.kbs);
    const int nk = 2 * nkb;
    const int64_t k00 = kb0 * KBLK;

    floatx16_t acc[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    float2 ab_pt = make_float2(0.f, 0.f);  // per-tensor scale and zero: FP32 s, z
    if constexpr (PT) ab_pt = dq_affine<BITS>(wfmt, ((const float *)p.meta)[0], ((const float *)p.meta)[1]);

    // Activations of step ks into dst: 4 direct loads per wavefront, each writing
    // 1 KiB of LDS (8 rows); lane L of load i fills slot L % 8 of row
    // 32 wave + 8 i + L / 8 with the chunk that belongs there under the swizzle.
    auto load_act = [&](int ks, _Float16 *dst) {
        const int64_t k0 = k00 + (int64_t)ks * QBK;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int row = 32 * wave + 8 * i + (lane >> 3), slot = lane & 7;
            const int c = slot ^ ((row >> 1) & 7);
            const int64_t r = (m0 + row < p.M) ? m0 + row : p.M - 1;  // rows past M: clamped, never stored
            __builtin_amdgcn_global_load_lds((glb_void *)(p.act + r * p.K + k0 + 8 * c),
                                             (lds_void *)(dst + (32 * wave + 8 * i) * QBK), 16, 0, 0);
        }
    };
    // packed weights of step ks for this thread: 32 indices of each plane (one 32-bit
    // word, the thread's half of the step) and the group's metadata word
    struct WReg {
        uint32_t b[BITS];
        uint32_t m;
    };
    auto load_w = [&](int ks, WReg &w) {
        const int64_t k0 = k00 + (int64_t)ks * QBK;
        const int64_t kb = k0 / KBLK;
        const int dw = 2 * (ks & 1) + hf;  // word of the 128-k plane word (k00 is a multiple of 128)
#pragma unroll
        for (int t = 0; t < BITS; ++t) w.b[t] = ((const uint32_t *)(p.planes + (kb * BITS + t) * p.N_pad + n))[dw];
        if constexpr (!PT) w.m = ((const uint32_t *)p.meta)[(int64_t)((uint32_t)k0 / (uint32_t)p.G) * p.N_pad + n];
        else w.m = 0u;
    };
    // weights 32 hf .. 32 hf + 31 of the step for column col, in four parts of 8 (one
    // 16-byte LDS store each): the affine coefficients and the Eq. 6-undone words first
    struct DqPrep {
        float2 ab;
        uint32_t raw[BITS];
    };
    auto dq_prep = [&](const WReg &w) {
        DqPrep d;
        if constexpr (PT) d.ab = ab_pt;
        else d.ab = dq_affine<BITS>(wfmt, dq_h2f(w.m & 0xFFFFu), dq_h2f(w.m >> 16));
#pragma unroll
        for (int t = 0; t < BITS; ++t) d.raw[t] = undo_eq6(w.b[t]);
        return d;
    };
    auto dq_part = [&](const DqPrep &d, int it, _Float16 *dst) {
        uint32_t packed[4];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            uint32_t qb = 0;  // byte e: bit e of each plane's index, i.e. weight 3 - e
#pragma unroll
            for (int t = 0; t < BITS; ++t) qb |= spread_nibble(d.raw[t], 2 * it + u) << t;
            const float r3 = fmaf(d.ab.x, ubyte_f(qb, 0), d.ab.y), r2 = fmaf(d.ab.x, ubyte_f(qb, 1), d.ab.y);
            const float r1 = fmaf(d.ab.x, ubyte_f(qb, 2), d.ab.y), r0 = fmaf(d.ab.x, ubyte_f(qb, 3), d.ab.y);
            packed[2 * u] = (uint32_t)__half_as_ushort(__float2half_rn(r0)) |
                            ((uint32_t)__half_as_ushort(__float2half_rn(r1)) << 16);
            packed[2 * u + 1] = (uint32_t)__half_as_ushort(__float2half_rn(r2)) |
                                ((uint32_t)__half_as_ushort(__float2half_rn(r3)) << 16);
        }
        *(uint4 *)(dst + col * QST + 32 * hf + 8 * it) = make_uint4(packed[0], packed[1], packed[2], packed[3]);
    };

    // One K step: MFMAs on (as, bs) while the next step's activations stream into
    // as_n and the next step's weights (wn_, requested one step earlier) are
    // dequantized into bs_n, a quarter per 16-deep sub-step, interleaved with the
    // MFMAs; the weights two steps ahead are requested into wl_.  Indices past the
    // last step are clamped to it, so every load and store is unconditional (the
    // buffers they fill at the last step are never read).
    auto step = [&](int ks, const _Float16 *as, const _Float16 *bs, _Float16 *as_n, _Float16 *bs_n,
                    const WReg &wn_, WReg &wl_) {
        load_act(ks + 1 < nk ? ks + 1 : nk - 1, as_n);
        load_w(ks + 2 < nk ? ks + 2 : nk - 1, wl_);
        const DqPrep dq = dq_prep(wn_);
        // operand fragments double-buffered across the four 16-deep sub-steps
        half8_t a[2][4], b[2][2];
        auto read_frags = [&](int kk, int f) {
            const int c = 2 * kk + (lane >> 5);  // 16-byte chunk of the K step this lane supplies
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = wm + 32 * i + (lane & 31);
                a[f][i] = *(const half8_t *)(as + row * QBK + 8 * (c ^ ((row >> 1) & 7)));
            }
#pragma unroll
            for (int j = 0; j < 2; ++j) b[f][j] = *(const half8_t *)(bs + (wn + 32 * j + (lane & 31)) * QST + 8 * c);
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
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[f][i], b[f][j], acc[i][j], 0, 0, 0);
            dq_part(dq, kk, bs_n);
            // issue order: MFMAs spaced by the next sub-step's LDS reads and a share of
            // the dequantization arithmetic
            if (kk + 1 < QBK / 16) {
#pragma unroll
                for (int t = 0; t < 6; ++t) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one MFMA
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
                    __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);  // VALU
                }
                __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
                __builtin_amdgcn_sched_group_barrier(0x002, 20, 0);
                __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // the LDS store
            } else {
#pragma unroll
                for (int t = 0; t < 8; ++t) {
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);
                }
                __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        __builtin_amdgcn_s_waitcnt(0);  // this wavefront's loads (direct LDS ones included) have landed
        __syncthreads();
    };

    WReg wA, wB;
    load_act(0, As0);
    load_w(0, wA);
    load_w(1, wB);  // nk >= 2
    {
        const DqPrep dq = dq_prep(wA);
#pragma unroll
        for (int it = 0; it < 4; ++it) dq_part(dq, it, Bs0);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    for (int ks = 0; ks < nk; ks += 2) {           // nk is even
        step(ks, As0, Bs0, As1, Bs1, wB, wA);      // dequantizes step ks + 1 from wB, loads ks + 2 into wA
        step(ks + 1, As1, Bs1, As0, Bs0, wA, wB);  // dequantizes step ks + 2 from wA, loads ks + 3 into wB
    }

    // epilogue: lane holds column (lane % 32), rows 8*(v/4) + 4*(lane/32) + v%4 of each block
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int64_t c = n0 + wn + 32 * j + (lane & 31);
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int64_t row = m0 + wm + 32 * i + 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
                dq_store(p, row, c, acc[i][j][v]);
            }
        }
}

// ---------------------------------------------------------------- few tokens
//
// 1-bit weights (BINARY, one scale per column or per tensor) and up to 16 tokens per
// workgroup: v_mfma_f32_16x16x32_f16 on 16-token slabs.  A workgroup owns 256
// columns (64 per wavefront, four 16-column MFMA blocks) and kbs 128-blocks of K.
//
// The order of k inside an MFMA is free as long as both operands follow it, so it is
// chosen to make the weight decode cheap.  Lane (r, g) = (lane % 16, lane / 16) of a
// 16-column block takes the 32-bit word g (weights 32 g .. 32 g + 31 of the 128-block)
// of column r and undoes the Eq. 6 inversion on the whole word (a set bit marks a +1).
// Shifted left by h (0 .. 15), the word holds its bits 15 - h and 31 - h at the sign
// positions of an FP16 pair, so one shift and one three-input bit operation (the
// inverted sign bits over 0x3C003C00) give two FP16 weights +-1; MFMA step st uses
// h = 4 st .. 4 st + 3.
// Bit b of a word is weight 4 (b / 4) + 3 - b % 4 (the first weight of a 4-group in
// its bit 3), so pair h = 4 st + t holds weights 4 (3 - st) + t (low half) and
// 4 (7 - st) + t (high half).  The activations are staged in LDS in exactly that
// order, in chunks of at most 16 128-blocks (64 KiB); 16-byte slot j of a block's
// 256 bytes in row r is stored at slot j ^ r, so the operand reads of the 16 rows
// hit distinct banks.  The packed words are requested
// nontemporally eight 128-blocks ahead (a ring of registers); the column scale
// multiplies the FP32 result.  At a few tokens the decode, not the matrix cores, is
// the work: no decoded weight is reused beyond the slab's 16 tokens.
constexpr int SK_CHUNK = 16;  // 128-blocks of activations staged in LDS at once
constexpr int SK_RING = 8;    // 128-blocks of weight words in flight per lane
constexpr int SK_STAGE = 4;   // staging items per thread: 16 rows x SK_CHUNK blocks x 4 words / 256
typedef float floatx4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

inline size_t skinny_lds_bytes(int kbs) {
    const int ch = kbs < SK_CHUNK ? kbs : SK_CHUNK;
    return (size_t)16 * ch * KBLK * 2;
}

// undo_eq6 with the multiply by 7 done on 16-bit halves (full rate; each half of
// (w >> 3) & 0x11111111 times 7 stays below 2^16).
__device__ __forceinline__ uint32_t undo_eq6_pk(uint32_t w) {
    typedef unsigned short u16x2_t __attribute__((ext_vector_type(2)));
    const u16x2_t t = __builtin_bit_cast(u16x2_t, (w >> 3) & 0x11111111u);
    return w ^ __builtin_bit_cast(uint32_t, t * (u16x2_t){7, 7});
}

// A workgroup barrier that orders LDS only (global loads in flight stay in flight).
__device__ __forceinline__ void dq_lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__global__ __launch_bounds__(256) void dequant_skinny_kernel(DequantParams p, int per_tensor) {
    extern __shared__ __attribute__((aligned(16))) _Float16 As[];  // [16][row_h] halves
    const int ch = p.kbs < SK_CHUNK ? p.kbs : SK_CHUNK;
    const int row_h = ch * KBLK;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int r = lane & 15, g = lane >> 4;
    const int64_t ncol0 = (int64_t)blockIdx.x * NTILE + wave * 64;
    const int64_t kb0 = (int64_t)blockIdx.z * p.kbs;
    const int nkb = (int)(p.KB - kb0 < p.kbs ? p.KB - kb0 : p.kbs);
    const int64_t m0 = (int64_t)blockIdx.y * 16;

    // Activation staging, one item per (row, block, word g2) = the 32 activations of
    // word g2 of the block, 64 contiguous bytes (four 16-byte loads); all of a thread's
    // loads are issued before any of its LDS stores (at most 4 items per thread: nc <=
    // 16), and each item gives the four operand chunks of steps st = 0..3: the 4
    // activations from 4 (3 - st) (low halves) and from 4 (7 - st) (high halves)
    // interleaved.  Rows past M are zero; item indices past the chunk are clamped and
    // not stored.  A wavefront's loads return in issue order, so the first chunk's are
    // issued before the weight ring: behind it they would wait for the weight stream.
    uint4 xv[SK_STAGE][4];
    auto stage_load = [&](int c0, int nc) {
        const int items = 16 * nc * 4;
#pragma unroll
        for (int u = 0; u < SK_STAGE; ++u) {
            const int i = tid + 256 * u, ic = i < items ? i : items - 1;
            const int row = ic / (nc * 4), rest = ic % (nc * 4);
            const int64_t mr = m0 + row < p.M ? m0 + row : p.M - 1;
            const uint4 *src = (const uint4 *)(p.act + mr * p.K + (kb0 + c0 + (rest >> 2)) * KBLK + 32 * (rest & 3));
#pragma unroll
            for (int j = 0; j < 4; ++j) xv[u][j] = src[j];
        }
    };
    auto stage_store = [&](int nc) {
        const int items = 16 * nc * 4;
#pragma unroll
        for (int u = 0; u < SK_STAGE; ++u) {
            const int i = tid + 256 * u;
            if (i < items) {
                const int row = i / (nc * 4), rest = i % (nc * 4);
                const int blk = rest >> 2, g2 = rest & 3;
                const bool live = m0 + row < p.M;
                const uint32_t X[16] = {xv[u][0].x, xv[u][0].y, xv[u][0].z, xv[u][0].w, xv[u][1].x, xv[u][1].y,
                                        xv[u][1].z, xv[u][1].w, xv[u][2].x, xv[u][2].y, xv[u][2].z, xv[u][2].w,
                                        xv[u][3].x, xv[u][3].y, xv[u][3].z, xv[u][3].w};
#pragma unroll
                for (int st = 0; st < 4; ++st) {
                    const uint32_t lx = X[2 * (3 - st)], ly = X[2 * (3 - st) + 1];
                    const uint32_t hx = X[2 * (7 - st)], hy = X[2 * (7 - st) + 1];
                    uint4 v = make_uint4(__builtin_amdgcn_perm(hx, lx, 0x05040100u), __builtin_amdgcn_perm(hx, lx, 0x07060302u),
                                         __builtin_amdgcn_perm(hy, ly, 0x05040100u), __builtin_amdgcn_perm(hy, ly, 0x07060302u));
                    if (!live) v = make_uint4(0u, 0u, 0u, 0u);
                    *(uint4 *)(As + row * row_h + blk * KBLK + 8 * ((4 * g2 + st) ^ row)) = v;
                }
            }
        }
    };
    stage_load(0, nkb < ch ? nkb : ch);
    __builtin_amdgcn_sched_barrier(0);  // keep the activation loads ahead of the weight ring

    // word g of column ncol0 + 16 cb + r in 128-block kbl of the range (clamped to the
    // last block: loads past the range repeat it and are never used)
    uint32_t w[SK_RING][4];
    const uint32_t *wbase = (const uint32_t *)(p.planes + kb0 * p.N_pad + ncol0 + r) + g;
    auto load_w = [&](int kbl, uint32_t(&d)[4]) {
        const int64_t kb = kbl < nkb ? kbl : nkb - 1;
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) d[cb] = __builtin_nontemporal_load(wbase + (kb * p.N_pad + 16 * cb) * 4);
    };
#pragma unroll
    for (int u = 0; u < SK_RING; ++u) load_w(u, w[u]);

    floatx4_t acc[4];
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) acc[cb] = floatx4_t{0.f, 0.f, 0.f, 0.f};

    // the MFMAs of 128-block kb_l (LDS column blk) with the weight words d
    auto block = [&](int blk, const uint32_t(&d)[4]) {
        const _Float16 *arow = As + r * row_h + blk * KBLK;
        uint32_t y[4];
#pragma unroll
        for (int cb = 0; cb < 4; ++cb) y[cb] = undo_eq6_pk(d[cb]);
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            const half8_t a = *(const half8_t *)(arow + 8 * ((4 * g + st) ^ r));
#pragma unroll
            for (int cb = 0; cb < 4; ++cb) {
                u32x4_t bw;
#pragma unroll
                for (int t = 0; t < 4; ++t) bw[t] = (~(y[cb] << (4 * st + t)) & 0x80008000u) | 0x3C003C00u;
                acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, __builtin_bit_cast(half8_t, bw), acc[cb], 0, 0, 0);
            }
        }
    };

    // the first chunk, loaded before the weight ring, in straight-line code (so the
    // compiler's waits count only the activation loads ahead of the ring)
    stage_store(nkb < ch ? nkb : ch);
    dq_lds_barrier();
    for (int c0 = 0; c0 < nkb; c0 += ch) {
        const int nc = nkb - c0 < ch ? nkb - c0 : ch;
        if (c0) {
            dq_lds_barrier();  // every wavefront is done with the previous chunk
            stage_load(c0, nc);
            stage_store(nc);
            dq_lds_barrier();
        }

        // whole groups of SK_RING blocks: no condition in the body, so the waits for the
        // ring's loads stay exact
        int kk = 0;
        for (; kk + SK_RING <= nc; kk += SK_RING) {
#pragma unroll
            for (int u = 0; u < SK_RING; ++u) {
                block(kk + u, w[u]);
                load_w(c0 + kk + u + SK_RING, w[u]);
                // keep the blocks in order (hoisting every decode to the top of the group
                // would wait for all of the ring's loads at once)
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        // the rest of the last chunk (its words are already in the ring)
#pragma unroll
        for (int u = 0; u < SK_RING; ++u)
            if (kk + u < nc) block(kk + u, w[u]);
    }

    // epilogue: acc[cb][j] is token 4 (lane / 16) + j, column 16 cb + lane % 16
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
        const int64_t col = ncol0 + 16 * cb + r;
        const float sc = per_tensor ? ((const float *)p.meta)[lane_value_dq(0)]
                                    : dq_h2f(((const uint32_t *)p.meta)[lane_value_dq(col)] & 0xFFFFu);
#pragma unroll
        for (int j = 0; j < 4; ++j) dq_store(p, m0 + 4 * g + j, col, acc[cb][j] * sc);
    }
}

// Sums the K-split partials of output (m, n) in split order, then the output
// epilogue (accumulate, dtype).  One lane per column, 256 per workgroup.
__global__ __launch_bounds__(256) void dequant_reduce_kernel(DequantParams p) {
    const int64_t n = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t m = blockIdx.y;
    if (n >= p.N) return;
    float y = 0.f;
    for (int s = 0; s < p.splits; ++s) y += p.part[((int64_t)s * p.M + m) * p.N_pad + n];
    const int64_t o = m * p.N + n;
    if (p.out_dtype == LUTGEMM_OUT_FP32) {
        if (p.accumulate) y += ((const float *)p.out)[o];
        ((float *)p.out)[o] = y;
    } else {
        if (p.accumulate) y += __half2float(((const __half *)p.out)[o]);
        ((__half *)p.out)[o] = __float2half_rn(y);
    }
}

// Kernel and K split of the comparison path.  1-bit weights with one scale per column
// (or tensor) and at most 64 tokens: the 16-token-slab kernel, K split until the grid
// has about 2 x 256 workgroups (at least 4 blocks per split).  Otherwise the pipelined
// 256 x 256 kernel when M >= 128 and it has at least 32 tiles, K split into as many
// ranges as keep the grid within one workgroup per CU (256; a second, partial round
// costs more than the split saves); else 128 x 128 tiles, K split until the grid has
// about 256 workgroups.  A split costs FP32 partial sums of splits x M x N_pad
// and the reduce launch.  LUTGEMM_TUNE_DEQUANT_KIND and LUTGEMM_TUNE_DEQUANT_SPLITS
// force the kernel and the split count (clamped to the 128-blocks of K).
DequantPlan plan_dequant(const Layout &L, int64_t M) {
    DequantPlan P{};
    const int force = tuning(LUTGEMM_TUNE_DEQUANT_KIND);
    const int force_splits = tuning(LUTGEMM_TUNE_DEQUANT_SPLITS);
    const int64_t tiles256 = (L.N_pad / QBN) * ((M + QBM - 1) / QBM);
    // splits = ceil(target / base), or floor (at least 1) when one round of workgroups
    // must not spill over the target (one workgroup per CU)
    auto split_for = [&](int64_t base, int64_t target, int64_t min_kbs, bool floor_div = false) {
        int64_t splits = base >= target ? 1 : floor_div ? target / base : (target + base - 1) / base;
        const int64_t max_splits = L.KB / min_kbs > 1 ? L.KB / min_kbs : 1;
        if (splits > max_splits) splits = max_splits;
        if (force_splits > 0) splits = force_splits < L.KB ? force_splits : L.KB;
        const int64_t kbs = (L.KB + splits - 1) / splits;
        P.kbs = (int)kbs;
        P.splits = (int)((L.KB + kbs - 1) / kbs);
    };
    const bool slab_ok = L.wfmt == LUTGEMM_WFMT_BINARY && (L.per_tensor || L.Q == 1);
    if (slab_ok && (force == 2 || (force < 0 && M <= 64))) {
        P.kind = 2;
        split_for((L.N_pad / NTILE) * ((M + 15) / 16), 512, 4);
    } else if (force == 1 || (force < 0 && M >= 128 && tiles256 * 8 >= 256)) {
        P.kind = 1;
        split_for(tiles256, 256, 1, true);
    } else {
        P.kind = 0;
        split_for((L.N_pad / DBN) * ((M + DBM - 1) / DBM), 256, 1);
    }
    P.ws_bytes = P.splits > 1 ? align256((size_t)P.splits * M * L.N_pad * 4) : 0;
    return P;
}

int launch_dequant(const DequantParams &p, const Layout &L, const DequantPlan &plan, void *stream) {
    hipStream_t s = (hipStream_t)stream;
    const int pt = L.per_tensor ? 1 : 0;
    const unsigned sp = (unsigned)plan.splits;
    if (plan.kind == 2) {
        const dim3 grid((unsigned)(L.N_pad / NTILE), (unsigned)((p.M + 15) / 16), sp);
        hipLaunchKernelGGL(dequant_skinny_kernel, grid, dim3(256), skinny_lds_bytes(plan.kbs), s, p, pt);
    } else if (plan.kind == 1) {
        const dim3 big((unsigned)(L.N_pad / QBN), (unsigned)((p.M + QBM - 1) / QBM), sp);
        const dim3 blk(512);
        if (pt) {
            if (L.bits == 1) hipLaunchKernelGGL((dequant_mfma_big_kernel<1, true>), big, blk, 0, s, p, L.wfmt);
            else if (L.bits == 2) hipLaunchKernelGGL((dequant_mfma_big_kernel<2, true>), big, blk, 0, s, p, L.wfmt);
            else hipLaunchKernelGGL((dequant_mfma_big_kernel<4, true>), big, blk, 0, s, p, L.wfmt);
        } else {
            if (L.bits == 1) hipLaunchKernelGGL((dequant_mfma_big_kernel<1, false>), big, blk, 0, s, p, L.wfmt);
            else if (L.bits == 2) hipLaunchKernelGGL((dequant_mfma_big_kernel<2, false>), big, blk, 0, s, p, L.wfmt);
            else hipLaunchKernelGGL((dequant_mfma_big_kernel<4, false>), big, blk, 0, s, p, L.wfmt);
        }
    } else {
        const dim3 grid((unsigned)(L.N_pad / DBN), (unsigned)((p.M + DBM - 1) / DBM), sp);
        if (L.bits == 1)
            hipLaunchKernelGGL(dequant_mfma_kernel<1>, grid, dim3(256), 0, s, p, L.wfmt, pt);
        else if (L.bits == 2)
            hipLaunchKernelGGL(dequant_mfma_kernel<2>, grid, dim3(256), 0, s, p, L.wfmt, pt);
        else
            hipLaunchKernelGGL(dequant_mfma_kernel<4>, grid, dim3(256), 0, s, p, L.wfmt, pt);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || plan.splits == 1) return (int)e;
    hipLaunchKernelGGL(dequant_reduce_kernel, dim3((unsigned)(L.N_pad / 256), (unsigned)p.M), dim3(256), 0, s, p);
    return (int)hipGetLastError();
}

}  // namespace lutgemm
