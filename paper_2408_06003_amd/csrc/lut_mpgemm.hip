// Bit-serial LUT mpGEMM (LUT Tensor Core, Section 3.1 bit-serial tables with
// Eq. 3, 5 and 6; LMMA semantics O = A x W^T + Acc, Section 3.3.1).
//
// gfx950 mapping.  Each lane owns one output column and a wavefront covers 64
// consecutive columns, so one table entry read from LDS is reused by every
// column of the workgroup (the "elongated N" reuse of Section 3.2.2), all lanes
// of a wavefront read the same 16-entry table at any time (no LDS bank
// conflicts), and a wavefront's weight loads are 1 KiB contiguous 128-bit loads.
//
// Per workgroup and K range, the half tables of Eq. 5 (8 entries per 4
// activations, HBM format) are expanded once into full 16-entry signed tables
// in LDS, F[s i] = (s ? -T[i] : T[i]), so the stored Eq. 6 index addresses the
// entry directly and no per-lookup negation is needed.  Entries are INT32:
// exact integers on the INT8 path, and FP16 values times 2^20 on the FP path
// (exact for |T| >= 2^-10, otherwise within 2^-21; tables are normalized to
// |T| < 4 by the precompute), which lets one v_add3_u32 accumulate two lookups.
//
// A lookup costs one byte-select AND (SDWA) to form the LDS address, one
// ds_read_b32, and half of a v_add3_u32.  Each bit-plane t has its own INT32
// accumulator; at the end of every 128-wide K block the planes are combined as
// sum_t 2^t acc_t and the Eq. 3 epilogue s' (A - z' S) is applied in FP32.
//
// K is split across workgroups when the grid would otherwise be too small to
// fill 256 CUs; the last workgroup to finish a column tile (arrival counter)
// sums the partials in split order, so results are bitwise reproducible.
#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>

#include "lutgemm_internal.h"

namespace lutgemm {

__device__ __forceinline__ float h2f(uint32_t bits16) {
    return __half2float(__ushort_as_half((unsigned short)bits16));
}

// (byte B of w) & 0x3C: a 4-bit index pre-shifted left by 2 becomes an INT32
// table offset in one VALU op (SDWA byte select).
template <int B>
__device__ __forceinline__ uint32_t idx4(uint32_t w) {
    uint32_t r;
    if constexpr (B == 0)
        asm("v_and_b32_sdwa %0, 60, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_0"
            : "=v"(r) : "v"(w));
    else if constexpr (B == 1)
        asm("v_and_b32_sdwa %0, 60, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_1"
            : "=v"(r) : "v"(w));
    else if constexpr (B == 2)
        asm("v_and_b32_sdwa %0, 60, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_2"
            : "=v"(r) : "v"(w));
    else
        asm("v_and_b32_sdwa %0, 60, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_3"
            : "=v"(r) : "v"(w));
    return r;
}

__device__ __forceinline__ int lds_i32(const char *base, uint32_t off) {
    return *(const int *)(base + off);
}

// Expand one half table (8 entries, 16 bytes) into a 16-entry INT32 signed table.
template <bool INT8>
__device__ __forceinline__ void expand_table(const uint4 h, int *dst) {
    const uint32_t w[4] = {h.x, h.y, h.z, h.w};
    int v[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        if (INT8) {
            v[2 * i] = (int)(int16_t)(uint16_t)(w[i] & 0xFFFFu);
            v[2 * i + 1] = (int)(int16_t)(uint16_t)(w[i] >> 16);
        } else {
            v[2 * i] = (int)rintf(h2f(w[i] & 0xFFFFu) * (float)(1 << FIX_SHIFT));
            v[2 * i + 1] = (int)rintf(h2f(w[i] >> 16) * (float)(1 << FIX_SHIFT));
        }
    }
    int4 *d4 = (int4 *)dst;
    d4[0] = make_int4(v[0], v[1], v[2], v[3]);
    d4[1] = make_int4(v[4], v[5], v[6], v[7]);
    d4[2] = make_int4(-v[0], -v[1], -v[2], -v[3]);
    d4[3] = make_int4(-v[4], -v[5], -v[6], -v[7]);
}

// Reinterpreted scale and zero (Eq. 2) of quantization group q, column n.
struct SZ {
    float sp, zp;
};

// Branch-free so that the lookup adds stay in the basic block of their LDS reads.
__device__ __forceinline__ SZ load_sz(const LutParams &p, int q, int64_t n) {
    const float *mf = (const float *)p.meta;
    const int64_t idx = p.per_tensor ? 0 : (int64_t)q * p.N_pad + n;
    const uint32_t mz = ((const uint32_t *)p.meta)[idx];
    const float s = p.per_tensor ? mf[0] : h2f(mz & 0xFFFFu);
    const float z = p.per_tensor ? mf[1] : h2f(mz >> 16);
    SZ r;
    r.sp = p.cs * s;
    r.zp = fmaf(p.cz, z, p.c0);
    return r;
}

// Per-column weight scale of the INT8 path (per-tensor or per-channel).
__device__ __forceinline__ float int_weight_scale(const LutParams &p, bool per_tensor, int64_t n) {
    if (per_tensor) return ((const float *)p.meta)[0];
    return h2f(((const uint32_t *)p.meta)[n] & 0xFFFFu);
}

// Final value of output (m, n): scale, optional accumulate, dtype conversion.
template <bool INT8>
__device__ __forceinline__ void store_out(const LutParams &p, int wfmt, bool per_tensor, int64_t m,
                                          int64_t n, float yf, int yi) {
    if (n >= p.N) return;
    const int64_t o = m * p.N + n;
    if (INT8) {
        const int y = (wfmt == LUTGEMM_WFMT_TERNARY) ? (yi >> 1) : yi;  // (A + S) / 2 is exact
        if (p.out_dtype == LUTGEMM_OUT_INT32) {
            int v = y;
            if (p.accumulate) v += ((const int *)p.out)[o];
            ((int *)p.out)[o] = v;
            return;
        }
        float v = ((float)y * p.tok[m]) * int_weight_scale(p, per_tensor, n);
        if (p.out_dtype == LUTGEMM_OUT_FP32) {
            if (p.accumulate) v += ((const float *)p.out)[o];
            ((float *)p.out)[o] = v;
        } else {
            if (p.accumulate) v += __half2float(((const __half *)p.out)[o]);
            ((__half *)p.out)[o] = __float2half_rn(v);
        }
        return;
    }
    float v = p.tok[m] * yf;
    if (p.out_dtype == LUTGEMM_OUT_FP32) {
        if (p.accumulate) v += ((const float *)p.out)[o];
        ((float *)p.out)[o] = v;
    } else {
        if (p.accumulate) v += __half2float(((const __half *)p.out)[o]);
        ((__half *)p.out)[o] = __float2half_rn(v);
    }
}

// Publishes this split's partial (m rows [m0, m0 + rows)), and returns true in
// the workgroup that arrives last for its (token tile, column tile).
__device__ __forceinline__ bool publish_partial(const LutParams &p, int64_t m_alloc, int split,
                                                int64_t m0, int rows, const float *vals, int64_t n,
                                                int64_t tile_id) {
    __shared__ int s_last;
    for (int r = 0; r < rows; ++r) {
        float *dst = p.part + ((int64_t)split * m_alloc + m0 + r) * p.N_pad + n;
        __hip_atomic_store(dst, vals[r], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t old =
            __hip_atomic_fetch_add(p.counters + tile_id, 1u, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
        s_last = (old == (uint32_t)(p.splits - 1));
        if (s_last) __hip_atomic_store(p.counters + tile_id, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    if (s_last) __threadfence();
    return s_last != 0;
}

__device__ __forceinline__ float read_partial(const LutParams &p, int64_t m_alloc, int split, int64_t m,
                                              int64_t n) {
    const float *src = p.part + ((int64_t)split * m_alloc + m) * p.N_pad + n;
    return __hip_atomic_load(src, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ------------------------------------------------------------------ single token

template <int BITS, int KBS, bool INT8>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void lut_gemv_kernel(LutParams p, int wfmt, int per_tensor_i) {
    __shared__ __attribute__((aligned(16))) int F[KBS * GPB * 16];
    const bool per_tensor = per_tensor_i != 0;
    const int tid = threadIdx.x;
    const int64_t n = (int64_t)blockIdx.x * NTILE + tid;
    const int split = blockIdx.y;
    const int64_t m = blockIdx.z;
    const int64_t kb0 = (int64_t)split * KBS;
    const int nkb = (int)((p.KB - kb0) < KBS ? (p.KB - kb0) : KBS);

    // issue every weight load of this split first
    uint4 w[KBS][BITS];
#pragma unroll
    for (int kbl = 0; kbl < KBS; ++kbl) {
        if (kbl < nkb) {
#pragma unroll
            for (int t = 0; t < BITS; ++t)
                w[kbl][t] = p.planes[((kb0 + kbl) * BITS + t) * p.N_pad + n];
        }
    }
    // epilogue operands of every 128-block, fetched before the lookups so that no
    // scalar-memory load is outstanding among the LDS reads (they share lgkmcnt)
    float e_scale[KBS], e_zero[KBS];
    if (!INT8) {
        int q = (int)(kb0 / p.kpg);
        int phase = (int)(kb0 - (int64_t)q * p.kpg);
#pragma unroll
        for (int kbl = 0; kbl < KBS; ++kbl) {
            e_scale[kbl] = 0.f;
            e_zero[kbl] = 0.f;
            if (kbl < nkb) {
                const SZ sz = load_sz(p, q, n);
                e_scale[kbl] = sz.sp * (1.0f / (float)(1 << FIX_SHIFT));
                // zero-point term of Eq. 3, once per quantization group
                e_zero[kbl] = phase == 0 ? sz.sp * sz.zp * ((const float *)p.S)[m * p.Q + q] : 0.f;
            }
            if (++phase == p.kpg) {
                phase = 0;
                ++q;
            }
        }
    }
    int s_total = 0;
    if (INT8 && split == 0 && wfmt == LUTGEMM_WFMT_TERNARY) s_total = ((const int *)p.S)[m * p.Q];
    // stage the signed tables of this K range
    if (tid < nkb * GPB) expand_table<INT8>(p.T[m * p.J + kb0 * GPB + tid], F + tid * 16);
    __syncthreads();

    const char *Fb = (const char *)F;
    float yf = 0.f;
    int yi = s_total;
#pragma unroll
    for (int kbl = 0; kbl < KBS; ++kbl) {
        if (kbl < nkb) {
            int acc[BITS];
#pragma unroll
            for (int t = 0; t < BITS; ++t) {
                acc[t] = 0;
                const uint32_t wd[4] = {w[kbl][t].x, w[kbl][t].y, w[kbl][t].z, w[kbl][t].w};
#pragma unroll
                for (int d = 0; d < 4; ++d) {
                    const uint32_t lo = wd[d] << 2, hi = wd[d] >> 2;
                    const uint32_t a0 = idx4<0>(lo), a1 = idx4<0>(hi), a2 = idx4<1>(lo), a3 = idx4<1>(hi);
                    const uint32_t a4 = idx4<2>(lo), a5 = idx4<2>(hi), a6 = idx4<3>(lo), a7 = idx4<3>(hi);
                    const uint32_t g = (uint32_t)((kbl * GPB + d * 8) * 64);
                    acc[t] += lds_i32(Fb + g + 0 * 64, a0) + lds_i32(Fb + g + 1 * 64, a1);
                    acc[t] += lds_i32(Fb + g + 2 * 64, a2) + lds_i32(Fb + g + 3 * 64, a3);
                    acc[t] += lds_i32(Fb + g + 4 * 64, a4) + lds_i32(Fb + g + 5 * 64, a5);
                    acc[t] += lds_i32(Fb + g + 6 * 64, a6) + lds_i32(Fb + g + 7 * 64, a7);
                }
            }
            // |sum_t 2^t acc_t| <= 15 * 32 * 2^22 < 2^31 on the FP path: exact in INT32
            int tot = 0;
#pragma unroll
            for (int t = 0; t < BITS; ++t) tot += acc[t] << t;
            if (INT8)
                yi += tot;
            else
                yf = fmaf(e_scale[kbl], (float)tot, yf) - e_zero[kbl];
        }
    }

    if (p.splits == 1) {
        store_out<INT8>(p, wfmt, per_tensor, m, n, yf, yi);
        return;
    }
    const float val = INT8 ? __int_as_float(yi) : yf;
    const int64_t tile_id = m * (p.N_pad / NTILE) + blockIdx.x;
    if (publish_partial(p, p.M, split, m, 1, &val, n, tile_id)) {
        float sf = 0.f;
        int si = 0;
        for (int s = 0; s < p.splits; ++s) {
            const float v = read_partial(p, p.M, s, m, n);
            if (INT8)
                si += __float_as_int(v);
            else
                sf += v;
        }
        store_out<INT8>(p, wfmt, per_tensor, m, n, sf, si);
    }
}

// ------------------------------------------------------------------ several tokens

constexpr int CH = 2;  // 128-blocks of K staged in LDS at a time

template <int BITS, int MT, bool INT8>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void lut_gemm_kernel(LutParams p, int wfmt, int per_tensor_i) {
    __shared__ __attribute__((aligned(16))) int F[MT * CH * GPB * 16];
    const bool per_tensor = per_tensor_i != 0;
    const int tid = threadIdx.x;
    const int64_t n = (int64_t)blockIdx.x * NTILE + tid;
    const int split = blockIdx.y;
    const int64_t m0 = (int64_t)blockIdx.z * MT;
    const int64_t kb_begin = (int64_t)split * p.kbs;
    const int64_t kb_end = (kb_begin + p.kbs < p.KB) ? kb_begin + p.kbs : p.KB;
    const char *Fb = (const char *)F;

    float yf[MT];
    int yi[MT];
#pragma unroll
    for (int r = 0; r < MT; ++r) {
        yf[r] = 0.f;
        yi[r] = 0;
    }

    if (INT8 && split == 0 && wfmt == LUTGEMM_WFMT_TERNARY) {
#pragma unroll
        for (int r = 0; r < MT; ++r)
            if (m0 + r < p.M) yi[r] = ((const int *)p.S)[(m0 + r) * p.Q];
    }
    int q = (int)(kb_begin / p.kpg);
    int phase = (int)(kb_begin - (int64_t)q * p.kpg);
    for (int64_t kc = kb_begin; kc < kb_end; kc += CH) {
        const int nkb = (int)((kb_end - kc) < CH ? (kb_end - kc) : CH);
        uint4 w[CH][BITS];
#pragma unroll
        for (int kbl = 0; kbl < CH; ++kbl) {
            if (kbl < nkb) {
#pragma unroll
                for (int t = 0; t < BITS; ++t) w[kbl][t] = p.planes[((kc + kbl) * BITS + t) * p.N_pad + n];
            }
        }
        // epilogue operands of this chunk, fetched before the lookups (see the GEMV kernel)
        float e_scale[CH], e_zero[CH][MT];
#pragma unroll
        for (int kbl = 0; kbl < CH; ++kbl) {
            e_scale[kbl] = 0.f;
#pragma unroll
            for (int r = 0; r < MT; ++r) e_zero[kbl][r] = 0.f;
            if (!INT8 && kbl < nkb) {
                const SZ sz = load_sz(p, q, n);
                e_scale[kbl] = sz.sp * (1.0f / (float)(1 << FIX_SHIFT));
                if (phase == 0) {
#pragma unroll
                    for (int r = 0; r < MT; ++r) {
                        const int64_t mr = (m0 + r < p.M) ? m0 + r : p.M - 1;  // rows past M are never stored
                        e_zero[kbl][r] = sz.sp * sz.zp * ((const float *)p.S)[mr * p.Q + q];
                    }
                }
            }
            if (kbl < nkb && ++phase == p.kpg) {
                phase = 0;
                ++q;
            }
        }
        __syncthreads();  // previous chunk's tables are no longer read
        for (int e = tid; e < MT * CH * GPB; e += 256) {
            const int r = e / (CH * GPB);
            const int jl = e % (CH * GPB);
            int *dst = F + e * 16;
            if (m0 + r < p.M && jl < nkb * GPB) {
                expand_table<INT8>(p.T[(m0 + r) * p.J + kc * GPB + jl], dst);
            } else {
                int4 *d4 = (int4 *)dst;
                d4[0] = d4[1] = d4[2] = d4[3] = make_int4(0, 0, 0, 0);
            }
        }
        __syncthreads();

#pragma unroll
        for (int kbl = 0; kbl < CH; ++kbl) {
            if (kbl < nkb) {
                int acc[MT][BITS];
#pragma unroll
                for (int t = 0; t < BITS; ++t) {
#pragma unroll
                    for (int r = 0; r < MT; ++r) acc[r][t] = 0;
                    const uint32_t wd[4] = {w[kbl][t].x, w[kbl][t].y, w[kbl][t].z, w[kbl][t].w};
#pragma unroll
                    for (int d = 0; d < 4; ++d) {
                        const uint32_t lo = wd[d] << 2, hi = wd[d] >> 2;
                        const uint32_t a[8] = {idx4<0>(lo), idx4<0>(hi), idx4<1>(lo), idx4<1>(hi),
                                               idx4<2>(lo), idx4<2>(hi), idx4<3>(lo), idx4<3>(hi)};
                        const uint32_t g = (uint32_t)((kbl * GPB + d * 8) * 64);
#pragma unroll
                        for (int r = 0; r < MT; ++r) {
                            const char *Fr = Fb + r * (CH * GPB * 64) + g;
#pragma unroll
                            for (int i = 0; i < 8; i += 2)
                                acc[r][t] += lds_i32(Fr + i * 64, a[i]) + lds_i32(Fr + (i + 1) * 64, a[i + 1]);
                        }
                    }
                }
                int tot[MT];
#pragma unroll
                for (int r = 0; r < MT; ++r) {
                    tot[r] = 0;
#pragma unroll
                    for (int t = 0; t < BITS; ++t) tot[r] += acc[r][t] << t;
                }
#pragma unroll
                for (int r = 0; r < MT; ++r) {
                    if (INT8)
                        yi[r] += tot[r];
                    else
                        yf[r] = fmaf(e_scale[kbl], (float)tot[r], yf[r]) - e_zero[kbl][r];
                }
            }
        }
    }
    const int rows = (int)((p.M - m0) < MT ? (p.M - m0) : MT);
    if (p.splits == 1) {
#pragma unroll
        for (int r = 0; r < MT; ++r)
            if (r < rows) store_out<INT8>(p, wfmt, per_tensor, m0 + r, n, yf[r], yi[r]);
        return;
    }
    float vals[MT];
#pragma unroll
    for (int r = 0; r < MT; ++r) vals[r] = INT8 ? __int_as_float(yi[r]) : yf[r];
    const int64_t m_alloc = (int64_t)gridDim.z * MT;
    const int64_t tile_id = (int64_t)blockIdx.z * (p.N_pad / NTILE) + blockIdx.x;
    if (publish_partial(p, m_alloc, split, m0, MT, vals, n, tile_id)) {
        for (int r = 0; r < rows; ++r) {
            float sf = 0.f;
            int si = 0;
            for (int s = 0; s < p.splits; ++s) {
                const float v = read_partial(p, m_alloc, s, m0 + r, n);
                if (INT8)
                    si += __float_as_int(v);
                else
                    sf += v;
            }
            store_out<INT8>(p, wfmt, per_tensor, m0 + r, n, sf, si);
        }
    }
}

// ------------------------------------------------------------------ dispatch

template <int BITS, bool INT8>
static void launch_gemv_kbs(const LutParams &p, const Layout &L, const LutPlan &plan, hipStream_t s) {
    dim3 grid((unsigned)plan.n_tiles, (unsigned)plan.splits, (unsigned)plan.m_tiles);
    const int pt = L.per_tensor ? 1 : 0;
    switch (plan.kbs) {
    case 1: hipLaunchKernelGGL((lut_gemv_kernel<BITS, 1, INT8>), grid, dim3(256), 0, s, p, L.wfmt, pt); break;
    case 2: hipLaunchKernelGGL((lut_gemv_kernel<BITS, 2, INT8>), grid, dim3(256), 0, s, p, L.wfmt, pt); break;
    case 4:
        if constexpr (BITS <= 2)
            hipLaunchKernelGGL((lut_gemv_kernel<BITS, 4, INT8>), grid, dim3(256), 0, s, p, L.wfmt, pt);
        break;
    default:
        if constexpr (BITS == 1)
            hipLaunchKernelGGL((lut_gemv_kernel<BITS, 8, INT8>), grid, dim3(256), 0, s, p, L.wfmt, pt);
        break;
    }
}

template <int BITS, bool INT8>
static void launch_gemm_mt(const LutParams &p, const Layout &L, const LutPlan &plan, hipStream_t s) {
    dim3 grid((unsigned)plan.n_tiles, (unsigned)plan.splits, (unsigned)plan.m_tiles);
    const int pt = L.per_tensor ? 1 : 0;
    if (plan.mt == 4)
        hipLaunchKernelGGL((lut_gemm_kernel<BITS, 4, INT8>), grid, dim3(256), 0, s, p, L.wfmt, pt);
    else
        hipLaunchKernelGGL((lut_gemm_kernel<BITS, 8, INT8>), grid, dim3(256), 0, s, p, L.wfmt, pt);
}

template <bool INT8>
static void launch_bits(const LutParams &p, const Layout &L, const LutPlan &plan, hipStream_t s) {
    if (plan.kind == 0) {
        if (L.bits == 1) launch_gemv_kbs<1, INT8>(p, L, plan, s);
        else if (L.bits == 2) launch_gemv_kbs<2, INT8>(p, L, plan, s);
        else launch_gemv_kbs<4, INT8>(p, L, plan, s);
    } else {
        if (L.bits == 1) launch_gemm_mt<1, INT8>(p, L, plan, s);
        else if (L.bits == 2) launch_gemm_mt<2, INT8>(p, L, plan, s);
        else launch_gemm_mt<4, INT8>(p, L, plan, s);
    }
}

int launch_lut(const LutParams &p, const Layout &L, const LutPlan &plan, void *stream) {
    hipStream_t s = (hipStream_t)stream;
    if (L.act == LUTGEMM_ACT_INT8)
        launch_bits<true>(p, L, plan, s);
    else
        launch_bits<false>(p, L, plan, s);
    return (int)hipGetLastError();
}

}  // namespace lutgemm
