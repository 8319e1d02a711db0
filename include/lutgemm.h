/*
 * lutgemm.h -- C ABI of an MI355X (gfx950) library for LUT-based
 * mixed-precision GEMM (mpGEMM) between low-bit weights and FP16 / INT8
 * activations, after "LUT Tensor Core: A Software-Hardware Co-Design for
 * LUT-Based Low-Bit LLM Inference" (arXiv 2408.06003).
 *
 * The operation (the paper's LMMA semantics, Section 3.3.1):
 *
 *     O[M, N] = A[M, K] x W[N, K]^T  (+ O[M, N] when accumulating)
 *
 * with real weights r = s (q - z) (Section 3.1.2, Eq. 1) and the dot product
 * evaluated by table lookup (Section 3.1, Eq. 3-6):
 *   - lutgemm_precompute builds, for every 4 activations, the 8-entry half
 *     table of signed partial sums made possible by reading weight bits {0,1}
 *     as {-1,+1} (Eq. 4-5), as an independent operator (Section 3.1.1);
 *   - lutgemm_pack_weights is the offline weight mapping: bit-serial planes
 *     (Section 3.1), reinterpretation (Eq. 2) and offline bit-level negation
 *     (Eq. 6);
 *   - lutgemm_mpgemm is the bit-serial lookup-accumulate with the
 *     scale / zero-point epilogue of Eq. 3.
 * lutgemm_mpgemm_dequant is a dequantize-to-FP16 + matrix-core comparison path
 * (the "indirect mpGEMM with dequantization" of Section 2.2).
 *
 * Conventions for every entry point:
 *   - Device pointers must be 16-byte aligned device memory; host pointers are
 *     marked as such.  The caller allocates and owns every buffer; the library
 *     never allocates, frees or retains a pointer after the call returns.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Work is enqueued
 *     asynchronously; no call synchronizes the host with the device.
 *   - Arguments are validated on the host before anything is enqueued: on any
 *     status other than LUTGEMM_SUCCESS nothing was launched.  A failed launch
 *     returns LUTGEMM_ERROR_HIP.
 *   - Calls on distinct streams with distinct workspaces are thread-safe.
 */
#ifndef LUTGEMM_H
#define LUTGEMM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    LUTGEMM_SUCCESS = 0,
    LUTGEMM_ERROR_INVALID_VALUE = 1,     /* null pointer, negative size, misaligned pointer, bad enum */
    LUTGEMM_ERROR_NOT_SUPPORTED = 2,     /* a valid but unsupported combination (see lutgemm_validate) */
    LUTGEMM_ERROR_INSUFFICIENT_SIZE = 3, /* a buffer smaller than its size query */
    LUTGEMM_ERROR_HIP = 4                /* the HIP runtime reported an error */
} lutgemm_status_t;

/* Weight formats (Section 3.1.2).  `codes` is [N][K], K contiguous. */
enum {
    LUTGEMM_WFMT_UINT = 0,    /* uint8 codes q in [0, 2^b), r = s (q - z); s, z FP16 per group   */
    LUTGEMM_WFMT_BINARY = 1,  /* uint8 codes q in {0,1} standing for {-1,+1}, r = s (2q - 1)        */
    LUTGEMM_WFMT_TERNARY = 2, /* int8 codes w in {-1,0,+1}, stored as q = w + 1 with b = 2, r = s w  */
    LUTGEMM_WFMT_TERNARY_3IN5 = 3 /* int8 codes w in {-1,0,+1}, r = s w, packed three weights per 5-bit
                                     code (Section 5, non-integer weights): one table of the 27
                                     patterns of 3 activations (half of it stored, by the symmetry
                                     of Eq. 4) and one lookup per 3 weights; w_bits = 2, per-tensor
                                     or per-channel scale (group_size 0 or K)                        */
};

/* Activation / table types. */
enum {
    LUTGEMM_ACT_FP16 = 0,     /* FP16 activations -> FP16 tables, FP32 accumulation              */
    LUTGEMM_ACT_INT8 = 1,     /* FP16 activations quantized per token to INT8 (absmax) -> INT16
                                 tables, exact INT32 accumulation (BINARY / TERNARY weights)     */
    LUTGEMM_ACT_FP16_LUT8 = 2 /* FP16 activations, tables quantized to INT8 with one FP32 scale
                                 per table (Section 3.1.3): an approximation (relative error of
                                 the output about 3e-3), 12 instead of 16 table bytes per 4
                                 activations (8 INT8 codes + FP32 scale); not
                                 with TERNARY_3IN5                                               */
};

/* Output types. */
enum {
    LUTGEMM_OUT_FP16 = 0,
    LUTGEMM_OUT_FP32 = 1,
    LUTGEMM_OUT_INT32 = 2     /* INT8 path only: the exact integer dot product sum_k q_a w       */
};

/*
 * Problem description.
 *   K, N        reduction length and number of output columns (weight rows); K % 128 == 0, N >= 1
 *   w_bits      b: 1, 2 or 4 for UINT; 1 for BINARY; 2 for TERNARY and TERNARY_3IN5
 *   wfmt        LUTGEMM_WFMT_*
 *   group_size  quantization group along K: a multiple of 128 that divides K (K = per channel),
 *               or 0 = a single scale (and zero) for the whole tensor
 *   scale_fp32  0: scales (and zeros) are FP16; 1: the scale is FP32 (per-tensor only, no zeros)
 *   act         LUTGEMM_ACT_*
 */
typedef struct {
    int64_t K;
    int64_t N;
    int32_t w_bits;
    int32_t wfmt;
    int32_t group_size;
    int32_t scale_fp32;
    int32_t act;
    int32_t reserved; /* must be 0 */
} lutgemm_problem_t;

/* Static string for a status code. */
const char *lutgemm_status_string(lutgemm_status_t status);

/* Library version string. */
const char *lutgemm_version(void);

/* Text of the HIP error behind the calling thread's most recent
 * LUTGEMM_ERROR_HIP ("" if none).  Valid until the thread's next call. */
const char *lutgemm_last_error(void);

/*
 * Host-only check of a problem and token count M (M >= 1; pass M = 1 when M does
 * not matter).  Needs no GPU.  Returns LUTGEMM_ERROR_INVALID_VALUE for malformed
 * input (null, K or N <= 0, unknown enum, reserved != 0) and
 * LUTGEMM_ERROR_NOT_SUPPORTED for: K % 128 != 0; group_size not 0 and not a
 * multiple of 128 dividing K; w_bits not allowed for wfmt; scale_fp32 with
 * group_size != 0 or with UINT; ACT_INT8 with UINT weights or with a group
 * smaller than K; K > 2^20, N > 2^24 or M > 2^19; M > 2 with
 * ceil(M/8) * ceil(N/256) >= 2^24; TERNARY_3IN5 with a group other than 0 or K,
 * with ceil(N/16) * M >= 2^24, or with ACT_FP16_LUT8.
 */
lutgemm_status_t lutgemm_validate(const lutgemm_problem_t *problem, int64_t M);

/* Bytes of the packed-weight buffer (opaque layout).  0 for an invalid problem. */
size_t lutgemm_packed_weight_size(const lutgemm_problem_t *problem);

/*
 * Bytes of the table buffer written by lutgemm_precompute for M tokens.  The
 * layout is public so that another kernel can produce it (e.g. fused into the
 * operator that produces the activations, Section 3.1.1), with J = K/4 table
 * groups and Q = K/group_size quantization groups (Q = 1 per-tensor):
 *   offset 0:      T[M][J][8]   half tables, FP16 (ACT_FP16) or INT16 (ACT_INT8);
 *                  T[m][j][i] = sum_{e<4} x_{4j+e} (2 b_e - 1) where b_0 = 0 and
 *                  b_e = bit (3-e) of i (Eq. 5: the first activation of the group
 *                  is the pattern's MSB), x = a * 2^-e_m (FP16) or q_a (INT8)
 *   offset s_off:  S[M][Q]      sum of x over each quantization group, FP32 or INT32
 *   offset t_off:  t[M]         per-token factor, FP32: 2^e_m for ACT_FP16, where
 *                  max_k |a[m,k]| = f 2^e_m with f in [0.5, 1) (1 for an all-zero row);
 *                  the absmax scale s_a = amax / 127 for ACT_INT8
 * with s_off = align256(16 M J) and t_off = align256(s_off + 4 M Q).
 * ACT_FP16_LUT8 instead of the FP16 T:
 *   offset 0:      T8[M][J][8]  INT8 codes of each half table: amax = max_i |T[i]| (T as
 *                  for ACT_FP16, FP32), T8[i] = clamp(rint(T[i] * (127 / amax)), -127, 127)
 *   offset sc_off: sc[M][J]     FP32 amax / 127 (0 for an all-zero table)
 * with sc_off = align256(8 M J), s_off = align256(sc_off + 4 M J); S and t as for ACT_FP16.
 * TERNARY_3IN5 instead: J = 32 ceil(K/96) triples and
 *   offset 0:      T[M][J][16]  triple tables, FP16 or INT16, entries 14 and 15 zero;
 *                  T[m][j][i] = sum_{e<3} x_{3j+e} w_e(13 + i) for i < 14, where
 *                  w_e(v) is digit e of v in base 3 (most significant first) minus 1
 *                  and x_k = 0 for k >= K (entry i is the triple pattern 13 + i; its
 *                  negation is pattern 13 - i, Eq. 4)
 *   offset s_off:  unused (no zero point)
 *   offset t_off:  t[M] as above
 * with s_off = align256(32 M J).
 * 0 for an invalid problem.
 */
size_t lutgemm_table_size(const lutgemm_problem_t *problem, int64_t M);

/* Offsets of S and t inside the table buffer (see lutgemm_table_size). */
lutgemm_status_t lutgemm_table_offsets(const lutgemm_problem_t *problem, int64_t M,
                                       size_t *s_offset, size_t *t_offset);

/* Leading bytes of every nonempty workspace that are zero between calls. */
#define LUTGEMM_WORKSPACE_ZERO_BYTES ((size_t)1 << 20)

/*
 * Bytes of scratch memory lutgemm_mpgemm needs for M tokens (partial sums when K
 * is split across workgroups, and the arrival counters and exact split-sum words
 * with which the single-token split-K kernel completes the split itself); may be 0.
 * The workspace must be zero-filled before its first use.  Its first
 * LUTGEMM_WORKSPACE_ZERO_BYTES hold the counters and split-sum words: every call
 * leaves them zero again (the kernel re-arms them) and nothing else is ever stored
 * there, so one zero fill per allocation suffices even when the workspace is shared
 * by calls on different problems.  A workspace must not be shared by calls that
 * run concurrently.
 */
size_t lutgemm_workspace_size(const lutgemm_problem_t *problem, int64_t M);

/*
 * Offline weight packing (Section 3.1.2, Eq. 2 and Eq. 6; Section 3.1 bit-serial
 * planes).  Enqueues one kernel on `stream`.
 *   codes   device [N][K]: uint8 (UINT, BINARY) or int8 (TERNARY).  UINT codes are
 *           taken modulo 2^b, BINARY codes modulo 2; TERNARY values outside
 *           {-1,0,1} are clamped.
 *   scales  device: FP16 [N][K/group] (FP32 or FP16 [1] when group_size == 0)
 *   zeros   device FP16, same shape as scales, UINT only (NULL otherwise)
 *   packed  device, packed_bytes >= lutgemm_packed_weight_size(problem)
 * Each weight bit-plane is stored as 4-bit table indices: the pattern of 4
 * consecutive weights (the first weight is the MSB) with the low 3 bits inverted
 * when the MSB is set (Eq. 6); scale and zero are stored as given and
 * reinterpreted (s' = s/2, z' = 2z + 1 - 2^b, Eq. 2) in FP32 where they are used;
 * per column, a fixed-point exponent derived from its scales and zeros (the unit in
 * which lutgemm_mpgemm sums K splits exactly) is stored beside them.
 * TERNARY_3IN5: every 3 consecutive weights (padded with 0 past K) become a sign
 * bit and a 4-bit index into the triple table (5 bits per 3 weights).
 */
lutgemm_status_t lutgemm_pack_weights(const lutgemm_problem_t *problem, const void *codes,
                                      const void *scales, const void *zeros, void *packed,
                                      size_t packed_bytes, void *stream);

/*
 * Table precompute (Section 3.1.1 "independent operator"; Eq. 4-5): one kernel
 * that reads act [M][K] FP16 (device) and writes the table buffer described at
 * lutgemm_table_size.  For ACT_INT8 it first quantizes each token:
 * amax = max |a|, q_a = clamp(rint(a * (127 / amax)), -127, 127) in FP32
 * (q_a = 0 when amax == 0).  For ACT_FP16_LUT8 it quantizes each finished table
 * (Section 3.1.3).
 */
lutgemm_status_t lutgemm_precompute(const lutgemm_problem_t *problem, int64_t M, const void *act,
                                    void *tables, size_t table_bytes, void *stream);

/*
 * LUT mpGEMM (Section 3.1 bit-serial lookup with Eq. 3, 5-6; LMMA semantics
 * O = A x W^T + Acc, Section 3.3.1).
 *   tables     device, written by lutgemm_precompute (or the same layout; FP16 tables
 *              must hold entries of the normalized token, |x| < 1 as the layout
 *              defines, so |T| < 4: the single-token kernels sum K splits in fixed
 *              point with a unit derived from that bound, and larger entries give
 *              unspecified results there)
 *   packed     device, written by lutgemm_pack_weights
 *   out        device [M][N] row-major, of out_dtype; read first when accumulate != 0
 *   out_dtype  LUTGEMM_OUT_FP16 / FP32; LUTGEMM_OUT_INT32 for ACT_INT8 only
 *   accumulate 0: O = A W^T;  1: O = O + A W^T (INT32: exact integer add;
 *              FP: one FP32 add of the finished product, then the conversion)
 *   workspace  device, workspace_bytes >= lutgemm_workspace_size(problem, M);
 *              may be NULL when that size is 0
 * FP path: O = t_m sum_q s'_q (sum_b 2^b sum_j L_{b,j} - z'_q S_q), FP32.
 * INT8 path: acc = sum_k q_a w exactly; O = acc (INT32) or (float(acc) s_a) s_w.
 * TERNARY_3IN5: O = t_m s (sum_j L_j) (FP path, FP32) with one lookup per triple.
 * The result is bitwise reproducible run to run.
 */
lutgemm_status_t lutgemm_mpgemm(const lutgemm_problem_t *problem, int64_t M, const void *tables,
                                const void *packed, void *out, int32_t out_dtype,
                                int32_t accumulate, void *workspace, size_t workspace_bytes,
                                void *stream);

/* Size of the static scratch array behind lutgemm_mpgemm_noalloc, per GPU. */
#define LUTGEMM_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)

/*
 * lutgemm_mpgemm without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation).  Same arguments, kernels and results as lutgemm_mpgemm; the
 * K-split partial sums go to a static device array of
 * LUTGEMM_NOALLOC_SCRATCH_BYTES per GPU that the library holds until the process
 * ends (its address is looked up on the first call with each device current; it
 * is zero when the library is loaded and every call leaves it zeroed).
 * Calls needing more scratch than that (lutgemm_workspace_size) return
 * LUTGEMM_ERROR_NOT_SUPPORTED and launch nothing, with the sizes in
 * lutgemm_last_error().  No call allocates or frees memory.  All calls on one GPU
 * share its array: calls that overlap on one GPU (other streams, other threads)
 * race on it and must be serialized by the caller.
 */
lutgemm_status_t lutgemm_mpgemm_noalloc(const lutgemm_problem_t *problem, int64_t M, const void *tables,
                                        const void *packed, void *out, int32_t out_dtype,
                                        int32_t accumulate, void *stream);

/*
 * Bytes of scratch memory lutgemm_mpgemm_fused needs for M tokens; may be 0.  As
 * for lutgemm_workspace_size: zero-filled before its first use, left zero-filled by
 * every call, not shared by calls that run concurrently.
 */
size_t lutgemm_fused_workspace_size(const lutgemm_problem_t *problem, int64_t M);

/*
 * Table precompute fused into the LUT mpGEMM (Section 3.1.1 splits the
 * precompute out of the lookup so that it can be fused; this fuses it on the
 * consumer side): O = A x W^T (+ O) from act [M][K] FP16 (device) and the packed
 * weights.  Single tokens (M <= 2): every workgroup builds the tables of its K
 * range in LDS from the activations -- with the weights the whole-K lookup kernel
 * takes (at most a few MB) the same activation quantization (ACT_INT8) or
 * power-of-two token scaling (ACT_FP16) and the same FP16 / INT16 table entries as
 * lutgemm_precompute + lutgemm_mpgemm, one kernel; with larger weights and
 * ACT_FP16 the split-K kernel, whose tables are exact FP32 sums of the
 * activations as given (no token scaling, no FP16 rounding of entries), plus the
 * split sum; with larger weights and ACT_INT8 the same kernel, each workgroup
 * reading the whole token for the absmax and building the exact INT16 entries of
 * the precompute's quantization for its K range.  Several tokens (2 < M <= 64) with ACT_FP16 on layers of at most
 * 64 x 256 columns: the multi-token kernel reads the FP16 activations of its
 * tokens and K range, scales each token by the power of two 2^-e with e from its
 * absmax over that K range, and builds the same FP16 entries as
 * lutgemm_precompute (tuning key LUTGEMM_TUNE_MT_FUSED forces it on or off; every
 * column tile repeats the build, so beyond those sizes precompute + mpGEMM is
 * faster).  TERNARY_3IN5: one kernel for every M, tables built per workgroup for
 * its token.  Otherwise (larger M or N with ACT_FP16, ACT_INT8 with M > 2,
 * ACT_FP16_LUT8) it runs lutgemm_precompute into the workspace followed by
 * lutgemm_mpgemm: with several tokens every workgroup would have to read all of its
 * tokens for the INT8 quantizer's absmax.
 *   act        device FP16 [M][K]
 *   packed, out, out_dtype, accumulate   as for lutgemm_mpgemm
 *   workspace  device, workspace_bytes >= lutgemm_fused_workspace_size(problem, M);
 *              may be NULL when that size is 0
 * INT8 activations: results are bitwise those of lutgemm_precompute +
 * lutgemm_mpgemm.  FP16 activations: the zero-point term is summed per 128-block
 * instead of per quantization group, and the split-K kernel's entries are not
 * rounded to FP16, so results agree with the two-call path to within that
 * rounding (TERNARY_3IN5, and the multi-token kernel on weights without zero
 * points: bitwise, unless an entry or partial sum is subnormal).  Bitwise
 * reproducible run to run.
 */
lutgemm_status_t lutgemm_mpgemm_fused(const lutgemm_problem_t *problem, int64_t M, const void *act,
                                      const void *packed, void *out, int32_t out_dtype,
                                      int32_t accumulate, void *workspace, size_t workspace_bytes,
                                      void *stream);

/*
 * Comparison path (Section 2.2, dequantization-based mpGEMM): rebuilds FP16
 * weights s (q - z) from the same packed buffer and multiplies them with FP16
 * activations act [M][K] on the matrix cores (FP32 accumulation).  ACT_FP16 and
 * ACT_FP16_LUT8 problems (the activations are used as they are), not
 * TERNARY_3IN5 (LUTGEMM_ERROR_NOT_SUPPORTED); out_dtype FP16 or FP32; accumulate
 * as for lutgemm_mpgemm.
 *   workspace  device, 16-byte aligned, workspace_bytes >=
 *              lutgemm_dequant_workspace_size(problem, M); may be NULL when that is 0
 * With a K split the partial sums are added in split order by a second kernel, so
 * results are bitwise reproducible run to run.
 */
lutgemm_status_t lutgemm_mpgemm_dequant(const lutgemm_problem_t *problem, int64_t M,
                                        const void *act, const void *packed, void *out,
                                        int32_t out_dtype, int32_t accumulate, void *workspace,
                                        size_t workspace_bytes, void *stream);

/*
 * Bytes of scratch memory lutgemm_mpgemm_dequant needs for M tokens: FP32 partial
 * sums [splits][M][N_pad] when its kernel splits K across workgroups (small grids),
 * else 0 (also for problems the comparison path does not support).  Any contents
 * on entry; not shared by calls that run concurrently.
 */
size_t lutgemm_dequant_workspace_size(const lutgemm_problem_t *problem, int64_t M);

/*
 * The launch plan lutgemm_mpgemm_dequant uses for M tokens (host only, launches
 * nothing): *kernel = 0 for 128 x 128 tiles, 1 for the pipelined 256 x 256 tiles, 2
 * for 16-token slabs (1-bit weights); *splits = K ranges (1: no split).  Errors as
 * for lutgemm_mpgemm_dequant.
 */
lutgemm_status_t lutgemm_dequant_plan(const lutgemm_problem_t *problem, int64_t M, int32_t *kernel,
                                      int32_t *splits);

/*
 * Overrides of the launch planner, for tests and experiments only (normal use needs
 * none).  Each key holds one integer, set when the library is loaded from the
 * environment variable named beside it (if that is set) or else to its default;
 * no entry point reads the environment after that.  Setting -1 restores the
 * default.  The values are process-wide and apply to calls made after the setter
 * returns; changing them while other threads call the library gives those calls
 * either the old or the new value.  Kernel choices forced this way must still
 * suit the problem (the planner clamps splits and block counts to the problem).
 */
enum {
    LUTGEMM_TUNE_TARGET_BLOCKS = 0, /* LUTGEMM_TARGET_BLOCKS: workgroups a launch aims for (256)      */
    LUTGEMM_TUNE_WHOLEK_MAX_KB = 1, /* LUTGEMM_WHOLEK_MAX_KB: largest packed weights, in kB, that the
                                       single-token whole-K kernel takes (10000)                     */
    LUTGEMM_TUNE_GEMV_KIND = 2,     /* LUTGEMM_GEMV_KIND: kernel for M <= 2, 0 whole-K, 2 split-K,
                                       1 the multi-token kernel (default -1: planned)                */
    LUTGEMM_TUNE_GEMV_CFG = 3,      /* LUTGEMM_GEMV_CFG: lane decomposition of the whole-K kernel (-1) */
    LUTGEMM_TUNE_SPLITS = 4,        /* LUTGEMM_SPLITS: K splits of the whole-K kernel (0: planned)     */
    LUTGEMM_TUNE_KBS = 5,           /* LUTGEMM_KBS: 128-blocks per workgroup of the split-K kernel
                                       (0: planned)                                                  */
    LUTGEMM_TUNE_MT16 = 6,          /* LUTGEMM_MT16: 0 keeps 8-token tiles from M = 16 on (1)         */
    LUTGEMM_TUNE_MT_TARGET = 7,     /* LUTGEMM_MT_TARGET: multi-token grid target, in units of
                                       TARGET_BLOCKS (8)                                              */
    LUTGEMM_TUNE_MT_SPLITS = 8,     /* LUTGEMM_MT_SPLITS: K splits of the multi-token kernel
                                       (0: planned)                                                  */
    LUTGEMM_TUNE_MT_ORDER = 9,      /* LUTGEMM_MT_ORDER: multi-token workgroup order (-1: planned)    */
    LUTGEMM_TUNE_DEQUANT_KIND = 10, /* LUTGEMM_DEQUANT_KIND: comparison kernel, 0 128x128 tiles,
                                       1 pipelined 256x256 tiles, 2 16-token slabs (1-bit weights
                                       with one scale per column or tensor only; ignored for
                                       others) (-1: planned)                                         */
    LUTGEMM_TUNE_LOG = 11,          /* LUTGEMM_LOG: 1 prints each launch plan to stderr (0)           */
    LUTGEMM_TUNE_SPLIT_PRE = 12,    /* LUTGEMM_SPLIT_PRE: weight words per lane the split-K kernel
                                       requests before its tables arrive, 0, 2, 4 or 8 = all
                                       (-1: half of the lane's words)                              */
    LUTGEMM_TUNE_DEQUANT_SPLITS = 13, /* LUTGEMM_DEQUANT_SPLITS: K splits of the comparison kernel
                                       (0: planned)                                                  */
    LUTGEMM_TUNE_MT_FUSED = 14,     /* LUTGEMM_MT_FUSED: lutgemm_mpgemm_fused with FP16 activations and
                                       M > 2: 1 builds the tables inside the multi-token kernel, 0
                                       runs precompute + mpGEMM (-1: planned, the former for
                                       M <= 64 on layers of at most 64 x 256 columns)              */
    LUTGEMM_TUNE_MT4 = 15,          /* LUTGEMM_MT4: 0 keeps 8-token tiles for M <= 4 (1: 4-token
                                       tiles)                                                        */
    LUTGEMM_TUNE_SPLIT_EXACT = 16,  /* LUTGEMM_SPLIT_EXACT: 1 completes the single-token K split by one
                                       64-bit atomic per output where every split's partial sum is an
                                       integer (INT8 activations, or FP16 activations on weights with
                                       one scale per column or tensor); 0 always sums FP32 partials
                                       in split order (1)                                            */
    LUTGEMM_TUNE_COUNT = 17
};

/* Sets planner override `key` (LUTGEMM_TUNE_*) to `value` (-1: its default).
 * LUTGEMM_ERROR_INVALID_VALUE for an unknown key or a value outside [-1, 2^24]
 * (TARGET_BLOCKS: 0 is rejected too). */
lutgemm_status_t lutgemm_set_tuning(int32_t key, int32_t value);

/* Current value of planner override `key`; -2 for an unknown key. */
int32_t lutgemm_get_tuning(int32_t key);

/*
 * Measurement utility (not part of the method): reads `bytes` (rounded down to a
 * multiple of 16) of device memory at `src` with 128-bit loads from `blocks`
 * workgroups of 256 lanes and writes one 32-bit word per workgroup to `sink`
 * (device, >= 4 * blocks bytes).  Timing it on the byte counts of an mpGEMM call
 * gives the achievable streaming-read bandwidth the LUT kernels are compared with.
 * Returns LUTGEMM_ERROR_INVALID_VALUE for null or misaligned pointers, bytes < 16
 * or blocks outside [1, 65536].
 */
lutgemm_status_t lutgemm_calibrate_stream_read(const void *src, size_t bytes, void *sink,
                                               int32_t blocks, void *stream);

/*
 * The same measurement with the read pattern chosen by the caller, to search for
 * the fastest single-launch read of a byte count: each of the `blocks` x 256
 * lanes keeps `unroll` (1, 2, 4, 8 or 16) 16-byte loads in flight; flags bit 0
 * marks the loads nontemporal, bit 1 gives each workgroup one contiguous range
 * (else tiles of 256 x unroll words are dealt to the workgroups in turn).
 * lutgemm_calibrate_stream_read is unroll 4, flags 0.  Returns
 * LUTGEMM_ERROR_INVALID_VALUE as above and for any other unroll or flags value.
 */
lutgemm_status_t lutgemm_calibrate_stream_read_ex(const void *src, size_t bytes, void *sink,
                                                  int32_t blocks, int32_t unroll, int32_t flags,
                                                  void *stream);

#ifdef __cplusplus
}
#endif

#endif /* LUTGEMM_H */
