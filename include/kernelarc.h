/*
 * kernelarc.h -- C ABI of the MI355X (gfx950) BF16 linear-plus-residual library.
 *
 * The operation is the attention output projection with residual addition of
 * the KernelArc paper (Sec. "L1-030: attention output projection with
 * residual" and Alg. 3): the destination aliases the residual and the
 * library computes O <- W^T A + O with alpha = beta = 1, written there in
 * column-major cuBLASLt notation.  In the row-major, nn.Linear reading used
 * here (W stored [out, in] = [N, K]):
 *
 *     Y[i,j] = bf16( sum_k X[i,k] * W[j,k]  +  R[i,j] )
 *
 * with every product and partial sum in fp32 and a single round-to-nearest-
 * even conversion of the fp32 result (accumulator plus residual) to bf16.
 * The order in which the k-terms are summed is not part of the contract;
 * it is fixed per plan, so one plan gives bitwise-identical results for
 * identical inputs (no floating-point atomics anywhere).
 *
 * Types and layout (all entry points):
 *   - X, W, R, Y are device pointers on the calling thread's current HIP
 *     device, holding bf16 values as raw 16-bit patterns;
 *   - X is [M,K], W is [N,K], R and Y are [M,N]; all dense row-major with no
 *     padding (leading dimensions K, K, N, N);
 *   - the caller owns every buffer; the library never allocates, frees or
 *     retains them.  Internal state is limited to a per-device property
 *     cache, a per-thread cache of plan choices, and a per-device split-K
 *     workspace (64 MiB of fp32 partials and 64 Ki arrival counters) that
 *     the first call needing it allocates and keeps until the process ends.
 *
 * Execution: calls enqueue work on `stream` and return without synchronising
 * the stream or the device; a fault in a kernel surfaces at the caller's next
 * synchronisation.  The call that allocates the split-K workspace (the first
 * one on a device whose plan splits K) clears its counters with a kernel on
 * `stream`; under stream capture that call cannot allocate and returns
 * KERNELARC_ERR_UNSUPPORTED instead, so make one such call before capturing.
 * Calls on one stream are ordered; the split-K workspace of a device is
 * shared, so calls that may run concurrently on different streams of the
 * same device must not both pick a split-K plan
 * (kernelarc_plan_uses_workspace).
 *
 * Errors: every entry point returns a status (KERNELARC_OK on success) and
 * never throws, aborts or prints.  kernelarc_last_error() gives a detail
 * string for the calling thread's most recent failure.
 */
#ifndef KERNELARC_H
#define KERNELARC_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum kernelarc_status {
    KERNELARC_OK = 0,
    KERNELARC_ERR_INVALID_ARG = 1, /* negative size, NULL operand, bad overlap, size limit  */
    KERNELARC_ERR_UNSUPPORTED = 2, /* no gfx950 device, or a forced plan that cannot run it */
    KERNELARC_ERR_LAUNCH = 3,      /* the HIP runtime refused a launch or an allocation     */
};

/*
 * Y = X W^T + R  (Alg. 3: O <- W^T A + O, alpha = beta = 1; the destination
 * may alias the residual).
 *
 * M: rows of X, R, Y (the flattened token count); N: rows of W, columns of R
 * and Y; K: columns of X and W.  M, N, K >= 0 and each below 2^31.
 * Y == R (the same address) computes in place.  Any other overlap of Y's
 * byte range with X, W or R is rejected with KERNELARC_ERR_INVALID_ARG.
 * M == 0 or N == 0: nothing to do, returns KERNELARC_OK without a launch.
 * K == 0: Y = R.
 * Pointers that are 16-byte aligned with K a multiple of 8 take the MFMA
 * kernels; anything else takes a slower generic kernel with the same result
 * contract.
 */
int kernelarc_gemm_bf16_residual(int64_t M, int64_t N, int64_t K,
                                 const void *X, const void *W, const void *R,
                                 void *Y, hipStream_t stream);

/*
 * Y = X W^T  (the same operation without a residual; the plain BF16 GEMM of
 * the paper's Sec. "Guided Sequential GEMM Boundary Study").  Arguments and
 * errors as above; K == 0 gives Y = +0.
 */
int kernelarc_gemm_bf16(int64_t M, int64_t N, int64_t K,
                        const void *X, const void *W, void *Y, hipStream_t stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops that must not call hipMalloc, harnesses that forbid
 * it): kernelarc_gemm_bf16_residual with the same plans, kernels and result
 * (bit for bit), except that R == NULL computes the plain product Y = X W^T
 * and that the split-K partials go to a static scratch area compiled into
 * the library instead of the allocated per-device workspace.  The call
 * allocates nothing (no hipMalloc, no allocating library routine) and never
 * synchronises.
 *
 * The scratch holds at most 16 Mi fp32 partials (64 MiB) and 64 Ki arrival
 * counters per device; each device the library runs on keeps its copy until
 * the process ends.  A plan needing more is rejected with
 * KERNELARC_ERR_UNSUPPORTED (the plan choice never picks such a split, so
 * this does not happen for shapes the library accepts).  The first call on a
 * device clears the counters with a kernel on `stream`; the kernels leave
 * them at zero.  Every call on one device shares that device's scratch and
 * its contents persist between calls: calls that may overlap in time on one
 * device (different streams, concurrently replayed graphs) race on it and
 * must be serialised by the caller.  Arguments and other errors as
 * kernelarc_gemm_bf16_residual.
 */
int kernelarc_gemm_bf16_residual_noalloc(int64_t M, int64_t N, int64_t K,
                                         const void *X, const void *W, const void *R,
                                         void *Y, hipStream_t stream);

/*
 * Plan introspection and forced-plan execution (for tests, the benchmark
 * and offline tuning; Alg. 3's per-M plan cache, static validated table and
 * heuristic fallback correspond to kernelarc_select_plan).
 *
 * A plan is one kernel variant (tile shape, staging depth, split-K rule).
 * Plan ids run from 0 to kernelarc_plan_count() - 1.  None of these touch
 * the GPU.
 */
int kernelarc_plan_count(void);

/*
 * Name of the plan the library runs for this shape (Alg. 3's per-M plan
 * choice) when the pointers are 16-byte aligned: written NUL-terminated into
 * buf, which holds len bytes.  Returns KERNELARC_OK; KERNELARC_ERR_INVALID_ARG
 * for negative sizes, buf == NULL, or len too small for the name (then
 * nothing is written).  Plan names are shorter than 64 bytes.  Does not touch
 * the GPU.
 */
int kernelarc_plan_name(int64_t M, int64_t N, int64_t K, int residual, char *buf, size_t len);

/* Static, NUL-terminated name of plan id `plan`, or NULL for an unknown id. */
const char *kernelarc_plan_label(int plan);

/*
 * 1 if `plan` can compute this shape (size limits and the K % 8 rule of the
 * MFMA plans; pointer alignment is checked at call time), 0 if not, and -1
 * for an unknown plan or negative sizes.
 */
int kernelarc_plan_supports(int plan, int64_t M, int64_t N, int64_t K, int residual);

/*
 * The plan the library runs for this shape when the pointers are 16-byte
 * aligned, or -1 for negative sizes.  Depends on the shape only, never on
 * data.
 */
int kernelarc_select_plan(int64_t M, int64_t N, int64_t K, int residual);

/* 1 if `plan` on this shape uses the per-device split-K workspace, else 0. */
int kernelarc_plan_uses_workspace(int plan, int64_t M, int64_t N, int64_t K);

/*
 * Y = X W^T (+ R if R != NULL) computed with the given plan.  Returns
 * KERNELARC_ERR_UNSUPPORTED if the plan cannot compute this shape or these
 * pointers' alignment, otherwise as kernelarc_gemm_bf16_residual.
 */
int kernelarc_gemm_bf16_with_plan(int plan, int64_t M, int64_t N, int64_t K,
                                  const void *X, const void *W, const void *R,
                                  void *Y, hipStream_t stream);

/*
 * General form: the library epilogue of the paper's GEMM sites (cuBLASLt's
 * D = alpha W^T A + beta C, Alg. 3 and the decoder-layer case study, whose
 * two residual GEMMs are this operator with K = hidden or K = intermediate
 * size), in the same row-major reading, with a bias row and leading
 * dimensions:
 *
 *     Y[i,j] = bf16( alpha * sum_k X[i*ldx+k] W[j*ldw+k]
 *                    + beta * C[i*ldc+j] + bias[j] )
 *
 * fp32 accumulation; alpha * acc, then + beta * C as one fused multiply-add,
 * then + bias, in fp32; one round-to-nearest-even to bf16.  With
 * alpha = beta = 1, bias == NULL and dense leading dimensions the result is
 * bit-identical to kernelarc_gemm_bf16_residual (C != NULL) or
 * kernelarc_gemm_bf16 (C == NULL).
 *
 * ldx, ldw, ldc, ldy: row strides in elements (ldx, ldw >= K; ldc, ldy >= N;
 * each below 2^31).  C may be NULL (no C term); when beta == 0, C is not
 * read at all.  bias is N bf16 values or NULL.  Y may equal C when
 * ldy == ldc (in place); any other overlap of Y's rows with X, W, C or the
 * bias is rejected with KERNELARC_ERR_INVALID_ARG.  Pointers 16-byte aligned
 * with K, ldx and ldw multiples of 8 take the MFMA and GEMV kernels (16-byte
 * R/Y accesses also need ldc and ldy multiples of 8, otherwise 2-byte ones);
 * anything else takes the generic kernel.
 */
int kernelarc_gemm_bf16_ex(int64_t M, int64_t N, int64_t K, float alpha,
                           const void *X, int64_t ldx, const void *W, int64_t ldw,
                           float beta, const void *C, int64_t ldc, const void *bias,
                           void *Y, int64_t ldy, hipStream_t stream);

/* The general form with a forced plan (KERNELARC_ERR_UNSUPPORTED if the plan
 * cannot compute it). */
int kernelarc_gemm_bf16_ex_with_plan(int plan, int64_t M, int64_t N, int64_t K, float alpha,
                                     const void *X, int64_t ldx, const void *W, int64_t ldw,
                                     float beta, const void *C, int64_t ldc, const void *bias,
                                     void *Y, int64_t ldy, hipStream_t stream);

/* The plan kernelarc_gemm_bf16_ex runs for these sizes, strides and scalars
 * when the pointers are suitably aligned; -1 for negative sizes. */
int kernelarc_select_plan_ex(int64_t M, int64_t N, int64_t K, int has_c, int64_t ldx, int64_t ldw,
                             int64_t ldc, int64_t ldy, float alpha, float beta, int has_bias);

/*
 * Gated MLP input projection with the SiLU-multiply (SwiGLU): the decoder
 * layer's gate and up projections and the activation that joins them
 * (decoder-layer case study, Alg. 7: BF16 gate/up projections followed by a
 * SiLU-multiply, and the fused gate/up GEMM with a SwiGLU epilogue), in one
 * kernel:
 *
 *     H[i,j] = bf16( silu(G[i,j]) * U[i,j] ),   silu(z) = z / (1 + e^-z),
 *     G = X Wg^T,  U = X Wu^T
 *
 * X is [M,K] (the normalised hidden states), Wg and Wu are [N,K] (gate and
 * up weights, nn.Linear orientation, N = intermediate size), H is [M,N];
 * all dense row-major bf16 device buffers owned by the caller.  G and U are
 * accumulated in fp32 and never rounded to bf16; SiLU and the product are
 * evaluated in fp32 (SiLU within a few fp32 ulps) and rounded once to bf16,
 * nearest-even.  A merged [2N,K] gate_up weight is passed as Wg = W and
 * Wu = W + N*K.  Wg and Wu may overlap each other (they are only read); H
 * overlapping X, Wg or Wu is rejected with KERNELARC_ERR_INVALID_ARG.
 * M, K >= 0 and below 2^31, 0 <= N < 2^30.  M == 0 or N == 0: no launch.
 * K == 0: H = 0.  16-byte aligned pointers with K a multiple of 8 take the
 * MFMA tile kernels; anything else takes a generic kernel with the same
 * contract.  Non-finite sums propagate as the formula does in IEEE
 * arithmetic (silu(-inf) is NaN).
 */
int kernelarc_swiglu_bf16(int64_t M, int64_t N, int64_t K, const void *X,
                          const void *Wg, const void *Wu, void *H, hipStream_t stream);

/* SwiGLU with a forced plan (KERNELARC_ERR_UNSUPPORTED if the plan cannot
 * compute it: only tile plans whose waves hold gate/up block pairs, and the
 * generic plan). */
int kernelarc_swiglu_bf16_with_plan(int plan, int64_t M, int64_t N, int64_t K, const void *X,
                                    const void *Wg, const void *Wu, void *H, hipStream_t stream);

/* The plan kernelarc_swiglu_bf16 runs for these sizes with aligned
 * pointers; -1 for negative sizes. */
int kernelarc_select_plan_swiglu(int64_t M, int64_t N, int64_t K);

/* 1 if `plan` can compute SwiGLU at these sizes, 0 if not, -1 for an unknown
 * plan or negative sizes. */
int kernelarc_plan_supports_swiglu(int plan, int64_t M, int64_t N, int64_t K);

/*
 * INT8 linear layer with a dequantisation epilogue (W8A8), and the INT8
 * SwiGLU gate/up projection of the decoder-layer case study (Alg. 7: its
 * INT8 path computes the gate/up GEMM with a fused dequantisation and SwiGLU
 * epilogue).  Symmetric quantisation with one binary32 scale per row of the
 * activations (token) and one per output channel, no zero points:
 *
 *     A[i,j] = sum_k qX[i,k] qW[j,k]               (exact, int32)
 *     Y[i,j] = bf16( sx[i] * sw[j] * A[i,j]  (+ R[i,j]) )
 *     H[i,j] = bf16( silu(sx[i] swg[j] Ag[i,j]) * (sx[i] swu[j] Au[i,j]) )
 *
 * qX is [M,K], qW, qWg, qWu are [N,K] int8 (nn.Linear orientation), sx is
 * [M] and sw, swg, swu are [N] floats; R (optional, NULL for none) and Y, H
 * are [M,N] bf16; all dense row-major device buffers owned by the caller.
 * The integer sums are exact (K <= 65536 keeps them in int32; a larger K is
 * rejected with KERNELARC_ERR_INVALID_ARG); A is converted to fp32 and
 * multiplied by sx[i] * sw[j] (formed in fp32); the residual is added in
 * fp32; one round-to-nearest-even to bf16.  Y may equal R (in place); any
 * other overlap of the output with an operand or a scale vector is
 * rejected.  Scale vectors must be 4-byte aligned.  M == 0 or N == 0: no
 * launch.  16-byte aligned int8 operands with K a multiple of 16 take the
 * MFMA tile kernels (v_mfma_i32_32x32x32_i8); anything else a generic kernel
 * with the same contract.
 */
int kernelarc_gemm_i8(int64_t M, int64_t N, int64_t K, const void *qX, const float *sx,
                      const void *qW, const float *sw, const void *R, void *Y, hipStream_t stream);

/* The INT8 GEMM with a forced plan (KERNELARC_ERR_UNSUPPORTED if the plan
 * cannot compute it: only tile plans and the generic plan can). */
int kernelarc_gemm_i8_with_plan(int plan, int64_t M, int64_t N, int64_t K, const void *qX,
                                const float *sx, const void *qW, const float *sw, const void *R,
                                void *Y, hipStream_t stream);

/* INT8 SwiGLU (see above): 0 <= N < 2^30. */
int kernelarc_swiglu_i8(int64_t M, int64_t N, int64_t K, const void *qX, const float *sx,
                        const void *qWg, const float *swg, const void *qWu, const float *swu,
                        void *H, hipStream_t stream);

/* INT8 SwiGLU with a forced plan (tile plans that pair gate and up blocks,
 * and the generic plan). */
int kernelarc_swiglu_i8_with_plan(int plan, int64_t M, int64_t N, int64_t K, const void *qX,
                                  const float *sx, const void *qWg, const float *swg,
                                  const void *qWu, const float *swu, void *H, hipStream_t stream);

/* The plan the INT8 GEMM (swiglu == 0) or INT8 SwiGLU (swiglu != 0) runs for
 * these sizes with aligned operands; -1 for negative sizes. */
int kernelarc_select_plan_i8(int64_t M, int64_t N, int64_t K, int swiglu);

/* 1 if `plan` can compute the INT8 GEMM / SwiGLU at these sizes, 0 if not,
 * -1 for an unknown plan or negative sizes. */
int kernelarc_plan_supports_i8(int plan, int64_t M, int64_t N, int64_t K, int swiglu);

/*
 * FP8 forms: the INT8 entry points above with OCP FP8 E4M3 operands (the
 * "FN" variant: bias 7, no infinities, S.1111.111 is NaN, largest finite
 * 448) in place of int8, the same per-row and per-column float scales,
 * layout, residual, aliasing and error rules:
 *
 *     Y[i,j] = bf16( sx[i] * sw[j] * S[i,j]  (+ R[i,j]) ),  S = sum_k x8(qX[i,k]) x8(qW[j,k])
 *     H[i,j] = bf16( silu(sx[i] swg[j] Sg[i,j]) * (sx[i] swu[j] Su[i,j]) )
 *
 * The products of decoded values are exact in fp32 and S is accumulated in
 * fp32 (the summation order is not part of the contract); K has no limit
 * beyond 2^31.  qX, qW, qWg, qWu hold E4M3 bit patterns (one byte each).
 * 16-byte aligned operands with K a multiple of 16 take the MFMA tile
 * kernels (v_mfma_scale_f32_32x32x64_f8f6f4 with unit scales, twice the
 * bf16 rate); anything else a generic kernel with the same contract.
 */
int kernelarc_gemm_f8(int64_t M, int64_t N, int64_t K, const void *qX, const float *sx,
                      const void *qW, const float *sw, const void *R, void *Y, hipStream_t stream);

int kernelarc_gemm_f8_with_plan(int plan, int64_t M, int64_t N, int64_t K, const void *qX,
                                const float *sx, const void *qW, const float *sw, const void *R,
                                void *Y, hipStream_t stream);

int kernelarc_swiglu_f8(int64_t M, int64_t N, int64_t K, const void *qX, const float *sx,
                        const void *qWg, const float *swg, const void *qWu, const float *swu,
                        void *H, hipStream_t stream);

int kernelarc_swiglu_f8_with_plan(int plan, int64_t M, int64_t N, int64_t K, const void *qX,
                                  const float *sx, const void *qWg, const float *swg,
                                  const void *qWu, const float *swu, void *H, hipStream_t stream);

/* Plan choice and plan capability of the FP8 forms (as for INT8). */
int kernelarc_select_plan_f8(int64_t M, int64_t N, int64_t K, int swiglu);

int kernelarc_plan_supports_f8(int plan, int64_t M, int64_t N, int64_t K, int swiglu);

/*
 * Grouped (per-expert) linear layer and SwiGLU over an expert-major padded
 * layout: the mixture-of-experts case study (Alg. 4) places token-expert
 * pairs in expert-contiguous rows of a [G x M_pad] buffer (gap rows
 * zero-filled) and runs each projection as one strided-batched GEMM.  For
 * each group (expert) g and each valid row i < rows(g):
 *
 *     Y[g,i,j] = bf16( sum_k X[g,i,k] W[g,j,k] )                   (fp32 sums)
 *     H[g,i,j] = bf16( silu(X[g,i,:].Wg[g,j,:]) * (X[g,i,:].Wu[g,j,:]) )
 *
 * X is [G,M_pad,K], W, Wg, Wu are [G,N,K], Y, H are [G,M_pad,N]; dense
 * row-major bf16 device buffers owned by the caller.  counts is a device
 * array of G int32 valid-row counts, each clamped to [0, M_pad] (NULL: every
 * row of every group is valid); it is read by the kernels, so it may be
 * produced on the device just before the call (no host round trip).  Rows
 * at or past rows(g) -- the gap rows -- are neither read nor written.  The
 * arithmetic per row is that of kernelarc_gemm_bf16 / kernelarc_swiglu_bf16.
 * G * M_pad and K below 2^31 (N below 2^30 for SwiGLU); G, M_pad or N = 0:
 * no launch.  An output overlapping X, a weight or counts is rejected.
 * 16-byte aligned pointers with K a multiple of 8 take the MFMA tile kernels
 * (one launch over all groups; tiles wholly in gap rows exit at once);
 * anything else takes a generic kernel with the same contract.
 */
int kernelarc_gemm_bf16_grouped(int64_t G, int64_t M_pad, int64_t N, int64_t K, const void *X,
                                const void *W, const int32_t *counts, void *Y, hipStream_t stream);

int kernelarc_swiglu_bf16_grouped(int64_t G, int64_t M_pad, int64_t N, int64_t K, const void *X,
                                  const void *Wg, const void *Wu, const int32_t *counts, void *H,
                                  hipStream_t stream);

/* The grouped forms with a forced plan (tile plans without split-K, and the
 * generic plan; KERNELARC_ERR_UNSUPPORTED otherwise). */
int kernelarc_gemm_bf16_grouped_with_plan(int plan, int64_t G, int64_t M_pad, int64_t N, int64_t K,
                                          const void *X, const void *W, const int32_t *counts,
                                          void *Y, hipStream_t stream);

int kernelarc_swiglu_bf16_grouped_with_plan(int plan, int64_t G, int64_t M_pad, int64_t N, int64_t K,
                                            const void *X, const void *Wg, const void *Wu,
                                            const int32_t *counts, void *H, hipStream_t stream);

/* The plan the grouped GEMM (swiglu == 0) or grouped SwiGLU runs for these
 * sizes with aligned pointers; -1 for negative sizes. */
int kernelarc_select_plan_grouped(int64_t G, int64_t M_pad, int64_t N, int64_t K, int swiglu);

/* 1 if `plan` can compute the grouped form at these sizes, 0 if not, -1 for
 * an unknown plan or negative sizes. */
int kernelarc_plan_supports_grouped(int plan, int64_t G, int64_t M_pad, int64_t N, int64_t K,
                                    int swiglu);

/* Static description of a status code. */
const char *kernelarc_status_string(int status);

/* Detail of the calling thread's most recent failed call ("" if none). */
const char *kernelarc_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* KERNELARC_H */
