/*
 * Plain CPU oracle for the fused linear-plus-residual operator
 *
 *     Y[i,j] = sum_k X[i,k] * W[j,k]  +  R[i,j]          (R optional)
 *
 * its general form (alpha, beta, bias, leading dimensions), the gated
 * MLP input projection H = silu(X Wg^T) * (X Wu^T) (SwiGLU), and INT8
 * versions of the linear layer and of SwiGLU with per-row and per-column
 * dequantisation scales, FP8 (E4M3) versions with the same scales, and
 * grouped (per-expert) forms of the linear layer and of SwiGLU over an
 * expert-major padded layout.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously correct
 * reference that the GPU library is checked against.  Only the test suite,
 * the smoke check and the CPU-baseline leg of the benchmark load it; the
 * product library never links, calls or falls back to it, and it shares no
 * code, header, table or helper with the HIP sources.
 *
 * What it follows (KernelArc paper):
 *   - Sec. "L1-030: attention output projection with residual" and Alg. 3:
 *     the destination aliases the residual and the library computes
 *     O <- W^T A + O with alpha = beta = 1 (cuBLASLt column-major notation).
 *     Read in row-major, nn.Linear orientation (W stored [out, in] = [N, K]),
 *     that is Y = X W^T + R.
 *   - Sec. "Guided Sequential GEMM Boundary Study": BF16 operands.
 *   - The inputs are bf16 bit patterns; every value is widened exactly to
 *     double, every product of two bf16 values is exact in double, and the
 *     k-sum runs in ascending k in double (no reassociation: build with
 *     -O2 -ffp-contract=off and without -ffast-math).  The result is returned
 *     in double and is NOT rounded to bf16.
 *
 * Pins: tests/test_oracle_pins.py (exact rational brute force, a hand-worked
 * fixture, numpy's float64 matmul, W = 0, W = I, rank-1 integer closed form,
 * row/K permutation and transpose invariants, and planted-mistake runs; for
 * SwiGLU, brute force with a high-precision decimal exponential, scipy's
 * logistic function, closed forms at e, the odd and even parts of SiLU,
 * saturated tails and zero operands).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* bf16 is the top half of an IEEE binary32: widen by a 16-bit left shift. */
static double bf16_bits_to_double(uint16_t bits)
{
    uint32_t u = (uint32_t)bits << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

/* One output element, straight from the definition. */
static double element(int64_t i, int64_t j, int64_t N, int64_t K,
                      const uint16_t *X, const uint16_t *W, const uint16_t *R)
{
    double acc = 0.0;
    for (int64_t k = 0; k < K; ++k)
        acc += bf16_bits_to_double(X[i * K + k]) * bf16_bits_to_double(W[j * K + k]);
    if (R)
        acc += bf16_bits_to_double(R[i * N + j]);
    return acc;
}

/*
 * Full output.  X is [M,K], W is [N,K], R is [M,N] or NULL, all row-major
 * bf16 bit patterns; Y is [M,N] doubles.  Returns 0, or -1 on a negative
 * dimension or a NULL buffer that is needed.
 */
int ka_oracle_linear(int64_t M, int64_t N, int64_t K,
                     const uint16_t *X, const uint16_t *W, const uint16_t *R,
                     double *Y)
{
    if (M < 0 || N < 0 || K < 0) return -1;
    if (M * N > 0 && !Y) return -1;
    if (M * K > 0 && !X) return -1;
    if (N * K > 0 && !W) return -1;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < M; ++i)
        for (int64_t j = 0; j < N; ++j)
            Y[i * N + j] = element(i, j, N, K, X, W, R);
    return 0;
}

/*
 * Both operators over the whole output from one evaluation of each k-sum:
 * Yp = the product alone (R absent) and Yr = the product plus R, element for
 * element the values ka_oracle_linear gives without and with R (the same
 * sum in the same order, then the same single addition of R).  Used where
 * the whole output of both forms is checked at sizes where two passes would
 * double the CPU time.  R is required.
 */
int ka_oracle_linear_pair(int64_t M, int64_t N, int64_t K,
                          const uint16_t *X, const uint16_t *W, const uint16_t *R,
                          double *Yp, double *Yr)
{
    if (M < 0 || N < 0 || K < 0) return -1;
    if (M * N > 0 && (!Yp || !Yr || !R)) return -1;
    if (M * K > 0 && !X) return -1;
    if (N * K > 0 && !W) return -1;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < M; ++i)
        for (int64_t j = 0; j < N; ++j) {
            const double acc = element(i, j, N, K, X, W, NULL);
            Yp[i * N + j] = acc;
            Yr[i * N + j] = acc + bf16_bits_to_double(R[i * N + j]);
        }
    return 0;
}

/*
 * The same definition evaluated only at the n listed positions
 * (rows[t], cols[t]); used for sampled checks at sizes where the full
 * product is too slow on the CPU.  Indices must lie in [0,M) x [0,N).
 */
int ka_oracle_linear_at(int64_t M, int64_t N, int64_t K,
                        const uint16_t *X, const uint16_t *W, const uint16_t *R,
                        int64_t n, const int64_t *rows, const int64_t *cols,
                        double *out)
{
    if (M < 0 || N < 0 || K < 0 || n < 0) return -1;
    for (int64_t t = 0; t < n; ++t)
        if (rows[t] < 0 || rows[t] >= M || cols[t] < 0 || cols[t] >= N) return -1;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t t = 0; t < n; ++t)
        out[t] = element(rows[t], cols[t], N, K, X, W, R);
    return 0;
}

/*
 * Round doubles to bf16 bit patterns, round-to-nearest, ties to even
 * (IEEE 754 roundTiesToEven applied to the bf16 format: 8 significant bits,
 * exponent range of binary32).  Written from the definition: the spacing of
 * bf16 values around |x| is a power of two, so x is scaled by that spacing,
 * rounded to the nearest integer (ties to even, the default rounding mode of
 * rint) and scaled back.  Results above the largest finite bf16 after
 * rounding become infinity; NaN becomes the quiet NaN 0x7FC0 with x's sign.
 */
void ka_oracle_round_bf16(int64_t n, const double *in, uint16_t *out)
{
    for (int64_t t = 0; t < n; ++t) {
        double x = in[t];
        uint16_t sign = signbit(x) ? 0x8000u : 0u;
        if (isnan(x)) { out[t] = (uint16_t)(sign | 0x7FC0u); continue; }
        double a = fabs(x);
        if (isinf(a)) { out[t] = (uint16_t)(sign | 0x7F80u); continue; }
        if (a == 0.0) { out[t] = sign; continue; }
        int e;
        frexp(a, &e);               /* a = f * 2^e, f in [0.5, 1) */
        int exp2 = e - 1;           /* a in [2^exp2, 2^(exp2+1)) */
        if (exp2 < -126) exp2 = -126; /* subnormal bf16: fixed spacing */
        double spacing = ldexp(1.0, exp2 - 7);
        double r = rint(a / spacing) * spacing;
        const double max_finite = ldexp(255.0, 120); /* (2 - 2^-7) * 2^127 */
        if (r > max_finite) { out[t] = (uint16_t)(sign | 0x7F80u); continue; }
        float rf = (float)r;        /* exact: r is a bf16 value */
        uint32_t u;
        memcpy(&u, &rf, sizeof u);
        out[t] = (uint16_t)(sign | (uint16_t)(u >> 16));
    }
}

/*
 * General form: the library epilogue the paper's GEMM sites invoke
 * (D = alpha * W^T A + beta * C in cuBLASLt's column-major notation, Alg. 3
 * and the decoder-layer case study, whose two residual GEMMs are this
 * operator with K = hidden size or K = intermediate size), read row-major
 * as for the plain operator, with a bias row and leading dimensions:
 *
 *     D[i,j] = alpha * sum_k X[i*ldx + k] W[j*ldw + k]
 *              + beta * C[i*ldc + j] + bias[j]
 *
 * alpha and beta are binary32 values (widened exactly); C and bias are bf16
 * bit patterns or NULL.  When beta == 0, C is not read (so it may be NULL or
 * hold non-finite values), as in BLAS; alpha always multiplies the product.
 * Evaluated in double: the k-sum ascending, then the alpha product, then
 * the C term, then the bias.  D is dense [M,N] doubles, not rounded.
 */
static double element_ex(int64_t i, int64_t j, int64_t K, double alpha,
                         const uint16_t *X, int64_t ldx, const uint16_t *W, int64_t ldw,
                         double beta, const uint16_t *C, int64_t ldc, const uint16_t *bias)
{
    double s = 0.0;
    for (int64_t k = 0; k < K; ++k)
        s += bf16_bits_to_double(X[i * ldx + k]) * bf16_bits_to_double(W[j * ldw + k]);
    double d = alpha * s;
    if (C && beta != 0.0)
        d += beta * bf16_bits_to_double(C[i * ldc + j]);
    if (bias)
        d += bf16_bits_to_double(bias[j]);
    return d;
}

static int check_ex(int64_t M, int64_t N, int64_t K, const uint16_t *X, int64_t ldx,
                    const uint16_t *W, int64_t ldw, float beta, const uint16_t *C, int64_t ldc)
{
    if (M < 0 || N < 0 || K < 0) return -1;
    if (M > 0 && K > 0 && (!X || ldx < K)) return -1;
    if (N > 0 && K > 0 && (!W || ldw < K)) return -1;
    if (M > 0 && N > 0 && beta != 0.0f && C && ldc < N) return -1;
    return 0;
}

int ka_oracle_linear_ex(int64_t M, int64_t N, int64_t K, float alpha,
                        const uint16_t *X, int64_t ldx, const uint16_t *W, int64_t ldw,
                        float beta, const uint16_t *C, int64_t ldc, const uint16_t *bias,
                        double *D)
{
    if (check_ex(M, N, K, X, ldx, W, ldw, beta, C, ldc) != 0) return -1;
    if (M * N > 0 && !D) return -1;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < M; ++i)
        for (int64_t j = 0; j < N; ++j)
            D[i * N + j] = element_ex(i, j, K, (double)alpha, X, ldx, W, ldw, (double)beta, C, ldc, bias);
    return 0;
}

/* The general form at the n positions (rows[t], cols[t]). */
int ka_oracle_linear_ex_at(int64_t M, int64_t N, int64_t K, float alpha,
                           const uint16_t *X, int64_t ldx, const uint16_t *W, int64_t ldw,
                           float beta, const uint16_t *C, int64_t ldc, const uint16_t *bias,
                           int64_t n, const int64_t *rows, const int64_t *cols, double *out)
{
    if (check_ex(M, N, K, X, ldx, W, ldw, beta, C, ldc) != 0 || n < 0) return -1;
    for (int64_t t = 0; t < n; ++t)
        if (rows[t] < 0 || rows[t] >= M || cols[t] < 0 || cols[t] >= N) return -1;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t t = 0; t < n; ++t)
        out[t] = element_ex(rows[t], cols[t], K, (double)alpha, X, ldx, W, ldw, (double)beta, C, ldc, bias);
    return 0;
}

/*
 * Gated MLP input projection with the SiLU-multiply (SwiGLU): the decoder
 * layer's gate and up projections and the activation that joins them
 * (decoder-layer case study, Alg. 7: its BF16 gate/up projections followed
 * by a SiLU-multiply, and its fused gate/up GEMM with a SwiGLU epilogue):
 *
 *     G[i,j] = sum_k X[i,k] Wg[j,k]        U[i,j] = sum_k X[i,k] Wu[j,k]
 *     H[i,j] = silu(G[i,j]) * U[i,j]       silu(z) = z / (1 + e^(-z))
 *
 * The paper names the operation without writing it out; SiLU is the
 * sigmoid-weighted linear unit z * sigmoid(z), and SwiGLU gates the up
 * projection with SiLU of the gate projection.  X is [M,K], Wg and Wu are
 * [N,K] (nn.Linear orientation, N = intermediate size), H is [M,N] doubles.
 * G and U are the k-sums in double (ascending k), never rounded to bf16:
 * the fused epilogue has no intermediate tensor.  H is not rounded.
 */
static double silu(double z)
{
    return z / (1.0 + exp(-z));
}

static double element_swiglu(int64_t i, int64_t j, int64_t K, const uint16_t *X,
                             const uint16_t *Wg, const uint16_t *Wu)
{
    double g = 0.0;
    double u = 0.0;
    for (int64_t k = 0; k < K; ++k) {
        double x = bf16_bits_to_double(X[i * K + k]);
        g += x * bf16_bits_to_double(Wg[j * K + k]);
        u += x * bf16_bits_to_double(Wu[j * K + k]);
    }
    return silu(g) * u;
}

static int check_swiglu(int64_t M, int64_t N, int64_t K, const uint16_t *X,
                        const uint16_t *Wg, const uint16_t *Wu)
{
    if (M < 0 || N < 0 || K < 0) return -1;
    if (M * K > 0 && !X) return -1;
    if (N * K > 0 && (!Wg || !Wu)) return -1;
    return 0;
}

int ka_oracle_swiglu(int64_t M, int64_t N, int64_t K, const uint16_t *X,
                     const uint16_t *Wg, const uint16_t *Wu, double *H)
{
    if (check_swiglu(M, N, K, X, Wg, Wu) != 0) return -1;
    if (M * N > 0 && !H) return -1;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < M; ++i)
        for (int64_t j = 0; j < N; ++j)
            H[i * N + j] = element_swiglu(i, j, K, X, Wg, Wu);
    return 0;
}

/* SwiGLU at the n positions (rows[t], cols[t]). */
int ka_oracle_swiglu_at(int64_t M, int64_t N, int64_t K, const uint16_t *X,
                        const uint16_t *Wg, const uint16_t *Wu, int64_t n,
                        const int64_t *rows, const int64_t *cols, double *out)
{
    if (check_swiglu(M, N, K, X, Wg, Wu) != 0 || n < 0) return -1;
    for (int64_t t = 0; t < n; ++t)
        if (rows[t] < 0 || rows[t] >= M || cols[t] < 0 || cols[t] >= N) return -1;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t t = 0; t < n; ++t)
        out[t] = element_swiglu(rows[t], cols[t], K, X, Wg, Wu);
    return 0;
}

/*
 * INT8 linear layer with a dequantisation epilogue, and the INT8 SwiGLU
 * gate/up projection (decoder-layer case study, Alg. 7: its INT8 path
 * quantises the normalised activations and the gate/up weights and computes
 * the gate/up GEMM with a fused dequantisation and SwiGLU epilogue, or an
 * integer GEMM followed by a separate dequantisation/SwiGLU step).  The
 * paper does not give the quantisation granularity; the reading here is the
 * symmetric W8A8 scheme: one scale per activation row (token) and one per
 * weight row (output channel), no zero points:
 *
 *     A[i,j] = sum_k qX[i,k] qW[j,k]                   (exact integer)
 *     Y[i,j] = sx[i] sw[j] A[i,j]  (+ R[i,j])
 *     H[i,j] = silu(sx[i] swg[j] Ag[i,j]) * (sx[i] swu[j] Au[i,j])
 *
 * qX is [M,K], qW, qWg, qWu are [N,K] int8; sx [M] and sw, swg, swu [N] are
 * binary32 scales; R is an optional bf16 [M,N] residual.  The integer sums
 * are exact (int64); the dequantised value is formed in double as
 * (sx * sw) * A (the scale product is exact in double), then + R; silu as
 * above.  Results are doubles, not rounded.
 */
static int64_t dot_i8(const int8_t *x, const int8_t *w, int64_t K)
{
    int64_t acc = 0;
    for (int64_t k = 0; k < K; ++k)
        acc += (int64_t)x[k] * (int64_t)w[k];
    return acc;
}

static double element_i8(int64_t i, int64_t j, int64_t N, int64_t K, const int8_t *qX,
                         const float *sx, const int8_t *qW, const float *sw, const uint16_t *R)
{
    double y = (double)sx[i] * (double)sw[j] * (double)dot_i8(qX + i * K, qW + j * K, K);
    if (R)
        y += bf16_bits_to_double(R[i * N + j]);
    return y;
}

static double element_i8_swiglu(int64_t i, int64_t j, int64_t K, const int8_t *qX, const float *sx,
                                const int8_t *qWg, const float *swg, const int8_t *qWu, const float *swu)
{
    double g = (double)sx[i] * (double)swg[j] * (double)dot_i8(qX + i * K, qWg + j * K, K);
    double u = (double)sx[i] * (double)swu[j] * (double)dot_i8(qX + i * K, qWu + j * K, K);
    return silu(g) * u;
}

static int check_i8(int64_t M, int64_t N, int64_t K, const void *qX, const float *sx,
                    const void *qW, const float *sw)
{
    if (M < 0 || N < 0 || K < 0) return -1;
    if (M > 0 && (!sx || (K > 0 && !qX))) return -1;
    if (N > 0 && (!sw || (K > 0 && !qW))) return -1;
    return 0;
}

/* The exact integer sums A = qX qW^T (int64), for the integer checks. */
int ka_oracle_i8_dot(int64_t M, int64_t N, int64_t K, const int8_t *qX, const int8_t *qW, int64_t *A)
{
    if (M < 0 || N < 0 || K < 0) return -1;
    if (M * N > 0 && (!A || (K > 0 && (!qX || !qW)))) return -1;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < M; ++i)
        for (int64_t j = 0; j < N; ++j)
            A[i * N + j] = dot_i8(qX + i * K, qW + j * K, K);
    return 0;
}

int ka_oracle_i8_linear(int64_t M, int64_t N, int64_t K, const int8_t *qX, const float *sx,
                        const int8_t *qW, const float *sw, const uint16_t *R, double *Y)
{
    if (check_i8(M, N, K, qX, sx, qW, sw) != 0) return -1;
    if (M * N > 0 && !Y) return -1;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < M; ++i)
        for (int64_t j = 0; j < N; ++j)
            Y[i * N + j] = element_i8(i, j, N, K, qX, sx, qW, sw, R);
    return 0;
}

int ka_oracle_i8_linear_at(int64_t M, int64_t N, int64_t K, const int8_t *qX, const float *sx,
                           const int8_t *qW, const float *sw, const uint16_t *R, int64_t n,
                           const int64_t *rows, const int64_t *cols, double *out)
{
    if (check_i8(M, N, K, qX, sx, qW, sw) != 0 || n < 0) return -1;
    for (int64_t t = 0; t < n; ++t)
        if (rows[t] < 0 || rows[t] >= M || cols[t] < 0 || cols[t] >= N) return -1;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t t = 0; t < n; ++t)
        out[t] = element_i8(rows[t], cols[t], N, K, qX, sx, qW, sw, R);
    return 0;
}

int ka_oracle_i8_swiglu(int64_t M, int64_t N, int64_t K, const int8_t *qX, const float *sx,
                        const int8_t *qWg, const float *swg, const int8_t *qWu, const float *swu,
                        double *H)
{
    if (check_i8(M, N, K, qX, sx, qWg, swg) != 0 || check_i8(M, N, K, qX, sx, qWu, swu) != 0) return -1;
    if (M * N > 0 && !H) return -1;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < M; ++i)
        for (int64_t j = 0; j < N; ++j)
            H[i * N + j] = element_i8_swiglu(i, j, K, qX, sx, qWg, swg, qWu, swu);
    return 0;
}

int ka_oracle_i8_swiglu_at(int64_t M, int64_t N, int64_t K, const int8_t *qX, const float *sx,
                           const int8_t *qWg, const float *swg, const int8_t *qWu, const float *swu,
                           int64_t n, const int64_t *rows, const int64_t *cols, double *out)
{
    if (check_i8(M, N, K, qX, sx, qWg, swg) != 0 || check_i8(M, N, K, qX, sx, qWu, swu) != 0 || n < 0)
        return -1;
    for (int64_t t = 0; t < n; ++t)
        if (rows[t] < 0 || rows[t] >= M || cols[t] < 0 || cols[t] >= N) return -1;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t t = 0; t < n; ++t)
        out[t] = element_i8_swiglu(rows[t], cols[t], K, qX, sx, qWg, swg, qWu, swu);
    return 0;
}

/*
 * Grouped (batched) linear layer over an expert-major padded layout
 * (mixture-of-experts case study, Alg. 4: token-expert pairs are placed in
 * expert-contiguous rows of a [E x M_pad] buffer, gap rows zero-filled, and
 * every projection runs as one strided-batched GEMM).  Expert e owns rows
 * [e*M_pad, (e+1)*M_pad) of X and Y and its own weight W[e]:
 *
 *     Y[e,i,j] = sum_k X[e,i,k] W[e,j,k]            for i < rows(e)
 *     H[e,i,j] = silu(X[e,i,:].Wg[e,j,:]) * (X[e,i,:].Wu[e,j,:])   (SwiGLU form)
 *
 * X is [E,M_pad,K], W (Wg, Wu) [E,N,K], Y (H) [E,M_pad,N], bf16 patterns;
 * counts[e] is the number of valid rows of expert e, clamped to [0, M_pad]
 * (NULL: every row is valid).  Rows at or past rows(e) are not computed and
 * their outputs are left as they were (the gap rows).  Each valid element is
 * the plain (or SwiGLU) definition above, in double, not rounded.
 */
static int64_t group_rows(const int32_t *counts, int64_t e, int64_t Mpad)
{
    if (!counts) return Mpad;
    int64_t c = counts[e];
    return c < 0 ? 0 : (c > Mpad ? Mpad : c);
}

static int check_grouped(int64_t E, int64_t Mpad, int64_t N, int64_t K, const void *X, const void *W)
{
    if (E < 0 || Mpad < 0 || N < 0 || K < 0) return -1;
    if (E * Mpad * K > 0 && !X) return -1;
    if (E * N * K > 0 && !W) return -1;
    return 0;
}

int ka_oracle_grouped_linear(int64_t E, int64_t Mpad, int64_t N, int64_t K, const uint16_t *X,
                             const uint16_t *W, const int32_t *counts, double *Y)
{
    if (check_grouped(E, Mpad, N, K, X, W) != 0) return -1;
    if (E * Mpad * N > 0 && !Y) return -1;
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t e = 0; e < E; ++e)
        for (int64_t i = 0; i < Mpad; ++i) {
            if (i >= group_rows(counts, e, Mpad)) continue;
            for (int64_t j = 0; j < N; ++j)
                Y[(e * Mpad + i) * N + j] = element(i, j, N, K, X + e * Mpad * K, W + e * N * K, NULL);
        }
    return 0;
}

int ka_oracle_grouped_swiglu(int64_t E, int64_t Mpad, int64_t N, int64_t K, const uint16_t *X,
                             const uint16_t *Wg, const uint16_t *Wu, const int32_t *counts, double *H)
{
    if (check_grouped(E, Mpad, N, K, X, Wg) != 0 || check_grouped(E, Mpad, N, K, X, Wu) != 0) return -1;
    if (E * Mpad * N > 0 && !H) return -1;
#pragma omp parallel for collapse(2) schedule(dynamic, 1)
    for (int64_t e = 0; e < E; ++e)
        for (int64_t i = 0; i < Mpad; ++i) {
            if (i >= group_rows(counts, e, Mpad)) continue;
            for (int64_t j = 0; j < N; ++j)
                H[(e * Mpad + i) * N + j] =
                    element_swiglu(i, j, K, X + e * Mpad * K, Wg + e * N * K, Wu + e * N * K);
        }
    return 0;
}

/*
 * Either grouped form at the n positions (groups[t], rows[t], cols[t]); a
 * position in a gap row is an error (-1).  swiglu != 0 selects the SwiGLU
 * form (W2 the up weights), else the plain form (W2 unused).
 */
int ka_oracle_grouped_at(int64_t E, int64_t Mpad, int64_t N, int64_t K, const uint16_t *X,
                         const uint16_t *W, const uint16_t *W2, const int32_t *counts, int swiglu,
                         int64_t n, const int64_t *groups, const int64_t *rows, const int64_t *cols,
                         double *out)
{
    if (check_grouped(E, Mpad, N, K, X, W) != 0 || n < 0) return -1;
    if (swiglu && check_grouped(E, Mpad, N, K, X, W2) != 0) return -1;
    for (int64_t t = 0; t < n; ++t)
        if (groups[t] < 0 || groups[t] >= E || rows[t] < 0 || rows[t] >= group_rows(counts, groups[t], Mpad) ||
            cols[t] < 0 || cols[t] >= N)
            return -1;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t t = 0; t < n; ++t) {
        const int64_t e = groups[t];
        out[t] = swiglu ? element_swiglu(rows[t], cols[t], K, X + e * Mpad * K, W + e * N * K, W2 + e * N * K)
                        : element(rows[t], cols[t], N, K, X + e * Mpad * K, W + e * N * K, NULL);
    }
    return 0;
}

/*
 * FP8 (E4M3) linear layer and SwiGLU with dequantisation scales: the
 * precision axis the paper's strategy skills name (FP8 / BF16 choices), in
 * the same scaled form as the INT8 path above, with FP8 E4M3 operands in
 * place of int8 (one binary32 scale per activation row and per output
 * channel):
 *
 *     Y[i,j] = sx[i] sw[j] sum_k x8(qX[i,k]) x8(qW[j,k])  (+ R[i,j])
 *     H[i,j] = silu(sx[i] swg[j] Sg[i,j]) * (sx[i] swu[j] Su[i,j])
 *
 * x8() decodes the OCP 8-bit E4M3 format (the "FN" variant): sign bit,
 * 4 exponent bits with bias 7, 3 mantissa bits; exponent field 0 gives
 * subnormals m/8 * 2^-6; exponent field 15 with mantissa 7 is NaN (there are
 * no infinities), so the largest finite magnitude is 1.75 * 2^8 = 448.
 * Every decoded value and every product of two is exact in double; the
 * k-sum runs ascending in double; then (sx * sw) * S (+ R); silu as above.
 */
static double fp8_e4m3_to_double(uint8_t b)
{
    int sign = b >> 7;
    int e = (b >> 3) & 15;
    int m = b & 7;
    double v;
    if (e == 15 && m == 7)
        v = NAN;
    else if (e == 0)
        v = ldexp((double)m, -9);            /* m/8 * 2^-6 */
    else
        v = ldexp((double)(8 + m), e - 10);  /* (1 + m/8) * 2^(e-7) */
    return sign ? -v : v;
}

static double dot_f8(const uint8_t *x, const uint8_t *w, int64_t K)
{
    double acc = 0.0;
    for (int64_t k = 0; k < K; ++k)
        acc += fp8_e4m3_to_double(x[k]) * fp8_e4m3_to_double(w[k]);
    return acc;
}

static double element_f8(int64_t i, int64_t j, int64_t N, int64_t K, const uint8_t *qX,
                         const float *sx, const uint8_t *qW, const float *sw, const uint16_t *R)
{
    double y = (double)sx[i] * (double)sw[j] * dot_f8(qX + i * K, qW + j * K, K);
    if (R)
        y += bf16_bits_to_double(R[i * N + j]);
    return y;
}

static double element_f8_swiglu(int64_t i, int64_t j, int64_t K, const uint8_t *qX, const float *sx,
                                const uint8_t *qWg, const float *swg, const uint8_t *qWu, const float *swu)
{
    double g = (double)sx[i] * (double)swg[j] * dot_f8(qX + i * K, qWg + j * K, K);
    double u = (double)sx[i] * (double)swu[j] * dot_f8(qX + i * K, qWu + j * K, K);
    return silu(g) * u;
}

/* Decode n E4M3 bytes (the format definition above) into doubles. */
void ka_oracle_fp8_decode(int64_t n, const uint8_t *in, double *out)
{
    for (int64_t t = 0; t < n; ++t)
        out[t] = fp8_e4m3_to_double(in[t]);
}

int ka_oracle_f8_linear(int64_t M, int64_t N, int64_t K, const uint8_t *qX, const float *sx,
                        const uint8_t *qW, const float *sw, const uint16_t *R, double *Y)
{
    if (check_i8(M, N, K, qX, sx, qW, sw) != 0) return -1;
    if (M * N > 0 && !Y) return -1;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < M; ++i)
        for (int64_t j = 0; j < N; ++j)
            Y[i * N + j] = element_f8(i, j, N, K, qX, sx, qW, sw, R);
    return 0;
}

int ka_oracle_f8_linear_at(int64_t M, int64_t N, int64_t K, const uint8_t *qX, const float *sx,
                           const uint8_t *qW, const float *sw, const uint16_t *R, int64_t n,
                           const int64_t *rows, const int64_t *cols, double *out)
{
    if (check_i8(M, N, K, qX, sx, qW, sw) != 0 || n < 0) return -1;
    for (int64_t t = 0; t < n; ++t)
        if (rows[t] < 0 || rows[t] >= M || cols[t] < 0 || cols[t] >= N) return -1;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t t = 0; t < n; ++t)
        out[t] = element_f8(rows[t], cols[t], N, K, qX, sx, qW, sw, R);
    return 0;
}

int ka_oracle_f8_swiglu(int64_t M, int64_t N, int64_t K, const uint8_t *qX, const float *sx,
                        const uint8_t *qWg, const float *swg, const uint8_t *qWu, const float *swu,
                        double *H)
{
    if (check_i8(M, N, K, qX, sx, qWg, swg) != 0 || check_i8(M, N, K, qX, sx, qWu, swu) != 0) return -1;
    if (M * N > 0 && !H) return -1;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < M; ++i)
        for (int64_t j = 0; j < N; ++j)
            H[i * N + j] = element_f8_swiglu(i, j, K, qX, sx, qWg, swg, qWu, swu);
    return 0;
}

int ka_oracle_f8_swiglu_at(int64_t M, int64_t N, int64_t K, const uint8_t *qX, const float *sx,
                           const uint8_t *qWg, const float *swg, const uint8_t *qWu, const float *swu,
                           int64_t n, const int64_t *rows, const int64_t *cols, double *out)
{
    if (check_i8(M, N, K, qX, sx, qWg, swg) != 0 || check_i8(M, N, K, qX, sx, qWu, swu) != 0 || n < 0)
        return -1;
    for (int64_t t = 0; t < n; ++t)
        if (rows[t] < 0 || rows[t] >= M || cols[t] < 0 || cols[t] >= N) return -1;
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t t = 0; t < n; ++t)
        out[t] = element_f8_swiglu(rows[t], cols[t], K, qX, sx, qWg, swg, qWu, swu);
    return 0;
}

/* Number of threads the OpenMP loops above use (1 without OpenMP). */
int ka_oracle_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Sets the number of threads the OpenMP loops use from now on (n >= 1; no
 * effect without OpenMP).  Used to time the oracle on one core. */
void ka_oracle_set_threads(int n)
{
#ifdef _OPENMP
    if (n >= 1) omp_set_num_threads(n);
#else
    (void)n;
#endif
}
