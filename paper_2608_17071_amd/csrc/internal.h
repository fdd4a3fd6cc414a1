// Private declarations shared by the library's translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace kernelarc {

// ---------------------------------------------------------------- plans ----
// One plan = one kernel variant plus its split-K rule.  The plan table and
// the selection rules live in api.hip; the launchers live beside their
// kernels.
enum PlanId : int {
    PLAN_GENERIC = 0,          // scalar LDS-tiled kernel: any K, any alignment
    PLAN_GEMV = 1,             // M <= 4: contiguous W stream, VALU dot products
};

// MFMA macro-tile kernel configurations (tile_kernel.h):
// BM x BN output tile, BK deep stages, STAGES-deep LDS ring, waves.
enum TileCfg : int {
    TC_256x256_K64_S2_W8 = 0,
    TC_256x256_K64_S2_W4_M16A = 1,  // 4 waves of 128x128, 16x16x32 MFMA, AGPR accumulators (bf16)
    TC_256x128_K64_S3_W8 = 2,
    TC_256x128_K64_S3_W8_L = 3,    // lagged refill
    TC_128x128_K64_S2_W4 = 4,
    TC_128x128_K64_S3_W4 = 5,
    TC_128x128_K64_S4_W4_L = 6,
    TC_64x64_K128_S3_W4 = 7,
    TC_64x64_K64_S4_W4 = 8,
    TC_64x128_K64_S4_W4 = 9,
    TC_COUNT = 10,
};

struct TileShape {
    int bm, bn, bk, workgroups_per_cu;
};
TileShape tile_shape(int cfg);

// One call: Y = bf16(alpha * X W^T + beta * R + bias) with row strides
// (in elements).  The plain entry points pass dense strides (K, K, N, N),
// alpha = beta = 1 and no bias; R and bias may be null.
struct Problem {
    int64_t M, N, K;
    const uint16_t *X, *W, *R;   // R may be null (no residual term)
    uint16_t *Y;
    int64_t ldx, ldw, ldr, ldy;
    float alpha, beta;
    const uint16_t *bias;        // [N] or null
};

// The plain operator's arguments alone (dense strides, alpha = beta = 1, no
// bias): what the kernels of the plain entry points receive, so their
// argument block and its loads stay as small as the operation needs.
struct DenseProblem {
    int64_t M, N, K;
    const uint16_t *X, *W, *R;
    uint16_t *Y;
};

// Gated MLP input projection (SwiGLU): Y = bf16(silu(X W^T) * (X W2^T)),
// W the gate and W2 the up weights, all dense.  The tile kernels stage the
// two weight panels side by side as one B tile of twice the output width.
struct GluProblem {
    int64_t M, N, K;
    const uint16_t *X, *W, *W2;  // X [M,K]; W (gate), W2 (up) [N,K]
    uint16_t *Y;                 // [M,N]
};

// INT8 operands with dequantisation scales (symmetric W8A8: one scale per
// row of X, one per row of W):
//   Y = bf16(sx[i] sw[j] A[i,j] (+ R[i,j])),  A = qX qW^T summed exactly in int32.
struct I8Problem {
    int64_t M, N, K;
    const int8_t *X, *W;         // [M,K], [N,K]
    const uint16_t *R;           // [M,N] bf16 or null
    uint16_t *Y;                 // [M,N] bf16
    const float *sx, *sw;        // [M], [N]
};

// INT8 SwiGLU: Y = bf16(silu(sx swg Ag) * (sx swu Au)) with Ag = qX qW^T
// (gate) and Au = qX qW2^T (up).
struct I8GluProblem {
    int64_t M, N, K;
    const int8_t *X, *W, *W2;
    uint16_t *Y;
    const float *sx, *sw, *sw2;  // [M], gate [N], up [N]
};

// FP8 (OCP E4M3) operands with the same dequantisation scales as the INT8
// forms: Y = bf16(sx[i] sw[j] S[i,j] (+ R)), S the fp32 sum of the products
// of the decoded values.  Bit patterns are held as uint8.
struct F8Problem {
    int64_t M, N, K;
    const uint8_t *X, *W;
    const uint16_t *R;
    uint16_t *Y;
    const float *sx, *sw;
};
struct F8GluProblem {
    int64_t M, N, K;
    const uint8_t *X, *W, *W2;
    uint16_t *Y;
    const float *sx, *sw, *sw2;
};

// Grouped (per-expert) form of a dense problem over an expert-major padded
// layout: group g owns rows [g*Mpad, (g+1)*Mpad) of X and Y and its own
// weights (W + g*N*K, and W2 for SwiGLU); its valid rows are counts[g]
// clamped to [0, Mpad] (counts null: all Mpad).  M is unused (the kernels
// set it per group); rows past the valid ones are neither read nor written.
template <class Base>
struct Grouped : Base {
    int64_t G, Mpad;
    const int32_t *counts;
};
template <class P>
struct grouped_trait {
    static constexpr bool value = false;
    using base = P;
};
template <class B>
struct grouped_trait<Grouped<B>> {
    static constexpr bool value = true;
    using base = B;
};

// Uniform access to every form inside the kernels.
__host__ __device__ inline int64_t ldx_of(const Problem &p) { return p.ldx; }
__host__ __device__ inline int64_t ldw_of(const Problem &p) { return p.ldw; }
__host__ __device__ inline int64_t ldr_of(const Problem &p) { return p.ldr; }
__host__ __device__ inline int64_t ldy_of(const Problem &p) { return p.ldy; }
__host__ __device__ inline float alpha_of(const Problem &p) { return p.alpha; }
__host__ __device__ inline float beta_of(const Problem &p) { return p.beta; }
__host__ __device__ inline const uint16_t *bias_of(const Problem &p) { return p.bias; }
__host__ __device__ inline int64_t ldx_of(const DenseProblem &p) { return p.K; }
__host__ __device__ inline int64_t ldw_of(const DenseProblem &p) { return p.K; }
__host__ __device__ inline int64_t ldr_of(const DenseProblem &p) { return p.N; }
__host__ __device__ inline int64_t ldy_of(const DenseProblem &p) { return p.N; }
__host__ __device__ inline float alpha_of(const DenseProblem &) { return 1.0f; }
__host__ __device__ inline float beta_of(const DenseProblem &) { return 1.0f; }
__host__ __device__ inline const uint16_t *bias_of(const DenseProblem &) { return nullptr; }

__host__ __device__ inline int64_t ldx_of(const GluProblem &p) { return p.K; }
__host__ __device__ inline int64_t ldw_of(const GluProblem &p) { return p.K; }
__host__ __device__ inline int64_t ldr_of(const GluProblem &p) { return p.N; }
__host__ __device__ inline int64_t ldy_of(const GluProblem &p) { return p.N; }
__host__ __device__ inline float alpha_of(const GluProblem &) { return 1.0f; }
__host__ __device__ inline float beta_of(const GluProblem &) { return 1.0f; }
__host__ __device__ inline const uint16_t *bias_of(const GluProblem &) { return nullptr; }
__host__ __device__ inline int64_t ldx_of(const I8Problem &p) { return p.K; }
__host__ __device__ inline int64_t ldw_of(const I8Problem &p) { return p.K; }
__host__ __device__ inline int64_t ldr_of(const I8Problem &p) { return p.N; }
__host__ __device__ inline int64_t ldy_of(const I8Problem &p) { return p.N; }
__host__ __device__ inline float alpha_of(const I8Problem &) { return 1.0f; }
__host__ __device__ inline float beta_of(const I8Problem &) { return 1.0f; }
__host__ __device__ inline const uint16_t *bias_of(const I8Problem &) { return nullptr; }
__host__ __device__ inline int64_t ldx_of(const I8GluProblem &p) { return p.K; }
__host__ __device__ inline int64_t ldw_of(const I8GluProblem &p) { return p.K; }
__host__ __device__ inline int64_t ldr_of(const I8GluProblem &p) { return p.N; }
__host__ __device__ inline int64_t ldy_of(const I8GluProblem &p) { return p.N; }
__host__ __device__ inline float alpha_of(const I8GluProblem &) { return 1.0f; }
__host__ __device__ inline float beta_of(const I8GluProblem &) { return 1.0f; }
__host__ __device__ inline const uint16_t *bias_of(const I8GluProblem &) { return nullptr; }
__host__ __device__ inline int64_t ldx_of(const F8Problem &p) { return p.K; }
__host__ __device__ inline int64_t ldw_of(const F8Problem &p) { return p.K; }
__host__ __device__ inline int64_t ldr_of(const F8Problem &p) { return p.N; }
__host__ __device__ inline int64_t ldy_of(const F8Problem &p) { return p.N; }
__host__ __device__ inline float alpha_of(const F8Problem &) { return 1.0f; }
__host__ __device__ inline float beta_of(const F8Problem &) { return 1.0f; }
__host__ __device__ inline const uint16_t *bias_of(const F8Problem &) { return nullptr; }
__host__ __device__ inline int64_t ldx_of(const F8GluProblem &p) { return p.K; }
__host__ __device__ inline int64_t ldw_of(const F8GluProblem &p) { return p.K; }
__host__ __device__ inline int64_t ldr_of(const F8GluProblem &p) { return p.N; }
__host__ __device__ inline int64_t ldy_of(const F8GluProblem &p) { return p.N; }
__host__ __device__ inline float alpha_of(const F8GluProblem &) { return 1.0f; }
__host__ __device__ inline float beta_of(const F8GluProblem &) { return 1.0f; }
__host__ __device__ inline const uint16_t *bias_of(const F8GluProblem &) { return nullptr; }
__host__ __device__ inline const uint16_t *resid_of(const F8Problem &p) { return p.R; }
__host__ __device__ inline const uint16_t *resid_of(const F8GluProblem &) { return nullptr; }
__host__ __device__ inline const uint16_t *resid_of(const I8Problem &p) { return p.R; }
__host__ __device__ inline const uint16_t *resid_of(const I8GluProblem &) { return nullptr; }
__host__ __device__ inline const uint16_t *resid_of(const Problem &p) { return p.R; }
__host__ __device__ inline const uint16_t *resid_of(const DenseProblem &p) { return p.R; }
__host__ __device__ inline const uint16_t *resid_of(const GluProblem &) { return nullptr; }

// True unless the call is the plain operator (then the dense kernels run).
inline bool is_general(const Problem &p) {
    return p.ldx != p.K || p.ldw != p.K || (p.R && p.ldr != p.N) || p.ldy != p.N || p.alpha != 1.0f ||
           (p.R && p.beta != 1.0f) || p.bias != nullptr;
}
inline DenseProblem dense_of(const Problem &p) { return DenseProblem{p.M, p.N, p.K, p.X, p.W, p.R, p.Y}; }

// Bytes a buffer resource must cover for `rows` rows of `cols` elements at
// row stride `ld` (the last row ends at its last element).
__host__ __device__ inline int64_t strided_bytes(int64_t rows, int64_t cols, int64_t ld) {
    return rows > 0 && cols > 0 ? ((rows - 1) * ld + cols) * 2 : 0;
}

// Per-device split-K workspace: fp32 partials followed by tile counters.
struct Workspace {
    float *partials;
    int64_t partial_floats;
    unsigned *counters;
    int64_t counter_count;
};

// Launchers: validate nothing (plan.hip has done it), enqueue, return the
// hipError_t of the launch.
hipError_t launch_generic(const Problem &p, hipStream_t s);
hipError_t launch_gemv(const Problem &p, hipStream_t s);
// full_tiles > 0 with split > 1: tiles past the first full_tiles (band
// order) are split in K, the others run whole (see tile_kernel.h).
hipError_t launch_tile(int cfg, const Problem &p, int split, int64_t full_tiles, const Workspace *ws, hipStream_t s);
hipError_t launch_stream(const Problem &p, int bk, int stages, int rows, int split, const Workspace *ws,
                         hipStream_t s);
bool stream_config_exists(int bk, int stages, int rows);
// INT8 operands through the 16- and 32-row streaming configurations.
hipError_t launch_stream_i8(const I8Problem &p, int bk, int stages, int rows, int split, const Workspace *ws,
                            hipStream_t s);
// SwiGLU: the generic kernel, and the tile kernels of the configurations
// that can pair gate and up blocks (tile_glu_ok).
hipError_t launch_generic_glu(const GluProblem &p, hipStream_t s);
hipError_t launch_tile_glu(int cfg, const GluProblem &p, int split, int64_t full_tiles, const Workspace *ws,
                           hipStream_t s);
bool tile_glu_ok(int cfg);
// INT8: generic kernels (any K, any alignment) and the tile kernels (K a
// multiple of 16; SwiGLU on the configurations of tile_glu_ok).
// Grouped forms (bf16): the tile kernels without split-K, and generic kernels.
hipError_t launch_tile_grouped(int cfg, const Grouped<DenseProblem> &p, hipStream_t s);
hipError_t launch_tile_grouped_glu(int cfg, const Grouped<GluProblem> &p, hipStream_t s);
hipError_t launch_generic_grouped(const Grouped<DenseProblem> &p, hipStream_t s);
hipError_t launch_generic_grouped_glu(const Grouped<GluProblem> &p, hipStream_t s);
__host__ __device__ inline int64_t group_rows(const int32_t *counts, int64_t g, int64_t Mpad) {
    if (!counts) return Mpad;
    const int64_t c = counts[g];
    return c < 0 ? 0 : (c > Mpad ? Mpad : c);
}
// FP8: tile kernels (configurations of tile_f8_ok; SwiGLU also tile_glu_ok)
// and generic kernels.
bool tile_f8_ok(int cfg);
// 16x16x32 MFMA tile configurations (bf16 operands only).
bool tile_is_m16(int cfg);
hipError_t launch_tile_f8(int cfg, const F8Problem &p, int split, int64_t full_tiles, const Workspace *ws,
                          hipStream_t s);
hipError_t launch_tile_f8_glu(int cfg, const F8GluProblem &p, int split, int64_t full_tiles, const Workspace *ws,
                              hipStream_t s);
hipError_t launch_generic_f8(const F8Problem &p, hipStream_t s);
hipError_t launch_generic_f8_glu(const F8GluProblem &p, hipStream_t s);
// OCP E4M3 (bias 7, no infinities, S.1111.111 = NaN) to fp32, exact.
__device__ __forceinline__ float fp8_e4m3_to_f32(uint8_t b) {
    const uint32_t sign = static_cast<uint32_t>(b & 0x80) << 24;
    const uint32_t e = (b >> 3) & 15, m = b & 7;
    float v;
    if (e == 15 && m == 7) v = __builtin_nanf("");
    else if (e == 0) v = static_cast<float>(m) * 0.001953125f;              // m * 2^-9
    else v = __uint_as_float(((e + 120) << 23) | (m << 20));                  // (1 + m/8) 2^(e-7)
    return __uint_as_float(__float_as_uint(v) | sign);
}
hipError_t launch_generic_i8(const I8Problem &p, hipStream_t s);
hipError_t launch_generic_i8_glu(const I8GluProblem &p, hipStream_t s);
hipError_t launch_tile_i8(int cfg, const I8Problem &p, int split, int64_t full_tiles, const Workspace *ws,
                          hipStream_t s);
hipError_t launch_tile_i8_glu(int cfg, const I8GluProblem &p, int split, int64_t full_tiles, const Workspace *ws,
                              hipStream_t s);

// Shape rules of the kernels, used by the plan table (host only).
bool gemv_fits(int64_t M, int64_t N, int64_t K, int64_t ldw);
int stream_split_for(int64_t M, int64_t N, int64_t K, int bk, int rows);
int64_t stream_workspace_floats(int64_t M, int64_t N, int split, int rows);
int64_t stream_counter_count(int64_t N, int rows);

// ------------------------------------------------------- device helpers ----
// bf16 <-> fp32.  Widening is exact (bf16 is the top half of a binary32).
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// fp32 -> bf16, round to nearest, ties to even; NaN stays NaN (quiet, sign
// and leading payload bits kept), finite values beyond the bf16 range round
// to infinity.  gfx950 does this in one instruction (v_cvt_pk_bf16_f32);
// its results equal the bit-level definition -- add 0x7fff plus the lowest
// kept bit, truncate; NaN -> top half with the quiet bit set -- for every
// one of the 2^32 inputs.
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

// The epilogue's value before rounding: alpha * acc, then + beta * r as one
// fused multiply-add when there is a residual.  With alpha = beta = 1 this is
// exactly acc + r (one rounding), the plain operator's value.
__device__ __forceinline__ float combine(float acc, float r, bool has_r, float alpha, float beta) {
    const float a = alpha * acc;
    return has_r ? __builtin_fmaf(beta, r, a) : a;
}

// silu(z) = z * sigmoid(z) = z / (1 + e^-z) in fp32: e^-z as 2^(-z log2 e)
// (v_exp_f32) and the reciprocal by v_rcp_f32, each within about 1 ulp, so
// the result is within a few fp32 ulps (plus |z| 2^-24 relative from the
// scaled exponent), far below one bf16 rounding.  For z <= -88.7 the power
// overflows to infinity and the result is -0; for large z it is z.
__device__ __forceinline__ float silu_f32(float z) {
    const float t = __builtin_amdgcn_exp2f(-z * 1.44269504088896341f);
    return z * __builtin_amdgcn_rcpf(1.0f + t);
}

// Two values at once (one v_cvt_pk_bf16_f32): lo in bits 0-15, hi in 16-31.
typedef float f32x2_pair __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_pair __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t f32x2_to_bf16x2_rne(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_pair{lo, hi}, bf16x2_pair));
}

}  // namespace kernelarc
