// Generic kernels: Y = alpha X W^T (+ beta R) (+ bias) for any shape, any
// row strides and any pointer alignment; SwiGLU, the INT8 and FP8 forms
// and the grouped (per-expert) forms for any shape and alignment.
//
// This is the correctness fallback (K not a multiple of 8, pointers not
// 16-byte aligned).  Each 256-thread workgroup computes a 64x64 output tile;
// each thread owns a 4x4 sub-block strided by 16 in both directions.  Both
// operands are staged through LDS as fp32 in 16-deep K slices with bounds-
// checked scalar loads; products of bf16 values are exact in fp32 and the
// k-terms are accumulated in ascending order.
#include "internal.h"

#include <type_traits>

namespace kernelarc {
namespace {

constexpr int GT = 64;   // output tile edge
constexpr int GK = 16;   // K slice

__device__ __forceinline__ void generic_body(const Problem &p, int64_t tile, int64_t tiles_n) {
    __shared__ float xs[GK][GT + 1];
    __shared__ float ws[GK][GT + 1];

    const int tx = threadIdx.x & 15;
    const int ty = threadIdx.x >> 4;
    const int64_t m0 = (tile / tiles_n) * GT;
    const int64_t n0 = (tile % tiles_n) * GT;

    float acc[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) acc[a][b] = 0.0f;

    for (int64_t k0 = 0; k0 < p.K; k0 += GK) {
        // 64 rows x 16 k of each operand = 1024 values = 4 per thread.
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int idx = threadIdx.x + 256 * t;
            const int r = idx / GK;
            const int kk = idx % GK;
            const int64_t k = k0 + kk;
            const int64_t xm = m0 + r;
            const int64_t wn = n0 + r;
            xs[kk][r] = (xm < p.M && k < p.K) ? bf16_to_f32(p.X[xm * p.ldx + k]) : 0.0f;
            ws[kk][r] = (wn < p.N && k < p.K) ? bf16_to_f32(p.W[wn * p.ldw + k]) : 0.0f;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < GK; ++kk) {
            float xv[4], wv[4];
#pragma unroll
            for (int a = 0; a < 4; ++a) xv[a] = xs[kk][ty + 16 * a];
#pragma unroll
            for (int b = 0; b < 4; ++b) wv[b] = ws[kk][tx + 16 * b];
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int b = 0; b < 4; ++b) acc[a][b] = fmaf(xv[a], wv[b], acc[a][b]);
        }
        __syncthreads();
    }

#pragma unroll
    for (int a = 0; a < 4; ++a) {
        const int64_t i = m0 + ty + 16 * a;
        if (i >= p.M) continue;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const int64_t j = n0 + tx + 16 * b;
            if (j >= p.N) continue;
            const float r = p.R ? bf16_to_f32(p.R[i * p.ldr + j]) : 0.0f;
            float y = combine(acc[a][b], r, p.R != nullptr, p.alpha, p.beta);
            if (p.bias) y += bf16_to_f32(p.bias[j]);
            p.Y[i * p.ldy + j] = f32_to_bf16_rne(y);
        }
    }
}

__global__ __launch_bounds__(256) void generic_kernel(Problem p, int64_t tiles_n) {
    generic_body(p, blockIdx.x, tiles_n);
}

// Grouped: workgroup id = (group, tile within the group's [Mpad, N] output).
__global__ __launch_bounds__(256) void generic_grouped_kernel(Grouped<DenseProblem> p, int64_t tiles_n,
                                                              int64_t tiles_per_group) {
    const int64_t g = blockIdx.x / tiles_per_group;
    const int64_t tile = blockIdx.x - g * tiles_per_group;
    const int64_t rows = group_rows(p.counts, g, p.Mpad);
    if ((tile / tiles_n) * GT >= rows) return;
    const Problem q{rows, p.N, p.K, p.X + g * p.Mpad * p.K, p.W + g * p.N * p.K, nullptr, p.Y + g * p.Mpad * p.N,
                    p.K, p.K, p.N, p.N, 1.0f, 1.0f, nullptr};
    generic_body(q, tile, tiles_n);
}

// SwiGLU fallback: the same tiling with both weight operands staged, the
// gate and up sums kept side by side, and silu(g) * u rounded once.
__device__ __forceinline__ void generic_glu_body(const GluProblem &p, int64_t tile, int64_t tiles_n) {
    __shared__ float xs[GK][GT + 1];
    __shared__ float gs[GK][GT + 1];
    __shared__ float us[GK][GT + 1];

    const int tx = threadIdx.x & 15;
    const int ty = threadIdx.x >> 4;
    const int64_t m0 = (tile / tiles_n) * GT;
    const int64_t n0 = (tile % tiles_n) * GT;

    float g[4][4], u[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) g[a][b] = u[a][b] = 0.0f;

    for (int64_t k0 = 0; k0 < p.K; k0 += GK) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int idx = threadIdx.x + 256 * t;
            const int r = idx / GK;
            const int kk = idx % GK;
            const int64_t k = k0 + kk;
            const int64_t xm = m0 + r;
            const int64_t wn = n0 + r;
            const bool kin = k < p.K;
            xs[kk][r] = (xm < p.M && kin) ? bf16_to_f32(p.X[xm * p.K + k]) : 0.0f;
            gs[kk][r] = (wn < p.N && kin) ? bf16_to_f32(p.W[wn * p.K + k]) : 0.0f;
            us[kk][r] = (wn < p.N && kin) ? bf16_to_f32(p.W2[wn * p.K + k]) : 0.0f;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < GK; ++kk) {
            float xv[4], gv[4], uv[4];
#pragma unroll
            for (int a = 0; a < 4; ++a) xv[a] = xs[kk][ty + 16 * a];
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                gv[b] = gs[kk][tx + 16 * b];
                uv[b] = us[kk][tx + 16 * b];
            }
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    g[a][b] = fmaf(xv[a], gv[b], g[a][b]);
                    u[a][b] = fmaf(xv[a], uv[b], u[a][b]);
                }
        }
        __syncthreads();
    }

#pragma unroll
    for (int a = 0; a < 4; ++a) {
        const int64_t i = m0 + ty + 16 * a;
        if (i >= p.M) continue;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const int64_t j = n0 + tx + 16 * b;
            if (j >= p.N) continue;
            p.Y[i * p.N + j] = f32_to_bf16_rne(silu_f32(g[a][b]) * u[a][b]);
        }
    }
}

__global__ __launch_bounds__(256) void generic_glu_kernel(GluProblem p, int64_t tiles_n) {
    generic_glu_body(p, blockIdx.x, tiles_n);
}

__global__ __launch_bounds__(256) void generic_grouped_glu_kernel(Grouped<GluProblem> p, int64_t tiles_n,
                                                                  int64_t tiles_per_group) {
    const int64_t g = blockIdx.x / tiles_per_group;
    const int64_t tile = blockIdx.x - g * tiles_per_group;
    const int64_t rows = group_rows(p.counts, g, p.Mpad);
    if ((tile / tiles_n) * GT >= rows) return;
    const GluProblem q{rows, p.N, p.K, p.X + g * p.Mpad * p.K, p.W + g * p.N * p.K, p.W2 + g * p.N * p.K,
                       p.Y + g * p.Mpad * p.N};
    generic_glu_body(q, tile, tiles_n);
}

// INT8 and FP8 fallbacks: the same 64x64 tiling with the operands staged
// as int32 (exact int32 sums) or as decoded fp32 (E4M3 values and their
// products are exact in fp32); dequantisation (and the residual, or SwiGLU)
// in fp32 as the tile kernels do it.
template <class T>
__device__ __forceinline__ T widen(int8_t v) { return v; }
template <class T>
__device__ __forceinline__ T widen(uint8_t v) { return fp8_e4m3_to_f32(v); }

template <bool GLU_, class P>
__device__ __forceinline__ void generic_i8_body(const P &p, int64_t tiles_n) {
    using T = typename std::conditional<std::is_same<decltype(p.X), const int8_t *>::value, int, float>::type;
    __shared__ T xs[GK][GT + 1];
    __shared__ T gs[GK][GT + 1];
    __shared__ T us[GLU_ ? GK : 1][GT + 1];

    const int tx = threadIdx.x & 15;
    const int ty = threadIdx.x >> 4;
    const int64_t tile = blockIdx.x;
    const int64_t m0 = (tile / tiles_n) * GT;
    const int64_t n0 = (tile % tiles_n) * GT;

    T g[4][4], u[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) g[a][b] = u[a][b] = 0;

    for (int64_t k0 = 0; k0 < p.K; k0 += GK) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int idx = threadIdx.x + 256 * t;
            const int r = idx / GK;
            const int kk = idx % GK;
            const int64_t k = k0 + kk;
            const int64_t xm = m0 + r;
            const int64_t wn = n0 + r;
            const bool kin = k < p.K;
            xs[kk][r] = (xm < p.M && kin) ? widen<T>(p.X[xm * p.K + k]) : T(0);
            gs[kk][r] = (wn < p.N && kin) ? widen<T>(p.W[wn * p.K + k]) : T(0);
            if constexpr (GLU_) us[kk][r] = (wn < p.N && kin) ? widen<T>(p.W2[wn * p.K + k]) : T(0);
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < GK; ++kk) {
            T xv[4], gv[4], uv[4];
#pragma unroll
            for (int a = 0; a < 4; ++a) xv[a] = xs[kk][ty + 16 * a];
#pragma unroll
            for (int b = 0; b < 4; ++b) {
                gv[b] = gs[kk][tx + 16 * b];
                if constexpr (GLU_) uv[b] = us[kk][tx + 16 * b];
            }
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    g[a][b] += xv[a] * gv[b];
                    if constexpr (GLU_) u[a][b] += xv[a] * uv[b];
                }
        }
        __syncthreads();
    }

#pragma unroll
    for (int a = 0; a < 4; ++a) {
        const int64_t i = m0 + ty + 16 * a;
        if (i >= p.M) continue;
        const float sr = p.sx[i];
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const int64_t j = n0 + tx + 16 * b;
            if (j >= p.N) continue;
            float y;
            if constexpr (GLU_) {
                const float gv = static_cast<float>(g[a][b]) * (sr * p.sw[j]);
                const float uv = static_cast<float>(u[a][b]) * (sr * p.sw2[j]);
                y = silu_f32(gv) * uv;
            } else {
                y = static_cast<float>(g[a][b]) * (sr * p.sw[j]);
                if (p.R) y += bf16_to_f32(p.R[i * p.N + j]);
            }
            p.Y[i * p.N + j] = f32_to_bf16_rne(y);
        }
    }
}

__global__ __launch_bounds__(256) void generic_i8_kernel(I8Problem p, int64_t tiles_n) {
    generic_i8_body<false>(p, tiles_n);
}

__global__ __launch_bounds__(256) void generic_i8_glu_kernel(I8GluProblem p, int64_t tiles_n) {
    generic_i8_body<true>(p, tiles_n);
}

__global__ __launch_bounds__(256) void generic_f8_kernel(F8Problem p, int64_t tiles_n) {
    generic_i8_body<false>(p, tiles_n);
}

__global__ __launch_bounds__(256) void generic_f8_glu_kernel(F8GluProblem p, int64_t tiles_n) {
    generic_i8_body<true>(p, tiles_n);
}

}  // namespace

hipError_t launch_generic_i8(const I8Problem &p, hipStream_t s) {
    const int64_t tiles_n = (p.N + GT - 1) / GT;
    const int64_t tiles = ((p.M + GT - 1) / GT) * tiles_n;
    hipLaunchKernelGGL(generic_i8_kernel, dim3(static_cast<unsigned>(tiles)), dim3(256), 0, s, p, tiles_n);
    return hipGetLastError();
}

hipError_t launch_generic_f8(const F8Problem &p, hipStream_t s) {
    const int64_t tiles_n = (p.N + GT - 1) / GT;
    const int64_t tiles = ((p.M + GT - 1) / GT) * tiles_n;
    hipLaunchKernelGGL(generic_f8_kernel, dim3(static_cast<unsigned>(tiles)), dim3(256), 0, s, p, tiles_n);
    return hipGetLastError();
}

hipError_t launch_generic_f8_glu(const F8GluProblem &p, hipStream_t s) {
    const int64_t tiles_n = (p.N + GT - 1) / GT;
    const int64_t tiles = ((p.M + GT - 1) / GT) * tiles_n;
    hipLaunchKernelGGL(generic_f8_glu_kernel, dim3(static_cast<unsigned>(tiles)), dim3(256), 0, s, p, tiles_n);
    return hipGetLastError();
}

hipError_t launch_generic_i8_glu(const I8GluProblem &p, hipStream_t s) {
    const int64_t tiles_n = (p.N + GT - 1) / GT;
    const int64_t tiles = ((p.M + GT - 1) / GT) * tiles_n;
    hipLaunchKernelGGL(generic_i8_glu_kernel, dim3(static_cast<unsigned>(tiles)), dim3(256), 0, s, p, tiles_n);
    return hipGetLastError();
}

hipError_t launch_generic_grouped(const Grouped<DenseProblem> &p, hipStream_t s) {
    const int64_t tiles_n = (p.N + GT - 1) / GT;
    const int64_t per = ((p.Mpad + GT - 1) / GT) * tiles_n;
    hipLaunchKernelGGL(generic_grouped_kernel, dim3(static_cast<unsigned>(p.G * per)), dim3(256), 0, s, p, tiles_n,
                       per);
    return hipGetLastError();
}

hipError_t launch_generic_grouped_glu(const Grouped<GluProblem> &p, hipStream_t s) {
    const int64_t tiles_n = (p.N + GT - 1) / GT;
    const int64_t per = ((p.Mpad + GT - 1) / GT) * tiles_n;
    hipLaunchKernelGGL(generic_grouped_glu_kernel, dim3(static_cast<unsigned>(p.G * per)), dim3(256), 0, s, p,
                       tiles_n, per);
    return hipGetLastError();
}

hipError_t launch_generic_glu(const GluProblem &p, hipStream_t s) {
    const int64_t tiles_n = (p.N + GT - 1) / GT;
    const int64_t tiles = ((p.M + GT - 1) / GT) * tiles_n;
    hipLaunchKernelGGL(generic_glu_kernel, dim3(static_cast<unsigned>(tiles)), dim3(256), 0, s, p, tiles_n);
    return hipGetLastError();
}

hipError_t launch_generic(const Problem &p, hipStream_t s) {
    const int64_t tiles_m = (p.M + GT - 1) / GT;
    const int64_t tiles_n = (p.N + GT - 1) / GT;
    const int64_t tiles = tiles_m * tiles_n;
    hipLaunchKernelGGL(generic_kernel, dim3(static_cast<unsigned>(tiles)), dim3(256), 0, s, p,
                       tiles_n);
    return hipGetLastError();
}

}  // namespace kernelarc
