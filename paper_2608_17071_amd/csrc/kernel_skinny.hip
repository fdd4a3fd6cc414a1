// Skinny-M kernel (M <= 64): Y = X W^T (+ R) when the time is the single
// pass over W (N*K*2 bytes) and the multiply is cheap.
//
// Roles are swapped relative to the macro-tile kernel: the MFMA A operand is
// a 16-row block of W and the B operand is X^T, so one
// v_mfma_f32_16x16x32_bf16 yields C[n][m] for 16 weight rows and 16 tokens;
// M is padded to 16 * MB with zeros (buffer loads past X's end read 0).
//
// Work split (the paper's split-K / reduction skills, Sec. "Strategy skills"):
//   * a workgroup of 8 waves owns 16 rows of W and one K slice; its 8 waves
//     each stream a contiguous sub-range of that slice, UNROLL MFMA steps of
//     32 k at a time, so every wave keeps UNROLL 16-byte W loads in flight;
//     W loads are marked non-temporal (W is touched once), X stays in L2;
//   * the 8 partial C blocks are summed through LDS in wave order;
//   * when N/16 alone gives too few workgroups for 256 CUs, K is also split
//     across S workgroups: each writes its fp32 partial block to the split-K
//     workspace, and the last of the S to arrive (a per-strip counter, agent-
//     scope release/acquire) adds the S blocks in slice order, applies the
//     epilogue and resets the counter for the next call;
//   * epilogue: fp32 sum + fp32(R), one nearest-even rounding to bf16; Y may
//     alias R (each element is read and written by the same thread).
// All sums run in a fixed order, so repeated calls are bitwise identical.
#include "internal.h"

namespace kernelarc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

constexpr int RSRC_WORD3 = 0x00020000;
constexpr uint32_t OOB_OFFSET = 0x80000000u;
constexpr int WAVES = 8;
constexpr int THREADS = 64 * WAVES;
constexpr int ROWS = 16;        // W rows per workgroup
constexpr int UNROLL = 8;       // MFMA steps (32 k each) per batch of loads
constexpr int AUX_NT = 2;       // non-temporal load
constexpr int WAITCNT_VM0 = 0x0F70;   // s_waitcnt vmcnt(0)

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), static_cast<short>(0),
                                             static_cast<int>(bytes), RSRC_WORD3);
}

__device__ __forceinline__ bf16x8 as_bf16x8(i32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// One batch: U MFMA steps of 32 k starting at k0 -- U loads of W (16 rows)
// and U*MB loads of X (16 tokens each); chunks at or past kend read zero.
template <int MB, int U>
__device__ __forceinline__ void issue_batch(i32x4 (&wv)[U], i32x4 (&xv)[U][MB],
                                            const __amdgpu_buffer_rsrc_t &rw,
                                            const __amdgpu_buffer_rsrc_t &rx, uint32_t w_row,
                                            const uint32_t (&x_row)[MB], int64_t k0, int64_t kend,
                                            int chunk) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int64_t k = k0 + u * 32 + chunk * 8;
        const bool ok = k < kend;
        const uint32_t kb = static_cast<uint32_t>(k * 2);
        wv[u] = __builtin_amdgcn_raw_buffer_load_b128(rw, ok ? w_row + kb : OOB_OFFSET, 0, AUX_NT);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
            xv[u][mb] = __builtin_amdgcn_raw_buffer_load_b128(rx, ok ? x_row[mb] + kb : OOB_OFFSET, 0, 0);
    }
}

template <int MB, int U>
__device__ __forceinline__ void mfma_batch(f32x4 (&acc)[MB], const i32x4 (&wv)[U], const i32x4 (&xv)[U][MB]) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
            acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(wv[u]), as_bf16x8(xv[u][mb]), acc[mb],
                                                              0, 0, 0);
}

template <int MB>
__global__ __launch_bounds__(THREADS) void skinny_kernel(DenseProblem p, int split, int64_t kslice,
                                                         float *ws, unsigned *counters) {
    constexpr int MP = 16 * MB;                         // padded token count
    constexpr int U = MB <= 2 ? 8 : 4;                  // MFMA steps per batch of loads
    __shared__ float red[WAVES][ROWS][MP];              // per-wave partial C^T blocks
    __shared__ int is_last;

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t strip = blockIdx.x / split;
    const int s = blockIdx.x % split;
    const int64_t n0 = strip * ROWS;
    const int64_t K = p.K;

    // W rows [n0, n0+16) as one panel; rows past N read as zero.
    const int64_t rows_w = (p.N - n0) < ROWS ? (p.N - n0) : ROWS;
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(p.W + n0 * K, static_cast<uint32_t>(rows_w * K * 2));
    const __amdgpu_buffer_rsrc_t rx = make_rsrc(p.X, static_cast<uint32_t>(p.M * K * 2));

    // This wave's k range: slice s of the row, then part `wave` of the slice.
    const int64_t ks0 = s * kslice;
    const int64_t ks1 = (ks0 + kslice) < K ? (ks0 + kslice) : K;
    const int64_t part = (((ks1 - ks0) + WAVES * 32 - 1) / (WAVES * 32)) * 32;
    const int64_t kw0 = ks0 + wave * part;
    int64_t kw1 = kw0 + part;
    if (kw1 > ks1) kw1 = ks1;

    // Lane l supplies row l % 16 and the 8-wide chunk l / 16 of each step.
    const int r = lane & 15;
    const int chunk = lane >> 4;
    const uint32_t w_row = static_cast<uint32_t>(r * K * 2);
    uint32_t x_row[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) x_row[mb] = static_cast<uint32_t>((mb * 16 + r) * K * 2);

    const int64_t M = p.M;
    const int64_t N = p.N;
    // Output element idx of this strip: token m = idx / 16, row n0 + idx % 16.
    // The residual of this thread's elements is fetched now so its DRAM
    // latency overlaps the W stream (the same thread writes them at the end).
    constexpr int PER_THREAD = (ROWS * MP + THREADS - 1) / THREADS;
    float rpre[PER_THREAD];
#pragma unroll
    for (int t = 0; t < PER_THREAD; ++t) {
        const int idx = threadIdx.x + t * THREADS;
        const int64_t m = idx >> 4;
        const int64_t n = n0 + (idx & 15);
        rpre[t] = (p.R && idx < ROWS * MP && m < M && n < N) ? bf16_to_f32(p.R[m * N + n]) : 0.0f;
    }

    f32x4 acc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};

    // Two register buffers: batch b+1's loads are in flight while batch b is
    // multiplied (the wait before the MFMAs only needs batch b's data).
    // Loads past kw1 are out of range: no traffic, zeros.
    i32x4 wa[U], wb[U];
    i32x4 xa[U][MB], xb[U][MB];
    constexpr int64_t STEP = U * 32;
    issue_batch<MB, U>(wa, xa, rw, rx, w_row, x_row, kw0, kw1, chunk);
    for (int64_t k0 = kw0; k0 < kw1; k0 += 2 * STEP) {
        issue_batch<MB, U>(wb, xb, rw, rx, w_row, x_row, k0 + STEP, kw1, chunk);
        __builtin_amdgcn_sched_barrier(0);
        mfma_batch<MB, U>(acc, wa, xa);
        __builtin_amdgcn_sched_barrier(0);
        if (k0 + STEP >= kw1) break;
        issue_batch<MB, U>(wa, xa, rw, rx, w_row, x_row, k0 + 2 * STEP, kw1, chunk);
        __builtin_amdgcn_sched_barrier(0);
        mfma_batch<MB, U>(acc, wb, xb);
        __builtin_amdgcn_sched_barrier(0);
    }

    // C[n][m] of a 16x16 block: lane l holds n = 4*(l/16) + i, m = l % 16.
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int i = 0; i < 4; ++i) red[wave][4 * (lane >> 4) + i][mb * 16 + (lane & 15)] = acc[mb][i];
    __syncthreads();

    if (split == 1) {
#pragma unroll
        for (int t = 0; t < PER_THREAD; ++t) {
            const int idx = threadIdx.x + t * THREADS;
            const int nl = idx & 15;
            const int m = idx >> 4;
            const int64_t n = n0 + nl;
            if (idx >= ROWS * MP || m >= M || n >= N) continue;
            float y = 0.0f;
#pragma unroll
            for (int w = 0; w < WAVES; ++w) y += red[w][nl][m];
            p.Y[m * N + n] = f32_to_bf16_rne(y + rpre[t]);
        }
        return;
    }

    // Cross-workgroup split: publish this slice's block with device-scope
    // stores (write-through the XCD's L2), count the arrival once they have
    // completed, and let the last arrival read all blocks with device-scope
    // loads (no L2-wide write-back or invalidate needed).
    float *blk = ws + (strip * split + s) * (ROWS * MP);
    for (int idx = threadIdx.x; idx < ROWS * MP; idx += THREADS) {
        const int nl = idx & 15;
        const int m = idx >> 4;
        float y = 0.0f;
#pragma unroll
        for (int w = 0; w < WAVES; ++w) y += red[w][nl][m];
        __hip_atomic_store(blk + idx, y, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __builtin_amdgcn_s_waitcnt(WAITCNT_VM0);   // this wave's block stores are complete
    __syncthreads();
    if (threadIdx.x == 0) {
        const unsigned prev = __hip_atomic_fetch_add(counters + strip, 1u, __ATOMIC_RELAXED,
                                                     __HIP_MEMORY_SCOPE_AGENT);
        is_last = (prev == static_cast<unsigned>(split - 1));
    }
    __syncthreads();
    if (!is_last) return;
    const float *first = ws + strip * split * (ROWS * MP);
#pragma unroll
    for (int t = 0; t < PER_THREAD; ++t) {
        const int idx = threadIdx.x + t * THREADS;
        const int nl = idx & 15;
        const int m = idx >> 4;
        const int64_t n = n0 + nl;
        if (idx >= ROWS * MP || m >= M || n >= N) continue;
        float y = 0.0f;
        for (int sl = 0; sl < split; ++sl)
            y += __hip_atomic_load(first + sl * (ROWS * MP) + idx, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        p.Y[m * N + n] = f32_to_bf16_rne(y + rpre[t]);
    }
    if (threadIdx.x == 0)
        __hip_atomic_store(counters + strip, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int MB>
hipError_t launch_mb(const Problem &p, int split, const Workspace *ws, hipStream_t s) {
    const int64_t strips = (p.N + ROWS - 1) / ROWS;
    const int64_t kslice = ((p.K + split - 1) / split + 31) / 32 * 32;
    float *partials = split > 1 ? ws->partials : nullptr;
    unsigned *counters = split > 1 ? ws->counters : nullptr;
    hipLaunchKernelGGL(skinny_kernel<MB>, dim3(static_cast<unsigned>(strips * split)), dim3(THREADS), 0,
                       s, dense_of(p), split, kslice, partials, counters);
    return hipGetLastError();
}

}  // namespace

// Split rule: N/16 strips; add K slices until there are at least 256
// workgroups (one per CU), keeping every wave at >= 8 MFMA steps of work.
int skinny_split_for(int64_t M, int64_t N, int64_t K) {
    (void)M;
    const int64_t strips = (N + ROWS - 1) / ROWS;
    int split = 1;
    while (strips * split < 256 && K / (split * 2) >= WAVES * UNROLL * 32 && split < 16) split *= 2;
    return split;
}

int64_t skinny_workspace_floats(int64_t M, int64_t N, int split) {
    if (split <= 1) return 0;
    const int64_t mp = ((M + 15) / 16) * 16;
    return ((N + ROWS - 1) / ROWS) * split * ROWS * mp;
}

int64_t skinny_counter_count(int64_t N) { return (N + ROWS - 1) / ROWS; }

hipError_t launch_skinny(const Problem &p, int split, const Workspace *ws, hipStream_t s) {
    const int mb = static_cast<int>((p.M + 15) / 16);
    switch (mb) {
        case 1: return launch_mb<1>(p, split, ws, s);
        case 2: return launch_mb<2>(p, split, ws, s);
        case 3: return launch_mb<3>(p, split, ws, s);
        case 4: return launch_mb<4>(p, split, ws, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace kernelarc
