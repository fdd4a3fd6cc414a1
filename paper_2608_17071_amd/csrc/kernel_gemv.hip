// GEMV kernel for M <= 4 tokens: Y = alpha X W^T (+ beta R) (+ bias) as a
// pure stream over W.
//
// With one to four tokens the multiply is negligible and the time is the
// single pass over W (N*K*2 bytes).  The measured best way to stream HBM on
// MI355X is one contiguous kilobyte per wave instruction, so here every load
// instruction reads 512 consecutive k of ONE weight row (16 bytes per lane);
// the 16-row fragments an MFMA needs would scatter each instruction over 16
// rows.  The dot products run on the VALU with v_dot2_f32_bf16 (bf16 pairs,
// fp32 accumulation) -- at M <= 4 that is a few percent of the VALU's rate.
//
//   * X (M rows of K, each row padded to whole kilobytes in LDS, at most
//     64 KB) is copied to LDS once per workgroup with LDS-direct loads (1 KB
//     each, all in flight together, and in flight together with the first
//     batch of weight loads); lane l reads the 8 values of X that face its
//     16 bytes of W.
//   * a wave owns RPW consecutive rows and walks them k-segment by
//     k-segment (all rows of a segment share one read of X from LDS), two
//     batches of BATCH loads in flight;
//   * per row and token the 64 lane partials are added by a fixed xor
//     butterfly, then one lane adds fp32(R) and rounds once to bf16.  The
//     residual is fetched at kernel start (from an empty resource when there
//     is none, so the load needs no branch and nothing waits for it until
//     the end).  Y may alias R.
#include "internal.h"

namespace kernelarc {
namespace {

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int RSRC_WORD3 = 0x00020000;
constexpr uint32_t OOB_OFFSET = 0x80000000u;
constexpr int AUX_NT = 2;
constexpr int WAVES = 4;
constexpr int THREADS = 64 * WAVES;
constexpr int BATCH = 4;                 // loads per batch (one kilobyte each)
constexpr int WAITCNT_VM_BATCH = 0x0F70 | BATCH;   // s_waitcnt vmcnt(BATCH)
constexpr int MAX_ROWS_PER_WAVE = 4;     // a batch must hold whole segments
constexpr int X_LDS_BYTES = 64 * 1024;   // X lives in LDS: M rows of x_pitch(K) bytes

// LDS bytes of one row of X: K * 2 rounded up to whole 1 KB loads.
__host__ __device__ inline int64_t x_pitch(int64_t K) { return (K * 2 + 1023) / 1024 * 1024; }

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), static_cast<short>(0),
                                             static_cast<int>(bytes), RSRC_WORD3);
}

// acc + sum of the 8 products of two rows of 8 bf16 (each int holds a pair).
// The four pairs are named members on purpose: a loop subscripting the
// vector inside __builtin_bit_cast was lowered to four uses of element 0.
__device__ __forceinline__ float dot2(int w, int x, float acc) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), __builtin_bit_cast(bf16x2, x), acc,
                                           false);
}

__device__ __forceinline__ float dot8(i32x4 w, i32x4 x, float acc) {
    acc = dot2(w.x, x.x, acc);
    acc = dot2(w.y, x.y, acc);
    acc = dot2(w.z, x.z, acc);
    acc = dot2(w.w, x.w, acc);
    return acc;
}

// Sum over the 64 lanes of a wave, in a fixed butterfly order.
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

// P = Problem: the general form (row strides, alpha, beta, bias);
// P = DenseProblem: dense operands, the residual added as is (the plain
// operator).
template <int MT, int RPW, class P>
__global__ __launch_bounds__(THREADS) void gemv_kernel(P p) {
    constexpr bool GEN = std::is_same<P, Problem>::value;
    extern __shared__ __attribute__((aligned(16))) char xs[];   // X, M * K * 2 bytes

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t K = p.K;
    const int64_t N = p.N;
    const int64_t row0 = (static_cast<int64_t>(blockIdx.x) * WAVES + wave) * RPW;
    const int segs = static_cast<int>((K + 511) / 512);

    // Residual of the outputs this wave writes: lane t * RPW + r owns row
    // row0 + r of token t.
    const int my_t = lane / RPW;
    const int my_r = lane % RPW;
    const bool writer = my_t < MT && my_t < p.M && row0 + my_r < N;
    const int64_t ldx = ldx_of(p), ldw = ldw_of(p), ldr = ldr_of(p), ldy = ldy_of(p);
    const uint32_t r_off = writer ? static_cast<uint32_t>((my_t * ldr + row0 + my_r) * 2) : OOB_OFFSET;
    const __amdgpu_buffer_rsrc_t rr = make_rsrc(
        p.R ? p.R : p.Y, p.R ? static_cast<uint32_t>(GEN ? strided_bytes(p.M, N, ldr) : p.M * N * 2) : 0u);
    const uint16_t rbits = __builtin_amdgcn_raw_buffer_load_b16(rr, r_off, 0, 0);
    uint16_t bbits = 0;
    if constexpr (GEN) {
        const __amdgpu_buffer_rsrc_t rbias =
            make_rsrc(bias_of(p) ? bias_of(p) : p.Y, bias_of(p) ? static_cast<uint32_t>(N * 2) : 0u);
        bbits = __builtin_amdgcn_raw_buffer_load_b16(rbias, writer ? static_cast<uint32_t>((row0 + my_r) * 2) : OOB_OFFSET, 0, 0);
    }

    // X -> LDS: every wave issues its share of the 1 KB LDS-direct loads
    // (row t of X goes to xs + t * x_pitch(K); a row's tail past K reads
    // zero), then one wait and one barrier.
    const int64_t xp = GEN ? x_pitch(K) : K * 2;
    if constexpr (GEN) {
        const int per_row = static_cast<int>(xp / 1024);
        for (int t = 0; t < p.M; ++t) {
            const __amdgpu_buffer_rsrc_t rxs = make_rsrc(p.X + t * ldx, static_cast<uint32_t>(K * 2));
            for (int c = wave; c < per_row; c += WAVES)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rxs, (lds_void *)(xs + t * xp + c * 1024), 16,
                                                         static_cast<uint32_t>(c * 1024 + lane * 16), 0, 0, 0);
        }
    } else {
        // dense X: M*K*2 contiguous bytes, the tail past it reads zero
        const uint32_t xbytes = static_cast<uint32_t>(p.M * K * 2);
        const __amdgpu_buffer_rsrc_t rxs = make_rsrc(p.X, xbytes);
        const int xloads = static_cast<int>((xbytes + 1023) / 1024);
        for (int q = wave; q < xloads; q += WAVES)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rxs, (lds_void *)(xs + q * 1024), 16,
                                                     static_cast<uint32_t>(q * 1024 + lane * 16), 0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);

    const __amdgpu_buffer_rsrc_t rw = make_rsrc(p.W, static_cast<uint32_t>(GEN ? strided_bytes(N, K, ldw) : N * K * 2));
    float acc[RPW][MT];
#pragma unroll
    for (int r = 0; r < RPW; ++r)
#pragma unroll
        for (int t = 0; t < MT; ++t) acc[r][t] = 0.0f;

    // The wave's loads, segment-major: a batch holds SPB segments of all RPW
    // rows; load b of a batch is segment b / RPW, row b % RPW.
    static_assert(RPW >= 1 && BATCH % RPW == 0, "a batch holds whole segments (SPB >= 1)");
    constexpr int SPB = BATCH / RPW;
    auto issue = [&](i32x4 (&wv)[BATCH], int seg0) {
#pragma unroll
        for (int b = 0; b < BATCH; ++b) {
            const int64_t k = static_cast<int64_t>(seg0 + b / RPW) * 512 + lane * 8;
            const int64_t row = row0 + b % RPW;
            const uint32_t off = (row < N && k < K) ? static_cast<uint32_t>(row * ldw * 2 + k * 2) : OOB_OFFSET;
            wv[b] = __builtin_amdgcn_raw_buffer_load_b128(rw, off, 0, AUX_NT);
        }
    };
    auto consume = [&](const i32x4 (&wv)[BATCH], int seg0) {
        // Exactly one later batch has been issued: wait for this one as a
        // whole.  No branches (segments past K and tokens past M read a
        // valid LDS address and multiply zeros).
        __builtin_amdgcn_s_waitcnt(WAITCNT_VM_BATCH);
#pragma unroll
        for (int sb = 0; sb < SPB; ++sb) {
            const int64_t k = static_cast<int64_t>(seg0 + sb) * 512 + lane * 8;
            const bool k_ok = k < K;
#pragma unroll
            for (int t = 0; t < MT; ++t) {
                const bool ok = k_ok && t < p.M;
                const int tt = t < p.M ? t : 0;
                const i32x4 xr = *reinterpret_cast<const i32x4 *>(xs + tt * xp + (k_ok ? k : 0) * 2);
                const i32x4 xv = ok ? xr : i32x4{0, 0, 0, 0};
#pragma unroll
                for (int r = 0; r < RPW; ++r) acc[r][t] = dot8(wv[sb * RPW + r], xv, acc[r][t]);
            }
        }
    };

    // The first weight batch goes out before X has landed, so the two
    // round trips overlap.  Loads complete in issue order: once at most
    // that batch is outstanding, this wave's X loads (and the residual) are
    // in LDS; the barrier then covers every wave's.  (__syncthreads() would
    // wait for the weight batch too.)
    i32x4 wa[BATCH], wb[BATCH];
    issue(wa, 0);
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_waitcnt vmcnt(%0)\n\ts_barrier" ::"n"(BATCH) : "memory");
    __builtin_amdgcn_sched_barrier(0);
    // (With the exit below the compiler waits for every load at the head
    // of the loop; a loop without it, consuming batches in pairs past K,
    // keeps two batches in flight but measured slower on M = 1 shapes.)
    for (int s0 = 0; s0 < segs; s0 += 2 * SPB) {
        issue(wb, s0 + SPB);
        __builtin_amdgcn_sched_barrier(0);
        consume(wa, s0);
        __builtin_amdgcn_sched_barrier(0);
        if (s0 + SPB >= segs) break;
        issue(wa, s0 + 2 * SPB);
        __builtin_amdgcn_sched_barrier(0);
        consume(wb, s0 + SPB);
        __builtin_amdgcn_sched_barrier(0);
    }

    // Lane-sum every (row, token); lane t * RPW + r keeps its own.
    float mine = 0.0f;
#pragma unroll
    for (int r = 0; r < RPW; ++r)
#pragma unroll
        for (int t = 0; t < MT; ++t) {
            const float v = wave_sum(acc[r][t]);
            if (lane == t * RPW + r) mine = v;
        }
    if (writer) {
        float y;
        if constexpr (GEN) {
            y = combine(mine, bf16_to_f32(rbits), p.R != nullptr, alpha_of(p), beta_of(p));
            if (bias_of(p)) y += bf16_to_f32(bbits);
        } else {
            y = mine;
            if (p.R) y += bf16_to_f32(rbits);
        }
        p.Y[my_t * ldy + row0 + my_r] = f32_to_bf16_rne(y);
    }
}

template <int MT, class P>
hipError_t launch_mt(const P &p, int rpw, hipStream_t s) {
    constexpr bool GEN = std::is_same<P, Problem>::value;
    const int64_t rows_per_wg = static_cast<int64_t>(rpw) * WAVES;
    const dim3 grid(static_cast<unsigned>((p.N + rows_per_wg - 1) / rows_per_wg));
    // whole 1 KB loads per row (general form) or over the dense X
    const size_t lds = static_cast<size_t>(GEN ? p.M * x_pitch(p.K) : (p.M * p.K * 2 + 1023) / 1024 * 1024);
    switch (rpw) {
        case 1: hipLaunchKernelGGL((gemv_kernel<MT, 1, P>), grid, dim3(THREADS), lds, s, p); break;
        case 2: hipLaunchKernelGGL((gemv_kernel<MT, 2, P>), grid, dim3(THREADS), lds, s, p); break;
        case 4: hipLaunchKernelGGL((gemv_kernel<MT, 4, P>), grid, dim3(THREADS), lds, s, p); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <int MT>
hipError_t launch_mt(const Problem &p, int rpw, hipStream_t s) {
    return is_general(p) ? launch_mt<MT, Problem>(p, rpw, s) : launch_mt<MT, DenseProblem>(dense_of(p), rpw, s);
}

}  // namespace

int gemv_rows_per_wave(int64_t M, int64_t N, int64_t K) {
    (void)M;
    (void)K;
    // One row per wave up to 8192 rows (measured best: many short streams),
    // then 2 or 4 (a power of two dividing the batch).
    int rpw = 1;
    while (rpw < MAX_ROWS_PER_WAVE && static_cast<int64_t>(rpw) * 8192 < N) rpw *= 2;
    return rpw;
}

bool gemv_fits(int64_t M, int64_t N, int64_t K, int64_t ldw) {
    return M >= 1 && M <= 4 && K % 8 == 0 && M * x_pitch(K) <= X_LDS_BYTES &&
           strided_bytes(N, K, ldw) < (int64_t{1} << 31);
}

hipError_t launch_gemv(const Problem &p, hipStream_t s) {
    const int rpw = gemv_rows_per_wave(p.M, p.N, p.K);
    switch (p.M) {
        case 1: return launch_mt<1>(p, rpw, s);
        case 2: return launch_mt<2>(p, rpw, s);
        case 3: return launch_mt<3>(p, rpw, s);
        case 4: return launch_mt<4>(p, rpw, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace kernelarc
