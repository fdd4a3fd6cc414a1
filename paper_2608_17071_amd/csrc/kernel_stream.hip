// Streaming MFMA kernel for few rows (M <= 64): Y = X W^T (+ R) as one pass
// over the weight (also the general form: row strides, alpha, beta, bias).
//
// With at most 64 rows of X the work is bound by reading W (N*K*2 bytes)
// from HBM, and the time a load takes to come back (microseconds under load)
// decides the rate unless each CU keeps several tens of kilobytes in flight.
// The tile kernels synchronise their waves at every K step; here no wave
// ever waits for another inside the K loop:
//   * a workgroup of 4 waves owns one block of ROWS = 16, 32 or 64 rows of
//     W and one K slice; each wave takes a contiguous quarter of the
//     slice's BK steps and runs its own pipeline;
//   * W goes through LDS-direct loads into the wave's private ring of
//     STAGES buffers (ROWS rows x BK, 16-byte chunk c of row r at slot
//     c ^ swz(r)), requested STAGES-1 steps ahead; one load instruction
//     reads 64/(BK/8) whole row segments of BK*2 contiguous bytes, and the
//     wave's own vmcnt says when a buffer has landed;
//   * X (at most 64 rows, L2-resident after first use) is staged in the
//     same ring beside W (16- and 32-row blocks) or read straight into
//     MFMA A fragments one step ahead (64-row blocks);
//   * v_mfma_f32_16x16x32_bf16 with A = 16 rows of X x 32 k and B = 16 rows
//     of W x 32 k: MB = ceil(M/16) x ROWS/16 blocks per 32-k step, fp32
//     accumulation in K order.
// Fewer rows per workgroup give more workgroups without a K split (16-row
// blocks: one workgroup per CU at N = 4096 and no cross-workgroup hand-off)
// at the price of reading X once per 16 rows of W instead of once per 64;
// X is small and stays in L2.
// INT8 operands (16- and 32-row blocks only): a stage holds the same bytes,
// i.e. twice the K elements, v_mfma_i32_16x16x64_i8 takes the same 16 bytes
// per lane as the bf16 16x16x32 form and accumulates exactly in int32 (the
// wave and split-K partials are added as integers), and the epilogue
// multiplies by the row and column scales before adding R.
// After the loop the four wave partials are added in LDS in wave order; a
// split of K across workgroups goes through the fp32 workspace, where the
// last workgroup of a row block adds the slices in slice order.  The
// epilogue adds fp32(R) (the general form: alpha*acc + beta*R + bias) and
// rounds once to bf16; each output element is read (R) and written (Y) by
// one lane, so Y may alias R.
#include "internal.h"

namespace kernelarc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int RSRC_WORD3 = 0x00020000;
constexpr uint32_t OOB_OFFSET = 0x80000000u;
constexpr int AUX_SC1 = 16;   // device-scope (cross-XCD coherent) access
constexpr int AUX_NT = 2;     // non-temporal: each weight byte is read once
constexpr int WAVES = 4;
constexpr int THREADS = 64 * WAVES;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), static_cast<short>(0),
                                             static_cast<int>(bytes), RSRC_WORD3);
}

constexpr int waitcnt_vm(int n) { return (n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8); }

// Slot of 16-byte chunk c of row r is c ^ swz(r); a fragment read (16
// consecutive rows at one chunk) then touches 16 distinct bank groups.
template <int CHUNKS>
__device__ __forceinline__ int swz(int r) {
    if constexpr (CHUNKS == 16) return r & 15;
    else return (r & 7) ^ ((r >> 3) & 1);
}

struct StreamSplit {
    int split;          // K slices per row block (1: none)
    int64_t kslice;     // slice length, a multiple of BK
    float *partials;    // [row block][slice][wave][token block][lane] f32x4
    unsigned *counters; // one arrival counter per row block, zero between calls
};

// RB 16-row blocks of W per workgroup.
// X path: with RB = 4 the X fragments go straight from L2 into registers one
// step ahead.  Loads complete in issue order, so waiting for step t+1's X
// (issued after step t+PF-1's W) also waits for that W: a deeper W ring
// would buy nothing, and these configurations keep PF = 1.  With RB < 4
// each stage holds the step's 16*MB rows of X after its W rows, both moved
// by LDS-direct loads; every load of a wave is then counted in stage order
// and the ring is as deep as asked, capped by the vmcnt range and by LDS.
template <int MB, int BK, int STAGES_, int RB_>
struct StreamCfg {
    static constexpr int RB = RB_, ROWS = 16 * RB;
    static constexpr bool XL = RB < 4;                    // X staged through LDS
    static constexpr int CHUNKS = BK / 8, ROW_BYTES = BK * 2, RPI = 64 / CHUNKS;
    static constexpr int W_BYTES = ROWS * ROW_BYTES;
    static constexpr int X_BYTES = XL ? 16 * MB * ROW_BYTES : 0;
    static constexpr int STAGE_BYTES = W_BYTES + X_BYTES;
    static constexpr int W_LOADS = W_BYTES / 1024;       // load instructions per stage
    static constexpr int KS = BK / 32;                    // MFMA k steps per stage
    static constexpr int X_LOADS = XL ? X_BYTES / 1024 : MB * KS;
    static constexpr int PF_VM = 63 / (W_LOADS + X_LOADS);
    static constexpr int ST_LDS = 160 * 1024 / (WAVES * STAGE_BYTES);
    static constexpr int ST_CAP = PF_VM + 1 < ST_LDS ? PF_VM + 1 : ST_LDS;
    static constexpr int STAGES = STAGES_ < ST_CAP ? STAGES_ : ST_CAP;   // per-wave buffers
    static constexpr int PF = STAGES - 1;                 // steps requested ahead
    static constexpr int WAVE_BYTES = STAGES * STAGE_BYTES;
    static constexpr int LDS_BYTES = WAVES * WAVE_BYTES;
    static constexpr int RED_BYTES = WAVES * MB * RB * 64 * 16;   // wave partials, f32x4 per lane
    // After the wave partials are added, wave w writes row block OWN_J(w)
    // and the EPW accumulator values [e0, e0 + EPW) of each lane's f32x4.
    static constexpr int EPW = RB;
    static_assert(RB == 1 || RB == 2 || RB == 4, "row blocks");
    static_assert(W_BYTES % 1024 == 0 && X_BYTES % 1024 == 0, "whole load instructions per stage");
    static_assert(XL || STAGES == 2, "register X path: one step ahead");
    static_assert(BK == 64 || BK == 128, "BK");
    static_assert(MB >= 1 && MB <= 4, "token blocks");
    static_assert(RED_BYTES <= LDS_BYTES, "reduction fits in the stage buffers");
    static_assert(LDS_BYTES <= 160 * 1024, "LDS capacity");
    static_assert(STAGES >= 2 && PF * (W_LOADS + X_LOADS) < 64, "vmcnt range");
};

// P = DenseProblem (bf16, the plain operator), Problem (bf16, the general
// form: row strides, alpha, beta, bias) or I8Problem (int8 with scales).
template <int MB, int BK, int STAGES, int RB, class P>
__global__ __launch_bounds__(THREADS) void stream_kernel(P p, int64_t nblocks, StreamSplit sk) {
    using C = StreamCfg<MB, BK, STAGES, RB>;
    constexpr bool I8 = std::is_same<P, I8Problem>::value;
    constexpr bool GEN = std::is_same<P, Problem>::value;
    const int64_t ldx = ldx_of(p), ldw = ldw_of(p), ldr = ldr_of(p), ldy = ldy_of(p);
    static_assert(!I8 || C::XL, "INT8 operands take the LDS-staged X path");
    constexpr int EB = I8 ? 1 : 2;                 // bytes per operand element
    constexpr int BKE = C::ROW_BYTES / EB;         // K elements per stage
    constexpr int CKE = 16 / EB;                   // K elements per 16-byte chunk
    using AccV = typename std::conditional<I8, i32x4, f32x4>::type;
    __shared__ __attribute__((aligned(1024))) char lds[C::LDS_BYTES];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int64_t nb = blockIdx.x % nblocks;
    const int64_t slice = blockIdx.x / nblocks;
    const int64_t n0 = nb * C::ROWS;
    // Outputs this wave writes after the reduction: row block j_own, values
    // [e0, e0 + EPW) of each f32x4.
    const int j_own = wave * RB / WAVES;
    const int e0 = (wave % (WAVES / RB)) * RB;
    const int64_t K = p.K;

    // K range of the workgroup, then of this wave (a quarter of its steps).
    const int64_t kbeg = slice * sk.kslice;
    const int64_t kend = (kbeg + sk.kslice) < K ? (kbeg + sk.kslice) : K;
    const int64_t steps = kend > kbeg ? (kend - kbeg + BKE - 1) / BKE : 0;
    const int64_t step0 = kbeg / BKE + steps * wave / WAVES;
    const int nsteps = static_cast<int>(steps * (wave + 1) / WAVES - steps * wave / WAVES);

    // Residual of the outputs of this lane's row block in the epilogue
    // (all four values; the wave writes EPW of them): fetched now, so its
    // latency hides under the K loop.  Every element is read here before any lane writes
    // Y, so Y may alias R.
    const int64_t N = p.N;
    const __amdgpu_buffer_rsrc_t ry = make_rsrc(p.Y, static_cast<uint32_t>(strided_bytes(p.M, N, ldy)));
    // Without a residual the R resource is empty: its loads read zero.
    const __amdgpu_buffer_rsrc_t rr =
        make_rsrc(p.R ? p.R : p.Y, p.R ? static_cast<uint32_t>(strided_bytes(p.M, N, ldr)) : 0u);
    const int64_t n_out = n0 + 16 * j_own + (lane & 15);
    // Offsets of output (16i + 4*(l/16) + e, n_out) in Y and R: rows past M
    // fall outside the resources; a column past N is pointed out of range.
    // Computed without branches so the loads below issue back to back.
    const bool col_ok = n_out < N;
    auto out_off = [&](int64_t ld, int i, int e) {
        const uint32_t off = static_cast<uint32_t>(((16 * i + 4 * (lane >> 4) + e) * ld + n_out) * 2);
        return col_ok ? off : OOB_OFFSET;
    };
    uint16_t rres[MB][4];
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) rres[i][e] = __builtin_amdgcn_raw_buffer_load_b16(rr, out_off(ldr, i, e), 0, 0);
    // General form: the bias of the lane's output column.
    [[maybe_unused]] float bias_v = 0.0f;
    if constexpr (GEN) {
        if (p.bias)
            bias_v = bf16_to_f32(__builtin_amdgcn_raw_buffer_load_b16(
                make_rsrc(p.bias, static_cast<uint32_t>(N * 2)), col_ok ? static_cast<uint32_t>(n_out * 2) : OOB_OFFSET,
                0, 0));
    }
    // INT8: the column scale of the lane's output column and the row
    // scales of its rows, requested with R.
    [[maybe_unused]] float scw = 0.0f, scx[MB][4];
    if constexpr (I8) {
        const __amdgpu_buffer_rsrc_t rsw = make_rsrc(p.sw, static_cast<uint32_t>(N * 4));
        const __amdgpu_buffer_rsrc_t rsx = make_rsrc(p.sx, static_cast<uint32_t>(p.M * 4));
        scw = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                            rsw, col_ok ? static_cast<uint32_t>(n_out * 4) : OOB_OFFSET, 0, 0));
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
            for (int e = 0; e < 4; ++e)
                scx[i][e] = __builtin_bit_cast(
                    float, __builtin_amdgcn_raw_buffer_load_b32(
                               rsx, static_cast<uint32_t>((16 * i + 4 * (lane >> 4) + e) * 4), 0, 0));
    }

    const int64_t rows_w = (p.N - n0) < C::ROWS ? (p.N - n0) : C::ROWS;
    const __amdgpu_buffer_rsrc_t rw =
        make_rsrc(p.W + n0 * ldw, static_cast<uint32_t>(GEN ? strided_bytes(rows_w, K, ldw) : rows_w * K * EB));
    const __amdgpu_buffer_rsrc_t rx =
        make_rsrc(p.X, static_cast<uint32_t>(GEN ? strided_bytes(p.M, K, ldx) : p.M * K * EB));

    // W staging map: lane l of load q fills slot l % CHUNKS of row
    // RPI*q + l / CHUNKS with global chunk slot ^ swz(row).
    uint32_t w_off[C::W_LOADS];
    int w_k[C::W_LOADS];
#pragma unroll
    for (int q = 0; q < C::W_LOADS; ++q) {
        const int r = q * C::RPI + lane / C::CHUNKS;
        const int c = (lane % C::CHUNKS) ^ swz<C::CHUNKS>(r);
        w_off[q] = static_cast<uint32_t>(r * ldw * EB + c * 16);
        w_k[q] = c * CKE;
    }
    // X staging map (RB < 4), the same map over the 16*MB rows of X (rows
    // past M fall outside the resource and read zero).
    uint32_t x_off[C::XL ? C::X_LOADS : 1];
    int x_kc[C::XL ? C::X_LOADS : 1];
    if constexpr (C::XL) {
#pragma unroll
        for (int q = 0; q < C::X_LOADS; ++q) {
            const int r = q * C::RPI + lane / C::CHUNKS;
            const int c = (lane % C::CHUNKS) ^ swz<C::CHUNKS>(r);
            x_off[q] = static_cast<uint32_t>(r * ldx * EB + c * 16);
            x_kc[q] = c * CKE;
        }
    }
    // A fragment of token block i at k step s (register path): token
    // 16i + l % 16, k chunk 4s + l / 16 of the stage.
    const uint32_t x_row = static_cast<uint32_t>((lane & 15) * ldx * 2);
    const int x_k = 8 * (lane >> 4);
    char *ring = lds + wave * C::WAVE_BYTES;

    // Loads of one step: chunks at or past the end of the wave's range
    // (rem = k values left in the step, 0 for a step past the range) are
    // pointed out of range; they move no data and only complete in order.
    auto rem_of = [&](int64_t step, bool valid) {
        const int64_t left = kend - step * BKE;
        return valid ? static_cast<int>(left < BKE ? left : BKE) : 0;
    };
    auto issue_w = [&](int buf, int64_t step, int rem) {
        const uint32_t kb2 = static_cast<uint32_t>(step * C::ROW_BYTES);
#pragma unroll
        for (int q = 0; q < C::W_LOADS; ++q) {
            const uint32_t off = w_k[q] < rem ? w_off[q] + kb2 : OOB_OFFSET;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_void *)(ring + buf * C::STAGE_BYTES + q * 1024), 16,
                                                     off, 0, 0, AUX_NT);
        }
        if constexpr (C::XL) {
#pragma unroll
            for (int q = 0; q < C::X_LOADS; ++q) {
                const uint32_t off = x_kc[q] < rem ? x_off[q] + kb2 : OOB_OFFSET;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rx, (lds_void *)(ring + buf * C::STAGE_BYTES + C::W_BYTES + q * 1024), 16, off, 0, 0, 0);
            }
        }
    };
    // X fragments of sub-step s of a step, token blocks 0..MB-1.
    auto issue_x = [&](bf16x8 (&xs)[MB], int64_t step, int s, int rem) {
        const int kr = 32 * s + x_k;
        const uint32_t base = x_row + static_cast<uint32_t>((step * BK + kr) * 2);
#pragma unroll
        for (int i = 0; i < MB; ++i) {
            const uint32_t off = kr < rem ? base + static_cast<uint32_t>(16 * i * ldx * 2) : OOB_OFFSET;
            xs[i] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rx, off, 0, 0));
        }
    };

    AccV acc[MB][RB];
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < RB; ++j) acc[i][j] = AccV{0, 0, 0, 0};

    // B fragment of row block j at k step s: row 16j + l % 16, chunk
    // 4s + l / 16.
    const int frag_row = lane & 15;
    const int frag_hi = lane >> 4;

    // Pipeline: step t's W is in buffer t % STAGES, requested PF = STAGES-1
    // steps ahead (iteration t requests step t+PF into the buffer that step
    // t-1 used); X sub-step s of step t+1 is loaded into the registers of
    // sub-step s of step t as soon as those have been multiplied (one step
    // of lookahead).  Steps past the wave's range load nothing (out of
    // range) and only keep the vmcnt bookkeeping uniform.  The waits count
    // loads in issue order, so every W issue is fenced with scheduling
    // barriers: no X load may be moved ahead of the W loads it is counted
    // after.
    // With X through LDS (RB < 4) the stage loads are the wave's only
    // loads in the loop: after step t's come exactly those of steps
    // t+1 .. t+PF, in the prologue as in the steady state.
    bf16x8 xf[C::KS][MB];
    if (nsteps > 0) {
#pragma unroll
        for (int u = 0; u < C::PF; ++u) issue_w(u, step0 + u, rem_of(step0 + u, u < nsteps));
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (!C::XL) {
            const int rem0 = rem_of(step0, true);
#pragma unroll
            for (int s = 0; s < C::KS; ++s) issue_x(xf[s], step0, s, rem0);
        }
    }
    int buf = 0;
    for (int t = 0; t < nsteps; ++t) {
        const int64_t step = step0 + t;
        const int pbuf = buf == 0 ? C::STAGES - 1 : buf - 1;   // the buffer step t-1 used
        __builtin_amdgcn_sched_barrier(0);
        issue_w(pbuf, step + C::PF, rem_of(step + C::PF, t + C::PF < nsteps));
        __builtin_amdgcn_sched_barrier(0);
        const int rem1 = rem_of(step + 1, t + 1 < nsteps);
        // Step t's loads have landed once only what was issued after them
        // may be outstanding: the stages of steps t+1 .. t+PF (X through
        // LDS), or the W of step t+1 and the X of step t (register X path,
        // PF = 1: one X set per iteration, after that iteration's W).
        __builtin_amdgcn_s_waitcnt(waitcnt_vm(C::PF * (C::W_LOADS + C::X_LOADS)));
        __builtin_amdgcn_sched_barrier(0);
        const char *base = ring + buf * C::STAGE_BYTES + frag_row * C::ROW_BYTES;
#pragma unroll
        for (int s = 0; s < C::KS; ++s) {
            bf16x8 wf[RB];
#pragma unroll
            for (int j = 0; j < RB; ++j) {
                const int slot = (4 * s + frag_hi) ^ swz<C::CHUNKS>(16 * j + frag_row);
                wf[j] = *reinterpret_cast<const bf16x8 *>(base + 16 * j * C::ROW_BYTES + slot * 16);
            }
            if constexpr (C::XL) {
#pragma unroll
                for (int i = 0; i < MB; ++i) {
                    const int slot = (4 * s + frag_hi) ^ swz<C::CHUNKS>(16 * i + frag_row);
                    xf[s][i] = *reinterpret_cast<const bf16x8 *>(base + C::W_BYTES + 16 * i * C::ROW_BYTES +
                                                                 slot * 16);
                }
            }
#pragma unroll
            for (int i = 0; i < MB; ++i)
#pragma unroll
                for (int j = 0; j < RB; ++j) {
                    if constexpr (I8)
                        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4, xf[s][i]),
                                                                          __builtin_bit_cast(i32x4, wf[j]),
                                                                          acc[i][j], 0, 0, 0);
                    else
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xf[s][i], wf[j], acc[i][j], 0, 0, 0);
                }
            if constexpr (!C::XL) issue_x(xf[s], step + 1, s, rem1);
        }
        buf = buf + 1 == C::STAGES ? 0 : buf + 1;
    }

    // Add the four wave partials in LDS (wave order).  Wave w then holds
    // row block j_own of every token block.
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    __syncthreads();
    AccV *red = reinterpret_cast<AccV *>(lds);
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < RB; ++j) red[((wave * MB + i) * RB + j) * 64 + lane] = acc[i][j];
    __syncthreads();
    AccV sum[MB];
#pragma unroll
    for (int i = 0; i < MB; ++i) {
        sum[i] = red[((0 * MB + i) * RB + j_own) * 64 + lane];
#pragma unroll
        for (int w = 1; w < WAVES; ++w) sum[i] += red[((w * MB + i) * RB + j_own) * 64 + lane];
    }

    if (sk.split > 1) {
        // Publish this slice with device-scope stores; once every wave's
        // stores have completed the arrival is counted, and the last slice
        // to arrive adds all slices (device-scope loads) in slice order.
        // A slice holds one copy of the workgroup's sums: wave w stores and
        // later reads back only the EPW values of each f32x4 that it writes
        // to Y (all four with 64-row blocks, one with 16-row blocks).
        constexpr int EPW = C::EPW, CH = 4 / EPW;
        constexpr int BLOCK_FLOATS = MB * RB * 64 * 4;
        const float *first = sk.partials + nb * sk.split * BLOCK_FLOATS;
        const __amdgpu_buffer_rsrc_t rp = make_rsrc(first, static_cast<uint32_t>(sk.split) * BLOCK_FLOATS * 4u);
        const uint32_t mine = static_cast<uint32_t>(slice) * BLOCK_FLOATS * 4u;
        const int c_own = e0 / EPW;
        auto part_off = [&](int i) {
            return static_cast<uint32_t>((((i * RB + j_own) * CH + c_own) * 64 + lane) * EPW * 4);
        };
        using E = typename std::conditional<I8, int, float>::type;
        using B64 = decltype(__builtin_amdgcn_raw_buffer_load_b64(rp, 0u, 0, 0));
        static_assert(sizeof(B64) == 8, "64-bit buffer access");
#pragma unroll
        for (int i = 0; i < MB; ++i) {
            if constexpr (EPW == 4) {
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, sum[i]), rp, mine + part_off(i), 0,
                                                       AUX_SC1);
            } else if constexpr (EPW == 2) {
                const i32x2 v = {__builtin_bit_cast(int, static_cast<E>(sum[i][e0])),
                                 __builtin_bit_cast(int, static_cast<E>(sum[i][e0 + 1]))};
                __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(B64, v), rp, mine + part_off(i), 0, AUX_SC1);
            } else {
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, static_cast<E>(sum[i][e0])), rp,
                                                      mine + part_off(i), 0, AUX_SC1);
            }
        }
        __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
        __syncthreads();
        int *flag = reinterpret_cast<int *>(lds);   // every wave has read its sums (barrier above)
        if (threadIdx.x == 0) {
            const unsigned prev =
                __hip_atomic_fetch_add(sk.counters + nb, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            *flag = prev == static_cast<unsigned>(sk.split - 1);
        }
        __syncthreads();
        const bool last = *flag != 0;
        if (!last) return;
        // Eight slices per round trip; a slice past the last reads out of
        // range and is not added, so the sum runs over the slices in order.
        E tot[MB][EPW];
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
            for (int k = 0; k < EPW; ++k) tot[i][k] = 0;
        constexpr int D = 8;
        for (int t0 = 0; t0 < sk.split; t0 += D) {
            E v[D][MB][EPW];
#pragma unroll
            for (int d = 0; d < D; ++d)
#pragma unroll
                for (int i = 0; i < MB; ++i) {
                    const uint32_t off = static_cast<uint32_t>(t0 + d) * BLOCK_FLOATS * 4u + part_off(i);
                    if constexpr (EPW == 4) {
                        const i32x4 w = __builtin_amdgcn_raw_buffer_load_b128(rp, off, 0, AUX_SC1);
#pragma unroll
                        for (int k = 0; k < 4; ++k) v[d][i][k] = __builtin_bit_cast(E, static_cast<int>(w[k]));
                    } else if constexpr (EPW == 2) {
                        // Vector elements go through a value (static_cast) before
                        // __builtin_bit_cast: applied to an element of a vector
                        // lvalue, it reads the vector's first element instead.
                        const i32x2 w = __builtin_bit_cast(i32x2, __builtin_amdgcn_raw_buffer_load_b64(rp, off, 0, AUX_SC1));
                        v[d][i][0] = __builtin_bit_cast(E, static_cast<int>(w[0]));
                        v[d][i][1] = __builtin_bit_cast(E, static_cast<int>(w[1]));
                    } else {
                        v[d][i][0] = __builtin_bit_cast(E, __builtin_amdgcn_raw_buffer_load_b32(rp, off, 0, AUX_SC1));
                    }
                }
#pragma unroll
            for (int d = 0; d < D; ++d) {
                if (t0 + d >= sk.split) break;
#pragma unroll
                for (int i = 0; i < MB; ++i)
#pragma unroll
                    for (int k = 0; k < EPW; ++k) tot[i][k] += v[d][i][k];
            }
        }
#pragma unroll
        for (int i = 0; i < MB; ++i)
#pragma unroll
            for (int k = 0; k < EPW; ++k) sum[i][e0 + k] = tot[i][k];
        if (threadIdx.x == 0)
            __hip_atomic_store(sk.counters + nb, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }

    // Epilogue: sum[i][e] is Y[16i + 4*(l/16) + e][n0 + 16*j_own + l%16].
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if (RB < WAVES && (e < e0 || e >= e0 + C::EPW)) continue;   // another wave's value
            float y;
            if constexpr (I8) y = static_cast<float>(sum[i][e]) * (scx[i][e] * scw);
            else y = sum[i][e];
            if constexpr (GEN) {
                y = combine(y, bf16_to_f32(rres[i][e]), p.R != nullptr, p.alpha, p.beta);
                if (p.bias) y += bias_v;
            } else if (p.R) {
                y += bf16_to_f32(rres[i][e]);
            }
            __builtin_amdgcn_raw_buffer_store_b16(f32_to_bf16_rne(y), ry, out_off(ldy, i, e), 0, 0);
        }
}

// P: DenseProblem or I8Problem; a K slice is a whole number of stages
// (BK bf16 or 2*BK int8 elements).
template <int MB, int BK, int STAGES, int RB, class P>
hipError_t launch_mb(const P &p, int split, const Workspace *ws, hipStream_t s) {
    constexpr int BKE = std::is_same<P, I8Problem>::value ? 2 * BK : BK;
    const int64_t nblocks = (p.N + 16 * RB - 1) / (16 * RB);
    StreamSplit sk{1, ((p.K + BKE - 1) / BKE) * BKE, nullptr, nullptr};
    if (split > 1) {
        sk.split = split;
        sk.kslice = (((p.K + split - 1) / split + BKE - 1) / BKE) * BKE;
        sk.partials = ws->partials;
        sk.counters = ws->counters;
    }
    hipLaunchKernelGGL((stream_kernel<MB, BK, STAGES, RB, P>), dim3(static_cast<unsigned>(nblocks * sk.split)),
                       dim3(THREADS), 0, s, p, nblocks, sk);
    return hipGetLastError();
}

template <int BK, int STAGES, int RB, class P>
hipError_t launch_bk(const P &p, int split, const Workspace *ws, hipStream_t s) {
    switch ((p.M + 15) / 16) {
        case 1: return launch_mb<1, BK, STAGES, RB>(p, split, ws, s);
        case 2: return launch_mb<2, BK, STAGES, RB>(p, split, ws, s);
        case 3: return launch_mb<3, BK, STAGES, RB>(p, split, ws, s);
        case 4: return launch_mb<4, BK, STAGES, RB>(p, split, ws, s);
        default: return hipErrorInvalidValue;
    }
}

// The configurations with 16- and 32-row blocks, for either operand type.
template <class P>
hipError_t launch_rows(const P &p, int bk, int stages, int rows, int split, const Workspace *ws, hipStream_t s) {
    if (rows == 16 && bk == 128 && stages == 2) return launch_bk<128, 2, 1>(p, split, ws, s);
    if (rows == 32 && bk == 64 && stages == 4) return launch_bk<64, 4, 2>(p, split, ws, s);
    return hipErrorInvalidValue;
}

}  // namespace

// K slices per row block: enough workgroups for one per CU, each wave at
// least one BK step of its slice.
int stream_split_for(int64_t M, int64_t N, int64_t K, int bk, int rows) {
    (void)M;
    const int64_t nblocks = (N + rows - 1) / rows;
    int64_t split = nblocks > 0 ? 256 / nblocks : 1;
    const int64_t by_depth = K / (WAVES * bk);
    if (split > by_depth) split = by_depth;
    if (split > 16) split = 16;
    return split < 1 ? 1 : static_cast<int>(split);
}

int64_t stream_workspace_floats(int64_t M, int64_t N, int split, int rows) {
    const int64_t nblocks = (N + rows - 1) / rows;
    return nblocks * split * (rows / 16) * ((M + 15) / 16) * 64 * 4;
}

int64_t stream_counter_count(int64_t N, int rows) { return (N + rows - 1) / rows; }

bool stream_config_exists(int bk, int stages, int rows) {
    return (rows == 64 && stages == 2 && bk == 64) || (rows == 16 && bk == 128 && stages == 2) ||
           (rows == 32 && bk == 64 && stages == 4);
}

hipError_t launch_stream(const Problem &p, int bk, int stages, int rows, int split, const Workspace *ws,
                         hipStream_t s) {
    if (p.M < 1 || p.M > 64) return hipErrorInvalidValue;
    if (is_general(p)) {
        if (rows == 64 && bk == 64 && stages == 2) return launch_bk<64, 2, 4>(p, split, ws, s);
        return launch_rows(p, bk, stages, rows, split, ws, s);
    }
    const DenseProblem d = dense_of(p);
    if (rows == 64 && bk == 64 && stages == 2) return launch_bk<64, 2, 4>(d, split, ws, s);
    return launch_rows(d, bk, stages, rows, split, ws, s);
}

hipError_t launch_stream_i8(const I8Problem &p, int bk, int stages, int rows, int split, const Workspace *ws,
                            hipStream_t s) {
    if (p.M < 1 || p.M > 64 || rows == 64) return hipErrorInvalidValue;
    return launch_rows(p, bk, stages, rows, split, ws, s);
}

}  // namespace kernelarc
