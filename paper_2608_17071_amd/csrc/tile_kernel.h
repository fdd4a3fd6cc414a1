// MFMA macro-tile kernels for Y = alpha X W^T (+ beta R) (+ bias): the
// compute-bound path.  Operands may be row-strided (leading dimensions).
//
// One workgroup of WAVES_M x WAVES_N waves computes a BM x BN output tile;
// each wave owns a (BM/WAVES_M) x (BN/WAVES_N) block made of 32x32
// accumulator blocks of v_mfma_f32_32x32x16_bf16 (bf16 in, fp32 accumulate).
//
// Data path (the paper's Table 2 tiers -- tensor-core substrate,
// asynchronous copy, software pipelining, epilogue and tile scheduling --
// re-derived for CDNA4 rather than Hopper):
//   * staging: buffer_load_dwordx4 with the LDS bit moves 16 bytes per lane
//     from HBM/L2 straight into LDS, no VGPR round trip.  One instruction
//     fills RPI = 64 / (BK/8) rows of one operand; every row segment it reads
//     is BK*2 contiguous bytes.
//   * pipeline: a ring of STAGES LDS buffers; STAGES-1 K steps are in flight
//     while one is multiplied (the loads' latency, about 2 us under full
//     load, is what a shallow pipeline exposes).
//   * LDS layout: BK*2 bytes per row; 16-byte chunk c of row r sits at slot
//     c ^ swz(r).  A fragment read (ds_read_b128) touches 32 consecutive
//     rows at one chunk; the swizzle spreads every 8 (and every 16)
//     consecutive rows over distinct bank groups.
//   * buffer resources bound each operand panel, so rows past M or N read
//     as zero without a branch; K-tail chunks are pointed out of range.
//   * schedule: fragment reads run PD sub-steps ahead of the MFMAs and the
//     refill loads go among the last sub-steps' MFMAs, after the step's
//     barrier; the order is pinned slot by slot (sched_barrier).
//   * epilogue: fp32 accumulator + fp32(R), one nearest-even rounding to
//     bf16, staged through LDS so R is read and Y written 16 bytes per
//     lane; each element is read (R) and written (Y) by the same lane, so Y
//     may alias R.
//   * tile scheduler: workgroups are handed to the 8 XCDs round-robin; ids
//     are remapped so each XCD takes a contiguous range of tiles, walked in
//     GROUP_M-row bands, so tiles resident on one XCD share panels in its L2.
#pragma once

#include "internal.h"

#include <utility>

namespace kernelarc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) void lds_void;

// Word 3 of a raw (unswizzled, stride 0) gfx9 buffer resource.
constexpr int RSRC_WORD3 = 0x00020000;
// A byte offset that is out of range for every panel (panels are < 2^31 B).
constexpr uint32_t OOB_OFFSET = 0x80000000u;
constexpr int XCDS = 8;
// Cache policy of buffer accesses: sc1 = device scope (coherent across XCDs);
// nt = non-temporal, for the residual and the output, which a launch reads
// or writes once (1-2.6 % faster on the MFMA-sized shapes).
constexpr int AUX_SC1 = 16;
constexpr int AUX_NT = 2;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), static_cast<short>(0),
                                             static_cast<int>(bytes), RSRC_WORD3);
}

// s_waitcnt immediate for gfx9: vmcnt = n (6 bits), expcnt and lgkmcnt not waited.
constexpr int waitcnt_vm(int n) { return (n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8); }

// Slot of 16-byte chunk c of row r: c ^ swz(r).  16 chunks per row
// (BK=128), 8 (BK=64) or 4 (BK=32).  A fragment read touches one chunk of
// 32 consecutive rows (32x32 MFMA) or two or four chunks of 16 (16x16 MFMA,
// lane quarters reading chunks that differ in their low bit); each swizzle
// puts the rows such a read serves together in distinct 16-byte bank groups.
// The fragment readers compute swz from the row within a 16-row block, so
// every swizzle repeats every 16 rows (checked below).
template <int CHUNKS>
__host__ __device__ constexpr int swz(int r) {
    if constexpr (CHUNKS == 16) return r & 15;
    else if constexpr (CHUNKS == 8) return (r & 7) ^ ((r >> 3) & 1);
    else return (((r >> 1) & 1) << 1) | ((r >> 2) & 1);   // 64-byte rows: pairs of rows share 128 bytes
}
template <int CHUNKS>
constexpr bool swz_repeats_every_16_rows() {
    for (int r = 0; r < 64; ++r)
        if (swz<CHUNKS>(r) != swz<CHUNKS>(r & 15)) return false;
    return true;
}
static_assert(swz_repeats_every_16_rows<4>() && swz_repeats_every_16_rows<8>() && swz_repeats_every_16_rows<16>(),
              "fragment reads assume 16-row periodic swizzles");

template <int BM_, int BN_, int BK_, int WAVES_M_, int WAVES_N_, int STAGES_, int WAVES_PER_EU_, bool LAG_ = false,
          bool M16_ = false, bool AACC_ = false>
struct Cfg {
    static constexpr int BM = BM_, BN = BN_, BK = BK_, STAGES = STAGES_;
    static constexpr int WAVES_M = WAVES_M_, WAVES_N = WAVES_N_;
    static constexpr int TILE_WAVES = WAVES_M * WAVES_N;
    static constexpr int WAVES = TILE_WAVES, THREADS = 64 * WAVES;
    static constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;   // per-wave block
    static constexpr int TM = WM / 32, TN = WN / 32;             // 32x32 blocks per wave
    // MFMA shape: 32x32x16 (default) or, with M16, 16x16x32 (bf16 plain and
    // general forms only): each 32x32 accumulator block is then four 16x16
    // blocks, quad q = 2*(row half) + (column half) in its elements 4q..4q+3.
    // Same operand bytes and MFMA cycles per K; half the accumulator
    // register traffic per product.
    static constexpr bool M16 = M16_;
    // AACC (with M16, bf16 only): the MFMAs are issued as inline assembly
    // whose accumulator operands are AGPRs, so the 16x16 accumulator blocks
    // stay in the AGPR file for the whole K loop.  This is what lets one wave
    // hold a 128x128 block (256 accumulator registers, the whole AGPR file)
    // with its fragments and addresses in VGPRs; with the builtin the
    // compiler moves accumulators between the two files every step.
    static constexpr bool AACC = AACC_;

    static constexpr int KSTEPS = BK / (M16 ? 32 : 16);           // MFMA sub-steps per stage
    // Fragment prefetch distance: the LDS reads of sub-step s + PD are
    // issued among the MFMAs of sub-step s (PD + 1 register sets).
    static constexpr int PD = 1;
    // Refill timing (STAGES >= 3 only when set): the buffer freed at step
    // kt-1's barrier is refilled with step kt+STAGES-1 by loads spread over
    // all of step kt's MFMAs (STAGES-2 steps of latency slack, no burst);
    // when clear, the buffer freed at step kt's own barrier is refilled
    // with step kt+STAGES among the MFMAs after that barrier.
    static constexpr bool LAG = LAG_;
    static constexpr int ROW_BYTES = BK * 2, CHUNKS = BK / 8, RPI = 64 / CHUNKS;
    static constexpr int A_BYTES = BM * ROW_BYTES, B_BYTES = BN * ROW_BYTES;
    static constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
    static constexpr int LDS_BYTES = STAGES * STAGE_BYTES;
    static constexpr int A_LOADS = BM / RPI / TILE_WAVES;         // DMA instructions per wave per stage
    static constexpr int B_LOADS = BN / RPI / TILE_WAVES;
    static constexpr int LOADS = A_LOADS + B_LOADS;
    static constexpr int WAVES_PER_EU = WAVES_PER_EU_;
    // Epilogue staging: one 32-row slab of a wave's block in fp32, rows
    // padded by 4 floats; lanes then read 8 consecutive columns each.
    static constexpr int EPI_STRIDE = WN + 4;
    static constexpr int EPI_WAVE_FLOATS = 32 * EPI_STRIDE;
    static constexpr int LANES_PER_ROW = WN / 8;
    static constexpr int ROWS_PER_PASS = 64 / LANES_PER_ROW;

    static_assert(BK == 32 || BK == 64 || BK == 128, "BK");
    static_assert(TM >= 1 && TN >= 1 && WM % 32 == 0 && WN % 32 == 0, "wave block");
    static_assert(A_LOADS >= 1 && B_LOADS >= 1 && BM % (RPI * TILE_WAVES) == 0 && BN % (RPI * TILE_WAVES) == 0,
                  "staging split");
    static_assert(STAGES >= 2, "pipeline depth");
    static_assert(WAVES <= 16, "workgroup size");
    static_assert(LDS_BYTES <= 160 * 1024, "LDS capacity");
    static_assert(TILE_WAVES * EPI_WAVE_FLOATS * 4 <= LDS_BYTES, "epilogue staging fits");
    static_assert(LOADS * (STAGES - 2) < 64, "vmcnt range");
    static_assert(PD >= 1 && PD <= KSTEPS, "fragment prefetch distance");
    static_assert(!LAG || STAGES >= 3, "lagged refill needs three stages");
    static_assert(!AACC || M16, "AGPR accumulators are a 16x16 MFMA option");
};

// Load block (RPI rows of the stage's B tile) that B load qb of a wave
// fills.  SwiGLU: the B tile alternates 32-row blocks of gate and up rows
// (block 2b holds gate rows 32b.., block 2b+1 the up rows of the same
// outputs); a wave's first B_LOADS/2 loads fill gate blocks and the rest up
// blocks, so which weight a load reads is fixed at compile time.
template <class C, bool GLU>
__device__ __forceinline__ int b_block(int wave, int qb) {
    if constexpr (!GLU) {
        return wave * C::B_LOADS + qb;
    } else {
        constexpr int HALF = C::B_LOADS / 2, PER = 32 / C::RPI;   // load blocks per 32-row block
        const bool up = qb >= HALF;
        const int idx = wave * HALF + (up ? qb - HALF : qb);     // among the gate (or up) load blocks
        return (idx / PER) * 2 * PER + (up ? PER : 0) + idx % PER;
    }
}

// Enqueue LDS-direct load q (A loads first, then B) of the K step at
// element kbase (byte kbytes within a row) into one stage buffer.  Chunks
// at or past K are pointed out of range and arrive as zeros.  rb2 is the
// up-weight panel of SwiGLU (unused otherwise).  FULL: the caller knows the
// whole step lies below K, so the lane's offset stays fixed and the step's
// byte offset goes in the scalar offset (no per-load vector arithmetic).
template <class C, int q, bool GLU, bool FULL = false>
__device__ __forceinline__ void issue_load(char *stage, const __amdgpu_buffer_rsrc_t &ra,
                                           const __amdgpu_buffer_rsrc_t &rb, const __amdgpu_buffer_rsrc_t &rb2,
                                           const uint32_t *a_off, const int *a_k, const uint32_t *b_off,
                                           const int *b_k, int wave, int64_t kbase, uint32_t kbytes, int64_t K) {
    if constexpr (FULL) {
        if constexpr (q < C::A_LOADS) {
            const int blk = wave * C::A_LOADS + q;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void *)(stage + blk * 1024), 16, a_off[q], kbytes, 0, 0);
        } else {
            constexpr int qb = q - C::A_LOADS;
            const int blk = b_block<C, GLU>(wave, qb);
            const __amdgpu_buffer_rsrc_t &r = (GLU && qb >= C::B_LOADS / 2) ? rb2 : rb;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void *)(stage + C::A_BYTES + blk * 1024), 16, b_off[qb],
                                                     kbytes, 0, 0);
        }
    } else if constexpr (q < C::A_LOADS) {
        const int blk = wave * C::A_LOADS + q;
        const uint32_t off = (kbase + a_k[q] < K) ? a_off[q] + kbytes : OOB_OFFSET;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void *)(stage + blk * 1024), 16, off, 0, 0, 0);
    } else {
        constexpr int qb = q - C::A_LOADS;
        const int blk = b_block<C, GLU>(wave, qb);
        const uint32_t off = (kbase + b_k[qb] < K) ? b_off[qb] + kbytes : OOB_OFFSET;
        const __amdgpu_buffer_rsrc_t &r = (GLU && qb >= C::B_LOADS / 2) ? rb2 : rb;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void *)(stage + C::A_BYTES + blk * 1024), 16,
                                                 off, 0, 0, 0);
    }
}

constexpr int gcd_int(int a, int b) { return b == 0 ? a : gcd_int(b, a % b); }

// Compile-time loop: f(std::integral_constant<int, I>) for I = B .. E-1.
template <int B, class F, int... I>
__device__ __forceinline__ void static_for_impl(F &&f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, B + I>{}), ...);
}
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F &&f) {
    if constexpr (E > B) static_for_impl<B>(f, std::make_integer_sequence<int, E - B>{});
}

// BKE: K elements per stage (BK for bf16 operands, 2*BK for int8 ones: a
// stage always holds ROW_BYTES bytes of each row).
template <class C, bool GLU, int BKE>
__device__ __forceinline__ void issue_stage(char *stage, const __amdgpu_buffer_rsrc_t &ra,
                                            const __amdgpu_buffer_rsrc_t &rb, const __amdgpu_buffer_rsrc_t &rb2,
                                            const uint32_t *a_off, const int *a_k, const uint32_t *b_off,
                                            const int *b_k, int wave, int kt, int64_t K) {
    const int64_t kbase = static_cast<int64_t>(kt) * BKE;
    const uint32_t kbytes = static_cast<uint32_t>(kt) * C::ROW_BYTES;
    static_for<0, C::LOADS>([&](auto q) {
        issue_load<C, decltype(q)::value, GLU>(stage, ra, rb, rb2, a_off, a_k, b_off, b_k, wave, kbase, kbytes,
                                               K);
    });
}

// Fragment read r of one sub-step, in the order the sub-step's MFMAs first
// use them (a0, b0 .. b[TN-1], a1 .. a[TM-1]): lane l reads row l % 32 of a
// 32-row block at byte column col.
template <class C, int r>
__device__ __forceinline__ void read_frag(const char *a_base, const char *b_base, int col, bf16x8 *fa,
                                          bf16x8 *fb) {
    if constexpr (r == 0)
        fa[0] = *reinterpret_cast<const bf16x8 *>(a_base + col);
    else if constexpr (r <= C::TN)
        fb[r - 1] = *reinterpret_cast<const bf16x8 *>(b_base + (r - 1) * 32 * C::ROW_BYTES + col);
    else
        fa[r - C::TN] = *reinterpret_cast<const bf16x8 *>(a_base + (r - C::TN) * 32 * C::ROW_BYTES + col);
}

// Fragment read r of a 16x16x32 sub-step (M16), in the order the MFMAs
// first use them (a0, b0 .. b[2TN-1], a1 .. a[2TM-1]): lane l reads row
// l % 16 of a 16-row block at byte column col.
template <class C, int r>
__device__ __forceinline__ void read_frag16(const char *a_base, const char *b_base, int col, bf16x8 *fa,
                                            bf16x8 *fb) {
    constexpr int FTN = 2 * C::TN;
    if constexpr (r == 0)
        fa[0] = *reinterpret_cast<const bf16x8 *>(a_base + col);
    else if constexpr (r <= FTN)
        fb[r - 1] = *reinterpret_cast<const bf16x8 *>(b_base + (r - 1) * 16 * C::ROW_BYTES + col);
    else
        fa[r - FTN] = *reinterpret_cast<const bf16x8 *>(a_base + (r - FTN) * 16 * C::ROW_BYTES + col);
}

// FP8 fragment read r (same order as read_frag): 32 bytes per lane, the two
// 16-byte chunks at byte columns col and col2 of the lane's row (the 64 K
// bytes of one v_mfma_scale_f32_32x32x64_f8f6f4 split between the lane
// halves; A and B use the same byte-to-K assignment, so the sum over K is
// the full one whatever order the instruction takes its bytes in).
template <class C, int r>
__device__ __forceinline__ void read_frag8(const char *a_base, const char *b_base, int col, int col2, i32x8 *fa,
                                           i32x8 *fb) {
    const char *base = r == 0 ? a_base
                       : r <= C::TN ? b_base + (r - 1) * 32 * C::ROW_BYTES
                                    : a_base + (r - C::TN) * 32 * C::ROW_BYTES;
    const i32x4 lo = *reinterpret_cast<const i32x4 *>(base + col);
    const i32x4 hi = *reinterpret_cast<const i32x4 *>(base + col2);
    const i32x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    if constexpr (r == 0) fa[0] = v;
    else if constexpr (r <= C::TN) fb[r - 1] = v;
    else fa[r - C::TN] = v;
}

// Workgroup barrier that keeps the newest N LDS-direct loads of each wave
// in flight.  A __syncthreads() here would drain every outstanding load
// (its fence waits for vmcnt(0)) and so empty the staging ring at every K
// step.  The wave's LDS reads are complete before it arrives (lgkmcnt(0)),
// so the buffer they read may be refilled once all waves have passed; the
// memory clobber keeps the compiler from moving LDS accesses across it.
template <int N>
__device__ __forceinline__ void stage_barrier() {
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
}

// Workgroup barrier for LDS only: the wave's LDS accesses are complete
// before it arrives, its global stores may still be in flight.
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Adds 16 raw bytes (fp32 or int32 bits) to quad q of a 32x32 block (exact
// for int32).
__device__ __forceinline__ void add_quad(f32x16 &a, int q, const f32x4 &v) {
    a[4 * q] += v[0];
    a[4 * q + 1] += v[1];
    a[4 * q + 2] += v[2];
    a[4 * q + 3] += v[3];
}
__device__ __forceinline__ void add_quad(i32x16 &a, int q, const f32x4 &bits) {
    const i32x4 v = __builtin_bit_cast(i32x4, bits);
    a[4 * q] += v[0];
    a[4 * q + 1] += v[1];
    a[4 * q + 2] += v[2];
    a[4 * q + 3] += v[3];
}

// 16 raw bytes added to an fp32 or int32 quad (exact for int32).
__device__ __forceinline__ void add_bits(f32x4 &a, const f32x4 &bits) { a += bits; }
__device__ __forceinline__ void add_bits(i32x4 &a, const f32x4 &bits) { a += __builtin_bit_cast(i32x4, bits); }

// v_mfma_f32_16x16x32_bf16 with the accumulator in AGPRs (see Cfg::AACC).
__device__ __forceinline__ void mfma16_agpr(f32x4 &acc, const bf16x8 &a, const bf16x8 &b) {
    asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}
// The INT8 form: 16 x 64 int8 operands (the same 16 bytes per lane), exact
// int32 sums.
__device__ __forceinline__ void mfma16_agpr(i32x4 &acc, const bf16x8 &a, const bf16x8 &b) {
    asm volatile("v_mfma_i32_16x16x64_i8 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}

// Split-K bookkeeping of one launch (split == 1: none).
struct SplitK {
    int split;          // K slices per split tile (1: none)
    int64_t kslice;     // slice length, a multiple of BK
    float *partials;    // [split tile][slice][BM*BN] fp32, fragment order
    unsigned *counters; // one arrival counter per split tile, zero between calls
    // Tail split: tiles [0, full_tiles) of the band order run whole and only
    // the rest are split (0: every tile is split when split > 1).  Used when
    // whole rounds of workgroups leave a partial last round.
    int64_t full_tiles;
};

// P = Problem: the general form (row strides, alpha, beta, bias);
// P = DenseProblem: dense operands, and the epilogue adds R as is (the plain
// operator); P = GluProblem: SwiGLU, the B tile holds BN/2 gate and BN/2 up
// rows (alternate 32-row blocks) and the output tile is BM x BN/2;
// P = I8Problem, I8GluProblem: the same with int8 operands (a stage holds
// twice the K elements, v_mfma_i32_32x32x32_i8 accumulates exactly in
// int32) and dequantisation by the row and column scales in the epilogue;
// P = F8Problem, F8GluProblem: the same with FP8 E4M3 operands
// (v_mfma_scale_f32_32x32x64_f8f6f4 with unit scales, fp32 accumulation,
// sub-steps of 64 K bytes);
// P = Grouped<DenseProblem>, Grouped<GluProblem>: one launch over the groups
// of an expert-major padded layout; the m-tiles of the groups are stacked
// (tiles_m = G * m-tiles per group), each workgroup rebases the problem on
// its group, and tiles wholly past the group's valid rows exit at once.
template <class C, class P>
__global__ __attribute__((amdgpu_flat_work_group_size(C::THREADS, C::THREADS),
                          amdgpu_waves_per_eu(C::WAVES_PER_EU, C::WAVES_PER_EU)))
void tile_kernel(P p, int64_t tiles_m, int64_t tiles_n, int group_m, SplitK sk) {
    using PB = typename grouped_trait<P>::base;
    constexpr bool GROUPED = grouped_trait<P>::value;
    constexpr bool GEN = std::is_same<PB, Problem>::value;
    constexpr bool I8 = std::is_same<PB, I8Problem>::value || std::is_same<PB, I8GluProblem>::value;
    constexpr bool F8 = std::is_same<PB, F8Problem>::value || std::is_same<PB, F8GluProblem>::value;
    constexpr bool Q8 = I8 || F8;                  // 1-byte operands with dequantisation scales
    constexpr bool GLU = std::is_same<PB, GluProblem>::value || std::is_same<PB, I8GluProblem>::value ||
                         std::is_same<PB, F8GluProblem>::value;
    static_assert(!C::M16 || !F8, "16x16 MFMA tiles take bf16 or int8 problems");
    constexpr int EB = Q8 ? 1 : 2;                 // bytes per operand element
    constexpr int BKE = C::ROW_BYTES / EB;         // K elements per stage
    constexpr int CKE = 16 / EB;                   // K elements per 16-byte chunk
    using AccV = typename std::conditional<I8, i32x16, f32x16>::type;
    // Output columns of the tile and of one wave's block.
    constexpr int BNO = GLU ? C::BN / 2 : C::BN, WNO = GLU ? C::WN / 2 : C::WN;
    static_assert(!GLU || (C::TN % 2 == 0 && C::B_LOADS % 2 == 0 && 32 % C::RPI == 0), "gate/up pairing");
    const int64_t ldx = ldx_of(p), ldw = ldw_of(p), ldr = ldr_of(p), ldy = ldy_of(p);
    __shared__ __attribute__((aligned(1024))) char lds[C::LDS_BYTES + (C::AACC ? 256 : 0)];   // + prefetch sink

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    char *const glds = lds;

    // Workgroup -> (K slice, tile).  Workgroups go to the 8 XCDs round-robin;
    // each XCD takes a contiguous range of work (slice-major ids), walked in
    // GROUP_M-row bands.  With a tail split each XCD takes an equal share of
    // the whole tiles first and then an equal share of the tail pieces.
    const int64_t tiles = tiles_m * tiles_n;
    int64_t tm, tn, slice, tile;
    bool piece;   // a K slice of a split tile
    {
        const int64_t x = blockIdx.x % XCDS, local = blockIdx.x / XCDS;
        if (sk.split > 1 && sk.full_tiles > 0) {
            const int64_t rest = tiles - sk.full_tiles;
            const int64_t f8 = sk.full_tiles / XCDS, p8 = rest * sk.split / XCDS;
            if (local < f8) {
                tile = x * f8 + local;
                slice = 0;
                piece = false;
            } else {
                const int64_t q = x * p8 + (local - f8);
                slice = q / rest;
                tile = sk.full_tiles + (q - slice * rest);
                piece = true;
            }
        } else {
            const int64_t T = tiles * sk.split;
            const int64_t per = T / XCDS, rem = T % XCDS;
            const int64_t logical = x * per + (x < rem ? x : rem) + local;
            slice = logical / tiles;
            tile = logical - slice * tiles;
            piece = sk.split > 1;
        }
        const int64_t band = static_cast<int64_t>(group_m) * tiles_n;
        const int64_t g = tile / band;
        const int64_t first_m = g * group_m;
        const int64_t rows = (tiles_m - first_m) < group_m ? (tiles_m - first_m) : group_m;
        const int64_t in_band = tile - g * band;
        tm = first_m + in_band % rows;
        tn = in_band / rows;
    }
    if constexpr (GROUPED) {
        const int64_t tpg = (p.Mpad + C::BM - 1) / C::BM;   // m-tiles per group
        const int64_t g = tm / tpg;
        tm -= g * tpg;
        const int64_t rows = group_rows(p.counts, g, p.Mpad);
        if (tm * C::BM >= rows) return;                    // the whole tile is gap rows
        p.M = rows;
        p.X += g * p.Mpad * p.K;
        p.Y += g * p.Mpad * p.N;
        p.W += g * p.N * p.K;
        if constexpr (GLU) p.W2 += g * p.N * p.K;
    }
    const int64_t m0 = tm * C::BM;
    const int64_t n0 = tn * BNO;
    const int64_t K = p.K;
    // This workgroup's K range [kbeg, kend); loads at or past kend read zero.
    const int64_t kbeg = piece ? slice * sk.kslice : 0;
    const int64_t kend = piece ? ((kbeg + sk.kslice) < K ? (kbeg + sk.kslice) : K) : K;

    // Operand panels bounded by buffer resources: rows past M (N) read 0.
    const int64_t rows_a = (p.M - m0) < C::BM ? (p.M - m0) : C::BM;
    const int64_t rows_b = (p.N - n0) < BNO ? (p.N - n0) : BNO;
    const __amdgpu_buffer_rsrc_t ra =
        make_rsrc(p.X + m0 * ldx, static_cast<uint32_t>(GEN ? strided_bytes(rows_a, K, ldx) : rows_a * K * EB));
    const __amdgpu_buffer_rsrc_t rb =
        make_rsrc(p.W + n0 * ldw, static_cast<uint32_t>(GEN ? strided_bytes(rows_b, K, ldw) : rows_b * K * EB));
    const __amdgpu_buffer_rsrc_t rb2 = [&] {
        if constexpr (GLU) return make_rsrc(p.W2 + n0 * ldw, static_cast<uint32_t>(rows_b * K * EB));
        else return rb;
    }();

    // Staging map: lane l of load block blk fills slot l % CHUNKS of row
    // RPI*blk + l / CHUNKS, which holds global chunk (l % CHUNKS) ^ swz(row).
    uint32_t a_off[C::A_LOADS], b_off[C::B_LOADS];
    int a_k[C::A_LOADS], b_k[C::B_LOADS];
    const int slot = lane % C::CHUNKS;
#pragma unroll
    for (int q = 0; q < C::A_LOADS; ++q) {
        const int r = (wave * C::A_LOADS + q) * C::RPI + lane / C::CHUNKS;
        const int c = slot ^ swz<C::CHUNKS>(r);
        a_off[q] = static_cast<uint32_t>(r * ldx * EB + c * 16);
        a_k[q] = c * CKE;
    }
#pragma unroll
    for (int q = 0; q < C::B_LOADS; ++q) {
        const int r = b_block<C, GLU>(wave, q) * C::RPI + lane / C::CHUNKS;   // row of the B tile
        const int c = slot ^ swz<C::CHUNKS>(r);
        const int wr = GLU ? (r >> 6) * 32 + (r & 31) : r;                    // row of its weight panel
        b_off[q] = static_cast<uint32_t>(wr * ldw * EB + c * 16);
        b_k[q] = c * CKE;
    }

    // L2 prefetch of A (AGPR tile only).  The tiles of one tile row that run
    // together on an XCD (consecutive tn within a band) stage the same A
    // rows, and their loads of a new K step miss the XCD's L2 together.  Tile
    // tn % 4 owns a quarter of the rows: at the end of each K step its waves
    // touch the step PF_AHEAD ahead of the K loop in each owned row (16 rows
    // a wave, one dword per 128-byte line, a second one when a row's slice
    // straddles two lines), so that the line is in L2 when the staging loads
    // of all four tiles ask for it.  The dwords land in an LDS sink that
    // nothing reads; the prefetch is the newest load at every barrier, so
    // the counted wait leaves it in flight.  A tile with no neighbour for an
    // owned row (narrow problems, other bands) only fetches that line early.
    constexpr int PFN = C::AACC ? 1 : 0;             // prefetch loads per wave per step
    static_assert(!PFN || (C::STAGES == 2 && !C::LAG), "the counted waits place one prefetch per barrier");
    constexpr int PF_AHEAD = C::STAGES + 1;          // one step past the refill
    uint32_t pf_off = OOB_OFFSET;
    if constexpr (C::AACC) {
        const int64_t r = 64 * (tn & 3) + 16 * wave + (lane & 15);
        const bool straddles =
            (reinterpret_cast<uintptr_t>(p.X + (m0 + r) * ldx) & (C::ROW_BYTES - 1)) != 0;
        if (lane < 16 || (lane < 32 && straddles))
            pf_off = static_cast<uint32_t>(r * ldx * EB + (lane < 16 ? 0 : C::ROW_BYTES - 4));
    }
    auto prefetch_a = [&](int step) {
        if constexpr (C::AACC) {
            const bool in_range = static_cast<int64_t>(step) * BKE < kend && pf_off != OOB_OFFSET;
            const uint32_t off = in_range ? pf_off + static_cast<uint32_t>(step) * C::ROW_BYTES : OOB_OFFSET;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void *)(lds + C::LDS_BYTES), 4, off, 0, 0, 0);
        }
    };

    // Accumulators: 32x32 blocks (acc), or with M16 16x16 blocks (acc16),
    // where quad q of 32x32 block (i, j) -- its elements 4q .. 4q+3 -- is
    // 16x16 block (2i + q/2, 2j + q%2).  Everything after the K loop reads
    // and writes them through quad_of / set_quad in 32x32-block terms.
    using AccQ = typename std::conditional<I8, i32x4, f32x4>::type;
    AccV acc[C::M16 ? 1 : C::TM][C::M16 ? 1 : C::TN];
    AccQ acc16[C::M16 ? 2 * C::TM : 1][C::M16 ? 2 * C::TN : 1];
    auto quad_of = [&](int i, int j, int q) -> AccQ {
        if constexpr (C::M16) return acc16[2 * i + (q >> 1)][2 * j + (q & 1)];
        else return AccQ{acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
    };
    auto quad_set = [&](int i, int j, int q, const AccQ &v) {
        if constexpr (C::M16) acc16[2 * i + (q >> 1)][2 * j + (q & 1)] = v;
        else {
            acc[i][j][4 * q] = v[0];
            acc[i][j][4 * q + 1] = v[1];
            acc[i][j][4 * q + 2] = v[2];
            acc[i][j][4 * q + 3] = v[3];
        }
    };
    auto quad_ref_add = [&](int i, int j, int q, const f32x4 &bits) {
        if constexpr (C::M16) add_bits(acc16[2 * i + (q >> 1)][2 * j + (q & 1)], bits);
        else add_quad(acc[i][j], q, bits);
    };
    auto zero_acc = [&] {
        if constexpr (C::M16) {
#pragma unroll
            for (int i = 0; i < 2 * C::TM; ++i)
#pragma unroll
                for (int j = 0; j < 2 * C::TN; ++j) acc16[i][j] = AccQ{0, 0, 0, 0};
        } else {
#pragma unroll
            for (int i = 0; i < C::TM; ++i)
#pragma unroll
                for (int j = 0; j < C::TN; ++j)
#pragma unroll
                    for (int e = 0; e < 16; ++e) acc[i][j][e] = 0;
        }
    };
    zero_acc();

    // Fragment reads: row (lane % 32) of each 32-row block, chunk 2*ks + hi
    // (32x32x16); with M16, row (lane % 16) of each 16-row block, one of
    // the sub-step's four chunks per lane quarter hi = lane / 16.  Rows 16
    // apart share their swizzle.
    const int frag_row = C::M16 ? (lane & 15) : (lane & 31);
    const int hi = C::M16 ? (lane >> 4) : (lane >> 5);
    const int wm0 = (wave / C::WAVES_N) * C::WM;
    const int wn0 = (wave % C::WAVES_N) * C::WN;
    const int a_row_byte = (wm0 + frag_row) * C::ROW_BYTES;
    const int b_row_byte = (wn0 + frag_row) * C::ROW_BYTES;
    const int frag_swz = swz<C::CHUNKS>(frag_row);

    // The workgroup's BK steps [g0, g0 + iters); loads past kend read zero.
    const int g0 = static_cast<int>(kbeg / BKE);
    const int iters = kend > kbeg ? static_cast<int>((kend + BKE - 1) / BKE) - g0 : 0;
    const int64_t gend = kend;

    // Epilogue constants (the residual may be requested before the K loop).
    const int64_t N = p.N;
    const int64_t rows_y = (p.M - m0) < C::BM ? (p.M - m0) : C::BM;
    const uint32_t ybytes = static_cast<uint32_t>(GEN ? strided_bytes(rows_y, N, ldy) : rows_y * N * 2);
    const uint32_t rbytes = static_cast<uint32_t>(GEN ? strided_bytes(rows_y, N, ldr) : rows_y * N * 2);
    const __amdgpu_buffer_rsrc_t ry = make_rsrc(p.Y + m0 * ldy, ybytes);
    // Without a residual the R resource is empty (its loads read zero).
    const uint16_t *const R = resid_of(p);
    const __amdgpu_buffer_rsrc_t rr = make_rsrc(R ? R + m0 * ldr : p.Y, R ? rbytes : 0u);
    const bool has_r = R != nullptr;
    // 16-byte R/Y accesses need every row to start 16-byte aligned.
    const bool vec = (N & 7) == 0 && (ldy & 7) == 0 && (!has_r || (ldr & 7) == 0);
    // Epilogue staging geometry for the wave's WNO output columns.
    constexpr int EPS = WNO + 4, LPR = WNO / 8, RPP = 64 / LPR;
    static_assert(GLU || (EPS == C::EPI_STRIDE && LPR == C::LANES_PER_ROW && RPP == C::ROWS_PER_PASS), "staging");
    const int pr = lane / LPR;                          // row within a pass
    const int pc = (lane % LPR) * 8;                    // first of 8 columns
    const int64_t col0 = n0 + wn0 / (C::WN / WNO) + pc;
    constexpr int PASSES = 32 / RPP;
    auto row_of = [&](int i, int v) { return static_cast<int64_t>(wm0 + i * 32 + v * RPP + pr); };
    auto base_of = [&](int i, int v) { return static_cast<uint32_t>(row_of(i, v) * ldy * 2 + col0 * 2); };
    auto rbase_of = [&](int i, int v) {
        return GEN ? static_cast<uint32_t>(row_of(i, v) * ldr * 2 + col0 * 2) : base_of(i, v);
    };
    // All of a slab's R is read before any of its Y is written (each element
    // by the same lane), so the loads do not wait behind the stores and Y
    // may alias R.
    auto load_r = [&](int i, i32x4 (&rv)[PASSES]) {
#pragma unroll
        for (int v = 0; v < PASSES; ++v)
            rv[v] = __builtin_amdgcn_raw_buffer_load_b128(rr, col0 < N ? rbase_of(i, v) : OOB_OFFSET, 0, AUX_NT);
    };
    // Two slabs of R in registers: slab i+1 is requested before slab i is
    // staged and stored, so only slab 0's latency is exposed.  The AGPR tile
    // (whose fragment registers are free after the K loop) requests every
    // slab of its block at once, so the whole block waits for one latency.
    constexpr bool R_ALL = C::AACC;
    constexpr int RV = R_ALL ? C::TM : 2;
    i32x4 rv[RV][PASSES];
    auto rslot = [](int i) { return R_ALL ? i : (i & 1); };
    const bool has_bias = GEN && bias_of(p) != nullptr;
    const float alpha = alpha_of(p), beta = beta_of(p);
    // The value before rounding: the plain operator's acc + r, or the
    // general form's alpha * acc + beta * r (the two agree at alpha = beta = 1).
    auto value = [&](float acc, float r) {
        if constexpr (GEN) return combine(acc, r, has_r, alpha, beta);
        else return has_r ? acc + r : acc;
    };
    // INT8 dequantisation scales.  The column scales and the first slab's
    // row scales are requested before the K loop so that their latency
    // hides behind it; each later slab's row scales are requested one slab
    // ahead.  Plain: the scales of the lane's 8 columns and of its row in
    // each pass; SwiGLU: the gate and up scales of the lane's column in each
    // block pair and the scales of the slab's 16 accumulator rows.
    constexpr int NSX = !Q8 ? 1 : GLU ? 16 : PASSES;
    constexpr int NSW = !Q8 ? 1 : GLU ? C::TN : 8;
    float sxr[2][NSX], swc[NSW];
    [[maybe_unused]] __amdgpu_buffer_rsrc_t rsx;
    auto ld = [](const __amdgpu_buffer_rsrc_t &r, uint32_t off) {
        return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
    };
    // Row scales of slab i into sxr[i & 1].
    auto load_sx = [&](int i) {
        if constexpr (GLU) {
#pragma unroll
            for (int e = 0; e < 16; ++e)
                sxr[i & 1][e] = ld(rsx, static_cast<uint32_t>((wm0 + i * 32 + 8 * (e >> 2) + 4 * hi + (e & 3)) * 4));
        } else {
#pragma unroll
            for (int v = 0; v < PASSES; ++v) sxr[i & 1][v] = ld(rsx, static_cast<uint32_t>(row_of(i, v) * 4));
        }
    };
    if constexpr (Q8) {
        rsx = make_rsrc(p.sx + m0, static_cast<uint32_t>(rows_y * 4));
        const __amdgpu_buffer_rsrc_t rsw = make_rsrc(p.sw, static_cast<uint32_t>(N * 4));
        if constexpr (GLU) {
            const __amdgpu_buffer_rsrc_t rsw2 = make_rsrc(p.sw2, static_cast<uint32_t>(N * 4));
#pragma unroll
            for (int j = 0; j < C::TN / 2; ++j) {
                const int64_t c = n0 + wn0 / 2 + j * 32 + frag_row;
                swc[j] = ld(rsw, c < N ? static_cast<uint32_t>(c * 4) : OOB_OFFSET);
                swc[C::TN / 2 + j] = ld(rsw2, c < N ? static_cast<uint32_t>(c * 4) : OOB_OFFSET);
            }
        } else {
#pragma unroll
            for (int t = 0; t < 8; ++t)
                swc[t] = ld(rsw, col0 + t < N ? static_cast<uint32_t>((col0 + t) * 4) : OOB_OFFSET);
        }
        load_sx(0);
    }

    // Small tiles request the first slab of R before the K loop (a few
    // registers); it is then in flight with the first loads instead of after
    // the loop, or after the split-K hand-off.
    constexpr bool EARLY_R = C::TM * C::TN <= 4 && C::WAVES_PER_EU <= 2 && C::WAVES <= 4;
    if constexpr (EARLY_R)
        if (vec && has_r) load_r(0, rv[0]);

    // Software pipeline.  Per K step: the MFMAs of its KSTEPS sub-steps;
    // among the MFMAs of sub-step s, the LDS reads of sub-step s + PD's
    // fragments.  The barrier sits before the last PD sub-steps: there every
    // wave has read the whole step (its buffer may be refilled) and the next
    // step has landed, so the reads that run ahead into the next step and
    // the refill (step kt + STAGES into this buffer) go among those last
    // MFMAs, whose operands are already in registers.  The instruction order
    // is pinned slot by slot (one MFMA and its share of reads and loads).
    // One MFMA sub-step covers 32 bytes of K per row (bf16 32x32x16, int8
    // 32x32x32) or 64 (FP8 32x32x64).
    constexpr int KS = F8 ? C::KSTEPS / 2 : C::KSTEPS, PD = C::PD, NSETS = PD + 1;
    static_assert(KS >= PD, "fragment prefetch distance");
    // Sub-step g of the workgroup's range (g = step * KS + ks) multiplies the
    // fragments of register set g % NSETS.  When KS is not a multiple of
    // NSETS the loop body covers UNROLL steps, each with its phase fixed at
    // compile time, so every set index stays a constant; the step count is
    // then rounded up to a multiple of UNROLL, and the extra step, past the
    // end of the K range, multiplies stage buffers its loads filled with
    // zeros (out-of-range chunks arrive as zeros), adding exact zeros.
    constexpr int UNROLL = NSETS / gcd_int(KS, NSETS);
    // Per sub-step: MF MFMAs and FR fragment reads (A blocks then B blocks
    // of 32 rows, or of 16 rows with M16: twice as many of each block kind,
    // four 16x16 products per 32x32 accumulator block).
    constexpr int FTM = C::M16 ? 2 * C::TM : C::TM, FTN = C::M16 ? 2 * C::TN : C::TN;
    constexpr int MF = FTM * FTN, FR = FTM + FTN, POST = PD * MF, SLOTS = KS * MF;
    // Loads a wave may leave in flight at a step's barrier (step kt+1 must
    // have landed): the steps requested after it, and with the lagged
    // refill also the loads of this step's refill issued before the barrier,
    // and with the A prefetch the PFN loads issued at the end of step kt-1.
    constexpr int LPRE = C::LAG ? ((KS - PD) * MF * C::LOADS) / SLOTS : 0;
    constexpr int VM_KEEP = C::LAG ? C::LOADS * (C::STAGES - 3) + LPRE : C::LOADS * (C::STAGES - 2);
    constexpr int VM_KEEP0 = C::LOADS * (C::STAGES - 2);   // prologue: step g0 landed
    int colk[KS], colk2[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        if constexpr (F8) {
            colk[ks] = ((4 * ks + 2 * hi) ^ frag_swz) * 16;
            colk2[ks] = ((4 * ks + 2 * hi + 1) ^ frag_swz) * 16;
        } else if constexpr (C::M16) {
            // Lane quarter h takes chunk (h & 1) * 2 + (h >> 1) of the
            // sub-step (A and B alike, so the sum over k is unchanged): a
            // ds_read_b128 serves lanes l and l + 32 together, and their
            // chunks must differ in the low bit, as in the 32x32 layout,
            // for the XOR-swizzled rows to fall in distinct banks.
            colk[ks] = ((4 * ks + ((hi & 1) << 1) + (hi >> 1)) ^ frag_swz) * 16;
            colk2[ks] = 0;
        } else {
            colk[ks] = ((2 * ks + hi) ^ frag_swz) * 16;
            colk2[ks] = 0;
        }
    }
    using Frag = typename std::conditional<F8, i32x8, bf16x8>::type;
    Frag fa[NSETS][FTM], fb[NSETS][FTN];
    auto read_any = [&](auto rc, const char *src, int col, int col2, Frag *ta, Frag *tb) {
        if constexpr (F8)
            read_frag8<C, decltype(rc)::value>(src + a_row_byte, src + C::A_BYTES + b_row_byte, col, col2, ta, tb);
        else if constexpr (C::M16)
            read_frag16<C, decltype(rc)::value>(src + a_row_byte, src + C::A_BYTES + b_row_byte, col, ta, tb);
        else
            read_frag<C, decltype(rc)::value>(src + a_row_byte, src + C::A_BYTES + b_row_byte, col, ta, tb);
    };

    // Prologue: steps g0 .. g0+STAGES-2 requested, step g0 landed in every
    // wave, the fragments of its first PD sub-steps requested, then step
    // g0+STAGES-1 into the last buffer and the first A prefetch (AGPR tile),
    // so that a prefetch is the newest load at every barrier.  Past the end
    // of the range the loads only write zeros into buffers whose contents
    // are never used.
    // The counted waits assume the steps' loads are issued in step order:
    // scheduling barriers keep the compiler from interleaving them.
#pragma unroll
    for (int s = 0; s < C::STAGES - 1; ++s) {
        issue_stage<C, GLU, BKE>(glds + s * C::STAGE_BYTES, ra, rb, rb2, a_off, a_k, b_off, b_k, wave, g0 + s,
                                 gend);
        __builtin_amdgcn_sched_barrier(0);
    }
    stage_barrier<VM_KEEP0>();
    static_for<0, PD>([&](auto ksc) {
        constexpr int ks = decltype(ksc)::value;
        static_for<0, FR>([&](auto rc) { read_any(rc, glds, colk[ks], colk2[ks], fa[ks], fb[ks]); });
    });
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (!C::LAG)
        issue_stage<C, GLU, BKE>(glds + (C::STAGES - 1) * C::STAGE_BYTES, ra, rb, rb2, a_off, a_k, b_off, b_k,
                                 wave, g0 + C::STAGES - 1, gend);
    __builtin_amdgcn_sched_barrier(0);
    prefetch_a(g0 + PF_AHEAD - 1);
    __builtin_amdgcn_sched_barrier(0);

    int cur_stage = 0;
    auto k_step = [&](int it, auto phc, auto fullc) {
        constexpr int PH = decltype(phc)::value;   // it % UNROLL
        constexpr bool FULL = decltype(fullc)::value;   // the refill step lies wholly below kend
        const int next_stage = cur_stage + 1 == C::STAGES ? 0 : cur_stage + 1;
        char *const cur = glds + cur_stage * C::STAGE_BYTES;
        const char *const nxt = glds + next_stage * C::STAGE_BYTES;
        // The buffer refilled during this step and the step it receives.
        const int prev_stage = cur_stage == 0 ? C::STAGES - 1 : cur_stage - 1;
        char *const dst = C::LAG ? glds + prev_stage * C::STAGE_BYTES : cur;
        const int refill = g0 + it + (C::LAG ? C::STAGES - 1 : C::STAGES);
        const int64_t kbase = static_cast<int64_t>(refill) * BKE;
        const uint32_t kbytes = static_cast<uint32_t>(refill) * C::ROW_BYTES;
        static_for<0, KS>([&](auto ksc) {
            constexpr int ks = decltype(ksc)::value;
            if constexpr (ks == KS - PD) stage_barrier<VM_KEEP + PFN>();
            constexpr int set = (PH * KS + ks) % NSETS;
            constexpr int tgt = ks + PD;              // sub-step whose fragments are read
            constexpr int tset = (PH * KS + tgt) % NSETS;
            const char *const src = tgt < KS ? cur : nxt;
            const int tcol = colk[tgt % KS], tcol2 = colk2[tgt % KS];
            static_for<0, MF>([&](auto tc) {
                constexpr int t = decltype(tc)::value;
                constexpr int i = t / FTN, j = t % FTN;
                if constexpr (C::M16)
                {
                    if constexpr (C::AACC)
                        mfma16_agpr(acc16[i][j], fa[set][i], fb[set][j]);
                    else if constexpr (I8)
                        acc16[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4, fa[set][i]),
                                                                            __builtin_bit_cast(i32x4, fb[set][j]),
                                                                            acc16[i][j], 0, 0, 0);
                    else
                        acc16[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[set][i], fb[set][j], acc16[i][j], 0,
                                                                              0, 0);
                }
                else if constexpr (I8)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(__builtin_bit_cast(i32x4, fa[set][i]),
                                                                      __builtin_bit_cast(i32x4, fb[set][j]),
                                                                      acc[i][j], 0, 0, 0);
                else if constexpr (F8)
                    // A and B as E4M3 (format codes 0), unit E8M0 scales (127).
                    acc[i][j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(fa[set][i], fb[set][j], acc[i][j], 0,
                                                                                0, 0, 127, 0, 127);
                else
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[set][i], fb[set][j], acc[i][j], 0, 0, 0);
                // AGPR tile: the reads before the barrier go in the first
                // three quarters of the sub-step's slots, so that they have
                // landed when the barrier waits for them; the reads after
                // it go in the first quarter, one per slot, ahead of most of
                // the refill loads (a wave's LDS reads complete after its
                // earlier LDS-direct loads have written their data).
                constexpr int RS = !C::AACC ? MF : ks < KS - PD ? MF * 3 / 4 : MF / 4;
                if constexpr (t < RS)
                    static_for<t * FR / RS, (t + 1) * FR / RS>(
                        [&](auto rc) { read_any(rc, src, tcol, tcol2, fa[tset], fb[tset]); });
                if constexpr (C::LAG) {
                    constexpr int u = ks * MF + t;
                    static_for<u * C::LOADS / SLOTS, (u + 1) * C::LOADS / SLOTS>([&](auto q) {
                        issue_load<C, decltype(q)::value, GLU, FULL>(dst, ra, rb, rb2, a_off, a_k, b_off, b_k, wave,
                                                               kbase, kbytes, gend);
                    });
                } else if constexpr (ks >= KS - PD) {
                    constexpr int u = (ks - (KS - PD)) * MF + t;
                    static_for<u * C::LOADS / POST, (u + 1) * C::LOADS / POST>([&](auto q) {
                        issue_load<C, decltype(q)::value, GLU, FULL>(dst, ra, rb, rb2, a_off, a_k, b_off, b_k, wave,
                                                               kbase, kbytes, gend);
                    });
                }
                __builtin_amdgcn_sched_barrier(0);
                if constexpr (PFN > 0 && ks == KS - 1 && t == MF - 1) {
                    prefetch_a(g0 + it + PF_AHEAD);
                    __builtin_amdgcn_sched_barrier(0);
                }
            });
        });
        cur_stage = next_stage;
    };
    const int iters_run = (iters + UNROLL - 1) / UNROLL * UNROLL;
    int it = 0;
    if constexpr (UNROLL == 1) {
        // Iterations whose refill step lies wholly below kend skip the
        // per-chunk K check: a second copy of the loop body takes the rest
        // (a partial last step, the steps past the range).
        const int full_iters = static_cast<int>(kend / BKE) - g0 - (C::LAG ? C::STAGES - 1 : C::STAGES);
        for (; it < full_iters; ++it) k_step(it, std::integral_constant<int, 0>{}, std::true_type{});
    }
    for (; it < iters_run; it += UNROLL)
        static_for<0, UNROLL>([&](auto ph) { k_step(it + decltype(ph)::value, ph, std::false_type{}); });
    // The compiler does not see the inline-assembly MFMAs, so it cannot
    // space their last AGPR writes from the first reads below: 32 idle
    // cycles cover the longest required gap of a 16x16x32 MFMA.
    if constexpr (C::AACC) asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");

    // Epilogue.  Accumulator element e of a 32x32 block sits at row
    // 8*(e/4) + 4*hi + e%4 and column lane % 32.  Each 32-row slab of the
    // wave's block goes through LDS as fp32 so that every lane then owns 8
    // consecutive columns: R is read and Y written 16 bytes at a time
    // through buffer resources bounded to the tile's rows (rows past M are
    // dropped by the range check; columns past N are pointed out of range).
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));   // trailing LDS-direct loads have landed
    __syncthreads();                             // every wave is done with the stage buffers

    if (piece) {
        // Split-K hand-off.  Partial tiles cross workgroups only through
        // device-scope (sc1) stores, which write through the XCD's L2, and
        // device-scope loads, which bypass stale L2 lines, so no L2-wide
        // write-back or invalidate is needed.  Slices are laid out in
        // fragment order (each store instruction writes 1 KB contiguous).
        // Each split tile owns an arrival counter, zero between calls.
        constexpr int TILE_FLOATS = C::BM * C::BN;
        constexpr int NB = C::TM * C::TN * 4;        // accumulator quads per lane
        const int64_t stile = tile - sk.full_tiles;   // index among the split tiles
        unsigned *const arrived = sk.counters + stile;
        const float *first = sk.partials + stile * sk.split * TILE_FLOATS;
        const __amdgpu_buffer_rsrc_t rp =
            make_rsrc(first, static_cast<uint32_t>(sk.split) * TILE_FLOATS * 4u);
        const uint32_t mine = static_cast<uint32_t>(slice) * TILE_FLOATS * 4u;
        const int wblk = wave * C::TM * C::TN;
        auto publish = [&] {
#pragma unroll
            for (int i = 0; i < C::TM; ++i)
#pragma unroll
                for (int j = 0; j < C::TN; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const f32x4 v = __builtin_bit_cast(f32x4, quad_of(i, j, q));
                        const uint32_t off = mine + (((wblk + i * C::TN + j) * 4 + q) * 64 + lane) * 16;
                        __builtin_amdgcn_raw_buffer_store_b128(v, rp, off, 0, AUX_SC1);
                    }
            __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));   // this wave's slice stores are complete
        };
        int *flag = reinterpret_cast<int *>(lds);
        // Every slice publishes itself and then counts its arrival; the last
        // to arrive adds the slices in slice order.  With 64x64 wave blocks
        // (16 quads per lane: the sum still fits beside the accumulators) the
        // last arriver takes its own slice from its registers instead of
        // reading it back (one slice less through memory: 5 % at M = 512,
        // N = K = 5120); other blocks read every slice back (for 32x32 wave
        // blocks the register form measured 1-2 % slower).
        constexpr bool SHORT = NB == 16;
        publish();
        __syncthreads();                          // every wave's stores are complete
        if (threadIdx.x == 0) {
            const unsigned prev = __hip_atomic_fetch_add(arrived, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            *flag = prev == static_cast<unsigned>(sk.split - 1);
        }
        __syncthreads();
        const bool last = *flag != 0;
        __syncthreads();                          // the flag is read before LDS is reused
        if (!last) return;
        if constexpr (SHORT) {
            // D slices per round trip (their loads fit in 64 registers); the
            // own slice and slices past the last are not loaded.
            constexpr int D = 64 / (NB * 4) > 8 ? 8 : (64 / (NB * 4) < 1 ? 1 : 64 / (NB * 4));
            AccQ sum[NB];
#pragma unroll
            for (int b = 0; b < NB; ++b) sum[b] = AccQ{0, 0, 0, 0};
            for (int t0 = 0; t0 < sk.split; t0 += D) {
                f32x4 v[D][NB];
#pragma unroll
                for (int d = 0; d < D; ++d) {
                    const int t = t0 + d;
                    const bool other = t < sk.split && t != static_cast<int>(slice);
                    const uint32_t base = static_cast<uint32_t>(t) * TILE_FLOATS * 4u;
#pragma unroll
                    for (int b = 0; b < NB; ++b)
                        v[d][b] = __builtin_bit_cast(
                            f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                       rp, other ? base + ((wblk * 4 + b) * 64 + lane) * 16 : OOB_OFFSET, 0, AUX_SC1));
                }
#pragma unroll
                for (int d = 0; d < D; ++d) {
                    const int t = t0 + d;
                    if (t >= sk.split) break;
#pragma unroll
                    for (int i = 0; i < C::TM; ++i)
#pragma unroll
                        for (int j = 0; j < C::TN; ++j)
#pragma unroll
                            for (int q = 0; q < 4; ++q) {
                                const int b = (i * C::TN + j) * 4 + q;
                                if (t == static_cast<int>(slice)) sum[b] += quad_of(i, j, q);
                                else add_bits(sum[b], v[d][b]);
                            }
                }
            }
#pragma unroll
            for (int i = 0; i < C::TM; ++i)
#pragma unroll
                for (int j = 0; j < C::TN; ++j)
#pragma unroll
                    for (int q = 0; q < 4; ++q) quad_set(i, j, q, sum[(i * C::TN + j) * 4 + q]);
        } else {
            zero_acc();
            // Small tiles: D slices per round trip (as many as 128 registers
            // hold); a slice past the last reads out of range and is not added,
            // so the sum still runs over the slices in order.  Large tiles
            // (a slice fills 128 registers) go one slice at a time.
            constexpr int D = NB * 4 >= 128 ? 1 : (128 / (NB * 4) > 8 ? 8 : 128 / (NB * 4));
            if constexpr (D == 1) {
                for (int t = 0; t < sk.split; ++t) {
                    const uint32_t base = static_cast<uint32_t>(t) * TILE_FLOATS * 4u;
#pragma unroll
                    for (int i = 0; i < C::TM; ++i)
#pragma unroll
                        for (int j = 0; j < C::TN; ++j)
#pragma unroll
                            for (int q = 0; q < 4; ++q) {
                                const uint32_t off = base + (((wblk + i * C::TN + j) * 4 + q) * 64 + lane) * 16;
                                quad_ref_add(i, j, q,
                                             __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                                               rp, off, 0, AUX_SC1)));
                            }
                }
            } else {
                for (int t0 = 0; t0 < sk.split; t0 += D) {
                    f32x4 v[D][NB];
#pragma unroll
                    for (int d = 0; d < D; ++d) {
                        const uint32_t base = static_cast<uint32_t>(t0 + d) * TILE_FLOATS * 4u;
#pragma unroll
                        for (int b = 0; b < NB; ++b)
                            v[d][b] = __builtin_bit_cast(
                                f32x4, __builtin_amdgcn_raw_buffer_load_b128(rp, base + ((wblk * 4 + b) * 64 + lane) * 16,
                                                                             0, AUX_SC1));
                    }
#pragma unroll
                    for (int d = 0; d < D; ++d) {
                        if (t0 + d >= sk.split) break;
#pragma unroll
                        for (int i = 0; i < C::TM; ++i)
#pragma unroll
                            for (int j = 0; j < C::TN; ++j)
#pragma unroll
                                for (int q = 0; q < 4; ++q) quad_ref_add(i, j, q, v[d][(i * C::TN + j) * 4 + q]);
                    }
                }
            }
        }
        if (threadIdx.x == 0) __hip_atomic_store(arrived, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if constexpr (R_ALL) {
        if (vec && has_r)
#pragma unroll
            for (int i = 0; i < C::TM; ++i) load_r(i, rv[i]);
    } else if constexpr (!EARLY_R) {
        if (vec && has_r) load_r(0, rv[0]);
    }
    // The bias of the lane's 8 columns (fixed for the whole tile).
    float bv[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (has_bias) {
        const __amdgpu_buffer_rsrc_t rbias = make_rsrc(bias_of(p), static_cast<uint32_t>(N * 2));
#pragma unroll
        for (int t = 0; t < 8; ++t)
            bv[t] = bf16_to_f32(__builtin_amdgcn_raw_buffer_load_b16(
                rbias, col0 + t < N ? static_cast<uint32_t>((col0 + t) * 2) : OOB_OFFSET, 0, 0));
    }
    float *ep = reinterpret_cast<float *>(lds) + wave * C::EPI_WAVE_FLOATS;
#pragma unroll
    for (int i = 0; i < C::TM; ++i) {
        if (!R_ALL && vec && has_r && i + 1 < C::TM) load_r(i + 1, rv[rslot(i + 1)]);
        if constexpr (Q8)
            if (i + 1 < C::TM) load_sx(i + 1);
        {
            if constexpr (GLU) {
                // Block 2j holds the gate sums and block 2j+1 the up sums of
                // the same 32 outputs, element for element.
#pragma unroll
                for (int j = 0; j < C::TN / 2; ++j)
#pragma unroll
                    for (int e = 0; e < 16; ++e) {
                        float g, u;
                        if constexpr (Q8) {
                            const float sr = sxr[i & 1][e];
                            g = static_cast<float>(quad_of(i, 2 * j, e >> 2)[e & 3]) * (sr * swc[j]);
                            u = static_cast<float>(quad_of(i, 2 * j + 1, e >> 2)[e & 3]) * (sr * swc[C::TN / 2 + j]);
                        } else {
                            g = quad_of(i, 2 * j, e >> 2)[e & 3];
                            u = quad_of(i, 2 * j + 1, e >> 2)[e & 3];
                        }
                        if constexpr (C::M16)
                            ep[(16 * (e >> 3) + 4 * hi + (e & 3)) * EPS + j * 32 + 16 * ((e >> 2) & 1) + frag_row] =
                                silu_f32(g) * u;
                        else
                            ep[(8 * (e >> 2) + 4 * hi + (e & 3)) * EPS + j * 32 + frag_row] = silu_f32(g) * u;
                    }
            } else {
#pragma unroll
                for (int j = 0; j < C::TN; ++j)
#pragma unroll
                    for (int e = 0; e < 16; ++e) {
                        if constexpr (C::M16)   // quad q = e/4: rows 16*(q/2) + 4*hi + e%4, columns 16*(q%2) + lane%16
                            ep[(16 * (e >> 3) + 4 * hi + (e & 3)) * EPS + j * 32 + 16 * ((e >> 2) & 1) + frag_row] =
                                static_cast<float>(quad_of(i, j, e >> 2)[e & 3]);
                        else
                            ep[(8 * (e >> 2) + 4 * hi + (e & 3)) * EPS + j * 32 + frag_row] =
                                static_cast<float>(quad_of(i, j, e >> 2)[e & 3]);
                    }
            }
        }
        // The slab's staging area is the wave's own, so only LDS order
        // matters here: the Y stores of the previous slab keep flowing
        // (a __syncthreads() would wait for them to complete).
        lds_barrier();
        {
#pragma unroll
            for (int v = 0; v < PASSES; ++v) {
                const float *src = ep + (v * RPP + pr) * EPS + pc;
                float y[8];
#pragma unroll
                for (int t = 0; t < 8; ++t) y[t] = src[t];
                if constexpr (Q8 && !GLU) {
                    const float sr = sxr[i & 1][v];
#pragma unroll
                    for (int t = 0; t < 8; ++t) y[t] *= sr * swc[t];
                }
                const uint32_t base = base_of(i, v);
                if (vec) {
                    if constexpr (GEN) {
#pragma unroll
                        for (int t = 0; t < 4; ++t) {
                            const uint32_t w = static_cast<uint32_t>(rv[rslot(i)][v][t]);
                            y[2 * t] = value(y[2 * t], bf16_to_f32(static_cast<uint16_t>(w & 0xffffu)));
                            y[2 * t + 1] = value(y[2 * t + 1], bf16_to_f32(static_cast<uint16_t>(w >> 16)));
                        }
                        if (has_bias) {
#pragma unroll
                            for (int t = 0; t < 8; ++t) y[t] += bv[t];
                        }
                    } else if (has_r) {
#pragma unroll
                        for (int t = 0; t < 4; ++t) {
                            const uint32_t w = static_cast<uint32_t>(rv[rslot(i)][v][t]);
                            y[2 * t] += bf16_to_f32(static_cast<uint16_t>(w & 0xffffu));
                            y[2 * t + 1] += bf16_to_f32(static_cast<uint16_t>(w >> 16));
                        }
                    }
                    i32x4 out;
#pragma unroll
                    for (int t = 0; t < 4; ++t) out[t] = static_cast<int>(f32x2_to_bf16x2_rne(y[2 * t], y[2 * t + 1]));
                    __builtin_amdgcn_raw_buffer_store_b128(out, ry, col0 < N ? base : OOB_OFFSET, 0, AUX_NT);
                } else {
                    uint16_t rs[8];
                    const int cols = static_cast<int>(N - col0);   // columns of this lane's 8 that exist
                    const uint32_t rbase = rbase_of(i, v);
#pragma unroll
                    for (int t = 0; t < 8; ++t) rs[t] = __builtin_amdgcn_raw_buffer_load_b16(rr, t < cols ? rbase + 2 * t : OOB_OFFSET, 0, 0);
#pragma unroll
                    for (int t = 0; t < 8; ++t) {
                        float yt = value(y[t], bf16_to_f32(rs[t]));
                        if (has_bias) yt += bv[t];
                        __builtin_amdgcn_raw_buffer_store_b16(f32_to_bf16_rne(yt), ry, t < cols ? base + 2 * t : OOB_OFFSET, 0, 0);
                    }
                }
            }
        }
        lds_barrier();   // the staging area is read before the next slab overwrites it
    }
}

// Split-K arguments of one launch; false when a tail split cannot hand
// the XCDs equal shares of both kinds of work.
// BKE: K elements per stage (C::BK for bf16 operands, 2 * C::BK for int8).
template <class C, int BKE = C::BK>
bool split_args(int64_t K, int64_t tiles, int split, int64_t full_tiles, const Workspace *ws, SplitK &sk) {
    sk = SplitK{1, ((K + BKE - 1) / BKE) * BKE, nullptr, nullptr, 0};
    if (split > 1) {
        sk.split = split;
        sk.kslice = (((K + split - 1) / split + BKE - 1) / BKE) * BKE;
        sk.partials = ws->partials;
        sk.counters = ws->counters;
        sk.full_tiles = full_tiles;
        if (full_tiles > 0 && (full_tiles >= tiles || full_tiles % XCDS != 0 ||
                               ((tiles - full_tiles) * split) % XCDS != 0))
            return false;
    }
    return true;
}

template <class C>
hipError_t launch_cfg(const Problem &p, int group_m, int split, int64_t full_tiles, const Workspace *ws,
                      hipStream_t s) {
    const int64_t tiles_m = (p.M + C::BM - 1) / C::BM;
    const int64_t tiles_n = (p.N + C::BN - 1) / C::BN;
    const int64_t tiles = tiles_m * tiles_n;
    SplitK sk;
    if (!split_args<C>(p.K, tiles, split, full_tiles, ws, sk)) return hipErrorInvalidValue;
    const int64_t wgs = sk.full_tiles + (tiles - sk.full_tiles) * sk.split;
    if (is_general(p))
        hipLaunchKernelGGL((tile_kernel<C, Problem>), dim3(static_cast<unsigned>(wgs)), dim3(C::THREADS), 0, s, p,
                           tiles_m, tiles_n, group_m, sk);
    else
        hipLaunchKernelGGL((tile_kernel<C, DenseProblem>), dim3(static_cast<unsigned>(wgs)), dim3(C::THREADS), 0, s,
                           dense_of(p), tiles_m, tiles_n, group_m, sk);
    return hipGetLastError();
}

template <class C>
hipError_t launch_cfg_i8(const I8Problem &p, int group_m, int split, int64_t full_tiles, const Workspace *ws,
                         hipStream_t s) {
    {
        const int64_t tiles_m = (p.M + C::BM - 1) / C::BM;
        const int64_t tiles_n = (p.N + C::BN - 1) / C::BN;
        const int64_t tiles = tiles_m * tiles_n;
        SplitK sk;
        if (!split_args<C, 2 * C::BK>(p.K, tiles, split, full_tiles, ws, sk)) return hipErrorInvalidValue;
        const int64_t wgs = sk.full_tiles + (tiles - sk.full_tiles) * sk.split;
        hipLaunchKernelGGL((tile_kernel<C, I8Problem>), dim3(static_cast<unsigned>(wgs)), dim3(C::THREADS), 0, s, p,
                           tiles_m, tiles_n, group_m, sk);
        return hipGetLastError();
    }
}

// SwiGLU needs an even number of 32-column blocks per wave (gate/up pairs)
// and an even number of B loads per wave (half gate, half up).  (With 16x16
// MFMAs the gate and up blocks of a pair still hold their values in the same
// element order, so the pairing is the same.)
template <class C>
constexpr bool glu_ok() { return C::TN % 2 == 0 && C::B_LOADS % 2 == 0 && 32 % C::RPI == 0; }

template <class C>
hipError_t launch_cfg_glu(const GluProblem &p, int group_m, int split, int64_t full_tiles, const Workspace *ws,
                          hipStream_t s) {
    if constexpr (!glu_ok<C>()) {
        return hipErrorInvalidValue;
    } else {
        const int64_t tiles_m = (p.M + C::BM - 1) / C::BM;
        const int64_t tiles_n = (p.N + C::BN / 2 - 1) / (C::BN / 2);
        const int64_t tiles = tiles_m * tiles_n;
        SplitK sk;
        if (!split_args<C>(p.K, tiles, split, full_tiles, ws, sk)) return hipErrorInvalidValue;
        const int64_t wgs = sk.full_tiles + (tiles - sk.full_tiles) * sk.split;
        hipLaunchKernelGGL((tile_kernel<C, GluProblem>), dim3(static_cast<unsigned>(wgs)), dim3(C::THREADS), 0, s,
                           p, tiles_m, tiles_n, group_m, sk);
        return hipGetLastError();
    }
}

template <class C>
hipError_t launch_cfg_i8_glu(const I8GluProblem &p, int group_m, int split, int64_t full_tiles, const Workspace *ws,
                             hipStream_t s) {
    if constexpr (!glu_ok<C>() || C::M16) {   // (the INT8 SwiGLU epilogue reads the 32x32 layout)
        return hipErrorInvalidValue;
    } else {
        const int64_t tiles_m = (p.M + C::BM - 1) / C::BM;
        const int64_t tiles_n = (p.N + C::BN / 2 - 1) / (C::BN / 2);
        const int64_t tiles = tiles_m * tiles_n;
        SplitK sk;
        if (!split_args<C, 2 * C::BK>(p.K, tiles, split, full_tiles, ws, sk)) return hipErrorInvalidValue;
        const int64_t wgs = sk.full_tiles + (tiles - sk.full_tiles) * sk.split;
        hipLaunchKernelGGL((tile_kernel<C, I8GluProblem>), dim3(static_cast<unsigned>(wgs)), dim3(C::THREADS), 0, s,
                           p, tiles_m, tiles_n, group_m, sk);
        return hipGetLastError();
    }
}

// Tile shape, K depth, wave grid, pipeline depth and occupancy of each tile
// configuration: Cfg<BM, BN, BK, WAVES_M, WAVES_N, STAGES, WAVES_PER_EU, LAG, M16, AACC>.
using C256x256w8 = Cfg<256, 256, 64, 2, 4, 2, 2>;
using C256x256w4m16a = Cfg<256, 256, 64, 2, 2, 2, 1, false, true, true>;
using C256x128s3w8 = Cfg<256, 128, 64, 4, 2, 3, 2>;
using C256x128s3w8L = Cfg<256, 128, 64, 4, 2, 3, 2, true>;
using C128x128w4 = Cfg<128, 128, 64, 2, 2, 2, 2>;
using C128x128s3 = Cfg<128, 128, 64, 2, 2, 3, 1>;
using C128x128s4L = Cfg<128, 128, 64, 2, 2, 4, 1, true>;
using C64x64k128s3 = Cfg<64, 64, 128, 2, 2, 3, 1>;
using C64x64k64s4 = Cfg<64, 64, 64, 2, 2, 4, 2>;
using C64x128k64s4 = Cfg<64, 128, 64, 2, 2, 4, 1>;

// Workgroups per CU that each configuration's LDS and registers allow, and
// the dispatch from a TileCfg value to its type: f(C{}, per_cu).
template <class F>
auto with_cfg(int cfg, F &&f) -> decltype(f(C256x256w8{}, 1)) {
    switch (cfg) {
        case TC_256x256_K64_S2_W8: return f(C256x256w8{}, 1);
        case TC_256x256_K64_S2_W4_M16A: return f(C256x256w4m16a{}, 1);
        case TC_256x128_K64_S3_W8: return f(C256x128s3w8{}, 1);
        case TC_256x128_K64_S3_W8_L: return f(C256x128s3w8L{}, 1);
        case TC_128x128_K64_S2_W4: return f(C128x128w4{}, 2);
        case TC_128x128_K64_S3_W4: return f(C128x128s3{}, 1);
        case TC_128x128_K64_S4_W4_L: return f(C128x128s4L{}, 1);
        case TC_64x64_K128_S3_W4: return f(C64x64k128s3{}, 1);
        case TC_64x64_K64_S4_W4: return f(C64x64k64s4{}, 2);
        case TC_64x128_K64_S4_W4: return f(C64x128k64s4{}, 1);
        default: return f(nullptr, 0);
    }
}

// Grouped forms: one launch of G * m-tiles-per-group * n-tiles workgroups,
// no split-K.
template <class C, class B>
hipError_t launch_cfg_grouped(const Grouped<B> &p, hipStream_t s) {
    constexpr bool GLU = std::is_same<B, GluProblem>::value;
    if constexpr (GLU && !glu_ok<C>()) {
        return hipErrorInvalidValue;
    } else {
        constexpr int BNO = GLU ? C::BN / 2 : C::BN;
        const int64_t tiles_m = p.G * ((p.Mpad + C::BM - 1) / C::BM);
        const int64_t tiles_n = (p.N + BNO - 1) / BNO;
        SplitK sk;
        if (!split_args<C>(p.K, tiles_m * tiles_n, 1, 0, nullptr, sk)) return hipErrorInvalidValue;
        hipLaunchKernelGGL((tile_kernel<C, Grouped<B>>), dim3(static_cast<unsigned>(tiles_m * tiles_n)),
                           dim3(C::THREADS), 0, s, p, tiles_m, tiles_n, 8, sk);
        return hipGetLastError();
    }
}

// FP8 needs sub-steps of 64 K bytes that split into fragment-prefetch sets.
template <class C>
constexpr bool f8_ok() { return !C::M16 && C::KSTEPS / 2 > C::PD && (C::KSTEPS / 2) % (C::PD + 1) == 0; }

template <class C, class P>
hipError_t launch_cfg_q8(const P &p, int group_m, int split, int64_t full_tiles, const Workspace *ws,
                         hipStream_t s) {
    constexpr bool GLU = std::is_same<P, F8GluProblem>::value;
    if constexpr (!f8_ok<C>() || (GLU && !glu_ok<C>())) {
        return hipErrorInvalidValue;
    } else {
        constexpr int BNO = GLU ? C::BN / 2 : C::BN;
        const int64_t tiles_m = (p.M + C::BM - 1) / C::BM;
        const int64_t tiles_n = (p.N + BNO - 1) / BNO;
        const int64_t tiles = tiles_m * tiles_n;
        SplitK sk;
        if (!split_args<C, 2 * C::BK>(p.K, tiles, split, full_tiles, ws, sk)) return hipErrorInvalidValue;
        const int64_t wgs = sk.full_tiles + (tiles - sk.full_tiles) * sk.split;
        hipLaunchKernelGGL((tile_kernel<C, P>), dim3(static_cast<unsigned>(wgs)), dim3(C::THREADS), 0, s, p, tiles_m,
                           tiles_n, group_m, sk);
        return hipGetLastError();
    }
}

}  // namespace
}  // namespace kernelarc
