// MFMA macro-tile kernels for Y = X W^T (+ R): the compute-bound path.
//
// One workgroup of four waves computes a BM x BN output tile; each wave owns
// a (BM/2) x (BN/2) quadrant built from 32x32 accumulator blocks of
// v_mfma_f32_32x32x16_bf16 (bf16 inputs, fp32 accumulation).
//
// Data path per 64-deep K step (the paper's Table 2 tiers 2-7 -- tensor-core
// substrate, asynchronous copy, software pipelining, epilogue and tile
// scheduling -- re-derived for CDNA4 rather than Hopper):
//   * staging: buffer_load_dwordx4 with the LDS bit moves 16 bytes per lane
//     straight from HBM/L2 into LDS (no VGPR round trip).  Each instruction
//     covers 8 rows x 128 contiguous bytes of one operand, so every row read
//     is a whole 128-byte line.  Two stages: the loads for step kt+1 are in
//     flight while step kt is multiplied.
//   * LDS layout: 128 bytes per row (64 bf16 of K); the 16-byte chunk c of
//     row r is stored at slot c ^ swz(r).  A wave's ds_read_b128 of one
//     fragment touches 32 rows at one chunk; the swizzle spreads any 8 (or
//     16) consecutive rows over distinct bank groups.
//   * buffer resources bound each operand panel, so rows past M/N read as
//     zero without any branch; K-tail chunks are pointed out of range.
//   * epilogue: fp32 accumulator + fp32(R) rounded once to bf16 (nearest
//     even); each output element is read (R) and written (Y) by the same
//     lane, so Y may alias R.
//   * tile scheduler: workgroups are handed to the 8 XCDs round-robin; the
//     id is remapped so each XCD works on a contiguous range of tiles, and
//     that range is walked in GROUP_M-row super-tiles so that the tiles
//     resident on one XCD share X and W panels in its L2.
#include "internal.h"

namespace kernelarc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

// Word 3 of a raw (unswizzled, stride 0) gfx9 buffer resource.
constexpr int RSRC_WORD3 = 0x00020000;
// A byte offset that is out of range for every panel (panels are < 2^31 B).
constexpr uint32_t OOB_OFFSET = 0x80000000u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), static_cast<short>(0),
                                             static_cast<int>(bytes), RSRC_WORD3);
}

// Slot of 16-byte chunk c of row r is c ^ swz(r).
__device__ __forceinline__ int swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

constexpr int XCDS = 8;

// blockIdx -> (tile_m, tile_n).  Dispatch places workgroup b on XCD b % 8;
// XCD x is given the logical ids [start_x, start_x + count_x) in order, and
// logical ids run over GROUP_M-row bands column by column.
__device__ __forceinline__ void schedule(int64_t bid, int64_t tiles_m, int64_t tiles_n, int group_m,
                                         int64_t &tm, int64_t &tn) {
    const int64_t T = tiles_m * tiles_n;
    const int64_t per = T / XCDS;
    const int64_t rem = T % XCDS;
    const int64_t x = bid % XCDS;
    const int64_t local = bid / XCDS;
    const int64_t logical = x * per + (x < rem ? x : rem) + local;
    const int64_t band = static_cast<int64_t>(group_m) * tiles_n;
    const int64_t g = logical / band;
    const int64_t first_m = g * group_m;
    const int64_t rows = (tiles_m - first_m) < group_m ? (tiles_m - first_m) : group_m;
    const int64_t in_band = logical - g * band;
    tm = first_m + in_band % rows;
    tn = in_band / rows;
}

template <int BM_, int BN_, int WAVES_PER_EU_>
struct Cfg {
    static constexpr int BM = BM_, BN = BN_, BK = 64;
    static constexpr int WAVES = 4, THREADS = 256;
    static constexpr int WM = BM / 2, WN = BN / 2;        // per-wave quadrant
    static constexpr int TM = WM / 32, TN = WN / 32;      // 32x32 blocks per wave
    static constexpr int A_BYTES = BM * BK * 2, B_BYTES = BN * BK * 2;
    static constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
    static constexpr int STAGES = 2;
    static constexpr int LDS_BYTES = STAGES * STAGE_BYTES;
    static constexpr int A_LOADS = BM / 8 / WAVES;        // 8-row blocks per wave per step
    static constexpr int B_LOADS = BN / 8 / WAVES;
    static constexpr int WAVES_PER_EU = WAVES_PER_EU_;
    // Epilogue staging: one 32-row slab of a wave's quadrant in fp32, rows
    // padded by 4 floats; lanes then read 8 consecutive columns each.
    static constexpr int EPI_STRIDE = WN + 4;
    static constexpr int EPI_WAVE_FLOATS = 32 * EPI_STRIDE;
    static constexpr int LANES_PER_ROW = WN / 8;
    static constexpr int ROWS_PER_PASS = 64 / LANES_PER_ROW;
    static_assert(4 * EPI_WAVE_FLOATS * 4 <= LDS_BYTES, "epilogue staging fits in the stage buffers");
};

// Enqueue the LDS-direct loads of K step kt into one stage.  Load block blk
// (8 rows) of a wave has the parity of q (A_LOADS and B_LOADS are even), so
// the lane's source chunk is c_even ^ (q & 1); chunks at or past K are
// pointed out of range and arrive as zeros.
template <class C>
__device__ __forceinline__ void issue_stage(char *stage, const __amdgpu_buffer_rsrc_t &ra,
                                            const __amdgpu_buffer_rsrc_t &rb, const uint32_t *a_off,
                                            const uint32_t *b_off, int wave, int kt, int64_t K,
                                            int c_even) {
    const int64_t kbase = static_cast<int64_t>(kt) * C::BK;
    const bool ok_even = kbase + c_even * 8 < K;
    const bool ok_odd = kbase + (c_even ^ 1) * 8 < K;
    const uint32_t kbytes = static_cast<uint32_t>(kt) * (C::BK * 2);
#pragma unroll
    for (int q = 0; q < C::A_LOADS; ++q) {
        const int blk = wave * C::A_LOADS + q;
        const bool ok = (q & 1) ? ok_odd : ok_even;
        const uint32_t off = ok ? a_off[q] + kbytes : OOB_OFFSET;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void *)(stage + blk * 1024), 16, off, 0, 0, 0);
    }
#pragma unroll
    for (int q = 0; q < C::B_LOADS; ++q) {
        const int blk = wave * C::B_LOADS + q;
        const bool ok = (q & 1) ? ok_odd : ok_even;
        const uint32_t off = ok ? b_off[q] + kbytes : OOB_OFFSET;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_void *)(stage + C::A_BYTES + blk * 1024),
                                                 16, off, 0, 0, 0);
    }
}

// MFMA operands of K sub-step ks (16 deep) from one stage: lane l reads row
// l % 32 of each 32-row block at chunk 2*ks + l / 32, whose slot is
// (2*ks) ^ slot_base with slot_base = (l / 32) ^ swz(l % 32).
template <class C>
__device__ __forceinline__ void load_fragments(const char *a_base, const char *b_base, int slot_base,
                                               int ks, bf16x8 *af, bf16x8 *bfr) {
    const int col = ((2 * ks) ^ slot_base) * 16;
#pragma unroll
    for (int i = 0; i < C::TM; ++i) af[i] = *reinterpret_cast<const bf16x8 *>(a_base + i * 32 * 128 + col);
#pragma unroll
    for (int j = 0; j < C::TN; ++j) bfr[j] = *reinterpret_cast<const bf16x8 *>(b_base + j * 32 * 128 + col);
}

// Sub-step scheduling: MFMA number T of a sub-step is followed by its share
// of the LDS reads (next sub-step's fragments) and of the VMEM loads (next
// stage), spread evenly over the MFMAS MFMAs.
template <int MFMAS, int READS, int LOADS, int T>
__device__ __forceinline__ void interleave() {
    constexpr int MFMA = 0x008, VMEM_READ = 0x020, DS_READ = 0x100;
    constexpr int r = ((T + 1) * READS) / MFMAS - (T * READS) / MFMAS;
    constexpr int l = ((T + 1) * LOADS) / MFMAS - (T * LOADS) / MFMAS;
    __builtin_amdgcn_sched_group_barrier(MFMA, 1, 0);
    if constexpr (l > 0) __builtin_amdgcn_sched_group_barrier(VMEM_READ, l, 0);
    if constexpr (r > 0) __builtin_amdgcn_sched_group_barrier(DS_READ, r, 0);
    if constexpr (T + 1 < MFMAS) interleave<MFMAS, READS, LOADS, T + 1>();
}

// Instruction order of one K step, pinned because the default schedule
// funnels every fragment through one register set and waits for each LDS
// read just before its MFMAs (one wave per SIMD cannot hide that).  Order:
// the fragment reads of sub-step 0; then sub-step 0's MFMAs interleaved with
// the next stage's LDS-direct loads and sub-step 1's fragment reads; then
// each further sub-step's MFMAs interleaved with the following sub-step's
// reads; the last sub-step's MFMAs alone.
template <class C>
__device__ __forceinline__ void schedule_k_step() {
    constexpr int FRAGS = C::TM + C::TN;          // LDS reads per sub-step
    constexpr int MFMAS = C::TM * C::TN;          // MFMAs per sub-step
    constexpr int LOADS = C::A_LOADS + C::B_LOADS;
    __builtin_amdgcn_sched_group_barrier(0x100, FRAGS, 0);
    interleave<MFMAS, FRAGS, LOADS, 0>();
    interleave<MFMAS, FRAGS, 0, 0>();
    interleave<MFMAS, FRAGS, 0, 0>();
    __builtin_amdgcn_sched_group_barrier(0x008, MFMAS, 0);
}

template <class C>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256),
                          amdgpu_waves_per_eu(C::WAVES_PER_EU, C::WAVES_PER_EU)))
void tile_kernel(Problem p, int64_t tiles_m, int64_t tiles_n, int group_m) {
    __shared__ __attribute__((aligned(1024))) char lds[C::LDS_BYTES];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

    int64_t tm, tn;
    schedule(blockIdx.x, tiles_m, tiles_n, group_m, tm, tn);
    const int64_t m0 = tm * C::BM;
    const int64_t n0 = tn * C::BN;
    const int64_t K = p.K;

    // Operand panels bounded by buffer resources: rows past M (N) read 0.
    const int64_t rows_a = (p.M - m0) < C::BM ? (p.M - m0) : C::BM;
    const int64_t rows_b = (p.N - n0) < C::BN ? (p.N - n0) : C::BN;
    const __amdgpu_buffer_rsrc_t ra = make_rsrc(p.X + m0 * K, static_cast<uint32_t>(rows_a * K * 2));
    const __amdgpu_buffer_rsrc_t rb = make_rsrc(p.W + n0 * K, static_cast<uint32_t>(rows_b * K * 2));

    // Per-lane source offsets (bytes, K step 0) of the chunks this lane
    // stages: lane l fills slot l % 8 of row 8*blk + l / 8, which holds
    // global chunk (l % 8) ^ swz(row) = (l % 8) ^ (l / 8) ^ (blk & 1).
    static_assert(C::A_LOADS % 2 == 0 && C::B_LOADS % 2 == 0, "load blocks come in pairs");
    const int lane_row = lane >> 3;
    const int c_even = (lane & 7) ^ lane_row;
    uint32_t a_off[C::A_LOADS], b_off[C::B_LOADS];
#pragma unroll
    for (int q = 0; q < C::A_LOADS; ++q) {
        const int r = (wave * C::A_LOADS + q) * 8 + lane_row;
        a_off[q] = static_cast<uint32_t>(r * K * 2 + (c_even ^ (q & 1)) * 16);
    }
#pragma unroll
    for (int q = 0; q < C::B_LOADS; ++q) {
        const int r = (wave * C::B_LOADS + q) * 8 + lane_row;
        b_off[q] = static_cast<uint32_t>(r * K * 2 + (c_even ^ (q & 1)) * 16);
    }

    f32x16 acc[C::TM][C::TN];
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

    // Fragment read offsets: lane reads row (lane % 32) of each 32-row block
    // at chunk 2*ks + lane / 32, i.e. slot (2*ks + hi) ^ swz(lane % 32).
    const int frag_row = lane & 31;
    const int hi = lane >> 5;
    const int wm0 = (wave >> 1) * C::WM;
    const int wn0 = (wave & 1) * C::WN;
    const int a_row_byte = (wm0 + frag_row) * 128;
    const int b_row_byte = (wn0 + frag_row) * 128;
    const int slot_base = hi ^ swz(frag_row);

    const int nk = static_cast<int>((K + C::BK - 1) / C::BK);

    if (nk > 0) issue_stage<C>(lds, ra, rb, a_off, b_off, wave, 0, K, c_even);

    for (int kt = 0; kt < nk; ++kt) {
        __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): this wave's stage kt is in LDS
        __syncthreads();                        // all waves' too; stage kt+1's buffer is free
        const char *cur = lds + (kt & 1) * C::STAGE_BYTES;
        const char *a_base = cur + a_row_byte;
        const char *b_base = cur + C::A_BYTES + b_row_byte;
        bf16x8 af[2][C::TM], bfr[2][C::TN];
        load_fragments<C>(a_base, b_base, slot_base, 0, af[0], bfr[0]);
        // Unconditional so the scheduler can interleave it: past the end of
        // K every offset is out of range and the loads only write zeros into
        // the idle stage.
        issue_stage<C>(lds + ((kt + 1) & 1) * C::STAGE_BYTES, ra, rb, a_off, b_off, wave, kt + 1, K, c_even);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            if (ks < 3) load_fragments<C>(a_base, b_base, slot_base, ks + 1, af[(ks + 1) & 1], bfr[(ks + 1) & 1]);
#pragma unroll
            for (int i = 0; i < C::TM; ++i)
#pragma unroll
                for (int j = 0; j < C::TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[ks & 1][i], bfr[ks & 1][j],
                                                                        acc[i][j], 0, 0, 0);
        }
        schedule_k_step<C>();
    }

    // Epilogue.  Accumulator element e of a 32x32 block sits at row
    // 8*(e/4) + 4*hi + e%4 and column lane % 32.  Each 32-row slab of the
    // wave's quadrant goes through LDS as fp32 so that every lane then owns
    // 8 consecutive columns: R is read and Y written 16 bytes at a time
    // through buffer resources bounded to the tile's rows (rows past M are
    // dropped by the range check; columns past N are pointed out of range).
    __builtin_amdgcn_s_waitcnt(0x0F70);   // the trailing LDS-direct loads have landed
    __syncthreads();                        // every wave is done with the stage buffers
    float *ep = reinterpret_cast<float *>(lds) + wave * C::EPI_WAVE_FLOATS;
    const int64_t N = p.N;
    const int64_t rows_y = (p.M - m0) < C::BM ? (p.M - m0) : C::BM;
    const uint32_t ybytes = static_cast<uint32_t>(rows_y * N * 2);
    const __amdgpu_buffer_rsrc_t ry = make_rsrc(p.Y + m0 * N, ybytes);
    const __amdgpu_buffer_rsrc_t rr = make_rsrc(p.R ? p.R + m0 * N : p.Y + m0 * N, ybytes);
    const bool has_r = p.R != nullptr;
    const bool vec = (N & 7) == 0;
    const int pr = lane / C::LANES_PER_ROW;             // row within a pass
    const int pc = (lane % C::LANES_PER_ROW) * 8;       // first of 8 columns
    const int64_t col0 = n0 + wn0 + pc;
#pragma unroll
    for (int i = 0; i < C::TM; ++i) {
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
#pragma unroll
            for (int e = 0; e < 16; ++e)
                ep[(8 * (e >> 2) + 4 * hi + (e & 3)) * C::EPI_STRIDE + j * 32 + frag_row] = acc[i][j][e];
        __syncthreads();
#pragma unroll
        for (int v = 0; v < 32 / C::ROWS_PER_PASS; ++v) {
            const int r = v * C::ROWS_PER_PASS + pr;
            const float *src = ep + r * C::EPI_STRIDE + pc;
            float y[8];
#pragma unroll
            for (int t = 0; t < 8; ++t) y[t] = src[t];
            const int64_t row_local = wm0 + i * 32 + r;
            const uint32_t base = static_cast<uint32_t>(row_local * N * 2 + col0 * 2);
            if (vec) {
                const uint32_t off = col0 < N ? base : OOB_OFFSET;
                if (has_r) {
                    const i32x4 rv = __builtin_amdgcn_raw_buffer_load_b128(rr, off, 0, 0);
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        const uint32_t w = static_cast<uint32_t>(rv[t]);
                        y[2 * t] += bf16_to_f32(static_cast<uint16_t>(w & 0xffffu));
                        y[2 * t + 1] += bf16_to_f32(static_cast<uint16_t>(w >> 16));
                    }
                }
                i32x4 out;
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    out[t] = static_cast<int>(static_cast<uint32_t>(f32_to_bf16_rne(y[2 * t])) |
                                              (static_cast<uint32_t>(f32_to_bf16_rne(y[2 * t + 1])) << 16));
                __builtin_amdgcn_raw_buffer_store_b128(out, ry, off, 0, 0);
            } else {
#pragma unroll
                for (int t = 0; t < 8; ++t) {
                    const uint32_t off = (col0 + t) < N ? base + 2 * t : OOB_OFFSET;
                    float yt = y[t];
                    if (has_r) yt += bf16_to_f32(__builtin_amdgcn_raw_buffer_load_b16(rr, off, 0, 0));
                    __builtin_amdgcn_raw_buffer_store_b16(f32_to_bf16_rne(yt), ry, off, 0, 0);
                }
            }
        }
        __syncthreads();
    }
}

template <class C>
hipError_t launch_cfg(const Problem &p, int group_m, hipStream_t s) {
    const int64_t tiles_m = (p.M + C::BM - 1) / C::BM;
    const int64_t tiles_n = (p.N + C::BN - 1) / C::BN;
    const int64_t tiles = tiles_m * tiles_n;
    hipLaunchKernelGGL(tile_kernel<C>, dim3(static_cast<unsigned>(tiles)), dim3(C::THREADS), 0, s, p,
                       tiles_m, tiles_n, group_m);
    return hipGetLastError();
}

using Cfg256x256 = Cfg<256, 256, 1>;
using Cfg256x128 = Cfg<256, 128, 1>;
using Cfg128x128 = Cfg<128, 128, 2>;

}  // namespace

hipError_t launch_tile(int plan, const Problem &p, int num_cus, hipStream_t s) {
    (void)num_cus;
    switch (plan) {
        case PLAN_TILE_256x256: return launch_cfg<Cfg256x256>(p, 8, s);
        case PLAN_TILE_256x128: return launch_cfg<Cfg256x128>(p, 8, s);
        case PLAN_TILE_128x128: return launch_cfg<Cfg128x128>(p, 8, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace kernelarc
