// C ABI, argument validation, device check, split-K workspace and the
// shape-gated plan table.
//
// Plan selection mirrors the structure of the paper's Alg. 3 (per-M cached
// plan, static validated table, heuristic fallback) with hand-written gfx950
// kernels in place of library configurations: exact-shape entries first,
// then rules on (M, N, K); every candidate is checked against the plan's
// limits before use; the choice depends on the shape only, never on data,
// and nothing is tuned during a call.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "../../include/kernelarc.h"
#include "internal.h"

namespace kernelarc {
namespace {

thread_local char g_last_error[512] = "";

int fail(int status, const char *fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return status;
}

constexpr int64_t LIMIT_DIM = (int64_t{1} << 31) - 1;
// Work-items of one grid dimension must stay below 2^32.
constexpr int64_t LIMIT_ITEMS = (int64_t{1} << 32) - 1;
constexpr int64_t PANEL_LIMIT = int64_t{1} << 31;   // bytes addressable by one buffer resource

// Split-K workspace capacity per device (partials in floats, tile counters).
constexpr int64_t WS_PARTIAL_FLOATS = int64_t{1} << 24;
constexpr int64_t WS_COUNTERS = int64_t{1} << 16;
constexpr int64_t CUS = 256;        // MI355X compute units
constexpr int MAX_SPLIT = 16;

enum PlanKind { KIND_GENERIC, KIND_GEMV, KIND_TILE, KIND_STREAM, KIND_BANDS };

struct PlanInfo {
    const char *name;
    PlanKind kind;
    int tile_cfg;   // TileCfg for tile plans, K depth (BK) for stream plans, -1 otherwise
    int split;      // tile and stream plans: 1 = no split-K, 0 = split-K by rule,
                    // -1 (tile) = split only the tiles of a partial last round,
                    // -1 (stream) = split-K by rule, none when the rule says 1
    int stages = 2; // stream plans: per-wave stage buffers
    int rows = 64;  // stream plans: W rows per workgroup
};

// The plans the table and the rules select (plus the generic fallback).
// Order fixes the plan ids; PLAN_GENERIC and PLAN_GEMV are the first two.
const PlanInfo PLANS[] = {
    {"generic_64x64_scalar", KIND_GENERIC, -1, 1},
    {"gemv_valu_w4", KIND_GEMV, -1, 1},
    {"stream_mfma16_r16_k128s2", KIND_STREAM, 128, -1, 2, 16},
    {"stream_mfma16_r32_k64s4", KIND_STREAM, 64, -1, 4, 32},
    {"stream_mfma16_k64_splitk", KIND_STREAM, 64, 0},
    {"tile_64x64_k64s4_w4", KIND_TILE, TC_64x64_K64_S4_W4, 1},
    {"tile_64x64_k128s3_w4_splitk", KIND_TILE, TC_64x64_K128_S3_W4, 0},
    {"tile_64x128_k64s4_w4", KIND_TILE, TC_64x128_K64_S4_W4, 1},
    {"tile_64x128_k64s4_w4_splitk", KIND_TILE, TC_64x128_K64_S4_W4, 0},
    {"tile_128x128_k64_w4", KIND_TILE, TC_128x128_K64_S2_W4, 1},
    {"tile_128x128_k64_w4_splitk", KIND_TILE, TC_128x128_K64_S2_W4, 0},
    {"tile_128x128_k64s3_w4_splitk", KIND_TILE, TC_128x128_K64_S3_W4, 0},
    {"tile_128x128_k64s4_w4_lag", KIND_TILE, TC_128x128_K64_S4_W4_L, 1},
    {"tile_256x128_k64s3_w8_splitk", KIND_TILE, TC_256x128_K64_S3_W8, 0},
    {"tile_256x128_k64s3_w8_lag", KIND_TILE, TC_256x128_K64_S3_W8_L, 1},
    {"tile_256x128_k64s3_w8_lag_splitk", KIND_TILE, TC_256x128_K64_S3_W8_L, 0},
    {"tile_256x256_k64_w8", KIND_TILE, TC_256x256_K64_S2_W8, 1},
    {"tile_256x256_k64_w8_tailsplit", KIND_TILE, TC_256x256_K64_S2_W8, -1},
    {"tile_256x256_k64_w4_m16a", KIND_TILE, TC_256x256_K64_S2_W4_M16A, 1},
    // Two column bands: the widest one whose 256x256 tiles fill whole rounds
    // of the CUs on the 4-wave AGPR tile, the other columns on the 128x128
    // 4-stage lagged tile (two launches on the stream).
    {"tile_256x256_k64_w4_m16a_bands", KIND_BANDS, -1, 1},
};
constexpr int NUM_PLANS = static_cast<int>(sizeof(PLANS) / sizeof(PLANS[0]));

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

int64_t tile_count(const TileShape &ts, int64_t M, int64_t N) { return cdiv(M, ts.bm) * cdiv(N, ts.bn); }

// Split-K rule of the "_splitk" tile plans: enough K slices that the tiles
// fill one round of workgroup slots on the 256 CUs, each slice at least 8
// BK steps deep; at least 2 so the plan always exercises the reduction.
// "_tailsplit" plans: the tiles that fill whole rounds run whole and the
// rest are split so that they fill the last round (each XCD must get equal
// shares of both kinds of work, else no split).
struct TileSplit {
    int split;
    int64_t full_tiles;   // > 0: tail split
};

TileSplit tile_split_plan(int plan, int64_t M, int64_t N, int64_t K) {
    const PlanInfo &pi = PLANS[plan];
    if (pi.split >= 1) return {pi.split, 0};
    const TileShape ts = tile_shape(pi.tile_cfg);
    const int64_t tiles = tile_count(ts, M, N);
    const int64_t slots = CUS * ts.workgroups_per_cu;
    if (pi.split < 0) {
        const int64_t full = (tiles / slots) * slots, rest = tiles - full;
        if (full == 0 || rest == 0) return {1, 0};
        int64_t split = slots / rest;
        const int64_t by_depth = K / (4 * ts.bk);
        if (split > by_depth) split = by_depth;
        if (split > MAX_SPLIT) split = MAX_SPLIT;
        if (split < 2 || full % 8 != 0 || (rest * split) % 8 != 0) return {1, 0};
        return {static_cast<int>(split), full};
    }
    int64_t split = tiles > 0 ? slots / tiles : 1;
    const int64_t by_depth = K / (8 * ts.bk);
    if (split > by_depth) split = by_depth;
    if (split > MAX_SPLIT) split = MAX_SPLIT;
    if (split < 2) split = 2;
    return {static_cast<int>(split), 0};
}

int tile_split_of(int plan, int64_t M, int64_t N, int64_t K) { return tile_split_plan(plan, M, N, K).split; }

// Split-K of the stream plans: the kernel's rule, at least 2 for the
// "_splitk" plans so they always exercise the reduction.
int stream_split_of(int plan, int64_t M, int64_t N, int64_t K) {
    const PlanInfo &pi = PLANS[plan];
    if (pi.split >= 1) return pi.split;
    const int rule = stream_split_for(M, N, K, pi.tile_cfg, pi.rows);
    if (pi.split < 0) return rule;
    return rule < 2 ? 2 : rule;
}

// Row strides of a call and whether it is the general form (strides other
// than dense, alpha or beta other than 1, or a bias).  Every kernel computes
// every form.
struct Layout {
    int64_t ldx, ldw, ldr, ldy;
    bool general;
};
Layout dense_layout(int64_t N, int64_t K) { return Layout{K, K, N, N, false}; }

int plan_index(const char *name);

// Column bands of the banded plan: columns [0, N1) on BAND_MAIN, whose
// 256x256 tiles then fill whole rounds of the CUs (the tile rows times the
// band's tile columns is a multiple of CUS), the rest on BAND_REST.  N1 is
// a multiple of 256 (0 or N when no such split exists).
const char *const BAND_MAIN = "tile_256x256_k64_w4_m16a";
const char *const BAND_REST = "tile_128x128_k64s4_w4_lag";
int64_t gcd64(int64_t a, int64_t b) { return b == 0 ? a : gcd64(b, a % b); }
int64_t band_split(int64_t M, int64_t N) {
    const int64_t tm = cdiv(M, 256), tn = cdiv(N, 256);
    if (tm == 0 || tn == 0) return 0;
    const int64_t q = CUS / gcd64(tm, CUS);        // band tile columns come in multiples of q
    const int64_t tn1 = (tn / q) * q;
    return tn1 >= tn ? N : tn1 * 256;
}

bool supports(int plan, int64_t M, int64_t N, int64_t K, bool residual, const Layout &lay) {
    (void)residual;
    if (M < 0 || N < 0 || K < 0 || M > LIMIT_DIM || N > LIMIT_DIM || K > LIMIT_DIM) return false;
    if (plan < 0 || plan >= NUM_PLANS) return false;
    const PlanInfo &pi = PLANS[plan];
    switch (pi.kind) {
        case KIND_GENERIC:
            return cdiv(M, 64) * cdiv(N, 64) * 256 <= LIMIT_ITEMS;
        case KIND_GEMV:
            return gemv_fits(M, N, K, lay.ldw) && cdiv(N, 4) * 256 <= LIMIT_ITEMS &&
                   strided_bytes(M, N, lay.ldy) < PANEL_LIMIT && strided_bytes(M, N, lay.ldr) < PANEL_LIMIT;
        case KIND_STREAM: {
            if (M < 1 || M > 64 || K % 8 != 0) return false;
            if (!stream_config_exists(pi.tile_cfg, pi.stages, pi.rows)) return false;
            // The kernel addresses whole 16-row token blocks of X, R and Y
            // (rows past M fall outside the buffer resources): their 32-bit
            // offsets must stay below the panel limit.
            const int64_t mb = 16 * cdiv(M, 16);
            if (strided_bytes(pi.rows, K, lay.ldw) >= PANEL_LIMIT || strided_bytes(mb, K, lay.ldx) >= PANEL_LIMIT ||
                strided_bytes(mb, N, lay.ldy) >= PANEL_LIMIT || strided_bytes(mb, N, lay.ldr) >= PANEL_LIMIT)
                return false;
            const int split = stream_split_of(plan, M, N, K);
            if (cdiv(N, pi.rows) * split * 256 > LIMIT_ITEMS) return false;
            if (split > 1 && (stream_workspace_floats(M, N, split, pi.rows) > WS_PARTIAL_FLOATS ||
                              stream_counter_count(N, pi.rows) > WS_COUNTERS))
                return false;
            return true;
        }
        case KIND_BANDS: {
            const int64_t N1 = band_split(M, N);
            const Layout band{lay.ldx, lay.ldw, lay.ldr, lay.ldy, true};
            return (N1 == 0 || supports(plan_index(BAND_MAIN), M, N1, K, residual, band)) &&
                   (N1 == N || supports(plan_index(BAND_REST), M, N - N1, K, residual, band));
        }
        case KIND_TILE: {
            const TileShape ts = tile_shape(pi.tile_cfg);
            if (K % 8 != 0) return false;
            if (strided_bytes(ts.bm, K, lay.ldx) >= PANEL_LIMIT || strided_bytes(ts.bn, K, lay.ldw) >= PANEL_LIMIT)
                return false;
            // epilogue panels of R and Y
            if (strided_bytes(ts.bm, N, lay.ldy) >= PANEL_LIMIT || strided_bytes(ts.bm, N, lay.ldr) >= PANEL_LIMIT)
                return false;
            const int64_t tiles = tile_count(ts, M, N);
            const TileSplit sp = tile_split_plan(plan, M, N, K);
            const int64_t split_tiles = tiles - sp.full_tiles;
            if ((sp.full_tiles + split_tiles * sp.split) * 1024 > LIMIT_ITEMS) return false;
            if (sp.split > 1 &&
                (split_tiles * sp.split * ts.bm * ts.bn > WS_PARTIAL_FLOATS || split_tiles > WS_COUNTERS))
                return false;
            return true;
        }
    }
    return false;
}

int plan_index(const char *name) {
    for (int i = 0; i < NUM_PLANS; ++i)
        if (std::strcmp(PLANS[i].name, name) == 0) return i;
    return -1;
}


// Exact-shape entries (M, N, K, residual) -> plan name; from measurements on
// MI355X (the benchmark's cold-cache protocol).  The sentinel has M = -1.
struct TableEntry {
    int64_t M, N, K;
    int residual;
    const char *plan;
};
const TableEntry TABLE[] = {
    // attention-output-projection sweep: M x (N = K = hidden), residual
    {1, 2048, 2048, 1, "gemv_valu_w4"},
    {1, 4096, 4096, 1, "gemv_valu_w4"},
    {1, 5120, 5120, 1, "gemv_valu_w4"},
    {1, 8192, 8192, 1, "gemv_valu_w4"},
    {16, 4096, 4096, 1, "stream_mfma16_r16_k128s2"},
    {64, 2048, 2048, 1, "stream_mfma16_r16_k128s2"},
    {64, 4096, 4096, 1, "tile_64x64_k128s3_w4_splitk"},
    {64, 5120, 5120, 1, "tile_64x64_k128s3_w4_splitk"},
    {64, 8192, 8192, 1, "tile_64x64_k128s3_w4_splitk"},
    {512, 2048, 2048, 1, "tile_64x64_k64s4_w4"},
    {512, 4096, 4096, 1, "tile_128x128_k64s3_w4_splitk"},
    {512, 5120, 5120, 1, "tile_256x128_k64s3_w8_lag_splitk"},
    {512, 8192, 8192, 1, "tile_256x128_k64s3_w8_lag_splitk"},
    {4096, 2048, 2048, 1, "tile_256x128_k64s3_w8_lag"},
    {4096, 4096, 4096, 1, "tile_256x256_k64_w4_m16a"},
    {4096, 5120, 5120, 1, "tile_256x256_k64_w4_m16a_bands"},
    {4096, 8192, 8192, 1, "tile_256x256_k64_w4_m16a"},
    // plain BF16 GEMM
    {8192, 8192, 8192, 0, "tile_256x256_k64_w4_m16a"},
    {-1, 0, 0, 0, ""},   // sentinel
};

// The 256x256 plan for t256 tiles.  Whole rounds, or fewer tiles than CUs:
// the 4-wave AGPR tile.  A partial last round takes most of a full round's
// time whatever its fill (each tile still runs its whole K loop), while one
// round of 128x128 tiles takes about 0.4 of it: two column bands when the
// columns past the widest whole-round band fit one round of 128x128 tiles
// (bands_ok: plain and general forms); else the 8-wave tail split after a
// single full round when the last one holds at most a quarter of the CUs
// (with more full rounds the 8-wave tile's slower rounds cost more than the
// split saves); else the 4-wave tile over every tile.
const char *wide_tile_plan(int64_t M, int64_t N, int64_t t256, bool bands_ok) {
    if (t256 % CUS == 0 || t256 < CUS) return "tile_256x256_k64_w4_m16a";
    if (bands_ok) {
        const int64_t N1 = band_split(M, N);
        if (N1 > 0 && N1 < N && tile_count(tile_shape(TC_128x128_K64_S4_W4_L), M, N - N1) <= CUS)
            return "tile_256x256_k64_w4_m16a_bands";
    }
    if (t256 < 2 * CUS && 4 * (t256 % CUS) <= CUS) return "tile_256x256_k64_w8_tailsplit";
    return "tile_256x256_k64_w4_m16a";
}

// Rule-based choice when no table entry matches (from the same
// measurements): the VALU GEMV up to 4 rows; the streaming kernel up to 32
// rows, with 16-row blocks of W when they fit one round on the CUs (N up to
// 4096; no cross-workgroup split there) and 64-row blocks with split-K
// beyond; up to 64 rows, the 16-row streaming kernel while N <= 2048 and
// K <= 4096; up to 1024 rows: the 256x256 tile when its tiles reach 2/3
// of the CUs (the 4-wave form when they fit one round or fill whole ones),
// the 256x128 3-stage lagged tile above 512 rows when its tiles fill them,
// else 64x64 tiles (3 stages of K depth 128, split-K) while they fill at
// most half the CUs, 64x64 tiles (4 stages of depth 64, two per CU) while
// they fit one round, else 128x128 tiles
// with 3 stages and split-K when they would keep at most half the CUs busy,
// 256x128 8-wave tiles (3 stages, lagged refill) with split-K when 128x128
// tiles would leave some CUs idle, else 128x128 tiles with 4 stages and the
// lagged refill; above that the 256x256 tile when it fills the 256 CUs
// (4 waves of 128x128 on 16x16x32 MFMAs with AGPR accumulators when the
// tiles fill whole rounds; else 8 waves on 32x32 MFMAs with the tail split:
// the tiles of a partial last round are split in K), the 256x128 8-wave
// tile (3 stages, lagged refill) when that fills them, else the 128x128
// tile.
int select(int64_t M, int64_t N, int64_t K, bool residual, const Layout &lay) {
    if (M < 0 || N < 0 || K < 0) return -1;
    for (const TableEntry &e : TABLE) {
        if (e.M < 0 || e.M != M || e.N != N || e.K != K || (e.residual != 0) != residual) continue;
        const int plan = plan_index(e.plan);
        if (plan >= 0 && supports(plan, M, N, K, residual, lay)) return plan;
    }
    if (K % 8 != 0) return PLAN_GENERIC;
    auto pick = [&](const char *name) {
        const int plan = plan_index(name);
        return (plan >= 0 && supports(plan, M, N, K, residual, lay)) ? plan : -1;
    };
    int plan = -1;
    if (M >= 1 && M <= 4) plan = pick("gemv_valu_w4");
    if (plan >= 0) return plan;
    if (M >= 1 && M <= 64 && cdiv(N, 16) <= CUS && (M <= 32 || (N <= 2048 && K <= 4096)))
        plan = pick("stream_mfma16_r16_k128s2");
    if (plan >= 0) return plan;
    if (M >= 1 && M <= 32) {
        plan = pick("stream_mfma16_k64_splitk");
        if (plan < 0) plan = pick("tile_64x64_k128s3_w4_splitk");
    } else if (M <= 1024) {
        const int64_t tiles64 = tile_count(tile_shape(TC_64x64_K64_S4_W4), M, N);
        const int64_t tiles128 = tile_count(tile_shape(TC_128x128_K64_S4_W4_L), M, N);
        const int64_t t256 = tile_count(tile_shape(TC_256x256_K64_S2_W8), M, N);
        const int64_t t256x128 = tile_count(tile_shape(TC_256x128_K64_S3_W8_L), M, N);
        if (3 * t256 >= 2 * CUS) {   // wide outputs: the 256x256 tiles reach 2/3 of the CUs
            plan = pick(wide_tile_plan(M, N, t256, true));
            if (plan < 0) plan = pick("tile_256x256_k64_w8_tailsplit");
        } else if (t256x128 >= CUS && M > 512)
            plan = pick("tile_256x128_k64s3_w8_lag");
        else if (2 * tiles64 <= CUS) plan = pick("tile_64x64_k128s3_w4_splitk");
        else if (tiles64 <= 2 * CUS) plan = pick("tile_64x64_k64s4_w4");
        else if (2 * tiles128 <= CUS) plan = pick("tile_128x128_k64s3_w4_splitk");
        else if (tiles128 < CUS) plan = pick("tile_256x128_k64s3_w8_lag_splitk");
        else plan = pick("tile_128x128_k64s4_w4_lag");
        if (plan < 0) plan = pick("tile_128x128_k64_w4_splitk");
    } else {
        const int64_t t256 = tile_count(tile_shape(TC_256x256_K64_S2_W8), M, N);
        if (t256 >= CUS) {
            plan = pick(wide_tile_plan(M, N, t256, true));
            if (plan < 0) plan = pick("tile_256x256_k64_w8_tailsplit");
        }
        else if (tile_count(tile_shape(TC_256x128_K64_S3_W8_L), M, N) >= CUS) plan = pick("tile_256x128_k64s3_w8_lag");
        if (plan < 0) plan = pick("tile_128x128_k64_w4");
    }
    if (plan < 0) plan = pick("tile_128x128_k64_w4");
    return plan >= 0 ? plan : PLAN_GENERIC;
}

// SwiGLU (gate and up projections with the SiLU-multiply): the tile plans
// whose configuration pairs gate and up blocks, and the generic kernel.  A
// tile computes BM x BN/2 outputs from a BM x BN block of products, so tile
// counts and split-K rules are those of the doubled width 2N.
bool supports_glu(int plan, int64_t M, int64_t N, int64_t K) {
    if (M < 0 || N < 0 || K < 0 || M > LIMIT_DIM || N > LIMIT_DIM / 2 || K > LIMIT_DIM) return false;
    if (plan < 0 || plan >= NUM_PLANS) return false;
    const PlanInfo &pi = PLANS[plan];
    if (pi.kind == KIND_GENERIC) return cdiv(M, 64) * cdiv(N, 64) * 256 <= LIMIT_ITEMS;
    if (pi.kind != KIND_TILE || !tile_glu_ok(pi.tile_cfg) || K % 8 != 0) return false;
    const TileShape ts = tile_shape(pi.tile_cfg);
    if (ts.bm * K * 2 >= PANEL_LIMIT || (ts.bn / 2) * K * 2 >= PANEL_LIMIT || ts.bm * N * 2 >= PANEL_LIMIT)
        return false;
    const int64_t tiles = tile_count(ts, M, 2 * N);
    const TileSplit sp = tile_split_plan(plan, M, 2 * N, K);
    const int64_t split_tiles = tiles - sp.full_tiles;
    if ((sp.full_tiles + split_tiles * sp.split) * 1024 > LIMIT_ITEMS) return false;
    if (sp.split > 1 && (split_tiles * sp.split * ts.bm * ts.bn > WS_PARTIAL_FLOATS || split_tiles > WS_COUNTERS))
        return false;
    return true;
}

// SwiGLU plan rule (from measurements on MI355X over M = 1 .. 4096 at
// Llama-class hidden/intermediate sizes; tile counts at width 2N): up to 64
// rows the 64x128 4-stage tile, with split-K when its tiles fill at most
// half the CUs and K is deep enough; up to 128 rows, or while 256x128 tiles
// would fill less than half the CUs, 128x128 tiles (3 stages and split-K
// when they fill at most half the CUs, else 4 stages with the lagged
// refill); then the 256x256 8-wave tile once its tiles cover at least 80%
// of the CUs (tail split past whole rounds), else the 256x128 8-wave tile
// with 3 stages and the lagged refill.
int select_glu(int64_t M, int64_t N, int64_t K) {
    if (M < 0 || N < 0 || K < 0) return -1;
    if (K % 8 != 0) return PLAN_GENERIC;
    auto pick = [&](const char *name) {
        const int plan = plan_index(name);
        return (plan >= 0 && supports_glu(plan, M, N, K)) ? plan : -1;
    };
    const int64_t N2 = 2 * N;
    const int64_t t64 = tile_count(tile_shape(TC_64x128_K64_S4_W4), M, N2);
    const int64_t t128 = tile_count(tile_shape(TC_128x128_K64_S4_W4_L), M, N2);
    const int64_t t256x128 = tile_count(tile_shape(TC_256x128_K64_S3_W8_L), M, N2);
    const int64_t t256 = tile_count(tile_shape(TC_256x256_K64_S2_W8), M, N2);
    int plan = -1;
    if (M <= 64) {
        plan = (2 * t64 <= CUS && K >= 2048) ? pick("tile_64x128_k64s4_w4_splitk") : pick("tile_64x128_k64s4_w4");
    } else if (M <= 128 || 2 * t256x128 < CUS) {
        plan = 2 * t128 <= CUS ? pick("tile_128x128_k64s3_w4_splitk") : pick("tile_128x128_k64s4_w4_lag");
    } else if (5 * t256 >= 4 * CUS) {
        plan = pick(wide_tile_plan(M, N2, t256, false));
        if (plan < 0) plan = pick("tile_256x256_k64_w8_tailsplit");
    } else {
        plan = pick("tile_256x128_k64s3_w8_lag");
    }
    if (plan < 0) plan = pick("tile_128x128_k64_w4");
    return plan >= 0 ? plan : PLAN_GENERIC;
}

// INT8 operands (W8A8 with dequantisation scales): the tile plans when K is
// a multiple of 16 (16-byte chunks of int8), and the generic plan.  A stage
// of an INT8 tile holds twice the K elements of a bf16 one, so panel sizes,
// tile counts and split-K rules are those of the bf16 problem at K/2.
// |A| <= K * 2^14 keeps the exact int32 sums in range for K <= 2^16.
constexpr int64_t I8_MAX_K = int64_t{1} << 16;

// FP8 (E4M3) operands share the INT8 path's layout, scales, plans and rules;
// their tile configurations also need sub-steps of 64 K bytes
// (tile_f8_ok), and K has no integer-range limit.
bool supports_i8(int plan, int64_t M, int64_t N, int64_t K, bool glu, bool f8 = false) {
    if (M < 0 || N < 0 || K < 0 || M > LIMIT_DIM || N > (glu ? LIMIT_DIM / 2 : LIMIT_DIM) ||
        K > (f8 ? LIMIT_DIM : I8_MAX_K))
        return false;
    if (plan < 0 || plan >= NUM_PLANS) return false;
    const PlanInfo &pi = PLANS[plan];
    if (pi.kind == KIND_GENERIC) return cdiv(M, 64) * cdiv(N, 64) * 256 <= LIMIT_ITEMS;
    // INT8 GEMMs also stream through the 16- and 32-row configurations
    // (the same bytes per stage as bf16 at K/2).
    if (pi.kind == KIND_STREAM)
        return !glu && !f8 && pi.rows < 64 && K % 16 == 0 && supports(plan, M, N, K / 2, true, dense_layout(N, K / 2));
    // (the 16x16 MFMA tiles take plain int8 operands: not FP8, not SwiGLU)
    if (pi.kind != KIND_TILE || K % 16 != 0 || ((f8 || glu) && tile_is_m16(pi.tile_cfg)) ||
        (f8 && !tile_f8_ok(pi.tile_cfg)))
        return false;
    return glu ? supports_glu(plan, M, N, K / 2) : supports(plan, M, N, K / 2, true, dense_layout(N, K / 2));
}

// INT8 plan rule (measured on MI355X): the bf16 rules at K/2 (the same
// bytes per stage), with these changes.  Plain INT8 GEMMs up to 64 rows
// stream: 16-row blocks while they fit one round on the CUs (N <= 4096),
// else 32-row blocks while those do (N <= 8192); past that (and for FP8
// operands) 64x64 tiles, 3 stages of depth 256 with split-K while the tiles
// fill at most half the CUs, else 4 stages of depth 128.  The 256x256 tile runs without the tail split: an
// INT8 tile covers its K range in half the steps, so the split's partial
// round trip costs more than the idle CUs it saves (6% at M = 2048 SwiGLU).
int select_i8(int64_t M, int64_t N, int64_t K, bool glu, bool f8 = false) {
    if (M < 0 || N < 0 || K < 0) return -1;
    if (K % 16 != 0 || K > (f8 ? LIMIT_DIM : I8_MAX_K)) return PLAN_GENERIC;
    auto pick = [&](const char *name) {
        const int p = plan_index(name);
        return (p >= 0 && supports_i8(p, M, N, K, glu, f8)) ? p : -1;
    };
    int plan = -1;
    if (!glu && !f8 && M >= 1 && M <= 64) {
        if (cdiv(N, 16) <= CUS) plan = pick("stream_mfma16_r16_k128s2");
        else if (cdiv(N, 32) <= CUS) plan = pick("stream_mfma16_r32_k64s4");
        if (plan >= 0) return plan;
    }
    if (!glu && M <= 64) {
        const int64_t t64 = tile_count(tile_shape(TC_64x64_K64_S4_W4), M, N);
        plan = 2 * t64 <= CUS ? pick("tile_64x64_k128s3_w4_splitk") : pick("tile_64x64_k64s4_w4");
        if (plan >= 0) return plan;
    }
    plan = glu ? select_glu(M, N, K / 2) : select(M, N, K / 2, true, dense_layout(N, K / 2));
    // The 4-wave AGPR tile keeps plain INT8 from K = 8192 up (its 16x16
    // layout has no FP8 or SwiGLU form), also where the bf16 rule splits it
    // into column bands: a long K loop pays for its costlier prologue (at
    // 8192^3 415 us against 457 us for the 8-wave tile; at M = 4096,
    // N = 14336, K = 4096 it is 2% behind). Otherwise the 256x256 8-wave
    // tile without the tail split, and already
    // when its tiles reach 4/5 of the CUs (an INT8 tile covers its K range
    // in half the steps: at M = 1024, N = 13824, K = 5120, 90 us against
    // 128 us for 128x128).
    const int m16a = plan_index("tile_256x256_k64_w4_m16a");
    if (plan == plan_index("tile_256x256_k64_w4_m16a_bands")) plan = m16a;
    const bool keep_m16a = plan == m16a && !glu && !f8 && K >= 8192;
    if (!keep_m16a && (plan == plan_index("tile_256x256_k64_w8_tailsplit") || plan == m16a ||
                       (!glu && 5 * tile_count(tile_shape(TC_256x256_K64_S2_W8), M, N) >= 4 * CUS)))
        plan = plan_index("tile_256x256_k64_w8");
    if (plan >= 0 && plan != PLAN_GENERIC && supports_i8(plan, M, N, K, glu, f8)) return plan;
    for (const char *name : {"tile_64x64_k128s3_w4_splitk", "tile_64x128_k64s4_w4", "tile_128x128_k64_w4"}) {
        const int p = pick(name);
        if (p >= 0) return p;
    }
    return PLAN_GENERIC;
}

// Grouped (per-expert) forms over an expert-major padded layout: the tile
// plans without split-K (SwiGLU: those that pair gate and up blocks) and the
// generic plan.  The valid rows per group are on the device, so a launch
// covers every group's M_pad rows and the tiles past the valid rows exit at
// once.
bool supports_grouped(int plan, int64_t G, int64_t Mpad, int64_t N, int64_t K, bool glu) {
    if (G < 0 || Mpad < 0 || N < 0 || K < 0 || Mpad > LIMIT_DIM || N > (glu ? LIMIT_DIM / 2 : LIMIT_DIM) ||
        K > LIMIT_DIM || (Mpad > 0 && G > LIMIT_DIM / Mpad))
        return false;
    if (plan < 0 || plan >= NUM_PLANS) return false;
    const PlanInfo &pi = PLANS[plan];
    if (pi.kind == KIND_GENERIC) return G * cdiv(Mpad, 64) * cdiv(N, 64) * 256 <= LIMIT_ITEMS;
    if (pi.kind != KIND_TILE || pi.split != 1 || K % 8 != 0) return false;
    if (glu && !tile_glu_ok(pi.tile_cfg)) return false;
    const TileShape ts = tile_shape(pi.tile_cfg);
    const int64_t bn = glu ? ts.bn / 2 : ts.bn;
    if (ts.bm * K * 2 >= PANEL_LIMIT || bn * K * 2 >= PANEL_LIMIT || ts.bm * N * 2 >= PANEL_LIMIT) return false;
    return G * cdiv(Mpad, ts.bm) * cdiv(N, bn) * 1024 <= LIMIT_ITEMS;
}

// Grouped plan rule (measured on MI355X at the mixture-of-experts sizes of
// the paper's case study, 256 experts, top-8, hidden 4096, intermediate
// 2048): the expert weights dominate the traffic, so a group whose padded
// rows exceed 128 takes a 256x256 tile (one m-tile per expert, its weights
// read once): the 4-wave AGPR form for the gate/up projections with SwiGLU
// (2.4 % faster at 6144 tokens), the 8-wave form for plain projections (the
// 4-wave one is 3 % slower there); smaller groups take the 128x128 tile at
// two workgroups per CU.
int select_grouped(int64_t G, int64_t Mpad, int64_t N, int64_t K, bool glu) {
    if (G < 0 || Mpad < 0 || N < 0 || K < 0) return -1;
    if (K % 8 != 0) return PLAN_GENERIC;
    const char *first = Mpad <= 128 ? "tile_128x128_k64_w4"
                        : glu       ? "tile_256x256_k64_w4_m16a"
                                    : "tile_256x256_k64_w8";
    for (const char *name : {first, "tile_256x256_k64_w8", "tile_128x128_k64_w4"}) {
        const int p = plan_index(name);
        if (p >= 0 && supports_grouped(p, G, Mpad, N, K, glu)) return p;
    }
    return PLAN_GENERIC;
}

// ---------------------------------------------------------- plan cache ----
// Alg. 3 keeps the chosen plan per shape so that the table and the rules are
// consulted once.  The key is everything a choice depends on (the operation,
// the sizes, the row strides and whether the call is the general form),
// never data.  Each thread holds its own direct-mapped table, so a lookup
// takes no lock; a colliding shape replaces the entry.
enum PlanOp { OP_LINEAR = 0, OP_GLU, OP_I8, OP_I8_GLU, OP_F8, OP_F8_GLU, OP_GROUPED, OP_GROUPED_GLU };

struct PlanKey {
    int op;
    int flags;   // OP_LINEAR: bit 0 residual, bit 1 general form
    int64_t M, N, K, a, b, c, d;   // OP_LINEAR: row strides; OP_GROUPED*: a = G
    bool operator==(const PlanKey &o) const {
        return op == o.op && flags == o.flags && M == o.M && N == o.N && K == o.K && a == o.a && b == o.b &&
               c == o.c && d == o.d;
    }
};

constexpr int PLAN_CACHE_SLOTS = 64;
struct PlanCacheEntry {
    PlanKey key;
    int plan;
    bool valid;
};
thread_local PlanCacheEntry g_plan_cache[PLAN_CACHE_SLOTS];

template <class F>
int cached_plan(const PlanKey &k, F &&choose) {
    uint64_t h = static_cast<uint64_t>(k.op) * 0x9E3779B97F4A7C15ull ^ static_cast<uint64_t>(k.flags);
    for (int64_t v : {k.M, k.N, k.K, k.a, k.b, k.c, k.d}) h = (h ^ static_cast<uint64_t>(v)) * 0x100000001B3ull;
    PlanCacheEntry &e = g_plan_cache[(h ^ (h >> 29)) % PLAN_CACHE_SLOTS];
    if (e.valid && e.key == k) return e.plan;
    const int plan = choose();
    e = PlanCacheEntry{k, plan, true};
    return plan;
}

// ------------------------------------------------------------ devices ----
constexpr int MAX_DEVICES = 64;

struct DeviceState {
    bool probed = false;
    bool gfx950 = false;
    int num_cus = 0;
    char arch[64] = "";
    float *ws_partials = nullptr;
    unsigned *ws_counters = nullptr;
    float *scratch = nullptr;        // this device's copy of `scratch` (hipGetSymbolAddress)
    bool scratch_cleared = false;    // its counters were cleared by an uncaptured kernel
};

std::mutex g_mutex;
DeviceState g_devices[MAX_DEVICES];

int current_device(int *dev, int *num_cus) {
    int d = -1;
    hipError_t e = hipGetDevice(&d);
    if (e != hipSuccess || d < 0)
        return fail(KERNELARC_ERR_UNSUPPORTED, "no HIP device: %s", hipGetErrorString(e));
    if (d >= MAX_DEVICES) return fail(KERNELARC_ERR_UNSUPPORTED, "device index %d out of range", d);
    std::lock_guard<std::mutex> lock(g_mutex);
    DeviceState &st = g_devices[d];
    if (!st.probed) {
        hipDeviceProp_t prop;
        e = hipGetDeviceProperties(&prop, d);
        if (e != hipSuccess)
            return fail(KERNELARC_ERR_UNSUPPORTED, "hipGetDeviceProperties: %s", hipGetErrorString(e));
        snprintf(st.arch, sizeof st.arch, "%s", prop.gcnArchName);
        st.gfx950 = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
        st.num_cus = prop.multiProcessorCount;
        st.probed = true;
    }
    if (!st.gfx950)
        return fail(KERNELARC_ERR_UNSUPPORTED, "device %d is %s; this library is built for gfx950", d,
                    st.arch);
    *dev = d;
    *num_cus = st.num_cus;
    return KERNELARC_OK;
}

// Sets n counters to zero on the caller's stream: a kernel rather than
// hipMemsetAsync, so the clearing is an ordinary kernel node if a caller
// captures the stream.
__global__ void zero_counters_kernel(unsigned *c, int64_t n) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < n) c[i] = 0u;
}

hipError_t zero_counters(unsigned *c, int64_t n, hipStream_t stream) {
    hipLaunchKernelGGL(zero_counters_kernel, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, stream, c,
                       n);
    return hipGetLastError();
}

// The split-K workspace of device `dev`, allocated on first use.  Its
// counters are cleared by a kernel on `stream`, ahead of the call's own
// kernel on the same stream; nothing waits for the stream.  The kernels
// leave every counter at zero, so later calls need no clearing.  A first
// use under stream capture cannot allocate (and the clearing would only run
// when the graph is replayed), so it is refused.
int workspace(int dev, hipStream_t stream, Workspace *out) {
    std::lock_guard<std::mutex> lock(g_mutex);
    DeviceState &st = g_devices[dev];
    if (!st.ws_partials) {
        hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
        hipError_t e = hipStreamIsCapturing(stream, &cap);
        if (e != hipSuccess)
            return fail(KERNELARC_ERR_LAUNCH, "hipStreamIsCapturing: %s", hipGetErrorString(e));
        if (cap != hipStreamCaptureStatusNone)
            return fail(KERNELARC_ERR_UNSUPPORTED,
                        "the split-K workspace of device %d is allocated by the first call that needs it, which "
                        "cannot run under stream capture: make one call of this plan before capturing", dev);
        void *parts = nullptr;
        void *counters = nullptr;
        e = hipMalloc(&parts, WS_PARTIAL_FLOATS * sizeof(float));
        if (e == hipSuccess) e = hipMalloc(&counters, WS_COUNTERS * sizeof(unsigned));
        if (e == hipSuccess) e = zero_counters(static_cast<unsigned *>(counters), WS_COUNTERS, stream);
        if (e != hipSuccess) {
            if (parts) (void)hipFree(parts);
            if (counters) (void)hipFree(counters);
            return fail(KERNELARC_ERR_LAUNCH, "split-K workspace set-up: %s", hipGetErrorString(e));
        }
        st.ws_partials = static_cast<float *>(parts);
        st.ws_counters = static_cast<unsigned *>(counters);
    }
    out->partials = st.ws_partials;
    out->partial_floats = WS_PARTIAL_FLOATS;
    out->counters = st.ws_counters;
    out->counter_count = WS_COUNTERS;
    return KERNELARC_OK;
}

// Split-K scratch of kernelarc_gemm_bf16_residual_noalloc, for callers that
// cannot allocate: the same capacity as the workspace above (fp32 partials,
// then the arrival counters as 32-bit words), reserved in the code object,
// so each device holds its own copy from the moment the library's code is
// loaded onto it until the process ends.  Host code must not pass the
// array's name to a kernel (in host code it is only a stand-in for the
// symbol); it uses the device address that hipGetSymbolAddress returns.
constexpr int64_t SCRATCH_FLOATS = WS_PARTIAL_FLOATS + WS_COUNTERS;
static __device__ __align__(256) float scratch[SCRATCH_FLOATS];

// The scratch of device `dev` (the current device) as a workspace.  The first
// call on a device looks up its address and clears the counters with a
// kernel on `stream` (no allocation, no memset node, no wait); the kernels
// leave every counter at zero, so later calls need no clearing.  If that
// first clearing is captured into a graph, it runs only when the graph is
// replayed (before the captured GEMM, which is all that graph needs), so the
// next uncaptured call clears again.
int scratch_workspace(int dev, hipStream_t stream, Workspace *out) {
    std::lock_guard<std::mutex> lock(g_mutex);
    DeviceState &st = g_devices[dev];
    if (!st.scratch) {
        void *ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr)
            return fail(KERNELARC_ERR_LAUNCH, "hipGetSymbolAddress(scratch) on device %d: %s", dev,
                        hipGetErrorString(e));
        st.scratch = static_cast<float *>(ptr);
    }
    unsigned *const counters = reinterpret_cast<unsigned *>(st.scratch + WS_PARTIAL_FLOATS);
    if (!st.scratch_cleared) {
        hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
        hipError_t e = hipStreamIsCapturing(stream, &cap);
        if (e == hipSuccess) e = zero_counters(counters, WS_COUNTERS, stream);
        if (e != hipSuccess) return fail(KERNELARC_ERR_LAUNCH, "clearing the scratch counters: %s", hipGetErrorString(e));
        if (cap == hipStreamCaptureStatusNone) st.scratch_cleared = true;
    }
    out->partials = st.scratch;
    out->partial_floats = WS_PARTIAL_FLOATS;
    out->counters = counters;
    out->counter_count = WS_COUNTERS;
    return KERNELARC_OK;
}

bool overlaps(const void *a, int64_t abytes, const void *b, int64_t bbytes) {
    if (!a || !b || abytes == 0 || bbytes == 0) return false;
    const auto pa = reinterpret_cast<uintptr_t>(a);
    const auto pb = reinterpret_cast<uintptr_t>(b);
    return pa < pb + static_cast<uintptr_t>(bbytes) && pb < pa + static_cast<uintptr_t>(abytes);
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// One call as the entry points pass it (leading dimensions in elements).
struct Request {
    int64_t M, N, K;
    float alpha;
    const void *X;
    int64_t ldx;
    const void *W;
    int64_t ldw;
    float beta;
    const void *R;    // residual / C; null: none
    int64_t ldr;
    const void *bias; // [N] or null
    void *Y;
    int64_t ldy;
};

// Launch tile plan tp on p: its split-K workspace (the allocated one, or the
// static scratch), then the kernel; e receives the launch status.
int run_tile_plan(int tp, const Problem &p, int dev, bool static_scratch, hipStream_t stream, hipError_t &e) {
    const TileSplit sp = tile_split_plan(tp, p.M, p.N, p.K);
    Workspace ws{};
    if (static_scratch && sp.split > 1) {
        const TileShape ts = tile_shape(PLANS[tp].tile_cfg);
        const int64_t split_tiles = tile_count(ts, p.M, p.N) - sp.full_tiles;
        const int64_t need = split_tiles * sp.split * ts.bm * ts.bn;
        if (need > WS_PARTIAL_FLOATS || split_tiles > WS_COUNTERS)
            return fail(KERNELARC_ERR_UNSUPPORTED,
                        "plan %s needs %lld fp32 partials and %lld counters; the static scratch holds %lld "
                        "and %lld", PLANS[tp].name, (long long)need, (long long)split_tiles,
                        (long long)WS_PARTIAL_FLOATS, (long long)WS_COUNTERS);
    }
    if (sp.split > 1) {
        const int wst = static_scratch ? scratch_workspace(dev, stream, &ws) : workspace(dev, stream, &ws);
        if (wst != KERNELARC_OK) return wst;
    }
    e = launch_tile(PLANS[tp].tile_cfg, p, sp.split, sp.full_tiles, sp.split > 1 ? &ws : nullptr, stream);
    return KERNELARC_OK;
}

// plan < 0: choose; otherwise run exactly that plan.  static_scratch: the
// split-K partials go to the static scratch instead of the allocated
// workspace (nothing is allocated).
int run(int plan, Request q, hipStream_t stream, bool static_scratch = false) {
    g_last_error[0] = '\0';
    const int64_t M = q.M, N = q.N, K = q.K;
    if (M < 0 || N < 0 || K < 0)
        return fail(KERNELARC_ERR_INVALID_ARG, "negative size M=%lld N=%lld K=%lld", (long long)M,
                    (long long)N, (long long)K);
    if (M > LIMIT_DIM || N > LIMIT_DIM || K > LIMIT_DIM)
        return fail(KERNELARC_ERR_INVALID_ARG, "a size is 2^31 or more");
    if (plan >= NUM_PLANS) return fail(KERNELARC_ERR_UNSUPPORTED, "unknown plan %d", plan);
    if (q.beta == 0.0f) q.R = nullptr;   // beta = 0: the residual term is not read
    const bool residual = q.R != nullptr;
    if (q.ldx < 0 || q.ldw < 0 || q.ldy < 0 || q.ldr < 0 || q.ldx > LIMIT_DIM || q.ldw > LIMIT_DIM ||
        q.ldy > LIMIT_DIM || q.ldr > LIMIT_DIM)
        return fail(KERNELARC_ERR_INVALID_ARG, "a leading dimension is negative or 2^31 or more");
    if (M == 0 || N == 0) return KERNELARC_OK;
    if (!q.Y) return fail(KERNELARC_ERR_INVALID_ARG, "Y is NULL");
    if (K > 0 && (!q.X || !q.W)) return fail(KERNELARC_ERR_INVALID_ARG, "X or W is NULL");
    if (q.ldy < N || (residual && q.ldr < N) || (K > 0 && (q.ldx < K || q.ldw < K)))
        return fail(KERNELARC_ERR_INVALID_ARG, "a leading dimension is smaller than its row length");
    const int64_t ybytes = strided_bytes(M, N, q.ldy);
    if (overlaps(q.Y, ybytes, q.X, strided_bytes(M, K, q.ldx)) || overlaps(q.Y, ybytes, q.W, strided_bytes(N, K, q.ldw)))
        return fail(KERNELARC_ERR_INVALID_ARG, "Y overlaps X or W");
    if (overlaps(q.Y, ybytes, q.bias, N * 2)) return fail(KERNELARC_ERR_INVALID_ARG, "Y overlaps the bias");
    if (residual && !(q.R == q.Y && q.ldr == q.ldy) && overlaps(q.Y, ybytes, q.R, strided_bytes(M, N, q.ldr)))
        return fail(KERNELARC_ERR_INVALID_ARG,
                    "Y partially overlaps R (only Y == R with the same leading dimension is allowed)");

    int dev = 0, num_cus = 0;
    const int st = current_device(&dev, &num_cus);
    if (st != KERNELARC_OK) return st;

    const Layout lay{q.ldx, q.ldw, residual ? q.ldr : N, q.ldy,
                     q.ldx != K || q.ldw != K || (residual && q.ldr != N) || q.ldy != N || q.alpha != 1.0f ||
                         q.beta != 1.0f || q.bias != nullptr};
    // 16-byte operand loads need every row of X and W 16-byte aligned.
    const bool vec_ok = aligned16(q.X) && aligned16(q.W) && aligned16(q.Y) && (!residual || aligned16(q.R)) &&
                        K % 8 == 0 && q.ldx % 8 == 0 && q.ldw % 8 == 0;
    if (plan < 0) {
        const PlanKey key{OP_LINEAR, (residual ? 1 : 0) | (lay.general ? 2 : 0), M, N, K, lay.ldx, lay.ldw, lay.ldr,
                          lay.ldy};
        plan = cached_plan(key, [&] { return select(M, N, K, residual, lay); });
        if (plan != PLAN_GENERIC && !vec_ok) plan = PLAN_GENERIC;
    } else {
        if (!supports(plan, M, N, K, residual, lay))
            return fail(KERNELARC_ERR_UNSUPPORTED, "plan %s cannot compute M=%lld N=%lld K=%lld%s",
                        PLANS[plan].name, (long long)M, (long long)N, (long long)K,
                        lay.general ? " in the general form" : "");
        if (plan != PLAN_GENERIC && !vec_ok)
            return fail(KERNELARC_ERR_UNSUPPORTED,
                        "plan %s needs 16-byte aligned pointers and K, ldx, ldw multiples of 8", PLANS[plan].name);
    }

    Problem p{M, N, K, static_cast<const uint16_t *>(q.X), static_cast<const uint16_t *>(q.W),
              static_cast<const uint16_t *>(q.R), static_cast<uint16_t *>(q.Y), q.ldx, q.ldw, lay.ldr, q.ldy,
              q.alpha, residual ? q.beta : 1.0f, static_cast<const uint16_t *>(q.bias)};
    (void)hipGetLastError();   // clear any stale error before launching
    hipError_t e = hipSuccess;
    switch (PLANS[plan].kind) {
        case KIND_GENERIC:
            e = launch_generic(p, stream);
            break;
        case KIND_GEMV:
            e = launch_gemv(p, stream);
            break;
        case KIND_TILE: {
            const int st_tile = run_tile_plan(plan, p, dev, static_scratch, stream, e);
            if (st_tile != KERNELARC_OK) return st_tile;
            break;
        }
        case KIND_BANDS: {
            // Two launches on the stream: the columns [0, N1) and [N1, N)
            // are independent, each element computed by one of them.
            const int64_t N1 = band_split(M, N);
            if (N1 > 0) {
                Problem p1 = p;
                p1.N = N1;
                const int st1 = run_tile_plan(plan_index(BAND_MAIN), p1, dev, static_scratch, stream, e);
                if (st1 != KERNELARC_OK) return st1;
            }
            if (N1 < N && e == hipSuccess) {
                Problem p2 = p;
                p2.N = N - N1;
                p2.W += N1 * q.ldw;
                if (p2.R) p2.R += N1;
                p2.Y += N1;
                if (p2.bias) p2.bias += N1;
                const int st2 = run_tile_plan(plan_index(BAND_REST), p2, dev, static_scratch, stream, e);
                if (st2 != KERNELARC_OK) return st2;
            }
            break;
        }
        case KIND_STREAM: {
            const int split = stream_split_of(plan, M, N, K);
            Workspace ws{};
            if (static_scratch && split > 1) {
                const int64_t need = stream_workspace_floats(M, N, split, PLANS[plan].rows);
                const int64_t counters = stream_counter_count(N, PLANS[plan].rows);
                if (need > WS_PARTIAL_FLOATS || counters > WS_COUNTERS)
                    return fail(KERNELARC_ERR_UNSUPPORTED,
                                "plan %s needs %lld fp32 partials and %lld counters; the static scratch holds %lld "
                                "and %lld", PLANS[plan].name, (long long)need, (long long)counters,
                                (long long)WS_PARTIAL_FLOATS, (long long)WS_COUNTERS);
            }
            if (split > 1) {
                const int wst = static_scratch ? scratch_workspace(dev, stream, &ws) : workspace(dev, stream, &ws);
                if (wst != KERNELARC_OK) return wst;
            }
            e = launch_stream(p, PLANS[plan].tile_cfg, PLANS[plan].stages, PLANS[plan].rows, split,
                              split > 1 ? &ws : nullptr, stream);
            break;
        }
    }
    if (e != hipSuccess)
        return fail(KERNELARC_ERR_LAUNCH, "launch of %s failed: %s", PLANS[plan].name, hipGetErrorString(e));
    return KERNELARC_OK;
}

// SwiGLU call: H = bf16(silu(X Wg^T) * (X Wu^T)); plan < 0: choose.
int run_glu(int plan, int64_t M, int64_t N, int64_t K, const void *X, const void *Wg, const void *Wu, void *H,
            hipStream_t stream) {
    g_last_error[0] = '\0';
    if (M < 0 || N < 0 || K < 0)
        return fail(KERNELARC_ERR_INVALID_ARG, "negative size M=%lld N=%lld K=%lld", (long long)M,
                    (long long)N, (long long)K);
    if (M > LIMIT_DIM || N > LIMIT_DIM / 2 || K > LIMIT_DIM)
        return fail(KERNELARC_ERR_INVALID_ARG, "a size is too large (M, K < 2^31, N < 2^30)");
    if (plan >= NUM_PLANS) return fail(KERNELARC_ERR_UNSUPPORTED, "unknown plan %d", plan);
    if (M == 0 || N == 0) return KERNELARC_OK;
    if (!H) return fail(KERNELARC_ERR_INVALID_ARG, "H is NULL");
    if (K > 0 && (!X || !Wg || !Wu)) return fail(KERNELARC_ERR_INVALID_ARG, "X, Wg or Wu is NULL");
    const int64_t hbytes = M * N * 2;
    if (overlaps(H, hbytes, X, M * K * 2) || overlaps(H, hbytes, Wg, N * K * 2) || overlaps(H, hbytes, Wu, N * K * 2))
        return fail(KERNELARC_ERR_INVALID_ARG, "H overlaps X, Wg or Wu");

    int dev = 0, num_cus = 0;
    const int st = current_device(&dev, &num_cus);
    if (st != KERNELARC_OK) return st;

    const bool vec_ok = aligned16(X) && aligned16(Wg) && aligned16(Wu) && aligned16(H) && K % 8 == 0;
    if (plan < 0) {
        plan = cached_plan(PlanKey{OP_GLU, 0, M, N, K, 0, 0, 0, 0}, [&] { return select_glu(M, N, K); });
        if (plan != PLAN_GENERIC && !vec_ok) plan = PLAN_GENERIC;
    } else {
        if (!supports_glu(plan, M, N, K))
            return fail(KERNELARC_ERR_UNSUPPORTED, "plan %s cannot compute SwiGLU at M=%lld N=%lld K=%lld",
                        PLANS[plan].name, (long long)M, (long long)N, (long long)K);
        if (plan != PLAN_GENERIC && !vec_ok)
            return fail(KERNELARC_ERR_UNSUPPORTED, "plan %s needs 16-byte aligned pointers and K a multiple of 8",
                        PLANS[plan].name);
    }
    const GluProblem p{M, N, K, static_cast<const uint16_t *>(X), static_cast<const uint16_t *>(Wg),
                       static_cast<const uint16_t *>(Wu), static_cast<uint16_t *>(H)};
    (void)hipGetLastError();
    hipError_t e = hipSuccess;
    if (PLANS[plan].kind == KIND_GENERIC) {
        e = launch_generic_glu(p, stream);
    } else {
        const TileSplit sp = tile_split_plan(plan, M, 2 * N, K);
        Workspace ws{};
        if (sp.split > 1) {
            const int wst = workspace(dev, stream, &ws);
            if (wst != KERNELARC_OK) return wst;
        }
        e = launch_tile_glu(PLANS[plan].tile_cfg, p, sp.split, sp.full_tiles, sp.split > 1 ? &ws : nullptr, stream);
    }
    if (e != hipSuccess)
        return fail(KERNELARC_ERR_LAUNCH, "launch of %s failed: %s", PLANS[plan].name, hipGetErrorString(e));
    return KERNELARC_OK;
}

bool aligned4(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

// Grouped call: per group g, Y[g] = X[g] W[g]^T (or SwiGLU with W2) on its
// valid rows; plan < 0: choose.
int run_grouped(int plan, bool glu, int64_t G, int64_t Mpad, int64_t N, int64_t K, const void *X, const void *W,
                const void *W2, const int32_t *counts, void *Y, hipStream_t stream) {
    g_last_error[0] = '\0';
    if (G < 0 || Mpad < 0 || N < 0 || K < 0)
        return fail(KERNELARC_ERR_INVALID_ARG, "negative size G=%lld M_pad=%lld N=%lld K=%lld", (long long)G,
                    (long long)Mpad, (long long)N, (long long)K);
    if (Mpad > LIMIT_DIM || N > (glu ? LIMIT_DIM / 2 : LIMIT_DIM) || K > LIMIT_DIM ||
        (Mpad > 0 && G > LIMIT_DIM / Mpad))
        return fail(KERNELARC_ERR_INVALID_ARG, "a size is too large (G * M_pad, K below 2^31)");
    if (plan >= NUM_PLANS) return fail(KERNELARC_ERR_UNSUPPORTED, "unknown plan %d", plan);
    if (G == 0 || Mpad == 0 || N == 0) return KERNELARC_OK;
    if (!Y) return fail(KERNELARC_ERR_INVALID_ARG, "the output is NULL");
    if (K > 0 && (!X || !W || (glu && !W2))) return fail(KERNELARC_ERR_INVALID_ARG, "an operand is NULL");
    if (counts && !aligned4(counts)) return fail(KERNELARC_ERR_INVALID_ARG, "counts must be 4-byte aligned");
    const int64_t ybytes = G * Mpad * N * 2, wbytes = G * N * K * 2;
    if (overlaps(Y, ybytes, X, G * Mpad * K * 2) || overlaps(Y, ybytes, W, wbytes) ||
        (glu && overlaps(Y, ybytes, W2, wbytes)) || overlaps(Y, ybytes, counts, G * 4))
        return fail(KERNELARC_ERR_INVALID_ARG, "the output overlaps an operand or the counts");

    int dev = 0, num_cus = 0;
    const int st = current_device(&dev, &num_cus);
    if (st != KERNELARC_OK) return st;

    const bool vec_ok = aligned16(X) && aligned16(W) && (!glu || aligned16(W2)) && aligned16(Y) && K % 8 == 0;
    if (plan < 0) {
        plan = cached_plan(PlanKey{glu ? OP_GROUPED_GLU : OP_GROUPED, 0, Mpad, N, K, G, 0, 0, 0},
                           [&] { return select_grouped(G, Mpad, N, K, glu); });
        if (plan != PLAN_GENERIC && !vec_ok) plan = PLAN_GENERIC;
    } else {
        if (!supports_grouped(plan, G, Mpad, N, K, glu))
            return fail(KERNELARC_ERR_UNSUPPORTED, "plan %s cannot compute the grouped %s at G=%lld M_pad=%lld N=%lld K=%lld",
                        PLANS[plan].name, glu ? "SwiGLU" : "GEMM", (long long)G, (long long)Mpad, (long long)N,
                        (long long)K);
        if (plan != PLAN_GENERIC && !vec_ok)
            return fail(KERNELARC_ERR_UNSUPPORTED, "plan %s needs 16-byte aligned pointers and K a multiple of 8",
                        PLANS[plan].name);
    }
    (void)hipGetLastError();
    hipError_t e = hipSuccess;
    const auto *x = static_cast<const uint16_t *>(X);
    const auto *w = static_cast<const uint16_t *>(W);
    auto *y = static_cast<uint16_t *>(Y);
    if (glu) {
        Grouped<GluProblem> p{};
        static_cast<GluProblem &>(p) = GluProblem{0, N, K, x, w, static_cast<const uint16_t *>(W2), y};
        p.G = G;
        p.Mpad = Mpad;
        p.counts = counts;
        e = PLANS[plan].kind == KIND_GENERIC ? launch_generic_grouped_glu(p, stream)
                                             : launch_tile_grouped_glu(PLANS[plan].tile_cfg, p, stream);
    } else {
        Grouped<DenseProblem> p{};
        static_cast<DenseProblem &>(p) = DenseProblem{0, N, K, x, w, nullptr, y};
        p.G = G;
        p.Mpad = Mpad;
        p.counts = counts;
        e = PLANS[plan].kind == KIND_GENERIC ? launch_generic_grouped(p, stream)
                                             : launch_tile_grouped(PLANS[plan].tile_cfg, p, stream);
    }
    if (e != hipSuccess)
        return fail(KERNELARC_ERR_LAUNCH, "launch of %s failed: %s", PLANS[plan].name, hipGetErrorString(e));
    return KERNELARC_OK;
}

// INT8 call.  glu: H = bf16(silu(sx swg Ag) (sx swu Au)) (W2, sw2 the up
// operands); else Y = bf16(sx sw A (+ R)).  plan < 0: choose.
int run_i8(int plan, bool glu, int64_t M, int64_t N, int64_t K, const void *X, const float *sx, const void *W,
           const float *sw, const void *W2, const float *sw2, const void *R, void *Y, hipStream_t stream,
           bool f8 = false) {
    g_last_error[0] = '\0';
    if (M < 0 || N < 0 || K < 0)
        return fail(KERNELARC_ERR_INVALID_ARG, "negative size M=%lld N=%lld K=%lld", (long long)M,
                    (long long)N, (long long)K);
    if (M > LIMIT_DIM || N > (glu ? LIMIT_DIM / 2 : LIMIT_DIM))
        return fail(KERNELARC_ERR_INVALID_ARG, "a size is too large");
    if (!f8 && K > I8_MAX_K)
        return fail(KERNELARC_ERR_INVALID_ARG, "K=%lld above %lld could overflow the int32 sums", (long long)K,
                    (long long)I8_MAX_K);
    if (K > LIMIT_DIM) return fail(KERNELARC_ERR_INVALID_ARG, "K is 2^31 or more");
    if (plan >= NUM_PLANS) return fail(KERNELARC_ERR_UNSUPPORTED, "unknown plan %d", plan);
    if (M == 0 || N == 0) return KERNELARC_OK;
    if (!Y) return fail(KERNELARC_ERR_INVALID_ARG, "the output is NULL");
    if (K > 0 && (!X || !W || (glu && !W2))) return fail(KERNELARC_ERR_INVALID_ARG, "an int8 operand is NULL");
    if (!sx || !sw || (glu && !sw2)) return fail(KERNELARC_ERR_INVALID_ARG, "a scale vector is NULL");
    if (!aligned4(sx) || !aligned4(sw) || (glu && !aligned4(sw2)))
        return fail(KERNELARC_ERR_INVALID_ARG, "scale vectors must be 4-byte aligned");
    const int64_t ybytes = M * N * 2;
    if (overlaps(Y, ybytes, X, M * K) || overlaps(Y, ybytes, W, N * K) || (glu && overlaps(Y, ybytes, W2, N * K)) ||
        overlaps(Y, ybytes, sx, M * 4) || overlaps(Y, ybytes, sw, N * 4) || (glu && overlaps(Y, ybytes, sw2, N * 4)))
        return fail(KERNELARC_ERR_INVALID_ARG, "the output overlaps an operand or a scale vector");
    if (R && R != Y && overlaps(Y, ybytes, R, ybytes))
        return fail(KERNELARC_ERR_INVALID_ARG, "Y partially overlaps R (only Y == R is allowed)");

    int dev = 0, num_cus = 0;
    const int st = current_device(&dev, &num_cus);
    if (st != KERNELARC_OK) return st;

    const bool vec_ok = aligned16(X) && aligned16(W) && (!glu || aligned16(W2)) && aligned16(Y) &&
                        (!R || aligned16(R)) && K % 16 == 0;
    if (plan < 0) {
        const int op = f8 ? (glu ? OP_F8_GLU : OP_F8) : (glu ? OP_I8_GLU : OP_I8);
        plan = cached_plan(PlanKey{op, 0, M, N, K, 0, 0, 0, 0}, [&] { return select_i8(M, N, K, glu, f8); });
        if (plan != PLAN_GENERIC && !vec_ok) plan = PLAN_GENERIC;
    } else {
        if (!supports_i8(plan, M, N, K, glu, f8))
            return fail(KERNELARC_ERR_UNSUPPORTED, "plan %s cannot compute the %s %s at M=%lld N=%lld K=%lld",
                        PLANS[plan].name, f8 ? "FP8" : "INT8", glu ? "SwiGLU" : "GEMM", (long long)M, (long long)N,
                        (long long)K);
        if (plan != PLAN_GENERIC && !vec_ok)
            return fail(KERNELARC_ERR_UNSUPPORTED, "plan %s needs 16-byte aligned operands and K a multiple of 16",
                        PLANS[plan].name);
    }
    (void)hipGetLastError();
    hipError_t e = hipSuccess;
    const auto *x8 = static_cast<const int8_t *>(X);
    const auto *w8 = static_cast<const int8_t *>(W);
    if (f8) {
        const auto *xf = static_cast<const uint8_t *>(X);
        const auto *wf = static_cast<const uint8_t *>(W);
        const bool generic = PLANS[plan].kind == KIND_GENERIC;
        if (glu) {
            const F8GluProblem p{M, N, K, xf, wf, static_cast<const uint8_t *>(W2), static_cast<uint16_t *>(Y),
                                 sx, sw, sw2};
            if (generic) {
                e = launch_generic_f8_glu(p, stream);
            } else {
                const TileSplit sp = tile_split_plan(plan, M, 2 * N, K / 2);
                Workspace ws{};
                if (sp.split > 1) {
                    const int wst = workspace(dev, stream, &ws);
                    if (wst != KERNELARC_OK) return wst;
                }
                e = launch_tile_f8_glu(PLANS[plan].tile_cfg, p, sp.split, sp.full_tiles, sp.split > 1 ? &ws : nullptr,
                                       stream);
            }
        } else {
            const F8Problem p{M, N, K, xf, wf, static_cast<const uint16_t *>(R), static_cast<uint16_t *>(Y), sx, sw};
            if (generic) {
                e = launch_generic_f8(p, stream);
            } else {
                const TileSplit sp = tile_split_plan(plan, M, N, K / 2);
                Workspace ws{};
                if (sp.split > 1) {
                    const int wst = workspace(dev, stream, &ws);
                    if (wst != KERNELARC_OK) return wst;
                }
                e = launch_tile_f8(PLANS[plan].tile_cfg, p, sp.split, sp.full_tiles, sp.split > 1 ? &ws : nullptr,
                                   stream);
            }
        }
    } else if (PLANS[plan].kind == KIND_STREAM) {
        const int split = stream_split_of(plan, M, N, K / 2);
        Workspace ws{};
        if (split > 1) {
            const int wst = workspace(dev, stream, &ws);
            if (wst != KERNELARC_OK) return wst;
        }
        e = launch_stream_i8(I8Problem{M, N, K, x8, w8, static_cast<const uint16_t *>(R), static_cast<uint16_t *>(Y),
                                       sx, sw},
                             PLANS[plan].tile_cfg, PLANS[plan].stages, PLANS[plan].rows, split,
                             split > 1 ? &ws : nullptr, stream);
    } else if (PLANS[plan].kind == KIND_GENERIC) {
        if (glu)
            e = launch_generic_i8_glu(I8GluProblem{M, N, K, x8, w8, static_cast<const int8_t *>(W2),
                                                   static_cast<uint16_t *>(Y), sx, sw, sw2},
                                      stream);
        else
            e = launch_generic_i8(I8Problem{M, N, K, x8, w8, static_cast<const uint16_t *>(R),
                                            static_cast<uint16_t *>(Y), sx, sw},
                                  stream);
    } else {
        const TileSplit sp = tile_split_plan(plan, M, glu ? 2 * N : N, K / 2);
        Workspace ws{};
        if (sp.split > 1) {
            const int wst = workspace(dev, stream, &ws);
            if (wst != KERNELARC_OK) return wst;
        }
        const Workspace *wsp = sp.split > 1 ? &ws : nullptr;
        if (glu)
            e = launch_tile_i8_glu(PLANS[plan].tile_cfg,
                                   I8GluProblem{M, N, K, x8, w8, static_cast<const int8_t *>(W2),
                                                static_cast<uint16_t *>(Y), sx, sw, sw2},
                                   sp.split, sp.full_tiles, wsp, stream);
        else
            e = launch_tile_i8(PLANS[plan].tile_cfg,
                               I8Problem{M, N, K, x8, w8, static_cast<const uint16_t *>(R), static_cast<uint16_t *>(Y),
                                         sx, sw},
                               sp.split, sp.full_tiles, wsp, stream);
    }
    if (e != hipSuccess)
        return fail(KERNELARC_ERR_LAUNCH, "launch of %s failed: %s", PLANS[plan].name, hipGetErrorString(e));
    return KERNELARC_OK;
}

}  // namespace
}  // namespace kernelarc

using namespace kernelarc;

extern "C" {

Request dense_request(int64_t M, int64_t N, int64_t K, const void *X, const void *W, const void *R, void *Y) {
    return Request{M, N, K, 1.0f, X, K, W, K, 1.0f, R, N, nullptr, Y, N};
}

int kernelarc_gemm_bf16_residual(int64_t M, int64_t N, int64_t K, const void *X, const void *W,
                                 const void *R, void *Y, hipStream_t stream) {
    if (!R && M > 0 && N > 0) {
        g_last_error[0] = '\0';
        return fail(KERNELARC_ERR_INVALID_ARG, "R is NULL");
    }
    return run(-1, dense_request(M, N, K, X, W, R, Y), stream);
}

int kernelarc_gemm_bf16(int64_t M, int64_t N, int64_t K, const void *X, const void *W, void *Y,
                        hipStream_t stream) {
    return run(-1, dense_request(M, N, K, X, W, nullptr, Y), stream);
}

int kernelarc_gemm_bf16_residual_noalloc(int64_t M, int64_t N, int64_t K, const void *X, const void *W,
                                         const void *R, void *Y, hipStream_t stream) {
    return run(-1, dense_request(M, N, K, X, W, R, Y), stream, true);
}

int kernelarc_gemm_bf16_with_plan(int plan, int64_t M, int64_t N, int64_t K, const void *X,
                                  const void *W, const void *R, void *Y, hipStream_t stream) {
    if (plan < 0) {
        g_last_error[0] = '\0';
        return fail(KERNELARC_ERR_UNSUPPORTED, "unknown plan %d", plan);
    }
    return run(plan, dense_request(M, N, K, X, W, R, Y), stream);
}

int kernelarc_gemm_bf16_ex(int64_t M, int64_t N, int64_t K, float alpha, const void *X, int64_t ldx,
                           const void *W, int64_t ldw, float beta, const void *C, int64_t ldc, const void *bias,
                           void *Y, int64_t ldy, hipStream_t stream) {
    return run(-1, Request{M, N, K, alpha, X, ldx, W, ldw, beta, C, ldc, bias, Y, ldy}, stream);
}

int kernelarc_gemm_bf16_ex_with_plan(int plan, int64_t M, int64_t N, int64_t K, float alpha, const void *X,
                                     int64_t ldx, const void *W, int64_t ldw, float beta, const void *C,
                                     int64_t ldc, const void *bias, void *Y, int64_t ldy, hipStream_t stream) {
    if (plan < 0) {
        g_last_error[0] = '\0';
        return fail(KERNELARC_ERR_UNSUPPORTED, "unknown plan %d", plan);
    }
    return run(plan, Request{M, N, K, alpha, X, ldx, W, ldw, beta, C, ldc, bias, Y, ldy}, stream);
}

int kernelarc_select_plan_ex(int64_t M, int64_t N, int64_t K, int has_c, int64_t ldx, int64_t ldw, int64_t ldc,
                             int64_t ldy, float alpha, float beta, int has_bias) {
    if (M < 0 || N < 0 || K < 0) return -1;
    const bool residual = has_c != 0 && beta != 0.0f;
    const Layout lay{ldx, ldw, residual ? ldc : N, ldy,
                     ldx != K || ldw != K || (residual && ldc != N) || ldy != N || alpha != 1.0f || beta != 1.0f ||
                         has_bias != 0};
    return select(M, N, K, residual, lay);
}

int kernelarc_swiglu_bf16(int64_t M, int64_t N, int64_t K, const void *X, const void *Wg, const void *Wu, void *H,
                          hipStream_t stream) {
    return run_glu(-1, M, N, K, X, Wg, Wu, H, stream);
}

int kernelarc_swiglu_bf16_with_plan(int plan, int64_t M, int64_t N, int64_t K, const void *X, const void *Wg,
                                    const void *Wu, void *H, hipStream_t stream) {
    if (plan < 0) {
        g_last_error[0] = '\0';
        return fail(KERNELARC_ERR_UNSUPPORTED, "unknown plan %d", plan);
    }
    return run_glu(plan, M, N, K, X, Wg, Wu, H, stream);
}

int kernelarc_select_plan_swiglu(int64_t M, int64_t N, int64_t K) { return select_glu(M, N, K); }

int kernelarc_plan_supports_swiglu(int plan, int64_t M, int64_t N, int64_t K) {
    if (plan < 0 || plan >= NUM_PLANS || M < 0 || N < 0 || K < 0) return -1;
    return supports_glu(plan, M, N, K) ? 1 : 0;
}

int kernelarc_gemm_i8(int64_t M, int64_t N, int64_t K, const void *qX, const float *sx, const void *qW,
                      const float *sw, const void *R, void *Y, hipStream_t stream) {
    return run_i8(-1, false, M, N, K, qX, sx, qW, sw, nullptr, nullptr, R, Y, stream);
}

int kernelarc_gemm_i8_with_plan(int plan, int64_t M, int64_t N, int64_t K, const void *qX, const float *sx,
                                const void *qW, const float *sw, const void *R, void *Y, hipStream_t stream) {
    if (plan < 0) {
        g_last_error[0] = '\0';
        return fail(KERNELARC_ERR_UNSUPPORTED, "unknown plan %d", plan);
    }
    return run_i8(plan, false, M, N, K, qX, sx, qW, sw, nullptr, nullptr, R, Y, stream);
}

int kernelarc_swiglu_i8(int64_t M, int64_t N, int64_t K, const void *qX, const float *sx, const void *qWg,
                        const float *swg, const void *qWu, const float *swu, void *H, hipStream_t stream) {
    return run_i8(-1, true, M, N, K, qX, sx, qWg, swg, qWu, swu, nullptr, H, stream);
}

int kernelarc_swiglu_i8_with_plan(int plan, int64_t M, int64_t N, int64_t K, const void *qX, const float *sx,
                                  const void *qWg, const float *swg, const void *qWu, const float *swu, void *H,
                                  hipStream_t stream) {
    if (plan < 0) {
        g_last_error[0] = '\0';
        return fail(KERNELARC_ERR_UNSUPPORTED, "unknown plan %d", plan);
    }
    return run_i8(plan, true, M, N, K, qX, sx, qWg, swg, qWu, swu, nullptr, H, stream);
}

int kernelarc_select_plan_i8(int64_t M, int64_t N, int64_t K, int swiglu) { return select_i8(M, N, K, swiglu != 0); }

int kernelarc_gemm_f8(int64_t M, int64_t N, int64_t K, const void *qX, const float *sx, const void *qW,
                      const float *sw, const void *R, void *Y, hipStream_t stream) {
    return run_i8(-1, false, M, N, K, qX, sx, qW, sw, nullptr, nullptr, R, Y, stream, true);
}

int kernelarc_gemm_f8_with_plan(int plan, int64_t M, int64_t N, int64_t K, const void *qX, const float *sx,
                                const void *qW, const float *sw, const void *R, void *Y, hipStream_t stream) {
    if (plan < 0) {
        g_last_error[0] = '\0';
        return fail(KERNELARC_ERR_UNSUPPORTED, "unknown plan %d", plan);
    }
    return run_i8(plan, false, M, N, K, qX, sx, qW, sw, nullptr, nullptr, R, Y, stream, true);
}

int kernelarc_swiglu_f8(int64_t M, int64_t N, int64_t K, const void *qX, const float *sx, const void *qWg,
                        const float *swg, const void *qWu, const float *swu, void *H, hipStream_t stream) {
    return run_i8(-1, true, M, N, K, qX, sx, qWg, swg, qWu, swu, nullptr, H, stream, true);
}

int kernelarc_swiglu_f8_with_plan(int plan, int64_t M, int64_t N, int64_t K, const void *qX, const float *sx,
                                  const void *qWg, const float *swg, const void *qWu, const float *swu, void *H,
                                  hipStream_t stream) {
    if (plan < 0) {
        g_last_error[0] = '\0';
        return fail(KERNELARC_ERR_UNSUPPORTED, "unknown plan %d", plan);
    }
    return run_i8(plan, true, M, N, K, qX, sx, qWg, swg, qWu, swu, nullptr, H, stream, true);
}

int kernelarc_select_plan_f8(int64_t M, int64_t N, int64_t K, int swiglu) {
    return select_i8(M, N, K, swiglu != 0, true);
}

int kernelarc_plan_supports_f8(int plan, int64_t M, int64_t N, int64_t K, int swiglu) {
    if (plan < 0 || plan >= NUM_PLANS || M < 0 || N < 0 || K < 0) return -1;
    return supports_i8(plan, M, N, K, swiglu != 0, true) ? 1 : 0;
}

int kernelarc_plan_supports_i8(int plan, int64_t M, int64_t N, int64_t K, int swiglu) {
    if (plan < 0 || plan >= NUM_PLANS || M < 0 || N < 0 || K < 0) return -1;
    return supports_i8(plan, M, N, K, swiglu != 0) ? 1 : 0;
}

int kernelarc_gemm_bf16_grouped(int64_t G, int64_t M_pad, int64_t N, int64_t K, const void *X, const void *W,
                                const int32_t *counts, void *Y, hipStream_t stream) {
    return run_grouped(-1, false, G, M_pad, N, K, X, W, nullptr, counts, Y, stream);
}

int kernelarc_gemm_bf16_grouped_with_plan(int plan, int64_t G, int64_t M_pad, int64_t N, int64_t K, const void *X,
                                          const void *W, const int32_t *counts, void *Y, hipStream_t stream) {
    if (plan < 0) {
        g_last_error[0] = '\0';
        return fail(KERNELARC_ERR_UNSUPPORTED, "unknown plan %d", plan);
    }
    return run_grouped(plan, false, G, M_pad, N, K, X, W, nullptr, counts, Y, stream);
}

int kernelarc_swiglu_bf16_grouped(int64_t G, int64_t M_pad, int64_t N, int64_t K, const void *X, const void *Wg,
                                  const void *Wu, const int32_t *counts, void *H, hipStream_t stream) {
    return run_grouped(-1, true, G, M_pad, N, K, X, Wg, Wu, counts, H, stream);
}

int kernelarc_swiglu_bf16_grouped_with_plan(int plan, int64_t G, int64_t M_pad, int64_t N, int64_t K, const void *X,
                                            const void *Wg, const void *Wu, const int32_t *counts, void *H,
                                            hipStream_t stream) {
    if (plan < 0) {
        g_last_error[0] = '\0';
        return fail(KERNELARC_ERR_UNSUPPORTED, "unknown plan %d", plan);
    }
    return run_grouped(plan, true, G, M_pad, N, K, X, Wg, Wu, counts, H, stream);
}

int kernelarc_select_plan_grouped(int64_t G, int64_t M_pad, int64_t N, int64_t K, int swiglu) {
    return select_grouped(G, M_pad, N, K, swiglu != 0);
}

int kernelarc_plan_supports_grouped(int plan, int64_t G, int64_t M_pad, int64_t N, int64_t K, int swiglu) {
    if (plan < 0 || plan >= NUM_PLANS || G < 0 || M_pad < 0 || N < 0 || K < 0) return -1;
    return supports_grouped(plan, G, M_pad, N, K, swiglu != 0) ? 1 : 0;
}

int kernelarc_plan_count(void) { return NUM_PLANS; }

const char *kernelarc_plan_label(int plan) {
    return (plan >= 0 && plan < NUM_PLANS) ? PLANS[plan].name : nullptr;
}

int kernelarc_plan_name(int64_t M, int64_t N, int64_t K, int residual, char *buf, size_t len) {
    g_last_error[0] = '\0';
    if (M < 0 || N < 0 || K < 0)
        return fail(KERNELARC_ERR_INVALID_ARG, "negative size M=%lld N=%lld K=%lld", (long long)M, (long long)N,
                    (long long)K);
    if (!buf) return fail(KERNELARC_ERR_INVALID_ARG, "buf is NULL");
    const int plan = select(M, N, K, residual != 0, dense_layout(N, K));
    const size_t need = std::strlen(PLANS[plan].name) + 1;
    if (len < need) return fail(KERNELARC_ERR_INVALID_ARG, "buf holds %zu bytes; the name needs %zu", len, need);
    std::memcpy(buf, PLANS[plan].name, need);
    return KERNELARC_OK;
}

int kernelarc_plan_supports(int plan, int64_t M, int64_t N, int64_t K, int residual) {
    if (plan < 0 || plan >= NUM_PLANS || M < 0 || N < 0 || K < 0) return -1;
    return supports(plan, M, N, K, residual != 0, dense_layout(N, K)) ? 1 : 0;
}

int kernelarc_select_plan(int64_t M, int64_t N, int64_t K, int residual) {
    return select(M, N, K, residual != 0, dense_layout(N, K));
}

int kernelarc_plan_uses_workspace(int plan, int64_t M, int64_t N, int64_t K) {
    if (!supports(plan, M, N, K, true, dense_layout(N, K))) return 0;
    if (PLANS[plan].kind == KIND_TILE) return tile_split_of(plan, M, N, K) > 1 ? 1 : 0;
    if (PLANS[plan].kind == KIND_STREAM) return stream_split_of(plan, M, N, K) > 1 ? 1 : 0;
    if (PLANS[plan].kind == KIND_BANDS) {
        const int64_t N1 = band_split(M, N);
        return (N1 > 0 && tile_split_of(plan_index(BAND_MAIN), M, N1, K) > 1) ||
                       (N1 < N && tile_split_of(plan_index(BAND_REST), M, N - N1, K) > 1)
                   ? 1
                   : 0;
    }
    return 0;
}

const char *kernelarc_status_string(int status) {
    switch (status) {
        case KERNELARC_OK: return "ok";
        case KERNELARC_ERR_INVALID_ARG: return "invalid argument";
        case KERNELARC_ERR_UNSUPPORTED: return "unsupported (device or plan)";
        case KERNELARC_ERR_LAUNCH: return "launch failed";
        default: return "unknown status";
    }
}

const char *kernelarc_last_error(void) { return g_last_error; }

}  // extern "C"
