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
constexpr int64_t WS_PARTIAL_FLOATS = int64_t{1} << 20;
constexpr int64_t WS_COUNTERS = int64_t{1} << 16;

struct PlanInfo {
    const char *name;
    int bm, bn;   // macro-tile edge for tile plans, 0 otherwise
};

const PlanInfo PLANS[PLAN_COUNT] = {
    {"generic_64x64_scalar", 0, 0},
    {"skinny_mfma16_w8", 0, 0},
    {"skinny_mfma16_w8_splitk", 0, 0},
    {"tile_256x256x64_mfma32_w4", 256, 256},
    {"tile_256x128x64_mfma32_w4", 256, 128},
    {"tile_128x128x64_mfma32_w4", 128, 128},
};

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

int skinny_split_of(int plan, int64_t M, int64_t N, int64_t K) {
    if (plan == PLAN_SKINNY) return 1;
    const int rule = skinny_split_for(M, N, K);
    return rule < 2 ? 2 : rule;
}

bool supports(int plan, int64_t M, int64_t N, int64_t K, bool residual) {
    (void)residual;
    if (M < 0 || N < 0 || K < 0 || M > LIMIT_DIM || N > LIMIT_DIM || K > LIMIT_DIM) return false;
    switch (plan) {
        case PLAN_GENERIC:
            return cdiv(M, 64) * cdiv(N, 64) * 256 <= LIMIT_ITEMS;
        case PLAN_SKINNY:
        case PLAN_SKINNY_SPLITK: {
            if (M < 1 || M > 64 || K % 8 != 0) return false;
            if (N * K * 2 >= PANEL_LIMIT || 64 * K * 2 >= PANEL_LIMIT) return false;
            const int split = skinny_split_of(plan, M, N, K);
            if (cdiv(N, 16) * split * 512 > LIMIT_ITEMS) return false;
            if (split > 1 && (skinny_workspace_floats(M, N, split) > WS_PARTIAL_FLOATS ||
                              skinny_counter_count(N) > WS_COUNTERS))
                return false;
            return true;
        }
        case PLAN_TILE_256x256:
        case PLAN_TILE_256x128:
        case PLAN_TILE_128x128: {
            const PlanInfo &pi = PLANS[plan];
            if (K % 8 != 0) return false;
            if (int64_t{pi.bm} * K * 2 >= PANEL_LIMIT || int64_t{pi.bn} * K * 2 >= PANEL_LIMIT) return false;
            if (int64_t{pi.bm} * N * 2 >= PANEL_LIMIT) return false;   // epilogue panel of R / Y
            return cdiv(M, pi.bm) * cdiv(N, pi.bn) * 256 <= LIMIT_ITEMS;
        }
        default:
            return false;
    }
}

// Exact-shape entries (M, N, K, residual) -> plan; filled from measurements.
struct TableEntry {
    int64_t M, N, K;
    int residual;
    int plan;
};
const TableEntry TABLE[] = {
    {0, 0, 0, 0, -1},   // sentinel
};

// Relative cost of one output element for each macro tile (larger tiles
// reuse each staged byte more often) and how many workgroups a CU holds.
int select(int64_t M, int64_t N, int64_t K, bool residual) {
    if (M < 0 || N < 0 || K < 0) return -1;
    for (const TableEntry &e : TABLE)
        if (e.plan >= 0 && e.M == M && e.N == N && e.K == K && (e.residual != 0) == residual &&
            supports(e.plan, M, N, K, residual))
            return e.plan;
    if (K % 8 != 0) return PLAN_GENERIC;
    if (M >= 1 && M <= 64) {
        const int plan = skinny_split_for(M, N, K) > 1 ? PLAN_SKINNY_SPLITK : PLAN_SKINNY;
        if (supports(plan, M, N, K, residual)) return plan;
        if (supports(PLAN_SKINNY, M, N, K, residual)) return PLAN_SKINNY;
    }
    struct Cand {
        int plan;
        double per_elem;
        int per_cu;
    };
    const Cand cands[] = {
        {PLAN_TILE_256x256, 1.00, 1},
        {PLAN_TILE_256x128, 1.12, 1},
        {PLAN_TILE_128x128, 1.35, 2},
    };
    const int64_t cus = 256;
    int best = -1;
    double best_cost = 0.0;
    for (const Cand &c : cands) {
        if (!supports(c.plan, M, N, K, residual)) continue;
        const PlanInfo &pi = PLANS[c.plan];
        const int64_t tiles = cdiv(M, pi.bm) * cdiv(N, pi.bn);
        const int64_t rounds = cdiv(tiles, cus * c.per_cu);
        const double cost = static_cast<double>(rounds) * c.per_cu * pi.bm * pi.bn * c.per_elem;
        if (best < 0 || cost < best_cost) {
            best = c.plan;
            best_cost = cost;
        }
    }
    return best >= 0 ? best : PLAN_GENERIC;
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

// The split-K workspace of device `dev`, allocated and zeroed on first use.
int workspace(int dev, hipStream_t stream, Workspace *out) {
    std::lock_guard<std::mutex> lock(g_mutex);
    DeviceState &st = g_devices[dev];
    if (!st.ws_partials) {
        void *parts = nullptr;
        void *counters = nullptr;
        hipError_t e = hipMalloc(&parts, WS_PARTIAL_FLOATS * sizeof(float));
        if (e == hipSuccess) e = hipMalloc(&counters, WS_COUNTERS * sizeof(unsigned));
        if (e == hipSuccess) e = hipMemsetAsync(counters, 0, WS_COUNTERS * sizeof(unsigned), stream);
        if (e == hipSuccess) e = hipStreamSynchronize(stream);
        if (e != hipSuccess) {
            if (parts) (void)hipFree(parts);
            if (counters) (void)hipFree(counters);
            return fail(KERNELARC_ERR_LAUNCH, "split-K workspace allocation: %s", hipGetErrorString(e));
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

bool overlaps(const void *a, int64_t abytes, const void *b, int64_t bbytes) {
    if (!a || !b || abytes == 0 || bbytes == 0) return false;
    const auto pa = reinterpret_cast<uintptr_t>(a);
    const auto pb = reinterpret_cast<uintptr_t>(b);
    return pa < pb + static_cast<uintptr_t>(bbytes) && pb < pa + static_cast<uintptr_t>(abytes);
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// plan < 0: choose; otherwise run exactly that plan.
int run(int plan, int64_t M, int64_t N, int64_t K, const void *X, const void *W, const void *R,
        void *Y, bool residual, hipStream_t stream) {
    g_last_error[0] = '\0';
    if (M < 0 || N < 0 || K < 0)
        return fail(KERNELARC_ERR_INVALID_ARG, "negative size M=%lld N=%lld K=%lld", (long long)M,
                    (long long)N, (long long)K);
    if (M > LIMIT_DIM || N > LIMIT_DIM || K > LIMIT_DIM)
        return fail(KERNELARC_ERR_INVALID_ARG, "a size is 2^31 or more");
    if (plan >= PLAN_COUNT) return fail(KERNELARC_ERR_UNSUPPORTED, "unknown plan %d", plan);
    if (M == 0 || N == 0) return KERNELARC_OK;
    if (!Y) return fail(KERNELARC_ERR_INVALID_ARG, "Y is NULL");
    if (K > 0 && (!X || !W)) return fail(KERNELARC_ERR_INVALID_ARG, "X or W is NULL");
    if (residual && !R) return fail(KERNELARC_ERR_INVALID_ARG, "R is NULL");
    const int64_t ybytes = M * N * 2;
    if (overlaps(Y, ybytes, X, M * K * 2) || overlaps(Y, ybytes, W, N * K * 2))
        return fail(KERNELARC_ERR_INVALID_ARG, "Y overlaps X or W");
    if (residual && R != Y && overlaps(Y, ybytes, R, ybytes))
        return fail(KERNELARC_ERR_INVALID_ARG, "Y partially overlaps R (only Y == R is allowed)");

    int dev = 0, num_cus = 0;
    const int st = current_device(&dev, &num_cus);
    if (st != KERNELARC_OK) return st;

    const bool vec_ok = aligned16(X) && aligned16(W) && aligned16(Y) && (!residual || aligned16(R)) &&
                        K % 8 == 0;
    if (plan < 0) {
        plan = select(M, N, K, residual);
        if (plan != PLAN_GENERIC && !vec_ok) plan = PLAN_GENERIC;
    } else {
        if (!supports(plan, M, N, K, residual))
            return fail(KERNELARC_ERR_UNSUPPORTED, "plan %s cannot compute M=%lld N=%lld K=%lld",
                        PLANS[plan].name, (long long)M, (long long)N, (long long)K);
        if (plan != PLAN_GENERIC && !vec_ok)
            return fail(KERNELARC_ERR_UNSUPPORTED, "plan %s needs 16-byte aligned pointers and K %% 8 == 0",
                        PLANS[plan].name);
    }

    Problem p{M, N, K, static_cast<const uint16_t *>(X), static_cast<const uint16_t *>(W),
              residual ? static_cast<const uint16_t *>(R) : nullptr, static_cast<uint16_t *>(Y)};
    (void)hipGetLastError();   // clear any stale error before launching
    hipError_t e = hipSuccess;
    switch (plan) {
        case PLAN_GENERIC:
            e = launch_generic(p, stream);
            break;
        case PLAN_SKINNY:
        case PLAN_SKINNY_SPLITK: {
            const int split = skinny_split_of(plan, M, N, K);
            Workspace ws{};
            if (split > 1) {
                const int wst = workspace(dev, stream, &ws);
                if (wst != KERNELARC_OK) return wst;
            }
            e = launch_skinny(p, split, split > 1 ? &ws : nullptr, stream);
            break;
        }
        default:
            e = launch_tile(plan, p, num_cus, stream);
            break;
    }
    if (e != hipSuccess)
        return fail(KERNELARC_ERR_LAUNCH, "launch of %s failed: %s", PLANS[plan].name, hipGetErrorString(e));
    return KERNELARC_OK;
}

}  // namespace
}  // namespace kernelarc

using namespace kernelarc;

extern "C" {

int kernelarc_gemm_bf16_residual(int64_t M, int64_t N, int64_t K, const void *X, const void *W,
                                 const void *R, void *Y, hipStream_t stream) {
    return run(-1, M, N, K, X, W, R, Y, true, stream);
}

int kernelarc_gemm_bf16(int64_t M, int64_t N, int64_t K, const void *X, const void *W, void *Y,
                        hipStream_t stream) {
    return run(-1, M, N, K, X, W, nullptr, Y, false, stream);
}

int kernelarc_gemm_bf16_with_plan(int plan, int64_t M, int64_t N, int64_t K, const void *X,
                                  const void *W, const void *R, void *Y, hipStream_t stream) {
    if (plan < 0) {
        g_last_error[0] = '\0';
        return fail(KERNELARC_ERR_UNSUPPORTED, "unknown plan %d", plan);
    }
    return run(plan, M, N, K, X, W, R, Y, R != nullptr, stream);
}

int kernelarc_plan_count(void) { return PLAN_COUNT; }

const char *kernelarc_plan_name(int plan) {
    return (plan >= 0 && plan < PLAN_COUNT) ? PLANS[plan].name : nullptr;
}

int kernelarc_plan_supports(int plan, int64_t M, int64_t N, int64_t K, int residual) {
    if (plan < 0 || plan >= PLAN_COUNT || M < 0 || N < 0 || K < 0) return -1;
    return supports(plan, M, N, K, residual != 0) ? 1 : 0;
}

int kernelarc_select_plan(int64_t M, int64_t N, int64_t K, int residual) {
    return select(M, N, K, residual != 0);
}

int kernelarc_plan_uses_workspace(int plan, int64_t M, int64_t N, int64_t K) {
    if (plan == PLAN_SKINNY_SPLITK && supports(plan, M, N, K, true)) return 1;
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
