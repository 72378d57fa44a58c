// C ABI of the PAM library: argument validation, plan selection, workspace
// handling and launches.  The arithmetic lives in the HIP sources
// (pam_gemm_dma.hip, pam_kernels.hip, pa_ops.hip, pam_exact_grad.hip).

#include <hip/hip_runtime.h>
#include <hsa/hsa.h>
#include <hsa/hsa_ext_amd.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>

#include "pam.h"
#include "pam_internal.h"

namespace {

thread_local std::string g_last_error;

pam_status_t fail(pam_status_t s, const std::string &msg) {
    g_last_error = msg;
    return s;
}

pam_status_t fail_hip(hipError_t e, const char *what) {
    g_last_error = std::string(what) + ": " + hipGetErrorString(e);
    return PAM_ERROR_LAUNCH;
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr int64_t kMaxDim = 0x7FFFFFFF;
constexpr int64_t kMaxSplits = 64;
// 128 rows of a panel, in bytes, must fit the kernels' 32-bit offsets.
constexpr int64_t kMaxLd = (int64_t)1 << 22;

// With splits > 1, the first whole_tiles tiles (batch-major, then tile row,
// then tile column) take the whole K and the rest are split into `splits` K
// slices of k_per_split; whole_tiles == 0: every tile is split.
struct Plan {
    int tile_m, tile_n, kgroups, splits;
    int64_t k_per_split;
    int64_t whole_tiles;
};

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

struct Shape {
    int bm, bn, kw;
    int waves;      // waves per workgroup
    int per_cu;     // workgroups resident per compute unit (register budget)
    double rate;    // PAM-MACs per second with every compute unit full (fitted to MI355X runs)
};
// 128 x 128 and 128 x 64 tiles with one k-group; 128 x 64 tiles whose two
// k-groups split each chunk's k steps, and 64 x 64 tiles with one or four
// (more waves without partial sums in HBM: the groups add their partial
// tiles in LDS, at more staging work per MAC).  Resident workgroups per
// compute unit follow from the float32 kernel's registers and LDS: the
// 128 x 128 tile holds four waves per SIMD, the 128 x 64 tile with two
// k-groups three, the others two.
const Shape kShapes[] = {{128, 128, 1, 4, 4, 27.55e12},
                         {128, 64, 1, 2, 4, 23.69e12},
                         {128, 64, 2, 4, 3, 24.51e12},
                         {64, 64, 1, 1, 8, 20.31e12},
                         {64, 64, 4, 4, 2, 20.71e12}};
constexpr int kComputeUnits = 256;
constexpr int kSimdsPerCu = 4;
// Vector-ALU throughput of one SIMD holding 0..4 waves of this kernel,
// relative to four: one wave issues alone, two pair their adds and fmas
// but leave barrier and LDS waits exposed.
constexpr double kSimdEfficiency[5] = {0.0, 0.4495, 0.8693, 0.8743, 1.0};
constexpr double kWorkgroupFixedS = 3.15e-6;  // first loads, epilogue stores
constexpr double kSplitFixedS = 12.7e-6;      // second launch, workspace
// Effective rate of writing and re-reading partial sums: up to a few hundred
// MB they largely stay in the last-level cache, so above the HBM rate.
constexpr double kPartialBytesPerS = 24.7e12;
// Workgroups start as soon as slots free up, so a partial last round costs
// less than a full one the more rounds precede it (they end staggered).
constexpr double kTailDamping = 0.925;
// Compute units run at different clocks under load, so the last round of
// workgroups does not end at once: the launch ends a fraction of the last
// workgroups' duration after the average, scaled by how many slots the last
// round leaves without a shorter partial-round workgroup to absorb it.  A
// round that started together (the first) ends closer together than one
// whose workgroups started staggered behind earlier rounds.
constexpr double kRoundImbalance = 0.0408;
constexpr double kStaggeredImbalance = 0.1415;
// Split-K plans must beat the best unsplit plan by this factor (they change
// the summation order and take a workspace).
constexpr double kSplitMargin = 0.98;
// Plans with whole-K tiles beside split ones run in one launch; the planner
// offers them up to this many tiles.
constexpr int64_t kMaxHybridTiles = 1 << 20;
// Shortest K for which one full round of whole-K 128 x 128 tiles is replaced
// by the quarter-round hybrid plan (choose_plan).
constexpr int64_t kOneRoundHybridMinK = 512;
// Split counts the plan search considers.
constexpr int kSplitChoices[] = {1, 2, 3, 4, 5, 6, 7, 8, 12, 16, 24, 32, 48, 56, 64};

double cu_efficiency(int waves_per_cu) {
    const int base = waves_per_cu / kSimdsPerCu;
    const int extra = waves_per_cu % kSimdsPerCu;
    return (extra * kSimdEfficiency[std::min(base + 1, 4)] + (kSimdsPerCu - extra) * kSimdEfficiency[std::min(base, 4)]) /
           kSimdsPerCu;
}

Plan make_plan(const Shape &c, int64_t k, int64_t splits, int64_t whole_tiles = 0) {
    Plan p{c.bm, c.bn, c.kw, 1, k, 0};
    if (splits > 1) {
        const int64_t per = ceil_div(ceil_div(k, splits), pamk::kChunkK * c.kw) * pamk::kChunkK * c.kw;
        p.k_per_split = per;
        p.splits = (int)ceil_div(k, per);
        p.whole_tiles = p.splits > 1 ? whole_tiles : 0;
    }
    return p;
}

// Time of `wgs` workgroups of wg_s seconds each, dispatched after `before`
// full rounds of others: full rounds at the shape's rate, then a partial
// round whose workgroups share compute units with fewer others (faster each,
// slower in total), then the uneven end of the last round.
double rounds_time(const Shape &c, int64_t wgs, double wg_s, int64_t before) {
    const int64_t slots = (int64_t)c.per_cu * kComputeUnits;
    const int64_t rounds = wgs / slots;
    const int64_t rest = wgs % slots;
    double t = double(rounds) * wg_s;
    if (rest > 0) {
        const int q = (int)ceil_div(rest, kComputeUnits);
        const double partial = wg_s * (double(q) / c.per_cu) * cu_efficiency(c.per_cu * c.waves) /
                               cu_efficiency(q * c.waves);
        const double even = wg_s * double(rest) / double(slots);
        t += even + (partial - even) / (1.0 + kTailDamping * double(before + rounds));
    }
    if (before + rounds > 0) {
        const bool staggered = before + rounds + (rest > 0 ? 1 : 0) > 1;
        t += (staggered ? kStaggeredImbalance : kRoundImbalance) * wg_s * (1.0 - double(rest) / double(slots));
    }
    return t;
}

// Estimated time of a plan: the whole-K tiles' full rounds, then the K
// slices of the split tiles together with the whole-K tiles of a partial
// round (counted as the slices they displace), plus for split-K a second
// launch and the partial sums' round trip through memory.
double plan_time(const Shape &c, const Plan &p, int64_t m, int64_t n, int64_t k, int64_t batch) {
    const int64_t bk = pamk::kChunkK * c.kw;
    const int64_t slots = (int64_t)c.per_cu * kComputeUnits;
    const int64_t tiles = ceil_div(m, c.bm) * ceil_div(n, c.bn) * batch;
    const double per_chunk = double(c.bm) * c.bn * bk * slots / c.rate;
    const double wg_whole = per_chunk * double(ceil_div(k, bk)) + kWorkgroupFixedS;
    if (p.splits <= 1)
        return rounds_time(c, tiles, wg_whole, 0);
    const int64_t whole = std::min(p.whole_tiles, tiles);
    const int64_t split_tiles = tiles - whole;
    const int64_t before = whole / slots;
    const int64_t rem = whole % slots;
    const double wg_slice = per_chunk * double(ceil_div(p.k_per_split, bk)) + kWorkgroupFixedS;
    const int64_t displaced = rem > 0 ? (int64_t)std::ceil(double(rem) * wg_whole / wg_slice) : 0;
    double t = double(before) * wg_whole + rounds_time(c, split_tiles * p.splits + displaced, wg_slice, before);
    t += kSplitFixedS + double(p.splits + 1) * double(split_tiles) * c.bm * c.bn * 4.0 / kPartialBytesPerS;
    return t;
}

// How a plan's work items are launched: whole-K tiles, then `splits` slices
// of each split tile.  A plan with whole-K tiles beside split ones runs as
// one launch; otherwise launches take as many whole matrices as fit.
struct Layout {
    int64_t tiles;        // per matrix
    int64_t total;        // tiles of the whole batch
    int64_t splits;       // K slices of a split tile (1: none)
    int64_t whole_tiles;  // > 0: a hybrid plan
    int64_t per_launch;   // matrices per launch
    int64_t ws_tiles;     // split tiles the workspace holds at once
    size_t ws_bytes;
};

// The layout of a plan, or false (with the reason in *why) when its
// workgroups do not fit the launch limits.
bool layout_quiet(const Plan &plan, int64_t m, int64_t n, int64_t batch, Layout *out, const char **why) {
    Layout L{};
    L.tiles = ceil_div(m, plan.tile_m) * ceil_div(n, plan.tile_n);
    if (L.tiles > kMaxDim || batch > kMaxDim * kMaxDim / L.tiles) {
        *why = "too many output tiles (m, n or batch too large)";
        return false;
    }
    L.total = L.tiles * batch;
    L.splits = plan.splits > 1 ? plan.splits : 1;
    if (plan.whole_tiles >= L.total)
        L.splits = 1;
    L.whole_tiles = L.splits > 1 ? plan.whole_tiles : 0;
    const bool hybrid = L.whole_tiles > 0;
    if (L.tiles * L.splits > pamk::kMaxLaunchItems ||
        (hybrid && L.whole_tiles + (L.total - L.whole_tiles) * L.splits > pamk::kMaxLaunchItems)) {
        *why = "too many workgroups for one launch (output too large for the plan)";
        return false;
    }
    L.per_launch = hybrid ? batch : std::max<int64_t>(1, pamk::kMaxLaunchItems / (L.tiles * L.splits));
    L.ws_tiles = hybrid ? L.total - L.whole_tiles : (L.splits > 1 ? std::min(batch, L.per_launch) * L.tiles : 0);
    L.ws_bytes = (size_t)L.splits * (size_t)L.ws_tiles * (size_t)plan.tile_m * (size_t)plan.tile_n * sizeof(float);
    if (L.ws_tiles == 0)
        L.ws_bytes = 0;
    *out = L;
    return true;
}

pam_status_t layout_of(const Plan &plan, int64_t m, int64_t n, int64_t batch, Layout *out) {
    const char *why = "";
    if (!layout_quiet(plan, m, n, batch, out, &why))
        return fail(PAM_ERROR_INVALID_VALUE, why);
    return PAM_SUCCESS;
}

// No limit on the split-K workspace: the caller provides it.
constexpr size_t kAnyWorkspace = ~(size_t)0;

// The cheapest plan by plan_time whose split-K partial sums fit in
// max_ws_bytes (0: no split-K): for each tile shape every split count
// (slices of at least four chunks), and, for the one-k-group tiles, hybrid
// plans that split only the last tiles (those of a partial last round, of
// the last round and that one, or a quarter or half of a round's slots)
// while the rest take the whole K.  A hybrid's slices are short, at least
// four per tile and about one per 20 chunks up to 16: the launch then ends
// on short workgroups (measured: fewer, longer slices end later than the
// model's imbalance term predicts).  A plan with split-K must beat the best
// unsplit one by kSplitMargin.
Plan choose_plan(int64_t m, int64_t n, int64_t k, int64_t batch, size_t max_ws_bytes) {
    double best_t[2] = {0.0, 0.0};
    Plan best[2] = {};
    bool have[2] = {false, false};
    auto consider = [&](const Shape &c, const Plan &p) {
        const int split = p.splits > 1 ? 1 : 0;
        if (split) {
            Layout L;
            const char *why;
            if (!layout_quiet(p, m, n, batch, &L, &why) || L.ws_bytes > max_ws_bytes)
                return;
        }
        const double t = plan_time(c, p, m, n, k, batch);
        if (!have[split] || t < best_t[split]) {
            best_t[split] = t;
            best[split] = p;
            have[split] = true;
        }
    };
    for (const auto &c : kShapes) {
        const int64_t most = max_ws_bytes == 0 ? 1 : std::max<int64_t>(1, std::min(kMaxSplits, k / (4 * pamk::kChunkK * c.kw)));
        const int64_t slots = (int64_t)c.per_cu * kComputeUnits;
        const int64_t tiles = ceil_div(m, c.bm) * ceil_div(n, c.bn) * batch;
        const int64_t rest = tiles % slots;
        const int64_t hybrid_min = std::max<int64_t>(4, std::min<int64_t>(16, ceil_div(k, pamk::kChunkK) / 20));
        for (const int s : kSplitChoices) {
            if (s > most)
                break;
            consider(c, make_plan(c, k, s));
            if (s < hybrid_min || c.kw != 1 || tiles > kMaxHybridTiles)
                continue;
            const int64_t tails[4] = {rest, rest + slots, slots / 4, slots / 2};
            for (int i = 0; i < 4; ++i) {
                bool seen = false;
                for (int j = 0; j < i; ++j)
                    seen = seen || tails[j] == tails[i];
                if (!seen && tails[i] > 0 && tails[i] < tiles)
                    consider(c, make_plan(c, k, s, tiles - tails[i]));
            }
        }
    }
    if (have[1] && best_t[1] < kSplitMargin * best_t[0])
        return best[1];
    // One full round of whole-K 128 x 128 tiles ends when the slowest compute
    // unit does; whole-K tiles in three quarters of the slots beside the last
    // quarter's tiles in K slices let the faster units take more of the
    // slices.  Measured against the single round (1024 tiles, interleaved):
    // K = 512 2-3%, 768 4%, 1024 5%, 2048 8-9% faster; K = 256 3% slower.
    // The cost model above does not see it (its end-of-round term would
    // then misjudge other plans), so the plan is taken as measured.
    const Shape &big = kShapes[0];
    const int64_t big_slots = (int64_t)big.per_cu * kComputeUnits;
    if (best[0].tile_m == big.bm && best[0].tile_n == big.bn && best[0].kgroups == 1 &&
        ceil_div(m, big.bm) * ceil_div(n, big.bn) * batch == big_slots && k >= kOneRoundHybridMinK) {
        const int64_t slices = std::max<int64_t>(4, std::min<int64_t>(16, ceil_div(k, pamk::kChunkK) / 20));
        const Plan h = make_plan(big, k, slices, big_slots - big_slots / 4);
        Layout L;
        const char *why;
        if (h.splits > 1 && layout_quiet(h, m, n, batch, &L, &why) && L.ws_bytes <= max_ws_bytes)
            return h;
    }
    return best[0];
}

// Output tiles of the smallest tile shape over the whole batch, at most
// 2^40 (petabytes of output): the plan and launch arithmetic on tile counts
// (times split counts and slots) then stays far inside int64.
pam_status_t check_output_size(int64_t m, int64_t n, int64_t batch) {
    const int64_t tiles = ceil_div(std::max<int64_t>(m, 1), 64) * ceil_div(std::max<int64_t>(n, 1), 64);
    if (batch > 0 && tiles > ((int64_t)1 << 40) / batch)
        return fail(PAM_ERROR_INVALID_VALUE, "too many output tiles (m * n * batch too large)");
    return PAM_SUCCESS;
}

pam_status_t validate(pam_op_t ta, pam_op_t tb, int64_t m, int64_t n, int64_t k, const float *A, int64_t lda,
                      int64_t sa, const float *B, int64_t ldb, int64_t sb, const float *C, int64_t ldc, int64_t sc,
                      int64_t batch) {
    char buf[256];
    if ((ta != PAM_OP_N && ta != PAM_OP_T) || (tb != PAM_OP_N && tb != PAM_OP_T))
        return fail(PAM_ERROR_INVALID_VALUE, "transA/transB must be PAM_OP_N or PAM_OP_T");
    if (m < 0 || n < 0 || k < 0 || batch < 0) {
        snprintf(buf, sizeof buf, "negative size (m=%lld n=%lld k=%lld batch=%lld)", (long long)m, (long long)n,
                 (long long)k, (long long)batch);
        return fail(PAM_ERROR_INVALID_VALUE, buf);
    }
    if (m > kMaxDim || n > kMaxDim || k > kMaxDim)
        return fail(PAM_ERROR_INVALID_VALUE, "m, n and k must be below 2^31");
    if (check_output_size(m, n, batch) != PAM_SUCCESS)
        return PAM_ERROR_INVALID_VALUE;
    if (sa < 0 || sb < 0 || sc < 0)
        return fail(PAM_ERROR_INVALID_VALUE, "batch strides must be >= 0");
    if (lda >= kMaxLd || ldb >= kMaxLd)
        return fail(PAM_ERROR_NOT_SUPPORTED, "lda and ldb must be below 2^22 (per-thread 32-bit offsets)");
    const int64_t min_lda = std::max<int64_t>(1, ta == PAM_OP_N ? k : m);
    const int64_t min_ldb = std::max<int64_t>(1, tb == PAM_OP_N ? n : k);
    const int64_t min_ldc = std::max<int64_t>(1, n);
    if (lda < min_lda || ldb < min_ldb || ldc < min_ldc) {
        snprintf(buf, sizeof buf, "leading dimension too small (lda=%lld>=%lld ldb=%lld>=%lld ldc=%lld>=%lld)",
                 (long long)lda, (long long)min_lda, (long long)ldb, (long long)min_ldb, (long long)ldc,
                 (long long)min_ldc);
        return fail(PAM_ERROR_INVALID_VALUE, buf);
    }
    if (batch > 0) {
        if (m * k > 0 && A == nullptr)
            return fail(PAM_ERROR_INVALID_VALUE, "A is NULL");
        if (k * n > 0 && B == nullptr)
            return fail(PAM_ERROR_INVALID_VALUE, "B is NULL");
        if (m * n > 0 && C == nullptr)
            return fail(PAM_ERROR_INVALID_VALUE, "C is NULL");
    }
    return PAM_SUCCESS;
}

pam_status_t check_device() {
    static thread_local int checked_device = -1;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return fail_hip(e, "hipGetDevice");
    if (dev == checked_device)
        return PAM_SUCCESS;
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess)
        return fail_hip(e, "hipGetDeviceProperties");
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return fail(PAM_ERROR_NOT_SUPPORTED, std::string("device is ") + prop.gcnArchName + ", library built for gfx950");
    checked_device = dev;
    return PAM_SUCCESS;
}

// A caller-provided workspace (pointer and size), or none (then the plan
// does not split K).
struct Workspace {
    void *ptr;
    size_t bytes;
};

pam_status_t check_workspace(const Workspace *ws, size_t need) {
    if (need == 0)
        return PAM_SUCCESS;
    char buf[160];
    if (ws == nullptr || ws->bytes < need) {
        snprintf(buf, sizeof buf, "workspace of %zu bytes is smaller than the %zu this product's plan needs",
                 ws == nullptr ? (size_t)0 : ws->bytes, need);
        return fail(PAM_ERROR_INVALID_VALUE, buf);
    }
    if (ws->ptr == nullptr)
        return fail(PAM_ERROR_INVALID_VALUE, "workspace is NULL");
    if ((reinterpret_cast<uintptr_t>(ws->ptr) & 15u) != 0)
        return fail(PAM_ERROR_INVALID_VALUE, "workspace must be 16-byte aligned");
    return PAM_SUCCESS;
}

// The product under `plan`; a split plan keeps its partial sums in `ext`,
// which must hold the plan's workspace bytes.  Allocates nothing.
pam_status_t run_gemm(pam_op_t ta, pam_op_t tb, int64_t m, int64_t n, int64_t k, const float *A, int64_t lda,
                      int64_t sa, const float *B, int64_t ldb, int64_t sb, float *C, int64_t ldc, int64_t sc,
                      int64_t batch, const Plan &plan, hipStream_t stream, int round_drop = 0,
                      const Workspace *ext = nullptr, bool bf16 = false) {
    if (m == 0 || n == 0 || batch == 0)
        return PAM_SUCCESS;
    Layout L{};
    if (k > 0) {
        pam_status_t st = layout_of(plan, m, n, batch, &L);
        if (st != PAM_SUCCESS)
            return st;
        st = check_workspace(ext, L.ws_bytes);
        if (st != PAM_SUCCESS)
            return st;
    }
    pam_status_t st = check_device();
    if (st != PAM_SUCCESS)
        return st;
    if (k == 0) {
        hipError_t e = pamk::launch_fill_zero(C, (int32_t)m, (int32_t)n, ldc, sc, batch, stream);
        return e == hipSuccess ? PAM_SUCCESS : fail_hip(e, "fill kernel launch");
    }

    pamk::GemmParams p{};
    p.lda = lda;
    p.ldb = ldb;
    p.ldc = ldc;
    p.strideA = sa;
    p.strideB = sb;
    p.strideC = sc;
    p.m = (int32_t)m;
    p.n = (int32_t)n;
    p.k = (int32_t)k;
    p.k_per_split = (int32_t)std::min<int64_t>(plan.k_per_split, kMaxDim);
    p.tiles_n = (int32_t)ceil_div(n, plan.tile_n);
    // Operand copies of 16 bytes: four float32 or eight bfloat16 elements.
    const int64_t per16 = bf16 ? 8 : 4;
    p.vec_a = aligned16(A) && lda % per16 == 0 && (batch == 1 || sa % per16 == 0);
    p.vec_b = aligned16(B) && ldb % per16 == 0 && (batch == 1 || sb % per16 == 0);
    p.vec_c = aligned16(C) && ldc % 4 == 0 && (batch == 1 || sc % 4 == 0);
    p.round_drop = round_drop;
    p.tiles = (int32_t)L.tiles;
    p.splits = (int32_t)L.splits;
    float *ws = L.ws_bytes > 0 ? static_cast<float *>(ext->ptr) : nullptr;

    for (int64_t b0 = 0; b0 < batch; b0 += L.per_launch) {
        const int64_t nb = std::min(L.per_launch, batch - b0);
        const size_t es = bf16 ? 2 : 4;   // operand element bytes
        p.A = reinterpret_cast<const float *>(reinterpret_cast<const char *>(A) + (size_t)(b0 * sa) * es);
        p.B = reinterpret_cast<const float *>(reinterpret_cast<const char *>(B) + (size_t)(b0 * sb) * es);
        p.C = C + b0 * sc;
        p.W = ws;
        if (L.whole_tiles > 0) {
            p.whole = (int32_t)L.whole_tiles;
            p.split_tiles = (int32_t)(L.total - L.whole_tiles);
        } else if (L.splits > 1) {
            p.whole = 0;
            p.split_tiles = (int32_t)(nb * L.tiles);
        } else {
            p.whole = (int32_t)(nb * L.tiles);
            p.split_tiles = 0;
        }
        hipError_t e = pamk::launch_pam_gemm(plan.tile_m, plan.tile_n, plan.kgroups, ta == PAM_OP_T, tb == PAM_OP_T,
                                             bf16, p, stream);
        if (e != hipSuccess)
            return fail_hip(e, "gemm kernel launch");
        if (p.split_tiles > 0) {
            e = pamk::launch_split_tile_reduce(plan.tile_m, plan.tile_n, p, stream);
            if (e != hipSuccess)
                return fail_hip(e, "split-K reduce launch");
        }
    }
    return PAM_SUCCESS;
}

int query_simds_per_cu(int device) {
    // HSA agent enumeration order matches HIP device order for GPU agents.
    struct Ctx {
        int want, seen, simds;
    } ctx{device, 0, 0};
    if (hsa_init() != HSA_STATUS_SUCCESS)
        return 0;
    hsa_iterate_agents(
        [](hsa_agent_t agent, void *data) -> hsa_status_t {
            auto *c = static_cast<Ctx *>(data);
            hsa_device_type_t type;
            if (hsa_agent_get_info(agent, HSA_AGENT_INFO_DEVICE, &type) != HSA_STATUS_SUCCESS)
                return HSA_STATUS_SUCCESS;
            if (type != HSA_DEVICE_TYPE_GPU)
                return HSA_STATUS_SUCCESS;
            if (c->seen++ == c->want) {
                uint32_t v = 0;
                if (hsa_agent_get_info(agent, (hsa_agent_info_t)HSA_AMD_AGENT_INFO_NUM_SIMDS_PER_CU, &v) ==
                    HSA_STATUS_SUCCESS)
                    c->simds = (int)v;
                return HSA_STATUS_INFO_BREAK;
            }
            return HSA_STATUS_SUCCESS;
        },
        &ctx);
    hsa_shut_down();
    return ctx.simds;
}

// Exact-derivative products: 128 x 128 tiles, two workgroups per compute
// unit; K is split while the tiles would not fill two rounds and each slice
// keeps >= 4 chunks.  Partial sums [split][m][n].
int64_t exact_grad_splits(int64_t m, int64_t n, int64_t k) {
    const int64_t tiles = ceil_div(m, 128) * ceil_div(n, 128);
    int64_t splits = 1;
    while (tiles * splits < 4 * kComputeUnits && splits < kMaxSplits && k / (splits * 2) >= 4 * pamk::kChunkK)
        splits *= 2;
    return splits;
}

size_t exact_grad_workspace(int64_t m, int64_t n, int64_t k, int64_t *splits_out, int64_t *per_out) {
    const int64_t splits = exact_grad_splits(m, n, k);
    const int64_t per = ceil_div(ceil_div(k, splits), pamk::kChunkK) * pamk::kChunkK;
    const int64_t used = ceil_div(k, per);
    *splits_out = used;
    *per_out = per;
    return used > 1 ? (size_t)used * (size_t)m * (size_t)n * sizeof(float) : 0;
}

// ext == nullptr: one K slice (no workspace); otherwise the split plan, its
// partial sums in *ext.
pam_status_t run_exact_grad(pam_op_t transA, int64_t m, int64_t n, int64_t k, const float *A, int64_t lda,
                            const float *B, int64_t ldb, const float *Mod, int64_t ldm, float *C, int64_t ldc,
                            hipStream_t stream, const Workspace *ext) {
    pam_status_t st = validate(transA, PAM_OP_N, m, n, k, A, lda, 0, B, ldb, 0, C, ldc, 0, 1);
    if (st != PAM_SUCCESS)
        return st;
    if (ldm < std::max<int64_t>(1, n))
        return fail(PAM_ERROR_INVALID_VALUE, "ldm must be >= max(1, n)");
    if (m == 0 || n == 0)
        return PAM_SUCCESS;
    if (Mod == nullptr)
        return fail(PAM_ERROR_INVALID_VALUE, "Mod is NULL");
    int64_t splits = 1, per = std::max<int64_t>(k, 1);
    size_t need = 0;
    if (k > 0 && ext != nullptr)
        need = exact_grad_workspace(m, n, k, &splits, &per);
    st = check_workspace(ext, need);
    if (st != PAM_SUCCESS)
        return st;
    st = check_device();
    if (st != PAM_SUCCESS)
        return st;
    if (k == 0) {
        hipError_t e = pamk::launch_fill_zero(C, (int32_t)m, (int32_t)n, ldc, 0, 1, stream);
        return e == hipSuccess ? PAM_SUCCESS : fail_hip(e, "fill kernel launch");
    }
    pamk::GemmParams p{};
    p.A = A;
    p.B = B;
    p.Mod = Mod;
    p.lda = lda;
    p.ldb = ldb;
    p.ldm = ldm;
    p.ldc = ldc;
    p.m = (int32_t)m;
    p.n = (int32_t)n;
    p.k = (int32_t)k;
    p.k_per_split = (int32_t)std::min<int64_t>(per, kMaxDim);
    p.splits = (int32_t)splits;
    p.tiles_n = (int32_t)ceil_div(n, 128);
    p.vec_a = aligned16(A) && lda % 4 == 0;
    p.vec_b = aligned16(B) && ldb % 4 == 0;
    float *ws = need > 0 ? static_cast<float *>(ext->ptr) : nullptr;
    p.C = C;
    p.W = ws;
    hipError_t e = pamk::launch_pam_exact_grad(transA == PAM_OP_T, p, stream);
    if (e != hipSuccess)
        return fail_hip(e, "exact-derivative kernel launch");
    if (ws) {
        e = pamk::launch_splitk_reduce(ws, C, (int32_t)m, (int32_t)n, ldc, 0, p.splits, 1, stream);
        if (e != hipSuccess)
            return fail_hip(e, "split-K reduce launch");
    }
    return PAM_SUCCESS;
}

}  // namespace

extern "C" {

pam_status_t pam_mul(const float *a, const float *b, float *out, int64_t n, hipStream_t stream) {
    if (n < 0)
        return fail(PAM_ERROR_INVALID_VALUE, "n must be >= 0");
    if (n == 0)
        return PAM_SUCCESS;
    if (a == nullptr || b == nullptr || out == nullptr)
        return fail(PAM_ERROR_INVALID_VALUE, "a, b and out must be non-NULL");
    pam_status_t st = check_device();
    if (st != PAM_SUCCESS)
        return st;
    hipError_t e = pamk::launch_pam_mul(a, b, out, n, stream);
    if (e != hipSuccess)
        return fail_hip(e, "pam_mul kernel launch");
    return PAM_SUCCESS;
}

pam_status_t pam_pad(const float *a, const float *b, float *out, int64_t n, hipStream_t stream) {
    if (n < 0)
        return fail(PAM_ERROR_INVALID_VALUE, "n must be >= 0");
    if (n == 0)
        return PAM_SUCCESS;
    if (a == nullptr || b == nullptr || out == nullptr)
        return fail(PAM_ERROR_INVALID_VALUE, "a, b and out must be non-NULL");
    pam_status_t st = check_device();
    if (st != PAM_SUCCESS)
        return st;
    hipError_t e = pamk::launch_pad(a, b, out, n, stream);
    if (e != hipSuccess)
        return fail_hip(e, "pam_pad kernel launch");
    return PAM_SUCCESS;
}

pam_status_t pam_palog2(const float *a, float *out, int64_t n, hipStream_t stream) {
    if (n < 0)
        return fail(PAM_ERROR_INVALID_VALUE, "n must be >= 0");
    if (n == 0)
        return PAM_SUCCESS;
    if (a == nullptr || out == nullptr)
        return fail(PAM_ERROR_INVALID_VALUE, "a and out must be non-NULL");
    pam_status_t st = check_device();
    if (st != PAM_SUCCESS)
        return st;
    hipError_t e = pamk::launch_palog2(a, out, n, stream);
    if (e != hipSuccess)
        return fail_hip(e, "pam_palog2 kernel launch");
    return PAM_SUCCESS;
}

pam_status_t pam_paexp2(const float *a, float *out, int64_t n, hipStream_t stream) {
    if (n < 0)
        return fail(PAM_ERROR_INVALID_VALUE, "n must be >= 0");
    if (n == 0)
        return PAM_SUCCESS;
    if (a == nullptr || out == nullptr)
        return fail(PAM_ERROR_INVALID_VALUE, "a and out must be non-NULL");
    pam_status_t st = check_device();
    if (st != PAM_SUCCESS)
        return st;
    hipError_t e = pamk::launch_paexp2(a, out, n, stream);
    if (e != hipSuccess)
        return fail_hip(e, "pam_paexp2 kernel launch");
    return PAM_SUCCESS;
}

pam_status_t pam_gemm(pam_op_t transA, pam_op_t transB, int64_t m, int64_t n, int64_t k, const float *A, int64_t lda,
                      const float *B, int64_t ldb, float *C, int64_t ldc, hipStream_t stream) {
    pam_status_t st = validate(transA, transB, m, n, k, A, lda, 0, B, ldb, 0, C, ldc, 0, 1);
    if (st != PAM_SUCCESS)
        return st;
    if (m == 0 || n == 0)
        return PAM_SUCCESS;
    return run_gemm(transA, transB, m, n, k, A, lda, 0, B, ldb, 0, C, ldc, 0, 1, choose_plan(m, n, k, 1, 0), stream);
}

pam_status_t pam_gemm_batched(pam_op_t transA, pam_op_t transB, int64_t m, int64_t n, int64_t k, const float *A,
                              int64_t lda, int64_t strideA, const float *B, int64_t ldb, int64_t strideB, float *C,
                              int64_t ldc, int64_t strideC, int64_t batch, hipStream_t stream) {
    pam_status_t st = validate(transA, transB, m, n, k, A, lda, strideA, B, ldb, strideB, C, ldc, strideC, batch);
    if (st != PAM_SUCCESS)
        return st;
    if (m == 0 || n == 0 || batch == 0)
        return PAM_SUCCESS;
    return run_gemm(transA, transB, m, n, k, A, lda, strideA, B, ldb, strideB, C, ldc, strideC, batch,
                    choose_plan(m, n, k, batch, 0), stream);
}

pam_status_t pam_gemm_narrow(pam_op_t transA, pam_op_t transB, int64_t m, int64_t n, int64_t k, const float *A,
                             int64_t lda, int64_t strideA, const float *B, int64_t ldb, int64_t strideB, float *C,
                             int64_t ldc, int64_t strideC, int64_t batch, int32_t mantissa_bits,
                             hipStream_t stream) {
    if (mantissa_bits < 0 || mantissa_bits > 23)
        return fail(PAM_ERROR_INVALID_VALUE, "mantissa_bits must be in [0, 23]");
    pam_status_t st = validate(transA, transB, m, n, k, A, lda, strideA, B, ldb, strideB, C, ldc, strideC, batch);
    if (st != PAM_SUCCESS)
        return st;
    if (m == 0 || n == 0 || batch == 0)
        return PAM_SUCCESS;
    return run_gemm(transA, transB, m, n, k, A, lda, strideA, B, ldb, strideB, C, ldc, strideC, batch,
                    choose_plan(m, n, k, batch, 0), stream, 23 - mantissa_bits);
}

pam_status_t pam_gemm_batched_noalloc(pam_op_t transA, pam_op_t transB, int64_t m, int64_t n, int64_t k,
                                      const float *A, int64_t lda, int64_t strideA, const float *B, int64_t ldb,
                                      int64_t strideB, float *C, int64_t ldc, int64_t strideC, int64_t batch,
                                      int32_t mantissa_bits, hipStream_t stream) {
    if (mantissa_bits < 0 || mantissa_bits > 23)
        return fail(PAM_ERROR_INVALID_VALUE, "mantissa_bits must be in [0, 23]");
    pam_status_t st = validate(transA, transB, m, n, k, A, lda, strideA, B, ldb, strideB, C, ldc, strideC, batch);
    if (st != PAM_SUCCESS)
        return st;
    if (m == 0 || n == 0 || batch == 0)
        return PAM_SUCCESS;
    const Plan plan = choose_plan(m, n, std::max<int64_t>(k, 1), batch, pamk::kScratchBytes);
    Layout L{};
    if (k > 0) {
        st = layout_of(plan, m, n, batch, &L);
        if (st != PAM_SUCCESS)
            return st;
        if (L.ws_bytes > pamk::kScratchBytes) {
            char buf[160];
            snprintf(buf, sizeof buf, "split-K partial sums of %zu bytes exceed the %zu-byte static scratch",
                     L.ws_bytes, pamk::kScratchBytes);
            return fail(PAM_ERROR_INVALID_VALUE, buf);
        }
    }
    st = check_device();
    if (st != PAM_SUCCESS)
        return st;
    void *scratch = nullptr;
    if (L.ws_bytes > 0) {
        const hipError_t e = pamk::scratch_address(&scratch);
        if (e != hipSuccess)
            return fail_hip(e, "hipGetSymbolAddress of the static scratch");
    }
    const Workspace ws{scratch, pamk::kScratchBytes};
    return run_gemm(transA, transB, m, n, k, A, lda, strideA, B, ldb, strideB, C, ldc, strideC, batch, plan, stream,
                    23 - mantissa_bits, &ws);
}

pam_status_t pam_gemm_workspace_size(int64_t m, int64_t n, int64_t k, int64_t batch, size_t *bytes) {
    if (bytes == nullptr)
        return fail(PAM_ERROR_INVALID_VALUE, "bytes is NULL");
    *bytes = 0;
    if (m < 0 || n < 0 || k < 0 || batch < 0)
        return fail(PAM_ERROR_INVALID_VALUE, "m, n, k and batch must be >= 0");
    if (m > kMaxDim || n > kMaxDim || k > kMaxDim)
        return fail(PAM_ERROR_INVALID_VALUE, "m, n and k must be below 2^31");
    if (check_output_size(m, n, batch) != PAM_SUCCESS)
        return PAM_ERROR_INVALID_VALUE;
    if (m == 0 || n == 0 || k == 0 || batch == 0)
        return PAM_SUCCESS;
    Layout L;
    const pam_status_t st = layout_of(choose_plan(m, n, k, batch, kAnyWorkspace), m, n, batch, &L);
    if (st != PAM_SUCCESS)
        return st;
    *bytes = L.ws_bytes;
    return PAM_SUCCESS;
}

pam_status_t pam_gemm_batched_ws(pam_op_t transA, pam_op_t transB, int64_t m, int64_t n, int64_t k,
                                 const float *A, int64_t lda, int64_t strideA, const float *B, int64_t ldb,
                                 int64_t strideB, float *C, int64_t ldc, int64_t strideC, int64_t batch,
                                 int32_t mantissa_bits, void *workspace, size_t workspace_bytes,
                                 hipStream_t stream) {
    if (mantissa_bits < 0 || mantissa_bits > 23)
        return fail(PAM_ERROR_INVALID_VALUE, "mantissa_bits must be in [0, 23]");
    pam_status_t st = validate(transA, transB, m, n, k, A, lda, strideA, B, ldb, strideB, C, ldc, strideC, batch);
    if (st != PAM_SUCCESS)
        return st;
    if (m == 0 || n == 0 || batch == 0)
        return PAM_SUCCESS;
    const Workspace ws{workspace, workspace_bytes};
    return run_gemm(transA, transB, m, n, k, A, lda, strideA, B, ldb, strideB, C, ldc, strideC, batch,
                    choose_plan(m, n, k, batch, kAnyWorkspace), stream, 23 - mantissa_bits, &ws);
}

pam_status_t pam_gemm_batched_bf16(pam_op_t transA, pam_op_t transB, int64_t m, int64_t n, int64_t k,
                                   const uint16_t *A, int64_t lda, int64_t strideA, const uint16_t *B, int64_t ldb,
                                   int64_t strideB, float *C, int64_t ldc, int64_t strideC, int64_t batch,
                                   void *workspace, size_t workspace_bytes, hipStream_t stream) {
    const float *a = reinterpret_cast<const float *>(A);
    const float *b = reinterpret_cast<const float *>(B);
    pam_status_t st = validate(transA, transB, m, n, k, a, lda, strideA, b, ldb, strideB, C, ldc, strideC, batch);
    if (st != PAM_SUCCESS)
        return st;
    if (m == 0 || n == 0 || batch == 0)
        return PAM_SUCCESS;
    const Workspace ws{workspace, workspace_bytes};
    return run_gemm(transA, transB, m, n, k, a, lda, strideA, b, ldb, strideB, C, ldc, strideC, batch,
                    choose_plan(m, n, k, batch, workspace != nullptr ? kAnyWorkspace : 0), stream, 0,
                    workspace != nullptr ? &ws : nullptr, true);
}

pam_status_t pam_round_mantissa(const float *a, float *out, int64_t n, int32_t mantissa_bits, hipStream_t stream) {
    if (mantissa_bits < 0 || mantissa_bits > 23)
        return fail(PAM_ERROR_INVALID_VALUE, "mantissa_bits must be in [0, 23]");
    if (n < 0)
        return fail(PAM_ERROR_INVALID_VALUE, "n must be >= 0");
    if (n == 0)
        return PAM_SUCCESS;
    if (a == nullptr || out == nullptr)
        return fail(PAM_ERROR_INVALID_VALUE, "a and out must be non-NULL");
    pam_status_t st = check_device();
    if (st != PAM_SUCCESS)
        return st;
    hipError_t e;
    if (mantissa_bits == 23)
        e = (a == out) ? hipSuccess
                       : hipMemcpyAsync(out, a, (size_t)n * sizeof(float), hipMemcpyDeviceToDevice, stream);
    else
        e = pamk::launch_round_mantissa(a, out, n, 23 - mantissa_bits, stream);
    if (e != hipSuccess)
        return fail_hip(e, "pam_round_mantissa launch");
    return PAM_SUCCESS;
}

pam_status_t pam_gemm_exact_grad(pam_op_t transA, int64_t m, int64_t n, int64_t k, const float *A, int64_t lda,
                                 const float *B, int64_t ldb, const float *Mod, int64_t ldm, float *C, int64_t ldc,
                                 hipStream_t stream) {
    return run_exact_grad(transA, m, n, k, A, lda, B, ldb, Mod, ldm, C, ldc, stream, nullptr);
}

pam_status_t pam_gemm_exact_grad_workspace_size(int64_t m, int64_t n, int64_t k, size_t *bytes) {
    if (bytes == nullptr)
        return fail(PAM_ERROR_INVALID_VALUE, "bytes is NULL");
    *bytes = 0;
    if (m < 0 || n < 0 || k < 0)
        return fail(PAM_ERROR_INVALID_VALUE, "m, n and k must be >= 0");
    if (m > kMaxDim || n > kMaxDim || k > kMaxDim)
        return fail(PAM_ERROR_INVALID_VALUE, "m, n and k must be below 2^31");
    if (m == 0 || n == 0 || k == 0)
        return PAM_SUCCESS;
    int64_t splits, per;
    *bytes = exact_grad_workspace(m, n, k, &splits, &per);
    return PAM_SUCCESS;
}

pam_status_t pam_gemm_exact_grad_ws(pam_op_t transA, int64_t m, int64_t n, int64_t k, const float *A, int64_t lda,
                                    const float *B, int64_t ldb, const float *Mod, int64_t ldm, float *C,
                                    int64_t ldc, void *workspace, size_t workspace_bytes, hipStream_t stream) {
    const Workspace ws{workspace, workspace_bytes};
    return run_exact_grad(transA, m, n, k, A, lda, B, ldb, Mod, ldm, C, ldc, stream, &ws);
}

pam_status_t pam_gemm_plan_for_workspace(int64_t m, int64_t n, int64_t k, int64_t batch, size_t max_workspace_bytes,
                                         pam_plan_t *plan) {
    if (plan == nullptr)
        return fail(PAM_ERROR_INVALID_VALUE, "plan is NULL");
    if (m <= 0 || n <= 0 || k < 0 || batch <= 0)
        return fail(PAM_ERROR_INVALID_VALUE, "m, n, batch must be > 0 and k >= 0");
    if (m > kMaxDim || n > kMaxDim || k > kMaxDim)
        return fail(PAM_ERROR_INVALID_VALUE, "m, n and k must be below 2^31");
    if (check_output_size(m, n, batch) != PAM_SUCCESS)
        return PAM_ERROR_INVALID_VALUE;
    const Plan p = choose_plan(m, n, std::max<int64_t>(k, 1), batch, max_workspace_bytes);
    plan->tile_m = p.tile_m;
    plan->tile_n = p.tile_n;
    plan->splits = p.splits;
    plan->kgroups = p.kgroups;
    plan->whole_tiles = p.whole_tiles;
    return PAM_SUCCESS;
}

pam_status_t pam_gemm_plan(int64_t m, int64_t n, int64_t k, int64_t batch, pam_plan_t *plan) {
    return pam_gemm_plan_for_workspace(m, n, k, batch, kAnyWorkspace, plan);
}

// The plan of `plan` for these sizes (tile shape and split count checked).
pam_status_t plan_from(const pam_plan_t *plan, int64_t k, Plan *out) {
    if (plan == nullptr)
        return fail(PAM_ERROR_INVALID_VALUE, "plan is NULL");
    const bool tile_ok = (plan->kgroups == 1 && ((plan->tile_m == 128 && plan->tile_n == 128) ||
                                                 (plan->tile_m == 128 && plan->tile_n == 64) ||
                                                 (plan->tile_m == 64 && plan->tile_n == 64))) ||
                         (plan->kgroups == 4 && plan->tile_m == 64 && plan->tile_n == 64) ||
                         (plan->kgroups == 2 && plan->tile_m == 128 && plan->tile_n == 64);
    if (!tile_ok)
        return fail(PAM_ERROR_INVALID_VALUE,
                    "(tile_m, tile_n, kgroups) must be (128,128,1), (128,64,1), (128,64,2), (64,64,1) or "
                    "(64,64,4)");
    if (plan->splits < 1 || plan->splits > kMaxSplits)
        return fail(PAM_ERROR_INVALID_VALUE, "splits must be in [1, 64]");
    if (plan->whole_tiles < 0)
        return fail(PAM_ERROR_INVALID_VALUE, "whole_tiles must be >= 0");
    Plan p{plan->tile_m, plan->tile_n, plan->kgroups, 1, std::max<int64_t>(k, 1), 0};
    if (plan->splits > 1 && k > 0) {
        const int64_t per = ceil_div(ceil_div(k, plan->splits), pamk::kChunkK) * pamk::kChunkK;
        p.k_per_split = per;
        p.splits = (int)ceil_div(k, per);
        p.whole_tiles = plan->whole_tiles;
    }
    *out = p;
    return PAM_SUCCESS;
}

pam_status_t pam_gemm_plan_workspace_size(int64_t m, int64_t n, int64_t k, int64_t batch, const pam_plan_t *plan,
                                          size_t *bytes) {
    if (bytes == nullptr)
        return fail(PAM_ERROR_INVALID_VALUE, "bytes is NULL");
    *bytes = 0;
    if (m < 0 || n < 0 || k < 0 || batch < 0)
        return fail(PAM_ERROR_INVALID_VALUE, "m, n, k and batch must be >= 0");
    if (m > kMaxDim || n > kMaxDim || k > kMaxDim)
        return fail(PAM_ERROR_INVALID_VALUE, "m, n and k must be below 2^31");
    if (check_output_size(m, n, batch) != PAM_SUCCESS)
        return PAM_ERROR_INVALID_VALUE;
    Plan p;
    pam_status_t st = plan_from(plan, k, &p);
    if (st != PAM_SUCCESS)
        return st;
    if (m == 0 || n == 0 || k == 0 || batch == 0)
        return PAM_SUCCESS;
    Layout L;
    st = layout_of(p, m, n, batch, &L);
    if (st != PAM_SUCCESS)
        return st;
    *bytes = L.ws_bytes;
    return PAM_SUCCESS;
}

pam_status_t pam_gemm_batched_with_plan(pam_op_t transA, pam_op_t transB, int64_t m, int64_t n, int64_t k,
                                        const float *A, int64_t lda, int64_t strideA, const float *B, int64_t ldb,
                                        int64_t strideB, float *C, int64_t ldc, int64_t strideC, int64_t batch,
                                        const pam_plan_t *plan, void *workspace, size_t workspace_bytes,
                                        hipStream_t stream) {
    pam_status_t st = validate(transA, transB, m, n, k, A, lda, strideA, B, ldb, strideB, C, ldc, strideC, batch);
    if (st != PAM_SUCCESS)
        return st;
    Plan p;
    st = plan_from(plan, k, &p);
    if (st != PAM_SUCCESS)
        return st;
    if (m == 0 || n == 0 || batch == 0)
        return PAM_SUCCESS;
    const Workspace ws{workspace, workspace_bytes};
    return run_gemm(transA, transB, m, n, k, A, lda, strideA, B, ldb, strideB, C, ldc, strideC, batch, p, stream, 0,
                    &ws);
}

pam_status_t pam_device_info(int device, pam_device_info_t *info) {
    if (info == nullptr)
        return fail(PAM_ERROR_INVALID_VALUE, "info is NULL");
    std::memset(info, 0, sizeof *info);
    hipDeviceProp_t prop;
    hipError_t e = hipGetDeviceProperties(&prop, device);
    if (e != hipSuccess)
        return fail_hip(e, "hipGetDeviceProperties");
    int clock_khz = 0;
    e = hipDeviceGetAttribute(&clock_khz, hipDeviceAttributeClockRate, device);
    if (e != hipSuccess)
        return fail_hip(e, "hipDeviceGetAttribute(ClockRate)");
    info->compute_units = prop.multiProcessorCount;
    info->simds_per_cu = query_simds_per_cu(device);
    info->wavefront_size = prop.warpSize;
    // gfx950 SIMDs retire 32 lanes per clock for the ops the PAM matrix
    // product is built from (int32 add, float32 add / mul / fma); other
    // vector ops retire 16.
    info->lanes_per_simd = 32;
    info->clock_khz = clock_khz;
    info->valu_lane_ops_per_s =
        double(info->compute_units) * info->simds_per_cu * info->lanes_per_simd * double(clock_khz) * 1e3;
    std::snprintf(info->arch, sizeof info->arch, "%s", prop.gcnArchName);
    return PAM_SUCCESS;
}

const char *pam_status_string(pam_status_t s) {
    switch (s) {
    case PAM_SUCCESS:
        return "PAM_SUCCESS";
    case PAM_ERROR_INVALID_VALUE:
        return "PAM_ERROR_INVALID_VALUE";
    case PAM_ERROR_LAUNCH:
        return "PAM_ERROR_LAUNCH";
    case PAM_ERROR_NOT_SUPPORTED:
        return "PAM_ERROR_NOT_SUPPORTED";
    }
    return "PAM_ERROR_UNKNOWN";
}

const char *pam_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
