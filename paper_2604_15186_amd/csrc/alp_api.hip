// C ABI of the ALP allocation search: validation, device memory, launch geometry and timing.
// The arithmetic of the search runs in the kernels of alp_kernels.hip; this file only checks
// arguments, moves the tables and query values to the device and the results back.
#include <hip/hip_runtime.h>

#include <stdarg.h>
#include <stdlib.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <array>
#include <chrono>
#include <new>
#include <vector>

#include <rocprofiler-sdk-roctx/roctx.h>

#include "alp.h"
#include "alp_internal.h"

namespace {
// Names the dispatches that follow for a tracer (rocprofv3 --marker-trace shows the range around
// the kernels it covers); with no tracer attached both calls return at once.
struct Marked {
    explicit Marked(const char *what) { roctxRangePushA(what); }
    ~Marked() { roctxRangePop(); }
    Marked(const Marked &) = delete;
    Marked &operator=(const Marked &) = delete;
};
}  // namespace

using alp::kCapacityMax;

namespace {

thread_local char g_last_error[512] = "";

int32_t fail(int32_t status, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return status;
}

int32_t hip_fail(hipError_t e, const char *what)
{
    if (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation)
        return fail(ALP_ENOMEM, "%s: %s", what, hipGetErrorString(e));
    return fail(ALP_EDEVICE, "%s: %s", what, hipGetErrorString(e));
}

// Test hook: while the environment variable ALP_TEST_FAIL_ALLOC is set to a value other than
// "0", every device and pinned host allocation of the library fails as if memory were exhausted,
// so that tests reach the ALP_ENOMEM paths.
bool forced_alloc_failure()
{
    const char *v = getenv("ALP_TEST_FAIL_ALLOC");
    return v && v[0] && !(v[0] == '0' && v[1] == 0);
}

hipError_t alloc_device(void **ptr, size_t bytes)
{
    *ptr = nullptr;
    if (forced_alloc_failure())
        return hipErrorOutOfMemory;
    return hipMalloc(ptr, bytes);
}

hipError_t alloc_pinned(void **ptr, size_t bytes, unsigned flags)
{
    *ptr = nullptr;
    if (forced_alloc_failure())
        return hipErrorOutOfMemory;
    return hipHostMalloc(ptr, bytes, flags);
}

// Device buffer that only grows.  The larger buffer is allocated before the old one is
// released, so a failed growth leaves the buffer as it was.
struct DevBuf {
    void *ptr = nullptr;
    size_t cap = 0;
    bool guarded = false;           // work that may still use the buffer is queued on `stream`
    bool zeroed = false;            // a grown buffer is cleared (on `stream`) before its first use
    hipStream_t stream = nullptr;
    hipError_t ensure(size_t bytes)
    {
        if (bytes <= cap)
            return hipSuccess;
        void *grown = nullptr;
        hipError_t e = alloc_device(&grown, bytes);
        if (e != hipSuccess)
            return e;
        if (zeroed && (e = hipMemsetAsync(grown, 0, bytes, stream)) != hipSuccess) {
            (void)hipFree(grown);
            return e;
        }
        if (ptr) {
            // Queued asynchronous searches may still read or write the old buffer.
            if (guarded && (e = hipStreamSynchronize(stream)) != hipSuccess) {
                (void)hipFree(grown);
                return e;
            }
            (void)hipFree(ptr);
        }
        ptr = grown;
        cap = bytes;
        return hipSuccess;
    }
    void release()
    {
        if (ptr)
            (void)hipFree(ptr);
        ptr = nullptr;
        cap = 0;
    }
};

// Restores the caller's current device on scope exit.
struct DeviceGuard {
    int prev = -1;
    hipError_t status = hipSuccess;
    explicit DeviceGuard(int dev)
    {
        status = hipGetDevice(&prev);
        if (status == hipSuccess && prev != dev)
            status = hipSetDevice(dev);
    }
    ~DeviceGuard()
    {
        if (prev >= 0)
            (void)hipSetDevice(prev);
    }
};

}  // namespace

struct alp_ctx {
    int device = 0;
    hipStream_t stream = nullptr;
    alp_space_t space{};
    alp::SpaceDev sp{};
    uint64_t N = 0;
    uint32_t B = 0;
    uint64_t H = 0;
    int num_cus = 0;

    DevBuf tables;                 // W | n | p | allowed | rate | lat
    alp::TablesDev tdev{};

    DevBuf q_inst, rec, ext, inner, done, winners, idx, evals, tmax;   // q_inst: inst | cap | lambda
    DevBuf pair;                            // pair tables of the scan's pair form
    DevBuf fused_regions;                   // one-launch scan: per-block option records
    DevBuf fused_words;                     // one-launch scan: per-item best word and counter,
                                            // 0 between launches
    DevBuf split_dp;                        // allocate_kernel's knapsack table
    DevBuf pruned_table, pruned_orders, pruned_counts;   // pruned search scratch
    DevBuf place_in, place_out;                          // placement records
    alp_pruned_t *host_pruned = nullptr;    // mapped pinned results of pruned searches
    alp_pruned_t *host_pruned_dev = nullptr;
    size_t host_pruned_cap = 0;
    uint32_t *host_split = nullptr;         // mapped pinned: alp_plan_t (6 words) + budgets[16]
    uint32_t *host_split_dev = nullptr;
    uint32_t *host_query = nullptr;         // pinned staging of batch queries: inst | cap | lambda
    size_t host_query_cap = 0;
    alp_result_t *host_results = nullptr;   // pinned host memory the kernels write results to
    alp_result_t *host_results_dev = nullptr;  // its device-visible address
    size_t host_results_cap = 0;
    uint32_t *host_signal = nullptr;        // mapped word a single search's record signals in
    uint32_t *host_signal_dev = nullptr;    // (FinishArgs::signal), and its device address
    uint32_t call_seq = 0;                  // the last sequence number signalled

    uint32_t variant = 0, bpi_override = 0, tpb_override = 0, chunks_override = 0;
    int occupancy_cache[4][4][17] = {};   // [variant][log2 slots][threads / 64]: blocks per CU
    uint32_t timing_every = 0;          // 0: no timing; N: every N-th timed-API call
    uint64_t calls_seen = 0, timed_calls = 0;
    int timing = 0;                     // the current call records its kernel times
    hipEvent_t ev[4] = {nullptr, nullptr, nullptr, nullptr};
    // Timed asynchronous searches: their events (begin and end of the option terms, then of the
    // scan) wait in `pending` until the times are read; spent ones are reused.
    std::vector<std::array<hipEvent_t, 4>> ev_pending, ev_spare;
    std::vector<uint8_t> ev_pending_terms;  // per pending entry: its first two events are stamped
                                            // (a separate option-term kernel ran)
    bool last_terms = true;                 // the last launch_search ran the option-term kernel
    float last_ms[3] = {0, 0, 0};
    double total_ms[3] = {0, 0, 0};     // sums of last_ms since timing was last set
    void tally(int k) { total_ms[k] += last_ms[k]; }
    uint32_t last_blocks = 0;
    // The fixed scratch array of alp_search_batch_async_noalloc on this context's device, or
    // nullptr with static_status saying why its address could not be taken.
    uint8_t *static_scratch = nullptr;
    hipError_t static_status = hipSuccess;
};

namespace {

uint64_t ceil_div(uint64_t a, uint64_t b) { return (a + b - 1) / b; }

// Start of a call of an entry point whose kernels can be timed: it is timed if it is the first,
// or an N-th after it, since timing was set to every N-th call.
void begin_call(alp_ctx *c)
{
    c->timing = c->timing_every != 0 && c->calls_seen % c->timing_every == 0;
    c->calls_seen += c->timing_every != 0;
    c->timed_calls += c->timing;
}

int32_t validate_space(const alp_space_t *s, uint32_t *O_out, uint64_t *N_out)
{
    if (!s)
        return fail(ALP_EINVAL, "space is NULL");
    if (s->num_llms < 1 || s->num_llms > ALP_MAX_LLMS)
        return fail(ALP_EINVAL, "num_llms %u outside 1..%d", s->num_llms, ALP_MAX_LLMS);
    if (s->num_tp < 1 || s->num_tp > ALP_MAX_TP)
        return fail(ALP_EINVAL, "num_tp %u outside 1..%d", s->num_tp, ALP_MAX_TP);
    if (s->num_frac < 1 || s->num_frac > ALP_MAX_FRAC)
        return fail(ALP_EINVAL, "num_frac %u outside 1..%d", s->num_frac, ALP_MAX_FRAC);
    if (s->units_per_gpu < 1 || s->units_per_gpu > 16)
        return fail(ALP_EINVAL, "units_per_gpu %u outside 1..16", s->units_per_gpu);
    if (s->max_replicas < 1 || s->max_replicas > ALP_MAX_REPLICAS)
        return fail(ALP_EINVAL, "max_replicas %u outside 1..%d", s->max_replicas, ALP_MAX_REPLICAS);
    if (s->num_points < 1 || s->num_points > ALP_MAX_POINTS)
        return fail(ALP_EINVAL, "num_points %u outside 1..%d", s->num_points, ALP_MAX_POINTS);
    for (uint32_t i = 0; i < s->num_tp; ++i) {
        if (s->tp_values[i] < 1 || s->tp_values[i] > 64)
            return fail(ALP_EINVAL, "tp_values[%u]=%u outside 1..64", i, s->tp_values[i]);
        if (i && s->tp_values[i] <= s->tp_values[i - 1])
            return fail(ALP_EINVAL, "tp_values not strictly ascending");
    }
    for (uint32_t j = 0; j < s->num_frac; ++j) {
        if (s->frac_units[j] < 1 || s->frac_units[j] > s->units_per_gpu)
            return fail(ALP_EINVAL, "frac_units[%u]=%u outside 1..%u", j, s->frac_units[j],
                        s->units_per_gpu);
        if (j && s->frac_units[j] <= s->frac_units[j - 1])
            return fail(ALP_EINVAL, "frac_units not strictly ascending");
    }
    const uint32_t O = s->num_tp * s->num_frac * s->max_replicas;
    if (O > ALP_MAX_OPTIONS)
        return fail(ALP_EINVAL, "%u options per LLM exceed %d", O, ALP_MAX_OPTIONS);
    uint64_t N = 1;
    for (uint32_t m = 0; m < s->num_llms; ++m) {
        if (N > (UINT64_C(1) << 63) / O)
            return fail(ALP_ERANGE, "candidate space O^M reaches 2^63");
        N *= O;
    }
    if (N >= (UINT64_C(1) << 63))
        return fail(ALP_ERANGE, "candidate space O^M reaches 2^63");
    *O_out = O;
    *N_out = N;
    return ALP_OK;
}

int32_t validate_tables(const alp_space_t *s, uint32_t B, const uint64_t *W, const uint32_t *n,
                        const uint32_t *p, const uint8_t *allowed, const uint32_t *rate,
                        const uint32_t *lat, uint64_t H)
{
    if (!W || !n || !p || !allowed || !rate || !lat)
        return fail(ALP_EINVAL, "a table pointer is NULL");
    if (H < 1 || H >= (UINT64_C(1) << 48))
        return fail(ALP_EINVAL, "hbm_bytes_per_gpu outside 1..2^48-1");
    const uint32_t M = s->num_llms, nt = s->num_tp, nf = s->num_frac, K = s->num_points;
    for (uint32_t b = 0; b < B; ++b) {
        uint64_t worst = 0;   // largest possible L_w over deployable, fitting options
        for (uint32_t m = 0; m < M; ++m) {
            const uint64_t lm = (uint64_t)b * M + m;
            if (W[lm] >= (UINT64_C(1) << 48))
                return fail(ALP_EINVAL, "instance %u llm %u: weight_bytes >= 2^48", b, m);
            if (n[lm] < 1 || n[lm] >= (1u << 31) || p[lm] < 1 || p[lm] >= (1u << 31))
                return fail(ALP_EINVAL, "instance %u llm %u: n_milli/p_milli outside 1..2^31-1", b, m);
            uint64_t worst_m = 0;
            for (uint32_t i = 0; i < nt; ++i) {
                for (uint32_t j = 0; j < nf; ++j) {
                    const uint64_t tab = (lm * nt + i) * nf + j;
                    if (allowed[tab] > 1)
                        return fail(ALP_EINVAL, "instance %u llm %u: allowed must be 0 or 1", b, m);
                    const uint32_t *r = rate + tab * K, *l = lat + tab * K;
                    uint32_t max_lat = 0;
                    for (uint32_t k = 0; k < K; ++k) {
                        if (r[k] >= (1u << 31) || l[k] >= (1u << 31))
                            return fail(ALP_EINVAL, "instance %u llm %u: rate/latency >= 2^31", b, m);
                        if (k && r[k] <= r[k - 1])
                            return fail(ALP_EINVAL,
                                        "instance %u llm %u tp#%u share#%u: rates not strictly ascending",
                                        b, m, i, j);
                        max_lat = l[k] > max_lat ? l[k] : max_lat;
                    }
                    const bool fits = W[lm] * s->units_per_gpu <=
                                      (uint64_t)s->tp_values[i] * s->frac_units[j] * H;
                    if (allowed[tab] && fits) {
                        const uint64_t c = (uint64_t)max_lat * n[lm] / p[lm];
                        worst_m = c > worst_m ? c : worst_m;
                    }
                }
            }
            worst += worst_m;
            if (worst >= 0xFFFFFFFFull)
                return fail(ALP_ERANGE,
                            "instance %u: latency sum can reach %llu us, beyond the 32-bit objective",
                            b, (unsigned long long)worst);
        }
    }
    return ALP_OK;
}

uint32_t capacity_of(const alp_ctx *c, uint32_t gpu_budget)
{
    const uint64_t cap = (uint64_t)c->space.units_per_gpu * gpu_budget;
    return cap > kCapacityMax ? kCapacityMax : (uint32_t)cap;
}

uint32_t slots_for(uint32_t O)
{
    return O <= 64 ? 1 : O <= 128 ? 2 : O <= 256 ? 4 : 8;
}

// Resident blocks per CU of a scan kernel (occupancy query), cached per context.
int blocks_per_cu(alp_ctx *c, uint32_t variant, uint32_t slots, uint32_t threads)
{
    const uint32_t ls = slots == 1 ? 0 : slots == 2 ? 1 : slots == 4 ? 2 : 3;
    int &slot = c->occupancy_cache[variant & 3][ls][(threads / 64) & 15];
    if (slot <= 0)
        slot = alp::scan_blocks_per_cu(variant, slots, threads, c->sp);
    return slot;
}

// Blocks per item for a grid of `count` items.  Blocks are dispatched as resident slots free
// up, so a grid runs in rounds of `resident` blocks; a last round that is only partly filled
// leaves the chip idle while it runs, and one round alone ends with a long tail.  The grid is
// sized for about kRounds full rounds: among the block counts that end exactly at a round
// boundary (k * resident / count per item, k = 1 .. kRounds), the one with the least time per
// unit of work -- (rounds + a quarter-round tail) / blocks -- is taken.
uint64_t blocks_per_item_for_rounds(uint64_t count, uint64_t resident, uint64_t max_bpi)
{
    constexpr uint64_t kRounds = 4;
    if (count == 0 || resident == 0)
        return 1;
    uint64_t best = 1;
    double best_cost = (double)ceil_div(count, resident) + 0.25;
    for (uint64_t k = 1; k <= kRounds; ++k) {
        uint64_t bpi = k * resident / count;
        if (bpi > max_bpi)
            bpi = max_bpi;
        if (bpi < 1)
            continue;
        const double cost = ((double)ceil_div(count * bpi, resident) + 0.25) / (double)bpi;
        if (cost < best_cost) {
            best_cost = cost;
            best = bpi;
        }
    }
    return best;
}

// Launch geometry of a scan of `count` items.  ERANGE when no launch can cover the space: the
// fixed-range form counts a wave's rows in 32 bits, so a wave must get fewer than 2^32 rows
// (the automatic plan adds blocks until it does; a blocks_per_item override that leaves a wave
// more is rejected), and a launch holds fewer than 2^31 blocks.
// Largest space (candidates per item) searched in one launch.
constexpr uint64_t kFusedCandidatesMax = UINT64_C(1) << 25;

int32_t plan_scan(alp_ctx *c, uint32_t count, alp::ScanGeometry &out, bool allow_fused = true)
{
    alp::ScanGeometry g{};
    const alp::SpaceDev &sp = c->sp;
    // Variants 4 and 5 are the row-minimum scan with a fixed choice of work distribution;
    // ALP_LAUNCH_SEPARATE_TERMS added to 0, 1, 4 or 5 keeps the option terms in their own kernel.
    const uint32_t variant = c->variant & ~ALP_LAUNCH_SEPARATE_TERMS;
    g.variant = variant == 0 || variant >= 4 ? 1 : variant;
    g.slots = slots_for(sp.O);
    const uint64_t cus = c->num_cus > 0 ? (uint64_t)c->num_cus : 256;
    // Pair form (variant 1; forced by variant 6, chosen for 5 or more LLMs while the batch's
    // tables stay within 4 MiB, i.e. resident in L2): LLMs M-3 and M-2 folded into one inner
    // table of O^2 records, so a row carries O^2 candidates per lane-slot and the per-row work
    // is spread over 128 times more of them.  (132 4-LLM items, 17 MiB of tables: slower.)
    // Rows are split into sub-rows of at most 1,024 records, claimed within blocks of 16 waves,
    // 32 waves per CU per round and four rounds of blocks, about 8 sub-rows per wave.
    constexpr uint64_t kPairBytesMax = UINT64_C(4) << 20;
    if (g.variant == 1 && sp.M >= 3 && (variant == 6 || (variant == 0 && sp.M >= 5)) &&
        (uint64_t)count * alp::pair_stride(sp.O) * sizeof(uint2) <= kPairBytesMax) {
        uint64_t rows = 1;
        for (uint32_t m = 3; m < sp.M; ++m)
            rows *= sp.O;
        const uint32_t n16 = alp::pair_stride(sp.O) / 16;
        uint32_t chunks = n16;
        for (uint32_t k = 1; k <= n16; ++k)
            if (n16 % k == 0 && alp::pair_stride(sp.O) / k <= 1024) {
                chunks = k;
                break;
            }
        if (c->chunks_override && n16 % c->chunks_override == 0)
            chunks = c->chunks_override;
        const uint64_t sub_rows = rows * chunks;
        if (sub_rows < (UINT64_C(1) << 32)) {
            g.pair = 1;
            g.dynamic = 1;
            g.chunks = chunks;
            g.rows = sub_rows;
            g.threads = c->tpb_override ? c->tpb_override : 1024;
            const uint64_t wpb = g.threads / 64;
            const uint64_t items = std::max<uint64_t>(1, count);
            const uint64_t waves =
                std::max<uint64_t>(1, std::min<uint64_t>(cus * 32 * 4, items * sub_rows / 8));
            uint64_t bpi = c->bpi_override ? c->bpi_override
                                           : std::max<uint64_t>(1, ceil_div(waves, items * wpb));
            g.rows_per_wave = ceil_div(g.rows, bpi * wpb);
            if (!c->bpi_override)
                bpi = ceil_div(g.rows, g.rows_per_wave * wpb);
            if (bpi * items >= (UINT64_C(1) << 31))
                return fail(ALP_ERANGE, "batch too large for one launch (%llu blocks)",
                            (unsigned long long)(bpi * items));
            g.blocks_per_item = (uint32_t)bpi;
            out = g;
            return ALP_OK;
        }
    }
    if (g.variant != 2) {
        g.rows = 1;
        for (uint32_t m = 2; m < sp.M; ++m)
            g.rows *= sp.O;
        g.chunks = 1;
        // Fixed ranges of whole rows per wave: blocks of 8 waves (fewer blocks, fewer
        // end-of-block reductions), at most one wave per row, and each wave gets at least
        // kMinRecordsPerWave of the inner LLM's records (rows times records per row) when the
        // item has that many, so that a wave's fixed costs (setup, end-of-wave re-scan, block
        // reduction) stay small.
        constexpr uint64_t kMinRecordsPerWave = 512;
        const uint64_t per_row = sp.M >= 2 ? alp::inner_stride(sp.O) : 1;
        const uint64_t min_rows = std::max<uint64_t>(1, kMinRecordsPerWave / per_row);
        g.threads = c->tpb_override ? c->tpb_override
                                    : (uint32_t)(64 * (g.rows < 8 ? g.rows : 8));
        uint32_t wpb = g.threads / 64;
        const uint64_t max_waves = g.rows >= min_rows ? g.rows / min_rows : 1;
        uint64_t bpi = c->bpi_override;
        if (!bpi)
            bpi = blocks_per_item_for_rounds(
                count, cus * (uint64_t)blocks_per_cu(c, g.variant, g.slots, g.threads),
                ceil_div(max_waves, wpb));
        // Rows handed out within each block instead (row-minimum scan, needs fewer than 2^32
        // sub-rows per item): forced by variant 5 or a row split, else chosen when fixed ranges
        // would leave a wave fewer than 16 rows.  Waves then finish together however the SIMD
        // shares its issue slots among them, and rows may be split into sub-rows of the inner
        // LLM's records.  Plan: at most 16 waves per CU over the whole batch and at least two
        // of the finest sub-rows per wave; blocks of 8 waves while that leaves CUs without a
        // block, else of 16; rows split so that a wave gets about 4 sub-rows (a wave claims its next
        // sub-row late, so whole sub-rows balance well and keep the per-sub-row work small).
        const bool splittable = g.variant == 1 && sp.M >= 2;
        const uint32_t n16 = alp::inner_stride(sp.O) / 16;      // chunks must divide this
        bool dyn = g.variant == 1 && variant != 4 &&
                   (variant == 5 || c->chunks_override > 1 ||
                    ceil_div(g.rows, bpi * wpb) < 16);
        if (dyn && g.rows * (splittable ? n16 : 1) >= (UINT64_C(1) << 32))
            dyn = false;
        if (dyn) {
            const uint64_t finest = g.rows * (splittable ? n16 : 1);
            const uint64_t items = std::max<uint64_t>(1, count);
            const uint64_t waves = std::max<uint64_t>(
                1, std::min<uint64_t>(cus * 16, items * std::max<uint64_t>(1, finest / 2)));
            if (!c->tpb_override)
                g.threads = (uint32_t)(64 * std::min<uint64_t>(waves <= cus * 8 ? 8 : 16,
                                                               std::max<uint64_t>(1, finest)));
            wpb = g.threads / 64;
            if (!c->bpi_override)
                bpi = std::max<uint64_t>(1, ceil_div(waves, items * wpb));
            if (splittable && c->chunks_override && n16 % c->chunks_override == 0) {
                g.chunks = c->chunks_override;
            } else if (splittable) {
                g.chunks = n16;
                for (uint32_t k = 1; k <= n16; ++k)
                    if (n16 % k == 0 && g.rows * k >= 4 * bpi * wpb) {
                        g.chunks = k;
                        break;
                    }
            }
            g.rows *= g.chunks;
        }
        g.dynamic = dyn ? 1u : 0u;
        constexpr uint64_t kWaveRowsMax = UINT64_C(0xFFFFFFFF);
        if (g.variant == 1 && !dyn && ceil_div(g.rows, bpi * wpb) > kWaveRowsMax) {
            if (c->bpi_override)
                return fail(ALP_ERANGE,
                            "blocks_per_item %u leaves a wave %llu rows (at most 2^32 - 1); "
                            "raise blocks_per_item", c->bpi_override,
                            (unsigned long long)ceil_div(g.rows, bpi * wpb));
            bpi = ceil_div(g.rows, kWaveRowsMax * wpb);
        }
        g.rows_per_wave = ceil_div(g.rows, bpi * wpb);
        if (!c->bpi_override)
            bpi = ceil_div(g.rows, g.rows_per_wave * wpb);
        if (bpi * std::max<uint64_t>(1, count) >= (UINT64_C(1) << 31))
            return fail(ALP_ERANGE, "batch too large for one launch (%llu blocks)",
                        (unsigned long long)(bpi * std::max<uint64_t>(1, count)));
        g.blocks_per_item = (uint32_t)bpi;
        // One launch for spaces of at most 2^25 candidates (the winner fits one 64-bit word in
        // any space below 2^32), unless the option terms are asked to run in their own kernel.
        // Larger spaces take the two-launch form: every block of the one-launch scan repeats the
        // item's option terms (a prologue of about 2.7 us), which a long scan pays for more
        // than it saves the option-term kernel (a 4-LLM search of 2^28 candidates: 29.3 us per
        // step in two launches, 30.7 in one; a 3-LLM search of 2^21: 11.9 in two, 9.3 in one).
        // The block keeps the item's curves and records in LDS: at most 56 KiB of them, with
        // the kernel's own few KiB within 64 KiB (every space of fewer than 2^32 candidates
        // fits; the test only guards the layout).
        g.fused = g.variant == 1 && allow_fused && c->N <= kFusedCandidatesMax &&
                  alp::fused_lds_bytes(sp) <= (UINT64_C(56) << 10) &&
                  !(c->variant & ALP_LAUNCH_SEPARATE_TERMS) ? 1u : 0u;
    } else {
        g.threads = c->tpb_override ? c->tpb_override : 256;
        const uint64_t resident =
            cus * (uint64_t)blocks_per_cu(c, g.variant, g.slots, g.threads);
        uint64_t bpi = c->bpi_override ? c->bpi_override : (count ? ceil_div(resident, count) : 1);
        const uint64_t max_bpi = ceil_div(c->N, g.threads);
        if (!c->bpi_override && bpi > max_bpi)
            bpi = max_bpi;
        if (bpi < 1)
            bpi = 1;
        g.per_thread = ceil_div(c->N, bpi * g.threads);
        if (bpi * std::max<uint64_t>(1, count) >= (UINT64_C(1) << 31))
            return fail(ALP_ERANGE, "batch too large for one launch (%llu blocks)",
                        (unsigned long long)(bpi * std::max<uint64_t>(1, count)));
        g.blocks_per_item = (uint32_t)bpi;
    }
    out = g;
    return ALP_OK;
}

int32_t ensure_host_query(alp_ctx *c, size_t count)
{
    if (count <= c->host_query_cap)
        return ALP_OK;
    void *grown = nullptr;
    hipError_t e = alloc_pinned(&grown, 3 * count * sizeof(uint32_t), hipHostMallocDefault);
    if (e != hipSuccess)
        return hip_fail(e, "hipHostMalloc(queries)");
    if (c->host_query)
        (void)hipHostFree(c->host_query);
    c->host_query = (uint32_t *)grown;
    c->host_query_cap = count;
    return ALP_OK;
}

// Uploads batch queries (instance, capacity, target) through pinned staging; q gets the device
// arrays.
int32_t upload_queries(alp_ctx *c, uint32_t count, const uint32_t *inst, const uint32_t *cap,
                       const uint32_t *lambda, alp::QueryDev &q)
{
    int32_t st = ensure_host_query(c, count);
    if (st != ALP_OK)
        return st;
    const size_t bytes = (size_t)count * sizeof(uint32_t);
    hipError_t e;
    if ((e = c->q_inst.ensure(3 * bytes)) != hipSuccess)
        return hip_fail(e, "hipMalloc(queries)");
    memcpy(c->host_query, inst, bytes);
    memcpy(c->host_query + count, cap, bytes);
    memcpy(c->host_query + 2 * (size_t)count, lambda, bytes);
    if ((e = hipMemcpyAsync(c->q_inst.ptr, c->host_query, 3 * bytes, hipMemcpyHostToDevice,
                            c->stream)) != hipSuccess)
        return hip_fail(e, "copy queries");
    q = alp::QueryDev{};
    q.inst = (const uint32_t *)c->q_inst.ptr;
    q.capacity = q.inst + count;
    q.lambda = q.inst + 2 * (size_t)count;
    return ALP_OK;
}

int32_t ensure_host_results(alp_ctx *c, size_t count)
{
    if (!c->host_signal) {
        void *h = nullptr, *d = nullptr;
        hipError_t e = alloc_pinned(&h, 64, hipHostMallocMapped);
        if (e != hipSuccess)
            return hip_fail(e, "hipHostMalloc(signal)");
        if ((e = hipHostGetDevicePointer(&d, h, 0)) != hipSuccess) {
            (void)hipHostFree(h);
            return hip_fail(e, "hipHostGetDevicePointer(signal)");
        }
        c->host_signal = (uint32_t *)h;
        c->host_signal_dev = (uint32_t *)d;
        __atomic_store_n(c->host_signal, 0u, __ATOMIC_RELEASE);
    }
    if (count <= c->host_results_cap)
        return ALP_OK;
    void *grown = nullptr, *grown_dev = nullptr;
    hipError_t e = alloc_pinned(&grown, count * sizeof(alp_result_t), hipHostMallocMapped);
    if (e != hipSuccess)
        return hip_fail(e, "hipHostMalloc(results)");
    if ((e = hipHostGetDevicePointer(&grown_dev, grown, 0)) != hipSuccess) {
        (void)hipHostFree(grown);
        return hip_fail(e, "hipHostGetDevicePointer(results)");
    }
    if (c->host_results)
        (void)hipHostFree(c->host_results);
    c->host_results = (alp_result_t *)grown;
    c->host_results_dev = (alp_result_t *)grown_dev;
    c->host_results_cap = count;
    return ALP_OK;
}

// Device scratch of one search launch: per-option records, the inner (or pair) table, the
// per-item counters and the block winners.
struct SearchScratch {
    uint2 *rec = nullptr, *ext = nullptr, *inner = nullptr, *pair = nullptr;
    uint32_t *done = nullptr, *best = nullptr;
    alp::Winner *winners = nullptr;
    uint2 *regions = nullptr;                  // one-launch form
    uint32_t *fdone = nullptr, *fgroup = nullptr;
    unsigned long long *fbest = nullptr;
};

// Byte sizes of the scratch parts of a launch of `count` items with geometry g.  done[count],
// then best[count] at least 4 KiB further: the two per-item words take one atomic per block
// each, and counters in one line would queue behind each other.
struct ScratchSizes {
    uint64_t rec, inner, pair, counters, best_at, winners;
};

ScratchSizes scratch_sizes(const alp::SpaceDev &sp, uint32_t count, const alp::ScanGeometry &g)
{
    ScratchSizes z;
    z.rec = (uint64_t)count * sp.M * sp.O * sizeof(uint2);
    z.inner = (uint64_t)count * alp::inner_stride(sp.O) * sizeof(uint2);
    z.pair = g.pair ? (uint64_t)count * alp::pair_stride(sp.O) * sizeof(uint2) : 0;
    z.best_at = ((uint64_t)count + 2047) / 1024 * 1024;
    z.counters = (z.best_at + count) * sizeof(uint32_t);
    z.winners = (uint64_t)count * g.blocks_per_item * sizeof(alp::Winner);
    return z;
}

// The context's own scratch buffers, grown to the launch's sizes.
int32_t context_scratch(alp_ctx *c, uint32_t count, const alp::ScanGeometry &g, SearchScratch &s)
{
    hipError_t e;
    if (g.fused) {
        // Per block: its option records; per item: the best word (8 B), then the counters.
        const uint64_t blocks = (uint64_t)count * g.blocks_per_item;
        if ((e = c->fused_regions.ensure(blocks * alp::fused_region(c->sp.M, c->sp.O) *
                                         sizeof(uint2))) != hipSuccess)
            return hip_fail(e, "hipMalloc(block records)");
        const uint64_t groups = (g.blocks_per_item + alp::kFusedGroup - 1) / alp::kFusedGroup;
        if ((e = c->fused_words.ensure((uint64_t)count * (12 + 4 * groups))) != hipSuccess)
            return hip_fail(e, "hipMalloc(item words)");
        s.regions = (uint2 *)c->fused_regions.ptr;
        s.fbest = (unsigned long long *)c->fused_words.ptr;
        s.fdone = (uint32_t *)(s.fbest + count);
        s.fgroup = s.fdone + count;
        return ALP_OK;
    }
    const ScratchSizes z = scratch_sizes(c->sp, count, g);
    if ((e = c->rec.ensure(z.rec)) != hipSuccess)
        return hip_fail(e, "hipMalloc(rec)");
    if ((e = c->ext.ensure(z.rec)) != hipSuccess)
        return hip_fail(e, "hipMalloc(ext)");
    if ((e = c->inner.ensure(z.inner)) != hipSuccess)
        return hip_fail(e, "hipMalloc(inner)");
    if ((e = c->done.ensure(z.counters)) != hipSuccess)
        return hip_fail(e, "hipMalloc(done)");
    if ((e = c->winners.ensure(z.winners)) != hipSuccess)
        return hip_fail(e, "hipMalloc(winners)");
    if (g.pair && (e = c->pair.ensure(z.pair)) != hipSuccess)
        return hip_fail(e, "hipMalloc(pair table)");
    s.rec = (uint2 *)c->rec.ptr;
    s.ext = (uint2 *)c->ext.ptr;
    s.inner = (uint2 *)c->inner.ptr;
    s.pair = g.pair ? (uint2 *)c->pair.ptr : nullptr;
    s.done = (uint32_t *)c->done.ptr;
    s.best = s.done + z.best_at;
    s.winners = (alp::Winner *)c->winners.ptr;
    return ALP_OK;
}

// Queues the option-term and scan kernels (with the fused final reduction and result decode) of
// `count` searches described by q on the context stream, using scratch s for geometry g.
// Results go to `out` (device-visible); with device queries (raw), rejected ones to EINVAL
// records.  ev (4 events or nullptr): begin and end of the option-term kernel, then of the scan,
// stamped by the dispatches.
int32_t launch_search_with(alp_ctx *c, const alp::QueryDev &q, uint32_t count, alp_result_t *out,
                           const alp::RawQueries *raw, hipEvent_t *ev, const alp::ScanGeometry &g,
                           const SearchScratch &s, uint32_t *signal = nullptr, uint32_t seq = 0)
{
    const bool timed = ev != nullptr;
    const alp::SpaceDev &sp = c->sp;
    const uint64_t nwin = (uint64_t)count * g.blocks_per_item;
    hipError_t e;
    c->last_terms = !g.fused;
    if (g.fused) {
        alp::FinishArgs fa{};
        fa.sp = sp;
        fa.out = out;
        fa.signal = signal;
        fa.seq = seq;
        alp::FusedArgs fz{};
        fz.tb = c->tdev;
        if (raw)
            fz.raw = *raw;
        fz.regions = s.regions;
        fz.region = alp::fused_region(sp.M, sp.O);
        fz.done = s.fdone;
        fz.group_done = s.fgroup;
        fz.best = s.fbest;
        if ((e = alp::launch_scan(sp, q, count, nullptr, nullptr, g, nullptr, fa, c->stream,
                                  timed ? ev[2] : nullptr, timed ? ev[3] : nullptr, &fz)) !=
            hipSuccess)
            return hip_fail(e, "scan launch");
        c->last_blocks = (uint32_t)nwin;
        return ALP_OK;
    }
    alp::FinishArgs fa;
    fa.sp = sp;
    fa.ext = s.ext;
    fa.done = s.done;
    fa.best = s.best;
    fa.out = out;
    fa.invalid = raw ? raw->invalid : nullptr;
    fa.signal = signal;
    fa.seq = seq;
    alp::ScanReset reset;
    reset.done = s.done;
    reset.best = s.best;
    reset.winners = s.winners;
    reset.n_winners = nwin;
    if ((e = alp::launch_option_terms(sp, c->tdev, q, count, s.rec, s.ext, s.inner, reset,
                                      c->stream, raw, timed ? ev[0] : nullptr,
                                      timed ? ev[1] : nullptr)) != hipSuccess)
        return hip_fail(e, "option_terms launch");
    const uint2 *inner = s.inner;
    if (g.pair) {
        if ((e = alp::launch_pair_terms(sp, count, s.rec, s.inner, s.pair, c->stream)) !=
            hipSuccess)
            return hip_fail(e, "pair_terms launch");
        inner = s.pair;
    }
    if ((e = alp::launch_scan(sp, q, count, s.rec, inner, g, s.winners, fa, c->stream,
                              timed ? ev[2] : nullptr, timed ? ev[3] : nullptr)) != hipSuccess)
        return hip_fail(e, "scan launch");
    c->last_blocks = (uint32_t)nwin;
    return ALP_OK;
}

// launch_search_with on the context's own (growing) scratch buffers.
int32_t launch_search(alp_ctx *c, const alp::QueryDev &q, uint32_t count, alp_result_t *out,
                      const alp::RawQueries *raw, hipEvent_t *ev, uint32_t *signal = nullptr,
                      uint32_t seq = 0)
{
    alp::ScanGeometry g;
    int32_t st = plan_scan(c, count, g);
    if (st != ALP_OK)
        return st;
    SearchScratch s;
    if ((st = context_scratch(c, count, g, s)) != ALP_OK)
        return st;
    // The range stays out of launch_search_with itself: the entry point that must not allocate
    // calls it too, and a tracer may allocate host memory to record a range.
    Marked mark(g.fused ? "alp search: one-launch scan and finish"
                        : "alp search: option terms, scan and finish");
    return launch_search_with(c, q, count, out, raw, ev, g, s, signal, seq);
}

// Synchronous searches: results in the context's mapped host buffer.  A single untimed search
// has its record signalled in host memory (FinishArgs::signal): the caller reads it as soon as
// the kernel's last block has written it, rather than after the kernel's completion reaches
// the host.  After the first millisecond the wait also polls the stream, once a millisecond
// (a poll costs microseconds, so it stays off the path of short searches); a stream that ends
// (or fails) without the signal falls back to the synchronisation, which reports any error.
int32_t run_search(alp_ctx *c, const alp::QueryDev &q, uint32_t count)
{
    int32_t st = ensure_host_results(c, count);
    if (st != ALP_OK)
        return st;
    const bool signalled = count == 1 && !c->timing;
    uint32_t seq = 0;
    if (signalled && ++c->call_seq == 0)
        ++c->call_seq;                         // 0 is the word's initial value
    if (signalled)
        seq = c->call_seq;
    if ((st = launch_search(c, q, count, c->host_results_dev, nullptr, c->timing ? c->ev : nullptr,
                            signalled ? c->host_signal_dev : nullptr, seq)) != ALP_OK)
        return st;
    hipError_t e = hipSuccess;
    bool seen = false;
    auto poll_at = std::chrono::steady_clock::now() + std::chrono::milliseconds(1);
    for (uint32_t k = 1; signalled; ++k) {
        if (__atomic_load_n(c->host_signal, __ATOMIC_ACQUIRE) == seq) {
            seen = true;
            break;
        }
        if ((k & 255) == 0 && std::chrono::steady_clock::now() >= poll_at) {
            if (hipStreamQuery(c->stream) != hipErrorNotReady)
                break;
            poll_at = std::chrono::steady_clock::now() + std::chrono::milliseconds(1);
        }
        __builtin_ia32_pause();
    }
    if (!seen && (e = hipStreamSynchronize(c->stream)) != hipSuccess)
        return hip_fail(e, "hipStreamSynchronize");
    if (c->timing) {
        c->last_ms[0] = 0.0f;                  // no option-term kernel in the one-launch form
        for (int k = c->last_terms ? 0 : 1; k < 2; ++k) {
            if ((e = hipEventElapsedTime(&c->last_ms[k], c->ev[2 * k], c->ev[2 * k + 1])) !=
                hipSuccess)
                return hip_fail(e, "hipEventElapsedTime");
            c->tally(k);
        }
        c->last_ms[2] = 0.0f;
    }
    return ALP_OK;
}

// Reads the times of the timed asynchronous searches queued so far (waiting for them), adds
// them to the totals and leaves the last one in last_ms.
int32_t collect_async_times(alp_ctx *c)
{
    hipError_t e;
    for (size_t i = 0; i < c->ev_pending.size(); ++i) {
        auto &t = c->ev_pending[i];
        const bool terms = c->ev_pending_terms[i] != 0;
        c->last_ms[0] = 0.0f;
        if ((e = hipEventSynchronize(t[3])) != hipSuccess ||
            (terms && (e = hipEventElapsedTime(&c->last_ms[0], t[0], t[1])) != hipSuccess) ||
            (e = hipEventElapsedTime(&c->last_ms[1], t[2], t[3])) != hipSuccess)
            return hip_fail(e, "reading the times of queued searches");
        c->last_ms[2] = 0.0f;
        c->tally(0);
        c->tally(1);
        c->ev_spare.push_back(t);
    }
    c->ev_pending.clear();
    c->ev_pending_terms.clear();
    return ALP_OK;
}

int32_t check_instance(const alp_ctx *c, uint32_t inst)
{
    if (inst >= c->B)
        return fail(ALP_EINVAL, "instance %u out of range (%u loaded)", inst, c->B);
    return ALP_OK;
}

}  // namespace

extern "C" {

int32_t alp_load_profiles(alp_ctx **out, const alp_space_t *space, uint32_t num_instances,
                          const uint64_t *weight_bytes, const uint32_t *n_milli,
                          const uint32_t *p_milli, const uint8_t *allowed,
                          const uint32_t *rate_milli, const uint32_t *lat_us,
                          uint64_t hbm_bytes_per_gpu, int32_t device, void *hip_stream)
{
    if (!out)
        return fail(ALP_EINVAL, "out is NULL");
    uint32_t O = 0;
    uint64_t N = 0;
    int32_t st = validate_space(space, &O, &N);
    if (st != ALP_OK)
        return st;
    if (num_instances < 1)
        return fail(ALP_EINVAL, "num_instances must be >= 1");
    st = validate_tables(space, num_instances, weight_bytes, n_milli, p_milli, allowed, rate_milli,
                         lat_us, hbm_bytes_per_gpu);
    if (st != ALP_OK)
        return st;

    int ndev = 0;
    hipError_t e = hipGetDeviceCount(&ndev);
    if (e != hipSuccess || ndev <= 0)
        return fail(ALP_EDEVICE, "no HIP device available");
    if (device < 0 || device >= ndev)
        return fail(ALP_EDEVICE, "device %d out of range (%d devices)", device, ndev);
    DeviceGuard guard(device);
    if (guard.status != hipSuccess)
        return hip_fail(guard.status, "hipSetDevice");

    alp_ctx *c = new (std::nothrow) alp_ctx();
    if (!c)
        return fail(ALP_ENOMEM, "host allocation failed");
    c->device = device;
    c->stream = (hipStream_t)hip_stream;
    for (DevBuf *b : {&c->q_inst, &c->rec, &c->ext, &c->inner, &c->done, &c->winners, &c->pair,
                      &c->fused_regions, &c->fused_words}) {
        b->guarded = true;                              // used by alp_search_batch_async
        b->stream = c->stream;
    }
    c->fused_words.zeroed = true;
    c->space = *space;
    c->N = N;
    c->B = num_instances;
    c->H = hbm_bytes_per_gpu;
    alp::SpaceDev &sp = c->sp;
    sp.M = space->num_llms;
    sp.n_tp = space->num_tp;
    sp.n_fq = space->num_frac;
    sp.D = space->max_replicas;
    sp.K = space->num_points;
    sp.Q = space->units_per_gpu;
    sp.O = O;
    sp.mul_O = alp::div_multiplier(O);
    sp.mul_D = alp::div_multiplier(sp.D);
    sp.tp8 = sp.fq8 = 0;
    for (uint32_t i = 0; i < sp.n_tp; ++i)
        sp.tp8 |= (uint64_t)space->tp_values[i] << (8 * i);
    for (uint32_t j = 0; j < sp.n_fq; ++j)
        sp.fq8 |= (uint64_t)space->frac_units[j] << (8 * j);
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, device) == hipSuccess)
        c->num_cus = prop.multiProcessorCount;

    const uint64_t BM = (uint64_t)num_instances * sp.M;
    const uint64_t BMT = BM * sp.n_tp * sp.n_fq;
    const uint64_t BMTK = BMT * sp.K;
    auto align = [](uint64_t v) { return (v + 255) & ~UINT64_C(255); };
    const uint64_t offW = 0, offn = align(offW + BM * 8), offp = align(offn + BM * 4),
                   offA = align(offp + BM * 4), offR = align(offA + BMT),
                   offL = align(offR + BMTK * 4), total = align(offL + BMTK * 4);
    if ((e = c->tables.ensure(total)) != hipSuccess) {
        st = hip_fail(e, "hipMalloc(tables)");
        alp_free(c);
        return st;
    }
    uint8_t *base = (uint8_t *)c->tables.ptr;
    struct {
        uint64_t off;
        const void *src;
        uint64_t bytes;
    } parts[] = {{offW, weight_bytes, BM * 8}, {offn, n_milli, BM * 4}, {offp, p_milli, BM * 4},
                 {offA, allowed, BMT}, {offR, rate_milli, BMTK * 4}, {offL, lat_us, BMTK * 4}};
    for (auto &pp : parts) {
        if ((e = hipMemcpyAsync(base + pp.off, pp.src, pp.bytes, hipMemcpyHostToDevice,
                                c->stream)) != hipSuccess) {
            st = hip_fail(e, "copy tables");
            alp_free(c);
            return st;
        }
    }
    if ((e = hipStreamSynchronize(c->stream)) != hipSuccess) {
        st = hip_fail(e, "hipStreamSynchronize");
        alp_free(c);
        return st;
    }
    c->tdev.W = (const uint64_t *)(base + offW);
    c->tdev.n = (const uint32_t *)(base + offn);
    c->tdev.p = (const uint32_t *)(base + offp);
    c->tdev.allowed = (const uint8_t *)(base + offA);
    c->tdev.rate = (const uint32_t *)(base + offR);
    c->tdev.lat = (const uint32_t *)(base + offL);
    c->tdev.H = hbm_bytes_per_gpu;
    for (int k = 0; k < 4; ++k) {
        if ((e = hipEventCreate(&c->ev[k])) != hipSuccess) {
            st = hip_fail(e, "hipEventCreate");
            alp_free(c);
            return st;
        }
    }
    // Set-up of the allocation-free entry point: the device address of this GPU's fixed scratch
    // array (the device is current here).  A failure only disables that entry point.
    void *fixed = nullptr;
    c->static_status = alp::static_scratch_address(device, &fixed);
    c->static_scratch = c->static_status == hipSuccess ? (uint8_t *)fixed : nullptr;
    *out = c;
    return ALP_OK;
}

int32_t alp_search(alp_ctx *ctx, uint32_t instance, uint32_t gpu_budget, uint32_t target_milli,
                   alp_result_t *out)
{
    if (!ctx || !out)
        return fail(ALP_EINVAL, "ctx or out is NULL");
    int32_t st = check_instance(ctx, instance);
    if (st != ALP_OK)
        return st;
    DeviceGuard guard(ctx->device);
    if (guard.status != hipSuccess)
        return hip_fail(guard.status, "hipSetDevice");
    begin_call(ctx);
    alp::QueryDev q{};
    q.inst1 = instance;
    q.cap1 = capacity_of(ctx, gpu_budget);
    q.lambda1 = target_milli;
    if ((st = run_search(ctx, q, 1)) != ALP_OK)
        return st;
    *out = ctx->host_results[0];
    return out->status == ALP_OK ? ALP_OK : ALP_INFEASIBLE;
}

int32_t alp_search_batch(alp_ctx *ctx, uint32_t count, const uint32_t *instances,
                         const uint32_t *gpu_budget, const uint32_t *target_milli,
                         alp_result_t *out)
{
    if (!ctx)
        return fail(ALP_EINVAL, "ctx is NULL");
    if (count == 0)
        return ALP_OK;
    if (!gpu_budget || !target_milli || !out)
        return fail(ALP_EINVAL, "gpu_budget, target_milli or out is NULL");
    std::vector<uint32_t> inst(count), cap(count);
    for (uint32_t i = 0; i < count; ++i) {
        inst[i] = instances ? instances[i] : i;
        int32_t st = check_instance(ctx, inst[i]);
        if (st != ALP_OK)
            return st;
        cap[i] = capacity_of(ctx, gpu_budget[i]);
    }
    DeviceGuard guard(ctx->device);
    if (guard.status != hipSuccess)
        return hip_fail(guard.status, "hipSetDevice");
    begin_call(ctx);
    alp::QueryDev q{};
    int32_t st = upload_queries(ctx, count, inst.data(), cap.data(), target_milli, q);
    if (st != ALP_OK)
        return st;
    if ((st = run_search(ctx, q, count)) != ALP_OK)
        return st;
    memcpy(out, ctx->host_results, (size_t)count * sizeof(alp_result_t));
    return ALP_OK;
}

int32_t alp_search_batch_async(alp_ctx *ctx, uint32_t count, const uint32_t *instances,
                               const uint32_t *gpu_budget, const uint32_t *target_milli,
                               alp_result_t *out)
{
    if (!ctx)
        return fail(ALP_EINVAL, "ctx is NULL");
    if (count == 0)
        return ALP_OK;
    if (!gpu_budget || !target_milli || !out)
        return fail(ALP_EINVAL, "gpu_budget, target_milli or out is NULL");
    DeviceGuard guard(ctx->device);
    if (guard.status != hipSuccess)
        return hip_fail(guard.status, "hipSetDevice");
    begin_call(ctx);
    hipError_t e;
    // q_inst holds inst | cap | lambda, then the per-item rejection flags.
    const size_t bytes = (size_t)count * sizeof(uint32_t);
    if ((e = ctx->q_inst.ensure(4 * bytes)) != hipSuccess)
        return hip_fail(e, "hipMalloc(queries)");
    uint32_t *qi = (uint32_t *)ctx->q_inst.ptr;
    alp::RawQueries raw{instances, gpu_budget, target_milli, ctx->B, ctx->space.units_per_gpu,
                        qi, qi + count, qi + 2 * (size_t)count, qi + 3 * (size_t)count};
    alp::QueryDev q{};
    q.inst = qi;
    q.capacity = qi + count;
    q.lambda = qi + 2 * (size_t)count;
    hipEvent_t *ev = nullptr;
    if (ctx->timing) {
        if (ctx->ev_spare.empty()) {
            std::array<hipEvent_t, 4> t{};
            for (auto &x : t)
                if ((e = hipEventCreate(&x)) != hipSuccess) {
                    for (auto &y : t)
                        if (y)
                            (void)hipEventDestroy(y);
                    return hip_fail(e, "hipEventCreate");
                }
            ctx->ev_spare.push_back(t);
        }
        ctx->ev_pending.push_back(ctx->ev_spare.back());
        ctx->ev_spare.pop_back();
        ev = ctx->ev_pending.back().data();
    }
    int32_t st = launch_search(ctx, q, count, out, &raw, ev);
    if (st != ALP_OK && ev) {                      // nothing (complete) was queued for them
        ctx->ev_spare.push_back(ctx->ev_pending.back());
        ctx->ev_pending.pop_back();
    } else if (ev) {
        ctx->ev_pending_terms.push_back(ctx->last_terms ? 1 : 0);
    }
    return st;
}

int32_t alp_search_batch_async_noalloc(alp_ctx *ctx, uint32_t count, const uint32_t *instances,
                                       const uint32_t *gpu_budget, const uint32_t *target_milli,
                                       alp_result_t *out)
{
    if (!ctx)
        return fail(ALP_EINVAL, "ctx is NULL");
    if (count == 0)
        return ALP_OK;
    if (!gpu_budget || !target_milli || !out)
        return fail(ALP_EINVAL, "gpu_budget, target_milli or out is NULL");
    if (!ctx->static_scratch)
        return fail(ALP_EDEVICE, "the fixed scratch array of device %d has no address: %s",
                    ctx->device, hipGetErrorString(ctx->static_status));
    // The one-launch form needs its per-item words to be 0 between launches, which a shared
    // array carved differently from call to call cannot promise: the option terms run in their
    // own kernel here, which resets what the scan needs.
    alp::ScanGeometry g;
    int32_t st = plan_scan(ctx, count, g, false);
    if (st != ALP_OK)
        return st;
    // Carve the fixed array: queries (inst | cap | lambda | rejection flags), then the search
    // scratch, each part 256-byte aligned.
    const ScratchSizes z = scratch_sizes(ctx->sp, count, g);
    auto align = [](uint64_t v) { return (v + 255) & ~UINT64_C(255); };
    const uint64_t off_q = 0, off_rec = align(off_q + 4ull * count * sizeof(uint32_t)),
                   off_ext = align(off_rec + z.rec), off_inner = align(off_ext + z.rec),
                   off_pair = align(off_inner + z.inner), off_cnt = align(off_pair + z.pair),
                   off_win = align(off_cnt + z.counters), total = off_win + z.winners;
    if (total > ALP_STATIC_SCRATCH_BYTES)
        return fail(ALP_ERANGE,
                    "%u searches need %llu bytes of scratch; the fixed array holds %u "
                    "(use alp_search_batch_async, or fewer searches per call)",
                    count, (unsigned long long)total, (unsigned)ALP_STATIC_SCRATCH_BYTES);
    DeviceGuard guard(ctx->device);
    if (guard.status != hipSuccess)
        return hip_fail(guard.status, "hipSetDevice");
    uint8_t *base = ctx->static_scratch;
    uint32_t *qi = (uint32_t *)(base + off_q);
    alp::RawQueries raw{instances, gpu_budget, target_milli, ctx->B, ctx->space.units_per_gpu,
                        qi, qi + count, qi + 2 * (size_t)count, qi + 3 * (size_t)count};
    alp::QueryDev q{};
    q.inst = qi;
    q.capacity = qi + count;
    q.lambda = qi + 2 * (size_t)count;
    SearchScratch s;
    s.rec = (uint2 *)(base + off_rec);
    s.ext = (uint2 *)(base + off_ext);
    s.inner = (uint2 *)(base + off_inner);
    s.pair = g.pair ? (uint2 *)(base + off_pair) : nullptr;
    s.done = (uint32_t *)(base + off_cnt);
    s.best = s.done + z.best_at;
    s.winners = (alp::Winner *)(base + off_win);
    return launch_search_with(ctx, q, count, out, &raw, nullptr, g, s);
}

int32_t alp_max_throughput(alp_ctx *ctx, uint32_t count, const uint32_t *instances,
                           const uint32_t *gpu_budget, uint32_t *out_tmax)
{
    if (!ctx)
        return fail(ALP_EINVAL, "ctx is NULL");
    if (count == 0)
        return ALP_OK;
    if (!gpu_budget || !out_tmax)
        return fail(ALP_EINVAL, "gpu_budget or out_tmax is NULL");
    std::vector<uint32_t> inst(count), cap(count), zero(count, 0);
    for (uint32_t i = 0; i < count; ++i) {
        inst[i] = instances ? instances[i] : i;
        int32_t st = check_instance(ctx, inst[i]);
        if (st != ALP_OK)
            return st;
        cap[i] = capacity_of(ctx, gpu_budget[i]);
    }
    DeviceGuard guard(ctx->device);
    if (guard.status != hipSuccess)
        return hip_fail(guard.status, "hipSetDevice");
    alp::QueryDev q{};
    int32_t st = upload_queries(ctx, count, inst.data(), cap.data(), zero.data(), q);
    if (st != ALP_OK)
        return st;
    hipError_t e;
    const size_t bytes = (size_t)count * sizeof(uint32_t);
    const uint64_t items_bytes = (uint64_t)count * ctx->sp.M * ctx->sp.O * sizeof(uint2);
    if ((e = ctx->tmax.ensure(bytes)) != hipSuccess || (e = ctx->rec.ensure(items_bytes)) != hipSuccess ||
        (e = ctx->ext.ensure(items_bytes)) != hipSuccess)
        return hip_fail(e, "hipMalloc(max_throughput)");
    Marked mark("alp max_throughput: option terms and reduction");
    if ((e = alp::launch_option_terms(ctx->sp, ctx->tdev, q, count, (uint2 *)ctx->rec.ptr,
                                      (uint2 *)ctx->ext.ptr, nullptr, alp::ScanReset{}, ctx->stream)) !=
        hipSuccess)
        return hip_fail(e, "option_terms launch");
    if ((e = alp::launch_tmax(ctx->sp, q, count, (const uint2 *)ctx->ext.ptr,
                              (uint32_t *)ctx->tmax.ptr, ctx->stream)) != hipSuccess)
        return hip_fail(e, "tmax launch");
    std::vector<uint32_t> host(count);
    if ((e = hipMemcpyAsync(host.data(), ctx->tmax.ptr, bytes, hipMemcpyDeviceToHost, ctx->stream)) != hipSuccess)
        return hip_fail(e, "copy results");
    if ((e = hipStreamSynchronize(ctx->stream)) != hipSuccess)
        return hip_fail(e, "hipStreamSynchronize");
    memcpy(out_tmax, host.data(), bytes);
    return ALP_OK;
}

int32_t alp_allocate_workflows(alp_ctx *ctx, uint32_t count, const uint32_t *instances,
                               const uint32_t *target_milli, uint32_t total_gpus, uint32_t policy,
                               alp_plan_t *plan, uint32_t *gpus, alp_result_t *results)
{
    if (!ctx)
        return fail(ALP_EINVAL, "ctx is NULL");
    if (count < 1 || count > 16)
        return fail(ALP_EINVAL, "count %u outside 1..16", count);
    if (total_gpus > 1024)
        return fail(ALP_EINVAL, "total_gpus %u above 1024", total_gpus);
    if (policy > ALP_WELFARE_SOCIAL)
        return fail(ALP_EINVAL, "policy %u unknown", policy);
    if (!target_milli || !plan || !gpus || !results)
        return fail(ALP_EINVAL, "target_milli, plan, gpus or results is NULL");
    const uint32_t G1 = total_gpus + 1, items = count * G1;
    std::vector<uint32_t> inst(items), cap(items), lam(items);
    for (uint32_t w = 0; w < count; ++w) {
        const uint32_t iw = instances ? instances[w] : w;
        int32_t st = check_instance(ctx, iw);
        if (st != ALP_OK)
            return st;
        for (uint32_t g = 0; g < G1; ++g) {
            inst[w * G1 + g] = iw;
            cap[w * G1 + g] = capacity_of(ctx, g);
            lam[w * G1 + g] = target_milli[w];
        }
    }
    DeviceGuard guard(ctx->device);
    if (guard.status != hipSuccess)
        return hip_fail(guard.status, "hipSetDevice");
    begin_call(ctx);
    hipError_t e;
    if (!ctx->host_split) {
        if ((e = alloc_pinned((void **)&ctx->host_split, 32 * sizeof(uint32_t), hipHostMallocMapped)) !=
            hipSuccess)
            return hip_fail(e, "hipHostMalloc(split)");
        if ((e = hipHostGetDevicePointer((void **)&ctx->host_split_dev, ctx->host_split, 0)) != hipSuccess) {
            (void)hipHostFree(ctx->host_split);
            ctx->host_split = nullptr;
            return hip_fail(e, "hipHostGetDevicePointer(split)");
        }
    }
    if ((e = ctx->split_dp.ensure((uint64_t)(count + 1) * G1 * sizeof(uint64_t) +
                                  2ull * count * G1 * sizeof(uint32_t))) != hipSuccess)
        return hip_fail(e, "hipMalloc(split)");
    alp::QueryDev q{};
    int32_t st = upload_queries(ctx, items, inst.data(), cap.data(), lam.data(), q);
    if (st != ALP_OK)
        return st;
    // All (workflow, budget) searches; run_search synchronises, so the results are complete.
    if ((st = run_search(ctx, q, items)) != ALP_OK)
        return st;
    alp_plan_t *dplan = reinterpret_cast<alp_plan_t *>(ctx->host_split_dev);
    uint32_t *dgpus = ctx->host_split_dev + 8;
    if (ctx->timing && (e = hipEventRecord(ctx->ev[2], ctx->stream)) != hipSuccess)
        return hip_fail(e, "hipEventRecord");
    Marked mark("alp allocate");
    if ((e = alp::launch_allocate(ctx->host_results_dev, count, total_gpus, policy,
                                  (uint64_t *)ctx->split_dp.ptr, dplan, dgpus, ctx->stream)) != hipSuccess)
        return hip_fail(e, "allocate launch");
    if (ctx->timing && (e = hipEventRecord(ctx->ev[3], ctx->stream)) != hipSuccess)
        return hip_fail(e, "hipEventRecord");
    if ((e = hipStreamSynchronize(ctx->stream)) != hipSuccess)
        return hip_fail(e, "hipStreamSynchronize");
    if (ctx->timing) {
        if ((e = hipEventElapsedTime(&ctx->last_ms[2], ctx->ev[2], ctx->ev[3])) != hipSuccess)
            return hip_fail(e, "hipEventElapsedTime");
        ctx->tally(2);
    }
    memcpy(plan, ctx->host_split, sizeof(alp_plan_t));
    if (plan->status != ALP_OK)
        return ALP_INFEASIBLE;
    for (uint32_t w = 0; w < count; ++w) {
        gpus[w] = ctx->host_split[8 + w];
        results[w] = ctx->host_results[w * G1 + gpus[w]];
    }
    return ALP_OK;
}

namespace {

// Step-1 vectors of F units over M LLMs without lower bounds (an upper bound of the count with
// them): partitions of F into at most M parts when ordered, else C(F + M - 1, M - 1).
// Saturating.
uint64_t pruned_vector_bound(uint32_t F, uint32_t M, bool ordered)
{
    std::vector<uint64_t> row(F + 1, 0), prev(F + 1, 0);
    if (ordered) {
        prev[0] = 1;                                   // at most 0 parts
        for (uint32_t k = 1; k <= M; ++k) {            // at most k parts
            for (uint32_t n = 0; n <= F; ++n) {
                uint64_t v = prev[n] + (n >= k ? row[n - k] : 0);
                row[n] = v < prev[n] ? UINT64_MAX : v;
            }
            prev.swap(row);
        }
        return prev[F];
    }
    // C(F + M - 1, M - 1) by Pascal's rule
    std::vector<uint64_t> c(M, 0);
    c[0] = 1;
    for (uint32_t i = 1; i <= F + M - 1; ++i)
        for (uint32_t j = std::min<uint32_t>(i, M - 1); j >= 1; --j) {
            const uint64_t v = c[j] + c[j - 1];
            c[j] = v < c[j] ? UINT64_MAX : v;
        }
    return c[M - 1];
}

}  // namespace

int32_t alp_search_pruned(alp_ctx *ctx, uint32_t count, const uint32_t *instances,
                          const uint32_t *gpu_budget, const uint32_t *target_milli, uint32_t flags,
                          alp_pruned_t *out)
{
    if (!ctx)
        return fail(ALP_EINVAL, "ctx is NULL");
    if (flags > (ALP_PRUNE_ORDER | ALP_PRUNE_MIN_FRACTION))
        return fail(ALP_EINVAL, "flags 0x%x unknown", flags);
    if (count == 0)
        return ALP_OK;
    if (!gpu_budget || !target_milli || !out)
        return fail(ALP_EINVAL, "gpu_budget, target_milli or out is NULL");
    const alp::SpaceDev &sp = ctx->sp;
    std::vector<uint32_t> inst(count), cap(count);
    uint32_t F_max = 0;
    for (uint32_t i = 0; i < count; ++i) {
        inst[i] = instances ? instances[i] : i;
        int32_t st = check_instance(ctx, inst[i]);
        if (st != ALP_OK)
            return st;
        const uint64_t F = (uint64_t)sp.Q * gpu_budget[i];
        if (F > ALP_PRUNED_MAX_UNITS)
            return fail(ALP_EINVAL, "query %u: Q*G = %llu above %u for the pruned search", i,
                        (unsigned long long)F, ALP_PRUNED_MAX_UNITS);
        cap[i] = (uint32_t)F;
        F_max = std::max(F_max, cap[i]);
    }
    // the bound grows with the number of units: checking the largest query covers all
    if (pruned_vector_bound(F_max, sp.M, flags & ALP_PRUNE_ORDER) > ALP_PRUNED_MAX_VECTORS)
        return fail(ALP_ERANGE, "Q*G = %u: more than 2^34 fraction vectors per query", F_max);
    const uint64_t F1 = (uint64_t)F_max + 1;
    const uint32_t bpi = (uint32_t)ceil_div(alp::pruned_prefixes(sp.M, F_max), 256);
    const uint64_t nblocks = (uint64_t)count * bpi;
    if (nblocks >= (UINT64_C(1) << 31))
        return fail(ALP_ERANGE, "batch too large for one launch (%llu blocks)",
                    (unsigned long long)nblocks);
    DeviceGuard guard(ctx->device);
    if (guard.status != hipSuccess)
        return hip_fail(guard.status, "hipSetDevice");
    begin_call(ctx);
    const uint64_t items_bytes = (uint64_t)count * sp.M * sp.O * sizeof(uint2);
    hipError_t e;
    if ((e = ctx->rec.ensure(items_bytes)) != hipSuccess || (e = ctx->ext.ensure(items_bytes)) != hipSuccess ||
        (e = ctx->inner.ensure((uint64_t)count * alp::inner_stride(sp.O) * sizeof(uint2))) != hipSuccess ||
        (e = ctx->done.ensure((uint64_t)count * sizeof(uint32_t))) != hipSuccess ||
        (e = ctx->winners.ensure(nblocks * sizeof(alp::Winner))) != hipSuccess ||
        (e = ctx->pruned_counts.ensure(nblocks * sizeof(uint64_t))) != hipSuccess ||
        (e = ctx->pruned_table.ensure((uint64_t)count * sp.M * sp.Q * F1 * sizeof(uint64_t))) != hipSuccess ||
        (e = ctx->pruned_orders.ensure((uint64_t)count * alp::pruned_order_bytes())) != hipSuccess)
        return hip_fail(e, "hipMalloc(pruned search)");
    if (count > ctx->host_pruned_cap) {
        void *grown = nullptr, *grown_dev = nullptr;
        if ((e = alloc_pinned(&grown, count * sizeof(alp_pruned_t), hipHostMallocMapped)) !=
            hipSuccess)
            return hip_fail(e, "hipHostMalloc(pruned results)");
        if ((e = hipHostGetDevicePointer(&grown_dev, grown, 0)) != hipSuccess) {
            (void)hipHostFree(grown);
            return hip_fail(e, "hipHostGetDevicePointer(pruned results)");
        }
        if (ctx->host_pruned)
            (void)hipHostFree(ctx->host_pruned);
        ctx->host_pruned = (alp_pruned_t *)grown;
        ctx->host_pruned_dev = (alp_pruned_t *)grown_dev;
        ctx->host_pruned_cap = count;
    }
    alp::QueryDev q{};
    int32_t st = upload_queries(ctx, count, inst.data(), cap.data(), target_milli, q);
    if (st != ALP_OK)
        return st;
    uint2 *rec = (uint2 *)ctx->rec.ptr, *ext = (uint2 *)ctx->ext.ptr;
    uint32_t *done = (uint32_t *)ctx->done.ptr;
    if (ctx->timing && (e = hipEventRecord(ctx->ev[0], ctx->stream)) != hipSuccess)
        return hip_fail(e, "hipEventRecord");
    alp::ScanReset reset;
    reset.done = done;                       // the pruned scan publishes every block's winner
    Marked mark("alp pruned search: option terms, table and scan");
    if ((e = alp::launch_option_terms(sp, ctx->tdev, q, count, rec, ext, (uint2 *)ctx->inner.ptr,
                                      reset, ctx->stream)) != hipSuccess)
        return hip_fail(e, "option_terms launch");
    if (ctx->timing && (e = hipEventRecord(ctx->ev[1], ctx->stream)) != hipSuccess)
        return hip_fail(e, "hipEventRecord");
    if ((e = alp::launch_pruned_table(sp, ctx->tdev, q, count, F_max, flags, rec,
                                      (uint64_t *)ctx->pruned_table.ptr, ctx->pruned_orders.ptr,
                                      ctx->stream)) != hipSuccess)
        return hip_fail(e, "pruned table launch");
    if (ctx->timing && (e = hipEventRecord(ctx->ev[2], ctx->stream)) != hipSuccess)
        return hip_fail(e, "hipEventRecord");
    if ((e = alp::launch_pruned_scan(sp, count, F_max, flags,
                                     (const uint64_t *)ctx->pruned_table.ptr, ctx->pruned_orders.ptr, bpi,
                                     (alp::Winner *)ctx->winners.ptr,
                                     (uint64_t *)ctx->pruned_counts.ptr, ext, done,
                                     ctx->host_pruned_dev, ctx->stream)) != hipSuccess)
        return hip_fail(e, "pruned scan launch");
    if (ctx->timing && (e = hipEventRecord(ctx->ev[3], ctx->stream)) != hipSuccess)
        return hip_fail(e, "hipEventRecord");
    if ((e = hipStreamSynchronize(ctx->stream)) != hipSuccess)
        return hip_fail(e, "hipStreamSynchronize");
    if (ctx->timing) {
        // ms[0]: option terms, ms[1]: fraction enumeration, ms[2]: admissible-option table
        if ((e = hipEventElapsedTime(&ctx->last_ms[0], ctx->ev[0], ctx->ev[1])) != hipSuccess ||
            (e = hipEventElapsedTime(&ctx->last_ms[2], ctx->ev[1], ctx->ev[2])) != hipSuccess ||
            (e = hipEventElapsedTime(&ctx->last_ms[1], ctx->ev[2], ctx->ev[3])) != hipSuccess)
            return hip_fail(e, "hipEventElapsedTime");
        for (int k = 0; k < 3; ++k)
            ctx->tally(k);
    }
    ctx->last_blocks = (uint32_t)nblocks;
    memcpy(out, ctx->host_pruned, count * sizeof(alp_pruned_t));
    return ALP_OK;
}

int32_t alp_place(alp_ctx *ctx, uint32_t count, const alp_result_t *allocations,
                  const uint32_t *gpu_budget, alp_placement_t *out)
{
    if (!ctx)
        return fail(ALP_EINVAL, "ctx is NULL");
    if (count == 0)
        return ALP_OK;
    if (!allocations || !gpu_budget || !out)
        return fail(ALP_EINVAL, "allocations, gpu_budget or out is NULL");
    const alp_space_t &sp = ctx->space;
    // Budgets of at most 16 GPUs first (four to a wave), then the others.
    std::vector<alp::PlaceIn> in(count);
    uint32_t small = 0;
    for (uint32_t i = 0; i < count; ++i)
        small += gpu_budget[i] <= 16;
    uint32_t next_small = 0, next_large = small;
    for (uint32_t i = 0; i < count; ++i) {
        const alp_result_t &r = allocations[i];
        if (gpu_budget[i] > ALP_PLACE_MAX_GPUS)
            return fail(ALP_EINVAL, "allocation %u: %u GPUs, at most %u", i, gpu_budget[i],
                        ALP_PLACE_MAX_GPUS);
        alp::PlaceIn &p = in[gpu_budget[i] <= 16 ? next_small++ : next_large++];
        memset(&p, 0, sizeof(p));
        p.dst = i;
        p.gpus = (uint8_t)gpu_budget[i];
        p.llms = (uint8_t)sp.num_llms;
        p.feasible = r.status == ALP_OK;
        if (!p.feasible)
            continue;
        for (uint32_t m = 0; m < sp.num_llms; ++m) {
            bool tp_ok = false, q_ok = false;
            for (uint32_t j = 0; j < sp.num_tp; ++j)
                tp_ok |= r.tp[m] == sp.tp_values[j];
            for (uint32_t j = 0; j < sp.num_frac; ++j)
                q_ok |= r.frac_units[m] == sp.frac_units[j];
            if (!tp_ok || !q_ok || r.tp[m] > ALP_NODE_GPUS || r.replicas[m] < 1 ||
                r.replicas[m] > sp.max_replicas)
                return fail(ALP_EINVAL, "allocation %u: LLM %u's choice is not of the space", i, m);
            p.tp[m] = r.tp[m];
            p.q[m] = r.frac_units[m];
            p.d[m] = r.replicas[m];
        }
    }
    DeviceGuard guard(ctx->device);
    if (guard.status != hipSuccess)
        return hip_fail(guard.status, "hipSetDevice");
    begin_call(ctx);
    hipError_t e;
    if ((e = ctx->place_in.ensure(count * sizeof(alp::PlaceIn))) != hipSuccess ||
        (e = ctx->place_out.ensure(count * sizeof(alp_placement_t))) != hipSuccess)
        return hip_fail(e, "hipMalloc(placement)");
    if (ctx->timing && (e = hipEventRecord(ctx->ev[0], ctx->stream)) != hipSuccess)
        return hip_fail(e, "hipEventRecord");
    if ((e = hipMemcpyAsync(ctx->place_in.ptr, in.data(), count * sizeof(alp::PlaceIn),
                            hipMemcpyHostToDevice, ctx->stream)) != hipSuccess)
        return hip_fail(e, "copy allocations");
    if (ctx->timing && (e = hipEventRecord(ctx->ev[1], ctx->stream)) != hipSuccess)
        return hip_fail(e, "hipEventRecord");
    Marked mark("alp place");
    if ((e = alp::launch_place(sp.units_per_gpu, small, count - small,
                               (const alp::PlaceIn *)ctx->place_in.ptr,
                               (alp_placement_t *)ctx->place_out.ptr, ctx->stream)) != hipSuccess)
        return hip_fail(e, "placement launch");
    if (ctx->timing && (e = hipEventRecord(ctx->ev[2], ctx->stream)) != hipSuccess)
        return hip_fail(e, "hipEventRecord");
    if ((e = hipMemcpyAsync(out, ctx->place_out.ptr, count * sizeof(alp_placement_t),
                            hipMemcpyDeviceToHost, ctx->stream)) != hipSuccess ||
        (e = hipStreamSynchronize(ctx->stream)) != hipSuccess)
        return hip_fail(e, "placement");
    if (ctx->timing) {
        // ms[1]: the placement kernel
        if ((e = hipEventElapsedTime(&ctx->last_ms[1], ctx->ev[1], ctx->ev[2])) != hipSuccess)
            return hip_fail(e, "hipEventElapsedTime");
        ctx->last_ms[0] = ctx->last_ms[2] = 0.0f;
        ctx->tally(1);
    }
    return ALP_OK;
}

int32_t alp_eval_candidates(alp_ctx *ctx, uint32_t instance, uint32_t gpu_budget,
                            uint32_t target_milli, const uint64_t *indices, uint64_t count,
                            alp_eval_t *out)
{
    if (!ctx)
        return fail(ALP_EINVAL, "ctx is NULL");
    int32_t st = check_instance(ctx, instance);
    if (st != ALP_OK)
        return st;
    if (count == 0)
        return ALP_OK;
    if (!indices || !out)
        return fail(ALP_EINVAL, "indices or out is NULL");
    for (uint64_t i = 0; i < count; ++i)
        if (indices[i] >= ctx->N)
            return fail(ALP_EINVAL, "indices[%llu]=%llu outside the %llu candidates",
                        (unsigned long long)i, (unsigned long long)indices[i],
                        (unsigned long long)ctx->N);
    DeviceGuard guard(ctx->device);
    if (guard.status != hipSuccess)
        return hip_fail(guard.status, "hipSetDevice");
    hipError_t e;
    const uint64_t item_bytes = (uint64_t)ctx->sp.M * ctx->sp.O * sizeof(uint2);
    if ((e = ctx->rec.ensure(item_bytes)) != hipSuccess || (e = ctx->ext.ensure(item_bytes)) != hipSuccess ||
        (e = ctx->idx.ensure(count * sizeof(uint64_t))) != hipSuccess ||
        (e = ctx->evals.ensure(count * sizeof(alp_eval_t))) != hipSuccess)
        return hip_fail(e, "hipMalloc(eval)");
    alp::QueryDev q{};
    q.inst1 = instance;
    q.cap1 = capacity_of(ctx, gpu_budget);
    q.lambda1 = target_milli;
    if ((e = hipMemcpyAsync(ctx->idx.ptr, indices, count * sizeof(uint64_t), hipMemcpyHostToDevice,
                            ctx->stream)) != hipSuccess)
        return hip_fail(e, "copy indices");
    Marked mark("alp evaluate");
    if ((e = alp::launch_option_terms(ctx->sp, ctx->tdev, q, 1, (uint2 *)ctx->rec.ptr,
                                      (uint2 *)ctx->ext.ptr, nullptr, alp::ScanReset{}, ctx->stream)) !=
        hipSuccess)
        return hip_fail(e, "option_terms launch");
    if ((e = alp::launch_eval(ctx->sp, q.cap1, (const uint2 *)ctx->rec.ptr, (const uint2 *)ctx->ext.ptr,
                              (const uint64_t *)ctx->idx.ptr, count, (alp_eval_t *)ctx->evals.ptr,
                              ctx->stream)) != hipSuccess)
        return hip_fail(e, "eval launch");
    if ((e = hipMemcpyAsync(out, ctx->evals.ptr, count * sizeof(alp_eval_t), hipMemcpyDeviceToHost,
                            ctx->stream)) != hipSuccess)
        return hip_fail(e, "copy evaluations");
    if ((e = hipStreamSynchronize(ctx->stream)) != hipSuccess)
        return hip_fail(e, "hipStreamSynchronize");
    return ALP_OK;
}

int32_t alp_set_launch(alp_ctx *ctx, uint32_t variant, uint32_t blocks_per_item,
                       uint32_t threads_per_block, uint32_t inner_chunks)
{
    if (!ctx)
        return fail(ALP_EINVAL, "ctx is NULL");
    const uint32_t base_variant = variant & ~ALP_LAUNCH_SEPARATE_TERMS;
    if (base_variant > 6 || ((variant & ALP_LAUNCH_SEPARATE_TERMS) && base_variant != 0 &&
                             base_variant != 1 && base_variant != 4 && base_variant != 5))
        return fail(ALP_EINVAL, "variant %u is not one of 0..6, or 0, 1, 4, 5 with "
                                "ALP_LAUNCH_SEPARATE_TERMS", variant);
    if (threads_per_block && (threads_per_block % 64 || threads_per_block > 1024))
        return fail(ALP_EINVAL, "threads_per_block must be a multiple of 64, at most 1024");
    if (blocks_per_item > (1u << 24))
        return fail(ALP_EINVAL, "blocks_per_item too large");
    // inner_chunks must divide the inner table's groups of 16 records (the pair table's, for
    // variant 6); the planner uses it only where it divides the table the launch scans.
    const uint32_t n16 = alp::inner_stride(ctx->sp.O) / 16;
    const uint32_t p16 = alp::pair_stride(ctx->sp.O) / 16;
    const uint32_t d16 = base_variant == 6 ? p16 : n16;
    if (inner_chunks && (inner_chunks > d16 || d16 % inner_chunks))
        return fail(ALP_EINVAL, "inner_chunks %u does not divide %u", inner_chunks, d16);
    ctx->variant = variant;
    ctx->bpi_override = blocks_per_item;
    ctx->tpb_override = threads_per_block;
    ctx->chunks_override = inner_chunks;
    return ALP_OK;
}

int32_t alp_set_timing(alp_ctx *ctx, int32_t enable)
{
    if (!ctx)
        return fail(ALP_EINVAL, "ctx is NULL");
    if (enable < 0)
        return fail(ALP_EINVAL, "enable %d is negative", enable);
    int32_t st = collect_async_times(ctx);
    if (st != ALP_OK)
        return st;
    for (int k = 0; k < 3; ++k)
        ctx->total_ms[k] = 0.0;
    ctx->timing_every = (uint32_t)enable;
    ctx->calls_seen = ctx->timed_calls = 0;
    ctx->timing = 0;
    return ALP_OK;
}

int32_t alp_kernel_time_totals(alp_ctx *ctx, double ms[3], uint64_t *timed_calls)
{
    if (!ctx || !ms)
        return fail(ALP_EINVAL, "ctx or ms is NULL");
    int32_t st = collect_async_times(ctx);
    if (st != ALP_OK)
        return st;
    for (int k = 0; k < 3; ++k)
        ms[k] = ctx->total_ms[k];
    if (timed_calls)
        *timed_calls = ctx->timed_calls;
    return ALP_OK;
}

int32_t alp_kernel_times(alp_ctx *ctx, float ms[3], uint32_t *scan_blocks)
{
    if (!ctx || !ms)
        return fail(ALP_EINVAL, "ctx or ms is NULL");
    int32_t st = collect_async_times(ctx);
    if (st != ALP_OK)
        return st;
    for (int k = 0; k < 3; ++k)
        ms[k] = ctx->last_ms[k];
    if (scan_blocks)
        *scan_blocks = ctx->last_blocks;
    return ALP_OK;
}

int32_t alp_num_candidates(const alp_ctx *ctx, uint64_t *out)
{
    if (!ctx || !out)
        return fail(ALP_EINVAL, "ctx or out is NULL");
    *out = ctx->N;
    return ALP_OK;
}

void alp_free(alp_ctx *ctx)
{
    if (!ctx)
        return;
    DeviceGuard guard(ctx->device);
    (void)hipStreamSynchronize(ctx->stream);           // queued asynchronous searches included
    for (int k = 0; k < 4; ++k)
        if (ctx->ev[k])
            (void)hipEventDestroy(ctx->ev[k]);
    for (auto *list : {&ctx->ev_pending, &ctx->ev_spare})
        for (auto &t : *list)
            for (hipEvent_t x : t)
                (void)hipEventDestroy(x);
    DevBuf *bufs[] = {&ctx->tables, &ctx->q_inst, &ctx->rec, &ctx->ext, &ctx->inner, &ctx->done,
                      &ctx->winners, &ctx->idx, &ctx->evals, &ctx->tmax, &ctx->split_dp,
                      &ctx->pruned_table, &ctx->pruned_orders, &ctx->pruned_counts,
                      &ctx->place_in, &ctx->place_out, &ctx->pair, &ctx->fused_regions,
                      &ctx->fused_words};
    for (DevBuf *b : bufs)
        b->release();
    if (ctx->host_results)
        (void)hipHostFree(ctx->host_results);
    if (ctx->host_signal)
        (void)hipHostFree(ctx->host_signal);
    if (ctx->host_query)
        (void)hipHostFree(ctx->host_query);
    if (ctx->host_split)
        (void)hipHostFree(ctx->host_split);
    if (ctx->host_pruned)
        (void)hipHostFree(ctx->host_pruned);
    delete ctx;
}

struct alp_stats_ctx {
    int device = 0;
    hipStream_t stream = nullptr;
    DevBuf totals, long_list, long_base, scratch, work;
    alp_stats_t *host_out = nullptr;        // mapped pinned: results, then the StatsTail
    alp_stats_t *host_out_dev = nullptr;
    // Whether the device totals and counters are zero (the kernels leave them so); false for
    // fresh memory and after a failed launch, when the next call zeroes them first.
    bool counters_clean = false;
    uint64_t *offsets = nullptr;            // pinned: the trace offsets, read for planning
    size_t offsets_cap = 0;                 // entries
    int timing = 0;
    hipEvent_t ev[2] = {nullptr, nullptr};
    float last_ms = 0.0f;
    // Calls left that sort every trace without the end-order sweep: set when a sweep found most
    // traces out of end order (each such trace is then loaded twice), counted down per call, so
    // that every kStatsProbeEvery-th call measures the order again.
    uint32_t direct_left = 0;
};

constexpr uint32_t kStatsProbeEvery = 8;

int32_t alp_stats_create(alp_stats_ctx **out, int32_t device, void *hip_stream)
{
    if (!out)
        return fail(ALP_EINVAL, "out is NULL");
    *out = nullptr;
    alp_stats_ctx *c = new (std::nothrow) alp_stats_ctx;
    if (!c)
        return fail(ALP_ENOMEM, "context allocation");
    c->device = device;
    c->stream = (hipStream_t)hip_stream;
    DeviceGuard guard(device);
    hipError_t e = guard.status;
    if (e == hipSuccess)
        e = alloc_pinned((void **)&c->host_out, (ALP_MAX_LLMS + 1) * sizeof(alp_stats_t),
                         hipHostMallocMapped);
    if (e == hipSuccess)
        e = hipHostGetDevicePointer((void **)&c->host_out_dev, c->host_out, 0);
    for (int k = 0; k < 2 && e == hipSuccess; ++k)
        e = hipEventCreate(&c->ev[k]);
    if (e == hipSuccess)
        e = c->totals.ensure((alp::kStatsTotalsWords + alp::kStatsTailWords) * sizeof(uint64_t));
    if (e != hipSuccess) {
        alp_stats_free(c);
        return hip_fail(e, "statistics context");
    }
    *out = c;
    return ALP_OK;
}

int32_t alp_trace_stats(alp_stats_ctx *c, uint32_t num_llms, uint32_t num_traces,
                        const uint64_t *offsets, const uint32_t *llm, const uint64_t *start_us,
                        const uint64_t *end_us, alp_stats_t *out)
{
    constexpr uint64_t kMaxTrace = 1ull << 24, kLdsMax = 2048;   // 2 x 2048 x 8 B of LDS
    if (!c || !offsets || !out)
        return fail(ALP_EINVAL, "ctx, offsets or out is NULL");
    if (num_llms < 1 || num_llms > ALP_MAX_LLMS)
        return fail(ALP_EINVAL, "num_llms %u outside 1..%d", num_llms, ALP_MAX_LLMS);
    if (num_traces < 1 || num_traces >= (1u << 31))
        return fail(ALP_EINVAL, "num_traces %u outside 1..2^31-1", num_traces);
    DeviceGuard guard(c->device);
    if (guard.status != hipSuccess)
        return hip_fail(guard.status, "hipSetDevice");
    hipError_t e;
    const size_t n_off = (size_t)num_traces + 1;
    if (c->offsets_cap < n_off) {
        // Pinned, so the copy goes straight to it (no staging through a bounce buffer).
        void *grown = nullptr;
        if ((e = alloc_pinned(&grown, n_off * sizeof(uint64_t), hipHostMallocDefault)) !=
            hipSuccess)
            return hip_fail(e, "hipHostMalloc(offsets)");
        if (c->offsets)
            (void)hipHostFree(c->offsets);
        c->offsets = (uint64_t *)grown;
        c->offsets_cap = n_off;
    }
    if ((e = hipMemcpyAsync(c->offsets, offsets, n_off * sizeof(uint64_t),
                            hipMemcpyDeviceToHost, c->stream)) != hipSuccess ||
        (e = hipStreamSynchronize(c->stream)) != hipSuccess)
        return hip_fail(e, "copy offsets");
    if (c->offsets[0] != 0)
        return fail(ALP_EINVAL, "offsets[0] = %llu, not 0", (unsigned long long)c->offsets[0]);
    std::vector<uint32_t> longs;
    std::vector<uint64_t> bases;
    uint64_t max_short = 0, scratch_pairs = 0;
    for (uint32_t r = 0; r < num_traces; ++r) {
        if (c->offsets[r + 1] < c->offsets[r])
            return fail(ALP_EINVAL, "offsets decrease at trace %u", r);
        const uint64_t n = c->offsets[r + 1] - c->offsets[r];
        if (n > kMaxTrace)
            return fail(ALP_ERANGE, "trace %u has %llu calls (at most 2^24)", r, (unsigned long long)n);
        if (n > kLdsMax) {
            uint64_t P = 256;
            while (P < n)
                P <<= 1;
            longs.push_back(r);
            bases.push_back(scratch_pairs);
            scratch_pairs += P;
        } else if (n > max_short) {
            max_short = n;
        }
    }
    if (c->offsets[num_traces] > 0 && (!llm || !start_us || !end_us))
        return fail(ALP_EINVAL, "llm, start_us or end_us is NULL");
    uint32_t lds_cap = 256;
    while (lds_cap < max_short)
        lds_cap <<= 1;
    if (!longs.empty()) {
        if ((e = c->long_list.ensure(longs.size() * sizeof(uint32_t))) != hipSuccess ||
            (e = c->long_base.ensure(bases.size() * sizeof(uint64_t))) != hipSuccess ||
            (e = c->scratch.ensure(scratch_pairs * 2 * sizeof(uint64_t))) != hipSuccess)
            return hip_fail(e, "hipMalloc(statistics scratch)");
        if ((e = hipMemcpyAsync(c->long_list.ptr, longs.data(), longs.size() * sizeof(uint32_t),
                                hipMemcpyHostToDevice, c->stream)) != hipSuccess ||
            (e = hipMemcpyAsync(c->long_base.ptr, bases.data(), bases.size() * sizeof(uint64_t),
                                hipMemcpyHostToDevice, c->stream)) != hipSuccess)
            return hip_fail(e, "copy long traces");
    }
    if ((e = c->work.ensure((uint64_t)num_traces * sizeof(uint32_t))) != hipSuccess)
        return hip_fail(e, "hipMalloc(statistics work list)");
    uint64_t *totals = (uint64_t *)c->totals.ptr;
    const bool sweep = c->direct_left == 0;
    if (!sweep)
        --c->direct_left;
    if (c->timing && (e = hipEventRecord(c->ev[0], c->stream)) != hipSuccess)
        return hip_fail(e, "hipEventRecord");
    const bool zero_first = !c->counters_clean;
    c->counters_clean = false;                       // until the kernels have run to the end
    Marked mark("alp trace statistics");
    if ((e = alp::launch_trace_stats(num_llms, num_traces, offsets, llm, start_us, end_us, lds_cap,
                                     (uint32_t)max_short, (uint32_t)longs.size(), (const uint32_t *)c->long_list.ptr,
                                     (const uint64_t *)c->long_base.ptr, (uint64_t *)c->scratch.ptr,
                                     totals, (uint32_t *)c->work.ptr, sweep, zero_first,
                                     c->host_out_dev, c->stream)) != hipSuccess)
        return hip_fail(e, "statistics launch");
    if (c->timing && (e = hipEventRecord(c->ev[1], c->stream)) != hipSuccess)
        return hip_fail(e, "hipEventRecord");
    if ((e = hipStreamSynchronize(c->stream)) != hipSuccess)
        return hip_fail(e, "statistics");
    c->counters_clean = true;
    // The status and the work list's length, written by the last block after the records.
    alp::StatsTail tail;
    memcpy(&tail, c->host_out + ALP_MAX_LLMS, sizeof(tail));
    const uint32_t host_flags = tail.flags;
    const uint64_t short_traces = num_traces - longs.size();
    if (sweep && 2 * (uint64_t)tail.listed > short_traces)
        c->direct_left = kStatsProbeEvery - 1;
    if (c->timing && (e = hipEventElapsedTime(&c->last_ms, c->ev[0], c->ev[1])) != hipSuccess)
        return hip_fail(e, "hipEventElapsedTime");
    if (host_flags & 1u)
        return fail(ALP_EINVAL, "a call's llm index is not below num_llms");
    if (host_flags & 2u)
        return fail(ALP_EINVAL, "a call ends before it starts");
    if (host_flags & 4u)
        return fail(ALP_ERANGE, "a start time of 2^60 us or more, or a duration of 2^32 us or more");
    if (host_flags & 8u)
        return fail(ALP_ERANGE, "n or p of 2^31 thousandths or more");
    memcpy(out, c->host_out, num_llms * sizeof(alp_stats_t));
    return ALP_OK;
}

int32_t alp_stats_set_timing(alp_stats_ctx *ctx, int32_t enable)
{
    if (!ctx)
        return fail(ALP_EINVAL, "ctx is NULL");
    ctx->timing = enable ? 1 : 0;
    return ALP_OK;
}

int32_t alp_stats_time(alp_stats_ctx *ctx, float *ms)
{
    if (!ctx || !ms)
        return fail(ALP_EINVAL, "ctx or ms is NULL");
    *ms = ctx->last_ms;
    return ALP_OK;
}

void alp_stats_free(alp_stats_ctx *c)
{
    if (!c)
        return;
    DeviceGuard guard(c->device);
    if (c->stream)
        (void)hipStreamSynchronize(c->stream);
    else
        (void)hipDeviceSynchronize();
    for (int k = 0; k < 2; ++k)
        if (c->ev[k])
            (void)hipEventDestroy(c->ev[k]);
    DevBuf *bufs[] = {&c->totals, &c->long_list, &c->long_base, &c->scratch, &c->work};
    for (DevBuf *b : bufs)
        b->release();
    if (c->host_out)
        (void)hipHostFree(c->host_out);
    if (c->offsets)
        (void)hipHostFree(c->offsets);
    delete c;
}

const char *alp_status_str(int32_t status)
{
    switch (status) {
    case ALP_OK: return "ALP_OK";
    case ALP_EINVAL: return "ALP_EINVAL";
    case ALP_ERANGE: return "ALP_ERANGE";
    case ALP_ENOMEM: return "ALP_ENOMEM";
    case ALP_EDEVICE: return "ALP_EDEVICE";
    case ALP_INFEASIBLE: return "ALP_INFEASIBLE";
    default: return "ALP_UNKNOWN";
    }
}

const char *alp_last_error(void) { return g_last_error; }

}  // extern "C"
