// Internal declarations shared by the ABI layer (alp_api.hip) and the gfx950 kernels
// (alp_kernels.hip).  Not installed; the public interface is include/alp.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "alp.h"

namespace alp {

// Share-unit value stored for an option that cannot be used at the query's target (not
// deployable, weights do not fit, or the replica load exceeds saturation).  Real share units
// are at most 64 * 16 * 16 = 16384 per LLM and 131072 per candidate, budgets are clamped
// below the sentinel, so any candidate containing such an option fails the budget test.
constexpr uint32_t kSentinelUnits = 1u << 24;
constexpr uint32_t kCapacityMax = kSentinelUnits - 1;
constexpr uint32_t kNoLatency = 0xFFFFFFFFu;

// Search-space shape passed by value to kernels.  mul_O and mul_D are the multipliers of
// div_by(): ceil(2^32 / O) and ceil(2^32 / D), 0 for a divisor of 1.  The tensor-parallel
// degrees (at most 64) and GPU shares (at most 16 units) are bytes of tp8 and fq8 (byte i the
// i-th value), so that a lane picks its own by a shift: a by-value array indexed differently
// by different lanes is read from the kernel-argument memory, one slow round trip.
struct SpaceDev {
    uint32_t M, n_tp, n_fq, D, K, Q, O;
    uint32_t mul_O, mul_D;
    uint64_t tp8, fq8;
    __host__ __device__ uint32_t tp(uint32_t i) const { return (uint32_t)(tp8 >> (8 * i)) & 0xFFu; }
    __host__ __device__ uint32_t fq(uint32_t j) const { return (uint32_t)(fq8 >> (8 * j)) & 0xFFu; }
};

// The multiplier div_by() takes for divisor v (1 <= v < 2^32).
__host__ __device__ inline uint32_t div_multiplier(uint32_t v)
{
    return v > 1 ? (uint32_t)((UINT64_C(0xFFFFFFFF) + v) / v) : 0u;
}

// floor(a / v) for a * v < 2^32, given mul = div_multiplier(v): with mul = (2^32 + e) / v,
// 0 <= e < v, a * mul / 2^32 = a / v + a e / (v 2^32) and the added part is below 1 / v, less
// than the distance from a / v to the next integer.
__host__ __device__ inline uint32_t div_by(uint32_t a, uint32_t mul)
{
    return mul ? (uint32_t)(((uint64_t)a * mul) >> 32) : a;
}

// Device copies of the profile tables of all instances (layouts as in alp_load_profiles).
struct TablesDev {
    const uint64_t *W;
    const uint32_t *n;
    const uint32_t *p;
    const uint8_t *allowed;
    const uint32_t *rate;
    const uint32_t *lat;
    uint64_t H;
};

// Per-item query: device arrays for batches, or by-value scalars for a single query.
// The three arrays are set together or not at all.
struct QueryDev {
    const uint32_t *inst;       // instance of item i, or nullptr -> inst1
    const uint32_t *capacity;   // share-unit capacity Q*G of item i (clamped), or nullptr -> cap1
    const uint32_t *lambda;     // target rate of item i, or nullptr -> lambda1
    uint32_t inst1, cap1, lambda1;
};

// Records per item of the inner-LLM table: options rounded up to a multiple of 16.
__host__ __device__ inline uint32_t inner_stride(uint32_t O) { return (O + 15u) & ~15u; }
// Records per item of the pair table (LLMs M-3 and M-2 folded into one inner LLM of O^2
// options), padded to 16.
__host__ __device__ inline uint32_t pair_stride(uint32_t O) { return (O * O + 15u) & ~15u; }

// Per-block winner of a scan: lexicographic (L, x) minimum; L = kNoLatency if none.
struct Winner {
    uint32_t L;
    uint32_t pad;
    uint64_t x;
};

// The scan kernels write alp_result_t as six 64-bit words in this field order.
static_assert(sizeof(alp_result_t) == 48, "alp_result_t layout");
static_assert(offsetof(alp_result_t, latency_us) == 8 && offsetof(alp_result_t, throughput_milli) == 12 &&
                  offsetof(alp_result_t, gpu_units) == 16 && offsetof(alp_result_t, status) == 20 &&
                  offsetof(alp_result_t, tp) == 24 && offsetof(alp_result_t, frac_units) == 32 &&
                  offsetof(alp_result_t, replicas) == 40,
              "alp_result_t layout");

// What the last block of an item needs to produce the item's result.
struct FinishArgs {
    SpaceDev sp;
    const uint2 *ext;          // per-option (tau, u | flags) of the query
    uint32_t *done;            // per-item finished-block counter, zeroed by the option-term kernel
    uint32_t *best;            // per-item smallest block latency seen so far (atomic minimum),
                               // kNoLatency from the option-term kernel
    alp_result_t *out;         // per-item results (device-visible, may be mapped host memory)
    const uint32_t *invalid;   // per-item: nonzero = the query was rejected (result EINVAL);
                               // nullptr = every query valid
    // A search of one item whose caller waits for its record in host memory: once the record is
    // written, seq is stored to *signal (mapped host memory) with a release at system scope, so
    // a host that reads seq there also reads the whole record.  nullptr: no signal.
    uint32_t *signal = nullptr;
    uint32_t seq = 0;
};

// Launch geometry of one scan.
struct ScanGeometry {
    uint32_t variant;          // 1: row-minimum, 2: thread-per-candidate, 3: exact-tracking lanes
    uint32_t threads;          // per block
    uint32_t blocks_per_item;
    uint64_t rows;             // variants 1, 3: rows of O prefixes per item (variant 1: sub-rows,
                               // rows times chunks)
    uint64_t rows_per_wave;    // variants 1, 3
    uint32_t chunks;           // variant 1: ranges of the inner LLM's records per row
    uint32_t dynamic;          // variant 1: sub-rows handed out within each block (1) or fixed
                               // per wave (0, requires chunks == 1)
    uint64_t per_thread;       // variant 2: candidates per thread
    uint32_t slots;            // variants 1, 3: options of the last LLM per lane (1, 2, 4, 8)
    uint32_t pair;             // variant 1: the inner table is the pair table (rows fix M - 3
                               // digits, O^2 records each)
    uint32_t fused;            // variant 1: one launch -- every block computes its item's option
                               // terms itself, and the item's winner is one 64-bit word (spaces of
                               // fewer than 2^32 candidates, never with the pair table)
};

// Queries of a search batch given in device memory, prepared by the option-term kernel: item i
// searches instance inst[i] (i when inst is nullptr; one >= B is rejected and searched as
// instance 0), capacity min(units_per_gpu * budget[i], kCapacityMax), target target[i].  The
// kernel writes the prepared arrays (the QueryDev the scan reads) and the rejection flags.
struct RawQueries {
    const uint32_t *inst, *budget, *target;
    uint32_t B, units_per_gpu;
    uint32_t *q_inst, *q_cap, *q_lambda, *invalid;
};

// The one-launch form of the scan (ScanGeometry::fused): each block computes the option terms
// of its item from the tables into its own region of device memory and reads them back through
// the scalar cache; the item's best candidate so far is the word best[item] = ~(L << 32 | x)
// (x < 2^32), raised by an atomic maximum, 0 for none; done[item] counts finished blocks.  The
// last block of an item resets both words to 0, so they are 0 between launches (the host zeroes
// them when it allocates them).
struct FusedArgs {
    TablesDev tb;
    RawQueries raw;            // device queries when raw.budget is set (the QueryDev otherwise)
    uint2 *regions;            // per block: M * O option records, then inner_stride(O) records
    uint32_t region;           // records per block region
    uint32_t *done;            // per item: finished block groups
    uint32_t *group_done;      // per item and group of kFusedGroup blocks: finished blocks
    unsigned long long *best;
};
// Blocks of an item counted together before the item's count (two-level counting, so that at
// most this many blocks update one counter word).
constexpr uint32_t kFusedGroup = 64;

// What the option-term kernel resets for the scan that follows it: per item, the finished-block
// counter (done = 0) and the smallest block latency (best = kNoLatency, if best is set); every
// block winner slot (winners[0..n_winners) = no candidate).
struct ScanReset {
    uint32_t *done = nullptr;
    uint32_t *best = nullptr;
    Winner *winners = nullptr;
    uint64_t n_winners = 0;
};

hipError_t launch_option_terms(const SpaceDev &sp, const TablesDev &tb, const QueryDev &q,
                               uint32_t count, uint2 *rec, uint2 *ext, uint2 *inner,
                               const ScanReset &reset, hipStream_t st,
                               const RawQueries *raw = nullptr,
                               hipEvent_t t0 = nullptr, hipEvent_t t1 = nullptr);
// Pair table of count items: pair[item][j3 * O + j2] = (c of LLM M-3 option j3 + c of LLM M-2
// option j2, Q*G - both share units), from the option-term kernel's rec and inner tables;
// padding records never fit.
hipError_t launch_pair_terms(const SpaceDev &sp, uint32_t count, const uint2 *rec,
                             const uint2 *inner, uint2 *pair, hipStream_t st);
// fz: the one-launch form's arguments (g.fused), else nullptr.
hipError_t launch_scan(const SpaceDev &sp, const QueryDev &q, uint32_t count, const uint2 *rec,
                       const uint2 *inner, const ScanGeometry &g, Winner *winners,
                       const FinishArgs &fa, hipStream_t st, hipEvent_t t0 = nullptr,
                       hipEvent_t t1 = nullptr, const FusedArgs *fz = nullptr);
// Dynamic LDS of a one-launch scan block: the item's profile curves (for every (LLM, tp,
// share): rate padded to ALP_MAX_POINTS points, then -- after all rates -- lat, K points) and
// their deployability flags ...
__host__ __device__ inline size_t fused_lds_curves(const SpaceDev &sp)
{
    return (size_t)sp.M * sp.n_tp * sp.n_fq;
}
__host__ __device__ inline size_t fused_lds_lat_offset(const SpaceDev &sp)
{
    return fused_lds_curves(sp) * ALP_MAX_POINTS * sizeof(uint32_t);
}
__host__ __device__ inline size_t fused_lds_deploy_offset(const SpaceDev &sp)
{
    return fused_lds_lat_offset(sp) + fused_lds_curves(sp) * sp.K * sizeof(uint32_t);
}
// ... followed by the inner LLM's records (inner_stride(O) of them), 8-byte aligned.
__host__ __device__ inline size_t fused_lds_inner_offset(const SpaceDev &sp)
{
    return (fused_lds_deploy_offset(sp) + fused_lds_curves(sp) + 7) & ~(size_t)7;
}
// ... then every option's (tau, share units) for the result record.
__host__ __device__ inline size_t fused_lds_ext_offset(const SpaceDev &sp)
{
    return fused_lds_inner_offset(sp) + (size_t)inner_stride(sp.O) * 8;
}
__host__ __device__ inline size_t fused_lds_bytes(const SpaceDev &sp)
{
    return fused_lds_ext_offset(sp) + (size_t)sp.M * sp.O * 8;
}
// Records per block region of the one-launch form.
__host__ __device__ inline uint32_t fused_region(uint32_t M, uint32_t O)
{
    return (M * O + inner_stride(O) + 7u) & ~7u;    // 64-byte multiple
}
hipError_t launch_eval(const SpaceDev &sp, uint32_t capacity, const uint2 *rec, const uint2 *ext,
                       const uint64_t *idx, uint64_t count, alp_eval_t *out, hipStream_t st);
hipError_t launch_tmax(const SpaceDev &sp, const QueryDev &q, uint32_t count, const uint2 *ext,
                       uint32_t *out, hipStream_t st);

// Budget split over W workflows from their per-budget search results (res[w * (G + 1) + g]),
// see alp_allocate_workflows.  dp: device scratch of (W + 1) * (G + 1) uint64 followed by
// 2 * W * (G + 1) uint32.  Writes *plan and gpus[0..W).
hipError_t launch_allocate(const alp_result_t *res, uint32_t W, uint32_t G, uint32_t policy,
                           uint64_t *dp, alp_plan_t *plan, uint32_t *gpus, hipStream_t st);

// The paper's pruned search for count items (see alp_search_pruned), after the option-term
// kernel (rec, ext; it also zeroes done[]).  launch_pruned_table fills `table`
// (count * M * Q * (F_max + 1) entries) and `orders` (count records of pruned_order_bytes());
// launch_pruned_scan runs blocks_per_item blocks of 256 threads per item, covering
// pruned_prefixes(M, F_max) threads; winners and counts hold count * blocks_per_item entries.
// Writes out[0..count).
uint64_t pruned_prefixes(uint32_t M, uint32_t F_max);
size_t pruned_order_bytes();
hipError_t launch_pruned_table(const SpaceDev &sp, const TablesDev &tb, const QueryDev &q,
                               uint32_t count, uint32_t F_max, uint32_t flags, const uint2 *rec,
                               uint64_t *table, void *orders, hipStream_t st);
hipError_t launch_pruned_scan(const SpaceDev &sp, uint32_t count, uint32_t F_max, uint32_t flags,
                              const uint64_t *table, const void *orders, uint32_t blocks_per_item,
                              Winner *winners, uint64_t *counts, const uint2 *ext, uint32_t *done,
                              alp_pruned_t *out, hipStream_t st);

static_assert(sizeof(alp_stats_t) == 32 && offsetof(alp_stats_t, calls) == 8 &&
                  offsetof(alp_stats_t, active_us) == 24,
              "alp_stats_t layout");
static_assert(sizeof(alp_pruned_t) == 64 && offsetof(alp_pruned_t, fraction_vectors) == 48 &&
                  offsetof(alp_pruned_t, unpruned_vectors) == 56,
              "alp_pruned_t layout");

// Workflow statistics (see alp_trace_stats).  Traces up to lds_cap calls (a power of two,
// 256..2048) are swept or sorted in LDS; the num_long others (long_traces[]) are sorted in
// scratch, trace k at 2 * long_base[k] words (2 * pow2(length) words each).  totals:
// kStatsTotalsWords + kStatsTailWords words: kStatsCopies copies of the per-LLM sums,
// kStatsCopyStride words apart (trace r adds to copy r mod kStatsCopies, so that thousands of
// traces do not queue on the same atomic words), then the status flags (one word), the length
// of the work list and the count of finished slots (the low and high half of the next), and
// kStatsSlots 32-bit counters of finished blocks.  They must be zero when the kernels start; the last block leaves them zero,
// so zero_first is needed only for fresh memory or after a failed launch.  sweep: traces in end order are swept without a sort and the others listed in work
// (R entries) for the sort pass; otherwise every trace is sorted.  max_short: the most calls of
// a trace within lds_cap (direct sorts launch only the group sizes it reaches).  Writes
// out[0..M) and the StatsTail at out[ALP_MAX_LLMS].
constexpr uint32_t kStatsCopies = 64;
constexpr uint32_t kStatsCopyStride = 32;                 // >= 3 * ALP_MAX_LLMS, 256 B apart
constexpr uint32_t kStatsTotalsWords = kStatsCopies * kStatsCopyStride;
constexpr uint32_t kStatsSlots = 64;
constexpr uint32_t kStatsTailWords = 2 + kStatsSlots / 2;
struct StatsTail {
    uint32_t flags;                   // status bits (see alp_trace_stats)
    uint32_t listed;                  // traces the sweep left to the sort pass
    uint32_t pad[6];
};
static_assert(sizeof(StatsTail) == sizeof(alp_stats_t), "the tail takes one record's place");
hipError_t launch_trace_stats(uint32_t M, uint32_t R, const uint64_t *offsets, const uint32_t *llm,
                              const uint64_t *start, const uint64_t *end, uint32_t lds_cap,
                              uint32_t max_short, uint32_t num_long, const uint32_t *long_traces,
                              const uint64_t *long_base, uint64_t *scratch, uint64_t *totals,
                              uint32_t *work, bool sweep, bool zero_first, alp_stats_t *out,
                              hipStream_t st);

// One allocation to place: budget, LLM count, whether the search found it, per-LLM choices,
// and the index of its output record.
struct PlaceIn {
    uint8_t gpus, llms, feasible, pad;
    uint8_t tp[ALP_MAX_LLMS], q[ALP_MAX_LLMS], d[ALP_MAX_LLMS];
    uint32_t dst;
};

// Placement (see alp_place); Q share units per GPU.  in[0..small) have budgets of at most 16
// GPUs (placed four to a wave), in[small..small + large) the others (one to a wave); each
// writes out[in[i].dst].
hipError_t launch_place(uint32_t Q, uint32_t small, uint32_t large, const PlaceIn *in,
                        alp_placement_t *out, hipStream_t st);

static_assert(sizeof(alp_placement_t) == 272 && offsetof(alp_placement_t, slot) == 16,
              "alp_placement_t layout");

// Device address of the fixed scratch array of alp_search_batch_async_noalloc on `device`, which
// must be the current device.  Looked up once per device; later calls return the kept address.
hipError_t static_scratch_address(int device, void **ptr);

// Resident blocks per CU of the scan kernels at a given block size (occupancy query).
int scan_blocks_per_cu(uint32_t variant, uint32_t slots, uint32_t threads, const SpaceDev &sp);

}  // namespace alp
