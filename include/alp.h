/*
 * alp.h -- C ABI of the MI355X (gfx950) Aggregate LLM Pipeline allocation search.
 *
 * The search follows "Scepsy" (arXiv 2604.15186).  An agentic workflow is abstracted as a
 * pipeline of its LLMs (Section 4).  For LLM m the inputs are its workflow statistics n_m
 * (invocations per workflow request) and p_m (request-level parallelism) (Section 4, step 2),
 * and its per-replica throughput--latency profile, one curve per tensor-parallel degree and GPU
 * share (Section 4, step 3).  A candidate allocation picks, per LLM, a tensor-parallel degree
 * tp, a GPU share q (in units of 1/Q GPU) and a replica count d (the three search dimensions
 * of Section 1 and Section 5).  The predictor (Section 4, steps 4-5) gives
 *   L_w = sum_m L_m(lambda * n_m / d_m) * n_m / p_m     (Eq. 1, the latency at each replica's load)
 *   T_w = min_m d_m * T_m / n_m                         (Eq. 2, T_m the saturation throughput)
 * and the search returns the allocation of lowest L_w that sustains the target workflow rate
 * (T_w >= lambda), fits every LLM's weights into its GPU share (Section 5, step 1) and uses at
 * most the GPU budget (Section 3, step 3: the objective is the lowest latency that still meets
 * the workflow's target rate).  Every candidate of the space is evaluated; ties go to the lowest
 * index.
 *
 * Fixed point: rates in milli-requests/s, latencies in microseconds, n_m and p_m in thousandths.
 * Per-replica rate r = ceil(lambda * n / (1000 d)); latency at r is lat[0] for r <= rate[0],
 * linear between profile points (rounded down) and undefined above rate[K-1] (the option cannot
 * sustain the load); contribution c = floor(latency * n / p); normalised throughput
 * tau = floor(1000 d rate[K-1] / n); share units u = tp * q * d; memory fit W * Q <= tp * q * H.
 *
 * Numbering.  Option o of an LLM = (i * num_frac + j) * max_replicas + (d - 1) for
 * tp = tp_values[i], q = frac_units[j] (replicas vary fastest).  Candidate
 * x = sum_m o_m * O^(M-1-m) with O options per LLM (LLM 0 is the most significant digit).
 *
 * Conventions.  Every function returns an alp_status (int32_t).  No exception crosses the ABI.
 * Host pointers unless stated.  Inputs are owned by the caller and deep-copied where kept.
 * Out-parameters are written only on ALP_OK (and ALP_INFEASIBLE where stated).  A failed call
 * leaves the context usable and unchanged.  A context is not thread-safe; distinct contexts are
 * independent.  alp_last_error() describes the last failure of the calling thread.
 *
 * Test hook: while the environment variable ALP_TEST_FAIL_ALLOC is set (to anything but "0"),
 * every device and pinned host allocation the library attempts fails, and the call returns
 * ALP_ENOMEM; buffers a context already holds are kept, so later calls that need no larger ones
 * still succeed.
 */
#ifndef ALP_H
#define ALP_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    ALP_OK = 0,
    ALP_EINVAL = 1,      /* malformed argument or table */
    ALP_ERANGE = 2,      /* values would overflow the fixed-point objective or index space */
    ALP_ENOMEM = 3,      /* device or host allocation failed */
    ALP_EDEVICE = 4,     /* no usable device, or a HIP call failed */
    ALP_INFEASIBLE = 5   /* no candidate meets target, memory fit and budget */
} alp_status;

#define ALP_MAX_LLMS 8
#define ALP_MAX_TP 8
#define ALP_MAX_FRAC 8
#define ALP_MAX_REPLICAS 16
#define ALP_MAX_POINTS 16
#define ALP_MAX_OPTIONS 512      /* num_tp * num_frac * max_replicas */
#define ALP_NO_INDEX UINT64_MAX

/* Shape of the search space, shared by every instance of a context (Section 5: the scheduler
 * enumerates GPU fractions, tensor-parallel degrees and replica counts per LLM).
 *   num_llms      M, 1..8
 *   tp_values     strictly ascending tensor-parallel degrees, 1..64 (Section 5, step 3 caps tp
 *                 at the high-bandwidth interconnect degree; an MI355X node has 8)
 *   frac_units    strictly ascending GPU shares in units of 1/units_per_gpu, 1..units_per_gpu
 *   units_per_gpu Q, 1..16 (4 = quarters)
 *   max_replicas  D, replica counts 1..D, D in 1..16
 *   num_points    K profile points per (tp, share) curve, 1..16
 * O = num_tp * num_frac * max_replicas must be <= ALP_MAX_OPTIONS and O^M < 2^63. */
typedef struct {
    uint32_t num_llms;
    uint32_t num_tp;
    uint32_t tp_values[ALP_MAX_TP];
    uint32_t num_frac;
    uint32_t frac_units[ALP_MAX_FRAC];
    uint32_t units_per_gpu;
    uint32_t max_replicas;
    uint32_t num_points;
} alp_space_t;

/* Search result (48 bytes).  status is ALP_OK or ALP_INFEASIBLE (or ALP_EINVAL for a query
 * alp_search_batch_async rejected); otherwise than ALP_OK, index is ALP_NO_INDEX and the other
 * fields are 0.  latency_us = L_w (Eq. 1), throughput_milli = T_w
 * (Eq. 2), gpu_units = sum of tp * q * d; per LLM the chosen tp, share (units of 1/Q) and
 * replica count, entries beyond num_llms 0. */
typedef struct {
    uint64_t index;
    uint32_t latency_us;
    uint32_t throughput_milli;
    uint32_t gpu_units;
    uint32_t status;
    uint8_t tp[ALP_MAX_LLMS];
    uint8_t frac_units[ALP_MAX_LLMS];
    uint8_t replicas[ALP_MAX_LLMS];
} alp_result_t;

/* Evaluation of one candidate (16 bytes).
 *   flags bit0: every LLM's option is deployable and its weights fit (Section 5, step 1)
 *         bit1: every LLM sustains its per-replica load (r <= rate[K-1]; same as T_w >= lambda)
 *         bit2: sum of share units <= Q * gpu_budget
 *   latency_us       L_w (Eq. 1) if bit0 and bit1, else UINT32_MAX
 *   throughput_milli T_w (Eq. 2) if bit0, else 0
 *   gpu_units        sum of tp * q * d */
typedef struct {
    uint32_t flags;
    uint32_t latency_us;
    uint32_t throughput_milli;
    uint32_t gpu_units;
} alp_eval_t;

typedef struct alp_ctx alp_ctx;

/* Loads and validates the profiles of num_instances workflow instances and copies them to the
 * device (Section 4, steps 2-3 produce these tables).  Host arrays, row-major, B = num_instances:
 *   weight_bytes  uint64 [B][M]               model weights in bytes, < 2^48
 *   n_milli       uint32 [B][M]               n_m * 1000, 1 .. 2^31-1
 *   p_milli       uint32 [B][M]               p_m * 1000, 1 .. 2^31-1
 *   allowed       uint8  [B][M][num_tp][num_frac]     0/1: the (tp, share) pair may be deployed
 *   rate_milli    uint32 [B][M][num_tp][num_frac][K]  per-replica rates, strictly ascending in
 *                                                     k, < 2^31; the last is saturation
 *   lat_us        uint32 [B][M][num_tp][num_frac][K]  latency at that rate, < 2^31 (the caller
 *                                                     picks mean or a percentile, Section 4 step 5)
 * hbm_bytes_per_gpu H, 1 .. 2^48-1.  device: HIP device ordinal.  hip_stream: hipStream_t all
 * work of the context is ordered on (NULL: the device's null stream); it must outlive the ctx.
 * Errors: EINVAL (shape, ranges, ordering, NULL pointer), ERANGE (some instance's largest
 * possible L_w over deployable options reaches 2^32-1), EDEVICE, ENOMEM.  On success *out
 * owns device memory until alp_free. */
int32_t alp_load_profiles(alp_ctx **out, const alp_space_t *space, uint32_t num_instances,
                          const uint64_t *weight_bytes, const uint32_t *n_milli,
                          const uint32_t *p_milli, const uint8_t *allowed,
                          const uint32_t *rate_milli, const uint32_t *lat_us,
                          uint64_t hbm_bytes_per_gpu, int32_t device, void *hip_stream);

/* Exhaustive constrained argmin for one instance at GPU budget gpu_budget (whole GPUs) and
 * target workflow rate target_milli: the search objective of Section 3 (the lowest latency at
 * which the workflow sustains its target rate), with the latency of every candidate predicted by
 * Eq. 1 and its throughput by Eq. 2 (Section 4), over every candidate of the space; among equal
 * latencies the lowest candidate index.  A candidate is feasible iff every LLM's option is
 * deployable and its weights fit its share (Section 5, step 1), T_w >= target_milli, and
 * sum tp * q * d <= units_per_gpu * gpu_budget.  Synchronous: returns once the search's last
 * block has written the result to host memory (its exit may still be in flight on the context
 * stream, ahead of any later work queued there).  Returns
 * ALP_OK with the result in *out, or ALP_INFEASIBLE with out->status = ALP_INFEASIBLE and
 * out->index = ALP_NO_INDEX.  EINVAL: ctx or out NULL, or instance >= num_instances (nothing
 * written).  ERANGE: the space cannot be covered by one launch.  ENOMEM/EDEVICE: allocation or
 * HIP failure. */
int32_t alp_search(alp_ctx *ctx, uint32_t instance, uint32_t gpu_budget, uint32_t target_milli,
                   alp_result_t *out);

/* count independent searches in one launch sequence (the multi-workflow level of Section 5 runs
 * one search per workflow).  instances may be NULL (0..count-1).  out[i].status is ALP_OK or
 * ALP_INFEASIBLE per query; the call returns ALP_OK unless an argument or device error occurs.
 * count = 0 is a no-op. */
int32_t alp_search_batch(alp_ctx *ctx, uint32_t count, const uint32_t *instances,
                         const uint32_t *gpu_budget, const uint32_t *target_milli,
                         alp_result_t *out);

/* Batched searches with the queries and the results in device memory, queued on the context's
 * HIP stream without waiting (Section 5, the same search as alp_search_batch).  instances
 * (NULL = 0..count-1), gpu_budget and target_milli are device arrays of count entries; out is a
 * device array of count records.  The call returns once the work is queued: the inputs must
 * stay unchanged, and out is complete, only when the stream has reached the end of this work
 * (synchronise the stream, or order later work after it on the same stream).  A query whose
 * instance is out of range gets status ALP_EINVAL in its record and does not affect the others;
 * the other records are as alp_search_batch writes them.  Returns ALP_EINVAL for a NULL ctx or
 * array (instances aside), or the first error in queuing the work.  With timing enabled, the
 * call's kernel times are read (waiting for its work) by the next alp_kernel_times,
 * alp_kernel_time_totals or alp_set_timing call.  Successive calls on one context, and calls of
 * the synchronous functions after it, are ordered by the stream; a call that needs larger
 * scratch buffers than earlier ones first waits for the stream. */
int32_t alp_search_batch_async(alp_ctx *ctx, uint32_t count, const uint32_t *instances,
                               const uint32_t *gpu_budget, const uint32_t *target_milli,
                               alp_result_t *out);

/* ---- Searches that allocate nothing ----------------------------------------------------------
 * For callers that cannot allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  The same searches as alp_search_batch_async (same
 * arguments, device-resident queries and results, queued on the context stream without waiting,
 * the same result records), but every buffer the search needs beyond its inputs and outputs
 * (prepared queries, per-option records, the inner or pair table, per-item counters, block
 * winners) lives in one fixed device array of ALP_STATIC_SCRATCH_BYTES per GPU, whose address
 * alp_load_profiles takes; the call itself allocates nothing, device or host, and creates no
 * events (it is not counted or timed by alp_set_timing).  The kernels reset what must start at
 * zero, so the array's leftover contents from the previous call do not matter.  The array is
 * shared by every context and every call on its GPU: calls that overlap in time on one GPU (two
 * streams, two contexts, two threads) race on it and give undefined results, so the caller
 * serialises them (calls queued on one stream are ordered).  Returns ALP_ERANGE, before queuing
 * anything, if the batch needs more than the array holds (alp_last_error states both sizes;
 * about 11 KiB per 5-LLM search plus the 128 KiB pair table, 6 KiB per 3-LLM search), and
 * ALP_EDEVICE if the array's address could not be taken at load. */
#define ALP_STATIC_SCRATCH_BYTES (8u << 20)
int32_t alp_search_batch_async_noalloc(alp_ctx *ctx, uint32_t count, const uint32_t *instances,
                                       const uint32_t *gpu_budget, const uint32_t *target_milli,
                                       alp_result_t *out);

/* Largest workflow throughput T_w (Eq. 2) any candidate with deployable, fitting options
 * reaches within the budget, ignoring the target; 0 if none fits.  A target above it is
 * infeasible, a target at or below it is feasible.  instances may be NULL. */
int32_t alp_max_throughput(alp_ctx *ctx, uint32_t count, const uint32_t *instances,
                           const uint32_t *gpu_budget, uint32_t *out_tmax);

/* Several workflows sharing a pool of GPUs (Section 5, scheduling of several workflows: the
 * scheduler decides how many GPUs each workflow gets, searches each workflow's allocation
 * independently, and combines the per-workflow utilities with egalitarian or social welfare).
 * Workflow w is loaded instance instances[w] with target rate target_milli[w].  It gets g_w whole
 * GPUs, sum g_w <= total_gpus, and its search result at budget g_w; its utility is minus that
 * latency (a workflow with no feasible allocation makes the split infeasible).
 *   ALP_WELFARE_EGALITARIAN: minimise the largest workflow latency, ties by the latency sum;
 *   ALP_WELFARE_SOCIAL:      minimise the latency sum;
 * remaining ties go to the lexicographically smallest budget vector (workflow 0 first), so GPUs
 * that improve nothing stay unassigned. */
#define ALP_WELFARE_EGALITARIAN 0u
#define ALP_WELFARE_SOCIAL 1u

/* Outcome of alp_allocate_workflows (24 bytes). */
typedef struct {
    uint32_t status;           /* ALP_OK or ALP_INFEASIBLE */
    uint32_t policy;
    uint32_t max_latency_us;   /* largest workflow latency of the split (0 if infeasible) */
    uint32_t gpus_used;        /* sum of the budgets */
    uint64_t sum_latency_us;   /* sum of the workflow latencies */
} alp_plan_t;

/* Runs every (workflow, budget 0..total_gpus) search in one batch on the device, then the
 * split.  count in 1..16, total_gpus in 0..1024, instances may be NULL (0..count-1).
 * On ALP_OK and ALP_INFEASIBLE writes *plan; on ALP_OK also gpus[w] and results[w] (workflow
 * w's search result at g_w).  Returns ALP_INFEASIBLE if no split makes every workflow feasible. */
int32_t alp_allocate_workflows(alp_ctx *ctx, uint32_t count, const uint32_t *instances,
                               const uint32_t *target_milli, uint32_t total_gpus, uint32_t policy,
                               alp_plan_t *plan, uint32_t *gpus, alp_result_t *results);

/* ---- The paper's pruned search (Section 5, steps 1-3) ----------------------------------------
 * The paper's own scheduler enumerates GPU fractions instead of every candidate, and so need not
 * reach the exhaustive optimum; this entry point runs it on the device, for comparison.
 *   Step 1: LLM m receives f_m units of 1/Q GPU with sum f_m = Q*G.  ALP_PRUNE_ORDER: LLMs are
 *           ordered by profiled latency ratio (the Eq. 1 contribution at the smallest TP degree,
 *           the largest share and the first profiled point, largest first, ties by LLM index) and
 *           no LLM receives more units than the one before it.  ALP_PRUNE_MIN_FRACTION: each LLM
 *           receives at least max(1, ceil(W_m * Q / H)) units (its weights), and at most Q*G
 *           minus the lower bounds of the LLMs after it.
 *   Step 2: the fractions are packed contiguously in that order over the Q*G units, GPU by GPU.
 *   Step 3: option (tp, q, d) is admissible for an LLM iff tp * q * d equals its fraction and d
 *           replicas of tp ranks of q units, the ranks of one replica on distinct GPUs, fit its
 *           packed GPUs.
 * The result is the feasible admissible candidate of lowest L_w, ties to the lowest index. */
#define ALP_PRUNE_ORDER 1u
#define ALP_PRUNE_MIN_FRACTION 2u
#define ALP_PRUNED_MAX_UNITS 2048u           /* Q*G per query */
#define ALP_PRUNED_MAX_VECTORS (1ull << 34)  /* step-1 vectors per query, before bounds */

/* One pruned search (64 bytes). */
typedef struct {
    alp_result_t best;            /* as alp_search's result; ALP_INFEASIBLE if none */
    uint64_t fraction_vectors;    /* fraction vectors enumerated in step 1 */
    uint64_t unpruned_vectors;    /* C(Q*G + M - 1, M - 1): every split of Q*G units, saturating */
} alp_pruned_t;

/* Pruned searches of count queries (instances may be NULL: 0..count-1), one launch sequence.
 * flags: any of ALP_PRUNE_ORDER | ALP_PRUNE_MIN_FRACTION (else EINVAL).  Each query needs
 * Q * gpu_budget[i] <= ALP_PRUNED_MAX_UNITS (else EINVAL) and at most ALP_PRUNED_MAX_VECTORS
 * step-1 vectors counted without the lower bounds (else ERANGE).  Writes out[0..count) on
 * ALP_OK; each out[i].best.status is ALP_OK or ALP_INFEASIBLE. */
int32_t alp_search_pruned(alp_ctx *ctx, uint32_t count, const uint32_t *instances,
                          const uint32_t *gpu_budget, const uint32_t *target_milli, uint32_t flags,
                          alp_pruned_t *out);

/* ---- Workflow statistics from execution traces (Section 4, step 2) --------------------------
 * A trace is one workflow-level request: the LLM-level calls it made, each with its LLM index
 * and a half-open [start, end) interval in microseconds (tools and other non-LLM components are
 * left out by the caller).  For every LLM m:
 *   n_m = calls of m per workflow request = calls_m / traces;
 *   p_m = request-level parallelism from overlapping timestamps = the total duration of m's
 *         calls divided by the time during which at least one call of m runs, summed over the
 *         traces (so that n_m * L_m / p_m in Eq. 1 is the time per request m is active).
 * Both in thousandths, rounded down; p = 1000 if m has calls but none of positive length, and
 * n = p = 0 if m has no calls.  The results are the n_milli / p_milli inputs of
 * alp_load_profiles. */
typedef struct {
    uint32_t n_milli;
    uint32_t p_milli;
    uint64_t calls;        /* calls of the LLM over all traces */
    uint64_t busy_us;      /* sum of their durations */
    uint64_t active_us;    /* sum over traces of the time at least one of them runs */
} alp_stats_t;

typedef struct alp_stats_ctx alp_stats_ctx;

/* A statistics context on `device`, ordering its work on hip_stream (NULL: the default
 * stream).  It owns the device scratch of the computation until alp_stats_free. */
int32_t alp_stats_create(alp_stats_ctx **out, int32_t device, void *hip_stream);

/* Statistics of num_traces traces.  Device pointers: offsets[num_traces + 1] (ascending from 0;
 * trace r's calls are [offsets[r], offsets[r + 1])), llm[E], start_us[E], end_us[E] with
 * E = offsets[num_traces].  num_llms in 1..8; a trace has at most 2^24 calls; start < 2^60 and
 * end - start < 2^32.  Writes out[0..num_llms) (host).  EINVAL for a malformed input (offsets,
 * llm >= num_llms, end < start), ERANGE for out-of-range timestamps or a result of 2^31 or
 * more.  Synchronous on the context's stream.  Any call order within a trace gives the same
 * result; traces whose calls are in order of end time (as logged on completion) and that span
 * under 2^32 us take the fast path (no sort).  A context whose call finds most traces out of
 * end order sorts every trace directly on its next 7 calls, then checks the order again.  The
 * context's scratch grows to 4 bytes per trace plus, for traces beyond 2,048 calls, 16 bytes
 * per call rounded up to a power of two per trace. */
int32_t alp_trace_stats(alp_stats_ctx *ctx, uint32_t num_llms, uint32_t num_traces,
                        const uint64_t *offsets, const uint32_t *llm, const uint64_t *start_us,
                        const uint64_t *end_us, alp_stats_t *out);

/* Enables HIP-event timing; alp_stats_time gives the milliseconds of the last computation's
 * kernels (initialisation to final division). */
int32_t alp_stats_set_timing(alp_stats_ctx *ctx, int32_t enable);
int32_t alp_stats_time(alp_stats_ctx *ctx, float *ms);

void alp_stats_free(alp_stats_ctx *ctx);

/* ---- Placement of allocations on GPU nodes (Section 6, hierarchical placement) -------------
 * The search counts GPU share units only (sum tp * q * d <= Q * G); whether the allocation can
 * be laid out on real GPUs is a packing question.  alp_place answers it with the paper's
 * most-constrained-first heuristic.  The G GPUs of a budget form nodes of ALP_NODE_GPUS (the last
 * may hold fewer), every node one all-to-all xGMI domain; each GPU holds Q units.  LLM m needs
 * d_m replicas of tp_m ranks of q_m units, the ranks of a replica on distinct GPUs of one node.
 * Replicas are placed tensor-parallel first, larger (tp * q) first, ties by LLM index.  A
 * tensor-parallel replica takes, in some node, tp GPUs with room: among the node's GPUs with
 * room ordered by (free units, index), a run of tp consecutive ones scored by imbalance (most
 * minus least free units), then the node's free units (the smaller domain first, keeping large
 * domains for larger models), then the run's free units, then node and position.  A single-GPU
 * replica packs onto an occupied GPU with room (fewest free units, then lowest index), else onto
 * the lowest empty GPU of the node with the fewest free units. */
#define ALP_NODE_GPUS 8u
#define ALP_PLACE_MAX_GPUS 64u
#define ALP_PLACE_MAX_REPLICAS 128u
#define ALP_PLACE_NONE 0xFFFFu

/* One placement (272 bytes). */
typedef struct {
    uint32_t status;          /* ALP_OK: every replica placed; ALP_INFEASIBLE: one found no room,
                                 or the allocation itself was infeasible */
    uint32_t replicas;        /* replicas placed */
    uint32_t gpus_used;       /* GPUs holding at least one rank */
    uint32_t nodes_used;
    uint16_t slot[ALP_PLACE_MAX_REPLICAS];  /* per replica, LLM 0's first: node << 8 | mask of
                                               the node's GPUs; ALP_PLACE_NONE if not placed */
} alp_placement_t;

/* Places count allocations (search results of this context's space: tp, frac_units, replicas
 * per LLM; an ALP_INFEASIBLE result places nothing) on gpu_budget[i] <= ALP_PLACE_MAX_GPUS GPUs
 * each, one thread per allocation.  Host arrays; synchronous on the context's stream.  EINVAL for
 * a budget above the maximum or a record whose choices are not of the space. */
int32_t alp_place(alp_ctx *ctx, uint32_t count, const alp_result_t *allocations,
                  const uint32_t *gpu_budget, alp_placement_t *out);

/* The predictor at listed candidates (the element-wise check of the search): for each index
 * x of indices[0..count) (host array, each < O^M, else EINVAL and nothing written) of
 * `instance`, at gpu_budget and target_milli, out[i] (host) gets the flags and values of
 * alp_eval_t: L_w by Eq. 1 with every LLM at its per-replica load (Section 4, step 5), T_w by
 * Eq. 2, the share units, and the feasibility conditions the search applies (Section 5, step 1;
 * the target rate and the budget, Section 3).  Synchronous on the context stream.  count = 0 is
 * a no-op. */
int32_t alp_eval_candidates(alp_ctx *ctx, uint32_t instance, uint32_t gpu_budget,
                            uint32_t target_milli, const uint64_t *indices, uint64_t count,
                            alp_eval_t *out);

/* Added to variant 0, 1, 4 or 5 of alp_set_launch: the option terms run in their own kernel
 * before the scan (the two-launch form), also where one launch would do. */
#define ALP_LAUNCH_SEPARATE_TERMS 16u

/* Launch choices, for tests and tuning.  variant: 0 automatic, 1 row-minimum scan (default),
 * 2 thread-per-candidate scan, 3 exact-tracking lane scan, 4 row-minimum scan with fixed row
 * ranges per wave, 5 row-minimum scan with rows handed out within each block (variant 1 picks
 * between the two; rows can only be split with the second, so variant 4 ignores inner_chunks),
 * 6 row-minimum scan over the pair table (LLMs M-3 and M-2 folded into one inner LLM of O^2
 * options, 3 or more LLMs; variant 0 uses it for 5 or more LLMs while the batch's pair tables
 * stay within 4 MiB).  Spaces of at most 2^25 candidates searched with the row-minimum scan
 * without the pair table run in one launch: every block computes its item's option terms itself
 * (unless ALP_LAUNCH_SEPARATE_TERMS is added).  blocks_per_item and threads_per_block (a multiple
 * of 64, at most 1024):
 * 0 = automatic.  inner_chunks (variants 1, 5, 6): ranges each row's inner-LLM records are
 * split into, dividing ceil(O / 16) (variant 6: the pair table's ceil(O^2 / 16)); 0 =
 * automatic.  Results do not depend on these choices. */
int32_t alp_set_launch(alp_ctx *ctx, uint32_t variant, uint32_t blocks_per_item,
                       uint32_t threads_per_block, uint32_t inner_chunks);

/* HIP-event timing of the searches' kernels on the context stream.  enable = 0: off; N >= 1: the
 * calls of alp_search, alp_search_batch, alp_search_batch_async, alp_allocate_workflows,
 * alp_search_pruned and alp_place are counted from this call on, and the first and every N-th
 * after it are timed (the option-term and scan dispatches are stamped with their begin and end;
 * stamping keeps the GPU idle for a few microseconds between the kernels, so timing a sample of
 * the calls of a long run leaves the run's throughput nearly unchanged).  Setting resets the
 * count and the sums below; a negative enable is ALP_EINVAL.
 * alp_kernel_times writes, for the last timed search or batch, the milliseconds of the
 * option-term kernel (ms[0]; 0 when the search ran in one launch) and of the candidate scan
 * kernel, which includes the final reduction and the result write (ms[1]); ms[2] is the budget-split kernel of alp_allocate_workflows, 0
 * after the other searches.  After alp_search_pruned: ms[1] is the fraction enumeration and ms[2]
 * the admissible-option table.  After alp_place: ms[1] is the placement kernel, the others 0.
 * *scan_blocks receives the scan (or enumeration) grid size of the last search.
 * alp_kernel_time_totals writes the sums of those three figures over the timed calls since
 * timing was last set, and (if timed_calls is not NULL) their number, so that a caller timing
 * many calls reads them once. */
int32_t alp_set_timing(alp_ctx *ctx, int32_t enable);
int32_t alp_kernel_times(alp_ctx *ctx, float ms[3], uint32_t *scan_blocks);
int32_t alp_kernel_time_totals(alp_ctx *ctx, double ms[3], uint64_t *timed_calls);

/* Candidates per instance, O^M. */
int32_t alp_num_candidates(const alp_ctx *ctx, uint64_t *out);

/* Releases the context (NULL is a no-op). */
void alp_free(alp_ctx *ctx);

const char *alp_status_str(int32_t status);
const char *alp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ALP_H */
