// gfx950 kernels of the ALP allocation search (Scepsy, arXiv 2604.15186, Sections 4-5).
//
// Pipeline of one search (or a batch of independent searches, one "item" each):
//   1. option_terms_kernel: per (item, LLM m, option o) the Eq. 1 contribution c and the share
//      units u (replaced by a sentinel when the option is unusable at the target), plus the
//      Eq. 2 normalised throughput tau and validity flags for result decoding.
//   2. scan_min_kernel<S, ...> (or, for cross-checks, scan_flat_kernel / scan_lane_kernel<S>): every
//      candidate x = (o_0 .. o_{M-1}) is evaluated -- L_w = sum c, feasible iff sum u <= Q*G --
//      and the lexicographic (L_w, x) minimum is reduced per wave, per block, and written as one
//      16-byte winner per block.
//   3. The last block of each item to finish (an agent-scope counter) takes the minimum over the
//      item's block winners, decodes the winning index and recomputes T_w (Eq. 2) and the share
//      units from the per-option records.
// Everything is integer; results are bit-identical for every launch geometry.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "alp_device.h"
#include "alp_internal.h"

namespace alp {

namespace {

constexpr uint32_t kMaxOuter = ALP_MAX_LLMS - 2;   // digits above the last two LLMs
constexpr int32_t kNeverFits = -(1 << 30);          // remaining units no lane can satisfy

}  // namespace

// ---------------------------------------------------------------------------------------------
// 1. Per-option terms.  One thread per (item, m, o).
//    rec[item][m][o] = (c, usable ? u : sentinel), c = 0 when unusable
//    ext[item][m][o] = (tau, u | ok << 16 | thr_ok << 17)
//    inner[item][o]  = (c, capacity - (usable ? u : sentinel)) for m = M-2 (if inner != nullptr):
//                      the share units left for the other LLMs once LLM M-2 takes option o
//    done[item]      = 0, best[item] = kNoLatency, winners[] = no candidate (see ScanReset)
__global__ void __launch_bounds__(256)
option_terms_kernel(SpaceDev sp, TablesDev tb, QueryDev q, uint32_t count, uint2 *__restrict__ rec,
                    uint2 *__restrict__ ext, uint2 *__restrict__ inner, ScanReset reset,
                    RawQueries raw)
{
    const uint64_t per_item = (uint64_t)sp.M * sp.O;
    const uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= per_item * count)
        return;
    const uint32_t item = (uint32_t)(t / per_item);
    const uint32_t rem = (uint32_t)(t - (uint64_t)item * per_item);
    const uint32_t m = div_by(rem, sp.mul_O), o = rem - m * sp.O;
    // State of the scan's fused reduction.
    if (reset.done && rem == 0)
        reset.done[item] = 0;
    if (reset.best && rem == 0)
        reset.best[item] = kNoLatency;
    for (uint64_t i = t; i < reset.n_winners; i += per_item * count) {
        Winner w;
        w.L = kNoLatency;
        w.pad = 0;
        w.x = ~0ull;
        reset.winners[i] = w;
    }
    uint32_t inst, capacity;
    uint64_t lambda;
    if (raw.budget) {
        // Queries in device memory: prepared here; item's first thread writes what the scan and
        // the result need.
        // (budget and target first, as in the one-launch scan)
        const uint64_t cap = (uint64_t)raw.units_per_gpu * raw.budget[item];
        lambda = raw.target[item];
        inst = raw.inst ? raw.inst[item] : item;
        const bool bad = inst >= raw.B;
        inst = bad ? 0u : inst;
        capacity = cap > kCapacityMax ? kCapacityMax : (uint32_t)cap;
        if (rem == 0) {
            raw.q_inst[item] = inst;
            raw.q_cap[item] = capacity;
            raw.q_lambda[item] = (uint32_t)lambda;
            raw.invalid[item] = bad ? 1u : 0u;
        }
    } else {
        uint32_t lam;
        load_query(q, item, inst, capacity, lam);
        lambda = lam;
    }

    const OptionTerm term = option_term(sp, tb, inst, m, o, (uint32_t)lambda);
    const uint64_t c = term.c;
    const bool ok = term.ok, thr = term.thr;
    const uint32_t tau = term.tau;
    const uint32_t u = term.u;
    const bool usable = ok && thr;
    const uint32_t units = usable ? u : kSentinelUnits;
    rec[t] = make_uint2(usable ? (uint32_t)c : 0u, units);
    ext[t] = make_uint2((uint32_t)tau, u | ((uint32_t)ok << 16) | ((uint32_t)thr << 17));
    if (inner && sp.M >= 2 && m == sp.M - 2) {
        const uint32_t stride = inner_stride(sp.O);
        uint2 *row = inner + (uint64_t)item * stride;
        row[o] = make_uint2(usable ? (uint32_t)c : 0u, (uint32_t)((int32_t)capacity - (int32_t)units));
        // Padding up to a multiple of 16 records: never feasible (no lane's units fit).
        for (uint32_t pad = sp.O + o; pad < stride; pad += sp.O)
            row[pad] = make_uint2(0u, (uint32_t)kNeverFits);
    }
}


// ---------------------------------------------------------------------------------------------
// 2a. Row-minimum scan (default).
//
// Candidates are grouped in "rows": the digits o_0..o_{M-3} are fixed (their latency sum oc and
// share units ou are wave-uniform, in SGPRs) and o_{M-2} (the "inner" LLM, index j) and
// o_{M-1} (the "last" LLM) vary.  Lane l owns the last LLM's options l, l+64, ... (S per lane),
// whose records stay in VGPRs for the whole kernel.  With w = u_last + ou per lane and the
// inner record (c_j, y_j = capacity - u_j) read with scalar loads, candidate (j, lane option)
// is feasible iff w <= y_j, and its latency is oc + c_last + c_j, where oc + c_last is the
// same for all j of the row.  So the lane's best candidate of the row is found by
//     bq = min over feasible j of c_j
// which costs two VALU operations per candidate: v_cmpx (feasibility into EXEC) and v_min_u32
// (EXEC restored by one scalar move).
//
// The argmin index is recovered exactly at the end.  Candidate indices order as (row, j,
// option), and a wave walks its rows in increasing order.  Each lane-slot keeps its smallest
// row latency oc + c_last + bq and the first row reaching it (a later row replaces it only
// when strictly smaller).  At the end each wave takes its smallest latency L* and the lowest
// row reaching it; the block takes the smallest (L*, row) over its waves, (Lb, rb), and all of
// its waves scan their share of row rb again for the lowest feasible j with c_j = Lb - oc -
// c_last per lane-slot; the smallest (j, option) completes the block's lowest index reaching
// Lb.
//
// Work distribution.  Either each wave owns a fixed range of whole rows, or (DYNAMIC) a block
// owns a range of sub-rows -- a row may be split into consecutive ranges of the inner LLM's
// records -- and its waves claim them one at a time from an LDS counter.  A SIMD favours its
// older waves when issuing, so with fixed ranges the younger waves of a small search finish
// late while the SIMD idles; claiming lets every wave of a block finish within one sub-row of
// the others.

// One record (c, y) against every slot of the lane.  A lane's slots are ordered by share units
// (w_0 <= w_1 <= ...), so the feasible lanes of slot s+1 are a subset of those of slot s: each
// v_cmpx narrows EXEC to (w_s <= y), v_min_u32 folds c into bq_s on exactly those lanes, and one
// scalar move restores EXEC after the last slot.  Per candidate: one compare, one minimum.
// The compiler treats each asm statement as opaque and separates consecutive ones by a wait
// state, so the hot loop issues several records per statement.
#define ALP_CM(Y, C, W, B)                                                                         \
    "v_cmpx_ge_i32_e32 vcc, %[" Y "], %[" W "]\n\t"                                                \
    "v_min_u32_e32 %[" B "], %[" C "], %[" B "]\n\t"
#define ALP_RESTORE "s_mov_b64 exec, %[full]\n\t"

__device__ __forceinline__ void masked_min_step(uint32_t (&bq)[1], const int32_t (&w)[1],
                                                uint32_t y, uint32_t c, uint64_t full)
{
    asm volatile(ALP_CM("y", "c", "w0", "b0") ALP_RESTORE
                 : [b0] "+v"(bq[0])
                 : [y] "s"(y), [c] "s"(c), [w0] "v"(w[0]), [full] "s"(full)
                 : "vcc");
}

__device__ __forceinline__ void masked_min_step(uint32_t (&bq)[2], const int32_t (&w)[2],
                                                uint32_t y, uint32_t c, uint64_t full)
{
    asm volatile(ALP_CM("y", "c", "w0", "b0") ALP_CM("y", "c", "w1", "b1") ALP_RESTORE
                 : [b0] "+v"(bq[0]), [b1] "+v"(bq[1])
                 : [y] "s"(y), [c] "s"(c), [w0] "v"(w[0]), [w1] "v"(w[1]), [full] "s"(full)
                 : "vcc");
}

__device__ __forceinline__ void masked_min_step(uint32_t (&bq)[4], const int32_t (&w)[4],
                                                uint32_t y, uint32_t c, uint64_t full)
{
    asm volatile(ALP_CM("y", "c", "w0", "b0") ALP_CM("y", "c", "w1", "b1")
                 ALP_CM("y", "c", "w2", "b2") ALP_CM("y", "c", "w3", "b3") ALP_RESTORE
                 : [b0] "+v"(bq[0]), [b1] "+v"(bq[1]), [b2] "+v"(bq[2]), [b3] "+v"(bq[3])
                 : [y] "s"(y), [c] "s"(c), [w0] "v"(w[0]), [w1] "v"(w[1]), [w2] "v"(w[2]),
                   [w3] "v"(w[3]), [full] "s"(full)
                 : "vcc");
}

__device__ __forceinline__ void masked_min_step(uint32_t (&bq)[8], const int32_t (&w)[8],
                                                uint32_t y, uint32_t c, uint64_t full)
{
    asm volatile(ALP_CM("y", "c", "w0", "b0") ALP_CM("y", "c", "w1", "b1")
                 ALP_CM("y", "c", "w2", "b2") ALP_CM("y", "c", "w3", "b3")
                 ALP_CM("y", "c", "w4", "b4") ALP_CM("y", "c", "w5", "b5")
                 ALP_CM("y", "c", "w6", "b6") ALP_CM("y", "c", "w7", "b7") ALP_RESTORE
                 : [b0] "+v"(bq[0]), [b1] "+v"(bq[1]), [b2] "+v"(bq[2]), [b3] "+v"(bq[3]),
                   [b4] "+v"(bq[4]), [b5] "+v"(bq[5]), [b6] "+v"(bq[6]), [b7] "+v"(bq[7])
                 : [y] "s"(y), [c] "s"(c), [w0] "v"(w[0]), [w1] "v"(w[1]), [w2] "v"(w[2]),
                   [w3] "v"(w[3]), [w4] "v"(w[4]), [w5] "v"(w[5]), [w6] "v"(w[6]),
                   [w7] "v"(w[7]), [full] "s"(full)
                 : "vcc");
}

#define ALP_ARGS8(v)                                                                               \
    [y0] "s"(v[0].y), [c0] "s"(v[0].x), [y1] "s"(v[1].y), [c1] "s"(v[1].x), [y2] "s"(v[2].y),      \
        [c2] "s"(v[2].x), [y3] "s"(v[3].y), [c3] "s"(v[3].x), [y4] "s"(v[4].y), [c4] "s"(v[4].x),  \
        [y5] "s"(v[5].y), [c5] "s"(v[5].x), [y6] "s"(v[6].y), [c6] "s"(v[6].x), [y7] "s"(v[7].y),  \
        [c7] "s"(v[7].x)

// Eight consecutive records (v[0..7]) for lanes with one or two slots.
__device__ __forceinline__ void masked_min_8(uint32_t (&bq)[1], const int32_t (&w)[1],
                                             const uint2 (&v)[8], uint64_t full)
{
#define ALP_R1(T) ALP_CM("y" #T, "c" #T, "w0", "b0") ALP_RESTORE
    asm volatile(ALP_R1(0) ALP_R1(1) ALP_R1(2) ALP_R1(3) ALP_R1(4) ALP_R1(5) ALP_R1(6) ALP_R1(7)
                 : [b0] "+v"(bq[0])
                 : [w0] "v"(w[0]), [full] "s"(full), ALP_ARGS8(v)
                 : "vcc");
#undef ALP_R1
}

__device__ __forceinline__ void masked_min_8(uint32_t (&bq)[2], const int32_t (&w)[2],
                                             const uint2 (&v)[8], uint64_t full)
{
#define ALP_R2(T) ALP_CM("y" #T, "c" #T, "w0", "b0") ALP_CM("y" #T, "c" #T, "w1", "b1") ALP_RESTORE
    asm volatile(ALP_R2(0) ALP_R2(1) ALP_R2(2) ALP_R2(3) ALP_R2(4) ALP_R2(5) ALP_R2(6) ALP_R2(7)
                 : [b0] "+v"(bq[0]), [b1] "+v"(bq[1])
                 : [w0] "v"(w[0]), [w1] "v"(w[1]), [full] "s"(full), ALP_ARGS8(v)
                 : "vcc");
#undef ALP_R2
}

template <int S>
__device__ __forceinline__ void masked_min_8(uint32_t (&bq)[S], const int32_t (&w)[S],
                                             const uint2 (&v)[8], uint64_t full)
{
#pragma unroll
    for (int t = 0; t < 8; ++t)
        masked_min_step(bq, w, v[t].y, v[t].x, full);
}

// Outer-digit latency and share-unit sums of row r (digits o_0..o_{M-3} of r, base O), least
// significant digit (k = n_outer - 1) first.
template <typename Int>
__device__ __forceinline__ void outer_sums_t(const uint2 *R, uint32_t O, uint32_t n_outer, Int r,
                                             uint32_t &oc, int32_t &ou)
{
    oc = 0;
    ou = 0;
#pragma unroll
    for (int k = (int)kMaxOuter - 1; k >= 0; --k) {
        if ((uint32_t)k < n_outer) {
            const uint32_t d = (uint32_t)(r % O);
            r /= O;
            const uint2 v = R[(uint64_t)k * O + d];
            oc += v.x;
            ou += (int32_t)v.y;
        }
    }
}

// 32-bit division whenever r allows it.
__device__ __forceinline__ void outer_sums(const uint2 *R, uint32_t O, uint32_t n_outer,
                                           uint64_t r, uint32_t &oc, int32_t &ou)
{
    if ((r >> 32) == 0)
        outer_sums_t<uint32_t>(R, O, n_outer, (uint32_t)r, oc, ou);
    else
        outer_sums_t<uint64_t>(R, O, n_outer, r, oc, ou);
}

// One record (c, y) at inner index j against every slot of the lane, for the end-of-wave
// re-scan: where the slot is feasible (w_s <= y) and c equals the slot's target, jf_s takes
// min(jf_s, j).  A slot that needs nothing has w_s above every y.
template <int S>
__device__ __forceinline__ void masked_find_step(uint32_t (&jf)[S], const int32_t (&w)[S],
                                                 const uint32_t (&target)[S], uint32_t y,
                                                 uint32_t c, uint32_t j, uint64_t full)
{
#pragma unroll
    for (int s = 0; s < S; ++s)
        asm volatile("v_cmpx_ge_i32_e32 vcc, %[y], %[w]\n\t"
                     "v_cmpx_eq_u32_e32 vcc, %[c], %[t]\n\t"
                     "v_min_u32_e32 %[f], %[j], %[f]\n\t" ALP_RESTORE
                     : [f] "+v"(jf[s])
                     : [y] "s"(y), [c] "s"(c), [j] "s"(j), [w] "v"(w[s]), [t] "v"(target[s]),
                       [full] "s"(full)
                     : "vcc");
}

// NOUT >= 0: the number of outer digits (M - 2) is fixed at compile time; NOUT < 0: any M.
// Scalar loads of records the same kernel wrote (the one-launch form): the compiler would read
// memory written earlier in the kernel with vector loads and move every value to a scalar
// register on its own, so these loads are spelled out.  The block's stores have reached L2
// (waited for before its barrier) and no scalar cache line of the region was read before them.
typedef uint32_t u32x16 __attribute__((ext_vector_type(16)));

// A wave-uniform address as a scalar value (every lane holds the same pointer).
__device__ __forceinline__ const uint2 *uniform_ptr(const uint2 *p)
{
    const uint64_t a = (uint64_t)p;
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)a);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));
    return (const uint2 *)(((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ void scalar_load16(const uint2 *p, uint2 (&a)[8], uint2 (&b)[8])
{
    u32x16 x, y;
    asm volatile("s_load_dwordx16 %0, %2, 0x0\n\t"
                 "s_load_dwordx16 %1, %2, 0x40\n\t"
                 "s_waitcnt lgkmcnt(0)"
                 : "=s"(x), "=s"(y)
                 : "s"(uniform_ptr(p))
                 : "memory");
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        a[t] = make_uint2(x[2 * t], x[2 * t + 1]);
        b[t] = make_uint2(y[2 * t], y[2 * t + 1]);
    }
}

// The same, and lane 0 claims a sub-row meanwhile (see piped_min_8_claim): one wait for both.
__device__ __forceinline__ void scalar_load16_claim(const uint2 *p, uint2 (&a)[8], uint2 (&b)[8],
                                                    uint32_t la, uint64_t full,
                                                    uint32_t &claimed)
{
    u32x16 x, y;
    asm volatile("s_load_dwordx16 %[x], %[p], 0x0\n\t"
                 "s_load_dwordx16 %[y], %[p], 0x40\n\t"
                 "s_mov_b64 exec, 1\n\t"
                 "ds_add_rtn_u32 %[cl], %[la], %[one]\n\t"
                 "s_mov_b64 exec, %[full]\n\t"
                 "s_waitcnt lgkmcnt(0)"
                 : [x] "=&s"(x), [y] "=&s"(y), [cl] "=&v"(claimed)
                 : [p] "s"(uniform_ptr(p)), [la] "v"(la), [one] "v"(1u), [full] "s"(full)
                 : "memory");
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        a[t] = make_uint2(x[2 * t], x[2 * t + 1]);
        b[t] = make_uint2(y[2 * t], y[2 * t + 1]);
    }
}

__device__ __forceinline__ uint2 scalar_load1(const uint2 *p)
{
    uint64_t v;
    asm volatile("s_load_dwordx2 %0, %1, 0x0\n\t"
                 "s_waitcnt lgkmcnt(0)"
                 : "=s"(v)
                 : "s"(uniform_ptr(p))
                 : "memory");
    return make_uint2((uint32_t)v, (uint32_t)(v >> 32));
}

// Software-pipelined record loop (one or two slots per lane): each statement loads the next 8
// records while it processes the current 8 (x[2t] = c, x[2t + 1] = y of record t), and waits for
// the load only at its end, so a wave waits for the scalar cache once per row rather than once
// per 16 records.  Loaded registers are complete when the statement ends: nothing in flight
// crosses a statement.
#define ALP_ARGSX(x)                                                                               \
    [c0] "s"(x[0]), [y0] "s"(x[1]), [c1] "s"(x[2]), [y1] "s"(x[3]), [c2] "s"(x[4]),                \
        [y2] "s"(x[5]), [c3] "s"(x[6]), [y3] "s"(x[7]), [c4] "s"(x[8]), [y4] "s"(x[9]),            \
        [c5] "s"(x[10]), [y5] "s"(x[11]), [c6] "s"(x[12]), [y6] "s"(x[13]), [c7] "s"(x[14]),       \
        [y7] "s"(x[15])
#define ALP_P1(T) ALP_CM("y" #T, "c" #T, "w0", "b0") ALP_RESTORE
#define ALP_P2(T) ALP_CM("y" #T, "c" #T, "w0", "b0") ALP_CM("y" #T, "c" #T, "w1", "b1") ALP_RESTORE
#define ALP_P1_8 ALP_P1(0) ALP_P1(1) ALP_P1(2) ALP_P1(3) ALP_P1(4) ALP_P1(5) ALP_P1(6) ALP_P1(7)
#define ALP_P2_8 ALP_P2(0) ALP_P2(1) ALP_P2(2) ALP_P2(3) ALP_P2(4) ALP_P2(5) ALP_P2(6) ALP_P2(7)

__device__ __forceinline__ u32x16 piped_min_8(uint32_t (&bq)[1], const int32_t (&w)[1],
                                              const u32x16 &x, uint64_t full, const uint2 *pn)
{
    u32x16 nx;
    asm volatile("s_load_dwordx16 %[nx], %[pn], 0x0\n\t" ALP_P1_8 "s_waitcnt lgkmcnt(0)"
                 : [nx] "=&s"(nx), [b0] "+v"(bq[0])
                 : [pn] "s"(uniform_ptr(pn)), [w0] "v"(w[0]), [full] "s"(full), ALP_ARGSX(x)
                 : "vcc", "memory");
    return nx;
}

__device__ __forceinline__ u32x16 piped_min_8(uint32_t (&bq)[2], const int32_t (&w)[2],
                                              const u32x16 &x, uint64_t full, const uint2 *pn)
{
    u32x16 nx;
    asm volatile("s_load_dwordx16 %[nx], %[pn], 0x0\n\t" ALP_P2_8 "s_waitcnt lgkmcnt(0)"
                 : [nx] "=&s"(nx), [b0] "+v"(bq[0]), [b1] "+v"(bq[1])
                 : [pn] "s"(uniform_ptr(pn)), [w0] "v"(w[0]), [w1] "v"(w[1]), [full] "s"(full),
                   ALP_ARGSX(x)
                 : "vcc", "memory");
    return nx;
}

// The same, and lane 0 claims the wave's next sub-row meanwhile: an LDS atomic add of 1 at byte
// address la (lane 0's result in claimed), complete when the statement ends.
__device__ __forceinline__ u32x16 piped_min_8_claim(uint32_t (&bq)[1], const int32_t (&w)[1],
                                                    const u32x16 &x, uint64_t full,
                                                    const uint2 *pn, uint32_t la,
                                                    uint32_t &claimed)
{
    u32x16 nx;
    asm volatile("s_load_dwordx16 %[nx], %[pn], 0x0\n\t"
                 "s_mov_b64 exec, 1\n\t"
                 "ds_add_rtn_u32 %[cl], %[la], %[one]\n\t"
                 "s_mov_b64 exec, %[full]\n\t" ALP_P1_8 "s_waitcnt lgkmcnt(0)"
                 : [nx] "=&s"(nx), [cl] "=&v"(claimed), [b0] "+v"(bq[0])
                 : [pn] "s"(uniform_ptr(pn)), [la] "v"(la), [one] "v"(1u), [w0] "v"(w[0]),
                   [full] "s"(full), ALP_ARGSX(x)
                 : "vcc", "memory");
    return nx;
}

__device__ __forceinline__ u32x16 piped_min_8_claim(uint32_t (&bq)[2], const int32_t (&w)[2],
                                                    const u32x16 &x, uint64_t full,
                                                    const uint2 *pn, uint32_t la,
                                                    uint32_t &claimed)
{
    u32x16 nx;
    asm volatile("s_load_dwordx16 %[nx], %[pn], 0x0\n\t"
                 "s_mov_b64 exec, 1\n\t"
                 "ds_add_rtn_u32 %[cl], %[la], %[one]\n\t"
                 "s_mov_b64 exec, %[full]\n\t" ALP_P2_8 "s_waitcnt lgkmcnt(0)"
                 : [nx] "=&s"(nx), [cl] "=&v"(claimed), [b0] "+v"(bq[0]), [b1] "+v"(bq[1])
                 : [pn] "s"(uniform_ptr(pn)), [la] "v"(la), [one] "v"(1u), [w0] "v"(w[0]),
                   [w1] "v"(w[1]), [full] "s"(full), ALP_ARGSX(x)
                 : "vcc", "memory");
    return nx;
}

// The last 8 records of a row (nothing more to load).
__device__ __forceinline__ void piped_last_8(uint32_t (&bq)[1], const int32_t (&w)[1],
                                             const u32x16 &x, uint64_t full)
{
    asm volatile(ALP_P1_8
                 : [b0] "+v"(bq[0])
                 : [w0] "v"(w[0]), [full] "s"(full), ALP_ARGSX(x)
                 : "vcc");
}

__device__ __forceinline__ void piped_last_8(uint32_t (&bq)[2], const int32_t (&w)[2],
                                             const u32x16 &x, uint64_t full)
{
    asm volatile(ALP_P2_8
                 : [b0] "+v"(bq[0]), [b1] "+v"(bq[1])
                 : [w0] "v"(w[0]), [w1] "v"(w[1]), [full] "s"(full), ALP_ARGSX(x)
                 : "vcc");
}
#undef ALP_P1_8
#undef ALP_P2_8
#undef ALP_P1
#undef ALP_P2
#undef ALP_ARGSX

// A row's first 8 inner records and its NOUT outer records (digits o_0..o_{NOUT-1}) in one
// round trip; the outer records' latency and share-unit sums go to oc and ou.
template <int NOUT, int N>
__device__ __forceinline__ u32x16 row_start_loads(const uint2 *R, uint32_t O,
                                                  const uint32_t (&digit)[N], const uint2 *first,
                                                  uint32_t &oc, int32_t &ou)
{
    static_assert(NOUT >= 0 && NOUT <= 3 && NOUT <= N, "outer digits loaded together");
    u32x16 x;
    uint64_t o[3] = {0, 0, 0};
    const uint2 *pa = uniform_ptr(first);
    if constexpr (NOUT == 0) {
        asm volatile("s_load_dwordx16 %[a], %[pa], 0x0\n\t"
                     "s_waitcnt lgkmcnt(0)"
                     : [a] "=&s"(x)
                     : [pa] "s"(pa)
                     : "memory");
    } else if constexpr (NOUT == 1) {
        asm volatile("s_load_dwordx2 %[o0], %[p0], 0x0\n\t"
                     "s_load_dwordx16 %[a], %[pa], 0x0\n\t"
                     "s_waitcnt lgkmcnt(0)"
                     : [a] "=&s"(x), [o0] "=&s"(o[0])
                     : [pa] "s"(pa), [p0] "s"(uniform_ptr(R + digit[0]))
                     : "memory");
    } else if constexpr (NOUT == 2) {
        asm volatile("s_load_dwordx2 %[o0], %[p0], 0x0\n\t"
                     "s_load_dwordx2 %[o1], %[p1], 0x0\n\t"
                     "s_load_dwordx16 %[a], %[pa], 0x0\n\t"
                     "s_waitcnt lgkmcnt(0)"
                     : [a] "=&s"(x), [o0] "=&s"(o[0]), [o1] "=&s"(o[1])
                     : [pa] "s"(pa), [p0] "s"(uniform_ptr(R + digit[0])),
                       [p1] "s"(uniform_ptr(R + O + digit[1]))
                     : "memory");
    } else {
        asm volatile("s_load_dwordx2 %[o0], %[p0], 0x0\n\t"
                     "s_load_dwordx2 %[o1], %[p1], 0x0\n\t"
                     "s_load_dwordx2 %[o2], %[p2], 0x0\n\t"
                     "s_load_dwordx16 %[a], %[pa], 0x0\n\t"
                     "s_waitcnt lgkmcnt(0)"
                     : [a] "=&s"(x), [o0] "=&s"(o[0]), [o1] "=&s"(o[1]), [o2] "=&s"(o[2])
                     : [pa] "s"(pa), [p0] "s"(uniform_ptr(R + digit[0])),
                       [p1] "s"(uniform_ptr(R + O + digit[1])),
                       [p2] "s"(uniform_ptr(R + 2 * O + digit[2]))
                     : "memory");
    }
    oc = 0;
    ou = 0;
#pragma unroll
    for (int k = 0; k < NOUT; ++k) {
        oc += (uint32_t)o[k];
        ou += (int32_t)(uint32_t)(o[k] >> 32);
    }
    return x;
}

// FUSED: the one-launch form (see FusedArgs) -- the block first computes its item's option
// terms into its own region (the inner LLM's records with the query's capacity folded in, as
// the option-term kernel writes them), waits for the stores to reach L2 and reads them back
// through the scalar cache like the separate kernel's; the finish keeps the item's winner in one
// 64-bit word.  Requires no pair table and fewer than 2^32 candidates per item.
template <int S, int NOUT, bool DYNAMIC, bool FUSED>
__global__ void __launch_bounds__(1024) __attribute__((amdgpu_waves_per_eu(S <= 2 ? 8 : 1)))
scan_min_kernel(const uint2 *__restrict__ rec, const uint2 *__restrict__ inner_all, QueryDev q,
                uint32_t M, uint32_t O, uint64_t rows, uint64_t rows_per_wave, uint32_t chunks,
                uint32_t blocks_per_item, uint32_t nblocks, Winner *__restrict__ winners,
                FinishArgs fa, uint32_t pair, FusedArgs fz)
{
    // pair = 1: the inner table is the pair table of LLMs M-3 and M-2 (index j = j3 * O + j2,
    // O^2 records), so rows fix the M - 3 outer digits; candidates keep their index order.
    // `rows` counts sub-rows: each row (one choice of the outer digits) may be split into
    // `chunks` consecutive ranges of the inner LLM's records (DYNAMIC only), so that small
    // spaces still give every wave several sub-rows; candidates stay in index order (row,
    // record, option).  Without DYNAMIC, chunks = 1 and each wave walks a fixed range of rows.
    if constexpr (FUSED) {
        // Kernel arguments are read through the scalar cache, a memory round trip for each
        // 64-byte line first read.  One field of every line the prologue reads (the space, M
        // and O, the block regions, the queries and tables, the block size) is taken here as
        // an input of an empty statement, so all lines arrive in the first round trip rather
        // than one after another, some after the query.
        asm volatile("" ::"s"(M), "s"(rows), "s"(nblocks), "s"(fa.sp.tp8), "s"(fa.out),
                     "s"(fz.tb.rate), "s"(fz.raw.budget), "s"(fz.regions), "s"(fz.best),
                     "s"(blockDim.x));
    }
    if (!DYNAMIC)
        chunks = 1;
    const uint32_t lb = xcd_logical_block(blockIdx.x, nblocks);
    const uint32_t item = lb / blocks_per_item;
    const uint32_t sub = lb - item * blocks_per_item;
    const uint32_t lane = threadIdx.x & 63;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint32_t wpb = blockDim.x >> 6;
    int32_t capacity;
    const uint2 *R, *inner;
    uint32_t f_inst = 0;          // FUSED: the query
    uint64_t f_lambda = 0;
    bool f_rejected = false;
    FusedLds flds{};
    const uint2 *s_inner = nullptr;     // FUSED: the inner LLM's records, in LDS
    __shared__ uint2 s_last[FUSED ? ALP_MAX_OPTIONS : 1];
    // FUSED: the item's profile curves and their deployability in dynamic LDS (layout as
    // fused_lds_bytes counts it); tp * q of every (tp, share) pair, each LLM's inputs and the
    // reciprocals of 1000 d (see FusedLds).
    extern __shared__ uint4 s_dyn[];
    __shared__ LlmInputs s_llm[FUSED ? ALP_MAX_LLMS : 1];
    __shared__ uint32_t s_tpq[FUSED ? ALP_MAX_TP * ALP_MAX_FRAC : 1];
    __shared__ double s_inv_dd[FUSED ? ALP_MAX_REPLICAS : 1];
    if constexpr (FUSED) {
        uint32_t cap;
        if (fz.raw.budget) {
            // budget and target read first: the instance's read is conditional, and a
            // conditional read is waited for where the paths join
            const uint64_t c64 = (uint64_t)fz.raw.units_per_gpu * fz.raw.budget[item];
            f_lambda = fz.raw.target[item];
            f_inst = fz.raw.inst ? fz.raw.inst[item] : item;
            f_rejected = f_inst >= fz.raw.B;
            f_inst = f_rejected ? 0u : f_inst;
            cap = c64 > kCapacityMax ? kCapacityMax : (uint32_t)c64;
        } else {
            uint32_t lam;
            load_query(q, item, f_inst, cap, lam);
            f_lambda = lam;
        }
        capacity = (int32_t)cap;
        uint2 *blk = fz.regions + (uint64_t)blockIdx.x * fz.region;
        uint2 *blk_inner = blk + M * O;
        const uint32_t stride = inner_stride(O);
        // The item's profile curves (one per LLM, tp and share; shared by the replica counts)
        // staged in LDS by one load per point, all in flight together, the rates padded to
        // ALP_MAX_POINTS points with the last one; each curve's deployability, tp * q of every
        // pair, each LLM's inputs and the reciprocals of 1000 d.
        const SpaceDev &sp = fa.sp;
        const uint32_t K = sp.K, curves = M * sp.n_tp * sp.n_fq, pairs = sp.n_tp * sp.n_fq;
        const uint64_t base = (uint64_t)f_inst * curves;
        uint8_t *s_base = reinterpret_cast<uint8_t *>(s_dyn);
        uint32_t *s_rate = reinterpret_cast<uint32_t *>(s_base);
        uint32_t *s_lat = reinterpret_cast<uint32_t *>(s_base + fused_lds_lat_offset(sp));
        uint8_t *s_deploy = s_base + fused_lds_deploy_offset(sp);
        uint2 *s_inner_w = reinterpret_cast<uint2 *>(s_base + fused_lds_inner_offset(sp));
        uint2 *s_ext_w = reinterpret_cast<uint2 *>(s_base + fused_lds_ext_offset(sp));
        flds = FusedLds{s_rate, s_lat, s_deploy, s_tpq, s_llm, s_inv_dd, s_ext_w};
        s_inner = s_inner_w;
        // Stores point a (rate padded past K - 1).
        const uint64_t lm0 = (uint64_t)f_inst * M;
        auto put_point = [&](uint32_t a, uint32_t rate, uint32_t lat) {
            const uint32_t c = a / K, k = a - c * K;
            s_lat[a] = lat;
            s_rate[c * ALP_MAX_POINTS + k] = rate;
            if (k == K - 1)
                for (uint32_t kk = K; kk < ALP_MAX_POINTS; ++kk)
                    s_rate[c * ALP_MAX_POINTS + kk] = rate;
        };
        // tp and q of curve (or pair) a.
        auto curve_tp = [&](uint32_t a) { return sp.tp(a % pairs / sp.n_fq); };
        auto curve_fq = [&](uint32_t a) { return sp.fq(a % pairs % sp.n_fq); };
        // Every thread's first point, curve, pair and LLM are read together, at indices clamped
        // into the item's tables (a thread past the end reads the last entry and stores
        // nothing), so that the reads are in flight at once; further points and curves (blocks
        // smaller than the item's tables) follow.  Waves past every table (points are the most
        // entries, but for the D reciprocals) skip it.
        const uint32_t points = curves * K;
        if (wave * 64 < (points > sp.D ? points : sp.D)) {
            const uint32_t t = threadIdx.x;
            const uint32_t ap = t < points ? t : points - 1, ac = t < curves ? t : curves - 1;
            const uint32_t am = t < M ? t : M - 1;
            const uint32_t rate = fz.tb.rate[base * K + ap], lat = fz.tb.lat[base * K + ap];
            const uint8_t allowed = fz.tb.allowed[base + ac];
            const uint64_t W = fz.tb.W[lm0 + ac / pairs];
            const uint32_t n = fz.tb.n[lm0 + am], p = fz.tb.p[lm0 + am];
            const uint32_t tp = curve_tp(ac), fq = curve_fq(ac);
            if (t < sp.D)
                s_inv_dd[t] = recip_low<1, 40>(1000u * (t + 1));
            if (t < points)
                put_point(t, rate, lat);
            if (t < curves)
                s_deploy[t] = deployable(sp, fz.tb.H, allowed != 0, W, tp * fq);
            if (t < pairs)
                s_tpq[t] = tp * fq;                  // curve t < pairs is pair t's
            if (t < M)
                s_llm[t] = llm_inputs(n, p);
        }
        for (uint32_t a = threadIdx.x + blockDim.x; a < curves * K; a += blockDim.x)
            put_point(a, fz.tb.rate[base * K + a], fz.tb.lat[base * K + a]);
        for (uint32_t a = threadIdx.x + blockDim.x; a < curves; a += blockDim.x)
            s_deploy[a] = deployable(sp, fz.tb.H, fz.tb.allowed[base + a] != 0,
                                     fz.tb.W[lm0 + a / pairs], curve_tp(a) * curve_fq(a));
        __syncthreads();
        for (uint32_t a = threadIdx.x; a < M * O; a += blockDim.x) {
            const uint32_t m = div_by(a, sp.mul_O), o = a - m * O;
            const OptionTerm t = flds.term(sp, m, o, (uint32_t)f_lambda);
            s_ext_w[a] = make_uint2(t.tau, t.u);
            const bool usable = t.ok && t.thr;
            const uint2 r = make_uint2(usable ? t.c : 0u, usable ? t.u : kSentinelUnits);
            blk[a] = r;
            if (m == M - 1)
                s_last[o] = r;
            if (M >= 2 && m == M - 2) {
                const uint2 in = make_uint2(r.x, (uint32_t)((int32_t)cap - (int32_t)r.y));
                blk_inner[o] = in;
                s_inner_w[o] = in;
            }
        }
        for (uint32_t a = O + threadIdx.x; a < stride; a += blockDim.x) {
            blk_inner[a] = make_uint2(0u, (uint32_t)kNeverFits);
            s_inner_w[a] = make_uint2(0u, (uint32_t)kNeverFits);
        }
        // The region is read back through the scalar cache, which reads L2: wait until every
        // store has reached it, then let the other waves go.
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        R = blk;
        inner = blk_inner;
    } else {
        capacity = (int32_t)query_value(q.capacity, q.cap1, item);
        R = rec + (uint64_t)item * M * O;
        inner = inner_all + (uint64_t)item * (pair ? pair_stride(O) : inner_stride(O));
    }

    // The last LLM's options of this lane: lane, lane + 64, ...  They are processed in order
    // of share units (insertion sort of the S values held by the lane), which lets the hot
    // loop nest the EXEC masks of the slots; o_last keeps each slot's option index.
    const uint2 *last = R + (uint64_t)(M - 1) * O;
    uint32_t c_last[S], o_last[S];
    int32_t u_last[S];
#pragma unroll
    for (int s = 0; s < S; ++s) {
        const uint32_t o = lane + 64u * s;
        o_last[s] = o;
        if (o < O) {
            const uint2 v = FUSED ? s_last[o] : last[o];
            c_last[s] = v.x;
            u_last[s] = (int32_t)v.y;
        } else {
            c_last[s] = 0;
            u_last[s] = 1 << 28;              // above every capacity, even after adding ou
        }
    }
#pragma unroll
    for (int a = 1; a < S; ++a) {
#pragma unroll
        for (int b = a; b > 0; --b) {
            const bool swap = u_last[b] < u_last[b - 1];
            const int32_t u0 = u_last[b - 1], u1 = u_last[b];
            const uint32_t c0 = c_last[b - 1], c1 = c_last[b], o0 = o_last[b - 1], o1 = o_last[b];
            u_last[b - 1] = swap ? u1 : u0;
            u_last[b] = swap ? u0 : u1;
            c_last[b - 1] = swap ? c1 : c0;
            c_last[b] = swap ? c0 : c1;
            o_last[b - 1] = swap ? o1 : o0;
            o_last[b] = swap ? o0 : o1;
        }
    }
    const bool has_inner = M >= 2;
    const uint32_t n_inner_padded = pair ? pair_stride(O) : inner_stride(O);
    const uint32_t chunk_len = n_inner_padded / chunks;   // a multiple of 16
    const uint32_t n_inner = has_inner ? (pair ? O * O : O) : 1;
    constexpr int NMAX = NOUT >= 0 ? NOUT : (int)kMaxOuter;
    // One or two slots and at most three outer digits: the pipelined record loop -- except
    // for the one-launch form with claimed sub-rows (the single small searches, rows of a few
    // hundred records at 4 waves per SIMD), where its extra scalar registers cost more reloads
    // per row than the loads it overlaps save.
    constexpr bool kPiped = S <= 2 && NOUT >= 0 && NOUT <= 3 && !(FUSED && DYNAMIC);
    const uint32_t n_outer =
        NOUT >= 0 ? (uint32_t)NOUT : (M >= 2 + pair ? M - 2 - pair : 0);

    uint32_t waveL = kNoLatency;
    uint64_t waveX = ~0ull;
    // Without DYNAMIC, wave gw owns the sub-rows [r_begin, r_end).  With DYNAMIC, the block owns
    // [r_begin, r_end) (rows_per_wave * wpb sub-rows, fewer than 2^32) and hands them out one at
    // a time from an LDS counter: waves that the SIMD issues less often (younger waves) simply
    // take fewer sub-rows, so the waves of a block finish together.  Wave w starts with sub-row
    // w; each wave's sub-rows increase, as the first-row bookkeeping below requires.
    const uint64_t gw = (uint64_t)sub * wpb + wave;
    const uint64_t per = DYNAMIC ? rows_per_wave * wpb : rows_per_wave;
    const uint64_t r_begin = (DYNAMIC ? (uint64_t)sub : gw) * per;
    const uint64_t r_end = r_begin + per < rows ? r_begin + per : rows;
    __shared__ uint32_t s_next, s_ended;
    if (threadIdx.x == 0) {
        s_next = wpb;
        s_ended = 0;
    }
    __syncthreads();
    const uint32_t first = DYNAMIC ? wave : 0u;

    const uint64_t full = __builtin_amdgcn_read_exec();
    uint32_t bestL[S], bestR[S];              // per lane-slot: smallest row latency, its first row
#pragma unroll
    for (int s = 0; s < S; ++s) {
        bestL[s] = kNoLatency;
        bestR[s] = 0;
    }
    uint32_t Lstar = kNoLatency;              // the wave's smallest latency
    if (r_begin + first < r_end) {
        uint32_t digit[NMAX > 0 ? NMAX : 1];
        uint32_t chunk = 0;
        // Division by O and by chunks through reciprocals: q = mulhi(n, floor((2^32-1)/d)) is
        // floor(n/d) or one less (n < 2^32), and one correction step makes it exact.
        const uint32_t inv_o = 0xFFFFFFFFu / O, inv_ch = 0xFFFFFFFFu / chunks;
        auto divmod = [](uint32_t n, uint32_t d, uint32_t inv, uint32_t &r) {
            uint32_t q = __umulhi(n, inv);
            r = n - q * d;
            if (r >= d) {
                ++q;
                r -= d;
            }
            return q;
        };
        if (!DYNAMIC) {
            uint64_t rr = r_begin;
#pragma unroll
            for (int k = NMAX - 1; k >= 0; --k) {
                digit[k] = 0;
                if (NOUT >= 0 || (uint32_t)k < n_outer) {
                    digit[k] = (uint32_t)(rr % O);
                    rr /= O;
                }
            }
        }
        uint32_t cur = first, next = 0;
        for (uint32_t rr = 0;; ++rr) {
            if (DYNAMIC) {
                if (r_begin + cur >= r_end)
                    break;
                uint32_t row = divmod((uint32_t)(r_begin + cur), chunks, inv_ch, chunk);
#pragma unroll
                for (int k = NMAX - 1; k >= 0; --k) {
                    digit[k] = 0;
                    if (NOUT >= 0 || (uint32_t)k < n_outer)
                        row = divmod(row, O, inv_o, digit[k]);
                }
            } else if (rr >= (uint32_t)(r_end - r_begin)) {
                break;
            }
            const uint32_t tag = DYNAMIC ? cur : rr;
            // The row's inner records (the table is padded to a multiple of 16 with records no
            // lane can use).
            const uint2 *const begin = DYNAMIC ? inner + chunk * chunk_len : inner;
            const uint2 *const last16 = (DYNAMIC ? begin + chunk_len : inner + n_inner_padded) - 16;
            uint32_t oc = 0;
            int32_t ou = 0;
            int32_t w[S];
            uint32_t bq[S];
            auto row_init = [&]() {
#pragma unroll
                for (int s = 0; s < S; ++s) {
                    w[s] = u_last[s] + ou;
                    bq[s] = kNoLatency;
                }
            };
            bool done_row = false;
            if constexpr (kPiped) {
                if (has_inner) {
                    // 8 records per statement, the next 8 loading meanwhile.  The claim goes
                    // out 8 records before the row's end, within a statement that completes
                    // it.
                    u32x16 a = row_start_loads<NOUT>(R, O, digit, begin, oc, ou);
                    row_init();
                    const uint2 *p = begin;
                    for (; p != last16; p += 16) {
                        const u32x16 b = piped_min_8(bq, w, a, full, p + 8);
                        a = piped_min_8(bq, w, b, full, p + 16);
                    }
                    if constexpr (DYNAMIC) {
                        typedef __attribute__((address_space(3))) uint32_t lds_u32;
                        const uint32_t la = (uint32_t)(uintptr_t)(lds_u32 *)&s_next;
                        const u32x16 b = piped_min_8_claim(bq, w, a, full, p + 8, la, next);
                        piped_last_8(bq, w, b, full);
                    } else {
                        const u32x16 b = piped_min_8(bq, w, a, full, p + 8);
                        piped_last_8(bq, w, b, full);
                    }
                    done_row = true;
                }
            }
            if (!done_row) {
#pragma unroll
                for (int k = 0; k < NMAX; ++k) {
                    if (NOUT >= 0 || (uint32_t)k < n_outer) {
                        const uint2 *rp = R + (uint64_t)k * O + digit[k];
                        const uint2 v = FUSED ? scalar_load1(rp) : *rp;
                        oc += v.x;
                        ou += (int32_t)v.y;
                    }
                }
                row_init();
            }
            if (done_row) {
            } else if (has_inner) {
                // 16 records per iteration: two 64-byte scalar loads issued together, so the
                // loop's own scalar work stays small next to the 2 x 16 x S VALU operations.
                auto batch = [&](const uint2 *p) {
                    uint2 v0[8], v1[8];
                    if constexpr (FUSED) {
                        scalar_load16(p, v0, v1);
                    } else {
#pragma unroll
                        for (int t = 0; t < 8; ++t) {
                            v0[t] = p[t];
                            v1[t] = p[8 + t];
                        }
                    }
                    masked_min_8(bq, w, v0, full);
                    masked_min_8(bq, w, v1, full);
                };
                for (const uint2 *p = begin; p != last16; p += 16)
                    batch(p);
                // Claim the wave's next sub-row with the last 16 records; claiming earlier
                // would commit a slowly issued wave to more work than the others while the
                // block's range runs out.  The one-launch form issues the claim with the
                // records' loads, under one wait.
                if constexpr (FUSED && DYNAMIC) {
                    typedef __attribute__((address_space(3))) uint32_t lds_u32;
                    const uint32_t la = (uint32_t)(uintptr_t)(lds_u32 *)&s_next;
                    uint2 v0[8], v1[8];
                    scalar_load16_claim(last16, v0, v1, la, full, next);
                    masked_min_8(bq, w, v0, full);
                    masked_min_8(bq, w, v1, full);
                } else {
                    if (DYNAMIC && lane == 0)
                        next = atomicAdd(&s_next, 1u);
                    batch(last16);
                }
            } else {
                if (DYNAMIC && lane == 0)
                    next = atomicAdd(&s_next, 1u);
                masked_min_step(bq, w, (uint32_t)capacity, 0u, full);
            }
            // Row minimum per lane-slot (saturating: no feasible j leaves kNoLatency).
#pragma unroll
            for (int s = 0; s < S; ++s) {
                const uint32_t L = __builtin_elementwise_add_sat(bq[s], c_last[s] + oc);
                const bool better = L < bestL[s];
                bestL[s] = better ? L : bestL[s];
                bestR[s] = better ? tag : bestR[s];
            }
            if (DYNAMIC) {
                cur = (uint32_t)__builtin_amdgcn_readfirstlane(next);
                continue;
            }
            // Next row: the odometer on the outer digits moves on (integer carry, stays in
            // scalar registers).
            uint32_t inc = 1;
#pragma unroll
            for (int k = NMAX - 1; k >= 0; --k) {
                if (NOUT >= 0 || (uint32_t)k < n_outer) {
                    const uint32_t d = digit[k] + inc;
                    inc = d == O ? 1u : 0u;
                    digit[k] = inc ? 0u : d;
                }
            }
        }

        uint32_t lmin = kNoLatency;
#pragma unroll
        for (int s = 0; s < S; ++s)
            lmin = bestL[s] < lmin ? bestL[s] : lmin;
        Lstar = wave_min_u32(lmin);
    }
    // The item's best latency so far as this wave sees it at the end of its loop (the loads of
    // a block's last waves see what blocks that ended earlier published).  A block whose
    // minimum lies above it cannot hold the item's winner and skips its re-scan.
    // Only the block's last wave to end its loop reads it: one coherent load per block, taken
    // as late as the block allows.
    uint32_t hint = kNoLatency;
    if (lane == 0 && blocks_per_item > 1 && atomicAdd(&s_ended, 1u) == wpb - 1) {
        if constexpr (FUSED) {
            const unsigned long long w =
                __hip_atomic_load(&fz.best[item], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            hint = w ? (uint32_t)(~w >> 32) : kNoLatency;
        } else {
            hint = __hip_atomic_load(&fa.best[item], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    // The wave's lowest sub-row reaching L* (its lane-slots' first rows at L*), as a sub-row
    // index of the item, and that row's outer sums, loaded now while the block's other waves
    // finish (claimed sub-rows number fewer than 2^32).
    uint64_t rwave = ~0ull;
    uint32_t oc_w = 0;
    int32_t ou_w = 0;
    if (Lstar != kNoLatency) {
        uint32_t rmin = 0xFFFFFFFFu;
#pragma unroll
        for (int s = 0; s < S; ++s)
            if (bestL[s] == Lstar && bestR[s] < rmin)
                rmin = bestR[s];
        rwave = r_begin + wave_min_u32(rmin);
        outer_sums(R, O, n_outer, DYNAMIC ? (uint32_t)rwave / chunks : rwave, oc_w, ou_w);
    }
    // The block's smallest latency Lb and the lowest sub-row rb reaching it: the (L*, row)
    // minimum over the waves.  Sub-rows are in candidate-index order, so the block's winner
    // is the lowest candidate of sub-row rb with latency Lb.
    __shared__ uint32_t s_wave_L[16], s_wave_oc[16], s_wave_H[16];
    __shared__ int32_t s_wave_ou[16];
    __shared__ uint64_t s_wave_R[16];
    if (lane == 0) {
        s_wave_L[wave] = Lstar;
        s_wave_R[wave] = rwave;
        s_wave_oc[wave] = oc_w;
        s_wave_ou[wave] = ou_w;
        s_wave_H[wave] = hint;
    }
    __syncthreads();
    // Lane k reads wave k's pair; one wave reduction (in every wave) gives the block's.
    const uint32_t mineL = lane < wpb ? s_wave_L[lane] : kNoLatency;
    const uint64_t mineR = lane < wpb ? s_wave_R[lane] : ~0ull;
    uint32_t Lblock = mineL;
    uint64_t rb = mineR;
    wave_min(Lblock, rb);
    const uint32_t block_hint = wave_min_u32(lane < wpb ? s_wave_H[lane] : kNoLatency);
    // Uniform over the block: every wave reduced the same LDS words.
    const bool held = Lblock != kNoLatency && Lblock <= block_hint;
    if (held) {
        // Every wave of the block searches its share of sub-row rb (4 records per step,
        // steps interleaved over the waves) for the lowest feasible j of each lane-slot with
        // c_j = Lb - oc - c_last: no wave re-walks a whole sub-row alone.  A feasible match
        // has latency exactly Lb, since no sum of usable terms reaches 2^32 - 1 (a wrapped
        // target is never met).  Sub-rows are distinct across waves, so exactly one wave
        // reported rb; its outer sums are taken from LDS.
        const uint64_t r = DYNAMIC ? (uint32_t)rb / chunks : rb;
        const uint32_t j0 = DYNAMIC ? (uint32_t)rb % chunks * chunk_len : 0u;
        const uint32_t src = (uint32_t)__builtin_ctzll(__ballot(mineL == Lblock && mineR == rb));
        const uint32_t oc = s_wave_oc[src];
        const int32_t ou = s_wave_ou[src];
        uint32_t target[S], jf[S];
        int32_t w[S];
#pragma unroll
        for (int s = 0; s < S; ++s) {
            target[s] = Lblock - c_last[s] - oc;
            w[s] = u_last[s] + ou;
            jf[s] = kNoLatency;
        }
        if (has_inner) {
            for (uint32_t jb = j0 + 4u * wave; jb < j0 + chunk_len; jb += 4u * wpb) {
                uint2 v[4];
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    if constexpr (FUSED) {
                        // the same LDS word in every lane: move it to scalar registers
                        const uint2 l = s_inner[jb + t];
                        v[t] = make_uint2((uint32_t)__builtin_amdgcn_readfirstlane((int)l.x),
                                          (uint32_t)__builtin_amdgcn_readfirstlane((int)l.y));
                    } else {
                        v[t] = inner[jb + t];
                    }
                }
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    masked_find_step(jf, w, target, v[t].y, v[t].x, jb + t, full);
            }
        } else if (wave == 0) {
            // One LLM: the row is the last LLM's options alone (j = 0).
#pragma unroll
            for (int s = 0; s < S; ++s)
                jf[s] = w[s] <= capacity && c_last[s] + oc == Lblock ? 0u : kNoLatency;
        }
        uint64_t xmin = ~0ull;
#pragma unroll
        for (int s = 0; s < S; ++s) {
            if (jf[s] != kNoLatency) {
                const uint64_t x = (r * n_inner + jf[s]) * (uint64_t)O + o_last[s];
                xmin = x < xmin ? x : xmin;
            }
        }
        waveL = Lblock;
        waveX = wave_min_u64(xmin);
    }
    if constexpr (FUSED)
        block_finish_fused(waveL, waveX, item, sub, blocks_per_item, fa, fz, flds, f_rejected,
                           block_hint, held);
    else
        block_finish(waveL, waveX, item, sub, blocks_per_item, winners, fa, block_hint, held);
}

// ---------------------------------------------------------------------------------------------
// 2c. Exact-tracking lane scan (cross-check variant).
//
// A wave walks "rows": fixed digits o_0..o_{M-3} (their c and u sums are wave-uniform and live
// in SGPRs) and every o_{M-2} in turn (one uniform 8-byte record per step, fetched with scalar
// loads).  Lane l owns the last LLM's options l, l+64, ... (S of them, records held in VGPRs for
// the whole kernel).  For a prefix with latency sum pc and remaining share units slack, the
// lane's candidate is feasible iff u_last <= slack and has latency pc + c_last; because c_last
// is constant per lane, "better than the lane's best so far" is pc < best_pc.  Per candidate:
// two compares, one mask AND (scalar), two selects.  Within a row a lane scans prefixes in
// increasing index order and only a strictly smaller pc replaces its best, so ties keep the
// lowest index; rows and lanes are merged lexicographically on (L, x).
template <int S>
__global__ void __launch_bounds__(1024)
scan_lane_kernel(const uint2 *__restrict__ rec, QueryDev q, uint32_t M, uint32_t O,
                 uint64_t rows, uint64_t rows_per_wave, uint32_t blocks_per_item,
                 uint32_t nblocks, Winner *__restrict__ winners, FinishArgs fa)
{
    const uint32_t lb = xcd_logical_block(blockIdx.x, nblocks);
    const uint32_t item = lb / blocks_per_item;
    const uint32_t sub = lb - item * blocks_per_item;
    const uint32_t lane = threadIdx.x & 63;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint32_t wpb = blockDim.x >> 6;
    const int32_t capacity = (int32_t)query_value(q.capacity, q.cap1, item);
    const uint2 *R = rec + (uint64_t)item * M * O;

    // The last LLM's options owned by this lane.
    const uint2 *last = R + (uint64_t)(M - 1) * O;
    uint32_t c_last[S];
    int32_t u_last[S];
#pragma unroll
    for (int s = 0; s < S; ++s) {
        const uint32_t o = lane + 64u * s;
        if (o < O) {
            const uint2 v = last[o];
            c_last[s] = v.x;
            u_last[s] = (int32_t)v.y;
        } else {
            c_last[s] = 0;
            u_last[s] = 0x7FFFFFFF;          // never within any slack
        }
    }

    // The LLM before the last one varies inside a row; with a single LLM there is no prefix:
    // one row of one empty prefix (inner record (0, 0)).
    const bool has_inner = M >= 2;
    const uint2 *inner = R + (uint64_t)(has_inner ? M - 2 : 0) * O;
    const uint32_t n_inner = has_inner ? O : 1;
    const uint32_t n_outer = M >= 2 ? M - 2 : 0;

    uint32_t bestL = kNoLatency;
    uint64_t bestX = ~0ull;

    const uint64_t gw = (uint64_t)sub * wpb + wave;
    const uint64_t r_begin = gw * rows_per_wave;
    const uint64_t r_end = r_begin + rows_per_wave < rows ? r_begin + rows_per_wave : rows;

    if (r_begin < r_end) {
        uint32_t digit[kMaxOuter];
        {
            uint64_t rr = r_begin;
#pragma unroll
            for (int k = (int)kMaxOuter - 1; k >= 0; --k) {
                digit[k] = 0;
                if ((uint32_t)k < n_outer) {
                    digit[k] = (uint32_t)(rr % O);
                    rr /= O;
                }
            }
        }
        for (uint64_t r = r_begin; r < r_end; ++r) {
            uint32_t oc = 0;
            int32_t ou = 0;
#pragma unroll
            for (uint32_t k = 0; k < kMaxOuter; ++k) {
                if (k < n_outer) {
                    const uint2 v = R[(uint64_t)k * O + digit[k]];
                    oc += v.x;
                    ou += (int32_t)v.y;
                }
            }
            const int32_t base_slack = capacity - ou;

            uint32_t best_pc[S], best_j[S];
#pragma unroll
            for (int s = 0; s < S; ++s) {
                best_pc[s] = kNoLatency;
                best_j[s] = 0;
            }
            auto step = [&](const uint2 v, const uint32_t jj) {
                const uint32_t pc = oc + v.x;
                const int32_t slack = base_slack - (int32_t)v.y;
#pragma unroll
                for (int s = 0; s < S; ++s) {
                    const bool take = (u_last[s] <= slack) & (pc < best_pc[s]);
                    best_pc[s] = take ? pc : best_pc[s];
                    best_j[s] = take ? jj : best_j[s];
                }
            };
            if (has_inner) {
                uint32_t jb = 0;
                for (; jb + 8 <= n_inner; jb += 8) {
#pragma unroll
                    for (uint32_t t = 0; t < 8; ++t)
                        step(inner[jb + t], jb + t);
                }
                for (; jb < n_inner; ++jb)
                    step(inner[jb], jb);
            } else {
                step(make_uint2(0u, 0u), 0u);
            }

            // Merge the row into the lane's running best.
#pragma unroll
            for (int s = 0; s < S; ++s) {
                if (best_pc[s] != kNoLatency) {
                    const uint32_t L = best_pc[s] + c_last[s];
                    const uint64_t x = ((r * n_inner + best_j[s]) * (uint64_t)O) + lane + 64u * s;
                    if (lex_less(L, x, bestL, bestX)) {
                        bestL = L;
                        bestX = x;
                    }
                }
            }
            // Next row: odometer on the outer digits (last outer digit fastest).
            bool carry = true;
#pragma unroll
            for (int k = (int)kMaxOuter - 1; k >= 0; --k) {
                if ((uint32_t)k < n_outer && carry) {
                    ++digit[k];
                    if (digit[k] == O)
                        digit[k] = 0;
                    else
                        carry = false;
                }
            }
        }
    }
    block_finish(bestL, bestX, item, sub, blocks_per_item, winners, fa);
}

// ---------------------------------------------------------------------------------------------
// 2b. Thread-per-candidate scan (cross-check variant): each thread evaluates a
// contiguous index range from the LDS-staged option table, decoding the start index once and
// counting the digits up from there.
__global__ void __launch_bounds__(1024)
scan_flat_kernel(const uint2 *__restrict__ rec, QueryDev q, uint32_t M, uint32_t O, uint64_t N,
                 uint64_t per_thread, uint32_t blocks_per_item, uint32_t nblocks,
                 Winner *__restrict__ winners, FinishArgs fa)
{
    extern __shared__ uint2 table[];
    const uint32_t lb = xcd_logical_block(blockIdx.x, nblocks);
    const uint32_t item = lb / blocks_per_item;
    const uint32_t sub = lb - item * blocks_per_item;
    const uint32_t capacity = query_value(q.capacity, q.cap1, item);
    const uint2 *R = rec + (uint64_t)item * M * O;
    for (uint32_t a = threadIdx.x; a < M * O; a += blockDim.x)
        table[a] = R[a];
    __syncthreads();

    uint32_t bestL = kNoLatency;
    uint64_t bestX = ~0ull;
    const uint64_t t = (uint64_t)sub * blockDim.x + threadIdx.x;
    const uint64_t x0 = t * per_thread;
    const uint64_t x1 = x0 + per_thread < N ? x0 + per_thread : N;
    if (x0 < x1) {
        uint32_t digit[ALP_MAX_LLMS];
        uint64_t rr = x0;
#pragma unroll
        for (int m = ALP_MAX_LLMS - 1; m >= 0; --m) {
            digit[m] = 0;
            if ((uint32_t)m < M) {
                digit[m] = (uint32_t)(rr % O);
                rr /= O;
            }
        }
        for (uint64_t x = x0; x < x1; ++x) {
            uint32_t L = 0, U = 0;
#pragma unroll
            for (uint32_t m = 0; m < ALP_MAX_LLMS; ++m) {
                if (m < M) {
                    const uint2 v = table[m * O + digit[m]];
                    L += v.x;
                    U += v.y;
                }
            }
            if (U <= capacity && L < bestL) {
                bestL = L;
                bestX = x;
            }
            bool carry = true;
#pragma unroll
            for (int m = ALP_MAX_LLMS - 1; m >= 0; --m) {
                if ((uint32_t)m < M && carry) {
                    ++digit[m];
                    if (digit[m] == O)
                        digit[m] = 0;
                    else
                        carry = false;
                }
            }
        }
    }
    block_finish(bestL, bestX, item, sub, blocks_per_item, winners, fa);
}

// ---------------------------------------------------------------------------------------------
// Evaluation of listed candidates (one thread each).
__global__ void __launch_bounds__(256)
eval_kernel(SpaceDev sp, uint32_t capacity, const uint2 *__restrict__ rec,
            const uint2 *__restrict__ ext, const uint64_t *__restrict__ idx, uint64_t count,
            alp_eval_t *__restrict__ out)
{
    const uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= count)
        return;
    uint64_t rr = idx[t];
    bool ok = true, thr = true;
    uint32_t L = 0, T = 0xFFFFFFFFu, U = 0;
    for (int m = (int)sp.M - 1; m >= 0; --m) {
        const uint32_t o = (uint32_t)(rr % sp.O);
        rr /= sp.O;
        const uint64_t a = (uint64_t)m * sp.O + o;
        const uint2 e = ext[a];
        ok &= ((e.y >> 16) & 1u) != 0;
        thr &= ((e.y >> 17) & 1u) != 0;
        U += e.y & 0xFFFFu;
        T = e.x < T ? e.x : T;
        L += rec[a].x;
    }
    alp_eval_t r;
    r.flags = (uint32_t)ok | ((uint32_t)thr << 1) | ((uint32_t)(U <= capacity) << 2);
    r.latency_us = (ok && thr) ? L : kNoLatency;
    r.throughput_milli = ok ? T : 0u;
    r.gpu_units = U;
    out[t] = r;
}

// ---------------------------------------------------------------------------------------------
// Largest reachable T_w within the budget, one block per item.  T_w >= t is reachable iff the
// cheapest deployable, fitting options with tau >= t of all LLMs together fit:
// need(t) = sum_m min{u : ok, tau >= t} <= capacity.  The maximum is one of the options' own
// taus.  Per LLM, the deployable options are ranked by tau descending (ties by option index)
// and a running minimum of their units is taken along that order; need(t) for each candidate
// t then costs one binary search per LLM.  O(M * O * (O + M log O)) work per item, in LDS; one
// thread per option where the block allows.
constexpr uint32_t kTmaxStride = 8;     // options per LLM padded to this (whole 16-byte reads)

__host__ __device__ inline uint32_t tmax_stride(uint32_t O)
{
    return (O + kTmaxStride - 1) / kTmaxStride * kTmaxStride;
}

__global__ void __launch_bounds__(1024)
tmax_kernel(SpaceDev sp, QueryDev q, const uint2 *__restrict__ ext, uint32_t *__restrict__ out)
{
    extern __shared__ uint4 t_lds4[];
    constexpr uint16_t kUnusable = 0xFFFFu;   // share units are at most 64 * 16 * 16 = 16384
    constexpr uint64_t kNoKey = ~0ull;        // not deployable (or padding): ranks last
    const uint32_t item = blockIdx.x;
    const uint32_t O = sp.O, MO = sp.M * O, P = tmax_stride(O), MP = sp.M * P;
    // Each option's rank key: (2^32 - 1 - tau) << 32 | index, so that ascending keys are tau
    // descending then index ascending, and one 64-bit compare orders two options.
    uint64_t *key = reinterpret_cast<uint64_t *>(t_lds4);   // [M][P]
    uint32_t *stau = reinterpret_cast<uint32_t *>(key + MP); // [M][P] deployable taus, descending
    uint16_t *units = (uint16_t *)(stau + MP);           // [M][P] share units, or kUnusable
    uint16_t *smin = units + MP;                         // [M][P] running minimum of units
    __shared__ uint32_t s_count[ALP_MAX_LLMS];
    __shared__ uint32_t s_best[16];
    const uint2 *E = ext + (uint64_t)item * MO;
    if (threadIdx.x < ALP_MAX_LLMS)
        s_count[threadIdx.x] = 0;
    for (uint32_t a = threadIdx.x; a < MP; a += blockDim.x) {
        const uint32_t m = a / P, o = a - m * P;
        uint2 e = make_uint2(0u, 0u);                    // padding: not deployable
        if (o < O)
            e = E[m * O + o];
        const bool usable = (e.y >> 16) & 1u;
        key[a] = usable ? (uint64_t)(0xFFFFFFFFu - e.x) << 32 | o : kNoKey;
        units[a] = usable ? (uint16_t)(e.y & 0xFFFFu) : kUnusable;
    }
    __syncthreads();
    // Rank of each deployable option within its LLM: the keys of the LLM below its own, read
    // two at a time (a compare and an add each).
    for (uint32_t a = threadIdx.x; a < MP; a += blockDim.x) {
        const uint64_t mine = key[a];
        if (mine == kNoKey)
            continue;
        const uint32_t m = a / P;
        const uint4 *K2 = reinterpret_cast<const uint4 *>(key + m * P);
        uint32_t rank = 0;
#pragma unroll 4
        for (uint32_t j2 = 0; j2 < P / 2; ++j2) {
            const uint4 kk = K2[j2];
            rank += ((uint64_t)kk.y << 32 | kk.x) < mine;
            rank += ((uint64_t)kk.w << 32 | kk.z) < mine;
        }
        stau[m * P + rank] = 0xFFFFFFFFu - (uint32_t)(mine >> 32);
        smin[m * P + rank] = units[a];
        atomicAdd(&s_count[m], 1u);
    }
    __syncthreads();
    // Running minimum along each LLM's order: wave w takes LLMs w, w + waves, ...; lane l holds
    // a contiguous run of the order, minimum within the run, then a prefix minimum of the runs
    // across the lanes.
    const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    for (uint32_t m = wave; m < sp.M; m += nw) {
        const uint32_t n = s_count[m], per = (n + 63) / 64;
        uint16_t *S = smin + m * P;
        const uint32_t lo = lane * per, hi = lo + per < n ? lo + per : n;
        uint32_t run = 0xFFFFFFFFu;
        for (uint32_t k = lo; k < hi; ++k)
            run = S[k] < run ? S[k] : run;
        // Inclusive prefix minimum over the lanes by DPP (row shifts by 1, 2, 4, 8, then lane
        // 15 into rows 1 and 3 and lane 31 into rows 2 and 3; lanes a move does not reach keep
        // the identity), then the exclusive one by a shift of the whole wave.
        uint32_t before = run;
        auto step = [&](auto c, auto rm) {
            constexpr int C = decltype(c)::value, RM = decltype(rm)::value;
            const uint32_t o = dpp_mov<C, RM>(0xFFFFFFFFu, before);
            before = o < before ? o : before;
        };
        step(std::integral_constant<int, 0x111>{}, std::integral_constant<int, 0xF>{});
        step(std::integral_constant<int, 0x112>{}, std::integral_constant<int, 0xF>{});
        step(std::integral_constant<int, 0x114>{}, std::integral_constant<int, 0xF>{});
        step(std::integral_constant<int, 0x118>{}, std::integral_constant<int, 0xF>{});
        step(std::integral_constant<int, 0x142>{}, std::integral_constant<int, 0xA>{});
        step(std::integral_constant<int, 0x143>{}, std::integral_constant<int, 0xC>{});
        uint32_t acc = dpp_mov<0x138>(0xFFFFFFFFu, before);
        for (uint32_t k = lo; k < hi; ++k) {
            acc = S[k] < acc ? S[k] : acc;
            S[k] = (uint16_t)acc;
        }
    }
    __syncthreads();
    const uint64_t capacity = (uint64_t)query_value(q.capacity, q.cap1, item);
    uint32_t best = 0;
    for (uint32_t a = threadIdx.x; a < MP; a += blockDim.x) {
        if (key[a] == kNoKey)
            continue;
        const uint32_t t = 0xFFFFFFFFu - (uint32_t)(key[a] >> 32);
        if (t <= best)
            continue;
        uint64_t need = 0;
        bool reachable = true;
        for (uint32_t m = 0; m < sp.M && reachable; ++m) {
            // options of m with tau >= t: the first c of its descending order
            uint32_t lo = 0, hi = s_count[m];
            const uint32_t *S = stau + m * P;
            while (lo < hi) {
                const uint32_t mid = (lo + hi) >> 1;
                if (S[mid] >= t)
                    lo = mid + 1;
                else
                    hi = mid;
            }
            if (lo == 0)
                reachable = false;
            else
                need += smin[m * P + lo - 1];
        }
        if (reachable && need <= capacity)
            best = t;
    }
    best = wave_max_u32(best);
    if (lane == 0)
        s_best[wave] = best;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t b = 0;
        for (uint32_t w = 0; w < nw; ++w)
            b = s_best[w] > b ? s_best[w] : b;
        out[item] = b;
    }
}

// ---------------------------------------------------------------------------------------------
// Launchers.  The option-term and scan launches take optional start/stop events that the
// dispatch itself stamps with the kernel's begin and end (no separate event packets between
// the kernels, which would leave the GPU idle for microseconds per search).

namespace {

// One thread per pair record: LLM M-3's record from rec (c, units or sentinel) and LLM M-2's
// from inner (c, Q*G - units); the sum of two usable terms stays below 2^32 - 1, and any unusable
// option leaves Q*G - units far below zero, so the pair never fits.
__global__ void __launch_bounds__(256)
pair_terms_kernel(uint32_t M, uint32_t O, uint32_t count, const uint2 *__restrict__ rec,
                  const uint2 *__restrict__ inner, uint2 *__restrict__ pair)
{
    const uint32_t stride = pair_stride(O);
    const uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (uint64_t)count * stride)
        return;
    const uint32_t item = (uint32_t)(t / stride), j = (uint32_t)(t - (uint64_t)item * stride);
    uint2 out = make_uint2(0u, (uint32_t)kNeverFits);
    if (j < O * O) {
        const uint32_t j3 = j / O, j2 = j - j3 * O;
        const uint2 a = rec[((uint64_t)item * M + (M - 3)) * O + j3];
        const uint2 b = inner[(uint64_t)item * inner_stride(O) + j2];
        out = make_uint2(a.x + b.x, (uint32_t)((int32_t)b.y - (int32_t)a.y));
    }
    pair[t] = out;
}

}  // namespace

hipError_t launch_pair_terms(const SpaceDev &sp, uint32_t count, const uint2 *rec,
                             const uint2 *inner, uint2 *pair, hipStream_t st)
{
    const uint64_t total = (uint64_t)count * pair_stride(sp.O);
    if (total == 0 || sp.M < 3)
        return hipSuccess;
    hipLaunchKernelGGL(pair_terms_kernel, dim3((uint32_t)((total + 255) / 256)), dim3(256), 0, st,
                       sp.M, sp.O, count, rec, inner, pair);
    return hipGetLastError();
}

hipError_t launch_option_terms(const SpaceDev &sp, const TablesDev &tb, const QueryDev &q,
                               uint32_t count, uint2 *rec, uint2 *ext, uint2 *inner,
                               const ScanReset &reset, hipStream_t st, const RawQueries *raw,
                               hipEvent_t t0, hipEvent_t t1)
{
    const uint64_t total = (uint64_t)count * sp.M * sp.O;
    if (total == 0)
        return hipSuccess;
    const uint32_t blocks = (uint32_t)((total + 255) / 256);
    RawQueries none{};
    hipExtLaunchKernelGGL(option_terms_kernel, dim3(blocks), dim3(256), 0, st, t0, t1, 0, sp, tb, q,
                          count, rec, ext, inner, reset, raw ? *raw : none);
    return hipGetLastError();
}

template <int S>
static hipError_t launch_lane(const SpaceDev &sp, const QueryDev &q, uint32_t count,
                              const uint2 *rec, const uint2 *inner, const ScanGeometry &g,
                              Winner *winners, const FinishArgs &fa, hipStream_t st,
                              hipEvent_t t0, hipEvent_t t1, const FusedArgs *fzp)
{
    FusedArgs fz{};
    if (fzp)
        fz = *fzp;
    const uint32_t nblocks = count * g.blocks_per_item;
    if (g.variant == 3)
        hipExtLaunchKernelGGL(HIP_KERNEL_NAME(scan_lane_kernel<S>), dim3(nblocks), dim3(g.threads),
                              0, st, t0, t1, 0, rec, q, sp.M, sp.O, g.rows, g.rows_per_wave,
                              g.blocks_per_item, nblocks, winners, fa);
    else {
        const uint32_t n_outer = sp.M >= 2 + g.pair ? sp.M - 2 - g.pair : 0;
#define ALP_LAUNCH_MIN_DF(NO, DYN, FU)                                                             \
    hipExtLaunchKernelGGL(HIP_KERNEL_NAME(scan_min_kernel<S, NO, DYN, FU>), dim3(nblocks),         \
                          dim3(g.threads), FU ? fused_lds_bytes(sp) : 0, st, t0, t1, 0, rec,       \
                          inner, q, sp.M, sp.O, g.rows,                                            \
                          g.rows_per_wave, DYN ? g.chunks : 1u, g.blocks_per_item, nblocks,        \
                          winners, fa, g.pair, fz)
#define ALP_LAUNCH_MIN(NO)                                                                         \
    do {                                                                                           \
        if (g.fused) {                                                                             \
            if (g.dynamic)                                                                         \
                ALP_LAUNCH_MIN_DF(NO, true, true);                                                 \
            else                                                                                   \
                ALP_LAUNCH_MIN_DF(NO, false, true);                                                \
        } else if (g.dynamic) {                                                                    \
            ALP_LAUNCH_MIN_DF(NO, true, false);                                                    \
        } else {                                                                                   \
            ALP_LAUNCH_MIN_DF(NO, false, false);                                                   \
        }                                                                                          \
    } while (0)
        switch (n_outer) {
        case 0: ALP_LAUNCH_MIN(0); break;
        case 1: ALP_LAUNCH_MIN(1); break;
        case 2: ALP_LAUNCH_MIN(2); break;
        case 3: ALP_LAUNCH_MIN(3); break;
        default: ALP_LAUNCH_MIN(-1); break;
        }
#undef ALP_LAUNCH_MIN
#undef ALP_LAUNCH_MIN_DF
    }
    return hipGetLastError();
}

hipError_t launch_scan(const SpaceDev &sp, const QueryDev &q, uint32_t count, const uint2 *rec,
                       const uint2 *inner, const ScanGeometry &g, Winner *winners,
                       const FinishArgs &fa, hipStream_t st, hipEvent_t t0, hipEvent_t t1,
                       const FusedArgs *fz)
{
    if (g.fused && (!fz || g.variant != 1 || g.pair))
        return hipErrorInvalidValue;
    if (count == 0)
        return hipSuccess;
    if (g.variant == 2) {
        uint64_t N = 1;
        for (uint32_t m = 0; m < sp.M; ++m)
            N *= sp.O;
        const uint32_t nblocks = count * g.blocks_per_item;
        const size_t lds = (size_t)sp.M * sp.O * sizeof(uint2);
        hipExtLaunchKernelGGL(scan_flat_kernel, dim3(nblocks), dim3(g.threads), lds, st, t0, t1, 0,
                              rec, q, sp.M, sp.O, N, g.per_thread, g.blocks_per_item, nblocks,
                              winners, fa);
        return hipGetLastError();
    }
    switch (g.slots) {
    case 1: return launch_lane<1>(sp, q, count, rec, inner, g, winners, fa, st, t0, t1, fz);
    case 2: return launch_lane<2>(sp, q, count, rec, inner, g, winners, fa, st, t0, t1, fz);
    case 4: return launch_lane<4>(sp, q, count, rec, inner, g, winners, fa, st, t0, t1, fz);
    case 8: return launch_lane<8>(sp, q, count, rec, inner, g, winners, fa, st, t0, t1, fz);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_eval(const SpaceDev &sp, uint32_t capacity, const uint2 *rec, const uint2 *ext,
                       const uint64_t *idx, uint64_t count, alp_eval_t *out, hipStream_t st)
{
    if (count == 0)
        return hipSuccess;
    const uint64_t blocks = (count + 255) / 256;
    hipLaunchKernelGGL(eval_kernel, dim3((uint32_t)blocks), dim3(256), 0, st, sp, capacity, rec,
                       ext, idx, count, out);
    return hipGetLastError();
}

hipError_t launch_tmax(const SpaceDev &sp, const QueryDev &q, uint32_t count, const uint2 *ext,
                       uint32_t *out, hipStream_t st)
{
    if (count == 0)
        return hipSuccess;
    const uint32_t MP = sp.M * tmax_stride(sp.O);
    const size_t lds = (size_t)MP * (sizeof(uint64_t) + sizeof(uint32_t) + 2 * sizeof(uint16_t));
    // one thread per option (padded), in whole waves, 64..1024
    const uint32_t threads = MP >= 1024 ? 1024u : (MP + 63) / 64 * 64;
    hipLaunchKernelGGL(tmax_kernel, dim3(count), dim3(threads), lds, st, sp, q, ext, out);
    return hipGetLastError();
}

int scan_blocks_per_cu(uint32_t variant, uint32_t slots, uint32_t threads, const SpaceDev &sp)
{
    int n = 0;
    hipError_t e = hipErrorInvalidValue;
    if (variant == 2) {
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, scan_flat_kernel, (int)threads,
                                                         (size_t)sp.M * sp.O * sizeof(uint2));
    } else {
        const bool exact = variant == 3;
        const uint32_t no = sp.M >= 2 ? sp.M - 2 : 0;
#define ALP_OCC_MIN(SL)                                                                            \
    (no == 0 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, scan_min_kernel<SL, 0, false, false>, (int)threads, 0) \
   : no == 1 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, scan_min_kernel<SL, 1, false, false>, (int)threads, 0) \
   : no == 2 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, scan_min_kernel<SL, 2, false, false>, (int)threads, 0) \
   : no == 3 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, scan_min_kernel<SL, 3, false, false>, (int)threads, 0) \
             : hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, scan_min_kernel<SL, -1, false, false>, (int)threads, 0))
        switch (slots) {
        case 1: e = exact ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, scan_lane_kernel<1>, (int)threads, 0) : ALP_OCC_MIN(1); break;
        case 2: e = exact ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, scan_lane_kernel<2>, (int)threads, 0) : ALP_OCC_MIN(2); break;
        case 4: e = exact ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, scan_lane_kernel<4>, (int)threads, 0) : ALP_OCC_MIN(4); break;
        case 8: e = exact ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, scan_lane_kernel<8>, (int)threads, 0) : ALP_OCC_MIN(8); break;
        default: break;
        }
#undef ALP_OCC_MIN
    }
    return (e == hipSuccess && n > 0) ? n : 1;
}

}  // namespace alp
