// gfx950 kernels for the workflow statistics of Scepsy (arXiv 2604.15186, Section 4, step 2):
// per LLM m, n_m = calls per workflow request and p_m = request-level parallelism, from
// execution traces (one trace per workflow request; each LLM call has an LLM index and a
// half-open [start, end) interval in microseconds).
//
//   p_m = (sum of m's call durations) / (sum over traces of the time at least one call of m
//         runs), so that n_m * L_m / p_m (Eq. 1) is the time per request during which m is
//         active.  n_m and p_m are reported in thousandths, rounded down.
//
// Kernels:
//   stats_init_kernel        zeroes the per-LLM totals, the error flags and the counters (once;
//                            afterwards the last block of each computation leaves them zeroed).
//   trace_sweep_kernel<MM>   one wave per trace of at most 2,048 calls (MM bounds the number of
//                            LLMs, so the per-LLM state fits in few registers).  A trace already
//                            in order of end time (calls logged on completion) is swept backwards
//                            in rows of 64 consecutive calls, without a sort: a call adds the part
//                            of it before the earliest start of the same LLM's later calls.  Other
//                            traces go to a work list.
//   trace_wave_kernel        instead of the sweep, when the traces come out of end order: one
//                            wave per trace of at most 512 calls sorts its calls by packed key
//                            (llm << 61 | start << 32 | duration, starts within 2^29 us of a
//                            reference) in registers and across lanes -- no LDS, no barrier --
//                            and sweeps them as below; other traces go to the work list.
//   trace_group_kernel<E,NT> the same for traces of 513 to 1,024 calls (two waves each) and of
//                            1,025 to 2,048 (four), 8 keys per thread, the exchanges between
//                            waves through LDS.
//   trace_sort_kernel        the work list: calls sorted by key (llm << 60 | start), packed into
//                            one 64-bit key when the starts span under 2^29 us, with a bitonic
//                            network in registers, across lanes and in LDS; the time covered by
//                            each LLM follows from an exclusive prefix maximum of
//                            (llm << 61 | end) -- an interval adds the part of it beyond the
//                            furthest end of the same LLM's earlier intervals.
//   trace_long_kernel        traces beyond 2,048 calls, sorted the same way in a global scratch
//                            region.
//   In each, per-LLM call counts, durations and covered time are summed per trace and added to
//   one of kStatsCopies copies of the totals with 64-bit atomics (integer sums: the result does
//   not depend on their order).  The last block of the sort and long passes computes n and p
//   per LLM from the totals and writes them with the error flags.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "alp_device.h"
#include "alp_internal.h"

namespace alp {

namespace {

constexpr uint64_t kPad = ~0ull;                       // sorts after every real key
constexpr uint64_t kStartLimit = 1ull << 60;
constexpr uint64_t kDurationLimit = 1ull << 32;
constexpr uint32_t kThreads = 256;
constexpr uint32_t kSortBlocks = 1024;                 // grid of the work-list sort

__global__ void stats_init_kernel(uint64_t *__restrict__ totals, uint32_t words)
{
    for (uint32_t k = threadIdx.x; k < words; k += blockDim.x)
        totals[k] = 0;
}

// Exclusive maximum over the threads' values, in thread order (every thread gets the maximum
// over the threads before it; 0 for thread 0).
__device__ __forceinline__ uint64_t block_exclusive_max(uint64_t v)
{
    __shared__ uint64_t s_wave[kThreads / 64];
    const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint64_t incl = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint64_t o = __shfl_up((unsigned long long)incl, off, 64);
        if (lane >= (uint32_t)off)
            incl = o > incl ? o : incl;
    }
    if (lane == 63)
        s_wave[wave] = incl;
    __syncthreads();
    uint64_t excl = __shfl_up((unsigned long long)incl, 1, 64);
    if (lane == 0)
        excl = 0;
    for (uint32_t w = 0; w < wave; ++w)
        excl = s_wave[w] > excl ? s_wave[w] : excl;
    return excl;
}

// The 32-bit value of lane (lane ^ Q), Q a power of two below 64: DPP quad permutations for 1
// and 2, a swizzle within 32 lanes for 4..16, a lane permute for 32.
template <int Q>
__device__ __forceinline__ uint32_t lane_xor(uint32_t v)
{
    if constexpr (Q == 1)
        return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false);
    else if constexpr (Q == 2)
        return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false);
    else if constexpr (Q < 32)
        return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, 0x1F | (Q << 10));
    else
        return (uint32_t)__builtin_amdgcn_ds_bpermute((int)((threadIdx.x ^ 32u) << 2), (int)v);
}

template <int Q>
__device__ __forceinline__ uint64_t lane_xor64(uint64_t v)
{
    return (uint64_t)lane_xor<Q>((uint32_t)v) | ((uint64_t)lane_xor<Q>((uint32_t)(v >> 32)) << 32);
}

// Bitonic sort of P (a power of two) entries in place, ascending by key then val when val is
// given (keys only otherwise).
template <bool WithVal>
__device__ __forceinline__ void bitonic_sort(uint64_t *key, uint64_t *val, uint32_t P)
{
    for (uint32_t size = 2; size <= P; size <<= 1) {
        for (uint32_t stride = size >> 1; stride > 0; stride >>= 1) {
            for (uint32_t t = threadIdx.x; t < P / 2; t += kThreads) {
                const uint32_t i = 2 * t - (t & (stride - 1));
                const uint32_t j = i + stride;
                const bool up = (i & size) == 0;
                const uint64_t ki = key[i], kj = key[j];
                bool greater = ki > kj;
                uint64_t vi = 0, vj = 0;
                if (WithVal) {
                    vi = val[i];
                    vj = val[j];
                    greater = greater || (ki == kj && vi > vj);
                }
                if (greater == up) {
                    key[i] = kj;
                    key[j] = ki;
                    if (WithVal) {
                        val[i] = vj;
                        val[j] = vi;
                    }
                }
            }
            __syncthreads();
        }
    }
}

// One compare-exchange of the bitonic network seen from one side: keep the minimum (else the
// maximum) of the own and the partner's key.
__device__ __forceinline__ uint64_t keep_one(uint64_t mine, uint64_t other, bool keep_min)
{
    // other < mine selects the minimum where keep_min holds; elsewhere it keeps mine unless
    // other is larger (equal keys: either is the same value).  One compare and a mask test.
    const bool take = (other < mine) == keep_min;
    return take ? other : mine;
}

// Position i is the pair's lower index iff bit `stride` of i is clear, and lies in a run of
// `size` sorted ascending iff bit `size` of i is clear; the lower index of an ascending pair,
// or the upper of a descending one, keeps the minimum.
__device__ __forceinline__ bool keeps_min(uint32_t i, uint32_t stride, uint32_t size)
{
    return ((i & stride) == 0) == ((i & size) == 0);
}

// Exchanges with partner lane (lane ^ Q) for stride Q * E, if that stride occurs in this run.
template <int E, int Q>
__device__ __forceinline__ void lane_stage(uint64_t (&k)[E], uint32_t size, uint32_t t)
{
    constexpr uint32_t stride = (uint32_t)(Q * E);
    if (2 * stride > size)
        return;
    const bool km = keeps_min(t * E, stride, size);   // the same for all E slots
    // Partners of up to 4 slots fetched before any is used: the cross-lane moves' latency
    // overlaps.
#pragma unroll
    for (int e0 = 0; e0 < E; e0 += 4) {
        uint64_t o[4];
#pragma unroll
        for (int e = e0; e < e0 + 4 && e < E; ++e)
            o[e - e0] = lane_xor64<Q>(k[e]);
#pragma unroll
        for (int e = e0; e < e0 + 4 && e < E; ++e)
            k[e] = keep_one(k[e], o[e - e0], km);
    }
}

// Bitonic sort of P = NT E keys held E per thread of NT in registers, ascending by position:
// thread t holds positions t E .. t E + E - 1 (a sort within one wave takes NT = 64 and t = the
// lane, so that no exchange reaches another wave).  An exchange whose partner is in the same
// thread runs in registers, one whose partner is in the same wave by cross-lane moves (lane ^
// stride / E), and only those whose partner is in another wave go through LDS, in a layout
// (slot e of thread t at e * NT + t) where a wave's 64 accesses are consecutive; two LDS
// buffers alternate, so each such exchange needs one barrier.  buf holds 2 P keys.
template <int E, int NT = kThreads>
__device__ __forceinline__ void bitonic_sort_regs(uint64_t (&k)[E], uint64_t *buf, uint32_t P,
                                                  uint32_t t)
{
    uint32_t flip = 0;
    for (uint32_t size = 2; size <= P; size <<= 1) {
        for (uint32_t stride = size >> 1; stride >= (uint32_t)E * 64; stride >>= 1) {
            uint64_t *b = buf + flip * P;
            flip ^= 1u;
#pragma unroll
            for (int e = 0; e < E; ++e)
                b[e * NT + t] = k[e];
            __syncthreads();
            const uint32_t pt = t ^ (stride / E);
            const bool km = keeps_min(t * E, stride, size);
#pragma unroll
            for (int e = 0; e < E; ++e)
                k[e] = keep_one(k[e], b[e * NT + pt], km);
        }
        lane_stage<E, 32>(k, size, t);
        lane_stage<E, 16>(k, size, t);
        lane_stage<E, 8>(k, size, t);
        lane_stage<E, 4>(k, size, t);
        lane_stage<E, 2>(k, size, t);
        lane_stage<E, 1>(k, size, t);
#pragma unroll
        for (int st = E / 2; st >= 1; st >>= 1) {
            if ((uint32_t)(2 * st) > size)
                continue;
#pragma unroll
            for (int e = 0; e < E; ++e) {
                if (e & st)
                    continue;
                const uint64_t a = k[e], b = k[e | st];
                const bool asc = ((t * E + e) & size) == 0;
                const bool swap = (a > b) == asc;         // equal keys: either way
                k[e] = swap ? b : a;
                k[e | st] = swap ? a : b;
            }
        }
    }
}

// The sweep over the sorted calls of one trace: each thread takes a contiguous chunk of the
// first `valid` entries; get(i, m, s, e) yields entry i.  Packed value of a call: (llm << 61 |
// end); the maximum of the packed values before a call has high bits equal to its LLM iff an
// earlier call of the same LLM exists, and then low bits equal to the furthest end among them.
// Per-LLM calls, durations and covered time are added to s_sum.
template <class Get>
__device__ __forceinline__ void sweep(uint32_t P, uint32_t valid, Get get,
                                      unsigned long long *s_sum)
{
    const uint32_t per = P / kThreads, base = threadIdx.x * per;
    uint64_t run = 0;
    for (uint32_t k = 0; k < per && base + k < valid; ++k) {
        uint32_t m;
        uint64_t s, e;
        get(base + k, m, s, e);
        const uint64_t pk = ((uint64_t)m << 61) | e;
        run = pk > run ? pk : run;
    }
    uint64_t prev = block_exclusive_max(run);
    constexpr uint64_t kLow61 = (1ull << 61) - 1;
    uint32_t cur = ~0u;
    uint64_t c_calls = 0, c_busy = 0, c_active = 0;
    auto flush = [&]() {
        if (cur != ~0u) {
            atomicAdd(&s_sum[3 * cur + 0], (unsigned long long)c_calls);
            atomicAdd(&s_sum[3 * cur + 1], (unsigned long long)c_busy);
            atomicAdd(&s_sum[3 * cur + 2], (unsigned long long)c_active);
        }
        c_calls = c_busy = c_active = 0;
    };
    for (uint32_t k = 0; k < per && base + k < valid; ++k) {
        uint32_t m;
        uint64_t s, e;
        get(base + k, m, s, e);
        if (m != cur) {
            flush();
            cur = m;
        }
        uint64_t from = s;
        if ((prev >> 61) == m) {
            const uint64_t reach = prev & kLow61;
            from = reach > s ? reach : s;
        }
        c_calls += 1;
        c_busy += e - s;
        c_active += e > from ? e - from : 0;
        const uint64_t pk = ((uint64_t)m << 61) | e;
        prev = pk > prev ? pk : prev;
    }
    flush();
}

// 64-bit DPP move (both halves; lanes the move does not write get `old`).
template <int C, int RM = 0xF>
__device__ __forceinline__ uint64_t dpp_mov64(uint64_t old, uint64_t v)
{
    return ((uint64_t)dpp_mov<C, RM>((uint32_t)(old >> 32), (uint32_t)(v >> 32)) << 32) |
           dpp_mov<C, RM>((uint32_t)old, (uint32_t)v);
}

// One LLM's sums over the wave (DPP row moves; lane 63 ends with them), added to s_sum[3q..].
__device__ __forceinline__ void wave_add_sums(uint32_t q, uint32_t calls, uint64_t busy,
                                              uint64_t active, unsigned long long *s_sum)
{
    wave_reduce_steps([&](auto c, auto rm) {
        constexpr int C = decltype(c)::value, RM = decltype(rm)::value;
        calls += dpp_mov<C, RM>(0u, calls);
        busy += dpp_mov64<C, RM>(0ull, busy);
        active += dpp_mov64<C, RM>(0ull, active);
    });
    if ((threadIdx.x & 63) == 63 && calls) {
        atomicAdd(&s_sum[3 * q + 0], (unsigned long long)calls);
        atomicAdd(&s_sum[3 * q + 1], (unsigned long long)busy);
        atomicAdd(&s_sum[3 * q + 2], (unsigned long long)active);
    }
}

// The passes that sort (the sweep of end-ordered traces is trace_sweep_kernel below).  kSort:
// the work list (or every trace of at most lds_cap calls), sorted in registers or LDS.  kLong:
// traces beyond lds_cap, sorted in a global scratch region.
enum StatsPass { kSort = 1, kLong = 2 };

struct StatsArgs {
    uint32_t M, lds_cap, R;
    const uint64_t *offsets;
    const uint32_t *llm;
    const uint64_t *start, *end;
    const uint32_t *long_traces;      // kLong: trace of each block
    const uint64_t *long_base;        // kLong: scratch offset of each block's trace (/ 2 words)
    uint64_t *scratch;
    unsigned long long *totals;       // kStatsCopies copies of the per-LLM sums
    uint32_t *flags;
    uint32_t *work;                   // the sweep appends, kSort reads: traces needing the sort
    uint32_t *work_count;
    uint32_t *done;                   // participants of the sort and long passes done
    uint32_t *slot_done;              // kStatsSlots counters of those participants
    uint32_t sort_grid, num_long;     // blocks of the sort and long launches
    alp_stats_t *out;                 // M records, then the StatsTail
};

// Wave-wide sum of 32-bit values (every lane gets it).
__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v)
{
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        v += (uint32_t)__shfl_xor((int)v, off, 64);
    return v;
}

// Exclusive maximum over the lanes of one wave (lane 0 gets 0).
__device__ __forceinline__ uint64_t wave_exclusive_max(uint64_t v, uint32_t lane)
{
    uint64_t incl = v;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint64_t o = __shfl_up((unsigned long long)incl, off, 64);
        if (lane >= (uint32_t)off)
            incl = o > incl ? o : incl;
    }
    const uint64_t excl = __shfl_up((unsigned long long)incl, 1, 64);
    return lane == 0 ? 0 : excl;
}

// The 32-bit value of lane (lane ^ Q) for any Q below 64: DPP for 1, 2, 3 (quad permutations),
// 7 (half-row mirror) and 15 (row mirror), a swizzle within 32 lanes up to 31, a lane permute
// from 32.
template <int Q>
__device__ __forceinline__ uint32_t lane_xor_any(uint32_t v)
{
    if constexpr (Q == 1 || Q == 2)
        return lane_xor<Q>(v);
    else if constexpr (Q == 3)
        return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x1B, 0xF, 0xF, false);
    else if constexpr (Q == 7)
        return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false);
    else if constexpr (Q == 15)
        return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false);
    else if constexpr (Q < 32)
        return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, 0x1F | (Q << 10));
    else
        return (uint32_t)__builtin_amdgcn_ds_bpermute((int)((threadIdx.x ^ (uint32_t)Q) << 2),
                                                       (int)v);
}

template <int Q>
__device__ __forceinline__ uint64_t lane_xor_any64(uint64_t v)
{
    return (uint64_t)lane_xor_any<Q>((uint32_t)v) |
           ((uint64_t)lane_xor_any<Q>((uint32_t)(v >> 32)) << 32);
}

constexpr uint32_t pow2_at_least(uint32_t v)
{
    uint32_t p = 1;
    while (p < v)
        p <<= 1;
    return p;
}

// One stage of a bitonic network whose comparators all put the minimum at the lower position:
// the first stage of a merge of SIZE pairs position i with its mirror i ^ (SIZE - 1) (MIRROR),
// the later ones with i ^ STRIDE.  Positions t E + e of NT threads, E keys each (E, NT powers of
// two or NT a multiple of 64); positions past NT E hold +inf without existing, so a pair whose
// upper position lies there leaves the lower one as it is.  Partners in the same thread are
// exchanged in registers, in the same wave across lanes, in other waves through buf (NT E keys,
// two barriers).
template <int E, int NT, int SIZE, int STRIDE, bool MIRROR>
__device__ __forceinline__ void mirror_stage(uint64_t (&k)[E], uint64_t *buf, uint32_t t)
{
    // partner of (t, e): thread t ^ TQ, register e ^ EQ
    constexpr uint32_t D = MIRROR ? SIZE - 1 : STRIDE;       // position xor
    constexpr uint32_t HALF = MIRROR ? SIZE / 2 : STRIDE;    // bit that marks the upper element
    constexpr uint32_t EQ = D % E, TQ = D / E;
    if constexpr (TQ == 0) {
#pragma unroll
        for (int e = 0; e < E; ++e) {
            if (e & HALF)
                continue;
            const int f = e ^ (int)EQ;
            const uint64_t a = k[e], b = k[f];
            const bool swap = a > b;
            k[e] = swap ? b : a;
            k[f] = swap ? a : b;
        }
    } else {
        const bool lower = (t & (HALF / E)) == 0;
        if constexpr (TQ < 64) {
            // Every partner value is fetched before any key changes: with EQ != 0 a key's
            // partner register may come earlier in the loop.
            uint64_t o[E];
#pragma unroll
            for (int e = 0; e < E; ++e)
                o[e] = lane_xor_any64<TQ>(k[e ^ EQ]);
#pragma unroll
            for (int e = 0; e < E; ++e)
                k[e] = keep_one(k[e], o[e], lower);
        } else {
#pragma unroll
            for (int e = 0; e < E; ++e)
                buf[e * NT + t] = k[e];
            __syncthreads();
            const uint32_t pt = t ^ TQ;
            if (pt < (uint32_t)NT) {
#pragma unroll
                for (int e = 0; e < E; ++e)
                    k[e] = keep_one(k[e], buf[(e ^ EQ) * NT + pt], lower);
            }
            __syncthreads();
        }
    }
}

template <int E, int NT, int SIZE, int STRIDE>
__device__ __forceinline__ void mirror_strides(uint64_t (&k)[E], uint64_t *buf, uint32_t t)
{
    if constexpr (STRIDE >= 1) {
        mirror_stage<E, NT, SIZE, STRIDE, false>(k, buf, t);
        mirror_strides<E, NT, SIZE, STRIDE / 2>(k, buf, t);
    }
}

// Ascending sort of the NT E keys (E per thread, thread t at positions t E ..), padded virtually
// to the next power of two: every merge of SIZE = 2, 4, .. is a mirror stage and half-cleaners.
template <int E, int NT, int SIZE = 2>
__device__ __forceinline__ void mirror_sort_regs(uint64_t (&k)[E], uint64_t *buf, uint32_t t)
{
    mirror_stage<E, NT, SIZE, SIZE / 2, true>(k, buf, t);
    mirror_strides<E, NT, SIZE, SIZE / 4>(k, buf, t);
    if constexpr (SIZE < (int)pow2_at_least(NT * E))
        mirror_sort_regs<E, NT, SIZE * 2>(k, buf, t);
}

// Per-LLM calls, durations and covered time of one trace's sorted keys, held by a group of NT
// threads (one wave, NT = 64, or a workgroup), added to s_sum: thread t holds positions
// t E .. t E + E - 1 of the valid calls and padding.  An exclusive prefix maximum of
// (llm << 61 | end) over the positions before a call tells whether an earlier call of the same
// LLM exists and the furthest end among them; the call adds its part beyond that end.  Key of a call: (llm << 61 | start - base
// << 32 | duration), the field start - base below 2^29.  The calls' fields are unpacked again
// where they are used rather than held, so that large E keep few registers.
template <int E, int NT>
__device__ __forceinline__ void group_sweep_regs(const uint64_t (&k)[E], uint32_t valid,
                                                 uint64_t base, unsigned long long *s_sum,
                                                 uint32_t t)
{
    const uint32_t first = t * E;
    auto llm_of = [](uint64_t kk) { return (uint32_t)(kk >> 61); };
    auto start_of = [&](uint64_t kk) { return base + ((kk >> 32) & ((1ull << 29) - 1)); };
    auto end_of = [&](uint64_t kk) { return start_of(kk) + (kk & 0xFFFFFFFFull); };
    uint64_t run = 0;
#pragma unroll
    for (int j = 0; j < E; ++j) {
        if (first + j < valid) {
            const uint64_t pk = ((uint64_t)llm_of(k[j]) << 61) | end_of(k[j]);
            run = pk > run ? pk : run;
        }
    }
    uint64_t prev;
    if constexpr (NT == 64)
        prev = wave_exclusive_max(run, t);
    else
        prev = block_exclusive_max(run);
    constexpr uint64_t kLow61 = (1ull << 61) - 1;
    uint32_t cur = ~0u;
    uint64_t c_calls = 0, c_busy = 0, c_active = 0;
#pragma unroll
    for (int j = 0; j < E; ++j) {
        if (first + j >= valid)
            continue;                                  // (sorted: every later j too)
        const uint32_t m = llm_of(k[j]);
        const uint64_t s = start_of(k[j]), e = s + (k[j] & 0xFFFFFFFFull);
        if (m != cur) {
            if (cur != ~0u) {
                atomicAdd(&s_sum[3 * cur + 0], (unsigned long long)c_calls);
                atomicAdd(&s_sum[3 * cur + 1], (unsigned long long)c_busy);
                atomicAdd(&s_sum[3 * cur + 2], (unsigned long long)c_active);
            }
            c_calls = c_busy = c_active = 0;
            cur = m;
        }
        uint64_t from = s;
        if ((prev >> 61) == m) {
            const uint64_t reach = prev & kLow61;
            from = reach > s ? reach : s;
        }
        c_calls += 1;
        c_busy += e - s;
        c_active += e > from ? e - from : 0;
        const uint64_t pk = ((uint64_t)m << 61) | e;
        prev = pk > prev ? pk : prev;
    }
    if (cur != ~0u) {
        atomicAdd(&s_sum[3 * cur + 0], (unsigned long long)c_calls);
        atomicAdd(&s_sum[3 * cur + 1], (unsigned long long)c_busy);
        atomicAdd(&s_sum[3 * cur + 2], (unsigned long long)c_active);
    }
}

// Keys of the calls lo .. lo + n - 1 (n <= NT E) for thread t of a group of NT: calls j NT + t
// (j < E; each load instruction reads consecutive calls), keyed by start relative to base.
// Malformed calls are reported in bad and left out, as in the block sort; a valid call outside
// [base, base + 2^29) sets far (the group then hands the trace to the block sort).  Loads go
// in groups of up to 4 keys, all in flight together and without branches: positions past the
// trace load its last call again and become padding.  (A branch per call made the compiler
// wait for each call's loads before the next; all E at once spill.)
template <int E, int NT>
__device__ __forceinline__ void load_keys(const StatsArgs &a, uint64_t lo, uint32_t n, uint32_t t,
                                          uint64_t base, uint64_t (&k)[E], uint32_t &bad,
                                          uint32_t &valid, bool &far)
{
    const uint32_t M = a.M;
    constexpr int kGroup = E < 4 ? E : 4;
#pragma unroll
    for (int j0 = 0; j0 < E; j0 += kGroup) {
        uint32_t mm[kGroup];
        uint64_t ss[kGroup], ee[kGroup];
#pragma unroll
        for (int g = 0; g < kGroup; ++g) {
            const uint32_t i = (uint32_t)(j0 + g) * NT + t;
            const uint64_t at = lo + (i < n ? i : n - 1);
            mm[g] = a.llm[at];
            ss[g] = a.start[at];
            ee[g] = a.end[at];
        }
#pragma unroll
        for (int g = 0; g < kGroup; ++g) {
            const uint32_t i = (uint32_t)(j0 + g) * NT + t;
            const uint32_t m = mm[g];
            const uint64_t st = ss[g], en = ee[g];
            const uint32_t b = m >= M ? 1u
                             : en < st ? 2u
                             : st >= kStartLimit || en - st >= kDurationLimit ? 4u : 0u;
            const uint64_t off = st - base;
            const bool ok = i < n && b == 0;
            bad |= i < n ? b : 0u;
            far = far || (ok && off >= (1ull << 29));
            const bool use = ok && off < (1ull << 29);
            k[j0 + g] = use ? ((uint64_t)m << 61) | (off << 32) | (en - st) : kPad;
            valid += use ? 1u : 0u;
        }
        __builtin_amdgcn_sched_barrier(0);
    }
}

// Statistics of trace r (slot = the block's trace slot in long_base for kLong) by one block.
template <int Pass, int MM = ALP_MAX_LLMS>
__device__ __forceinline__ void one_trace(const StatsArgs &a, uint32_t r, uint32_t slot,
                                          unsigned char *s_dyn)
{
    constexpr bool Global = Pass == kLong;
    const uint32_t M = a.M;
    const uint32_t *__restrict__ llm = a.llm;
    const uint64_t *__restrict__ start = a.start;
    const uint64_t *__restrict__ end = a.end;
    uint32_t *flags = a.flags;
    __shared__ unsigned long long s_sum[3 * ALP_MAX_LLMS];   // per LLM: calls, busy, active
    __shared__ uint32_t s_valid, s_far;
    const uint64_t lo = a.offsets[r], n = a.offsets[r + 1] - lo;
    if (n == 0 || (!Global && n > a.lds_cap))
        return;                                        // empty, or the global pass takes it
    uint32_t P = kThreads;                              // padded length: a power of two
    while (P < n)
        P <<= 1;
    uint64_t *key = Global ? a.scratch + 2 * a.long_base[slot]
                           : reinterpret_cast<uint64_t *>(s_dyn);
    uint64_t *val = key + P;
    for (uint32_t k = threadIdx.x; k < 3 * ALP_MAX_LLMS; k += kThreads)
        s_sum[k] = 0;
    if (threadIdx.x == 0) {
        s_valid = 0;
        s_far = 0;
    }
    __syncthreads();                                   // counters zeroed before any adds
    // Calls i = threadIdx.x + k * kThreads; out-of-range or invalid ones become padding.
    uint32_t bad = 0, valid = 0;
    auto load = [&](uint64_t i, uint32_t &m, uint64_t &s, uint64_t &e) -> bool {
        if (i >= n)
            return false;
        m = llm[lo + i];
        s = start[lo + i];
        e = end[lo + i];
        if (m >= M)
            bad |= 1u;
        else if (e < s)
            bad |= 2u;
        else if (s >= kStartLimit || e - s >= kDurationLimit)
            bad |= 4u;
        else
            return true;
        return false;
    };
    bool unpacked = Global;
    if constexpr (!Global) {
        // Packed keys in registers, as the direct sort's groups hold them: thread t loads calls
        // j * 256 + t (j < E = P / 256) and keys each by its start relative to the first call's
        // start - 2^28 (llm << 61 | start - base << 32 | duration), which halves the sort's LDS
        // traffic.  A trace with a start outside [base, base + 2^29) falls back to (key, end)
        // pairs in LDS, loaded again.
        const uint64_t base = start[lo] - (1ull << 28);      // modulo 2^64
        auto run = [&](auto e_const) {
            constexpr int E = decltype(e_const)::value;
            uint64_t k[E];
            uint32_t kb = 0, kv = 0;
            bool far = false;
            load_keys<E, kThreads>(a, lo, n, threadIdx.x, base, k, kb, kv, far);
            if (kb)
                atomicOr(flags, kb);
            const uint32_t wv = wave_sum_u32(kv);
            const bool wf = __ballot(far) != 0;
            if ((threadIdx.x & 63) == 0) {
                atomicAdd(&s_valid, wv);
                if (wf)
                    atomicOr(&s_far, 1u);
            }
            __syncthreads();
            if (s_far) {                                // uniform over the block
                unpacked = true;
                return;
            }
            const uint32_t nvalid = s_valid;
            if (nvalid == 0)
                return;
            bitonic_sort_regs<E>(k, key, P, threadIdx.x);
            group_sweep_regs<E, kThreads>(k, nvalid, base, s_sum, threadIdx.x);
        };
        switch (P) {
        case kThreads: run(std::integral_constant<int, 1>{}); break;
        case 2 * kThreads: run(std::integral_constant<int, 2>{}); break;
        case 4 * kThreads: run(std::integral_constant<int, 4>{}); break;
        default: run(std::integral_constant<int, 8>{}); break;
        }
        if (unpacked) {
            __syncthreads();                           // every thread has read s_valid
            if (threadIdx.x == 0)
                s_valid = 0;
            __syncthreads();
        }
    }
    if (unpacked) {
        for (uint64_t i = threadIdx.x; i < P; i += kThreads) {
            uint32_t m = 0;
            uint64_t s = 0, e = 0;
            const bool ok = load(i, m, s, e);
            valid += ok;
            key[i] = ok ? ((uint64_t)m << 60) | s : kPad;
            val[i] = ok ? e : 0;
        }
        if (bad)
            atomicOr(flags, bad);
        atomicAdd(&s_valid, valid);
        __syncthreads();
        const uint32_t nvalid = s_valid;
        bitonic_sort<true>(key, val, P);
        sweep(P, nvalid, [&](uint32_t i, uint32_t &m, uint64_t &s, uint64_t &e) {
            const uint64_t kk = key[i];
            m = (uint32_t)(kk >> 60);
            s = kk & (kStartLimit - 1);
            e = val[i];
        }, s_sum);
    }
    __syncthreads();
    unsigned long long *copy = a.totals + (uint64_t)(r % kStatsCopies) * kStatsCopyStride;
    for (uint32_t k = threadIdx.x; k < 3 * M; k += kThreads)
        if (s_sum[k])
            atomicAdd(&copy[k], s_sum[k]);
}

constexpr uint32_t kSweepWaves = 4;     // traces per workgroup of the sweep, one per wave
constexpr uint32_t kSweepBatch = 8;     // rows of 64 calls loaded together

// Inclusive maximum over lanes 0..L: row shifts by 1, 2, 4 and 8, then lane 15 into rows 1 and
// 3 and lane 31 into rows 2 and 3 (lanes a move does not reach keep 0, the identity).
__device__ __forceinline__ uint32_t wave_prefix_max(uint32_t v)
{
    auto step = [&](auto c, auto rm) {
        constexpr int C = decltype(c)::value, RM = decltype(rm)::value;
        const uint32_t o = dpp_mov<C, RM>(0u, v);
        v = o > v ? o : v;
    };
    step(std::integral_constant<int, 0x111>{}, std::integral_constant<int, 0xF>{});
    step(std::integral_constant<int, 0x112>{}, std::integral_constant<int, 0xF>{});
    step(std::integral_constant<int, 0x114>{}, std::integral_constant<int, 0xF>{});
    step(std::integral_constant<int, 0x118>{}, std::integral_constant<int, 0xF>{});
    step(std::integral_constant<int, 0x142>{}, std::integral_constant<int, 0xA>{});
    step(std::integral_constant<int, 0x143>{}, std::integral_constant<int, 0xC>{});
    return v;
}

struct SweepRows {
    uint32_t m[kSweepBatch];
    uint64_t s[kSweepBatch], e[kSweepBatch];
};

// Covered time of the traces whose calls are in order of end time (as a proxy logs them on
// completion), without a sort: one wave per trace of at most lds_cap calls.  Walking the calls
// backwards, the calls of LLM m after call j (ending no earlier) cover, within (-inf, e_j],
// exactly [lo, e_j], lo their earliest start (nothing if lo > e_j); so call j adds
// max(0, min(e_j, lo) - s_j).  The wave takes rows of 64 calls from the end: lane L of row k
// holds call n - 1 - 64 k - L, so a call's later calls are the lower lanes of its row and the
// rows already swept, and each load instruction reads 64 consecutive calls.  Times count back
// from the last call's end E, a = E - s and b = E - e, in 32 bits: then call j adds
// max(0, a_j - max(b_j, h)), h the largest a among m's later calls (0 if none) -- a prefix
// maximum over the lanes, per LLM, joined with the maximum carried over the rows before.  A
// trace out of end order, with a malformed call, reaching 2^60 us or spanning 2^32 us or more
// goes to the work list instead (the sort pass reports malformed calls).  MM bounds the number
// of LLMs (2, 4 or 8), so the per-LLM registers fit the workflow.
template <int MM>
__global__ void __launch_bounds__(64 * kSweepWaves) trace_sweep_kernel(StatsArgs a)
{
    const uint32_t lane = threadIdx.x & 63;
    const uint32_t r = (uint32_t)__builtin_amdgcn_readfirstlane(
        (int)(blockIdx.x * kSweepWaves + (threadIdx.x >> 6)));
    if (r >= a.R)
        return;                                        // uniform over the wave
    const uint64_t lo = a.offsets[r], n64 = a.offsets[r + 1] - lo;
    if (n64 == 0 || n64 > a.lds_cap)
        return;                                        // empty, or the global pass takes it
    const uint32_t n = (uint32_t)n64, M = a.M, rows = (n + 63) >> 6;
    const uint64_t E = a.end[lo + n - 1];
    bool bad = E >= kStartLimit;
    auto load = [&](SweepRows &R, uint32_t k0) {
#pragma unroll
        for (uint32_t j = 0; j < kSweepBatch; ++j) {
            if (k0 + j >= rows)
                break;                                 // uniform
            const int32_t idx = (int32_t)n - 1 - (int32_t)(64 * (k0 + j) + lane);
            // a lane before the trace's first call reads that call again (masked below)
            const uint64_t i = lo + (uint64_t)(idx < 0 ? 0 : idx);
            R.m[j] = a.llm[i];
            R.s[j] = a.start[i];
            R.e[j] = a.end[i];
        }
    };
    uint32_t calls[MM], carry[MM];
    uint64_t busy[MM], active[MM];
#pragma unroll
    for (int q = 0; q < MM; ++q) {
        calls[q] = carry[q] = 0;
        busy[q] = active[q] = 0;
    }
    uint32_t next_b = 0;                               // b of the call after the row's lane 0
    auto sweep_rows = [&](const SweepRows &R, uint32_t k0) {
#pragma unroll
        for (uint32_t j = 0; j < kSweepBatch; ++j) {
            if (k0 + j >= rows)
                break;                                 // uniform
            const bool valid = 64 * (k0 + j) + lane < n;
            const uint32_t m = R.m[j];
            const uint64_t a64 = E - R.s[j], b64 = E - R.e[j];
            const uint32_t av = (uint32_t)a64, bv = (uint32_t)b64;
            // In order: this call ends no later than the next one (lane - 1, or the previous
            // row's lane 63).
            const uint32_t bn = dpp_mov<0x138>(next_b, bv);
            const bool good = m < M && (a64 >> 32) == 0 && (b64 >> 32) == 0 && av >= bv &&
                              bv >= bn;
            bad = bad || __ballot(valid && !good) != 0;
            next_b = lane63(bv);
            uint32_t h = 0;
#pragma unroll
            for (int q = 0; q < MM; ++q) {
                if ((uint32_t)q >= M)
                    break;
                const uint32_t v = wave_prefix_max(valid && m == (uint32_t)q ? av : 0u);
                const uint32_t ex = dpp_mov<0x138>(0u, v);   // lanes below this one
                const uint32_t later = ex > carry[q] ? ex : carry[q];
                h = m == (uint32_t)q ? later : h;
                const uint32_t tot = lane63(v);
                carry[q] = tot > carry[q] ? tot : carry[q];
            }
            const uint32_t t = bv > h ? bv : h;
            const uint32_t act = av > t ? av - t : 0u;
#pragma unroll
            for (int q = 0; q < MM; ++q) {
                if (valid && m == (uint32_t)q) {
                    calls[q] += 1;
                    busy[q] += av - bv;
                    active[q] += act;
                }
            }
        }
    };
    // A batch of rows is loaded at once (up to 8 x 1.25 KB in flight per wave), then swept;
    // the other waves of the SIMD sweep while this one waits.
    for (uint32_t k0 = 0; k0 < rows && !bad; k0 += kSweepBatch) {
        SweepRows R;
        load(R, k0);
        sweep_rows(R, k0);
    }
    if (bad) {
        if (lane == 0)
            a.work[atomicAdd(a.work_count, 1u)] = r;
        return;
    }
    unsigned long long *copy = a.totals + (uint64_t)(r % kStatsCopies) * kStatsCopyStride;
#pragma unroll
    for (int q = 0; q < MM; ++q)
        if ((uint32_t)q < M)
            wave_add_sums((uint32_t)q, calls[q], busy[q], active[q], copy);
}

// Called, once its traces are summed, by every block of the sort and long passes that had
// work: participant i of P.  The last of them (over both launches) takes the totals -- reading
// each word and zeroing it for the next call, as it zeroes the flags, the work-list length and
// the counters -- and writes n and p per LLM, then the status and the work-list length for the
// host.  Participants count themselves in kStatsSlots counters (i mod kStatsSlots) and the last
// of each slot in one more, so that no counter takes more than a share of the increments.
// Every sum, flag and count is added and read by atomics, performed where all blocks see them;
// a block's own atomics have completed (its vector memory count drained) before it counts
// itself, so no cache needs writing back or invalidating (a device-wide fence per block would
// cost both for every block).  Status bits: 1 llm out of range, 2 end before start, 4 start or
// duration out of range, 8 a result beyond 2^31 - 1 (it could not be loaded as an ALP input).
__device__ __forceinline__ void finish_block(const StatsArgs &a, uint32_t i, uint32_t P)
{
    __shared__ uint32_t s_last, s_flags;
    __shared__ unsigned long long s_tot[3 * ALP_MAX_LLMS];
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // this thread's atomics are done
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t slot = i % kStatsSlots;
        const uint32_t in_slot = (P - slot + kStatsSlots - 1) / kStatsSlots;
        uint32_t last = 0;
        if (atomicAdd(&a.slot_done[slot], 1u) == in_slot - 1) {
            (void)atomicExch(&a.slot_done[slot], 0u);
            const uint32_t slots = P < kStatsSlots ? P : kStatsSlots;
            if (atomicAdd(a.done, 1u) == slots - 1) {
                (void)atomicExch(a.done, 0u);
                last = 1;
            }
        }
        s_last = last;
        s_flags = 0;
    }
    if (threadIdx.x < 3 * ALP_MAX_LLMS)
        s_tot[threadIdx.x] = 0;
    __syncthreads();
    if (!s_last)
        return;                                        // uniform over the block
    const uint32_t W = 3 * a.M;
    for (uint32_t k = threadIdx.x; k < kStatsCopies * W; k += kThreads) {
        const uint32_t c = k / W, f = k - c * W;
        const unsigned long long v =
            atomicExch(a.totals + (uint64_t)c * kStatsCopyStride + f, 0ull);
        if (v)
            atomicAdd(&s_tot[f], v);
    }
    __syncthreads();
    const uint32_t m = threadIdx.x;
    if (m < a.M) {
        const uint64_t calls = s_tot[3 * m], busy = s_tot[3 * m + 1], active = s_tot[3 * m + 2];
        uint64_t n = calls * 1000u / a.R, p;
        if (calls == 0)
            p = 0;
        else if (active == 0)
            p = 1000;
        else if (busy >= (1ull << 53))
            p = ~0ull;
        else
            p = busy * 1000u / active;
        if (n >= (1u << 31) || p >= (1u << 31)) {
            atomicOr(&s_flags, 8u);
            n = n >= (1u << 31) ? 0 : n;
            p = p >= (1u << 31) ? 0 : p;
        }
        alp_stats_t st;
        st.n_milli = (uint32_t)n;
        st.p_milli = (uint32_t)p;
        st.calls = calls;
        st.busy_us = busy;
        st.active_us = active;
        a.out[m] = st;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        StatsTail t = {};
        t.flags = atomicExch(a.flags, 0u) | s_flags;
        t.listed = atomicExch(a.work_count, 0u);
        *reinterpret_cast<StatsTail *>(a.out + ALP_MAX_LLMS) = t;
    }
}

constexpr uint32_t kWaveSortWaves = 4;       // traces per workgroup of the direct sort
constexpr uint32_t kWaveSortMax = 64 * 8;    // longest trace one wave sorts (8 keys per lane)

// Trace r (calls lo .. lo + n - 1, n <= 64 E) sorted and swept by one wave: the wave sorts the
// 64 E keys in registers and across lanes (no LDS, no barrier), sweeps them, and adds the
// per-LLM sums to s_sum (the wave's own) and then to the trace's copy of the totals.  Keys hold
// a call's start relative to base = (first call's start) - 2^28; a trace with a valid call
// outside [base, base + 2^29) goes to the work list for the block sort, which handles any span.
template <int E>
__device__ __forceinline__ void wave_trace(const StatsArgs &a, uint32_t r, uint64_t lo, uint32_t n,
                                           uint32_t lane, unsigned long long *s_sum)
{
    const uint32_t M = a.M;
    const uint64_t base = a.start[lo] - (1ull << 28);      // modulo 2^64
    uint64_t k[E];
    uint32_t bad = 0, valid = 0;
    bool far = false;
    load_keys<E, 64>(a, lo, n, lane, base, k, bad, valid, far);
    if (bad)
        atomicOr(a.flags, bad);
    if (__ballot(far)) {
        if (lane == 0)
            a.work[atomicAdd(a.work_count, 1u)] = r;
        return;
    }
    const uint32_t nvalid = wave_sum_u32(valid);
    if (nvalid == 0)
        return;
    bitonic_sort_regs<E, 64>(k, nullptr, 64 * E, lane);
    if (lane < 3 * M)
        s_sum[lane] = 0;
    group_sweep_regs<E, 64>(k, nvalid, base, s_sum, lane);
    unsigned long long *copy = a.totals + (uint64_t)(r % kStatsCopies) * kStatsCopyStride;
    if (lane < 3 * M) {
        const unsigned long long v = s_sum[lane];
        if (v)
            atomicAdd(&copy[lane], v);
    }
}

// Every trace of at most 512 calls sorted directly (the context found most traces out of end
// order): one wave per trace, kWaveSortWaves traces per workgroup; traces the wave does not take
// (a span beyond its packed keys) are listed for the block sort that follows.
__global__ void __launch_bounds__(64 * kWaveSortWaves) trace_wave_kernel(StatsArgs a)
{
    __shared__ unsigned long long s_sum[kWaveSortWaves][3 * ALP_MAX_LLMS];
    const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint32_t r = (uint32_t)__builtin_amdgcn_readfirstlane(
        (int)(blockIdx.x * kWaveSortWaves + wave));
    if (r >= a.R)
        return;                                        // uniform over the wave
    const uint64_t lo = a.offsets[r], n64 = a.offsets[r + 1] - lo;
    if (n64 == 0 || n64 > a.lds_cap || n64 > kWaveSortMax)
        return;                                        // empty, or another pass takes it
    const uint32_t n = (uint32_t)n64;
    unsigned long long *sum = s_sum[wave];
    if (n <= 64)
        wave_trace<1>(a, r, lo, n, lane, sum);
    else if (n <= 128)
        wave_trace<2>(a, r, lo, n, lane, sum);
    else if (n <= 256)
        wave_trace<4>(a, r, lo, n, lane, sum);
    else
        wave_trace<8>(a, r, lo, n, lane, sum);
}

// Every trace of LO + 1 to NT E calls sorted directly (8 keys per thread: 513 to 1,024 calls on
// two waves, 1,025 to 1,536 on three, 1,537 to 2,048 on four): one workgroup of NT threads per
// trace, keyed and handed on as in trace_wave_kernel, sorted by mirror_sort_regs (exchanges
// between waves through one LDS buffer of NT E keys).  8 keys per thread keep about 50 VGPRs;
// 16 or 32 keys per lane needed 89 and 171 (2 to 5 waves per SIMD instead of 8).
template <int E, int NT, int LO>
__global__ void __launch_bounds__(NT) trace_group_kernel(StatsArgs a)
{
    constexpr uint32_t P = NT * E;
    __shared__ uint64_t s_buf[P];
    __shared__ unsigned long long s_sum[3 * ALP_MAX_LLMS];
    __shared__ uint32_t s_valid, s_far;
    const uint32_t r = blockIdx.x, t = threadIdx.x;
    if (r >= a.R)
        return;                                        // uniform over the block
    const uint64_t lo = a.offsets[r], n64 = a.offsets[r + 1] - lo;
    if (n64 <= (uint64_t)LO || n64 > a.lds_cap)
        return;                                        // another pass takes it
    if (n64 > P) {
        // Below 2,048 keys: a larger group's.  2,048: to the block sort (the host keeps lds_cap
        // within 2,048, so this does not occur).
        if (P == 2048 && t == 0)
            a.work[atomicAdd(a.work_count, 1u)] = r;
        return;
    }
    const uint32_t n = (uint32_t)n64, M = a.M;
    if (t == 0) {
        s_valid = 0;
        s_far = 0;
    }
    if (t < 3 * M)
        s_sum[t] = 0;
    __syncthreads();
    const uint64_t base = a.start[lo] - (1ull << 28);      // modulo 2^64
    uint64_t k[E];
    uint32_t bad = 0, valid = 0;
    bool far = false;
    load_keys<E, NT>(a, lo, n, t, base, k, bad, valid, far);
    if (bad)
        atomicOr(a.flags, bad);
    const uint32_t wvalid = wave_sum_u32(valid);
    const bool wfar = __ballot(far) != 0;
    if ((t & 63) == 0) {
        atomicAdd(&s_valid, wvalid);
        if (wfar)
            atomicOr(&s_far, 1u);
    }
    __syncthreads();
    if (s_far) {                                       // uniform over the block
        if (t == 0)
            a.work[atomicAdd(a.work_count, 1u)] = r;
        return;
    }
    const uint32_t nvalid = s_valid;
    if (nvalid == 0)
        return;
    mirror_sort_regs<E, NT>(k, s_buf, t);
    group_sweep_regs<E, NT>(k, nvalid, base, s_sum, t);
    __syncthreads();
    unsigned long long *copy = a.totals + (uint64_t)(r % kStatsCopies) * kStatsCopyStride;
    if (t < 3 * M) {
        const unsigned long long v = s_sum[t];
        if (v)
            atomicAdd(&copy[t], v);
    }
}

// Sorts the traces of the work list (written by the sweep, or by the direct sort for the traces
// it leaves), a grid of blocks taking its entries in turn.
// Blocks of the sort launch that have work: the first min(listed, grid) blocks, and block 0
// always (it finishes when nothing is listed).
__device__ __forceinline__ uint32_t sort_participants(const StatsArgs &a)
{
    const uint32_t listed = *a.work_count;
    return listed == 0 ? 1u : (listed < a.sort_grid ? listed : a.sort_grid);
}

__global__ void __launch_bounds__(kThreads) trace_sort_kernel(StatsArgs a)
{
    extern __shared__ __align__(8) unsigned char s_dyn[];
    const uint32_t P = sort_participants(a);
    if (blockIdx.x >= P)
        return;                                        // nothing listed for this block
    const uint32_t listed = *a.work_count;
    for (uint32_t w = blockIdx.x; w < listed; w += gridDim.x) {
        if (w != blockIdx.x)
            __syncthreads();                           // the previous trace's sums are read
        one_trace<kSort>(a, a.work[w], 0, s_dyn);
    }
    finish_block(a, blockIdx.x, P + a.num_long);
}

__global__ void __launch_bounds__(kThreads) trace_long_kernel(StatsArgs a)
{
    one_trace<kLong>(a, a.long_traces[blockIdx.x], blockIdx.x, nullptr);
    const uint32_t P = sort_participants(a);           // the list is still intact here
    finish_block(a, P + blockIdx.x, P + a.num_long);
}

}  // namespace

hipError_t launch_trace_stats(uint32_t M, uint32_t R, const uint64_t *offsets, const uint32_t *llm,
                              const uint64_t *start, const uint64_t *end, uint32_t lds_cap,
                              uint32_t max_short, uint32_t num_long, const uint32_t *long_traces,
                              const uint64_t *long_base, uint64_t *scratch, uint64_t *totals,
                              uint32_t *work, bool sweep, bool zero_first, alp_stats_t *out,
                              hipStream_t st)
{
    hipError_t e;
    if (zero_first) {
        hipLaunchKernelGGL(stats_init_kernel, dim3(1), dim3(256), 0, st, totals,
                           kStatsTotalsWords + kStatsTailWords);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
    }
    StatsArgs a;
    a.M = M;
    a.lds_cap = lds_cap;
    a.R = R;
    a.offsets = offsets;
    a.llm = llm;
    a.start = start;
    a.end = end;
    a.long_traces = long_traces;
    a.long_base = long_base;
    a.scratch = scratch;
    a.totals = reinterpret_cast<unsigned long long *>(totals);
    a.flags = reinterpret_cast<uint32_t *>(totals + kStatsTotalsWords);
    a.work = work;
    a.work_count = reinterpret_cast<uint32_t *>(totals + kStatsTotalsWords + 1);
    a.done = reinterpret_cast<uint32_t *>(totals + kStatsTotalsWords + 1) + 1;
    a.slot_done = reinterpret_cast<uint32_t *>(totals + kStatsTotalsWords + 2);
    a.out = out;
    if (sweep) {
        const dim3 grid((R + kSweepWaves - 1) / kSweepWaves), block(64 * kSweepWaves);
        if (M <= 2)
            hipLaunchKernelGGL(trace_sweep_kernel<2>, grid, block, 0, st, a);
        else if (M <= 4)
            hipLaunchKernelGGL(trace_sweep_kernel<4>, grid, block, 0, st, a);
        else
            hipLaunchKernelGGL(trace_sweep_kernel<ALP_MAX_LLMS>, grid, block, 0, st, a);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
    } else {
        if (max_short > 1536) {
            hipLaunchKernelGGL(HIP_KERNEL_NAME(trace_group_kernel<8, 256, 1536>), dim3(R),
                               dim3(256), 0, st, a);
            if ((e = hipGetLastError()) != hipSuccess)
                return e;
        }
        if (max_short > 1024) {
            hipLaunchKernelGGL(HIP_KERNEL_NAME(trace_group_kernel<8, 192, 1024>), dim3(R),
                               dim3(192), 0, st, a);
            if ((e = hipGetLastError()) != hipSuccess)
                return e;
        }
        if (max_short > kWaveSortMax) {
            hipLaunchKernelGGL(HIP_KERNEL_NAME(trace_group_kernel<8, 128, kWaveSortMax>),
                               dim3(R), dim3(128), 0, st, a);
            if ((e = hipGetLastError()) != hipSuccess)
                return e;
        }
        hipLaunchKernelGGL(trace_wave_kernel, dim3((R + kWaveSortWaves - 1) / kWaveSortWaves),
                           dim3(64 * kWaveSortWaves), 0, st, a);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
    }
    // The work list's length is known only on the device: a grid of at most kSortBlocks
    // blocks takes its entries in turn (an empty list costs one short launch).
    const size_t lds = (size_t)2 * lds_cap * sizeof(uint64_t);
    const uint32_t sort_blocks = R > kSortBlocks ? kSortBlocks : R;
    a.sort_grid = sort_blocks;
    a.num_long = num_long;
    hipLaunchKernelGGL(trace_sort_kernel, dim3(sort_blocks), dim3(kThreads), lds, st, a);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    if (num_long) {
        hipLaunchKernelGGL(trace_long_kernel, dim3(num_long), dim3(kThreads), 0, st, a);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
    }
    return hipSuccess;
}

}  // namespace alp
