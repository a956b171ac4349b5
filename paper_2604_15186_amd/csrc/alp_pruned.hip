// gfx950 kernels of the paper's own pruned allocation search (Scepsy, arXiv 2604.15186,
// Section 5, steps 1-3), measured against the exhaustive search of alp_kernels.hip.
//
//   Step 1  every LLM m gets f_m units of 1/Q GPU, sum f_m = Q*G; with the ordering flag no LLM
//           gets more units than one of higher profiled latency ratio before it, with the
//           minimum-fraction flag every LLM gets at least the units that hold its weights and
//           at most Q*G minus the lower bounds of the LLMs after it.
//   Step 2  the fractions are packed contiguously, highest latency ratio first.
//   Step 3  an option (tp, q, d) is admissible for an LLM iff tp*q*d equals its fraction and
//           d replicas of tp ranks (q units each, the ranks of a replica on distinct GPUs) fit
//           its packed GPUs.
//
// Kernels:
//   pruned_prep_kernel       clears the option table and computes each item's step-1 order and
//                            bounds.
//   pruned_scatter_kernel    per (item, LLM, option): enters the option into the table entry
//                            (item, LLM, first-unit offset mod Q, fraction = its units) of every
//                            offset where it fits, keeping the smallest Eq. 1 contribution
//                            (lowest option among equal ones).  With the fraction vector fixed
//                            the LLMs are independent and L_w is a sum, so this table decides
//                            every vector.
//   pruned_scan_kernel<M>    one thread per prefix (the first fraction, or the first two beyond
//                            3 LLMs); the remaining fractions are enumerated in registers
//                            (compile-time depth), each vector summed from the table; the
//                            lexicographic (L_w, x) minimum and the vector count are reduced per
//                            block, and the item's last block writes the result.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "alp_device.h"
#include "alp_internal.h"

namespace alp {

namespace {

// Does an LLM whose units start at offset r (mod Q) and span f units fit d replicas of tp ranks
// of q units, the ranks of a replica on distinct GPUs?  A GPU holding h of its units takes at
// most min(floor(h / q), d) ranks, and the sum reaching tp * d suffices (deal the ranks to the
// replicas GPU by GPU in turn).  The units occupy a partial first GPU, full GPUs, and a partial
// last GPU.
__device__ __forceinline__ bool placement_fits(uint32_t Q, uint32_t r, uint32_t f, uint32_t tp,
                                               uint32_t q, uint32_t d)
{
    if (f == 0)
        return tp * d == 0;
    const uint32_t end = r + f;
    auto take = [&](uint32_t h) { const uint32_t c = h / q; return c < d ? c : d; };
    uint32_t ranks;
    if (end <= Q) {
        ranks = take(f);
    } else {
        const uint32_t full = end / Q - 1, tail = end % Q;
        ranks = take(Q - r) + full * take(Q) + (tail ? take(tail) : 0u);
    }
    return ranks >= tp * d;
}

// Table entries pack (c << 32 | option): the 64-bit minimum is the smallest contribution, then
// the lowest option.  No admissible option: all ones (c = kNoLatency).
constexpr uint64_t kNoEntry = ~0ull;

// Per-item constants of step 1, by position in the latency-ratio order (first M entries used).
struct Order {
    uint32_t lo[ALP_MAX_LLMS], hi[ALP_MAX_LLMS], lo_after[ALP_MAX_LLMS];
    uint64_t pw[ALP_MAX_LLMS];      // O^(M-1-m) of the LLM at the position
    uint64_t tab[ALP_MAX_LLMS];     // offset of its table rows in the item's table, in entries
    uint32_t F, empty;
};

// Fills the option table with kNoEntry and, in the first `count` threads, computes each item's
// step-1 order: latency ratios (contribution at tp[0], the largest share, the first profiled
// point), largest first with ties by LLM index, the lower bounds max(1, ceil(W Q / H)) with the
// minimum-fraction flag, and the upper bounds Q*G minus the lower bounds after each position.
__global__ void __launch_bounds__(256)
pruned_prep_kernel(SpaceDev sp, TablesDev tb, QueryDev q, uint32_t count, uint32_t F1,
                   uint32_t flags, uint64_t *__restrict__ table, Order *__restrict__ orders)
{
    const uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t < (uint64_t)count * sp.M * sp.Q * F1)
        table[t] = kNoEntry;
    if (t >= count)
        return;
    const uint32_t item = (uint32_t)t, M = sp.M;
    const uint32_t inst = query_value(q.inst, q.inst1, item);
    const uint32_t F = query_value(q.capacity, q.cap1, item);
    uint64_t ref[ALP_MAX_LLMS];
    uint32_t order[ALP_MAX_LLMS];
    for (uint32_t m = 0; m < M; ++m) {
        const uint64_t base = (uint64_t)inst * M + m;
        const uint64_t cell = (base * sp.n_tp + 0) * sp.n_fq + (sp.n_fq - 1);
        ref[m] = (uint64_t)tb.lat[cell * sp.K] * tb.n[base] / tb.p[base];
        order[m] = m;
    }
    for (uint32_t a = 1; a < M; ++a) {
        const uint32_t v = order[a];
        uint32_t b = a;
        while (b > 0 && ref[order[b - 1]] < ref[v]) {
            order[b] = order[b - 1];
            --b;
        }
        order[b] = v;
    }
    Order od;
    uint64_t after = 0;
    od.empty = 0;
    for (int k = (int)M - 1; k >= 0; --k) {
        const uint32_t m = order[k];
        const uint64_t base = (uint64_t)inst * M + m;
        uint64_t lo = 0;
        if (flags & ALP_PRUNE_MIN_FRACTION) {
            const uint64_t need = (tb.W[base] * sp.Q + tb.H - 1) / tb.H;
            lo = need > 1 ? need : 1;
        }
        if (after + lo > F) {
            od.empty = 1;
            lo = 0;
        }
        od.lo[k] = (uint32_t)lo;
        od.lo_after[k] = (uint32_t)after;
        od.hi[k] = after <= F ? F - (uint32_t)after : 0u;
        after += lo;
        uint64_t pw = 1;
        for (uint32_t j = m + 1; j < M; ++j)
            pw *= sp.O;
        od.pw[k] = pw;
        od.tab[k] = (uint64_t)m * sp.Q * F1;
    }
    od.F = F;
    orders[item] = od;
}

// One thread per (item, LLM, option): an option usable at the query (ok and within
// saturation) with u units is admissible for fraction f = u at every first-unit offset r
// (mod Q) where its replicas fit; it enters those entries by a 64-bit minimum.
__global__ void __launch_bounds__(256)
pruned_scatter_kernel(SpaceDev sp, const uint2 *__restrict__ rec, uint32_t count, uint32_t F1,
                      uint64_t *__restrict__ table)
{
    const uint64_t t = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= (uint64_t)count * sp.M * sp.O)
        return;
    const uint32_t o = (uint32_t)(t % sp.O);
    const uint64_t im = t / sp.O;                       // item * M + m
    const uint2 e = rec[t];
    const uint32_t u = e.y;                             // unusable options carry the sentinel
    if (u >= F1)
        return;
    const uint32_t ij = o / sp.D;
    const uint32_t tp = sp.tp(ij / sp.n_fq), q = sp.fq(ij % sp.n_fq), d = o % sp.D + 1;
    const uint64_t key = ((uint64_t)e.x << 32) | o;
    for (uint32_t r = 0; r < sp.Q; ++r)
        if (placement_fits(sp.Q, r, u, tp, q, d))
            atomicMin((unsigned long long *)&table[(im * sp.Q + r) * F1 + u],
                      (unsigned long long)key);
}

struct Walk {
    const uint64_t *table;
    uint32_t Q, F1;
    bool ordered;
    uint32_t L;                     // running best (L, x) and vector count of the thread
    uint64_t x;
    uint64_t count;
};

// Position K receives v units starting at unit `offset`; returns false if v is outside the
// position's range.  Adds the LLM's table entry when every LLM so far has an admissible option.
template <int M, int K>
__device__ __forceinline__ bool place_at(const Order &od, const Walk &w, uint32_t offset,
                                         uint32_t remaining, uint32_t prev, uint32_t v,
                                         uint32_t &L, uint64_t &x, bool &alive)
{
    uint32_t hi = od.hi[K];
    if (w.ordered && K > 0 && prev < hi)
        hi = prev;
    if (v < od.lo[K] || v > hi || v > remaining || remaining - v < od.lo_after[K])
        return false;
    if (alive) {
        const uint64_t e = w.table[od.tab[K] + (offset % w.Q) * w.F1 + v];
        if (e == kNoEntry) {
            alive = false;
        } else {
            L += (uint32_t)(e >> 32);
            x += (uint64_t)(uint32_t)e * od.pw[K];
        }
    }
    return true;
}

template <int M, int K>
__device__ __forceinline__ void walk_from(const Order &od, Walk &w, uint32_t offset,
                                          uint32_t remaining, uint32_t prev, uint32_t L,
                                          uint64_t x, bool alive)
{
    if constexpr (K == M - 1) {
        bool a = alive;
        if (!place_at<M, K>(od, w, offset, remaining, prev, remaining, L, x, a))
            return;
        w.count += 1;
        if (a && lex_less(L, x, w.L, w.x)) {
            w.L = L;
            w.x = x;
        }
    } else {
        // v ranges over [lo, min(hi, prev if ordered, remaining - lower bounds after K)]
        if (remaining < od.lo_after[K])
            return;
        uint32_t top = remaining - od.lo_after[K];
        if (od.hi[K] < top)
            top = od.hi[K];
        if (w.ordered && K > 0 && prev < top)
            top = prev;
        for (uint32_t v = od.lo[K]; v <= top; ++v) {
            uint32_t L2 = L;
            uint64_t x2 = x;
            bool a = alive;
            place_at<M, K>(od, w, offset, remaining, prev, v, L2, x2, a);
            walk_from<M, K + 1>(od, w, offset + v, remaining - v, v, L2, x2, a);
        }
    }
}

// Saturating C(n, k), k < 8, by Pascal's rule (additions only).
template <int KMAX>
__device__ uint64_t binomial_sat(uint32_t n, uint32_t k)
{
    uint64_t c[KMAX + 1];
#pragma unroll
    for (int j = 0; j <= KMAX; ++j)
        c[j] = j == 0 ? 1u : 0u;
    for (uint32_t i = 1; i <= n; ++i) {
#pragma unroll
        for (int j = KMAX; j >= 1; --j) {
            const uint64_t s = c[j] + c[j - 1];
            c[j] = s < c[j] ? ~0ull : s;
        }
    }
    uint64_t out = 0;
#pragma unroll
    for (int j = 0; j <= KMAX; ++j)
        if ((uint32_t)j == k)
            out = c[j];
    return out;
}

// Fractions fixed per thread: the first one for up to 3 LLMs, the first two beyond.
template <int M>
constexpr int kPrefix = M <= 3 ? 1 : 2;

// The item's table (M * Q * F1 entries) is copied to LDS first when `stage` is set (the
// launch then provides that much dynamic LDS): the walk's loads are dependent, and LDS latency
// is far below that of L2 or HBM.
template <int M>
__global__ void __launch_bounds__(256)
pruned_scan_kernel(SpaceDev sp, const Order *__restrict__ orders, uint32_t F1, uint32_t flags,
                   const uint64_t *__restrict__ table, uint32_t stage, uint32_t blocks_per_item,
                   Winner *__restrict__ winners, uint64_t *__restrict__ counts,
                   const uint2 *__restrict__ ext, uint32_t *__restrict__ done,
                   alp_pruned_t *__restrict__ out)
{
    extern __shared__ __align__(8) unsigned char s_dyn[];
    const uint32_t item = blockIdx.x / blocks_per_item;
    const uint32_t sub = blockIdx.x % blocks_per_item;
    const Order od = orders[item];
    const uint64_t per_item = (uint64_t)M * sp.Q * F1;
    const uint64_t *tab = table + item * per_item;
    if (stage) {
        uint64_t *s_tab = reinterpret_cast<uint64_t *>(s_dyn);
        for (uint32_t k = threadIdx.x; k < per_item; k += blockDim.x)
            s_tab[k] = tab[k];
        __syncthreads();
        tab = s_tab;
    }
    Walk w;
    w.table = tab;
    w.Q = sp.Q;
    w.F1 = F1;
    w.ordered = (flags & ALP_PRUNE_ORDER) != 0;
    w.L = kNoLatency;
    w.x = ~0ull;
    w.count = 0;

    const uint32_t F = od.F;
    const uint64_t t = (uint64_t)sub * blockDim.x + threadIdx.x;
    if (!od.empty) {
        if constexpr (M == 1) {
            if (t == 0)
                walk_from<M, 0>(od, w, 0, F, 0, 0, 0, true);
        } else if constexpr (kPrefix<M> == 1) {
            if (t <= F) {
                uint32_t L = 0;
                uint64_t x = 0;
                bool a = true;
                const uint32_t f0 = (uint32_t)t;
                if (place_at<M, 0>(od, w, 0, F, 0, f0, L, x, a))
                    walk_from<M, 1>(od, w, f0, F - f0, f0, L, x, a);
            }
        } else {
            const uint64_t F1i = (uint64_t)F + 1;
            if (t < F1i * F1i) {
                const uint32_t f0 = (uint32_t)(t / F1i), f1 = (uint32_t)(t % F1i);
                uint32_t L = 0;
                uint64_t x = 0;
                bool a = true;
                if (place_at<M, 0>(od, w, 0, F, 0, f0, L, x, a) &&
                    place_at<M, 1>(od, w, f0, F - f0, f0, f1, L, x, a))
                    walk_from<M, 2>(od, w, f0 + f1, F - f0 - f1, f1, L, x, a);
            }
        }
    }

    // Block totals: the vector count, then the (L, x) winner and the finished-block counter.
    __shared__ uint64_t s_count[4];
    uint64_t c = w.count;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        c += __shfl_xor((unsigned long long)c, off, 64);
    if ((threadIdx.x & 63) == 0)
        s_count[threadIdx.x >> 6] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t sum = 0;
        for (uint32_t k = 0; k < (blockDim.x >> 6); ++k)
            sum += s_count[k];
        counts[(uint64_t)item * blocks_per_item + sub] = sum;
    }
    if (!block_store_last(w.L, w.x, item, sub, blocks_per_item, winners, done) ||
        threadIdx.x >= 64)
        return;
    uint32_t L;
    uint64_t x;
    item_winner(item, blocks_per_item, winners, L, x);
    uint64_t total = 0;
    for (uint32_t k = threadIdx.x; k < blocks_per_item; k += 64)
        total += counts[(uint64_t)item * blocks_per_item + k];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        total += __shfl_xor((unsigned long long)total, off, 64);
    uint64_t *dst = reinterpret_cast<uint64_t *>(out + item);
    write_result(sp, ext + (uint64_t)item * M * sp.O, L, x, dst);
    if (threadIdx.x != 0)
        return;
    dst[6] = total;
    dst[7] = binomial_sat<M - 1>(F + M - 1, M - 1);
}

}  // namespace

// Largest per-item table staged in LDS (with the static LDS, well inside the 64 KiB a block
// gets without an opt-in).
constexpr uint64_t kStageBytes = 48 * 1024;

uint64_t pruned_prefixes(uint32_t M, uint32_t F_max)
{
    const uint64_t F1 = (uint64_t)F_max + 1;
    return M == 1 ? 1 : M <= 3 ? F1 : F1 * F1;
}

hipError_t launch_pruned_table(const SpaceDev &sp, const TablesDev &tb, const QueryDev &q,
                               uint32_t count, uint32_t F_max, uint32_t flags, const uint2 *rec,
                               uint64_t *table, void *orders, hipStream_t st)
{
    if (count == 0)
        return hipSuccess;
    const uint32_t F1 = F_max + 1;
    const uint64_t entries = (uint64_t)count * sp.M * sp.Q * F1;
    hipLaunchKernelGGL(pruned_prep_kernel, dim3((uint32_t)((entries + 255) / 256)), dim3(256), 0,
                       st, sp, tb, q, count, F1, flags, table, (Order *)orders);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    const uint64_t options = (uint64_t)count * sp.M * sp.O;
    hipLaunchKernelGGL(pruned_scatter_kernel, dim3((uint32_t)((options + 255) / 256)), dim3(256),
                       0, st, sp, rec, count, F1, table);
    return hipGetLastError();
}

hipError_t launch_pruned_scan(const SpaceDev &sp, uint32_t count, uint32_t F_max, uint32_t flags,
                              const uint64_t *table, const void *orders, uint32_t blocks_per_item,
                              Winner *winners, uint64_t *counts, const uint2 *ext, uint32_t *done,
                              alp_pruned_t *out, hipStream_t st)
{
    if (count == 0)
        return hipSuccess;
    const uint32_t F1 = F_max + 1;
    const dim3 grid(count * blocks_per_item), block(256);
    const Order *od = (const Order *)orders;
    const uint64_t item_bytes = (uint64_t)sp.M * sp.Q * F1 * sizeof(uint64_t);
    const uint32_t stage = item_bytes <= kStageBytes ? 1u : 0u;
    const size_t lds = stage ? (size_t)item_bytes : 0;
#define ALP_PRUNED_CASE(MM)                                                                        \
    case MM:                                                                                       \
        hipLaunchKernelGGL(pruned_scan_kernel<MM>, grid, block, lds, st, sp, od, F1, flags,       \
                           table, stage, blocks_per_item, winners, counts, ext, done, out);       \
        break;
    switch (sp.M) {
        ALP_PRUNED_CASE(1)
        ALP_PRUNED_CASE(2)
        ALP_PRUNED_CASE(3)
        ALP_PRUNED_CASE(4)
        ALP_PRUNED_CASE(5)
        ALP_PRUNED_CASE(6)
        ALP_PRUNED_CASE(7)
        ALP_PRUNED_CASE(8)
    default:
        return hipErrorInvalidValue;
    }
#undef ALP_PRUNED_CASE
    return hipGetLastError();
}

size_t pruned_order_bytes() { return sizeof(Order); }

}  // namespace alp
