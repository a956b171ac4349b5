// gfx950 kernel that splits a GPU pool over several workflows (Scepsy, arXiv 2604.15186,
// Section 5, scheduling multiple workflows).  Its input is the table of per-workflow search
// results at every budget 0..G, which the search kernels have already written.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "alp_internal.h"

namespace alp {

namespace {

// Budget split over workflows (Section 5, scheduling multiple workflows), one block.
// L(w, g) = latency of workflow w's search at g GPUs, or none.  Egalitarian: the smallest
// largest latency t* is found by thresholds (workflow w needs the fewest g with L(w, g) <= t;
// t is reachable iff those budgets fit in G; t* is one of the table's values); then, among
// splits whose latencies are all <= t*, the smallest latency sum comes from a knapsack over the
// budget, and taking each workflow's smallest budget that stays optimal gives the
// lexicographically smallest vector.  Social welfare: the same without the threshold.
__global__ void __launch_bounds__(256)
allocate_kernel(const alp_result_t *__restrict__ res, uint32_t W, uint32_t G, uint32_t policy,
                uint64_t *__restrict__ dp, alp_plan_t *__restrict__ plan, uint32_t *__restrict__ gpus)
{
    constexpr uint64_t kInf = ~0ull;
    __shared__ uint32_t red[256];
    const uint32_t G1 = G + 1;
    // Scratch after the knapsack table: latency table and its running minimum over budgets.
    uint32_t *lt = reinterpret_cast<uint32_t *>(dp + (uint64_t)(W + 1) * G1);
    uint32_t *pm = lt + (uint64_t)W * G1;
    for (uint32_t a = threadIdx.x; a < W * G1; a += blockDim.x) {
        const alp_result_t &r = res[a];
        lt[a] = r.status == ALP_OK ? r.latency_us : kNoLatency;
    }
    __syncthreads();
    for (uint32_t w = threadIdx.x; w < W; w += blockDim.x) {
        uint32_t m = kNoLatency;
        for (uint32_t g = 0; g < G1; ++g) {
            const uint32_t l = lt[w * G1 + g];
            m = l < m ? l : m;
            pm[w * G1 + g] = m;
        }
    }
    __syncthreads();
    auto lat = [&](uint32_t w, uint32_t g) -> uint32_t { return lt[w * G1 + g]; };
    // 1. Threshold (egalitarian only): workflow w needs the first g whose running minimum is
    //    <= t (binary search; the running minimum does not increase with g).
    uint32_t t_star = kNoLatency - 1;     // social: every feasible latency is allowed
    if (policy == ALP_WELFARE_EGALITARIAN) {
        uint32_t best = kNoLatency;
        for (uint32_t a = threadIdx.x; a < W * G1; a += blockDim.x) {
            const uint32_t t = lt[a];
            if (t == kNoLatency || t >= best)
                continue;
            uint32_t need = 0;
            bool reachable = true;
            for (uint32_t w = 0; w < W && reachable; ++w) {
                const uint32_t *row = pm + w * G1;
                if (row[G] > t) {
                    reachable = false;
                    break;
                }
                uint32_t lo = 0, hi = G;           // first g with row[g] <= t lies in [lo, hi]
                while (lo < hi) {
                    const uint32_t mid = (lo + hi) / 2;
                    if (row[mid] <= t)
                        hi = mid;
                    else
                        lo = mid + 1;
                }
                need += lo;
            }
            if (reachable && need <= G)
                best = t;
        }
        red[threadIdx.x] = best;
        __syncthreads();
        for (uint32_t s = blockDim.x / 2; s > 0; s >>= 1) {
            if (threadIdx.x < s && red[threadIdx.x + s] < red[threadIdx.x])
                red[threadIdx.x] = red[threadIdx.x + s];
            __syncthreads();
        }
        t_star = red[0];
        __syncthreads();
    }
    // 2. Knapsack over the budget, workflows from last to first: dp[w][b] = smallest latency sum
    //    of workflows w..W-1 within b GPUs (latencies <= t_star), kInf if none.
    for (uint32_t b = threadIdx.x; b < G1; b += blockDim.x)
        dp[(uint64_t)W * G1 + b] = 0;
    __syncthreads();
    for (int w = (int)W - 1; w >= 0; --w) {
        for (uint32_t b = threadIdx.x; b < G1; b += blockDim.x) {
            uint64_t best = kInf;
            if (t_star != kNoLatency) {
                for (uint32_t g = 0; g <= b; ++g) {
                    const uint32_t l = lat(w, g);
                    const uint64_t rest = dp[(uint64_t)(w + 1) * G1 + (b - g)];
                    if (l != kNoLatency && l <= t_star && rest != kInf && l + rest < best)
                        best = l + rest;
                }
            }
            dp[(uint64_t)w * G1 + b] = best;
        }
        __syncthreads();
    }
    // 3. Lexicographically smallest optimal budget vector.
    if (threadIdx.x != 0)
        return;
    alp_plan_t p;
    p.policy = policy;
    if (dp[G] == kInf) {
        p.status = ALP_INFEASIBLE;
        p.max_latency_us = 0;
        p.gpus_used = 0;
        p.sum_latency_us = 0;
        *plan = p;
        return;
    }
    uint32_t b = G, used = 0, mx = 0;
    for (uint32_t w = 0; w < W; ++w) {
        const uint64_t target = dp[(uint64_t)w * G1 + b];
        for (uint32_t g = 0; g <= b; ++g) {
            const uint32_t l = lat(w, g);
            const uint64_t rest = dp[(uint64_t)(w + 1) * G1 + (b - g)];
            if (l != kNoLatency && l <= t_star && rest != kInf && l + rest == target) {
                gpus[w] = g;
                used += g;
                mx = l > mx ? l : mx;
                b -= g;
                break;
            }
        }
    }
    p.status = ALP_OK;
    p.max_latency_us = mx;
    p.gpus_used = used;
    p.sum_latency_us = dp[G];
    *plan = p;
}

}  // namespace

hipError_t launch_allocate(const alp_result_t *res, uint32_t W, uint32_t G, uint32_t policy,
                           uint64_t *dp, alp_plan_t *plan, uint32_t *gpus, hipStream_t st)
{
    hipLaunchKernelGGL(allocate_kernel, dim3(1), dim3(256), 0, st, res, W, G, policy, dp, plan,
                       gpus);
    return hipGetLastError();
}

}  // namespace alp
