// gfx950 kernel that places allocations on the GPUs of their budgets (Scepsy, arXiv 2604.15186,
// Section 6, hierarchical placement), one allocation per thread.
//
// G GPUs form nodes of 8 (the last may hold fewer), each node one all-to-all xGMI domain; a GPU
// holds Q share units.  LLM m's allocation is d_m replicas of tp_m ranks of q_m units, the ranks
// of a replica on distinct GPUs of one node.  Most-constrained-first: tensor-parallel replicas
// before single-GPU ones, larger replicas (tp * q units) first, ties by LLM index.
//   * A tensor-parallel replica takes, in some node, tp GPUs with q units free each: among the
//     node's GPUs with room ordered by (free units, index), a run of tp consecutive ones --
//     scored by imbalance (most minus least free), then the node's free units (the smaller
//     domain is preferred, keeping large ones for later), then the run's free units, then node
//     and position.  (A least-imbalance set with the least free units is always such a run.)
//   * A single-GPU replica packs onto an occupied GPU with room (fewest free units, then lowest
//     index); failing that, onto the lowest empty GPU of the node with the fewest free units.
// The free units of the thread's GPUs live in LDS, GPU-major, so that the 256 threads of a block
// touch consecutive bytes.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "alp_internal.h"

namespace alp {

namespace {

constexpr uint32_t kThreads = 256;
constexpr uint32_t kNode = ALP_NODE_GPUS;

__global__ void __launch_bounds__(kThreads)
place_kernel(uint32_t Q, uint32_t count, const PlaceIn *__restrict__ in,
             alp_placement_t *__restrict__ out)
{
    __shared__ uint8_t s_free[ALP_PLACE_MAX_GPUS * kThreads];
    const uint32_t t = blockIdx.x * kThreads + threadIdx.x;
    if (t >= count)
        return;
    const PlaceIn a = in[t];
    const uint32_t G = a.gpus, M = a.llms;
    uint8_t *fr = s_free + threadIdx.x;                 // fr[g * kThreads]: free units of GPU g
    for (uint32_t g = 0; g < G; ++g)
        fr[g * kThreads] = (uint8_t)Q;
    uint16_t *slot = out[t].slot;
    uint32_t total = 0, first[ALP_MAX_LLMS];
    for (uint32_t m = 0; m < M; ++m) {
        first[m] = total;
        total += a.d[m];
    }
    for (uint32_t i = 0; i < ALP_PLACE_MAX_REPLICAS; ++i)
        slot[i] = 0xFFFFu;
    // Most-constrained-first order of the LLMs (their replicas are placed together).
    uint32_t order[ALP_MAX_LLMS], k = 0;
    for (uint32_t m = 0; m < M; ++m)
        if (a.d[m])
            order[k++] = m;
    for (uint32_t i = 1; i < k; ++i) {
        const uint32_t v = order[i];
        const uint32_t vkind = a.tp[v] == 1, vsize = (uint32_t)a.tp[v] * a.q[v];
        uint32_t j = i;
        while (j > 0) {
            const uint32_t u = order[j - 1];
            const uint32_t ukind = a.tp[u] == 1, usize = (uint32_t)a.tp[u] * a.q[u];
            const bool before = vkind < ukind || (vkind == ukind && (vsize > usize ||
                                                 (vsize == usize && v < u)));
            if (!before)
                break;
            order[j] = u;
            --j;
        }
        order[j] = v;
    }
    const uint32_t nodes = (G + kNode - 1) / kNode;
    bool placed = a.feasible != 0;
    uint32_t done = 0;
    for (uint32_t i = 0; i < k && placed; ++i) {
        const uint32_t m = order[i], tp = a.tp[m], q = a.q[m];
        for (uint32_t r = 0; r < a.d[m] && placed; ++r) {
            uint32_t node = 0, mask = 0;
            bool found = false;
            if (tp > 1) {
                uint32_t b_imb = 0, b_dom = 0, b_cap = 0;
                for (uint32_t n = 0; n < nodes; ++n) {
                    const uint32_t lo = n * kNode, hi = lo + kNode < G ? lo + kNode : G;
                    // rank of each GPU with room by (free, index): GPU of rank j is pos[j]
                    uint32_t pos[kNode], e = 0, dom = 0;
                    for (uint32_t g = lo; g < hi; ++g) {
                        const uint32_t f = fr[g * kThreads];
                        dom += f;
                        if (f < q)
                            continue;
                        uint32_t j = e++;
                        while (j > 0 && (fr[pos[j - 1] * kThreads] > f)) {
                            pos[j] = pos[j - 1];
                            --j;
                        }
                        pos[j] = g;
                    }
                    for (uint32_t s = 0; s + tp <= e; ++s) {
                        const uint32_t imb = fr[pos[s + tp - 1] * kThreads] - fr[pos[s] * kThreads];
                        uint32_t cap = 0, msk = 0;
                        for (uint32_t j = s; j < s + tp; ++j) {
                            cap += fr[pos[j] * kThreads];
                            msk |= 1u << (pos[j] - lo);
                        }
                        if (!found || imb < b_imb || (imb == b_imb && dom < b_dom) ||
                            (imb == b_imb && dom == b_dom && cap < b_cap)) {
                            found = true;
                            b_imb = imb;
                            b_dom = dom;
                            b_cap = cap;
                            node = n;
                            mask = msk;
                        }
                    }
                }
                if (found)
                    for (uint32_t j = 0; j < kNode; ++j)
                        if (mask >> j & 1u)
                            fr[(node * kNode + j) * kThreads] -= (uint8_t)q;
            } else {
                uint32_t best = G;
                for (uint32_t g = 0; g < G; ++g) {
                    const uint32_t f = fr[g * kThreads];
                    if (f < Q && f >= q && (best == G || f < fr[best * kThreads]))
                        best = g;
                }
                if (best == G) {
                    uint32_t best_free = 0;
                    for (uint32_t n = 0; n < nodes; ++n) {
                        const uint32_t lo = n * kNode, hi = lo + kNode < G ? lo + kNode : G;
                        uint32_t nf = 0, empty = G;
                        for (uint32_t g = lo; g < hi; ++g) {
                            const uint32_t f = fr[g * kThreads];
                            nf += f;
                            if (f == Q && empty == G)
                                empty = g;
                        }
                        if (empty != G && (best == G || nf < best_free)) {
                            best = empty;
                            best_free = nf;
                        }
                    }
                }
                if (best != G) {
                    found = true;
                    fr[best * kThreads] -= (uint8_t)q;
                    node = best / kNode;
                    mask = 1u << (best % kNode);
                }
            }
            if (!found) {
                placed = false;
                break;
            }
            slot[first[m] + r] = (uint16_t)(node << 8 | mask);
            ++done;
        }
    }
    uint32_t gpus = 0, used_nodes = 0;
    for (uint32_t n = 0; n < nodes; ++n) {
        uint32_t used = 0;
        for (uint32_t g = n * kNode; g < G && g < (n + 1) * kNode; ++g)
            used += fr[g * kThreads] < Q;
        gpus += used;
        used_nodes += used > 0;
    }
    out[t].status = placed ? ALP_OK : ALP_INFEASIBLE;
    out[t].replicas = done;
    out[t].gpus_used = gpus;
    out[t].nodes_used = used_nodes;
}

}  // namespace

hipError_t launch_place(uint32_t Q, uint32_t count, const PlaceIn *in, alp_placement_t *out,
                        hipStream_t st)
{
    if (count == 0)
        return hipSuccess;
    hipLaunchKernelGGL(place_kernel, dim3((count + kThreads - 1) / kThreads), dim3(kThreads), 0,
                       st, Q, count, in, out);
    return hipGetLastError();
}

}  // namespace alp
