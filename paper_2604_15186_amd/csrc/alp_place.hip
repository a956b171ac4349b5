// gfx950 kernel that places allocations on the GPUs of their budgets (Scepsy, arXiv 2604.15186,
// Section 6, hierarchical placement), one wave per allocation, lane g holding GPU g.
//
// G <= 64 GPUs form nodes of 8 (the last may hold fewer), each node one all-to-all xGMI domain;
// a GPU holds Q share units.  LLM m's allocation is d_m replicas of tp_m ranks of q_m units, the
// ranks of a replica on distinct GPUs of one node.  Most-constrained-first: tensor-parallel
// replicas before single-GPU ones, larger replicas (tp * q units) first, ties by LLM index.
//   * A tensor-parallel replica takes, in some node, tp GPUs with q units free each: among the
//     node's GPUs with room ordered by (free units, index), a run of tp consecutive ones --
//     scored by imbalance (most minus least free), then the node's free units (the smaller
//     domain is preferred, keeping large ones for later), then the run's free units, then node
//     and position.  (A least-imbalance set with the least free units is always such a run.)
//   * A single-GPU replica packs onto an occupied GPU with room (fewest free units, then lowest
//     index); failing that, onto the lowest empty GPU of the node with the fewest free units.
// Replicas are placed one after the other (each sees the units the earlier ones took); within a
// replica every lane scores its own GPU, or the run its GPU starts, from its node's free units
// (kept by every lane of the node, one byte per GPU), and a wave minimum over one packed 32-bit
// key per lane picks the choice with the order above.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "alp_device.h"
#include "alp_internal.h"

namespace alp {

namespace {

constexpr uint32_t kWavesPerBlock = 4;
constexpr uint32_t kNode = ALP_NODE_GPUS;
constexpr uint32_t kNone = 0xFFFFFFFFu;
static_assert(ALP_PLACE_MAX_GPUS == 64, "one lane per GPU of a wave");
static_assert(kNode == 8, "a node is an 8-lane group of the wave");

// Free units of the 8 GPUs of a node, one byte each (GPU j of the node in byte j of lo for
// j < 4, of hi for j >= 4): every lane of the node keeps the same copy, so scoring a replica
// needs no cross-lane traffic.
struct NodeFree {
    uint32_t lo, hi;
    __device__ __forceinline__ uint32_t get(uint32_t j) const
    {
        return __builtin_amdgcn_ubfe(j < 4 ? lo : hi, 8 * (j & 3), 8);
    }
    __device__ __forceinline__ void sub(uint32_t j, uint32_t v)
    {
        if (j < 4)
            lo -= v << (8 * j);
        else
            hi -= v << (8 * (j - 4));
    }
};

// Sorts 8 keys ascending in registers (a 19-comparator network).
__device__ __forceinline__ void sort8(uint32_t (&k)[8])
{
    auto cs = [&](int i, int j) {
        const uint32_t a = k[i], b = k[j];
        k[i] = a < b ? a : b;
        k[j] = a < b ? b : a;
    };
    cs(0, 1); cs(2, 3); cs(4, 5); cs(6, 7);
    cs(0, 2); cs(1, 3); cs(4, 6); cs(5, 7);
    cs(1, 2); cs(5, 6); cs(0, 4); cs(3, 7);
    cs(1, 5); cs(2, 6);
    cs(1, 4); cs(3, 6);
    cs(2, 4); cs(3, 5);
    cs(3, 4);
}

__global__ void __launch_bounds__(64 * kWavesPerBlock)
place_kernel(uint32_t Q, uint32_t count, const PlaceIn *__restrict__ in,
             alp_placement_t *__restrict__ out)
{
    const uint32_t lane = threadIdx.x & 63;
    const uint32_t t = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    if (t >= count)
        return;                                        // uniform over the wave
    const PlaceIn a = in[t];
    const uint32_t G = a.gpus, M = a.llms;
    const uint32_t node = lane / kNode, pos = lane % kNode;
    const bool gpu = lane < G;
    // GPUs of this lane's node (the last node may hold fewer), and the node's free units.
    const uint32_t node_gpus = G > node * kNode ? (G - node * kNode < kNode ? G - node * kNode : kNode)
                                                : 0u;
    NodeFree F{0u, 0u};
    for (uint32_t j = 0; j < node_gpus; ++j)
        F.sub(j, 0u - Q);                              // adds Q to byte j
    // Lane L keeps slots 2L and 2L + 1 (128 16-bit slots, "not placed" until set) and stores
    // them once at the end.
    uint32_t slots = 0xFFFFFFFFu;
    auto set_slot = [&](uint32_t s, uint32_t v) {
        if (lane == s >> 1)
            slots = s & 1u ? (slots & 0xFFFFu) | v << 16 : (slots & 0xFFFF0000u) | v;
    };
    uint32_t first[ALP_MAX_LLMS], total = 0;
    for (uint32_t m = 0; m < M; ++m) {
        first[m] = total;
        total += a.d[m];
    }
    // Most-constrained-first order of the LLMs (their replicas are placed together); the same
    // in every lane.
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
    bool placed = a.feasible != 0;
    uint32_t done = 0;
    for (uint32_t i = 0; i < k && placed; ++i) {
        const uint32_t m = order[i], tp = a.tp[m], q = a.q[m];
        for (uint32_t r = 0; r < a.d[m]; ++r) {
            const uint32_t f = F.get(pos);
            uint32_t fj[kNode], dom = 0;
#pragma unroll
            for (uint32_t j = 0; j < kNode; ++j) {
                fj[j] = F.get(j);
                dom += fj[j];
            }
            uint32_t key, bn, mask;
            if (tp > 1) {
                // GPUs of the node with room as keys (free, index), sorted; this lane's run is
                // the tp keys from its own on.
                uint32_t ks[kNode], rank = 0, rooms = 0;
                const uint32_t mine = f << 3 | pos;
#pragma unroll
                for (uint32_t j = 0; j < kNode; ++j) {
                    const bool rj = j < node_gpus && fj[j] >= q;
                    ks[j] = rj ? fj[j] << 3 | j : 0xFFFFu;
                    rooms += rj;
                    rank += rj && ks[j] < mine;
                }
                sort8(ks);
                uint32_t cap = 0, fmax = 0, run = 0;
#pragma unroll
                for (uint32_t i = 0; i < kNode; ++i) {
                    if (i >= rank && i < rank + tp && ks[i] != 0xFFFFu) {
                        cap += ks[i] >> 3;
                        fmax = ks[i] >> 3;                 // ascending: the last one is the most
                        run |= 1u << (ks[i] & 7u);
                    }
                }
                const bool room = gpu && f >= q;
                // imbalance <= Q <= 16, node and run free units <= 8 * 16, node < 8, rank < 8
                key = room && rank + tp <= rooms
                          ? (fmax - f) << 24 | dom << 16 | cap << 8 | node << 3 | rank
                          : kNone;
                const uint32_t best = wave_min_u32(key);
                if (best == kNone) {
                    placed = false;
                    break;
                }
                // The winning run, as seen by the lane that proposed it.
                bn = (best >> 3) & 7u;
                const uint64_t won = __ballot(key == best);
                mask = (uint32_t)__builtin_amdgcn_readlane((int)run,
                                                           (int)__builtin_ctzll(won));
            } else {
                // An occupied GPU with room, fewest free units, lowest index.
                key = gpu && f < Q && f >= q ? f << 8 | lane : kNone;
                uint32_t best = wave_min_u32(key), g = best & 0xFFu;
                if (best == kNone) {
                    // The lowest empty GPU of the node with the fewest free units.
                    uint32_t empty = 0;
#pragma unroll
                    for (uint32_t j = 0; j < kNode; ++j)
                        empty |= (uint32_t)(j < node_gpus && fj[j] == Q) << j;
                    key = pos == 0 && empty ? dom << 8 | node << 3 | (uint32_t)__builtin_ctz(empty)
                                            : kNone;
                    best = wave_min_u32(key);
                    if (best == kNone) {
                        placed = false;
                        break;
                    }
                    g = ((best >> 3) & 7u) * kNode + (best & 7u);
                }
                bn = g / kNode;
                mask = 1u << (g % kNode);
            }
            if (node == bn) {
#pragma unroll
                for (uint32_t j = 0; j < kNode; ++j)
                    if (mask >> j & 1u)
                        F.sub(j, q);
            }
            set_slot(first[m] + r, bn << 8 | mask);
            ++done;
        }
    }
    reinterpret_cast<uint32_t *>(out[t].slot)[lane] = slots;
    const uint64_t used = __ballot(gpu && F.get(pos) < Q);
    uint32_t used_nodes = 0;
    for (uint32_t n = 0; n < ALP_PLACE_MAX_GPUS / kNode; ++n)
        used_nodes += (used >> (n * kNode) & 0xFFu) != 0;
    if (lane == 0) {
        out[t].status = placed ? ALP_OK : ALP_INFEASIBLE;
        out[t].replicas = done;
        out[t].gpus_used = (uint32_t)__popcll(used);
        out[t].nodes_used = used_nodes;
    }
}

}  // namespace

hipError_t launch_place(uint32_t Q, uint32_t count, const PlaceIn *in, alp_placement_t *out,
                        hipStream_t st)
{
    if (count == 0)
        return hipSuccess;
    hipLaunchKernelGGL(place_kernel, dim3((count + kWavesPerBlock - 1) / kWavesPerBlock),
                       dim3(64 * kWavesPerBlock), 0, st, Q, count, in, out);
    return hipGetLastError();
}

}  // namespace alp
