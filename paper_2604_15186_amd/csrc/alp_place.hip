// gfx950 kernel that places allocations on the GPUs of their budgets (Scepsy, arXiv 2604.15186,
// Section 6, hierarchical placement): one wave per allocation, or one 16-lane row of a wave
// for budgets of at most 16 GPUs (four allocations per wave); lane g of the allocation's lanes
// holds GPU g.
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
// (kept by every lane of the node, one byte per GPU), and a minimum over the allocation's lanes
// of one packed 32-bit key per lane picks the choice with the order above.
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

// Free units of the 8 GPUs of a node, one byte each (GPU j of the node in byte j): every lane
// of the node keeps the same copy, so scoring a replica needs no cross-lane traffic.  One 64-bit
// value, shifted by the GPU (a choice between two halves would be compiled as an index into a
// per-lane array, kept in LDS).
struct NodeFree {
    uint64_t v;
    __device__ __forceinline__ uint32_t get(uint32_t j) const
    {
        return (uint32_t)(v >> (8 * j)) & 0xFFu;
    }
    __device__ __forceinline__ void sub(uint32_t j, uint32_t x)
    {
        v -= (uint64_t)x << (8 * j);
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

// Minimum over the L lanes of this lane's allocation, in every one of them: the whole wave (L =
// 64, a wave-uniform value) or its 16-lane row (quad swaps, then the row's half mirror and
// mirror).
template <uint32_t L>
__device__ __forceinline__ uint32_t group_min(uint32_t v)
{
    if constexpr (L == 64) {
        return wave_min_u32(v);
    } else {
        static_assert(L == 16, "an allocation takes the wave or one 16-lane row");
        auto step = [&](auto c) {
            constexpr int C = decltype(c)::value;
            const uint32_t o = dpp_mov<C>(v, v);
            v = o < v ? o : v;
        };
        step(std::integral_constant<int, 0xB1>{});
        step(std::integral_constant<int, 0x4E>{});
        step(std::integral_constant<int, 0x141>{});
        step(std::integral_constant<int, 0x140>{});
        return v;
    }
}

// v of lane `src` of the wave (src the same within each allocation's lanes).
template <uint32_t L>
__device__ __forceinline__ uint32_t group_read(uint32_t v, uint32_t src)
{
    if constexpr (L == 64)
        return (uint32_t)__builtin_amdgcn_readlane((int)v, (int)src);
    else
        return (uint32_t)__builtin_amdgcn_ds_bpermute((int)(src << 2), (int)v);
}

// L lanes per allocation: 64 (one allocation per wave, G <= 64) or 16 (four per wave, one per
// 16-lane row, G <= 16); lane g of an allocation's lanes holds its GPU g.  Every decision below
// depends only on the allocation, so its lanes take the same path.
template <uint32_t L>
__global__ void __launch_bounds__(64 * kWavesPerBlock)
place_kernel(uint32_t Q, uint32_t count, const PlaceIn *__restrict__ in,
             alp_placement_t *__restrict__ out)
{
    constexpr uint32_t kPerWave = 64 / L, kWords = 64 / L;   // allocations, slot words per lane
    const uint32_t lane = threadIdx.x & 63;
    const uint32_t gl = lane % L, first_lane = lane - gl;
    const uint32_t t = (blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6)) * kPerWave + lane / L;
    if (t >= count)
        return;                                        // uniform over the allocation's lanes
    // The allocation's fields as packed words (byte m of tp, q, d is LLM m's), so that nothing
    // below is indexed in a per-lane array: such arrays would be kept in LDS at an offset from
    // the flat thread index, whose workgroup size is read from the dispatch packet in host
    // memory -- a PCIe round trip that every wave would wait for.
    const PlaceIn a = in[t];
    const uint32_t G = a.gpus, M = a.llms;
    auto bytes64 = [](const uint8_t (&b)[ALP_MAX_LLMS]) {
        uint64_t v = 0;
#pragma unroll
        for (uint32_t m = 0; m < ALP_MAX_LLMS; ++m)
            v |= (uint64_t)b[m] << (8 * m);
        return v;
    };
    const uint64_t tp_w = bytes64(a.tp), q_w = bytes64(a.q), d_w = bytes64(a.d);
    auto byte_of = [](uint64_t v, uint32_t m) { return (uint32_t)(v >> (8 * m)) & 0xFFu; };
    const uint32_t node = gl / kNode, pos = gl % kNode;
    const bool gpu = gl < G;
    // GPUs of this lane's node (the last node may hold fewer), and the node's free units.
    const uint32_t node_gpus = G > node * kNode ? (G - node * kNode < kNode ? G - node * kNode : kNode)
                                                : 0u;
    NodeFree F{0ull};
    for (uint32_t j = 0; j < node_gpus; ++j)
        F.v += (uint64_t)Q << (8 * j);
    // Lane g keeps slots 2 kWords g .. 2 kWords g + 2 kWords - 1 (128 16-bit slots, "not
    // placed" until set) and stores them once at the end.
    uint32_t slots[kWords];
#pragma unroll
    for (uint32_t k = 0; k < kWords; ++k)
        slots[k] = 0xFFFFFFFFu;
    auto set_slot = [&](uint32_t s, uint32_t v) {
        if (gl == s / (2 * kWords)) {
            const uint32_t k = (s / 2) % kWords;
#pragma unroll
            for (uint32_t kk = 0; kk < kWords; ++kk)
                if (kk == k)
                    slots[kk] = s & 1u ? (slots[kk] & 0xFFFFu) | v << 16
                                       : (slots[kk] & 0xFFFF0000u) | v;
        }
    };
    // First slot of each LLM's replicas (byte m; at most 8 x 16 replicas in all).
    uint64_t first_w = 0;
    uint32_t total = 0;
#pragma unroll
    for (uint32_t m = 0; m < ALP_MAX_LLMS; ++m) {
        first_w |= (uint64_t)total << (8 * m);
        total += m < M ? byte_of(d_w, m) : 0u;
    }
    // Most-constrained-first order of the LLMs with replicas (their replicas are placed
    // together): ascending keys (single-GPU replicas after tensor-parallel ones, then larger
    // replicas first, then the LLM index), sorted by the network; order_w holds the LLMs, four
    // bits each.
    uint32_t keys[ALP_MAX_LLMS];
#pragma unroll
    for (uint32_t m = 0; m < ALP_MAX_LLMS; ++m) {
        const uint32_t tpm = byte_of(tp_w, m), size = tpm * byte_of(q_w, m);   // <= 128
        keys[m] = m < M && byte_of(d_w, m) ? (uint32_t)(tpm == 1) << 16 | (0xFFu - size) << 8 | m
                                           : 0xFFFFFFFFu;
    }
    sort8(keys);
    uint32_t order_w = 0, k = 0;
#pragma unroll
    for (uint32_t i = 0; i < ALP_MAX_LLMS; ++i) {
        order_w |= (keys[i] & 7u) << (4 * i);
        k += keys[i] != 0xFFFFFFFFu;
    }
    bool placed = a.feasible != 0;
    uint32_t done = 0;
    for (uint32_t i = 0; i < k && placed; ++i) {
        const uint32_t m = (order_w >> (4 * i)) & 7u, tp = byte_of(tp_w, m), q = byte_of(q_w, m);
        const uint32_t dm = byte_of(d_w, m), fm = byte_of(first_w, m);
        for (uint32_t r = 0; r < dm; ++r) {
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
                const uint32_t best = group_min<L>(key);
                if (best == kNone) {
                    placed = false;
                    break;
                }
                // The winning run, as seen by the lane that proposed it.
                bn = (best >> 3) & 7u;
                const uint64_t won = __ballot(key == best) >> first_lane;
                mask = group_read<L>(run, first_lane + (uint32_t)__builtin_ctzll(won));
            } else {
                // An occupied GPU with room, fewest free units, lowest index.
                key = gpu && f < Q && f >= q ? f << 8 | gl : kNone;
                uint32_t best = group_min<L>(key), g = best & 0xFFu;
                if (best == kNone) {
                    // The lowest empty GPU of the node with the fewest free units.
                    uint32_t empty = 0;
#pragma unroll
                    for (uint32_t j = 0; j < kNode; ++j)
                        empty |= (uint32_t)(j < node_gpus && fj[j] == Q) << j;
                    key = pos == 0 && empty ? dom << 8 | node << 3 | (uint32_t)__builtin_ctz(empty)
                                            : kNone;
                    best = group_min<L>(key);
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
            set_slot(fm + r, bn << 8 | mask);
            ++done;
        }
    }
    alp_placement_t *dst = out + a.dst;
#pragma unroll
    for (uint32_t kk = 0; kk < kWords; ++kk)
        reinterpret_cast<uint32_t *>(dst->slot)[gl * kWords + kk] = slots[kk];
    const uint64_t used_all = __ballot(gpu && F.get(pos) < Q) >> first_lane;
    const uint64_t used = L == 64 ? used_all : used_all & ((1ull << L) - 1);
    uint32_t used_nodes = 0;
    for (uint32_t n = 0; n < L / kNode; ++n)
        used_nodes += (used >> (n * kNode) & 0xFFu) != 0;
    if (gl == 0) {
        dst->status = placed ? ALP_OK : ALP_INFEASIBLE;
        dst->replicas = done;
        dst->gpus_used = (uint32_t)__popcll(used);
        dst->nodes_used = used_nodes;
    }
}

}  // namespace

hipError_t launch_place(uint32_t Q, uint32_t small, uint32_t large, const PlaceIn *in,
                        alp_placement_t *out, hipStream_t st)
{
    if (small) {
        const uint32_t per_block = kWavesPerBlock * 4;
        hipLaunchKernelGGL(place_kernel<16>, dim3((small + per_block - 1) / per_block),
                           dim3(64 * kWavesPerBlock), 0, st, Q, small, in, out);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess)
            return e;
    }
    if (large) {
        hipLaunchKernelGGL(place_kernel<64>, dim3((large + kWavesPerBlock - 1) / kWavesPerBlock),
                           dim3(64 * kWavesPerBlock), 0, st, Q, large, in + small, out);
        return hipGetLastError();
    }
    return hipSuccess;
}

}  // namespace alp
