// Device helpers shared by the gfx950 kernels: wave and block minima of (L, x), the end-of-item
// reduction of block winners with result decoding, and block renumbering across XCDs.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "alp_internal.h"

namespace alp {
namespace {

__device__ __forceinline__ bool lex_less(uint32_t aL, uint64_t ax, uint32_t bL, uint64_t bx)
{
    return aL < bL || (aL == bL && ax < bx);
}

// Wave-wide lexicographic minimum of (L, x); every lane ends with the result.
__device__ __forceinline__ void wave_min(uint32_t &L, uint64_t &x)
{
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        uint32_t oL = __shfl_xor(L, off, 64);
        uint64_t ox = __shfl_xor((unsigned long long)x, off, 64);
        if (lex_less(oL, ox, L, x)) {
            L = oL;
            x = ox;
        }
    }
}

// Wave-wide minima, returned as wave-uniform values.
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v)
{
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const uint32_t o = __shfl_xor(v, off, 64);
        v = o < v ? o : v;
    }
    return (uint32_t)__builtin_amdgcn_readfirstlane(v);
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v)
{
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const uint64_t o = __shfl_xor((unsigned long long)v, off, 64);
        v = o < v ? o : v;
    }
    // readfirstlane works on int: widen through uint32_t, never sign-extend.
    return ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(v >> 32)) << 32) |
           (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)v);
}

// Block-wide minimum; thread 0 writes the block's winner.
__device__ __forceinline__ void block_min_store(uint32_t L, uint64_t x, Winner *dst)
{
    __shared__ uint32_t sL[16];
    __shared__ uint64_t sx[16];
    wave_min(L, x);
    const uint32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    if (lane == 0) {
        sL[wave] = L;
        sx[wave] = x;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (uint32_t w = 1; w < nw; ++w)
            if (lex_less(sL[w], sx[w], L, x)) {
                L = sL[w];
                x = sx[w];
            }
        Winner r;
        r.L = L;
        r.pad = 0;
        r.x = x;
        *dst = r;
    }
}

// Lexicographic (L, x) minimum of an item's block winners, by one wave; every lane gets it.
__device__ __forceinline__ void item_winner(uint32_t item, uint32_t blocks_per_item,
                                            const Winner *winners, uint32_t &L, uint64_t &x)
{
    const uint32_t lane = threadIdx.x & 63;
    L = kNoLatency;
    x = ~0ull;
    for (uint32_t k = lane; k < blocks_per_item; k += 64) {
        const Winner w = winners[(uint64_t)item * blocks_per_item + k];
        if (lex_less(w.L, w.x, L, x)) {
            L = w.L;
            x = w.x;
        }
    }
    wave_min(L, x);
}

// The result record of winner (L, x) -- decoded per-LLM choices, T_w (Eq. 2: minimum over LLMs)
// and the share units, from the item's per-option records E -- written by one thread as the six
// 64-bit words of alp_result_t.  (Assembled in registers: a local struct indexed at run time
// would be placed in memory for every thread of the block.)
__device__ __forceinline__ void write_result(const SpaceDev &sp, const uint2 *E, uint32_t L,
                                             uint64_t x, uint64_t *dst)
{
    uint64_t word[6] = {ALP_NO_INDEX, 0, (uint64_t)ALP_INFEASIBLE << 32, 0, 0, 0};
    if (L != kNoLatency) {
        uint64_t rr = x;
        uint32_t T = 0xFFFFFFFFu, U = 0;
        uint64_t tp = 0, fq = 0, rep = 0;
        for (int m = (int)sp.M - 1; m >= 0; --m) {
            const uint32_t o = (uint32_t)(rr % sp.O);
            rr /= sp.O;
            const uint2 e = E[(uint64_t)m * sp.O + o];
            T = e.x < T ? e.x : T;                      // Eq. 2: minimum over LLMs
            U += e.y & 0xFFFFu;
            const uint32_t ij = o / sp.D;
            tp |= (uint64_t)(sp.tp[ij / sp.n_fq] & 0xFFu) << (8 * m);
            fq |= (uint64_t)(sp.fq[ij % sp.n_fq] & 0xFFu) << (8 * m);
            rep |= (uint64_t)((o % sp.D + 1) & 0xFFu) << (8 * m);
        }
        word[0] = x;
        word[1] = (uint64_t)L | ((uint64_t)T << 32);
        word[2] = (uint64_t)U | ((uint64_t)ALP_OK << 32);
        word[3] = tp;
        word[4] = fq;
        word[5] = rep;
    }
#pragma unroll
    for (int k = 0; k < 6; ++k)
        dst[k] = word[k];
}

// Result of one item from its block winners, by one wave.
__device__ __forceinline__ void finish_item(const FinishArgs &fa, uint32_t item,
                                            uint32_t blocks_per_item, const Winner *winners)
{
    uint32_t L;
    uint64_t x;
    item_winner(item, blocks_per_item, winners, L, x);
    if ((threadIdx.x & 63) == 0)
        write_result(fa.sp, fa.ext + (uint64_t)item * fa.sp.M * fa.sp.O, L, x,
                     reinterpret_cast<uint64_t *>(fa.out + item));
}

// Writes the block's winner and counts the block as finished (agent-scope fence and per-item
// counter, zeroed by option_terms_kernel); true in every thread of the item's last block, which
// then sees every other block's writes.
__device__ __forceinline__ bool block_store_last(uint32_t L, uint64_t x, uint32_t item,
                                                 uint32_t sub, uint32_t blocks_per_item,
                                                 Winner *winners, uint32_t *done)
{
    __shared__ uint32_t last_block;
    block_min_store(L, x, &winners[(uint64_t)item * blocks_per_item + sub]);
    if (blocks_per_item == 1) {
        // The block is the whole item: its own writes only need to reach its own threads.
        __threadfence_block();
        __syncthreads();
        return true;
    }
    if (threadIdx.x == 0) {
        __threadfence();
        const uint32_t prev = atomicAdd(&done[item], 1u);
        last_block = prev == blocks_per_item - 1 ? 1u : 0u;
    }
    __syncthreads();
    const bool last = last_block != 0;
    if (last)
        __threadfence();
    return last;
}

// Writes the block's winner; the last block of the item to finish (agent-scope fence and
// counter, zeroed by option_terms_kernel before the scan) reduces the item's winners and
// writes its result, so no separate reduction kernel is launched.
__device__ __forceinline__ void block_finish(uint32_t L, uint64_t x, uint32_t item,
                                             uint32_t sub, uint32_t blocks_per_item,
                                             Winner *winners, const FinishArgs &fa)
{
    __shared__ uint32_t last_block;
    block_min_store(L, x, &winners[(uint64_t)item * blocks_per_item + sub]);
    if (blocks_per_item == 1) {
        // The block is the whole item: no agent-scope fence (an L2 write-back across XCDs) or
        // counter; its winner only needs to reach its own first wave.
        __threadfence_block();
        __syncthreads();
        if (threadIdx.x < 64)
            finish_item(fa, item, 1, winners);
        return;
    }
    if (threadIdx.x == 0) {
        __threadfence();
        const uint32_t prev = atomicAdd(&fa.done[item], 1u);
        last_block = prev == blocks_per_item - 1 ? 1u : 0u;
    }
    __syncthreads();
    if (last_block && threadIdx.x < 64) {
        __threadfence();
        finish_item(fa, item, blocks_per_item, winners);
    }
}

// Workgroups are dispatched to the 8 XCDs round-robin; renumber them so that consecutive
// logical blocks (the blocks of one item, which read the same few-KiB option table) share an
// XCD and its L2.  A bijection on [0, nblocks).
__device__ __forceinline__ uint32_t xcd_logical_block(uint32_t b, uint32_t nblocks)
{
    const uint32_t per = nblocks >> 3;
    if (b >= (per << 3))
        return b;
    return (b & 7u) * per + (b >> 3);
}

__device__ __forceinline__ uint32_t query_value(const uint32_t *arr, uint32_t single, uint32_t i)
{
    return arr ? arr[i] : single;
}

}  // namespace
}  // namespace alp
