// Device helpers shared by the gfx950 kernels: wave and block minima of (L, x), the end-of-item
// reduction of block winners with result decoding, and block renumbering across XCDs.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "alp_internal.h"

namespace alp {
namespace {

__device__ __forceinline__ bool lex_less(uint32_t aL, uint64_t ax, uint32_t bL, uint64_t bx)
{
    return aL < bL || (aL == bL && ax < bx);
}

// Cross-lane reductions by DPP moves (no LDS round trip per step); every lane of the wave must
// be active.  dpp_mov returns, in each lane of the rows selected by ROWMASK, the value of the
// lane that CTRL names; other rows keep `old`.
template <int CTRL, int ROWMASK = 0xF>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t old, uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, CTRL, ROWMASK, 0xF, false);
}

// The six steps of a wave reduction; lane 63 ends with the whole wave's value.  Quad swaps
// (lane ^ 1, lane ^ 2), the row's half mirror and mirror (every lane then holds its 16-lane
// row's value), lane 15 of each row into rows 1 and 3, lane 31 into rows 2 and 3.
template <class Step>
__device__ __forceinline__ void wave_reduce_steps(Step step)
{
    step(std::integral_constant<int, 0xB1>{}, std::integral_constant<int, 0xF>{});
    step(std::integral_constant<int, 0x4E>{}, std::integral_constant<int, 0xF>{});
    step(std::integral_constant<int, 0x141>{}, std::integral_constant<int, 0xF>{});
    step(std::integral_constant<int, 0x140>{}, std::integral_constant<int, 0xF>{});
    step(std::integral_constant<int, 0x142>{}, std::integral_constant<int, 0xA>{});
    step(std::integral_constant<int, 0x143>{}, std::integral_constant<int, 0xC>{});
}

__device__ __forceinline__ uint32_t lane63(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_readlane((int)v, 63);
}

// Wave-wide lexicographic minimum of (L, x); every lane ends with the result (wave-uniform).
__device__ __forceinline__ void wave_min(uint32_t &L, uint64_t &x)
{
    uint32_t xl = (uint32_t)x, xh = (uint32_t)(x >> 32);
    wave_reduce_steps([&](auto c, auto m) {
        constexpr int C = decltype(c)::value, RM = decltype(m)::value;
        const uint32_t oL = dpp_mov<C, RM>(L, L);
        const uint32_t ol = dpp_mov<C, RM>(xl, xl), oh = dpp_mov<C, RM>(xh, xh);
        const bool take = lex_less(oL, ((uint64_t)oh << 32) | ol, L, ((uint64_t)xh << 32) | xl);
        L = take ? oL : L;
        xl = take ? ol : xl;
        xh = take ? oh : xh;
    });
    L = lane63(L);
    x = ((uint64_t)lane63(xh) << 32) | lane63(xl);
}

// Wave-wide minima, returned as wave-uniform values.
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v)
{
    wave_reduce_steps([&](auto c, auto m) {
        constexpr int C = decltype(c)::value, RM = decltype(m)::value;
        const uint32_t o = dpp_mov<C, RM>(v, v);
        v = o < v ? o : v;
    });
    return lane63(v);
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v)
{
    wave_reduce_steps([&](auto c, auto m) {
        constexpr int C = decltype(c)::value, RM = decltype(m)::value;
        const uint32_t o = dpp_mov<C, RM>(v, v);
        v = o > v ? o : v;
    });
    return lane63(v);
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v)
{
    uint32_t l = (uint32_t)v, h = (uint32_t)(v >> 32);
    wave_reduce_steps([&](auto c, auto m) {
        constexpr int C = decltype(c)::value, RM = decltype(m)::value;
        const uint32_t ol = dpp_mov<C, RM>(l, l), oh = dpp_mov<C, RM>(h, h);
        const bool take = oh < h || (oh == h && ol < l);
        l = take ? ol : l;
        h = take ? oh : h;
    });
    return ((uint64_t)lane63(h) << 32) | lane63(l);
}

// Block-wide lexicographic minimum of (L, x); wave 0 ends with it (wave-uniform), other waves
// keep their wave's minimum.
__device__ __forceinline__ void block_min(uint32_t &L, uint64_t &x)
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
    if (wave == 0) {
        // Lane w reads wave w's minimum; one more wave reduction.
        L = lane < nw ? sL[lane] : kNoLatency;
        x = lane < nw ? sx[lane] : ~0ull;
        wave_min(L, x);
    }
}

__device__ __forceinline__ void store_winner(uint32_t L, uint64_t x, Winner *dst)
{
    Winner r;
    r.L = L;
    r.pad = 0;
    r.x = x;
    *dst = r;
}

// Block-wide minimum; thread 0 writes the block's winner.
__device__ __forceinline__ void block_min_store(uint32_t L, uint64_t x, Winner *dst)
{
    block_min(L, x);
    if (threadIdx.x == 0)
        store_winner(L, x, dst);
}

// Lexicographic (L, x) minimum of an item's block winners, by one wave; every lane gets it.
// Each lane issues up to eight winner loads before comparing any, so the item's winners arrive
// in one memory round trip per 512 blocks.
__device__ __forceinline__ void item_winner(uint32_t item, uint32_t blocks_per_item,
                                            const Winner *winners, uint32_t &L, uint64_t &x)
{
    const uint32_t lane = threadIdx.x & 63;
    const Winner *base = winners + (uint64_t)item * blocks_per_item;
    L = kNoLatency;
    x = ~0ull;
    for (uint32_t k0 = 0; k0 < blocks_per_item; k0 += 8 * 64) {
        uint32_t wL[8];
        uint64_t wx[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const uint32_t k = k0 + 64u * t + lane;
            wL[t] = kNoLatency;
            wx[t] = ~0ull;
            if (k < blocks_per_item) {
                const Winner w = base[k];
                wL[t] = w.L;
                wx[t] = w.x;
            }
        }
#pragma unroll
        for (int t = 0; t < 8; ++t)
            if (lex_less(wL[t], wx[t], L, x)) {
                L = wL[t];
                x = wx[t];
            }
    }
    wave_min(L, x);
}

// Option index of LLM `m` in candidate x: floor(x / O^(M-1-m)) mod O (LLM 0 most significant),
// with 32-bit division whenever x allows it.
__device__ __forceinline__ uint32_t candidate_digit(const SpaceDev &sp, uint64_t x, uint32_t m)
{
    uint64_t scale = 1;
    for (uint32_t k = m + 1; k < sp.M; ++k)
        scale *= sp.O;
    if ((x >> 32) == 0)
        return (scale >> 32) != 0 ? 0u : (uint32_t)x / (uint32_t)scale % sp.O;
    return (uint32_t)((x / scale) % sp.O);
}

// The result record of winner (L, x) written as the six 64-bit words of alp_result_t, by all
// lanes of one wave with the same (L, x): lane m < M holds LLM m's option o, its normalised
// throughput T (Eq. 2 term) and share units U; the wave takes T_w as their minimum (Eq. 2) and
// sums U, and lane 0 writes.
__device__ __forceinline__ void write_result_lanes(const SpaceDev &sp, uint32_t o, uint32_t T,
                                                   uint32_t U, uint32_t L, uint64_t x,
                                                   uint64_t *dst, uint32_t status_if_none,
                                                   uint32_t *signal = nullptr, uint32_t seq = 0)
{
    const uint32_t lane = threadIdx.x & 63;
    uint64_t tp = 0, fq = 0, rep = 0;
    if (L != kNoLatency && lane < sp.M) {
        const uint32_t ij = o / sp.D;
        tp = (uint64_t)sp.tp(ij / sp.n_fq) << (8 * lane);
        fq = (uint64_t)sp.fq(ij % sp.n_fq) << (8 * lane);
        rep = (uint64_t)((o % sp.D + 1) & 0xFFu) << (8 * lane);
    } else {
        T = 0xFFFFFFFFu;
        U = 0;
    }
    // Combine the (at most 8) LLM lanes: Eq. 2 minimum, unit sum, disjoint byte fields.
    // DPP steps within each 8-lane half row: lane ^ 1, lane ^ 2, then the half mirror (lane i
    // and 7 - i); every lane 0..7 ends with the total.
    auto combine = [&](auto c) {
        constexpr int C = decltype(c)::value;
        const uint32_t oT = dpp_mov<C>(T, T);
        T = oT < T ? oT : T;
        U += dpp_mov<C>(U, U);
        auto or64 = [](uint64_t v) {
            return v | ((uint64_t)dpp_mov<C>((uint32_t)(v >> 32), (uint32_t)(v >> 32)) << 32) |
                   dpp_mov<C>((uint32_t)v, (uint32_t)v);
        };
        tp = or64(tp);
        fq = or64(fq);
        rep = or64(rep);
    };
    static_assert(ALP_MAX_LLMS <= 8, "the combine covers one 8-lane half row");
    combine(std::integral_constant<int, 0xB1>{});
    combine(std::integral_constant<int, 0x4E>{});
    combine(std::integral_constant<int, 0x141>{});
    if (lane != 0)
        return;
    const bool none = L == kNoLatency;
    dst[0] = none ? ALP_NO_INDEX : x;
    dst[1] = none ? 0 : (uint64_t)L | ((uint64_t)T << 32);
    dst[2] = none ? (uint64_t)status_if_none << 32 : (uint64_t)U | ((uint64_t)ALP_OK << 32);
    dst[3] = none ? 0 : tp;
    dst[4] = none ? 0 : fq;
    dst[5] = none ? 0 : rep;
    if (signal)
        __hip_atomic_store(signal, seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

// The result record of winner (L, x), with the per-LLM choices decoded from x and T and U read
// from the item's per-option records E (lane m loads LLM m's: one memory round trip for all).
__device__ __forceinline__ void write_result(const SpaceDev &sp, const uint2 *E, uint32_t L,
                                             uint64_t x, uint64_t *dst,
                                             uint32_t status_if_none = ALP_INFEASIBLE,
                                             uint32_t *signal = nullptr, uint32_t seq = 0)
{
    const uint32_t lane = threadIdx.x & 63;
    uint32_t o = 0, T = 0xFFFFFFFFu, U = 0;
    if (L != kNoLatency && lane < sp.M) {
        o = candidate_digit(sp, x, lane);
        const uint2 e = E[(uint64_t)lane * sp.O + o];
        T = e.x;
        U = e.y & 0xFFFFu;
    }
    write_result_lanes(sp, o, T, U, L, x, dst, status_if_none, signal, seq);
}

// Result record of one item whose winner is (L, x), by one wave.  E: the item's per-option
// records, or nullptr for their copy in fa.ext.
__device__ __forceinline__ void write_item_result(const FinishArgs &fa, uint32_t item, uint32_t L,
                                                  uint64_t x, const uint2 *E = nullptr)
{
    const bool rejected = fa.invalid && fa.invalid[item];
    if (!E)
        E = fa.ext + (uint64_t)item * fa.sp.M * fa.sp.O;
    write_result(fa.sp, E, rejected ? kNoLatency : L, x,
                 reinterpret_cast<uint64_t *>(fa.out + item),
                 rejected ? (uint32_t)ALP_EINVAL : (uint32_t)ALP_INFEASIBLE, fa.signal, fa.seq);
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
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");   // the winner, before the count
        const uint32_t prev = atomicAdd(&done[item], 1u);
        last_block = prev == blocks_per_item - 1 ? 1u : 0u;
    }
    __syncthreads();
    const bool last = last_block != 0;
    if (last)
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");   // every block's winner
    return last;
}

// Per-option records of one item the finishing block stages in LDS (M * O at most this many).
constexpr uint32_t kFinishStage = 2048;

// The block's winner and the item's completion: the last block of the item to finish reduces
// the item's winners and writes its result, so no separate reduction kernel is launched.
// Publishing a winner takes an agent-scope release (an L2 write-back), so a block first takes
// the atomic minimum of the item's best latency: if an earlier block already reached a smaller
// latency, this block cannot hold the item's winner and only counts itself (its slot keeps the
// "no candidate" the option-term kernel wrote).  Blocks at or below the minimum so far store
// their winner and release it before counting; later relaxed counts continue that release
// sequence, so the last block's acquire sees every stored winner.  The counter, the minimum and
// the slots are reset by option_terms_kernel before each scan.
//
// `hint`: the item's best latency as read earlier in this launch (kNoLatency if not read); the
// minimum only falls, so a block above the hint skips the atomic minimum too (a plain load
// does not queue at the atomic unit behind the other blocks' updates).  `held` false (uniform
// over the block) says that no wave holds a candidate at or below the hint: the block skips its
// reduction and only counts itself.
__device__ __forceinline__ void block_finish(uint32_t L, uint64_t x, uint32_t item,
                                             uint32_t sub, uint32_t blocks_per_item,
                                             Winner *winners, const FinishArgs &fa,
                                             uint32_t hint = kNoLatency, bool held = true)
{
    __shared__ uint32_t last_block;
    if (blocks_per_item == 1) {
        // The block is the whole item: its minimum, held by wave 0, is the item's winner (no
        // fence, counter or winner slot).
        block_min(L, x);
        if (threadIdx.x < 64)
            write_item_result(fa, item, L, x);
        return;
    }
    if (held)
        block_min(L, x);
    if (threadIdx.x == 0) {
        if (held && L != kNoLatency && L <= hint && L <= atomicMin(&fa.best[item], L)) {
            store_winner(L, x, &winners[(uint64_t)item * blocks_per_item + sub]);
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        }
        const uint32_t prev = atomicAdd(&fa.done[item], 1u);
        last_block = prev == blocks_per_item - 1 ? 1u : 0u;
    }
    __syncthreads();
    if (!last_block)
        return;
    // The item's per-option records (written by the previous kernel) are staged in LDS by the
    // other waves while wave 0 loads the winners, so the result's records cost no second
    // memory round trip.
    __shared__ uint2 s_ext[kFinishStage];
    const uint32_t nE = fa.sp.M * fa.sp.O;
    const bool staged = nE <= kFinishStage && blockDim.x > 64;
    if (staged && threadIdx.x >= 64) {
        const uint2 *E = fa.ext + (uint64_t)item * nE;
        for (uint32_t k = threadIdx.x - 64; k < nE; k += blockDim.x - 64)
            s_ext[k] = E[k];
    }
    uint32_t Lw = kNoLatency;
    uint64_t xw = ~0ull;
    if (threadIdx.x < 64) {
        // Acquire: every stored winner is visible (an invalidate; no write-back).
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        item_winner(item, blocks_per_item, winners, Lw, xw);
    }
    __syncthreads();
    if (threadIdx.x < 64)
        write_item_result(fa, item, Lw, xw, staged ? s_ext : nullptr);
}

// ALP terms of option o of LLM m of instance `inst` at target rate lambda (Eq. 1 and Eq. 2
// terms, the memory fit of Section 5 step 1):
//   ok     the (tp, share) pair is deployable and W * Q <= tp * q * H (weights sharded over tp fit
//          the share q / Q of one GPU's memory);
//   tau    floor(1000 d T / n), d replicas of saturation throughput T = rate[K-1], saturated at
//          2^32 - 1 (Eq. 2);
//   thr    the per-replica load r = ceil(lambda n / (1000 d)) does not exceed T;
//   c      floor(ell(r) n / p), ell the profile latency at r: lat[0] up to rate[0], linear between
//          points, rounded down (Eq. 1; 0 unless thr);
//   u      tp * q * d share units.
struct OptionTerm {
    uint32_t c, u, tau;
    bool ok, thr;
};

// A reciprocal of d (0 < d < 2^31) in double precision biased low: (1 - e) / d with
// 0.85 * 2^-B < e < 1.15 * 2^-B.  The single-precision hardware reciprocal (within 1 ulp, so a
// relative error below 2^-22 with the rounding of d to a float) starts S Newton steps; a step
// squares the relative error (below 2^-44 after one, 2^-88 after two) and rounds once (2^-53),
// and the last step forms its residual against 1 - 2^-B instead of 1, which subtracts 2^-B.
// The bounds hold for (S, B) = (1, 40) and (2, 50).
template <int S, int B>
__device__ __forceinline__ double recip_low(uint32_t d)
{
    static_assert((S == 1 && B == 40) || (S == 2 && B == 50), "bounds stated for these");
    constexpr double kOneLow = 1.0 - 1.0 / (double)(1ull << B);
    const double D = (double)d;
    double y = (double)__builtin_amdgcn_rcpf((float)d);
    if constexpr (S == 2)
        y = fma(y, fma(-D, y, 1.0), y);
    return fma(y, fma(-D, y, kOneLow), y);
}

// floor(x / d) for 0 < d <= 2^31 and a quotient below 2^32 - 1, given x as a double xf (exact
// or rounded once) and modulo 2^32 (x_lo), and inv = recip_low<1, 40>(d) (or <2, 50>).  The
// estimate xf * inv is below x / d (the bias outweighs the roundings of x and of the product,
// 2^-53 each) by less than 2^-7 (1.15 * 2^-40 + 2^-52 of a quotient below 2^32), so its integer
// part q is the quotient or one less; the remainder x - q d then lies in [0, 2 d), exact modulo
// 2^32, and one comparison with d decides.  Outside the domain the result is some value,
// without undefined behaviour (the estimate is clamped before its conversion).
__device__ __forceinline__ uint32_t udiv_low(double xf, uint32_t x_lo, uint32_t d, double inv)
{
    const uint32_t q = (uint32_t)fmin(xf * inv, 4294967295.0);
    return q + (x_lo - q * d >= d ? 1u : 0u);
}

// An LLM's inputs to its option terms: n and p (milli) with their reciprocals.
struct LlmInputs {
    double inv_n;              // recip_low<2, 50>(n): tau's quotient reaches 2^45
    double inv_p;              // recip_low<1, 40>(p)
    uint32_t n, p;
};

__device__ __forceinline__ LlmInputs llm_inputs(uint32_t n, uint32_t p)
{
    return LlmInputs{recip_low<2, 50>(n), recip_low<1, 40>(p), n, p};
}

// Whether an (LLM, tp, share) curve's options are deployable: the pair is allowed and the
// weights sharded over tp fit the share q / Q of one GPU (W * Q <= tp * q * H).
__device__ __forceinline__ bool deployable(const SpaceDev &sp, uint64_t H, bool allowed,
                                           uint64_t W, uint32_t tpq)
{
    return allowed && W * sp.Q <= (uint64_t)tpq * H;
}

// A profile curve in device memory: rate and lat, K points each.  The point count below r is
// taken over ALP_MAX_POINTS reads at indices clamped to K - 1 (a clamped read repeats the last
// rate, which is not below r), so that all reads are in flight together with no test between.
struct CurveK {
    const uint32_t *rate, *lat;
    uint32_t K;
    __device__ __forceinline__ uint32_t last_rate() const { return rate[K - 1]; }
    __device__ __forceinline__ uint32_t points_below(uint32_t r) const
    {
        uint32_t k = 0;
#pragma unroll
        for (uint32_t q = 0; q < ALP_MAX_POINTS; ++q)
            k += rate[q < K ? q : K - 1] < r ? 1u : 0u;
        return k;
    }
};

// A profile curve in LDS: rate padded to ALP_MAX_POINTS points with its last value (16-byte
// aligned, read as four vectors), lat with K points.  Rates and r are below 2^31, so rate - r
// has its top bit set exactly when rate < r; the count adds those bits.
struct CurveLds {
    const uint32_t *rate, *lat;
    uint32_t K;
    __device__ __forceinline__ uint32_t last_rate() const { return rate[K - 1]; }
    __device__ __forceinline__ uint32_t points_below(uint32_t r) const
    {
        const uint4 *r4 = reinterpret_cast<const uint4 *>(rate);
        uint32_t k = 0;
#pragma unroll
        for (uint32_t q = 0; q < ALP_MAX_POINTS / 4; ++q) {
            const uint4 v = r4[q];
            k += ((v.x - r) >> 31) + ((v.y - r) >> 31) + ((v.z - r) >> 31) + ((v.w - r) >> 31);
        }
        return k;
    }
};

// The terms of an option with d replicas of its LLM, from the LLM's profile curve for the
// option's (tp, share) pair, whether that curve is deployable, tpq = tp * q, the LLM's inputs,
// the target lambda and inv_dd = recip_low<1, 40>(1000 d).  Every quotient is one udiv_low:
//   * tau < 2^45 with the <2, 50> reciprocal of n (an estimate below the quotient by less than
//     1.3 * 2^-50 * 2^45 < 2^-4): an estimate at or above 2^32 saturates, below it is the
//     quotient or one less, and a quotient of 2^32 saturates too;
//   * thr is lambda n <= 1000 d T (for an integer T, ceil(y) <= T iff y <= T), a product test;
//     with thr, r <= T < 2^31 and lambda n + 1000 d - 1 < 2^46 is an exact double;
//   * ell < 2^31 lies between two latencies;
//   * c of a deployable option is below 2^32 - 1 by the bound alp_load_profiles checks (every
//     latency term of a deployable option at most the instance's latency bound), and the
//     record of an undeployable option ignores c.
// Lanes without thr compute r, ell and c from out-of-range values and drop them.
template <class Curve>
__device__ __forceinline__ OptionTerm option_term_core(uint32_t d, const Curve &cv,
                                                       bool deployable, uint32_t tpq,
                                                       const LlmInputs &l, uint32_t lambda,
                                                       double inv_dd)
{
    OptionTerm t;
    t.ok = deployable;
    t.u = tpq * d;
    const uint32_t dd = 1000u * d;
    const uint32_t T = cv.last_rate();
    const uint64_t dT = (uint64_t)dd * T;
    const double n_f = (double)l.n;
    const double tau_est = ((double)dd * (double)T) * l.inv_n;      // dT exact in a double
    const uint32_t tq = (uint32_t)fmin(tau_est, 4294967295.0);
    const bool tau_up = (uint32_t)dT - tq * l.n >= l.n && tq != 0xFFFFFFFFu;
    t.tau = tau_est >= 4294967296.0 ? 0xFFFFFFFFu : tq + (tau_up ? 1u : 0u);
    const uint64_t load = (uint64_t)lambda * l.n;
    t.thr = load <= dT;
    const uint32_t r = udiv_low(fma((double)lambda, n_f, (double)(dd - 1)),
                                (uint32_t)load + dd - 1, dd, inv_dd);
    // ell, the latency at r: linear between the points (r0, l0) and (r1, l1) of the segment
    // holding r, taken at rc = max(r, r0) and rounded down; k counts the points below r (rates
    // ascend strictly, r <= rate[K-1]).  k = 0 (r at or below rate[0]) evaluates the first
    // segment at r0, giving lat[0]; a one-point curve (r0 = r1) takes a unit-width segment from
    // r0, again lat[0].
    const uint32_t k = cv.points_below(r);
    const uint32_t k1 = k > 1 ? k : 1u;
    const uint32_t i1 = k1 < cv.K ? k1 : cv.K - 1, i0 = k1 - 1;
    const uint32_t r0 = cv.rate[i0], r1 = cv.rate[i1];
    const uint32_t l0 = cv.lat[i0], l1 = cv.lat[i1];
    const uint32_t w = r1 > r0 ? r1 - r0 : 1u;
    const uint32_t rc = r > r0 ? r : r0;
    const uint64_t num = (uint64_t)l0 * (r0 + w - rc) + (uint64_t)l1 * (rc - r0);
    const uint32_t ell = udiv_low((double)num, (uint32_t)num, w, recip_low<1, 40>(w));
    const uint32_t c = udiv_low((double)ell * n_f, ell * l.n, l.p, l.inv_p);
    t.c = t.thr ? c : 0u;
    return t;
}

__device__ __forceinline__ OptionTerm option_term(const SpaceDev &sp, const TablesDev &tb,
                                                  uint32_t inst, uint32_t m, uint32_t o,
                                                  uint32_t lambda)
{
    const uint32_t ij = div_by(o, sp.mul_D), d = o - ij * sp.D + 1;
    const uint32_t i = ij / sp.n_fq, j = ij - i * sp.n_fq;
    const uint64_t lm = (uint64_t)inst * sp.M + m;
    const uint64_t tab = (lm * sp.n_tp + i) * sp.n_fq + j;
    const uint32_t tpq = sp.tp(i) * sp.fq(j);
    const CurveK cv{tb.rate + tab * sp.K, tb.lat + tab * sp.K, sp.K};
    return option_term_core(d, cv, deployable(sp, tb.H, tb.allowed[tab] != 0, tb.W[lm], tpq),
                            tpq, llm_inputs(tb.n[lm], tb.p[lm]), lambda,
                            recip_low<1, 40>(1000u * d));
}

// The item's profile inputs a one-launch block keeps in LDS: every (LLM, tp, share) curve's
// rate (padded, as CurveLds reads it), lat and deployability, tp * q of every (tp, share) pair,
// each LLM's inputs and the reciprocals of 1000 d.
struct FusedLds {
    const uint32_t *rate;
    const uint32_t *lat;
    const uint8_t *deploy;
    const uint32_t *tpq;
    const LlmInputs *llm;
    const double *inv_dd;      // [d - 1]
    const uint2 *ext;          // every option's (tau, share units), written by the prologue
    __device__ __forceinline__ OptionTerm term(const SpaceDev &sp, uint32_t m, uint32_t o,
                                               uint32_t lambda) const
    {
        const uint32_t ij = div_by(o, sp.mul_D), d = o - ij * sp.D + 1;
        const uint32_t c = m * (sp.n_tp * sp.n_fq) + ij;
        const CurveLds cv{rate + c * ALP_MAX_POINTS, lat + c * sp.K, sp.K};
        return option_term_core(d, cv, deploy[c] != 0, tpq[ij], llm[m], lambda, inv_dd[d - 1]);
    }
};

// Result record of a one-launch item whose winner is (L, x), by one wave: lane m reads LLM m's
// option terms of the winner from the block's LDS.  A rejected query gets ALP_EINVAL.
__device__ __forceinline__ void write_fused_result(const FinishArgs &fa, const FusedLds &lds,
                                                   bool rejected, uint32_t L, uint64_t x,
                                                   uint32_t item)
{
    const SpaceDev &sp = fa.sp;
    const uint32_t lane = threadIdx.x & 63;
    if (rejected)
        L = kNoLatency;
    uint32_t o = 0, T = 0xFFFFFFFFu, U = 0;
    if (L != kNoLatency && lane < sp.M) {
        o = candidate_digit(sp, x, lane);
        const uint2 e = lds.ext[lane * sp.O + o];
        T = e.x;
        U = e.y;
    }
    write_result_lanes(sp, o, T, U, L, x, reinterpret_cast<uint64_t *>(fa.out + item),
                       rejected ? (uint32_t)ALP_EINVAL : (uint32_t)ALP_INFEASIBLE, fa.signal,
                       fa.seq);
}

// End of a one-launch block: the block's lowest (L, x) (x < 2^32) joins the item's word by an
// atomic maximum of ~(L << 32 | x), performed (returned) before the block counts itself.  Blocks
// count in groups of kFusedGroup (sub / kFusedGroup); the last block of a group counts the group
// in the item's counter (an item of one group counts its blocks there directly), and the block
// completing the last group reads the item's lowest candidate from the word, resets the words
// and writes the result.  `hint` and `held` as in block_finish.
__device__ __forceinline__ void block_finish_fused(uint32_t L, uint64_t x, uint32_t item,
                                                   uint32_t sub, uint32_t blocks_per_item,
                                                   const FinishArgs &fa, const FusedArgs &fz,
                                                   const FusedLds &lds, bool rejected,
                                                   uint32_t hint, bool held)
{
    __shared__ uint32_t last_block;
    __shared__ unsigned long long s_word;
    if (blocks_per_item == 1) {
        block_min(L, x);
        if (threadIdx.x < 64)
            write_fused_result(fa, lds, rejected, L, x, item);
        return;
    }
    if (held)
        block_min(L, x);
    if (threadIdx.x == 0) {
        if (held && L != kNoLatency && L <= hint) {
            (void)atomicMax(&fz.best[item], ~(((unsigned long long)L << 32) | x));
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        }
        const uint32_t groups = (blocks_per_item + kFusedGroup - 1) / kFusedGroup;
        const uint32_t g = sub / kFusedGroup;
        const uint32_t in_group = g + 1 < groups ? kFusedGroup : blocks_per_item - g * kFusedGroup;
        uint32_t *gd = fz.group_done + (uint64_t)item * groups + g;
        last_block = 0;
        // One group: the blocks count in the item's counter directly (one atomic fewer on the
        // way to the result).
        if (groups == 1 || atomicAdd(gd, 1u) == in_group - 1) {
            if (groups > 1)
                (void)atomicExch(gd, 0u);          // the group's count, 0 for the next launch
            if (atomicAdd(&fz.done[item], 1u) == (groups > 1 ? groups : blocks_per_item) - 1) {
                s_word = atomicExch(&fz.best[item], 0ull);
                (void)atomicExch(&fz.done[item], 0u);
                last_block = 1;
            }
        }
    }
    __syncthreads();
    if (!last_block || threadIdx.x >= 64)
        return;
    const unsigned long long w = ~s_word;
    const uint32_t Lw = s_word ? (uint32_t)(w >> 32) : kNoLatency;
    write_fused_result(fa, lds, rejected, Lw, (uint32_t)w, item);
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

// Item i's query (instance, capacity, target): the three reads under one test, in flight
// together (a test per read would wait for each before the next).
__device__ __forceinline__ void load_query(const QueryDev &q, uint32_t i, uint32_t &inst,
                                           uint32_t &cap, uint32_t &lambda)
{
    if (q.inst) {
        inst = q.inst[i];
        cap = q.capacity[i];
        lambda = q.lambda[i];
    } else {
        inst = q.inst1;
        cap = q.cap1;
        lambda = q.lambda1;
    }
}

}  // namespace
}  // namespace alp
