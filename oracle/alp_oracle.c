/*
 * alp_oracle.c -- ORACLE.  Test infrastructure only: the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark load this library; the GPU library never includes, links
 * or calls anything here, and nothing here is shared with it.
 *
 * A plain, slow, single-threaded statement of the Aggregate LLM Pipeline (ALP) allocation
 * search of "Scepsy" (arXiv 2604.15186):
 *   - per LLM m and per-LLM option (tp, GPU share q, replicas d), the workflow-level latency
 *     contribution L_m(lambda * n_m / d) * n_m / p_m of Eq. 1 (Section 4, step 4 and step 5,
 *     replicas divide the per-replica arrival rate) and the workflow-normalised maximum
 *     throughput d * T_m / n_m of Eq. 2 (throughput scales linearly with replicas, Section 4,
 *     step 3);
 *   - per candidate allocation (one option per LLM), L_w = sum of the contributions (Eq. 1),
 *     T_w = minimum of the normalised throughputs (Eq. 2), and the feasibility conditions:
 *     every LLM's option deployable and its weights fit in its GPU share (Section 5, step 1,
 *     minimum fractions that hold the parameters), the target rate is sustained (T_w >= lambda,
 *     Section 3: the lowest latency that still meets the workflow's target rate), and the GPU
 *     budget is respected;
 *   - the search result: the feasible candidate of lowest L_w, ties broken by lowest index;
 *   - the paper's own pruned search over GPU fractions (Section 5, steps 1-3), and the split of
 *     a GPU pool over several workflows (Section 5, scheduling multiple workflows).
 *
 * Fixed-point readings (the paper computes in reals):
 *   rates in milli-requests/s, latencies in microseconds, n_m and p_m in milli-units;
 *   the per-replica LLM rate is rounded up, the interpolated latency, the latency contribution
 *   and the normalised throughput are rounded down; between profiled points latency is linear
 *   in the rate, below the first point it is flat, above the last (saturation) point the option
 *   cannot sustain the load.  GPU shares are counted in units of 1/Q GPU; the budget is
 *   sum(tp * q * d) <= Q * G.  The memory fit is W_m * Q <= tp * q * H (weights sharded over tp
 *   must fit the share q/Q of H bytes).
 *
 * Candidate numbering: option o = (i * |FQ| + j) * D + (d - 1) for tp = tp[i], q = fq[j]
 * (replicas vary fastest); candidate x = sum_m o_m * O^(M-1-m) (LLM 0 most significant).
 *
 * Arithmetic is 64-bit unsigned throughout; inputs are assumed to satisfy the documented ranges
 * (values below 2^31, weights and HBM size below 2^48), which keep every product below 2^63.
 */
#include <stdint.h>
#include <stddef.h>
#include <stdlib.h>

#define ORC_U64_NONE UINT64_MAX

typedef struct {
    uint32_t M;                 /* LLMs in the workflow */
    uint32_t n_tp;              /* number of tensor-parallel degrees */
    uint32_t n_fq;              /* number of GPU-share choices */
    uint32_t D;                 /* replica counts 1..D */
    uint32_t K;                 /* profile points per (tp, share) */
    uint32_t Q;                 /* share units per GPU */
    const uint32_t *tp;         /* [n_tp] */
    const uint32_t *fq;         /* [n_fq] share in units of 1/Q */
    const uint64_t *W;          /* [M] weight bytes */
    const uint32_t *n;          /* [M] invocations per workflow request (milli) */
    const uint32_t *p;          /* [M] request-level parallelism (milli) */
    const uint8_t *allowed;     /* [M][n_tp][n_fq] */
    const uint32_t *rate;       /* [M][n_tp][n_fq][K] milli-req/s, strictly ascending in k */
    const uint32_t *lat;        /* [M][n_tp][n_fq][K] microseconds */
    uint64_t H;                 /* HBM bytes per GPU */
} orc_instance;

typedef struct {
    uint32_t ok;        /* deployable and weights fit the share */
    uint32_t thr_ok;    /* the per-replica load does not exceed saturation */
    uint64_t c;         /* latency contribution, microseconds (valid iff thr_ok) */
    uint64_t u;         /* GPU share units used: tp * q * d */
    uint64_t tau;       /* workflow-normalised max throughput, milli-req/s */
} orc_term;

typedef struct {
    uint32_t flags;     /* bit0: every option ok; bit1: every option thr_ok; bit2: budget ok */
    uint64_t L;         /* L_w, defined iff bit0 and bit1, else ORC_U64_NONE */
    uint64_t T;         /* T_w, defined iff bit0, else 0 */
    uint64_t U;         /* sum of share units */
} orc_eval_out;

typedef struct {
    uint64_t best_x;        /* ORC_U64_NONE if no feasible candidate in the range */
    uint64_t best_L;
    uint64_t n_feasible;
    uint64_t sum_L;         /* sum of L_w over feasible candidates, modulo 2^64 */
} orc_argmin_out;

uint32_t orc_num_options(const orc_instance *s) { return s->n_tp * s->n_fq * s->D; }

/* Linear interpolation of one profiled latency curve at per-replica rate r (milli-req/s).
 * Called only when r <= rate[K-1].  Below the first point the curve is flat. */
static uint64_t orc_latency_at(const uint32_t *rate, const uint32_t *lat, uint32_t K, uint64_t r)
{
    if (r <= rate[0])
        return lat[0];
    for (uint32_t k = 1; k < K; ++k) {
        if (r <= rate[k]) {
            uint64_t r0 = rate[k - 1], r1 = rate[k];
            uint64_t num = (uint64_t)lat[k - 1] * (r1 - r) + (uint64_t)lat[k] * (r - r0);
            return num / (r1 - r0);
        }
    }
    return lat[K - 1]; /* not reached when r <= rate[K-1] */
}

/* Per-LLM, per-option ALP terms at workflow rate lambda (Eq. 1 and Eq. 2 terms; Section 4,
 * step 5, the load of one of d replicas is lambda * n_m / d; Section 5 step 1, memory bound). */
int orc_option_term(const orc_instance *s, uint32_t m, uint32_t o, uint32_t lambda, orc_term *out)
{
    if (m >= s->M || o >= orc_num_options(s))
        return -1;
    uint32_t d = o % s->D + 1;
    uint32_t ij = o / s->D;
    uint32_t j = ij % s->n_fq;
    uint32_t i = ij / s->n_fq;
    uint64_t tp = s->tp[i], q = s->fq[j];
    size_t tab = ((size_t)m * s->n_tp + i) * s->n_fq + j;
    const uint32_t *rate = s->rate + tab * s->K;
    const uint32_t *lat = s->lat + tab * s->K;
    uint64_t n = s->n[m], p = s->p[m];

    out->ok = s->allowed[tab] && (s->W[m] * (uint64_t)s->Q <= tp * q * s->H);
    uint64_t T = rate[s->K - 1];                                   /* saturation throughput */
    uint64_t tau = 1000ull * d * T / n;                            /* d * T_m / n_m (Eq. 2) */
    out->tau = tau > 0xFFFFFFFFull ? 0xFFFFFFFFull : tau;
    uint64_t r = ((uint64_t)lambda * n + 1000ull * d - 1) / (1000ull * d); /* ceil(lambda n / d) */
    out->thr_ok = (r <= T);
    out->c = 0;
    if (out->thr_ok) {
        uint64_t ell = orc_latency_at(rate, lat, s->K, r);        /* L_m at the replica's load */
        out->c = ell * n / p;                                      /* times n_m / p_m (Eq. 1) */
    }
    out->u = tp * q * d;
    return 0;
}

/* Evaluates one candidate from the raw tables (no precomputation). */
int orc_eval(const orc_instance *s, uint32_t G, uint32_t lambda, uint64_t x, orc_eval_out *out)
{
    uint32_t O = orc_num_options(s);
    uint32_t digit[16];
    if (s->M == 0 || s->M > 16)
        return -1;
    for (uint32_t k = 0; k < s->M; ++k) {                         /* LLM M-1 is the last digit */
        uint32_t m = s->M - 1 - k;
        digit[m] = (uint32_t)(x % O);
        x /= O;
    }
    if (x != 0)
        return -1;                                                 /* index out of range */
    int all_ok = 1, all_thr = 1;
    uint64_t L = 0, T = ORC_U64_NONE, U = 0;
    for (uint32_t m = 0; m < s->M; ++m) {
        orc_term t;
        orc_option_term(s, m, digit[m], lambda, &t);
        all_ok &= (int)t.ok;
        all_thr &= (int)t.thr_ok;
        L += t.c;
        if (t.tau < T)
            T = t.tau;
        U += t.u;
    }
    int budget_ok = U <= (uint64_t)s->Q * G;
    out->flags = (uint32_t)all_ok | ((uint32_t)all_thr << 1) | ((uint32_t)budget_ok << 2);
    out->L = (all_ok && all_thr) ? L : ORC_U64_NONE;
    out->T = all_ok ? T : 0;
    out->U = U;
    return 0;
}

int orc_eval_many(const orc_instance *s, uint32_t G, uint32_t lambda, const uint64_t *x,
                  uint64_t count, orc_eval_out *out)
{
    for (uint64_t i = 0; i < count; ++i)
        if (orc_eval(s, G, lambda, x[i], &out[i]) != 0)
            return -1;
    return 0;
}

/* Exhaustive argmin over candidates [lo, hi): the feasible candidate of lowest L_w, lowest
 * index among ties (scanning in increasing index order, only a strictly lower L_w replaces the
 * current best).  The per-option terms do not depend on the candidate, so they are computed
 * once per (m, o) and looked up; every candidate is then combined by Eq. 1, Eq. 2 and the
 * budget exactly as orc_eval does. */
int orc_argmin(const orc_instance *s, uint32_t G, uint32_t lambda, uint64_t lo, uint64_t hi,
               orc_term *scratch /* [M * O] */, orc_argmin_out *out)
{
    uint32_t O = orc_num_options(s);
    if (s->M == 0 || s->M > 16)
        return -1;
    for (uint32_t m = 0; m < s->M; ++m)
        for (uint32_t o = 0; o < O; ++o)
            orc_option_term(s, m, o, lambda, &scratch[(size_t)m * O + o]);
    uint64_t capacity = (uint64_t)s->Q * G;
    out->best_x = ORC_U64_NONE;
    out->best_L = ORC_U64_NONE;
    out->n_feasible = 0;
    out->sum_L = 0;
    for (uint64_t x = lo; x < hi; ++x) {
        uint64_t rest = x, L = 0, U = 0;
        int feasible = 1;
        for (uint32_t k = 0; k < s->M; ++k) {
            uint32_t m = s->M - 1 - k;
            const orc_term *t = &scratch[(size_t)m * O + rest % O];
            rest /= O;
            feasible &= (int)(t->ok && t->thr_ok);
            L += t->c;
            U += t->u;
        }
        if (!feasible || U > capacity)
            continue;
        out->n_feasible += 1;
        out->sum_L += L;
        if (L < out->best_L) {
            out->best_L = L;
            out->best_x = x;
        }
    }
    return 0;
}

/* Largest workflow throughput any candidate reaches within the budget, ignoring the target:
 * max over candidates with every option ok and sum(u) <= Q*G of T_w (Eq. 2); 0 if none.
 * Brute force over [lo, hi). */
int orc_tmax_brute(const orc_instance *s, uint32_t G, uint64_t lo, uint64_t hi, uint64_t *out)
{
    uint64_t best = 0;
    for (uint64_t x = lo; x < hi; ++x) {
        orc_eval_out e;
        if (orc_eval(s, G, 0, x, &e) != 0)
            return -1;
        if ((e.flags & 1u) && (e.flags & 4u) && e.T > best)
            best = e.T;
    }
    *out = best;
    return 0;
}

/* The same maximum by thresholds: T_w(x) >= t holds iff every LLM's option has normalised
 * throughput >= t, so t is reachable within the budget iff the cheapest such options of all
 * LLMs together fit in Q*G.  Reachability only shrinks as t grows, and the maximum is one of
 * the options' own throughputs; try each. */
int orc_tmax_threshold(const orc_instance *s, uint32_t G, orc_term *scratch /* [M * O] */,
                       uint64_t *out)
{
    uint32_t O = orc_num_options(s);
    for (uint32_t m = 0; m < s->M; ++m)
        for (uint32_t o = 0; o < O; ++o)
            orc_option_term(s, m, o, 0, &scratch[(size_t)m * O + o]);
    uint64_t capacity = (uint64_t)s->Q * G, best = 0;
    for (size_t a = 0; a < (size_t)s->M * O; ++a) {
        if (!scratch[a].ok)
            continue;
        uint64_t t = scratch[a].tau;
        if (t <= best)
            continue;
        uint64_t need = 0;
        int reachable = 1;
        for (uint32_t m = 0; m < s->M && reachable; ++m) {
            uint64_t cheapest = ORC_U64_NONE;
            for (uint32_t o = 0; o < O; ++o) {
                const orc_term *e = &scratch[(size_t)m * O + o];
                if (e->ok && e->tau >= t && e->u < cheapest)
                    cheapest = e->u;
            }
            if (cheapest == ORC_U64_NONE)
                reachable = 0;
            else
                need += cheapest;
        }
        if (reachable && need <= capacity)
            best = t;
    }
    *out = best;
    return 0;
}

/* ---------------------------------------------------------------------------------------------
 * Several workflows sharing a GPU pool (Section 5, scheduling of several workflows): every
 * workflow w receives a whole number of GPUs g_w, sum g_w <= G, and its own search at budget g_w
 * gives its latency L[w][g_w] (ORC_U64_NONE when infeasible).  The per-workflow utilities are
 * combined by egalitarian welfare (policy 0: minimise the largest latency; ties by the smaller
 * latency sum) or by social welfare (policy 1: minimise the latency sum); remaining ties go to
 * the lexicographically smallest budget vector (g_0 first).
 *
 * Brute force: every budget vector in increasing lexicographic order, keeping a strictly better
 * one.  L is row-major [W][G+1].  Returns 0 with g[] filled, 1 if no split makes every
 * workflow feasible, -1 on bad arguments. */
int orc_allocate(uint32_t W, uint32_t G, const uint64_t *L, uint32_t policy, uint32_t *g_out,
                 uint64_t *max_out, uint64_t *sum_out)
{
    if (W == 0 || W > 16 || policy > 1)
        return -1;
    uint32_t g[16] = {0};
    int found = 0;
    uint64_t best_max = 0, best_sum = 0;
    for (;;) {
        uint32_t used = 0;
        int ok = 1;
        uint64_t mx = 0, sum = 0;
        for (uint32_t w = 0; w < W; ++w) {
            used += g[w];
            uint64_t l = L[(size_t)w * (G + 1) + g[w]];
            if (l == ORC_U64_NONE) {
                ok = 0;
                break;
            }
            if (l > mx)
                mx = l;
            sum += l;
        }
        if (ok && used <= G) {
            int better;
            if (!found)
                better = 1;
            else if (policy == 0)
                better = mx < best_max || (mx == best_max && sum < best_sum);
            else
                better = sum < best_sum;
            if (better) {
                found = 1;
                best_max = mx;
                best_sum = sum;
                for (uint32_t w = 0; w < W; ++w)
                    g_out[w] = g[w];
            }
        }
        /* next vector: the last workflow's budget varies fastest */
        int w = (int)W - 1;
        while (w >= 0 && g[w] == G) {
            g[w] = 0;
            --w;
        }
        if (w < 0)
            break;
        ++g[w];
    }
    if (!found)
        return 1;
    *max_out = best_max;
    *sum_out = best_sum;
    return 0;
}

/* ---------------------------------------------------------------------------------------------
 * The paper's own pruned search (Section 5, steps 1-3).  It looks at a subset of the candidates
 * and so need not reach the exhaustive optimum.  Read as follows.
 *
 *  1. Enumerate GPU fractions: LLM m receives f_m units of 1/Q GPU, sum f_m = Q*G.
 *     ORC_PRUNE_ORDER: the LLMs are ordered by profiled latency ratio -- ref_m, the contribution
 *     lat * n_m / p_m at the smallest TP degree, the largest share and the first profiled point,
 *     largest first, ties by LLM index -- and no LLM receives more units than the one before it.
 *     ORC_PRUNE_MIN: each LLM receives at least the units that hold its weights,
 *     lo_m = max(1, ceil(W_m * Q / H)), and at most Q*G minus the lower bounds of the LLMs after
 *     it in the order.  Without the flags the order is still used for packing, lo = 0 and the
 *     upper bound is Q*G.
 *  2. Pack the fractions contiguously in that order: the k-th LLM occupies units [a_k, a_k + f)
 *     of the Q*G units laid out GPU after GPU.
 *  3. Resolve parallelism: option (tp, q, d) is admissible for an LLM iff tp * q * d = f (the
 *     fraction is used exactly, every rank with the same share) and d replicas of tp ranks of q
 *     units each, the ranks of one replica on distinct GPUs, fit the LLM's packed GPUs.
 *
 * The result is the feasible admissible candidate of lowest L_w, ties to the lowest index.
 * ------------------------------------------------------------------------------------------- */

#define ORC_PRUNE_ORDER 1u
#define ORC_PRUNE_MIN 2u

typedef struct {
    uint64_t best_x;    /* ORC_U64_NONE if no admissible candidate is feasible */
    uint64_t best_L;
    uint64_t vectors;   /* fraction vectors enumerated in step 1 */
    uint64_t unpruned;  /* C(Q*G + M - 1, M - 1): every fraction vector, saturating */
} orc_pruned_out;

/* Does an LLM holding units [a, a + f) fit d replicas of tp ranks of q units, the ranks of a
 * replica on distinct GPUs?  GPU g, holding h_g of the LLM's units, takes at most floor(h_g/q)
 * ranks and at most one rank of each replica, so at most min(floor(h_g/q), d).  The sum of these
 * reaching tp * d is also enough: list the ranks GPU by GPU and deal them to the replicas in
 * turn; no GPU contributes more than d consecutive ranks, so no replica gets two on one GPU. */
int orc_fits(uint32_t Q, uint64_t a, uint64_t f, uint64_t tp, uint64_t q, uint64_t d)
{
    uint64_t ranks = 0;
    if (Q == 0 || q == 0)
        return 0;
    for (uint64_t g = a / Q; g * Q < a + f; ++g) {
        uint64_t from = g * Q > a ? g * Q : a;
        uint64_t to = (g + 1) * Q < a + f ? (g + 1) * Q : a + f;
        uint64_t c = (to - from) / q;
        ranks += c < d ? c : d;
    }
    return ranks >= tp * d;
}

uint64_t orc_binomial(uint64_t n, uint64_t k)
{
    if (k > n)
        return 0;
    unsigned __int128 c = 1;
    for (uint64_t i = 1; i <= k; ++i) {
        c = c * (n - k + i) / i;        /* exact: c is C(n - k + i, i) after this step */
        if (c > ORC_U64_NONE)
            return ORC_U64_NONE;
    }
    return (uint64_t)c;
}

typedef struct {
    const orc_instance *s;
    const orc_term *terms;     /* [M][O], NULL when only counting */
    uint32_t M, Q;
    uint32_t order[16];        /* LLM at each position */
    uint64_t lo[16], hi[16];   /* bounds per position */
    uint64_t f[16];            /* fraction per position */
    int ordered;
    uint64_t vectors, best_x, best_L;
} orc_enum;

/* Steps 2 and 3 for one fraction vector.  With the fractions fixed, the admissible options of
 * each LLM do not depend on the others' choices and L_w is a sum, so the lowest (L_w, x) over the
 * product of the admissible sets takes, per LLM, the smallest contribution and, among equal
 * ones, the lowest option (x orders LLM 0 first). */
static void orc_visit(orc_enum *e)
{
    e->vectors += 1;
    if (!e->terms)
        return;
    const orc_instance *s = e->s;
    uint32_t O = orc_num_options(s);
    uint64_t start[16], size[16], a = 0;
    for (uint32_t k = 0; k < e->M; ++k) {
        start[e->order[k]] = a;
        size[e->order[k]] = e->f[k];
        a += e->f[k];
    }
    uint64_t L = 0, x = 0;
    for (uint32_t m = 0; m < e->M; ++m) {
        uint64_t best_c = ORC_U64_NONE;
        uint32_t best_o = 0;
        for (uint32_t o = 0; o < O; ++o) {
            const orc_term *t = &e->terms[(size_t)m * O + o];
            if (!t->ok || !t->thr_ok || t->u != size[m])
                continue;
            uint32_t d = o % s->D + 1, ij = o / s->D;
            uint64_t tp = s->tp[ij / s->n_fq], q = s->fq[ij % s->n_fq];
            if (!orc_fits(e->Q, start[m], size[m], tp, q, d))
                continue;
            if (t->c < best_c) {
                best_c = t->c;
                best_o = o;
            }
        }
        if (best_c == ORC_U64_NONE)
            return;
        L += best_c;
        x = x * O + best_o;
    }
    if (L < e->best_L || (L == e->best_L && x < e->best_x)) {
        e->best_L = L;
        e->best_x = x;
    }
}

/* Step 1: every fraction vector, position by position; the last position takes the rest. */
static void orc_enum_from(orc_enum *e, uint32_t k, uint64_t remaining)
{
    uint64_t lo = e->lo[k], hi = e->hi[k];
    if (e->ordered && k > 0 && e->f[k - 1] < hi)
        hi = e->f[k - 1];
    if (k + 1 == e->M) {
        if (remaining >= lo && remaining <= hi) {
            e->f[k] = remaining;
            orc_visit(e);
        }
        return;
    }
    for (uint64_t v = lo; v <= hi && v <= remaining; ++v) {
        e->f[k] = v;
        orc_enum_from(e, k + 1, remaining - v);
    }
}

/* Bounds per position; returns 0 when the lower bounds alone exceed the total (no vector). */
static int orc_enum_bounds(orc_enum *e, uint64_t total, const uint64_t *lo_pos)
{
    uint64_t after = 0;
    for (uint32_t k = e->M; k-- > 0;) {
        if (after + lo_pos[k] > total)
            return 0;
        e->lo[k] = lo_pos[k];
        e->hi[k] = total - after;
        after += lo_pos[k];
    }
    return 1;
}

/* Number of fraction vectors of step 1 for M positions, total units, lower bounds per position
 * (upper bounds as in step 1), with or without the ordering. */
uint64_t orc_count_fractions(uint32_t M, uint64_t total, const uint64_t *lo_pos, int ordered)
{
    orc_enum e = {0};
    if (M == 0 || M > 16)
        return 0;
    e.M = M;
    e.ordered = ordered;
    if (orc_enum_bounds(&e, total, lo_pos))
        orc_enum_from(&e, 0, total);
    return e.vectors;
}

int orc_pruned(const orc_instance *s, uint32_t G, uint32_t lambda, uint32_t flags,
               orc_term *scratch /* [M * O] */, orc_pruned_out *out)
{
    uint32_t O = orc_num_options(s);
    if (s->M == 0 || s->M > 16 || flags > 3u)
        return -1;
    for (uint32_t m = 0; m < s->M; ++m)
        for (uint32_t o = 0; o < O; ++o)
            orc_option_term(s, m, o, lambda, &scratch[(size_t)m * O + o]);
    orc_enum e = {0};
    e.s = s;
    e.terms = scratch;
    e.M = s->M;
    e.Q = s->Q;
    e.ordered = (flags & ORC_PRUNE_ORDER) != 0;
    e.best_x = ORC_U64_NONE;
    e.best_L = ORC_U64_NONE;
    /* latency ratios: contribution at tp[0], the largest share, the first profiled point */
    uint64_t ref[16];
    for (uint32_t m = 0; m < s->M; ++m) {
        size_t tab = ((size_t)m * s->n_tp + 0) * s->n_fq + (s->n_fq - 1);
        ref[m] = (uint64_t)s->lat[tab * s->K] * s->n[m] / s->p[m];
        e.order[m] = m;
    }
    for (uint32_t a = 1; a < s->M; ++a) {                  /* insertion sort: ref desc, m asc */
        uint32_t v = e.order[a], b = a;
        while (b > 0 && ref[e.order[b - 1]] < ref[v]) {
            e.order[b] = e.order[b - 1];
            --b;
        }
        e.order[b] = v;
    }
    uint64_t total = (uint64_t)s->Q * G, lo_pos[16];
    for (uint32_t k = 0; k < s->M; ++k) {
        uint32_t m = e.order[k];
        uint64_t need = (s->W[m] * (uint64_t)s->Q + s->H - 1) / s->H;
        lo_pos[k] = (flags & ORC_PRUNE_MIN) ? (need > 1 ? need : 1) : 0;
    }
    if (orc_enum_bounds(&e, total, lo_pos))
        orc_enum_from(&e, 0, total);
    out->best_x = e.best_x;
    out->best_L = e.best_x == ORC_U64_NONE ? ORC_U64_NONE : e.best_L;
    out->vectors = e.vectors;
    out->unpruned = orc_binomial(total + s->M - 1, s->M - 1);
    return 0;
}

/* ---------------------------------------------------------------------------------------------
 * Workflow statistics from execution traces (Section 4, step 2).  A trace is one workflow
 * request: the LLM-level calls it made, each with its LLM, start and end timestamp (half-open
 * [start, end), microseconds).  For every LLM m:
 *   n_m = average number of calls per workflow request = calls_m / traces;
 *   p_m = average request-level parallelism, from overlapping timestamps: the calls' total
 *         duration divided by the time during which at least one call of m runs, summed over
 *         the traces.  (Then n_m * L_m / p_m of Eq. 1 is the time per request during which m is
 *         active.)  Three concurrent beams give p = 3.
 * Both in thousandths, rounded down; p = 1000 when m has calls but no measurable time, and
 * n = p = 0 when m has no calls.
 * ------------------------------------------------------------------------------------------- */

typedef struct {
    uint32_t n_milli, p_milli;
    uint64_t calls, busy_us, active_us;
} orc_stats;

static int orc_cmp_u64(const void *a, const void *b)
{
    uint64_t x = *(const uint64_t *)a, y = *(const uint64_t *)b;
    return x < y ? -1 : x > y;
}

/* offsets[R + 1] delimit each trace's calls.  scratch: 2 * (longest trace) uint64.  Returns 0, or
 * -1 for a malformed input (offsets not ascending from 0, llm >= M, end < start). */
int orc_trace_stats(uint32_t M, uint32_t R, const uint64_t *offsets, const uint32_t *llm,
                    const uint64_t *start, const uint64_t *end, uint64_t *scratch,
                    orc_stats *out)
{
    if (M == 0 || M > 16 || R == 0 || offsets[0] != 0)
        return -1;
    for (uint32_t m = 0; m < M; ++m) {
        out[m].calls = out[m].busy_us = out[m].active_us = 0;
    }
    for (uint32_t r = 0; r < R; ++r) {
        uint64_t lo = offsets[r], hi = offsets[r + 1];
        if (hi < lo)
            return -1;
        for (uint32_t m = 0; m < M; ++m) {
            /* this LLM's intervals in the trace, sorted by start (end as the tie-breaker) */
            uint64_t k = 0;
            for (uint64_t i = lo; i < hi; ++i) {
                if (llm[i] >= M || end[i] < start[i])
                    return -1;
                if (llm[i] != m)
                    continue;
                scratch[2 * k] = start[i];
                scratch[2 * k + 1] = end[i];
                ++k;
            }
            qsort(scratch, k, 2 * sizeof(uint64_t), orc_cmp_u64);
            /* sweep: the union grows by the part of each interval beyond the furthest end so far */
            uint64_t reach = 0, active = 0, busy = 0;
            for (uint64_t j = 0; j < k; ++j) {
                uint64_t s = scratch[2 * j], e = scratch[2 * j + 1];
                busy += e - s;
                uint64_t from = (j == 0 || s > reach) ? s : reach;
                if (e > from)
                    active += e - from;
                if (j == 0 || e > reach)
                    reach = e;
            }
            out[m].calls += k;
            out[m].busy_us += busy;
            out[m].active_us += active;
        }
    }
    for (uint32_t m = 0; m < M; ++m) {
        out[m].n_milli = (uint32_t)(out[m].calls * 1000u / R);
        if (out[m].calls == 0)
            out[m].p_milli = 0;
        else if (out[m].active_us == 0)
            out[m].p_milli = 1000;
        else
            out[m].p_milli = (uint32_t)(out[m].busy_us * 1000u / out[m].active_us);
    }
    return 0;
}

/* ---------------------------------------------------------------------------------------------
 * Placement of an allocation on the GPUs of a budget (Section 6, hierarchical placement).  The
 * G GPUs form nodes of 8 (the last node may hold fewer), every node one all-to-all xGMI domain,
 * each GPU Q share units.  LLM m's allocation is d_m replicas of tp_m ranks of q_m units; the
 * ranks of a replica sit on tp_m distinct GPUs of one node.
 *
 * The paper's most-constrained-first heuristic, read as follows.  Replicas are placed one by
 * one: tensor-parallel replicas (tp > 1) before the others, larger replicas (tp * q units)
 * first within each kind, ties by LLM index.  A tensor-parallel replica goes to tp GPUs of one
 * node that each have q units free: in each node the GPUs with room are ordered by free units
 * (then index), every run of tp consecutive ones is a candidate, scored by its imbalance (most
 * minus least free units), then by the capacity of its domain (the node's free units; the
 * least preferred, which keeps large domains for later), then by its own free units, then by
 * node and position.  A single-GPU replica goes onto
 * an already occupied GPU with room first, the one with the fewest free units (then the lowest
 * index); failing that onto an empty GPU of the node with the fewest free units in total (then
 * the lowest node), the lowest such GPU.  The allocation is placed if every replica finds room.
 * ------------------------------------------------------------------------------------------- */

#define ORC_NODE_GPUS 8u
#define ORC_PLACE_MAX_GPUS 64u
#define ORC_PLACE_MAX_REPLICAS 128u
#define ORC_PLACE_NONE 0xFFFFu

typedef struct {
    uint32_t placed;          /* 1 if every replica was placed */
    uint32_t replicas;        /* replicas placed */
    uint32_t gpus_used, nodes_used;
    uint16_t slot[ORC_PLACE_MAX_REPLICAS];  /* per replica (LLM-major): node << 8 | GPU mask */
} orc_placement;

static uint32_t orc_replica_order(uint32_t M, const uint32_t *tp, const uint32_t *q,
                                  const uint32_t *d, uint32_t *order)
{
    uint32_t k = 0;
    for (uint32_t m = 0; m < M; ++m)
        if (d[m] > 0)
            order[k++] = m;
    for (uint32_t a = 1; a < k; ++a) {          /* insertion sort by (tp == 1, -tp*q, m) */
        uint32_t v = order[a], b = a;
        for (; b > 0; --b) {
            uint32_t u = order[b - 1];
            int u_tp1 = tp[u] == 1, v_tp1 = tp[v] == 1;
            uint64_t us = (uint64_t)tp[u] * q[u], vs = (uint64_t)tp[v] * q[v];
            int v_first = v_tp1 < u_tp1 || (v_tp1 == u_tp1 && (vs > us || (vs == us && v < u)));
            if (!v_first)
                break;
            order[b] = u;
        }
        order[b] = v;
    }
    return k;
}

/* Places one replica; returns 0 and the slot, or -1 if there is no room. */
static int orc_place_one(uint32_t Q, uint32_t G, uint32_t *free_u, uint32_t tp, uint32_t q,
                         uint16_t *slot)
{
    uint32_t nodes = (G + ORC_NODE_GPUS - 1) / ORC_NODE_GPUS;
    if (tp > 1) {
        int found = 0;
        uint32_t b_imb = 0, b_dom = 0, b_cap = 0, b_node = 0, b_mask = 0;
        for (uint32_t n = 0; n < nodes; ++n) {
            uint32_t E[ORC_NODE_GPUS], k = 0, dom = 0;
            for (uint32_t g = n * ORC_NODE_GPUS; g < G && g < (n + 1) * ORC_NODE_GPUS; ++g) {
                dom += free_u[g];
                if (free_u[g] >= q)
                    E[k++] = g;
            }
            for (uint32_t a = 1; a < k; ++a) {  /* by (free, index) */
                uint32_t v = E[a], b = a;
                while (b > 0 && (free_u[E[b - 1]] > free_u[v] ||
                                 (free_u[E[b - 1]] == free_u[v] && E[b - 1] > v))) {
                    E[b] = E[b - 1];
                    --b;
                }
                E[b] = v;
            }
            for (uint32_t i = 0; i + tp <= k; ++i) {
                uint32_t imb = free_u[E[i + tp - 1]] - free_u[E[i]], cap = 0, mask = 0;
                for (uint32_t j = i; j < i + tp; ++j) {
                    cap += free_u[E[j]];
                    mask |= 1u << (E[j] - n * ORC_NODE_GPUS);
                }
                if (!found || imb < b_imb || (imb == b_imb && dom < b_dom) ||
                    (imb == b_imb && dom == b_dom && cap < b_cap)) {
                    found = 1;
                    b_imb = imb;
                    b_dom = dom;
                    b_cap = cap;
                    b_node = n;
                    b_mask = mask;
                }
            }
        }
        if (!found)
            return -1;
        for (uint32_t j = 0; j < ORC_NODE_GPUS; ++j)
            if (b_mask & (1u << j))
                free_u[b_node * ORC_NODE_GPUS + j] -= q;
        *slot = (uint16_t)(b_node << 8 | b_mask);
        return 0;
    }
    /* a single GPU: an occupied one with room (fewest free units), else an empty one */
    uint32_t best = G;
    for (uint32_t g = 0; g < G; ++g)
        if (free_u[g] < Q && free_u[g] >= q && (best == G || free_u[g] < free_u[best]))
            best = g;
    if (best == G) {
        uint64_t best_node_free = 0;
        for (uint32_t n = 0; n < nodes; ++n) {
            uint32_t empty = G;
            uint64_t node_free = 0;
            for (uint32_t g = n * ORC_NODE_GPUS; g < G && g < (n + 1) * ORC_NODE_GPUS; ++g) {
                node_free += free_u[g];
                if (free_u[g] == Q && q <= Q && empty == G)
                    empty = g;
            }
            if (empty != G && (best == G || node_free < best_node_free)) {
                best = empty;
                best_node_free = node_free;
            }
        }
    }
    if (best == G)
        return -1;
    free_u[best] -= q;
    *slot = (uint16_t)((best / ORC_NODE_GPUS) << 8 | 1u << (best % ORC_NODE_GPUS));
    return 0;
}

/* The heuristic.  tp, q, d per LLM (d = 0: the LLM has no replica).  Returns 0, or -1 for bad
 * arguments (G above 64, more than 128 replicas, tp above 8, q outside 1..Q). */
int orc_place(uint32_t Q, uint32_t G, uint32_t M, const uint32_t *tp, const uint32_t *q,
              const uint32_t *d, orc_placement *out)
{
    uint32_t free_u[ORC_PLACE_MAX_GPUS], order[16], total = 0;
    if (G > ORC_PLACE_MAX_GPUS || M == 0 || M > 16 || Q == 0)
        return -1;
    for (uint32_t m = 0; m < M; ++m) {
        if (d[m] && (tp[m] == 0 || tp[m] > ORC_NODE_GPUS || q[m] == 0 || q[m] > Q))
            return -1;
        total += d[m];
    }
    if (total > ORC_PLACE_MAX_REPLICAS)
        return -1;
    for (uint32_t g = 0; g < G; ++g)
        free_u[g] = Q;
    for (uint32_t i = 0; i < ORC_PLACE_MAX_REPLICAS; ++i)
        out->slot[i] = ORC_PLACE_NONE;
    uint32_t first[16], acc = 0;                 /* slot index of each LLM's first replica */
    for (uint32_t m = 0; m < M; ++m) {
        first[m] = acc;
        acc += d[m];
    }
    uint32_t k = orc_replica_order(M, tp, q, d, order);
    out->placed = 1;
    out->replicas = 0;
    for (uint32_t a = 0; a < k && out->placed; ++a) {
        uint32_t m = order[a];
        for (uint32_t r = 0; r < d[m]; ++r) {
            if (orc_place_one(Q, G, free_u, tp[m], q[m], &out->slot[first[m] + r]) != 0) {
                out->placed = 0;
                break;
            }
            out->replicas += 1;
        }
    }
    out->gpus_used = out->nodes_used = 0;
    for (uint32_t n = 0; n * ORC_NODE_GPUS < G; ++n) {
        uint32_t used = 0;
        for (uint32_t g = n * ORC_NODE_GPUS; g < G && g < (n + 1) * ORC_NODE_GPUS; ++g)
            used += free_u[g] < Q;
        out->gpus_used += used;
        out->nodes_used += used > 0;
    }
    return 0;
}

/* Exact feasibility by backtracking (small cases only): every replica tries every node and
 * every set of tp GPUs with room.  Returns 1 if some placement exists, 0 if none, -1 for bad
 * arguments. */
static int orc_place_rec(uint32_t Q, uint32_t G, uint32_t *free_u, uint32_t n_rep,
                         const uint32_t *rtp, const uint32_t *rq, uint32_t i, uint32_t from)
{
    if (i == n_rep)
        return 1;
    uint32_t nodes = (G + ORC_NODE_GPUS - 1) / ORC_NODE_GPUS;
    /* choices are numbered node * 256 + mask; replicas of the same kind are interchangeable,
     * so a replica identical to the previous one takes a choice no smaller than its choice */
    for (uint32_t n = 0; n < nodes; ++n) {
        uint32_t lo = n * ORC_NODE_GPUS, hi = lo + ORC_NODE_GPUS < G ? lo + ORC_NODE_GPUS : G;
        for (uint32_t mask = 1; mask < (1u << (hi - lo)); ++mask) {
            uint32_t choice = n * 256 + mask;
            if (choice < from || (uint32_t)__builtin_popcount(mask) != rtp[i])
                continue;
            int ok = 1;
            for (uint32_t j = 0; j < hi - lo && ok; ++j)
                if ((mask >> j & 1u) && free_u[lo + j] < rq[i])
                    ok = 0;
            if (!ok)
                continue;
            for (uint32_t j = 0; j < hi - lo; ++j)
                if (mask >> j & 1u)
                    free_u[lo + j] -= rq[i];
            uint32_t next_from = 0;
            if (i + 1 < n_rep && rtp[i + 1] == rtp[i] && rq[i + 1] == rq[i])
                next_from = choice;
            int r = orc_place_rec(Q, G, free_u, n_rep, rtp, rq, i + 1, next_from);
            for (uint32_t j = 0; j < hi - lo; ++j)
                if (mask >> j & 1u)
                    free_u[lo + j] += rq[i];
            if (r)
                return 1;
        }
    }
    return 0;
}

int orc_place_exact(uint32_t Q, uint32_t G, uint32_t M, const uint32_t *tp, const uint32_t *q,
                    const uint32_t *d)
{
    uint32_t free_u[ORC_PLACE_MAX_GPUS], rtp[ORC_PLACE_MAX_REPLICAS], rq[ORC_PLACE_MAX_REPLICAS];
    uint32_t n = 0;
    if (G > ORC_PLACE_MAX_GPUS || M == 0 || M > 16)
        return -1;
    for (uint32_t m = 0; m < M; ++m)
        for (uint32_t r = 0; r < d[m]; ++r) {
            if (n == ORC_PLACE_MAX_REPLICAS || tp[m] == 0 || tp[m] > ORC_NODE_GPUS || q[m] > Q)
                return -1;
            rtp[n] = tp[m];
            rq[n] = q[m];
            ++n;
        }
    for (uint32_t g = 0; g < G; ++g)
        free_u[g] = Q;
    return orc_place_rec(Q, G, free_u, n, rtp, rq, 0, 0);
}
