/*
 * tas_oracle.c - plain, sequential CPU oracle of the serving simulation.
 *
 * TEST INFRASTRUCTURE ONLY (see tas_oracle.h). It is written for a reader who
 * checks it against the paper by eye: one request array, one candidate list
 * re-ranked from scratch every iteration, linear victim searches, no
 * incremental structures beyond keeping the previous order as the start of an
 * insertion sort (which sorts any input; the previous order only makes it fast).
 *
 * Paper passages followed (arXiv 2606.18431):
 *   Formulation / Notation          request (a_i, s_pre, s_dec); T_i = C_i - a_i
 *   Eq. boost_function              b_gamma(w) = (1/gamma) ln(1/(1-exp(-gamma w)))
 *   Phase 2 (UniBoost-Base)         Phi(i,t) = a_i - b(max(w_i, s_pre)), argmin
 *   Phase 2 preemption protocol     hysteresis: preempt only if better by delta
 *   Phase 3 (MemGuard), Eq. memguard_level  w_hat = k 2^floor(log2(max(w,k)/k)),
 *                                   dispatched => non-evictable until the next
 *                                   threshold
 *   Algorithm 1                     per iteration: keys for every active
 *                                   request, greedy batch fill under M and the
 *                                   KV capacity, victim selection + swap-out,
 *                                   ExecuteOneStep, UpdateStats
 *   Phase 4                         t_p = inf{t : Fbar(t) <= (100-p)/100}
 *   Phase 4 (gamma-Ada), Eq. gamma_estimator, Algorithm 2 UpdateGamma
 *                                   gamma_hat = (ln Fbar(t95) - ln Fbar(t99)) /
 *                                   (t99 - t95) over a window of recent
 *                                   end-to-end latencies, EMA, clip
 *
 * Where the paper is silent, the readings are (each is listed, with its
 * reason, in the design notes of the repository):
 *   - signal w = P + dec (prompt plus emitted tokens; monotone in both phases)
 *   - boost in microseconds: table[level] = round(tau * b_gamma(k 2^level))
 *   - ExecuteOneStep: dt = base + tok * sum(n) + floor(sum(kv + n) / div)
 *   - swap-out = recompute preemption: KV dropped, emitted tokens kept, the
 *     request re-prefills P + dec tokens when readmitted
 *   - victim = worst (key, idx) resident not already in this batch; voluntary
 *     victims must be evictable (MemGuard) and worse than the candidate by
 *     delta; when none exists a resident candidate forces out the worst other
 *     resident, or itself; a waiting candidate that does not fit closes
 *     admissions for the rest of the iteration
 *   - the iteration that completes the prefill emits the first token; times
 *     are iteration ends; arrivals join at the next iteration start
 *   - SRPT key = remaining computed tokens P + D - 1 - kv; FCFS key = a_i
 *
 * Comparison policies (paper: Table 1 and the baselines of the evaluation):
 *   SPF   shortest prompt first: key = P (static)
 *   SJF   shortest job first with perfect knowledge of the output length (the
 *         ranking LTR learns): key = D (static)
 *   LTR   SJF (LTR+): the SJF key plus LTR's starvation control by quantum
 *         promotion (baselines of the evaluation, item 2; Table 1, the LTR
 *         row). After every iteration each request that was a candidate and
 *         did not run adds one to its starvation count; one that ran resets
 *         it. At the threshold S (a setting) the request is promoted: it
 *         ranks before every unpromoted request, promoted requests in order
 *         of promotion (key = j - 2^42 for a promotion at the end of
 *         iteration j, ties by index), for a quantum of Q iterations in which
 *         it runs (Q a setting); then it returns to its SJF key with a count
 *         of zero. No MemGuard, no hysteresis.
 *   LAS   least attained service: key = P + dec, the same signal as the boost
 *         (grows with every emitted token)
 *   TRAIL SRPT with perfect knowledge plus the swap-prevention threshold: a
 *         resident that has emitted at least 0.6 D tokens is never a voluntary
 *         victim (5 dec >= 3 D)
 *   SARATHI decode-prioritized continuous batching with round-robin decodes
 *         and piggy-backed prefill chunks: a request in its prefill waits in
 *         arrival order (key = a); once it has emitted a token it is in the
 *         decode queue, ordered by the time of its latest token (the request
 *         served longest ago goes first), below every prefill key:
 *         key = t_last - 2^42. Waiting requests never preempt running ones:
 *         no voluntary victims, only the forced eviction of a resident that
 *         cannot grow (the worst other resident, i.e. the latest prefill or
 *         the most recently served decode, else itself)
 *
 * Phase ladder (paper: Phase 1 DistBoost; Algorithm 2 Signal):
 *   DIST  DistBoost: two queues. A request in its prefill (no token emitted
 *         yet) has the prefill priority a - b(P) (the boost table at the level
 *         of its prompt); once it has emitted its first token it is in the
 *         decode queue, ordered by the time it entered it (its first-token
 *         time), and every decode-queue request ranks before every prefill-
 *         queue request: the decode batch first, prefill chunks fill the rest.
 *         Key = t_first - 2^42 in decode, below every prefill key.
 *   signal 1 (BOOST): the phase-aware signal of Algorithm 2: the prompt length
 *         while in prefill, the decode tokens emitted after it (the level,
 *         the key and MemGuard's guard all use it)
 *   signal 2 (BOOST): prefix caching (paper: interaction with prefix/radix
 *         caching): with h expected cached prompt tokens the effective work is
 *         max(w, P - h), i.e. P - h + dec when cached tokens are not counted as
 *         processed; the engine itself is unchanged
 *
 * Adaptive gamma (Phase 4, gamma-Ada), for BOOST instances that ask for it:
 *   - the window holds the end-to-end latencies (TTLT, us, capped at 2^32-1)
 *     of the last W completed requests; requests that complete in the same
 *     iteration enter it in batch order
 *   - at the start of every iteration (Algorithm 1 calls UpdateGamma before
 *     the keys), once the window holds at least min_samples latencies:
 *       t95, t99 = nearest-rank percentiles of the window
 *       gamma_hat = (tau ln 5) / max(t99 - t95, eps)   (per token: the
 *           estimator is per microsecond and one token of boost is tau us;
 *           ln 5 = ln(0.05 / 0.01) from the tail-band definition)
 *       gamma = clip((1 - beta) gamma + beta gamma_hat, gamma_min, gamma_max)
 *   - the boost table in use is that of the nearest point of a log-spaced
 *     grid of G values from gamma_min to gamma_max (nearest in log scale,
 *     midpoints sqrt(g_j g_{j+1}) going up), so priorities stay integers
 *   - every floating-point step is one IEEE double operation, in this order
 */
#include "tas_oracle.h"

#include <math.h>
#include <pthread.h>
#include <stdlib.h>
#include <string.h>

enum { PENDING = 0, WAITING = 1, RESIDENT = 2, DONE = 3 };
enum { P_FCFS = 0, P_SRPT = 1, P_BOOST = 2, P_SPF = 3, P_SJF = 4, P_LAS = 5, P_TRAIL = 6,
       P_DIST = 7, P_SARATHI = 8, P_LTR = 9 };
#define P_LAST P_LTR
#define DECODE_QUEUE_OFFSET ((int64_t)1 << 42) /* decode-queue keys lie below every prefill key */
#define PROMOTED_OFFSET ((int64_t)1 << 42)     /* LTR+: promoted keys lie below every SJF key */

#define ADA_GRID_MAX 64
#define ADA_WINDOW_MAX 2048

typedef struct {
    int32_t on;
    double gamma0, beta, gmin, gmax, eps, num; /* num = tau ln 5 */
    int32_t W, nmin, G;
    double grid[ADA_GRID_MAX], bound[ADA_GRID_MAX];
    int64_t table[ADA_GRID_MAX][TOR_LEVELS];
} ada_t;

typedef struct {
    int32_t N;
    const int64_t *a;
    const int32_t *P, *D;
    int32_t policy, k, memguard;
    int64_t delta;
    const int64_t *bt;
    int32_t M, T, c, Kb, bs, base, tok, div;
    int64_t max_iters;
    const ada_t *ada; /* NULL: gamma fixed */
    int32_t signal;   /* BOOST: 0 = P + dec, 1 = Algorithm 2's phase-aware signal,
                         2 = P - h + dec (expected prefix-cache hits h) */
    const int32_t *H; /* expected cached prompt tokens per request, or NULL */
    int32_t ltr_s, ltr_q; /* LTR+: starvation threshold and quantum, iterations */
} inst_t;

typedef struct {
    int8_t st;
    int8_t in_batch;
    int32_t kv;    /* tokens whose KV is resident */
    int32_t dec;   /* tokens emitted so far */
    int32_t guard; /* MemGuard level at the latest dispatch */
    int64_t key;   /* priority key, frozen at iteration start */
    int64_t t_first, t_last, tbt_max;
    int64_t evicted_at; /* iteration in which it was last evicted, or -1 */
    int32_t starve;     /* LTR+: iterations not served (unpromoted), or quantum left */
    int8_t promoted;    /* LTR+ */
    int64_t promo_key;  /* LTR+: the key while promoted */
} req_t;

typedef struct {
    int64_t *it;
    int64_t it_cap, n_it;
    int32_t *b;
    int64_t b_cap, n_b;
    int64_t *ev;
    int64_t ev_cap, n_ev;
    int full;
} log_t;

/* ------------------------------------------------------------ boost table */

/* ln(1 - exp(-x)) for x > 0, evaluated accurately on both sides of ln 2
 * (Maechler 2012, "Accurately computing log(1 - exp(-|a|))"). */
static double log1mexp(double x) {
    return x <= 0.6931471805599453 ? log(-expm1(-x)) : log1p(-exp(-x));
}

int tas_oracle_boost_table(double gamma, int32_t k, double tau_us, int64_t *out) {
    if (!(gamma > 0.0) || k < 1 || !(tau_us > 0.0)) return TOR_EINVAL;
    const double cap = 4398046511104.0; /* 2^42 */
    for (int j = 0; j < TOR_LEVELS; j++) {
        double w = (double)k * ldexp(1.0, j); /* quantized signal k * 2^j */
        double b = -log1mexp(gamma * w) / gamma; /* b_gamma(w), tokens */
        double us = tau_us * b;
        out[j] = us >= cap ? (int64_t)cap : (int64_t)llround(us);
    }
    return 0;
}

/* ------------------------------------------------------------ helpers */

static int64_t blocks(int64_t tokens, int32_t bs) { return (tokens + bs - 1) / bs; }

/* MemGuard level: floor(log2(max(w,k)/k)), capped at the table's last entry.
 * floor(log2(x)) of the real ratio equals that of floor(x) because every
 * threshold 2^j is an integer. */
static int32_t level_of(int64_t w, int32_t k) {
    int64_t q = (w > k ? w : k) / k;
    int32_t L = 0;
    while (q >= 2) {
        q >>= 1;
        L++;
    }
    return L < TOR_LEVELS - 1 ? L : TOR_LEVELS - 1;
}

int32_t tas_oracle_level(int64_t w, int32_t k) { return level_of(w, k); }

/* The boost signal of request r: P + dec, or (signal 1) P during the prefill
 * and the decode tokens emitted after it, or (signal 2) P - h + dec. */
static int64_t signal_of(const inst_t *I, int32_t r, const req_t *q) {
    if (I->signal == 1) return q->dec == 0 ? I->P[r] : q->dec;
    if (I->signal == 2) return (int64_t)I->P[r] - I->H[r] + q->dec;
    return (int64_t)I->P[r] + q->dec;
}

static int64_t key_of(const inst_t *I, int32_t r, const req_t *q) {
    switch (I->policy) {
    case P_FCFS:
        return I->a[r];
    case P_SRPT:
    case P_TRAIL:
        return (int64_t)I->P[r] + I->D[r] - 1 - q->kv;
    case P_SPF:
        return I->P[r];
    case P_SJF:
        return I->D[r];
    case P_LAS:
        return (int64_t)I->P[r] + q->dec;
    case P_DIST:
        if (q->dec > 0) return q->t_first - DECODE_QUEUE_OFFSET; /* decode queue */
        return I->a[r] - I->bt[level_of(I->P[r], I->k)];         /* prefill queue */
    case P_SARATHI:
        if (q->dec > 0) return q->t_last - DECODE_QUEUE_OFFSET; /* round robin */
        return I->a[r];                                         /* arrival order */
    case P_LTR:
        return q->promoted ? q->promo_key : I->D[r];
    default:
        return I->a[r] - I->bt[level_of(signal_of(I, r, q), I->k)];
    }
}

/* (ka, ia) > (kb, ib) in lexicographic order */
static int lex_gt(int64_t ka, int32_t ia, int64_t kb, int32_t ib) {
    return ka > kb || (ka == kb && ia > ib);
}

static void evict(req_t *q, int64_t *U, int32_t bs, int64_t iter) {
    *U -= blocks(q->kv, bs);
    q->kv = 0;
    q->st = WAITING;
    q->evicted_at = iter;
}

/* ------------------------------------------------------------ gamma-Ada */

/* One instance's adaptive-gamma parameters from prm[10] = {on, gamma0, beta,
 * gamma_min, gamma_max, eps_us, window, min_samples, grid points, tau_us}:
 * the log-spaced grid g_j = gamma_min (gamma_max/gamma_min)^(j/(G-1)), the
 * midpoints sqrt(g_j g_{j+1}) between neighbours and the boost table of every
 * grid point. Returns 0 or TOR_EINVAL. */
static int ada_setup(ada_t *A, const double *prm, int32_t policy, int32_t k) {
    memset(A, 0, sizeof *A);
    if (prm[0] == 0.0) return 0;
    if (prm[0] != 1.0 || policy != P_BOOST) return TOR_EINVAL;
    A->on = 1;
    A->gamma0 = prm[1], A->beta = prm[2], A->gmin = prm[3], A->gmax = prm[4], A->eps = prm[5];
    const double tau = prm[9];
    if (!(prm[6] >= 1 && prm[6] <= ADA_WINDOW_MAX && prm[7] >= 1 && prm[7] <= prm[6] &&
          prm[8] >= 2 && prm[8] <= ADA_GRID_MAX))
        return TOR_EINVAL;
    A->W = (int32_t)prm[6], A->nmin = (int32_t)prm[7], A->G = (int32_t)prm[8];
    if (!(A->beta >= 0.0 && A->beta <= 1.0 && A->gmin > 0.0 && A->gmax > A->gmin &&
          isfinite(A->gmax) && A->gamma0 >= A->gmin && A->gamma0 <= A->gmax && A->eps > 0.0 &&
          isfinite(A->eps) && tau > 0.0 && isfinite(tau)))
        return TOR_EINVAL;
    A->num = tau * log(5.0);
    for (int32_t j = 0; j < A->G; j++)
        A->grid[j] = A->gmin * pow(A->gmax / A->gmin, (double)j / (double)(A->G - 1));
    for (int32_t j = 0; j + 1 < A->G; j++) A->bound[j] = sqrt(A->grid[j] * A->grid[j + 1]);
    for (int32_t j = 0; j < A->G; j++)
        if (tas_oracle_boost_table(A->grid[j], k, tau, A->table[j])) return TOR_EINVAL;
    return 0;
}

/* The grid point nearest to gamma in log scale (a midpoint goes up). */
static int32_t ada_cell(const ada_t *A, double gamma) {
    int32_t j = 0;
    while (j + 1 < A->G && gamma >= A->bound[j]) j++;
    return j;
}

int tas_oracle_ada_grid(const double *prm, int32_t k, double *grid, double *bound,
                        int64_t *tables) {
    ada_t *A = (ada_t *)malloc(sizeof *A);
    if (!A) return TOR_EINVAL;
    int rc = ada_setup(A, prm, P_BOOST, k);
    if (rc == 0 && A->on) {
        memcpy(grid, A->grid, sizeof(double) * (size_t)A->G);
        memcpy(bound, A->bound, sizeof(double) * (size_t)(A->G - 1));
        memcpy(tables, A->table, sizeof(int64_t) * TOR_LEVELS * (size_t)A->G);
    }
    free(A);
    return rc;
}

/* ------------------------------------------------------------ one instance */

static int simulate(const inst_t *I0, uint32_t *ttft, uint32_t *ttlt, uint32_t *tbtmax,
                    int64_t *cnt, double *gamma_out, int64_t *switch_out, log_t *lg) {
    inst_t J = *I0; /* J.bt follows the adaptive gamma */
    const inst_t *I = &J;
    const ada_t *A = I->ada && I->ada->on ? I->ada : NULL;
    const int32_t N = I->N;
    if (I->signal == 2 && !I->H) return TOR_EINVAL;
    if (I->policy == P_LTR && (I->ltr_s < 1 || I->ltr_q < 1)) return TOR_EINVAL;
    for (int32_t i = 0; i < N; i++) {
        if (I->P[i] < 1 || I->D[i] < 1 || I->a[i] < 0 || (i && I->a[i] < I->a[i - 1]))
            return TOR_EINVAL;
        if (I->H && (I->H[i] < 0 || I->H[i] >= I->P[i])) return TOR_EINVAL;
        if (blocks((int64_t)I->P[i] + I->D[i] - 1, I->bs) > I->Kb) return TOR_EINFEASIBLE;
    }
    req_t *R = (req_t *)calloc((size_t)N, sizeof *R);
    int32_t *act = (int32_t *)malloc(sizeof(int32_t) * (size_t)N);
    int32_t *bidx = (int32_t *)malloc(sizeof(int32_t) * (size_t)I->M);
    int32_t *bn = (int32_t *)malloc(sizeof(int32_t) * (size_t)I->M);
    uint32_t *win = A ? (uint32_t *)malloc(sizeof(uint32_t) * (size_t)A->W) : NULL;
    int status = 0;
    if (!R || !act || !bidx || !bn || (A && !win)) {
        status = TOR_EINVAL;
        goto out;
    }
    for (int32_t i = 0; i < N; i++) R[i].evicted_at = -1;

    int64_t t = 0, U = 0, iters = 0, reqiters = 0, tokens = 0, ev_vol = 0, ev_forced = 0;
    int64_t maxU = 0, idle = 0;
    int32_t next = 0, nact = 0;
    /* gamma-Ada state: gamma, its grid cell, the latency window */
    double gamma = A ? A->gamma0 : 0.0, ghat = 0.0;
    int32_t cell = A ? ada_cell(A, gamma) : -1, wn = 0, whead = 0, wnew = 0;
    int64_t switches = 0;
    if (A) J.bt = A->table[cell];

    for (;;) {
        /* O2 arrivals: a_i <= t joins the waiting set (idx order). */
        while (next < N && I->a[next] <= t) {
            R[next].st = WAITING;
            act[nact++] = next++;
        }
        /* O3 idle server: jump to the next arrival. */
        if (nact == 0) {
            if (next == N) break;
            idle += I->a[next] - t;
            t = I->a[next];
            continue;
        }
        /* Phase 4 UpdateGamma, before the keys of this iteration. */
        if (A && wn >= A->nmin) {
            if (wnew) { /* the window changed since the last estimate */
                uint32_t t95 = tas_oracle_percentile(win, wn, 95);
                uint32_t t99 = tas_oracle_percentile(win, wn, 99);
                double d = (double)(t99 - t95);
                if (d < A->eps) d = A->eps;
                ghat = A->num / d;
                wnew = 0;
            }
            double g = (1.0 - A->beta) * gamma + A->beta * ghat;
            if (g < A->gmin) g = A->gmin;
            if (g > A->gmax) g = A->gmax;
            gamma = g;
            int32_t c2 = ada_cell(A, gamma);
            if (c2 != cell) {
                cell = c2;
                switches++;
                J.bt = A->table[cell];
            }
        }
        /* O4/O5 keys of every active request, then rank by (key, idx). */
        for (int32_t j = 0; j < nact; j++) R[act[j]].key = key_of(I, act[j], &R[act[j]]);
        for (int32_t j = 1; j < nact; j++) {
            int32_t x = act[j];
            int64_t kx = R[x].key;
            int32_t m = j;
            while (m > 0 && lex_gt(R[act[m - 1]].key, act[m - 1], kx, x)) {
                act[m] = act[m - 1];
                m--;
            }
            act[m] = x;
        }

        /* O6 greedy batch formation in priority order. */
        int32_t nb = 0, closed = 0;
        int64_t used = 0;
        for (int32_t j = 0; j < nact; j++) {
            if (nb == I->M || used == I->T) break;
            int32_t r = act[j];
            req_t *q = &R[r];
            if (q->evicted_at == iters) continue;
            if (q->st == WAITING && closed) continue;
            int64_t need = (int64_t)I->P[r] + q->dec - q->kv;
            int64_t n = need;
            if (n > I->c) n = I->c;
            if (n > I->T - used) n = I->T - used;
            int64_t dU = blocks(q->kv + n, I->bs) - blocks(q->kv, I->bs);
            for (;;) {
                if (U + dU <= I->Kb) {
                    if (q->st == WAITING) { /* dispatch */
                        q->st = RESIDENT;
                        q->guard = level_of(signal_of(I, r, q), I->k);
                    }
                    q->in_batch = 1;
                    bidx[nb] = r;
                    bn[nb] = (int32_t)n;
                    nb++;
                    used += n;
                    U += dU;
                    break;
                }
                /* voluntary victim: worst eligible resident outside the batch */
                int32_t v = -1;
                for (int32_t m = 0; m < nact; m++) {
                    int32_t x = act[m];
                    const req_t *p = &R[x];
                    if (x == r || p->st != RESIDENT || p->in_batch) continue;
                    if (I->memguard && !(level_of(signal_of(I, x, p), I->k) > p->guard))
                        continue;
                    if (I->policy == P_TRAIL && 5 * (int64_t)p->dec >= 3 * (int64_t)I->D[x])
                        continue; /* past the swap-prevention threshold */
                    if (I->policy == P_SARATHI) continue; /* no preemption by priority */
                    if (!lex_gt(p->key - I->delta, x, q->key, r)) continue;
                    if (v < 0 || lex_gt(p->key, x, R[v].key, v)) v = x;
                }
                if (v >= 0) {
                    evict(&R[v], &U, I->bs, iters);
                    ev_vol++;
                    if (lg && lg->n_ev < lg->ev_cap) {
                        int64_t *e = lg->ev + 4 * lg->n_ev++;
                        e[0] = iters, e[1] = v, e[2] = 0, e[3] = r;
                    } else if (lg)
                        lg->full = 1;
                    continue;
                }
                if (q->st == RESIDENT) {
                    /* forced: worst other resident outside the batch, else r */
                    for (int32_t m = 0; m < nact; m++) {
                        int32_t x = act[m];
                        const req_t *p = &R[x];
                        if (x == r || p->st != RESIDENT || p->in_batch) continue;
                        if (v < 0 || lex_gt(p->key, x, R[v].key, v)) v = x;
                    }
                    int self = v < 0;
                    if (self) v = r;
                    evict(&R[v], &U, I->bs, iters);
                    ev_forced++;
                    if (lg && lg->n_ev < lg->ev_cap) {
                        int64_t *e = lg->ev + 4 * lg->n_ev++;
                        e[0] = iters, e[1] = v, e[2] = 1, e[3] = r;
                    } else if (lg)
                        lg->full = 1;
                    if (self) break;
                    continue;
                }
                closed = 1; /* a waiting request that does not fit */
                break;
            }
        }
        /* O7 */
        if (nb == 0) {
            status = TOR_ESTATE;
            goto out;
        }
        if (U > maxU) maxU = U;

        /* O8 cost of the step. */
        int64_t sum_n = 0, sum_ctx = 0;
        for (int32_t b = 0; b < nb; b++) {
            sum_n += bn[b];
            sum_ctx += (int64_t)R[bidx[b]].kv + bn[b];
        }
        int64_t dt = I->base + (int64_t)I->tok * sum_n + sum_ctx / I->div;
        int64_t t_end = t + dt;
        if (lg) {
            if (lg->n_it < lg->it_cap) {
                int32_t nw = 0, nr = 0;
                for (int32_t m = 0; m < nact; m++) {
                    nw += R[act[m]].st == WAITING;
                    nr += R[act[m]].st == RESIDENT;
                }
                int64_t *e = lg->it + 8 * lg->n_it++;
                e[0] = t, e[1] = dt, e[2] = nb, e[3] = U, e[4] = nw, e[5] = nr;
                e[6] = cell;
                memcpy(&e[7], &gamma, sizeof gamma);
            } else
                lg->full = 1;
            for (int32_t b = 0; b < nb; b++) {
                if (lg->n_b < lg->b_cap) {
                    lg->b[2 * lg->n_b] = bidx[b];
                    lg->b[2 * lg->n_b + 1] = bn[b];
                    lg->n_b++;
                } else
                    lg->full = 1;
            }
        }

        /* LTR+ starvation control: every candidate of this iteration that did
         * not run counts one more iteration of starvation and is promoted at
         * the threshold; one that ran resets its count, or spends one
         * iteration of its quantum. Effective from the next iteration's keys. */
        if (I->policy == P_LTR) {
            for (int32_t j = 0; j < nact; j++) {
                req_t *q = &R[act[j]];
                if (q->in_batch) {
                    if (!q->promoted) {
                        q->starve = 0;
                    } else if (--q->starve == 0) {
                        q->promoted = 0; /* the quantum is spent */
                    }
                } else if (!q->promoted && ++q->starve >= I->ltr_s) {
                    q->promoted = 1;
                    q->starve = I->ltr_q;
                    q->promo_key = (iters + 1) - PROMOTED_OFFSET;
                }
            }
        }

        /* O9 execute: advance KV, emit tokens, record latencies, complete. */
        for (int32_t b = 0; b < nb; b++) {
            int32_t r = bidx[b];
            req_t *q = &R[r];
            q->in_batch = 0;
            q->kv += bn[b];
            if (q->kv == I->P[r] + q->dec) {
                q->dec++;
                if (q->dec == 1)
                    q->t_first = t_end;
                else if (t_end - q->t_last > q->tbt_max)
                    q->tbt_max = t_end - q->t_last;
                q->t_last = t_end;
                if (q->dec == I->D[r]) {
                    q->st = DONE;
                    U -= blocks(q->kv, I->bs);
                    q->kv = 0;
                    if (A) { /* UpdateStats: the window keeps the last W latencies */
                        int64_t e2e = t_end - I->a[r];
                        win[whead] = e2e > 0xFFFFFFFFll ? 0xFFFFFFFFu : (uint32_t)e2e;
                        whead = (whead + 1) % A->W;
                        if (wn < A->W) wn++;
                        wnew = 1;
                    }
                }
            }
        }

        /* O10 advance the clock and the counters. */
        t = t_end;
        iters++;
        reqiters += nb;
        tokens += sum_n;
        if (iters > I->max_iters) {
            status = TOR_ELIVELOCK;
            goto out;
        }
        int32_t w = 0;
        for (int32_t j = 0; j < nact; j++)
            if (R[act[j]].st != DONE) act[w++] = act[j];
        nact = w;
    }

    /* O11 per-request outputs, relative to arrival. */
    for (int32_t i = 0; i < N; i++) {
        int64_t f = R[i].t_first - I->a[i], l = R[i].t_last - I->a[i], g = R[i].tbt_max;
        if (f > 0xFFFFFFFFll || l > 0xFFFFFFFFll || g > 0xFFFFFFFFll) {
            status = TOR_EOVERFLOW;
            goto out;
        }
        ttft[i] = (uint32_t)f;
        ttlt[i] = (uint32_t)l;
        tbtmax[i] = (uint32_t)g;
    }
    cnt[0] = iters, cnt[1] = reqiters, cnt[2] = tokens, cnt[3] = ev_vol;
    cnt[4] = ev_forced, cnt[5] = t, cnt[6] = maxU, cnt[7] = idle;
    if (gamma_out) *gamma_out = gamma;
    if (switch_out) *switch_out = switches;
out:
    free(win);
    free(R);
    free(act);
    free(bidx);
    free(bn);
    return status;
}

/* ------------------------------------------------------------ percentiles */

static int cmp_u32(const void *x, const void *y) {
    uint32_t a = *(const uint32_t *)x, b = *(const uint32_t *)y;
    return (a > b) - (a < b);
}

uint32_t tas_oracle_percentile(const uint32_t *v, int32_t n, int32_t q) {
    if (n <= 0) return 0;
    uint32_t *s = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)n);
    memcpy(s, v, sizeof(uint32_t) * (size_t)n);
    qsort(s, (size_t)n, sizeof(uint32_t), cmp_u32);
    int64_t rank = ((int64_t)q * n + 99) / 100; /* ceil(q n / 100) */
    if (rank < 1) rank = 1;
    uint32_t out = s[rank - 1];
    free(s);
    return out;
}

/* ------------------------------------------------------------ driver */

typedef struct {
    int32_t n_req, n_inst;
    const int64_t *arrival;
    const int32_t *prompt, *decode, *cached;
    const int32_t *trace, *policy, *k, *memguard;
    const int64_t *delta, *table;
    const int32_t *eng;
    int64_t max_iters;
    uint32_t *ttft, *ttlt, *tbtmax, *pct;
    int64_t *counters;
    int32_t *status;
    const double *ada; /* [n_inst*10] or NULL */
    const int32_t *signal; /* [n_inst] or NULL */
    const int32_t *ltr;    /* [n_inst*2] or NULL */
    double *gamma_out;
    int64_t *switch_out;
    int32_t next; /* work counter */
} job_t;

static void fill_inst(inst_t *I, const int32_t *eng, int32_t n_req, const int64_t *a,
                      const int32_t *P, const int32_t *D, int32_t policy, int32_t k,
                      int32_t memguard, int64_t delta, const int64_t *bt, int64_t max_iters) {
    I->N = n_req, I->a = a, I->P = P, I->D = D;
    I->policy = policy, I->k = k, I->memguard = memguard, I->delta = delta, I->bt = bt;
    I->M = eng[0], I->T = eng[1], I->c = eng[2], I->Kb = eng[3], I->bs = eng[4];
    I->base = eng[5], I->tok = eng[6], I->div = eng[7];
    I->max_iters = max_iters;
    I->ada = NULL;
    I->signal = 0;
    I->H = NULL;
    I->ltr_s = I->ltr_q = 0;
}

static void run_one(job_t *J, int32_t i) {
    int32_t tr = J->trace[i];
    size_t off = (size_t)tr * (size_t)J->n_req;
    inst_t I;
    fill_inst(&I, J->eng, J->n_req, J->arrival + off, J->prompt + off, J->decode + off,
              J->policy[i], J->k[i], J->memguard[i], J->delta[i], J->table + (size_t)i * 24,
              J->max_iters);
    size_t o = (size_t)i * (size_t)J->n_req;
    ada_t *A = NULL;
    int st = 0;
    if (J->signal) I.signal = J->signal[i];
    if (J->cached) I.H = J->cached + off;
    if (J->ltr) I.ltr_s = J->ltr[2 * (size_t)i], I.ltr_q = J->ltr[2 * (size_t)i + 1];
    if (J->ada && J->ada[(size_t)i * 10] != 0.0) {
        A = (ada_t *)malloc(sizeof *A);
        st = A ? ada_setup(A, J->ada + (size_t)i * 10, J->policy[i], J->k[i]) : TOR_EINVAL;
        I.ada = A;
    }
    if (st == 0)
        st = simulate(&I, J->ttft + o, J->ttlt + o, J->tbtmax + o, J->counters + (size_t)i * 8,
                      J->gamma_out ? J->gamma_out + i : NULL,
                      J->switch_out ? J->switch_out + i : NULL, NULL);
    free(A);
    J->status[i] = st;
    if (st == 0) {
        const uint32_t *m[3] = {J->ttft + o, J->ttlt + o, J->tbtmax + o};
        const int32_t qs[3] = {50, 90, 99};
        for (int a = 0; a < 3; a++)
            for (int b = 0; b < 3; b++)
                J->pct[(size_t)i * 9 + a * 3 + b] = tas_oracle_percentile(m[a], J->n_req, qs[b]);
    }
}

static void *worker(void *arg) {
    job_t *J = (job_t *)arg;
    for (;;) {
        int32_t i = __atomic_fetch_add(&J->next, 1, __ATOMIC_RELAXED);
        if (i >= J->n_inst) break;
        run_one(J, i);
    }
    return NULL;
}

int tas_oracle_run(int32_t n_traces, int32_t n_req, const int64_t *arrival,
                   const int32_t *prompt, const int32_t *decode, const int32_t *cached,
                   int32_t n_inst,
                   const int32_t *trace, const int32_t *policy, const int32_t *k,
                   const int32_t *memguard, const int64_t *delta, const int64_t *table,
                   const int32_t *eng, int64_t max_iters, uint32_t *ttft, uint32_t *ttlt,
                   uint32_t *tbtmax, int64_t *counters, uint32_t *pct, int32_t *status,
                   const double *ada, const int32_t *signal, const int32_t *ltr,
                   double *gamma_out, int64_t *switch_out, int32_t n_threads) {
    if (n_traces < 1 || n_req < 1 || n_inst < 0) return TOR_EINVAL;
    for (int32_t i = 0; i < n_inst; i++) {
        if (trace[i] < 0 || trace[i] >= n_traces || policy[i] < 0 || policy[i] > P_LAST ||
            k[i] < 1)
            return TOR_EINVAL;
        if (policy[i] == P_LTR && (!ltr || ltr[2 * i] < 1 || ltr[2 * i + 1] < 1))
            return TOR_EINVAL;
        if (signal && signal[i] != 0 &&
            (signal[i] < 1 || signal[i] > 2 || policy[i] != P_BOOST || (signal[i] == 2 && !cached)))
            return TOR_EINVAL;
    }
    if (eng[0] < 1 || eng[1] < 1 || eng[2] < 1 || eng[2] > eng[1] || eng[3] < 1 || eng[4] < 1 ||
        eng[5] < 1 || eng[6] < 0 || eng[7] < 1)
        return TOR_EINVAL;
    job_t J = {.n_req = n_req, .n_inst = n_inst, .arrival = arrival, .prompt = prompt,
               .decode = decode, .cached = cached, .trace = trace, .policy = policy, .k = k,
               .memguard = memguard, .delta = delta, .table = table, .eng = eng,
               .max_iters = max_iters, .ttft = ttft, .ttlt = ttlt, .tbtmax = tbtmax,
               .pct = pct, .counters = counters, .status = status, .ada = ada,
               .signal = signal, .ltr = ltr, .gamma_out = gamma_out, .switch_out = switch_out,
               .next = 0};
    if (n_threads < 1) n_threads = 1;
    if (n_threads > n_inst) n_threads = n_inst > 0 ? n_inst : 1;
    pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)n_threads);
    int started = 0;
    for (int32_t w = 1; w < n_threads; w++)
        if (pthread_create(&th[w], NULL, worker, &J) == 0) started++;
        else break;
    worker(&J);
    for (int32_t w = 1; w <= started; w++) pthread_join(th[w], NULL);
    free(th);
    for (int32_t i = 0; i < n_inst; i++)
        if (status[i]) return status[i];
    return 0;
}

int tas_oracle_log(int32_t n_req, const int64_t *arrival, const int32_t *prompt,
                   const int32_t *decode, const int32_t *cached, int32_t policy, int32_t k,
                   int32_t memguard,
                   int64_t delta, const int64_t *table, const double *ada, int32_t signal,
                   const int32_t *ltr, const int32_t *eng, int64_t max_iters, uint32_t *ttft,
                   uint32_t *ttlt, uint32_t *tbtmax, int64_t *counters, int64_t *log_iter,
                   int64_t iter_cap, int32_t *log_batch, int64_t batch_cap, int64_t *log_evict,
                   int64_t evict_cap, int64_t *n_iter, int64_t *n_batch, int64_t *n_evict) {
    if (policy < 0 || policy > P_LAST ||
        (signal != 0 && (signal < 1 || signal > 2 || policy != P_BOOST || (signal == 2 && !cached))))
        return TOR_EINVAL;
    inst_t I;
    fill_inst(&I, eng, n_req, arrival, prompt, decode, policy, k, memguard, delta, table,
              max_iters);
    I.signal = signal;
    I.H = cached;
    if (ltr) I.ltr_s = ltr[0], I.ltr_q = ltr[1];
    ada_t *A = NULL;
    if (ada && ada[0] != 0.0) {
        A = (ada_t *)malloc(sizeof *A);
        int rc = A ? ada_setup(A, ada, policy, k) : TOR_EINVAL;
        if (rc) {
            free(A);
            return rc;
        }
        I.ada = A;
    }
    log_t lg = {log_iter, iter_cap, 0, log_batch, batch_cap, 0, log_evict, evict_cap, 0, 0};
    int st = simulate(&I, ttft, ttlt, tbtmax, counters, NULL, NULL, &lg);
    free(A);
    *n_iter = lg.n_it, *n_batch = lg.n_b, *n_evict = lg.n_ev;
    if (lg.full) return TOR_EINVAL;
    return st;
}

/* ------------------------------------------------------------ JSQ cluster */

/* Replicas behind a join-shortest-queue router (paper: composability with
 * global dispatch policies). Request j of the global trace goes, at its
 * arrival a_j, to the replica holding the fewest requests at that moment
 * (dispatched to it and not completed by a_j; ties to the lowest replica),
 * each replica scheduling its own requests as one instance.
 *
 * The schedule of a replica up to time a_j depends only on the requests it
 * received before j (they arrive no later than a_j, and an iteration that
 * starts before a_j is formed before request j exists). So the count at a_j
 * is read from a full simulation of the replica over the requests it holds
 * so far: those whose completion time a + TTLT exceeds a_j are still there.
 * Only the replica that receives j changes, so it alone is simulated again. */
int tas_oracle_jsq(int32_t n_req, const int64_t *arrival, const int32_t *prompt,
                   const int32_t *decode, const int32_t *cached, int32_t replicas,
                   int32_t policy, int32_t k, int32_t memguard, int64_t delta,
                   const int64_t *table, const double *ada, int32_t signal, const int32_t *ltr,
                   const int32_t *eng, int64_t max_iters, uint32_t *ttft, uint32_t *ttlt,
                   uint32_t *tbtmax, int32_t *assign, int64_t *counters, double *gamma_out,
                   int64_t *switch_out) {
    if (n_req < 1 || replicas < 1 || policy < 0 || policy > P_LAST || k < 1 ||
        (signal != 0 && (signal < 1 || signal > 2 || policy != P_BOOST || (signal == 2 && !cached))))
        return TOR_EINVAL;
    for (int32_t j = 1; j < n_req; j++)
        if (arrival[j] < arrival[j - 1]) return TOR_EINVAL;
    const int32_t R = replicas;
    ada_t *A = NULL;
    if (ada && ada[0] != 0.0) {
        A = (ada_t *)malloc(sizeof *A);
        int rc = A ? ada_setup(A, ada, policy, k) : TOR_EINVAL;
        if (rc) {
            free(A);
            return rc;
        }
    }
    /* per replica: the global indices it holds, its gathered trace, and the
     * outputs of its latest full simulation */
    int32_t *cnt = (int32_t *)calloc((size_t)R, sizeof(int32_t));
    int32_t *idx = (int32_t *)malloc(sizeof(int32_t) * (size_t)R * (size_t)n_req);
    int64_t *ra = (int64_t *)malloc(sizeof(int64_t) * (size_t)R * (size_t)n_req);
    int32_t *rp = (int32_t *)malloc(sizeof(int32_t) * (size_t)R * (size_t)n_req * 3);
    uint32_t *out = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)R * (size_t)n_req * 3);
    int status = 0;
    if (!cnt || !idx || !ra || !rp || !out) {
        status = TOR_EINVAL;
        goto done;
    }
    for (int32_t j = 0; j <= n_req && status == 0; j++) {
        /* route j (skipped after the last request, which only simulates) */
        int32_t best = -1, best_n = 0;
        for (int32_t r = 0; r < R && j < n_req; r++) {
            const size_t o = (size_t)r * (size_t)n_req;
            int32_t held = 0;
            for (int32_t m = 0; m < cnt[r]; m++)
                held += ra[o + m] + (int64_t)out[(o + m) * 3 + 1] > arrival[j];
            if (best < 0 || held < best_n) best = r, best_n = held;
        }
        for (int32_t r = 0; r < R; r++) {
            if (j < n_req && r != best) continue;
            if (j == n_req && cnt[r] == 0) continue;
            const size_t o = (size_t)r * (size_t)n_req;
            if (j < n_req) {
                const int32_t m = cnt[r]++;
                idx[o + m] = j;
                ra[o + m] = arrival[j];
                rp[(o + m) * 3] = prompt[j];
                rp[(o + m) * 3 + 1] = decode[j];
                rp[(o + m) * 3 + 2] = cached ? cached[j] : 0;
                assign[j] = r;
            }
            /* the replica's trace as plain arrays */
            const int32_t n = cnt[r];
            int32_t *P = (int32_t *)malloc(sizeof(int32_t) * (size_t)n * 3);
            uint32_t *o3 = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)n * 3);
            if (!P || !o3) {
                free(P);
                free(o3);
                status = TOR_EINVAL;
                break;
            }
            for (int32_t m = 0; m < n; m++) {
                P[m] = rp[(o + m) * 3];
                P[n + m] = rp[(o + m) * 3 + 1];
                P[2 * n + m] = rp[(o + m) * 3 + 2];
            }
            inst_t I;
            fill_inst(&I, eng, n, ra + o, P, P + n, policy, k, memguard, delta, table, max_iters);
            I.signal = signal;
            I.H = cached ? P + 2 * n : NULL;
            I.ada = A;
            if (ltr) I.ltr_s = ltr[0], I.ltr_q = ltr[1];
            int64_t c8[8];
            double g = 0.0;
            int64_t sw = 0;
            status = simulate(&I, o3, o3 + n, o3 + 2 * n, c8, &g, &sw, NULL);
            if (status == 0) {
                for (int32_t m = 0; m < n; m++)
                    for (int q = 0; q < 3; q++) out[(o + m) * 3 + q] = o3[(size_t)q * n + m];
                if (j == n_req) { /* final: outputs in global order */
                    for (int32_t m = 0; m < n; m++) {
                        ttft[idx[o + m]] = out[(o + m) * 3];
                        ttlt[idx[o + m]] = out[(o + m) * 3 + 1];
                        tbtmax[idx[o + m]] = out[(o + m) * 3 + 2];
                    }
                    memcpy(counters + (size_t)r * 8, c8, sizeof c8);
                    if (gamma_out) gamma_out[r] = g;
                    if (switch_out) switch_out[r] = sw;
                }
            }
            free(P);
            free(o3);
            if (status) break;
        }
    }
    if (status == 0)
        for (int32_t r = 0; r < R; r++)
            if (cnt[r] == 0) { /* a replica that received nothing */
                memset(counters + (size_t)r * 8, 0, 8 * sizeof(int64_t));
                if (gamma_out) gamma_out[r] = A ? A->gamma0 : 0.0;
                if (switch_out) switch_out[r] = 0;
            }
done:
    free(cnt);
    free(idx);
    free(ra);
    free(rp);
    free(out);
    free(A);
    return status;
}
