/*
 * tas_oracle.h - CPU oracle of the tail-aware serving simulation.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product library links or calls
 * this code; only the tests, the smoke check and the benchmark's CPU-baseline
 * leg do. It shares no header, type or helper with the HIP path.
 *
 * What it computes: for every instance (one request trace, one scheduling
 * policy setting), an iteration-level simulation of a continuous-batching
 * LLM server (paper: Algorithm 1, UniBoost, gamma fixed or adaptive) whose per-step
 * execution is replaced by an integer cost model, followed by the per-request
 * latencies TTFT / TTLT / max inter-token gap and their nearest-rank
 * percentiles (paper: section "Phase 4", the definition of t_p).
 *
 * All arguments are host pointers. Arrays are flat, C-contiguous:
 *   arrival [n_traces*n_req] int64 us, non-decreasing within a trace
 *   prompt, decode [n_traces*n_req] int32 tokens, >= 1
 *   cached [n_traces*n_req] int32 expected prefix-cache hit tokens, 0 <= h < P,
 *   or NULL (needed only by signal 2)
 *   per instance i: trace[i], policy[i] (0 FCFS, 1 SRPT, 2 BOOST, 3 SPF,
 *   4 SJF, 5 LAS, 6 TRAIL, 7 DIST, 8 SARATHI, 9 LTR), k[i] >= 1,
 *   memguard[i] in {0,1}, delta[i] >= 0 us, table[i*24 .. i*24+23] int64 us
 *   eng[8] = {max_seqs, max_tokens, chunk, kv_blocks, block_tokens,
 *             iter_base_us, iter_tok_us, iter_ctx_div}
 * Outputs (caller-owned):
 *   ttft, ttlt, tbtmax [n_inst*n_req] uint32 us
 *   counters [n_inst*8] int64: iterations, request-iterations, tokens,
 *     voluntary evictions, forced evictions, final clock, max KV blocks,
 *     idle us
 *   pct [n_inst*9] uint32: {TTFT, TTLT, TBTmax} x {P50, P90, P99}
 *   status [n_inst] int32: 0 or one of the TOR_E* codes
 *
 * Adaptive gamma (paper: Phase 4, gamma-Ada; Algorithm 2 UpdateGamma), per
 * instance, optional (ada == NULL: none): ada[i*10 .. i*10+9] = {on (0/1),
 * gamma0, beta in [0,1], gamma_min, gamma_max, eps_us, window (1..2048),
 * min_samples (1..window), grid points (2..64), tau_us}. An adaptive instance
 * (BOOST only) ignores its table: it uses the table of the grid point nearest
 * to the current gamma (see tas_oracle.c). Outputs gamma_out [n_inst] (final
 * gamma, 0 when not adaptive) and switch_out [n_inst] (grid-cell changes) may
 * be NULL.
 *
 * ltr [n_inst*2] (NULL: no LTR instance): for an LTR instance (SJF (LTR+),
 * the evaluation's baselines) ltr[2i] = the starvation threshold S >= 1 and
 * ltr[2i+1] = the promotion quantum Q >= 1, both in iterations (see
 * tas_oracle.c); ignored for the other policies. tas_oracle_log and
 * tas_oracle_jsq take the pair of their one setting (or NULL).
 *
 * signal [n_inst] (NULL: all 0): the boost signal of a BOOST instance, 0 =
 * prompt plus emitted tokens, 1 = Algorithm 2's phase-aware signal (prompt
 * length in prefill, emitted tokens in decode), 2 = prompt minus expected
 * cached tokens plus emitted tokens (prefix caching).
 */
#ifndef TAS_ORACLE_H
#define TAS_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TOR_LEVELS 24
#define TOR_EINVAL (-1)
#define TOR_EINFEASIBLE (-2)
#define TOR_EOVERFLOW (-5)
#define TOR_ELIVELOCK (-6)
#define TOR_ESTATE (-7)

/* Boost table from the gamma-Boost function (paper, Eq. boost_function):
 * out[j] = min(2^42, round(tau * b_gamma(k * 2^j))), b_gamma(w) =
 * (1/gamma) * ln(1 / (1 - exp(-gamma*w))). Returns 0, or TOR_EINVAL. */
int tas_oracle_boost_table(double gamma, int32_t k, double tau_us, int64_t *out);

/* Run all instances on n_threads host threads (instances are independent).
 * Returns 0 if every instance finished, else the first nonzero status. */
int tas_oracle_run(int32_t n_traces, int32_t n_req, const int64_t *arrival,
                   const int32_t *prompt, const int32_t *decode, const int32_t *cached,
                   int32_t n_inst,
                   const int32_t *trace, const int32_t *policy, const int32_t *k,
                   const int32_t *memguard, const int64_t *delta, const int64_t *table,
                   const int32_t *eng, int64_t max_iters, uint32_t *ttft, uint32_t *ttlt,
                   uint32_t *tbtmax, int64_t *counters, uint32_t *pct, int32_t *status,
                   const double *ada, const int32_t *signal, const int32_t *ltr,
                   double *gamma_out, int64_t *switch_out, int32_t n_threads);

/* Run ONE instance and record its schedule, for invariant checks.
 * log_iter[it*8 + {0..7}] = {t_start, dt, batch size, KV blocks in use
 *   after formation, waiting count, resident count after formation, grid
 *   cell of the boost table used (-1 when gamma is fixed), the bits of gamma
 *   (IEEE double)}; ada: 10 parameters as above, or NULL;
 * log_batch[...] = (request index, tokens) pairs, iteration after iteration;
 * log_evict[...] = (iteration, evicted request, forced flag, the candidate
 *   whose admission caused it) records of 4.
 * Capacities are in records. *n_iter, *n_batch, *n_evict receive the counts.
 * Returns the instance status, or TOR_EINVAL if a log buffer is too small. */
int tas_oracle_log(int32_t n_req, const int64_t *arrival, const int32_t *prompt,
                   const int32_t *decode, const int32_t *cached, int32_t policy, int32_t k,
                   int32_t memguard,
                   int64_t delta, const int64_t *table, const double *ada, int32_t signal,
                   const int32_t *ltr, const int32_t *eng, int64_t max_iters, uint32_t *ttft,
                   uint32_t *ttlt, uint32_t *tbtmax, int64_t *counters, int64_t *log_iter,
                   int64_t iter_cap, int32_t *log_batch, int64_t batch_cap, int64_t *log_evict,
                   int64_t evict_cap, int64_t *n_iter, int64_t *n_batch, int64_t *n_evict);

/* The adaptive-gamma grid of prm[10] (layout as above, on = 1): grid[G],
 * midpoints bound[G-1], boost tables tables[G*24]. Returns 0 or TOR_EINVAL. */
int tas_oracle_ada_grid(const double *prm, int32_t k, double *grid, double *bound,
                        int64_t *tables);

/* MemGuard level of signal w at granularity k: floor(log2(max(w,k)/k)),
 * capped at 23 (paper, Eq. memguard_level). */
int32_t tas_oracle_level(int64_t w, int32_t k);

/* Nearest-rank percentile of n values: the value at sorted position
 * ceil(q*n/100) - 1. */
uint32_t tas_oracle_percentile(const uint32_t *v, int32_t n, int32_t q);

/* Replicas behind a join-shortest-queue router (paper: composability with
 * global dispatch policies): the n_req requests of one global trace are
 * dispatched, at their arrival and in index order, to the replica holding
 * the fewest requests not yet completed (ties to the lowest replica); every
 * replica runs the one setting given (policy .. signal as for
 * tas_oracle_log; ada[10] or NULL). Outputs: ttft, ttlt, tbtmax [n_req] in
 * global order, assign [n_req] (the replica of each request), counters
 * [replicas*8], gamma_out and switch_out [replicas] (may be NULL). */
int tas_oracle_jsq(int32_t n_req, const int64_t *arrival, const int32_t *prompt,
                   const int32_t *decode, const int32_t *cached, int32_t replicas,
                   int32_t policy, int32_t k, int32_t memguard, int64_t delta,
                   const int64_t *table, const double *ada, int32_t signal, const int32_t *ltr,
                   const int32_t *eng, int64_t max_iters, uint32_t *ttft, uint32_t *ttlt,
                   uint32_t *tbtmax, int32_t *assign, int64_t *counters, double *gamma_out,
                   int64_t *switch_out);

#ifdef __cplusplus
}
#endif
#endif
