/*
 * tas.h - C ABI of the batched tail-aware serving simulation on MI355X.
 *
 * A sweep is a set of INSTANCES. Each instance pairs one synthetic request
 * trace with one scheduling-policy setting and is simulated independently,
 * iteration by iteration, as a continuous-batching LLM server:
 *
 *   - request i is (a_i arrival us, P_i prompt tokens known at arrival,
 *     D_i decode tokens unknown to a blind policy)
 *     (arXiv 2606.18431, section "Formulation", Notation);
 *   - every iteration ranks the waiting and resident requests by a priority
 *     key, smaller first, ties by request index:
 *       TAS_FCFS   key = a_i                                   (Table 1, FCFS)
 *       TAS_SRPT   key = P_i + D_i - 1 - kv_i  (exact remaining tokens;
 *                  Table 1, SRPT with perfect length knowledge)
 *       TAS_SPF    key = P_i                (Table 1, shortest prefix first)
 *       TAS_SJF    key = D_i   (Table 1, SJF with perfect output-length rank)
 *       TAS_LAS    key = P_i + dec_i        (Table 1 and baselines, least
 *                  attained service)
 *       TAS_TRAIL  key as TAS_SRPT; a resident that emitted at least 0.6 D_i
 *                  tokens is never a voluntary victim (baselines, TRAIL+
 *                  swap-prevention threshold)
 *       TAS_BOOST  key = a_i - boost_us[level(P_i + dec_i)]    (Phase 2 unified
 *                  key Phi = a - b_gamma(w~) with w~ = max(w, s_pre); Phase 3
 *                  MemGuard quantization level = floor(log2(max(w,k)/k)));
 *                  with signal = 1 the level is that of Algorithm 2's
 *                  phase-aware signal: P_i before the first token, dec_i after;
 *                  with signal = 2 that of P_i - h_i + dec_i, h_i the expected
 *                  prefix-cache hit tokens (section "Interaction with other
 *                  system optimization", prefix/radix caching: effective work
 *                  max(w, s_pre - h) with cached tokens not counted as
 *                  processed); the engine still prefills all P_i tokens
 *       TAS_DIST   DistBoost (Phase 1): before its first token a request is
 *                  in the prefill queue, key a_i - boost_us[level(P_i)]; after
 *                  it, in the decode queue, key t_first - 2^42, so the decode
 *                  queue in order of entry fills the batch first and prefill
 *                  chunks fill the rest
 *       TAS_LTR    SJF (LTR+; the evaluation's baselines, item 2, and Table 1's
 *                  LTR row): the SJF key D_i plus starvation control by
 *                  quantum promotion. After every iteration a candidate that
 *                  did not run adds one to its starvation count and one that
 *                  ran resets it; at ltr_starve the request is promoted: key
 *                  j - 2^42 for a promotion at the end of iteration j (ahead
 *                  of every unpromoted request, promoted ones in order of
 *                  promotion), for ltr_quantum iterations in which it runs,
 *                  after which it returns to key D_i with a count of zero
 *       TAS_SARATHI decode-prioritized continuous batching with round-robin
 *                  decodes and piggy-backed prefill chunks (the evaluation's
 *                  baselines, Sarathi): key a_i before the first token, then
 *                  t_last - 2^42 with t_last the time of the request's latest
 *                  token, so decodes rotate (longest unserved first) ahead of
 *                  prefills in arrival order; a waiting request never evicts a
 *                  resident (only a resident that cannot grow forces one out)
 *   - a greedy pass fills the batch under a sequence cap, a token budget and a
 *     KV-block budget, evicting (recompute preemption) the worst resident when
 *     KV runs out; MemGuard and the hysteresis delta restrict voluntary
 *     evictions (Algorithm 1; Phase 2 preemption protocol; Phase 3);
 *   - the iteration costs base + tok * sum(tokens) + floor(sum(context)/div) us
 *     (the engine's forward step, Algorithm 1 ExecuteOneStep, replaced by an
 *     integer cost model);
 *   - each request's TTFT, TTLT and maximum inter-token gap are recorded, and
 *     reduced per instance to nearest-rank P50/P90/P99 (Phase 4, t_p);
 *   - optionally (TAS_BOOST, tas_setting.ada = 1) gamma adapts online (Phase 4,
 *     gamma-Ada; Algorithm 2 UpdateGamma, run before the keys of every
 *     iteration): once the window of the last `ada_window` end-to-end
 *     latencies (TTLT of completed requests, in completion order; requests
 *     finishing in one iteration in batch order) holds `ada_min_samples`
 *     values, gamma_hat = (tau_us ln 5) / max(t99 - t95, ada_eps_us) with
 *     nearest-rank t95, t99 of the window (the tail-band slope of
 *     Eq. gamma_estimator, ln 5 = ln(0.05/0.01), per token of boost), and
 *     gamma = clip((1 - beta) gamma + beta gamma_hat, gamma_min, gamma_max),
 *     each step one rounded IEEE double operation. The boost table in use is
 *     that of the grid point nearest gamma in log scale on the grid
 *     g_j = gamma_min (gamma_max/gamma_min)^(j/(G-1)), j < G (midpoints
 *     sqrt(g_j g_{j+1}) round up), so priorities stay integers.
 *
 * Everything is integer arithmetic; results are deterministic and independent
 * of the launch configuration.
 *
 * Memory. Host pointers are marked HOST, device pointers DEVICE. The caller
 * owns all memory: the workspace and every output buffer are device
 * allocations made by the caller (for instance PyTorch tensors), which must
 * stay allocated and untouched until the stream has been synchronised and the
 * context destroyed. The context holds host metadata only; tas_destroy frees
 * that and nothing else. One context is used by one host thread at a time.
 *
 * Streams. `stream` is a hipStream_t passed as void*; NULL is the default
 * stream. tas_run, tas_percentiles, tas_latencies and tas_counters enqueue
 * work and return without waiting; calls on one context must use one stream,
 * or the caller orders them.
 *
 * Errors. Functions return TAS_OK (0) or a negative TAS_E* code; no C++
 * exception crosses the ABI. Per-instance device errors are sticky and are
 * reported by tas_status.
 */
#ifndef TAS_H
#define TAS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    TAS_OK = 0,
    TAS_EINVAL = -1,      /* invalid argument or input (see tas_create)        */
    TAS_EINFEASIBLE = -2, /* a request needs more KV than the budget holds     */
    TAS_ENOMEM = -3,      /* workspace too small                               */
    TAS_EHIP = -4,        /* a HIP runtime call failed                         */
    TAS_EOVERFLOW = -5,   /* a latency does not fit 32 bits of microseconds   */
    TAS_ELIVELOCK = -6,   /* an instance exceeded max_iters iterations         */
    TAS_ESTATE = -7,      /* internal consistency check failed                 */
    TAS_ECAPACITY = -8    /* an instance outgrew its on-chip candidate list    */
};

enum { TAS_FCFS = 0, TAS_SRPT = 1, TAS_BOOST = 2, TAS_SPF = 3, TAS_SJF = 4, TAS_LAS = 5,
       TAS_TRAIL = 6, TAS_DIST = 7, TAS_SARATHI = 8, TAS_LTR = 9 };

#define TAS_LEVELS 24

/* Request traces, trace-major structure-of-arrays (all HOST, read during
 * tas_create only). Every trace holds n_req requests sorted by arrival. */
typedef struct {
    int32_t n_traces;
    int32_t n_req;              /* 1 <= n_req < 2^20                           */
    const int64_t *arrival_us;  /* [n_traces*n_req], 0 <= a < 2^41, sorted     */
    const int32_t *prompt;      /* [n_traces*n_req], >= 1                      */
    const int32_t *decode;      /* [n_traces*n_req], >= 1; P + D < 2^24        */
    const int32_t *cached;      /* [n_traces*n_req] expected prefix-cache hit
                                   tokens, 0 <= h < P, or NULL; read only by
                                   settings with signal = 2                    */
} tas_traces;

/* One instance: a trace and a policy setting. */
typedef struct {
    int32_t trace;    /* index into the traces                                 */
    int32_t policy;   /* one of the TAS_FCFS .. TAS_LTR policies above         */
    int32_t k;        /* MemGuard granularity in tokens (BOOST, DIST), >= 1    */
    int32_t memguard; /* 1: a dispatched request is non-evictable until its
                         level passes the level it was dispatched at (BOOST)  */
    int64_t delta_us; /* hysteresis: a voluntary victim's key must exceed the
                         candidate's by more than delta (BOOST), >= 0          */
    double gamma;     /* BOOST: > 0 builds boost_us from the gamma-Boost curve
                         (tas_boost_table); 0 uses boost_us as given           */
    int32_t table_given; /* 1: boost_us is an explicit table (gamma ignored)  */
    int32_t ada;         /* 1: adaptive gamma from `gamma` (BOOST, no explicit
                            table); 0: the ada_* fields are ignored           */
    int64_t boost_us[TAS_LEVELS]; /* explicit table: non-increasing, in
                                     [0, 2^42]                                 */
    /* adaptive gamma (ada = 1), see the top of this file */
    double ada_beta;       /* EMA weight per iteration, in [0, 1]              */
    double ada_gamma_min;  /* clip bounds and grid ends: 0 < gamma_min <       */
    double ada_gamma_max;  /*   gamma_max, gamma_min <= gamma <= gamma_max     */
    double ada_eps_us;     /* floor of t99 - t95, > 0                          */
    int32_t ada_window;    /* latencies kept, in [1, TAS_ADA_WINDOW_MAX]       */
    int32_t ada_min_samples; /* window size before the first update, in
                                [1, ada_window]                                */
    int32_t ada_grid;      /* grid points G, in [2, TAS_ADA_GRID_MAX]          */
    int32_t signal;        /* BOOST: 0 = P + dec; 1 = the phase-aware signal of
                              Algorithm 2 (P in prefill, dec in decode); 2 =
                              P - h + dec with h from tas_traces.cached; 0
                              for every other policy                          */
    /* SJF (LTR+), see TAS_LTR above; both 0 for every other policy */
    int32_t ltr_starve;    /* iterations without service that promote, in
                              [1, 32767]                                       */
    int32_t ltr_quantum;   /* iterations of service a promotion grants, in
                              [1, 32767]                                       */
} tas_setting;

#define TAS_ADA_WINDOW_MAX 2048
#define TAS_ADA_GRID_MAX 64

/* Engine limits, cost model and the instance list (HOST). */
typedef struct {
    int32_t max_seqs;      /* sequences per iteration, >= 1                    */
    int32_t max_tokens;    /* tokens per iteration, >= chunk                   */
    int32_t chunk;         /* prefill chunk, 1 <= chunk <= 32767               */
    int32_t kv_blocks;     /* KV budget in blocks, >= 1                        */
    int32_t block_tokens;  /* tokens per KV block, >= 1                        */
    int32_t iter_base_us;  /* iteration cost: base + tok*sum(n)                */
    int32_t iter_tok_us;   /*   + floor(sum(kv+n) / ctx_div), base >= 1        */
    int32_t iter_ctx_div;  /*   ctx_div >= 1                                   */
    int64_t max_iters;     /* per-instance iteration limit (TAS_ELIVELOCK)     */
    double tau_us;         /* microseconds per token of boost, > 0             */
    int32_t list_cap;      /* on-chip candidate entries per instance, in
                              [max_seqs + 64, 4032]; 0 picks max_seqs + 128,
                              or max_seqs + 768 when some instance adapts
                              gamma, rounded up to 64                          */
    int32_t spill_cap;     /* waiting entries per instance kept in HBM beyond
                              the on-chip list; 0 = n_req                      */
    int32_t n_inst;
    int32_t retry_cap;     /* an instance that holds more residents than
                              list_cap reruns from scratch with this larger
                              list (tas_run enqueues the second pass); 0 picks
                              min(4032, max(2048, 4 list_cap)). Beyond it:
                              TAS_ECAPACITY                                    */
    const tas_setting *inst; /* [n_inst]                                       */
    int32_t jsq_replicas;  /* 0 or 1: every instance is one server. 2 ..
                              TAS_MAX_REPLICAS: every instance is a cluster of
                              that many replicas behind a join-shortest-queue
                              router (section "Composability with Global
                              Dispatch Policies"): its trace is the global
                              arrival stream; request j goes, at a_j, to the
                              replica holding the fewest requests not completed
                              by a_j (ties to the lowest replica), and each
                              replica schedules its requests with the
                              instance's setting (an adaptive setting adapts
                              gamma per replica)                              */
} tas_params;

#define TAS_MAX_REPLICAS 16

typedef struct tas_ctx tas_ctx;

/* Bytes of device workspace tas_create needs for these inputs, or 0 if the
 * arguments are invalid. */
size_t tas_workspace_bytes(const tas_traces *traces, const tas_params *params);

/* Validate the inputs, build every boost table, lay out the workspace and
 * copy the traces and settings into it (synchronous host-to-device copies).
 * The inputs are the paper's problem statement (section "Formulation",
 * Notation: requests (a_i, P_i, D_i) arriving online) plus the policy
 * settings (Eq. boost_function for the tables; Phase 3 k and MemGuard; Phase
 * 2 hysteresis delta) and the engine limits of Algorithm 1 (batch size, token
 * budget, KV blocks).
 * d_ws: DEVICE buffer of ws_bytes >= tas_workspace_bytes(...), 256-byte
 * aligned, owned by the caller. *out receives a new context.
 * Returns TAS_EINVAL if: n_req < 1 or >= 2^20; an arrival is negative,
 * >= 2^41 or out of order; P or D < 1; P + D >= 2^24; a trace index is out of
 * range; policy unknown; k < 1 (BOOST); delta < 0; memguard or delta nonzero
 * for a policy other than BOOST; gamma <= 0 without table_given (BOOST,
 * DIST); an explicit table not non-increasing or outside [0, 2^42] (DIST:
 * [0, 2^40], also for a table built from gamma); signal not 0, or 1 or 2 for
 * BOOST; signal 2 without traces->cached; a cached value < 0 or >= its P;
 * ada not 0 or 1; ada = 1 with a policy
 * other than BOOST, with table_given, or with an ada_* field outside its
 * range; chunk > max_tokens; any engine limit
 * < 1; chunk > 32767; tau <= 0; list_cap < max_seqs + 64 or > 4032;
 * jsq_replicas < 0 or > TAS_MAX_REPLICAS; jsq_replicas > 1 with the lists
 * (and adaptive-gamma windows) of all replicas beyond the 160 KB of LDS.
 * TAS_EINFEASIBLE if ceil((P + D - 1) / block_tokens) > kv_blocks for some
 * request. TAS_ENOMEM if ws_bytes is too small. TAS_EHIP if a copy fails. */
int tas_create(const tas_traces *traces, const tas_params *params, void *d_ws, size_t ws_bytes,
               tas_ctx **out);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops, harnesses that forbid hipMalloc): tas_create with
 * the workspace in a static device array of TAS_STATIC_WORKSPACE_BYTES that
 * the library holds on each GPU it runs on until the process ends. No device
 * memory is allocated. Returns TAS_ENOMEM when tas_workspace_bytes exceeds
 * TAS_STATIC_WORKSPACE_BYTES, TAS_EHIP when the array's address cannot be
 * obtained, otherwise as tas_create. All contexts created this way on one
 * GPU share its array: creating one overwrites the workspace of the previous
 * one, which must no longer be used, and calls on two such contexts that
 * overlap on one GPU race. The array keeps the last call's contents; what
 * must start at zero is cleared by this call, as by tas_create. */
#define TAS_STATIC_WORKSPACE_BYTES ((size_t)64 << 20)
int tas_create_static(const tas_traces *traces, const tas_params *params, tas_ctx **out);

/* Enqueue the simulation of every instance on `stream` (one workgroup per
 * instance), followed by the retry pass for instances that outgrew list_cap.
 * Each instance runs Algorithm 1's loop (arrivals, keys, the greedy batch with
 * KVNeed / SelectVictim / SwapOut, ExecuteOneStep as the integer cost model,
 * UpdateStats; with ada = 1 also UpdateGamma of Algorithm 2) until its last
 * request completes.
 * Per-request latencies, counters and errors land in the workspace. The
 * workgroups (up to 16384 instances, without replicas) take the instances
 * longest first: a launch lasts until its last instance ends. The first call
 * ranks them by an estimate of their work from the inputs (the sum over the
 * trace of D + ceil(P / chunk), times 5/4 for SRPT, TRAIL, LAS and Sarathi),
 * later calls by the work each instance did in the previous call, counted in
 * loop steps of its wavefront (4 per iteration, 5 per formation pass over up
 * to 64 candidates, 3 per emission chunk: their measured relative cost), a
 * measure that, unlike its wall-clock time, does not depend on where it ran.
 * Consecutive workgroups
 * go to different XCDs, so the sorted order also spreads each kind of
 * instance over them. The results do not depend on the order. Calls on one
 * context share its workspace: a call on another stream must be ordered
 * after the previous one by the caller. */
int tas_run(tas_ctx *ctx, void *stream);

/* Enqueue the nearest-rank percentile reduction: d_out DEVICE uint32
 * [n_inst][3][3] = {TTFT, TTLT, TBTmax} x {P50, P90, P99}, the value at
 * sorted position ceil(q*n_req/100) - 1 (Phase 4, t_p). Call after tas_run on
 * the same stream. */
int tas_percentiles(tas_ctx *ctx, uint32_t *d_out, void *stream);

/* Nearest-rank percentiles over groups of `group` adjacent instances (the
 * replicas of one cluster behind a global router; paper: global dispatch
 * policies and cluster scale): d_out DEVICE uint32 [n_inst/group][3][3], the
 * value at sorted position ceil(q*m/100) - 1 of the group's m = group*n_req
 * latencies pooled. Call after tas_run on the same stream. TAS_EINVAL unless
 * group >= 1 divides n_inst and group*n_req < 2^31. */
int tas_percentiles_grouped(tas_ctx *ctx, int32_t group, uint32_t *d_out, void *stream);

/* Enqueue device-to-device copies of the per-request latencies, DEVICE
 * uint32 [n_inst][n_req] each, microseconds relative to arrival: TTFT, TTLT
 * (T_i = C_i - a_i of section "Formulation") and the largest gap between two
 * consecutive tokens (the TBT of Table 2, per request its maximum); any
 * pointer may be NULL to skip that array. */
int tas_latencies(tas_ctx *ctx, uint32_t *d_ttft, uint32_t *d_ttlt, uint32_t *d_tbtmax,
                  void *stream);

/* Enqueue a copy of the per-instance counters, DEVICE int64 [n_inst][8]
 * (Algorithm 1's loop as run: its iterations and batches, the SwapOut
 * evictions, the KV blocks of KVNeed): iterations, request-iterations (sum of
 * batch sizes), computed tokens,
 * voluntary evictions, forced evictions, final clock us, peak KV blocks,
 * idle us. For a cluster (jsq_replicas > 1): sums over its replicas, except
 * the final clock and the peak KV blocks, which are the largest. */
int tas_counters(tas_ctx *ctx, int64_t *d_out, void *stream);

/* Enqueue copies of the adaptive-gamma state at the end of each instance:
 * d_gamma DEVICE double [n_inst] (the final gamma; 0 for an instance without
 * adaptive gamma) and d_switches DEVICE int64 [n_inst] (how often the boost
 * table changed grid point). Either pointer may be NULL. */
int tas_gamma(tas_ctx *ctx, double *d_gamma, int64_t *d_switches, void *stream);

/* Clusters behind the join-shortest-queue router (jsq_replicas > 1):
 * enqueue copies of the replica each request went to, d_assign DEVICE int32
 * [n_inst][n_req], of each replica's counters (as tas_counters), d_counters
 * DEVICE int64 [n_inst][jsq_replicas][8], and of each replica's final
 * adaptive gamma and grid-cell changes (as tas_gamma), d_gamma DEVICE double
 * and d_switches DEVICE int64 [n_inst][jsq_replicas]. Any pointer may be
 * NULL. TAS_EINVAL for a context without replicas. */
int tas_replicas(tas_ctx *ctx, int32_t *d_assign, int64_t *d_counters, double *d_gamma,
                 int64_t *d_switches, void *stream);

/* Synchronise the stream of the last enqueued call and return TAS_OK or the
 * first per-instance error (lowest instance index), e.g. TAS_ELIVELOCK,
 * TAS_EOVERFLOW, TAS_ECAPACITY; TAS_EHIP if the stream reports a failure. */
int tas_status(tas_ctx *ctx);

/* The schedule of the latest tas_run: d_work DEVICE int64 [n_inst], the key
 * the next tas_run orders the instances by, largest first (before the first
 * run: the work estimates; after a run: each instance's work in it in loop
 * steps, as tas_run describes), and d_order DEVICE int32 [n_inst], the instance each workgroup took
 * (a permutation; the index order before the first run). Either pointer may
 * be NULL. TAS_EINVAL where no order is kept (replicas, or more than 16384
 * instances). */
int tas_schedule(tas_ctx *ctx, int64_t *d_work, int32_t *d_order, void *stream);

/* Per-instance status codes, DEVICE int32 [n_inst] (enqueued copy). */
int tas_instance_status(tas_ctx *ctx, int32_t *d_out, void *stream);

/* Free the context's host metadata; device memory is untouched. */
void tas_destroy(tas_ctx *ctx);

/* A static English description of a return code. */
const char *tas_strerror(int code);

/* The gamma-Boost table (Eq. boost_function): out[j] = min(2^42,
 * round(tau_us * b_gamma(k 2^j))) with b_gamma(w) = (1/gamma) ln(1/(1 -
 * exp(-gamma w))), evaluated in double precision on the host. out: HOST
 * int64[TAS_LEVELS]. Returns TAS_EINVAL unless gamma > 0, k >= 1, tau > 0. */
int tas_boost_table(double gamma, int32_t k, double tau_us, int64_t *out);

/* The adaptive-gamma grid of a setting (ada = 1 and valid ada_* fields, as
 * tas_create requires): grid[j] = gamma_min (gamma_max/gamma_min)^(j/(G-1)),
 * bound[j] = sqrt(grid[j] grid[j+1]) for j < G-1, and tables[j*TAS_LEVELS ..]
 * = the tas_boost_table of grid[j] (k and tau_us as given), all evaluated in
 * double precision on the host (Phase 4 with the boost curve of
 * Eq. boost_function). grid, bound, tables: HOST arrays of G, G-1 and
 * G*TAS_LEVELS elements. Returns TAS_EINVAL for an invalid setting. */
int tas_ada_grid(const tas_setting *s, double tau_us, double *grid, double *bound,
                 int64_t *tables);

/* The boost table an instance uses (as built by tas_create). out: HOST
 * int64[TAS_LEVELS]. */
int tas_instance_table(const tas_ctx *ctx, int32_t inst, int64_t *out);

/* The on-chip candidate-list capacity the context uses per instance. */
int32_t tas_list_cap(const tas_ctx *ctx);

#ifdef __cplusplus
}
#endif
#endif
