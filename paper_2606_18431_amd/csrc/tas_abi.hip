// tas_abi.hip - host side of the C ABI declared in include/tas.h.
//
// tas_create validates the inputs on the host (so every rejection is testable
// without a GPU), builds each instance's boost table, lays the workspace out
// and copies the traces and settings into it once. tas_run / tas_percentiles
// only enqueue kernels; nothing on the path allocates.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "tas.h"
#include "tas_internal.h"

struct tas_ctx {
    int32_t n_traces = 0, n_req = 0, n_inst = 0, list_cap = 0, spill_cap = 0, retry_cap = 0;
    int32_t replicas = 1;  // > 1: replicas behind a join-shortest-queue router
    bool ordered = false;  // order the next launch by `work` (estimates, then loop steps)
    int64_t lds_bytes = 0, lds_retry = 0;
    tas::SimArgs args{};
    std::vector<tas::DevSetting> settings;
    std::vector<tas::DevAda> ada;
    hipStream_t last_stream = nullptr;
};

namespace {

constexpr int64_t kMaxLds = 160 * 1024;  // gfx950 LDS per workgroup
constexpr int64_t kTwo41 = int64_t(1) << 41;
constexpr int64_t kTwo42 = int64_t(1) << 42;
constexpr int64_t kTwo40 = int64_t(1) << 40;  // DistBoost tables: decode keys stay below
constexpr int32_t kLtrMax = (1 << 15) - 1;    // LTR+ counts live in 15 bits of the flag word

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

struct Layout {
    size_t arrival, prompt, decode, cached, settings, ada, tfirst, tlast, ttft, ttlt, tbtmax,
        counters, status, gamma, switches, spill, ovf, jidx, assign, rcounters, rgamma, rswitches,
        work, order, total;
};

// Replicas per instance behind the join-shortest-queue router (1: none).
int32_t replicas_of(const tas_params *p) { return p->jsq_replicas > 1 ? p->jsq_replicas : 1; }

// Dynamic LDS of a launch: one list per instance, or the router block and
// one 16-aligned list per replica (replicas use four-word slots).
int64_t launch_lds(int32_t list_cap, int32_t wmax, int32_t replicas, bool compact) {
    if (replicas <= 1) return tas::lds_bytes_for(list_cap, wmax, compact);
    const int64_t one = tas::lds_bytes_for(list_cap, wmax);
    return tas::kJsqLdsBytes + (int64_t)replicas * ((one + 15) & ~int64_t(15));
}

// Compact list slots (24 LDS bytes per entry instead of 32) hold w = P + dec
// and kv in 16 bits and left - 1 in 15: usable when every request has
// P + D <= 65535 and D <= 32768, and the instance is a single server.
bool compact_ok(const tas_traces *t, const tas_params *p) {
    if (replicas_of(p) > 1) return false;
    for (int32_t i = 0; i < p->n_inst; i++)  // LTR+ keeps its counts in those bits
        if (p->inst[i].policy == TAS_LTR) return false;
    const size_t tn = (size_t)t->n_traces * (size_t)t->n_req;
    for (size_t i = 0; i < tn; i++) {
        const int64_t P = t->prompt[i], D = t->decode[i];
        if (P + D > tas::kCompactMaxPD || D > tas::kCompactMaxD) return false;
    }
    return true;
}

// Adaptive-gamma instances and their largest window (clamped: an invalid
// window is rejected by check_setting).
int32_t ada_count(const tas_params *p, int32_t *wmax) {
    int32_t n = 0, w = 0;
    for (int32_t i = 0; i < p->n_inst; i++) {
        if (p->inst[i].ada == 0) continue;
        n++;
        w = std::max(w, std::min(std::max(p->inst[i].ada_window, 0), tas::kAdaWindowMax));
    }
    *wmax = w;
    return n;
}

// First pass: room for about max_seqs residents plus a window of waiting
// entries, small enough for several instances per compute unit. Instances
// that hold more residents than that rerun in a second pass with a large list.
// The kernel is bound by each wavefront's dependent instruction chain, so the
// number of instances sharing a compute unit (its LDS divided by an
// instance's) matters more than the last waiting entries on chip: the list
// holds max_seqs + 128 entries, shrunk (not below max_seqs + 64, in steps of
// 8) to the largest size at which 16, or else 12, instances fit. (On the
// large sweep, 256 sequences: 352 compact entries, 16 per compute unit.)
// With adaptive gamma every grid change reorders the queue; requests admitted
// under the old order keep their KV until the budget binds, so residents
// outside the batch accumulate (beyond 3 max_seqs on the large sweep):
// launches with adaptive instances start with 768 more entries, so that a
// rerun is rare (the adaptive build keeps only residents + 128 on chip, so
// the larger list costs occupancy, not longer passes).
int32_t default_list_cap(int32_t max_seqs, bool adaptive, bool compact) {
    if (adaptive) {
        const int64_t lc = ((int64_t)max_seqs + 768 + 63) / 64 * 64;
        return (int32_t)std::min<int64_t>(lc, tas::kMaxListCap);
    }
    const int64_t lo = (int64_t)max_seqs + 64, hi = (int64_t)max_seqs + 128;
    for (const int64_t per_cu : {16, 12}) {
        int64_t l = hi;
        while (l >= lo && tas::lds_bytes_for((int32_t)std::min<int64_t>(l, tas::kMaxListCap), 0,
                                             compact) * per_cu > kMaxLds)
            l = (l - 1) / 8 * 8;
        if (l >= lo) return (int32_t)std::min<int64_t>(l, tas::kMaxListCap);
    }
    return (int32_t)std::min<int64_t>(hi, tas::kMaxListCap);
}
int32_t default_retry_cap(int32_t list_cap) {
    return (int32_t)std::min<int64_t>(std::max<int64_t>(4 * (int64_t)list_cap, 2048),
                                      tas::kMaxListCap);
}

bool engine_ok(const tas_params *p) {
    return p->max_seqs >= 1 && p->max_tokens >= 1 && p->chunk >= 1 && p->chunk <= p->max_tokens &&
           p->chunk <= tas::kMaxChunk &&
           p->kv_blocks >= 1 && p->block_tokens >= 1 && p->iter_base_us >= 1 &&
           p->iter_tok_us >= 0 && p->iter_ctx_div >= 1 && p->max_iters >= 1 &&
           p->tau_us > 0.0 && std::isfinite(p->tau_us) && p->n_inst >= 0 &&
           p->jsq_replicas >= 0 && p->jsq_replicas <= tas::kMaxReplicas &&
           p->list_cap >= 0 && p->spill_cap >= 0 && (p->n_inst == 0 || p->inst != nullptr);
}

bool shape_ok(const tas_traces *t) {
    return t && t->n_traces >= 1 && t->n_req >= 1 && t->n_req < (1 << 20) && t->arrival_us &&
           t->prompt && t->decode;
}

// Effective capacities and slot layout; false if invalid. *rc == *lc means
// no second pass.
bool caps(const tas_traces *t, const tas_params *p, int32_t *lc, int32_t *rc, int32_t *sc,
          bool *cp) {
    int32_t wmax;
    const bool adaptive = ada_count(p, &wmax) > 0;
    const bool compact = compact_ok(t, p);
    const int32_t l =
        p->list_cap ? p->list_cap : default_list_cap(p->max_seqs, adaptive, compact);
    if ((int64_t)l < (int64_t)p->max_seqs + 64 || l > tas::kMaxListCap) return false;
    const int32_t nr = replicas_of(p);
    if (launch_lds(l, wmax, nr, compact) > kMaxLds) return false;
    int32_t r = p->retry_cap ? p->retry_cap : default_retry_cap(l);
    if (r < l) r = l;
    while (r > l && launch_lds(r, wmax, nr, compact) > kMaxLds) r -= 64;  // room for the window
    if (r > tas::kMaxListCap || tas::lds_bytes_for(r, wmax, compact) > kMaxLds) return false;
    *lc = l;
    *rc = r;
    *sc = p->spill_cap ? p->spill_cap : t->n_req;
    *cp = compact;
    return true;
}

bool layout(const tas_traces *t, const tas_params *p, int32_t rc, int32_t sc, Layout *L) {
    const size_t tn = (size_t)t->n_traces * (size_t)t->n_req;
    const size_t in = (size_t)p->n_inst * (size_t)t->n_req;
    size_t o = 0;
    L->arrival = o, o = align256(o + tn * 8);
    L->prompt = o, o = align256(o + tn * 4);
    L->decode = o, o = align256(o + tn * 4);
    L->cached = o, o = align256(o + (t->cached ? tn * 4 : 0));
    L->settings = o, o = align256(o + (size_t)p->n_inst * sizeof(tas::DevSetting));
    int32_t wmax;
    L->ada = o, o = align256(o + (size_t)ada_count(p, &wmax) * sizeof(tas::DevAda));
    L->tfirst = o, o = align256(o + in * 8);
    L->tlast = o, o = align256(o + in * 8);
    L->ttft = o, o = align256(o + in * 4);
    L->ttlt = o, o = align256(o + in * 4);
    L->tbtmax = o, o = align256(o + in * 4);
    L->counters = o, o = align256(o + (size_t)p->n_inst * 8 * 8);
    L->status = o, o = align256(o + (size_t)p->n_inst * 4);
    L->gamma = o, o = align256(o + (size_t)p->n_inst * 8);
    L->switches = o, o = align256(o + (size_t)p->n_inst * 8);
    const size_t nr = (size_t)replicas_of(p), slots = (size_t)p->n_inst * nr;
    L->spill = o, o = align256(o + slots * (size_t)sc * sizeof(tas::Rec));
    L->ovf = o, o = align256(o + slots * (size_t)(rc + tas::kStage) * sizeof(tas::Rec));
    const bool cl = nr > 1;  // the router's lists, assignment and per-replica counters
    L->jidx = o, o = align256(o + (cl ? slots * (size_t)t->n_req * 4 : 0));
    L->assign = o, o = align256(o + (cl ? in * 4 : 0));
    L->rcounters = o, o = align256(o + (cl ? slots * 8 * 8 : 0));
    L->rgamma = o, o = align256(o + (cl ? slots * 8 : 0));
    L->rswitches = o, o = align256(o + (cl ? slots * 8 : 0));
    L->work = o, o = align256(o + (size_t)p->n_inst * 8);
    L->order = o, o = align256(o + (size_t)p->n_inst * 4);
    L->total = o;
    return true;
}

// ln(1 - exp(-x)) for x > 0, accurate on both sides of ln 2 (Maechler 2012).
double log1mexp(double x) { return x <= 0.6931471805599453 ? std::log(-std::expm1(-x)) : std::log1p(-std::exp(-x)); }

bool ada_ok(const tas_setting &s) {
    return s.policy == TAS_BOOST && !s.table_given && s.ada_beta >= 0.0 && s.ada_beta <= 1.0 &&
           s.ada_gamma_min > 0.0 && s.ada_gamma_max > s.ada_gamma_min &&
           std::isfinite(s.ada_gamma_max) && s.gamma >= s.ada_gamma_min &&
           s.gamma <= s.ada_gamma_max && s.ada_eps_us > 0.0 && std::isfinite(s.ada_eps_us) &&
           s.ada_window >= 1 && s.ada_window <= TAS_ADA_WINDOW_MAX && s.ada_min_samples >= 1 &&
           s.ada_min_samples <= s.ada_window && s.ada_grid >= 2 && s.ada_grid <= TAS_ADA_GRID_MAX;
}

int check_setting(const tas_setting &s, int32_t n_traces, double tau_us, bool has_cached) {
    if (s.trace < 0 || s.trace >= n_traces) return TAS_EINVAL;
    if (s.ada != 0 && (s.ada != 1 || !ada_ok(s))) return TAS_EINVAL;
    if (s.signal != 0 && (s.signal < 1 || s.signal > 2 || s.policy != TAS_BOOST)) return TAS_EINVAL;
    if (s.signal == 2 && !has_cached) return TAS_EINVAL;
    if (s.policy < TAS_FCFS || s.policy > TAS_LTR) return TAS_EINVAL;
    if (s.delta_us < 0) return TAS_EINVAL;
    if (s.policy == TAS_LTR) {
        if (s.ltr_starve < 1 || s.ltr_starve > kLtrMax || s.ltr_quantum < 1 ||
            s.ltr_quantum > kLtrMax)
            return TAS_EINVAL;
    } else if (s.ltr_starve != 0 || s.ltr_quantum != 0) {
        return TAS_EINVAL;
    }
    const bool boosted = s.policy == TAS_BOOST || s.policy == TAS_DIST;
    if (s.policy != TAS_BOOST) {
        if (s.memguard != 0 || s.delta_us != 0) return TAS_EINVAL;
        if (!boosted) return TAS_OK;
    }
    if (s.k < 1 || (s.memguard != 0 && s.memguard != 1)) return TAS_EINVAL;
    if (s.delta_us >= kTwo42) return TAS_EINVAL;
    const int64_t cap = s.policy == TAS_DIST ? kTwo40 : kTwo42;
    if (s.table_given) {
        for (int j = 0; j < TAS_LEVELS; j++) {
            if (s.boost_us[j] < 0 || s.boost_us[j] > cap) return TAS_EINVAL;
            if (j && s.boost_us[j] > s.boost_us[j - 1]) return TAS_EINVAL;
        }
    } else if (!(s.gamma > 0.0) || !std::isfinite(s.gamma)) {
        return TAS_EINVAL;
    } else if (s.policy == TAS_DIST) {
        int64_t bt[TAS_LEVELS];
        if (tas_boost_table(s.gamma, s.k, tau_us, bt) || bt[0] > cap) return TAS_EINVAL;
    }
    return TAS_OK;
}

// The kernel of a pass: one workgroup per instance, or per cluster of
// replicas behind the router.
int launch(const tas::SimArgs &a, int64_t lds_bytes, void *stream) {
    return a.replicas > 1 ? tas_launch_cluster(a, lds_bytes, stream)
                          : tas_launch_sim(a, lds_bytes, stream);
}

}  // namespace

// Device workspace for callers that cannot allocate (tas_create_static): a
// file-scope array of TAS_STATIC_WORKSPACE_BYTES on every GPU the library
// runs on, held until the process ends. Host code never passes the array's
// name to a kernel or a copy: it uses the address hipGetSymbolAddress gives
// on each device.
static __device__ __align__(256) unsigned char scratch[TAS_STATIC_WORKSPACE_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void *scratch_addr[kMaxDevices];  // per device, looked up on its first use

// The device address of `scratch` on the current device.
int scratch_ptr(void **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return TAS_EHIP;
    std::lock_guard<std::mutex> g(scratch_mu);
    if (!scratch_addr[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return TAS_EHIP;
        scratch_addr[dev] = p;
    }
    *out = scratch_addr[dev];
    return TAS_OK;
}

}  // namespace

extern "C" {

int tas_boost_table(double gamma, int32_t k, double tau_us, int64_t *out) {
    if (!out || !(gamma > 0.0) || !std::isfinite(gamma) || k < 1 || !(tau_us > 0.0)) return TAS_EINVAL;
    const double cap = (double)kTwo42;
    for (int j = 0; j < TAS_LEVELS; j++) {
        const double w = (double)k * std::ldexp(1.0, j);  // quantized signal k 2^j
        const double b = -log1mexp(gamma * w) / gamma;     // b_gamma(w) in tokens
        const double us = tau_us * b;
        out[j] = us >= cap ? kTwo42 : (int64_t)std::llround(us);
    }
    return TAS_OK;
}

int tas_ada_grid(const tas_setting *s, double tau_us, double *grid, double *bound,
                 int64_t *tables) {
    if (!s || !grid || !bound || !tables || s->ada != 1 || !ada_ok(*s) || s->k < 1 ||
        !(tau_us > 0.0) || !std::isfinite(tau_us))
        return TAS_EINVAL;
    const int G = s->ada_grid;
    const double lo = s->ada_gamma_min, hi = s->ada_gamma_max;
    for (int j = 0; j < G; j++) grid[j] = lo * std::pow(hi / lo, (double)j / (double)(G - 1));
    for (int j = 0; j + 1 < G; j++) bound[j] = std::sqrt(grid[j] * grid[j + 1]);
    for (int j = 0; j < G; j++)
        if (tas_boost_table(grid[j], s->k, tau_us, tables + (size_t)j * TAS_LEVELS))
            return TAS_EINVAL;
    return TAS_OK;
}

size_t tas_workspace_bytes(const tas_traces *t, const tas_params *p) {
    if (!shape_ok(t) || !p || !engine_ok(p)) return 0;
    int32_t lc, rc, sc;
    bool cp;
    if (!caps(t, p, &lc, &rc, &sc, &cp)) return 0;
    Layout L;
    layout(t, p, rc, sc, &L);
    return L.total;
}

int tas_create_static(const tas_traces *t, const tas_params *p, tas_ctx **out) {
    if (!out) return TAS_EINVAL;
    *out = nullptr;
    const size_t need = tas_workspace_bytes(t, p);
    if (need > TAS_STATIC_WORKSPACE_BYTES) return TAS_ENOMEM;
    void *ws = nullptr;
    if (need > 0) {  // (invalid inputs: tas_create names the error)
        const int rc = scratch_ptr(&ws);
        if (rc) return rc;
    }
    return tas_create(t, p, ws, TAS_STATIC_WORKSPACE_BYTES, out);
}

int tas_create(const tas_traces *t, const tas_params *p, void *d_ws, size_t ws_bytes,
               tas_ctx **out) {
    if (!out) return TAS_EINVAL;
    *out = nullptr;
    if (!shape_ok(t) || !p || !engine_ok(p)) return TAS_EINVAL;
    int32_t lc, rc, sc;
    bool cp;
    if (!caps(t, p, &lc, &rc, &sc, &cp)) return TAS_EINVAL;
    const int32_t N = t->n_req;
    const size_t tn = (size_t)t->n_traces * (size_t)N;
    // traces: sorted, in range; P, D >= 1; P + D < 2^24
    for (size_t i = 0; i < tn; i++) {
        const int64_t a = t->arrival_us[i];
        const int32_t P = t->prompt[i], D = t->decode[i];
        if (a < 0 || a >= kTwo41 || P < 1 || D < 1 || (int64_t)P + D >= (int64_t(1) << 24))
            return TAS_EINVAL;
        if (i % (size_t)N && a < t->arrival_us[i - 1]) return TAS_EINVAL;
        if (t->cached && (t->cached[i] < 0 || t->cached[i] >= P)) return TAS_EINVAL;
    }
    for (int32_t i = 0; i < p->n_inst; i++) {
        int rc = check_setting(p->inst[i], t->n_traces, p->tau_us, t->cached != nullptr);
        if (rc) return rc;
    }
    for (size_t i = 0; i < tn; i++) {
        const int64_t need = ((int64_t)t->prompt[i] + t->decode[i] - 1 + p->block_tokens - 1) /
                             p->block_tokens;
        if (need > p->kv_blocks) return TAS_EINFEASIBLE;
    }
    Layout L;
    layout(t, p, rc, sc, &L);
    if (!d_ws || ws_bytes < L.total || ((uintptr_t)d_ws & 255u)) return TAS_ENOMEM;

    tas_ctx *c = new (std::nothrow) tas_ctx();
    if (!c) return TAS_ENOMEM;
    c->n_traces = t->n_traces, c->n_req = N, c->n_inst = p->n_inst;
    c->list_cap = lc, c->spill_cap = sc, c->retry_cap = rc;
    int32_t wmax;
    const int32_t n_ada = ada_count(p, &wmax);
    c->replicas = replicas_of(p);
    c->lds_bytes = launch_lds(lc, wmax, c->replicas, cp);
    c->lds_retry = launch_lds(rc, wmax, c->replicas, cp);
    c->settings.resize((size_t)p->n_inst);
    c->ada.resize((size_t)n_ada);
    int32_t ai = 0;
    bool ext = n_ada > 0;  // the extended kernel build is needed
    for (int32_t i = 0; i < p->n_inst; i++) {
        const tas_setting &s = p->inst[i];
        tas::DevSetting &d = c->settings[(size_t)i];
        std::memset(&d, 0, sizeof d);
        const bool boosted = s.policy == TAS_BOOST || s.policy == TAS_DIST;
        d.trace = s.trace, d.policy = s.policy, d.k = boosted ? s.k : 1;
        d.memguard = s.policy == TAS_BOOST ? s.memguard : 0;
        d.delta = s.policy == TAS_BOOST ? s.delta_us : 0;
        d.ada = -1;
        d.signal = s.signal;
        d.ltr_s = s.ltr_starve, d.ltr_q = s.ltr_quantum;
        if (s.signal || s.policy == TAS_DIST || s.policy == TAS_SARATHI || s.policy == TAS_LTR)
            ext = true;
        if (boosted) {
            if (s.table_given) std::memcpy(d.bt, s.boost_us, sizeof d.bt);
            else tas_boost_table(s.gamma, s.k, p->tau_us, d.bt);
        }
        if (s.ada) {
            tas::DevAda &A = c->ada[(size_t)ai];
            std::memset(&A, 0, sizeof A);
            double grid[tas::kAdaGridMax];
            tas_ada_grid(&s, p->tau_us, grid, A.bound, &A.table[0][0]);
            for (int j = s.ada_grid - 1; j < tas::kAdaGridMax; j++) A.bound[j] = INFINITY;
            A.beta = s.ada_beta, A.gmin = s.ada_gamma_min, A.gmax = s.ada_gamma_max;
            A.eps = s.ada_eps_us, A.num = p->tau_us * std::log(5.0), A.gamma0 = s.gamma;
            A.window = s.ada_window, A.min_samples = s.ada_min_samples, A.grid = s.ada_grid;
            int cell = 0;  // the grid point nearest gamma0 in log scale
            while (cell + 1 < s.ada_grid && s.gamma >= A.bound[cell]) cell++;
            A.cell0 = cell;
            std::memcpy(d.bt, A.table[cell], sizeof d.bt);
            d.ada = ai++;
        }
    }
    char *ws = (char *)d_ws;
    bool ok = hipMemcpy(ws + L.arrival, t->arrival_us, tn * 8, hipMemcpyHostToDevice) == hipSuccess &&
              hipMemcpy(ws + L.prompt, t->prompt, tn * 4, hipMemcpyHostToDevice) == hipSuccess &&
              hipMemcpy(ws + L.decode, t->decode, tn * 4, hipMemcpyHostToDevice) == hipSuccess;
    if (ok && t->cached)
        ok = hipMemcpy(ws + L.cached, t->cached, tn * 4, hipMemcpyHostToDevice) == hipSuccess;
    if (ok && p->n_inst > 0)
        ok = hipMemcpy(ws + L.settings, c->settings.data(),
                       c->settings.size() * sizeof(tas::DevSetting),
                       hipMemcpyHostToDevice) == hipSuccess;
    if (ok && n_ada > 0)
        ok = hipMemcpy(ws + L.ada, c->ada.data(), c->ada.size() * sizeof(tas::DevAda),
                       hipMemcpyHostToDevice) == hipSuccess;
    if (ok && p->n_inst > 0) {
        // The first launch's order comes from an estimate of each instance's
        // work, in place of the loop steps a launch records for the next
        // one: the requests' minimum iterations in a batch, sum(D + ceil(P /
        // c)) over the trace, weighted 5/4 for policies that re-key every
        // batch member at every token (the list is repaired after each
        // iteration). Sorted longest first, and dealt round robin over the
        // XCDs that take consecutive workgroups, it keeps any one setting of
        // the sweep from landing on a single XCD (as index order does).
        std::vector<int64_t> work((size_t)t->n_traces, 0), est((size_t)p->n_inst);
        for (int32_t tr = 0; tr < t->n_traces; tr++)
            for (int32_t j = 0; j < N; j++) {
                const size_t x = (size_t)tr * (size_t)N + (size_t)j;
                work[(size_t)tr] += t->decode[x] + (t->prompt[x] + p->chunk - 1) / p->chunk;
            }
        for (int32_t i = 0; i < p->n_inst; i++) {
            const int32_t pol = p->inst[i].policy;
            const bool rekey = pol == TAS_SRPT || pol == TAS_TRAIL || pol == TAS_LAS ||
                               pol == TAS_SARATHI;
            est[(size_t)i] = work[(size_t)p->inst[i].trace] * (rekey ? 5 : 4);
        }
        std::vector<int32_t> iota((size_t)p->n_inst);
        for (int32_t i = 0; i < p->n_inst; i++) iota[(size_t)i] = i;
        ok = hipMemcpy(ws + L.order, iota.data(), iota.size() * 4, hipMemcpyHostToDevice) ==
                 hipSuccess &&
             hipMemcpy(ws + L.work, est.data(), est.size() * 8, hipMemcpyHostToDevice) ==
                 hipSuccess;
    }
    // the fixed-gamma kernel build leaves the adaptive outputs alone: zero them
    if (ok && p->n_inst > 0)
        ok = hipMemset(ws + L.gamma, 0, L.spill - L.gamma) == hipSuccess;
    if (!ok) {
        delete c;
        return TAS_EHIP;
    }
    tas::SimArgs &a = c->args;
    a.arrival = (const int64_t *)(ws + L.arrival);
    a.prompt = (const int32_t *)(ws + L.prompt);
    a.decode = (const int32_t *)(ws + L.decode);
    a.cached = t->cached ? (const int32_t *)(ws + L.cached) : nullptr;
    a.inst = (const tas::DevSetting *)(ws + L.settings);
    a.tfirst = (int64_t *)(ws + L.tfirst);
    a.tlast = (int64_t *)(ws + L.tlast);
    a.ttft = (uint32_t *)(ws + L.ttft);
    a.ttlt = (uint32_t *)(ws + L.ttlt);
    a.tbtmax = (uint32_t *)(ws + L.tbtmax);
    a.counters = (int64_t *)(ws + L.counters);
    a.status = (int32_t *)(ws + L.status);
    a.spill = (tas::Rec *)(ws + L.spill);
    a.ovf = (tas::Rec *)(ws + L.ovf);
    a.max_iters = p->max_iters;
    a.n_req = N, a.n_inst = p->n_inst;
    a.M = p->max_seqs, a.T = p->max_tokens, a.c = p->chunk, a.Kb = p->kv_blocks;
    a.bs = p->block_tokens, a.base = p->iter_base_us, a.tok = p->iter_tok_us;
    a.div = p->iter_ctx_div, a.list_cap = lc, a.spill_cap = sc;
    a.div_magic = a.div >= 2 ? ~0ull / (uint64_t)a.div + 1 : 0;
    a.ovf_stride = rc + tas::kStage, a.retry = 0;
    a.ada = (const tas::DevAda *)(ws + L.ada);
    a.gamma_out = (double *)(ws + L.gamma);
    a.switch_out = (int64_t *)(ws + L.switches);
    a.ada_window = wmax;
    a.ext = ext ? 1 : 0;
    a.cp = cp ? 1 : 0;
    a.replicas = c->replicas;
    a.wave_lds = (int32_t)((tas::lds_bytes_for(lc, wmax) + 15) & ~int64_t(15));
    a.jidx = (int32_t *)(ws + L.jidx);
    a.assign = (int32_t *)(ws + L.assign);
    a.rcounters = (int64_t *)(ws + L.rcounters);
    a.rgamma = (double *)(ws + L.rgamma);
    a.rswitches = (int64_t *)(ws + L.rswitches);
    const bool orderable = c->replicas == 1 && p->n_inst <= tas::kMaxOrdered;
    a.order = orderable ? (const int32_t *)(ws + L.order) : nullptr;
    a.work = orderable ? (int64_t *)(ws + L.work) : nullptr;
    c->ordered = orderable;  // the first launch is ordered by the work estimate
    *out = c;
    return TAS_OK;
}


int tas_run(tas_ctx *c, void *stream) {
    if (!c) return TAS_EINVAL;
    c->last_stream = (hipStream_t)stream;
    if (c->ordered && c->args.order &&
        tas_launch_order(c->args.work, const_cast<int32_t *>(c->args.order), c->n_inst, stream))
        return TAS_EHIP;
    if (launch(c->args, c->lds_bytes, stream)) return TAS_EHIP;
    c->ordered = c->args.order != nullptr;
    if (c->retry_cap > c->list_cap) {  // rerun instances that outgrew the small list
        tas::SimArgs a2 = c->args;
        a2.list_cap = c->retry_cap;
        a2.retry = 1;
        a2.wave_lds = (int32_t)((tas::lds_bytes_for(c->retry_cap, c->args.ada_window) + 15) &
                                ~int64_t(15));
        if (launch(a2, c->lds_retry, stream)) return TAS_EHIP;
    }
    return TAS_OK;
}

int tas_percentiles(tas_ctx *c, uint32_t *d_out, void *stream) {
    if (!c || !d_out) return TAS_EINVAL;
    c->last_stream = (hipStream_t)stream;
    return tas_launch_pctl(c->args.ttft, c->args.ttlt, c->args.tbtmax, c->n_inst, c->n_req, d_out,
                           stream)
               ? TAS_EHIP
               : TAS_OK;
}

int tas_percentiles_grouped(tas_ctx *c, int32_t group, uint32_t *d_out, void *stream) {
    if (!c || !d_out || group < 1 || c->n_inst % group != 0 ||
        (int64_t)c->n_req * group > INT32_MAX)
        return TAS_EINVAL;
    c->last_stream = (hipStream_t)stream;
    // the rows of `group` adjacent instances are one contiguous run of values
    return tas_launch_pctl(c->args.ttft, c->args.ttlt, c->args.tbtmax, c->n_inst / group,
                           c->n_req * group, d_out, stream)
               ? TAS_EHIP
               : TAS_OK;
}

int tas_latencies(tas_ctx *c, uint32_t *d_ttft, uint32_t *d_ttlt, uint32_t *d_tbtmax,
                  void *stream) {
    if (!c) return TAS_EINVAL;
    c->last_stream = (hipStream_t)stream;
    const size_t bytes = (size_t)c->n_inst * (size_t)c->n_req * 4;
    const uint32_t *src[3] = {c->args.ttft, c->args.ttlt, c->args.tbtmax};
    uint32_t *dst[3] = {d_ttft, d_ttlt, d_tbtmax};
    for (int m = 0; m < 3; m++)
        if (dst[m] && bytes &&
            hipMemcpyAsync(dst[m], src[m], bytes, hipMemcpyDeviceToDevice,
                           (hipStream_t)stream) != hipSuccess)
            return TAS_EHIP;
    return TAS_OK;
}

int tas_counters(tas_ctx *c, int64_t *d_out, void *stream) {
    if (!c || !d_out) return TAS_EINVAL;
    c->last_stream = (hipStream_t)stream;
    if (c->n_inst == 0) return TAS_OK;
    return hipMemcpyAsync(d_out, c->args.counters, (size_t)c->n_inst * 64,
                          hipMemcpyDeviceToDevice, (hipStream_t)stream) == hipSuccess
               ? TAS_OK
               : TAS_EHIP;
}

int tas_gamma(tas_ctx *c, double *d_gamma, int64_t *d_switches, void *stream) {
    if (!c) return TAS_EINVAL;
    c->last_stream = (hipStream_t)stream;
    if (c->n_inst == 0) return TAS_OK;
    const size_t bytes = (size_t)c->n_inst * 8;
    if (d_gamma && hipMemcpyAsync(d_gamma, c->args.gamma_out, bytes, hipMemcpyDeviceToDevice,
                                  (hipStream_t)stream) != hipSuccess)
        return TAS_EHIP;
    if (d_switches && hipMemcpyAsync(d_switches, c->args.switch_out, bytes,
                                     hipMemcpyDeviceToDevice, (hipStream_t)stream) != hipSuccess)
        return TAS_EHIP;
    return TAS_OK;
}

int tas_replicas(tas_ctx *c, int32_t *d_assign, int64_t *d_counters, double *d_gamma,
                 int64_t *d_switches, void *stream) {
    if (!c || c->replicas < 2) return TAS_EINVAL;
    c->last_stream = (hipStream_t)stream;
    if (c->n_inst == 0) return TAS_OK;
    const hipStream_t s = (hipStream_t)stream;
    const size_t slots = (size_t)c->n_inst * (size_t)c->replicas;
    const size_t na = (size_t)c->n_inst * (size_t)c->n_req * 4;
    if ((d_assign && hipMemcpyAsync(d_assign, c->args.assign, na, hipMemcpyDeviceToDevice, s)) ||
        (d_counters && hipMemcpyAsync(d_counters, c->args.rcounters, slots * 64,
                                      hipMemcpyDeviceToDevice, s)) ||
        (d_gamma && hipMemcpyAsync(d_gamma, c->args.rgamma, slots * 8, hipMemcpyDeviceToDevice, s)) ||
        (d_switches && hipMemcpyAsync(d_switches, c->args.rswitches, slots * 8,
                                      hipMemcpyDeviceToDevice, s)))
        return TAS_EHIP;
    return TAS_OK;
}

int tas_schedule(tas_ctx *c, int64_t *d_work, int32_t *d_order, void *stream) {
    if (!c || !c->args.order) return TAS_EINVAL;
    c->last_stream = (hipStream_t)stream;
    if (c->n_inst == 0) return TAS_OK;
    const hipStream_t s = (hipStream_t)stream;
    const size_t n = (size_t)c->n_inst;
    if ((d_work && hipMemcpyAsync(d_work, c->args.work, n * 8, hipMemcpyDeviceToDevice, s)) ||
        (d_order && hipMemcpyAsync(d_order, c->args.order, n * 4, hipMemcpyDeviceToDevice, s)))
        return TAS_EHIP;
    return TAS_OK;
}

int tas_instance_status(tas_ctx *c, int32_t *d_out, void *stream) {
    if (!c || !d_out) return TAS_EINVAL;
    c->last_stream = (hipStream_t)stream;
    if (c->n_inst == 0) return TAS_OK;
    return hipMemcpyAsync(d_out, c->args.status, (size_t)c->n_inst * 4, hipMemcpyDeviceToDevice,
                          (hipStream_t)stream) == hipSuccess
               ? TAS_OK
               : TAS_EHIP;
}

int tas_status(tas_ctx *c) {
    if (!c) return TAS_EINVAL;
    if (hipStreamSynchronize(c->last_stream) != hipSuccess) return TAS_EHIP;
    if (c->n_inst == 0) return TAS_OK;
    std::vector<int32_t> st((size_t)c->n_inst);
    if (hipMemcpy(st.data(), c->args.status, st.size() * 4, hipMemcpyDeviceToHost) != hipSuccess)
        return TAS_EHIP;
    for (int32_t v : st)
        if (v) return v;
    return TAS_OK;
}

void tas_destroy(tas_ctx *c) { delete c; }

int tas_instance_table(const tas_ctx *c, int32_t inst, int64_t *out) {
    if (!c || !out || inst < 0 || inst >= c->n_inst) return TAS_EINVAL;
    std::memcpy(out, c->settings[(size_t)inst].bt, sizeof(int64_t) * TAS_LEVELS);
    return TAS_OK;
}

int32_t tas_list_cap(const tas_ctx *c) { return c ? c->list_cap : 0; }

const char *tas_strerror(int code) {
    switch (code) {
    case TAS_OK: return "ok";
    case TAS_EINVAL: return "invalid argument";
    case TAS_EINFEASIBLE: return "a request needs more KV blocks than the budget";
    case TAS_ENOMEM: return "workspace too small or misaligned";
    case TAS_EHIP: return "HIP runtime error";
    case TAS_EOVERFLOW: return "a latency exceeds 2^32-1 microseconds";
    case TAS_ELIVELOCK: return "an instance exceeded max_iters";
    case TAS_ESTATE: return "internal consistency check failed";
    case TAS_ECAPACITY: return "an instance outgrew its candidate-list or spill capacity";
    default: return "unknown error";
    }
}

}  // extern "C"
