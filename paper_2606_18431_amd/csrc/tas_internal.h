// tas_internal.h - device-side layouts shared by the host ABI and the kernels.
#pragma once
#include <stdint.h>

namespace tas {

constexpr int kWave = 64;
constexpr int kLevels = 24;
constexpr int kStage = 64;              // staging slots behind the candidate list
constexpr int64_t kKeyOff = int64_t(1) << 42;
constexpr int kIdxBits = 21;            // packed key = (key + 2^42) << 21 | idx
constexpr uint64_t kIdxMask = (uint64_t(1) << kIdxBits) - 1;

constexpr int kAdaGridMax = 64;       // grid points of the adaptive gamma
constexpr int kAdaWindowMax = 2048;   // latencies in its window

// Policy parameters of one instance, as the kernel reads them.
struct DevSetting {
    int32_t trace;
    int32_t policy;
    int32_t k;
    int32_t memguard;
    int64_t delta;
    int64_t bt[kLevels];  // boost in us per MemGuard level (non-increasing);
                          // with adaptive gamma, the table of the first grid cell
    int32_t ada;          // index into SimArgs::ada, or -1
    int32_t signal;       // BOOST: 1 = Algorithm 2's phase-aware signal,
                          // 2 = P - h + dec (expected prefix-cache hits h)
    int32_t ltr_s, ltr_q; // LTR+: starvation threshold and quantum (iterations)
    int32_t pad_;
};

// Adaptive gamma of one instance (host-built): the update constants, the
// grid midpoints (a cell is the number of midpoints <= gamma) and the boost
// table of every grid point.
struct DevAda {
    double beta, gmin, gmax, eps, num;  // num = tau ln 5
    double gamma0;
    int32_t window, min_samples, grid, cell0;
    double bound[kAdaGridMax];          // [grid - 1] midpoints, then +infinity
    int64_t table[kAdaGridMax][kLevels];
};

// A candidate-list record as it is parked in HBM (spilled waiting entries and
// the overflow of a large re-sort). 32 bytes.
struct Rec {
    uint64_t pk;   // packed (key, idx)
    int32_t w;     // signal: prompt + emitted tokens
    int32_t left;  // tokens still to emit
    int32_t kv;    // tokens with resident KV
    uint32_t gs;   // flags, guard, level and this iteration's chunk (see the kernel)
    uint32_t tl;   // time of the last emitted token, modulo 2^32 (us)
    uint32_t gm;   // largest inter-token gap so far (us)
};

struct SimArgs {
    const int64_t *arrival;  // [n_traces][n_req]
    const int32_t *prompt;
    const int32_t *decode;
    const DevSetting *inst;  // [n_inst]
    int64_t *tfirst;         // [n_inst][n_req] absolute time of the first token
    int64_t *tlast;          // [n_inst][n_req] absolute time of the last token
    uint32_t *ttft;          // [n_inst][n_req] outputs, relative to arrival
    uint32_t *ttlt;
    uint32_t *tbtmax;        // written at completion from the on-chip running maximum
    int64_t *counters;       // [n_inst][8]
    int32_t *status;         // [n_inst]
    Rec *spill;              // [n_inst][spill_cap]
    Rec *ovf;                // [n_inst][ovf_stride]
    int64_t max_iters;
    uint64_t div_magic;      // floor((2^64 - 1) / div) + 1 when div >= 2
    int32_t n_req;
    int32_t n_inst;
    int32_t M, T, c, Kb, bs, base, tok, div;
    int32_t list_cap;
    int32_t spill_cap;
    int32_t ovf_stride;  // records per instance in `ovf` (largest list + 64)
    int32_t retry;       // second pass: only instances whose first pass ran out of list
    const DevAda *ada;   // [number of adaptive instances]
    double *gamma_out;   // [n_inst] final adaptive gamma (0 without)
    int64_t *switch_out; // [n_inst] grid-cell changes
    int32_t ada_window;  // largest window over the adaptive instances (LDS), 0 if none
    int32_t ext;         // some instance needs the extended build (adaptive gamma,
                         // the phase-aware or cache-aware signal, DistBoost)
    int32_t cp;          // compact list slots: every request has P + D < 2^16, D <= 2^15
    const int32_t *cached;  // [n_traces][n_req] expected prefix-cache hits, or
                            // null (read by the cache-aware signal only)
    // replicas behind a join-shortest-queue router (cluster_kernel only)
    int32_t replicas;       // waves per workgroup, one replica each
    int32_t wave_lds;       // LDS bytes per replica (16-aligned)
    int32_t *jidx;          // [n_inst][replicas][n_req] global indices per replica
    int32_t *assign;        // [n_inst][n_req] replica of each request
    int64_t *rcounters;     // [n_inst][replicas][8] counters per replica
    double *rgamma;         // [n_inst][replicas] final adaptive gamma (0 without)
    int64_t *rswitches;     // [n_inst][replicas] grid-cell changes
    // launch order: workgroup b simulates instance order[b] (null: b), and
    // each instance's work in loop steps, the next launch's order key (null:
    // not kept)
    const int32_t *order;
    int64_t *work;
};

constexpr int32_t kMaxOrdered = 16384;  // instances the order kernel sorts in LDS

constexpr int kMaxReplicas = 16;
constexpr int64_t kJsqLdsBytes = kMaxReplicas * 4 * 3 + kMaxReplicas * 8 * 8;

// Bytes of the adaptive-gamma block: its state (gamma, gamma_hat, counters),
// then the window in completion order and sorted, 4 bytes per latency each.
constexpr int64_t kAdaStateBytes = 48;
inline int64_t ada_lds_bytes(int32_t window) {
    return window > 0 ? kAdaStateBytes + int64_t(window) * 8 : 0;
}

// LDS bytes per candidate-list slot: the packed key (8 B), the last token
// time and gap maximum (8 B), and the state {gs, w, kv, left} in 16 B, or in
// 8 B with compact slots.
constexpr int64_t kSlotBytes = 8 + 8 + 16;
constexpr int64_t kCompactSlotBytes = 8 + 8 + 8;
constexpr int32_t kCompactMaxPD = (1 << 16) - 1;  // compact slots: P + D <= this
constexpr int32_t kCompactMaxD = 1 << 15;         // and D <= this

// Dynamic LDS bytes per workgroup for a list capacity, the largest
// adaptive-gamma window (0: none) and the slot layout.
inline int64_t lds_bytes_for(int32_t list_cap, int32_t ada_window = 0, bool compact = false) {
    const int64_t cap = int64_t(list_cap) + kStage;  // the list and its overflow region
    // the slots; alignment of the boost table; the boost table; the
    // adaptive-gamma block
    return cap * (compact ? kCompactSlotBytes : kSlotBytes) + 8 + kLevels * 8 +
           ada_lds_bytes(ada_window);
}
constexpr int kMaxChunk = (1 << 15) - 1;  // the chunk size lives in 15 bits of the flag word
// At most 64 chunks of 64 entries (list + overflow region): chunk bitmaps are
// 64-bit and per-chunk masks live one chunk per lane.
constexpr int kMaxListCap = 64 * 64 - kStage;

}  // namespace tas

// Launchers implemented next to the kernels.
int tas_launch_sim(const tas::SimArgs &a, int64_t lds_bytes, void *stream);
int tas_launch_cluster(const tas::SimArgs &a, int64_t lds_bytes, void *stream);
int tas_launch_order(const int64_t *work, int32_t *order, int32_t n, void *stream);
int tas_launch_pctl(const uint32_t *ttft, const uint32_t *ttlt, const uint32_t *tbtmax,
                    int32_t n_inst, int32_t n_req, uint32_t *out, void *stream);
