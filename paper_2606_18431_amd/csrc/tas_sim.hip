// tas_sim.hip - the iteration-level serving simulation, one wavefront per
// instance (one trace x one policy setting), for gfx950.
//
// What each iteration computes (arXiv 2606.18431, Algorithm 1; Phase 2
// unified key and hysteresis; Phase 3 MemGuard; Phase 4 adaptive gamma):
//   0. with adaptive gamma, gamma follows the tail of the recent end-to-end
//      latencies, and the boost table that of its nearest grid point;
//   1. arrivals with a_i <= t join the waiting set;
//   2. every waiting or resident request has a key; candidates are taken in
//      ascending (key, idx) order;
//   3. greedy batch formation under max_seqs, max_tokens and the KV budget;
//      when the KV budget is exceeded the worst eligible resident outside the
//      batch is evicted (recompute preemption); a resident candidate with no
//      eligible victim forces out the worst other resident or itself; a
//      waiting candidate that does not fit closes admissions;
//   4. the step costs base + tok*sum(n) + floor(sum(kv+n)/div) us; tokens are
//      emitted, first/last token times and the max inter-token gap recorded.
//
// Design (MI355X): instances are independent, so one 64-lane wavefront owns
// one instance and needs no workgroup barrier. The active requests live in
// LDS as one array sorted by the packed key (key + 2^42) << 21 | idx, with
// their state in structure-of-arrays form, so the batch-formation pass is a
// sequence of 64-wide chunks with DPP prefix sums (token budget, KV blocks,
// sequence count) and a ballot to find the first candidate that does not
// fit; only that candidate takes the sequential eviction path. Keys of
// waiting requests never change (MemGuard recomputes a key only when the
// quantized signal moves, Phase 3), so the list is repaired incrementally:
// finished entries stay behind as holes until a compaction pass, entries whose
// key moved are extracted and merged back. Waiting requests beyond the
// on-chip capacity spill to HBM with the invariant that every spilled key
// exceeds every waiting key on chip; a radix select over the spill refills
// the list.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tas_internal.h"

namespace tas {
namespace {

#define DEV __device__ __forceinline__

// The checking build (a library of its own, compiled with
// TAS_CHECK_INVARIANTS=1) verifies the state of every instance after each
// iteration and fails the instance with S_ESTATE at the first violation;
// its results are otherwise those of the ordinary build.
#ifndef TAS_CHECK_INVARIANTS
#define TAS_CHECK_INVARIANTS 0
#endif
constexpr bool kCheck = TAS_CHECK_INVARIANTS != 0;
#define UNLIKELY(x) __builtin_expect(!!(x), 0)
#define LIKELY(x) __builtin_expect(!!(x), 1)

// record flag word (gs)
constexpr uint32_t G_GUARD = 0x1fu;      // MemGuard level at the latest dispatch
constexpr uint32_t G_RES = 1u << 5;      // resident: holds KV
constexpr uint32_t G_FIRST = 1u << 6;    // first token emitted
constexpr uint32_t G_INB = 1u << 7;      // in this iteration's batch
constexpr uint32_t G_EVI = 1u << 8;      // evicted during this iteration
constexpr uint32_t G_DONE = 1u << 9;     // completed: a hole until compaction
constexpr uint32_t G_DIRTY = 1u << 10;   // key moved: re-insert
constexpr uint32_t G_MARK = 1u << 11;    // selected for spilling
constexpr int G_LVL_SHIFT = 12;          // current MemGuard level (5 bits)
constexpr uint32_t G_LVL = 0x1fu << G_LVL_SHIFT;
constexpr uint32_t G_FLAGS = 0x1ffffu;   // the flags and levels: bits 0..16
constexpr int kLeftShift = 17;           // compact slots: left - 1 in bits 17..31
// LTR+ (which has no MemGuard level, and never uses compact slots): the
// level's lowest bit marks a promoted request, bits 17..31 hold its
// starvation count, or while promoted the quantum left
constexpr uint32_t G_PROMO = 1u << G_LVL_SHIFT;
constexpr int kLtrShift = 17;
constexpr int kHoleLimit = 16;           // compact once this many holes accumulate

enum { S_OK = 0, S_EOVERFLOW = -5, S_ELIVELOCK = -6, S_ESTATE = -7, S_ECAPACITY = -8 };
// Policies: the paper's boosted priority (BOOST), its comparators FCFS and
// oracle-length SRPT, and the further comparison policies of its Table 1 and
// evaluation baselines: shortest prompt first (SPF), shortest job first with
// perfect output-length knowledge (SJF), least attained service (LAS) and
// SRPT with TRAIL's swap-prevention threshold (TRAIL); and the Phase 1
// strawman DistBoost (DIST).
enum { P_FCFS = 0, P_SRPT = 1, P_BOOST = 2, P_SPF = 3, P_SJF = 4, P_LAS = 5, P_TRAIL = 6,
       P_DIST = 7, P_SARATHI = 8, P_LTR = 9 };
// LTR+ ranks a promoted request ahead of every unpromoted one (SJF keys are
// D >= 1): key j - 2^42 for a promotion at the end of iteration j.
constexpr int64_t kPromotedOff = int64_t(1) << 42;
// DistBoost ranks its decode queue (key: the time a request entered it, its
// first-token time) ahead of its prefill queue: decode keys are shifted down
// by 2^42, below every prefill key a - bt (boost tables are capped at 2^40).
constexpr int64_t kDecodeQueueOff = int64_t(1) << 42;

// ------------------------------------------------------------ wave helpers

DEV int lane() { return (int)__lane_id(); }
DEV uint64_t ballot(bool p) { return (uint64_t)__ballot(p); }
DEV int popc(uint64_t m) { return __popcll(m); }
DEV int ffs0(uint64_t m) { return __ffsll((unsigned long long)m) - 1; }
DEV int fls0(uint64_t m) { return 63 - __clzll((unsigned long long)m); }
DEV int mbcnt(uint64_t m) {
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                          __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}
DEV int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }
DEV int rl(int x, int l) { return __builtin_amdgcn_readlane(x, l); }
DEV uint64_t rlu(uint64_t x, int l) {
    uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)x, l);
    uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(x >> 32), l);
    return ((uint64_t)hi << 32) | lo;
}
DEV int64_t rl64(int64_t x, int l) { return (int64_t)rlu((uint64_t)x, l); }
DEV uint64_t uniu(uint64_t x) { return rlu(x, __builtin_amdgcn_readfirstlane(lane())); }
// One wavefront is the whole workgroup and its LDS operations execute in
// issue order, so ordering LDS traffic between lanes only needs the compiler
// not to move memory operations across this point.
DEV void wsync() { __asm__ volatile("" ::: "memory"); }
// Before reading back HBM this wavefront wrote (spill, overflow, timestamps).
DEV void hbm_fence() { __builtin_amdgcn_s_waitcnt(0); __asm__ volatile("" ::: "memory"); }

// DPP lane moves (GFX9 encodings): row_shr:n shifts within 16-lane rows,
// row_bcast:15 / :31 carry a row's last lane into the next row(s), wave_shr:1
// shifts across the whole wavefront. Disabled or out-of-range lanes take `old`.
constexpr int kShr1 = 0x111, kShr2 = 0x112, kShr4 = 0x114, kShr8 = 0x118;
constexpr int kBc15 = 0x142, kBc31 = 0x143, kWShr1 = 0x138;

template <int CTRL, int RM = 0xf>
DEV int dpp(int old, int x) {
    return __builtin_amdgcn_update_dpp(old, x, CTRL, RM, 0xf, false);
}
template <int CTRL, int RM = 0xf>
DEV uint64_t dppu(uint64_t old, uint64_t x) {
    const uint32_t lo = (uint32_t)dpp<CTRL, RM>((int)(uint32_t)old, (int)(uint32_t)x);
    const uint32_t hi = (uint32_t)dpp<CTRL, RM>((int)(uint32_t)(old >> 32), (int)(uint32_t)(x >> 32));
    return ((uint64_t)hi << 32) | lo;
}

// inclusive prefix sum over the wavefront
DEV int scan_add(int x) {
    x += dpp<kShr1>(0, x);
    x += dpp<kShr2>(0, x);
    x += dpp<kShr4>(0, x);
    x += dpp<kShr8>(0, x);
    x += dpp<kBc15, 0xa>(0, x);
    x += dpp<kBc31, 0xc>(0, x);
    return x;
}
DEV int wsum(int x) { return rl(scan_add(x), 63); }
DEV int wmin(int x) {
    x = min(x, dpp<kShr1>(INT32_MAX, x));
    x = min(x, dpp<kShr2>(INT32_MAX, x));
    x = min(x, dpp<kShr4>(INT32_MAX, x));
    x = min(x, dpp<kShr8>(INT32_MAX, x));
    x = min(x, dpp<kBc15, 0xa>(INT32_MAX, x));
    x = min(x, dpp<kBc31, 0xc>(INT32_MAX, x));
    return rl(x, 63);
}
DEV uint64_t scan_maxu(uint64_t x) {
    uint64_t y;
    y = dppu<kShr1>(0ull, x), x = y > x ? y : x;
    y = dppu<kShr2>(0ull, x), x = y > x ? y : x;
    y = dppu<kShr4>(0ull, x), x = y > x ? y : x;
    y = dppu<kShr8>(0ull, x), x = y > x ? y : x;
    y = dppu<kBc15, 0xa>(0ull, x), x = y > x ? y : x;
    y = dppu<kBc31, 0xc>(0ull, x), x = y > x ? y : x;
    return x;
}
DEV uint64_t scan_minu(uint64_t x) {
    uint64_t y;
    y = dppu<kShr1>(~0ull, x), x = y < x ? y : x;
    y = dppu<kShr2>(~0ull, x), x = y < x ? y : x;
    y = dppu<kShr4>(~0ull, x), x = y < x ? y : x;
    y = dppu<kShr8>(~0ull, x), x = y < x ? y : x;
    y = dppu<kBc15, 0xa>(~0ull, x), x = y < x ? y : x;
    y = dppu<kBc31, 0xc>(~0ull, x), x = y < x ? y : x;
    return x;
}
DEV uint64_t wminu(uint64_t x) { return rlu(scan_minu(x), 63); }
// the value of the previous lane (lane 0 gets `fill`)
DEV uint64_t prev_lane_u64(uint64_t x, uint64_t fill) { return dppu<kWShr1>(fill, x); }

// ------------------------------------------------------------ keys

DEV uint64_t pack(int64_t key, int idx) {
    return ((uint64_t)(key + kKeyOff) << kIdxBits) | (uint64_t)(uint32_t)idx;
}
DEV int64_t key_of(uint64_t pk) { return (int64_t)(pk >> kIdxBits) - kKeyOff; }
DEV int idx_of(uint64_t pk) { return (int)(pk & kIdxMask); }

// MemGuard level floor(log2(max(w,k)/k)) capped at 23, without a division:
// with e = floor(log2 w) - floor(log2 k), the level is e when w >= k 2^e and
// e - 1 otherwise (Eq. memguard_level). Branch-free (lanes with w < k take 0
// by a select), so a wave evaluates it without splitting.
DEV int level_of(int w, int k, int lk) {
    const int e = (31 - __clz(w | 1)) - lk;
    const int L = ((w >> (e & 31)) >= k) ? e : e - 1;
    return w < k ? 0 : (L < kLevels - 1 ? L : kLevels - 1);
}

// ------------------------------------------------------------ LDS layout

// LDS holds the candidate list as three parallel arrays: the slot state
// {gs, w, kv, left} (what formation reads, one load per lane), the packed
// key (searches and merges) and the pair {tl, gm} of the last token time and
// the largest inter-token gap so far (emission only). The gap maximum stays
// on chip until the request completes, so the per-token work touches no HBM.
// The slot state takes 16 bytes, or 8 in the compact layout used when every
// request has P + D < 2^16 and D <= 2^15: w and kv in 16 bits each, left - 1
// in the flag word's bits 17..31 (the flags use bits 0..16). An entry is then
// 24 bytes instead of 32, which lets 16 instead of 12 instances share a
// compute unit's LDS at the large sweep's list size.
struct Lds {
    uint4 *q;   // four-word slots
    uint2 *q2;  // compact slots
    uint64_t *k;
    uint2 *tg;
    int64_t *bt;
    struct AdaLds *as;  // adaptive gamma: state, then the window in completion
    uint32_t *wr, *ws;  // order (a ring) and sorted
};

// Adaptive-gamma state of one instance (LDS, written by lane 0).
struct AdaLds {
    double gamma, ghat;      // current gamma, latest estimate
    int32_t wn, whead;       // latencies in the window, ring slot of the oldest
    int32_t cell, wnew;      // grid cell in use; 1: the window changed since ghat
    int64_t switches;        // grid-cell changes
    int32_t window, min_samples;
};
static_assert(sizeof(AdaLds) == kAdaStateBytes, "adaptive-gamma LDS block");

struct R {  // one candidate-list record in registers
    uint64_t pk = 0;
    int w = 0, left = 0, kv = 0;
    uint32_t gs = 0, tl = 0, gm = 0;
};

DEV R from_rec(const Rec &r) {
    R x;
    x.pk = r.pk, x.w = r.w, x.left = r.left, x.kv = r.kv, x.gs = r.gs, x.tl = r.tl, x.gm = r.gm;
    return x;
}
DEV Rec to_rec(const R &x) {
    Rec r;
    r.pk = x.pk, r.w = x.w, r.left = x.left, r.kv = x.kv, r.gs = x.gs, r.tl = x.tl, r.gm = x.gm;
    return r;
}
DEV R shfl_rec(const R &x, int src) {
    R y;
    y.pk = (uint64_t)__shfl((unsigned long long)x.pk, src);
    y.w = __shfl(x.w, src);
    y.left = __shfl(x.left, src);
    y.kv = __shfl(x.kv, src);
    y.gs = (uint32_t)__shfl((int)x.gs, src);
    y.tl = (uint32_t)__shfl((int)x.tl, src);
    y.gm = (uint32_t)__shfl((int)x.gm, src);
    return y;
}
DEV bool is_waiting(uint32_t g) { return (g & (G_RES | G_DONE)) == 0; }

// Destination lanes of a wavefront permutation: the lanes in m go, in order,
// to lanes base, base + 1, ...; the other lanes fill the remaining slots in
// order. Requires base + popc(m) <= 64.
DEV int place_dest(uint64_t m, int base) {
    const int before = mbcnt(m);
    if ((m >> lane()) & 1ull) return base + before;
    const int k = lane() - before;  // rank among the lanes outside m
    return k < base ? k : k + popc(m);
}
DEV uint32_t perm32(int dest, uint32_t v) {
    return (uint32_t)__builtin_amdgcn_ds_permute(dest * 4, (int)v);
}
// Move a record across lanes (a register transpose: no LDS storage is used).
// Every lane must be active, and dest must be a permutation.
DEV R permute_rec(const R &x, int dest) {
    R y;
    const uint32_t lo = perm32(dest, (uint32_t)x.pk), hi = perm32(dest, (uint32_t)(x.pk >> 32));
    y.pk = ((uint64_t)hi << 32) | lo;
    y.w = (int)perm32(dest, (uint32_t)x.w);
    y.left = (int)perm32(dest, (uint32_t)x.left);
    y.kv = (int)perm32(dest, (uint32_t)x.kv);
    y.gs = perm32(dest, x.gs);
    y.tl = perm32(dest, x.tl);
    y.gm = perm32(dest, x.gm);
    return y;
}

// ------------------------------------------------------------ the simulator

// BSH: log2 of the KV block size when it is a power of two (the common
// 16-token block gets its own instantiation), -1 otherwise. The policy is a
// run-time value: one copy of the code serves every policy, so workgroups of
// different policies on one compute unit share the instruction cache.
// CL: one replica of a cluster behind a join-shortest-queue router; its
// arrivals are the global requests the router has dispatched to it so far.
// CP: compact slots (see Lds).
template <int BSH, bool EXT, bool CL = false, bool CP = false>
struct Sim {
    const SimArgs &A;
    Lds S;
    // instance constants (memguard and delta are zero unless pol is BOOST)
    int inst, N, M, T, c, Kb, bs, base, tok, div, pol, k, lk, memguard, lcap, scap;
    int ltr_s, ltr_q;  // LTR+: starvation threshold and quantum (iterations)
    int64_t delta, max_iters;
    uint64_t div_magic;  // ceil(2^64 / div) for div >= 2
    const int64_t *arr;
    const int32_t *Pp, *Dp;
    int64_t *tfirst, *tlast;
    uint32_t *tbo;  // the instance's max-gap outputs, written at completion
    Rec *spill, *ovf;
    // state
    int64_t t;
    int U, L, nW, nR, n_holes, lo_hole, spill_n, next, pf, completed, status;
    uint64_t spill_min;
    int64_t pa;
    int pP, pD;
    int64_t iters, reqiters, tokens, ev_vol, ev_forced, maxU, idle;
    // loop steps for the launch-order key: formation passes and emission
    // chunks (32-bit: a wrap only perturbs the order of a huge instance)
    uint32_t fpass, echunks;
    // CL: the replica (wave) index, the global indices dispatched to it in
    // order (HBM, written and read by this wave only, through L2), how many,
    // the prefetched global index of each lane, and the completions of the
    // latest iteration
    int wv, Nk, pidx, last_done;
    int32_t *jl;
    // per-iteration formation results
    int cnt, used;
    int64_t sum_ctx;
    uint64_t emit_chunks;  // 64-entry chunks holding batch members or evictions
    bool emit_all;         // ranks moved during formation: visit every chunk
    // Repeated batch: the next iteration's formation would select every
    // resident with one token each and nothing else (see run), so it is
    // skipped. Emission reports whether every batch member emitted a token
    // and how many new KV blocks the members need for their next token.
    bool rep, all_emit;
    int du_next;
    int nmoved;  // entries whose key the latest emission moved
    // the key of the waiting candidate that closed admissions in the latest
    // formation (~0: none), the smallest key of the arrivals taken since
    // (~0: none) and a count of spill_excess calls
    uint64_t close_pk, arr_min_pk;
    int n_spilled;
    // victim masks, lane c = chunk c: residents, and those a voluntary
    // eviction may take (MemGuard). Kept across iterations: bits change in
    // place on admission, eviction and completion; any edit that moves ranks
    // clears vm_ok and the next victim search rebuilds them.
    uint64_t vm_res, vm_ev;
    bool vm_ok;
    // adaptive gamma (null without): constants, and lane j < grid - 1 holds
    // the midpoint above grid point j (+infinity beyond)
    const DevAda *ad;
    double bnd;
    bool phase_signal;  // BOOST with Algorithm 2's signal: P in prefill, dec after
    bool cache_signal;  // BOOST with the cache-aware signal P - h + dec
    const int32_t *Hp;  // expected prefix-cache hits of the trace (cache_signal)

    DEV Sim(const SimArgs &a, const DevSetting &st, int i, unsigned char *smem, int w = 0) : A(a) {
        inst = i;
        N = a.n_req, M = a.M, T = a.T, c = a.c, Kb = a.Kb, bs = a.bs;
        base = a.base, tok = a.tok, div = a.div, lcap = a.list_cap, scap = a.spill_cap;
        k = st.k > 0 ? st.k : 1;
        lk = 31 - __clz(k);
        pol = st.policy;
        ltr_s = st.ltr_s, ltr_q = st.ltr_q;
        memguard = st.memguard;
        delta = st.delta;
        max_iters = a.max_iters;
        div_magic = a.div_magic;
        const size_t toff = (size_t)st.trace * (size_t)N;
        arr = a.arrival + toff, Pp = a.prompt + toff, Dp = a.decode + toff;
        const size_t ioff = (size_t)i * (size_t)N;
        tfirst = a.tfirst + ioff, tlast = a.tlast + ioff, tbo = a.tbtmax + ioff;
        wv = w, Nk = 0, pidx = 0, last_done = 0;
        jl = nullptr;
        const size_t slot = CL ? (size_t)i * (size_t)a.replicas + (size_t)w : (size_t)i;
        spill = a.spill + slot * (size_t)scap;
        ovf = a.ovf + slot * (size_t)a.ovf_stride;
        if constexpr (CL) jl = a.jidx + slot * (size_t)N;
        const int cap = lcap + kStage;  // the list may use its overflow region during formation
        size_t o = 0;
        S.q = nullptr, S.q2 = nullptr;
        if constexpr (CP) S.q2 = (uint2 *)(smem + o), o += (size_t)cap * 8;
        else S.q = (uint4 *)(smem + o), o += (size_t)cap * 16;
        S.k = (uint64_t *)(smem + o), o += (size_t)cap * 8;
        S.tg = (uint2 *)(smem + o), o += (size_t)cap * 8;
        S.bt = (int64_t *)(smem + o), o += (size_t)kLevels * 8;
        for (int j = lane(); j < kLevels; j += kWave) S.bt[j] = st.bt[j];
        ad = nullptr;
        bnd = 0.0;
        phase_signal = EXT && st.signal == 1;
        cache_signal = EXT && st.signal == 2;
        Hp = cache_signal ? a.cached + toff : nullptr;
        if constexpr (EXT) {
            S.as = (AdaLds *)(smem + o), o += kAdaStateBytes;
            S.wr = (uint32_t *)(smem + o), o += (size_t)a.ada_window * 4;
            S.ws = (uint32_t *)(smem + o);
            ad = st.ada >= 0 ? a.ada + st.ada : nullptr;
        }
        if (EXT && ad) {  // the table of the first cell is st.bt
            bnd = ad->bound[lane()];
            if (lane() == 0) {
                AdaLds &G = *S.as;
                G.gamma = ad->gamma0, G.ghat = 0.0;
                G.wn = G.whead = G.wnew = 0;
                G.cell = ad->cell0;
                G.switches = 0;
                G.window = ad->window, G.min_samples = ad->min_samples;
            }
        }
        t = 0;
        U = L = nW = nR = n_holes = spill_n = next = pf = completed = status = 0;
        lo_hole = INT32_MAX;
        spill_min = ~0ull;
        iters = reqiters = tokens = ev_vol = ev_forced = maxU = idle = 0;
        fpass = echunks = 0;
        cnt = used = 0;
        sum_ctx = 0;
        emit_chunks = 0;
        emit_all = false;
        rep = all_emit = false;
        du_next = 0;
        nmoved = 0;
        close_pk = arr_min_pk = ~0ull;
        n_spilled = 0;
        vm_res = vm_ev = 0;
        vm_ok = false;
        wsync();
    }

    DEV void fail(int code) {
        if (status == 0) status = code;
    }

    // ---------------------------------------------------------- slots

    // The state of slot i as loaded: the flag word in .x (compact: with
    // left - 1 above the flags), the rest unpacked by sw / skv / sleft.
    DEV uint4 ldq(int i) const {
        if constexpr (CP) {
            const uint2 v = S.q2[i];
            return make_uint4(v.x, v.y, 0u, 0u);
        } else {
            return S.q[i];
        }
    }
    DEV int sw(const uint4 &v) const { return CP ? (int)(v.y & 0xffffu) : (int)v.y; }
    DEV int skv(const uint4 &v) const { return CP ? (int)(v.y >> 16) : (int)v.z; }
    DEV int sleft(const uint4 &v) const {
        return CP ? (int)(v.x >> kLeftShift) + 1 : (int)v.w;
    }
    DEV void stq(int i, uint32_t x, int w, int kv, int left) const {
        if constexpr (CP) {
            S.q2[i] = make_uint2((x & G_FLAGS) | ((uint32_t)(left - 1) << kLeftShift),
                                 (uint32_t)w | ((uint32_t)kv << 16));
        } else {
            S.q[i] = make_uint4(x, (uint32_t)w, (uint32_t)kv, (uint32_t)left);
        }
    }
    // the flag word alone (flag edits keep the compact layout's left bits)
    DEV uint32_t ldx(int i) const { return CP ? S.q2[i].x : S.q[i].x; }
    DEV void stx(int i, uint32_t x) const {
        if constexpr (CP) S.q2[i].x = x;
        else S.q[i].x = x;
    }
    // the flag word (as loaded, flags edited) and kv of a slot whose w is w
    DEV void stxkv(int i, uint32_t x, int w, int kv) const {
        if constexpr (CP) {
            S.q2[i] = make_uint2(x, (uint32_t)w | ((uint32_t)kv << 16));
        } else {
            S.q[i].x = x;
            S.q[i].z = (uint32_t)kv;
        }
    }
    DEV void ldr(int i, R &x) const {
        const uint4 q = ldq(i);
        x.gs = q.x, x.w = sw(q), x.kv = skv(q), x.left = sleft(q);
        x.pk = S.k[i];
        const uint2 tg = S.tg[i];
        x.tl = tg.x, x.gm = tg.y;
    }
    DEV void str(int i, const R &x) const {
        stq(i, x.gs, x.w, x.kv, x.left);
        S.k[i] = x.pk;
        S.tg[i] = make_uint2(x.tl, x.gm);
    }
    // Entries the list keeps before spilling waiting ones. The adaptive build
    // sizes the waiting window from the residents (max(M, residents) + 128,
    // within lcap): its grid changes let residents outside the batch pile up,
    // and a list padded with waiting entries costs every pass over it.
    DEV int cap_now() const {
        if constexpr (EXT) {
            if (pol == P_LTR) return lcap;  // LTR+ keeps every request on chip
            return min(lcap, max(M, nR) + 128);
        } else {
            return lcap;
        }
    }
    // floor(s / div). Below 2^32 a multiply by the rounded-up reciprocal is
    // exact: s * ceil(2^64/div) / 2^64 exceeds s/div by less than 2^-32 <= 1/div.
    DEV uint64_t ctx_quot(uint64_t s) const {
        if (div == 1) return s;
        if (s >> 32) return s / (uint64_t)div;
        const uint32_t x = (uint32_t)s;
        return ((uint64_t)x * (div_magic >> 32) + __umulhi(x, (uint32_t)div_magic)) >> 32;
    }
    DEV int blocks(int x) const {
        if constexpr (BSH >= 0) {
            return (x + (1 << BSH) - 1) >> BSH;
        } else {
            return (x + bs - 1) / bs;
        }
    }

    // ---------------------------------------------------------- arrivals

    // requests this instance (replica) may take: the trace, or those
    // dispatched to the replica so far
    DEV int n_known() const { return CL ? Nk : N; }

    DEV void load_pf() {
        const int r = pf + lane();
        if (r < n_known()) {
            if constexpr (CL) {
                pidx = __hip_atomic_load(&jl[r], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                pa = arr[pidx], pP = Pp[pidx], pD = Dp[pidx];
            } else {
                pa = arr[r], pP = Pp[r], pD = Dp[r];
            }
        } else {
            pa = INT64_MAX, pP = 1, pD = 1;
            if constexpr (CL) pidx = 0;
        }
    }

    DEV R new_record(int idx, int64_t a, int P, int D) const {
        R x;
        x.w = P, x.left = D;
        int64_t key;
        uint32_t lvl = 0;
        if (pol == P_FCFS || (EXT && pol == P_SARATHI)) {
            key = a;  // Sarathi: prefills wait in arrival order
        } else if (pol == P_SRPT || pol == P_TRAIL) {
            key = (int64_t)P + D - 1;  // remaining computed tokens
        } else if (pol == P_SPF || pol == P_LAS) {
            key = P;  // prompt length; the attained service P + dec at dec = 0
        } else if (pol == P_SJF || (EXT && pol == P_LTR)) {
            key = D;  // output length (LTR+: until a promotion)
        } else {
            int sig = P;  // the signal before the first token
            if constexpr (EXT) {
                // cached tokens are not work (lanes past the trace hold no request)
                if (cache_signal && idx < N) sig = P - Hp[idx];
            }
            lvl = (uint32_t)level_of(sig, k, lk);
            key = a - S.bt[lvl];
        }
        x.gs = lvl << G_LVL_SHIFT;
        x.pk = pack(key, idx);
        return x;
    }

    // Arrivals with a <= t join the waiting set, up to 64 per round.
    DEV void take_arrivals() {
        for (int round = 0; round <= (N >> 6) + 1 && status == 0; round++) {
            int off = next - pf;
            if (off >= kWave) {
                pf = next;
                load_pf();
                off = 0;
            }
            const int r = pf + lane();
            const bool arrive = lane() >= off && r < n_known() && pa <= t;
            const int n_arr = popc(ballot(arrive));
            if (LIKELY(n_arr == 0)) return;
            const R x = new_record(CL ? pidx : r, pa, pP, pD);
            const R y = off ? shfl_rec(x, min(off + lane(), kWave - 1)) : x;
            if constexpr (!CL && !EXT)
                arr_min_pk = min(arr_min_pk, wminu(lane() < n_arr ? y.pk : ~0ull));
            nW += n_arr;
            next += n_arr;
            add_entries(y, n_arr);
            if (off + n_arr < kWave) return;
        }
    }

    // ---------------------------------------------------------- list edits

    // Number of list entries with pk < x (x wave-uniform): the last key of
    // every 64-entry chunk, then one chunk. Requires L <= 64 * 64.
    DEV int lower_bound(uint64_t x) const {
        if (L == 0) return 0;
        const int nch = (L + kWave - 1) >> 6;
        const int probe = min(lane() * kWave + kWave - 1, L - 1);
        const uint64_t cm = lane() < nch ? S.k[probe] : ~0ull;
        const int c0 = popc(ballot(lane() < nch && cm < x));
        if (c0 >= nch) return L;
        const int r = c0 * kWave + lane();
        const uint64_t v = r < L ? S.k[r] : ~0ull;
        return c0 * kWave + popc(ballot(r < L && v < x));
    }

    // Merge K records held by lanes [0, K) into the sorted list.
    // Requires L + K <= lcap + kStage (the list's overflow region).
    DEV void merge_new(const R &x, int K) {
        if (K <= 0) return;
        const bool act = lane() < K;
        int rn = 0;
        for (int j = 0; j < K; j++) rn += (act && rlu(x.pk, j) < x.pk) ? 1 : 0;
        const uint64_t xmin = wminu(act ? x.pk : ~0ull);
        const int minpos = lower_bound(xmin);
        int pos_in = 0;  // lane j < K: list entries at ranks >= minpos smaller than x_j
        if (minpos < L) {
            for (int b = ((L - 1) >> 6) << 6; b >= 0 && b + kWave > minpos; b -= kWave) {
                const int r = b + lane();
                const bool mv = r >= minpos && r < L;
                const uint64_t pr = mv ? S.k[r] : ~0ull;
                int sh = 0;
                for (int j = 0; j < K; j++) {
                    const uint64_t xj = rlu(x.pk, j);
                    sh += (mv && xj < pr) ? 1 : 0;
                    const int cj = popc(ballot(mv && pr < xj));
                    if (lane() == j) pos_in += cj;
                }
                const bool go = mv && sh > 0;
                if (ballot(go)) vm_ok = false;
                R y;
                if (go) ldr(r, y);
                wsync();
                if (go) str(r + sh, y);
                wsync();
            }
        }
        if (act) str(minpos + pos_in + rn, x);
        wsync();
        L += K;
    }

    // Remove the entries whose flags intersect `mask`, from rank `from` on.
    DEV void compact_remove(int from, uint32_t mask) {
        vm_ok = false;
        int out = from;
        for (int b = (from >> 6) << 6; b < L; b += kWave) {
            const int r = b + lane();
            const bool v = r >= from && r < L;
            R y;
            if (v) ldr(r, y);
            const bool keep = v && !(y.gs & mask);
            const uint64_t km = ballot(keep);
            wsync();
            if (keep) {
                const int d = out + mbcnt(km);
                if (d != r) str(d, y);
            }
            wsync();
            out += popc(km);
        }
        L = out;
    }

    DEV void drop_holes() {
        if (n_holes == 0) return;
        compact_remove(lo_hole, G_DONE);
        n_holes = 0;
        lo_hole = INT32_MAX;
    }

    // Keep at most cap_now() entries: drop holes, then spill the largest
    // waiting entries to HBM.
    DEV void spill_excess() {
        const int cap = cap_now();
        if (L <= cap) return;
        drop_holes();
        const int E = L - cap;
        if (E <= 0) return;
        n_spilled++;
        if (EXT && pol == P_LTR) {
            // a spilled request's starvation count would have to advance in
            // HBM every iteration: an LTR+ instance keeps every request on
            // chip, and one that outgrows the list reruns with a larger one
            fail(S_ECAPACITY);
            return;
        }
        if (spill_n + E > scap) {
            fail(S_ECAPACITY);
            return;
        }
        int found = 0, lowest = L;
        for (int b = ((L - 1) >> 6) << 6; b >= 0 && found < E; b -= kWave) {
            const int r = b + lane();
            const bool isw = r < L && is_waiting(ldx(r));
            const uint64_t m = ballot(isw);
            const int above = popc(m) - mbcnt(m) - 1;
            const bool take = isw && above < E - found;
            if (take) {
                R y;
                ldr(r, y);
                spill[spill_n + found + above] = to_rec(y);
                stx(r, y.gs | G_MARK);
            }
            const uint64_t tm = ballot(take);
            found += popc(tm);
            if (tm) lowest = b + ffs0(tm);
        }
        wsync();
        if (found < E) {
            fail(S_ECAPACITY);
            return;
        }
        const uint64_t mn = uniu(S.k[lowest]);
        spill_min = (spill_n == 0 || mn < spill_min) ? mn : spill_min;
        spill_n += E;
        nW -= E;
        compact_remove(lowest, G_MARK);
    }

    // Add K records (lanes [0, K)) to the list; waiting ones whose key exceeds
    // the spill's minimum go straight to the spill. L <= cap_now() on entry.
    DEV void add_entries(R y, int K) {
        if (spill_n > 0) {
            const bool toS = lane() < K && is_waiting(y.gs) && y.pk > spill_min;
            const uint64_t sm = ballot(toS);
            const int ns = popc(sm);
            if (ns) {
                if (spill_n + ns > scap) {
                    fail(S_ECAPACITY);
                    return;
                }
                if (toS) spill[spill_n + mbcnt(sm)] = to_rec(y);
                spill_n += ns;
                nW -= ns;
                const uint64_t km = ballot(lane() < K && !toS);
                y = permute_rec(y, place_dest(km, 0));
                K -= ns;
            }
        }
        if (K > 0) merge_new(y, K);
        if (L > cap_now()) spill_excess();
    }

    // The want-th smallest spilled key: radix select over 4-bit digits, the
    // 16 bin counts held one per lane (no LDS histogram).
    DEV uint64_t select_kth(int want) {
        hbm_fence();
        uint64_t prefix = 0;
        int rank = want;
        for (int d = 15; d >= 0; d--) {
            const int sh = 4 * d;
            int cnt = 0;  // lane b < 16: matching entries whose digit is b
            for (int rd = 0; rd < spill_n; rd += kWave) {
                const int i = rd + lane();
                uint64_t key = 0;
                bool match = false;
                if (i < spill_n) {
                    key = spill[i].pk;
                    match = d == 15 || (key >> (sh + 4)) == (prefix >> (sh + 4));
                }
                if (!ballot(match)) continue;
                const int dig = (int)((key >> sh) & 15u);
                for (int b = 0; b < 16; b++) {
                    const int nb = popc(ballot(match && dig == b));
                    if (lane() == b) cnt += nb;
                }
            }
            const int inc = scan_add(lane() < 16 ? cnt : 0);
            const int exc = inc - cnt;
            const uint64_t hm = ballot(lane() < 16 && exc < rank && rank <= inc);
            if (hm == 0) {
                fail(S_ESTATE);
                return 0;
            }
            const int bin = ffs0(hm);
            rank -= rl(exc, bin);
            prefix |= (uint64_t)bin << sh;
        }
        return prefix;
    }

    // Bring the smallest spilled entries back on chip (as many as fit).
    DEV void refill() {
        drop_holes();
        refill_into(cap_now() - L);
    }

    DEV void refill_into(int room) {
        const int want = min(spill_n, room);
        if (want <= 0) return;
        const uint64_t theta = want < spill_n ? select_kth(want) : ~0ull;
        if (status) return;
        hbm_fence();
        int wr = 0, got = 0;
        uint64_t newmin = ~0ull;
        const int n0 = spill_n;
        for (int rd = 0; rd < n0; rd += kWave) {
            const int i = rd + lane();
            const bool v = i < n0;
            Rec s = {};
            if (v) s = spill[i];
            const bool sel = v && s.pk <= theta;
            const bool keep = v && !sel;
            const uint64_t km = ballot(keep), sm = ballot(sel);
            if (keep) {
                const int d = wr + mbcnt(km);
                if (d != i) spill[d] = s;
                if (s.pk < newmin) newmin = s.pk;
            }
            wr += popc(km);
            const int ks = popc(sm);
            if (ks) {
                const R x = permute_rec(from_rec(s), place_dest(sm, 0));
                merge_new(x, ks);
                got += ks;
            }
        }
        if (got != want) fail(S_ESTATE);
        spill_n = wr;
        nW += got;
        spill_min = wminu(newmin);
    }

    // ---------------------------------------------------------- formation

    // Victim masks for the whole list: one LDS read and two ballots per chunk.
    // Batch members below the candidate are excluded by rank (victims lie
    // above it, where nothing is in the batch yet), so the masks ignore INB.
    DEV void build_victim_masks() {
        const int nch = (L + kWave - 1) >> 6;
        vm_res = vm_ev = 0;
        for (int c = 0; c < nch; c++) {
            const int r = c * kWave + lane();
            const uint32_t g = r < L ? ldx(r) : 0u;
            const bool rs = (g & G_RES) != 0;
            bool ev = rs;
            if (memguard) ev = rs && ((g >> G_LVL_SHIFT) & 31u) > (g & G_GUARD);
            if (pol == P_TRAIL && ballot(rs)) {
                // swap prevention: a request that emitted at least 0.6 D of its
                // D tokens is not a voluntary victim (5 (D - left) >= 3 D)
                int64_t Dv = 0, lv = 0;
                if (rs) {
                    const int idx = idx_of(S.k[r]);
                    Dv = idx < N ? Dp[idx] : 0;
                    lv = CP ? (int)(g >> kLeftShift) + 1 : (int)S.q[r].w;
                }
                ev = rs && !(2 * Dv >= 5 * lv);
            }
            const uint64_t m1 = ballot(rs), m2 = ballot(ev);
            if (lane() == c) vm_res = m1, vm_ev = m2;
        }
        vm_ok = true;
    }

    // A request at rank r became resident (dispatch: MemGuard keeps it
    // non-evictable until its level moves) or stopped being one.
    DEV void vm_set(int r, bool resident) {
        if (!vm_ok) return;
        if (resident && pol == P_TRAIL) {  // eligibility depends on progress: rebuild
            vm_ok = false;
            return;
        }
        const uint64_t bit = 1ull << (r & 63);
        if (lane() == (r >> 6)) {
            if (resident) {
                vm_res |= bit;
                if (!memguard) vm_ev |= bit;
            } else {
                vm_res &= ~bit;
                vm_ev &= ~bit;
            }
        }
    }

    // Highest rank > q set in the per-chunk mask vm, or -1.
    DEV int top_above(uint64_t vm, int q) const {
        const int qc = q >> 6, qb = q & 63;
        uint64_t m = vm;
        if (lane() < qc) m = 0;
        else if (lane() == qc) m &= qb == 63 ? 0ull : (~0ull << (qb + 1));
        const uint64_t nz = ballot(m != 0);
        if (!nz) return -1;
        const int ch = fls0(nz);
        return ch * kWave + fls0(rlu(m, ch));
    }

    // Highest rank > q holding a resident outside the batch that may be
    // evicted for candidate q (voluntary: MemGuard and hysteresis apply).
    // The list is sorted, so the highest such rank is the worst (key, idx).
    DEV int find_victim(int q, bool voluntary) {
        if constexpr (EXT) {
            if (voluntary && pol == P_SARATHI) return -1;  // no preemption by priority
        }
        if (UNLIKELY(!vm_ok)) build_victim_masks();
        const int v = top_above(voluntary ? vm_ev : vm_res, q);
        if (voluntary && v >= 0 && delta > 0) {
            // the worst eligible key fails the hysteresis test => all fail
            const uint64_t pv = uniu(S.k[v]), pkq = uniu(S.k[q]);
            const int64_t kd = key_of(pv) - delta, kq = key_of(pkq);
            if (!(kd > kq || (kd == kq && idx_of(pv) > idx_of(pkq)))) return -1;
        }
        return v;
    }

    DEV void do_evict(int v) {
        const uint4 qv = ldq(v);
        const int kvv = uni(skv(qv)), wv_ = uni(sw(qv));
        const uint32_t g = (uint32_t)uni((int)qv.x);
        wsync();
        if (lane() == 0)
            stxkv(v, (g & ~G_RES) | G_EVI | (pol == P_SRPT || pol == P_TRAIL ? G_DIRTY : 0u), wv_, 0);
        wsync();
        U -= blocks(kvv);
        nW++;
        nR--;
        emit_chunks |= 1ull << (v >> 6);
        vm_set(v, false);
    }

    // Admission of candidate q with n tokens: its KV advances now (emission
    // finds the tokens scheduled this iteration already counted).
    DEV void admit_one(int q, uint32_t g, int n, int du, int kvv, int wq) {
        const bool res = (g & G_RES) != 0;
        if (lane() == 0) {
            uint32_t g2 = g | G_INB;
            if (!res) g2 = (g2 & ~G_GUARD) | G_RES | ((g >> G_LVL_SHIFT) & 31u);
            stxkv(q, g2, wq, kvv + n);
        }
        wsync();
        cnt++;
        used += n;
        U += du;
        sum_ctx += kvv + n;
        if (!res) {
            nW--, nR++;
            vm_set(q, true);
        }
        emit_chunks |= 1ull << (q >> 6);
    }

    // Candidate q did not fit: evictions, or closing admissions. r_ahead
    // counts residents at ranks > q.
    // (g, n, du, kvv, wq: its flag word, chunk size, KV blocks, KV tokens and w)
    DEV void slow_path(int q, uint32_t g, int n, int du, int kvv, int wq, bool &closed,
                       int &r_ahead) {
        const bool res = (g & G_RES) != 0;
        for (int it = 0; it <= L + 1; it++) {
            if (U + du <= Kb) {
                admit_one(q, g, n, du, kvv, wq);
                return;
            }
            int v = find_victim(q, true);
            if (v >= 0) {
                do_evict(v);
                r_ahead--;
                ev_vol++;
                continue;
            }
            if (res) {
                v = find_victim(q, false);
                if (v >= 0) {
                    do_evict(v);
                    r_ahead--;
                    ev_forced++;
                    continue;
                }
                do_evict(q);
                ev_forced++;
                return;
            }
            closed = true;
            close_pk = uniu(S.k[q]);
            return;
        }
        fail(S_ESTATE);
    }

    // Spilled entries come next in the candidate order (formation reached
    // the first on-chip key above the spill's minimum with admissions open):
    // bring the smallest of them on chip. Every entry below rank p has been
    // processed and keeps its rank; every on-chip waiting key is below p.
    DEV void mid_refill(int p) {
        if (n_holes > 0) {
            const int from = max(p, lo_hole);
            const int L0 = L;
            compact_remove(from, G_DONE);
            n_holes -= L0 - L;
            if (n_holes == 0) lo_hole = INT32_MAX;
        }
        int room = cap_now() + kStage - L;  // may use the overflow region
        if (room <= 0) room = lcap + kStage - L;
        if (room <= 0) {
            fail(S_ECAPACITY);
            return;
        }
        refill_into(room);
        emit_all = true;
    }

    DEV void formation() {
        close_pk = ~0ull;
        cnt = 0, used = 0;
        sum_ctx = 0;
        emit_chunks = 0;
        emit_all = false;
        bool closed = false;
        int r_ahead = nR;  // residents at ranks >= p
        int p = 0;
        int bstar = spill_n > 0 ? lower_bound(spill_min) : INT32_MAX;
        // the next chunk's records, loaded while this one is processed; valid
        // while formation walks whole chunks without touching the list
        const int lim = lcap + kStage;
        uint4 nx = make_uint4(0u, 0u, 0u, 0u);
        bool have_nx = false;
        // every pass advances p or refills from the spill, so the walk ends
        // within L + spill_cap passes; a walk that does not is a broken state
        for (int pass = 0;; pass++) {
            fpass++;
            if (UNLIKELY(pass > lcap + kStage + scap + 2)) {
                fail(S_ESTATE);
                return;
            }
            if (cnt >= M || used >= T || (closed && r_ahead <= 0)) break;
            if (UNLIKELY(!closed && p >= bstar)) {  // bstar <= L: spilled entries come next
                mid_refill(p);
                if (status) return;
                bstar = spill_n > 0 ? lower_bound(spill_min) : INT32_MAX;
                have_nx = false;
                continue;
            }
            if (p >= L) break;
            const int end = closed ? L : min(L, bstar);
            const int r = p + lane();
            const bool valid = r < end;
            // (lanes past the slots read the last one; they are not valid)
            uint4 qr = nx;
            if (!have_nx) qr = ldq(min(r, lim - 1));
            nx = ldq(min(r + kWave, lim - 1));
            const uint32_t g = valid ? qr.x : 0u;
            const int w = sw(qr);
            const int kvv = skv(qr);
            const bool res = (g & G_RES) != 0;
            const bool cand = valid && !(g & (G_EVI | G_DONE)) && (res || !closed);
            // one round of scans: the candidates admitted from this chunk
            // are a prefix of its candidates, and only the last of them can
            // be clipped by the token budget
            const int m = cand ? min(w - kvv, c) : 0;
            const int kvc = cand ? kvv : 0;
            const int dfull = cand ? blocks(kvv + m) - blocks(kvv) : 0;
            const int mi = scan_add(m);
            const int dfi = scan_add(dfull);
            const int kvi = scan_add(kvc);
            const uint64_t cm = ballot(cand);
            const int cb = cnt + mbcnt(cm);
            const int ub = used + mi - m;
            const bool adm = cand && cb < M && ub < T;
            const int n = adm ? min(m, T - ub) : 0;
            const int du = adm ? blocks(kvv + n) - blocks(kvv) : 0;
            const int dui = dfi - dfull + du;
            const bool fit = U + dui <= Kb;
            const uint64_t bad = ballot(adm && !fit);
            const uint64_t am = ballot(adm);
            const uint64_t okm = bad ? (am & ((1ull << ffs0(bad)) - 1ull)) : am;
            const bool ok = ((okm >> lane()) & 1ull) != 0;
            if (ok) {  // admitted: the KV advances by this iteration's chunk now
                uint32_t g2 = g | G_INB;
                if (!res) g2 = (g2 & ~G_GUARD) | G_RES | ((g >> G_LVL_SHIFT) & 31u);
                stxkv(r, g2, w, kvv + n);
            }
            if (okm) {
                const int last = fls0(okm);
                const int used_new = rl(ub + n, last);
                const uint64_t nm = ballot(ok && !res);
                const int nadm_w = popc(nm);
                cnt += popc(okm);
                sum_ctx += rl(kvi, last) + (used_new - used);
                used = used_new;
                U += rl(dui, last);
                nW -= nadm_w;
                nR += nadm_w;
                if (pol == P_TRAIL && nadm_w) vm_ok = false;  // eligibility depends on progress
                if (UNLIKELY(vm_ok && nadm_w)) {  // dispatched waiting entries become residents
                    // lanes of this chunk land in aligned chunks p>>6 and (p>>6)+1
                    const int c0 = p >> 6, sh = p & 63;
                    const uint64_t lo = nm << sh, hi = sh ? (nm >> (64 - sh)) : 0ull;
                    const bool ev_too = !memguard;
                    if (lane() == c0) vm_res |= lo, vm_ev |= ev_too ? lo : 0ull;
                    if (lane() == c0 + 1) vm_res |= hi, vm_ev |= ev_too ? hi : 0ull;
                }
                emit_chunks |= (1ull << ((p + ffs0(okm)) >> 6)) | (1ull << ((p + last) >> 6));
            }
            const uint64_t resm = ballot(valid && res);
            wsync();
            if (bad) {
                const int ql = ffs0(bad);
                // residents among lanes [0, ql] are passed (q included if resident);
                // waiting entries admitted in this chunk sit below q
                r_ahead -= popc(resm & (ql == 63 ? ~0ull : ((2ull << ql) - 1ull)));
                slow_path(p + ql, (uint32_t)rl((int)g, ql), rl(n, ql), rl(du, ql), rl(kvv, ql),
                          rl(w, ql), closed, r_ahead);
                if (status) return;
                p = p + ql + 1;
                have_nx = false;
            } else {
                r_ahead -= popc(resm);
                const int p2 = min(p + kWave, end);
                have_nx = p2 == p + kWave;
                p = p2;
            }
        }
    }

    // ---------------------------------------------------------- execute

    // Returns the lowest rank whose key moved (INT32_MAX if none). Batch
    // members are the entries whose flags meet `mem` (G_INB; in a repeated
    // batch also G_RES), with `n1` added to their scheduled tokens (1 in a
    // repeated batch, whose entries carry no token count).
    DEV int emission(int64_t t_end, uint32_t mem, int n1) {
        int lo = INT32_MAX, lohole = INT32_MAX, nd = 0, ufree = 0, nmv = 0;
        nmoved = 0;
        bool bad_idx = false;
        uint64_t noemit = 0;  // batch members that emitted no token
        int dnext = 0;        // members whose next token opens a KV block
        const uint32_t t32 = (uint32_t)t_end;
        const int nch = (L + kWave - 1) >> 6;
        // LTR+ updates every candidate's starvation count: visit every chunk
        const bool all = emit_all || (EXT && pol == P_LTR);
        uint64_t todo = all ? (nch >= 64 ? ~0ull : ((1ull << nch) - 1ull)) : emit_chunks;
        if (!todo) return INT32_MAX;
        echunks += popc(todo);
        // chunks are visited in ascending order, the next one's records loaded
        // while this one is processed (a chunk's edits stay inside it). Lanes
        // past the list end read its last slot and are masked out.
        int b = ffs0(todo) * kWave;
        todo &= todo - 1;
        uint4 q;
        uint64_t pk;
        uint2 tg;
        {
            const int i0 = min(b + lane(), L - 1);
            q = ldq(i0), pk = S.k[i0], tg = S.tg[i0];
        }
        for (;;) {
            const int bn = todo ? ffs0(todo) * kWave : -1;
            todo &= todo - 1;
            uint4 qn = make_uint4(0u, 0u, 0u, 0u);
            uint64_t pkn = 0;
            uint2 tgn = make_uint2(0u, 0u);
            if (bn >= 0) {
                const int i1 = min(bn + lane(), L - 1);
                qn = ldq(i1), pkn = S.k[i1], tgn = S.tg[i1];
            }
            const int r = b + lane();
            const uint32_t g = r < L ? q.x : 0u;
            // Per lane, as selects: the flag tests below are lane-dependent,
            // and a branch on them would cost scalar exec-mask work in every
            // chunk. Members (flags meet `mem`) advance; entries evicted in
            // this iteration lose the eviction mark.
            const bool memb = (g & mem) != 0;
            const bool evi = !memb && (g & G_EVI) != 0;
            int w = sw(q), left = sleft(q);
            const int kv0 = skv(q);
            int kv = kv0 + n1;  // includes this iteration's chunk (added at admission)
            const int idx = idx_of(pk);
            bad_idx = bad_idx || (memb && idx >= N);
            const bool emit = memb && kv == w && idx < N;
            const bool first = emit && !(g & G_FIRST);
            // times are kept modulo 2^32: a gap of 2^32 us or more overflows
            // the request's TTLT too
            const uint32_t gap = t32 - tg.x;
            const uint32_t gm = emit && !first && gap > tg.y ? gap : tg.y;
            w += emit ? 1 : 0;
            left -= emit ? 1 : 0;
            const bool fin = emit && left == 0;
            uint32_t gs = (memb ? g & ~G_INB : g & ~G_EVI) | (first ? G_FIRST : 0u);
            gs = fin ? (gs | G_DONE) & ~G_RES : gs;
            ufree += fin ? blocks(kv) : 0;
            if (first) tfirst[idx] = t_end;
            if (fin) {
                tlast[idx] = t_end;
                tbo[idx] = gm;
            }
            kv = fin ? 0 : (memb ? kv : kv0);
            const bool live = emit && !fin;  // emitted and has tokens left
            bool chg = false;
            uint64_t pk2 = pk;
            if (pol == P_LAS) {
                // the attained service grew by one token
                chg = live;
                pk2 = chg ? pack((int64_t)w, idx) : pk;
            } else if (pol == P_SRPT || pol == P_TRAIL) {
                // remaining computed tokens (an evicted entry holds no KV)
                chg = (memb && !fin) || evi;
                pk2 = chg ? pack((int64_t)w + left - 1 - kv, idx) : pk;
            } else if (pol == P_BOOST) {
                const int lo_ = (int)((gs >> G_LVL_SHIFT) & 31u);
                int sig = w;  // P + dec
                if constexpr (EXT) {
                    // every lane reads: keep non-member lanes in bounds
                    const int ix = min(idx, N - 1);
                    if (phase_signal) sig = w - Pp[ix];  // dec >= 1 after this token
                    if (cache_signal) sig = w - Hp[ix];  // P - h + dec
                }
                const int ln = level_of(sig, k, lk);
                chg = live && ln != lo_;
                if (chg) {  // a level crossing (rare): re-key by the table step
                    pk2 = pack(key_of(pk) + S.bt[lo_] - S.bt[ln], idx);
                    gs = (gs & ~G_LVL) | ((uint32_t)ln << G_LVL_SHIFT);
                }
            }
            if constexpr (EXT) {
                if (pol == P_DIST && first && left > 0) {  // enters DistBoost's decode queue
                    pk2 = pack(t_end - kDecodeQueueOff, idx);
                    chg = true;
                } else if (pol == P_SARATHI && live) {
                    // round robin: back of the decode queue after each token
                    pk2 = pack(t_end - kDecodeQueueOff, idx);
                    chg = true;
                }
                if (pol == P_LTR && memb && !fin) {  // it ran: the count resets, or
                    if (!(gs & G_PROMO)) {           // a promotion spends its quantum
                        gs &= G_FLAGS;
                    } else if ((gs >> kLtrShift) <= 1u) {
                        gs = (gs & G_FLAGS & ~G_PROMO) | G_DIRTY;  // back to key D
                        pk2 = pack((int64_t)(w - Pp[idx]) + left, idx);
                        chg = true;
                    } else {
                        gs -= 1u << kLtrShift;
                    }
                }
            }
            // SRPT's and TRAIL's re-keyed entries carry no re-insertion mark:
            // compaction extracts those that fall out of order
            const bool dirty = chg && pol != P_SRPT && pol != P_TRAIL;
            gs |= dirty ? G_DIRTY : 0u;
            const bool mute = memb && !emit;
            const bool opens = live && blocks(kv + 1) != blocks(kv);
            if (memb || evi) {
                stq(r, gs, w, kv, left);
                S.k[r] = pk2;
                S.tg[r] = make_uint2(emit ? t32 : tg.x, gm);
            }
            if constexpr (EXT) {
                // LTR+: a candidate that did not run starves one more
                // iteration; at the threshold it is promoted for a quantum
                if (pol == P_LTR && !memb && r < L && !(g & (G_DONE | G_PROMO))) {
                    const uint32_t cnt = (g >> kLtrShift) + 1u;
                    uint32_t gx = (g & G_FLAGS & ~G_EVI) | (cnt << kLtrShift);
                    if ((int)cnt >= ltr_s) {
                        gx = (g & G_FLAGS & ~G_EVI) | G_PROMO | G_DIRTY |
                             ((uint32_t)ltr_q << kLtrShift);
                        pk2 = pack(iters + 1 - kPromotedOff, idx);
                        S.k[r] = pk2;
                        chg = true;
                    }
                    stx(r, gx);
                }
            }
            const uint64_t cm = ballot(chg), fm = ballot(fin);
            noemit |= ballot(mute);
            dnext += popc(ballot(opens));
            if (cm) {
                nmv += popc(cm);
                if (lo == INT32_MAX) lo = b + ffs0(cm);
            }
            if (fm) {
                if (lohole == INT32_MAX) lohole = b + ffs0(fm);
                nd += popc(fm);
                if (vm_ok && lane() == (b >> 6)) vm_res &= ~fm, vm_ev &= ~fm;
                if constexpr (EXT) {
                    if (ad) {  // end-to-end latencies enter the window in batch order
                        uint32_t lat = 0;
                        if (fin) {
                            const int64_t e2e = t_end - arr[idx_of(pk)];
                            lat = e2e > 0xFFFFFFFFll ? 0xFFFFFFFFu : (uint32_t)e2e;
                        }
                        for (uint64_t m = fm; m; m &= m - 1)
                            ada_push((uint32_t)rl((int)lat, ffs0(m)));
                    }
                }
            }
            if (bn < 0) break;
            b = bn, q = qn, pk = pkn, tg = tgn;
        }
        wsync();
        if (ballot(bad_idx)) fail(S_ESTATE);
        all_emit = noemit == 0;
        nmoved = nmv;
        du_next = dnext;
        if (nd) {
            U -= wsum(ufree);
            completed += nd;
            nR -= nd;
            n_holes += nd;
            lo_hole = min(lo_hole, lohole);
        }
        return lo;
    }

    // From rank `from` on: remove holes; extract entries whose key moved
    // (flagged, or below the running maximum of the entries kept before them)
    // into `stage` (lanes [0, min(count, 64))) and, beyond 64, the HBM
    // overflow. Returns the number extracted. No holes lie below `from`.
    DEV int compact_extract(int from, R &stage) {
        vm_ok = false;
        const int start = (from >> 6) << 6;
        uint64_t pmax = start > 0 ? uniu(S.k[start - 1]) : 0ull;
        int out = start, nx = 0;
        for (int b = start; b < L; b += kWave) {
            const int r = b + lane();
            const bool v = r < L;
            R y;
            if (v) ldr(r, y);
            const bool dead = v && (y.gs & G_DONE);
            const bool dirty = v && (y.gs & G_DIRTY);
            const uint64_t val = (v && !dead && !dirty) ? y.pk : 0ull;
            const uint64_t inc = scan_maxu(val);
            uint64_t exc = prev_lane_u64(inc, 0ull);
            if (pmax > exc) exc = pmax;
            const bool ext = v && !dead && (dirty || y.pk < exc);
            const bool keep = v && !dead && !ext;
            const uint64_t km = ballot(keep), xm = ballot(ext);
            wsync();
            if (keep) {
                const int d = out + mbcnt(km);
                if (d != r) str(d, y);
            }
            if (ext) {
                y.gs &= ~G_DIRTY;
                const int xi = nx + mbcnt(xm);
                if (xi >= kStage) ovf[xi - kStage] = to_rec(y);
            }
            wsync();
            if (xm && nx < kStage) {  // the first kStage extracted stay in registers
                const uint64_t sm = ballot(ext && nx + mbcnt(xm) < kStage);
                const R z = permute_rec(y, place_dest(sm, nx));
                if (lane() >= nx && lane() < nx + popc(sm)) stage = z;
            }
            const uint64_t cm = rlu(inc, 63);
            if (cm > pmax) pmax = cm;
            out += popc(km);
            nx += popc(xm);
        }
        L = out;
        n_holes = 0;
        lo_hole = INT32_MAX;
        return nx;
    }

    // Whether the entries from rank `from` on, completed ones aside, are in
    // ascending order; if so, their re-keyed entries stay where they are
    // (their flags are cleared). No holes lie below `from`.
    DEV bool settle_in_place(int from) {
        const int start = (from >> 6) << 6;
        uint64_t pmax = start > 0 ? uniu(S.k[start - 1]) : 0ull;
        for (int b = start; b < L; b += kWave) {
            const int r = b + lane();
            const bool v = r < L && !(ldx(r) & G_DONE);
            const uint64_t pk = r < L ? S.k[r] : 0ull;
            const uint64_t inc = scan_maxu(v ? pk : 0ull);
            uint64_t exc = prev_lane_u64(inc, 0ull);
            if (pmax > exc) exc = pmax;
            if (ballot(v && pk < exc)) return false;
            const uint64_t cm = rlu(inc, 63);
            if (cm > pmax) pmax = cm;
        }
        for (int b = start; b < L; b += kWave) {
            const int r = b + lane();
            if (r < L) {
                const uint32_t g = ldx(r);
                if (g & G_DIRTY) stx(r, g & ~G_DIRTY);
            }
        }
        wsync();
        return true;
    }

    // The list is in key order except for the resident entry at rank r, whose
    // key moved: put it at its rank among the others, shifting the entries
    // in between by one slot (one pass over them, instead of extracting the
    // tail of the list and merging it back). Holes keep their stale keys,
    // which are in order, and move with the others.
    DEV void move_one(int r) {
        vm_ok = false;
        R x;
        ldr(r, x);  // every lane reads the entry (one address)
        x.gs &= ~G_DIRTY;
        const uint64_t key = x.pk;
        // its new rank: the entries other than it with smaller keys. Entries
        // before r had keys below its old key and after r above it, so only
        // one side is counted, chunk by chunk, until a chunk lies beyond.
        int to;
        const bool right = r + 1 < L && uniu(S.k[r + 1]) < key;
        if (right) {
            to = r;
            for (int b = ((r + 1) >> 6) << 6; b < L; b += kWave) {
                const int i = b + lane();
                const bool lt = i > r && i < L && S.k[i] < key;
                const uint64_t m = ballot(lt);
                to += popc(m);
                if (popc(m) < min(L, b + kWave) - max(b, r + 1)) break;
            }
        } else {
            to = r;
            for (int b = ((r - 1) >> 6) << 6; b >= 0 && r > 0; b -= kWave) {
                const int i = b + lane();
                const bool gt = i < r && S.k[i] > key;
                const uint64_t m = ballot(gt);
                to -= popc(m);
                if (popc(m) < min(r, b + kWave) - b) break;
            }
        }
        wsync();
        if (to > r) {  // entries r+1 .. to move down one slot, in ascending chunks
            for (int b = ((r + 1) >> 6) << 6; b <= to; b += kWave) {
                const int i = b + lane();
                const bool mv = i > r && i <= to;
                R y;
                if (mv) ldr(i, y);
                wsync();
                if (mv) str(i - 1, y);
                wsync();
            }
            if (lo_hole > r && lo_hole <= to) lo_hole--;
        } else if (to < r) {  // entries to .. r-1 move up one slot, in descending chunks
            for (int b = ((r - 1) >> 6) << 6; b >= 0 && b + kWave > to; b -= kWave) {
                const int i = b + lane();
                const bool mv = i >= to && i < r;
                R y;
                if (mv) ldr(i, y);
                wsync();
                if (mv) str(i + 1, y);
                wsync();
            }
            if (lo_hole >= to && lo_hole < r) lo_hole++;
        }
        if (lane() == 0) str(to, x);
        wsync();
    }

    // emit_chunks := the 64-entry chunks holding residents (in a repeated
    // batch, every resident is a member)
    DEV void resident_chunks() {
        uint64_t m = 0;
        for (int b = 0; b < L; b += kWave) {
            const int r = b + lane();
            if (ballot(r < L && (ldx(r) & G_RES))) m |= 1ull << (b >> 6);
        }
        emit_chunks = m;
    }

    DEV void maintenance(int lo_mod) {
        if constexpr (EXT) {
            // Sarathi moves every decode that emitted to the same, latest key:
            // when all decodes were in the batch (steady decoding) the list
            // is still in order and nothing needs re-inserting
            if (pol == P_SARATHI && lo_mod < L && n_holes < kHoleLimit && L <= cap_now() &&
                settle_in_place(min(lo_mod, lo_hole)))
                lo_mod = L;
        }
        if (nmoved == 1 && lo_mod < L && n_holes < kHoleLimit && L <= cap_now() &&
            (ldx(lo_mod) & G_RES)) {
            move_one(lo_mod);  // one resident re-keyed (a level crossing, say)
            lo_mod = L;
        }
        if (UNLIKELY(lo_mod < L || n_holes >= kHoleLimit || L > cap_now())) {
            R stage;
            const int nx = compact_extract(min(min(lo_mod, lo_hole), L), stage);
            if (nx > kStage) hbm_fence();
            if (L > cap_now()) spill_excess();  // a refill during formation used the overflow region
            if (nx > 0 && status == 0) {
                add_entries(stage, min(nx, kStage));
                for (int b = kStage; b < nx && status == 0; b += kStage) {
                    const int kb = min(nx - b, kStage);
                    R x;
                    if (lane() < kb) x = from_rec(ovf[b - kStage + lane()]);
                    add_entries(x, kb);
                }
            }
        }
        if (status == 0) take_arrivals();
    }

    // ---------------------------------------------------------- adaptive gamma

    // Entries of the sorted window (n of them) below x.
    DEV int window_below(uint32_t x, int n) const {
        int c = 0;
        for (int b = 0; b < n; b += kWave) {
            const int r = b + lane();
            c += popc(ballot(r < n && S.ws[r] < x));
        }
        return c;
    }

    // UpdateStats (Algorithm 1): the end-to-end latency x (wave-uniform) of a
    // completed request enters the window; when it is full the oldest leaves.
    // The ring keeps completion order, the sorted copy serves the percentiles.
    DEV void ada_push(uint32_t x) {
        AdaLds &G = *S.as;
        int n = uni(G.wn);
        const int W = uni(G.window), head = uni(G.whead);
        if (n == W) {  // drop the oldest: close the gap at its first copy
            const uint32_t old = (uint32_t)uni((int)S.wr[head]);
            const int po = window_below(old, n);
            for (int b = ((po + 1) >> 6) << 6; b < n; b += kWave) {
                const int r = b + lane();
                const bool mv = r > po && r < n;
                uint32_t v = 0;
                if (mv) v = S.ws[r];
                wsync();
                if (mv) S.ws[r - 1] = v;
                wsync();
            }
            n--;
        }
        const int pn = window_below(x, n);  // open a slot at the insertion rank
        for (int b = ((n - 1) >> 6) << 6; b >= 0 && b + kWave > pn; b -= kWave) {
            const int r = b + lane();
            const bool mv = r >= pn && r < n;
            uint32_t v = 0;
            if (mv) v = S.ws[r];
            wsync();
            if (mv) S.ws[r + 1] = v;
            wsync();
        }
        if (lane() == 0) {
            S.ws[pn] = x;
            S.wr[head] = x;
            G.whead = head + 1 == W ? 0 : head + 1;
            G.wn = n + 1;
            G.wnew = 1;
        }
        wsync();
    }

    // UpdateGamma (Phase 4, Algorithm 2), before the keys of every iteration:
    // with at least min_samples latencies in the window, gamma_hat =
    // tau ln 5 / max(t99 - t95, eps) from the nearest-rank t95, t99 (only
    // recomputed when the window changed), then gamma = clip((1 - beta) gamma
    // + beta gamma_hat); each is one rounded double operation (no contraction).
    // A new grid cell re-keys every waiting and resident request.
    DEV void ada_update() {
#pragma clang fp contract(off)
        AdaLds &G = *S.as;
        const int wn = uni(G.wn);
        if (wn < uni(G.min_samples)) return;
        double gh = G.ghat;
        if (uni(G.wnew)) {
            const int r95 = (95 * wn + 99) / 100, r99 = (99 * wn + 99) / 100;
            const uint32_t t95 = S.ws[r95 - 1], t99 = S.ws[r99 - 1];
            double d = (double)(t99 - t95);
            if (d < ad->eps) d = ad->eps;
            gh = ad->num / d;
        }
        double g = (1.0 - ad->beta) * G.gamma + ad->beta * gh;
        if (g < ad->gmin) g = ad->gmin;
        if (g > ad->gmax) g = ad->gmax;
        const int cell = popc(ballot(g >= bnd));
        const int old = uni(G.cell);
        wsync();
        if (lane() == 0) {
            G.ghat = gh, G.wnew = 0;
            G.gamma = g;
            if (cell != old) G.cell = cell, G.switches++;
        }
        wsync();
        if (cell != old) ada_rekey(cell);
    }

    // The boost table changes to that of `cell`: keys a - bt[level] of the
    // spilled, waiting and resident entries shift by bt_old - bt_new of their
    // level; every on-chip entry is then re-inserted, so waiting entries above
    // the new spill minimum move to the spill and the list is sorted again.
    DEV void ada_rekey(int cell) {
        const int64_t *nt = ad->table[cell];
        hbm_fence();
        uint64_t mn = ~0ull;
        for (int b = 0; b < spill_n; b += kWave) {
            const int i = b + lane();
            if (i < spill_n) {
                const uint64_t pk = spill[i].pk;
                const int lv = min((int)((spill[i].gs >> G_LVL_SHIFT) & 31u), kLevels - 1);
                const uint64_t pk2 = pack(key_of(pk) + S.bt[lv] - nt[lv], idx_of(pk));
                spill[i].pk = pk2;
                mn = pk2 < mn ? pk2 : mn;
            }
        }
        spill_min = wminu(mn);
        for (int b = 0; b < L; b += kWave) {
            const int r = b + lane();
            if (r < L) {
                const uint32_t g = ldx(r);
                if (!(g & G_DONE)) {
                    const int lv = min((int)((g >> G_LVL_SHIFT) & 31u), kLevels - 1);
                    const uint64_t pk = S.k[r];
                    S.k[r] = pack(key_of(pk) + S.bt[lv] - nt[lv], idx_of(pk));
                    stx(r, g | G_DIRTY);
                }
            }
        }
        int64_t v = 0;
        if (lane() < kLevels) v = nt[lane()];
        wsync();
        if (lane() < kLevels) S.bt[lane()] = v;
        wsync();
        R stage;
        const int nx = compact_extract(0, stage);  // every live entry is flagged
        if (nx > kStage) hbm_fence();
        if (nx > 0 && status == 0) {
            add_entries(stage, min(nx, kStage));
            for (int b = kStage; b < nx && status == 0; b += kStage) {
                const int kb = min(nx - b, kStage);
                R x;
                if (lane() < kb) x = from_rec(ovf[b - kStage + lane()]);
                add_entries(x, kb);
            }
        }
    }

    // ---------------------------------------------------------- checks

    // The batch just formed respects the sequence cap, the token budget and
    // the KV budget, and every member computes at least one token.
    DEV void check_batch() {
        if (cnt < 1 || cnt > M || used < cnt || used > T || U < 0 || U > Kb) fail(S_ESTATE);
    }

    // The state between iterations: the list's residents, waiting entries
    // and holes match their counts; the KV in use is the residents' blocks,
    // within the budget; the keys of the entries other than holes ascend
    // strictly; holes lie at or after lo_hole; no mark of an iteration (in
    // the batch, evicted, selected for spilling, key moved) survives it; an
    // entry's KV lies within its signal and a waiting entry holds none; the
    // spill holds waiting entries only, its minimum is exact; and every
    // request taken so far is done, on chip or spilled.
    DEV void check_state() {
        bool bad = U < 0 || U > Kb || L < 0 || L > cap_now() || spill_n < 0 || spill_n > scap;
        int nres = 0, nwait = 0, nhole = 0, blk = 0;
        uint64_t pmax = 0;  // 1 + the largest key of the live entries so far (0: none)
        for (int b = 0; b < L && !bad; b += kWave) {
            const int r = b + lane();
            const bool v = r < L;
            const int i = min(r, L - 1);  // lanes past the list read its last slot
            const uint4 q = ldq(i);
            const uint32_t g = q.x;
            const uint64_t pk = S.k[i];
            const bool done = v && (g & G_DONE) != 0;
            const bool live = v && !done;
            const bool rs = live && (g & G_RES) != 0;
            const bool wt = live && (g & G_RES) == 0;
            const int w = sw(q), kv = skv(q), left = sleft(q);
            nres += rs ? 1 : 0;
            nwait += wt ? 1 : 0;
            nhole += done ? 1 : 0;
            blk += rs ? blocks(kv) : 0;
            const uint64_t inc = scan_maxu(live ? pk + 1 : 0ull);
            uint64_t exc = prev_lane_u64(inc, 0ull);
            if (pmax > exc) exc = pmax;
            bool e = v && (g & (G_INB | G_EVI | G_MARK)) != 0;
            e = e || (live && (g & G_DIRTY) != 0);
            e = e || (live && pk + 1 <= exc);  // not above a live key before it
            e = e || (done && r < lo_hole);
            e = e || (live && (kv < 0 || kv > w || left < 1 || idx_of(pk) >= N));
            e = e || (wt && kv != 0);
            bad = bad || ballot(e) != 0;
            const uint64_t cm = rlu(inc, 63);
            if (cm > pmax) pmax = cm;
        }
        if (!bad) {
            nres = wsum(nres), nwait = wsum(nwait), nhole = wsum(nhole), blk = wsum(blk);
            bad = nres != nR || nwait != nW || nhole != n_holes || blk != U ||
                  completed + nR + nW + spill_n != next;
        }
        if (!bad && spill_n > 0) {
            hbm_fence();
            uint64_t mn = ~0ull;
            bool e = false;
            for (int b = 0; b < spill_n; b += kWave) {
                const int i = b + lane();
                if (i < spill_n) {
                    const Rec x = spill[i];
                    if (x.pk < mn) mn = x.pk;
                    e = e || (x.gs & (G_RES | G_DONE | G_INB | G_EVI | G_MARK | G_DIRTY)) != 0 ||
                        x.kv != 0 || x.left < 1 || idx_of(x.pk) >= N;
                }
            }
            bad = ballot(e) != 0 || wminu(mn) != spill_min;
        }
        if (bad) fail(S_ESTATE);
    }

    // ---------------------------------------------------------- driver

    DEV void run() {
        load_pf();
        take_arrivals();
        for (;;) {
            if (status) break;
            if (UNLIKELY(nW + nR == 0)) {
                if (spill_n > 0) {
                    refill();
                    if (status) break;
                    if (nW + nR == 0) {
                        fail(S_ESTATE);
                        break;
                    }
                    continue;
                }
                if (next >= N) break;
                int off = next - pf;
                if (off >= kWave) {
                    pf = next;
                    load_pf();
                    off = 0;
                }
                const int64_t an = rl64(pa, off);
                idle += an - t;
                t = an;
                take_arrivals();
                continue;
            }
            if constexpr (EXT) {
                if (ad) {
                    ada_update();
                    if (status) break;
                }
            }
            const int64_t ev0 = ev_vol + ev_forced;
            const bool rp = rep;
            if (rp) {
                // the previous batch again: every resident, one token each
                // (its context grows by one token per member)
                U += du_next;
                cnt = nR;
                used = nR;
                sum_ctx += nR;
            } else {
                formation();
                if (status) break;
                if (cnt == 0) {
                    fail(S_ESTATE);
                    break;
                }
            }
            if constexpr (kCheck) {
                check_batch();
                if (status) break;
            }
            // formation evicted nothing, refilled nothing, stopped short of
            // the token budget and took every resident
            const bool rep_form = ev_vol + ev_forced == ev0 && !emit_all && used < T && cnt == nR;
            if (U > maxU) maxU = U;
            const int64_t dt = (int64_t)base + (int64_t)tok * used + (int64_t)ctx_quot((uint64_t)sum_ctx);
            const int64_t t_end = t + dt;
            const int c0 = completed;
            const int lo_mod = emission(t_end, rp ? (G_INB | G_RES) : G_INB, rp ? 1 : 0);
            t = t_end;
            iters++;
            reqiters += cnt;
            tokens += used;
            if (iters > max_iters) {
                fail(S_ELIVELOCK);
                break;
            }
            // Every member emitted (so every resident needs one token), none
            // completed or moved, the list needs no repair and the next
            // step's KV growth fits: then the next formation takes the same
            // residents and nothing else, as long as no request arrives. A
            // waiting candidate it meets with admissions open met them in
            // this formation too, did not fit and found no eligible victim;
            // the KV held by the members before it has not shrunk, its own
            // chunk has not shrunk, and the residents after it are the same
            // with the same keys and eligibility, so it closes admissions
            // again. (Adaptive gamma may re-key at the next step: excluded.)
            bool nrep = rep_form && all_emit && completed == c0 && lo_mod == INT32_MAX &&
                        L <= cap_now() && U + du_next <= Kb;
            if constexpr (EXT) nrep = nrep && ad == nullptr;
            // Arrivals (merged on chip or sent to the spill) that rank after
            // the candidate that closed admissions are met after it closes
            // them again, and skipped: the batch still repeats, as long as
            // nothing was spilled to make room (the on-chip list keeps every
            // waiting entry it had). The members' chunks are recounted, as
            // the merged arrivals may shift them. (Fixed build only: its
            // registers would cost the extended build occupancy.)
            const int next0 = next, sp0 = n_spilled;
            arr_min_pk = ~0ull;
            maintenance(lo_mod);
            rep = nrep && (next == next0 || (!EXT && arr_min_pk > close_pk && n_spilled == sp0 &&
                                             close_pk != ~0ull));
            if (!EXT && rep && next != next0) resident_chunks();
            if constexpr (kCheck) {
                if (status == 0) check_state();
            }
        }
        finish();
    }

    // CL: simulate while the replica has work and its clock is below `limit`,
    // the next arrival time of the global trace (an iteration that starts
    // before it is formed without that request); then wait for the router.
    // With limit = INT64_MAX it runs to the end of what was dispatched.
    DEV void run_until(int64_t limit) {
        if (status) return;
        take_arrivals();  // the router may have dispatched since the last call
        for (;;) {
            if (status) return;
            if (UNLIKELY(nW + nR == 0)) {
                if (spill_n > 0) {
                    refill();
                    if (status) return;
                    if (nW + nR == 0) {
                        fail(S_ESTATE);
                        return;
                    }
                    continue;
                }
                if (next >= Nk) return;  // idle: nothing dispatched yet
                int off = next - pf;
                if (off >= kWave) {
                    pf = next;
                    load_pf();
                    off = 0;
                }
                const int64_t an = rl64(pa, off);  // <= limit: dispatched requests have arrived
                idle += an - t;
                t = an;
                take_arrivals();
                continue;
            }
            if (t >= limit) return;
            if (ad) {  // each replica adapts its own gamma
                ada_update();
                if (status) return;
            }
            formation();
            if (status) return;
            if (cnt == 0) {
                fail(S_ESTATE);
                return;
            }
            if constexpr (kCheck) {
                check_batch();
                if (status) return;
            }
            if (U > maxU) maxU = U;
            const int64_t dt = (int64_t)base + (int64_t)tok * used + (int64_t)ctx_quot((uint64_t)sum_ctx);
            const int64_t t_end = t + dt;
            const int c0 = completed;
            const int lo_mod = emission(t_end, G_INB, 0);
            last_done = completed - c0;
            t = t_end;
            iters++;
            reqiters += cnt;
            tokens += used;
            if (iters > max_iters) {
                fail(S_ELIVELOCK);
                return;
            }
            maintenance(lo_mod);
            if constexpr (kCheck) {
                if (status == 0) check_state();
            }
        }
    }

    // CL: requests the replica holds at time aj (dispatched and not completed
    // by aj). Only the latest iteration can end after aj, and its
    // completions then have not happened yet.
    DEV int held_at(int64_t aj) const { return Nk - completed + (t > aj ? last_done : 0); }

    // CL: the router sends global request j to this replica.
    DEV void dispatch(int j) {
        if (lane() == 0) {
            __hip_atomic_store(&jl[Nk], j, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            A.assign[(size_t)inst * (size_t)N + (size_t)j] = wv;
        }
        // the prefetch window [pf, pf + 64) takes the new entry now, as a
        // reload from the list would (pf <= next <= Nk)
        if (lane() == Nk - pf) pidx = j, pa = arr[j], pP = Pp[j], pD = Dp[j];
        Nk++;
        hbm_fence();
    }

    // CL: latencies of the replica's requests in global order, its counters
    // (HBM, and in `cn` for the instance's totals) and status (`st`).
    DEV void finish_cl(int64_t *cn, int32_t *st) {
        hbm_fence();
        if (status == 0 && completed != Nk) fail(S_ESTATE);
        if (status == 0) {
            const size_t ioff = (size_t)inst * (size_t)N;
            bool bad = false;
            for (int b = 0; b < Nk; b += kWave) {
                const int kk = b + lane();
                if (kk < Nk) {
                    const int i = __hip_atomic_load(&jl[kk], __ATOMIC_RELAXED,
                                                    __HIP_MEMORY_SCOPE_AGENT);
                    const int64_t a = arr[i];
                    const int64_t f = tfirst[i] - a, l = tlast[i] - a;
                    if (f < 0 || f > 0xFFFFFFFFll || l < 0 || l > 0xFFFFFFFFll) bad = true;
                    A.ttft[ioff + i] = (uint32_t)f;
                    A.ttlt[ioff + i] = (uint32_t)l;
                }
            }
            if (ballot(bad)) fail(S_EOVERFLOW);
        }
        if (lane() == 0) {
            const int64_t v[8] = {iters, reqiters, tokens, ev_vol, ev_forced, t, maxU, idle};
            const size_t slot = (size_t)inst * (size_t)A.replicas + (size_t)wv;
            int64_t *rc = A.rcounters + slot * 8;
            for (int q = 0; q < 8; q++) rc[q] = v[q], cn[q] = v[q];
            A.rgamma[slot] = ad ? S.as->gamma : 0.0;
            A.rswitches[slot] = ad ? S.as->switches : 0;
            *st = status;
        }
    }

    DEV void finish() {
        hbm_fence();
        if (status == 0 && completed != N) fail(S_ESTATE);
        if (status == 0) {
            const size_t ioff = (size_t)inst * (size_t)N;
            bool bad = false;
            for (int b = 0; b < N; b += kWave) {
                const int i = b + lane();
                if (i < N) {
                    const int64_t a = arr[i];
                    const int64_t f = tfirst[i] - a, l = tlast[i] - a;
                    if (f < 0 || f > 0xFFFFFFFFll || l < 0 || l > 0xFFFFFFFFll) bad = true;
                    A.ttft[ioff + i] = (uint32_t)f;
                    A.ttlt[ioff + i] = (uint32_t)l;
                }
            }
            if (ballot(bad)) fail(S_EOVERFLOW);
        }
        if (lane() == 0) {
            int64_t *cn = A.counters + (size_t)inst * 8;
            cn[0] = iters, cn[1] = reqiters, cn[2] = tokens, cn[3] = ev_vol;
            cn[4] = ev_forced, cn[5] = t, cn[6] = maxU, cn[7] = idle;
            // the next launch's order key: the loop steps this wave ran,
            // weighted by their measured cost (an iteration's fixed work 4,
            // a formation pass over up to 64 candidates 5, an emission chunk
            // 3). Unlike wall-clock time it does not depend on the slot the
            // instance ran in.
            if (A.work) A.work[inst] = 4 * iters + 5 * (int64_t)fpass + 3 * (int64_t)echunks;
            if constexpr (EXT) {  // (zero from tas_create for the other build)
                A.gamma_out[inst] = ad ? S.as->gamma : 0.0;
                A.switch_out[inst] = ad ? S.as->switches : 0;
            }
            A.status[inst] = status;
        }
    }
};

template <int BSH, bool EXT, bool CP>
DEV void run_instance(const SimArgs &a, const DevSetting &st, int inst, unsigned char *smem) {
    Sim<BSH, EXT, false, CP> s(a, st, inst, smem);
    s.run();
}

// A cluster of replicas behind a join-shortest-queue router (global dispatch
// policies): one wavefront per replica, all in one workgroup. For every
// request of the global trace, in order, each replica first simulates the
// iterations that start before its arrival; then the request goes to the
// replica holding the fewest requests at that instant (ties to the lowest
// replica). Every wave passes the same barrier once per request, whatever
// its own state, so the workgroup cannot split at a barrier.
struct JsqLds {
    int32_t held[2][kMaxReplicas];  // by the parity of the global request index
    int32_t status[kMaxReplicas];
    int64_t cn[kMaxReplicas][8];
};
static_assert(sizeof(JsqLds) == kJsqLdsBytes, "router block size");

template <int BSH>
DEV void run_cluster(const SimArgs &a, const DevSetting &st, int inst, unsigned char *smem) {
    JsqLds *J = (JsqLds *)smem;
    const int R = a.replicas, w = (int)(threadIdx.x >> 6), N = a.n_req;
    Sim<BSH, true, true> s(a, st, inst, smem + kJsqLdsBytes + (size_t)w * (size_t)a.wave_lds, w);
    const int64_t *arr = a.arrival + (size_t)st.trace * (size_t)N;
    s.load_pf();  // nothing dispatched yet: an empty window, kept current by dispatch
    for (int j = 0;; j++) {  // j = N: run what was dispatched to the end
        const int64_t aj = j < N ? arr[j] : INT64_MAX;
        s.run_until(aj);
        if (j == N) break;
        // One barrier per request: the counts alternate between two
        // buffers. A wave that runs ahead writes the other one, and it
        // comes back to this one only after passing the next request's
        // barrier, which every wave reaches after reading this one.
        int32_t *held = J->held[j & 1];
        if (lane() == 0) held[w] = s.held_at(aj);
        __syncthreads();
        int best = 0, bn = held[0];
        for (int r = 1; r < R; r++) {
            const int h = held[r];
            if (h < bn) best = r, bn = h;
        }
        if (best == w) s.dispatch(j);
    }
    s.finish_cl(J->cn[w], &J->status[w]);
    __syncthreads();
    if (w == 0) {  // instance totals: sums, the latest clock, the largest KV peak
        const int q = lane();
        if (q < 8) {
            int64_t v = 0;
            for (int r = 0; r < R; r++) {
                const int64_t x = J->cn[r][q];
                v = (q == 5 || q == 6) ? (x > v ? x : v) : v + x;
            }
            a.counters[(size_t)inst * 8 + q] = v;
        }
        if (q == 0) {
            int32_t e = 0;
            for (int r = 0; r < R && e == 0; r++) e = J->status[r];
            a.status[inst] = e;
        }
    }
}

// EXT: the extended build (adaptive gamma, the phase-aware and cache-aware signals,
// DistBoost, Sarathi), launched when some instance uses one of them (its extra state
// and code cost the other policies registers). CP: compact list slots.
template <bool EXT, bool CP>
__global__ __launch_bounds__(64) void sim_kernel(SimArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    if ((int)blockIdx.x >= a.n_inst) return;
    const int inst = a.order ? a.order[blockIdx.x] : (int)blockIdx.x;
    if (a.retry && a.status[inst] != S_ECAPACITY) return;
    const DevSetting &st = a.inst[inst];
    if (a.bs == 16) run_instance<4, EXT, CP>(a, st, inst, smem);
    else run_instance<-1, EXT, CP>(a, st, inst, smem);
}

// MAXW: the largest number of waves (replicas) the build serves; 8 leaves
// each wave twice the registers of 16.
template <int BSH, int MAXW>
__global__ __launch_bounds__(64 * MAXW) void cluster_kernel(SimArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int inst = blockIdx.x;
    if (inst >= a.n_inst) return;
    if (a.retry && a.status[inst] != S_ECAPACITY) return;
    run_cluster<BSH>(a, a.inst[inst], inst, smem);
}

}  // namespace
}  // namespace tas

int tas_launch_cluster(const tas::SimArgs &a, int64_t lds_bytes, void *stream) {
    if (a.n_inst <= 0) return 0;
    if (a.replicas < 2 || a.replicas > tas::kMaxReplicas) return -4;
    hipStream_t s = (hipStream_t)stream;
    const bool small = a.replicas <= 8, b16 = a.bs == 16;
    const void *fn = small ? (b16 ? (const void *)tas::cluster_kernel<4, 8>
                                  : (const void *)tas::cluster_kernel<-1, 8>)
                           : (b16 ? (const void *)tas::cluster_kernel<4, tas::kMaxReplicas>
                                  : (const void *)tas::cluster_kernel<-1, tas::kMaxReplicas>);
    if (lds_bytes > 65536) {
        if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)lds_bytes) != hipSuccess)
            return -4;
    }
    const dim3 grid((unsigned)a.n_inst), block((unsigned)(64 * a.replicas));
    if (small && b16)
        hipLaunchKernelGGL((tas::cluster_kernel<4, 8>), grid, block, (size_t)lds_bytes, s, a);
    else if (small)
        hipLaunchKernelGGL((tas::cluster_kernel<-1, 8>), grid, block, (size_t)lds_bytes, s, a);
    else if (b16)
        hipLaunchKernelGGL((tas::cluster_kernel<4, tas::kMaxReplicas>), grid, block,
                           (size_t)lds_bytes, s, a);
    else
        hipLaunchKernelGGL((tas::cluster_kernel<-1, tas::kMaxReplicas>), grid, block,
                           (size_t)lds_bytes, s, a);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

int tas_launch_sim(const tas::SimArgs &a, int64_t lds_bytes, void *stream) {
    if (a.n_inst <= 0) return 0;
    hipStream_t s = (hipStream_t)stream;
    void (*const fns[2][2])(tas::SimArgs) = {
        {tas::sim_kernel<false, false>, tas::sim_kernel<false, true>},
        {tas::sim_kernel<true, false>, tas::sim_kernel<true, true>}};
    void (*fn)(tas::SimArgs) = fns[a.ext ? 1 : 0][a.cp ? 1 : 0];
    if (lds_bytes > 65536) {
        if (hipFuncSetAttribute((const void *)fn, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)lds_bytes) != hipSuccess)
            return -4;
    }
    hipLaunchKernelGGL(fn, dim3((unsigned)a.n_inst), dim3(64), (size_t)lds_bytes, s, a);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}
