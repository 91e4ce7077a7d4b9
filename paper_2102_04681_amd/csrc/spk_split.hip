// spk_split.hip -- the persistent step kernel with the soonest deliveries
// split from the rest (binned delivery).
//
// Only the events of delay 1 from the spikes of step t are needed to update
// the neurons at t + 1; the events of longer delays are needed later.  Each
// workgroup (one per compute unit) therefore runs two roles at once, on
// disjoint waves and LDS:
//   - the tile role (waves 0-7) owns a target tile: it sums the arriving
//     events into LDS accumulators, updates the tile's neurons (state kept in
//     LDS for the whole launch) and publishes the tile's spikes;
//   - the push role (waves 8-15) is one of the XCD's push blocks: it takes an
//     equal share of the spikes of t, files their delay-1 events first
//     ("critical" pages, one per target tile), signals the XCD, and then
//     files the events of the other delays ("bulk" pages, per arrival slot
//     and tile) while the tiles update.
// The tile role drains the bulk pages of arrival t + 1 as soon as the bulk
// phase of t - 1 is done (every event of a delay >= 2 arriving at t + 1 was
// filed by then), so that only the critical pages remain between the push of
// t and the update of t + 1.  Rows keep each XCD group's smallest-delay
// synapses first, with their end in the row descriptor, so the critical part
// of a row is one contiguous run.  With a smallest delay above 1 nothing is
// critical and the whole push runs beside the updates.
//
// The roles meet only through global words: tiles -> push (a grid-wide
// count of published spike lists; a tile never counts step t before every
// tile has counted t - 1), push -> tiles (per push block, the number of
// critical and of bulk phases it has finished).  Inside a role, waves synchronise through an
// LDS counter (the hardware barrier would stop both roles).  Spike lists
// cross XCDs with agent-scope stores and loads; pages are written and read
// on one XCD and read after an L1 invalidate.  Every wait is bounded and an
// abort flag polled by all waiters lets the grid drain.
#include <hip/hip_runtime.h>

#include "spk_dev.h"

namespace spk {

namespace {

constexpr int kSplitThreads = 1024;
constexpr uint32_t kRoleWaves = 8;                        // waves per role
constexpr uint32_t kRoleThreads = kRoleWaves * kWave;     // 512
constexpr int kSplitRounds = kMaxTileW / kRoleThreads;    // neurons per tile thread
constexpr uint32_t kSplitChunk = 256;                     // spikes resolved per push chunk
constexpr uint32_t kSplitMaxT = kGroups * kRunMaxR;       // tiles
constexpr int kSplitDrain = 16;                           // page loads in flight per tile thread
constexpr uint64_t kSplitSpinTicks = 10ull * 100000000ull;  // 10 s of the 100 MHz clock
constexpr uint32_t kSplitStoppedFlag = 4u;                // sticky in the network's device flags

__device__ __forceinline__ uint32_t xcc_id_split()
{
    return __builtin_amdgcn_s_getreg((20) | (0 << 6) | ((4 - 1) << 11)) & 0xfu;  // HW_REG_XCC_ID[3:0]
}

// Wait until *p >= target (wrap-safe); false if the wait gave up or another
// workgroup did.
__device__ __forceinline__ bool split_spin(const uint32_t *p, uint32_t target, uint32_t *abort_flag)
{
    const uint64_t t0 = wall_clock64();
    for (uint32_t k = 0;; k++) {
        if ((int32_t)(ld_ag(p) - target) >= 0) return true;
        if ((k & 31u) == 31u) {
            if (ld_ag(abort_flag)) return false;
            if (wall_clock64() - t0 > kSplitSpinTicks) {
                atomicOr(abort_flag, kRunAbortTimeout);
                return false;
            }
        }
        __builtin_amdgcn_s_sleep(1);
    }
}

// Wait (the first wave of a role) until every one of the n <= 64 progress
// words p[0..n) has reached target (wrap-safe); false if the wait gave up or
// another workgroup did.  Exact per-block progress, not a count: a fast block
// that is a step ahead cannot stand in for a slow one.
__device__ __forceinline__ bool split_spin_all(const uint32_t *p, uint32_t n, uint32_t target, uint32_t *abort_flag)
{
    const uint32_t lane = lane_id();
    const uint64_t t0 = wall_clock64();
    for (uint32_t k = 0;; k++) {
        const uint32_t v = ld_ag(p + (lane < n ? lane : 0u));
        if (__all(lane >= n || (int32_t)(v - target) >= 0)) return true;
        if ((k & 31u) == 31u) {
            if (ld_ag(abort_flag)) return false;
            if (wall_clock64() - t0 > kSplitSpinTicks) {
                if (lane == 0) atomicOr(abort_flag, kRunAbortTimeout);
                return false;
            }
        }
        __builtin_amdgcn_s_sleep(1);
    }
}

// The waves of one role: local thread index, scalar wave index, and a
// barrier on an LDS arrival counter (every wave of the role calls sync()).
// The wait is bounded (2^24 polls, about a second); a role that gives up
// raises the abort flag, and every global wait then ends.
struct Role {
    uint32_t tid, w, epoch;
    uint32_t *bar;
    uint32_t *abort_flag;
    __device__ __forceinline__ void sync()
    {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
        epoch += kRoleWaves;
        if (lane_id() == 0) __hip_atomic_fetch_add(bar, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
        for (uint32_t k = 0;
             (int32_t)(__hip_atomic_load(bar, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) - epoch) < 0; k++) {
            if (k == (1u << 24)) {
                if (lane_id() == 0) atomicOr(abort_flag, kRunAbortTimeout);
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
    }
};

// Exclusive scan of one u32 per role thread; the total in *total.
__device__ __forceinline__ uint32_t role_scan_u32(Role &g, uint32_t x, uint32_t *ws, uint32_t *total)
{
    const uint32_t lane = lane_id();
    uint32_t inc = x;
    for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t y = __shfl_up(inc, o);
        if (lane >= (uint32_t)o) inc += y;
    }
    if (lane == kWave - 1) ws[g.w] = inc;
    g.sync();
    uint32_t before = 0, tot = 0;
    for (uint32_t k = 0; k < kRoleWaves; k++) {
        const uint32_t v = ws[k];
        before += k < g.w ? v : 0u;
        tot += v;
    }
    g.sync();
    *total = tot;
    return before + inc - x;
}

__device__ __forceinline__ uint64_t role_sum_u64(Role &g, uint64_t x, unsigned long long *ws)
{
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
    if (lane_id() == 0) ws[g.w] = x;
    g.sync();
    uint64_t tot = 0;
    for (uint32_t k = 0; k < kRoleWaves; k++) tot += ws[k];
    g.sync();
    return tot;
}

// Spike counts of slot's T tile segments -> exclusive prefix in pre[]; total.
__device__ __forceinline__ uint32_t role_spike_set(Role &g, const StepArgs &a, uint32_t slot, uint32_t *pre, uint32_t *ws)
{
    const uint32_t T = a.tl.T, W = a.tl.W;
    const uint32_t b = g.tid * 2;
    const uint32_t *cnt = a.spk_cnt + (uint64_t)slot * T;
    uint32_t c0 = ld_ag(cnt + (b < T ? b : 0)), c1 = ld_ag(cnt + (b + 1 < T ? b + 1 : 0));
    c0 = b < T ? (c0 < W ? c0 : W) : 0u;
    c1 = b + 1 < T ? (c1 < W ? c1 : W) : 0u;
    uint32_t tot;
    const uint32_t ex = role_scan_u32(g, c0 + c1, ws, &tot);
    if (b < T) pre[b] = ex;
    if (b + 1 < T) pre[b + 1] = ex + c0;
    if (g.tid == 0) pre[T] = tot;
    g.sync();
    return tot;
}

template <bool FIXED, bool CMP>
struct SplitLDS {
    using AccT = typename Acc<FIXED>::T;
    using Rec = typename SynRec<CMP>::T;
    static constexpr int R = 16;                               // push: events per thread per load phase
    static constexpr uint32_t kStageN = R * kRoleThreads / 2;  // events bucket-sorted at once
    struct {
        float V[kMaxTileW];
        uint8_t ref[kMaxTileW];     // LIF: refractory steps left; source: fires at the current step
        uint8_t kp[kMaxTileW];      // Poisson count of the current step
        AccT acc[kMaxTileW];
        uint64_t pois[256];
        uint16_t guide[256];
        uint32_t cbase[kRoleWaves * kSplitDrain];
        uint32_t clen[kRoleWaves * kSplitDrain];
        uint32_t ws[16];
        unsigned long long ws64[16];
        uint32_t bar, nspk, stop, ovf;
    } t;
    struct {
        Rec stage[kStageN];
        uint32_t pre[kSplitMaxT + 1];
        uint32_t cpre[kSplitChunk + 1];
        uint32_t plen[kSplitChunk];
        uint32_t blen[kSplitChunk];       // the bulk run's length (it follows the critical run)
        uint64_t pbase[kSplitChunk];
        uint64_t cbase[R * kRoleWaves];
        uint32_t clen[R * kRoleWaves];
        uint32_t bcnt[kSplitMaxBuckets];  // events per bucket in this half, then rank cursor
        uint32_t bst[kSplitMaxBuckets];   // bucket starts in the stage
        uint32_t wb[kSplitMaxBuckets];    // page position of stage entry q is wb[b] + q
        uint32_t fill[kSplitMaxBuckets];  // bulk pages: records in (arrival slot, tile), persistent
        uint32_t cfill[kRunMaxR];         // critical pages: records per tile
        uint32_t ws[16], ws2[16];
        unsigned long long ws64[16];
        uint32_t bar, stop;
    } p;
    uint32_t x, r, stop;
};

// ---------------------------------------------------------------- tile role

// Per-step draws for step t (Poisson counts; sources: whether they fire).
template <bool FIXED, bool CMP>
__device__ __forceinline__ void split_draws(const StepArgs &a, SplitLDS<FIXED, CMP> &L, const Role &g, uint32_t tile_lo,
                            uint32_t tile_n, uint64_t t)
{
    const ModelArgs &m = a.m;
#pragma unroll 4
    for (int u = 0; u < kSplitRounds; u++) {
        const uint32_t q = u * kRoleThreads + g.tid;
        if (q >= tile_n) continue;
        const uint32_t gi = tile_lo + q;
        if (m.pois_len) {
            const uint32_t h = hash_hi32(step_hash(m.keys.pois, gi, t));
            uint32_t k = L.t.guide[h >> 24];
            while ((uint64_t)h >= L.t.pois[k]) k++;
            L.t.kp[q] = (uint8_t)k;
        }
        if (m.kind == SPK_SOURCE)
            L.t.ref[q] = (uint64_t)hash_hi32(step_hash(m.keys.bern, gi, t)) < m.src_thr ? 1 : 0;
    }
}

// Sum the records of one page set into the accumulators: the critical pages
// (crit: one per push block of the group) or the bulk pages of arrival slot
// `slot`.  Returns the records summed (counted in the fill counters,
// including records that overflowed to the global accumulators).
template <bool FIXED, bool CMP>
__device__ __forceinline__ uint64_t split_drain(const StepArgs &a, const RunArgs &ra, SplitLDS<FIXED, CMP> &L, Role &g,
                                uint32_t x, uint32_t c, bool crit, uint32_t slot)
{
    const uint32_t tid = g.tid, lane = lane_id(), w = g.w;
    const uint32_t cap = a.page_cap, G1 = ra.R, T8 = a.tl.T8;
    constexpr uint32_t kPer = CMP ? 2u : 1u;
    constexpr uint32_t kChunk = kPer * kWave;
    const uint32_t g1 = tid < G1 ? tid : 0u;
    const uint32_t page = crit ? (x * G1 + g1) * T8 + c : page_of(a, x, g1, slot, c);
    uint32_t pf = crit ? ra.cfill[page] : a.pfill[page];
    pf = tid < G1 ? pf : 0u;
    const uint32_t ne = pf < cap ? pf : cap;
    uint32_t C;
    const uint32_t cex = role_scan_u32(g, (ne + kChunk - 1) / kChunk, L.t.ws, &C);
    const uint64_t got = role_sum_u64(g, pf, L.t.ws64);
    const uint32_t nchp = (ne + kChunk - 1) / kChunk;
    constexpr uint32_t kWin = kSplitDrain * kRoleWaves;
    for (uint32_t i0 = 0; i0 < C; i0 += kWin) {
        for (uint32_t q = tid; q < kWin; q += kRoleThreads) L.t.clen[q] = 0;
        g.sync();
        if (tid < G1) {
            const uint32_t cb = cex > i0 ? cex : i0, ce = cex + nchp < i0 + kWin ? cex + nchp : i0 + kWin;
            const uint32_t pbase = page * cap;
            for (uint32_t q = cb; q < ce; q++) {
                const uint32_t o = (q - cex) * kChunk;
                L.t.cbase[q - i0] = (pbase + o) / kPer;
                L.t.clen[q - i0] = ne - o < kChunk ? ne - o : kChunk;
            }
        }
        g.sync();
        if constexpr (CMP) {
            const uint32_t *pw = (const uint32_t *)(crit ? ra.cpages16 : a.pages16);
            uint32_t rr[kSplitDrain];
            uint32_t okm = 0;
#pragma unroll
            for (int u = 0; u < kSplitDrain; u++) {
                const uint32_t cw = u * kRoleWaves + w;
                const uint32_t len = L.t.clen[cw], cb = L.t.cbase[cw];
                const bool ok = 2 * lane < len;
                const uint32_t idx = ok ? cb + lane : 0u;
                okm |= ((uint32_t)ok | (uint32_t)(2 * lane + 1 < len) << 1) << (2 * u);
                rr[u] = pw[idx];  // unconditional load from a clamped index
            }
#pragma unroll
            for (int u = 0; u < kSplitDrain; u++) {
#pragma unroll
                for (int hf = 0; hf < 2; hf++) {
                    if (!((okm >> (2 * u + hf)) & 1u)) continue;
                    const uint32_t rec = hf ? rr[u] >> 16 : rr[u] & 0xffffu;
                    Acc<FIXED>::add(&L.t.acc[rec & kPageLocalMask], class_units(a, rec >> kPageClassShift));
                }
            }
        } else {
            const int2 *pp = crit ? ra.cpages : a.pages;
            int2 rr[kSplitDrain];
            uint32_t okm = 0;
#pragma unroll
            for (int u = 0; u < kSplitDrain; u++) {
                const uint32_t cw = u * kRoleWaves + w;
                const uint32_t len = L.t.clen[cw], cb = L.t.cbase[cw];
                const bool ok = lane < len;
                const uint32_t idx = ok ? cb + lane : 0u;
                okm |= (uint32_t)ok << u;
                rr[u] = pp[idx];
            }
#pragma unroll
            for (int u = 0; u < kSplitDrain; u++)
                if ((okm >> u) & 1u)
                    Acc<FIXED>::add(&L.t.acc[(uint32_t)rr[u].x], units_of<FIXED>(rr[u].y, a.m.shift64));
        }
        g.sync();
    }
    return got;
}

// Events of arrival slot `slot` that did not fit their pages.
template <bool FIXED, bool CMP>
__device__ __forceinline__ void split_overflow(const StepArgs &a, SplitLDS<FIXED, CMP> &L, Role &g, uint32_t tile,
                               uint32_t tile_n, uint32_t slot)
{
    const uint64_t st = (uint64_t)slot * a.tl.T + tile;
    if (g.tid == 0) L.t.ovf = ld_ag(&a.ovf_flag[st]);
    g.sync();
    if (!L.t.ovf) return;  // uniform: read from LDS by every thread
    for (uint32_t q = g.tid; q < tile_n; q += kRoleThreads) {
        const uint64_t gi = st * a.tl.W + q;
        if (FIXED) {
            int32_t *o = (int32_t *)a.acc_ovf + gi;
            L.t.acc[q] += (int32_t)ld_ag((const uint32_t *)o);
            st_ag((uint32_t *)o, 0u);
        } else {
            unsigned long long *o = (unsigned long long *)a.acc_ovf + gi;
            L.t.acc[q] += __hip_atomic_load(o, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(o, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    g.sync();
    if (g.tid == 0) st_ag(&a.ovf_flag[st], 0u);
}

// Update of the tile's neurons; spikes compacted by wavefront ballots and
// stored straight into the tile's segment of the spike list of t.
template <bool FIXED, bool CMP>
__device__ __forceinline__ void split_update(const StepArgs &a, SplitLDS<FIXED, CMP> &L, Role &g, uint32_t x, uint32_t tile,
                             uint32_t tile_lo, uint32_t tile_n, uint64_t t, uint64_t delivered, uint32_t sslot)
{
    const ModelArgs &m = a.m;
    const uint32_t lane = lane_id();
    const uint64_t seg = (uint64_t)sslot * a.tl.T + tile;
    uint32_t *dst = a.spk_ids + seg * a.tl.W;
#pragma unroll 4
    for (int u = 0; u < kSplitRounds; u++) {
        const uint32_t q = u * kRoleThreads + g.tid;
        bool spk = false;
        if (q < tile_n) {
            const uint32_t K = m.pois_len ? L.t.kp[q] : 0u;
            float I;
            if (FIXED) {
                const int32_t qt = (int32_t)L.t.acc[q] + (int32_t)K * m.ext_wq + m.bias_q;
                I = ldexpf((float)qt, -m.shift);
            } else {
                const float isyn = fixed64_to_float(L.t.acc[q], m.shift64);
                const float ext = __fmul_rn((float)K, m.ext_w);
                I = __fadd_rn(__fadd_rn(isyn, ext), m.i_bias);
            }
            float V = L.t.V[q];
            if (m.kind == SPK_SOURCE) {
                const float av = __fsub_rn(m.v_rest, V);
                const float bv = __fmul_rn(m.k, av);
                const float cv = __fadd_rn(V, bv);
                V = __fadd_rn(cv, I);
                spk = L.t.ref[q] != 0;
            } else {
                uint32_t r = L.t.ref[q];
                if (r > 0) {
                    r -= 1;
                    V = m.v_reset;
                } else {
                    const float av = __fsub_rn(m.v_rest, V);
                    const float bv = __fmul_rn(m.k, av);
                    const float cv = __fadd_rn(V, bv);
                    V = __fadd_rn(cv, I);
                    if (V >= m.v_th) {
                        spk = true;
                        V = m.v_reset;
                        r = m.ref_steps;
                    }
                }
                L.t.ref[q] = (uint8_t)r;
            }
            L.t.V[q] = V;
        }
        const uint64_t mask = __ballot(spk);
        if (mask) {
            const int leader = __ffsll((unsigned long long)mask) - 1;
            uint32_t wb = 0;
            if ((int)lane == leader) wb = atomicAdd(&L.t.nspk, (uint32_t)__popcll(mask));
            wb = __shfl(wb, leader);
            if (spk) {
                const uint32_t rank = __builtin_amdgcn_mbcnt_hi(
                    (uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
                st_ag(dst + wb + rank, tile_lo + q);
            }
        }
    }
    g.sync();
    if (g.tid == 0) {
        const uint32_t ns = L.t.nspk;
        st_ag(&a.spk_cnt[seg], ns);
        if (ns) atomicAdd(&a.counts8[t * kGroups + x], ns);
        if (delivered)
            atomicAdd((unsigned long long *)&a.delivered8[t * kGroups + x], (unsigned long long)delivered);
    }
}

template <bool FIXED, bool CMP>
__device__ __forceinline__ void tile_role(const RunArgs &ra, SplitLDS<FIXED, CMP> &L, uint32_t x, uint32_t c)
{
    const StepArgs &a = ra.s;
    RunCtl *ctl = ra.ctl;
    const uint32_t rt = threadIdx.x;
    Role g{rt, (uint32_t)__builtin_amdgcn_readfirstlane(rt / kWave), 0u, &L.t.bar, &ctl->abort_flag};
    const Tiling tl = a.tl;
    const uint32_t tile = x * tl.T8 + c;
    const uint32_t tile_lo = tile * tl.W;
    const uint32_t tile_n = tile_lo < a.n ? (a.n - tile_lo < tl.W ? a.n - tile_lo : tl.W) : 0u;
    const ModelArgs &m = a.m;
    for (uint32_t q = g.tid; q < tile_n; q += kRoleThreads) {
        L.t.V[q] = a.V[tile_lo + q];
        L.t.ref[q] = a.ref[tile_lo + q];
    }
    if (m.pois_len)
        for (uint32_t q = g.tid; q < 256; q += kRoleThreads) {
            L.t.pois[q] = a.pois[q < m.pois_len ? q : 0u];
            L.t.guide[q] = a.pois_guide[q];
        }
    for (uint32_t q = g.tid; q < tl.W; q += kRoleThreads) L.t.acc[q] = 0;
    g.sync();
    if (!ra.n_steps) return;
    split_draws(a, L, g, tile_lo, tile_n, ra.t0);
    // events of delay >= 2 arriving at t0 were filed by the previous launch
    uint64_t pre = split_drain(a, ra, L, g, x, c, false, (uint32_t)(ra.t0 % a.pslots));
    const uint32_t R = ra.R;
    // with a smallest delay above one step nothing filed at t arrives at t + 1
    const bool split = a.dmin == 1;
    for (uint64_t s = 0; s < ra.n_steps; s++) {
        const uint64_t t = ra.t0 + s;
        if (s > 0) {
            // split: the critical phase of t - 1 is done on this XCD (which
            // implies every tile published t - 1).  Otherwise wait for that
            // publication itself: a tile may not count step t before every
            // tile has counted t - 1, or the per-XCD counts would mix steps.
            if (g.w == 0) {
                const bool ok = split ? split_spin_all(&ctl->critp[x * kRunMaxR], R, (uint32_t)s, &ctl->abort_flag)
                                      : split_spin(&ctl->gen, (uint32_t)s, &ctl->abort_flag);
                if (g.tid == 0) {
                    L.t.stop = ok ? 0u : 1u;
                    if (!ok) atomicOr(a.flags, kSplitStoppedFlag);
                    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
                    __builtin_amdgcn_s_waitcnt(0);
                }
            }
            g.sync();
            if (L.t.stop) return;
        }
        const uint32_t pslot = (uint32_t)(t % a.pslots);
        uint64_t delivered = pre + (split ? split_drain(a, ra, L, g, x, c, true, 0u) : 0ull);
        split_overflow(a, L, g, tile, tile_n, pslot);
        if (g.tid == 0) L.t.nspk = 0;
        g.sync();
        split_update(a, L, g, x, tile, tile_lo, tile_n, t, delivered, (uint32_t)(t % a.spk_slots));
        // publish: every store of the role has completed, then count the tile
        __builtin_amdgcn_s_waitcnt(0);
        g.sync();
        if (g.tid == 0) {
            const uint32_t e = (uint32_t)s + 1;
            const uint32_t o = atomicAdd(&ctl->gx[x * kCtlStride], 1u);
            if (o == tl.T8 * e - 1) {
                const uint32_t gg = atomicAdd(&ctl->gcnt, 1u);
                if (gg == kGroups * e - 1) st_ag(&ctl->gen, e);
            }
        }
        if (s + 1 == ra.n_steps) break;
        // next step: draws, then the bulk pages of arrival t + 1 (complete
        // once the bulk phase of t - 1 is done)
        for (uint32_t q = g.tid; q < tl.W; q += kRoleThreads) L.t.acc[q] = 0;
        split_draws(a, L, g, tile_lo, tile_n, t + 1);
        if (g.w == 0) {  // the bulk phase of t - 1 is done by every push block of the XCD
            const bool ok = split_spin_all(&ctl->bulkp[x * kRunMaxR], R, (uint32_t)s, &ctl->abort_flag);
            if (g.tid == 0) {
                L.t.stop = ok ? 0u : 1u;
                if (!ok) atomicOr(a.flags, kSplitStoppedFlag);
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
                __builtin_amdgcn_s_waitcnt(0);
            }
        }
        g.sync();
        if (L.t.stop) return;
        pre = split_drain(a, ra, L, g, x, c, false, (uint32_t)((t + 1) % a.pslots));
    }
    for (uint32_t q = g.tid; q < tile_n; q += kRoleThreads) {
        a.V[tile_lo + q] = L.t.V[q];
        if (m.kind != SPK_SOURCE) a.ref[tile_lo + q] = L.t.ref[q];
    }
}

// ---------------------------------------------------------------- push role

// File the events of the runs in L.p.plen / L.p.pbase (K spikes) into the
// block's pages.  CRIT: bucket = tile c of the group, the critical page of c;
// otherwise bucket = delay index j * T8 + c, the bulk page of arrival slot
// (t + dmin + j) mod pslots.
template <bool FIXED, bool CMP, bool CRIT>
__device__ __forceinline__ void push_runs(const RunArgs &ra, SplitLDS<FIXED, CMP> &L, Role &g, uint32_t x, uint32_t r, uint64_t t,
                          uint32_t K)
{
    using Rec = typename SynRec<CMP>::T;
    constexpr int R = SplitLDS<FIXED, CMP>::R;
    const StepArgs &a = ra.s;
    const uint32_t tid = g.tid, lane = lane_id(), w = g.w;
    const Tiling tl = a.tl;
    const uint32_t NB = CRIT ? tl.T8 : a.lists * tl.T8;
    const uint32_t xlo = x * tl.Gw;
    const uint64_t cap = a.page_cap;
    const uint32_t slot_of_j0 = (uint32_t)((t + a.dmin) % a.pslots);
    uint32_t len = 0;
    uint64_t base = 0;
    if (tid < K) {
        len = L.p.plen[tid];
        base = L.p.pbase[tid];
    }
    uint32_t C;
    const uint32_t nch = (len + kWave - 1) / kWave;
    const uint32_t coff = role_scan_u32(g, nch, L.p.ws, &C);
    constexpr uint32_t kWin = R * kRoleWaves;
    for (uint32_t i0 = 0; i0 < C; i0 += kWin) {
        for (uint32_t q = tid; q < kWin; q += kRoleThreads) L.p.clen[q] = 0;
        g.sync();
        if (tid < K) {
            const uint32_t cb = coff > i0 ? coff : i0, ce = coff + nch < i0 + kWin ? coff + nch : i0 + kWin;
            for (uint32_t q = cb; q < ce; q++) {
                const uint32_t o = (q - coff) * kWave;
                L.p.cbase[q - i0] = base + o;
                L.p.clen[q - i0] = len - o < kWave ? len - o : kWave;
            }
        }
        g.sync();
        Rec rec[R];
        uint32_t okm = 0;
#pragma unroll
        for (int u = 0; u < R; u++) {
            const uint32_t cl = u * kRoleWaves + w;
            const uint32_t ln = L.p.clen[cl];
            const uint64_t cb = L.p.cbase[cl];
            const bool ok = lane < ln;
            const uint64_t idx = ok ? cb + lane : 0ull;
            okm |= (uint32_t)ok << u;
            rec[u] = SynRec<CMP>::load(a, idx);  // unconditional load from a clamped index
        }
#pragma unroll
        for (int h = 0; h < 2; h++) {
            if (i0 + (uint32_t)h * (R / 2) * kRoleWaves >= C) break;
            constexpr int RH = R / 2;
            uint32_t tr[RH];
#pragma unroll
            for (int rr = 0; rr < RH; rr++) {
                const int q = h * RH + rr;
                tr[rr] = 0xffffffffu;
                if (!((okm >> q) & 1u)) continue;
                const uint32_t key = rec_key(rec[q]);
                const uint32_t local = rec_target(key) - xlo;
                const uint32_t b = (CRIT ? 0u : rec_delay(key) * tl.T8) + (local >> tl.logW);
                const uint32_t rank = atomicAdd(&L.p.bcnt[b], 1u);
                tr[rr] = (b << 16) | rank;
                const uint32_t sv = (b << 16) | (local & (tl.W - 1));
                if constexpr (CMP) rec[q] = sv | (rec_class(key) << kPageClassShift);
                else rec[q].x = (int)sv;
            }
            g.sync();
            uint32_t staged;
            {
                const uint32_t P = (NB + kRoleThreads - 1) / kRoleThreads;
                const uint32_t b0 = tid * P;
                uint32_t sum = 0;
                for (uint32_t k = 0; k < P; k++)
                    if (b0 + k < NB) sum += L.p.bcnt[b0 + k];
                uint32_t ex = role_scan_u32(g, sum, h ? L.p.ws : L.p.ws2, &staged);
                for (uint32_t k = 0; k < P; k++) {
                    if (b0 + k < NB) {
                        const uint32_t bb = b0 + k, cnt = L.p.bcnt[bb];
                        uint32_t *f;
                        if (CRIT) {
                            f = &L.p.cfill[bb];
                        } else {
                            const uint32_t j = bb / tl.T8, cc = bb - j * tl.T8;
                            uint32_t sl = slot_of_j0 + j;
                            sl = sl >= a.pslots ? sl - a.pslots : sl;
                            f = &L.p.fill[sl * tl.T8 + cc];
                        }
                        L.p.bst[bb] = ex;
                        L.p.wb[bb] = *f - ex;
                        *f += cnt;
                        L.p.bcnt[bb] = 0;
                        ex += cnt;
                    }
                }
            }
            g.sync();
            Rec *stage = L.p.stage;
#pragma unroll
            for (int rr = 0; rr < RH; rr++) {
                if (tr[rr] == 0xffffffffu) continue;
                stage[L.p.bst[tr[rr] >> 16] + (tr[rr] & 0xffffu)] = rec[h * RH + rr];
            }
            g.sync();
            for (uint32_t q = tid; q < staged; q += kRoleThreads) {
                const Rec r2 = stage[q];
                const uint32_t key = rec_key(r2);
                const uint32_t b = key >> 16, low = key & 0xffffu;
                const uint32_t pos = L.p.wb[b] + q;
                uint32_t page, sl;
                if (CRIT) {
                    page = (x * ra.R + r) * tl.T8 + b;
                    sl = (uint32_t)((t + 1) % a.pslots);
                } else {
                    const uint32_t j = b / tl.T8, cc = b - j * tl.T8;
                    sl = slot_of_j0 + j;
                    sl = sl >= a.pslots ? sl - a.pslots : sl;
                    page = page_of(a, x, r, sl, cc);
                }
                if (pos < cap) {
                    const uint64_t e = (uint64_t)page * cap + pos;
                    if constexpr (CMP) (CRIT ? ra.cpages16 : a.pages16)[e] = (uint16_t)low;
                    else (CRIT ? ra.cpages : a.pages)[e] = make_int2((int)low, r2.y);
                } else {
                    const uint32_t cc = CRIT ? b : b % tl.T8;
                    long long units;
                    uint32_t local;
                    if constexpr (CMP) {
                        units = class_units(a, low >> kPageClassShift);
                        local = low & kPageLocalMask;
                    } else {
                        units = units_of<FIXED>(r2.y, a.m.shift64);
                        local = low;
                    }
                    overflow_add<FIXED, true>(a, sl, x * tl.T8 + cc, local, units);
                }
            }
        }
    }
    g.sync();
}

// The spikes [k0, k1) of the share, one chunk: IDs, row descriptors and the
// run of each row for this pass (critical: the smallest-delay part of group
// x's run; bulk: the rest) into L.p.plen / L.p.pbase.
template <bool FIXED, bool CMP>
__device__ __forceinline__ uint64_t load_chunk(const RunArgs &ra, SplitLDS<FIXED, CMP> &L, Role &g, uint32_t x, uint32_t c0,
                               uint32_t K, uint32_t sslot, bool crit, bool split, uint64_t rbase, bool rec_raster)
{
    const StepArgs &a = ra.s;
    uint64_t emitted = 0;
    if (g.tid < K) {
        const uint32_t k = c0 + g.tid;
        const uint32_t s = spike_at<true>(a, L.p.pre, sslot, k);
        if (rec_raster) a.raster[rbase + k] = s;
        const RowDesc *d = a.desc + s;
        const uint32_t lo = x ? d->gend[x - 1] : 0u, hi = d->gend[x];
        const uint32_t mid = split ? d->dend[x] : lo;  // end of the critical part
        const uint32_t b = crit ? lo : mid, e = crit ? mid : hi;
        L.p.plen[g.tid] = e - b;
        L.p.blen[g.tid] = hi - mid;
        L.p.pbase[g.tid] = d->start + b;
        emitted = d->gend[kGroups - 1];
    }
    g.sync();
    return emitted;
}

template <bool FIXED, bool CMP>
__device__ __forceinline__ void push_role(const RunArgs &ra, SplitLDS<FIXED, CMP> &L, uint32_t x, uint32_t r)
{
    const StepArgs &a = ra.s;
    RunCtl *ctl = ra.ctl;
    const uint32_t rt = threadIdx.x - kRoleThreads;
    Role g{rt, (uint32_t)__builtin_amdgcn_readfirstlane(rt / kWave), 0u, &L.p.bar, &ctl->abort_flag};
    const Tiling tl = a.tl;
    const uint32_t NF = a.pslots * tl.T8;
    for (uint32_t f = g.tid; f < NF; f += kRoleThreads) {
        const uint32_t sl = f / tl.T8;
        L.p.fill[f] = a.pfill[page_of(a, x, r, sl, f - sl * tl.T8)];
    }
    for (uint32_t b = g.tid; b < kSplitMaxBuckets; b += kRoleThreads) L.p.bcnt[b] = 0;
    g.sync();
    // the smallest delay's events are critical only when it is one step
    const bool split = a.dmin == 1;
    uint64_t rbase = a.raster_cap ? a.raster_offs[ra.t0] : 0;
    const uint32_t G1 = ra.R;
    for (uint64_t s = 0; s < ra.n_steps; s++) {
        const uint64_t t = ra.t0 + s;
        if (g.tid == 0) {  // every tile has published the spikes of t
            L.p.stop = split_spin(&ctl->gen, (uint32_t)s + 1, &ctl->abort_flag) ? 0u : 1u;
            if (L.p.stop) atomicOr(a.flags, kSplitStoppedFlag);
        }
        g.sync();
        if (L.p.stop) return;
        const uint32_t sslot = (uint32_t)(t % a.spk_slots);
        const uint32_t M = role_spike_set(g, a, sslot, L.p.pre, L.p.ws);
        const uint32_t k0 = (uint32_t)((uint64_t)M * r / G1), k1 = (uint32_t)((uint64_t)M * (r + 1) / G1);
        const bool rec_raster = a.raster_cap && x == 0 && rbase + M <= a.raster_cap;
        uint64_t emitted = 0;
        // critical phase: events of delay 1, one page per tile
        for (uint32_t c = g.tid; c < tl.T8; c += kRoleThreads) L.p.cfill[c] = 0;
        g.sync();
        for (uint32_t c0 = k0; c0 < k1; c0 += kSplitChunk) {
            const uint32_t K = k1 - c0 < kSplitChunk ? k1 - c0 : kSplitChunk;
            emitted += load_chunk(ra, L, g, x, c0, K, sslot, true, split, rbase, rec_raster);
            if (split) push_runs<FIXED, CMP, true>(ra, L, g, x, r, t, K);
        }
        for (uint32_t c = g.tid; c < tl.T8; c += kRoleThreads) ra.cfill[(x * G1 + r) * tl.T8 + c] = L.p.cfill[c];
        __builtin_amdgcn_s_waitcnt(0);
        g.sync();
        if (g.tid == 0) st_ag(&ctl->critp[x * kRunMaxR + r], (uint32_t)s + 1);
        // bulk phase: the other delays, pages per (arrival slot, tile)
        const uint32_t s0 = (uint32_t)(t % a.pslots);
        for (uint32_t c = g.tid; c < tl.T8; c += kRoleThreads) L.p.fill[s0 * tl.T8 + c] = 0;
        g.sync();  // the reset is read by other threads (pushes, publish) even with no spikes
        const bool one_chunk = k1 - k0 <= kSplitChunk;
        for (uint32_t c0 = k0; c0 < k1; c0 += kSplitChunk) {
            const uint32_t K = k1 - c0 < kSplitChunk ? k1 - c0 : kSplitChunk;
            if (one_chunk) {  // the chunk's runs are in LDS: the bulk run follows the critical one
                if (g.tid < K) {
                    L.p.pbase[g.tid] += L.p.plen[g.tid];
                    L.p.plen[g.tid] = L.p.blen[g.tid];
                }
                g.sync();
            } else {
                load_chunk(ra, L, g, x, c0, K, sslot, false, split, rbase, false);
            }
            push_runs<FIXED, CMP, false>(ra, L, g, x, r, t, K);
        }
        for (uint32_t f = g.tid; f < NF; f += kRoleThreads) {
            const uint32_t sl = f / tl.T8;
            a.pfill[page_of(a, x, r, sl, f - sl * tl.T8)] = L.p.fill[f];
        }
        if (x == 0) {
            const uint64_t tot = role_sum_u64(g, emitted, L.p.ws64);
            if (g.tid == 0 && tot) atomicAdd((unsigned long long *)&a.events8[t * kGroups], (unsigned long long)tot);
        }
        if (a.raster_cap) {
            const bool ok = rbase + M <= a.raster_cap;
            if (x == 0 && r == 0 && g.tid == 0) {
                a.raster_offs[t + 1] = ok ? rbase + M : rbase;
                if (!ok) atomicOr(a.flags, 2u);
            }
            rbase = ok ? rbase + M : rbase;
        }
        __builtin_amdgcn_s_waitcnt(0);
        g.sync();
        if (g.tid == 0) st_ag(&ctl->bulkp[x * kRunMaxR + r], (uint32_t)s + 1);
    }
}

template <bool FIXED, bool CMP>
__global__ __launch_bounds__(kSplitThreads) void k_split(RunArgs ra)
{
    __shared__ SplitLDS<FIXED, CMP> L;
    const StepArgs &a = ra.s;
    RunCtl *ctl = ra.ctl;
    const uint32_t tid = threadIdx.x;
    if (tid == 0) {
        const uint32_t raw = xcc_id_split();
        const uint32_t x = raw & (kGroups - 1);
        if (raw >= kGroups) atomicOr(&ctl->abort_flag, kRunAbortPlacement);
        L.x = x;
        L.r = atomicAdd(&ctl->ticket[x * kCtlStride], 1u);
        L.t.bar = 0;
        L.p.bar = 0;
        L.t.stop = 0;
        L.p.stop = 0;
        atomicAdd(&ctl->start, 1u);
        L.stop = split_spin(&ctl->start, gridDim.x, &ctl->abort_flag) ? 0u : 1u;
        if (L.stop) atomicOr(a.flags, kSplitStoppedFlag);
    }
    __syncthreads();
    if (L.stop) return;
    if (tid < kGroups && ld_ag(&ctl->ticket[tid * kCtlStride]) != ra.R) atomicOr(&L.stop, 1u);
    if (tid == 0 && ld_ag(&ctl->abort_flag)) atomicOr(&L.stop, 1u);
    __syncthreads();
    if (L.stop) {
        if (tid == 0) {
            atomicOr(&ctl->abort_flag, kRunAbortPlacement);
            atomicOr(a.flags, kSplitStoppedFlag);
        }
        return;
    }
    const uint32_t x = L.x, r = L.r;
    if (tid < kRoleThreads) {
        if (r < a.tl.T8) tile_role(ra, L, x, r);
    } else {
        push_role(ra, L, x, r);
    }
    if (tid == 0 && x == 0 && r == 0) *(uint64_t *)a.t_base = ra.t0 + ra.n_steps;
}

template <bool FIXED, bool CMP>
hipError_t launch_split_t(const RunArgs &ra, hipStream_t s)
{
    RunArgs arg = ra;
    void *args[] = {&arg};
    return hipLaunchCooperativeKernel((const void *)k_split<FIXED, CMP>, dim3(kGroups * ra.R),
                                      dim3(kSplitThreads), args, 0, s);
}

}  // namespace

bool split_supported(const StepArgs &a, uint32_t R)
{
    const Tiling &tl = a.tl;
    if (a.direct || R == 0 || R > kRunMaxR || tl.T8 > R || tl.T != kGroups * tl.T8 || tl.W > kMaxTileW) return false;
    if (a.m.pois_len > 256 || a.pg1 != R || a.spk_slots < 3 || a.page_cap % 16) return false;
    if (a.lists * tl.T8 > kSplitMaxBuckets || a.pslots * tl.T8 > kSplitMaxBuckets) return false;
    // LDS: 8-byte records with 64-bit accumulators do not fit beside each other
    return a.compact || a.m.fixed;
}

hipError_t launch_split(const RunArgs &ra, hipStream_t s)
{
    const StepArgs &a = ra.s;
    if (!split_supported(a, ra.R) || !ra.cfill) return hipErrorInvalidValue;
    if (a.compact ? !a.syn32 || !a.pages16 || !ra.cpages16 : !a.syn || !a.pages || !ra.cpages)
        return hipErrorInvalidValue;
    if (a.m.fixed) {
        if (a.compact) return launch_split_t<true, true>(ra, s);
        return launch_split_t<true, false>(ra, s);
    }
    if (a.compact) return launch_split_t<false, true>(ra, s);
    return hipErrorInvalidValue;
}

}  // namespace spk
