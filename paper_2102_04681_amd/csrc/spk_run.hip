// spk_run.hip -- the persistent step kernel: many simulation steps in one
// cooperative launch of one workgroup per compute unit.
//
// The step is the same as the graph path's (spk_step.hip): the events that
// arrive at t are summed in LDS, the neurons are updated, the spikes of t are
// compacted, and (binned delivery) the rows of the neurons that fired are read
// once and their events filed by (arrival step, target tile) into pages.  The
// difference is what persists between steps and how the hand-offs happen:
//   - each workgroup keeps its tile's membrane potentials, refractory
//     counters and the next step's Poisson draws in LDS for the whole launch,
//     and (as a push block) the fill counters of the pages it owns;
//   - the two hand-offs of a step happen inside the kernel instead of at
//     kernel boundaries, through progress words (binned delivery): a tile
//     advances its word once it has published its spike list of t (for a
//     one-step batch the word also carries the spike count), and the push
//     blocks start once every tile's word has advanced; a push block
//     advances its word once it has filed its events, and a tile starts its
//     next drain once the 32 words of its XCD have advanced: every page is
//     written and read on one XCD (its L2 is the point of coherence, so only
//     the compute unit's L1 is invalidated there).  Direct delivery has one
//     hand-off per step, a grid barrier;
//   - with binned delivery and a smallest delay of D >= 2 steps, steps run in
//     batches of D: nothing filed in a batch arrives within it, so the tile
//     drains the batch's D arrival slots at once and takes each neuron
//     through the D updates in registers, and one push phase files the
//     events of all D steps' spikes.
// Workgroups find their XCD from the hardware register and take a ticket
// within it, so the group of tiles a workgroup serves is always on the XCD it
// runs on.  Spike lists cross XCDs through agent-scope loads and stores.
//
// Every wait is bounded (10 s of the real-time clock); a workgroup that gives
// up sets an abort flag that every other waiter also polls, so the grid
// always drains.  The host reads the flag after the launch.
//
// The variants for batches of several LIF steps (updates in registers) are
// compiled from this file in a translation unit of their own
// (spk_run_batch.hip, SPK_RUN_BATCH = 1): instantiated beside the one-step
// variants, they changed the compiler's register allocation of those.
#include <hip/hip_runtime.h>

#ifndef SPK_RUN_BATCH
#define SPK_RUN_BATCH 0
#endif

#include "spk_dev.h"

namespace spk {

namespace {

constexpr int kRunThreads = 1024;
static_assert(kRunThreads == (int)kBlockThreads, "the block-wide helpers assume workgroups of kBlockThreads");

// The thread index, opaque to the optimiser: address arithmetic derived from
// it is then recomputed in each phase instead of being hoisted out of the
// step loop, where the kernel has no registers to spare and the hoisted
// values would be spilled (each reload waits for every load in flight).
__device__ __forceinline__ uint32_t tid_here()
{
    uint32_t t = threadIdx.x;
    asm volatile("" : "+v"(t));
    return t;
}
constexpr int kRunRounds = kMaxTileW / kRunThreads;      // neurons per thread
constexpr uint32_t kRunChunk = 256;                      // spikes resolved per push chunk
constexpr uint32_t kRunMaxT = kGroups * kRunMaxR;        // tiles
constexpr uint64_t kSpinTicks = 10ull * 100000000ull;    // 10 s of the 100 MHz clock
constexpr uint32_t kRunStoppedFlag = 4u;                 // sticky in the network's device flags

__device__ __forceinline__ uint32_t xcc_id()
{
    return __builtin_amdgcn_s_getreg((20) | (0 << 6) | ((4 - 1) << 11)) & 0xfu;  // HW_REG_XCC_ID[3:0]
}

// Wait until *p >= target; false if the wait gave up or another workgroup did.
__device__ bool spin_ge(const uint32_t *p, uint32_t target, uint32_t *abort_flag)
{
    const uint64_t t0 = wall_clock64();
    for (uint32_t k = 0;; k++) {
        if (ld_ag(p) >= target) return true;
        if ((k & 31u) == 31u) {
            if (ld_ag(abort_flag)) return false;
            if (wall_clock64() - t0 > kSpinTicks) {
                atomicOr(abort_flag, kRunAbortTimeout);
                return false;
            }
        }
        __builtin_amdgcn_s_sleep(1);
    }
}

// Wait (one wave) until every one of the n <= 64 words p[0..n) has reached
// target (wrap-safe); false if the wait gave up or another workgroup did.
__device__ bool spin_all_ge(const uint32_t *p, uint32_t n, uint32_t target, uint32_t *abort_flag)
{
    const uint32_t lane = lane_id();
    const uint64_t t0 = wall_clock64();
    for (uint32_t k = 0;; k++) {
        const uint32_t v = ld_ag(p + (lane < n ? lane : 0u));
        if (__all(lane >= n || (int32_t)(v - target) >= 0)) return true;
        if ((k & 31u) == 31u) {
            if (ld_ag(abort_flag)) return false;
            if (wall_clock64() - t0 > kSpinTicks) {
                if (lane == 0) atomicOr(abort_flag, kRunAbortTimeout);
                return false;
            }
        }
        __builtin_amdgcn_s_sleep(1);
    }
}

template <bool FIXED, bool CMP>
struct RunLDS {
    using AccT = typename Acc<FIXED>::T;
    using Rec = typename SynRec<CMP>::T;
    static constexpr int R = CMP ? 16 : 8;                // events per thread per window
    static constexpr uint32_t kStageN = R * kRunThreads;  // events bucket-sorted at once (a window)
    // persistent for the whole launch
    float V[kMaxTileW];
    uint8_t ref[kMaxTileW];     // LIF: refractory steps left; source: fires at the current step
    uint8_t kp[kMaxTileW];      // Poisson counts: of the current step, or of step u of a batch at u * W
    uint64_t pois[256];
    uint16_t guide[256];
    uint32_t fill[kRunMaxFill]; // push block: records in each of its pages, (arrival slot, tile)
    union {
        struct {
            AccT acc[kMaxTileW];
            // unused: keeps the arrays below at the LDS offsets the direct
            // gather was measured fastest at (without it 1e6 Bernoulli
            // sources at 10 Hz take 77.7 instead of 75.8 us per step)
            uint16_t pad_[kMaxTileW];
            uint32_t pre[kRunMaxT + 1];                      // binned: chunk prefix; direct: spike prefix
            uint32_t cbase[kRunThreads / kWave * 16];
            uint32_t clen[kRunThreads / kWave * 16];
            uint32_t wpre[kRunThreads / kWave][kWave + 1];
            uint64_t wbeg[kRunThreads / kWave][kWave];
            unsigned long long dlv[kRunMaxD];  // binned: events delivered at each step of the batch
            uint32_t ovfm;                     // binned: bit u: step u of the batch has overflowed events
            uint32_t pfv[kRunMaxR];            // binned, one step: records in each push block's page
            uint32_t nb[kRunMaxD];             // batched update: spikes of each step of the batch
        } t;
        struct {
            Rec stage[kStageN];
            uint32_t pre[kRunMaxT * kRunMaxD + 1];  // spikes before segment (step of the batch, tile)
            uint32_t uslot[kRunMaxD];               // spike-list slot of each step of the batch
            unsigned long long emit[kRunMaxD];      // events emitted per step of the batch
            unsigned long long rbu[kRunMaxD];       // raster position of spike k of step u: rbu[u] + k
            uint32_t rokm;                          // bit u: the spikes of step u fit in the raster
            uint64_t cbase[R * (kRunThreads / kWave)];
            uint32_t clen[R * (kRunThreads / kWave)];
            uint32_t bcnt[kRunMaxBuckets];  // events per bucket in this window, then rank cursor
            uint32_t bst[kRunMaxBuckets];   // bucket starts in the stage
            uint32_t wb[kRunMaxBuckets];    // page position of stage entry q is wb[b] + q
            uint32_t pb[kRunMaxBuckets];    // first record of the bucket's page (pages x capacity < 2^32)
        } p;
    } u;
    uint32_t ws[16], ws2[16];
    unsigned long long ws64[16];
    uint32_t mstep[kRunMaxD];   // spikes of each step of the last pushed batch
    uint32_t nspk2[3];          // spike counters of the update, alternating between steps; [2] = 0
    uint32_t pstop[4];          // wait_tiles: a polling wave gave up
    uint32_t pq[2][4];          // look_tiles: a polling wave saw its words complete (by look parity)
    uint32_t ptot[4];           // one-step batches: the spikes of each polling wave's 64 tiles
    uint32_t x, r, stop;
    // the neuron model's constants, read by the update from here into vector
    // registers (kept in scalar registers they spill across the long kernel)
    float mk, v_rest, v_th, v_reset, i_bias, ext_w;
    int32_t ext_wq, bias_q, shift, shift64;
    uint32_t ref_steps, pois_len;
    // compact records: accumulator units of each weight class, read by the
    // drain with one LDS load per record instead of a chain of selects among
    // kernel arguments
    long long wtab[kMaxClasses];
    // the per-step statistics of the tile's last step (thread 0's), added to
    // the global counters after the tile's publication, which then does
    // not wait for these atomics (nothing orders them with it)
    uint32_t st_ns;
    unsigned long long st_ev, st_dlv;
};

// Per-step draws of the tile's neurons for steps t .. t + nsteps - 1: the
// Poisson count of step t + u at kp[u * W + q] and, for source neurons (one
// step at a time), whether they fire.  They do not depend on the network's
// activity, so they are computed while the workgroup waits at a barrier.
template <bool FIXED, bool CMP>
__device__ void run_draws(const StepArgs &a, RunLDS<FIXED, CMP> &L, uint32_t tile_lo, uint32_t tile_n,
                          uint64_t t, uint32_t nsteps)
{
    const ModelArgs &m = a.m;
    const uint32_t W = a.tl.W;
    for (uint32_t u = 0; u < nsteps; u++) {
#pragma unroll
        for (int r = 0; r < kRunRounds; r++) {  // (unrolled: the rounds' hashes are independent)
            const uint32_t q = r * kRunThreads + threadIdx.x;
            if (q >= tile_n) continue;
            const uint32_t gi = tile_lo + q;
            if (m.pois_len) {  // K = min { k : hi32 < T_k }, searched from the guide entry
                const uint32_t h = hash_hi32(step_hash(m.keys.pois, gi, t + u));
                uint32_t k = L.guide[h >> 24];
                while ((uint64_t)h >= L.pois[k]) k++;
                L.kp[u * W + q] = (uint8_t)k;
            }
            if (m.kind == SPK_SOURCE)
                L.ref[q] = (uint64_t)hash_hi32(step_hash(m.keys.bern, gi, t)) < m.src_thr ? 1 : 0;
        }
    }
}

// The same draws one round of one step at a time (unit k: step k / nr, round
// k % nr, nr = draw_units_per_step), so that a workgroup can look at the
// tiles' words between units and stop once its wait is over (measured:
// units of one round see the last tile published sooner than units of two
// or four: 27.7 -> 27.1 us per step on the 3e9-synapse network).
__device__ __forceinline__ uint32_t draw_units_per_step(uint32_t tile_n)
{
    return (tile_n + kRunThreads - 1) / kRunThreads;
}
template <bool FIXED, bool CMP>
__device__ void run_draw_unit(const StepArgs &a, RunLDS<FIXED, CMP> &L, uint32_t tile_lo, uint32_t tile_n,
                              uint64_t t, uint32_t k)
{
    const ModelArgs &m = a.m;
    const uint32_t W = a.tl.W, nr = draw_units_per_step(tile_n), u = k / nr, j = k - u * nr;
    const uint32_t q = j * kRunThreads + threadIdx.x;
    if (q >= tile_n) return;
    const uint32_t gi = tile_lo + q;
    if (m.pois_len) {
        const uint32_t h = hash_hi32(step_hash(m.keys.pois, gi, t + u));
        uint32_t kk = L.guide[h >> 24];
        while ((uint64_t)h >= L.pois[kk]) kk++;
        L.kp[u * W + q] = (uint8_t)kk;
    }
    if (m.kind == SPK_SOURCE)
        L.ref[q] = (uint64_t)hash_hi32(step_hash(m.keys.bern, gi, t)) < m.src_thr ? 1 : 0;
}

// Grid barrier: every workgroup's stores have completed before it arrives.
// The last arrival of an XCD counts the XCD; the last XCD releases epoch e
// into every XCD's copy of the release word.
// Between arriving and waiting, the workgroup computes the next step's draws.
template <bool FIXED, bool CMP>
__device__ bool grid_sync(const RunArgs &ra, RunLDS<FIXED, CMP> &L, uint32_t x, uint32_t e, bool draws,
                          uint32_t tile_lo, uint32_t tile_n, uint64_t t_draw, uint32_t n_draw)
{
    RunCtl *c = ra.ctl;
    __builtin_amdgcn_s_waitcnt(0);  // this thread's stores have completed
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t o = atomicAdd(&c->gx[x * kCtlStride], 1u);
        if (o == ra.R * e - 1) {
            const uint32_t g = atomicAdd(&c->gcnt, 1u);
            if (g == kGroups * e - 1)
                for (uint32_t xx = 0; xx < kGroups; xx++) st_ag(&c->gen[xx * kTileWordStride], e);
        }
    }
    if (draws) run_draws(ra.s, L, tile_lo, tile_n, t_draw, n_draw);
    if (threadIdx.x == 0) {
        L.stop = spin_ge(&c->gen[x * kTileWordStride], e, &c->abort_flag) ? 0u : 1u;
        if (L.stop) atomicOr(ra.s.flags, kRunStoppedFlag);
    }
    __syncthreads();
    return L.stop == 0;
}

// End of a push phase (binned delivery): every thread's page and fill
// stores have completed, then the block's progress word advances to e.
__device__ void publish_push(const RunArgs &ra, uint32_t x, uint32_t r, uint32_t e)
{
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) st_ag(&ra.ctl->pushp[x * kRunMaxR + r], e);
}

// End of a tile phase (binned delivery): every thread's spike-list stores
// have completed, then the tile's progress word of batch parity e & 1 takes
// the stamp of batch e and the spike count ns of its step (one-step batches;
// 0 otherwise).
__device__ void publish_tile(const RunArgs &ra, uint32_t tile, uint32_t e, const uint32_t *ns)
{
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) st_ag(&ra.ctl->tilep[e & 1u][tile * kTileWordStride], e << kTileCntBits | *ns);
}

// Wait (one wave) until each of the n <= 64 words p[0..n) carries the stamp e
// in its bits kTileCntBits and up; leaves lane k's word in *v.  On entry *v
// holds the lane's word as last seen: a lane whose word already carries e
// loads it no more.  False if the wait gave up or another workgroup did.
__device__ bool spin_all_stamp(const uint32_t *p, uint32_t n, uint32_t e, uint32_t *abort_flag, uint32_t *v)
{
    const uint32_t lane = lane_id(), want = e & (0xffffffffu >> kTileCntBits);
    const uint64_t t0 = wall_clock64();
    for (uint32_t k = 0;; k++) {
        if (lane < n && (*v >> kTileCntBits) != want) *v = ld_ag(p + lane * kTileWordStride);
        if (__all(lane >= n || (*v >> kTileCntBits) == want)) return true;
        if ((k & 31u) == 31u) {
            if (ld_ag(abort_flag)) return false;
            if (wall_clock64() - t0 > kSpinTicks) {
                if (lane == 0) atomicOr(abort_flag, kRunAbortTimeout);
                return false;
            }
        }
        __builtin_amdgcn_s_sleep(1);
    }
}

// A polling wave's part of a one-step batch's spike prefix, from the words
// of its tiles w * 64 .. w * 64 + n - 1 (all lanes active): the exclusive
// prefix of their spike counts (each at most W) at pre[w * 64 + lane], their
// sum at ptot[w]; load_spike_batch adds the sums of the waves before.
template <bool FIXED, bool CMP>
__device__ __forceinline__ void poller_prefix(RunLDS<FIXED, CMP> &L, uint32_t w, uint32_t lane, uint32_t n,
                                              uint32_t v, uint32_t W)
{
    uint32_t cnt = lane < n ? v & ((1u << kTileCntBits) - 1u) : 0u;
    cnt = cnt < W ? cnt : W;
    const uint32_t inc = wave_scan_incl_u32(cnt);
    if (lane < n) L.u.p.pre[w * kWave + lane] = inc - cnt;
    if (lane == kWave - 1) L.ptot[w] = inc;
}

// Start of a push phase (binned delivery): waves 0-3 wait until the progress
// word of every tile (64 per wave) carries batch e: then every spike list of
// the batch is complete, and every tile has drained the pages of the batch's
// arrival steps, which this push phase may start to refill.  For a one-step
// batch the words' spike counts go into the spike prefix (poller_prefix).
// Words are kept per batch parity: a tile publishes batch e + 1 only after
// the push phases of batch e of its own XCD, and batch e + 2 only after
// those of batch e + 1 of every XCD, so the words of parity e & 1 still hold
// batch e for every push block that waits for it.
// pv: the polling lane's word as last seen (look_tiles), updated here.
template <bool FIXED, bool CMP>
__device__ bool wait_tiles(const RunArgs &ra, RunLDS<FIXED, CMP> &L, uint32_t e, bool counts, uint32_t &pv)
{
    RunCtl *c = ra.ctl;
    const uint32_t T = ra.s.tl.T, w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    if (w * kWave < T) {
        const uint32_t n = T - w * kWave < kWave ? T - w * kWave : kWave, lane = lane_id();
        const bool ok = spin_all_stamp(&c->tilep[e & 1u][w * kWave * kTileWordStride], n, e, &c->abort_flag, &pv);
        if (counts && ok) poller_prefix(L, w, lane, n, pv, ra.s.tl.W);
        if (lane == 0) {
            L.pstop[w] = ok ? 0u : 1u;
            if (!ok) atomicOr(ra.s.flags, kRunStoppedFlag);
        }
    }
    __syncthreads();
    uint32_t stop = 0;
    for (uint32_t k = 0; k * kWave < T; k++) stop |= L.pstop[k];
    return stop == 0;
}

// One look at the tiles' progress words (as wait_tiles, without waiting),
// with work() done while the loads are in flight: true if every tile has
// published batch e (and then, with counts, the spike prefix is in place).
// pv: the polling lane's word as last seen; a lane whose word already
// carries batch e loads it no more (fewer loads from every workgroup while
// the last tiles finish).
template <bool FIXED, bool CMP, class Work>
__device__ bool look_tiles(const RunArgs &ra, RunLDS<FIXED, CMP> &L, uint32_t e, bool counts, uint32_t par,
                           uint32_t &pv, Work &&work)
{
    const uint32_t T = ra.s.tl.T, w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave), lane = lane_id();
    const bool poller = w * kWave < T;
    const uint32_t n = poller ? (T - w * kWave < kWave ? T - w * kWave : kWave) : 0u;
    const uint32_t want = e & (0xffffffffu >> kTileCntBits);
    if (lane < n && (pv >> kTileCntBits) != want)
        pv = ld_ag(&ra.ctl->tilep[e & 1u][(w * kWave + lane) * kTileWordStride]);
    work();
    if (poller) {
        const bool ok = __all(lane >= n || (pv >> kTileCntBits) == want);
        if (counts && ok) poller_prefix(L, w, lane, n, pv, ra.s.tl.W);
        if (lane == 0) L.pq[par][w] = ok ? 1u : 0u;
    }
    __syncthreads();
    bool all = true;
    for (uint32_t k = 0; k * kWave < T; k++) all = all && L.pq[par][k] != 0;
    return all;  // (pq[par] is written again two looks later, after a barrier)
}

// Start of a tile phase (binned delivery): the first wave waits until every
// push block of the XCD has finished push phase e; then the compute unit's L1
// is invalidated so that plain loads see the pages in the XCD's L2.
template <bool FIXED, bool CMP>
__device__ bool wait_pushes(const RunArgs &ra, RunLDS<FIXED, CMP> &L, uint32_t x, uint32_t e)
{
    RunCtl *c = ra.ctl;
    if (threadIdx.x < kWave) {
        const bool ok = spin_all_ge(&c->pushp[x * kRunMaxR], ra.R, e, &c->abort_flag);
        if (threadIdx.x == 0) {
            L.stop = ok ? 0u : 1u;
            if (!ok) atomicOr(ra.s.flags, kRunStoppedFlag);
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        __builtin_amdgcn_s_waitcnt(0);
    }
    __syncthreads();
    return L.stop == 0;
}

// Tile phase, binned delivery: sum the records of the pages of the Db
// arrival steps t_first .. t_first + Db - 1 (one page per push block of the
// group and step) into the LDS accumulators, those of step u at
// acc[u * W ...].  A table of 64-record chunks of all the pages is built per
// window of kDrain chunks per wave; every wave loads its chunks at once.
// The caller has zeroed acc[0 .. Db * W).  Leaves in L.u.t.dlv the events
// delivered at each step, including any that overflowed into the global
// accumulators (merged here).
// ONE (Db = 1): the first part of every page (an equal number of records per
// page, within the page capacity) is loaded together with the pages' fill
// counters, before the counts are known, and records past a page's count are
// dropped; only the rest of a longer page goes through the chunk tables.
// The pages of an arrival step are not written while it is drained, so the
// records read are the filed ones or stale ones beyond the count.
template <bool FIXED, bool CMP, bool ONE>
__device__ void run_drain(const StepArgs &a, RunLDS<FIXED, CMP> &L, uint32_t x, uint32_t c, uint32_t tile,
                          uint32_t tile_n, uint32_t pslot0, uint32_t Db)
{
    const uint32_t tid = tid_here();
    const Tiling tl = a.tl;
    constexpr uint32_t kPer = CMP ? 2u : 1u;
    constexpr uint32_t kChunk = kPer * kWave;
    const uint32_t cap = a.page_cap, G1 = a.pg1, P = Db * G1;
    // (pslot0: the arrival slot of the first step; Db <= pslots: one wrap at most)
    // thread p < P: page p = u * G1 + g, push block g's page of arrival step t_first + u
    const uint32_t pu = ONE || tid >= P ? 0u : tid / G1, pg = tid < P ? tid - pu * G1 : 0u;
    const uint32_t psl = pslot0 + pu < a.pslots ? pslot0 + pu : pslot0 + pu - a.pslots;
    const uint32_t page = page_of(a, x, pg, psl, c);
    uint32_t pf = a.pfill[page];
    // thread u < Db: the overflow flag of (arrival step t_first + u, tile)
    const uint32_t osl = tid < Db ? (pslot0 + tid < a.pslots ? pslot0 + tid : pslot0 + tid - a.pslots) : 0u;
    uint32_t ovf = ld_ag(&a.ovf_flag[(uint64_t)osl * tl.T + tile]);
    // the wave index is uniform: held in a scalar register, the chunk-table
    // addresses below cost no vector registers
    const uint32_t w = __builtin_amdgcn_readfirstlane(tid / kWave), lane = tid & (kWave - 1);
    constexpr uint32_t nw = kRunThreads / kWave;
    // ONE, full records: chunk q = u * nw + w of the speculative loads is
    // chunk q % spc of push block q / spc's page.  Compact records: 2 nw load
    // slots of 512 records (one 16-byte load per lane: the same bytes in a
    // quarter of the load instructions, which the compute unit's queue of
    // loads in flight admits at once), two per wave; slot v = 2 w + j is part
    // v % lpp of push block v / lpp's page.  spc * kChunk records per page (S)
    constexpr int kSpecU = CMP ? 2 : 16;
    constexpr uint32_t kSlotRec = 8u * kWave;  // compact: records per load slot
    const uint32_t lpp = CMP ? kSpecU * nw / G1 : 1u;
    const uint32_t spc = ONE ? (CMP ? lpp * (kSlotRec / kChunk) : kSpecU * nw / G1) : 1u, S = spc * kChunk;
    // q / spc for q < 256 as (q * spc_inv) >> 16: exact, since q (spc_inv -
    // 2^16 / spc) spc < q spc < 2^16 (a division per chunk cost ~0.5 us per
    // step); v / lpp the same way
    const uint32_t spc_inv = (65536u + spc - 1u) / spc, lpp_inv = (65536u + lpp - 1u) / lpp;
    using Ld = typename std::conditional<CMP, uint4, int2>::type;
    Ld sr[ONE ? kSpecU : 1];
    if constexpr (ONE) {
#pragma unroll
        for (int u = 0; u < kSpecU; u++) {
            if constexpr (CMP) {
                const uint32_t v = kSpecU * w + u, g = (v * lpp_inv) >> 16, o = (v - g * lpp) * kSlotRec + lane * 8u;
                const bool ok = g < G1 && o < cap;  // (cap is a multiple of 16: all 8 records of a lane)
                const uint32_t idx = ok ? (page_of(a, x, g, pslot0, c) * cap + o) / 8u : 0u;
                sr[u] = ((const uint4 *)a.pages16)[idx];
            } else {
                const uint32_t q = u * nw + w, g = (q * spc_inv) >> 16, o = (q - g * spc) * kChunk + lane * kPer;
                const bool ok = g < G1 && o < cap;
                sr[u] = a.pages[ok ? page_of(a, x, g, pslot0, c) * cap + o : 0u];
            }
        }
    }
    ovf = tid < Db ? ovf : 0u;
    if (tid < Db) L.u.t.dlv[tid] = 0;
    if (tid == 0) L.u.t.ovfm = 0;
    pf = tid < P ? pf : 0u;
    const uint32_t ne_all = pf < cap ? pf : cap;
    if (ONE && tid < kRunMaxR) L.u.t.pfv[tid] = ne_all;
    // records left for the chunk tables (ONE: those past the speculative part)
    const uint32_t o0 = ONE ? S : 0u;
    const uint32_t ne = ne_all > o0 ? ne_all - o0 : 0u;
    uint32_t C;
    // chunks of the chunk tables: compact records 512 (one 16-byte load per
    // lane), full records 64 (one 8-byte load per lane)
    constexpr uint32_t kPerL = CMP ? 8u : 1u, kChunkL = kPerL * kWave;
    const uint32_t cex = block_scan_u32((ne + kChunkL - 1) / kChunkL, L.ws, &C);  // (publishes the resets)
    if (pf) atomicAdd(&L.u.t.dlv[pu], (unsigned long long)pf);
    if (ovf) atomicOr(&L.u.t.ovfm, 1u << tid);
    if constexpr (ONE) {
#pragma unroll
        for (int u = 0; u < kSpecU; u++) {
            if constexpr (CMP) {
                const uint32_t v = kSpecU * w + u, g = (v * lpp_inv) >> 16, o = (v - g * lpp) * kSlotRec + lane * 8u;
                const uint32_t f = g < G1 ? L.u.t.pfv[g] : 0u;
                const uint32_t wd[4] = {sr[u].x, sr[u].y, sr[u].z, sr[u].w};
#pragma unroll
                for (int k = 0; k < 4; k++) {
                    // both records' units read before either add
                    const uint32_t r0 = wd[k] & 0xffffu, r1 = wd[k] >> 16;
                    const long long u0 = L.wtab[(r0 >> kPageClassShift) & (kMaxClasses - 1)];
                    const long long u1 = L.wtab[(r1 >> kPageClassShift) & (kMaxClasses - 1)];
                    if (o + 2 * k < f) Acc<FIXED>::add(&L.u.t.acc[r0 & kPageLocalMask], u0);
                    if (o + 2 * k + 1 < f) Acc<FIXED>::add(&L.u.t.acc[r1 & kPageLocalMask], u1);
                }
            } else {
                const uint32_t q = u * nw + w, g = (q * spc_inv) >> 16, o = (q - g * spc) * kChunk + lane * kPer;
                const uint32_t f = g < G1 ? L.u.t.pfv[g] : 0u;
                if (o < f) Acc<FIXED>::add(&L.u.t.acc[(uint32_t)sr[u].x], units_of<FIXED>(sr[u].y, a.m.shift64));
            }
        }
    }
    // chunks per wave and window: the same registers for both formats
    constexpr int kDrain = CMP ? 4 : 16;
    constexpr uint32_t kWin = kDrain * nw;
    const uint32_t nchp = (ne + kChunkL - 1) / kChunkL;
    for (uint32_t i0 = 0; i0 < C; i0 += kWin) {
        for (uint32_t q = tid; q < kWin; q += kRunThreads) L.u.t.clen[q] = 0;
        lds_sync();
        if (tid < P) {
            const uint32_t cb = cex > i0 ? cex : i0, ce = cex + nchp < i0 + kWin ? cex + nchp : i0 + kWin;
            // (16-byte aligned for compact records: cap is a multiple of 16, o0 of 8)
            const uint32_t pbase = page * cap + o0;
            for (uint32_t q = cb; q < ce; q++) {
                const uint32_t o = (q - cex) * kChunkL;
                L.u.t.cbase[q - i0] = (pbase + o) / kPerL;
                L.u.t.clen[q - i0] = (ne - o < kChunkL ? ne - o : kChunkL) | (pu << 16);
            }
        }
        lds_sync();
        if constexpr (CMP) {
            const uint4 *pq = (const uint4 *)a.pages16;
            uint4 rr[kDrain];
            uint32_t okm = 0;  // bit 8u + i: record i of the lane's 8 in chunk u
#pragma unroll
            for (int u = 0; u < kDrain; u++) {
                const uint32_t cw = u * nw + w;
                const uint32_t len = L.u.t.clen[cw] & 0xffffu, cb = L.u.t.cbase[cw];
                const uint32_t o = lane * kPerL;
                const uint32_t nv = o < len ? (len - o < kPerL ? len - o : kPerL) : 0u;
                okm |= ((1u << nv) - 1u) << (8 * u);
                rr[u] = pq[nv ? cb + lane : 0u];  // unconditional load from a clamped index
            }
#pragma unroll
            for (int u = 0; u < kDrain; u++) {
                const uint32_t ao = (L.u.t.clen[u * nw + w] >> 16) << tl.logW;
                const uint32_t wd[4] = {rr[u].x, rr[u].y, rr[u].z, rr[u].w};
#pragma unroll
                for (int k = 0; k < 4; k++) {
                    const uint32_t r0 = wd[k] & 0xffffu, r1 = wd[k] >> 16;
                    const long long u0 = L.wtab[(r0 >> kPageClassShift) & (kMaxClasses - 1)];
                    const long long u1 = L.wtab[(r1 >> kPageClassShift) & (kMaxClasses - 1)];
                    if ((okm >> (8 * u + 2 * k)) & 1u) Acc<FIXED>::add(&L.u.t.acc[ao + (r0 & kPageLocalMask)], u0);
                    if ((okm >> (8 * u + 2 * k + 1)) & 1u)
                        Acc<FIXED>::add(&L.u.t.acc[ao + (r1 & kPageLocalMask)], u1);
                }
            }
        } else {
            int2 rr[kDrain];
            uint32_t okm = 0;
#pragma unroll
            for (int u = 0; u < kDrain; u++) {
                const uint32_t cw = u * nw + w;
                const uint32_t len = L.u.t.clen[cw] & 0xffffu, cb = L.u.t.cbase[cw];
                const bool ok = lane < len;
                const uint32_t idx = ok ? cb + lane : 0u;
                okm |= (uint32_t)ok << u;
                rr[u] = a.pages[idx];
            }
#pragma unroll
            for (int u = 0; u < kDrain; u++)
                if ((okm >> u) & 1u) {
                    const uint32_t ao = (L.u.t.clen[u * nw + w] >> 16) << tl.logW;
                    Acc<FIXED>::add(&L.u.t.acc[ao + (uint32_t)rr[u].x], units_of<FIXED>(rr[u].y, a.m.shift64));
                }
        }
        lds_sync();
    }
    lds_sync();  // the counts and flags above are complete (also when there was no chunk)
    const uint32_t om = L.u.t.ovfm;
    if (om) {  // events that did not fit their page, accumulated by global atomics
        for (uint32_t u = 0; u < Db; u++) {
            if (!((om >> u) & 1u)) continue;
            const uint32_t sl = pslot0 + u < a.pslots ? pslot0 + u : pslot0 + u - a.pslots;
            const uint64_t st = (uint64_t)sl * tl.T + tile;
            for (uint32_t q = tid; q < tile_n; q += kRunThreads) {
                const uint64_t gi = st * tl.W + q;
                if (FIXED) {
                    int32_t *o = (int32_t *)a.acc_ovf + gi;
                    L.u.t.acc[u * tl.W + q] += (int32_t)ld_ag((const uint32_t *)o);
                    st_ag((uint32_t *)o, 0u);
                } else {
                    unsigned long long *o = (unsigned long long *)a.acc_ovf + gi;
                    L.u.t.acc[u * tl.W + q] += __hip_atomic_load(o, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_store(o, 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
            }
            if (tid == 0) st_ag(&a.ovf_flag[st], 0u);
        }
    }
}

// A step's spike, event and delivery counts of one tile added to the
// group's global counters (global atomics, thread 0).
__device__ __forceinline__ void step_stats(const StepArgs &a, uint32_t x, uint64_t t, uint32_t ns,
                                           unsigned long long ev, unsigned long long dlv)
{
    if (ns) atomicAdd(&a.counts8[t * kGroups + x], ns);
    if (ev) atomicAdd((unsigned long long *)&a.events8[t * kGroups + x], ev);
    if (dlv) atomicAdd((unsigned long long *)&a.delivered8[t * kGroups + x], dlv);
}

// Forward Euler step of the membrane in single precision (Sec. IV-A; the
// delta-current LIF reading, each operation rounded on its own):
// (V + k (v_rest - V)) + I.
__device__ __forceinline__ float lif_integrate(float V, float I, float mk, float v_rest)
{
    const float av = __fsub_rn(v_rest, V);
    const float bv = __fmul_rn(mk, av);
    const float cv = __fadd_rn(V, bv);
    return __fadd_rn(cv, I);
}

// One LIF step with threshold, reset and refractory count; true if the neuron
// fires.  Without branches: the membrane is integrated for refractory neurons
// too and the result dropped, so that all lanes of a wave run the same
// instructions (a wave nearly always holds both kinds of neuron).
__device__ __forceinline__ bool lif_step(float &V, uint32_t &r, float I, float mk, float v_rest, float v_th,
                                         float v_reset, uint32_t ref_steps)
{
    const float vn = lif_integrate(V, I, mk, v_rest);
    const bool refr = r > 0;
    const bool fire = !refr && vn >= v_th;
    V = refr || fire ? v_reset : vn;
    r = refr ? r - 1u : (fire ? ref_steps : 0u);
    return fire;
}

// Tile phase: the update of the tile's neurons from the LDS accumulators, the
// state and the draws in LDS (input: the accumulators from acc[aoff] on);
// spikes compacted by wavefront ballots straight into the tile's segment of
// the spike list of t.
template <bool FIXED, bool CMP, bool DIRECT>
__device__ void run_update(const RunArgs &ra, RunLDS<FIXED, CMP> &L, uint32_t x, uint32_t tile,
                           uint32_t tile_lo, uint32_t tile_n, uint64_t t, uint32_t tslot, uint64_t delivered,
                           uint32_t aoff, uint32_t kpoff, uint32_t *cnt, uint32_t *cnt_next, bool late)
{
    const StepArgs &a = ra.s;
    const ModelArgs &m = a.m;
    const uint32_t tid = threadIdx.x, lane = lane_id();
    // the model's constants from LDS (vector registers), see RunLDS
    const float mk = L.mk, v_rest = L.v_rest, v_th = L.v_th, v_reset = L.v_reset, i_bias = L.i_bias,
                ext_w = L.ext_w;
    const int32_t ext_wq = L.ext_wq, bias_q = L.bias_q, shift = L.shift, shift64 = L.shift64;
    const uint32_t ref_steps = L.ref_steps, pois_len = L.pois_len;
    uint64_t ev = 0;
    uint64_t bal[kRunRounds];  // per round: the wave's firing lanes (wave-uniform)
    uint32_t nw_spk = 0;       // the wave's spikes over all rounds
    if constexpr (!DIRECT) {
        // binned delivery: the rounds of one neuron kind (uniform: chosen
        // once, outside the rounds), the LIF step without branches
        auto rounds = [&](auto src_tag) {
            constexpr bool SRC = decltype(src_tag)::value;
#pragma unroll
            for (int u = 0; u < kRunRounds; u++) {
                const uint32_t q = u * kRunThreads + tid;
                bool spk = false;
                if (q < tile_n) {
                    const uint32_t kq = L.kp[kpoff + q];  // (read unconditionally: a select, not a branch)
                    const uint32_t K = pois_len ? kq : 0u;
                    float I;
                    if (FIXED) {
                        const int32_t qt = (int32_t)L.u.t.acc[aoff + q] + (int32_t)K * ext_wq + bias_q;
                        I = ldexpf((float)qt, -shift);
                    } else {
                        const float isyn = fixed64_to_float(L.u.t.acc[aoff + q], shift64);
                        const float ext = __fmul_rn((float)K, ext_w);
                        I = __fadd_rn(__fadd_rn(isyn, ext), i_bias);
                    }
                    float V = L.V[q];
                    uint32_t r = L.ref[q];
                    if constexpr (SRC) {
                        V = lif_integrate(V, I, mk, v_rest);
                        spk = r != 0;  // the step's Bernoulli decision
                    } else {
                        spk = lif_step(V, r, I, mk, v_rest, v_th, v_reset, ref_steps);
                        L.ref[q] = (uint8_t)r;
                    }
                    L.V[q] = V;
                }
                bal[u] = __ballot(spk);
                nw_spk += (uint32_t)__popcll(bal[u]);
            }
        };
        if (m.kind == SPK_SOURCE) rounds(std::true_type{});
        else rounds(std::false_type{});
    } else {
        // direct delivery keeps the kind checked per round, with the branches
        // on the refractory count (measured: the hoisted, branch-free rounds
        // cost the gather of 1e6 Bernoulli sources 1.4 us per step, and gain
        // nothing on 2.5e5 LIF neurons)
#pragma unroll
        for (int u = 0; u < kRunRounds; u++) {
            const uint32_t q = u * kRunThreads + tid;
            bool spk = false;
            if (q < tile_n) {
                const uint32_t K = pois_len ? L.kp[kpoff + q] : 0u;
                float I;
                if (FIXED) {
                    const int32_t qt = (int32_t)L.u.t.acc[aoff + q] + (int32_t)K * ext_wq + bias_q;
                    I = ldexpf((float)qt, -shift);
                } else {
                    const float isyn = fixed64_to_float(L.u.t.acc[aoff + q], shift64);
                    const float ext = __fmul_rn((float)K, ext_w);
                    I = __fadd_rn(__fadd_rn(isyn, ext), i_bias);
                }
                float V = L.V[q];
                if (m.kind == SPK_SOURCE) {
                    const float av = __fsub_rn(v_rest, V);
                    const float bv = __fmul_rn(mk, av);
                    const float cv = __fadd_rn(V, bv);
                    V = __fadd_rn(cv, I);
                    spk = L.ref[q] != 0;
                } else {
                    uint32_t r = L.ref[q];
                    if (r > 0) {
                        r -= 1;
                        V = v_reset;
                    } else {
                        const float av = __fsub_rn(v_rest, V);
                        const float bv = __fmul_rn(mk, av);
                        const float cv = __fadd_rn(V, bv);
                        V = __fadd_rn(cv, I);
                        if (V >= v_th) {
                            spk = true;
                            V = v_reset;
                            r = ref_steps;
                        }
                    }
                    L.ref[q] = (uint8_t)r;
                }
                L.V[q] = V;
                if (spk) ev += a.outdeg[tile_lo + q];
            }
            bal[u] = __ballot(spk);
            nw_spk += (uint32_t)__popcll(bal[u]);
        }
    }
    // compaction: one LDS counter update per wave, then every round's firing
    // lanes stored at consecutive positions of the tile's segment of the
    // spike list (tslot: the spike-list slot of t)
    const uint64_t seg = (uint64_t)tslot * a.tl.T + tile;
    uint32_t *dst = a.spk_ids + seg * a.tl.W;
    if (nw_spk) {
        uint32_t wb = 0;
        if (lane == 0) wb = atomicAdd(cnt, nw_spk);
        wb = (uint32_t)__builtin_amdgcn_readlane((int)wb, 0);  // (lane 0 took the positions)
#pragma unroll
        for (int u = 0; u < kRunRounds; u++) {
            const uint64_t mask = bal[u];
            if ((mask >> lane) & 1ull) {
                const uint32_t rank = __builtin_amdgcn_mbcnt_hi(
                    (uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
                st_ag(dst + wb + rank, tile_lo + u * kRunThreads + tid);
            }
            wb += (uint32_t)__popcll(mask);
        }
    }
    if (DIRECT) ev = block_sum_u64(ev, L.ws64);
    else lds_sync();
    const uint32_t ns = *cnt;
    // the other counter, last read before the barrier that began this step,
    // restarts at zero for the next step
    if (tid == 0) *cnt_next = 0;
    if (tid == 0) {
        st_ag(&a.spk_cnt[seg], ns);
        if (late) {  // (step_stats, after the publication)
            L.st_ns = ns;
            L.st_ev = ev;
            L.st_dlv = delivered;
        } else {
            step_stats(a, x, t, ns, ev, delivered);
        }
    }
}

// Tile phase of a batch of Db >= 2 steps of LIF neurons (binned delivery):
// the inputs of every step of the batch are in the accumulators already
// (acc[u * W ...], the smallest delay is at least Db), so each thread takes
// its neurons through the Db steps in registers, with the arithmetic of
// run_update, and compacts each step's spikes straight into that step's
// segment of the spike list (one counter nb[u] per step: no barrier between
// steps).  Then one barrier, and every step's count is published.
template <bool FIXED, bool CMP>
__device__ void run_update_batch(const RunArgs &ra, RunLDS<FIXED, CMP> &L, uint32_t x, uint32_t tile,
                                 uint32_t tile_lo, uint32_t tile_n, uint64_t t_first, uint32_t ss, uint32_t Db)
{
    using AccT = typename RunLDS<FIXED, CMP>::AccT;
    const StepArgs &a = ra.s;
    const uint32_t tid = tid_here(), lane = tid & (kWave - 1), W = a.tl.W;
    const float mk = L.mk, v_rest = L.v_rest, v_th = L.v_th, v_reset = L.v_reset, i_bias = L.i_bias,
                ext_w = L.ext_w;
    const int32_t ext_wq = L.ext_wq, bias_q = L.bias_q, shift = L.shift, shift64 = L.shift64;
    const uint32_t ref_steps = L.ref_steps, pois_len = L.pois_len;
    for (uint32_t q0 = 0; q0 < tile_n; q0 += kRunThreads) {  // (uniform trip count: ballots below)
        const uint32_t q = q0 + tid;
        const bool live = q < tile_n;
        const uint32_t qc = live ? q : 0u;
        float V = L.V[qc];
        uint32_t r = L.ref[qc];
        AccT acc_n = L.u.t.acc[qc];  // step u + 1's input, loaded one step ahead
        uint32_t K_n = L.kp[qc];  // (read unconditionally: a select below, not a branch)
        for (uint32_t u = 0; u < Db; u++) {
            const AccT acc = acc_n;
            const uint32_t K = pois_len ? K_n : 0u;
            if (u + 1 < Db) {
                acc_n = L.u.t.acc[(u + 1) * W + qc];
                K_n = L.kp[(u + 1) * W + qc];
            }
            float I;
            if (FIXED) {
                const int32_t qt = (int32_t)acc + (int32_t)K * ext_wq + bias_q;
                I = ldexpf((float)qt, -shift);
            } else {
                const float isyn = fixed64_to_float(acc, shift64);
                const float ext = __fmul_rn((float)K, ext_w);
                I = __fadd_rn(__fadd_rn(isyn, ext), i_bias);
            }
            bool spk = lif_step(V, r, I, mk, v_rest, v_th, v_reset, ref_steps);
            spk = spk && live;
            const uint64_t bal = __ballot(spk);
            if (bal) {  // (uniform) one counter update per wave and step
                uint32_t wb = 0;
                if (lane == 0) wb = atomicAdd(&L.u.t.nb[u], (uint32_t)__popcll(bal));
                wb = (uint32_t)__builtin_amdgcn_readlane((int)wb, 0);  // (lane 0 took the positions)
                if (spk) {  // straight to step u's segment of the spike list
                    const uint32_t rank =
                        __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
                    const uint32_t su = ss + u < a.spk_slots ? ss + u : ss + u - a.spk_slots;
                    st_ag(a.spk_ids + ((uint64_t)su * a.tl.T + tile) * W + wb + rank, tile_lo + q);
                }
            }
        }
        if (live) {
            L.V[q] = V;
            L.ref[q] = (uint8_t)r;
        }
    }
    lds_sync();
    const uint64_t T = a.tl.T;
    if (tid < Db) {
        const uint64_t t = t_first + tid;
        const uint32_t ns = L.u.t.nb[tid];
        st_ag(&a.spk_cnt[(uint64_t)(ss + tid < a.spk_slots ? ss + tid : ss + tid - a.spk_slots) * T + tile], ns);
        if (ns) atomicAdd(&a.counts8[t * kGroups + x], ns);
        const unsigned long long delivered = L.u.t.dlv[tid];
        if (delivered) atomicAdd((unsigned long long *)&a.delivered8[t * kGroups + x], delivered);
    }
}

// Spike counts of the Db steps t_first .. t_first + Db - 1 as one list in
// (step, tile) order: pre[u * T + tile] = spikes before segment (u, tile),
// pre[Db * T] = all of them; uslot[u] = the spike-list slot of step u.  A
// one-step batch finds each polling wave's part in place already
// (poller_prefix) and adds the sums of the waves before.
template <bool FIXED, bool CMP>
__device__ uint32_t load_spike_batch(const StepArgs &a, RunLDS<FIXED, CMP> &L, uint32_t slot0, uint32_t Db)
{
    const uint32_t T = a.tl.T, W = a.tl.W, NS = Db * T;
    if (Db == 1) {
        // the polling waves left each wave's exclusive prefix in pre[] and
        // its sum in ptot[] (T <= 256: one tile per thread)
        uint32_t before = 0, tot = 0;
#pragma unroll
        for (uint32_t k = 0; k < kRunMaxT / kWave; k++) {
            const uint32_t v = k * kWave < T ? L.ptot[k] : 0u;
            before += k < threadIdx.x / kWave ? v : 0u;
            tot += v;
        }
        if (threadIdx.x < T) L.u.p.pre[threadIdx.x] += before;
        if (threadIdx.x == 0) {
            L.u.p.pre[T] = tot;
            L.u.p.uslot[0] = slot0;
        }
        lds_sync();
        return tot;
    }
    constexpr uint32_t kPerMax = kRunMaxT * kRunMaxD / kRunThreads;  // segments per thread, at most
    const uint32_t per = (NS + kRunThreads - 1) / kRunThreads;
    const uint32_t b0 = threadIdx.x * per;
    // (slot0: the spike-list slot of the first step; Db <= spk_slots / 2: one wrap at most)
    uint32_t c[kPerMax], sum = 0;
#pragma unroll
    for (uint32_t k = 0; k < kPerMax; k++) {  // unconditional loads from clamped indices
        const uint32_t seg = b0 + k < NS && k < per ? b0 + k : 0u;
        const uint32_t u = seg / T, tile = seg - u * T;
        const uint32_t slot = slot0 + u < a.spk_slots ? slot0 + u : slot0 + u - a.spk_slots;
        const uint32_t v = ld_u32<true>(a.spk_cnt + (uint64_t)slot * T + tile);
        c[k] = b0 + k < NS && k < per ? (v < W ? v : W) : 0u;
        sum += c[k];
    }
    if (threadIdx.x < Db) {
        const uint32_t u = threadIdx.x;
        L.u.p.uslot[u] = slot0 + u < a.spk_slots ? slot0 + u : slot0 + u - a.spk_slots;
    }
    uint32_t tot;
    uint32_t ex = block_scan_u32(sum, L.ws, &tot);
#pragma unroll
    for (uint32_t k = 0; k < kPerMax; k++)
        if (k < per && b0 + k < NS) {
            L.u.p.pre[b0 + k] = ex;
            ex += c[k];
        }
    if (threadIdx.x == 0) L.u.p.pre[NS] = tot;
    lds_sync();
    return tot;
}

// k-th spike of the batch (k < total): its neuron, and in *u the step of the
// batch it belongs to.
template <bool FIXED, bool CMP>
__device__ __forceinline__ uint32_t spike_at_batch(const StepArgs &a, const RunLDS<FIXED, CMP> &L, uint32_t NS,
                                                   uint32_t k, uint32_t *u)
{
    const uint32_t *pre = L.u.p.pre;
    uint32_t lo = 0, hi = NS - 1;
    while (lo < hi) {
        const uint32_t mid = (lo + hi + 1) >> 1;
        if (pre[mid] <= k) lo = mid; else hi = mid - 1;
    }
    const uint32_t T = a.tl.T, uu = NS == T ? 0u : lo / T, tile = lo - uu * T;
    *u = uu;
    return ld_u32<true>(a.spk_ids + ((uint64_t)L.u.p.uslot[uu] * T + tile) * a.tl.W + (k - pre[lo]));
}

// Push phase (binned delivery): push block (x, r) takes the r-th equal share
// of the spikes of the Db steps t_first .. t_first + Db - 1 (Db = 1 unless
// the smallest delay allows batches: every event of these spikes arrives
// after the batch), reads the runs of their rows that target group x and
// appends the events to its own pages: bucket b = a_off * T8 + c with the
// arrival offset a_off = (step of the batch) + (delay index j) and c the tile
// of the group; page (arrival slot (t_first + dmin + a_off) mod pslots, c).
// Also appends its share of the spike IDs to the raster (group 0).  Returns
// the batch's spike count (every push block sees the whole list) and, for
// batches of several steps, leaves each step's count in L.mstep.
template <bool FIXED, bool CMP>
__device__ uint32_t run_push(const RunArgs &ra, RunLDS<FIXED, CMP> &L, uint32_t x, uint32_t r, uint64_t t_first,
                             uint32_t ps, uint32_t ss, uint32_t Db, uint64_t rbase)
{
    using Rec = typename SynRec<CMP>::T;
    using LT = RunLDS<FIXED, CMP>;
    constexpr int R = LT::R;
    const StepArgs &a = ra.s;
    const uint32_t tid = tid_here(), lane = tid & (kWave - 1), w = __builtin_amdgcn_readfirstlane(tid / kWave);
    constexpr uint32_t nw = kRunThreads / kWave;
    const Tiling tl = a.tl;
    const uint32_t NB = (Db + a.lists - 1) * tl.T8, G1 = ra.R, NS = Db * tl.T;
    // the pages of the batch's arrival slots were drained in the batch: they
    // restart empty (ps, ss: the arrival and spike-list slots of t_first)
    for (uint32_t q = tid; q < Db * tl.T8; q += kRunThreads) {
        const uint32_t u = div_t8(tl, q), c = q - u * tl.T8;
        L.fill[(ps + u < a.pslots ? ps + u : ps + u - a.pslots) * tl.T8 + c] = 0;
    }
    for (uint32_t b = tid; b < NB; b += kRunThreads) L.u.p.bcnt[b] = 0;
    if (tid < Db) L.u.p.emit[tid] = 0;
    const uint32_t M = load_spike_batch(a, L, ss, Db);  // (its barriers publish the resets)
    if (Db > 1) {
        if (tid == 0) {  // each step's count, and where its spikes go in the raster (if they fit)
            uint64_t rb = rbase;
            uint32_t okm = 0;
            for (uint32_t u = 0; u < Db; u++) {
                const uint32_t Mu = L.u.p.pre[(u + 1) * tl.T] - L.u.p.pre[u * tl.T];
                const bool ok = a.raster_cap && rb + Mu <= a.raster_cap;
                L.u.p.rbu[u] = rb - L.u.p.pre[u * tl.T];  // (mod 2^64)
                okm |= (uint32_t)ok << u;
                rb = ok ? rb + Mu : rb;
                L.mstep[u] = Mu;
            }
            L.u.p.rokm = okm;
        }
        lds_sync();
    }
    // one step: its spikes go to the raster from rbase on, if they fit
    const bool one_fits = a.raster_cap && rbase + M <= a.raster_cap;
    uint32_t k0, k1;
    equal_share(M, r, G1, &k0, &k1);
    const bool rec_raster = a.raster_cap && x == 0;
    const uint32_t xlo = x * tl.Gw;
    const uint64_t cap = a.page_cap;
    const uint32_t dm = a.dmin % a.pslots;  // (ps + dm < 2 pslots)
    const uint32_t slot_of_a0 = ps + dm < a.pslots ? ps + dm : ps + dm - a.pslots;
    for (uint32_t c0 = k0; c0 < k1; c0 += kRunChunk) {
        const uint32_t K = k1 - c0 < kRunChunk ? k1 - c0 : kRunChunk;
        uint32_t len = 0, uo = 0;
        uint64_t base = 0;
        if (tid < K) {
            const uint32_t k = c0 + tid;
            const uint32_t s = spike_at_batch(a, L, NS, k, &uo);
            if (rec_raster && (Db == 1 ? one_fits : ((L.u.p.rokm >> uo) & 1u) != 0))
                a.raster[(Db == 1 ? rbase : L.u.p.rbu[uo]) + k] = s;
            const RowDesc *d = a.desc + s;
            const uint32_t lo = x ? d->gend[x - 1] : 0u, hi = d->gend[x];
            len = hi - lo;
            base = d->start + lo;
            if (x == 0) atomicAdd(&L.u.p.emit[uo], (unsigned long long)d->gend[kGroups - 1]);
        }
        uint32_t C;
        const uint32_t nch = (len + kWave - 1) / kWave;
        const uint32_t coff = block_scan_u32(nch, L.ws, &C);  // this thread's row: chunks [coff, coff + nch)
        constexpr uint32_t kWin = R * nw;
        for (uint32_t i0 = 0; i0 < C; i0 += kWin) {
            for (uint32_t q = tid; q < kWin; q += kRunThreads) L.u.p.clen[q] = 0;
            lds_sync();
            if (tid < K) {
                const uint32_t cb = coff > i0 ? coff : i0, ce = coff + nch < i0 + kWin ? coff + nch : i0 + kWin;
                for (uint32_t q = cb; q < ce; q++) {
                    const uint32_t o = (q - coff) * kWave;
                    L.u.p.cbase[q - i0] = base + o;
                    L.u.p.clen[q - i0] = (len - o < kWave ? len - o : kWave) | (uo << 8);
                }
            }
            lds_sync();
            Rec rec[R];
            uint32_t okm = 0;
            uint64_t uom = 0;  // step of the batch of each chunk, 4 bits each
#pragma unroll
            for (int u = 0; u < R; u++) {
                const uint32_t cl = u * nw + w;
                const uint32_t lw = L.u.p.clen[cl];
                const uint32_t len = lw & 0xffu;
                const uint64_t cb = L.u.p.cbase[cl];
                const bool ok = lane < len;
                const uint64_t idx = ok ? cb + lane : 0ull;
                okm |= (uint32_t)ok << u;
                uom |= (uint64_t)(lw >> 8) << (4 * u);
                rec[u] = SynRec<CMP>::load(a, idx);  // unconditional load from a clamped index
            }
            // rank every event of the window within its bucket (LDS counters);
            // no rank is used before the loop ends, so that the atomics are in
            // flight together rather than one LDS round trip each.  The
            // record becomes (bucket << 16) | page entry.
            uint32_t rk[R];
#pragma unroll
            for (int q = 0; q < R; q++) {
                rk[q] = 0;
                if (!((okm >> q) & 1u)) continue;
                const uint32_t key = rec_key(rec[q]);
                const uint32_t ao = rec_delay(key) + (uint32_t)((uom >> (4 * q)) & 0xfu);
                const uint32_t local = rec_target(key) - xlo;
                const uint32_t b = __umul24(ao, tl.T8) + (local >> tl.logW);  // (ao, T8 < 2^24)
                rk[q] = atomicAdd(&L.u.p.bcnt[b], 1u);
                const uint32_t sv = (b << 16) | (local & (tl.W - 1));
                if constexpr (CMP) rec[q] = sv | (rec_class(key) << kPageClassShift);
                else rec[q].x = (int)sv;
            }
            lds_sync();
            // bucket starts in the stage; the page position of staged event q
            // of bucket b is wb[b] + q (mod 2^32); the fill counters advance
            uint32_t staged;
            {
                const uint32_t P = (NB + kRunThreads - 1) / kRunThreads;
                const uint32_t b0 = tid * P;
                uint32_t sum = 0;
                for (uint32_t k = 0; k < P; k++)
                    if (b0 + k < NB) sum += L.u.p.bcnt[b0 + k];
                uint32_t ex = block_scan_u32_open(sum, L.ws2, &staged);
                for (uint32_t k = 0; k < P; k++) {
                    if (b0 + k < NB) {
                        const uint32_t bb = b0 + k, cnt = L.u.p.bcnt[bb];
                        const uint32_t ao = div_t8(tl, bb), cc = bb - ao * tl.T8;
                        uint32_t sl = slot_of_a0 + ao;
                        sl = sl >= a.pslots ? sl - a.pslots : sl;
                        uint32_t &f = L.fill[sl * tl.T8 + cc];
                        L.u.p.bst[bb] = ex;
                        L.u.p.wb[bb] = f - ex;
                        L.u.p.pb[bb] = page_of(a, x, r, sl, cc) * a.page_cap;
                        f += cnt;
                        L.u.p.bcnt[bb] = 0;
                        ex += cnt;
                    }
                }
            }
            lds_sync();
            Rec *stage = L.u.p.stage;
#pragma unroll
            for (int q = 0; q < R; q++)
                if ((okm >> q) & 1u) stage[L.u.p.bst[rec_key(rec[q]) >> 16] + rk[q]] = rec[q];
            lds_sync();
            // coalesced appends: consecutive staged events of a bucket go to
            // consecutive page positions
            for (uint32_t q = tid; q < staged; q += kRunThreads) {
                const Rec r2 = stage[q];
                const uint32_t key = rec_key(r2);
                const uint32_t b = key >> 16, low = key & 0xffffu;
                const uint32_t pos = L.u.p.wb[b] + q;
                if (pos < cap) {
                    const uint32_t e = L.u.p.pb[b] + pos;
                    if constexpr (CMP) a.pages16[e] = (uint16_t)low;
                    else a.pages[e] = make_int2((int)low, r2.y);
                } else {
                    const uint32_t ao = div_t8(tl, b), cc = b - ao * tl.T8;
                    uint32_t sl = slot_of_a0 + ao;
                    sl = sl >= a.pslots ? sl - a.pslots : sl;
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
            lds_sync();  // the stage and wb are rewritten by the next window
        }
        lds_sync();  // the chunk tables are rewritten by the next chunk
    }
    lds_sync();
    // publish the fill counters of all pages of this block
    const uint32_t NF = a.pslots * tl.T8;
    for (uint32_t f = tid; f < NF; f += kRunThreads) {
        const uint32_t sl = div_t8(tl, f);
        a.pfill[page_of(a, x, r, sl, f - sl * tl.T8)] = L.fill[f];
    }
    // events emitted at each step of the batch, counted once per spike (group 0)
    if (x == 0 && tid < Db && L.u.p.emit[tid])
        atomicAdd((unsigned long long *)&a.events8[(t_first + tid) * kGroups], L.u.p.emit[tid]);
    return M;
}

// Direct delivery (one delay): the tile reads, for every spike of t - dmin,
// the run of its row that falls into the tile.
template <bool FIXED, bool CMP>
__device__ uint64_t run_gather(const StepArgs &a, RunLDS<FIXED, CMP> &L, uint32_t tile, uint32_t tile_lo,
                               uint64_t t, uint32_t tslot)
{
    uint64_t mine = 0;
    if (t >= a.dmin) {
        // the spike-list slot of t - dmin (tslot: that of t; dmin < spk_slots)
        const uint32_t dslot = tslot >= a.dmin ? tslot - a.dmin : tslot + a.spk_slots - a.dmin;
        const uint32_t P = load_spike_set<true>(a, dslot, L.u.t.pre, L.ws);
        mine = gather_direct<FIXED, CMP, true>(a, L.u.t.acc, L.u.t.pre, L.u.t.wpre, L.u.t.wbeg, tile, tile_lo, P,
                                               dslot, -1, L.wtab);
    }
    const uint64_t tot = block_sum_u64(mine, L.ws64);
    return tot;
}

// Raster bookkeeping shared by both deliveries: offsets of step t + 1 and the
// capacity flag, by one workgroup; every workgroup advances its own copy of
// the running base.
__device__ __forceinline__ uint64_t raster_advance(const StepArgs &a, uint64_t t, uint64_t rbase, uint32_t M,
                                                   bool writer)
{
    const bool ok = rbase + M <= a.raster_cap;
    if (writer && threadIdx.x == 0) {
        a.raster_offs[t + 1] = ok ? rbase + M : rbase;
        if (!ok) atomicOr(a.flags, 2u);
    }
    return ok ? rbase + M : rbase;
}

// BATCH: binned delivery of LIF neurons in batches of several steps, whose
// updates run in registers (run_update_batch); a variant of its own, so that
// the one-step kernels keep their register allocation.
template <bool FIXED, bool CMP, bool DIRECT, bool BATCH>
__global__ __launch_bounds__(kRunThreads) void k_run(RunArgs ra)
{
    __shared__ RunLDS<FIXED, CMP> L;
    const StepArgs &a = ra.s;
    RunCtl *ctl = ra.ctl;
    const uint32_t tid = threadIdx.x;

    // placement: the XCD this workgroup runs on, and a ticket within it
    if (tid == 0) {
        const ModelArgs &mm = ra.s.m;
        L.mk = mm.k;
        L.v_rest = mm.v_rest;
        L.v_th = mm.v_th;
        L.v_reset = mm.v_reset;
        L.i_bias = mm.i_bias;
        L.ext_w = mm.ext_w;
        L.ext_wq = mm.ext_wq;
        L.bias_q = mm.bias_q;
        L.shift = mm.shift;
        L.shift64 = mm.shift64;
        L.ref_steps = mm.ref_steps;
        L.pois_len = mm.pois_len;
        for (uint32_t k = 0; k < kMaxClasses; k++) L.wtab[k] = a.wval[k];
        const uint32_t raw = xcc_id();
        const uint32_t x = raw & (kGroups - 1);
        if (raw >= kGroups) atomicOr(&ctl->abort_flag, kRunAbortPlacement);
        L.x = x;
        L.r = atomicAdd(&ctl->ticket[x * kCtlStride], 1u);
        L.nspk2[0] = 0;
        L.nspk2[2] = 0;
        atomicAdd(&ctl->start, 1u);
        L.stop = spin_ge(&ctl->start, gridDim.x, &ctl->abort_flag) ? 0u : 1u;
        if (L.stop) atomicOr(a.flags, kRunStoppedFlag);
    }
    __syncthreads();
    if (L.stop) return;
    if (tid < kGroups && ld_ag(&ctl->ticket[tid * kCtlStride]) != ra.R) atomicOr(&L.stop, 1u);
    if (tid == 0 && ld_ag(&ctl->abort_flag)) atomicOr(&L.stop, 1u);
    __syncthreads();
    if (L.stop) {  // every workgroup reads the same tickets: all leave here together
        if (tid == 0) {
            atomicOr(&ctl->abort_flag, kRunAbortPlacement);
            atomicOr(a.flags, kRunStoppedFlag);
        }
        return;
    }
    const uint32_t x = __builtin_amdgcn_readfirstlane(L.x), r = __builtin_amdgcn_readfirstlane(L.r);
    const Tiling tl = a.tl;
    const bool has_tile = r < tl.T8;
    const uint32_t tile = x * tl.T8 + r;
    const uint32_t tile_lo = tile * tl.W;
    const uint32_t tile_n = has_tile && tile_lo < a.n ? (a.n - tile_lo < tl.W ? a.n - tile_lo : tl.W) : 0u;
    const ModelArgs &m = a.m;

    // persistent LDS state
    for (uint32_t q = tid; q < tile_n; q += kRunThreads) {
        L.V[q] = a.V[tile_lo + q];
        L.ref[q] = a.ref[tile_lo + q];
    }
    if (m.pois_len)
        for (uint32_t q = tid; q < 256; q += kRunThreads) {
            L.pois[q] = a.pois[q < m.pois_len ? q : 0u];
            L.guide[q] = a.pois_guide[q];
        }
    if (!DIRECT) {
        const uint32_t NF = a.pslots * tl.T8;
        for (uint32_t f = tid; f < NF; f += kRunThreads) {
            const uint32_t sl = div_t8(tl, f);
            L.fill[f] = a.pfill[page_of(a, x, r, sl, f - sl * tl.T8)];
        }
    }
    __syncthreads();
    // LIF neurons: the draws of a whole batch at once (source neurons: of one step)
    const bool lif = m.kind != SPK_SOURCE;
    const uint32_t Dd = DIRECT || !lif ? 1u : ra.D;
    if (ra.n_steps) run_draws(a, L, tile_lo, tile_n, ra.t0, (uint32_t)(ra.n_steps < Dd ? ra.n_steps : Dd));
    uint64_t rbase = a.raster_cap ? a.raster_offs[ra.t0] : 0;
    uint32_t eg = 0, ex = 0;
    // binned: draws of the next batch left for after its push phase (units
    // dr_k .. dr_n - 1 of steps from dr_t on)
    uint64_t dr_t = 0;
    uint32_t dr_k = 0, dr_n = 0, look = 0;
    __syncthreads();

    // Steps run in batches of D (binned delivery with a smallest delay >= D;
    // D = 1 otherwise): the tile phases of the batch back to back, then one
    // push phase for all of the batch's spikes.  Every event that arrives
    // within a batch comes from a spike before it, so it has been filed.
    const uint32_t D = DIRECT ? 1u : ra.D;
    uint64_t s = 0;
    // the arrival slot and the spike-list slot of t_first, advanced by Db per
    // batch (Db <= pslots, spk_slots: one wrap at most) instead of a 64-bit
    // remainder per use
    uint32_t ps = (uint32_t)(ra.t0 % a.pslots), ss = (uint32_t)(ra.t0 % a.spk_slots);
    while (s < ra.n_steps) {
        const uint32_t Db = (uint32_t)(ra.n_steps - s < D ? ra.n_steps - s : D);
        const uint64_t t_first = ra.t0 + s;
        s += Db;
        const bool more = s < ra.n_steps;
        // binned: the last step's statistics wait in LDS until the tile has
        // published (step_stats); direct delivery adds them at once (measured:
        // deferred past the grid barrier, 1e6 sources at 10 Hz took 76.2
        // instead of 74.8 us per step)
        bool late = false;
        if (has_tile) {
            // binned: the draws not made before the last push phase
            for (; dr_k < dr_n; dr_k++) run_draw_unit(a, L, tile_lo, tile_n, dr_t, dr_k);
            // the push phase reused this LDS: accumulators restart at zero, and
            // the spike count of the previous step has been read by every
            // thread (binned: while the other push blocks finish; the barrier
            // of the wait orders these stores before the drain)
            for (uint32_t q = tid; q < Db * tl.W; q += kRunThreads) L.u.t.acc[q] = 0;
            if (tid == 0) L.nspk2[0] = 0;
            if constexpr (BATCH)
                if (tid < Db) L.u.t.nb[tid] = 0;
            // binned: every push block of the XCD has filed the previous batch
            if (!DIRECT && !wait_pushes(ra, L, x, ex)) return;
            if (!DIRECT) {  // all steps of the batch
                if (!BATCH && Db == 1) run_drain<FIXED, CMP, true>(a, L, x, r, tile, tile_n, ps, 1);
                else run_drain<FIXED, CMP, false>(a, L, x, r, tile, tile_n, ps, Db);
            }
            bool batched = false;
            if constexpr (BATCH) {
                batched = lif && Db > 1;
                if (batched) run_update_batch(ra, L, x, tile, tile_lo, tile_n, t_first, ss, Db);
            }
            late = !DIRECT && !batched;
            if (!batched) for (uint32_t u = 0; u < Db; u++) {
                const uint64_t t = t_first + u;
                if (u) {  // the spike list of t - 1 (LDS) has been published by every thread
                    if (!lif) run_draws(a, L, tile_lo, tile_n, t, 1);
                    __syncthreads();
                }
                const uint32_t tslot = ss + u < a.spk_slots ? ss + u : ss + u - a.spk_slots;
                const uint64_t delivered = DIRECT ? run_gather(a, L, tile, tile_lo, t, tslot) : L.u.t.dlv[u];
                run_update<FIXED, CMP, DIRECT>(ra, L, x, tile, tile_lo, tile_n, t, tslot, delivered, u * tl.W,
                                               lif ? u * tl.W : 0u, &L.nspk2[u & 1u], &L.nspk2[(u + 1u) & 1u],
                                               late && u + 1 == Db);
            }
        }
        const uint32_t Dn = (uint32_t)(ra.n_steps - s < Dd ? ra.n_steps - s : Dd);  // (0 after the last batch)
        if (DIRECT) {
            if (!grid_sync(ra, L, x, ++eg, has_tile && more, tile_lo, tile_n, t_first + Db, Dn)) return;
        } else {  // binned: the tiles' progress words instead of a grid barrier
            ++eg;
            if (has_tile) publish_tile(ra, tile, eg, &L.nspk2[Db == 1 ? 0u : 2u]);
            if (late && tid == 0) step_stats(a, x, t_first + Db - 1, L.st_ns, L.st_ev, L.st_dlv);
            // the next batch's draws while the others finish: a unit at a
            // time between looks at the tiles' words; once every tile has
            // published, the rest waits until after the push phase (the last
            // tiles to finish would otherwise hold every push phase up by
            // their draws)
            {
                bool ready = false;
                dr_t = t_first + Db;
                dr_k = 0;
                dr_n = has_tile && more ? Dn * draw_units_per_step(tile_n) : 0u;
                // a polling lane's word as last seen: none yet (a stamp other than eg's)
                uint32_t pv = ((eg ^ 1u) & (0xffffffffu >> kTileCntBits)) << kTileCntBits;
                while (!ready && dr_k < dr_n)
                    ready = look_tiles(ra, L, eg, Db == 1, look++ & 1u, pv,
                                       [&] { run_draw_unit(a, L, tile_lo, tile_n, dr_t, dr_k++); });
                if (!ready && !wait_tiles(ra, L, eg, Db == 1, pv)) return;
            }
        }
        if (DIRECT) {
            const uint64_t t = t_first;
            if (a.raster_cap) {  // the spike list of t is complete: workgroup (0, 0) records it
                const bool writer = x == 0 && r == 0;
                const uint32_t M = load_spike_set<true>(a, (uint32_t)(t % a.spk_slots), L.u.p.pre, L.ws);
                if (writer && rbase + M <= a.raster_cap)
                    for (uint32_t k = tid; k < M; k += kRunThreads)
                        a.raster[rbase + k] = spike_at<true>(a, L.u.p.pre, (uint32_t)(t % a.spk_slots), k);
                rbase = raster_advance(a, t, rbase, M, writer);
                __syncthreads();  // pre[] is the tile's scratch again
            }
        } else {
            const uint32_t M = run_push(ra, L, x, r, t_first, ps, ss, Db, rbase);
            if (a.raster_cap)
                for (uint32_t u = 0; u < Db; u++)
                    rbase = raster_advance(a, t_first + u, rbase, Db == 1 ? M : L.mstep[u], x == 0 && r == 0);
            publish_push(ra, x, r, ++ex);  // the tiles of the XCD wait for it (wait_pushes)
        }
        ps = ps + Db < a.pslots ? ps + Db : ps + Db - a.pslots;
        ss = ss + Db < a.spk_slots ? ss + Db : ss + Db - a.spk_slots;
    }

    for (uint32_t q = tid; q < tile_n; q += kRunThreads) {
        a.V[tile_lo + q] = L.V[q];
        if (m.kind != SPK_SOURCE) a.ref[tile_lo + q] = L.ref[q];
    }
    if (tid == 0 && x == 0 && r == 0) *(uint64_t *)a.t_base = ra.t0 + ra.n_steps;
}

template <bool FIXED, bool CMP, bool DIRECT, bool BATCH>
hipError_t launch_run_t(const RunArgs &ra, hipStream_t s)
{
    RunArgs arg = ra;
    void *args[] = {&arg};
    return hipLaunchCooperativeKernel((const void *)k_run<FIXED, CMP, DIRECT, BATCH>, dim3(kGroups * ra.R),
                                      dim3(kRunThreads), args, 0, s);
}

template <bool FIXED, bool CMP>
hipError_t launch_run_fc(const RunArgs &ra, hipStream_t s)
{
#if SPK_RUN_BATCH
    return launch_run_t<FIXED, CMP, false, true>(ra, s);
#else
    if (ra.s.direct) return launch_run_t<FIXED, CMP, true, false>(ra, s);
    return launch_run_t<FIXED, CMP, false, false>(ra, s);
#endif
}

hipError_t launch_run_any(const RunArgs &ra, hipStream_t s)
{
    const bool F = ra.s.m.fixed, C = ra.s.compact;
    if (F && C) return launch_run_fc<true, true>(ra, s);
    if (F && !C) return launch_run_fc<true, false>(ra, s);
    if (!F && C) return launch_run_fc<false, true>(ra, s);
    return launch_run_fc<false, false>(ra, s);
}

}  // namespace

#if SPK_RUN_BATCH
// Binned delivery, LIF neurons, batches of ra.D >= 2 steps.
hipError_t launch_run_batched(const RunArgs &ra, hipStream_t s) { return launch_run_any(ra, s); }
#else

bool run_supported(const StepArgs &a, uint32_t R)
{
    const Tiling &tl = a.tl;
    if (R == 0 || R > kRunMaxR || tl.T8 > R || tl.T != kGroups * tl.T8 || tl.W > kMaxTileW) return false;
    if (a.m.pois_len > 256 || a.proc) return false;
    if (a.direct) return a.lists == 1 && a.spk_slots > a.dmin;
    return a.pg1 == R && a.pslots * tl.T8 <= kRunMaxFill && a.lists * tl.T8 <= kRunMaxBuckets && a.spk_slots >= 2 &&
           a.page_cap % 16 == 0 && tl.W <= 65536;
}

bool run_batch_supported(const StepArgs &a, uint32_t D)
{
    if (a.direct) return D == 1;
    return D >= 1 && D <= kRunMaxD && D <= a.dmin && a.spk_slots >= 2 * D && a.tl.T <= kRunMaxT &&
           (D + a.lists - 1) * a.tl.T8 <= kRunMaxBuckets && D + a.lists - 1 <= a.pslots &&
           D * a.tl.W <= kMaxTileW && D * a.pg1 <= kRunThreads;
}

hipError_t launch_run(const RunArgs &ra, hipStream_t s)
{
    if (!run_supported(ra.s, ra.R) || !run_batch_supported(ra.s, ra.D)) return hipErrorInvalidValue;
    const StepArgs &a = ra.s;
    if (a.compact ? !a.syn32 || (!a.direct && !a.pages16) : !a.syn || (!a.direct && !a.pages))
        return hipErrorInvalidValue;
    if (!a.direct && ra.D > 1 && a.m.kind != SPK_SOURCE) return launch_run_batched(ra, s);
    return launch_run_any(ra, s);
}
#endif

}  // namespace spk
