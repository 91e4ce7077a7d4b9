// spk_step.hip -- the simulation step on gfx950 (MI355X): spike transmission
// (paper Sec. III-C) fused with the neuron update that produces the spikes.
//
// Why this shape (measured on MI355X): scattered global atomics reach only
// ~21 G/s device-wide whatever the footprint, while LDS integer atomics reach
// ~4 T/s (u32) and ~2.7 T/s (u64); LDS fp32 atomics are ~20x slower than u32.
// So every synaptic event is accumulated in LDS, as an integer:
//   - fixed mode: int32 in units of 2^-S (weights quantised, Sec. "fixed point"
//     of the public header);
//   - fp32 mode: int64 in units of 2^-S64, where S64 is chosen at creation so
//     that every fp32 weight is an exact multiple and no sum can overflow;
//     the sum is therefore exact and is rounded once to fp32.
// The target neurons are cut into tiles of W neurons, one workgroup per tile
// ("tile" kernel); each XCD owns a contiguous group of T8 tiles (blockIdx % 8
// selects the XCD).  A step t is:
//   1. tile kernel: accumulate the events arriving at t in LDS, update the
//      tile's neurons, compact the spikes of t into the tile's own segment of
//      the spike list (no global atomics);
//   2. push kernel (binned delivery): read the row of every neuron that fired
//      at t once, and sort its events by (arrival step t + d, target tile) in
//      LDS into pages owned by the block (no global atomics); the tile kernel
//      of step t + d drains them.
// With a single delay and long rows the tile kernel instead reads, for every
// spike due at t, the run of that spike's row that falls into its tile
// ("direct" delivery, per-row tile offsets).  Rows are grouped by target tile
// (Sec. III-A keeps them sorted by target), so both runs are contiguous: the
// paper's cache-aware transmission, with the locality made explicit as LDS
// tiles instead of left to the cache.
//
// Delays (Sec. V): each stored synapse carries its delay index; an event of
// delay d from a spike at t lands in the page of arrival slot (t + d) mod dmax.
#include <hip/hip_runtime.h>

#include "spk_dev.h"

namespace spk {

namespace {

constexpr int kPushThreads = 1024;
constexpr int kTileThreads = 1024;
static_assert(kPushThreads == (int)kBlockThreads && kTileThreads == (int)kBlockThreads,
              "the block-wide helpers assume workgroups of kBlockThreads");
constexpr int kPushR = 16;                                // events per thread per load phase
constexpr uint32_t kLoadPhase = kPushR * kPushThreads;    // events loaded at once
constexpr uint32_t kStage = kLoadPhase / 2;               // events bucket-sorted at once
constexpr uint32_t kMaxChunkSpikes = 1024;                // rows resolved per push chunk
constexpr int kRounds = kMaxTileW / kTileThreads;         // neurons per tile thread
static_assert(kMaxTiles <= 2 * kTileThreads, "spike-count prefix takes at most two tiles per thread");

// ------------------------------------------------------------ push kernel

struct PushLDS {
    int2 stage[kStage];              // bucket-sorted events {bucket << 16 | local, weight}; compact
                                     // format: u32 bucket << 16 | class << 13 | local
    uint32_t pre[kMaxTiles + 1];     // prefix of the source tiles' spike counts
    uint32_t cpre[kMaxChunkSpikes + 1];  // prefix of the rows' 64-event chunk counts
    uint64_t cbase[kPushR * (kPushThreads / kWave)];  // first synapse of every chunk of the window
    uint32_t clen[kPushR * (kPushThreads / kWave)];   // its number of events (0 past the end)
    uint32_t plen[kMaxChunkSpikes];
    uint64_t pbase[kMaxChunkSpikes];
    uint32_t bcnt[kMaxBuckets];      // events per bucket in this half, then rank cursor
    uint32_t bst[kMaxBuckets];       // bucket starts in the stage
    uint32_t wb[kMaxBuckets];        // page position of stage entry q is wb[b] + q
    uint32_t fill[kMaxBuckets];      // records already in the bucket's page
    uint32_t pidx[kMaxBuckets];      // page of the bucket
    uint32_t ws[16], ws2[16];
    unsigned long long ws64[16];
};

// Block (x, g1) takes the g1-th equal share of the spikes of step t, reads
// the runs of their rows that target group x, and appends the events to its
// own pages, bucket b = j * T8 + c (delay index j, tile c of the group).
// Dependent memory round trips: spike counts, spike IDs, row descriptors,
// synapses; the page writes are not waited for.  Compact synapses (CMP) give
// 2-byte page records class << 13 | local.
template <bool FIXED, bool CMP>
__global__ __launch_bounds__(kPushThreads) void k_push(StepArgs a, uint32_t i, int64_t t_explicit)
{
    using Rec = typename SynRec<CMP>::T;
    __shared__ PushLDS L;
    const uint64_t t = step_index(a, i, t_explicit);
    const uint32_t x = blockIdx.x % kGroups, g1 = blockIdx.x / kGroups, G1 = a.pg1;
    const uint32_t tid = threadIdx.x;
    const Tiling tl = a.tl;
    const bool dbg = a.dbg_spikes != nullptr;
    const uint32_t NB = (dbg ? 1u : a.lists) * tl.T8;
    const uint32_t sslot = (uint32_t)(t % a.spk_slots);

    // 0. the spike counts of every source tile (their prefix gives each
    //    block an equal share of the spikes) and the block's fill counters
    for (uint32_t b = tid; b < NB; b += kPushThreads) {
        const uint32_t p = page_of(a, x, g1, arrival_slot(a, t, b / tl.T8, dbg), b % tl.T8);
        L.pidx[b] = p;
        L.fill[b] = a.pfill[p];
        L.bcnt[b] = 0;
    }
    const uint32_t M = dbg ? a.dbg_n : load_spike_set(a, sslot, L.pre, L.ws);
    const uint32_t k0 = (uint32_t)((uint64_t)M * g1 / G1), k1 = (uint32_t)((uint64_t)M * (g1 + 1) / G1);
    const uint32_t xlo = x * tl.Gw;
    const uint64_t cap = a.page_cap;
    uint64_t emitted = 0;
    for (uint32_t c0 = k0; c0 < k1; c0 += kMaxChunkSpikes) {
        const uint32_t K = k1 - c0 < kMaxChunkSpikes ? k1 - c0 : kMaxChunkSpikes;
        // 1. this group's run of every row of the chunk
        uint32_t len = 0;
        uint64_t base = 0;
        if (tid < K) {
            const uint32_t k = c0 + tid;
            uint32_t s = dbg ? a.dbg_spikes[k] : spike_at(a, L.pre, sslot, k);
            // a caller's spike list (debug delivery) is checked here: an ID
            // out of range delivers nothing and raises a flag
            const bool bad = s >= a.n;
            if (bad && x == 0) atomicOr(a.flags, kFlagBadSpike);
            s = bad ? 0u : s;
            const RowDesc *d = a.desc + s;
            const uint32_t lo = x ? d->gend[x - 1] : 0u, hi = d->gend[x];
            len = bad ? 0u : hi - lo;
            base = d->start + lo;
            emitted += bad ? 0u : d->gend[kGroups - 1];
        }
        // rows are cut into chunks of 64 events; wave w takes chunks w, w + nw,
        // ...: lane l reads event l of the chunk (one uniform lookup per chunk)
        uint32_t C;
        const uint32_t nch = (len + kWave - 1) / kWave;
        const uint32_t coff = block_scan_u32(nch, L.ws, &C);
        if (tid < K) {
            L.cpre[tid] = coff;
            L.plen[tid] = len;
            L.pbase[tid] = base;
        }
        lds_sync();
        const uint32_t lane = lane_id(), w = tid / kWave;
        constexpr uint32_t nw = kPushThreads / kWave;
        // 2. load phases of kPushR chunks per wave: issue every load, then
        //    bucket-sort and append in two halves (the second half's loads
        //    land while the first is sorted)
        constexpr uint32_t kWin = kPushR * nw;  // chunks per load phase
        for (uint32_t i0 = 0; i0 < C; i0 += kWin) {
            // the window's chunks (start, length), written by each row's thread
            for (uint32_t c = tid; c < kWin; c += kPushThreads) L.clen[c] = 0;
            lds_sync();
            if (tid < K) {
                const uint32_t cb = coff > i0 ? coff : i0, ce = coff + nch < i0 + kWin ? coff + nch : i0 + kWin;
                for (uint32_t c = cb; c < ce; c++) {
                    const uint32_t o = (c - coff) * kWave;
                    L.cbase[c - i0] = base + o;
                    L.clen[c - i0] = len - o < kWave ? len - o : kWave;
                }
            }
            lds_sync();
            // every load is issued unconditionally (lanes past the end read
            // synapse 0 and drop it): a load under a branch would get its own
            // wait for all earlier loads
            Rec rec[kPushR];
            uint32_t okm = 0;  // bit u: rec[u] is an event
#pragma unroll
            for (int u = 0; u < kPushR; u++) {
                const uint32_t cl = u * nw + w;
                const bool ok = lane < L.clen[cl];
                const uint64_t idx = ok ? L.cbase[cl] + lane : 0ull;
                okm |= (uint32_t)ok << u;
                rec[u] = SynRec<CMP>::load(a, idx);
            }
#pragma unroll
            for (int h = 0; h < 2; h++) {
                if (i0 + (uint32_t)h * (kPushR / 2) * nw >= C) break;
                constexpr int R = kPushR / 2;
                uint32_t tr[R];
#pragma unroll
                for (int rr = 0; rr < R; rr++) {
                    const int r = h * R + rr;
                    tr[rr] = 0xffffffffu;
                    if (!((okm >> r) & 1u)) continue;
                    const uint32_t key = rec_key(rec[r]);
                    const uint32_t j = rec_delay(key);
                    if (dbg && a.dbg_j >= 0 && (int32_t)j != a.dbg_j) continue;
                    const uint32_t local = rec_target(key) - xlo;
                    const uint32_t b = (dbg ? 0u : j) * tl.T8 + (local >> tl.logW);
                    const uint32_t rank = atomicAdd(&L.bcnt[b], 1u);
                    tr[rr] = (b << 16) | rank;
                    const uint32_t sv = (b << 16) | (local & (tl.W - 1));
                    if constexpr (CMP) rec[r] = sv | (rec_class(key) << kPageClassShift);
                    else rec[r].x = (int)sv;
                }
                lds_sync();
                // bucket starts in the stage; the page position of staged event
                // q of bucket b is wb[b] + q (mod 2^32); the fill counters advance
                uint32_t staged;
                {
                    const uint32_t P = (NB + kPushThreads - 1) / kPushThreads;
                    const uint32_t b0 = tid * P;
                    uint32_t sum = 0;
                    for (uint32_t k = 0; k < P; k++)
                        if (b0 + k < NB) sum += L.bcnt[b0 + k];
                    uint32_t ex = block_scan_u32_open(sum, h ? L.ws : L.ws2, &staged);
                    for (uint32_t k = 0; k < P; k++) {
                        if (b0 + k < NB) {
                            const uint32_t bb = b0 + k, cnt = L.bcnt[bb], f = L.fill[bb];
                            L.bst[bb] = ex;
                            L.wb[bb] = f - ex;
                            L.fill[bb] = f + cnt;
                            L.bcnt[bb] = 0;
                            ex += cnt;
                        }
                    }
                }
                lds_sync();
                Rec *stage = (Rec *)L.stage;
#pragma unroll
                for (int rr = 0; rr < R; rr++) {
                    if (tr[rr] == 0xffffffffu) continue;
                    stage[L.bst[tr[rr] >> 16] + (tr[rr] & 0xffffu)] = rec[h * R + rr];
                }
                lds_sync();
                // no barrier after the write-out: the next half's first barrier
                // follows every thread's write-out, and only then are wb and the
                // stage rewritten
                for (uint32_t q = tid; q < staged; q += kPushThreads) {
                    const Rec r2 = stage[q];
                    const uint32_t key = rec_key(r2);
                    const uint32_t b = key >> 16, low = key & 0xffffu;
                    const uint32_t pos = L.wb[b] + q;
                    if (pos < cap) {
                        const uint64_t e = (uint64_t)L.pidx[b] * cap + pos;
                        if constexpr (CMP) a.pages16[e] = (uint16_t)low;
                        else a.pages[e] = make_int2((int)low, r2.y);
                    } else {
                        const uint32_t c = b % tl.T8;
                        long long units;
                        uint32_t local;
                        if constexpr (CMP) {
                            units = class_units(a, low >> kPageClassShift);
                            local = low & kPageLocalMask;
                        } else {
                            units = units_of<FIXED>(r2.y, a.m.shift64);
                            local = low;
                        }
                        overflow_add<FIXED>(a, arrival_slot(a, t, b / tl.T8, dbg), x * tl.T8 + c, local, units);
                    }
                }
            }
        }
    }
    lds_sync();
    for (uint32_t b = tid; b < NB; b += kPushThreads) a.pfill[L.pidx[b]] = L.fill[b];
    if (!dbg && x == 0) {  // events emitted at t, counted once per spike
        const uint64_t tot = block_sum_u64(emitted, L.ws64);
        if (tid == 0 && tot) atomicAdd((unsigned long long *)&a.events8[t * kGroups], (unsigned long long)tot);
    }
}

// ------------------------------------------------------------ tile kernel

template <bool FIXED>
struct TileLDS {
    typename Acc<FIXED>::T acc[kMaxTileW];
    uint16_t spk[kMaxTileW];
    uint32_t pre[kMaxTiles + 1];   // direct: spike-count prefix; binned: page prefix
    uint32_t cbase[kTileThreads / kWave * 16];  // binned: first record of every chunk of the window
    uint32_t clen[kTileThreads / kWave * 16];   // its number of records (0 past the end)
    uint32_t wpre[kTileThreads / kWave][kWave + 1];
    uint64_t wbeg[kTileThreads / kWave][kWave];
    uint32_t ws[16];
    unsigned long long ws64[16];
    uint32_t nspk;
    uint64_t pois[256];
    uint16_t guide[256];
    // compact records: accumulator units of each weight class (one LDS load
    // per record instead of a chain of selects among the kernel arguments)
    long long wtab[kMaxClasses];
};

template <bool FIXED, bool CMP>
__global__ __launch_bounds__(kTileThreads) void k_tile(StepArgs a, uint32_t i, int64_t t_explicit)
{
    __shared__ TileLDS<FIXED> L;
    const uint64_t t = step_index(a, i, t_explicit);
    const uint32_t tid = threadIdx.x, lane = lane_id();
    const Tiling tl = a.tl;
    const uint32_t x = blockIdx.x % kGroups, cl = blockIdx.x / kGroups;
    const uint32_t tile = x * tl.T8 + cl;
    const uint32_t tile_lo = tile * tl.W;
    const uint32_t tile_n = tile_lo < a.n ? (a.n - tile_lo < tl.W ? a.n - tile_lo : tl.W) : 0u;
    const ModelArgs &m = a.m;
    const bool debug = a.dbg_out != nullptr;
    const uint32_t pslot = debug || a.direct ? 0u : (uint32_t)(t % a.pslots);

    // 0. loads that do not depend on delivery are issued first.  Loads
    //    complete in issue order, so the small ones that are waited for soon
    //    (drive table, page fill counts, overflow flag) go before the tile's
    //    neuron state, which stays in flight until the update needs it.
    //    All are unconditional loads from clamped indices (see the push kernel).
    uint64_t pz = 0;
    uint16_t gz = 0;
    const bool drive = m.pois_len && !debug;
    if (drive) {
        pz = a.pois[tid < m.pois_len ? tid : 0u];
        gz = a.pois_guide[tid & 255u];
    }
    uint32_t pf = 0, ovf = 0;
    if (!a.direct) {
        pf = a.pfill[page_of(a, x, tid < a.pg1 ? tid : 0u, pslot, cl)];  // masked where used
        ovf = a.ovf_flag[(uint64_t)pslot * tl.T + tile];
    }
    float Vr[kRounds];
    uint32_t Rr[kRounds];
#pragma unroll
    for (int u = 0; u < kRounds; u++) {
        const uint32_t q = u * kTileThreads + tid;
        const uint32_t gi = q < tile_n ? tile_lo + q : 0u;
        Vr[u] = a.V[gi];
        Rr[u] = a.ref[gi];
    }
    for (uint32_t q = tid; q < tl.W; q += kTileThreads) L.acc[q] = 0;
    if (drive) {
        if (tid < m.pois_len) L.pois[tid] = pz;
        if (tid < 256) L.guide[tid] = gz;
    }
    if (tid == 0) {
        L.nspk = 0;
        for (uint32_t k = 0; k < kMaxClasses; k++) L.wtab[k] = a.wval[k];
    }

    // 1. accumulate every event arriving at t (the state loads above stay
    //    in flight: the barriers below order LDS traffic only)
    uint64_t delivered = 0;
    lds_sync();
    if (a.direct) {
        // spikes of step t - d for every delay d, through the runs of their
        // rows in this tile (only the synapses of delay d when there are several)
        uint64_t mine = 0;
        if (debug) {
            mine = gather_direct<FIXED, CMP, false>(a, L.acc, L.pre, L.wpre, L.wbeg, tile, tile_lo, a.dbg_n, 0, a.dbg_j,
                                                   L.wtab);
        } else {
            for (uint32_t j = 0; j < a.lists; j++) {
                const uint64_t d = (uint64_t)a.dmin + j;
                if (t < d) break;
                const uint32_t dslot = (uint32_t)((t - d) % a.spk_slots);
                const uint32_t P = load_spike_set(a, dslot, L.pre, L.ws);
                mine += gather_direct<FIXED, CMP, false>(a, L.acc, L.pre, L.wpre, L.wbeg, tile, tile_lo, P, dslot,
                                                         a.lists > 1 ? (int32_t)j : -1, L.wtab);
                lds_sync();
            }
        }
        delivered = block_sum_u64(mine, L.ws64);
    } else {
        // pages cut into chunks of 64 loads (a load is one full record, or two
        // compact ones: page capacities are multiples of 16 records, so a pair
        // never straddles pages); wave w drains chunks w, w + nw, ...
        constexpr uint32_t kPer = CMP ? 2u : 1u;
        constexpr uint32_t kChunk = kPer * kWave;
        const uint32_t cap = a.page_cap, G1 = a.pg1;
        pf = tid < G1 ? pf : 0u;
        const uint32_t ne = pf < cap ? pf : cap;  // records stored in page tid
        uint32_t C;
        const uint32_t cex = block_scan_u32((ne + kChunk - 1) / kChunk, L.ws, &C);
        delivered = block_sum_u64(pf, L.ws64);  // includes events that overflowed
        const uint32_t w = tid / kWave;
        constexpr uint32_t nw = kTileThreads / kWave;
        constexpr int kDrain = 16;  // loads in flight per lane before their atomics
        constexpr uint32_t kWin = kDrain * nw;
        const uint32_t nchp = (ne + kChunk - 1) / kChunk;
        for (uint32_t i0 = 0; i0 < C; i0 += kWin) {
            // the window's chunks (first record, length), written by each page's thread
            for (uint32_t c = tid; c < kWin; c += kTileThreads) L.clen[c] = 0;
            lds_sync();
            if (tid < G1) {
                const uint32_t cb = cex > i0 ? cex : i0, ce = cex + nchp < i0 + kWin ? cex + nchp : i0 + kWin;
                const uint32_t pbase = page_of(a, x, tid, pslot, cl) * cap;
                for (uint32_t c = cb; c < ce; c++) {
                    const uint32_t o = (c - cex) * kChunk;
                    L.cbase[c - i0] = (pbase + o) / kPer;
                    L.clen[c - i0] = ne - o < kChunk ? ne - o : kChunk;
                }
            }
            lds_sync();
            if constexpr (CMP) {
                const uint32_t *pw = (const uint32_t *)a.pages16;
                uint32_t r[kDrain];
                uint32_t okm = 0;  // bits 2u, 2u + 1: the two records of r[u]
#pragma unroll
                for (int u = 0; u < kDrain; u++) {
                    const uint32_t cw = u * nw + w;
                    const uint32_t len = L.clen[cw];
                    const bool ok = 2 * lane < len;
                    const uint32_t idx = ok ? L.cbase[cw] + lane : 0u;
                    okm |= ((uint32_t)ok | (uint32_t)(2 * lane + 1 < len) << 1) << (2 * u);
                    r[u] = pw[idx];  // unconditional, see the push kernel
                }
#pragma unroll
                for (int u = 0; u < kDrain; u++) {
                    // both records' units read before either add
                    const uint32_t r0 = r[u] & 0xffffu, r1 = r[u] >> 16;
                    const long long u0 = L.wtab[(r0 >> kPageClassShift) & (kMaxClasses - 1)];
                    const long long u1 = L.wtab[(r1 >> kPageClassShift) & (kMaxClasses - 1)];
                    if ((okm >> (2 * u)) & 1u) Acc<FIXED>::add(&L.acc[r0 & kPageLocalMask], u0);
                    if ((okm >> (2 * u + 1)) & 1u) Acc<FIXED>::add(&L.acc[r1 & kPageLocalMask], u1);
                }
            } else {
                int2 r[kDrain];
                uint32_t okm = 0;
#pragma unroll
                for (int u = 0; u < kDrain; u++) {
                    const uint32_t cw = u * nw + w;
                    const bool ok = lane < L.clen[cw];
                    const uint32_t idx = ok ? L.cbase[cw] + lane : 0u;
                    okm |= (uint32_t)ok << u;
                    r[u] = a.pages[idx];  // unconditional, see the push kernel
                }
#pragma unroll
                for (int u = 0; u < kDrain; u++)
                    if ((okm >> u) & 1u) Acc<FIXED>::add(&L.acc[(uint32_t)r[u].x], units_of<FIXED>(r[u].y, m.shift64));
            }
            lds_sync();  // the window's map is read before the next one is written
        }
        if (tid < G1) a.pfill[page_of(a, x, tid, pslot, cl)] = 0;
        lds_sync();
        if (ovf) {  // events that did not fit their page (global fallback)
            const uint64_t st = (uint64_t)pslot * tl.T + tile;
            for (uint32_t q = tid; q < tile_n; q += kTileThreads) {
                const uint64_t gi = st * tl.W + q;
                if (FIXED) {
                    int32_t *o = (int32_t *)a.acc_ovf + gi;
                    L.acc[q] += *o;
                    *o = 0;
                } else {
                    unsigned long long *o = (unsigned long long *)a.acc_ovf + gi;
                    L.acc[q] += *o;
                    *o = 0;
                }
            }
            if (tid == 0) a.ovf_flag[st] = 0;
        }
    }
    lds_sync();

    if (debug) {  // delivery check: hand the accumulated input back, no update
        for (uint32_t q = tid; q < tile_n; q += kTileThreads) {
            if (FIXED) ((int32_t *)a.dbg_out)[tile_lo + q] = (int32_t)L.acc[q];
            else ((float *)a.dbg_out)[tile_lo + q] = fixed64_to_float(L.acc[q], m.shift64);
        }
        return;
    }

    // 2. neuron update (forward Euler in fp32, every operation rounded on its
    //    own), spikes collected in LDS
    uint64_t ev = 0;
#pragma unroll
    for (int u = 0; u < kRounds; u++) {
        const uint32_t q = u * kTileThreads + tid;
        bool spk = false;
        if (q < tile_n) {
            const uint32_t gi = tile_lo + q;
            uint32_t K = 0;
            if (m.pois_len) {  // K = min { k : hi32 < T_k }, searched from the guide entry
                const uint32_t h = hash_hi32(step_hash(m.keys.pois, gi, t));
                uint32_t k = L.guide[h >> 24];
                while ((uint64_t)h >= L.pois[k]) k++;
                K = k;
            }
            float I;
            if (FIXED) {
                const int32_t qt = (int32_t)L.acc[q] + (int32_t)K * m.ext_wq + m.bias_q;
                I = ldexpf((float)qt, -m.shift);
            } else {
                const float isyn = fixed64_to_float(L.acc[q], m.shift64);
                const float ext = __fmul_rn((float)K, m.ext_w);
                I = __fadd_rn(__fadd_rn(isyn, ext), m.i_bias);
            }
            float V = Vr[u];
            if (m.kind == SPK_SOURCE) {
                const float av = __fsub_rn(m.v_rest, V);
                const float bv = __fmul_rn(m.k, av);
                const float cv = __fadd_rn(V, bv);
                V = __fadd_rn(cv, I);
                spk = (uint64_t)hash_hi32(step_hash(m.keys.bern, gi, t)) < m.src_thr;
            } else {
                uint32_t r = Rr[u];
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
                a.ref[gi] = (uint8_t)r;
            }
            a.V[gi] = V;
            if (spk && a.direct) ev += a.outdeg[gi];  // binned: counted by the push kernel
        }
        const uint64_t mask = __ballot(spk);
        if (mask) {  // wavefront-ballot compaction into the tile's LDS list
            const int leader = __ffsll((unsigned long long)mask) - 1;
            uint32_t wb = 0;
            if ((int)lane == leader) wb = atomicAdd(&L.nspk, (uint32_t)__popcll(mask));
            wb = (uint32_t)__builtin_amdgcn_readlane((int)wb, leader);
            if (spk) {
                const uint32_t rank = __builtin_amdgcn_mbcnt_hi(
                    (uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
                L.spk[wb + rank] = (uint16_t)q;
            }
        }
    }
    if (a.direct) ev = block_sum_u64(ev, L.ws64);
    else lds_sync();

    // 3. publish into the tile's own segment of the spike list of t
    const uint32_t ns = L.nspk;
    const uint64_t seg = (uint64_t)(t % a.spk_slots) * tl.T + tile;
    uint32_t *dst = a.spk_ids + seg * tl.W;
    for (uint32_t q = tid; q < ns; q += kTileThreads) dst[q] = tile_lo + L.spk[q];
    if (tid == 0) {
        a.spk_cnt[seg] = ns;
        if (ns) atomicAdd(&a.counts8[t * kGroups + x], ns);
        if (ev) atomicAdd((unsigned long long *)&a.events8[t * kGroups + x], (unsigned long long)ev);
        if (delivered)
            atomicAdd((unsigned long long *)&a.delivered8[t * kGroups + x], (unsigned long long)delivered);
    }
}

// ---------------------------------------------------------------- record

__global__ __launch_bounds__(kTileThreads) void k_record(StepArgs a, uint32_t i, int64_t t_explicit)
{
    __shared__ uint32_t pre[kMaxTiles + 1];
    __shared__ uint32_t ws[16];
    const uint64_t t = step_index(a, i, t_explicit);
    const uint32_t slot = (uint32_t)(t % a.spk_slots);
    const uint32_t M = load_spike_set(a, slot, pre, ws);
    const uint64_t base = a.raster_offs[t];
    const bool ok = base + M <= a.raster_cap;
    if (ok)
        for (uint32_t k = threadIdx.x; k < M; k += kTileThreads) a.raster[base + k] = spike_at(a, pre, slot, k);
    if (threadIdx.x == 0) {
        a.raster_offs[t + 1] = ok ? base + M : base;
        if (!ok) atomicOr(a.flags, 2u);
    }
}

__global__ void k_advance(uint64_t *t_base, uint32_t steps)
{
    if (threadIdx.x == 0) *t_base += steps;
}

__global__ __launch_bounds__(256) void k_stream_copy(const uint4 *src, uint4 *dst, uint64_t n16)
{
    for (uint64_t k = (uint64_t)blockIdx.x * 256 + threadIdx.x; k < n16; k += (uint64_t)gridDim.x * 256)
        dst[k] = src[k];
}

// Fill n words with zero (a kernel, not a memset: usable in captured graphs).
__global__ __launch_bounds__(256) void k_zero_u32(uint32_t *p, uint64_t n)
{
    for (uint64_t k = (uint64_t)blockIdx.x * 256 + threadIdx.x; k < n; k += (uint64_t)gridDim.x * 256) p[k] = 0;
}

// Streaming read of n16 16-byte words, four loads in flight per thread; the
// xor of everything read is stored only if it equals a value a memset never
// produces, so the loads cannot be dropped and nothing is written.
__global__ __launch_bounds__(256) void k_stream_read(const uint4 *src, uint64_t n16, uint32_t *sink)
{
    const uint64_t stride = (uint64_t)gridDim.x * 256;
    uint64_t k = (uint64_t)blockIdx.x * 256 + threadIdx.x;
    uint32_t acc = 0;
    for (; k + 3 * stride < n16; k += 4 * stride) {
        const uint4 a = src[k], b = src[k + stride], c = src[k + 2 * stride], d = src[k + 3 * stride];
        acc ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w;
    }
    for (; k < n16; k += stride) {
        const uint4 a = src[k];
        acc ^= a.x ^ a.y ^ a.z ^ a.w;
    }
    if (acc == 0x13579bdfu) sink[0] = acc;
}

}  // namespace

uint32_t push_blocks_per_group()
{
    const int g = cu_count() / (int)kGroups;
    return g < 1 ? 1u : (uint32_t)g;
}

hipError_t launch_push(const StepArgs &a, uint32_t i, int64_t t_explicit, hipStream_t s)
{
    if (a.proc) return launch_push_proc(a, i, t_explicit, s);
    const uint32_t nj = a.dbg_spikes ? 1u : a.lists;
    if (a.direct || a.tl.T > kMaxTiles || a.tl.T != kGroups * a.tl.T8 || nj * a.tl.T8 > kMaxBuckets ||
        a.tl.W > 65536 || a.pg1 == 0 || a.pg1 > kPushThreads || a.pslots == 0 || a.page_cap == 0)
        return hipErrorInvalidValue;
    if (a.compact ? (!a.syn32 || !a.pages16) : (!a.syn || !a.pages)) return hipErrorInvalidValue;
    const dim3 grid(kGroups * a.pg1), block(kPushThreads);
    if (a.compact) {
        if (a.m.fixed) hipLaunchKernelGGL((k_push<true, true>), grid, block, 0, s, a, i, t_explicit);
        else hipLaunchKernelGGL((k_push<false, true>), grid, block, 0, s, a, i, t_explicit);
    } else {
        if (a.m.fixed) hipLaunchKernelGGL((k_push<true, false>), grid, block, 0, s, a, i, t_explicit);
        else hipLaunchKernelGGL((k_push<false, false>), grid, block, 0, s, a, i, t_explicit);
    }
    return hipGetLastError();
}

hipError_t launch_tile(const StepArgs &a, uint32_t i, int64_t t_explicit, hipStream_t s)
{
    if (a.tl.W > kMaxTileW || a.m.pois_len > 256 || a.tl.T != kGroups * a.tl.T8 || a.tl.T > kMaxTiles ||
        (!a.direct && (a.pg1 == 0 || a.pg1 > kTileThreads || a.pslots == 0)) || a.spk_slots == 0 ||
        (a.direct && a.spk_slots <= a.dmin && !a.dbg_out))
        return hipErrorInvalidValue;
    // rows are read only by direct delivery (procedural synapses are never
    // stored, and always binned); pages only by binned delivery
    const bool rows_ok = a.proc ? !a.direct : (a.compact ? a.syn32 != nullptr : a.syn != nullptr);
    const bool pages_ok = a.direct || (a.compact ? a.pages16 != nullptr : a.pages != nullptr);
    if (!rows_ok || !pages_ok) return hipErrorInvalidValue;
    if (!a.direct && (a.page_cap % 16)) return hipErrorInvalidValue;  // record pairs stay in their page
    const dim3 grid(a.tl.T), block(kTileThreads);
    if (a.compact) {
        if (a.m.fixed) hipLaunchKernelGGL((k_tile<true, true>), grid, block, 0, s, a, i, t_explicit);
        else hipLaunchKernelGGL((k_tile<false, true>), grid, block, 0, s, a, i, t_explicit);
    } else {
        if (a.m.fixed) hipLaunchKernelGGL((k_tile<true, false>), grid, block, 0, s, a, i, t_explicit);
        else hipLaunchKernelGGL((k_tile<false, false>), grid, block, 0, s, a, i, t_explicit);
    }
    return hipGetLastError();
}

hipError_t launch_record(const StepArgs &a, uint32_t i, int64_t t_explicit, hipStream_t s)
{
    if (a.tl.T > kMaxTiles) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_record, dim3(1), dim3(kTileThreads), 0, s, a, i, t_explicit);
    return hipGetLastError();
}

hipError_t launch_advance(uint64_t *t_base, uint32_t steps, hipStream_t s)
{
    hipLaunchKernelGGL(k_advance, dim3(1), dim3(64), 0, s, t_base, steps);
    return hipGetLastError();
}

hipError_t zero_words(uint32_t *p, uint64_t n, hipStream_t s)
{
    if (n == 0) return hipSuccess;
    uint64_t blocks = (n + 255) / 256;
    const uint64_t most = (uint64_t)cu_count() * 8;
    blocks = blocks < most ? blocks : most;
    hipLaunchKernelGGL(k_zero_u32, dim3((uint32_t)(blocks ? blocks : 1)), dim3(256), 0, s, p, n);
    return hipGetLastError();
}

hipError_t stream_read(const void *src, uint64_t bytes, uint32_t *sink, hipStream_t s)
{
    hipLaunchKernelGGL(k_stream_read, dim3(cu_count() * 16), dim3(256), 0, s, (const uint4 *)src, bytes / 16, sink);
    return hipGetLastError();
}

hipError_t stream_copy(const void *src, void *dst, uint64_t bytes, hipStream_t s)
{
    hipLaunchKernelGGL(k_stream_copy, dim3(cu_count() * 16), dim3(256), 0, s, (const uint4 *)src,
                       (uint4 *)dst, bytes / 16);
    return hipGetLastError();
}

}  // namespace spk
