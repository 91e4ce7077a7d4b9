// spk_proc.hip -- procedural connectivity: the synapses of a fixed
// out-degree network are never stored; the row of every neuron that fires
// is generated again from the network's parameters when its events are
// filed (the paper's Sec. V names procedural connectivity as future work:
// store only the parameters that create the network and generate the
// adjacency on the fly).
//
// A synapse j of source s is the generator's draw: target
// range(H(seed, TGT, s, j), n), delay index range(H(seed, DELAY, s, j),
// lists), weight by source population or w_lo + (w_hi - w_lo) u24(H(seed,
// W, s, j)).  The push kernel here replaces the stored-row push of binned
// delivery (spk_step.hip): push block (x, g1) takes the same equal share of
// the step's spikes, generates every synapse of their rows (each XCD group
// keeps the 1/8 that target it), and files the kept events into the same
// pages with the same counting sort, so the tile kernel is unchanged.  The
// cost moves from the synapse stream (no bytes read per event) to hashing
// (one mixer round per generated synapse, eight synapses generated per kept
// event); the memory of the synapses (4 or 8 bytes each) is not needed.
//
// Generation is wave-local: lanes walk consecutive synapses of the wave's
// slice of the rows, draw each one's target, keep those of the block's
// group, and compact them with a ballot into a ring of the wave in LDS as
// (target, spike, synapse index); the delay (and a per-synapse weight) is
// drawn when an entry is taken from the ring, where every lane holds a kept
// synapse (drawn before compaction, one kept lane in eight would make the
// whole wave run those mixer rounds).  Every window takes kProcR events per
// lane from the rings and sorts them by (arrival slot, tile) as the
// stored-row push does.
#include <hip/hip_runtime.h>

#include "spk_dev.h"

namespace spk {

namespace {

constexpr int kProcThreads = 1024;
static_assert(kProcThreads == (int)kBlockThreads, "the block-wide helpers assume workgroups of kBlockThreads");
constexpr uint32_t kProcChunk = 1024;                      // spikes generated per chunk
constexpr uint32_t kProcWaves = kProcThreads / kWave;
constexpr uint32_t kRing = 128;                            // events a wave holds between windows
constexpr uint32_t kNoSpike = 0xffffffffu;
static_assert(kProcChunk <= (1u << 16), "ring entries hold the spike of the chunk in 16 bits");

template <bool CMP>
struct ProcLDS {
    using Rec = typename SynRec<CMP>::T;
    static constexpr int R = CMP ? 12 : 8;                    // events per lane per window
    static constexpr uint32_t kWin = R * kProcThreads;        // events sorted at once
    Rec stage[kWin];                 // bucket-sorted events {bucket << 16 | local, weight}; compact:
                                     // u32 bucket << 16 | class << 13 | local
    uint2 ring[kProcWaves][kRing];   // kept synapses of each wave, not yet taken: {target,
                                     // spike of the chunk << 16 | synapse index}
    uint32_t sid[kProcChunk];        // the chunk's spikes (kNoSpike: an ID out of range)
    uint32_t pre[kMaxTiles + 1];     // prefix of the source tiles' spike counts
    uint32_t bcnt[kMaxBuckets];      // events per bucket in this window, then rank cursor
    uint32_t bst[kMaxBuckets];       // bucket starts in the stage
    uint32_t wb[kMaxBuckets];        // page position of stage entry q is wb[b] + q
    uint32_t fill[kMaxBuckets];      // records already in the bucket's page
    uint32_t pidx[kMaxBuckets];      // page of the bucket
    uint32_t more[kProcWaves];       // the wave has events left to generate or take
    uint32_t ws[16];
    unsigned long long ws64[16];
};

// The stored-format record of synapse j of source s (its target tgt is
// known): compact {class << 30 | delay index << 24 | target} with class =
// source population, or full {delay index << 24 | target, weight bits}.
// pw: the weight stream's prefix of row s, mix64(keys.w ^ s) (per-synapse
// weights: the synapse's draw is mix64(pw ^ j), i.e. key_hash(keys.w, s, j)).
template <bool CMP>
__device__ __forceinline__ typename SynRec<CMP>::T proc_record(const StepArgs &a, uint32_t s, uint32_t j,
                                                              uint32_t tgt, uint32_t jd, uint64_t pw)
{
    const uint32_t key = (jd << kTargetBits) | tgt;
    if constexpr (CMP) {
        return key | ((s < a.pr.n_exc ? 0u : 1u) << kClassShift);
    } else {
        float w;
        if (a.pr.w_uniform) {
            const uint64_t h = mix64(pw ^ (uint64_t)j);
            const float u = (float)(uint32_t)(h >> 40) * (1.0f / 16777216.0f);
            w = __fadd_rn(a.pr.w_lo, __fmul_rn(__fsub_rn(a.pr.w_hi, a.pr.w_lo), u));
        } else {
            w = s < a.pr.n_exc ? a.pr.w_exc : a.pr.w_inh;
        }
        const int32_t wb = a.m.fixed ? (int32_t)__builtin_rintf(__fmul_rn(w, a.pr.qscale)) : __float_as_int(w);
        return make_int2((int)key, wb);
    }
}
template <bool CMP>
__device__ __forceinline__ typename SynRec<CMP>::T proc_record(const StepArgs &a, uint32_t s, uint32_t j,
                                                              uint32_t tgt, uint32_t jd)
{
    return proc_record<CMP>(a, s, j, tgt, jd, CMP || !a.pr.w_uniform ? 0ull : mix64(a.m.keys.w ^ (uint64_t)s));
}

template <bool FIXED, bool CMP>
__global__ __launch_bounds__(kProcThreads) void k_push_proc(StepArgs a, uint32_t i, int64_t t_explicit)
{
    using Rec = typename SynRec<CMP>::T;
    __shared__ ProcLDS<CMP> L;
    constexpr int kProcR = ProcLDS<CMP>::R;
    const uint64_t t = step_index(a, i, t_explicit);
    const uint32_t x = blockIdx.x % kGroups, g1 = blockIdx.x / kGroups, G1 = a.pg1;
    const uint32_t tid = threadIdx.x, lane = lane_id();
    const uint32_t w = __builtin_amdgcn_readfirstlane(tid / kWave);
    const Tiling tl = a.tl;
    const bool dbg = a.dbg_spikes != nullptr;
    const uint32_t NB = (dbg ? 1u : a.lists) * tl.T8;
    const uint32_t sslot = (uint32_t)(t % a.spk_slots);
    const uint32_t kout = a.pr.k_out;

    const uint32_t abase = arrival_slot(a, t, 0, dbg);
    for (uint32_t b = tid; b < NB; b += kProcThreads) {
        const uint32_t j = div_t8(tl, b);
        const uint32_t p = page_of(a, x, g1, arrival_slot_from(a, abase, j, dbg), b - j * tl.T8);
        L.pidx[b] = p;
        L.fill[b] = a.pfill[p];
        L.bcnt[b] = 0;
    }
    const uint32_t M = dbg ? a.dbg_n : load_spike_set(a, sslot, L.pre, L.ws);
    uint32_t k0, k1;
    equal_share(M, g1, G1, &k0, &k1);
    const uint32_t xlo = x * tl.Gw;
    const uint64_t cap = a.page_cap;
    uint64_t emitted = 0;
    for (uint32_t c0 = k0; c0 < k1 && kout; c0 += kProcChunk) {
        const uint32_t K = k1 - c0 < kProcChunk ? k1 - c0 : kProcChunk;
        if (tid < K) {
            const uint32_t k = c0 + tid;
            const uint32_t s = dbg ? a.dbg_spikes[k] : spike_at(a, L.pre, sslot, k);
            // a caller's spike list (debug delivery) is checked here: an ID
            // out of range generates nothing and raises a flag
            const bool bad = s >= a.n;
            if (bad && x == 0) atomicOr(a.flags, kFlagBadSpike);
            L.sid[tid] = bad ? kNoSpike : s;
            emitted += bad ? 0u : kout;
        }
        lds_sync();
        // the wave's slice [vb, ve) of the chunk's K * kout synapses; lane l
        // generates synapse v = vcur + l, i.e. synapse j of spike si
        const uint32_t V = K * kout;
        const uint32_t vb = (uint32_t)((uint64_t)V * w / kProcWaves);
        const uint32_t ve = (uint32_t)((uint64_t)V * (w + 1) / kProcWaves);
        uint32_t vcur = vb;                      // (wave-uniform)
        uint32_t si = (vb + lane) / kout, j = (vb + lane) - si * kout;
        uint32_t sicur = kNoSpike, scur = kNoSpike;  // the lane's spike (index, ID) whose
        uint64_t pt = 0;                              // target-stream prefix pt is held
        uint32_t head = 0, cnt = 0;              // the wave's ring (wave-uniform)
        for (;;) {
            Rec rec[kProcR];
            uint32_t okm = 0;  // bit u: rec[u] is an event
#pragma unroll
            for (int u = 0; u < kProcR; u++) {
                while (cnt < kWave && vcur < ve) {
                    const bool live = vcur + lane < ve;
                    bool keep = false;
                    uint32_t tgt = 0;
                    if (live) {
                        if (si != sicur) {  // (once per kout synapses)
                            sicur = si;
                            scur = L.sid[si];
                            pt = mix64(a.m.keys.tgt ^ (uint64_t)scur);
                        }
                        if (scur != kNoSpike) {
                            tgt = hash_range(mix64(pt ^ (uint64_t)j), a.n);
                            keep = tgt - xlo < tl.Gw;  // (unsigned) the target is in group x
                        }
                    }
                    const uint64_t bal = __ballot(keep);
                    if (keep) {
                        const uint32_t rank =
                            __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
                        L.ring[w][(head + cnt + rank) & (kRing - 1)] = make_uint2(tgt, si << 16 | j);
                    }
                    cnt += (uint32_t)__popcll(bal);
                    vcur += kWave;
                    j += kWave;
                    while (j >= kout) {
                        j -= kout;
                        si++;
                    }
                }
                lds_wave_sync();  // the ring's new entries are visible to every lane
                const uint32_t avail = cnt < kWave ? cnt : kWave;
                bool ok = lane < avail;
                const uint2 ge = L.ring[w][(head + lane) & (kRing - 1)];  // (read unconditionally; used if ok)
                rec[u] = Rec{};
                if (ok) {  // the kept synapse's delay (and weight) draws
                    const uint32_t s = L.sid[ge.y >> 16], j2 = ge.y & 0xffffu;
                    const uint32_t jd = a.lists > 1 ? hash_range(key_hash(a.m.keys.delay, s, j2), a.lists) : 0u;
                    ok = !(dbg && a.dbg_j >= 0 && (int32_t)jd != a.dbg_j);
                    rec[u] = proc_record<CMP>(a, s, j2, ge.x, jd);
                }
                okm |= (uint32_t)ok << u;
                head += avail;
                cnt -= avail;
                lds_wave_sync();  // taken before the ring is written again
            }
            if (lane == 0) L.more[w] = cnt > 0 || vcur < ve ? 1u : 0u;
            // rank every event of the window within its bucket (LDS counters)
            uint32_t tr[kProcR];
#pragma unroll
            for (int q = 0; q < kProcR; q++) {
                tr[q] = 0xffffffffu;
                if (!((okm >> q) & 1u)) continue;
                const uint32_t key = rec_key(rec[q]);
                const uint32_t local = rec_target(key) - xlo;
                const uint32_t b = (dbg ? 0u : rec_delay(key)) * tl.T8 + (local >> tl.logW);
                const uint32_t rank = atomicAdd(&L.bcnt[b], 1u);
                tr[q] = (b << 16) | rank;
                const uint32_t sv = (b << 16) | (local & (tl.W - 1));
                if constexpr (CMP) rec[q] = sv | (rec_class(key) << kPageClassShift);
                else rec[q].x = (int)sv;
            }
            lds_sync();
            // bucket starts in the stage; the page position of staged event q
            // of bucket b is wb[b] + q (mod 2^32); the fill counters advance
            uint32_t staged;
            {
                const uint32_t P = (NB + kProcThreads - 1) / kProcThreads;
                const uint32_t b0 = tid * P;
                uint32_t sum = 0;
                for (uint32_t k = 0; k < P; k++)
                    if (b0 + k < NB) sum += L.bcnt[b0 + k];
                uint32_t ex = block_scan_u32_open(sum, L.ws, &staged);
                for (uint32_t k = 0; k < P; k++) {
                    if (b0 + k < NB) {
                        const uint32_t bb = b0 + k, c = L.bcnt[bb], f = L.fill[bb];
                        L.bst[bb] = ex;
                        L.wb[bb] = f - ex;
                        L.fill[bb] = f + c;
                        L.bcnt[bb] = 0;
                        ex += c;
                    }
                }
            }
            lds_sync();
#pragma unroll
            for (int q = 0; q < kProcR; q++) {
                if (tr[q] == 0xffffffffu) continue;
                L.stage[L.bst[tr[q] >> 16] + (tr[q] & 0xffffu)] = rec[q];
            }
            lds_sync();
            // coalesced appends: consecutive staged events of a bucket go to
            // consecutive page positions
            for (uint32_t q = tid; q < staged; q += kProcThreads) {
                const Rec r2 = L.stage[q];
                const uint32_t key = rec_key(r2);
                const uint32_t b = key >> 16, low = key & 0xffffu;
                const uint32_t pos = L.wb[b] + q;
                if (pos < cap) {
                    const uint64_t e = (uint64_t)L.pidx[b] * cap + pos;
                    if constexpr (CMP) a.pages16[e] = (uint16_t)low;
                    else a.pages[e] = make_int2((int)low, r2.y);
                } else {
                    long long units;
                    uint32_t local;
                    if constexpr (CMP) {
                        units = class_units(a, low >> kPageClassShift);
                        local = low & kPageLocalMask;
                    } else {
                        units = units_of<FIXED>(r2.y, a.m.shift64);
                        local = low;
                    }
                    const uint32_t jb = div_t8(tl, b);
                    overflow_add<FIXED>(a, arrival_slot_from(a, abase, jb, dbg), x * tl.T8 + b - jb * tl.T8, local,
                                        units);
                }
            }
            uint32_t any = 0;
            for (uint32_t k = 0; k < kProcWaves; k++) any |= L.more[k];
            lds_sync();  // the stage, wb and more[] are read before the next window writes them
            if (!any) break;
        }
    }
    lds_sync();
    for (uint32_t b = tid; b < NB; b += kProcThreads) a.pfill[L.pidx[b]] = L.fill[b];
    if (!dbg && x == 0) {  // events emitted at t, counted once per spike
        const uint64_t tot = block_sum_u64(emitted, L.ws64);
        if (tid == 0 && tot) atomicAdd((unsigned long long *)&a.events8[t * kGroups], (unsigned long long)tot);
    }
}

// Rows generated once (the graph path's default for procedural networks).
// Between the push and the tile kernels lies a kernel boundary, so pages
// need not stay on one XCD: push block b of NBLK (= pg1, one per compute
// unit) takes the b-th equal share of the step's spikes, generates every
// synapse of their rows once (no group filter: an eighth of the target draws
// of k_push_proc) and files each event into its own page of the target's
// tile, page (group of the tile, b, arrival slot, tile of the group); the
// tile kernel drains the pages of all NBLK push blocks.  Each lane generates
// consecutive synapses of the block's share (the wave's slice), kOnceR per
// window, with the target, delay and weight streams' prefixes of the lane's
// row held in registers; the events are sorted by (delay index, tile) over
// all T tiles of the network, as k_push_proc does within a group.
constexpr uint32_t kOnceChunk = 256;  // spikes per chunk

template <bool CMP>
struct OnceLDS {
    using Rec = typename SynRec<CMP>::T;
    static constexpr int R = CMP ? 12 : 6;                    // events per lane per window
    static constexpr uint32_t kWin = R * kProcThreads;
    Rec stage[kWin];                 // bucket-sorted events {bucket << 16 | page record}
    uint32_t sid[kOnceChunk];        // the chunk's spikes (kNoSpike: an ID out of range)
    uint32_t pre[kMaxTiles + 1];     // prefix of the source tiles' spike counts
    uint32_t bcnt[kOnceMaxB];        // events per bucket in this window, then rank cursor
    uint32_t bst[kOnceMaxB];         // bucket starts in the stage
    uint32_t wb[kOnceMaxB];          // page position of stage entry q is wb[b] + q
    uint32_t fill[kOnceMaxB];        // records already in the bucket's page
    uint32_t pidx[kOnceMaxB];        // page of the bucket
    uint32_t more[kProcWaves];       // the wave has synapses left to generate
    uint32_t ws[16];
    unsigned long long ws64[16];
};

template <bool FIXED, bool CMP>
__global__ __launch_bounds__(kProcThreads) void k_push_proc_once(StepArgs a, uint32_t i, int64_t t_explicit)
{
    using Rec = typename SynRec<CMP>::T;
    __shared__ OnceLDS<CMP> L;
    constexpr int kOnceR = OnceLDS<CMP>::R;
    const uint64_t t = step_index(a, i, t_explicit);
    const uint32_t b = blockIdx.x, NBLK = gridDim.x;
    const uint32_t tid = threadIdx.x, lane = lane_id();
    const uint32_t w = __builtin_amdgcn_readfirstlane(tid / kWave);
    const Tiling tl = a.tl;
    const bool dbg = a.dbg_spikes != nullptr;
    const uint32_t T = tl.T, NB = (dbg ? 1u : a.lists) * T;  // bucket (delay index, tile) = j * T + tile
    const uint32_t sslot = (uint32_t)(t % a.spk_slots);
    const uint32_t kout = a.pr.k_out;

    const uint32_t abase = arrival_slot(a, t, 0, dbg);
    for (uint32_t q = tid; q < NB; q += kProcThreads) {
        // (q / T = (q / 8) / T8: T = 8 T8)
        const uint32_t j = div_t8(tl, q >> 3), tt = q - j * T, x = div_t8(tl, tt);
        const uint32_t p = page_of(a, x, b, arrival_slot_from(a, abase, j, dbg), tt - x * tl.T8);
        L.pidx[q] = p;
        L.fill[q] = a.pfill[p];
        L.bcnt[q] = 0;
    }
    const uint32_t M = dbg ? a.dbg_n : load_spike_set(a, sslot, L.pre, L.ws);
    uint32_t k0, k1;
    equal_share(M, b, NBLK, &k0, &k1);
    const uint64_t cap = a.page_cap;
    const bool uniform_w = !CMP && a.pr.w_uniform;
    uint64_t emitted = 0;
    for (uint32_t c0 = k0; c0 < k1 && kout; c0 += kOnceChunk) {
        const uint32_t K = k1 - c0 < kOnceChunk ? k1 - c0 : kOnceChunk;
        if (tid < K) {
            const uint32_t k = c0 + tid;
            const uint32_t s = dbg ? a.dbg_spikes[k] : spike_at(a, L.pre, sslot, k);
            // a caller's spike list (debug delivery) is checked here: an ID
            // out of range generates nothing and raises a flag
            const bool bad = s >= a.n;
            if (bad && b == 0) atomicOr(a.flags, kFlagBadSpike);
            L.sid[tid] = bad ? kNoSpike : s;
            emitted += bad ? 0u : kout;
        }
        lds_sync();
        // the wave's slice [vb, ve) of the chunk's K * kout synapses; lane l
        // generates synapse v = vcur + l, i.e. synapse j of spike si
        const uint32_t V = K * kout;
        const uint32_t vb = (uint32_t)((uint64_t)V * w / kProcWaves);
        const uint32_t ve = (uint32_t)((uint64_t)V * (w + 1) / kProcWaves);
        uint32_t vcur = vb;                                // (wave-uniform)
        uint32_t si = (vb + lane) / kout, j = (vb + lane) - si * kout;
        uint32_t sicur = kNoSpike, scur = kNoSpike;        // the lane's row (index, ID) and
        uint64_t pt = 0, pd = 0, pw = 0;                   // its streams' prefixes
        for (;;) {
            Rec rec[kOnceR];
            uint32_t okm = 0;  // bit u: rec[u] is an event
#pragma unroll
            for (int u = 0; u < kOnceR; u++) {
                bool ok = false;
                rec[u] = Rec{};
                if (vcur + lane < ve) {
                    if (si != sicur) {  // (once per kout synapses)
                        sicur = si;
                        scur = L.sid[si];
                        pt = mix64(a.m.keys.tgt ^ (uint64_t)scur);
                        pd = mix64(a.m.keys.delay ^ (uint64_t)scur);
                        if (uniform_w) pw = mix64(a.m.keys.w ^ (uint64_t)scur);
                    }
                    if (scur != kNoSpike) {
                        const uint32_t tgt = hash_range(mix64(pt ^ (uint64_t)j), a.n);
                        const uint32_t jd = a.lists > 1 ? hash_range(mix64(pd ^ (uint64_t)j), a.lists) : 0u;
                        ok = !(dbg && a.dbg_j >= 0 && (int32_t)jd != a.dbg_j);
                        rec[u] = proc_record<CMP>(a, scur, j, tgt, jd, pw);
                    }
                }
                okm |= (uint32_t)ok << u;
                vcur += kWave;
                j += kWave;
                while (j >= kout) {
                    j -= kout;
                    si++;
                }
            }
            if (lane == 0) L.more[w] = vcur < ve ? 1u : 0u;
            // rank every event of the window within its bucket (LDS counters)
            uint32_t tr[kOnceR];
#pragma unroll
            for (int q = 0; q < kOnceR; q++) {
                tr[q] = 0xffffffffu;
                if (!((okm >> q) & 1u)) continue;
                const uint32_t key = rec_key(rec[q]);
                const uint32_t tgt = rec_target(key);
                const uint32_t bk = (dbg ? 0u : rec_delay(key)) * T + (tgt >> tl.logW);
                const uint32_t rank = atomicAdd(&L.bcnt[bk], 1u);
                tr[q] = (bk << 16) | rank;
                const uint32_t sv = (bk << 16) | (tgt & (tl.W - 1));
                if constexpr (CMP) rec[q] = sv | (rec_class(key) << kPageClassShift);
                else rec[q].x = (int)sv;
            }
            lds_sync();
            // bucket starts in the stage; the page position of staged event q
            // of bucket b is wb[b] + q (mod 2^32); the fill counters advance
            uint32_t staged;
            {
                const uint32_t P = (NB + kProcThreads - 1) / kProcThreads;
                const uint32_t b0 = tid * P;
                uint32_t sum = 0;
                for (uint32_t k = 0; k < P; k++)
                    if (b0 + k < NB) sum += L.bcnt[b0 + k];
                uint32_t ex = block_scan_u32_open(sum, L.ws, &staged);
                for (uint32_t k = 0; k < P; k++) {
                    if (b0 + k < NB) {
                        const uint32_t bb = b0 + k, c = L.bcnt[bb], f = L.fill[bb];
                        L.bst[bb] = ex;
                        L.wb[bb] = f - ex;
                        L.fill[bb] = f + c;
                        L.bcnt[bb] = 0;
                        ex += c;
                    }
                }
            }
            lds_sync();
#pragma unroll
            for (int q = 0; q < kOnceR; q++) {
                if (tr[q] == 0xffffffffu) continue;
                L.stage[L.bst[tr[q] >> 16] + (tr[q] & 0xffffu)] = rec[q];
            }
            lds_sync();
            // coalesced appends: consecutive staged events of a bucket go to
            // consecutive page positions
            for (uint32_t q = tid; q < staged; q += kProcThreads) {
                const Rec r2 = L.stage[q];
                const uint32_t key = rec_key(r2);
                const uint32_t bk = key >> 16, low = key & 0xffffu;
                const uint32_t pos = L.wb[bk] + q;
                if (pos < cap) {
                    const uint64_t e = (uint64_t)L.pidx[bk] * cap + pos;
                    if constexpr (CMP) a.pages16[e] = (uint16_t)low;
                    else a.pages[e] = make_int2((int)low, r2.y);
                } else {
                    long long units;
                    uint32_t local;
                    if constexpr (CMP) {
                        units = class_units(a, low >> kPageClassShift);
                        local = low & kPageLocalMask;
                    } else {
                        units = units_of<FIXED>(r2.y, a.m.shift64);
                        local = low;
                    }
                    const uint32_t jb = div_t8(tl, bk >> 3);
                    overflow_add<FIXED>(a, arrival_slot_from(a, abase, jb, dbg), bk - jb * T, local, units);
                }
            }
            uint32_t any = 0;
            for (uint32_t k = 0; k < kProcWaves; k++) any |= L.more[k];
            lds_sync();  // the stage, wb and more[] are read before the next window writes them
            if (!any) break;
        }
    }
    lds_sync();
    for (uint32_t q = tid; q < NB; q += kProcThreads) a.pfill[L.pidx[q]] = L.fill[q];
    if (!dbg) {  // events emitted at t (each spike is in one block's share)
        const uint64_t tot = block_sum_u64(emitted, L.ws64);
        if (tid == 0 && tot) atomicAdd((unsigned long long *)&a.events8[t * kGroups], (unsigned long long)tot);
    }
}

// Rows of the given sources as generated, synapse j of row r at out_off[r] + j:
// target, weight bits as the full format stores them (compact classes: the
// class's bits from the table), delay.
__global__ __launch_bounds__(256) void k_export_proc(StepArgs a, ClassTab tab, const uint32_t *rows,
                                                     const uint64_t *out_off, uint32_t *col, uint32_t *wbits,
                                                     uint8_t *delay)
{
    const uint32_t s = rows[blockIdx.x];
    const uint64_t o = out_off[blockIdx.x];
    const uint64_t pt = mix64(a.m.keys.tgt ^ (uint64_t)s);
    for (uint32_t j = threadIdx.x; j < a.pr.k_out; j += 256) {
        const uint32_t tgt = hash_range(mix64(pt ^ (uint64_t)j), a.n);
        const uint32_t jd = a.lists > 1 ? hash_range(key_hash(a.m.keys.delay, s, j), a.lists) : 0u;
        uint32_t wb;
        if (a.compact) {
            wb = tab.bits[s < a.pr.n_exc ? 0 : 1];
        } else {
            wb = (uint32_t)proc_record<false>(a, s, j, tgt, jd).y;
        }
        col[o + j] = tgt;
        wbits[o + j] = wb;
        delay[o + j] = (uint8_t)(a.dmin + jd);
    }
}

// Per-target sum of the |weight| terms of every in-synapse (the units of the
// stored-row range pass: |quantised w| in fixed mode, |w| in units of 2^-24
// rounded up in fp32 mode), one global atomic per generated synapse.
__global__ __launch_bounds__(256) void k_proc_in_abs_sum(StepArgs a, unsigned long long *insum)
{
    const uint32_t s = blockIdx.x;
    const uint64_t pt = mix64(a.m.keys.tgt ^ (uint64_t)s);
    for (uint32_t j = threadIdx.x; j < a.pr.k_out; j += 256) {
        const uint32_t tgt = hash_range(mix64(pt ^ (uint64_t)j), a.n);
        const int2 r = proc_record<false>(a, s, j, tgt, 0u);
        unsigned long long q;
        if (a.m.fixed) q = (unsigned long long)(r.y < 0 ? -(long long)r.y : (long long)r.y);
        else q = (unsigned long long)ceil(ldexp((double)fabsf(__int_as_float(r.y)), 24));
        atomicAdd(&insum[tgt], q);
    }
}

}  // namespace

hipError_t launch_push_proc(const StepArgs &a, uint32_t i, int64_t t_explicit, hipStream_t s)
{
    const uint32_t nj = a.dbg_spikes ? 1u : a.lists;
    if (a.pr.once) {  // rows generated once: pg1 push blocks, pages of every group
        if (!a.proc || a.direct || a.tl.T > kMaxTiles || a.tl.T != kGroups * a.tl.T8 || nj * a.tl.T > kOnceMaxB ||
            a.tl.W > 8192 || a.pg1 == 0 || a.pslots == 0 || a.page_cap == 0 || a.pr.k_out > kMaxRow)
            return hipErrorInvalidValue;
        if (a.compact ? !a.pages16 : !a.pages) return hipErrorInvalidValue;
        const dim3 grid(a.pg1), block(kProcThreads);
        if (a.compact) {
            if (a.m.fixed) hipLaunchKernelGGL((k_push_proc_once<true, true>), grid, block, 0, s, a, i, t_explicit);
            else hipLaunchKernelGGL((k_push_proc_once<false, true>), grid, block, 0, s, a, i, t_explicit);
        } else {
            if (a.m.fixed) hipLaunchKernelGGL((k_push_proc_once<true, false>), grid, block, 0, s, a, i, t_explicit);
            else hipLaunchKernelGGL((k_push_proc_once<false, false>), grid, block, 0, s, a, i, t_explicit);
        }
        return hipGetLastError();
    }
    if (!a.proc || a.direct || a.tl.T > kMaxTiles || a.tl.T != kGroups * a.tl.T8 || nj * a.tl.T8 > kMaxBuckets ||
        a.tl.W > 8192 || a.pg1 == 0 || a.pslots == 0 || a.page_cap == 0 || a.pr.k_out > kMaxRow)
        return hipErrorInvalidValue;
    if (a.compact ? !a.pages16 : !a.pages) return hipErrorInvalidValue;
    const dim3 grid(kGroups * a.pg1), block(kProcThreads);
    if (a.compact) {
        if (a.m.fixed) hipLaunchKernelGGL((k_push_proc<true, true>), grid, block, 0, s, a, i, t_explicit);
        else hipLaunchKernelGGL((k_push_proc<false, true>), grid, block, 0, s, a, i, t_explicit);
    } else {
        if (a.m.fixed) hipLaunchKernelGGL((k_push_proc<true, false>), grid, block, 0, s, a, i, t_explicit);
        else hipLaunchKernelGGL((k_push_proc<false, false>), grid, block, 0, s, a, i, t_explicit);
    }
    return hipGetLastError();
}

hipError_t export_proc(const StepArgs &a, const ClassTab &tab, const uint32_t *rows, uint64_t n_rows,
                       const uint64_t *out_off, uint32_t *col, uint32_t *wbits, uint8_t *delay, hipStream_t s)
{
    if (!n_rows) return hipSuccess;
    if (n_rows > 0x7fffffffull || !a.proc) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_export_proc, dim3((uint32_t)n_rows), dim3(256), 0, s, a, tab, rows, out_off, col, wbits,
                       delay);
    return hipGetLastError();
}

hipError_t proc_in_abs_sum(const StepArgs &a, uint64_t *insum, hipStream_t s)
{
    if (!a.proc || a.n == 0) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_proc_in_abs_sum, dim3(a.n), dim3(256), 0, s, a, (unsigned long long *)insum);
    return hipGetLastError();
}

}  // namespace spk
