// spk_dev.h -- device helpers shared by the step kernels (spk_step.hip) and
// the persistent step kernel (spk_run.hip): workgroup barriers and scans,
// spike-list and page addressing, accumulator units, synapse records.
#pragma once

#include <hip/hip_runtime.h>

#include "spk_internal.h"

namespace spk {
namespace {


// Loads and stores at agent scope (the sc1 cache policy): they do not hit in
// the non-coherent per-XCD caches, so data written this way by one workgroup
// is seen by a workgroup on another XCD once the writer's store has completed
// (vmcnt) and the reader has observed that through an atomic.  Used by the
// persistent kernel for the spike lists, which every XCD reads.
__device__ __forceinline__ uint32_t ld_ag(const uint32_t *p)
{
    return __hip_atomic_load(const_cast<uint32_t *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_ag(uint32_t *p, uint32_t v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <bool COH>
__device__ __forceinline__ uint32_t ld_u32(const uint32_t *p)
{
    if constexpr (COH) return ld_ag(p);
    else return *p;
}

__device__ __forceinline__ uint32_t lane_id() { return threadIdx.x & (kWave - 1); }

// Workgroup barrier that orders LDS traffic only.  __syncthreads() carries
// workgroup-scope fences on global memory as well, which can make a wave
// wait for its outstanding global loads (one full memory round trip per
// phase); here global loads issued before the barrier stay in flight across
// it.  Used wherever threads of a block communicate through LDS alone.
// Neither barrier waits for global stores to complete: code that hands
// global data to other workgroups waits for them explicitly (s_waitcnt).
__device__ __forceinline__ void lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ void lds_wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ uint64_t step_index(const StepArgs &a, uint32_t i, int64_t t_explicit)
{
    return t_explicit >= 0 ? (uint64_t)t_explicit : *a.t_base + i;
}

// Inclusive prefix sum of one u32 per lane over a whole wave (every lane
// active): DPP row shifts by 1, 2, 4 and 8 lanes scan each row of 16 lanes
// (a lane with no source adds 0), then each row adds the totals of the rows
// before it, read from lanes 15, 31 and 47.  No LDS traffic, unlike a
// shuffle (ds_bpermute) per step.
__device__ __forceinline__ uint32_t wave_scan_incl_u32(uint32_t x)
{
    int v = (int)x;
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, true);  // row_shr:1
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, true);  // row_shr:2
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, true);  // row_shr:4
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, true);  // row_shr:8
    const uint32_t t0 = (uint32_t)__builtin_amdgcn_readlane(v, 15), t1 = (uint32_t)__builtin_amdgcn_readlane(v, 31),
                   t2 = (uint32_t)__builtin_amdgcn_readlane(v, 47);
    const uint32_t row = lane_id() >> 4;
    const uint32_t before = (row >= 1 ? t0 : 0u) + (row >= 2 ? t1 : 0u) + (row >= 3 ? t2 : 0u);
    return (uint32_t)v + before;
}

// Every kernel that uses the block-wide helpers below runs workgroups of
// kBlockThreads threads (a constant, so that the per-wave partials are read
// with all loads at once instead of a loop bounded by blockDim).
constexpr uint32_t kBlockThreads = 1024;
constexpr uint32_t kBlockWaves = kBlockThreads / kWave;

// The per-wave partials ws[0 .. kBlockWaves) of a block-wide scan: their sum
// before wave w and their total.  kBlockWaves is one DPP row: every row of
// 16 lanes reads the 16 partials (one LDS read per lane) and scans them.
static_assert(kBlockWaves == 16, "one partial per lane of a DPP row");
__device__ __forceinline__ void wave_partials(const uint32_t *ws, uint32_t w, uint32_t *before, uint32_t *tot)
{
    int v = (int)ws[lane_id() & (kBlockWaves - 1)];
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, true);  // row_shr:1
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, true);  // row_shr:2
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, true);  // row_shr:4
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, true);  // row_shr:8
    *tot = (uint32_t)__builtin_amdgcn_readlane(v, kBlockWaves - 1);
    *before = w ? (uint32_t)__builtin_amdgcn_readlane(v, (int)w - 1) : 0u;
}

// Block-wide exclusive scan of one u32 per thread.
__device__ uint32_t block_scan_u32(uint32_t x, uint32_t *ws /*>=16*/, uint32_t *total)
{
    const uint32_t lane = lane_id(), w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const uint32_t inc = wave_scan_incl_u32(x);
    if (lane == kWave - 1) ws[w] = inc;
    lds_sync();
    uint32_t before, tot;
    wave_partials(ws, w, &before, &tot);
    lds_sync();
    *total = tot;
    return before + inc - x;
}

// Same, without the trailing barrier: ws must not be written again before
// the caller's next barrier.
__device__ uint32_t block_scan_u32_open(uint32_t x, uint32_t *ws /*>=16*/, uint32_t *total)
{
    const uint32_t lane = lane_id(), w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const uint32_t inc = wave_scan_incl_u32(x);
    if (lane == kWave - 1) ws[w] = inc;
    lds_sync();
    uint32_t before, tot;
    wave_partials(ws, w, &before, &tot);
    *total = tot;
    return before + inc - x;
}

// One step of a 64-bit row scan: x plus the value of the lane C & 0xf below
// in its row of 16 (0 where there is none), both halves moved by DPP.
template <int C>
__device__ __forceinline__ uint64_t dpp_shr_add_u64(uint64_t x)
{
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)x, C, 0xf, 0xf, true);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(x >> 32), C, 0xf, 0xf, true);
    return x + (((uint64_t)hi << 32) | lo);
}

// Sum of one u64 per lane over a whole wave (every lane active), the same in
// every lane: each row of 16 lanes is scanned with DPP row shifts, and the
// four row sums are read from lanes 15, 31, 47 and 63.
__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t x)
{
    x = dpp_shr_add_u64<0x111>(x);  // row_shr:1
    x = dpp_shr_add_u64<0x112>(x);  // row_shr:2
    x = dpp_shr_add_u64<0x114>(x);  // row_shr:4
    x = dpp_shr_add_u64<0x118>(x);  // row_shr:8
    const int lo = (int)(uint32_t)x, hi = (int)(uint32_t)(x >> 32);
    uint64_t tot = 0;
#pragma unroll
    for (int r = 0; r < kWave / 16; r++)
        tot += ((uint64_t)(uint32_t)__builtin_amdgcn_readlane(hi, 16 * r + 15) << 32) |
               (uint32_t)__builtin_amdgcn_readlane(lo, 16 * r + 15);
    return tot;
}

__device__ __forceinline__ uint64_t block_sum_u64(uint64_t x, unsigned long long *ws /*>=16*/)
{
    const uint32_t lane = lane_id(), w = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    x = wave_sum_u64(x);
    if (lane == 0) ws[w] = x;
    lds_sync();
    // each row of 16 lanes sums the 16 partials (one LDS read per lane)
    uint64_t v = ws[lane & (kBlockWaves - 1)];
    v = dpp_shr_add_u64<0x111>(v);
    v = dpp_shr_add_u64<0x112>(v);
    v = dpp_shr_add_u64<0x114>(v);
    v = dpp_shr_add_u64<0x118>(v);
    const uint64_t tot = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), 15) << 32) |
                         (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, 15);
    lds_sync();
    return tot;
}

// The spike list of one slot is spread over per-tile segments: pre[] gets
// the exclusive prefix of the T segment counts (T <= 2048, two per thread of
// a 1024-thread block); returns the total.  COH: agent-scope loads.
template <bool COH = false>
__device__ uint32_t load_spike_set(const StepArgs &a, uint32_t slot, uint32_t *pre, uint32_t *ws)
{
    const uint32_t T = a.tl.T, W = a.tl.W;
    const uint32_t b = threadIdx.x * 2;
    const uint32_t *cnt = a.spk_cnt + (uint64_t)slot * T;
    uint32_t c0 = ld_u32<COH>(cnt + (b < T ? b : 0)), c1 = ld_u32<COH>(cnt + (b + 1 < T ? b + 1 : 0));
    c0 = b < T ? (c0 < W ? c0 : W) : 0u;
    c1 = b + 1 < T ? (c1 < W ? c1 : W) : 0u;
    uint32_t tot;
    const uint32_t ex = block_scan_u32(c0 + c1, ws, &tot);
    if (b < T) pre[b] = ex;
    if (b + 1 < T) pre[b + 1] = ex + c0;
    if (threadIdx.x == 0) pre[T] = tot;
    lds_sync();
    return tot;
}

// k-th spike of the slot (k < total): largest tile with pre[tile] <= k.
template <bool COH = false>
__device__ __forceinline__ uint32_t spike_at(const StepArgs &a, const uint32_t *pre, uint32_t slot,
                                             uint32_t k)
{
    uint32_t lo = 0, hi = a.tl.T - 1;
    while (lo < hi) {
        const uint32_t mid = (lo + hi + 1) >> 1;
        if (pre[mid] <= k) lo = mid; else hi = mid - 1;
    }
    return ld_u32<COH>(a.spk_ids + ((uint64_t)slot * a.tl.T + lo) * a.tl.W + (k - pre[lo]));
}

// x / T8 for x * T8 < 2^32: the high half of x * ceil(2^32 / T8) (exact:
// the rounding of the reciprocal adds less than x / 2^32 < 1 / T8).
__device__ __forceinline__ uint32_t div_t8(const Tiling &tl, uint32_t x)
{
    return tl.T8 == 1 ? x : __umulhi(x, tl.T8inv);
}

// Page (x, g1, slot, c) of the binned delivery; records at page * page_cap.
__device__ __forceinline__ uint32_t page_of(const StepArgs &a, uint32_t x, uint32_t g1, uint32_t slot,
                                            uint32_t c)
{
    return ((x * a.pg1 + g1) * a.pslots + slot) * a.tl.T8 + c;
}

__device__ __forceinline__ uint32_t arrival_slot(const StepArgs &a, uint64_t t, uint32_t j, bool dbg)
{
    return dbg ? 0u : (uint32_t)((t + a.dmin + j) % a.pslots);
}

// The same from base = arrival_slot(a, t, 0, dbg), without a 64-bit
// remainder per use (j < lists <= pslots: one wrap at most).
__device__ __forceinline__ uint32_t arrival_slot_from(const StepArgs &a, uint32_t base, uint32_t j, bool dbg)
{
    const uint32_t sl = base + j;
    return dbg ? 0u : (sl < a.pslots ? sl : sl - a.pslots);
}

// [M r / G, M (r + 1) / G) in 32-bit arithmetic (M = mq G + mr): the r-th of
// G equal shares of M items.
__device__ __forceinline__ void equal_share(uint32_t M, uint32_t r, uint32_t G, uint32_t *k0, uint32_t *k1)
{
    const uint32_t mq = M / G, mr = M - mq * G;
    *k0 = mq * r + mr * r / G;
    *k1 = mq * (r + 1) + mr * (r + 1) / G;
}

// Accumulator conversions.  fp32 mode: exact int64 multiple of 2^-S64.
__device__ __forceinline__ long long to_fixed64(int32_t wbits, int32_t s64)
{
    return __double2ll_rn(ldexp((double)__int_as_float(wbits), s64));
}
// The unit is chosen so that |acc| < 2^53: the conversion to double is
// exact, the scaling by 2^-S64 is exact, and the one rounding is to fp32.
__device__ __forceinline__ float fixed64_to_float(unsigned long long acc, int32_t s64)
{
    return (float)ldexp((double)(long long)acc, -s64);
}

// Accumulator units of one event: the stored weight bits converted
// (full format), or the class's precomputed value (compact format).
template <bool FIXED>
__device__ __forceinline__ long long units_of(int32_t wbits, int32_t s64)
{
    return FIXED ? (long long)wbits : to_fixed64(wbits, s64);
}
// Selected without a dynamic index into the kernel arguments (which would
// go through scratch memory).
__device__ __forceinline__ long long class_units(const StepArgs &a, uint32_t cls)
{
    const long long w01 = cls & 1u ? a.wval[1] : a.wval[0];
    const long long w23 = cls & 1u ? a.wval[3] : a.wval[2];
    return cls & 2u ? w23 : w01;
}

template <bool FIXED> struct Acc;
template <> struct Acc<true> {
    using T = int32_t;
    static __device__ __forceinline__ void add(T *p, long long units) { atomicAdd(p, (int32_t)units); }
};
template <> struct Acc<false> {
    using T = unsigned long long;
    static __device__ __forceinline__ void add(T *p, long long units)
    {
        atomicAdd(p, (unsigned long long)units);
    }
};

// Synapse record of each format, and its key (class, delay index, target).
template <bool CMP> struct SynRec;
template <> struct SynRec<false> {
    using T = int2;
    static __device__ __forceinline__ T load(const StepArgs &a, uint64_t e) { return a.syn[e]; }
};
template <> struct SynRec<true> {
    using T = uint32_t;
    static __device__ __forceinline__ T load(const StepArgs &a, uint64_t e) { return a.syn32[e]; }
};
// Global fallback for a full page (rare): same units as the LDS accumulator,
// one accumulator per (arrival slot, neuron).
// COH: the flag is read with an agent-scope load (persistent kernel, where
// the tile resets it during the launch).
template <bool FIXED, bool COH = false>
__device__ __forceinline__ void overflow_add(const StepArgs &a, uint32_t slot, uint32_t tile,
                                             uint32_t local, long long units)
{
    const uint64_t st = (uint64_t)slot * a.tl.T + tile;
    const uint64_t i = st * a.tl.W + local;
    if (FIXED) atomicAdd((int32_t *)a.acc_ovf + i, (int32_t)units);
    else atomicAdd((unsigned long long *)a.acc_ovf + i, (unsigned long long)units);
    if (ld_u32<COH>(&a.ovf_flag[st]) == 0) atomicOr(&a.ovf_flag[st], 1u);
}

// Accumulate the tile's events directly from the rows of the given spikes
// (direct mode): each wave takes 64 spikes at a time, lane l resolving spike
// l's run for this tile; the 64 runs are then streamed lane-parallel.  With
// jf >= 0 only synapses of delay index jf are delivered.  Returns the number
// of events this thread delivered.
//   acc: the tile's LDS accumulators; pre: the spike-count prefix of the slot
//   (load_spike_set); wpre, wbeg: per-wave scratch; wtab: the accumulator
//   units of each weight class (compact records) in LDS.  COH: spike IDs are
//   read with agent-scope loads (persistent kernel).
template <bool FIXED, bool CMP, bool COH>
__device__ uint32_t gather_direct(const StepArgs &a, typename Acc<FIXED>::T *acc, const uint32_t *pre,
                                  uint32_t (*wpre)[kWave + 1], uint64_t (*wbeg)[kWave], uint32_t tile,
                                  uint32_t tile_lo, uint32_t P, uint32_t slot, int32_t jf, const long long *wtab)
{
    using Rec = typename SynRec<CMP>::T;
    // (the wave count as a constant in the persistent kernel; the graph
    // path's tile kernel, which holds both deliveries, compiles to faster
    // code with it read from blockDim: measured on both)
    const uint32_t lane = lane_id(), w = threadIdx.x / kWave, nw = COH ? kBlockWaves : blockDim.x / kWave;
    const uint32_t T1 = a.tl.T + 1;
    uint32_t mine = 0;
    // spikes per wave and round: all waves share the spikes (few spikes with
    // long runs: fewer per wave, so that every wave streams records)
    uint32_t G = (P + nw - 1) / nw;
    G = G < 1u ? 1u : (G > (uint32_t)kWave ? (uint32_t)kWave : G);
    for (uint32_t p0 = w * G; p0 < P; p0 += nw * G) {
        uint32_t len = 0;
        uint64_t beg = 0;
        if (lane < G && p0 + lane < P) {
            uint32_t s = a.dbg_spikes ? a.dbg_spikes[p0 + lane] : spike_at<COH>(a, pre, slot, p0 + lane);
            // a caller's spike list (debug delivery) is checked here: an ID
            // out of range delivers nothing and raises a flag
            const bool bad = s >= a.n;
            if (bad && tile == 0) atomicOr(a.flags, kFlagBadSpike);
            s = bad ? 0u : s;
            const uint16_t *to = a.toff + (uint64_t)s * T1 + tile;
            const uint32_t b = to[0], e = to[1];
            beg = a.row_ptr[s] + b;
            len = bad ? 0u : e - b;
        }
        const uint32_t inc = wave_scan_incl_u32(len);
        const uint32_t tot = (uint32_t)__builtin_amdgcn_readlane((int)inc, kWave - 1);
        wpre[w][lane] = inc - len;
        wbeg[w][lane] = beg;
        if (lane == 0) wpre[w][kWave] = tot;
        lds_wave_sync();
        constexpr int U = 8;  // loads in flight per lane
        for (uint32_t f0 = 0; f0 < tot; f0 += kWave * U) {
            uint64_t idx[U];
#pragma unroll
            for (int u = 0; u < U; u++) {
                const uint32_t f = f0 + u * kWave + lane;
                const uint32_t fc = f < tot ? f : 0u;
                uint32_t lo = 0, hi = kWave - 1;
                while (lo < hi) {
                    const uint32_t mid = (lo + hi + 1) >> 1;
                    if (wpre[w][mid] <= fc) lo = mid; else hi = mid - 1;
                }
                idx[u] = f < tot ? wbeg[w][lo] + (fc - wpre[w][lo]) : 0ull;
            }
            Rec r[U];
#pragma unroll
            for (int u = 0; u < U; u++) r[u] = SynRec<CMP>::load(a, idx[u]);  // unconditional, see push
#pragma unroll
            for (int u = 0; u < U; u++) {
                if (f0 + u * kWave + lane >= tot) continue;
                const uint32_t key = rec_key(r[u]);
                if (jf >= 0 && (int32_t)rec_delay(key) != jf) continue;
                long long units;
                if constexpr (CMP) units = wtab[rec_class(key)];
                else units = units_of<FIXED>(r[u].y, a.m.shift64);
                Acc<FIXED>::add(&acc[rec_target(key) - tile_lo], units);
                mine++;
            }
        }
        __builtin_amdgcn_wave_barrier();
    }
    return mine;
}

}  // namespace
}  // namespace spk
