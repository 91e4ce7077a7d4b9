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
// selects the XCD).  Events reach their tile in one of two ways:
//   - direct: the tile reads, for every due spike, the run of that spike's
//     target-sorted row that falls into the tile (per-piece tile offsets);
//     used when rows are long compared with the tile count;
//   - binned: a "bin" kernel reads each due row's run for the XCD's group
//     (per-piece group offsets), counting-sorts it by tile in LDS and appends
//     coalesced runs to per-tile bins that the tile kernel then drains.
// The rows are sorted by target (Sec. III-A), so both runs are contiguous:
// this is the paper's cache-aware transmission, with the locality made
// explicit as LDS tiles instead of left to the cache.
//
// Per-delay adjacency lists (Sec. V): at step t, list j (delay dmin+j)
// delivers the spikes of step t - dmin - j.  Spike lists live in a ring of
// dmax + 2 slots, one list per (slot, XCD group); counts stay on the device.
#include <hip/hip_runtime.h>

#include "spk_internal.h"

namespace spk {

namespace {

constexpr int kBinThreads = 512;
constexpr int kTileThreads = 1024;
constexpr uint32_t kChunk = 4096;              // events staged per binning round
constexpr uint32_t kMaxChunkPieces = 512;      // pieces resolved per binning chunk
constexpr uint32_t kDue = kMaxLists * kGroups; // (list, source group) spike lists

__device__ __forceinline__ uint32_t lane_id() { return threadIdx.x & (kWave - 1); }

__device__ __forceinline__ uint64_t step_index(const StepArgs &a, uint32_t i, int64_t t_explicit)
{
    return t_explicit >= 0 ? (uint64_t)t_explicit : *a.t_base + i;
}

// Block-wide exclusive scan of one u32 per thread (blockDim <= 1024).
__device__ uint32_t block_scan_u32(uint32_t x, uint32_t *ws /*>=16*/, uint32_t *total)
{
    const uint32_t lane = lane_id(), w = threadIdx.x / kWave, nw = blockDim.x / kWave;
    uint32_t inc = x;
    for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t y = __shfl_up(inc, o);
        if (lane >= (uint32_t)o) inc += y;
    }
    if (lane == kWave - 1) ws[w] = inc;
    __syncthreads();
    uint32_t before = 0, tot = 0;
    for (uint32_t k = 0; k < nw; k++) {
        const uint32_t v = ws[k];
        before += k < w ? v : 0u;
        tot += v;
    }
    __syncthreads();
    *total = tot;
    return before + inc - x;
}

__device__ __forceinline__ uint64_t block_sum_u64(uint64_t x, unsigned long long *ws /*>=16*/)
{
    const uint32_t lane = lane_id(), w = threadIdx.x / kWave, nw = blockDim.x / kWave;
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
    if (lane == 0) ws[w] = x;
    __syncthreads();
    uint64_t tot = 0;
    for (uint32_t k = 0; k < nw; k++) tot += ws[k];
    __syncthreads();
    return tot;
}

// The spike lists due at step t: one entry per (delay list, source group).
struct Due {
    uint32_t pre[kDue + 1];   // exclusive prefix of the entry counts
    uint64_t base[kDue];      // offset of the entry's spike list in the ring
    uint32_t list[kDue];      // delay list of the entry
    uint32_t ne;
};

__device__ void build_due(const StepArgs &a, uint64_t t, Due &d, uint32_t *ws)
{
    const uint32_t nl = a.list_hi - a.list_lo;
    const uint32_t ne = nl * kGroups;
    uint32_t c = 0;
    const uint32_t e = threadIdx.x;
    if (e < ne) {
        const uint32_t jj = a.list_lo + e / kGroups, xs = e % kGroups;
        const uint64_t del = (uint64_t)a.dmin + jj;
        uint64_t base = 0;
        if (a.dbg_spikes) {
            c = xs == 0 ? *a.dbg_count : 0u;
        } else if (t >= del) {
            const uint64_t slot = (t - del) % a.ring_slots;
            c = a.ring_count[(slot * kGroups + xs) * kPad];
            if (c > a.tl.Gw) c = a.tl.Gw;
            base = (slot * kGroups + xs) * (uint64_t)a.tl.Gw;
        }
        d.base[e] = base;
        d.list[e] = jj;
    }
    uint32_t tot;
    const uint32_t ex = block_scan_u32(e < ne ? c : 0u, ws, &tot);
    if (e < ne) d.pre[e] = ex;
    if (threadIdx.x == 0) {
        d.pre[ne] = tot;
        d.ne = ne;
    }
    __syncthreads();
}

// piece p of the due set -> (row index j*n + s); p < d.pre[d.ne]
__device__ __forceinline__ uint64_t due_row(const StepArgs &a, const Due &d, uint32_t p)
{
    uint32_t lo = 0, hi = d.ne - 1;  // largest e with pre[e] <= p
    while (lo < hi) {
        const uint32_t mid = (lo + hi + 1) >> 1;
        if (d.pre[mid] <= p) lo = mid; else hi = mid - 1;
    }
    const uint32_t k = p - d.pre[lo];
    const uint32_t s = a.dbg_spikes ? a.dbg_spikes[k] : a.ring[d.base[lo] + k];
    return (uint64_t)d.list[lo] * a.n + s;
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

template <bool FIXED> struct Acc;
template <> struct Acc<true> {
    using T = int32_t;
    static __device__ __forceinline__ void add(T *p, int32_t wbits, int32_t) { atomicAdd(p, wbits); }
};
template <> struct Acc<false> {
    using T = unsigned long long;
    static __device__ __forceinline__ void add(T *p, int32_t wbits, int32_t s64)
    {
        atomicAdd(p, (unsigned long long)to_fixed64(wbits, s64));
    }
};

// Global fallback for bin overflow (rare): same units as the LDS accumulator.
template <bool FIXED>
__device__ __forceinline__ void overflow_add(const StepArgs &a, uint32_t tile, uint32_t local, int32_t wbits)
{
    const uint64_t i = (uint64_t)tile * a.tl.W + local;
    if (FIXED) atomicAdd((int32_t *)a.acc_ovf + i, wbits);
    else atomicAdd((unsigned long long *)a.acc_ovf + i, (unsigned long long)to_fixed64(wbits, a.m.shift64));
    if (a.ovf_flag[tile] == 0) atomicOr(&a.ovf_flag[tile], 1u);
}

// ------------------------------------------------------------- bin kernel

struct BinLDS {
    Due due;
    union {
        int2 stage[kChunk];        // tile-sorted events {tile<<16 | local, weight}
        uint16_t pmap[kChunk];     // piece of every event of the round
    } u;
    uint32_t poff[kMaxChunkPieces + 1];
    uint64_t pbase[kMaxChunkPieces];
    uint32_t tcnt[256], tst[256];
    uint64_t gbase[256];
    uint32_t ws[16];
};

// Block-wide exclusive max-scan of one u32 per thread.
__device__ uint32_t block_scan_max_u32(uint32_t x, uint32_t *ws)
{
    const uint32_t lane = lane_id(), w = threadIdx.x / kWave, nw = blockDim.x / kWave;
    uint32_t inc = x;
    for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t y = __shfl_up(inc, o);
        if (lane >= (uint32_t)o) inc = y > inc ? y : inc;
    }
    const uint32_t ex_w = __shfl_up(inc, 1);
    if (lane == kWave - 1) ws[w] = inc;
    __syncthreads();
    uint32_t before = 0;
    for (uint32_t k = 0; k < w; k++) before = ws[k] > before ? ws[k] : before;
    __syncthreads();
    const uint32_t ex = lane ? (ex_w > before ? ex_w : before) : before;
    (void)nw;
    return ex;
}

template <bool FIXED>
__global__ __launch_bounds__(kBinThreads) void k_bin(StepArgs a, uint32_t i, int64_t t_explicit)
{
    __shared__ BinLDS L;
    const uint64_t t = step_index(a, i, t_explicit);
    const uint32_t x = blockIdx.x % kGroups, g = blockIdx.x / kGroups;
    const uint32_t G1 = gridDim.x / kGroups;
    const uint32_t tid = threadIdx.x;
    const Tiling tl = a.tl;
    build_due(a, t, L.due, L.ws);
    const uint32_t P = L.due.pre[L.due.ne];
    // pieces per chunk: one chunk per block when possible
    uint32_t K = (P + G1 - 1) / G1;
    K = K < 1 ? 1 : (K > a.bin_chunk ? a.bin_chunk : K);
    const uint32_t chunks = (P + K - 1) / K;
    const uint32_t xlo = x * tl.Gw;
    for (uint32_t c = g; c < chunks; c += G1) {
        // 1. this XCD's run of every piece of the chunk
        uint32_t len = 0;
        uint64_t base = 0;
        if (tid < K && c * K + tid < P) {
            const uint64_t row = due_row(a, L.due, c * K + tid);
            const uint64_t pb = a.row_ptr[row];
            const uint32_t plen = (uint32_t)(a.row_ptr[row + 1] - pb);
            const uint32_t gl = a.goff[row * kGroups + x];
            const uint32_t gh = x + 1 < kGroups ? a.goff[row * kGroups + x + 1] : plen;
            len = gh - gl;
            base = pb + gl;
        }
        uint32_t E;
        const uint32_t off = block_scan_u32(len, L.ws, &E);
        if (tid < K) {
            L.poff[tid] = off;
            L.pbase[tid] = base;
        }
        if (tid == 0) L.poff[K] = E;
        __syncthreads();
        // 2. in rounds of kChunk events: map events to pieces, count by tile,
        //    reserve bin space, stage tile-sorted in LDS, write coalesced runs
        for (uint32_t e0 = 0; e0 < E; e0 += kChunk) {
            const uint32_t nsub = E - e0 < kChunk ? E - e0 : kChunk;
            constexpr int R = kChunk / kBinThreads;
            // piece map: mark each piece's first event of the round, then a
            // max-scan spreads the mark over the piece's events
            for (uint32_t q = tid; q < nsub; q += kBinThreads) L.u.pmap[q] = 0;
            for (uint32_t q = tid; q < tl.T8; q += kBinThreads) L.tcnt[q] = 0;
            __syncthreads();
            if (tid < K) {
                const uint32_t ps = L.poff[tid], pe = L.poff[tid + 1];
                const uint32_t st = ps > e0 ? ps : e0;
                if (st < pe && st < e0 + nsub) L.u.pmap[st - e0] = (uint16_t)tid;
            }
            __syncthreads();
            {
                uint32_t v[R], mx = 0;
#pragma unroll
                for (int r = 0; r < R; r++) {
                    const uint32_t q = tid * R + r;
                    v[r] = q < nsub ? L.u.pmap[q] : 0u;
                    mx = v[r] > mx ? v[r] : mx;
                }
                uint32_t run = block_scan_max_u32(mx, L.ws);
#pragma unroll
                for (int r = 0; r < R; r++) {
                    const uint32_t q = tid * R + r;
                    run = v[r] > run ? v[r] : run;
                    if (q < nsub) L.u.pmap[q] = (uint16_t)run;
                }
            }
            __syncthreads();
            int2 rec[R];
            uint32_t tr[R];
            uint64_t idx[R];
#pragma unroll
            for (int r = 0; r < R; r++) {
                const uint32_t f = r * kBinThreads + tid;
                idx[r] = ~0ull;
                if (f < nsub) {
                    const uint32_t k = L.u.pmap[f];
                    idx[r] = L.pbase[k] + (e0 + f - L.poff[k]);
                }
            }
#pragma unroll
            for (int r = 0; r < R; r++)
                if (idx[r] != ~0ull) rec[r] = a.syn[idx[r]];
#pragma unroll
            for (int r = 0; r < R; r++) {
                tr[r] = 0xffffffffu;
                if (idx[r] != ~0ull) {
                    const uint32_t local = (uint32_t)rec[r].x - xlo;
                    const uint32_t tc = local >> tl.logW;
                    const uint32_t rank = atomicAdd(&L.tcnt[tc], 1u);
                    tr[r] = (tc << 16) | rank;
                    rec[r].x = (int)((tc << 16) | (local & (tl.W - 1)));
                }
            }
            __syncthreads();
            {
                uint32_t cnt = tid < tl.T8 ? L.tcnt[tid] : 0u, tot;
                const uint32_t st = block_scan_u32(cnt, L.ws, &tot);
                if (tid < tl.T8) {
                    L.tst[tid] = st;
                    L.gbase[tid] = cnt ? atomicAdd(&a.bin_fill[(x * tl.T8 + tid) * kPad], cnt) : 0u;
                }
            }
            __syncthreads();
#pragma unroll
            for (int r = 0; r < R; r++) {
                if (tr[r] == 0xffffffffu) continue;
                L.u.stage[L.tst[tr[r] >> 16] + (tr[r] & 0xffffu)] = rec[r];
            }
            __syncthreads();
            for (uint32_t q = tid; q < nsub; q += kBinThreads) {
                int2 r2 = L.u.stage[q];
                const uint32_t tc = (uint32_t)r2.x >> 16;
                r2.x &= 0xffff;
                const uint32_t tile = x * tl.T8 + tc;
                const uint64_t pos = L.gbase[tc] + (q - L.tst[tc]);
                if (pos < a.bin_cap) a.bins[(uint64_t)tile * a.bin_cap + pos] = r2;
                else overflow_add<FIXED>(a, tile, (uint32_t)r2.x, r2.y);
            }
            __syncthreads();
        }
    }
}

// ------------------------------------------------------------ tile kernel

template <bool FIXED>
struct TileLDS {
    typename Acc<FIXED>::T acc[kMaxTileW];
    uint16_t spk[kMaxTileW];
    Due due;
    uint32_t wpre[kTileThreads / kWave][kWave + 1];
    uint64_t wbeg[kTileThreads / kWave][kWave];
    uint32_t ws[16];
    unsigned long long ws64[16];
    uint32_t nspk, base;
    uint64_t pois[256];
};

// Accumulate the tile's events directly from the due rows (direct mode):
// each wave takes 64 pieces at a time, lane l resolving piece l's run for
// this tile; the 64 runs are then streamed lane-parallel.
template <bool FIXED>
__device__ uint64_t gather_direct(const StepArgs &a, TileLDS<FIXED> &L, uint32_t tile, uint32_t tile_lo)
{
    const uint32_t lane = lane_id(), w = threadIdx.x / kWave, nw = kTileThreads / kWave;
    const uint32_t P = L.due.pre[L.due.ne];
    const uint32_t T1 = a.tl.T + 1;
    uint64_t mine = 0;
    for (uint32_t p0 = w * kWave; p0 < P; p0 += nw * kWave) {
        uint32_t len = 0;
        uint64_t beg = 0;
        if (p0 + lane < P) {
            const uint64_t row = due_row(a, L.due, p0 + lane);
            const uint16_t *to = a.toff + row * T1 + tile;
            const uint32_t b = to[0], e = to[1];
            beg = a.row_ptr[row] + b;
            len = e - b;
        }
        uint32_t inc = len;
        for (int o = 1; o < kWave; o <<= 1) {
            const uint32_t y = __shfl_up(inc, o);
            if (lane >= (uint32_t)o) inc += y;
        }
        const uint32_t tot = __shfl(inc, kWave - 1);
        L.wpre[w][lane] = inc - len;
        L.wbeg[w][lane] = beg;
        if (lane == 0) L.wpre[w][kWave] = tot;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
        constexpr int U = 4;  // loads in flight per lane
        for (uint32_t f0 = 0; f0 < tot; f0 += kWave * U) {
            uint64_t idx[U];
#pragma unroll
            for (int u = 0; u < U; u++) {
                const uint32_t f = f0 + u * kWave + lane;
                idx[u] = ~0ull;
                if (f < tot) {
                    uint32_t lo = 0, hi = kWave - 1;
                    while (lo < hi) {
                        const uint32_t mid = (lo + hi + 1) >> 1;
                        if (L.wpre[w][mid] <= f) lo = mid; else hi = mid - 1;
                    }
                    idx[u] = L.wbeg[w][lo] + (f - L.wpre[w][lo]);
                }
            }
            int2 r[U];
#pragma unroll
            for (int u = 0; u < U; u++)
                if (idx[u] != ~0ull) r[u] = a.syn[idx[u]];
#pragma unroll
            for (int u = 0; u < U; u++)
                if (idx[u] != ~0ull) Acc<FIXED>::add(&L.acc[(uint32_t)r[u].x - tile_lo], r[u].y, a.m.shift64);
        }
        mine += lane == 0 ? tot : 0u;
        __builtin_amdgcn_wave_barrier();
    }
    return mine;
}

template <bool FIXED>
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

    for (uint32_t q = tid; q < tl.W; q += kTileThreads) L.acc[q] = 0;
    if (m.pois_len && !debug)
        for (uint32_t k = tid; k < m.pois_len; k += kTileThreads) L.pois[k] = a.pois[k];
    if (tid == 0) L.nspk = 0;
    if (a.direct) build_due(a, t, L.due, L.ws);
    __syncthreads();

    // 1. accumulate every event due at t for this tile
    uint64_t delivered = 0;
    if (a.direct) {
        delivered = block_sum_u64(gather_direct<FIXED>(a, L, tile, tile_lo), L.ws64);
    } else {
        const uint32_t filled = a.bin_fill[tile * kPad];
        const uint32_t nb = filled < a.bin_cap ? filled : (uint32_t)a.bin_cap;
        const int2 *bin = a.bins + (uint64_t)tile * a.bin_cap;
        // kDrain independent loads in flight per thread before their atomics
        constexpr int kDrain = 8;
        for (uint32_t q0 = tid; q0 < nb; q0 += kTileThreads * kDrain) {
            int2 r[kDrain];
#pragma unroll
            for (int u = 0; u < kDrain; u++) {
                const uint32_t q = q0 + u * kTileThreads;
                r[u] = q < nb ? bin[q] : make_int2(-1, 0);
            }
#pragma unroll
            for (int u = 0; u < kDrain; u++)
                if (r[u].x >= 0) Acc<FIXED>::add(&L.acc[(uint32_t)r[u].x], r[u].y, m.shift64);
        }
        delivered = filled;
        __syncthreads();
        if (tid == 0) a.bin_fill[tile * kPad] = 0;
        if (a.ovf_flag[tile]) {  // events that did not fit the bin (global fallback)
            for (uint32_t q = tid; q < tile_n; q += kTileThreads) {
                const uint64_t gi = (uint64_t)tile * tl.W + q;
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
            __syncthreads();
            if (tid == 0) a.ovf_flag[tile] = 0;
        }
    }
    __syncthreads();

    if (debug) {  // delivery check: hand the accumulated input back, no update
        for (uint32_t q = tid; q < tile_n; q += kTileThreads) {
            if (FIXED) ((int32_t *)a.dbg_out)[tile_lo + q] = (int32_t)L.acc[q];
            else ((float *)a.dbg_out)[tile_lo + q] = fixed64_to_float(L.acc[q], m.shift64);
        }
        return;
    }

    // 2. neuron update (forward Euler in fp32, every operation rounded on its
    //    own), spikes collected in LDS
    const uint32_t slot = (uint32_t)(t % a.ring_slots);
    uint64_t ev = 0;
    constexpr int kRounds = kMaxTileW / kTileThreads;  // neurons per thread
    for (uint32_t q00 = 0; q00 < tile_n; q00 += kTileThreads * kRounds) {
    // all state loads of this thread's neurons are issued before any update
    float Vr[kRounds];
    uint32_t Rr[kRounds];
#pragma unroll
    for (int u = 0; u < kRounds; u++) {
        const uint32_t q = q00 + u * kTileThreads + tid;
        Vr[u] = 0.0f;
        Rr[u] = 0;
        if (q < tile_n) {
            Vr[u] = a.V[tile_lo + q];
            if (m.kind != SPK_SOURCE) Rr[u] = a.ref[tile_lo + q];
        }
    }
#pragma unroll
    for (int u = 0; u < kRounds; u++) {
        const uint32_t q = q00 + u * kTileThreads + tid;
        bool spk = false;
        if (q < tile_n) {
            const uint32_t gi = tile_lo + q;
            uint32_t K = 0;
            if (m.pois_len) {  // K = min { k : hi32 < T_k }
                const uint64_t h = hash_hi32(step_hash(m.keys.pois, gi, t));
                uint32_t lo = 0, hi = m.pois_len - 1;
                while (lo < hi) {
                    const uint32_t mid = (lo + hi) >> 1;
                    if (h < L.pois[mid]) hi = mid; else lo = mid + 1;
                }
                K = lo;
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
            if (spk) ev += a.outdeg[gi];
        }
        const uint64_t mask = __ballot(spk);
        if (mask) {  // wavefront-ballot compaction into the tile's LDS list
            const int leader = __ffsll((unsigned long long)mask) - 1;
            uint32_t wb = 0;
            if ((int)lane == leader) wb = atomicAdd(&L.nspk, (uint32_t)__popcll(mask));
            wb = __shfl(wb, leader);
            if (spk) {
                const uint32_t rank = __builtin_amdgcn_mbcnt_hi(
                    (uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
                L.spk[wb + rank] = (uint16_t)q;
            }
        }
    }
    }
    ev = block_sum_u64(ev, L.ws64);

    // 3. publish: one reservation per tile in the XCD group's spike list
    if (tid == 0) {
        const uint32_t ns = L.nspk;
        uint32_t base = 0;
        if (ns) {
            base = atomicAdd(&a.ring_count[((uint64_t)slot * kGroups + x) * kPad], ns);
            atomicAdd(&a.counts8[t * kGroups + x], ns);
            atomicAdd((unsigned long long *)&a.events8[t * kGroups + x], (unsigned long long)ev);
        }
        if (delivered)
            atomicAdd((unsigned long long *)&a.delivered8[t * kGroups + x], (unsigned long long)delivered);
        L.base = base;
    }
    if (blockIdx.x == 0 && tid < kGroups)  // next step's lists start empty
        a.ring_count[(((t + 1) % a.ring_slots) * kGroups + tid) * kPad] = 0;
    __syncthreads();
    const uint32_t ns = L.nspk, base = L.base;
    uint32_t *dst = a.ring + ((uint64_t)slot * kGroups + x) * tl.Gw;
    for (uint32_t q = tid; q < ns; q += kTileThreads) {
        if (base + q < tl.Gw) dst[base + q] = tile_lo + L.spk[q];
        else atomicOr(a.flags, 1u);
    }
}

// ---------------------------------------------------------------- record

__global__ __launch_bounds__(256) void k_record(StepArgs a, uint32_t i, int64_t t_explicit)
{
    const uint64_t t = step_index(a, i, t_explicit);
    const uint64_t slot = t % a.ring_slots;
    uint64_t base = a.raster_offs[t];
    bool ok = true;
    for (uint32_t xs = 0; xs < kGroups; xs++) {
        uint32_t c = a.ring_count[(slot * kGroups + xs) * kPad];
        if (c > a.tl.Gw) c = a.tl.Gw;
        if (base + c > a.raster_cap) {
            ok = false;
            break;
        }
        const uint32_t *src = a.ring + (slot * kGroups + xs) * a.tl.Gw;
        for (uint32_t k = threadIdx.x; k < c; k += blockDim.x) a.raster[base + k] = src[k];
        base += c;
    }
    if (threadIdx.x == 0) {
        a.raster_offs[t + 1] = ok ? base : a.raster_offs[t];
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

}  // namespace

uint32_t bin_grid() { return (uint32_t)(kGroups * ((3 * cu_count() + kGroups - 1) / kGroups)); }

hipError_t launch_bin(const StepArgs &a, uint32_t i, int64_t t_explicit, hipStream_t s)
{
    if (a.tl.T8 > 256 || a.bin_chunk == 0 || a.bin_chunk > kMaxChunkPieces ||
        a.list_hi <= a.list_lo || a.list_hi - a.list_lo > kMaxLists || a.tl.W > 65536)
        return hipErrorInvalidValue;
    if (a.m.fixed)
        hipLaunchKernelGGL(k_bin<true>, dim3(bin_grid()), dim3(kBinThreads), 0, s, a, i, t_explicit);
    else
        hipLaunchKernelGGL(k_bin<false>, dim3(bin_grid()), dim3(kBinThreads), 0, s, a, i, t_explicit);
    return hipGetLastError();
}

hipError_t launch_tile(const StepArgs &a, uint32_t i, int64_t t_explicit, hipStream_t s)
{
    if (a.tl.W > kMaxTileW || a.m.pois_len > 256 || a.list_hi <= a.list_lo ||
        a.list_hi - a.list_lo > kMaxLists || a.tl.T != kGroups * a.tl.T8)
        return hipErrorInvalidValue;
    if (a.m.fixed)
        hipLaunchKernelGGL(k_tile<true>, dim3(a.tl.T), dim3(kTileThreads), 0, s, a, i, t_explicit);
    else
        hipLaunchKernelGGL(k_tile<false>, dim3(a.tl.T), dim3(kTileThreads), 0, s, a, i, t_explicit);
    return hipGetLastError();
}

hipError_t launch_record(const StepArgs &a, uint32_t i, int64_t t_explicit, hipStream_t s)
{
    hipLaunchKernelGGL(k_record, dim3(1), dim3(256), 0, s, a, i, t_explicit);
    return hipGetLastError();
}

hipError_t launch_advance(uint64_t *t_base, uint32_t steps, hipStream_t s)
{
    hipLaunchKernelGGL(k_advance, dim3(1), dim3(64), 0, s, t_base, steps);
    return hipGetLastError();
}

hipError_t stream_copy(const void *src, void *dst, uint64_t bytes, hipStream_t s)
{
    hipLaunchKernelGGL(k_stream_copy, dim3(cu_count() * 16), dim3(256), 0, s, (const uint4 *)src,
                       (uint4 *)dst, bytes / 16);
    return hipGetLastError();
}

}  // namespace spk
