// spk_gen.hip -- connectivity expansion on the GPU (paper Sec. III-B: the
// network description is expanded on the device, not uploaded synapse by
// synapse) for gfx950 (MI355X, wave64).
//
// Layout produced: one row per source neuron at [row_ptr[s], row_ptr[s+1]),
// synapse = int2 {j << 24 | target, weight bits} (full format) or u32
// {class << 30 | j << 24 | target} (compact format: at most four distinct
// weights, looked up by class), j = delay - delay_min.
// Every row is grouped by target range (the paper keeps rows sorted by target,
// Sec. III-A, so that each target range of a row is one contiguous run; only
// the grouping matters for delivery, the order inside a range does not).
// Direct delivery groups by target tile and writes per-tile starts.  Binned
// delivery groups by XCD group and, inside each group's run, puts the
// synapses of the smallest delay first; it writes per-group ends and the end
// of each group's smallest-delay part (the events that arrive soonest).
//
// Build with -ffp-contract=off: weights are computed with explicitly rounded
// fp32 operations.
#include <hip/hip_runtime.h>

#include <cstdlib>
#include <cstring>

#include "spk_internal.h"

namespace spk {

namespace {

constexpr int kBlock = 256;

__device__ __forceinline__ float u24(uint64_t h)
{
    return (float)(uint32_t)(h >> 40) * (1.0f / 16777216.0f);
}

__device__ __forceinline__ float syn_weight(const ConnArgs &c, uint32_t src, uint64_t hw)
{
    if (c.w_uniform) {
        float span = __fsub_rn(c.w_hi, c.w_lo);
        return __fadd_rn(c.w_lo, __fmul_rn(span, u24(hw)));
    }
    return src < c.n_exc ? c.w_exc : c.w_inh;
}

// stored weight bits: fp32, or round(w * 2^S) as int32 in fixed mode
__device__ __forceinline__ int32_t weight_bits(const ConnArgs &c, float w)
{
    if (c.fixed) return (int32_t)__builtin_rintf(__fmul_rn(w, c.qscale));
    return __float_as_int(w);
}

__device__ __forceinline__ int2 make_syn(uint32_t j, uint32_t tgt, int32_t wbits)
{
    return make_int2((int)((j << kTargetBits) | tgt), wbits);
}

// Synapse e of a row, in the format of the network.  Compact classes:
// generated rows have one weight per source population (class 0 excitatory,
// 1 inhibitory); explicit rows name their weight's class in cls_w.
__device__ __forceinline__ void put_syn(const ConnArgs &c, void *syn, uint64_t e, uint32_t j, uint32_t tgt,
                                        uint32_t src, float w)
{
    if (c.compact) {
        uint32_t cls = src < c.n_exc ? 0u : 1u;
        if (c.kind == SPK_CONN_EXPLICIT) {
            cls = 0;
            for (uint32_t k = 1; k < kMaxClasses; k++)
                if (c.cls_w[k] == __float_as_uint(w)) cls = k;
        }
        ((uint32_t *)syn)[e] = (cls << kClassShift) | (j << kTargetBits) | tgt;
    } else {
        ((int2 *)syn)[e] = make_syn(j, tgt, weight_bits(c, w));
    }
}

__device__ __forceinline__ uint32_t lane_id() { return threadIdx.x & (kWave - 1); }

// Block-wide exclusive scan of one u32 per thread (kBlock threads).
__device__ uint32_t block_scan_u32(uint32_t x, uint32_t *ws, uint32_t *total)
{
    const uint32_t lane = lane_id(), w = threadIdx.x / kWave;
    uint32_t inc = x;
    for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t y = __shfl_up(inc, o);
        if (lane >= (uint32_t)o) inc += y;
    }
    if (lane == kWave - 1) ws[w] = inc;
    __syncthreads();
    uint32_t before = 0, tot = 0;
    for (uint32_t k = 0; k < kBlock / kWave; k++) {
        before += k < w ? ws[k] : 0u;
        tot += ws[k];
    }
    __syncthreads();
    *total = tot;
    return before + inc - x;
}

// ------------------------------------------------------------ bucketing
// Per-row counting sort in LDS: histogram, exclusive scan (the bucket
// starts), then every synapse goes to start[bucket] + its rank.  Buckets:
// target tiles (direct delivery) or (XCD group, smallest delay or not)
// (binned delivery).

struct RowLDS {
    uint32_t cur[kMaxTiles];
    uint32_t ws[kBlock / kWave];
};

__device__ __forceinline__ void zero_tiles(RowLDS &L, uint32_t T)
{
    for (uint32_t k = threadIdx.x; k < T; k += kBlock) L.cur[k] = 0;
    __syncthreads();
}

// histogram -> exclusive starts, in place
__device__ void scan_tiles(RowLDS &L, uint32_t T)
{
    __syncthreads();
    const uint32_t P = (T + kBlock - 1) / kBlock;
    const uint32_t b = threadIdx.x * P;
    uint32_t sum = 0;
    for (uint32_t k = 0; k < P; k++)
        if (b + k < T) sum += L.cur[b + k];
    uint32_t tot;
    uint32_t ex = block_scan_u32(sum, L.ws, &tot);
    for (uint32_t k = 0; k < P; k++) {
        if (b + k < T) {
            const uint32_t v = L.cur[b + k];
            L.cur[b + k] = ex;
            ex += v;
        }
    }
    __syncthreads();
}

// Range boundaries of row s from the bucket starts in L.cur (before placement).
__device__ void write_row_index(const ConnArgs &c, const RowIndex &ix, RowLDS &L, uint32_t s,
                                uint64_t start, uint32_t len)
{
    const Tiling &tl = c.tl;
    if (ix.toff) {
        uint16_t *to = ix.toff + (uint64_t)s * (tl.T + 1);
        for (uint32_t k = threadIdx.x; k <= tl.T; k += kBlock)
            to[k] = (uint16_t)(k < tl.T ? L.cur[k] : len);
    }
    if (ix.desc && threadIdx.x == 0) {
        RowDesc d{};
        d.start = start;
        for (uint32_t x = 0; x < kGroups; x++) {
            d.gend[x] = (uint16_t)(x + 1 < kGroups ? L.cur[2 * (x + 1)] : len);
            d.dend[x] = (uint16_t)L.cur[2 * x + 1];
        }
        ix.desc[s] = d;
    }
    __syncthreads();
}

// Bucket of a synapse (target tgt, delay index j) in its row.
__device__ __forceinline__ uint32_t bucket_of(const ConnArgs &c, const RowIndex &ix, uint32_t tgt, uint32_t j)
{
    const uint32_t tile = tgt >> c.tl.logW;
    if (ix.desc) return 2 * (tile / c.tl.T8) + (j != 0 ? 1u : 0u);
    return tile;
}
__device__ __forceinline__ uint32_t n_buckets(const ConnArgs &c, const RowIndex &ix)
{
    return ix.desc ? 2 * kGroups : c.tl.T;
}

// ----------------------------------------------- rows drawn per source
// Bernoulli rows (one hash per ordered pair) and fixed out-degree rows
// (k_out uniform targets with replacement): one block per source.

// With hist (Bernoulli rows), the pass also keeps each row's bucket counts
// for the placement pass, which then need not count the row again:
// hist[s * (T + 2 * kGroups) ...] = the row's synapses per target tile
// (direct delivery's buckets), then per (XCD group, smallest delay or not)
// (binned delivery's), as u16 (a row longer than kMaxRow is refused before
// placement).  With keys as well, it keeps the first cap synapses of the row
// as keys (j << 24 | target) at keys[s * cap ...], in no particular order:
// where no row is longer than cap, the placement pass reads them instead of
// drawing the row again.
__global__ __launch_bounds__(kBlock) void k_gen_count_rows(ConnArgs c, uint32_t *cnt, uint16_t *hist,
                                                          uint32_t *keys, uint32_t cap)
{
    __shared__ uint32_t tot;
    __shared__ uint32_t hb[kMaxTiles + 2 * kGroups];  // per tile, then per (group, delay class)
    __shared__ uint32_t hj[kMaxTiles];                  // per tile, smallest delay only (several delays)
    const uint32_t s = blockIdx.x;
    if (c.kind != SPK_CONN_BERNOULLI) {
        if (threadIdx.x == 0) cnt[s] = c.k_out;
        return;
    }
    const uint32_t T = c.tl.T, HB = T + 2 * kGroups;
    if (threadIdx.x == 0) tot = 0;
    if (hist)
        for (uint32_t k = threadIdx.x; k < HB; k += kBlock) {
            hb[k] = 0;
            if (k < T) hj[k] = 0;
        }
    __syncthreads();
    const uint64_t rk = mix64(c.keys.conn ^ (uint64_t)s);
    const uint64_t rd = mix64(c.keys.delay ^ (uint64_t)s);
    const uint32_t lane = lane_id();
    uint32_t mine = 0;
    for (uint32_t t0 = 0; t0 < c.n; t0 += kBlock) {  // (uniform trip count: ballots below)
        const uint32_t tgt = t0 + threadIdx.x;
        const bool hit = tgt < c.n && (uint64_t)hash_hi32(mix64(rk ^ (uint64_t)tgt)) < c.conn_thr;
        uint32_t j = 0;
        if (hist && hit) {  // (per-tile counters: few conflicts; the 16 group buckets follow from them)
            const uint32_t tile = tgt >> c.tl.logW;
            atomicAdd(&hb[tile], 1u);
            j = c.lists > 1 ? hash_range(mix64(rd ^ (uint64_t)tgt), c.lists) : 0u;
            if (c.lists > 1 && j == 0) atomicAdd(&hj[tile], 1u);
        }
        if (keys) {  // one position counter update per wave
            const uint64_t bal = __ballot(hit);
            uint32_t base = 0;
            if (lane == 0 && bal) base = atomicAdd(&tot, (uint32_t)__popcll(bal));
            base = __shfl(base, 0);
            const uint32_t pos =
                base + __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
            if (hit && pos < cap) keys[(uint64_t)s * cap + pos] = (j << kTargetBits) | tgt;
        } else {
            mine += hit ? 1u : 0u;
        }
    }
    for (int o = 32; o > 0; o >>= 1) mine += __shfl_xor(mine, o);
    if (lane == 0 && mine) atomicAdd(&tot, mine);
    __syncthreads();
    if (threadIdx.x == 0) cnt[s] = tot;
    if (hist && threadIdx.x < kGroups) {  // group g: smallest delay, then the others
        uint32_t all = 0, j0 = 0;
        for (uint32_t k = threadIdx.x * c.tl.T8; k < (threadIdx.x + 1) * c.tl.T8; k++) {
            all += hb[k];
            j0 += c.lists > 1 ? hj[k] : hb[k];
        }
        hb[T + 2 * threadIdx.x] = j0;
        hb[T + 2 * threadIdx.x + 1] = all - j0;
    }
    __syncthreads();
    if (hist)
        for (uint32_t k = threadIdx.x; k < HB; k += kBlock)
            hist[(uint64_t)s * HB + k] = (uint16_t)(hb[k] < 65535u ? hb[k] : 65535u);
}

// Draw the row twice: once to count per bucket (unless the count pass kept
// the counts in hist), once to place (unless it kept the row's keys).
__global__ __launch_bounds__(kBlock) void k_gen_fill_rows(ConnArgs c, const uint64_t *row_ptr,
                                                         void *syn, RowIndex ix, const uint16_t *hist,
                                                         const uint32_t *keys, uint32_t cap)
{
    __shared__ RowLDS L;
    const uint32_t s = blockIdx.x, tid = threadIdx.x;
    const uint64_t beg = row_ptr[s];
    const uint32_t len = (uint32_t)(row_ptr[s + 1] - beg);
    const uint32_t nb = n_buckets(c, ix);
    zero_tiles(L, nb);
    const uint64_t rd = mix64(c.keys.delay ^ (uint64_t)s);
    const uint64_t rw = mix64(c.keys.w ^ (uint64_t)s);
    if (c.kind == SPK_CONN_BERNOULLI) {
        const uint64_t rk = mix64(c.keys.conn ^ (uint64_t)s);
        if (hist) {  // the count pass's bucket counts of this row
            const uint32_t HB = c.tl.T + 2 * kGroups, off = ix.desc ? c.tl.T : 0u;
            for (uint32_t k = tid; k < nb; k += kBlock) L.cur[k] = hist[(uint64_t)s * HB + off + k];
        } else {
            for (uint32_t tgt = tid; tgt < c.n; tgt += kBlock) {
                if (!((uint64_t)hash_hi32(mix64(rk ^ (uint64_t)tgt)) < c.conn_thr)) continue;
                const uint32_t j = c.lists > 1 ? hash_range(mix64(rd ^ (uint64_t)tgt), c.lists) : 0;
                atomicAdd(&L.cur[bucket_of(c, ix, tgt, j)], 1u);
            }
        }
        scan_tiles(L, nb);
        write_row_index(c, ix, L, s, beg, len);
        if (keys) {  // the row's synapses as the count pass kept them (len <= cap)
            for (uint32_t k = tid; k < len; k += kBlock) {
                const uint32_t key = keys[(uint64_t)s * cap + k];
                const uint32_t tgt = rec_target(key), j = rec_delay(key);
                const float w = syn_weight(c, s, mix64(rw ^ (uint64_t)tgt));
                const uint32_t pos = atomicAdd(&L.cur[bucket_of(c, ix, tgt, j)], 1u);
                put_syn(c, syn, beg + pos, j, tgt, s, w);
            }
            return;
        }
        for (uint32_t tgt = tid; tgt < c.n; tgt += kBlock) {
            if (!((uint64_t)hash_hi32(mix64(rk ^ (uint64_t)tgt)) < c.conn_thr)) continue;
            const uint32_t j = c.lists > 1 ? hash_range(mix64(rd ^ (uint64_t)tgt), c.lists) : 0;
            const float w = syn_weight(c, s, mix64(rw ^ (uint64_t)tgt));
            const uint32_t pos = atomicAdd(&L.cur[bucket_of(c, ix, tgt, j)], 1u);
            put_syn(c, syn, beg + pos, j, tgt, s, w);
        }
    } else {
        const uint64_t rt = mix64(c.keys.tgt ^ (uint64_t)s);
        for (uint32_t q = tid; q < c.k_out; q += kBlock) {
            const uint32_t tgt = hash_range(mix64(rt ^ (uint64_t)q), c.n);
            const uint32_t j = c.lists > 1 ? hash_range(mix64(rd ^ (uint64_t)q), c.lists) : 0;
            atomicAdd(&L.cur[bucket_of(c, ix, tgt, j)], 1u);
        }
        scan_tiles(L, nb);
        write_row_index(c, ix, L, s, beg, len);
        for (uint32_t q = tid; q < c.k_out; q += kBlock) {
            const uint32_t tgt = hash_range(mix64(rt ^ (uint64_t)q), c.n);
            const uint32_t j = c.lists > 1 ? hash_range(mix64(rd ^ (uint64_t)q), c.lists) : 0;
            const float w = syn_weight(c, s, mix64(rw ^ (uint64_t)q));
            const uint32_t pos = atomicAdd(&L.cur[bucket_of(c, ix, tgt, j)], 1u);
            put_syn(c, syn, beg + pos, j, tgt, s, w);
        }
    }
}

// ------------------------------------------------- fixed in-degree rows
// One block per target draws its sources; synapses are regrouped by source
// through global atomic cursors (unordered), then bucketed by bucket_rows.
// For networks of up to kInRanges * kInRange neurons, blocks of kInThreads
// take a run of targets each and count their draws per source in LDS, one
// range of kInRange sources at a time: one global update per (block,
// source) instead of one per synapse, for a few more passes of hashes.
__device__ __forceinline__ uint32_t in_source(const ConnArgs &c, uint64_t re, uint64_t ri,
                                              uint32_t q)
{
    if (q < c.k_in_exc) return hash_range(mix64(re ^ (uint64_t)q), c.n_exc);
    return c.n_exc + hash_range(mix64(ri ^ (uint64_t)(q - c.k_in_exc)), c.n - c.n_exc);
}

__global__ __launch_bounds__(kBlock) void k_gen_in_count(ConnArgs c, uint32_t *cnt)
{
    const uint32_t tgt = blockIdx.x;
    const uint64_t re = mix64(c.keys.src_e ^ (uint64_t)tgt);
    const uint64_t ri = mix64(c.keys.src_i ^ (uint64_t)tgt);
    const uint32_t kin = c.k_in_exc + c.k_in_inh;
    for (uint32_t q = threadIdx.x; q < kin; q += kBlock)
        atomicAdd(&cnt[in_source(c, re, ri, q)], 1u);
}

constexpr uint32_t kInThreads = 1024, kInRange = 32768, kInRanges = 8, kInBlocks = 1024;

// The draws of targets [t0, t1) that land in sources [r0, r0 + rn), counted
// into h[src - r0].
__device__ void in_range_counts(const ConnArgs &c, uint32_t t0, uint32_t t1, uint32_t r0, uint32_t rn,
                                uint32_t *h)
{
    const uint32_t kin = c.k_in_exc + c.k_in_inh;
    for (uint32_t tgt = t0; tgt < t1; tgt++) {
        const uint64_t re = mix64(c.keys.src_e ^ (uint64_t)tgt);
        const uint64_t ri = mix64(c.keys.src_i ^ (uint64_t)tgt);
        for (uint32_t q = threadIdx.x; q < kin; q += kInThreads) {
            const uint32_t k = in_source(c, re, ri, q) - r0;
            if (k < rn) atomicAdd(&h[k], 1u);
        }
    }
}

__global__ __launch_bounds__(kInThreads) void k_gen_in_count_lds(ConnArgs c, uint32_t tpb, uint32_t *cnt)
{
    __shared__ uint32_t h[kInRange];
    const uint32_t t0 = blockIdx.x * tpb;
    if (t0 >= c.n) return;
    const uint32_t t1 = c.n - t0 < tpb ? c.n : t0 + tpb;
    for (uint32_t r0 = 0; r0 < c.n; r0 += kInRange) {
        const uint32_t rn = c.n - r0 < kInRange ? c.n - r0 : kInRange;
        for (uint32_t k = threadIdx.x; k < rn; k += kInThreads) h[k] = 0;
        __syncthreads();
        in_range_counts(c, t0, t1, r0, rn, h);
        __syncthreads();
        for (uint32_t k = threadIdx.x; k < rn; k += kInThreads)
            if (h[k]) atomicAdd(&cnt[r0 + k], h[k]);
        __syncthreads();
    }
}

__global__ __launch_bounds__(kInThreads) void k_gen_in_fill_lds(ConnArgs c, uint32_t tpb, const uint64_t *row_ptr,
                                                               uint32_t *cursor, void *syn)
{
    __shared__ uint32_t h[kInRange];
    const uint32_t t0 = blockIdx.x * tpb;
    if (t0 >= c.n) return;
    const uint32_t t1 = c.n - t0 < tpb ? c.n : t0 + tpb;
    const uint32_t kin = c.k_in_exc + c.k_in_inh;
    for (uint32_t r0 = 0; r0 < c.n; r0 += kInRange) {
        const uint32_t rn = c.n - r0 < kInRange ? c.n - r0 : kInRange;
        for (uint32_t k = threadIdx.x; k < rn; k += kInThreads) h[k] = 0;
        __syncthreads();
        in_range_counts(c, t0, t1, r0, rn, h);
        __syncthreads();
        // this block's first position in each row of the range
        for (uint32_t k = threadIdx.x; k < rn; k += kInThreads)
            if (h[k]) h[k] = atomicAdd(&cursor[r0 + k], h[k]);
        __syncthreads();
        for (uint32_t tgt = t0; tgt < t1; tgt++) {
            const uint64_t re = mix64(c.keys.src_e ^ (uint64_t)tgt);
            const uint64_t ri = mix64(c.keys.src_i ^ (uint64_t)tgt);
            const uint64_t rd = mix64(c.keys.delay ^ (uint64_t)tgt);
            const uint64_t rw = mix64(c.keys.w ^ (uint64_t)tgt);
            for (uint32_t q = threadIdx.x; q < kin; q += kInThreads) {
                const uint32_t src = in_source(c, re, ri, q);
                if (src - r0 >= rn) continue;
                const uint32_t j = c.lists > 1 ? hash_range(mix64(rd ^ (uint64_t)q), c.lists) : 0;
                const float w = syn_weight(c, src, mix64(rw ^ (uint64_t)q));
                const uint32_t pos = atomicAdd(&h[src - r0], 1u);
                put_syn(c, syn, row_ptr[src] + pos, j, tgt, src, w);
            }
        }
        __syncthreads();
    }
}

__global__ __launch_bounds__(kBlock) void k_gen_in_fill(ConnArgs c, const uint64_t *row_ptr,
                                                       uint32_t *cursor, void *syn)
{
    const uint32_t tgt = blockIdx.x;
    const uint64_t re = mix64(c.keys.src_e ^ (uint64_t)tgt);
    const uint64_t ri = mix64(c.keys.src_i ^ (uint64_t)tgt);
    const uint64_t rd = mix64(c.keys.delay ^ (uint64_t)tgt);
    const uint64_t rw = mix64(c.keys.w ^ (uint64_t)tgt);
    const uint32_t kin = c.k_in_exc + c.k_in_inh;
    for (uint32_t q = threadIdx.x; q < kin; q += kBlock) {
        const uint32_t src = in_source(c, re, ri, q);
        const uint32_t j = c.lists > 1 ? hash_range(mix64(rd ^ (uint64_t)q), c.lists) : 0;
        const float w = syn_weight(c, src, mix64(rw ^ (uint64_t)q));
        const uint32_t pos = atomicAdd(&cursor[src], 1u);
        put_syn(c, syn, row_ptr[src] + pos, j, tgt, src, w);
    }
}

// Explicit adjacency (host-given rows, already in row order): encode.
__global__ __launch_bounds__(kBlock) void k_csr_fill(ConnArgs c, uint64_t nnz, const uint32_t *in_col,
                                                    const float *in_w, const uint8_t *in_delay,
                                                    void *syn)
{
    for (uint64_t e = (uint64_t)blockIdx.x * kBlock + threadIdx.x; e < nnz;
         e += (uint64_t)gridDim.x * kBlock) {
        const uint32_t j = in_delay ? (uint32_t)in_delay[e] - c.dmin : 0u;
        put_syn(c, syn, e, j, in_col[e], 0u, in_w[e]);
    }
}

// Group the synapses of every row of src by bucket into dst (same row_ptr)
// and write the row's range boundaries.  Blocks stride over rows.
template <class R>
__global__ __launch_bounds__(kBlock) void k_bucket_rows(ConnArgs c, const uint64_t *row_ptr,
                                                       const R *src, R *dst, RowIndex ix)
{
    __shared__ RowLDS L;
    for (uint32_t s = blockIdx.x; s < c.n; s += gridDim.x) {
        const uint64_t beg = row_ptr[s];
        const uint32_t len = (uint32_t)(row_ptr[s + 1] - beg);
        const uint32_t nb = n_buckets(c, ix);
        zero_tiles(L, nb);
        for (uint32_t e = threadIdx.x; e < len; e += kBlock) {
            const uint32_t key = rec_key(src[beg + e]);
            atomicAdd(&L.cur[bucket_of(c, ix, rec_target(key), rec_delay(key))], 1u);
        }
        scan_tiles(L, nb);
        write_row_index(c, ix, L, s, beg, len);
        for (uint32_t e = threadIdx.x; e < len; e += kBlock) {
            const R r = src[beg + e];
            const uint32_t key = rec_key(r);
            const uint32_t pos = atomicAdd(&L.cur[bucket_of(c, ix, rec_target(key), rec_delay(key))], 1u);
            dst[beg + pos] = r;
        }
        __syncthreads();
    }
}

// ------------------------------------------------------------------ scan
// Exclusive scan of m u32 counts into u64 offsets (m+1 entries), plus the
// largest count.  Three passes: block-local scan, scan of block sums,
// add-back.
constexpr int kScanPer = 8;
constexpr int kScanTile = kBlock * kScanPer;

__device__ __forceinline__ uint64_t block_exclusive_scan(uint64_t x, uint64_t *total)
{
    __shared__ uint64_t ws[kBlock / kWave];
    const uint32_t lane = lane_id(), w = threadIdx.x / kWave;
    uint64_t inc = x;
    for (int o = 1; o < kWave; o <<= 1) {
        uint64_t y = __shfl_up(inc, o);
        if (lane >= (uint32_t)o) inc += y;
    }
    if (lane == kWave - 1) ws[w] = inc;
    __syncthreads();
    uint64_t before = 0, tot = 0;
    for (uint32_t k = 0; k < kBlock / kWave; k++) {
        if (k < w) before += ws[k];
        tot += ws[k];
    }
    __syncthreads();
    *total = tot;
    return before + inc - x;
}

__global__ __launch_bounds__(kBlock) void k_scan1(const uint32_t *cnt, uint64_t m, uint64_t *out,
                                                 uint64_t *bsum, uint32_t *maxp)
{
    const uint64_t base = (uint64_t)blockIdx.x * kScanTile + (uint64_t)threadIdx.x * kScanPer;
    uint32_t v[kScanPer];
    uint64_t sum = 0;
    uint32_t mx = 0;
    for (int k = 0; k < kScanPer; k++) {
        v[k] = base + k < m ? cnt[base + k] : 0u;
        sum += v[k];
        mx = v[k] > mx ? v[k] : mx;
    }
    uint64_t tot;
    uint64_t off = block_exclusive_scan(sum, &tot);
    for (int k = 0; k < kScanPer; k++) {
        if (base + k < m) out[base + k] = off;
        off += v[k];
    }
    for (int o = 32; o > 0; o >>= 1) {
        uint32_t y = __shfl_xor(mx, o);
        mx = y > mx ? y : mx;
    }
    if (lane_id() == 0 && mx) atomicMax(maxp, mx);
    if (threadIdx.x == 0) bsum[blockIdx.x] = tot;
}

__global__ __launch_bounds__(kBlock) void k_scan2(uint64_t *bsum, uint64_t nb)
{
    uint64_t carry = 0;
    for (uint64_t base = 0; base < nb; base += kBlock) {
        uint64_t i = base + threadIdx.x;
        uint64_t x = i < nb ? bsum[i] : 0;
        uint64_t tot;
        uint64_t ex = block_exclusive_scan(x, &tot);
        if (i < nb) bsum[i] = carry + ex;
        carry += tot;
    }
    if (threadIdx.x == 0) bsum[nb] = carry;
}

__global__ __launch_bounds__(kBlock) void k_scan3(uint64_t *out, uint64_t m, const uint64_t *bsum,
                                                 uint64_t nb)
{
    const uint64_t base = (uint64_t)blockIdx.x * kScanTile;
    const uint64_t add = bsum[blockIdx.x];
    for (int k = 0; k < kScanPer; k++) {
        uint64_t i = base + (uint64_t)k * kBlock + threadIdx.x;
        if (i < m) out[i] += add;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) out[m] = bsum[nb];
}

// --------------------------------------------------------- bookkeeping

__global__ __launch_bounds__(kBlock) void k_out_degree(const uint64_t *row_ptr, uint32_t n,
                                                      uint32_t *outdeg)
{
    const uint32_t s = blockIdx.x * kBlock + threadIdx.x;
    if (s < n) outdeg[s] = (uint32_t)(row_ptr[s + 1] - row_ptr[s]);
}

// Per-target sum of |weight| over all in-synapses: exact in quantised units
// (fixed mode), or an upper bound in units of 2^-24 (fp32 mode: each term
// rounded up), used to size the accumulators.  Compact synapses take the
// term of their class from the table (the same value).
__global__ __launch_bounds__(kBlock) void k_in_abs_sum(const void *syn, uint64_t nnz, int fixed,
                                                      int compact, ClassTab tab,
                                                      unsigned long long *insum)
{
    for (uint64_t e = (uint64_t)blockIdx.x * kBlock + threadIdx.x; e < nnz;
         e += (uint64_t)gridDim.x * kBlock) {
        if (compact) {
            const uint32_t x = ((const uint32_t *)syn)[e];
            atomicAdd(&insum[rec_target(x)], (unsigned long long)tab.abs[rec_class(x)]);
            continue;
        }
        const int2 x = ((const int2 *)syn)[e];
        unsigned long long q;
        if (fixed) {
            q = (unsigned long long)(x.y < 0 ? -(long long)x.y : (long long)x.y);
        } else {
            const float w = fabsf(__int_as_float(x.y));
            q = (unsigned long long)ceil(ldexp((double)w, 24));
        }
        atomicAdd(&insum[(uint32_t)x.x & kTargetMask], q);
    }
}

// Largest sum of |weight| into any neuron of a Bernoulli network, with no
// atomic per synapse: thread j evaluates the connection predicate of every
// source s of its block's source range into j (the generator's hash of the
// pair) and adds the term of each synapse it finds, in the units of
// k_in_abs_sum; the sources' row keys are staged in LDS.  One source range
// (grid.y = 1): a block's largest sum goes to *out by one atomic; several
// (small networks, to fill the device): partial sums go to insum[j].
// Cost: n^2 hashes (one pass of the generator), against nnz global atomics.
__device__ __forceinline__ unsigned long long abs_term(const ConnArgs &c, uint32_t src, uint64_t hw)
{
    const float w = syn_weight(c, src, hw);
    if (c.fixed) {
        const int32_t q = weight_bits(c, w);
        return (unsigned long long)(q < 0 ? -(long long)q : (long long)q);
    }
    return (unsigned long long)ceil(ldexp((double)fabsf(w), 24));
}

__global__ __launch_bounds__(kBlock) void k_bern_in_abs_max(ConnArgs c, uint32_t src_chunk, unsigned long long *out,
                                                           unsigned long long *insum)
{
    __shared__ uint64_t rk[kBlock], rw[kBlock];
    __shared__ unsigned long long wmax[kBlock / kWave];
    const uint32_t j = blockIdx.x * kBlock + threadIdx.x;
    const uint32_t sb = blockIdx.y * src_chunk;
    const uint32_t se = c.n - sb < src_chunk ? c.n : sb + src_chunk;
    const unsigned long long te = abs_term(c, 0, 0), ti = abs_term(c, c.n_exc, 0);  // population weights
    unsigned long long sum = 0;
    for (uint32_t s0 = sb; s0 < se; s0 += kBlock) {
        __syncthreads();
        const uint64_t sl = (uint64_t)s0 + threadIdx.x;
        rk[threadIdx.x] = mix64(c.keys.conn ^ sl);
        rw[threadIdx.x] = mix64(c.keys.w ^ sl);
        __syncthreads();
        const uint32_t ns = se - s0 < kBlock ? se - s0 : kBlock;
        if (j >= c.n) continue;
        for (uint32_t k = 0; k < ns; k++) {
            if (!((uint64_t)hash_hi32(mix64(rk[k] ^ (uint64_t)j)) < c.conn_thr)) continue;
            const uint32_t src = s0 + k;
            sum += c.w_uniform ? abs_term(c, src, mix64(rw[k] ^ (uint64_t)j)) : (src < c.n_exc ? te : ti);
        }
    }
    if (gridDim.y > 1) {
        if (j < c.n && sum) atomicAdd(&insum[j], sum);
        return;
    }
    for (int o = 32; o > 0; o >>= 1) {
        const unsigned long long y = __shfl_xor(sum, o);
        sum = y > sum ? y : sum;
    }
    if (lane_id() == 0) wmax[threadIdx.x / kWave] = sum;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long mx = 0;
        for (uint32_t k = 0; k < kBlock / kWave; k++) mx = wmax[k] > mx ? wmax[k] : mx;
        if (mx) atomicMax(out, mx);
    }
}

// Largest sum of |weight| into one neuron of a fixed out-degree network
// with population weights, without a global atomic per synapse.  Every
// synapse is drawn again (the generator's target hash; its term depends only
// on the class of its source population), counted per target tile by blocks
// of kFoSrc sources (one global reservation per block and tile), then filed
// into per-tile buckets as (class << 14 | neuron within the tile); one block
// per tile counts its neurons' in-synapses per class in LDS and takes the
// largest sum of class counts x class terms.
constexpr uint32_t kFoSrc = 256;  // sources per block of the counting and filing passes

__global__ __launch_bounds__(kBlock) void k_fo_count(ConnArgs c, uint32_t *base, uint32_t *tile_total)
{
    __shared__ uint32_t cnt[kMaxTiles];
    const uint32_t T = c.tl.T, tid = threadIdx.x;
    const uint32_t s0 = blockIdx.x * kFoSrc, s1 = s0 + kFoSrc < c.n ? s0 + kFoSrc : c.n;
    for (uint32_t k = tid; k < T; k += kBlock) cnt[k] = 0;
    __syncthreads();
    for (uint32_t s = s0; s < s1; s++) {
        const uint64_t rt = mix64(c.keys.tgt ^ (uint64_t)s);
        for (uint32_t q = tid; q < c.k_out; q += kBlock)
            atomicAdd(&cnt[hash_range(mix64(rt ^ (uint64_t)q), c.n) >> c.tl.logW], 1u);
    }
    __syncthreads();
    for (uint32_t k = tid; k < T; k += kBlock)
        base[(uint64_t)blockIdx.x * T + k] = cnt[k] ? atomicAdd(&tile_total[k], cnt[k]) : 0u;
}

// Filing: the block's synapses are drawn again kFoStage at a time,
// counting-sorted by target tile in LDS, and each tile's run is written
// contiguously after what the block filed there before (its reservation).
constexpr uint32_t kFoThreads = 1024;
constexpr uint32_t kFoPer = 32;                          // synapses per thread and round
constexpr uint32_t kFoStage = kFoPer * kFoThreads;       // synapses sorted at once

__global__ __launch_bounds__(kFoThreads) void k_fo_file(ConnArgs c, const uint32_t *base, const uint64_t *tile_start,
                                                       uint16_t *entries)
{
    __shared__ uint16_t stage[kFoStage];   // (class << 14 | neuron in tile), sorted by tile
    __shared__ uint16_t stile[kFoStage];   // the tile of each staged entry
    __shared__ uint32_t cnt[kMaxTiles], off[kMaxTiles], cur[kMaxTiles];
    __shared__ uint32_t ws[kFoThreads / kWave];
    const uint32_t T = c.tl.T, tid = threadIdx.x, lane = lane_id(), w = tid / kWave;
    const uint32_t s0 = blockIdx.x * kFoSrc, s1 = s0 + kFoSrc < c.n ? s0 + kFoSrc : c.n;
    const uint64_t V = (uint64_t)(s1 - s0) * c.k_out;
    for (uint32_t k = tid; k < T; k += kFoThreads) cur[k] = base[(uint64_t)blockIdx.x * T + k];
    // this thread's next synapse: v = v0 + tid + kFoThreads * u, i.e. synapse j of source s0 + si
    uint32_t si = tid / c.k_out, j = tid - si * c.k_out;
    for (uint64_t v0 = 0; v0 < V; v0 += kFoStage) {
        for (uint32_t k = tid; k < T; k += kFoThreads) cnt[k] = 0;
        __syncthreads();
        uint32_t ent[kFoPer];  // tile << 16 | entry, rank in the tile's run of this round in ...
        uint32_t rnk[kFoPer];
#pragma unroll
        for (int u = 0; u < (int)kFoPer; u++) {
            const uint64_t v = v0 + tid + (uint64_t)kFoThreads * u;
            ent[u] = 0xffffffffu;
            if (v < V) {
                const uint32_t s = s0 + si;
                const uint32_t tgt = hash_range(key_hash(c.keys.tgt, s, j), c.n), tile = tgt >> c.tl.logW;
                const uint32_t cls = s < c.n_exc ? 0u : 1u;
                ent[u] = (tile << 16) | (cls << 14) | (tgt & (c.tl.W - 1));
                rnk[u] = atomicAdd(&cnt[tile], 1u);
            }
            j += kFoThreads;
            while (j >= c.k_out) {
                j -= c.k_out;
                si++;
            }
        }
        __syncthreads();
        // exclusive scan of the round's tile counts (T <= 2048: two per thread)
        {
            const uint32_t b = 2 * tid;
            const uint32_t c0 = b < T ? cnt[b] : 0u, c1 = b + 1 < T ? cnt[b + 1] : 0u;
            uint32_t inc = c0 + c1;
            for (int o = 1; o < kWave; o <<= 1) {
                const uint32_t y = __shfl_up(inc, o);
                if (lane >= (uint32_t)o) inc += y;
            }
            if (lane == kWave - 1) ws[w] = inc;
            __syncthreads();
            uint32_t before = 0;
            for (uint32_t k = 0; k < w; k++) before += ws[k];
            const uint32_t ex = before + inc - (c0 + c1);
            if (b < T) off[b] = ex;
            if (b + 1 < T) off[b + 1] = ex + c0;
        }
        __syncthreads();
        uint32_t staged = 0;
#pragma unroll
        for (int u = 0; u < (int)kFoPer; u++) {
            if (ent[u] == 0xffffffffu) continue;
            const uint32_t tile = ent[u] >> 16, q = off[tile] + rnk[u];
            stage[q] = (uint16_t)(ent[u] & 0xffffu);
            stile[q] = (uint16_t)tile;
            staged++;
        }
        const uint32_t n_round = (uint32_t)(V - v0 < kFoStage ? V - v0 : kFoStage);
        __syncthreads();
        // consecutive staged entries of a tile go to consecutive positions
        for (uint32_t q = tid; q < n_round; q += kFoThreads) {
            const uint32_t tile = stile[q];
            entries[tile_start[tile] + cur[tile] + (q - off[tile])] = stage[q];
        }
        __syncthreads();
        for (uint32_t k = tid; k < T; k += kFoThreads) cur[k] += cnt[k];
        (void)staged;
    }
}

__global__ __launch_bounds__(1024) void k_fo_max(ConnArgs c, const uint64_t *tile_start, const uint16_t *entries,
                                                ClassTab tab, unsigned long long *out)
{
    __shared__ uint32_t cnt[2][kMaxTileW];
    __shared__ unsigned long long wmax[1024 / kWave];
    const uint32_t tile = blockIdx.x, tid = threadIdx.x, W = c.tl.W;
    for (uint32_t k = tid; k < W; k += 1024) cnt[0][k] = cnt[1][k] = 0;
    __syncthreads();
    const uint64_t e0 = tile_start[tile], e1 = tile_start[tile + 1];
    for (uint64_t e = e0 + tid; e < e1; e += 1024) {
        const uint32_t v = entries[e];
        atomicAdd(&cnt[v >> 14][v & 0x3fffu], 1u);
    }
    __syncthreads();
    unsigned long long m = 0;
    for (uint32_t k = tid; k < W; k += 1024) {
        const unsigned long long x = (unsigned long long)cnt[0][k] * tab.abs[0] + (unsigned long long)cnt[1][k] * tab.abs[1];
        m = x > m ? x : m;
    }
    for (int o = 32; o > 0; o >>= 1) {
        const unsigned long long y = __shfl_xor(m, o);
        m = y > m ? y : m;
    }
    if ((tid & (kWave - 1)) == 0) wmax[tid / kWave] = m;
    __syncthreads();
    if (tid == 0) {
        for (uint32_t k = 1; k < 1024 / kWave; k++) m = wmax[k] > m ? wmax[k] : m;
        atomicMax(out, m);
    }
}

__global__ __launch_bounds__(kBlock) void k_max_u64(const uint64_t *x, uint64_t m,
                                                   unsigned long long *out)
{
    unsigned long long mx = 0;
    for (uint64_t i = (uint64_t)blockIdx.x * kBlock + threadIdx.x; i < m;
         i += (uint64_t)gridDim.x * kBlock)
        mx = x[i] > mx ? x[i] : mx;
    for (int o = 32; o > 0; o >>= 1) {
        unsigned long long y = __shfl_xor(mx, o);
        mx = y > mx ? y : mx;
    }
    if (lane_id() == 0 && mx) atomicMax(out, mx);
}

// V0 = v0_lo + (v0_hi - v0_lo) * U[0,1), refractory counters 0.
__global__ __launch_bounds__(kBlock) void k_init_state(ModelArgs m, float v0_lo, float v0_hi,
                                                      float *V, uint8_t *ref)
{
    const uint32_t i = blockIdx.x * kBlock + threadIdx.x;
    if (i >= m.n) return;
    const float span = __fsub_rn(v0_hi, v0_lo);
    V[i] = __fadd_rn(v0_lo, __fmul_rn(span, u24(key_hash(m.keys.v0, i, 0))));
    ref[i] = 0;
}

// ---------------------------------------------------------------- export

// One block per requested row: decode (target, delay, weight bits).
__global__ __launch_bounds__(kBlock) void k_export_gather(const uint64_t *row_ptr, const void *syn,
                                                         int compact, ClassTab tab, uint32_t dmin,
                                                         const uint32_t *rows, const uint64_t *out_off,
                                                         uint32_t *col, uint32_t *wbits, uint8_t *delay)
{
    const uint64_t r = blockIdx.x;
    const uint32_t s = rows[r];
    const uint64_t beg = row_ptr[s], L = row_ptr[s + 1] - beg;
    const uint64_t o = out_off[r];
    for (uint64_t e = threadIdx.x; e < L; e += kBlock) {
        uint32_t key, wb;
        if (compact) {
            key = ((const uint32_t *)syn)[beg + e];
            wb = tab.bits[rec_class(key)];
        } else {
            const int2 x = ((const int2 *)syn)[beg + e];
            key = (uint32_t)x.x;
            wb = (uint32_t)x.y;
        }
        col[o + e] = rec_target(key);
        wbits[o + e] = wb;
        delay[o + e] = (uint8_t)(dmin + rec_delay(key));
    }
}

uint32_t grid_for(uint64_t threads, uint32_t cap = 1u << 20)
{
    uint64_t g = (threads + kBlock - 1) / kBlock;
    if (g == 0) g = 1;
    return g > cap ? cap : (uint32_t)g;
}

}  // namespace

// -------------------------------------------------------- launch wrappers

int cu_count()
{
    static int cus = 0;
    if (!cus) {
        int dev = 0, v = 0;
        if (hipGetDevice(&dev) == hipSuccess &&
            hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && v > 0)
            cus = v;
        else
            cus = 256;
    }
    return cus;
}

hipError_t gen_count_rows(const ConnArgs &c, uint32_t *cnt, uint16_t *hist, uint32_t *keys, uint32_t cap,
                          hipStream_t s)
{
    if (c.tl.T > kMaxTiles || (keys && (!hist || c.n > kTargetMask + 1u))) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_gen_count_rows, dim3(c.n), dim3(kBlock), 0, s, c, cnt, hist, keys, cap);
    return hipGetLastError();
}

hipError_t gen_fill_rows(const ConnArgs &c, const uint64_t *row_ptr, void *syn, RowIndex ix,
                         const uint16_t *hist, const uint32_t *keys, uint32_t cap, hipStream_t s)
{
    if (c.tl.T > kMaxTiles || (keys && !hist)) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_gen_fill_rows, dim3(c.n), dim3(kBlock), 0, s, c, row_ptr, syn, ix, hist, keys, cap);
    return hipGetLastError();
}

// block-local counting where the source ranges are few (see above);
// SPK_GEN_IN_ATOMICS=1 forces the per-synapse path (a test knob)
static bool in_rows_lds(const ConnArgs &c)
{
    const char *e = std::getenv("SPK_GEN_IN_ATOMICS");
    if (e && std::strcmp(e, "1") == 0) return false;
    return c.n <= kInRanges * kInRange;
}
static uint32_t in_rows_tpb(const ConnArgs &c) { return (c.n + kInBlocks - 1) / kInBlocks; }

hipError_t gen_in_count(const ConnArgs &c, uint32_t *cnt, hipStream_t s)
{
    if (in_rows_lds(c)) {
        const uint32_t tpb = in_rows_tpb(c);
        hipLaunchKernelGGL(k_gen_in_count_lds, dim3((c.n + tpb - 1) / tpb), dim3(kInThreads), 0, s, c, tpb, cnt);
    } else {
        hipLaunchKernelGGL(k_gen_in_count, dim3(c.n), dim3(kBlock), 0, s, c, cnt);
    }
    return hipGetLastError();
}

hipError_t gen_in_fill(const ConnArgs &c, const uint64_t *row_ptr, uint32_t *cursor, void *syn,
                       hipStream_t s)
{
    if (in_rows_lds(c)) {
        const uint32_t tpb = in_rows_tpb(c);
        hipLaunchKernelGGL(k_gen_in_fill_lds, dim3((c.n + tpb - 1) / tpb), dim3(kInThreads), 0, s, c, tpb, row_ptr,
                           cursor, syn);
    } else {
        hipLaunchKernelGGL(k_gen_in_fill, dim3(c.n), dim3(kBlock), 0, s, c, row_ptr, cursor, syn);
    }
    return hipGetLastError();
}

hipError_t csr_fill(const ConnArgs &c, uint64_t nnz, const uint32_t *in_col, const float *in_w,
                    const uint8_t *in_delay, void *syn, hipStream_t s)
{
    if (!nnz) return hipSuccess;
    hipLaunchKernelGGL(k_csr_fill, dim3(grid_for(nnz, 65536)), dim3(kBlock), 0, s, c, nnz, in_col,
                       in_w, in_delay, syn);
    return hipGetLastError();
}

hipError_t bucket_rows(const ConnArgs &c, const uint64_t *row_ptr, const void *src, void *dst,
                       RowIndex ix, hipStream_t s)
{
    if (c.tl.T > kMaxTiles) return hipErrorInvalidValue;
    const uint32_t g = c.n < 65536u ? c.n : 65536u;
    if (c.compact)
        hipLaunchKernelGGL(k_bucket_rows<uint32_t>, dim3(g ? g : 1), dim3(kBlock), 0, s, c, row_ptr,
                           (const uint32_t *)src, (uint32_t *)dst, ix);
    else
        hipLaunchKernelGGL(k_bucket_rows<int2>, dim3(g ? g : 1), dim3(kBlock), 0, s, c, row_ptr,
                           (const int2 *)src, (int2 *)dst, ix);
    return hipGetLastError();
}

size_t scan_scratch_elems(uint64_t m) { return (size_t)((m + kScanTile - 1) / kScanTile) + 1; }

hipError_t scan_counts(const uint32_t *cnt, uint64_t m, uint64_t *out, uint64_t *block_sums,
                       uint32_t *max_count, hipStream_t s)
{
    const uint64_t nb = (m + kScanTile - 1) / kScanTile;
    if (nb == 0) {
        return hipMemsetAsync(out, 0, sizeof(uint64_t), s);
    }
    hipLaunchKernelGGL(k_scan1, dim3((uint32_t)nb), dim3(kBlock), 0, s, cnt, m, out, block_sums,
                       max_count);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_scan2, dim3(1), dim3(kBlock), 0, s, block_sums, nb);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_scan3, dim3((uint32_t)nb), dim3(kBlock), 0, s, out, m, block_sums, nb);
    return hipGetLastError();
}

hipError_t out_degree(const uint64_t *row_ptr, uint32_t n, uint32_t *outdeg, hipStream_t s)
{
    hipLaunchKernelGGL(k_out_degree, dim3(grid_for(n)), dim3(kBlock), 0, s, row_ptr, n, outdeg);
    return hipGetLastError();
}

hipError_t in_abs_sum(const void *syn, uint64_t nnz, bool fixed, bool compact, const ClassTab &tab,
                      uint64_t *insum, hipStream_t s)
{
    if (!nnz) return hipSuccess;
    hipLaunchKernelGGL(k_in_abs_sum, dim3(grid_for(nnz, 65536)), dim3(kBlock), 0, s, syn, nnz,
                       fixed ? 1 : 0, compact ? 1 : 0, tab, (unsigned long long *)insum);
    return hipGetLastError();
}

uint32_t bern_src_ranges(uint32_t n)
{
    // about 4096 blocks: split the sources when the targets alone give fewer
    const uint32_t tb = (n + kBlock - 1) / kBlock;
    uint32_t S = (4096 + tb - 1) / tb;
    S = S < 1 ? 1 : (S > 64 ? 64 : S);
    return S;
}

hipError_t bern_in_abs_max(const ConnArgs &c, uint64_t *out, uint64_t *insum, hipStream_t s)
{
    if (c.kind != SPK_CONN_BERNOULLI) return hipErrorInvalidValue;
    const uint32_t S = bern_src_ranges(c.n);
    const uint32_t chunk = ((c.n + S - 1) / S + kBlock - 1) / kBlock * kBlock;
    const uint32_t Sused = chunk ? (c.n + chunk - 1) / chunk : 1;
    if (Sused > 1 && !insum) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_bern_in_abs_max, dim3(grid_for(c.n), Sused ? Sused : 1), dim3(kBlock), 0, s, c, chunk,
                       (unsigned long long *)out, (unsigned long long *)insum);
    hipError_t e = hipGetLastError();
    if (e == hipSuccess && Sused > 1) e = max_u64(insum, c.n, out, s);
    return e;
}

uint32_t fo_blocks(uint32_t n) { return (n + kFoSrc - 1) / kFoSrc; }

hipError_t fo_count(const ConnArgs &c, uint32_t *base, uint32_t *tile_total, hipStream_t s)
{
    if (c.kind != SPK_CONN_FIXED_OUT || c.tl.T > kMaxTiles) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_fo_count, dim3(fo_blocks(c.n)), dim3(kBlock), 0, s, c, base, tile_total);
    return hipGetLastError();
}

hipError_t fo_file(const ConnArgs &c, const uint32_t *base, const uint64_t *tile_start, uint16_t *entries,
                   hipStream_t s)
{
    if (c.kind != SPK_CONN_FIXED_OUT || c.tl.T > kMaxTiles || c.tl.W > (1u << 14) || c.k_out == 0)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_fo_file, dim3(fo_blocks(c.n)), dim3(kFoThreads), 0, s, c, base, tile_start, entries);
    return hipGetLastError();
}

hipError_t fo_max(const ConnArgs &c, const uint64_t *tile_start, const uint16_t *entries, const ClassTab &tab,
                  uint64_t *out, hipStream_t s)
{
    if (c.tl.W > kMaxTileW || c.tl.T == 0) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_fo_max, dim3(c.tl.T), dim3(1024), 0, s, c, tile_start, entries, tab,
                       (unsigned long long *)out);
    return hipGetLastError();
}

hipError_t max_u64(const uint64_t *x, uint64_t m, uint64_t *out, hipStream_t s)
{
    hipLaunchKernelGGL(k_max_u64, dim3(grid_for(m, 4096)), dim3(kBlock), 0, s, x, m,
                       (unsigned long long *)out);
    return hipGetLastError();
}

hipError_t init_state(const ModelArgs &m, float v0_lo, float v0_hi, float *V, uint8_t *ref,
                      hipStream_t s)
{
    hipLaunchKernelGGL(k_init_state, dim3(grid_for(m.n)), dim3(kBlock), 0, s, m, v0_lo, v0_hi, V, ref);
    return hipGetLastError();
}

hipError_t export_gather(const uint64_t *row_ptr, const void *syn, bool compact, const ClassTab &tab,
                         uint32_t dmin, const uint32_t *rows, uint64_t n_rows, const uint64_t *out_off,
                         uint32_t *col, uint32_t *wbits, uint8_t *delay, hipStream_t s)
{
    if (!n_rows) return hipSuccess;
    if (n_rows > 0x7fffffffull) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_export_gather, dim3((uint32_t)n_rows), dim3(kBlock), 0, s, row_ptr, syn,
                       compact ? 1 : 0, tab, dmin, rows, out_off, col, wbits, delay);
    return hipGetLastError();
}

}  // namespace spk
