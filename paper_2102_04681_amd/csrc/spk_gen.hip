// spk_kernels.hip -- HIP kernels of libspk for gfx950 (MI355X, wave64).
//
// Build with -ffp-contract=off: the neuron update must round every fp32
// operation separately (forward Euler in single precision, Sec. IV-A of the
// paper), so no multiply-add may be fused.  The update additionally uses
// the explicit _rn intrinsics.
#include <hip/hip_runtime.h>

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

__device__ __forceinline__ uint32_t lane_id() { return threadIdx.x & (kWave - 1); }

__device__ __forceinline__ uint32_t mbcnt(uint64_t mask)
{
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                     __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t x)
{
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
    return x;
}

__device__ __forceinline__ uint64_t pack(int2 e)
{
    return ((uint64_t)(uint32_t)e.x << 32) | (uint64_t)(uint32_t)e.y;
}
__device__ __forceinline__ int2 unpack(uint64_t k)
{
    return make_int2((int)(uint32_t)(k >> 32), (int)(uint32_t)k);
}

// ------------------------------------------------------------ generation
// Per-delay adjacency lists (Sec. V): list j holds the synapses of delay
// dmin + j; "piece" (j, s) = the synapses of source s in list j, stored
// contiguously at [row_ptr[j*n+s], row_ptr[j*n+s+1]).

// Count pieces of Bernoulli / fixed out-degree rows: one block per source.
__global__ __launch_bounds__(kBlock) void k_gen_count_rows(ConnArgs c, uint32_t *cnt)
{
    __shared__ uint32_t lc[kMaxLists];
    const uint32_t s = blockIdx.x, tid = threadIdx.x;
    for (uint32_t j = tid; j < c.lists; j += kBlock) lc[j] = 0;
    __syncthreads();
    const uint64_t rd = mix64(c.keys.delay ^ (uint64_t)s);
    uint32_t mine = 0;
    if (c.kind == SPK_CONN_BERNOULLI) {
        const uint64_t rk = mix64(c.keys.conn ^ (uint64_t)s);
        for (uint32_t tgt = tid; tgt < c.n; tgt += kBlock) {
            if ((uint64_t)hash_hi32(mix64(rk ^ (uint64_t)tgt)) < c.conn_thr) {
                if (c.lists > 1) atomicAdd(&lc[hash_range(mix64(rd ^ (uint64_t)tgt), c.lists)], 1u);
                else mine++;
            }
        }
    } else {
        for (uint32_t q = tid; q < c.k_out; q += kBlock) {
            if (c.lists > 1) atomicAdd(&lc[hash_range(mix64(rd ^ (uint64_t)q), c.lists)], 1u);
            else mine++;
        }
    }
    if (c.lists == 1 && mine) atomicAdd(&lc[0], mine);
    __syncthreads();
    for (uint32_t j = tid; j < c.lists; j += kBlock) cnt[(uint64_t)j * c.n + s] = lc[j];
}

// Fill pieces of Bernoulli / fixed out-degree rows (unordered inside a
// piece; k_sort_* establish the order).
__global__ __launch_bounds__(kBlock) void k_gen_fill_rows(ConnArgs c, const uint64_t *row_ptr,
                                                         int2 *syn)
{
    __shared__ uint32_t cur[kMaxLists];
    const uint32_t s = blockIdx.x, tid = threadIdx.x;
    for (uint32_t j = tid; j < c.lists; j += kBlock) cur[j] = 0;
    __syncthreads();
    const uint64_t rd = mix64(c.keys.delay ^ (uint64_t)s);
    const uint64_t rw = mix64(c.keys.w ^ (uint64_t)s);
    if (c.kind == SPK_CONN_BERNOULLI) {
        const uint64_t rk = mix64(c.keys.conn ^ (uint64_t)s);
        for (uint32_t tgt = tid; tgt < c.n; tgt += kBlock) {
            if (!((uint64_t)hash_hi32(mix64(rk ^ (uint64_t)tgt)) < c.conn_thr)) continue;
            uint32_t j = c.lists > 1 ? hash_range(mix64(rd ^ (uint64_t)tgt), c.lists) : 0;
            float w = syn_weight(c, s, mix64(rw ^ (uint64_t)tgt));
            uint32_t pos = atomicAdd(&cur[j], 1u);
            syn[row_ptr[(uint64_t)j * c.n + s] + pos] = make_int2((int)tgt, weight_bits(c, w));
        }
    } else {
        const uint64_t rt = mix64(c.keys.tgt ^ (uint64_t)s);
        for (uint32_t q = tid; q < c.k_out; q += kBlock) {
            uint32_t tgt = hash_range(mix64(rt ^ (uint64_t)q), c.n);
            uint32_t j = c.lists > 1 ? hash_range(mix64(rd ^ (uint64_t)q), c.lists) : 0;
            float w = syn_weight(c, s, mix64(rw ^ (uint64_t)q));
            uint32_t pos = atomicAdd(&cur[j], 1u);
            syn[row_ptr[(uint64_t)j * c.n + s] + pos] = make_int2((int)tgt, weight_bits(c, w));
        }
    }
}

// Fixed in-degree: one block per target draws its sources; the synapses
// are regrouped by source through global atomic counters.
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
    const uint64_t rd = mix64(c.keys.delay ^ (uint64_t)tgt);
    const uint32_t kin = c.k_in_exc + c.k_in_inh;
    for (uint32_t q = threadIdx.x; q < kin; q += kBlock) {
        uint32_t src = in_source(c, re, ri, q);
        uint32_t j = c.lists > 1 ? hash_range(mix64(rd ^ (uint64_t)q), c.lists) : 0;
        atomicAdd(&cnt[(uint64_t)j * c.n + src], 1u);
    }
}

__global__ __launch_bounds__(kBlock) void k_gen_in_fill(ConnArgs c, const uint64_t *row_ptr,
                                                       uint32_t *cursor, int2 *syn)
{
    const uint32_t tgt = blockIdx.x;
    const uint64_t re = mix64(c.keys.src_e ^ (uint64_t)tgt);
    const uint64_t ri = mix64(c.keys.src_i ^ (uint64_t)tgt);
    const uint64_t rd = mix64(c.keys.delay ^ (uint64_t)tgt);
    const uint64_t rw = mix64(c.keys.w ^ (uint64_t)tgt);
    const uint32_t kin = c.k_in_exc + c.k_in_inh;
    for (uint32_t q = threadIdx.x; q < kin; q += kBlock) {
        uint32_t src = in_source(c, re, ri, q);
        uint32_t j = c.lists > 1 ? hash_range(mix64(rd ^ (uint64_t)q), c.lists) : 0;
        float w = syn_weight(c, src, mix64(rw ^ (uint64_t)q));
        uint64_t piece = (uint64_t)j * c.n + src;
        uint32_t pos = atomicAdd(&cursor[piece], 1u);
        syn[row_ptr[piece] + pos] = make_int2((int)tgt, weight_bits(c, w));
    }
}

// Explicit adjacency (host-given rows): one thread per source row.
__global__ __launch_bounds__(kBlock) void k_csr_count(ConnArgs c, const uint64_t *in_ptr,
                                                     const uint8_t *in_delay, uint32_t *cnt)
{
    const uint32_t s = blockIdx.x * kBlock + threadIdx.x;
    if (s >= c.n) return;
    for (uint64_t e = in_ptr[s]; e < in_ptr[s + 1]; e++) {
        uint32_t j = in_delay ? (uint32_t)in_delay[e] - c.dmin : 0;
        cnt[(uint64_t)j * c.n + s] += 1;
    }
}

__global__ __launch_bounds__(kBlock) void k_csr_fill(ConnArgs c, const uint64_t *in_ptr,
                                                    const uint32_t *in_col, const float *in_w,
                                                    const uint8_t *in_delay,
                                                    const uint64_t *row_ptr, int2 *syn)
{
    const uint32_t s = blockIdx.x * kBlock + threadIdx.x;
    if (s >= c.n) return;
    uint32_t fill[kMaxLists];
    for (uint32_t j = 0; j < c.lists; j++) fill[j] = 0;
    for (uint64_t e = in_ptr[s]; e < in_ptr[s + 1]; e++) {
        uint32_t j = in_delay ? (uint32_t)in_delay[e] - c.dmin : 0;
        uint64_t piece = (uint64_t)j * c.n + s;
        syn[row_ptr[piece] + fill[j]] = make_int2((int)in_col[e], weight_bits(c, in_w[e]));
        fill[j] += 1;
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

// ------------------------------------------------------------------ sort
// Every piece is sorted by (target, weight bits).  Pieces of up to
// kSmallSort synapses: one wave each, rank by counting; longer pieces are
// listed for a block-wide bitonic sort in LDS.
constexpr uint32_t kSmallSort = 256;

__global__ __launch_bounds__(kBlock) void k_sort_small(const uint64_t *row_ptr, int2 *syn, uint64_t m,
                                                      uint32_t *large, uint32_t *n_large)
{
    __shared__ uint64_t keys[kBlock / kWave][kSmallSort];
    const uint32_t lane = lane_id(), w = threadIdx.x / kWave;
    for (uint64_t b0 = (uint64_t)blockIdx.x * (kBlock / kWave); b0 < m;
         b0 += (uint64_t)gridDim.x * (kBlock / kWave)) {
        const uint64_t piece = b0 + w;
        uint64_t beg = 0;
        uint32_t L = 0;
        if (piece < m) {
            beg = row_ptr[piece];
            uint64_t len = row_ptr[piece + 1] - beg;
            if (len > kSmallSort) {
                if (lane == 0) large[atomicAdd(n_large, 1u)] = (uint32_t)piece;
            } else {
                L = (uint32_t)len;
            }
        }
        if (L < 2) L = 0;
        for (uint32_t e = lane; e < L; e += kWave) keys[w][e] = pack(syn[beg + e]);
        __syncthreads();
        for (uint32_t e = lane; e < L; e += kWave) {
            const uint64_t k = keys[w][e];
            uint32_t r = 0;
            for (uint32_t q = 0; q < L; q++) {
                const uint64_t kq = keys[w][q];
                r += (kq < k) | ((kq == k) & (q < e));
            }
            syn[beg + r] = unpack(k);
        }
        __syncthreads();
    }
}

constexpr int kSortThreads = 1024;

__global__ __launch_bounds__(kSortThreads) void k_sort_large(const uint64_t *row_ptr, int2 *syn,
                                                            const uint32_t *large)
{
    extern __shared__ uint64_t sk[];
    const uint32_t piece = large[blockIdx.x];
    const uint64_t beg = row_ptr[piece];
    const uint32_t L = (uint32_t)(row_ptr[piece + 1] - beg);
    uint32_t P2 = 1;
    while (P2 < L) P2 <<= 1;
    for (uint32_t e = threadIdx.x; e < P2; e += kSortThreads)
        sk[e] = e < L ? pack(syn[beg + e]) : ~0ull;
    __syncthreads();
    for (uint32_t k = 2; k <= P2; k <<= 1) {
        for (uint32_t j = k >> 1; j > 0; j >>= 1) {
            for (uint32_t e = threadIdx.x; e < P2; e += kSortThreads) {
                const uint32_t x = e ^ j;
                if (x > e) {
                    const uint64_t a = sk[e], b = sk[x];
                    const bool up = (e & k) == 0;
                    if ((a > b) == up) {
                        sk[e] = b;
                        sk[x] = a;
                    }
                }
            }
            __syncthreads();
        }
    }
    for (uint32_t e = threadIdx.x; e < L; e += kSortThreads) syn[beg + e] = unpack(sk[e]);
}

// --------------------------------------------------------- bookkeeping

__global__ __launch_bounds__(kBlock) void k_out_degree(const uint64_t *row_ptr, uint32_t n,
                                                      uint32_t lists, uint32_t *outdeg)
{
    const uint32_t s = blockIdx.x * kBlock + threadIdx.x;
    if (s >= n) return;
    uint64_t d = 0;
    for (uint32_t j = 0; j < lists; j++) {
        const uint64_t r = (uint64_t)j * n + s;
        d += row_ptr[r + 1] - row_ptr[r];
    }
    outdeg[s] = (uint32_t)d;
}

// Per-target sum of |weight| over all in-synapses: exact in quantised units
// (fixed mode), or an upper bound in units of 2^-24 (fp32 mode: each term
// rounded up), used to size the accumulators.
__global__ __launch_bounds__(kBlock) void k_in_abs_sum(const int2 *syn, uint64_t nnz, int fixed,
                                                      unsigned long long *insum)
{
    for (uint64_t e = (uint64_t)blockIdx.x * kBlock + threadIdx.x; e < nnz;
         e += (uint64_t)gridDim.x * kBlock) {
        const int2 x = syn[e];
        unsigned long long q;
        if (fixed) {
            q = (unsigned long long)(x.y < 0 ? -(long long)x.y : (long long)x.y);
        } else {
            const float w = fabsf(__int_as_float(x.y));
            q = (unsigned long long)ceil(ldexp((double)w, 24));
        }
        atomicAdd(&insum[(uint32_t)x.x], q);
    }
}

// Sub-piece boundaries of target-sorted pieces: off[p*bounds + b] is the
// offset (from the piece start) of the first synapse with target >= b*width.
// Also the longest sub-piece (targets in [b*width, (b+1)*width)).
__global__ __launch_bounds__(kBlock) void k_piece_offsets(const uint64_t *row_ptr, const int2 *syn,
                                                         uint64_t pieces, uint32_t bounds,
                                                         uint32_t width, uint16_t *off,
                                                         uint32_t *max_sub)
{
    uint32_t mx = 0;
    for (uint64_t k = (uint64_t)blockIdx.x * kBlock + threadIdx.x; k < pieces * bounds;
         k += (uint64_t)gridDim.x * kBlock) {
        const uint64_t p = k / bounds;
        const uint32_t b = (uint32_t)(k % bounds);
        const uint64_t beg = row_ptr[p];
        const uint32_t L = (uint32_t)(row_ptr[p + 1] - beg);
        const uint64_t lo_t = (uint64_t)b * width, hi_t = lo_t + width;
        uint32_t lo = 0, hi = L;  // first index with target >= lo_t
        while (lo < hi) {
            const uint32_t mid = (lo + hi) >> 1;
            if ((uint64_t)(uint32_t)syn[beg + mid].x < lo_t) lo = mid + 1; else hi = mid;
        }
        const uint32_t first = lo;
        hi = L;  // first index with target >= hi_t
        while (lo < hi) {
            const uint32_t mid = (lo + hi) >> 1;
            if ((uint64_t)(uint32_t)syn[beg + mid].x < hi_t) lo = mid + 1; else hi = mid;
        }
        off[k] = (uint16_t)first;
        mx = lo - first > mx ? lo - first : mx;
    }
    for (int o = 32; o > 0; o >>= 1) {
        const uint32_t y = __shfl_xor(mx, o);
        mx = y > mx ? y : mx;
    }
    if (lane_id() == 0 && mx) atomicMax(max_sub, mx);
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

__global__ __launch_bounds__(kBlock) void k_export_lens(const uint64_t *row_ptr, uint32_t n,
                                                       uint32_t lists, const uint32_t *rows,
                                                       uint64_t n_rows, uint64_t *lens)
{
    const uint64_t k = (uint64_t)blockIdx.x * kBlock + threadIdx.x;
    if (k >= n_rows * lists) return;
    const uint64_t r = k / lists, j = k % lists;
    const uint64_t piece = j * n + rows[r];
    lens[k] = row_ptr[piece + 1] - row_ptr[piece];
}

__global__ __launch_bounds__(kBlock) void k_export_gather(const uint64_t *row_ptr, const int2 *syn,
                                                         uint32_t n, uint32_t lists, uint32_t dmin,
                                                         const uint32_t *rows,
                                                         const uint64_t *piece_off, uint32_t *col,
                                                         uint32_t *wbits, uint8_t *delay)
{
    const uint64_t k = blockIdx.x;  // (row r, list j) = (k / lists, k % lists)
    const uint64_t r = k / lists, j = k % lists;
    const uint64_t piece = j * n + rows[r];
    const uint64_t beg = row_ptr[piece], L = row_ptr[piece + 1] - beg;
    const uint64_t o = piece_off[k];
    for (uint64_t e = threadIdx.x; e < L; e += kBlock) {
        const int2 x = syn[beg + e];
        col[o + e] = (uint32_t)x.x;
        wbits[o + e] = (uint32_t)x.y;
        delay[o + e] = (uint8_t)(dmin + j);
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

hipError_t gen_count_rows(const ConnArgs &c, uint32_t *cnt, hipStream_t s)
{
    hipLaunchKernelGGL(k_gen_count_rows, dim3(c.n), dim3(kBlock), 0, s, c, cnt);
    return hipGetLastError();
}

hipError_t gen_fill_rows(const ConnArgs &c, const uint64_t *row_ptr, int2 *syn, hipStream_t s)
{
    hipLaunchKernelGGL(k_gen_fill_rows, dim3(c.n), dim3(kBlock), 0, s, c, row_ptr, syn);
    return hipGetLastError();
}

hipError_t gen_in_count(const ConnArgs &c, uint32_t *cnt, hipStream_t s)
{
    hipLaunchKernelGGL(k_gen_in_count, dim3(c.n), dim3(kBlock), 0, s, c, cnt);
    return hipGetLastError();
}

hipError_t gen_in_fill(const ConnArgs &c, const uint64_t *row_ptr, uint32_t *cursor, int2 *syn,
                       hipStream_t s)
{
    hipLaunchKernelGGL(k_gen_in_fill, dim3(c.n), dim3(kBlock), 0, s, c, row_ptr, cursor, syn);
    return hipGetLastError();
}

hipError_t csr_count(const ConnArgs &c, const uint64_t *in_ptr, const uint8_t *in_delay,
                     uint32_t *cnt, hipStream_t s)
{
    hipLaunchKernelGGL(k_csr_count, dim3(grid_for(c.n)), dim3(kBlock), 0, s, c, in_ptr, in_delay, cnt);
    return hipGetLastError();
}

hipError_t csr_fill(const ConnArgs &c, const uint64_t *in_ptr, const uint32_t *in_col,
                    const float *in_w, const uint8_t *in_delay, const uint64_t *row_ptr,
                    int2 *syn, hipStream_t s)
{
    hipLaunchKernelGGL(k_csr_fill, dim3(grid_for(c.n)), dim3(kBlock), 0, s, c, in_ptr, in_col, in_w,
                       in_delay, row_ptr, syn);
    return hipGetLastError();
}

size_t scan_scratch_elems(uint64_t m) { return (size_t)((m + kScanTile - 1) / kScanTile) + 1; }

hipError_t scan_counts(const uint32_t *cnt, uint64_t m, uint64_t *out, uint64_t *block_sums,
                       uint32_t *max_piece, hipStream_t s)
{
    const uint64_t nb = (m + kScanTile - 1) / kScanTile;
    if (nb == 0) {
        return hipMemsetAsync(out, 0, sizeof(uint64_t), s);
    }
    hipLaunchKernelGGL(k_scan1, dim3((uint32_t)nb), dim3(kBlock), 0, s, cnt, m, out, block_sums,
                       max_piece);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_scan2, dim3(1), dim3(kBlock), 0, s, block_sums, nb);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_scan3, dim3((uint32_t)nb), dim3(kBlock), 0, s, out, m, block_sums, nb);
    return hipGetLastError();
}

hipError_t sort_small_pieces(const uint64_t *row_ptr, int2 *syn, uint64_t m, uint32_t *large,
                             uint32_t *n_large, hipStream_t s)
{
    uint64_t g = (m + 3) / 4;
    if (g > 65536) g = 65536;
    if (g == 0) g = 1;
    hipLaunchKernelGGL(k_sort_small, dim3((uint32_t)g), dim3(kBlock), 0, s, row_ptr, syn, m, large,
                       n_large);
    return hipGetLastError();
}

hipError_t sort_large_pieces(const uint64_t *row_ptr, int2 *syn, const uint32_t *large,
                             uint32_t n_large, uint32_t pow2, hipStream_t s)
{
    if (!n_large) return hipSuccess;
    const size_t lds = (size_t)pow2 * sizeof(uint64_t);
    hipError_t e = hipFuncSetAttribute((const void *)k_sort_large,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_sort_large, dim3(n_large), dim3(kSortThreads), lds, s, row_ptr, syn, large);
    return hipGetLastError();
}

hipError_t out_degree(const uint64_t *row_ptr, uint32_t n, uint32_t lists, uint32_t *outdeg,
                      hipStream_t s)
{
    hipLaunchKernelGGL(k_out_degree, dim3(grid_for(n)), dim3(kBlock), 0, s, row_ptr, n, lists, outdeg);
    return hipGetLastError();
}

hipError_t in_abs_sum(const int2 *syn, uint64_t nnz, bool fixed, uint64_t *insum, hipStream_t s)
{
    if (!nnz) return hipSuccess;
    hipLaunchKernelGGL(k_in_abs_sum, dim3(grid_for(nnz, 65536)), dim3(kBlock), 0, s, syn, nnz,
                       fixed ? 1 : 0, (unsigned long long *)insum);
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

hipError_t piece_offsets(const uint64_t *row_ptr, const int2 *syn, uint64_t pieces, uint32_t bounds,
                         uint32_t width, uint16_t *off, uint32_t *max_sub, hipStream_t s)
{
    if (!pieces) return hipSuccess;
    hipLaunchKernelGGL(k_piece_offsets, dim3(grid_for(pieces * bounds, 1u << 22)), dim3(kBlock), 0, s,
                       row_ptr, syn, pieces, bounds, width, off, max_sub);
    return hipGetLastError();
}

hipError_t export_lens(const uint64_t *row_ptr, uint32_t n, uint32_t lists, const uint32_t *rows,
                       uint64_t n_rows, uint64_t *lens, hipStream_t s)
{
    hipLaunchKernelGGL(k_export_lens, dim3(grid_for(n_rows * lists)), dim3(kBlock), 0, s, row_ptr, n,
                       lists, rows, n_rows, lens);
    return hipGetLastError();
}

hipError_t export_gather(const uint64_t *row_ptr, const int2 *syn, uint32_t n, uint32_t lists,
                         uint32_t dmin, const uint32_t *rows, uint64_t n_rows,
                         const uint64_t *piece_off, uint32_t *col, uint32_t *wbits,
                         uint8_t *delay, hipStream_t s)
{
    const uint64_t pieces = n_rows * lists;
    if (!pieces) return hipSuccess;
    if (pieces > 0x7fffffffull) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_export_gather, dim3((uint32_t)pieces), dim3(kBlock), 0, s, row_ptr, syn, n,
                       lists, dmin, rows, piece_off, col, wbits, delay);
    return hipGetLastError();
}

}  // namespace spk
