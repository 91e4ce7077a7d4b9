// spk_internal.h -- declarations shared by the HIP kernels and the host
// runtime of libspk (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "spk.h"

namespace spk {

constexpr uint32_t kMaxLists = SPK_MAX_DELAY_LISTS;
constexpr int kWave = 64;
constexpr uint32_t kGroups = 8;        // one target group per XCD (blockIdx % 8 == XCD)
constexpr uint32_t kMaxTileW = 8192;   // neurons per tile (LDS accumulators + spike list)
constexpr uint32_t kTileCntBits = 14;  // a tile's spike count (<= kMaxTileW) in a progress word
constexpr uint32_t kMaxT8 = 256;       // tiles per group
constexpr uint32_t kMaxTiles = kGroups * kMaxT8;
constexpr uint32_t kMaxBuckets = 2048; // (delay, tile) buckets of one group in the push kernel
constexpr uint32_t kMaxRow = 65535;    // synapses per source row (16-bit run offsets)
constexpr uint32_t kOnceMaxB = 4992;   // (delay, tile) buckets of the procedural rows-once push
// Two synapse formats.  Full: int2 {j << 24 | target, weight bits}.  Compact
// (networks with at most kMaxClasses distinct weights, e.g. one weight per
// source population, as in the paper's static models): u32
// {class << 30 | j << 24 | target}, the weight taken from a table.  The
// target needs at most 24 bits (n <= 2^24), the delay index j = d - dmin < 64.
constexpr uint32_t kTargetBits = 24;
constexpr uint32_t kTargetMask = (1u << kTargetBits) - 1u;
constexpr uint32_t kDelayMask = 0x3fu;
constexpr uint32_t kMaxClasses = 4;
constexpr uint32_t kClassShift = 30;
__host__ __device__ __forceinline__ uint32_t rec_target(uint32_t x) { return x & kTargetMask; }
__host__ __device__ __forceinline__ uint32_t rec_delay(uint32_t x) { return (x >> kTargetBits) & kDelayMask; }
__host__ __device__ __forceinline__ uint32_t rec_class(uint32_t x) { return x >> kClassShift; }
__host__ __device__ __forceinline__ uint32_t rec_key(int2 r) { return (uint32_t)r.x; }
__host__ __device__ __forceinline__ uint32_t rec_key(uint32_t r) { return r; }

// Device flag bits of a network (StepArgs::flags): bit 1 the raster capacity
// was exceeded, bit 2 a persistent launch stopped early, bit 3 a spike ID
// given for debug delivery was out of range.
constexpr uint32_t kFlagBadSpike = 8u;

// A compact page record (u16): class << 13 | local target (W <= 8192).
constexpr uint32_t kPageClassShift = 13;
constexpr uint32_t kPageLocalMask = (1u << kPageClassShift) - 1u;

// Stream tags of the counter-based hash: one independent stream per kind of
// random decision (connection, target, source, weight, delay, initial V,
// Poisson drive, Bernoulli firing).
enum Tag : uint32_t {
    TAG_CONN = 1, TAG_TGT = 2, TAG_SRC_E = 3, TAG_SRC_I = 4, TAG_W = 5,
    TAG_DELAY = 6, TAG_V0 = 7, TAG_POIS = 8, TAG_BERN = 9
};

// SplitMix64 output function (Steele, Lea & Flood, OOPSLA 2014): add the
// golden gamma, two xor-shift-multiply rounds, final xor-shift.
__host__ __device__ __forceinline__ uint64_t mix64(uint64_t z)
{
    z += 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// H(seed, tag, a, b) = mix(mix(mix(mix(seed) ^ tag) ^ a) ^ b).  The first two
// rounds depend only on (seed, tag) and are precomputed on the host as a
// stream key; kernels finish with key_hash(key, a, b).
__host__ __device__ __forceinline__ uint64_t stream_key(uint64_t seed, uint32_t tag)
{
    return mix64(mix64(seed) ^ (uint64_t)tag);
}
__host__ __device__ __forceinline__ uint64_t key_hash(uint64_t key, uint64_t a, uint64_t b)
{
    return mix64(mix64(key ^ a) ^ b);
}
// Per-step draws of neuron i at step t (Poisson drive, Bernoulli firing):
// one round over the stream key and the packed counter t * 2^32 + i.
__host__ __device__ __forceinline__ uint64_t step_hash(uint64_t key, uint32_t i, uint64_t t)
{
    return mix64(key ^ ((t << 32) | (uint64_t)i));
}
__host__ __device__ __forceinline__ uint32_t hash_hi32(uint64_t h) { return (uint32_t)(h >> 32); }
// integer in [0, n): multiply-shift of the high 32 bits (Lemire)
__host__ __device__ __forceinline__ uint32_t hash_range(uint64_t h, uint32_t n)
{
    return (uint32_t)(((uint64_t)hash_hi32(h) * (uint64_t)n) >> 32);
}

struct Keys {
    uint64_t conn, tgt, src_e, src_i, w, delay, v0, pois, bern;
};

// Target tiling.  Tile k covers neurons [k*W, (k+1)*W); group x (one per
// XCD) covers tiles [x*T8, (x+1)*T8), i.e. neurons [x*Gw, (x+1)*Gw).
struct Tiling {
    uint32_t W, logW;   // tile width, a power of two
    uint32_t T8;        // tiles per group
    uint32_t T;         // tiles = 8 * T8
    uint32_t Gw;        // group width = T8 * W
    uint32_t T8inv;     // ceil(2^32 / T8) (0 when T8 = 1): x / T8 by one high multiply
};

// Where the runs of one source row start, per XCD group (binned delivery):
// group x owns [start + (x ? gend[x-1] : 0), start + gend[x]); gend[7] is the
// row length.  Inside group x's run the synapses of the smallest delay come
// first, up to start + dend[x].  One cache line per row.
struct alignas(64) RowDesc {
    uint64_t start;
    uint16_t gend[kGroups];
    uint16_t dend[kGroups];
    uint64_t spare[3];
};
static_assert(sizeof(RowDesc) == 64, "one row descriptor is 64 bytes");

// Connectivity generation parameters.
struct ConnArgs {
    uint32_t n, n_exc;
    uint32_t kind;          // SPK_CONN_*
    uint32_t lists;         // delay_max - delay_min + 1
    uint32_t dmin;
    uint32_t k_out, k_in_exc, k_in_inh;
    uint64_t conn_thr;      // Bernoulli: connect iff hi32 < conn_thr
    uint32_t w_uniform;
    float w_exc, w_inh, w_lo, w_hi;
    uint32_t fixed;         // store quantised weights
    float qscale;           // 2^fixed_shift
    uint32_t compact;       // write u32 records; generated rows: class = source population
                            // (0 exc, 1 inh); explicit rows: class k where cls_w[k] = weight bits
    uint32_t cls_w[kMaxClasses];
    Keys keys;
    Tiling tl;
};

// Where a bucketing pass writes the tile boundaries of every row: per-tile
// starts (direct delivery, T+1 per row) or per-group descriptors (binned).
struct RowIndex {
    uint16_t *toff;         // n * (T+1) or null
    RowDesc *desc;          // n or null
};

// Neuron model constants for the update.
struct ModelArgs {
    uint32_t n;
    uint32_t kind;          // SPK_LIF / SPK_SOURCE
    uint32_t fixed;         // 1: int32 accumulators in units of 2^-shift
    int32_t shift;
    int32_t shift64;        // fp32 mode: int64 accumulators in units of 2^-shift64
    float k, v_rest, v_th, v_reset, i_bias, ext_w;
    int32_t ext_wq, bias_q;
    uint32_t ref_steps;
    uint32_t pois_len;      // 0 = no drive
    uint64_t src_thr;
    Keys keys;
};

// Procedural connectivity (fixed out-degree networks whose synapses are
// generated again when their source fires, never stored): what the synapse
// draw needs beyond the stream keys.
struct ProcArgs {
    uint32_t k_out, n_exc, w_uniform;
    uint32_t once;          // rows generated once by one of pg1 push blocks (pages across XCDs)
    float w_lo, w_hi, w_exc, w_inh;
    float qscale;           // 2^fixed_shift (fixed mode)
};

// Everything the step kernels touch.
struct StepArgs {
    ModelArgs m;
    Tiling tl;
    uint32_t n, lists, dmin;
    uint32_t direct;             // 1: tiles read their runs of the due rows (one delay)
    uint32_t compact;            // 1: u32 synapses and u16 page records, weights from wval
    uint32_t proc;               // 1: procedural synapses (binned delivery; no rows stored)
    ProcArgs pr;
    int64_t wval[kMaxClasses];   // compact: weight of each class in accumulator units
    const uint64_t *row_ptr;     // n + 1
    const int2 *syn;             // full: {j << 24 | target, weight bits (fp32 or quantised int32)}
    const uint32_t *syn32;       // compact: class << 30 | j << 24 | target
    const RowDesc *desc;         // binned: n
    const uint16_t *toff;        // direct: T + 1 per row
    const uint32_t *outdeg;      // n
    float *V;                    // n
    uint8_t *ref;                // n
    // spike lists: one segment of W IDs per (slot, tile) and its count
    uint32_t spk_slots;
    uint32_t *spk_ids;           // spk_slots * T * W
    uint32_t *spk_cnt;           // spk_slots * T
    uint32_t *counts8;           // max_steps * 8
    uint64_t *events8;           // max_steps * 8: events emitted per group
    uint64_t *delivered8;        // max_steps * 8: events delivered per group
    // binned delivery: pages of {local target, weight bits} records, one per
    // (group x, push block g1, arrival slot, tile of the group), each owned by
    // its push block; fill counters in the same order
    int2 *pages;                 // full records {local target, weight bits}
    uint16_t *pages16;           // compact records class << 13 | local target
    uint32_t *pfill;
    uint32_t page_cap;           // records per page
    uint32_t pslots;             // arrival slots (delay_max)
    uint32_t pg1;                // push blocks per group
    void *acc_ovf;               // pslots * T * W accumulators for page overflow (int64 or int32)
    uint32_t *ovf_flag;          // pslots * T
    const uint64_t *pois;        // pois_len thresholds
    const uint16_t *pois_guide;  // 256: first k with T_k > b * 2^24
    uint32_t *flags;             // bit 1: raster overflow
    uint32_t *raster;
    uint64_t *raster_offs;       // max_steps + 1
    uint64_t raster_cap;
    const uint64_t *t_base;      // device step counter (steps completed before this batch)
    // debug delivery: deliver this spike list (only delay index dbg_j, or
    // every delay when dbg_j < 0) into dbg_out, no update
    const uint32_t *dbg_spikes;
    uint32_t dbg_n;
    int32_t dbg_j;
    void *dbg_out;
};

// Persistent step kernel (spk_run.hip): one cooperative launch of R
// workgroups per XCD runs many steps.  Control words, zeroed before every
// launch; each counter sits on its own 128-byte line.
constexpr uint32_t kCtlStride = 32;
constexpr uint32_t kRunMaxR = 32;          // workgroups per XCD (one per compute unit)
constexpr uint32_t kRunMaxFill = 2048;     // pages per push block: arrival slots x tiles of a group
constexpr uint32_t kRunMaxD = 16;          // steps per batch (binned delivery)
constexpr uint32_t kRunMaxBuckets = 1024;  // (arrival offset, tile) buckets of a push block
// Tile progress words lie 4 KB apart: every workgroup polls all of them, and
// spread over memory channels the polls queue less (measured: 35.5 -> 35.1 us
// per step on the 3e9-synapse network, 6.18 -> 5.99 on the delay-15 one).
constexpr uint32_t kTileWordStride = 1024;
constexpr uint32_t kRunAbortTimeout = 1u;  // a barrier wait gave up
constexpr uint32_t kRunAbortPlacement = 2u;  // workgroups not spread R per XCD: nothing was run
struct RunCtl {
    uint32_t ticket[kGroups * kCtlStride];  // workgroups placed on each XCD
    uint32_t gx[kGroups * kCtlStride];      // grid barrier: arrivals per XCD
    uint32_t pushp[kGroups * kRunMaxR];     // binned: push phases finished, per push block
    // binned: per batch parity and tile (kTileWordStride words apart), the batch published
    // (epoch in bits kTileCntBits and up) with, for a one-step batch, the
    // tile's spike count of that step (bits below)
    uint32_t tilep[2][kGroups * kRunMaxR * kTileWordStride];
    uint32_t start, pad0[kCtlStride - 1];   // placement barrier
    uint32_t gcnt, pad1[kCtlStride - 1];    // grid barrier: XCDs complete
    // grid barrier: the released epoch, one copy per XCD (kTileWordStride
    // words apart), each polled by the XCD's workgroups only (measured: 17.08
    // -> 16.96 us per step on the 250,000-neuron network, 79.6 -> 79.3 on the
    // 1e6-source one)
    uint32_t gen[kGroups * kTileWordStride];
    uint32_t abort_flag, pad3[kCtlStride - 1];
};
struct RunArgs {
    StepArgs s;
    RunCtl *ctl;
    uint64_t t0, n_steps;   // steps [t0, t0 + n_steps)
    uint32_t R;             // workgroups per XCD
    uint32_t D;             // binned delivery: steps per batch (1 .. min(d_min, kRunMaxD))
};

// spk_gen.hip -- connectivity expansion
// hist: optional (Bernoulli rows), n * (T + 2 * kGroups) u16 bucket counts
// kept for gen_fill_rows, which then need not count the rows again; keys
// (with hist): n * cap u32, the first cap synapses of every row kept as
// (delay index << 24 | target), so that gen_fill_rows need not draw the rows
// again either (valid where no row is longer than cap).
hipError_t gen_count_rows(const ConnArgs &c, uint32_t *cnt, uint16_t *hist, uint32_t *keys, uint32_t cap,
                          hipStream_t s);
hipError_t gen_fill_rows(const ConnArgs &c, const uint64_t *row_ptr, void *syn, RowIndex ix,
                         const uint16_t *hist, const uint32_t *keys, uint32_t cap, hipStream_t s);
hipError_t gen_in_count(const ConnArgs &c, uint32_t *cnt, hipStream_t s);
hipError_t gen_in_fill(const ConnArgs &c, const uint64_t *row_ptr, uint32_t *cursor, void *syn,
                       hipStream_t s);
hipError_t csr_fill(const ConnArgs &c, uint64_t nnz, const uint32_t *in_col, const float *in_w,
                    const uint8_t *in_delay, void *syn, hipStream_t s);
hipError_t bucket_rows(const ConnArgs &c, const uint64_t *row_ptr, const void *src, void *dst,
                       RowIndex ix, hipStream_t s);
hipError_t scan_counts(const uint32_t *cnt, uint64_t m, uint64_t *out, uint64_t *block_sums,
                       uint32_t *max_count, hipStream_t s);
size_t scan_scratch_elems(uint64_t m);
hipError_t out_degree(const uint64_t *row_ptr, uint32_t n, uint32_t *outdeg, hipStream_t s);
// Per-class values of compact synapses: the stored weight bits (fp32, or the
// quantised int32 in fixed mode) and the |weight| term of in_abs_sum.
struct ClassTab {
    uint32_t bits[kMaxClasses];
    uint64_t abs[kMaxClasses];
};
hipError_t in_abs_sum(const void *syn, uint64_t nnz, bool fixed, bool compact, const ClassTab &tab,
                      uint64_t *insum, hipStream_t s);
hipError_t max_u64(const uint64_t *x, uint64_t m, uint64_t *out, hipStream_t s);
// Fixed out-degree networks with population weights: the largest in_abs_sum
// from the synapses drawn again and filed by target tile (no atomic per
// synapse).  fo_count: per (block of sources, tile) reservations base
// (fo_blocks(n) x T) and tile totals (T, zero on entry); fo_file: entries
// (class << 14 | neuron in tile) at tile_start[tile] + reservation; fo_max:
// one block per tile, the largest sum into *out (zero on entry).
uint32_t fo_blocks(uint32_t n);
hipError_t fo_count(const ConnArgs &c, uint32_t *base, uint32_t *tile_total, hipStream_t s);
hipError_t fo_file(const ConnArgs &c, const uint32_t *base, const uint64_t *tile_start, uint16_t *entries,
                   hipStream_t s);
hipError_t fo_max(const ConnArgs &c, const uint64_t *tile_start, const uint16_t *entries, const ClassTab &tab,
                  uint64_t *out, hipStream_t s);
// Bernoulli networks: the largest in_abs_sum over neurons, by evaluating the
// pair predicate per target (no atomic per synapse); *out must be zero on
// entry, and so must insum (n entries), needed when bern_src_ranges(n) > 1.
uint32_t bern_src_ranges(uint32_t n);
hipError_t bern_in_abs_max(const ConnArgs &c, uint64_t *out, uint64_t *insum, hipStream_t s);
hipError_t init_state(const ModelArgs &m, float v0_lo, float v0_hi, float *V, uint8_t *ref,
                      hipStream_t s);
hipError_t export_gather(const uint64_t *row_ptr, const void *syn, bool compact, const ClassTab &tab,
                         uint32_t dmin, const uint32_t *rows, uint64_t n_rows, const uint64_t *out_off,
                         uint32_t *col, uint32_t *wbits, uint8_t *delay, hipStream_t s);
int cu_count();

// spk_step.hip -- one simulation step = tile (+ push) (+ record); i = step
// index inside the current batch (t = *t_base + i), or explicit t when
// t_explicit >= 0.
hipError_t launch_tile(const StepArgs &a, uint32_t i, int64_t t_explicit, hipStream_t s);
hipError_t launch_push(const StepArgs &a, uint32_t i, int64_t t_explicit, hipStream_t s);
hipError_t launch_record(const StepArgs &a, uint32_t i, int64_t t_explicit, hipStream_t s);
hipError_t launch_advance(uint64_t *t_base, uint32_t steps, hipStream_t s);

// spk_proc.hip -- procedural connectivity: the push of a step with every
// fired row generated again (binned delivery), the rows of given sources as
// generated (export), and the per-target sum of |weight| terms (range pass,
// one atomic per generated synapse).
hipError_t launch_push_proc(const StepArgs &a, uint32_t i, int64_t t_explicit, hipStream_t s);
hipError_t export_proc(const StepArgs &a, const ClassTab &tab, const uint32_t *rows, uint64_t n_rows,
                       const uint64_t *out_off, uint32_t *col, uint32_t *wbits, uint8_t *delay, hipStream_t s);
hipError_t proc_in_abs_sum(const StepArgs &a, uint64_t *insum, hipStream_t s);
hipError_t stream_copy(const void *src, void *dst, uint64_t bytes, hipStream_t s);
hipError_t stream_read(const void *src, uint64_t bytes, uint32_t *sink, hipStream_t s);
hipError_t zero_words(uint32_t *p, uint64_t n, hipStream_t s);
uint32_t push_blocks_per_group();

// spk_run.hip -- the persistent step kernel (all steps of a call in one launch)
bool run_supported(const StepArgs &a, uint32_t R);
bool run_batch_supported(const StepArgs &a, uint32_t D);  // steps per batch D is valid for this network
hipError_t launch_run(const RunArgs &ra, hipStream_t s);
hipError_t launch_run_batched(const RunArgs &ra, hipStream_t s);  // spk_run_batch.hip

}  // namespace spk
