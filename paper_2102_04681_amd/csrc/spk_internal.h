// spk_internal.h -- declarations shared by the HIP kernels and the host
// runtime of libspk (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "spk.h"

namespace spk {

constexpr uint32_t kMaxLists = SPK_MAX_DELAY_LISTS;
constexpr int kWave = 64;

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
__host__ __device__ __forceinline__ uint32_t hash_hi32(uint64_t h) { return (uint32_t)(h >> 32); }
// integer in [0, n): multiply-shift of the high 32 bits (Lemire)
__host__ __device__ __forceinline__ uint32_t hash_range(uint64_t h, uint32_t n)
{
    return (uint32_t)(((uint64_t)hash_hi32(h) * (uint64_t)n) >> 32);
}

struct Keys {
    uint64_t conn, tgt, src_e, src_i, w, delay, v0, pois, bern;
};

// Connectivity generation parameters.
struct ConnArgs {
    uint32_t n, n_exc;
    uint32_t kind;          // SPK_CONN_*
    uint32_t lists;         // D = delay_max - delay_min + 1
    uint32_t dmin;
    uint32_t k_out, k_in_exc, k_in_inh;
    uint64_t conn_thr;      // Bernoulli: connect iff hi32 < conn_thr
    uint32_t w_uniform;
    float w_exc, w_inh, w_lo, w_hi;
    uint32_t fixed;         // store quantised weights
    float qscale;           // 2^fixed_shift
    Keys keys;
};

// Everything the update kernel needs about the neuron model.
struct ModelArgs {
    uint32_t n;
    uint32_t kind;          // SPK_LIF / SPK_SOURCE
    uint32_t fixed;
    int32_t shift;
    float k, v_rest, v_th, v_reset, i_bias, ext_w;
    int32_t ext_wq, bias_q;
    uint32_t ref_steps;
    uint32_t pois_len;      // 0 = no drive
    uint64_t src_thr;
    Keys keys;
};

struct NetDev {
    uint32_t n, lists, dmin, ring_slots, cap;
    const uint64_t *row_ptr;   // lists*n + 1: list j, source s -> row_ptr[j*n + s]
    const int2 *syn;           // {target, weight bits (fp32 or quantised int32)}
    const uint32_t *outdeg;    // n
    float *V;                  // n
    uint8_t *ref;              // n
    void *acc;                 // n: fp32 or int32 input of the current step
    uint32_t *ring;            // ring * cap spike IDs
    uint32_t *ring_count;      // ring
    uint32_t *counts;          // max_steps
    uint64_t *events;          // max_steps
    uint64_t *delivered;       // max_steps
    const uint64_t *pois;      // pois_len thresholds
    uint32_t *flags;           // bit 0: spike-list overflow, bit 1: raster overflow
    uint32_t *raster;          // raster_cap
    uint64_t *raster_offs;     // max_steps + 1
    uint64_t raster_cap;
};

// Delivery work description: spike lists of lists [list_lo, list_hi) due
// at step t, or a single debug spike list delivered through those lists.
struct DeliverArgs {
    NetDev net;
    uint32_t fixed;
    uint32_t bpp;              // 64-synapse column blocks per piece
    uint64_t t;
    uint32_t list_lo, list_hi;
    void *acc;                 // accumulation target
    const uint32_t *dbg_spikes;  // non-null: debug mode
    const uint32_t *dbg_count;
    uint64_t *delivered;       // per-step counter to add to, or null
    uint32_t *zero_count;      // ring_count slot to clear, or null
};

// kernels.hip -- launch wrappers (return the launch error)
hipError_t gen_count_rows(const ConnArgs &c, uint32_t *cnt, hipStream_t s);
hipError_t gen_fill_rows(const ConnArgs &c, const uint64_t *row_ptr, int2 *syn, hipStream_t s);
hipError_t gen_in_count(const ConnArgs &c, uint32_t *cnt, hipStream_t s);
hipError_t gen_in_fill(const ConnArgs &c, const uint64_t *row_ptr, uint32_t *cursor, int2 *syn,
                       hipStream_t s);
hipError_t csr_count(const ConnArgs &c, const uint64_t *in_ptr, const uint8_t *in_delay,
                     uint32_t *cnt, hipStream_t s);
hipError_t csr_fill(const ConnArgs &c, const uint64_t *in_ptr, const uint32_t *in_col,
                    const float *in_w, const uint8_t *in_delay, const uint64_t *row_ptr,
                    int2 *syn, hipStream_t s);
hipError_t scan_counts(const uint32_t *cnt, uint64_t m, uint64_t *out, uint64_t *block_sums,
                       uint32_t *max_piece, hipStream_t s);
size_t scan_scratch_elems(uint64_t m);
hipError_t sort_small_pieces(const uint64_t *row_ptr, int2 *syn, uint64_t m, uint32_t *large,
                             uint32_t *n_large, hipStream_t s);
hipError_t sort_large_pieces(const uint64_t *row_ptr, int2 *syn, const uint32_t *large,
                             uint32_t n_large, uint32_t pow2, hipStream_t s);
hipError_t out_degree(const uint64_t *row_ptr, uint32_t n, uint32_t lists, uint32_t *outdeg,
                      hipStream_t s);
hipError_t in_abs_sum(const int2 *syn, uint64_t nnz, uint64_t *insum, hipStream_t s);
hipError_t max_u64(const uint64_t *x, uint64_t m, uint64_t *out, hipStream_t s);
hipError_t init_state(const ModelArgs &m, float v0_lo, float v0_hi, float *V, uint8_t *ref,
                      hipStream_t s);
hipError_t deliver(const DeliverArgs &a, int grid, hipStream_t s);
hipError_t update(const ModelArgs &m, const NetDev &net, uint64_t t, hipStream_t s);
hipError_t record(const NetDev &net, uint64_t t, hipStream_t s);
hipError_t export_lens(const uint64_t *row_ptr, uint32_t n, uint32_t lists, const uint32_t *rows,
                       uint64_t n_rows, uint64_t *lens, hipStream_t s);
hipError_t export_gather(const uint64_t *row_ptr, const int2 *syn, uint32_t n, uint32_t lists,
                         uint32_t dmin, const uint32_t *rows, uint64_t n_rows,
                         const uint64_t *piece_off, uint32_t *col, uint32_t *wbits,
                         uint8_t *delay, hipStream_t s);
hipError_t stream_copy(const void *src, void *dst, uint64_t bytes, hipStream_t s);
int deliver_grid();

}  // namespace spk
