/*
 * spk.h -- C ABI of libspk: spike transmission fused with the neuron update,
 * for one AMD Instinct MI355X (gfx950).
 *
 * Method: Bautembach, Oikonomidis, Argyros, "Multi-GPU SNN Simulation with
 * Static Load Balancing" (arXiv 2102.04681).
 *   - Sec. III-A: neurons and synapses live in struct-of-arrays pools; the
 *     topology is an adjacency list with sorted rows; spiking neuron IDs go
 *     into one of 'delay' spike arrays and are delivered that many steps
 *     later.
 *   - Sec. III-B: the network is described by connectivity parameters and
 *     expanded on the GPU ("uploaded to the GPU where it is expanded").
 *   - Sec. III-C: every spike is delivered to all neighbours of its row.
 *   - Sec. IV-A: single-precision forward Euler integration.
 *   - Sec. V:    per-synapse delays (the paper proposes one adjacency list
 *                per delay; here every stored synapse carries its delay and
 *                an event is filed under its arrival step when its source
 *                fires -- the same deliveries).
 *
 * Conventions (all entry points):
 *   - Every function returns spk_status (0 = SPK_OK, negative = error) and
 *     never throws; spk_last_error() gives a message for the calling thread.
 *   - The library owns all device memory of a network (allocated at create,
 *     released by spk_destroy).  The caller owns every host buffer passed
 *     in and passes its length explicitly; host buffers are only read or
 *     written during the call.
 *   - All device work of a network is ordered on one HIP stream: the one
 *     given at creation (e.g. torch.cuda.current_stream().cuda_stream), or a
 *     stream the library creates when NULL is given.  spk_step is
 *     asynchronous; every spk_read_* / spk_export_* call synchronises that
 *     stream before returning.
 *   - A network is not thread-safe: calls on one network must not overlap.
 *   - Errors: SPK_EINVAL bad argument or parameter, SPK_ENOMEM device or host
 *     allocation failed, SPK_EHIP a HIP runtime error (message included),
 *     SPK_EOVERFLOW a capacity or fixed-point range would be exceeded,
 *     SPK_ESTATE call not valid in the network's current state.
 */
#ifndef SPK_H
#define SPK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPK_ABI_VERSION 5u
#define SPK_MAX_DELAY_LISTS 64u  /* delay_max - delay_min + 1 must not exceed this */
/* Device scratch of spk_deliver_noalloc, per device (bytes). */
#define SPK_NOALLOC_SCRATCH_BYTES (32ull << 20)

typedef enum {
    SPK_OK = 0,
    SPK_EINVAL = -1,
    SPK_ENOMEM = -2,
    SPK_EHIP = -3,
    SPK_EOVERFLOW = -4,
    SPK_ESTATE = -5
} spk_status;

enum { SPK_LIF = 0, SPK_SOURCE = 1 };
enum { SPK_CONN_BERNOULLI = 0, SPK_CONN_FIXED_OUT = 1, SPK_CONN_FIXED_IN = 2,
       SPK_CONN_EXPLICIT = 3 };
enum { SPK_ACC_F32 = 0, SPK_ACC_FIXED = 1 };
/* Delivery strategy (same results, different speed): AUTO picks from the
 * network's shape; DIRECT makes each target tile read its runs of the due
 * rows at arrival (best for one delay and long rows); BINNED reads every
 * fired row once, right after the spike, and files its events by (arrival
 * step, target tile) in pages that the tile drains at arrival.  BINNED needs
 * (delay_max - delay_min + 1) * tiles / 8 <= 2048. */
enum { SPK_DELIVERY_AUTO = 0, SPK_DELIVERY_DIRECT = 1, SPK_DELIVERY_BINNED = 2 };
/* Synapse storage (same results, different size): FULL keeps 8 bytes per
 * synapse (delay index and target in 32 bits, the 32-bit weight beside them);
 * COMPACT keeps 4 (delay index, target and a 2-bit weight class; the weight of
 * each class is held once), which needs a network with at most 4 distinct
 * weights: population weights (the paper's static models keep one weight per
 * source population, Sec. III-A), or an explicit adjacency with at most 4
 * distinct weights.  AUTO picks COMPACT whenever it applies. */
enum { SPK_FORMAT_AUTO = 0, SPK_FORMAT_FULL = 1, SPK_FORMAT_COMPACT = 2, SPK_FORMAT_PROCEDURAL = 3 };
/* PROCEDURAL (Sec. V, future work: procedural connectivity) stores no
 * synapses at all: the row of a neuron that fires is generated again from
 * the network's seed and parameters when its events are filed, the same
 * synapses the other formats store.  Generated fixed out-degree networks
 * only; binned delivery, steps run as graphs (SPK_EINVAL otherwise); each
 * fired row costs one hash per synapse in each of the 8 XCD groups instead
 * of 4 or 8 bytes per synapse read.  spk_stats_t.bytes_per_synapse is 0. */
/* How spk_step runs the steps (same results, different speed).  GRAPH: each
 * step is a tile kernel (+ push kernel for binned delivery), batches of steps
 * replayed from captured HIP graphs.  PERSISTENT: all steps of one spk_step
 * call in a single cooperative launch of one workgroup per compute unit that
 * keeps the neuron state in LDS and hands each step over through barriers
 * inside the kernel; it needs one tile per compute unit or fewer (n <= 2^21
 * on MI355X), direct delivery with a single delay, or binned delivery with
 * delay_max * tiles / 8 <= 2048.  AUTO takes PERSISTENT where it applies and
 * the device runs it (checked once at creation), else GRAPH; asking for
 * PERSISTENT where it does not apply is SPK_EINVAL at creation. */
enum { SPK_STEP_AUTO = 0, SPK_STEP_GRAPH = 1, SPK_STEP_PERSISTENT = 2 };

/* Network parameters (plain data).
 *
 * Neurons: IDs [0, n); excitatory = [0, round(frac_exc*n)), inhibitory = rest.
 *   SPK_LIF: delta-current leaky integrate-and-fire, forward Euler in fp32
 *     (Sec. IV-A), per step  V <- (V + k*(v_rest - V)) + I,  k = fp32(dt/tau),
 *     spike when V >= v_th, then V = v_reset and round(t_ref/dt) steps held
 *     at v_reset with arriving input dropped.  V0 ~ U[v0_lo, v0_hi).
 *   SPK_SOURCE: fires independently with probability src_rate_hz*dt per
 *     step; V integrates its input the same way (no threshold).
 * Connectivity (Sec. III-B): Bernoulli(p) per ordered pair; fixed out-degree
 *   k_out (uniform targets, with replacement); fixed in-degree k_in_exc from
 *   the excitatory and k_in_inh from the inhibitory range (with
 *   replacement); or explicit (spk_create_from_csr).  Self-connections are
 *   allowed.  Weight = w_exc / w_inh by source population, or per synapse
 *   w_lo + (w_hi-w_lo)*U[0,1) when w_uniform.  Delay (steps) uniform over
 *   [delay_min, delay_max], 1 <= delay_min <= delay_max <= 253, at most 64
 *   distinct delays.
 * Drive: ext_lambda > 0 adds K*ext_w per neuron and step, K ~ Poisson(lambda);
 *   i_bias is added every step.
 * Accumulation: SPK_ACC_F32 keeps fp32 weights and sums each neuron's input
 *   exactly (64-bit fixed point whose unit is chosen at creation so that every
 *   weight is an exact multiple), then rounds the sum once to fp32;
 *   SPK_ACC_FIXED quantises weights to round(w * 2^fixed_shift) and sums
 *   int32.  Both are deterministic and bit-reproducible.
 * Every random draw is a pure function of (seed, stream, coordinates) via a
 *   SplitMix64-based counter hash, so networks are reproducible exactly.
 * Capacities: max_steps bounds the per-step records (counts, events) and the
 *   total number of steps; raster_capacity bounds the recorded spike IDs
 *   (0 = no raster).  Limits: n <= 2^24, at most 65535 synapses per source
 *   row.
 * Tuning (environment, read at creation): SPK_TILES_PER_XCD caps the tiles
 *   per XCD group (1..256, default 32); SPK_PAGE_CAP sets the records per
 *   page of binned delivery (default: an equal share of 2 GiB);
 *   SPK_BATCH_STEPS caps the
 *   steps per batch (1..16, default 8; spk_stats_t.batch_steps);
 *   SPK_GEN_KEYS=0 makes the Bernoulli generator draw every row a second
 *   time to place it instead of keeping the first pass's synapses (the
 *   results are the same). */
typedef struct {
    uint32_t abi_version;      /* must be SPK_ABI_VERSION */
    uint32_t n;
    uint64_t seed;
    uint32_t neuron_kind;      /* SPK_LIF or SPK_SOURCE */
    uint32_t conn_kind;        /* SPK_CONN_* */
    double frac_exc;
    double dt_ms, tau_m_ms, t_ref_ms;
    float v_rest, v_th, v_reset, v0_lo, v0_hi, i_bias;
    double p;
    uint32_t k_out, k_in_exc, k_in_inh;
    uint32_t w_uniform;
    float w_exc, w_inh, w_lo, w_hi;
    uint32_t delay_min, delay_max;
    double ext_lambda;
    float ext_w;
    uint32_t acc_mode;         /* SPK_ACC_F32 or SPK_ACC_FIXED */
    double src_rate_hz;
    int32_t fixed_shift;       /* 0..30 */
    uint32_t delivery;         /* SPK_DELIVERY_*: how events reach their target tile */
    uint32_t syn_format;       /* SPK_FORMAT_*: synapse storage */
    uint32_t step_mode;        /* SPK_STEP_*: how steps are launched */
    uint64_t max_steps;        /* >= 1 */
    uint64_t raster_capacity;  /* spike IDs; 0 = no raster */
} spk_params;

typedef struct {
    uint64_t n, nnz, steps;
    uint64_t device_bytes;     /* device memory owned by the network */
    uint32_t n_exc, ref_steps, ring_slots, delay_lists;
    uint32_t max_row;          /* longest source row (synapses) */
    uint32_t pois_len;
    int32_t fixed_shift;       /* fixed mode: S; fp32 mode: the unit 2^-S64 of the exact sums */
    float k;
    double bytes_per_synapse;  /* synapse storage / nnz: 8 (FULL), 4 (COMPACT), 0 (PROCEDURAL) */
    uint32_t tile_width;       /* target neurons per tile (one workgroup each) */
    uint32_t tiles;
    uint32_t delivery;         /* SPK_DELIVERY_DIRECT or SPK_DELIVERY_BINNED as chosen */
    uint32_t page_cap;         /* binned delivery: records per page (beyond: global atomics) */
    uint32_t step_mode;        /* SPK_STEP_GRAPH or SPK_STEP_PERSISTENT as chosen */
    uint32_t batch_steps;      /* persistent kernel, binned delivery: steps run as
                                  one batch (tile phases back to back, then one filing pass);
                                  up to the smallest delay (at most 8, or SPK_BATCH_STEPS up
                                  to 16), 1 otherwise */
    /* Setup timing (Sec. IV-C): host wall time of the creating call, GPU time
     * (HIP events on the network's stream) of the connectivity generation
     * kernels (row counts, fill and regrouping; excludes allocation), and of the
     * accumulator-range pass (largest sum of |weights| into one neuron).
     * gen_ms is zero for networks made by spk_create_from_csr (rows are
     * uploaded and grouped there, not generated); range_ms is zero for fixed
     * in-degree networks with population weights, whose range is known
     * without a pass (every neuron has the same in-synapses' weights). */
    double setup_ms, gen_ms, range_ms;
} spk_stats_t;

typedef struct spk_net spk_net;

/* Fill *out with the parameters of workload `index` (0..4):
 *   0  1 000 LIF, Bernoulli p=0.02, w +0.27/-4.5 mV, delay 1, 1 000 steps
 *   1  250 000 LIF, p=0.02, weights x 80/(0.02 n), 10 000 steps
 *   2  100 000 LIF, in-degree 8 000 exc + 2 000 inh, J=0.1, g=5, delay 15,
 *      Poisson drive at twice threshold rate, 10 000 steps
 *   3  1 000 000 Bernoulli sources at rate_hz, dt 1 ms, fan-out 1 000,
 *      w ~ U[0,1e-3), 1 000 steps
 *   4  2 000 000 LIF, fan-out 1 500, weights x 80/1500, delays 1..20, 5 000 steps
 * driven != 0 adds an external Poisson drive at twice the threshold rate
 * (lambda = 2*(v_th-v_rest)*(dt/tau)/w_exc, ext_w = w_exc) to LIF workloads
 * that have none; without it workloads 0, 1 and 4 are silent.
 * rate_hz is used by workload 3 only.  Errors: SPK_EINVAL for a bad index. */
spk_status spk_preset(int index, int driven, double rate_hz, uint64_t seed, spk_params *out);

/* Create a network and generate its connectivity on the GPU (Sec. III-B).
 * stream: a hipStream_t, or NULL for a library-owned stream.  On success
 * *out owns all device memory; release with spk_destroy.  Errors:
 * SPK_EINVAL (parameters), SPK_ENOMEM, SPK_EHIP, SPK_EOVERFLOW (fixed-point
 * range: the sum of |quantised weights| into one neuron plus the largest
 * drive must fit in int32). */
spk_status spk_create(const spk_params *params, void *stream, spk_net **out);

/* Create a network from an explicit adjacency list (row per source neuron,
 * any order inside rows; Fig. 'adj').  row_ptr: n+1 entries, row_ptr[0]=0;
 * col, w: row_ptr[n] entries; delay: row_ptr[n] entries or NULL (= delay_min).
 * params->n and params->conn_kind are ignored.  Host buffers, read only
 * during the call. */
spk_status spk_create_from_csr(const spk_params *params, uint32_t n, const uint64_t *row_ptr,
                               const uint32_t *col, const float *w, const uint8_t *delay,
                               void *stream, spk_net **out);

/* Enqueue n_steps simulation steps on the network's stream (asynchronous).
 * Each step t: deliver every synapse whose spike is due at t (source spiked
 * at t - d for a synapse of delay d; Sec. III-A, III-C, V), update all
 * neurons, compact the spiking IDs into the spike list of step t, record.
 * Errors: SPK_EOVERFLOW if steps would exceed max_steps. */
spk_status spk_step(spk_net *net, uint64_t n_steps);

/* Wait for all enqueued work (the host waits once per call instead of
 * downloading spike counts every step as the paper's loop does, Sec. III-E,
 * IV-D).  Reports device-side flags: SPK_EOVERFLOW (raster capacity or
 * fixed-point range exceeded), SPK_EINVAL once after spk_deliver_noalloc
 * was given a spike ID >= n, and SPK_EHIP if a persistent launch stopped
 * early (a barrier wait exceeded its 10 s bound): the state is then
 * undefined. */
spk_status spk_sync(spk_net *net);

/* Per-step records for steps [t0, t0+n) (host output buffers of n entries,
 * written by the call; the call waits for enqueued work first): spike
 * counts |S(t)| (the spike arrays of Sec. III-A), synaptic events emitted
 * at t (sum of the out-degrees of the neurons that spiked at t: one event
 * per (spike, outgoing synapse), the unit of Sec. IV-A's throughput) and
 * synaptic events delivered at t (synapses whose spike arrived at t, the
 * delay of Sec. III-A, V applied); steps not run yet read as 0.  Errors:
 * SPK_EINVAL if t0 + n exceeds max_steps, or a null buffer with n > 0;
 * device flags as spk_sync. */
spk_status spk_read_spike_counts(spk_net *net, uint64_t t0, uint64_t n, uint32_t *out);
spk_status spk_read_events(spk_net *net, uint64_t t0, uint64_t n, uint64_t *out);
spk_status spk_read_delivered(spk_net *net, uint64_t t0, uint64_t n, uint64_t *out);

/* Spike raster of steps [t0, t0+n) (the IDs each step's spike array holds,
 * Sec. III-A): host buffers offs (n+1 entries, offs[0] = 0) and ids (cap
 * entries); IDs of each step ascending.  Requires raster_capacity > 0 at
 * creation.  Errors: SPK_EOVERFLOW if the raster capacity was exceeded
 * during the run or cap is too small, SPK_EINVAL if t0 + n exceeds the
 * steps run or offs is NULL, SPK_ESTATE if recording is off. */
spk_status spk_read_raster(spk_net *net, uint64_t t0, uint64_t n, uint64_t *offs,
                           uint32_t *ids, uint64_t cap);

/* The neuron pool's state after the steps run so far (Sec. III-A: the
 * per-neuron struct-of-arrays the update reads and writes): membrane
 * potentials (fp32) and refractory counters (steps left) into host buffers
 * of n entries; either may be NULL.  Waits for enqueued work first. */
spk_status spk_read_state(spk_net *net, float *v, uint8_t *ref);

/* Spike transmission alone (Sec. III-C): deliver the listed spikes (host
 * array of n_spikes IDs < n) through the synapses of delay `delay` (0 =
 * every delay) with the same kernels the simulation uses, into a scratch
 * input buffer (allocated and freed by the call) that is copied to the host
 * buffer out_f32 (fp32 mode) or out_i32 (fixed mode, units of
 * 2^-fixed_shift); n entries; the other output may be NULL.  Network state
 * is not changed.  Errors: SPK_EINVAL (ID >= n, bad delay, missing output),
 * SPK_ENOMEM, SPK_EHIP. */
spk_status spk_debug_deliver(spk_net *net, const uint32_t *spikes, uint64_t n_spikes,
                             uint32_t delay, float *out_f32, int32_t *out_i32);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the
 * delivery of spk_debug_deliver with the spike list (d_spikes, n_spikes IDs)
 * and the output (d_out: n floats in fp32 mode, n int32 in fixed mode, units
 * of 2^-fixed_shift) in the caller's device memory, enqueued on the
 * network's stream and not waited for.  The pages, fill counters and
 * overflow accumulators the delivery needs come from one fixed scratch area
 * per device (SPK_NOALLOC_SCRATCH_BYTES, a static device array the library
 * holds until the process ends, cleared by a kernel at the start of every
 * call); the call allocates nothing, frees nothing, uses no memset and does
 * not synchronise.  Every call on one device shares that area: calls that
 * overlap on one device (any network, any stream) race, so the caller
 * orders them (one stream, or events).  Networks with direct delivery need
 * no scratch.  Results equal spk_debug_deliver's.  Network state is not
 * changed.  Errors (returned at once): SPK_EINVAL (null output, bad delay,
 * n_spikes >= 2^30), SPK_EOVERFLOW (the network's tiles need more overflow
 * accumulators than the scratch holds: n rounded up to whole tiles x 8
 * (fp32) or 4 (fixed) bytes, plus pages, must fit), SPK_EHIP.  Spike IDs
 * >= n are not read through: they deliver nothing, and the next spk_sync
 * (or read) reports SPK_EINVAL once. */
spk_status spk_deliver_noalloc(spk_net *net, const uint32_t *d_spikes, uint64_t n_spikes, uint32_t delay,
                               void *d_out);

/* Export the adjacency-list rows (Sec. III-A, Fig. 'adj': all synapses of
 * the given source neurons; procedural networks generate them, Sec. V), each
 * row in canonical order (target, delay, weight bits).  Host buffers:
 * offs: n_rows+1 entries; col/delay and w (fp32 mode) or wq (fixed mode) of
 * cap entries; unused outputs may be NULL.  Errors: SPK_EOVERFLOW if cap is
 * too small, SPK_EINVAL for a row >= n. */
spk_status spk_export_rows(spk_net *net, const uint32_t *rows, uint64_t n_rows, uint64_t *offs,
                           uint32_t *col, float *w, int32_t *wq, uint8_t *delay, uint64_t cap);

/* The Poisson threshold table of the external drive (the benchmark models'
 * Poisson input, Sec. IV): thr[k] = floor(CDF(k) * 2^32), last entry 2^32;
 * *len entries (0 without drive) into the host buffer thr of cap entries.
 * Errors: SPK_EOVERFLOW if cap is too small. */
spk_status spk_poisson_table(spk_net *net, uint64_t *thr, uint32_t cap, uint32_t *len);

/* The network's derived configuration and setup timings (spk_stats_t
 * above; setup_ms is the creation time of Sec. IV-C) into *out. */
spk_status spk_stats(spk_net *net, spk_stats_t *out);

/* Kernel timing.  With profiling on, spk_step records HIP events on the
 * network's stream around every kernel it launches: in GRAPH mode it launches
 * each step's kernels directly (no graph) -- the tile kernel (delivery into
 * LDS + neuron update + spike list) and, for binned delivery, the push kernel
 * (the new spikes' events into arrival pages); in PERSISTENT mode the one
 * launch of each spk_step call.  spk_read_kernel_ms returns the summed
 * durations (ms) of push, tile and persistent launches, the number of steps
 * and the number of persistent launches since the last spk_set_profiling
 * call; outputs may be NULL. */
spk_status spk_set_profiling(spk_net *net, int on);
spk_status spk_read_kernel_ms(spk_net *net, double *push_ms, double *tile_ms, double *run_ms,
                              uint64_t *steps, uint64_t *run_launches);

/* Plain device-to-device copy of `bytes` bytes (multiple of 16) through the
 * library's streaming copy kernel on the network's stream, timed with HIP
 * events: used to calibrate HBM traffic counters.  *ms may be NULL. */
spk_status spk_hbm_copy(spk_net *net, uint64_t bytes, int reps, double *ms);

/* Plain streaming read of `bytes` bytes (multiple of 16) of a device buffer
 * the call allocates and fills first, `reps` times, on the network's stream,
 * timed with HIP events: the read bandwidth the synapse stream can reach.
 * *ms (summed over reps) may be NULL.  Errors: SPK_EINVAL, SPK_ENOMEM,
 * SPK_EHIP. */
spk_status spk_hbm_read(spk_net *net, uint64_t bytes, int reps, double *ms);

void spk_destroy(spk_net *net);                 /* NULL-safe */
const char *spk_last_error(void);               /* thread-local; never NULL */
uint32_t spk_abi_version(void);

#ifdef __cplusplus
}
#endif
#endif
