/*
 * spk_oracle.h -- CPU oracle for the spike-transmission + neuron-update path.
 *
 * TEST INFRASTRUCTURE ONLY.  This is a plain, slow, single-threaded C
 * implementation of what the GPU library computes, written from the paper
 * (Bautembach, Oikonomidis, Argyros, "Multi-GPU SNN Simulation with Static
 * Load Balancing", arXiv 2102.04681).  Only the test suite, the smoke check
 * and the benchmark's CPU-baseline leg may load it.  It shares no code,
 * header, table or constant with the GPU library.
 *
 * Paper passages followed:
 *   Sec. III-A  neuron/synapse pools, sorted adjacency rows, a spike array
 *               per pending delay (IDs of spiking neurons are delivered
 *               'delay' steps later);
 *   Sec. III-B  connectivity descriptor "connect range1 to range2 with
 *               probability p";
 *   Sec. III-C  spike transmission: every spike is delivered to every
 *               neighbour in its adjacency row;
 *   Sec. IV-A   single precision + forward Euler integration;
 *   Sec. V      per-delay adjacency lists for per-synapse delays.
 * The paper gives no neuron equations, no RNG and no parameter values; the
 * readings used here (LIF form, operation order, RNG, refractory rule,
 * Poisson drive, fixed-point mode) are listed in the design notes and in
 * the comments of spk_oracle.c.
 */
#ifndef SPK_ORACLE_H
#define SPK_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { ORC_OK = 0, ORC_EINVAL = -1, ORC_ENOMEM = -2, ORC_EOVERFLOW = -4 };
enum { ORC_LIF = 0, ORC_SOURCE = 1 };
enum { ORC_CONN_BERNOULLI = 0, ORC_CONN_FIXED_OUT = 1, ORC_CONN_FIXED_IN = 2,
       ORC_CONN_EXPLICIT = 3 };
enum { ORC_ACC_F32 = 0, ORC_ACC_FIXED = 1 };
/* stream tags of the counter-based hash */
enum { ORC_TAG_CONN = 1, ORC_TAG_TGT = 2, ORC_TAG_SRC_E = 3, ORC_TAG_SRC_I = 4,
       ORC_TAG_W = 5, ORC_TAG_DELAY = 6, ORC_TAG_V0 = 7, ORC_TAG_POIS = 8,
       ORC_TAG_BERN = 9 };

typedef struct {
    uint64_t seed;
    uint32_t n;            /* neuron count */
    uint32_t neuron_kind;  /* ORC_LIF or ORC_SOURCE */
    double frac_exc;       /* excitatory = IDs [0, round(frac_exc*n)) */
    double dt_ms, tau_m_ms, t_ref_ms;
    float v_rest, v_th, v_reset, v0_lo, v0_hi, i_bias;
    uint32_t conn_kind;
    double p;              /* Bernoulli connection probability */
    uint32_t k_out;        /* fixed out-degree */
    uint32_t k_in_exc, k_in_inh; /* fixed in-degree per population */
    float w_exc, w_inh;    /* weight by source population */
    uint32_t w_uniform;    /* 1: per-synapse w = w_lo + (w_hi-w_lo)*u24 */
    float w_lo, w_hi;
    uint32_t delay_min, delay_max; /* steps, >= 1 */
    double ext_lambda;     /* Poisson drive: mean count per neuron per step */
    float ext_w;           /* weight of one external event */
    double src_rate_hz;    /* ORC_SOURCE firing rate */
    uint32_t acc_mode;     /* ORC_ACC_F32 or ORC_ACC_FIXED */
    int32_t fixed_shift;   /* S: weights quantised to round(w * 2^S) */
} orc_params;

/* Derived constants, exposed for tests. */
typedef struct {
    uint32_t n_exc;
    float k;               /* dt / tau_m rounded once to fp32 */
    uint32_t ref_steps;
    uint32_t ring;         /* input slots = delay_max + 1 */
    uint64_t conn_thr;     /* Bernoulli threshold on the high 32 hash bits */
    uint64_t src_thr;
    uint32_t pois_len;
    int32_t ext_wq, bias_q, w_exc_q, w_inh_q;
    uint64_t nnz;
    uint32_t max_row;
} orc_derived;

typedef struct orc_net orc_net;

/* SplitMix64 (Steele, Lea, Flood 2014): the output function applied to state z. */
uint64_t orc_splitmix64(uint64_t z);
/* Counter-based hash H(seed, tag, a, b) (connectivity, weights, delays, V0). */
uint64_t orc_hash(uint64_t seed, uint32_t tag, uint64_t a, uint64_t b);
/* Per-step draw of neuron i at step t (< 2^32): one mixer round over the
 * stream key and the counter t * 2^32 + i (Poisson drive, Bernoulli firing). */
uint64_t orc_hash_step(uint64_t seed, uint32_t tag, uint32_t i, uint32_t t);
/* Poisson CDF thresholds T_k (k = 0..len-1); returns len or <0 on error. */
int orc_poisson_table(double lambda, uint64_t *thr, int cap);

/* Create a network.  build_csr = 0 skips connectivity (rows can still be
 * generated one at a time with orc_row for Bernoulli / fixed out-degree). */
int orc_create(const orc_params *P, int build_csr, orc_net **out);
/* Create from an explicit CSR (rows need not be sorted; they are sorted). */
int orc_create_explicit(const orc_params *P, uint32_t n, const uint64_t *row_ptr,
                        const uint32_t *col, const float *w, const uint8_t *delay,
                        orc_net **out);
void orc_destroy(orc_net *net);
int orc_get_derived(const orc_net *net, orc_derived *out);
uint64_t orc_nnz(const orc_net *net);
int orc_get_csr(const orc_net *net, uint64_t *row_ptr, uint32_t *col, float *w,
                uint8_t *delay);
/* Canonical row s (sorted by target, delay, weight bits). */
int orc_row(orc_net *net, uint32_t s, uint32_t *tgt, float *w, uint8_t *delay,
            uint64_t cap, uint64_t *len);
/* Fixed in-degree networks: the in-synapses of target tgt in draw order
 * (source, weight, delay), generated on their own (no CSR needed). */
int orc_in_row(const orc_net *net, uint32_t tgt, uint32_t *src, float *w, uint8_t *delay,
               uint64_t cap, uint64_t *len);
/* Delivery definition: out[i] = sum over listed spikes s, over synapses
 * s->i whose delay equals 'delay' (0 = any delay), of w (double) and of the
 * quantised weight (int64).  Either output may be NULL. */
int orc_deliver(orc_net *net, const uint32_t *spikes, uint64_t n_spikes,
                uint32_t delay, double *out_f, int64_t *out_q);
/* Run n steps.  counts/events/delivered: n entries each (may be NULL):
 * spikes, synapses of the spikes emitted at the step, synapses whose spike
 * arrives at the step.  raster: IDs of every step ascending, concatenated;
 * offs: n+1 entries (may be NULL).  A network created without its CSR
 * (Bernoulli or fixed out-degree) generates the row of each spike when it
 * is delivered. */
int orc_run(orc_net *net, uint64_t n_steps, uint32_t *counts, uint64_t *events,
            uint64_t *delivered, uint32_t *raster, uint64_t raster_cap, uint64_t *offs);
/* Bernoulli networks: whether source s connects to tgt, and the weight and
 * delay that synapse has (drawn whether or not it exists). */
int orc_pair(const orc_net *net, uint32_t s, uint32_t tgt, int *connected, float *w,
             uint8_t *delay);
int orc_get_state(const orc_net *net, float *v, uint8_t *ref);
uint64_t orc_step_index(const orc_net *net);
/* The update of one neuron in isolation: state (v, ref) at the start of step
 * t, synaptic input (isyn_f in fp32 mode, isyn_q in fixed mode), neuron id i.
 * Writes the new state and whether it spiked. */
int orc_update_one(const orc_net *net, uint64_t t, uint32_t i, float v, uint8_t ref,
                   float isyn_f, int64_t isyn_q, float *v_out, uint8_t *ref_out,
                   int *spiked);
/* Per-target sum of |quantised weight| over in-synapses (for the overflow
 * guard); requires the CSR. */
int orc_in_abs_sum_q(const orc_net *net, int64_t *out);

#ifdef __cplusplus
}
#endif
#endif
