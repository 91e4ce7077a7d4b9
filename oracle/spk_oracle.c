/*
 * spk_oracle.c -- CPU oracle (TEST INFRASTRUCTURE ONLY; see spk_oracle.h).
 *
 * Build: gcc -O2 -std=c99 -ffp-contract=off -fPIC -shared spk_oracle.c -lm
 * No -ffast-math and no FMA contraction: every fp32 operation below is one
 * IEEE-754 single-precision operation with round-to-nearest-even.
 *
 * What is computed, and where it comes from:
 *  - Connectivity (Sec. III-B): a descriptor says "connect every neuron of
 *    range1 to every neuron of range2 with probability p".  Here: Bernoulli
 *    (each ordered pair independently), fixed out-degree and fixed in-degree
 *    draws, or an explicit list.  Each draw is a pure function of a
 *    counter-based hash so that the GPU generator can reproduce it exactly.
 *  - Adjacency rows are kept sorted (Sec. III-A; Fig. 'adj'); the canonical
 *    order is (target, delay, weight bits).  Self-connections are allowed
 *    (Fig. 'adj' rows list their own neuron).
 *  - Step t (Sec. III-A, III-C): every neuron is updated; the spiking ones
 *    are collected; every spike is delivered to all neighbours in its row,
 *    arriving 'delay' steps later (a spike array per pending delay in the
 *    paper; here an input slot per pending step, which is equivalent).
 *  - Neuron model: the paper states fp32 forward Euler (Sec. IV-A) but no
 *    equation.  Reading: delta-current leaky integrate-and-fire,
 *        a = v_rest - V;  b = k*a;  c = V + b;  V = c + I   (k = dt/tau_m)
 *    each step rounded in fp32, threshold V >= v_th, reset to v_reset and
 *    ref_steps = round(t_ref/dt) refractory steps during which V is held at
 *    v_reset and arriving input is dropped.
 *  - Fixed-point accumulation mode (deterministic): weights quantised to
 *    wq = rint(w * 2^S) (int32), inputs summed exactly as integers, one
 *    conversion I = float(Iq) * 2^-S per neuron and step.
 */
#include "spk_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#define ORC_POIS_CAP 256

struct orc_net {
    orc_params P;
    orc_derived D;
    uint32_t dspan;        /* delay_max - delay_min + 1 */
    int have_csr;
    uint64_t *row_ptr;     /* n+1 */
    uint32_t *col;
    float *w;
    uint8_t *delay;
    int32_t *wq;           /* fixed mode only */
    float *V;
    uint8_t *ref;
    float *slot_f;         /* ring * n, fp32 mode */
    int64_t *slot_q;       /* ring * n, fixed mode */
    uint64_t *arrive;      /* ring: synapses whose spike arrives at each pending step */
    uint64_t pois_thr[ORC_POIS_CAP];
    uint64_t t;
};

/* ------------------------------------------------------------------ hash */

/* SplitMix64 output function (Steele, Lea, Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014): advance the state by the
 * golden gamma, then two xor-shift-multiply rounds and a final xor-shift. */
uint64_t orc_splitmix64(uint64_t z)
{
    z = z + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* H(seed, tag, a, b): chain the mixer over seed, stream tag and two
 * coordinates.  Used for every random decision of the model.  The chain up
 * to the first coordinate is the prefix of every draw that shares
 * (seed, tag, a), e.g. all synapses of one source row. */
static uint64_t hash_prefix(uint64_t seed, uint32_t tag, uint64_t a)
{
    uint64_t h = orc_splitmix64(seed);
    h = orc_splitmix64(h ^ (uint64_t)tag);
    return orc_splitmix64(h ^ a);
}

uint64_t orc_hash(uint64_t seed, uint32_t tag, uint64_t a, uint64_t b)
{
    return orc_splitmix64(hash_prefix(seed, tag, a) ^ b);
}

/* Per-step draws (Poisson drive, Bernoulli firing of neuron i at step t):
 * one mixer round over the stream key and the packed counter (t, i),
 *     H_step(seed, tag, i, t) = mix(key(seed, tag) ^ (t * 2^32 + i)),
 * key(seed, tag) = mix(mix(seed) ^ tag); distinct (i, t) give distinct
 * counters and hence distinct outputs. */
uint64_t orc_hash_step(uint64_t seed, uint32_t tag, uint32_t i, uint32_t t)
{
    uint64_t key = orc_splitmix64(orc_splitmix64(seed) ^ (uint64_t)tag);
    return orc_splitmix64(key ^ (((uint64_t)t << 32) | (uint64_t)i));
}

static uint32_t hi32(uint64_t h) { return (uint32_t)(h >> 32); }

/* uniform in [0,1): the top 24 bits scaled by 2^-24 (exact in fp32) */
static float u24(uint64_t h) { return (float)(uint32_t)(h >> 40) * (1.0f / 16777216.0f); }

/* integer in [0, n): Lemire's multiply-shift of the high 32 bits */
static uint32_t range_n(uint64_t h, uint32_t n)
{
    return (uint32_t)(((uint64_t)hi32(h) * (uint64_t)n) >> 32);
}

/* threshold on hi32 for an event of probability p: hi32 < floor(p * 2^32) */
static uint64_t prob_thr(double p)
{
    if (p <= 0.0) return 0;
    if (p >= 1.0) return 4294967296ull;
    return (uint64_t)floor(p * 4294967296.0);
}

/* ------------------------------------------------------ Poisson table */

/* Thresholds T_k = floor(CDF_lambda(k) * 2^32), CDF built in double from
 * the pmf recursion p_0 = e^-lambda, p_k = p_{k-1} * lambda / k.  The last
 * entry is 2^32 so that every 32-bit draw maps to some k:
 *     K = min { k : hi32(h) < T_k }. */
int orc_poisson_table(double lambda, uint64_t *thr, int cap)
{
    if (!(lambda > 0.0) || lambda > 100.0 || cap < 2) return ORC_EINVAL;
    double p = exp(-lambda);
    double cdf = p;
    int k = 0;
    for (;;) {
        double T = floor(cdf * 4294967296.0);
        if (T >= 4294967295.0 || k == cap - 1) {
            thr[k] = 4294967296ull;
            return k + 1;
        }
        thr[k] = (uint64_t)T;
        k = k + 1;
        p = (p * lambda) / (double)k;
        cdf = cdf + p;
    }
}

static uint32_t poisson_draw(const orc_net *net, uint64_t h)
{
    uint64_t x = hi32(h);
    uint32_t k = 0;
    while (!(x < net->pois_thr[k])) k++;
    return k;
}

/* ------------------------------------------------------------- derived */

static int quantise(float w, int S, int32_t *out)
{
    float x = rintf(ldexpf(w, S));
    if (!(fabsf(x) < 2147483648.0f)) return ORC_EOVERFLOW;
    *out = (int32_t)x;
    return ORC_OK;
}

static int derive(orc_net *net)
{
    const orc_params *P = &net->P;
    orc_derived *D = &net->D;
    if (P->n == 0 || P->n > 2000000000u) return ORC_EINVAL;
    if (!(P->dt_ms > 0.0) || !(P->tau_m_ms > 0.0) || P->t_ref_ms < 0.0) return ORC_EINVAL;
    if (P->delay_min < 1 || P->delay_max < P->delay_min || P->delay_max > 255) return ORC_EINVAL;
    if (P->frac_exc < 0.0 || P->frac_exc > 1.0) return ORC_EINVAL;
    if (P->neuron_kind > ORC_SOURCE || P->conn_kind > ORC_CONN_EXPLICIT) return ORC_EINVAL;
    if (P->acc_mode > ORC_ACC_FIXED) return ORC_EINVAL;
    D->n_exc = (uint32_t)llround(P->frac_exc * (double)P->n);
    D->k = (float)(P->dt_ms / P->tau_m_ms);
    long long rs = llround(P->t_ref_ms / P->dt_ms);
    if (rs < 0 || rs > 255) return ORC_EINVAL;
    D->ref_steps = (uint32_t)rs;
    D->ring = P->delay_max + 1;
    net->dspan = P->delay_max - P->delay_min + 1;
    if (P->p < 0.0 || P->p > 1.0) return ORC_EINVAL;
    D->conn_thr = prob_thr(P->p);
    D->src_thr = prob_thr(P->src_rate_hz * P->dt_ms * 1e-3);
    if (P->ext_lambda > 0.0) {
        int L = orc_poisson_table(P->ext_lambda, net->pois_thr, ORC_POIS_CAP);
        if (L < 0) return L;
        D->pois_len = (uint32_t)L;
    } else {
        D->pois_len = 0;
    }
    if (P->acc_mode == ORC_ACC_FIXED) {
        if (P->fixed_shift < 0 || P->fixed_shift > 30) return ORC_EINVAL;
        int S = P->fixed_shift;
        if (quantise(P->ext_w, S, &D->ext_wq) || quantise(P->i_bias, S, &D->bias_q) ||
            quantise(P->w_exc, S, &D->w_exc_q) || quantise(P->w_inh, S, &D->w_inh_q))
            return ORC_EOVERFLOW;
    }
    if (P->conn_kind == ORC_CONN_FIXED_IN &&
        ((P->k_in_exc > 0 && D->n_exc == 0) || (P->k_in_inh > 0 && D->n_exc == P->n)))
        return ORC_EINVAL;
    return ORC_OK;
}

/* ------------------------------------------------------------ synapses */

typedef struct {
    uint32_t tgt;
    uint8_t d;
    float w;
} orc_syn;

static uint32_t wbits(float w)
{
    uint32_t u;
    memcpy(&u, &w, 4);
    return u;
}

/* canonical order inside a row: target, then delay, then weight bits */
static int syn_cmp(const void *a, const void *b)
{
    const orc_syn *x = (const orc_syn *)a, *y = (const orc_syn *)b;
    if (x->tgt != y->tgt) return x->tgt < y->tgt ? -1 : 1;
    if (x->d != y->d) return x->d < y->d ? -1 : 1;
    uint32_t u = wbits(x->w), v = wbits(y->w);
    if (u != v) return u < v ? -1 : 1;
    return 0;
}

/* Weight of a synapse from source s: per synapse w_lo + (w_hi - w_lo) * u24
 * of its W-stream hash h (two fp32 operations), else the weight of the
 * source's population (Sec. III-A: the static models keep one weight per
 * population; h is not used). */
static float weight_of(const orc_net *net, uint32_t s, uint64_t h)
{
    const orc_params *P = &net->P;
    if (P->w_uniform) {
        float span = P->w_hi - P->w_lo;
        float t = span * u24(h);
        return P->w_lo + t;
    }
    return s < net->D.n_exc ? P->w_exc : P->w_inh;
}

/* Delay (steps) of a synapse from its DELAY-stream hash h: uniform over
 * [delay_min, delay_max] (h is not used for a single delay). */
static uint8_t delay_of(const orc_net *net, uint64_t h)
{
    if (net->dspan == 1) return (uint8_t)net->P.delay_min;
    return (uint8_t)(net->P.delay_min + range_n(h, net->dspan));
}

/* The same for the synapse drawn at coordinates (a, b) of the streams. */
static float syn_weight(const orc_net *net, uint32_t s, uint64_t a, uint64_t b)
{
    return weight_of(net, s, net->P.w_uniform ? orc_hash(net->P.seed, ORC_TAG_W, a, b) : 0);
}

static uint8_t syn_delay(const orc_net *net, uint64_t a, uint64_t b)
{
    return delay_of(net, net->dspan > 1 ? orc_hash(net->P.seed, ORC_TAG_DELAY, a, b) : 0);
}

/* Generate the row of source s into buf (cap entries); Bernoulli and fixed
 * out-degree only.  sorted: put the row in canonical order (the stored
 * rows' order; fixed-point sums do not depend on it).  Returns the row
 * length, or -1 if cap is too small. */
static long long gen_row(const orc_net *net, uint32_t s, orc_syn *buf, uint64_t cap, int sorted)
{
    const orc_params *P = &net->P;
    uint64_t len = 0;
    if (P->conn_kind == ORC_CONN_BERNOULLI) {
        /* every ordered pair (s, tgt) independently, targets ascending */
        for (uint32_t tgt = 0; tgt < P->n; tgt++) {
            if (!(hi32(orc_hash(P->seed, ORC_TAG_CONN, s, tgt)) < net->D.conn_thr)) continue;
            if (len >= cap) return -1;
            buf[len].tgt = tgt;
            buf[len].d = syn_delay(net, s, tgt);
            buf[len].w = syn_weight(net, s, s, tgt);
            len++;
        }
    } else if (P->conn_kind == ORC_CONN_FIXED_OUT) {
        /* k_out independent uniform targets; duplicates are kept.  Draw j of
         * the row is H(seed, tag, s, j), finished from the row's prefixes. */
        if (P->k_out > cap) return -1;
        uint64_t pt = hash_prefix(P->seed, ORC_TAG_TGT, s);
        uint64_t pd = hash_prefix(P->seed, ORC_TAG_DELAY, s);
        uint64_t pw = hash_prefix(P->seed, ORC_TAG_W, s);
        for (uint32_t j = 0; j < P->k_out; j++) {
            buf[j].tgt = range_n(orc_splitmix64(pt ^ j), P->n);
            buf[j].d = delay_of(net, net->dspan > 1 ? orc_splitmix64(pd ^ j) : 0);
            buf[j].w = weight_of(net, s, P->w_uniform ? orc_splitmix64(pw ^ j) : 0);
        }
        len = P->k_out;
    } else {
        return -2;
    }
    if (sorted) qsort(buf, (size_t)len, sizeof(orc_syn), syn_cmp);
    return (long long)len;
}

static int alloc_csr(orc_net *net, uint64_t nnz)
{
    net->D.nnz = nnz;
    size_t m = nnz ? (size_t)nnz : 1;
    net->col = (uint32_t *)malloc(m * sizeof(uint32_t));
    net->w = (float *)malloc(m * sizeof(float));
    net->delay = (uint8_t *)malloc(m);
    if (!net->col || !net->w || !net->delay) return ORC_ENOMEM;
    return ORC_OK;
}

/* Bernoulli / fixed out-degree: concatenate the generated rows. */
static int build_rows(orc_net *net)
{
    const orc_params *P = &net->P;
    uint32_t n = P->n;
    uint64_t cap = P->conn_kind == ORC_CONN_BERNOULLI ? n : P->k_out;
    orc_syn *buf = (orc_syn *)malloc((size_t)(cap ? cap : 1) * sizeof(orc_syn));
    net->row_ptr = (uint64_t *)malloc(((size_t)n + 1) * sizeof(uint64_t));
    if (!buf || !net->row_ptr) { free(buf); return ORC_ENOMEM; }
    /* pass 1: lengths (a fixed out-degree row always has k_out entries) */
    net->row_ptr[0] = 0;
    for (uint32_t s = 0; s < n; s++) {
        long long L = P->conn_kind == ORC_CONN_FIXED_OUT ? (long long)P->k_out
                                                           : gen_row(net, s, buf, cap, 0);
        if (L < 0) { free(buf); return ORC_EINVAL; }
        net->row_ptr[s + 1] = net->row_ptr[s] + (uint64_t)L;
    }
    int rc = alloc_csr(net, net->row_ptr[n]);
    if (rc) { free(buf); return rc; }
    /* pass 2: fill */
    for (uint32_t s = 0; s < n; s++) {
        long long L = gen_row(net, s, buf, cap, 1);
        uint64_t o = net->row_ptr[s];
        for (long long e = 0; e < L; e++) {
            net->col[o + e] = buf[e].tgt;
            net->delay[o + e] = buf[e].d;
            net->w[o + e] = buf[e].w;
        }
    }
    free(buf);
    return ORC_OK;
}

/* Fixed in-degree: every target draws k_in_exc sources from the excitatory
 * range and k_in_inh from the inhibitory range (with replacement); the
 * synapses are then regrouped by source row (counting sort) and each row
 * is sorted canonically. */
/* Fixed in-degree (Sec. III-B): in-synapse j of target tgt.  The first
 * k_in_exc draw their source uniformly from the excitatory range, the rest
 * from the inhibitory range (with replacement). */
static uint32_t fixed_in_src(const orc_net *net, uint32_t tgt, uint32_t j)
{
    const orc_params *P = &net->P;
    uint32_t ne = net->D.n_exc, ni = P->n - ne;
    return j < P->k_in_exc
        ? range_n(orc_hash(P->seed, ORC_TAG_SRC_E, tgt, j), ne)
        : ne + range_n(orc_hash(P->seed, ORC_TAG_SRC_I, tgt, j - P->k_in_exc), ni);
}

static int build_fixed_in(orc_net *net)
{
    const orc_params *P = &net->P;
    uint32_t n = P->n;
    uint32_t kin = P->k_in_exc + P->k_in_inh;
    uint64_t nnz = (uint64_t)n * kin;
    uint64_t *cnt = (uint64_t *)calloc((size_t)n + 1, sizeof(uint64_t));
    net->row_ptr = (uint64_t *)malloc(((size_t)n + 1) * sizeof(uint64_t));
    if (!cnt || !net->row_ptr) { free(cnt); return ORC_ENOMEM; }
    for (uint32_t tgt = 0; tgt < n; tgt++)
        for (uint32_t j = 0; j < kin; j++) cnt[fixed_in_src(net, tgt, j)]++;
    net->row_ptr[0] = 0;
    for (uint32_t s = 0; s < n; s++) net->row_ptr[s + 1] = net->row_ptr[s] + cnt[s];
    int rc = alloc_csr(net, nnz);
    if (rc) { free(cnt); return rc; }
    for (uint32_t s = 0; s < n; s++) cnt[s] = net->row_ptr[s];
    for (uint32_t tgt = 0; tgt < n; tgt++)
        for (uint32_t j = 0; j < kin; j++) {
            uint32_t src = fixed_in_src(net, tgt, j);
            uint64_t o = cnt[src]++;
            net->col[o] = tgt;
            net->delay[o] = syn_delay(net, tgt, j);
            net->w[o] = syn_weight(net, src, tgt, j);
        }
    free(cnt);
    return ORC_OK;
}

/* sort every row of the stored CSR canonically */
static int sort_rows(orc_net *net)
{
    uint32_t n = net->P.n;
    uint64_t maxlen = 0;
    for (uint32_t s = 0; s < n; s++) {
        uint64_t L = net->row_ptr[s + 1] - net->row_ptr[s];
        if (L > maxlen) maxlen = L;
    }
    orc_syn *buf = (orc_syn *)malloc((size_t)(maxlen ? maxlen : 1) * sizeof(orc_syn));
    if (!buf) return ORC_ENOMEM;
    for (uint32_t s = 0; s < n; s++) {
        uint64_t o = net->row_ptr[s], L = net->row_ptr[s + 1] - o;
        for (uint64_t e = 0; e < L; e++) {
            buf[e].tgt = net->col[o + e];
            buf[e].d = net->delay[o + e];
            buf[e].w = net->w[o + e];
        }
        qsort(buf, (size_t)L, sizeof(orc_syn), syn_cmp);
        for (uint64_t e = 0; e < L; e++) {
            net->col[o + e] = buf[e].tgt;
            net->delay[o + e] = buf[e].d;
            net->w[o + e] = buf[e].w;
        }
    }
    free(buf);
    return ORC_OK;
}

/* statistics of the stored CSR + fixed-point weights + overflow guard */
static int finish_csr(orc_net *net)
{
    uint32_t n = net->P.n;
    net->have_csr = 1;
    net->D.max_row = 0;
    for (uint32_t s = 0; s < n; s++) {
        uint64_t L = net->row_ptr[s + 1] - net->row_ptr[s];
        if (L > net->D.max_row) net->D.max_row = (uint32_t)L;
    }
    if (net->P.acc_mode != ORC_ACC_FIXED) return ORC_OK;
    uint64_t nnz = net->D.nnz;
    net->wq = (int32_t *)malloc((size_t)(nnz ? nnz : 1) * sizeof(int32_t));
    if (!net->wq) return ORC_ENOMEM;
    for (uint64_t e = 0; e < nnz; e++)
        if (quantise(net->w[e], net->P.fixed_shift, &net->wq[e])) return ORC_EOVERFLOW;
    /* Guard: the largest input one neuron can receive in one step (all its
     * in-synapses at once, the largest Poisson count, the bias) must fit in
     * int32, otherwise the fixed-point sums could wrap. */
    int64_t *acc = (int64_t *)calloc(n, sizeof(int64_t));
    if (!acc) return ORC_ENOMEM;
    orc_in_abs_sum_q(net, acc);
    int64_t kmax = net->D.pois_len ? (int64_t)net->D.pois_len - 1 : 0;
    int64_t extra = kmax * llabs((long long)net->D.ext_wq) + llabs((long long)net->D.bias_q);
    int rc = ORC_OK;
    for (uint32_t i = 0; i < n; i++)
        if (acc[i] + extra > 2147483647ll) { rc = ORC_EOVERFLOW; break; }
    free(acc);
    return rc;
}

int orc_in_abs_sum_q(const orc_net *net, int64_t *out)
{
    if (!net->have_csr || !net->wq) return ORC_EINVAL;
    memset(out, 0, (size_t)net->P.n * sizeof(int64_t));
    for (uint64_t e = 0; e < net->D.nnz; e++)
        out[net->col[e]] += llabs((long long)net->wq[e]);
    return ORC_OK;
}

/* --------------------------------------------------------------- state */

static int init_state(orc_net *net)
{
    const orc_params *P = &net->P;
    uint32_t n = P->n;
    size_t slots = (size_t)net->D.ring * n;
    net->V = (float *)malloc((size_t)n * sizeof(float));
    net->ref = (uint8_t *)calloc(n, 1);
    if (P->acc_mode == ORC_ACC_FIXED)
        net->slot_q = (int64_t *)calloc(slots, sizeof(int64_t));
    else
        net->slot_f = (float *)calloc(slots, sizeof(float));
    net->arrive = (uint64_t *)calloc(net->D.ring, sizeof(uint64_t));
    if (!net->V || !net->ref || (!net->slot_q && !net->slot_f) || !net->arrive) return ORC_ENOMEM;
    /* V0 = v0_lo + (v0_hi - v0_lo) * u, u uniform in [0,1) */
    float span = P->v0_hi - P->v0_lo;
    for (uint32_t i = 0; i < n; i++) {
        float t = span * u24(orc_hash(P->seed, ORC_TAG_V0, i, 0));
        net->V[i] = P->v0_lo + t;
    }
    net->t = 0;
    return ORC_OK;
}

static orc_net *alloc_net(const orc_params *P)
{
    orc_net *net = (orc_net *)calloc(1, sizeof(orc_net));
    if (net) net->P = *P;
    return net;
}

int orc_create(const orc_params *P, int build_csr, orc_net **out)
{
    *out = NULL;
    if (P->conn_kind == ORC_CONN_EXPLICIT) return ORC_EINVAL;
    orc_net *net = alloc_net(P);
    if (!net) return ORC_ENOMEM;
    int rc = derive(net);
    if (!rc && build_csr) {
        if (P->conn_kind == ORC_CONN_FIXED_IN) {
            rc = build_fixed_in(net);
            if (!rc) rc = sort_rows(net);
        } else {
            rc = build_rows(net);
        }
        if (!rc) rc = finish_csr(net);
    }
    if (!rc) rc = init_state(net);
    if (rc) { orc_destroy(net); return rc; }
    *out = net;
    return ORC_OK;
}

int orc_create_explicit(const orc_params *P, uint32_t n, const uint64_t *row_ptr,
                        const uint32_t *col, const float *w, const uint8_t *delay,
                        orc_net **out)
{
    *out = NULL;
    orc_net *net = alloc_net(P);
    if (!net) return ORC_ENOMEM;
    net->P.n = n;
    net->P.conn_kind = ORC_CONN_EXPLICIT;
    int rc = derive(net);
    if (!rc && row_ptr[0] != 0) rc = ORC_EINVAL;
    for (uint32_t s = 0; !rc && s < n; s++)
        if (row_ptr[s + 1] < row_ptr[s]) rc = ORC_EINVAL;
    if (!rc) {
        uint64_t nnz = row_ptr[n];
        net->row_ptr = (uint64_t *)malloc(((size_t)n + 1) * sizeof(uint64_t));
        rc = net->row_ptr ? alloc_csr(net, nnz) : ORC_ENOMEM;
        if (!rc) {
            memcpy(net->row_ptr, row_ptr, ((size_t)n + 1) * sizeof(uint64_t));
            for (uint64_t e = 0; e < nnz && !rc; e++) {
                uint8_t d = delay ? delay[e] : (uint8_t)P->delay_min;
                if (col[e] >= n || d < P->delay_min || d > P->delay_max) rc = ORC_EINVAL;
                net->col[e] = col[e];
                net->w[e] = w[e];
                net->delay[e] = d;
            }
        }
        if (!rc) rc = sort_rows(net);
        if (!rc) rc = finish_csr(net);
    }
    if (!rc) rc = init_state(net);
    if (rc) { orc_destroy(net); return rc; }
    *out = net;
    return ORC_OK;
}

void orc_destroy(orc_net *net)
{
    if (!net) return;
    free(net->row_ptr); free(net->col); free(net->w); free(net->delay); free(net->wq);
    free(net->V); free(net->ref); free(net->slot_f); free(net->slot_q); free(net->arrive);
    free(net);
}

int orc_get_derived(const orc_net *net, orc_derived *out)
{
    *out = net->D;
    return ORC_OK;
}

uint64_t orc_nnz(const orc_net *net) { return net->have_csr ? net->D.nnz : 0; }

int orc_get_csr(const orc_net *net, uint64_t *row_ptr, uint32_t *col, float *w,
                uint8_t *delay)
{
    if (!net->have_csr) return ORC_EINVAL;
    uint64_t nnz = net->D.nnz;
    if (row_ptr) memcpy(row_ptr, net->row_ptr, ((size_t)net->P.n + 1) * sizeof(uint64_t));
    if (col) memcpy(col, net->col, (size_t)nnz * sizeof(uint32_t));
    if (w) memcpy(w, net->w, (size_t)nnz * sizeof(float));
    if (delay) memcpy(delay, net->delay, (size_t)nnz);
    return ORC_OK;
}

int orc_row(orc_net *net, uint32_t s, uint32_t *tgt, float *w, uint8_t *delay,
            uint64_t cap, uint64_t *len)
{
    if (s >= net->P.n) return ORC_EINVAL;
    if (net->have_csr) {
        uint64_t o = net->row_ptr[s], L = net->row_ptr[s + 1] - o;
        *len = L;
        if (L > cap) return ORC_EOVERFLOW;
        for (uint64_t e = 0; e < L; e++) {
            tgt[e] = net->col[o + e];
            w[e] = net->w[o + e];
            delay[e] = net->delay[o + e];
        }
        return ORC_OK;
    }
    uint64_t bcap = net->P.conn_kind == ORC_CONN_BERNOULLI ? net->P.n : net->P.k_out;
    orc_syn *buf = (orc_syn *)malloc((size_t)(bcap ? bcap : 1) * sizeof(orc_syn));
    if (!buf) return ORC_ENOMEM;
    long long L = gen_row(net, s, buf, bcap, 1);
    if (L < 0) { free(buf); return ORC_EINVAL; }
    *len = (uint64_t)L;
    if ((uint64_t)L > cap) { free(buf); return ORC_EOVERFLOW; }
    for (long long e = 0; e < L; e++) {
        tgt[e] = buf[e].tgt;
        w[e] = buf[e].w;
        delay[e] = buf[e].d;
    }
    free(buf);
    return ORC_OK;
}

/* ------------------------------------------------------------ delivery */

int orc_in_row(const orc_net *net, uint32_t tgt, uint32_t *src, float *w, uint8_t *delay,
               uint64_t cap, uint64_t *len)
{
    const orc_params *P = &net->P;
    if (P->conn_kind != ORC_CONN_FIXED_IN || tgt >= P->n) return ORC_EINVAL;
    uint32_t kin = P->k_in_exc + P->k_in_inh;
    *len = kin;
    if (kin > cap) return ORC_EOVERFLOW;
    for (uint32_t j = 0; j < kin; j++) {
        src[j] = fixed_in_src(net, tgt, j);
        delay[j] = syn_delay(net, tgt, j);
        w[j] = syn_weight(net, src[j], tgt, j);
    }
    return ORC_OK;
}

int orc_pair(const orc_net *net, uint32_t s, uint32_t tgt, int *connected, float *w, uint8_t *delay)
{
    const orc_params *P = &net->P;
    if (P->conn_kind != ORC_CONN_BERNOULLI || s >= P->n || tgt >= P->n) return ORC_EINVAL;
    /* Sec. III-B: every ordered pair is connected independently with
     * probability p */
    *connected = hi32(orc_hash(P->seed, ORC_TAG_CONN, s, tgt)) < net->D.conn_thr;
    *w = syn_weight(net, s, s, tgt);
    *delay = syn_delay(net, s, tgt);
    return ORC_OK;
}

int orc_deliver(orc_net *net, const uint32_t *spikes, uint64_t n_spikes,
                uint32_t delay, double *out_f, int64_t *out_q)
{
    uint32_t n = net->P.n;
    if (out_f) memset(out_f, 0, (size_t)n * sizeof(double));
    if (out_q) memset(out_q, 0, (size_t)n * sizeof(int64_t));
    uint64_t bcap = 0;
    orc_syn *buf = NULL;
    if (!net->have_csr) {
        if (net->P.conn_kind != ORC_CONN_BERNOULLI && net->P.conn_kind != ORC_CONN_FIXED_OUT)
            return ORC_EINVAL;
        bcap = net->P.conn_kind == ORC_CONN_BERNOULLI ? n : net->P.k_out;
        buf = (orc_syn *)malloc((size_t)(bcap ? bcap : 1) * sizeof(orc_syn));
        if (!buf) return ORC_ENOMEM;
    }
    for (uint64_t k = 0; k < n_spikes; k++) {
        uint32_t s = spikes[k];
        if (s >= n) { free(buf); return ORC_EINVAL; }
        if (net->have_csr) {
            for (uint64_t e = net->row_ptr[s]; e < net->row_ptr[s + 1]; e++) {
                if (delay && net->delay[e] != delay) continue;
                if (out_f) out_f[net->col[e]] += (double)net->w[e];
                if (out_q) {
                    int32_t q;
                    if (quantise(net->w[e], net->P.fixed_shift, &q)) { free(buf); return ORC_EOVERFLOW; }
                    out_q[net->col[e]] += q;
                }
            }
        } else {
            long long L = gen_row(net, s, buf, bcap, 0);
            for (long long e = 0; e < L; e++) {
                if (delay && buf[e].d != delay) continue;
                if (out_f) out_f[buf[e].tgt] += (double)buf[e].w;
                if (out_q) {
                    int32_t q;
                    if (quantise(buf[e].w, net->P.fixed_shift, &q)) { free(buf); return ORC_EOVERFLOW; }
                    out_q[buf[e].tgt] += q;
                }
            }
        }
    }
    free(buf);
    return ORC_OK;
}

/* -------------------------------------------------------------- update */

/* One neuron, one step.  isyn_f / isyn_q is the synaptic input that arrived
 * for step t. */
static int update_neuron(const orc_net *net, uint64_t t, uint32_t i, float *v, uint8_t *ref,
                         float isyn_f, int64_t isyn_q)
{
    const orc_params *P = &net->P;
    const orc_derived *D = &net->D;
    uint32_t K = 0;
    if (D->pois_len) K = poisson_draw(net, orc_hash_step(P->seed, ORC_TAG_POIS, i, (uint32_t)t));
    float I;
    if (P->acc_mode == ORC_ACC_FIXED) {
        int64_t q = isyn_q + (int64_t)K * D->ext_wq + D->bias_q;
        if (q > 2147483647ll || q < -2147483648ll) return -1;
        I = ldexpf((float)(int32_t)q, -P->fixed_shift);
    } else {
        float ext = (float)K * P->ext_w;
        float s = isyn_f + ext;
        I = s + P->i_bias;
    }
    if (P->neuron_kind == ORC_SOURCE) {
        float a = P->v_rest - *v;
        float b = D->k * a;
        float c = *v + b;
        *v = c + I;
        return hi32(orc_hash_step(P->seed, ORC_TAG_BERN, i, (uint32_t)t)) < D->src_thr ? 1 : 0;
    }
    if (*ref > 0) {
        *ref = (uint8_t)(*ref - 1);
        *v = P->v_reset;
        return 0;
    }
    float a = P->v_rest - *v;
    float b = D->k * a;
    float c = *v + b;
    *v = c + I;
    if (*v >= P->v_th) {
        *v = P->v_reset;
        *ref = (uint8_t)D->ref_steps;
        return 1;
    }
    return 0;
}

int orc_update_one(const orc_net *net, uint64_t t, uint32_t i, float v, uint8_t ref,
                   float isyn_f, int64_t isyn_q, float *v_out, uint8_t *ref_out,
                   int *spiked)
{
    if (i >= net->P.n) return ORC_EINVAL;
    int s = update_neuron(net, t, i, &v, &ref, isyn_f, isyn_q);
    if (s < 0) return ORC_EOVERFLOW;
    *v_out = v;
    *ref_out = ref;
    *spiked = s;
    return ORC_OK;
}

/* ----------------------------------------------------------------- run */

/* Add one synapse (target tgt, weight w, delay d) of a spike of step t to
 * the input of step t + d. */
static void push_synapse(orc_net *net, uint64_t t, uint32_t tgt, float w, int32_t wq, uint8_t d)
{
    uint32_t R = net->D.ring;
    size_t slot = (size_t)((t + d) % R) * net->P.n + tgt;
    if (net->P.acc_mode == ORC_ACC_FIXED) net->slot_q[slot] += wq;
    else                                  net->slot_f[slot] += w;
    net->arrive[(t + d) % R] += 1;
}

int orc_run(orc_net *net, uint64_t n_steps, uint32_t *counts, uint64_t *events,
            uint64_t *delivered, uint32_t *raster, uint64_t raster_cap, uint64_t *offs)
{
    const orc_params *P = &net->P;
    uint32_t n = P->n, R = net->D.ring;
    int fixed = P->acc_mode == ORC_ACC_FIXED;
    /* Without the stored CSR (Bernoulli and fixed out-degree networks too
     * large to store here), the row of every spike is generated when the
     * spike is delivered: the same rows, in canonical order in fp32 mode
     * (where the order of the fp32 additions matters) and in draw order in
     * fixed-point mode (integer sums do not depend on it). */
    uint64_t bcap = 0;
    orc_syn *buf = NULL;
    if (!net->have_csr) {
        if (P->conn_kind != ORC_CONN_BERNOULLI && P->conn_kind != ORC_CONN_FIXED_OUT) return ORC_EINVAL;
        bcap = P->conn_kind == ORC_CONN_BERNOULLI ? n : P->k_out;
        buf = (orc_syn *)malloc((size_t)(bcap ? bcap : 1) * sizeof(orc_syn));
        if (!buf) return ORC_ENOMEM;
    }
    uint32_t *S = (uint32_t *)malloc((size_t)n * sizeof(uint32_t));
    if (!S) { free(buf); return ORC_ENOMEM; }
    uint64_t rl = 0;
    if (offs) offs[0] = 0;
    int rc = ORC_OK;
    for (uint64_t step = 0; step < n_steps; step++) {
        uint64_t t = net->t;
        size_t base = (size_t)(t % R) * n;
        uint32_t ns = 0;
        /* 1. update every neuron with the input that arrived for step t */
        for (uint32_t i = 0; i < n; i++) {
            float xf = 0.0f;
            int64_t xq = 0;
            if (fixed) { xq = net->slot_q[base + i]; net->slot_q[base + i] = 0; }
            else       { xf = net->slot_f[base + i]; net->slot_f[base + i] = 0.0f; }
            int s = update_neuron(net, t, i, &net->V[i], &net->ref[i], xf, xq);
            if (s < 0) { rc = ORC_EOVERFLOW; goto done; }
            if (s) S[ns++] = i;
        }
        uint64_t arrived = net->arrive[t % R];
        net->arrive[t % R] = 0;
        /* 2. deliver every spike of step t to all neighbours in its row;
         *    a synapse of delay d feeds the input of step t + d */
        uint64_t ev = 0;
        for (uint32_t k = 0; k < ns; k++) {
            uint32_t s = S[k];
            if (net->have_csr) {
                for (uint64_t e = net->row_ptr[s]; e < net->row_ptr[s + 1]; e++)
                    push_synapse(net, t, net->col[e], net->w[e], fixed ? net->wq[e] : 0, net->delay[e]);
                ev += net->row_ptr[s + 1] - net->row_ptr[s];
            } else {
                long long L = gen_row(net, s, buf, bcap, !fixed);
                if (L < 0) { rc = ORC_EINVAL; goto done; }
                for (long long e = 0; e < L; e++) {
                    int32_t q = 0;
                    if (fixed && quantise(buf[e].w, P->fixed_shift, &q)) { rc = ORC_EOVERFLOW; goto done; }
                    push_synapse(net, t, buf[e].tgt, buf[e].w, q, buf[e].d);
                }
                ev += (uint64_t)L;
            }
        }
        /* 3. record */
        if (counts) counts[step] = ns;
        if (events) events[step] = ev;
        if (delivered) delivered[step] = arrived;
        if (raster) {
            if (rl + ns > raster_cap) { rc = ORC_EOVERFLOW; goto done; }
            memcpy(raster + rl, S, (size_t)ns * sizeof(uint32_t));
        }
        rl += ns;
        if (offs) offs[step + 1] = rl;
        net->t = t + 1;
    }
done:
    free(S);
    free(buf);
    return rc;
}

int orc_get_state(const orc_net *net, float *v, uint8_t *ref)
{
    if (v) memcpy(v, net->V, (size_t)net->P.n * sizeof(float));
    if (ref) memcpy(ref, net->ref, net->P.n);
    return ORC_OK;
}

uint64_t orc_step_index(const orc_net *net) { return net->t; }
