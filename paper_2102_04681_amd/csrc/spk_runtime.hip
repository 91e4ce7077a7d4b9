// spk_runtime.hip -- host runtime and C ABI of libspk (declared in spk.h).
//
// A network owns its device memory and orders all work on one HIP stream.
// Creation expands the connectivity parameters on the GPU (paper Sec. III-B:
// the layout description is expanded on the device) into one row per source
// neuron, grouped by target tile (Sec. III-A keeps rows sorted by target),
// with each synapse carrying its delay (Sec. V), and records where every row
// crosses the tile or XCD-group boundaries.  Steps run either as one
// persistent cooperative launch per spk_step call (spk_run.hip), or as the
// tile kernel (delivery into LDS + update + spike list), then for binned
// delivery the push kernel (the new spikes' events into per-arrival pages),
// then the optional raster record, batches of steps captured once into a HIP
// graph and replayed.  Spike counts stay on the device, so stepping never
// waits for the host.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "spk_internal.h"

using namespace spk;

namespace {

thread_local std::string g_err;

spk_status fail(spk_status st, const std::string &msg)
{
    g_err = msg;
    return st;
}

#define SPK_HIP(expr)                                                                   \
    do {                                                                                \
        hipError_t e_ = (expr);                                                         \
        if (e_ != hipSuccess)                                                           \
            return fail(e_ == hipErrorOutOfMemory ? SPK_ENOMEM : SPK_EHIP,              \
                        std::string(#expr) + ": " + hipGetErrorString(e_));             \
    } while (0)

#define SPK_TRY(expr)                   \
    do {                                \
        spk_status s_ = (expr);         \
        if (s_ != SPK_OK) return s_;    \
    } while (0)

constexpr uint32_t kPoisCap = 256;
constexpr uint32_t kBatch = 32;                    // steps per captured graph
constexpr uint64_t kPageBudget = 256ull << 20;     // page records across all pages (2 GiB)
constexpr uint64_t kDebugPageCap = 4096;           // records per page for spk_debug_deliver
constexpr uint64_t kRunMaxSteps = 1ull << 24;      // steps per persistent launch (barrier epochs fit u32)
constexpr uint32_t kFlagRunStopped = 4u;           // device flag: a persistent launch stopped early

// Scratch of spk_deliver_noalloc: one fixed area per device, held until the
// process ends, shared by every call on that device (the caller orders
// them).  In host code the array's name stands for a host-side shadow, not a
// device address: kernels get the address hipGetSymbolAddress returned for
// the device, looked up once per device when a network is created there.
constexpr uint64_t kNoAllocScratchBytes = SPK_NOALLOC_SCRATCH_BYTES;
__device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];

// Address of this device's scratch (the device is current); looked up once.
spk_status scratch_lookup(int device)
{
    if (device < 0 || device >= kMaxDevices) return fail(SPK_EINVAL, "device index beyond the scratch table");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[device]) return SPK_OK;
    void *p = nullptr;
    SPK_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(SPK_EHIP, "hipGetSymbolAddress returned no address for the scratch area");
    g_scratch_ptr[device] = p;
    return SPK_OK;
}

void *scratch_of(int device)
{
    if (device < 0 || device >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    return g_scratch_ptr[device];
}

uint64_t prob_threshold(double p)
{
    if (!(p > 0.0)) return 0;
    if (p >= 1.0) return 4294967296ull;
    return (uint64_t)std::floor(p * 4294967296.0);
}

// Poisson(lambda) thresholds on a 32-bit uniform draw: T_k = floor(CDF(k)*2^32)
// with the CDF summed in double from p_0 = exp(-lambda), p_k = p_{k-1}*lambda/k;
// the table ends with 2^32 once the CDF reaches 1 - 2^-32.
int poisson_thresholds(double lambda, std::vector<uint64_t> &thr)
{
    thr.clear();
    if (!(lambda > 0.0) || lambda > 100.0) return -1;
    double pk = std::exp(-lambda), cdf = pk;
    for (uint32_t k = 0;; k++) {
        const double T = std::floor(cdf * 4294967296.0);
        if (T >= 4294967295.0 || k == kPoisCap - 1) {
            thr.push_back(4294967296ull);
            return (int)thr.size();
        }
        thr.push_back((uint64_t)T);
        pk = (pk * lambda) / (double)(k + 1);
        cdf = cdf + pk;
    }
}

// Guide table of the indexed search (Chen & Asau 1974): for the 256 ranges of
// the top 8 bits of the draw, the first k whose threshold exceeds the range
// start; the search for K = min{k : h < T_k} starts there.
std::vector<uint16_t> poisson_guide(const std::vector<uint64_t> &thr)
{
    std::vector<uint16_t> g(256, 0);
    uint32_t k = 0;
    for (uint32_t b = 0; b < 256; b++) {
        const uint64_t lo = (uint64_t)b << 24;
        while (k + 1 < thr.size() && thr[k] <= lo) k++;
        g[b] = (uint16_t)k;
    }
    return g;
}

bool quantise(float w, int S, int32_t *out)
{
    const float x = std::rint(std::ldexp(w, S));
    if (!(std::fabs(x) < 2147483648.0f)) return false;
    *out = (int32_t)x;
    return true;
}

// Tiles of W neurons (a power of two, at most kMaxTileW), 8 groups of T8
// tiles; the smallest W that keeps T8 <= max_t8 (default 32: one tile per
// compute unit).  SPK_TILES_PER_XCD overrides max_t8 (a tuning knob).
Tiling make_tiling(uint32_t n)
{
    uint32_t max_t8 = 32;
    if (const char *e = std::getenv("SPK_TILES_PER_XCD")) {
        const long v = std::strtol(e, nullptr, 10);
        if (v >= 1 && v <= (long)kMaxT8) max_t8 = (uint32_t)v;
    }
    Tiling tl{};
    uint32_t W = 64, logW = 6;
    while (W < kMaxTileW && (n + 8ull * W - 1) / (8ull * W) > max_t8) {
        W <<= 1;
        logW++;
    }
    tl.W = W;
    tl.logW = logW;
    tl.T8 = (uint32_t)((n + 8ull * W - 1) / (8ull * W));
    tl.T = kGroups * tl.T8;
    tl.Gw = tl.T8 * W;
    tl.T8inv = tl.T8 > 1 ? (uint32_t)(((1ull << 32) + tl.T8 - 1) / tl.T8) : 0u;
    return tl;
}

}  // namespace

struct spk_net {
    spk_params P{};
    // derived constants
    uint32_t n = 0, n_exc = 0, lists = 1, dmin = 1, dmax = 1, ref_steps = 0;
    uint32_t pois_len = 0, max_row = 0;
    float k = 0.f;
    uint64_t conn_thr = 0, src_thr = 0, nnz = 0;
    int32_t ext_wq = 0, bias_q = 0, shift64 = 0;
    Keys keys{};
    std::vector<uint64_t> pois;
    std::vector<uint16_t> guide;
    Tiling tl{};
    bool direct = false;
    uint32_t spk_slots = 1, pslots = 1, pg1 = 1, page_cap = 0;
    // device
    hipStream_t stream = nullptr, cap_stream = nullptr;
    bool own_stream = false;
    int device = 0;
    uint64_t *row_ptr = nullptr;
    // synapses: full (int2) or compact (u32 with a weight class)
    bool compact = false;
    bool proc = false;  // procedural synapses: generated when their source fires, not stored
    bool proc_once = false;  // ... each fired row generated once (pages of every group per push block)
    uint32_t n_cls = 0;
    float cls_w[kMaxClasses] = {};
    ClassTab ctab{};
    long long wval[kMaxClasses] = {};
    int2 *syn = nullptr;
    uint32_t *syn32 = nullptr;
    RowDesc *desc = nullptr;
    uint16_t *toff = nullptr;
    uint32_t *outdeg = nullptr;
    float *V = nullptr;
    uint8_t *ref = nullptr;
    uint32_t *spk_ids = nullptr, *spk_cnt = nullptr, *counts8 = nullptr, *flags = nullptr;
    uint64_t *events8 = nullptr, *delivered8 = nullptr, *pois_dev = nullptr, *t_base = nullptr;
    uint16_t *guide_dev = nullptr;
    int2 *pages = nullptr;
    uint16_t *pages16 = nullptr;
    uint32_t *pfill = nullptr, *ovf_flag = nullptr;
    void *acc_ovf = nullptr;
    uint32_t *raster = nullptr;
    uint64_t *raster_offs = nullptr;
    void *dbg_out = nullptr;
    uint64_t t = 0;
    uint64_t device_bytes = 0;
    std::vector<void *> allocs;
    std::map<uint32_t, hipGraphExec_t> graphs;
    // persistent step kernel
    bool persistent = false;
    uint32_t run_R = 0;
    uint32_t run_D = 1;  // persistent kernel, binned delivery: steps per batch
    RunCtl *ctl = nullptr;
    // profiling
    bool profiling = false;
    std::vector<hipEvent_t> ev_free;
    std::vector<std::pair<hipEvent_t, hipEvent_t>> ev_push, ev_tile, ev_run;
    double ms_push = 0, ms_tile = 0, ms_run = 0;
    uint64_t launches = 0, run_launches = 0;
    // setup timing
    double setup_ms = 0, gen_ms = 0, range_ms = 0;
};

namespace {

// GPU time of the work enqueued on a stream between start() and stop(),
// added to *acc by stop() (which waits for the work).
struct SegTimer {
    hipEvent_t e0 = nullptr, e1 = nullptr;
    SegTimer() = default;
    SegTimer(const SegTimer &) = delete;
    SegTimer &operator=(const SegTimer &) = delete;
    ~SegTimer()
    {
        if (e0) (void)hipEventDestroy(e0);
        if (e1) (void)hipEventDestroy(e1);
    }
    hipError_t start(hipStream_t s)
    {
        hipError_t e = e0 ? hipSuccess : hipEventCreate(&e0);
        if (e == hipSuccess && !e1) e = hipEventCreate(&e1);
        return e == hipSuccess ? hipEventRecord(e0, s) : e;
    }
    hipError_t stop(hipStream_t s, double *acc)
    {
        hipError_t e = hipEventRecord(e1, s);
        if (e == hipSuccess) e = hipEventSynchronize(e1);
        float t = 0.f;
        if (e == hipSuccess) e = hipEventElapsedTime(&t, e0, e1);
        if (e == hipSuccess) *acc += t;
        return e;
    }
};

template <class T>
spk_status dalloc(spk_net *net, T **p, size_t count)
{
    *p = nullptr;
    const size_t bytes = (count ? count : 1) * sizeof(T);
    void *q = nullptr;
    hipError_t e = hipMalloc(&q, bytes);
    if (e != hipSuccess)
        return fail(SPK_ENOMEM, "hipMalloc of " + std::to_string(bytes) + " bytes: " +
                                    hipGetErrorString(e));
    net->allocs.push_back(q);
    net->device_bytes += bytes;
    *p = (T *)q;
    return SPK_OK;
}

void dfree(spk_net *net, void *p)
{
    if (!p) return;
    auto it = std::find(net->allocs.begin(), net->allocs.end(), p);
    if (it != net->allocs.end()) net->allocs.erase(it);
    (void)hipFree(p);
}

ModelArgs model_args(const spk_net *net)
{
    ModelArgs m{};
    m.n = net->n;
    m.kind = net->P.neuron_kind;
    m.fixed = net->P.acc_mode == SPK_ACC_FIXED;
    m.shift = net->P.fixed_shift;
    m.shift64 = net->shift64;
    m.k = net->k;
    m.v_rest = net->P.v_rest;
    m.v_th = net->P.v_th;
    m.v_reset = net->P.v_reset;
    m.i_bias = net->P.i_bias;
    m.ext_w = net->P.ext_w;
    m.ext_wq = net->ext_wq;
    m.bias_q = net->bias_q;
    m.ref_steps = net->ref_steps;
    m.pois_len = net->pois_len;
    m.src_thr = net->src_thr;
    m.keys = net->keys;
    return m;
}

StepArgs step_args(const spk_net *net)
{
    StepArgs a{};
    a.m = model_args(net);
    a.tl = net->tl;
    a.n = net->n;
    a.lists = net->lists;
    a.dmin = net->dmin;
    a.direct = net->direct ? 1u : 0u;
    a.row_ptr = net->row_ptr;
    a.compact = net->compact ? 1u : 0u;
    a.proc = net->proc ? 1u : 0u;
    a.pr.k_out = net->P.k_out;
    a.pr.once = net->proc_once ? 1u : 0u;
    a.pr.n_exc = net->n_exc;
    a.pr.w_uniform = net->P.w_uniform;
    a.pr.w_lo = net->P.w_lo;
    a.pr.w_hi = net->P.w_hi;
    a.pr.w_exc = net->P.w_exc;
    a.pr.w_inh = net->P.w_inh;
    a.pr.qscale = std::ldexp(1.0f, net->P.fixed_shift);
    for (uint32_t k = 0; k < kMaxClasses; k++) a.wval[k] = net->wval[k];
    a.syn = net->syn;
    a.syn32 = net->syn32;
    a.desc = net->desc;
    a.toff = net->toff;
    a.outdeg = net->outdeg;
    a.V = net->V;
    a.ref = net->ref;
    a.spk_slots = net->spk_slots;
    a.spk_ids = net->spk_ids;
    a.spk_cnt = net->spk_cnt;
    a.counts8 = net->counts8;
    a.events8 = net->events8;
    a.delivered8 = net->delivered8;
    a.pages = net->pages;
    a.pages16 = net->pages16;
    a.pfill = net->pfill;
    a.page_cap = net->page_cap;
    a.pslots = net->pslots;
    a.pg1 = net->pg1;
    a.acc_ovf = net->acc_ovf;
    a.ovf_flag = net->ovf_flag;
    a.pois = net->pois_dev;
    a.pois_guide = net->guide_dev;
    a.flags = net->flags;
    a.raster = net->raster;
    a.raster_offs = net->raster_offs;
    a.raster_cap = net->P.raster_capacity;
    a.t_base = net->t_base;
    a.dbg_j = -1;
    return a;
}

ConnArgs conn_args(const spk_net *net)
{
    ConnArgs c{};
    c.n = net->n;
    c.n_exc = net->n_exc;
    c.kind = net->P.conn_kind;
    c.lists = net->lists;
    c.dmin = net->dmin;
    c.k_out = net->P.k_out;
    c.k_in_exc = net->P.k_in_exc;
    c.k_in_inh = net->P.k_in_inh;
    c.conn_thr = net->conn_thr;
    c.w_uniform = net->P.w_uniform;
    c.w_exc = net->P.w_exc;
    c.w_inh = net->P.w_inh;
    c.w_lo = net->P.w_lo;
    c.w_hi = net->P.w_hi;
    c.fixed = net->P.acc_mode == SPK_ACC_FIXED;
    c.qscale = std::ldexp(1.0f, net->P.fixed_shift);
    c.compact = net->compact ? 1u : 0u;
    for (uint32_t k = 0; k < kMaxClasses; k++) {
        float w = net->cls_w[k < net->n_cls ? k : 0];
        std::memcpy(&c.cls_w[k], &w, 4);
    }
    c.keys = net->keys;
    c.tl = net->tl;
    return c;
}

// Synapse format.  classes = the distinct weights (null: per-synapse weights).
// Class k stores its weight bits (fp32, or the quantised int32 in fixed mode)
// and the |weight| term of the accumulator-range bound, both as the full
// format would per synapse.
spk_status choose_format(spk_net *net, const float *classes, uint32_t n_cls)
{
    const uint32_t f = net->P.syn_format;
    const bool ok = classes && n_cls >= 1 && n_cls <= kMaxClasses;
    if (f == SPK_FORMAT_COMPACT && !ok)
        return fail(SPK_EINVAL, "the compact synapse format needs at most 4 distinct weights");
    net->compact = ok && f != SPK_FORMAT_FULL;
    net->n_cls = 0;
    net->ctab = ClassTab{};
    if (!net->compact) return SPK_OK;
    const bool fixed = net->P.acc_mode == SPK_ACC_FIXED;
    net->n_cls = n_cls;
    for (uint32_t k = 0; k < kMaxClasses; k++) {
        const float w = classes[k < n_cls ? k : 0];
        net->cls_w[k] = w;
        if (fixed) {
            int32_t q = 0;
            if (!quantise(w, net->P.fixed_shift, &q))
                return fail(SPK_EOVERFLOW, "a weight does not fit int32 at this fixed_shift");
            net->ctab.bits[k] = (uint32_t)q;
            net->ctab.abs[k] = (uint64_t)std::llabs((long long)q);
        } else {
            std::memcpy(&net->ctab.bits[k], &w, 4);
            net->ctab.abs[k] = (uint64_t)std::ceil(std::ldexp((double)std::fabs(w), 24));
        }
    }
    return SPK_OK;
}

// How the accumulator range of a generated Bernoulli network is found: per
// target from the pair predicate (n^2 hashes, ~1.7e12 per s) when that costs
// less than one global atomic per synapse (~2.4e10 per s).
// SPK_RANGE_PASS=targets / atomics forces either (a tuning knob, for tests).
bool range_by_targets(const spk_net *net)
{
    if (net->P.conn_kind != SPK_CONN_BERNOULLI) return false;
    if (const char *e = std::getenv("SPK_RANGE_PASS")) return std::strcmp(e, "targets") == 0;
    return (double)net->nnz * 70.0 > (double)net->n * (double)net->n;
}

// Fixed out-degree networks with population weights (generated, compact
// classes = source populations): the range from the synapses drawn again and
// filed by target tile, counted per class in LDS (no global atomic per
// synapse).  SPK_RANGE_PASS=atomics forces the per-synapse atomic pass.
bool range_by_tiles(const spk_net *net)
{
    if (net->P.conn_kind != SPK_CONN_FIXED_OUT || !net->compact || net->n_cls > 2) return false;
    if (const char *e = std::getenv("SPK_RANGE_PASS")) return std::strcmp(e, "atomics") != 0;
    return true;
}

// Largest in_abs_sum of a fixed out-degree network by tiles (range_by_tiles);
// *ok = false (and nothing changed) when its temporary buckets (2 bytes per
// synapse) cannot be allocated.
spk_status fo_range(spk_net *net, uint64_t *m, bool *ok)
{
    hipStream_t s = net->stream;
    const ConnArgs c = conn_args(net);
    const uint32_t T = net->tl.T, nb = fo_blocks(net->n);
    *ok = false;
    uint16_t *entries = nullptr;
    if (dalloc(net, &entries, (size_t)std::max<uint64_t>(net->nnz, 1)) != SPK_OK) {
        (void)hipGetLastError();  // the failed allocation is not an error of a later call
        return SPK_OK;
    }
    uint32_t *base = nullptr, *tot = nullptr;
    uint64_t *start = nullptr, *mx = nullptr;
    SPK_TRY(dalloc(net, &base, (size_t)nb * T));
    SPK_TRY(dalloc(net, &tot, T));
    SPK_TRY(dalloc(net, &start, T + 1));
    SPK_TRY(dalloc(net, &mx, 1));
    SPK_HIP(hipMemsetAsync(tot, 0, (size_t)T * 4, s));
    SPK_HIP(hipMemsetAsync(mx, 0, 8, s));
    SegTimer tm;
    SPK_HIP(tm.start(s));
    SPK_HIP(fo_count(c, base, tot, s));
    std::vector<uint32_t> ht(T);
    SPK_HIP(hipMemcpyAsync(ht.data(), tot, (size_t)T * 4, hipMemcpyDeviceToHost, s));
    SPK_HIP(hipStreamSynchronize(s));
    std::vector<uint64_t> hs(T + 1, 0);
    for (uint32_t k = 0; k < T; k++) hs[k + 1] = hs[k] + ht[k];
    if (hs[T] != net->nnz) return fail(SPK_EHIP, "range pass: filed synapses do not add up to nnz");
    SPK_HIP(hipMemcpyAsync(start, hs.data(), (size_t)(T + 1) * 8, hipMemcpyHostToDevice, s));
    SPK_HIP(fo_file(c, base, start, entries, s));
    SPK_HIP(fo_max(c, start, entries, net->ctab, mx, s));
    SPK_HIP(tm.stop(s, &net->range_ms));
    SPK_HIP(hipMemcpyAsync(m, mx, 8, hipMemcpyDeviceToHost, s));
    SPK_HIP(hipStreamSynchronize(s));  // (hs is host memory read by the copy above)
    dfree(net, entries); dfree(net, base); dfree(net, tot); dfree(net, start); dfree(net, mx);
    *ok = true;
    return SPK_OK;
}

// The term of one synapse of weight w in the accumulator-range bound, as the
// range pass computes it: |quantised w| (fixed mode) or |w| in units of
// 2^-24 rounded up (fp32 mode).
spk_status abs_term(const spk_net *net, float w, uint64_t *out)
{
    if (net->P.acc_mode == SPK_ACC_FIXED) {
        int32_t q = 0;
        if (!quantise(w, net->P.fixed_shift, &q))
            return fail(SPK_EOVERFLOW, "a weight does not fit int32 at this fixed_shift");
        *out = (uint64_t)std::llabs((long long)q);
    } else {
        *out = (uint64_t)std::ceil(std::ldexp((double)std::fabs(w), 24));
    }
    return SPK_OK;
}

// Per-class accumulator units, once the unit is known.
void class_units(spk_net *net)
{
    const bool fixed = net->P.acc_mode == SPK_ACC_FIXED;
    for (uint32_t k = 0; k < kMaxClasses; k++) {
        if (!net->compact) {
            net->wval[k] = 0;
        } else if (fixed) {
            net->wval[k] = (long long)(int32_t)net->ctab.bits[k];
        } else {
            // exact: every weight is a multiple of the unit 2^-S64 (as the
            // per-event conversion of the full format, rounded to nearest)
            net->wval[k] = std::llrint(std::ldexp((double)net->cls_w[k], net->shift64));
        }
    }
}

// Synapse storage of the chosen format.
spk_status alloc_syn(spk_net *net, void **p, uint64_t nnz)
{
    uint8_t *q = nullptr;
    SPK_TRY(dalloc(net, &q, (size_t)nnz * (net->compact ? 4 : 8)));
    *p = q;
    return SPK_OK;
}

const void *syn_ptr(const spk_net *net)
{
    return net->compact ? (const void *)net->syn32 : (const void *)net->syn;
}

// Validate parameters and compute the derived constants.
spk_status derive(spk_net *net, bool explicit_csr)
{
    const spk_params &P = net->P;
    if (P.abi_version != SPK_ABI_VERSION) return fail(SPK_EINVAL, "abi_version mismatch");
    if (P.n == 0 || P.n > (1u << kTargetBits))
        return fail(SPK_EINVAL, "n must be in [1, 2^24]");
    if (!(P.dt_ms > 0.0) || !(P.tau_m_ms > 0.0) || !(P.t_ref_ms >= 0.0))
        return fail(SPK_EINVAL, "dt_ms, tau_m_ms must be > 0 and t_ref_ms >= 0");
    if (P.delay_min < 1 || P.delay_max < P.delay_min || P.delay_max > 253)
        return fail(SPK_EINVAL, "delays must satisfy 1 <= delay_min <= delay_max <= 253");
    if (P.delay_max - P.delay_min + 1 > kMaxLists)
        return fail(SPK_EINVAL, "at most 64 distinct delays");
    if (!(P.frac_exc >= 0.0 && P.frac_exc <= 1.0)) return fail(SPK_EINVAL, "frac_exc in [0,1]");
    if (P.neuron_kind > SPK_SOURCE) return fail(SPK_EINVAL, "neuron_kind");
    if (P.acc_mode > SPK_ACC_FIXED) return fail(SPK_EINVAL, "acc_mode");
    if (P.delivery > SPK_DELIVERY_BINNED) return fail(SPK_EINVAL, "delivery");
    if (P.syn_format > SPK_FORMAT_PROCEDURAL) return fail(SPK_EINVAL, "syn_format");
    if (P.syn_format == SPK_FORMAT_PROCEDURAL) {
        if (explicit_csr || P.conn_kind != SPK_CONN_FIXED_OUT || P.k_out == 0)
            return fail(SPK_EINVAL, "procedural synapses need a generated fixed out-degree network (k_out >= 1)");
        if (P.delivery == SPK_DELIVERY_DIRECT)
            return fail(SPK_EINVAL, "procedural synapses are delivered binned (each fired row generated once)");
        if (P.step_mode == SPK_STEP_PERSISTENT)
            return fail(SPK_EINVAL, "procedural synapses run as graphs of steps, not in the persistent kernel");
        net->proc = true;
    }
    if (P.step_mode > SPK_STEP_PERSISTENT) return fail(SPK_EINVAL, "step_mode");
    if (!explicit_csr && P.conn_kind > SPK_CONN_FIXED_IN) return fail(SPK_EINVAL, "conn_kind");
    if (!(P.p >= 0.0 && P.p <= 1.0)) return fail(SPK_EINVAL, "p in [0,1]");
    if (P.max_steps == 0) return fail(SPK_EINVAL, "max_steps must be >= 1");
    if (!(P.ext_lambda >= 0.0) || P.ext_lambda > 100.0) return fail(SPK_EINVAL, "ext_lambda in [0,100]");
    if (!explicit_csr && P.conn_kind == SPK_CONN_FIXED_OUT && P.k_out > kMaxRow)
        return fail(SPK_EINVAL, "k_out exceeds the longest supported row (65535)");
    net->n = P.n;
    net->n_exc = (uint32_t)std::llround(P.frac_exc * (double)P.n);
    net->k = (float)(P.dt_ms / P.tau_m_ms);
    const long long rs = std::llround(P.t_ref_ms / P.dt_ms);
    if (rs < 0 || rs > 255) return fail(SPK_EINVAL, "t_ref/dt must round to 0..255 steps");
    net->ref_steps = (uint32_t)rs;
    net->dmin = P.delay_min;
    net->dmax = P.delay_max;
    net->lists = P.delay_max - P.delay_min + 1;
    net->conn_thr = prob_threshold(P.p);
    net->src_thr = prob_threshold(P.src_rate_hz * P.dt_ms * 1e-3);
    net->tl = make_tiling(P.n);
    if (!explicit_csr && P.conn_kind == SPK_CONN_FIXED_IN &&
        ((P.k_in_exc > 0 && net->n_exc == 0) || (P.k_in_inh > 0 && net->n_exc == P.n)))
        return fail(SPK_EINVAL, "fixed in-degree needs a non-empty source population");
    if (P.ext_lambda > 0.0) {
        const int L = poisson_thresholds(P.ext_lambda, net->pois);
        if (L < 0) return fail(SPK_EINVAL, "ext_lambda");
        net->pois_len = (uint32_t)L;
        net->guide = poisson_guide(net->pois);
    }
    if (P.acc_mode == SPK_ACC_FIXED) {
        if (P.fixed_shift < 0 || P.fixed_shift > 30) return fail(SPK_EINVAL, "fixed_shift in 0..30");
        int32_t dummy;
        const int S = P.fixed_shift;
        if (!quantise(P.ext_w, S, &net->ext_wq) || !quantise(P.i_bias, S, &net->bias_q) ||
            !quantise(P.w_exc, S, &dummy) || !quantise(P.w_inh, S, &dummy) ||
            !quantise(P.w_lo, S, &dummy) || !quantise(P.w_hi, S, &dummy))
            return fail(SPK_EOVERFLOW, "a weight does not fit int32 at this fixed_shift");
    }
    if (!explicit_csr) {  // population weights: class 0 excitatory, 1 inhibitory
        const float w[2] = {P.w_exc, P.w_inh};
        SPK_TRY(choose_format(net, P.w_uniform ? nullptr : w, 2));
    }
    const uint64_t seed = P.seed;
    net->keys.conn = stream_key(seed, TAG_CONN);
    net->keys.tgt = stream_key(seed, TAG_TGT);
    net->keys.src_e = stream_key(seed, TAG_SRC_E);
    net->keys.src_i = stream_key(seed, TAG_SRC_I);
    net->keys.w = stream_key(seed, TAG_W);
    net->keys.delay = stream_key(seed, TAG_DELAY);
    net->keys.v0 = stream_key(seed, TAG_V0);
    net->keys.pois = stream_key(seed, TAG_POIS);
    net->keys.bern = stream_key(seed, TAG_BERN);
    return SPK_OK;
}

spk_status setup_stream(spk_net *net, void *stream)
{
    SPK_HIP(hipGetDevice(&net->device));
    SPK_TRY(scratch_lookup(net->device));
    if (stream) {
        net->stream = (hipStream_t)stream;
    } else {
        SPK_HIP(hipStreamCreateWithFlags(&net->stream, hipStreamNonBlocking));
        net->own_stream = true;
    }
    SPK_HIP(hipStreamCreateWithFlags(&net->cap_stream, hipStreamNonBlocking));
    return SPK_OK;
}

// Row offsets from per-row counts.
spk_status finish_counts(spk_net *net, const uint32_t *cnt)
{
    hipStream_t s = net->stream;
    const uint64_t n = net->n;
    uint64_t *bsum = nullptr;
    uint32_t *maxp = nullptr;
    SPK_TRY(dalloc(net, &net->row_ptr, n + 1));
    SPK_TRY(dalloc(net, &bsum, scan_scratch_elems(n) + 1));
    SPK_TRY(dalloc(net, &maxp, 1));
    SPK_HIP(hipMemsetAsync(maxp, 0, 4, s));
    SegTimer tm;
    SPK_HIP(tm.start(s));
    SPK_HIP(scan_counts(cnt, n, net->row_ptr, bsum, maxp, s));
    SPK_HIP(tm.stop(s, &net->gen_ms));
    uint64_t nnz = 0;
    uint32_t mr = 0;
    SPK_HIP(hipMemcpyAsync(&nnz, net->row_ptr + n, 8, hipMemcpyDeviceToHost, s));
    SPK_HIP(hipMemcpyAsync(&mr, maxp, 4, hipMemcpyDeviceToHost, s));
    SPK_HIP(hipStreamSynchronize(s));
    dfree(net, bsum);
    dfree(net, maxp);
    net->nnz = nnz;
    net->max_row = mr;
    return SPK_OK;
}

// Delivery strategy and the row index it needs.  Direct: every tile reads
// its run of each due row (rows long compared with the tile count, one
// delay, offsets small next to the synapses).  Binned: the push kernel sorts
// each fired row's events by (arrival step, tile) into pages.
spk_status choose_delivery(spk_net *net, RowIndex *ix)
{
    if (net->max_row > kMaxRow)
        return fail(SPK_EINVAL, "a source row of " + std::to_string(net->max_row) +
                                    " synapses exceeds the supported " + std::to_string(kMaxRow));
    const Tiling &tl = net->tl;
    const double mean_row = (double)net->nnz / (double)net->n;
    const double toff_bytes = (double)net->n * (tl.T + 1) * 2.0;
    const bool binned_ok = (uint64_t)net->lists * tl.T8 <= kMaxBuckets;
    bool direct = net->lists == 1 && mean_row >= 2.0 * tl.T && toff_bytes <= 0.5 * 8.0 * (double)net->nnz;
    // With a smallest delay of two steps or more, no event filed at t is
    // needed at t + 1: binned delivery lets the persistent kernel run steps
    // in batches and file a whole batch's events at once (or file them beside
    // the updates), which beats reading the due rows at arrival.
    if (direct && net->dmin >= 2 && net->P.step_mode != SPK_STEP_GRAPH && binned_ok) direct = false;
    if (!binned_ok || net->P.delivery == SPK_DELIVERY_DIRECT) direct = true;
    if (net->P.delivery == SPK_DELIVERY_BINNED) {
        if (!binned_ok)
            return fail(SPK_EINVAL, "binned delivery supports at most 2048 (delay, tile) buckets per "
                                    "XCD group; use fewer delays or direct delivery");
        direct = false;
    }
    net->direct = direct;
    *ix = RowIndex{};
    if (direct) {
        SPK_TRY(dalloc(net, &net->toff, (size_t)net->n * (tl.T + 1)));
        ix->toff = net->toff;
    } else {
        SPK_TRY(dalloc(net, &net->desc, net->n));
        ix->desc = net->desc;
    }
    return SPK_OK;
}

// Out-degrees, accumulator range, delivery buffers.
spk_status finish_rows(spk_net *net)
{
    hipStream_t s = net->stream;
    SPK_TRY(dalloc(net, &net->outdeg, net->n));
    if (net->proc) {  // every row has k_out synapses
        const std::vector<uint32_t> deg(net->n, net->P.k_out);
        SPK_HIP(hipMemcpyAsync(net->outdeg, deg.data(), (size_t)net->n * 4, hipMemcpyHostToDevice, s));
        SPK_HIP(hipStreamSynchronize(s));
    } else {
        SPK_HIP(out_degree(net->row_ptr, net->n, net->outdeg, s));
    }

    // Accumulator range.  Fixed mode: all in-synapses of one neuron at once,
    // plus the largest Poisson count and the bias, must fit in int32.  fp32
    // mode: choose the 64-bit fixed-point unit 2^-S64 as fine as the largest
    // possible sum allows.
    const bool fixed = net->P.acc_mode == SPK_ACC_FIXED;
    uint64_t m = 0;
    bool done = false;
    if (range_by_tiles(net)) SPK_TRY(fo_range(net, &m, &done));
    if (done) {
        // (the range is known)
    } else if (net->P.conn_kind == SPK_CONN_FIXED_IN && !net->P.w_uniform) {
        // every neuron has exactly k_in_exc excitatory and k_in_inh
        // inhibitory in-synapses, each with its population's weight: the
        // largest sum is every neuron's, no pass over the synapses needed
        uint64_t te = 0, ti = 0;
        SPK_TRY(abs_term(net, net->P.w_exc, &te));
        SPK_TRY(abs_term(net, net->P.w_inh, &ti));
        m = (uint64_t)net->P.k_in_exc * te + (uint64_t)net->P.k_in_inh * ti;
    } else if (range_by_targets(net)) {
        // Bernoulli: the pair predicate evaluated per target (n^2 hashes)
        // costs less than a global atomic per synapse above ~1.4 % density
        uint64_t *mx = nullptr, *insum = nullptr;
        SPK_TRY(dalloc(net, &mx, 1));
        SPK_HIP(hipMemsetAsync(mx, 0, 8, s));
        if (bern_src_ranges(net->n) > 1) {
            SPK_TRY(dalloc(net, &insum, net->n));
            SPK_HIP(hipMemsetAsync(insum, 0, (size_t)net->n * 8, s));
        }
        SegTimer tm;
        SPK_HIP(tm.start(s));
        SPK_HIP(bern_in_abs_max(conn_args(net), mx, insum, s));
        SPK_HIP(tm.stop(s, &net->range_ms));
        SPK_HIP(hipMemcpyAsync(&m, mx, 8, hipMemcpyDeviceToHost, s));
        SPK_HIP(hipStreamSynchronize(s));
        dfree(net, mx);
        if (insum) dfree(net, insum);
    } else {
        uint64_t *insum = nullptr, *mx = nullptr;
        SPK_TRY(dalloc(net, &insum, net->n));
        SPK_TRY(dalloc(net, &mx, 1));
        SPK_HIP(hipMemsetAsync(insum, 0, (size_t)net->n * 8, s));
        SPK_HIP(hipMemsetAsync(mx, 0, 8, s));
        SegTimer tm;
        SPK_HIP(tm.start(s));
        if (net->proc) SPK_HIP(proc_in_abs_sum(step_args(net), insum, s));
        else SPK_HIP(in_abs_sum(syn_ptr(net), net->nnz, fixed, net->compact, net->ctab, insum, s));
        SPK_HIP(max_u64(insum, net->n, mx, s));
        SPK_HIP(tm.stop(s, &net->range_ms));
        SPK_HIP(hipMemcpyAsync(&m, mx, 8, hipMemcpyDeviceToHost, s));
        SPK_HIP(hipStreamSynchronize(s));
        dfree(net, insum);
        dfree(net, mx);
    }
    if (fixed) {
        const uint64_t kmax = net->pois_len ? net->pois_len - 1 : 0;
        const uint64_t extra = kmax * (uint64_t)std::llabs((long long)net->ext_wq) +
                               (uint64_t)std::llabs((long long)net->bias_q);
        if (m + extra > 2147483647ull)
            return fail(SPK_EOVERFLOW, "fixed-point inputs could exceed int32; lower fixed_shift");
    } else {
        // every reachable |sum| stays below 2^52 (M <= 2^e): exact in double
        const double M = std::ldexp((double)m, -24);
        const int e = M > 0.0 ? (int)std::ceil(std::log2(M)) : 0;
        net->shift64 = std::max(0, std::min(100, 52 - e));
    }
    class_units(net);

    // Steps per batch of the persistent kernel (binned delivery): up
    // to the smallest delay, so that nothing a batch files arrives within it,
    // and within the bucket, slot and LDS limits.
    const Tiling &tl = net->tl;
    net->run_D = 1;
    if (!net->direct) {
        // Default at most 8 steps: longer batches save hand-offs but give a
        // push block more events than one 16K-event sorting window holds
        // (measured on the delay-15 network: 7.3 us per step at 8, 7.4 at
        // 10, 7.6 at 12, 7.9 at 15).  SPK_BATCH_STEPS sets the cap (1..16).
        uint32_t cap = 8;
        if (const char *e = std::getenv("SPK_BATCH_STEPS")) {
            const long v = std::strtol(e, nullptr, 10);
            if (v >= 1) cap = (uint32_t)std::min<long>(v, kRunMaxD);
        }
        uint32_t D = std::min<uint32_t>(net->dmin, cap);
        // the tile keeps one accumulator array per step of the batch in LDS
        while (D > 1 && ((uint64_t)(D + net->lists - 1) * tl.T8 > kRunMaxBuckets || D * tl.W > kMaxTileW)) D--;
        net->run_D = D;
    }
    // Spike lists: direct delivery reads the lists of steps t - dmax .. t - dmin
    // while writing that of t; binned delivery consumes the list of t within t,
    // but in the persistent kernel one XCD may publish t + 1 while another
    // still reads t, so there are three; with batches of
    // D steps, one XCD may publish the next batch while another reads this one.
    net->spk_slots = net->direct ? net->dmax + 1 : std::max<uint32_t>(3, 2 * net->run_D);
    if (!net->direct) {
        // Pages: (group, push block, arrival slot, tile).  A page never holds
        // more than nnz records (each synapse arrives at most once per slot),
        // so small networks never overflow; large ones get an equal share of
        // the budget and fall back to global atomics beyond it.
        net->pslots = net->dmax;
        net->pg1 = push_blocks_per_group();
        // procedural rows are generated once, by one push block per compute
        // unit, whose pages cover every group (graph path: the kernel boundary
        // makes them visible on every XCD), where its buckets fit
        net->proc_once = net->proc && (uint64_t)net->lists * tl.T <= kOnceMaxB;
        if (const char *e = std::getenv("SPK_PROC_ONCE"))  // 0: the per-group push (tests)
            if (e[0] == '0') net->proc_once = false;
        if (net->proc_once) net->pg1 *= kGroups;
        const uint64_t n_pages = (uint64_t)kGroups * net->pg1 * net->pslots * tl.T8;
        uint64_t cap = std::min<uint64_t>(kPageBudget / n_pages, std::max<uint64_t>(net->nnz, 1));
        if (const char *e = std::getenv("SPK_PAGE_CAP")) {
            const long long v = std::strtoll(e, nullptr, 10);
            if (v >= 1 && v <= (1ll << 30)) cap = (uint64_t)v;
        }
        cap = std::max<uint64_t>(16, (cap + 15) / 16 * 16);
        if (n_pages * cap >= (1ull << 32))  // page records are addressed with 32-bit indices
            return fail(SPK_EINVAL, "page capacity too large: pages x records must stay below 2^32");
        net->page_cap = (uint32_t)cap;
        const size_t acc_elems = (size_t)net->pslots * tl.T * tl.W;
        if (net->compact) SPK_TRY(dalloc(net, &net->pages16, n_pages * cap));
        else SPK_TRY(dalloc(net, &net->pages, n_pages * cap));
        SPK_TRY(dalloc(net, &net->pfill, n_pages));
        SPK_TRY(dalloc(net, &net->ovf_flag, (size_t)net->pslots * tl.T));
        SPK_TRY(dalloc(net, (uint64_t **)&net->acc_ovf, acc_elems));
        SPK_HIP(hipMemsetAsync(net->pfill, 0, n_pages * 4, s));
        SPK_HIP(hipMemsetAsync(net->ovf_flag, 0, (size_t)net->pslots * tl.T * 4, s));
        SPK_HIP(hipMemsetAsync(net->acc_ovf, 0, acc_elems * 8, s));
    }
    SPK_HIP(hipStreamSynchronize(s));
    return SPK_OK;
}

// Procedural synapses: nothing is generated or stored at creation; every
// row has k_out synapses, drawn when its source fires (binned delivery).
spk_status generate_proc(spk_net *net)
{
    net->nnz = (uint64_t)net->n * net->P.k_out;
    net->max_row = net->P.k_out;
    if ((uint64_t)net->lists * net->tl.T8 > kMaxBuckets)
        return fail(SPK_EINVAL, "binned delivery supports at most 2048 (delay, tile) buckets per XCD group");
    net->direct = false;
    return finish_rows(net);
}

spk_status generate(spk_net *net)
{
    if (net->proc) return generate_proc(net);
    hipStream_t s = net->stream;
    uint32_t *cnt = nullptr;
    SPK_TRY(dalloc(net, &cnt, net->n));
    SPK_HIP(hipMemsetAsync(cnt, 0, (size_t)net->n * 4, s));
    ConnArgs c = conn_args(net);
    const bool in_rows = net->P.conn_kind == SPK_CONN_FIXED_IN;
    // Bernoulli rows: the count pass keeps every row's bucket counts (u16,
    // both deliveries' buckets), so the placement pass draws each row once
    // (SPK_GEN_HIST=0 skips it, as when it cannot be allocated: a test knob)
    uint16_t *hist = nullptr;
    const uint64_t hist_elems = (uint64_t)net->n * (net->tl.T + 2 * kGroups);
    const char *gh = std::getenv("SPK_GEN_HIST");
    const bool want_hist = !(gh && std::strcmp(gh, "0") == 0);
    if (net->P.conn_kind == SPK_CONN_BERNOULLI && want_hist && hist_elems * 2 <= (4ull << 30) &&
        dalloc(net, &hist, hist_elems) != SPK_OK) {
        hist = nullptr;          // (then the placement pass counts for itself)
        (void)hipGetLastError();  // the failed allocation is not an error of the launches below
    }
    // ... and keeps each row's synapses, up to cap = mean + 10 sd + 64 per
    // row, so that the placement pass need not draw the rows again (unless a
    // row turns out longer, or the keys would take more than 32 GB)
    uint32_t *keys = nullptr;
    uint32_t cap = 0;
    const char *gk = std::getenv("SPK_GEN_KEYS");
    if (hist && !(gk && std::strcmp(gk, "0") == 0)) {
        const double p = net->P.p, nn = (double)net->n;
        const double capd = std::ceil(p * nn + 10.0 * std::sqrt(nn * p * (1.0 - p)) + 64.0);
        if (capd <= (double)kMaxRow && (double)net->n * capd * 4.0 <= (double)(32ull << 30)) {
            cap = (uint32_t)capd;
            if (dalloc(net, &keys, (size_t)net->n * cap) != SPK_OK) {
                keys = nullptr;
                (void)hipGetLastError();
            }
        }
    }
    SegTimer tm;
    SPK_HIP(tm.start(s));
    if (in_rows) SPK_HIP(gen_in_count(c, cnt, s));
    else SPK_HIP(gen_count_rows(c, cnt, hist, keys, cap, s));
    SPK_HIP(tm.stop(s, &net->gen_ms));
    SPK_TRY(finish_counts(net, cnt));
    if (keys && net->max_row > cap) {  // a row did not fit: placement draws the rows again
        dfree(net, keys);
        keys = nullptr;
    }
    RowIndex ix{};
    SPK_TRY(choose_delivery(net, &ix));
    void *syn = nullptr;
    SPK_TRY(alloc_syn(net, &syn, net->nnz));
    if (net->compact) net->syn32 = (uint32_t *)syn;
    else net->syn = (int2 *)syn;
    if (in_rows) {  // drawn per target: regroup by source, then bucket
        void *tmp = nullptr;
        SPK_TRY(alloc_syn(net, &tmp, net->nnz));
        SPK_HIP(hipMemsetAsync(cnt, 0, (size_t)net->n * 4, s));
        SPK_HIP(tm.start(s));
        SPK_HIP(gen_in_fill(c, net->row_ptr, cnt, tmp, s));
        SPK_HIP(bucket_rows(c, net->row_ptr, tmp, syn, ix, s));
        SPK_HIP(tm.stop(s, &net->gen_ms));
        dfree(net, tmp);
    } else {        // drawn per source, bucketed while drawn
        SPK_HIP(tm.start(s));
        SPK_HIP(gen_fill_rows(c, net->row_ptr, syn, ix, hist, keys, cap, s));
        SPK_HIP(tm.stop(s, &net->gen_ms));
    }
    SPK_HIP(hipStreamSynchronize(s));
    dfree(net, cnt);
    dfree(net, hist);
    dfree(net, keys);
    return finish_rows(net);
}

// State, spike lists and per-step records.
spk_status alloc_state(spk_net *net)
{
    const uint32_t n = net->n;
    const uint64_t T = net->P.max_steps;
    const Tiling &tl = net->tl;
    hipStream_t s = net->stream;
    const uint64_t segs = (uint64_t)net->spk_slots * tl.T;
    SPK_TRY(dalloc(net, &net->V, n));
    SPK_TRY(dalloc(net, &net->ref, n));
    SPK_TRY(dalloc(net, &net->spk_ids, segs * tl.W));
    SPK_TRY(dalloc(net, &net->spk_cnt, segs));
    SPK_TRY(dalloc(net, &net->counts8, T * kGroups));
    SPK_TRY(dalloc(net, &net->events8, T * kGroups));
    SPK_TRY(dalloc(net, &net->delivered8, T * kGroups));
    SPK_TRY(dalloc(net, &net->flags, 1));
    SPK_TRY(dalloc(net, (uint32_t **)&net->dbg_out, n));
    SPK_TRY(dalloc(net, &net->t_base, 1));
    SPK_TRY(dalloc(net, &net->raster_offs, T + 1));
    SPK_TRY(dalloc(net, &net->raster, net->P.raster_capacity));
    SPK_TRY(dalloc(net, &net->pois_dev, net->pois_len ? net->pois_len : 1));
    SPK_TRY(dalloc(net, &net->guide_dev, 256));
    SPK_HIP(hipMemsetAsync(net->spk_cnt, 0, segs * 4, s));
    SPK_HIP(hipMemsetAsync(net->counts8, 0, T * kGroups * 4, s));
    SPK_HIP(hipMemsetAsync(net->events8, 0, T * kGroups * 8, s));
    SPK_HIP(hipMemsetAsync(net->delivered8, 0, T * kGroups * 8, s));
    SPK_HIP(hipMemsetAsync(net->flags, 0, 4, s));
    SPK_HIP(hipMemsetAsync(net->t_base, 0, 8, s));
    SPK_HIP(hipMemsetAsync(net->raster_offs, 0, (T + 1) * 8, s));
    SPK_HIP(hipMemsetAsync(net->guide_dev, 0, 512, s));
    if (net->pois_len) {
        SPK_HIP(hipMemcpyAsync(net->pois_dev, net->pois.data(), net->pois_len * 8,
                               hipMemcpyHostToDevice, s));
        SPK_HIP(hipMemcpyAsync(net->guide_dev, net->guide.data(), 512, hipMemcpyHostToDevice, s));
    }
    ModelArgs m = model_args(net);
    SPK_HIP(init_state(m, net->P.v0_lo, net->P.v0_hi, net->V, net->ref, s));
    SPK_HIP(hipStreamSynchronize(s));  // host tables above are stack/vector memory
    return SPK_OK;
}

spk_status check_ready(spk_net *net)
{
    if (!net) return fail(SPK_EINVAL, "null network");
    return SPK_OK;
}

spk_status sync_flags(spk_net *net, uint32_t *flags_out)
{
    SPK_HIP(hipStreamSynchronize(net->stream));
    uint32_t f = 0;
    SPK_HIP(hipMemcpy(&f, net->flags, 4, hipMemcpyDeviceToHost));
    if (flags_out) *flags_out = f;
    if (f & kFlagRunStopped)
        return fail(SPK_EHIP, "a persistent step launch stopped early (a barrier wait exceeded its "
                              "bound); the network state is undefined");
    if (f & kFlagBadSpike) {  // reported once, then cleared: the network is unchanged
        const uint32_t g = f & ~kFlagBadSpike;
        SPK_HIP(hipMemcpy(net->flags, &g, 4, hipMemcpyHostToDevice));
        return fail(SPK_EINVAL, "a spike ID given to spk_deliver_noalloc was >= n; those spikes "
                                "delivered nothing");
    }
    return SPK_OK;
}

RunArgs run_args(const spk_net *net, uint64_t t0, uint64_t n_steps)
{
    RunArgs ra{};
    ra.s = step_args(net);
    ra.ctl = net->ctl;
    ra.t0 = t0;
    ra.n_steps = n_steps;
    ra.R = net->run_R;
    ra.D = net->direct ? 1u : net->run_D;
    return ra;
}

hipError_t launch_persistent(const spk_net *net, const RunArgs &ra, hipStream_t s)
{
    (void)net;
    return launch_run(ra, s);
}

// A zero-step launch of the persistent kernel: checks that the workgroups
// were placed evenly over the XCDs (it only loads and stores back state).
spk_status probe_persistent(spk_net *net, bool *ok)
{
    hipStream_t s = net->stream;
    *ok = false;
    SPK_HIP(hipMemsetAsync(net->ctl, 0, sizeof(RunCtl), s));
    hipError_t e = launch_persistent(net, run_args(net, net->t, 0), s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    uint32_t abort_flag = 1;
    if (e == hipSuccess) e = hipMemcpy(&abort_flag, &net->ctl->abort_flag, 4, hipMemcpyDeviceToHost);
    if (e == hipSuccess && abort_flag == 0) {
        *ok = true;
        return SPK_OK;
    }
    (void)hipGetLastError();
    (void)hipStreamSynchronize(s);
    SPK_HIP(hipMemsetAsync(net->flags, 0, 4, s));  // the probe's stop flag
    SPK_HIP(hipStreamSynchronize(s));
    return SPK_OK;
}

// Step mode.  The persistent kernel needs a cooperative launch of one
// workgroup per compute unit spread evenly over the XCDs; a launch of zero
// steps checks that once (it only loads and stores back the state).
spk_status choose_step_mode(spk_net *net)
{
    net->persistent = false;
    const uint32_t mode = net->P.step_mode;
    if (mode == SPK_STEP_GRAPH) return SPK_OK;
    int coop = 0;
    SPK_HIP(hipDeviceGetAttribute(&coop, hipDeviceAttributeCooperativeLaunch, net->device));
    const int cus = cu_count();
    net->run_R = cus > 0 && cus % (int)kGroups == 0 ? (uint32_t)(cus / (int)kGroups) : 0u;
    const StepArgs a = step_args(net);
    const bool run_fits = coop && run_supported(a, net->run_R) && run_batch_supported(a, net->direct ? 1u : net->run_D);
    if (!run_fits) {
        if (mode == SPK_STEP_PERSISTENT)
            return fail(SPK_EINVAL, "the persistent step kernel does not apply to this network or device "
                                    "(tiles per XCD, delays, or cooperative launch)");
        return SPK_OK;
    }
    SPK_TRY(dalloc(net, &net->ctl, 1));
    bool ok = false;
    SPK_TRY(probe_persistent(net, &ok));
    if (ok) {
        net->persistent = true;
        return SPK_OK;
    }
    dfree(net, net->ctl);
    net->ctl = nullptr;
    if (mode == SPK_STEP_PERSISTENT)
        return fail(SPK_EHIP, "the persistent step kernel could not be placed evenly over the XCDs");
    return SPK_OK;
}

spk_status collect_profile(spk_net *net)
{
    SPK_HIP(hipStreamSynchronize(net->stream));
    for (int which = 0; which < 3; which++) {
        auto &v = which == 2 ? net->ev_run : which ? net->ev_tile : net->ev_push;
        double &acc = which == 2 ? net->ms_run : which ? net->ms_tile : net->ms_push;
        for (auto &pr : v) {
            float ms = 0;
            SPK_HIP(hipEventElapsedTime(&ms, pr.first, pr.second));
            acc += ms;
            net->ev_free.push_back(pr.first);
            net->ev_free.push_back(pr.second);
        }
        v.clear();
    }
    return SPK_OK;
}

spk_status get_event(spk_net *net, hipEvent_t *e)
{
    if (!net->ev_free.empty()) {
        *e = net->ev_free.back();
        net->ev_free.pop_back();
        return SPK_OK;
    }
    SPK_HIP(hipEventCreate(e));
    return SPK_OK;
}

// One step's kernels on stream s (step i of a batch, or explicit t).
spk_status enqueue_step(spk_net *net, const StepArgs &a, hipStream_t s, uint32_t i, int64_t t_explicit)
{
    SPK_HIP(launch_tile(a, i, t_explicit, s));
    if (!net->direct) SPK_HIP(launch_push(a, i, t_explicit, s));
    if (net->P.raster_capacity) SPK_HIP(launch_record(a, i, t_explicit, s));
    return SPK_OK;
}

// A graph of B steps followed by the step-counter advance, built once.
spk_status batch_graph(spk_net *net, uint32_t B, hipGraphExec_t *out)
{
    auto it = net->graphs.find(B);
    if (it != net->graphs.end()) {
        *out = it->second;
        return SPK_OK;
    }
    const StepArgs a = step_args(net);
    hipStream_t cs = net->cap_stream;
    SPK_HIP(hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal));
    spk_status st = SPK_OK;
    for (uint32_t i = 0; i < B && st == SPK_OK; i++) st = enqueue_step(net, a, cs, i, -1);
    if (st == SPK_OK && launch_advance(net->t_base, B, cs) != hipSuccess)
        st = fail(SPK_EHIP, "advance launch");
    hipGraph_t g = nullptr;
    hipError_t e = hipStreamEndCapture(cs, &g);
    if (st != SPK_OK) {
        if (g) (void)hipGraphDestroy(g);
        return st;
    }
    SPK_HIP(e);
    hipGraphExec_t ge = nullptr;
    e = hipGraphInstantiate(&ge, g, nullptr, nullptr, 0);
    (void)hipGraphDestroy(g);
    SPK_HIP(e);
    net->graphs[B] = ge;
    *out = ge;
    return SPK_OK;
}

void destroy_net(spk_net *net)
{
    if (!net) return;
    if (net->stream) (void)hipStreamSynchronize(net->stream);
    for (auto &kv : net->graphs) (void)hipGraphExecDestroy(kv.second);
    for (auto *v : {&net->ev_push, &net->ev_tile, &net->ev_run})
        for (auto &pr : *v) {
            (void)hipEventDestroy(pr.first);
            (void)hipEventDestroy(pr.second);
        }
    for (auto e : net->ev_free) (void)hipEventDestroy(e);
    for (void *p : net->allocs) (void)hipFree(p);
    if (net->cap_stream) (void)hipStreamDestroy(net->cap_stream);
    if (net->own_stream && net->stream) (void)hipStreamDestroy(net->stream);
    delete net;
}

spk_status read_groups(spk_net *net, const void *dev, size_t elem, uint64_t t0, uint64_t n, void *out)
{
    (void)net;
    std::vector<uint8_t> buf(n * kGroups * elem);
    if (n) SPK_HIP(hipMemcpy(buf.data(), (const uint8_t *)dev + t0 * kGroups * elem, buf.size(),
                             hipMemcpyDeviceToHost));
    for (uint64_t k = 0; k < n; k++) {
        uint64_t sum = 0;
        for (uint32_t x = 0; x < kGroups; x++) {
            if (elem == 4) {
                uint32_t v;
                std::memcpy(&v, &buf[(k * kGroups + x) * 4], 4);
                sum += v;
            } else {
                uint64_t v;
                std::memcpy(&v, &buf[(k * kGroups + x) * 8], 8);
                sum += v;
            }
        }
        if (elem == 4) ((uint32_t *)out)[k] = (uint32_t)sum;
        else ((uint64_t *)out)[k] = sum;
    }
    return SPK_OK;
}

}  // namespace

// ===================================================================== ABI

extern "C" {

uint32_t spk_abi_version(void) { return SPK_ABI_VERSION; }

const char *spk_last_error(void) { return g_err.c_str(); }

spk_status spk_preset(int index, int driven, double rate_hz, uint64_t seed, spk_params *out)
{
    if (!out) return fail(SPK_EINVAL, "null output");
    spk_params p{};
    p.abi_version = SPK_ABI_VERSION;
    p.seed = seed;
    p.neuron_kind = SPK_LIF;
    p.frac_exc = 0.8;
    p.dt_ms = 0.1;
    p.tau_m_ms = 20.0;
    p.t_ref_ms = 5.0;
    p.v_rest = -60.0f;
    p.v_th = -50.0f;
    p.v_reset = -60.0f;
    p.v0_lo = -60.0f;
    p.v0_hi = -50.0f;
    p.delay_min = p.delay_max = 1;
    p.acc_mode = SPK_ACC_F32;
    p.fixed_shift = 20;
    switch (index) {
    case 0:
        p.n = 1000; p.conn_kind = SPK_CONN_BERNOULLI; p.p = 0.02;
        p.w_exc = 0.27f; p.w_inh = -4.5f; p.max_steps = 1000;
        break;
    case 1: {
        p.n = 250000; p.conn_kind = SPK_CONN_BERNOULLI; p.p = 0.02;
        const double sc = 80.0 / (0.02 * p.n);
        p.w_exc = (float)(0.27 * sc); p.w_inh = (float)(-4.5 * sc); p.max_steps = 10000;
        break;
    }
    case 2:
        p.n = 100000; p.conn_kind = SPK_CONN_FIXED_IN; p.k_in_exc = 8000; p.k_in_inh = 2000;
        p.w_exc = 0.1f; p.w_inh = -0.5f; p.delay_min = p.delay_max = 15;
        p.ext_lambda = 1.0; p.ext_w = 0.1f; p.max_steps = 10000;
        break;
    case 3:
        p.n = 1000000; p.neuron_kind = SPK_SOURCE; p.frac_exc = 1.0; p.dt_ms = 1.0;
        p.conn_kind = SPK_CONN_FIXED_OUT; p.k_out = 1000; p.w_uniform = 1; p.w_lo = 0.0f;
        p.w_hi = 1e-3f; p.src_rate_hz = rate_hz; p.max_steps = 1000;
        break;
    case 4: {
        p.n = 2000000; p.conn_kind = SPK_CONN_FIXED_OUT; p.k_out = 1500;
        const double sc = 80.0 / 1500.0;
        p.w_exc = (float)(0.27 * sc); p.w_inh = (float)(-4.5 * sc);
        p.delay_min = 1; p.delay_max = 20; p.max_steps = 5000;
        break;
    }
    default:
        return fail(SPK_EINVAL, "preset index must be 0..4");
    }
    if (driven && p.neuron_kind == SPK_LIF && p.ext_lambda == 0.0) {
        const double theta = (double)p.v_th - (double)p.v_rest;
        p.ext_lambda = 2.0 * theta * (p.dt_ms / p.tau_m_ms) / (double)p.w_exc;
        p.ext_w = p.w_exc;
    }
    *out = p;
    return SPK_OK;
}

spk_status spk_create(const spk_params *params, void *stream, spk_net **out)
{
    if (!params || !out) return fail(SPK_EINVAL, "null argument");
    *out = nullptr;
    const auto t_begin = std::chrono::steady_clock::now();
    spk_net *net = new (std::nothrow) spk_net();
    if (!net) return fail(SPK_ENOMEM, "host allocation");
    net->P = *params;
    spk_status st = derive(net, false);
    if (st == SPK_OK) st = setup_stream(net, stream);
    if (st == SPK_OK) st = generate(net);
    if (st == SPK_OK) st = alloc_state(net);
    if (st == SPK_OK) st = choose_step_mode(net);
    if (st == SPK_OK) st = sync_flags(net, nullptr);
    if (st != SPK_OK) {
        std::string msg = g_err;
        destroy_net(net);
        g_err = msg;
        return st;
    }
    net->setup_ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t_begin).count();
    *out = net;
    return SPK_OK;
}

spk_status spk_create_from_csr(const spk_params *params, uint32_t n, const uint64_t *row_ptr,
                               const uint32_t *col, const float *w, const uint8_t *delay,
                               void *stream, spk_net **out)
{
    if (!params || !out || !row_ptr || (row_ptr[n] && (!col || !w)))
        return fail(SPK_EINVAL, "null argument");
    *out = nullptr;
    const auto t_begin = std::chrono::steady_clock::now();
    spk_net *net = new (std::nothrow) spk_net();
    if (!net) return fail(SPK_ENOMEM, "host allocation");
    net->P = *params;
    net->P.n = n;
    net->P.conn_kind = SPK_CONN_EXPLICIT;
    auto run = [&]() -> spk_status {
        SPK_TRY(derive(net, true));
        if (row_ptr[0] != 0) return fail(SPK_EINVAL, "row_ptr[0] must be 0");
        uint64_t max_row = 0;
        for (uint32_t s = 0; s < n; s++) {
            if (row_ptr[s + 1] < row_ptr[s]) return fail(SPK_EINVAL, "row_ptr not monotone");
            max_row = std::max<uint64_t>(max_row, row_ptr[s + 1] - row_ptr[s]);
        }
        const uint64_t nnz = row_ptr[n];
        std::vector<uint32_t> distinct;  // weight bit patterns, first-seen order, up to 5
        for (uint64_t e = 0; e < nnz && distinct.size() <= kMaxClasses; e++) {
            uint32_t b;
            std::memcpy(&b, &w[e], 4);
            if (std::find(distinct.begin(), distinct.end(), b) == distinct.end()) distinct.push_back(b);
        }
        {
            float cls[kMaxClasses] = {};
            const bool fits = distinct.size() <= kMaxClasses;
            for (size_t k = 0; fits && k < distinct.size(); k++) std::memcpy(&cls[k], &distinct[k], 4);
            if (fits && distinct.empty()) cls[0] = 0.0f;
            SPK_TRY(choose_format(net, fits ? cls : nullptr,
                                  fits ? std::max<uint32_t>(1, (uint32_t)distinct.size()) : 0));
        }
        for (uint64_t e = 0; e < nnz; e++) {
            if (col[e] >= n) return fail(SPK_EINVAL, "target id out of range");
            const uint32_t d = delay ? delay[e] : net->P.delay_min;
            if (d < net->P.delay_min || d > net->P.delay_max)
                return fail(SPK_EINVAL, "delay out of [delay_min, delay_max]");
            if (net->P.acc_mode == SPK_ACC_FIXED) {
                int32_t q;
                if (!quantise(w[e], net->P.fixed_shift, &q))
                    return fail(SPK_EOVERFLOW, "a weight does not fit int32 at this fixed_shift");
            }
        }
        net->nnz = nnz;
        net->max_row = (uint32_t)std::min<uint64_t>(max_row, 0xffffffffull);
        SPK_TRY(setup_stream(net, stream));
        hipStream_t s = net->stream;
        RowIndex ix{};
        SPK_TRY(choose_delivery(net, &ix));
        uint32_t *in_col = nullptr;
        float *in_w = nullptr;
        uint8_t *in_d = nullptr;
        void *tmp = nullptr, *syn = nullptr;
        SPK_TRY(dalloc(net, &net->row_ptr, (size_t)n + 1));
        SPK_TRY(alloc_syn(net, &syn, nnz));
        if (net->compact) net->syn32 = (uint32_t *)syn;
        else net->syn = (int2 *)syn;
        SPK_TRY(alloc_syn(net, &tmp, nnz));
        SPK_TRY(dalloc(net, &in_col, nnz));
        SPK_TRY(dalloc(net, &in_w, nnz));
        SPK_HIP(hipMemcpyAsync(net->row_ptr, row_ptr, ((size_t)n + 1) * 8, hipMemcpyHostToDevice, s));
        if (nnz) {
            SPK_HIP(hipMemcpyAsync(in_col, col, nnz * 4, hipMemcpyHostToDevice, s));
            SPK_HIP(hipMemcpyAsync(in_w, w, nnz * 4, hipMemcpyHostToDevice, s));
        }
        if (delay) {
            SPK_TRY(dalloc(net, &in_d, nnz));
            if (nnz) SPK_HIP(hipMemcpyAsync(in_d, delay, nnz, hipMemcpyHostToDevice, s));
        }
        ConnArgs c = conn_args(net);
        SPK_HIP(csr_fill(c, nnz, in_col, in_w, in_d, tmp, s));
        SPK_HIP(bucket_rows(c, net->row_ptr, tmp, syn, ix, s));
        SPK_HIP(hipStreamSynchronize(s));
        dfree(net, tmp);
        dfree(net, in_col);
        dfree(net, in_w);
        dfree(net, in_d);
        SPK_TRY(finish_rows(net));
        SPK_TRY(alloc_state(net));
        SPK_TRY(choose_step_mode(net));
        return sync_flags(net, nullptr);
    };
    spk_status st = run();
    if (st != SPK_OK) {
        std::string msg = g_err;
        destroy_net(net);
        g_err = msg;
        return st;
    }
    net->setup_ms = std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t_begin).count();
    *out = net;
    return SPK_OK;
}

spk_status spk_step(spk_net *net, uint64_t n_steps)
{
    SPK_TRY(check_ready(net));
    if (net->t + n_steps > net->P.max_steps)
        return fail(SPK_EOVERFLOW, "max_steps exceeded");
    hipStream_t s = net->stream;
    if (net->persistent) {  // one cooperative launch per (at most 2^24) steps
        uint64_t left = n_steps;
        while (left) {
            const uint64_t B = std::min<uint64_t>(left, kRunMaxSteps);
            hipEvent_t e0 = nullptr, e1 = nullptr;
            if (net->profiling) {
                SPK_TRY(get_event(net, &e0));
                SPK_TRY(get_event(net, &e1));
            }
            SPK_HIP(hipMemsetAsync(net->ctl, 0, sizeof(RunCtl), s));
            if (e0) SPK_HIP(hipEventRecord(e0, s));
            SPK_HIP(launch_persistent(net, run_args(net, net->t, B), s));
            if (e1) {
                SPK_HIP(hipEventRecord(e1, s));
                net->ev_run.push_back({e0, e1});
                net->run_launches++;
                net->launches += B;
            }
            left -= B;
            net->t += B;
        }
        return SPK_OK;
    }
    if (net->profiling) {  // plain launches with events around every kernel
        const StepArgs a = step_args(net);
        for (uint64_t k = 0; k < n_steps; k++) {
            const int64_t t = (int64_t)(net->t + k);
            hipEvent_t e0 = nullptr, e1 = nullptr, e2 = nullptr, e3 = nullptr;
            SPK_TRY(get_event(net, &e0));
            SPK_TRY(get_event(net, &e1));
            SPK_HIP(hipEventRecord(e0, s));
            SPK_HIP(launch_tile(a, 0, t, s));
            SPK_HIP(hipEventRecord(e1, s));
            net->ev_tile.push_back({e0, e1});
            if (!net->direct) {
                SPK_TRY(get_event(net, &e2));
                SPK_TRY(get_event(net, &e3));
                SPK_HIP(hipEventRecord(e2, s));
                SPK_HIP(launch_push(a, 0, t, s));
                SPK_HIP(hipEventRecord(e3, s));
                net->ev_push.push_back({e2, e3});
            }
            if (net->P.raster_capacity) SPK_HIP(launch_record(a, 0, t, s));
            net->launches++;
        }
        if (n_steps) SPK_HIP(launch_advance(net->t_base, (uint32_t)n_steps, s));
        net->t += n_steps;
        return SPK_OK;
    }
    uint64_t left = n_steps;
    while (left) {
        const uint32_t B = (uint32_t)std::min<uint64_t>(left, kBatch);
        hipGraphExec_t ge = nullptr;
        SPK_TRY(batch_graph(net, B, &ge));
        SPK_HIP(hipGraphLaunch(ge, s));
        left -= B;
        net->t += B;
    }
    return SPK_OK;
}

spk_status spk_sync(spk_net *net)
{
    SPK_TRY(check_ready(net));
    return sync_flags(net, nullptr);
}

spk_status spk_read_spike_counts(spk_net *net, uint64_t t0, uint64_t n, uint32_t *out)
{
    SPK_TRY(check_ready(net));
    if (t0 + n > net->P.max_steps || (n && !out)) return fail(SPK_EINVAL, "range");
    SPK_TRY(sync_flags(net, nullptr));
    return read_groups(net, net->counts8, 4, t0, n, out);
}

spk_status spk_read_events(spk_net *net, uint64_t t0, uint64_t n, uint64_t *out)
{
    SPK_TRY(check_ready(net));
    if (t0 + n > net->P.max_steps || (n && !out)) return fail(SPK_EINVAL, "range");
    SPK_TRY(sync_flags(net, nullptr));
    return read_groups(net, net->events8, 8, t0, n, out);
}

spk_status spk_read_delivered(spk_net *net, uint64_t t0, uint64_t n, uint64_t *out)
{
    SPK_TRY(check_ready(net));
    if (t0 + n > net->P.max_steps || (n && !out)) return fail(SPK_EINVAL, "range");
    SPK_TRY(sync_flags(net, nullptr));
    return read_groups(net, net->delivered8, 8, t0, n, out);
}

spk_status spk_read_raster(spk_net *net, uint64_t t0, uint64_t n, uint64_t *offs, uint32_t *ids,
                           uint64_t cap)
{
    SPK_TRY(check_ready(net));
    if (!net->P.raster_capacity) return fail(SPK_ESTATE, "raster recording is off");
    if (t0 + n > net->t || !offs) return fail(SPK_EINVAL, "range");
    uint32_t f = 0;
    SPK_TRY(sync_flags(net, &f));
    if (f & 2u) return fail(SPK_EOVERFLOW, "raster capacity exceeded during the run");
    std::vector<uint64_t> o(n + 1);
    SPK_HIP(hipMemcpy(o.data(), net->raster_offs + t0, (n + 1) * 8, hipMemcpyDeviceToHost));
    const uint64_t total = o[n] - o[0];
    if (total > cap || (total && !ids)) return fail(SPK_EOVERFLOW, "ids buffer too small");
    if (total) SPK_HIP(hipMemcpy(ids, net->raster + o[0], total * 4, hipMemcpyDeviceToHost));
    for (uint64_t k = 0; k <= n; k++) offs[k] = o[k] - o[0];
    for (uint64_t k = 0; k < n; k++) std::sort(ids + offs[k], ids + offs[k + 1]);
    return SPK_OK;
}

spk_status spk_read_state(spk_net *net, float *v, uint8_t *ref)
{
    SPK_TRY(check_ready(net));
    SPK_TRY(sync_flags(net, nullptr));
    if (v) SPK_HIP(hipMemcpy(v, net->V, (size_t)net->n * 4, hipMemcpyDeviceToHost));
    if (ref) SPK_HIP(hipMemcpy(ref, net->ref, net->n, hipMemcpyDeviceToHost));
    return SPK_OK;
}

spk_status spk_debug_deliver(spk_net *net, const uint32_t *spikes, uint64_t n_spikes, uint32_t delay,
                             float *out_f32, int32_t *out_i32)
{
    SPK_TRY(check_ready(net));
    const bool fixed = net->P.acc_mode == SPK_ACC_FIXED;
    if ((fixed && !out_i32) || (!fixed && !out_f32))
        return fail(SPK_EINVAL, "output buffer for this accumulation mode is required");
    if (n_spikes > 0x3fffffffull || (n_spikes && !spikes)) return fail(SPK_EINVAL, "spikes");
    for (uint64_t k = 0; k < n_spikes; k++)
        if (spikes[k] >= net->n) return fail(SPK_EINVAL, "spike id out of range");
    if (delay && (delay < net->dmin || delay >= net->dmin + net->lists))
        return fail(SPK_EINVAL, "delay not in [delay_min, delay_max]");
    hipStream_t s = net->stream;
    SPK_TRY(sync_flags(net, nullptr));
    const Tiling &tl = net->tl;
    // scratch: the spike list, and for binned delivery pages of one arrival
    // slot with their fill counters and overflow accumulators, so that the
    // network's own pages (events in flight) are left untouched
    std::vector<void *> tmp;
    auto scratch = [&](void **p, size_t bytes) -> spk_status {
        uint8_t *q = nullptr;
        SPK_TRY(dalloc(net, &q, bytes));
        tmp.push_back(q);
        *p = q;
        return SPK_OK;
    };
    spk_status st = SPK_OK;
    do {
        uint32_t *d_sp = nullptr;
        if ((st = scratch((void **)&d_sp, n_spikes * 4 + 4)) != SPK_OK) break;
        StepArgs a = step_args(net);
        a.dbg_spikes = d_sp;
        a.dbg_n = (uint32_t)n_spikes;
        a.dbg_j = delay ? (int32_t)(delay - net->dmin) : -1;
        a.dbg_out = net->dbg_out;
        hipError_t e = hipSuccess;
        if (n_spikes) e = hipMemcpyAsync(d_sp, spikes, n_spikes * 4, hipMemcpyHostToDevice, s);
        if (e == hipSuccess && !net->direct) {
            const uint64_t n_pages = (uint64_t)kGroups * net->pg1 * tl.T8;
            const uint64_t cap = std::min<uint64_t>(kDebugPageCap, std::max<uint64_t>(16, net->page_cap));
            const size_t acc_elems = (size_t)tl.T * tl.W;
            void *pg = nullptr;
            if ((st = scratch(&pg, n_pages * cap * (net->compact ? 2 : 8))) != SPK_OK) break;
            a.pages = net->compact ? nullptr : (int2 *)pg;
            a.pages16 = net->compact ? (uint16_t *)pg : nullptr;
            if ((st = scratch((void **)&a.pfill, n_pages * 4)) != SPK_OK) break;
            if ((st = scratch((void **)&a.ovf_flag, (size_t)tl.T * 4)) != SPK_OK) break;
            if ((st = scratch(&a.acc_ovf, acc_elems * 8)) != SPK_OK) break;
            a.page_cap = (uint32_t)cap;
            a.pslots = 1;
            e = hipMemsetAsync(a.pfill, 0, n_pages * 4, s);
            if (e == hipSuccess) e = hipMemsetAsync(a.ovf_flag, 0, (size_t)tl.T * 4, s);
            if (e == hipSuccess) e = hipMemsetAsync(a.acc_ovf, 0, acc_elems * 8, s);
            if (e == hipSuccess) e = launch_push(a, 0, 0, s);
        }
        if (e == hipSuccess) e = launch_tile(a, 0, 0, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e == hipSuccess)
            e = hipMemcpy(fixed ? (void *)out_i32 : (void *)out_f32, net->dbg_out,
                          (size_t)net->n * 4, hipMemcpyDeviceToHost);
        if (e != hipSuccess) st = fail(SPK_EHIP, hipGetErrorString(e));
    } while (0);
    (void)hipStreamSynchronize(s);
    for (void *p : tmp) dfree(net, p);
    return st;
}

spk_status spk_deliver_noalloc(spk_net *net, const uint32_t *d_spikes, uint64_t n_spikes, uint32_t delay,
                               void *d_out)
{
    SPK_TRY(check_ready(net));
    if (!d_out) return fail(SPK_EINVAL, "output buffer required");
    if (n_spikes > 0x3fffffffull || (n_spikes && !d_spikes)) return fail(SPK_EINVAL, "spikes");
    if (delay && (delay < net->dmin || delay >= net->dmin + net->lists))
        return fail(SPK_EINVAL, "delay not in [delay_min, delay_max]");
    uint8_t *base = (uint8_t *)scratch_of(net->device);
    if (!base) return fail(SPK_ESTATE, "no scratch address for the network's device");
    hipStream_t s = net->stream;
    const Tiling &tl = net->tl;
    StepArgs a = step_args(net);
    a.dbg_spikes = n_spikes ? d_spikes : nullptr;
    a.dbg_n = (uint32_t)n_spikes;
    a.dbg_j = delay ? (int32_t)(delay - net->dmin) : -1;
    a.dbg_out = d_out;  // (no spikes: the tile kernel writes zeros)
    hipError_t e = hipSuccess;
    if (!net->direct) {
        // Carve the scratch: fill counters, overflow flags and overflow
        // accumulators of one arrival slot, then pages of as many records as
        // the rest holds (at most the debug capacity; events beyond it take
        // the overflow accumulators, with the same sums)
        auto up = [](uint64_t b) { return (b + 255) / 256 * 256; };
        const uint64_t n_pages = (uint64_t)kGroups * net->pg1 * tl.T8;
        const uint64_t acc_bytes = (uint64_t)tl.T * tl.W * (net->P.acc_mode == SPK_ACC_FIXED ? 4 : 8);
        const uint64_t o_fill = 0, o_flag = up(n_pages * 4), o_acc = o_flag + up((uint64_t)tl.T * 4);
        const uint64_t o_pages = o_acc + up(acc_bytes);
        const uint64_t rec = net->compact ? 2 : 8;
        const uint64_t room = o_pages < kNoAllocScratchBytes ? kNoAllocScratchBytes - o_pages : 0;
        uint64_t cap = std::min<uint64_t>(room / (n_pages * rec), std::min<uint64_t>(kDebugPageCap, net->page_cap));
        cap = cap / 16 * 16;
        if (cap < 16)
            return fail(SPK_EOVERFLOW, "network too large for the fixed scratch of spk_deliver_noalloc (" +
                                           std::to_string(kNoAllocScratchBytes >> 20) + " MiB per device)");
        a.pfill = (uint32_t *)(base + o_fill);
        a.ovf_flag = (uint32_t *)(base + o_flag);
        a.acc_ovf = base + o_acc;
        a.pages = net->compact ? nullptr : (int2 *)(base + o_pages);
        a.pages16 = net->compact ? (uint16_t *)(base + o_pages) : nullptr;
        a.page_cap = (uint32_t)cap;
        a.pslots = 1;
        // counters, flags and accumulators start at zero (a fill kernel: the
        // last call's contents stay in the scratch)
        e = zero_words((uint32_t *)base, o_pages / 4, s);
        if (e == hipSuccess && n_spikes) e = launch_push(a, 0, 0, s);
    }
    if (e == hipSuccess) e = launch_tile(a, 0, 0, s);
    if (e != hipSuccess) return fail(SPK_EHIP, hipGetErrorString(e));
    return SPK_OK;
}

spk_status spk_export_rows(spk_net *net, const uint32_t *rows, uint64_t n_rows, uint64_t *offs,
                           uint32_t *col, float *w, int32_t *wq, uint8_t *delay, uint64_t cap)
{
    SPK_TRY(check_ready(net));
    if (!offs || (n_rows && !rows)) return fail(SPK_EINVAL, "null argument");
    for (uint64_t r = 0; r < n_rows; r++)
        if (rows[r] >= net->n) return fail(SPK_EINVAL, "row id out of range");
    SPK_TRY(sync_flags(net, nullptr));
    offs[0] = 0;
    if (!n_rows) return SPK_OK;
    hipStream_t s = net->stream;
    std::vector<uint32_t> deg(net->n);
    SPK_HIP(hipMemcpy(deg.data(), net->outdeg, (size_t)net->n * 4, hipMemcpyDeviceToHost));
    uint64_t tot = 0;
    for (uint64_t r = 0; r < n_rows; r++) {
        tot += deg[rows[r]];
        offs[r + 1] = tot;
    }
    if (tot > cap) return fail(SPK_EOVERFLOW, "export buffers too small");
    uint32_t *d_rows = nullptr, *d_col = nullptr, *d_wb = nullptr;
    uint64_t *d_off = nullptr;
    uint8_t *d_del = nullptr;
    SPK_TRY(dalloc(net, &d_rows, n_rows));
    SPK_TRY(dalloc(net, &d_off, n_rows));
    SPK_TRY(dalloc(net, &d_col, tot));
    SPK_TRY(dalloc(net, &d_wb, tot));
    SPK_TRY(dalloc(net, &d_del, tot));
    SPK_HIP(hipMemcpyAsync(d_rows, rows, n_rows * 4, hipMemcpyHostToDevice, s));
    SPK_HIP(hipMemcpyAsync(d_off, offs, n_rows * 8, hipMemcpyHostToDevice, s));
    if (net->proc)
        SPK_HIP(export_proc(step_args(net), net->ctab, d_rows, n_rows, d_off, d_col, d_wb, d_del, s));
    else
        SPK_HIP(export_gather(net->row_ptr, syn_ptr(net), net->compact, net->ctab, net->dmin, d_rows, n_rows,
                              d_off, d_col, d_wb, d_del, s));
    std::vector<uint32_t> hc(tot), hw(tot);
    std::vector<uint8_t> hd(tot);
    if (tot) {
        SPK_HIP(hipMemcpyAsync(hc.data(), d_col, tot * 4, hipMemcpyDeviceToHost, s));
        SPK_HIP(hipMemcpyAsync(hw.data(), d_wb, tot * 4, hipMemcpyDeviceToHost, s));
        SPK_HIP(hipMemcpyAsync(hd.data(), d_del, tot, hipMemcpyDeviceToHost, s));
    }
    SPK_HIP(hipStreamSynchronize(s));
    dfree(net, d_rows); dfree(net, d_off);
    dfree(net, d_col); dfree(net, d_wb); dfree(net, d_del);
    // canonical order per row: (target, delay, stored weight bits)
    std::vector<uint64_t> idx;
    for (uint64_t r = 0; r < n_rows; r++) {
        const uint64_t a = offs[r], b = offs[r + 1];
        idx.resize(b - a);
        for (uint64_t e = a; e < b; e++) idx[e - a] = e;
        std::sort(idx.begin(), idx.end(), [&](uint64_t x, uint64_t y) {
            if (hc[x] != hc[y]) return hc[x] < hc[y];
            if (hd[x] != hd[y]) return hd[x] < hd[y];
            return hw[x] < hw[y];
        });
        for (uint64_t e = a; e < b; e++) {
            const uint64_t src = idx[e - a];
            if (col) col[e] = hc[src];
            if (delay) delay[e] = hd[src];
            if (w) std::memcpy(&w[e], &hw[src], 4);
            if (wq) wq[e] = (int32_t)hw[src];
        }
    }
    return SPK_OK;
}

spk_status spk_poisson_table(spk_net *net, uint64_t *thr, uint32_t cap, uint32_t *len)
{
    SPK_TRY(check_ready(net));
    if (!len) return fail(SPK_EINVAL, "null len");
    *len = net->pois_len;
    if (net->pois_len > cap || (net->pois_len && !thr)) return fail(SPK_EOVERFLOW, "cap");
    for (uint32_t k = 0; k < net->pois_len; k++) thr[k] = net->pois[k];
    return SPK_OK;
}

spk_status spk_stats(spk_net *net, spk_stats_t *out)
{
    SPK_TRY(check_ready(net));
    if (!out) return fail(SPK_EINVAL, "null output");
    spk_stats_t st{};
    st.n = net->n;
    st.nnz = net->nnz;
    st.steps = net->t;
    st.device_bytes = net->device_bytes;
    st.n_exc = net->n_exc;
    st.ref_steps = net->ref_steps;
    st.ring_slots = net->spk_slots;
    st.delay_lists = net->lists;
    st.max_row = net->max_row;
    st.pois_len = net->pois_len;
    st.fixed_shift = net->P.acc_mode == SPK_ACC_FIXED ? net->P.fixed_shift : net->shift64;
    st.k = net->k;
    st.bytes_per_synapse = net->proc ? 0.0 : net->compact ? 4.0 : 8.0;
    st.tile_width = net->tl.W;
    st.tiles = net->tl.T;
    st.delivery = net->direct ? SPK_DELIVERY_DIRECT : SPK_DELIVERY_BINNED;
    st.page_cap = net->page_cap;
    st.step_mode = net->persistent ? SPK_STEP_PERSISTENT : SPK_STEP_GRAPH;
    st.batch_steps = net->persistent && !net->direct ? net->run_D : 1u;
    st.setup_ms = net->setup_ms;
    st.gen_ms = net->gen_ms;
    st.range_ms = net->range_ms;
    *out = st;
    return SPK_OK;
}

spk_status spk_set_profiling(spk_net *net, int on)
{
    SPK_TRY(check_ready(net));
    SPK_TRY(collect_profile(net));
    net->profiling = on != 0;
    net->ms_push = net->ms_tile = net->ms_run = 0;
    net->launches = net->run_launches = 0;
    return SPK_OK;
}

spk_status spk_read_kernel_ms(spk_net *net, double *push_ms, double *tile_ms, double *run_ms,
                              uint64_t *steps, uint64_t *run_launches)
{
    SPK_TRY(check_ready(net));
    SPK_TRY(collect_profile(net));
    if (push_ms) *push_ms = net->ms_push;
    if (tile_ms) *tile_ms = net->ms_tile;
    if (run_ms) *run_ms = net->ms_run;
    if (steps) *steps = net->launches;
    if (run_launches) *run_launches = net->run_launches;
    return SPK_OK;
}

spk_status spk_hbm_copy(spk_net *net, uint64_t bytes, int reps, double *ms)
{
    SPK_TRY(check_ready(net));
    if (bytes == 0 || bytes % 16 || reps < 1) return fail(SPK_EINVAL, "bytes multiple of 16, reps >= 1");
    hipStream_t s = net->stream;
    void *a = nullptr, *b = nullptr;
    SPK_TRY(dalloc(net, (uint8_t **)&a, bytes));
    SPK_TRY(dalloc(net, (uint8_t **)&b, bytes));
    hipEvent_t e0 = nullptr, e1 = nullptr;
    spk_status st = SPK_OK;
    do {
        hipError_t e = hipMemsetAsync(a, 1, bytes, s);
        if (e == hipSuccess) e = stream_copy(a, b, bytes, s);  // warm-up
        if (e == hipSuccess) e = hipEventCreate(&e0);
        if (e == hipSuccess) e = hipEventCreate(&e1);
        if (e == hipSuccess) e = hipEventRecord(e0, s);
        for (int r = 0; r < reps && e == hipSuccess; r++) e = stream_copy(a, b, bytes, s);
        if (e == hipSuccess) e = hipEventRecord(e1, s);
        if (e == hipSuccess) e = hipEventSynchronize(e1);
        float t = 0;
        if (e == hipSuccess) e = hipEventElapsedTime(&t, e0, e1);
        if (e != hipSuccess) { st = fail(SPK_EHIP, hipGetErrorString(e)); break; }
        if (ms) *ms = t;
    } while (0);
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    dfree(net, a);
    dfree(net, b);
    return st;
}

spk_status spk_hbm_read(spk_net *net, uint64_t bytes, int reps, double *ms)
{
    SPK_TRY(check_ready(net));
    if (bytes == 0 || bytes % 16 || reps < 1) return fail(SPK_EINVAL, "bytes multiple of 16, reps >= 1");
    hipStream_t s = net->stream;
    uint8_t *a = nullptr;
    uint32_t *sink = nullptr;
    SPK_TRY(dalloc(net, &a, bytes));
    SPK_TRY(dalloc(net, &sink, 1));
    hipEvent_t e0 = nullptr, e1 = nullptr;
    spk_status st = SPK_OK;
    do {
        hipError_t e = hipMemsetAsync(a, 1, bytes, s);
        if (e == hipSuccess) e = stream_read(a, bytes, sink, s);  // warm-up
        if (e == hipSuccess) e = hipEventCreate(&e0);
        if (e == hipSuccess) e = hipEventCreate(&e1);
        if (e == hipSuccess) e = hipEventRecord(e0, s);
        for (int r = 0; r < reps && e == hipSuccess; r++) e = stream_read(a, bytes, sink, s);
        if (e == hipSuccess) e = hipEventRecord(e1, s);
        if (e == hipSuccess) e = hipEventSynchronize(e1);
        float t = 0;
        if (e == hipSuccess) e = hipEventElapsedTime(&t, e0, e1);
        if (e != hipSuccess) { st = fail(SPK_EHIP, hipGetErrorString(e)); break; }
        if (ms) *ms = t;
    } while (0);
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    dfree(net, a);
    dfree(net, sink);
    return st;
}

void spk_destroy(spk_net *net) { destroy_net(net); }

}  // extern "C"
