// Host runtime behind the C ABI of include/snn.h: configuration checks,
// derived constants, the workspace plan over caller memory, launch
// sequencing of one step, graph-building phases and statistics.
#include "snn_internal.h"
#include "snn.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

using namespace snn;

// Scratch of snn_step_static: the list scans' status words, in device memory
// the library holds on every device it runs on, so that the call allocates
// nothing. In host code `scratch` is only a stand-in for the symbol; the
// kernels get the device address obtained once per device at snn_create.
constexpr int64_t kScratchWords = 131072;  // 1 MiB of 64-bit status words
static __device__ __align__(256) unsigned long long scratch[kScratchWords];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
unsigned long long *g_scratch[kMaxDevices] = {};  // device address of `scratch`, per device

// The device address of `scratch` on the current device `dev` (looked up on
// the first call for that device).
hipError_t static_scratch(int dev, unsigned long long **out)
{
    *out = nullptr;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void *ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) {
            (void)hipGetLastError();
            return e;
        }
        g_scratch[dev] = (unsigned long long *)ptr;
    }
    *out = g_scratch[dev];
    return hipSuccess;
}
}  // namespace

struct snn_ctx {
    snn_config cfg;
    hipStream_t stream = nullptr;
    int device = 0;
    std::string err;

    // derived configuration
    int32_t n = 0, nw = 0, nblk = 0, nacc = 1, n_slices = 0, chunks = 1, delay = 1;
    int32_t n_plastic_rows = 0, ref_steps = 0, dlv_blocks = 0;
    int32_t stdp_mult = 1, stdp_width = 0, stdp_groups = 0, stdp_chunks = 1, stdp_grid = 0;
    int32_t info_blocks = 1, syn_slots = 1;
    int32_t n_cu = 1;  // compute units of the device: one row-STDP workgroup each
    int32_t hw = 1;  // 64-bit history words per neuron
    int32_t algo = 0;  // plasticity_algorithm: 0 lazy + event, 1 lazy, 2 naive
    bool ct = false;  // compressed targets: 16-bit slice-local indices for slice delivery
    int32_t max_row = 0;  // longest row of the built graph
    float *sx_pre = nullptr, *sx_post = nullptr;  // per-synapse traces (naive)
    // kernel timing: events [step][part][start, stop] for the first t_cap
    // steps run by snn_step after snn_record_kernel_times; t_rec marks parts
    // that launched a kernel
    std::vector<hipEvent_t> tev;
    std::vector<uint8_t> t_rec;
    int32_t t_cap = 0, t_used = 0;
    ~snn_ctx()
    {
        for (hipEvent_t e : tev) (void)hipEventDestroy(e);
    }
    float k_m = 0, v_th = 0, v_reset = 0, v_inf = 0, d_e = 0, d_i = 0, j_ext = 0;
    float d_minus = 0, c_pot = 0, c_dep = 0, mu = 0;
    float dpow[kMaxAge + 1] = {};
    uint32_t fire_thr = 0;

    // workspace plan
    size_t ws_need = 0;
    uint8_t *ws = nullptr;
    float *v = nullptr, *ie = nullptr, *ii = nullptr, *ypost = nullptr, *xpre = nullptr;
    long long *apart = nullptr;  // fixed-point partial inputs [C][nacc][n]
    float *ain = nullptr;        // fp32 input [nacc][n] (teacher forcing / views)
    int32_t *ref = nullptr, *t_last = nullptr, *pend = nullptr;
    uint64_t *hist = nullptr, *mask = nullptr, *txmask = nullptr;
    uint8_t *code = nullptr;  // per-neuron history codes (k_neuron), n + 16 bytes
    uint64_t *recent = nullptr;
    StepClock *clk = nullptr;  // per-step scalars on the device (step index, input source)
    // list-scan status words: k_neuron uses the first neuron_grid(n); a delay
    // block's step k the row k of status_stride words
    unsigned long long *status = nullptr;
    int32_t status_stride = 0, status_words = 0;
    int32_t *spk_pos = nullptr;  // [D][n] spike-list positions (D > 1 with plasticity), else unused
    int32_t *ring = nullptr, *ring_cnt = nullptr;
    int32_t *rows = nullptr, *row_cnt = nullptr, *err_flag = nullptr, *maxlen = nullptr;
    int32_t *tx_cnt = nullptr;  // transmitted spikes of the step in progress (count)
    unsigned long long *static_status = nullptr;  // `scratch` on this context's device
    // forced rows partitioned by target range over the XCDs (StdpArgs::xcd):
    // the number of ranges (and the least the LDS reservation allows), the
    // ranges, their slice boundaries, the largest range's code table bytes,
    // and the forced rows' segment ends written by the neuron update
    // ([n_plastic_rows][8])
    bool xcd = false;
    int32_t xparts = 0, xparts_min = 0;
    int32_t xlo[kXcds + 1] = {}, xcd_piv[kXcds + 1] = {};
    int32_t xcd_table = 0;
    int32_t *segb = nullptr;
    int64_t *row_ptr = nullptr, *scratch = nullptr, *bsum = nullptr;
    int64_t *gstats = nullptr, *info_stats = nullptr, *syn_stats = nullptr, *dlv_stats = nullptr;
    RowInfo *info = nullptr, *txinfo = nullptr;
    int32_t dlv_slots = 0;
    // delay blocks (no plasticity, D >= 2): steps per block, partial inputs
    int32_t batch_max = 0;
    bool fuse = false;  // plastic: parts (2) and (3) of snn_step in one launch
    int32_t fuse_slots = 0;  // workgroups of the fused pass resident at once
    long long *abatch = nullptr;  // [batch_max][C][nacc][n]
    // plastic blocks (BlockArgs): most steps per block (0: off), targets per
    // group and groups; the group pivots (graph buffer), the plan's lists
    // and counts and the block clock (workspace)
    int32_t pb_max = 0, pb_width = 0, pb_groups = 0;
    int32_t *gpiv = nullptr;
    PbEvent *pev = nullptr;
    int32_t *pev_cnt = nullptr;
    uint8_t *pdcode = nullptr;
    uint64_t *phq = nullptr;
    BlockClock *bclk = nullptr;
    // source blocks (SourceArgs: Bernoulli sources, D = 1, plastic): most
    // steps per block (0: off) and the per-step versions of the arrays the
    // synapse pass reads, for the steps before a block's last
    int32_t sb_max = 0, sv_code_stride = 0;
    uint64_t *sv_hist = nullptr, *sv_recent = nullptr;
    float *sv_ypost = nullptr;
    uint8_t *sv_code = nullptr;
    int32_t *sv_tx = nullptr, *sv_rows = nullptr, *sv_cnt = nullptr;
    RowInfo *sv_txinfo = nullptr, *sv_info = nullptr;
    StepClock *sv_clk = nullptr;

    // graph
    uint8_t *g = nullptr;
    size_t g_bytes = 0;
    int64_t n_edges = -1, counted_edges = -1;
    int32_t *col = nullptr;
    uint16_t *col16 = nullptr;  // compressed targets (ct)
    float *w = nullptr;
    int32_t *piv = nullptr;
    int graph_state = 0;  // 0 none, 1 counted, 2 buffer bound, 3 built
    int32_t counted_kind = -1;
    double counted_p = 0.0;

    // time, as the host sees it: t is the step in progress or the next one
    // (the device clock counts neuron updates: t + 1 while a step is in
    // progress); a step is in progress when last_neuron_t == t
    int64_t t = 0, last_neuron_t = -1, last_deliver_t = -1;
};

// A captured sequence of steps (snn_graph_capture).
struct snn_graph {
    hipGraphExec_t exec = nullptr;
    int32_t steps = 0;
};

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

snn_status fail(snn_ctx *c, snn_status st, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    if (c) c->err = buf;
    return st;
}

snn_status check_hip(snn_ctx *c, hipError_t e, const char *what)
{
    if (e == hipSuccess) return SNN_OK;
    return fail(c, SNN_EDEVICE, "%s: %s", what, hipGetErrorString(e));
}

bool finite_all(std::initializer_list<double> xs)
{
    for (double x : xs)
        if (!std::isfinite(x)) return false;
    return true;
}

snn_status validate(snn_ctx *c, const snn_config &k)
{
    if (k.n < 1 || k.n >= (1 << 24)) return fail(c, SNN_EINVAL, "n must be in [1, 2^24)");
    if (k.n_exc < 0 || k.n_exc > k.n) return fail(c, SNN_EINVAL, "n_exc must be in [0, n]");
    if (k.delay_steps < 1 || k.delay_steps > SNN_MAX_DELAY)
        return fail(c, SNN_EINVAL, "delay_steps must be in [1, 64]");
    if (k.neuron_model < 0 || k.neuron_model > 2)
        return fail(c, SNN_EINVAL, "unknown neuron_model %d", k.neuron_model);
    if (k.plastic < 0 || k.plastic > 2) return fail(c, SNN_EINVAL, "unknown plastic %d", k.plastic);
    const int nacc = k.neuron_model == SNN_LIF_CUBA ? 2 : 1;
    if (k.slice_width < kWave || k.slice_width % kWave != 0)
        return fail(c, SNN_EINVAL, "slice_width must be a positive multiple of 64");
    if ((int64_t)k.slice_width * 8 * nacc > kLdsBytes)
        return fail(c, SNN_EINVAL, "slice_width * 8 B * %d accumulators exceeds 160 KiB of LDS",
                    nacc);
    if (k.spike_chunks < 1 || k.spike_chunks > 64)
        return fail(c, SNN_EINVAL, "spike_chunks must be in [1, 64]");
    if (k.stdp_slice_mult < 0 || k.stdp_slice_mult > 4096)
        return fail(c, SNN_EINVAL, "stdp_slice_mult must be in [0, 4096]");
    if (k.stdp_chunks < 0 || k.stdp_chunks > 1024)
        return fail(c, SNN_EINVAL, "stdp_chunks must be in [0, 1024]");
    if (k.stdp_layout < 0 || k.stdp_layout > 1)
        return fail(c, SNN_EINVAL, "stdp_layout must be 0 or 1");
    if (k.history_bits != 0 && k.history_bits != 64 && k.history_bits != 128)
        return fail(c, SNN_EINVAL, "history_bits must be 64 or 128 (0: 64)");
    if (k.plasticity_algorithm < 0 || k.plasticity_algorithm > 2)
        return fail(c, SNN_EINVAL, "plasticity_algorithm must be 0, 1 or 2");
    if (k.stdp_filter < 0 || k.stdp_filter > 3)
        return fail(c, SNN_EINVAL, "stdp_filter must be in [0, 3]");
    if (k.compressed_targets < 0 || k.compressed_targets > 1)
        return fail(c, SNN_EINVAL, "compressed_targets must be 0 or 1");
    if (k.stdp_xcd != 0 && k.stdp_xcd != 1 && k.stdp_xcd != 2 && k.stdp_xcd != 4 &&
        k.stdp_xcd != 8)
        return fail(c, SNN_EINVAL, "stdp_xcd must be 0, 1, 2, 4 or 8");
    if (k.plastic_blocks < -1 || k.plastic_blocks > SNN_MAX_DELAY)
        return fail(c, SNN_EINVAL, "plastic_blocks must be in [-1, 64]");
    if (k.plastic_block_width != 0 &&
        ((k.plastic_block_width != 64 && k.plastic_block_width != 128 &&
          k.plastic_block_width != 256) ||
         k.slice_width % k.plastic_block_width != 0))
        return fail(c, SNN_EINVAL,
                    "plastic_block_width must be 0, or 64, 128 or 256 dividing slice_width");
    if (k.stdp_filter == 1 && (int64_t)k.n + 16 > kCodeMax)
        return fail(c, SNN_EINVAL, "stdp_filter 1 needs n + 16 <= %d", kCodeMax);
    if (k.stdp_filter == 2 && (k.n + 63) / 64 > kRecentMaxWords)
        return fail(c, SNN_EINVAL, "stdp_filter 2 needs n <= %d", kRecentMaxWords * 64);
    const int64_t slices = (k.n + k.slice_width - 1) / k.slice_width;
    if (slices * k.spike_chunks > (1 << 20))
        return fail(c, SNN_EINVAL, "slices * spike_chunks must not exceed 2^20");
    if (k.poisson_len < 0 || k.poisson_len > SNN_MAX_POISSON)
        return fail(c, SNN_EINVAL, "poisson_len must be in [0, 32]");
    for (int q = 1; q < k.poisson_len; ++q)
        if (k.poisson_cdf[q] < k.poisson_cdf[q - 1])
            return fail(c, SNN_EINVAL, "poisson_cdf must be non-decreasing");
    if (!finite_all({k.dt_ms, k.tau_m_ms, k.v_th, k.v_reset, k.v_inf, k.tau_ref_ms, k.tau_e_ms,
                     k.tau_i_ms, k.j_ext, k.p_fire, k.tau_plus_ms, k.tau_minus_ms, k.lambda,
                     k.alpha, k.mu, k.w0}))
        return fail(c, SNN_EINVAL, "configuration contains a NaN or infinity");
    if (!(k.dt_ms > 0)) return fail(c, SNN_EINVAL, "dt_ms must be > 0");
    if (k.neuron_model != SNN_BERNOULLI_SOURCE) {
        if (!(k.tau_m_ms > 0)) return fail(c, SNN_EINVAL, "tau_m_ms must be > 0");
        if (!(k.tau_ref_ms >= 0)) return fail(c, SNN_EINVAL, "tau_ref_ms must be >= 0");
    } else if (!(k.p_fire >= 0 && k.p_fire <= 1)) {
        return fail(c, SNN_EINVAL, "p_fire must be in [0, 1]");
    }
    if (k.neuron_model == SNN_LIF_CUBA && !(k.tau_e_ms > 0 && k.tau_i_ms > 0))
        return fail(c, SNN_EINVAL, "tau_e_ms and tau_i_ms must be > 0");
    if (k.plastic != SNN_PLASTIC_NONE) {
        if (!(k.tau_plus_ms > 0 && k.tau_minus_ms > 0))
            return fail(c, SNN_EINVAL, "STDP time constants must be > 0");
        if (!(k.mu >= 0 && k.mu < 1)) return fail(c, SNN_EINVAL, "mu must be in [0, 1)");
        if (!(k.w0 > 0)) return fail(c, SNN_EINVAL, "w0 must be > 0");
        if (!(k.lambda >= 0 && k.alpha >= 0))
            return fail(c, SNN_EINVAL, "lambda and alpha must be >= 0");
    }
    return SNN_OK;
}

// The plastic targets' slices (all targets, or the excitatory ones).
int32_t xcd_plastic_slices(const snn_ctx *c)
{
    const int32_t limit = c->cfg.plastic == SNN_PLASTIC_EXC_EXC ? c->cfg.n_exc : c->n;
    return (limit + c->cfg.slice_width - 1) / c->cfg.slice_width;
}

// Cuts the plastic targets' slices into `parts` ranges (entries past the
// last range repeat its end) and sizes the largest range's code table.
void set_xcd_ranges(snn_ctx *c, int parts)
{
    const int32_t sp = xcd_plastic_slices(c);
    int32_t span = 0;
    for (int x = 0; x <= kXcds; ++x) {
        const int xx = std::min(x, parts);
        c->xcd_piv[x] = (int32_t)((int64_t)xx * sp / parts);
        c->xlo[x] = (int32_t)std::min<int64_t>((int64_t)c->xcd_piv[x] * c->cfg.slice_width, c->n);
        if (x > 0) span = std::max(span, c->xlo[x] - c->xlo[x - 1]);
    }
    c->xparts = parts;
    c->xcd_table = (span + 15) / 16 * 16;
}

// The automatic range count, once the edge count is known: the most ranges
// (of 2, 4, 8, at least the count the LDS reservation was made for) whose
// segments still hold about three quarters of a part, taking a forced row's
// plastic entries as its share of the edges spread evenly over the targets.
void choose_xcd_ranges(snn_ctx *c)
{
    if (!c->xcd || c->cfg.stdp_xcd != 1) return;
    const int32_t sp = xcd_plastic_slices(c);
    const int64_t limit = std::min<int64_t>((int64_t)sp * c->cfg.slice_width, c->n);
    const double seg = (double)c->n_edges / c->n * (double)limit / c->n;
    const int part = kStdpXcdUnroll * kWave;
    int parts = c->xparts_min;
    for (int p = kXcds; p > c->xparts_min; p /= 2)
        if (p <= sp && seg / p >= 0.75 * part) {
            parts = p;
            break;
        }
    set_xcd_ranges(c, parts);
}

// Constants derived here on the host from the physical parameters (double,
// rounded once to fp32).
void derive(snn_ctx *c)
{
    const snn_config &k = c->cfg;
    c->n = k.n;
    c->nw = (k.n + 63) / 64;
    c->nblk = (k.n + kBlock - 1) / kBlock;
    c->nacc = k.neuron_model == SNN_LIF_CUBA ? 2 : 1;
    c->hw = k.history_bits == 128 ? 2 : 1;
    c->algo = k.plasticity_algorithm;
    c->ct = k.compressed_targets != 0;
    c->n_slices = (k.n + k.slice_width - 1) / k.slice_width;
    c->chunks = k.spike_chunks;
    c->delay = k.delay_steps;
    c->n_plastic_rows = k.plastic == SNN_PLASTIC_ALL ? k.n
                      : k.plastic == SNN_PLASTIC_EXC_EXC ? k.n_exc : 0;
    c->k_m = k.neuron_model == SNN_BERNOULLI_SOURCE ? 0.f : (float)(k.dt_ms / k.tau_m_ms);
    c->v_th = (float)k.v_th;
    c->v_reset = (float)k.v_reset;
    c->v_inf = (float)k.v_inf;
    c->d_e = k.neuron_model == SNN_LIF_CUBA ? (float)std::exp(-k.dt_ms / k.tau_e_ms) : 0.f;
    c->d_i = k.neuron_model == SNN_LIF_CUBA ? (float)std::exp(-k.dt_ms / k.tau_i_ms) : 0.f;
    c->j_ext = (float)k.j_ext;
    c->ref_steps = k.neuron_model == SNN_BERNOULLI_SOURCE
                       ? 0 : (int32_t)std::lround(k.tau_ref_ms / k.dt_ms);
    const double thr = std::floor(k.p_fire * 4294967296.0);
    c->fire_thr = thr <= 0 ? 0u : thr >= 4294967295.0 ? 0xFFFFFFFFu : (uint32_t)thr;
    if (k.plastic != SNN_PLASTIC_NONE) {
        const double dp = std::exp(-k.dt_ms / k.tau_plus_ms);
        static_assert(sizeof(c->dpow) == sizeof(float) * (kMaxAge + 1), "decay table size");
        for (int q = 0; q <= kMaxAge; ++q) c->dpow[q] = (float)std::pow(dp, (double)q);
        c->d_minus = (float)std::exp(-k.dt_ms / k.tau_minus_ms);
        c->c_pot = (float)(k.lambda * std::pow(k.w0, 1.0 - k.mu));
        c->c_dep = (float)(k.lambda * k.alpha);
        c->mu = (float)k.mu;
    }
    const int64_t work = (int64_t)c->n_slices * c->chunks;
    c->dlv_blocks = (int32_t)((work + 7) / 8 * 8);
    c->dlv_slots = c->dlv_blocks > kGlobalMaxBlocks ? c->dlv_blocks : kGlobalMaxBlocks;
    // Delay blocks of up to D-1 steps, their inputs within kBatchBytes of
    // workspace (none for plastic networks or D = 1). A block's delivery
    // item is (step, slice) with one chunk: the steps give the parallelism.
    c->batch_max = 0;
    if (k.plastic == SNN_PLASTIC_NONE && c->delay >= 2) {
        const int64_t per_step = (int64_t)c->nacc * c->n * (int64_t)sizeof(long long);
        int64_t bm = std::min<int64_t>(c->delay - 1, batch_steps_max(k.neuron_model));
        bm = std::min<int64_t>(bm, kBatchBytes / per_step);
        if (bm * c->n_slices > (1 << 24)) bm = 0;
        c->batch_max = (int32_t)std::max<int64_t>(bm, 0);
        const int64_t bb = (c->batch_max * c->n_slices + 7) / 8 * 8;
        if (bb > c->dlv_slots) c->dlv_slots = (int32_t)bb;
    }
    c->info_blocks = c->nblk;  // statistics slots of the neuron-kernel / flush snapshots
    // Plastic blocks (BlockArgs) of up to D-1 steps (at most kPbMaxSteps): lazy
    // plasticity, D >= 2, up to kPbMaxN neurons. Target groups of 64, 128
    // or 256 neurons inside slices, one workgroup each: the narrowest that
    // needs no more workgroups than the device has CUs, else the widest.
    c->pb_max = c->pb_width = c->pb_groups = 0;
    if (c->n_plastic_rows > 0 && c->algo != 2 && c->delay >= 2 && k.n <= kPbMaxN &&
        k.plastic_blocks >= 0) {
        int32_t bm = std::min<int32_t>(c->delay - 1, kPbMaxSteps);
        if (k.plastic_blocks > 0) bm = std::min<int32_t>(bm, k.plastic_blocks);
        int32_t gw = k.plastic_block_width;
        if (gw == 0) {
            for (int cand : {64, 128, 256}) {
                if (k.slice_width % cand != 0) continue;
                gw = cand;
                if (((int64_t)k.n + cand - 1) / cand <= (int64_t)c->n_cu) break;
            }
        }
        c->pb_max = bm;
        c->pb_width = gw;
        c->pb_groups = (k.n + gw - 1) / gw;
    }
}

// Workspace plan: a bump allocator over the caller's buffer.
struct Plan {
    size_t off = 0;
    uint8_t *base = nullptr;
    template <typename T> T *take(int64_t count)
    {
        T *p = base ? (T *)(base + off) : nullptr;
        off = align_up(off + (size_t)count * sizeof(T));
        return p;
    }
};

void plan_workspace(snn_ctx *c, uint8_t *base)
{
    Plan p;
    p.base = base;
    const int64_t n = c->n;
    c->v = p.take<float>(n);
    c->ref = p.take<int32_t>(n);
    c->ie = p.take<float>(n);
    c->ii = p.take<float>(n);
    c->hist = p.take<uint64_t>(n * c->hw);
    c->ypost = p.take<float>(n);
    c->t_last = p.take<int32_t>(n);
    c->xpre = p.take<float>(n);
    c->apart = p.take<long long>((int64_t)c->chunks * c->nacc * n);
    c->ain = p.take<float>((int64_t)c->nacc * n);
    c->mask = p.take<uint64_t>(c->nw);
    c->txmask = p.take<uint64_t>(c->nw);
    c->code = p.take<uint8_t>((int64_t)c->n + 16);
    c->recent = p.take<uint64_t>(c->nw);
    c->clk = p.take<StepClock>(1);
    c->status_stride = neuron_steps_grid(c->n);
    c->status_words = std::max<int32_t>(neuron_grid(c->n), kBatchMax * c->status_stride);
    c->status = p.take<unsigned long long>(c->status_words);
    c->spk_pos = p.take<int32_t>(c->delay > 1 ? (int64_t)c->delay * n : 1);
    c->ring = p.take<int32_t>((int64_t)c->delay * n);
    c->ring_cnt = p.take<int32_t>(c->delay);
    c->rows = p.take<int32_t>(n);
    c->row_cnt = p.take<int32_t>(1);
    c->tx_cnt = p.take<int32_t>(1);
    c->segb = p.take<int32_t>(c->xcd ? (int64_t)c->n_plastic_rows * kXcds : 1);
    c->err_flag = p.take<int32_t>(1);
    c->maxlen = p.take<int32_t>(1);
    c->row_ptr = p.take<int64_t>(n + 1);
    c->pend = p.take<int32_t>(n);
    c->scratch = p.take<int64_t>(n + 1);
    c->bsum = p.take<int64_t>((n + 1 + 1023) / 1024 + 1);
    c->gstats = p.take<int64_t>(kGFields);
    c->info = p.take<RowInfo>(c->n_plastic_rows > 0 ? c->n_plastic_rows : 1);
    c->txinfo = p.take<RowInfo>(n);  // transmitted rows: start, and plasticity snapshot
    c->info_stats = p.take<int64_t>((int64_t)c->info_blocks * kStFields);
    c->syn_stats = p.take<int64_t>(c->syn_slots);
    c->dlv_stats = p.take<int64_t>(2 * (int64_t)c->dlv_slots);
    c->abatch = p.take<long long>(c->batch_max > 0 ? (int64_t)c->batch_max * c->nacc * n : 1);
    c->pev = p.take<PbEvent>(c->pb_max > 0 ? (int64_t)(c->pb_max + 1) * n : 1);
    c->pev_cnt = p.take<int32_t>(2 * kBatchMax);  // consecutive blocks alternate halves
    c->pdcode = p.take<uint8_t>(c->pb_max > 0 ? (n + 15) / 16 * 16 : 1);
    c->phq = p.take<uint64_t>(c->pb_max > 0 ? 2 * n * c->hw : 1);
    c->bclk = p.take<BlockClock>(1);
    {
        const int64_t v = c->sb_max > 1 ? c->sb_max - 1 : 0;  // versions
        const int64_t npl = std::max<int32_t>(c->n_plastic_rows, 1);
        c->sv_code_stride = (int32_t)((n + 16 + 15) / 16 * 16);
        c->sv_hist = p.take<uint64_t>(v ? v * n * c->hw : 1);
        c->sv_ypost = p.take<float>(v ? v * n : 1);
        c->sv_code = p.take<uint8_t>(v ? v * c->sv_code_stride : 1);
        c->sv_recent = p.take<uint64_t>(v ? v * c->nw : 1);
        c->sv_tx = p.take<int32_t>(v ? v * n : 1);
        c->sv_txinfo = p.take<RowInfo>(v ? v * n : 1);
        c->sv_rows = p.take<int32_t>(v ? v * npl : 1);
        c->sv_info = p.take<RowInfo>(v ? v * npl : 1);
        c->sv_cnt = p.take<int32_t>(v ? 2 * v : 1);
        c->sv_clk = p.take<StepClock>(v ? v : 1);
    }
    c->ws_need = p.off;
}

snn_status require_ws(snn_ctx *c)
{
    if (!c->ws) return fail(c, SNN_ESTATE, "no workspace bound");
    return SNN_OK;
}

snn_status require_graph(snn_ctx *c)
{
    if (!c->ws) return fail(c, SNN_ESTATE, "no workspace bound");
    if (c->graph_state != 3) return fail(c, SNN_ESTATE, "graph not built");
    return SNN_OK;
}

GraphArgs graph_args(snn_ctx *c)
{
    GraphArgs a{};
    a.row_ptr = c->row_ptr;
    a.col = c->col;
    a.w = c->w;
    a.piv = c->piv;
    a.pend = c->pend;
    a.err = c->err_flag;
    a.maxlen = c->maxlen;
    a.seed = c->cfg.seed;
    a.n = c->n;
    a.n_exc = c->cfg.n_exc;
    a.width = c->cfg.slice_width;
    a.n_slices = c->n_slices;
    a.plastic = c->cfg.plastic;
    a.col16 = c->col16;
    return a;
}

int ring_slot(const snn_ctx *c, int64_t step)
{
    const int64_t d = c->delay;
    return (int)(((step % d) + d) % d);
}

snn_status zero_stats(snn_ctx *c)
{
    hipError_t e = launch_fill_i64(c->stream, c->gstats, kGFields, 0);
    if (e == hipSuccess)
        e = launch_fill_i64(c->stream, c->info_stats, (int64_t)c->info_blocks * kStFields, 0);
    if (e == hipSuccess) e = launch_fill_i64(c->stream, c->syn_stats, c->syn_slots, 0);
    if (e == hipSuccess) e = launch_fill_i64(c->stream, c->dlv_stats, 2 * (int64_t)c->dlv_slots, 0);
    return check_hip(c, e, "reset statistics");
}

// Finish a graph build: pivots, plastic prefixes, error check, group size.
snn_status finish_graph(snn_ctx *c)
{
    GraphArgs a = graph_args(c);
    snn_status st = check_hip(c, launch_pivots(c->stream, a), "pivot kernel");
    if (st) return st;
    if (c->pb_max > 0) {  // pivots at the target groups of the plastic blocks
        GraphArgs ga = a;
        ga.piv = c->gpiv;
        ga.width = c->pb_width;
        ga.n_slices = c->pb_groups;
        st = check_hip(c, launch_pivots(c->stream, ga), "group pivot kernel");
        if (st) return st;
    }
    if (c->ct) {
        st = check_hip(c, launch_encode_targets(c->stream, a, c->n_edges), "target compression");
        if (st) return st;
    }
    if (c->algo == 2) {  // per-synapse traces start at 0
        st = check_hip(c, launch_fill_f32(c->stream, c->sx_pre, c->n_edges, 0.f), "traces");
        if (!st) st = check_hip(c, launch_fill_f32(c->stream, c->sx_post, c->n_edges, 0.f),
                                "traces");
        if (st) return st;
    }
    st = check_hip(c, launch_fill_i32(c->stream, c->maxlen, 1, 0), "row length");
    if (!st) st = check_hip(c, launch_row_maxlen(c->stream, a), "row length");
    if (st) return st;
    int32_t err = 0, maxlen = 0;
    st = check_hip(c, hipMemcpyAsync(&err, c->err_flag, sizeof err, hipMemcpyDeviceToHost,
                                     c->stream), "read error flag");
    if (!st)
        st = check_hip(c, hipMemcpyAsync(&maxlen, c->maxlen, sizeof maxlen,
                                         hipMemcpyDeviceToHost, c->stream), "read row length");
    if (st) return st;
    st = check_hip(c, hipStreamSynchronize(c->stream), "graph build");
    if (st) return st;
    if (err & kErrIndex) return fail(c, SNN_EINVAL, "edge index outside [0, n)");
    if (err & kErrRowTooLong)
        return fail(c, SNN_EINVAL, "a row has more than %d edges", kMaxSortRow);
    c->max_row = maxlen;
    c->graph_state = 3;
    return SNN_OK;
}

// Turns pending fixed-point partial inputs into the fp32 input the next
// neuron update would compute, so it can be viewed or overwritten (the
// device clock says which the next update reads; afterwards the fp32 one).
snn_status materialize_input(snn_ctx *c)
{
    return check_hip(c, launch_materialize_input(c->stream, c->apart, (int64_t)c->nacc * c->n,
                                                 c->clk, c->ain, (int64_t)c->nacc * c->n),
                     "materialise input");
}

// Status words cleared (no stale step tag can match a later scan).
hipError_t clear_status(snn_ctx *c)
{
    return launch_fill_i64(c->stream, (int64_t *)c->status, c->status_words, 0);
}

// The device clock read back (synchronises the stream); the host's view of
// t follows it (a replayed capture advances the device only).
snn_status sync_clock(snn_ctx *c, int64_t *dev_t)
{
    StepClock ck{};
    snn_status st = check_hip(c, hipMemcpyAsync(&ck, c->clk, sizeof ck, hipMemcpyDeviceToHost,
                                                c->stream), "read the step clock");
    if (!st) st = check_hip(c, hipStreamSynchronize(c->stream), "read the step clock");
    if (st) return st;
    const bool in_step = c->last_neuron_t == c->t;
    c->t = in_step ? ck.t - 1 : ck.t;
    c->last_neuron_t = ck.t - 1;
    if (!in_step) c->last_deliver_t = ck.t - 1;
    *dev_t = ck.t;
    return SNN_OK;
}

// Events of part `part` (0 neurons and lists, 1 plasticity, 2 delivery)
// of the current step when timing is on; marks the part as timed.
KernelEvents part_events(snn_ctx *c, int part)
{
    KernelEvents ev;
    if (c->t_used < c->t_cap) {
        const size_t q = (size_t)c->t_used * kTimedParts + part;
        ev.start = c->tev[2 * q];
        ev.stop = c->tev[2 * q + 1];
        c->t_rec[q] = 1;
    }
    return ev;
}

NeuronArgs neuron_args(snn_ctx *c)
{
    NeuronArgs a{};
    a.v = c->v;
    a.ref = c->ref;
    a.ie = c->ie;
    a.ii = c->ii;
    a.hist = c->hist;
    a.hw = c->hw;
    a.ypost = c->ypost;
    a.t_last = c->t_last;
    a.apart = c->apart;
    a.ain = c->ain;
    a.part_stride = (int64_t)c->nacc * c->n;
    a.max_parts = c->chunks;
    a.clk = c->clk;
    a.mask = c->mask;
    a.txmask = c->txmask;
    a.code = c->code;
    a.recent = c->recent;
    a.n = c->n;
    a.n_exc = c->cfg.n_exc;
    a.model = c->cfg.neuron_model;
    a.n_plastic_rows = c->algo == 2 ? 0 : c->n_plastic_rows;  // naive: no lazy rows
    a.dm1 = c->delay - 1;
    a.ref_steps = c->ref_steps;
    a.poisson_len = c->cfg.neuron_model == SNN_LIF_DELTA ? c->cfg.poisson_len : 0;
    a.k_m = c->k_m;
    a.v_th = c->v_th;
    a.v_reset = c->v_reset;
    a.v_inf = c->v_inf;
    a.d_e = c->d_e;
    a.d_i = c->d_i;
    a.j_ext = c->j_ext;
    a.d_minus = c->d_minus;
    a.fire_thr = c->fire_thr;
    a.seed = c->cfg.seed;
    for (int q = 0; q < kMaxPoisson; ++q) a.poisson[q] = c->cfg.poisson_cdf[q];
    return a;
}

// parity: the block's place in the call (consecutive blocks use the two
// halves of the list counts in turn)
BlockArgs block_args(snn_ctx *c, int32_t steps, int32_t parity)
{
    BlockArgs b{};
    b.row_ptr = c->row_ptr;
    b.pend = c->pend;
    b.hist = c->hist;
    b.t_last = c->t_last;
    b.xpre = c->xpre;
    b.status = c->status;
    b.status_stride = c->status_stride;
    b.status_words = c->status_words;
    b.ev = c->pev;
    b.ev_cnt = c->pev_cnt + (parity & 1) * kBatchMax;
    b.ev_cnt_next = c->pev_cnt + (~parity & 1) * kBatchMax;
    b.dcode = c->pdcode;
    b.hq = c->phq;
    b.n_cu = c->n_cu;
    b.df_parts = (int32_t)std::max<int64_t>(1, ((int64_t)c->max_row + 7 + kPbDfPart - 1) /
                                                   kPbDfPart);
    b.bclk = c->bclk;
    b.clk = c->clk;
    b.info_stats = c->info_stats;
    b.info_slots = c->info_blocks;
    b.err = c->err_flag;
    b.steps = steps;
    b.n = c->n;
    b.n_exc = c->cfg.n_exc;
    b.n_plastic_rows = c->n_plastic_rows;
    b.hw = c->hw;
    b.delay = c->delay;
    b.nacc = c->nacc;
    b.col = c->col;
    b.col16 = c->ct ? c->col16 : nullptr;
    b.w = c->w;
    b.gpiv = c->gpiv;
    b.n_edges = c->n_edges;
    b.gwidth = c->pb_width;
    b.width = c->cfg.slice_width;
    b.n_groups = c->pb_groups;
    b.apart = c->apart;
    b.part_stride = (int64_t)c->nacc * c->n;
    b.dlv_stats = c->dlv_stats;
    b.dlv_slots = c->dlv_slots;
    b.syn_stats = c->syn_stats;
    b.syn_slots = c->syn_slots;
    b.gstats = c->gstats;
    b.event = c->algo == 0 ? 1 : 0;
    b.c_pot = c->c_pot;
    b.c_dep = c->c_dep;
    b.mu = c->mu;
    b.ring = c->ring;
    b.ring_cnt = c->ring_cnt;
    b.spk_pos = c->spk_pos;
    b.rows = c->rows;
    b.row_cnt = c->row_cnt;
    b.mask = c->mask;
    b.txmask = c->txmask;
    b.recent = c->recent;
    for (int q = 0; q <= kMaxAge; ++q) b.dpow[q] = c->dpow[q];
    return b;
}

CompactArgs compact_args(snn_ctx *c)
{
    CompactArgs b{};
    b.ring = c->ring;
    b.ring_cnt = c->ring_cnt;
    b.tx_cnt = c->tx_cnt;
    b.row_list = c->rows;
    b.row_cnt = c->row_cnt;
    b.status = c->status;
    b.spk_pos = c->spk_pos;
    b.delay = c->delay;
    b.gstats = c->gstats;
    b.n = c->n;
    b.nw = c->nw;
    b.n_plastic_rows = c->algo == 2 ? 0 : c->n_plastic_rows;
    b.info = c->info;
    b.txinfo = c->txinfo;
    b.row_ptr = c->row_ptr;
    b.pend = c->pend;
    b.hist = c->hist;
    b.hw = c->hw;
    b.t_last = c->t_last;
    b.xpre = c->xpre;
    b.err = c->err_flag;
    b.info_stats = c->n_plastic_rows > 0 && c->algo != 2 ? c->info_stats : nullptr;
    b.segb = c->xcd ? c->segb : nullptr;
    b.piv = c->piv;
    b.piv_stride = c->n_slices + 1;
    b.xparts = c->xparts;
    for (int x = 0; x <= kXcds; ++x) b.xcd_piv[x] = c->xcd_piv[x];
    for (int q = 0; q <= kMaxAge; ++q) b.dpow[q] = c->dpow[q];
    return b;
}

snn_status launch_step_neurons(snn_ctx *c)
{
    NeuronArgs a = neuron_args(c);
    CompactArgs b = compact_args(c);
    snn_status st =
        check_hip(c, launch_neuron(c->stream, a, b, part_events(c, 0)), "neuron kernel");
    if (st) return st;
    c->last_neuron_t = c->t;
    return SNN_OK;
}

size_t dlv_lds_bytes(const snn_ctx *c)
{
    size_t b = sizeof(DlvShared) + (size_t)c->cfg.slice_width * c->nacc * sizeof(long long);
    if (c->n_plastic_rows > 0 && c->algo != 2)
        b += (size_t)c->cfg.slice_width * (c->hw * sizeof(uint64_t) + sizeof(float));
    return b;
}

// Arguments of the synapse pass over the forced rows (flush: all rows).
StdpArgs stdp_args(snn_ctx *c, bool flush, int64_t waves = 0)
{
    if (waves <= 0) waves = (int64_t)c->n_cu * (kStdpRowsBlock / kWave);
    StdpArgs a{};
    a.info = c->info;
    a.row_cnt = flush ? nullptr : c->row_cnt;
    a.n_rows_all = c->n_plastic_rows;
    a.n_info = std::max<int32_t>(c->n_plastic_rows, 1);
    a.t_last = c->t_last;
    a.xpre = c->xpre;
    a.clk = c->clk;
    a.tx_cnt = c->tx_cnt;
    a.col = c->col;
    a.w = c->w;
    a.piv = c->piv;
    a.hist = c->hist;
    a.hw = c->hw;
    a.ypost = c->ypost;
    a.n = c->n;
    a.n_slices = c->n_slices;
    a.mult = c->stdp_mult;
    a.width = c->stdp_width;
    a.n_groups = c->stdp_groups;
    a.chunks = c->stdp_chunks;
    a.n_work = c->stdp_groups * c->stdp_chunks;
    a.target_limit = c->cfg.plastic == SNN_PLASTIC_EXC_EXC ? c->cfg.n_exc : c->n;
    a.c_pot = c->c_pot;
    a.c_dep = c->c_dep;
    a.mu = c->mu;
    a.stats = c->syn_stats;
    // codes and bitmap are rebuilt by every neuron update (not by set_state)
    const bool fresh = c->last_neuron_t >= 0;
    const int f = c->cfg.stdp_filter;
    const bool fits_code = (int64_t)c->n + 16 <= kCodeMax, fits_map = c->nw <= kRecentMaxWords;
    // lazy but not event-driven: every synapse of a row walks every step
    const bool filt = fresh && c->algo == 0;
    a.code = filt && (f == 1 || (f == 0 && fits_code)) ? c->code : nullptr;
    a.recent = filt && (f == 2 || (f == 0 && !fits_code && fits_map)) ? c->recent : nullptr;
    a.event = c->algo == 0;
    // forced rows over the XCDs: each range's codes (none when not event-driven)
    a.xcd = c->xcd && !flush;
    a.xparts = c->xparts;
    a.segb = c->segb;
    for (int x = 0; x <= kXcds; ++x) a.xlo[x] = c->xlo[x];
    if (a.xcd) {
        a.code = filt ? c->code : nullptr;
        a.recent = nullptr;
    }
    a.nw = c->nw;
    // row-wise layout: a row's parts (counting the row start's offset in its
    // line) may spread over P waves. P minimises the parts one wave takes in
    // sequence, ceil(rows P / waves) ceil(parts / P), for the expected number
    // of rows: all plastic rows in a flush, else the forced rows (staggered:
    // one in 64 hw per step); ties keep the smaller P (fewer snapshot loads).
    const int part = (c->hw == 2 ? kStdpRowsUnroll2 : kStdpRowsUnroll) * kWave;
    const int64_t parts = std::max(1, (c->max_row + kStoreLine - 1 + part - 1) / part);
    const int64_t rows = std::max<int64_t>(1, flush ? c->n_plastic_rows
                                                    : c->n_plastic_rows / (64 * c->hw));
    int64_t best = -1;
    a.parts = 1;
    for (int pp = 1; pp <= kStdpRowsSplit && pp <= parts; ++pp) {
        const int64_t chain = ((rows * pp + waves - 1) / waves) * ((parts + pp - 1) / pp);
        if (best < 0 || chain < best) {
            best = chain;
            a.parts = pp;
        }
    }
    for (int q = 0; q <= kMaxAge; ++q) a.dpow[q] = c->dpow[q];
    return a;
}

// The plasticity part for rows forced by the 64-step history window (their
// snapshots were taken by the neuron kernel); rows transmitting at t are
// brought up to date by the delivery part. A flush (every plastic row up to
// step t-1, no pre-synaptic spike) takes its snapshots first. The synapse
// pass commits t_last and the pre traces.
snn_status launch_plasticity(snn_ctx *c, bool flush, hipStream_t s, KernelEvents ev = {})
{
    if (flush) {
        RowInfoArgs r{};
        r.rows = nullptr;
        r.row_cnt = nullptr;
        r.n_rows_all = c->n_plastic_rows;
        r.dm1 = c->delay - 1;
        r.clk = c->clk;
        r.row_ptr = c->row_ptr;
        r.pend = c->pend;
        r.hist = c->hist;
        r.hw = c->hw;
        r.t_last = c->t_last;
        r.xpre = c->xpre;
        r.info = c->info;
        r.err = c->err_flag;
        r.stats = c->info_stats;
        for (int q = 0; q <= kMaxAge; ++q) r.dpow[q] = c->dpow[q];
        snn_status st = check_hip(c, launch_row_info(s, r, c->n_plastic_rows),
                                  "STDP row snapshot kernel");
        if (st) return st;
    }
    StdpArgs a = stdp_args(c, flush);
    if (c->cfg.stdp_layout == 0)
        return check_hip(c, launch_stdp_rows(s, a, c->n_cu, ev), "STDP kernel");
    const size_t lds = (size_t)c->stdp_width * (c->hw * sizeof(uint64_t) + sizeof(float));
    return check_hip(c, launch_stdp(s, a, c->stdp_grid, lds, ev), "STDP kernel");
}

snn_status launch_step_plasticity(snn_ctx *c)
{
    if (c->n_plastic_rows == 0) return SNN_OK;
    if (c->algo == 2) {  // naive: every plastic synapse of every row
        NaiveArgs a{};
        a.row_ptr = c->row_ptr;
        a.pend = c->pend;
        a.col = c->col;
        a.w = c->w;
        a.sx_pre = c->sx_pre;
        a.sx_post = c->sx_post;
        a.mask = c->mask;
        a.txmask = c->txmask;
        a.n_rows = c->n_plastic_rows;
        a.nw = c->nw;
        a.d_plus = c->dpow[1];
        a.d_minus = c->d_minus;
        a.c_pot = c->c_pot;
        a.c_dep = c->c_dep;
        a.mu = c->mu;
        a.stats = c->syn_stats;
        a.syn_count = c->gstats + kGNaiveSyn;
        return check_hip(c, launch_stdp_naive(c->stream, a, c->n_cu, part_events(c, 1)),
                         "naive STDP");
    }
    return launch_plasticity(c, false, c->stream, part_events(c, 1));
}


DeliverArgs deliver_args(snn_ctx *c)
{
    DeliverArgs a{};
    a.row_ptr = c->row_ptr;
    a.col = c->col;
    a.w = c->w;
    a.piv = c->piv;
    a.ring = c->ring;
    a.ring_cnt = c->ring_cnt;
    a.tx_cnt = c->tx_cnt;
    a.clk = c->clk;
    a.delay = c->delay;
    a.apart = c->apart;
    a.ain = c->ain;
    a.part_stride = (int64_t)c->nacc * c->n;
    a.n = c->n;
    a.n_exc = c->cfg.n_exc;
    a.width = c->cfg.slice_width;
    a.n_slices = c->n_slices;
    a.chunks = c->chunks;
    a.nacc = c->nacc;
    a.n_work = c->n_slices * c->chunks;
    a.stats = c->dlv_stats;
    a.col16 = c->col16;
    a.plastic = c->n_plastic_rows > 0 && c->algo != 2;
    a.event = c->algo == 0;
    a.txinfo = c->txinfo;
    a.hist = c->hist;
    a.hw = c->hw;
    a.ypost = c->ypost;
    a.t_last = c->t_last;
    a.xpre = c->xpre;
    a.c_pot = c->c_pot;
    a.c_dep = c->c_dep;
    a.mu = c->mu;
    for (int q = 0; q <= kMaxAge; ++q) a.dpow[q] = c->dpow[q];
    return a;
}

// Parts (2) and (3) of a step in one launch (k_synapse_pass): delivery on
// its usual work items, the forced rows on the CU slots left over. ver >= 0:
// the step of a source block whose lists, histories, post traces, history
// summaries, counts and clock are the block's version ver (SourceArgs).
snn_status launch_step_synapse_pass(snn_ctx *c, KernelEvents ev, int ver = -1)
{
    DeliverArgs d = deliver_args(c);
    const int nd = c->dlv_blocks;
    const int ns = std::max(8, c->fuse_slots - nd);
    StdpArgs a = stdp_args(c, false, (int64_t)ns * (kDlvBlock / kWave));
    if (ver >= 0) {
        const int64_t n = c->n, npl = c->n_plastic_rows;
        d.ring = c->sv_tx + ver * n;
        d.ring_cnt = d.tx_cnt = c->sv_cnt + 2 * ver;
        d.clk = c->sv_clk + ver;
        d.txinfo = c->sv_txinfo + ver * n;
        d.hist = c->sv_hist + ver * n * c->hw;
        d.ypost = c->sv_ypost + ver * n;
        a.info = c->sv_info + ver * npl;
        a.row_cnt = c->sv_cnt + 2 * ver + 1;
        a.tx_cnt = c->sv_cnt + 2 * ver;
        a.clk = c->sv_clk + ver;
        a.hist = d.hist;
        a.ypost = d.ypost;
        if (a.code) a.code = c->sv_code + ver * (int64_t)c->sv_code_stride;
        if (a.recent) a.recent = c->sv_recent + ver * (int64_t)c->nw;
    }
    const size_t table = a.xcd      ? (a.code ? (size_t)c->xcd_table : 0)
                         : a.code   ? (((size_t)c->n + 15) / 16) * 16
                         : a.recent ? (size_t)c->nw * sizeof(uint64_t)
                                    : 0;
    const size_t dlv = dlv_lds_bytes(c) - sizeof(DlvShared) + fused_dlv_shared_bytes(c->hw);
    const size_t lds = std::max(dlv, table + (size_t)fused_queue_bytes(c->hw));
    snn_status st =
        check_hip(c, launch_synapse_pass(c->stream, d, a, nd, ns, lds, ev), "synapse pass kernel");
    if (st) return st;
    c->last_deliver_t = c->t;
    return SNN_OK;
}

snn_status launch_step_delivery(snn_ctx *c, int32_t mode)
{
    DeliverArgs a = deliver_args(c);
    snn_status st;
    if (mode == SNN_DELIVER_LDS_SLICE) {
        // the transmitting rows' plasticity is fused into slice delivery
        st = check_hip(c, launch_deliver_lds(c->stream, a, c->dlv_blocks, dlv_lds_bytes(c),
                                             part_events(c, 2)),
                       "slice delivery kernel");
        if (st) return st;
        c->last_deliver_t = c->t;
        return SNN_OK;
    }
    const KernelEvents ev = part_events(c, 2);
    KernelEvents last{ev.start, ev.stop};
    if (a.plastic) {
        // bring the transmitting rows up to date first (row-wise, L2 gathers)
        StdpArgs r = stdp_args(c, false);
        r.info = c->txinfo;
        r.n_info = c->n;
        r.tx_rows = 1;
        // transmitting rows: the row-wise form, gathering every target's
        // history and post trace (no summary staged)
        r.xcd = 0;
        r.code = nullptr;
        r.recent = nullptr;
        st = check_hip(c, launch_stdp_rows(c->stream, r, c->n_cu, {ev.start, nullptr}),
                       "STDP of transmitting rows");
        if (st) return st;
        last.start = nullptr;
    }
    st = check_hip(c, launch_fill_ll(c->stream, c->apart, a.part_stride, 0), "clear input");
    if (st) return st;
    st = check_hip(c, launch_deliver_global(c->stream, a, kGlobalMaxBlocks, last),
                   "global delivery kernel");
    if (st) return st;
    c->last_deliver_t = c->t;
    return SNN_OK;
}


}  // namespace

extern "C" {

const char *snn_status_string(snn_status s)
{
    switch (s) {
    case SNN_OK: return "ok";
    case SNN_EINVAL: return "invalid argument";
    case SNN_ENOMEM: return "buffer too small";
    case SNN_EDEVICE: return "device error";
    case SNN_ESTATE: return "call out of order";
    }
    return "unknown status";
}

snn_status snn_create(const snn_config *cfg, void *hip_stream, snn_ctx **out)
{
    if (!out) return SNN_EINVAL;
    *out = nullptr;
    if (!cfg) return SNN_EINVAL;
    snn_ctx *c = new (std::nothrow) snn_ctx();
    if (!c) return SNN_ENOMEM;
    c->cfg = *cfg;
    c->stream = (hipStream_t)hip_stream;
    *out = c;
    snn_status st = validate(c, *cfg);
    if (st) return st;
    if (hipGetDevice(&c->device) != hipSuccess)
        return fail(c, SNN_EDEVICE, "no HIP device");
    {
        const hipError_t e = static_scratch(c->device, &c->static_status);
        if (e != hipSuccess)
            return fail(c, SNN_EDEVICE, "the library's device scratch: %s", hipGetErrorString(e));
    }
    int lds_max = 0;
    if (hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, c->device) !=
        hipSuccess)
        return fail(c, SNN_EDEVICE, "cannot query the LDS size");
    if (hipDeviceGetAttribute(&c->n_cu, hipDeviceAttributeMultiprocessorCount, c->device) !=
            hipSuccess ||
        c->n_cu < 1)
        return fail(c, SNN_EDEVICE, "cannot query the compute-unit count");
    const int stat = deliver_lds_static_bytes();
    const int stat_stdp = stdp_static_bytes();
    if (stat < 0 || stat_stdp < 0) return fail(c, SNN_EDEVICE, "cannot query the kernels");
    int64_t need = (int64_t)sizeof(DlvShared) +
                   (int64_t)cfg->slice_width * 8 * (cfg->neuron_model == SNN_LIF_CUBA ? 2 : 1);
    const int hw = cfg->history_bits == 128 ? 2 : 1;
    if (cfg->plastic != SNN_PLASTIC_NONE) need += (int64_t)cfg->slice_width * (8 * hw + 4);
    if (need + stat > lds_max)
        return fail(c, SNN_EINVAL,
                    "slice delivery needs %lld B of LDS (staging, accumulator%s) besides %d B "
                    "of static LDS; the device allows %d", (long long)need,
                    cfg->plastic != SNN_PLASTIC_NONE ? ", histories and post traces" : "", stat,
                    lds_max);
    derive(c);
    if (c->n_plastic_rows > 0) {
        // STDP target groups: mult * W neurons, staged at 12 B each in LDS
        const int64_t per = hw * sizeof(uint64_t) + sizeof(float);
        int mult = cfg->stdp_slice_mult;
        if (mult == 0) {
            mult = 4096 / cfg->slice_width;
            if (mult < 1) mult = 1;
            if (mult > c->n_slices) mult = c->n_slices;
            while (mult > 1 && (int64_t)mult * cfg->slice_width * per + stat_stdp > lds_max) --mult;
        }
        if ((int64_t)mult * cfg->slice_width * per + stat_stdp > lds_max)
            return fail(c, SNN_EINVAL,
                        "STDP staging of %d x %d neurons needs %lld B of LDS; the device "
                        "allows %d", mult, cfg->slice_width,
                        (long long)(mult * cfg->slice_width * per + stat_stdp), lds_max);
        c->stdp_mult = mult;
        c->stdp_width = mult * cfg->slice_width;
        c->stdp_groups = (c->n_slices + mult - 1) / mult;
        int chunks = cfg->stdp_chunks;
        if (chunks == 0) {
            chunks = (512 + c->stdp_groups - 1) / c->stdp_groups;
            if (chunks > 256) chunks = 256;
        }
        c->stdp_chunks = chunks;
        const int64_t work = (int64_t)c->stdp_groups * chunks;
        if (work > (1 << 20)) return fail(c, SNN_EINVAL, "too many STDP work items");
        c->stdp_grid = (int32_t)((work + 7) / 8 * 8);
        c->syn_slots = c->stdp_grid > c->n_cu ? c->stdp_grid : c->n_cu;
    }
    // The fused synapse pass: its static LDS beside the larger of the two
    // parts' dynamic LDS gives the workgroups a CU holds; it is used when
    // the delivery items leave at least half a slot per CU to the forced
    // rows (fewer waves starve them: slower than two launches).
    // Forced rows by target range over the XCDs: on where asked for, codes
    // or no summary are in use, every range has slices and a range's codes
    // fit in LDS. The LDS reservation is made here for the fewest ranges
    // allowed (largest table): a fixed count, or (automatic) the fewest
    // whose codes fit beside the forced rows' queues within the delivery
    // role's LDS, which the count chosen when the graph is bound does not
    // undercut.
    if (c->n_plastic_rows > 0 && c->algo != 2 && cfg->stdp_layout == 0 && cfg->stdp_xcd != 0 &&
        (cfg->stdp_filter == 0 || cfg->stdp_filter == 1)) {
        const int32_t sp = xcd_plastic_slices(c);
        const int64_t dlv = need - (int64_t)sizeof(DlvShared) + (int64_t)fused_dlv_shared_bytes(c->hw);
        int parts = 0;
        for (int p = 2; p <= kXcds && !parts; p *= 2) {
            if (cfg->stdp_xcd > 1 && p != cfg->stdp_xcd) continue;
            if (p > sp) break;
            set_xcd_ranges(c, p);
            const bool fits = c->xcd_table <= kCodeMax &&
                              (cfg->stdp_xcd > 1 || c->xcd_table + fused_queue_bytes(c->hw) <= dlv);
            if (fits) parts = p;
        }
        if (!parts && cfg->stdp_xcd == 1) {  // else the fewest whose codes fit at all
            for (int p = 2; p <= kXcds && p <= sp && !parts; p *= 2) {
                set_xcd_ranges(c, p);
                if (c->xcd_table <= kCodeMax) parts = p;
            }
        }
        c->xcd = parts > 0;
        c->xparts_min = parts;
        if (parts) set_xcd_ranges(c, parts);
    }
    if (c->n_plastic_rows > 0 && c->algo != 2 && cfg->stdp_layout == 0) {
        const int fstat = synapse_pass_static_bytes();
        if (fstat < 0) return fail(c, SNN_EDEVICE, "cannot query the kernels");
        // the history summary the forced rows stage (as stdp_args chooses it)
        const int f = cfg->stdp_filter;
        const bool fits_code = (int64_t)c->n + 16 <= kCodeMax, fits_map = c->nw <= kRecentMaxWords;
        const int64_t code_b = ((int64_t)c->n + 15) / 16 * 16, map_b = (int64_t)c->nw * 8;
        const int64_t table = c->xcd ? c->xcd_table
                              : f == 1 ? code_b
                              : f == 2 ? map_b
                              : f == 0 ? (fits_code ? code_b : fits_map ? map_b : 0)
                                       : 0;
        const int64_t dlv = need - (int64_t)sizeof(DlvShared) + (int64_t)fused_dlv_shared_bytes(c->hw);
        const int64_t dyn = std::max<int64_t>(dlv, table + fused_queue_bytes(c->hw));
        const int64_t per_cu = std::min<int64_t>(2, lds_max / (dyn + fstat));
        c->fuse_slots = (int32_t)(c->n_cu * per_cu);
        c->fuse = per_cu >= 1 && c->fuse_slots - c->dlv_blocks >= c->n_cu / 2;
        // the forced-row workgroups of the pass keep a statistics slot each
        if (c->fuse && c->syn_slots < c->fuse_slots) c->syn_slots = c->fuse_slots;
    }
    // Source blocks (SourceArgs): plastic networks of Bernoulli sources with
    // D = 1, lazy plasticity, whose step runs the fused synapse pass on whole
    // forced rows; at most kSrcMaxSteps steps (or plastic_blocks) per block.
    c->sb_max = 0;
    if (c->n_plastic_rows > 0 && c->algo != 2 && c->delay == 1 &&
        cfg->neuron_model == SNN_BERNOULLI_SOURCE && c->fuse && !c->xcd &&
        cfg->plastic_blocks >= 0)
        c->sb_max = cfg->plastic_blocks > 0 ? std::min<int32_t>(cfg->plastic_blocks, kSrcMaxSteps)
                                            : kSrcMaxSteps;
    plan_workspace(c, nullptr);
    return SNN_OK;
}

void snn_destroy(snn_ctx *ctx) { delete ctx; }

const char *snn_last_error(const snn_ctx *ctx) { return ctx ? ctx->err.c_str() : "null context"; }

snn_status snn_workspace_size(const snn_ctx *ctx, size_t *bytes)
{
    if (!ctx || !bytes) return SNN_EINVAL;
    *bytes = ctx->ws_need;
    return SNN_OK;
}

snn_status snn_bind_workspace(snn_ctx *c, void *device_ptr, size_t bytes)
{
    if (!c) return SNN_EINVAL;
    if (!device_ptr) return fail(c, SNN_EINVAL, "workspace pointer is NULL");
    if ((uintptr_t)device_ptr % kAlign) return fail(c, SNN_EINVAL, "workspace not 256-byte aligned");
    if (bytes < c->ws_need)
        return fail(c, SNN_ENOMEM, "workspace has %zu bytes, needs %zu", bytes, c->ws_need);
    c->ws = (uint8_t *)device_ptr;
    plan_workspace(c, c->ws);
    hipError_t e = launch_init_state(c->stream, c->v, c->ref, c->ie, c->ii, c->hist, c->ypost,
                                     c->t_last, c->xpre, c->n, c->hw);
    if (e == hipSuccess)
        e = launch_fill_ll(c->stream, c->apart, (int64_t)c->chunks * c->nacc * c->n, 0);
    if (e == hipSuccess) e = launch_fill_f32(c->stream, c->ain, (int64_t)c->nacc * c->n, 0.f);
    if (e == hipSuccess) e = launch_fill_i32(c->stream, c->ring_cnt, c->delay, 0);
    if (e == hipSuccess) e = launch_fill_i32(c->stream, c->row_cnt, 1, 0);
    if (e == hipSuccess) e = launch_fill_i32(c->stream, c->tx_cnt, 1, 0);
    if (e == hipSuccess) e = clear_status(c);
    if (e == hipSuccess) e = launch_set_clock(c->stream, c->clk, 0, 1, 1);
    if (e == hipSuccess) e = launch_fill_i32(c->stream, c->err_flag, 1, 0);
    if (e == hipSuccess) e = launch_fill_i32(c->stream, c->pend, c->n, 0);
    if (e == hipSuccess) e = launch_fill_i32(c->stream, c->pev_cnt, 2 * kBatchMax, 0);
    snn_status st = check_hip(c, e, "workspace initialisation");
    if (st) return st;
    c->t = 0;
    c->last_neuron_t = c->last_deliver_t = -1;
    c->graph_state = 0;
    return zero_stats(c);
}

snn_status snn_graph_count_random(snn_ctx *c, int32_t kind, double p_or_fanout,
                                  int64_t *n_edges)
{
    if (!c || !n_edges) return SNN_EINVAL;
    snn_status st = require_ws(c);
    if (st) return st;
    GraphArgs a = graph_args(c);
    a.col = nullptr;
    a.w = nullptr;
    hipError_t e;
    if (kind == SNN_GRAPH_BERNOULLI) {
        if (!(p_or_fanout >= 0 && p_or_fanout <= 1))
            return fail(c, SNN_EINVAL, "connection probability must be in [0, 1]");
        const double thr = std::floor(p_or_fanout * 4294967296.0);
        a.thr = thr >= 4294967295.0 ? 0xFFFFFFFFu : (uint32_t)thr;
        e = launch_graph_count_bernoulli(c->stream, a);
        if (e == hipSuccess) e = launch_scan_i64(c->stream, c->row_ptr + 1, c->n, c->bsum);
    } else if (kind == SNN_GRAPH_FIXED_FANOUT) {
        if (!(p_or_fanout >= 0 && p_or_fanout < (1 << 24)) ||
            p_or_fanout != std::floor(p_or_fanout))
            return fail(c, SNN_EINVAL, "fan-out must be an integer in [0, 2^24)");
        a.fanout = (int32_t)p_or_fanout;
        e = launch_graph_fill_fanout(c->stream, a);
    } else {
        return fail(c, SNN_EINVAL, "unknown graph kind %d", kind);
    }
    st = check_hip(c, e, "graph count");
    if (st) return st;
    int64_t total = 0;
    st = check_hip(c, hipMemcpyAsync(&total, c->row_ptr + c->n, sizeof total,
                                     hipMemcpyDeviceToHost, c->stream), "read edge count");
    if (st) return st;
    st = check_hip(c, hipStreamSynchronize(c->stream), "graph count");
    if (st) return st;
    c->counted_edges = total;
    c->counted_kind = kind;
    c->counted_p = p_or_fanout;
    c->graph_state = 1;
    *n_edges = total;
    return SNN_OK;
}

snn_status snn_graph_size(const snn_ctx *c, int64_t n_edges, size_t *bytes)
{
    if (!c || !bytes || n_edges < 0) return SNN_EINVAL;
    *bytes = (c->algo == 2 ? 4 : 2) * align_up((size_t)n_edges * sizeof(int32_t)) +
             align_up((size_t)c->n * (size_t)(c->n_slices + 1) * 4) +
             (c->ct ? align_up((size_t)n_edges * sizeof(uint16_t)) : 0) +
             (c->pb_max > 0 ? align_up((size_t)c->n * (size_t)(c->pb_groups + 1) * 4) : 0);
    return SNN_OK;
}

snn_status snn_bind_graph(snn_ctx *c, void *device_ptr, size_t bytes, int64_t n_edges)
{
    if (!c) return SNN_EINVAL;
    snn_status st = require_ws(c);
    if (st) return st;
    if (!device_ptr) return fail(c, SNN_EINVAL, "graph pointer is NULL");
    if ((uintptr_t)device_ptr % kAlign) return fail(c, SNN_EINVAL, "graph buffer not 256-byte aligned");
    if (n_edges < 0) return fail(c, SNN_EINVAL, "n_edges must be >= 0");
    if (c->graph_state == 1 && n_edges != c->counted_edges)
        return fail(c, SNN_EINVAL, "n_edges %lld differs from the counted %lld",
                    (long long)n_edges, (long long)c->counted_edges);
    size_t need = 0;
    snn_graph_size(c, n_edges, &need);
    if (bytes < need) return fail(c, SNN_ENOMEM, "graph buffer has %zu bytes, needs %zu", bytes, need);
    c->g = (uint8_t *)device_ptr;
    c->g_bytes = bytes;
    c->n_edges = n_edges;
    choose_xcd_ranges(c);
    const size_t arr = align_up((size_t)n_edges * sizeof(int32_t));
    c->col = (int32_t *)c->g;
    c->w = (float *)(c->g + arr);
    c->piv = (int32_t *)(c->g + 2 * arr);
    const size_t pivb = align_up((size_t)c->n * (size_t)(c->n_slices + 1) * 4);
    c->sx_pre = c->algo == 2 ? (float *)(c->g + 2 * arr + pivb) : nullptr;
    c->sx_post = c->algo == 2 ? (float *)(c->g + 3 * arr + pivb) : nullptr;
    const size_t ctb = c->ct ? align_up((size_t)n_edges * sizeof(uint16_t)) : 0;
    c->col16 = c->ct ? (uint16_t *)(c->g + (c->algo == 2 ? 4 : 2) * arr + pivb) : nullptr;
    c->gpiv = c->pb_max > 0 ? (int32_t *)(c->g + (c->algo == 2 ? 4 : 2) * arr + pivb + ctb)
                            : nullptr;
    if (c->graph_state != 1) c->counted_kind = -1;
    c->graph_state = 2;
    return SNN_OK;
}

snn_status snn_build_graph_random(snn_ctx *c, float w_exc, float w_inh)
{
    if (!c) return SNN_EINVAL;
    snn_status st = require_ws(c);
    if (st) return st;
    if (c->graph_state != 2 || c->counted_kind < 0)
        return fail(c, SNN_ESTATE, "call snn_graph_count_random and snn_bind_graph first");
    if (!std::isfinite(w_exc) || !std::isfinite(w_inh))
        return fail(c, SNN_EINVAL, "weights must be finite");
    GraphArgs a = graph_args(c);
    a.w_exc = w_exc;
    a.w_inh = w_inh;
    hipError_t e = launch_fill_i32(c->stream, c->err_flag, 1, 0);
    if (c->counted_kind == SNN_GRAPH_BERNOULLI) {
        const double thr = std::floor(c->counted_p * 4294967296.0);
        a.thr = thr >= 4294967295.0 ? 0xFFFFFFFFu : (uint32_t)thr;
        if (e == hipSuccess) e = launch_graph_fill_bernoulli(c->stream, a);
    } else {
        a.fanout = (int32_t)c->counted_p;
        if (e == hipSuccess) e = launch_graph_fill_fanout(c->stream, a);
        if (e == hipSuccess && a.fanout > 1) {
            int p2 = 2;
            while (p2 < a.fanout) p2 <<= 1;
            if (a.fanout > kMaxSortRow) return fail(c, SNN_EINVAL, "fan-out above %d", kMaxSortRow);
            e = launch_row_sort(c->stream, a, p2);
        }
    }
    st = check_hip(c, e, "graph fill");
    if (st) return st;
    return finish_graph(c);
}

snn_status snn_build_graph_edges(snn_ctx *c, const int32_t *src, const int32_t *dst,
                                 const float *w)
{
    if (!c) return SNN_EINVAL;
    snn_status st = require_ws(c);
    if (st) return st;
    if (c->graph_state < 2) return fail(c, SNN_ESTATE, "call snn_bind_graph first");
    const int64_t e = c->n_edges;
    if (e > 0 && (!src || !dst || !w)) return fail(c, SNN_EINVAL, "edge arrays are NULL");
    GraphArgs a = graph_args(c);
    hipError_t he = launch_fill_i32(c->stream, c->err_flag, 1, 0);
    if (he == hipSuccess) he = launch_fill_i32(c->stream, c->maxlen, 1, 0);
    if (he == hipSuccess) he = launch_fill_i64(c->stream, c->row_ptr, (int64_t)c->n + 1, 0);
    if (he == hipSuccess) he = launch_edges_count(c->stream, a, src, dst, e);
    if (he == hipSuccess) he = launch_scan_i64(c->stream, c->row_ptr + 1, c->n, c->bsum);
    if (he == hipSuccess)
        he = launch_copy_bytes(c->stream, c->scratch, c->row_ptr, (int64_t)c->n * 8);
    if (he == hipSuccess) he = launch_edges_scatter(c->stream, a, src, dst, w, e, c->scratch);
    if (he == hipSuccess) he = launch_row_maxlen(c->stream, a);
    st = check_hip(c, he, "edge grouping");
    if (st) return st;
    int32_t maxlen = 0, err = 0;
    st = check_hip(c, hipMemcpyAsync(&maxlen, c->maxlen, 4, hipMemcpyDeviceToHost, c->stream),
                   "read row length");
    if (!st)
        st = check_hip(c, hipMemcpyAsync(&err, c->err_flag, 4, hipMemcpyDeviceToHost, c->stream),
                       "read error flag");
    if (!st) st = check_hip(c, hipStreamSynchronize(c->stream), "edge grouping");
    if (st) return st;
    if (err & kErrIndex) return fail(c, SNN_EINVAL, "edge index outside [0, n)");
    if (maxlen > kMaxSortRow) return fail(c, SNN_EINVAL, "a row has more than %d edges", kMaxSortRow);
    if (maxlen > 1) {
        int p2 = 2;
        while (p2 < maxlen) p2 <<= 1;
        st = check_hip(c, launch_row_sort(c->stream, a, p2), "row sort");
        if (st) return st;
    }
    return finish_graph(c);
}

snn_status snn_update_neurons(snn_ctx *c)
{
    if (!c) return SNN_EINVAL;
    snn_status st = require_graph(c);
    if (st) return st;
    if (c->last_neuron_t == c->t)
        return fail(c, SNN_ESTATE, "step %lld is in progress: finish it with snn_advance",
                    (long long)c->t);
    return launch_step_neurons(c);
}

snn_status snn_update_plasticity(snn_ctx *c)
{
    if (!c) return SNN_EINVAL;
    snn_status st = require_graph(c);
    if (st) return st;
    if (c->last_neuron_t != c->t)
        return fail(c, SNN_ESTATE, "update neurons of step %lld first", (long long)c->t);
    return launch_step_plasticity(c);
}

snn_status snn_deliver_spikes(snn_ctx *c, int32_t mode)
{
    if (!c) return SNN_EINVAL;
    snn_status st = require_graph(c);
    if (st) return st;
    if (mode != SNN_DELIVER_LDS_SLICE && mode != SNN_DELIVER_GLOBAL_ATOMIC)
        return fail(c, SNN_EINVAL, "unknown delivery mode %d", mode);
    if (c->last_neuron_t != c->t)
        return fail(c, SNN_ESTATE, "update neurons of step %lld first", (long long)c->t);
    return launch_step_delivery(c, mode);
}

snn_status snn_advance(snn_ctx *c)
{
    if (!c) return SNN_EINVAL;
    snn_status st = require_graph(c);
    if (st) return st;
    if (c->last_neuron_t != c->t)
        return fail(c, SNN_ESTATE, "step %lld has not run", (long long)c->t);
    c->t += 1;  // the device clock advanced with the neuron update
    return SNN_OK;
}

snn_status snn_step(snn_ctx *c, int32_t n_steps, int32_t mode)
{
    if (!c) return SNN_EINVAL;
    snn_status st = require_graph(c);
    if (st) return st;
    if (n_steps < 0) return fail(c, SNN_EINVAL, "n_steps must be >= 0");
    if (mode != SNN_DELIVER_LDS_SLICE && mode != SNN_DELIVER_GLOBAL_ATOMIC)
        return fail(c, SNN_EINVAL, "unknown delivery mode %d", mode);
    if (c->last_neuron_t == c->t)
        return fail(c, SNN_ESTATE, "step %lld is in progress: finish it with snn_advance",
                    (long long)c->t);
    // a small network without plasticity runs whole steps in one workgroup
    // (unless kernel times are being recorded per step)
    const bool small = mode == SNN_DELIVER_LDS_SLICE && c->n_plastic_rows == 0 &&
                       c->n <= kSmallRounds * kSmallBlock &&
                       (int64_t)c->nacc * c->n <= kSmallMaxAcc && c->t_used >= c->t_cap;
    for (int32_t q = 0; small && q < n_steps;) {
        const int32_t k = std::min<int32_t>(n_steps - q, kSmallChunk);
        NeuronArgs a = neuron_args(c);
        SmallArgs b{};
        b.ring = c->ring;
        b.ring_cnt = c->ring_cnt;
        b.delay = c->delay;
        b.row_ptr = c->row_ptr;
        b.col = c->col;
        b.w = c->w;
        b.apart = c->apart;
        b.gstats = c->gstats;
        b.dlv_stats = c->dlv_stats;
        b.status = c->status;
        b.status_words = c->status_words;
        b.n_exc = c->cfg.n_exc;
        b.nacc = c->nacc;
        b.steps = k;
        if ((st = check_hip(c, launch_small_steps(c->stream, a, b), "small-network steps")))
            return st;
        c->t += k;
        c->last_neuron_t = c->last_deliver_t = c->t - 1;
        q += k;
    }
    if (small) return SNN_OK;
    // a network without plasticity and D >= 2 runs in delay blocks (see
    // BatchArgs): one delivery launch for the inputs of steps t+1 .. t+B,
    // then one neuron launch for steps t .. t+B-1
    const bool blocks = mode == SNN_DELIVER_LDS_SLICE && c->batch_max > 0 && c->t_used >= c->t_cap;
    for (int32_t q = 0; blocks && q < n_steps;) {
        const int32_t B = std::min<int32_t>(n_steps - q, c->batch_max);
        DeliverArgs d = deliver_args(c);
        d.batch = B;
        d.abatch = c->abatch;
        d.chunks = 1;
        d.n_work = B * c->n_slices;
        const int grid = (d.n_work + 7) / 8 * 8;
        if ((st = check_hip(c, launch_deliver_lds(c->stream, d, grid, dlv_lds_bytes(c)),
                            "delay-block delivery")))
            return st;
        NeuronArgs a = neuron_args(c);
        BatchArgs b{};
        b.ring = c->ring;
        b.ring_cnt = c->ring_cnt;
        b.delay = c->delay;
        b.status = c->status;
        b.status_stride = c->status_stride;
        b.abatch = c->abatch;
        b.apart = c->apart;
        b.gstats = c->gstats;
        b.err = c->err_flag;
        b.steps = B;
        if ((st = check_hip(c, launch_neuron_steps(c->stream, a, b), "delay-block neurons")))
            return st;
        c->t += B;
        c->last_neuron_t = c->last_deliver_t = c->t - 1;
        q += B;
    }
    if (blocks) return SNN_OK;
    // a plastic network of Bernoulli sources with D = 1 runs in source
    // blocks (see SourceArgs): one launch for the neuron updates and lists
    // of up to sb_max steps, then the synapse pass of each step on its
    // versions (the last step's are the state arrays). The scans' status
    // words are cleared before and after, so that no word a different launch
    // shape left can match a step tag. With kernel timing on, the block's
    // launch is timed as the neuron part of its first step and each pass as
    // the delivery part of its step.
    const bool sblocks = mode == SNN_DELIVER_LDS_SLICE && c->sb_max > 0;
    if (sblocks && n_steps > 0) {
        if ((st = check_hip(c, clear_status(c), "clear the list scans"))) return st;
        NeuronArgs a = neuron_args(c);
        CompactArgs l = compact_args(c);
        for (int32_t q = 0; q < n_steps;) {
            const int32_t B = std::min<int32_t>(n_steps - q, c->sb_max);
            SourceArgs b{};
            b.status = c->status;
            b.status_stride = c->status_stride;
            b.steps = B;
            b.info_slots = c->info_blocks;
            b.code_stride = c->sv_code_stride;
            b.hist = c->sv_hist;
            b.ypost = c->sv_ypost;
            b.code = c->sv_code;
            b.recent = c->sv_recent;
            b.tx = c->sv_tx;
            b.txinfo = c->sv_txinfo;
            b.rows = c->sv_rows;
            b.info = c->sv_info;
            b.cnt = c->sv_cnt;
            b.clk = c->sv_clk;
            if ((st = check_hip(c, launch_source_steps(c->stream, a, l, b, part_events(c, 0)),
                                "source block")))
                return st;
            c->last_neuron_t = c->t;  // the history summaries are current
            for (int32_t k = 0; k < B; ++k) {
                if ((st = launch_step_synapse_pass(c, part_events(c, 2), k < B - 1 ? k : -1)))
                    return st;
                if (c->t_used < c->t_cap) c->t_used += 1;
                c->t += 1;
            }
            q += B;
        }
        if ((st = check_hip(c, clear_status(c), "clear the list scans"))) return st;
        c->last_neuron_t = c->last_deliver_t = c->t - 1;
        return SNN_OK;
    }
    // a plastic network with D >= 2 runs in blocks of up to D-1 steps (see
    // BlockArgs): the plan, then the run of the block, and after the last
    // block the per-step lists
    const bool pblocks = mode == SNN_DELIVER_LDS_SLICE && c->pb_max > 0 && c->t_used >= c->t_cap;
    if (pblocks && n_steps > 0) {
        const NeuronArgs a = neuron_args(c);
        for (int32_t q = 0, k = 0; q < n_steps; ++k) {
            const int32_t B = std::min<int32_t>(n_steps - q, c->pb_max);
            const BlockArgs b = block_args(c, B, k);
            if ((st = check_hip(c, launch_block_plan(c->stream, b), "plastic block plan")))
                return st;
            if ((st = check_hip(c, launch_block_run(c->stream, a, b), "plastic block run")))
                return st;
            if ((st = check_hip(c, launch_block_deferred(c->stream, b), "plastic block deferred")))
                return st;
            c->t += B;
            q += B;
        }
        if ((st = check_hip(c, launch_block_finish(c->stream, block_args(c, 1, 0)),
                            "plastic block lists")))
            return st;
        c->last_neuron_t = c->last_deliver_t = c->t - 1;
        return SNN_OK;
    }
    // parts (2) and (3) of plastic networks in one launch where it fits
    // (kernel timing records it as the delivery part)
    const bool fuse = mode == SNN_DELIVER_LDS_SLICE && c->fuse;
    for (int32_t q = 0; q < n_steps; ++q) {
        if ((st = launch_step_neurons(c))) return st;
        if (fuse) {
            if ((st = launch_step_synapse_pass(c, part_events(c, 2)))) return st;
        } else {
            if ((st = launch_step_plasticity(c))) return st;
            if ((st = launch_step_delivery(c, mode))) return st;
        }
        if (c->t_used < c->t_cap) c->t_used += 1;
        c->t += 1;
    }
    return SNN_OK;
}

snn_status snn_step_static(snn_ctx *c, int32_t n_steps, int32_t mode)
{
    if (!c) return SNN_EINVAL;
    if (c->status_words > kScratchWords)
        return fail(c, SNN_EINVAL,
                    "the list scans need %d status words; the library's scratch holds %lld "
                    "(networks up to %lld neurons)", c->status_words, (long long)kScratchWords,
                    (long long)(kScratchWords / kBatchMax) * 512);
    snn_status st = require_graph(c);
    if (st) return st;
    if (!c->static_status) return fail(c, SNN_EDEVICE, "no device scratch on this device");
    if (n_steps < 0) return fail(c, SNN_EINVAL, "n_steps must be >= 0");
    if (n_steps == 0) return SNN_OK;
    // the array keeps the last call's words (any context on this device):
    // cleared first, with a kernel (no memset node in a captured call)
    st = check_hip(c, launch_fill_i64(c->stream, (int64_t *)c->static_status, c->status_words, 0),
                   "clear the scratch");
    if (st) return st;
    unsigned long long *own = c->status;
    c->status = c->static_status;
    st = snn_step(c, n_steps, mode);
    c->status = own;
    return st;
}

snn_status snn_record_kernel_times(snn_ctx *c, int32_t max_steps)
{
    if (!c) return SNN_EINVAL;
    if (max_steps < 0 || max_steps > (1 << 20))
        return fail(c, SNN_EINVAL, "max_steps must be in [0, 2^20]");
    snn_status st = check_hip(c, hipStreamSynchronize(c->stream), "kernel timing");
    if (st) return st;
    for (hipEvent_t e : c->tev) (void)hipEventDestroy(e);
    c->tev.assign((size_t)max_steps * kTimedParts * 2, nullptr);
    c->t_rec.assign((size_t)max_steps * kTimedParts, 0);
    c->t_cap = c->t_used = 0;
    for (hipEvent_t &e : c->tev) {
        if (hipEventCreate(&e) != hipSuccess) {
            (void)hipGetLastError();
            e = nullptr;
            for (hipEvent_t x : c->tev)
                if (x) (void)hipEventDestroy(x);
            c->tev.clear();
            c->t_rec.clear();
            return fail(c, SNN_EDEVICE, "cannot create timing events");
        }
    }
    c->t_cap = max_steps;
    return SNN_OK;
}

snn_status snn_get_kernel_times(snn_ctx *c, double *mean_ms, int32_t *steps)
{
    if (!c || !mean_ms || !steps) return SNN_EINVAL;
    snn_status st = check_hip(c, hipStreamSynchronize(c->stream), "kernel timing");
    if (st) return st;
    for (int part = 0; part < kTimedParts; ++part) {
        double sum = 0;
        int cnt = 0;
        for (int q = 0; q < c->t_used; ++q) {
            const size_t k = (size_t)q * kTimedParts + part;
            if (!c->t_rec[k]) continue;
            float ms = 0;
            st = check_hip(c, hipEventElapsedTime(&ms, c->tev[2 * k], c->tev[2 * k + 1]),
                           "kernel timing");
            if (st) return st;
            sum += ms;
            ++cnt;
        }
        mean_ms[part] = cnt ? sum / cnt : 0.0;
    }
    *steps = c->t_used;
    return SNN_OK;
}

snn_status snn_flush_plasticity(snn_ctx *c)
{
    if (!c) return SNN_EINVAL;
    snn_status st = require_graph(c);
    if (st) return st;
    if (c->last_neuron_t == c->t)
        return fail(c, SNN_ESTATE, "step %lld is in progress: finish it with snn_advance",
                    (long long)c->t);
    if (c->n_plastic_rows == 0 || c->t == 0 || c->algo == 2) return SNN_OK;  // naive: current
    return launch_plasticity(c, true, c->stream);
}

snn_status snn_probe_rows(snn_ctx *c, int32_t n_rows, int32_t write, uint64_t seed, double *ms,
                          int64_t *synapses)
{
    if (!c || !ms || !synapses) return SNN_EINVAL;
    snn_status st = require_graph(c);
    if (st) return st;
    if (c->n_plastic_rows == 0) return fail(c, SNN_ESTATE, "the network has no plastic rows");
    if (n_rows < 1 || n_rows > (1 << 24))
        return fail(c, SNN_EINVAL, "n_rows must be in [1, 2^24]");
    hipEvent_t ev[2] = {nullptr, nullptr};
    hipError_t e = hipEventCreate(&ev[0]);
    if (e == hipSuccess) e = hipEventCreate(&ev[1]);
    if (e == hipSuccess)
        e = launch_probe_rows(c->stream, c->n_cu, c->row_ptr, c->pend, c->col, c->w, n_rows,
                              c->n_plastic_rows, seed, write ? 1 : 0,
                              (unsigned long long *)c->scratch, KernelEvents{ev[0], ev[1]});
    std::vector<int32_t> pend((size_t)c->n_plastic_rows);
    if (e == hipSuccess)
        e = hipMemcpyAsync(pend.data(), c->pend, pend.size() * sizeof(int32_t),
                           hipMemcpyDeviceToHost, c->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
    float t = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&t, ev[0], ev[1]);
    for (hipEvent_t x : ev)
        if (x) (void)hipEventDestroy(x);
    st = check_hip(c, e, "row probe");
    if (st) return st;
    // the rows the kernel drew: SplitMix64 of seed ^ (5 << 58 | r << 24), high word
    int64_t cnt = 0;
    for (int32_t r = 0; r < n_rows; ++r) {
        uint64_t z = (seed ^ ((5ull << 58) | ((uint64_t)r << 24))) + 0x9E3779B97F4A7C15ull;
        z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
        z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
        z ^= z >> 31;
        cnt += pend[(uint32_t)(z >> 32) % (uint32_t)c->n_plastic_rows];
    }
    *ms = t;
    *synapses = cnt;
    return SNN_OK;
}

snn_status snn_get_state(snn_ctx *c, snn_state_view *out)
{
    if (!c || !out) return SNN_EINVAL;
    snn_status st = require_ws(c);
    if (st) return st;
    st = materialize_input(c);
    if (st) return st;
    int64_t dev_t = 0;
    st = sync_clock(c, &dev_t);
    if (st) return st;
    std::memset(out, 0, sizeof *out);
    out->t = c->t;
    out->v = c->v;
    out->refractory = c->ref;
    out->i_exc = c->ie;
    out->i_inh = c->ii;
    out->hist = c->hist;
    out->trace_post = c->ypost;
    out->t_last = c->t_last;
    out->trace_pre = c->xpre;
    out->input_exc = c->ain;
    out->input_inh = c->nacc == 2 ? c->ain + c->n : nullptr;
    out->spike_mask = c->mask;
    // the last neuron update ran step dev_t - 1; the last delivery sent the
    // spikes of step dev_t - D
    const int sl = ring_slot(c, dev_t > 0 ? dev_t - 1 : 0);
    out->spike_list = c->ring + (int64_t)sl * c->n;
    out->spike_count = c->ring_cnt + sl;
    const int tl = ring_slot(c, dev_t > 0 ? dev_t - c->delay : 0);
    out->tx_list = c->ring + (int64_t)tl * c->n;
    out->tx_count = c->ring_cnt + tl;
    out->stdp_rows = c->rows;
    out->stdp_row_count = c->row_cnt;
    out->ring_lists = c->ring;
    out->ring_counts = c->ring_cnt;
    return SNN_OK;
}

snn_status snn_set_state(snn_ctx *c, const snn_state_view *in)
{
    if (!c || !in) return SNN_EINVAL;
    snn_status st = require_ws(c);
    if (st) return st;
    if (in->t < 0) return fail(c, SNN_EINVAL, "t must be >= 0");
    const int64_t n = c->n;
    if (in->input_exc || in->input_inh) {
        st = materialize_input(c);  // a field not given keeps its current value
        if (st) return st;
    }
    struct Item { void *dst; const void *src; int64_t bytes; };
    const Item items[] = {
        {c->v, in->v, n * 4},           {c->ref, in->refractory, n * 4},
        {c->ie, in->i_exc, n * 4},      {c->ii, in->i_inh, n * 4},
        {c->hist, in->hist, n * 8 * c->hw},     {c->ypost, in->trace_post, n * 4},
        {c->t_last, in->t_last, n * 4}, {c->xpre, in->trace_pre, n * 4},
        {c->ain, in->input_exc, n * 4},
        {c->nacc == 2 ? c->ain + n : nullptr, in->input_inh, n * 4},
        {c->ring, in->ring_lists, (int64_t)c->delay * n * 4},
        {c->ring_cnt, in->ring_counts, (int64_t)c->delay * 4},
    };
    for (const Item &it : items) {
        if (!it.src || !it.dst) continue;
        st = check_hip(c, launch_copy_bytes(c->stream, it.dst, it.src, it.bytes), "state copy");
        if (st) return st;
    }
    if (c->delay > 1 && (in->ring_lists || in->ring_counts)) {
        st = check_hip(c,
                       launch_ring_positions(c->stream, c->ring, c->ring_cnt, c->spk_pos, c->n,
                                             c->delay),
                       "ring positions");
        if (st) return st;
    }
    // the clock: step t, the fp32 input when one was given; the scans' status
    // words cleared (their step tags refer to the old clock)
    const bool inp = in->input_exc || in->input_inh;
    hipError_t e = launch_set_clock(c->stream, c->clk, in->t, inp ? 1 : -1, 1);
    if (e == hipSuccess) e = clear_status(c);
    st = check_hip(c, e, "set the step clock");
    if (st) return st;
    c->t = in->t;
    c->last_neuron_t = c->last_deliver_t = -1;
    return SNN_OK;
}

snn_status snn_get_graph(const snn_ctx *c, snn_graph_view *out)
{
    if (!c || !out) return SNN_EINVAL;
    std::memset(out, 0, sizeof *out);
    if (!c->ws || c->graph_state < 2) return SNN_ESTATE;
    out->n_edges = c->n_edges;
    out->n_slices = c->n_slices;
    out->row_ptr = c->row_ptr;
    out->col = c->col;
    out->w = c->w;
    out->pivots = c->piv;
    out->plastic_end = c->pend;
    out->col16 = c->col16;
    out->stdp_ranges = c->xcd ? c->xparts : 0;
    out->block_steps = c->pb_max > 0 ? c->pb_max : c->sb_max;
    out->block_width = c->pb_width;
    out->block_pivots = c->gpiv;
    return SNN_OK;
}

snn_status snn_get_stats(snn_ctx *c, snn_stats *out)
{
    if (!c || !out) return SNN_EINVAL;
    snn_status st = require_ws(c);
    if (st) return st;
    std::vector<int64_t> g(kGFields), si((size_t)c->info_blocks * kStFields),
        sy((size_t)c->syn_slots), dv(2 * (size_t)c->dlv_slots);
    int32_t err = 0;
    hipError_t e = hipMemcpyAsync(g.data(), c->gstats, g.size() * 8, hipMemcpyDeviceToHost,
                                  c->stream);
    if (e == hipSuccess)
        e = hipMemcpyAsync(&err, c->err_flag, sizeof err, hipMemcpyDeviceToHost, c->stream);
    if (e == hipSuccess)
        e = hipMemcpyAsync(si.data(), c->info_stats, si.size() * 8, hipMemcpyDeviceToHost,
                           c->stream);
    if (e == hipSuccess)
        e = hipMemcpyAsync(sy.data(), c->syn_stats, sy.size() * 8, hipMemcpyDeviceToHost,
                           c->stream);
    if (e == hipSuccess)
        e = hipMemcpyAsync(dv.data(), c->dlv_stats, dv.size() * 8, hipMemcpyDeviceToHost,
                           c->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
    st = check_hip(c, e, "read statistics");
    if (st) return st;
    std::memset(out, 0, sizeof *out);
    out->steps = g[kGSteps];
    out->spikes = g[kGSpikes];
    out->stdp_synapse_updates = g[kGNaiveSyn];  // naive plasticity (0 otherwise)
    out->device_errors = err;
    for (int b = 0; b < c->info_blocks; ++b) {
        out->stdp_rows += si[(size_t)b * kStFields + kStRows];
        out->stdp_forced_rows += si[(size_t)b * kStFields + kStForced];
        out->stdp_synapse_updates += si[(size_t)b * kStFields + kStSyn];
        out->stdp_forced_synapse_updates += si[(size_t)b * kStFields + kStForcedSyn];
    }
    for (int64_t v : sy) out->stdp_forced_weights_written += v;
    out->stdp_weights_written = out->stdp_forced_weights_written;
    for (int b = 0; b < c->dlv_slots; ++b) {
        out->delivered_events += dv[2 * (size_t)b];
        out->stdp_weights_written += dv[2 * (size_t)b + 1];
    }
    return SNN_OK;
}

snn_status snn_reset_stats(snn_ctx *c)
{
    if (!c) return SNN_EINVAL;
    snn_status st = require_ws(c);
    if (st) return st;
    return zero_stats(c);
}

snn_status snn_graph_capture(snn_ctx *c, int32_t n_steps, int32_t mode, snn_graph **out)
{
    if (!c || !out) return SNN_EINVAL;
    *out = nullptr;
    snn_status st = require_graph(c);
    if (st) return st;
    if (n_steps < 1) return fail(c, SNN_EINVAL, "n_steps must be >= 1");
    if (!c->stream) return fail(c, SNN_EINVAL, "the null stream cannot be captured");
    if (c->t_used < c->t_cap)
        return fail(c, SNN_ESTATE, "kernel times are being recorded");
    if (c->last_neuron_t == c->t)
        return fail(c, SNN_ESTATE, "step %lld is in progress: finish it with snn_advance",
                    (long long)c->t);
    // the capture records the launches only: the host's view of time is put back
    const int64_t t0 = c->t, ln = c->last_neuron_t, ld = c->last_deliver_t;
    st = check_hip(c, hipStreamBeginCapture(c->stream, hipStreamCaptureModeThreadLocal),
                   "begin capture");
    if (st) return st;
    st = snn_step(c, n_steps, mode);
    const std::string step_err = c->err;
    hipGraph_t g = nullptr;
    const hipError_t e = hipStreamEndCapture(c->stream, &g);
    c->t = t0;
    c->last_neuron_t = ln;
    c->last_deliver_t = ld;
    if (st) {
        if (g) (void)hipGraphDestroy(g);
        c->err = step_err;
        return st;
    }
    st = check_hip(c, e, "end capture");
    if (st) return st;
    hipGraphExec_t ex = nullptr;
    const hipError_t ei = hipGraphInstantiate(&ex, g, nullptr, nullptr, 0);
    (void)hipGraphDestroy(g);
    st = check_hip(c, ei, "instantiate the captured steps");
    if (st) return st;
    snn_graph *h = new (std::nothrow) snn_graph();
    if (!h) {
        (void)hipGraphExecDestroy(ex);
        return fail(c, SNN_ENOMEM, "host allocation failed");
    }
    h->exec = ex;
    h->steps = n_steps;
    *out = h;
    return SNN_OK;
}

snn_status snn_graph_launch(snn_ctx *c, snn_graph *g)
{
    if (!c || !g || !g->exec) return SNN_EINVAL;
    snn_status st = require_graph(c);
    if (st) return st;
    if (c->last_neuron_t == c->t)
        return fail(c, SNN_ESTATE, "step %lld is in progress: finish it with snn_advance",
                    (long long)c->t);
    st = check_hip(c, hipGraphLaunch(g->exec, c->stream), "launch the captured steps");
    if (st) return st;
    c->t += g->steps;
    c->last_neuron_t = c->last_deliver_t = c->t - 1;
    return SNN_OK;
}

void snn_graph_destroy(snn_graph *g)
{
    if (!g) return;
    if (g->exec) (void)hipGraphExecDestroy(g->exec);
    delete g;
}

}  // extern "C"
