/*
 * Plain CPU oracle for one clock-based SNN simulation step: neuron update,
 * synapse (STDP) update and spike delivery, following the three-step loop of
 * Bautembach, Oikonomidis & Argyros, "Even Faster SNN Simulation with
 * Lazy+Event-driven Plasticity and Shared Atomics" (Sec. I).
 *
 * TEST INFRASTRUCTURE ONLY. This file is the correctness reference that the
 * HIP library is compared against. Only the tests, the smoke check and the
 * CPU-baseline leg of the benchmark may load it; the library never does.
 * It shares no source, header, table or constant with the HIP path: it
 * derives its own constants from the physical parameters and implements the
 * counter-based random generator from its published definition.
 *
 * What it computes, deliberately in the slow, obvious form:
 *   - Neuron update (Sec. I, step 1) in fp32 with a fixed operation order,
 *     so that spikes can be compared bit for bit. Build with
 *     -ffp-contract=off (no fused multiply-add).
 *   - Plasticity (Sec. III-A, Fig. 2(a), the naive form): EVERY plastic
 *     synapse is advanced EVERY step, reading the pre-synaptic spike from
 *     bit (delay-1) of the source's history word and the post-synaptic spike
 *     from bit 0 of the target's history word. Each synapse carries its own
 *     weight and pre/post traces (the 12 B-per-synapse state of Sec. III-A),
 *     kept in double here.
 *   - Delivery (Sec. III-B, Fig. 3(a), the naive row-wise form): every
 *     transmitting row adds its weights to its targets, summed in double and
 *     rounded once to fp32.
 *
 * Readings of points the paper leaves open are listed with each function.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define OR_LIF_DELTA 0
#define OR_LIF_CUBA 1
#define OR_BERNOULLI 2

#define OR_PLASTIC_NONE 0
#define OR_PLASTIC_EXC_EXC 1
#define OR_PLASTIC_ALL 2

#define OR_GRAPH_BERNOULLI 0
#define OR_GRAPH_FIXED_FANOUT 1

#define OR_MAX_POISSON 32

typedef struct oracle_cfg {
    int32_t n, n_exc, delay, model, plastic, poisson_len;
    double dt, tau_m, v_th, v_reset, v_inf, tau_ref, tau_e, tau_i;
    double j_ext, p_fire;
    double tau_plus, tau_minus, lambda, alpha, mu, w0;
    uint64_t seed;
    uint32_t poisson_cdf[OR_MAX_POISSON];
} oracle_cfg;

typedef struct oracle {
    oracle_cfg c;
    /* constants derived here from the physical parameters */
    float k_m, v_th, v_reset, v_inf, d_e, d_i, j_ext;
    int32_t ref_steps;
    uint32_t fire_thr;
    double d_plus, d_minus, c_pot, c_dep;
    /* graph: CSR grouped by source, rows sorted ascending (Sec. III) */
    int64_t n_edges;
    int64_t *row_ptr;
    int32_t *col;
    double *w;
    double *x_pre, *x_post;
    /* neurons */
    float *v, *ie, *ii;
    int32_t *r;
    uint64_t *hist;
    uint64_t *hist_old; /* the 64 steps before those of hist: bit b = step t-64-b */
    float *a_e, *a_i; /* input consumed by the next neuron update */
    /* outputs of the last step */
    uint64_t *mask;
    int32_t *list;
    int32_t count;
    int64_t spikes_total; /* spikes emitted since creation */
    int64_t t;
} oracle;

/* ---------------------------------------------------------------------- */
/* Counter-based random numbers: the SplitMix64 output function (Steele, Lea
 * & Flood 2014) applied to seed XOR key, key = stream<<58 | a<<24 | b. */

uint64_t oracle_splitmix64(uint64_t state)
{
    uint64_t z = state + 0x9E3779B97F4A7C15ULL;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

uint64_t oracle_rng(uint64_t seed, uint32_t stream, uint64_t a, uint64_t b)
{
    uint64_t key = ((uint64_t)stream << 58) | (a << 24) | b;
    return oracle_splitmix64(seed ^ key);
}

static uint32_t rng32(uint64_t seed, uint32_t stream, uint64_t a, uint64_t b)
{
    return (uint32_t)(oracle_rng(seed, stream, a, b) >> 32);
}

static uint32_t prob_threshold(double p)
{
    double x = floor(p * 4294967296.0);
    if (x < 0.0) return 0;
    if (x > 4294967295.0) return 0xFFFFFFFFu;
    return (uint32_t)x;
}

/* ---------------------------------------------------------------------- */

static void derive_constants(oracle *o)
{
    const oracle_cfg *c = &o->c;
    o->k_m = (float)(c->dt / c->tau_m);
    o->v_th = (float)c->v_th;
    o->v_reset = (float)c->v_reset;
    o->v_inf = (float)c->v_inf;
    o->d_e = (float)exp(-c->dt / c->tau_e);
    o->d_i = (float)exp(-c->dt / c->tau_i);
    o->j_ext = (float)c->j_ext;
    o->ref_steps = (int32_t)lround(c->tau_ref / c->dt);
    o->fire_thr = prob_threshold(c->p_fire);
    o->d_plus = exp(-c->dt / c->tau_plus);
    o->d_minus = exp(-c->dt / c->tau_minus);
    /* power-law STDP (Morrison et al. 2007 form):
     *   potentiation  dw = +lambda * w0^(1-mu) * w^mu * x_pre
     *   depression    dw = -lambda * alpha * w * x_post            */
    o->c_pot = c->lambda * pow(c->w0, 1.0 - c->mu);
    o->c_dep = c->lambda * c->alpha;
}

oracle *oracle_new(const oracle_cfg *cfg)
{
    oracle *o = (oracle *)calloc(1, sizeof(oracle));
    if (!o) return NULL;
    o->c = *cfg;
    derive_constants(o);
    int64_t n = cfg->n, nw = (n + 63) / 64;
    o->v = (float *)calloc(n, sizeof(float));
    o->ie = (float *)calloc(n, sizeof(float));
    o->ii = (float *)calloc(n, sizeof(float));
    o->r = (int32_t *)calloc(n, sizeof(int32_t));
    o->hist = (uint64_t *)calloc(n, sizeof(uint64_t));
    o->hist_old = (uint64_t *)calloc(n, sizeof(uint64_t));
    o->a_e = (float *)calloc(n, sizeof(float));
    o->a_i = (float *)calloc(n, sizeof(float));
    o->mask = (uint64_t *)calloc(nw ? nw : 1, sizeof(uint64_t));
    o->list = (int32_t *)calloc(n ? n : 1, sizeof(int32_t));
    o->row_ptr = (int64_t *)calloc(n + 1, sizeof(int64_t));
    if (!o->v || !o->ie || !o->ii || !o->r || !o->hist || !o->hist_old || !o->a_e || !o->a_i ||
        !o->mask || !o->list || !o->row_ptr) {
        free(o);
        return NULL;
    }
    return o;
}

void oracle_free(oracle *o)
{
    if (!o) return;
    free(o->v); free(o->ie); free(o->ii); free(o->r); free(o->hist); free(o->hist_old);
    free(o->a_e); free(o->a_i); free(o->mask); free(o->list);
    free(o->row_ptr); free(o->col); free(o->w); free(o->x_pre); free(o->x_post);
    free(o);
}

/* ---------------------------------------------------------------------- */
/* Graph construction. */

static int synapse_is_plastic(const oracle *o, int32_t k, int32_t j)
{
    if (o->c.plastic == OR_PLASTIC_ALL) return 1;
    if (o->c.plastic == OR_PLASTIC_EXC_EXC) return k < o->c.n_exc && j < o->c.n_exc;
    return 0;
}

static int alloc_edges(oracle *o, int64_t e)
{
    o->n_edges = e;
    o->col = (int32_t *)malloc((e ? e : 1) * sizeof(int32_t));
    o->w = (double *)malloc((e ? e : 1) * sizeof(double));
    if (!o->col || !o->w) return -1;
    if (o->c.plastic != OR_PLASTIC_NONE) {
        o->x_pre = (double *)calloc(e ? e : 1, sizeof(double));
        o->x_post = (double *)calloc(e ? e : 1, sizeof(double));
        if (!o->x_pre || !o->x_post) return -1;
    }
    return 0;
}

static int cmp_i32(const void *a, const void *b)
{
    int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

/* Row k's fixed-fan-out targets: F draws with replacement,
 * j = (u32 * n) >> 32 from stream 1 at (k, draw), sorted ascending. */
void oracle_fanout_row(uint64_t seed, int32_t n, int32_t fanout, int32_t k,
                       int32_t *out)
{
    for (int32_t b = 0; b < fanout; ++b)
        out[b] = (int32_t)(((uint64_t)rng32(seed, 1, (uint64_t)k, (uint64_t)b) *
                            (uint64_t)n) >> 32);
    qsort(out, (size_t)fanout, sizeof(int32_t), cmp_i32);
}

/* Row k of the fixed-probability graph (kind 0 below): the targets j != k
 * whose stream-0 draw at (k, j) is below floor(p * 2^32), ascending. out
 * holds n entries; returns the row length. */
int32_t oracle_bernoulli_row(uint64_t seed, int32_t n, double p, int32_t k, int32_t *out)
{
    const uint32_t thr = prob_threshold(p);
    int32_t c = 0;
    for (int32_t j = 0; j < n; ++j)
        if (j != k && rng32(seed, 0, (uint64_t)k, (uint64_t)j) < thr) out[c++] = j;
    return c;
}

/* Random graph, weights by source type (w_exc for sources below n_exc).
 * kind 0: each ordered pair (k, j), j != k, is present when the stream-0
 *         draw at (k, j) is below floor(p * 2^32).
 * kind 1: fixed fan-out, see oracle_fanout_row.
 * Returns the number of edges, or -1 on allocation failure. */
int64_t oracle_build_random(oracle *o, int32_t kind, double p_or_fanout,
                            float w_exc, float w_inh)
{
    const int32_t n = o->c.n;
    const uint64_t seed = o->c.seed;
    if (kind == OR_GRAPH_BERNOULLI) {
        const uint32_t thr = prob_threshold(p_or_fanout);
#pragma omp parallel for schedule(dynamic, 64)
        for (int32_t k = 0; k < n; ++k) {
            int64_t cnt = 0;
            for (int32_t j = 0; j < n; ++j)
                if (j != k && rng32(seed, 0, (uint64_t)k, (uint64_t)j) < thr) ++cnt;
            o->row_ptr[k + 1] = cnt;
        }
        o->row_ptr[0] = 0;
        for (int32_t k = 0; k < n; ++k) o->row_ptr[k + 1] += o->row_ptr[k];
        if (alloc_edges(o, o->row_ptr[n])) return -1;
#pragma omp parallel for schedule(dynamic, 64)
        for (int32_t k = 0; k < n; ++k) {
            int64_t e = o->row_ptr[k];
            for (int32_t j = 0; j < n; ++j)
                if (j != k && rng32(seed, 0, (uint64_t)k, (uint64_t)j) < thr)
                    o->col[e++] = j;
        }
    } else {
        const int32_t f = (int32_t)p_or_fanout;
        for (int32_t k = 0; k <= n; ++k) o->row_ptr[k] = (int64_t)k * f;
        if (alloc_edges(o, (int64_t)n * f)) return -1;
#pragma omp parallel for schedule(dynamic, 256)
        for (int32_t k = 0; k < n; ++k)
            oracle_fanout_row(seed, n, f, k, o->col + (int64_t)k * f);
    }
#pragma omp parallel for schedule(dynamic, 256)
    for (int32_t k = 0; k < n; ++k) {
        double wk = (double)(k < o->c.n_exc ? w_exc : w_inh);
        for (int64_t e = o->row_ptr[k]; e < o->row_ptr[k + 1]; ++e) o->w[e] = wk;
    }
    return o->n_edges;
}

typedef struct { int32_t dst; float w; } edge_t;

static int cmp_edge(const void *a, const void *b)
{
    const edge_t *x = (const edge_t *)a, *y = (const edge_t *)b;
    if (x->dst != y->dst) return (x->dst > y->dst) - (x->dst < y->dst);
    return (x->w > y->w) - (x->w < y->w);
}

/* Graph from an explicit edge list (host arrays); rows sorted by target,
 * ties by weight. Returns 0, or -1 on a bad index / allocation failure. */
int oracle_build_edges(oracle *o, const int32_t *src, const int32_t *dst,
                       const float *w, int64_t e)
{
    const int32_t n = o->c.n;
    for (int64_t i = 0; i < e; ++i)
        if (src[i] < 0 || src[i] >= n || dst[i] < 0 || dst[i] >= n) return -1;
    memset(o->row_ptr, 0, (size_t)(n + 1) * sizeof(int64_t));
    for (int64_t i = 0; i < e; ++i) o->row_ptr[src[i] + 1]++;
    for (int32_t k = 0; k < n; ++k) o->row_ptr[k + 1] += o->row_ptr[k];
    if (alloc_edges(o, e)) return -1;
    edge_t *tmp = (edge_t *)malloc((e ? e : 1) * sizeof(edge_t));
    int64_t *fill = (int64_t *)malloc((size_t)(n + 1) * sizeof(int64_t));
    if (!tmp || !fill) { free(tmp); free(fill); return -1; }
    memcpy(fill, o->row_ptr, (size_t)(n + 1) * sizeof(int64_t));
    for (int64_t i = 0; i < e; ++i) {
        int64_t p = fill[src[i]]++;
        tmp[p].dst = dst[i];
        tmp[p].w = w[i];
    }
    for (int32_t k = 0; k < n; ++k) {
        int64_t a = o->row_ptr[k], b = o->row_ptr[k + 1];
        qsort(tmp + a, (size_t)(b - a), sizeof(edge_t), cmp_edge);
        for (int64_t q = a; q < b; ++q) { o->col[q] = tmp[q].dst; o->w[q] = tmp[q].w; }
    }
    free(tmp);
    free(fill);
    return 0;
}

/* Slice pivots of one sorted row, by their definition (Fig. 1): pivot s is
 * the number of entries whose target lies below s*W, for s = 0 .. S with
 * S = ceil(n / W). Counting, not searching. */
void oracle_pivots(const int32_t *row, int64_t len, int32_t n, int32_t width,
                   int32_t *out)
{
    int32_t s_count = (n + width - 1) / width;
    for (int32_t s = 0; s <= s_count; ++s) {
        int64_t lim = (int64_t)s * width, c = 0;
        for (int64_t q = 0; q < len; ++q)
            if (row[q] < lim) ++c;
        out[s] = (int32_t)c;
    }
}

/* ---------------------------------------------------------------------- */
/* Step 1: neuron update (Sec. I). All arithmetic in fp32, in this order.
 *   LIF_DELTA: if refractory: count down, hold at reset, no spike, input
 *              dropped; else V <- ((V + (V_inf - V) * k_m) + A) + X, spike
 *              when V >= V_th, then reset and start ref_steps of refractoriness.
 *   LIF_CUBA:  I_e <- I_e * d_e + A_e, I_i <- I_i * d_i + A_i (always);
 *              if not refractory: V <- V + (((V_inf - V) + I_e) + I_i) * k_m.
 *   BERNOULLI: spike when the stream-4 draw at (t, i) is below floor(p 2^32).
 * X = J_ext * k with k ~ Poisson from the stream-3 draw at (t, i) and the
 * inverse-CDF table: k = number of table entries <= the draw.            */
static int neuron_update(oracle *o, int32_t i, int64_t t)
{
    const oracle_cfg *c = &o->c;
    if (c->model == OR_BERNOULLI)
        return rng32(c->seed, 4, (uint64_t)t, (uint64_t)i) < o->fire_thr;

    float v = o->v[i];
    int s = 0;
    if (c->model == OR_LIF_CUBA) {
        float ie = o->ie[i] * o->d_e;
        ie = ie + o->a_e[i];
        float ii = o->ii[i] * o->d_i;
        ii = ii + o->a_i[i];
        o->ie[i] = ie;
        o->ii[i] = ii;
        if (o->r[i] > 0) {
            o->r[i] -= 1;
            v = o->v_reset;
        } else {
            float a = o->v_inf - v;
            a = a + ie;
            a = a + ii;
            float b = a * o->k_m;
            v = v + b;
            if (v >= o->v_th) { s = 1; v = o->v_reset; o->r[i] = o->ref_steps; }
        }
    } else {
        if (o->r[i] > 0) {
            o->r[i] -= 1;
            v = o->v_reset;
        } else {
            float x = 0.0f;
            if (c->poisson_len > 0) {
                uint32_t u = rng32(c->seed, 3, (uint64_t)t, (uint64_t)i);
                int32_t k = 0;
                for (int32_t q = 0; q < c->poisson_len; ++q)
                    if (c->poisson_cdf[q] <= u) ++k;
                x = o->j_ext * (float)k;
            }
            float a = o->v_inf - v;
            float b = a * o->k_m;
            float cc = v + b;
            v = cc + o->a_e[i];
            v = v + x;
            if (v >= o->v_th) { s = 1; v = o->v_reset; o->r[i] = o->ref_steps; }
        }
    }
    o->v[i] = v;
    return s;
}

/* One synapse, one step of the plasticity rule (the user callback of
 * Fig. 2(a)). Both traces decay first; a pre-synaptic spike depresses using
 * the post trace (post spikes strictly before this step), then counts into
 * the pre trace; a post-synaptic spike then potentiates using the pre trace
 * (which already includes a pre spike of this same step), then counts into
 * the post trace. Weights are clamped at zero after depression. */
static void stdp_synapse_step(double *w, double *x_pre, double *x_post, int pre,
                              int post, double d_plus, double d_minus,
                              double c_pot, double c_dep, double mu)
{
    *x_pre *= d_plus;
    *x_post *= d_minus;
    if (pre) {
        *w = *w - c_dep * (*w) * (*x_post);
        if (*w < 0.0) *w = 0.0;
        *x_pre += 1.0;
    }
    if (post) {
        *w = *w + c_pot * pow(*w, mu) * (*x_pre);
        *x_post += 1.0;
    }
}

/* One full simulation step: (1) neurons, (2) synapses, (3) delivery. */
void oracle_step(oracle *o)
{
    const oracle_cfg *c = &o->c;
    const int32_t n = c->n;
    const int64_t t = o->t;
    const int dm1 = c->delay - 1;

    /* (1) neurons; history word: shift in this step's spike at bit 0 */
#pragma omp parallel for schedule(static)
    for (int32_t i = 0; i < n; ++i) {
        int s = neuron_update(o, i, t);
        o->hist_old[i] = (o->hist_old[i] << 1) | (o->hist[i] >> 63);
        o->hist[i] = (o->hist[i] << 1) | (uint64_t)s;
    }
    int64_t nw = (n + 63) / 64;
    memset(o->mask, 0, (size_t)(nw ? nw : 1) * sizeof(uint64_t));
    o->count = 0;
    for (int32_t i = 0; i < n; ++i)
        if (o->hist[i] & 1ULL) {
            o->mask[i >> 6] |= 1ULL << (i & 63);
            o->list[o->count++] = i;
        }
    o->spikes_total += o->count;

    /* (2) synapses: every plastic synapse, every step (Fig. 2(a)):
     * pre = source history bit (delay-1), post = target history bit 0 */
    if (c->plastic != OR_PLASTIC_NONE) {
#pragma omp parallel for schedule(dynamic, 64)
        for (int32_t k = 0; k < n; ++k) {
            int pre = (int)((o->hist[k] >> dm1) & 1ULL);
            for (int64_t e = o->row_ptr[k]; e < o->row_ptr[k + 1]; ++e) {
                int32_t j = o->col[e];
                if (!synapse_is_plastic(o, k, j)) continue;
                int post = (int)(o->hist[j] & 1ULL);
                stdp_synapse_step(&o->w[e], &o->x_pre[e], &o->x_post[e], pre, post,
                                  o->d_plus, o->d_minus, o->c_pot, o->c_dep, c->mu);
            }
        }
    }

    /* (3) delivery (Fig. 3(a)): each transmitting row adds its current
     * weights to its targets; double sums, rounded once to fp32. A source
     * transmits at step t the spike it emitted at t - (delay-1). */
    double *acc_e = (double *)calloc((size_t)n + 1, sizeof(double));
    double *acc_i = (double *)calloc((size_t)n + 1, sizeof(double));
    for (int32_t k = 0; k < n; ++k) {
        if (!((o->hist[k] >> dm1) & 1ULL)) continue;
        double *acc = (c->model == OR_LIF_CUBA && k >= c->n_exc) ? acc_i : acc_e;
        for (int64_t e = o->row_ptr[k]; e < o->row_ptr[k + 1]; ++e) acc[o->col[e]] += o->w[e];
    }
    for (int32_t j = 0; j < n; ++j) {
        o->a_e[j] = (float)acc_e[j];
        o->a_i[j] = (float)acc_i[j];
    }
    free(acc_e);
    free(acc_i);
    o->t = t + 1;
}

void oracle_run(oracle *o, int64_t steps)
{
    for (int64_t q = 0; q < steps; ++q) oracle_step(o);
}

/* ---------------------------------------------------------------------- */
/* State access. */

int64_t oracle_time(const oracle *o) { return o->t; }
void oracle_set_time(oracle *o, int64_t t) { o->t = t; }
int64_t oracle_num_edges(const oracle *o) { return o->n_edges; }
int32_t oracle_spike_count(const oracle *o) { return o->count; }
int64_t oracle_spikes_total(const oracle *o) { return o->spikes_total; }

void oracle_set_neurons(oracle *o, const float *v, const int32_t *r, const float *ie,
                        const float *ii, const uint64_t *hist)
{
    size_t n = (size_t)o->c.n;
    if (v) memcpy(o->v, v, n * sizeof(float));
    if (r) memcpy(o->r, r, n * sizeof(int32_t));
    if (ie) memcpy(o->ie, ie, n * sizeof(float));
    if (ii) memcpy(o->ii, ii, n * sizeof(float));
    if (hist) memcpy(o->hist, hist, n * sizeof(uint64_t));
}

void oracle_get_neurons(const oracle *o, float *v, int32_t *r, float *ie, float *ii,
                        uint64_t *hist)
{
    size_t n = (size_t)o->c.n;
    if (v) memcpy(v, o->v, n * sizeof(float));
    if (r) memcpy(r, o->r, n * sizeof(int32_t));
    if (ie) memcpy(ie, o->ie, n * sizeof(float));
    if (ii) memcpy(ii, o->ii, n * sizeof(float));
    if (hist) memcpy(hist, o->hist, n * sizeof(uint64_t));
}

/* The spike history of the 64 steps before those of the history word (for
 * comparing and forcing a simulator that keeps 128 steps of history). */
void oracle_set_history_old(oracle *o, const uint64_t *h)
{
    if (h) memcpy(o->hist_old, h, (size_t)o->c.n * sizeof(uint64_t));
}

void oracle_get_history_old(const oracle *o, uint64_t *h)
{
    if (h) memcpy(h, o->hist_old, (size_t)o->c.n * sizeof(uint64_t));
}

void oracle_set_input(oracle *o, const float *a_e, const float *a_i)
{
    size_t n = (size_t)o->c.n;
    if (a_e) memcpy(o->a_e, a_e, n * sizeof(float));
    if (a_i) memcpy(o->a_i, a_i, n * sizeof(float));
}

void oracle_get_input(const oracle *o, float *a_e, float *a_i)
{
    size_t n = (size_t)o->c.n;
    if (a_e) memcpy(a_e, o->a_e, n * sizeof(float));
    if (a_i) memcpy(a_i, o->a_i, n * sizeof(float));
}

void oracle_get_spikes(const oracle *o, uint64_t *mask, int32_t *list)
{
    int64_t nw = (o->c.n + 63) / 64;
    if (mask) memcpy(mask, o->mask, (size_t)nw * sizeof(uint64_t));
    if (list) memcpy(list, o->list, (size_t)o->count * sizeof(int32_t));
}

void oracle_get_graph(const oracle *o, int64_t *row_ptr, int32_t *col, double *w)
{
    if (row_ptr) memcpy(row_ptr, o->row_ptr, (size_t)(o->c.n + 1) * sizeof(int64_t));
    if (col) memcpy(col, o->col, (size_t)o->n_edges * sizeof(int32_t));
    if (w) memcpy(w, o->w, (size_t)o->n_edges * sizeof(double));
}

/* The weights of the given edges (count indices into the edge arrays). */
void oracle_get_weights_at(const oracle *o, const int64_t *idx, int64_t count, double *out)
{
    for (int64_t q = 0; q < count; ++q) out[q] = o->w[idx[q]];
}

void oracle_get_traces(const oracle *o, double *x_pre, double *x_post)
{
    if (!o->x_pre) return;
    if (x_pre) memcpy(x_pre, o->x_pre, (size_t)o->n_edges * sizeof(double));
    if (x_post) memcpy(x_post, o->x_post, (size_t)o->n_edges * sizeof(double));
}

/* Number of threads the parallel loops use (for reporting). */
int32_t oracle_threads(void)
{
#ifdef _OPENMP
    return (int32_t)omp_get_max_threads();
#else
    return 1;
#endif
}

void oracle_set_threads(int32_t nt)
{
#ifdef _OPENMP
    if (nt > 0) omp_set_num_threads(nt);
#else
    (void)nt;
#endif
}

/* ---------------------------------------------------------------------- */
/* Independent per-synapse replays for networks of Bernoulli sources, where
 * every spike is a function of (seed, step, neuron) only. They let a test
 * check single outputs of a full-size network without building it.        */

static int bern_spike(const oracle *o, int64_t u, int32_t i)
{
    if (u < 0) return 0;
    return rng32(o->c.seed, 4, (uint64_t)u, (uint64_t)i) < o->fire_thr;
}

/* Weight of one plastic synapse k -> j after the plasticity part of step
 * t_end, replayed naively from step 0 with initial weight w_init. */
double oracle_bernoulli_synapse(const oracle *o, int32_t k, int32_t j, double w_init,
                                int64_t t_end)
{
    double w = w_init, xp = 0.0, xq = 0.0;
    const int dm1 = o->c.delay - 1;
    for (int64_t u = 0; u <= t_end; ++u)
        stdp_synapse_step(&w, &xp, &xq, bern_spike(o, u - dm1, k), bern_spike(o, u, j),
                          o->d_plus, o->d_minus, o->c_pot, o->c_dep, o->c.mu);
    return w;
}

/* Delivered input A(t+1) of a fixed-fan-out network of Bernoulli sources
 * with all synapses plastic, for every target: rows transmitting at step t
 * add their weights as they stand after step t's plasticity. */
void oracle_bernoulli_input(const oracle *o, int32_t fanout, double w_init, int64_t t,
                            float *a_out)
{
    const int32_t n = o->c.n;
    const int dm1 = o->c.delay - 1;
    int32_t *tx = (int32_t *)malloc((size_t)n * sizeof(int32_t));
    int32_t ntx = 0;
    for (int32_t k = 0; k < n; ++k)
        if (bern_spike(o, t - dm1, k)) tx[ntx++] = k;
    int32_t *tg = (int32_t *)malloc((size_t)ntx * fanout * sizeof(int32_t));
    double *wt = (double *)malloc((size_t)ntx * fanout * sizeof(double));
#pragma omp parallel for schedule(dynamic, 4)
    for (int32_t q = 0; q < ntx; ++q) {
        int32_t *row = tg + (int64_t)q * fanout;
        oracle_fanout_row(o->c.seed, n, fanout, tx[q], row);
        for (int32_t b = 0; b < fanout; ++b)
            wt[(int64_t)q * fanout + b] =
                o->c.plastic == OR_PLASTIC_NONE
                    ? w_init
                    : oracle_bernoulli_synapse(o, tx[q], row[b], w_init, t);
    }
    double *acc = (double *)calloc((size_t)n, sizeof(double));
    for (int64_t e = 0; e < (int64_t)ntx * fanout; ++e) acc[tg[e]] += wt[e];
    for (int32_t j = 0; j < n; ++j) a_out[j] = (float)acc[j];
    free(acc); free(wt); free(tg); free(tx);
}
