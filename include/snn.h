/*
 * snn.h - C ABI of libsnn.so, the MI355X (gfx950) synapse pass of a
 * clock-based spiking-neural-network simulator.
 *
 * Method: Bautembach, Oikonomidis & Argyros, "Even Faster SNN Simulation with
 * Lazy+Event-driven Plasticity and Shared Atomics". One simulation step is
 * the three-part loop of Sec. I:
 *   (1) update neurons and note which fire,
 *   (2) update synapses, recovering pre- and post-synaptic spikes,
 *   (3) deliver spikes to the neurons' neighbours.
 * Every part runs in hand-written HIP kernels:
 *   - (1) emits a 64-bit firing mask word per 64 neurons (one wave64 ballot),
 *     an ascending spike list (each workgroup learns where its stretch starts
 *     by a look-back over the counts of the workgroups before it), and shifts
 *     each neuron's firing history of one or two 64-bit words (least
 *     significant bit = most recent step, Fig. 2);
 *   - a ring of the last D spike lists implements the network-wide delay;
 *   - (2) is lazy + event-driven STDP (Sec. III-A, Fig. 2(b,c)): only rows
 *     that transmit this step are brought up to date, replaying the missed
 *     steps by walking the set bits of each target's history; rows idle for
 *     as many steps as the history holds are forced so no post-synaptic
 *     spike leaves the window;
 *   - (3) is slice delivery (Sec. III-B, Fig. 3(b)): the target domain is cut
 *     into slices of W neurons and one workgroup accumulates one slice in
 *     LDS with LDS atomics; a global-atomic row-wise variant (Fig. 3(a)) is
 *     kept for comparison. Both accumulate exact 64-bit fixed-point sums
 *     (32 fractional bits), so delivered inputs do not depend on the order of
 *     the atomic updates; each input is rounded once to fp32;
 *   - the graph is a CSR grouped by source with sorted rows plus per-row
 *     slice pivots (Fig. 1), built on the device.
 *
 * Conventions for every call:
 *   - Ownership. The caller owns all device memory and the HIP stream. The
 *     library never allocates device memory: it works inside the workspace
 *     and graph buffers the caller binds, which stay borrowed until
 *     snn_destroy. The library owns only the host-side snn_ctx.
 *   - Pointers. "device" pointers must be addresses in device memory of the
 *     device that was current at snn_create; "host" pointers are ordinary
 *     process memory. Nothing is retained beyond the call unless stated.
 *   - Streams. All device work is enqueued on the stream given to
 *     snn_create, in call order. Calls that return values computed on the
 *     device synchronise that stream and say so.
 *   - Errors. Every call returns an snn_status and never throws or aborts.
 *     Arguments are checked before any launch; on failure nothing is
 *     enqueued and snn_last_error(ctx) describes the problem. Asynchronous
 *     kernel faults surface as SNN_EDEVICE at the next synchronising call.
 *   - Threads. A context is bound to one stream and is not thread-safe.
 *   - Time. The step index and the source of the next input live on the
 *     device (in the workspace): the neuron update advances the step there,
 *     and no launch of a step depends on its index, so a step captured into
 *     a HIP graph (snn_graph_capture) replays correctly. The host's view of
 *     the step follows the calls made, and is read back from the device by
 *     the calls that synchronise (snn_get_state).
 */
#ifndef SNN_H
#define SNN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum snn_status {
    SNN_OK = 0,
    SNN_EINVAL = 1,  /* bad argument or configuration */
    SNN_ENOMEM = 2,  /* a caller-provided buffer is too small */
    SNN_EDEVICE = 3, /* a HIP call or kernel failed */
    SNN_ESTATE = 4   /* call out of order (e.g. step before the graph exists) */
} snn_status;

/* Neuron dynamics of part (1). All use dt-step Euler integration in fp32. */
enum snn_neuron_model {
    SNN_LIF_DELTA = 0,       /* V += (V_inf - V) dt/tau_m + A + J_ext k_Poisson */
    SNN_LIF_CUBA = 1,        /* exponential exc/inh currents, tau_e / tau_i */
    SNN_BERNOULLI_SOURCE = 2 /* fires with probability p_fire per step */
};

/* Which synapses are plastic (part (2)). */
enum snn_plasticity {
    SNN_PLASTIC_NONE = 0,
    SNN_PLASTIC_EXC_EXC = 1, /* source and target both below n_exc */
    SNN_PLASTIC_ALL = 2
};

/* Delivery algorithm for part (3). */
enum snn_delivery {
    SNN_DELIVER_LDS_SLICE = 0,    /* Fig. 3(b): per-slice LDS accumulation */
    SNN_DELIVER_GLOBAL_ATOMIC = 1 /* Fig. 3(a): row-wise global atomics */
};

/* Random graph families for snn_graph_count_random. */
enum snn_graph_kind {
    SNN_GRAPH_BERNOULLI = 0,   /* each ordered pair j != k with probability p */
    SNN_GRAPH_FIXED_FANOUT = 1 /* F uniform targets per source, with replacement */
};

#define SNN_MAX_POISSON 32
#define SNN_MAX_DELAY 64

/* Network configuration: physical parameters only; the library derives its
 * own fp32 constants (dt/tau_m, exp(-dt/tau), ...) from them. */
typedef struct snn_config {
    int32_t n;            /* neurons, 1 .. 2^24-1 */
    int32_t n_exc;        /* excitatory neurons are 0 .. n_exc-1 (0 <= n_exc <= n) */
    int32_t delay_steps;  /* D, 1 .. 64: a spike emitted at step t reaches the
                             neuron update of step t+D */
    int32_t slice_width;  /* W for LDS delivery: multiple of 64, and the
                             W * 8 B fixed-point accumulator (x2 for CUBA),
                             with plasticity W * (8 * history words + 4) B
                             of staged histories and post traces, and about
                             29 KiB of segment staging must fit in the
                             device's LDS (160 KiB); SNN_EINVAL otherwise */
    int32_t spike_chunks; /* C in 1..64: workgroups that share one slice, each
                             taking 1/C of the spike list (partial sums are
                             added by the next neuron update) */
    int32_t stdp_slice_mult; /* STDP target groups span stdp_slice_mult * W
                             neurons (0 = about 4096); their history words and
                             post traces (12 B each) are staged in LDS */
    int32_t stdp_chunks;  /* workgroups sharing one STDP target group, each
                             taking 1/stdp_chunks of the rows (0 = auto) */
    int32_t stdp_layout;  /* forced rows (idle for 64 steps): 0 = row-wise,
                             waves over each row's synapses, histories
                             looked up as below; 1 = slice-organised, the
                             target group's histories staged in LDS */
    int32_t stdp_filter;  /* row-wise layout, per-neuron summary staged in LDS:
                             0 = automatic (codes if n + 16 <= 97280, else
                             the bitmap if n <= 778240, else none), 1 = history
                             codes (which single step of the window held a
                             spike; more than one: gather), 2 = spike-recency
                             bitmap (gather for targets that fired in the
                             window), 3 = none (gather for every synapse) */
    int32_t history_bits; /* spike history per neuron: 64 (or 0) or 128 steps.
                             Rows idle for that many steps are forced, so 128
                             halves the forced updates of silent rows; the
                             weights are the same either way */
    int32_t plasticity_algorithm; /* 0 = lazy + event-driven (Fig. 2(c)); 1 =
                             lazy only (Fig. 2(b)): rows are still updated
                             only when they transmit or are forced, but each
                             synapse steps through every step of the window;
                             2 = naive (Fig. 2(a)): every plastic synapse
                             every step with its own pre and post traces,
                             which the graph buffer then holds (8 B more per
                             synapse). All three reach the same weights up to
                             rounding; they differ in work */
    int32_t compressed_targets; /* 1 = the graph also holds each target's 16-bit
                             slice-local index, target mod W (Sec. V:
                             compressed slice-local indices; W is bounded by
                             the LDS accumulator, so it always fits), which
                             slice delivery reads instead of the 32-bit target
                             (half the target bytes). Row-wise kernels read
                             the 32-bit targets. 0 = off */
    int32_t stdp_xcd;     /* forced rows partitioned by target range over
                             the XCDs (row-wise layout, history codes or no
                             summary: stdp_filter 0 or 1): 0 = off; 2, 4 or 8
                             = that many ranges; 1 = automatic (the most
                             ranges whose segments still fill about three
                             quarters of a 256-entry part, given the edge
                             count when the graph is bound, and whose codes
                             fit in LDS). The plastic targets are cut into
                             ranges of whole slices; range x belongs to the
                             workgroups on XCDs b mod 8 in [8x/p, 8(x+1)/p),
                             which update the entries of every forced row
                             whose targets lie in range x, so the histories
                             they gather stay in those XCDs' L2. Off where
                             the plastic targets have fewer slices than
                             ranges or no range's codes fit. Same weights
                             either way */
    int32_t plastic_blocks; /* plastic networks (lazy plasticity, slice
                             delivery) with D >= 2 and n <= 65536: snn_step
                             runs blocks of up to min(D-1, 15) steps, each
                             workgroup owning a group of targets through
                             the whole block; plastic networks of
                             Bernoulli sources with D = 1 whose step fuses
                             parts (2) and (3): snn_step runs the neuron
                             updates of up to 16 steps in one launch, then
                             each step's synapse pass (see snn_step). 0 =
                             on; k > 0 = on, at most k steps per block; -1
                             = off (the parts step by step). Same results
                             either way */
    int32_t plastic_block_width; /* targets per group of those blocks: 64, 128
                             or 256, dividing slice_width; 0 = automatic */
    int32_t neuron_model; /* enum snn_neuron_model */
    int32_t plastic;      /* enum snn_plasticity */
    int32_t poisson_len;  /* entries used in poisson_cdf (0 = no external drive) */
    double dt_ms, tau_m_ms, v_th, v_reset, v_inf, tau_ref_ms, tau_e_ms, tau_i_ms;
    double j_ext;         /* mV per external Poisson event */
    double p_fire;        /* Bernoulli source firing probability per step */
    double tau_plus_ms, tau_minus_ms;     /* STDP trace time constants */
    double lambda, alpha, mu, w0;         /* power-law STDP: dw+ = lambda w0^(1-mu)
                                             w^mu x_pre, dw- = -lambda alpha w x_post */
    uint64_t seed;        /* counter-based random streams (graph, drive, sources) */
    /* External drive: k ~ Poisson drawn by inversion, k = #{q : cdf[q] <= u}
     * for the 32-bit draw u of stream 3 at (step, neuron). */
    uint32_t poisson_cdf[SNN_MAX_POISSON];
} snn_config;

typedef struct snn_ctx snn_ctx;

/* A captured sequence of steps (snn_graph_capture); opaque, host-side. */
typedef struct snn_graph snn_graph;

/* Device views of the simulation state, all inside the bound workspace. Each
 * array has n entries unless stated. Returned by snn_get_state (pointers
 * into the workspace, valid until snn_destroy); passed to snn_set_state
 * (caller device buffers to copy from; NULL fields are left unchanged). */
typedef struct snn_state_view {
    int64_t t;              /* index of the next step to run */
    float *v;               /* membrane potential (mV) */
    int32_t *refractory;    /* remaining refractory steps */
    float *i_exc, *i_inh;   /* CUBA currents (mV) */
    uint64_t *hist;         /* firing history, history_bits/64 words per neuron
                               (neuron-major): word 0 bit i = spike at step
                               t-1-i, word 1 bit i = spike at step t-65-i */
    float *trace_post;      /* post-synaptic trace as of the last neuron update */
    int32_t *t_last;        /* step each plastic row was last brought up to date */
    float *trace_pre;       /* pre-synaptic row trace at t_last */
    float *input_exc;       /* fp32 input A(t) the next neuron update uses */
    float *input_inh;       /* (CUBA inhibitory input; NULL otherwise) */
    uint64_t *spike_mask;   /* last neuron update: ceil(n/64) words, bits >= n zero */
    int32_t *spike_list;    /* last neuron update: ascending indices */
    int32_t *spike_count;   /* device int32 */
    int32_t *tx_list;       /* spikes transmitted by the last delivery step
                               (those of step t-D), ascending */
    int32_t *tx_count;      /* device int32 */
    int32_t *stdp_rows;     /* plastic rows forced by the history window at the
                               last neuron update (brought up to date by
                               snn_update_plasticity), ascending; transmitting
                               plastic rows are brought up to date by delivery */
    int32_t *stdp_row_count;/* device int32 */
    int32_t *ring_lists;    /* delay ring: D x n spike lists (each ascending),
                               slot = step mod D */
    int32_t *ring_counts;   /* delay ring: D counts */
} snn_state_view;

/* Device views of the graph (inside the bound graph buffer / workspace).
 * Targets and weights are separate arrays indexed by edge. */
typedef struct snn_graph_view {
    int64_t n_edges;
    int32_t n_slices;      /* S = ceil(n / W) */
    int64_t *row_ptr;      /* n+1 entries: row k is edges row_ptr[k] .. row_ptr[k+1]-1 */
    int32_t *col;          /* targets, ascending within each row */
    float *w;              /* weights, 1:1 with col */
    int32_t *pivots;       /* n x (S+1), row-relative: entries pivots[k][s] ..
                              pivots[k][s+1]-1 of row k target [sW, (s+1)W) */
    int32_t *plastic_end;  /* n: row-relative end of the plastic prefix */
    uint16_t *col16;       /* compressed_targets: n_edges slice-local indices
                              (col mod W), 1:1 with col; else NULL. Derived
                              from col by the graph build */
    int32_t stdp_ranges;   /* target ranges the forced rows are split into
                              (stdp_xcd; 0 = whole rows), fixed when the
                              graph is bound */
    int32_t block_steps;   /* most steps per plastic block or source block
                              of snn_step (plastic_blocks; 0 = steps run one
                              by one) */
    int32_t block_width;   /* targets per group of those blocks (0 = none) */
    int32_t *block_pivots; /* n x (n / block_width rounded up, + 1),
                              row-relative like pivots, at the group
                              boundaries; NULL without blocks */
} snn_graph_view;

typedef struct snn_stats {
    int64_t steps;                 /* completed steps */
    int64_t spikes;                /* spikes emitted */
    int64_t delivered_events;      /* (transmitted spike, outgoing synapse) pairs */
    int64_t stdp_rows;             /* rows brought up to date (incl. forced, flush) */
    int64_t stdp_forced_rows;      /* rows forced by the history window */
    int64_t stdp_synapse_updates;  /* plastic synapses advanced */
    int64_t stdp_weights_written;  /* weights that changed and were stored */
    int64_t stdp_forced_synapse_updates;  /* of stdp_synapse_updates: in forced rows
                                             (snn_update_plasticity) */
    int64_t stdp_forced_weights_written;  /* of stdp_weights_written: by
                                             snn_update_plasticity and flushes
                                             (with global-atomic delivery also
                                             the transmitting rows) */
    int64_t device_errors;         /* conditions flagged by kernels: 4 = a plastic row
                                      fell more than 64 steps behind (its update was
                                      skipped), so its weights are no longer exact;
                                      8 = a transmitting neuron had no entry in the
                                      delay ring (a state set whose ring lists
                                      disagree with the histories); 16 = a list scan
                                      gave up waiting for an earlier workgroup */
} snn_stats;

/* Human-readable name of a status code (static string). */
const char *snn_status_string(snn_status s);

/* Creates a context for cfg on the current HIP device and stream hip_stream
 * (a hipStream_t; NULL = the null stream). Validates cfg (SNN_EINVAL with a
 * message in *out's error if *out could be created, else only the status).
 * Derived constants are computed here on the host. */
snn_status snn_create(const snn_config *cfg, void *hip_stream, snn_ctx **out);

/* Releases the host context. Does not touch caller device memory. NULL is
 * accepted. Work already enqueued is not waited for. */
void snn_destroy(snn_ctx *ctx);

/* Last error message of ctx (empty string if none; never NULL). */
const char *snn_last_error(const snn_ctx *ctx);

/* Bytes of device workspace for neuron state, spike lists, the delay ring,
 * row pointers and statistics, and the per-step lists, snapshots and
 * histories of the blocks snn_step runs (plastic_blocks; for source blocks
 * about 93 bytes per neuron and step of a block besides its last: 350 MB
 * for 250,000 neurons). Depends only on the configuration. */
snn_status snn_workspace_size(const snn_ctx *ctx, size_t *bytes);

/* Binds a device buffer of at least snn_workspace_size bytes (256-byte
 * aligned) and initialises the state: V, currents, histories, traces and
 * inputs 0, t_last = -1, t = 0, statistics 0. SNN_ENOMEM if too small. */
snn_status snn_bind_workspace(snn_ctx *ctx, void *device_ptr, size_t bytes);

/* First half of the random graph builder (Fig. 1 data structures, built on
 * the device as in Sec. IV-B): draws the edge count of every row and scans
 * them into row_ptr. kind SNN_GRAPH_BERNOULLI: pair (k, j), j != k, exists
 * when the stream-0 draw at (k, j) is below floor(p 2^32). kind
 * SNN_GRAPH_FIXED_FANOUT: row k has F = p_or_fanout targets
 * (u32 * n) >> 32 from stream 1 at (k, draw). Synchronises the stream and
 * returns the total in *n_edges. Needs a bound workspace. */
snn_status snn_graph_count_random(snn_ctx *ctx, int32_t kind, double p_or_fanout,
                                  int64_t *n_edges);

/* Bytes of the graph buffer for n_edges edges: int32 targets, fp32 weights
 * and the n x (S+1) pivot table. */
snn_status snn_graph_size(const snn_ctx *ctx, int64_t n_edges, size_t *bytes);

/* Binds a device graph buffer of at least snn_graph_size(n_edges) bytes. */
snn_status snn_bind_graph(snn_ctx *ctx, void *device_ptr, size_t bytes, int64_t n_edges);

/* Second half of the random builder (after snn_graph_count_random and
 * snn_bind_graph with the same edge count): fills sorted rows, weights by
 * source type (w_exc for sources below n_exc, else w_inh), slice pivots and
 * plastic prefixes. Synchronises the stream to check for errors. */
snn_status snn_build_graph_random(snn_ctx *ctx, float w_exc, float w_inh);

/* Builds the graph from an edge list in device memory (src, dst, w each with
 * the n_edges entries given to snn_bind_graph) into the data structures of
 * Fig. 1: an adjacency list grouped by source with every row sorted by
 * target (ties by weight), the synapse array aligned with it, and per row
 * the slice pivots (pivot s = the number of the row's entries whose target
 * lies below s * W, the leading 0 stored explicitly) plus the plastic prefix
 * length. Construction runs on the device, as in Sec. IV-B. Edge arrays are
 * borrowed for the call only. Rows longer than 16384 edges are rejected
 * (SNN_EINVAL), as are indices outside [0, n); SNN_ESTATE before
 * snn_bind_graph. Synchronises the stream. */
snn_status snn_build_graph_edges(snn_ctx *ctx, const int32_t *src, const int32_t *dst,
                                 const float *w);

/* Part (1) of step t (Sec. I): integrates every neuron with its input A(t),
 * writes the firing mask, the ascending spike list into ring slot t mod D,
 * shifts the histories, updates the post-synaptic trace, lists the plastic
 * rows idle for the whole history (forced), snapshots the plastic rows to
 * update at t, and advances the device's step index. SNN_ESTATE while step t
 * is in progress (call snn_advance first). */
snn_status snn_update_neurons(snn_ctx *ctx);

/* Part (2) of step t (Sec. III-A, Fig. 2(c)) for the forced rows: brings
 * them up to step t (lazy), visiting only set history bits (event-driven).
 * Rows transmitting at t are brought up to date by snn_deliver_spikes,
 * immediately before their weights are delivered. */
snn_status snn_update_plasticity(snn_ctx *ctx);

/* Part (3) of step t: delivers the spikes emitted at t-D+1 (ring slot
 * (t-D+1) mod D), producing A(t+1). Each transmitting plastic row is first
 * brought up to step t, with its pre-synaptic spike at t (the remainder of
 * part (2)); with SNN_DELIVER_LDS_SLICE inside the slice kernel, so the row
 * is read once. mode is an enum snn_delivery value. */
snn_status snn_deliver_spikes(snn_ctx *ctx, int32_t mode);

/* Ends step t (t <- t+1 on the host; the device index advanced with part
 * (1)). SNN_ESTATE if part (1) of step t has not run. */
snn_status snn_advance(snn_ctx *ctx);

/* n_steps full steps: parts (1), (2), (3) with delivery mode, then advance.
 * Enqueues only; never synchronises; its launches can be captured into a
 * HIP graph (snn_graph_capture). The result equals that of the separate
 * part calls in every state and statistic; with SNN_DELIVER_LDS_SLICE and
 * no kernel times being recorded, networks without plasticity take fewer
 * launches: up to 4096 neurons run many steps in one workgroup, and with
 * D >= 2 the inputs of up to D-1 steps (at most 16; 8 for CUBA) come from
 * spikes already in the delay ring, so one delivery launch computes them
 * all before one neuron launch runs those steps (Sec. I: the input of step
 * t depends on the spikes of step t-D only). Plastic networks with D >= 2
 * and n <= 65536 (lazy plasticity, snn_config.plastic_blocks) run in blocks
 * of up to D-1 steps (at most 15): the weight a row delivers at t depends
 * only on spikes of its targets and on pre spikes that arrived by t (Sec.
 * III-A: each synapse sees its pre spike D-1 steps after emission), so the
 * rows to update and deliver at each step of the block are known when it
 * starts, and one launch lists them, then one launch runs every step of
 * the block with each workgroup owning a group of targets (their neuron
 * update, and the plasticity and delivery of every listed row's synapses
 * onto them; a forced update that is its row's last of the block delivers
 * nothing and is computed after the block's last step, from the targets'
 * histories at its step); a last launch per call rebuilds the per-step
 * lists. Plastic networks of Bernoulli sources with D = 1 (lazy plasticity,
 * snn_config.plastic_blocks, the fused pass below on whole forced rows) run
 * the neuron part of up to 16 steps in one launch: a source fires on a
 * counter-based draw that no input changes, so the spikes, histories and
 * the rows each step brings up to date (with the t_last and pre trace each
 * update leaves for the next) are known before any of those steps' synapse
 * passes; the launch writes, for each step, the lists, snapshots and
 * histories its pass reads, and the passes then run one per step, in order.
 * Other
 * plastic networks run parts (2) and (3) in one launch where its LDS
 * leaves the forced rows at least half a workgroup slot per CU beside the
 * delivery work items: the forced rows and the transmitting rows of a step
 * are disjoint. */
snn_status snn_step(snn_ctx *ctx, int32_t n_steps, int32_t mode);

/* snn_step for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same steps, states and statistics as snn_step(ctx, n_steps, mode), with the
 * scratch of the steps' list scans (one 64-bit status word per workgroup
 * and step of a launch) in an array the library holds on each device it runs
 * on (1 MiB, kept until the process ends) instead of the bound workspace.
 * The caller still binds the workspace and graph buffers that hold the
 * state. Allocates nothing (no hipMalloc, hipFree or allocating library
 * call); enqueues a clear of the words it uses, then the steps. Every call on
 * one device shares the array: calls that overlap on a device (contexts on
 * different streams) race and must be ordered by the caller. SNN_EINVAL for
 * networks above 4,194,304 neurons (more status words than the array holds)
 * or n_steps < 0; otherwise the errors of snn_step. */
snn_status snn_step_static(snn_ctx *ctx, int32_t n_steps, int32_t mode);

/* Kernel timing for profiling. After this call the next max_steps steps run
 * by snn_step record, per step, the device time of its kernels in three
 * parts: [0] neuron update with its spike / row lists, [1] plasticity,
 * [2] delivery (for the global-atomic mode from the start of the
 * transmitting rows' plasticity to the end of delivery; where snn_step runs
 * parts (2) and (3) in one launch, that launch, with [1] not recorded). Each launch places its own events around the kernel
 * (no extra stream work). 0 stops recording and frees the events. Calls the
 * stream's synchronisation first. */
snn_status snn_record_kernel_times(snn_ctx *ctx, int32_t max_steps);

/* Mean device time per recorded step of each part in milliseconds
 * (mean_ms: 3 doubles, host; 0 for a part that launched nothing) and the
 * number of steps recorded.
 * Synchronises the stream. */
snn_status snn_get_kernel_times(snn_ctx *ctx, double *mean_ms, int32_t *steps);

/* Measurement only: the access pattern of the forced-row update (Sec.
 * III-A: a row's targets and weights are read in full, Fig. 2(c)) without
 * its arithmetic, as the ceiling of what that pattern reaches at a given
 * row count. Streams the targets and weights of n_rows pseudo-random plastic
 * rows (row r draws its index from the stream-5 generator at (r, 0), mod
 * the plastic rows), a wave per part of 512 synapses with non-temporal
 * loads, on the grid of the row-wise STDP kernel; with write != 0 it also
 * stores every weight back unchanged. *ms (host) receives the device time
 * of the one launch, *synapses (host) the synapses covered. Changes no
 * state. Synchronises the stream. SNN_ESTATE without a built graph or
 * without plastic rows; SNN_EINVAL for n_rows outside [1, 2^24]. */
snn_status snn_probe_rows(snn_ctx *ctx, int32_t n_rows, int32_t write, uint64_t seed,
                          double *ms, int64_t *synapses);

/* Captures n_steps steps (snn_step(ctx, n_steps, mode)) into an
 * instantiated HIP graph on the context's stream, for callers that replay a
 * fixed step sequence without host launch work (Sec. I: the step loop).
 * Nothing runs: the capture records the launches only, and the host's view
 * of time is left as it was. Every launch reads the step index and the input
 * source from the device (see Time above) and makes no allocation or memset,
 * so each replay (snn_graph_launch) runs the next n_steps steps and equals
 * snn_step(ctx, n_steps, mode) there. The path a step takes (small
 * networks, delay blocks, plastic blocks, the fused pass) is fixed at
 * capture. *out (host)
 * receives the handle, owned by the caller (snn_graph_destroy); it stays
 * valid while the context and its buffers do. SNN_EINVAL for n_steps < 1 or
 * a context on the null stream (HIP cannot capture it); SNN_ESTATE while
 * kernel times are being recorded, a step is in progress or no graph is
 * built; SNN_EDEVICE if HIP refuses the capture. */
snn_status snn_graph_capture(snn_ctx *ctx, int32_t n_steps, int32_t mode, snn_graph **out);

/* Enqueues one replay of a captured step sequence on the context's stream
 * and advances the host's step index by its length. Never synchronises.
 * SNN_ESTATE while a step is in progress. */
snn_status snn_graph_launch(snn_ctx *ctx, snn_graph *graph);

/* Releases a captured step sequence (NULL is accepted). Replays already
 * enqueued are not waited for. */
void snn_graph_destroy(snn_graph *graph);

/* Brings every plastic row up to the last completed step t-1 (no pre-
 * synaptic spike), so that all weights equal those of per-step updates.
 * Under lazy plasticity (Sec. III-A) a row's weights are brought up to date
 * only when the row transmits or is forced, so between those updates they
 * lag behind the naive per-step form (Fig. 2(a)); after this call every
 * weight equals the naive one up to rounding. Enqueues only (row snapshots,
 * then the row-wise update); a no-op without plastic rows, at t = 0 or with
 * naive plasticity, whose weights are always current. SNN_ESTATE before the
 * graph is built. */
snn_status snn_flush_plasticity(snn_ctx *ctx);

/* Fills *out with device pointers into the workspace and the step index.
 * Delivery accumulates inputs exactly in 64-bit fixed point (32 fractional
 * bits) over C partial sums; this call first converts them into the fp32
 * input the next neuron update would use, so input_exc/input_inh are
 * readable (and writable) fp32 arrays. It reads the step index back from
 * the device, so it synchronises the stream. Every list is ascending as the
 * step wrote it. */
snn_status snn_get_state(snn_ctx *ctx, snn_state_view *out);

/* Copies every non-NULL array of *in (caller device buffers) into the state
 * and sets t = in->t, on the host and on the device. Used for teacher
 * forcing and checkpoint restore. With an input array given, the next
 * neuron update reads the fp32 input. The output-only fields (spike
 * mask/list/count, tx, stdp rows) are ignored. */
snn_status snn_set_state(snn_ctx *ctx, const snn_state_view *in);

/* Device pointers of the graph arrays. */
snn_status snn_get_graph(const snn_ctx *ctx, snn_graph_view *out);

/* Synchronises the stream and returns accumulated counters. */
snn_status snn_get_stats(snn_ctx *ctx, snn_stats *out);

/* Zeroes the counters (enqueued on the stream). */
snn_status snn_reset_stats(snn_ctx *ctx);

#ifdef __cplusplus
}
#endif

#endif /* SNN_H */
