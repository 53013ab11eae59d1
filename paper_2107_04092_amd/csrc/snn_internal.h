// Internal interface between the host runtime (snn_api.hip) and the gfx950
// kernels (snn_kernels.hip). Not part of the public C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <type_traits>
#include <stdint.h>

namespace snn {

constexpr int kBlock = 256;          // threads per workgroup of the element kernels
constexpr int kNeuronBlock = 1024;   // threads per workgroup of the neuron update on large
                                     // networks (one list-scan status word per workgroup)
constexpr int kNeuronSmallN = 65536; // up to this many neurons the update takes kBlock threads
                                     // per workgroup
constexpr int kWave = 64;            // CDNA wavefront width
constexpr int kXcds = 8;             // XCDs of the device: workgroup b runs on XCD b mod 8
constexpr int kMaxPoisson = 32;
constexpr int kMaxSortRow = 16384;   // longest row the LDS row sort accepts
constexpr int kStdpBlock = 512;      // threads of the slice STDP kernel
constexpr int kStdpBatch = 512;      // rows whose segments are staged at once
constexpr int kStdpUnroll = 4;       // elements per thread with loads in flight
constexpr int kStdpWindow = kStdpBlock * kStdpUnroll;  // elements per segment map
constexpr int kGlobalMaxBlocks = 2048;
constexpr int kLdsBytes = 160 * 1024;
// slice widths are bounded by the 8-byte accumulators in LDS, so a slice-local
// index (compressed targets) always fits 16 bits
static_assert(kLdsBytes / 8 <= 65536, "slice-local index must fit 16 bits");
// Spike histories: hw 64-bit words per neuron (1 or 2), neuron-major; word 0
// bit b = step t-b, word 1 bit b = step t-64-b. A plastic row is forced once
// its last update is 64 hw steps old, so every window fits the history.
constexpr int kMaxHistWords = 2;
constexpr int kMaxAge = 64 * kMaxHistWords;

// Delivered inputs are accumulated exactly as 64-bit fixed-point integers with
// 32 fractional bits (sums of |x| < 2^31 mV, resolution 2^-32 mV); integer
// atomics make the sum independent of the order of the atomic updates.
constexpr float kFixScale = 4294967296.0f;        // 2^32
constexpr float kFixUnit = 2.3283064365386963e-10f; // 2^-32

// Per-block statistics slots of the STDP kernel.
enum StdpStat { kStRows = 0, kStForced = 1, kStSyn = 2, kStForcedSyn = 3, kStFields = 4 };

// Global counters.
enum GlobalStat { kGSpikes = 0, kGNaiveSyn = 1, kGSteps = 2, kGFields = 8 };

// Error bits raised by kernels (device int32, ORed).
enum DevError {
    kErrIndex = 1, kErrRowTooLong = 2, kErrWindow = 4, kErrRing = 8,
    kErrLookback = 16  // a list scan waited too long for an earlier workgroup
};

// Per-step scalars, kept on the device (one struct in the workspace). Every
// kernel of a step reads them there rather than from its launch arguments,
// and the neuron update advances the step index, so the launches of a step
// are the same whatever step they run (a captured step replays correctly).
struct StepClock {
    long long t;           // neuron updates run so far: the index of the next step
    int32_t input_forced;  // 1: the next neuron update reads the fp32 input `ain`
    int32_t n_parts;       // 0: it adds this many fixed-point partial sums instead
    long long pad_[2];
};

// Look-back status words of the list scans, one per workgroup (and step of
// a multi-step launch): bits 0-23 and 24-47 two counts, bits 48-61 the step
// they belong to (mod 2^14), bits 62-63 the kind: the workgroup's own counts
// (aggregate) or those of it and every workgroup before it (inclusive).
constexpr unsigned long long kStatusAgg = 1ull << 62;
constexpr unsigned long long kStatusInc = 2ull << 62;
constexpr int kLookbackSpins = 1 << 16;  // bound of the wait for an earlier workgroup (rounds)
constexpr int kLookbackDelay = 16;       // s_sleep units (64 clocks) before the first read

struct NeuronArgs {
    float *v;
    int32_t *ref;
    float *ie, *ii;
    uint64_t *hist;
    float *ypost;
    const int32_t *t_last;
    const long long *apart; // fixed-point partial inputs [n_parts][nacc][n]
    const float *ain;       // fp32 input [nacc][n], used when clk->input_forced
    int64_t part_stride;    // nacc * n
    int32_t max_parts;      // most partial sums a delivery writes (the chunk count)
    StepClock *clk;         // step index and input source (advanced by the update)
    uint64_t *mask;         // spikes emitted at t
    uint64_t *txmask;       // spikes transmitted at t (emitted at t-D+1)
    uint8_t *code;          // per neuron: 0 no spike in the last 64 steps, 1 + i one spike
                            // at step t-i, kCodeMulti more than one (see k_neuron)
    uint64_t *recent;       // neurons with a spike in the last 64 steps (hist != 0)
    int32_t n, n_exc, model, n_plastic_rows, dm1, ref_steps, poisson_len, hw;
    float k_m, v_th, v_reset, v_inf, d_e, d_i, j_ext, d_minus;
    uint32_t fire_thr;
    uint64_t seed;
    uint32_t poisson[kMaxPoisson];
};

struct RowInfo;

// The lists k_neuron builds: spikes of step t (into the delay ring), forced
// plastic rows, and the snapshots of the rows to update at t. The lists are
// ascending: each workgroup's stretch starts at the counts of all earlier
// workgroups, which it learns by a decoupled look-back over their status
// words; the last workgroup publishes the counts and advances the step.
struct CompactArgs {
    int32_t *ring, *ring_cnt;      // delay ring: D lists of n and D counts; step t: slot t mod D
    // the number of rows transmitting at t (the count of ring slot
    // (t-D+1) mod D) at a fixed address, so that the synapse pass needs no
    // load that waits for the clock to find it
    int32_t *tx_cnt;
    int32_t *row_list, *row_cnt;   // forced plastic rows
    unsigned long long *status;    // look-back status words, one per workgroup
    // position of each neuron in the spike list of the step it last fired
    // (only D > 1 with plasticity): [D][n], slot of the step as in the ring
    int32_t *spk_pos;
    int64_t *gstats;
    int32_t n, nw, n_plastic_rows, hw, delay;
    // snapshots of the plastic rows to update at step t (see RowInfo): forced
    // rows aligned with row_list; transmitting rows aligned with the
    // delay-ring list of step t-D+1 (txinfo[r].k = that list's entry r)
    RowInfo *info;
    RowInfo *txinfo;
    const int64_t *row_ptr;
    const int32_t *pend;
    const uint64_t *hist;
    const int32_t *t_last;
    const float *xpre;
    int32_t *err;
    int64_t *info_stats;     // [gridDim.x][kStFields]
    // target-range segments of the forced rows (see StdpArgs::segb), when
    // segb is given: segment x < xparts of row k ends at pivot
    // piv[k][xcd_piv[x + 1]]
    int32_t *segb;
    const int32_t *piv;
    int32_t piv_stride, xparts;
    int32_t xcd_piv[kXcds + 1];
    float dpow[kMaxAge + 1];
};

// Snapshot of one row to bring up to date, taken before the synapse pass;
// the pass reads only snapshots, so the workgroup that commits t_last and
// xpre never races with another that still needs the old values.
struct RowInfo {
    long long rs;    // first edge of the row
    int32_t k;       // row (source neuron)
    int32_t len;     // plastic prefix length; 0 = nothing to do
    int32_t age_pre; // age (1 .. 64 hw) | pre << 8
    float xp0;       // pre trace at the previous update
    float xp_now;    // pre trace after this update
    int32_t pad;
};

struct RowInfoArgs {
    const int32_t *rows;     // list mode: rows to update; nullptr in flush mode
    const int32_t *row_cnt;
    int32_t n_rows_all;      // flush mode: rows 0 .. n_rows_all-1
    int32_t dm1, hw;
    const StepClock *clk;    // flush: rows are brought up to the last completed step
    const int64_t *row_ptr;
    const int32_t *pend;
    const uint64_t *hist;
    const int32_t *t_last;
    const float *xpre;
    RowInfo *info;
    int32_t *err;            // kErrWindow when a row fell more than 64 hw steps behind
    int64_t *stats;          // [gridDim.x][kStFields]
    float dpow[kMaxAge + 1]; // d_plus^i, i = 0..kMaxAge
};

struct StdpArgs {
    const RowInfo *info;
    const int32_t *row_cnt;  // list mode row count (nullptr: flush, n_rows_all)
    // tx_rows: the rows are the transmitted spikes of step t (info = their
    // snapshots, tx_cnt their count)
    int32_t tx_rows;
    const int32_t *tx_cnt;
    int32_t n_rows_all;
    int32_t n_info;  // entries of info (snapshot loads are clamped to it)
    int32_t *t_last;         // committed here: t_last = t, xpre = xp_now
    float *xpre;
    const StepClock *clk;    // t = clk->t - 1: the step whose neuron update ran last
    const int32_t *col;      // synapse targets (sorted per row)
    float *w;                // synapse weights
    const int32_t *piv;      // [n][S+1] delivery pivots, used at multiples of `mult`
    const uint64_t *hist;
    const float *ypost;
    int32_t n, n_slices, mult, width, n_groups, chunks, n_work, target_limit, hw;
    int32_t event;           // 1: replay only the set history bits; 0: every step (lazy only)
    float c_pot, c_dep, mu;
    int64_t *stats;          // [gridDim.x] weights written
    // row-wise layout: per-neuron history codes or the spike-recency bitmap
    // staged in LDS (at most one of them; both nullptr: gather everything)
    const uint8_t *code;
    const uint64_t *recent;
    int32_t nw;              // words of `recent`
    int32_t parts;           // row-wise layout: waves sharing one row (>= 1)
    // Forced rows partitioned by target range over the XCDs (xcd != 0): the
    // plastic targets are cut into xparts (2, 4 or 8) ranges of whole
    // slices, [xlo[x], xlo[x+1]); range x belongs to the 8 / xparts XCDs
    // b mod 8 in [x 8 / xparts, (x + 1) 8 / xparts), whose waves bring up
    // to date the entries of every forced row with targets in range x: the
    // target histories they gather stay in those XCDs' L2, and they stage
    // the history codes of range x only. The entries of forced row r (list
    // position) in range x are segb[8 r + x - 1] (0 for x = 0) ..
    // segb[8 r + x] - 1, boundaries moved to 128-byte lines of the weight
    // array so that no line is shared by two ranges (a target next to a
    // boundary may fall outside the range: it is gathered).
    int32_t xcd, xparts;
    const int32_t *segb;
    int32_t xlo[kXcds + 1];
    float dpow[kMaxAge + 1];
};

struct DeliverArgs {
    const int64_t *row_ptr;
    const int32_t *col;
    float *w;
    const int32_t *piv;      // [n][S+1]
    // the transmitted spikes of step t = clk->t - 1: delay-ring slot
    // (t - D + 1) mod D (a delay block: slots of its steps, below)
    const int32_t *ring, *ring_cnt;
    const int32_t *tx_cnt;   // the transmitted spikes' count of the step (see CompactArgs)
    StepClock *clk;
    long long *apart;        // fixed-point partial inputs [C][nacc][n]
    float *ain;              // fp32 input [nacc][n], written directly when C == 1
    int64_t part_stride;
    int32_t n, n_exc, width, n_slices, chunks, nacc, n_work, hw;
    const uint16_t *col16;   // compressed targets: slice-local indices (nullptr: read `col`)
    int64_t *stats;          // [gridDim.x][2]: events delivered, weights written
    // delay block (no plasticity): batch > 0 delivers, before the block's
    // neuron launch, the spikes emitted at steps t0 + 1 - D .. t0 + batch - D
    // (t0 = clk->t, the block's first step), work item (b, slice, chunk)
    // writing fixed-point partial c of step b to abatch (the host passes one
    // chunk, so each item writes the whole sum); n_work counts all batch items
    int32_t batch, delay;
    long long *abatch;       // [batch][chunks][nacc][n]
    // plasticity of the transmitting rows, fused into slice delivery
    int32_t plastic;         // 0: no plastic rows
    int32_t event;           // as in StdpArgs
    const RowInfo *txinfo;   // aligned with the transmitted list
    const uint64_t *hist;
    const float *ypost;
    int32_t *t_last;
    float *xpre;
    float c_pot, c_dep, mu;
    float dpow[kMaxAge + 1];
};

// Naive plasticity (every plastic synapse every step, per-synapse traces).
struct NaiveArgs {
    const int64_t *row_ptr;
    const int32_t *pend;     // plastic prefix length per row
    const int32_t *col;
    float *w;
    float *sx_pre, *sx_post; // per-synapse pre and post traces
    const uint64_t *mask;    // spikes of step t (post)
    const uint64_t *txmask;  // spikes transmitted at t (pre)
    int32_t n_rows, nw;
    float d_plus, d_minus, c_pot, c_dep, mu;
    int64_t *stats;          // [gridDim.x] weights written
    int64_t *syn_count;      // synapse updates (one counter)
};

struct GraphArgs {
    int64_t *row_ptr;        // n+1
    int32_t *col;
    uint16_t *col16;         // compressed targets (encoded from col), or nullptr
    float *w;
    int32_t *piv;
    int32_t *pend;
    int32_t *err;
    int32_t *maxlen;
    uint64_t seed;
    int32_t n, n_exc, width, n_slices, plastic, fanout;
    uint32_t thr;
    float w_exc, w_inh;
};

// Several whole steps of a small network without plasticity in one launch of
// one workgroup (k_small_steps): neuron update, spike list into the delay
// ring, and delivery into an LDS accumulator that the next step's neuron
// update reads, so no step waits for a kernel boundary or an HBM round trip.
struct SmallArgs {
    int32_t *ring, *ring_cnt;   // delay ring: D lists of n, D counts
    int32_t delay;
    const int64_t *row_ptr;
    const int32_t *col;
    const float *w;
    long long *apart;           // after the last step: part 0 = the pending input
    int64_t *gstats;            // kGSpikes
    int64_t *dlv_stats;         // slot 0: events delivered
    // the list scans' status words, cleared at the end (the steps run here
    // leave stale step tags in them)
    unsigned long long *status;
    int32_t status_words;
    int32_t n_exc, nacc, steps;
};
constexpr int kSmallBlock = 1024;
constexpr int kSmallRounds = 4;     // neurons per thread: n <= 4096
constexpr int kSmallMaxAcc = 8192;  // nacc * n accumulators (64 KiB of LDS)
constexpr int kSmallChunk = 4096;   // steps per launch

// Delay-blocked steps of a network without plasticity and delay D >= 2
// (k_neuron_steps after a batched k_deliver_lds). The input of step t comes
// from the spikes of step t-D only, so the inputs of steps t0+1 .. t0+B
// (B <= D-1) depend on spikes already in the delay ring when step t0
// starts: one delivery launch computes all B of them, then one neuron
// launch runs steps t0 .. t0+B-1, each thread keeping its neuron's state in
// registers across the B steps.
struct BatchArgs {
    int32_t *ring, *ring_cnt;   // delay ring: D lists of n, D counts
    int32_t delay;
    unsigned long long *status; // [kBatchMax][status_stride] look-back status words (step
                                // k of the block: row k, one word per workgroup)
    int32_t status_stride;
    const long long *abatch;    // [B][nacc][n] fixed-point inputs of steps t0+1 .. t0+B
    long long *apart;           // partial 0 receives the input of step t0+B
    int64_t *gstats;            // kGSpikes
    int32_t *err;
    int32_t steps;
};
constexpr int kBatchMax = 16;  // steps per delay block
// steps per delay block for neuron model m (CUBA: two inputs per step)
constexpr int batch_steps_max(int m) { return m == 1 ? kBatchMax / 2 : kBatchMax; }
constexpr int64_t kBatchBytes = 256ll << 20;  // most workspace for a block's partial inputs

// Blocks of steps of a plastic network with D >= 2 (k_block_plan, then
// k_block_run). Delivery at step t sends the spikes emitted at t-D+1, and
// the weight of synapse k->j at t depends only on the pre spikes of k that
// arrived by t (emitted by t-D+1) and on the post spikes of j. So the rows
// to bring up to date and to deliver at each of the steps t0 .. t0+B-1
// (B <= D-1) follow from the histories when t0 starts, and a workgroup that
// owns a range of targets can run all B steps alone: the neuron update of
// its targets, then the plasticity and delivery of every listed row's
// entries that fall in its range, into an accumulator in LDS that its next
// neuron update reads. No workgroup waits for another within the block.
//   The plan (one thread per row) walks each row through the block's steps
// as the neuron update would (transmitting: history bit D-1 of the step;
// forced: idle for 64 hw steps), and writes each step's list of row updates
// (PbEvent), each workgroup's share placed by one atomic add per list, and
// commits t_last and x_pre after the block. A forced update that is its row's last
// event of the block delivers nothing and no later event of the block reads
// its weights: it goes to one more list, the deferred updates, which the run
// computes after the block's last step from the targets' histories at the
// update's step (the history at block start and the block's spike bits). A group finds a row's entries with
// targets in the group from the pivot table at group granularity
// (gpiv[k][g] = the row-relative first entry of row k with a target >=
// g gwidth, g = 0..n_groups; the pivot kernel with gwidth for the slice
// width). After the last
// block of a call, k_block_finish rebuilds from the histories what the
// step-by-step path keeps per step: the delay-ring lists of the last D
// steps with their positions, the masks and forced-row list of the last
// step; and clears the list scans' status words.
struct BlockClock {
    long long t0;          // the block's first step
    int32_t input_forced;  // the input of step t0, as the step clock said
    int32_t n_parts;
    long long pad_[2];
};
// One row to bring up to date (and deliver) at a step of a block.
struct PbEvent {
    int32_t rs;      // first edge of the row
    uint32_t lenf;   // plastic prefix length (bits 0-15), age (16-23), pre spike (24),
                     // transmitting (25), inhibitory source of a CUBA network (26),
                     // step in the block (27-30)
    float xp0;       // pre trace at the row's previous update
    int32_t k;       // the row
};
constexpr int kPbPlanBlock = 512;   // threads of the plan (one row each, a half wave per step's scan)
constexpr int kPbBlock = 512;       // threads of a target group's workgroup
constexpr int kPbMaxWidth = 256;    // most targets per group (one neuron per thread)
constexpr int kPbSegs = 2 * kPbBlock;  // a step's records staged at once (two per thread)
constexpr int kPbUnroll = 16;       // flattened entries per thread per window
constexpr int kPbWindow = kPbBlock * kPbUnroll;
constexpr int kPbRecords = 5120;    // a block's records a workgroup holds in LDS
constexpr int kPbMaxN = 65536;      // largest network the blocks run
constexpr int kPbMaxSteps = kBatchMax - 1;  // steps per block: lists 0 .. B-1, deferred list B
constexpr int kPbDfPart = 8 * 64;   // entries per part of a deferred row (8 per lane)
static_assert(kPbPlanBlock / 32 >= kPbMaxSteps + 1, "a half wave per list scan");
static_assert(kPbMaxSteps < 16, "step in the block fits PbEvent::lenf");
static_assert(kPbSegs < 65535, "16-bit segment map");
struct BlockArgs {
    // plan
    const int64_t *row_ptr;
    const int32_t *pend;
    const uint64_t *hist;
    int32_t *t_last;
    float *xpre;
    unsigned long long *status;  // look-back words of the step-by-step kernels (the finish
    int32_t status_stride;       // clears them)
    PbEvent *ev;                 // [steps + 1][n]: step k's rows at ev + k n, the deferred
                                 // forced updates at ev + steps n
    int32_t *ev_cnt;             // [kBatchMax]: the lists' lengths (0 when the plan starts)
    int32_t *ev_cnt_next;        // [kBatchMax]: the other block's, cleared by the plan
    uint8_t *dcode;              // [n, padded to 16] run -> deferred: per target, the first
                                 // spike step of the block (bits 0-3), the latest spike before
                                 // it against a forced window (4-7)
    uint64_t *hq;                // [n][2 hw] run -> deferred: history words at block start,
                                 // then the block's spikes (bit 0: its last step)
    int32_t n_cu;
    int32_t df_parts;            // parts of kDfPart entries of the longest row (deferred)
    BlockClock *bclk;            // written by the plan, read by the run
    StepClock *clk;              // read by the plan, advanced by the run
    int64_t *info_stats;         // plan: rows, forced rows, synapses (kStFields per slot)
    int32_t info_slots;
    int32_t *err;
    int32_t steps, n, n_exc, n_plastic_rows, hw, delay, nacc;
    // run
    const int32_t *col;
    const uint16_t *col16;       // compressed targets (slice-local), or nullptr
    float *w;
    const int32_t *gpiv;         // [n][n_groups + 1]
    int64_t n_edges;
    int32_t gwidth, width, n_groups;
    long long *apart;            // partial 0 receives the input of step t0 + B
    int64_t part_stride;
    int64_t *dlv_stats;          // [dlv_slots][2]: events delivered, weights written (transmitting rows)
    int32_t dlv_slots;
    int64_t *syn_stats;          // [syn_slots]: weights written (forced rows)
    int32_t syn_slots;
    int64_t *gstats;
    int32_t event;               // 1: replay only the set history bits; 0: every step
    float c_pot, c_dep, mu;
    // finish
    int32_t *ring, *ring_cnt, *spk_pos, *rows, *row_cnt;
    uint64_t *mask, *txmask, *recent;
    int32_t status_words;
    float dpow[kMaxAge + 1];
};
// Blocks of steps of a plastic network of Bernoulli sources with D = 1
// (k_source_steps, then one synapse pass per step). A source fires on a
// counter-based draw that no input changes, so one launch runs the neuron
// update of B steps: each thread walks its neuron through them (spike,
// history, post trace) and its row through the updates of each step
// (transmitting, or forced by the history window), with t_last and x_pre
// carried in registers from one update to the next exactly as the synapse
// passes will commit them. For every step it writes what that step's pass
// reads: the histories, post traces and history summaries after the step,
// its transmitted and forced lists, ascending (one decoupled look-back per
// step, the B scans together), their snapshots, their counts and a copy of
// the clock. The last step of the block writes to the state arrays
// themselves (ring slot, lists, counts, masks, clock), so after the block
// the state is that of the step-by-step path; the steps before it write to
// versions of those arrays in the workspace (step k at k times the stride
// of each). The passes then run one per step, in order.
struct SourceArgs {
    unsigned long long *status;  // [kBatchMax][status_stride]: step k's scan in row k
    int32_t status_stride;
    int32_t steps;               // B: 1 .. kSrcMaxSteps
    int32_t info_slots;          // statistics slots of CompactArgs::info_stats
    int32_t code_stride;         // bytes per version of `code`
    uint64_t *hist;              // versions: [B-1][n][hw]
    float *ypost;                // [B-1][n]
    uint8_t *code;               // [B-1][code_stride]
    uint64_t *recent;            // [B-1][nw]
    int32_t *tx;                 // [B-1][n]: the transmitted (= spike) list of the step
    RowInfo *txinfo;             // [B-1][n]
    int32_t *rows;               // [B-1][n_plastic_rows]: the forced rows
    RowInfo *info;               // [B-1][n_plastic_rows]
    int32_t *cnt;                // [B-1][2]: transmitted and forced counts
    StepClock *clk;              // [B-1]: t = t0 + k + 1, as after the step's neuron update
};
constexpr int kSrcMaxSteps = kBatchMax;  // steps per source block (one scan per half wave)

hipError_t launch_block_plan(hipStream_t s, const BlockArgs &b);
hipError_t launch_block_run(hipStream_t s, const NeuronArgs &a, const BlockArgs &b);
hipError_t launch_block_deferred(hipStream_t s, const BlockArgs &b);
hipError_t launch_block_finish(hipStream_t s, const BlockArgs &b);

// Optional events placed by a launch itself around the kernel
// (hipExtLaunchKernelGGL): its device time without marker or dispatch gaps.
struct KernelEvents {
    hipEvent_t start = nullptr, stop = nullptr;
};
// timed parts of a step: neuron update with its lists, plasticity, delivery
constexpr int kTimedParts = 3;
// k_source_steps (see SourceArgs) and its workgroups for n neurons
hipError_t launch_source_steps(hipStream_t s, const NeuronArgs &a, const CompactArgs &c,
                               const SourceArgs &b, KernelEvents ev = {});
int source_steps_grid(int32_t n);

// ---- launchers (k_*.hip); all enqueue on `s` and return the launch
// status of the last kernel they started.
hipError_t launch_init_state(hipStream_t s, float *v, int32_t *ref, float *ie, float *ii,
                             uint64_t *hist, float *ypost, int32_t *t_last, float *xpre,
                             int32_t n, int32_t hw);
hipError_t launch_fill_f32(hipStream_t s, float *p, int64_t count, float value);
hipError_t launch_fill_i64(hipStream_t s, int64_t *p, int64_t count, int64_t value);
hipError_t launch_fill_i32(hipStream_t s, int32_t *p, int64_t count, int32_t value);
hipError_t launch_fill_ll(hipStream_t s, long long *p, int64_t count, long long value);
hipError_t launch_copy_bytes(hipStream_t s, void *dst, const void *src, int64_t bytes);
// k_small_steps: steps a.t .. a.t + b.steps - 1 (a describes step a.t)
hipError_t launch_small_steps(hipStream_t s, const NeuronArgs &a, const SmallArgs &b,
                              KernelEvents ev = {});
hipError_t launch_neuron(hipStream_t s, const NeuronArgs &a, const CompactArgs &b,
                         KernelEvents ev = {});
// workgroups of k_neuron and k_neuron_steps for n neurons (one status word each)
int neuron_grid(int32_t n);
int neuron_steps_grid(int32_t n);
// k_neuron_steps: steps a.t .. a.t + b.steps - 1 (a describes step a.t)
hipError_t launch_neuron_steps(hipStream_t s, const NeuronArgs &a, const BatchArgs &b);
// pos[q n + ring[q n + r]] = r for every delay-ring slot q < d and r < its count
hipError_t launch_ring_positions(hipStream_t s, const int32_t *ring, const int32_t *cnt,
                                 int32_t *pos, int32_t n, int32_t d);
hipError_t launch_row_info(hipStream_t s, const RowInfoArgs &a, int64_t max_rows);
hipError_t launch_stdp(hipStream_t s, const StdpArgs &a, int blocks, size_t lds, KernelEvents ev = {});
hipError_t launch_stdp_rows(hipStream_t s, const StdpArgs &a, int blocks, KernelEvents ev = {});
hipError_t launch_stdp_naive(hipStream_t s, const NaiveArgs &a, int blocks, KernelEvents ev = {});
// k_probe_rows: measurement only (sink: one scratch word)
hipError_t launch_probe_rows(hipStream_t s, int blocks, const int64_t *row_ptr,
                             const int32_t *pend, const int32_t *col, float *w, int32_t n_rows,
                             int32_t n_plastic, uint64_t seed, int32_t write,
                             unsigned long long *sink, KernelEvents ev);
constexpr int kStdpRowsBlock = 1024;   // threads of the row-wise STDP kernel
constexpr int kStdpRowsUnroll = 8;     // synapses per lane and row part (64-step histories)
constexpr int kStdpRowsUnroll2 = 8;    // the same with 128-step histories (4: 28.3 against
                                       // 26.4 us for the stress network's fused pass)
constexpr int kStdpXcdUnroll = 4;      // the same in the target-range form (both lengths)
constexpr int kDlvBlock = 512;         // threads per workgroup of slice delivery
constexpr int kDlvBatch = 704;         // spikes whose segments slice delivery stages at once
                                       // (two per thread: 1,250 spikes over two chunks fit
                                       // one batch, 4.5 standard deviations above the mean)
constexpr int kDlvUnroll = 8;          // flattened elements per thread per window
constexpr int kDlvWindow = kDlvBlock * kDlvUnroll;
// Slice delivery's staging arrays, at the start of its dynamic LDS. MapT is
// the element type of the segment map: int, or uint16_t where LDS is tight
// (the fused pass with 128-step histories), at the cost of a few registers.
template <typename MapT>
struct DlvSharedT {
    long long start[kDlvBatch];        // segment starts (edge index)
    long long sh[kDlvBlock / 64];      // scan scratch
    unsigned long long written;        // weights written by the workgroup
    long long total;                   // the scan's running total between its rounds
    int off[kDlvBatch + 1];            // segment offsets in the batch
    // per segment: plastic elements (bits 0-17), row age (bits 18-25: the
    // replay window), inhibitory source of a CUBA network (bit 26)
    int info[kDlvBatch];
    // pre trace at the last update (the trace after this one, x0 d+^age + 1,
    // is computed where it is needed, as the neuron update computed it)
    float xp0[kDlvBatch];
    MapT map[kDlvWindow];              // element -> 1 + segment of the window (0: none)
    float dpow[kMaxAge + 1];           // decay table
    int shi[kDlvBlock / 64];           // scan scratch
    int nlong;                         // segments longer than the direct-map limit
    int pad_[1];
};
using DlvShared = DlvSharedT<int>;
using DlvShared16 = DlvSharedT<uint16_t>;
// the fused pass's map type: 16-bit with 128-step histories (two workgroups
// per CU on the stress network), else int
template <int HW>
using FusedMap = typename std::conditional<HW == 2, uint16_t, int>::type;
inline size_t fused_dlv_shared_bytes(int hw)
{
    return hw == 2 ? sizeof(DlvShared16) : sizeof(DlvShared);
}
static_assert(sizeof(DlvShared) % 16 == 0 && sizeof(DlvShared16) % 16 == 0,
              "the accumulators follow 16-byte aligned");
constexpr int kStoreLine = 32;         // weights per store line of the row-wise STDP (128 B)
constexpr int kStdpRowsSplit = 8;      // most waves that share one row


// LDS of the row-wise STDP workgroup's candidate queues (one per wave: target
// and weight of up to U x 64 synapses)
constexpr int stdp_rows_queue_bytes(int hw)
{
    return (kStdpRowsBlock / kWave) * (hw == 2 ? kStdpRowsUnroll2 : kStdpRowsUnroll) * kWave * 8;
}
// the per-neuron summary it stages beside the queues (160 KB of LDS per workgroup)
constexpr int kCodeMax = 163840 - stdp_rows_queue_bytes(1) - 1024;  // bytes of history codes
// The row-wise STDP kernel runs one workgroup per CU, and the fused synapse
// pass (k_synapse_pass) fills the slots of every CU (one or two workgroups
// per CU, as the LDS of both parts allows): both grids come from the CU
// count of the device (hipDeviceAttributeMultiprocessorCount).
constexpr int fused_queue_bytes(int hw)
{
    return (kDlvBlock / kWave) * (hw == 2 ? kStdpRowsUnroll2 : kStdpRowsUnroll) * kWave * 8;
}
constexpr int kRecentMaxWords = kCodeMax / 8;  // words of the spike-recency bitmap
constexpr uint8_t kCodeMulti = 255;    // history code: two or more spikes in the window
int stdp_static_bytes();  // static LDS of the slice STDP kernel (-1 on error)
hipError_t launch_deliver_lds(hipStream_t s, const DeliverArgs &a, int blocks, size_t lds, KernelEvents ev = {});
// k_synapse_pass: slice delivery on workgroups [0, nd) (nd a multiple of 8),
// forced-row STDP on ns more, kDlvBlock threads each; lds covers both
hipError_t launch_synapse_pass(hipStream_t s, const DeliverArgs &d, const StdpArgs &a, int nd,
                               int ns, size_t lds, KernelEvents ev = {});
hipError_t launch_deliver_global(hipStream_t s, const DeliverArgs &a, int blocks, KernelEvents ev = {});
int deliver_lds_static_bytes();  // static LDS of the slice kernel (-1 on error)
int synapse_pass_static_bytes();  // static LDS of the fused synapse pass (-1 on error)
// the fp32 input from the partial sums when clk->input_forced is 0 (then
// set to 1 by a second kernel, so that every workgroup reads the flag first)
hipError_t launch_materialize_input(hipStream_t s, const long long *apart, int64_t part_stride,
                                    StepClock *clk, float *ain, int64_t count);
// clk->t = t unless t < 0, the input flags unless input_forced < 0
hipError_t launch_set_clock(hipStream_t s, StepClock *clk, int64_t t, int32_t input_forced,
                            int32_t n_parts);
hipError_t launch_scan_i64(hipStream_t s, int64_t *data, int64_t count, int64_t *bsum);
hipError_t launch_graph_count_bernoulli(hipStream_t s, const GraphArgs &a);
hipError_t launch_graph_fill_bernoulli(hipStream_t s, const GraphArgs &a);
hipError_t launch_graph_fill_fanout(hipStream_t s, const GraphArgs &a);
hipError_t launch_edges_count(hipStream_t s, const GraphArgs &a, const int32_t *src,
                              const int32_t *dst, int64_t e);
hipError_t launch_edges_scatter(hipStream_t s, const GraphArgs &a, const int32_t *src,
                                const int32_t *dst, const float *w, int64_t e,
                                int64_t *cursor);
hipError_t launch_row_maxlen(hipStream_t s, const GraphArgs &a);
hipError_t launch_row_sort(hipStream_t s, const GraphArgs &a, int pow2len);
hipError_t launch_pivots(hipStream_t s, const GraphArgs &a);
// col16 from col (snn_config.compressed_targets): slice-local indices
hipError_t launch_encode_targets(hipStream_t s, const GraphArgs &a, int64_t n_edges);

}  // namespace snn
