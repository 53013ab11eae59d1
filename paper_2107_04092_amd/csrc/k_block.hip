// gfx950 kernels of a block of steps of a plastic network with D >= 2 (see
// BlockArgs): the plan of the block's rows, the target groups' run of its
// steps, and the per-step lists rebuilt after the last block.
//
// Built with -ffp-contract=off: the neuron update reproduces a fixed fp32
// operation order.
#include "snn_neuron.h"

#include <algorithm>

namespace snn {
namespace {

// ---------------------------------------------------------------------------
// The plan of steps t0 .. t0+B-1 (t0 = clk->t), one thread per row k.
//
// Row k transmits at t when it spiked at t-D+1, which the history word holds
// when the block starts (bit b = step t0-1-b, so bit D-2-q for t = t0+q). A
// plastic row is brought up to date when it transmits, or, idle, once its
// last update is 64 hw steps old (forced), exactly as the step-by-step
// neuron update decides; each such event is a snapshot of the row at its
// step, taken from the t_last and x_pre that the row's earlier events in the
// block left. A row is forced at most once per block (64 hw > B steps apart)
// and only before its first transmission; a forced update that is the row's
// last event of the block goes to the deferred list (list B) instead of its
// step's. The steps are walked twice: once for the event flags (each list's
// count in the workgroup, which one atomic add per list turns into the
// workgroup's place in the list), then for the snapshots (PbEvent), written
// at their positions. A list is ascending inside each workgroup's share; the
// shares come in the order the workgroups arrive, and no result depends on
// the order (the run accumulates in exact fixed point and every synapse's
// update is its own).

__global__ __launch_bounds__(kPbPlanBlock) void k_block_plan(BlockArgs b)
{
    constexpr int NWV = kPbPlanBlock / kWave;
    __shared__ uint64_t s_m[kBatchMax][NWV];
    __shared__ int s_lb[kBatchMax];
    __shared__ int s_wp[kBatchMax][NWV];  // events of list q in the waves before
    __shared__ int s_rq[NWV][kWave];      // a wave's lanes with an event
    __shared__ float s_dpow[kMaxAge + 1];
    __shared__ unsigned long long s_st[kStFields];
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const int k = blockIdx.x * kPbPlanBlock + tid;
    const bool live = k < b.n;
    const bool plastic = k < b.n_plastic_rows;  // (n_plastic_rows <= n)
    const int B = b.steps, D = b.delay, hw = b.hw;
    // the row's values, then the clock: one round trip
    uint64_t h0 = 0ull;
    int64_t rs = 0;
    int tl0 = 0, pend_k = 0;
    float xp0 = 0.f;
    if (live) {
        h0 = b.hist[(int64_t)k * hw];
        rs = b.row_ptr[k];
    }
    if (plastic) {
        tl0 = b.t_last[k];
        xp0 = b.xpre[k];
        pend_k = b.pend[k];
    }
    const StepClock ck = load_clock(b.clk);
    const int64_t t0 = ck.t;
    if (blockIdx.x == 0 && tid == 0) {
        BlockClock bc{};
        bc.t0 = t0;
        bc.input_forced = ck.input_forced;
        bc.n_parts = ck.n_parts;
        *b.bclk = bc;
    }
    for (int q = tid; q <= kMaxAge; q += kPbPlanBlock) s_dpow[q] = b.dpow[q];
    if (tid < kStFields) s_st[tid] = 0ull;
    // the steps with an event, and the deferred one
    uint32_t evm = 0, fm = 0;
    {
        int tl = tl0;
        for (int q = 0; q < B; ++q) {  // uniform
            const int64_t t = t0 + q;
            const bool tx = live && ((h0 >> (D - 2 - q)) & 1ull);
            bool ev = tx;
            if (plastic) {
                if (tx) {
                    if (t - (int64_t)tl > 0) tl = (int)t;
                } else if (t - (int64_t)tl >= 64 * hw) {
                    ev = true;
                    fm |= 1u << q;
                    tl = (int)t;
                }
            }
            evm |= (uint32_t)ev << q;
        }
    }
    // (a forced update is the row's last event when no higher bit is set)
    const uint32_t dfm = fm != 0u && (evm >> (__ffs((int)fm))) == 0u ? fm : 0u;
    for (int q = 0; q <= B; ++q) {  // uniform
        const bool ev = q < B ? ((evm & ~dfm) >> q) & 1u : dfm != 0u;
        const uint64_t m = ballot64(ev);
        if (lane == 0) s_m[q][wave] = m;
    }
    __syncthreads();  // s_m, s_dpow, s_st
    // this workgroup's place in list tid; the other block's counts cleared
    // for the next plan (the launches that read them have ended)
    if (tid <= B) {
        int own = 0;
        for (int w = 0; w < NWV; ++w) {
            s_wp[tid][w] = own;
            own += __popcll(s_m[tid][w]);
        }
        s_lb[tid] = own ? atomicAdd(b.ev_cnt + tid, own) : 0;
    }
    if (blockIdx.x == 0 && tid < kBatchMax) b.ev_cnt_next[tid] = 0;
    __syncthreads();  // s_lb
    // the snapshots, at their positions (the workgroup's place in the list,
    // then earlier waves, then earlier lanes). A wave's rows with an event
    // are compacted first: a lane walks one such row's events in order (each
    // snapshot starts from the one before), with the wave's lanes busy.
    const uint64_t hm = ballot64(evm != 0u);
    if (evm != 0u) s_rq[wave][lane_rank(hm)] = lane;
    __builtin_amdgcn_wave_barrier();
    const int nq = (int)__popcll(hm);  // wave-uniform
    const int src = lane < nq ? s_rq[wave][lane] : lane;
    const int kr = blockIdx.x * kPbPlanBlock + wave * kWave + src;  // the lane's row
    const uint32_t r_evm = (uint32_t)__shfl((int)evm, src);
    const uint32_t r_dfm = (uint32_t)__shfl((int)dfm, src);
    const uint64_t r_h0 = (uint64_t)__shfl((long long)h0, src);
    const int64_t r_rs = (int64_t)__shfl((long long)rs, src);
    const int r_tl0 = __shfl(tl0, src), r_pend = __shfl(pend_k, src);
    const float r_xp0 = __shfl(xp0, src);
    const bool r_plastic = kr < b.n_plastic_rows;
    const uint64_t below = src == 0 ? 0ull : (~0ull >> (64 - src));
    int tl = r_tl0;
    float xp = r_xp0;
    long long n_rows = 0, n_forced = 0, n_syn = 0, n_fsyn = 0;
    for (uint32_t m = lane < nq ? r_evm : 0u; m; m &= m - 1u) {
        const int q = __ffs((int)m) - 1;
        const int64_t t = t0 + q;
        const int tx = (int)((r_h0 >> (D - 2 - q)) & 1ull);
        RowInfo ri = RowInfo{};
        int ok = 0;
        if (r_plastic) {
            ok = make_row_info_d(ri, kr, t, tl, r_rs, r_pend, xp, tx, hw,
                                 s_dpow[row_age_index(t, tl, hw)], b.err);
            if (ok) {
                tl = (int)t;
                xp = ri.xp_now;
                n_rows += 1;
                n_syn += ri.len;
                if (!tx) {
                    n_forced += 1;
                    n_fsyn += ri.len;
                }
            }
        }
        // nothing to bring up to date (ok == 0): the row is only delivered
        PbEvent pe;
        pe.rs = (int32_t)r_rs;
        pe.lenf = ok ? ((uint32_t)ri.len & 0xffffu) | ((uint32_t)(ri.age_pre & 0xff) << 16) |
                           ((uint32_t)((ri.age_pre >> 8) & 1) << 24)
                     : 0u;
        pe.lenf |= ((uint32_t)tx << 25) | ((uint32_t)(b.nacc == 2 && kr >= b.n_exc) << 26) |
                   ((uint32_t)q << 27);
        pe.xp0 = ok ? ri.xp0 : 0.f;
        pe.k = kr;
        const int lq = (r_dfm >> q) & 1u ? B : q;  // the list
        const int pos = s_lb[lq] + s_wp[lq][wave] + (int)__popcll(s_m[lq][wave] & below);
        // (the counts of a list never exceed n unless they did not start at 0)
        if (pos < b.n)
            b.ev[(int64_t)lq * b.n + pos] = pe;
        else
            atomicOr(b.err, kErrRing);
    }
    if (lane < nq && r_plastic && tl != r_tl0) {  // the row as its last event left it
        b.t_last[kr] = tl;
        b.xpre[kr] = xp;
    }
    n_rows = wave_sum_i64(n_rows);
    n_forced = wave_sum_i64(n_forced);
    n_syn = wave_sum_i64(n_syn);
    n_fsyn = wave_sum_i64(n_fsyn);
    if (lane == 0) {
        if (n_rows) atomicAdd(s_st + kStRows, (unsigned long long)n_rows);
        if (n_forced) atomicAdd(s_st + kStForced, (unsigned long long)n_forced);
        if (n_syn) atomicAdd(s_st + kStSyn, (unsigned long long)n_syn);
        if (n_fsyn) atomicAdd(s_st + kStForcedSyn, (unsigned long long)n_fsyn);
    }
    __syncthreads();  // s_st complete
    if (tid < kStFields && s_st[tid])
        add_stat(b.info_stats + (int64_t)(blockIdx.x % b.info_slots) * kStFields + tid,
                 (long long)s_st[tid]);
}

// ---------------------------------------------------------------------------
// The run of the block: workgroup of target group g (targets [g gw, g gw +
// gw), gw = gwidth, inside one slice), every step t = t0 + q:
//   (1) the neuron update of the group's targets (thread j: neuron g gw + j,
//       its state in registers from the first step to the last), with the
//       input of step t: the state's input at t0, afterwards the LDS
//       accumulator; the new history words and post traces go to LDS;
//   (2) the step's rows (the plan's list): for each, its entries with a
//       target in the group, staged as in slice delivery (prefix sums of
//       the lengths, a map from each flattened entry to its row), then
//       every entry: the plastic ones brought up to date from the target's
//       history in LDS (a forced row: only those; its other entries are not
//       read), and a transmitting row's entries added to the accumulator
//       (64-bit fixed point, LDS atomics), which step t+1's neuron update
//       reads.
// A synapse belongs to the group of its target, so each weight is read and
// written by one workgroup only, and the steps of a workgroup are ordered by
// its barriers.
//
// The workgroup first loads the records of all its rows of the block (row
// start plus the group's offset and length, plastic length, age, flags, pre
// trace) into LDS, so a step stages its rows without a round trip to
// memory. The steps are pipelined: the next step's rows are staged and
// mapped while this step's entries are computed, and once the step's last
// barrier has ordered its weight stores, the next step's entries (its
// first window) are loaded, one set of loads in flight at a time (a wave's
// loads complete in the order they were issued, and the loads a step waits
// for are always the oldest). Further windows and batches of a step are
// loaded when the step reaches them; a block with more records than LDS
// holds loads each step's records when it runs.
//
// At the end the state goes back, the accumulator becomes partial sum 0 (the
// input of step t0 + B), each target's history words at block start and its
// code for the deferred updates are written (see k_block_deferred), and
// workgroup 0 advances the step clock, which no workgroup of the run reads
// (they read the plan's copy).

constexpr int kPbDirect = 32;  // segments up to this long are mapped by their own thread
constexpr long long kMask40 = (1ll << 40) - 1;
// a record's flags: age (bits 0-7), pre spike (8), delivered (9), inhibitory (10)
// per loaded entry: record in the batch (bits 0-9), plastic (10), present
// (11), offset in the segment (12-25), edge index parity (26)
constexpr int kPkSeg = 0x3ff, kPkPlastic = 1 << 10, kPkIn = 1 << 11, kPkOff = 12;
constexpr int kPkOffMask = 0x3fff, kPkOdd = 26;
static_assert(kPbSegs <= kPkSeg + 1, "record index fits the entry word");
static_assert(kMaxSortRow <= kPkOffMask + 1, "segment offset fits the entry word");
// a queued update: record in the batch (bits 0-9), offset (10-23), target in the group (24-31)
static_assert(kPbMaxWidth <= 256, "target in the group fits the queue word");
// The graphs of the blocks (at most kPbMaxN rows of at most kMaxSortRow
// entries) have fewer than 2^31 edges: 32-bit edge indices.
static_assert((int64_t)kPbMaxN * kMaxSortRow < (1ll << 31), "32-bit edge index");

struct PbEntries {
    float wv[kPbUnroll];     // weight as loaded
    uint32_t cv[kPbUnroll];  // target as loaded (compressed: the 32-bit word holding it)
    int pk[kPbUnroll];
};

template <int HW, bool CT>
__global__ __launch_bounds__(kPbBlock) void k_block_run(NeuronArgs a, BlockArgs b)
{
    constexpr int NWV = kPbBlock / kWave;
    constexpr int QH = 4;  // entry slots between queue flushes
    __shared__ int r_start[kPbRecords];   // first entry of the row in the group (edge index)
    __shared__ int r_lens[kPbRecords];    // entries (bits 0-15), plastic entries (16-31)
    __shared__ int r_info[kPbRecords];
    __shared__ float r_xp0[kPbRecords];
    __shared__ int s_off[2][kPbSegs + 1];
    __shared__ uint16_t s_map[2][kPbWindow];  // entry -> 1 + record in the batch
    __shared__ long long s_tot[2];            // entries (bits 0-39), long segments (40+)
    __shared__ float q_w[NWV][QH * kWave];
    __shared__ int q_p[NWV][QH * kWave];
    __shared__ uint64_t s_hist[kPbMaxWidth * HW];
    __shared__ float s_y[kPbMaxWidth];
    __shared__ long long s_acc[2 * kPbMaxWidth];
    __shared__ float s_dpow[kMaxAge + 1];
    __shared__ long long sh[NWV];
    __shared__ int shi[NWV];
    __shared__ int s_cnt[kBatchMax], s_base[kBatchMax + 1];
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    // neighbouring groups (which read neighbouring entries of each row) on
    // one XCD: workgroup b runs on XCD b mod 8
    const int nb = gridDim.x;  // multiple of 8
    const int g = (blockIdx.x & 7) * (nb >> 3) + (blockIdx.x >> 3);
    if (g >= b.n_groups) return;  // whole workgroup, before any barrier
    const int n = a.n, G = b.n_groups;
    const int glo = g * b.gwidth;
    const int wn = min(b.gwidth, n - glo);  // > 0
    const int cbase = CT ? glo % b.width : glo;  // subtracted from a loaded target
    const int i = glo + tid;
    const bool live = tid < wn;
    const int B = b.steps;
    const long long ne = (long long)b.n_edges;
    // the neuron state and the input of the first step (both in flight
    // while the block clock is read)
    NState st = {};
    float ae0 = 0.f, ai0 = 0.f;
    const BlockClock bc = *b.bclk;
    const int64_t t0 = bc.t0;
    if (live) {
        InputLoads in0;
        nstate_load<-1, HW>(a, i, st);
        if (a.model != 2) {
            input_issue(a, i, in0);
            input_combine(a, in0, bc.input_forced, bc.n_parts, i, ae0, ai0);
        }
    }
    if (tid < kBatchMax) s_cnt[tid] = tid < B ? min(max(b.ev_cnt[tid], 0), n) : 0;
    for (int q = tid; q <= kMaxAge; q += kPbBlock) s_dpow[q] = b.dpow[q];
    __syncthreads();  // s_cnt
    if (tid == 0) {
        int acc = 0;
        for (int q = 0; q < kBatchMax; ++q) {
            s_base[q] = acc;
            acc += s_cnt[q];
        }
        s_base[kBatchMax] = acc;
    }
    const float c_pot = b.c_pot, c_dep = b.c_dep, mu = b.mu;
    const int32_t *__restrict__ col = b.col;
    const uint32_t *__restrict__ col32 = reinterpret_cast<const uint32_t *>(b.col16);
    float *__restrict__ wgt = b.w;
    long long events = 0, w_tx = 0, w_forced = 0, spikes = 0;
    uint32_t blk = 0u;  // the block's spikes (bit 0: the latest step)
    __syncthreads();  // s_base

    // LDS records r0 .. r0 + count - 1 from the lists from entry j0 of step
    // q0 on (across the steps' lists in order): the row's start plus the
    // group's offset and length (the group pivots of the row, loaded once
    // the row is known), clamped to the graph (only a failed plan scan,
    // which leaves list entries unwritten, could point elsewhere)
    auto load_records = [&](int q0, int j0, int r0, int count) {
        constexpr int RU = kPbRecords / kPbBlock;  // all records of LDS in one round
        static_assert(kPbRecords % kPbBlock == 0, "whole rounds of records");
        for (int x0 = 0; x0 < count; x0 += RU * kPbBlock) {
            PbEvent pe[RU];
#pragma unroll
            for (int u = 0; u < RU; ++u) {
                const int x = min(x0 + u * kPbBlock + tid, max(count - 1, 0));
                // (the step of flattened entry x: at most kBatchMax lists)
                int q = q0, j = j0 + x;
                while (q < B - 1 && j >= s_cnt[q]) {
                    j -= s_cnt[q];
                    ++q;
                }
                j = min(j, max(s_cnt[q] - 1, 0));
                pe[u] = b.ev[(int64_t)q * n + j];
            }
            int p0[RU], p1[RU];
#pragma unroll
            for (int u = 0; u < RU; ++u) {
                const int32_t *gp = b.gpiv + (int64_t)min(max(pe[u].k, 0), n - 1) * (G + 1) + g;
                p0[u] = gp[0];
                p1[u] = gp[1];
            }
#pragma unroll
            for (int u = 0; u < RU; ++u) {
                const int x = x0 + u * kPbBlock + tid;
                if (x >= count) continue;
                int sl = max(p1[u] - p0[u], 0);
                const uint32_t f = pe[u].lenf;
                const int plen = min(max((int)(f & 0xffffu) - p0[u], 0), sl);
                const int deliver = (f >> 25) & 1;
                if (!deliver) sl = plen;  // a forced row: its plastic entries only
                const long long st0 = min(max((long long)pe[u].rs + p0[u], 0ll), ne);
                sl = (int)min((long long)sl, ne - st0);
                r_start[r0 + x] = (int)st0;
                r_lens[r0 + x] = sl | (min(plen, sl) << 16);
                r_info[r0 + x] = (int)((f >> 16) & 0xff) | (int)(((f >> 24) & 1) << 8) |
                                 (deliver << 9) | (int)(((f >> 26) & 1) << 10);
                r_xp0[r0 + x] = pe[u].xp0;
            }
        }
    };
    // a batch of nbt records from LDS record rb on, into staging buffer x:
    // offsets scanned, the map of its first window; ends with a barrier
    auto build_map = [&](int x, int nbt, int w0, int we, bool direct) {
        if (direct) {  // short segments: each thread writes its own segments' entries
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                const int j = 2 * tid + r;
                if (j < nbt) {
                    const int a0 = max(s_off[x][j], w0), a1 = min(s_off[x][j + 1], w0 + we);
                    for (int y = a0; y < a1; ++y) s_map[x][y - w0] = (uint16_t)(j + 1);
                }
            }
            __syncthreads();
        } else {  // mark each segment's first entry in the window, then max-scan
            for (int y = tid; y < we; y += kPbBlock) s_map[x][y] = 0;
            __syncthreads();
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                const int j = 2 * tid + r;
                if (j < nbt) {
                    const int a0 = max(s_off[x][j], w0), a1 = min(s_off[x][j + 1], w0 + we);
                    if (a0 < a1) s_map[x][a0 - w0] = (uint16_t)(j + 1);
                }
            }
            __syncthreads();
            fill_segment_map<kPbBlock, kPbUnroll, uint16_t>(s_map[x], we, shi, 0);
        }
    };
    auto prep = [&](int x, int rb, int nbt) {
        int len[2];
        long long packed = 0;
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int j = 2 * tid + r;
            len[r] = j < nbt ? (r_lens[rb + j] & 0xffff) : 0;
            packed += (long long)len[r] | ((long long)(len[r] > kPbDirect) << 40);
        }
        const long long incl = block_incl_scan_i64_n<kPbBlock>(packed, sh);
        long long ex = (incl - packed) & kMask40;
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            s_off[x][2 * tid + r] = (int)ex;
            ex += len[r];
        }
        if (tid == kPbBlock - 1) {
            s_off[x][kPbSegs] = (int)(incl & kMask40);
            s_tot[x] = incl;
        }
        __syncthreads();
        const long long tq = s_tot[x];
        const int total = (int)(tq & kMask40);
        if (total > 0) build_map(x, nbt, 0, min(total, kPbWindow), (tq >> 40) == 0);
    };
    // loads of window [w0, w0 + we) of staging buffer x (records from rb):
    // every slot loads from a valid address, the results are looked at when
    // the entries are computed
    auto issue = [&](int x, int rb, int w0, int we, PbEntries &E) {
#pragma unroll
        for (int u = 0; u < kPbUnroll; ++u) {
            const int y = u * kPbBlock + tid;
            const bool in = y < we;
            // a slot no lane of the wave uses loads nothing (wave-uniform)
            if (u * kPbBlock + wave * kWave >= we) {
                E.pk[u] = 0;
                continue;
            }
            const int l = in ? (int)s_map[x][y] - 1 : 0;
            const int off = w0 + y - s_off[x][l];
            const int r = rb + l;
            const int e = in ? r_start[r] + off : 0;  // < n_edges
            E.cv[u] = CT ? col32[e >> 1] : (uint32_t)col[e];
            E.wv[u] = wgt[e];
            E.pk[u] = in ? l | (off < (r_lens[r] >> 16) ? kPkPlastic : 0) | kPkIn |
                               (off << kPkOff) | ((e & 1) << kPkOdd)
                         : 0;
        }
    };
    // The entries of one window: a transmitting row's entry whose weight
    // does not change is delivered at once; the entries whose weight
    // changes (a pre spike, or a post spike of the target within the row's
    // window) go to the wave's queue, which is then updated 64 at a time
    // with every lane busy (the replay loops run over those entries only),
    // stored, and delivered where the row transmits.
    auto compute = [&](int rb, const PbEntries &E) {
        float *qw = q_w[wave];
        int *qp = q_p[wave];
#pragma unroll
        for (int hf = 0; hf < kPbUnroll / QH; ++hf) {
            int qn = 0;
#pragma unroll
            for (int v = 0; v < QH; ++v) {
                const int u = hf * QH + v;
                const int pk = E.pk[u];
                if (!ballot64(pk & kPkIn)) continue;  // an unused slot of the wave
                const int l = pk & kPkSeg;
                const int info = (pk & kPkIn) ? r_info[rb + l] : 0;
                const uint32_t c = CT ? (((pk >> kPkOdd) & 1) ? E.cv[u] >> 16 : E.cv[u] & 0xffffu)
                                      : E.cv[u];
                const int j = (int)c - cbase;
                const bool ok = (pk & kPkIn) && (unsigned)j < (unsigned)wn;
                if ((pk & kPkIn) && !ok) atomicOr(b.err, kErrIndex);  // not this group's target
                bool cand = false;
                if (ok && (pk & kPkPlastic)) {
                    uint64_t m0, m1;
                    window_masks(info & 0xff, m0, m1);
                    const uint64_t h0 = s_hist[j * HW] & m0;
                    const uint64_t h1 = HW == 2 ? s_hist[j * 2 + 1] & m1 : 0ull;
                    cand = h0 || h1 || ((info >> 8) & 1) || !b.event;
                }
                if (ok && !cand && ((info >> 9) & 1)) {
                    atomicAdd((unsigned long long *)(s_acc + j +
                                                     (((info >> 10) & 1) ? kPbMaxWidth : 0)),
                              (unsigned long long)to_fix(E.wv[u]));
                    ++events;
                }
                const uint64_t bl = ballot64(cand);
                if (cand) {
                    const int e = qn + lane_rank(bl);
                    qw[e] = E.wv[u];
                    qp[e] = l | (((pk >> kPkOff) & kPkOffMask) << 10) | (j << 24);
                }
                qn += (int)__popcll(bl);
            }
            __builtin_amdgcn_wave_barrier();
            for (int e0 = 0; e0 < qn; e0 += kWave) {  // wave-uniform
                const int e = e0 + lane;
                if (e >= qn) continue;
                float w = qw[e];
                const unsigned p = (unsigned)qp[e];
                const int r = rb + (int)(p & kPkSeg);
                const int off = (int)((p >> 10) & kPkOffMask), j = (int)(p >> 24);
                const int info = r_info[r];
                const int age = info & 0xff, pre = (info >> 8) & 1;
                uint64_t m0, m1;
                window_masks(age, m0, m1);
                const uint64_t h0 = s_hist[j * HW] & m0;
                const uint64_t h1 = HW == 2 ? s_hist[j * 2 + 1] & m1 : 0ull;
                const float y = pre ? s_y[j] : 0.f;
                const float xp0 = r_xp0[r];
                // the pre trace after this update, as the plan's snapshot has it
                const float xpn = __fadd_rn(__fmul_rn(xp0, s_dpow[age]), (float)pre);
                w = b.event ? stdp_synapse(w, h0, h1, age, pre, xp0, xpn, y, s_dpow, c_pot, c_dep, mu)
                            : stdp_synapse_steps(w, h0, h1, age, pre, xp0, xpn, y, s_dpow[1],
                                                 c_pot, c_dep, mu);
                wgt[r_start[r] + off] = w;
                if (pre)
                    ++w_tx;
                else
                    ++w_forced;
                if ((info >> 9) & 1) {
                    atomicAdd((unsigned long long *)(s_acc + j +
                                                     (((info >> 10) & 1) ? kPbMaxWidth : 0)),
                              (unsigned long long)to_fix(w));
                    ++events;
                }
            }
            __builtin_amdgcn_wave_barrier();  // the queue is rewritten next
        }
    };
    // the windows of a staged batch from window w_from on (each mapped,
    // loaded and computed in turn)
    auto windows = [&](int x, int rb, int nbt, int w_from, PbEntries &E) {
        const long long tq = s_tot[x];
        const int total = (int)(tq & kMask40);
        for (int w0 = w_from; w0 < total; w0 += kPbWindow) {
            const int we = min(kPbWindow, total - w0);
            if (w0 > 0) {
                __syncthreads();  // every read of the map of the window before
                build_map(x, nbt, w0, we, (tq >> 40) == 0);
            }
            issue(x, rb, w0, we, E);
            compute(rb, E);
        }
    };
    auto neuron_step = [&](int q) {
        const int64_t t = t0 + q;
        if (live) {
            float ae = 0.f, ai = 0.f;
            if (a.model != 2) {
                if (q == 0) {
                    ae = ae0;
                    ai = ai0;
                } else {
                    ae = from_fix(s_acc[tid]);
                    if (b.nacc == 2) ai = from_fix(s_acc[kPbMaxWidth + tid]);
                }
            }
            const int sp = neuron_advance<-1, HW>(a, i, t, ae, ai, st);
            spikes += sp;
            blk = (blk << 1) | (uint32_t)sp;
            s_hist[tid * HW] = st.h0;
            if (HW == 2) s_hist[tid * 2 + 1] = st.h1;
            s_y[tid] = st.y;
        }
        if (tid < kPbMaxWidth) {
            s_acc[tid] = 0;
            s_acc[kPbMaxWidth + tid] = 0;
        }
    };

    const uint64_t hs0 = st.h0, hs1 = st.h1;  // the history words at block start
    PbEntries E;
    const int total_rec = s_base[kBatchMax];
    if (total_rec <= kPbRecords) {
        // every record of the block in LDS; step 0 staged and its first
        // window loaded
        load_records(0, 0, 0, total_rec);
        __syncthreads();
        const int nb0 = min(s_cnt[0], kPbSegs);
        prep(0, s_base[0], nb0);
        issue(0, s_base[0], 0, min((int)(s_tot[0] & kMask40), kPbWindow), E);
        for (int q = 0; q < B; ++q) {
            const int x = q & 1;
            neuron_step(q);
            // (2a) the next step's first batch staged and its first window
            // mapped (the staging's barriers publish the neuron update)
            if (q + 1 < B)
                prep(x ^ 1, s_base[q + 1], min(s_cnt[q + 1], kPbSegs));
            else
                __syncthreads();  // the neuron update's histories and traces
            // (2b) this step's entries: the loaded first window, the rest
            const int nb1 = min(s_cnt[q], kPbSegs);
            compute(s_base[q], E);
            windows(x, s_base[q], nb1, kPbWindow, E);
            for (int e0 = kPbSegs; e0 < s_cnt[q]; e0 += kPbSegs) {  // further batches
                __syncthreads();  // every read of the staging of the batch before
                const int nbt = min(kPbSegs, s_cnt[q] - e0);
                prep(x, s_base[q] + e0, nbt);
                windows(x, s_base[q] + e0, nbt, 0, E);
            }
            __syncthreads();  // every atomic and weight store of step q done
            // (3) the next step's first window loaded
            if (q + 1 < B) issue(x ^ 1, s_base[q + 1], 0,
                                 min((int)(s_tot[x ^ 1] & kMask40), kPbWindow), E);
        }
    } else {
        // more records than LDS holds: each batch of each step's records is
        // loaded when the step reaches it
        for (int q = 0; q < B; ++q) {
            neuron_step(q);
            for (int e0 = 0; e0 < s_cnt[q]; e0 += kPbSegs) {
                __syncthreads();  // every read of the records and staging before
                const int nbt = min(kPbSegs, s_cnt[q] - e0);
                load_records(q, e0, 0, nbt);
                __syncthreads();
                prep(0, 0, nbt);
                windows(0, 0, nbt, 0, E);
            }
            __syncthreads();  // every atomic of step q done (and the neuron update published)
        }
    }
    if (live) {
        nstate_store<-1, HW>(a, i, st);
        a.code[i] = hist_code(st.h0, st.h1);
        b.apart[i] = s_acc[tid];
        if (b.nacc == 2) b.apart[n + i] = s_acc[kPbMaxWidth + tid];
        uint64_t *hqi = b.hq + (int64_t)i * (2 * HW);
        hqi[0] = hs0;
        if (HW == 2) hqi[1] = hs1;
        hqi[HW] = blk;
        // the code of the deferred updates: the first step of the block with
        // a spike (15: none), and the bit L of the latest spike before it
        // against the window of a forced update at step q (L + q + 1 < 64 hw,
        // q < 15): 0 if always inside, 15 if never, else L - (64 hw - 16)
        const int first = blk ? B - 1 - (31 - __clz((int)blk)) : 15;
        const int last = hs0 ? __ffsll((long long)hs0) - 1
                             : (HW == 2 && hs1) ? 63 + __ffsll((long long)hs1) : 1 << 20;
        const int lc = last <= 64 * HW - 16 ? 0 : last >= 64 * HW - 1 ? 15 : last - (64 * HW - 16);
        b.dcode[i] = (uint8_t)(first | (lc << 4));
    }
    events = block_sum_i64_n<kPbBlock>(events, sh);
    w_tx = block_sum_i64_n<kPbBlock>(w_tx, sh);
    w_forced = block_sum_i64_n<kPbBlock>(w_forced, sh);
    spikes = block_sum_i64_n<kPbBlock>(spikes, sh);
    if (tid == 0) {
        int64_t *ds = b.dlv_stats + 2 * (int64_t)(g % b.dlv_slots);
        if (events) add_stat(ds, events);
        if (w_tx) add_stat(ds + 1, w_tx);
        if (w_forced) add_stat(b.syn_stats + (g % b.syn_slots), w_forced);
        if (spikes) add_stat(b.gstats + kGSpikes, spikes);
        if (g == 0) {
            add_stat(b.gstats + kGSteps, B);
            b.clk->t = t0 + B;
            b.clk->input_forced = 0;  // the next input is partial sum 0
            b.clk->n_parts = 1;
        }
    }
}

// ---------------------------------------------------------------------------
// The deferred forced updates of a block (the plan's list B), after its run,
// streamed by the whole device: one workgroup per CU, the rows' plastic
// entries (from each row's first 8-aligned entry on) cut into parts of
// kDfPart, spread over the waves (each lane 8 consecutive targets and
// weights in 16-byte loads), the next part loaded while the current one is
// computed.
//   An update at step t = t0 + q changes the synapses whose target spiked in
// the window (t - a, t] (every one without event-driven replay). The
// target's history word at t is its word at block start shifted up by q + 1
// steps, under the block's spike bits of steps t0 .. t (Sec. III-A's bit
// history). A forced update has the longest age, a = 64 hw (> q), so a
// synapse changes iff its target spiked in the block at a step <= q, or
// before the block at bit L of the start words with L + q + 1 < a: one byte
// per target holds both (the first spike step in the block; L against the
// last 15 bits of the window), staged in LDS. The synapses that pass are
// queued and brought up to date 64 at a time from the full words (hq), which
// decide exactly (an update of another age queues every entry).

constexpr int kDfBlock = 1024;
constexpr int kDfPart = kPbDfPart;      // entries per part of a row
constexpr int kDfU = kDfPart / kWave;   // entries per lane per part
static_assert(kDfU == 8, "two 16-byte loads of targets and of weights per lane");
static_assert(kPbMaxN <= 65536, "target in 16 bits of the queue word");

struct DfPart {
    int4 c[2];
    float4 w[2];
    long long base, lo, hi;  // first entry of the part (8-aligned), the row's plastic entries
    int age, qs;
    float xp0;
    int valid;
};

template <int HW>
__global__ __launch_bounds__(kDfBlock) void k_block_deferred(BlockArgs b)
{
    constexpr int NWV = kDfBlock / kWave;
    constexpr int A = 64 * HW;  // the age of a forced update
    __shared__ uint8_t s_code[kPbMaxN];
    __shared__ int q_p[NWV][kDfPart];    // target (bits 0-15), entry in the part (16-24)
    __shared__ float q_w[NWV][kDfPart];  // weight
    __shared__ float s_dpow[kMaxAge + 1];
    __shared__ long long sh[NWV];
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    const int n = b.n, B = b.steps;
    const int nd = min(max(b.ev_cnt[B], 0), n);
    const PbEvent *__restrict__ evd = b.ev + (int64_t)B * n;
    const int32_t *__restrict__ col = b.col;
    float *__restrict__ wgt = b.w;
    const uint64_t *__restrict__ hq = b.hq;
    const long long ne = (long long)b.n_edges;  // < 2^31
    const float c_pot = b.c_pot, c_dep = b.c_dep, mu = b.mu;
    // the targets' codes (padded to 16 bytes), loaded first: every later
    // load of the wave completes after them
    constexpr int kCodeLoads = kPbMaxN / 16 / kDfBlock;
    uint4 cl[kCodeLoads];
    const int ncv = (n + 15) / 16;
#pragma unroll
    for (int u = 0; u < kCodeLoads; ++u)
        cl[u] = reinterpret_cast<const uint4 *>(b.dcode)[min(u * kDfBlock + tid, ncv - 1)];
    // Items: part p of row r is item r P + p (P = parts of the longest
    // row); the wave takes items w0 + j stride, j = 0 .. nit - 1. Lane l
    // holds the record of the row of item (j & ~63) + l, read out for the
    // current item j (no load inside the part stream waits on a record).
    const int P = b.df_parts;
    const int stride = gridDim.x * NWV;
    const int w0 = blockIdx.x * NWV + wave;
    const long long nitems = (long long)nd * P;
    const int nit = w0 < nitems ? (int)((nitems - 1 - w0) / stride + 1) : 0;
    PbEvent le = PbEvent{};
    int j = 0;
    long long base = 0, r_lo = 0, r_hi = 0;  // the current item's part, its row's entries
    int r_age = 0, r_qs = 0;
    float r_xp0 = 0.f;
    auto set_item = [&]() {  // j < nit
        if ((j & 63) == 0) {
            const long long it = w0 + (long long)(j + lane) * stride;
            le = j + lane < nit ? evd[it / P] : PbEvent{};
        }
        const int src = j & 63;
        const long long rs = __builtin_amdgcn_readlane(le.rs, src);
        const uint32_t f = (uint32_t)__builtin_amdgcn_readlane((int)le.lenf, src);
        r_xp0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(le.xp0), src));
        r_lo = min(max(rs, 0ll), ne);
        r_hi = min(r_lo + (long long)(f & 0xffffu), ne);
        base = (r_lo & ~7ll) + (long long)((w0 + (long long)j * stride) % P) * kDfPart;
        r_age = min((int)((f >> 16) & 0xff), kMaxAge);
        r_qs = (int)((f >> 27) & 15);
    };
    if (nit > 0) set_item();
    // the next part's loads, from a valid address whether or not the part
    // exists, so that every part issues the same loads
    auto issue = [&](DfPart &p) {
        p.valid = j < nit && base < r_hi;
        p.base = base;
        p.lo = r_lo;
        p.hi = r_hi;
        p.age = r_age;
        p.qs = r_qs;
        p.xp0 = r_xp0;
        // (entries up to 7 past the last edge lie in the next array of the
        // graph buffer; they are never used)
        const long long e0 = p.valid ? min(base + lane * kDfU, (r_hi - 1) & ~7ll) : 0ll;
        const int4 *cv = reinterpret_cast<const int4 *>(col + e0);
        const float4 *wv = reinterpret_cast<const float4 *>(wgt + e0);
        p.c[0] = cv[0];
        p.c[1] = cv[1];
        p.w[0] = wv[0];
        p.w[1] = wv[1];
        if (j < nit && ++j < nit) set_item();  // wave-uniform
    };
    DfPart P0, P1;
    issue(P0);
    issue(P1);
#pragma unroll
    for (int u = 0; u < kCodeLoads; ++u)
        if (u * kDfBlock + tid < ncv) reinterpret_cast<uint4 *>(s_code)[u * kDfBlock + tid] = cl[u];
    for (int x = tid; x <= kMaxAge; x += kDfBlock) s_dpow[x] = b.dpow[x];
    __syncthreads();
    long long written = 0;
    // The history words of the first kDfRounds rounds of the queue are
    // gathered before the next part's loads are issued (a wave's loads
    // complete in order: waiting for a later gather waits for every earlier
    // load), so that part loads while this one is brought up to date.
    constexpr int kDfRounds = 2;
    auto words_of = [&](int j, uint64_t &s0, uint64_t &s1, uint64_t &blk) {
        const uint4 *hj = reinterpret_cast<const uint4 *>(hq + (int64_t)j * (2 * HW));
        const uint4 v0 = hj[0];
        if (HW == 2) {
            const uint4 v1 = hj[1];
            s1 = (uint64_t)v0.z | ((uint64_t)v0.w << 32);
            blk = (uint64_t)v1.x | ((uint64_t)v1.y << 32);
        } else {
            s1 = 0ull;
            blk = (uint64_t)v0.z | ((uint64_t)v0.w << 32);
        }
        s0 = (uint64_t)v0.x | ((uint64_t)v0.y << 32);
    };
    // a part, then the next part's loads into p
    auto step = [&](DfPart &p) {
        if (!p.valid) {  // wave-uniform
            issue(p);
            return;
        }
        const int age = p.age, qs = min(p.qs, B - 1);
        const long long pbase = p.base;
        const float xp0 = p.xp0;
        const bool filt = b.event && age == A;  // the codes decide
        const int cj[kDfU] = {p.c[0].x, p.c[0].y, p.c[0].z, p.c[0].w,
                              p.c[1].x, p.c[1].y, p.c[1].z, p.c[1].w};
        const float wj[kDfU] = {p.w[0].x, p.w[0].y, p.w[0].z, p.w[0].w,
                                p.w[1].x, p.w[1].y, p.w[1].z, p.w[1].w};
        const long long e0 = pbase + lane * kDfU;
        bool cand[kDfU];
#pragma unroll
        for (int v = 0; v < kDfU; ++v) {
            const long long e = e0 + v;
            const bool in = e >= p.lo && e < p.hi;
            const bool okj = (unsigned)cj[v] < (unsigned)n;
            if (in && !okj) atomicOr(b.err, kErrIndex);
            const int c = s_code[okj ? cj[v] : 0];
            cand[v] = in && okj && (!filt || (c & 15) <= qs || (c >> 4) + qs < 15);
        }
        int *qp = q_p[wave];
        float *qw = q_w[wave];
        int qn = 0;
#pragma unroll
        for (int v = 0; v < kDfU; ++v) {
            const uint64_t bl = ballot64(cand[v]);
            if (cand[v]) {
                const int x = qn + lane_rank(bl);
                qp[x] = cj[v] | ((lane * kDfU + v) << 16);
                qw[x] = wj[v];
            }
            qn += (int)__popcll(bl);
        }
        __builtin_amdgcn_wave_barrier();
        uint64_t g0[kDfRounds], g1[kDfRounds], gb[kDfRounds];
        int gp[kDfRounds];
#pragma unroll
        for (int r = 0; r < kDfRounds; ++r) {  // every lane, clamped into the queue
            const int x = min(r * kWave + lane, max(qn - 1, 0));
            gp[r] = qn > 0 ? qp[x] : 0;
            words_of(gp[r] & 0xffff, g0[r], g1[r], gb[r]);
        }
        issue(p);
        uint64_t m0, m1;
        window_masks(age, m0, m1);
        const int sft = B - 1 - qs;
        const float xpn = __fadd_rn(__fmul_rn(xp0, s_dpow[age]), 0.f);  // no pre spike
        auto update = [&](int x, int pk, uint64_t s0, uint64_t s1, uint64_t blk) {
            const uint64_t h0 = ((s0 << (qs + 1)) | (blk >> sft)) & m0;
            const uint64_t h1 = HW == 2 ? ((s1 << (qs + 1)) | (s0 >> (63 - qs))) & m1 : 0ull;
            if (b.event && !(h0 | h1)) return;  // unchanged
            float w = qw[x];
            w = b.event ? stdp_synapse(w, h0, h1, age, 0, xp0, xpn, 0.f, s_dpow, c_pot, c_dep, mu)
                        : stdp_synapse_steps(w, h0, h1, age, 0, xp0, xpn, 0.f, s_dpow[1], c_pot,
                                             c_dep, mu);
            wgt[pbase + (pk >> 16)] = w;
            ++written;
        };
#pragma unroll
        for (int r = 0; r < kDfRounds; ++r) {
            const int x = r * kWave + lane;
            if (x < qn) update(x, gp[r], g0[r], g1[r], gb[r]);
        }
        for (int x0 = kDfRounds * kWave; x0 < qn; x0 += kWave) {  // wave-uniform; rare
            const int x = x0 + lane;
            if (x >= qn) continue;
            const int pk = qp[x];
            uint64_t s0, s1, blk;
            words_of(pk & 0xffff, s0, s1, blk);
            update(x, pk, s0, s1, blk);
        }
        __builtin_amdgcn_wave_barrier();  // the queue is rewritten next
    };
    while (P0.valid || P1.valid || j < nit) {  // wave-uniform
        step(P0);
        step(P1);
    }
    written = block_sum_i64_n<kDfBlock>(written, sh);
    if (tid == 0 && written) add_stat(b.syn_stats + (blockIdx.x % b.syn_slots), written);
}

// ---------------------------------------------------------------------------
// After the last block of a call, what the step-by-step path keeps per step,
// rebuilt from the histories (the run writes none of it): workgroup q < D,
// the spike list of step t-1-q (bit q of history word 0; t = clk->t) in
// ascending order into its ring slot, with its count and each neuron's
// position; workgroup D, the spike, transmit and recency masks of step t-1
// and its forced rows (plastic, brought up to date at t-1 without
// transmitting), ascending. Every workgroup clears a share of the list
// scans' status words, so that no stale step tag matches a later scan.

constexpr int kPbFinishBlock = 1024;

__global__ __launch_bounds__(kPbFinishBlock) void k_block_finish(BlockArgs b)
{
    constexpr int NWV = kPbFinishBlock / kWave;
    __shared__ int s_cnt[NWV];
    __shared__ int s_base;
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const int q = blockIdx.x;
    const int n = b.n, hw = b.hw, D = b.delay;
    const int64_t t = load_clock(b.clk).t;
    for (int64_t x = (int64_t)q * kPbFinishBlock + tid; x < b.status_words;
         x += (int64_t)gridDim.x * kPbFinishBlock)
        b.status[x] = 0ull;
    if (q == 0 && tid < kBatchMax) {  // both blocks' list counts, for the next call's plans
        b.ev_cnt[tid] = 0;
        b.ev_cnt_next[tid] = 0;
    }
    if (tid == 0) s_base = 0;
    const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
    const bool lists = q < D;
    const int slot = ring_slot(t - 1 - q, D);
    int32_t *list = lists ? b.ring + (int64_t)slot * n : b.rows;
    int32_t *pos = b.spk_pos + (int64_t)slot * n;  // (lists only)
    for (int i0 = 0; i0 < n; i0 += kPbFinishBlock) {  // uniform
        const int i = i0 + tid;
        bool s = false;
        if (lists) {
            s = i < n && ((b.hist[(int64_t)i * hw] >> q) & 1ull);
        } else {
            uint64_t h0 = 0ull, h1 = 0ull;
            if (i < n) {
                h0 = b.hist[(int64_t)i * hw];
                if (hw == 2) h1 = b.hist[(int64_t)i * hw + 1];
            }
            const bool tx = (h0 >> (D - 1)) & 1ull;
            s = i < b.n_plastic_rows && !tx && (int64_t)b.t_last[i] == t - 1;
            const uint64_t m = ballot64(i < n && (h0 & 1ull));
            const uint64_t txm = ballot64(i < n && tx);
            const uint64_t rcm = ballot64(i < n && (h0 | h1) != 0ull);
            const int64_t word = (int64_t)(i0 / kWave) + wave;
            if (lane == 0 && word * kWave < n) {
                b.mask[word] = m;
                b.txmask[word] = txm;
                b.recent[word] = rcm;
            }
        }
        const uint64_t m = ballot64(s);
        if (lane == 0) s_cnt[wave] = __popcll(m);
        __syncthreads();  // s_cnt, and s_base of the previous round
        int p = s_base, tot = 0;
        for (int w = 0; w < NWV; ++w) {
            if (w < wave) p += s_cnt[w];
            tot += s_cnt[w];
        }
        if (s) {
            const int r = p + __popcll(m & below);
            list[r] = i;
            if (lists) pos[i] = r;
        }
        __syncthreads();  // every read of s_cnt and s_base
        if (tid == 0) s_base = p + tot;  // (thread 0: p is the round's base)
    }
    __syncthreads();
    if (tid == 0) {
        if (lists)
            b.ring_cnt[slot] = s_base;
        else
            *b.row_cnt = s_base;
    }
}

template <int HW, bool CT>
hipError_t launch_run(hipStream_t s, const NeuronArgs &a, const BlockArgs &b)
{
    const int grid = (b.n_groups + 7) / 8 * 8;
    hipLaunchKernelGGL((k_block_run<HW, CT>), dim3(grid), dim3(kPbBlock), 0, s, a, b);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_block_plan(hipStream_t s, const BlockArgs &b)
{
    if (b.steps < 1 || b.steps > kPbMaxSteps || b.steps > b.delay - 1 || b.n < 1 ||
        b.n > kPbMaxN || b.ev_cnt == b.ev_cnt_next)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_block_plan, dim3(blocks_for(b.n, kPbPlanBlock)), dim3(kPbPlanBlock), 0,
                       s, b);
    return hipGetLastError();
}

hipError_t launch_block_run(hipStream_t s, const NeuronArgs &a, const BlockArgs &b)
{
    if (b.steps < 1 || b.steps > kPbMaxSteps || b.gwidth < 1 || b.gwidth > kPbMaxWidth ||
        b.n_edges < 1 || b.n_edges > INT32_MAX ||
        b.width % b.gwidth != 0 || (int64_t)b.n_groups * b.gwidth < a.n ||
        (int64_t)(b.n_groups - 1) * b.gwidth >= a.n || a.n != b.n || b.nacc < 1 || b.nacc > 2 ||
        b.dlv_slots < 1 || b.syn_slots < 1)
        return hipErrorInvalidValue;
    const bool ct = b.col16 != nullptr;
    if (a.hw == 2) return ct ? launch_run<2, true>(s, a, b) : launch_run<2, false>(s, a, b);
    return ct ? launch_run<1, true>(s, a, b) : launch_run<1, false>(s, a, b);
}

hipError_t launch_block_deferred(hipStream_t s, const BlockArgs &b)
{
    if (b.steps < 1 || b.steps > kPbMaxSteps || b.n < 1 || b.n > kPbMaxN || b.n_edges < 1 ||
        b.n_edges > INT32_MAX || b.n_cu < 1 || b.syn_slots < 1 || (b.hw != 1 && b.hw != 2) ||
        b.df_parts < 1 || b.df_parts > (kMaxSortRow + 7 + kDfPart - 1) / kDfPart)
        return hipErrorInvalidValue;
    const int grid = (int)std::min<int64_t>(
        (int64_t)b.n_cu, ((int64_t)b.n * b.df_parts + kDfBlock / kWave - 1) / (kDfBlock / kWave));
    if (b.hw == 2)
        hipLaunchKernelGGL(k_block_deferred<2>, dim3(grid), dim3(kDfBlock), 0, s, b);
    else
        hipLaunchKernelGGL(k_block_deferred<1>, dim3(grid), dim3(kDfBlock), 0, s, b);
    return hipGetLastError();
}

hipError_t launch_block_finish(hipStream_t s, const BlockArgs &b)
{
    if (b.delay < 2 || b.delay > 64 || b.n < 1) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_block_finish, dim3(b.delay + 1), dim3(kPbFinishBlock), 0, s, b);
    return hipGetLastError();
}

}  // namespace snn
