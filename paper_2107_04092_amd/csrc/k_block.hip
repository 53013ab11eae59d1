// gfx950 kernels of a block of steps of a plastic network with D >= 2 (see
// BlockArgs): the plan of the block's rows, the target groups' run of its
// steps, and the per-step lists rebuilt after the last block.
//
// Built with -ffp-contract=off: the neuron update reproduces a fixed fp32
// operation order.
#include "snn_neuron.h"

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
// step (RowInfo), taken from the t_last and x_pre that the row's earlier
// events in the block left. The steps are walked twice: once for the event
// flags (each step's counts, scanned over the workgroups by a decoupled
// look-back, one scan per step), then for the snapshots, written at their
// positions in the step's ascending list.

__global__ __launch_bounds__(kPbPlanBlock) void k_block_plan(BlockArgs b)
{
    constexpr int NWV = kPbPlanBlock / kWave;
    __shared__ uint64_t s_m[kBatchMax][NWV];
    __shared__ int s_lb[2 * kBatchMax];
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
    // the steps with an event
    uint32_t evm = 0;
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
                    tl = (int)t;
                }
            }
            evm |= (uint32_t)ev << q;
            const uint64_t m = ballot64(ev);
            if (lane == 0) s_m[q][wave] = m;
        }
    }
    __syncthreads();  // s_m, s_dpow, s_st
    // this workgroup's events of step tid, published for the step's scan
    int own = 0;
    if (tid < B) {
        for (int w = 0; w < NWV; ++w) own += __popcll(s_m[tid][w]);
        publish_status(b.status + (int64_t)tid * b.status_stride + blockIdx.x,
                       status_word(own, 0, t0 + tid, blockIdx.x == 0 ? kStatusInc : kStatusAgg));
    }
    lookback32<kPbPlanBlock>(b.status, b.status_stride, B, (int)blockIdx.x, t0, s_lb, b.err);
    if (tid < B && blockIdx.x > 0)
        publish_status(b.status + (int64_t)tid * b.status_stride + blockIdx.x,
                       status_word(s_lb[2 * tid] + own, 0, t0 + tid, kStatusInc));
    // the snapshots, at their positions: earlier workgroups, earlier waves,
    // earlier lanes
    const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
    int tl = tl0;
    float xp = xp0;
    long long n_rows = 0, n_forced = 0, n_syn = 0, n_fsyn = 0;
    for (int q = 0; q < B; ++q) {
        if (!((evm >> q) & 1u)) continue;
        const int64_t t = t0 + q;
        const int tx = (int)((h0 >> (D - 2 - q)) & 1ull);
        RowInfo ri = RowInfo{};
        int ok = 0;
        if (plastic) {
            ok = make_row_info_d(ri, k, t, tl, rs, pend_k, xp, tx, hw,
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
        if (!ok) {  // nothing to bring up to date: the row is only delivered
            ri = RowInfo{};
            ri.k = k;
            ri.rs = rs;
        }
        ri.pad = tx;
        int pos = s_lb[2 * q] + __popcll(s_m[q][wave] & below);
        for (int w = 0; w < wave; ++w) pos += __popcll(s_m[q][w]);
        // (only a failed scan puts a position out of range)
        if (pos < b.n)
            b.ev[(int64_t)q * b.n + pos] = ri;
        else
            atomicOr(b.err, kErrRing);
    }
    if (plastic && tl != tl0) {  // the row as its last event in the block left it
        b.t_last[k] = tl;
        b.xpre[k] = xp;
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
    // the last workgroup's scans saw every workgroup: the step totals
    if (blockIdx.x == gridDim.x - 1 && tid < B) b.ev_cnt[tid] = s_lb[2 * tid] + own;
}

// ---------------------------------------------------------------------------
// The run of the block: workgroup of target group g (targets [g gw, g gw +
// gw), gw = gwidth, inside one slice), every step t = t0 + q:
//   (1) the neuron update of the group's targets (thread j: neuron g gw + j,
//       its state in registers from the first step to the last), with the
//       input of step t: the state's input at t0, afterwards the LDS
//       accumulator; the new history words and post traces go to LDS;
//   (2) the step's rows (the plan's list): for each, its entries with a
//       target in the group (gpiv), staged as in slice delivery (segment
//       starts, prefix sums of the lengths, a map from each flattened entry
//       to its segment), then every entry: the plastic ones brought up to
//       date from the target's history in LDS (a forced row: only those; its
//       other entries are not read), and a transmitting row's entries added
//       to the accumulator (64-bit fixed point, LDS atomics), which step
//       t+1's neuron update reads.
// A synapse belongs to the group of its target, so each weight is read and
// written by one workgroup only, and the steps of a workgroup are ordered by
// its barriers.
//
// The steps are pipelined so that a step waits for no round trip to memory
// started by itself: once step q's last barrier has ordered its weight
// stores, the entries of step q+1 (the first window of its first batch,
// staged and mapped during step q in the other of two staging buffers) are
// loaded, with the group pivots of step q+3's rows and the snapshots of
// step q+4; step q+1 consumes only loads started one or more steps before
// (a wave's loads complete in the order they were issued). Further windows
// and batches of a step (more entries or rows than one staging holds) are
// loaded when the step reaches them.
//
// At the end the state goes back, the accumulator becomes partial sum 0 (the
// input of step t0 + B), and workgroup 0 advances the step clock, which no
// workgroup of the run reads (they read the plan's copy).

constexpr int kPbDirect = 32;  // segments up to this long are mapped by their own thread
constexpr long long kMask40 = (1ll << 40) - 1;
// per segment of the staging: plastic entries (bits 0-17), age (18-25), pre
// (26), inhibitory source of a CUBA network (27), delivered (28)
constexpr int kInfoPlen = 0x3ffff;
// per loaded entry: segment (bits 0-9), plastic (10), present (11), its
// offset in the segment (12-31; segments are at most kMaxSortRow long)
constexpr int kPkSeg = 0x3ff, kPkPlastic = 1 << 10, kPkIn = 1 << 11, kPkOff = 12;
static_assert(kPbBatch <= kPkSeg + 1, "segment index fits the entry word");
static_assert(kMaxSortRow < (1 << (31 - kPkOff)), "segment offset fits the entry word");

struct PbStage {
    long long start[kPbBatch];  // segment starts (edge index)
    long long total;            // entries (bits 0-39), segments longer than kPbDirect (40+)
    int off[kPbBatch + 1];      // segment offsets
    int info[kPbBatch];
    float xp0[kPbBatch];
    float xpn[kPbBatch];
    uint16_t map[kPbWindow];    // entry -> 1 + segment
};

struct PbEntries {
    float wv[kPbUnroll];      // weight as loaded
    int cv[kPbUnroll];        // target as loaded (slice-local with compressed targets)
    int pk[kPbUnroll];
};

template <int HW, bool CT>
__global__ __launch_bounds__(kPbBlock) void k_block_run(NeuronArgs a, BlockArgs b)
{
    __shared__ PbStage S[2];
    __shared__ uint64_t s_hist[kPbMaxWidth * HW];
    __shared__ float s_y[kPbMaxWidth];
    __shared__ long long s_acc[2 * kPbMaxWidth];
    __shared__ float s_dpow[kMaxAge + 1];
    __shared__ long long sh[kPbBlock / kWave];
    __shared__ int shi[kPbBlock / kWave];
    __shared__ int s_cnt[kBatchMax];
    const int tid = threadIdx.x;
    // neighbouring groups (which read neighbouring entries of each row) on
    // one XCD: workgroup b runs on XCD b mod 8
    const int nb = gridDim.x;  // multiple of 8
    const int g = (blockIdx.x & 7) * (nb >> 3) + (blockIdx.x >> 3);
    if (g >= b.n_groups) return;  // whole workgroup, before any barrier
    const int n = a.n;
    const int glo = g * b.gwidth;
    const int wn = min(b.gwidth, n - glo);  // > 0
    const int cbase = CT ? glo % b.width : glo;  // subtracted from a loaded target
    const int i = glo + tid;
    const bool live = tid < wn;
    const int B = b.steps;
    const int G1 = b.n_groups + 1;
    const long long ne1 = (long long)b.n_edges - 1;  // (same-type min / max)
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
    const float c_pot = b.c_pot, c_dep = b.c_dep, mu = b.mu;
    const int32_t *__restrict__ col = b.col;
    const uint16_t *__restrict__ col16 = b.col16;
    float *__restrict__ wgt = b.w;
    long long events = 0, w_tx = 0, w_forced = 0, spikes = 0;
    __syncthreads();  // s_cnt, s_dpow

    auto nbt_of = [&](int q) { return q < B ? min(s_cnt[q], kPbBatch) : 0; };
    // snapshots e0 + 2 tid, e0 + 2 tid + 1 of step q's list (a valid index
    // for every lane: the loads go out unconditionally, and lanes past the
    // count are told apart when staged)
    auto load_rows = [&](int q, int e0, RowInfo (&R)[kPbRounds]) {
        const int c = q < B ? s_cnt[q] : 0;
        const RowInfo *src = b.ev + (int64_t)min(q, B - 1) * n;
#pragma unroll
        for (int r = 0; r < kPbRounds; ++r)
            R[r] = src[min(e0 + kPbRounds * tid + r, max(c - 1, 0))];
    };
    // the group's pivots of those rows
    auto load_piv = [&](const RowInfo (&R)[kPbRounds], int (&p0)[kPbRounds],
                        int (&p1)[kPbRounds]) {
#pragma unroll
        for (int r = 0; r < kPbRounds; ++r) {
            const int k = min(max(R[r].k, 0), n - 1);
            const int32_t *gp = b.gpiv + (int64_t)k * G1 + g;
            p0[r] = gp[0];
            p1[r] = gp[1];
        }
    };
    // segments of nbt rows into s, offsets scanned; ends with a barrier
    auto stage = [&](PbStage &s, const RowInfo (&R)[kPbRounds], const int (&p0)[kPbRounds],
                     const int (&p1)[kPbRounds], int nbt) {
        int len[kPbRounds];
        long long packed = 0;
#pragma unroll
        for (int r = 0; r < kPbRounds; ++r) {
            const int j = kPbRounds * tid + r;
            len[r] = 0;
            if (j < nbt) {
                const RowInfo &ri = R[r];
                int sl = max(p1[r] - p0[r], 0);
                const int deliver = ri.pad & 1;
                const int plen = ri.age_pre != 0 ? min(max(ri.len - p0[r], 0), sl) : 0;
                if (!deliver) sl = plen;  // a forced row: its plastic entries only
                len[r] = sl;
                const int inh = (b.nacc == 2 && ri.k >= b.n_exc) ? 1 : 0;
                s.start[j] = ri.rs + p0[r];
                s.info[j] = plen | ((ri.age_pre & 0xff) << 18) | (((ri.age_pre >> 8) & 1) << 26) |
                            (inh << 27) | (deliver << 28);
                s.xp0[j] = ri.xp0;
                s.xpn[j] = ri.xp_now;
            }
            packed += (long long)len[r] | ((long long)(len[r] > kPbDirect) << 40);
        }
        const long long incl = block_incl_scan_i64_n<kPbBlock>(packed, sh);
        long long ex = (incl - packed) & kMask40;
#pragma unroll
        for (int r = 0; r < kPbRounds; ++r) {
            s.off[kPbRounds * tid + r] = (int)ex;
            ex += len[r];
        }
        if (tid == kPbBlock - 1) {
            s.off[kPbBatch] = (int)(incl & kMask40);
            s.total = incl;
        }
        __syncthreads();
    };
    // the segment map of window [w0, w0 + we) of s; ends with a barrier
    auto build_map = [&](PbStage &s, int nbt, int w0, int we, bool direct) {
        if (direct) {  // short segments: each thread writes its own segments' entries
#pragma unroll
            for (int r = 0; r < kPbRounds; ++r) {
                const int j = kPbRounds * tid + r;
                if (j < nbt) {
                    const int a0 = max(s.off[j], w0), a1 = min(s.off[j + 1], w0 + we);
                    for (int x = a0; x < a1; ++x) s.map[x - w0] = (uint16_t)(j + 1);
                }
            }
            __syncthreads();
        } else {  // mark each segment's first entry in the window, then max-scan
            for (int x = tid; x < we; x += kPbBlock) s.map[x] = 0;
            __syncthreads();
#pragma unroll
            for (int r = 0; r < kPbRounds; ++r) {
                const int j = kPbRounds * tid + r;
                if (j < nbt) {
                    const int a0 = max(s.off[j], w0), a1 = min(s.off[j + 1], w0 + we);
                    if (a0 < a1) s.map[a0 - w0] = (uint16_t)(j + 1);
                }
            }
            __syncthreads();
            fill_segment_map<kPbBlock, kPbUnroll, uint16_t>(s.map, we, shi, 0);
        }
    };
    // loads of the entries of window [w0, w0 + we) of s: every slot loads
    // from a valid address (clamped to the graph), the results are looked at
    // when the entries are computed
    auto issue = [&](const PbStage &s, int w0, int we, PbEntries &E) {
#pragma unroll
        for (int u = 0; u < kPbUnroll; ++u) {
            const int x = u * kPbBlock + tid;
            const bool in = x < we;
            const int l = in ? (int)s.map[x] - 1 : 0;
            const int off = w0 + x - s.off[l];
            const long long e = in ? min(max(s.start[l] + off, 0ll), ne1) : 0;
            E.cv[u] = CT ? (int)col16[e] : col[e];
            E.wv[u] = wgt[e];
            E.pk[u] = in ? l | (off < (s.info[l] & kInfoPlen) ? kPkPlastic : 0) | kPkIn |
                               (off << kPkOff)
                         : 0;
        }
    };
    // entries loaded before the step before this one stored its weights:
    // those of rows brought up to date at both steps are loaded again
    // an entry's edge index (clamped as when it was loaded)
    auto edge = [&](const PbStage &s, int pk) {
        return min(max(s.start[pk & kPkSeg] + (long long)(pk >> kPkOff), 0ll), ne1);
    };
    auto compute = [&](const PbStage &s, const PbEntries &E) {
#pragma unroll
        for (int u = 0; u < kPbUnroll; ++u) {
            const int pk = E.pk[u];
            if (!(pk & kPkIn)) continue;
            const int l = pk & kPkSeg;
            const int info = s.info[l];
            const int j = E.cv[u] - cbase;
            if ((unsigned)j >= (unsigned)wn) {  // not this group's target
                atomicOr(b.err, kErrIndex);
                continue;
            }
            float w = E.wv[u];
            if (pk & kPkPlastic) {
                const int age = (info >> 18) & 0xff, pre = (info >> 26) & 1;
                uint64_t m0, m1;
                window_masks(age, m0, m1);
                const uint64_t h0 = s_hist[j * HW] & m0;
                const uint64_t h1 = HW == 2 ? s_hist[j * 2 + 1] & m1 : 0ull;
                if (h0 || h1 || pre || !b.event) {
                    const float y = pre ? s_y[j] : 0.f;
                    w = b.event ? stdp_synapse(w, h0, h1, age, pre, s.xp0[l], s.xpn[l], y, s_dpow,
                                               c_pot, c_dep, mu)
                                : stdp_synapse_steps(w, h0, h1, age, pre, s.xp0[l], s.xpn[l], y,
                                                     s_dpow[1], c_pot, c_dep, mu);
                    wgt[edge(s, pk)] = w;
                    if (pre)
                        ++w_tx;
                    else
                        ++w_forced;
                }
            }
            if ((info >> 28) & 1) {
                atomicAdd((unsigned long long *)(s_acc + j + (((info >> 27) & 1) ? kPbMaxWidth : 0)),
                          (unsigned long long)to_fix(w));
                ++events;
            }
        }
    };
    // everything of the step staged in s beyond its first window, and its
    // further batches (each loaded, staged and mapped when reached)
    auto rest_of_step = [&](int q, PbStage &s, PbEntries &E) {
        const int cnt = s_cnt[q];
        for (int e0 = 0; e0 < cnt; e0 += kPbBatch) {
            const int nbt = min(kPbBatch, cnt - e0);
            if (e0 > 0) {
                __syncthreads();  // every read of the staging of the batch before
                RowInfo R[kPbRounds];
                int p0[kPbRounds], p1[kPbRounds];
                load_rows(q, e0, R);
                load_piv(R, p0, p1);
                stage(s, R, p0, p1, nbt);
            }
            const long long tq = s.total;
            const int total = (int)(tq & kMask40);
            const bool direct = (tq >> 40) == 0;
            for (int w0 = e0 > 0 ? 0 : kPbWindow; w0 < total; w0 += kPbWindow) {
                const int we = min(kPbWindow, total - w0);
                __syncthreads();  // every read of the map of the window before
                build_map(s, nbt, w0, we, direct);
                issue(s, w0, we, E);
                compute(s, E);
            }
        }
    };

    // prologue: step 0 staged and its first window loaded, the snapshots of
    // steps 1-3 and the pivots of steps 1-2 loaded
    PbEntries E;
    RowInfo R1[kPbRounds], R2[kPbRounds], R3[kPbRounds];
    int P1a[kPbRounds], P1b[kPbRounds], P2a[kPbRounds], P2b[kPbRounds];
    {
        RowInfo R0[kPbRounds];
        int p0[kPbRounds], p1[kPbRounds];
        load_rows(0, 0, R0);
        load_rows(1, 0, R1);
        load_rows(2, 0, R2);
        load_rows(3, 0, R3);
        load_piv(R0, p0, p1);
        load_piv(R1, P1a, P1b);
        load_piv(R2, P2a, P2b);
        stage(S[0], R0, p0, p1, nbt_of(0));
        const long long tq = S[0].total;
        const int total = (int)(tq & kMask40);
        if (total > 0) build_map(S[0], nbt_of(0), 0, min(total, kPbWindow), (tq >> 40) == 0);
        issue(S[0], 0, min(total, kPbWindow), E);
    }
    for (int q = 0; q < B; ++q) {
        PbStage &cur = S[q & 1];
        PbStage &nxt = S[(q + 1) & 1];
        const int64_t t = t0 + q;
        // (1) neuron update; the accumulator it read is cleared
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
            spikes += neuron_advance<-1, HW>(a, i, t, ae, ai, st);
            s_hist[tid * HW] = st.h0;
            if (HW == 2) s_hist[tid * 2 + 1] = st.h1;
            s_y[tid] = st.y;
        }
        s_acc[tid] = 0;
        s_acc[kPbMaxWidth + tid] = 0;
        // (2a) step q+1 staged and its first window mapped (the staging's
        // barriers publish the neuron update)
        if (q + 1 < B) {
            const int nb1 = nbt_of(q + 1);
            stage(nxt, R1, P1a, P1b, nb1);
            const long long tq = nxt.total;
            const int total = (int)(tq & kMask40);
            if (total > 0) build_map(nxt, nb1, 0, min(total, kPbWindow), (tq >> 40) == 0);
        } else {
            __syncthreads();  // the neuron update's histories and traces
        }
        // (2b) the entries of step q
        compute(cur, E);
        rest_of_step(q, cur, E);
        __syncthreads();  // every atomic and weight store of step q done
        // (3) the loads for the steps ahead
        if (q + 1 < B) {
            const int total = (int)(nxt.total & kMask40);
            issue(nxt, 0, min(total, kPbWindow), E);
#pragma unroll
            for (int r = 0; r < kPbRounds; ++r) {
                R1[r] = R2[r];
                R2[r] = R3[r];
                P1a[r] = P2a[r];
                P1b[r] = P2b[r];
            }
            load_piv(R2, P2a, P2b);
            load_rows(q + 4, 0, R3);
        }
    }
    if (live) {
        nstate_store<-1, HW>(a, i, st);
        a.code[i] = hist_code(st.h0, st.h1);
        b.apart[i] = s_acc[tid];
        if (b.nacc == 2) b.apart[n + i] = s_acc[kPbMaxWidth + tid];
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
    if (b.steps < 1 || b.steps > kBatchMax || b.steps > b.delay - 1 || b.n < 1 ||
        b.n > kPbMaxN || b.status_stride < blocks_for(b.n, kPbPlanBlock) ||
        (int64_t)b.status_stride * kBatchMax > b.status_words)
        return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_block_plan, dim3(blocks_for(b.n, kPbPlanBlock)), dim3(kPbPlanBlock), 0,
                       s, b);
    return hipGetLastError();
}

hipError_t launch_block_run(hipStream_t s, const NeuronArgs &a, const BlockArgs &b)
{
    if (b.steps < 1 || b.steps > kBatchMax || b.gwidth < 1 || b.gwidth > kPbMaxWidth ||
        b.n_edges < 1 ||
        b.width % b.gwidth != 0 || (int64_t)b.n_groups * b.gwidth < a.n ||
        (int64_t)(b.n_groups - 1) * b.gwidth >= a.n || a.n != b.n || b.nacc < 1 || b.nacc > 2 ||
        b.dlv_slots < 1 || b.syn_slots < 1)
        return hipErrorInvalidValue;
    const bool ct = b.col16 != nullptr;
    if (a.hw == 2) return ct ? launch_run<2, true>(s, a, b) : launch_run<2, false>(s, a, b);
    return ct ? launch_run<1, true>(s, a, b) : launch_run<1, false>(s, a, b);
}

hipError_t launch_block_finish(hipStream_t s, const BlockArgs &b)
{
    if (b.delay < 2 || b.delay > 64 || b.n < 1) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_block_finish, dim3(b.delay + 1), dim3(kPbFinishBlock), 0, s, b);
    return hipGetLastError();
}

}  // namespace snn
