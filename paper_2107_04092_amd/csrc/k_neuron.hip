// gfx950 kernels of the neuron part of a step: state initialisation and
// fills, and the neuron update (firing masks, histories, post traces) that
// also builds the spike / transmitted / forced lists with row snapshots.
//
// Built with -ffp-contract=off: the neuron update must reproduce a fixed
// fp32 operation order, so no multiply-add is ever fused.
#include "snn_neuron.h"

namespace snn {
namespace {

// ---------------------------------------------------------------------------
// state initialisation and fills (kernels instead of memsets so that a
// captured step never contains a memset node)

__global__ __launch_bounds__(kBlock) void k_init_state(float *v, int32_t *ref, float *ie,
                                                       float *ii, uint64_t *hist, float *ypost,
                                                       int32_t *t_last, float *xpre, int32_t n,
                                                       int32_t hw)
{
    const int i = blockIdx.x * kBlock + threadIdx.x;
    if (i >= n) return;
    v[i] = 0.f;
    ref[i] = 0;
    ie[i] = 0.f;
    ii[i] = 0.f;
    for (int q = 0; q < hw; ++q) hist[(int64_t)i * hw + q] = 0ull;
    ypost[i] = 0.f;
    // Rows start staggered over 64 hw phases. No spike precedes step 0 and
    // the pre trace starts at 0, so any t_last <= -1 gives the same weights;
    // staggering spreads the forced updates of idle rows evenly over steps.
    t_last[i] = -1 - (i & (64 * hw - 1));
    xpre[i] = 0.f;
}

template <typename T>
__global__ __launch_bounds__(kBlock) void k_fill(T *p, int64_t count, T value)
{
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < count; i += stride)
        p[i] = value;
}

// ---------------------------------------------------------------------------
// (1) neuron update, one wave64 per mask word and one neuron per thread, and
// the lists of the step: spikes (into the delay ring), forced plastic rows
// and the snapshots of the rows to bring up to date (see CompactArgs).
//
// List offsets: the lists are ascending, workgroup by workgroup. Each
// workgroup publishes its spike and forced-row counts in a status word and
// learns the counts of all earlier workgroups by a decoupled look-back over
// theirs (lookback), so no workgroup waits on a shared counter: same-address
// device atomics serialise. Transmitting rows need no list of their own: a
// row transmitting at t spiked at t-D+1, when its position in that step's
// spike list was recorded (spk_pos); its snapshot goes to the same position,
// so snapshots line up with the delay-ring list delivery reads. The step
// index and the input source come from the device clock (StepClock); the
// last workgroup publishes the counts and advances the clock.

// The whole update of neuron i from and to the state arrays, in three parts:
// the loads, issued before the clock is read (so the state and the clock
// arrive in one round trip); the update at step t with the input source of
// the clock, which returns spiked / transmitting / forced and, for a plastic
// row, its t_last; and the stores (neuron_commit), which the caller issues
// after its last wait for a load: with stores outstanding, a wait for any
// load also waits for every earlier store.
struct NeuronLoads {
    NState st;
    int t_last;
    InputLoads in;
};
__device__ __forceinline__ void neuron_issue(const NeuronArgs &a, int i, NeuronLoads &L)
{
    nstate_load<-1, 0>(a, i, L.st);
    L.t_last = i < a.n_plastic_rows ? a.t_last[i] : 0;
    if (a.model != 2) input_issue(a, i, L.in);
}
__device__ __forceinline__ void neuron_update(const NeuronArgs &a, const StepClock &ck, int i,
                                              int64_t t, NeuronLoads &L, int &s, int &tx,
                                              int &forced, bool &fired_recently, int &t_last_i)
{
    NState &st = L.st;
    t_last_i = L.t_last;
    float ae = 0.f, ai = 0.f;
    if (a.model != 2) input_combine(a, L.in, ck.input_forced, ck.n_parts, i, ae, ai);
    s = neuron_advance<-1, 0>(a, i, t, ae, ai, st);
    fired_recently = (st.h0 | st.h1) != 0ull;
    tx = (int)((st.h0 >> a.dm1) & 1ull);
    if (i < a.n_plastic_rows) forced = !tx && (t - (int64_t)t_last_i >= 64 * a.hw);
}
__device__ __forceinline__ void neuron_commit(const NeuronArgs &a, int i, const NState &st)
{
    nstate_store<-1, 0>(a, i, st);
    a.code[i] = hist_code(st.h0, st.h1);
}

// NB threads per workgroup: 1024 on large networks (fewer workgroups to look
// back over), 256 up to kNeuronSmallN neurons, where 1024 would leave most
// CUs without a workgroup.
template <int NB>
__global__ __launch_bounds__(NB) void k_neuron(NeuronArgs a, CompactArgs lst)
{
    constexpr int NWV = NB / kWave;
    __shared__ int s_cnt[2][NWV];
    __shared__ unsigned long long s_st[4];
    __shared__ int s_lb[8];
    const int tid = threadIdx.x;
    const int wave = tid / kWave, lane = tid % kWave;
    const bool plastic = lst.n_plastic_rows > 0;
    const int D = lst.delay;
    const int i = blockIdx.x * NB + tid;
    if (tid < 4) s_st[tid] = 0ull;
    // the state loads, then the clock (vector loads, which the state loads
    // do not wait for): one round trip
    NeuronLoads L;
    if (i < a.n) neuron_issue(a, i, L);
    const StepClock ck = load_clock(a.clk);
    const int64_t t = ck.t;
    int s = 0, tx = 0, forced = 0, tl = 0;
    bool fired_recently = false;
    if (i < a.n) neuron_update(a, ck, i, t, L, s, tx, forced, fired_recently, tl);
    // the count of the transmitted list (D > 1: written D-1 steps ago), for
    // the fixed address the synapse pass reads: loaded now, stored at the end
    const bool tx_writer = blockIdx.x == 0 && tid == 0 && a.dm1 > 0;
    const int tx_count = tx_writer ? lst.ring_cnt[ring_slot(t - a.dm1, D)] : 0;
    const uint64_t m = ballot64(s), fm = ballot64(forced);
    const uint64_t txm = ballot64(tx), rcm = ballot64(fired_recently);
    if (lane == 0) {
        s_cnt[0][wave] = __popcll(m);
        s_cnt[1][wave] = __popcll(fm);
    }
    // The values a row snapshot needs, loaded for the rows to bring up to
    // date at t only (transmitting plastic rows, forced rows), and a
    // transmitting row's position in the spike list of step t-D+1: the loads
    // are issued now and arrive during the list scan.
    const bool snap_tx = tx && plastic;
    int64_t rs = 0;
    int pend_i = 0, txpos = -1;
    float xp = 0.f, dp = 0.f;
    if (snap_tx || forced) {
        rs = lst.row_ptr[i];
        if (i < lst.n_plastic_rows) {
            pend_i = lst.pend[i];
            xp = lst.xpre[i];
            dp = lst.dpow[row_age_index(t, tl, lst.hw)];
        }
        if (snap_tx && a.dm1 > 0) txpos = lst.spk_pos[(int64_t)ring_slot(t - a.dm1, D) * a.n + i];
    }
    // a forced row's pivots at the range boundaries (forced rows split by
    // target range): loaded with the snapshot values, read under the same
    // condition (left unset otherwise, so no merge waits for the loads)
    int pv[kXcds - 1];
    if (forced && lst.segb) {
        // (all seven: the boundaries past the last range repeat its end, so
        // each index is a pivot of the row; no load waits inside a branch)
        const int32_t *pr = lst.piv + (int64_t)i * lst.piv_stride;
#pragma unroll
        for (int x = 0; x < kXcds - 1; ++x) pv[x] = pr[lst.xcd_piv[x + 1]];
    }
    __syncthreads();  // s_cnt, s_st
    int agg_s = 0, agg_f = 0;
#pragma unroll
    for (int q = 0; q < NWV; ++q) {
        agg_s += s_cnt[0][q];
        agg_f += s_cnt[1][q];
    }
    if (tid == 0)
        publish_status(lst.status + blockIdx.x,
                       status_word(agg_s, agg_f, t, blockIdx.x == 0 ? kStatusInc : kStatusAgg));
    lookback<NB, 1>(lst.status, 0, 1, (int)blockIdx.x, t, s_lb, lst.err);
    const int pre_s = s_lb[6], pre_f = s_lb[7];  // spikes and forced rows of earlier workgroups
    // the values loaded before the scan (arrived during it) are taken here,
    // before thread 0's status store: a later wait for them would also wait
    // for that store
    asm volatile("" ::"v"(rs), "v"(pend_i), "v"(xp), "v"(dp), "v"(txpos), "v"(tx_count));
    if (tid == 0 && blockIdx.x > 0)
        publish_status(lst.status + blockIdx.x,
                       status_word(pre_s + agg_s, pre_f + agg_f, t, kStatusInc));
    if (tx_writer) *lst.tx_cnt = tx_count;
    // snapshots of the rows to bring up to date (taken before any kernel
    // commits t_last / x_pre)
    RowInfo ri = RowInfo{};
    int ri_ok = 0;
    if (snap_tx) {
        // the row transmits at t exactly when tx (history bit D-1 of step t)
        if (i < lst.n_plastic_rows)
            ri_ok = make_row_info_d(ri, i, t, tl, rs, pend_i, xp, 1, lst.hw, dp, lst.err);
        if (!ri_ok) {  // nothing to bring up to date: the row is only delivered
            ri = RowInfo{};
            ri.k = i;
            ri.rs = rs;
        }
    } else if (forced) {
        ri_ok = make_row_info_d(ri, i, t, tl, rs, pend_i, xp, 0, lst.hw, dp, lst.err);
    }
    if (lst.info_stats) {
        const bool f = forced && ri_ok;
        const long long v0 = __popcll(ballot64(ri_ok)), v1 = __popcll(ballot64(f));
        const long long v2 = wave_sum_i64(ri_ok ? ri.len : 0), v3 = wave_sum_i64(f ? ri.len : 0);
        if (lane == 0) {
            if (v0) atomicAdd(s_st + 0, (unsigned long long)v0);
            if (v1) atomicAdd(s_st + 1, (unsigned long long)v1);
            if (v2) atomicAdd(s_st + 2, (unsigned long long)v2);
            if (v3) atomicAdd(s_st + 3, (unsigned long long)v3);
        }
    }
    // this wave's offsets: the earlier workgroups, then the earlier waves
    const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
    int p0 = pre_s, p2 = pre_f;
    for (int q = 0; q < wave; ++q) {
        p0 += s_cnt[0][q];
        p2 += s_cnt[1][q];
    }
    const int slot = ring_slot(t, D);
    // (the bounds checks only catch a failed scan; otherwise every offset is
    // in range)
    if (s) {
        const int pos = p0 + __popcll(m & below);
        if (pos < a.n) {
            lst.ring[(int64_t)slot * a.n + pos] = i;
            if (plastic && a.dm1 > 0) lst.spk_pos[(int64_t)slot * a.n + i] = pos;
            if (a.dm1 == 0) txpos = pos;  // D = 1: transmitted as it fires
        } else {
            atomicOr(lst.err, kErrRing);
        }
    }
    if (snap_tx) {
        if (txpos >= 0 && txpos < a.n)
            lst.txinfo[txpos] = ri;
        else
            atomicOr(lst.err, kErrRing);
    }
    if (forced) {
        const int q = p2 + __popcll(fm & below);
        if (q < lst.n_plastic_rows) {
            lst.row_list[q] = i;
            lst.info[q] = ri;
            if (lst.segb) {
                // segment ends, moved to the nearest 128-byte line of the
                // weight array (monotone: the pivots are)
                int e[kXcds];
#pragma unroll
                for (int x = 0; x < kXcds - 1; ++x) {
                    // (an empty asm pins the pivot here: no conversion of it
                    // is hoisted to its load, where it would wait for it)
                    asm volatile("" : "+v"(pv[x]));
                    const int64_t al = ((rs + pv[x] + kStoreLine / 2) & ~(int64_t)(kStoreLine - 1));
                    e[x] = x < lst.xparts - 1 ? (int)min(max(al - rs, (int64_t)0), (int64_t)pend_i)
                                              : pend_i;
                }
                e[kXcds - 1] = pend_i;
                int4 *dst = reinterpret_cast<int4 *>(lst.segb + (int64_t)q * kXcds);
                dst[0] = make_int4(e[0], e[1], e[2], e[3]);
                dst[1] = make_int4(e[4], e[5], e[6], e[7]);
            }
        } else {
            atomicOr(lst.err, kErrRing);
        }
    }
    // the neuron's state and the masks: stored after the last wait for a
    // load (the snapshot values above)
    if (i < a.n) neuron_commit(a, i, L.st);
    if (lane == 0) {
        const int64_t word = (int64_t)blockIdx.x * NWV + wave;
        if (word * kWave < a.n) {
            a.mask[word] = m;
            a.txmask[word] = txm;
            a.recent[word] = rcm;
        }
    }
    if (lst.info_stats) {
        __syncthreads();  // s_st complete
        if (tid == 0) {
            int64_t *sl = lst.info_stats + (int64_t)blockIdx.x * kStFields;
            add_stat(sl + kStRows, (long long)s_st[0]);
            add_stat(sl + kStForced, (long long)s_st[1]);
            add_stat(sl + kStSyn, (long long)s_st[2]);
            add_stat(sl + kStForcedSyn, (long long)s_st[3]);
        }
    }
    if (tid == 0 && blockIdx.x == gridDim.x - 1) {
        // every workgroup has read the clock: the look-back saw all of them
        const int n_spk = pre_s + agg_s, n_forced = pre_f + agg_f;
        lst.ring_cnt[slot] = n_spk;
        if (a.dm1 == 0) *lst.tx_cnt = n_spk;  // D = 1: this step's spikes transmit
        *lst.row_cnt = n_forced;
        add_stat(lst.gstats + kGSpikes, n_spk);
        add_stat(lst.gstats + kGSteps, 1);
        a.clk->t = t + 1;
    }
}

// ---------------------------------------------------------------------------
// Small networks without plasticity: b.steps whole steps in one workgroup,
// each thread holding the state of its neurons (one per round of
// kSmallBlock) in registers from the first step to the last. Each step:
// (1) the neuron update of every neuron (the same arithmetic as k_neuron;
// from the second step on the input is the LDS accumulator, exact like the
// fixed-point partial sums), fire and transmit masks, and the spike list in
// ascending order into ring slot t mod D; (3) delivery of ring slot
// (t-D+1) mod D, a wave per transmitted row, lanes over its targets, 64-bit
// fixed-point LDS atomics. At the end the state goes back to the arrays and
// the accumulator becomes partial sum 0, where the next neuron update (of
// either path) reads it.

template <int M, int H>
__global__ __launch_bounds__(kSmallBlock) void k_small_steps(NeuronArgs a, SmallArgs b)
{
    constexpr int NWV = kSmallBlock / kWave;
    extern __shared__ long long acc[];  // nacc * n
    __shared__ int s_cnt[kSmallRounds * NWV];
    __shared__ int s_total;
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const int n = a.n;
    const int rounds = (n + kSmallBlock - 1) / kSmallBlock;  // <= kSmallRounds
    const int span = b.nacc * n;
    const StepClock ck = *a.clk;
    long long events = 0, spikes = 0;
    NState st[kSmallRounds];
#pragma unroll
    for (int r = 0; r < kSmallRounds; ++r) {
        const int i = r * kSmallBlock + tid;
        if (r < rounds && i < n) nstate_load<M, H>(a, i, st[r]);
    }
    for (int k = 0; k < b.steps; ++k) {
        const int64_t t = ck.t + k;
        const int slot = (int)(t % b.delay);
        int32_t *list = b.ring + (int64_t)slot * n;
        // (1) neuron update
        int sp[kSmallRounds];
#pragma unroll
        for (int r = 0; r < kSmallRounds; ++r) {
            sp[r] = 0;
            if (r >= rounds) continue;  // workgroup-uniform
            const int i = r * kSmallBlock + tid;
            uint64_t hw0 = 0ull, hw1 = 0ull;
            if (i < n) {
                float ae = 0.f, ai = 0.f;
                if (M != 2) {
                    if (k == 0) {
                        neuron_input(a, ck.input_forced, ck.n_parts, i, ae, ai);
                    } else {
                        ae = from_fix(acc[i]);
                        if (M == 1) ai = from_fix(acc[n + i]);
                    }
                }
                sp[r] = neuron_advance<M, H>(a, i, t, ae, ai, st[r]);
                hw0 = st[r].h0;
                hw1 = st[r].h1;
            }
            const uint64_t m = ballot64(sp[r]);
            const uint64_t txm = ballot64((hw0 >> a.dm1) & 1ull);
            const uint64_t rcm = ballot64((hw0 | hw1) != 0ull);
            if (lane == 0) {
                const int word = r * NWV + wave;
                if (word * kWave < n) {
                    a.mask[word] = m;
                    a.txmask[word] = txm;
                    a.recent[word] = rcm;
                }
                s_cnt[word] = __popcll(m);
            }
        }
        __syncthreads();  // every input read, every count written
        for (int x = tid; x < span; x += kSmallBlock) acc[x] = 0;
        if (tid == 0) {  // exclusive offsets in (round, wave) = ascending order
            int o = 0;
            for (int q = 0; q < rounds * NWV; ++q) {
                const int c = s_cnt[q];
                s_cnt[q] = o;
                o += c;
            }
            s_total = o;
            b.ring_cnt[slot] = o;
        }
        __syncthreads();
        const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
        for (int r = 0; r < kSmallRounds; ++r) {
            if (r >= rounds) continue;
            const uint64_t m = ballot64(sp[r]);
            if (sp[r]) list[s_cnt[r * NWV + wave] + __popcll(m & below)] = r * kSmallBlock + tid;
        }
        spikes += s_total;
        __syncthreads();  // the list (global) and the cleared accumulator
        // (3) delivery of the spikes of step t-D+1 (this step's for D = 1)
        const int tslot = (int)((t - (b.delay - 1) + (int64_t)b.delay * 64) % b.delay);
        const int32_t *tlist = b.ring + (int64_t)tslot * n;
        const int ntx = min(max(b.ring_cnt[tslot], 0), n);
        for (int q = wave; q < ntx; q += NWV) {  // wave-uniform
            const int src = min(max(tlist[q], 0), n - 1);
            const int64_t rs = b.row_ptr[src], re = b.row_ptr[src + 1];
            const int half = (b.nacc == 2 && src >= b.n_exc) ? n : 0;
            for (int64_t e = rs + lane; e < re; e += kWave)
                atomicAdd((unsigned long long *)(acc + b.col[e] + half),
                          (unsigned long long)to_fix(b.w[e]));
            if (lane == 0) events += re - rs;
        }
        __syncthreads();  // accumulation done before the next step reads it
    }
#pragma unroll
    for (int r = 0; r < kSmallRounds; ++r) {
        const int i = r * kSmallBlock + tid;
        if (r < rounds && i < n) {
            nstate_store<M, H>(a, i, st[r]);
            a.code[i] = hist_code(st[r].h0, st[r].h1);
        }
    }
    for (int x = tid; x < span; x += kSmallBlock) b.apart[x] = acc[x];
    // the list scans of the other kernels find no stale step tag after these steps
    for (int x = tid; x < b.status_words; x += kSmallBlock) b.status[x] = 0ull;
    if (lane == 0 && events) atomicAdd((unsigned long long *)b.dlv_stats, (unsigned long long)events);
    if (tid == 0) {
        add_stat(b.gstats + kGSpikes, spikes);
        add_stat(b.gstats + kGSteps, b.steps);
        a.clk->t = ck.t + b.steps;
        a.clk->input_forced = 0;  // the next input is partial sum 0
        a.clk->n_parts = 1;
    }
}

// ---------------------------------------------------------------------------
// Delay block of a network without plasticity: b.steps (<= D-1) steps of the
// neuron update, one neuron per thread with its state in registers. Step t0
// (= clk->t) reads its input like k_neuron (the fp32 input or the partial
// sums); step t0 + k, k >= 1, reads slot k-1 of abatch, the whole input as
// one fixed-point sum, written beforehand by the batched delivery. Every
// slot's load is issued before the first step, so the steps wait for one
// round trip in all. The spike flags of every step are kept (a bit per step
// per thread, ballots in LDS), and the spike lists go into the delay ring at
// the end, ascending: one list scan per step (status row k of b.status),
// the B scans looked back over together. The masks, codes and the state
// written are those of the last step, and apart part 0 receives slot B-1,
// the pending input of the next step. Workgroups of 512 threads: the B
// steps of a thread run one after another, so fewer waves share a SIMD than
// with 1024.
constexpr int kStepsBlock = 512;
template <int M, int H>
__global__ __launch_bounds__(kStepsBlock) void k_neuron_steps(NeuronArgs a, BatchArgs b)
{
    constexpr int NWV = kStepsBlock / kWave;
    static_assert(kStepsBlock / 32 >= kBatchMax, "a half wave per step's list scan");
    __shared__ uint64_t s_m[kBatchMax][NWV];
    __shared__ int s_lb[2 * kBatchMax];
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const int n = a.n;
    const int i = blockIdx.x * kStepsBlock + tid;
    const bool live = i < n;
    const int ic = live ? i : 0;
    const int64_t ps = a.part_stride;  // nacc * n
    const StepClock ck = *a.clk;
    const int64_t t0 = ck.t;
    // steps per launch: CUBA holds two inputs per step in registers
    constexpr int KB = batch_steps_max(M);
    const int B = b.steps;  // 1 .. KB (checked by the launcher)
    // slot k = input of step t0 + k + 1 (Bernoulli sources read only the
    // last). Every load is issued unconditionally from a valid slot (past B:
    // slot B-1 again): a load under a branch would be waited for inside it.
    long long pe[KB], pi[KB];
#pragma unroll
    for (int k = 0; k < KB; ++k) {
        const int kk = M == 2 ? B - 1 : min(k, B - 1);
        const long long *p = b.abatch + (int64_t)kk * ps;
        pe[k] = M == 2 && k > 0 ? 0 : p[ic];
        pi[k] = M == 1 ? p[n + ic] : 0;
    }
    NState st = {};
    if (live) nstate_load<M, H>(a, i, st);
    uint32_t fired = 0;
#pragma unroll
    for (int k = 0; k < KB; ++k) {
        if (k >= B) break;
        float ae = 0.f, ai = 0.f;
        if (live && M != 2) {
            if (k == 0) {
                neuron_input(a, ck.input_forced, ck.n_parts, i, ae, ai);
            } else {
                ae = from_fix(pe[k - 1]);
                if (M == 1) ai = from_fix(pi[k - 1]);
            }
        }
        int sp = 0;
        if (live) sp = neuron_advance<M, H>(a, i, t0 + k, ae, ai, st);
        fired |= (uint32_t)sp << k;
        const uint64_t m = ballot64(sp);
        if (lane == 0) s_m[k][wave] = m;
    }
    if (live) {
        nstate_store<M, H>(a, i, st);
        a.code[i] = hist_code(st.h0, st.h1);
        long long le = pe[0], li = pi[0];  // Bernoulli sources: slot B-1 is pe[0]
        if (M != 2) {
#pragma unroll
            for (int k = 1; k < KB; ++k) {
                if (k == B - 1) {
                    le = pe[k];
                    li = pi[k];
                }
            }
        }
        b.apart[i] = le;
        if (M == 1) b.apart[n + i] = li;
    }
    {
        const uint64_t m = ballot64(live && ((fired >> (B - 1)) & 1u));
        const uint64_t txm = ballot64(live && ((st.h0 >> a.dm1) & 1ull));
        const uint64_t rcm = ballot64(live && (st.h0 | st.h1) != 0ull);
        const int64_t word = (int64_t)blockIdx.x * NWV + wave;
        if (lane == 0 && word * kWave < n) {
            a.mask[word] = m;
            a.txmask[word] = txm;
            a.recent[word] = rcm;
        }
    }
    __syncthreads();  // every step's ballots
    // the workgroup's spike count of each step (thread k), published for the scans
    int own = 0;
    if (tid < B) {
        for (int w = 0; w < NWV; ++w) own += __popcll(s_m[tid][w]);
        publish_status(b.status + (int64_t)tid * b.status_stride + blockIdx.x,
                       status_word(own, 0, t0 + tid, blockIdx.x == 0 ? kStatusInc : kStatusAgg));
    }
    lookback32<kStepsBlock>(b.status, b.status_stride, B, (int)blockIdx.x, t0, s_lb, b.err);
    // the spikes of step k before this workgroup: s_lb[2 k]
    if (tid < B && blockIdx.x > 0)
        publish_status(b.status + (int64_t)tid * b.status_stride + blockIdx.x,
                       status_word(s_lb[2 * tid] + own, 0, t0 + tid, kStatusInc));
    const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
    for (int k = 0; k < KB; ++k) {
        if (k >= B || !((fired >> k) & 1u)) continue;
        int pos = s_lb[2 * k] + __popcll(s_m[k][wave] & below);
        for (int w = 0; w < wave; ++w) pos += __popcll(s_m[k][w]);
        // (only a failed scan puts an offset out of range)
        if (pos < n)
            b.ring[(int64_t)ring_slot(t0 + k, b.delay) * n + pos] = i;
        else
            atomicOr(b.err, kErrRing);
    }
    if (blockIdx.x == gridDim.x - 1) {
        // every workgroup has read the clock: the scans saw all of them
        if (tid < B) {
            const int cnt = s_lb[2 * tid] + own;
            b.ring_cnt[ring_slot(t0 + tid, b.delay)] = cnt;
            add_stat(b.gstats + kGSpikes, cnt);
        }
    }
    if (tid == 0 && blockIdx.x == gridDim.x - 1) {
        add_stat(b.gstats + kGSteps, B);
        a.clk->t = t0 + B;
        a.clk->input_forced = 0;  // the next input is partial sum 0
        a.clk->n_parts = 1;
    }
}

// Steps t0 .. t0+B-1 of a plastic network of Bernoulli sources with D = 1
// (see SourceArgs), one neuron per thread, kStepsBlock threads per
// workgroup (a half wave per step's list scan). A row transmits at the step
// its neuron fires; a plastic row is forced at a step where it neither
// transmits nor was updated in the last 64 hw steps, as in k_neuron. The
// walk through the steps records the spike and forced bits and the state of
// each step; after the scans a second walk over the row's updates makes
// their snapshots, each starting from the t_last and pre trace the one
// before left (what the passes commit in between, step by step).
template <int H>
__global__ __launch_bounds__(kStepsBlock) void k_source_steps(NeuronArgs a, CompactArgs lst,
                                                              SourceArgs b)
{
    constexpr int NWV = kStepsBlock / kWave;
    static_assert(kStepsBlock / 32 >= kSrcMaxSteps, "a half wave per step's list scan");
    __shared__ uint64_t s_m[kSrcMaxSteps][NWV];  // transmitted rows of step k, per wave
    __shared__ uint64_t s_f[kSrcMaxSteps][NWV];  // forced rows
    __shared__ int s_lb[2 * kBatchMax];
    __shared__ unsigned long long s_st[4];
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const int n = a.n, npl = lst.n_plastic_rows;  // npl > 0
    const int i = blockIdx.x * kStepsBlock + tid;
    const bool live = i < n, prow = i < npl;
    const int ic = live ? i : 0, ip = prow ? i : 0;
    const int B = b.steps;  // 1 .. kSrcMaxSteps (checked by the launcher)
    if (tid < 4) s_st[tid] = 0ull;
    // the state and the row's values, then the clock: one round trip (every
    // load unconditional, from a valid index)
    NState st;
    nstate_load<-1, H>(a, ic, st);
    const int tl0 = a.t_last[ip];
    const int64_t rs = lst.row_ptr[ic];
    const int pend_k = lst.pend[ip];
    const float xp0 = lst.xpre[ip];
    const StepClock ck = load_clock(a.clk);
    const int64_t t0 = ck.t;
    const int64_t nh = (int64_t)n * H;
    uint32_t fired = 0, forced = 0;
    int tl = tl0;
    for (int k = 0; k < B; ++k) {
        const int64_t t = t0 + k;
        const int s = live ? neuron_advance<-1, H>(a, ic, t, 0.f, 0.f, st) : 0;
        const int f = live && prow && !s && t - (int64_t)tl >= 64 * H;
        if (live && prow && (s || f) && t > (int64_t)tl) tl = (int)t;
        fired |= (uint32_t)s << k;
        forced |= (uint32_t)f << k;
        const uint64_t m = ballot64(s), fm = ballot64(f);
        const uint64_t rcm = ballot64(live && (st.h0 | st.h1) != 0ull);
        if (lane == 0) {
            s_m[k][wave] = m;
            s_f[k][wave] = fm;
        }
        if (k < B - 1) {  // the step's versions (the last step's go to the state arrays)
            if (live) {
                uint64_t *hp = b.hist + k * nh + (int64_t)i * H;
                hp[0] = st.h0;
                if (H == 2) hp[1] = st.h1;
                b.ypost[(int64_t)k * n + i] = st.y;
                b.code[(int64_t)k * b.code_stride + i] = hist_code(st.h0, st.h1);
            }
            const int64_t word = (int64_t)blockIdx.x * NWV + wave;
            if (lane == 0 && word * kWave < n) b.recent[(int64_t)k * lst.nw + word] = rcm;
        } else {
            const int64_t word = (int64_t)blockIdx.x * NWV + wave;
            if (lane == 0 && word * kWave < n) {
                a.mask[word] = m;
                a.txmask[word] = m;  // D = 1: the spikes of the step transmit
                a.recent[word] = rcm;
            }
        }
    }
    if (live) neuron_commit(a, i, st);
    __syncthreads();  // every step's ballots, s_st
    // the workgroup's transmitted and forced counts of step `tid`, published
    // for the scans
    int own_s = 0, own_f = 0;
    if (tid < B) {
        for (int w = 0; w < NWV; ++w) {
            own_s += __popcll(s_m[tid][w]);
            own_f += __popcll(s_f[tid][w]);
        }
        publish_status(b.status + (int64_t)tid * b.status_stride + blockIdx.x,
                       status_word(own_s, own_f, t0 + tid,
                                   blockIdx.x == 0 ? kStatusInc : kStatusAgg));
    }
    lookback32<kStepsBlock>(b.status, b.status_stride, B, (int)blockIdx.x, t0, s_lb, lst.err);
    if (tid < B && blockIdx.x > 0)
        publish_status(b.status + (int64_t)tid * b.status_stride + blockIdx.x,
                       status_word(s_lb[2 * tid] + own_s, s_lb[2 * tid + 1] + own_f, t0 + tid,
                                   kStatusInc));
    // the row's updates in step order, each at its place in its step's list:
    // the earlier workgroups, then the earlier waves, then the earlier lanes
    const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
    int tlw = tl0;
    float xp = xp0;
    long long n_rows = 0, n_forced = 0, n_syn = 0, n_fsyn = 0;
    for (uint32_t ev = fired | forced; ev; ev &= ev - 1u) {
        const int k = __ffs((int)ev) - 1;
        const int64_t t = t0 + k;
        const int tx = (int)((fired >> k) & 1u);
        const bool last = k == B - 1;
        RowInfo ri = RowInfo{};
        int ok = 0;
        if (prow) {
            ok = make_row_info_d(ri, i, t, tlw, rs, pend_k, xp, tx, H,
                                 lst.dpow[row_age_index(t, tlw, H)], lst.err);
            if (ok) {
                tlw = (int)t;
                xp = ri.xp_now;
                n_rows += 1;
                n_syn += ri.len;
                if (!tx) {
                    n_forced += 1;
                    n_fsyn += ri.len;
                }
            }
        }
        if (tx) {
            if (!ok) {  // nothing to bring up to date: the row is only delivered
                ri = RowInfo{};
                ri.k = i;
                ri.rs = rs;
            }
            int pos = s_lb[2 * k] + __popcll(s_m[k][wave] & below);
            for (int w = 0; w < wave; ++w) pos += __popcll(s_m[k][w]);
            // (only a failed scan puts a position out of range)
            if (pos < n) {
                (last ? lst.ring : b.tx + (int64_t)k * n)[pos] = i;
                (last ? lst.txinfo : b.txinfo + (int64_t)k * n)[pos] = ri;
            } else {
                atomicOr(lst.err, kErrRing);
            }
        } else {
            int pos = s_lb[2 * k + 1] + __popcll(s_f[k][wave] & below);
            for (int w = 0; w < wave; ++w) pos += __popcll(s_f[k][w]);
            if (pos < npl) {
                (last ? lst.row_list : b.rows + (int64_t)k * npl)[pos] = i;
                (last ? lst.info : b.info + (int64_t)k * npl)[pos] = ri;
            } else {
                atomicOr(lst.err, kErrRing);
            }
        }
    }
    if (lst.info_stats) {
        n_rows = wave_sum_i64(n_rows);
        n_forced = wave_sum_i64(n_forced);
        n_syn = wave_sum_i64(n_syn);
        n_fsyn = wave_sum_i64(n_fsyn);
        if (lane == 0) {
            if (n_rows) atomicAdd(s_st + 0, (unsigned long long)n_rows);
            if (n_forced) atomicAdd(s_st + 1, (unsigned long long)n_forced);
            if (n_syn) atomicAdd(s_st + 2, (unsigned long long)n_syn);
            if (n_fsyn) atomicAdd(s_st + 3, (unsigned long long)n_fsyn);
        }
        __syncthreads();  // s_st complete
        if (tid < 4 && s_st[tid]) {
            int64_t *sl = lst.info_stats + (int64_t)(blockIdx.x % b.info_slots) * kStFields;
            const int f = tid == 0 ? kStRows : tid == 1 ? kStForced : tid == 2 ? kStSyn
                                                                                : kStForcedSyn;
            add_stat(sl + f, (long long)s_st[tid]);
        }
    }
    // copies of the clock as the passes before the last expect it
    if (blockIdx.x == 0 && tid < B - 1) {
        StepClock c = ck;
        c.t = t0 + tid + 1;
        b.clk[tid] = c;
    }
    if (blockIdx.x == gridDim.x - 1) {
        // every workgroup has read the clock: the scans saw all of them
        if (tid < B) {
            const int cs = s_lb[2 * tid] + own_s, cf = s_lb[2 * tid + 1] + own_f;
            if (tid == B - 1) {
                lst.ring_cnt[0] = cs;
                *lst.tx_cnt = cs;
                *lst.row_cnt = cf;
            } else {
                b.cnt[2 * tid] = cs;
                b.cnt[2 * tid + 1] = cf;
            }
            add_stat(lst.gstats + kGSpikes, cs);
        }
        if (tid == 0) {
            add_stat(lst.gstats + kGSteps, B);
            a.clk->t = t0 + B;
        }
    }
}

// Positions of the delay-ring entries: grid (ceil(n / kBlock), d).
__global__ __launch_bounds__(kBlock) void k_ring_positions(const int32_t *ring,
                                                           const int32_t *cnt, int32_t *pos,
                                                           int32_t n)
{
    const int q = blockIdx.y;
    const int r = blockIdx.x * kBlock + threadIdx.x;
    if (r >= min(max(cnt[q], 0), n)) return;
    const int k = ring[(int64_t)q * n + r];
    if (k >= 0 && k < n) pos[(int64_t)q * n + k] = r;
}

// The fp32 input the next neuron update would compute from the partial sums
// (nothing when the clock says it reads the fp32 input already).
__global__ __launch_bounds__(kBlock) void k_materialize_input(const long long *apart,
                                                              int64_t stride,
                                                              const StepClock *clk, float *ain,
                                                              int64_t count)
{
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const StepClock ck = *clk;
    if (i >= count || ck.input_forced) return;
    long long v = apart[i];
    for (int c = 1; c < ck.n_parts; ++c) v += apart[c * stride + i];
    ain[i] = from_fix(v);
}

// Sets the clock: step t unless t < 0, the input source unless
// input_forced < 0.
__global__ void k_set_clock(StepClock *clk, int64_t t, int32_t input_forced, int32_t n_parts)
{
    if (threadIdx.x != 0) return;
    if (t >= 0) clk->t = t;
    if (input_forced >= 0) {
        clk->input_forced = input_forced;
        clk->n_parts = n_parts;
    }
}

template <int M, int H>
hipError_t launch_steps(hipStream_t s, const NeuronArgs &a, const BatchArgs &b)
{
    hipLaunchKernelGGL((k_neuron_steps<M, H>), dim3(blocks_for(a.n, kStepsBlock)),
                       dim3(kStepsBlock), 0, s, a, b);
    return hipGetLastError();
}

template <int M, int H>
hipError_t launch_small(hipStream_t s, const NeuronArgs &a, const SmallArgs &b, size_t lds,
                        KernelEvents ev)
{
    static std::mutex mu;
    static int granted = 48 * 1024;
    const hipError_t e =
        allow_dynamic_lds((const void *)k_small_steps<M, H>, (int)lds, mu, granted);
    if (e != hipSuccess) return e;
    launch_kernel(k_small_steps<M, H>, dim3(1), dim3(kSmallBlock), lds, s, ev, a, b);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_init_state(hipStream_t s, float *v, int32_t *ref, float *ie, float *ii,
                             uint64_t *hist, float *ypost, int32_t *t_last, float *xpre,
                             int32_t n, int32_t hw)
{
    hipLaunchKernelGGL(k_init_state, dim3(blocks_for(n)), dim3(kBlock), 0, s, v, ref, ie, ii,
                       hist, ypost, t_last, xpre, n, hw);
    return hipGetLastError();
}

hipError_t launch_fill_f32(hipStream_t s, float *p, int64_t count, float value)
{
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill<float>, dim3(blocks_for(count, kBlock, 4096)), dim3(kBlock), 0,
                       s, p, count, value);
    return hipGetLastError();
}

hipError_t launch_fill_i64(hipStream_t s, int64_t *p, int64_t count, int64_t value)
{
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill<int64_t>, dim3(blocks_for(count, kBlock, 4096)), dim3(kBlock),
                       0, s, p, count, value);
    return hipGetLastError();
}

hipError_t launch_fill_i32(hipStream_t s, int32_t *p, int64_t count, int32_t value)
{
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill<int32_t>, dim3(blocks_for(count, kBlock, 4096)), dim3(kBlock),
                       0, s, p, count, value);
    return hipGetLastError();
}

hipError_t launch_fill_ll(hipStream_t s, long long *p, int64_t count, long long value)
{
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_fill<long long>, dim3(blocks_for(count, kBlock, 4096)), dim3(kBlock),
                       0, s, p, count, value);
    return hipGetLastError();
}

hipError_t launch_copy_bytes(hipStream_t s, void *dst, const void *src, int64_t bytes)
{
    if (bytes <= 0) return hipSuccess;
    return hipMemcpyAsync(dst, src, (size_t)bytes, hipMemcpyDeviceToDevice, s);
}

hipError_t launch_small_steps(hipStream_t s, const NeuronArgs &a, const SmallArgs &b,
                              KernelEvents ev)
{
    const size_t lds = (size_t)b.nacc * a.n * sizeof(long long);
    const int m = a.model == 1 ? 1 : a.model == 2 ? 2 : 0;
    switch (m * 2 + (a.hw == 2)) {
    case 0: return launch_small<0, 1>(s, a, b, lds, ev);
    case 1: return launch_small<0, 2>(s, a, b, lds, ev);
    case 2: return launch_small<1, 1>(s, a, b, lds, ev);
    case 3: return launch_small<1, 2>(s, a, b, lds, ev);
    case 4: return launch_small<2, 1>(s, a, b, lds, ev);
    default: return launch_small<2, 2>(s, a, b, lds, ev);
    }
}

hipError_t launch_neuron_steps(hipStream_t s, const NeuronArgs &a, const BatchArgs &b)
{
    const int m = a.model == 1 ? 1 : a.model == 2 ? 2 : 0;
    if (b.steps < 1 || b.steps > batch_steps_max(m)) return hipErrorInvalidValue;
    switch (m * 2 + (a.hw == 2)) {
    case 0: return launch_steps<0, 1>(s, a, b);
    case 1: return launch_steps<0, 2>(s, a, b);
    case 2: return launch_steps<1, 1>(s, a, b);
    case 3: return launch_steps<1, 2>(s, a, b);
    case 4: return launch_steps<2, 1>(s, a, b);
    default: return launch_steps<2, 2>(s, a, b);
    }
}

hipError_t launch_neuron(hipStream_t s, const NeuronArgs &a, const CompactArgs &c,
                         KernelEvents ev)
{
    if (a.n <= kNeuronSmallN)
        launch_kernel(k_neuron<kBlock>, dim3(blocks_for(a.n, kBlock)), dim3(kBlock), 0, s, ev,
                      a, c);
    else
        launch_kernel(k_neuron<kNeuronBlock>, dim3(blocks_for(a.n, kNeuronBlock)),
                      dim3(kNeuronBlock), 0, s, ev, a, c);
    return hipGetLastError();
}

hipError_t launch_source_steps(hipStream_t s, const NeuronArgs &a, const CompactArgs &c,
                               const SourceArgs &b, KernelEvents ev)
{
    if (b.steps < 1 || b.steps > kSrcMaxSteps || a.model != 2 || c.delay != 1 ||
        c.n_plastic_rows < 1 || c.n_plastic_rows > a.n || (a.hw != 1 && a.hw != 2) ||
        b.info_slots < 1 || b.status_stride < source_steps_grid(a.n) || c.segb)
        return hipErrorInvalidValue;
    if (a.hw == 2)
        launch_kernel(k_source_steps<2>, dim3(source_steps_grid(a.n)), dim3(kStepsBlock), 0, s,
                      ev, a, c, b);
    else
        launch_kernel(k_source_steps<1>, dim3(source_steps_grid(a.n)), dim3(kStepsBlock), 0, s,
                      ev, a, c, b);
    return hipGetLastError();
}

int source_steps_grid(int32_t n) { return blocks_for(n, kStepsBlock); }

int neuron_grid(int32_t n) { return blocks_for(n, n <= kNeuronSmallN ? kBlock : kNeuronBlock); }
int neuron_steps_grid(int32_t n) { return blocks_for(n, kStepsBlock); }

hipError_t launch_ring_positions(hipStream_t s, const int32_t *ring, const int32_t *cnt,
                                 int32_t *pos, int32_t n, int32_t d)
{
    hipLaunchKernelGGL(k_ring_positions, dim3(blocks_for(n), d), dim3(kBlock), 0, s, ring, cnt,
                       pos, n);
    return hipGetLastError();
}

hipError_t launch_materialize_input(hipStream_t s, const long long *apart, int64_t part_stride,
                                    StepClock *clk, float *ain, int64_t count)
{
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_materialize_input, dim3(blocks_for(count)), dim3(kBlock), 0, s, apart,
                       part_stride, clk, ain, count);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_set_clock(s, clk, -1, 1, 1);
}

hipError_t launch_set_clock(hipStream_t s, StepClock *clk, int64_t t, int32_t input_forced,
                            int32_t n_parts)
{
    hipLaunchKernelGGL(k_set_clock, dim3(1), dim3(kWave), 0, s, clk, t, input_forced, n_parts);
    return hipGetLastError();
}

}  // namespace snn
