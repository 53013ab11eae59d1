// gfx950 kernels of the neuron part of a step: state initialisation and
// fills, and the neuron update (firing masks, histories, post traces) that
// also builds the spike / transmitted / forced lists with row snapshots.
//
// Built with -ffp-contract=off: the neuron update must reproduce a fixed
// fp32 operation order, so no multiply-add is ever fused.
#include "snn_device.h"

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
// (1) neuron update, one wave64 per mask word and kNeuronRounds neurons per
// thread, and the lists of the step: spikes (into the delay ring), forced
// plastic rows and the snapshots of the rows to bring up to date (see
// CompactArgs).
//
// List offsets: each workgroup reserves its stretch of the spike list and of
// the forced-row list with ONE 64-bit atomic on a packed word (spikes in bits
// 0-23, forced rows in bits 24-47, a workgroup ticket in bits 48-63; counts
// stay below n < 2^24). Same-address device-scope atomics serialise, so a
// workgroup covers many neurons (fewer reservations). The workgroup whose ticket comes
// last holds every other contribution in the returned value: it publishes
// the counts and clears the word for the next step. Transmitting rows need
// no reservation: a row transmitting at t spiked at t-D+1, when its position
// in that step's spike list was recorded (spk_pos); its snapshot goes to the
// same position, so snapshots line up with the delay-ring list delivery reads.

// A neuron's state as one update reads and writes it: potential,
// refractory count, CUBA currents, post trace and history words.
struct NState {
    float v, ie, ii, y;
    int r;
    uint64_t h0, h1;
};

// M >= 0 fixes the neuron model at compile time for a network without
// plasticity (the small-network kernel); M < 0 reads both from the arguments.
// H > 0 fixes the history width in words the same way.
template <int M>
__device__ __forceinline__ int nmodel(const NeuronArgs &a) { return M >= 0 ? M : a.model; }
template <int M>
__device__ __forceinline__ bool nplastic(const NeuronArgs &a)
{
    return M >= 0 ? false : a.n_plastic_rows > 0;
}
template <int H>
__device__ __forceinline__ int nhw(const NeuronArgs &a) { return H > 0 ? H : a.hw; }

template <int M, int H>
__device__ __forceinline__ void nstate_load(const NeuronArgs &a, int i, NState &st)
{
    st.v = st.ie = st.ii = st.y = 0.f;
    st.r = 0;
    if (nmodel<M>(a) != 2) {
        st.v = a.v[i];
        st.r = a.ref[i];
        if (nmodel<M>(a) == 1) {
            st.ie = a.ie[i];
            st.ii = a.ii[i];
        }
    }
    const uint64_t *hp = a.hist + (int64_t)i * nhw<H>(a);
    st.h0 = hp[0];
    st.h1 = nhw<H>(a) == 2 ? hp[1] : 0ull;
    if (nplastic<M>(a)) st.y = a.ypost[i];
}

template <int M, int H>
__device__ __forceinline__ void nstate_store(const NeuronArgs &a, int i, const NState &st)
{
    if (nmodel<M>(a) != 2) {
        a.v[i] = st.v;
        a.ref[i] = st.r;
        if (nmodel<M>(a) == 1) {
            a.ie[i] = st.ie;
            a.ii[i] = st.ii;
        }
    }
    uint64_t *hp = a.hist + (int64_t)i * nhw<H>(a);
    hp[0] = st.h0;
    if (nhw<H>(a) == 2) hp[1] = st.h1;
    if (nplastic<M>(a)) a.ypost[i] = st.y;
}

// The input A(t) of neuron i from the state: the fp32 input, or the sum of
// the fixed-point partial sums of delivery.
__device__ __forceinline__ void neuron_input(const NeuronArgs &a, int i, float &ae, float &ai)
{
    ai = 0.f;
    if (a.input_forced) {
        ae = a.ain[i];
        if (a.model == 1) ai = a.ain[a.n + i];
    } else {
        long long se = a.apart[i];
        for (int c = 1; c < a.n_parts; ++c) se += a.apart[c * a.part_stride + i];
        ae = from_fix(se);
        if (a.model == 1) {
            long long si = a.apart[a.n + i];
            for (int c = 1; c < a.n_parts; ++c) si += a.apart[c * a.part_stride + a.n + i];
            ai = from_fix(si);
        }
    }
}

// The external Poisson count of neuron i at step t: the number of CDF
// thresholds at or below one 32-bit draw (inversion). Unrolled over the
// table's capacity, so the thresholds are loaded once, not waited for inside
// a loop.
__device__ __forceinline__ int poisson_count(const NeuronArgs &a, int64_t t, int i)
{
    const uint32_t u = rng32(a.seed, 3, (uint64_t)t, (uint64_t)i);
    int k = 0;
#pragma unroll
    for (int q = 0; q < kMaxPoisson; ++q)
        if (q < a.poisson_len) k += (a.poisson[q] <= u);
    return k;
}

// One neuron's update at step t (i < n) on its state in registers, with
// input (ae, ai): its dynamics in a fixed fp32 operation order, its post
// trace and its history words. Returns whether it spiked.
template <int M, int H>
__device__ __forceinline__ int neuron_advance(const NeuronArgs &a, int i, int64_t t, float ae,
                                              float ai, NState &st)
{
    int s = 0;
    if (nmodel<M>(a) == 2) {
        s = rng32(a.seed, 4, (uint64_t)t, (uint64_t)i) < a.fire_thr;
    } else {
        float v = st.v;
        int r = st.r;
        if (nmodel<M>(a) == 1) {
            const float ie = __fadd_rn(__fmul_rn(st.ie, a.d_e), ae);
            const float ii = __fadd_rn(__fmul_rn(st.ii, a.d_i), ai);
            st.ie = ie;
            st.ii = ii;
            if (r > 0) {
                r -= 1;
                v = a.v_reset;
            } else {
                float x = __fsub_rn(a.v_inf, v);
                x = __fadd_rn(x, ie);
                x = __fadd_rn(x, ii);
                v = __fadd_rn(v, __fmul_rn(x, a.k_m));
                if (v >= a.v_th) {
                    s = 1;
                    v = a.v_reset;
                    r = a.ref_steps;
                }
            }
        } else {
            if (r > 0) {
                r -= 1;
                v = a.v_reset;
            } else {
                float x = 0.f;
                if (a.poisson_len > 0) {
                    x = __fmul_rn(a.j_ext, (float)poisson_count(a, t, i));
                }
                const float d = __fsub_rn(a.v_inf, v);
                const float b = __fmul_rn(d, a.k_m);
                const float c = __fadd_rn(v, b);
                v = __fadd_rn(c, ae);
                v = __fadd_rn(v, x);
                if (v >= a.v_th) {
                    s = 1;
                    v = a.v_reset;
                    r = a.ref_steps;
                }
            }
        }
        st.v = v;
        st.r = r;
    }
    if (nplastic<M>(a)) {
        // post trace seen by a pre spike at step t: posts strictly before t
        st.y = __fmul_rn(__fadd_rn(st.y, (float)(st.h0 & 1ull)), a.d_minus);
    }
    st.h1 = nhw<H>(a) == 2 ? (st.h1 << 1) | (st.h0 >> 63) : 0ull;
    st.h0 = (st.h0 << 1) | (uint64_t)s;
    return s;
}

// History code for the row-wise STDP: the position + 1 of the only spike of
// the last 64 hw steps (bit b = step t-b), 0 for none, kCodeMulti for more.
__device__ __forceinline__ uint8_t hist_code(uint64_t h0, uint64_t h1)
{
    const int np = __popcll(h0) + __popcll(h1);
    const int pos = h0 ? __ffsll((long long)h0) : 64 + __ffsll((long long)h1);
    return np == 0 ? (uint8_t)0 : np == 1 ? (uint8_t)pos : kCodeMulti;
}

// The whole update of neuron i at step t from and to the state arrays;
// returns spiked / transmitting / forced.
__device__ __forceinline__ void neuron_update(const NeuronArgs &a, int i, int64_t t, int &s,
                                              int &tx, int &forced, bool &fired_recently)
{
    NState st;
    nstate_load<-1, 0>(a, i, st);
    float ae = 0.f, ai = 0.f;
    if (a.model != 2) neuron_input(a, i, ae, ai);
    s = neuron_advance<-1, 0>(a, i, t, ae, ai, st);
    nstate_store<-1, 0>(a, i, st);
    a.code[i] = hist_code(st.h0, st.h1);
    fired_recently = (st.h0 | st.h1) != 0ull;
    tx = (int)((st.h0 >> a.dm1) & 1ull);
    if (i < a.n_plastic_rows) forced = !tx && (t - (int64_t)a.t_last[i] >= 64 * a.hw);
}

// NB threads per workgroup: 1024 on large networks (one list reservation
// per workgroup; same-address atomics serialise), 256 up to kNeuronSmallN
// neurons, where 1024 would leave most CUs without a workgroup.
template <int NB>
__global__ __launch_bounds__(NB) void k_neuron(NeuronArgs a, CompactArgs lst)
{
    // (n < 2^24 neurons with 1024 threads, at most kNeuronSmallN with fewer)
    static_assert((NB == kNeuronBlock ? (1 << 24) : kNeuronSmallN) / (NB * kNeuronRounds) <=
                      65536,
                  "workgroup ticket must fit in 16 bits");
    constexpr int NWV = NB / kWave;
    constexpr int R = kNeuronRounds;
    __shared__ int s_cnt[2][R * NWV];
    __shared__ unsigned long long s_st[4];
    __shared__ unsigned long long s_base;
    const int tid = threadIdx.x;
    const int wave = tid / kWave, lane = tid % kWave;
    const bool plastic = lst.n_plastic_rows > 0;
    if (tid < 4) s_st[tid] = 0ull;
    // The values a row snapshot needs are loaded with the neuron's own state
    // for every plastic neuron (first edge for every neuron when there is
    // plasticity), so that the few snapshots taken below cost no second
    // dependent round trip.
    int64_t v_rs[R];
    int v_pend[R], v_tl[R];
    float v_xp[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int i = (blockIdx.x * R + r) * NB + tid;
        v_rs[r] = 0;
        v_pend[r] = v_tl[r] = 0;
        v_xp[r] = 0.f;
        if (plastic && i < a.n) {
            v_rs[r] = lst.row_ptr[i];
            if (i < lst.n_plastic_rows) {
                v_pend[r] = lst.pend[i];
                v_tl[r] = lst.t_last[i];
                v_xp[r] = lst.xpre[i];
            }
        }
    }
    // round r covers neurons [(b R + r) B, (b R + r + 1) B) of workgroup b
    int s[R], tx[R], forced[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int i = (blockIdx.x * R + r) * NB + tid;
        s[r] = tx[r] = forced[r] = 0;
        bool fired_recently = false;
        if (i < a.n) neuron_update(a, i, a.t, s[r], tx[r], forced[r], fired_recently);
        const uint64_t m = ballot64(s[r]), txm = ballot64(tx[r]), fm = ballot64(forced[r]);
        const uint64_t rcm = ballot64(fired_recently);
        if (lane == 0) {
            const int64_t word = (int64_t)(blockIdx.x * R + r) * NWV + wave;
            if (word * kWave < a.n) {
                a.mask[word] = m;
                a.txmask[word] = txm;
                a.recent[word] = rcm;
            }
            s_cnt[0][r * NWV + wave] = __popcll(m);
            s_cnt[1][r * NWV + wave] = __popcll(fm);
        }
    }
    // snapshots of the rows to bring up to date (taken before any kernel
    // commits t_last / x_pre), and the position of a transmitting row in the
    // spike list of step t-D+1; their loads overlap the barrier and the
    // reservation below
    RowInfo ri[R];
    int ri_ok[R], txpos[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int i = (blockIdx.x * R + r) * NB + tid;
        ri[r] = RowInfo{};
        ri_ok[r] = 0;
        txpos[r] = -1;
        // the row transmits at t exactly when tx (history bit D-1 of step t)
        if (tx[r] && plastic) {
            if (lst.dm1 > 0) txpos[r] = lst.tx_pos[i];
            if (i < lst.n_plastic_rows)
                ri_ok[r] = make_row_info_v(ri[r], i, lst.t, v_tl[r], v_rs[r], v_pend[r],
                                           v_xp[r], 1, lst.hw, lst.dpow, lst.err);
            if (!ri_ok[r]) {  // nothing to bring up to date: the row is only delivered
                ri[r] = RowInfo{};
                ri[r].k = i;
                ri[r].rs = v_rs[r];
            }
        } else if (forced[r]) {
            ri_ok[r] = make_row_info_v(ri[r], i, lst.t, v_tl[r], v_rs[r], v_pend[r], v_xp[r], 0,
                                       lst.hw, lst.dpow, lst.err);
        }
    }
    __syncthreads();  // publishes s_cnt, s_st
    if (tid == 0) {
        int spk = 0, fr = 0;
#pragma unroll
        for (int q = 0; q < R * NWV; ++q) {
            spk += s_cnt[0][q];
            fr += s_cnt[1][q];
        }
        const unsigned long long mine =
            (unsigned long long)spk | ((unsigned long long)fr << 24) | (1ull << 48);
        const unsigned long long old = atomicAdd(lst.acc, mine);
        s_base = old;
        if ((int)(old >> 48) == (int)gridDim.x - 1) {
            const int n_spk = (int)(old & 0xffffffull) + spk;
            const int n_forced = (int)((old >> 24) & 0xffffffull) + fr;
            (void)atomicExch(lst.acc, 0ull);
            *lst.spk_cnt = n_spk;
            *lst.row_cnt = n_forced;
            lst.gstats[kGSpikes] += n_spk;
        }
    }
    if (lst.info_stats) {
        long long v0 = 0, v1 = 0, v2 = 0, v3 = 0;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const bool f = forced[r] && ri_ok[r];
            v0 += ri_ok[r] ? 1 : 0;
            v1 += f ? 1 : 0;
            v2 += ri_ok[r] ? ri[r].len : 0;
            v3 += f ? ri[r].len : 0;
        }
        v0 = wave_sum_i64(v0);
        v1 = wave_sum_i64(v1);
        v2 = wave_sum_i64(v2);
        v3 = wave_sum_i64(v3);
        if (lane == 0) {
            if (v0) atomicAdd(s_st + 0, (unsigned long long)v0);
            if (v1) atomicAdd(s_st + 1, (unsigned long long)v1);
            if (v2) atomicAdd(s_st + 2, (unsigned long long)v2);
            if (v3) atomicAdd(s_st + 3, (unsigned long long)v3);
        }
    }
    __syncthreads();  // publishes s_base, s_st
    const unsigned long long base = s_base;
    const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
    int o0 = (int)(base & 0xffffffull), o2 = (int)((base >> 24) & 0xffffffull);
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int i = (blockIdx.x * R + r) * NB + tid;
        // this wave's offsets in round r: every wave of the earlier rounds,
        // then the earlier waves of this one
        int p0 = o0, p2 = o2;
        for (int q = 0; q < r * NWV + wave; ++q) {
            p0 += s_cnt[0][q];
            p2 += s_cnt[1][q];
        }
        const uint64_t m = ballot64(s[r]), fm = ballot64(forced[r]);
        // (the bounds checks only catch an accumulator left non-zero by a
        // failed step; with a cleared one every offset is in range)
        if (s[r]) {
            const int pos = p0 + __popcll(m & below);
            if (pos < a.n) {
                lst.spk_list[pos] = i;
                if (plastic && lst.dm1 > 0) lst.spk_pos[i] = pos;
                if (lst.dm1 == 0) txpos[r] = pos;  // D = 1: transmitted as it fires
            } else {
                atomicOr(lst.err, kErrRing);
            }
        }
        if (tx[r] && plastic) {
            if (txpos[r] >= 0 && txpos[r] < a.n)
                lst.txinfo[txpos[r]] = ri[r];
            else
                atomicOr(lst.err, kErrRing);
        }
        if (forced[r]) {
            const int q = p2 + __popcll(fm & below);
            if (q < lst.n_plastic_rows) {
                lst.row_list[q] = i;
                lst.info[q] = ri[r];
            } else {
                atomicOr(lst.err, kErrRing);
            }
        }
    }
    if (lst.info_stats && tid == 0) {
        int64_t *slot = lst.info_stats + (int64_t)blockIdx.x * kStFields;
        slot[kStRows] += (int64_t)s_st[0];
        slot[kStForced] += (int64_t)s_st[1];
        slot[kStSyn] += (int64_t)s_st[2];
        slot[kStForcedSyn] += (int64_t)s_st[3];
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
    long long events = 0, spikes = 0;
    NState st[kSmallRounds];
#pragma unroll
    for (int r = 0; r < kSmallRounds; ++r) {
        const int i = r * kSmallBlock + tid;
        if (r < rounds && i < n) nstate_load<M, H>(a, i, st[r]);
    }
    for (int k = 0; k < b.steps; ++k) {
        const int64_t t = a.t + k;
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
                        neuron_input(a, i, ae, ai);
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
    if (lane == 0 && events) atomicAdd((unsigned long long *)b.dlv_stats, (unsigned long long)events);
    if (tid == 0) b.gstats[kGSpikes] += spikes;
}

// ---------------------------------------------------------------------------
// Delay block of a network without plasticity: b.steps (<= D-1) steps of the
// neuron update, one neuron per thread with its state in registers. Step
// a.t reads its input like k_neuron (forced input or the partial sums in
// apart); step a.t + k, k >= 1, reads slot k-1 of abatch, the whole input
// as one fixed-point sum, written beforehand by the batched delivery. Every
// slot's load is issued before the first step, so the steps wait for one
// round trip in all. The spike flags of every step are kept (a bit per step
// per thread, ballots in LDS), and the spike lists go into the delay ring at
// the end: one packed reservation per workgroup and step (counts in bits
// 0-23, a ticket in bits 48-63; the workgroup whose ticket comes last
// publishes the count and clears the word), the B reservations of a
// workgroup in flight together. The masks, codes and the state written are
// those of the last step, and apart part 0 receives slot B-1, the pending
// input of the next step. Workgroups of 512 threads: the B steps of a
// thread run one after another, so fewer waves share a SIMD than with 1024,
// and half as many reservations queue per step as with 256.
constexpr int kStepsBlock = 512;
static_assert((1 << 24) / kStepsBlock <= 65536, "workgroup ticket must fit in 16 bits");
template <int M, int H>
__global__ __launch_bounds__(kStepsBlock) void k_neuron_steps(NeuronArgs a, BatchArgs b)
{
    constexpr int NWV = kStepsBlock / kWave;
    __shared__ uint64_t s_m[kBatchMax][NWV];
    __shared__ int s_off[kBatchMax];
    const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
    const int n = a.n;
    const int i = blockIdx.x * kStepsBlock + tid;
    const bool live = i < n;
    const int ic = live ? i : 0;
    const int64_t ps = a.part_stride;  // nacc * n
    // steps per launch: CUBA holds two inputs per step in registers
    constexpr int KB = batch_steps_max(M);
    const int B = b.steps;  // 1 .. KB (checked by the launcher)
    // slot k = input of step a.t + k + 1 (Bernoulli sources read only the
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
                neuron_input(a, i, ae, ai);
            } else {
                ae = from_fix(pe[k - 1]);
                if (M == 1) ai = from_fix(pi[k - 1]);
            }
        }
        int sp = 0;
        if (live) sp = neuron_advance<M, H>(a, i, a.t + k, ae, ai, st);
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
    if (tid < B) {
        const int k = tid;
        int cnt = 0;
        for (int w = 0; w < NWV; ++w) cnt += __popcll(s_m[k][w]);
        const unsigned long long old =
            atomicAdd(b.acc + k * kAccStride, (unsigned long long)cnt | (1ull << 48));
        s_off[k] = (int)(old & 0xffffffull);
        if ((int)(old >> 48) == (int)gridDim.x - 1) {
            const int total = (int)(old & 0xffffffull) + cnt;
            (void)atomicExch(b.acc + k * kAccStride, 0ull);
            const int64_t d = b.delay;
            b.ring_cnt[(int)((a.t + k) % d)] = total;
            atomicAdd((unsigned long long *)(b.gstats + kGSpikes), (unsigned long long)total);
        }
    }
    __syncthreads();  // every offset
    const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
    for (int k = 0; k < B; ++k) {
        if (!((fired >> k) & 1u)) continue;
        int pos = s_off[k] + __popcll(s_m[k][wave] & below);
        for (int w = 0; w < wave; ++w) pos += __popcll(s_m[k][w]);
        // (only an accumulator left non-zero by a failed launch is out of range)
        if (pos < n)
            b.ring[(int64_t)((a.t + k) % b.delay) * n + pos] = i;
        else
            atomicOr(b.err, kErrRing);
    }
}

// Sorts a list of distinct neuron indices (capacity n entries, values in
// [0, n)) into ascending order (one workgroup; not on the step's path):
// scatter into a bitmap of nw = ceil(n/64) words, then read it back in order.
// Entries past min(*cnt, n) are not read; out-of-range values are dropped.
// With pos, records each index's new position.
constexpr int kSortListBlock = 1024;
__global__ __launch_bounds__(kSortListBlock) void k_sort_list(int32_t *list, const int32_t *cnt,
                                                              uint64_t *bitmap, int32_t *pos,
                                                              int32_t n, int32_t nw)
{
    __shared__ long long sh[kSortListBlock / kWave];
    const int tid = threadIdx.x;
    const int len = min(max(*cnt, 0), n);
    for (int q = tid; q < nw; q += kSortListBlock) bitmap[q] = 0ull;
    __syncthreads();
    for (int q = tid; q < len; q += kSortListBlock) {
        const int k = list[q];
        if (k >= 0 && k < n)
            atomicOr((unsigned long long *)(bitmap + (k >> 6)), 1ull << (k & 63));
    }
    __syncthreads();
    long long done = 0;
    for (int w0 = 0; w0 < nw; w0 += kSortListBlock) {
        const int wi = w0 + tid;
        // agent-scope loads: the bits were set by atomics at L2
        const uint64_t bits =
            wi < nw ? __hip_atomic_load(bitmap + wi, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                    : 0ull;
        const long long incl = block_incl_scan_i64_n<kSortListBlock>(__popcll(bits), sh);
        int o = (int)(done + incl - __popcll(bits));
        for (uint64_t b = bits; b; b &= b - 1, ++o) {
            const int k = wi * 64 + __ffsll((long long)b) - 1;
            list[o] = k;
            if (pos) pos[k] = o;
        }
        done += block_sum_i64_n<kSortListBlock>(__popcll(bits), sh);
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

// The fp32 input the next neuron update would compute from the partial sums.
__global__ __launch_bounds__(kBlock) void k_materialize_input(const long long *apart,
                                                              int64_t stride, int32_t parts,
                                                              float *ain, int64_t count)
{
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    if (i >= count) return;
    long long v = apart[i];
    for (int c = 1; c < parts; ++c) v += apart[c * stride + i];
    ain[i] = from_fix(v);
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
    hipExtLaunchKernelGGL(k_small_steps<M, H>, dim3(1), dim3(kSmallBlock), lds, s, ev.start,
                          ev.stop, 0, a, b);
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
    if (a.n <= kNeuronSmallN) {
        constexpr int NB = kBlock;
        hipExtLaunchKernelGGL(k_neuron<NB>, dim3(blocks_for(a.n, NB * kNeuronRounds)), dim3(NB),
                              0, s, ev.start, ev.stop, 0, a, c);
    } else {
        constexpr int NB = kNeuronBlock;
        hipExtLaunchKernelGGL(k_neuron<NB>, dim3(blocks_for(a.n, NB * kNeuronRounds)), dim3(NB),
                              0, s, ev.start, ev.stop, 0, a, c);
    }
    return hipGetLastError();
}

hipError_t launch_sort_list(hipStream_t s, int32_t *list, const int32_t *cnt, uint64_t *bitmap,
                            int32_t *pos, int32_t n)
{
    hipLaunchKernelGGL(k_sort_list, dim3(1), dim3(kSortListBlock), 0, s, list, cnt, bitmap, pos, n,
                       (n + 63) / 64);
    return hipGetLastError();
}

hipError_t launch_ring_positions(hipStream_t s, const int32_t *ring, const int32_t *cnt,
                                 int32_t *pos, int32_t n, int32_t d)
{
    hipLaunchKernelGGL(k_ring_positions, dim3(blocks_for(n), d), dim3(kBlock), 0, s, ring, cnt,
                       pos, n);
    return hipGetLastError();
}

hipError_t launch_materialize_input(hipStream_t s, const long long *apart, int64_t part_stride,
                                    int32_t n_parts, float *ain, int64_t count)
{
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_materialize_input, dim3(blocks_for(count)), dim3(kBlock), 0, s, apart,
                       part_stride, n_parts, ain, count);
    return hipGetLastError();
}

}  // namespace snn
