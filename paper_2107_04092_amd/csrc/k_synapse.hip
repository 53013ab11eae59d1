// gfx950 kernels of the synapse pass: row snapshots for a flush, lazy +
// event-driven STDP (slice-organised and row-wise layouts), slice delivery
// with LDS accumulation and the transmitting rows' plasticity fused in, and
// the global-atomic delivery variant.
#include "snn_device.h"

namespace snn {
namespace {

// ---------------------------------------------------------------------------
// (2) lazy + event-driven STDP (Sec. III-A, Fig. 2(b,c)).
//
// Row k was last brought up to date at step t_last; its age is t - t_last
// (1..64). For synapse k->j the post spikes in the window are the set bits
// age-1..0 of hist[j] (bit i = spike at step t-i); they are visited oldest
// first via count-leading-zeros, each potentiating with the pre trace
// decayed to its step (x_pre(t-i) = xp0 d+^(age-i)). A row transmitting at t
// then depresses with the post trace y_j(t), and a post at t itself
// potentiates with the pre trace that includes the pre spike at t.
//
// Snapshots of every plastic row for a flush (bring all rows to step t, no
// pre-synaptic spike). During a step the neuron kernel takes them.

__global__ __launch_bounds__(kBlock) void k_row_info(RowInfoArgs a)
{
    __shared__ float s_dpow[kMaxAge + 1];
    __shared__ long long sh[kBlock / kWave];
    const int tid = threadIdx.x;
    for (int q = tid; q <= kMaxAge; q += kBlock) s_dpow[q] = a.dpow[q];
    __syncthreads();
    const int r = blockIdx.x * kBlock + tid;
    long long st_rows = 0, st_syn = 0;
    if (r < a.n_rows_all) {
        RowInfo ri;
        if (make_row_info(ri, r, a.clk->t - 1, false, a.dm1, a.hw, a.row_ptr, a.pend, a.hist, a.t_last, a.xpre,
                          s_dpow, a.err)) {
            st_rows = 1;
            st_syn = ri.len;
        }
        a.info[r] = ri;
    }
    st_rows = block_sum_i64(st_rows, sh);
    st_syn = block_sum_i64(st_syn, sh);
    if (tid == 0) {
        int64_t *slot = a.stats + (int64_t)blockIdx.x * kStFields;
        add_stat(slot + kStRows, st_rows);
        add_stat(slot + kStSyn, st_syn);
    }
}

// Slice-organised synapse pass, the STDP counterpart of slice delivery.
// Work item q = (target group g, row chunk cr); group g is the W_s = mult * W
// targets [g W_s, (g+1) W_s), so its segment of row k is entries
// piv[k][g mult] .. piv[k][(g+1) mult] of the delivery pivots. The group's
// history words and post traces are staged in LDS once; every synapse reads
// them from LDS instead of gathering them from L2 (random L2 gathers are
// bounded by the outstanding misses each CU's L1 can track). For a batch of
// rows the workgroup stages each row's segment (start, window mask, pre,
// traces) and prefix-sums the lengths; the concatenated segments are then
// walked in windows of 4 elements per thread, with an LDS map from element
// to segment, so lanes stay busy whatever the segment lengths and
// consecutive lanes read consecutive entries. Work items are dealt out so
// that each XCD gets a contiguous range of target groups. The workgroups of
// group 0 commit t_last and xpre of their rows; no workgroup reads those.

__global__ __launch_bounds__(kStdpBlock) void k_stdp(StdpArgs a)
{
    extern __shared__ unsigned char stage[];  // W_s x hw history words, then W_s post traces
    __shared__ long long s_start[kStdpBatch];
    __shared__ int s_off[kStdpBatch + 1];
    __shared__ int s_ap[kStdpBatch];
    __shared__ float s_xp0[kStdpBatch];
    __shared__ float s_xpn[kStdpBatch];
    __shared__ int s_map[kStdpWindow];
    __shared__ float s_dpow[kMaxAge + 1];
    __shared__ long long sh[kStdpBlock / kWave];
    __shared__ int shi[kStdpBlock / kWave];
    const int tid = threadIdx.x;
    const int nb = gridDim.x;  // multiple of 8
    const int q = (blockIdx.x & 7) * (nb >> 3) + (blockIdx.x >> 3);
    if (q >= a.n_work) return;  // whole workgroup, before any barrier
    const int g = q / a.chunks, cr = q - g * a.chunks;
    const int64_t t = a.clk->t - 1;
    const int nrows = a.row_cnt ? *a.row_cnt : a.n_rows_all;
    const int lo = (int)((int64_t)nrows * cr / a.chunks);
    const int hi = (int)((int64_t)nrows * (cr + 1) / a.chunks);
    if (g == 0) {
        for (int r = lo + tid; r < hi; r += kStdpBlock) {
            const RowInfo ri = a.info[r];
            if (ri.age_pre != 0) {
                a.t_last[ri.k] = (int32_t)t;
                a.xpre[ri.k] = ri.xp_now;
            }
        }
    }
    const int j0 = g * a.width;
    if (j0 >= a.target_limit) return;  // no plastic synapse targets this group (g > 0)
    const int hw = a.hw;
    uint64_t *s_hist = (uint64_t *)stage;
    float *s_y = (float *)(stage + (size_t)a.width * hw * sizeof(uint64_t));
    const int jn = min(a.width, a.n - j0);  // > 0
    stage_lds<kStdpBlock, 4>(s_hist, a.hist + (int64_t)j0 * hw, jn * hw);
    stage_lds<kStdpBlock, 4>(s_y, a.ypost + j0, jn);
    for (int x = tid; x <= kMaxAge; x += kStdpBlock) s_dpow[x] = a.dpow[x];
    const int pv_lo = g * a.mult;
    const int pv_hi = min((g + 1) * a.mult, a.n_slices);
    const int piv_stride = a.n_slices + 1;
    const int32_t *__restrict__ col = a.col;
    float *__restrict__ wgt = a.w;
    const float c_pot = a.c_pot, c_dep = a.c_dep, mu = a.mu;
    long long written = 0;
    for (int b0 = lo; b0 < hi; b0 += kStdpBatch) {
        const int nbt = min(kStdpBatch, hi - b0);
        int len = 0;
        if (tid < nbt) {
            const RowInfo ri = a.info[b0 + tid];
            if (ri.len > 0) {
                const int32_t *pv = a.piv + (int64_t)ri.k * piv_stride;
                const int p0 = pv[pv_lo];
                const int p1 = min(pv[pv_hi], ri.len);
                len = max(0, p1 - p0);
                s_start[tid] = ri.rs + p0;
                s_ap[tid] = ri.age_pre;
                s_xp0[tid] = ri.xp0;
                s_xpn[tid] = ri.xp_now;
            }
        }
        const long long incl = block_incl_scan_i64_n<kStdpBlock>(len, sh);
        if (tid < nbt) s_off[tid] = (int)(incl - len);
        if (tid == kStdpBlock - 1) s_off[nbt] = (int)incl;
        __syncthreads();
        const int total = s_off[nbt];
        for (int e0 = 0; e0 < total; e0 += kStdpWindow) {
            const int we = min(kStdpWindow, total - e0);
            for (int x = tid; x < we; x += kStdpBlock) s_map[x] = -1;
            __syncthreads();
            if (tid < nbt) {
                const int a0 = max(s_off[tid], e0), a1 = min(s_off[tid + 1], e0 + we);
                if (a0 < a1) s_map[a0 - e0] = tid;
            }
            __syncthreads();
            fill_segment_map<kStdpBlock>(s_map, we, shi);
            int jl[kStdpUnroll], slot[kStdpUnroll];
            long long gi[kStdpUnroll];
            float wv[kStdpUnroll];
            int cv[kStdpUnroll];
#pragma unroll
            for (int u = 0; u < kStdpUnroll; ++u) {
                const int x = u * kStdpBlock + tid;  // < kStdpWindow
                const int lm = s_map[x];
                const int l = x < we ? lm : 0;
                slot[u] = l;
                gi[u] = x < we ? s_start[l] + (e0 + x - s_off[l]) : 0;  // edge 0 exists
                cv[u] = col[gi[u]];
                wv[u] = wgt[gi[u]];
            }
#pragma unroll
            for (int u = 0; u < kStdpUnroll; ++u)
                jl[u] = u * kStdpBlock + tid < we ? cv[u] - j0 : -1;
#pragma unroll
            for (int u = 0; u < kStdpUnroll; ++u) {
                if (jl[u] < 0) continue;
                const int l = slot[u];
                const int ap = s_ap[l];
                const int pre = ap >> 8;
                uint64_t m0, m1;
                window_masks(ap & 0xff, m0, m1);
                const uint64_t h0 = s_hist[jl[u] * hw] & m0;
                const uint64_t h1 = hw == 2 ? s_hist[jl[u] * hw + 1] & m1 : 0ull;
                if (a.event && !h0 && !h1 && !pre) continue;  // nothing happened to it
                const float y = pre ? s_y[jl[u]] : 0.f;
                wgt[gi[u]] = a.event ? stdp_synapse(wv[u], h0, h1, ap & 0xff, pre, s_xp0[l],
                                                    s_xpn[l], y, s_dpow, c_pot, c_dep, mu)
                                     : stdp_synapse_steps(wv[u], h0, h1, ap & 0xff, pre, s_xp0[l],
                                                          s_xpn[l], y, s_dpow[1], c_pot, c_dep,
                                                          mu);
                ++written;
            }
            __syncthreads();  // map rewritten by the next window
        }
        __syncthreads();  // staging arrays are rewritten by the next batch
    }
    written = block_sum_i64_n<kStdpBlock>(written, sh);
    if (tid == 0) add_stat(a.stats + blockIdx.x, written);
}

// Row-wise layout: waves walk the rows to update in parts of up to U*64
// plastic synapses, lanes over a part's synapses in the row's own order.
// Histories and post traces come from L2 unless a per-neuron summary staged
// in LDS answers:
//   - history codes (k_neuron), when the codes of all neurons fit in LDS: a
//     synapse whose target did not fire within the window is skipped, one
//     whose target fired once takes its window bit from the code, and only
//     targets with two or more spikes have their history word gathered;
//   - else the spike-recency bitmap (1 bit per neuron: fired within the
//     window), which skips the synapses of silent targets.
// Rows with a pre spike (transmitting rows, in the global-atomic delivery
// mode) need every target's post trace and gather histories and traces.
//
// Parts start at 128-byte lines of the weight array, and a line that holds a
// changed weight is stored whole (its unchanged weights included), so the
// L2 writes no partial line back to HBM. Two parts are held per wave: the
// targets and weights of one are loaded while the other is looked up,
// updated and stored (both are in flight from the start); the next row's
// snapshot is fetched one part ahead.

constexpr uint64_t kLineMask = (1ull << kStoreLine) - 1;

template <int U>
struct RowPart {
    RowInfo ri;  // snapshot of the part's row (age_pre 0: nothing to do)
    int i;       // index in the row list (>= nrows: no part)
    int base;    // element index of lane 0 (line-aligned, may be negative)
    int j[U];    // targets (-1: no synapse)
    float w[U];  // weights
};

// History words 0 and 1 of neuron j (one 16-byte load with two words).
template <int HW>
__device__ __forceinline__ void gather_hist(const uint64_t *hist, int j, uint64_t &h0,
                                            uint64_t &h1)
{
    if (HW == 2) {
        const ulonglong2 v = ((const ulonglong2 *)hist)[j];
        h0 = v.x;
        h1 = v.y;
    } else {
        h0 = hist[j];
        h1 = 0ull;
    }
}

// Issues the loads of part p. Every lane loads from an address inside the
// row (clamped) and selects afterwards: a load whose result is used under a
// lane condition makes the compiler wait for it inside that condition, which
// would serialise the U loads of a lane.
template <int U>
__device__ __forceinline__ void rows_issue(RowPart<U> &p, const int32_t *col, const float *wgt,
                                           int lane)
{
    const int len = p.ri.age_pre != 0 ? p.ri.len : 0;
    if (len == 0) {  // wave-uniform
#pragma unroll
        for (int u = 0; u < U; ++u) {
            p.j[u] = -1;
            p.w[u] = 0.f;
        }
        return;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int q = p.base + u * kWave + lane;
        const int qc = min(max(q, 0), len - 1);
        // streaming (non-temporal) loads: the row is read once, and the
        // gathered histories stay in L2
        p.j[u] = __builtin_nontemporal_load(col + p.ri.rs + qc);
        p.w[u] = __builtin_nontemporal_load(wgt + p.ri.rs + qc);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const int q = p.base + u * kWave + lane;
        if (q < 0 || q >= len) p.j[u] = -1;
    }
}

template <int NT, int U, int HW>
__device__ __forceinline__ void stdp_rows_body(const StdpArgs &a, int bid, int nblocks,
                                               unsigned char *s_sum)
{
    __shared__ float s_dpow[kMaxAge + 1];
    const int tid = threadIdx.x;
    const int32_t *__restrict__ col = a.col;
    float *__restrict__ wgt = a.w;
    const uint64_t *__restrict__ hist = a.hist;
    const float *__restrict__ ypost = a.ypost;
    const float c_pot = a.c_pot, c_dep = a.c_dep, mu = a.mu;
    const int lane = tid % kWave;
    const int line0 = lane & ~(kStoreLine - 1);  // first lane of this lane's store line
    const int gw = (bid * NT + tid) / kWave;
    const int nwv = nblocks * (NT / kWave);
    // The prologue costs two round trips: first, together, the summary's
    // staging loads (one round of eight 8-byte loads per thread holds 32 KB:
    // the recency bitmap up to 262,144 neurons, the codes up to 32,768), the
    // row count and the first two rows' snapshots (loaded from indices
    // clamped to the snapshot array, kept only below the count); then the
    // first two parts' targets and weights.
    StageRegs<8, uint64_t> g_sum;
    const int sum_words = a.code ? (a.n + 7) / 8 : a.recent ? a.nw : 0;
    const uint64_t *sum_src = a.code ? (const uint64_t *)a.code : a.recent;
    if (sum_words > 0) stage_issue<NT>(g_sum, sum_src, sum_words);
    const int64_t t = a.clk->t - 1;
    const int nrows = a.tx_rows ? *a.tx_cnt : a.row_cnt ? *a.row_cnt : a.n_rows_all;
    long long written = 0;

    // cursor: the next part to issue (row snapshot, row-list index, base);
    // la: snapshot of the row after the cursor's
    // Work items are (row, phase) pairs, phase m in [0, P): the wave holding
    // a pair takes parts m, m + P, m + 2P, ... of the row, so a row of up to
    // P parts is spread over P waves. The cursor index counts pairs.
    const int P = a.parts;
    const int npairs = nrows * P;
    auto row_of = [&](int i) { return P == 1 ? i : i / P; };
    auto phase_of = [&](int i) { return P == 1 ? 0 : i % P; };
    RowInfo cur = a.info[min(row_of(gw), a.n_info - 1)];
    RowInfo la = a.info[min(row_of(gw + nwv), a.n_info - 1)];
    int cur_i = gw, la_i = gw + nwv;
    if (cur_i >= npairs) cur = RowInfo{};
    if (la_i >= npairs) la = RowInfo{};
    int cur_base = -(int)(cur.rs & (kStoreLine - 1)) + phase_of(cur_i) * (U * kWave);
    auto issue = [&](RowPart<U> &p) {
        p.ri = cur;
        p.i = cur_i;
        p.base = cur_base;
        rows_issue(p, col, wgt, lane);
        if (cur.age_pre != 0 && cur_base + P * U * kWave < cur.len) {  // the pair's next part
            cur_base += P * U * kWave;
        } else {  // the lookahead pair
            cur = la;
            cur_base = -(int)(la.rs & (kStoreLine - 1)) + phase_of(la_i) * (U * kWave);
            cur_i = la_i;
            la_i += nwv;
            la = RowInfo{};
            if (la_i < npairs) la = a.info[row_of(la_i)];
        }
    };
    // the first two parts go out before the staged words are stored
    RowPart<U> A, B;
    issue(A);
    issue(B);
    for (int q = tid; q <= kMaxAge; q += NT) s_dpow[q] = a.dpow[q];
    const uint8_t *s_code = s_sum;
    const uint64_t *s_recent = (const uint64_t *)s_sum;
    if (sum_words > 0) stage_finish<NT>((uint64_t *)s_sum, g_sum, sum_src, sum_words);
    __syncthreads();

    // Look-ups, update and stores of part p (the other part's loads are in
    // flight meanwhile); then p takes the next part's loads. The part's
    // candidate synapses (targets that fired within the summary's reach) are
    // appended densely to a queue of this wave in LDS (target, weight),
    // updated 64 per pass with every lane busy (all passes' history gathers
    // first, then the updates), and each owner lane takes its new weight and
    // changed flag back for the line stores: the divergent per-synapse loops
    // run over candidates only, not over every lane of every slot.
    const int tbytes = a.code ? ((a.n + 15) / 16) * 16 : a.recent ? a.nw * 8 : 0;
    int32_t *q_j = (int32_t *)(s_sum + tbytes) + (tid / kWave) * (2 * U * kWave);
    float *q_w = (float *)(q_j + U * kWave);
    auto step = [&](RowPart<U> &p) {
        const RowInfo ri = p.ri;
        const int age = ri.age_pre & 0xff, pre = ri.age_pre >> 8;
        uint64_t m0, m1;
        window_masks(age, m0, m1);
        if (HW == 1) m1 = 0ull;
        bool cand[U];
        if (!pre && a.code) {
#pragma unroll
            for (int u = 0; u < U; ++u) cand[u] = p.j[u] >= 0 && s_code[max(p.j[u], 0)] != 0;
        } else if (!pre && a.recent) {
            uint64_t rw[U];
#pragma unroll
            for (int u = 0; u < U; ++u) rw[u] = s_recent[max(p.j[u], 0) >> 6];
#pragma unroll
            for (int u = 0; u < U; ++u)
                cand[u] = p.j[u] >= 0 && ((rw[u] >> (p.j[u] & 63)) & 1ull);
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u) cand[u] = p.j[u] >= 0;
        }
        // queue offsets: wave-uniform base and ballot per slot (SGPRs); a
        // lane's entry of slot u is qb[u] + its rank among the slot's lanes
        uint64_t bl[U];
        int qb[U];
        int qn = 0;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            bl[u] = ballot64(cand[u]);
            qb[u] = qn;
            qn += (int)__popcll(bl[u]);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (cand[u]) {
                const int e = qb[u] + lane_rank(bl[u]);
                q_j[e] = p.j[u];
                q_w[e] = p.w[u];
            }
        }
        __builtin_amdgcn_wave_barrier();
        // passes of 64 entries, in two halves of U/2 passes (fewer registers
        // held); the second half runs only for more than U/2 x 64 entries
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            constexpr int H = U / 2;
            if (half * H * kWave >= qn) break;  // wave-uniform
            uint64_t h[H], g[H];
            float y[H], qw[H];
            int cd[H];
#pragma unroll
            for (int q = 0; q < H; ++q) {
                const int e0 = (half * H + q) * kWave;
                h[q] = g[q] = 0ull;
                y[q] = qw[q] = 0.f;
                cd[q] = 0;
                if (e0 < qn) {  // wave-uniform
                    const int e = e0 + lane;
                    const int j = e < qn ? q_j[e] : 0;
                    qw[q] = q_w[e];
                    if (!pre && a.code) {
                        cd[q] = s_code[j];
                        gather_hist<HW>(hist, cd[q] == kCodeMulti ? j : 0, h[q], g[q]);
                    } else {
                        gather_hist<HW>(hist, j, h[q], g[q]);
                    }
                    if (pre) y[q] = ypost[j];
                }
            }
#pragma unroll
            for (int q = 0; q < H; ++q) {
                const int e = (half * H + q) * kWave + lane;
                if (e < qn) {
                    uint64_t h0 = h[q], h1 = g[q];
                    if (!pre && a.code && cd[q] != kCodeMulti) {
                        const int ps = (cd[q] - 1) & 127;  // single spike: ps steps ago
                        h0 = ps < 64 ? 1ull << (ps & 63) : 0ull;
                        h1 = ps >= 64 ? 1ull << (ps & 63) : 0ull;
                    }
                    h0 &= m0;
                    h1 &= m1;
                    const bool chg = h0 || h1 || pre || !a.event;
                    float w = qw[q];
                    if (chg) {
                        w = a.event ? stdp_synapse(w, h0, h1, age, pre, ri.xp0, ri.xp_now, y[q],
                                                   s_dpow, c_pot, c_dep, mu)
                                    : stdp_synapse_steps(w, h0, h1, age, pre, ri.xp0,
                                                         ri.xp_now, y[q], s_dpow[1], c_pot,
                                                         c_dep, mu);
                        ++written;
                    }
                    q_w[e] = w;
                    q_j[e] = chg ? 1 : 0;
                }
            }
        }
        __builtin_amdgcn_wave_barrier();
        if (ri.age_pre != 0 && p.base == -(int)(ri.rs & (kStoreLine - 1)) && lane == 0) {  // first part
            a.t_last[ri.k] = (int32_t)t;
            a.xpre[ri.k] = ri.xp_now;
        }
        const int len = ri.age_pre != 0 ? ri.len : 0;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int e = qb[u] + lane_rank(bl[u]);  // < (u + 1) * 64: inside the queue
            const int rj = q_j[e];
            const float rw = q_w[e];
            const bool c = (bl[u] >> lane) & 1ull;
            const bool chg = c && rj != 0;
            const float w = c ? rw : p.w[u];
            const int qi = p.base + u * kWave + lane;
            const uint64_t m = ballot64(chg);
            if (((m >> line0) & kLineMask) && qi >= 0 && qi < len)
                __builtin_nontemporal_store(w, wgt + ri.rs + qi);
        }
        issue(p);
    };
    while (A.i < npairs) {
        step(A);
        if (B.i >= npairs) break;
        step(B);
    }
    // one atomic per wave: no workgroup barrier waits for the weight stores
    written = wave_sum_i64(written);
    if (lane == 0 && written)
        atomicAdd((unsigned long long *)(a.stats + bid), (unsigned long long)written);
}

// Target-range form of the forced-row update (StdpArgs::xcd): workgroup b
// runs on XCD b mod 8 and belongs to range x = (b mod 8) / (8 / xparts);
// its waves take, for every forced row, only the entries whose targets lie
// in range x of the plastic targets (the row's segment x, bounds from the
// neuron update). The targets' histories a wave gathers then stay in the
// L2 of its XCDs, and the history codes staged in LDS cover range x only.
// The host picks xparts so that a segment is about one part (U x 64
// entries); segment bounds sit on 128-byte lines of the weight array, so
// no line is stored by two ranges. Otherwise as stdp_rows_body: a
// candidate queue per wave, two parts in flight, whole lines stored.
template <int U>
struct RowPartX {
    RowInfo ri;
    int i;       // row-list index (>= nrows: no part)
    int base;    // element index of lane 0 (line-aligned)
    int s0, s1;  // the segment's entries
    int j[U];    // targets (-1: none)
    float w[U];
};

template <int NT, int U, int HW>
__device__ __forceinline__ void stdp_rows_xcd_body(const StdpArgs &a, int bid, int nblocks,
                                                   unsigned char *s_sum)
{
    __shared__ float s_dpow[kMaxAge + 1];
    constexpr int NWV = NT / kWave;
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    const int G = kXcds / a.xparts;            // XCDs per range
    const int x = (bid % kXcds) / G;           // this workgroup's range
    const int rho0 = x * G;                    // its range's first XCD
    int grp_wgs = 0;                           // workgroups of the range
    for (int q = 0; q < G; ++q) grp_wgs += (nblocks - (rho0 + q) + kXcds - 1) / kXcds;
    const int gw = ((bid / kXcds) * G + (bid % kXcds - rho0)) * NWV + wave;  // wave among the range's
    const int nwv = grp_wgs * NWV;
    const int32_t *__restrict__ col = a.col;
    float *__restrict__ wgt = a.w;
    const uint64_t *__restrict__ hist = a.hist;
    const float c_pot = a.c_pot, c_dep = a.c_dep, mu = a.mu;
    const int line0 = lane & ~(kStoreLine - 1);
    const int64_t t = a.clk->t - 1;
    const int nrows = *a.row_cnt;
    const int lo = a.xlo[x], span = a.xlo[x + 1] - lo;  // this XCD's targets
    long long written = 0;

    // cursor: the next part to issue; la: the row after the cursor's
    RowInfo cur = RowInfo{}, la = RowInfo{};
    int cur_i = gw, la_i = gw + nwv;
    int cur_s0 = 0, cur_s1 = 0, la_s0 = 0, la_s1 = 0;
    auto load_row = [&](int r, RowInfo &ri, int &s0, int &s1) {
        if (r < nrows) {
            ri = a.info[r];
            const int32_t *e = a.segb + (int64_t)r * kXcds;
            s0 = x ? e[x - 1] : 0;
            s1 = e[x];
        }
    };
    load_row(cur_i, cur, cur_s0, cur_s1);
    load_row(la_i, la, la_s0, la_s1);
    auto first_base = [](const RowInfo &ri, int s0) {
        return s0 - (int)((ri.rs + s0) & (kStoreLine - 1));
    };
    int cur_base = first_base(cur, cur_s0);
    auto issue = [&](RowPartX<U> &p) {
        p.ri = cur;
        p.i = cur_i;
        p.base = cur_base;
        p.s0 = cur_s0;
        p.s1 = cur_s1;
        const bool any = cur_i < nrows && cur_s1 > cur_s0;  // wave-uniform
#pragma unroll
        for (int u = 0; u < U; ++u) {
            p.j[u] = -1;
            p.w[u] = 0.f;
        }
        if (any) {
            // clamped loads, selected afterwards (a load used under a lane
            // condition would be waited for inside it); non-temporal: the
            // row is read once, the gathered histories stay in L2
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int q = p.base + u * kWave + lane;
                const int qc = min(max(q, cur_s0), cur_s1 - 1);
                p.j[u] = __builtin_nontemporal_load(col + cur.rs + qc);
                p.w[u] = __builtin_nontemporal_load(wgt + cur.rs + qc);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int q = p.base + u * kWave + lane;
                if (q < cur_s0 || q >= cur_s1) p.j[u] = -1;
            }
        }
        if (any && cur_base + U * kWave < cur_s1) {  // the segment's next part
            cur_base += U * kWave;
        } else {  // the next row
            cur = la;
            cur_i = la_i;
            cur_s0 = la_s0;
            cur_s1 = la_s1;
            cur_base = first_base(cur, cur_s0);
            la_i += nwv;
            la = RowInfo{};
            la_s0 = la_s1 = 0;
            load_row(la_i, la, la_s0, la_s1);
        }
    };
    RowPartX<U> A, B;
    issue(A);
    issue(B);
    for (int q = tid; q <= kMaxAge; q += NT) s_dpow[q] = a.dpow[q];
    const uint8_t *s_code = s_sum;
    const int tbytes = a.code ? ((span + 15) / 16) * 16 : 0;
    if (a.code && span > 0)
        stage_lds<NT, 4>((uint4 *)s_sum, (const uint4 *)(a.code + lo), (span + 15) / 16);
    __syncthreads();

    int32_t *q_j = (int32_t *)(s_sum + tbytes) + wave * (2 * U * kWave);
    float *q_w = (float *)(q_j + U * kWave);
    // the history code of target j: staged for range x; outside it (a
    // target next to a range boundary) the history is gathered
    auto code_of = [&](int j) -> int {
        const int jj = j - lo;
        const bool in = (unsigned)jj < (unsigned)span;
        const int c = s_code[in ? jj : 0];
        return in ? c : (int)kCodeMulti;
    };
    auto step = [&](RowPartX<U> &p) {
        const RowInfo ri = p.ri;
        const int age = ri.age_pre & 0xff, pre = ri.age_pre >> 8;
        uint64_t m0, m1;
        window_masks(age, m0, m1);
        if (HW == 1) m1 = 0ull;
        bool cand[U];
        if (!pre && a.code) {
#pragma unroll
            for (int u = 0; u < U; ++u) cand[u] = p.j[u] >= 0 && code_of(max(p.j[u], 0)) != 0;
        } else {
#pragma unroll
            for (int u = 0; u < U; ++u) cand[u] = p.j[u] >= 0;
        }
        uint64_t bl[U];
        int qb[U];
        int qn = 0;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            bl[u] = ballot64(cand[u]);
            qb[u] = qn;
            qn += (int)__popcll(bl[u]);
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (cand[u]) {
                const int e = qb[u] + lane_rank(bl[u]);
                q_j[e] = p.j[u];
                q_w[e] = p.w[u];
            }
        }
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            constexpr int H = U / 2;
            if (half * H * kWave >= qn) break;  // wave-uniform
            uint64_t h[H], g[H];
            float qw[H];
            int cd[H];
#pragma unroll
            for (int q = 0; q < H; ++q) {
                const int e0 = (half * H + q) * kWave;
                h[q] = g[q] = 0ull;
                qw[q] = 0.f;
                cd[q] = 0;
                if (e0 < qn) {  // wave-uniform
                    const int e = e0 + lane;
                    const int j = e < qn ? q_j[e] : 0;
                    qw[q] = q_w[e];
                    cd[q] = (!pre && a.code) ? code_of(j) : (int)kCodeMulti;
                    gather_hist<HW>(hist, cd[q] == kCodeMulti ? j : 0, h[q], g[q]);
                }
            }
#pragma unroll
            for (int q = 0; q < H; ++q) {
                const int e = (half * H + q) * kWave + lane;
                if (e < qn) {
                    uint64_t h0 = h[q], h1 = g[q];
                    if (cd[q] != kCodeMulti) {
                        const int ps = (cd[q] - 1) & 127;  // single spike: ps steps ago
                        h0 = ps < 64 ? 1ull << (ps & 63) : 0ull;
                        h1 = ps >= 64 ? 1ull << (ps & 63) : 0ull;
                    }
                    h0 &= m0;
                    h1 &= m1;
                    const bool chg = h0 || h1 || !a.event;
                    float w = qw[q];
                    if (chg) {
                        w = a.event ? stdp_synapse(w, h0, h1, age, 0, ri.xp0, ri.xp_now, 0.f,
                                                   s_dpow, c_pot, c_dep, mu)
                                    : stdp_synapse_steps(w, h0, h1, age, 0, ri.xp0, ri.xp_now,
                                                         0.f, s_dpow[1], c_pot, c_dep, mu);
                        ++written;
                    }
                    q_w[e] = w;
                    q_j[e] = chg ? 1 : 0;
                }
            }
        }
        __builtin_amdgcn_wave_barrier();
        // the waves of range 0 commit the row's t_last and pre trace (every
        // row has a first part there, empty or not)
        if (x == 0 && p.i < nrows && ri.age_pre != 0 && p.base == first_base(ri, 0) &&
            lane == 0) {
            a.t_last[ri.k] = (int32_t)t;
            a.xpre[ri.k] = ri.xp_now;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int e = qb[u] + lane_rank(bl[u]);  // < (u + 1) * 64: inside the queue
            const int rj = q_j[e];
            const float rw = q_w[e];
            const bool c = (bl[u] >> lane) & 1ull;
            const bool chg = c && rj != 0;
            const float w = c ? rw : p.w[u];
            const int qi = p.base + u * kWave + lane;
            const uint64_t m = ballot64(chg);
            if (((m >> line0) & kLineMask) && qi >= p.s0 && qi < p.s1)
                __builtin_nontemporal_store(w, wgt + ri.rs + qi);
        }
        issue(p);
    };
    while (A.i < nrows) {
        step(A);
        if (B.i >= nrows) break;
        step(B);
    }
    written = wave_sum_i64(written);
    if (lane == 0 && written)
        atomicAdd((unsigned long long *)(a.stats + bid), (unsigned long long)written);
}

// One instance per history length: the 128-step one keeps a second history
// word per gathered synapse in registers.
template <int HW>
__global__ __launch_bounds__(kStdpRowsBlock) void k_stdp_rows(StdpArgs a)
{
    extern __shared__ uint4 dyn_sum[];
    if (a.xcd)
        stdp_rows_xcd_body<kStdpRowsBlock, kStdpXcdUnroll, HW>(
            a, blockIdx.x, gridDim.x, (unsigned char *)dyn_sum);
    else
        stdp_rows_body<kStdpRowsBlock, HW == 1 ? kStdpRowsUnroll : kStdpRowsUnroll2, HW>(
            a, blockIdx.x, gridDim.x, (unsigned char *)dyn_sum);
}

// Naive plasticity (Fig. 2(a)), the baseline the lazy forms are measured
// against: every plastic synapse every step, each with its own pre and post
// trace. Per step and synapse k->j both traces decay; a pre spike (k
// transmits at t) depresses with the post trace and bumps the pre trace; a
// post spike (j fires at t) potentiates with the pre trace and bumps the
// post trace. A wave per row, U synapses per lane; the fire mask of step t
// is staged in LDS for the post spikes.
constexpr int kNaiveBlock = 1024;
constexpr int kNaiveUnroll = 4;

__global__ __launch_bounds__(kNaiveBlock) void k_stdp_naive(NaiveArgs a)
{
    extern __shared__ uint64_t s_fire[];
    const int tid = threadIdx.x, lane = tid % kWave;
    stage_lds<kNaiveBlock, 4>(s_fire, a.mask, a.nw);
    __syncthreads();
    const int gw = (blockIdx.x * kNaiveBlock + tid) / kWave;
    const int nwv = gridDim.x * (kNaiveBlock / kWave);
    const float dp = a.d_plus, dm = a.d_minus, c_pot = a.c_pot, c_dep = a.c_dep, mu = a.mu;
    long long written = 0, updates = 0;
    for (int k = gw; k < a.n_rows; k += nwv) {
        const int pre = (int)((a.txmask[k >> 6] >> (k & 63)) & 1ull);  // wave-uniform
        const int64_t rs = a.row_ptr[k];
        const int len = a.pend[k];
        updates += len;
        for (int b = 0; b < len; b += kWave * kNaiveUnroll) {
            int j[kNaiveUnroll];
            float w[kNaiveUnroll], xp[kNaiveUnroll], xq[kNaiveUnroll];
#pragma unroll
            for (int u = 0; u < kNaiveUnroll; ++u) {  // clamped loads, selected below
                const int e = min(b + u * kWave + lane, len - 1);
                j[u] = a.col[rs + e];
                w[u] = a.w[rs + e];
                xp[u] = a.sx_pre[rs + e];
                xq[u] = a.sx_post[rs + e];
            }
#pragma unroll
            for (int u = 0; u < kNaiveUnroll; ++u) {
                const int e = b + u * kWave + lane;
                if (e >= len) continue;
                const int post = (int)((s_fire[j[u] >> 6] >> (j[u] & 63)) & 1ull);
                float x = xp[u] * dp, y = xq[u] * dm, ww = w[u];
                if (pre) {
                    ww = ww - c_dep * ww * y;
                    ww = fmaxf(ww, 0.f);
                    x = x + 1.f;
                }
                if (post) {
                    ww = ww + c_pot * pow_mu(ww, mu) * x;
                    y = y + 1.f;
                }
                if (pre || post) {
                    a.w[rs + e] = ww;
                    ++written;
                }
                a.sx_pre[rs + e] = x;
                a.sx_post[rs + e] = y;
            }
        }
    }
    written = wave_sum_i64(written);
    if (lane == 0) {
        if (written)
            atomicAdd((unsigned long long *)(a.stats + blockIdx.x), (unsigned long long)written);
        if (updates) atomicAdd((unsigned long long *)a.syn_count, (unsigned long long)updates);
    }
}

// ---------------------------------------------------------------------------
// (3) delivery.
//
// Slice delivery (Sec. III-B, Fig. 3(b)): work item q = (slice s, chunk c)
// owns targets [sW, (s+1)W) for the transmitted spikes at list positions
// c, c + C, c + 2C, ... The slice accumulator lives in LDS as exact 64-bit
// fixed point. For a batch of spikes the workgroup first gathers each
// spike's in-slice segment (row start + piv[k][s], length piv[k][s+1] -
// piv[k][s]) into LDS and prefix-sums the lengths; a map from each entry of
// the concatenated segments to its segment is then filled (by the segments'
// own threads when all are short, else by marking starts and a max-scan);
// then every thread takes flattened elements of the concatenated segments,
// so lanes stay busy
// whatever the segment lengths and consecutive lanes read consecutive
// entries of a segment (coalesced loads). Each element adds its weight into
// acc[target - sW] with an LDS 64-bit integer atomic. With C = 1 the
// workgroup owns the slice and stores the fp32 input directly; with C > 1 it
// stores fixed-point partial sum c. Workgroup b runs on XCD b mod 8, so work
// items are dealt out so that each XCD gets a contiguous range of slices
// (neighbouring segments of one row share cache lines).
//
// With plastic rows, each transmitting row is brought up to date here,
// immediately before its weights are delivered (Sec. III-A: a synapse need
// only be current to transmit; Sec. I: steps (2) and (3) walk the same
// rows): the slice's history words and post traces are staged in LDS beside
// the accumulator, and every plastic element of a segment is updated, stored
// and then delivered, so the row's targets and weights are read once. The
// workgroups of slice 0 commit t_last and the pre traces of their spikes.
//
// In a delay block (networks without plasticity) the grid also spans the
// block's steps: item (b, slice) takes ring slot (t_emit0 + b) mod D and
// writes the fixed-point input of its step to abatch, one chunk per item.
//
// The spike count is read first and only the spikes below it are read
// (a network with few spikes per step would otherwise read a whole batch of
// snapshots per workgroup), and the workgroup's statistics are reduced
// before its final stores, so no barrier waits for them.

constexpr int kDlvDirectMax = 32;  // segments up to this long are mapped by their own thread
// spikes a thread stages per batch (spike j = r kDlvBlock + tid)
constexpr int kDlvRounds = (kDlvBatch + kDlvBlock - 1) / kDlvBlock;
static_assert(kDlvRounds == 2, "two staged spikes per thread");

// The body of one workgroup (bid of nb, nb a multiple of 8) in its dynamic
// LDS: the staging arrays (DlvShared), then nacc * W accumulators [, W
// histories, W traces]. Keeping the staging arrays in the dynamic region
// lets a launch that also runs other work reuse the bytes.
template <bool CT, typename MapT>
__device__ __forceinline__ void deliver_lds_body(const DeliverArgs &a, int bid, int nb,
                                                 unsigned char *dyn)
{
    DlvSharedT<MapT> &S = *reinterpret_cast<DlvSharedT<MapT> *>(dyn);
    long long *acc = reinterpret_cast<long long *>(dyn + sizeof(DlvSharedT<MapT>));
    long long *s_start = S.start;
    int *s_off = S.off;
    int *s_info = S.info;
    float *s_xp0 = S.xp0;
    MapT *s_map = S.map;
    float *s_dpow = S.dpow;
    long long *sh = S.sh;
    int *shi = S.shi;
    unsigned long long &s_written = S.written;
    int &s_nlong = S.nlong;
    const int tid = threadIdx.x;
    const int qa = (bid & 7) * (nb >> 3) + (bid >> 3);
    if (qa >= a.n_work) return;  // whole workgroup, before any barrier
    // a delay block's item (b, slice, chunk) takes step b's ring list and
    // writes partial sums of step b (b varies slowest: an XCD's range of
    // items covers neighbouring slices)
    // step t = clk->t - 1 delivers the spikes of step t - D + 1; a delay
    // block starting at step t0 = clk->t delivers those of t0 + 1 - D + b
    const int64_t t = a.clk->t - 1;
    int slot = ring_slot(t - (a.delay - 1), a.delay);
    long long *parts = a.apart;
    int q = qa;
    if (a.batch > 0) {
        const int per = a.n_slices * a.chunks;
        const int bb = qa / per;
        q = qa - bb * per;
        slot = ring_slot(t + 2 - a.delay + bb, a.delay);
        parts = a.abatch + (int64_t)bb * a.chunks * a.part_stride;
    } else if (qa == 0 && threadIdx.x == 0) {
        // the next neuron update reads this delivery's output: the fp32
        // input with one chunk, else the C partial sums
        a.clk->input_forced = a.chunks == 1 ? 1 : 0;
        a.clk->n_parts = a.chunks;
    }
    // (the count of a single step's transmitted list is at a fixed address:
    // loading it does not wait for the clock)
    const int32_t *list = a.ring + (int64_t)slot * a.n;
    const int32_t *cntp = a.batch > 0 ? a.ring_cnt + slot : a.tx_cnt;
    const int s = q / a.chunks, c = q - s * a.chunks;
    const int C = a.chunks;
    const int base = s * a.width;
    const int span = a.nacc * a.width;
    // the count first (one scalar load), then the first batch's snapshots
    // (or list entries) below it, before the staging loads, so the two
    // round trips overlap: spikes j = rr kDlvBlock + tid
    const int cnt = *cntp;
    RowInfo ri0[kDlvRounds];
    int k0[kDlvRounds];
#pragma unroll
    for (int rr = 0; rr < kDlvRounds; ++rr) {
        const int j = rr * kDlvBlock + tid;
        ri0[rr] = RowInfo{};
        k0[rr] = 0;
        if (j < kDlvBatch && c + C * j < cnt) {
            if (a.plastic)
                ri0[rr] = a.txinfo[c + C * j];
            else
                k0[rr] = list[c + C * j];
        }
    }
    const int hw = a.hw;
    const int jn = min(a.width, a.n - base);  // > 0
    // the slice's histories and post traces: loads out now, stored below
    StageRegs<4, uint64_t> g_hist;
    StageRegs<4, float> g_y;
    if (a.plastic) {
        stage_issue<kDlvBlock>(g_hist, a.hist + (int64_t)base * hw, jn * hw);
        stage_issue<kDlvBlock>(g_y, a.ypost + base, jn);
    }
    const int piv_stride = a.n_slices + 1;
    // the first batch's pivots, as soon as its snapshots are in (spikes
    // below the count only)
    int k0p[kDlvRounds], p0p[kDlvRounds], p1p[kDlvRounds];
    int64_t rsp[kDlvRounds];
#pragma unroll
    for (int rr = 0; rr < kDlvRounds; ++rr) {
        const int j = rr * kDlvBlock + tid;
        k0p[rr] = p0p[rr] = p1p[rr] = 0;
        rsp[rr] = 0;
        if (j < kDlvBatch && c + C * j < cnt) {
            k0p[rr] = min(max(a.plastic ? ri0[rr].k : k0[rr], 0), a.n - 1);
            const int32_t *pv = a.piv + (int64_t)k0p[rr] * piv_stride + s;
            p0p[rr] = pv[0];
            p1p[rr] = pv[1];
            rsp[rr] = a.plastic ? ri0[rr].rs : a.row_ptr[k0p[rr]];
        }
    }
    if (tid == 0) s_written = 0ull;  // published by the batch loop's barriers
    for (int x = tid; x < span; x += kDlvBlock) acc[x] = 0;
    uint64_t *s_hist = (uint64_t *)(acc + span);
    float *s_y = (float *)(s_hist + (size_t)a.width * hw);
    if (a.plastic) {
        stage_finish<kDlvBlock>(s_hist, g_hist, a.hist + (int64_t)base * hw, jn * hw);
        stage_finish<kDlvBlock>(s_y, g_y, a.ypost + base, jn);
        for (int x = tid; x <= kMaxAge; x += kDlvBlock) s_dpow[x] = a.dpow[x];
    }
    const int32_t *__restrict__ col = a.col;
    float *__restrict__ wgt = a.w;
    const float c_pot = a.c_pot, c_dep = a.c_dep, mu = a.mu;
    long long ev = 0, written = 0;
    for (int b0 = 0;; b0 += kDlvBatch) {
        // stage segment starts and lengths (spikes tid and kDlvBlock + tid)
        int len[kDlvRounds];
#pragma unroll
        for (int rr = 0; rr < kDlvRounds; ++rr) {
            const int j = rr * kDlvBlock + tid;
            const int r = c + C * (b0 + j);
            len[rr] = 0;
            if (j >= kDlvBatch || r >= a.n) continue;
            int k, p0, p1;
            int64_t rs;
            RowInfo ri = RowInfo{};
            if (a.plastic) ri = b0 == 0 ? ri0[rr] : a.txinfo[r];
            const int plen_row = ri.len, ap = ri.age_pre;
            const float xp0 = ri.xp0, xpn = ri.xp_now;
            if (b0 == 0) {  // prefetched above
                k = k0p[rr];
                rs = rsp[rr];
                p0 = p0p[rr];
                p1 = p1p[rr];
            } else {
                k = min(max(a.plastic ? ri.k : list[r], 0), a.n - 1);  // past the count: stale
                const int32_t *pv = a.piv + (int64_t)k * piv_stride + s;
                p0 = pv[0];
                p1 = pv[1];
                rs = a.plastic ? ri.rs : a.row_ptr[k];
            }
            if (r < cnt) {
                len[rr] = p1 - p0;
                s_start[j] = rs + p0;
                const int plen = ap != 0 ? min(max(plen_row - p0, 0), len[rr]) : 0;
                const int inh = (a.nacc == 2 && k >= a.n_exc) ? 1 : 0;
                s_info[j] = plen | ((ap & 0xff) << 18) | (inh << 26);
                s_xp0[j] = xp0;
                if (a.plastic && s == 0 && ap != 0) {
                    a.t_last[k] = (int32_t)t;
                    a.xpre[k] = xpn;
                }
            }
        }
        const int nbt = min(kDlvBatch, max(0, (cnt - c + C - 1) / C - b0));
        // segment offsets in spike order, one scan per round that holds
        // spikes; each packs the number of long segments in bits 40+
        long long carry = 0;
#pragma unroll
        for (int rr = 0; rr < kDlvRounds; ++rr) {
            if (rr > 0 && nbt <= rr * kDlvBlock) break;  // workgroup-uniform
            const int j = rr * kDlvBlock + tid;
            const long long packed =
                (long long)len[rr] | ((long long)(len[rr] > kDlvDirectMax) << 40);
            const long long incl_p = block_incl_scan_i64_n<kDlvBlock>(packed, sh) + carry;
            if (j < nbt) s_off[j] = (int)((incl_p & ((1ll << 40) - 1)) - len[rr]);
            if (tid == kDlvBlock - 1) S.total = incl_p;
            __syncthreads();
            carry = S.total;
        }
        if (tid == 0) {  // totals (spikes >= nbt add 0)
            s_off[nbt] = (int)(carry & ((1ll << 40) - 1));
            s_nlong = (int)(carry >> 40);
        }
        __syncthreads();
        const int total = s_off[nbt];
        const bool direct = s_nlong == 0;
        ev += tid == 0 ? total : 0;
        for (int e0 = 0; e0 < total; e0 += kDlvWindow) {
            const int we = min(kDlvWindow, total - e0);
            if (direct) {
                // short segments: each thread writes its own segments' entries
#pragma unroll
                for (int rr = 0; rr < kDlvRounds; ++rr) {
                    const int j = rr * kDlvBlock + tid;
                    if (j < nbt) {
                        const int a0 = max(s_off[j], e0), a1 = min(s_off[j + 1], e0 + we);
                        for (int x = a0; x < a1; ++x) s_map[x - e0] = (MapT)(j + 1);
                    }
                }
                __syncthreads();
            } else {
                // mark each segment's first entry in the window, then max-scan
                for (int x = tid; x < we; x += kDlvBlock) s_map[x] = 0;
                __syncthreads();
#pragma unroll
                for (int rr = 0; rr < kDlvRounds; ++rr) {
                    const int j = rr * kDlvBlock + tid;
                    if (j < nbt) {
                        const int a0 = max(s_off[j], e0), a1 = min(s_off[j + 1], e0 + we);
                        if (a0 < a1) s_map[a0 - e0] = (MapT)(j + 1);
                    }
                }
                __syncthreads();
                fill_segment_map<kDlvBlock, kDlvUnroll, MapT>(s_map, we, shi, 0);
            }
            int tgt[kDlvUnroll], slot[kDlvUnroll], off[kDlvUnroll];
            long long gi[kDlvUnroll];
            float wv[kDlvUnroll];
            // loads from safe addresses for every element slot, selected after
            // all of them are in flight (a load used under a lane condition
            // would be waited for inside it)
            int cv[kDlvUnroll];
#pragma unroll
            for (int u = 0; u < kDlvUnroll; ++u) {
                const int x = u * kDlvBlock + tid;  // < kDlvWindow
                const int lm = (int)s_map[x] - 1;  // entries are 1 + segment
                const int l = x < we ? lm : 0;
                slot[u] = l;
                off[u] = e0 + x - s_off[l];
                gi[u] = x < we ? s_start[l] + off[u] : 0;  // edge 0 exists when total > 0
                // compressed targets are the slice-local index itself
                if (CT)
                    cv[u] = (int)a.col16[gi[u]];
                else
                    cv[u] = col[gi[u]] - base;
                wv[u] = wgt[gi[u]];
            }
#pragma unroll
            for (int u = 0; u < kDlvUnroll; ++u) {
                const bool in = u * kDlvBlock + tid < we;
                tgt[u] = in ? cv[u] : -1;
                if (!in) wv[u] = 0.f;
            }
            if (a.plastic) {
#pragma unroll
                for (int u = 0; u < kDlvUnroll; ++u) {
                    if (tgt[u] < 0) continue;
                    const int l = slot[u];
                    const int info = s_info[l];
                    if (off[u] >= (info & 0x3ffff)) continue;  // not plastic
                    const int age = (info >> 18) & 0xff;
                    uint64_t m0, m1;
                    window_masks(age, m0, m1);
                    const uint64_t h1 = hw == 2 ? s_hist[tgt[u] * 2 + 1] & m1 : 0ull;
                    const uint64_t h0 = s_hist[tgt[u] * hw] & m0;
                    // the pre trace after this update, as the snapshot holds it
                    const float xp0 = s_xp0[l];
                    const float xpn = __fadd_rn(__fmul_rn(xp0, s_dpow[age]), 1.f);
                    wv[u] = a.event ? stdp_synapse(wv[u], h0, h1, age, 1, xp0, xpn,
                                                   s_y[tgt[u]], s_dpow, c_pot, c_dep, mu)
                                    : stdp_synapse_steps(wv[u], h0, h1, age, 1, xp0, xpn,
                                                         s_y[tgt[u]], s_dpow[1], c_pot, c_dep,
                                                         mu);
                    wgt[gi[u]] = wv[u];
                    ++written;
                }
            }
#pragma unroll
            for (int u = 0; u < kDlvUnroll; ++u)
                if (tgt[u] >= 0)
                    atomicAdd((unsigned long long *)(acc + tgt[u] +
                                                     (((s_info[slot[u]] >> 26) & 1) ? a.width : 0)),
                              (unsigned long long)to_fix(wv[u]));
            if (e0 + kDlvWindow < total) __syncthreads();  // map rewritten by the next window
        }
        if (c + C * (b0 + kDlvBatch) >= cnt) break;
        __syncthreads();  // staging arrays are rewritten by the next batch
    }
    // (ev is thread 0's alone)
    written = wave_sum_i64(written);
    if (tid % kWave == 0 && written) atomicAdd(&s_written, (unsigned long long)written);
    __syncthreads();  // the accumulation barrier: every LDS atomic is done
    if (tid == 0) {
        add_stat(a.stats + 2 * (int64_t)bid, ev);
        add_stat(a.stats + 2 * (int64_t)bid + 1, (long long)s_written);
    }
    if (a.chunks == 1 && a.batch == 0) {
        for (int x = tid; x < a.width; x += kDlvBlock) {
            const int j = base + x;
            if (j < a.n) {
                a.ain[j] = from_fix(acc[x]);
                if (a.nacc == 2) a.ain[a.n + j] = from_fix(acc[a.width + x]);
            }
        }
    } else {
        long long *out = parts + (int64_t)c * a.part_stride;
        for (int x = tid; x < a.width; x += kDlvBlock) {
            const int j = base + x;
            if (j < a.n) {
                out[j] = acc[x];
                if (a.nacc == 2) out[a.n + j] = acc[a.width + x];
            }
        }
    }
}

// (four waves per SIMD: two workgroups share a CU)
template <bool CT>
__global__ __launch_bounds__(kDlvBlock, 4) void k_deliver_lds(DeliverArgs a)
{
    extern __shared__ uint4 dyn_dlv[];
    deliver_lds_body<CT, int>(a, blockIdx.x, gridDim.x, reinterpret_cast<unsigned char *>(dyn_dlv));
}

// Fused synapse pass of one step: the forced rows' plasticity and slice
// delivery (with the transmitting rows' plasticity) in one launch. A forced
// row does not transmit at t, so the two parts touch disjoint rows, and
// neither reads what the other writes (targets' histories, post traces and
// history summaries are only read): workgroups [0, nd) deliver, the others
// take forced-row parts, side by side, in one launch's ramp and drain. The
// dynamic LDS is the larger role's (each role lays its own out from the
// start), so two workgroups share a CU where it is at most half the CU's;
// four waves per SIMD bound the registers to match. With 128-step
// histories the delivery role keeps its segment map in 16 bits.
template <bool CT, int HW>
__global__ __launch_bounds__(kDlvBlock, 4) void k_synapse_pass(DeliverArgs d, StdpArgs s,
                                                               int32_t nd)
{
    extern __shared__ uint4 dyn_pass[];
    if ((int)blockIdx.x < nd)
        deliver_lds_body<CT, FusedMap<HW>>(d, blockIdx.x, nd,
                                           reinterpret_cast<unsigned char *>(dyn_pass));
    else if (s.xcd)
        stdp_rows_xcd_body<kDlvBlock, kStdpXcdUnroll, HW>(
            s, blockIdx.x - nd, gridDim.x - nd, (unsigned char *)dyn_pass);
    else
        stdp_rows_body<kDlvBlock, HW == 1 ? kStdpRowsUnroll : kStdpRowsUnroll2, HW>(
            s, blockIdx.x - nd, gridDim.x - nd, (unsigned char *)dyn_pass);
}

// Row-wise delivery with global atomics (Fig. 3(a)): a wave per transmitted
// spike, lanes over its row, hardware 64-bit integer atomics on the same
// fixed-point accumulator in HBM/L2. A lane loads U entries before issuing
// their atomics, so a 1000-synapse row needs about one load latency.
constexpr int kGlobalUnroll = 16;

__global__ __launch_bounds__(kBlock) void k_deliver_global(DeliverArgs a)
{
    __shared__ long long sh[kBlock / kWave];
    const int tid = threadIdx.x, lane = tid % kWave;
    const int gw = (blockIdx.x * kBlock + tid) / kWave;
    const int nwv = gridDim.x * (kBlock / kWave);
    const int64_t t = a.clk->t - 1;
    const int slot = ring_slot(t - (a.delay - 1), a.delay);
    const int32_t *list = a.ring + (int64_t)slot * a.n;
    const int cnt = a.ring_cnt[slot];
    if (blockIdx.x == 0 && tid == 0) {  // the next neuron update adds the one sum
        a.clk->input_forced = 0;
        a.clk->n_parts = 1;
    }
    const int32_t *__restrict__ col = a.col;
    const float *__restrict__ wgt = a.w;
    long long ev = 0;
    for (int x = gw; x < cnt; x += nwv) {
        const int k = list[x];
        const int64_t rs = a.row_ptr[k], re = a.row_ptr[k + 1];
        long long *dst = (a.nacc == 2 && k >= a.n_exc) ? a.apart + a.n : a.apart;
        for (int64_t e0 = rs; e0 < re; e0 += kWave * kGlobalUnroll) {
            int tgt[kGlobalUnroll];
            float wv[kGlobalUnroll];
#pragma unroll
            for (int u = 0; u < kGlobalUnroll; ++u) {
                const int64_t e = e0 + u * kWave + lane;
                const int64_t ec = e < re ? e : rs;  // safe address, selected below
                tgt[u] = col[ec];
                wv[u] = wgt[ec];
            }
#pragma unroll
            for (int u = 0; u < kGlobalUnroll; ++u) {
                if (e0 + u * kWave + lane >= re) tgt[u] = -1;
            }
#pragma unroll
            for (int u = 0; u < kGlobalUnroll; ++u)
                if (tgt[u] >= 0)
                    atomicAdd((unsigned long long *)(dst + tgt[u]),
                              (unsigned long long)to_fix(wv[u]));
        }
        if (lane == 0) ev += re - rs;
    }
    ev = block_sum_i64(ev, sh);
    if (tid == 0) add_stat(a.stats + 2 * (int64_t)blockIdx.x, ev);
}

// ---------------------------------------------------------------------------
// Measurement probe, not part of a step: the access pattern of the forced-row
// STDP without its arithmetic. Each wave streams whole plastic rows, chosen
// pseudo-randomly (row rng32(seed, 5, r, 0) mod plastic rows for r <
// n_rows), two parts of 8 synapses per lane in flight, with non-temporal
// loads of the targets and weights, and with `write` stores every weight
// back unchanged. `sink` only keeps the loads alive (written with vanishing
// probability); the synapse count is left to the host, since atomics on one
// word from every wave would serialise.
__global__ __launch_bounds__(kStdpRowsBlock) void k_probe_rows(const int64_t *row_ptr,
                                                               const int32_t *pend,
                                                               const int32_t *col, float *w,
                                                               int32_t n_rows, int32_t n_plastic,
                                                               uint64_t seed, int32_t write,
                                                               unsigned long long *sink)
{
    constexpr int U = 2 * kStdpRowsUnroll;  // two parts in flight, as the STDP kernel holds
    const int lane = threadIdx.x % kWave;
    const int gw = (blockIdx.x * kStdpRowsBlock + threadIdx.x) / kWave;
    const int nwv = gridDim.x * (kStdpRowsBlock / kWave);
    uint32_t keep = 0;
    for (int r = gw; r < n_rows; r += nwv) {  // wave-uniform
        const int k = (int)(rng32(seed, 5, (uint64_t)r, 0) % (uint32_t)n_plastic);
        const int64_t rs = row_ptr[k];
        const int len = pend[k];
        for (int base = 0; base < len; base += U * kWave) {
            int32_t j[U];
            float x[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int qc = min(base + u * kWave + lane, len - 1);
                j[u] = __builtin_nontemporal_load(col + rs + qc);
                x[u] = __builtin_nontemporal_load(w + rs + qc);
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                keep ^= (uint32_t)j[u] ^ __float_as_uint(x[u]);
                const int q = base + u * kWave + lane;
                if (write && q < len) __builtin_nontemporal_store(x[u], w + rs + q);
            }
        }
    }
    if (keep == 0x9e3779b9u) atomicAdd(sink, 1ull);
}

}  // namespace

hipError_t launch_row_info(hipStream_t s, const RowInfoArgs &a, int64_t max_rows)
{
    hipLaunchKernelGGL(k_row_info, dim3(blocks_for(max_rows)), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_stdp(hipStream_t s, const StdpArgs &a, int blocks, size_t lds, KernelEvents ev)
{
    static std::mutex mu;
    static int granted = 64 * 1024;
    const hipError_t e = allow_dynamic_lds((const void *)k_stdp, (int)lds, mu, granted);
    if (e != hipSuccess) return e;
    launch_kernel(k_stdp, dim3(blocks), dim3(kStdpBlock), lds, s, ev, a);
    return hipGetLastError();
}

hipError_t launch_stdp_rows(hipStream_t s, const StdpArgs &a, int blocks, KernelEvents ev)
{
    static std::mutex mu;
    static int granted[2] = {64 * 1024, 64 * 1024};
    size_t xspan = 0;  // the largest target range of the XCD form
    for (int x = 0; x < kXcds; ++x) xspan = std::max(xspan, (size_t)(a.xlo[x + 1] - a.xlo[x]));
    const size_t table = a.xcd      ? (a.code ? (xspan + 15) / 16 * 16 : 0)
                         : a.code   ? (((size_t)a.n + 15) / 16) * 16
                         : a.recent ? (size_t)a.nw * sizeof(uint64_t)
                                    : 0;
    const size_t lds = table + stdp_rows_queue_bytes(a.hw);
    if (a.xcd && (blocks < kXcds || (a.xparts != 2 && a.xparts != 4 && a.xparts != 8)))
        return hipErrorInvalidValue;
    const void *kern = a.hw == 2 ? (const void *)k_stdp_rows<2> : (const void *)k_stdp_rows<1>;
    const hipError_t e = allow_dynamic_lds(kern, (int)lds, mu, granted[a.hw == 2]);
    if (e != hipSuccess) return e;
    if (a.hw == 2)
        launch_kernel(k_stdp_rows<2>, dim3(blocks), dim3(kStdpRowsBlock), lds, s, ev, a);
    else
        launch_kernel(k_stdp_rows<1>, dim3(blocks), dim3(kStdpRowsBlock), lds, s, ev, a);
    return hipGetLastError();
}

hipError_t launch_stdp_naive(hipStream_t s, const NaiveArgs &a, int blocks, KernelEvents ev)
{
    static std::mutex mu;
    static int granted = 64 * 1024;
    const size_t lds = (size_t)a.nw * sizeof(uint64_t);
    const hipError_t e = allow_dynamic_lds((const void *)k_stdp_naive, (int)lds, mu, granted);
    if (e != hipSuccess) return e;
    launch_kernel(k_stdp_naive, dim3(blocks), dim3(kNaiveBlock), lds, s, ev, a);
    return hipGetLastError();
}

hipError_t launch_deliver_lds(hipStream_t s, const DeliverArgs &a, int blocks, size_t lds, KernelEvents ev)
{
    static std::mutex mu;
    static int granted[2] = {64 * 1024, 64 * 1024};
    const bool ct = a.col16 != nullptr;
    const void *kern = ct ? (const void *)k_deliver_lds<true> : (const void *)k_deliver_lds<false>;
    const hipError_t e = allow_dynamic_lds(kern, (int)lds, mu, granted[ct]);
    if (e != hipSuccess) return e;
    if (ct)
        launch_kernel(k_deliver_lds<true>, dim3(blocks), dim3(kDlvBlock), lds, s, ev, a);
    else
        launch_kernel(k_deliver_lds<false>, dim3(blocks), dim3(kDlvBlock), lds, s, ev, a);
    return hipGetLastError();
}

hipError_t launch_probe_rows(hipStream_t s, int blocks, const int64_t *row_ptr,
                             const int32_t *pend, const int32_t *col, float *w, int32_t n_rows,
                             int32_t n_plastic, uint64_t seed, int32_t write,
                             unsigned long long *sink, KernelEvents ev)
{
    if (n_rows < 1 || n_plastic < 1 || blocks < 1) return hipErrorInvalidValue;
    launch_kernel(k_probe_rows, dim3(blocks), dim3(kStdpRowsBlock), 0, s, ev, row_ptr, pend, col, w, n_rows, n_plastic, seed,
                          write, sink);
    return hipGetLastError();
}

hipError_t launch_synapse_pass(hipStream_t s, const DeliverArgs &d, const StdpArgs &a, int nd,
                               int ns, size_t lds, KernelEvents ev)
{
    static std::mutex mu;
    static int granted[4] = {64 * 1024, 64 * 1024, 64 * 1024, 64 * 1024};
    const int k = (d.col16 != nullptr ? 2 : 0) + (a.hw == 2 ? 1 : 0);
    const void *kerns[4] = {(const void *)k_synapse_pass<false, 1>,
                            (const void *)k_synapse_pass<false, 2>,
                            (const void *)k_synapse_pass<true, 1>,
                            (const void *)k_synapse_pass<true, 2>};
    // (the XCD form needs a forced-row workgroup on every XCD)
    if (nd % 8 != 0 || ns < 1 || (a.xcd && ns < kXcds)) return hipErrorInvalidValue;
    if (a.xcd && a.xparts != 2 && a.xparts != 4 && a.xparts != 8) return hipErrorInvalidValue;
    const hipError_t e = allow_dynamic_lds(kerns[k], (int)lds, mu, granted[k]);
    if (e != hipSuccess) return e;
    const dim3 g(nd + ns), b(kDlvBlock);
    switch (k) {
    case 0: launch_kernel((k_synapse_pass<false, 1>), g, b, lds, s, ev, d, a, nd); break;
    case 1: launch_kernel((k_synapse_pass<false, 2>), g, b, lds, s, ev, d, a, nd); break;
    case 2: launch_kernel((k_synapse_pass<true, 1>), g, b, lds, s, ev, d, a, nd); break;
    default: launch_kernel((k_synapse_pass<true, 2>), g, b, lds, s, ev, d, a, nd); break;
    }
    return hipGetLastError();
}

hipError_t launch_deliver_global(hipStream_t s, const DeliverArgs &a, int blocks, KernelEvents ev)
{
    launch_kernel(k_deliver_global, dim3(blocks), dim3(kBlock), 0, s, ev, a);
    return hipGetLastError();
}

int deliver_lds_static_bytes()
{
    return std::max(static_lds_bytes((const void *)k_deliver_lds<false>),
                    static_lds_bytes((const void *)k_deliver_lds<true>));
}
int stdp_static_bytes() { return static_lds_bytes((const void *)k_stdp); }
int synapse_pass_static_bytes()
{
    int m = -1;
    for (const void *k : {(const void *)k_synapse_pass<false, 1>, (const void *)k_synapse_pass<false, 2>,
                          (const void *)k_synapse_pass<true, 1>, (const void *)k_synapse_pass<true, 2>}) {
        const int b = static_lds_bytes(k);
        if (b < 0) return -1;
        m = std::max(m, b);
    }
    return m;
}

}  // namespace snn
