// gfx950 kernels of the synapse pass: row snapshots for a flush, lazy +
// event-driven STDP (slice-organised and row-wise layouts), slice delivery
// with LDS accumulation and the transmitting rows' plasticity fused in, the
// global-atomic delivery variant, and the one-launch synapse pass of a step.
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
// pre-synaptic spike). During a step the compaction kernel takes them.

__global__ __launch_bounds__(kBlock) void k_row_info(RowInfoArgs a)
{
    __shared__ float s_dpow[65];
    __shared__ long long sh[kBlock / kWave];
    const int tid = threadIdx.x;
    for (int q = tid; q < 65; q += kBlock) s_dpow[q] = a.dpow[q];
    __syncthreads();
    const int r = blockIdx.x * kBlock + tid;
    long long st_rows = 0, st_syn = 0;
    if (r < a.n_rows_all) {
        RowInfo ri;
        if (make_row_info(ri, r, a.t, false, a.dm1, a.row_ptr, a.pend, a.hist, a.t_last, a.xpre,
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
        slot[kStRows] += st_rows;
        slot[kStSyn] += st_syn;
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
    extern __shared__ unsigned char stage[];  // W_s history words, then W_s post traces
    __shared__ long long s_start[kStdpBatch];
    __shared__ uint64_t s_win[kStdpBatch];
    __shared__ int s_off[kStdpBatch + 1];
    __shared__ int s_ap[kStdpBatch];
    __shared__ float s_xp0[kStdpBatch];
    __shared__ float s_xpn[kStdpBatch];
    __shared__ int s_map[kStdpWindow];
    __shared__ float s_dpow[65];
    __shared__ long long sh[kStdpBlock / kWave];
    __shared__ int shi[kStdpBlock / kWave];
    const int tid = threadIdx.x;
    const int nb = gridDim.x;  // multiple of 8
    const int q = (blockIdx.x & 7) * (nb >> 3) + (blockIdx.x >> 3);
    if (q >= a.n_work) return;  // whole workgroup, before any barrier
    const int g = q / a.chunks, cr = q - g * a.chunks;
    const int nrows = a.row_cnt ? *a.row_cnt : a.n_rows_all;
    const int lo = (int)((int64_t)nrows * cr / a.chunks);
    const int hi = (int)((int64_t)nrows * (cr + 1) / a.chunks);
    if (g == 0) {
        for (int r = lo + tid; r < hi; r += kStdpBlock) {
            const RowInfo ri = a.info[r];
            if (ri.age_pre != 0) {
                a.t_last[ri.k] = (int32_t)a.t;
                a.xpre[ri.k] = ri.xp_now;
            }
        }
    }
    const int j0 = g * a.width;
    if (j0 >= a.target_limit) return;  // no plastic synapse targets this group (g > 0)
    uint64_t *s_hist = (uint64_t *)stage;
    float *s_y = (float *)(stage + (size_t)a.width * sizeof(uint64_t));
    const int jn = min(a.width, a.n - j0);
    for (int x = tid; x < jn; x += kStdpBlock) {
        s_hist[x] = a.hist[j0 + x];
        s_y[x] = a.ypost[j0 + x];
    }
    for (int x = tid; x < 65; x += kStdpBlock) s_dpow[x] = a.dpow[x];
    const int pv_lo = g * a.mult;
    const int pv_hi = min((g + 1) * a.mult, a.n_slices);
    const int piv_stride = a.n_slices + 1;
    Edge *__restrict__ edges = a.edges;
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
                const int age = ri.age_pre & 0xff;
                s_start[tid] = ri.rs + p0;
                s_win[tid] = age >= 64 ? ~0ull : ((1ull << age) - 1ull);
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
#pragma unroll
            for (int u = 0; u < kStdpUnroll; ++u) {
                const int x = u * kStdpBlock + tid;
                jl[u] = -1;
                if (x < we) {
                    const int l = s_map[x];
                    slot[u] = l;
                    gi[u] = s_start[l] + (e0 + x - s_off[l]);
                    const Edge ed = edges[gi[u]];
                    jl[u] = ed.col - j0;
                    wv[u] = ed.w;
                }
            }
#pragma unroll
            for (int u = 0; u < kStdpUnroll; ++u) {
                if (jl[u] < 0) continue;
                const int l = slot[u];
                const int ap = s_ap[l];
                const int pre = ap >> 8;
                const uint64_t h = s_hist[jl[u]] & s_win[l];
                if (!h && !pre) continue;  // nothing happened to this synapse
                edges[gi[u]].w = stdp_synapse(wv[u], h, ap & 0xff, pre, s_xp0[l], s_xpn[l],
                                          pre ? s_y[jl[u]] : 0.f, s_dpow, c_pot, c_dep, mu);
                ++written;
            }
            __syncthreads();  // map rewritten by the next window
        }
        __syncthreads();  // staging arrays are rewritten by the next batch
    }
    written = block_sum_i64_n<kStdpBlock>(written, sh);
    if (tid == 0) a.stats[blockIdx.x] += written;
}

// Row-wise layout: a wave per row to update, lanes over its plastic
// synapses in the row's own order, U synapses per lane with their edge loads
// and their history (and post-trace) gathers in flight together. Histories
// and traces come from L2 instead of LDS. With the spike-recency bitmap
// staged in LDS, a synapse of a row without a pre spike whose target has not
// fired within 64 steps is skipped without touching its history word in L2:
// most of them, at low rates. NT threads per workgroup; workgroup `bid` of
// `nblocks`.

template <int NT, int U>
__device__ __forceinline__ void stdp_rows_body(const StdpArgs &a, int bid, int nblocks,
                                               uint64_t *s_recent)
{
    __shared__ float s_dpow[65];
    __shared__ long long sh[NT / kWave];
    const int tid = threadIdx.x;
    for (int q = tid; q < 65; q += NT) s_dpow[q] = a.dpow[q];
    const bool filt = a.recent != nullptr;
    if (filt)
        for (int q = tid; q < a.nw; q += NT) s_recent[q] = a.recent[q];
    __syncthreads();
    Edge *__restrict__ edges = a.edges;
    const uint64_t *__restrict__ hist = a.hist;
    const float *__restrict__ ypost = a.ypost;
    const float c_pot = a.c_pot, c_dep = a.c_dep, mu = a.mu;
    const int lane = tid % kWave;
    const int gw = (bid * NT + tid) / kWave;
    const int nwv = nblocks * (NT / kWave);
    const int nrows = a.row_cnt ? *a.row_cnt : a.n_rows_all;
    long long written = 0;
    for (int r = gw; r < nrows; r += nwv) {
        const RowInfo ri = a.info[r];
        if (ri.age_pre == 0) continue;  // wave-uniform
        if (lane == 0) {
            a.t_last[ri.k] = (int32_t)a.t;
            a.xpre[ri.k] = ri.xp_now;
        }
        const int len = ri.len;
        const int age = ri.age_pre & 0xff, pre = ri.age_pre >> 8;
        const uint64_t win = age >= 64 ? ~0ull : ((1ull << age) - 1ull);
        const long long rs = ri.rs;
        for (int base = 0; base < len; base += kWave * U) {
            int j[U];
            float w[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int q = base + u * kWave + lane;
                Edge ed{-1, 0.f};
                if (q < len) ed = edges[rs + q];
                j[u] = ed.col;
                w[u] = ed.w;
            }
            if (filt && !pre) {
#pragma unroll
                for (int u = 0; u < U; ++u)
                    if (j[u] >= 0 && !((s_recent[j[u] >> 6] >> (j[u] & 63)) & 1ull)) j[u] = -1;
            }
            uint64_t h[U];
#pragma unroll
            for (int u = 0; u < U; ++u) h[u] = j[u] >= 0 ? (hist[j[u]] & win) : 0ull;
            float y[U];
#pragma unroll
            for (int u = 0; u < U; ++u) y[u] = (pre && j[u] >= 0) ? ypost[j[u]] : 0.f;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (j[u] < 0 || (!h[u] && !pre)) continue;
                edges[rs + base + u * kWave + lane].w = stdp_synapse(
                    w[u], h[u], age, pre, ri.xp0, ri.xp_now, y[u], s_dpow, c_pot, c_dep, mu);
                ++written;
            }
        }
    }
    written = block_sum_i64_n<NT>(written, sh);
    if (tid == 0) a.stats[bid] += written;
}

__global__ __launch_bounds__(kStdpRowsBlock) void k_stdp_rows(StdpArgs a)
{
    extern __shared__ uint64_t dyn_recent[];
    stdp_rows_body<kStdpRowsBlock, kStdpRowsUnroll>(a, blockIdx.x, gridDim.x, dyn_recent);
}

// ---------------------------------------------------------------------------
// (3) delivery.
//
// Slice delivery (Sec. III-B, Fig. 3(b)): work item q = (slice s, chunk c)
// owns targets [sW, (s+1)W) for the c-th 1/C of the transmitted spikes. The
// slice accumulator lives in LDS as exact 64-bit fixed point. For a batch of
// spikes the workgroup first gathers each spike's in-slice segment
// (row start + piv[k][s], length piv[k][s+1] - piv[k][s]) into LDS and
// prefix-sums the lengths; then every thread takes flattened elements of the
// concatenated segments, so lanes stay busy whatever the segment lengths and
// consecutive lanes read consecutive entries of a segment. Each element adds
// its weight into acc[target - sW] with an LDS 64-bit integer atomic. With
// C = 1 the workgroup owns the slice and stores the fp32 input directly;
// with C > 1 it stores fixed-point partial sum c. Workgroup b runs on XCD
// b mod 8, so work items are dealt out so that each XCD gets a contiguous
// range of slices (neighbouring segments of one row share cache lines).

constexpr int kDlvBlock = 512;
constexpr int kDlvBatch = 512;   // spikes whose segments are staged at once
constexpr int kDlvUnroll = 4;
constexpr int kDlvWindow = kDlvBlock * kDlvUnroll;

// With plastic rows, each transmitting row is brought up to date here,
// immediately before its weights are delivered (Sec. III-A: a synapse need
// only be current to transmit; Sec. I: steps (2) and (3) walk the same
// rows): the slice's history words and post traces are staged in LDS beside
// the accumulator, and every plastic element of a segment is updated, stored
// and then delivered, so the row's targets and weights are read once. The
// workgroups of slice 0 commit t_last and the pre traces of their spikes.
// Workgroup `bid` of `nb` (a multiple of 8); `acc` is the dynamic LDS.
__device__ __forceinline__ void deliver_lds_body(const DeliverArgs &a, int bid, int nb,
                                                 long long *acc)
{
    // acc: nacc * W accumulators [, W histories, W post traces]
    __shared__ long long s_start[kDlvBatch];
    __shared__ uint64_t s_win[kDlvBatch];
    __shared__ int s_off[kDlvBatch + 1];
    __shared__ int s_half[kDlvBatch];
    __shared__ int s_plen[kDlvBatch];
    __shared__ int s_age[kDlvBatch];
    __shared__ float s_xp0[kDlvBatch];
    __shared__ float s_xpn[kDlvBatch];
    __shared__ int s_map[kDlvWindow];
    __shared__ float s_dpow[65];
    __shared__ long long sh[kDlvBlock / kWave];
    __shared__ int shi[kDlvBlock / kWave];
    const int tid = threadIdx.x;
    const int q = (bid & 7) * (nb >> 3) + (bid >> 3);
    if (q >= a.n_work) return;  // whole workgroup, before any barrier
    const int s = q / a.chunks, c = q - s * a.chunks;
    const int base = s * a.width;
    const int span = a.nacc * a.width;
    for (int x = tid; x < span; x += kDlvBlock) acc[x] = 0;
    const int cnt = *a.cnt;
    const int lo = (int)((int64_t)cnt * c / a.chunks);
    const int hi = (int)((int64_t)cnt * (c + 1) / a.chunks);
    uint64_t *s_hist = (uint64_t *)(acc + span);
    float *s_y = (float *)(s_hist + a.width);
    if (a.plastic) {
        const int jn = min(a.width, a.n - base);
        for (int x = tid; x < jn; x += kDlvBlock) {
            s_hist[x] = a.hist[base + x];
            s_y[x] = a.ypost[base + x];
        }
        for (int x = tid; x < 65; x += kDlvBlock) s_dpow[x] = a.dpow[x];
        if (s == 0) {
            for (int x = lo + tid; x < hi; x += kDlvBlock) {
                const RowInfo ri = a.txinfo[x];
                if (ri.age_pre != 0) {
                    a.t_last[ri.k] = (int32_t)a.t;
                    a.xpre[ri.k] = ri.xp_now;
                }
            }
        }
    }
    const int piv_stride = a.n_slices + 1;
    Edge *__restrict__ edges = a.edges;
    const float c_pot = a.c_pot, c_dep = a.c_dep, mu = a.mu;
    long long ev = 0, written = 0;
    for (int b0 = lo; b0 < hi; b0 += kDlvBatch) {
        const int nbt = min(kDlvBatch, hi - b0);
        // stage segment starts and lengths (one spike per thread)
        int len = 0;
        if (tid < nbt) {
            const RowInfo ri = a.txinfo[b0 + tid];
            const int k = ri.k;
            const int32_t *pv = a.piv + (int64_t)k * piv_stride + s;
            const int p0 = pv[0], p1 = pv[1];
            s_start[tid] = ri.rs + p0;
            s_half[tid] = (a.nacc == 2 && k >= a.n_exc) ? a.width : 0;
            len = p1 - p0;
            int plen = 0;
            if (a.plastic) {
                if (ri.age_pre != 0) {
                    plen = min(max(ri.len - p0, 0), len);
                    const int age = ri.age_pre & 0xff;
                    s_age[tid] = age;
                    s_win[tid] = age >= 64 ? ~0ull : ((1ull << age) - 1ull);
                    s_xp0[tid] = ri.xp0;
                    s_xpn[tid] = ri.xp_now;
                }
            }
            s_plen[tid] = plen;
        }
        const long long incl = block_incl_scan_i64_n<kDlvBlock>(len, sh);
        if (tid < nbt) s_off[tid] = (int)(incl - len);
        if (tid == kDlvBlock - 1) s_off[nbt] = (int)incl;  // = total (threads >= nbt add 0)
        __syncthreads();
        const int total = s_off[nbt];
        ev += tid == 0 ? total : 0;
        for (int e0 = 0; e0 < total; e0 += kDlvWindow) {
            const int we = min(kDlvWindow, total - e0);
            for (int x = tid; x < we; x += kDlvBlock) s_map[x] = -1;
            __syncthreads();
            if (tid < nbt) {
                const int a0 = max(s_off[tid], e0), a1 = min(s_off[tid + 1], e0 + we);
                if (a0 < a1) s_map[a0 - e0] = tid;
            }
            __syncthreads();
            fill_segment_map<kDlvBlock>(s_map, we, shi);
            int tgt[kDlvUnroll], slot[kDlvUnroll], off[kDlvUnroll];
            long long gi[kDlvUnroll];
            float wv[kDlvUnroll];
#pragma unroll
            for (int u = 0; u < kDlvUnroll; ++u) {
                const int x = u * kDlvBlock + tid;
                tgt[u] = -1;
                wv[u] = 0.f;
                if (x < we) {
                    const int l = s_map[x];
                    slot[u] = l;
                    off[u] = e0 + x - s_off[l];
                    gi[u] = s_start[l] + off[u];
                    const Edge ed = edges[gi[u]];
                    tgt[u] = ed.col - base;
                    wv[u] = ed.w;
                }
            }
            if (a.plastic) {
#pragma unroll
                for (int u = 0; u < kDlvUnroll; ++u) {
                    if (tgt[u] < 0) continue;
                    const int l = slot[u];
                    if (off[u] >= s_plen[l]) continue;  // not plastic
                    const uint64_t h = s_hist[tgt[u]] & s_win[l];
                    wv[u] = stdp_synapse(wv[u], h, s_age[l], 1, s_xp0[l], s_xpn[l], s_y[tgt[u]],
                                         s_dpow, c_pot, c_dep, mu);
                    edges[gi[u]].w = wv[u];
                    ++written;
                }
            }
#pragma unroll
            for (int u = 0; u < kDlvUnroll; ++u)
                if (tgt[u] >= 0)
                    atomicAdd((unsigned long long *)(acc + tgt[u] + s_half[slot[u]]),
                              (unsigned long long)to_fix(wv[u]));
            __syncthreads();  // map rewritten by the next window
        }
        __syncthreads();  // staging arrays are rewritten by the next batch
    }
    __syncthreads();
    if (a.chunks == 1) {
        for (int x = tid; x < a.width; x += kDlvBlock) {
            const int j = base + x;
            if (j < a.n) {
                a.ain[j] = from_fix(acc[x]);
                if (a.nacc == 2) a.ain[a.n + j] = from_fix(acc[a.width + x]);
            }
        }
    } else {
        long long *out = a.apart + (int64_t)c * a.part_stride;
        for (int x = tid; x < a.width; x += kDlvBlock) {
            const int j = base + x;
            if (j < a.n) {
                out[j] = acc[x];
                if (a.nacc == 2) out[a.n + j] = acc[a.width + x];
            }
        }
    }
    ev = block_sum_i64_n<kDlvBlock>(ev, sh);
    written = block_sum_i64_n<kDlvBlock>(written, sh);
    if (tid == 0) {
        a.stats[2 * (int64_t)bid] += ev;
        a.stats[2 * (int64_t)bid + 1] += written;
    }
}

__global__ __launch_bounds__(kDlvBlock) void k_deliver_lds(DeliverArgs a)
{
    extern __shared__ long long dyn_acc[];
    deliver_lds_body(a, blockIdx.x, gridDim.x, dyn_acc);
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
    const int cnt = *a.cnt;
    const Edge *__restrict__ edges = a.edges;
    long long ev = 0;
    for (int x = gw; x < cnt; x += nwv) {
        const int k = a.list[x];
        const int64_t rs = a.row_ptr[k], re = a.row_ptr[k + 1];
        long long *dst = (a.nacc == 2 && k >= a.n_exc) ? a.apart + a.n : a.apart;
        for (int64_t e0 = rs; e0 < re; e0 += kWave * kGlobalUnroll) {
            int tgt[kGlobalUnroll];
            float wv[kGlobalUnroll];
#pragma unroll
            for (int u = 0; u < kGlobalUnroll; ++u) {
                const int64_t e = e0 + u * kWave + lane;
                Edge ed{-1, 0.f};
                if (e < re) ed = edges[e];
                tgt[u] = ed.col;
                wv[u] = ed.w;
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
    if (tid == 0) a.stats[2 * (int64_t)blockIdx.x] += ev;
}

}  // namespace

hipError_t launch_row_info(hipStream_t s, const RowInfoArgs &a, int64_t max_rows)
{
    hipLaunchKernelGGL(k_row_info, dim3(blocks_for(max_rows)), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_stdp(hipStream_t s, const StdpArgs &a, int blocks, size_t lds)
{
    static std::mutex mu;
    static int granted = 64 * 1024;
    const hipError_t e = allow_dynamic_lds((const void *)k_stdp, (int)lds, mu, granted);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_stdp, dim3(blocks), dim3(kStdpBlock), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_stdp_rows(hipStream_t s, const StdpArgs &a, int blocks)
{
    const size_t lds = a.recent ? (size_t)a.nw * sizeof(uint64_t) : 0;
    hipLaunchKernelGGL(k_stdp_rows, dim3(blocks), dim3(kStdpRowsBlock), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_deliver_lds(hipStream_t s, const DeliverArgs &a, int blocks, size_t lds)
{
    static std::mutex mu;
    static int granted = 64 * 1024;
    const hipError_t e = allow_dynamic_lds((const void *)k_deliver_lds, (int)lds, mu, granted);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_deliver_lds, dim3(blocks), dim3(kDlvBlock), lds, s, a);
    return hipGetLastError();
}

hipError_t launch_deliver_global(hipStream_t s, const DeliverArgs &a, int blocks)
{
    hipLaunchKernelGGL(k_deliver_global, dim3(blocks), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

int deliver_lds_static_bytes() { return static_lds_bytes((const void *)k_deliver_lds); }
int stdp_static_bytes() { return static_lds_bytes((const void *)k_stdp); }

}  // namespace snn
