// gfx950 kernels of the neuron part of a step: state initialisation and
// fills, the neuron update (firing masks, histories, post traces) and the
// compaction of spike / transmitted / forced lists with row snapshots.
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
// (1) neuron update. One thread per neuron, one wave64 per mask word.

__global__ __launch_bounds__(kBlock) void k_neuron(NeuronArgs a)
{
    const int tid = threadIdx.x;
    const int i = blockIdx.x * kBlock + tid;
    int s = 0, tx = 0, forced = 0;
    bool fired_recently = false;
    if (i < a.n) {
        if (a.model == 2) {
            s = rng32(a.seed, 4, (uint64_t)a.t, (uint64_t)i) < a.fire_thr;
        } else {
            float ae, ai = 0.f;
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
            float v = a.v[i];
            int r = a.ref[i];
            if (a.model == 1) {
                const float ie = __fadd_rn(__fmul_rn(a.ie[i], a.d_e), ae);
                const float ii = __fadd_rn(__fmul_rn(a.ii[i], a.d_i), ai);
                a.ie[i] = ie;
                a.ii[i] = ii;
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
                        const uint32_t u = rng32(a.seed, 3, (uint64_t)a.t, (uint64_t)i);
                        int k = 0;
                        for (int q = 0; q < a.poisson_len; ++q) k += (a.poisson[q] <= u);
                        x = __fmul_rn(a.j_ext, (float)k);
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
            a.v[i] = v;
            a.ref[i] = r;
        }
        uint64_t *hp = a.hist + (int64_t)i * a.hw;
        uint64_t h = hp[0];
        uint64_t h1 = a.hw == 2 ? hp[1] : 0ull;
        if (a.n_plastic_rows > 0) {
            // post trace seen by a pre spike at step t: posts strictly before t
            const float y = __fmul_rn(__fadd_rn(a.ypost[i], (float)(h & 1ull)), a.d_minus);
            a.ypost[i] = y;
        }
        h1 = a.hw == 2 ? (h1 << 1) | (h >> 63) : 0ull;
        h = (h << 1) | (uint64_t)s;
        hp[0] = h;
        if (a.hw == 2) hp[1] = h1;
        // history code for the row-wise STDP of this step: the position + 1 of
        // the only spike of the last 64 hw steps (bit b = step t-b), 0 for none
        const int np = __popcll(h) + __popcll(h1);
        const int pos = h ? __ffsll((long long)h) : 64 + __ffsll((long long)h1);
        a.code[i] = np == 0 ? (uint8_t)0 : np == 1 ? (uint8_t)pos : kCodeMulti;
        fired_recently = np != 0;
        tx = (int)((h >> a.dm1) & 1ull);
        if (i < a.n_plastic_rows) forced = !tx && (a.t - (int64_t)a.t_last[i] >= 64 * a.hw);
    }
    const uint64_t m = ballot64(s), txm = ballot64(tx), fm = ballot64(forced);
    const uint64_t rcm = ballot64(fired_recently);
    const int wave = tid / kWave, lane = tid % kWave;
    const int64_t word = (int64_t)blockIdx.x * (kBlock / kWave) + wave;
    __shared__ int s_cnt[3][kBlock / kWave];
    if (lane == 0) {
        if (word * kWave < a.n) {
            a.mask[word] = m;
            a.txmask[word] = txm;
            a.fmask[word] = fm;
            a.recent[word] = rcm;
        }
        s_cnt[0][wave] = __popcll(m);
        s_cnt[1][wave] = __popcll(txm);
        s_cnt[2][wave] = __popcll(fm);
    }
    __syncthreads();
    if (tid == 0) {
        int c0 = 0, c1 = 0, c2 = 0;
#pragma unroll
        for (int q = 0; q < kBlock / kWave; ++q) {
            c0 += s_cnt[0][q];
            c1 += s_cnt[1][q];
            c2 += s_cnt[2][q];
        }
        a.blk_spk[blockIdx.x] = c0;
        a.blk_tx[blockIdx.x] = c1;
        a.blk_f[blockIdx.x] = c2;
    }
}

// Ascending lists from the masks: each workgroup adds the counts of the
// workgroups before it, then ranks its bits. Spikes go to the delay-ring
// slot of step t; forced plastic rows to the forced list with their
// snapshots; each transmitting plastic row gets its snapshot at its position
// in the transmitted list (the ring list of step t-D+1, which holds the same
// neurons in the same ascending order).
__global__ __launch_bounds__(kBlock) void k_compact(CompactArgs a)
{
    __shared__ long long sh[kBlock / kWave];
    __shared__ int s_pc[3][kBlock / kWave];
    __shared__ float s_dpow[kMaxAge + 1];
    const int tid = threadIdx.x, b = blockIdx.x;
    for (int q = tid; q <= kMaxAge; q += kBlock) s_dpow[q] = a.dpow[q];
    long long p0 = 0, p1 = 0, p2 = 0;
    for (int q = tid; q < b; q += kBlock) {
        p0 += a.blk_spk[q];
        p1 += a.blk_tx[q];
        p2 += a.blk_f[q];
    }
    // pack two prefix sums into one reduction (each < 2^31)
    const long long packed = block_sum_i64((p0 << 32) | p1, sh);
    p0 = packed >> 32;
    p1 = packed & 0xffffffffll;
    p2 = block_sum_i64(p2, sh);
    const int wave = tid / kWave, lane = tid % kWave;
    const int64_t word = (int64_t)b * (kBlock / kWave) + wave;
    const bool inb = word < a.nw;
    const uint64_t m = inb ? a.mask[word] : 0ull;
    const uint64_t txm = inb ? a.txmask[word] : 0ull;
    const uint64_t fm = inb ? a.fmask[word] : 0ull;
    if (lane == 0) {
        s_pc[0][wave] = __popcll(m);
        s_pc[1][wave] = __popcll(txm);
        s_pc[2][wave] = __popcll(fm);
    }
    __syncthreads();
    int o0 = (int)p0, o1 = (int)p1, o2 = (int)p2, t0 = 0, t2 = 0;
#pragma unroll
    for (int q = 0; q < kBlock / kWave; ++q) {
        if (q < wave) {
            o0 += s_pc[0][q];
            o1 += s_pc[1][q];
            o2 += s_pc[2][q];
        }
        t0 += s_pc[0][q];
        t2 += s_pc[2][q];
    }
    const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
    const int i = (int)(word * kWave) + lane;
    if ((m >> lane) & 1ull) a.spk_list[o0 + __popcll(m & below)] = i;
    long long st_rows = 0, st_forced = 0, st_syn = 0, st_fsyn = 0;
    if ((txm >> lane) & 1ull) {
        RowInfo ri;
        if (i < a.n_plastic_rows &&
            make_row_info(ri, i, a.t, true, a.dm1, a.hw, a.row_ptr, a.pend, a.hist, a.t_last, a.xpre,
                          s_dpow, a.err)) {
            st_rows = 1;
            st_syn = ri.len;
        } else {
            ri.k = i;
            ri.rs = a.row_ptr[i];
            ri.len = 0;
            ri.age_pre = 0;
            ri.xp0 = ri.xp_now = 0.f;
            ri.pad = 0;
        }
        a.txinfo[o1 + __popcll(txm & below)] = ri;
    }
    if ((fm >> lane) & 1ull) {
        const int r = o2 + __popcll(fm & below);
        a.row_list[r] = i;
        RowInfo ri;
        if (make_row_info(ri, i, a.t, true, a.dm1, a.hw, a.row_ptr, a.pend, a.hist, a.t_last, a.xpre,
                          s_dpow, a.err)) {
            st_rows += 1;
            st_forced = 1;
            st_syn += ri.len;
            st_fsyn = ri.len;
        }
        a.info[r] = ri;
    }
    if (b == (int)gridDim.x - 1 && tid == 0) {
        *a.spk_cnt = (int)p0 + t0;
        *a.row_cnt = (int)p2 + t2;
        a.gstats[kGSpikes] += (int)p0 + t0;
    }
    if (a.info_stats) {
        st_rows = block_sum_i64(st_rows, sh);
        st_forced = block_sum_i64(st_forced, sh);
        st_syn = block_sum_i64(st_syn, sh);
        st_fsyn = block_sum_i64(st_fsyn, sh);
        if (tid == 0) {
            int64_t *slot = a.info_stats + (int64_t)b * kStFields;
            slot[kStRows] += st_rows;
            slot[kStForced] += st_forced;
            slot[kStSyn] += st_syn;
            slot[kStForcedSyn] += st_fsyn;
        }
    }
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

hipError_t launch_neuron(hipStream_t s, const NeuronArgs &a, KernelEvents ev)
{
    hipExtLaunchKernelGGL(k_neuron, dim3(blocks_for(a.n)), dim3(kBlock), 0, s,
                          ev.start, ev.stop, 0, a);
    return hipGetLastError();
}

hipError_t launch_compact(hipStream_t s, const CompactArgs &a, KernelEvents ev)
{
    hipExtLaunchKernelGGL(k_compact, dim3(blocks_for(a.n)), dim3(kBlock), 0, s,
                          ev.start, ev.stop, 0, a);
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
