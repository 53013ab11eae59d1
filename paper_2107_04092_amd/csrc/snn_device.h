// Device helpers shared by the gfx950 kernels of the synapse pass: the
// counter-based generator, wave/workgroup reductions and scans, the segment
// map of flattened row segments, fixed-point accumulation, row snapshots and
// the per-synapse STDP update.
#pragma once

#include "snn_internal.h"

#include <hip/hip_ext.h>

#include <mutex>
#include <utility>

namespace snn {
namespace {

// ---------------------------------------------------------------------------
// helpers

// SplitMix64 output function (Steele, Lea & Flood 2014) of seed XOR key, with
// key = stream << 58 | a << 24 | b: a counter-based draw per (stream, a, b).
__device__ __forceinline__ uint32_t rng32(uint64_t seed, uint32_t stream, uint64_t a,
                                          uint64_t b)
{
    uint64_t z = (seed ^ (((uint64_t)stream << 58) | (a << 24) | b)) + 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    return (uint32_t)(z >> 32);
}

__device__ __forceinline__ uint64_t ballot64(bool p) { return __builtin_amdgcn_ballot_w64(p); }

// w^mu for w >= 0 and 0 <= mu < 1, as 2^(mu log2 w) on the hardware
// transcendental unit (v_log_f32 / v_exp_f32, about 1 ulp each): relative
// error around 1e-7, against a few hundred instructions for a libm powf.
__device__ __forceinline__ float pow_mu(float w, float mu)
{
    if (mu == 0.f) return 1.f;
    // computed unconditionally and selected: no divergent branch per call
    const float p = __builtin_amdgcn_exp2f(mu * __builtin_amdgcn_logf(w));
    return w > 0.f ? p : 0.f;
}

// fp32 -> fixed point (x * 2^32 is exact in fp32; only |x| < 2^-9 loses bits)
__device__ __forceinline__ long long to_fix(float x) { return __float2ll_rn(x * kFixScale); }
// fixed point -> fp32, one correctly rounded conversion (the scaling is exact)
__device__ __forceinline__ float from_fix(long long s) { return __ll2float_rn(s) * kFixUnit; }

// Adds v to a 64-bit counter in global memory without waiting for it (an
// atomic whose result is unused needs no round trip; a read-modify-write
// would wait for the read).
__device__ __forceinline__ void add_stat(int64_t *p, long long v)
{
    if (v) (void)atomicAdd((unsigned long long *)p, (unsigned long long)v);
}

// Wave-wide scans by DPP lane moves (VALU operations: no LDS round trip per
// step, unlike shuffles). dpp_mov<CTRL, RM> returns, per lane, x of the lane
// CTRL selects, or id where that lane does not exist or the lane's row is
// not in the row mask RM.
template <int CTRL, int RM>
__device__ __forceinline__ int dpp_mov(int x, int id)
{
    return __builtin_amdgcn_update_dpp(id, x, CTRL, RM, 0xf, false);
}
template <int CTRL, int RM>
__device__ __forceinline__ long long dpp_mov(long long x, long long id)
{
    const int lo = __builtin_amdgcn_update_dpp((int)id, (int)x, CTRL, RM, 0xf, false);
    const int hi = __builtin_amdgcn_update_dpp((int)(id >> 32), (int)(x >> 32), CTRL, RM, 0xf,
                                               false);
    return (long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo);
}
constexpr int kDppRowShr1 = 0x111, kDppRowShr2 = 0x112, kDppRowShr4 = 0x114,
              kDppRowShr8 = 0x118, kDppRowBcast15 = 0x142, kDppRowBcast31 = 0x143,
              kDppWaveShr1 = 0x138;

// Inclusive scan over the 64 lanes with the associative op (identity id):
// shifts by 1, 2, 4, 8 inside each row of 16 lanes, then lane 15 of rows 0
// and 2 into rows 1 and 3, then lane 31 into rows 2 and 3.
template <typename T, typename Op>
__device__ __forceinline__ T wave_incl_scan(T x, T id, Op op)
{
    x = op(x, dpp_mov<kDppRowShr1, 0xf>(x, id));
    x = op(x, dpp_mov<kDppRowShr2, 0xf>(x, id));
    x = op(x, dpp_mov<kDppRowShr4, 0xf>(x, id));
    x = op(x, dpp_mov<kDppRowShr8, 0xf>(x, id));
    x = op(x, dpp_mov<kDppRowBcast15, 0xa>(x, id));
    x = op(x, dpp_mov<kDppRowBcast31, 0xc>(x, id));
    return x;
}
// The value of the previous lane (lane 0: id).
template <typename T>
__device__ __forceinline__ T wave_shr1(T x, T id)
{
    return dpp_mov<kDppWaveShr1, 0xf>(x, id);
}
struct AddOp {
    template <typename T>
    __device__ __forceinline__ T operator()(T a, T b) const { return a + b; }
};
struct MaxOp {
    template <typename T>
    __device__ __forceinline__ T operator()(T a, T b) const { return a > b ? a : b; }
};

__device__ __forceinline__ int wave_sum_i32(int v)
{
    return __builtin_amdgcn_readlane(wave_incl_scan(v, 0, AddOp{}), kWave - 1);
}

__device__ __forceinline__ long long wave_sum_i64(long long v)
{
    const long long s = wave_incl_scan(v, 0ll, AddOp{});
    const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)s, kWave - 1);
    const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(s >> 32), kWave - 1);
    return (long long)(((unsigned long long)hi << 32) | lo);
}

// Copies count > 0 elements from global memory into LDS with an NT-thread
// workgroup, R loads in flight per thread before their stores (a plain
// strided loop would wait for each load before the next).
template <int NT, int R, typename T>
__device__ __forceinline__ void stage_lds(T *dst, const T *__restrict__ src, int count,
                                          int from = 0)
{
    for (int x0 = from; x0 < count; x0 += NT * R) {
        T v[R];
#pragma unroll
        for (int r = 0; r < R; ++r) v[r] = src[min(x0 + r * NT + (int)threadIdx.x, count - 1)];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int x = x0 + r * NT + (int)threadIdx.x;
            if (x < count) dst[x] = v[r];
        }
    }
}

// The same in two halves, so that other loads can go out in between: the
// first R NT elements are loaded into registers by stage_issue, stored by
// stage_finish, which then copies the rest.
template <int R, typename T>
struct StageRegs {
    T v[R];
};

template <int NT, int R, typename T>
__device__ __forceinline__ void stage_issue(StageRegs<R, T> &g, const T *__restrict__ src,
                                            int count)
{
#pragma unroll
    for (int r = 0; r < R; ++r) g.v[r] = src[min(r * NT + (int)threadIdx.x, count - 1)];
}

template <int NT, int R, typename T>
__device__ __forceinline__ void stage_finish(T *dst, const StageRegs<R, T> &g,
                                             const T *__restrict__ src, int count)
{
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int x = r * NT + (int)threadIdx.x;
        if (x < count) dst[x] = g.v[r];
    }
    stage_lds<NT, R>(dst, src, count, NT * R);
}

// Number of lanes below this one whose bit is set in a wave-uniform mask.
__device__ __forceinline__ int lane_rank(uint64_t m)
{
    return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                          __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Sum over a kBlock-thread workgroup; every thread gets the total.
__device__ __forceinline__ long long block_sum_i64(long long v, long long *sh)
{
    v = wave_sum_i64(v);
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    __syncthreads();
    if (lane == 0) sh[wave] = v;
    __syncthreads();
    long long t = 0;
#pragma unroll
    for (int q = 0; q < kBlock / kWave; ++q) t += sh[q];
    return t;
}

// Sum / inclusive scan over a NT-thread workgroup (sh: NT/64 entries).
template <int NT>
__device__ __forceinline__ long long block_sum_i64_n(long long v, long long *sh)
{
    v = wave_sum_i64(v);
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    __syncthreads();
    if (lane == 0) sh[wave] = v;
    __syncthreads();
    long long t = 0;
#pragma unroll
    for (int q = 0; q < NT / kWave; ++q) t += sh[q];
    return t;
}

template <int NT>
__device__ __forceinline__ long long block_incl_scan_i64_n(long long v, long long *sh)
{
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    v = wave_incl_scan(v, 0ll, AddOp{});
    __syncthreads();
    if (lane == kWave - 1) sh[wave] = v;
    __syncthreads();
    for (int q = 0; q < wave; ++q) v += sh[q];
    return v;
}

// Segment map of a window of flattened elements. On entry mark[x] holds the
// index of the (non-empty) segment that starts at x, or `none`; on exit every
// entry holds the index of the segment containing x (an inclusive max-scan,
// valid because segment indices grow with their start offsets; `none` is
// below every index). NT threads, E consecutive entries each; len <= E NT.
// Ends with a barrier.
template <int NT, int E = 4, typename T = int>
__device__ __forceinline__ void fill_segment_map(T *mark, int len, int *sh, int none = -1)
{
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    int v[E], m = none;
#pragma unroll
    for (int q = 0; q < E; ++q) {
        const int x = E * tid + q;
        const int u = x < len ? (int)mark[x] : none;
        m = max(m, u);
        v[q] = m;
    }
    const int inc = wave_incl_scan(m, none, MaxOp{});
    if (lane == kWave - 1) sh[wave] = inc;
    __syncthreads();
    int excl = wave_shr1(inc, none);
    for (int q = 0; q < wave; ++q) excl = max(excl, sh[q]);
#pragma unroll
    for (int q = 0; q < E; ++q) {
        const int x = E * tid + q;
        if (x < len) mark[x] = (T)max(excl, v[q]);
    }
    __syncthreads();
}


// The decay-table index of a row of t_last t_last_k brought up to step t:
// its age, at most the history's 64 hw steps (0 for a row already current).
__device__ __forceinline__ int row_age_index(int64_t t, int t_last_k, int hw)
{
    const int age = (int)(t - (int64_t)t_last_k);
    return age <= 0 ? 0 : min(age, 64 * hw);
}

// Snapshot of plastic row k for an update at step t (see RowInfo) from the
// row's values: t_last, first edge rs, plastic prefix length, pre trace at
// t_last, and whether the row transmits at t; dp_age = d_plus^age at
// row_age_index. Returns 1 if the row has something to bring up to date.
__device__ __forceinline__ int make_row_info_d(RowInfo &ri, int k, int64_t t, int t_last_k,
                                               int64_t rs, int pend_k, float xpre_k, int pre,
                                               int hw, float dp_age, int32_t *err)
{
    int age = (int)(t - (int64_t)t_last_k);
    ri.k = k;
    ri.rs = rs;
    ri.pad = 0;
    ri.xp0 = xpre_k;
    if (age <= 0) {  // flush: already current
        ri.len = 0;
        ri.age_pre = 0;
        ri.xp_now = ri.xp0;
        return 0;
    }
    if (age > 64 * hw) {
        // the plasticity part was skipped for this row: posts older than the
        // history are lost; flag it and stay inside the table
        atomicOr(err, kErrWindow);
        age = 64 * hw;
    }
    ri.len = pend_k;
    ri.age_pre = age | (pre << 8);
    ri.xp_now = __fadd_rn(__fmul_rn(ri.xp0, dp_age), (float)pre);
    return 1;
}

// The same with the decay table.
__device__ __forceinline__ int make_row_info_v(RowInfo &ri, int k, int64_t t, int t_last_k,
                                               int64_t rs, int pend_k, float xpre_k, int pre,
                                               int hw, const float *dpow, int32_t *err)
{
    return make_row_info_d(ri, k, t, t_last_k, rs, pend_k, xpre_k, pre, hw,
                           dpow[row_age_index(t, t_last_k, hw)], err);
}

// The same reading the values from the state arrays.
__device__ __forceinline__ int make_row_info(RowInfo &ri, int k, int64_t t, bool pre_allowed,
                                             int dm1, int hw, const int64_t *row_ptr,
                                             const int32_t *pend, const uint64_t *hist,
                                             const int32_t *t_last, const float *xpre,
                                             const float *dpow, int32_t *err)
{
    const int pre = pre_allowed ? (int)((hist[(int64_t)k * hw] >> dm1) & 1ull) : 0;
    return make_row_info_v(ri, k, t, t_last[k], row_ptr[k], pend[k], xpre[k], pre, hw, dpow,
                           err);
}

// Masks of the window of a row of age `age` (bits age-1 .. 0 of the
// history, word 0 = the last 64 steps, word 1 = the 64 before).
__device__ __forceinline__ void window_masks(int age, uint64_t &m0, uint64_t &m1)
{
    m0 = age >= 64 ? ~0ull : ((1ull << age) - 1ull);
    m1 = age >= 128 ? ~0ull : age > 64 ? ((1ull << (age - 64)) - 1ull) : 0ull;
}

// One synapse k->j brought from t_last to t (age = t - t_last; h0, h1 the
// window bits of the target's history words 0 and 1; pre = transmitting at
// t). Returns the new weight.
__device__ __forceinline__ float stdp_synapse(float w, uint64_t h0, uint64_t h1, int age,
                                              int pre, float xp0, float xp_now, float y,
                                              const float *dpow, float c_pot, float c_dep,
                                              float mu)
{
    while (h1) {  // posts 64 .. 127 steps ago, oldest first
        const int bit = 63 - __clzll((long long)h1);
        h1 ^= 1ull << bit;
        w = w + c_pot * pow_mu(w, mu) * __fmul_rn(xp0, dpow[age - 64 - bit]);
    }
    uint64_t older = h0 & ~1ull;
    while (older) {  // posts before t, oldest first
        const int bit = 63 - __clzll((long long)older);
        older ^= 1ull << bit;
        w = w + c_pot * pow_mu(w, mu) * __fmul_rn(xp0, dpow[age - bit]);
    }
    if (pre) {  // pre at t sees the posts strictly before t
        w = w - c_dep * w * y;
        w = fmaxf(w, 0.f);
    }
    if (h0 & 1ull) w = w + c_pot * pow_mu(w, mu) * xp_now;  // post at t
    return w;
}

// The same update stepping through every step of the window (lazy but not
// event-driven, Fig. 2(b)): the pre trace decays one step at a time and every
// history bit is tested. Differs from stdp_synapse only in the rounding of
// the decayed pre trace.
__device__ __forceinline__ float stdp_synapse_steps(float w, uint64_t h0, uint64_t h1, int age,
                                                    int pre, float xp0, float xp_now, float y,
                                                    float d_plus, float c_pot, float c_dep,
                                                    float mu)
{
    float xp = xp0;
    for (int s = age - 1; s >= 1; --s) {  // steps t-s before t, oldest first
        xp = xp * d_plus;
        const uint64_t bit = s < 64 ? (h0 >> s) & 1ull : (h1 >> (s - 64)) & 1ull;
        if (bit) w = w + c_pot * pow_mu(w, mu) * xp;
    }
    if (pre) {
        w = w - c_dep * w * y;
        w = fmaxf(w, 0.f);
    }
    if (h0 & 1ull) w = w + c_pot * pow_mu(w, mu) * xp_now;
    return w;
}

// Delay-ring slot of a step (steps before 0 wrap like the ring).
__device__ __forceinline__ int ring_slot(int64_t step, int d)
{
    const int64_t r = step % d;
    return (int)(r < 0 ? r + d : r);
}

// A list scan's status word (see kStatusAgg): counts a and b of step t.
__device__ __forceinline__ unsigned long long status_word(int a, int b, int64_t t,
                                                          unsigned long long kind)
{
    return (unsigned long long)(uint32_t)a | ((unsigned long long)(uint32_t)b << 24) |
           ((unsigned long long)(t & 0x3fff) << 48) | kind;
}

// The step clock read with vector loads (relaxed, device scope): unlike a
// scalar load, its wait does not join the wait for the kernel arguments.
__device__ __forceinline__ StepClock load_clock(const StepClock *c)
{
    StepClock k{};
    k.t = __hip_atomic_load(&c->t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const long long f = __hip_atomic_load(reinterpret_cast<const long long *>(&c->input_forced),
                                          __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    k.input_forced = (int32_t)(uint32_t)f;
    k.n_parts = (int32_t)(f >> 32);
    return k;
}

__device__ __forceinline__ void publish_status(unsigned long long *p, unsigned long long w)
{
    __hip_atomic_store(p, w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Exclusive prefix, over the workgroups before workgroup b, of the two
// counts of `nscan` (<= R) list scans, by decoupled look-back. Scan r keeps
// its status words at status + r * stride (one per workgroup) and belongs to
// step t0 + r. The NT threads read a window of NT predecessors at once
// (thread i: workgroup base - 1 - i). In each scan the nearest predecessor
// that has published an inclusive prefix ends the walk; every workgroup
// between it and b must have published its own counts for that step, else
// the window is read again. Workgroup 0 publishes an inclusive prefix
// without waiting, so every walk ends once the workgroups before b have
// started, which in-order dispatch guarantees. The wait is bounded: after
// kLookbackSpins rounds the error flag is raised and the counts found so far
// are used (list writers check their offsets). Called by every thread of
// the workgroup with workgroup-uniform arguments. The state of each scan
// lives in LDS (sh: 8 R ints); on return sh[8 r + 6] and sh[8 r + 7] hold
// scan r's two prefixes.
template <int NT, int R>
__device__ void lookback(unsigned long long *status, int64_t stride, int nscan, int b,
                         int64_t t0, int *sh, int32_t *err)
{
    // sh[8 r + ...]: 0 nearest inclusive in the window (NT: none), 1 lanes
    // not yet published, 2-3 the window's sums, 4 window end, 5 done, 6-7 prefixes
    const int tid = threadIdx.x, lane = tid % kWave;
    // thread tid reads the predecessor at distance 1 + d in the window: wave
    // 0, whose thread 0 has just stored this workgroup's status, takes the
    // farthest distances (none in a grid of at most NT - 63 workgroups), so
    // the reads the scan waits for are not queued behind that store
    const int d = (tid + NT - kWave) % NT;
    if (tid < R) {
        int *q = sh + 8 * tid;
        q[4] = b;
        q[5] = b == 0 || tid >= nscan;
        q[6] = q[7] = 0;
    }
    // the earlier workgroups publish at about the same time as this one: a
    // read issued at once mostly finds their words not yet visible and
    // costs a second round trip (measured: 0.6 us more per launch)
    if (b > 0) __builtin_amdgcn_s_sleep(kLookbackDelay);
    __syncthreads();
    for (int rounds = 0;; ++rounds) {
        bool all = true;
#pragma unroll
        for (int r = 0; r < R; ++r) all = all && sh[8 * r + 5] != 0;
        if (all) break;
        if (rounds >= kLookbackSpins) {
            if (tid == 0) atomicOr(err, kErrLookback);
            break;
        }
        unsigned long long w[R];
#pragma unroll
        for (int r = 0; r < R; ++r) {  // every read of the round in flight together
            const int p = sh[8 * r + 4] - 1 - d;
            w[r] = 0ull;
            if (!sh[8 * r + 5] && p >= 0)
                w[r] = __hip_atomic_load(status + r * stride + p, __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_AGENT);
        }
        __syncthreads();  // window ends read before the per-round fields are reset
        if (tid < R) {
            sh[8 * tid] = NT;
            sh[8 * tid + 1] = sh[8 * tid + 2] = sh[8 * tid + 3] = 0;
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < R; ++r) {  // the nearest inclusive prefix of the window
            if (sh[8 * r + 5]) continue;
            const unsigned tag = (unsigned)((t0 + r) & 0x3fff);
            const bool inc = sh[8 * r + 4] - 1 - d >= 0 && (w[r] >> 62) == 2ull &&
                             (unsigned)((w[r] >> 48) & 0x3fff) == tag;
            const uint64_t bl = ballot64(inc);  // (d rises with the lane)
            if (bl && lane == __ffsll((long long)bl) - 1) atomicMin(&sh[8 * r], d);
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < R; ++r) {  // counts up to it; predecessors not yet published
            if (sh[8 * r + 5]) continue;
            const unsigned tag = (unsigned)((t0 + r) & 0x3fff);
            const bool need = sh[8 * r + 4] - 1 - d >= 0 && d <= sh[8 * r];
            const bool cur = (w[r] >> 62) != 0ull && (unsigned)((w[r] >> 48) & 0x3fff) == tag;
            const uint64_t bad = ballot64(need && !cur);
            int va = need && cur ? (int)(w[r] & 0xffffffull) : 0;
            int vb = need && cur ? (int)((w[r] >> 24) & 0xffffffull) : 0;
            va = wave_sum_i32(va);
            vb = wave_sum_i32(vb);
            if (lane == 0) {
                if (bad) atomicAdd(&sh[8 * r + 1], (int)__popcll(bad));
                if (va) atomicAdd(&sh[8 * r + 2], va);
                if (vb) atomicAdd(&sh[8 * r + 3], vb);
            }
        }
        __syncthreads();
        if (tid < R && !sh[8 * tid + 5] && sh[8 * tid + 1] == 0) {  // the window is complete
            int *q = sh + 8 * tid;
            q[6] += q[2];
            q[7] += q[3];
            if (q[0] < NT || q[4] <= NT)
                q[5] = 1;
            else
                q[4] -= NT;
        }
        __syncthreads();
        bool retry = false;
#pragma unroll
        for (int r = 0; r < R; ++r) retry = retry || (!sh[8 * r + 5] && sh[8 * r + 1] != 0);
        if (retry) __builtin_amdgcn_s_sleep(4);
    }
}

// The same for up to NT/32 scans, one per half wave: scan r is looked back
// over by threads 32 r .. 32 r + 31, a window of 32 predecessors at a time,
// with ballots and lane moves inside the wave, so the scans need no
// workgroup barrier until the end. On return out[2 r], out[2 r + 1] (LDS)
// hold scan r's two prefixes. Bounded as above.
template <int NT>
__device__ void lookback32(unsigned long long *status, int64_t stride, int nscan, int b,
                           int64_t t0, int *out, int32_t *err)
{
    static_assert(NT % kWave == 0, "whole waves");
    const int tid = threadIdx.x, lane = tid % kWave;
    const int r = tid >> 5, gi = tid & 31, half = lane >> 5;
    const bool active = r < nscan;
    const unsigned tag = (unsigned)((t0 + r) & 0x3fff);
    int base = b, acc_a = 0, acc_b = 0;
    bool done = !active || b == 0;
    if (b > 0) __builtin_amdgcn_s_sleep(kLookbackDelay);  // as in lookback
    for (int rounds = 0;; ++rounds) {
        if (!ballot64(!done)) break;  // both scans of the wave complete
        if (rounds >= kLookbackSpins) {
            if (!done && gi == 0) atomicOr(err, kErrLookback);
            break;
        }
        const int p = base - 1 - gi;
        unsigned long long w = 0ull;
        if (!done && p >= 0)
            w = __hip_atomic_load(status + r * stride + p, __ATOMIC_RELAXED,
                                  __HIP_MEMORY_SCOPE_AGENT);
        const bool cur = (w >> 62) != 0ull && (unsigned)((w >> 48) & 0x3fff) == tag;
        const uint32_t incm =
            (uint32_t)(ballot64(cur && p >= 0 && (w >> 62) == 2ull) >> (32 * half));
        const int ip = incm ? __ffs((int)incm) - 1 : 32;  // nearest inclusive prefix
        const bool need = !done && p >= 0 && gi <= ip;
        const uint32_t badm = (uint32_t)(ballot64(need && !cur) >> (32 * half));
        int va = need && cur ? (int)(w & 0xffffffull) : 0;
        int vb = need && cur ? (int)((w >> 24) & 0xffffffull) : 0;
        {  // sums inside the half wave: lanes 31 and 63 of a wave scan
            const int sa = wave_incl_scan(va, 0, AddOp{}), sb = wave_incl_scan(vb, 0, AddOp{});
            const int a31 = __builtin_amdgcn_readlane(sa, 31), a63 = __builtin_amdgcn_readlane(sa, 63);
            const int b31 = __builtin_amdgcn_readlane(sb, 31), b63 = __builtin_amdgcn_readlane(sb, 63);
            va = half ? a63 - a31 : a31;
            vb = half ? b63 - b31 : b31;
        }
        if (!done && badm == 0) {
            acc_a += va;
            acc_b += vb;
            if (ip < 32 || base <= 32)
                done = true;
            else
                base -= 32;
        }
        if (ballot64(!done && badm != 0)) __builtin_amdgcn_s_sleep(4);
    }
    if (active && gi == 0) {
        out[2 * r] = acc_a;
        out[2 * r + 1] = acc_b;
    }
    __syncthreads();
}

inline int blocks_for(int64_t count, int per = kBlock, int64_t cap = 1 << 20)
{
    int64_t b = (count + per - 1) / per;
    if (b < 1) b = 1;
    if (b > cap) b = cap;
    return (int)b;
}

// Launches a kernel; with events, the launch places them around the kernel
// itself (hipExtLaunchKernelGGL), else it is a plain launch, which a stream
// capture can record.
template <typename... KArgs, typename... Args>
inline void launch_kernel(void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t lds,
                          hipStream_t s, KernelEvents ev, Args &&...args)
{
    if (ev.start || ev.stop)
        hipExtLaunchKernelGGL(kernel, grid, block, lds, s, ev.start, ev.stop, 0,
                              std::forward<Args>(args)...);
    else
        hipLaunchKernelGGL(kernel, grid, block, lds, s, std::forward<Args>(args)...);
}

// Raises a kernel's dynamic-LDS limit to `bytes` (once per size increase).
inline hipError_t allow_dynamic_lds(const void *kernel, int bytes, std::mutex &mu, int &granted)
{
    std::lock_guard<std::mutex> lock(mu);
    if (bytes <= granted) return hipSuccess;
    const hipError_t e =
        hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (e != hipSuccess) {
        (void)hipGetLastError();  // do not leave the error for the next launch
        return e;
    }
    granted = bytes;
    return hipSuccess;
}

inline int static_lds_bytes(const void *kernel)
{
    hipFuncAttributes attr{};
    if (hipFuncGetAttributes(&attr, kernel) != hipSuccess) {
        (void)hipGetLastError();
        return -1;
    }
    return (int)attr.sharedSizeBytes;
}

}  // namespace
}  // namespace snn
