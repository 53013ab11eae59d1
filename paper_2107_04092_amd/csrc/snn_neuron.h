// Neuron-update helpers shared by the kernels that run the neuron part of a
// step (k_neuron.hip: one step, small networks, delay blocks; k_block.hip:
// plastic blocks): the state one update reads and writes, its input, and the
// update itself in a fixed fp32 operation order. Every file that includes
// this is built with -ffp-contract=off.
#pragma once

#include "snn_device.h"

namespace snn {
namespace {

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

// The input A(t) of neuron i from the state: the fp32 input (forced), or the
// sum of the n_parts fixed-point partial sums of delivery. Which one the
// clock says is known only when its load returns, so the fp32 input and up
// to kSpecParts partial sums (a.max_parts of them) are loaded before it is
// looked at: one round trip instead of two.
constexpr int kSpecParts = 8;
struct InputLoads {
    float fe, fi;
    long long pe[kSpecParts], pi[kSpecParts];
};
__device__ __forceinline__ void input_issue(const NeuronArgs &a, int i, InputLoads &L)
{
    const bool cuba = a.model == 1;
    L.fe = a.ain[i];
    L.fi = cuba ? a.ain[a.n + i] : 0.f;
#pragma unroll
    for (int c = 0; c < kSpecParts; ++c) {
        L.pe[c] = c < a.max_parts ? a.apart[c * a.part_stride + i] : 0;
        L.pi[c] = cuba && c < a.max_parts ? a.apart[c * a.part_stride + a.n + i] : 0;
    }
}
__device__ __forceinline__ void input_combine(const NeuronArgs &a, const InputLoads &L, int forced,
                                              int n_parts, int i, float &ae, float &ai)
{
    const bool cuba = a.model == 1;
    ai = 0.f;
    if (forced) {
        ae = L.fe;
        ai = L.fi;
        return;
    }
    long long se = 0, si = 0;
#pragma unroll
    for (int c = 0; c < kSpecParts; ++c) {
        if (c < n_parts) {
            se += L.pe[c];
            si += L.pi[c];
        }
    }
    for (int c = kSpecParts; c < n_parts; ++c) {  // beyond the speculative loads
        se += a.apart[c * a.part_stride + i];
        if (cuba) si += a.apart[c * a.part_stride + a.n + i];
    }
    ae = from_fix(se);
    if (cuba) ai = from_fix(si);
}
__device__ __forceinline__ void neuron_input(const NeuronArgs &a, int forced, int n_parts, int i,
                                             float &ae, float &ai)
{
    InputLoads L;
    input_issue(a, i, L);
    input_combine(a, L, forced, n_parts, i, ae, ai);
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

}  // namespace
}  // namespace snn
