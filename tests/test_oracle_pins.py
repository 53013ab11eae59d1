"""Pins of the CPU oracle against things other than itself (no GPU needed).

Each test fixes part of the oracle with a value printed in the paper, a
published reference output, a closed form, an independent formulation
(brute force over explicit spike lists) or an invariant, chosen so that a
dropped term, a wrong sign, a wrong history bit or a swapped operand fails.
"""

import json
import math
import os

import numpy as np
import pytest

import workloads as wl
from workloads.presets import (LIF_DELTA, LIF_CUBA, BERNOULLI_SOURCE, PLASTIC_ALL,
                               PLASTIC_EXC_EXC, PLASTIC_NONE, GRAPH_BERNOULLI,
                               GRAPH_FIXED_FANOUT)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
pytestmark = pytest.mark.filterwarnings("ignore")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# --------------------------------------------------------------------------
# counter-based generator

def test_splitmix64_published_vectors(orc):
    g = _golden("splitmix64.json")
    gamma = 0x9E3779B97F4A7C15
    for seed, outs in g["sequences"].items():
        for q, want in enumerate(outs):
            want = int(want, 0)
            state = (int(seed) + q * gamma) % (1 << 64)
            assert orc.splitmix64(state) == want
            assert int(wl.splitmix64_mix(np.uint64(state))) == want


def test_rng_two_implementations_agree(orc):
    rs = np.random.default_rng(1)
    for _ in range(200):
        seed = int(rs.integers(0, 1 << 63))
        stream = int(rs.integers(0, 64))
        a = int(rs.integers(0, 1 << 34))
        b = int(rs.integers(0, 1 << 24))
        assert orc.rng_u64(seed, stream, a, b) == int(wl.rng_u64(seed, stream, a, b))


# --------------------------------------------------------------------------
# pivots (Fig. 1)

def test_pivots_fig1_worked_example(orc):
    g = _golden("fig1_pivots.json")
    for row, piv in zip(g["rows"], g["pivots"]):
        got = orc.pivots(np.array(row), g["n"], g["width"])
        assert got.tolist() == piv


def test_pivots_slice_containment(orc):
    rs = np.random.default_rng(2)
    for n, w in [(1000, 64), (777, 100), (64, 64), (5, 1024)]:
        row = np.sort(rs.integers(0, n, size=rs.integers(0, 300)))
        piv = orc.pivots(row, n, w)
        s = (n + w - 1) // w
        assert piv[0] == 0 and piv[s] == len(row)
        assert np.all(np.diff(piv) >= 0)
        for q in range(s):
            seg = row[piv[q]:piv[q + 1]]
            assert np.all(seg >= q * w) and np.all(seg < (q + 1) * w)


# --------------------------------------------------------------------------
# neuron update

def _single(model=LIF_DELTA, **kw):
    base = dict(n=1, n_exc=1, model=model, graph_kind=GRAPH_BERNOULLI, p_or_fanout=0.0,
                w_exc=0.0, w_inh=0.0, delay=1)
    base.update(kw)
    return wl.Preset(name="single", **base)


def _empty_graph(o):
    z = np.zeros(0, np.int32)
    o.build_edges(z, z, np.zeros(0, np.float32))


def test_lif_euler_closed_form_and_period(orc):
    p = _single()
    o = orc.Oracle(p)
    _empty_graph(o)
    o.set_neurons(v=np.array([-60.0], np.float32))
    k = 0.1 / 20.0
    spikes, vs = [], []
    for t in range(1100):
        o.step()
        if o.spikes()[1].size:
            spikes.append(t)
        vs.append(float(o.neurons()["v"][0]))
    # V_n = V_inf - (V_inf - V_0)(1 - k)^n for n integration steps
    for n in (1, 10, 100, 300, 478):
        want = -49.0 - 11.0 * (1.0 - k) ** n
        assert abs(vs[n - 1] - want) < 2e-4, (n, vs[n - 1], want)
    assert abs(vs[99] - (-55.66347)) < 1e-4
    # first crossing after ceil(ln 11 / -ln 0.995) = 479 updates; 50 refractory
    # steps give an isolated period of 529 steps
    assert spikes == [478, 1007]
    assert vs[478] == -60.0 and vs[528] == -60.0 and vs[529] > -60.0


def test_lif_cuba_pulse_closed_form(orc):
    p = _single(model=LIF_CUBA, n=2, n_exc=1, v_inf=-70.0, v_th=0.0, v0_lo=-70, v0_hi=-70)
    o = orc.Oracle(p)
    _empty_graph(o)
    o.set_neurons(v=np.array([-70.0, -70.0], np.float32))
    q_e, q_i = 5.0, -3.0
    o.set_input(np.array([q_e, 0.0], np.float32), np.array([q_i, 2.0], np.float32))
    k = 0.1 / 20.0
    d_e, d_i = math.exp(-0.1 / 5.0), math.exp(-0.1 / 10.0)

    def g(d, n):
        return ((1 - k) ** (n + 1) - d ** (n + 1)) / ((1 - k) - d)

    for n in range(400):
        o.step()
        if n in (0, 1, 5, 50, 399):
            st = o.neurons()
            u0 = k * (q_e * g(d_e, n) + q_i * g(d_i, n))
            u1 = k * (2.0 * g(d_i, n))
            assert abs(st["v"][0] + 70.0 - u0) <= 1e-5 * abs(u0) + 2e-5
            assert abs(st["v"][1] + 70.0 - u1) <= 1e-5 * abs(u1) + 2e-5
            assert abs(st["i_exc"][0] - q_e * d_e ** n) <= 1e-5 * q_e
            assert abs(st["i_inh"][0] - q_i * d_i ** n) <= 1e-5 * abs(q_i)
        o.set_input(np.zeros(2, np.float32), np.zeros(2, np.float32))


def test_lif_refractory_drops_input(orc):
    p = _single(n=1)
    o = orc.Oracle(p)
    _empty_graph(o)
    o.set_neurons(v=np.array([-60.0], np.float32), refractory=np.array([3], np.int32))
    for _ in range(3):
        o.set_input(np.array([100.0], np.float32))
        o.step()
        st = o.neurons()
        assert st["v"][0] == -60.0 and o.spikes()[1].size == 0
    assert st["refractory"][0] == 0
    o.set_input(np.array([100.0], np.float32))
    o.step()
    assert o.spikes()[1].tolist() == [0] and o.neurons()["refractory"][0] == 50


def test_bernoulli_source_spikes_match_rng(orc):
    p = wl.preset("stress", n=3000, p_or_fanout=4, plastic=PLASTIC_NONE)
    o = orc.Oracle(p)
    o.build_random()
    thr = np.uint32(math.floor(p.p_fire * 2 ** 32))
    total = 0
    for t in range(200):
        o.step()
        mask, lst = o.spikes()
        want = np.nonzero(wl.rng_u32(p.seed, wl.STREAM_SPIKE, t,
                                     np.arange(p.n, dtype=np.uint64)) < thr)[0]
        assert lst.tolist() == want.tolist()
        total += len(lst)
    rate = total / (200 * p.n)
    assert abs(rate - p.p_fire) < 5 * math.sqrt(p.p_fire / (200 * p.n))


def test_mask_list_history_invariants(orc):
    p = wl.preset("tiny")
    o = orc.Oracle(p)
    o.build_random()
    o.set_neurons(**wl.initial_state(p))
    prev = np.zeros(p.n, np.uint64)
    seen = 0
    for _ in range(1200):
        o.step()
        mask, lst = o.spikes()
        hist = o.neurons()["hist"]
        bits = np.unpackbits(mask.view(np.uint8), bitorder="little")
        assert bits[p.n:].sum() == 0
        assert np.nonzero(bits[:p.n])[0].tolist() == lst.tolist()
        assert np.array_equal((hist & np.uint64(1)).astype(np.uint8), bits[:p.n])
        assert np.array_equal(hist >> np.uint64(1), prev & np.uint64((1 << 63) - 1))
        prev = hist
        seen += len(lst)
    assert seen > 0


def test_128_step_history_equals_spike_lists(orc):
    """The history word and the older word together hold exactly the spikes
    of the last 128 steps (bit b of the pair = step t-b), rebuilt here from
    the recorded spike lists."""
    p = wl.preset("stress", n=700, p_or_fanout=20, p_fire=0.05, plastic=0)
    o = orc.Oracle(p)
    o.build_random()
    lists = []
    for _ in range(300):
        o.step()
        lists.append(o.spikes()[1].copy())
    st = o.neurons()
    for b in range(128):
        fired = np.zeros(p.n, bool)
        fired[lists[-1 - b]] = True
        word = st["hist"] if b < 64 else st["hist_old"]
        bit = (word >> np.uint64(b % 64)) & np.uint64(1)
        assert np.array_equal(bit.astype(bool), fired), b


def test_poisson_drive_table_and_samples(orc):
    from scipy.stats import poisson
    mu = 2.0
    tab = wl.poisson_cdf_table(mu)
    ks = np.arange(len(tab))
    ref = np.floor(poisson.cdf(ks, mu) * 2.0 ** 32)
    assert np.all(np.abs(tab.astype(np.float64) - np.minimum(ref, 2 ** 32 - 1)) <= 1)
    assert tab[-1] == 2 ** 32 - 1
    # A neuron with no leak and an unreachable threshold integrates J_ext * k.
    p = wl.Preset(name="drive", n=256, n_exc=256, model=LIF_DELTA,
                  graph_kind=GRAPH_BERNOULLI, p_or_fanout=0.0, w_exc=0, w_inh=0,
                  tau_m=1e15, v_inf=0.0, v_th=1e30, v0_lo=0, v0_hi=0,
                  poisson_mu=mu, j_ext=1.0)
    o = orc.Oracle(p, tab)
    _empty_graph(o)
    o.set_neurons(v=np.zeros(p.n, np.float32))
    T = 400
    o.step(T)
    want = np.zeros(p.n, np.int64)
    for t in range(T):
        u = wl.rng_u32(p.seed, wl.STREAM_POISSON, t, np.arange(p.n, dtype=np.uint64))
        want += np.searchsorted(tab, u, side="right")
    v = o.neurons()["v"]
    assert np.array_equal(v.astype(np.int64), want)
    m = want.sum() / (p.n * T)
    assert abs(m - mu) < 5 * math.sqrt(mu / (p.n * T))
    var = (want / T).var() * T  # per-step variance estimate across neurons
    assert abs(var - mu) < 0.25 * mu


# --------------------------------------------------------------------------
# graph generators

def test_bernoulli_graph_matches_definition(orc):
    p = wl.preset("tiny", n=300, n_exc=240, p_or_fanout=0.1)
    o = orc.Oracle(p)
    e = o.build_random()
    rp, col, w = o.graph()
    thr = np.uint32(math.floor(0.1 * 2 ** 32))
    for k in range(p.n):
        u = wl.rng_u32(p.seed, wl.STREAM_GRAPH_PAIR, k, np.arange(p.n, dtype=np.uint64))
        js = np.nonzero(u < thr)[0]
        js = js[js != k]
        assert col[rp[k]:rp[k + 1]].tolist() == js.tolist()
        assert orc.bernoulli_row(p.seed, p.n, 0.1, k).tolist() == js.tolist()
        assert np.all(w[rp[k]:rp[k + 1]] == np.float32(p.w_exc if k < p.n_exc else p.w_inh))
    mean = p.n * (p.n - 1) * 0.1
    assert abs(e - mean) < 5 * math.sqrt(mean * 0.9)


def test_fanout_graph_matches_definition(orc):
    p = wl.preset("stress", n=5000, p_or_fanout=100, plastic=PLASTIC_NONE)
    o = orc.Oracle(p)
    assert o.build_random() == 5000 * 100
    rp, col, _ = o.graph()
    for k in (0, 1, 2500, 4999):
        u = wl.rng_u32(p.seed, wl.STREAM_FANOUT, k, np.arange(100, dtype=np.uint64))
        want = np.sort((u.astype(np.uint64) * np.uint64(p.n)) >> np.uint64(32))
        assert col[rp[k]:rp[k + 1]].tolist() == want.tolist()
    # targets uniform over [0, n): chi-square over 10 bins
    h = np.bincount(col * 10 // p.n, minlength=10)
    chi2 = ((h - len(col) / 10) ** 2 / (len(col) / 10)).sum()
    assert chi2 < 40


# --------------------------------------------------------------------------
# delivery (Fig. 3(a))

def _forced_net(orc, model, n, n_exc, src, dst, w, delay=1, plastic=PLASTIC_NONE, **kw):
    p = wl.Preset(name="forced", n=n, n_exc=n_exc, model=model,
                  graph_kind=GRAPH_BERNOULLI, p_or_fanout=0.0, w_exc=0, w_inh=0,
                  delay=delay, v_inf=-65.0, v_th=-50.0, plastic=plastic, **kw)
    o = orc.Oracle(p)
    o.build_edges(np.asarray(src), np.asarray(dst), np.asarray(w, np.float32))
    return o, p


def _force(o, n, firing):
    v = np.full(n, -1000.0, np.float32)
    v[list(firing)] = 1000.0
    o.set_neurons(v=v, refractory=np.zeros(n, np.int32))
    o.set_input(np.zeros(n, np.float32), np.zeros(n, np.float32))


def _fig1_edges():
    g = _golden("fig1_pivots.json")
    src, dst, w = [], [], []
    for k, (row, wk) in enumerate(zip(g["rows"], [1.0, 0.5, -0.25])):
        src += [k] * len(row)
        dst += row
        w += [wk] * len(row)
    return src, dst, w


def test_delivery_hand_computed(orc):
    src, dst, w = _fig1_edges()
    o, p = _forced_net(orc, LIF_DELTA, 9, 9, src, dst, w)
    _force(o, 9, [0, 2])
    o.step()
    a, b = o.input()
    # rows 0 (w=1) and 2 (w=-0.25) fire; row 1 does not
    assert a.tolist() == [1.0, 0.75, 1.0, -0.25, 0.75, -0.25, 0.75, 1.0, 0.0]
    assert not b.any()
    # CUBA splits the sum by source type (sources 0, 1 excitatory, 2 inhibitory)
    o, p = _forced_net(orc, LIF_CUBA, 9, 2, src, dst, w)
    _force(o, 9, [0, 1, 2])
    o.step()
    a, b = o.input()
    assert a.tolist() == [1.5, 1.5, 1.0, 0.0, 1.5, 0.5, 1.0, 1.5, 0.5]
    assert b.tolist() == [0.0, -0.25, 0.0, -0.25, -0.25, -0.25, -0.25, 0.0, 0.0]


def test_delivery_respects_delay(orc):
    src, dst, w = _fig1_edges()
    o, p = _forced_net(orc, LIF_DELTA, 9, 9, src, dst, w, delay=4)
    _force(o, 9, [1])
    o.step()                      # step 0: neuron 1 emits
    for t in (1, 2, 3):
        assert not o.input()[0].any(), t
        _force(o, 9, [])
        o.step()
    # emitted at step 0, transmitted at step 3 (delay-1 = 3), input for step 4
    a, _ = o.input()
    assert a.tolist() == [0.5, 0.5, 0.0, 0.0, 0.5, 0.5, 0.0, 0.5, 0.5]


def test_delivery_conservation(orc):
    p = wl.preset("tiny")
    o = orc.Oracle(p)
    o.build_random()
    o.set_neurons(**wl.initial_state(p))
    rp, col, w = o.graph()
    checked = 0
    for _ in range(1500):
        o.step()
        _, lst = o.spikes()
        a, _ = o.input()
        want = sum(w[rp[k]:rp[k + 1]].sum() for k in lst)
        mag = sum(np.abs(w[rp[k]:rp[k + 1]]).sum() for k in lst)
        assert abs(a.astype(np.float64).sum() - want) <= 1e-6 * mag + 1e-12
        checked += len(lst)
    assert checked > 100


# --------------------------------------------------------------------------
# plasticity (Fig. 2(a)) against brute force over explicit spike lists

def _stdp_consts(p):
    return dict(dp=math.exp(-p.dt / p.tau_plus), dm=math.exp(-p.dt / p.tau_minus),
                cpot=p.lam * p.w0 ** (1 - p.mu), cdep=p.lam * p.alpha, mu=p.mu)


def brute_force_weight(w, pres, posts, c):
    """All-to-all pairing: each pre event sees every earlier post, each post
    event sees every pre at or before it; events in time order, a pre before
    a post of the same step. Sums of exponentials, no traces."""
    ev = sorted([(u, 0) for u in pres] + [(v, 1) for v in posts])
    for time, kind in ev:
        if kind == 0:
            xq = sum(c["dm"] ** (time - v) for v in posts if v < time)
            w = max(0.0, w - c["cdep"] * w * xq)
        else:
            xp = sum(c["dp"] ** (time - u) for u in pres if u <= time)
            w = w + c["cpot"] * w ** c["mu"] * xp
    return w


def test_stdp_single_pair_hand_values(orc):
    w0 = 0.1 * 0.11 ** (1 / 0.6)
    for sched, want in [({10: [0], 15: [1]}, +1.0728409e-3),
                        ({10: [1], 15: [0]}, -1.0728409e-3),
                        ({10: [0, 1]}, +1.1e-3)]:
        o, p = _forced_net(orc, LIF_DELTA, 2, 2, [0], [1], [0.1], plastic=PLASTIC_ALL,
                           w0=w0)
        for t in range(20):
            _force(o, 2, sched.get(t, []))
            o.step()
        dw = o.weights()[0] - np.float64(np.float32(0.1))
        assert abs(dw - want) < 2e-9, (sched, dw, want)


@pytest.mark.parametrize("delay,plastic", [(1, PLASTIC_ALL), (3, PLASTIC_ALL),
                                           (2, PLASTIC_EXC_EXC)])
def test_stdp_matches_brute_force(orc, delay, plastic):
    p = wl.preset("stress", n=48, n_exc=32, p_or_fanout=8, p_fire=0.05, delay=delay,
                  plastic=plastic)
    o = orc.Oracle(p)
    o.build_random()
    T = 300
    o.step(T)
    thr = np.uint32(math.floor(p.p_fire * 2 ** 32))
    sp = np.stack([wl.rng_u32(p.seed, wl.STREAM_SPIKE, t, np.arange(p.n, dtype=np.uint64))
                   < thr for t in range(T)])
    c = _stdp_consts(p)
    rp, col, w = o.graph()
    w_init = float(np.float32(0.1))
    changed = 0
    for k in range(p.n):
        pres = [u + delay - 1 for u in np.nonzero(sp[:, k])[0] if u + delay - 1 < T]
        for e in range(rp[k], rp[k + 1]):
            j = col[e]
            plastic_syn = plastic == PLASTIC_ALL or (k < p.n_exc and j < p.n_exc)
            if not plastic_syn:
                assert w[e] == w_init
                continue
            posts = list(np.nonzero(sp[:, j])[0])
            want = brute_force_weight(w_init, pres, posts, c)
            assert abs(w[e] - want) <= 1e-12 * abs(want) + 1e-15, (k, j, w[e], want)
            changed += w[e] != w_init
    assert changed > 50


def test_bernoulli_replays_match_dense_oracle(orc):
    p = wl.preset("stress", n=2000, p_or_fanout=50, p_fire=0.02)
    o = orc.Oracle(p)
    o.build_random()
    T = 90
    o.step(T)
    rp, col, w = o.graph()
    for k in (0, 7, 1999):
        for e in range(rp[k], rp[k] + 5):
            want = o.bernoulli_synapse(k, int(col[e]), float(np.float32(0.1)), T - 1)
            assert abs(w[e] - want) <= 1e-13
    a, _ = o.input()
    a2 = o.bernoulli_input(50, float(np.float32(0.1)), T - 1)
    assert np.array_equal(a, a2)
