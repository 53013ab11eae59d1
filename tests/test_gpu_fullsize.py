"""Full-size networks in the launch configurations the benchmark times: the
stress network (250,000 Bernoulli sources, fan-out 1,000, 250M plastic
synapses), the Brunel network (390M synapses) and Brunel with STDP (25,000
neurons, 62.5M synapses, 40M of them plastic).

The oracle cannot step a network this size in seconds, but every spike here
is a counter-based draw, so single outputs are computable one by one: the
spike mask from the generator, a row's targets and pivots from its draws, a
synapse's weight by replaying it naively from step 0, and each target's
delivered input from the transmitting rows' replayed weights."""

import numpy as np
import pytest

import workloads as wl
from paper_2107_04092_amd import snn

from gpu_common import (gpu_net, oracle_net, to_np, hist_np, assert_close, log, rate_hz,
                        teacher_forced_run, compare_all_plastic_weights, same_state)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("hbits", [64, 128])
def test_stress_full_size_sampled_parity(hbits):
    from oracle import oracle
    p = wl.preset("stress")
    log("full-size stress: build n=%d fanout=%d W=%d C=%d history=%d" % (
        p.n, p.p_or_fanout, p.slice_width, p.spike_chunks, hbits))
    net = gpu_net(p, history_bits=hbits)
    o = oracle_net(p, build=False)
    F = int(p.p_or_fanout)
    w_init = float(np.float32(p.w_exc))
    T = 150
    net.step(T, snn.SNN_DELIVER_LDS_SLICE)
    s = net.state()
    log("  stepped %d" % T)
    # spikes of the last step, bit-exact
    thr = np.uint32(np.floor(p.p_fire * 2 ** 32))
    fired = wl.rng_u32(p.seed, wl.STREAM_SPIKE, T - 1, np.arange(p.n, dtype=np.uint64)) < thr
    want_mask = np.packbits(np.concatenate([fired, np.zeros((-p.n) % 64, bool)]),
                            bitorder="little").view(np.uint64)
    assert np.array_equal(hist_np(s["spike_mask"]), want_mask)
    cnt = int(to_np(s["spike_count"])[0])
    assert np.array_equal(to_np(s["spike_list"])[:cnt], np.nonzero(fired)[0])
    # delivered input of every target after step T-1 (weights after its STDP)
    a_want = o.bernoulli_input(F, w_init, T - 1)
    assert_close(to_np(s["input_exc"]), a_want, "full-size delivered input")
    log("  input checked")
    # graph rows and pivots of sampled rows
    g = net.graph()
    rp = to_np(g["row_ptr"])
    assert rp[-1] == p.n * F
    rs = np.random.default_rng(11)
    rows = np.concatenate([[0, p.n - 1], rs.integers(0, p.n, 60)])
    col = g["col"]
    piv = g["pivots"]
    for k in rows:
        row = to_np(col[rp[k]:rp[k + 1]])
        assert np.array_equal(row, oracle.fanout_row(p.seed, p.n, F, int(k))), k
        assert np.array_equal(to_np(piv[k]), oracle.pivots(row, p.n, p.slice_width)), k
    # weights of sampled rows after a flush, against per-synapse replays
    net.flush_plasticity()
    w = g["w"]
    for k in rows[:24]:
        row = to_np(col[rp[k]:rp[k + 1]])
        gw = to_np(w[rp[k]:rp[k + 1]])
        ow = np.array([o.bernoulli_synapse(int(k), int(j), w_init, T - 1) for j in row])
        assert_close(gw, ow, "row %d weights" % k)
    log("  weights checked")
    st = net.stats()
    assert st["delivered_events"] == st["spikes"] * F
    # one more step with the global-atomic variant: same input
    net.step(1, snn.SNN_DELIVER_GLOBAL_ATOMIC)
    a_want = o.bernoulli_input(F, w_init, T)
    assert_close(to_np(net.state()["input_exc"]), a_want, "full-size global-atomic input")


def test_stress_full_size_source_blocks_equal_stepwise():
    """The full-size stress network in the benchmark's launch configuration
    (source blocks of 16 steps: one neuron launch, then a fused synapse pass
    per step) against the same network stepped one neuron launch and one
    pass at a time, over 300 steps in uneven calls: every state array, every
    list and all 250M weights bit for bit."""
    p = wl.preset("stress")
    log("full-size stress: source blocks vs stepwise")
    a = gpu_net(p)
    b = gpu_net(p, plastic_blocks=-1)
    assert a.graph()["block_steps"] == 16 and b.graph()["block_steps"] == 0
    done = 0
    for n_steps in (150, 1, 149):
        a.step(n_steps, snn.SNN_DELIVER_LDS_SLICE)
        b.step(n_steps, snn.SNN_DELIVER_LDS_SLICE)
        done += n_steps
        same_state(a, b, "after %d steps" % done)
        log("  %d steps equal" % done)


def test_brunel_full_size_delay_block():
    """Full-size Brunel network (62,500 LIF neurons with Poisson drive,
    p = 0.1: 390M synapses, D = 15) in the launch configuration the benchmark
    times: delay blocks of 14 steps. Teacher forcing over one block: from the
    state after 100 steps, the oracle (no graph) runs the block's 14 neuron
    updates, each fed the input the delivered spikes imply; those inputs are
    summed from the oracle's own rows of every spiking source. Spikes of
    every step of the block, potentials, refractory counts and histories
    must be bit-exact (the weights 0.1 and -0.5 sum exactly), and the pending
    input after the block within the delivery tolerance."""
    from oracle import oracle
    p = wl.preset("brunel")
    D, n = p.delay, p.n
    log("full-size brunel: n=%d p=%g D=%d W=%d C=%d" % (n, p.p_or_fanout, D, p.slice_width,
                                                       p.spike_chunks))
    net = gpu_net(p)
    T0, B = 100, D - 1
    net.step(T0, snn.SNN_DELIVER_LDS_SLICE)
    s0 = net.state()  # views of the device state: copied before the next steps
    ring0 = to_np(s0["ring_lists"]).reshape(D, -1).copy()
    cnt0 = to_np(s0["ring_counts"]).copy()
    v0, ref0, hist0 = to_np(s0["v"]).copy(), to_np(s0["refractory"]).copy(), hist_np(s0["hist"]).copy()
    a0 = to_np(s0["input_exc"]).copy()
    ev0 = net.stats()["delivered_events"]
    net.step(B, snn.SNN_DELIVER_LDS_SLICE)
    s1 = net.state()
    ring1 = to_np(s1["ring_lists"]).reshape(D, -1)
    cnt1 = to_np(s1["ring_counts"])
    log("  stepped %d + %d" % (T0, B))
    rows = {}

    def row(k):
        if k not in rows:
            rows[k] = oracle.bernoulli_row(p.seed, n, p.p_or_fanout, int(k))
        return rows[k]

    def input_from(spk):
        # the input a list of spiking sources delivers, in double from the
        # oracle's rows, rounded once to fp32
        acc = np.zeros(n, np.float64)
        for k in spk:
            acc[row(k)] += np.float64(np.float32(p.w_exc if k < p.n_exc else p.w_inh))
        return acc.astype(np.float32)

    o = oracle_net(p, build=False)
    o.t = T0
    o.set_neurons(v=v0, refractory=ref0, hist=hist0)
    events = 0
    for b in range(B):
        t = T0 + b
        if b == 0:
            a = a0  # pending input at T0: the state
        else:
            e = t - D  # emission step of the spikes arriving at t
            a = input_from(ring0[e % D, :cnt0[e % D]])
        o.set_input(a_exc=a)
        o.step(1)
        mask, lst = o.spikes()
        slot = t % D
        assert np.array_equal(ring1[slot, :cnt1[slot]], lst), ("spikes of step", t)
    # the block delivered the spikes emitted at T0+1-D .. T0+B-D
    for e in range(T0 + 1 - D, T0 + B + 1 - D):
        events += sum(len(row(k)) for k in ring0[e % D, :cnt0[e % D]])
    ost = o.neurons()
    assert np.array_equal(to_np(s1["v"]).view(np.uint32), ost["v"].view(np.uint32))
    assert np.array_equal(to_np(s1["refractory"]), ost["refractory"])
    assert np.array_equal(hist_np(s1["hist"]), ost["hist"])
    e = T0 + B - D  # pending input of step T0+B
    assert_close(to_np(s1["input_exc"]), input_from(ring0[e % D, :cnt0[e % D]]),
                 "pending input after the block")
    assert net.stats()["delivered_events"] - ev0 == events
    # the GPU's rows of some of the spiking sources
    g = net.graph()
    rp = to_np(g["row_ptr"])
    for k in list(rows)[:16]:
        assert np.array_equal(to_np(g["col"][rp[k]:rp[k + 1]]), row(k)), k
    log("  block checked: %d spiking rows, %d events" % (len(rows), events))


@pytest.mark.parametrize("blocks", [0, -1], ids=["blocks", "stepwise"])
def test_brunel_plus_full_size_teacher_forced(blocks):
    """Brunel with STDP at its stated size (25,000 LIF neurons with Poisson
    drive, p = 0.1: 62.5M synapses, STDP on the 40M exc->exc ones, D = 15)
    in the benchmark's launch configuration (W = 1024, four chunks, 16-bit
    slice-local targets), each step a block of one step (plan and target
    groups) or the three parts with the fused synapse pass. 150
    teacher-forced steps: every step spikes, histories, potentials and
    refractory counts are bit-exact, the delivered input is within
    tolerance, and so are the weights of every row made current (forced
    rows from step 63 on, transmitting rows from step 14 on); after a flush,
    every plastic weight."""
    p = wl.preset("brunel_plus")
    log("full-size brunel_plus: n=%d p=%g D=%d W=%d C=%d blocks=%d" % (
        p.n, p.p_or_fanout, p.delay, p.slice_width, p.spike_chunks, blocks))
    net, o, cnt = teacher_forced_run(p, 150, snn.SNN_DELIVER_LDS_SLICE, progress=25,
                                     plastic_blocks=blocks)
    log("  %d rows, %d weights, %d spikes checked" % (cnt["rows"], cnt["weights"], cnt["spikes"]))
    assert cnt["spikes"] > 0 and cnt["rows"] > 0 and cnt["weights"] > 0
    st = net.stats()
    assert st["stdp_forced_rows"] > 0
    assert st["device_errors"] == 0
    net.flush_plasticity()
    n_w = compare_all_plastic_weights(net, o)
    log("  all %d plastic weights equal after the flush" % n_w)
    assert n_w > 39_000_000


def test_brunel_plus_full_size_free_running_rate():
    """Brunel with STDP at its stated size runs free for 1 s of network time
    (10,000 steps) on both sides: the mean firing rates agree within 2%. The
    two runs share every external Poisson draw but drift apart spike by spike
    as the weights' roundings differ, so only the rate is compared."""
    p = wl.preset("brunel_plus")
    steps = 10_000
    log("full-size brunel_plus free run: %d steps" % steps)
    net = gpu_net(p)
    o = oracle_net(p)
    for done in range(0, steps, 1000):
        net.step(1000, snn.SNN_DELIVER_LDS_SLICE)
        o.step(1000)
        log("  %d/%d steps: gpu %d spikes, oracle %d" % (
            done + 1000, steps, net.stats()["spikes"], o.spikes_total))
    g, r = net.stats()["spikes"], o.spikes_total
    rg, ro = rate_hz(g, p.n, steps), rate_hz(r, p.n, steps)
    log("  gpu %.3f Hz, oracle %.3f Hz" % (rg, ro))
    assert net.stats()["device_errors"] == 0
    assert r >= 100_000
    assert abs(rg - ro) <= 0.02 * ro


def test_brunel_plus_full_size_blocks_equal_stepwise():
    """The benchmark's Brunel+ network (62.5M synapses) run 300 steps in
    blocks of 14 and step by step: every state array, delay-ring list,
    weight and statistic bit for bit."""
    from test_gpu_blocks import same_state
    p = wl.preset("brunel_plus")
    a = gpu_net(p)
    assert a.graph()["block_steps"] == 14
    a.step(300, snn.SNN_DELIVER_LDS_SLICE)
    a.synchronize()
    b = gpu_net(p, plastic_blocks=-1)
    b.step(300, snn.SNN_DELIVER_LDS_SLICE)
    log("  300 steps each: %d spikes, %d forced rows" % (a.stats()["spikes"],
                                                        a.stats()["stdp_forced_rows"]))
    same_state(a, b, "full-size brunel_plus")
    assert a.stats()["stdp_forced_rows"] > 0
