"""Full-size stress network (250,000 Bernoulli sources, fan-out 1,000, 250M
plastic synapses) in the launch configuration the benchmark times.

The oracle cannot step a network this size in seconds, but every spike here
is a counter-based draw, so single outputs are computable one by one: the
spike mask from the generator, a row's targets and pivots from its draws, a
synapse's weight by replaying it naively from step 0, and each target's
delivered input from the transmitting rows' replayed weights."""

import numpy as np
import pytest

import workloads as wl
from paper_2107_04092_amd import snn

from gpu_common import gpu_net, oracle_net, to_np, hist_np, assert_close, log

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
