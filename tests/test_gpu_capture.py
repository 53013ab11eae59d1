"""A step captured into a HIP graph replays correctly.

Every launch of a step reads the step index and the input source from the
device clock in the workspace, and the neuron update advances it there, so
the launches recorded once run any later step. One captured step replayed
100 times, with the program's own eager work (state reads, which also turn
the pending partial sums into the fp32 input) and synchronisations between
the replays, must equal the eager steps after every replay and equal one
snn_step(100) bit for bit at the end (fixed-point delivery, ascending lists
and per-synapse STDP are all deterministic)."""

import numpy as np
import pytest

import workloads as wl
from workloads.presets import PLASTIC_EXC_EXC, PLASTIC_NONE
from paper_2107_04092_amd import snn

from gpu_common import gpu_net, to_np, log

pytestmark = pytest.mark.gpu
LDS, GLOBAL = snn.SNN_DELIVER_LDS_SLICE, snn.SNN_DELIVER_GLOBAL_ATOMIC

CASES = [
    # name, preset overrides, slice width, chunks, mode: one path of snn_step each
    ("stress", dict(n=3000, p_or_fanout=100, p_fire=0.03, delay=3), 512, 2, LDS),   # plastic blocks
    ("stress", dict(n=3000, p_or_fanout=100, p_fire=0.03, delay=3, blocks=-1), 512, 2, LDS),  # fused pass
    ("stress", dict(n=3000, p_or_fanout=100, p_fire=0.03), 512, 1, GLOBAL),         # global atomics
    ("vogels", dict(n=3000, n_exc=2400, plastic=PLASTIC_EXC_EXC, w0=0.05), 512, 2, LDS),
    ("brunel", dict(n=5000, n_exc=4000), 1024, 2, LDS),                              # delay blocks
    ("tiny", dict(), 256, 1, LDS),                                                   # one workgroup
]

KEYS = ("v", "refractory", "i_exc", "i_inh", "hist", "trace_post", "t_last", "trace_pre",
        "input_exc", "input_inh", "spike_mask", "ring_counts")


def _same_state(a, b, what):
    sa, sb = a.state(), b.state()
    assert sa["t"] == sb["t"], (what, "t", sa["t"], sb["t"])
    for k in KEYS:
        ga, gb = to_np(sa[k]), to_np(sb[k])
        assert np.array_equal(ga.view(np.uint8), gb.view(np.uint8)), (what, k)
    d = a.cfg.delay_steps
    ra = to_np(sa["ring_lists"]).reshape(d, -1)
    rb = to_np(sb["ring_lists"]).reshape(d, -1)
    for q, c in enumerate(to_np(sa["ring_counts"])):
        assert np.array_equal(ra[q, :c], rb[q, :c]), (what, "ring slot", q)


@pytest.mark.parametrize("case", CASES, ids=lambda c: "%s-d%d-m%d%s" % (
    c[0], c[1].get("delay", 1 if c[0] != "brunel" else 15), c[4],
    "-stepwise" if c[1].get("blocks") == -1 else ""))
def test_captured_step_replays_equal_eager_steps(case):
    import torch
    name, kw, width, chunks, mode = case
    kw = dict(kw)
    cfg = dict(plastic_blocks=kw.pop("blocks", 0))
    p = wl.preset(name, **kw)
    log("capture %s %s W=%d C=%d mode=%d %s" % (name, kw, width, chunks, mode, cfg))
    side = torch.cuda.Stream()
    a = gpu_net(p, width, chunks, stream=side, **cfg)  # captured step, replayed
    b = gpu_net(p, width, chunks, **cfg)               # eager, one step at a time
    c = gpu_net(p, width, chunks, **cfg)               # eager, one call of 100 steps
    for net in (a, b, c):
        net.step(3, mode)
    g = a.capture(1, mode)
    try:
        assert a.state()["t"] == 3  # the capture ran nothing
        c.step(100, mode)
        for k in range(100):
            a.replay(g)
            b.step(1, mode)
            _same_state(a, b, "replay %d" % k)
        _same_state(a, c, "after 100 replays")
        for net in (a, c):
            net.flush_plasticity()
            net.synchronize()
        assert np.array_equal(to_np(a.graph()["w"]), to_np(c.graph()["w"]))
        ta, tc = a.stats(), c.stats()
        for key in ("steps", "spikes", "delivered_events", "stdp_rows", "stdp_synapse_updates",
                    "stdp_weights_written", "device_errors"):
            assert ta[key] == tc[key], key
        assert ta["steps"] == 103 and ta["spikes"] > 0 and ta["device_errors"] == 0
    finally:
        snn.snn_graph_destroy(g)


def test_capture_refuses_the_null_stream_and_steps_in_progress():
    import torch
    p = wl.preset("stress", n=1000, p_or_fanout=20, p_fire=0.03)
    net = gpu_net(p, 256, 1)  # the default stream
    if net.stream.cuda_stream == 0:
        with pytest.raises(snn.SnnError) as e:
            net.capture(1)
        assert e.value.status == snn.SNN_EINVAL
    side = gpu_net(p, 256, 1, stream=torch.cuda.Stream())
    side.update_neurons()
    with pytest.raises(snn.SnnError) as e:
        side.capture(1)
    assert e.value.status == snn.SNN_ESTATE
    with pytest.raises(snn.SnnError) as e:
        side.update_neurons()  # step 0 is in progress
    assert e.value.status == snn.SNN_ESTATE
    side.update_plasticity()
    side.deliver_spikes()
    side.advance()
    g = side.capture(2)
    side.replay(g)
    side.replay(g)
    assert side.state()["t"] == 5
    snn.snn_graph_destroy(g)


@pytest.mark.parametrize("delay", [1, 4])
def test_device_lists_are_ascending(delay):
    """The neuron update writes its lists in ascending order (each workgroup's
    stretch starts at the counts of the earlier ones): spike lists of every
    ring slot and the forced-row list, read without any sorting, at a rate
    that gives thousands of spikes per step over many workgroups."""
    p = wl.preset("stress", n=200_000, p_or_fanout=20, p_fire=0.02, delay=delay)
    net = gpu_net(p, 2048, 2)
    t = 0
    for chunk in (1, 60, 70):
        net.step(chunk, LDS)
        t += chunk
        s = net.state()
        d = p.delay
        ring = to_np(s["ring_lists"]).reshape(d, -1)
        cnt = to_np(s["ring_counts"])
        for q in range(d):
            assert cnt[q] > 0 or t < d  # (slots of steps before 0 are empty)
            assert np.all(np.diff(ring[q, :cnt[q]]) > 0), ("ring slot", q)
        nf = int(to_np(s["stdp_row_count"])[0])
        rows = to_np(s["stdp_rows"])[:nf]
        assert nf > 0 and np.all(np.diff(rows) > 0)
        # the spike list of the last step is the fire mask's set bits
        mask = to_np(s["spike_mask"]).view(np.uint64)
        bits = np.unpackbits(mask.view(np.uint8), bitorder="little")[:p.n]
        n_spk = int(to_np(s["spike_count"])[0])
        assert np.array_equal(to_np(s["spike_list"])[:n_spk], np.nonzero(bits)[0])
    assert net.stats()["device_errors"] == 0
