"""Teacher-forced parity of the HIP step against the CPU oracle.

Each step the GPU receives the oracle's neuron state and pending input; the
synaptic state (weights, row ages and traces, post traces, delay ring) evolves
on the GPU from identical spikes. Spike masks, spike lists, histories,
potentials and refractory counters must match bit for bit; delivered inputs
and the weights of the rows STDP just made current must match within
|g - o| <= 1e-5 |o| + 1e-7; after a final flush every plastic weight must.
"""

import numpy as np
import pytest

import workloads as wl
from workloads.presets import PLASTIC_ALL, PLASTIC_EXC_EXC, PLASTIC_NONE, BERNOULLI_SOURCE, \
    LIF_DELTA, GRAPH_BERNOULLI
from paper_2107_04092_amd import snn

from gpu_common import (teacher_forced_run, compare_all_plastic_weights, gpu_net, oracle_net,
                        compare_step, compare_rows, force_from_oracle, to_np, log, assert_close)

pytestmark = pytest.mark.gpu
LDS, GLOBAL = snn.SNN_DELIVER_LDS_SLICE, snn.SNN_DELIVER_GLOBAL_ATOMIC

CASES = [
    # name, preset overrides, steps, slice width, chunks
    ("tiny", dict(), 300, 256, 1),
    ("tiny", dict(n=1037, n_exc=830), 300, 320, 3),
    ("vogels", dict(), 300, 1024, 2),
    # CUBA with STDP on exc->exc: the packed segment word carries the
    # plastic length, the row age and the inhibitory half together
    ("vogels", dict(n=3000, n_exc=2400, plastic=PLASTIC_EXC_EXC, w0=0.05), 200, 512, 2),
    ("brunel", dict(n=5000, n_exc=4000), 200, 1024, 1),
    ("brunel_plus", dict(n=2500, n_exc=2000), 300, 512, 2),
    ("stress", dict(n=6000, p_or_fanout=200, p_fire=0.02), 200, 1024, 4),
    ("stress", dict(n=3000, p_or_fanout=150, p_fire=0.03, delay=3), 160, 640, 1),
]


MODES = [((LDS, 0, 1), "lds-rowstdp-codes"), ((LDS, 0, 2), "lds-rowstdp-bitmap"),
         ((LDS, 1, 0), "lds-slicestdp"), ((GLOBAL, 0, 3), "global-rowstdp-gather")]


def _parity_params():
    """Every case in every mode; plastic networks with D >= 2 in the slice
    mode run snn_step's steps as blocks (of one step here), and so do
    plastic networks of Bernoulli sources with D = 1 whose step fuses the
    synapse pass (row-wise layout), so they run once more with the blocks
    switched off (parts one by one)."""
    out = []
    for case in CASES:
        p = wl.preset(case[0], **case[1])
        for (mode, layout, filt), mname in MODES:
            both = p.plastic != PLASTIC_NONE and mode == LDS and (
                p.delay >= 2 or (p.model == BERNOULLI_SOURCE and layout == 0))
            for blocks in ([0, -1] if both else [0]):
                cid = "%s-%s-%s%s" % (case[0], case[1].get("n", ""), mname,
                                      "-stepwise" if blocks == -1 else "")
                out.append(pytest.param(case, mode, layout, filt, blocks, id=cid))
    return out


@pytest.mark.parametrize("hbits", [64, 128], ids=["h64", "h128"])
@pytest.mark.parametrize("case,mode,layout,filt,blocks", _parity_params())
def test_teacher_forced_parity(case, mode, layout, filt, hbits, blocks):
    name, kw, steps, width, chunks = case
    p = wl.preset(name, **kw)
    log("parity %s %s mode=%d layout=%d filter=%d history=%d W=%d C=%d steps=%d blocks=%d" % (
        name, kw, mode, layout, filt, hbits, width, chunks, steps, blocks))
    net, o, cnt = teacher_forced_run(p, steps, mode, slice_width=width, spike_chunks=chunks,
                                     stdp_layout=layout, stdp_filter=filt, history_bits=hbits,
                                     plastic_blocks=blocks)
    assert cnt["spikes"] > 0
    if p.plastic != PLASTIC_NONE:
        assert cnt["rows"] > 0 and cnt["weights"] > 0
        net.flush_plasticity()
        compare_all_plastic_weights(net, o)
        st = net.stats()
        assert st["stdp_forced_rows"] > 0  # rows idle for the whole history were forced
    st = net.stats()
    assert st["steps"] == steps
    assert st["spikes"] == cnt["spikes"]


@pytest.mark.parametrize("width,chunks,fanout,mult,schunks,hbits", [
    (64, 1, 300, 1, 1, 64), (2048, 2, 300, 0, 0, 64), (4096, 1, 3000, 1, 1, 64),
    (1024, 64, 300, 3, 7, 64), (640, 1, 300, 4, 300, 128), (1024, 3, 400, 0, 0, 128),
    (2048, 1, 300, 2, 5, 128)])
def test_slice_shapes(width, chunks, fanout, mult, schunks, hbits):
    """Delivery segments from 1 to ~600 entries, one to many chunks, more
    spikes (and rows) per workgroup than one staging batch holds; STDP target
    groups of 1..8 slices shared by 1..300 workgroups."""
    p = wl.preset("stress", n=4000, p_or_fanout=fanout, p_fire=0.3 if chunks == 1 else 0.02)
    log("slice shape W=%d C=%d F=%d mult=%d stdp_chunks=%d" % (width, chunks, fanout, mult,
                                                                 schunks))
    layout = 1 if mult else 0
    net, o, _ = teacher_forced_run(p, 70, LDS, slice_width=width, spike_chunks=chunks,
                                   stdp_slice_mult=mult, stdp_chunks=schunks, stdp_layout=layout,
                                   history_bits=hbits)
    net.flush_plasticity()
    compare_all_plastic_weights(net, o)


def test_three_part_calls_equal_step():
    """update_neurons / update_plasticity / deliver_spikes / advance == step."""
    p = wl.preset("stress", n=2000, p_or_fanout=100, p_fire=0.03)
    a = gpu_net(p, slice_width=512)
    b = gpu_net(p, slice_width=512)
    for t in range(100):
        a.step(1, LDS)
        b.update_neurons()
        b.update_plasticity()
        b.deliver_spikes(LDS)
        b.advance()
    a.flush_plasticity()
    b.flush_plasticity()
    sa, sb = a.state(), b.state()
    for key in ("hist", "input_exc", "t_last", "trace_pre", "trace_post"):
        assert np.array_equal(to_np(sa[key]), to_np(sb[key])), key
    assert np.array_equal(to_np(a.graph()["w"]), to_np(b.graph()["w"]))


SMALL_CASES = [
    ("tiny", dict()),
    ("tiny", dict(n=1037, n_exc=830, delay=3)),
    ("vogels", dict()),
    ("stress", dict(n=3000, p_or_fanout=50, p_fire=0.03, plastic=PLASTIC_NONE, delay=2)),
]


@pytest.mark.parametrize("case", SMALL_CASES, ids=lambda c: "%s-%s" % (c[0], c[1].get("n", "")))
def test_small_network_steps_equal_three_part_calls(case):
    """Small networks without plasticity run several steps per launch in one
    workgroup (the input carried in LDS between steps): states, delay ring and
    statistics equal those of the separate kernels, bit for bit."""
    name, kw = case
    p = wl.preset(name, **kw)
    a = gpu_net(p)
    b = gpu_net(p)
    for k in (1, 37, 63):  # several launches, the first of a single step
        a.step(k, LDS)
        for _ in range(k):
            b.update_neurons()
            b.update_plasticity()
            b.deliver_spikes(LDS)
            b.advance()
    sa, sb = a.state(), b.state()
    for key in ("v", "refractory", "i_exc", "i_inh", "hist", "input_exc", "input_inh",
                "spike_mask", "ring_counts"):
        if sa[key] is None:
            continue
        assert np.array_equal(to_np(sa[key]), to_np(sb[key])), key
    ra, rb = to_np(sa["ring_lists"]).reshape(p.delay, -1), to_np(sb["ring_lists"]).reshape(
        p.delay, -1)
    for q, c in enumerate(to_np(sa["ring_counts"])):  # entries past a count are stale
        assert np.array_equal(ra[q, :c], rb[q, :c]), ("ring slot", q)
    ta, tb = a.stats(), b.stats()
    for key in ("steps", "spikes", "delivered_events"):
        assert ta[key] == tb[key], key
    assert ta["spikes"] > 0


SMALL_FREE_CASES = [
    # name, preset overrides, history bits
    ("tiny", dict(), 64),
    ("tiny", dict(), 128),
    ("tiny", dict(delay=3), 64),
    ("vogels", dict(), 64),
    ("vogels", dict(), 128),
]


@pytest.mark.parametrize("case", SMALL_FREE_CASES,
                         ids=lambda c: "%s-d%d-h%d" % (c[0], c[1].get("delay", 1), c[2]))
def test_small_network_free_run_matches_oracle(case):
    """Small networks without plasticity run several steps per launch in one
    workgroup, carrying the input between steps in an LDS accumulator. Both
    presets' weights (+0.27/-4.5 and +1.62/-9 in fp32) sum exactly in the
    64-bit fixed point and in the oracle's double sums, so the two free runs
    stay bit-exact: after launches of 1, 37, 63 and 4096 steps the spikes of
    the last step, the histories, potentials, refractory counts (and CUBA
    currents) equal the oracle's, and the pending input is within the
    delivery tolerance."""
    name, kw, hbits = case
    p = wl.preset(name, **kw)
    log("small free run %s %s history=%d" % (name, kw, hbits))
    net = gpu_net(p, history_bits=hbits)
    o = oracle_net(p)
    t = 0
    for chunk in (1, 37, 63, 4096):
        net.step(chunk, LDS)
        o.step(chunk)
        t += chunk
        compare_step(net, o, "small free run", t, check_rows=False)
        log("  %d steps equal" % t)
    st = net.stats()
    assert st["spikes"] == o.spikes_total > 0
    assert st["device_errors"] == 0


DELAY_BLOCK_CASES = [
    # name, preset overrides, slice width, chunks
    ("brunel", dict(n=8000, n_exc=6400), 1024, 4),               # D = 15: blocks of 14
    ("brunel", dict(n=8000, n_exc=6400, delay=2), 512, 1),       # blocks of 1, one chunk
    ("brunel", dict(n=6000, n_exc=4800, delay=24), 1024, 3),     # blocks of 16 (the cap)
    ("vogels", dict(n=6000, n_exc=4800, delay=4), 1024, 2),      # CUBA: two accumulators
    ("vogels", dict(n=5000, n_exc=4000, delay=12), 512, 1),      # CUBA: blocks of 8 (its cap)
    ("stress", dict(n=9000, p_or_fanout=60, p_fire=0.02, plastic=PLASTIC_NONE, delay=5),
     2048, 4),
]


@pytest.mark.parametrize("hbits", [64, 128], ids=["h64", "h128"])
@pytest.mark.parametrize("case", DELAY_BLOCK_CASES,
                         ids=lambda c: "%s-%s-d%s" % (c[0], c[1].get("n", ""), c[1].get("delay", "")))
def test_delay_blocks_equal_three_part_calls(case, hbits):
    """Networks without plasticity and D >= 2 run in delay blocks (one
    delivery launch for up to D-1 steps' inputs, then one neuron launch for
    those steps): states, delay ring and statistics equal those of the
    separate kernels, bit for bit, across blocks cut short by the step count."""
    name, kw, width, chunks = case
    p = wl.preset(name, **kw)
    log("delay blocks %s %s W=%d C=%d history=%d" % (name, kw, width, chunks, hbits))
    a = gpu_net(p, slice_width=width, spike_chunks=chunks, history_bits=hbits)
    b = gpu_net(p, slice_width=width, spike_chunks=chunks, history_bits=hbits)
    for k in (1, 37, 63):
        a.step(k, LDS)
        for _ in range(k):
            b.update_neurons()
            b.update_plasticity()
            b.deliver_spikes(LDS)
            b.advance()
        sa, sb = a.state(), b.state()
        for key in ("v", "refractory", "i_exc", "i_inh", "hist", "input_exc", "input_inh",
                    "spike_mask", "ring_counts"):
            if sa[key] is None:
                continue
            assert np.array_equal(to_np(sa[key]), to_np(sb[key])), (key, k)
        ra = to_np(sa["ring_lists"]).reshape(p.delay, -1)
        rb = to_np(sb["ring_lists"]).reshape(p.delay, -1)
        for q, c in enumerate(to_np(sa["ring_counts"])):
            assert np.array_equal(ra[q, :c], rb[q, :c]), ("ring slot", q)
    ta, tb = a.stats(), b.stats()
    for key in ("steps", "spikes", "delivered_events", "device_errors"):
        assert ta[key] == tb[key], key
    assert ta["spikes"] > 0 and ta["delivered_events"] > 0
    assert ta["device_errors"] == 0


def test_delay_blocks_free_run_matches_oracle():
    """A Brunel network with 15-step delays runs free in delay blocks. Its
    weights (0.1 and -0.5 in fp32) sum exactly in both the fixed-point and the
    double accumulation, so the free run stays bit-exact: after every chunk,
    spikes, histories and potentials equal the oracle's, and the pending input
    is within the delivery tolerance."""
    p = wl.preset("brunel", n=5000, n_exc=4000)
    net = gpu_net(p, slice_width=1024, spike_chunks=2)
    o = oracle_net(p)
    t = 0
    for chunk in (14, 29, 3, 50):
        net.step(chunk, LDS)
        o.step(chunk)
        t += chunk
        compare_step(net, o, "delay blocks", t, check_rows=False)
    assert net.stats()["spikes"] > 0


def test_fused_pass_statistics_with_few_stdp_slots():
    """The fused synapse pass gives each of its forced-row workgroups (here
    496 of them) a statistics slot, also when the slice-STDP grid (one
    chunk) would size the slots for fewer: every spike delivers exactly its
    fan-out, and the weight counts match the separate kernels'."""
    p = wl.preset("stress", n=3000, p_or_fanout=100, p_fire=0.03)
    a = gpu_net(p, slice_width=512, spike_chunks=2, stdp_chunks=1)
    b = gpu_net(p, slice_width=512, spike_chunks=2, stdp_chunks=1)
    for t in range(70):
        a.step(1, LDS)
        b.update_neurons()
        b.update_plasticity()
        b.deliver_spikes(LDS)
        b.advance()
    sa, sb = a.stats(), b.stats()
    assert sa["delivered_events"] == sa["spikes"] * 100
    for key in ("spikes", "delivered_events", "stdp_forced_rows", "stdp_synapse_updates",
                "stdp_weights_written", "device_errors"):
        assert sa[key] == sb[key], key
    assert np.array_equal(to_np(a.graph()["w"]), to_np(b.graph()["w"]))


def test_out_of_order_calls_rejected():
    p = wl.preset("stress", n=500, p_or_fanout=10, p_fire=0.03)
    net = gpu_net(p, slice_width=128)
    with pytest.raises(snn.SnnError) as e:
        net.update_plasticity()
    assert e.value.status == snn.SNN_ESTATE
    with pytest.raises(snn.SnnError):
        net.deliver_spikes(7)


@pytest.mark.parametrize("hbits", [64, 128])
def test_silent_network(hbits):
    """No spikes at all: empty lists, zero input, rows only forced."""
    p = wl.preset("stress", n=1500, p_or_fanout=50, p_fire=0.0)
    net, o, cnt = teacher_forced_run(p, 300, LDS, slice_width=512, spike_chunks=2,
                                     history_bits=hbits)
    assert cnt["spikes"] == 0
    st = net.stats()
    assert st["delivered_events"] == 0
    # row k starts 1 + (k mod H) steps old: forced at H-1 - (k mod H) + H i
    H = hbits
    want = sum(len(range(H - 1 - (k % H), 300, H)) for k in range(1500))
    assert st["stdp_forced_rows"] == want
    assert st["stdp_weights_written"] == 0
    assert not to_np(net.state()["input_exc"]).any()


@pytest.mark.parametrize("mode", [LDS, GLOBAL], ids=["lds", "global"])
def test_all_spikes_hit_one_target(mode):
    """Maximum atomic contention: 3000 sources, all edges into neuron 5."""
    n = 3000
    src = np.arange(n)
    dst = np.full(n, 5)
    w = np.full(n, 0.25, np.float32)  # sums of quarters are exact in fp32
    p = wl.Preset(name="contention", n=n, n_exc=n, model=BERNOULLI_SOURCE,
                  graph_kind=GRAPH_BERNOULLI, p_or_fanout=0, w_exc=0, w_inh=0,
                  p_fire=0.5, slice_width=1024)
    net = gpu_net(p, build=False, slice_width=1024, spike_chunks=3)
    net.build_edges(src, dst, w)
    o = oracle_net(p, build=False)
    o.build_edges(src, dst, w)
    for t in range(20):
        o.step()
        net.step(1, mode)
        compare_step(net, o, "contention", t, check_rows=False)
        a = to_np(net.state()["input_exc"])
        assert a[5] == o.input()[0][5] and a[5] > 100


def test_weights_span_sign_and_cancel():
    """Brunel weights +0.1/-0.5 summed into one input: cancellation cases."""
    p = wl.preset("brunel", n=3000, n_exc=2400, delay=1)
    net, o, cnt = teacher_forced_run(p, 150, LDS, slice_width=64, spike_chunks=1)
    assert cnt["spikes"] > 100


def test_checkpoint_restore_resumes_identically():
    """get_state -> copy -> set_state into a fresh network continues identically
    (spikes are Bernoulli draws, so no teacher forcing is needed)."""
    import torch
    p = wl.preset("stress", n=2500, p_or_fanout=100, p_fire=0.03, delay=4)
    a = gpu_net(p, slice_width=512)
    a.step(90, LDS)
    s = a.state()
    snap = {k: v.clone() for k, v in s.items() if isinstance(v, torch.Tensor)}
    w_snap = a.graph()["w"].clone()
    a.step(50, LDS)
    b = gpu_net(p, slice_width=512)
    b.graph()["w"].copy_(w_snap)
    keys = ("v", "refractory", "i_exc", "i_inh", "hist", "trace_post", "t_last", "trace_pre",
            "input_exc", "ring_lists", "ring_counts")
    b.set_state(int(s["t"]), **{k: snap[k] for k in keys})
    b.step(50, LDS)
    sa, sb = a.state(), b.state()
    for k in ("hist", "t_last", "trace_pre", "trace_post"):
        assert np.array_equal(to_np(sa[k]), to_np(sb[k])), k
    assert_close(to_np(sb["input_exc"]), to_np(sa["input_exc"]), "input after restore")
    assert_close(to_np(b.graph()["w"]), to_np(a.graph()["w"]), "weights after restore")


def test_checkpoint_restore_between_delay_blocks():
    """A Brunel network (delay blocks of 14) saved after 20 steps and restored
    into a fresh network, with a forced input for its next step, continues
    exactly as the original does through the same calls: the ring, the
    pending input and the neuron state carry every block boundary."""
    import torch
    p = wl.preset("brunel", n=6000, n_exc=4800)
    a = gpu_net(p, slice_width=1024, spike_chunks=2)
    a.step(20, LDS)
    s = a.state()
    keys = ("v", "refractory", "hist", "input_exc", "ring_lists", "ring_counts")
    snap = {k: s[k].clone() for k in keys}
    t = int(s["t"])
    b = gpu_net(p, slice_width=1024, spike_chunks=2)
    b.set_state(t, **snap)
    # the same forced input on both: the next step reads it, later ones the blocks
    bump = snap["input_exc"] + 0.25
    for net in (a, b):
        net.set_state(t, input_exc=bump)
        net.step(47, LDS)
    sa, sb = a.state(), b.state()
    for k in ("v", "refractory", "hist", "input_exc", "spike_mask", "ring_counts"):
        assert np.array_equal(to_np(sa[k]), to_np(sb[k])), k
    ra = to_np(sa["ring_lists"]).reshape(p.delay, -1)
    rb = to_np(sb["ring_lists"]).reshape(p.delay, -1)
    for q, c in enumerate(to_np(sa["ring_counts"])):
        assert np.array_equal(ra[q, :c], rb[q, :c]), ("ring slot", q)
    assert a.stats()["spikes"] > 0 and a.stats()["device_errors"] == 0


@pytest.mark.parametrize("mode", [LDS, GLOBAL], ids=["lds", "global"])
@pytest.mark.parametrize("delay", [1, 3])
def test_free_run_with_state_reads(mode, delay):
    """Bernoulli sources run free on both sides. Reading the state mid-run
    puts the step's lists in ascending order (and re-records the delay-ring
    positions the transmitting rows' snapshots use); later steps must not
    notice. Spike lists come back ascending and equal the oracle's."""
    p = wl.preset("stress", n=3000, p_or_fanout=120, p_fire=0.03, delay=delay)
    net = gpu_net(p, slice_width=512, spike_chunks=2)
    o = oracle_net(p)
    for chunk in (37, 41, 12):
        net.step(chunk, mode)
        o.step(chunk)
        s = net.state()
        mask, lst = o.spikes()
        assert np.array_equal(to_np(s["spike_mask"]).view(np.uint64), mask)
        cnt = int(to_np(s["spike_count"])[0])
        assert np.array_equal(to_np(s["spike_list"])[:cnt], lst)
        ring = to_np(s["ring_lists"]).reshape(delay, -1)
        rc = to_np(s["ring_counts"])
        for q in range(delay):
            assert np.all(np.diff(ring[q, :rc[q]]) > 0), "ring slot %d not ascending" % q
    net.flush_plasticity()
    compare_all_plastic_weights(net, o)
    assert net.stats()["device_errors"] == 0


CT_CASES = [
    # name, preset overrides, steps, slice width, chunks
    ("stress", dict(n=6000, p_or_fanout=200, p_fire=0.02), 200, 1024, 4),
    ("stress", dict(n=3000, p_or_fanout=150, p_fire=0.03, delay=3), 160, 640, 1),
    ("brunel_plus", dict(n=2500, n_exc=2000), 300, 512, 2),
    ("vogels", dict(), 200, 1024, 2),
    # sparse rows over 18 slices of 4096
    ("stress", dict(n=70_000, p_or_fanout=3, p_fire=0.05), 150, 4096, 1),
]


@pytest.mark.parametrize("hbits", [64, 128], ids=["h64", "h128"])
@pytest.mark.parametrize("mode", [LDS, GLOBAL], ids=["lds", "global"])
@pytest.mark.parametrize("case", CT_CASES, ids=lambda c: "%s-%s" % (c[0], c[1].get("n", "")))
def test_compressed_targets_parity(case, mode, hbits):
    """16-bit slice-local targets (read by slice delivery): the same parity
    bar as the 32-bit targets."""
    name, kw, steps, width, chunks = case
    p = wl.preset(name, **kw)
    log("compressed-target parity %s %s mode=%d history=%d W=%d C=%d" % (
        name, kw, mode, hbits, width, chunks))
    net, o, cnt = teacher_forced_run(p, steps, mode, slice_width=width, spike_chunks=chunks,
                                     history_bits=hbits, compressed_targets=1)
    assert cnt["spikes"] > 0
    if p.plastic != PLASTIC_NONE:
        assert cnt["rows"] > 0
        net.flush_plasticity()
        compare_all_plastic_weights(net, o)
    assert net.stats()["device_errors"] == 0


ALGO_CASES = [
    ("brunel_plus", dict(n=2500, n_exc=2000), 260, 512, 2),
    ("stress", dict(n=6000, p_or_fanout=200, p_fire=0.02), 200, 1024, 4),
    ("stress", dict(n=3000, p_or_fanout=150, p_fire=0.03, delay=3), 160, 640, 1),
]


@pytest.mark.parametrize("algo,hbits", [(1, 64), (1, 128), (2, 64)],
                         ids=["lazy-h64", "lazy-h128", "naive"])
@pytest.mark.parametrize("mode", [LDS, GLOBAL], ids=["lds", "global"])
@pytest.mark.parametrize("case", ALGO_CASES, ids=lambda c: "%s-%s" % (c[0], c[1].get("n", "")))
def test_plasticity_algorithms(case, mode, algo, hbits):
    """Lazy without event-driven replay (every step of the window) and the
    naive per-synapse, per-step form (Fig. 2(a,b)) reach the oracle's weights
    too; naive keeps every weight current, so all are compared as it runs."""
    name, kw, steps, width, chunks = case
    p = wl.preset(name, **kw)
    log("algorithm %d history %d %s %s mode=%d" % (algo, hbits, name, kw, mode))
    net = gpu_net(p, width, chunks, plasticity_algorithm=algo, history_bits=hbits)
    o = oracle_net(p)
    cache = {}
    n_w = 0
    for t in range(steps):
        force_from_oracle(net, o, t)
        o.step()
        net.step(1, mode)
        rows = compare_step(net, o, "algo %d" % algo, t)
        n_w += compare_rows(net, o, rows, "STDP rows at t=%d" % t, cache)
        if algo == 2 and t % 40 == 39:
            compare_all_plastic_weights(net, o)
    assert n_w > 0
    st = net.stats()
    if algo == 2:
        assert st["stdp_forced_rows"] == 0
        assert st["stdp_synapse_updates"] > 0
    net.flush_plasticity()
    compare_all_plastic_weights(net, o)


XCD_CASES = [
    # name, preset overrides, steps, slice width, chunks, target ranges: the
    # plastic targets span at least as many slices as ranges
    ("stress", dict(n=6000, p_or_fanout=200, p_fire=0.02), 200, 256, 2, 8),
    ("stress", dict(n=3000, p_or_fanout=150, p_fire=0.03, delay=3), 160, 128, 1, 4),
    ("brunel_plus", dict(n=2500, n_exc=2000), 260, 128, 2, 2),
    ("vogels", dict(n=3000, n_exc=2400, plastic=PLASTIC_EXC_EXC, w0=0.05), 200, 192, 2, 8),
]


@pytest.mark.parametrize("hbits", [64, 128], ids=["h64", "h128"])
@pytest.mark.parametrize("filt,algo", [(0, 0), (1, 0), (0, 1)], ids=["auto", "codes", "lazy"])
@pytest.mark.parametrize("case", XCD_CASES,
                         ids=lambda c: "%s-%s-x%d" % (c[0], c[1].get("n", ""), c[5]))
def test_xcd_forced_rows_parity(case, filt, algo, hbits):
    """Forced rows split by target range over the XCDs (the waves of a
    range's XCDs take the entries of every forced row whose targets lie in
    that range, with the range's history codes in LDS): the same
    teacher-forced bar as the row-wise form."""
    name, kw, steps, width, chunks, parts = case
    p = wl.preset(name, **kw)
    log("xcd parity %s %s filter=%d algo=%d history=%d W=%d C=%d ranges=%d" % (
        name, kw, filt, algo, hbits, width, chunks, parts))
    net, o, cnt = teacher_forced_run(p, steps, LDS, slice_width=width, spike_chunks=chunks,
                                     stdp_filter=filt, plasticity_algorithm=algo,
                                     history_bits=hbits, stdp_xcd=parts)
    assert cnt["rows"] > 0 and cnt["weights"] > 0
    assert net.graph()["stdp_ranges"] == parts
    st = net.stats()
    assert st["stdp_forced_rows"] > 0 and st["device_errors"] == 0
    net.flush_plasticity()
    compare_all_plastic_weights(net, o)


@pytest.mark.parametrize("parts", [1, 2, 4, 8], ids=["auto", "x2", "x4", "x8"])
@pytest.mark.parametrize("chunks", [2, 32], ids=["fused", "two-launches"])
@pytest.mark.parametrize("hbits", [64, 128], ids=["h64", "h128"])
def test_xcd_partition_equals_rowwise(chunks, hbits, parts):
    """The forced rows split by target range and the row-wise form give the
    same weights bit for bit (the same arithmetic per synapse, history bits
    from the same codes or words), inside the fused pass and in the separate
    forced-row launch (32 chunks leave the pass too few slots), for every
    range count and the automatic one."""
    p = wl.preset("stress", n=6000, p_or_fanout=300, p_fire=0.02, delay=2)
    a = gpu_net(p, 256, chunks, history_bits=hbits, stdp_xcd=parts)  # by target range
    b = gpu_net(p, 256, chunks, history_bits=hbits)                  # row-wise
    assert a.graph()["stdp_ranges"] == (parts if parts > 1 else 2)  # 150 entries: 2 ranges
    assert b.graph()["stdp_ranges"] == 0
    for k in (1, 70, 150):
        a.step(k, LDS)
        b.step(k, LDS)
    sa, sb = a.state(), b.state()
    for key in ("hist", "t_last", "trace_pre", "trace_post", "input_exc"):
        assert np.array_equal(to_np(sa[key]), to_np(sb[key])), key
    assert np.array_equal(to_np(a.graph()["w"]), to_np(b.graph()["w"]))
    ta, tb = a.stats(), b.stats()
    for key in ("stdp_forced_rows", "stdp_synapse_updates", "stdp_weights_written",
                "device_errors"):
        assert ta[key] == tb[key], key
    assert ta["stdp_forced_rows"] > 0 and ta["device_errors"] == 0
