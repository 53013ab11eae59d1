"""Blocks of steps of plastic networks with D >= 2 (snn_config.plastic_blocks).

A block of B <= D-1 steps is one plan launch (each step's rows, from the
histories) and one run launch in which each workgroup owns a group of
targets through all B steps (their neuron update; the plasticity and
delivery of every listed row's entries onto them). The weight a row
delivers at step t depends only on its targets' spikes and on pre spikes
that arrived by t (Sec. III-A, a synapse sees its pre spike D-1 steps after
emission), so no workgroup needs another's results within the block.

Checked here:
  - bit-equality with the step-by-step path (three parts per step, or the
    fused pass) over hundreds of steps: every state array, every delay-ring
    list, the forced-row list, all weights and all statistics, for LIF and
    CUBA networks, 64- and 128-step histories, lazy and lazy + event-driven
    plasticity, group widths 64 / 128 / 256, ragged last groups, compressed
    targets on and off, block lengths from 1 to 16, and sequences that mix
    blocks with the separate part calls;
  - teacher-forced oracle parity with blocks of one step (the oracle's state
    and input handed over before every step; spikes, histories and
    potentials bit-exact, inputs and weights within |g-o| <= 1e-5|o| + 1e-7);
  - the group pivots against a lower bound computed on the host;
  - captured blocks replayed against eager steps.
The full-size Brunel+ network (25,000 neurons, 62.5M synapses) is compared
with the step-by-step path in test_gpu_fullsize.py.
"""

import numpy as np
import pytest

import workloads as wl
from workloads.presets import PLASTIC_ALL, PLASTIC_EXC_EXC, LIF_CUBA
from paper_2107_04092_amd import snn

from gpu_common import (gpu_net, to_np, log, teacher_forced_run, compare_all_plastic_weights,
                        same_state)

pytestmark = pytest.mark.gpu
LDS = snn.SNN_DELIVER_LDS_SLICE

CASES = [
    # name, preset overrides, slice width, chunks, extra config, steps
    ("brunel_plus", dict(n=2500, n_exc=2000), 512, 2, dict(), 300),
    ("brunel_plus", dict(n=2517, n_exc=2001), 512, 1, dict(plastic_block_width=128), 260),
    ("brunel_plus", dict(n=3000, n_exc=2400), 1024, 4,
     dict(plastic_block_width=256, history_bits=128), 300),
    ("brunel_plus", dict(n=2500, n_exc=2000, delay=2), 512, 2, dict(), 200),
    ("brunel_plus", dict(n=2500, n_exc=2000, delay=40), 512, 2,
     dict(plastic_blocks=5, compressed_targets=0), 230),
    ("brunel_plus", dict(n=2500, n_exc=2000), 512, 2, dict(plasticity_algorithm=1), 200),
    ("vogels", dict(n=3000, n_exc=2400, plastic=PLASTIC_EXC_EXC, w0=0.05, delay=4), 512, 2,
     dict(), 250),
    ("vogels", dict(n=3000, n_exc=2400, plastic=PLASTIC_EXC_EXC, w0=0.05, delay=4), 512, 1,
     dict(history_bits=128, plastic_block_width=64), 250),
    ("stress", dict(n=3000, p_or_fanout=150, p_fire=0.03, delay=3), 640, 1, dict(), 200),
    ("stress", dict(n=4100, p_or_fanout=300, p_fire=0.02, delay=17), 1024, 3,
     dict(history_bits=128), 200),
    # heavy activity: about 1,200 rows per step (more than one staging batch
    # of 1,024), over 8,192 entries per group and step (several windows),
    # and more records per block than a workgroup holds in LDS (each step's
    # records loaded when it runs)
    ("stress", dict(n=6000, p_or_fanout=1000, p_fire=0.2, delay=17), 1024, 2,
     dict(plastic_block_width=64), 60),
    # the same activity in blocks short enough to keep their records in LDS
    ("stress", dict(n=6000, p_or_fanout=1000, p_fire=0.2, delay=3), 1024, 2,
     dict(plastic_block_width=64), 60),
]


SHORT = dict(plastic_block_width="gw", plastic_blocks="B", history_bits="h",
             compressed_targets="ct", plasticity_algorithm="algo")


@pytest.mark.parametrize("case", CASES, ids=lambda c: "%s-n%d-d%d-%s" % (
    c[0], c[1]["n"], wl.preset(c[0], **c[1]).delay,
    "-".join("%s%s" % (SHORT[k], v) for k, v in sorted(c[4].items())) or "auto"))
def test_blocks_equal_stepwise(case):
    name, kw, width, chunks, extra, steps = case
    p = wl.preset(name, **kw)
    log("blocks vs stepwise %s %s W=%d C=%d %s steps=%d" % (name, kw, width, chunks, extra,
                                                            steps))
    a = gpu_net(p, width, chunks, **extra)
    b = gpu_net(p, width, chunks, **dict(extra, plastic_blocks=-1))
    ga = a.graph()
    assert ga["block_steps"] == min(p.delay - 1, 15, extra.get("plastic_blocks", 0) or 15)
    assert ga["block_width"] == extra.get("plastic_block_width", ga["block_width"])
    assert b.graph()["block_steps"] == 0
    # uneven calls: a block cut short at the end of each call
    done = 0
    for k, n_steps in enumerate((steps // 3, 1, steps - steps // 3 - 1)):
        a.step(n_steps, LDS)
        b.step(n_steps, LDS)
        done += n_steps
        same_state(a, b, "after %d steps" % done)
    st = a.stats()
    assert st["spikes"] > 0 and st["stdp_forced_rows"] > 0 and st["delivered_events"] > 0
    for net in (a, b):
        net.flush_plasticity()
    same_state(a, b, "after the flush")


def test_blocks_mixed_with_part_calls():
    """Blocks, then the separate part calls, then blocks again: the lists the
    last launch of a call rebuilds are those the part calls need."""
    p = wl.preset("brunel_plus", n=2500, n_exc=2000)
    a = gpu_net(p, 512, 2)
    b = gpu_net(p, 512, 2, plastic_blocks=-1)
    for net in (a, b):
        net.step(37, LDS)
        for _ in range(9):
            net.update_neurons()
            net.update_plasticity()
            net.deliver_spikes(LDS)
            net.advance()
        net.step(50, LDS)
    same_state(a, b, "mixed")


def test_block_pivots_match_host_lower_bound():
    import torch
    p = wl.preset("brunel_plus", n=2517, n_exc=2001)
    for gw in (64, 128, 256):
        net = gpu_net(p, 512, 2, plastic_block_width=gw)
        g = net.graph()
        assert g["block_width"] == gw
        n = net.n
        groups = (n + gw - 1) // gw
        piv = to_np(g["block_pivots"]).reshape(n, groups + 1)
        rp = to_np(g["row_ptr"])
        col = to_np(g["col"])
        for k in range(0, n, 97):
            row = col[rp[k]:rp[k + 1]]
            want = np.searchsorted(row, np.arange(groups + 1) * gw, side="left")
            want[-1] = len(row)
            assert np.array_equal(piv[k], want), (gw, k)
        del net
        torch.cuda.synchronize()


TF_CASES = [
    ("brunel_plus", dict(n=2500, n_exc=2000), 300, 512, 2),
    ("stress", dict(n=3000, p_or_fanout=150, p_fire=0.03, delay=3), 160, 640, 1),
    ("vogels", dict(n=3000, n_exc=2400, plastic=PLASTIC_EXC_EXC, w0=0.05, delay=4), 200, 512, 2),
]


@pytest.mark.parametrize("hbits", [64, 128], ids=["h64", "h128"])
@pytest.mark.parametrize("case", TF_CASES, ids=lambda c: "%s-%s" % (c[0], c[1].get("n", "")))
def test_blocks_teacher_forced_parity(case, hbits):
    """Blocks of one step under teacher forcing: the run kernel's neuron
    update, plasticity and delivery against the oracle at every step."""
    name, kw, steps, width, chunks = case
    p = wl.preset(name, **kw)
    log("block parity %s %s history=%d steps=%d" % (name, kw, hbits, steps))
    net, o, cnt = teacher_forced_run(p, steps, LDS, slice_width=width, spike_chunks=chunks,
                                     history_bits=hbits, plastic_blocks=1)
    assert net.graph()["block_steps"] == 1
    assert cnt["spikes"] > 0 and cnt["rows"] > 0 and cnt["weights"] > 0
    net.flush_plasticity()
    compare_all_plastic_weights(net, o)
    st = net.stats()
    assert st["steps"] == steps and st["spikes"] == cnt["spikes"]
    assert st["stdp_forced_rows"] > 0 and st["device_errors"] == 0


def test_captured_blocks_replay_equal_eager_steps():
    import torch
    p = wl.preset("brunel_plus", n=2500, n_exc=2000)
    side = torch.cuda.Stream()
    a = gpu_net(p, 512, 2, stream=side)  # 30 steps captured: blocks of 14, 14, 2
    c = gpu_net(p, 512, 2)               # eager
    for net in (a, c):
        net.step(5, LDS)
    g = a.capture(30, LDS)
    try:
        assert a.state()["t"] == 5  # the capture ran nothing
        for k in range(8):
            a.replay(g)
            c.step(30, LDS)
            same_state(a, c, "replay %d" % k)
    finally:
        snn.snn_graph_destroy(g)
