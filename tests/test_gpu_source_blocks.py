"""Blocks of steps of plastic networks of Bernoulli sources with D = 1
(snn_config.plastic_blocks; the stress network's configuration).

A source fires on a counter-based draw that no input changes (the stress
workload: each neuron fires independently with a fixed probability per
step), so one launch runs the neuron updates of up to 16 steps: each
neuron's spikes, histories and post traces, and each row's updates of every
step (transmitting, or forced by the history window) with their snapshots,
t_last and the pre trace carried from one update to the next (Sec. III-A:
a row is brought up to date only when it transmits or its history window is
about to overflow). The synapse pass of each step then runs on that step's
versions of the lists, histories and summaries.

Checked here:
  - bit-equality with the step-by-step path (one neuron launch and one fused
    synapse pass per step) over hundreds of steps in uneven calls: every
    state array, the ring, spike, transmitted and forced lists (ascending),
    all weights and all statistics; 64- and 128-step histories, history
    codes and the recency bitmap, lazy and lazy + event-driven plasticity,
    exc->exc plasticity (rows without plasticity transmit only), 16- and
    32-bit targets, one to four chunks, ragged sizes, networks of one
    workgroup and of one wave, block lengths capped (down to one step),
    heavy activity;
  - free runs against the oracle (both sides draw the same spikes): after
    calls of 1 to 132 steps (blocks cut at every call's end), spikes,
    lists, histories and the last step's delivered input, and the weights
    of the rows the last step made current; every plastic weight after a
    flush;
  - sequences that mix blocks with the separate part calls;
  - captured blocks replayed against eager steps.
Teacher-forced oracle parity of the same path (blocks of one step) runs in
test_gpu_parity.py, and the full-size stress network against per-synapse
oracle replays in test_gpu_fullsize.py.
"""

import numpy as np
import pytest

import workloads as wl
from workloads.presets import PLASTIC_EXC_EXC
from paper_2107_04092_amd import snn

from gpu_common import (gpu_net, oracle_net, to_np, log, same_state, compare_step, compare_rows,
                        compare_all_plastic_weights)

pytestmark = pytest.mark.gpu
LDS = snn.SNN_DELIVER_LDS_SLICE

CASES = [
    # preset overrides, slice width, chunks, extra config, steps
    (dict(n=3000, p_or_fanout=150, p_fire=0.03), 640, 1, dict(), 200),
    (dict(n=6000, p_or_fanout=200, p_fire=0.02), 1024, 4, dict(history_bits=128), 300),
    (dict(n=3001, p_or_fanout=100, p_fire=0.05), 512, 2, dict(plastic_blocks=5), 200),
    (dict(n=4000, p_or_fanout=150, p_fire=0.03), 512, 2, dict(stdp_filter=2), 200),
    (dict(n=4000, p_or_fanout=150, p_fire=0.03), 512, 2,
     dict(stdp_filter=2, history_bits=128, compressed_targets=0), 200),
    (dict(n=4000, p_or_fanout=150, p_fire=0.03), 512, 2, dict(plasticity_algorithm=1), 150),
    (dict(n=5000, n_exc=4000, plastic=PLASTIC_EXC_EXC, p_or_fanout=200, p_fire=0.02), 1024, 2,
     dict(), 250),
    # heavy activity: about 1,200 spikes and forced rows per step
    (dict(n=6000, p_or_fanout=1000, p_fire=0.2), 1024, 2, dict(history_bits=128), 60),
    # one workgroup (one wave, and a ragged wave); blocks of one step
    (dict(n=64, p_or_fanout=20, p_fire=0.05), 64, 1, dict(), 200),
    (dict(n=300, p_or_fanout=30, p_fire=0.05), 128, 2, dict(history_bits=128), 200),
    (dict(n=2000, p_or_fanout=100, p_fire=0.05), 512, 2, dict(plastic_blocks=1), 150),
]

SHORT = dict(plastic_blocks="B", history_bits="h", compressed_targets="ct",
             plasticity_algorithm="algo", stdp_filter="f")


def _id(c):
    kw, width, chunks, extra, _ = c
    return "n%d-W%d-C%d-%s" % (kw["n"], width, chunks,
                               "-".join("%s%s" % (SHORT[k], v) for k, v in sorted(extra.items()))
                               or "auto")


@pytest.mark.parametrize("case", CASES, ids=_id)
def test_source_blocks_equal_stepwise(case):
    kw, width, chunks, extra, steps = case
    p = wl.preset("stress", **kw)
    assert p.delay == 1
    log("source blocks vs stepwise %s W=%d C=%d %s steps=%d" % (kw, width, chunks, extra,
                                                                steps))
    a = gpu_net(p, width, chunks, **extra)
    b = gpu_net(p, width, chunks, **dict(extra, plastic_blocks=-1))
    assert a.graph()["block_steps"] == min(16, extra.get("plastic_blocks", 0) or 16)
    assert a.graph()["block_width"] == 0
    assert b.graph()["block_steps"] == 0
    # uneven calls: a block cut short at the end of each call
    done = 0
    for n_steps in (steps // 3, 1, 17, steps - steps // 3 - 18):
        a.step(n_steps, LDS)
        b.step(n_steps, LDS)
        done += n_steps
        same_state(a, b, "after %d steps" % done)
    st = a.stats()
    assert st["spikes"] > 0 and st["stdp_forced_rows"] > 0 and st["delivered_events"] > 0
    for net in (a, b):
        net.flush_plasticity()
    same_state(a, b, "after the flush")


def test_source_blocks_mixed_with_part_calls():
    """Blocks, then the separate part calls, then blocks again."""
    p = wl.preset("stress", n=3000, p_or_fanout=150, p_fire=0.03)
    a = gpu_net(p, 640, 2)
    b = gpu_net(p, 640, 2, plastic_blocks=-1)
    for net in (a, b):
        net.step(37, LDS)
        for _ in range(9):
            net.update_neurons()
            net.update_plasticity()
            net.deliver_spikes(LDS)
            net.advance()
        net.step(50, LDS)
    same_state(a, b, "mixed")


def test_captured_source_blocks_replay_equal_eager_steps():
    import torch
    p = wl.preset("stress", n=3000, p_or_fanout=150, p_fire=0.03)
    side = torch.cuda.Stream()
    a = gpu_net(p, 640, 2, stream=side)  # 37 steps captured: blocks of 16, 16, 5
    c = gpu_net(p, 640, 2)               # eager
    for net in (a, c):
        net.step(5, LDS)
    g = a.capture(37, LDS)
    try:
        assert a.state()["t"] == 5  # the capture ran nothing
        for k in range(6):
            a.replay(g)
            c.step(37, LDS)
            same_state(a, c, "replay %d" % k)
    finally:
        snn.snn_graph_destroy(g)


@pytest.mark.parametrize("hbits", [64, 128], ids=["h64", "h128"])
@pytest.mark.parametrize("kw", [dict(n=3000, p_or_fanout=150, p_fire=0.03),
                                # several updates of a row in one block: rows
                                # that transmit twice, forced rows that
                                # transmit later in the block
                                dict(n=2000, p_or_fanout=200, p_fire=0.1)],
                         ids=["p0.03", "p0.1"])
def test_source_blocks_free_run_matches_oracle(kw, hbits):
    p = wl.preset("stress", **kw)
    log("source blocks free run %s history=%d" % (kw, hbits))
    net = gpu_net(p, 640, 2, history_bits=hbits)
    assert net.graph()["block_steps"] == 16
    o = oracle_net(p)
    cache = {}
    t = n_w = 0
    for chunk in (16, 37, 1, 64, 50, 132):
        net.step(chunk, LDS)
        o.step(chunk)
        t += chunk
        rows = compare_step(net, o, "source blocks", t)
        n_w += compare_rows(net, o, rows, "rows made current at t=%d" % t, cache)
    assert n_w > 0
    net.flush_plasticity()
    compare_all_plastic_weights(net, o)
    st = net.stats()
    assert st["spikes"] == o.spikes_total > 0
    assert st["stdp_forced_rows"] > 0 and st["device_errors"] == 0
