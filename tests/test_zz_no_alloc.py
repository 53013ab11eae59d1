"""snn_step_static, the entry point for callers that cannot allocate: the
same steps as snn_step, with the list scans' scratch in the library's own
device array instead of the workspace. Compared with snn_step bit for bit on
two calls in a row, the second on a smaller network; a network whose scans
need more words than the array holds is refused before any launch."""

import numpy as np
import pytest

import workloads as wl
from workloads.presets import PLASTIC_NONE
from paper_2107_04092_amd import snn

from gpu_common import gpu_net, to_np, log

pytestmark = pytest.mark.gpu
LDS = snn.SNN_DELIVER_LDS_SLICE

KEYS = ("v", "refractory", "i_exc", "i_inh", "hist", "trace_post", "t_last", "trace_pre",
        "input_exc", "input_inh", "spike_mask", "ring_counts", "stdp_row_count")


def _same(a, b, d, what):
    sa, sb = a.state(), b.state()
    assert sa["t"] == sb["t"], what
    for k in KEYS:
        assert np.array_equal(to_np(sa[k]).view(np.uint8), to_np(sb[k]).view(np.uint8)), (what, k)
    ra, rb = to_np(sa["ring_lists"]).reshape(d, -1), to_np(sb["ring_lists"]).reshape(d, -1)
    for q, c in enumerate(to_np(sa["ring_counts"])):
        assert np.array_equal(ra[q, :c], rb[q, :c]), (what, "ring slot", q)
    a.flush_plasticity()
    b.flush_plasticity()
    assert np.array_equal(to_np(a.graph()["w"]), to_np(b.graph()["w"])), (what, "weights")
    ta, tb = a.stats(), b.stats()
    for k in ("steps", "spikes", "delivered_events", "stdp_rows", "stdp_weights_written",
              "device_errors"):
        assert ta[k] == tb[k], (what, k)
    assert ta["spikes"] > 0 and ta["device_errors"] == 0


@pytest.mark.parametrize("case", [
    # (preset, overrides, slice width, chunks, steps): two calls in a row, the
    # second smaller; then a delay-block network (16 status rows per call)
    [("stress", dict(n=6000, p_or_fanout=120, p_fire=0.03, delay=3), 1024, 2, 77),
     ("stress", dict(n=3000, p_or_fanout=60, p_fire=0.03, delay=3), 512, 1, 50)],
    [("brunel", dict(n=6000, n_exc=4800), 1024, 2, 45),
     ("tiny", dict(), 256, 1, 30)],
    # Bernoulli sources with D = 1: source blocks (16 status rows per block)
    [("stress", dict(n=6000, p_or_fanout=120, p_fire=0.03), 1024, 2, 77),
     ("stress", dict(n=3000, p_or_fanout=60, p_fire=0.03), 512, 1, 50)],
], ids=["plastic", "delay-blocks", "source-blocks"])
def test_static_step_equals_step(case):
    for name, kw, width, chunks, steps in case:
        p = wl.preset(name, **kw)
        log("static step %s %s W=%d C=%d steps=%d" % (name, kw, width, chunks, steps))
        a = gpu_net(p, width, chunks)
        b = gpu_net(p, width, chunks)
        a.step(steps, LDS)
        b.step_static(steps, LDS)
        _same(a, b, p.delay, "%s n=%d" % (name, p.n))


def test_static_step_refuses_networks_beyond_its_scratch():
    p = wl.preset("stress", n=4_300_000, p_or_fanout=1, plastic=PLASTIC_NONE)
    net = gpu_net(p, 4096, 1, build=False)
    with pytest.raises(snn.SnnError) as e:
        net.step_static(1)
    assert e.value.status == snn.SNN_EINVAL
    assert "status words" in str(e.value)
