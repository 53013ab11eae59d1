"""Kernel timing: the events each launch places around its kernel give
positive device times for the parts a step runs, and stop when asked."""

import pytest

import workloads as wl
from paper_2107_04092_amd import snn

from gpu_common import gpu_net

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("mode", [snn.SNN_DELIVER_LDS_SLICE, snn.SNN_DELIVER_GLOBAL_ATOMIC])
def test_kernel_times_cover_the_parts_of_a_step(mode):
    p = wl.preset("stress", n=3000, p_or_fanout=100, p_fire=0.02)
    net = gpu_net(p, slice_width=512, spike_chunks=2)
    net.record_kernel_times(5)
    net.step(8, mode)  # more steps than recorded
    t, steps = net.kernel_times()
    assert steps == 5
    assert t["neuron"] > 0 and t["delivery"] > 0
    if mode == snn.SNN_DELIVER_LDS_SLICE:
        # the fused synapse pass: plasticity and delivery in one launch,
        # recorded as the delivery part
        assert t["plasticity"] == 0
    else:
        assert t["plasticity"] > 0
    net.record_kernel_times(0)
    net.step(2, mode)
    assert net.kernel_times()[1] == 0


def test_kernel_times_of_separate_parts():
    """A network whose delivery items leave too few slots for the fused pass
    (16 slices x 32 chunks) runs plasticity and delivery as two launches."""
    p = wl.preset("stress", n=8192, p_or_fanout=100, p_fire=0.02)
    net = gpu_net(p, slice_width=512, spike_chunks=32)
    net.record_kernel_times(4)
    net.step(4, snn.SNN_DELIVER_LDS_SLICE)
    t, steps = net.kernel_times()
    assert steps == 4
    for part in snn.KERNEL_PARTS:
        assert t[part] > 0, part


def test_kernel_times_without_plasticity():
    p = wl.preset("tiny")
    net = gpu_net(p, slice_width=256)
    net.record_kernel_times(3)
    net.step(3, snn.SNN_DELIVER_LDS_SLICE)
    t, steps = net.kernel_times()
    assert steps == 3 and t["plasticity"] == 0 and t["delivery"] > 0
