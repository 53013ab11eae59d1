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
    for part in snn.KERNEL_PARTS:
        assert t[part] > 0, part
    net.record_kernel_times(0)
    net.step(2, mode)
    assert net.kernel_times()[1] == 0


def test_kernel_times_without_plasticity():
    p = wl.preset("tiny")
    net = gpu_net(p, slice_width=256)
    net.record_kernel_times(3)
    net.step(3, snn.SNN_DELIVER_LDS_SLICE)
    t, steps = net.kernel_times()
    assert steps == 3 and t["plasticity"] == 0 and t["delivery"] > 0
