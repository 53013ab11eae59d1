"""Free-running simulations: the GPU's mean firing rate must match the
oracle's within 2% (runs long enough for >= 1e5 spikes, so Poisson noise is
about 0.3%)."""

import pytest

import workloads as wl
from paper_2107_04092_amd import snn

from gpu_common import gpu_net, oracle_net, rate_hz, log

pytestmark = pytest.mark.gpu


def _free_run(p, steps, mode, chunk=5000):
    net = gpu_net(p)
    o = oracle_net(p)
    done = 0
    while done < steps:
        k = min(chunk, steps - done)
        net.step(k, mode)
        o.step(k)
        done += k
        log("  %s: %d/%d steps" % (p.name, done, steps))
    g = net.stats()["spikes"]
    return g, o.spikes_total


@pytest.mark.parametrize("name,kw,steps,mode", [
    ("tiny", dict(), 100_000, snn.SNN_DELIVER_LDS_SLICE),
    ("vogels", dict(), 100_000, snn.SNN_DELIVER_LDS_SLICE),
    ("brunel_plus", dict(n=2500, n_exc=2000, slice_width=512), 10_000,
     snn.SNN_DELIVER_LDS_SLICE),
    ("brunel_plus", dict(n=2500, n_exc=2000, slice_width=512), 10_000,
     snn.SNN_DELIVER_GLOBAL_ATOMIC),
])
def test_free_running_rate_within_2_percent(name, kw, steps, mode):
    p = wl.preset(name, **kw)
    log("rate %s %s steps=%d mode=%d" % (name, kw, steps, mode))
    g, o = _free_run(p, steps, mode)
    rg, ro = rate_hz(g, p.n, steps), rate_hz(o, p.n, steps)
    log("  gpu %.3f Hz (%d spikes), oracle %.3f Hz (%d spikes)" % (rg, g, ro, o))
    assert o >= 100_000
    assert abs(rg - ro) <= 0.02 * ro
