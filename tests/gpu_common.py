"""Shared helpers of the GPU parity tests: build the same seeded network on the
GPU (through the C ABI) and in the CPU oracle, and compare them under the
tolerances the parity bar fixes."""

import math
import sys

import numpy as np

import workloads as wl
from paper_2107_04092_amd import snn

RTOL = 1e-5   # delivered inputs and STDP weights: |g - o| <= RTOL |o| + ATOL
ATOL = 1e-7


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def torch_mod():
    import torch
    return torch


def gpu_net(p, slice_width=None, spike_chunks=None, build=True, stream=None, **cfg_kw):
    torch = torch_mod()
    tab = wl.poisson_cdf_table(p.poisson_mu)
    cfg = snn.config_from_preset(p, tab, slice_width=slice_width, spike_chunks=spike_chunks,
                                 **cfg_kw)
    net = snn.Network(cfg, stream=stream)
    if build:
        net.build_random(p.graph_kind, p.p_or_fanout, p.w_exc, p.w_inh)
        st = wl.initial_state(p)
        net.set_state(0, v=torch.from_numpy(st["v"]))
    return net


def oracle_net(p, build=True):
    from oracle import oracle
    o = oracle.Oracle(p, wl.poisson_cdf_table(p.poisson_mu))
    if build:
        o.build_random()
        o.set_neurons(**wl.initial_state(p))
    return o


def to_np(t):
    return t.detach().cpu().numpy()


def hist_np(t):
    return to_np(t).view(np.uint64)


def assert_close(g, o, what, rtol=RTOL, atol=ATOL, terms=None):
    g = np.asarray(g, dtype=np.float64)
    o = np.asarray(o, dtype=np.float64)
    assert g.shape == o.shape, (what, g.shape, o.shape)
    err = np.abs(g - o)
    bad = err > rtol * np.abs(o) + atol
    if bad.any():
        i = int(np.nonzero(bad)[0][0])
        diag = ""
        if terms is not None:
            diag = " |g-o|/sum|terms| = %.3g" % (err[i] / max(terms[i], 1e-30))
        raise AssertionError("%s: %d of %d outside rtol %g atol %g; first at %d: gpu %.9g "
                             "oracle %.9g%s" % (what, int(bad.sum()), bad.size, rtol, atol, i,
                                                g[i], o[i], diag))


def oracle_hist(st, words):
    """The oracle's spike history in the GPU layout (words per neuron, neuron-major)."""
    if words == 1:
        return st["hist"]
    return np.stack([st["hist"], st["hist_old"]], axis=1).reshape(-1)


def force_from_oracle(net, o, t):
    """Teacher forcing: hand the oracle's neuron state and pending input to the GPU."""
    torch = torch_mod()
    st = o.neurons()
    a_e, a_i = o.input()
    h = np.ascontiguousarray(oracle_hist(st, net.history_words))
    kw = dict(v=torch.from_numpy(st["v"]), refractory=torch.from_numpy(st["refractory"]),
              hist=torch.from_numpy(h.view(np.int64)),
              input_exc=torch.from_numpy(a_e))
    if net.cfg.neuron_model == snn.SNN_LIF_CUBA:
        kw.update(i_exc=torch.from_numpy(st["i_exc"]), i_inh=torch.from_numpy(st["i_inh"]),
                  input_inh=torch.from_numpy(a_i))
    net.set_state(t, **kw)


def plastic_index(rp, pend, rows):
    """Edge indices of the plastic prefixes of the given rows."""
    starts = rp[rows]
    lens = pend[rows]
    if lens.sum() == 0:
        return np.zeros(0, np.int64)
    return np.concatenate([np.arange(s, s + l) for s, l in zip(starts, lens) if l > 0])


def compare_step(net, o, mode_name, t, check_rows=True):
    """Bit-exact spikes/histories/potentials; tolerance on inputs and weights."""
    s = net.state()
    mask, lst = o.spikes()
    ost = o.neurons()
    g_mask = hist_np(s["spike_mask"])
    assert np.array_equal(g_mask, mask), ("spike mask", t, mode_name)
    cnt = int(to_np(s["spike_count"])[0])
    assert cnt == len(lst), ("spike count", t, cnt, len(lst))
    assert np.array_equal(to_np(s["spike_list"])[:cnt], lst), ("spike list", t)
    assert np.array_equal(hist_np(s["hist"]), oracle_hist(ost, net.history_words)), ("history", t)
    assert np.array_equal(to_np(s["v"]).view(np.uint32), ost["v"].view(np.uint32)), ("V", t)
    assert np.array_equal(to_np(s["refractory"]), ost["refractory"]), ("refractory", t)
    a_e, a_i = o.input()
    assert_close(to_np(s["input_exc"]), a_e, "delivered input (t=%d, %s)" % (t, mode_name))
    if net.cfg.neuron_model == snn.SNN_LIF_CUBA:
        assert_close(to_np(s["input_inh"]), a_i, "delivered inh input (t=%d)" % t)
        assert np.array_equal(to_np(s["i_exc"]).view(np.uint32), ost["i_exc"].view(np.uint32))
        assert np.array_equal(to_np(s["i_inh"]).view(np.uint32), ost["i_inh"].view(np.uint32))
    rows = None
    if check_rows and net.cfg.plastic != snn.SNN_PLASTIC_NONE:
        # rows made current at this step: those forced by the history window
        # and the plastic rows that transmitted
        nf = int(to_np(s["stdp_row_count"])[0])
        nt = int(to_np(s["tx_count"])[0])
        n_plastic = net.n if net.cfg.plastic == snn.SNN_PLASTIC_ALL else net.cfg.n_exc
        tx = to_np(s["tx_list"])[:nt]
        rows = np.unique(np.concatenate([to_np(s["stdp_rows"])[:nf], tx[tx < n_plastic]]))
    return rows


def compare_rows(net, o, rows, what, graph_cache):
    """Weights of the plastic prefixes of `rows`: GPU (just made current) vs oracle."""
    if rows is None or len(rows) == 0:
        return 0
    g = graph_cache.setdefault("g", net.graph())
    if "rp" not in graph_cache:
        graph_cache["rp"] = to_np(g["row_ptr"])
        graph_cache["pend"] = to_np(g["plastic_end"])
    idx = plastic_index(graph_cache["rp"], graph_cache["pend"], rows)
    if len(idx) == 0:
        return 0
    torch = torch_mod()
    gw = to_np(g["w"][torch.from_numpy(idx).to(g["w"].device)])
    ow = o.weights_at(idx)
    assert_close(gw, ow, what)
    return len(idx)


def teacher_forced_run(p, steps, mode, slice_width=None, spike_chunks=None, check_every=1,
                       progress=0, **cfg_kw):
    """Runs `steps` teacher-forced steps; returns (net, oracle, counters).
    With progress > 0 a line is logged every `progress` steps."""
    net = gpu_net(p, slice_width, spike_chunks, **cfg_kw)
    o = oracle_net(p)
    cache = {}
    n_rows = n_w = n_spk = 0
    for t in range(steps):
        if progress and t % progress == 0:
            log("  teacher-forced step %d/%d (%d rows, %d weights checked)" % (
                t, steps, n_rows, n_w))
        force_from_oracle(net, o, t)
        o.step()
        net.step(1, mode)
        if t % check_every == 0 or t == steps - 1:
            rows = compare_step(net, o, "mode %d" % mode, t)
            n_w += compare_rows(net, o, rows, "STDP rows at t=%d" % t, cache)
            n_rows += 0 if rows is None else len(rows)
        n_spk += len(o.spikes()[1])
    return net, o, dict(rows=n_rows, weights=n_w, spikes=n_spk)


def compare_all_plastic_weights(net, o):
    """After a flush every plastic weight is current on both sides."""
    g = net.graph()
    rp = to_np(g["row_ptr"])
    pend = to_np(g["plastic_end"])
    idx = plastic_index(rp, pend, np.arange(net.n))
    gw = to_np(g["w"])
    ow = o.weights()
    assert_close(gw[idx], ow[idx], "all plastic weights after flush")
    # non-plastic weights never change
    mask = np.ones(len(gw), bool)
    mask[idx] = False
    assert np.array_equal(gw[mask].astype(np.float64), ow[mask])
    return len(idx)


def rate_hz(spikes, n, steps, dt_ms=0.1):
    return spikes / n / (steps * dt_ms * 1e-3)


def poisson_sigma(count):
    return math.sqrt(max(count, 1))


KEYS = ("v", "refractory", "i_exc", "i_inh", "hist", "trace_post", "t_last", "trace_pre",
        "input_exc", "input_inh", "spike_mask", "ring_counts", "spike_count", "tx_count",
        "stdp_row_count")
STAT_KEYS = ("steps", "spikes", "delivered_events", "stdp_rows", "stdp_forced_rows",
             "stdp_synapse_updates", "stdp_weights_written", "stdp_forced_synapse_updates",
             "stdp_forced_weights_written", "device_errors")


def same_state(a, b, what, weights=True):
    sa, sb = a.state(), b.state()
    assert sa["t"] == sb["t"], (what, "t", sa["t"], sb["t"])
    for k in KEYS:
        ga, gb = to_np(sa[k]), to_np(sb[k])
        assert np.array_equal(ga.view(np.uint8), gb.view(np.uint8)), (what, k)
    for lst, cnt in (("spike_list", "spike_count"), ("tx_list", "tx_count"),
                     ("stdp_rows", "stdp_row_count")):
        c = int(to_np(sa[cnt])[0])
        assert np.array_equal(to_np(sa[lst])[:c], to_np(sb[lst])[:c]), (what, lst)
    d = a.cfg.delay_steps
    ra = to_np(sa["ring_lists"]).reshape(d, -1)
    rb = to_np(sb["ring_lists"]).reshape(d, -1)
    for q, c in enumerate(to_np(sa["ring_counts"])):
        assert np.array_equal(ra[q, :c], rb[q, :c]), (what, "ring slot", q)
        assert np.all(np.diff(ra[q, :c]) > 0), (what, "ring slot ascending", q)
    if weights:
        wa, wb = to_np(a.graph()["w"]), to_np(b.graph()["w"])
        assert np.array_equal(wa.view(np.uint32), wb.view(np.uint32)), (what, "weights")
    ta, tb = a.stats(), b.stats()
    for k in STAT_KEYS:
        assert ta[k] == tb[k], (what, k, ta[k], tb[k])
    assert ta["device_errors"] == 0, what
