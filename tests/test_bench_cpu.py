"""bench.py without a GPU: the one-GPU guard, the algorithmic byte counts the
roofline divides, and the source digest that keys the committed traffic
counters."""

import importlib.util
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def bench_module():
    spec = importlib.util.spec_from_file_location("bench", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


STATS = {"stdp_forced_synapse_updates": 1000, "stdp_forced_weights_written": 300,
         "stdp_forced_rows": 7, "delivered_events": 5000, "spikes": 50,
         "stdp_weights_written": 900, "stdp_rows": 57}


@pytest.mark.parametrize("hw", [1, 2])
def test_stdp_bytes_by_hand(hw):
    b = bench_module()
    n, launches = 100, 3
    want = 8 * 1000 + 4 * 300 + (32 + 8 * hw) * 7 + 8 * hw * n * launches
    assert b.stdp_bytes(STATS, n, launches, hw) == want


@pytest.mark.parametrize("hw", [1, 2])
@pytest.mark.parametrize("chunks", [1, 2])
def test_delivery_bytes_by_hand(hw, chunks):
    b = bench_module()
    n, s, nacc, launches = 100, 4, 1, 3
    wb = 4 * nacc * n if chunks == 1 else 8 * chunks * nacc * n
    want = (2 + 4) * 5000 + 4 * (900 - 300) + 20 * 50 * s + (wb + (8 * hw + 4) * n) * launches
    assert b.delivery_bytes(STATS, n, s, chunks, nacc, launches, "lds", 2, hw) == want
    glob = 16 * 5000 + 20 * 50 + 8 * nacc * n * launches
    assert b.delivery_bytes(STATS, n, s, chunks, nacc, launches, "global", 4, hw) == glob


def test_survey_bytes_by_hand():
    """The survey's per-step count on the stress network in steady state
    (2,639 rows made current, 1,388 of them forced, 1,251 spikes of 1,000
    synapses, 123 slices, two chunks): 48.3 MB as the count is written,
    38.3 MB less the fused pass's single read of the transmitting rows."""
    b = bench_module()
    steps, n = 10, 250_000
    st = {"stdp_synapse_updates": 2_639_000 * steps, "stdp_rows": 2_639 * steps,
          "stdp_forced_synapse_updates": 1_388_000 * steps, "delivered_events": 1_251_000 * steps,
          "spikes": 1_251 * steps}
    sb = b.survey_bytes(st, steps, n, 123, 2, 1, fused=True)
    stdp = 12 * 2_639_000 + 16 * 2_639 + 16 * n
    dlv = 8 * 1_251_000 + 1_251 * 124 * 4 + 2 * n * 4
    assert sb["stdp"] == pytest.approx(stdp) and sb["delivery"] == pytest.approx(dlv)
    assert sb["as_written"] == pytest.approx(48.34e6, rel=1e-3)
    assert sb["algorithmic"] == pytest.approx(stdp + dlv - 8 * 1_251_000, rel=1e-12)
    assert sb["algorithmic"] == pytest.approx(38.33e6, rel=1e-3)
    # no deduction where delivery re-reads the rows (global atomics), and no
    # STDP bytes without plastic rows
    assert b.survey_bytes(st, steps, n, 123, 2, 1, fused=False)["fused_deduction"] == 0
    st0 = dict(st, stdp_rows=0, stdp_synapse_updates=0, stdp_forced_synapse_updates=0)
    assert b.survey_bytes(st0, steps, n, 123, 2, 1, fused=True)["stdp"] == 0


def test_cpu_model_reads_the_host():
    b = bench_module()
    name, ncpu = b.cpu_model()
    assert ncpu >= 1
    assert name is None or isinstance(name, str)


def test_digest_ignores_comments_and_layout():
    b = bench_module()
    a = "int f(int x) { // a comment\n  return x + 1; /* block\n comment */ }\n"
    c = "int f(int x) {\n\n  return    x + 1;   }"
    norm = lambda t: " ".join(b._COMMENT.sub(" ", t).split())
    assert norm(a) == norm(c)
    assert norm(a) != norm(a.replace("x + 1", "x + 2"))
    assert len(b.kernel_source_digest()) == 16


def test_traffic_is_dropped_for_other_sources(monkeypatch):
    b = bench_module()
    d = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))
    kernel = next(iter(d["stress"]))
    monkeypatch.setattr(b, "kernel_source_digest", lambda: d["stress"][kernel]["source_digest"])
    assert b.load_traffic(kernel, "stress") == float(d["stress"][kernel]["bytes_per_launch"])
    monkeypatch.setattr(b, "kernel_source_digest", lambda: "0" * 16)
    assert b.load_traffic(kernel, "stress") is None


def test_write_traffic_scales_by_the_reference_copy(tmp_path, monkeypatch):
    """profiles/traffic.json from two counter databases: each kernel's KiB per
    dispatch (after the first quarter) scaled by the reference copy's reading
    for its known size."""
    import sqlite3
    b = bench_module()
    dbs = []
    for counter, copy_kib, kern in (("FETCH_SIZE", 1024.0, [10.0, 100.0, 100.0, 100.0]),
                                    ("WRITE_SIZE", 2048.0, [7.0, 50.0, 50.0, 50.0])):
        path = str(tmp_path / (counter + ".db"))
        con = sqlite3.connect(path)
        con.execute("create table counters_collection (kernel_name text, counter_name text, "
                    "value real)")
        rows = [("__amd_rocclr_copyBuffer", counter, copy_kib)]
        rows += [("void snn::(anonymous namespace)::k_synapse_pass<true, 2>(a, b, int)",
                  counter, v) for v in kern]
        con.executemany("insert into counters_collection values (?, ?, ?)", rows)
        con.commit()
        con.close()
        dbs.append(path)
    monkeypatch.setattr(b, "ROOT", str(tmp_path))
    os.makedirs(tmp_path / "profiles")
    monkeypatch.setattr(b, "kernel_source_digest", lambda: "abc")
    b.write_traffic(dbs[0], dbs[1], "stress", 2)  # 2 MiB = 2048 KiB each way
    d = json.load(open(tmp_path / "profiles" / "traffic.json"))
    e = d["stress"]["k_synapse_pass"]
    assert e["fetch_kib"] == 100.0 and e["write_kib"] == 50.0
    assert e["fetch_scale"] == 2.0 and e["write_scale"] == 1.0
    assert e["bytes_per_launch"] == round((100.0 * 2.0 + 50.0 * 1.0) * 1024)
    assert e["source_digest"] == "abc" and e["dispatches"] == 3


def test_stdp_xcd_choices_map_to_the_config_field(monkeypatch):
    b = bench_module()
    assert b.XCD_ARG == {"off": 0, "auto": 1, "2": 2, "4": 4, "8": 8}
    for arg, want in (([], 0), (["--stdp-xcd", "auto"], 1), (["--stdp-xcd", "4"], 4)):
        monkeypatch.setattr(sys, "argv", ["bench.py"] + arg)
        assert b.XCD_ARG[b.parse().stdp_xcd] == want


def test_plastic_block_choices_map_to_the_config_field(monkeypatch):
    b = bench_module()
    for arg, want in (([], 0), (["--plastic-blocks", "off"], -1),
                      (["--plastic-blocks", "5"], 5)):
        monkeypatch.setattr(sys, "argv", ["bench.py"] + arg)
        assert b.block_arg(b.parse().plastic_blocks) == want
    for bad in ("0", "65", "x"):
        with pytest.raises(ValueError):
            b.block_arg(bad)
