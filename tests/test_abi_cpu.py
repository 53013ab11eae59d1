"""The C-ABI library loads, exports every declared symbol, agrees with the
binding on struct layouts, and rejects bad configurations before touching a
device. No GPU needed (no compute calls)."""

import ctypes
import os
import re
import subprocess

import pytest

from paper_2107_04092_amd import snn
import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "snn.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(snn_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = snn.load()
    names = _declared()
    assert len(names) >= 20
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(snn._SIGNATURES), set(names) ^ set(snn._SIGNATURES)


def _c_layout(tmp_path):
    prog = tmp_path / "layout.c"
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "snn.h"', 'int main(void){']
    for struct, cls in (("snn_config", snn.snn_config), ("snn_state_view", snn.snn_state_view),
                        ("snn_graph_view", snn.snn_graph_view), ("snn_stats", snn.snn_stats)):
        lines.append('printf("%s sizeof %%zu\\n", sizeof(%s));' % (struct, struct))
        for f, _ in cls._fields_:
            cf = "lambda" if f == "lambda_" else f
            lines.append('printf("%s %s %%zu\\n", offsetof(%s, %s));' % (struct, f, struct, cf))
    lines.append("return 0;}")
    prog.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", "-I", os.path.dirname(HEADER), str(prog), "-o", str(exe)],
                   check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout
    return {tuple(l.split()[:2]): int(l.split()[2]) for l in out.splitlines()}


def test_struct_layouts_match_header(tmp_path):
    lay = _c_layout(tmp_path)
    for struct, cls in (("snn_config", snn.snn_config), ("snn_state_view", snn.snn_state_view),
                        ("snn_graph_view", snn.snn_graph_view), ("snn_stats", snn.snn_stats)):
        assert lay[(struct, "sizeof")] == ctypes.sizeof(cls), struct
        for f, _ in cls._fields_:
            assert lay[(struct, f)] == getattr(cls, f).offset, (struct, f)


@pytest.mark.parametrize("field,value,msg", [
    ("n", 0, "n must be"),
    ("n_exc", 2000, "n_exc"),
    ("delay_steps", 0, "delay_steps"),
    ("delay_steps", 65, "delay_steps"),
    ("slice_width", 100, "multiple of 64"),
    ("slice_width", 40960 + 64, "160 KiB"),
    ("spike_chunks", 0, "spike_chunks"),
    ("neuron_model", 7, "neuron_model"),
    ("plastic", 9, "plastic"),
    ("stdp_layout", 2, "stdp_layout"),
    ("stdp_filter", 4, "stdp_filter"),
    ("plasticity_algorithm", 3, "plasticity_algorithm"),
    ("history_bits", 96, "history_bits"),
    ("compressed_targets", 2, "compressed_targets"),
    ("plastic_blocks", -2, "plastic_blocks"),
    ("plastic_blocks", 65, "plastic_blocks"),
    ("plastic_block_width", 96, "plastic_block_width"),
    ("plastic_block_width", 512, "plastic_block_width"),
    ("poisson_len", 33, "poisson_len"),
    ("dt_ms", float("nan"), "NaN"),
    ("tau_m_ms", 0.0, "tau_m_ms"),
])
def test_create_rejects_bad_config(field, value, msg):
    cfg = snn.config_from_preset(wl.preset("tiny"))
    setattr(cfg, field, value)
    with pytest.raises(snn.SnnError) as e:
        snn.snn_create(cfg, 0)
    assert e.value.status == snn.SNN_EINVAL
    assert msg in str(e.value)


def test_create_rejects_bad_stdp_and_cuba_config():
    cfg = snn.config_from_preset(wl.preset("brunel_plus"))
    cfg.mu = 1.0
    with pytest.raises(snn.SnnError, match="mu"):
        snn.snn_create(cfg, 0)
    cfg = snn.config_from_preset(wl.preset("vogels"))
    cfg.slice_width = 40960  # two accumulators do not fit
    with pytest.raises(snn.SnnError, match="160 KiB"):
        snn.snn_create(cfg, 0)
    cfg = snn.config_from_preset(wl.preset("stress"))
    cfg.p_fire = 1.5
    with pytest.raises(snn.SnnError, match="p_fire"):
        snn.snn_create(cfg, 0)
    cfg = snn.config_from_preset(wl.preset("brunel_plus"), slice_width=320)
    cfg.plastic_block_width = 128  # target groups must tile the slices
    with pytest.raises(snn.SnnError, match="plastic_block_width"):
        snn.snn_create(cfg, 0)



def test_poisson_table_must_be_monotone():
    tab = list(wl.poisson_cdf_table(2.0))
    tab[3], tab[4] = tab[4], tab[3]
    cfg = snn.config_from_preset(wl.preset("brunel"), poisson_table=tab)
    with pytest.raises(snn.SnnError, match="non-decreasing"):
        snn.snn_create(cfg, 0)


def test_status_strings():
    lib = snn.load()
    for s in range(5):
        assert lib.snn_status_string(s)
    assert lib.snn_last_error(None) == b"null context"
