"""ctypes binding of the CPU oracle (snn_oracle.c).

TEST INFRASTRUCTURE ONLY: the correctness reference for the HIP library.
Only the tests, the smoke check and the CPU-baseline leg of the benchmark may
import this module; the library itself never does and fails loudly without
its own HIP build.

Parity status of each oracle function (what pins it, see tests/test_oracle_*.py):
  oracle_rng            pinned: published SplitMix64 output vectors
  oracle_pivots         pinned: worked example of Fig. 1
  neuron update (LIF)   pinned: Euler closed form, threshold step 479, period 529
  neuron update (Bern.) pinned: empirical rate vs p, mask/list/history invariants
  Poisson drive         pinned: table vs scipy Poisson CDF, sample moments
  STDP (naive, Fig. 2a) pinned: brute-force all-to-all pairing from spike lists,
                        hand-computed single-pair weight changes
  delivery (Fig. 3a)    pinned: hand-built graph with known sums, conservation
  graph generators      pinned: edge counts vs binomial expectation, no autapses,
                        sortedness, fan-out target uniformity; single rows
                        (fanout_row, bernoulli_row) vs the draw definition
  whole-network rates   parity unpinned (the paper's model definitions and
                        raster data are not available)
"""

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "snn_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

MAX_POISSON = 32


def build(force=True):
    """Compile the oracle with gcc (IEEE fp32/fp64, no FMA contraction)."""
    if not force and os.path.exists(_LIB) and \
            os.path.getmtime(_LIB) >= os.path.getmtime(_SRC):
        return _LIB
    tmp = _LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
           "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


class OracleCfg(ctypes.Structure):
    _fields_ = [
        ("n", ctypes.c_int32), ("n_exc", ctypes.c_int32), ("delay", ctypes.c_int32),
        ("model", ctypes.c_int32), ("plastic", ctypes.c_int32),
        ("poisson_len", ctypes.c_int32),
        ("dt", ctypes.c_double), ("tau_m", ctypes.c_double), ("v_th", ctypes.c_double),
        ("v_reset", ctypes.c_double), ("v_inf", ctypes.c_double),
        ("tau_ref", ctypes.c_double), ("tau_e", ctypes.c_double),
        ("tau_i", ctypes.c_double), ("j_ext", ctypes.c_double),
        ("p_fire", ctypes.c_double), ("tau_plus", ctypes.c_double),
        ("tau_minus", ctypes.c_double), ("lam", ctypes.c_double),
        ("alpha", ctypes.c_double), ("mu", ctypes.c_double), ("w0", ctypes.c_double),
        ("seed", ctypes.c_uint64),
        ("poisson_cdf", ctypes.c_uint32 * MAX_POISSON),
    ]


_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    i32, i64, u64, f32, f64 = (ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64,
                               ctypes.c_float, ctypes.c_double)
    sig = {
        "oracle_splitmix64": (u64, [u64]),
        "oracle_rng": (u64, [u64, ctypes.c_uint32, u64, u64]),
        "oracle_new": (P, [ctypes.POINTER(OracleCfg)]),
        "oracle_free": (None, [P]),
        "oracle_build_random": (i64, [P, i32, f64, f32, f32]),
        "oracle_build_edges": (i32, [P, P, P, P, i64]),
        "oracle_fanout_row": (None, [u64, i32, i32, i32, P]),
        "oracle_bernoulli_row": (i32, [u64, i32, f64, i32, P]),
        "oracle_pivots": (None, [P, i64, i32, i32, P]),
        "oracle_step": (None, [P]),
        "oracle_run": (None, [P, i64]),
        "oracle_time": (i64, [P]),
        "oracle_set_time": (None, [P, i64]),
        "oracle_num_edges": (i64, [P]),
        "oracle_spike_count": (i32, [P]),
        "oracle_spikes_total": (i64, [P]),
        "oracle_set_neurons": (None, [P, P, P, P, P, P]),
        "oracle_get_neurons": (None, [P, P, P, P, P, P]),
        "oracle_set_history_old": (None, [P, P]),
        "oracle_get_history_old": (None, [P, P]),
        "oracle_set_input": (None, [P, P, P]),
        "oracle_get_input": (None, [P, P, P]),
        "oracle_get_spikes": (None, [P, P, P]),
        "oracle_get_graph": (None, [P, P, P, P]),
        "oracle_get_traces": (None, [P, P, P]),
        "oracle_get_weights_at": (None, [P, P, i64, P]),
        "oracle_threads": (i32, []),
        "oracle_set_threads": (None, [i32]),
        "oracle_bernoulli_synapse": (f64, [P, i32, i32, f64, i64]),
        "oracle_bernoulli_input": (None, [P, i32, f64, i64, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def rng_u64(seed, stream, a, b):
    return int(_load().oracle_rng(seed, stream, a, b))


def splitmix64(state):
    return int(_load().oracle_splitmix64(state))


def pivots(row, n, width):
    row = np.ascontiguousarray(row, dtype=np.int32)
    s = (n + width - 1) // width
    out = np.zeros(s + 1, dtype=np.int32)
    _load().oracle_pivots(_ptr(row), len(row), n, width, _ptr(out))
    return out


def fanout_row(seed, n, fanout, k):
    out = np.zeros(fanout, dtype=np.int32)
    _load().oracle_fanout_row(seed, n, fanout, k, _ptr(out))
    return out


def bernoulli_row(seed, n, p, k):
    out = np.zeros(n, dtype=np.int32)
    c = _load().oracle_bernoulli_row(seed, n, p, k, _ptr(out))
    return out[:c].copy()


def threads():
    return int(_load().oracle_threads())


def set_threads(nt):
    _load().oracle_set_threads(int(nt))


def make_cfg(p, poisson_table=None):
    """Fill the oracle's config from a workloads.Preset (physical values)."""
    c = OracleCfg()
    c.n, c.n_exc, c.delay, c.model, c.plastic = p.n, p.n_exc, p.delay, p.model, p.plastic
    c.dt, c.tau_m, c.v_th, c.v_reset, c.v_inf = p.dt, p.tau_m, p.v_th, p.v_reset, p.v_inf
    c.tau_ref, c.tau_e, c.tau_i, c.j_ext, c.p_fire = (p.tau_ref, p.tau_e, p.tau_i,
                                                      p.j_ext, p.p_fire)
    c.tau_plus, c.tau_minus, c.lam, c.alpha, c.mu, c.w0 = (p.tau_plus, p.tau_minus, p.lam,
                                                            p.alpha, p.mu, p.w0)
    c.seed = p.seed
    tab = np.zeros(0, dtype=np.uint32) if poisson_table is None else poisson_table
    if len(tab) > MAX_POISSON:
        raise ValueError("Poisson table too long")
    c.poisson_len = len(tab)
    for q, v in enumerate(tab):
        c.poisson_cdf[q] = int(v)
    return c


class Oracle:
    """One oracle network. Arrays in and out are numpy (host) arrays."""

    def __init__(self, preset, poisson_table=None):
        lib = _load()
        self.p = preset
        self.n = preset.n
        self._cfg = make_cfg(preset, poisson_table)
        self._h = lib.oracle_new(ctypes.byref(self._cfg))
        if not self._h:
            raise MemoryError("oracle_new failed")
        self._lib = lib

    def close(self):
        if self._h:
            self._lib.oracle_free(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # graph -------------------------------------------------------------
    def build_random(self, kind=None, p_or_fanout=None, w_exc=None, w_inh=None):
        p = self.p
        e = self._lib.oracle_build_random(
            self._h, p.graph_kind if kind is None else kind,
            p.p_or_fanout if p_or_fanout is None else p_or_fanout,
            p.w_exc if w_exc is None else w_exc, p.w_inh if w_inh is None else w_inh)
        if e < 0:
            raise MemoryError("oracle graph allocation failed")
        return int(e)

    def build_edges(self, src, dst, w):
        src = np.ascontiguousarray(src, dtype=np.int32)
        dst = np.ascontiguousarray(dst, dtype=np.int32)
        w = np.ascontiguousarray(w, dtype=np.float32)
        if self._lib.oracle_build_edges(self._h, _ptr(src), _ptr(dst), _ptr(w), len(src)):
            raise ValueError("bad edge list")
        return len(src)

    @property
    def n_edges(self):
        return int(self._lib.oracle_num_edges(self._h))

    def graph(self):
        e = self.n_edges
        rp = np.zeros(self.n + 1, dtype=np.int64)
        col = np.zeros(e, dtype=np.int32)
        w = np.zeros(e, dtype=np.float64)
        self._lib.oracle_get_graph(self._h, _ptr(rp), _ptr(col), _ptr(w))
        return rp, col, w

    def weights(self):
        return self.graph()[2]

    def weights_at(self, idx):
        """Weights of the given edge indices (without copying every weight)."""
        idx = np.ascontiguousarray(idx, dtype=np.int64)
        out = np.zeros(len(idx), dtype=np.float64)
        if len(idx):
            if idx.min() < 0 or idx.max() >= self.n_edges:
                raise IndexError("edge index out of range")
            self._lib.oracle_get_weights_at(self._h, _ptr(idx), len(idx), _ptr(out))
        return out

    def traces(self):
        e = self.n_edges
        xp = np.zeros(e, dtype=np.float64)
        xq = np.zeros(e, dtype=np.float64)
        self._lib.oracle_get_traces(self._h, _ptr(xp), _ptr(xq))
        return xp, xq

    # state -------------------------------------------------------------
    @property
    def t(self):
        return int(self._lib.oracle_time(self._h))

    @t.setter
    def t(self, v):
        self._lib.oracle_set_time(self._h, int(v))

    def set_neurons(self, v=None, refractory=None, i_exc=None, i_inh=None, hist=None,
                    hist_old=None):
        conv = lambda a, dt: None if a is None else np.ascontiguousarray(a, dtype=dt)
        arrs = [conv(v, np.float32), conv(refractory, np.int32), conv(i_exc, np.float32),
                conv(i_inh, np.float32), conv(hist, np.uint64)]
        old = conv(hist_old, np.uint64)
        for a in arrs + [old]:
            if a is not None and a.shape != (self.n,):
                raise ValueError("neuron array shape mismatch")
        self._lib.oracle_set_neurons(self._h, *[_ptr(a) for a in arrs])
        if old is not None:
            self._lib.oracle_set_history_old(self._h, _ptr(old))

    def neurons(self):
        n = self.n
        out = {"v": np.zeros(n, np.float32), "refractory": np.zeros(n, np.int32),
               "i_exc": np.zeros(n, np.float32), "i_inh": np.zeros(n, np.float32),
               "hist": np.zeros(n, np.uint64)}
        self._lib.oracle_get_neurons(self._h, _ptr(out["v"]), _ptr(out["refractory"]),
                                     _ptr(out["i_exc"]), _ptr(out["i_inh"]),
                                     _ptr(out["hist"]))
        out["hist_old"] = np.zeros(n, np.uint64)
        self._lib.oracle_get_history_old(self._h, _ptr(out["hist_old"]))
        return out

    def set_input(self, a_exc=None, a_inh=None):
        a = None if a_exc is None else np.ascontiguousarray(a_exc, dtype=np.float32)
        b = None if a_inh is None else np.ascontiguousarray(a_inh, dtype=np.float32)
        self._lib.oracle_set_input(self._h, _ptr(a), _ptr(b))

    def input(self):
        a = np.zeros(self.n, np.float32)
        b = np.zeros(self.n, np.float32)
        self._lib.oracle_get_input(self._h, _ptr(a), _ptr(b))
        return a, b

    def spikes(self):
        nw = (self.n + 63) // 64
        mask = np.zeros(nw, np.uint64)
        cnt = int(self._lib.oracle_spike_count(self._h))
        lst = np.zeros(cnt, np.int32)
        self._lib.oracle_get_spikes(self._h, _ptr(mask), _ptr(lst))
        return mask, lst

    @property
    def spikes_total(self):
        return int(self._lib.oracle_spikes_total(self._h))

    def step(self, n=1):
        if n == 1:
            self._lib.oracle_step(self._h)
        else:
            self._lib.oracle_run(self._h, int(n))

    # Bernoulli-source replays --------------------------------------------
    def bernoulli_synapse(self, k, j, w_init, t_end):
        return float(self._lib.oracle_bernoulli_synapse(self._h, k, j, w_init, t_end))

    def bernoulli_input(self, fanout, w_init, t):
        out = np.zeros(self.n, np.float32)
        self._lib.oracle_bernoulli_input(self._h, int(fanout), float(w_init), int(t),
                                         _ptr(out))
        return out
