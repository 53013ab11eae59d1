"""ctypes binding of libsnn.so (include/snn.h), argument marshalling only.

Each `snn_*` function here has the name and meaning of the C function of the
same name. Every step of the simulation runs in the library's HIP kernels;
PyTorch only provides device memory (uint8 workspace tensors) and the HIP
stream. There is no fallback: importing this module without the built
library raises.

`Network` bundles the calls for one network: it allocates the workspace and
graph buffers as torch tensors and returns zero-copy torch views of the
device state.
"""

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libsnn.so")

SNN_OK, SNN_EINVAL, SNN_ENOMEM, SNN_EDEVICE, SNN_ESTATE = range(5)
SNN_LIF_DELTA, SNN_LIF_CUBA, SNN_BERNOULLI_SOURCE = range(3)
SNN_PLASTIC_NONE, SNN_PLASTIC_EXC_EXC, SNN_PLASTIC_ALL = range(3)
SNN_DELIVER_LDS_SLICE, SNN_DELIVER_GLOBAL_ATOMIC = range(2)
SNN_GRAPH_BERNOULLI, SNN_GRAPH_FIXED_FANOUT = range(2)
SNN_MAX_POISSON = 32

_i32, _i64, _u32, _u64, _f32, _f64 = (ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32,
                                      ctypes.c_uint64, ctypes.c_float, ctypes.c_double)
_P = ctypes.c_void_p


class snn_config(ctypes.Structure):
    _fields_ = [
        ("n", _i32), ("n_exc", _i32), ("delay_steps", _i32), ("slice_width", _i32),
        ("spike_chunks", _i32), ("stdp_slice_mult", _i32), ("stdp_chunks", _i32),
        ("stdp_layout", _i32), ("stdp_filter", _i32), ("history_bits", _i32),
        ("plasticity_algorithm", _i32), ("compressed_targets", _i32), ("stdp_xcd", _i32),
        ("plastic_blocks", _i32), ("plastic_block_width", _i32), ("neuron_model", _i32),
        ("plastic", _i32), ("poisson_len", _i32),
        ("dt_ms", _f64), ("tau_m_ms", _f64), ("v_th", _f64), ("v_reset", _f64),
        ("v_inf", _f64), ("tau_ref_ms", _f64), ("tau_e_ms", _f64), ("tau_i_ms", _f64),
        ("j_ext", _f64), ("p_fire", _f64), ("tau_plus_ms", _f64), ("tau_minus_ms", _f64),
        ("lambda_", _f64), ("alpha", _f64), ("mu", _f64), ("w0", _f64),
        ("seed", _u64), ("poisson_cdf", _u32 * SNN_MAX_POISSON),
    ]


class snn_state_view(ctypes.Structure):
    _fields_ = [("t", _i64)] + [(name, _P) for name in (
        "v", "refractory", "i_exc", "i_inh", "hist", "trace_post", "t_last", "trace_pre",
        "input_exc", "input_inh", "spike_mask", "spike_list", "spike_count", "tx_list",
        "tx_count", "stdp_rows", "stdp_row_count", "ring_lists", "ring_counts")]


class snn_graph_view(ctypes.Structure):
    _fields_ = [("n_edges", _i64), ("n_slices", _i32), ("row_ptr", _P),
                ("col", _P), ("w", _P), ("pivots", _P), ("plastic_end", _P), ("col16", _P),
                ("stdp_ranges", _i32), ("block_steps", _i32), ("block_width", _i32),
                ("block_pivots", _P)]


class snn_stats(ctypes.Structure):
    _fields_ = [(name, _i64) for name in (
        "steps", "spikes", "delivered_events", "stdp_rows", "stdp_forced_rows",
        "stdp_synapse_updates", "stdp_weights_written", "stdp_forced_synapse_updates",
        "stdp_forced_weights_written", "device_errors")]


_SIGNATURES = {
    "snn_status_string": (ctypes.c_char_p, [_i32]),
    "snn_create": (_i32, [ctypes.POINTER(snn_config), _P, ctypes.POINTER(_P)]),
    "snn_destroy": (None, [_P]),
    "snn_record_kernel_times": (_i32, [_P, _i32]),
    "snn_get_kernel_times": (_i32, [_P, ctypes.POINTER(ctypes.c_double),
                                    ctypes.POINTER(_i32)]),
    "snn_last_error": (ctypes.c_char_p, [_P]),
    "snn_workspace_size": (_i32, [_P, ctypes.POINTER(ctypes.c_size_t)]),
    "snn_bind_workspace": (_i32, [_P, _P, ctypes.c_size_t]),
    "snn_graph_count_random": (_i32, [_P, _i32, _f64, ctypes.POINTER(_i64)]),
    "snn_graph_size": (_i32, [_P, _i64, ctypes.POINTER(ctypes.c_size_t)]),
    "snn_bind_graph": (_i32, [_P, _P, ctypes.c_size_t, _i64]),
    "snn_build_graph_random": (_i32, [_P, _f32, _f32]),
    "snn_build_graph_edges": (_i32, [_P, _P, _P, _P]),
    "snn_update_neurons": (_i32, [_P]),
    "snn_update_plasticity": (_i32, [_P]),
    "snn_deliver_spikes": (_i32, [_P, _i32]),
    "snn_advance": (_i32, [_P]),
    "snn_step": (_i32, [_P, _i32, _i32]),
    "snn_step_static": (_i32, [_P, _i32, _i32]),
    "snn_flush_plasticity": (_i32, [_P]),
    "snn_probe_rows": (_i32, [_P, _i32, _i32, ctypes.c_uint64, ctypes.POINTER(ctypes.c_double),
                              ctypes.POINTER(_i64)]),
    "snn_get_state": (_i32, [_P, ctypes.POINTER(snn_state_view)]),
    "snn_set_state": (_i32, [_P, ctypes.POINTER(snn_state_view)]),
    "snn_get_graph": (_i32, [_P, ctypes.POINTER(snn_graph_view)]),
    "snn_get_stats": (_i32, [_P, ctypes.POINTER(snn_stats)]),
    "snn_reset_stats": (_i32, [_P]),
    "snn_graph_capture": (_i32, [_P, _i32, _i32, ctypes.POINTER(_P)]),
    "snn_graph_launch": (_i32, [_P, _P]),
    "snn_graph_destroy": (None, [_P]),
}

_lib = None


def load():
    """Loads libsnn.so from the package directory; raises if it is missing."""
    global _lib
    if _lib is None:
        # torch's HIP runtime first: the library then binds to the same
        # runtime (same soname) instead of loading a second one
        import torch  # noqa: F401
        if not os.path.exists(LIB_PATH):
            raise ImportError(
                "libsnn.so is not built (run python -m paper_2107_04092_amd.build); "
                "there is no fallback implementation")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


class SnnError(RuntimeError):
    def __init__(self, status, message):
        super().__init__("%s (status %d): %s" % (
            load().snn_status_string(status).decode(), status, message))
        self.status = status


def _check(ctx, status):
    if status != SNN_OK:
        msg = load().snn_last_error(ctx).decode() if ctx else ""
        raise SnnError(status, msg)


# ---- same-name wrappers of the C functions ---------------------------------

def snn_create(cfg, stream_handle):
    ctx = _P()
    st = load().snn_create(ctypes.byref(cfg), _P(stream_handle), ctypes.byref(ctx))
    if st != SNN_OK:
        msg = load().snn_last_error(ctx).decode() if ctx.value else ""
        if ctx.value:
            load().snn_destroy(ctx)
        raise SnnError(st, msg)
    return ctx


def snn_destroy(ctx):
    load().snn_destroy(ctx)


def snn_workspace_size(ctx):
    b = ctypes.c_size_t()
    _check(ctx, load().snn_workspace_size(ctx, ctypes.byref(b)))
    return b.value


def snn_bind_workspace(ctx, ptr, nbytes):
    _check(ctx, load().snn_bind_workspace(ctx, _P(ptr), nbytes))


def snn_graph_count_random(ctx, kind, p_or_fanout):
    e = _i64()
    _check(ctx, load().snn_graph_count_random(ctx, kind, float(p_or_fanout), ctypes.byref(e)))
    return e.value


def snn_graph_size(ctx, n_edges):
    b = ctypes.c_size_t()
    _check(ctx, load().snn_graph_size(ctx, n_edges, ctypes.byref(b)))
    return b.value


def snn_bind_graph(ctx, ptr, nbytes, n_edges):
    _check(ctx, load().snn_bind_graph(ctx, _P(ptr), nbytes, n_edges))


def snn_build_graph_random(ctx, w_exc, w_inh):
    _check(ctx, load().snn_build_graph_random(ctx, w_exc, w_inh))


def snn_build_graph_edges(ctx, src_ptr, dst_ptr, w_ptr):
    _check(ctx, load().snn_build_graph_edges(ctx, _P(src_ptr), _P(dst_ptr), _P(w_ptr)))


def snn_update_neurons(ctx):
    _check(ctx, load().snn_update_neurons(ctx))


def snn_update_plasticity(ctx):
    _check(ctx, load().snn_update_plasticity(ctx))


def snn_deliver_spikes(ctx, mode):
    _check(ctx, load().snn_deliver_spikes(ctx, mode))


def snn_advance(ctx):
    _check(ctx, load().snn_advance(ctx))


def snn_step(ctx, n_steps, mode):
    _check(ctx, load().snn_step(ctx, n_steps, mode))


def snn_step_static(ctx, n_steps, mode):
    _check(ctx, load().snn_step_static(ctx, n_steps, mode))


def snn_flush_plasticity(ctx):
    _check(ctx, load().snn_flush_plasticity(ctx))


def snn_probe_rows(ctx, n_rows, write, seed):
    """Device milliseconds and synapses of one row-stream probe launch."""
    ms = ctypes.c_double()
    syn = _i64()
    _check(ctx, load().snn_probe_rows(ctx, n_rows, write, seed, ctypes.byref(ms),
                                      ctypes.byref(syn)))
    return ms.value, syn.value


def snn_get_state(ctx):
    v = snn_state_view()
    _check(ctx, load().snn_get_state(ctx, ctypes.byref(v)))
    return v


def snn_set_state(ctx, view):
    _check(ctx, load().snn_set_state(ctx, ctypes.byref(view)))


def snn_get_graph(ctx):
    v = snn_graph_view()
    _check(ctx, load().snn_get_graph(ctx, ctypes.byref(v)))
    return v


def snn_get_stats(ctx):
    s = snn_stats()
    _check(ctx, load().snn_get_stats(ctx, ctypes.byref(s)))
    return s


def snn_reset_stats(ctx):
    _check(ctx, load().snn_reset_stats(ctx))


def snn_graph_capture(ctx, n_steps, mode):
    g = _P()
    _check(ctx, load().snn_graph_capture(ctx, n_steps, mode, ctypes.byref(g)))
    return g


def snn_graph_launch(ctx, graph):
    _check(ctx, load().snn_graph_launch(ctx, graph))


def snn_graph_destroy(graph):
    load().snn_graph_destroy(graph)


def snn_record_kernel_times(ctx, max_steps):
    _check(ctx, load().snn_record_kernel_times(ctx, int(max_steps)))


KERNEL_PARTS = ("neuron", "plasticity", "delivery")


def snn_get_kernel_times(ctx):
    """Mean device milliseconds per step of each part, and the steps recorded."""
    ms = (ctypes.c_double * len(KERNEL_PARTS))()
    steps = _i32()
    _check(ctx, load().snn_get_kernel_times(ctx, ms, ctypes.byref(steps)))
    return dict(zip(KERNEL_PARTS, list(ms))), steps.value


# ---- configuration marshalling ---------------------------------------------

def config_from_preset(p, poisson_table=(), slice_width=None, spike_chunks=None,
                       stdp_slice_mult=0, stdp_chunks=0, stdp_layout=0, stdp_filter=0,
                       history_bits=64, plasticity_algorithm=0, compressed_targets=None,
                       stdp_xcd=0, plastic_blocks=0, plastic_block_width=0):
    """snn_config from a preset-like object with the physical parameters."""
    c = snn_config()
    c.n, c.n_exc, c.delay_steps = p.n, p.n_exc, p.delay
    c.slice_width = p.slice_width if slice_width is None else slice_width
    c.spike_chunks = p.spike_chunks if spike_chunks is None else spike_chunks
    c.stdp_slice_mult, c.stdp_chunks = stdp_slice_mult, stdp_chunks
    c.stdp_layout = stdp_layout
    c.stdp_filter = stdp_filter
    c.history_bits = history_bits
    c.plasticity_algorithm = plasticity_algorithm
    c.compressed_targets = (getattr(p, "compressed_targets", 0) if compressed_targets is None
                            else compressed_targets)
    c.stdp_xcd = stdp_xcd
    c.plastic_blocks, c.plastic_block_width = plastic_blocks, plastic_block_width
    c.neuron_model, c.plastic = p.model, p.plastic
    c.dt_ms, c.tau_m_ms, c.v_th, c.v_reset, c.v_inf = p.dt, p.tau_m, p.v_th, p.v_reset, p.v_inf
    c.tau_ref_ms, c.tau_e_ms, c.tau_i_ms = p.tau_ref, p.tau_e, p.tau_i
    c.j_ext, c.p_fire = p.j_ext, p.p_fire
    c.tau_plus_ms, c.tau_minus_ms = p.tau_plus, p.tau_minus
    c.lambda_, c.alpha, c.mu, c.w0 = p.lam, p.alpha, p.mu, p.w0
    c.seed = p.seed
    tab = list(poisson_table)
    if len(tab) > SNN_MAX_POISSON:
        raise ValueError("Poisson table longer than %d" % SNN_MAX_POISSON)
    c.poisson_len = len(tab)
    for q, v in enumerate(tab):
        c.poisson_cdf[q] = int(v)
    return c


# ---- one network over torch-owned device memory ------------------------------

class Network:
    """A network on the current HIP device, bound to one torch stream."""

    def __init__(self, cfg, stream=None, device=None):
        import torch
        self._torch = torch
        self.device = torch.device("cuda", torch.cuda.current_device()) if device is None \
            else torch.device(device)
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        self.cfg = cfg
        self.n = cfg.n
        self.history_words = 2 if cfg.history_bits == 128 else 1
        self.ctx = snn_create(cfg, self.stream.cuda_stream)
        nbytes = snn_workspace_size(self.ctx)
        with torch.cuda.stream(self.stream):
            self.ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.device)
        self._ws_off = (-self.ws.data_ptr()) % 256
        snn_bind_workspace(self.ctx, self.ws.data_ptr() + self._ws_off, nbytes)
        self.g = None
        self.n_edges = None

    def close(self):
        if getattr(self, "ctx", None):
            snn_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # graph ---------------------------------------------------------------
    def _bind_graph(self, n_edges):
        torch = self._torch
        nbytes = snn_graph_size(self.ctx, n_edges)
        with torch.cuda.stream(self.stream):
            self.g = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.device)
        self._g_off = (-self.g.data_ptr()) % 256
        snn_bind_graph(self.ctx, self.g.data_ptr() + self._g_off, nbytes, n_edges)
        self.n_edges = n_edges

    def build_random(self, kind, p_or_fanout, w_exc, w_inh):
        e = snn_graph_count_random(self.ctx, kind, p_or_fanout)
        self._bind_graph(e)
        snn_build_graph_random(self.ctx, w_exc, w_inh)
        return e

    def build_edges(self, src, dst, w):
        torch = self._torch
        src = torch.as_tensor(src, dtype=torch.int32).to(self.device).contiguous()
        dst = torch.as_tensor(dst, dtype=torch.int32).to(self.device).contiguous()
        w = torch.as_tensor(w, dtype=torch.float32).to(self.device).contiguous()
        if not (src.numel() == dst.numel() == w.numel()):
            raise ValueError("edge arrays differ in length")
        self._bind_graph(src.numel())
        self.stream.wait_stream(torch.cuda.current_stream(self.device))
        snn_build_graph_edges(self.ctx, src.data_ptr(), dst.data_ptr(), w.data_ptr())
        return src.numel()

    # stepping ------------------------------------------------------------
    def step(self, n=1, mode=SNN_DELIVER_LDS_SLICE):
        snn_step(self.ctx, n, mode)

    def step_static(self, n=1, mode=SNN_DELIVER_LDS_SLICE):
        snn_step_static(self.ctx, n, mode)

    def update_neurons(self):
        snn_update_neurons(self.ctx)

    def update_plasticity(self):
        snn_update_plasticity(self.ctx)

    def deliver_spikes(self, mode=SNN_DELIVER_LDS_SLICE):
        snn_deliver_spikes(self.ctx, mode)

    def advance(self):
        snn_advance(self.ctx)

    def flush_plasticity(self):
        snn_flush_plasticity(self.ctx)

    def capture(self, n_steps=1, mode=SNN_DELIVER_LDS_SLICE):
        """A captured sequence of n_steps steps (replay with replay())."""
        return snn_graph_capture(self.ctx, n_steps, mode)

    def replay(self, graph):
        snn_graph_launch(self.ctx, graph)

    def probe_rows(self, n_rows, write=False, seed=1):
        return snn_probe_rows(self.ctx, n_rows, 1 if write else 0, seed)

    def stats(self):
        s = snn_get_stats(self.ctx)
        return {name: getattr(s, name) for name, _ in snn_stats._fields_}

    def reset_stats(self):
        snn_reset_stats(self.ctx)

    def record_kernel_times(self, max_steps):
        snn_record_kernel_times(self.ctx, max_steps)

    def kernel_times(self):
        return snn_get_kernel_times(self.ctx)

    def synchronize(self):
        self.stream.synchronize()

    # views ---------------------------------------------------------------
    def _view(self, buf, ptr, count, dtype):
        torch = self._torch
        if not ptr or count == 0:
            return torch.empty(0, dtype=dtype, device=self.device)
        off = ptr - buf.data_ptr()
        nbytes = count * torch.empty(0, dtype=dtype).element_size()
        if off < 0 or off + nbytes > buf.numel():
            raise RuntimeError("view outside its buffer")
        return buf[off:off + nbytes].view(dtype)

    def state(self):
        """Zero-copy torch views of the device state (see snn_state_view)."""
        torch = self._torch
        v = snn_get_state(self.ctx)
        n, nw, d = self.n, (self.n + 63) // 64, self.cfg.delay_steps
        ws = self.ws
        out = {"t": v.t}
        for name, dt, cnt in (("v", torch.float32, n), ("refractory", torch.int32, n),
                              ("i_exc", torch.float32, n), ("i_inh", torch.float32, n),
                              ("hist", torch.int64, n * self.history_words),
                              ("trace_post", torch.float32, n),
                              ("t_last", torch.int32, n), ("trace_pre", torch.float32, n),
                              ("input_exc", torch.float32, n), ("input_inh", torch.float32, n),
                              ("spike_mask", torch.int64, nw), ("spike_list", torch.int32, n),
                              ("spike_count", torch.int32, 1), ("tx_list", torch.int32, n),
                              ("tx_count", torch.int32, 1), ("stdp_rows", torch.int32, n),
                              ("stdp_row_count", torch.int32, 1),
                              ("ring_lists", torch.int32, d * n),
                              ("ring_counts", torch.int32, d)):
            out[name] = self._view(ws, getattr(v, name), cnt, dt)
        return out

    def set_state(self, t, **arrays):
        """Copies the given device tensors (names of snn_state_view) into the state."""
        torch = self._torch
        view = snn_state_view()
        view.t = int(t)
        keep = []
        for name, arr in arrays.items():
            if arr is None:
                continue
            if not isinstance(arr, torch.Tensor):
                raise TypeError("%s must be a torch tensor" % name)
            arr = arr.to(self.device).contiguous()
            keep.append(arr)
            setattr(view, name, arr.data_ptr())
        self.stream.wait_stream(torch.cuda.current_stream(self.device))
        snn_set_state(self.ctx, view)
        # the copies are enqueued on self.stream: keep sources alive until done
        self.stream.synchronize()
        del keep

    def graph(self):
        torch = self._torch
        v = snn_get_graph(self.ctx)
        n, s, e = self.n, v.n_slices, v.n_edges
        return {
            "n_edges": e, "n_slices": s,
            "row_ptr": self._view(self.ws, v.row_ptr, n + 1, torch.int64),
            "col": self._view(self.g, v.col, e, torch.int32),
            "w": self._view(self.g, v.w, e, torch.float32),
            "pivots": self._view(self.g, v.pivots, n * (s + 1), torch.int32).view(n, s + 1),
            "plastic_end": self._view(self.ws, v.plastic_end, n, torch.int32),
            "col16": (self._view(self.g, v.col16, e, torch.int16) if v.col16 else None),
            "stdp_ranges": v.stdp_ranges,
            "block_steps": v.block_steps, "block_width": v.block_width,
            "block_pivots": (self._view(self.g, v.block_pivots,
                                        n * ((n + v.block_width - 1) // v.block_width + 1),
                                        torch.int32) if v.block_pivots else None),
        }
