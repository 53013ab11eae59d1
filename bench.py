"""Benchmark of the synapse pass on one MI355X.

Workload (default): the stress network - 250,000 Bernoulli(0.005) sources,
fan-out 1,000 uniform-random targets with replacement (250M synapses, int32
targets + fp32 weights), power-law STDP on every synapse, delay 1 step.

One step = neuron update (with the spike and row lists), lazy + event-driven STDP
of the forced rows, and slice (LDS) delivery with the transmitting rows'
STDP. Before the timed region the network runs max(--warmup, 2 x history
length) untimed steps, so that every history window is full and the forced
rows have left their staggered start: the timed steps are steady state
whatever --warmup says. Timed region: K steps issued by one snn_step call,
bracketed by device synchronisation. Then K more steps run with the
library's kernel timing: every kernel launch places HIP events around
itself on the library's stream, which gives per-kernel device times (the
events widen the gaps between kernels, so the timed region runs without
them).

The roofline figure of the dominant kernel (the fused synapse pass, or the
forced-row STDP where the step runs it alone) divides the method's
algorithmic bytes per step by the kernel's device time. Those bytes follow
the survey's per-step count (targets and weights read and changed weights
written per STDP synapse update, row state per triggered row, the gathered
histories and post traces once per neuron, the age scan, 8 B per delivered
event, the pivots of each delivered row, the slice write-back), less the
delivery re-read of the transmitting rows' targets and weights, which a
fused pass reads once. The bytes this implementation moves by design
(fixed-point partials, snapshots, staging) are reported beside it.

Prints one JSON line. `--gpus N` with N > 1 exits: the benchmark runs on one GPU.
"""

import argparse
import hashlib
import re
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
METRIC = "synaptic events/sec (delivery+STDP) on 1 MI355X; % of HBM roofline"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=1000)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--config", default="stress")
    ap.add_argument("--mode", choices=["lds", "global"], default="lds")
    ap.add_argument("--slice-width", type=int, default=None)
    ap.add_argument("--chunks", type=int, default=None)
    ap.add_argument("--stdp-layout", choices=["rows", "slice"], default="rows")
    ap.add_argument("--stdp-filter", choices=["auto", "codes", "bitmap", "none"],
                    default="auto")
    ap.add_argument("--history-bits", type=int, choices=[64, 128], default=None,
                    help="spike history per neuron (default: the preset's)")
    ap.add_argument("--targets", choices=["preset", "32", "16"], default="preset",
                    help="synapse targets: 32-bit, or 16-bit slice-local (compressed)")
    ap.add_argument("--plasticity", choices=["lazy-event", "lazy", "naive"],
                    default="lazy-event",
                    help="plasticity algorithm (Fig. 2(c), (b), (a))")
    ap.add_argument("--stdp-xcd", choices=sorted(XCD_ARG), default="off",
                    help="forced rows partitioned over the XCDs by target range")
    ap.add_argument("--plastic-blocks", default="on",
                    help="plastic networks with D >= 2: on (blocks of up to D-1 steps), off "
                         "(three parts per step) or the most steps per block")
    ap.add_argument("--block-width", type=int, choices=[0, 64, 128, 256], default=0,
                    help="targets per group of the plastic blocks (0: automatic)")
    ap.add_argument("--stdp-mult", type=int, default=0)
    ap.add_argument("--stdp-chunks", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="time budget of the oracle on all its threads")
    ap.add_argument("--cpu-seconds-1t", type=float, default=10.0,
                    help="time budget of the oracle on one thread (0: skip)")
    ap.add_argument("--no-instrumented", action="store_true",
                    help="no per-kernel event timing (plain timed steps)")
    ap.add_argument("--no-row-probe", action="store_true",
                    help="skip the row-stream probe (the forced-row STDP access pattern "
                         "without its arithmetic, at the same row count)")
    ap.add_argument("--write-traffic", nargs=2, metavar=("FETCH_DB", "WRITE_DB"),
                    help="no run: write profiles/traffic.json for --config from two "
                         "rocprofv3 --pmc result databases of a run with --copy-probe-mib "
                         "(FETCH_SIZE, then WRITE_SIZE)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="after the timed region, run one device-to-device copy of this many "
                         "MiB: the reference kernel that scales rocprofv3 FETCH_SIZE/WRITE_SIZE "
                         "readings to bytes")
    return ap.parse_args()


# --stdp-xcd: the config's stdp_xcd (0 off, 1 automatic, else the range count)
XCD_ARG = {"off": 0, "auto": 1, "2": 2, "4": 4, "8": 8}


def block_arg(v):
    """--plastic-blocks: the config's plastic_blocks (0 on, -1 off, k at most k steps)."""
    if v == "on":
        return 0
    if v == "off":
        return -1
    k = int(v)
    if not 1 <= k <= 64:
        raise ValueError("--plastic-blocks: on, off or 1..64")
    return k

_COMMENT = re.compile(r"//[^\n]*|/\*.*?\*/", re.S)


def kernel_source_digest():
    """Digest of the library's code with comments and layout removed, so that
    counters taken on a source stay valid across comment-only edits."""
    h = hashlib.sha256()
    for f in ("k_neuron.hip", "k_synapse.hip", "k_graph.hip", "snn_device.h", "snn_api.hip",
              "snn_internal.h"):
        with open(os.path.join(ROOT, "paper_2107_04092_amd", "csrc", f)) as fh:
            code = _COMMENT.sub(" ", fh.read())
        h.update(" ".join(code.split()).encode())
    return h.hexdigest()[:16]


def write_traffic(fetch_db, write_db, workload_key, copy_mib):
    """HBM bytes per launch of each kernel from two rocprofv3 counter runs
    (FETCH_SIZE, then WRITE_SIZE, in KiB per dispatch), each scaled by what
    the same counter reads for the reference copy of copy_mib MiB each way
    (__amd_rocclr_copyBuffer); averaged over the dispatches after the first
    quarter. Written to profiles/traffic.json under workload_key with the
    current source digest."""
    import sqlite3
    import collections
    vals = collections.defaultdict(lambda: collections.defaultdict(list))
    for db, counter in ((fetch_db, "FETCH_SIZE"), (write_db, "WRITE_SIZE")):
        con = sqlite3.connect(db)
        for name, cn, v in con.execute(
                "select kernel_name, counter_name, value from counters_collection"):
            if cn != counter:
                continue
            k = name.replace("snn::(anonymous namespace)::", "").split("(")[0]
            k = k.replace("void ", "").split("<")[0].strip()
            vals[k][cn].append(float(v))
        con.close()
    ref = vals["__amd_rocclr_copyBuffer"]
    kib = copy_mib * 1024.0
    fs, ws = kib / max(ref["FETCH_SIZE"]), kib / max(ref["WRITE_SIZE"])
    path = os.path.join(ROOT, "profiles", "traffic.json")
    d = json.load(open(path)) if os.path.exists(path) else {}
    out = {}
    for k in ("k_neuron", "k_source_steps", "k_synapse_pass", "k_deliver_lds", "k_stdp_rows"):
        f, w = vals[k]["FETCH_SIZE"], vals[k]["WRITE_SIZE"]
        if not f or not w:
            continue
        f, w = f[len(f) // 4:], w[len(w) // 4:]
        fk, wk = sum(f) / len(f), sum(w) / len(w)
        out[k] = {"fetch_kib": round(fk, 1), "write_kib": round(wk, 1),
                  "fetch_scale": round(fs, 4), "write_scale": round(ws, 4),
                  "bytes_per_launch": round((fk * fs + wk * ws) * 1024),
                  "dispatches": len(f), "source_digest": kernel_source_digest()}
    d[workload_key] = out
    with open(path, "w") as fh:
        json.dump(d, fh, indent=1)
    print(json.dumps({workload_key: out}, indent=1))


def load_traffic(kernel, workload_key):
    """HBM bytes per launch from committed rocprofv3 counter summaries, if they
    were taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        d = json.load(open(path))
        ent = d[workload_key][kernel]
        if ent.get("source_digest") != kernel_source_digest():
            return None
        return float(ent["bytes_per_launch"])
    except (KeyError, ValueError, TypeError):
        return None


def survey_bytes(st, steps, n, n_slices, chunks, nacc, fused):
    """The method's algorithmic bytes per step, counted as the survey's
    measurement section writes them (per-step averages of the counters):
      STDP      12 B per synapse update (target and weight read, weight
                written), 16 B per triggered row (t_last and pre trace read
                and written), 12 B per neuron (the gathered history word and
                post trace, once), 4 B per neuron (the age scan);
      delivery  8 B per delivered event (target and weight), (S+1) x 4 B of
                pivots per delivered row, C x nacc x 4 B per neuron of slice
                write-back;
      fused     less 8 B per synapse update of a transmitting row: a pass that
                makes those rows current inside delivery reads their targets
                and weights once (the survey's fused-pass deduction).
    Delivered rows are the spikes emitted in the same steps (equal to the
    transmitted ones in steady state). Returns a dict of floats."""
    u = st["stdp_synapse_updates"] / steps
    r = st["stdp_rows"] / steps
    ev = st["delivered_events"] / steps
    tx = st["spikes"] / steps
    u_tx = (st["stdp_synapse_updates"] - st["stdp_forced_synapse_updates"]) / steps
    plastic = st["stdp_rows"] > 0
    stdp = (12 * u + 16 * r + 12 * n + 4 * n) if plastic else 0.0
    dlv = 8 * ev + tx * (n_slices + 1) * 4 + chunks * n * 4 * nacc
    deduct = 8 * min(ev, u_tx) if (fused and plastic) else 0.0
    return {"stdp": stdp, "delivery": dlv, "as_written": stdp + dlv,
            "fused_deduction": deduct, "algorithmic": stdp + dlv - deduct}


def stdp_bytes(st, n, launches, hw=1):
    """Bytes the forced-row STDP kernel (snn_update_plasticity) of this
    implementation moves, with hw 64-bit history words per neuron: per
    synapse update 8 B (32-bit target and weight read), per changed weight
    4 B (store), per row 32 + 8 hw B (list entry, row pointer, plastic end,
    source history, t_last and pre trace read and written), per launch
    8 hw B per neuron (the target histories)."""
    return (8 * st["stdp_forced_synapse_updates"] + 4 * st["stdp_forced_weights_written"] +
            (32 + 8 * hw) * st["stdp_forced_rows"] + 8 * hw * n * launches)


def delivery_bytes(st, n, n_slices, chunks, nacc, launches, mode, target_bytes=4, hw=1):
    """Bytes this implementation's delivery with the transmitting rows' STDP
    moves: per event the target (4 B, or 2 B compressed in LDS mode) and the weight
    (4 B), and 4 B per weight STDP changed there. LDS mode
    adds per (transmitted spike, slice) 20 B (row snapshot or list entry,
    pivot pair), per launch 8 hw + 4 B per neuron for the targets' histories
    and post traces (plastic networks) and the slice write-back: nacc * n * 4 B of
    fp32 inputs with one chunk, else C * nacc * n * 8 B of fixed-point
    partial sums. The global mode adds per spike 20 B, per event the 8 B
    atomic update, and per launch the clear of nacc * n * 8 B."""
    ev, tx = st["delivered_events"], st["spikes"]
    wtx = st["stdp_weights_written"] - st["stdp_forced_weights_written"]
    plastic = (8 * hw + 4) * n if st["stdp_rows"] > 0 else 0
    if mode == "lds":
        wb = 4 * nacc * n if chunks == 1 else 8 * chunks * nacc * n
        return ((target_bytes + 4) * ev + 4 * wtx + 20 * tx * n_slices +
                (wb + plastic) * launches)
    return 16 * ev + 20 * tx + 8 * nacc * n * launches


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo) and its logical CPUs."""
    name = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    name = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return name, os.cpu_count()


def cpu_baseline(p, seconds, seconds_1t):
    """The oracle as it stands on this host's cores: naive dense STDP over all
    synapses every step plus row-wise delivery, a prefix of the same workload
    with all of the oracle's OpenMP threads, then one more prefix on one
    thread (each bounded by its time budget)."""
    from oracle import oracle
    import workloads as wl
    o = oracle.Oracle(p, wl.poisson_cdf_table(p.poisson_mu))
    t0 = time.time()
    o.build_random()
    o.set_neurons(**wl.initial_state(p))
    build_s = time.time() - t0
    rp = o.graph()[0]

    def run(budget, max_steps):
        events = steps = 0
        t0 = time.time()
        while True:
            o.step()
            steps += 1
            _, lst = o.spikes()
            events += int((rp[lst + 1] - rp[lst]).sum())
            el = time.time() - t0
            if el >= budget or steps >= max_steps:
                return events, steps, el

    threads = oracle.threads()
    ev, steps, el = run(seconds, 200)
    one = None
    if seconds_1t > 0:
        oracle.set_threads(1)
        try:
            ev1, steps1, el1 = run(seconds_1t, 200)
        finally:
            oracle.set_threads(threads)
        one = {"value": ev1 / el1, "unit": "synaptic events/s", "cores": 1,
               "steps": steps1, "s_per_step": round(el1 / steps1, 4)}
    model, ncpu = cpu_model()
    return {"value": ev / el, "unit": "synaptic events/s", "cores": threads,
            "kind": "oracle",
            "sample": "%s workload at full size (n=%d, %d synapses), steps 1-%d after a "
                      "%.1f s build, %d OpenMP threads; dense per-synapse STDP every step + "
                      "row-wise delivery; %.3f s/step"
                      % (p.name, p.n, o.n_edges, steps, build_s, threads, el / steps),
            "single_thread": one,
            "cpu_model": model, "host_logical_cpus": ncpu}


def check_device_errors(net, where):
    """Ends the benchmark if a kernel flagged an error condition (a row
    behind its history window, a ring inconsistency): its numbers would be
    those of a wrong simulation."""
    err = net.stats()["device_errors"]
    if err:
        print("bench.py: device error flags 0x%x after the %s; no result" % (err, where),
              file=sys.stderr)
        sys.exit(1)


def main():
    args = parse()
    if args.write_traffic:
        if args.copy_probe_mib <= 0:
            sys.exit("bench.py: --write-traffic needs the --copy-probe-mib of the profiled run")
        write_traffic(args.write_traffic[0], args.write_traffic[1], args.config,
                      args.copy_probe_mib)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: the synapse pass is benchmarked on one GPU only; "
              "--gpus %d is not supported" % args.gpus, file=sys.stderr)
        sys.exit(2)
    import torch
    import workloads as wl
    from workloads.presets import PLASTIC_EXC_EXC
    from paper_2107_04092_amd import snn

    p = wl.preset(args.config)
    hbits = args.history_bits or p.history_bits
    width = args.slice_width or p.slice_width
    chunks = args.chunks or p.spike_chunks
    mode = snn.SNN_DELIVER_LDS_SLICE if args.mode == "lds" else snn.SNN_DELIVER_GLOBAL_ATOMIC
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream(dev)

    cfg = snn.config_from_preset(p, wl.poisson_cdf_table(p.poisson_mu),
                                 slice_width=width, spike_chunks=chunks,
                                 stdp_slice_mult=args.stdp_mult, stdp_chunks=args.stdp_chunks,
                                 stdp_layout=0 if args.stdp_layout == "rows" else 1,
                                 stdp_filter=["auto", "codes", "bitmap", "none"].index(
                                     args.stdp_filter),
                                 history_bits=hbits,
                                 plasticity_algorithm=["lazy-event", "lazy", "naive"].index(
                                     args.plasticity),
                                 compressed_targets=(None if args.targets == "preset" else
                                                     int(args.targets == "16")),
                                 stdp_xcd=XCD_ARG[args.stdp_xcd],
                                 plastic_blocks=block_arg(args.plastic_blocks),
                                 plastic_block_width=args.block_width)
    t0 = time.time()
    net = snn.Network(cfg, stream=stream, device=dev)
    e = net.build_random(p.graph_kind, p.p_or_fanout, p.w_exc, p.w_inh)
    st0 = wl.initial_state(p)
    net.set_state(0, v=torch.from_numpy(st0["v"]))
    torch.cuda.synchronize()
    setup_s = time.time() - t0

    # untimed steps: the requested warm-up, and at least two history lengths,
    # so that every window is full and the forced rows are past their
    # staggered start (steady state)
    untimed = max(args.warmup, 2 * hbits)
    net.step(untimed, mode)
    torch.cuda.synchronize()
    check_device_errors(net, "untimed steps")
    net.reset_stats()

    # timed region: exactly K steps
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record(stream)
    t_wall = time.perf_counter()
    net.step(args.steps, mode)
    end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_wall
    ms_total = start.elapsed_time(end)
    st = net.stats()
    check_device_errors(net, "timed steps")
    ms_per_step = ms_total / args.steps
    events_per_s = st["delivered_events"] / (ms_total * 1e-3)
    stdp_per_s = st["stdp_synapse_updates"] / (ms_total * 1e-3)

    n_slices = (p.n + width - 1) // width
    nacc = 2 if p.model == snn.SNN_LIF_CUBA else 1
    # 16-bit targets are read by slice delivery only; row-wise STDP reads 32-bit
    tb = 2 if cfg.compressed_targets and args.mode == "lds" else 4
    b_stdp = stdp_bytes(st, p.n, args.steps, hbits // 64) / args.steps
    b_dlv = delivery_bytes(st, p.n, n_slices, chunks, nacc, args.steps, args.mode,
                           tb, hbits // 64) / args.steps

    kernels = None
    roofline = None
    combined = None
    if not args.no_instrumented:
        # per-kernel device times: K more steps in which every kernel launch
        # places HIP events around itself on the library's stream (events in
        # the launches widen the gaps between kernels, not the kernels, so
        # the timed region above runs without them)
        net.reset_stats()
        net.record_kernel_times(args.steps)
        net.step(args.steps, mode)
        kt, nrec = net.kernel_times()
        net.record_kernel_times(0)
        st2 = net.stats()
        b_stdp = stdp_bytes(st2, p.n, args.steps, hbits // 64) / args.steps
        b_dlv = delivery_bytes(st2, p.n, n_slices, chunks, nacc, args.steps,
                               args.mode, tb, hbits // 64) / args.steps
        t_neu, t_stdp, t_dlv = kt["neuron"], kt["plasticity"], kt["delivery"]
        # a plastic network of Bernoulli sources with D = 1 runs its neuron
        # updates in source blocks: one launch per block of steps
        nsteps = (net.graph()["block_steps"] or 1) if (
            p.model == snn.SNN_BERNOULLI_SOURCE and p.delay == 1 and p.plastic != 0
            and args.mode == "lds") else 1
        kernels = {
            "steps_timed": nrec,
            "neuron_us": round(t_neu * 1e3, 3),
            "neuron_steps_per_launch": nsteps,
            "neuron_us_per_step": round(t_neu * 1e3 / nsteps, 3),
            "plasticity_us": round(t_stdp * 1e3, 3),
            "delivery_us": round(t_dlv * 1e3, 3),
            "fused_synapse_pass": bool(p.plastic != 0 and t_stdp == 0 and t_dlv > 0),
            "plasticity_bytes_per_launch": int(b_stdp),
            "delivery_bytes_per_launch": int(b_dlv),
            "delivery_GBs": (round(b_dlv / (t_dlv * 1e-3) / 1e9, 1)
                             if t_dlv and not (p.plastic != 0 and t_stdp == 0) else None),
        }
        if args.plasticity == "naive":
            kname = "k_stdp_naive"
        elif args.stdp_layout == "rows":
            kname = "k_stdp_rows"
        else:
            kname = "k_stdp"
        # a plastic network whose step ran plasticity and delivery in one
        # launch (the fused synapse pass) records it as the delivery part
        fused = p.plastic != 0 and t_stdp == 0 and t_dlv > 0 and b_stdp > 0
        sb = survey_bytes(st2, args.steps, p.n, n_slices, chunks, nacc,
                          fused or (args.mode == "lds" and p.plastic != 0))
        if fused:
            kname = "k_synapse_pass"
            t_k = t_dlv
            alg = sb["algorithmic"]
            written = sb["as_written"]
            impl = b_stdp + b_dlv
        elif t_stdp > 0:
            # the forced rows' share of the STDP count, the kernel's own
            # (delivery makes the transmitting rows current)
            f = st2["stdp_forced_synapse_updates"] / args.steps
            rf = st2["stdp_forced_rows"] / args.steps
            t_k = t_stdp
            alg = written = 12 * f + 16 * rf + 16 * p.n
            impl = b_stdp
        if fused or t_stdp > 0:
            ach = alg / (t_k * 1e-3) / 1e9
            traffic = load_traffic(kname, p.name)
            roofline = {"bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS,
                        "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4),
                        "traffic": traffic, "kernel": kname,
                        "kernel_us": round(t_k * 1e3, 3),
                        "bytes_per_launch": int(alg),
                        "bytes_as_written": int(written),
                        "frac_as_written": round(written / (t_k * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                        "implementation_bytes_per_launch": int(impl),
                        "traffic_over_algorithmic": (round(traffic / alg, 3)
                                                     if traffic else None)}
            comb = sb["algorithmic"] / ((t_stdp + t_dlv) * 1e-3) / 1e9
            combined = {"achieved_GBs": round(comb, 1), "frac": round(comb / HBM_PEAK_GBS, 4),
                        "us_per_step": round((t_stdp + t_dlv) * 1e3, 3),
                        "survey_bytes_per_step": {k: int(v) for k, v in sb.items()}}

    ceiling = None
    if roofline is not None and kname in ("k_stdp_rows", "k_synapse_pass") and \
            not args.no_row_probe:
        # the forced-row access pattern without its arithmetic, at the same
        # row count: targets and weights streamed (8 B per synapse), then
        # also every weight stored back (12 B per synapse); median of 5
        rows = max(1, int(round(st2["stdp_forced_rows"] / max(nrec, 1))))

        def probe(r):
            meas = {}
            for write in (False, True):
                runs = sorted(net.probe_rows(r, write=write, seed=q + 1) for q in range(5))
                ms, syn = runs[2]
                bps = 12 if write else 8
                meas[write] = (syn * bps / (ms * 1e-3) / 1e9, ms)
            return meas

        meas = probe(rows)
        ceiling = {"kernel": "k_probe_rows", "rows": rows,
                   "read_GBs": round(meas[False][0], 1),
                   "read_frac": round(meas[False][0] / HBM_PEAK_GBS, 4),
                   "read_us": round(meas[False][1] * 1e3, 2),
                   "read_write_GBs": round(meas[True][0], 1),
                   "read_write_frac": round(meas[True][0] / HBM_PEAK_GBS, 4),
                   "read_write_us": round(meas[True][1] * 1e3, 2)}
        # the same pattern at 2, 4, 8 and 16 times the rows (within the
        # plastic rows): how far launch size alone moves the fraction
        sweep = []
        for mult in (2, 4, 8, 16):
            r = min(rows * mult, p.n_exc if p.plastic == PLASTIC_EXC_EXC else p.n)
            m = probe(r)
            sweep.append({"rows": r, "read_frac": round(m[False][0] / HBM_PEAK_GBS, 4),
                          "read_write_frac": round(m[True][0] / HBM_PEAK_GBS, 4),
                          "read_write_us": round(m[True][1] * 1e3, 2)})
        ceiling["sweep"] = sweep

    if args.copy_probe_mib > 0:
        nbytes = args.copy_probe_mib << 20
        src = torch.empty(nbytes, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(p, args.cpu_seconds, args.cpu_seconds_1t)

    out = {
        "metric": METRIC,
        "value": events_per_s,
        "unit": "synaptic events/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "untimed_steps": untimed,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": "%s: n=%d, %s %s, %d synapses, delay %d, plasticity %s, "
                        "delivery %s, slice width %d, chunks %d"
                        % (p.name, p.n,
                           "fan-out" if p.graph_kind == 1 else "p",
                           p.p_or_fanout, e, p.delay,
                           ["none", "exc-exc", "all"][p.plastic], args.mode, width, chunks),
            "n": p.n, "synapses": e, "slice_width": width, "spike_chunks": chunks,
            "delivery": args.mode, "stdp_layout": args.stdp_layout,
            "stdp_filter": args.stdp_filter, "history_bits": hbits,
            "target_bits": 16 if cfg.compressed_targets else 32,
            "plasticity": args.plasticity,
            "stdp_slice_mult": args.stdp_mult, "stdp_chunks": args.stdp_chunks,
            "stdp_xcd": args.stdp_xcd, "seed": p.seed,
            "plastic_blocks": net.graph()["block_steps"],
            "block_width": net.graph()["block_width"],
        },
        "roofline": roofline,
        "cpu_baseline": cpu,
        "stdp_synapse_updates_per_s": stdp_per_s,
        "delivery_plus_stdp": combined,
        "row_stream_ceiling": ceiling,
        "kernels": kernels,
        "stats": {k: int(v) for k, v in st.items()},
        "implementation_bytes_per_step": {"stdp": int(b_stdp), "delivery": int(b_dlv)},
        "setup_s": round(setup_s, 3),
        "host_wall_s": round(wall, 4),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
