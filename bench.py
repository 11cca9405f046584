"""Throughput of the credit-assignment hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu]
    python bench.py --extra                      # every workload, table on stderr
    python bench.py --probe-sweep                # streaming probe launch shapes beside the GAE step

Workload: GAE over a 4096 x 256 float32 rollout buffer with termination and truncation flags,
truncation continuations and per-row bootstraps (seeded synthetic data). One step is one call
of rlcs_gae: load, coefficient build, scan, carry, epilogue and store of advantages and returns,
all inside one kernel launch.

Cold HBM: the timed steps rotate over enough independent input/output sets (well beyond the
256 MB Infinity Cache) that every step reads its inputs from HBM.

Prints one JSON line on stdout:
  value      effective bandwidth = algorithmic bytes / (timed time / K), GB/s
  roofline   the same figure against the 8 TB/s HBM peak
  copy_reference  a streaming kernel moving the same 22 B per step over the same sets, timed
                the same way (the ceiling at this size), and the empty-launch floor
  cpu_baseline  the fp64 oracle on the host, rows split over the host's cores (the single-thread
                rate in its `sample`), each timed for about --cpu-seconds
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import sqlite3
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
N, T = 4096, 256
GAMMA, LAM = 0.99, 0.95
METRIC = "effective HBM GB/s (% of MI355X peak) + Gsteps/s, GAE 4096×256 fp32"


def algorithmic_bytes(N, T, *, dtype_bytes=4, trunc=True, boot=True, outputs=2):
    """Each input read once and each output written once, dense: r, v (data), term (1 B),
    trunc (1 B) and bv (data) when truncation is on, boot [N], advantages and returns (4 B)."""
    per = 2 * dtype_bytes + 1 + (1 + dtype_bytes if trunc else 0) + 4 * outputs
    return N * T * per + (N * dtype_bytes if boot else 0)


def eager_steps(warmup, steps, sets):
    """Eager calls before the timed steps: at least `warmup`, and enough that every set the
    timed steps touch (set i % sets for i < steps) has been written by an eager call."""
    return max(warmup, min(steps, sets))


def replay_check_set(steps, sets):
    """The set whose advantages the timed steps are compared with: the last one they write."""
    return (steps - 1) % sets


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--sets", type=int, default=32, help="rotated input/output sets (cold HBM)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-context", action="store_true",
                    help="skip the full-call timing and the warm figure, which launch the GAE kernel "
                         "outside the cold timed path: for kernel-trace runs (the copy reference, "
                         "whose probe kernels are told apart by name, still runs)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--extra", action="store_true",
                    help="time every estimator of every workload (table on stderr, no JSON line)")
    ap.add_argument("--only", default="", help="with --extra: only workloads whose label starts so")
    ap.add_argument("--probe-sweep", action="store_true",
                    help="time the streaming probe in several launch shapes beside the GAE step on "
                         "the headline sets (a table on stdout) and exit")
    ap.add_argument("--variant", type=int, default=0,
                    help="with --extra: force a kernel variant through the library's test hook "
                         "(rlcs_testing_set_variant; 1 = whole rows and two-pass whitening)")
    ap.add_argument("--summarize-counters", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="print the counter summary of two rocprofv3 --pmc runs and exit")
    ap.add_argument("--summarize-trace", metavar="TRACE_DIR",
                    help="print per-kernel durations of a rocprofv3 --kernel-trace run and exit")
    ap.add_argument("--profile-pass", action="store_true",
                    help="eager launches of the timed kernel plus a plain copy of known size, "
                         "for rocprofv3 runs (no JSON line); with --extra, of every workload")
    ap.add_argument("--manifest", default="",
                    help="with --extra --profile-pass: write the workload list (JSON) here")
    ap.add_argument("--summarize-extra", nargs=4, metavar=("TRACE_DIR", "FETCH_DIR", "WRITE_DIR", "MANIFEST"),
                    help="per-workload kernel durations and HBM traffic of three rocprofv3 runs of "
                         "--extra --profile-pass (kernel trace, FETCH_SIZE, WRITE_SIZE) and exit")
    return ap.parse_args()


def probe_lib():
    """libprobe.so (built beside the library): the streaming reference kernel with GAE's byte
    split and the empty launch."""
    import ctypes
    from paper_2608_17641_amd.build import PROBE_LIB
    if not os.path.exists(PROBE_LIB):
        raise RuntimeError(f"{PROBE_LIB} is missing: run __graft_entry__.build()")
    lib = ctypes.CDLL(PROBE_LIB)
    P = ctypes.c_void_p
    lib.probe_stream_gae.argtypes = [P] * 7 + [ctypes.c_int64, ctypes.c_int, P]
    lib.probe_stream_gae.restype = ctypes.c_int
    lib.probe_empty.argtypes = [P]
    lib.probe_empty.restype = ctypes.c_int
    lib.probe_stream_gae_shape.argtypes = [P] * 7 + [ctypes.c_int64, ctypes.c_int, ctypes.c_int,
                                                     ctypes.c_int64, ctypes.c_int, P]
    lib.probe_stream_gae_shape.restype = ctypes.c_int
    return lib


def probe_stream_call(lib, s, threads):
    """One streaming pass over set `s` (the GAE call's own buffers: r, v, bv, term, trunc read,
    adv and ret written)."""
    import torch
    st = torch.cuda.current_stream().cuda_stream
    rc = lib.probe_stream_gae(s["r"].data_ptr(), s["v"].data_ptr(), s["bv"].data_ptr(),
                              s["term"].data_ptr(), s["trunc"].data_ptr(), s["adv"].data_ptr(),
                              s["ret"].data_ptr(), s["r"].numel(), threads, st)
    if rc != 0:
        raise RuntimeError(f"probe_stream_gae returned {rc}")


# The events around a timed region are created with hipEventDisableSystemFence: they serve for
# timing only, so recording them skips the system-scope cache write-back and invalidation that a
# default event performs (the host synchronizes with the device by itself after the end event,
# outside the timed region). Measured on the 20 eager GAE steps behind the hold (us per step,
# medians of six): 5.27 with default events, 5.11 with these; at 2000 steps 4.85 either way.
HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000
_HIP = {}


def hip_runtime():
    """The HIP runtime that PyTorch loaded (ctypes), found among the process's mapped files so
    that no second copy of the runtime is loaded."""
    if "lib" not in _HIP:
        import ctypes
        import torch
        torch.cuda.init()
        with open("/proc/self/maps") as f:
            paths = {ln.split()[-1] for ln in f if "libamdhip64" in ln.split()[-1]}
        if len(paths) != 1:
            raise RuntimeError(f"expected one mapped HIP runtime, found {sorted(paths)}")
        lib = ctypes.CDLL(paths.pop())
        P = ctypes.c_void_p
        lib.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(P), ctypes.c_uint]
        lib.hipEventRecord.argtypes = [P, P]
        lib.hipEventSynchronize.argtypes = [P]
        lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), P, P]
        lib.hipEventDestroy.argtypes = [P]
        _HIP["lib"] = lib
    return _HIP["lib"]


class TimingEvent:
    """A HIP event for timing only (hipEventDisableSystemFence), recorded on PyTorch's current
    stream; record() and elapsed_time() as torch.cuda.Event's."""

    def __init__(self):
        import ctypes
        self._lib = hip_runtime()
        self._ev = ctypes.c_void_p()
        rc = self._lib.hipEventCreateWithFlags(ctypes.byref(self._ev), HIP_EVENT_DISABLE_SYSTEM_FENCE)
        if rc != 0:
            raise RuntimeError(f"hipEventCreateWithFlags returned {rc}")

    def record(self):
        import ctypes
        import torch
        rc = self._lib.hipEventRecord(self._ev, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        if rc != 0:
            raise RuntimeError(f"hipEventRecord returned {rc}")

    def elapsed_time(self, end):
        """Milliseconds from this event to `end` (waits for `end`)."""
        import ctypes
        rc = self._lib.hipEventSynchronize(end._ev)
        ms = ctypes.c_float()
        rc = rc or self._lib.hipEventElapsedTime(ctypes.byref(ms), self._ev, end._ev)
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime returned {rc}")
        return ms.value

    def __del__(self):
        if getattr(self, "_ev", None) and self._ev.value:
            self._lib.hipEventDestroy(self._ev)


# Up to this many steps the timed calls are launched eagerly; more are replayed from one HIP
# graph. Either way they queue behind the hold below, on a stream of their own. An eager launch
# costs about 0.3 us more on the GPU than a graph node, and a graph about 7.5 us once at its
# start. Measured on the GAE step behind the hold with the timing events above (us per step,
# medians of six; eager / graph): K = 20: 5.17 / 5.27; K = 50: 5.17 / 5.01; K = 2000 graph 4.87.
EAGER_MAX_STEPS = 25

# Untimed calls replayed from a graph right before the timed ones. They keep the GPU streaming
# the same work (as the other steps of a training loop keep it busy) while the host queues the
# timed calls, so that the timed calls neither wait for the host nor start on clocks that fell
# while the GPU idled: behind a 2-3 ms spin kernel instead, the first timed 2000-step replay of
# a process took 5.09-5.18 us per step and the later ones 4.78-4.88. A multiple of the number of
# rotated sets, so the first timed call's set was last touched a whole rotation earlier, as in
# the steady state of the timed calls themselves.
HOLD_CALLS = 2048


def hold_calls(sets):
    """Untimed calls before the timed ones: HOLD_CALLS rounded up to a multiple of `sets`."""
    sets = max(1, int(sets))
    return sets * -(-HOLD_CALLS // sets)


def timing_protocol(steps):
    """How `steps` timed calls are issued: 'eager' or 'graph'."""
    return "eager" if steps <= EAGER_MAX_STEPS else "graph"


def time_steps(fn, steps, start=None, end=None, sets=1):
    """Milliseconds for exactly `steps` calls fn(0) .. fn(steps - 1) on the current stream,
    between two events. The timed calls queue behind hold_calls(sets) untimed calls fn(0) ..
    replayed from a graph (fn(i) uses rotated set i % sets); they are launched eagerly for few
    steps, and replayed from one HIP graph (captured and replayed once beforehand) for more."""
    import torch
    start = start or TimingEvent()
    end = end or TimingEvent()
    hold = torch.cuda.CUDAGraph()
    with torch.cuda.graph(hold):
        for i in range(hold_calls(sets)):
            fn(i)
    graph = None
    if timing_protocol(steps) == "graph":
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for i in range(steps):
                fn(i)
        graph.replay()
    hold.replay()
    torch.cuda.synchronize()
    hold.replay()
    start.record()
    if graph is None:
        for i in range(steps):
            fn(i)
    else:
        graph.replay()
    end.record()
    torch.cuda.synchronize()
    del graph, hold
    return start.elapsed_time(end)


def _per_step_us(fn, steps, sets=1):
    """Mean microseconds per call of `steps` calls timed as the GAE steps are."""
    return time_steps(fn, steps, sets=sets) * 1e3 / steps


def copy_reference(sets, steps):
    """The streaming ceiling at this size: probe_stream_gae over the same rotated sets as the
    GAE steps (22 B per step: the three data inputs and two flag arrays read, both outputs
    written, densely), in 64- and 256-lane workgroups, timed like the GAE steps; and the
    empty-launch floor, issued like the timed GAE steps."""
    lib = probe_lib()
    S = len(sets)
    for i in range(S):
        probe_stream_call(lib, sets[i], 64)
    out = {}
    for threads in (64, 256):
        out[threads] = _per_step_us(lambda i: probe_stream_call(lib, sets[i % S], threads), steps, S)
    import torch
    empty = _per_step_us(lambda i: lib.probe_empty(torch.cuda.current_stream().cuda_stream), steps)
    return out, empty


# Launch shapes of the streaming probe timed by --probe-sweep: (label, lanes per workgroup,
# vectors per lane, persistent grid size or 0, dependent continuation loads).
PROBE_SHAPES = [
    ("64 lanes, 1 vector/lane", 64, 1, 0, 0),
    ("64 lanes, 1 vector/lane, dependent bv", 64, 1, 0, 1),
    ("256 lanes, 1 vector/lane", 256, 1, 0, 0),
    ("256 lanes, 1 vector/lane, dependent bv", 256, 1, 0, 1),
    ("64 lanes, 2 vectors/lane", 64, 2, 0, 0),
    ("64 lanes, 2 vectors/lane, dependent bv", 64, 2, 0, 1),
    ("64 lanes, 4 vectors/lane", 64, 4, 0, 0),
    ("256 lanes, 2 vectors/lane", 256, 2, 0, 0),
    ("persistent 1024 x 64 lanes", 64, 1, 1024, 0),
    ("persistent 2048 x 64 lanes", 64, 1, 2048, 0),
    ("persistent 512 x 256 lanes", 256, 1, 512, 0),
    ("persistent 1024 x 256 lanes", 256, 1, 1024, 0),
]


def probe_sweep(step, sets, steps):
    """The GAE step, the streaming probe in every PROBE_SHAPES launch shape, and the empty launch,
    each timed like the headline (`steps` calls over the rotated sets, cold); GB/s counts GAE's
    algorithmic bytes for every row."""
    import torch
    lib = probe_lib()
    S = len(sets)
    nbytes = algorithmic_bytes(N, T)
    rows = [("rlcs_gae", _per_step_us(step, steps, S))]
    for label, threads, per_lane, groups, dep in PROBE_SHAPES:
        def call(i, threads=threads, per_lane=per_lane, groups=groups, dep=dep):
            s = sets[i % S]
            rc = lib.probe_stream_gae_shape(s["r"].data_ptr(), s["v"].data_ptr(), s["bv"].data_ptr(),
                                            s["term"].data_ptr(), s["trunc"].data_ptr(),
                                            s["adv"].data_ptr(), s["ret"].data_ptr(), s["r"].numel(),
                                            threads, per_lane, groups, dep,
                                            torch.cuda.current_stream().cuda_stream)
            if rc != 0:
                raise RuntimeError(f"probe_stream_gae_shape returned {rc}")
        for i in range(S):
            call(i)
        rows.append((f"probe: {label}", _per_step_us(call, steps, S)))
    rows.append(("empty launch", _per_step_us(
        lambda i: lib.probe_empty(torch.cuda.current_stream().cuda_stream), steps)))
    print(f"# GAE {N}x{T} fp32 sets, {steps} steps per row ({timing_protocol(steps)}), cold; "
          f"GB/s = {nbytes} B / time")
    for label, us in rows:
        print(f"{label:<48} {us:8.3f} us {nbytes / us / 1e3:8.1f} GB/s {100 * nbytes / us / 1e3 / PEAK_HBM_GBS:6.1f} %",
              flush=True)


def cpu_baseline(ro, seconds):
    """The fp64 oracle on the same workload, repeated for about `seconds` each way: on one
    thread, and with the rows split over the host's cores (at most 16 threads; the oracle's C
    calls release the GIL). Reported: the all-cores rate, the single-thread one in `sample`."""
    import concurrent.futures as cf
    import oracle
    a = (ro["r"], ro["v"], ro["term"], ro["trunc"], ro["bv"], ro["boot"])
    oracle.gae(*a, gamma=GAMMA, lam=LAM)  # warm-up (also builds/loads the library)

    def timed(fn):
        reps, t0 = 0, time.perf_counter()
        while True:
            fn()
            reps += 1
            el = time.perf_counter() - t0
            if el >= seconds:
                return el / reps, reps, el

    one, reps1, el1 = timed(lambda: oracle.gae(*a, gamma=GAMMA, lam=LAM))
    threads = max(1, min(16, len(os.sched_getaffinity(0))))
    bounds = np.linspace(0, N, threads + 1).astype(int)
    slices = [tuple(x[lo:hi] for x in a) for lo, hi in zip(bounds[:-1], bounds[1:])]
    with cf.ThreadPoolExecutor(threads) as ex:
        def all_rows():
            list(ex.map(lambda sl: oracle.gae(*sl, gamma=GAMMA, lam=LAM), slices))
        all_rows()
        par, reps, el = timed(all_rows)
    nbytes = algorithmic_bytes(N, T)
    return {
        "value": round(nbytes / par / 1e9, 3),
        "unit": "GB/s",
        "cores": threads,
        "kind": "oracle",
        "sample": f"GAE {N}x{T} fp32+trunc, full workload: {threads} threads (rows split), "
                  f"{reps}x in {el:.1f} s, {par * 1e3:.2f} ms/call, {N * T / par / 1e9:.3f} Gsteps/s; "
                  f"1 thread: {reps1}x in {el1:.1f} s, {one * 1e3:.1f} ms/call, "
                  f"{nbytes / one / 1e9:.3f} GB/s, {N * T / one / 1e9:.4f} Gsteps/s (fp64 sequential C)",
    }


COPY_BYTES = 64 << 20
KERNEL_TAG = "wave_rows_kernel<rlcs::GaeOp, float, 4, true, 4>"
COUNTERS_FILE = os.path.join(ROOT, "profiles", "gae_4096x256_f32_counters.md")


def kernel_source_hash():
    """sha256 over the HIP sources of the library (kernels and launch code; not the measurement
    probe built beside it) and the build script that holds the compiler flags."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_17641_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if name.startswith("rlcs_") and name.endswith((".h", ".hip")):
            with open(os.path.join(csrc, name), "rb") as f:
                h.update(name.encode() + b"\0" + f.read())
    with open(os.path.join(ROOT, "paper_2608_17641_amd", "build.py"), "rb") as f:
        h.update(b"build.py\0" + f.read())
    return h.hexdigest()


def recorded_traffic():
    """HBM bytes per launch from the committed counter summary, if it was taken on the
    current kernel sources; otherwise None."""
    try:
        text = open(COUNTERS_FILE).read()
    except OSError:
        return None
    fields = dict(l.split(":", 1) for l in text.splitlines() if ":" in l and not l.startswith(" "))
    if fields.get("source_sha256", "").strip() != kernel_source_hash():
        return None
    try:
        return int(fields["traffic_bytes_per_launch"].strip())
    except (KeyError, ValueError):
        return None


def _rocpd(path):
    dbs = sorted(glob.glob(os.path.join(path, "**", "*.db"), recursive=True)) if os.path.isdir(path) else [path]
    if not dbs:
        raise SystemExit(f"no rocprofv3 database under {path}")
    return sqlite3.connect(dbs[0])


def _is_copy(name):
    return "copyBuffer" in name or "copy_kernel" in name


def _calibration_kib(rows, counter):
    """Mean counter value of the calibration copies of COPY_BYTES: the copy dispatches that end
    a profile pass (rows are (dispatch_id, kernel name, value) in dispatch order)."""
    tail = []
    for _, name, val in reversed(rows):
        if not _is_copy(name):
            break
        tail.append(val)
    if not tail:
        raise SystemExit(f"{counter}: no calibration copy at the end of the run")
    return statistics.mean(tail)


def summarize_counters(fetch_dir, write_dir):
    """Counter summary (FETCH_SIZE, WRITE_SIZE per dispatch of the timed kernel, each scaled by
    the same counter on a plain device copy of COPY_BYTES) in the committed format."""
    out = {}
    for counter, path in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        cur = _rocpd(path).cursor()
        rows = cur.execute("select dispatch_id, kernel_name, value from counters_collection "
                           "where counter_name = ? order by dispatch_id", (counter,)).fetchall()
        mine = [v for _, n, v in rows if KERNEL_TAG in n]
        if not mine:
            raise SystemExit(f"{counter}: kernel not found in {path}")
        copy_kib = _calibration_kib(rows, counter)
        out[counter] = (statistics.mean(mine), len(mine), copy_kib, (COPY_BYTES / 1024) / copy_kib)
    fetch, write = out["FETCH_SIZE"], out["WRITE_SIZE"]
    traffic = int(round((fetch[0] * fetch[3] + write[0] * write[3]) * 1024))
    alg = algorithmic_bytes(N, T)
    lines = [
        f"# HBM traffic of {KERNEL_TAG}",
        f"# workload: GAE {N}x{T} fp32, term+trunc, bootstrap (bench.py --profile-pass)",
        "commands (repo root, on the MI355X host):",
        "  rocprofv3 --pmc FETCH_SIZE -d prof/pmc_fetch -o run -- python bench.py --profile-pass --steps 200 --warmup 20",
        "  rocprofv3 --pmc WRITE_SIZE -d prof/pmc_write -o run -- python bench.py --profile-pass --steps 200 --warmup 20",
        "  python bench.py --summarize-counters prof/pmc_fetch prof/pmc_write",
        f"FETCH_SIZE_KiB_per_dispatch: {fetch[0]:.1f}",
        f"FETCH_SIZE_dispatches: {fetch[1]}",
        f"FETCH_SIZE_copy_KiB: {fetch[2]:.1f}",
        f"FETCH_SIZE_scale: {fetch[3]:.4f}",
        f"WRITE_SIZE_KiB_per_dispatch: {write[0]:.1f}",
        f"WRITE_SIZE_dispatches: {write[1]}",
        f"WRITE_SIZE_copy_KiB: {write[2]:.1f}",
        f"WRITE_SIZE_scale: {write[3]:.4f}",
        f"traffic_bytes_per_launch: {traffic}",
        f"algorithmic_bytes_per_launch: {alg}",
        f"traffic_over_algorithmic: {traffic / alg:.4f}",
        f"source_sha256: {kernel_source_hash()}",
    ]
    print("\n".join(lines))


def summarize_trace(trace_dir):
    """Per-kernel duration statistics from a rocprofv3 --kernel-trace run."""
    cur = _rocpd(trace_dir).cursor()
    rows = cur.execute("select name, start, end from kernels").fetchall()
    by = {}
    for n, a, b in rows:
        by.setdefault(n, []).append((b - a) / 1e3)
    print(f"{'kernel':<70} {'calls':>6} {'avg_us':>8} {'median_us':>9} {'min_us':>7} {'max_us':>8}")
    for n, v in sorted(by.items(), key=lambda kv: -sum(kv[1])):
        v.sort()
        print(f"{n[:70]:<70} {len(v):>6} {statistics.mean(v):>8.3f} {v[len(v) // 2]:>9.3f} "
              f"{v[0]:>7.3f} {v[-1]:>8.3f}")


def _blocks(path, value_col):
    """The library's dispatches of a --extra --profile-pass run, in launch order, between each
    pair of markers: a list of [(kernel name, value)] per block. `value_col` is 'duration'
    (kernel trace, ns) or a counter name (counter run, per dispatch)."""
    cur = _rocpd(path).cursor()
    if value_col == "duration":
        rows = cur.execute("select dispatch_id, name, duration from kernels order by dispatch_id").fetchall()
    else:
        rows = cur.execute("select dispatch_id, kernel_name, value from counters_collection "
                           "where counter_name = ? order by dispatch_id", (value_col,)).fetchall()
    blocks, inside = [], False
    for _, name, val in rows:
        if MARKER_KERNEL in name:
            inside = not inside
            if inside:
                blocks.append([])
        elif "rlcs::" in name and inside:
            blocks[-1].append((name, val))
    if inside:
        raise SystemExit(f"{path}: unmatched block marker")
    return blocks, rows


def _copy_scale(rows, counter):
    return (COPY_BYTES / 1024) / _calibration_kib(rows, counter)


def _short(name):
    name = name.replace("rlcs::", "").replace("void ", "")
    return name.split("(")[0][:42]


def summarize_extra(trace_dir, fetch_dir, write_dir, manifest):
    """Per workload: each library kernel's average duration (kernel trace) and its HBM bytes
    per call (FETCH_SIZE and WRITE_SIZE, scaled by the same counters on a plain copy of
    COPY_BYTES), against the dense algorithmic bytes."""
    man = json.load(open(manifest))
    trace, _ = _blocks(trace_dir, "duration")
    fetch, frows = _blocks(fetch_dir, "FETCH_SIZE")
    write, wrows = _blocks(write_dir, "WRITE_SIZE")
    fs, ws = _copy_scale(frows, "FETCH_SIZE"), _copy_scale(wrows, "WRITE_SIZE")
    for what, b in (("trace", trace), ("FETCH_SIZE", fetch), ("WRITE_SIZE", write)):
        if len(b) != len(man):
            raise SystemExit(f"{what}: {len(b)} marked blocks, manifest lists {len(man)}")
    print(f"FETCH_SIZE_scale: {fs:.4f}\nWRITE_SIZE_scale: {ws:.4f}")
    print(f"{'workload':<18} {'estimator':<16} {'kernel':<44} {'avg_us':>8} {'GB/s':>7} {'%peak':>6} "
          f"{'traffic_B':>11} {'alg_B':>11} {'ratio':>6}")
    for m, tb, fb, wb in zip(man, trace, fetch, write):
        calls = m["calls"]
        kinds = sorted({n for n, _ in tb}, key=[n for n, _ in tb].index)
        per_call_us = sum(v for _, v in tb) / 1e3 / calls
        traffic = (sum(v for _, v in fb) * fs + sum(v for _, v in wb) * ws) * 1024 / calls
        for k in kinds if len(kinds) > 1 else ():
            d = [v / 1e3 for n, v in tb if n == k]
            f = [v for n, v in fb if n == k]
            w = [v for n, v in wb if n == k]
            kt = (statistics.mean(f) * fs + statistics.mean(w) * ws) * 1024
            print(f"{m['label']:<18} {m['name']:<16} {'- ' + _short(k):<44} {statistics.mean(d):>8.3f} "
                  f"{'':>7} {'':>6} {kt:>11.0f}")
        gbs = m["bytes"] / (per_call_us * 1e-6) / 1e9
        what = _short(kinds[0]) if len(kinds) == 1 else "(per call: the kernels above)"
        print(f"{m['label']:<18} {m['name']:<16} {what:<44} {per_call_us:>8.3f} {gbs:>7.0f} "
              f"{100 * gbs / PEAK_HBM_GBS:>5.1f}% {traffic:>11.0f} {m['bytes']:>11} "
              f"{traffic / m['bytes']:>6.3f}")


def profile_pass(step, args, dev):
    """Eager launches for kernel-trace / counter runs, then a plain device copy of COPY_BYTES
    (read COPY_BYTES, write COPY_BYTES) that calibrates the HBM byte counters."""
    import torch
    for i in range(args.warmup):
        step(i)
    for i in range(args.steps):
        step(i)
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(f"profile pass: {args.warmup + args.steps} launches, 3 copies of {COPY_BYTES} B", flush=True)


# Dense algorithmic bytes per step (data elements of `eb` bytes, 1-byte flags, 4-byte outputs)
# and the data inputs each estimator reads, for the --extra workloads.
EXTRA_EST = {
    "gae": (("r", "v"), 2), "vtrace": (("r", "v", "log_rho"), 2),
    "retrace": (("r", "q", "eq", "log_rho"), 2), "td_lambda": (("r", "v"), 1),
    "discounted": (("r",), 1), "elig_trace": (("x",), 1), "episodic_prefix": (("x",), 1),
}


def extra_bytes(name, N, T, eb, trunc, boot):
    data, outs = EXTRA_EST[name]
    backward = name not in ("elig_trace", "episodic_prefix")
    per = len(data) * eb + 1 + (1 + (eb if backward else 0) if trunc else 0) + 4 * outs
    return N * T * per + (N * eb if (boot and backward) else 0)


def run_extra(dev, only=""):
    """Time every estimator of every workload (cold where the data exceeds the Infinity Cache,
    otherwise over rotated sets), after a parity check of sampled rows against the oracle.
    Prints a table on stderr."""
    import torch
    import oracle
    import workloads
    import paper_2608_17641_amd as rl

    def to_dev(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).to(dev).view(torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    def call(name, d, ws, gamma, lam, trunc, boot):
        tr = d["trunc"] if trunc else None
        bv = d["bv"] if trunc else None
        bt = d["boot"] if boot else None
        if name == "gae":
            return rl.rlcs_gae(d["r"], d["v"], d["term"], tr, bv, bt, d["o0"], d["o1"], gamma=gamma, lam=lam, ws=ws)
        if name == "vtrace":
            return rl.rlcs_vtrace(d["r"], d["v"], d["log_rho"], d["term"], tr, bv, bt, d["o0"], d["o1"], gamma=gamma, ws=ws)
        if name == "retrace":
            return rl.rlcs_retrace(d["r"], d["q"], d["eq"], d["log_rho"], d["term"], tr, bv, bt, d["o0"], d["o1"],
                                   gamma=gamma, lam=lam, ws=ws)
        if name == "td_lambda":
            return (rl.rlcs_td_lambda(d["r"], d["v"], d["term"], tr, bv, bt, d["o0"], gamma=gamma, lam=lam, ws=ws),)
        if name == "discounted":
            return (rl.rlcs_discounted(d["r"], d["term"], tr, bv, bt, d["o0"], gamma=gamma, ws=ws),)
        if name == "elig_trace":
            return (rl.rlcs_elig_trace(d["x"], d["term"], tr, d["o0"], gamma=gamma, lam=lam, ws=ws),)
        return (rl.rlcs_episodic_prefix(d["x"], d["term"], tr, d["o0"], ws=ws),)

    def ref(name, ro, rows, gamma, lam, trunc, boot):
        g = lambda k: ro[k][rows]
        tr = g("trunc") if trunc else None
        bv = g("bv") if trunc else None
        bt = g("boot") if boot else None
        if name == "gae":
            return oracle.gae(g("r"), g("v"), g("term"), tr, bv, bt, gamma=gamma, lam=lam)
        if name == "vtrace":
            return oracle.vtrace(g("r"), g("v"), g("log_rho"), g("term"), tr, bv, bt, gamma=gamma)
        if name == "retrace":
            return oracle.retrace(g("r"), g("q"), g("eq"), g("log_rho"), g("term"), tr, bv, bt, gamma=gamma, lam=lam)
        if name == "td_lambda":
            return (oracle.td_lambda(g("r"), g("v"), g("term"), tr, bv, bt, gamma=gamma, lam=lam),)
        if name == "discounted":
            return (oracle.discounted(g("r"), g("term"), tr, bv, bt, gamma=gamma),)
        if name == "elig_trace":
            return (oracle.elig_trace(g("x"), g("term"), tr, gamma=gamma, lam=lam),)
        return (oracle.episodic_prefix(g("x"), g("term"), tr),)

    plan = [("gae_8x128", 8, 128, "f32", dict(p_term=0.01, p_trunc=0.0), False, True, 0.99, 0.95, ("gae",))]
    seven = tuple(EXTRA_EST)
    plan.append(("all7_4096x32", 4096, 32, "f32", dict(p_term=0.02, p_trunc=0.01), True, True, 0.99, 0.95, seven))
    plan.append(("4096x256", 4096, 256, "f32", dict(p_term=0.02, p_trunc=0.01), True, True, 0.99, 0.95, ("gae", "vtrace")))
    plan.append(("4096x256_plain", 4096, 256, "f32", dict(p_term=0.02, p_trunc=0.0), False, True, 0.99, 0.95, ("gae",)))
    plan.append(("rlhf_64x4096", 64, 4096, "f32", None, False, False, 1.0, 0.95, ("gae", "td_lambda")))
    # dense rows of a multiple of the vector width that do not tile a wave: the flat rows kernel
    plan.append(("flat_4096x200", 4096, 200, "f32", dict(p_term=0.02, p_trunc=0.01), True, True, 0.99, 0.95,
                 ("gae", "vtrace", "elig_trace")))
    plan.append(("flat_4096x1000", 4096, 1000, "f32", dict(p_term=0.02, p_trunc=0.01), True, True, 0.99, 0.95,
                 ("gae", "td_lambda")))
    plan.append(("flat_bf16_16384x200", 16384, 200, "bf16", dict(p_term=0.005, p_trunc=0.005), True, True, 0.99,
                 0.95, ("gae", "retrace")))
    # rows of a length that is not a multiple of the vector width: the flat rows kernel (four or
    # sixteen waves) where a workgroup's rows can start and end on vector boundaries
    plan.append(("ragged_4096x255", 4096, 255, "f32", dict(p_term=0.02, p_trunc=0.01), True, True, 0.99, 0.95,
                 ("gae", "vtrace", "elig_trace")))
    plan.append(("ragged_4096x499", 4096, 499, "f32", dict(p_term=0.02, p_trunc=0.01), True, True, 0.99, 0.95,
                 ("gae", "vtrace")))
    plan.append(("ragged_1024x1001", 1024, 1001, "f32", dict(p_term=0.02, p_trunc=0.01), True, True, 0.99, 0.95,
                 ("gae",)))
    plan.append(("ragged_bf16_16384x100", 16384, 100, "bf16", dict(p_term=0.005, p_trunc=0.005), True, True, 0.99,
                 0.95, ("gae", "retrace")))
    for n_ in (16384, 65536):
        for t_ in (64, 512, 2048):
            plan.append((f"bf16_{n_}x{t_}", n_, t_, "bf16", dict(p_term=0.005, p_trunc=0.005), True, True, 0.99, 0.95, seven))
    print(f"{'workload':<18} {'estimator':<16} {'us/step':>9} {'GB/s':>8} {'%peak':>6} {'Gsteps/s':>9} {'sets':>5} {'max_rel_err':>11}",
          file=sys.stderr, flush=True)
    for label, n_, t_, dt, kw, trunc, boot, gamma, lam, ests in plan:
        if not label.startswith(only):
            continue
        ro = (workloads.make_rlhf_rollout(n_, t_, 0) if kw is None
              else workloads.make_rollout(n_, t_, 0, dtype=dt, **kw))
        eb = 2 if dt == "bf16" else 4
        base = {k: to_dev(v) for k, v in ro.items()}
        set_bytes = sum(v.numel() * v.element_size() for v in base.values()) + 8 * n_ * t_
        S = max(1, min(32, -(-600_000_000 // set_bytes)))
        sets = []
        for i in range(S):
            d = base if i == 0 else {k: v.clone() for k, v in base.items()}
            d = dict(d)
            d["o0"] = torch.empty((n_, t_), dtype=torch.float32, device=dev)
            d["o1"] = torch.empty((n_, t_), dtype=torch.float32, device=dev)
            sets.append(d)
        ws = rl.make_workspace(n_, t_, dev)
        rows = np.unique(np.concatenate([[0, n_ - 1], np.random.default_rng(1).integers(0, n_, 32)]))
        for name in ests:
            outs = call(name, sets[0], ws, gamma, lam, trunc, boot)
            torch.cuda.synchronize()
            refs = ref(name, ro, rows, gamma, lam, trunc, boot)
            rel = 0.0
            for o, r_ in zip(outs, refs):
                got = o.index_select(0, torch.from_numpy(rows).to(dev)).double().cpu().numpy()
                rel = max(rel, float(np.max(np.abs(got - r_))) / (1 + float(np.max(np.abs(r_)))))
            if rel > (1e-3 if dt == "bf16" else 1e-5):
                raise SystemExit(f"parity failure in {label} {name}: {rel}")
            nbytes = extra_bytes(name, n_, t_, eb, trunc, boot)
            _measure(label, name, lambda d: call(name, d, ws, gamma, lam, trunc, boot), sets, nbytes,
                     n_ * t_, rel)
        del sets, base, ws
        torch.cuda.empty_cache()
    for label, n_, t_, a_ in (("rf_4096x256x4", 4096, 256, 4), ("rf_512x4096x4", 512, 4096, 4),
                              ("rf_4096x256x18", 4096, 256, 18), ("rf_4096x256x64", 4096, 256, 64),
                              ("rf_1024x256x256", 1024, 256, 256)):
        if label.startswith(only):
            run_retrace_full(label, n_, t_, a_, dev)
    for label, t_, n_ in (("tm_256x4096", 256, 4096), ("tm_4096x64", 4096, 64),
                          ("tm_2048x128", 2048, 128), ("tm_64x65536", 64, 65536)):
        if label.startswith(only):
            run_time_major(label, t_, n_, dev)
    if "tm_noflags_16384x64".startswith(only):
        run_time_major("tm_noflags_16384x64", 16384, 64, dev, noflags=True)
    for label, n_, t_, ld in (("sr_4096x256_ld320", 4096, 256, 320), ("sr_64x4096_ld4160", 64, 4096, 4160)):
        if label.startswith(only):
            run_strided_rows(label, n_, t_, ld, dev)
    for label, n_, t_, f_ in (("vec_4096x256x16", 4096, 256, 16), ("vec_65536x8x16", 65536, 8, 16),
                              ("vec_64x1024x256", 64, 1024, 256), ("vec_1x128x1M", 1, 128, 1 << 20)):
        if label.startswith(only):
            run_vector_trace(label, n_, t_, f_, dev)
    for label, n_, t_ in (("mt_64x4096", 64, 4096), ("mt_4096x256", 4096, 256),
                          ("mt_1024x2048", 1024, 2048)):
        if label.startswith(only):
            run_masked(label, n_, t_, dev)


def run_retrace_full(label, n_, t_, a_, dev):
    """Full-form Retrace (fp32, truncation), parity on sampled rows, then graph-timed."""
    import torch
    import oracle
    import workloads
    import paper_2608_17641_amd as rl
    ro = workloads.make_retrace_full(n_, t_, a_, 0)
    base = {k: torch.from_numpy(np.ascontiguousarray(v)).to(dev) for k, v in ro.items()}
    set_bytes = sum(v.numel() * v.element_size() for v in base.values()) + 8 * n_ * t_
    S = max(1, min(32, -(-600_000_000 // set_bytes)))
    sets = []
    for i in range(S):
        d = dict(base if i == 0 else {k: v.clone() for k, v in base.items()})
        d["o0"] = torch.empty((n_, t_), dtype=torch.float32, device=dev)
        d["o1"] = torch.empty((n_, t_), dtype=torch.float32, device=dev)
        sets.append(d)

    def call(d):
        rl.rlcs_retrace_full(d["r"], d["q3"], d["pi3"], d["actions"], d["mu"], d["term"], d["trunc"],
                             d["bv"], d["boot"], d["o0"], d["o1"], gamma=0.99, lam=0.95)

    call(sets[0])
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, n_ - 1], np.random.default_rng(1).integers(0, n_, 32)]))
    g = lambda k: ro[k][rows]
    rd, rq = oracle.retrace_full(g("r"), g("q3"), g("pi3"), g("actions"), g("mu"), g("term"),
                                 g("trunc"), g("bv"), g("boot"), gamma=0.99, lam=0.95)
    rel = 0.0
    for o, r_ in ((sets[0]["o0"], rd), (sets[0]["o1"], rq)):
        got = o.index_select(0, torch.from_numpy(rows).to(dev)).double().cpu().numpy()
        rel = max(rel, float(np.max(np.abs(got - r_))) / (1 + float(np.max(np.abs(r_)))))
    if rel > 1e-5:
        raise SystemExit(f"parity failure in {label}: {rel}")
    # r, Q and pi [A], action (4 B), mu, term, trunc, bv, two outputs; bootstrap per row
    nbytes = n_ * t_ * (4 + 8 * a_ + 4 + 4 + 1 + 1 + 4 + 8) + 4 * n_
    _measure(label, "retrace_full", call, sets, nbytes, n_ * t_, rel)


def _rotated_sets(base, S, outs):
    """S input/output sets: set 0 is `base`, the others copies; fresh float32 outputs."""
    import torch
    sets = []
    for i in range(S):
        d = dict(base if i == 0 else {k: v.clone() for k, v in base.items()})
        for name, like in outs.items():
            d[name] = torch.empty_like(like, dtype=torch.float32)
        sets.append(d)
    return sets


def extra_calls(nbytes, sets):
    """Timed calls per --extra row: about 8 GB of algorithmic bytes (a few ms at these rates, so
    that the fixed cost at the two events, about 9 us, stays near 1 %), at least 20 and at most
    2000 calls, rounded up to a whole number of rotations over `sets`."""
    k = int(max(20, min(2000, -(-8e9 // max(1, nbytes)))))
    return sets * -(-k // sets)


def _graph_time(call, sets, nbytes):
    """Mean microseconds per call over extra_calls() graph-replayed calls cycling through
    `sets`, timed behind an untimed replay of the same graph."""
    import torch
    S = len(sets)
    K = extra_calls(nbytes, S)
    for i in range(3):
        call(sets[i % S])
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for i in range(K):
            call(sets[i % S])
    graph.replay()
    torch.cuda.synchronize()
    a, b = TimingEvent(), TimingEvent()
    graph.replay()
    a.record(); graph.replay(); b.record()
    torch.cuda.synchronize()
    del graph
    return a.elapsed_time(b) * 1e3 / K


def _report(label, name, us, nbytes, steps, S, rel):
    gbs = nbytes / (us * 1e-6) / 1e9
    print(f"{label:<18} {name:<16} {us:>9.3f} {gbs:>8.1f} {100 * gbs / PEAK_HBM_GBS:>5.1f}% "
          f"{steps / (us * 1e-6) / 1e9:>9.1f} {S:>5} {rel:>11.2e}", file=sys.stderr, flush=True)


# With --extra --profile-pass: eager launches per workload for rocprofv3 runs instead of graph
# timing. Each workload's launches sit between two one-element int16 fills (a marker no other
# step of the run launches), and `manifest` lists the workloads in launch order.
_PROFILE = {"on": False, "calls": 20, "manifest": []}
MARKER_KERNEL = "FillFunctor<short>"


def _measure(label, name, call, sets, nbytes, steps, rel):
    """Graph-time `call` over the rotated `sets` and print a table line, or, in a profile pass,
    launch it eagerly after a block marker and record the workload in the manifest."""
    import torch
    if not _PROFILE["on"]:
        _report(label, name, _graph_time(call, sets, nbytes), nbytes, steps, len(sets), rel)
        return
    dev = next(v for v in sets[0].values() if torch.is_tensor(v)).device
    torch.cuda.synchronize()
    torch.full((1,), 7, dtype=torch.int16, device=dev)
    for i in range(_PROFILE["calls"]):
        call(sets[i % len(sets)])
    torch.full((1,), 7, dtype=torch.int16, device=dev)
    torch.cuda.synchronize()
    _PROFILE["manifest"].append({"label": label, "name": name, "calls": _PROFILE["calls"],
                                 "bytes": int(nbytes), "steps": int(steps)})
    print(f"profile pass: {label} {name} x{_PROFILE['calls']}", file=sys.stderr, flush=True)


def run_time_major(label, t_, n_, dev, noflags=False):
    """GAE and V-Trace on a time-major [T, N] fp32 buffer with truncation: parity on sampled
    environments, then graph-timed. Same dense byte count as the row-major form. `noflags`: GAE
    alone, a termination array with no flag set, no truncation, gamma = lambda = 1 (every
    look-back runs to the column's edge)."""
    import torch
    import oracle
    import workloads
    import paper_2608_17641_amd as rl
    ro = workloads.make_rollout_time_major(t_, n_, 0, p_term=0.0 if noflags else 0.02,
                                           p_trunc=0.0 if noflags else 0.01)
    base = {k: torch.from_numpy(np.ascontiguousarray(v)).to(dev) for k, v in ro.items()}
    set_bytes = sum(v.numel() * v.element_size() for v in base.values()) + 8 * n_ * t_
    S = max(1, min(32, -(-600_000_000 // set_bytes)))
    sets = _rotated_sets(base, S, {"o0": base["r"], "o1": base["r"]})
    ws = rl.make_workspace_columns(n_, t_, dev)
    cols = np.unique(np.concatenate([[0, n_ - 1], np.random.default_rng(1).integers(0, n_, 32)]))
    g = lambda k: np.ascontiguousarray(ro[k][:, cols]) if ro[k].ndim == 2 else ro[k][cols]
    for name in (("gae",) if noflags else ("gae", "vtrace")):
        if noflags:
            call = lambda d: rl.rlcs_gae_strided(d["r"].t(), d["v"].t(), d["term"].t(), None, None,
                                                 d["boot"], d["o0"].t(), d["o1"].t(), gamma=1.0,
                                                 lam=1.0, ws=ws)
            refs = oracle.time_major(oracle.gae, g("r"), g("v"), g("term"), None, None, g("boot"),
                                     gamma=1.0, lam=1.0)
        elif name == "gae":
            call = lambda d: rl.rlcs_gae_strided(d["r"].t(), d["v"].t(), d["term"].t(), d["trunc"].t(),
                                                 d["bv"].t(), d["boot"], d["o0"].t(), d["o1"].t(),
                                                 gamma=0.99, lam=0.95, ws=ws)
            refs = oracle.time_major(oracle.gae, g("r"), g("v"), g("term"), g("trunc"), g("bv"),
                                     g("boot"), gamma=0.99, lam=0.95)
        else:
            call = lambda d: rl.rlcs_vtrace_strided(d["r"].t(), d["v"].t(), d["log_rho"].t(),
                                                    d["term"].t(), d["trunc"].t(), d["bv"].t(),
                                                    d["boot"], d["o0"].t(), d["o1"].t(), gamma=0.99,
                                                    ws=ws)
            refs = oracle.time_major(oracle.vtrace, g("r"), g("v"), g("log_rho"), g("term"),
                                     g("trunc"), g("bv"), g("boot"), gamma=0.99)
        call(sets[0])
        torch.cuda.synchronize()
        rel = 0.0
        for o, r_ in zip((sets[0]["o0"], sets[0]["o1"]), refs):
            got = o.index_select(1, torch.from_numpy(cols).to(dev)).double().cpu().numpy()
            rel = max(rel, float(np.max(np.abs(got - r_))) / (1 + float(np.max(np.abs(r_)))))
        if rel > 1e-5:
            raise SystemExit(f"parity failure in {label} {name}: {rel}")
        nbytes = extra_bytes(name, n_, t_, 4, not noflags, True)
        _measure(label, name + "_tm", call, sets, nbytes, n_ * t_, rel)


def run_strided_rows(label, n_, t_, ld, dev):
    """GAE on [N, T] rows that are the first T steps of [N, ld] rows (fp32, truncation):
    parity on sampled rows, then graph-timed. Same dense byte count as the row-major form."""
    import torch
    import oracle
    import workloads
    import paper_2608_17641_amd as rl
    ro = workloads.make_rollout(n_, t_, 0, p_term=0.02, p_trunc=0.01)

    def wide(a):
        t = torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        if t.dim() != 2:
            return t
        buf = torch.zeros((n_, ld), dtype=t.dtype, device=dev)
        buf[:, :t_] = t
        return buf[:, :t_]
    base = {k: wide(v) for k, v in ro.items()}
    S = max(1, min(32, -(-600_000_000 // (n_ * ld * 30))))
    sets = []
    for i in range(S):
        d = dict(base if i == 0 else {k: wide(v) for k, v in ro.items()})
        d["o0"] = torch.empty((n_, ld), dtype=torch.float32, device=dev)[:, :t_]
        d["o1"] = torch.empty((n_, ld), dtype=torch.float32, device=dev)[:, :t_]
        sets.append(d)
    ws = rl.make_workspace_columns(n_, t_, dev)
    call = lambda d: rl.rlcs_gae_strided(d["r"], d["v"], d["term"], d["trunc"], d["bv"], d["boot"],
                                         d["o0"], d["o1"], gamma=0.99, lam=0.95, ws=ws)
    call(sets[0])
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, n_ - 1], np.random.default_rng(1).integers(0, n_, 32)]))
    g = lambda k: ro[k][rows]
    refs = oracle.gae(g("r"), g("v"), g("term"), g("trunc"), g("bv"), g("boot"), gamma=0.99, lam=0.95)
    rel = 0.0
    for o, r_ in zip((sets[0]["o0"], sets[0]["o1"]), refs):
        got = o.index_select(0, torch.from_numpy(rows).to(dev)).double().cpu().numpy()
        rel = max(rel, float(np.max(np.abs(got - r_))) / (1 + float(np.max(np.abs(r_)))))
    if rel > 1e-5:
        raise SystemExit(f"parity failure in {label}: {rel}")
    nbytes = extra_bytes("gae", n_, t_, 4, True, True)
    _measure(label, "gae_strided", call, sets, nbytes, n_ * t_, rel)


def run_vector_trace(label, n_, t_, f_, dev):
    """Eligibility traces of F-vectors (fp32, both flags): parity on sampled rows, then
    graph-timed. Dense bytes: x and z (4 B each per feature) and two flag bytes per step."""
    import torch
    import oracle
    import workloads
    import paper_2608_17641_amd as rl
    ro = workloads.make_vector_trace(n_, t_, f_, 0)
    base = {k: torch.from_numpy(np.ascontiguousarray(v)).to(dev) for k, v in ro.items()}
    set_bytes = sum(v.numel() * v.element_size() for v in base.values()) + 4 * n_ * t_ * f_
    S = max(1, min(32, -(-600_000_000 // set_bytes)))
    sets = _rotated_sets(base, S, {"z": base["x"]})
    ws = rl.make_workspace_columns(n_ * f_, t_, dev)
    call = lambda d: rl.rlcs_elig_trace_vec(d["x"], d["term"], d["trunc"], d["z"], gamma=0.99,
                                            lam=0.95, ws=ws)
    call(sets[0])
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, n_ - 1], np.random.default_rng(1).integers(0, n_, 8)]))
    feats = np.unique(np.concatenate([[0, f_ - 1], np.random.default_rng(2).integers(0, f_, 64)]))
    xs = np.ascontiguousarray(ro["x"][rows][:, :, feats])
    ref = oracle.elig_trace_vec(xs, ro["term"][rows], ro["trunc"][rows], gamma=0.99, lam=0.95)
    got = sets[0]["z"][torch.from_numpy(rows).to(dev)][:, :, torch.from_numpy(feats).to(dev)]
    got = got.double().cpu().numpy()
    rel = float(np.max(np.abs(got - ref))) / (1 + float(np.max(np.abs(ref))))
    if rel > 1e-5:
        raise SystemExit(f"parity failure in {label}: {rel}")
    nbytes = n_ * t_ * (8 * f_ + 2)
    _measure(label, "elig_trace_vec", call, sets, nbytes, n_ * t_ * f_, rel)


def run_masked(label, n_, t_, dev):
    """Masked GAE on multi-turn rows (fp32, gamma 1), plain and whitened: parity on sampled
    rows (whitened: the statistics are recomputed by the oracle over the whole batch), then
    graph-timed. Dense bytes: r, v (4 B each), mask and term (1 B each), adv and ret (4 B
    each) per step; whitening is counted as fused (no extra bytes)."""
    import torch
    import oracle
    import workloads
    import paper_2608_17641_amd as rl
    ro = workloads.make_multiturn(n_, t_, 0)
    base = {k: torch.from_numpy(np.ascontiguousarray(v)).to(dev) for k, v in ro.items()}
    set_bytes = sum(v.numel() * v.element_size() for v in base.values()) + 8 * n_ * t_
    S = max(1, min(32, -(-600_000_000 // set_bytes)))
    sets = _rotated_sets(base, S, {"o0": base["r"], "o1": base["r"]})
    ws = torch.zeros(rl.rlcs_workspace_size_masked(n_, t_), dtype=torch.uint8, device=dev)
    adv_ref, _ = oracle.gae_masked(ro["r"], ro["v"], ro["mask"], ro["term"], None, None, ro["boot"],
                                   gamma=1.0, lam=0.95)
    nbytes = n_ * t_ * 18
    rows = np.unique(np.concatenate([[0, n_ - 1], np.random.default_rng(1).integers(0, n_, 32)]))
    for norm in (False, True):
        call = lambda d: rl.rlcs_gae_masked(d["r"], d["v"], d["mask"], d["term"], None, None,
                                            d["boot"], d["o0"], d["o1"], gamma=1.0, lam=0.95,
                                            normalize=norm, ws=ws)
        call(sets[0])
        torch.cuda.synchronize()
        ref = oracle.normalize_advantages(adv_ref, ro["mask"], eps=1e-8) if norm else adv_ref
        got = sets[0]["o0"].index_select(0, torch.from_numpy(rows).to(dev)).double().cpu().numpy()
        r_ = ref[rows]
        rel = float(np.max(np.abs(got - r_))) / (1 + float(np.max(np.abs(r_))))
        if rel > 1e-5:
            raise SystemExit(f"parity failure in {label} norm={norm}: {rel}")
        _measure(label, "gae_masked" + ("_norm" if norm else ""), call, sets, nbytes, n_ * t_, rel)


def main():
    args = parse()
    if args.summarize_counters:
        summarize_counters(*args.summarize_counters)
        return
    if args.summarize_trace:
        summarize_trace(args.summarize_trace)
        return
    if args.summarize_extra:
        summarize_extra(*args.summarize_extra)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); rows are independent, so "
              "a multi-GPU run would shard rows with no exchange and is not implemented.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import workloads
    import paper_2608_17641_amd as rl
    from paper_2608_17641_amd.build import build

    build(force=False)  # only if nothing is built yet
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    # Everything below runs on a stream of its own (default priority), as a caller's training
    # loop would; on the null stream the same eager GAE steps took 0.1-0.2 us more each.
    torch.cuda.set_stream(torch.cuda.Stream(dev))
    if args.extra:
        if args.profile_pass:
            _PROFILE["on"] = True
        if args.variant:
            rl.testing_set_variant(args.variant)
        run_extra(dev, args.only)
        if args.profile_pass:
            src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
            dst = torch.empty_like(src)
            for _ in range(3):
                dst.copy_(src)
            torch.cuda.synchronize()
            if args.manifest:
                with open(args.manifest, "w") as f:
                    json.dump(_PROFILE["manifest"], f, indent=0)
            print(f"profile pass: {len(_PROFILE['manifest'])} workloads, 3 copies of {COPY_BYTES} B",
                  flush=True)
        return

    ro = workloads.make_rollout(N, T, seed=0, p_term=0.02, p_trunc=0.01)
    names = ("r", "v", "term", "trunc", "bv", "boot")
    base = {k: torch.from_numpy(ro[k]).to(dev) for k in names}
    S = max(1, args.sets)
    sets = []
    for _ in range(S):
        s = {k: v.clone() for k, v in base.items()}
        s["adv"] = torch.empty((N, T), dtype=torch.float32, device=dev)
        s["ret"] = torch.empty((N, T), dtype=torch.float32, device=dev)
        sets.append(s)

    def step(i):
        s = sets[i % S]
        rl.rlcs_gae(s["r"], s["v"], s["term"], s["trunc"], s["bv"], s["boot"], s["adv"], s["ret"],
                    gamma=GAMMA, lam=LAM)

    if args.profile_pass:
        profile_pass(step, args, dev)
        return
    if args.probe_sweep:
        for i in range(S):
            step(i)
        probe_sweep(step, sets, args.steps)
        return

    # parity of the timed configuration before timing
    import oracle
    step(0)
    torch.cuda.synchronize()
    o_adv, o_ret = oracle.gae(ro["r"], ro["v"], ro["term"], ro["trunc"], ro["bv"], ro["boot"],
                              gamma=GAMMA, lam=LAM)
    for got, ref in ((sets[0]["adv"], o_adv), (sets[0]["ret"], o_ret)):
        err = float(np.max(np.abs(got.double().cpu().numpy() - ref)))
        if err > 1e-5 * (1 + float(np.max(np.abs(ref)))):
            raise SystemExit(f"parity failure before timing: max err {err}")

    # Eager warm-up writes every set that the timed steps write into, so that their result can
    # be compared with an eager result of the same set.
    for i in range(eager_steps(args.warmup, args.steps, S)):
        step(i)
    torch.cuda.synchronize()
    check_set = replay_check_set(args.steps, S)
    eager_adv = sets[check_set]["adv"].clone()

    # The timed steps: eager launches for few steps, a HIP graph replay for more, queued behind
    # untimed steps that keep the GPU busy until the first timed one (so that host-side launch
    # cost, Python and ctypes, does not starve the GPU); each step is one rlcs_gae kernel launch
    # either way.
    start, end = TimingEvent(), TimingEvent()
    total_ms = time_steps(step, args.steps, start, end, sets=S)
    if not torch.equal(sets[check_set]["adv"], eager_adv):
        raise SystemExit("the timed steps' result differs from the eager launch")
    per_step_s = total_ms / 1e3 / args.steps
    nbytes = algorithmic_bytes(N, T)
    gbs = nbytes / per_step_s / 1e9

    out = {
        "metric": METRIC,
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(total_ms / args.steps, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "timing": f"{timing_protocol(args.steps)}: " + ("eager launches"
                  if timing_protocol(args.steps) == "eager" else "one HIP graph replay") +
                  f" on a stream of their own, queued behind {hold_calls(S)} untimed steps (one "
                  "graph replay); HIP events for timing only (hipEventDisableSystemFence) on that stream "
                  "around exactly K steps",
        "config": {"workload": f"GAE {N}x{T} fp32, term+trunc, bootstrap, cold HBM ({S} rotated input/output sets)",
                   "N": N, "T": T, "algorithmic_bytes": nbytes,
                   "gsteps_per_s": round(N * T / per_step_s / 1e9, 2),
                   "pct_of_peak": round(100 * gbs / PEAK_HBM_GBS, 2)},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 2), "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                     "traffic": recorded_traffic()},
    }
    out.update(copy_context(nbytes, per_step_s, sets, args))
    if not args.no_context:
        out.update(context(step, nbytes, args, start, end))
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(ro, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def copy_context(nbytes, per_step_s, sets, args):
    """The streaming ceiling beside the headline (also on stderr): probe_stream_gae over the same
    rotated sets, and the empty-launch floor. It launches only the probe kernels, so it also runs
    in kernel-trace runs (--no-context), whose trace then holds the probe's durations."""
    copies, empty_us = copy_reference(sets, args.steps)
    copy_us = min(copies.values())
    for threads, us in copies.items():
        print(f"copy reference (probe_stream_gae, {threads}-lane workgroups, GAE's 22 B per step, "
              f"cold): {us:.3f} us = {nbytes / us / 1e3:.1f} GB/s", file=sys.stderr)
    print(f"the GAE step takes {per_step_s * 1e6 / copy_us:.3f}x the faster copy's time; empty "
          f"launch {empty_us:.3f} us", file=sys.stderr)
    return {
        "copy_reference": {"kernel": "probe_stream_gae (libprobe.so): r, v, bv, term, trunc read "
                                     "and adv, ret written densely, 22 B per step, non-temporal "
                                     "16-byte vectors, same rotated sets, timed like the GAE steps, cold",
                           "us_64_lanes": round(copies[64], 3), "us_256_lanes": round(copies[256], 3),
                           "us": round(copy_us, 3), "GB/s": round(nbytes / copy_us / 1e3, 1),
                           "frac_of_peak": round(nbytes / copy_us / 1e3 / PEAK_HBM_GBS, 4),
                           "kernel_time_over_copy": round(per_step_s * 1e6 / copy_us, 3),
                           "empty_launch_us": round(empty_us, 3)},
    }


def context(step, nbytes, args, start, end):
    """Context figures next to the headline (also on stderr): the full-call time of one eager
    call through the Python binding by the paper's protocol (per-call events, median of 50, min
    over 5 trials), and the warm (cache-resident) step."""
    import torch
    trials = []
    for _ in range(5):
        ts = []
        for i in range(50):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            a.record(); step(i); b.record()
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        trials.append(float(np.median(ts)))
    full_us = min(trials) * 1e3
    print(f"full-call (per-call events, min of 5 medians): {full_us:.2f} us", file=sys.stderr)
    # Warm (context only): every step on set 0, Infinity-Cache resident after the first.
    warm_us = time_steps(lambda i: step(0), args.steps, start, end) * 1e3 / args.steps
    print(f"warm (one set, Infinity-Cache resident): {warm_us:.3f} us = {nbytes / warm_us / 1e3:.1f} GB/s "
          f"effective", file=sys.stderr)
    return {
        "full_call_us": round(full_us, 2),
        "warm": {"what": "same steps on one input/output set, Infinity-Cache resident (context only)",
                 "us": round(warm_us, 3), "GB/s": round(nbytes / warm_us / 1e3, 1)},
    }

if __name__ == "__main__":
    main()
