"""Host logic of bench.py: byte accounting and the rocprofv3 summaries (on small synthetic
profiler databases with the columns rocprofv3 writes)."""
import json
import os
import sqlite3

import pytest

import bench


def _db(path, kernels=(), counters=()):
    os.makedirs(path, exist_ok=True)
    con = sqlite3.connect(os.path.join(path, "run_results.db"))
    con.execute("create table kernels (dispatch_id integer, name text, start integer, "
                "\"end\" integer, duration integer)")
    con.execute("create table counters_collection (dispatch_id integer, kernel_name text, "
                "counter_name text, value real, grid_size integer)")
    for i, (n, d) in enumerate(kernels):
        con.execute("insert into kernels values (?, ?, ?, ?, ?)", (i, n, 1000 * i, 1000 * i + d, d))
    for i, (n, c, v, g) in enumerate(counters):
        con.execute("insert into counters_collection values (?, ?, ?, ?, ?)", (i, n, c, v, g))
    con.commit()
    con.close()


MARK = "void at::native::vectorized_elementwise_kernel<4, at::native::FillFunctor<short>>"
GAE = "void rlcs::rows_kernel<rlcs::GaeOp, float, 4, 4, true, true>(rlcs::Args, long, int)"
NORM = "void rlcs::masked_normalize_kernel(rlcs::MaskedArgs)"
MASK = "void rlcs::masked_gae_kernel<float, 4, 4, true, false, true, true>(rlcs::MaskedArgs)"
COPY = "__amd_rocclr_copyBuffer"
OTHER = "void at::native::index_select_kernel<float>"


def test_algorithmic_bytes_headline():
    # r, v, bv fp32; term, trunc u8; adv, ret fp32 -> 22 B per step, plus a 4-byte bootstrap per row
    assert bench.algorithmic_bytes(4096, 256) == 4096 * 256 * 22 + 4096 * 4
    assert bench.algorithmic_bytes(8, 128, trunc=False) == 8 * 128 * 17 + 8 * 4
    assert bench.extra_bytes("gae", 4096, 256, 4, True, True) == bench.algorithmic_bytes(4096, 256)
    assert bench.extra_bytes("elig_trace", 10, 10, 2, True, True) == 100 * (2 + 1 + 1 + 4)


def test_summarize_extra(tmp_path, capsys):
    # two workloads: two GAE calls, then one whitened masked call (two kernels); a parity call and
    # a torch kernel outside the markers must be ignored
    seq = [(GAE, 999), (MARK, 1), (GAE, 5000), (OTHER, 7), (GAE, 7000), (MARK, 1),
           (MASK, 999), (MARK, 1), (MASK, 3000), (NORM, 2000), (MARK, 1), (COPY, 9)]
    _db(str(tmp_path / "t"), kernels=seq)
    copy_kib = (bench.COPY_BYTES / 1024) / 2  # a counter that reads half the copy: scale 2
    fvals = {GAE: 100.0, MASK: 40.0, NORM: 10.0, MARK: 0.0, OTHER: 1.0}
    _db(str(tmp_path / "f"), counters=[(n, "FETCH_SIZE", fvals.get(n, copy_kib), 1) for n, _ in seq])
    _db(str(tmp_path / "w"), counters=[(n, "WRITE_SIZE", fvals.get(n, bench.COPY_BYTES / 1024), 1)
                                       for n, _ in seq])
    man = [{"label": "a", "name": "gae", "calls": 2, "bytes": 4_000_000, "steps": 10},
           {"label": "b", "name": "gae_masked_norm", "calls": 1, "bytes": 1_000_000, "steps": 10}]
    mp = tmp_path / "m.json"
    mp.write_text(json.dumps(man))
    bench.summarize_extra(str(tmp_path / "t"), str(tmp_path / "f"), str(tmp_path / "w"), str(mp))
    out = capsys.readouterr().out.splitlines()
    assert "FETCH_SIZE_scale: 2.0000" in out and "WRITE_SIZE_scale: 1.0000" in out
    # per workload: label, estimator, kernel (several words), avg_us, GB/s, %peak, traffic, alg, ratio
    per_call = [l.split() for l in out if l[:2] in ("a ", "b ") and l.split()[2] != "-"]
    assert len(per_call) == 2
    # workload a: (5 + 7) / 2 = 6 us per call; traffic (2 * 100 + 100) KiB per call
    assert per_call[0][0] == "a" and float(per_call[0][-6]) == pytest.approx(6.0)
    assert int(per_call[0][-3]) == 300 * 1024
    # workload b: both kernels of the call, 3 + 2 us; traffic (2 * 50 + 50) KiB
    assert per_call[1][0] == "b" and float(per_call[1][-6]) == pytest.approx(5.0)
    assert int(per_call[1][-3]) == 150 * 1024


def test_summarize_extra_rejects_mismatch(tmp_path):
    seq = [(MARK, 1), (GAE, 5000), (MARK, 1), (COPY, 9)]
    for d, kind in (("t", None), ("f", "FETCH_SIZE"), ("w", "WRITE_SIZE")):
        if kind is None:
            _db(str(tmp_path / d), kernels=seq)
        else:
            _db(str(tmp_path / d), counters=[(n, kind, 1.0, 1) for n, _ in seq])
    mp = tmp_path / "m.json"
    mp.write_text(json.dumps([{"label": "a", "name": "x", "calls": 1, "bytes": 1, "steps": 1}] * 2))
    with pytest.raises(SystemExit):
        bench.summarize_extra(str(tmp_path / "t"), str(tmp_path / "f"), str(tmp_path / "w"), str(mp))


def test_bench_refuses_more_than_one_gpu():
    """The bench measures one GPU: any other --gpus exits with status 2 and says why, before
    touching a GPU."""
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(os.path.dirname(bench.__file__), "bench.py"),
                        "--gpus", "2"], capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


@pytest.mark.parametrize("steps,warmup,sets", [(20, 5, 32), (2000, 200, 32), (1, 0, 32), (5, 100, 32),
                                               (64, 5, 32), (33, 0, 32), (7, 3, 1)])
def test_replay_check_set_was_written_eagerly(steps, warmup, sets):
    """The timed steps' result is compared with the eager result of the same set: that set must be
    one the eager calls before timing wrote (the driver's --steps 20 --warmup 5 among them)."""
    eager = {i % sets for i in range(bench.eager_steps(warmup, steps, sets))}
    replayed = {i % sets for i in range(steps)}
    assert replayed <= eager
    assert bench.replay_check_set(steps, sets) in eager
    assert bench.eager_steps(warmup, steps, sets) >= warmup


def test_timing_protocol():
    """Few timed steps are launched eagerly, many are replayed from one graph."""
    assert bench.timing_protocol(20) == "eager"
    assert bench.timing_protocol(bench.EAGER_MAX_STEPS) == "eager"
    assert bench.timing_protocol(bench.EAGER_MAX_STEPS + 1) == "graph"
    assert bench.timing_protocol(2000) == "graph"


@pytest.mark.parametrize("sets", [1, 3, 7, 20, 32, 33, 5000])
def test_hold_ends_a_whole_rotation(sets):
    """The untimed calls before the timed ones number at least HOLD_CALLS and a whole number of
    rotations, so the first timed call (set 0) follows the hold's call on the last set, and its
    own set was last touched a full rotation before."""
    h = bench.hold_calls(sets)
    assert h >= bench.HOLD_CALLS and h % sets == 0 and h - sets < max(bench.HOLD_CALLS, sets)
    assert (h - 1) % sets == sets - 1


def test_probe_library_rejects_bad_shapes():
    """The streaming probe's argument checks run before any HIP call (no GPU needed): every
    combination outside the supported shapes returns 1."""
    import ctypes
    import os
    from paper_2608_17641_amd.build import PROBE_LIB
    if not os.path.exists(PROBE_LIB):
        pytest.skip("libprobe.so not built")
    lib = bench.probe_lib()
    fake = [ctypes.c_void_p(0x10000 * (k + 1)) for k in range(7)]  # 16-byte aligned, never dereferenced
    n = 4096
    for threads, per_lane, groups, dep in ((128, 1, 0, 0), (64, 3, 0, 0), (64, 2, 512, 0),
                                           (64, 1, 512, 1), (64, 1, -1, 0), (64, 1, 0, 2)):
        assert lib.probe_stream_gae_shape(*fake, n, threads, per_lane, groups, dep, None) == 1
    assert lib.probe_stream_gae_shape(*fake, 4098, 64, 1, 0, 0, None) == 1   # not whole vectors
    assert lib.probe_stream_gae_shape(None, *fake[1:], n, 64, 1, 0, 0, None) == 1
    assert lib.probe_stream_gae_shape(*fake, 0, 64, 1, 0, 0, None) == 0      # nothing to stream


@pytest.mark.parametrize("nbytes,sets", [(17440, 32), (2899968, 32), (23085056, 16),
                                         (2147614720, 1), (10**12, 3)])
def test_extra_calls(nbytes, sets):
    """Every --extra row times 20 to 2000 calls (more only to end on a whole rotation), a whole
    number of rotations over its sets, and at least about 8 GB unless capped at 2000."""
    k = bench.extra_calls(nbytes, sets)
    assert k % sets == 0 and 20 <= k < 2000 + sets
    assert k >= 2000 or k * nbytes >= 8e9
