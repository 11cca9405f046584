"""GPU parity of the column scans through the C ABI: the time-major [T, N] entry points of every
estimator and the F-vector eligibility traces, against the fp64 oracle on the same seeded
inputs, under every kernel variant (64-column walks, columns split over workgroups, narrow
column groups of 16 or 32 columns per workgroup, narrow groups split over workgroups). Bar: max |gpu - oracle| <= tol * (1 + max
|oracle|) per output, tol = 1e-5 for float32 inputs and 1e-3 for bfloat16 inputs."""
import contextlib

import numpy as np
import pytest

from cases import TOL, assert_parity, to_device
import oracle
import workloads

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2608_17641_amd as rl  # noqa: E402

DEV = torch.device("cuda:0")
G, L = 0.99, 0.95


@contextlib.contextmanager
def variant(v):
    rl.testing_set_variant(v)
    try:
        yield
    finally:
        rl.testing_set_variant(0)


def strided(t, ld):
    """`t` [T, N] copied into the first N columns of a [T, ld] buffer (a strided view)."""
    if ld == t.shape[1]:
        return t
    buf = torch.full((t.shape[0], ld), 7, dtype=t.dtype, device=t.device)
    buf[:, : t.shape[1]] = t
    return buf[:, : t.shape[1]]


TM_ESTIMATORS = ("gae", "vtrace", "retrace", "td_lambda", "discounted", "elig_trace",
                 "prefix_ends", "prefix_starts")


def run_strided(name, d, *, trunc=True, boot=True, ws=None):
    """Estimator `name` on [N, T] views `d` of any layout, through the strided entry points."""
    tr = d["trunc"] if trunc else None
    bv = d["bv"] if trunc else None
    bt = d["boot"] if boot else None
    if name == "gae":
        a, b = rl.rlcs_gae_strided(d["r"], d["v"], d["term"], tr, bv, bt, gamma=G, lam=L, ws=ws)
        return {"adv": a, "ret": b}
    if name == "vtrace":
        a, b = rl.rlcs_vtrace_strided(d["r"], d["v"], d["log_rho"], d["term"], tr, bv, bt, gamma=G,
                                      rho_bar=1.0, c_bar=0.9, ws=ws)
        return {"vs": a, "pg": b}
    if name == "retrace":
        a, b = rl.rlcs_retrace_strided(d["r"], d["q"], d["eq"], d["log_rho"], d["term"], tr, bv, bt,
                                       gamma=G, lam=L, c_bar=1.0, ws=ws)
        return {"delta": a, "q_ret": b}
    if name == "td_lambda":
        return {"ret": rl.rlcs_td_lambda_strided(d["r"], d["v"], d["term"], tr, bv, bt, gamma=G,
                                                 lam=L, ws=ws)}
    if name == "discounted":
        return {"ret": rl.rlcs_discounted_strided(d["r"], d["term"], tr, bv, bt, gamma=G, ws=ws)}
    if name == "elig_trace":
        return {"z": rl.rlcs_elig_trace_strided(d["x"], d["term"], tr, gamma=G, lam=L, ws=ws)}
    b = "starts_at" if name == "prefix_starts" else "ends_at"
    return {"c": rl.rlcs_episodic_prefix_strided(d["x"], d["term"], tr, boundary=b, ws=ws)}


def run_tm(name, d, *, trunc=True, boot=True, ws=None):
    """Time-major [T, N] tensors in `d`: passed as their [N, T] transposes; outputs [T, N]."""
    dt = {k: (v.t() if v.dim() == 2 else v) for k, v in d.items()}
    out = run_strided(name, dt, trunc=trunc, boot=boot, ws=ws)
    return {k: (None if v is None else v.t()) for k, v in out.items()}


def ref_tm(name, ro, *, trunc=True, boot=True):
    tm = oracle.time_major
    tr = ro["trunc"] if trunc else None
    bv = ro["bv"] if trunc else None
    bt = ro["boot"] if boot else None
    if name == "gae":
        a, b = tm(oracle.gae, ro["r"], ro["v"], ro["term"], tr, bv, bt, gamma=G, lam=L)
        return {"adv": a, "ret": b}
    if name == "vtrace":
        a, b = tm(oracle.vtrace, ro["r"], ro["v"], ro["log_rho"], ro["term"], tr, bv, bt,
                  gamma=G, rho_bar=1.0, c_bar=0.9)
        return {"vs": a, "pg": b}
    if name == "retrace":
        a, b = tm(oracle.retrace, ro["r"], ro["q"], ro["eq"], ro["log_rho"], ro["term"], tr, bv,
                  bt, gamma=G, lam=L, c_bar=1.0)
        return {"delta": a, "q_ret": b}
    if name == "td_lambda":
        return {"ret": tm(oracle.td_lambda, ro["r"], ro["v"], ro["term"], tr, bv, bt, gamma=G,
                          lam=L)}
    if name == "discounted":
        return {"ret": tm(oracle.discounted, ro["r"], ro["term"], tr, bv, bt, gamma=G)}
    if name == "elig_trace":
        return {"z": tm(oracle.elig_trace, ro["x"], ro["term"], tr, gamma=G, lam=L)}
    b = "starts_at" if name == "prefix_starts" else "ends_at"
    return {"c": tm(oracle.episodic_prefix, ro["x"], ro["term"], tr, boundary=b)}


def device_tm(ro, ld=None):
    d = {}
    for k, v in ro.items():
        t = to_device(v, DEV)
        d[k] = strided(t, ld) if (ld is not None and t.dim() == 2) else t
    return d


@pytest.mark.parametrize("v", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("T,N", [(1, 1), (7, 3), (33, 64), (256, 100), (1000, 65), (4097, 5)])
def test_time_major_every_estimator(T, N, v):
    ro = workloads.make_rollout_time_major(T, N, seed=T * 7 + N, p_term=0.05, p_trunc=0.05)
    d = device_tm(ro)
    ws = rl.make_workspace_columns(N, T, DEV)
    with variant(v):
        for name in TM_ESTIMATORS:
            out = run_tm(name, d, ws=ws)
            torch.cuda.synchronize()
            assert_parity(out, ref_tm(name, ro), TOL["f32"], label=f"tm {name} T={T} N={N} v={v}")
    assert int(ws[8:12].view(torch.int32).item()) == 0


@pytest.mark.parametrize("v", [1, 2, 3, 4])
def test_time_major_bf16_plain_and_strided(v):
    T, N = 300, 130
    ro = workloads.make_rollout_time_major(T, N, seed=3, dtype="bf16", p_term=0.03, p_trunc=0.03)
    ws = rl.make_workspace_columns(N, T, DEV)
    with variant(v):
        for ld in (None, 160):
            d = device_tm(ro, ld)
            for name in TM_ESTIMATORS:
                out = run_tm(name, d, ws=ws)
                torch.cuda.synchronize()
                assert_parity(out, ref_tm(name, ro), TOL["bf16"], label=f"tm bf16 {name} ld={ld}")
                if ld is not None:
                    for o in out.values():
                        assert o.stride() == (ld, 1)  # [T, N] view of [T, ld] storage
            for name in ("gae", "discounted", "elig_trace"):
                out = run_tm(name, d, trunc=False, boot=False, ws=ws)
                torch.cuda.synchronize()
                assert_parity(out, ref_tm(name, ro, trunc=False, boot=False), TOL["bf16"],
                              label=f"tm bf16 plain {name} ld={ld}")


def test_time_major_strided_padding_untouched():
    """Columns n >= N of a strided [T, ld] output are never written."""
    T, N, ld = 70, 40, 48
    ro = workloads.make_rollout_time_major(T, N, seed=9)
    d = device_tm(ro, ld)
    adv_buf = torch.full((T, ld), -3.0, device=DEV)
    ret_buf = torch.full((T, ld), -4.0, device=DEV)
    rl.rlcs_gae_strided(d["r"].t(), d["v"].t(), d["term"].t(), d["trunc"].t(), d["bv"].t(),
                        d["boot"], adv_buf[:, :N].t(), ret_buf[:, :N].t(), gamma=G, lam=L)
    torch.cuda.synchronize()
    assert torch.all(adv_buf[:, N:] == -3.0) and torch.all(ret_buf[:, N:] == -4.0)
    assert_parity({"adv": adv_buf[:, :N], "ret": ret_buf[:, :N]}, ref_tm("gae", ro), TOL["f32"],
                  label="tm strided")


@pytest.mark.parametrize("v", [0, 1, 2, 3, 4])
def test_time_major_headline_shape(v):
    """GAE on the 4096-environment x 256-step workload stored time-major, whole."""
    T, N = 256, 4096
    ro = workloads.make_rollout_time_major(T, N, seed=0, p_term=0.02, p_trunc=0.01)
    d = device_tm(ro)
    ws = rl.make_workspace_columns(N, T, DEV)
    with variant(v):
        out = run_tm("gae", d, ws=ws)
        torch.cuda.synchronize()
    assert_parity(out, ref_tm("gae", ro), TOL["f32"], label=f"tm 256x4096 v={v}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("T,N,ld", [(1, 17, None), (64, 1000, None), (65, 1000, 1030), (300, 1000, None),
                                    (64, 1600, 1700), (1100, 4100, None), (2000, 530, 600),
                                    (5000, 4096, None)])
def test_time_major_narrow_groups(T, N, ld, dtype):
    """Narrow column groups (16 float32 or 32 bfloat16 columns per workgroup, whole columns):
    group counts below, at and above multiples of 64 (runs of 64 workgroups deal eight
    consecutive groups to each XCD; the rest keep their order), one 4-wave chunk, 16-wave chunks
    walked with and without the load pipeline, strided buffers. Forced here; the automatic choice (columns of at most
    256 steps in at least 256 groups) runs in the headline-shape test."""
    ro = workloads.make_rollout_time_major(T, N, seed=T + N, dtype=dtype, p_term=0.03, p_trunc=0.03)
    d = device_tm(ro, ld)
    with variant(3):
        for name in (TM_ESTIMATORS if T * N <= 2_000_000 else ("gae", "elig_trace")):
            out = run_tm(name, d)
            torch.cuda.synchronize()
            assert_parity(out, ref_tm(name, ro), TOL[dtype], label=f"narrow {name} T={T} N={N} {dtype}")


def test_time_major_deterministic_and_workspace_reuse():
    T, N = 500, 70
    ro = workloads.make_rollout_time_major(T, N, seed=4)
    d = device_tm(ro)
    ws = rl.make_workspace_columns(4 * N, 2 * T, DEV)
    with variant(2):
        a1, _ = rl.rlcs_gae_strided(d["r"].t(), d["v"].t(), d["term"].t(), d["trunc"].t(),
                                    d["bv"].t(), d["boot"], gamma=G, lam=L, ws=ws)
        for T2, N2 in ((37, 3), (999, 200), (64, 64)):
            ro2 = workloads.make_rollout_time_major(T2, N2, seed=T2)
            out = run_tm("vtrace", device_tm(ro2), ws=ws)
            torch.cuda.synchronize()
            assert_parity(out, ref_tm("vtrace", ro2), TOL["f32"], label=f"reuse {T2}x{N2}")
        a2, _ = rl.rlcs_gae_strided(d["r"].t(), d["v"].t(), d["term"].t(), d["trunc"].t(),
                                    d["bv"].t(), d["boot"], gamma=G, lam=L, ws=ws)
        torch.cuda.synchronize()
    assert torch.equal(a1, a2)
    assert int(ws[8:12].view(torch.int32).item()) == 0


def test_time_major_no_flags_long_lookback():
    """No flags at all: every split tile composes the maps of all later tiles of its column."""
    T, N = 3000, 17
    ro = workloads.make_rollout_time_major(T, N, seed=12, p_term=0.0, p_trunc=0.0)
    d = device_tm(ro)
    ws = rl.make_workspace_columns(N, T, DEV)
    with variant(2):
        for name in ("discounted", "prefix_ends"):
            out = run_tm(name, d, trunc=False, ws=ws)
            torch.cuda.synchronize()
            assert_parity(out, ref_tm(name, ro, trunc=False), TOL["f32"], label=f"no flags {name}")


@pytest.mark.parametrize("v", [0, 4])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_block_aggregates_with_rare_flags(dtype, v):
    """Columns of 256 split tiles with gamma * lambda = 1 (c_bar = inf for V-Trace) and rare
    flags (episodes of about 250 steps): look-backs run past their first tiles into block
    aggregates, some of which hold an episode edge. Against the oracle, and bitwise run to run;
    vector traces of 128 tiles the same way. Automatic choice (tiles of 64 columns) and split
    narrow groups."""
    T, N = 16384, 70
    ro = workloads.make_rollout_time_major(T, N, seed=21, dtype=dtype, p_term=0.002, p_trunc=0.002)
    d = {k: (v.t() if v.dim() == 2 else v) for k, v in device_tm(ro).items()}
    ws = rl.make_workspace_columns(N, T, DEV)
    tm = oracle.time_major
    calls = {
        "gae": (lambda: rl.rlcs_gae_strided(d["r"], d["v"], d["term"], d["trunc"], d["bv"], d["boot"],
                                            gamma=1.0, lam=1.0, ws=ws),
                lambda: tm(oracle.gae, ro["r"], ro["v"], ro["term"], ro["trunc"], ro["bv"], ro["boot"],
                           gamma=1.0, lam=1.0)),
        "vtrace": (lambda: rl.rlcs_vtrace_strided(d["r"], d["v"], d["log_rho"], d["term"], d["trunc"],
                                                  d["bv"], d["boot"], gamma=1.0, rho_bar=1.0,
                                                  c_bar=float("inf"), ws=ws),
                   lambda: tm(oracle.vtrace, ro["r"], ro["v"], ro["log_rho"], ro["term"], ro["trunc"],
                              ro["bv"], ro["boot"], gamma=1.0, rho_bar=1.0, c_bar=float("inf"))),
        "elig_trace": (lambda: (rl.rlcs_elig_trace_strided(d["x"], d["term"], d["trunc"], gamma=1.0,
                                                           lam=1.0, ws=ws),),
                       lambda: (tm(oracle.elig_trace, ro["x"], ro["term"], ro["trunc"], gamma=1.0,
                                   lam=1.0),)),
        "prefix": (lambda: (rl.rlcs_episodic_prefix_strided(d["x"], d["term"], d["trunc"],
                                                            boundary="ends_at", ws=ws),),
                   lambda: (tm(oracle.episodic_prefix, ro["x"], ro["term"], ro["trunc"],
                               boundary="ends_at"),)),
    }
    for name, (gpu, ref) in calls.items():
        with variant(v):
            first = [o.clone() for o in gpu() if o is not None]
            again = [o for o in gpu() if o is not None]
            torch.cuda.synchronize()
        for a, b in zip(first, again):
            assert torch.equal(a, b), f"{name}: not bitwise reproducible"
        expect = [r for r in ref() if r is not None]
        assert_parity({str(i): o.t() for i, o in enumerate(first)},
                      {str(i): r for i, r in enumerate(expect)}, TOL[dtype],
                      label=f"block aggregates {name} {dtype}")
    assert int(ws[8:12].view(torch.int32).item()) == 0
    vr = workloads.make_vector_trace(2, 8192, 40, seed=22, p_term=0.002, p_trunc=0.002)
    dv = {k: to_device(v, DEV) for k, v in vr.items()}
    wsv = rl.make_workspace_columns(2 * 40, 8192, DEV)
    with variant(v):
        z = rl.rlcs_elig_trace_vec(dv["x"], dv["term"], dv["trunc"], gamma=1.0, lam=1.0, ws=wsv)
        torch.cuda.synchronize()
    zr = oracle.elig_trace_vec(vr["x"], vr["term"], vr["trunc"], gamma=1.0, lam=1.0)
    assert_parity({"z": z}, {"z": zr}, TOL["f32"], label="block aggregates vector traces")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("T,N", [(4096, 128), (1024, 64), (1024, 40), (8192, 64), (512, 7)])
def test_narrow_split_dealt_tiles(T, N, dtype):
    """Split narrow groups with the tiles dealt statically to XCDs, the automatic choice for these
    shapes in float32 (a grid resident at once, a multiple of 8 tiles per group, 128-step tiles
    or at most 16 tiles; ragged groups): every estimator against the oracle, and bitwise against
    the same tiles drawn in arrival order (variant 4)."""
    ro = workloads.make_rollout_time_major(T, N, seed=T + 3 * N, dtype=dtype, p_term=0.01,
                                           p_trunc=0.01)
    d = device_tm(ro)
    ws = rl.make_workspace_columns(N, T, DEV)
    for name in TM_ESTIMATORS:
        dealt = {k: o.clone() for k, o in run_tm(name, d, ws=ws).items()}
        with variant(4):
            drawn = run_tm(name, d, ws=ws)
        torch.cuda.synchronize()
        for k in dealt:
            assert torch.equal(dealt[k], drawn[k]), f"{name} {k}: dealt and drawn tiles differ"
        assert_parity(dealt, ref_tm(name, ro), TOL[dtype], label=f"dealt {name} T={T} N={N} {dtype}")
    assert int(ws[8:12].view(torch.int32).item()) == 0


@pytest.mark.parametrize("v", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("trunc", [False, True])
def test_forward_column_scans_without_termination_array(v, trunc):
    """Forward column scans given no termination array (truncation given or not): a kernel reads
    a missing flag array from the data input instead and must drop what it reads there, also for
    the previous step's flag that a lane takes from memory (once read as a flag, a data byte cut
    the carry at every lane boundary). Time-major eligibility traces and prefix sums, and vector
    traces on the column scans."""
    T, N = 1000, 65
    ro = workloads.make_rollout_time_major(T, N, seed=41, p_term=0.05, p_trunc=0.05)
    d = device_tm(ro)
    ws = rl.make_workspace_columns(N, T, DEV)
    tr_d = d["trunc"].t() if trunc else None
    tr_o = ro["trunc"] if trunc else None
    with variant(v):
        z = rl.rlcs_elig_trace_strided(d["x"].t(), None, tr_d, gamma=G, lam=L, ws=ws)
        c = rl.rlcs_episodic_prefix_strided(d["x"].t(), None, tr_d, boundary="ends_at", ws=ws)
        torch.cuda.synchronize()
    zr = oracle.time_major(oracle.elig_trace, ro["x"], None, tr_o, gamma=G, lam=L)
    cr = oracle.time_major(oracle.episodic_prefix, ro["x"], None, tr_o, boundary="ends_at")
    assert_parity({"z": z.t()}, {"z": zr}, TOL["f32"], label=f"time-major elig, no term, v={v}")
    assert_parity({"c": c.t()}, {"c": cr}, TOL["f32"], label=f"time-major prefix, no term, v={v}")
    rv = workloads.make_vector_trace(300, 605, 4, seed=42, p_term=0.05, p_trunc=0.05)
    wsv = rl.make_workspace_columns(300 * 4, 605, DEV)
    with variant(v):
        zv = rl.rlcs_elig_trace_vec(to_device(rv["x"], DEV), None,
                                    to_device(rv["trunc"], DEV) if trunc else None,
                                    gamma=G, lam=L, ws=wsv)
        torch.cuda.synchronize()
    zvr = oracle.elig_trace_vec(rv["x"], None, rv["trunc"] if trunc else None, gamma=G, lam=L)
    assert_parity({"z": zv}, {"z": zvr}, TOL["f32"], label=f"vector traces, no term, v={v}")


# ---------------------------------------------------------------- vector eligibility traces

def run_vec(ro, *, trunc=True, ws=None):
    d = {k: to_device(v, DEV) for k, v in ro.items()}
    z = rl.rlcs_elig_trace_vec(d["x"], d["term"], d["trunc"] if trunc else None, gamma=G, lam=L,
                               ws=ws)
    torch.cuda.synchronize()
    ref = oracle.elig_trace_vec(ro["x"], ro["term"], ro["trunc"] if trunc else None, gamma=G,
                                lam=L)
    return z, ref


@pytest.mark.parametrize("v", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("N,T,F", [(1, 1, 1), (3, 7, 5), (64, 256, 16), (7, 1000, 33),
                                   (2, 4097, 3), (5, 40, 300), (1, 33, 64)])
def test_elig_trace_vec_shapes(N, T, F, v):
    ro = workloads.make_vector_trace(N, T, F, seed=N + T + F, p_term=0.04, p_trunc=0.04)
    ws = rl.make_workspace_columns(N * F, T, DEV)
    with variant(v):
        z, ref = run_vec(ro, ws=ws)
        assert_parity({"z": z}, {"z": ref}, TOL["f32"], label=f"vec {N}x{T}x{F} v={v}")
        z, ref = run_vec(ro, trunc=False, ws=ws)
        assert_parity({"z": z}, {"z": ref}, TOL["f32"], label=f"vec plain {N}x{T}x{F} v={v}")


def test_elig_trace_vec_bf16_and_large():
    ro = workloads.make_vector_trace(200, 129, 24, seed=5, dtype="bf16")
    z, ref = run_vec(ro)
    assert_parity({"z": z}, {"z": ref}, TOL["bf16"], label="vec bf16")
    ro = workloads.make_vector_trace(4096, 64, 16, seed=6)
    z, ref = run_vec(ro)
    assert_parity({"z": z}, {"z": ref}, TOL["f32"], label="vec 4096x64x16")


@pytest.mark.parametrize("N,T,F,dtype", [
    (256, 2048, 4, "f32"), (257, 1999, 4, "f32"), (300, 65, 8, "f32"), (256, 511, 16, "f32"),
    (256, 512, 16, "f32"), (260, 65, 16, "f32"), (256, 255, 32, "f32"), (256, 33, 64, "f32"),
    (256, 64, 128, "f32"), (256, 31, 256, "f32"), (256, 32, 256, "f32"), (1000, 100, 16, "f32"),
    (256, 1024, 8, "bf16"), (256, 257, 16, "bf16"), (256, 63, 64, "bf16"), (256, 16, 512, "bf16"),
    (256, 5, 512, "bf16"),
    # short rows, several to a workgroup (the last one partly filled)
    (601, 32, 16, "f32"), (3100, 5, 16, "f32"), (33000, 1, 8, "f32"), (600, 7, 64, "f32"),
    (257, 33, 16, "f32"), (5001, 13, 4, "f32"), (300, 3, 512, "bf16"), (33001, 2, 8, "bf16"),
    (1000, 9, 32, "bf16"),
    # 8 and 16 waves to a row (LDS beyond 64 KB)
    (256, 1024, 16, "f32"), (256, 777, 16, "f32"), (256, 4096, 4, "f32"), (256, 64, 256, "f32"),
    (256, 2048, 8, "bf16"), (256, 1000, 16, "bf16")])
def test_elig_trace_vec_rows(N, T, F, dtype):
    """Shapes the row kernel of vector traces takes (F a multiple of the vector width with a
    power-of-two number of vectors, at least 256 workgroups, every wave count it uses, one row
    or several short ones to a workgroup, T a multiple of 4 or not): with and without
    truncation, and with no flags at all."""
    ro = workloads.make_vector_trace(N, T, F, seed=N + T + F, dtype=dtype, p_term=0.04,
                                     p_trunc=0.04)
    z, ref = run_vec(ro)
    assert_parity({"z": z}, {"z": ref}, TOL[dtype], label=f"vec rows {N}x{T}x{F} {dtype}")
    z, ref = run_vec(ro, trunc=False)
    assert_parity({"z": z}, {"z": ref}, TOL[dtype], label=f"vec rows plain {N}x{T}x{F} {dtype}")
    d = to_device(ro["x"], DEV)
    z = rl.rlcs_elig_trace_vec(d, None, None, gamma=G, lam=L)
    torch.cuda.synchronize()
    ref = oracle.elig_trace_vec(ro["x"], None, None, gamma=G, lam=L)
    assert_parity({"z": z}, {"z": ref}, TOL[dtype], label=f"vec rows no flags {N}x{T}x{F} {dtype}")


def test_elig_trace_vec_one_feature_matches_scalar_entry_point():
    """F = 1 and the scalar row-major trace compute the same recurrence on the same data."""
    ro = workloads.make_vector_trace(33, 500, 1, seed=8)
    d = {k: to_device(v, DEV) for k, v in ro.items()}
    zv = rl.rlcs_elig_trace_vec(d["x"], d["term"], d["trunc"], gamma=G, lam=L)[:, :, 0]
    zs = rl.rlcs_elig_trace(d["x"][:, :, 0].contiguous(), d["term"], d["trunc"], gamma=G, lam=L)
    torch.cuda.synchronize()
    ref = oracle.elig_trace(ro["x"][:, :, 0], ro["term"], ro["trunc"], gamma=G, lam=L)
    assert_parity({"z": zv}, {"z": ref}, TOL["f32"], label="vec F=1")
    assert_parity({"z": zs}, {"z": ref}, TOL["f32"], label="scalar")


def test_workspace_shared_by_row_major_and_column_calls():
    """One workspace serves split row-major calls and split column calls in any order."""
    from cases import gpu_run, make_inputs, oracle_run, device_inputs
    n = max(rl.rlcs_workspace_size(64, 8192), rl.rlcs_workspace_size_columns(200, 999),
            rl.rlcs_workspace_size_columns(16 * 40, 300))
    ws = torch.zeros(n, dtype=torch.uint8, device=DEV)
    with variant(2):
        for rnd in range(2):
            ro = make_inputs("gae", 64, 8192, seed=rnd)
            out = gpu_run("gae", device_inputs(ro, DEV), ws=ws)
            torch.cuda.synchronize()
            assert_parity(out, oracle_run("gae", ro), TOL["f32"], label=f"row-major {rnd}")
            ro2 = workloads.make_rollout_time_major(999, 200, seed=rnd)
            out = run_tm("vtrace", device_tm(ro2), ws=ws)
            torch.cuda.synchronize()
            assert_parity(out, ref_tm("vtrace", ro2), TOL["f32"], label=f"time-major {rnd}")
            ro3 = workloads.make_vector_trace(16, 300, 40, seed=rnd)
            z, ref = run_vec(ro3, ws=ws)
            assert_parity({"z": z}, {"z": ref}, TOL["f32"], label=f"vector {rnd}")
            ro4 = make_inputs("elig_trace", 3, 5000, seed=rnd)
            out = gpu_run("elig_trace", device_inputs(ro4, DEV), ws=ws)
            torch.cuda.synchronize()
            assert_parity(out, oracle_run("elig_trace", ro4), TOL["f32"], label=f"row-major elig {rnd}")
    assert int(ws[8:12].view(torch.int32).item()) == 0


def strided_rows(t, ld):
    """`t` [N, T] copied into the first T steps of [N, ld] rows (a view with stride (ld, 1))."""
    buf = torch.full((t.shape[0], ld), 5, dtype=t.dtype, device=t.device)
    buf[:, : t.shape[1]] = t
    return buf[:, : t.shape[1]]


@pytest.mark.parametrize("v", [0, 1, 2, 4])
@pytest.mark.parametrize("N,T,ld", [(1, 1, 3), (9, 33, 40), (100, 256, 300), (5, 1000, 1001)])
def test_strided_rows_every_estimator(N, T, ld, v):
    """Row-major rows with a row stride above T (the first T steps of wider rows)."""
    ro = workloads.make_rollout(N, T, seed=N + T, p_term=0.05, p_trunc=0.05)
    d = {k: (strided_rows(to_device(a, DEV), ld) if a.ndim == 2 else to_device(a, DEV))
         for k, a in ro.items()}
    ws = rl.make_workspace_columns(N, T, DEV)
    from cases import oracle_run
    with variant(v):
        for name in TM_ESTIMATORS:
            out = run_strided(name, d, ws=ws)
            torch.cuda.synchronize()
            for o in out.values():
                assert o.stride() == (ld, 1) or T == 1
            assert_parity(out, oracle_run(name, ro, gamma=G, lam=L, c_bar=1.0 if name != "vtrace" else 0.9),
                          TOL["f32"], label=f"strided rows {name} {N}x{T} ld={ld} v={v}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("N,T,ld", [(100, 256, 320), (37, 64, 72), (6, 4096, 4160), (300, 8, 16),
                                    (3, 2048, 2056), (25, 33, 37), (9, 1001, 1003), (40, 100, 128)])
def test_strided_rows_vector_path(N, T, ld, dtype):
    """Aligned storage: the vector path of the rows kernel, lane by lane (lanes whose steps reach
    into the gaps between rows go element-wise, lanes wholly in a gap skip). Every estimator
    against the oracle; the gaps of the outputs are never written."""
    ro = workloads.make_rollout(N, T, seed=N * 7 + T, dtype=dtype, p_term=0.05, p_trunc=0.05)
    d = {k: (strided_rows(to_device(a, DEV), ld) if a.ndim == 2 else to_device(a, DEV))
         for k, a in ro.items()}
    from cases import oracle_run
    for name in TM_ESTIMATORS:
        out = run_strided(name, d)
        torch.cuda.synchronize()
        assert_parity(out, oracle_run(name, ro, gamma=G, lam=L, c_bar=1.0 if name != "vtrace" else 0.9),
                      TOL[dtype], label=f"strided rows {name} {N}x{T} ld={ld} {dtype}")
    bufs = [torch.full((N, ld), -3.0, device=DEV) for _ in range(2)]
    adv, ret = rl.rlcs_gae_strided(d["r"], d["v"], d["term"], d["trunc"], d["bv"], d["boot"],
                                   bufs[0][:, :T], bufs[1][:, :T], gamma=G, lam=L)
    torch.cuda.synchronize()
    assert_parity({"adv": adv, "ret": ret}, oracle_run("gae", ro, gamma=G, lam=L),
                  TOL[dtype], label=f"strided rows gae, given outputs {N}x{T} ld={ld} {dtype}")
    for b in bufs:
        assert bool((b[:, T:] == -3.0).all())


def test_strided_dense_layout_runs_the_row_major_path():
    """stride (T, 1) is the plain row-major layout: same results as the row-major entry point,
    bit for bit."""
    ro = workloads.make_rollout(64, 300, seed=3)
    d = {k: to_device(a, DEV) for k, a in ro.items()}
    a1, r1 = rl.rlcs_gae_strided(d["r"], d["v"], d["term"], d["trunc"], d["bv"], d["boot"], gamma=G, lam=L)
    a2, r2 = rl.rlcs_gae(d["r"], d["v"], d["term"], d["trunc"], d["bv"], d["boot"], gamma=G, lam=L)
    torch.cuda.synchronize()
    assert torch.equal(a1, a2) and torch.equal(r1, r2)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("T,N,ld", [(4096, 64, None), (2048, 128, 136), (65, 16, None), (129, 1, 3),
                                    (1000, 33, None), (8192, 48, 50), (20000, 32, None)])
def test_time_major_narrow_split_auto(T, N, ld, dtype):
    """Few long columns (fewer than 256 tiles of 64 columns by 64 steps, or fewer than 64
    columns): the automatic choice splits narrow groups along T (64- and 128-step tiles).
    Against the oracle, and bitwise run to run."""
    ro = workloads.make_rollout_time_major(T, N, seed=T + 3 * N, dtype=dtype, p_term=0.01,
                                           p_trunc=0.01)
    d = device_tm(ro, ld)
    ws = rl.make_workspace_columns(N, T, DEV)
    for name in TM_ESTIMATORS:
        out = run_tm(name, d, ws=ws)
        again = run_tm(name, d, ws=ws)
        torch.cuda.synchronize()
        for k in out:
            if out[k] is not None:
                assert torch.equal(out[k], again[k]), f"{name} {k}: not bitwise reproducible"
        assert_parity(out, ref_tm(name, ro), TOL[dtype], label=f"narrow split {name} T={T} N={N}")
    assert int(ws[8:12].view(torch.int32).item()) == 0
