"""GPU parity: every entry point, called through the C ABI, against the fp64 oracle on the same
seeded inputs. Bar: max |gpu - oracle| <= tol * (1 + max |oracle|) per output tensor, with
tol = 1e-5 for float32 inputs and 1e-3 for bfloat16 inputs (arithmetic is float32 in both)."""
import contextlib

import numpy as np
import pytest

from cases import (ESTIMATORS, OUTPUTS, SEVEN, TOL, assert_parity, device_inputs, gpu_run,
                   make_inputs, oracle_run, to_device)
import workloads

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2608_17641_amd as rl  # noqa: E402

DEV = torch.device("cuda:0")


@contextlib.contextmanager
def variant(v):
    rl.testing_set_variant(v)
    try:
        yield
    finally:
        rl.testing_set_variant(0)


def check(name, ro, *, trunc=True, boot=True, ws=None, label="", **params):
    d = device_inputs(ro, DEV)
    out = gpu_run(name, d, trunc=trunc, boot=boot, ws=ws, **params)
    torch.cuda.synchronize()
    ref = oracle_run(name, ro, trunc=trunc, boot=boot, **params)
    return assert_parity(out, ref, TOL[ro.dtype], label=f"{name} {label}")


# ------------------------------------------------------------------ the five workloads

def test_gae_8x128_plain():
    ro = workloads.make_rollout(8, 128, 0, p_term=0.01, p_trunc=0.0)
    check("gae", ro, trunc=False, gamma=0.99, lam=0.95)


@pytest.mark.parametrize("name", ESTIMATORS)
def test_all_estimators_4096x32_with_truncation(name):
    ro = make_inputs(name, 4096, 32, 0, p_term=0.02, p_trunc=0.01)
    check(name, ro, gamma=0.99, lam=0.95)


@pytest.mark.parametrize("name", ["gae", "vtrace"])
@pytest.mark.parametrize("trunc", [True, False])
def test_headline_4096x256(name, trunc):
    ro = workloads.make_rollout(4096, 256, 0, p_term=0.02, p_trunc=0.01)
    check(name, ro, trunc=trunc, gamma=0.99, lam=0.95)


@pytest.mark.parametrize("name", ["gae", "td_lambda"])
@pytest.mark.parametrize("var", [0, 1, 2])
def test_rlhf_64x4096(name, var):
    ro = workloads.make_rlhf_rollout(64, 4096, 0)
    ws = rl.make_workspace(64, 4096, DEV)
    with variant(var):
        check(name, ro, trunc=False, boot=False, ws=ws, gamma=1.0, lam=0.95, label=f"variant {var}")
    assert int(ws[8:12].view(torch.int32).item()) == 0  # workspace error flag


# ------------------------------------------------------------------ shapes and variants

ODD_T = [1, 2, 3, 5, 7, 31, 33, 63, 65, 255, 257, 1023, 1025, 1100, 4095, 4097]


@pytest.mark.parametrize("T", ODD_T)
@pytest.mark.parametrize("var", [1, 2])
def test_odd_lengths_all_estimators(T, var):
    N = 37
    ws = rl.make_workspace(N, T, DEV)
    with variant(var):
        for i, name in enumerate(ESTIMATORS):
            ro = make_inputs(name, N, T, seed=T * 10 + i, p_term=0.05, p_trunc=0.05)
            check(name, ro, ws=ws, gamma=0.97, lam=0.9, label=f"T={T} variant {var}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("T", [24, 96, 200, 1000, 3000, 5000, 8200])
def test_vector_lengths_not_dividing_the_chunk(T, dtype):
    """T a multiple of the vector width whose rows do not fill a workgroup's chunks exactly:
    the vector path with the lanes outside the workgroup's rows skipped."""
    N = 37
    ws = rl.make_workspace(N, T, DEV)
    with variant(1):
        for i, name in enumerate(ESTIMATORS):
            ro = make_inputs(name, N, T, seed=T * 10 + i, dtype=dtype, p_term=0.05, p_trunc=0.05)
            check(name, ro, ws=ws, gamma=0.97, lam=0.9, label=f"T={T} {dtype}")


@pytest.mark.parametrize("T", [3, 64, 129, 2050])
@pytest.mark.parametrize("var", [1, 2])
def test_odd_lengths_bf16(T, var):
    N = 29
    ws = rl.make_workspace(N, T, DEV)
    with variant(var):
        for i, name in enumerate(ESTIMATORS):
            ro = make_inputs(name, N, T, seed=500 + T + i, dtype="bf16", p_term=0.05, p_trunc=0.05)
            check(name, ro, ws=ws, gamma=0.97, lam=0.9, label=f"bf16 T={T} variant {var}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("T", [4, 8, 16, 32, 64, 128, 256, 512])
def test_rows_tiling_a_wave(T, dtype):
    """Power-of-two rows of K to 64*K steps (K = 4 float32, 8 bfloat16 steps per lane): the
    wave-rows kernel, whole rows per wave. Row counts that leave the last wave partial, one
    row, and many rows; with and without truncation and bootstrap."""
    K = 4 if dtype == "f32" else 8
    if T < K or T > 64 * K:
        pytest.skip("not a wave-rows shape for this dtype")
    for N in (1, 3, 1000 // T + 1, 4099):
        for i, name in enumerate(ESTIMATORS):
            ro = make_inputs(name, N, T, seed=N * 7 + T + i, dtype=dtype, p_term=0.05, p_trunc=0.05)
            check(name, ro, gamma=0.97, lam=0.9, label=f"{N}x{T} {dtype}")
            if name in ("gae", "vtrace", "td_lambda"):
                check(name, ro, trunc=False, boot=False, gamma=0.97, lam=0.9,
                      label=f"{N}x{T} {dtype} plain")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("T", [8, 12, 20, 24, 36, 40, 72, 100, 132, 136, 192, 200, 240, 252, 264,
                               300, 384, 500, 504, 512, 600, 1000, 1020, 1024, 1028, 1100, 1500,
                               2000, 2048, 3000, 4092, 4096])
def test_rows_flat(T, dtype):
    """Dense rows of a multiple of K steps, at most one sixteen-wave chunk (float32) or one wave
    (bfloat16), except powers of two that tile a wave: the flat rows kernel, floor(256*K / T)
    whole rows per four-wave workgroup, or floor(1024*K / T) per sixteen-wave one for float32
    rows of more than 1024 steps, rows straddling waves. Row counts that leave the last
    workgroup partial, one row, and many rows; with and without truncation and bootstrap."""
    K = 4 if dtype == "f32" else 8
    flat_max = 1024 * K if dtype == "f32" else 64 * K
    if T % K or T <= K or T > flat_max or ((T & (T - 1)) == 0 and T <= 64 * K):
        pytest.skip("not a flat-rows shape for this dtype")
    R = 256 * K // T or 1024 * K // T
    for N in (1, R + 1, 3 * R - 1, 4099 if T <= 256 * K else 601):
        for i, name in enumerate(ESTIMATORS):
            ro = make_inputs(name, N, T, seed=N * 13 + T + i, dtype=dtype, p_term=0.05, p_trunc=0.05)
            check(name, ro, gamma=0.97, lam=0.9, label=f"{N}x{T} {dtype}")
            if name in ("gae", "vtrace", "td_lambda"):
                check(name, ro, trunc=False, boot=False, gamma=0.97, lam=0.9,
                      label=f"{N}x{T} {dtype} plain")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("T", [5, 9, 33, 100, 101, 129, 250, 251, 255, 257, 300, 499, 514, 771, 1001,
                               1022, 1023])
def test_rows_flat_ragged(T, dtype):
    """Rows whose length is not a multiple of K: the flat rows kernel where a workgroup's rows
    start and end on vector boundaries (a row edge inside a lane's K steps), the lane-by-lane
    rows kernel where they cannot (N*T not a multiple of K, or rows too long): both against the
    oracle, with and without truncation and bootstrap."""
    K = 4 if dtype == "f32" else 8
    for N in (K, 3 * K, 4 * K + 1, 1000 * K):
        for i, name in enumerate(ESTIMATORS):
            ro = make_inputs(name, N, T, seed=N * 17 + T + i, dtype=dtype, p_term=0.05, p_trunc=0.05)
            check(name, ro, gamma=0.97, lam=0.9, label=f"{N}x{T} {dtype}")
            if name in ("gae", "vtrace", "td_lambda"):
                check(name, ro, trunc=False, boot=False, gamma=0.97, lam=0.9,
                      label=f"{N}x{T} {dtype} plain")


@pytest.mark.parametrize("N,T", [(1, 1), (1, 4096), (1, 1 << 20), (3, 100_000), (5000, 3)])
@pytest.mark.parametrize("var", [0, 1, 2])
def test_extreme_shapes(N, T, var):
    ws = rl.make_workspace(N, T, DEV)
    with variant(var):
        for name in ("gae", "vtrace", "retrace", "elig_trace", "prefix_starts"):
            ro = make_inputs(name, N, T, seed=N + T, p_term=0.001, p_trunc=0.001)
            check(name, ro, ws=ws, gamma=0.999, lam=0.97, label=f"{N}x{T} variant {var}")


def test_no_flags_no_bootstrap():
    ro = workloads.make_rollout(64, 300, 3, p_term=0.0, p_trunc=0.0)
    ro["term"] = None
    for name in ("gae", "td_lambda", "discounted", "vtrace", "retrace", "elig_trace",
                 "prefix_ends"):
        check(name, ro, trunc=False, boot=False, gamma=0.99, lam=0.95)


def test_both_flags_and_parameter_extremes():
    ro = workloads.make_rollout(50, 70, 4, p_term=0.3, p_trunc=0.3)
    for gamma, lam in ((0.0, 0.0), (1.0, 1.0), (1.0, 0.0), (0.5, 1.0)):
        for name in ("gae", "td_lambda", "discounted", "retrace", "elig_trace"):
            check(name, ro, gamma=gamma, lam=lam, label=f"g={gamma} l={lam}")
    for rho_bar, c_bar in ((float("inf"), float("inf")), (0.5, 2.0)):
        check("vtrace", ro, gamma=0.9, rho_bar=rho_bar, c_bar=c_bar)
        check("retrace", ro, gamma=0.9, lam=0.8, c_bar=c_bar)


def test_misaligned_pointers_take_scalar_path():
    """Contiguous views that start 4 bytes (fp32) / 2 bytes (bf16) past a 16-byte boundary."""
    N, T = 33, 77
    for dtype in ("f32", "bf16"):
        ro = workloads.make_rollout(N, T, 5, dtype=dtype, p_term=0.05, p_trunc=0.05)
        d = {}
        for k, a in ro.items():
            t = to_device(a, DEV)
            base = torch.empty(t.numel() + 1, dtype=t.dtype, device=DEV)
            view = base[1:].view(t.shape)
            view.copy_(t)
            d[k] = view
        for name in ("gae", "vtrace", "retrace", "td_lambda", "discounted", "elig_trace"):
            out = gpu_run(name, d, gamma=0.99, lam=0.95)
            torch.cuda.synchronize()
            assert_parity(out, oracle_run(name, ro, gamma=0.99, lam=0.95), TOL[dtype],
                          label=f"misaligned {dtype} {name}")


def test_optional_outputs():
    ro = workloads.make_rollout(40, 64, 6)
    d = device_inputs(ro, DEV)
    adv, ret = rl.rlcs_gae(d["r"], d["v"], d["term"], d["trunc"], d["bv"], d["boot"], gamma=0.99,
                           lam=0.95, want_ret=False)
    assert ret is None
    vs, pg = rl.rlcs_vtrace(d["r"], d["v"], d["log_rho"], d["term"], d["trunc"], d["bv"],
                            d["boot"], gamma=0.99, want_pg=False)
    dl, qr = rl.rlcs_retrace(d["r"], d["q"], d["eq"], d["log_rho"], d["term"], d["trunc"],
                             d["bv"], d["boot"], gamma=0.99, lam=0.95, want_q_ret=False)
    torch.cuda.synchronize()
    assert pg is None and qr is None
    assert_parity({"adv": adv}, {"adv": oracle_run("gae", ro)["adv"]}, 1e-5)
    assert_parity({"vs": vs}, {"vs": oracle_run("vtrace", ro)["vs"]}, 1e-5)
    assert_parity({"delta": dl}, {"delta": oracle_run("retrace", ro)["delta"]}, 1e-5)


def test_empty_shapes_are_noops():
    for N, T in ((0, 10), (10, 0), (0, 0)):
        x = torch.zeros((N, T), device=DEV)
        out = torch.full((N, T), 7.0, device=DEV)
        rl.rlcs_elig_trace(x, z=out, gamma=0.9, lam=0.9)
        a, r = rl.rlcs_gae(x, x, adv=out, gamma=0.9, lam=0.9, want_ret=False)
        torch.cuda.synchronize()
        assert out.numel() == 0 or bool((out == 7.0).all())


# ------------------------------------------------------------------ invariants

@pytest.mark.parametrize("T", [32, 256, 1000, 5000])
def test_run_to_run_bitwise(T):
    N = 300
    ro = workloads.make_rollout(N, T, 7)
    d = device_inputs(ro, DEV)
    ws = rl.make_workspace(N, T, DEV)
    for var in (1, 2):
        with variant(var):
            for name in SEVEN:
                a = gpu_run(name, d, ws=ws)
                b = gpu_run(name, d, ws=ws)
                torch.cuda.synchronize()
                for k in a:
                    assert torch.equal(a[k], b[k]), (name, k, T, var)


@pytest.mark.parametrize("T", [32, 64, 256])
def test_row_permutation(T):
    """Rows are independent: permuting the input rows permutes the outputs, bit for bit, when
    every row sits at the same lane offset within its wave (T divides 64*K)."""
    N = 1024
    ro = workloads.make_rollout(N, T, 8)
    perm = np.random.default_rng(9).permutation(N)
    rop = workloads.Rollout(N, T, "f32", **{k: (v[perm] if v.ndim else v) for k, v in ro.items()})
    d, dp = device_inputs(ro, DEV), device_inputs(rop, DEV)
    pt = torch.from_numpy(perm).to(DEV)
    for name in SEVEN:
        a, b = gpu_run(name, d), gpu_run(name, dp)
        torch.cuda.synchronize()
        for k in a:
            assert torch.equal(a[k].index_select(0, pt), b[k]), (name, k)


@pytest.mark.parametrize("var", [1, 2])
def test_severing_invariance(var):
    """Section 5.2: with a flag at step t, backward outputs at steps <= t do not change when
    anything after t changes (and forward outputs after t do not change when anything before
    t changes)."""
    N, T, t = 64, 3000, 1700
    ro = workloads.make_rollout(N, T, 10, p_term=0.0, p_trunc=0.0)
    ro["term"][:, t] = 1
    pert = workloads.Rollout(N, T, "f32", **{k: v.copy() for k, v in ro.items()})
    rng = np.random.default_rng(11)
    for k in ("r", "v", "bv", "log_rho", "q", "eq"):
        pert[k][:, t + 1:] = rng.standard_normal((N, T - t - 1)).astype(np.float32)
    pert["boot"] = rng.standard_normal(N).astype(np.float32)
    pert_f = workloads.Rollout(N, T, "f32", **{k: v.copy() for k, v in ro.items()})
    pert_f["x"][:, :t + 1] = rng.standard_normal((N, t + 1)).astype(np.float32)
    ws = rl.make_workspace(N, T, DEV)
    with variant(var):
        for name in ("gae", "vtrace", "retrace", "td_lambda", "discounted"):
            a = gpu_run(name, device_inputs(ro, DEV), ws=ws)
            b = gpu_run(name, device_inputs(pert, DEV), ws=ws)
            torch.cuda.synchronize()
            for k in a:
                assert torch.equal(a[k][:, :t + 1], b[k][:, :t + 1]), (name, k)
                assert not torch.equal(a[k][:, t + 1:], b[k][:, t + 1:])
        a = gpu_run("prefix_ends", device_inputs(ro, DEV), ws=ws)["c"]
        b = gpu_run("prefix_ends", device_inputs(pert_f, DEV), ws=ws)["c"]
        torch.cuda.synchronize()
        assert torch.equal(a[:, t + 1:], b[:, t + 1:])


def test_workspace_reused_across_shapes():
    """One workspace serves consecutive split-row calls of different shapes."""
    ws = rl.make_workspace(64, 8192, DEV)
    with variant(2):
        for (N, T) in ((64, 8192), (3, 5000), (64, 8192), (17, 2049), (1, 30000)):
            for name in ("gae", "elig_trace"):
                ro = make_inputs(name, N, T, seed=N * T)
                check(name, ro, ws=ws, label=f"{N}x{T}")
    assert int(ws[8:12].view(torch.int32).item()) == 0


# ------------------------------------------------------------------ full-form Retrace

def _retrace_full_run(ro, *, trunc=True, boot=True, gamma=0.99, lam=0.95, c_bar=1.0, act=None,
                      term=True):
    d = device_inputs(ro, DEV)
    if act is not None:
        d["actions"] = torch.from_numpy(act).to(DEV)
    dl, qr = rl.rlcs_retrace_full(d["r"], d["q3"], d["pi3"], d["actions"], d["mu"],
                                  d["term"] if term else None,
                                  d["trunc"] if trunc else None, d["bv"] if trunc else None,
                                  d["boot"] if boot else None, gamma=gamma, lam=lam, c_bar=c_bar)
    torch.cuda.synchronize()
    import oracle
    a = ro["actions"] if act is None else act
    rd, rq = oracle.retrace_full(ro["r"], ro["q3"], ro["pi3"], a, ro["mu"], ro["term"] if term else None,
                                 ro["trunc"] if trunc else None, ro["bv"] if trunc else None,
                                 ro["boot"] if boot else None, gamma=gamma, lam=lam, c_bar=c_bar)
    return {"delta": dl, "q_ret": qr}, {"delta": rd, "q_ret": rq}


@pytest.mark.parametrize("A", [1, 3, 4, 6, 7, 18, 28])
@pytest.mark.parametrize("T", [1, 7, 33, 256, 1000, 4097])
def test_retrace_full_shapes(A, T):
    N = 23
    ro = workloads.make_retrace_full(N, T, A, seed=A * 1000 + T, p_term=0.05, p_trunc=0.05)
    out, ref = _retrace_full_run(ro, c_bar=0.9)
    assert_parity(out, ref, 1e-5, label=f"retrace_full A={A} T={T}")
    out, ref = _retrace_full_run(ro, c_bar=0.9, term=False)
    assert_parity(out, ref, 1e-5, label=f"retrace_full no term A={A} T={T}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("A", [29, 30, 33, 64, 100, 256])
@pytest.mark.parametrize("T", [1, 33, 4097])
def test_retrace_full_long_action_axes(A, T, dtype):
    """More actions than a chunk's whole slices hold in LDS: the action axis staged in slices
    of 32 actions (one slice at A = 29 and 30; A = 33 and 100 leave a partial last slice, 64
    and 256 whole ones; an odd count of bfloat16 actions per row splits 16-byte blocks between
    rows)."""
    N = 5 if T > 1000 else 23
    ro = workloads.make_retrace_full(N, T, A, seed=A * 31 + T, dtype=dtype, p_term=0.05, p_trunc=0.05)
    out, ref = _retrace_full_run(ro, c_bar=0.9)
    assert_parity(out, ref, TOL[dtype], label=f"retrace_full A={A} T={T} {dtype}")


@pytest.mark.parametrize("A", [5, 64])
def test_retrace_full_reports_out_of_range_actions(A):
    """An action outside [0, A) takes Q and pi as 0 at its step (as the oracle does) and sets
    the workspace's error word to 2; a call without such actions leaves it at 0."""
    ro = workloads.make_retrace_full(64, 100, A, seed=79 + A, p_term=0.05, p_trunc=0.05)
    d = device_inputs(ro, DEV)
    ws = torch.zeros(64, dtype=torch.uint8, device=DEV)
    rl.rlcs_retrace_full(d["r"], d["q3"], d["pi3"], d["actions"], d["mu"], d["term"], d["trunc"],
                         d["bv"], d["boot"], gamma=0.97, lam=0.9, ws=ws)
    torch.cuda.synchronize()
    assert int(ws[8:12].view(torch.int32).item()) == 0
    act = ro["actions"].copy()
    act[::3, ::7] = A
    act[1::5, 2::9] = -3
    d["actions"] = torch.from_numpy(act).to(DEV)
    dl, qr = rl.rlcs_retrace_full(d["r"], d["q3"], d["pi3"], d["actions"], d["mu"], d["term"],
                                  d["trunc"], d["bv"], d["boot"], gamma=0.97, lam=0.9, ws=ws)
    torch.cuda.synchronize()
    assert int(ws[8:12].view(torch.int32).item()) == 2
    import oracle
    rd, rq = oracle.retrace_full(ro["r"], ro["q3"], ro["pi3"], act, ro["mu"], ro["term"],
                                 ro["trunc"], ro["bv"], ro["boot"], gamma=0.97, lam=0.9)
    assert_parity({"delta": dl, "q_ret": qr}, {"delta": rd, "q_ret": rq}, 1e-5,
                  label=f"out-of-range actions A={A}")


@pytest.mark.parametrize("A", [4, 8, 18, 24])
def test_retrace_full_bf16_and_plain(A):
    ro = workloads.make_retrace_full(300, 129, A, seed=A, dtype="bf16", p_term=0.05, p_trunc=0.05)
    out, ref = _retrace_full_run(ro)
    assert_parity(out, ref, 1e-3, label=f"retrace_full bf16 A={A}")
    ro = workloads.make_retrace_full(300, 256, A, seed=A + 1, p_term=0.05, p_trunc=0.0)
    out, ref = _retrace_full_run(ro, trunc=False, boot=False)
    assert_parity(out, ref, 1e-5, label=f"retrace_full plain A={A}")


def _misaligned(t):
    """A copy of `t` whose storage starts one element past a 16-byte boundary."""
    buf = torch.empty(t.numel() + 1, dtype=t.dtype, device=t.device)
    buf[1:].copy_(t.reshape(-1))
    return buf[1:].view(t.shape)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("A", [3, 4, 18, 40])
def test_retrace_full_unaligned_slices(A, dtype):
    """Q and pi not 16-byte aligned: the slices are staged element-wise."""
    ro = workloads.make_retrace_full(37, 301, A, seed=5 + A, dtype=dtype, p_term=0.05, p_trunc=0.05)
    d = device_inputs(ro, DEV)
    q, pi = _misaligned(d["q3"]), _misaligned(d["pi3"])
    assert q.data_ptr() % 16 != 0 and pi.data_ptr() % 16 != 0
    dl, qr = rl.rlcs_retrace_full(d["r"], q, pi, d["actions"], d["mu"], d["term"], d["trunc"],
                                  d["bv"], d["boot"], gamma=0.97, lam=0.9, c_bar=1.0)
    torch.cuda.synchronize()
    import oracle
    rd, rq = oracle.retrace_full(ro["r"], ro["q3"], ro["pi3"], ro["actions"], ro["mu"], ro["term"],
                                 ro["trunc"], ro["bv"], ro["boot"], gamma=0.97, lam=0.9, c_bar=1.0)
    assert_parity({"delta": dl, "q_ret": qr}, {"delta": rd, "q_ret": rq}, TOL[dtype],
                  label=f"retrace_full unaligned A={A} {dtype}")


def test_retrace_full_out_of_range_actions():
    A = 5
    ro = workloads.make_retrace_full(64, 100, A, seed=77, p_term=0.05, p_trunc=0.05)
    act = ro["actions"].copy()
    act[::3, ::7] = A
    act[1::5, 2::9] = -3
    out, ref = _retrace_full_run(ro, act=act)
    assert_parity(out, ref, 1e-5, label="retrace_full out-of-range actions")


def test_retrace_full_4096x256():
    ro = workloads.make_retrace_full(4096, 256, 4, seed=0, p_term=0.02, p_trunc=0.01)
    out, ref = _retrace_full_run(ro)
    assert_parity(out, ref, 1e-5, label="retrace_full 4096x256x4")
