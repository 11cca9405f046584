"""Seeded random GPU parity sweep: 600 cases drawn from one fixed seed, each one estimator on one
shape, dtype, flag density, layout (row-major, strided rows, time-major) and kernel variant,
against the fp64 oracle on the same inputs. The cases cover what hand-picked shapes can miss:
odd sizes, rows that straddle vectors and workgroups, row strides and time-major strides of any
residue, optional inputs (the termination array among them) present or not. A second sweep of 200 cases does the same for
eligibility traces of F-vectors. Each case prints itself before it runs. RLCS_RANDOM_CASES,
RLCS_RANDOM_VEC_CASES and RLCS_RANDOM_SEED (environment) draw longer or other sweeps."""
import os

import numpy as np
import pytest

from cases import TOL, assert_parity, oracle_run, to_device
import workloads

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2608_17641_amd as rl  # noqa: E402

DEV = torch.device("cuda:0")
NAMES = ("gae", "vtrace", "retrace", "td_lambda", "discounted", "elig_trace", "prefix_ends",
         "prefix_starts")
OUT_KEYS = {"gae": ("adv", "ret"), "vtrace": ("vs", "pg"), "retrace": ("delta", "q_ret"),
            "td_lambda": ("ret",), "discounted": ("ret",), "elig_trace": ("z",),
            "prefix_ends": ("c",), "prefix_starts": ("c",)}


def _cases(n=int(os.environ.get("RLCS_RANDOM_CASES", "600")),
           seed=int(os.environ.get("RLCS_RANDOM_SEED", "20261202"))):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        layout = ("rows", "strided", "tm")[rng.integers(0, 3)]
        N = int(rng.choice([1, 2, 3, 7, 16, 33, 64, 100, 257, 600, 1100, 4100]))
        T = int(rng.choice([1, 2, 3, 4, 5, 8, 31, 33, 64, 65, 100, 128, 129, 255, 256, 257, 512, 1000,
                            1025, 3000, 5000]))
        T = max(1, min(T, 3_000_000 // N))  # at most 3M steps a case
        pad = int(rng.integers(0, 40))
        out.append(dict(i=i, name=NAMES[rng.integers(0, len(NAMES))], N=N, T=T,
                        dtype=("f32", "bf16")[rng.integers(0, 2)], layout=layout, pad=pad,
                        p=float(rng.choice([0.0, 0.001, 0.005, 0.05, 0.3])),
                        trunc=bool(rng.integers(0, 2)), boot=bool(rng.integers(0, 2)),
                        variant=int(rng.integers(0, 5)), seed=int(rng.integers(0, 2 ** 31))))
        # one case in four has no termination array; taken from the case's seed, so that the
        # draws of every other field stay as they were
        out[-1]["term"] = out[-1]["seed"] % 4 != 0
    return out


def _view(t, layout, pad):
    """An [N, T] view of `t` in the case's layout (a copy into fresh storage for strided ones)."""
    if t.dim() != 2 or layout == "rows":
        return t
    N, T = t.shape
    if layout == "strided":
        buf = torch.full((N, T + pad), 3, dtype=t.dtype, device=t.device)
        buf[:, :T] = t
        return buf[:, :T]
    buf = torch.full((T, N + pad), 3, dtype=t.dtype, device=t.device)
    buf[:, :N] = t.t()
    return buf[:, :N].t()


def _run(name, d, trunc, boot, ws, strided):
    tr = d["trunc"] if trunc else None
    bv = d["bv"] if trunc else None
    bt = d["boot"] if boot else None
    sfx = "_strided" if strided else ""
    f = lambda base: getattr(rl, "rlcs_" + base + sfx)
    if name == "gae":
        return f("gae")(d["r"], d["v"], d.get("term"), tr, bv, bt, gamma=0.97, lam=0.9, ws=ws)
    if name == "vtrace":
        return f("vtrace")(d["r"], d["v"], d["log_rho"], d.get("term"), tr, bv, bt, gamma=0.97,
                           rho_bar=1.0, c_bar=0.9, ws=ws)
    if name == "retrace":
        return f("retrace")(d["r"], d["q"], d["eq"], d["log_rho"], d.get("term"), tr, bv, bt,
                            gamma=0.97, lam=0.9, c_bar=1.0, ws=ws)
    if name == "td_lambda":
        return (f("td_lambda")(d["r"], d["v"], d.get("term"), tr, bv, bt, gamma=0.97, lam=0.9, ws=ws),)
    if name == "discounted":
        return (f("discounted")(d["r"], d.get("term"), tr, bv, bt, gamma=0.97, ws=ws),)
    if name == "elig_trace":
        return (f("elig_trace")(d["x"], d.get("term"), tr, gamma=0.97, lam=0.9, ws=ws),)
    b = "starts_at" if name == "prefix_starts" else "ends_at"
    return (f("episodic_prefix")(d["x"], d.get("term"), tr, boundary=b, ws=ws),)


@pytest.mark.parametrize("case", _cases(), ids=lambda c: f"c{c['i']}")
def test_random_case(case):
    c = case
    print(f"case {c}", flush=True)
    ro = workloads.make_rollout(c["N"], c["T"], c["seed"], dtype=c["dtype"], p_term=c["p"],
                                p_trunc=c["p"])
    if not c["term"]:
        del ro["term"]
    d = {k: _view(to_device(v, DEV), c["layout"], c["pad"]) for k, v in ro.items()}
    strided = c["layout"] != "rows"
    ws = (rl.make_workspace_columns(c["N"], c["T"], DEV) if strided
          else rl.make_workspace(c["N"], c["T"], DEV))
    rl.testing_set_variant(c["variant"])
    try:
        outs = _run(c["name"], d, c["trunc"], c["boot"], ws, strided)
        torch.cuda.synchronize()
    finally:
        rl.testing_set_variant(0)
    ref = oracle_run(c["name"], ro, trunc=c["trunc"], boot=c["boot"], gamma=0.97, lam=0.9,
                     c_bar=0.9 if c["name"] == "vtrace" else 1.0)
    got = {k: o for k, o in zip(OUT_KEYS[c["name"]], outs) if o is not None}
    assert_parity(got, {k: ref[k] for k in got}, TOL[c["dtype"]], label=f"random case {c['i']}")
    assert int(ws[8:12].view(torch.int32).item()) == 0


def _vec_cases(n=int(os.environ.get("RLCS_RANDOM_VEC_CASES", "200")),
               seed=int(os.environ.get("RLCS_RANDOM_SEED", "20261202")) + 1):
    """Vector eligibility traces: most cases shaped for the row kernel (F a multiple of the vector
    width with a power-of-two number of vectors, T up to the most its waves hold, enough rows for
    256 workgroups or more), the rest any shape, under any variant."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        dtype = ("f32", "bf16")[rng.integers(0, 2)]
        if rng.random() < 0.7:
            V = 4 if dtype == "f32" else 8
            F = V * int(rng.choice([1, 2, 4, 8, 16, 32, 64]))
            per_wave = 64 // (F // V) * 4
            most = per_wave * 16
            if rng.random() < 0.4:  # at most a wave's steps: several rows to a workgroup
                T = int(rng.integers(1, per_wave + 1))
            else:
                T = int(rng.integers(per_wave // 2 + 1, most + 1))
            rows = max(1, per_wave // T)  # about the rows of a one-wave workgroup
            N = int(rng.choice([256, 257, 300, 513])) * rows + int(rng.integers(0, rows))
            variant = int(rng.choice([0, 0, 0, 0, 1, 3]))
        else:
            N = int(rng.choice([1, 7, 64, 255, 600]))
            F = int(rng.choice([1, 3, 12, 16, 24, 40]))
            T = int(rng.choice([1, 2, 3, 5, 31, 33, 64, 100, 129, 257, 1000, 2049]))
            variant = int(rng.integers(0, 5))
        T = max(1, min(T, 8_000_000 // (N * F)))  # at most 8M elements a case
        out.append(dict(i=i, N=N, T=T, F=F, dtype=dtype, p=float(rng.choice([0.0, 0.005, 0.05, 0.3])),
                        term=bool(rng.integers(0, 4) > 0), trunc=bool(rng.integers(0, 2)),
                        variant=variant, seed=int(rng.integers(0, 2 ** 31))))
    return out


@pytest.mark.parametrize("case", _vec_cases(), ids=lambda c: f"v{c['i']}")
def test_random_vec_case(case):
    import oracle
    c = case
    print(f"case {c}", flush=True)
    ro = workloads.make_vector_trace(c["N"], c["T"], c["F"], seed=c["seed"], dtype=c["dtype"],
                                     p_term=c["p"], p_trunc=c["p"])
    term = ro["term"] if c["term"] else None
    trunc = ro["trunc"] if c["trunc"] else None
    ws = rl.make_workspace_columns(c["N"] * c["F"], c["T"], DEV)
    rl.testing_set_variant(c["variant"])
    try:
        z = rl.rlcs_elig_trace_vec(to_device(ro["x"], DEV),
                                   None if term is None else to_device(term, DEV),
                                   None if trunc is None else to_device(trunc, DEV),
                                   gamma=0.97, lam=0.9, ws=ws)
        torch.cuda.synchronize()
    finally:
        rl.testing_set_variant(0)
    ref = oracle.elig_trace_vec(ro["x"], term, trunc, gamma=0.97, lam=0.9)
    assert_parity({"z": z}, {"z": ref}, TOL[c["dtype"]], label=f"random vec case {c['i']}")
    assert int(ws[8:12].view(torch.int32).item()) == 0
