"""Shared helpers for the GPU parity tests: run an estimator through the C ABI (via the thin
binding) and through the oracle on the same seeded host arrays, and compare them."""
from __future__ import annotations

import numpy as np

import oracle
import workloads

# Estimator name -> output names, in the order the binding returns them.
OUTPUTS = {
    "gae": ("adv", "ret"),
    "vtrace": ("vs", "pg"),
    "retrace": ("delta", "q_ret"),
    "td_lambda": ("ret",),
    "discounted": ("ret",),
    "elig_trace": ("z",),
    "prefix_ends": ("c",),
    "prefix_starts": ("c",),
    "affine_back": ("out",),
    "affine_fwd": ("out",),
}
ESTIMATORS = tuple(OUTPUTS)
SEVEN = ("gae", "vtrace", "retrace", "td_lambda", "discounted", "elig_trace", "prefix_ends")

TOL = {"f32": 1e-5, "bf16": 1e-3}


def make_inputs(name, N, T, seed=0, dtype="f32", **kw):
    if name.startswith("affine"):
        return workloads.make_affine(N, T, seed, dtype=dtype)
    return workloads.make_rollout(N, T, seed, dtype=dtype, **kw)


def to_device(arr, device):
    import torch
    if arr is None:
        return None
    if arr.dtype == np.int32:
        return torch.from_numpy(np.ascontiguousarray(arr)).to(device)
    if arr.dtype == np.uint16:
        return torch.from_numpy(arr.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(arr)).to(device)


def device_inputs(ro, device):
    return {k: to_device(v, device) for k, v in ro.items()}


def gpu_run(name, d, *, trunc=True, boot=True, gamma=0.99, lam=0.95, rho_bar=1.0, c_bar=1.0,
            ws=None, outputs=None):
    """Run estimator `name` on device inputs `d`; returns {output: torch tensor}."""
    import paper_2608_17641_amd as rl
    tr = d.get("trunc") if trunc else None
    bv = d.get("bv") if trunc else None
    bt = d.get("boot") if boot else None
    if name == "gae":
        a, r = rl.rlcs_gae(d["r"], d["v"], d["term"], tr, bv, bt, gamma=gamma, lam=lam, ws=ws)
        return {"adv": a, "ret": r}
    if name == "vtrace":
        a, b = rl.rlcs_vtrace(d["r"], d["v"], d["log_rho"], d["term"], tr, bv, bt, gamma=gamma,
                              rho_bar=rho_bar, c_bar=c_bar, ws=ws)
        return {"vs": a, "pg": b}
    if name == "retrace":
        a, b = rl.rlcs_retrace(d["r"], d["q"], d["eq"], d["log_rho"], d["term"], tr, bv, bt,
                               gamma=gamma, lam=lam, c_bar=c_bar, ws=ws)
        return {"delta": a, "q_ret": b}
    if name == "td_lambda":
        return {"ret": rl.rlcs_td_lambda(d["r"], d["v"], d["term"], tr, bv, bt, gamma=gamma,
                                         lam=lam, ws=ws)}
    if name == "discounted":
        return {"ret": rl.rlcs_discounted(d["r"], d["term"], tr, bv, bt, gamma=gamma, ws=ws)}
    if name == "elig_trace":
        return {"z": rl.rlcs_elig_trace(d["x"], d["term"], tr, gamma=gamma, lam=lam, ws=ws)}
    if name in ("prefix_ends", "prefix_starts"):
        b = "starts_at" if name == "prefix_starts" else "ends_at"
        return {"c": rl.rlcs_episodic_prefix(d["x"], d["term"], tr, boundary=b, ws=ws)}
    if name in ("affine_back", "affine_fwd"):
        return {"out": rl.rlcs_affine_scan(d["alpha"], d["beta"], d["carry"] if boot else None,
                                           reverse=(name == "affine_back"), ws=ws)}
    raise KeyError(name)


def oracle_run(name, ro, *, trunc=True, boot=True, gamma=0.99, lam=0.95, rho_bar=1.0, c_bar=1.0,
               rows=None):
    """Oracle outputs (fp64 numpy) for estimator `name`, optionally only for `rows`."""
    def g(k):
        a = ro.get(k)
        if a is None:
            return None
        return a[rows] if rows is not None else a

    tr = g("trunc") if trunc else None
    bv = g("bv") if trunc else None
    bt = g("boot") if boot else None
    if name == "gae":
        a, r = oracle.gae(g("r"), g("v"), g("term"), tr, bv, bt, gamma=gamma, lam=lam)
        return {"adv": a, "ret": r}
    if name == "vtrace":
        a, b = oracle.vtrace(g("r"), g("v"), g("log_rho"), g("term"), tr, bv, bt, gamma=gamma,
                             rho_bar=rho_bar, c_bar=c_bar)
        return {"vs": a, "pg": b}
    if name == "retrace":
        a, b = oracle.retrace(g("r"), g("q"), g("eq"), g("log_rho"), g("term"), tr, bv, bt,
                              gamma=gamma, lam=lam, c_bar=c_bar)
        return {"delta": a, "q_ret": b}
    if name == "td_lambda":
        return {"ret": oracle.td_lambda(g("r"), g("v"), g("term"), tr, bv, bt, gamma=gamma, lam=lam)}
    if name == "discounted":
        return {"ret": oracle.discounted(g("r"), g("term"), tr, bv, bt, gamma=gamma)}
    if name == "elig_trace":
        return {"z": oracle.elig_trace(g("x"), g("term"), tr, gamma=gamma, lam=lam)}
    if name in ("prefix_ends", "prefix_starts"):
        b = "starts_at" if name == "prefix_starts" else "ends_at"
        return {"c": oracle.episodic_prefix(g("x"), g("term"), tr, boundary=b)}
    if name in ("affine_back", "affine_fwd"):
        return {"out": oracle.affine_scan(g("alpha"), g("beta"), g("carry") if boot else None,
                                          reverse=(name == "affine_back"))}
    raise KeyError(name)


def max_err(gpu: np.ndarray, ref: np.ndarray):
    """(max |gpu - ref|, 1 + max |ref|)."""
    gpu = np.asarray(gpu, np.float64)
    if ref.size == 0:
        return 0.0, 1.0
    return float(np.max(np.abs(gpu - ref))), 1.0 + float(np.max(np.abs(ref)))


def assert_parity(gpu: dict, ref: dict, tol: float, label=""):
    """max_i |gpu_i - ref_i| <= tol * (1 + max_i |ref_i|), per output tensor."""
    worst = {}
    for k, r in ref.items():
        g = gpu[k]
        if hasattr(g, "cpu"):
            g = g.float().cpu().numpy()
        assert g.shape == r.shape, (label, k, g.shape, r.shape)
        assert np.all(np.isfinite(g)), f"{label} {k}: non-finite GPU output"
        err, scale = max_err(g, r)
        worst[k] = err / scale
        assert err <= tol * scale, (f"{label} {k}: max err {err:.3e} > {tol:g} * {scale:.3f}; "
                                    + mismatch_report(g, r, tol * scale))
    return worst


def mismatch_report(g: np.ndarray, r: np.ndarray, bound: float, show: int = 12) -> str:
    """Where a failed comparison differs: how many elements exceed the bound, the first ones
    (index, GPU value, oracle value), and the byte span they cover in a float32 output."""
    bad = np.argwhere(np.abs(np.asarray(g, np.float64) - r) > bound)
    if bad.size == 0:
        return "no element above the bound"
    flat = np.ravel_multi_index(bad.T, r.shape)
    first = ", ".join(f"{tuple(int(x) for x in i)}: {float(g[tuple(i)]):.6g} vs {float(r[tuple(i)]):.6g}"
                      for i in bad[:show])
    return (f"{len(bad)} of {r.size} elements differ, flat float32 byte offsets "
            f"{4 * int(flat.min())}..{4 * int(flat.max()) + 3}; first: {first}")
