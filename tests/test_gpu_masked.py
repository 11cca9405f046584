"""GPU parity of GAE with observation-skip masking and advantage whitening (rlcs_gae_masked)
through the C ABI, against the fp64 oracle on the same seeded inputs. Bar: max |gpu - oracle|
<= tol * (1 + max |oracle|) per output, tol = 1e-5 for float32 inputs and 1e-3 for bfloat16
inputs (whitened outputs included: the oracle whitens its own fp64 advantages)."""
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


def run(ro, mask, *, trunc=True, boot=True, normalize=False, eps=1e-8, gamma=G, lam=L, term=True):
    d = {k: to_device(v, DEV) for k, v in ro.items()}
    te = d["term"] if term else None
    m = None if mask is None else to_device(mask, DEV)
    tr = d["trunc"] if trunc else None
    bv = d["bv"] if trunc else None
    bt = d["boot"] if boot else None
    adv, ret = rl.rlcs_gae_masked(d["r"], d["v"], m, te, tr, bv, bt, gamma=gamma, lam=lam,
                                  normalize=normalize, eps=eps)
    torch.cuda.synchronize()
    a, r = oracle.gae_masked(ro["r"], ro["v"], mask, ro["term"] if term else None,
                             ro["trunc"] if trunc else None,
                             ro["bv"] if trunc else None, ro["boot"] if boot else None, gamma=gamma,
                             lam=lam)
    if normalize:
        a = oracle.normalize_advantages(a, mask, eps=eps)
    return {"adv": adv, "ret": ret}, {"adv": a, "ret": r}


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("N,T", [(1, 1), (5, 7), (64, 256), (33, 1000), (8, 4097), (3, 9000),
                                 (300, 33)])
def test_gae_masked_random_masks(N, T, dtype):
    ro = workloads.make_rollout(N, T, seed=N * 31 + T, dtype=dtype, p_term=0.03, p_trunc=0.03)
    mask = (np.random.default_rng(T).random((N, T)) < 0.6).astype(np.uint8)
    for norm in (False, True):
        out, ref = run(ro, mask, normalize=norm)
        assert_parity(out, ref, TOL[dtype], label=f"masked {N}x{T} {dtype} norm={norm}")
    out, ref = run(ro, None)
    assert_parity(out, ref, TOL[dtype], label=f"unmasked {N}x{T} {dtype}")
    out, ref = run(ro, mask, trunc=False, boot=False)
    assert_parity(out, ref, TOL[dtype], label=f"masked plain {N}x{T} {dtype}")
    for norm in (False, True):  # no termination array (with truncation, then without)
        out, ref = run(ro, mask, term=False, normalize=norm)
        assert_parity(out, ref, TOL[dtype], label=f"masked no term {N}x{T} {dtype} norm={norm}")
    out, ref = run(ro, mask, term=False, trunc=False)
    assert_parity(out, ref, TOL[dtype], label=f"masked no flags {N}x{T} {dtype}")


def test_gae_masked_equals_gae_without_mask():
    ro = workloads.make_rollout(200, 300, seed=5, p_term=0.02, p_trunc=0.01)
    d = {k: to_device(v, DEV) for k, v in ro.items()}
    a1, r1 = rl.rlcs_gae_masked(d["r"], d["v"], None, d["term"], d["trunc"], d["bv"], d["boot"],
                                gamma=G, lam=L)
    a2, r2 = rl.rlcs_gae(d["r"], d["v"], d["term"], d["trunc"], d["bv"], d["boot"], gamma=G, lam=L)
    torch.cuda.synchronize()
    ref, _ = oracle.gae(ro["r"], ro["v"], ro["term"], ro["trunc"], ro["bv"], ro["boot"], gamma=G,
                        lam=L)
    assert_parity({"a": a1}, {"a": ref}, TOL["f32"], label="masked entry, no mask")
    assert_parity({"a": a2}, {"a": ref}, TOL["f32"], label="gae entry")


@pytest.mark.parametrize("N,T", [(64, 4096), (16, 8192), (512, 512)])
def test_gae_masked_multiturn(N, T):
    ro = workloads.make_multiturn(N, T, seed=N + T)
    for norm in (False, True):
        out, ref = run(ro, ro["mask"], normalize=norm, gamma=1.0, lam=0.95)
        assert_parity(out, ref, TOL["f32"], label=f"multiturn {N}x{T} norm={norm}")


def test_gae_masked_edge_cases():
    ro = workloads.make_rollout(40, 50, seed=9, p_term=0.05, p_trunc=0.05)
    zeros = np.zeros((40, 50), np.uint8)
    out, ref = run(ro, zeros)                       # every step skipped
    assert_parity(out, ref, TOL["f32"], label="all masked")
    assert float(out["adv"].abs().max()) == 0.0
    out, ref = run(ro, zeros, normalize=True)       # nothing takes part: mean 0, var 0
    assert_parity(out, ref, 1e-5, label="all masked, whitened")
    one = zeros.copy(); one[7, 13] = 1              # one step takes part: var 0
    out, ref = run(ro, one, normalize=True, eps=1e-2)
    assert_parity(out, ref, 1e-5, label="one unmasked, whitened")


def test_gae_masked_deterministic():
    ro = workloads.make_multiturn(64, 4096, seed=2)
    d = {k: to_device(v, DEV) for k, v in ro.items()}
    outs = [rl.rlcs_gae_masked(d["r"], d["v"], d["mask"], d["term"], None, None, d["boot"],
                               gamma=1.0, lam=0.95, normalize=True)[0] for _ in range(3)]
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1]) and torch.equal(outs[1], outs[2])


def test_gae_masked_workspace_reuse():
    """One whitening workspace serves calls of several shapes in turn, one-pass and two-pass.
    Only its 64-byte header is zero-filled; every record and partial starts as 0xff bytes."""
    ws = torch.full((rl.rlcs_workspace_size_masked(600, 1),), 255, dtype=torch.uint8, device=DEV)
    ws[:64] = 0
    for N, T, seed, var in ((600, 40, 1, 0), (7, 3000, 2, 0), (600, 40, 1, 1), (600, 40, 1, 0),
                            (64, 1024, 3, 1), (64, 1024, 3, 0)):
        ro = workloads.make_multiturn(N, T, seed=seed, mean_action=20, mean_obs=30)
        d = {k: to_device(v, DEV) for k, v in ro.items()}
        with variant(var):
            adv, _ = rl.rlcs_gae_masked(d["r"], d["v"], d["mask"], d["term"], None, None,
                                        d["boot"], gamma=1.0, lam=0.95, normalize=True, ws=ws)
        torch.cuda.synchronize()
        a, _ = oracle.gae_masked(ro["r"], ro["v"], ro["mask"], ro["term"], None, None, ro["boot"],
                                 gamma=1.0, lam=0.95)
        assert_parity({"adv": adv}, {"adv": oracle.normalize_advantages(a, ro["mask"], eps=1e-8)},
                      TOL["f32"], label=f"reuse {N}x{T} variant {var}")
        # the workspace's first 16 bytes hold the call's mean and 1/sqrt(var + eps), taken over
        # the kernel's float32 advantages: float32 rounding against the oracle's fp64 ones
        st = ws[:16].view(torch.float64).cpu().numpy()
        sel = a[ro["mask"] != 0]
        assert abs(st[0] - sel.mean()) <= 1e-6 * (1 + np.abs(sel).max())
        assert st[1] == pytest.approx(1 / np.sqrt(sel.var(ddof=1) + 1e-8), rel=1e-5)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("N,T", [(4096, 256), (64, 4096), (1000, 33), (3, 8192), (513, 1)])
def test_gae_masked_one_pass_and_two_pass_whitening(N, T, dtype):
    """Whitening in one kernel (every workgroup resident, advantages held in registers) and in
    two (a second kernel rewrites them), each against the oracle. Where every row lies within
    one wave the two forms scan each row alike, and the returns agree bit for bit."""
    ro = workloads.make_rollout(N, T, seed=N + 3 * T, dtype=dtype, p_term=0.03, p_trunc=0.03)
    mask = (np.random.default_rng(N + T).random((N, T)) < 0.7).astype(np.uint8)
    rets = []
    for var in (0, 1):
        with variant(var):
            out, ref = run(ro, mask, normalize=True)
        assert_parity(out, ref, TOL[dtype], label=f"{N}x{T} {dtype} variant {var}")
        rets.append(out["ret"])
    K = 4 if dtype == "f32" else 8
    if T % K == 0 and (64 * K) % T == 0:
        assert torch.equal(rets[0], rets[1])


@pytest.mark.parametrize("N,T", [(4500, 1024), (9000, 256)])
def test_gae_masked_whitened_many_workgroups(N, T):
    """More workgroups than one normalize workgroup adds up directly (4096): the partials are
    first added in blocks."""
    ro = workloads.make_multiturn(N, T, seed=N, mean_action=20, mean_obs=30)
    out, ref = run(ro, ro["mask"], normalize=True, gamma=1.0, lam=0.95, trunc=False)
    assert_parity(out, ref, TOL["f32"], label=f"whitened {N}x{T}")


def test_gae_masked_unaligned_outputs_whitened():
    """Advantages not 16-byte aligned: element-wise loads, stores and whitening."""
    N, T = 37, 301
    ro = workloads.make_rollout(N, T, seed=21, p_term=0.03, p_trunc=0.03)
    mask = (np.random.default_rng(21).random((N, T)) < 0.5).astype(np.uint8)
    d = {k: to_device(v, DEV) for k, v in ro.items()}
    buf = torch.zeros(N * T + 1, dtype=torch.float32, device=DEV)
    adv = buf[1:].view(N, T)
    assert adv.data_ptr() % 16 != 0
    rl.rlcs_gae_masked(d["r"], d["v"], to_device(mask, DEV), d["term"], d["trunc"], d["bv"],
                       d["boot"], adv, None, gamma=G, lam=L, normalize=True, want_ret=False)
    torch.cuda.synchronize()
    a, _ = oracle.gae_masked(ro["r"], ro["v"], mask, ro["term"], ro["trunc"], ro["bv"], ro["boot"],
                             gamma=G, lam=L)
    assert_parity({"adv": adv}, {"adv": oracle.normalize_advantages(a, mask, eps=1e-8)},
                  TOL["f32"], label="unaligned whitened")
