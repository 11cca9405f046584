"""The entry point that allocates nothing, rlcs_gae_masked_noalloc, through the C ABI: its
outputs against those of rlcs_gae_masked given a workspace of its own (same kernels, so the
results agree bit for bit; the bar is the parity tolerance) on two calls in a row, the second
with a smaller input, so that the built-in workspace holds the first call's contents when the
second starts; whitened and plain; and its size limit."""
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
from paper_2608_17641_amd import _native  # noqa: E402

DEV = torch.device("cuda:0")
G, L = 0.99, 0.95


def _inputs(N, T, seed, dtype):
    ro = workloads.make_rollout(N, T, seed=seed, dtype=dtype, p_term=0.03, p_trunc=0.02)
    mask = (np.random.default_rng(seed + 1).random((N, T)) < 0.6).astype(np.uint8)
    d = {k: to_device(v, DEV) for k, v in ro.items()}
    return ro, mask, d, to_device(mask, DEV)


def _both(d, m, N, T, normalize):
    """(noalloc outputs, outputs of the entry point with a caller workspace)."""
    a0 = torch.empty((N, T), dtype=torch.float32, device=DEV)
    r0 = torch.empty((N, T), dtype=torch.float32, device=DEV)
    print(f"rlcs_gae_masked_noalloc N={N} T={T} normalize={normalize}", flush=True)
    rl.rlcs_gae_masked_noalloc(d["r"], d["v"], m, d["term"], d["trunc"], d["bv"], d["boot"], a0, r0,
                               gamma=G, lam=L, normalize=normalize)
    ws = torch.zeros(rl.rlcs_workspace_size_masked(N, T), dtype=torch.uint8, device=DEV)
    a1, r1 = rl.rlcs_gae_masked(d["r"], d["v"], m, d["term"], d["trunc"], d["bv"], d["boot"],
                                gamma=G, lam=L, normalize=normalize, ws=ws)
    torch.cuda.synchronize()
    return {"adv": a0, "ret": r0}, {"adv": a1, "ret": r1}


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_noalloc_matches_workspace_entry_point(dtype):
    # first call: the most rows the built-in workspace holds; second: a smaller call
    for N, T, seed in ((65536, 24, 3), (1000, 300, 4)):
        ro, mask, d, m = _inputs(N, T, seed, dtype)
        for normalize in (True, False):
            got, want = _both(d, m, N, T, normalize)
            want_np = {k: v.double().cpu().numpy() for k, v in want.items()}
            assert_parity(got, want_np, TOL[dtype], label=f"noalloc {N}x{T} {dtype} norm={normalize}")
            # same kernels on the same inputs: bitwise equal as well
            assert torch.equal(got["adv"], want["adv"]) and torch.equal(got["ret"], want["ret"])
        if N <= 1000:
            a, r = oracle.gae_masked(ro["r"], ro["v"], mask, ro["term"], ro["trunc"], ro["bv"],
                                     ro["boot"], gamma=G, lam=L)
            ref = {"adv": oracle.normalize_advantages(a, mask, eps=1e-8), "ret": r}
            rl.rlcs_gae_masked_noalloc(d["r"], d["v"], m, d["term"], d["trunc"], d["bv"], d["boot"],
                                       got["adv"], got["ret"], gamma=G, lam=L, normalize=True)
            torch.cuda.synchronize()
            assert_parity(got, ref, TOL[dtype], label=f"noalloc vs oracle {N}x{T} {dtype}")


def test_noalloc_rejects_more_rows_than_its_workspace():
    fake = 0x10000
    lib = _native.load()
    for norm in (0, 1):
        rc = lib.rlcs_gae_masked_noalloc(fake, fake, None, None, None, None, None, fake, None,
                                         65537, 4, G, L, norm, 1e-8, _native.RLCS_F32, None)
        assert rc == _native.RLCS_ERR_WORKSPACE
