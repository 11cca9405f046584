"""GPU parity past 2^31 elements: every offset computation of the rows kernel and the column
scans runs in 64-bit. One bfloat16 rollout of 65600 x 32768 steps (2.15e9 elements, about 30 GB
of device memory with the outputs) is generated on the device with a seeded torch generator;
sampled rows (row-major GAE and eligibility traces) and sampled environments (the same buffers
read time-major through the strided entry point) are copied back and checked against the fp64
oracle on exactly the same values. Bar: 1e-3 relative, the bfloat16-input bar."""
import numpy as np
import pytest

from cases import TOL, assert_parity
import oracle

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2608_17641_amd as rl  # noqa: E402

DEV = torch.device("cuda:0")
G, L = 0.99, 0.95


def _host_bf16(t):
    """A bfloat16 device tensor as the uint16 bit patterns the oracle widens."""
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


@pytest.fixture(scope="module")
def big():
    N, T = 65600, 32768
    assert N * T > 2 ** 31
    free, _ = torch.cuda.mem_get_info(DEV)
    if free < 40 * 2 ** 30:
        pytest.skip("needs about 40 GB of free device memory")
    g = torch.Generator(device=DEV)
    g.manual_seed(7)
    d = {
        "r": torch.randn((N, T), generator=g, device=DEV, dtype=torch.bfloat16),
        "v": torch.randn((N, T), generator=g, device=DEV, dtype=torch.bfloat16),
        "term": (torch.rand((N, T), generator=g, device=DEV) < 0.002).to(torch.uint8),
        "boot": torch.randn((N,), generator=g, device=DEV, dtype=torch.bfloat16),
    }
    torch.cuda.synchronize()
    yield N, T, d
    del d
    torch.cuda.empty_cache()


def test_rows_past_2_31_elements(big):
    N, T, d = big
    adv, ret = rl.rlcs_gae(d["r"], d["v"], d["term"], None, None, d["boot"], gamma=G, lam=L)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, N // 2, N - 2, N - 1],
                                     np.random.default_rng(3).integers(0, N, 4)]))
    idx = torch.from_numpy(rows).to(DEV)
    sub = {k: (_host_bf16(v.index_select(0, idx)) if v.dtype == torch.bfloat16 else
               v.index_select(0, idx).cpu().numpy()) for k, v in d.items()}
    a_ref, r_ref = oracle.gae(sub["r"], sub["v"], sub["term"], None, None, sub["boot"], gamma=G, lam=L)
    assert_parity({"adv": adv.index_select(0, idx), "ret": ret.index_select(0, idx)},
                  {"adv": a_ref, "ret": r_ref}, TOL["bf16"], label="GAE rows past 2^31")
    del adv, ret
    z = rl.rlcs_elig_trace(d["r"], d["term"], None, gamma=G, lam=L)
    torch.cuda.synchronize()
    z_ref = oracle.elig_trace(sub["r"], sub["term"], None, gamma=G, lam=L)
    assert_parity({"z": z.index_select(0, idx)}, {"z": z_ref}, TOL["bf16"], label="elig rows past 2^31")


def test_time_major_past_2_31_elements(big):
    """The same buffers read time-major: [T', N'] = [65600, 32768], environment n at column n."""
    N, T, d = big
    Tt, Nt = N, T  # 65600 steps of 32768 environments
    bt = d["boot"].new_zeros((Nt,))
    bt[: min(Nt, N)] = d["boot"][: min(Nt, N)]
    ws = rl.make_workspace_columns(Nt, Tt, DEV)
    adv, ret = rl.rlcs_gae_strided(d["r"].t(), d["v"].t(), d["term"].t(), None, None, bt,
                                   gamma=G, lam=L, ws=ws)
    torch.cuda.synchronize()
    cols = np.unique(np.concatenate([[0, Nt - 1], np.random.default_rng(4).integers(0, Nt, 3)]))
    idx = torch.from_numpy(cols).to(DEV)
    # environment n's steps are column n of the [Tt, Nt] storage; as [N, T] rows for the oracle
    sub = {k: d[k].index_select(1, idx).t().contiguous() for k in ("r", "v", "term")}
    host = {k: (_host_bf16(v) if v.dtype == torch.bfloat16 else v.cpu().numpy()) for k, v in sub.items()}
    boot = _host_bf16(bt.index_select(0, idx))
    a_ref, r_ref = oracle.gae(host["r"], host["v"], host["term"], None, None, boot, gamma=G, lam=L)
    # outputs are [N', T'] views of [T', N'] storage
    assert_parity({"adv": adv.index_select(0, idx), "ret": ret.index_select(0, idx)},
                  {"adv": a_ref, "ret": r_ref}, TOL["bf16"], label="GAE time-major past 2^31")
