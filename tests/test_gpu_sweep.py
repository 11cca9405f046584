"""GPU parity at the large bfloat16 sweep sizes: full-size runs, oracle on sampled rows."""
import numpy as np
import pytest

from cases import SEVEN, TOL, assert_parity, device_inputs, gpu_run, oracle_run
import workloads

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

DEV = torch.device("cuda:0")


SWEEP = [(16384, 64), (16384, 512), (16384, 2048), (65536, 64), (65536, 512), (65536, 2048)]


@pytest.mark.parametrize("N,T", SWEEP)
def test_bf16_sweep_sampled_rows(N, T):
    """Full-size bfloat16 runs of all seven estimators; the oracle checks 66 sampled rows
    (first, last and 64 random ones) of every output."""
    ro = workloads.make_rollout(N, T, 0, dtype="bf16", p_term=0.005, p_trunc=0.005)
    d = device_inputs(ro, DEV)
    rows = np.unique(np.concatenate([[0, N - 1], np.random.default_rng(1).integers(0, N, 64)]))
    rows_t = torch.from_numpy(rows).to(DEV)
    for name in SEVEN + ("prefix_starts",):
        out = gpu_run(name, d, gamma=0.99, lam=0.95)
        sampled = {k: v.index_select(0, rows_t) for k, v in out.items()}
        torch.cuda.synchronize()
        ref = oracle_run(name, ro, gamma=0.99, lam=0.95, rows=rows)
        assert_parity(sampled, ref, TOL["bf16"], label=f"{name} {N}x{T}")
        del out, sampled
    del d
    torch.cuda.empty_cache()
