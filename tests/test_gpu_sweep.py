"""GPU parity at the large bfloat16 sweep sizes (N in {16384, 65536} x T in {64, 512, 2048}):
full-size runs of all seven estimators, compared with the oracle element by element over the
whole tensors. The oracle runs on blocks of rows in parallel host threads (its C routines
release Python's lock); the bar is the whole-tensor form, max |gpu - oracle| <= 1e-3 * (1 +
max |oracle|) per output, with both maxima taken over every block."""
import concurrent.futures as cf
import os

import numpy as np
import pytest

from cases import SEVEN, TOL, device_inputs, gpu_run, mismatch_report, oracle_run
import workloads

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

DEV = torch.device("cuda:0")
SWEEP = [(16384, 64), (16384, 512), (16384, 2048), (65536, 64), (65536, 512), (65536, 2048)]
BLOCK_STEPS = 1 << 22  # oracle block: rows holding about 4M steps
THREADS = max(1, min(16, len(os.sched_getaffinity(0))))


@pytest.mark.parametrize("N,T", SWEEP)
def test_bf16_sweep_whole_tensors(N, T):
    ro = workloads.make_rollout(N, T, 0, dtype="bf16", p_term=0.005, p_trunc=0.005)
    d = device_inputs(ro, DEV)
    rows_per_block = max(1, BLOCK_STEPS // T)
    blocks = [(lo, min(N, lo + rows_per_block)) for lo in range(0, N, rows_per_block)]
    print(f"sweep {N}x{T}: {len(blocks)} oracle blocks on {THREADS} threads", flush=True)
    with cf.ThreadPoolExecutor(THREADS) as ex:
        for name in SEVEN + ("prefix_starts",):
            out = gpu_run(name, d, gamma=0.99, lam=0.95)
            host = {k: v.cpu().numpy() for k, v in out.items()}  # float32, whole tensors
            del out

            def check_block(b):
                lo, hi = b
                ref = oracle_run(name, ro, gamma=0.99, lam=0.95, rows=slice(lo, hi))
                return {k: (float(np.max(np.abs(host[k][lo:hi].astype(np.float64) - r))),
                            float(np.max(np.abs(r)))) for k, r in ref.items()}

            worst = {}
            for res in ex.map(check_block, blocks):
                for k, (err, mag) in res.items():
                    e0, m0 = worst.get(k, (0.0, 0.0))
                    worst[k] = (max(e0, err), max(m0, mag))
            for k, (err, mag) in worst.items():
                bound = TOL["bf16"] * (1.0 + mag)
                if err > bound:  # locate the first block that breaks the bar, for the report
                    for lo, hi in blocks:
                        r = oracle_run(name, ro, gamma=0.99, lam=0.95, rows=slice(lo, hi))[k]
                        g = host[k][lo:hi]
                        if np.max(np.abs(g.astype(np.float64) - r)) > bound:
                            raise AssertionError(f"{name} {k} {N}x{T}: max err {err:.3e} > {bound:.3e}; "
                                                 f"rows {lo}..{hi}: " + mismatch_report(g, r, bound))
                assert err <= bound
            del host
    del d
    torch.cuda.empty_cache()
