"""Throughput of the credit-assignment hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu] [--extra]

Workload: GAE over a 4096 x 256 float32 rollout buffer with termination and truncation flags,
truncation continuations and per-row bootstraps (seeded synthetic data). One step is one call
of rlcs_gae: load, coefficient build, scan, carry, epilogue and store of advantages and returns,
all inside one kernel launch.

Cold HBM: the timed steps rotate over enough independent input/output sets (well beyond the
256 MB Infinity Cache) that every step reads its inputs from HBM.

Prints one JSON line on stdout:
  value      effective bandwidth = algorithmic bytes / (timed time / K), GB/s
  roofline   the same figure against the 8 TB/s HBM peak
  cpu_baseline  the fp64 oracle on the host, single thread, on a bounded sample
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
N, T = 4096, 256
GAMMA, LAM = 0.99, 0.95
METRIC = "effective HBM GB/s (% of MI355X peak) + Gsteps/s, GAE 4096×256 fp32"


def algorithmic_bytes(N, T, *, dtype_bytes=4, trunc=True, boot=True, outputs=2):
    """Each input read once and each output written once, dense: r, v (data), term (1 B),
    trunc (1 B) and bv (data) when truncation is on, boot [N], advantages and returns (4 B)."""
    per = 2 * dtype_bytes + 1 + (1 + dtype_bytes if trunc else 0) + 4 * outputs
    return N * T * per + (N * dtype_bytes if boot else 0)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--sets", type=int, default=32, help="rotated input/output sets (cold HBM)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--extra", action="store_true", help="also time the other workloads (stderr)")
    return ap.parse_args()


def cpu_baseline(ro, seconds):
    """The fp64 oracle on the same workload, single thread, repeated for about `seconds`."""
    import oracle
    a = (ro["r"], ro["v"], ro["term"], ro["trunc"], ro["bv"], ro["boot"])
    oracle.gae(*a, gamma=GAMMA, lam=LAM)  # warm-up (also builds/loads the library)
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.gae(*a, gamma=GAMMA, lam=LAM)
        reps += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    per_call = el / reps
    return {
        "value": round(algorithmic_bytes(N, T) / per_call / 1e9, 3),
        "unit": "GB/s",
        "cores": 1,
        "kind": "oracle",
        "sample": f"GAE {N}x{T} fp32+trunc, full workload repeated {reps}x in {el:.1f} s "
                  f"(fp64 sequential C, {per_call * 1e3:.1f} ms/call, "
                  f"{N * T / per_call / 1e9:.4f} Gsteps/s)",
    }


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); rows are independent, so "
              "a multi-GPU run would shard rows with no exchange and is not part of this build.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import workloads
    import paper_2608_17641_amd as rl
    from paper_2608_17641_amd.build import is_stale, build

    if is_stale():
        build(force=False)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    ro = workloads.make_rollout(N, T, seed=0, p_term=0.02, p_trunc=0.01)
    names = ("r", "v", "term", "trunc", "bv", "boot")
    base = {k: torch.from_numpy(ro[k]).to(dev) for k in names}
    S = max(1, args.sets)
    sets = []
    for _ in range(S):
        s = {k: v.clone() for k, v in base.items()}
        s["adv"] = torch.empty((N, T), dtype=torch.float32, device=dev)
        s["ret"] = torch.empty((N, T), dtype=torch.float32, device=dev)
        sets.append(s)

    def step(i):
        s = sets[i % S]
        rl.rlcs_gae(s["r"], s["v"], s["term"], s["trunc"], s["bv"], s["boot"], s["adv"], s["ret"],
                    gamma=GAMMA, lam=LAM)

    # parity of the timed configuration before timing
    import oracle
    step(0)
    torch.cuda.synchronize()
    o_adv, o_ret = oracle.gae(ro["r"], ro["v"], ro["term"], ro["trunc"], ro["bv"], ro["boot"],
                              gamma=GAMMA, lam=LAM)
    for got, ref in ((sets[0]["adv"], o_adv), (sets[0]["ret"], o_ret)):
        err = float(np.max(np.abs(got.double().cpu().numpy() - ref)))
        if err > 1e-5 * (1 + float(np.max(np.abs(ref)))):
            raise SystemExit(f"parity failure before timing: max err {err}")

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    eager_adv = sets[(args.steps - 1) % S]["adv"].clone()

    # The timed steps are replayed from a HIP graph so that host-side launch cost (Python,
    # ctypes) does not starve the GPU; each graph node is one rlcs_gae kernel launch.
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for i in range(args.steps):
            step(i)
    graph.replay()
    torch.cuda.synchronize()
    if not torch.equal(sets[(args.steps - 1) % S]["adv"], eager_adv):
        raise SystemExit("graph replay differs from the eager launch")
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    graph.replay()
    end.record()
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(end)
    per_step_s = total_ms / 1e3 / args.steps
    nbytes = algorithmic_bytes(N, T)
    gbs = nbytes / per_step_s / 1e9

    # Context (stderr): full-call time of one eager call through the Python binding, the
    # paper's protocol (per-call events, median of 50, min over 5 trials).
    trials = []
    for _ in range(5):
        ts = []
        for i in range(50):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            a.record(); step(i); b.record()
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        trials.append(float(np.median(ts)))
    print(f"full-call (per-call events, min of 5 medians): {min(trials) * 1e3:.2f} us", file=sys.stderr)

    out = {
        "metric": METRIC,
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(total_ms / args.steps, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"GAE {N}x{T} fp32, term+trunc, bootstrap, cold HBM "
                               f"({S} rotated input/output sets)",
                   "N": N, "T": T, "algorithmic_bytes": nbytes,
                   "gsteps_per_s": round(N * T / per_step_s / 1e9, 2),
                   "pct_of_peak": round(100 * gbs / PEAK_HBM_GBS, 2)},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 2), "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4), "traffic": None},
    }
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(ro, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
