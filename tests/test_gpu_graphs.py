"""HIP graph capture of the entry points: the calls that keep state in a workspace (split rows,
split time-major columns, whitening partials) and the staged one (full-form Retrace) are
captured together, replayed three times with eager work and synchronisations in between, and
every replay is compared bit for bit with the eager results (every path is deterministic)."""
import pytest

from cases import to_device
import workloads

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2608_17641_amd as rl  # noqa: E402

DEV = torch.device("cuda:0")
G, L = 0.99, 0.95


def test_graph_replays_equal_eager():
    rows = {k: to_device(v, DEV) for k, v in workloads.make_rollout(64, 8192, seed=1).items()}
    tm = {k: to_device(v, DEV) for k, v in workloads.make_rollout_time_major(1024, 256, seed=2).items()}
    mt = {k: to_device(v, DEV) for k, v in workloads.make_multiturn(64, 2048, seed=3).items()}
    rf = {k: to_device(v, DEV) for k, v in workloads.make_retrace_full(256, 129, 5, seed=4).items()}
    ws_rows = rl.make_workspace(64, 8192, DEV)
    ws_cols = rl.make_workspace_columns(256, 1024, DEV)
    ws_mask = torch.zeros(rl.rlcs_workspace_size_masked(64, 2048), dtype=torch.uint8, device=DEV)

    def outputs():
        return [torch.empty((64, 8192), device=DEV), torch.empty((64, 8192), device=DEV),
                torch.empty((1024, 256), device=DEV).t(), torch.empty((1024, 256), device=DEV).t(),
                torch.empty((64, 2048), device=DEV), torch.empty((64, 2048), device=DEV),
                torch.empty((256, 129), device=DEV), torch.empty((256, 129), device=DEV)]

    def run(o):
        rl.rlcs_gae(rows["r"], rows["v"], rows["term"], rows["trunc"], rows["bv"], rows["boot"],
                    o[0], o[1], gamma=G, lam=L, ws=ws_rows)
        rl.rlcs_gae_strided(tm["r"].t(), tm["v"].t(), tm["term"].t(), tm["trunc"].t(), tm["bv"].t(),
                            tm["boot"], o[2], o[3], gamma=G, lam=L, ws=ws_cols)
        rl.rlcs_gae_masked(mt["r"], mt["v"], mt["mask"], mt["term"], None, None, mt["boot"], o[4],
                           o[5], gamma=1.0, lam=L, normalize=True, ws=ws_mask)
        rl.rlcs_retrace_full(rf["r"], rf["q3"], rf["pi3"], rf["actions"], rf["mu"], rf["term"],
                             rf["trunc"], rf["bv"], rf["boot"], o[6], o[7], gamma=G, lam=L)

    eager = outputs()
    run(eager)
    torch.cuda.synchronize()
    for o in eager:
        assert bool(torch.isfinite(o).all())

    captured = outputs()
    run(captured)  # warm-up on the capture buffers (first-call set-up happens outside the graph)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run(captured)
    for rep in range(3):
        for o in captured:
            o.fill_(float("nan"))
        other = outputs()
        run(other)  # eager work on the same workspaces between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for i, (e, c) in enumerate(zip(eager, captured)):
            assert torch.equal(e, c), f"replay {rep}: output {i} differs from the eager result"
        for i, (e, c) in enumerate(zip(eager, other)):
            assert torch.equal(e, c), f"eager call {rep}: output {i} differs"
    assert int(ws_rows[8:12].view(torch.int32).item()) == 0
    assert int(ws_cols[8:12].view(torch.int32).item()) == 0
