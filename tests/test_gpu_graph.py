"""Back-to-back calls captured in a HIP graph: the single-token split-K kernels complete
their K split inside the kernel with per-tile arrival counters that each call re-arms,
and consecutive kernel nodes of a graph may run with no memory fence in between.
Each call of the graph gets a different token, so a call that found a counter not yet
re-armed (and took a stale partial sum, or stored no output) would differ from the
eager result.  The graph is replayed several times, with eager work and
synchronizations in between, and every call of every replay is compared bit for bit
with the same call made eagerly."""
import numpy as np
import pytest

import workloads as W
from helpers import GpuProblem

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2408_06003_amd as L  # noqa: E402

CALLS = 12
TOKENS = 4


@pytest.mark.parametrize("cid,sid,entry", [(3, 0, "two-call"), (3, 0, "fused"), (5, 0, "two-call"),
                                           (5, 0, "fused"), (2, 0, "two-call")])
def test_graph_of_split_calls_matches_eager(cid, sid, entry, tune):
    tune(GEMV_KIND=2)  # the split-K kernel with in-kernel completion
    print(f"\n[case] graph of {CALLS} split-K calls, config {cid}/{sid}, {entry}", flush=True)
    inp = W.make_inputs(cid, sid, M=1)
    gp = GpuProblem(inp)
    g = gp.g
    M = 1
    rng = np.random.default_rng(17)
    acts = []
    for t in range(TOKENS):
        a = inp.act.astype(np.float32) * np.float32(0.5 + rng.random())
        a = np.roll(a, 37 * t, axis=1)
        acts.append(torch.from_numpy(a.astype(np.float16)).cuda())
    od = torch.int32 if inp.act_kind == W.ACT_INT8 else torch.float16
    outs = [torch.zeros((M, inp.N), dtype=od, device="cuda") for _ in range(CALLS)]
    ws_fused = g.fused_workspace(M)
    ws = g.workspace(M)
    plan_splits = L.workspace_size(gp.p, M) > 0
    assert plan_splits or entry == "fused", "the forced split-K plan needs a workspace"
    tables = g.tables(M)

    def call(i):
        a = acts[i % TOKENS]
        if entry == "fused":
            L.mpgemm_fused(gp.p, M, a, g.packed, outs[i], g.out_dtype_code(od), False, workspace=ws_fused)
        else:
            L.precompute(gp.p, M, a, tables)
            L.mpgemm(gp.p, M, tables, g.packed, outs[i], g.out_dtype_code(od), False, workspace=ws)

    # eager reference, each call on its own
    refs = []
    for i in range(CALLS):
        call(i)
        torch.cuda.synchronize()
        refs.append(outs[i].clone())
    for i in range(TOKENS, CALLS):
        assert torch.equal(refs[i], refs[i % TOKENS]), "eager calls are not reproducible"

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        for i in range(CALLS):
            call(i)
    torch.cuda.synchronize()
    for rep in range(4):
        for o in outs:
            o.zero_()
        call(rep % CALLS)  # eager work between replays
        torch.cuda.synchronize()
        outs[rep % CALLS].zero_()
        graph.replay()
        torch.cuda.synchronize()
        for i in range(CALLS):
            assert torch.equal(outs[i], refs[i]), f"replay {rep}, call {i}: differs from the eager result"
    if ws is not None:
        assert not ws[:L.WORKSPACE_ZERO_BYTES].any(), "arrival counters not re-armed"
    if ws_fused is not None:
        assert not ws_fused[:L.WORKSPACE_ZERO_BYTES].any(), "arrival counters not re-armed"
