"""The operator inside HIP graphs (how bench.py times it, and how a caller
removes the host's per-launch latency): calls captured on torch's capturing
stream replay with results bit-identical to eager calls.  Every replay is
checked, with eager work and synchronisations between replays, and the
outputs poisoned before each one (so a replay that wrote nothing fails)."""
import numpy as np
import pytest
import torch

from paper_2505_08098_amd import workloads as W

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _capture(fn):
    side = torch.cuda.Stream(DEV)
    side.wait_stream(torch.cuda.current_stream(DEV))
    with torch.cuda.stream(side):
        fn()                                   # eager warm-up on the side stream
    torch.cuda.current_stream(DEV).wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        out = fn()
    torch.cuda.synchronize()
    return g, out


@pytest.mark.parametrize("k,piece", [(2, "4"), (1, None), (5, None)])
def test_forward_graph_replays_equal_eager(gpu, k, piece, monkeypatch):
    if piece:
        monkeypatch.setenv("F3S_PIECE_BLOCKS", piece)   # split windows: two launches
    c = W.make_config(k)
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    assert piece is None or plan.info["n_split"] > 0
    q, kk, v = (_dev(c[x]) for x in ("Q", "K", "V"))
    O = torch.empty((c["N"], c["d"]), dtype=torch.float32, device=DEV)
    lse = torch.empty(c["N"], dtype=torch.float32, device=DEV)
    ref, ref_lse = gpu.forward(plan, q, kk, v, scale=c["scale"])
    torch.cuda.synchronize()
    g, _ = _capture(lambda: gpu.forward(plan, q, kk, v, scale=c["scale"], out=O, lse=lse))
    for r in range(4):
        O.fill_(float("nan"))
        lse.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(O, ref) and torch.equal(lse, ref_lse), r
        _ = (q.float() * 2).sum().item()          # eager work between replays


def test_backward_graph_replays_equal_eager(gpu):
    c = W.make_config(2)
    plan = gpu.Plan(_dev(c["row_ptr"]), _dev(c["col_idx"]), c["N"])
    plan_t = plan.transpose()
    q, kk, v = (_dev(c[x]) for x in ("Q", "K", "V"))
    g16 = _dev(np.random.default_rng(3).standard_normal(c["Q"].shape).astype(np.float16))
    O, lse = gpu.forward(plan, q, kk, v, scale=c["scale"])
    ref = gpu.backward(plan, plan_t, q, kk, v, O, g16, lse, scale=c["scale"])
    torch.cuda.synchronize()
    graph, outs = _capture(lambda: gpu.backward(plan, plan_t, q, kk, v, O, g16, lse,
                                                scale=c["scale"]))
    for r in range(3):
        for x in outs:
            x.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for a, b in zip(outs, ref):
            assert torch.equal(a, b), r
