"""The structured inference call (fq_frame_apply_tff) captured into a HIP graph: several
replays, with eager work and synchronizations between them, each give exactly the eager
call's output (the library records no memset into a graph; every step is a kernel)."""
import numpy as np
import pytest

import oracle as O
from fq_inputs import tff
from fq_testutil import need_gpu

pytestmark = pytest.mark.gpu


def _frame(torch, fq, d, k, rho, seed):
    R1, R2 = tff.rotation_factors(d, np.random.SeedSequence(seed))
    return fq.Frame(d, k, rho, torch.from_numpy(R1.astype(np.float32)).cuda(),
                    torch.from_numpy(R2.astype(np.float32)).cuda())


@pytest.mark.parametrize("n", [1, 8])
def test_frame_apply_tff_graph_replays_match_eager(n):
    torch = need_gpu()
    import paper_2403_06082_amd as fq
    Fo = _frame(torch, fq, 200, 55, 4, 5)
    Fi = _frame(torch, fq, 136, 37, 4, 6)
    rng = np.random.default_rng(n)
    codes = rng.integers(0, 4, size=(Fo.K, Fi.K))
    words = torch.from_numpy(O.pack2(codes).view(np.int32)).cuda()
    sc = torch.from_numpy(rng.uniform(0.01, 0.1, Fo.K).astype(np.float32)).cuda()
    ze = torch.from_numpy(rng.integers(0, 4, Fo.K).astype(np.float32)).cuda()
    X = torch.from_numpy(rng.standard_normal((n, 136)).astype(np.float32)).cuda()
    ws = torch.empty(fq.fq_frame_apply_tff_workspace_bytes(Fo, Fi), dtype=torch.uint8,
                     device="cuda")
    Y = torch.empty((n, 200), dtype=torch.float32, device="cuda")
    fq.fq_frame_apply_tff(X, words, sc, ze, Fo, Fi, Y=Y, ws=ws)
    torch.cuda.synchronize()
    ref = Y.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fq.fq_frame_apply_tff(X, words, sc, ze, Fo, Fi, Y=Y, ws=ws,
                              stream=torch.cuda.current_stream())
    for i in range(4):
        Y.fill_(float("nan"))
        ws.fill_(0xFF)                                     # eager work between replays
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(Y, ref), f"replay {i}"
    # the inputs change between replays: the graph reads them in place
    X.mul_(2.0)
    g.replay()
    torch.cuda.synchronize()
    Y2 = torch.empty_like(Y)
    fq.fq_frame_apply_tff(X, words, sc, ze, Fo, Fi, Y=Y2, ws=ws)
    torch.cuda.synchronize()
    assert torch.equal(Y, Y2)
