"""The library's calls captured into a HIP graph give, on every replay, the
same bits as the same calls run eagerly (the library issues no memset or
allocation, so its calls are safe to capture)."""
import numpy as np
import pytest
import torch

from paper_2412_04787_amd import dqt, workloads as W

from gpu_util import DEV, log, make_weight, weight_codes_dev

pytestmark = pytest.mark.gpu


def test_graph_replays_match_eager(lib):
    M, d_in, d_out = 1024, 256, 384
    q = W.draw_ternary((d_out, d_in), 5, 97, 1)
    w = make_weight(d_out, d_in, "ternary", -1, 1, 0.02, tensor_id=3)
    X = torch.from_numpy(W.draw_normal((M, d_in), 1.0, 5, 97, 2)).to(torch.bfloat16).to(DEV)
    dY = torch.from_numpy(W.draw_normal((M, d_out), 1e-2, 5, 97, 3)).to(torch.bfloat16).to(DEV)
    Wq0 = weight_codes_dev(q, "ternary")
    ws = dqt.workspace(dqt.dqt_linear_bwd_workspace(w, M))
    fws = dqt.workspace(dqt.dqt_linear_fwd_workspace(w))

    def make_bufs():
        return dict(Wq=Wq0.clone(), Xq=torch.empty((M, d_in), dtype=torch.int8, device=DEV),
                    xdq=torch.empty((M,), dtype=torch.float32, device=DEV),
                    Y=torch.empty((M, d_out), dtype=torch.bfloat16, device=DEV),
                    dX=torch.empty((M, d_in), dtype=torch.bfloat16, device=DEV),
                    dW=torch.empty((d_out, d_in), dtype=torch.float32, device=DEV),
                    cnt=torch.zeros((2,), dtype=torch.int64, device=DEV))

    def step(b):
        dqt.dqt_linear_fwd(w, b["Wq"], X, M, dqt.DQT_I8, b["Xq"], b["xdq"], b["Y"], fws)
        dqt.dqt_linear_bwd(w, b["Wq"], b["Xq"], dqt.DQT_I8, b["xdq"], dY, M, dqt.DQT_BF16,
                           b["dX"], b["dW"], ws)
        dqt.dqt_sr_update(w, b["Wq"], b["dW"], 1e-2, 11, 1, b["cnt"])

    eager = make_bufs()
    step(eager)                       # eager reference of one step from the initial codes
    torch.cuda.synchronize()

    g_bufs = make_bufs()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(g_bufs)
    torch.cuda.synchronize()
    for rep in range(3):
        log(f"graph replay {rep}")
        g_bufs["Wq"].copy_(Wq0)       # eager work between replays
        g_bufs["cnt"].zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k in ("Xq", "xdq", "Y", "dX", "dW", "Wq", "cnt"):
            assert torch.equal(g_bufs[k], eager[k]), (rep, k)
