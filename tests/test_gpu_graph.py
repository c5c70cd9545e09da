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


def test_graph_replays_of_fused_adamw_and_variant_calls(lib):
    """The fused backward + SR call, AdamW with SR and the force-to-update
    variant (whose selection state lives in the workspace) replay from a
    graph with the eager results, replay after replay."""
    M, d_in, d_out = 1024, 256, 384
    q = W.draw_ternary((d_out, d_in), 6, 98, 1)
    w = make_weight(d_out, d_in, "ternary", -1, 1, 0.02, tensor_id=4)
    X = torch.from_numpy(W.draw_normal((M, d_in), 1.0, 6, 98, 2)).to(torch.bfloat16).to(DEV)
    dY = torch.from_numpy(W.draw_normal((M, d_out), 1e-2, 6, 98, 3)).to(torch.bfloat16).to(DEV)
    g = torch.from_numpy(W.draw_normal((d_out, d_in), 1e-2, 6, 98, 4)).to(DEV)
    Wq0 = weight_codes_dev(q, "ternary")
    hp = dqt.adamw(1e-3, 0.9, 0.95, 1e-8, 0.1)
    bf = dqt.DQT_BF16

    def make_bufs():
        b = dict(Wq=Wq0.clone(), Wa=Wq0.clone(), Wv=Wq0.clone(),
                 Xq=torch.empty((M, d_in), dtype=torch.int8, device=DEV),
                 xdq=torch.empty((M,), dtype=torch.float32, device=DEV),
                 dX=torch.empty((M, d_in), dtype=torch.bfloat16, device=DEV),
                 m=torch.zeros((d_out, d_in), dtype=torch.float32, device=DEV),
                 v=torch.zeros((d_out, d_in), dtype=torch.float32, device=DEV),
                 cnt=torch.zeros((6,), dtype=torch.int64, device=DEV))
        b["io"] = dqt.linear_io([dict(w=w, Wq=b["Wq"], Xq=b["Xq"], xdq=b["xdq"], dY=dY, dX=b["dX"])])
        b["ioa"] = dqt.linear_io([dict(w=w, Wq=b["Wa"], dW=g)])
        b["iov"] = dqt.linear_io([dict(w=w, Wq=b["Wv"], dW=g)])
        b["ws"] = dqt.workspace(dqt.dqt_linear_bwd_batch_workspace(b["io"], M))
        b["vws"] = dqt.workspace(dqt.dqt_update_variant_workspace(1))
        return b

    def step(b):
        dqt.dqt_act_quant(X, dqt.DQT_I8, b["Xq"], b["xdq"])
        dqt.dqt_linear_bwd_sr_batch(b["io"], M, dqt.DQT_I8, bf, bf, bf, 1e-2, 11, 2, b["cnt"][0:2],
                                    b["ws"])
        dqt.dqt_adamw_sr_update_batch(b["ioa"], [b["m"]], [b["v"]], hp, 11, 2, b["cnt"][2:4])
        dqt.dqt_update_variant_batch(b["iov"], 1e-2, 11, 2, dqt.DQT_UPD_FORCE_CHANGE, 0.2,
                                     b["cnt"][4:6], b["vws"])

    eager = make_bufs()
    step(eager)
    torch.cuda.synchronize()
    g_bufs = make_bufs()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(g_bufs)
    torch.cuda.synchronize()
    for rep in range(3):
        log(f"graph replay {rep}")
        for k in ("Wq", "Wa", "Wv"):
            g_bufs[k].copy_(Wq0)      # eager work between replays
        g_bufs["m"].zero_()
        g_bufs["v"].zero_()
        g_bufs["cnt"].zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k in ("Xq", "xdq", "dX", "Wq", "Wa", "Wv", "m", "v", "cnt"):
            assert torch.equal(g_bufs[k], eager[k]), (rep, k)
