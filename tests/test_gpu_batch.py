"""Batch entry points: a batch of linears gives the results of the
single-linear calls (bit-exact where those are bit-exact) and matches the
oracle, including linears that share one quantised input."""
import numpy as np
import pytest
import torch

from oracle import dqt_oracle as O
from paper_2412_04787_amd import dqt, workloads as W

from gpu_util import (DEV, gemm_close, log, make_weight, run_fwd, to_dev, weight_codes_dev,
                      weight_codes_host)

pytestmark = pytest.mark.gpu
SEED = 4321

BATCHES = [
    # (M, [(d_in, d_out, input_index)], wfmt, qmin, qmax, act, env)
    (1000, [(256, 256, 0), (256, 384, 0), (256, 128, 0), (384, 256, 1)], "ternary", -1, 1, "i8", "bf16"),
    (777, [(96, 208, 0), (96, 48, 0), (208, 96, 1)], "i8", -127, 127, "i8", "bf16"),
    (640, [(128, 256, 0), (256, 128, 1)], "ternary", -1, 1, "e4m3", "bf16"),
    (300, [(64, 80, 0), (80, 64, 1), (64, 64, 0)], "ternary", -1, 1, "i8", "f32"),
    (2048, [(768, 768, 0)] * 3 + [(768, 768, 1), (768, 2048, 2), (768, 2048, 2), (2048, 768, 3)],
     "ternary", -1, 1, "i8", "bf16"),
    # two dW tiles over a long batch: dW split over the batch (partials and
    # their reduction) inside the launch it shares with dX
    (4096, [(256, 256, 0), (256, 128, 0)], "ternary", -1, 1, "i8", "bf16"),
    # 4-bit codes: forward, dX, dW and the SR update
    (600, [(256, 128, 0), (128, 256, 1), (256, 256, 0)], "i4", -8, 7, "i8", "bf16"),
    (300, [(64, 80, 0), (80, 64, 1)], "i4", -4, 3, "i8", "f32"),
    # 3-bit codes (8 weights in 3 bytes)
    (600, [(256, 128, 0), (128, 256, 1), (256, 256, 0)], "i3", -4, 3, "i8", "bf16"),
    (300, [(64, 80, 0), (80, 64, 1)], "i3", -2, 1, "e4m3", "f32"),
]


@pytest.mark.parametrize("bi", range(len(BATCHES)))
def test_batch_matches_oracle_and_singles(lib, bi):
    M, lins, wfmt, qmin, qmax, act, env = BATCHES[bi]
    log(f"batch {bi}: M={M} {lins} {wfmt} {act} {env}")
    n_in = max(l[2] for l in lins) + 1
    widths = {}
    for (d_in, _, ii) in lins:
        widths[ii] = d_in
    Xs, Xseen, Xq, xdq = {}, {}, {}, {}
    for ii in range(n_in):
        Xs[ii], Xseen[ii] = to_dev(W.draw_normal((M, widths[ii]), 1.0, SEED, bi, 1, ii), env)
        Xq[ii] = torch.empty((M, widths[ii]), dtype=torch.int8 if act == "i8" else torch.uint8, device=DEV)
        xdq[ii] = torch.empty((M,), dtype=torch.float32, device=DEV)
        dqt.dqt_act_quant(Xs[ii], dqt.DQT_I8 if act == "i8" else dqt.DQT_FP8E4M3, Xq[ii], xdq[ii])
    ents, qs, alphas, dys = [], [], [], []
    tdt = torch.bfloat16 if env == "bf16" else torch.float32
    for li, (d_in, d_out, ii) in enumerate(lins):
        if wfmt == "ternary":
            q = W.draw_ternary((d_out, d_in), SEED, bi, 2, li)
        else:
            q = W.draw_int((d_out, d_in), qmin, qmax, SEED, bi, 2, li)
        alpha = np.float32(0.01 + 0.003 * li)
        w = make_weight(d_out, d_in, wfmt, qmin, qmax, alpha, tensor_id=li)
        dY, dYs = to_dev(W.draw_normal((M, d_out), 1e-2, SEED, bi, 3, li), env)
        ents.append(dict(w=w, Wq=weight_codes_dev(q, wfmt), Xq=Xq[ii], xdq=xdq[ii],
                         Y=torch.empty((M, d_out), dtype=tdt, device=DEV), dY=dY,
                         dX=torch.empty((M, d_in), dtype=tdt, device=DEV),
                         dW=torch.empty((d_out, d_in), dtype=torch.float32, device=DEV)))
        qs.append(q)
        alphas.append(alpha)
        dys.append(dYs)
    io = dqt.linear_io(ents)
    a_code = dqt.DQT_I8 if act == "i8" else dqt.DQT_FP8E4M3
    f_code = dqt.DQT_BF16 if env == "bf16" else dqt.DQT_F32
    fws = dqt.workspace(dqt.dqt_linear_fwd_batch_workspace(io))
    bws = dqt.workspace(dqt.dqt_linear_bwd_batch_workspace(io, M))
    dqt.dqt_linear_fwd_batch(io, M, a_code, f_code, fws)
    dqt.dqt_linear_bwd_batch(io, M, a_code, f_code, f_code, f_code, bws)
    torch.cuda.synchronize()
    for li, (d_in, d_out, ii) in enumerate(lins):
        e = ents[li]
        wq_, d_ = O.act_quant(Xseen[ii], act)
        # forward: bit-exact (int8) / tolerance (e4m3) against the oracle
        Y_ref, acc = O.linear_fwd(wq_, d_, act, qs[li], alphas[li], env)
        gotY = e["Y"].float().cpu().numpy()
        if act == "i8":
            assert np.array_equal(gotY, Y_ref), li
        else:
            a = np.abs(O.act_values(wq_, act)) @ np.abs(qs[li].astype(np.float64)).T
            f = (d_ * alphas[li]).astype(np.float64)[:, None]
            ok, nb, em = gemm_close(gotY, acc * f, a * f, bf16_out=(env == "bf16"))
            assert ok, (li, nb, em)
        _, _, dX64, dW64 = O.linear_bwd(dys[li], qs[li], alphas[li], wq_, d_, act, env, env)
        bx = float(alphas[li]) * O.gemm_abs_bound(dys[li], qs[li].astype(np.float64))
        ok, nb, em = gemm_close(e["dX"].float().cpu().numpy(), dX64, bx, bf16_out=(env == "bf16"))
        assert ok, ("dX", li, nb, em)
        bw = O.gemm_abs_bound(dys[li].T, O.act_dequant(wq_, d_, act, env))
        ok, nb, em = gemm_close(e["dW"].cpu().numpy(), dW64, bw)
        assert ok, ("dW", li, nb, em)
        # single-linear calls give the same forward and dX bits
        w = e["w"]
        Y1 = torch.empty_like(e["Y"])
        ws1 = dqt.workspace(dqt.dqt_linear_fwd_workspace(w))
        dqt.dqt_linear_fwd(w, e["Wq"], None, M, a_code, e["Xq"], e["xdq"], Y1, ws1)
        dX1 = torch.empty_like(e["dX"])
        wsb1 = dqt.workspace(dqt.dqt_linear_bwd_workspace(w, M))
        dqt.dqt_linear_bwd(w, e["Wq"], e["Xq"], a_code, e["xdq"], e["dY"], M, f_code, dX1, None,
                           wsb1)
        torch.cuda.synchronize()
        assert torch.equal(Y1, e["Y"]), li
        assert torch.equal(dX1, e["dX"]), li
    # SR batch == per-tensor SR on the same gradients
    before = [weight_codes_host(e["Wq"], wfmt, lin[0]) for e, lin in zip(ents, lins)]
    cnt = torch.zeros((2,), dtype=torch.int64, device=DEV)
    dqt.dqt_sr_update_batch(io, 5e-3, 9, 2, cnt)
    total = 0
    for li, (d_in, d_out, ii) in enumerate(lins):
        got = weight_codes_host(ents[li]["Wq"], wfmt, d_in)
        g = ents[li]["dW"].cpu().numpy()
        want, nch, _ = O.sr_update(before[li].ravel(), g.ravel(), 5e-3, alphas[li], qmin, qmax, 9, 2, li)
        assert np.array_equal(got.ravel(), want), li
        total += nch
    assert int(cnt[0].item()) == total


def test_batch_rejects_mixed_formats_and_sizes(lib):
    w1 = make_weight(64, 64, "ternary", -1, 1, 0.01)
    w2 = make_weight(64, 64, "i8", -127, 127, 0.01)
    t = torch.empty((64 * 64,), dtype=torch.int8, device=DEV)
    io = dqt.linear_io([dict(w=w1, Wq=t), dict(w=w2, Wq=t)])
    with pytest.raises(dqt.DqtError) as e:
        dqt.dqt_linear_fwd_batch(io, 16, dqt.DQT_I8, dqt.DQT_F32)
    assert e.value.status == dqt.DQT_ERR_UNSUPPORTED
    io9 = dqt.linear_io([dict(w=w1, Wq=t)] * 9)
    with pytest.raises(dqt.DqtError) as e:
        dqt.dqt_sr_update_batch(io9, 1e-3, 0, 1)
    assert e.value.status == dqt.DQT_ERR_SHAPE


def test_workspace_contents_do_not_matter(lib):
    """The persistent GEMM's tile counters live in the workspace and are
    cleared by every call before its kernels run, so a workspace left with
    any contents (another call's counters, or garbage) gives the same bits
    call after call."""
    M = 1000
    ents = []
    for li, (d_in, d_out) in enumerate([(256, 512), (512, 256), (256, 256)]):
        q = W.draw_ternary((d_out, d_in), 5, 97, li)
        w = make_weight(d_out, d_in, "ternary", -1, 1, 0.02, li)
        X_dev, _ = to_dev(W.draw_normal((M, d_in), 1.0, 5, 97, 10 + li), "bf16")
        dY_dev, _ = to_dev(W.draw_normal((M, d_out), 1e-2, 5, 97, 20 + li), "bf16")
        Xq, xdq, _ = run_fwd(w, weight_codes_dev(q, "ternary"), X_dev, "i8", "bf16")
        ents.append(dict(w=w, Wq=weight_codes_dev(q, "ternary"), Xq=Xq, xdq=xdq,
                         Y=torch.empty((M, d_out), dtype=torch.bfloat16, device=DEV), dY=dY_dev,
                         dX=torch.empty((M, d_in), dtype=torch.bfloat16, device=DEV),
                         dW=torch.empty((d_out, d_in), dtype=torch.float32, device=DEV)))
    io = dqt.linear_io(ents)
    ws = dqt.workspace(max(dqt.dqt_linear_fwd_batch_workspace(io),
                           dqt.dqt_linear_bwd_batch_workspace(io, M)))
    first = None
    for rep, fill in enumerate([0x00, 0xFF, 0x7F, None]):
        if fill is not None:
            ws.view(torch.uint8).fill_(fill)
        dqt.dqt_linear_fwd_batch(io, M, dqt.DQT_I8, dqt.DQT_BF16, ws)
        dqt.dqt_linear_bwd_batch(io, M, dqt.DQT_I8, dqt.DQT_BF16, dqt.DQT_BF16, dqt.DQT_BF16, ws)
        torch.cuda.synchronize()
        got = [(e["Y"].clone(), e["dX"].clone(), e["dW"].clone()) for e in ents]
        if first is None:
            first = got
            continue
        for li, (a, b) in enumerate(zip(first, got)):
            for k in range(3):
                assert torch.equal(a[k], b[k]), (rep, li, k)
