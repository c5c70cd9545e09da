"""The fused backward + SR call (Sec. 3.2 Eq. 5 consuming the backward's dW)
at the sizes the train step runs it: every linear of a LLaMA block in one
call, at the block's full token count, so that every block of the persistent
grid runs several SR-epilogue tiles in a row (about 3 per compute unit at
hidden 2048, about 12 at hidden 4096).

Each case runs the same inputs through
  (1) dqt_linear_bwd_batch writing dW, then dqt_sr_update_batch on that dW;
  (2) dqt_linear_bwd_sr_batch (dW never stored),
on two copies of the codes, and checks
  * the fused codes equal the two-call codes on every weight, bit for bit;
  * the change / non-finite counters are equal;
  * the fused dX equals the two-call dX bit for bit;
  * the codes equal the oracle's SR update of the two-call dW (every weight
    at hidden 768; sampled rows spanning several tiles at 2048 / 4096);
  * dW and dX equal the oracle's fp64 products within the GEMM tolerance on
    sampled rows and columns.
"""
import numpy as np
import pytest
import torch

from oracle import dqt_oracle as O
from paper_2412_04787_amd import dqt, workloads as W

from gpu_util import DEV, gemm_close, log, weight_codes_host

pytestmark = pytest.mark.gpu

SEED, STEP = 11, 3


def _block(name, with_dx):
    """Device state of one workload's block: codes (two copies), quantised
    inputs, upstream gradients, outputs."""
    wl = W.WORKLOADS[name]
    M = wl.M
    act = dqt.DQT_I8 if wl.act == "i8" else dqt.DQT_FP8E4M3
    wfmt = {"ternary": dqt.DQT_TERNARY2, "i4": dqt.DQT_INT4, "i3": dqt.DQT_INT3}.get(wl.wfmt,
                                                                                   dqt.DQT_I8)
    Xq, xdq, Xd = {}, {}, {}
    for name_in in wl.inputs:
        X = torch.from_numpy(W.input_draw(wl, name_in)).to(torch.bfloat16).to(DEV)
        Xq[name_in] = torch.empty(X.shape, dtype=torch.int8 if wl.act == "i8" else torch.uint8,
                                  device=DEV)
        xdq[name_in] = torch.empty((M,), dtype=torch.float32, device=DEV)
        Xd[name_in] = X
    aio = dqt.act_io([(Xd[n], Xq[n], xdq[n]) for n in wl.inputs])
    dqt.dqt_act_quant_batch(aio, dqt.DQT_BF16, M, act)
    torch.cuda.synchronize()
    del Xd, aio
    lin_state = []
    for li, lin in enumerate(wl.linears):
        W0, _ = W.weight_draws(wl, li)
        q, alpha = O.absmean_init(W0, wl.qmin, wl.qmax)
        q = q.astype(np.int8)
        if wl.wfmt == "ternary":
            codes = O.pack_ternary(q)
        elif wl.wfmt == "i4":
            codes = O.pack_int4(q)
        elif wl.wfmt == "i3":
            codes = O.pack_int3(q)
        else:
            codes = q
        c1 = torch.from_numpy(np.ascontiguousarray(codes)).to(DEV)
        c2 = c1.clone()
        dY = torch.from_numpy(W.grad_draw(wl, li)).to(torch.bfloat16).to(DEV)
        w = dqt.weight(lin.d_out, lin.d_in, wfmt, wl.qmin, wl.qmax, float(alpha), 40 + li)
        lin_state.append(dict(lin=lin, q=q, alpha=np.float32(alpha), w=w, c_two=c1, c_fused=c2,
                              dY=dY))
    return wl, act, Xq, xdq, lin_state


def _sample_rows(d_out, rng, k=6):
    """Rows in the first, a middle and the last 256-row tile, plus random ones."""
    base = [0, 255 % d_out, min(256, d_out - 1), d_out // 2, d_out - 1]
    return np.unique(np.array(base + list(rng.integers(0, d_out, size=k)), dtype=np.int64))


def _run_case(name, with_dx, full_oracle):
    wl, act, Xq, xdq, st = _block(name, with_dx)
    M = wl.M
    log(f"full fused SR case {name}: M={M} with_dx={with_dx} weights={wl.n_weights}")
    bf = dqt.DQT_BF16
    two, fused = [], []
    for s in st:
        lin = s["lin"]
        dx2 = torch.empty((M, lin.d_in), dtype=torch.bfloat16, device=DEV) if with_dx else None
        dxf = torch.empty((M, lin.d_in), dtype=torch.bfloat16, device=DEV) if with_dx else None
        dW = torch.empty((lin.d_out, lin.d_in), dtype=torch.float32, device=DEV)
        common = dict(w=s["w"], Xq=Xq[lin.input], xdq=xdq[lin.input], dY=s["dY"])
        two.append(dict(common, Wq=s["c_two"], dX=dx2, dW=dW))
        fused.append(dict(common, Wq=s["c_fused"], dX=dxf, dW=None))
    io2, iof = dqt.linear_io(two), dqt.linear_io(fused)
    ws = dqt.workspace(max(dqt.dqt_linear_bwd_batch_workspace(io2, M),
                           dqt.dqt_linear_bwd_batch_workspace(iof, M)))
    # the workspace's contents on entry do not matter (tile counters included)
    ws.view(torch.uint8).fill_(0xA5)
    cnt2 = torch.zeros((2,), dtype=torch.int64, device=DEV)
    cntf = torch.zeros((2,), dtype=torch.int64, device=DEV)
    lr = wl.lr
    dqt.dqt_linear_bwd_batch(io2, M, act, bf, bf, bf, ws)
    dqt.dqt_sr_update_batch(io2, lr, SEED, STEP, cnt2)
    dqt.dqt_linear_bwd_sr_batch(iof, M, act, bf, bf, bf, lr, SEED, STEP, cntf, ws)
    torch.cuda.synchronize()
    assert torch.equal(cnt2, cntf), (cnt2.tolist(), cntf.tolist())
    log(f"  counters {cntf.tolist()}")
    rng = np.random.default_rng(5)
    total_changed = 0
    for li, s in enumerate(st):
        lin = s["lin"]
        # fused vs two calls: every weight
        if not torch.equal(s["c_two"], s["c_fused"]):
            a = weight_codes_host(s["c_two"], wl.wfmt, lin.d_in)
            b = weight_codes_host(s["c_fused"], wl.wfmt, lin.d_in)
            bad = np.argwhere(a != b)
            raise AssertionError(f"{lin.name}: {len(bad)} codes differ, first at {bad[:4].tolist()}")
        if with_dx:
            a, b = two[li]["dX"], fused[li]["dX"]
            assert torch.equal(a, b), f"{lin.name}: dX differs"
        got = weight_codes_host(s["c_fused"], wl.wfmt, lin.d_in)
        q = s["q"]
        if full_oracle:
            g = two[li]["dW"].cpu().numpy()
            want, nch, _ = O.sr_update(q.ravel(), g.ravel(), lr, s["alpha"], wl.qmin, wl.qmax,
                                       SEED, STEP, s["w"].tensor_id)
            assert np.array_equal(got.ravel(), want), f"{lin.name}: codes vs oracle"
            total_changed += nch
        rows = _sample_rows(lin.d_out, rng)
        g_rows = two[li]["dW"][torch.from_numpy(rows).to(DEV)].cpu().numpy()
        idx = (rows[:, None] * lin.d_in + np.arange(lin.d_in)[None, :]).astype(np.uint64)
        want_r, _, _ = O.sr_update(q[rows].ravel(), g_rows.ravel(), lr, s["alpha"], wl.qmin,
                                   wl.qmax, SEED, STEP, s["w"].tensor_id, idx=idx.ravel())
        assert np.array_equal(got[rows].ravel(), want_r), f"{lin.name}: sampled rows vs oracle"
        # dW against the oracle's fp64 product on sampled rows x columns
        cols = np.unique(np.concatenate([[0, lin.d_in - 1], rng.integers(0, lin.d_in, size=30)]))
        xq_c = Xq[lin.input][:, torch.from_numpy(cols).to(DEV)].cpu().numpy()
        d = xdq[lin.input].cpu().numpy()
        xt = O.act_dequant(xq_c, d, wl.act, "bf16")                    # [M, cols] float64
        dy_r = s["dY"][:, torch.from_numpy(rows).to(DEV)].float().cpu().numpy().astype(np.float64)
        ref = dy_r.T @ xt
        bound = np.abs(dy_r.T) @ np.abs(xt)
        ok, nbad, emax = gemm_close(g_rows[:, cols], ref, bound)
        assert ok, (lin.name, "dW", nbad, emax)
        if with_dx:
            mrows = _sample_rows(M, rng, k=4)
            dy_m = s["dY"][torch.from_numpy(mrows).to(DEV)].float().cpu().numpy().astype(np.float64)
            qf = q.astype(np.float64)
            ref = float(s["alpha"]) * (dy_m @ qf)
            bound = float(s["alpha"]) * (np.abs(dy_m) @ np.abs(qf))
            got_dx = fused[li]["dX"][torch.from_numpy(mrows).to(DEV)].float().cpu().numpy()
            ok, nbad, emax = gemm_close(got_dx, ref, bound, bf16_out=True)
            assert ok, (lin.name, "dX", nbad, emax)
    if full_oracle:
        assert int(cntf[0].item()) == total_changed
    assert int(cntf[1].item()) == 0


def test_fused_sr_full_llama_h768(lib):
    """Whole h768 block, M = 8192, dX for every linear: the bench's step call;
    every code checked against the oracle."""
    _run_case("llama_h768", True, True)


def test_fused_sr_full_llama_h768_split_dw(lib):
    """The same block without dX: the plan splits the dW reduction over the
    tokens, so the update runs in the kernel that sums the partials."""
    _run_case("llama_h768", False, True)


def test_fused_sr_full_llama_h2048(lib):
    """Hidden 2048 / FFN 5632, M = 16384, int8 codes -127..127: ~3 SR
    epilogue tiles per compute unit."""
    _run_case("llama_h2048", True, False)


def test_fused_sr_full_llama_h4096(lib):
    """Hidden 4096 / FFN 11008, M = 8192, ternary codes, e4m3 activations:
    ~12 SR epilogue tiles per compute unit."""
    _run_case("llama_h4096", True, False)


def test_fused_sr_full_llama_h2048_int4(lib):
    """Hidden 2048 block with 4-bit codes -8..7."""
    _run_case("llama_h2048_int4", True, False)


def test_fused_sr_full_llama_h2048_int3(lib):
    """Hidden 2048 block with 3-bit codes -4..3 (8 weights in 3 bytes)."""
    _run_case("llama_h2048_int3", True, False)


def test_fused_sr_full_llama_h768_staged(lib, monkeypatch):
    """The h768 block with dW staged in the workspace and the update run as
    a streaming pass (DQT_SR_EPILOGUE=staged) instead of in the epilogue."""
    monkeypatch.setenv("DQT_SR_EPILOGUE", "staged")
    _run_case("llama_h768", True, True)
