"""Backward with the SR update fused into the backward call (dW never
reaches the caller's memory: updated in the dW product's epilogue, or staged
in the workspace for a streaming pass):
the codes, the counters and dX equal those of the backward call that writes
dW followed by the SR update call on that dW, bit for bit, and the codes
equal the oracle's SR update (Sec. 3.2 Eq. 5) of that dW."""
import numpy as np
import pytest
import torch

from oracle import dqt_oracle as O
from paper_2412_04787_amd import dqt, workloads as W

from gpu_util import DEV, log, make_weight, to_dev, weight_codes_dev, weight_codes_host

pytestmark = pytest.mark.gpu
SEED = 2024

CASES = [
    # (M, [(d_in, d_out, input_index, wants_dX)], wfmt, qmin, qmax, act, lr, inf_at)
    # ragged batch and tiles (384 = 1.5 tiles, 1000 tokens), one shared input
    (1000, [(256, 256, 0, True), (256, 384, 0, True), (256, 128, 0, True), (384, 256, 1, True)],
     "ternary", -1, 1, "i8", 5e-3, None),
    # int8 codes, small shapes
    (777, [(96, 208, 0, True), (96, 48, 0, True), (208, 96, 1, True)], "i8", -127, 127, "i8", 2e-2,
     None),
    # e4m3 activations
    (640, [(128, 256, 0, True), (256, 128, 1, True)], "ternary", -1, 1, "e4m3", 5e-3, None),
    # two dW tiles over a long batch: dW split over the batch, the update in
    # the kernel that sums the partials
    (4096, [(256, 256, 0, True), (256, 128, 0, True)], "ternary", -1, 1, "i8", 5e-3, None),
    # dX for some linears only (dX first, then dW and the update of all)
    (512, [(256, 256, 0, True), (256, 128, 0, False), (128, 256, 1, True)], "i8", -8, 7, "i8", 5e-2,
     None),
    # no dX at all (dW-only launch); a large step that saturates
    (512, [(256, 256, 0, False), (256, 512, 0, False)], "ternary", -1, 1, "i8", 1.0, None),
    # a non-finite upstream gradient entry: a row of dW is inf/NaN, its
    # weights stay and are counted
    (320, [(256, 256, 0, True), (256, 256, 1, True)], "ternary", -1, 1, "i8", 5e-3, (1, 7, 33)),
    (320, [(128, 256, 0, True)], "i8", -127, 127, "i8", 5e-3, (0, 5, 100)),
    # the largest batch (8 linears, three inputs)
    (640, [(128, 128, 0, True), (128, 256, 0, True), (128, 64, 0, True), (256, 128, 1, True),
           (64, 128, 2, True), (128, 192, 0, True), (256, 64, 1, False), (64, 64, 2, True)],
     "ternary", -1, 1, "i8", 1e-2, None),
    # widths that are not multiples of 32 (partial 32-wide blocks of dW in
    # both directions), a token count that is not a multiple of 64
    (300, [(80, 48, 0, True), (48, 272, 1, True), (208, 80, 2, False)], "ternary", -1, 1, "i8",
     5e-3, None),
    (200, [(16, 96, 0, True), (272, 16, 1, True)], "i8", -127, 127, "e4m3", 5e-3, None),
    # 4-bit codes (ragged batch, dX for all; and a batch-split dW)
    (1000, [(256, 384, 0, True), (384, 128, 1, True)], "i4", -8, 7, "i8", 2e-2, None),
    (4096, [(256, 256, 0, True)], "i4", -4, 3, "i8", 2e-2, (0, 9, 3)),
    # 4-bit codes with e4m3 activations
    (640, [(128, 256, 0, True), (256, 128, 1, True)], "i4", -8, 7, "e4m3", 2e-2, None),
    # 3-bit codes: ragged batch; a batch-split dW with a non-finite gradient;
    # e4m3 activations
    (1000, [(256, 384, 0, True), (384, 128, 1, True)], "i3", -4, 3, "i8", 2e-2, None),
    (4096, [(256, 256, 0, True)], "i3", -4, 3, "i8", 2e-2, (0, 9, 3)),
    (640, [(128, 256, 0, True), (256, 128, 1, True)], "i3", -4, 3, "e4m3", 2e-2, None),
]


@pytest.mark.parametrize("mode", ["fused", "staged"])
@pytest.mark.parametrize("ci", range(len(CASES)))
def test_fused_sr_matches_two_calls_and_oracle(lib, ci, mode, monkeypatch):
    """mode: the update in the dW epilogue, or on dW staged in the workspace
    (DQT_SR_EPILOGUE); a batch-split dW always updates in the reduction."""
    monkeypatch.setenv("DQT_SR_EPILOGUE", mode)
    M, lins, wfmt, qmin, qmax, act, lr, inf_at = CASES[ci]
    log(f"fused SR case {ci} ({mode}): M={M} {lins} {wfmt} {act} lr={lr} inf_at={inf_at}")
    a_code = dqt.DQT_I8 if act == "i8" else dqt.DQT_FP8E4M3
    bf = dqt.DQT_BF16
    n_in = max(l[2] for l in lins) + 1
    widths = {ii: d_in for (d_in, _, ii, _) in lins}
    Xq, xdq = {}, {}
    for ii in range(n_in):
        X, _ = to_dev(W.draw_normal((M, widths[ii]), 1.0, SEED, ci, 1, ii), "bf16")
        Xq[ii] = torch.empty((M, widths[ii]), dtype=torch.int8 if act == "i8" else torch.uint8,
                             device=DEV)
        xdq[ii] = torch.empty((M,), dtype=torch.float32, device=DEV)
        dqt.dqt_act_quant(X, a_code, Xq[ii], xdq[ii])
    two, fused, qs = [], [], []
    for li, (d_in, d_out, ii, wants_dx) in enumerate(lins):
        if wfmt == "ternary":
            q = W.draw_ternary((d_out, d_in), SEED, ci, 2, li)
        else:
            q = W.draw_int((d_out, d_in), qmin, qmax, SEED, ci, 2, li)
        alpha = np.float32(0.01 + 0.002 * li)
        w = make_weight(d_out, d_in, wfmt, qmin, qmax, alpha, tensor_id=3 + li)
        dY, _ = to_dev(W.draw_normal((M, d_out), 1e-2, SEED, ci, 3, li), "bf16")
        if inf_at is not None and inf_at[0] == li:
            dY[inf_at[1], inf_at[2]] = float("inf")
        common = dict(w=w, Xq=Xq[ii], xdq=xdq[ii], dY=dY)
        dx = lambda: (torch.empty((M, d_in), dtype=torch.bfloat16, device=DEV) if wants_dx else None)
        two.append(dict(common, Wq=weight_codes_dev(q, wfmt), dX=dx(),
                        dW=torch.empty((d_out, d_in), dtype=torch.float32, device=DEV)))
        fused.append(dict(common, Wq=weight_codes_dev(q, wfmt), dX=dx(), dW=None))
        qs.append((q, alpha, w))
    io2, iof = dqt.linear_io(two), dqt.linear_io(fused)
    ws2 = dqt.workspace(dqt.dqt_linear_bwd_batch_workspace(io2, M))
    wsf = dqt.workspace(dqt.dqt_linear_bwd_batch_workspace(iof, M))
    cnt2 = torch.zeros((2,), dtype=torch.int64, device=DEV)
    cntf = torch.zeros((2,), dtype=torch.int64, device=DEV)
    seed, step = 77, 5
    wsf.view(torch.uint8).fill_(0xFF)     # a workspace's contents on entry do not matter
    dqt.dqt_linear_bwd_batch(io2, M, a_code, bf, bf, bf, ws2)
    dqt.dqt_sr_update_batch(io2, lr, seed, step, cnt2)
    dqt.dqt_linear_bwd_sr_batch(iof, M, a_code, bf, bf, bf, lr, seed, step, cntf, wsf)
    torch.cuda.synchronize()
    assert torch.equal(cnt2, cntf), (cnt2.tolist(), cntf.tolist())
    total_changed = total_nf = 0
    for li, (d_in, d_out, ii, wants_dx) in enumerate(lins):
        q, alpha, w = qs[li]
        got = weight_codes_host(fused[li]["Wq"], wfmt, d_in)
        ref2 = weight_codes_host(two[li]["Wq"], wfmt, d_in)
        assert np.array_equal(got, ref2), ("codes vs two calls", li, int((got != ref2).sum()))
        if wants_dx:
            a, b = two[li]["dX"], fused[li]["dX"]
            assert torch.equal(a.isnan(), b.isnan()), li
            assert torch.equal(torch.nan_to_num(a.float()), torch.nan_to_num(b.float())), ("dX", li)
        g = two[li]["dW"].cpu().numpy()
        want, nch, nnf = O.sr_update(q.ravel(), g.ravel(), lr, alpha, qmin, qmax, seed, step,
                                     3 + li)
        assert np.array_equal(got.ravel(), want), ("codes vs oracle", li)
        total_changed += nch
        total_nf += nnf
    assert int(cntf[0].item()) == total_changed
    assert int(cntf[1].item()) == total_nf
    if inf_at is not None:
        assert total_nf > 0


def test_fused_sr_argument_checks(lib):
    w = make_weight(64, 64, "ternary", -1, 1, 0.01)
    t = torch.empty((64 * 64,), dtype=torch.int8, device=DEV)
    f = torch.empty((64, 64), dtype=torch.float32, device=DEV)
    bf, f32 = dqt.DQT_BF16, dqt.DQT_F32
    io_dw = dqt.linear_io([dict(w=w, Wq=t, Xq=t, xdq=f, dY=f, dW=f)])
    ws = dqt.workspace(dqt.dqt_linear_bwd_batch_workspace(io_dw, 64))
    with pytest.raises(dqt.DqtError) as e:    # dW would not be written
        dqt.dqt_linear_bwd_sr_batch(io_dw, 64, dqt.DQT_I8, bf, bf, bf, 1e-3, 0, 1, None, ws)
    assert e.value.status == dqt.DQT_ERR_UNSUPPORTED
    io = dqt.linear_io([dict(w=w, Wq=t, Xq=t, xdq=f, dY=f)])
    with pytest.raises(dqt.DqtError) as e:    # fp32 environment: use the two calls
        dqt.dqt_linear_bwd_sr_batch(io, 64, dqt.DQT_I8, f32, f32, bf, 1e-3, 0, 1, None, ws)
    assert e.value.status == dqt.DQT_ERR_UNSUPPORTED
    with pytest.raises(dqt.DqtError) as e:
        dqt.dqt_linear_bwd_sr_batch(io, 64, dqt.DQT_I8, bf, bf, bf, -1.0, 0, 1, None, ws)
    assert e.value.status == dqt.DQT_ERR_RANGE
    with pytest.raises(dqt.DqtError) as e:
        dqt.dqt_linear_bwd_sr_batch(io, 64, dqt.DQT_I8, bf, bf, bf, 1e-3, 0, 1, None, None)
    assert e.value.status == dqt.DQT_ERR_WORKSPACE
    # M = 0 moves nothing and launches nothing
    before = t.clone()
    dqt.dqt_linear_bwd_sr_batch(io, 0, dqt.DQT_I8, bf, bf, bf, 1e-3, 0, 1, None, ws)
    torch.cuda.synchronize()
    assert torch.equal(before, t)


def test_fused_sr_is_deterministic_at_block_size(lib):
    """The step's fused call on the hidden-768 block (M = 8192, seven
    linears, several dW tiles per compute unit) twice from the same codes:
    codes, dX and counts identical bit for bit (fixed reduction orders, no
    atomics in any value)."""
    import os
    import sys
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import bench
    log("fused backward + SR determinism: llama_h768")
    blk = bench.Block(W.WORKLOADS["llama_h768"], torch, dqt, W)

    def only(kind):
        def rec(k, fn):
            if k == kind:
                fn()
        return rec
    bench.run_step(blk, dqt, 1, None, only("act_quant"))
    bench.run_step(blk, dqt, 1, None, only("fwd"))
    torch.cuda.synchronize()
    codes0 = [c.clone() for c in blk.codes]
    outs = []
    for _ in range(2):
        for c, c0 in zip(blk.codes, codes0):
            c.copy_(c0)
        blk.counters.zero_()
        bench.run_step(blk, dqt, 5, None, only("bwd_sr"), sr="fused")
        torch.cuda.synchronize()
        outs.append(([c.clone() for c in blk.codes], [x.clone() for x in blk.dX], blk.counters.clone()))
    (ca, xa, na), (cb, xb, nb) = outs
    assert all(torch.equal(a, b) for a, b in zip(ca, cb))
    assert all(torch.equal(a, b) for a, b in zip(xa, xb))
    assert torch.equal(na, nb) and int(na[0].item()) > 0
    assert any(not torch.equal(a, b) for a, b in zip(ca, codes0))
