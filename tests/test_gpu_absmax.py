"""The literal absmax re-quantisation control of Sec. 5.1 on the GPU against
the oracle (reading R14): new codes, the new scale of every tensor and the
counts, bit for bit, for every code format in one batch each."""
import numpy as np
import pytest
import torch

from oracle import dqt_oracle as O
from paper_2412_04787_amd import dqt, workloads as W

from gpu_util import DEV, log, make_weight, weight_codes_dev, weight_codes_host

pytestmark = pytest.mark.gpu

CASES = [
    # (wfmt, qmin, qmax, shapes, lr, gscale)
    ("ternary", -1, 1, [(256, 384), (96, 64), (1024, 512)], 1e-2, 1.0),
    ("i8", -127, 127, [(208, 96), (64, 32)], 1e-3, 3.0),
    ("i4", -8, 7, [(192, 160), (16, 16)], 1e-2, 1.0),
    ("i3", -4, 3, [(160, 208), (48, 80)], 1e-2, 1.0),
]


@pytest.mark.parametrize("ci", range(len(CASES)))
def test_absmax_requant_matches_oracle(lib, ci):
    wfmt, qmin, qmax, shapes, lr, gscale = CASES[ci]
    log(f"absmax control case {ci}: {wfmt} {shapes}")
    ents, host = [], []
    for s, (d_out, d_in) in enumerate(shapes):
        q = (W.draw_ternary((d_out, d_in), 8, 81, s) if wfmt == "ternary"
             else W.draw_int((d_out, d_in), qmin, qmax, 8, 81, s))
        g = W.draw_normal((d_out, d_in), gscale, 8, 82, ci, s)
        if s == 0:
            g[3, 5] = np.nan
        alpha = np.float32(0.02 + 0.001 * s)
        w = make_weight(d_out, d_in, wfmt, qmin, qmax, alpha, s)
        ents.append(dict(w=w, Wq=weight_codes_dev(q, wfmt), dW=torch.from_numpy(g).to(DEV)))
        host.append((q, g, alpha, w))
    io = dqt.linear_io(ents)
    alpha_out = torch.zeros((len(shapes),), dtype=torch.float32, device=DEV)
    counters = torch.zeros((2,), dtype=torch.int64, device=DEV)
    dqt.dqt_absmax_requant_batch(io, lr, alpha_out, counters)
    torch.cuda.synchronize()
    tot_c = tot_f = 0
    for s, (q, g, alpha, w) in enumerate(host):
        want, a2, nch, nnf = O.absmax_requant(q, g, lr, alpha, qmin, qmax)
        got = weight_codes_host(ents[s]["Wq"], wfmt, w.d_in)
        assert np.array_equal(got.ravel(), want), (s, int((got.ravel() != want).sum()))
        assert alpha_out[s].item() == float(a2), (s, alpha_out[s].item(), float(a2))
        tot_c += nch
        tot_f += nnf
    assert counters.tolist() == [tot_c, tot_f]
    assert tot_f == 1


def test_absmax_requant_zero_matrix_keeps_scale(lib):
    w = make_weight(64, 64, "ternary", -1, 1, 0.125)
    q = np.zeros((64, 64), np.int8)
    ents = [dict(w=w, Wq=weight_codes_dev(q, "ternary"),
                 dW=torch.zeros((64, 64), dtype=torch.float32, device=DEV))]
    alpha_out = torch.zeros((1,), dtype=torch.float32, device=DEV)
    dqt.dqt_absmax_requant_batch(dqt.linear_io(ents), 1e-3, alpha_out)
    torch.cuda.synchronize()
    assert alpha_out.item() == 0.125
    assert not weight_codes_host(ents[0]["Wq"], "ternary", 64).any()
