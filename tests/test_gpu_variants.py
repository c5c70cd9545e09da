"""The analysis variants of the update on the GPU against the oracle (Sec. 5;
reading R12 of the oracle): nearest rounding and the two interventions on
the smallest fraction of updates, whose threshold the GPU finds by an exact
radix select; codes and counts bit-exact."""
import numpy as np
import pytest
import torch

from oracle import dqt_oracle as O
from paper_2412_04787_amd import dqt, workloads as W

from gpu_util import DEV, log, make_weight, weight_codes_dev, weight_codes_host

pytestmark = pytest.mark.gpu
SEED = 808

SHAPES = [
    # (d_out, d_in, wfmt, qmin, qmax, alpha, lr, grad kind)
    (256, 384, "ternary", -1, 1, 0.02, 5e-3, "normal"),
    (208, 96, "i8", -127, 127, 0.004, 2e-2, "normal"),
    (64, 48, "i8", -8, 7, 0.05, 0.5, "ties"),          # few distinct |delta|: ties at tau
    (2048, 1024, "ternary", -1, 1, 0.01, 1e-2, "normal"),
    (96, 256, "i4", -8, 7, 0.02, 0.1, "normal"),
    (112, 208, "i3", -4, 3, 0.02, 0.1, "normal"),
]
MODES = [(dqt.DQT_UPD_SR, 0.2), (dqt.DQT_UPD_NEAREST, 0.2), (dqt.DQT_UPD_FORCE_REMAIN, 0.2),
         (dqt.DQT_UPD_FORCE_CHANGE, 0.2), (dqt.DQT_UPD_FORCE_CHANGE, 1.0),
         (dqt.DQT_UPD_FORCE_REMAIN, 0.0)]


def _grad(shape, kind, si):
    g = W.draw_normal(shape, 1e-2, SEED, si, 2).astype(np.float32)
    if kind == "ties":
        vals = np.array([-0.02, -0.005, 0.0, 0.005, 0.01, 0.04], np.float32)
        g = vals[np.abs((g * 1e4).astype(np.int64)) % vals.size].reshape(shape)
    flat = g.reshape(-1)
    flat[[3, 17]] = [np.inf, np.nan]
    return g


@pytest.mark.parametrize("mi", range(len(MODES)))
@pytest.mark.parametrize("si", range(len(SHAPES)))
def test_update_variant_matches_oracle(lib, si, mi):
    d_out, d_in, wfmt, qmin, qmax, alpha, lr, kind = SHAPES[si]
    mode, frac = MODES[mi]
    log(f"variant shape {si} {SHAPES[si]} mode {mode} frac {frac}")
    q = (W.draw_ternary((d_out, d_in), SEED, si, 1) if wfmt == "ternary"
         else W.draw_int((d_out, d_in), qmin, qmax, SEED, si, 1))
    g = _grad((d_out, d_in), kind, si)
    w = make_weight(d_out, d_in, wfmt, qmin, qmax, alpha, tensor_id=si)
    Wq = weight_codes_dev(q, wfmt)
    dW = torch.from_numpy(g).to(DEV)      # held: linear_io keeps only the pointer
    io = dqt.linear_io([dict(w=w, Wq=Wq, dW=dW)])
    ws = dqt.workspace(dqt.dqt_update_variant_workspace(1))
    cnt = torch.zeros((2,), dtype=torch.int64, device=DEV)
    dqt.dqt_update_variant_batch(io, lr, 31, 4, mode, frac, cnt, ws)
    torch.cuda.synchronize()
    want, nch, nnf = O.update_variant(q.ravel(), g.ravel(), lr, alpha, qmin, qmax, 31, 4, si, mode,
                                      frac)
    got = weight_codes_host(Wq, wfmt, d_in).ravel()
    assert np.array_equal(got, want), int((got != want).sum())
    assert cnt.tolist() == [nch, nnf]


def test_update_variant_batch_equals_singles(lib):
    shapes = [(256, 256), (128, 512), (384, 128)]
    ents, singles = [], []
    for li, (d_out, d_in) in enumerate(shapes):
        q = W.draw_ternary((d_out, d_in), SEED, 50, li)
        w = make_weight(d_out, d_in, "ternary", -1, 1, 0.01 + 0.002 * li, tensor_id=li)
        g = torch.from_numpy(W.draw_normal((d_out, d_in), 1e-2, SEED, 51, li)).to(DEV)
        ents.append(dict(w=w, Wq=weight_codes_dev(q, "ternary"), dW=g))
        singles.append(dict(w=w, Wq=weight_codes_dev(q, "ternary"), dW=g))
    ws = dqt.workspace(dqt.dqt_update_variant_workspace(len(shapes)))
    c1 = torch.zeros((2,), dtype=torch.int64, device=DEV)
    c2 = torch.zeros((2,), dtype=torch.int64, device=DEV)
    dqt.dqt_update_variant_batch(dqt.linear_io(ents), 1e-2, 2, 9, dqt.DQT_UPD_FORCE_CHANGE, 0.2, c1, ws)
    ws1 = dqt.workspace(dqt.dqt_update_variant_workspace(1))
    for s in singles:
        dqt.dqt_update_variant_batch(dqt.linear_io([s]), 1e-2, 2, 9, dqt.DQT_UPD_FORCE_CHANGE, 0.2, c2,
                                     ws1)
    torch.cuda.synchronize()
    assert torch.equal(c1, c2)
    for e, s in zip(ents, singles):
        assert torch.equal(e["Wq"], s["Wq"])


@pytest.mark.parametrize("mode", [dqt.DQT_UPD_FORCE_CHANGE, dqt.DQT_UPD_FORCE_REMAIN])
def test_update_variant_large_batch_equals_singles(lib, mode):
    """A batch of 17.8 M weights takes 8 chunks of 8 weights per thread in its
    selection passes (a single 8.4 M-weight tensor takes 4), the last block of
    a tensor partly empty: codes and counts equal those of the single calls,
    whose selection the small cases above pin to the oracle."""
    shapes = [(2048, 4096), (2048, 4096), (1040, 1024)]
    log(f"variant large batch mode {mode}: {shapes}")
    ents, singles = [], []
    for li, (d_out, d_in) in enumerate(shapes):
        q = torch.from_numpy(W.draw_ternary((d_out, d_in), SEED, 70, li))
        w = make_weight(d_out, d_in, "ternary", -1, 1, 0.01, tensor_id=li)
        g = torch.randn((d_out, d_in), generator=torch.Generator().manual_seed(li), dtype=torch.float32) * 1e-2
        g = g.to(DEV)
        ents.append(dict(w=w, Wq=weight_codes_dev(q.numpy(), "ternary"), dW=g))
        singles.append(dict(w=w, Wq=weight_codes_dev(q.numpy(), "ternary"), dW=g))
    c1 = torch.zeros((2,), dtype=torch.int64, device=DEV)
    c2 = torch.zeros((2,), dtype=torch.int64, device=DEV)
    ws = dqt.workspace(dqt.dqt_update_variant_workspace(len(shapes)))
    dqt.dqt_update_variant_batch(dqt.linear_io(ents), 1e-2, 5, 3, mode, 0.2, c1, ws)
    ws1 = dqt.workspace(dqt.dqt_update_variant_workspace(1))
    for s in singles:
        dqt.dqt_update_variant_batch(dqt.linear_io([s]), 1e-2, 5, 3, mode, 0.2, c2, ws1)
    torch.cuda.synchronize()
    for a, b in zip(ents, singles):
        assert torch.equal(a["Wq"], b["Wq"])
    assert torch.equal(c1, c2)
    assert int(c1[0].item()) > 0
