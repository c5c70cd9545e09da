"""The LLaMA-shaped model with DQT linears (model_step.py) on the GPU: the
autograd glue of a group of DQT linears (fused RMSNorm + quantisation in
front, the norm's backward after) against a float reference, and a few
train steps of a small model (loss near ln(vocab) at the start, finite, codes
moving by Eq. 5)."""
import math

import numpy as np
import pytest
import torch

from oracle import dqt_oracle as O
from paper_2412_04787_amd import model_step as MS

from gpu_util import DEV, log

pytestmark = pytest.mark.gpu


def _codes_host(grp, li):
    d_out, d_in = grp.d_outs[li], grp.d_in
    return O.unpack_ternary(grp.codes[li].cpu().numpy(), d_in).astype(np.float64)


def test_group_forward_backward_matches_reference(lib):
    """One norm-fed group (q, k, v of the small model): Y against the
    dequantised linear of the library's own quantised input, dx and dgamma
    against float autograd of RMSNorm with the straight-through quantiser."""
    cfg = MS.MODELS["tiny"]
    log(f"model group glue {cfg}")
    model = MS.DQTModel(cfg)
    grp = model.groups[0]["attn_in"]
    T, H = cfg.tokens, cfg.hidden
    rng = np.random.default_rng(11)
    x = torch.from_numpy(rng.standard_normal((T, H), dtype=np.float32)).to(torch.bfloat16).to(DEV)
    x.requires_grad_(True)
    gamma = torch.from_numpy((1 + 0.1 * rng.standard_normal(H)).astype(np.float32)).to(DEV)
    gamma.requires_grad_(True)
    q_before = [_codes_host(grp, li) for li in range(3)]
    alphas = [w.alpha for w in grp.weights]
    fn = MS._DQTGroupFn.get()
    Ys = fn.apply(x, gamma, grp)
    dYs = [torch.from_numpy(rng.standard_normal((T, H), dtype=np.float32) * 0.01)
           .to(torch.bfloat16).to(DEV) for _ in range(3)]
    # forward: the library's own quantised input, dequantised, times alpha q
    n_ref = torch.nn.functional.rms_norm(x.detach().float(), (H,), weight=gamma.detach(),
                                         eps=cfg.eps).cpu().numpy().astype(np.float64)
    Xq, xdq = O.act_quant(n_ref.astype(np.float32), "i8")
    for li in range(3):
        Yref = (Xq.astype(np.float64) * xdq[:, None].astype(np.float64)) @ (alphas[li] * q_before[li]).T
        got = Ys[li].detach().float().cpu().numpy()
        err = np.linalg.norm(got - Yref) / np.linalg.norm(Yref)
        assert err < 2e-2, (li, err)
    torch.autograd.backward(Ys, dYs)
    torch.cuda.synchronize()
    # reference backward: dn = sum_l dY_l (alpha_l q_l) (straight through the
    # quantiser), then float autograd through RMSNorm
    dn = sum(dYs[li].float().cpu().numpy().astype(np.float64) @ (alphas[li] * q_before[li])
             for li in range(3))
    xr = x.detach().float().cpu().requires_grad_(True)
    gr = gamma.detach().cpu().requires_grad_(True)
    y = torch.nn.functional.rms_norm(xr, (H,), weight=gr, eps=cfg.eps)
    dx_ref, dg_ref = torch.autograd.grad(y, (xr, gr), torch.from_numpy(dn.astype(np.float32)))
    dx = x.grad.float().cpu().numpy()
    dg = gamma.grad.cpu().numpy()
    ex = np.linalg.norm(dx - dx_ref.numpy()) / np.linalg.norm(dx_ref.numpy())
    eg = np.linalg.norm(dg - dg_ref.numpy()) / np.linalg.norm(dg_ref.numpy())
    log(f"dx rel err {ex:.2e}, dgamma rel err {eg:.2e}")
    assert ex < 2e-2 and eg < 2e-2, (ex, eg)
    # the backward applied Eq. 5 to the codes: they moved, and stayed on the grid
    moved = sum(int(np.count_nonzero(_codes_host(grp, li) != q_before[li])) for li in range(3))
    assert moved == int(model.counters[0].item()) and moved > 0
    for li in range(3):
        assert set(np.unique(_codes_host(grp, li)).tolist()) <= {-1.0, 0.0, 1.0}


def test_tiny_model_trains(lib):
    cfg = MS.MODELS["tiny"]
    log(f"tiny model steps {cfg}")
    model = MS.DQTModel(cfg)
    losses = []
    for s in range(4):
        tok, tgt = MS.synthetic_batch(cfg, s)
        losses.append(float(model.train_step(tok, tgt).item()))
    log(f"losses {losses}")
    assert all(math.isfinite(v) for v in losses)
    assert abs(losses[0] - math.log(cfg.vocab)) < 0.5
    changed, nonfinite = model.counters.tolist()
    assert changed > 0 and nonfinite == 0
    # each step moves a small fraction of the weights (Sec. 5.2 reports
    # fractions below a few percent for the 8-bit grid and far less for ternary)
    assert changed / 4 < 0.05 * cfg.dqt_weights
