"""RMSNorm + activation quantisation on the GPU against the oracle (reading
R13), bit for bit: codes, scales and 1 / rms per row, for bf16 and fp32
inputs, int8 and e4m3 codes, ragged token counts, the LLaMA widths, a zero
row and rows of very different magnitudes."""
import numpy as np
import pytest
import torch

from oracle import dqt_oracle as O
from paper_2412_04787_amd import dqt, workloads as W

from gpu_util import DEV, log

pytestmark = pytest.mark.gpu

CASES = [
    # (M, K, x dtype, act, eps)
    (37, 48, "bf16", "i8", 1e-6),
    (257, 768, "bf16", "i8", 1e-5),
    (130, 2048, "f32", "e4m3", 1e-6),
    (64, 4096, "bf16", "e4m3", 1e-5),
    (33, 11008, "bf16", "i8", 1e-6),
    (5, 5632, "f32", "i8", 1e-5),
]


@pytest.mark.parametrize("ci", range(len(CASES)))
def test_rmsnorm_act_quant_matches_oracle(lib, ci):
    M, K, xdt, act, eps = CASES[ci]
    log(f"rmsnorm+quant case {ci}: M={M} K={K} {xdt} {act} eps={eps}")
    X = W.draw_normal((M, K), 1.0, 17, 71, ci)
    X *= np.exp(np.linspace(-4, 4, M, dtype=np.float32))[:, None]   # magnitudes across rows
    X[M // 2] = 0.0                                                  # a zero row
    g = (1.0 + 0.3 * W.draw_normal((K,), 1.0, 17, 72, ci)).astype(np.float32)
    Xt = torch.from_numpy(X)
    if xdt == "bf16":
        Xt = Xt.to(torch.bfloat16)
    Xd = Xt.to(DEV)
    xv = Xt.float().numpy()                # the values the device sees
    code = dqt.DQT_I8 if act == "i8" else dqt.DQT_FP8E4M3
    Xq = torch.empty((M, K), dtype=torch.int8 if act == "i8" else torch.uint8, device=DEV)
    xdq = torch.empty((M,), dtype=torch.float32, device=DEV)
    rinv = torch.empty((M,), dtype=torch.float32, device=DEV)
    dqt.dqt_rmsnorm_act_quant(Xd, torch.from_numpy(g).to(DEV), eps, code, Xq, xdq, rinv)
    torch.cuda.synchronize()
    wq, wd, wr, _ = O.rmsnorm_act_quant(xv, g, eps, act)
    assert np.array_equal(rinv.cpu().numpy(), wr), "1 / rms"
    assert np.array_equal(xdq.cpu().numpy(), wd), "scales"
    got = Xq.cpu().numpy()
    assert np.array_equal(got, wq), ("codes", int((got != wq).sum()))


def test_rmsnorm_act_quant_argument_checks(lib):
    X = torch.zeros((4, 64), dtype=torch.bfloat16, device=DEV)
    g = torch.ones((64,), dtype=torch.float32, device=DEV)
    q = torch.empty((4, 64), dtype=torch.int8, device=DEV)
    d = torch.empty((4,), dtype=torch.float32, device=DEV)
    for eps, st in ((0.0, dqt.DQT_ERR_RANGE), (float("nan"), dqt.DQT_ERR_RANGE)):
        with pytest.raises(dqt.DqtError) as e:
            dqt.dqt_rmsnorm_act_quant(X, g, eps, dqt.DQT_I8, q, d)
        assert e.value.status == st
    with pytest.raises(dqt.DqtError) as e:
        dqt.dqt_rmsnorm_act_quant(X[:, :40], g, 1e-5, dqt.DQT_I8, q, d)
    assert e.value.status == dqt.DQT_ERR_SHAPE
    with pytest.raises(dqt.DqtError) as e:
        dqt.dqt_rmsnorm_act_quant(X, None, 1e-5, dqt.DQT_I8, q, d)
    assert e.value.status == dqt.DQT_ERR_NULL


BWD_CASES = [
    # (M, K, n_dy, blocks)
    (37, 48, 1, 3),
    (257, 768, 2, 16),
    (130, 2048, 3, 1024),
    (5, 4096, 4, 2),
]


@pytest.mark.parametrize("ci", range(len(BWD_CASES)))
def test_rmsnorm_backward_matches_float_reference(lib, ci):
    """dqt_rmsnorm_backward (the norm's backward on the sum of a group's dX,
    for the model step) against float64 autograd of y = x r gamma, with r
    the forward's 1 / rms: dX within bf16 rounding, dgamma (the sum of the
    per-block partials) to fp32 accuracy."""
    M, K, n_dy, blocks = BWD_CASES[ci]
    log(f"rmsnorm backward case {ci}: M={M} K={K} n_dy={n_dy} blocks={blocks}")
    X = W.draw_normal((M, K), 1.0, 17, 73, ci)
    X *= np.exp(np.linspace(-2, 2, M, dtype=np.float32))[:, None]
    g = (1.0 + 0.3 * W.draw_normal((K,), 1.0, 17, 74, ci)).astype(np.float32)
    dys = [torch.from_numpy(W.draw_normal((M, K), 1e-2, 17, 75, ci, i)).to(torch.bfloat16).to(DEV)
           for i in range(n_dy)]
    Xd = torch.from_numpy(X).to(torch.bfloat16).to(DEV)
    gd = torch.from_numpy(g).to(DEV)
    Xq = torch.empty((M, K), dtype=torch.int8, device=DEV)
    xdq = torch.empty((M,), dtype=torch.float32, device=DEV)
    rinv = torch.empty((M,), dtype=torch.float32, device=DEV)
    dqt.dqt_rmsnorm_act_quant(Xd, gd, 1e-6, dqt.DQT_I8, Xq, xdq, rinv)
    dX = torch.empty_like(Xd)
    gpart = torch.empty((blocks, K), dtype=torch.float32, device=DEV)
    dqt.dqt_rmsnorm_backward(dys, Xd, gd, rinv, dX, gpart)
    torch.cuda.synchronize()
    x64 = torch.from_numpy(Xd.float().cpu().numpy().astype(np.float64)).requires_grad_(True)
    g64 = torch.from_numpy(g.astype(np.float64)).requires_grad_(True)
    r = torch.from_numpy(rinv.cpu().numpy().astype(np.float64))
    # y = x r(x) gamma, r(x) = (mean(x^2) + eps)^(-1/2), whose value is the forward's
    y = x64 * torch.rsqrt((x64 * x64).mean(-1, keepdim=True) + 1e-6) * g64
    dn = sum(d.float().cpu().double() for d in dys)
    dx_ref, dg_ref = torch.autograd.grad(y, (x64, g64), dn)
    got = dX.float().cpu().numpy().astype(np.float64)
    ref = dx_ref.numpy()
    # bf16 output (half an ulp of the value), plus the fp32 rounding of the
    # row's dot product (up to ~K 2^-24 relative, times |x| r^3 c)
    tol = np.abs(ref) * 2.0 ** -8 + 2e-4 * np.abs(ref).max()
    assert np.all(np.abs(got - ref) <= tol), np.max(np.abs(got - ref) / (np.abs(ref) + 1e-30))
    assert np.allclose(gpart.sum(0).cpu().numpy(), dg_ref.numpy(), rtol=1e-4, atol=1e-6 * np.abs(dg_ref.numpy()).max())
    assert np.allclose(r.numpy(), 1.0 / np.sqrt((X.astype(np.float64) ** 2).mean(-1) + 1e-6), rtol=2e-2)
