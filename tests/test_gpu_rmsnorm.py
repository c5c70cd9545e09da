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
