"""AdamW with SR on the GPU against the oracle (reading R11 of the oracle;
Sec. 4.1 trains DQT with AdamW modified to round stochastically): codes, m
and v bit-exact over several steps, counters exact, a batch equal to its
single-tensor calls, non-finite gradient entries kept."""
import numpy as np
import pytest
import torch

from oracle import dqt_oracle as O
from paper_2412_04787_amd import dqt, workloads as W

from gpu_util import DEV, log, make_weight, weight_codes_dev, weight_codes_host

pytestmark = pytest.mark.gpu
SEED = 606

CASES = [
    # (d_out, d_in, wfmt, qmin, qmax, alpha, hyper, n_bad)
    (256, 384, "ternary", -1, 1, 0.02, dict(lr=2e-3, beta1=0.9, beta2=0.95, eps=1e-8,
                                            weight_decay=0.1), 0),
    (208, 96, "i8", -127, 127, 0.004, dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8,
                                           weight_decay=0.0), 5),
    (64, 32, "i8", -8, 7, 0.05, dict(lr=0.5, beta1=0.5, beta2=0.6, eps=1e-3, weight_decay=0.3), 3),
    (2048, 2048, "ternary", -1, 1, 0.01, dict(lr=3e-4, beta1=0.9, beta2=0.95, eps=1e-8,
                                              weight_decay=0.01), 17),
    (192, 160, "i4", -8, 7, 0.01, dict(lr=1e-2, beta1=0.9, beta2=0.99, eps=1e-8,
                                        weight_decay=0.05), 4),
    (160, 208, "i3", -4, 3, 0.01, dict(lr=1e-2, beta1=0.9, beta2=0.99, eps=1e-8,
                                        weight_decay=0.05), 6),
]


def _bits(a):
    return np.asarray(a, dtype=np.float32).view(np.uint32)


@pytest.mark.parametrize("ci", range(len(CASES)))
def test_adamw_sr_matches_oracle_over_steps(lib, ci):
    d_out, d_in, wfmt, qmin, qmax, alpha, hp, n_bad = CASES[ci]
    log(f"adamw case {ci}: {d_out}x{d_in} {wfmt} {hp} bad={n_bad}")
    n = d_out * d_in
    if wfmt == "ternary":
        q = W.draw_ternary((d_out, d_in), SEED, ci, 1)
    else:
        q = W.draw_int((d_out, d_in), qmin, qmax, SEED, ci, 1)
    w = make_weight(d_out, d_in, wfmt, qmin, qmax, alpha, tensor_id=9 + ci)
    Wq = weight_codes_dev(q, wfmt)
    m_d = torch.zeros((d_out, d_in), dtype=torch.float32, device=DEV)
    v_d = torch.zeros((d_out, d_in), dtype=torch.float32, device=DEV)
    cnt = torch.zeros((2,), dtype=torch.int64, device=DEV)
    hpc = dqt.adamw(**hp)
    qh = q.ravel().astype(np.int64)
    mh = np.zeros(n, np.float32)
    vh = np.zeros(n, np.float32)
    tot_c = tot_f = 0
    for step in (1, 2, 3):
        g = W.draw_normal((d_out, d_in), 1e-2, SEED, ci, 2, step).astype(np.float32)
        if n_bad:
            pos = np.random.default_rng(ci * 10 + step).choice(n, n_bad, replace=False)
            g.ravel()[pos] = np.array([np.inf, -np.inf, np.nan] * n_bad, np.float32)[:n_bad]
        dW = torch.from_numpy(g).to(DEV)
        dqt.dqt_adamw_sr_update(w, Wq, dW, m_d, v_d, hpc, SEED, step, cnt)
        torch.cuda.synchronize()
        qh, mh, vh, nc, nf = O.adamw_sr_update(qh, g.ravel(), mh, vh, hp["lr"], alpha,
                                               hp["beta1"], hp["beta2"], hp["eps"],
                                               hp["weight_decay"], qmin, qmax, SEED, step, 9 + ci)
        tot_c += nc
        tot_f += nf
        got_q = weight_codes_host(Wq, wfmt, d_in).ravel()
        assert np.array_equal(got_q, qh), (step, int((got_q != qh).sum()))
        assert np.array_equal(_bits(m_d.cpu().numpy().ravel()), _bits(mh)), step
        assert np.array_equal(_bits(v_d.cpu().numpy().ravel()), _bits(vh)), step
        assert cnt.tolist() == [tot_c, tot_f], (step, cnt.tolist(), tot_c, tot_f)
    assert tot_c > 0


def test_adamw_sr_batch_equals_single_calls(lib):
    shapes = [(256, 256), (128, 512), (384, 128)]
    hp = dqt.adamw(1e-3, 0.9, 0.95, 1e-8, 0.05)
    ents, singles = [], []
    for li, (d_out, d_in) in enumerate(shapes):
        q = W.draw_ternary((d_out, d_in), SEED, 40, li)
        w = make_weight(d_out, d_in, "ternary", -1, 1, 0.01 + 0.001 * li, tensor_id=li)
        g = torch.from_numpy(W.draw_normal((d_out, d_in), 1e-2, SEED, 41, li)).to(DEV)
        m0 = torch.from_numpy(W.draw_normal((d_out, d_in), 1e-3, SEED, 42, li)).to(DEV)
        v0 = torch.from_numpy(np.abs(W.draw_normal((d_out, d_in), 1e-4, SEED, 43, li))).to(DEV)
        ents.append(dict(w=w, Wq=weight_codes_dev(q, "ternary"), dW=g, m=m0.clone(), v=v0.clone()))
        singles.append(dict(w=w, Wq=weight_codes_dev(q, "ternary"), dW=g, m=m0.clone(), v=v0.clone()))
    io = dqt.linear_io([dict(w=e["w"], Wq=e["Wq"], dW=e["dW"]) for e in ents])
    c1 = torch.zeros((2,), dtype=torch.int64, device=DEV)
    c2 = torch.zeros((2,), dtype=torch.int64, device=DEV)
    dqt.dqt_adamw_sr_update_batch(io, [e["m"] for e in ents], [e["v"] for e in ents], hp, 5, 4, c1)
    for s in singles:
        dqt.dqt_adamw_sr_update(s["w"], s["Wq"], s["dW"], s["m"], s["v"], hp, 5, 4, c2)
    torch.cuda.synchronize()
    assert torch.equal(c1, c2)
    for e, s in zip(ents, singles):
        assert torch.equal(e["Wq"], s["Wq"])
        assert torch.equal(e["m"], s["m"]) and torch.equal(e["v"], s["v"])


def test_adamw_sr_at_a_large_step(lib):
    """At a large step the bias corrections are 1 - b^t with b^t formed by
    binary exponentiation on both sides: same codes, m and v as the oracle."""
    d_out, d_in, alpha = 128, 256, 0.02
    q = W.draw_ternary((d_out, d_in), SEED, 60, 1)
    g = W.draw_normal((d_out, d_in), 1e-2, SEED, 60, 2).astype(np.float32)
    m0 = W.draw_normal((d_out, d_in), 1e-3, SEED, 60, 3).astype(np.float32)
    v0 = np.abs(W.draw_normal((d_out, d_in), 1e-4, SEED, 60, 4)).astype(np.float32)
    w = make_weight(d_out, d_in, "ternary", -1, 1, alpha, tensor_id=1)
    Wq = weight_codes_dev(q, "ternary")
    m_d, v_d = torch.from_numpy(m0.copy()).to(DEV), torch.from_numpy(v0.copy()).to(DEV)
    dW = torch.from_numpy(g).to(DEV)
    step = 123457
    hp = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01)
    dqt.dqt_adamw_sr_update(w, Wq, dW, m_d, v_d, dqt.adamw(**hp), SEED, step)
    torch.cuda.synchronize()
    want, mw, vw, _, _ = O.adamw_sr_update(q.ravel(), g.ravel(), m0.ravel(), v0.ravel(), hp["lr"],
                                           alpha, hp["beta1"], hp["beta2"], hp["eps"],
                                           hp["weight_decay"], -1, 1, SEED, step, 1)
    assert np.array_equal(weight_codes_host(Wq, "ternary", d_in).ravel(), want)
    assert np.array_equal(_bits(m_d.cpu().numpy().ravel()), _bits(mw))
    assert np.array_equal(_bits(v_d.cpu().numpy().ravel()), _bits(vw))
