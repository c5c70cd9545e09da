"""Pins of the oracle's AdamW-with-SR update (Sec. 4.1 names AdamW with
stochastic rounding; the convention is reading R11 of the oracle): the
target against torch's own AdamW in float64, reductions to the plain SR
update and to pure weight decay, and the non-finite rule."""
import numpy as np
import pytest
import torch

from oracle import dqt_oracle as O


def _draws(n, seed):
    rng = np.random.default_rng(seed)
    q = rng.integers(-3, 4, size=n).astype(np.int64)
    gs = [rng.normal(0.0, s, size=n).astype(np.float32) for s in (1e-2, 3e-3, 2e-2)]
    return q, gs


@pytest.mark.parametrize("wd", [0.0, 0.1])
def test_target_matches_torch_adamw_float64(wd):
    """x = q + delta equals torch.optim.AdamW's updated weight / alpha (the
    weight reset to alpha q before every step, the moments carried), and m, v
    equal its exp_avg, exp_avg_sq, to fp32 rounding, over three steps."""
    n = 4096
    q, gs = _draws(n, 11)
    alpha, lr, b1, b2, eps = 0.02, 1e-3, 0.9, 0.95, 1e-8
    p = torch.zeros(n, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.AdamW([p], lr=lr, betas=(b1, b2), eps=eps, weight_decay=wd)
    m = np.zeros(n, np.float32)
    v = np.zeros(n, np.float32)
    w0 = alpha * q.astype(np.float64)
    for t, g in enumerate(gs, start=1):
        with torch.no_grad():
            p.copy_(torch.from_numpy(w0))
        p.grad = torch.from_numpy(g.astype(np.float64))
        opt.step()
        want_delta = (p.detach().numpy() - w0) / alpha
        k = O.adamw_scalars(lr, alpha, b1, b2, eps, wd, t)
        delta, m, v = O.adamw_target(q, g, m, v, k)
        st = opt.state[p]
        # m sums terms of either sign: fp32 rounding is relative to the terms
        m_ref = st["exp_avg"].numpy()
        np.testing.assert_allclose(m, m_ref, rtol=2e-6, atol=1e-6 * np.abs(m_ref).max())
        np.testing.assert_allclose(v, st["exp_avg_sq"].numpy(), rtol=2e-6, atol=1e-14)
        scale = np.abs(want_delta).max()
        np.testing.assert_allclose(delta, want_delta, rtol=1e-5, atol=1e-6 * scale)


def test_reduces_to_plain_sr_of_the_gradient_sign():
    """b1 = b2 = 0, eps = 0, no decay: m' = g, v' = g^2, u = g / |g|, so the
    update is the plain SR update with gradient sign(g) and the same step
    size (lr / alpha exact), bit for bit, with the same draws."""
    n = 20000
    rng = np.random.default_rng(5)
    q = rng.integers(-1, 2, size=n).astype(np.int64)
    g = rng.normal(0, 1e-3, size=n).astype(np.float32)
    g[g == 0] = np.float32(1e-3)
    m = rng.normal(0, 1, size=n).astype(np.float32)      # forgotten at b1 = 0
    v = np.abs(rng.normal(0, 1, size=n)).astype(np.float32)
    lr, alpha = 0.375, 0.5                               # c = 0.75 exactly
    got, m1, v1, nch, nnf = O.adamw_sr_update(q, g, m, v, lr, alpha, 0.0, 0.0, 0.0, 0.0, -1, 1,
                                              seed=9, step=3, tensor_id=2)
    want, nch2, _ = O.sr_update(q, np.sign(g).astype(np.float32), lr, alpha, -1, 1, 9, 3, 2)
    assert np.array_equal(got, want)
    assert nch == nch2 and nnf == 0
    assert np.array_equal(m1, g) and np.array_equal(v1, (g * g).astype(np.float32))
    # an integer step moves deterministically: c = 1 -> q - sign(g), clipped
    got1, *_ = O.adamw_sr_update(q, g, m, v, 0.5, 0.5, 0.0, 0.0, 0.0, 0.0, -1, 1, 9, 3, 2)
    assert np.array_equal(got1, np.clip(q - np.sign(g).astype(np.int64), -1, 1))


def test_weight_decay_alone():
    """g = 0, m = v = 0: delta = -lr wd q.  lr wd = 1 sends every code to 0;
    lr wd = 0.3 keeps a code of +-1 with probability 0.7 (Eq. 1)."""
    n = 200000
    q = np.where(np.arange(n) % 2 == 0, 1, -1).astype(np.int64)
    z = np.zeros(n, np.float32)
    got, m1, v1, nch, _ = O.adamw_sr_update(q, z, z, z, 1.0, 0.05, 0.9, 0.999, 1e-8, 1.0, -1, 1,
                                            seed=1, step=7, tensor_id=0)
    assert np.all(got == 0) and nch == n
    assert np.all(m1 == 0) and np.all(v1 == 0)
    got, *_ = O.adamw_sr_update(q, z, z, z, 0.5, 0.05, 0.9, 0.999, 1e-8, 0.6, -1, 1,
                                seed=1, step=7, tensor_id=0)
    kept = np.mean(got == q)
    p = 1.0 - float(np.float32(np.float32(0.5) * np.float32(0.6)))
    sd = np.sqrt(p * (1 - p) / n)
    assert abs(kept - p) < 5 * sd, (kept, p)
    assert np.all((got == q) | (got == 0))


def test_nonfinite_gradient_keeps_weight_and_moments():
    q = np.array([1, -1, 0, 1, 0], np.int64)
    g = np.array([np.inf, np.nan, -np.inf, 1e-3, -1e-3], np.float32)
    m = np.array([0.5, -0.25, 0.125, 0.0, 0.0], np.float32)
    v = np.array([1.0, 2.0, 3.0, 0.0, 0.0], np.float32)
    got, m1, v1, nch, nnf = O.adamw_sr_update(q, g, m, v, 1e-2, 0.01, 0.9, 0.999, 1e-8, 0.0,
                                              -1, 1, seed=3, step=1, tensor_id=4)
    assert nnf == 3
    assert np.array_equal(got[:3], q[:3])
    assert np.array_equal(m1[:3], m[:3]) and np.array_equal(v1[:3], v[:3])
    assert np.all(np.isfinite(m1)) and np.all(np.isfinite(v1))


def test_pow_by_squaring_is_repeated_multiplication_for_small_t():
    for b in (0.9, 0.95, 0.999, 0.5):
        r = 1.0
        for t in range(0, 40):
            assert O.pow_by_squaring(b, t) == pytest.approx(r, rel=1e-13, abs=0)
            assert O.pow_by_squaring(b, t) == pytest.approx(b ** t, rel=1e-13, abs=0)
            r *= b
