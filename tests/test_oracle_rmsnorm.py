"""Pins of the oracle's RMSNorm + activation quantisation (reading R13: the
LLaMA block's RMSNorm ahead of the 8-bit activations of Sec. 3.2), checked
against what mathematics and independent code fix, not against itself."""
import struct

import numpy as np
import torch

from oracle import dqt_oracle as O


def _f32(x: float) -> float:
    """Round a Python float (binary64) to binary32."""
    return struct.unpack("f", struct.pack("f", x))[0]


def _brute_sum_squares(row):
    """The fixed order of R13 written as plain loops over lanes, chunks and
    elements, one binary32 rounding after each operation."""
    K = len(row)
    nchunk = K // 8
    lane = [0.0] * 64
    for l in range(64):
        for c in range(l, nchunk, 64):
            for j in range(8):
                x = float(row[8 * c + j])
                lane[l] = _f32(lane[l] + _f32(x * x))
    for d in (32, 16, 8, 4, 2, 1):
        lane = [_f32(lane[l] + lane[l ^ d]) for l in range(64)]
    return lane[0]


def test_sum_of_squares_matches_brute_force_loops():
    rng = np.random.default_rng(0)
    for K in (16, 48, 512, 528, 1040):
        X = (rng.standard_normal((3, K)) * np.exp(rng.uniform(-6, 6, (3, K)))).astype(np.float32)
        got = O.rms_sum_squares(X)
        for m in range(3):
            assert got[m] == np.float32(_brute_sum_squares(X[m])), (K, m)


def test_sum_of_squares_exact_on_small_integers():
    """Squares of small integers and their sums are exact in fp32, so every
    order gives the exact integer sum: any dropped or repeated element
    shows."""
    rng = np.random.default_rng(1)
    for K in (16, 64, 520, 4096, 11008):
        X = rng.integers(-20, 21, size=(4, K)).astype(np.float32)
        exact = (X.astype(np.int64) ** 2).sum(axis=1)
        assert np.array_equal(O.rms_sum_squares(X).astype(np.int64), exact), K


def test_rmsnorm_against_torch_float64():
    rng = np.random.default_rng(2)
    for K, eps in ((64, 1e-6), (768, 1e-5), (4096, 1e-6)):
        X = rng.standard_normal((5, K)).astype(np.float32) * np.float32(3.0)
        g = (1.0 + 0.1 * rng.standard_normal(K)).astype(np.float32)
        y, r = O.rmsnorm(X, g, eps)
        ref = torch.nn.functional.rms_norm(torch.from_numpy(X).double(), (K,),
                                           torch.from_numpy(g).double(), eps=eps).numpy()
        assert np.allclose(y, ref, rtol=2e-6, atol=1e-30), K
        rref = 1.0 / np.sqrt((X.astype(np.float64) ** 2).mean(axis=1) + eps)
        assert np.allclose(r, rref, rtol=1e-6)


def test_constant_row_closed_form_and_scale_invariance():
    K = 256
    g = np.linspace(0.5, 2.0, K).astype(np.float32)
    X = np.full((2, K), 0.125, np.float32)
    X[1] = -0.125
    y, r = O.rmsnorm(X, g, 0.0)
    assert np.array_equal(r, np.array([8.0, 8.0], np.float32))
    assert np.array_equal(y[0], g) and np.array_equal(y[1], -g)
    # with eps = 0 a power-of-two scale of the input leaves y bit for bit
    rng = np.random.default_rng(3)
    X = rng.standard_normal((4, 1024)).astype(np.float32)
    y1, _ = O.rmsnorm(X, g.repeat(4), 0.0)
    y2, _ = O.rmsnorm(X * np.float32(32.0), g.repeat(4), 0.0)
    assert np.array_equal(y1, y2)


def test_rmsnorm_act_quant_composes_and_zero_row():
    rng = np.random.default_rng(4)
    K = 512
    X = rng.standard_normal((6, K)).astype(np.float32)
    X[2] = 0.0
    g = (1.0 + 0.2 * rng.standard_normal(K)).astype(np.float32)
    for kind, top in (("i8", 127), ("e4m3", 0x7E)):
        Xq, d, r, y = O.rmsnorm_act_quant(X, g, 1e-5, kind)
        # the largest |y| of each nonzero row maps to the largest code
        for m in (0, 1, 3):
            k = int(np.argmax(np.abs(y[m])))
            code = int(Xq[m, k]) if kind == "i8" else int(Xq[m, k]) & 0x7F
            assert code == (top if kind == "e4m3" else int(np.sign(y[m, k])) * top)
        # a zero row: r = 1 / sqrt(eps), y = 0, codes 0 and the eps scale
        assert r[2] == np.float32(1.0) / np.sqrt(np.float32(1e-5))
        assert not Xq[2].any() and d[2] == np.float32(1e-5) / np.float32(127 if kind == "i8" else 448)
