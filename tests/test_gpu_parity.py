"""GPU parity: every entry point of libdqt against the CPU oracle on the same
seeded inputs.  Bit-exact for the random stream, activation quantisation, the
int8 forward and the SR update; within the stated tolerance for the fp8
forward and the backward products."""
import numpy as np
import pytest
import torch

from oracle import dqt_oracle as O
from paper_2412_04787_amd import dqt, workloads as W

from gpu_util import (DEV, act_code, gemm_close, log, make_weight, run_bwd, run_fwd, to_dev,
                      weight_codes_dev, weight_codes_host)

pytestmark = pytest.mark.gpu

SEED = 1234


def draws(shape, std, *stream):
    return W.draw_normal(shape, std, SEED, 99, *stream)


# ------------------------------------------------------------------ RNG

@pytest.mark.parametrize("seed,step,tid,i0,n", [
    (0, 1, 0, 0, 1 << 16),
    (12345, 7, 3, 5, 100_003),
    ((1 << 63) + 17, 0xFFFFFFFF, 0xABCDEF01, (1 << 40) + 3, 4099),
])
def test_rng_stream_bit_exact(lib, seed, step, tid, i0, n):
    out = torch.empty((n,), dtype=torch.int32, device=DEV)
    dqt.dqt_debug_rng(seed, step, tid, i0, out)
    got = out.cpu().numpy().view(np.uint32)
    want = O.rng_u32(seed, step, tid, np.arange(i0, i0 + n, dtype=np.uint64))
    assert np.array_equal(got, want)


# ------------------------------------------------------------ act quant

@pytest.mark.parametrize("M,K", [(1, 16), (37, 272), (513, 768), (64, 11008), (5, 20480)])
@pytest.mark.parametrize("x_t", ["f32", "bf16"])
@pytest.mark.parametrize("act", ["i8", "e4m3"])
def test_act_quant_bit_exact(lib, M, K, x_t, act):
    X = draws((M, K), 1.0, 1, M, K)
    X[0, :] *= 1e-9            # eps path
    if M > 3:
        X[3, :] = 0.0          # all-zero row
        X[2, 5] = 37.5         # one outlier
    X_dev, X_seen = to_dev(X, x_t)
    Xq = torch.empty((M, K), dtype=torch.uint8, device=DEV)
    xdq = torch.empty((M,), dtype=torch.float32, device=DEV)
    dqt.dqt_act_quant(X_dev, act_code(act), Xq, xdq)
    want_q, want_d = O.act_quant(X_seen, act)
    assert np.array_equal(xdq.cpu().numpy(), want_d)
    assert np.array_equal(Xq.cpu().numpy(), want_q.view(np.uint8))


def _rounding_cases(act):
    """fp32 values at unit scale: every code's value, the midpoints between
    neighbouring codes (the ties), one ulp either side of each, tiny and
    subnormal values, both signs."""
    if act == "e4m3":
        grid = np.array(sorted({float(O.act_values(np.array([c], dtype=np.uint8), "e4m3")[0])
                                for c in range(0x7F)}), dtype=np.float64)
    else:
        grid = np.arange(-128.0, 128.0)
    grid = np.abs(grid) if act == "e4m3" else grid
    mids = (grid[:-1] + grid[1:]) / 2
    v = np.concatenate([grid, mids]).astype(np.float32)
    v = np.concatenate([v, np.nextafter(v, np.float32(np.inf)), np.nextafter(v, np.float32(-np.inf)),
                        np.float32([1e-30, 1e-40, 2.0 ** -10, 2.0 ** -11, 3 * 2.0 ** -11])])
    v = np.concatenate([v, -v])
    top = np.float32(448.0 if act == "e4m3" else 127.0)
    return v[np.abs(v) <= top], top


@pytest.mark.parametrize("act", ["i8", "e4m3"])
def test_act_quant_rounding_at_every_tie(lib, act):
    """Rows whose absmax is the format's largest value quantise at scale 1
    exactly, so each code is the rounding of the value itself: every tie
    between neighbouring codes and its neighbours against the oracle."""
    v, top = _rounding_cases(act)
    K = 512
    rows = (v.size + K - 2) // (K - 1)
    X = np.zeros((rows, K), dtype=np.float32)
    X[:, 0] = top                                  # absmax of every row
    X[:, 1:].flat[:v.size] = v
    X_dev, X_seen = to_dev(X, "f32")
    assert np.array_equal(X_seen, X)
    Xq = torch.empty((rows, K), dtype=torch.uint8, device=DEV)
    xdq = torch.empty((rows,), dtype=torch.float32, device=DEV)
    dqt.dqt_act_quant(X_dev, act_code(act), Xq, xdq)
    want_q, want_d = O.act_quant(X_seen, act)
    assert np.array_equal(xdq.cpu().numpy(), want_d)
    assert np.array_equal(Xq.cpu().numpy(), want_q.view(np.uint8))


@pytest.mark.parametrize("x_t", ["f32", "bf16"])
@pytest.mark.parametrize("act", ["i8", "e4m3"])
def test_act_quant_batch_matches_oracle(lib, x_t, act):
    """Inputs of six row lengths in one call: rows of up to 256 chunks share
    one launch whose blocks run 1, 4, 8 or 16 chunks per lane (by input),
    longer rows take the whole-wave kernel."""
    M = 257
    Ks = [768, 2048, 272, 11008, 16, 512]
    ents, seen = [], []
    for i, K in enumerate(Ks):
        X = draws((M, K), 1.0, 11, i, K)
        X[7, :] = 0.0
        X_dev, X_seen = to_dev(X, x_t)
        Xq = torch.empty((M, K), dtype=torch.uint8, device=DEV)
        xdq = torch.empty((M,), dtype=torch.float32, device=DEV)
        ents.append((X_dev, Xq, xdq))
        seen.append(X_seen)
    io = dqt.act_io(ents)
    dqt.dqt_act_quant_batch(io, dqt.dtype_code(ents[0][0]), M, act_code(act))
    for (X_dev, Xq, xdq), X_seen in zip(ents, seen):
        want_q, want_d = O.act_quant(X_seen, act)
        assert np.array_equal(xdq.cpu().numpy(), want_d)
        assert np.array_equal(Xq.cpu().numpy(), want_q.view(np.uint8))


# -------------------------------------------------------------- forward

FWD_SHAPES = [(1, 16, 16), (300, 272, 400), (512, 256, 256), (129, 48, 144), (1000, 1024, 208),
              (257, 320, 96),   # d_in 320: packed codes with a half step at the end
              (70, 64, 80),     # d_in 64: the whole reduction one half step
              (1, 128, 16)]     # one token, one step
FWD_KINDS = [  # act, wfmt, qmin, qmax, x_t, y_out
    ("i8", "ternary", -1, 1, "f32", "f32"),
    ("i8", "ternary", -1, 1, "bf16", "bf16"),
    ("i8", "i8", -127, 127, "bf16", "f32"),
    ("i8", "i8", -128, 127, "f32", "bf16"),
    ("e4m3", "ternary", -1, 1, "bf16", "f32"),
    ("e4m3", "ternary", -1, 1, "f32", "bf16"),
    ("i8", "i4", -8, 7, "bf16", "bf16"),
    ("i8", "i4", -4, 3, "f32", "f32"),
    ("e4m3", "i4", -8, 7, "bf16", "f32"),
    ("i8", "i3", -4, 3, "bf16", "bf16"),
    ("e4m3", "i3", -4, 3, "f32", "f32"),
]


def _weights(d_out, d_in, wfmt, qmin, qmax, *stream):
    if wfmt == "ternary":
        return W.draw_ternary((d_out, d_in), SEED, 99, 50, *stream)
    return W.draw_int((d_out, d_in), qmin, qmax, SEED, 99, 51, *stream)


@pytest.mark.parametrize("shape", FWD_SHAPES)
@pytest.mark.parametrize("kind", FWD_KINDS)
def test_forward(lib, shape, kind):
    M, d_in, d_out = shape
    act, wfmt, qmin, qmax, x_t, y_out = kind
    log(f"forward M={M} d_in={d_in} d_out={d_out} {kind}")
    q = _weights(d_out, d_in, wfmt, qmin, qmax, M, d_in, d_out)
    alpha = np.float32(0.0161)
    w = make_weight(d_out, d_in, wfmt, qmin, qmax, alpha)
    Wq = weight_codes_dev(q, wfmt)
    X_dev, X_seen = to_dev(draws((M, d_in), 1.0, 2, M, d_in), x_t)
    Xq, xdq, Y = run_fwd(w, Wq, X_dev, act, y_out)
    want_q, want_d = O.act_quant(X_seen, act)
    assert np.array_equal(Xq.cpu().numpy().view(np.uint8), want_q.view(np.uint8))
    Y_ref, acc = O.linear_fwd(want_q, want_d, act, q, alpha, y_out)
    got = Y.float().cpu().numpy()
    if act == "i8":
        assert np.array_equal(got, Y_ref), np.argwhere(got != Y_ref)[:5]
    else:
        a = np.abs(O.act_values(want_q, act)) @ np.abs(q.astype(np.float64)).T
        f = (want_d * alpha).astype(np.float64)[:, None]
        ok, nbad, emax = gemm_close(got, acc * f, a * f, bf16_out=(y_out == "bf16"))
        assert ok, (nbad, emax)


PACKED_SHAPES = [(512, 256, 256), (1000, 1024, 208), (257, 320, 96), (70, 64, 80), (1, 128, 16)]


@pytest.mark.parametrize("shape", PACKED_SHAPES)
@pytest.mark.parametrize("act", ["i8", "e4m3"])
def test_forward_packed_form_with_the_smallest_workspace(lib, shape, act):
    """Ternary codes with d_in a multiple of 64 given only the 256 counter
    bytes of workspace run from the packed codes, expanded in registers
    (int8 bytes, or FP4 values against e4m3 activations): int8 bit for bit
    equal to the expanded form and the oracle, e4m3 within the tolerance."""
    M, d_in, d_out = shape
    log(f"forward packed form M={M} d_in={d_in} d_out={d_out} {act}")
    q = _weights(d_out, d_in, "ternary", -1, 1, M, d_in, d_out, 7)
    alpha = np.float32(0.0173)
    w = make_weight(d_out, d_in, "ternary", -1, 1, alpha)
    Wq = weight_codes_dev(q, "ternary")
    X_dev, X_seen = to_dev(draws((M, d_in), 1.0, 3, M, d_in), "bf16")
    code = dqt.DQT_I8 if act == "i8" else dqt.DQT_FP8E4M3
    Xq = torch.empty((M, d_in), dtype=torch.int8 if act == "i8" else torch.uint8, device=DEV)
    xdq = torch.empty((M,), dtype=torch.float32, device=DEV)
    full = dqt.dqt_linear_fwd_workspace(w)
    assert full >= 256 + d_out * d_in            # the expansion's bytes
    outs = []
    for nbytes in (full, 256):
        ws = dqt.workspace(nbytes)
        Y = torch.empty((M, d_out), dtype=torch.float32, device=DEV)
        dqt.dqt_linear_fwd(w, Wq, X_dev, M, code, Xq, xdq, Y, ws)
        outs.append(Y.cpu().numpy())
    # one byte short of the counters is refused
    with pytest.raises(dqt.DqtError):
        Y = torch.empty((M, d_out), dtype=torch.float32, device=DEV)
        dqt.dqt_linear_fwd(w, Wq, X_dev, M, code, Xq, xdq, Y, dqt.workspace(256)[:-1])
    want_q, want_d = O.act_quant(X_seen, act)
    Y_ref, acc = O.linear_fwd(want_q, want_d, act, q, alpha, "f32")
    if act == "i8":
        assert np.array_equal(outs[0], Y_ref) and np.array_equal(outs[1], Y_ref)
    else:
        a = np.abs(O.act_values(want_q, act)) @ np.abs(q.astype(np.float64)).T
        f = (want_d * alpha).astype(np.float64)[:, None]
        for got in outs:
            ok, nbad, emax = gemm_close(got, acc * f, a * f, bf16_out=False)
            assert ok, (nbad, emax)


# ------------------------------------------------------------- backward

BWD_SHAPES = [(1, 16, 16), (300, 272, 400), (512, 256, 256), (2100, 96, 160), (4097, 128, 48)]
BWD_KINDS = [  # act, wfmt, qmin, qmax, xt (= dY dtype), dx_out
    ("i8", "ternary", -1, 1, "f32", "f32"),
    ("i8", "ternary", -1, 1, "bf16", "bf16"),
    ("i8", "i8", -127, 127, "bf16", "f32"),
    ("e4m3", "ternary", -1, 1, "bf16", "bf16"),
    ("i8", "i8", -128, 127, "f32", "bf16"),
    ("e4m3", "ternary", -1, 1, "f32", "f32"),
    ("i8", "i4", -8, 7, "bf16", "bf16"),
    ("i8", "i4", -2, 1, "f32", "f32"),
    ("e4m3", "i4", -4, 3, "bf16", "bf16"),
    ("i8", "i3", -4, 3, "bf16", "bf16"),
    ("i8", "i3", -2, 1, "f32", "f32"),
]


@pytest.mark.parametrize("shape", BWD_SHAPES)
@pytest.mark.parametrize("kind", BWD_KINDS)
def test_backward(lib, shape, kind):
    M, d_in, d_out = shape
    act, wfmt, qmin, qmax, xt, dx_out = kind
    log(f"backward M={M} d_in={d_in} d_out={d_out} {kind}")
    q = _weights(d_out, d_in, wfmt, qmin, qmax, M, d_in, d_out, 7)
    alpha = np.float32(0.0213)
    w = make_weight(d_out, d_in, wfmt, qmin, qmax, alpha)
    Wq = weight_codes_dev(q, wfmt)
    X_dev, X_seen = to_dev(draws((M, d_in), 1.0, 3, M, d_in), xt)
    dY_dev, dY_seen = to_dev(draws((M, d_out), 1e-2, 4, M, d_out), xt)
    Xq, xdq, _ = run_fwd(w, Wq, X_dev, act, "f32")
    dX, dW = run_bwd(w, Wq, Xq, act, xdq, dY_dev, xt, dx_out)
    want_q, want_d = O.act_quant(X_seen, act)
    _, _, dX64, dW64 = O.linear_bwd(dY_seen, q, alpha, want_q, want_d, act, xt, dx_out)
    xt_vals = O.act_dequant(want_q, want_d, act, xt)
    bx = float(alpha) * O.gemm_abs_bound(dY_seen, q.astype(np.float64))
    ok, nbad, emax = gemm_close(dX.float().cpu().numpy(), dX64, bx, bf16_out=(dx_out == "bf16"))
    assert ok, ("dX", nbad, emax)
    bw = O.gemm_abs_bound(dY_seen.T, xt_vals)
    ok, nbad, emax = gemm_close(dW.cpu().numpy(), dW64, bw)
    assert ok, ("dW", nbad, emax)


@pytest.mark.parametrize("act,wfmt,qmin,qmax", [("i8", "i8", -128, 127), ("e4m3", "ternary", -1, 1)])
def test_maximum_reduction_length(lib, act, wfmt, qmin, qmax):
    """d_in = 65536, the largest the library takes: the forward (one token's
    int32 sum at 127 * 128 * 65536 for int8 codes, exact), dX, dW and the SR
    update of the same weights against the oracle."""
    M, d_in, d_out = 40, 65536, 32
    log(f"maximum d_in: M={M} d_in={d_in} d_out={d_out} {act} {wfmt}")
    q = _weights(d_out, d_in, wfmt, qmin, qmax, M, d_in, d_out, 11)
    q[0, :] = qmin                                  # the largest |sum| of row 0 of Y
    alpha = np.float32(0.0137)
    w = make_weight(d_out, d_in, wfmt, qmin, qmax, alpha, tensor_id=2)
    Wq = weight_codes_dev(q, wfmt)
    X = draws((M, d_in), 1.0, 12, M, d_in)
    X[0, :] = -1.0
    X_dev, X_seen = to_dev(X, "bf16")
    Xq, xdq, Y = run_fwd(w, Wq, X_dev, act, "f32")
    want_q, want_d = O.act_quant(X_seen, act)
    Y_ref, acc = O.linear_fwd(want_q, want_d, act, q, alpha, "f32")
    if act == "i8":
        assert int(np.max(np.abs(acc))) == 127 * 128 * 65536
        assert np.array_equal(Y.cpu().numpy(), Y_ref)
    else:
        a = np.abs(O.act_values(want_q, act)) @ np.abs(q.astype(np.float64)).T
        f = (want_d * alpha).astype(np.float64)[:, None]
        ok, nbad, emax = gemm_close(Y.cpu().numpy(), acc * f, a * f, bf16_out=False)
        assert ok, (nbad, emax)
    dY_dev, dY_seen = to_dev(draws((M, d_out), 1e-2, 13, M, d_out), "bf16")
    dX, dW = run_bwd(w, Wq, Xq, act, xdq, dY_dev, "bf16", "f32")
    _, _, dX64, dW64 = O.linear_bwd(dY_seen, q, alpha, want_q, want_d, act, "bf16", "f32")
    bx = float(alpha) * O.gemm_abs_bound(dY_seen, q.astype(np.float64))
    ok, nbad, emax = gemm_close(dX.cpu().numpy(), dX64, bx)
    assert ok, ("dX", nbad, emax)
    bw = O.gemm_abs_bound(dY_seen.T, O.act_dequant(want_q, want_d, act, "bf16"))
    ok, nbad, emax = gemm_close(dW.cpu().numpy(), dW64, bw)
    assert ok, ("dW", nbad, emax)
    counters = torch.zeros((2,), dtype=torch.int64, device=DEV)
    dqt.dqt_sr_update(w, Wq, dW, 3e-3, 9, 1, counters)
    g = dW.cpu().numpy()
    want, n_changed, n_nonfinite = O.sr_update(q.ravel(), g.ravel(), 3e-3, alpha, qmin, qmax, 9, 1, 2)
    assert np.array_equal(weight_codes_host(Wq, wfmt, d_in).ravel(), want)
    assert int(counters[0].item()) == n_changed and int(counters[1].item()) == n_nonfinite


def test_backward_empty_tokens_writes_zero_dw(lib):
    w = make_weight(48, 32, "ternary", -1, 1, 0.01)
    Wq = weight_codes_dev(np.zeros((48, 32), np.int8), "ternary")
    dW = torch.full((48, 32), 7.0, dtype=torch.float32, device=DEV)
    dY = torch.empty((0, 48), dtype=torch.float32, device=DEV)
    Xq = torch.empty((0, 32), dtype=torch.int8, device=DEV)
    xdq = torch.empty((1,), dtype=torch.float32, device=DEV)
    for xt in (dqt.DQT_F32, dqt.DQT_BF16):
        dW.fill_(7.0)
        dYt = dY if xt == dqt.DQT_F32 else dY.to(torch.bfloat16)
        ws = dqt.workspace(dqt.dqt_linear_bwd_workspace(w, 0))
        dqt.dqt_linear_bwd(w, Wq, Xq, dqt.DQT_I8, xdq, dYt, 0, xt, None, dW, ws)
        assert torch.count_nonzero(dW).item() == 0
    assert torch.count_nonzero(dW).item() == 0


def test_backward_is_deterministic(lib):
    M, d_in, d_out = 3000, 256, 128
    w = make_weight(d_out, d_in, "ternary", -1, 1, 0.02)
    q = _weights(d_out, d_in, "ternary", -1, 1, 77)
    Wq = weight_codes_dev(q, "ternary")
    X_dev, _ = to_dev(draws((M, d_in), 1.0, 5), "bf16")
    dY_dev, _ = to_dev(draws((M, d_out), 1e-2, 6), "bf16")
    Xq, xdq, _ = run_fwd(w, Wq, X_dev, "i8", "bf16")
    a = run_bwd(w, Wq, Xq, "i8", xdq, dY_dev, "bf16", "bf16")
    b = run_bwd(w, Wq, Xq, "i8", xdq, dY_dev, "bf16", "bf16")
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


# ------------------------------------------------------------- SR update

SR_CASES = [  # d_out, d_in, wfmt, qmin, qmax, lr, alpha, gscale
    (16, 16, "ternary", -1, 1, 1e-3, 0.016, 1.0),
    (256, 256, "ternary", -1, 1, 1e-3, 0.016, 0.2),
    (400, 272, "ternary", -1, 1, 0.5, 0.01, 1.0),
    (144, 48, "i8", -127, 127, 3e-4, 1e-4, 1.0),
    (768, 2048, "i8", -128, 127, 1e-2, 1e-3, 3.0),
    (1024, 1024, "ternary", -1, 1, 3e-4, 0.0159, 0.01),
    (256, 384, "i4", -8, 7, 1e-2, 2e-3, 1.0),
    (144, 48, "i4", -4, 3, 0.3, 0.02, 1.0),
    (256, 384, "i3", -4, 3, 1e-2, 2e-3, 1.0),
    (144, 48, "i3", -4, 3, 0.3, 0.02, 1.0),
]


@pytest.mark.parametrize("case", SR_CASES)
def test_sr_update_bit_exact(lib, case):
    d_out, d_in, wfmt, qmin, qmax, lr, alpha, gscale = case
    log(f"sr_update {case}")
    q = _weights(d_out, d_in, wfmt, qmin, qmax, d_out, d_in, 9)
    g = draws((d_out, d_in), gscale, 8, d_out, d_in)
    flat = g.reshape(-1)
    flat[::997] *= 1e6                    # saturating moves
    flat[5] = np.nan
    flat[11] = np.inf
    flat[12] = -np.inf
    flat[::1013] = 0.0                     # on-grid: no move
    w = make_weight(d_out, d_in, wfmt, qmin, qmax, alpha, tensor_id=5)
    Wq = weight_codes_dev(q, wfmt)
    dW = torch.from_numpy(g).to(DEV)
    counters = torch.zeros((2,), dtype=torch.int64, device=DEV)
    dqt.dqt_sr_update(w, Wq, dW, lr, 42, 3, counters)
    got = weight_codes_host(Wq, wfmt, d_in)
    want, n_changed, n_nonfinite = O.sr_update(q.ravel(), g.ravel(), lr, alpha, qmin, qmax, 42, 3, 5)
    want = want.reshape(d_out, d_in)
    assert np.array_equal(got, want), np.argwhere(got != want)[:5]
    c = counters.cpu().numpy()
    assert int(c[0]) == n_changed and int(c[1]) == n_nonfinite
    # counters accumulate
    dqt.dqt_sr_update(w, Wq, dW, lr, 42, 4, counters)
    assert int(counters[1].item()) == 2 * n_nonfinite


def test_sr_update_ternary_small_steps_any_codes(lib):
    """Ternary codes as raw bytes (invalid code 3 included, which the rule
    reads as q = 2 and clips), steps |delta| < 1 on most chunks (the common
    case of training), some chunks with |delta| >= 1 or a non-finite
    gradient, and enough elements that draws equal to the threshold's top
    16 bits occur: every weight against the oracle."""
    d_out, d_in = 1024, 1024
    n = d_out * d_in
    rng = np.random.default_rng(2024)
    raw = rng.integers(0, 256, size=(d_out, d_in // 4), dtype=np.uint8)
    q = O.unpack_ternary(raw, d_in)
    g = rng.uniform(-0.999, 0.999, size=(d_out, d_in)).astype(np.float32)
    flat = g.reshape(-1)
    flat[40_003::65_537] = 2.5            # |delta| >= 1 in a few chunks
    flat[123_457] = np.nan
    lr, alpha, seed, step, tid = 1.0, 1.0, 5, 9, 3
    # the oracle's draws: elements whose primary draw equals the top 16 bits
    # of floor(|delta| 2^32) take the secondary draw
    c = O.sr_step_size(lr, alpha)
    delta = -(c * flat)
    u = O.rng_u32(seed, step, tid, np.arange(n, dtype=np.uint64))
    with np.errstate(invalid="ignore"):
        h = np.floor(np.abs(delta.astype(np.float64)) * 65536.0)
    ties = int(np.count_nonzero((np.abs(delta) < 1) & ((u >> 16) == h)))
    assert ties >= 3, ties
    w = make_weight(d_out, d_in, "ternary", -1, 1, alpha, tensor_id=tid)
    Wq = torch.from_numpy(raw.copy()).to(DEV)
    counters = torch.zeros((2,), dtype=torch.int64, device=DEV)
    dqt.dqt_sr_update(w, Wq, torch.from_numpy(g).to(DEV), lr, seed, step, counters)
    got = weight_codes_host(Wq, "ternary", d_in)
    want, n_changed, n_nonfinite = O.sr_update(q.ravel(), flat, lr, alpha, -1, 1, seed, step, tid)
    assert np.array_equal(got.ravel(), want), np.argwhere(got.ravel() != want)[:5]
    assert int(counters[0].item()) == n_changed and int(counters[1].item()) == n_nonfinite == 1


@pytest.mark.parametrize("wfmt,qmin,qmax", [("i4", -8, 7), ("i4", -4, 3), ("i4", -1, 1),
                                             ("i3", -4, 3), ("i3", -2, 1)])
def test_sr_update_packed_small_steps(lib, wfmt, qmin, qmax):
    """4-bit and 3-bit codes, steps |delta| < 1 on most chunks (the lane
    arithmetic of small steps), codes mostly at the grid's edges, a few
    outside the grid (which the rule clips, on any step), some chunks with
    |delta| >= 1 or a non-finite gradient, and draws equal to the
    threshold's top 16 bits: every weight and both counts against the
    oracle."""
    d_out, d_in = 1024, 1024
    n = d_out * d_in
    rng = np.random.default_rng(7 + qmax)
    lo_f, hi_f = (-8, 7) if wfmt == "i4" else (-4, 3)
    q = rng.choice([qmin, qmax, qmin + 1, qmax - 1], size=(d_out, d_in)).astype(np.int8)
    q = np.clip(q, qmin, qmax).astype(np.int8)
    q.reshape(-1)[::4099] = rng.integers(lo_f, hi_f + 1, size=q.reshape(-1)[::4099].shape)  # off-grid too
    g = rng.uniform(-0.999, 0.999, size=(d_out, d_in)).astype(np.float32)
    flat = g.reshape(-1)
    flat[40_003::65_537] = 2.5            # |delta| >= 1 in a few chunks
    flat[123_457] = np.nan
    lr, alpha, seed, step, tid = 1.0, 1.0, 11, 2, 4
    c = O.sr_step_size(lr, alpha)
    delta = -(c * flat)
    u = O.rng_u32(seed, step, tid, np.arange(n, dtype=np.uint64))
    with np.errstate(invalid="ignore"):
        h = np.floor(np.abs(delta.astype(np.float64)) * 65536.0)
    assert int(np.count_nonzero((np.abs(delta) < 1) & ((u >> 16) == h))) >= 3
    assert np.count_nonzero((q < qmin) | (q > qmax)) > 0 or (qmin, qmax) == (lo_f, hi_f)
    w = make_weight(d_out, d_in, wfmt, qmin, qmax, alpha, tensor_id=tid)
    Wq = weight_codes_dev(q, wfmt)
    counters = torch.zeros((2,), dtype=torch.int64, device=DEV)
    dqt.dqt_sr_update(w, Wq, torch.from_numpy(g).to(DEV), lr, seed, step, counters)
    got = weight_codes_host(Wq, wfmt, d_in)
    want, n_changed, n_nonfinite = O.sr_update(q.ravel(), flat, lr, alpha, qmin, qmax, seed, step, tid)
    assert np.array_equal(got.ravel(), want), np.argwhere(got.ravel() != want)[:5]
    assert int(counters[0].item()) == n_changed and int(counters[1].item()) == n_nonfinite == 1


@pytest.mark.parametrize("wfmt,qmin,qmax", [("ternary", -1, 1), ("i4", -8, 7), ("i3", -4, 3), ("i8", -128, 127)])
def test_sr_update_degenerate_steps_change_nothing(lib, wfmt, qmin, qmax):
    """lr = 0 with any gradient, and any lr with a zero gradient (both signs
    of zero): every code stays, nothing is counted."""
    d_out, d_in = 256, 512
    q = _weights(d_out, d_in, wfmt, qmin, qmax, 31)
    w = make_weight(d_out, d_in, wfmt, qmin, qmax, 0.01, tensor_id=1)
    g = draws((d_out, d_in), 1.0, 32, d_out, d_in)
    zero = np.zeros_like(g)
    zero.reshape(-1)[1::2] = -0.0
    for lr, grad in ((0.0, g), (0.5, zero)):
        Wq = weight_codes_dev(q, wfmt)
        counters = torch.zeros((2,), dtype=torch.int64, device=DEV)
        dqt.dqt_sr_update(w, Wq, torch.from_numpy(grad).to(DEV), lr, 3, 7, counters)
        assert np.array_equal(weight_codes_host(Wq, wfmt, d_in), q)
        assert counters.tolist() == [0, 0]


@pytest.mark.parametrize("wfmt,qmin,qmax", [("ternary", -1, 1), ("i4", -4, 3), ("i8", -127, 127)])
def test_sr_update_overflowing_step(lib, wfmt, qmin, qmax):
    """lr / alpha near the top of fp32 (c = 5e37, past the 2^100 bound of
    the small-step paths): c g overflows to an infinite step for about half
    of the gradients (|g| > 6.8) and is finite but far beyond the grid for
    the rest; every code saturates toward its step's sign (the gradients are
    finite, so nothing counts as non-finite), and zero gradients stay put."""
    d_out, d_in = 128, 256
    alpha = np.float32(2e-38)                    # the smallest normal fp32 is 1.18e-38
    q = _weights(d_out, d_in, wfmt, qmin, qmax, 41)
    w = make_weight(d_out, d_in, wfmt, qmin, qmax, alpha, tensor_id=6)
    g = draws((d_out, d_in), 10.0, 42, d_out, d_in)
    g.reshape(-1)[::7] = 0.0
    c = O.sr_step_size(1.0, alpha)
    with np.errstate(over="ignore"):
        assert np.count_nonzero(np.isinf(c * g)) > g.size // 4
    Wq = weight_codes_dev(q, wfmt)
    counters = torch.zeros((2,), dtype=torch.int64, device=DEV)
    dqt.dqt_sr_update(w, Wq, torch.from_numpy(g).to(DEV), 1.0, 8, 2, counters)
    want, n_changed, n_nonfinite = O.sr_update(q.ravel(), g.ravel(), 1.0, alpha, qmin, qmax, 8, 2, 6)
    assert np.array_equal(weight_codes_host(Wq, wfmt, d_in).ravel(), want)
    assert counters.tolist() == [n_changed, n_nonfinite] and n_nonfinite == 0


def test_sr_update_without_counters_and_repeatable(lib):
    d_out, d_in = 512, 512
    q = _weights(d_out, d_in, "ternary", -1, 1, 3)
    g = draws((d_out, d_in), 1.0, 10)
    w = make_weight(d_out, d_in, "ternary", -1, 1, 0.01, tensor_id=1)
    dW = torch.from_numpy(g).to(DEV)
    A = weight_codes_dev(q, "ternary")
    B = weight_codes_dev(q, "ternary")
    dqt.dqt_sr_update(w, A, dW, 1e-2, 7, 1)
    dqt.dqt_sr_update(w, B, dW, 1e-2, 7, 1)
    assert torch.equal(A, B)
    C = weight_codes_dev(q, "ternary")
    dqt.dqt_sr_update(w, C, dW, 1e-2, 7, 2)
    assert not torch.equal(A, C)


def test_sr_worked_example_on_gpu(lib):
    """-1 + 0.02 goes to 0 with probability 2% (Sec. 5), over ~1e7 weights."""
    d_out, d_in = 2560, 4096
    n = d_out * d_in
    alpha, lr = 1.0, 1.0
    q = np.full((d_out, d_in), -1, np.int8)
    w = make_weight(d_out, d_in, "ternary", -1, 1, alpha, tensor_id=2)
    Wq = weight_codes_dev(q, "ternary")
    dW = torch.full((d_out, d_in), -0.02, dtype=torch.float32, device=DEV)
    counters = torch.zeros((2,), dtype=torch.int64, device=DEV)
    dqt.dqt_sr_update(w, Wq, dW, lr, 0, 1, counters)
    got = weight_codes_host(Wq, "ternary", d_in)
    moved = int(np.count_nonzero(got == 0))
    assert set(np.unique(got).tolist()) <= {-1, 0}
    assert moved == int(counters[0].item())
    p = float(np.float32(0.02))
    sd = np.sqrt(p * (1 - p) / n)
    assert abs(moved / n - p) < 5 * sd
    # and bit-exact against the oracle on a sample of elements
    idx = np.random.default_rng(0).choice(n, 20000, replace=False).astype(np.uint64)
    want, _, _ = O.sr_update(np.full(idx.size, -1), np.full(idx.size, -0.02, np.float32),
                             lr, alpha, -1, 1, 0, 1, 2, idx=idx)
    assert np.array_equal(got.ravel()[idx.astype(np.int64)], want)


@pytest.mark.parametrize("wfmt,qmin,qmax,alpha", [("ternary", -1, 1, 0.016),
                                                  ("i8", -128, 127, 2e-4)])
def test_sr_update_large_sampled(lib, wfmt, qmin, qmax, alpha):
    """16M weights: several 4096-weight tiles per block of the persistent
    grid.  Bit-exact on a sample (every weight of the first and last tiles and
    of 150k random positions), counters against the host's own count."""
    d_out, d_in = 4096, 4096
    n = d_out * d_in
    log(f"sr_update large {wfmt} {d_out}x{d_in}")
    q = _weights(d_out, d_in, wfmt, qmin, qmax, 4096, 7)
    g = draws((d_out, d_in), 1.0, 11, wfmt == "ternary")
    flat = g.reshape(-1)
    flat[3::7919] *= 1e4
    flat[17::100_003] = np.nan
    flat[29::100_019] = np.inf
    n_nonfinite = int(np.count_nonzero(~np.isfinite(flat)))
    lr = 3e-4 if wfmt == "ternary" else 1e-3
    w = make_weight(d_out, d_in, wfmt, qmin, qmax, alpha, tensor_id=6)
    Wq = weight_codes_dev(q, wfmt)
    counters = torch.zeros((2,), dtype=torch.int64, device=DEV)
    dqt.dqt_sr_update(w, Wq, torch.from_numpy(g).to(DEV), lr, 77, 5, counters)
    got = weight_codes_host(Wq, wfmt, d_in).ravel()
    rng = np.random.default_rng(5)
    idx = np.unique(np.concatenate([np.arange(4096), np.arange(n - 4096, n),
                                    rng.choice(n, 150_000, replace=False)])).astype(np.uint64)
    ii = idx.astype(np.int64)
    want, _, _ = O.sr_update(q.ravel()[ii], flat[ii], lr, alpha, qmin, qmax, 77, 5, 6, idx=idx)
    assert np.array_equal(got[ii], want)
    c = counters.cpu().numpy()
    assert int(c[0]) == int(np.count_nonzero(got != q.ravel()))
    assert int(c[1]) == n_nonfinite


# ------------------------------------------------------- full train step

def _full_step(wl, li, M=None, sample_rows=None, sample_cols=None):
    """One linear of a workload at its full shape: fwd + bwd + SR on the GPU,
    checked against the oracle (all outputs, or sampled rows/cols)."""
    lin = wl.linears[li]
    M = wl.M if M is None else M
    log(f"full step {wl.name}/{lin.name} M={M} d_in={lin.d_in} d_out={lin.d_out}")
    W0, qdraw = W.weight_draws(wl, li)
    if wl.init == "uniform":
        q, alpha = qdraw, np.float32(O.absmean(W0))
    else:
        q, alpha = O.absmean_init(W0, wl.qmin, wl.qmax)
    w = make_weight(lin.d_out, lin.d_in, wl.wfmt, wl.qmin, wl.qmax, alpha, tensor_id=li)
    Wq = weight_codes_dev(q, wl.wfmt)
    X_dev, X_seen = to_dev(W.input_draw(wl, lin.input, M), wl.x_dtype)
    dY_dev, dY_seen = to_dev(W.grad_draw(wl, li, M), wl.dy_dtype)
    Xq, xdq, Y = run_fwd(w, Wq, X_dev, wl.act, wl.y_out)
    dX, dW = run_bwd(w, Wq, Xq, wl.act, xdq, dY_dev, wl.xt, wl.dx_out)
    torch.cuda.synchronize()
    # SR parity on the oracle's own gradient values (no GPU value feeds the oracle)
    want_q, want_d = O.act_quant(X_seen, wl.act)
    assert np.array_equal(Xq.cpu().numpy().view(np.uint8), want_q.view(np.uint8))
    assert np.array_equal(xdq.cpu().numpy(), want_d)
    rows = np.arange(M) if sample_rows is None else sample_rows
    Y_ref, acc = O.linear_fwd(want_q[rows], want_d[rows], wl.act, q, alpha, wl.y_out)
    got_Y = Y.float().cpu().numpy()[rows]
    if wl.act == "i8":
        assert np.array_equal(got_Y, Y_ref)
    else:
        a = np.abs(O.act_values(want_q[rows], wl.act)) @ np.abs(q.astype(np.float64)).T
        f = (want_d[rows] * alpha).astype(np.float64)[:, None]
        ok, nbad, emax = gemm_close(got_Y, acc * f, a * f, bf16_out=(wl.y_out == "bf16"))
        assert ok, ("Y", nbad, emax)
    qf = q.astype(np.float64)
    dX64 = float(alpha) * (dY_seen[rows].astype(np.float64) @ qf)
    bx = float(alpha) * O.gemm_abs_bound(dY_seen[rows], qf)
    ok, nbad, emax = gemm_close(dX.float().cpu().numpy()[rows], dX64, bx,
                                bf16_out=(wl.dx_out == "bf16"))
    assert ok, ("dX", nbad, emax)
    cols = np.arange(lin.d_in) if sample_cols is None else sample_cols
    xt_vals = O.act_dequant(want_q[:, cols], want_d, wl.act, wl.xt)
    dW64 = dY_seen.astype(np.float64).T @ xt_vals
    bw = O.gemm_abs_bound(dY_seen.T, xt_vals)
    ok, nbad, emax = gemm_close(dW.cpu().numpy()[:, cols], dW64, bw)
    assert ok, ("dW", nbad, emax)
    # SR: the oracle's fp32 dW on the checked columns (zero elsewhere, where
    # nothing may move) drives both sides
    g = dW64.astype(np.float32)
    g_full = np.zeros((lin.d_out, lin.d_in), np.float32)
    g_full[:, cols] = g
    dW_dev = torch.from_numpy(g_full).to(DEV)
    counters = torch.zeros((2,), dtype=torch.int64, device=DEV)
    dqt.dqt_sr_update(w, Wq, dW_dev, wl.lr, wl.seed, wl.sr_step, counters)
    got_q = weight_codes_host(Wq, wl.wfmt, lin.d_in)
    idx = (np.arange(lin.d_out)[:, None] * lin.d_in + cols[None, :]).ravel().astype(np.uint64)
    want_new, n_changed, _ = O.sr_update(q[:, cols].ravel(), g.ravel(), wl.lr, alpha, wl.qmin,
                                         wl.qmax, wl.seed, wl.sr_step, li, idx=idx)
    assert np.array_equal(got_q[:, cols].ravel(), want_new)
    untouched = np.ones(lin.d_in, bool)
    untouched[cols] = False
    assert np.array_equal(got_q[:, untouched], q[:, untouched])
    assert int(counters[0].item()) == n_changed
    log(f"  ok; SR changed {n_changed} of {q.size} weights")


def test_full_step_single_256(lib):
    _full_step(W.WORKLOADS["single_256"], 0)


@pytest.mark.parametrize("li", range(7))
def test_full_step_llama_h768(lib, li):
    _full_step(W.WORKLOADS["llama_h768"], li)


@pytest.mark.parametrize("wname", ["llama_h2048", "llama_h4096", "llama_h2048_int4"])
@pytest.mark.parametrize("li", [0, 4, 6])
def test_full_step_large_sampled(lib, wname, li):
    wl = W.WORKLOADS[wname]
    lin = wl.linears[li]
    rng = np.random.default_rng(li)
    rows = np.sort(rng.choice(wl.M, 96, replace=False))
    cols = np.sort(rng.choice(lin.d_in, 64, replace=False))
    _full_step(wl, li, sample_rows=rows, sample_cols=cols)
