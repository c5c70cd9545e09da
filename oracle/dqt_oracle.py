"""CPU oracle for the DQT linear train step (Direct Quantized Training,
arXiv 2412.04787).

TEST INFRASTRUCTURE, NOT PRODUCT CODE.  Only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import or call anything in ``oracle/``.  The HIP library never calls it, and
this module imports nothing from the HIP package: the two share no code,
tables or constants.

Everything here is plain numpy, written for readability, not speed.  Exact
integer work is done in int64 (or in float64 where every partial sum is an
integer far below 2**53, which makes float64 exact).  Real-valued sums are
float64.  Where the method itself fixes an fp32 operation (the per-token
activation scale, the SR step size, the update delta), the oracle performs that
same single fp32 operation with numpy ``float32`` scalars/arrays, which round
to nearest-even with no fused multiply-add.

Paper map (section / equation of the DQT paper):
  * Sec. 3.1, Eq. 1 ........ stochastic rounding SR(x)           -> sr_update
  * Sec. 3.2, Eq. 2-4 ...... AbsMean init quantisation            -> absmean_init
  * Sec. 3.2 (BitNet 8-bit activations, forward with W~) ......... -> act_quant,
                                                                      linear_fwd
  * Sec. 3.2 (backprop to the gradient of W~, no STE on weights) -> linear_bwd
  * Sec. 3.2, Eq. 5 ........ direct update W^ = SR(W')            -> sr_update
  * Sec. 5.2 ............... fraction of weights changed per step -> n_changed
  * Sec. 4.1 (AdamW modified with SR; reading R11) ............... -> adamw_sr_update
  * Sec. 5 (rounding without SR; forcing the smallest 20 %; R12) -> update_variant
  * Sec. 3.2 inputs of the linears after the block's RMSNorm (R13) -> rmsnorm_act_quant

Readings of points the paper leaves open:
  R1  SR acts in grid units: with W~ = q * alpha (alpha = 1/s, Eq. 3) and
      W' = W~ - lr * grad, the updated code is SR(W' / alpha).  This is what
      the worked example of Sec. 5 (a value -1 + 0.02 goes to 0 with
      probability 2%) requires.
  R2  Ternary grid is {-1, 0, 1}; n-bit grid is [qmin, qmax] given by the
      caller (Eq. 3 gives -2^(n-1) .. 2^(n-1)-1; 8-bit configs may use
      -127..127).
  R3  alpha is fixed at initialisation and never recomputed (Eq. 2-4 are
      skipped during training, Sec. 3.2).
  R4  Activations: per-token absmax to int8 with the constant 127, eps 1e-5
      and clamp to [-128, 127]; or to OCP e4m3 with the constant 448.
  R5  The backward treats activation quantisation as pass-through and uses
      the dequantised activation X~ (in the environment dtype) for dW.
  R6  The optimiser target is the plain step W' = W~ - lr * grad.
  R7  Random bits: Philox4x32-10 with the counter layout of ``rng_u32``;
      Bernoulli(p) is realised as U < ceil(p * 2**32) with U uniform on
      [0, 2**32).
  R8  A non-finite gradient entry leaves its weight unchanged and is counted.
  R11 AdamW with SR (Sec. 4.1 names AdamW, modified to round stochastically,
      and gives no further detail): the target W' is the AdamW step with
      decoupled weight decay and bias correction,
        m <- b1 m + (1 - b1) g,  v <- b2 v + (1 - b2) g^2,
        W' = W~ (1 - lr wd) - lr * mhat / (sqrt(vhat) + eps),
        mhat = m / (1 - b1^t),  vhat = v / (1 - b2^t),
      taken in grid units (R1) and rounded by Eq. 1 with the draws of R7;
      m and v are fp32.  The element-wise arithmetic is fixed in fp32 (see
      ``adamw_sr_update``); a non-finite gradient entry, or a NaN step, leaves
      the weight, m and v unchanged and is counted.
  R12 Analysis variants of Sec. 5 (with alpha fixed, R3): the deterministic
      control rounds x = q + delta to the nearest grid value (ties to even)
      instead of stochastically; for the interventions on the smallest
      fraction of a step's updates, updates are ranked per tensor by |delta| (fp32 bit patterns as unsigned
      integers, non-finite gradients ranked last): with k = floor(frac n) and
      tau the k-th smallest key, the bottom set is {key <= tau} (ties at tau
      may enlarge it).  Force-to-remain keeps the bottom codes; force-to-
      update rounds x away from q (ceil for delta > 0, floor for delta < 0),
      then clips; every other element takes the plain SR update.
  R13 RMSNorm before the activation quantisation (the LLaMA block's norm,
      not specified by the paper): y = x / sqrt(mean(x^2) + eps) * gamma in
      fp32, the sum of squares in the fixed order of ``rms_sum_squares``
      (64 lane sums over chunks of 8 elements, then a butterfly), each
      operation one correctly rounded fp32 operation; y then goes through
      ``act_quant``.
  R14 The deterministic control of Sec. 5.1 read literally: absmax
      quantisation of the updated real-valued matrix W' = W~ - lr g with a
      new per-tensor scale alpha' = max|W'| / qmax each step (see
      ``absmax_requant``); a non-finite g counts as 0 and is counted.
"""

from __future__ import annotations

import numpy as np

# ---------------------------------------------------------------------------
# Number formats.  Each converter is written from the format's definition:
# enumerate / bracket the representable values and pick the nearest one, ties
# to the value whose last significand bit is 0.
# ---------------------------------------------------------------------------


def bf16_round(x) -> np.ndarray:
    """fp32 -> bf16 bit pattern (uint16), round to nearest, ties to even.

    bf16 keeps the sign, the 8 exponent bits and the top 7 fraction bits of an
    fp32 value.  For a finite input the two candidates are the value with the
    low 16 bits cleared (toward zero) and the next bf16 value away from zero;
    the nearer one wins, and on a tie the one with an even last bit.
    Only finite inputs are expected here.
    """
    x = np.asarray(x, dtype=np.float32)
    bits = x.view(np.uint32).astype(np.uint64)
    toward_zero = (bits >> np.uint64(16))  # bf16 pattern, magnitude rounded down
    away = toward_zero + np.uint64(1)      # next magnitude up (carries into exp)
    v_tz = (toward_zero << np.uint64(16)).astype(np.uint32).view(np.float32).astype(np.float64)
    v_aw = (away << np.uint64(16)).astype(np.uint32).view(np.float32).astype(np.float64)
    xv = x.astype(np.float64)
    d_tz = np.abs(xv - v_tz)
    d_aw = np.abs(v_aw - xv)
    pick_away = (d_aw < d_tz) | ((d_aw == d_tz) & ((toward_zero & np.uint64(1)) == np.uint64(1)))
    out = np.where(pick_away, away, toward_zero)
    return out.astype(np.uint16)


def bf16_to_f32(b) -> np.ndarray:
    """bf16 bit pattern (uint16) -> fp32 value (exact)."""
    b = np.asarray(b, dtype=np.uint16).astype(np.uint32)
    return (b << np.uint32(16)).view(np.float32)


def _e4m3_table() -> np.ndarray:
    """Value of every OCP E4M3 ('fn') code, NaN for the two NaN codes.

    Layout: 1 sign bit, 4 exponent bits (bias 7), 3 fraction bits.
    exponent 0 is subnormal: value = frac/8 * 2**(1-7).
    S.1111.111 is NaN; there are no infinities, so the largest finite
    magnitude is 1.75 * 2**8 = 448.
    """
    vals = np.empty(256, dtype=np.float64)
    for code in range(256):
        sign = -1.0 if code & 0x80 else 1.0
        e = (code >> 3) & 0xF
        f = code & 0x7
        if e == 0xF and f == 0x7:
            vals[code] = np.nan
        elif e == 0:
            vals[code] = sign * (f / 8.0) * 2.0 ** (1 - 7)
        else:
            vals[code] = sign * (1.0 + f / 8.0) * 2.0 ** (e - 7)
    return vals


E4M3_VALUES = _e4m3_table()
E4M3_MAX = 448.0


def e4m3_encode(x) -> np.ndarray:
    """fp32 -> OCP E4M3 code (uint8): round to nearest, ties to even fraction,
    saturating to +-448.  The sign bit is kept (so -0.0 -> 0x80).

    Brute force: for each magnitude, find the nearest of the 127 non-negative
    finite codes (0x00..0x7E, increasing in value), ties to the even code.
    """
    x = np.asarray(x, dtype=np.float32).astype(np.float64)
    sign = np.signbit(x)
    a = np.minimum(np.abs(x), E4M3_MAX)
    pos = E4M3_VALUES[:0x7F]                        # 0x00 .. 0x7E, sorted
    hi = np.searchsorted(pos, a, side="left")       # first code with value >= a
    hi = np.clip(hi, 0, 0x7E)
    lo = np.clip(hi - 1, 0, 0x7E)
    d_lo = np.abs(a - pos[lo])
    d_hi = np.abs(pos[hi] - a)
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & (hi % 2 == 0))
    code = np.where(pick_hi, hi, lo).astype(np.uint8)
    return np.where(sign, code | np.uint8(0x80), code).astype(np.uint8)


def e4m3_decode(code) -> np.ndarray:
    """OCP E4M3 code -> float64 value (exact)."""
    return E4M3_VALUES[np.asarray(code, dtype=np.uint8)]


# ---------------------------------------------------------------------------
# Weight storage: packed ternary codes.
# ---------------------------------------------------------------------------


def pack_ternary(q: np.ndarray) -> np.ndarray:
    """int8 ternary [d_out, d_in] -> packed uint8 [d_out, d_in/4].

    Weight (n, k) is stored as the 2-bit code q + 1 in byte k // 4 of row n,
    at bit offset 2 * (k % 4).
    """
    q = np.asarray(q)
    d_out, d_in = q.shape
    assert d_in % 4 == 0
    codes = (q.astype(np.int64) + 1).reshape(d_out, d_in // 4, 4)
    assert codes.min() >= 0 and codes.max() <= 2
    packed = np.zeros((d_out, d_in // 4), dtype=np.int64)
    for j in range(4):
        packed |= codes[:, :, j] << (2 * j)
    return packed.astype(np.uint8)


def unpack_ternary(packed: np.ndarray, d_in: int) -> np.ndarray:
    """Inverse of pack_ternary: packed uint8 [d_out, d_in/4] -> int8 [d_out, d_in]."""
    packed = np.asarray(packed, dtype=np.uint8).astype(np.int64)
    d_out = packed.shape[0]
    out = np.empty((d_out, d_in // 4, 4), dtype=np.int64)
    for j in range(4):
        out[:, :, j] = ((packed >> (2 * j)) & 3) - 1
    return out.reshape(d_out, d_in).astype(np.int8)


# ---------------------------------------------------------------------------
# Sec. 3.2, Eq. 2-4: AbsMean initial quantisation (one-time, not per step).
# ---------------------------------------------------------------------------


def pack_int4(q: np.ndarray) -> np.ndarray:
    """Codes in [-8, 7] [rows, cols] -> 4-bit two's-complement nibbles, two
    per byte (weight k in the low nibble of byte k // 2 when k is even)."""
    q = np.asarray(q).astype(np.int64)
    assert q.ndim == 2 and q.shape[1] % 2 == 0 and q.min() >= -8 and q.max() <= 7
    nib = (q & 0xF).astype(np.uint8)
    return (nib[:, 0::2] | (nib[:, 1::2] << 4)).astype(np.uint8)


def unpack_int4(packed: np.ndarray, d_in: int) -> np.ndarray:
    p = np.asarray(packed, dtype=np.uint8)
    lo = (p & 0xF).astype(np.int64)
    hi = (p >> 4).astype(np.int64)
    out = np.empty((p.shape[0], d_in), dtype=np.int64)
    out[:, 0::2] = np.where(lo >= 8, lo - 16, lo)
    out[:, 1::2] = np.where(hi >= 8, hi - 16, hi)
    return out.astype(np.int8)


def pack_int3(q: np.ndarray) -> np.ndarray:
    """Codes in [-4, 3] [rows, cols] -> 3-bit two's-complement fields, 8 per
    3 bytes: the group of weights 8g .. 8g + 7 is the 24-bit number
    sum_j (q_(8g+j) mod 8) 2^(3j), stored little-endian in bytes 3g .. 3g + 2."""
    q = np.asarray(q).astype(np.int64)
    assert q.ndim == 2 and q.shape[1] % 8 == 0 and q.min() >= -4 and q.max() <= 3
    rows, cols = q.shape
    fields = (q & 7).reshape(rows, cols // 8, 8)
    word = np.zeros((rows, cols // 8), dtype=np.int64)
    for j in range(8):
        word += fields[:, :, j] << (3 * j)
    out = np.empty((rows, cols // 8, 3), dtype=np.uint8)
    for b in range(3):
        out[:, :, b] = (word >> (8 * b)) & 0xFF
    return out.reshape(rows, 3 * cols // 8)


def unpack_int3(packed: np.ndarray, d_in: int) -> np.ndarray:
    p = np.asarray(packed, dtype=np.uint8).reshape(-1, d_in // 8, 3).astype(np.int64)
    word = p[:, :, 0] | (p[:, :, 1] << 8) | (p[:, :, 2] << 16)
    out = np.empty((p.shape[0], d_in // 8, 8), dtype=np.int64)
    for j in range(8):
        f = (word >> (3 * j)) & 7
        out[:, :, j] = np.where(f >= 4, f - 8, f)
    return out.reshape(p.shape[0], d_in).astype(np.int8)


def absmean(W) -> float:
    """Eq. 2: the mean absolute value over every element of the tensor (fp64)."""
    W = np.asarray(W, dtype=np.float64)
    return float(np.mean(np.abs(W)))


def absmean_init(W0, qmin: int, qmax: int):
    """Eq. 3-4: s = Q_p / AbsMean(W);  q = Clip(Round(W * s), Q_n, Q_p).

    Returns the integer codes q (int8) and the dequantisation scale
    alpha = 1/s = AbsMean(W) / Q_p rounded once to fp32, so that the quantised
    weight of Eq. 4 is q * alpha.  Round() is half-to-even (``np.rint``).
    The products W * s are formed in fp64.
    """
    am = absmean(W0)
    s = qmax / am
    q = np.clip(np.rint(np.asarray(W0, dtype=np.float64) * s), qmin, qmax)
    alpha = np.float32(am / qmax)
    return q.astype(np.int8), alpha


# ---------------------------------------------------------------------------
# Sec. 3.2: 8-bit activation quantisation (BitNet convention, reading R4).
# ---------------------------------------------------------------------------

ACT_EPS = np.float32(1e-5)


def act_quant(X, kind: str):
    """Per-token absmax quantisation of X [M, K] (fp32 values).

    g_m   = max(max_k |x_mk|, 1e-5)                 (fp32)
    int8: inv_m = 127 / g_m ; Xq = clamp(rint(x * inv_m), -128, 127)
          d_m   = g_m / 127
    e4m3: inv_m = 448 / g_m ; Xq = e4m3(x * inv_m) ; d_m = g_m / 448
    Each division and the product x * inv_m is one correctly rounded fp32
    operation.  Returns (Xq, d) with Xq int8 or uint8 (e4m3 codes) and d fp32.
    """
    X = np.asarray(X, dtype=np.float32)
    M = X.shape[0]
    g = np.empty(M, dtype=np.float32)
    for m in range(M):
        row_max = np.float32(np.max(np.abs(X[m]))) if X.shape[1] else np.float32(0)
        g[m] = max(row_max, ACT_EPS)
    if kind == "i8":
        qmax_act = np.float32(127.0)
    elif kind == "e4m3":
        qmax_act = np.float32(448.0)
    else:
        raise ValueError(kind)
    inv = (qmax_act / g).astype(np.float32)            # fp32 division
    d = (g / qmax_act).astype(np.float32)              # fp32 division
    scaled = (X * inv[:, None]).astype(np.float32)     # one fp32 multiply
    if kind == "i8":
        Xq = np.clip(np.rint(scaled), -128, 127).astype(np.int8)
    else:
        Xq = e4m3_encode(scaled)
    return Xq, d


# ---------------------------------------------------------------------------
# Next row: RMSNorm followed by the activation quantisation (reading R13).
# In a LLaMA block the inputs of the q/k/v and gate/up linears are RMSNorm
# outputs; the paper quantises those inputs to 8 bits (Sec. 3.2).
# ---------------------------------------------------------------------------

RMS_LANES = 64      # lane partial sums of the sum of squares
RMS_CHUNK = 8       # consecutive elements per chunk


def rms_sum_squares(X) -> np.ndarray:
    """Sum of squares of each row of X [M, K] (fp32 values) in the fixed
    fp32 order of reading R13: every square is one fp32 multiply; lane l of
    64 adds, in order, the squares of the chunks l, l + 64, l + 128, ... of
    8 consecutive elements (each chunk's elements in order) into a sum that
    starts at 0; then, for d = 32, 16, 8, 4, 2, 1, every lane sum becomes
    fl(s_l + s_(l xor d)).  Returns the fp32 sums [M]."""
    X = np.asarray(X, dtype=np.float32)
    M, K = X.shape
    sq = (X * X).astype(np.float32)
    nchunk = K // RMS_CHUNK
    lanes = np.zeros((M, RMS_LANES), dtype=np.float32)
    # position p of lane l's sequence is element RMS_CHUNK * (l + 64 (p // 8)) + p % 8
    per_lane = (nchunk + RMS_LANES - 1) // RMS_LANES * RMS_CHUNK
    for p in range(per_lane):
        chunk = np.arange(RMS_LANES) + RMS_LANES * (p // RMS_CHUNK)
        elem = RMS_CHUNK * chunk + p % RMS_CHUNK
        live = chunk < nchunk
        add = np.where(live[None, :], sq[:, np.minimum(elem, K - 1)], np.float32(0))
        lanes = np.where(live[None, :], (lanes + add).astype(np.float32), lanes)
    idx = np.arange(RMS_LANES)
    for d in (32, 16, 8, 4, 2, 1):
        lanes = (lanes + lanes[:, idx ^ d]).astype(np.float32)
    return lanes[:, 0].copy()


def rmsnorm(X, gamma, eps):
    """RMSNorm of each row (R13): r_m = fl(1 / fl(sqrt(fl(fl(s_m / K) +
    eps)))) with s_m = rms_sum_squares, then y_mk = fl(fl(x_mk r_m) gamma_k);
    every operation one correctly rounded fp32 operation.  Returns (y, r)."""
    X = np.asarray(X, dtype=np.float32)
    K = X.shape[1]
    s = rms_sum_squares(X)
    mean = (s / np.float32(K)).astype(np.float32)
    v = (mean + np.float32(eps)).astype(np.float32)
    with np.errstate(divide="ignore"):
        r = (np.float32(1.0) / np.sqrt(v).astype(np.float32)).astype(np.float32)
    y = ((X * r[:, None]).astype(np.float32) * np.asarray(gamma, dtype=np.float32)[None, :])
    return y.astype(np.float32), r


def rmsnorm_act_quant(X, gamma, eps, kind: str):
    """RMSNorm, then the per-token quantisation of act_quant applied to its
    output.  Returns (Xq, d, r, y)."""
    y, r = rmsnorm(X, gamma, eps)
    Xq, d = act_quant(y, kind)
    return Xq, d, r, y


def act_values(Xq, kind: str) -> np.ndarray:
    """Integer / e4m3 activation codes as exact float64 values."""
    if kind == "i8":
        return np.asarray(Xq, dtype=np.int8).astype(np.float64)
    return e4m3_decode(Xq)


def act_dequant(Xq, d, kind: str, xt: str) -> np.ndarray:
    """X~[m, k] = Xq[m, k] * d_m as one fp32 multiply, then cast to the
    environment dtype xt ('f32' or 'bf16').  Returned as float64 values."""
    v = act_values(Xq, kind).astype(np.float32)
    xt32 = (v * np.asarray(d, dtype=np.float32)[:, None]).astype(np.float32)
    if xt == "f32":
        return xt32.astype(np.float64)
    if xt == "bf16":
        return bf16_to_f32(bf16_round(xt32)).astype(np.float64)
    raise ValueError(xt)


def cast_out(y32: np.ndarray, out: str) -> np.ndarray:
    """Cast fp32 results to the output dtype; returns fp32 (bf16 values widened)."""
    y32 = np.asarray(y32, dtype=np.float32)
    if out == "f32":
        return y32
    if out == "bf16":
        return bf16_to_f32(bf16_round(y32))
    raise ValueError(out)


# ---------------------------------------------------------------------------
# Sec. 3.2: forward with the quantised weights and quantised activations.
# ---------------------------------------------------------------------------


def linear_fwd(Xq, d, kind: str, q, alpha, out: str = "f32"):
    """Y = X~ W~^T with X~ = Xq * d_m and W~ = q * alpha (nn.Linear layout:
    q is [d_out, d_in], Y is [M, d_out]).

    acc[m, n] = sum_k Xq[m, k] * q[n, k] is formed exactly (every product and
    partial sum is an integer, or for e4m3 a multiple of 2**-9, well inside
    float64's 53-bit significand, so a float64 matmul is exact in any order).
    Then f_m = fl32(d_m * alpha) and y = fl32(fl32(acc) * f_m), cast to `out`.
    """
    a = act_values(Xq, kind)
    w = np.asarray(q, dtype=np.int8).astype(np.float64)
    acc = a @ w.T
    if kind == "i8":
        assert np.all(np.abs(acc) < 2.0 ** 31)
    f = (np.asarray(d, dtype=np.float32) * np.float32(alpha)).astype(np.float32)
    y32 = (acc.astype(np.float32) * f[:, None]).astype(np.float32)
    return cast_out(y32, out), acc


# ---------------------------------------------------------------------------
# Sec. 3.2: backward.  No straight-through estimator on the weights: the
# gradient is taken with respect to W~ itself; activation quantisation is
# treated as pass-through (reading R5).
# ---------------------------------------------------------------------------


def linear_bwd(dY, q, alpha, Xq, d, kind: str, xt: str, dx_out: str = "f32"):
    """dX = dY W~ = alpha * (dY @ q)          [M, d_in]
    dW = dY^T X~                              [d_out, d_in], fp32

    Sums in float64; dX is cast to `dx_out`, dW rounded once to fp32.
    Returns (dX, dW, dX64, dW64) where the *64 arrays are the unrounded sums.
    """
    dY = np.asarray(dY, dtype=np.float64)
    w = np.asarray(q, dtype=np.int8).astype(np.float64)
    xt_vals = act_dequant(Xq, d, kind, xt)
    dX64 = float(alpha) * (dY @ w)
    dW64 = dY.T @ xt_vals
    dX = cast_out(dX64.astype(np.float32), dx_out)
    dW = dW64.astype(np.float32)
    return dX, dW, dX64, dW64


# ---------------------------------------------------------------------------
# Random bits: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random
# numbers: as easy as 1, 2, 3", SC'11).  Counter-based: the output depends
# only on (counter, key), so there is no state to carry between steps.
# ---------------------------------------------------------------------------

PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9   # key schedule increments (golden ratio, sqrt(3)-1)
PHILOX_W1 = 0xBB67AE85
_MASK32 = np.uint64(0xFFFFFFFF)


def philox4x32_10(ctr, key):
    """Philox4x32 with 10 rounds, vectorised over numpy arrays.

    ctr: 4 arrays (or scalars) of uint32 words c0..c3;  key: 2 words k0, k1.
    One round: multiply c0 by M0 and c2 by M1 into 64-bit products, then
      (c0, c1, c2, c3) <- (hi(M1*c2) ^ c1 ^ k0, lo(M1*c2),
                           hi(M0*c0) ^ c3 ^ k1, lo(M0*c0));
    between rounds the key is bumped by (W0, W1) modulo 2**32.
    """
    c = [np.asarray(v, dtype=np.uint64) & _MASK32 for v in ctr]
    k0 = np.asarray(key[0], dtype=np.uint64) & _MASK32
    k1 = np.asarray(key[1], dtype=np.uint64) & _MASK32
    m0 = np.uint64(PHILOX_M0)
    m1 = np.uint64(PHILOX_M1)
    for rnd in range(10):
        if rnd > 0:
            k0 = (k0 + np.uint64(PHILOX_W0)) & _MASK32
            k1 = (k1 + np.uint64(PHILOX_W1)) & _MASK32
        p0 = c[0] * m0
        p1 = c[2] * m1
        c = [
            ((p1 >> np.uint64(32)) ^ c[1] ^ k0) & _MASK32,
            p1 & _MASK32,
            ((p0 >> np.uint64(32)) ^ c[3] ^ k1) & _MASK32,
            p0 & _MASK32,
        ]
    return [v.astype(np.uint32) for v in c]


def _half16(seed: int, step: int, tensor_id: int, idx: np.ndarray, dom: int) -> np.ndarray:
    """16-bit draw for each element index in idx from stream `dom` (0 or 1).

    Counter = (lo32(i >> 3), hi32(i >> 3) | dom << 31, step, tensor_id),
    key = (lo32(seed), hi32(seed)).  One Philox call serves 8 consecutive
    elements: element i takes output word (i & 7) >> 1, its low 16 bits when
    i is even and its high 16 bits when i is odd.
    """
    idx = np.asarray(idx, dtype=np.uint64)
    # one Philox call per distinct block of 8 elements
    blk, inv = np.unique(idx >> np.uint64(3), return_inverse=True)
    inv = inv.ravel()
    c0 = blk & _MASK32
    c1 = (blk >> np.uint64(32)) | np.uint64(dom << 31)
    c2 = np.full_like(blk, np.uint64(step & 0xFFFFFFFF))
    c3 = np.full_like(blk, np.uint64(tensor_id & 0xFFFFFFFF))
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    words = philox4x32_10((c0, c1, c2, c3), (seed & 0xFFFFFFFF, seed >> 32))
    words = np.stack(words).astype(np.uint64)           # [4, n_blocks]
    w_sel = ((idx & np.uint64(7)) >> np.uint64(1)).astype(np.int64)
    word = words[w_sel, inv]
    shift = (idx & np.uint64(1)) * np.uint64(16)
    return ((word >> shift) & np.uint64(0xFFFF)).astype(np.uint32)


def rng_u32(seed: int, step: int, tensor_id: int, idx) -> np.ndarray:
    """U(i) = (P16(i) << 16) | S16(i): a 32-bit uniform draw per element,
    P16 from stream 0 and S16 from stream 1 (reading R7)."""
    idx = np.atleast_1d(np.asarray(idx, dtype=np.uint64))
    p = _half16(seed, step, tensor_id, idx, 0)
    s = _half16(seed, step, tensor_id, idx, 1)
    return ((p.astype(np.uint64) << np.uint64(16)) | s.astype(np.uint64)).astype(np.uint32)


# ---------------------------------------------------------------------------
# Sec. 3.1 Eq. 1 and Sec. 3.2 Eq. 5: direct stochastic-rounding update.
# ---------------------------------------------------------------------------


def sr_step_size(lr, alpha) -> np.float32:
    """c = fl32(lr / alpha): the learning rate expressed in grid units."""
    return np.float32(np.float32(lr) / np.float32(alpha))


def sr_update(q, g, lr, alpha, qmin: int, qmax: int, seed: int, step: int,
              tensor_id: int, idx=None):
    """Eq. 5 in grid units (reading R1): q^ = Clip(SR(q + delta), qmin, qmax)
    with delta = -fl32(c * g) and c = fl32(lr / alpha).

    Eq. 1: with x = q + delta, SR(x) is floor(x) with probability
    ceil(x) - x, else ceil(x).  q is an integer, so floor/ceil of x are q plus
    floor/ceil of delta, and the probabilities are formed from delta alone
    (which keeps them exact):
      delta >= 0:  x rounds up   to q + floor(delta) + 1  w.p. delta - floor(delta)
      delta <  0:  x rounds down to q + ceil(delta)  - 1  w.p. ceil(delta) - delta
    A Bernoulli(p) event is U < ceil(p * 2**32) with U = rng_u32(...) (R7).

    q, g: flat arrays of the same length.  idx: flat element indices (default
    0..n-1) used to key the random draws.  Returns (q_new int64, n_changed,
    n_nonfinite).
    """
    q = np.asarray(q).astype(np.int64).ravel()
    g = np.asarray(g, dtype=np.float32).ravel()
    if idx is None:
        idx = np.arange(q.size, dtype=np.uint64)
    c = sr_step_size(lr, alpha)
    finite = np.isfinite(g)
    with np.errstate(over="ignore", invalid="ignore"):
        delta32 = -(c * np.where(finite, g, np.float32(0))).astype(np.float32)
    new = _sr_round(q, delta32, qmin, qmax, seed, step, tensor_id, idx)
    new = np.where(finite, new, q)
    n_changed = int(np.count_nonzero(new != q))
    n_nonfinite = int(np.count_nonzero(~finite))
    return new, n_changed, n_nonfinite


def _sr_round(q, delta32, qmin: int, qmax: int, seed: int, step: int, tensor_id: int, idx):
    """Eq. 1 on x = q + delta (grid units), clipped to [qmin, qmax]; delta
    is an fp32 array (an infinite delta saturates).  Element idx[i] keys the
    draw of element i (R7)."""
    delta = np.asarray(delta32, dtype=np.float32).astype(np.float64)
    U = rng_u32(seed, step, tensor_id, idx).astype(np.float64)
    big = ~np.isfinite(delta)                 # the step overflowed fp32
    d_ok = np.where(big, 0.0, delta)
    up_side = d_ok >= 0
    fl = np.floor(d_ok)
    ce = np.ceil(d_ok)
    p = np.where(up_side, d_ok - fl, ce - d_ok)          # exact in float64
    thresh = np.ceil(p * 2.0 ** 32)
    event = U < thresh
    base = np.where(up_side, fl, ce)
    move = base + np.where(event, np.where(up_side, 1.0, -1.0), 0.0)
    x_new = q.astype(np.float64) + move
    x_new = np.where(big, np.where(delta > 0, np.inf, -np.inf), x_new)
    return np.clip(x_new, qmin, qmax).astype(np.int64)


# ---------------------------------------------------------------------------
# Next row: AdamW with SR (Sec. 4.1; reading R11).
# ---------------------------------------------------------------------------


def pow_by_squaring(b: float, t: int) -> float:
    """b**t in float64 by binary exponentiation (t >= 0): square the base
    and multiply it in for every set bit of t, low bit first."""
    r, x = 1.0, float(b)
    while t > 0:
        if t & 1:
            r = r * x
        x = x * x
        t >>= 1
    return r


def adamw_scalars(lr, alpha, beta1, beta2, eps, weight_decay, t: int) -> dict:
    """Per-call constants, each formed in float64 from the fp32 inputs and
    rounded once to fp32:
      b1, b2, eps        the inputs;
      ob1 = 1 - b1, ob2 = 1 - b2;
      k2 = 1 / sqrt(1 - b2^t)          (sqrt(vhat) = sqrt(v) * k2);
      cu = lr / (alpha * (1 - b1^t))   (the bias-corrected step in grid units);
      cd = lr * weight_decay           (the decoupled decay per step)."""
    f = lambda x: np.float32(np.float64(x))
    b1 = np.float64(np.float32(beta1))
    b2 = np.float64(np.float32(beta2))
    lr64 = np.float64(np.float32(lr))
    a64 = np.float64(np.float32(alpha))
    wd64 = np.float64(np.float32(weight_decay))
    return dict(b1=f(b1), b2=f(b2), eps=np.float32(eps), ob1=f(1.0 - b1), ob2=f(1.0 - b2),
                k2=f(1.0 / np.sqrt(1.0 - pow_by_squaring(b2, t))),
                cu=f(lr64 / (a64 * (1.0 - pow_by_squaring(b1, t)))),
                cd=f(lr64 * wd64))


def adamw_target(q, g, m, v, k: dict):
    """One AdamW step in grid units, element-wise in fp32 (round to nearest
    even after every operation, no fused multiply-add; sqrt and division
    correctly rounded):
      m' = b1 m + ob1 g
      v' = b2 v + (ob2 g) g
      den = sqrt(v') k2 + eps
      u = m' / den
      delta = -(cu u + cd q)
    Returns (delta, m', v') as fp32 arrays: x = q + delta is W' / alpha."""
    f32 = np.float32
    q = np.asarray(q).astype(np.int64).astype(f32)
    g = np.asarray(g, dtype=f32)
    m = np.asarray(m, dtype=f32)
    v = np.asarray(v, dtype=f32)
    with np.errstate(over="ignore", invalid="ignore", divide="ignore"):
        m1 = (k["b1"] * m).astype(f32) + (k["ob1"] * g).astype(f32)
        v1 = (k["b2"] * v).astype(f32) + ((k["ob2"] * g).astype(f32) * g).astype(f32)
        den = (np.sqrt(v1.astype(f32)) * k["k2"]).astype(f32) + k["eps"]
        u = (m1.astype(f32) / den.astype(f32)).astype(f32)
        delta = -((k["cu"] * u).astype(f32) + (k["cd"] * q).astype(f32)).astype(f32)
    return delta.astype(f32), m1.astype(f32), v1.astype(f32)


def adamw_sr_update(q, g, m, v, lr, alpha, beta1, beta2, eps, weight_decay, qmin: int,
                    qmax: int, seed: int, step: int, tensor_id: int, idx=None):
    """AdamW with SR (R11): the AdamW target of ``adamw_target`` with
    t = step, rounded by Eq. 1 (``_sr_round``, draws keyed as in R7 by
    (seed, step, tensor_id, element)) and clipped to [qmin, qmax].  An element
    whose gradient is non-finite or whose delta is NaN keeps q, m and v.
    Returns (q_new int64, m_new, v_new, n_changed, n_nonfinite)."""
    q = np.asarray(q).astype(np.int64).ravel()
    g = np.asarray(g, dtype=np.float32).ravel()
    m = np.asarray(m, dtype=np.float32).ravel()
    v = np.asarray(v, dtype=np.float32).ravel()
    if idx is None:
        idx = np.arange(q.size, dtype=np.uint64)
    k = adamw_scalars(lr, alpha, beta1, beta2, eps, weight_decay, step)
    delta, m1, v1 = adamw_target(q, g, m, v, k)
    ok = np.isfinite(g) & ~np.isnan(delta)
    new = _sr_round(q, np.where(ok, delta, np.float32(0)), qmin, qmax, seed, step, tensor_id, idx)
    new = np.where(ok, new, q)
    m_new = np.where(ok, m1, m).astype(np.float32)
    v_new = np.where(ok, v1, v).astype(np.float32)
    return (new, m_new, v_new, int(np.count_nonzero(new != q)), int(np.count_nonzero(~ok)))


def sr_change_probability(q, g, lr, alpha, qmin: int, qmax: int) -> np.ndarray:
    """Per-element probability that the SR update changes the code (used for
    the Poisson-binomial check of n_changed).  Probabilities are taken at the
    2**-32 resolution of R7."""
    q = np.asarray(q).astype(np.int64).ravel()
    g = np.asarray(g, dtype=np.float32).ravel()
    c = sr_step_size(lr, alpha)
    delta = (-(c * g)).astype(np.float32).astype(np.float64)
    fl = np.floor(delta)
    frac = delta - fl
    p_hi = np.ceil(frac * 2.0 ** 32) / 2.0 ** 32        # P(x -> q + fl + 1)
    lo_val = np.clip(q + fl, qmin, qmax)
    hi_val = np.clip(q + fl + 1, qmin, qmax)
    return np.where(lo_val != q, 1.0 - p_hi, 0.0) + np.where(hi_val != q, p_hi, 0.0)


def linear_train_step(X, dY, q, alpha, qmin, qmax, *, act: str, xt: str,
                      y_out: str, dx_out: str, lr, seed, step, tensor_id):
    """One full DQT linear step: act-quant, forward, backward, SR update.

    Returns a dict of every intermediate, for comparison with the HIP path.
    """
    Xq, d = act_quant(X, act)
    Y, acc = linear_fwd(Xq, d, act, q, alpha, y_out)
    dX, dW, _, _ = linear_bwd(dY, q, alpha, Xq, d, act, xt, dx_out)
    q_new, n_changed, n_nonfinite = sr_update(q, dW, lr, alpha, qmin, qmax,
                                              seed, step, tensor_id)
    return dict(Xq=Xq, d=d, Y=Y, acc=acc, dX=dX, dW=dW,
                q_new=q_new.reshape(np.asarray(q).shape), n_changed=n_changed,
                n_nonfinite=n_nonfinite)


def gemm_abs_bound(A, B) -> np.ndarray:
    """|A| @ |B| in float64: the sum of absolute terms of each output of A @ B,
    used to scale componentwise tolerances."""
    return np.abs(np.asarray(A, dtype=np.float64)) @ np.abs(np.asarray(B, dtype=np.float64))


__all__ = [
    "bf16_round", "bf16_to_f32", "E4M3_VALUES", "e4m3_encode", "e4m3_decode",
    "pack_ternary", "unpack_ternary", "pack_int3", "unpack_int3", "absmean", "absmean_init", "act_quant",
    "act_values", "act_dequant", "cast_out", "linear_fwd", "linear_bwd",
    "philox4x32_10", "rng_u32", "sr_step_size", "sr_update",
    "sr_change_probability", "linear_train_step", "gemm_abs_bound",
]


# ---------------------------------------------------------------------------
# Next row: the analysis variants of Sec. 5 (reading R12).
# ---------------------------------------------------------------------------

UPD_SR, UPD_NEAREST, UPD_FORCE_REMAIN, UPD_FORCE_CHANGE = 0, 1, 2, 3


def delta_keys(g, lr, alpha) -> np.ndarray:
    """Ranking keys of R12: the fp32 bit pattern of |delta| = |fl32(c g)| as
    an unsigned integer (monotone in |delta|), 0xFFFFFFFF for a non-finite g."""
    g = np.asarray(g, dtype=np.float32).ravel()
    c = sr_step_size(lr, alpha)
    finite = np.isfinite(g)
    with np.errstate(over="ignore", invalid="ignore"):
        mag = np.abs((c * np.where(finite, g, np.float32(0))).astype(np.float32))
    keys = mag.astype(np.float32).view(np.uint32).copy()
    keys[~finite] = np.uint32(0xFFFFFFFF)
    return keys


def bottom_threshold(keys, frac):
    """tau = the k-th smallest key, k = floor(frac n) (frac as fp32, the
    product in float64); None when k = 0."""
    n = keys.size
    k = int(np.floor(np.float64(np.float32(frac)) * n))
    if k <= 0:
        return None
    return np.uint32(np.sort(keys)[k - 1])


def absmax_requant(q, g, lr, alpha, qmin: int, qmax: int):
    """The deterministic control of Sec. 5.1 read literally (R14): the
    updated matrix W' = W~ - lr g (W~ = q alpha) is quantised afresh with
    Eq. 3-4's form and the maximum in place of the mean,
      W'_i    = fl(fl(q_i alpha) - fl(lr g_i))       (g_i non-finite: g_i = 0)
      m       = max_i |W'_i|
      s'      = fl(qmax / m),  alpha' = fl(m / qmax)
      q'_i    = Clip(Round(fl(W'_i s')), qmin, qmax)  (Round: ties to even)
    with m = 0 giving s' = 0 and alpha' = alpha.  No stochastic rounding.
    Returns (q' int64, alpha' fp32, n_changed, n_nonfinite)."""
    q = np.asarray(q).astype(np.int64).ravel()
    g = np.asarray(g, dtype=np.float32).ravel()
    finite = np.isfinite(g)
    a = np.float32(alpha)
    w = (q.astype(np.float32) * a).astype(np.float32)
    with np.errstate(over="ignore", invalid="ignore"):
        u = (np.float32(lr) * np.where(finite, g, np.float32(0))).astype(np.float32)
    wp = (w - u).astype(np.float32)
    m = np.float32(np.max(np.abs(wp))) if wp.size else np.float32(0)
    if m == 0:
        s_new, alpha_new = np.float32(0), a
    else:
        s_new = np.float32(np.float32(qmax) / m)
        alpha_new = np.float32(m / np.float32(qmax))
    scaled = (wp * s_new).astype(np.float32)
    new = np.clip(np.rint(scaled), qmin, qmax).astype(np.int64)
    return new, alpha_new, int(np.count_nonzero(new != q)), int(np.count_nonzero(~finite))


def update_variant(q, g, lr, alpha, qmin: int, qmax: int, seed: int, step: int, tensor_id: int,
                   mode: int, frac: float = 0.2):
    """The update of Sec. 3.2 Eq. 5 with the interventions of Sec. 5 (R12):
    UPD_SR is ``sr_update``; UPD_NEAREST rounds x = q + delta to the nearest
    grid value, ties to even; UPD_FORCE_REMAIN / UPD_FORCE_CHANGE keep, or
    round away from q, the codes whose |delta| is in the bottom set of
    ``bottom_threshold`` and give the rest the plain SR update (same draws).
    A non-finite g keeps its code and is counted.  Returns (q_new,
    n_changed, n_nonfinite)."""
    q = np.asarray(q).astype(np.int64).ravel()
    g = np.asarray(g, dtype=np.float32).ravel()
    sr_new, _, nnf = sr_update(q, g, lr, alpha, qmin, qmax, seed, step, tensor_id)
    finite = np.isfinite(g)
    c = sr_step_size(lr, alpha)
    with np.errstate(over="ignore", invalid="ignore"):
        delta = (-(c * np.where(finite, g, np.float32(0)))).astype(np.float32).astype(np.float64)
    if mode == UPD_SR:
        new = sr_new
    elif mode == UPD_NEAREST:
        x = q.astype(np.float64) + delta               # exact: delta is fp32, q small
        new = np.where(finite, np.clip(np.rint(x), qmin, qmax), q).astype(np.int64)
    elif mode in (UPD_FORCE_REMAIN, UPD_FORCE_CHANGE):
        keys = delta_keys(g, lr, alpha)
        tau = bottom_threshold(keys, frac)
        bottom = np.zeros(q.size, bool) if tau is None else ((keys <= tau) & finite)
        if mode == UPD_FORCE_REMAIN:
            forced = q
        else:
            away = np.where(delta > 0, np.ceil(delta), np.where(delta < 0, np.floor(delta), 0.0))
            with np.errstate(invalid="ignore"):
                forced = np.clip(q.astype(np.float64) + away, qmin, qmax).astype(np.int64)
        new = np.where(bottom, forced, sr_new).astype(np.int64)
    else:
        raise ValueError(mode)
    return new, int(np.count_nonzero(new != q)), nnf
