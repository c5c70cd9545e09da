"""Pins of the oracle's analysis variants of the update (Sec. 5; reading R12
of the oracle): rounding to nearest against numpy's rint, the bottom-20 %
threshold against a plain sort, the two interventions on the paper's own
example, and every other element equal to the plain SR update."""
import numpy as np
import pytest

from oracle import dqt_oracle as O


def _case(n, seed, qmin=-1, qmax=1, scale=0.02):
    rng = np.random.default_rng(seed)
    q = rng.integers(qmin, qmax + 1, size=n).astype(np.int64)
    g = rng.normal(0, scale, size=n).astype(np.float32)
    return q, g


def test_nearest_is_rint_of_the_target():
    q, g = _case(50000, 1, -8, 7, scale=1.0)
    lr, alpha = 0.3, 0.25
    new, nch, _ = O.update_variant(q, g, lr, alpha, -8, 7, 0, 1, 0, O.UPD_NEAREST)
    c = np.float32(np.float32(lr) / np.float32(alpha))
    x = q + (-(c * g)).astype(np.float32).astype(np.float64)
    assert np.array_equal(new, np.clip(np.rint(x), -8, 7).astype(np.int64))
    # small updates never move (the failure the paper reports for it)
    small = np.abs((c * g).astype(np.float32)) < 0.5
    assert np.all(new[small] == q[small])
    # deterministic: the seed does not matter
    new2, *_ = O.update_variant(q, g, lr, alpha, -8, 7, 12345, 99, 7, O.UPD_NEAREST)
    assert np.array_equal(new, new2)


def test_nearest_ties_go_to_even():
    q = np.array([0, 0, 1, -1, 0, 0], np.int64)
    g = np.array([-0.5, 0.5, -0.5, 0.5, -1.5, 1.5], np.float32)   # c = 1: delta = -g
    new, *_ = O.update_variant(q, g, 1.0, 1.0, -8, 7, 0, 1, 0, O.UPD_NEAREST)
    assert new.tolist() == [0, 0, 2, -2, 2, -2]


@pytest.mark.parametrize("n,frac", [(97, 0.2), (1000, 0.2), (4096, 0.5), (10, 0.05), (33, 1.0)])
def test_bottom_threshold_is_the_kth_smallest(n, frac):
    q, g = _case(n, n)
    keys = O.delta_keys(g, 1e-2, 0.01)
    tau = O.bottom_threshold(keys, frac)
    k = int(np.floor(np.float64(np.float32(frac)) * n))
    if k == 0:
        assert tau is None
        return
    assert tau == sorted(int(x) for x in keys)[k - 1]
    # tie-free data: exactly k elements are in the bottom set
    if len(set(keys.tolist())) == n:
        assert int(np.count_nonzero(keys <= tau)) == k
    # keys order as |delta| does
    mag = np.abs((np.float32(1.0) * g).astype(np.float32))
    order = np.argsort(mag, kind="stable")
    assert np.all(np.diff(keys[order].astype(np.int64)) >= 0)


def test_paper_example_remain_and_update():
    """A code at -1 moved by +0.02 whose update is among the smallest 20 %:
    force-to-remain keeps -1, force-to-update gives 0 (Sec. 5)."""
    n = 100
    q = np.full(n, -1, np.int64)
    g = np.linspace(-0.9, -0.02, n).astype(np.float32)     # delta = +0.02 .. +0.9 (c = 1)
    g[0] = np.float32(-0.02)
    g[-1] = np.float32(-0.9)
    rem, *_ = O.update_variant(q, g, 1.0, 1.0, -1, 1, 0, 1, 0, O.UPD_FORCE_REMAIN, 0.2)
    chg, *_ = O.update_variant(q, g, 1.0, 1.0, -1, 1, 0, 1, 0, O.UPD_FORCE_CHANGE, 0.2)
    i = int(np.argmin(np.abs(g)))
    assert abs(float(g[i])) < 0.03
    assert rem[i] == -1 and chg[i] == 0
    keys = O.delta_keys(g, 1.0, 1.0)
    bottom = keys <= O.bottom_threshold(keys, 0.2)
    assert int(bottom.sum()) == 20
    assert np.all(rem[bottom] == -1) and np.all(chg[bottom] == 0)


@pytest.mark.parametrize("mode", [O.UPD_FORCE_REMAIN, O.UPD_FORCE_CHANGE])
def test_outside_the_bottom_set_is_the_plain_update(mode):
    q, g = _case(30000, 3, -127, 127, scale=0.05)
    g[[5, 77]] = [np.inf, np.nan]
    lr, alpha = 1e-2, 0.004
    new, nch, nnf = O.update_variant(q, g, lr, alpha, -127, 127, 8, 2, 5, mode, 0.2)
    sr, _, nnf2 = O.sr_update(q, g, lr, alpha, -127, 127, 8, 2, 5)
    keys = O.delta_keys(g, lr, alpha)
    bottom = (keys <= O.bottom_threshold(keys, 0.2)) & np.isfinite(g)
    assert np.array_equal(new[~bottom], sr[~bottom])
    assert nnf == nnf2 == 2 and new[5] == q[5] and new[77] == q[77]
    c = O.sr_step_size(lr, alpha)
    delta = (-(c * g)).astype(np.float32)
    if mode == O.UPD_FORCE_REMAIN:
        assert np.all(new[bottom] == q[bottom])
    else:
        d = delta[bottom]
        moved = new[bottom] - q[bottom]
        free = (d != 0) & ~(((q[bottom] == 127) & (d > 0)) | ((q[bottom] == -127) & (d < 0)))
        assert np.all(np.sign(moved[free]) == np.sign(d[free]))
        assert np.all(moved[free] != 0)
    assert nch == int(np.count_nonzero(new != q))


def test_non_finite_gradients_are_never_among_the_smallest_updates():
    """The bottom-20 % threshold with non-finite gradients present equals the
    k-th smallest |fl32(c g)| over the finite elements (k = floor(0.2 n) of
    all n): a non-finite gradient ranks above every finite one."""
    q, g = _case(30000, 6, -127, 127, scale=0.05)
    g[[3, 400, 29999]] = [np.inf, -np.inf, np.nan]
    lr, alpha = 1e-2, 0.004
    c = np.float32(np.float32(lr) / np.float32(alpha))
    fin = np.isfinite(g)
    mags = np.sort(np.abs((c * g[fin]).astype(np.float32)))
    k = int(np.floor(np.float64(np.float32(0.2)) * g.size))
    tau = O.bottom_threshold(O.delta_keys(g, lr, alpha), 0.2)
    assert tau == mags[k - 1].view(np.uint32)


def test_frac_zero_is_the_plain_update():
    q, g = _case(5000, 4)
    a, *_ = O.update_variant(q, g, 1e-2, 0.01, -1, 1, 3, 3, 3, O.UPD_FORCE_CHANGE, 0.0)
    b, *_ = O.sr_update(q, g, 1e-2, 0.01, -1, 1, 3, 3, 3)
    assert np.array_equal(a, b)


def test_int4_packing_layout():
    """4-bit codes: two's-complement nibbles, weight k in the low nibble of
    byte k // 2 when k is even; every value of [-8, 7] round-trips."""
    q = np.array([[-8, 7, 1, -1, 0, -2]], np.int64)
    p = O.pack_int4(q)
    assert p.tolist() == [[0x78, 0xF1, 0xE0]]
    allv = np.arange(-8, 8).reshape(1, 16)
    assert np.array_equal(O.unpack_int4(O.pack_int4(allv), 16), allv)


def test_int3_packing_layout():
    """3-bit codes (the n = 3 grid of Eq. 3, -4..3): a group of 8 weights is
    the 24-bit number sum_j (q_j mod 8) 2^(3j), little-endian.  For q = 0, 1,
    2, 3, -4, -3, -2, -1 the fields are 0..7, so the number is 0xFAC688:
    bytes 0x88, 0xC6, 0xFA.  Every value round-trips."""
    q = np.array([[0, 1, 2, 3, -4, -3, -2, -1, 3, 3, 3, 3, 3, 3, 3, 3]], np.int64)
    p = O.pack_int3(q)
    assert p.tolist() == [[0x88, 0xC6, 0xFA, 0xDB, 0xB6, 0x6D]]   # 3 x (011 repeated) = 0x6DB6DB
    rng = np.random.default_rng(9)
    allv = rng.integers(-4, 4, size=(5, 64))
    assert np.array_equal(O.unpack_int3(O.pack_int3(allv), 64), allv)


def test_absmax_requant_hand_example():
    """Sec. 5.1's control read literally, on a hand-computed case: alpha =
    0.5, lr = 0.25, ternary.  W~ = q alpha = [0.5, 0, -0.5, 0.5]; lr g = [0,
    0.25, -0.75, 1.0] (g = [0, 1, -3, 4]), so W' = [0.5, -0.25, 0.25, -0.5];
    m = 0.5, s' = 2, alpha' = 0.5; W' s' = [1, -0.5, 0.5, -1] rounds (ties to
    even) to [1, -0, 0, -1]."""
    q = np.array([1, 0, -1, 1])
    g = np.array([0.0, 1.0, -3.0, 4.0], np.float32)
    new, alpha_new, nch, nnf = O.absmax_requant(q, g, 0.25, 0.5, -1, 1)
    assert new.tolist() == [1, 0, 0, -1]
    assert alpha_new == np.float32(0.5) and (nch, nnf) == (2, 0)


def test_absmax_requant_drops_small_updates_and_rescales():
    """The property the paper measures: an update far below the grid step
    changes no code (SR would move a fraction of them), while one large entry
    rescales the whole tensor and sends the rest to zero."""
    rng = np.random.default_rng(21)
    q = rng.integers(-1, 2, size=4096)
    q[0] = 1                                        # max |W~| = alpha
    alpha = np.float32(0.02)
    g = (rng.standard_normal(4096) * 1e-3).astype(np.float32)
    g[0] = 0.0
    new, a2, nch, _ = O.absmax_requant(q, g, 1e-2, alpha, -1, 1)
    assert nch == 0 and np.array_equal(new, q)      # |lr g| <= 1e-4 << alpha / 2
    assert abs(float(a2) - float(alpha)) <= 1e-4
    sr_new, sr_changed, _ = O.sr_update(q, g * np.float32(100.0), 1e-2, alpha, -1, 1, 0, 1, 0)
    assert sr_changed > 0                           # SR moves some codes at a larger step
    g2 = np.zeros(4096, np.float32)
    g2[1] = -100.0                                  # W'_1 = q_1 alpha + 1
    new2, a3, _, _ = O.absmax_requant(q, g2, 1e-2, alpha, -1, 1)
    assert a3 == np.float32(np.float32(q[1] * alpha) + np.float32(1.0))
    assert new2[1] == 1 and np.count_nonzero(new2) == 1


def test_absmax_requant_int8_grid_matches_eq4_form():
    """On the 8-bit grid the new codes are Eq. 4 with s' = 127 / max|W'|:
    the entry holding the maximum maps to +-127 exactly; a non-finite
    gradient counts as zero and is counted; an all-zero W' keeps alpha."""
    rng = np.random.default_rng(22)
    q = rng.integers(-127, 128, size=1000)
    g = rng.standard_normal(1000).astype(np.float32)
    g[5] = np.nan
    new, a2, _, nnf = O.absmax_requant(q, g, 1e-3, 0.01, -127, 127)
    wp = (q.astype(np.float32) * np.float32(0.01)).astype(np.float32) - \
        (np.float32(1e-3) * np.where(np.isfinite(g), g, 0)).astype(np.float32)
    k = int(np.argmax(np.abs(wp)))
    assert abs(int(new[k])) == 127 and nnf == 1
    z, az, nz, _ = O.absmax_requant(np.zeros(16, np.int64), np.zeros(16, np.float32), 1e-3,
                                    0.25, -127, 127)
    assert not z.any() and az == np.float32(0.25) and nz == 0
