"""Pins for the oracle's random bits (Philox4x32-10 and the per-element
16+16-bit draw).  CPU only."""
import os

import numpy as np
import pytest

from oracle import dqt_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _kat_rows():
    rows = []
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            rows.append([int(t, 16) for t in line.split()])
    return rows


@pytest.mark.parametrize("row", _kat_rows())
def test_philox_known_answers(row):
    ctr, key, want = row[0:4], row[4:6], row[6:10]
    got = [int(v) for v in O.philox4x32_10(ctr, key)]
    assert got == want, [hex(v) for v in got]


def test_philox_vectorised_matches_scalar():
    ctr = [np.arange(5, dtype=np.uint64), np.full(5, 7), np.full(5, 9), np.full(5, 11)]
    vec = O.philox4x32_10(ctr, (123, 456))
    for j in range(5):
        one = O.philox4x32_10([j, 7, 9, 11], (123, 456))
        assert [int(v[j]) for v in vec] == [int(v) for v in one]


def test_half16_word_and_half_layout():
    """Element i of a block of 8 takes word (i & 7) >> 1, low half if even."""
    seed, step, tid = 0x1234_5678_9ABC_DEF0, 5, 3
    base = 8 * 1000
    idx = np.arange(base, base + 8, dtype=np.uint64)
    words = O.philox4x32_10([1000, 0, step, tid], (seed & 0xFFFFFFFF, seed >> 32))
    p = O._half16(seed, step, tid, idx, 0)
    for j in range(8):
        w = int(words[j >> 1])
        assert int(p[j]) == ((w >> (16 * (j & 1))) & 0xFFFF)
    # stream 1 sets the top bit of counter word 1
    words1 = O.philox4x32_10([1000, 1 << 31, step, tid], (seed & 0xFFFFFFFF, seed >> 32))
    s = O._half16(seed, step, tid, idx, 1)
    for j in range(8):
        w = int(words1[j >> 1])
        assert int(s[j]) == ((w >> (16 * (j & 1))) & 0xFFFF)


N_STAT = 1 << 20


def _chi2_uniform(values, nbins):
    counts = np.bincount(values, minlength=nbins)
    exp = values.size / nbins
    return float(np.sum((counts - exp) ** 2 / exp))


def test_u32_bytes_uniform_chi2():
    u = O.rng_u32(7, 1, 0, np.arange(N_STAT, dtype=np.uint64)).astype(np.int64)
    for shift in (0, 8, 16, 24):
        chi2 = _chi2_uniform((u >> shift) & 0xFF, 256)
        # chi^2 with 255 dof: mean 255, sd ~22.6; accept within 6 sd
        assert abs(chi2 - 255) < 6 * np.sqrt(2 * 255), (shift, chi2)


def test_u32_16bit_halves_uniform_chi2():
    u = O.rng_u32(11, 3, 2, np.arange(N_STAT, dtype=np.uint64)).astype(np.int64)
    for shift in (0, 16):
        chi2 = _chi2_uniform((u >> shift) & 0xFFFF, 1 << 16)
        dof = (1 << 16) - 1
        assert abs(chi2 - dof) < 6 * np.sqrt(2 * dof), (shift, chi2)


def test_u32_bit_balance():
    u = O.rng_u32(0, 1, 0, np.arange(N_STAT, dtype=np.uint64)).astype(np.uint64)
    sd = 0.5 / np.sqrt(N_STAT)
    for b in range(32):
        frac = float(np.mean((u >> np.uint64(b)) & np.uint64(1)))
        assert abs(frac - 0.5) < 6 * sd, (b, frac)


def test_streams_are_distinct_and_uncorrelated():
    idx = np.arange(1 << 18, dtype=np.uint64)
    a = O.rng_u32(0, 1, 0, idx).astype(np.float64)
    others = [O.rng_u32(0, 2, 0, idx), O.rng_u32(0, 1, 1, idx), O.rng_u32(1, 1, 0, idx),
              O.rng_u32(1 << 32, 1, 0, idx)]
    for b in others:
        b = b.astype(np.float64)
        assert np.count_nonzero(a == b) < 8
        r = np.corrcoef(a, b)[0, 1]
        assert abs(r) < 6 / np.sqrt(idx.size)
    # adjacent elements are uncorrelated too
    r = np.corrcoef(a[:-1], a[1:])[0, 1]
    assert abs(r) < 6 / np.sqrt(idx.size)


def test_high_element_indices():
    """Indices above 2**35 use the high counter word; still distinct draws."""
    idx = np.array([0, 8, (1 << 35), (1 << 35) + 8, (1 << 40) + 3], dtype=np.uint64)
    u = O.rng_u32(0, 1, 0, idx)
    assert len(set(int(v) for v in u)) == idx.size
