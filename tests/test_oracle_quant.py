"""Pins of the oracle's fp16 activation quantizer (quantize_fp16): brute-force
nearest odd level, closed forms, the error bound, the zero row, and the
equivalent signed-INT form floor(x / 2s)."""
import numpy as np
import pytest

from oracle import oracle as ref


def _rows(seed, M, K):
    g = np.random.default_rng(seed)
    x = g.standard_normal((M, K)) * g.uniform(0.01, 30.0, (M, 1))
    return x.astype(np.float16)


@pytest.mark.parametrize("q", range(1, 9))
def test_brute_force_nearest_odd_level(q):
    """Every element goes to the odd level nearest to t = x / s (fp32), ties
    to the larger level, inside +-(2^q - 1): checked against an explicit search
    over all levels."""
    x = _rows(10 + q, 6, 37)
    codes, s16 = ref.quantize_fp16(x, q)
    levels = np.arange(-(2 ** q - 1), 2 ** q, 2, dtype=np.float64)
    s = s16.astype(np.float32)
    for m in range(x.shape[0]):
        t = (x[m].astype(np.float32) / s[m]).astype(np.float64)
        for k in range(x.shape[1]):
            d = np.abs(levels - t[k])
            best = levels[np.flatnonzero(d == d.min())].max()
            assert 2 * int(codes[m, k]) + 1 == best, (q, m, k, t[k])


@pytest.mark.parametrize("q", range(1, 9))
def test_closed_forms(q):
    """Odd multiples of a power-of-two scale quantize exactly; the largest
    magnitude of a row lands on +-(2^q - 1)."""
    L = 2 ** q - 1
    s = np.float16(2.0 ** -4)
    odd = np.arange(-L, L + 1, 2)
    x = (odd * np.float64(s)).astype(np.float16)[None, :]
    codes, s16 = ref.quantize_fp16(x, q)
    assert s16[0] == s
    assert np.array_equal(2 * codes[0].astype(np.int64) + 1, odd)
    y = _rows(7, 5, 64)
    codes, _ = ref.quantize_fp16(y, q)
    v = 2 * codes.astype(np.int64) + 1
    for m in range(5):
        k = np.argmax(np.abs(y[m].astype(np.float64)))
        assert abs(v[m, k]) == L


@pytest.mark.parametrize("q", [1, 2, 3, 4, 8])
def test_error_bound(q):
    """|v s - x| <= s (a level is at most one t-unit away), up to the fp32
    rounding of t, where v is the level and s the row's fp16 scale."""
    x = _rows(20 + q, 32, 300)
    codes, s16 = ref.quantize_fp16(x, q)
    v = 2 * codes.astype(np.float64) + 1
    s = s16.astype(np.float64)[:, None]
    err = np.abs(v * s - x.astype(np.float64))
    assert np.all(err <= s * (1 + 2.0 ** -20))


def test_zero_row_and_signed_int_form():
    """A zero row has scale 0 and level +1 everywhere; every other element's
    code equals floor(t / 2) clipped to the signed q-bit range (the signed-INT
    quantizer with scale 2s)."""
    x = _rows(3, 4, 50)
    x[2] = 0
    for q in range(1, 9):
        codes, s16 = ref.quantize_fp16(x, q)
        assert s16[2] == 0 and np.all(codes[2] == 0)
        s = s16.astype(np.float32)
        for m in (0, 1, 3):
            t = x[m].astype(np.float32) / s[m]
            alt = np.clip(np.floor(t / np.float32(2)), -(2 ** (q - 1)), 2 ** (q - 1) - 1)
            assert np.array_equal(codes[m].astype(np.int64), alt.astype(np.int64))


def test_planted_mistakes_fail():
    """A truncating (instead of flooring) or a round-to-nearest-even rule would
    differ from the oracle on these inputs, so the pins above can tell."""
    x = np.array([[-3.0, -2.0, -1.0, -0.5, 0.0, 0.5, 1.0, 2.0, 3.0, 7.0]], np.float16)
    codes, s16 = ref.quantize_fp16(x, 3)
    t = x[0].astype(np.float32) / s16.astype(np.float32)[0]
    trunc = 2 * np.trunc(t / 2) + 1
    assert not np.array_equal(2 * codes[0].astype(np.int64) + 1, np.clip(trunc, -7, 7))
