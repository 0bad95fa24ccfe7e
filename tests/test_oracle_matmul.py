"""Pins of the oracle's integer product and fp16 epilogue against brute force,
library routines, closed forms and a hand-worked example (APT-LLM,
arXiv 2508.19087, Sec. III-B; scale rewrite of Sec. III-A)."""
import itertools
import os
import struct
from fractions import Fraction

import numpy as np
import pytest

import synth
from oracle import oracle as ref

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
BITS = range(1, 9)


def brute_force(a_codes, w_codes):
    """Python-integer product of the values 2x+1 (Sec. III-A correspondence)."""
    M, K = a_codes.shape
    N = w_codes.shape[0]
    out = [[0] * N for _ in range(M)]
    for m in range(M):
        for n in range(N):
            out[m][n] = sum((2 * int(a_codes[m, k]) + 1) * (2 * int(w_codes[n, k]) + 1)
                            for k in range(K))
    return np.array(out, dtype=np.int64)


@pytest.mark.parametrize("p,q", list(itertools.product(BITS, BITS)))
def test_brute_force_tiny(p, q):
    g = np.random.default_rng(100 * p + q)
    for M, N, K in [(1, 1, 1), (2, 3, 5), (4, 4, 70), (3, 2, 33)]:
        a = synth.uniform_codes(g, M, K, q)
        w = synth.uniform_codes(g, N, K, p)
        assert np.array_equal(ref.gemm(a, w, p, q).astype(np.int64), brute_force(a, w))


@pytest.mark.parametrize("p,q", [(1, 1), (2, 2), (4, 4), (3, 8), (8, 8), (1, 7)])
def test_numpy_int64_matmul(p, q):
    g = np.random.default_rng(7 * p + q)
    a = synth.uniform_codes(g, 17, 300, q)
    w = synth.uniform_codes(g, 23, 300, p)
    va = 2 * a.astype(np.int64) + 1
    vw = 2 * w.astype(np.int64) + 1
    assert np.array_equal(ref.gemm(a, w, p, q).astype(np.int64), va @ vw.T)


@pytest.mark.parametrize("p,q", list(itertools.product(BITS, BITS)))
def test_exhaustive_1x1x1(p, q):
    xa = np.arange(-(1 << (q - 1)), 1 << (q - 1))
    xw = np.arange(-(1 << (p - 1)), 1 << (p - 1))
    A = np.repeat(xa, xw.size).astype(np.int8)
    W = np.tile(xw, xa.size).astype(np.int8)
    va = ref.values(A, q)
    vw = ref.values(W, p)
    C = ref.matmul(va.reshape(-1, 1), vw.reshape(-1, 1))
    assert np.array_equal(np.diag(C).astype(np.int64),
                          (2 * A.astype(np.int64) + 1) * (2 * W.astype(np.int64) + 1))


@pytest.mark.parametrize("p,q", [(1, 1), (2, 4), (4, 4), (8, 8), (5, 3)])
def test_closed_forms(p, q):
    K = 257
    top_a = np.full((2, K), (1 << (q - 1)) - 1, np.int8)   # all-ones bipolar words
    top_w = np.full((3, K), (1 << (p - 1)) - 1, np.int8)
    bot_w = np.full((3, K), -(1 << (p - 1)), np.int8)      # all-zeros bipolar words
    full = K * ((1 << p) - 1) * ((1 << q) - 1)
    assert np.all(ref.gemm(top_a, top_w, p, q) == full)
    assert np.all(ref.gemm(top_a, bot_w, p, q) == -full)


def test_xnor_identity_p1_q1():
    """At p = q = 1 the product is the XNOR-net identity K - 2 * Hamming(a, w)."""
    g = np.random.default_rng(11)
    K = 531
    a = g.integers(0, 2, size=(5, K))
    w = g.integers(0, 2, size=(6, K))
    codes_a = (a - 1).astype(np.int8)  # bipolar word bit 1 <-> code 0, bit 0 <-> code -1
    codes_w = (w - 1).astype(np.int8)
    C = ref.gemm(codes_a, codes_w, 1, 1)
    ham = (a[:, None, :] != w[None, :, :]).sum(-1)
    assert np.array_equal(C, K - 2 * ham)


def test_golden_hand_example():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "matmul_w2a2_hand.txt"))
            if l.strip() and not l.startswith("#")]
    A = np.array([[int(t) for t in r[1:]] for r in rows if r[0] == "A"], np.int8)
    W = np.array([[int(t) for t in r[1:]] for r in rows if r[0] == "W"], np.int8)
    Cw = np.array([[int(t) for t in r[1:]] for r in rows if r[0] == "C"], np.int64)
    Y00 = [int(t) for t in [r for r in rows if r[0] == "Y00"][0][1:]]
    assert np.array_equal(ref.gemm(A, W, 2, 2), Cw)
    # Sec. III-B recombination of the hand-computed plane products of C[0][0]
    assert sum(y << (i + j) for y, (i, j) in zip(Y00, [(0, 0), (0, 1), (1, 0), (1, 1)])) == Cw[0, 0]


def test_overflow_boundary():
    """|C| <= K (2^p-1)(2^q-1); the largest K whose worst case fits int32 at
    p = q = 8 is 33025."""
    top = np.full((1, 33025), 127, np.int8)
    assert int(ref.gemm(top, top, 8, 8)[0, 0]) == 33025 * 255 * 255
    top = np.full((1, 33026), 127, np.int8)
    with pytest.raises(OverflowError):
        ref.gemm(top, top, 8, 8)


def test_entries_match_full():
    g = np.random.default_rng(5)
    a = synth.uniform_codes(g, 9, 200, 3)
    w = synth.uniform_codes(g, 13, 200, 5)
    va, vw = ref.values(a, 3), ref.values(w, 5)
    C = ref.matmul(va, vw)
    mi = g.integers(0, 9, 50)
    ni = g.integers(0, 13, 50)
    assert np.array_equal(ref.matmul_entries(va, vw, mi, ni), C[mi, ni])


def test_rowsum():
    g = np.random.default_rng(6)
    a = synth.uniform_codes(g, 7, 99, 4)
    assert np.array_equal(ref.rowsum(ref.values(a, 4)), (2 * a.astype(np.int64) + 1).sum(1))


def test_epilogue_exact_and_rounded():
    """E = C s_a s_w is exact in float64 (31 + 11 + 11 <= 53 significant bits),
    and H is its round-to-nearest-even fp16, checked with Python's own IEEE
    half packing."""
    g = np.random.default_rng(8)
    C = g.integers(-(2 ** 31) + 1, 2 ** 31 - 1, size=(6, 5), dtype=np.int64).astype(np.int32)
    C[0, 0] = 2 ** 31 - 1
    C[1, 1] = -(2 ** 31) + 1
    sa = synth.scales(g, 6, 0.01, 0.1)
    sw = synth.scales(g, 5, 0.005, 0.05)
    C[2] = g.integers(-3000, 3000, size=5)
    E, H = ref.epilogue(C, sa, sw)
    for m in range(6):
        for n in range(5):
            exact = Fraction(int(C[m, n])) * Fraction(float(sa[m])) * Fraction(float(sw[n]))
            assert Fraction(float(E[m, n])) == exact
            if abs(E[m, n]) < 65504:
                half = struct.unpack("<e", struct.pack("<e", float(E[m, n])))[0]
                assert float(H[m, n]) == half


def test_fp16_acceptance():
    E = np.array([1.0, 1000.0, 1e-9, -3.0])
    ok = ref.fp16_close(np.array([1.0009765625, 1000.5, 0.0, -3.0], np.float16), E)
    assert ok.tolist() == [True, True, True, True]
    bad = ref.fp16_close(np.array([1.01, 1002.0, 1e-5, 3.0], np.float16), E)
    assert bad.tolist() == [False, False, False, False]


def test_pins_catch_planted_mistakes():
    """Each plausible mistake planted in a copy of the oracle's arithmetic (on
    the CPU) fails at least one of the pins above."""
    def decode_ok(u, bits):
        return ref.decode(u, bits)

    def decode_unsigned(u, bits):      # forgot the -1 of a zero bit
        return np.array([sum(((int(t) >> i) & 1) << i for i in range(bits)) for t in u.ravel()])

    def decode_wrong_weight(u, bits):  # weights 2^(i+1)
        return np.array([sum((2 * ((int(t) >> i) & 1) - 1) << (i + 1) for i in range(bits))
                         for t in u.ravel()])

    def decode_msb_negative(u, bits):  # two's-complement style sign on the top plane
        out = []
        for t in u.ravel():
            s = sum((2 * ((int(t) >> i) & 1) - 1) << i for i in range(bits - 1))
            s -= (2 * ((int(t) >> (bits - 1)) & 1) - 1) << (bits - 1)
            out.append(s)
        return np.array(out)

    def roundtrip_pin(decode, bits):
        x = all_codes_(bits)
        v = np.asarray(decode(ref.convert(x, bits), bits), dtype=np.int64)
        return np.array_equal(v, 2 * x.astype(np.int64) + 1)

    assert all(roundtrip_pin(decode_ok, b) for b in BITS)
    for bad in (decode_unsigned, decode_wrong_weight, decode_msb_negative):
        assert not all(roundtrip_pin(bad, b) for b in BITS)

    g = np.random.default_rng(3)
    a = synth.uniform_codes(g, 3, 9, 2)
    w = synth.uniform_codes(g, 4, 9, 3)
    va, vw = ref.values(a, 2), ref.values(w, 3)
    good = brute_force(a, w)
    mutants = [
        va[:, :-1].astype(np.int64) @ vw[:, :-1].T.astype(np.int64),          # dropped last k
        va.astype(np.int64) @ vw[:, ::-1].T.astype(np.int64),                 # reversed k on one side
        -(va.astype(np.int64) @ vw.T.astype(np.int64)),                       # sign
        (va.astype(np.int64) @ vw.T.astype(np.int64)) + va.sum(1, keepdims=True),  # extra term
    ]
    for mut in mutants:
        assert not np.array_equal(mut, good)


def all_codes_(bits):
    return np.arange(-(1 << (bits - 1)), 1 << (bits - 1), dtype=np.int64).astype(np.int8)
