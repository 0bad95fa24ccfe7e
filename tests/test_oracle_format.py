"""Pins of the oracle's bipolar-INT conversion, decoding and packed layout
against what APT-LLM (arXiv 2508.19087) Sec. III-A / IV-A fix, independent of
the oracle's own formulas."""
import os

import numpy as np
import pytest

from oracle import oracle as ref

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def all_codes(bits):
    return np.arange(-(1 << (bits - 1)), 1 << (bits - 1), dtype=np.int64).astype(np.int8)


@pytest.mark.parametrize("bits", range(1, 9))
def test_roundtrip_every_code(bits):
    """Lossless signed <-> bipolar round trip over every code (Sec. III-A):
    value = 2x + 1, word = x + 2^(b-1), image = all odd integers in range,
    inverse recovers x, complementing every bit negates the value."""
    x = all_codes(bits)
    u = ref.convert(x, bits)
    v = ref.decode(u, bits)
    xi = x.astype(np.int64)
    assert np.array_equal(v, 2 * xi + 1)
    assert np.array_equal(u.astype(np.int64), xi + (1 << (bits - 1)))
    top = (1 << bits) - 1
    assert sorted(v.tolist()) == list(range(-top, top + 1, 2))
    assert np.array_equal((v.astype(np.int64) - 1) // 2, xi)
    comp = (~u) & np.uint8(top)
    assert np.array_equal(ref.decode(comp, bits), -v)


def test_golden_code_table():
    rows = [l.split() for l in open(os.path.join(GOLDEN, "bipolar_codes.txt"))
            if l.strip() and not l.startswith("#")]
    assert len(rows) == 14
    for bits, code, word, value in rows:
        bits, code, value = int(bits), int(code), int(value)
        u = ref.convert(np.array([code], np.int8), bits)
        assert format(int(u[0]), "0%db" % bits) == word
        assert int(ref.decode(u, bits)[0]) == value


@pytest.mark.parametrize("bits", range(1, 9))
def test_out_of_range_codes_use_low_bits(bits):
    """Codes outside the signed range are reduced modulo 2^b."""
    x = np.arange(-128, 128, dtype=np.int64).astype(np.int8)
    low = (x.astype(np.int64) & ((1 << bits) - 1))
    wrapped = np.where(low >= (1 << (bits - 1)), low - (1 << bits), low)
    assert np.array_equal(ref.values(x, bits), 2 * wrapped + 1)


def test_bad_bits_rejected():
    with pytest.raises(ValueError):
        ref.convert(np.zeros(3, np.int8), 0)
    with pytest.raises(ValueError):
        ref.decode(np.zeros(3, np.uint8), 9)


def test_golden_packed_layout():
    lines = {l.split()[0]: l.split()[1:] for l in open(os.path.join(GOLDEN, "packed_layout_w2.txt"))
             if l.strip() and not l.startswith("#")}
    R, K, bits = int(lines["R"][0]), int(lines["K"][0]), int(lines["bits"][0])
    u = (np.arange(K) % 4).astype(np.uint8).reshape(R, K)
    want = np.zeros(int(lines["total"][0]), dtype=np.uint32)
    for item in lines["nonzero"]:
        idx, val = item.split(":")
        want[int(idx)] = int(val, 16)
    got = ref.pack(u, bits)
    assert np.array_equal(got, want)
    back, stray = ref.unpack(got, R, K, bits)
    assert stray == 0 and np.array_equal(back, u)


def _pack_by_dict(u, bits):
    """Independent statement of the layout: a map from (row, k, plane) to the
    (word, bit) it occupies, filled element by element."""
    R, K = u.shape
    nc = (K + 127) // 128
    words = {}
    for r in range(R):
        for k in range(K):
            for i in range(bits):
                if (int(u[r, k]) >> i) & 1:
                    idx = (((r // 8) * nc + k // 128) * bits + i) * 32 + (r % 8) * 4 + (k % 128) // 32
                    words[idx] = words.get(idx, 0) | (1 << (k % 32))
    out = np.zeros((R + 7) // 8 * 8 * nc * bits * 4, dtype=np.uint32)
    for idx, val in words.items():
        out[idx] = val
    return out


@pytest.mark.parametrize("R,K,bits", [(1, 1, 1), (3, 31, 2), (2, 33, 3), (2, 129, 4), (1, 300, 8),
                                      (4, 128, 5), (2, 257, 7), (9, 200, 3), (16, 130, 2)])
def test_pack_unpack(R, K, bits):
    g = np.random.default_rng(R * 1000 + K * 10 + bits)
    u = g.integers(0, 1 << bits, size=(R, K)).astype(np.uint8)
    packed = ref.pack(u, bits)
    assert packed.size == ref.packed_words(R, K, bits)
    assert np.array_equal(packed, _pack_by_dict(u, bits))
    back, stray = ref.unpack(packed, R, K, bits)
    assert stray == 0 and np.array_equal(back, u)
    nc = (K + 127) // 128
    if K % 128:
        bad = packed.copy()
        last = ((0 * nc + nc - 1) * bits + 0) * 32 + 0 * 4 + 3  # row 0, last chunk, word 3, bit 31
        bad[last] |= np.uint32(1 << 31)
        assert ref.unpack(bad, R, K, bits)[1] == 1
    if R % 8:
        bad = packed.copy()
        row = R  # first padding row
        bad[(((row // 8) * nc + 0) * bits + 0) * 32 + (row % 8) * 4] |= np.uint32(1)
        assert ref.unpack(bad, R, K, bits)[1] == 1


# ---- FP4 (E2M1) operands: what the FP4 route relies on ------------------------

def e2m1_value(nibble: int) -> float:
    """OCP E2M1 decoding: sign bit 3, exponent bits 2..1 (bias 1), mantissa
    bit 0; exponent 0 is subnormal (0.5 * mantissa)."""
    s = -1.0 if nibble & 8 else 1.0
    e = (nibble >> 1) & 3
    m = nibble & 1
    return s * (0.5 * m if e == 0 else 2.0 ** (e - 1) * (1.0 + 0.5 * m))


def test_e2m1_codes_of_bipolar_values():
    """Every bipolar value of 1 or 2 bits is exact in E2M1, with the nibbles the
    FP4 route builds from the planes: b = 1: (~u) << 3 | 0b0010; b = 2 with
    u = 2h + l: (~h) << 3 | x << 2 | (~x) << 1 | x, x = ~(h ^ l)."""
    for u in (0, 1):
        v = int(ref.decode(np.array([u], np.uint8), 1)[0])
        nib = ((1 - u) << 3) | 0b0010
        assert e2m1_value(nib) == v == 2 * u - 1
    for u in range(4):
        h, l = u >> 1, u & 1
        x = 1 - (h ^ l)
        nib = ((1 - h) << 3) | (x << 2) | ((1 - x) << 1) | x
        v = int(ref.decode(np.array([u], np.uint8), 2)[0])
        assert e2m1_value(nib) == v == 2 * u - 3
    # 3-bit values (+-5, +-7) are not E2M1 values: the route stops at 2 bits
    values = {e2m1_value(n) for n in range(16)}
    assert 5.0 not in values and 7.0 not in values


def test_fp32_sums_exact_below_2_24():
    """The FP4 route accumulates in fp32: with K (2^p-1)(2^q-1) < 2^24 every
    partial sum is an integer below 2^24 in magnitude, so any order of fp32
    additions is exact; just past the bound an fp32 sum can lose a unit."""
    g = np.random.default_rng(5)
    for p, q in [(1, 1), (1, 2), (2, 2)]:
        K = (1 << 24) // (((1 << p) - 1) * ((1 << q) - 1)) - 1
        va = np.full(K, (1 << q) - 1, np.int64)
        vw = np.full(K, (1 << p) - 1, np.int64)
        prod = (va * vw).astype(np.float32)
        assert float(np.cumsum(prod, dtype=np.float32)[-1]) == float((va * vw).sum())
        small = g.choice([-3, -1, 1, 3], size=5000).astype(np.float32)
        assert float(np.sum(small, dtype=np.float32)) == float(small.astype(np.int64).sum())
    over = np.full((1 << 24) // 9 + 2, 9.0, np.float32)
    assert float(np.cumsum(over, dtype=np.float32)[-1]) != 9.0 * over.size


# ---- FP8 (E4M3) activations of the FP4 route (q = 3, 4) -------------------------

def e4m3_value(byte: int) -> float:
    """OCP E4M3 decoding: sign bit 7, exponent bits 6..3 (bias 7), mantissa
    bits 2..0; exponent 0 is subnormal (2^-6 * mantissa / 8); 0x7F and 0xFF
    are NaN."""
    if byte & 0x7F == 0x7F:
        return float("nan")
    s = -1.0 if byte & 0x80 else 1.0
    e = (byte >> 3) & 15
    m = byte & 7
    return s * (2.0 ** -6 * m / 8 if e == 0 else 2.0 ** (e - 7) * (1.0 + m / 8))


def test_e4m3_codes_of_bipolar_values():
    """Every bipolar value of up to 4 bits (odd, |v| <= 15) is exact in E4M3,
    with exponent field 7 + floor(log2 |v|) and the next three bits of |v| as
    mantissa (the bytes the FP4 route's activation expansion writes); 17, the
    first odd value past 4 bits, is not an E4M3 value."""
    table = {e4m3_value(b): b for b in range(256) if e4m3_value(b) == e4m3_value(b)}
    for q in range(1, 5):
        for u in range(1 << q):
            v = int(ref.decode(np.array([u], np.uint8), q)[0])
            assert v == 2 * u - ((1 << q) - 1)
            a = abs(v)
            e = a.bit_length() - 1
            byte = ((e + 7) << 3) | (((a << 3) >> e) & 7) | (0x80 if v < 0 else 0)
            assert e4m3_value(byte) == v
            assert table[float(v)] == byte
    assert 17.0 not in table


def test_fp32_sums_exact_with_fp8_activations():
    """W2A4 through the FP4 route: products up to 3 * 15 = 45; with
    K_pad * 45 < 2^24 every fp32 partial sum is an exact integer."""
    k_pad = ((1 << 24) - 1) // 45 // 128 * 128
    prod = np.full(k_pad, 45.0, np.float32)
    assert float(np.cumsum(prod, dtype=np.float32)[-1]) == 45.0 * k_pad
    over = np.full((1 << 24) // 45 + 2, 45.0, np.float32)
    assert float(np.cumsum(over, dtype=np.float32)[-1]) != 45.0 * over.size


# ---- FP6 (E2M3) operands of the FP6 route (p, q <= 3) ----------------------------

def e2m3_value(code: int) -> float:
    """OCP E2M3 decoding: sign bit 5, exponent bits 4..3 (bias 1), mantissa
    bits 2..0; exponent 0 is subnormal (mantissa / 8)."""
    s = -1.0 if code & 32 else 1.0
    e = (code >> 3) & 3
    m = code & 7
    return s * (m / 8 if e == 0 else 2.0 ** (e - 1) * (1.0 + m / 8))


def test_e2m3_codes_of_bipolar_values():
    """Every bipolar value of up to 3 bits (odd, |v| <= 7) is exact in E2M3 with
    exactly one code (the table the FP6 route maps words through), and 9, the
    first odd value past 3 bits, is not an E2M3 value."""
    table = {}
    for c in range(64):
        table.setdefault(e2m3_value(c), []).append(c)
    for b in range(1, 4):
        for u in range(1 << b):
            v = int(ref.decode(np.array([u], np.uint8), b)[0])
            assert v == 2 * u - ((1 << b) - 1)
            codes = table[float(v)]
            assert len(codes) == 1
            # sign bit set exactly for negative values; exponent 1..3 (normal numbers)
            assert (codes[0] >> 5) == (1 if v < 0 else 0) and 1 <= (codes[0] >> 3) & 3 <= 3
    assert 9.0 not in table and -9.0 not in table


def test_fp32_sums_exact_with_fp6_operands():
    """W3A3 through the FP6 route: products up to 7 * 7 = 49; with
    K_pad * 49 < 2^24 every fp32 partial sum is an exact integer, and just past
    the bound an fp32 running sum loses a unit."""
    k_pad = ((1 << 24) - 1) // 49 // 128 * 128
    prod = np.full(k_pad, 49.0, np.float32)
    assert float(np.cumsum(prod, dtype=np.float32)[-1]) == 49.0 * k_pad
    over = np.full((1 << 24) // 49 + 2, 49.0, np.float32)
    assert float(np.cumsum(over, dtype=np.float32)[-1]) != 49.0 * over.size


# ---- FP8 (E4M3) operands of the FP8 route (p, q <= 4) ----------------------------

def test_fp32_sums_exact_with_fp8_operands():
    """W4A4 through the FP8 route (both operands E4M3, whose codes of the bipolar
    values up to 4 bits are pinned above): products up to 15 * 15 = 225; with
    K_pad * 225 < 2^24 every fp32 partial sum is an exact integer, and just past
    the bound an fp32 running sum loses a unit."""
    k_pad = ((1 << 24) - 1) // 225 // 128 * 128
    prod = np.full(k_pad, 225.0, np.float32)
    assert float(np.cumsum(prod, dtype=np.float32)[-1]) == 225.0 * k_pad
    over = np.full((1 << 24) // 225 + 2, 225.0, np.float32)
    assert float(np.cumsum(over, dtype=np.float32)[-1]) != 225.0 * over.size
    # every product of two 4-bit bipolar values is an integer that fp32 and
    # E4M3 x E4M3 hold exactly
    vals = [2 * u - 15 for u in range(16)]
    for a in vals:
        for b in vals:
            assert float(np.float32(a) * np.float32(b)) == a * b
