"""Pins of the oracle's zero-point epilogue (linear quantizers with a zero,
Sec. III-A rewrite) against what the paper and arithmetic fix: the expanded
four-term form against the plain dequantize-then-multiply definition, the
paper's signed-INT -> bipolar parameter rewrite, the scale-only special case,
a closed form, and planted mistakes that the pins must reject."""
import numpy as np
import pytest

import synth
from oracle import oracle as ref


def _parts(prob):
    va, vw = ref.values(prob.a_codes, prob.q), ref.values(prob.w_codes, prob.p)
    C = ref.matmul(va, vw)
    return C, ref.rowsum(va), ref.rowsum(vw)


PQ = [(1, 1), (1, 2), (2, 2), (3, 4), (4, 4), (2, 8), (8, 3), (8, 8)]


@pytest.mark.parametrize("p,q", PQ)
def test_expanded_form_equals_definition(p, q):
    g = synth.rng(90, p, q)
    prob = synth.affine_problem("t", 5, 7, 300, p, q, g)
    C, Ra, Rw = _parts(prob)
    E, T = ref.affine_epilogue(C, Ra, Rw, prob.K, prob.a_scale, prob.a_zero, prob.w_scale,
                               prob.w_zero)
    D = ref.dequant_matmul(prob.a_codes, prob.w_codes, p, q, prob.a_scale, prob.a_zero,
                           prob.w_scale, prob.w_zero)
    # D sums K float64 products in BLAS order: a few ulps of T
    assert np.all(np.abs(E - D) <= 1e-12 * T)
    assert np.all(T > 0)


def test_signed_int_rewrite():
    """Sec. III-A: X = s x + z with signed code x equals s' x' + z' with the
    bipolar value x' = 2x + 1, s' = s / 2 and z' = z - s / 2; checked exactly
    in float64 for every code at b = 1..8 and fp16 parameters."""
    g = synth.rng(91)
    for b in range(1, 9):
        x = np.arange(-(1 << (b - 1)), 1 << (b - 1), dtype=np.int64)
        s = g.uniform(0.001, 0.1, size=16).astype(np.float16).astype(np.float64)
        z = g.uniform(-0.5, 0.5, size=16).astype(np.float16).astype(np.float64)
        signed = s[:, None] * x[None, :] + z[:, None]
        xb = ref.values(x.astype(np.int8), b).astype(np.float64)
        assert np.array_equal(xb, 2 * x + 1)
        bipolar = (s / 2)[:, None] * xb[None, :] + (z - s / 2)[:, None]
        assert np.array_equal(signed, bipolar)


def test_zero_zeros_reduce_to_scale_epilogue():
    g = synth.rng(92)
    prob = synth.affine_problem("t", 4, 9, 200, 2, 4, g)
    C, Ra, Rw = _parts(prob)
    z_a = np.zeros(prob.M, np.float16)
    z_w = np.zeros(prob.N, np.float16)
    E, _ = ref.affine_epilogue(C, Ra, Rw, prob.K, prob.a_scale, z_a, prob.w_scale, z_w)
    E0, _ = ref.epilogue(C, prob.a_scale, prob.w_scale)
    assert np.array_equal(E, E0)


@pytest.mark.parametrize("p,q", [(1, 1), (2, 4), (4, 4), (8, 8)])
def test_closed_form_constant_operands(p, q):
    """All codes at the top of the range: every dequantized activation is
    s'_a (2^q - 1) + z'_a and every weight s'_w (2^p - 1) + z'_w, so
    Y[m,n] = K (s'_a (2^q-1) + z'_a)(s'_w (2^p-1) + z'_w)."""
    M, N, K = 3, 4, 129
    g = synth.rng(93, p, q)
    a = np.full((M, K), (1 << (q - 1)) - 1, np.int8)
    w = np.full((N, K), (1 << (p - 1)) - 1, np.int8)
    sa, sw = synth.scales(g, M, 0.01, 0.1), synth.scales(g, N, 0.005, 0.05)
    za, zw = synth.zero_points(g, sa, q), synth.zero_points(g, sw, p)
    va, vw = ref.values(a, q), ref.values(w, p)
    E, _ = ref.affine_epilogue(ref.matmul(va, vw), ref.rowsum(va), ref.rowsum(vw), K, sa, za, sw, zw)
    A1 = sa.astype(np.float64) * ((1 << q) - 1) + za.astype(np.float64)
    W1 = sw.astype(np.float64) * ((1 << p) - 1) + zw.astype(np.float64)
    want = K * A1[:, None] * W1[None, :]
    assert np.allclose(E, want, rtol=1e-14, atol=0)


def test_planted_mistakes_are_caught():
    """Copies of the expanded form with one term dropped, a sign flipped or the
    row sums swapped must disagree with the definition."""
    g = synth.rng(94)
    prob = synth.affine_problem("t", 6, 5, 257, 3, 2, g)
    C, Ra, Rw = _parts(prob)
    D = ref.dequant_matmul(prob.a_codes, prob.w_codes, 3, 2, prob.a_scale, prob.a_zero,
                           prob.w_scale, prob.w_zero)
    sa = prob.a_scale.astype(np.float64)[:, None]
    za = prob.a_zero.astype(np.float64)[:, None]
    sw = prob.w_scale.astype(np.float64)[None, :]
    zw = prob.w_zero.astype(np.float64)[None, :]
    Cd, K = C.astype(np.float64), prob.K
    good = sa * sw * Cd + sa * zw * Ra[:, None] + za * sw * Rw[None, :] + K * za * zw
    assert np.allclose(good, D, rtol=1e-12, atol=1e-12)
    bad = [
        sa * sw * Cd + sa * zw * Ra[:, None] + za * sw * Rw[None, :],               # no K z z
        sa * sw * Cd + za * sw * Rw[None, :] + K * za * zw,                          # no s_a z_w R_a
        sa * sw * Cd - sa * zw * Ra[:, None] + za * sw * Rw[None, :] + K * za * zw,  # sign
        sa * sw * Cd + sa * zw * Rw[None, :] + za * sw * Ra[:, None] + K * za * zw,  # swapped sums
    ]
    for b in bad:
        assert not np.allclose(b, D, rtol=1e-6, atol=1e-9)


def test_tolerance_accepts_rne_and_rejects_far_values():
    g = synth.rng(95)
    prob = synth.affine_problem("t", 8, 16, 512, 2, 4, g)
    C, Ra, Rw = _parts(prob)
    E, T = ref.affine_epilogue(C, Ra, Rw, prob.K, prob.a_scale, prob.a_zero, prob.w_scale,
                               prob.w_zero)
    h = E.astype(np.float16)
    assert ref.fp16_affine_close(h, E, T).all()
    # a float32 evaluation of the four terms also passes
    f32 = (np.float32(1) * E.astype(np.float32)).astype(np.float16)
    assert ref.fp16_affine_close(f32, E, T).all()
    # a result 1% off fails wherever |E| is not tiny next to T
    far = (E * 1.01).astype(np.float16)
    sel = np.abs(E) > 0.01 * T
    assert sel.any() and not ref.fp16_affine_close(far, E, T)[sel].any()


def test_layer_affine_workload_ranges():
    """The zero-point layer workload stays inside fp16 range and its
    cancellation is moderate (the tolerance is relative to T)."""
    prob = synth.layer_w2a4_affine("q", 4)
    C, Ra, Rw = _parts(prob)
    E, T = ref.affine_epilogue(C, Ra, Rw, prob.K, prob.a_scale, prob.a_zero, prob.w_scale,
                               prob.w_zero)
    assert np.isfinite(E.astype(np.float16)).all()
    assert np.abs(E).max() < 60000
