"""GPU parity of every GEMM route against the oracle: bit-exact int32 over
all 64 (p, q) pairs, ragged shapes, config invariance, repeat determinism and
the fp16 scale epilogue."""
import itertools

import numpy as np
import pytest

import paper_2508_19087_amd as apt
import synth
from gpu_util import (assert_fp16_ok, assert_int32_equal, forced_configs, oracle_full,
                      pack_problem, run)

pytestmark = pytest.mark.gpu
PQ = list(itertools.product(range(1, 9), range(1, 9)))


@pytest.mark.parametrize("p,q", PQ)
def test_all_bit_widths_every_route(p, q):
    g = synth.rng(1000, p, q)
    for M, N, K in [(17, 33, 257), (70, 130, 300)]:
        prob = synth.random_problem(g, M, N, K, p, q)
        want = oracle_full(prob)
        packed = pack_problem(prob)
        for name, cfg in forced_configs(p, q, N, K):
            got, _ = run(prob, cfg=cfg, packed=packed)
            assert_int32_equal(got, want, "%s p=%d q=%d %dx%dx%d" % (name, p, q, M, N, K))


SHAPES = [(1, 1, 1), (1, 7, 31), (2, 5, 32), (3, 64, 33), (4, 3, 127), (5, 129, 128), (8, 256, 129),
          (9, 100, 1), (16, 512, 512), (17, 65, 4096), (64, 64, 64), (65, 257, 385),
          (128, 128, 256), (129, 255, 1000), (300, 513, 640)]


@pytest.mark.parametrize("M,N,K", SHAPES)
@pytest.mark.parametrize("p,q", [(1, 2), (2, 2), (4, 4), (3, 8), (8, 8), (2, 4)])
def test_ragged_shapes(M, N, K, p, q):
    prob = synth.random_problem(synth.rng(2000, M, N, K, p, q), M, N, K, p, q)
    want = oracle_full(prob)
    packed = pack_problem(prob)
    got, _ = run(prob, packed=packed)  # selected config
    assert_int32_equal(got, want, "auto")
    for name, cfg in forced_configs(p, q, N, K):
        got, _ = run(prob, cfg=cfg, packed=packed)
        assert_int32_equal(got, want, name)


@pytest.mark.parametrize("q", [2, 4])
def test_fp4_exact_at_its_bound(q):
    """The FP4 route sums in fp32 and takes W2Aq while K_pad (2^2-1)(2^q-1) < 2^24 (K_pad = K
    rounded up to 128; the padding products count too).  At the largest such K_pad with every
    product at its maximum (+9 with FP4 activations, +45 with FP8 ones), the running sum climbs
    to one step below 2^24; rows with mixed signs and a K whose last chunk is padded go
    through the same configs."""
    p = 2
    top = 3 * ((1 << q) - 1)
    k_pad = ((1 << 24) - 1) // top // 128 * 128
    fp4 = [(n, c) for n, c in forced_configs(p, q, 10, k_pad) if c.route == apt.APT_ROUTE_FP4_MFMA]
    assert fp4
    for K in (k_pad, k_pad - 57):
        g = synth.rng(2500, K, q)
        M, N = 3, 10
        a = np.full((M, K), (1 << (q - 1)) - 1, np.int8)  # largest code: value 2^q - 1
        w = np.ones((N, K), np.int8)                     # code 1: value +3
        w[1::2] = -2                                     # code -2: value -3
        a[2] = synth.uniform_codes(g, 1, K, q)[0]
        w[2] = synth.uniform_codes(g, 1, K, p)[0]
        prob = synth.Problem("fp4 bound", M, N, K, p, q, w, a)
        want = oracle_full(prob)
        assert want[0, 0] == top * K and want[0, 1] == -top * K
        packed = pack_problem(prob)
        for name, cfg in fp4:
            got, _ = run(prob, cfg=cfg, packed=packed)
            assert_int32_equal(got, want, "%s K=%d" % (name, K))


def test_fp6_exact_at_its_bound():
    """The FP6 route sums in fp32 and takes W3A3 while K_pad * 49 < 2^24 (the padding
    products count too).  At the largest such K_pad with every product +49 the running
    sum climbs to within one product of 2^24; rows with mixed signs, uniform codes and
    a K whose last chunk is padded go through every FP6 config."""
    p = q = 3
    k_pad = ((1 << 24) - 1) // 49 // 128 * 128
    fp6 = [(n, c) for n, c in forced_configs(p, q, 10, k_pad) if c.route == apt.APT_ROUTE_FP6_MFMA]
    assert fp6
    for K in (k_pad, k_pad - 57):
        g = synth.rng(2600, K)
        M, N = 3, 10
        a = np.full((M, K), 3, np.int8)   # code 3: value +7
        w = np.full((N, K), 3, np.int8)
        w[1::2] = -4                      # code -4: value -7
        a[2] = synth.uniform_codes(g, 1, K, q)[0]
        w[2] = synth.uniform_codes(g, 1, K, p)[0]
        prob = synth.Problem("fp6 bound", M, N, K, p, q, w, a)
        want = oracle_full(prob)
        assert want[0, 0] == 49 * K and want[0, 1] == -49 * K
        packed = pack_problem(prob)
        for name, cfg in fp6:
            got, _ = run(prob, cfg=cfg, packed=packed)
            assert_int32_equal(got, want, "%s K=%d" % (name, K))


def test_fp8_exact_at_its_bound():
    """The FP8 route sums in fp32 and takes W4A4 while K_pad * 225 < 2^24 (the
    padding products count too).  At the largest such K_pad with every product
    +225 the running sum climbs to within one product of 2^24; rows with mixed
    signs, uniform codes and a K whose last chunk is padded go through every FP8
    config."""
    p = q = 4
    k_pad = ((1 << 24) - 1) // 225 // 128 * 128
    fp8 = [(n, c) for n, c in forced_configs(p, q, 10, k_pad) if c.route == apt.APT_ROUTE_FP8_MFMA]
    assert fp8
    for K in (k_pad, k_pad - 57):
        g = synth.rng(2700, K)
        M, N = 3, 10
        a = np.full((M, K), 7, np.int8)   # code 7: value +15
        w = np.full((N, K), 7, np.int8)
        w[1::2] = -8                      # code -8: value -15
        a[2] = synth.uniform_codes(g, 1, K, q)[0]
        w[2] = synth.uniform_codes(g, 1, K, p)[0]
        prob = synth.Problem("fp8 bound", M, N, K, p, q, w, a)
        want = oracle_full(prob)
        assert want[0, 0] == 225 * K and want[0, 1] == -225 * K
        packed = pack_problem(prob)
        for name, cfg in fp8:
            got, _ = run(prob, cfg=cfg, packed=packed)
            assert_int32_equal(got, want, "%s K=%d" % (name, K))


def test_extreme_values_all_ones_and_zeros():
    """Worst-case magnitudes: all-ones / all-zeros bipolar words at p = q = 8."""
    for M, N, K in [(3, 5, 1000), (70, 80, 4100)]:
        a = np.full((M, K), 127, np.int8)
        w = np.full((N, K), 127, np.int8)
        w[1::2] = -128
        prob = synth.Problem("extreme", M, N, K, 8, 8, w, a)
        want = oracle_full(prob)
        assert want[0, 0] == K * 255 * 255 and want[0, 1] == -K * 255 * 255
        packed = pack_problem(prob)
        for name, cfg in [("auto", None)] + forced_configs(8, 8, N, K):
            got, _ = run(prob, cfg=cfg, packed=packed)
            assert_int32_equal(got, want, name)


def test_max_k_p8_q8():
    """Largest K whose worst case fits int32 at p = q = 8 (33025)."""
    K = 33025
    a = np.full((2, K), 127, np.int8)
    w = np.full((3, K), 127, np.int8)
    w[1] = -128
    prob = synth.Problem("maxk", 2, 3, K, 8, 8, w, a)
    want = oracle_full(prob)
    packed = pack_problem(prob)
    for name, cfg in [("auto", None)] + forced_configs(8, 8):
        got, _ = run(prob, cfg=cfg, packed=packed)
        assert_int32_equal(got, want, name)


def test_deterministic_repeats():
    """20 launches of each route give bit-identical outputs (an LDS race would
    show up as run-to-run differences)."""
    prob = synth.random_problem(synth.rng(3000), 300, 700, 1500, 4, 4)
    want = oracle_full(prob)
    packed = pack_problem(prob)
    for name, cfg in forced_configs(4, 4, 700, 1500):
        for _ in range(20):
            got, _ = run(prob, cfg=cfg, packed=packed)
            assert_int32_equal(got, want, name)


@pytest.mark.parametrize("M,N,K,p,q", [(1, 300, 640, 2, 2), (8, 129, 4096, 2, 4),
                                       (100, 200, 1000, 4, 4), (33, 70, 129, 8, 8)])
def test_fp16_epilogue(M, N, K, p, q):
    prob = synth.random_problem(synth.rng(4000, M, N, K), M, N, K, p, q, with_scales=True)
    want = oracle_full(prob)
    packed = pack_problem(prob)
    for name, cfg in [("auto", None)] + forced_configs(p, q, N, K):
        c32, c16 = run(prob, cfg=cfg, fp16=True, packed=packed)
        assert_int32_equal(c32, want, name)
        assert_fp16_ok(c16, want, prob, name)
        _, c16b = run(prob, cfg=cfg, int32=False, fp16=True, packed=packed)
        assert np.array_equal(c16b.view(np.uint16), c16.view(np.uint16))
