"""GPU parity on the five benchmark workloads at their full sizes, in the
configuration the library selects (the one the benchmark times): every int32
output bit-exact against the oracle and every fp16 output within 1e-3 relative
of the exact value (Sec. III-B: the exact product is sum_ij 2^(i+j) Y(i,j))."""
import pytest

import synth
from gpu_util import assert_fp16_ok, assert_int32_equal, oracle_full, run

pytestmark = pytest.mark.gpu


def test_w1a2_16x512x512():
    prob = synth.w1a2_small()
    got, _ = run(prob)
    assert_int32_equal(got, oracle_full(prob), prob.name)


@pytest.mark.parametrize("M", [1, 4, 8])
@pytest.mark.parametrize("N", [4096, 11008])
def test_w2a2_decode(M, N):
    prob = synth.w2a2_decode(M, N)
    c32, c16 = run(prob, fp16=True)
    want = oracle_full(prob)
    assert_int32_equal(c32, want, prob.name)
    assert_fp16_ok(c16, want, prob, prob.name)


def test_w4a4_prefill_2048x11008x4096():
    prob = synth.w4a4_prefill()
    got, _ = run(prob)
    assert_int32_equal(got, oracle_full(prob), prob.name)


@pytest.mark.parametrize("index", range(len(synth.SWEEP_BITS)))
def test_sweep_down_projection(index):
    prob = synth.sweep_down(index)
    got, _ = run(prob)
    assert_int32_equal(got, oracle_full(prob), prob.name)


@pytest.mark.parametrize("layer", list(synth.LAYER_SHAPES))
@pytest.mark.parametrize("M", [1, 1024])
def test_w2a4_layer(layer, M):
    prob = synth.layer_w2a4(layer, M)
    c32, c16 = run(prob, fp16=True)
    want = oracle_full(prob)
    assert_int32_equal(c32, want, prob.name)
    assert_fp16_ok(c16, want, prob, prob.name)
