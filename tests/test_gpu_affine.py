"""GPU parity of the zero-point epilogue (apt_gemm_affine) against the
oracle's exact value: every route and forced config on ragged shapes, the
W2A4 layer set at one token and at 1024 tokens (every output), and the int32
product written alongside it bit-exact."""
import numpy as np
import pytest

import paper_2508_19087_amd as apt
import synth
from gpu_util import assert_int32_equal, dev, forced_configs, pack_problem
from oracle import oracle as ref

pytestmark = pytest.mark.gpu


def run_affine(prob, cfg=None, packed=None, int32=True):
    import torch
    a, w = packed if packed is not None else pack_problem(prob)
    c16, c32 = apt.gemm_affine(a, w, dev(prob.a_scale), dev(prob.a_zero), dev(prob.w_scale),
                               dev(prob.w_zero), out_int32=int32, cfg=cfg)
    torch.cuda.synchronize()
    return c16.cpu().numpy(), (c32.cpu().numpy() if c32 is not None else None)


def expected(prob, rows=None):
    """(C, E, T) of the oracle for all rows or the given rows."""
    va = ref.values(prob.a_codes, prob.q)
    vw = ref.values(prob.w_codes, prob.p)
    sel = slice(None) if rows is None else rows
    C = ref.matmul(va[sel], vw)
    E, T = ref.affine_epilogue(C, ref.rowsum(va[sel]), ref.rowsum(vw), prob.K,
                               prob.a_scale[sel], prob.a_zero[sel], prob.w_scale, prob.w_zero)
    return C, E, T


def assert_affine_ok(got, E, T, what):
    ok = ref.fp16_affine_close(got, E, T)
    if not ok.all():
        bad = np.argwhere(~ok)
        m, n = bad[0]
        raise AssertionError("%s: %d fp16 outputs outside tolerance; first at (%d, %d): got %r "
                             "want %r (terms %r)" % (what, len(bad), m, n, float(got[m, n]),
                                                     E[m, n], T[m, n]))


@pytest.mark.parametrize("M,N,K,p,q", [(1, 7, 31, 2, 2), (5, 129, 300, 4, 4), (17, 65, 1000, 2, 4),
                                       (70, 130, 257, 3, 8), (129, 255, 640, 8, 8),
                                       (300, 513, 385, 1, 2)])
def test_affine_every_route(M, N, K, p, q):
    prob = synth.affine_problem("affine", M, N, K, p, q, synth.rng(3000, M, N, K, p, q))
    C, E, T = expected(prob)
    packed = pack_problem(prob)
    for name, cfg in [("auto", None)] + forced_configs(p, q, N, K):
        got16, got32 = run_affine(prob, cfg=cfg, packed=packed)
        what = "%s %dx%dx%d W%dA%d" % (name, M, N, K, p, q)
        assert_int32_equal(got32, C, what)
        assert_affine_ok(got16, E, T, what)


@pytest.mark.parametrize("layer", list(synth.LAYER_SHAPES))
def test_affine_layer_one_token(layer):
    prob = synth.layer_w2a4_affine(layer, 1)
    C, E, T = expected(prob)
    got16, got32 = run_affine(prob)
    assert_int32_equal(got32, C, prob.name)
    assert_affine_ok(got16, E, T, prob.name)


@pytest.mark.parametrize("layer", ["q", "gate", "down"])
def test_affine_layer_1024_tokens(layer):
    prob = synth.layer_w2a4_affine(layer, 1024)
    got16, got32 = run_affine(prob)
    C, E, T = expected(prob)
    assert_int32_equal(got32, C, prob.name)
    assert_affine_ok(got16, E, T, prob.name)


def test_affine_without_int32_output():
    prob = synth.affine_problem("affine", 33, 300, 500, 2, 4, synth.rng(3001))
    _, E, T = expected(prob)
    got16, got32 = run_affine(prob, int32=False)
    assert got32 is None
    assert_affine_ok(got16, E, T, "fp16 only")


def test_zero_zeros_match_scale_epilogue():
    """With all zero-points 0 the affine result is the plain scale epilogue's."""
    prob = synth.affine_problem("affine", 20, 200, 640, 4, 4, synth.rng(3002))
    prob.a_zero = np.zeros(prob.M, np.float16)
    prob.w_zero = np.zeros(prob.N, np.float16)
    C, E, T = expected(prob)
    got16, _ = run_affine(prob)
    E0, _ = ref.epilogue(C, prob.a_scale, prob.w_scale)
    assert np.array_equal(E, E0)
    assert ref.fp16_close(got16, E0).all()
