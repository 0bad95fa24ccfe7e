"""Seeded random problems through the GPU path: random sizes (ragged in every
dimension), random bit widths and a random forced config of those the library
can run for them, plus the selected config; int32 bit-exact against the oracle
and the fp16 scale epilogue within tolerance."""
import numpy as np
import pytest

import synth
from gpu_util import assert_fp16_ok, assert_int32_equal, forced_configs, oracle_full, pack_problem, run

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("case", range(40))
def test_random_problem_random_config(case):
    g = synth.rng(7000, case)
    M = int(g.integers(1, 300))
    N = int(g.integers(1, 700))
    K = int(g.integers(1, 1500))
    p, q = int(g.integers(1, 9)), int(g.integers(1, 9))
    prob = synth.random_problem(g, M, N, K, p, q, with_scales=True)
    want = oracle_full(prob)
    packed = pack_problem(prob)
    cfgs = forced_configs(p, q, N, K)
    name, cfg = cfgs[int(g.integers(0, len(cfgs)))]
    for label, c in (("auto", None), (name, cfg)):
        what = "case %d %s %dx%dx%d W%dA%d" % (case, label, M, N, K, p, q)
        got32, got16 = run(prob, cfg=c, fp16=True, packed=packed)
        assert_int32_equal(got32, want, what)
        assert_fp16_ok(got16, want, prob, what)


@pytest.mark.parametrize("case", range(40))
def test_random_problem_from_codes(case):
    """The same kind of random problems through apt_gemm_act (activations as
    int8 codes, converted inside the call) in the selected and a random forced
    config; int32 and fp16 against the oracle."""
    import torch

    import paper_2508_19087_amd as apt
    g = synth.rng(7100, case)
    M = int(g.integers(1, 300))
    N = int(g.integers(1, 700))
    K = int(g.integers(1, 1500))
    p, q = int(g.integers(1, 9)), int(g.integers(1, 9))
    prob = synth.random_problem(g, M, N, K, p, q, with_scales=True)
    want = oracle_full(prob)
    w = apt.pack(torch.from_numpy(prob.w_codes).cuda(), p)
    cfgs = forced_configs(p, q, N, K)
    name, cfg = cfgs[int(g.integers(0, len(cfgs)))]
    for label, c in (("auto", None), (name, cfg)):
        what = "case %d %s %dx%dx%d W%dA%d" % (case, label, M, N, K, p, q)
        c32, c16, _ = apt.gemm_act(torch.from_numpy(prob.a_codes).cuda(), q, w,
                                   a_scale=torch.from_numpy(prob.a_scale).cuda(),
                                   w_scale=torch.from_numpy(prob.w_scale).cuda(), out_fp16=True, cfg=c)
        torch.cuda.synchronize()
        assert_int32_equal(c32.cpu().numpy(), want, what)
        assert_fp16_ok(c16.cpu().numpy(), want, prob, what)
