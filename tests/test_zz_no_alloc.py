"""apt_gemm_noalloc (the GEMM whose workspace is the library's own device array)
against apt_gemm (caller workspace) on the same operands: int32 bit for bit,
fp16 bit for bit (same kernels) and both against the oracle, over two or more
calls in a row with a smaller problem after a larger one, so that a stale
fragment or stream-K counter left in the shared array would show."""
import numpy as np
import pytest

import paper_2508_19087_amd as apt
import synth
from gpu_util import assert_fp16_ok, assert_int32_equal, dev, oracle_full, pack_problem

pytestmark = pytest.mark.gpu

SCRATCH_BYTES = 64 << 20


def _call_noalloc(prob, a, w, cfg=None, fp16=True):
    import torch
    M, N, K = prob.M, prob.N, prob.K
    c32 = torch.full((M, N), -7, dtype=torch.int32, device="cuda")
    c16 = torch.full((M, N), 1.5, dtype=torch.float16, device="cuda") if fp16 else None
    sa = dev(prob.a_scale) if fp16 else None
    sw = dev(prob.w_scale) if fp16 else None
    st = apt.apt_gemm_noalloc(M, N, K, prob.p, prob.q, a.data.data_ptr(), w.data.data_ptr(),
                              a.rowsum.data_ptr(), w.rowsum.data_ptr(), c32.data_ptr(),
                              sa.data_ptr() if fp16 else None, sw.data_ptr() if fp16 else None,
                              c16.data_ptr() if fp16 else None, cfg,
                              torch.cuda.current_stream().cuda_stream)
    apt.check(st, "apt_gemm_noalloc")
    torch.cuda.synchronize()
    return c32.cpu().numpy(), (c16.cpu().numpy() if fp16 else None)


def _call_gemm(prob, a, w, cfg=None, fp16=True):
    import torch
    sa = dev(prob.a_scale) if fp16 else None
    sw = dev(prob.w_scale) if fp16 else None
    c32, c16 = apt.gemm(a, w, a_scale=sa, w_scale=sw, out_fp16=fp16, cfg=cfg)
    torch.cuda.synchronize()
    return c32.cpu().numpy(), (c16.cpu().numpy() if fp16 else None)


def _check(prob, cfg=None, what=""):
    a, w = pack_problem(prob)
    got32, got16 = _call_noalloc(prob, a, w, cfg)
    ref32, ref16 = _call_gemm(prob, a, w, cfg)
    want = oracle_full(prob)
    assert_int32_equal(got32, ref32, what + " vs apt_gemm")
    assert_int32_equal(got32, want, what + " vs oracle")
    assert np.array_equal(got16.view(np.uint16), ref16.view(np.uint16)), what + " fp16 vs apt_gemm"
    assert_fp16_ok(got16, want, prob, what)


def test_noalloc_matches_gemm_larger_then_smaller():
    # larger problem first (W4A4 on the MFMA route), then a smaller one (W2A3,
    # ragged), then the decode route (no workspace at all)
    big = synth.random_problem(synth.rng(6000), 1100, 2000, 3000, 4, 4, with_scales=True)
    small = synth.random_problem(synth.rng(6001), 70, 300, 500, 2, 3, with_scales=True)
    one = synth.random_problem(synth.rng(6002), 1, 1000, 4096, 2, 2, with_scales=True)
    _check(big, what="1100x2000x3000 W4A4")
    _check(small, what="70x300x500 W2A3")
    _check(one, what="1x1000x4096 W2A2")


def test_noalloc_stream_k_counters_cleared_between_calls():
    # a forced persistent grid shares tiles through counters and partial tiles
    # in the array; two calls in a row, the second smaller
    cfg = apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2, 7, 3)
    big = synth.random_problem(synth.rng(6003), 600, 700, 2000, 3, 5, with_scales=True)
    small = synth.random_problem(synth.rng(6004), 200, 300, 900, 3, 5, with_scales=True)
    assert apt.apt_gemm_workspace_bytes(600, 700, 2000, 3, 5, cfg) <= SCRATCH_BYTES
    _check(big, cfg, "600x700x2000 stream-K")
    _check(small, cfg, "200x300x900 stream-K")
    _check(big, cfg, "600x700x2000 stream-K again")


def test_noalloc_workload_shapes():
    # the W4A4 prefill and a down projection of the sweep, in the selected config
    for prob in (synth.w4a4_prefill(), synth.sweep_down(3)):
        prob.w_scale = synth.scales(synth.rng(6005), prob.N, 0.005, 0.05)
        prob.a_scale = synth.scales(synth.rng(6006), prob.M, 0.01, 0.1)
        _check(prob, what=prob.name)
