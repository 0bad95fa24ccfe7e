"""GPU tests of the library's runtime behaviour: launch status checking and
streams other than torch's current one."""
import ctypes

import numpy as np
import pytest

import paper_2508_19087_amd as apt
import synth
from gpu_util import assert_fp16_ok, assert_int32_equal, dev, oracle_full

pytestmark = pytest.mark.gpu


def _hip_runtime():
    """The HIP runtime library this process already loaded (through torch), opened
    by its exact path so that ctypes returns the same instance, not a second copy."""
    import torch
    torch.cuda.init()
    with open("/proc/self/maps") as f:
        paths = sorted({line.split()[-1] for line in f if "libamdhip64" in line})
    assert paths, "libamdhip64 is not loaded"
    L = ctypes.CDLL(paths[0])
    L.hipSetDevice.argtypes = [ctypes.c_int]
    L.hipSetDevice.restype = ctypes.c_int
    L.hipGetLastError.restype = ctypes.c_int
    L.hipPeekAtLastError.restype = ctypes.c_int
    return L


def test_stale_runtime_error_is_not_reported_as_launch_failure():
    """A failed, unrelated runtime call earlier in the thread (hipSetDevice on a
    device that does not exist) leaves the runtime's last-error state set; the
    library's launches check their own status, so packing and every route's GEMM
    still return APT_OK and the right result."""
    import torch
    hip = _hip_runtime()
    prob = synth.random_problem(synth.rng(5000), 40, 300, 700, 2, 3, with_scales=True)
    a_codes, w_codes = dev(prob.a_codes), dev(prob.w_codes)
    torch.cuda.synchronize()
    try:
        assert hip.hipSetDevice(1 << 20) != 0
        assert hip.hipPeekAtLastError() != 0  # the stale error is in place
        a = apt.pack(a_codes, prob.q, activations=True)
        w = apt.pack(w_codes, prob.p)
        want = oracle_full(prob)
        for route in (apt.APT_ROUTE_XOR, apt.APT_ROUTE_INT8_MFMA, apt.APT_ROUTE_PM1_MFMA):
            cfg = apt.apt_config_t.make(route)
            if route == apt.APT_ROUTE_INT8_MFMA:
                cfg = apt.apt_config_t.make(route, 128, 128, 128, 2, 2, 0, 3)
            c32, _ = apt.gemm(a, w, cfg=cfg)
            torch.cuda.synchronize()
            assert_int32_equal(c32.cpu().numpy(), want, "route %d after a stale error" % route)
        assert apt.apt_last_hip_error() == 0
    finally:
        hip.hipGetLastError()  # clear it, so that torch's own launch checks do not trip on it


def test_side_stream():
    """Packing and the GEMM on a stream other than torch's current one: the
    binding allocates outputs and workspace on that stream."""
    import torch
    prob = synth.random_problem(synth.rng(5001), 700, 1000, 1500, 4, 4, with_scales=True)
    want = oracle_full(prob)
    a_codes, w_codes = dev(prob.a_codes), dev(prob.w_codes)
    sa, sw = dev(prob.a_scale), dev(prob.w_scale)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    outs = []
    for _ in range(3):
        a = apt.pack(a_codes, prob.q, activations=True, stream=side)
        w = apt.pack(w_codes, prob.p, stream=side)
        c32, c16 = apt.gemm(a, w, a_scale=sa, w_scale=sw, out_fp16=True, stream=side)
        outs.append((c32, c16))
        # work on the current stream in the meantime may reuse freed blocks
        junk = torch.empty(64 << 20, dtype=torch.uint8, device="cuda").fill_(0xA5)
        del junk
    side.synchronize()
    for c32, c16 in outs:
        assert_int32_equal(c32.cpu().numpy(), want, "side stream")
        assert_fp16_ok(c16.cpu().numpy(), want, prob, "side stream")
    assert np.array_equal(outs[0][0].cpu().numpy(), outs[-1][0].cpu().numpy())
