"""GPU: independent calls in flight on several streams at once.

The library keeps no per-call state outside the caller's buffers (the
workspace carries the fragments, partial tiles and arrival counters), so two
batches whose GEMMs overlap on two streams, each with its own output and
workspace, and a decode chain on a third stream give the same results as the
same calls one after another.  Checked bit for bit against serial calls and
the oracle's matmul (Sec. III-B: the exact product of the bipolar values),
for the int8 route with one workgroup per tile, with a persistent round that
chains leftover tiles, and with stream-K tiles shared by several workgroups.
"""
import numpy as np
import pytest

import paper_2508_19087_amd as apt
from gpu_util import assert_int32_equal, dev
from oracle import oracle as ref

pytestmark = pytest.mark.gpu

M, N, K, P, Q = 384, 1536, 1000, 4, 4


def _codes(rng, rows, cols, bits):
    return rng.integers(-(1 << (bits - 1)), 1 << (bits - 1), (rows, cols), dtype=np.int8)


@pytest.mark.parametrize("grid", [0, 256, 7])
def test_two_batches_in_flight_match_serial_and_oracle(grid):
    import torch
    rng = np.random.default_rng(2508 + grid)
    w_codes = _codes(rng, N, K, P)
    x = [_codes(rng, M, K, Q) for _ in range(2)]
    w = apt.pack(dev(w_codes), P)
    cfg = apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 256, 128, 128, 4, 1, grid, 3)
    nbytes = apt.apt_gemm_act_workspace_bytes(M, N, K, P, Q, apt.APT_ACT_CODES, cfg)
    streams = [torch.cuda.current_stream(), torch.cuda.Stream()]
    srcs = [dev(xi) for xi in x]
    outs = [torch.full((M, N), -1, dtype=torch.int32, device="cuda") for _ in range(2)]
    wss = [torch.full((max(nbytes, 16),), 0x5A, dtype=torch.uint8, device="cuda") for _ in range(2)]

    def call(k, out, ws):
        st = apt.apt_gemm_act(M, N, K, P, Q, srcs[k].data_ptr(), apt.APT_ACT_CODES, w.data.data_ptr(),
                              w.rowsum.data_ptr(), out.data_ptr(), None, None, None, None, cfg,
                              ws.data_ptr(), nbytes, streams[k].cuda_stream)
        assert st == apt.APT_OK, apt.status_string(st)

    # serial reference through the same library, on one stream
    serial = []
    for k in range(2):
        o = torch.empty((M, N), dtype=torch.int32, device="cuda")
        ws = torch.empty((max(nbytes, 16),), dtype=torch.uint8, device="cuda")
        st = apt.apt_gemm_act(M, N, K, P, Q, srcs[k].data_ptr(), apt.APT_ACT_CODES, w.data.data_ptr(),
                              w.rowsum.data_ptr(), o.data_ptr(), None, None, None, None, cfg,
                              ws.data_ptr(), nbytes, streams[0].cuda_stream)
        assert st == apt.APT_OK
        torch.cuda.synchronize()
        serial.append(o.cpu().numpy())
    # several rounds of the two batches alternating between the two streams
    torch.cuda.synchronize()
    for _ in range(6):
        for k in range(2):
            call(k, outs[k], wss[k])
    torch.cuda.synchronize()
    for k in range(2):
        got = outs[k].cpu().numpy()
        np.testing.assert_array_equal(got, serial[k])
        assert_int32_equal(got, ref.gemm(x[k], w_codes, P, Q), "batch %d, grid %d" % (k, grid))


def test_prefill_beside_decode_chain():
    """A prefill batch on one stream and M = 1 decode GEMMs (XOR route, one
    launch from the token's codes) on another, overlapping: both equal their
    serial results."""
    import torch
    rng = np.random.default_rng(77)
    wp_codes = _codes(rng, N, K, P)
    wd_codes = _codes(rng, 2048, K, 2)
    xp = _codes(rng, M, K, Q)
    xd = _codes(rng, 1, K, 2)
    wp, wd = apt.pack(dev(wp_codes), P), apt.pack(dev(wd_codes), 2)
    side = torch.cuda.Stream()
    main = torch.cuda.current_stream()
    sp, sd = dev(xp), dev(xd)
    nbytes = apt.apt_gemm_act_workspace_bytes(M, N, K, P, Q, apt.APT_ACT_CODES, None)
    ws = torch.empty((max(nbytes, 16),), dtype=torch.uint8, device="cuda")
    cp = torch.full((M, N), -1, dtype=torch.int32, device="cuda")
    cd = torch.full((1, 2048), -1, dtype=torch.int32, device="cuda")

    def prefill():
        st = apt.apt_gemm_act(M, N, K, P, Q, sp.data_ptr(), apt.APT_ACT_CODES, wp.data.data_ptr(),
                              wp.rowsum.data_ptr(), cp.data_ptr(), None, None, None, None, None,
                              ws.data_ptr(), nbytes, main.cuda_stream)
        assert st == apt.APT_OK

    def decode():
        st = apt.apt_gemm_decode(1, 2048, K, 2, 2, sd.data_ptr(), apt.APT_ACT_CODES, wd.data.data_ptr(),
                                 cd.data_ptr(), None, None, None, None, None, side.cuda_stream)
        assert st == apt.APT_OK

    torch.cuda.synchronize()  # the buffers above were filled on the main stream
    for _ in range(4):
        prefill()
        for _ in range(3):
            decode()
    torch.cuda.synchronize()
    got_p, got_d = cp.cpu().numpy(), cd.cpu().numpy()
    assert_int32_equal(got_p, ref.gemm(xp, wp_codes, P, Q), "prefill")
    assert_int32_equal(got_d, ref.gemm(xd, wd_codes, 2, 2), "decode")
