"""GPU parity of apt_gemm_act, the GEMM from unpacked activations (int8 codes,
or fp16 values quantized per row inside the call; Sec. III-A conversion and the
bipolar form of the linear quantizer), for every route and launch shape the
config can force:

* int32 bit-exact against the oracle's matmul of the bipolar values (for fp16
  input, of the oracle's quantize_fp16 codes), fp16 within the epilogue
  tolerance, fp16 row scales bit-exact;
* bit-identical to the packer followed by apt_gemm in the same config.

The int8 MFMA route takes the rows straight into its operand fragments
(act_frag.hip), the XOR route's decode sizes the fused GEMV, every other route
the packer into the workspace; all three are covered, with ragged M and K, rows
past the last 32-row block, the padding chunk of an odd chunk count, unaligned
sources and the prefill workload at full size."""
import numpy as np
import pytest

import paper_2508_19087_amd as apt
import synth
from gpu_util import assert_int32_equal, dev, forced_configs
from oracle import oracle as ref

pytestmark = pytest.mark.gpu


def _stream():
    import torch
    return torch.cuda.current_stream().cuda_stream


def run_act(x, q, w, cfg=None, a_scale=None, w_scale=None, fp16_out=True, offset=0):
    """apt_gemm_act on x (numpy int8 codes or fp16 values) placed `offset`
    elements into a fresh device buffer; (status, c32, c16, scale bits)."""
    import torch
    M, K = x.shape
    N = w.rows
    fp16_src = x.dtype == np.float16
    kind = apt.APT_ACT_FP16 if fp16_src else apt.APT_ACT_CODES
    tdt = torch.float16 if fp16_src else torch.int8
    buf = torch.zeros(x.size + 64, dtype=tdt, device="cuda")
    view = buf[offset:offset + x.size]
    view.copy_(torch.from_numpy(np.ascontiguousarray(x).ravel()))
    c32 = torch.full((M, N), -12345, dtype=torch.int32, device="cuda")
    c16 = torch.full((M, N), 0x7E00, dtype=torch.int16, device="cuda") if fp16_out else None
    sc = torch.full((M,), 0x7E00, dtype=torch.int16, device="cuda") if fp16_src else None
    sa = dev(a_scale) if (a_scale is not None and not fp16_src) else None
    sw = dev(w_scale) if w_scale is not None else None
    nbytes = apt.apt_gemm_act_workspace_bytes(M, N, K, w.bits, q, kind, cfg)
    ws = torch.full((max(nbytes, 16),), 0x5A, dtype=torch.uint8, device="cuda")
    st = apt.apt_gemm_act(M, N, K, w.bits, q, view.data_ptr(), kind, w.data.data_ptr(),
                          w.rowsum.data_ptr(), c32.data_ptr(),
                          sa.data_ptr() if sa is not None else None,
                          sw.data_ptr() if sw is not None else None,
                          c16.data_ptr() if c16 is not None else None,
                          sc.data_ptr() if sc is not None else None, cfg,
                          ws.data_ptr() if nbytes else None, nbytes, _stream())
    torch.cuda.synchronize()
    return (st, c32.cpu().numpy(),
            c16.cpu().numpy().view(np.float16) if c16 is not None else None,
            sc.cpu().numpy().view(np.uint16) if sc is not None else None)


def unfused(x, q, w, cfg, a_scale, w_scale):
    """The same problem through the packer and apt_gemm."""
    import torch
    if x.dtype == np.float16:
        a, sa = apt.quantize_pack(dev(x), q)
    else:
        a, sa = apt.pack(dev(x), q, activations=True), dev(a_scale)
    c32, c16 = apt.gemm(a, w, a_scale=sa, w_scale=dev(w_scale), out_fp16=True, cfg=cfg)
    torch.cuda.synchronize()
    return c32.cpu().numpy(), c16.cpu().numpy().view(np.float16)


def check(M, N, K, p, q, cfg=None, fp16_src=False, seed=0, offset=0, against_unfused=True, what=""):
    g = synth.rng(96, seed, M, N, K, p, q, int(fp16_src))
    if fp16_src:
        x = synth.fp16_activations(g, M, K)
        codes, s16 = ref.quantize_fp16(x, q)
        a_scale = None
    else:
        x = codes = synth.uniform_codes(g, M, K, q)
        a_scale = s16 = synth.scales(g, M, *synth.A_SCALE_RANGE)
    w_codes = synth.uniform_codes(g, N, K, p)
    w_scale = synth.scales(g, N, *synth.W_SCALE_RANGE)
    w = apt.pack(dev(w_codes), p)
    st, c32, c16, sc = run_act(x, q, w, cfg, a_scale, w_scale, True, offset)
    what = "%s %s %dx%dx%d W%dA%d off=%d" % (what, "fp16" if fp16_src else "codes", M, N, K, p, q,
                                              offset)
    assert st == apt.APT_OK, what + ": " + apt.status_string(st)
    C = ref.gemm(codes, w_codes, p, q)
    assert_int32_equal(c32, C, what)
    E, _ = ref.epilogue(C, s16, w_scale)
    ok = ref.fp16_close(c16, E)
    assert ok.all(), "%s: %d fp16 outputs outside tolerance" % (what, (~ok).sum())
    if fp16_src:
        assert np.array_equal(sc, s16.view(np.uint16)), what + ": scales differ"
    if against_unfused:
        u32, u16 = unfused(x, q, w, cfg, a_scale, w_scale)
        assert np.array_equal(c32, u32), what + ": int32 differs from packer + apt_gemm"
        assert np.array_equal(c16.view(np.uint16), u16.view(np.uint16)), \
            what + ": fp16 differs from packer + apt_gemm"


@pytest.mark.parametrize("p,q", [(1, 1), (2, 4), (3, 3), (8, 8)])
def test_act_every_forced_config(p, q):
    """Every config the library can be forced to (XOR shapes, int8 tiles with
    their grids and split launches, FP4/FP6/FP8 operands, +-1 planes), on a
    ragged problem, codes and fp16."""
    M, N, K = 70, 300, 1000
    for name, cfg in forced_configs(p, q, N, K):
        for fp16_src in (False, True):
            check(M, N, K, p, q, cfg=cfg, fp16_src=fp16_src, seed=1, what=name)


@pytest.mark.parametrize("M", [1, 5, 8, 9, 31, 32, 33, 64, 100])
@pytest.mark.parametrize("K", [1, 100, 128, 129, 384, 4096, 4097])
def test_act_int8_fragments_ragged(M, K):
    """The fragment writer: ragged M (rows past the last block) and K (the
    padding chunk of an odd chunk count, elements past K), all bit widths of
    the activations through the int8 route."""
    cfg = apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2, 0, 3)
    for q in (1, 4, 7, 8):
        check(M, 96, K, 2, q, cfg=cfg, seed=2, what="int8 q=%d" % q)
    check(M, 96, K, 3, 5, cfg=cfg, fp16_src=True, seed=2, what="int8 fp16")


@pytest.mark.parametrize("offset", [1, 3, 8])
def test_act_unaligned_source(offset):
    cfg = apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2, 0, 3)
    for K in (512, 1000):
        check(40, 128, K, 2, 4, cfg=cfg, offset=offset, seed=3, what="int8")
        check(40, 128, K, 2, 4, cfg=cfg, fp16_src=True, offset=offset, seed=3, what="int8")
        check(40, 128, K, 2, 4, offset=offset, seed=3, what="auto")


@pytest.mark.parametrize("M,N,K,p,q", [(1, 4096, 4096, 2, 2), (8, 11008, 4096, 2, 2),
                                       (16, 512, 512, 1, 2), (512, 4096, 11008, 1, 1),
                                       (1024, 4096, 4096, 2, 4)])
def test_act_selected_config(M, N, K, p, q):
    """The selected config (fused XOR at decode sizes, XOR with packing for
    small problems, FP4 or int8 MFMA for the larger ones)."""
    check(M, N, K, p, q, seed=4, what="selected")
    check(M, N, K, p, q, fp16_src=True, seed=4, what="selected")


def test_act_prefill_full_size():
    """The W4A4 prefill (2048x11008x4096) from codes and from fp16 in the
    selected config, every output compared."""
    prob = synth.w4a4_prefill()
    w = apt.pack(dev(prob.w_codes), prob.p)
    st, c32, _, _ = run_act(prob.a_codes, prob.q, w, fp16_out=False)
    assert st == apt.APT_OK
    assert_int32_equal(c32, ref.gemm(prob.a_codes, prob.w_codes, prob.p, prob.q), prob.name)
    x = synth.fp16_activations(synth.rng(97), prob.M, prob.K)
    st, c32, _, sc = run_act(x, prob.q, w, fp16_out=False)
    assert st == apt.APT_OK
    codes, s16 = ref.quantize_fp16(x, prob.q)
    assert np.array_equal(sc, s16.view(np.uint16))
    assert_int32_equal(c32, ref.gemm(codes, prob.w_codes, prob.p, prob.q), prob.name + " fp16")


def test_act_binding_and_workspace():
    """The binding's helper, and a workspace one byte short refused."""
    import torch
    M, N, K, p, q = 64, 256, 1024, 2, 4
    g = synth.rng(98)
    x = synth.uniform_codes(g, M, K, q)
    w_codes = synth.uniform_codes(g, N, K, p)
    w = apt.pack(dev(w_codes), p)
    c32, _, _ = apt.gemm_act(dev(x), q, w)
    torch.cuda.synchronize()
    assert_int32_equal(c32.cpu().numpy(), ref.gemm(x, w_codes, p, q), "binding")
    cfg = apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2, 0, 3)
    nb = apt.apt_gemm_act_workspace_bytes(M, N, K, p, q, apt.APT_ACT_CODES, cfg)
    assert nb > 0
    ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    xd = dev(x)
    c = torch.empty((M, N), dtype=torch.int32, device="cuda")
    st = apt.apt_gemm_act(M, N, K, p, q, xd.data_ptr(), apt.APT_ACT_CODES, w.data.data_ptr(),
                          w.rowsum.data_ptr(), c.data_ptr(), None, None, None, None, cfg,
                          ws.data_ptr(), nb - 1, _stream())
    assert st == apt.APT_ERR_WORKSPACE
    st = apt.apt_gemm_act(M, N, K, p, q, xd.data_ptr(), apt.APT_ACT_CODES, w.data.data_ptr(),
                          None, c.data_ptr(), None, None, None, None, cfg,
                          ws.data_ptr(), nb, _stream())
    assert st == apt.APT_ERR_INVALID_ARG   # the MFMA routes need the weights' row sums


def test_act_special_fp16_rows():
    """Zero rows (scale 0), signed zeros, subnormal-only rows, fp16 extremes
    and exact ties of the quantizer, through the fragment writer (int8 route)
    and the packer path (XOR route, M > 8): int32 against the oracle's codes,
    scales bit-exact."""
    import torch
    K, q, p, N = 320, 3, 2, 64
    L = 2 ** q - 1
    x = np.zeros((12, K), np.float16)
    x[1, ::2] = np.float16(-0.0)
    x[2] = (np.arange(K) % 7 - 3).astype(np.float16) * np.float16(2.0 ** -24)
    x[3, :4] = [65504.0, -65504.0, 1.0, -1.0]
    s = 2.0 ** -3
    ties = np.arange(-L + 1, L, 2, dtype=np.float64)
    x[4, :len(ties)] = (ties * s).astype(np.float16)
    x[4, len(ties)] = np.float16(L * s)
    x[5:] = synth.fp16_activations(synth.rng(99), 7, K)
    w_codes = synth.uniform_codes(synth.rng(100), N, K, p)
    w = apt.pack(dev(w_codes), p)
    codes, s16 = ref.quantize_fp16(x, q)
    want = ref.gemm(codes, w_codes, p, q)
    for cfg in (apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2, 0, 3),
                apt.apt_config_t.make(apt.APT_ROUTE_XOR)):
        c32, _, sc = apt.gemm_act(dev(x), q, w, cfg=cfg)
        torch.cuda.synchronize()
        assert np.array_equal(sc.cpu().numpy().view(np.uint16), s16.view(np.uint16)), cfg.route
        assert_int32_equal(c32.cpu().numpy(), want, "special rows route %d" % cfg.route)
