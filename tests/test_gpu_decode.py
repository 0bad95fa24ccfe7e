"""GPU parity of apt_gemm_decode, the XOR-route decode GEMM that converts its
activation row inside the kernel (Sec. III-A conversion, for fp16 input after
the per-row quantizer; Sec. IV-A planes; Sec. III-B XOR recovery):

* int8 codes in: int32 bit-exact against the oracle's matmul of the bipolar
  values, fp16 within the epilogue tolerance;
* fp16 in: the row scales bit-exact against the oracle's quantize_fp16, the
  int32 output bit-exact against the matmul of the oracle's codes, fp16 within
  tolerance of the exact product with the oracle's scales;
* both bit-identical to the packer followed by apt_gemm on the XOR route.

Shapes cover ragged K (the row's tail inside a lane's 16 elements), rows longer
than the four rounds a lane holds in registers, every launch shape the config
can force, unaligned sources (element-wise loads), all 64 (p, q) pairs, the
largest K whose planes fit in LDS, and the decode workloads at full size."""
import numpy as np
import pytest

import paper_2508_19087_amd as apt
import synth
from gpu_util import assert_int32_equal, dev
from oracle import oracle as ref

pytestmark = pytest.mark.gpu


def _stream():
    import torch
    return torch.cuda.current_stream().cuda_stream


def decode_raw(x, q, w, cfg=None, a_scale=None, w_scale=None, fp16=False, offset=0):
    """apt_gemm_decode on x (int8 codes or fp16 values, numpy [M][K]) placed
    `offset` elements into a fresh device buffer.  Returns (status, c32, c16,
    scale bits) as numpy (outputs prefilled with sentinels)."""
    import torch
    M, K = x.shape
    N = w.rows
    tdt = torch.float16 if x.dtype == np.float16 else torch.int8
    buf = torch.zeros(x.size + 64, dtype=tdt, device="cuda")
    view = buf[offset:offset + x.size]
    view.copy_(torch.from_numpy(np.ascontiguousarray(x).ravel()))
    c32 = torch.full((M, N), -12345, dtype=torch.int32, device="cuda")
    c16 = torch.full((M, N), 0x7E00, dtype=torch.int16, device="cuda") if fp16 else None
    fp16_src = x.dtype == np.float16
    sc = torch.full((M,), 0x7E00, dtype=torch.int16, device="cuda") if fp16_src else None
    sa = dev(a_scale) if (a_scale is not None and not fp16_src) else None
    sw = dev(w_scale) if w_scale is not None else None
    st = apt.apt_gemm_decode(M, N, K, w.bits, q, view.data_ptr(),
                             apt.APT_ACT_FP16 if fp16_src else apt.APT_ACT_CODES,
                             w.data.data_ptr(), c32.data_ptr(),
                             sa.data_ptr() if sa is not None else None,
                             sw.data_ptr() if sw is not None else None,
                             c16.data_ptr() if c16 is not None else None,
                             sc.data_ptr() if sc is not None else None, cfg, _stream())
    torch.cuda.synchronize()
    return (st, c32.cpu().numpy(),
            c16.cpu().numpy().view(np.float16) if c16 is not None else None,
            sc.cpu().numpy().view(np.uint16) if sc is not None else None)


def check_codes(M, N, K, p, q, cfg=None, offset=0, seed=0, fp16=True, against_unfused=False):
    import torch
    g = synth.rng(90, seed, M, N, K, p, q)
    a_codes = synth.uniform_codes(g, M, K, q)
    w_codes = synth.uniform_codes(g, N, K, p)
    a_scale = synth.scales(g, M, *synth.A_SCALE_RANGE)
    w_scale = synth.scales(g, N, *synth.W_SCALE_RANGE)
    w = apt.pack(dev(w_codes), p)
    st, c32, c16, _ = decode_raw(a_codes, q, w, cfg, a_scale, w_scale, fp16, offset)
    what = "codes %dx%dx%d W%dA%d cfg=%s off=%d" % (M, N, K, p, q, cfg and cfg.as_dict(), offset)
    assert st == apt.APT_OK, what + ": " + apt.status_string(st)
    C = ref.gemm(a_codes, w_codes, p, q)
    assert_int32_equal(c32, C, what)
    if fp16:
        E, _ = ref.epilogue(C, a_scale, w_scale)
        ok = ref.fp16_close(c16, E)
        assert ok.all(), "%s: %d fp16 outputs outside tolerance" % (what, (~ok).sum())
    if against_unfused:
        a = apt.pack(dev(a_codes), q, activations=True)
        u32, u16 = apt.gemm(a, w, a_scale=dev(a_scale), w_scale=dev(w_scale), out_fp16=fp16,
                            cfg=apt.apt_config_t.make(apt.APT_ROUTE_XOR))
        torch.cuda.synchronize()
        assert np.array_equal(c32, u32.cpu().numpy()), what + ": differs from the unfused path"
        if fp16:
            assert np.array_equal(c16.view(np.uint16), u16.cpu().numpy().view(np.uint16)), what


def check_fp16(M, N, K, p, q, cfg=None, offset=0, seed=0, x=None, against_unfused=False):
    import torch
    g = synth.rng(91, seed, M, N, K, p, q)
    if x is None:
        x = synth.fp16_activations(g, M, K)
    w_codes = synth.uniform_codes(g, N, K, p)
    w_scale = synth.scales(g, N, *synth.W_SCALE_RANGE)
    w = apt.pack(dev(w_codes), p)
    st, c32, c16, sc = decode_raw(x, q, w, cfg, None, w_scale, True, offset)
    what = "fp16 %dx%dx%d W%dA%d cfg=%s off=%d" % (M, N, K, p, q, cfg and cfg.as_dict(), offset)
    assert st == apt.APT_OK, what + ": " + apt.status_string(st)
    codes, s16 = ref.quantize_fp16(x, q)
    assert np.array_equal(sc, s16.view(np.uint16)), "%s: scales differ at rows %s" % (
        what, np.flatnonzero(sc != s16.view(np.uint16))[:8])
    C = ref.gemm(codes, w_codes, p, q)
    assert_int32_equal(c32, C, what)
    E, _ = ref.epilogue(C, s16, w_scale)
    ok = ref.fp16_close(c16, E)
    assert ok.all(), "%s: %d fp16 outputs outside tolerance" % (what, (~ok).sum())
    if against_unfused:
        a, a_scale = apt.quantize_pack(dev(x), q)
        u32, u16 = apt.gemm(a, w, a_scale=a_scale, w_scale=dev(w_scale), out_fp16=True,
                            cfg=apt.apt_config_t.make(apt.APT_ROUTE_XOR))
        torch.cuda.synchronize()
        assert np.array_equal(c32, u32.cpu().numpy()), what + ": differs from the unfused path"
        assert np.array_equal(c16.view(np.uint16), u16.cpu().numpy().view(np.uint16)), what


# K: one element, inside the first lane, ragged across lanes, a whole chunk,
# ragged chunks, 5 and 7 register rounds of one wave (more than the 4 a lane
# holds), the K-split form (8 or more chunk rounds) with 3 rounds of 4 waves.
RAGGED_K = [1, 15, 17, 33, 128, 129, 1000, 4096, 5000, 7000, 7169, 11008]


@pytest.mark.parametrize("K", RAGGED_K)
@pytest.mark.parametrize("M", [1, 3, 8])
def test_decode_codes_ragged(M, K):
    check_codes(M, 70, K, 2, 4, seed=1)


@pytest.mark.parametrize("K", RAGGED_K)
@pytest.mark.parametrize("M", [1, 5])
def test_decode_fp16_ragged(M, K):
    check_fp16(M, 70, K, 2, 4, seed=2)


@pytest.mark.parametrize("p", range(1, 9))
@pytest.mark.parametrize("q", range(1, 9))
def test_decode_all_bit_pairs(p, q):
    check_codes(2, 33, 777, p, q, seed=3)
    check_fp16(2, 33, 777, p, q, seed=3)


XOR_SHAPES = ([dict(mt=mt, waves_m=w, waves_n=1) for mt in (1, 8) for w in (1, 2, 4)] +
              [dict(mt=mt, waves_n=b) for mt in (1, 8) for b in (2, 4)])


@pytest.mark.parametrize("shape", XOR_SHAPES, ids=lambda d: "-".join("%s%d" % kv for kv in d.items()))
@pytest.mark.parametrize("K", [100, 4096, 7000, 11008])
@pytest.mark.parametrize("M", [3, 8])
def test_decode_forced_shapes(shape, K, M):
    """One or eight activation rows per block row (mt), each wave shape."""
    cfg = apt.apt_config_t.make(apt.APT_ROUTE_XOR, **shape)
    check_codes(M, 200, K, 3, 3, cfg=cfg, seed=4)
    check_fp16(M, 200, K, 3, 3, cfg=cfg, seed=4)


@pytest.mark.parametrize("offset", [1, 3, 8])
@pytest.mark.parametrize("K", [64, 4096, 1000])
def test_decode_unaligned_source(offset, K):
    """Sources that are not 16-byte aligned, or K % 16 != 0, take the
    element-wise loads; the result does not change."""
    check_codes(2, 48, K, 2, 2, offset=offset, seed=5)
    check_fp16(2, 48, K, 2, 2, offset=offset, seed=5)


def test_decode_special_fp16_rows():
    """Zero rows (scale 0), signed zeros, subnormal-only rows, fp16 extremes
    and exact ties of the quantizer, through the fused kernel."""
    K, q = 320, 3
    L = 2 ** q - 1
    x = np.zeros((6, K), np.float16)
    x[1, ::2] = np.float16(-0.0)
    x[2] = (np.arange(K) % 7 - 3).astype(np.float16) * np.float16(2.0 ** -24)
    x[3, :4] = [65504.0, -65504.0, 1.0, -1.0]
    s = 2.0 ** -3
    ties = np.arange(-L + 1, L, 2, dtype=np.float64)
    x[4, :len(ties)] = (ties * s).astype(np.float16)
    x[4, len(ties)] = np.float16(L * s)
    x[5] = synth.fp16_activations(synth.rng(92), 1, K)[0]
    check_fp16(6, 40, K, 2, q, x=x)


def test_decode_matches_unfused_path():
    """Bit-identical to packer + apt_gemm (XOR route), codes and fp16."""
    for M, K in [(1, 4096), (2, 4096), (4, 11008), (8, 1000), (8, 4096)]:
        check_codes(M, 1024, K, 2, 4, seed=6, against_unfused=True)
        check_fp16(M, 1024, K, 2, 4, seed=6, against_unfused=True)


def test_decode_largest_k_in_lds():
    """q = 8 at K = 65536: the row's planes fill the 64 KB LDS copy; one
    element more is refused before any launch."""
    check_codes(1, 16, 65536, 1, 8, seed=7, fp16=False)
    check_fp16(1, 16, 65536, 1, 8, seed=7)
    import torch
    w = apt.pack(dev(synth.uniform_codes(synth.rng(93), 16, 65537, 1)), 1)
    x = torch.zeros((1, 65537), dtype=torch.int8, device="cuda")
    c = torch.empty((1, 16), dtype=torch.int32, device="cuda")
    st = apt.apt_gemm_decode(1, 16, 65537, 1, 8, x.data_ptr(), apt.APT_ACT_CODES, w.data.data_ptr(),
                             c.data_ptr(), None, None, None, None, None, _stream())
    assert st == apt.APT_ERR_UNSUPPORTED


def test_decode_eight_rows_lds_limit():
    """Eight rows at q = 8: K = 7168 is the longest whose eight-row copy fits
    in LDS; past it the library converts one row per block row (mt = 0), and a
    forced mt = 8 is refused."""
    mt8 = apt.apt_config_t.make(apt.APT_ROUTE_XOR, mt=8)
    check_codes(8, 64, 7168, 2, 8, cfg=mt8, seed=9, against_unfused=True)
    check_fp16(8, 64, 7168, 2, 8, cfg=mt8, seed=9, against_unfused=True)
    check_codes(8, 16384, 7169, 2, 8, seed=9)   # 2048 row groups: mt = 8 would be chosen
    check_fp16(8, 64, 7169, 2, 8, seed=9)
    import torch
    x = torch.zeros((8, 7169), dtype=torch.int8, device="cuda")
    w = apt.pack(dev(synth.uniform_codes(synth.rng(95), 64, 7169, 2)), 2)
    c = torch.empty((8, 64), dtype=torch.int32, device="cuda")
    st = apt.apt_gemm_decode(8, 64, 7169, 2, 8, x.data_ptr(), apt.APT_ACT_CODES, w.data.data_ptr(),
                             c.data_ptr(), None, None, None, None,
                             apt.apt_config_t.make(apt.APT_ROUTE_XOR, mt=8), _stream())
    assert st == apt.APT_ERR_UNSUPPORTED


def test_decode_int32_only_and_fp16_only():
    """Either output alone; fp16 source without a scale output pointer."""
    import torch
    M, N, K, p, q = 2, 96, 512, 2, 4
    g = synth.rng(94)
    x = synth.fp16_activations(g, M, K)
    w_codes = synth.uniform_codes(g, N, K, p)
    w_scale = synth.scales(g, N, *synth.W_SCALE_RANGE)
    w = apt.pack(dev(w_codes), p)
    xd = dev(x)
    c16 = torch.empty((M, N), dtype=torch.float16, device="cuda")
    st = apt.apt_gemm_decode(M, N, K, p, q, xd.data_ptr(), apt.APT_ACT_FP16, w.data.data_ptr(),
                             None, None, dev(w_scale).data_ptr(), c16.data_ptr(), None, None,
                             _stream())
    assert st == apt.APT_OK
    torch.cuda.synchronize()
    codes, s16 = ref.quantize_fp16(x, q)
    E, _ = ref.epilogue(ref.gemm(codes, w_codes, p, q), s16, w_scale)
    assert ref.fp16_close(c16.cpu().numpy(), E).all()
    c32, _, sc = apt.gemm_decode(xd, q, w)
    torch.cuda.synchronize()
    assert_int32_equal(c32.cpu().numpy(), ref.gemm(codes, w_codes, p, q), "binding")
    assert np.array_equal(sc.cpu().numpy().view(np.uint16), s16.view(np.uint16))


@pytest.mark.parametrize("M", [1, 4, 8])
@pytest.mark.parametrize("N,K", [(4096, 4096), (11008, 4096), (4096, 11008)])
def test_decode_full_size(M, N, K):
    """The decode workloads (W2A2 and the W2A4 layer shapes) at full size, in
    the launch shape the library chooses, every output compared."""
    check_codes(M, N, K, 2, 2, seed=8)
    check_fp16(M, N, K, 2, 4, seed=8)
