"""Host-side checks of the C ABI (no kernel launches): every declared symbol is
exported, sizes and selector outputs are as documented, and invalid arguments
are rejected with the documented status before anything reaches the GPU."""
import ctypes

import pytest

import paper_2508_19087_amd as apt
import synth


def test_exports_every_declared_symbol():
    names = apt.header_functions()
    assert set(names) == {"apt_packed_bytes", "apt_pack_weights", "apt_quantize_pack_activations",
                          "apt_quantize_pack_activations_fp16", "apt_select_config", "apt_gemm_workspace_bytes", "apt_gemm",
                          "apt_gemm_affine", "apt_search_workspace_bytes", "apt_search_config",
                          "apt_config_table_clear", "apt_config_table_size", "apt_last_hip_error",
                          "apt_gemm_noalloc", "apt_gemm_decode", "apt_gemm_act",
                          "apt_gemm_act_workspace_bytes",
                          "apt_status_string"}
    L = apt.lib()
    for n in names:
        assert hasattr(L, n), n


@pytest.mark.parametrize("rows,K,bits,want", [
    (1, 1, 1, 8 * 16), (1, 128, 1, 8 * 16), (1, 129, 1, 8 * 32), (3, 4096, 2, 8 * 32 * 2 * 16),
    (8, 1, 3, 8 * 3 * 16), (9, 1, 3, 16 * 3 * 16),
    (11008, 4096, 4, 11008 * 32 * 4 * 16), (2, 11008, 8, 8 * 86 * 8 * 16),
    (0, 5, 1, 0), (5, 0, 1, 0), (5, 5, 0, 0), (5, 5, 9, 0)])
def test_packed_bytes(rows, K, bits, want):
    assert apt.apt_packed_bytes(rows, K, bits) == want


def test_status_strings():
    for s in range(5):
        assert apt.status_string(s)
    assert apt.status_string(99) == "unknown status"


def test_last_hip_error_starts_clear():
    # validation failures never touch the runtime, so they leave it at 0
    assert apt.apt_gemm(0, 1, 1, 1, 1, None, None, None, None, None, None, None, None, None, None,
                        0, None) == apt.APT_ERR_INVALID_ARG
    assert apt.apt_last_hip_error() == 0


def _shapes():
    out = [(16, 512, 512, 1, 2), (2048, 11008, 4096, 4, 4)]
    for M in (1, 4, 8):
        out += [(M, 4096, 4096, 2, 2), (M, 11008, 4096, 2, 2)]
    for p, q in synth.SWEEP_BITS:
        out.append((512, 4096, 11008, p, q))
    for name, (N, K) in synth.LAYER_SHAPES.items():
        for M in (1, 1024):
            out.append((M, N, K, 2, 4))
    return out


def _int8_workspace(M, N, K, c, q=4):
    """Activation fragments, then (stream-K) per launch one counter per shared
    tile and two int32 partial tiles per workgroup, each region rounded up to
    256 bytes."""
    up = lambda x: (x + 255) // 256 * 256
    nce = ((K + 127) // 128 + 1) // 2 * 2
    # int8 or FP8 bytes, FP6 fields in 32 bytes per 32 elements, or FP4 nibbles (half as
    # many bytes: FP4 route with q <= 2)
    nib = c.route == apt.APT_ROUTE_FP4_MFMA and q <= 2
    ws = up((M + 31) // 32 * 32 * nce * (64 if nib else 128))
    launches = [(c.bm, c.bn, N, c.grid)]
    if c.split_n:
        launches = [(c.bm, c.bn, c.split_n, c.grid), (c.tail_bm, c.tail_bn, N - c.split_n, c.tail_grid)]
    waves = {(256, 256): 8, (512, 128): 8, (128, 128): 4}
    for bm, bn, cols, g in launches:
        tiles = -(-M // bm) * -(-cols // bn)
        grid = tiles if g == 0 else min(g, tiles * nce // 2)
        sk_tiles = tiles - tiles // grid * grid
        # leftover tiles more than half of the compute units the grid covers and
        # at most all of them stay whole, one per workgroup: no partials
        w = waves.get((bm, bn), 4 if (bm, bn, c.waves_m * c.waves_n) == (256, 128, 4) else 8)
        units = max(1, grid // (2 if w <= 4 else 1))
        whole = 2 * sk_tiles > units and sk_tiles <= units
        if sk_tiles and not whole:
            ws += up(2 * grid * bm * bn * 4) + up(sk_tiles * 4)
    return ws


def test_workspace_stream_k():
    c = apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 256, 256, 128, 4, 2, 256, 3)
    ws = apt.apt_gemm_workspace_bytes(2048, 11008, 4096, 4, 4, c)
    assert ws == 2048 * 4096 + 512 * 256 * 256 * 4 + 512  # 344 tiles: 88 shared
    assert ws == _int8_workspace(2048, 11008, 4096, c)
    c.grid = 0  # one workgroup per tile: fragments only
    assert apt.apt_gemm_workspace_bytes(2048, 11008, 4096, 4, 4, c) == 2048 * 4096
    c.grid = 344  # divides the tile count: no stream-K part
    assert apt.apt_gemm_workspace_bytes(2048, 11008, 4096, 4, 4, c) == 2048 * 4096
    # a tail launch over [8192, 11008) with 128x128 tiles on 512 workgroups
    c = apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 256, 256, 128, 4, 2, 0, 3, 0, 8192, 128, 128, 512)
    ws = apt.apt_gemm_workspace_bytes(2048, 11008, 4096, 4, 4, c)
    assert ws == 2048 * 4096 + 1024 * 128 * 128 * 4 + 1536  # 352 tail tiles, all shared
    assert ws == _int8_workspace(2048, 11008, 4096, c)
    # on 256 workgroups (128 compute units) the 96 leftover tail tiles stay whole
    c.tail_grid = 256
    assert apt.apt_gemm_workspace_bytes(2048, 11008, 4096, 4, 4, c) == 2048 * 4096
    assert _int8_workspace(2048, 11008, 4096, c) == 2048 * 4096
    # the prefill on one round of 512 workgroups: 176 leftover 256x128 tiles, whole
    c = apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 256, 128, 128, 4, 1, 512, 3)
    assert apt.apt_gemm_workspace_bytes(2048, 11008, 4096, 4, 4, c) == 2048 * 4096


@pytest.mark.parametrize("shape", _shapes())
def test_select_config_valid(shape):
    st, c = apt.apt_select_config(*shape)
    assert st == apt.APT_OK
    assert c.route in (apt.APT_ROUTE_XOR, apt.APT_ROUTE_INT8_MFMA, apt.APT_ROUTE_PM1_MFMA,
                       apt.APT_ROUTE_FP4_MFMA, apt.APT_ROUTE_FP6_MFMA, apt.APT_ROUTE_FP8_MFMA)
    if c.route == apt.APT_ROUTE_FP4_MFMA:
        M, N, K, p, q = shape
        k_pad = (K + 127) // 128 * 128
        assert p <= 2 and q <= 4 and k_pad * ((1 << p) - 1) * ((1 << q) - 1) < 1 << 24
    if shape[0] <= 8:
        assert c.route == apt.APT_ROUTE_XOR
    M, N, K, p, q = shape
    ws = apt.apt_gemm_workspace_bytes(*shape, c)
    if c.route in (apt.APT_ROUTE_INT8_MFMA, apt.APT_ROUTE_FP4_MFMA, apt.APT_ROUTE_FP6_MFMA,
                   apt.APT_ROUTE_FP8_MFMA):
        assert ws == _int8_workspace(M, N, K, c, q)
    else:
        assert ws == 0


def test_select_config_rejects():
    assert apt.apt_select_config(0, 1, 1, 1, 1)[0] == apt.APT_ERR_INVALID_ARG
    assert apt.apt_select_config(1, 1, 1, 9, 1)[0] == apt.APT_ERR_INVALID_ARG
    L = apt.lib()
    assert L.apt_select_config(1, 1, 1, 1, 1, None) == apt.APT_ERR_INVALID_ARG


# Fake, never-dereferenced device addresses: every call below must be rejected
# by host validation before any HIP call.
A, W, C = 0x7F0000000000, 0x7F0000100000, 0x7F0000200000
RA, RW, S = 0x7F0000300000, 0x7F0000400000, 0x7F0000500000


WS = 0x7F0000600000


def gemm(M=4, N=4, K=64, p=2, q=2, a=A, w=W, ra=RA, rw=RW, c32=C, sa=None, sw=None, c16=None,
         cfg=None, ws=None, ws_bytes=0):
    return apt.apt_gemm(M, N, K, p, q, a, w, ra, rw, c32, sa, sw, c16, cfg, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,want", [
    (dict(M=0), apt.APT_ERR_INVALID_ARG), (dict(N=-1), apt.APT_ERR_INVALID_ARG),
    (dict(K=0), apt.APT_ERR_INVALID_ARG), (dict(p=0), apt.APT_ERR_INVALID_ARG),
    (dict(q=9), apt.APT_ERR_INVALID_ARG), (dict(a=None), apt.APT_ERR_INVALID_ARG),
    (dict(w=None), apt.APT_ERR_INVALID_ARG), (dict(a=A + 4), apt.APT_ERR_INVALID_ARG),
    (dict(w=W + 8), apt.APT_ERR_INVALID_ARG), (dict(c32=None), apt.APT_ERR_INVALID_ARG),
    (dict(c16=C, sa=S), apt.APT_ERR_INVALID_ARG), (dict(c16=C, sw=S), apt.APT_ERR_INVALID_ARG),
    (dict(K=33026, p=8, q=8), apt.APT_ERR_UNSUPPORTED),
    (dict(K=1 << 30, p=2, q=2), apt.APT_ERR_UNSUPPORTED),
    (dict(cfg=apt.apt_config_t.make(7)), apt.APT_ERR_INVALID_ARG),
    (dict(cfg=apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 96, 128, 128, 2, 2)),
     apt.APT_ERR_INVALID_ARG),
    (dict(M=64, cfg=apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2), ra=None),
     apt.APT_ERR_INVALID_ARG),
    (dict(p=8, cfg=apt.apt_config_t.make(apt.APT_ROUTE_PM1_MFMA)), apt.APT_ERR_UNSUPPORTED),
    (dict(cfg=apt.apt_config_t.make(apt.APT_ROUTE_XOR, mt=3)), apt.APT_ERR_INVALID_ARG),
    (dict(cfg=apt.apt_config_t.make(apt.APT_ROUTE_XOR, waves_m=3)), apt.APT_ERR_INVALID_ARG),
    (dict(cfg=apt.apt_config_t.make(apt.APT_ROUTE_XOR, waves_n=8)), apt.APT_ERR_INVALID_ARG),
    # one activation row per block row: M block rows, at most 65535
    (dict(M=65536, cfg=apt.apt_config_t.make(apt.APT_ROUTE_XOR, mt=1)), apt.APT_ERR_UNSUPPORTED),
    (dict(M=64, cfg=apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2)),
     apt.APT_ERR_WORKSPACE),
    (dict(M=64, cfg=apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2), ws=WS,
          ws_bytes=64 * 256 - 1), apt.APT_ERR_WORKSPACE),
    (dict(M=64, cfg=apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2), ws=WS + 8,
          ws_bytes=1 << 20), apt.APT_ERR_INVALID_ARG),
    # persistent grid: 0..4096 workgroups
    (dict(M=64, cfg=apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2, -1, 3)),
     apt.APT_ERR_INVALID_ARG),
    (dict(M=64, cfg=apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2, 4097, 3)),
     apt.APT_ERR_INVALID_ARG),
    # (2 tiles on 4 workgroups: split in two parts each, with partial tiles)
    (dict(M=64, N=512, K=1024, cfg=apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 256, 256, 128, 4, 2,
                                                         4, 3), ws=WS,
          ws_bytes=64 * 1024), apt.APT_ERR_WORKSPACE),
    # tail launch: split_n a multiple of bn inside (0, N), a configured tail tile
    (dict(M=64, N=300, cfg=apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2, 0, 3, 0,
                                                 100, 128, 128)), apt.APT_ERR_INVALID_ARG),
    (dict(M=64, N=300, cfg=apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2, 0, 3, 0,
                                                 256, 96, 128)), apt.APT_ERR_INVALID_ARG),
    (dict(M=64, N=256, cfg=apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2, 0, 3, 0,
                                                 256, 128, 128)), apt.APT_ERR_INVALID_ARG),
    (dict(M=64, N=300, cfg=apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2, 0, 3, 0,
                                                 256, 128, 128, -2)), apt.APT_ERR_INVALID_ARG),
    # the int8 weight ring is 3 deep
    (dict(M=64, cfg=apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2, 0, 2)),
     apt.APT_ERR_INVALID_ARG),
    # FP4 route: weights of at most 2 bits, activations of at most 4 bits (FP4 up to
    # 2, FP8 up to 4), and fp32 sums below 2^24
    (dict(p=3, cfg=apt.apt_config_t.make(apt.APT_ROUTE_FP4_MFMA, 128, 128, 128, 2, 2)),
     apt.APT_ERR_UNSUPPORTED),
    (dict(q=5, cfg=apt.apt_config_t.make(apt.APT_ROUTE_FP4_MFMA, 128, 128, 128, 2, 2)),
     apt.APT_ERR_UNSUPPORTED),
    (dict(K=(1 << 24) // 45 + 1, p=2, q=4,
          cfg=apt.apt_config_t.make(apt.APT_ROUTE_FP4_MFMA, 128, 128, 128, 2, 2)),
     apt.APT_ERR_UNSUPPORTED),
    (dict(K=(1 << 24) // 9 + 1, p=2, q=2,
          cfg=apt.apt_config_t.make(apt.APT_ROUTE_FP4_MFMA, 128, 128, 128, 2, 2)),
     apt.APT_ERR_UNSUPPORTED),
    # the bound counts the padding elements of the last chunk: K below 2^24 / 9 whose
    # padded length is not
    (dict(K=(1 << 24) // 9 // 128 * 128 + 1, p=2, q=2,
          cfg=apt.apt_config_t.make(apt.APT_ROUTE_FP4_MFMA, 128, 128, 128, 2, 2)),
     apt.APT_ERR_UNSUPPORTED),
    (dict(M=64, p=1, q=2, cfg=apt.apt_config_t.make(apt.APT_ROUTE_FP4_MFMA, 128, 128, 128, 2, 2)),
     apt.APT_ERR_WORKSPACE),
    (dict(M=64, p=2, q=4, cfg=apt.apt_config_t.make(apt.APT_ROUTE_FP4_MFMA, 128, 128, 128, 2, 2)),
     apt.APT_ERR_WORKSPACE),
    (dict(M=64, p=1, q=2, cfg=apt.apt_config_t.make(apt.APT_ROUTE_FP4_MFMA, 96, 128, 128, 2, 2)),
     apt.APT_ERR_INVALID_ARG),
    # FP6 route: weights and activations of at most 3 bits, fp32 sums below 2^24
    (dict(p=4, q=3, cfg=apt.apt_config_t.make(apt.APT_ROUTE_FP6_MFMA, 128, 128, 128, 2, 2)),
     apt.APT_ERR_UNSUPPORTED),
    (dict(p=3, q=4, cfg=apt.apt_config_t.make(apt.APT_ROUTE_FP6_MFMA, 128, 128, 128, 2, 2)),
     apt.APT_ERR_UNSUPPORTED),
    (dict(K=(1 << 24) // 49 // 128 * 128 + 1, p=3, q=3,
          cfg=apt.apt_config_t.make(apt.APT_ROUTE_FP6_MFMA, 128, 128, 128, 2, 2)),
     apt.APT_ERR_UNSUPPORTED),
    (dict(M=64, p=3, q=3, cfg=apt.apt_config_t.make(apt.APT_ROUTE_FP6_MFMA, 128, 128, 128, 2, 2)),
     apt.APT_ERR_WORKSPACE),
    # FP8 route: weights and activations of at most 4 bits, fp32 sums below 2^24
    (dict(p=5, q=4, cfg=apt.apt_config_t.make(apt.APT_ROUTE_FP8_MFMA, 128, 128, 128, 2, 2)),
     apt.APT_ERR_UNSUPPORTED),
    (dict(p=4, q=5, cfg=apt.apt_config_t.make(apt.APT_ROUTE_FP8_MFMA, 128, 128, 128, 2, 2)),
     apt.APT_ERR_UNSUPPORTED),
    (dict(K=(1 << 24) // 225 // 128 * 128 + 1, p=4, q=4,
          cfg=apt.apt_config_t.make(apt.APT_ROUTE_FP8_MFMA, 128, 128, 128, 2, 2)),
     apt.APT_ERR_UNSUPPORTED),
    (dict(M=64, p=4, q=4, cfg=apt.apt_config_t.make(apt.APT_ROUTE_FP8_MFMA, 128, 128, 128, 2, 2)),
     apt.APT_ERR_WORKSPACE),
    # packed weights past 4 GiB do not fit the int8 kernels' 32-bit offsets
    (dict(M=64, N=1 << 20, K=1 << 16, p=1, q=1,
          cfg=apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2)),
     apt.APT_ERR_UNSUPPORTED),
    # the +-1 plane route's grid holds one workgroup per tile
    (dict(M=1 << 24, N=1 << 24, K=128, p=1, q=1, cfg=apt.apt_config_t.make(apt.APT_ROUTE_PM1_MFMA)),
     apt.APT_ERR_UNSUPPORTED),
    # tile counts past 2^31 do not fit the plans' 32-bit counts (operands within 4 GiB)
    (dict(M=1 << 24, N=1 << 24, K=128, p=1, q=1,
          cfg=apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2)),
     apt.APT_ERR_UNSUPPORTED),
])
def test_gemm_validation(kw, want):
    assert gemm(**kw) == want


def gemm_affine(M=4, N=4, K=64, p=2, q=2, a=A, w=W, ra=RA, rw=RW, sa=S, za=S + 64, sw=S + 128,
                zw=S + 192, c16=C, c32=None, cfg=None, ws=None, ws_bytes=0):
    return apt.apt_gemm_affine(M, N, K, p, q, a, w, ra, rw, sa, za, sw, zw, c16, c32, cfg, ws,
                               ws_bytes, None)


@pytest.mark.parametrize("kw,want", [
    (dict(ra=None), apt.APT_ERR_INVALID_ARG), (dict(rw=None), apt.APT_ERR_INVALID_ARG),
    (dict(sa=None), apt.APT_ERR_INVALID_ARG), (dict(za=None), apt.APT_ERR_INVALID_ARG),
    (dict(sw=None), apt.APT_ERR_INVALID_ARG), (dict(zw=None), apt.APT_ERR_INVALID_ARG),
    (dict(c16=None, c32=C), apt.APT_ERR_INVALID_ARG), (dict(M=0), apt.APT_ERR_INVALID_ARG),
    (dict(q=0), apt.APT_ERR_INVALID_ARG), (dict(a=A + 4), apt.APT_ERR_INVALID_ARG),
    (dict(K=33026, p=8, q=8), apt.APT_ERR_UNSUPPORTED),
    (dict(cfg=apt.apt_config_t.make(apt.APT_ROUTE_XOR, mt=5)), apt.APT_ERR_INVALID_ARG),
    (dict(M=64, cfg=apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2)),
     apt.APT_ERR_WORKSPACE),
])
def test_gemm_affine_validation(kw, want):
    assert gemm_affine(**kw) == want


@pytest.mark.parametrize("kw", [dict(rows=0), dict(K=0), dict(bits=0), dict(bits=9),
                                dict(codes=None), dict(packed=None), dict(packed=A + 4)])
def test_pack_validation(kw):
    args = dict(codes=A, rows=4, K=64, bits=3, packed=W, rowsum=None)
    args.update(kw)
    for fn in (apt.apt_pack_weights, apt.apt_quantize_pack_activations):
        st = fn(args["codes"], args["rows"], args["K"], args["bits"], args["packed"],
                args["rowsum"], None)
        assert st == apt.APT_ERR_INVALID_ARG


@pytest.mark.parametrize("kw", [dict(rows=0), dict(K=0), dict(bits=0), dict(bits=9),
                                dict(x=None), dict(packed=None), dict(packed=A + 4),
                                dict(scale=None)])
def test_quantize_fp16_validation(kw):
    """Rejected before any HIP call (the pointers are never dereferenced)."""
    args = dict(x=A, rows=4, K=64, bits=3, packed=W, rowsum=None, scale=A + 2)
    args.update(kw)
    st = apt.apt_quantize_pack_activations_fp16(args["x"], args["rows"], args["K"], args["bits"],
                                                args["packed"], args["rowsum"], args["scale"], None)
    assert st == apt.APT_ERR_INVALID_ARG


def test_pack_rejects_huge_rows():
    """K > 2^30 is refused before any HIP call (32-bit element indexing)."""
    K = (1 << 30) + 1
    for fn in (apt.apt_pack_weights, apt.apt_quantize_pack_activations):
        assert fn(A, 1, K, 2, W, None, None) == apt.APT_ERR_UNSUPPORTED
    assert apt.apt_quantize_pack_activations_fp16(A, 1, K, 2, W, None, A + 2, None) == \
        apt.APT_ERR_UNSUPPORTED


def gemm_decode(M=4, N=4, K=64, p=2, q=2, x=A, kind=apt.APT_ACT_CODES, w=W, c32=C, sa=S,
                sw=S + 128, c16=None, so=None, cfg=None):
    return apt.apt_gemm_decode(M, N, K, p, q, x, kind, w, c32, sa, sw, c16, so, cfg, None)


XOR = apt.APT_ROUTE_XOR


@pytest.mark.parametrize("kw,want", [
    (dict(M=0), apt.APT_ERR_INVALID_ARG), (dict(M=apt.APT_DECODE_MAX_M + 1), apt.APT_ERR_INVALID_ARG),
    (dict(N=0), apt.APT_ERR_INVALID_ARG), (dict(K=0), apt.APT_ERR_INVALID_ARG),
    (dict(p=9), apt.APT_ERR_INVALID_ARG), (dict(q=0), apt.APT_ERR_INVALID_ARG),
    (dict(kind=0), apt.APT_ERR_INVALID_ARG), (dict(kind=3), apt.APT_ERR_INVALID_ARG),
    (dict(x=None), apt.APT_ERR_INVALID_ARG), (dict(w=None), apt.APT_ERR_INVALID_ARG),
    (dict(w=W + 4), apt.APT_ERR_INVALID_ARG),
    (dict(kind=apt.APT_ACT_FP16, x=A + 1, sa=None), apt.APT_ERR_INVALID_ARG),
    (dict(c32=None), apt.APT_ERR_INVALID_ARG),
    (dict(c16=C, sa=None), apt.APT_ERR_INVALID_ARG),
    (dict(c16=C, sw=None), apt.APT_ERR_INVALID_ARG),
    (dict(kind=apt.APT_ACT_FP16), apt.APT_ERR_INVALID_ARG),       # a_scale with an fp16 source
    (dict(so=S + 64), apt.APT_ERR_INVALID_ARG),                   # scale output with codes
    (dict(cfg=apt.apt_config_t.make(XOR, mt=5)), apt.APT_ERR_INVALID_ARG),
    (dict(K=7169, p=1, q=8, cfg=apt.apt_config_t.make(XOR, mt=8)), apt.APT_ERR_UNSUPPORTED),
    (dict(cfg=apt.apt_config_t.make(XOR, waves_m=3)), apt.APT_ERR_INVALID_ARG),
    (dict(cfg=apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2)),
     apt.APT_ERR_INVALID_ARG),
    (dict(K=33026, p=8, q=8), apt.APT_ERR_UNSUPPORTED),
    (dict(K=65537, p=1, q=8), apt.APT_ERR_UNSUPPORTED),           # planes past 64 KB of LDS
    (dict(K=131073, p=1, q=4), apt.APT_ERR_UNSUPPORTED),
])
def test_gemm_decode_validation(kw, want):
    """Rejected before any HIP call (the pointers are never dereferenced)."""
    assert gemm_decode(**kw) == want


def gemm_act(M=4, N=4, K=64, p=2, q=2, x=A, kind=apt.APT_ACT_CODES, w=W, rw=RW, c32=C, sa=S,
             sw=S + 128, c16=None, so=None, cfg=None, ws=None, ws_bytes=0):
    return apt.apt_gemm_act(M, N, K, p, q, x, kind, w, rw, c32, sa, sw, c16, so, cfg, ws, ws_bytes,
                            None)


INT8_CFG = apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2)


@pytest.mark.parametrize("kw,want", [
    (dict(M=0), apt.APT_ERR_INVALID_ARG), (dict(N=0), apt.APT_ERR_INVALID_ARG),
    (dict(K=0), apt.APT_ERR_INVALID_ARG), (dict(p=0), apt.APT_ERR_INVALID_ARG),
    (dict(q=9), apt.APT_ERR_INVALID_ARG), (dict(kind=7), apt.APT_ERR_INVALID_ARG),
    (dict(x=None), apt.APT_ERR_INVALID_ARG), (dict(w=None), apt.APT_ERR_INVALID_ARG),
    (dict(w=W + 8), apt.APT_ERR_INVALID_ARG),
    (dict(kind=apt.APT_ACT_FP16, x=A + 1, sa=None), apt.APT_ERR_INVALID_ARG),
    (dict(c32=None), apt.APT_ERR_INVALID_ARG),
    (dict(c16=C, sw=None), apt.APT_ERR_INVALID_ARG), (dict(c16=C, sa=None), apt.APT_ERR_INVALID_ARG),
    (dict(kind=apt.APT_ACT_FP16), apt.APT_ERR_INVALID_ARG),        # a_scale with an fp16 source
    (dict(so=S + 64), apt.APT_ERR_INVALID_ARG),                    # scale output with codes
    (dict(K=33026, p=8, q=8), apt.APT_ERR_UNSUPPORTED),
    (dict(cfg=apt.apt_config_t.make(apt.APT_ROUTE_XOR, mt=3)), apt.APT_ERR_INVALID_ARG),
    (dict(M=64, cfg=INT8_CFG, rw=None), apt.APT_ERR_INVALID_ARG),  # MFMA routes need the weight row sums
    (dict(M=64, cfg=INT8_CFG), apt.APT_ERR_WORKSPACE),
    (dict(M=64, cfg=INT8_CFG, ws=S + 4, ws_bytes=1 << 30), apt.APT_ERR_INVALID_ARG),
    (dict(M=64, K=(1 << 30) + 128, p=1, q=1, cfg=INT8_CFG), apt.APT_ERR_UNSUPPORTED),
])
def test_gemm_act_validation(kw, want):
    """Rejected before any HIP call (the pointers are never dereferenced)."""
    assert gemm_act(**kw) == want


def test_gemm_act_workspace_bytes():
    """Fused XOR decode: none; int8 MFMA: the route's workspace plus row sums
    and scales; other routes: also the packed activations."""
    ws = apt.apt_gemm_act_workspace_bytes
    assert ws(1, 4096, 4096, 2, 2, apt.APT_ACT_CODES) == 0
    assert ws(1, 4096, 4096, 2, 2, apt.APT_ACT_FP16) == 0
    M, N, K = 1024, 4096, 4096
    route = apt.apt_gemm_workspace_bytes(M, N, K, 2, 4, INT8_CFG)
    r256 = lambda x: (x + 255) // 256 * 256  # noqa: E731
    assert ws(M, N, K, 2, 4, apt.APT_ACT_CODES, INT8_CFG) == r256(route) + r256(4 * M) + r256(2 * M)
    xor = apt.apt_config_t.make(apt.APT_ROUTE_XOR)
    assert ws(64, N, K, 2, 4, apt.APT_ACT_CODES, xor) == (
        r256(apt.apt_packed_bytes(64, K, 4)) + r256(4 * 64) + r256(2 * 64))
    fp4 = apt.apt_config_t.make(apt.APT_ROUTE_FP4_MFMA, 128, 128, 128, 2, 2)
    route = apt.apt_gemm_workspace_bytes(M, N, K, 2, 2, fp4)
    assert ws(M, N, K, 2, 2, apt.APT_ACT_FP16, fp4) == (
        r256(route) + r256(apt.apt_packed_bytes(M, K, 2)) + r256(4 * M) + r256(2 * M))
    # past 2^31 source bytes the rows go through the packer (planes in the workspace)
    big_m, big_k = 1 << 16, 1 << 15
    route = apt.apt_gemm_workspace_bytes(big_m, 256, big_k, 1, 1, INT8_CFG)
    assert route > 0
    assert ws(big_m, 256, big_k - 1, 1, 1, apt.APT_ACT_CODES, INT8_CFG) == (
        r256(apt.apt_gemm_workspace_bytes(big_m, 256, big_k - 1, 1, 1, INT8_CFG)) + r256(4 * big_m)
        + r256(2 * big_m))
    assert ws(big_m, 256, big_k, 1, 1, apt.APT_ACT_CODES, INT8_CFG) == (
        r256(route) + r256(apt.apt_packed_bytes(big_m, big_k, 1)) + r256(4 * big_m) + r256(2 * big_m))
    assert ws(0, N, K, 2, 2, apt.APT_ACT_CODES) == 0
    assert ws(4, N, K, 2, 2, 5) == 0


def test_config_struct_layout():
    assert ctypes.sizeof(apt.apt_config_t) == 16 * 4


def search(M=64, N=300, K=1000, p=2, q=4, a=A, w=W, ra=RA, rw=RW, c32=C, ws=None, ws_bytes=0):
    return apt.apt_search_config(M, N, K, p, q, a, w, ra, rw, c32, ws, ws_bytes, None)[0]


@pytest.mark.parametrize("kw,want", [
    (dict(M=0), apt.APT_ERR_INVALID_ARG), (dict(p=9), apt.APT_ERR_INVALID_ARG),
    (dict(a=None), apt.APT_ERR_INVALID_ARG), (dict(w=W + 4), apt.APT_ERR_INVALID_ARG),
    (dict(ra=None), apt.APT_ERR_INVALID_ARG), (dict(rw=None), apt.APT_ERR_INVALID_ARG),
    (dict(c32=None), apt.APT_ERR_INVALID_ARG),
    (dict(K=33026, p=8, q=8), apt.APT_ERR_UNSUPPORTED),
    (dict(), apt.APT_ERR_WORKSPACE),                      # q = 4: stream-K candidates need room
    (dict(ws=WS, ws_bytes=1024), apt.APT_ERR_WORKSPACE),
    (dict(ws=WS + 8, ws_bytes=1 << 40), apt.APT_ERR_INVALID_ARG),
])
def test_search_validation(kw, want):
    """Every case is rejected on the host before any HIP call."""
    assert search(**kw) == want


def test_search_best_pointer_required():
    L = apt.lib()
    st = L.apt_search_config(64, 300, 1000, 2, 4, A, W, RA, RW, C, WS, 1 << 40, None, None, None)
    assert st == apt.APT_ERR_INVALID_ARG


def test_search_workspace_covers_every_selectable_config():
    for shape in _shapes():
        need = apt.apt_search_workspace_bytes(*shape)
        assert need >= apt.apt_gemm_workspace_bytes(*shape, None)
        # each int8 tile shape with a persistent round of workgroups is a candidate
        M, N, K, p, q = shape
        for bm, bn, wm, wn in [(256, 256, 4, 2), (256, 128, 4, 2), (512, 128, 8, 1)]:
            c = apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, bm, bn, 128, wm, wn, 256, 3)
            assert need >= apt.apt_gemm_workspace_bytes(M, N, K, p, q, c)
    assert apt.apt_search_workspace_bytes(0, 1, 1, 1, 1) == 0


def test_config_table_starts_empty_and_clears():
    apt.apt_config_table_clear()
    assert apt.apt_config_table_size() == 0


def test_fp4_workspace_is_half_the_int8_fragments():
    """FP4 activations (q <= 2) take half a byte per element, FP8 ones (q = 3, 4) a byte."""
    i8 = apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2)
    f4 = apt.apt_config_t.make(apt.APT_ROUTE_FP4_MFMA, 128, 128, 128, 2, 2)
    for M, K in [(64, 1000), (100, 4096), (2048, 4096)]:
        a = apt.apt_gemm_workspace_bytes(M, 512, K, 2, 2, i8)
        b = apt.apt_gemm_workspace_bytes(M, 512, K, 2, 2, f4)
        nce = ((K + 127) // 128 + 1) // 2 * 2
        assert a == (M + 31) // 32 * 32 * nce * 128
        assert b == (M + 31) // 32 * 32 * nce * 64
        for q in (3, 4):
            assert apt.apt_gemm_workspace_bytes(M, 512, K, 2, q, f4) == a
    assert apt.apt_gemm_workspace_bytes(64, 512, 1000, 3, 2, f4) == 0  # p = 3: not runnable
    assert apt.apt_gemm_workspace_bytes(64, 512, 1000, 2, 5, f4) == 0  # q = 5: not runnable


def test_noalloc_rejects_before_any_launch():
    """apt_gemm_noalloc validates like apt_gemm and refuses a config whose
    workspace exceeds its fixed array, before it touches the runtime."""
    f = apt.apt_gemm_noalloc
    fake = 1 << 12  # aligned, never dereferenced: every case below fails validation
    assert f(0, 1, 1, 1, 1, fake, fake, fake, fake, fake, None, None, None, None,
             None) == apt.APT_ERR_INVALID_ARG
    assert f(4, 4, 4, 2, 2, fake, fake, fake, fake, None, None, None, None, None,
             None) == apt.APT_ERR_INVALID_ARG
    assert f(4, 4, 4, 2, 2, fake + 4, fake, fake, fake, fake, None, None, None, None,
             None) == apt.APT_ERR_INVALID_ARG
    assert f(4, 4, 40000, 8, 8, fake, fake, fake, fake, fake, None, None, None, None,
             None) == apt.APT_ERR_UNSUPPORTED
    # activation fragments of 65536 x 4096 bytes (256 MiB) exceed the 64 MiB array
    cfg = apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 256, 128, 128, 4, 1, 0, 3)
    assert apt.apt_gemm_workspace_bytes(65536, 4096, 4096, 4, 4, cfg) > 64 << 20
    assert f(65536, 4096, 4096, 4, 4, fake, fake, fake, fake, fake, None, None, None, cfg,
             None) == apt.APT_ERR_WORKSPACE
    assert f(65536, 4096, 4096, 4, 4, fake, fake, fake, fake, fake, None, None, None, None,
             None) == apt.APT_ERR_WORKSPACE
    # a forced persistent grid whose partial tiles do not fit is refused, not changed
    cfg = apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 256, 256, 128, 4, 2, 300, 3)
    assert apt.apt_gemm_workspace_bytes(1000, 1000, 4096, 4, 4, cfg) > 64 << 20
    assert f(1000, 1000, 4096, 4, 4, fake, fake, fake, fake, fake, None, None, None, cfg,
             None) == apt.APT_ERR_WORKSPACE
    assert apt.apt_last_hip_error() == 0


def test_shipped_table_configs_and_approximate_match():
    """The shipped table (searched configs of the workload shapes, Sec. V-B)
    answers the workload shapes and shapes near them (same p, q and M bucket,
    N and K within the matching radius); every config it gives is valid for its
    problem (it has a workspace size)."""
    import bench
    for prob in bench.workload_problems():
        st, c = apt.apt_select_config(prob.M, prob.N, prob.K, prob.p, prob.q)
        assert st == apt.APT_OK
        if c.route in (apt.APT_ROUTE_INT8_MFMA, apt.APT_ROUTE_FP4_MFMA):
            assert apt.apt_gemm_workspace_bytes(prob.M, prob.N, prob.K, prob.p, prob.q, c) > 0
    prefill = apt.select_config(2048, 11008, 4096, 4, 4)
    assert (prefill.route, prefill.bm, prefill.bn, prefill.waves_m, prefill.waves_n, prefill.grid) == \
        (apt.APT_ROUTE_INT8_MFMA, 256, 128, 4, 1, 512)
    near = apt.select_config(1900, 11000, 4200, 4, 4)
    assert near.as_dict() == prefill.as_dict()
    down = apt.select_config(512, 4096, 11008, 3, 3)
    assert apt.select_config(500, 4000, 11000, 3, 3).as_dict() == down.as_dict()


def test_fp6_workspace_and_bound():
    """FP6 activations take 32 bytes of fragment per 32 elements (as int8), and the
    route admits W3A3 up to K_pad * 49 < 2^24."""
    f6 = apt.apt_config_t.make(apt.APT_ROUTE_FP6_MFMA, 128, 128, 128, 2, 2)
    i8 = apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2)
    assert apt.apt_gemm_workspace_bytes(100, 300, 1000, 3, 3, f6) == \
        apt.apt_gemm_workspace_bytes(100, 300, 1000, 3, 3, i8) > 0
    k_ok = ((1 << 24) - 1) // 49 // 128 * 128
    assert apt.apt_gemm_workspace_bytes(64, 64, k_ok, 3, 3, f6) > 0
    assert apt.apt_gemm_workspace_bytes(64, 64, k_ok + 128, 3, 3, f6) == 0


def test_fp8_workspace_and_bound():
    """FP8 activations take one byte of fragment per element (as int8), and the
    route admits W4A4 up to K_pad * 225 < 2^24."""
    f8 = apt.apt_config_t.make(apt.APT_ROUTE_FP8_MFMA, 128, 128, 128, 2, 2)
    i8 = apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2)
    assert apt.apt_gemm_workspace_bytes(100, 300, 1000, 4, 4, f8) == \
        apt.apt_gemm_workspace_bytes(100, 300, 1000, 4, 4, i8) > 0
    k_ok = ((1 << 24) - 1) // 225 // 128 * 128
    assert apt.apt_gemm_workspace_bytes(64, 64, k_ok, 4, 4, f8) > 0
    assert apt.apt_gemm_workspace_bytes(64, 64, k_ok + 128, 4, 4, f8) == 0
