"""GPU parity of the fused fp16 activation quantizer and packer
(apt_quantize_pack_activations_fp16) against the oracle's quantize_fp16,
convert, pack and rowsum: packed words, row sums and scale bits bit-exact; and
end to end through the GEMM's int32 output and fp16 epilogue."""
import numpy as np
import pytest

import paper_2508_19087_amd as apt
import synth
from gpu_util import assert_int32_equal
from oracle import oracle as ref

pytestmark = pytest.mark.gpu


def gpu_quant(x, q, offset=0):
    """(packed words, row sums, scale bits) from the GPU for fp16 rows x, the
    input starting `offset` halves into a fresh buffer."""
    import torch
    M, K = x.shape
    buf = torch.zeros(x.size + 64, dtype=torch.float16, device="cuda")
    view = buf[offset:offset + x.size]
    view.copy_(torch.from_numpy(np.ascontiguousarray(x).ravel()))
    out = torch.full((apt.apt_packed_bytes(M, K, q),), 0xA5, dtype=torch.uint8, device="cuda")
    rs = torch.full((M,), -7, dtype=torch.int32, device="cuda")
    sc = torch.full((M,), 0x7E00, dtype=torch.int16, device="cuda")  # a NaN until written
    st = apt.apt_quantize_pack_activations_fp16(view.data_ptr(), M, K, q, out.data_ptr(),
                                                rs.data_ptr(), sc.data_ptr(),
                                                torch.cuda.current_stream().cuda_stream)
    assert st == apt.APT_OK, apt.status_string(st)
    torch.cuda.synchronize()
    return out.cpu().numpy().view(np.uint32), rs.cpu().numpy(), sc.cpu().numpy().view(np.uint16)


def expected(x, q):
    codes, s16 = ref.quantize_fp16(x, q)
    u = ref.convert(codes, q)
    return ref.pack(u, q), ref.rowsum(ref.decode(u, q)), s16.view(np.uint16), codes


def check(x, q, offset=0, what=""):
    words, rs, sc = gpu_quant(x, q, offset)
    w_words, w_rs, w_sc, codes = expected(x, q)
    assert np.array_equal(sc, w_sc), "%s: scales differ at rows %s" % (
        what, np.flatnonzero(sc != w_sc)[:8])
    if not np.array_equal(words, w_words):
        back, _ = ref.unpack(words, x.shape[0], x.shape[1], q)
        bad = np.argwhere(back != ref.convert(codes, q))
        raise AssertionError("%s: %d codes differ; first at %s (x=%r)"
                             % (what, len(bad), tuple(bad[0]), float(x[tuple(bad[0])])))
    assert np.array_equal(rs, w_rs), what


@pytest.mark.parametrize("q", range(1, 9))
@pytest.mark.parametrize("M,K", [(1, 1), (3, 31), (2, 33), (5, 127), (4, 128), (3, 129),
                                 (2, 1000), (7, 1024), (2, 1040), (9, 4096), (1, 11008)])
def test_quantize_pack_parity(q, M, K):
    x = synth.fp16_activations(synth.rng(70, q, M, K), M, K)
    check(x, q, what="q=%d %dx%d" % (q, M, K))


@pytest.mark.parametrize("offset", [1, 3, 8])
def test_quantize_pack_unaligned_input(offset):
    """Inputs not 16-byte aligned take the element-wise load path."""
    x = synth.fp16_activations(synth.rng(71, offset), 3, 4096)
    for q in (2, 4):
        check(x, q, offset, what="offset %d q=%d" % (offset, q))


@pytest.mark.parametrize("q", range(1, 9))
def test_quantize_pack_special_rows(q):
    """Zero rows (scale 0, level +1), signed zeros, subnormals only (scale may
    round to 0 or to a subnormal), the fp16 extremes, and exact ties: with a
    power-of-two scale, even multiples of it land halfway between two odd
    levels and go to the upper one."""
    K = 320
    L = 2 ** q - 1
    x = np.zeros((6, K), np.float16)
    x[1, ::2] = np.float16(-0.0)
    x[2] = (np.arange(K) % 7 - 3).astype(np.float16) * np.float16(2.0 ** -24)
    x[3, :4] = [65504.0, -65504.0, 1.0, -1.0]
    s = 2.0 ** -3
    ties = np.arange(-L + 1, L, 2, dtype=np.float64)          # even t in (-L, L)
    x[4, :len(ties)] = (ties * s).astype(np.float16)
    x[4, len(ties)] = np.float16(L * s)                         # sets absmax = L s
    x[5] = synth.fp16_activations(synth.rng(72, q), 1, K)[0]
    words, rs, sc = gpu_quant(x, q)
    w_words, w_rs, w_sc, codes = expected(x, q)
    assert w_sc[0] == 0 and w_sc[4] == np.float16(s).view(np.uint16)
    assert np.array_equal(2 * codes[4, :len(ties)].astype(np.int64) + 1, ties + 1)
    assert np.array_equal(sc, w_sc)
    assert np.array_equal(words, w_words)
    assert np.array_equal(rs, w_rs)


@pytest.mark.parametrize("M,K,q", [(2048, 4096, 4), (1, 4096, 2), (8, 11008, 2)])
def test_quantize_pack_full_size(M, K, q):
    """The activation shapes of the prefill (2048x4096, 4 bits) and decode
    (1 and 8 tokens, 2 bits) workloads, compared in full."""
    x = synth.fp16_activations(synth.rng(73, M, K, q), M, K)
    check(x, q, what="%dx%d q=%d" % (M, K, q))


@pytest.mark.parametrize("M,N,K,p,q", [(64, 512, 4096, 2, 4), (1, 4096, 4096, 2, 2),
                                       (33, 384, 1000, 4, 4)])
def test_quantized_activations_through_gemm(M, N, K, p, q):
    """fp16 activations -> GPU quantize+pack -> GEMM (int32 and the fp16
    epilogue with the produced scales) against the oracle's quantizer, matmul
    and epilogue."""
    import torch
    g = synth.rng(74, M, N, K)
    x = synth.fp16_activations(g, M, K)
    w_codes = synth.uniform_codes(g, N, K, p)
    w_scale = synth.scales(g, N, *synth.W_SCALE_RANGE)
    a, a_scale = apt.quantize_pack(torch.from_numpy(x).cuda(), q)
    w = apt.pack(torch.from_numpy(w_codes).cuda(), p)
    c32, c16 = apt.gemm(a, w, a_scale=a_scale, w_scale=torch.from_numpy(w_scale).cuda(),
                        out_fp16=True)
    torch.cuda.synchronize()
    codes, s16 = ref.quantize_fp16(x, q)
    C = ref.matmul(ref.values(codes, q), ref.values(w_codes, p))
    assert_int32_equal(c32.cpu().numpy(), C, "quantized %dx%dx%d" % (M, N, K))
    E, _ = ref.epilogue(C, s16, w_scale)
    assert ref.fp16_close(c16.cpu().numpy(), E).all()
    assert np.array_equal(a_scale.cpu().numpy().view(np.uint16), s16.view(np.uint16))
