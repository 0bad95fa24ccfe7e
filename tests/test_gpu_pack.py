"""GPU parity of the converter + bit-plane packer against the oracle's
reference packing of the documented layout (bit-exact), and of the row sums."""
import numpy as np
import pytest

import paper_2508_19087_amd as apt
import synth
from oracle import oracle as ref

pytestmark = pytest.mark.gpu


def gpu_pack(codes, bits, activations, offset=0):
    import torch
    buf = torch.zeros(codes.size + 64, dtype=torch.int8, device="cuda")
    view = buf[offset:offset + codes.size]
    view.copy_(torch.from_numpy(codes.ravel()))
    R, K = codes.shape
    out = torch.full((apt.apt_packed_bytes(R, K, bits),), 0xA5, dtype=torch.uint8, device="cuda")
    rs = torch.empty(R, dtype=torch.int32, device="cuda")
    fn = apt.apt_quantize_pack_activations if activations else apt.apt_pack_weights
    st = fn(view.data_ptr(), R, K, bits, out.data_ptr(), rs.data_ptr(),
            torch.cuda.current_stream().cuda_stream)
    assert st == apt.APT_OK, apt.status_string(st)
    torch.cuda.synchronize()
    return out.cpu().numpy().view(np.uint32), rs.cpu().numpy()


@pytest.mark.parametrize("bits", range(1, 9))
@pytest.mark.parametrize("R,K", [(1, 1), (3, 31), (2, 33), (5, 127), (4, 128), (3, 129), (2, 1000),
                                 (7, 1024), (2, 1040), (3, 4096), (1, 11008)])
def test_pack_parity(bits, R, K):
    g = np.random.default_rng(bits * 7919 + R * 31 + K)
    codes = synth.uniform_codes(g, R, K, bits)
    words, rs = gpu_pack(codes, bits, activations=(K % 2 == 0))
    u = ref.convert(codes, bits)
    assert np.array_equal(words, ref.pack(u, bits))
    back, stray = ref.unpack(words, R, K, bits)
    assert stray == 0 and np.array_equal(back, u)
    assert np.array_equal(rs, ref.rowsum(ref.decode(u, bits)))


@pytest.mark.parametrize("offset", [1, 3, 8])
def test_pack_unaligned_codes(offset):
    g = np.random.default_rng(offset)
    codes = synth.uniform_codes(g, 3, 4096, 4)
    words, rs = gpu_pack(codes, 4, True, offset=offset)
    assert np.array_equal(words, ref.pack(ref.convert(codes, 4), 4))
    assert np.array_equal(rs, ref.rowsum(ref.values(codes, 4)))


def test_pack_out_of_range_codes_use_low_bits():
    codes = np.arange(-128, 128, dtype=np.int64).astype(np.int8).reshape(2, 128)
    for bits in (1, 3, 5):
        words, rs = gpu_pack(codes, bits, False)
        assert np.array_equal(words, ref.pack(ref.convert(codes, bits), bits))
        assert np.array_equal(rs, ref.rowsum(ref.values(codes, bits)))
