"""Helpers shared by the GPU parity tests: run a problem through the C ABI
(via the binding) and compare with the oracle."""
from __future__ import annotations

import numpy as np

import paper_2508_19087_amd as apt
from oracle import oracle as ref

INT8_SHAPES = [(256, 256, 4, 2), (256, 256, 2, 4), (256, 128, 4, 2), (128, 128, 2, 2), (512, 128, 8, 1),
               (256, 128, 4, 1)]


def forced_configs(p: int, q: int, N: int = 0, K: int = 0):
    """(name, config) of every route and tile shape the library can be forced
    to; the XOR route with every launch shape; the int8 shapes with one workgroup per tile (grid 0) and with
    persistent stream-K grids: 256 workgroups, 7 (many workgroups share each
    tile) and 300; with N, also split launches (main tiles, then 128x128 tail
    tiles, one per workgroup and stream-K)."""
    del K
    out = [("xor", apt.apt_config_t.make(apt.APT_ROUTE_XOR))]
    # XOR route launch shapes: activation rows per block row (1 or 8), waves per
    # workgroup (one row group each), or the K split over 2 or 4 waves
    for mt in (1, 8):
        for waves in (1, 2, 4):
            c = apt.apt_config_t.make(apt.APT_ROUTE_XOR, waves_m=waves, waves_n=1, mt=mt)
            out.append(("xor_mt%d_w%d" % (mt, waves), c))
        for ks in (2, 4):
            c = apt.apt_config_t.make(apt.APT_ROUTE_XOR, waves_n=ks, mt=mt)
            out.append(("xor_mt%d_ks%d" % (mt, ks), c))
    for bm, bn, wm, wn in INT8_SHAPES:
        for grid in (0, 256, 7, 300):
            c = apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, bm, bn, 128, wm, wn, grid, 3)
            out.append(("int8_%dx%d_w%dx%d_g%d" % (bm, bn, wm, wn, grid), c))
        split = (N - 1) // bn * bn
        if N and split >= bn:
            tails = [(128, 128)] + ([(256, 128)] if (wm, wn) in ((4, 2), (8, 1), (4, 1)) else [])
            # paired launches: 256x256 or 512x128 + 256x128 (8 waves); 256x128 (4x1) + 128x128
            # or 256x128 (4 waves)
            for tbm, tbn in tails:
                for tg in (0, 5):
                    c = apt.apt_config_t.make(apt.APT_ROUTE_INT8_MFMA, bm, bn, 128, wm, wn, 0, 3, 0,
                                              split, tbm, tbn, tg)
                    out.append(("int8_%dx%d_w%dx%d_tail%dx%d@%d_g%d" % (bm, bn, wm, wn, tbm, tbn, split,
                                                                        tg), c))
    floats = []
    for route, tag, ok in ((apt.APT_ROUTE_FP4_MFMA, "fp4", p <= 2 and q <= 4),
                           (apt.APT_ROUTE_FP6_MFMA, "fp6", p <= 3 and q <= 3),
                           (apt.APT_ROUTE_FP8_MFMA, "fp8", p <= 4 and q <= 4)):
        if not ok:  # the same tile configs with FP4 weights (FP4 or FP8 activations) / FP6 / FP8 operands
            continue
        for name, c in out:
            if c.route == apt.APT_ROUTE_INT8_MFMA:
                f = apt.apt_config_t.make(route, c.bm, c.bn, c.bk, c.waves_m, c.waves_n, c.grid,
                                          c.lds_stages, c.mt, c.split_n, c.tail_bm, c.tail_bn,
                                          c.tail_grid)
                floats.append((tag + name[4:], f))
    out += floats
    if p <= 7 and q <= 7:
        out.append(("pm1", apt.apt_config_t.make(apt.APT_ROUTE_PM1_MFMA)))
    return out


def dev(arr):
    import torch
    return torch.from_numpy(np.ascontiguousarray(arr)).cuda()


def pack_problem(prob):
    a = apt.pack(dev(prob.a_codes), prob.q, activations=True)
    w = apt.pack(dev(prob.w_codes), prob.p)
    return a, w


def run(prob, cfg=None, int32=True, fp16=False, packed=None):
    """(C int32 numpy or None, C fp16 numpy or None) from the GPU path."""
    import torch
    a, w = packed if packed is not None else pack_problem(prob)
    sa = dev(prob.a_scale) if fp16 else None
    sw = dev(prob.w_scale) if fp16 else None
    c32, c16 = apt.gemm(a, w, out_int32=int32, a_scale=sa, w_scale=sw, out_fp16=fp16, cfg=cfg)
    torch.cuda.synchronize()
    return (c32.cpu().numpy() if c32 is not None else None,
            c16.cpu().numpy() if c16 is not None else None)


def oracle_full(prob):
    return ref.gemm(prob.a_codes, prob.w_codes, prob.p, prob.q)


def assert_int32_equal(got, want, what=""):
    if not np.array_equal(got, want):
        bad = np.argwhere(got != want)
        m, n = bad[0]
        raise AssertionError("%s: %d of %d int32 outputs differ; first at (%d, %d): got %d want %d"
                             % (what, len(bad), want.size, m, n, got[m, n], want[m, n]))


def assert_fp16_ok(got, C, prob, what=""):
    E, _ = ref.epilogue(C, prob.a_scale, prob.w_scale)
    ok = ref.fp16_close(got, E)
    if not ok.all():
        bad = np.argwhere(~ok)
        m, n = bad[0]
        raise AssertionError("%s: %d fp16 outputs outside tolerance; first at (%d, %d): got %r want %r"
                             % (what, len(bad), m, n, float(got[m, n]), E[m, n]))


def sample_rows(M: int, g: np.random.Generator, extra: int = 8):
    """Rows covering every 64-row band edge plus a few random rows."""
    rows = set([0, M - 1])
    for b in range(0, M, 64):
        rows.add(b)
        rows.add(min(M - 1, b + 63))
    rows.update(g.integers(0, M, extra).tolist())
    return np.array(sorted(rows), dtype=np.int64)


def check_sampled(prob, c32, seed: int = 0, n_entries: int = 100000, what=""):
    """Full comparison of sampled rows, sampled columns and random entries."""
    g = np.random.default_rng(seed)
    va = ref.values(prob.a_codes, prob.q)
    vw = ref.values(prob.w_codes, prob.p)
    rows = sample_rows(prob.M, g)
    assert_int32_equal(c32[rows], ref.matmul(va[rows], vw), what + " rows")
    cols = sample_rows(prob.N, g)
    assert_int32_equal(c32[:, cols], ref.matmul(va, vw[cols]), what + " cols")
    mi = g.integers(0, prob.M, n_entries)
    ni = g.integers(0, prob.N, n_entries)
    want = ref.matmul_entries(va, vw, mi, ni)
    got = c32[mi, ni]
    if not np.array_equal(got, want):
        k = int(np.argmax(got != want))
        raise AssertionError("%s: sampled entry (%d, %d) got %d want %d"
                             % (what, mi[k], ni[k], got[k], want[k]))
    return va, vw, rows
