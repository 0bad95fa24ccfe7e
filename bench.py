"""Benchmark of the WpAq bipolar-INT GEMM hot path on one MI355X.

One step is one pass of the whole path over one batch of synthetic input:
  decode  (M = 1):    the two 7B-class W2A2 decode GEMMs (N=4096 and N=11008,
                      K=4096) with int32 and fp16-epilogue outputs, each one
                      apt_gemm_decode launch that converts the token's codes
                      to bipolar planes inside the GEMV (--unfused-decode:
                      the packer, then apt_gemm);
  prefill (M = 2048): the W4A4 2048 x 11008 x 4096 GEMM with int32 output
                      from the activation codes, one apt_gemm_act call that
                      converts them straight into the int8 MFMA operand
                      fragments (--packed-prefill: the packer, then apt_gemm).
Weights are packed once before timing (they are static).  Every call goes
through the C ABI with the config chosen by the library's selector.  The
decode chain runs on a second stream beside the prefill, and consecutive
steps' prefills alternate between two streams with their own buffers (two
independent batches in flight; --one-batch: every prefill on one stream, a
figure the JSON line also reports; --serial-step: the whole step on one
stream).

Printed JSON line: whole-step effective TOPS (2 M N K summed over the three
GEMMs), the roofline of the dominant kernel (the prefill GEMM, int8 MFMA
bound) timed with HIP events on its stream around back-to-back calls, the
HBM-bound decode GEMM measured separately with cold weights, and the CPU
oracle timed on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import subprocess
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "effective TOPS and % of int8-MFMA/HBM roofline for WpAq GEMM, M=1 & M=2048"
PEAK_INT8_TOPS = 5000.0     # MI355X dense int8 MFMA, 5.0 POP/s
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E, 8 TB/s
MALL_BYTES = 256 << 20      # Infinity Cache; cold-weight runs rotate through > 2x this
PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = ["paper_2508_19087_amd/csrc/gemm_int8.h", "paper_2508_19087_amd/csrc/gemm_int8.hip",
                  "paper_2508_19087_amd/csrc/gemm_int8_inst.hip", "paper_2508_19087_amd/csrc/reassemble.h",
                  "paper_2508_19087_amd/csrc/select.hip", "paper_2508_19087_amd/csrc/act_frag.hip",
                  "paper_2508_19087_amd/csrc/rowcode.h"]


def kernel_hash() -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(open(os.path.join(ROOT, f), "rb").read())
    return h.hexdigest()[:16]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class Workload:
    """Device buffers of one bench step, built through the library's own calls."""

    def __init__(self):
        import numpy as np
        import torch

        import paper_2508_19087_amd as apt
        import synth
        self.apt, self.torch, self.np = apt, torch, np
        self.stream = torch.cuda.current_stream()
        self.sp = self.stream.cuda_stream
        # The decode GEMMs and the prefill GEMM are independent problems (other
        # tokens, other sequences), so a step issues the decode chain on a second
        # stream of default priority, where its kernels run beside the prefill
        # GEMM on the compute units its last partial round of tiles leaves idle.
        self.side = torch.cuda.Stream()
        self.side_sp = self.side.cuda_stream
        self.overlap = True
        self.unfused_decode = False
        self.packed_prefill = False
        self.dec = [synth.w2a2_decode(1, 4096), synth.w2a2_decode(1, synth.MLP)]
        self.pre = synth.w4a4_prefill()
        dev = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()  # noqa: E731
        self.items = []
        for prob, fp16 in [(self.dec[0], True), (self.dec[1], True), (self.pre, False)]:
            it = {"prob": prob, "fp16": fp16}
            w = apt.pack(dev(prob.w_codes), prob.p)  # weights: packed once
            it["w"] = w
            it["a_codes"] = dev(prob.a_codes)
            it["a_buf"] = torch.empty(apt.apt_packed_bytes(prob.M, prob.K, prob.q), dtype=torch.uint8,
                                      device="cuda")
            it["a_rs"] = torch.empty(prob.M, dtype=torch.int32, device="cuda")
            it["c32"] = torch.empty((prob.M, prob.N), dtype=torch.int32, device="cuda")
            wsb = apt.apt_gemm_workspace_bytes(prob.M, prob.N, prob.K, prob.p, prob.q, None)
            wsa = apt.apt_gemm_act_workspace_bytes(prob.M, prob.N, prob.K, prob.p, prob.q,
                                                   apt.APT_ACT_CODES, None)
            it["ws"] = torch.empty(max(wsb, wsa, 16), dtype=torch.uint8, device="cuda")
            it["ws_bytes"] = wsb
            it["ws_act_bytes"] = wsa
            if fp16:
                it["sa"], it["sw"] = dev(prob.a_scale), dev(prob.w_scale)
                it["c16"] = torch.empty((prob.M, prob.N), dtype=torch.float16, device="cuda")
            self.items.append(it)
        self.ops = sum(it["prob"].ops for it in self.items)
        # Two prefill batches in flight: consecutive steps' prefill calls
        # alternate between the main stream and a third one (default priority),
        # each with its own output, workspace and activation buffers, so the
        # next batch's fragment writer and first tiles start on the compute
        # units the current GEMM's last round leaves idle.  Stream order keeps
        # each buffer set's calls in sequence.
        self.batches = 2
        self.alt = torch.cuda.Stream()
        self.alt_sp = self.alt.cuda_stream
        # With another batch's GEMM in flight, the prefill takes the selected
        # config with one workgroup per tile (grid 0): the persistent round's
        # leftover tiles chained onto its own workgroups are the best schedule
        # for one call at a time, but with two calls in flight the second
        # call's workgroups fill the first one's idle compute units anyway,
        # and one workgroup per tile lets the two interleave (measured: 79.0
        # against 82.4 us per step; with one batch in flight 95.7 against 92.0).
        pre = self.items[2]["prob"]
        sel = apt.select_config(pre.M, pre.N, pre.K, pre.p, pre.q)
        self.pre_cfg_two = type(sel).from_buffer_copy(sel)
        if self.pre_cfg_two.route != apt.APT_ROUTE_XOR:
            self.pre_cfg_two.grid = 0
        wst = apt.apt_gemm_act_workspace_bytes(pre.M, pre.N, pre.K, pre.p, pre.q, apt.APT_ACT_CODES,
                                               self.pre_cfg_two)
        second = dict(self.items[2])
        for key in ("c32", "ws", "a_buf", "a_rs"):
            second[key] = torch.empty_like(self.items[2][key])
        first = dict(self.items[2])
        for st in (first, second):
            st["ws_two"] = torch.empty(max(wst, 16), dtype=torch.uint8, device="cuda")
            st["ws_two_bytes"] = wst
        self.pre_sets = [first, second]
        self.count = 0
        torch.cuda.synchronize()

    def pack_act(self, it, sp=None):
        p = it["prob"]
        sp = sp if sp is not None else self.sp
        st = self.apt.apt_quantize_pack_activations(it["a_codes"].data_ptr(), p.M, p.K, p.q,
                                                    it["a_buf"].data_ptr(), it["a_rs"].data_ptr(),
                                                    sp)
        self.apt.check(st, "apt_quantize_pack_activations")

    def gemm(self, it, w=None, sp=None):
        p = it["prob"]
        w = w if w is not None else it["w"]
        sp = sp if sp is not None else self.sp
        fp16 = it["fp16"]
        st = self.apt.apt_gemm(p.M, p.N, p.K, p.p, p.q, it["a_buf"].data_ptr(), w.data.data_ptr(),
                               it["a_rs"].data_ptr(), w.rowsum.data_ptr(), it["c32"].data_ptr(),
                               it["sa"].data_ptr() if fp16 else None,
                               it["sw"].data_ptr() if fp16 else None,
                               it["c16"].data_ptr() if fp16 else None, None,
                               it["ws"].data_ptr(), it["ws_bytes"], sp)
        self.apt.check(st, "apt_gemm")

    def decode(self, it, w=None, sp=None):
        """The decode GEMM from the token's codes in one launch: apt_gemm_decode
        converts the activation row inside the GEMV (same results as
        pack_act + gemm on the XOR route)."""
        p = it["prob"]
        w = w if w is not None else it["w"]
        sp = sp if sp is not None else self.sp
        st = self.apt.apt_gemm_decode(p.M, p.N, p.K, p.p, p.q, it["a_codes"].data_ptr(),
                                      self.apt.APT_ACT_CODES, w.data.data_ptr(), it["c32"].data_ptr(),
                                      it["sa"].data_ptr(), it["sw"].data_ptr(), it["c16"].data_ptr(),
                                      None, None, sp)
        self.apt.check(st, "apt_gemm_decode")

    def gemm_act(self, it, sp=None, two=False):
        """The GEMM from the activations' codes in one call (apt_gemm_act): on
        the int8 MFMA route the codes go straight into the operand fragments
        (same results as pack_act + gemm).  `two`: the config for two batches
        in flight (pre_cfg_two) and its workspace."""
        p = it["prob"]
        sp = sp if sp is not None else self.sp
        fp16 = it["fp16"]
        ws, wsb = (it["ws_two"], it["ws_two_bytes"]) if two else (it["ws"], it["ws_act_bytes"])
        st = self.apt.apt_gemm_act(p.M, p.N, p.K, p.p, p.q, it["a_codes"].data_ptr(),
                                   self.apt.APT_ACT_CODES, it["w"].data.data_ptr(),
                                   it["w"].rowsum.data_ptr(), it["c32"].data_ptr(),
                                   it["sa"].data_ptr() if fp16 else None,
                                   it["sw"].data_ptr() if fp16 else None,
                                   it["c16"].data_ptr() if fp16 else None, None,
                                   self.pre_cfg_two if two else None,
                                   ws.data_ptr(), wsb, sp)
        self.apt.check(st, "apt_gemm_act")

    def prefill(self, sp=None, it=None, two=False):
        """The prefill problem as the step runs it: apt_gemm_act from the codes,
        or with `packed_prefill` the packer and then apt_gemm (the selected
        config either way; `two`: apt_gemm_act in the two-batch config)."""
        it = it if it is not None else self.items[2]
        if self.packed_prefill:
            self.pack_act(it, sp)
            self.gemm(it, sp=sp)
        else:
            self.gemm_act(it, sp, two=two)

    def step(self):
        """One pass of the path over one batch: the two decode GEMMs from their
        tokens' codes (converted and decomposed into planes inside the GEMV,
        or with `unfused_decode` packed by the packer first), then the
        prefill GEMM from its codes (see prefill).  With `overlap`, the decode
        problems run on the side stream and the prefill on the main one, or,
        with two batches in flight, on the main and the third stream in turn
        (buffer set = step parity); without it, everything on the main one."""
        sp = self.side_sp if self.overlap else self.sp
        for it in self.items[:2]:
            if self.unfused_decode:
                self.pack_act(it, sp)
                self.gemm(it, sp=sp)
            else:
                self.decode(it, sp=sp)
        if self.overlap and self.batches == 2:
            k = self.count % 2
            self.count += 1
            self.prefill(sp=(self.sp, self.alt_sp)[k], it=self.pre_sets[k], two=True)
        else:
            self.prefill()


def prefill_call(wl):
    """The one call of the prefill GEMM the roofline describes (the step's
    form): apt_gemm_act from the codes (fragment writer + GEMM kernel), or
    with packed_prefill apt_gemm on activations packed beforehand (expansion
    + GEMM kernel)."""
    it = wl.items[2]
    if wl.packed_prefill:
        wl.pack_act(it)
        return lambda: wl.gemm(it)
    return lambda: wl.gemm_act(it)


def prefill_call_time(wl, calls: int) -> float:
    """Average seconds per prefill call (prefill_call), timed with HIP events
    on the workload's stream around `calls` back-to-back calls."""
    torch = wl.torch
    call = prefill_call(wl)
    for _ in range(3):
        call()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(wl.stream)
    for _ in range(calls):
        call()
    e1.record(wl.stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e-3 / calls


def quantize_fp16_rates(calls: int = 50):
    """The fused fp16 activation quantizer + packer on the activation shapes
    of the step (prefill 2048x4096 at 4 bits, decode 1x4096 at 2 bits):
    average microseconds per call over `calls` back-to-back calls between two
    events on the stream they run on, and the rate of its algorithmic bytes
    (fp16 input read once, packed planes, row sums and scales written once)
    against the HBM peak."""
    import torch

    import paper_2508_19087_amd as apt
    import synth
    out = []
    stream = torch.cuda.current_stream()
    for M, K, q in [(2048, synth.HIDDEN, 4), (1, synth.HIDDEN, 2)]:
        x = torch.from_numpy(synth.fp16_activations(synth.rng(80, M, K), M, K)).cuda()
        nb = apt.apt_packed_bytes(M, K, q)
        buf = torch.empty(nb, dtype=torch.uint8, device="cuda")
        rs = torch.empty(M, dtype=torch.int32, device="cuda")
        sc = torch.empty(M, dtype=torch.float16, device="cuda")

        def call():
            apt.check(apt.apt_quantize_pack_activations_fp16(
                x.data_ptr(), M, K, q, buf.data_ptr(), rs.data_ptr(), sc.data_ptr(),
                stream.cuda_stream), "apt_quantize_pack_activations_fp16")
        for _ in range(3):
            call()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(calls):
            call()
        e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / calls
        nbytes = 2 * M * K + nb + 4 * M + 2 * M
        gbs = nbytes / us / 1e3
        out.append({"M": M, "K": K, "q": q, "us": round(us, 2), "bytes": nbytes,
                    "GB/s": round(gbs, 1), "frac_hbm": round(gbs / PEAK_HBM_GBS, 4)})
    return out


def route_table(calls: int = 20):
    """Route choice evidence (Sec. V): every route the library has, forced on
    the prefill GEMM and on the two M=1 decode GEMMs of the step, warm
    weights, events around `calls` back-to-back apt_gemm calls."""
    import numpy as np
    import torch

    import paper_2508_19087_amd as apt
    import synth
    dev = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()  # noqa: E731
    C = apt.apt_config_t.make
    routes = [("selected", None),
              ("xor+popcount", C(apt.APT_ROUTE_XOR)),
              ("+-1 planes int8 MFMA", C(apt.APT_ROUTE_PM1_MFMA)),
              ("reassembled int8 MFMA 256x128 g256", C(apt.APT_ROUTE_INT8_MFMA, 256, 128, 128, 4, 2, 256, 3)),
              ("reassembled int8 MFMA 128x128 g512", C(apt.APT_ROUTE_INT8_MFMA, 128, 128, 128, 2, 2, 512, 3)),
              ("reassembled FP4 MFMA 128x128 g512", C(apt.APT_ROUTE_FP4_MFMA, 128, 128, 128, 2, 2, 512, 3))]
    out = {}
    # the step's GEMMs, the W1A1 down projection (FP4 route with FP4 activations) and the
    # W2A4 down projection at 1024 tokens (FP4 route with FP8 activations)
    for prob in [synth.w4a4_prefill(), synth.w2a2_decode(1, 4096), synth.w2a2_decode(1, synth.MLP),
                 synth.sweep_down(0), synth.layer_w2a4("down", 1024)]:
        a = apt.pack(dev(prob.a_codes), prob.q, activations=True)
        w = apt.pack(dev(prob.w_codes), prob.p)
        row = {}
        for name, cfg in routes:
            if cfg is not None and cfg.route == apt.APT_ROUTE_PM1_MFMA and max(prob.p, prob.q) > 7:
                continue
            if cfg is not None and cfg.route == apt.APT_ROUTE_FP4_MFMA and (prob.p > 2 or prob.q > 4):
                continue
            c32 = torch.empty((prob.M, prob.N), dtype=torch.int32, device="cuda")
            wsb = apt.apt_gemm_workspace_bytes(prob.M, prob.N, prob.K, prob.p, prob.q, cfg)
            ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
            sp = torch.cuda.current_stream().cuda_stream

            def call():
                apt.check(apt.apt_gemm(prob.M, prob.N, prob.K, prob.p, prob.q, a.data.data_ptr(),
                                       w.data.data_ptr(), a.rowsum.data_ptr(), w.rowsum.data_ptr(),
                                       c32.data_ptr(), None, None, None, cfg, ws.data_ptr(), wsb, sp),
                          "apt_gemm")
            for _ in range(3):
                call()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            for _ in range(calls):
                call()
            e1.record()
            torch.cuda.synchronize()
            row[name] = round(e0.elapsed_time(e1) * 1e3 / calls, 2)
        out[prob.name] = row
    return out


def search_table(calls: int = 20):
    """Config selection evidence (Sec. V-B): for every workload shape, the
    model's config and the best-kernel search module's pick (apt_search_config
    over every runnable config), each timed with events around `calls`
    back-to-back apt_gemm calls (warm weights, int32 output)."""
    import numpy as np
    import torch

    import paper_2508_19087_amd as apt
    import synth
    dev = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()  # noqa: E731
    probs = [synth.w1a2_small()]
    probs += [synth.w2a2_decode(M, N) for M in (1, 4, 8) for N in (4096, synth.MLP)]
    probs += [synth.w4a4_prefill()] + [synth.sweep_down(i) for i in range(len(synth.SWEEP_BITS))]
    probs += [synth.layer_w2a4(name, M) for M in (1, 1024) for name in ("q", "gate", "down")]

    def short(c):
        if c.route == apt.APT_ROUTE_XOR:
            return "xor"
        if c.route == apt.APT_ROUTE_PM1_MFMA:
            return "pm1"
        t = "%s %dx%d/%dx%d g%d" % ("fp4" if c.route == apt.APT_ROUTE_FP4_MFMA else "int8",
                                    c.bm, c.bn, c.waves_m, c.waves_n, c.grid)
        if c.split_n:
            t += " +%dx%d@%d g%d" % (c.tail_bm, c.tail_bn, c.split_n, c.tail_grid)
        return t

    rows = []
    apt.apt_config_table_clear()
    for prob in probs:
        a = apt.pack(dev(prob.a_codes), prob.q, activations=True)
        w = apt.pack(dev(prob.w_codes), prob.p)
        c32 = torch.empty((prob.M, prob.N), dtype=torch.int32, device="cuda")
        sp = torch.cuda.current_stream().cuda_stream

        def timed(cfg):
            wsb = apt.apt_gemm_workspace_bytes(prob.M, prob.N, prob.K, prob.p, prob.q, cfg)
            ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")

            def call():
                apt.check(apt.apt_gemm(prob.M, prob.N, prob.K, prob.p, prob.q, a.data.data_ptr(),
                                       w.data.data_ptr(), a.rowsum.data_ptr(), w.rowsum.data_ptr(),
                                       c32.data_ptr(), None, None, None, cfg, ws.data_ptr(), wsb, sp),
                          "apt_gemm")
            for _ in range(3):
                call()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            for _ in range(calls):
                call()
            e1.record()
            torch.cuda.synchronize()
            return e0.elapsed_time(e1) * 1e3 / calls

        model = apt.select_config(prob.M, prob.N, prob.K, prob.p, prob.q)
        t_model = timed(model)
        best, t_search = apt.search_config(a, w)
        t_best = timed(best)
        rows.append({"problem": prob.name, "M": prob.M, "N": prob.N, "K": prob.K, "p": prob.p,
                     "q": prob.q, "model": short(model), "model_us": round(t_model, 2),
                     "searched": short(best), "searched_us": round(t_best, 2),
                     "search_timing_us": round(t_search, 2), "searched_config": best.as_dict()})
        log("bench: search %s: model %s %.2f us, searched %s %.2f us"
            % (prob.name, short(model), t_model, short(best), t_best))
        del a, w, c32
    apt.apt_config_table_clear()
    return rows


def calibrate(calls: int = 20):
    """Calibration of the selector's MFMA model (csrc/select.hip): for each
    model tile shape and operand class (int8 operands at weight widths 2, 4 and
    8 with 4-bit activations; FP4 operands at W2A2), apt_gemm call times with
    M = 2048 at K = 2048 and 6144 (8 and 24 chunk pairs), over one full round
    of tiles (N chosen so), and for shapes with two workgroups per compute unit
    also over half a round (one per compute unit).  The K slope gives the
    microseconds per chunk pair, its intercept the fixed time."""
    import numpy as np
    import torch

    import paper_2508_19087_amd as apt
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    shapes = [(256, 256, 4, 2, 1), (512, 128, 8, 1, 1), (256, 128, 4, 1, 2), (256, 128, 4, 2, 1),
              (128, 128, 2, 2, 2)]
    classes = [("int8_w2", apt.APT_ROUTE_INT8_MFMA, 2, 4), ("int8_w4", apt.APT_ROUTE_INT8_MFMA, 4, 4),
               ("int8_w8", apt.APT_ROUTE_INT8_MFMA, 8, 4), ("fp4_w2a2", apt.APT_ROUTE_FP4_MFMA, 2, 2)]
    M, Ks = 2048, (2048, 6144)
    g = np.random.default_rng(11)
    sp = torch.cuda.current_stream().cuda_stream
    out = []
    for cname, route, p, q in classes:
        ops = {}
        for K in Ks:
            ac = torch.from_numpy(g.integers(-(1 << (q - 1)), 1 << (q - 1), (M, K), dtype=np.int8)).cuda()
            a = apt.pack(ac, q, activations=True)
            for bm, bn, wm, wn, per_cu in shapes:
                for label, tiles in (("full", cus * per_cu), ("alone", cus)):
                    if label == "alone" and per_cu == 1:
                        continue
                    N = tiles // (M // bm) * bn
                    key = (N, K)
                    if key not in ops:
                        wc = torch.from_numpy(g.integers(-(1 << (p - 1)), 1 << (p - 1), (N, K),
                                                         dtype=np.int8)).cuda()
                        ops[key] = apt.pack(wc, p)
                    w = ops[key]
                    cfg = apt.apt_config_t.make(route, bm, bn, 128, wm, wn, 0, 3)
                    wsb = apt.apt_gemm_workspace_bytes(M, N, K, p, q, cfg)
                    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
                    c32 = torch.empty((M, N), dtype=torch.int32, device="cuda")

                    def call():
                        apt.check(apt.apt_gemm(M, N, K, p, q, a.data.data_ptr(), w.data.data_ptr(),
                                               a.rowsum.data_ptr(), w.rowsum.data_ptr(), c32.data_ptr(),
                                               None, None, None, cfg, ws.data_ptr(), wsb, sp), "apt_gemm")
                    for _ in range(3):
                        call()
                    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    torch.cuda.synchronize()
                    e0.record()
                    for _ in range(calls):
                        call()
                    e1.record()
                    torch.cuda.synchronize()
                    us = e0.elapsed_time(e1) * 1e3 / calls
                    out.append({"class": cname, "shape": [bm, bn, wm, wn], "round": label, "M": M, "N": N,
                                "K": K, "us": round(us, 2)})
                    log("bench: calibrate %s %dx%d/%dx%d %s K=%d: %.2f us" % (cname, bm, bn, wm, wn, label,
                                                                              K, us))
                    del ws, c32
        del ops
    # the model's figures: pair time (slope over the 16 extra pairs), fixed time (intercept)
    fits = []
    for cname, _, _, _ in classes:
        for bm, bn, wm, wn, per_cu in shapes:
            def t(label, K):
                return [r["us"] for r in out if r["class"] == cname and r["shape"] == [bm, bn, wm, wn]
                        and r["round"] == label and r["K"] == K][0]
            pair = (t("full", 6144) - t("full", 2048)) / 16.0
            fixed = t("full", 2048) - 8 * pair
            alone = (t("alone", 6144) - t("alone", 2048)) / 16.0 if per_cu > 1 else pair
            fits.append({"class": cname, "shape": [bm, bn, wm, wn], "per_cu": per_cu,
                         "pair_us": round(pair, 3), "pair_alone_us": round(alone, 3),
                         "fixed_us": round(fixed, 2)})
    return {"cus": cus, "timings": out, "model": fits}


def format_sweep(calls: int = 20):
    """The operand formats of the reassembled MFMA route against each other:
    int8 against FP6 (E2M3) operands on W3A3 problems (the W3A3 down
    projection 512x4096x11008, 2048x11008x4096 and 1024x4096x4096) and int8
    against FP8 (E4M3) operands on W4A4 problems (2048x11008x4096, the prefill
    workload, and 512x4096x11008), on every tile shape with one workgroup per
    tile and with one persistent round; HIP events around `calls`
    back-to-back apt_gemm calls (warm weights, int32 output)."""
    import numpy as np
    import torch

    import paper_2508_19087_amd as apt
    import synth
    dev = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()  # noqa: E731
    shapes = [(256, 256, 4, 2, 1), (512, 128, 8, 1, 1), (256, 128, 4, 1, 2), (256, 128, 4, 2, 1),
              (128, 128, 2, 2, 2)]
    probs = [synth.sweep_down(3), synth.random_problem(synth.rng(9), 2048, 11008, 4096, 3, 3),
             synth.random_problem(synth.rng(10), 1024, 4096, 4096, 3, 3), synth.w4a4_prefill(),
             synth.random_problem(synth.rng(11), 512, 4096, 11008, 4, 4)]
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    sp = torch.cuda.current_stream().cuda_stream
    rows = []
    for prob in probs:
        a = apt.pack(dev(prob.a_codes), prob.q, activations=True)
        w = apt.pack(dev(prob.w_codes), prob.p)
        c32 = torch.empty((prob.M, prob.N), dtype=torch.int32, device="cuda")
        fl_name, fl_route = (("fp6_us", apt.APT_ROUTE_FP6_MFMA) if max(prob.p, prob.q) <= 3
                             else ("fp8_us", apt.APT_ROUTE_FP8_MFMA))
        for bm, bn, wm, wn, per_cu in shapes:
            for grid in (0, cus * per_cu):
                row = {"problem": "%dx%dx%d W%dA%d" % (prob.M, prob.N, prob.K, prob.p, prob.q),
                       "shape": "%dx%d/%dx%d g%d" % (bm, bn, wm, wn, grid)}
                for name, route in (("int8_us", apt.APT_ROUTE_INT8_MFMA), (fl_name, fl_route)):
                    cfg = apt.apt_config_t.make(route, bm, bn, 128, wm, wn, grid, 3)
                    wsb = apt.apt_gemm_workspace_bytes(prob.M, prob.N, prob.K, prob.p, prob.q, cfg)
                    ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")

                    def call():
                        apt.check(apt.apt_gemm(prob.M, prob.N, prob.K, prob.p, prob.q, a.data.data_ptr(),
                                               w.data.data_ptr(), a.rowsum.data_ptr(), w.rowsum.data_ptr(),
                                               c32.data_ptr(), None, None, None, cfg, ws.data_ptr(), wsb, sp),
                                  "apt_gemm")
                    for _ in range(3):
                        call()
                    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    torch.cuda.synchronize()
                    e0.record()
                    for _ in range(calls):
                        call()
                    e1.record()
                    torch.cuda.synchronize()
                    row[name] = round(e0.elapsed_time(e1) * 1e3 / calls, 2)
                    del ws
                rows.append(row)
                log("bench: formats %s %s int8 %.2f %s %.2f us" % (row["problem"], row["shape"],
                                                                    row["int8_us"], fl_name[:3],
                                                                    row[fl_name]))
        del a, w, c32
    return rows


def vendor_int8(calls: int = 50):
    """Context for the prefill GEMM: the vendor library's dense int8 GEMM
    (torch._int_mm, int32 result) on M=2048, N=11008, K=4096 with operands
    already int8 in memory (no bit-planes, no reassembly), the weight as an
    [N][K] row-major matrix (passed transposed) and as a [K][N] one; HIP events
    around `calls` back-to-back calls after 3 warm-up calls."""
    import torch
    g = torch.Generator().manual_seed(12)
    M, N, K = 2048, 11008, 4096
    a = torch.randint(-8, 8, (M, K), dtype=torch.int8, generator=g).cuda()
    w = torch.randint(-8, 8, (N, K), dtype=torch.int8, generator=g).cuda()
    wkn = w.t().contiguous()
    rows = []
    for name, b in (("weight [N][K] (transposed view)", w.t()), ("weight [K][N]", wkn)):
        out = torch._int_mm(a, b)
        ref = torch._int_mm(a, wkn) if name != "weight [K][N]" else out
        assert torch.equal(out, ref)
        for _ in range(3):
            torch._int_mm(a, b)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(calls):
            torch._int_mm(a, b)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / calls
        rows.append({"gemm": "torch._int_mm %dx%dx%d int8, %s" % (M, N, K, name), "us": round(us, 2),
                     "TOPS": round(2.0 * M * N * K / us / 1e6, 1)})
        log("bench: vendor int8 %s: %.2f us" % (name, us))
    # the library's own call on the same shape at W4A4, for the same timing method
    wl = Workload()
    us = prefill_call_time(wl, calls) * 1e6
    rows.append({"gemm": "apt_gemm W4A4 2048x11008x4096 (bit-planes, selected config)", "us": round(us, 2),
                 "TOPS": round(2.0 * M * N * K / us / 1e6, 1)})
    return rows


MFMA_ISSUE_MODES = [
    (0, "16 MFMAs per k-step, registers only (one wave per SIMD)"),
    (1, "+ 4 LDS reads of the next k-step's A fragments"),
    (2, "+ one workgroup barrier per chunk of 4 k-steps"),
    (3, "+ 4 buffer loads x 16 B per lane per k-step (B fragments, a chunk ahead)"),
    (4, "mode 2 + 4 buffer loads x 4 B per lane per k-step"),
    (5, "mode 2 + 2 buffer loads x 16 B per lane per k-step"),
    (6, "mode 2 + 4 x 16 B loads per k-step straight into LDS, read back a k-step ahead"),
    (7, "mode 3's per-SIMD pattern on two waves per SIMD (8 MFMAs + 2 loads per wave and k-step)"),
]


def mfma_issue(blocks: int = 256, chunks: int = 4000):
    """The MFMA-issue probe (probes/mfma_issue.hip, libapt_probe.so): cycles
    per v_mfma_i32_32x32x32_i8 per SIMD for each part of the GEMM loop's
    instruction pattern, with the shader clock read from s_memtime against
    s_memrealtime, on pseudo-random operand bytes, then modes 0, 3 and 7 on
    sparse bytes (one small nonzero byte per dword), on 4-bit bipolar values
    (random odd bytes in [-15, 15]) and on 4-bit codes (random bytes in
    [0, 15], what the reassembled int8 route multiplies at W4A4); mode 0's
    accumulators are checked against a closed form (result_checked)."""
    import ctypes
    lib = probe_lib()
    rows = []
    kinds = ["random", "sparse", "bipolar4", "code4"]
    runs = [(mode, what, 0) for mode, what in MFMA_ISSUE_MODES]
    runs += [(m, MFMA_ISSUE_MODES[m][1], d) for d in (1, 2, 3) for m in (0, 3, 7)]
    for mode, what, data in runs:
        res = (ctypes.c_double * 4)()
        rc = lib.apt_probe_mfma_issue(mode, blocks, chunks, data, res)
        if rc != 0:
            raise RuntimeError("mfma issue probe mode %d failed at step %d%s" %
                               (mode, rc, " (accumulator sums differ from the closed form)" if rc == 5 else ""))
        rows.append({"mode": mode, "operands": kinds[data], "pattern": what,
                     "cycles_per_mfma": round(res[0], 1),
                     "clock_GHz": round(res[1], 3), "us_per_chunk": round(res[2], 3),
                     "result_checked": bool(res[3])})
        log("bench: mfma issue mode %d: %.1f cycles per MFMA at %.2f GHz" % (mode, res[0], res[1]))
    return rows


def graph_of(torch, launch):
    """A HIP graph (torch.cuda.CUDAGraph) of launch(stream_ptr), captured on a
    side stream after one eager warm-up there."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        launch(side.cuda_stream)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        launch(torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    return g


def decode_cold(wl, reps: int = 4):
    """The M=1 decode GEMMs with cold weights: one GEMM per weight copy, with
    enough copies (> 2x the Infinity Cache) that every launch reads HBM.  The
    rotation is captured as one HIP graph and replayed between two events, so
    the launches follow each other as in a decode loop (no host launch gaps);
    every replay's output is checked against the eager result."""
    torch, apt = wl.torch, wl.apt
    out = {}
    for it in wl.items[:2]:
        p = it["prob"]
        wbytes = it["w"].data.numel()
        copies = max(8, int(2 * MALL_BYTES // wbytes) + 1)
        ws = []
        for _ in range(copies):
            ws.append(apt.Packed(it["w"].data.clone(), it["w"].rowsum.clone(), p.N, p.K, p.p))
        wl.pack_act(it)
        wl.gemm(it)
        torch.cuda.synchronize()
        ref32, ref16 = it["c32"].clone(), it["c16"].clone()

        def launch(sp):
            for w in ws:
                wl.gemm(it, w, sp)
        g = graph_of(torch, launch)
        times = []
        for r in range(reps):
            it["c32"].zero_()
            it["c16"].zero_()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            g.replay()
            e1.record()
            torch.cuda.synchronize()
            assert torch.equal(it["c32"], ref32) and torch.equal(it["c16"], ref16), "graph replay"
            if r > 0:
                times.append(e0.elapsed_time(e1) / copies)
        t = sorted(times)[len(times) // 2] * 1e-3
        bytes_alg = (p.N * p.K * p.p + p.M * p.K * p.q) / 8 + p.M * p.N * (4 + 2) + 2 * (p.M + p.N)
        out["m1_n%d_k%d" % (p.N, p.K)] = {
            "us_per_gemm": round(t * 1e6, 3), "algorithmic_bytes": int(bytes_alg),
            "achieved_GBs": round(bytes_alg / t / 1e9, 1), "peak_GBs": PEAK_HBM_GBS,
            "frac": round(bytes_alg / t / 1e9 / PEAK_HBM_GBS, 4), "weight_copies": copies,
            "effective_TOPS": round(p.ops / t / 1e12, 4),
            "method": "HIP graph of %d back-to-back GEMMs, one per cold weight copy" % copies}
        del ws, g
    out["read_ceiling_same_bytes"] = read_ceiling(torch, wl.items[1]["w"].data, reps)
    return out


def replay_us(torch, g, n, reps: int = 4, before=None, check=None) -> float:
    """Median microseconds per launch group of graph g (n groups per replay),
    replay 0 untimed; before() runs ahead of and check() after each replay."""
    times = []
    for r in range(reps):
        if before is not None:
            before()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        if check is not None:
            check()
        if r > 0:
            times.append(e0.elapsed_time(e1) * 1e3 / n)
    return sorted(times)[len(times) // 2]


def decode_token_cold(wl, reps: int = 4):
    """One token's decode GEMM as a whole, with cold weights: from the token's
    activations (int8 codes, or fp16 values quantized per row) to the int32
    and fp16 outputs.  Unfused = the packer (or the fp16 quantizer-packer)
    then apt_gemm, two launches; fused = apt_gemm_decode, one launch that
    converts the row inside the GEMV.  Each variant is one HIP graph over the
    cold weight copies; every replay's outputs are checked, and the fused
    outputs must equal the unfused ones bit for bit."""
    torch, apt, np = wl.torch, wl.apt, wl.np
    import synth
    out = {}
    for it in wl.items[:2]:
        p = it["prob"]
        wbytes = it["w"].data.numel()
        copies = max(8, int(2 * MALL_BYTES // wbytes) + 1)
        ws = [it["w"].data.clone() for _ in range(copies)]
        x16 = torch.from_numpy(synth.fp16_activations(synth.rng(81, p.N, p.K), p.M, p.K)).cuda()
        sa_q = torch.empty(p.M, dtype=torch.float16, device="cuda")
        c32 = torch.empty((p.M, p.N), dtype=torch.int32, device="cuda")
        c16 = torch.empty((p.M, p.N), dtype=torch.float16, device="cuda")
        rowsum = it["w"].rowsum

        def gemm(w, sp, sa):
            apt.check(apt.apt_gemm(p.M, p.N, p.K, p.p, p.q, it["a_buf"].data_ptr(), w.data_ptr(),
                                   it["a_rs"].data_ptr(), rowsum.data_ptr(), c32.data_ptr(),
                                   sa.data_ptr(), it["sw"].data_ptr(), c16.data_ptr(), None,
                                   it["ws"].data_ptr(), it["ws_bytes"], sp), "apt_gemm")

        def unfused_codes(sp):
            for w in ws:
                wl.pack_act(it, sp)
                gemm(w, sp, it["sa"])

        def fused_codes(sp):
            for w in ws:
                apt.check(apt.apt_gemm_decode(p.M, p.N, p.K, p.p, p.q, it["a_codes"].data_ptr(),
                                              apt.APT_ACT_CODES, w.data_ptr(), c32.data_ptr(),
                                              it["sa"].data_ptr(), it["sw"].data_ptr(),
                                              c16.data_ptr(), None, None, sp), "apt_gemm_decode")

        def unfused_fp16(sp):
            for w in ws:
                apt.check(apt.apt_quantize_pack_activations_fp16(
                    x16.data_ptr(), p.M, p.K, p.q, it["a_buf"].data_ptr(), it["a_rs"].data_ptr(),
                    sa_q.data_ptr(), sp), "apt_quantize_pack_activations_fp16")
                gemm(w, sp, sa_q)

        def fused_fp16(sp):
            for w in ws:
                apt.check(apt.apt_gemm_decode(p.M, p.N, p.K, p.p, p.q, x16.data_ptr(),
                                              apt.APT_ACT_FP16, w.data_ptr(), c32.data_ptr(), None,
                                              it["sw"].data_ptr(), c16.data_ptr(), sa_q.data_ptr(),
                                              None, sp), "apt_gemm_decode")
        row = {}
        for src, pair in (("codes", (unfused_codes, fused_codes)), ("fp16", (unfused_fp16, fused_fp16))):
            refs = None
            for name, fn in zip(("unfused", "fused"), pair):
                fn(wl.sp)
                torch.cuda.synchronize()
                got = (c32.clone(), c16.clone(), sa_q.clone())
                if refs is None:
                    refs = got
                else:
                    assert all(torch.equal(a, b) for a, b in zip(got[:2], refs[:2])), \
                        "fused %s output differs from the unfused path" % src
                    if src == "fp16":
                        assert torch.equal(got[2], refs[2]), "fused fp16 scales differ"
                g = graph_of(torch, fn)

                def zero():
                    c32.zero_()
                    c16.zero_()

                def check():
                    assert torch.equal(c32, refs[0]) and torch.equal(c16, refs[1]), "graph replay"
                row["%s_%s_us" % (src, name)] = round(replay_us(torch, g, copies, reps, zero, check), 3)
                del g
        row["launches"] = {"unfused": 2, "fused": 1}
        row["weight_copies"] = copies
        out["m1_n%d_k%d" % (p.N, p.K)] = row
        del ws
    return out


def probe_lib():
    """The measurement probes (probes/*.hip, libapt_probe.so; not part of
    libapt.so)."""
    import ctypes

    import torch  # noqa: F401  (the HIP runtime torch loaded serves the probe library too)
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2508_19087_amd", "libapt_probe.so"))
    lib.apt_probe_mfma_issue.argtypes = [ctypes.c_int] * 4 + [ctypes.POINTER(ctypes.c_double)]
    lib.apt_probe_mfma_issue.restype = ctypes.c_int
    lib.apt_probe_read_blocks.argtypes = [ctypes.c_int64, ctypes.c_int]
    lib.apt_probe_read_blocks.restype = ctypes.c_int64
    lib.apt_probe_read_xor.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_int,
                                       ctypes.c_void_p, ctypes.c_void_p]
    lib.apt_probe_read_xor.restype = ctypes.c_int
    return lib


READ_VECS, READ_NT = 2, 1  # read probe: 16-byte vectors per lane, non-temporal loads


def read_ceiling(torch, buf, reps: int = 4):
    """A read-only cold reference for a decode GEMM's weight bytes: the read
    probe (probes/read_stream.hip) reads every byte of each of enough copies of
    the buffer (> 2x the Infinity Cache) that every read comes from HBM, with
    16-byte non-temporal loads, two per lane, folded by XOR to one word per
    workgroup; replayed as one HIP graph like the GEMM rotation, and every
    replay's words are checked against the XOR of the buffer's words."""
    import numpy as np
    lib = probe_lib()
    n = buf.numel() * buf.element_size()
    copies = max(8, int(2 * MALL_BYTES // n) + 1)
    srcs = [buf.clone() for _ in range(copies)]
    nb = lib.apt_probe_read_blocks(n, READ_VECS)
    outs = [torch.empty(nb, dtype=torch.int32, device="cuda") for _ in srcs]

    def launch(sp):
        for x, o in zip(srcs, outs):
            rc = lib.apt_probe_read_xor(x.data_ptr(), n, READ_VECS, READ_NT, o.data_ptr(), sp)
            if rc != 0:
                raise RuntimeError("read probe launch failed (%d)" % rc)
    g = graph_of(torch, launch)
    want = np.bitwise_xor.reduce(buf.cpu().numpy().view(np.uint32))
    times = []
    for r in range(reps):
        for o in outs:
            o.zero_()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        got = np.bitwise_xor.reduce(torch.stack(outs).cpu().numpy().view(np.uint32), axis=1)
        assert (got == want).all(), "read probe replay"
        if r > 0:
            times.append(e0.elapsed_time(e1) / copies)
    t = sorted(times)[len(times) // 2] * 1e-3
    return {"bytes_read": n, "us": round(t * 1e6, 3), "read_GBs": round(n / t / 1e9, 1),
            "frac_hbm": round(n / t / 1e9 / PEAK_HBM_GBS, 4), "copies": copies,
            "method": "HIP graph of the read probe over each cold copy (16-byte non-temporal "
                      "loads, %d per lane; every byte read once, XOR-folded to one checked word "
                      "per workgroup)" % READ_VECS}


def decode_layer_cold(wl, reps: int = 4):
    """One token through the linears of the W2A4 7B-class decoder layer with
    cold weights: q/k/v fused along N (one packed [3*4096][4096] matrix against
    their shared input), o, gate/up fused (N = 2*11008) and down, four GEMMs
    with fp16 output per layer.  Three forms: the GEMMs alone on activations
    packed beforehand (four apt_gemm launches), and from each GEMM's fp16
    input: the fp16 quantizer-packer then apt_gemm (eight launches), or
    apt_gemm_decode (four launches, the row quantized inside each).  Enough
    layer copies (> 2x the Infinity Cache) are rotated in one HIP graph that
    every launch reads HBM; every replay's outputs are checked against the
    eager result, and the two fp16-input forms must agree bit for bit."""
    torch, apt, np = wl.torch, wl.apt, wl.np
    import synth
    dev = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()  # noqa: E731
    groups = [["q", "k", "v"], ["o"], ["gate", "up"], ["down"]]
    gemms = []
    bytes_alg = 0.0
    ops = 0
    for gi, parts in enumerate(groups):
        probs = [synth.layer_w2a4(name, 1) for name in parts]
        p0 = probs[0]
        w_codes = np.concatenate([pr.w_codes for pr in probs], 0)
        N, K, M = w_codes.shape[0], p0.K, 1
        g = {"N": N, "K": K, "p": p0.p, "q": p0.q}
        g["w"] = apt.pack(dev(w_codes), p0.p)
        g["a"] = apt.pack(dev(p0.a_codes), p0.q, activations=True)
        g["sa"] = dev(p0.a_scale)
        g["sw"] = dev(np.concatenate([pr.w_scale for pr in probs]))
        g["c16"] = torch.empty((M, N), dtype=torch.float16, device="cuda")
        g["x16"] = dev(synth.fp16_activations(synth.rng(82, gi), M, K))
        g["xq"] = torch.empty_like(g["a"].data)
        g["xq_rs"] = torch.empty(M, dtype=torch.int32, device="cuda")
        g["xq_s"] = torch.empty(M, dtype=torch.float16, device="cuda")
        wsb = apt.apt_gemm_workspace_bytes(M, N, K, p0.p, p0.q, None)
        g["ws"], g["ws_bytes"] = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda"), wsb
        gemms.append(g)
        bytes_alg += (N * K * p0.p + M * K * p0.q) / 8 + M * N * 2 + 2 * (M + N)
        ops += 2 * M * N * K
    layer_bytes = sum(g["w"].data.numel() for g in gemms)
    copies = max(8, int(2 * MALL_BYTES // layer_bytes) + 1)
    wcopies = [[apt.Packed(g["w"].data.clone(), g["w"].rowsum.clone(), g["N"], g["K"], g["p"])
                for g in gemms] for _ in range(copies)]

    def gemm(g, w, sp, a, a_rs, sa):
        apt.check(apt.apt_gemm(1, g["N"], g["K"], g["p"], g["q"], a.data_ptr(), w.data.data_ptr(),
                               a_rs.data_ptr(), w.rowsum.data_ptr(), None, sa.data_ptr(),
                               g["sw"].data_ptr(), g["c16"].data_ptr(), None, g["ws"].data_ptr(),
                               g["ws_bytes"], sp), "apt_gemm")

    def gemms_only(ws_list, sp):
        for g, w in zip(gemms, ws_list):
            gemm(g, w, sp, g["a"].data, g["a"].rowsum, g["sa"])

    def unfused_fp16(ws_list, sp):
        for g, w in zip(gemms, ws_list):
            apt.check(apt.apt_quantize_pack_activations_fp16(
                g["x16"].data_ptr(), 1, g["K"], g["q"], g["xq"].data_ptr(), g["xq_rs"].data_ptr(),
                g["xq_s"].data_ptr(), sp), "apt_quantize_pack_activations_fp16")
            gemm(g, w, sp, g["xq"], g["xq_rs"], g["xq_s"])

    def fused_fp16(ws_list, sp):
        for g, w in zip(gemms, ws_list):
            apt.check(apt.apt_gemm_decode(1, g["N"], g["K"], g["p"], g["q"], g["x16"].data_ptr(),
                                          apt.APT_ACT_FP16, w.data.data_ptr(), None, None,
                                          g["sw"].data_ptr(), g["c16"].data_ptr(), None, None, sp),
                      "apt_gemm_decode")
    res = {}
    fp16_ref = None
    for name, run, launches in (("gemms_only", gemms_only, 4), ("unfused_fp16", unfused_fp16, 8),
                                ("fused_fp16", fused_fp16, 4)):
        run([g["w"] for g in gemms], wl.sp)
        torch.cuda.synchronize()
        refs = [g["c16"].clone() for g in gemms]
        if name == "unfused_fp16":
            fp16_ref = refs
        elif name == "fused_fp16":
            assert all(torch.equal(a, b) for a, b in zip(refs, fp16_ref)), "fused layer differs"

        def launch(sp, run=run):
            for ws_list in wcopies:
                run(ws_list, sp)
        graph = graph_of(torch, launch)

        def zero():
            for g in gemms:
                g["c16"].zero_()

        def check(refs=refs):
            assert all(torch.equal(g["c16"], r) for g, r in zip(gemms, refs)), "layer graph replay"
        res[name] = (replay_us(torch, graph, copies, reps, zero, check), launches)
        del graph
    t = res["gemms_only"][0] * 1e-6
    return {"us_per_layer": round(t * 1e6, 3), "launches_per_layer": 4,
            "algorithmic_bytes": int(bytes_alg), "achieved_GBs": round(bytes_alg / t / 1e9, 1),
            "peak_GBs": PEAK_HBM_GBS, "frac": round(bytes_alg / t / 1e9 / PEAK_HBM_GBS, 4),
            "layer_copies": copies, "effective_TOPS": round(ops / t / 1e12, 4),
            "from_fp16_inputs": {k: {"us_per_layer": round(v[0], 3), "launches_per_layer": v[1]}
                                 for k, v in res.items() if k != "gemms_only"},
            "method": "HIP graph of %d layers (q/k/v fused, o, gate/up fused, down), one per cold "
                      "copy of the layer's weights; fp16 output; us_per_layer, frac: the GEMMs "
                      "on activations packed beforehand" % copies}


def decode_sweep(reps: int = 4):
    """Cold-weight time of one M=1 W2A4 GEMM (K = 4096, int32 output) against
    N, each as one HIP graph over enough weight copies (> 2x the Infinity
    Cache) that every launch reads HBM: the per-launch fixed cost and the
    streaming rate of the decode route."""
    import numpy as np
    import torch

    import paper_2508_19087_amd as apt
    g = np.random.default_rng(1)
    K, p, q = 4096, 2, 4
    rows = []
    for N in (4096, 12288, 22016, 44032, 88064):
        wc = torch.from_numpy(g.integers(-2, 2, (N, K), dtype=np.int8)).cuda()
        ac = torch.from_numpy(g.integers(-8, 8, (1, K), dtype=np.int8)).cuda()
        w = apt.pack(wc, p)
        a = apt.pack(ac, q, activations=True)
        nb = w.data.numel()
        copies = max(8, int(2 * MALL_BYTES // nb) + 1)
        ws = [apt.Packed(w.data.clone(), w.rowsum.clone(), N, K, p) for _ in range(copies)]
        c32 = torch.empty((1, N), dtype=torch.int32, device="cuda")

        def launch(sp, ws=ws, a=a, c32=c32, N=N):
            for wi in ws:
                apt.check(apt.apt_gemm(1, N, K, p, q, a.data.data_ptr(), wi.data.data_ptr(),
                                       a.rowsum.data_ptr(), wi.rowsum.data_ptr(), c32.data_ptr(),
                                       None, None, None, None, None, 0, sp), "apt_gemm")
        gr = graph_of(torch, launch)
        ts = []
        for r in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            gr.replay()
            e1.record()
            torch.cuda.synchronize()
            if r > 0:
                ts.append(e0.elapsed_time(e1) * 1e3 / copies)
        t = sorted(ts)[len(ts) // 2]
        bytes_alg = (N * K * p + K * q) / 8 + 4 * N
        ceil = read_ceiling(torch, w.data, reps)
        rows.append({"N": N, "K": K, "weight_bytes": nb, "copies": copies, "us": round(t, 3),
                     "GB/s": round(bytes_alg / t / 1e3, 1),
                     "frac_hbm": round(bytes_alg / t / 1e3 / PEAK_HBM_GBS, 4),
                     "read_ceiling_us": ceil["us"], "read_ceiling_frac_hbm": ceil["frac_hbm"]})
        log("bench: decode sweep N=%d %.2f us" % (N, t))
        del ws, gr
    # the launch floor in the same setting: a graph of one-element kernels
    one = torch.zeros(1, dtype=torch.int32, device="cuda")

    def tiny(sp):
        for _ in range(200):
            one.add_(1)
    gt = graph_of(torch, tiny)
    ts = []
    for r in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        gt.replay()
        e1.record()
        torch.cuda.synchronize()
        if r > 0:
            ts.append(e0.elapsed_time(e1) * 1e3 / 200)
    rows.append({"launch_floor_us": round(sorted(ts)[len(ts) // 2], 3),
                 "method": "HIP graph of 200 one-element kernels (torch add_), us per kernel"})
    return rows


DECODE_SHAPES = [(0, 0, 0), (8, 4, 1), (8, 0, 4), (1, 4, 1), (1, 2, 1), (1, 0, 4), (1, 0, 2)]


def decode_shapes(reps: int = 4):
    """XOR-route launch shapes for decode batches (M = 2, 4, 8) with cold
    weights: for each problem, the packed-activation GEMM (apt_gemm) and the
    fused forms (apt_gemm_decode from int8 codes and from fp16) in every
    (mt, waves_m, waves_n) of DECODE_SHAPES, (0, 0, 0) being the library's
    own choice.  Each entry is one HIP graph over enough weight copies
    (> 2x the Infinity Cache) that every launch reads HBM; every shape's
    int32 output must equal the first one's.  Prints a text table."""
    import torch

    import paper_2508_19087_amd as apt
    import synth
    sp0 = torch.cuda.current_stream().cuda_stream
    lines = []
    hdr = "%6s %6s %5s %2s %-7s" % ("N", "K", "WpAq", "M", "source") + "".join(
        "%9s" % ("auto" if s == (0, 0, 0) else "%d/%d/%d" % s) for s in DECODE_SHAPES) + "  best"
    lines.append(hdr)
    for (N, K, p, q) in [(4096, 4096, 2, 2), (11008, 4096, 2, 2), (4096, 4096, 2, 4), (11008, 4096, 2, 4),
                         (4096, 11008, 2, 4), (16384, 4096, 2, 4), (22016, 4096, 2, 4)]:
        g = synth.rng(83, N, K)
        w = apt.pack(torch.from_numpy(synth.uniform_codes(g, N, K, p)).cuda(), p)
        copies = max(8, int(2 * MALL_BYTES // w.data.numel()) + 1)
        ws = [w.data.clone() for _ in range(copies)]
        sw = torch.from_numpy(synth.scales(g, N, *synth.W_SCALE_RANGE)).cuda()
        for M in (2, 4, 8):
            xc = torch.from_numpy(synth.uniform_codes(g, M, K, q)).cuda()
            x16 = torch.from_numpy(synth.fp16_activations(g, M, K)).cuda()
            sa = torch.from_numpy(synth.scales(g, M, *synth.A_SCALE_RANGE)).cuda()
            a = apt.pack(xc, q, activations=True)
            c32 = torch.empty((M, N), dtype=torch.int32, device="cuda")
            c16 = torch.empty((M, N), dtype=torch.float16, device="cuda")
            so = torch.empty(M, dtype=torch.float16, device="cuda")
            for src in ("packed", "codes", "fp16"):
                ref, ts = None, []
                for mt, wm, wn in DECODE_SHAPES:
                    cfg = apt.apt_config_t.make(apt.APT_ROUTE_XOR, waves_m=wm, waves_n=wn, mt=mt)

                    def launch(sp, cfg=cfg, src=src):
                        for wi in ws:
                            if src == "packed":
                                st = apt.apt_gemm(M, N, K, p, q, a.data.data_ptr(), wi.data_ptr(), None,
                                                  None, c32.data_ptr(), sa.data_ptr(), sw.data_ptr(),
                                                  c16.data_ptr(), cfg, None, 0, sp)
                            elif src == "codes":
                                st = apt.apt_gemm_decode(M, N, K, p, q, xc.data_ptr(), apt.APT_ACT_CODES,
                                                         wi.data_ptr(), c32.data_ptr(), sa.data_ptr(),
                                                         sw.data_ptr(), c16.data_ptr(), None, cfg, sp)
                            else:
                                st = apt.apt_gemm_decode(M, N, K, p, q, x16.data_ptr(), apt.APT_ACT_FP16,
                                                         wi.data_ptr(), c32.data_ptr(), None,
                                                         sw.data_ptr(), c16.data_ptr(), so.data_ptr(),
                                                         cfg, sp)
                            apt.check(st, src)
                    launch(sp0)
                    torch.cuda.synchronize()
                    if ref is None:
                        ref = c32.clone()
                    assert torch.equal(c32, ref), "launch shapes disagree"
                    gr = graph_of(torch, launch)
                    ts.append(replay_us(torch, gr, copies, reps))
                    del gr
                best = min(range(len(ts)), key=lambda i: ts[i])
                bs = DECODE_SHAPES[best]
                lines.append("%6d %6d  W%dA%d %2d %-7s" % (N, K, p, q, M, src) +
                             "".join("%9.2f" % t for t in ts) +
                             "  %s" % ("auto" if bs == (0, 0, 0) else "%d/%d/%d" % bs))
                log("bench: decode shapes %s" % lines[-1])
        del ws
        torch.cuda.empty_cache()
    return "\n".join(lines)


def epilogue_table(calls: int = 50):
    """Cost of the zero-point epilogue: per call, the fp16 scale epilogue
    (apt_gemm) against the zero-point epilogue (apt_gemm_affine) on the same
    operands and selected config, fp16 output only; HIP events around `calls`
    back-to-back calls after 3 warm-up calls, median of 3."""
    import numpy as np
    import torch

    import paper_2508_19087_amd as apt
    import synth
    dev = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()  # noqa: E731
    probs = [synth.layer_w2a4_affine("gate", 1), synth.layer_w2a4_affine("gate", 1024),
             synth.affine_problem("w4a4_affine_2048x11008x4096", 2048, synth.MLP, synth.HIDDEN, 4, 4,
                                  synth.rng(7))]
    rows = []
    for prob in probs:
        M, N, K, p, q = prob.M, prob.N, prob.K, prob.p, prob.q
        a = apt.pack(dev(prob.a_codes), q, activations=True)
        w = apt.pack(dev(prob.w_codes), p)
        sa, sw, za, zw = dev(prob.a_scale), dev(prob.w_scale), dev(prob.a_zero), dev(prob.w_zero)
        c16 = torch.empty((M, N), dtype=torch.float16, device="cuda")
        wsb = apt.apt_gemm_workspace_bytes(M, N, K, p, q, None)
        ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")
        sp = torch.cuda.current_stream().cuda_stream

        def plain():
            apt.check(apt.apt_gemm(M, N, K, p, q, a.data.data_ptr(), w.data.data_ptr(),
                                   a.rowsum.data_ptr(), w.rowsum.data_ptr(), None, sa.data_ptr(),
                                   sw.data_ptr(), c16.data_ptr(), None, ws.data_ptr(), wsb, sp),
                      "apt_gemm")

        def affine():
            apt.check(apt.apt_gemm_affine(M, N, K, p, q, a.data.data_ptr(), w.data.data_ptr(),
                                          a.rowsum.data_ptr(), w.rowsum.data_ptr(), sa.data_ptr(),
                                          za.data_ptr(), sw.data_ptr(), zw.data_ptr(),
                                          c16.data_ptr(), None, None, ws.data_ptr(), wsb, sp),
                      "apt_gemm_affine")
        res = {}
        for name, fn in (("scale_us", plain), ("zero_point_us", affine)):
            ts = []
            for _ in range(3):
                for _ in range(3):
                    fn()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                torch.cuda.synchronize()
                e0.record()
                for _ in range(calls):
                    fn()
                e1.record()
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1) * 1e3 / calls)
            res[name] = round(sorted(ts)[1], 2)
        cfg = apt.select_config(M, N, K, p, q)
        rows.append({"problem": prob.name, "route": apt.ROUTE_NAMES[cfg.route], **res,
                     "extra": round(res["zero_point_us"] / res["scale_us"] - 1, 3)})
        log("bench: epilogues %s %s" % (prob.name, res))
    return rows


# Kernel latencies the paper reports for its own kernel on an RTX 3090 (int32
# output, average of many runs), in microseconds, by (M, N, K) and (p, q):
# the GEMM table (M = 64, N = K in 1024, 2048, 4096) and the LLM prefill and
# decode tables (M = 64 and M = 1; N, K in 1024/4096, 14336/4096, 4096/14336).
PAPER_US = {
    (64, 1024, 1024): {(1, 2): 6.83, (2, 2): 8.40, (3, 4): 11.6},
    (64, 2048, 2048): {(1, 2): 11.6, (2, 2): 11.8, (3, 4): 21.5},
    (64, 4096, 4096): {(1, 2): 18.6, (2, 2): 20.7, (3, 4): 42.3},
    (64, 1024, 4096): {(1, 2): 15.9, (2, 2): 15.7, (3, 4): 26.8},
    (64, 14336, 4096): {(1, 2): 52.8, (2, 2): 62.4, (3, 4): 203.0},
    (64, 4096, 14336): {(1, 2): 63.6, (2, 2): 71.7, (3, 4): 252.0},
    (1, 1024, 4096): {(1, 2): 15.9, (2, 2): 15.1, (3, 4): 21.4},
    (1, 14336, 4096): {(1, 2): 53.0, (2, 2): 51.2, (3, 4): 161.0},
    (1, 4096, 14336): {(1, 2): 64.1, (2, 2): 60.1, (3, 4): 216.0},
}


def paper_shapes(calls: int = 100, reps: int = 3):
    """Context for the paper's kernel tables: this library's selected config at
    the same shapes and widths, warm (the paper averages repeated runs), int32
    output, as one HIP graph of `calls` back-to-back calls replayed between two
    events (median of `reps` replays after one warm-up)."""
    import numpy as np
    import torch

    import paper_2508_19087_amd as apt
    rows = []
    g = np.random.default_rng(11)
    for (M, N, K), by_bits in PAPER_US.items():
        for (p, q), paper_us in by_bits.items():
            ac = torch.from_numpy(g.integers(-(1 << (q - 1)), 1 << (q - 1), (M, K), dtype=np.int8)).cuda()
            wc = torch.from_numpy(g.integers(-(1 << (p - 1)), 1 << (p - 1), (N, K), dtype=np.int8)).cuda()
            a = apt.pack(ac, q, activations=True)
            w = apt.pack(wc, p)
            c32 = torch.empty((M, N), dtype=torch.int32, device="cuda")
            wsb = apt.apt_gemm_workspace_bytes(M, N, K, p, q, None)
            ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")

            def launch(sp, M=M, N=N, K=K, p=p, q=q, a=a, w=w, c32=c32, ws=ws, wsb=wsb):
                for _ in range(calls):
                    apt.check(apt.apt_gemm(M, N, K, p, q, a.data.data_ptr(), w.data.data_ptr(),
                                           a.rowsum.data_ptr(), w.rowsum.data_ptr(), c32.data_ptr(),
                                           None, None, None, None, ws.data_ptr(), wsb, sp), "apt_gemm")
            gr = graph_of(torch, launch)
            ts = []
            for r in range(reps + 1):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                gr.replay()
                e1.record()
                torch.cuda.synchronize()
                if r > 0:
                    ts.append(e0.elapsed_time(e1) * 1e3 / calls)
            us = sorted(ts)[len(ts) // 2]
            cfg = apt.select_config(M, N, K, p, q)
            rows.append({"M": M, "N": N, "K": K, "p": p, "q": q, "route": apt.ROUTE_NAMES[cfg.route],
                         "us": round(us, 2), "paper_rtx3090_us": paper_us,
                         "paper_over_this": round(paper_us / us, 2),
                         "effective_TOPS": round(2 * M * N * K / us / 1e6, 2)})
            log("bench: paper shape %dx%dx%d W%dA%d %.2f us (paper %.1f)" % (M, N, K, p, q, us, paper_us))
            del gr
    return rows


def xor_crossover(calls: int = 50):
    """Where the XOR route beats the MFMA routes: for M = 16..256 and a few
    (N, K, p, q), the forced XOR route (its own launch shape) and
    the best of the 128x128 MFMA configs the model takes at such sizes (int8,
    and FP4 where it applies; one workgroup per tile and 512 workgroups), each
    as one HIP graph of `calls` calls (warm, int32 output), plus the selected
    config; then the least-squares fit of the XOR model the selector uses."""
    import math

    import numpy as np
    import torch

    import paper_2508_19087_amd as apt
    C = apt.apt_config_t.make
    g = np.random.default_rng(5)

    def timed(M, N, K, p, q, cfg, a, w, c32):
        wsb = apt.apt_gemm_workspace_bytes(M, N, K, p, q, cfg)
        ws = torch.empty(max(wsb, 16), dtype=torch.uint8, device="cuda")

        def launch(sp):
            for _ in range(calls):
                apt.check(apt.apt_gemm(M, N, K, p, q, a.data.data_ptr(), w.data.data_ptr(),
                                       a.rowsum.data_ptr(), w.rowsum.data_ptr(), c32.data_ptr(), None,
                                       None, None, cfg, ws.data_ptr(), wsb, sp), "apt_gemm")
        gr = graph_of(torch, launch)
        ts = []
        for r in range(4):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            gr.replay()
            e1.record()
            torch.cuda.synchronize()
            if r > 0:
                ts.append(e0.elapsed_time(e1) * 1e3 / calls)
        return sorted(ts)[1]
    rows = []
    for N, K in [(1024, 1024), (4096, 4096), (14336, 4096), (4096, 14336)]:
        for p, q in [(1, 2), (2, 2), (3, 4), (4, 4), (2, 8)]:
            for M in (16, 32, 64, 128, 256):
                ac = torch.from_numpy(g.integers(-(1 << (q - 1)), 1 << (q - 1), (M, K), dtype=np.int8)).cuda()
                wc = torch.from_numpy(g.integers(-(1 << (p - 1)), 1 << (p - 1), (N, K), dtype=np.int8)).cuda()
                a = apt.pack(ac, q, activations=True)
                w = apt.pack(wc, p)
                c32 = torch.empty((M, N), dtype=torch.int32, device="cuda")
                routes = [apt.APT_ROUTE_INT8_MFMA] + ([apt.APT_ROUTE_FP4_MFMA] if p <= 2 and q <= 2 else [])
                mfma = min(timed(M, N, K, p, q, C(r, 128, 128, 128, 2, 2, grid, 3), a, w, c32)
                           for r in routes for grid in (0, 512))
                xor = timed(M, N, K, p, q, C(apt.APT_ROUTE_XOR), a, w, c32)
                sel = apt.select_config(M, N, K, p, q)
                selected = timed(M, N, K, p, q, sel, a, w, c32)
                rows.append({"M": M, "N": N, "K": K, "p": p, "q": q, "xor_us": round(xor, 2),
                             "mfma_128x128_us": round(mfma, 2), "selected": apt.ROUTE_NAMES[sel.route],
                             "selected_us": round(selected, 2)})
            log("bench: xor crossover N=%d K=%d W%dA%d done" % (N, K, p, q))
    # the selector's XOR model: t = t0 + W (a + b q + c p q), W = 8 ceil(M / 8) N K / 32 word pairs
    # (8 activation rows per block row), fitted by least squares on the relative error
    t = np.array([r["xor_us"] for r in rows])
    W = np.array([8 * math.ceil(r["M"] / 8) * r["N"] * r["K"] / 32 for r in rows]) * 1e-6
    q = np.array([r["q"] for r in rows], dtype=float)
    pq = np.array([r["p"] * r["q"] for r in rows], dtype=float)
    X = np.vstack([np.ones_like(W), W, W * q, W * pq]).T
    coef = np.linalg.lstsq(X / t[:, None], np.ones_like(t), rcond=None)[0]
    err = np.abs(X @ coef / t - 1)
    return {"rows": rows, "xor_fit": {"t0_us": round(coef[0], 3), "a_ps_per_word": round(coef[1], 4),
                                      "b_ps_per_word_per_q": round(coef[2], 4),
                                      "c_ps_per_word_per_pq": round(coef[3], 4),
                                      "median_rel_err": round(float(np.median(err)), 3),
                                      "max_rel_err": round(float(err.max()), 3)}}


def stored_traffic():
    """HBM traffic of the prefill GEMM from the committed rocprofv3 counter
    summary, if it was taken on the current kernel sources."""
    path = os.path.join(PROFILES, "gemm_int8_w4a4_2048x11008x4096_traffic.json")
    if not os.path.exists(path):
        return None
    try:
        d = json.load(open(path))
    except Exception:
        return None
    if d.get("kernel_hash") != kernel_hash():
        return None
    return d.get("traffic_bytes_per_launch")


def cpu_baseline(target_s: float = 12.0):
    """The oracle on a bounded sample of the step: both M=1 decode GEMMs in
    full plus the first R rows of the prefill GEMM, conversion and decoding of
    the operands included.  Rate in effective TOPS."""
    import numpy as np

    import synth
    from oracle import oracle as ref
    dec = [synth.w2a2_decode(1, 4096), synth.w2a2_decode(1, synth.MLP)]
    pre = synth.w4a4_prefill()

    def run(rows):
        ops = 0
        t0 = time.perf_counter()
        for p in dec:
            C = ref.gemm(p.a_codes, p.w_codes, p.p, p.q)
            ref.epilogue(C, p.a_scale, p.w_scale)
            ops += p.ops
        va = ref.values(pre.a_codes[:rows], pre.q)
        vw = ref.values(pre.w_codes, pre.p)
        ref.matmul(va, vw)
        ops += 2 * rows * pre.N * pre.K
        return ops, time.perf_counter() - t0

    # calibrate: the fixed part (decode GEMMs, weight decoding) and the cost
    # of one prefill row, then size the sample to the target time
    t0 = time.perf_counter()
    for p in dec:
        ref.gemm(p.a_codes, p.w_codes, p.p, p.q)
    vw = ref.values(pre.w_codes, pre.p)
    t1 = time.perf_counter()
    va = ref.values(pre.a_codes[:64], pre.q)
    ref.matmul(va, vw)
    t2 = time.perf_counter()
    per_row = (t2 - t1) / 64
    rows = int(min(pre.M, max(16, (target_s - (t1 - t0)) / per_row)))
    # when the whole step is shorter than the target, time whole steps repeatedly
    passes = 1
    if rows == pre.M:
        passes = max(1, int(round(target_s / ((t1 - t0) + per_row * pre.M))))
    del vw, va
    ops = t = 0
    for _ in range(passes):
        o, dt = run(rows)
        ops += o
        t += dt
    return {"value": round(ops / t / 1e12, 6), "unit": "TOPS", "cores": ref.num_threads(),
            "kind": "oracle", "seconds": round(t, 2),
            "sample": ("%d pass(es) over: both M=1 W2A2 decode GEMMs in full (with fp16 epilogue) + "
                       "rows 0..%d of the 2048x11008x4096 W4A4 GEMM, bipolar conversion and decoding "
                       "included; %.3g effective ops in all" % (passes, rows - 1, ops)),
            "one_core": oracle_one_core()}


ONE_CORE_SCRIPT = """
import json, sys, time
sys.path.insert(0, sys.argv[1])
import synth
from oracle import oracle as ref
out = {"threads": ref.num_threads()}
for name, probs in (("w1a2_16x512x512", [synth.w1a2_small()]),
                    ("w2a2_decode_m1_both", [synth.w2a2_decode(1, 4096), synth.w2a2_decode(1, synth.MLP)])):
    ts = []
    for _ in range(3):
        t0 = time.perf_counter()
        for p in probs:
            C = ref.gemm(p.a_codes, p.w_codes, p.p, p.q)
            if p.a_scale is not None:
                ref.epilogue(C, p.a_scale, p.w_scale)
        ts.append(time.perf_counter() - t0)
    out[name] = {"seconds": round(sorted(ts)[1], 4), "ops": sum(p.ops for p in probs)}
print(json.dumps(out))
"""


def oracle_one_core():
    """The oracle on one core (OpenMP limited to one thread in a child process)
    for the small W1A2 GEMM and the two M=1 decode GEMMs: median of 3 runs,
    conversion and decoding included."""
    env = dict(os.environ, OMP_NUM_THREADS="1")
    r = subprocess.run([sys.executable, "-c", ONE_CORE_SCRIPT, ROOT], capture_output=True,
                       text=True, env=env, timeout=600)
    if r.returncode != 0:
        return {"error": r.stderr[-400:]}
    return json.loads(r.stdout.strip().splitlines()[-1])


COPY_BYTES = 256 << 20  # calibration copy for the HBM byte counters
TRAFFIC_JSON = "gemm_int8_w4a4_2048x11008x4096_traffic.json"


def counters_run(reps: int = 3, packed_prefill: bool = False):
    """For rocprofv3 --pmc: the prefill call (prefill_call) `reps` times after
    one warm-up call, then a plain device copy of COPY_BYTES (read and written once),
    whose counter readings calibrate the byte counters."""
    import torch
    wl = Workload()
    wl.packed_prefill = packed_prefill
    call = prefill_call(wl)
    for _ in range(reps + 1):
        call()
    src = torch.empty(COPY_BYTES, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    log("bench: counters run done (%d prefill GEMMs, copy of %d bytes)" % (reps + 1, COPY_BYTES))


def counters_xor(M: int, N: int, K: int, p: int, q: int, reps: int = 3):
    """For rocprofv3 --pmc on the XOR + popcount route: one M x N x K WpAq
    problem on seeded random codes, forced onto the XOR route (8 activation
    rows per workgroup), `reps` times after one warm-up call."""
    import numpy as np
    import torch

    import paper_2508_19087_amd as apt
    g = np.random.default_rng(5)
    ac = torch.from_numpy(g.integers(-(1 << (q - 1)), 1 << (q - 1), (M, K), dtype=np.int8)).cuda()
    wc = torch.from_numpy(g.integers(-(1 << (p - 1)), 1 << (p - 1), (N, K), dtype=np.int8)).cuda()
    a = apt.pack(ac, q, activations=True)
    w = apt.pack(wc, p)
    c32 = torch.empty((M, N), dtype=torch.int32, device="cuda")
    cfg = apt.apt_config_t.make(apt.APT_ROUTE_XOR, mt=8)
    sp = torch.cuda.current_stream().cuda_stream
    for _ in range(reps + 1):
        apt.check(apt.apt_gemm(M, N, K, p, q, a.data.data_ptr(), w.data.data_ptr(), a.rowsum.data_ptr(),
                               w.rowsum.data_ptr(), c32.data_ptr(), None, None, None, cfg, None, 0, sp),
                  "apt_gemm")
    torch.cuda.synchronize()
    log("bench: counters run done (%d XOR GEMMs, %dx%dx%d W%dA%d)" % (reps + 1, M, N, K, p, q))


def workload_problems():
    """Every workload configuration: the W1A2 16x512x512 GEMM, the W2A2 decode
    GEMMs (M = 1, 4, 8; N = 4096, 11008), the W4A4 prefill GEMM, the (p, q)
    sweep on the down projection and the W2A4 layer set at 1 and 1024 tokens."""
    import synth
    probs = [synth.w1a2_small()]
    probs += [synth.w2a2_decode(M, N) for M in (1, 4, 8) for N in (4096, synth.MLP)]
    probs += [synth.w4a4_prefill()]
    probs += [synth.sweep_down(i) for i in range(len(synth.SWEEP_BITS))]
    probs += [synth.layer_w2a4(name, M) for M in (1, 1024) for name in synth.LAYER_SHAPES]
    return probs


def settle_gpu(seconds: float):
    """Untimed load before a measurement mode: back-to-back W4A4
    1024x4096x4096 calls for `seconds`, so that the GPU's clocks have risen to
    the level they hold under load before anything is timed (the bench step
    does the same with its own steps)."""
    if seconds <= 0:
        return
    import torch

    import paper_2508_19087_amd as apt
    gen = torch.Generator().manual_seed(11)
    w = apt.pack(torch.randint(-8, 8, (4096, 4096), dtype=torch.int8, generator=gen).cuda(), 4)
    a = apt.pack(torch.randint(-8, 8, (1024, 4096), dtype=torch.int8, generator=gen).cuda(), 4,
                 activations=True)
    ws = torch.empty(max(apt.apt_gemm_workspace_bytes(1024, 4096, 4096, 4, 4), 256), dtype=torch.uint8,
                     device="cuda")
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(20):
            apt.gemm(a, w, workspace=ws)
        torch.cuda.synchronize()


def workloads_run(calls: int = 20, settle_s: float = 0.02):
    """For rocprofv3 --kernel-trace: every workload configuration packed
    first, then, workload by workload, untimed calls for `settle_s` seconds
    (loaded clocks), one torch fill of a marker buffer (a kernel that
    separates the workloads in the trace) and `calls` back-to-back apt_gemm
    calls in the selected config (int32 output, plus the fp16 epilogue where
    the workload has scales); then the same for the activation packers of
    the decode workloads (code and fp16 sources) and for apt_gemm_decode.
    Prints the plan as JSON."""
    import numpy as np
    import torch

    import paper_2508_19087_amd as apt
    dev = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()  # noqa: E731
    items = []
    for prob in workload_problems():
        a = apt.pack(dev(prob.a_codes), prob.q, activations=True)
        w = apt.pack(dev(prob.w_codes), prob.p)
        fp16 = prob.a_scale is not None
        items.append((prob, a, w, dev(prob.a_scale) if fp16 else None,
                      dev(prob.w_scale) if fp16 else None))
    marker = torch.empty(1, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    plan = []

    def group(entry, one_call):
        # untimed calls of the same kind first, for `settle_s`, so that the
        # timed ones run at loaded clocks (a segment of their own, marked
        # "settle" in the plan and left out of the summary); then `calls`
        # back-to-back calls after a marker fill
        marker.fill_(-1)
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < settle_s:
            for _ in range(10):
                one_call()
            torch.cuda.synchronize()
        plan.append({"settle": True})
        marker.fill_(len(plan))
        for _ in range(calls):
            one_call()
        torch.cuda.synchronize()
        plan.append(entry)

    for i, (prob, a, w, sa, sw) in enumerate(items):
        cfg = apt.select_config(prob.M, prob.N, prob.K, prob.p, prob.q)
        ws_bytes = apt.apt_gemm_workspace_bytes(prob.M, prob.N, prob.K, prob.p, prob.q, cfg)
        ws = torch.empty(max(ws_bytes, 256), dtype=torch.uint8, device="cuda")
        c32 = torch.empty((prob.M, prob.N), dtype=torch.int32, device="cuda")
        c16 = torch.empty((prob.M, prob.N), dtype=torch.float16, device="cuda") if sa is not None else None
        sp = torch.cuda.current_stream().cuda_stream

        def one_call():
            apt.check(apt.apt_gemm(prob.M, prob.N, prob.K, prob.p, prob.q, a.data.data_ptr(),
                                   w.data.data_ptr(), a.rowsum.data_ptr(), w.rowsum.data_ptr(),
                                   c32.data_ptr(), sa.data_ptr() if sa is not None else None,
                                   sw.data_ptr() if sw is not None else None,
                                   c16.data_ptr() if c16 is not None else None, cfg,
                                   ws.data_ptr(), ws_bytes, sp), "apt_gemm")
        group({"workload": prob.name, "M": prob.M, "N": prob.N, "K": prob.K, "p": prob.p,
               "q": prob.q, "ops": prob.ops, "fp16": c16 is not None, "calls": calls,
               "config": cfg.as_dict()}, one_call)
        del ws, c32, c16
    # the activation packers of the decode workloads (M <= 8, K = 4096): the
    # code source and the fp16 quantizer, `calls` back-to-back calls each
    seen = set()
    for prob, a, w, sa, sw in items:
        if prob.M > 8 or (prob.M, prob.K, prob.q) in seen:
            continue
        seen.add((prob.M, prob.K, prob.q))
        codes = dev(prob.a_codes)
        x16 = torch.from_numpy(np.ascontiguousarray(
            (prob.a_codes.astype(np.float32) * 0.37).astype(np.float16))).cuda()
        buf = torch.empty(apt.apt_packed_bytes(prob.M, prob.K, prob.q), dtype=torch.uint8, device="cuda")
        rs = torch.empty(prob.M, dtype=torch.int32, device="cuda")
        sc = torch.empty(prob.M, dtype=torch.float16, device="cuda")
        sp = torch.cuda.current_stream().cuda_stream
        for kind in ("codes", "fp16"):
            def one_call():
                if kind == "codes":
                    st = apt.apt_quantize_pack_activations(codes.data_ptr(), prob.M, prob.K, prob.q,
                                                           buf.data_ptr(), rs.data_ptr(), sp)
                else:
                    st = apt.apt_quantize_pack_activations_fp16(x16.data_ptr(), prob.M, prob.K, prob.q,
                                                                buf.data_ptr(), rs.data_ptr(),
                                                                sc.data_ptr(), sp)
                apt.check(st, "pack")
            group({"workload": "pack_%s_m%d_k%d_q%d" % (kind, prob.M, prob.K, prob.q),
                   "M": prob.M, "K": prob.K, "q": prob.q, "calls": calls, "pack": kind,
                   "bytes": prob.M * prob.K * (1 if kind == "codes" else 2)
                   + apt.apt_packed_bytes(prob.M, prob.K, prob.q) + 4 * prob.M}, one_call)
    # the decode workloads through apt_gemm_decode (one launch from the token's
    # codes or fp16 values, int32 and fp16 outputs)
    for i, (prob, a, w, sa, sw) in enumerate(items):
        if prob.M > 8 or sa is None:
            continue
        codes = dev(prob.a_codes)
        x16 = torch.from_numpy(np.ascontiguousarray(
            (prob.a_codes.astype(np.float32) * 0.37).astype(np.float16))).cuda()
        c32 = torch.empty((prob.M, prob.N), dtype=torch.int32, device="cuda")
        c16 = torch.empty((prob.M, prob.N), dtype=torch.float16, device="cuda")
        so = torch.empty(prob.M, dtype=torch.float16, device="cuda")
        sp = torch.cuda.current_stream().cuda_stream
        for kind in ("codes", "fp16"):
            def one_call():
                if kind == "codes":
                    st = apt.apt_gemm_decode(prob.M, prob.N, prob.K, prob.p, prob.q, codes.data_ptr(),
                                             apt.APT_ACT_CODES, w.data.data_ptr(), c32.data_ptr(),
                                             sa.data_ptr(), sw.data_ptr(), c16.data_ptr(), None, None, sp)
                else:
                    st = apt.apt_gemm_decode(prob.M, prob.N, prob.K, prob.p, prob.q, x16.data_ptr(),
                                             apt.APT_ACT_FP16, w.data.data_ptr(), c32.data_ptr(), None,
                                             sw.data_ptr(), c16.data_ptr(), so.data_ptr(), None, sp)
                apt.check(st, "apt_gemm_decode")
            group({"workload": prob.name, "M": prob.M, "N": prob.N, "K": prob.K, "p": prob.p,
                   "q": prob.q, "ops": prob.ops, "calls": calls, "decode": kind}, one_call)
    print(json.dumps(plan), flush=True)


def write_workload_stats(trace_csv: str, plan_json: str, command: str):
    """Per-workload kernel durations from the rocprofv3 kernel trace of
    workloads_run: the dispatches between consecutive marker fills belong to
    one workload; the first call of each is a warm-up and is left out."""
    import csv
    import statistics
    plan = json.load(open(plan_json))
    rows = sorted(csv.DictReader(open(trace_csv)), key=lambda r: int(r["Start_Timestamp"]))
    segs, cur = [], None
    for r in rows:
        name = r["Kernel_Name"]
        if "FillFunctor" in name or "fill" in name.lower():
            cur = []
            segs.append(cur)
        elif cur is not None and "rocclr" not in name:  # (host-to-device copies are not timed)
            cur.append((name, (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1000.0))
    assert len(segs) == len(plan), (len(segs), len(plan))
    keep = [i for i, pl in enumerate(plan) if not pl.get("settle")]
    plan, segs = [plan[i] for i in keep], [segs[i] for i in keep]
    lines = ["# Kernel durations of every workload configuration in its selected config (rocprofv3",
             "# kernel trace; per kernel: median and mean duration over the calls after the first,",
             "# in microseconds; 'per call' sums the kernels one apt_gemm call launches, 'TOPS' is",
             "# 2 M N K over that sum).  Weights and activations are packed before the timed calls,",
             "# except in the apt_gemm_decode lines, which take the tokens' codes or fp16 values.",
             "# Each workload's timed calls follow 20 ms of untimed calls of the same kind (loaded",
             "# clocks; the run starts with 0.3 s of untimed W4A4 1024x4096x4096 calls).",
             "# command (repository root on the MI355X box): " + command,
             ""]
    for pl, seg in zip(plan, segs):
        per_call = len(seg) // pl["calls"]
        assert per_call * pl["calls"] == len(seg), (pl["workload"], len(seg))
        body = seg[per_call:]  # skip the first call
        names = []
        for n, _ in body:
            if n not in names:
                names.append(n)
        total = 0.0
        parts = []
        for n in names:
            ts = [t for k, t in body if k == n]
            med = statistics.median(ts)
            total += med * len(ts) / (pl["calls"] - 1)
            short = re.sub(r"\(anonymous namespace\)::", "", n)
            short = short.split("(")[0].replace("void ", "").replace("apt::", "")
            parts.append("%s median %.2f mean %.2f" % (short, med, statistics.mean(ts)))
        if "pack" in pl:
            lines.append("%-32s %-28s per call %8.2f us  %8.1f GB/s" % (
                pl["workload"], "packer (%s source)" % pl["pack"], total, pl["bytes"] / total / 1e3))
            for ptxt in parts:
                lines.append("    " + ptxt)
            continue
        if "decode" in pl:
            lines.append("%-32s %-28s per call %8.2f us  %8.1f TOPS" % (
                pl["workload"], "apt_gemm_decode (%s)" % pl["decode"], total, pl["ops"] / total / 1e6))
            for ptxt in parts:
                lines.append("    " + ptxt)
            continue
        c = pl["config"]
        route = {1: "xor", 2: "pm1", 3: "int8", 4: "fp4", 5: "fp6", 6: "fp8"}[c["route"]]
        cfg = route if route == "xor" else "%s %dx%d/%dx%d g%d%s" % (
            route, c["bm"], c["bn"], c["waves_m"], c["waves_n"], c["grid"],
            " split %d" % c["split_n"] if c["split_n"] else "")
        lines.append("%-32s %-28s per call %8.2f us  %8.1f TOPS" % (
            pl["workload"], cfg, total, pl["ops"] / total / 1e6))
        for ptxt in parts:
            lines.append("    " + ptxt)
    print("\n".join(lines))


def write_traffic(fetch_dir: str, write_dir: str, commands: str):
    """HBM bytes per prefill apt_gemm call from two rocprofv3 --pmc runs of
    counters_run (FETCH_SIZE, then WRITE_SIZE; KiB per dispatch): the GEMM's
    kernels summed per call, each counter scaled by what it reads for the
    calibration copy (COPY_BYTES in each direction)."""
    import csv
    import glob
    import statistics

    def per_kernel(d, counter):
        f = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)[0]
        vals = {}
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] != counter:
                continue
            vals.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]) * 1024.0)
        return vals

    out = {"kernel_hash": kernel_hash(), "commands": commands}
    for tag, d, counter in [("fetch", fetch_dir, "FETCH_SIZE"), ("write", write_dir, "WRITE_SIZE")]:
        vals = per_kernel(d, counter)
        copy = [v for k, vs in vals.items() if "copyBuffer" in k for v in vs if v > COPY_BYTES / 4]
        factor = COPY_BYTES / statistics.median(copy)
        # the GEMM's kernels: every dispatch after the warm-up call
        gemm = {k: vs for k, vs in vals.items()
                if "expand_a_kernel" in k or "act_frag_kernel" in k or "gemm_int8_" in k}
        per_call = 0.0
        kernels = {}
        for k, vs in gemm.items():
            med = statistics.median(vs[1:] if len(vs) > 1 else vs)
            kernels[k] = round(med * factor)
            per_call += med * factor
        out[tag] = {"counter": counter, "calibration_factor": round(factor, 4),
                    "bytes_per_call": round(per_call), "kernels": kernels}
    out["traffic_bytes_per_launch"] = out["fetch"]["bytes_per_call"] + out["write"]["bytes_per_call"]
    path = os.path.join(PROFILES, TRAFFIC_JSON)
    json.dump(out, open(path, "w"), indent=1)
    print(json.dumps(out, indent=1))


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--settle", type=float, default=0.3,
                    help="seconds of untimed steps before the warm-up steps (other timing modes: "
                         "of untimed GEMM calls), so that the GPU's clocks have risen to their "
                         "loaded level (0 to skip)")
    ap.add_argument("--no-decode-cold", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--roofline-calls", type=int, default=50,
                    help="back-to-back prefill GEMM calls timed for the roofline")
    ap.add_argument("--counters-run", action="store_true",
                    help="run the prefill GEMM and a calibration copy for rocprofv3 --pmc, then exit")
    ap.add_argument("--counters-xor", nargs=5, type=int, metavar=("M", "N", "K", "P", "Q"),
                    help="run one problem on the XOR route for rocprofv3 --pmc, then exit")
    ap.add_argument("--write-traffic", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="summarize two rocprofv3 --pmc runs of --counters-run into profiles/")
    ap.add_argument("--routes", action="store_true",
                    help="print the route-choice table (us per call of every route) and exit")
    ap.add_argument("--search", action="store_true",
                    help="print the model's and the search module's config for every workload "
                         "shape, with their times, and exit")
    ap.add_argument("--xor-crossover", action="store_true",
                    help="print the XOR route against the MFMA routes for small M, with the XOR model fit, and exit")
    ap.add_argument("--paper-shapes", action="store_true",
                    help="print this library's times at the shapes of the paper's kernel tables and exit")
    ap.add_argument("--epilogues", action="store_true",
                    help="print the cost of the zero-point epilogue against the scale epilogue and exit")
    ap.add_argument("--decode-sweep", action="store_true",
                    help="print the cold-weight time of one M=1 W2A4 GEMM against N and exit")
    ap.add_argument("--calibrate", action="store_true",
                    help="print the selector model's calibration (pair and fixed times per tile "
                         "shape and operand class) and exit")
    ap.add_argument("--packed-prefill", action="store_true",
                    help="in the step and the roofline, pack the prefill activations with the packer "
                         "and run apt_gemm, instead of apt_gemm_act from the codes")
    ap.add_argument("--unfused-decode", action="store_true",
                    help="in the step, pack each decode token's activations with the packer and "
                         "then run apt_gemm, instead of apt_gemm_decode's one launch")
    ap.add_argument("--serial-step", action="store_true",
                    help="run the whole step on one stream (the decode GEMMs before the prefill) "
                         "instead of the decode chain on a second stream beside the prefill")
    ap.add_argument("--one-batch", action="store_true",
                    help="one prefill batch in flight: every step's prefill on the main stream "
                         "(the decode chain still on the second stream), instead of consecutive "
                         "steps' prefills alternating between two streams")
    ap.add_argument("--vendor-int8", action="store_true",
                    help="print the vendor library's dense int8 GEMM (torch._int_mm) on the prefill "
                         "shape with int8 operands, as context, and exit")
    ap.add_argument("--mfma-issue", action="store_true",
                    help="print the MFMA-issue probe's cycles per MFMA for each part of the GEMM "
                         "loop's instruction pattern and exit")
    ap.add_argument("--format-sweep", action="store_true",
                    help="print int8 against FP6 (W3A3) and FP8 (W4A4) operands on every tile shape and exit")
    ap.add_argument("--workloads", action="store_true",
                    help="for a rocprofv3 kernel trace: every workload configuration's selected "
                         "apt_gemm, 20 calls each, separated by marker fills; prints the plan")
    ap.add_argument("--write-workload-stats", nargs=3, metavar=("TRACE_CSV", "PLAN_JSON", "COMMAND"),
                    help="print the per-workload kernel durations of a --workloads trace and exit")
    ap.add_argument("--decode-shapes", action="store_true",
                    help="print the XOR launch shapes for 2-8 tokens (packed and fused activations) "
                         "with cold weights and exit")
    ap.add_argument("--decode-chain", action="store_true",
                    help="print one token's decode GEMMs and decoder layer from their activations, "
                         "unfused and fused, with cold weights, and exit")
    ap.add_argument("--traffic-commands", default="",
                    help="the commands that produced the --write-traffic directories")
    args = ap.parse_args()
    if args.write_traffic:
        write_traffic(args.write_traffic[0], args.write_traffic[1], args.traffic_commands)
        return
    if args.write_workload_stats:
        write_workload_stats(*args.write_workload_stats)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path "
              "(no sharding or collectives); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.counters_run:
        counters_run(packed_prefill=args.packed_prefill)
        return
    if any((args.workloads, args.vendor_int8, args.format_sweep, args.calibrate, args.routes,
            args.search, args.decode_shapes, args.decode_sweep, args.epilogues, args.paper_shapes,
            args.xor_crossover, args.decode_chain)):
        # these timing modes start at loaded clocks (the bench step settles
        # with its own steps)
        settle_gpu(args.settle)
    if args.workloads:
        workloads_run()
        return
    if args.vendor_int8:
        print(json.dumps(vendor_int8(), indent=1), flush=True)
        return
    if args.mfma_issue:
        print(json.dumps(mfma_issue(), indent=1), flush=True)
        return
    if args.format_sweep:
        print(json.dumps(format_sweep(), indent=1), flush=True)
        return
    if args.calibrate:
        print(json.dumps(calibrate(), indent=1), flush=True)
        return
    if args.counters_xor:
        counters_xor(*args.counters_xor)
        return
    if args.routes:
        print(json.dumps(route_table(), indent=1), flush=True)
        return
    if args.search:
        print(json.dumps(search_table(), indent=1), flush=True)
        return
    if args.decode_shapes:
        print(decode_shapes(), flush=True)
        return
    if args.decode_sweep:
        print(json.dumps(decode_sweep(), indent=1), flush=True)
        return
    if args.epilogues:
        print(json.dumps(epilogue_table(), indent=1), flush=True)
        return
    if args.paper_shapes:
        print(json.dumps(paper_shapes(), indent=1), flush=True)
        return
    if args.xor_crossover:
        print(json.dumps(xor_crossover(), indent=1), flush=True)
        return
    log("bench: building workload")
    wl = Workload()
    if args.decode_chain:
        res = {"token_chain": decode_token_cold(wl)}
        log("bench: one-token W2A4 decoder layer with cold weights")
        res["w2a4_layer_m1"] = decode_layer_cold(wl)
        print(json.dumps(res, indent=1), flush=True)
        return
    wl.overlap = not args.serial_step
    wl.batches = 1 if (args.one_batch or args.serial_step) else 2
    wl.unfused_decode = args.unfused_decode
    wl.packed_prefill = args.packed_prefill
    # Settle: the GPU raises its clocks over the first tenths of a second of
    # load (measured: 108 us per step after 10 warm-up steps, 93 us after
    # 1000), so steps run untimed for `settle` seconds before the W warm-up
    # steps, and the K timed steps see the clocks a loaded GPU runs at.
    settle_steps = 0
    t_settle = time.perf_counter()
    while time.perf_counter() - t_settle < args.settle:
        for _ in range(50):
            wl.step()
        settle_steps += 50
        torch.cuda.synchronize()
    settle_s = time.perf_counter() - t_settle
    for _ in range(args.warmup):
        wl.step()
    torch.cuda.synchronize()
    log("bench: timing %d steps" % args.steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        wl.step()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    step_s = (t1 - t0) / args.steps
    one_batch_s = None
    if wl.batches == 2:
        # the same steps with one prefill batch in flight, for comparison
        wl.batches = 1
        for _ in range(5):
            wl.step()
        torch.cuda.synchronize()
        t2 = time.perf_counter()
        for _ in range(args.steps):
            wl.step()
        torch.cuda.synchronize()
        one_batch_s = (time.perf_counter() - t2) / args.steps
        wl.batches = 2
    # The dominant kernel alone: back-to-back prefill GEMM calls between two
    # events on the stream they run on (an event per call would put a bubble
    # of several microseconds in the stream each time).
    gemm_s = prefill_call_time(wl, args.roofline_calls)
    pre = wl.pre
    achieved = pre.ops / gemm_s / 1e12
    traffic = stored_traffic()
    sel = wl.apt.select_config(pre.M, pre.N, pre.K, pre.p, pre.q)
    cfg = sel.as_dict()
    tiles = "%dx%d tiles (%dx%d waves)" % (sel.bm, sel.bn, sel.waves_m, sel.waves_n)
    if sel.split_n:
        tiles += " over columns [0, %d) and %dx%d tiles over the rest" % (sel.split_n, sel.tail_bm,
                                                                          sel.tail_bn)
    tiles += ", one workgroup per tile" if sel.grid == 0 else ", %d persistent workgroups" % sel.grid
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_INT8_TOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_INT8_TOPS, 4), "traffic": traffic,
                "kernel": ("apt_gemm W4A4 M=2048 N=11008 K=4096 on packed activations: expand_a_kernel"
                           if wl.packed_prefill else
                           "apt_gemm_act W4A4 M=2048 N=11008 K=4096 from the int8 codes: act_frag_kernel")
                          + " + gemm_int8 kernel (%s), %d back-to-back calls" % (tiles, args.roofline_calls),
                "avg_launch_us": round(gemm_s * 1e6, 2)}
    result = {
        "metric": METRIC, "value": round(wl.ops / step_s / 1e12, 3), "unit": "TOPS",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(step_s * 1e3, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "int8", "data": "synthetic",
        "config": {"workload": "W2A2 decode M=1 (N=4096 and N=11008, K=4096, int32 + fp16 epilogue) "
                               "+ W4A4 prefill M=2048 N=11008 K=4096 (int32); activations converted "
                               "and decomposed every step, weights packed once",
                   "schedule": ("decode chain on a second stream beside the prefill chain"
                                + ("; consecutive steps' prefills alternate between the main and a "
                                   "third stream (two batches in flight, separate buffers)"
                                   if wl.batches == 2 else "")
                                if wl.overlap else "one stream"),
                   "batches_in_flight": wl.batches if wl.overlap else 1,
                   "decode_activations": ("packer + apt_gemm" if wl.unfused_decode else
                                          "apt_gemm_decode (converted inside the GEMV)"),
                   "prefill_activations": ("packer + apt_gemm" if wl.packed_prefill else
                                           "apt_gemm_act (codes written straight into the int8 "
                                           "MFMA fragments)"),
                   "prefill_config": cfg,
                   "prefill_config_two_batches": (wl.pre_cfg_two.as_dict()
                                                  if wl.batches == 2 and not wl.packed_prefill
                                                  else None)},
        "roofline": roofline,
        "settle": {"seconds": round(settle_s, 3), "steps": settle_steps,
                   "note": "untimed steps before the warm-up steps, while the GPU raises its clocks"},
    }
    if one_batch_s is not None:
        result["one_batch_in_flight"] = {
            "ms_per_step": round(one_batch_s * 1e3, 4), "value": round(wl.ops / one_batch_s / 1e12, 3),
            "note": "the same K steps right after the timed ones with every prefill on the main "
                    "stream (one batch in flight; bench.py --one-batch times this as the headline)"}
    log("bench: fp16 activation quantizer")
    result["quantize_fp16"] = quantize_fp16_rates()
    if not args.no_decode_cold:
        log("bench: decode GEMMs with cold weights")
        result["decode_cold"] = decode_cold(wl)
        log("bench: one token's decode GEMM from its activations, unfused and fused")
        result["decode_cold"]["token_chain"] = decode_token_cold(wl)
        log("bench: one-token W2A4 decoder layer with cold weights")
        result["decode_cold"]["w2a4_layer_m1"] = decode_layer_cold(wl)
    if not args.no_cpu_baseline:
        log("bench: CPU oracle baseline")
        result["cpu_baseline"] = cpu_baseline(args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
