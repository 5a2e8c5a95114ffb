"""Benchmark of the multi-bitwidth additive-codebook linear layer on one MI355X.

One step is one pass of the whole hot path, every operation over R resident copies of its layer
(R distinct weight sets, like R layers of a model), with R chosen so that every burst at every k
streams at least 512 MiB of code planes, twice the 256 MB Infinity Cache:

  decode GEMV, for k in 1..4 (the headline):
    Llama-7B MLP pair, 11008 x 4096 (up) and 4096 x 11008 (down), 4 codebooks of 256 x 8 fp16,
    uint8 codes, bf16 x (heavy-tailed: 0.1 % of entries x 20) and bf16 y, batch 1, 8 and 16
  also in every step:
    16-bit codes: 14336 x 4096, 2 codebooks of 65536 x 8 fp16, fp16 x/y, batch 1, k = 1, 2
    4096 x 4096 (fp16 x/y), batch 1 and 4, k = 1..4; the same layers 4 and 16 per launch
      (aqmb_gemv_multi); the same shape with 4-bit codes (4 codebooks of 16), batch 1
    dequantization of the 4096 x 4096 layer to bf16, k = 1..4
    prefill GEMM, 2048 bf16 tokens x 4096 x 4096, bf16 out, k = 1..4
    prefix distortions D^(1..4) of the 4096 x 4096 layer against a dense fp16 W over 4096 fp16
      calibration inputs; beam search (k = 4, beam 8) of codes for every group of that W, with the
      plain squared error and with the data-aware error d^T H_j d

Each (operation, layer, k, batch) runs as a burst of R launches captured in a HIP graph and timed
with HIP events on the launch stream; the per-launch time is burst time / R.

`value` is the decode GEMV throughput of the headline workload in algorithmic GB/s: code planes
0..k-1, their codebooks, scales, x and y of every MLP-pair launch in the timed steps, over their
time. `roofline` is the MLP-pair GEMV kernel with the largest share of that time, against the
published HBM peak and against the measured ceilings that bind it.

Measured ceilings (`ceilings`, timed once after the steps with the kernels of
libaqmb_ceilings.so): attainable HBM read rate (streaming, and for a launch of each GEMV size on
the GEMV's grid), attainable write rate, random 16-byte LDS gathers from replicated codebooks (with
and without the batch-1 dot products), random 16-byte L2 gathers from 1 and 2 MiB tables, and the
bf16 MFMA rate on random operands.

`--counters MODE` runs eager launches for rocprofv3 counter passes instead (gemv: every MLP-pair and
4096 x 4096 GEMV; gemm: the prefill GEMM at k = 1 and 4; dequant: the 4096 x 4096 dequant to bf16 at
k = 1..4), then one plain 256 MiB copy that calibrates the byte counters.
Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0       # MI355X dense bf16 MFMA
F16_PEAK_TFLOPS = 2500.0        # MI355X dense fp16 MFMA
FP32_PLAIN_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12   # one non-packed fp32 op per lane and clock
BEAM_K, BEAM_WIDTH = 4, 8
STREAM_BYTES = 512 << 20        # code bytes every burst streams at least
KS = (1, 2, 3, 4)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def gemv_bytes(d_out, d_in, B, k, b):
    """Algorithmic bytes of one GEMV launch: k code planes, k codebooks, scales, x and y."""
    code_bytes = {4: 0.5, 8: 1, 16: 2}[B]
    return int(k * d_out * (d_in // 8) * code_bytes) + k * (1 << B) * 16 + 2 * d_out + 2 * b * (d_in + d_out)


# the sources the decode GEMV launches of the headline depend on (kernels and their dispatch)
GEMV_SOURCES = ("api.cpp", "device.h", "k_gemv.hip", "k_gemv_mma.hip")


def measured_traffic(kernel_key):
    """HBM bytes per launch of a kernel from the committed counter summary, if its sources still
    hash to what was measured (else None)."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "gemv_hbm_traffic.md")
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if ":" in line:
            key, val = line.rsplit(":", 1)                    # keys hold colons themselves
            if key.strip() in (f"traffic[{kernel_key}]", "sources_sha256"):
                fields[key.strip()] = val.strip()
    h = hashlib.sha256()
    for f in GEMV_SOURCES:
        h.update(open(os.path.join(ROOT, "paper_2606_12876_amd", "csrc", f), "rb").read())
    if fields.get("sources_sha256") != h.hexdigest() or f"traffic[{kernel_key}]" not in fields:
        return None
    return float(fields[f"traffic[{kernel_key}]"])


def gemv_kernel_name(spec, k, b, xdt):
    """The kernel aqmb_gemv runs for this layer (the library's dispatch rule, restated for labels)."""
    G = spec.d_in // 8
    if spec.B == 16:
        return f"gemv_b16_kernel<KC={min(k, 4)}>"
    wide = G > 512
    rb = (spec.d_out + 15) // 16
    if b >= 2 or (wide and (xdt == "f16" or k >= 3)):
        return ("gemv_mma_persist_kernel" if rb > 256 else "gemv_mma_kernel") + f"<K={k}> (batch {b})"
    return ("gemv_cw_persist_kernel" if rb > 256 else "gemv_cw_kernel") + f"<K={k}> (batch {b})"


class Ceilings:
    """The measured-ceiling kernels (libaqmb_ceilings.so), timed as graph bursts."""

    def __init__(self, torch, stream):
        path = os.path.join(ROOT, "paper_2606_12876_amd", "libaqmb_ceilings.so")
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build first")
        self.lib = ctypes.CDLL(path)
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
        self.lib.aqmbc_hbm_read.argtypes = [vp, sz, i32, vp, vp]
        self.lib.aqmbc_hbm_write.argtypes = [vp, sz, i32, vp]
        self.lib.aqmbc_lds_gather.argtypes = [vp, i32, i32, i32, i32, vp, vp]
        self.lib.aqmbc_lds_gather_paired.argtypes = [vp, i32, i32, vp, vp]
        self.lib.aqmbc_l2_gather.argtypes = [vp, i32, i32, i32, vp, vp]
        self.lib.aqmbc_mfma_bf16.argtypes = [vp, i32, i32, vp, vp]
        self.torch, self.stream = torch, stream
        self.sink = torch.zeros(16, dtype=torch.int32, device="cuda")
        self.n_cu = torch.cuda.get_device_properties(0).multi_processor_count

    def _st(self):
        return self.torch.cuda.current_stream().cuda_stream

    def _check(self, rc):
        if rc != 0:
            raise RuntimeError(f"ceiling kernel launch failed: hip error {rc}")

    def time(self, fn, reps=10):
        return time_graph(self.torch, self.stream, fn, reps)

    def hbm_read(self, nbytes, copies, n_wg):
        """us per launch reading nbytes with n_wg workgroups, rotating over `copies` buffers."""
        torch = self.torch
        buf = torch.ones(nbytes * copies // 2, dtype=torch.float16, device="cuda")
        base = buf.data_ptr()
        us = self.time(lambda: [self._check(self.lib.aqmbc_hbm_read(base + c * nbytes, nbytes, n_wg,
                                                                    self.sink.data_ptr(), self._st()))
                                for c in range(copies)]) / copies
        del buf
        return us

    def hbm_write(self, nbytes, copies):
        torch = self.torch
        buf = torch.empty(nbytes * copies // 2, dtype=torch.float16, device="cuda")
        base = buf.data_ptr()
        us = self.time(lambda: [self._check(self.lib.aqmbc_hbm_write(base + c * nbytes, nbytes, 4 * self.n_cu,
                                                                     self._st()))
                                for c in range(copies)]) / copies
        del buf
        return us

    def lds_gather(self, nrep, dot, rounds=200):
        """G gathers/s of replicated random 16-byte LDS reads (one 1024-thread workgroup per CU)."""
        torch = self.torch
        codes = torch.randint(0, 2 ** 31 - 1, (4096,), dtype=torch.int32, device="cuda")
        n = self.n_cu
        us = self.time(lambda: self._check(self.lib.aqmbc_lds_gather(codes.data_ptr(), n, rounds, nrep, int(dot),
                                                                     self.sink.data_ptr(), self._st())))
        return n * 1024 * 16 * rounds / (us * 1e-6) / 1e9

    def lds_gather_paired(self, rounds=200):
        """G gathers/s of random 16-byte LDS reads in the matrix-core GEMV's paired layout."""
        torch = self.torch
        codes = torch.randint(0, 2 ** 31 - 1, (4096,), dtype=torch.int32, device="cuda")
        n = self.n_cu
        us = self.time(lambda: self._check(self.lib.aqmbc_lds_gather_paired(codes.data_ptr(), n, rounds,
                                                                            self.sink.data_ptr(), self._st())))
        return n * 1024 * 16 * rounds / (us * 1e-6) / 1e9

    def l2_gather(self, table_bytes, n_wg, rounds=64):
        torch = self.torch
        log2n = int(np.log2(table_bytes // 16))
        table = torch.randn(table_bytes // 2, device="cuda").to(torch.float16)
        us = self.time(lambda: self._check(self.lib.aqmbc_l2_gather(table.data_ptr(), log2n, n_wg, rounds,
                                                                    self.sink.data_ptr(), self._st())))
        return n_wg * 1024 * 8 * rounds / (us * 1e-6) / 1e9

    def mfma_bf16(self, random_ops=True, rounds=4000):
        torch = self.torch
        ops = (torch.randn(512 * 8, device="cuda") if random_ops else torch.zeros(512 * 8, device="cuda")).to(torch.bfloat16)
        n = self.n_cu
        us = self.time(lambda: self._check(self.lib.aqmbc_mfma_bf16(ops.data_ptr(), n, rounds, self.sink.data_ptr(),
                                                                    self._st())), reps=5)
        flops = n * 4 * rounds * 8 * 2.0 * 32 * 32 * 16
        return flops / (us * 1e-6) / 1e12


def time_graph(torch, stream, fn, reps=5):
    """Microseconds per replay of a HIP graph of fn's launches (one warm replay first)."""
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    g.replay()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        g.replay()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / reps


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-ceilings", action="store_true")
    ap.add_argument("--counters", choices=["gemv", "gemm", "dequant"], default=None,
                    help="counter-collection run: eager launches (gemv: the MLP-pair GEMVs at every batch and k and "
                         "the 4096 x 4096 GEMV at batch 1 and 4, every k; gemm: the prefill GEMM at k = 1 and 4; "
                         "dequant: the 4096 x 4096 dequant to bf16 at every k), then one plain 256 MiB device copy "
                         "that calibrates the HBM byte counters")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): the library has no multi-GPU "
              f"path (no collectives, no sharded layers)", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2606_12876_amd as A
    from workloads import config, make_layer, make_activations, make_weights, make_calibration_inputs

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count

    def to_dev(a):
        a = np.ascontiguousarray(a)
        return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).to(dev)

    def copies(spec, R):
        """R layer handles: the seeded layer with its code planes rotated along rows by 61 r rows (distinct
        bytes, same statistics), rotated on the device."""
        L = make_layer(spec)
        desc = A.make_desc(spec.d_out, spec.d_in, spec.M, spec.B)
        codes = to_dev(L.codes)
        cb, sc = to_dev(L.codebooks), to_dev(L.scales)
        hs = []
        for r in range(R):
            c = codes if r == 0 else torch.roll(codes, shifts=(61 * r) % spec.d_out, dims=1).contiguous()
            hs.append(A.create(desc, c, cb, sc))
            del c
        torch.cuda.synchronize()
        return L, hs

    def n_copies(spec):
        plane = spec.d_out * (spec.d_in // 8) * {4: 0.5, 8: 1, 16: 2}[spec.B]
        return int(np.ceil(STREAM_BYTES / plane))

    DT = {"f16": (torch.float16, A.DType.F16), "bf16": (torch.bfloat16, A.DType.BF16)}

    # ---------------------------------------------------------------- counter runs
    if args.counters:
        run_counters(args.counters, A, torch, dev, config, make_layer, make_activations, copies, n_copies, DT, to_dev)
        return

    # ---------------------------------------------------------------- workloads
    ops = []     # dicts: name, shape, k, b, fn, n, bytes, flops, kernel

    # headline: the MLP pair, both layers
    gemv_layers = {}
    for name in ("mlp_up", "mlp_down", "b16", "square"):
        spec = config(name)
        R = n_copies(spec)
        log(f"creating {R} copies of {spec.name}")
        L, hs = copies(spec, R)
        tdt, adt = DT[spec.act_dtype]
        batches = spec.batches
        xs = {b: to_dev(make_activations(L, b)).view(tdt) for b in batches}
        ys = {b: [torch.empty((b, spec.d_out), dtype=tdt, device=dev) for _ in range(R)] for b in batches}
        gemv_layers[name] = (spec, L, hs, xs, ys, adt)
        for k in spec.ks:
            for b in batches:
                def fn(hs=hs, k=k, b=b, xs=xs, ys=ys, adt=adt):
                    for h, y in zip(hs, ys[b]):
                        A.gemv(h, k, xs[b], adt, b, y, adt)
                ops.append(dict(name="gemv", shape=spec.name, k=k, b=b, fn=fn, n=R,
                                bytes=gemv_bytes(spec.d_out, spec.d_in, spec.B, k, b),
                                rows_groups=spec.d_out * (spec.d_in // 8), code_bits=spec.B,
                                kernel=gemv_kernel_name(spec, k, b, spec.act_dtype)))

    # 4096 x 4096 several layers per launch
    spec2, L2, hs2, xs2, ys2, _ = gemv_layers["square"]
    for G in (4, 16):
        for k in KS:
            for b in (1, 4):
                def fn(G=G, k=k, b=b):
                    for r0 in range(0, len(hs2) - G + 1, G):
                        A.gemv_multi(hs2[r0:r0 + G], k, xs2[b], A.DType.F16, b, ys2[b][r0:r0 + G], A.DType.F16)
                ops.append(dict(name=f"gemv_multi{G}", shape=spec2.name, k=k, b=b, fn=fn, n=len(hs2) // G * G,
                                bytes=gemv_bytes(4096, 4096, 8, k, b), kernel="multi-layer"))

    # 4-bit codes, same shape
    import dataclasses
    spec4 = dataclasses.replace(spec2, name="square_4096x4096_B4", B=4, seed=spec2.seed + 100, batches=(1,))
    R4 = n_copies(spec4)
    log(f"creating {R4} copies of {spec4.name}")
    L4, hs4 = copies(spec4, R4)
    ys4 = [torch.empty((1, 4096), dtype=torch.float16, device=dev) for _ in range(R4)]
    for k in KS:
        def fn(k=k):
            for h, y in zip(hs4, ys4):
                A.gemv(h, k, xs2[1], A.DType.F16, 1, y, A.DType.F16)
        ops.append(dict(name="gemv4", shape=spec4.name, k=k, b=1, fn=fn, n=R4,
                        bytes=gemv_bytes(4096, 4096, 4, k, 1), kernel="gemv_b4_kernel"))

    # dequant to bf16 over 16 output buffers (512 MiB written per burst)
    n_w = 16
    Ws = [torch.empty((4096, 4096), dtype=torch.bfloat16, device=dev) for _ in range(n_w)]
    for k in KS:
        def fn(k=k):
            for r in range(n_w):
                A.dequant(hs2[r * 7], k, Ws[r], A.DType.BF16)
        ops.append(dict(name="dequant", shape=spec2.name, k=k, b=0, fn=fn, n=n_w,
                        bytes=k * 4096 * 512 + k * 4096 + 2 * 4096 + 2 * 4096 * 4096, kernel="dequant8_tile_kernel"))

    # prefill GEMM
    gspec = config("prefill")
    n_tok = gspec.n_tokens
    G_COPIES = 4
    Lg, glayers = copies(gspec, G_COPIES)
    Xg = to_dev(make_activations(Lg, n_tok, "bf16")).view(torch.bfloat16)
    Yg = [torch.empty((n_tok, gspec.d_out), dtype=torch.bfloat16, device=dev) for _ in range(G_COPIES)]
    gflop = 2.0 * n_tok * gspec.d_out * gspec.d_in
    # the library's fastest path: aqmb_gemm_ws with a workspace (two passes where the library
    # takes them, k >= 3 here; aqmb_gemm's one-pass kernel otherwise), and aqmb_gemm itself where
    # the two-pass path runs, for reference
    ws_bytes = {k: A.gemm_workspace_bytes(glayers[0], k, n_tok) for k in KS}
    gws = torch.empty((max(max(ws_bytes.values()), 512) // 2,), dtype=torch.int16, device=dev)
    for k in KS:
        def fn(k=k):
            for h, Y in zip(glayers, Yg):
                A.gemm_ws(h, k, Xg, n_tok, Y, A.DType.BF16, gws)
        two = ws_bytes[k] > 0
        ops.append(dict(name="gemm", shape=gspec.name, k=k, b=n_tok, fn=fn, n=G_COPIES, flops=gflop,
                        kernel=("gemm_wtile_kernel + gemm_dense_kernel" if two else f"gemm_kernel<K={k}>"),
                        workspace_bytes=ws_bytes[k]))
        if two:
            def fn1(k=k):
                for h, Y in zip(glayers, Yg):
                    A.gemm(h, k, Xg, n_tok, Y, A.DType.BF16)
            ops.append(dict(name="gemm_one_pass", shape=gspec.name, k=k, b=n_tok, fn=fn1, n=G_COPIES, flops=gflop,
                            kernel=f"gemm_kernel<K={k}>"))

    # prefix distortions and beam search (4096 x 4096 layer, dense fp16 W)
    n_cal = 4096
    Wd = to_dev(make_weights(L2)).view(torch.float16)
    Xd = to_dev(make_activations(L2, n_cal, "f16")).view(torch.float16)
    D_COPIES = 4
    Ds = [torch.empty((4,), dtype=torch.float64, device=dev) for _ in range(D_COPIES)]

    def dist_fn():
        for r in range(D_COPIES):
            A.prefix_distortion_noalloc(hs2[r], Wd, A.DType.F16, Xd, A.DType.F16, n_cal, Ds[r])
    ops.append(dict(name="distortion", shape=spec2.name, k=4, b=n_cal, fn=dist_fn, n=D_COPIES,
                    flops=2.0 * 5 * 4096 * 4096 * n_cal, kernel="distortion_kernel<4, 8> + distortion_reduce_kernel"))
    desc2 = A.make_desc(4096, 4096, 4, 8)
    beam_codes = torch.empty((BEAM_K, 4096, 512), dtype=torch.uint8, device=dev)
    beam_errs = torch.empty((4096, 512), dtype=torch.float32, device=dev)
    cb2, sc2 = to_dev(L2.codebooks), to_dev(L2.scales)

    def beam_fn():
        A.beam_search(desc2, BEAM_K, BEAM_WIDTH, Wd, cb2, sc2, beam_codes, beam_errs)
    beam_cands = 4096 * 512 * 256 * (1 + (BEAM_K - 1) * BEAM_WIDTH)
    ops.append(dict(name="beam", shape=spec2.name, k=BEAM_K, b=BEAM_WIDTH, fn=beam_fn, n=1,
                    flops=beam_cands * 23.0, kernel=f"beam_kernel<{BEAM_WIDTH}>"))
    # the data-aware search: the 8 x 8 diagonal blocks of X X^T / n of seeded calibration inputs
    # (input preparation with torch, outside the timed region)
    Xc = torch.from_numpy(make_calibration_inputs(L2, n_cal)).to(dev, torch.float32)     # [d_in][n]
    Xg = Xc.view(512, 8, n_cal)
    Hblk = (torch.bmm(Xg, Xg.transpose(1, 2).contiguous()) / n_cal).contiguous()        # [G][8][8] fp32
    wbeam_codes = torch.empty_like(beam_codes)
    wbeam_errs = torch.empty_like(beam_errs)

    def wbeam_fn():
        A.beam_search_weighted(desc2, BEAM_K, BEAM_WIDTH, Wd, cb2, sc2, Hblk, wbeam_codes, wbeam_errs)
    ops.append(dict(name="beam_weighted", shape=spec2.name, k=BEAM_K, b=BEAM_WIDTH, fn=wbeam_fn, n=1,
                    flops=beam_cands * 19.0, kernel=f"beam_weighted_kernel<{BEAM_WIDTH}>"))
    torch.cuda.synchronize()

    # eager reference of one headline burst, for the graph check below
    ref_op = [o for o in ops if o["name"] == "gemv" and o["shape"].startswith("mlp_up") and o["k"] == 4 and o["b"] == 1][0]
    ref_op["fn"]()
    torch.cuda.synchronize()
    yref = gemv_layers["mlp_up"][4][1][0].clone()

    log(f"capturing {len(ops)} bursts")
    graphs = []
    for o in ops:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            o["fn"]()
        graphs.append(g)
    torch.cuda.synchronize()

    def run_step(record):
        for i, g in enumerate(graphs):
            if record is not None:
                record[i][0].record(stream)
            g.replay()
            if record is not None:
                record[i][1].record(stream)

    for _ in range(args.warmup):
        run_step(None)
    torch.cuda.synchronize()
    gemv_layers["mlp_up"][4][1][0].zero_()
    graphs[ops.index(ref_op)].replay()
    torch.cuda.synchronize()
    assert torch.equal(gemv_layers["mlp_up"][4][1][0], yref), "graph replay differs from the eager GEMV"

    log(f"timing {args.steps} steps")
    events = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in ops]
              for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        run_step(events[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    for i, o in enumerate(ops):
        ms = sum(events[s][i][0].elapsed_time(events[s][i][1]) for s in range(args.steps))
        o["step_us"] = ms * 1e3 / args.steps
        o["us"] = o["step_us"] / o["n"]

    def gbps(o):
        return o["bytes"] / (o["us"] * 1e-6) / 1e9

    # ---------------------------------------------------------------- ceilings
    ceil = None
    if not args.no_ceilings:
        log("measuring ceilings")
        ceil = measure_ceilings(torch, stream, n_cu, ops)

    # ---------------------------------------------------------------- report
    head = [o for o in ops if o["name"] == "gemv" and o["shape"].startswith("mlp_")]
    value = sum(o["bytes"] * o["n"] for o in head) / (sum(o["step_us"] for o in head) * 1e-6) / 1e9
    per_k = {}
    for k in KS:
        e = {}
        for o in head:
            if o["k"] != k:
                continue
            key = f"{'up' if 'up' in o['shape'] else 'down'}_b{o['b']}"
            r = {"us": round(o["us"], 3), "GBps": round(gbps(o), 1), "frac_hbm": round(gbps(o) / HBM_PEAK_GBPS, 4),
                 "kernel": o["kernel"]}
            if ceil:
                r.update(binding_fracs(o, ceil))
            e[key] = r
        per_k[str(k)] = e
    dom = max(head, key=lambda o: o["step_us"])
    ach = gbps(dom)
    roofline = {"bound": "hbm", "kernel": f"{dom['kernel']} on {dom['shape']}, k={dom['k']}",
                "achieved": round(ach, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBPS, 4),
                "traffic": measured_traffic(f"{dom['shape']}:k{dom['k']}:b{dom['b']}"),
                "bytes_per_launch": dom["bytes"], "us_per_launch": round(dom["us"], 3),
                "share_of_headline_time": round(dom["step_us"] / sum(o["step_us"] for o in head), 4)}
    if ceil:
        roofline["ceilings"] = binding_fracs(dom, ceil)

    out = {
        "metric": "code-plane GEMV HBM GB/s (% peak) per bitwidth k; prefill GEMM TFLOP/s",
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / args.steps, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "decode GEMV of the Llama-7B MLP pair, 11008x4096 (up) and 4096x11008 (down), "
                               "M=4 codebooks of 256x8 fp16, uint8 codes, bf16 x (0.1% of entries x20) and bf16 y, "
                               "batch 1, 8 and 16, k=1..4",
                   "layer_copies": {n: len(v[2]) for n, v in gemv_layers.items()},
                   "launch": "HIP graph per burst of copies", "accumulate": "fp32",
                   "per_step_also": "16-bit-code 14336x4096 GEMV (k=1,2); 4096x4096 GEMV (batch 1, 4; single "
                                    "and 4/16 layers per launch; 4-bit codes); dequant 4096x4096 to bf16; "
                                    "2048-token prefill GEMM; prefix distortions; beam search (plain and data-aware)"},
        "per_k": per_k,
        "roofline": roofline,
    }
    out["gemv_other"] = other_gemv(ops, gbps, ceil)
    gemm = [o for o in ops if o["name"] == "gemm"]
    for o in gemm:
        o["tflops"] = o["flops"] / (o["us"] * 1e-6) / 1e12
    g4 = [o for o in gemm if o["k"] == 4][0]
    one_pass = {o["k"]: o for o in ops if o["name"] == "gemm_one_pass"}
    out["roofline_gemm"] = {"bound": "mfma", "kernel": f"{g4['kernel']} (k=4), 2048 x 4096 x 4096", "achieved": round(g4["tflops"], 1),
                            "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": round(g4["tflops"] / BF16_PEAK_TFLOPS, 4),
                            "traffic": None, "us_per_launch": round(g4["us"], 2),
                            "entry_point": "aqmb_gemm_ws (caller workspace; two passes at k >= 3: bf16 weight "
                                           "tiles, then a dense matrix-core GEMM, bit-identical to aqmb_gemm)",
                            "per_k": {str(o["k"]): {"us": round(o["us"], 2), "TFLOPs": round(o["tflops"], 1),
                                                    "frac_bf16_peak": round(o["tflops"] / BF16_PEAK_TFLOPS, 4),
                                                    "kernel": o["kernel"], "workspace_bytes": o["workspace_bytes"],
                                                    **({"one_pass_us": round(one_pass[o["k"]]["us"], 2)}
                                                       if o["k"] in one_pass else {})}
                                      for o in gemm}}
    if ceil:
        out["roofline_gemm"]["ceiling"] = {"kind": "mfma_bf16 on random operands (measured)",
                                           "TFLOPs": round(ceil["mfma_bf16_random_TFLOPs"], 1),
                                           "frac": round(g4["tflops"] / ceil["mfma_bf16_random_TFLOPs"], 4)}
    out["gemm_TFLOPs"] = round(len(gemm) * gflop / (sum(o["us"] for o in gemm) * 1e-6) / 1e12, 1)
    dq = [o for o in ops if o["name"] == "dequant"]
    out["roofline_dequant"] = {"bound": "hbm", "kernel": "dequant8_tile_kernel (bf16 out), 4096 x 4096", "unit": "GB/s",
                               "peak": HBM_PEAK_GBPS,
                               "per_k": {str(o["k"]): {"us": round(o["us"], 3), "GBps": round(gbps(o), 1),
                                                       "frac": round(gbps(o) / HBM_PEAK_GBPS, 4)} for o in dq}}
    if ceil:
        w = ceil["hbm_write_32MiB_GBps"]
        out["roofline_dequant"]["ceiling"] = {"kind": "plain 32 MiB write per launch (measured)", "GBps": round(w, 1)}
        for o in dq:
            out["roofline_dequant"]["per_k"][str(o["k"])]["frac_write_ceiling"] = round(gbps(o) / w, 4)
    od = [o for o in ops if o["name"] == "distortion"][0]
    achd = od["flops"] / (od["us"] * 1e-6) / 1e12
    out["roofline_distortion"] = {"bound": "mfma", "kernel": od["kernel"], "achieved": round(achd, 1),
                                  "peak": F16_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": round(achd / F16_PEAK_TFLOPS, 4),
                                  "traffic": None, "us_per_launch": round(od["us"], 2),
                                  "entry_point": "aqmb_prefix_distortion_noalloc (graph-captured)",
                                  "workload": f"D^(1..4) of a 4096x4096 layer, dense fp16 W, {n_cal} fp16 inputs"}
    ob = [o for o in ops if o["name"] == "beam"][0]
    achb = ob["flops"] / (ob["us"] * 1e-6) / 1e12
    out["roofline_beam"] = {"bound": "alu", "kernel": ob["kernel"] + f" (k={BEAM_K})", "achieved": round(achb, 2),
                            "peak": round(FP32_PLAIN_PEAK_TOPS, 2), "unit": "TFLOP/s",
                            "frac": round(achb / FP32_PLAIN_PEAK_TOPS, 4), "traffic": None,
                            "us_per_launch": round(ob["us"], 1), "candidates_per_s": round(beam_cands / (ob["us"] * 1e-6), 1),
                            "workload": f"codes for the 2097152 groups of a 4096x4096 fp16 W, k={BEAM_K} "
                                        f"codebooks of 256, beam {BEAM_WIDTH}"}
    ow = [o for o in ops if o["name"] == "beam_weighted"][0]
    achw = ow["flops"] / (ow["us"] * 1e-6) / 1e12
    out["roofline_beam_weighted"] = {
        "bound": "alu", "kernel": ow["kernel"] + f" (k={BEAM_K})", "achieved": round(achw, 2),
        "peak": round(FP32_PLAIN_PEAK_TOPS, 2), "unit": "TFLOP/s", "frac": round(achw / FP32_PLAIN_PEAK_TOPS, 4),
        "traffic": None, "us_per_launch": round(ow["us"], 1),
        "candidates_per_s": round(beam_cands / (ow["us"] * 1e-6), 1),
        "workload": f"codes for the 2097152 groups of a 4096x4096 fp16 W minimising d^T H_j d (H_j: 8x8 blocks of "
                    f"X X^T / n over {n_cal} calibration inputs), k={BEAM_K} codebooks of 256, beam {BEAM_WIDTH}"}
    if ceil:
        out["ceilings"] = {k: (round(v, 2) if isinstance(v, float) else v) for k, v in ceil.items()}
    tot = sum(o["step_us"] for o in ops)
    share = {}
    for o in ops:
        key = "gemv_mlp" if o in head else o["name"] if o["name"] != "gemv" else f"gemv_{o['shape'].split('_')[0]}"
        share[key] = share.get(key, 0.0) + o["step_us"] / tot
    out["time_share"] = {k: round(v, 4) for k, v in share.items()}

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(gemv_layers)
        dist_cpu, beam_cpu, wbeam_cpu = cpu_oracle_widened(L2, make_weights, make_activations, Hblk.cpu().numpy())
        out["roofline_distortion"]["cpu_oracle"] = dist_cpu
        out["roofline_beam"]["cpu_oracle"] = beam_cpu
        out["roofline_beam_weighted"]["cpu_oracle"] = wbeam_cpu
    print(json.dumps(out), flush=True)
    for v in gemv_layers.values():
        for h in v[2]:
            A.destroy(h)
    for h in hs4 + glayers:
        A.destroy(h)


def binding_fracs(o, ceil):
    """A GEMV launch against the measured ceilings: attainable HBM for a launch of its size on one
    workgroup per CU, and the gather rate its codewords need (LDS for 8-bit codes, L2 for 16-bit)."""
    r = {}
    att = ceil.get("hbm_read_per_launch_us", {}).get(str(launch_read_bytes(o)))
    if att:
        r["attainable_hbm_us"] = att
        r["frac_attainable_hbm"] = round(att / o["us"], 4)
    spec_rows = o.get("rows_groups")
    if spec_rows:
        # one codeword gather per code (the matrix-core kernel serves every batch row with it; the
        # direct-gather kernel at batch 1 also spends 4 fp16 dot products on it)
        gathers = spec_rows * o["k"]
        # the direct-gather kernel (batch 1) is bound by its gathers with their dot products; the
        # matrix-core kernel gathers from the conflict-free paired layout
        kind = ("l2_gather_G_per_s" if o.get("code_bits") == 16 else
                "lds_gather_paired_G_per_s" if "gemv_mma" in o.get("kernel", "") else "lds_gather_dot_G_per_s")
        rate = ceil.get(kind)
        if rate:
            t = gathers / (rate * 1e9) * 1e6
            r["gather_bound"] = kind
            r["gather_bound_us"] = round(t, 3)
            r["frac_gather_bound"] = round(t / o["us"], 4)
    return r


def launch_read_bytes(o):
    """Bytes the attainable-HBM probe reads for a GEMV launch: its algorithmic bytes, rounded up to 64 KiB."""
    return (o["bytes"] + 65535) // 65536 * 65536


def measure_ceilings(torch, stream, n_cu, ops):
    c = Ceilings(torch, stream)
    res = {}
    res["hbm_read_stream_1GiB_GBps"] = (1 << 30) / (c.hbm_read(1 << 30, 2, 4 * n_cu) * 1e-6) / 1e9
    # one launch of each GEMV size (rounded to whole MiB) on one 1024-thread workgroup per CU, 1 GiB rotated
    per = {}
    for o in ops:
        if o["name"] == "gemv":
            nb = launch_read_bytes(o)
            if str(nb) not in per:
                per[str(nb)] = round(c.hbm_read(nb, max(2, (1 << 30) // nb), n_cu), 3)
    res["hbm_read_per_launch_us"] = per
    res["hbm_read_per_launch_note"] = ("us per launch reading N bytes (key: a GEMV launch's algorithmic bytes rounded "
                                       "up to 64 KiB) with one 1024-thread workgroup per CU, rotating over 1 GiB of "
                                       "buffers, graph-replayed like the GEMV bursts")
    res["hbm_write_32MiB_GBps"] = (32 << 20) / (c.hbm_write(32 << 20, 16) * 1e-6) / 1e9
    res["lds_gather_G_per_s"] = c.lds_gather(8, False)
    res["lds_gather_dot_G_per_s"] = c.lds_gather(8, True)
    res["lds_gather_paired_G_per_s"] = c.lds_gather_paired()
    res["lds_gather_note"] = ("random 16-byte LDS reads from 4 codebooks of 256 codewords stored 8 times interleaved "
                              "(the direct-gather GEMV's layout), one 1024-thread workgroup per CU; _dot adds the 4 "
                              "fp16 dot products per codeword of the batch-1 GEMV; _paired: the matrix-core GEMV's conflict-free "
                              "layout (two codebooks per 256-byte row, 8 copies each)")
    l2 = {}
    for tb in (1 << 20, 2 << 20):
        l2[f"{tb >> 20}MiB"] = max(c.l2_gather(tb, n_cu), c.l2_gather(tb, 2 * n_cu))
    res["l2_gather_G_per_s_by_table"] = {k: round(v, 1) for k, v in l2.items()}
    res["l2_gather_G_per_s"] = l2["2MiB"]
    res["l2_gather_note"] = ("random 16-byte global loads from a 1 or 2 MiB table (the 16-bit-code codebooks at k = 1, 2), "
                             "8 in flight per lane, 1 or 2 workgroups of 1024 per CU (the faster)")
    res["mfma_bf16_random_TFLOPs"] = c.mfma_bf16(True)
    res["mfma_bf16_zeros_TFLOPs"] = c.mfma_bf16(False)
    return res


def other_gemv(ops, gbps, ceil):
    res = {}
    for o in ops:
        if o["name"] == "gemv" and o["shape"].startswith("mlp_"):
            continue
        if not o["name"].startswith("gemv"):
            continue
        key = f"{o['name']}:{o['shape']}"
        e = res.setdefault(key, {})
        per_layer = o["name"].startswith("gemv_multi")
        r = {"us_per_layer" if per_layer else "us": round(o["us"], 3), "GBps": round(gbps(o), 1),
             "frac_hbm": round(gbps(o) / HBM_PEAK_GBPS, 4)}
        if ceil and not per_layer:
            r.update(binding_fracs(o, ceil))
        e[f"k{o['k']}_b{o['b']}"] = r
    return res


def run_counters(mode, A, torch, dev, config, make_layer, make_activations, copies, n_copies, DT, to_dev):
    """Eager launches for rocprofv3 counter passes (no graphs: the profiler sees each dispatch), then one
    plain 256 MiB device copy that calibrates FETCH_SIZE and WRITE_SIZE."""
    meta = {"mode": f"counters-{mode}", "ops": []}
    if mode == "gemv":
        for name in ("mlp_up", "mlp_down", "square"):
            spec = config(name)
            R = n_copies(spec)
            L, hs = copies(spec, R)
            tdt, adt = DT[spec.act_dtype]
            for b in spec.batches:
                x = to_dev(make_activations(L, b)).view(tdt)
                ys = [torch.empty((b, spec.d_out), dtype=tdt, device=dev) for _ in range(R)]
                for k in spec.ks:
                    for h, y in zip(hs, ys):
                        A.gemv(h, k, x, adt, b, y, adt)
                    torch.cuda.synchronize()
                    meta["ops"].append({"shape": spec.name, "k": k, "b": b, "launches": R,
                                        "kernel": gemv_kernel_name(spec, k, b, spec.act_dtype),
                                        "bytes": gemv_bytes(spec.d_out, spec.d_in, spec.B, k, b)})
            for h in hs:
                A.destroy(h)
    elif mode == "dequant":
        spec = config("square")
        R = n_copies(spec)
        L, hs = copies(spec, R)
        n_w = 16                                             # 512 MiB of outputs per burst
        Ws = [torch.empty((spec.d_out, spec.d_in), dtype=torch.bfloat16, device=dev) for _ in range(n_w)]
        for k in spec.ks:
            for r in range(4 * n_w):
                A.dequant(hs[(r * 7) % R], k, Ws[r % n_w], A.DType.BF16)
            torch.cuda.synchronize()
            meta["ops"].append({"shape": spec.name, "k": k, "launches": 4 * n_w,
                                "bytes_read": k * spec.d_out * spec.d_in // 8 + k * 4096 + 2 * spec.d_out,
                                "bytes_written": 2 * spec.d_out * spec.d_in})
        for h in hs:
            A.destroy(h)
    else:
        spec = config("prefill")
        L, hs = copies(spec, 4)
        X = to_dev(make_activations(L, spec.n_tokens, "bf16")).view(torch.bfloat16)
        Y = torch.empty((spec.n_tokens, spec.d_out), dtype=torch.bfloat16, device=dev)
        ws = torch.empty((max(A.gemm_workspace_bytes(hs[0], 4, spec.n_tokens), 512) // 2,), dtype=torch.int16, device=dev)
        for k in (1, 4):
            for _ in range(4):
                for h in hs:
                    A.gemm_ws(h, k, X, spec.n_tokens, Y, A.DType.BF16, ws)
            torch.cuda.synchronize()
            meta["ops"].append({"shape": spec.name, "k": k, "launches": 16, "flops": 2.0 * spec.n_tokens * 4096 * 4096})
    copy_bytes = 256 << 20
    src = torch.ones(copy_bytes // 2, dtype=torch.float16, device=dev)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    meta["copy_bytes"] = copy_bytes
    print(json.dumps(meta), flush=True)


def cpu_baseline(gemv_layers, rows=4096):
    """The fp64 oracle on the host cores over a bounded sample of the headline workload: the first
    `rows` output rows of both MLP layers, every k, batch 1, 8 and 16, each call the oracle's
    reconstruction of W_k and its product with x (about 10-20 s), in the same algorithmic GB/s as
    the GPU figure (bytes of the sampled rows)."""
    import oracle
    from oracle import formats
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        blas_threads = 1
    from workloads import make_activations
    total_bytes, t_total = 0, 0.0
    for name in ("mlp_up", "mlp_down"):
        spec, L, _, _, _, _ = gemv_layers[name]
        C = formats.f16_bits_to_f64(L.codebooks)
        s = formats.f16_bits_to_f64(L.scales)[:rows]
        codes = np.ascontiguousarray(L.codes[:, :rows])
        xs = {b: formats.bf16_bits_to_f64(make_activations(L, b)) for b in spec.batches}
        for k in spec.ks:
            for b, x in xs.items():
                t0 = time.perf_counter()
                oracle.linear(x, codes, C, s, k)
                t_total += time.perf_counter() - t0
                total_bytes += gemv_bytes(rows, spec.d_in, 8, k, b)
    return {"value": round(total_bytes / t_total / 1e9, 4), "unit": "GB/s", "cores": int(blas_threads),
            "kind": "oracle",
            "sample": f"the first {rows} output rows of both MLP layers, k=1..4, batch 1, 8 and 16: 24 calls of "
                      "the oracle's fp64 reconstruction of W_k and its product with x (reconstruction "
                      "single-threaded, product on the BLAS threads)",
            "seconds": round(t_total, 2), "host_cpus": len(os.sched_getaffinity(0))}


def cpu_oracle_widened(layer, make_weights, make_activations, H_blocks):
    """The oracle beside the distortion evaluator and the beam search, on bounded samples of the
    same workloads (a few seconds each): the fp64 prefix distortions of the first 2048 rows over 1024
    calibration inputs (in TFLOP/s of the same 2 (M + 1) d_out d_in n count), and the binary32
    beam search of 64 groups (in candidates/s)."""
    import oracle
    from oracle import formats
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        blas_threads = 1
    rows, n, M, d_in = 2048, 1024, 4, 4096
    C = formats.f16_bits_to_f64(layer.codebooks)
    s = formats.f16_bits_to_f64(layer.scales)
    W = formats.f16_bits_to_f64(make_weights(layer))[:rows]
    X = formats.f16_bits_to_f64(make_activations(layer, n, "f16"))
    t0 = time.perf_counter()
    oracle.prefix_distortions(W, layer.codes[:, :rows], C, s[:rows], X)
    td = time.perf_counter() - t0
    dist = {"value": round(2.0 * (M + 1) * rows * d_in * n / td / 1e12, 4), "unit": "TFLOP/s",
            "cores": int(blas_threads), "kind": "oracle", "seconds": round(td, 2),
            "sample": f"fp64 prefix distortions of {rows} rows x {d_in} over {n} inputs (reconstruction "
                      f"single-threaded, products on BLAS)"}
    groups = [(i, j) for i in range(8) for j in range(8)]
    t0 = time.perf_counter()
    oracle.beam_search_codes_f32(formats.f16_bits_to_f64(make_weights(layer)[:8]), C[:BEAM_K], s[:8], BEAM_K,
                                 BEAM_WIDTH, groups=groups)
    tb = time.perf_counter() - t0
    cands = len(groups) * 256 * (1 + (BEAM_K - 1) * BEAM_WIDTH)
    beam = {"value": round(cands / tb, 1), "unit": "candidates/s", "cores": 1, "kind": "oracle",
            "seconds": round(tb, 2), "sample": f"binary32 beam search (k={BEAM_K}, beam {BEAM_WIDTH}) of "
                                                f"{len(groups)} groups, one thread"}
    t0 = time.perf_counter()
    oracle.beam_search_codes_weighted_f32(formats.f16_bits_to_f64(make_weights(layer)[:8]), C[:BEAM_K], s[:8],
                                          H_blocks.astype("float64"), BEAM_K, BEAM_WIDTH, groups=groups)
    tw = time.perf_counter() - t0
    wbeam = {"value": round(cands / tw, 1), "unit": "candidates/s", "cores": 1, "kind": "oracle",
             "seconds": round(tw, 2), "sample": f"binary32 data-aware beam search (k={BEAM_K}, beam {BEAM_WIDTH}) "
                                                 f"of {len(groups)} groups, one thread"}
    return dist, beam, wbeam


if __name__ == "__main__":
    main()
