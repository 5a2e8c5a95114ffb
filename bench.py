"""Benchmark of the multi-bitwidth additive-codebook linear layer on one MI355X.

One step is one pass of the whole hot path over a stack of R resident copies of the
workload layer (R distinct weight sets, like R layers of a model, so that the working set
exceeds the 256 MB Infinity Cache and every launch streams its codes from HBM):

  for k in 1..4:   decode GEMV at batch 1 and batch 4   (4096 x 4096, M = 4, uint8 codes, fp16 x/y)
                   dequantization to bf16                 (same layers)
                   prefill GEMM, 2048 bf16 tokens          (4096 x 4096 layer, bf16 out)
  once:            prefix distortions D^(1..4) of the decode layer against a dense fp16 W
                   over 4096 fp16 calibration inputs
                   beam search (k = 4, beam 8) of codes for every group of that W
  for k in 1..4:   decode GEMV at batch 1 of the same shape stored as 4 codebooks of 16
                   codewords (4-bit codes, 64 copies)

Each (operation, k, batch) runs as a burst of R launches captured in a HIP graph and timed
with HIP events on the launch stream; the per-launch time is burst time / R.

`value` is the decode GEMV throughput in algorithmic GB/s (code planes 0..k-1, their
codebooks, scales, x and y) over all GEMV launches of the timed steps. `roofline` describes the
GEMV kernel at batch 1, k = 4 (HBM-bound); `roofline_gemm` the prefill GEMM at k = 4
(MFMA-bound); `roofline_distortion` the distortion evaluator (fp16 MFMA-bound, algorithmic
flops 2 (M + 1) d_out d_in n: W X and one product per code plane); `roofline_beam` the code search
(ALU-bound: 23 binary32 operations per candidate, against the chip's non-packed, non-fused fp32
rate 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz = 39.3 Tops/s). The CPU baseline is the fp64
oracle timed on a bounded sample.

After the timed steps, `secondary` holds measurements taken once: the decode GEMV on the other
layer shapes (1024 x 1024; 11008 x 4096 and 4096 x 11008 at batch 1, 8, 16 with bf16 x/y; 14336
x 4096 with two codebooks of 65536 codewords), the prefill GEMM with 4-bit codes, and two
labelled reference points (the GEMV on one cache-resident layer; the platform BLAS bf16 GEMM of
the prefill shape on dense weights).

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
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


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def measured_traffic():
    """HBM bytes per launch of the dominant GEMV kernel, from the committed counter summary.

    The summary records a hash of the kernel sources it was measured on; once they change the
    figure no longer applies and None is returned.
    """
    import hashlib
    path = os.path.join(ROOT, "profiles", "gemv_k4_b1_hbm_traffic.md")
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if ":" in line and line.split(":", 1)[0] in ("traffic_bytes_per_launch", "sources_sha256"):
            key, val = line.split(":", 1)
            fields[key] = val.strip()
    h = hashlib.sha256()
    for f in ("paper_2606_12876_amd/csrc/k_gemv.hip", "paper_2606_12876_amd/csrc/device.h"):
        h.update(open(os.path.join(ROOT, f), "rb").read())
    if fields.get("sources_sha256") != h.hexdigest():
        return None
    return float(fields["traffic_bytes_per_launch"])


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--copies", type=int, default=64, help="resident layer copies per GEMV step")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-gemm", action="store_true")
    ap.add_argument("--no-secondary", action="store_true", help="skip the once-only measurements after the timed steps")
    ap.add_argument("--counters", action="store_true",
                    help="counter-collection run: eager GEMV launches (k = 4, batch 1) over the layer copies, "
                         "then one plain device copy of 256 MiB that calibrates the HBM byte counters")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): this build has no multi-GPU "
              f"path; see DESIGN.md for how the layer would shard", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2606_12876_amd as A
    from workloads import config, make_layer, make_activations

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()

    def to_dev(a):
        a = np.ascontiguousarray(a)
        return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).to(dev)

    # ---------------------------------------------------------------- decode workload
    spec = config("c2")
    R = args.copies
    d_out, d_in, M = spec.d_out, spec.d_in, spec.M
    log(f"creating {R} copies of the {d_out}x{d_in} M={M} layer")
    base = make_layer(spec)
    layers, xs1, xs4, ys1, ys4 = [], [], [], [], []
    rng = np.random.default_rng(1234)
    desc = A.make_desc(d_out, d_in, M, 8)
    for r in range(R):
        # copy r: the seeded layer with its code planes permuted along rows (distinct bytes, same statistics)
        codes = base.codes if r == 0 else np.ascontiguousarray(np.roll(base.codes, r * 61, axis=1))
        layers.append(A.create(desc, to_dev(codes), to_dev(base.codebooks), to_dev(base.scales)))
    x1 = make_activations(base, 1, "f16")
    x4 = make_activations(base, 4, "f16")
    for r in range(R):
        xs1.append(to_dev(x1).view(torch.float16))
        xs4.append(to_dev(x4).view(torch.float16))
        ys1.append(torch.empty((1, d_out), dtype=torch.float16, device=dev))
        ys4.append(torch.empty((4, d_out), dtype=torch.float16, device=dev))
    n_w = 16
    Ws = [torch.empty((d_out, d_in), dtype=torch.bfloat16, device=dev) for _ in range(n_w)]

    if args.counters:
        # No graphs here: the profiler sees every dispatch on its own.
        reps = 4
        for _ in range(reps):
            for r in range(R):
                A.gemv(layers[r], 4, xs1[r], A.DType.F16, 1, ys1[r], A.DType.F16)
        copy_bytes = 256 << 20
        src = torch.ones(copy_bytes // 2, dtype=torch.float16, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"mode": "counters", "gemv_launches": reps * R, "gemv_k": 4, "gemv_batch": 1,
                          "gemv_bytes_per_launch": 4 * (d_out * d_in // 8) + 4 * 256 * 8 * 2 + 2 * d_out
                          + 2 * (d_in + d_out), "copy_bytes": copy_bytes}), flush=True)
        return

    # ---------------------------------------------------------------- prefill workload
    gspec = config("c5")
    n_tok = gspec.n_tokens
    G_COPIES = 4
    if not args.no_gemm:
        gl = make_layer(gspec)
        gdesc = A.make_desc(gspec.d_out, gspec.d_in, gspec.M, 8)
        glayers = [A.create(gdesc, to_dev(gl.codes if r == 0 else np.roll(gl.codes, r * 61, axis=1)),
                            to_dev(gl.codebooks), to_dev(gl.scales)) for r in range(G_COPIES)]
        Xg = to_dev(make_activations(gl, n_tok, "bf16")).view(torch.bfloat16)
        Yg = [torch.empty((n_tok, gspec.d_out), dtype=torch.bfloat16, device=dev) for _ in range(G_COPIES)]
    # ---------------------------------------------------------------- distortion workload
    n_cal = 4096
    from workloads import make_weights
    Wd = to_dev(make_weights(base)).view(torch.float16)
    Xd = to_dev(make_activations(base, n_cal, "f16")).view(torch.float16)
    D_COPIES = 4
    Ds = [torch.empty((M,), dtype=torch.float64, device=dev) for _ in range(D_COPIES)]
    G_groups = d_in // 8
    beam_codes = torch.empty((BEAM_K, d_out, G_groups), dtype=torch.uint8, device=dev)
    beam_errs = torch.empty((d_out, G_groups), dtype=torch.float32, device=dev)
    cb_dev, sc_dev = to_dev(base.codebooks), to_dev(base.scales)
    # the same shape with 4-bit codes (4 codebooks of 16 codewords), R copies
    import dataclasses
    spec4 = dataclasses.replace(spec, name="c2_b4", B=4, seed=spec.seed + 100)
    base4 = make_layer(spec4)
    desc4 = A.make_desc(d_out, d_in, M, 4)
    layers4 = [A.create(desc4, to_dev(base4.codes if r == 0 else np.ascontiguousarray(np.roll(base4.codes, r * 61, axis=1))),
                        to_dev(base4.codebooks), to_dev(base4.scales)) for r in range(R)]
    torch.cuda.synchronize()

    ks = list(spec.ks)

    def gemv_burst(k, b):
        for r in range(R):
            x, y = (xs1[r], ys1[r]) if b == 1 else (xs4[r], ys4[r])
            A.gemv(layers[r], k, x, A.DType.F16, b, y, A.DType.F16)

    def dequant_burst(k):
        for r in range(n_w):
            A.dequant(layers[r], k, Ws[r], A.DType.BF16)

    def gemm_burst(k):
        for r in range(G_COPIES):
            A.gemm(glayers[r], k, Xg, n_tok, Yg[r], A.DType.BF16)

    # The same R layers decoded with aqmb_gemv_multi, G layers per launch (layers that share their
    # input, as fused q/k/v or gate/up projections do).
    MULTI_G = (4, 16)

    def gemv_multi_burst(k, b, G):
        for r0 in range(0, R - G + 1, G):
            xs, ys = (xs1, ys1) if b == 1 else (xs4, ys4)
            A.gemv_multi(layers[r0:r0 + G], k, xs[r0], A.DType.F16, b, ys[r0:r0 + G], A.DType.F16)

    def distortion_burst():
        for r in range(D_COPIES):
            A.prefix_distortion(layers[r], Wd, A.DType.F16, Xd, A.DType.F16, n_cal, Ds[r])

    def beam_burst():
        A.beam_search(desc, BEAM_K, BEAM_WIDTH, Wd, cb_dev, sc_dev, beam_codes, beam_errs)

    def gemv4_burst(k):
        for r in range(R):
            A.gemv(layers4[r], k, xs1[r], A.DType.F16, 1, ys1[r], A.DType.F16)

    ops = [("distortion", M, n_cal, distortion_burst, D_COPIES),   # (name, k, b, fn, launches)
           ("beam", BEAM_K, BEAM_WIDTH, beam_burst, 1)]
    for k in ks:
        ops.append(("gemv4", k, 1, lambda k=k: gemv4_burst(k), R))
    for k in ks:
        ops.append(("gemv", k, 1, lambda k=k: gemv_burst(k, 1), R))
        ops.append(("gemv", k, 4, lambda k=k: gemv_burst(k, 4), R))
        for G in MULTI_G:
            for b in (1, 4):
                ops.append((f"gemv_multi{G}", k, b, lambda k=k, b=b, G=G: gemv_multi_burst(k, b, G), R // G))
        ops.append(("dequant", k, 0, lambda k=k: dequant_burst(k), n_w))
        if not args.no_gemm:
            ops.append(("gemm", k, n_tok, lambda k=k: gemm_burst(k), G_COPIES))

    # Eager reference outputs for the graph check below.
    gemv_burst(4, 1)
    torch.cuda.synchronize()
    eager_y = ys1[0].clone()

    # Capture each burst in a HIP graph (the library only launches kernels on the given stream).
    graphs = []
    for (name, k, b, fn, n) in ops:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn()
        graphs.append(g)
    torch.cuda.synchronize()

    def gemv_bytes(k, b):
        return k * (d_out * d_in // 8) + k * 256 * 8 * 2 + 2 * d_out + 2 * b * (d_in + d_out)

    def run_step(record):
        for i, g in enumerate(graphs):
            if record is not None:
                e0, e1 = record[i]
                e0.record(stream)
                g.replay()
                e1.record(stream)
            else:
                g.replay()

    for w in range(args.warmup):
        run_step(None)
    torch.cuda.synchronize()
    # every replay recomputes the same outputs: check the graph against the eager result
    ys1[0].zero_()
    graphs[[i for i, o in enumerate(ops) if o[0] == "gemv" and o[1] == 4 and o[2] == 1][0]].replay()
    torch.cuda.synchronize()
    assert torch.equal(ys1[0], eager_y), "graph replay differs from the eager GEMV"

    events = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in ops]
              for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        run_step(events[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per_op_ms = np.zeros(len(ops))
    for s in range(args.steps):
        for i, (e0, e1) in enumerate(events[s]):
            per_op_ms[i] += e0.elapsed_time(e1)
    per_launch_us = {}
    for i, (name, k, b, fn, n) in enumerate(ops):
        per_launch_us[(name, k, b)] = per_op_ms[i] * 1e3 / (args.steps * n)

    gemv_total_bytes = sum(gemv_bytes(k, b) * R for (name, k, b, fn, n) in ops if name == "gemv")
    gemv_total_us = sum(per_launch_us[(name, k, b)] * R for (name, k, b, fn, n) in ops if name == "gemv")
    value = gemv_total_bytes / (gemv_total_us * 1e-6) / 1e9
    per_k = {}
    for k in ks:
        e = {}
        for b in (1, 4):
            t = per_launch_us[("gemv", k, b)]
            e[f"gemv_b{b}_us"] = round(t, 3)
            e[f"gemv_b{b}_GBps"] = round(gemv_bytes(k, b) / (t * 1e-6) / 1e9, 1)
            e[f"gemv_b{b}_frac_hbm"] = round(gemv_bytes(k, b) / (t * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)
        t = per_launch_us[("dequant", k, 0)]
        dq_bytes = k * d_out * d_in // 8 + k * 4096 + 2 * d_out + 2 * d_out * d_in
        e["dequant_us"] = round(t, 3)
        e["dequant_GBps"] = round(dq_bytes / (t * 1e-6) / 1e9, 1)
        if not args.no_gemm:
            t = per_launch_us[("gemm", k, n_tok)]
            fl = 2.0 * n_tok * gspec.d_out * gspec.d_in
            e["gemm_us"] = round(t, 2)
            e["gemm_TFLOPs"] = round(fl / (t * 1e-6) / 1e12, 1)
            e["gemm_frac_bf16_peak"] = round(fl / (t * 1e-6) / 1e12 / BF16_PEAK_TFLOPS, 4)
        per_k[str(k)] = e

    multi = {}
    for G in MULTI_G:
        mk = {}
        for k in ks:
            e = {}
            for b in (1, 4):
                t = per_launch_us[(f"gemv_multi{G}", k, b)] / G   # per layer
                e[f"b{b}_us_per_layer"] = round(t, 3)
                e[f"b{b}_GBps"] = round(gemv_bytes(k, b) / (t * 1e-6) / 1e9, 1)
                e[f"b{b}_frac_hbm"] = round(gemv_bytes(k, b) / (t * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)
            mk[str(k)] = e
        multi[str(G)] = mk

    t_dom = per_launch_us[("gemv", 4, 1)]
    ach = gemv_bytes(4, 1) / (t_dom * 1e-6) / 1e9
    gemv_kernel = "gemv_cw_kernel<K=4,NB=1>"
    roofline = {"bound": "hbm", "kernel": f"{gemv_kernel} (k=4, batch 1)", "achieved": round(ach, 1),
                "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBPS, 4),
                "traffic": measured_traffic(), "bytes_per_launch": gemv_bytes(4, 1), "us_per_launch": round(t_dom, 3)}
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
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"decode GEMV {d_out}x{d_in}, M={M} codebooks of 256x8 fp16, uint8 codes, "
                               f"fp16 x/y, batch 1 and 4, k=1..4; per k also dequant to bf16 and a "
                               f"{n_tok}-token bf16 prefill GEMM on a {gspec.d_out}x{gspec.d_in} layer",
                   "layer_copies": R, "launch": "HIP graph per burst of copies", "codes": "uint8",
                   "accumulate": "fp32"},
        "per_k": per_k,
        "gemv_multi": {"layers_per_launch": list(MULTI_G), "note": "aqmb_gemv_multi over the same layer "
                       "copies (one input per group); per-layer time and algorithmic GB/s", "per_G": multi},
        "roofline": roofline,
    }
    if not args.no_gemm:
        tg = per_launch_us[("gemm", 4, n_tok)]
        fl = 2.0 * n_tok * gspec.d_out * gspec.d_in
        achg = fl / (tg * 1e-6) / 1e12
        out["roofline_gemm"] = {"bound": "mfma", "kernel": "gemm_kernel (k=4)", "achieved": round(achg, 1),
                                "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s", "frac": round(achg / BF16_PEAK_TFLOPS, 4),
                                "traffic": None, "us_per_launch": round(tg, 2)}
        gemm_total_us = sum(per_launch_us[("gemm", k, n_tok)] for k in ks)
        out["gemm_TFLOPs"] = round(len(ks) * fl / (gemm_total_us * 1e-6) / 1e12, 1)
    td = per_launch_us[("distortion", M, n_cal)]
    fld = 2.0 * (M + 1) * d_out * d_in * n_cal
    achd = fld / (td * 1e-6) / 1e12
    out["roofline_distortion"] = {"bound": "mfma", "kernel": f"distortion_kernel<M={M}> + distortion_reduce_kernel",
                                  "achieved": round(achd, 1), "peak": F16_PEAK_TFLOPS, "unit": "TFLOP/s",
                                  "frac": round(achd / F16_PEAK_TFLOPS, 4), "traffic": None,
                                  "us_per_launch": round(td, 2),
                                  "workload": f"D^(1..{M}) of a {d_out}x{d_in} layer, dense fp16 W, "
                                              f"{n_cal} fp16 calibration inputs"}
    tb = per_launch_us[("beam", BEAM_K, BEAM_WIDTH)]
    cands = d_out * G_groups * 256 * (1 + (BEAM_K - 1) * BEAM_WIDTH)
    achb = cands * 23 / (tb * 1e-6) / 1e12
    out["roofline_beam"] = {"bound": "alu", "kernel": f"beam_kernel<{BEAM_WIDTH}> (k={BEAM_K})", "achieved": round(achb, 2),
                            "peak": round(FP32_PLAIN_PEAK_TOPS, 2), "unit": "TFLOP/s",
                            "frac": round(achb / FP32_PLAIN_PEAK_TOPS, 4), "traffic": None,
                            "us_per_launch": round(tb, 1), "candidates_per_s": round(cands / (tb * 1e-6), 1),
                            "workload": f"codes for the {d_out * G_groups} groups of a {d_out}x{d_in} fp16 W, "
                                        f"k={BEAM_K} codebooks of 256, beam {BEAM_WIDTH}"}
    def gemv4_bytes(k):
        return k * (d_out * d_in // 16) + k * 16 * 8 * 2 + 2 * d_out + 2 * (d_in + d_out)
    out["gemv_4bit"] = {"note": "the same shape with 4-bit codes (M = 4 codebooks of 16 codewords), batch 1, "
                        "fp16 x/y; algorithmic bytes k*d_out*d_in/16 + codebooks + scales + x + y",
                        "per_k": {str(k): {"us": round(per_launch_us[("gemv4", k, 1)], 3),
                                           "GBps": round(gemv4_bytes(k) / (per_launch_us[("gemv4", k, 1)] * 1e-6) / 1e9, 1)}
                                  for k in ks}}
    step_us = {n: 0.0 for n in ("gemv", "gemv_multi", "gemv4", "dequant", "gemm", "distortion", "beam")}
    for i, (name, k, b, fn, n) in enumerate(ops):
        step_us["gemv_multi" if name.startswith("gemv_multi") else name] += per_op_ms[i] * 1e3 / args.steps
    tot = sum(step_us.values())
    out["time_share"] = {n: round(v / tot, 4) for n, v in step_us.items() if v > 0}

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(base, x1, x4, ks, gemv_bytes)
        dist_cpu, beam_cpu = cpu_oracle_widened(base, make_weights, make_activations, M, d_in)
        out["roofline_distortion"]["cpu_oracle"] = dist_cpu
        out["roofline_beam"]["cpu_oracle"] = beam_cpu

    for h in layers + layers4:
        A.destroy(h)
    if not args.no_gemm:
        for h in glayers:
            A.destroy(h)
    if not args.no_secondary:
        out["secondary"] = secondary_measurements(A, torch, stream, to_dev, args.no_gemm)
    print(json.dumps(out), flush=True)


def _time_burst(torch, stream, fn, reps=5):
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


def secondary_measurements(A, torch, stream, to_dev, no_gemm):
    """Measured once after the timed steps (not part of a step): the decode GEMV on the other
    layer shapes, each over enough resident copies to stream from HBM; the prefill GEMM with
    4-bit codes; and two labelled ceilings: the GEMV on one cache-resident layer (warm), and the
    platform BLAS bf16 GEMM of the prefill shape (dense bf16 weights; a reference point only)."""
    import dataclasses
    from workloads import config, make_layer, make_activations
    res = {}
    dt = {"f16": (torch.float16, A.DType.F16), "bf16": (torch.bfloat16, A.DType.BF16)}

    def gemv_bytes(spec, k, b):
        code_b = 2 if spec.B == 16 else 1
        return (k * spec.d_out * (spec.d_in // 8) * code_b + k * (1 << spec.B) * 16 + 2 * spec.d_out
                + 2 * b * (spec.d_in + spec.d_out))

    shapes = {}
    for name, copies in (("c1", 64), ("c3_up", 24), ("c3_down", 24), ("c4", 20)):
        spec = config(name)
        log(f"secondary: {spec.name}, {copies} copies")
        L = make_layer(spec)
        desc = A.make_desc(spec.d_out, spec.d_in, spec.M, spec.B)
        hs = [A.create(desc, to_dev(L.codes if r == 0 else np.ascontiguousarray(np.roll(L.codes, r * 61, axis=1))),
                       to_dev(L.codebooks), to_dev(L.scales)) for r in range(copies)]
        tdt, adt = dt[spec.act_dtype]
        e = {}
        for b in spec.batches:
            x = to_dev(make_activations(L, b)).view(tdt)
            ys = [torch.empty((b, spec.d_out), dtype=tdt, device="cuda") for _ in range(copies)]
            for k in spec.ks:
                us = _time_burst(torch, stream, lambda: [A.gemv(h, k, x, adt, b, y, adt) for h, y in zip(hs, ys)]) / copies
                gbps = gemv_bytes(spec, k, b) / (us * 1e-6) / 1e9
                e[f"k{k}_b{b}"] = {"us": round(us, 3), "GBps": round(gbps, 1), "frac_hbm": round(gbps / HBM_PEAK_GBPS, 4)}
        shapes[spec.name] = e
        for h in hs:
            A.destroy(h)
    res["gemv_other_shapes"] = {"note": "per launch, graph replay over resident copies; algorithmic bytes "
                                "k*plane + k*codebook + scales + x + y", "per_shape": shapes}

    # warm: one layer of the 4096 x 4096 workload, launched repeatedly (codes cache-resident)
    spec = config("c2")
    L = make_layer(spec)
    h = A.create(A.make_desc(4096, 4096, 4, 8), to_dev(L.codes), to_dev(L.codebooks), to_dev(L.scales))
    x = to_dev(make_activations(L, 1, "f16")).view(torch.float16)
    y = torch.empty((1, 4096), dtype=torch.float16, device="cuda")
    warm = {}
    for k in spec.ks:
        us = _time_burst(torch, stream, lambda: [A.gemv(h, k, x, A.DType.F16, 1, y, A.DType.F16) for _ in range(64)]) / 64
        warm[str(k)] = {"us": round(us, 3), "GBps": round(gemv_bytes(spec, k, 1) / (us * 1e-6) / 1e9, 1)}
    A.destroy(h)
    res["gemv_warm_cache_resident"] = {"note": "one 4096x4096 layer launched 64 times in a row, batch 1: its "
                                       "codes stay in the caches (not an HBM figure)", "per_k": warm}

    if not no_gemm:
        gspec = config("c5")
        n = gspec.n_tokens
        fl = 2.0 * n * gspec.d_out * gspec.d_in
        s4 = dataclasses.replace(gspec, B=4, seed=gspec.seed + 100)
        L4 = make_layer(s4)
        d4 = A.make_desc(s4.d_out, s4.d_in, s4.M, 4)
        hs = [A.create(d4, to_dev(L4.codes if r == 0 else np.ascontiguousarray(np.roll(L4.codes, r * 61, axis=1))),
                       to_dev(L4.codebooks), to_dev(L4.scales)) for r in range(4)]
        X = to_dev(make_activations(L4, n, "bf16")).view(torch.bfloat16)
        Ys = [torch.empty((n, s4.d_out), dtype=torch.bfloat16, device="cuda") for _ in range(4)]
        g4 = {}
        for k in s4.ks:
            us = _time_burst(torch, stream, lambda: [A.gemm(hh, k, X, n, Y, A.DType.BF16) for hh, Y in zip(hs, Ys)]) / 4
            g4[str(k)] = {"us": round(us, 2), "TFLOPs": round(fl / (us * 1e-6) / 1e12, 1)}
        for hh in hs:
            A.destroy(hh)
        res["gemm_4bit"] = {"note": f"{n}-token prefill GEMM on a {s4.d_out}x{s4.d_in} layer with 4 codebooks of 16 "
                            "codewords (4-bit codes), bf16 out", "per_k": g4}
        # platform BLAS on dense bf16 weights of the same shape: a reference point, not part of the path
        Wt = torch.randn((gspec.d_in, gspec.d_out), dtype=torch.float32, device="cuda").mul_(0.02).to(torch.bfloat16)
        Wts = [Wt.clone() for _ in range(4)]
        Yb = torch.empty((n, gspec.d_out), dtype=torch.bfloat16, device="cuda")
        note = ("torch.matmul of the same shape on dense bf16 weights (the platform BLAS); a measurement "
                "reference, not part of the path")
        # eager launches (the BLAS is not captured in a graph); the first call warms it up
        for w in Wts:
            torch.matmul(X, w, out=Yb)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(5):
            for w in Wts:
                torch.matmul(X, w, out=Yb)
        e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / 20
        res["gemm_platform_blas_bf16"] = {"note": note, "us": round(us, 2), "TFLOPs": round(fl / (us * 1e-6) / 1e12, 1)}
    return res


def cpu_baseline(layer, x1bits, x4bits, ks, gemv_bytes):
    """The fp64 oracle on the host cores: reconstruct W_k and multiply, for batch 1 and 4 at every k,
    repeated until about 10 s have passed; reported in the GEMV's algorithmic GB/s."""
    import oracle
    from oracle import formats
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        blas_threads = 1
    C = formats.f16_bits_to_f64(layer.codebooks)
    s = formats.f16_bits_to_f64(layer.scales)
    x1 = formats.f16_bits_to_f64(x1bits)
    x4 = formats.f16_bits_to_f64(x4bits)
    total_bytes, t_total, passes = 0, 0.0, 0
    t_start = time.perf_counter()
    while True:
        for k in ks:
            t0 = time.perf_counter()
            oracle.linear(x1, layer.codes, C, s, k)
            oracle.linear(x4, layer.codes, C, s, k)
            t_total += time.perf_counter() - t0
            total_bytes += gemv_bytes(k, 1) + gemv_bytes(k, 4)
        passes += 1
        if time.perf_counter() - t_start > 10.0:
            break
    return {"value": round(total_bytes / t_total / 1e9, 4), "unit": "GB/s", "cores": int(blas_threads),
            "kind": "oracle",
            "sample": f"{passes} pass(es) of: reconstruct W_k in fp64 and multiply, batch 1 and 4, k=1..4, "
                      f"one {layer.spec.d_out}x{layer.spec.d_in} layer (gather single-threaded, product on BLAS)",
            "seconds": round(t_total, 2), "host_cpus": len(os.sched_getaffinity(0))}


def cpu_oracle_widened(layer, make_weights, make_activations, M, d_in):
    """The oracle beside the distortion evaluator and the beam search, on bounded samples of the
    same workloads (a few seconds each): the fp64 prefix distortions of the first 2048 rows over 1024
    calibration inputs (in TFLOP/s of the same 2 (M + 1) d_out d_in n count), and the binary32
    beam search of 64 groups (in candidates/s)."""
    import oracle
    from oracle import formats
    from workloads import LayerSpec, make_layer
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        blas_threads = 1
    rows, n = 2048, 1024
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
    return dist, beam


if __name__ == "__main__":
    main()
