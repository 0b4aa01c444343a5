#!/usr/bin/env python
"""Benchmark of the HyQuant hybrid-precision prefill path on one MI355X.

A step is one pass of the whole hot path over one synthetic layer:
hyq_select_vertical -> hyq_quantize -> hyq_attn_prefill, with Q/K/V already
resident in HBM.  Default workload: GQA 32 query / 8 KV heads, head dim 128,
32768 tokens, window 256, vertical budget 1%, 8-bit K/V, float32 output (the
launch configuration the parity tests check at full size).

The ``decode`` sub-record times the decode path (Algorithm 3 over the
cache Freeze builds) on the paper's decode-latency workload: batch 1, 32
query / 8 KV heads, 32k-token prefix, K4V4, top-5% vertical lines, window
128.  It measures one attention call per layer over 36 layer caches
(about 1.4 GB, so that the last-level cache cannot serve repeated reads),
against its roofline, HBM bandwidth.  A second line uses batch 16.  The
same kernel with every prefix token kept in bf16 is the in-house
full-precision comparison.

Prints one JSON line.  ``value`` is the algorithmic causal attention FLOPs
(4 * D * Hq * B * L(L+1)/2) per second of the whole step, in TFLOP/s;
``roofline`` describes the attention kernel alone (timed with HIP events on
the stream it runs on); ``cpu_baseline`` is the CPU oracle on a bounded
sample of the same layer.
"""
from __future__ import annotations

import argparse
import dataclasses
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

INT8_PEAK_TOPS = 5000.0        # MI355X dense int8 MFMA, TOP/s
F16_PEAK_TFLOPS = 2500.0       # MI355X dense f16/bf16 MFMA, TFLOP/s
FP4_PEAK_TFLOPS = 10100.0      # MI355X dense fp4/fp6 MFMA, TFLOP/s
BLENDED_PEAK = 1.0 / (0.5 / INT8_PEAK_TOPS + 0.5 / F16_PEAK_TFLOPS)   # int8 QK^T + f16 PV
HBM_PEAK_GBS = 8000.0


def causal_flops(B, Hq, L, D):
    return 4.0 * D * Hq * B * L * (L + 1) / 2.0


def src_digest(*names):
    """sha256 prefix of kernel sources (and the device headers they include)."""
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2608_27875_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def attn_src_digest():
    return src_digest("attn_prefill.hip", "codes_dev.h", "hyq_internal.h")


def decode_src_digest():
    return src_digest("decode.hip", "decode_split.h", "codes_dev.h", "quant_dev.h",
                      "hyq_internal.h")


def load_traffic(workload, fname="attn_traffic.json", digest=None):
    """HBM bytes per kernel launch from rocprofv3 FETCH_SIZE / WRITE_SIZE
    counters (profiles/<fname>), only if taken on this kernel source."""
    p = os.path.join(ROOT, "profiles", fname)
    if not os.path.exists(p):
        return None
    try:
        rec = json.load(open(p))
    except ValueError:
        return None
    if rec.get("kernel_src_sha") != (digest or attn_src_digest)() or \
            rec.get("workload") != workload:
        return None
    return rec.get("hbm_bytes_per_launch")


def host_identity():
    """The host the CPU baseline ran on: CPUs this process may use, the
    machine's CPU count and the CPU model string."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        affinity = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        affinity = None
    return {"affinity_cpus": affinity, "os_cpu_count": os.cpu_count(), "cpu_model": model}


def cpu_baseline(d, cfg, flops_total, budget_s):
    """The oracle (untuned) on a bounded sample: full selection and
    quantization of the layer, attention for a few heads x rows; the
    whole-layer time is extrapolated from the attention FLOPs of the sample."""
    import numpy as np
    from oracle import hyq_oracle as orc
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        blas_threads = None
    L, W, D, Hq = cfg["L"], cfg["W"], 128, cfg["Hq"]
    t0 = time.perf_counter()
    idx, _ = orc.select_vertical(d["Q"], d["K"], cfg["Hkv"], W, cfg["budget_ppm"])
    t_sel = time.perf_counter() - t0
    t0 = time.perf_counter()
    qz = orc.quantize(d["Q"], d["K"], d["V"], idx, W, cfg["bits"],
                      fmt=cfg.get("fmt_name", "int") if cfg["bits"] != 16 else "int")
    t_quant = time.perf_counter() - t0
    heads = [(0, h) for h in range(0, Hq, max(1, Hq // 4))][:4]
    rng = np.random.default_rng(0)
    n_rows = 64
    t_attn, f_attn = 0.0, 0.0
    while True:
        rows = np.sort(rng.choice(L, size=n_rows, replace=False))
        t0 = time.perf_counter()
        orc.attention(d["Q"], d["K"], d["V"], W, cfg["bits"], idx, qz, heads=heads, rows=rows)
        dt = time.perf_counter() - t0
        t_attn += dt
        f_attn += len(heads) * float(np.sum(4.0 * D * (rows + 1)))
        if t_attn + t_sel + t_quant > budget_s or n_rows >= 4096:
            break
        n_rows *= 2
    est = t_sel + t_quant + t_attn * (flops_total / f_attn)
    host = host_identity()
    # the oracle's attention is numpy matrix products (the BLAS thread pool);
    # its selection and quantization run on one thread
    cores = blas_threads or host["affinity_cpus"] or 1
    return {
        "value": flops_total / est / 1e12, "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
        "blas_threads": blas_threads, "host": host,
        "sample": (f"full selection ({t_sel:.2f} s) and quantization ({t_quant:.2f} s) of the layer; "
                   f"attention for {len(heads)} heads x {n_rows}-row random row sets "
                   f"({t_attn:.2f} s for {f_attn:.3e} FLOP); whole-layer time extrapolated "
                   f"to {est:.1f} s"),
    }


def decode_bytes(c, B):
    """Algorithmic HBM bytes of one decode attention call: every valid cache
    entry once (codes, scales, bf16 rows), the query and the output."""
    Hkv, D = c.Hkv, c.D
    nbq = -(-c.n_frozen // 64) + c.n_merged
    nq = c.n_frozen + 64 * c.n_merged
    row = D if c.bits_kv == 8 else D // 2
    per_head = 2 * nq * row + 2 * nbq * 4 + (c.n_vl + c.window + c.n_staged) * D * 2 * 2
    return B * Hkv * per_head + B * c.Hq * D * (2 + 4)


def decode_record(B, layers, steps, budget_ppm=50000, bits=4, N=32768, W=128, Hq=32, Hkv=8,
                  seed=0, label=None, probe=False, fmt=0, staging=128):
    """Freeze `layers` synthetic layers, then time hyq_decode_attn over all of
    them (one decode token of a `layers`-layer model)."""
    import numpy as np
    import torch

    import paper_2608_27875_amd as hyq
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    shape = hyq.Shape(B=B, Hq=Hq, Hkv=Hkv, L=N, window=W, budget_ppm=budget_ppm, bits_kv=bits,
                      kv_format=fmt, staging=staging)
    gen_ = torch.Generator(device=dev)
    gen_.manual_seed(seed)
    caches, qs, outs = [], [], []
    print(f"[bench] decode: freezing {layers} layers of {shape}", file=sys.stderr, flush=True)
    for _ in range(layers):
        Q = torch.randn((B, Hq, N, 128), generator=gen_, device=dev).to(torch.bfloat16)
        K = torch.randn((B, Hkv, N, 128), generator=gen_, device=dev).to(torch.bfloat16)
        V = torch.randn((B, Hkv, N, 128), generator=gen_, device=dev).to(torch.bfloat16)
        c = hyq.DecodeCache(shape, N + 64, dev)
        hyq.hyq_freeze(shape, Q, K, V, c, stream)
        del Q, K, V
        caches.append(c)
        qs.append(torch.randn((B, Hq, 128), generator=gen_, device=dev).to(torch.bfloat16))
        outs.append(torch.empty((B, Hq, 128), dtype=torch.float32, device=dev))
    torch.cuda.synchronize()

    def one_token():
        for c, q, o in zip(caches, qs, outs):
            hyq.hyq_decode_attn(c, q, o)   # on the current stream (the capture stream below)

    if probe:   # for rocprofv3 --pmc: one token, the 1 GiB copy kernel, one more token
        one_token()
        n = 1 << 28
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        one_token()
        torch.cuda.synchronize()
        print(f"[bench] decode traffic probe done: {layers} layers x 2 tokens; copy kernel reads "
              f"and writes {4 * n} bytes", file=sys.stderr, flush=True)
        return None

    def timed(run):
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(steps)]
        s = torch.cuda.current_stream()
        for e in ev:
            e[0].record(s)
            run()
            e[1].record(s)
        torch.cuda.synchronize()
        return float(np.median([e[0].elapsed_time(e[1]) for e in ev]))

    for _ in range(3):
        one_token()
    torch.cuda.synchronize()
    ref = [o.clone() for o in outs]
    ms_eager = timed(one_token)
    # the same launches replayed as one HIP graph (no host work between
    # kernels); every replay must reproduce the eager outputs bit for bit
    graph_ok, ms = False, ms_eager
    try:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            one_token()
        torch.cuda.synchronize()
        graph_ok = True
        for _ in range(3):
            for o in outs:
                o.zero_()
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            graph_ok &= all(torch.equal(o, r) for o, r in zip(outs, ref))
        if graph_ok:
            ms = timed(g.replay)
        del g
    except RuntimeError as e:
        print(f"[bench] decode graph capture failed: {e}", file=sys.stderr, flush=True)
    us_layer = ms * 1e3 / layers
    nbytes = decode_bytes(caches[0].c, B)
    gbs = nbytes / (us_layer * 1e-6) / 1e9
    workload = label or (f"decode_gqa{Hq}q{Hkv}kv_d128_B{B}_N{N}_W{W}_Ws{staging}_r{budget_ppm}ppm"
                         f"_kv{bits}bit" + ("_fp4" if fmt == hyq.FMT_FP4 else ""))
    rec = {"workload": workload,
           "layers": layers, "us_per_layer": round(us_layer, 3),
           "timing": "hip graph of the layer loop" if graph_ok else "eager launches",
           "us_per_layer_eager": round(ms_eager * 1e3 / layers, 3),
           "ms_per_token_all_layers": round(ms, 4),
           "bytes_per_layer": int(nbytes),
           "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
                        "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                        "traffic": load_traffic(workload, "decode_traffic.json", decode_src_digest),
                        "kernel": "decode_attn_kernel + decode_combine_kernel"}}
    del caches, qs, outs
    torch.cuda.empty_cache()
    return rec


def decode_section(layers, steps):
    """The decode measurements: K4V4 hybrid at batch 1 and 16, the same with
    FP4 (E2M1) codes at batch 1, and the all-bf16 comparison (every prefix
    token a vertical line) at batch 1."""
    r1 = decode_record(1, layers, steps)
    bf = decode_record(1, layers, steps, budget_ppm=1000000, bits=8,
                       label="decode_gqa32q8kv_d128_B1_N32768_all_bf16")
    r1["bf16_same_length"] = {"us_per_layer": bf["us_per_layer"],
                              "bytes_per_layer": bf["bytes_per_layer"],
                              "achieved_gbs": bf["roofline"]["achieved"],
                              "speedup_of_hybrid": round(bf["us_per_layer"] / r1["us_per_layer"], 3)}
    import paper_2608_27875_amd as hyq
    f4 = decode_record(1, layers, steps, fmt=hyq.FMT_FP4)
    r1["fp4_same_length"] = {k: f4[k] for k in ("workload", "us_per_layer", "bytes_per_layer")}
    r1["fp4_same_length"]["achieved_gbs"] = f4["roofline"]["achieved"]
    r16 = decode_record(16, max(2, layers // 9), steps)
    r1["batch16"] = {k: r16[k] for k in ("workload", "layers", "us_per_layer", "bytes_per_layer",
                                         "roofline")}
    return r1


def main():
    from paper_2608_27875_amd import gen   # the named workloads (numpy only)

    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=gen.GQA_32K, choices=sorted(gen.WORKLOADS),
                    help="named synthetic workload (default: the 32k GQA prefill)")
    ap.add_argument("--bits", type=int, default=None, help="override K/V bit-width (16, 8, 4)")
    ap.add_argument("--budget-ppm", type=int, default=None)
    ap.add_argument("--out-bf16", action="store_true")
    ap.add_argument("--cpu-budget-s", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--hq", type=int, default=None,
                    help="keep only the first HQ query heads (with their KV heads): e.g. --hq 4 "
                         "is one GPU's share of the 32k workload under 8-way head sharding")
    ap.add_argument("--no-bits16", action="store_true",
                    help="skip the full-precision (bits 16) attention of the same inputs")
    ap.add_argument("--fmt", choices=("int", "fp8", "fp4", "fp4q6"), default="int",
                    help="code format of the quantized path (fp8 = OCP E4M3, 8-bit only; "
                         "fp4 = OCP E2M1 K/V with E4M3 queries, fp4q6 the same with FP6 E2M3 "
                         "queries; both set bits 4)")
    ap.add_argument("--no-fp8", action="store_true",
                    help="skip the FP8-code run of the same inputs")
    ap.add_argument("--no-decode", action="store_true", help="skip the decode measurement")
    ap.add_argument("--no-band", action="store_true",
                    help="skip the per-query window (band) attention on the same inputs")
    ap.add_argument("--no-colmass", action="store_true",
                    help="skip the exact column-mass selector on the same inputs")
    ap.add_argument("--decode-only", action="store_true",
                    help="only the decode measurement (printed as its own JSON line)")
    ap.add_argument("--decode-layers", type=int, default=36)
    ap.add_argument("--traffic-probe", action="store_true",
                    help="for rocprofv3 --pmc runs: one step, a plain 1 GiB copy kernel of known "
                         "traffic (the counter scale), one more step; no timing")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: the operator is single-GPU (heads shard with no "
              "communication, see the design notes); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2608_27875_amd as hyq

    if args.decode_only:
        if args.traffic_probe:
            decode_record(1, args.decode_layers, 1, probe=True)
            return
        print(json.dumps({"decode": decode_section(args.decode_layers, args.steps)}), flush=True)
        return

    cfg = gen.workload(args.workload)
    if args.bits is not None:
        cfg["bits"] = args.bits
    if args.budget_ppm is not None:
        cfg["budget_ppm"] = args.budget_ppm
    print(f"[bench] generating workload {args.workload}: {cfg}", file=sys.stderr, flush=True)
    d = gen.generate_workload(args.workload, seed=args.seed)
    dev = torch.device("cuda:0")

    def t(x):
        return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to(dev)

    if args.hq is not None:
        g = cfg["Hq"] // cfg["Hkv"]
        if args.hq % g or not 0 < args.hq <= cfg["Hq"]:
            print(f"--hq must be a multiple of the group size {g} and at most {cfg['Hq']}",
                  file=sys.stderr)
            sys.exit(2)
        hkv = args.hq // g
        d["Q"], d["K"], d["V"] = d["Q"][:, :args.hq], d["K"][:, :hkv], d["V"][:, :hkv]
        d["planted"] = [d["planted"][b * cfg["Hkv"] + j] for b in range(cfg["B"])
                        for j in range(hkv)]
        cfg["Hq"], cfg["Hkv"] = args.hq, hkv
    Q, K, V = t(np.ascontiguousarray(d["Q"])), t(np.ascontiguousarray(d["K"])), \
        t(np.ascontiguousarray(d["V"]))
    fmt = {"fp8": hyq.FMT_FP8, "fp4": hyq.FMT_FP4, "fp4q6": hyq.FMT_FP4Q6}.get(args.fmt,
                                                                              hyq.FMT_INT)
    if fmt in (hyq.FMT_FP4, hyq.FMT_FP4Q6):
        cfg["bits"] = 4
    cfg["fmt_name"] = args.fmt
    shape = hyq.Shape(B=cfg["B"], Hq=cfg["Hq"], Hkv=cfg["Hkv"], L=cfg["L"], window=cfg["W"],
                      budget_ppm=cfg["budget_ppm"], bits_kv=cfg["bits"], kv_format=fmt)
    out_dtype = 1 if args.out_bf16 else 0
    bufs = hyq.alloc_buffers(shape, dev, out_dtype)
    z = bufs["sizes"]
    scale = 1.0 / math.sqrt(shape.D)
    stream = torch.cuda.current_stream()

    def step(ev=None):
        if ev:
            ev[0].record(stream)
        hyq.hyq_select_vertical(shape, Q, K, bufs["idx"], None, bufs["ws"], stream)
        if ev:
            ev[1].record(stream)
        hyq.hyq_quantize(shape, Q, K, V, bufs["idx"], bufs["q_codes"], bufs["q_scale"],
                         bufs["k_codes"], bufs["k_scale"], bufs["v_codes"], bufs["v_scale"],
                         bufs["kq_pos"], stream)
        if ev:
            ev[2].record(stream)
        hyq.hyq_attn_prefill(shape, Q, K, V, bufs["idx"], bufs["q_codes"], bufs["q_scale"],
                             bufs["k_codes"], bufs["k_scale"], bufs["v_codes"], bufs["v_scale"],
                             bufs["kq_pos"], scale, bufs["out"], out_dtype, stream)
        if ev:
            ev[3].record(stream)

    if args.traffic_probe:
        step()
        n = 1 << 28   # float32 elements: 1 GiB read + 1 GiB written
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.neg(src, out=dst)
        torch.cuda.synchronize()
        step()
        torch.cuda.synchronize()
        print(f"[bench] traffic probe done: copy kernel reads and writes {4 * n} bytes",
              file=sys.stderr, flush=True)
        return

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps
    # per-phase HIP-event times of the timed steps, reduced here once
    phase_ms = {name: [e[a].elapsed_time(e[a + 1]) for e in evs]
                for a, name in enumerate(("select", "quantize", "attention"))}
    phase_mean = {k: float(np.mean(v)) for k, v in phase_ms.items()}
    phase_median = {k: float(np.median(v)) for k, v in phase_ms.items()}
    attn_ms = phase_mean["attention"]

    def median_ms(run, reps, pre=None, warm=1):
        """Median over `reps` launches of run(), timed with HIP events on the
        library's stream; pre() (untimed, e.g. the quantization feeding an
        attention launch) runs before each."""
        for _ in range(warm):
            if pre:
                pre()
            run()
        torch.cuda.synchronize()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(reps)]
        for e in ev:
            if pre:
                pre()
            e[0].record(stream)
            run()
            e[1].record(stream)
        torch.cuda.synchronize()
        return float(np.median([e0.elapsed_time(e1) for e0, e1 in ev]))

    def attn_call(sx, bx):
        return lambda: hyq.hyq_attn_prefill(sx, Q, K, V, bx["idx"], bx["q_codes"], bx["q_scale"],
                                            bx["k_codes"], bx["k_scale"], bx["v_codes"],
                                            bx["v_scale"], bx["kq_pos"], scale, bx["out"],
                                            out_dtype, stream)

    # the same inputs through our own kernel with every key in full precision
    # (bits 16): the in-house exact-attention comparison
    bits16 = None
    if not args.no_bits16 and shape.bits_kv != 16:
        s16 = hyq.Shape(B=shape.B, Hq=shape.Hq, Hkv=shape.Hkv, L=shape.L, window=shape.window,
                        budget_ppm=shape.budget_ppm, bits_kv=16)
        b16 = hyq.alloc_buffers(s16, dev, out_dtype)
        print("[bench] bits-16 attention", file=sys.stderr, flush=True)

        ms16 = median_ms(attn_call(s16, b16), 5)
        bits16 = {"attention_ms_median": round(ms16, 4),
                  "tflops": round(causal_flops(shape.B, shape.Hq, shape.L, shape.D) /
                                  (ms16 * 1e-3) / 1e12, 2),
                  "speedup_of_hybrid": round(ms16 / phase_median["attention"], 3)}
        del b16

    def quant_attn_ms(sx, reps=10):
        """Median attention time for another bit-width / format on the same
        inputs and selection (each launch after its own quantization)."""
        bx = hyq.alloc_buffers(sx, dev, out_dtype)
        hyq.hyq_select_vertical(sx, Q, K, bx["idx"], None, bx["ws"], stream)

        def quant():
            hyq.hyq_quantize(sx, Q, K, V, bx["idx"], bx["q_codes"], bx["q_scale"],
                             bx["k_codes"], bx["k_scale"], bx["v_codes"], bx["v_scale"],
                             bx["kq_pos"], stream)
        ms = median_ms(attn_call(sx, bx), reps, pre=quant, warm=2)
        del bx
        return ms

    # the same inputs with 4-bit K/V codes: int4 (int8 queries, int8 MFMA)
    # and FP4 E2M1 (E4M3 queries, E2M1 keys as the scaled MFMA's 4-bit operand)
    four_bit = None
    if not args.no_fp8 and shape.bits_kv == 8 and fmt == hyq.FMT_INT:
        print("[bench] 4-bit codes (int4, fp4)", file=sys.stderr, flush=True)
        fl = causal_flops(shape.B, shape.Hq, shape.L, shape.D)
        four_bit = {}
        for name, fx in (("int4", hyq.FMT_INT), ("fp4", hyq.FMT_FP4), ("fp4q6", hyq.FMT_FP4Q6)):
            msx = quant_attn_ms(dataclasses.replace(shape, bits_kv=4, kv_format=fx))
            tfx = fl / (msx * 1e-3) / 1e12
            four_bit[name] = {"attention_ms_median": round(msx, 4), "tflops": round(tfx, 2),
                              "frac_int8_fp8_peak": round(tfx / INT8_PEAK_TOPS, 4)}
            if fx == hyq.FMT_FP4Q6:
                # E2M1 keys x E2M3 queries: the Q.K MFMA runs at the 4/6-bit rate
                four_bit[name]["frac_fp4_fp6_peak"] = round(tfx / FP4_PEAK_TFLOPS, 4)
                four_bit[name]["note"] = ("Q.K on the 4/6-bit MFMA rate; P.V stays f16 (2.5 PF), "
                                          "so the whole kernel cannot approach the 4-bit peak")

    # the same inputs with FP8 (E4M3) codes: quantize + attention
    fp8 = None
    if not args.no_fp8 and shape.bits_kv == 8 and fmt == hyq.FMT_INT:
        print("[bench] fp8 codes", file=sys.stderr, flush=True)
        ms8 = quant_attn_ms(dataclasses.replace(shape, kv_format=hyq.FMT_FP8))
        tf8 = causal_flops(shape.B, shape.Hq, shape.L, shape.D) / (ms8 * 1e-3) / 1e12
        fp8 = {"attention_ms_median": round(ms8, 4), "tflops": round(tf8, 2),
               "frac_fp8_peak": round(tf8 / INT8_PEAK_TOPS, 4)}

    # the same inputs and codes with the per-query window of eq. (win_def):
    # attention only (selection and quantization are the same)
    band = None
    if not args.no_band and shape.bits_kv != 16:
        sb = dataclasses.replace(shape, window_mode=hyq.WIN_BAND)
        print("[bench] per-query window (band) attention", file=sys.stderr, flush=True)

        msb = median_ms(attn_call(sb, bufs), 10)
        tfb = causal_flops(shape.B, shape.Hq, shape.L, shape.D) / (msb * 1e-3) / 1e12
        band = {"attention_ms_median": round(msb, 4), "tflops": round(tfb, 2),
                "frac_int8_peak": round(tfb / INT8_PEAK_TOPS, 4)}

    # the same inputs through the exact column-mass selector of eq. (vl_score):
    # selection only (its top-k feeds the same quantize and attention)
    colmass = None
    if not args.no_colmass and z["k"]:
        sc = dataclasses.replace(shape, selector=hyq.SEL_COLMASS)
        bc = hyq.alloc_buffers(sc, dev, out_dtype)
        print("[bench] column-mass selector", file=sys.stderr, flush=True)

        msc = median_ms(lambda: hyq.hyq_select_vertical(sc, Q, K, bc["idx"], None, bc["ws"],
                                                        stream), 10)
        # two QK^T passes over the tail rows: every causal key, then the prefix
        tr = min(shape.window, shape.L)
        rows = shape.B * shape.Hq * tr
        cflops = 2.0 * shape.D * rows * ((shape.L - tr) + (tr + 1) / 2.0 + z["P"])
        cidx = bc["idx"].cpu().numpy().reshape(-1, z["k"])
        pidx = bufs["idx"].cpu().numpy().reshape(-1, z["k"])
        crec, agree = [], []
        for bj in range(shape.B * shape.Hkv):
            pp = [p for p in d["planted"][bj].tolist() if p < z["P"]]
            if pp:
                crec.append(len(set(pp) & set(cidx[bj].tolist())) / min(len(pp), z["k"]))
            agree.append(len(set(pidx[bj].tolist()) & set(cidx[bj].tolist())) / z["k"])
        colmass = {"select_ms_median": round(msc, 4), "tflops": round(cflops / (msc * 1e-3) / 1e12, 2),
                   "frac_bf16_peak": round(cflops / (msc * 1e-3) / 1e12 / F16_PEAK_TFLOPS, 4),
                   "planted_recall": round(float(np.mean(crec)), 4) if crec else None,
                   "overlap_with_tail_proxy": round(float(np.mean(agree)), 4)}
        del bc

    # how well each selector finds vertical lines that the attention itself
    # makes (gen.shared_direction: a query direction shared by every query of
    # a KV group, planted keys along it), at the same shape and budget
    shared = None
    if not args.no_colmass and z["k"]:
        print("[bench] selector recall on shared-direction inputs", file=sys.stderr, flush=True)
        ds = gen.shared_direction(0, B=shape.B, Hq=shape.Hq, Hkv=shape.Hkv, L=shape.L,
                                  D=shape.D, W=shape.window, plant=cfg["plant"])
        Qs, Ks = t(ds["Q"]), t(ds["K"])
        shared = {"alpha": 7.0, "beta": 4.0}
        for name, selector in (("tail_proxy", hyq.SEL_PROXY), ("column_mass", hyq.SEL_COLMASS)):
            sx = dataclasses.replace(shape, selector=selector)
            bx = hyq.alloc_buffers(sx, dev, out_dtype)
            hyq.hyq_select_vertical(sx, Qs, Ks, bx["idx"], None, bx["ws"], stream)
            got = bx["idx"].cpu().numpy().reshape(-1, z["k"])
            rr = []
            for bj in range(shape.B * shape.Hkv):
                pp = [p for p in ds["planted"][bj].tolist() if p < z["P"]]
                if pp:
                    rr.append(len(set(pp) & set(got[bj].tolist())) / min(len(pp), z["k"]))
            shared[name + "_recall"] = round(float(np.mean(rr)), 4) if rr else None
            del bx
        del Qs, Ks, ds

    flops = causal_flops(shape.B, shape.Hq, shape.L, shape.D)
    value = flops / (ms_step * 1e-3) / 1e12
    attn_tflops = flops / (attn_ms * 1e-3) / 1e12
    # algorithmic bytes of the select and quantize kernels (one read of each
    # input row they need, one write of each output)
    sel_bytes = (shape.B * shape.Hq * min(shape.window, shape.L) * 256 +
                 shape.B * shape.Hkv * z["P"] * 256 + z["idx_bytes"]) if z["k"] else 0
    q_bytes = 0
    if shape.bits_kv != 16:
        q_bytes = (shape.B * shape.Hq * shape.L * 256 + 2 * shape.B * shape.Hkv * z["nQ"] * 256 +
                   z["q_codes_bytes"] + z["k_codes_bytes"] + z["v_codes_bytes"] +
                   z["q_scale_bytes"] + 2 * z["kv_scale_bytes"] + z["kq_pos_bytes"] + z["idx_bytes"])
    workload = (f"gqa{shape.Hq}q{shape.Hkv}kv_d{shape.D}_B{shape.B}_L{shape.L}_W{shape.window}"
                f"_r{shape.budget_ppm}ppm_kv{shape.bits_kv}bit" +
                {hyq.FMT_FP8: "_fp8", hyq.FMT_FP4: "_fp4", hyq.FMT_FP4Q6: "_fp4q6"}.get(fmt, ""))
    traffic = load_traffic(workload)
    planted = d["planted"]
    idx = bufs["idx"].cpu().numpy()
    recall = []
    for bj in range(shape.B * shape.Hkv):
        pp = [p for p in planted[bj].tolist() if p < z["P"]]
        if pp and z["k"]:
            recall.append(len(set(pp) & set(idx.reshape(-1, z["k"])[bj].tolist())) /
                          min(len(pp), z["k"]))
    rec = {
        "metric": "hybrid prefill attention TFLOP/s + % MFMA peak (GQA 32q/8kv, d128, 32k)",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": ("bf16" if shape.bits_kv == 16 else
                  "e4m3+f16" if fmt == hyq.FMT_FP8 else
                  "e2m1xe4m3+f16" if fmt == hyq.FMT_FP4 else
                  "e2m1xe2m3+f16" if fmt == hyq.FMT_FP4Q6 else "i8+f16"),
        "data": "synthetic (seeded Gaussian Q/K/V, planted vertical lines, x10 outlier K channels)",
        "config": {"workload": workload, "B": shape.B, "Hq": shape.Hq, "Hkv": shape.Hkv,
                   "L": shape.L, "D": shape.D, "window": shape.window,
                   "budget_ppm": shape.budget_ppm, "bits_kv": shape.bits_kv,
                   "out": "bf16" if out_dtype else "f32", "k": z["k"], "parallelism": "none"},
        "roofline": {"bound": "mfma", "achieved": round(attn_tflops, 2), "peak": INT8_PEAK_TOPS,
                     "unit": "TFLOP/s", "frac": round(attn_tflops / INT8_PEAK_TOPS, 4),
                     "traffic": traffic, "kernel": "attn_prefill_kernel"},
        "ms_per_layer": {"total": round(ms_step, 4), "attention": round(attn_ms, 4),
                         "select": round(phase_mean["select"], 4),
                         "quantize": round(phase_mean["quantize"], 4)},
        "ms_median": {"attention": round(phase_median["attention"], 4),
                      "select": round(phase_median["select"], 4),
                      "quantize": round(phase_median["quantize"], 4)},
        "bits16_same_inputs": bits16,
        "fp8_same_inputs": fp8,
        "four_bit_same_inputs": four_bit,
        "band_window_same_inputs": band,
        "colmass_selector_same_inputs": colmass,
        "selector_recall_shared_direction": shared,
        "attention_tflops": round(attn_tflops, 2),
        "frac_int8_peak": round(attn_tflops / INT8_PEAK_TOPS, 4),
        "frac_blended_ceiling": round(attn_tflops / BLENDED_PEAK, 4),
        "select_gbs": round(sel_bytes / (phase_mean["select"] * 1e-3) / 1e9, 1) if sel_bytes else None,
        "quantize_gbs": round(q_bytes / (phase_mean["quantize"] * 1e-3) / 1e9, 1) if q_bytes else None,
        "planted_recall": round(float(np.mean(recall)), 4) if recall else None,
    }
    rec["decode"] = None if args.no_decode else decode_section(args.decode_layers,
                                                                 min(args.steps, 20))
    if not args.no_cpu_baseline:
        print(f"[bench] cpu baseline (oracle, ~{args.cpu_budget_s:.0f} s)", file=sys.stderr,
              flush=True)
        rec["cpu_baseline"] = cpu_baseline(d, cfg, flops, args.cpu_budget_s)
    else:
        rec["cpu_baseline"] = None
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
