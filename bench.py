"""Benchmark of the SDQ decomposed linear layer on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--gpus 1]

A step is one pass of the hot path over one batch of synthetic input: for
every layer of the workload, per-token activation quantization
(sdq_quantize_act) followed by the decomposed GEMM (sdq_gemm).  The weights
were packed offline (sdq_pack, host); the packer's time is reported beside
the line, never inside the step.  Every input is resident in HBM when the
timed region starts: distinct copies of the packed weights, activations and
outputs (>= 512 MB, twice the 256 MB Infinity Cache) are rotated, and a
512 MB fill runs between the untimed and the timed graph replay, so that each
timed launch streams its weights from HBM whatever the step count.

The default workload is the LLaMA-7B MLP prefill (gate, up and down
projections at 2048 tokens, MX 1:8 e4m3 + 2:8 e2m1); the same line carries the
LLaMA-7B attention-projection decode (one token, INT 1:8 e4m3 + 3:8 int4)
under "decode", with its own HBM roofline.

Prints one JSON line: dense-equivalent TFLOP/s of the step (2*M*N*K per layer),
the roofline object of the dominant kernel (the GEMM) measured with HIP events
on the launch stream, and the CPU oracle timed on this host.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import synth  # noqa: E402

HBM_PEAK_GBS = 8000.0
FLUSH_BYTES = 512 * 1024 * 1024  # twice the Infinity Cache

WORKLOADS = {
    # name: (workload id, layer indices, M)
    "llama7b-attn-decode": (2, [0], 1),
    # q, k and v stacked along N, one launch (N = 12288)
    "llama7b-qkv-decode": (7, [0], 1),
    # gate and up stacked along N, one launch (N = 22016)
    "llama7b-gateup-decode": (8, [0], 1),
    "llama7b-mlp-prefill": (3, [0, 1, 2], 2048),
    "opt6.7b-ffn-decode": (4, [0, 1], 64),
    "tiny": (1, [0], 16),
    # the paper's dual configurations (int8 outliers against int8 activations,
    # fp4 inliers against MXFP4 activations) on the LLaMA-7B block; --fmt 0:
    # 1:8 + 6:8 (7:8 in all), 1: 2:8 + 4:8 (6:8), 2: 1:8 + 7:8 (8:8)
    "llama7b-block-dual": (6, [0, 1, 2, 3, 4, 5, 6], 4096),
}

# Dense MFMA peaks by operand type (MI355X, TFLOP/s or TOP/s).
MFMA_PEAK = {"fp8": 5033.0, "f16": 2516.6, "fp4": 10066.0, "int8": 5033.0}


def dual_mfma_peak() -> float:
    """Dense-equivalent peak of the dual GEMM's instruction mix: per 64 K of a
    32x32 tile one fp4 x fp4 instruction (32*32*64 products at the fp4 rate)
    and two int8 ones (32*32*32 each at the int8 rate); the dense-equivalent
    work is 2*32*32*64."""
    t = 2 * 32 * 32 * 64 / MFMA_PEAK["fp4"] + 2 * (2 * 32 * 32 * 32) / MFMA_PEAK["int8"]
    return 2 * 32 * 32 * 64 / t


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--workload", default="llama7b-mlp-prefill",
                   help="|".join(WORKLOADS) + "|sweep (with --layer/--M/--fmt)")
    p.add_argument("--no-decode", action="store_true",
                   help="leave out the LLaMA-7B attention decode figures that the default line carries")
    p.add_argument("--layer", type=int, default=0, help="block-sweep layer index (0..6)")
    p.add_argument("--M", type=int, default=0,
                   help="token count: block sweep (default 1) or the dual block workload (default 4096)")
    p.add_argument("--fmt", type=int, default=0,
                   help="format index of the block sweep, or of llama7b-block-dual (0: 1:8 int8 + 6:8 fp4, "
                        "1: 2:8 int8 + 4:8 fp4, 2: 1:8 int8 + 7:8 fp4)")
    p.add_argument("--inlier-scale", default="", choices=["", "e4m3", "ue6m2"],
                   help="INT family: two-level e4m3 or ufp8-e6m2 inlier scales instead of the workload's "
                        "fp16 (the quantized scale formats of the paper's Section 6.4 study)")
    p.add_argument("--qv", type=int, default=0, choices=[0, 16, 32, 64],
                   help="INT family: dense K per inlier scale (Q-Vector length; 0 = the family's 16)")
    p.add_argument("--scale-table", action="store_true",
                   help="INT workloads: GEMM time and bandwidth for every inlier scale format (fp16, e4m3, "
                        "e6m2) and Q-Vector (16, 32, 64), against the bits per weight; one JSON object")
    p.add_argument("--y-dtype", default="f32", choices=["f32", "bf16"],
                   help="GEMM output type (bf16: the fp32 result rounded to nearest even)")
    p.add_argument("--rotate-mb", type=float, default=512.0)
    p.add_argument("--cpu-seconds", type=float, default=10.0)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--context", action="store_true",
                   help="also time cache-resident and eager GEMM launches (context figures)")
    p.add_argument("--no-vendor", action="store_true",
                   help="skip the vendor dense-GEMM context figures (torch.matmul bf16, torch._scaled_mm fp8)")
    p.add_argument("--counters", type=int, default=0, metavar="L",
                   help="counter-collection mode: L eager GEMM launches over the rotated "
                        "weight copies, no graphs, no JSON line")
    p.add_argument("--copy-calibration", type=float, default=0.0, metavar="MB",
                   help="counter calibration: five plain device copies of MB megabytes")
    return p.parse_args()


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2406_13868_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        if f.endswith((".hip", ".h", ".cpp")):
            h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def profile_figures(kind: str, name: str):
    """Counter figures of a workload from a committed rocprofv3 summary
    (profiles/<kind>_<name>.txt, 'key: value' lines), used only while the
    kernel-source hash recorded with them matches the current sources."""
    path = os.path.join(ROOT, "profiles", f"{kind}_{name}.txt")
    if not os.path.exists(path):
        return None
    d = {}
    for ln in open(path):
        if ":" in ln and not ln.startswith("#"):
            k, v = ln.split(":", 1)
            d[k.strip()] = v.strip()
    if d.get("kernel_source_hash") != kernel_source_hash():
        return None
    d["source"] = f"profiles/{kind}_{name}.txt"
    return d


def host_description():
    """CPU model and the BLAS numpy calls, for the CPU baseline."""
    model = None
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                model = ln.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    blas = None
    try:
        cfg = np.show_config(mode="dicts")
        b = cfg["Build Dependencies"]["blas"]
        blas = f"{b.get('name')} {b.get('version', '')}".strip()
    except Exception:  # pragma: no cover - older numpy
        pass
    return model, blas


def main():
    a = parse()
    if a.gpus != 1:
        print(f"bench.py: runs on one GPU only (asked for --gpus {a.gpus}); across GPUs the "
              "layer would shard by output rows of W, with no exchange between them", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2406_13868_amd as sdq

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    sdq._lib.lib()

    if a.copy_calibration > 0:
        # a plain copy kernel of known size: FETCH_SIZE and WRITE_SIZE of one
        # dispatch should each read this many bytes
        n = int(a.copy_calibration * 1e6) // 16 * 16
        src = torch.randint(0, 255, (n,), dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n, "dispatches": 5}))
        return

    if a.scale_table:
        rows = []
        for sf in ("", "e4m3", "ue6m2"):
            for qv in (16, 32, 64):
                r = measure(a, torch, sdq, a.workload, a.M, full=False, scale=(sf, qv))
                ro = r["roofline"]
                rows.append({"scales": sf or "f16", "qv": qv, "bits_per_weight": r["extra"]["bits_per_weight"],
                             "gemm_us": ro["kernel_us"], "bound": ro["bound"], "achieved": ro["achieved"],
                             "unit": ro["unit"], "frac": ro["frac"],
                             "gemm_dense_equiv_tflops": r["extra"]["gemm_dense_equiv_tflops"]})
        print(json.dumps({"scale_table": rows, "workload": r["config"]["workload"],
                          "kernel_source_hash": kernel_source_hash()}))
        return
    res = measure(a, torch, sdq, a.workload, a.M, full=True, scale=(a.inlier_scale, a.qv))
    if res is None:  # counter-collection mode
        return
    line = {
        "metric": "dense-equivalent TFLOP/s and % roofline of sdq_gemm, LLaMA-7B layer shapes",
        "value": res["value"],
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": res["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": res["dtype"],
        "data": "synthetic (seeded generators shaped like the named layers; no weights or datasets)",
        "config": res["config"],
        "roofline": res["roofline"],
        "cpu_baseline": res["cpu_baseline"],
    }
    line.update(res["extra"])
    if a.workload == "llama7b-mlp-prefill" and not a.no_decode and a.counters == 0:
        d = measure(a, torch, sdq, "llama7b-attn-decode", 0, full=False)
        line["decode"] = {"workload": d["config"]["workload"], "formats": d["config"]["formats"],
                          "value": d["value"], "unit": "TFLOP/s", "ms_per_step": d["ms_per_step"],
                          "roofline": d["roofline"],
                          "gemm_dense_equiv_tflops": d["extra"]["gemm_dense_equiv_tflops"]}
    print(json.dumps(line))


def measure(a, torch, sdq, workload, M_arg, full, scale=("", 0)):
    """Time one workload: the step (activation quantization + GEMM of every
    layer) and the GEMM alone, both as HIP graphs over rotated copies, after a
    512 MB fill that leaves no weights in the Infinity Cache.  full: also the
    vendor context and the CPU oracle."""
    dev = torch.device("cuda:0")
    if workload == "sweep":
        wid = 5
        fmt = synth.WORKLOADS[5].formats[a.fmt]
        layers = [a.layer]
        M = M_arg or 1
        wl_name = f"llama7b block sweep {synth.WORKLOADS[5].layers[a.layer].name} M={M} {fmt.label}"
    else:
        wid, layers, M = WORKLOADS[workload]
        if M_arg and wid == 6:
            M = M_arg
        fmt = synth.WORKLOADS[wid].formats[a.fmt if wid == 6 else 0]
        wl_name = synth.WORKLOADS[wid].name
        if wid == 6:
            wl_name += f" M={M} {fmt.n_o}:8 int8 + {fmt.n_i}:8 fp4"
    W_def = synth.WORKLOADS[wid]
    cfg = sdq.Config.of(fmt)
    sfmt, qv = scale
    if sfmt or qv:
        import dataclasses
        if cfg.family != "int":
            raise SystemExit("--inlier-scale and --qv apply to the INT family only")
        cfg = dataclasses.replace(cfg, sfmt_i=sfmt, qv_i=qv)
        wl_name += f", {sfmt or 'fp16'}{' (two-level)' if sfmt == 'e4m3' else ''} inlier scales per {cfg.qv} K"
    if a.y_dtype != "f32" and full:
        import dataclasses
        cfg = dataclasses.replace(cfg, y_dtype=a.y_dtype)
        wl_name += f", {a.y_dtype} output"

    # ---------------------------------------------------------------- inputs
    Ls = [W_def.layers[i] for i in layers]
    Ws, Xs, blobs_host = [], [], []
    t_pack = t_pack1 = 0.0
    for li, L in zip(layers, Ls):
        W = synth.make_w(wid, li, L.N, L.K)
        X = synth.make_x(wid, M, L.K)
        t0 = time.perf_counter()
        blob = sdq.pack(W, cfg)
        t_pack += time.perf_counter() - t0
        if li == layers[0] and full:
            t0 = time.perf_counter()
            sdq.pack(W, cfg, n_threads=1)
            t_pack1 = time.perf_counter() - t0
        Ws.append(W)
        Xs.append(X)
        blobs_host.append(blob)
    phys = sum(b.nbytes for b in blobs_host)
    logical = sum(sdq.logical_bytes(cfg, L.N, L.K) for L in Ls)
    R = max(2, math.ceil(a.rotate_mb * 1e6 / phys))
    x_dtype = torch.bfloat16 if W_def.x_dtype == "bf16" else torch.float32
    blobs = [[torch.from_numpy(b).to(dev) for b in blobs_host] for _ in range(R)]
    Xd = [[torch.from_numpy(X).to(dev).to(x_dtype) for X in Xs] for _ in range(R)]
    Xq = [[torch.empty((M, L.K), dtype=torch.uint8, device=dev) for L in Ls] for _ in range(R)]
    sa = [[torch.empty((M,), dtype=torch.float32, device=dev) for _ in Ls] for _ in range(R)]
    dual = cfg.family == "dual"
    # the dual family's fp4 activations and their e8m0 scales
    Xi = [[torch.empty((M, L.K // 2), dtype=torch.uint8, device=dev) for L in Ls] for _ in range(R)] if dual else None
    Ea = [[torch.empty((M, L.K // 32), dtype=torch.uint8, device=dev) for L in Ls] for _ in range(R)] if dual else None
    Y = [[torch.empty((M, L.N), dtype=cfg.y_torch_dtype(), device=dev) for L in Ls] for _ in range(R)]
    # GEMM workspace (the two-pass path for many MX tokens), one for all layers:
    # the calls are ordered on one stream
    ws_bytes = 0 if dual else max(sdq.gemm_workspace_size(cfg, M, L.N, L.K) for L in Ls)
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev) if ws_bytes else None
    flush = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device=dev)

    def quant(r, j):
        if dual:
            sdq.quantize_act_dual(Xd[r][j], cfg, out=(Xq[r][j], sa[r][j], Xi[r][j], Ea[r][j]))
        else:
            sdq.quantize_act(Xd[r][j], cfg, out=Xq[r][j], scales=sa[r][j])

    for r in range(R):  # every rotated copy's Xq/s_a holds real codes before any GEMM-only launch
        for j in range(len(Ls)):
            quant(r, j)
    torch.cuda.synchronize()

    def gemm_one(r, j, L, q=None):
        q = j if q is None else q  # whose quantized activations
        if dual:
            sdq.gemm_dual(Xq[r][q], sa[r][q], Xi[r][q], Ea[r][q], blobs[r][j], L.N, L.K, cfg, out=Y[r][j])
        else:
            sdq.gemm(Xq[r][q], sa[r][q], blobs[r][j], L.N, L.K, cfg, out=Y[r][j], workspace=ws)

    # A layer that reads an earlier layer's input tensor (k and v read q's,
    # up reads gate's) multiplies that layer's quantized activations: the
    # tensor is quantized once per step, as the model computes it.
    shared = {j: [jj for jj in range(j) if Ls[jj].name == L.input_of][0]
              for j, L in enumerate(Ls) if L.input_of and any(P.name == L.input_of for P in Ls[:j])}

    def step(i):
        r = i % R
        for j, L in enumerate(Ls):
            if j in shared:
                gemm_one(r, j, L, shared[j])
            elif dual:  # quantize into this copy's buffers, then multiply
                quant(r, j)
                gemm_one(r, j, L)
            else:
                sdq.linear(Xd[r][j], blobs[r][j], L.N, L.K, cfg, out=Y[r][j], xq=Xq[r][j],
                           scales=sa[r][j], workspace=ws)

    def gemms(i):
        r = i % R
        for j, L in enumerate(Ls):
            gemm_one(r, j, L)

    def gemms_hot(i):
        for j, L in enumerate(Ls):
            gemm_one(0, j, L)

    def capture(fn, n, start):
        """HIP graph of n calls of fn (launch-bound loops replay without host gaps)."""
        g = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fn(start)
        torch.cuda.current_stream().wait_stream(side)
        with torch.cuda.graph(g):
            for i in range(n):
                fn(start + i)
        return g

    def timed(g, n, cold=True):
        """ms per call of one replay of g (n calls), timed with HIP events on the
        launch stream between two synchronizations; with cold, a 512 MB fill
        on the same stream first evicts the Infinity Cache (outside the events)."""
        torch.cuda.synchronize()
        st = torch.cuda.current_stream()
        if cold:
            flush.fill_(1)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        g.replay()
        e1.record(st)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n  # ms per call

    if a.counters > 0:
        # hardware-counter runs: eager launches of the GEMM kernel only, each on
        # a different weight copy, so that every dispatch streams from HBM
        for i in range(a.counters):
            gemms(i)
        torch.cuda.synchronize()
        print(json.dumps({"counter_launches": a.counters * len(Ls), "rotated_copies": R,
                          "kernel_source_hash": kernel_source_hash()}))
        return None

    def settled(g, n):
        """ms per call of a replay of g once replays have settled: two untimed
        replays (the first uploads the graph; the second still ran a few percent
        slower than every later one on 20-step graphs), then the median of three
        timed replays, each of all n calls."""
        timed(g, n)
        timed(g, n)
        return sorted(timed(g, n) for _ in range(3))[1]

    # ---------------------------------------------------------------- timed steps
    for i in range(a.warmup):
        step(i)
    torch.cuda.synchronize()
    g_step = capture(step, a.steps, a.warmup)
    ms_step = settled(g_step, a.steps)

    # ---------------------------------------------- the GEMM kernel alone (dominant kernel)
    n_g = max(a.steps, 2 * R, 64)
    g_gemm = capture(gemms, n_g, 0)
    gemm_us = settled(g_gemm, n_g) * 1e3
    gemm_hot_us = gemm_b2b_us = None
    if a.context and full:
        g_hot = capture(gemms_hot, n_g, 0)
        timed(g_hot, n_g, cold=False)
        gemm_hot_us = round(timed(g_hot, n_g, cold=False) * 1e3, 3)
        # eager launches (host launch rate included)
        torch.cuda.synchronize()
        stream = torch.cuda.current_stream()
        b0, b1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        b0.record(stream)
        for i in range(n_g):
            gemms(i)
        b1.record(stream)
        torch.cuda.synchronize()
        gemm_b2b_us = round(b0.elapsed_time(b1) * 1e3 / n_g, 3)
    del g_step, g_gemm

    flops = sum(2.0 * M * L.N * L.K for L in Ls)
    eff_frac = fmt.n_o / fmt.m_o + fmt.n_i / fmt.m_i
    y_bytes = 2 if cfg.y_dtype == "bf16" else 4
    alg_bytes = logical + sum(M * L.K + 4 * M + y_bytes * M * L.N for L in Ls)
    paths = [] if dual else sorted({sdq.gemm_path(cfg, M, L.N, L.K, workspace=True) for L in Ls})
    hbm_bound = cfg.family == "int" and M <= 64 or (cfg.family != "int" and M < 256)
    tkey = workload if workload != "sweep" else f"sweep_l{a.layer}_m{M}_f{a.fmt}"
    if wid == 6 and a.fmt:
        tkey += f"_f{a.fmt}"
    if sfmt or qv:
        tkey += f"_{sfmt or 'f16'}_qv{cfg.qv}_scales"
    gemm_s = gemm_us * 1e-6
    if hbm_bound:
        achieved = alg_bytes / gemm_s / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4)}
    else:
        achieved = flops / gemm_s / 1e12
        # the contraction's own low-precision dtype: fp8 (MX), int8 x int4 (INT,
        # priced at the int8 rate), and for the dual family the instruction mix
        # of its fp4 x fp4 and int8 x int8 branches
        peak = round(dual_mfma_peak(), 1) if dual else MFMA_PEAK["fp8" if cfg.family == "mx" else "int8"]
        roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4)}
        if dual:
            roof["frac_of_fp4_dense_peak"] = round(achieved / MFMA_PEAK["fp4"], 4)
        if cfg.family == "int":
            # the INT matrix path issues f16 instructions (the exact hi/lo split)
            roof["issued_dtype"] = "f16"
            roof["frac_of_issued_dtype_peak"] = round(achieved / MFMA_PEAK["f16"], 4)
        roof["effectual_tflops"] = round(flops * eff_frac / gemm_s / 1e12, 1)
        mf = profile_figures("mfma", tkey)
        if mf is not None:
            # issued matrix work from SQ_INSTS_VALU_MFMA_MOPS_* x 512 per GEMM call, and
            # the time those instructions take at their own dtypes' dense peaks
            issued = float(mf["issued_flop_per_call"]) * len(Ls)
            at_peak_s = float(mf["issued_us_at_peak_per_call"]) * 1e-6 * len(Ls)
            roof["mfma_issued_tflops"] = round(issued / gemm_s / 1e12, 1)
            roof["mfma_issued_frac"] = round(at_peak_s / gemm_s, 4)
            roof["mfma_busy_frac"] = float(mf["mfma_busy_frac"])
            roof["issued_over_effectual"] = round(issued / (flops * eff_frac), 3)
            roof["mfma_counters_source"] = mf["source"]
    tr = profile_figures("traffic", tkey)
    roof["traffic"] = int(float(tr["hbm_bytes_per_launch"])) if tr else None
    roof["traffic_source"] = (f"{tr['source']} (rocprofv3 --pmc FETCH_SIZE, WRITE_SIZE, copy-calibrated)"
                              if tr else None)
    roof["kernel_us"] = round(gemm_us / len(Ls), 3)
    # kernels per GEMM call: a two-pass path's time is both passes together
    roof["kernels_per_call"] = 2 if (sdq.PATH_DENSE in paths or sdq.PATH_SPLITK in paths) else 1
    roof["timing"] = (f"HIP events around a graph replay of {n_g} GEMM calls over {R} rotated copies, "
                      "after a 512 MB fill; median of three replays after two untimed ones")

    vendor = None if (a.no_vendor or not full) else vendor_context(torch, Ls, M, a.rotate_mb, max(a.steps, 20))
    cpu = None
    if full and not a.no_cpu_baseline:
        cpu = cpu_baseline(Ws, Xs, fmt, M, a.cpu_seconds, sfmt, qv)

    value = flops / (ms_step * 1e-3) / 1e12
    extra = {
        "gemm_us_graph": round(gemm_us, 3),
        "gemm_us_eager": gemm_b2b_us,
        "gemm_us_cache_resident": gemm_hot_us,
        "gemm_dense_equiv_tflops": round(flops / gemm_s / 1e12, 3),
        "vendor_dense_context": vendor,
        "logical_bytes": int(logical),
        "bits_per_weight": round(8.0 * logical / sum(L.N * L.K for L in Ls), 4),
        "physical_bytes": int(phys),
        "algorithmic_bytes_per_launch": int(alg_bytes),
        "rotated_copies": R,
        "packer_s_threaded": round(t_pack, 3),
        "packer_s_one_thread_first_layer": round(t_pack1, 3),
        "kernel_source_hash": kernel_source_hash(),
    }
    return {
        "value": round(value, 4),
        "ms_per_step": round(ms_step, 5),
        "dtype": {"int": "int8", "mx": "fp8", "dual": "int8+fp4"}[cfg.family],
        "config": {"workload": wl_name, "M": M, "layers": [[L.name, L.N, L.K] for L in Ls],
                   "formats": fmt.label,
                   "gemm_path": "dual mfma" if dual else ", ".join(
                       ["decode", "mfma", "dense (two passes)", "split-K (two passes)"][p - 1] for p in paths),
                   "activations_quantized": [L.name for j, L in enumerate(Ls) if j not in shared],
                   "parallelism": "none (one GPU)"},
        "roofline": roof,
        "cpu_baseline": cpu,
        "extra": extra,
    }


def vendor_context(torch, Ls, M, rotate_mb, n):
    """Dense GEMMs of the same shapes through the vendor library, timed like the
    SDQ GEMM (HIP graph of n launches over rotated weight copies, HIP events):
    a linear layer in bf16 (weight [N, K]), torch._scaled_mm in fp8 e4m3 with per-tensor scales
    (fp32 output), and with e8m0 scales per 32 K (MXFP8).  Context only: these
    read 16 or 8 bits per weight where the decomposed format reads 3.6-5."""
    dev = torch.device("cuda:0")
    out = {}
    for L in Ls:
        key = f"{M}x{L.N}x{L.K}"
        if key in out:
            continue
        g = torch.Generator(device=dev)
        g.manual_seed(0)
        a16 = torch.randn(M, L.K, device=dev, generator=g).to(torch.bfloat16)
        R = max(2, math.ceil(rotate_mb * 1e6 / (2 * L.N * L.K)))
        w16 = [torch.randn(L.N, L.K, device=dev, generator=g).to(torch.bfloat16) for _ in range(R)]
        a8 = a16.to(torch.float8_e4m3fn)
        w8 = [w.to(torch.float8_e4m3fn) for w in w16[: max(2, (R + 1) // 2)]]
        one = torch.ones((), device=dev)
        sa = torch.full((M, L.K // 32), 127, device=dev, dtype=torch.uint8).view(torch.float8_e8m0fnu)
        sb = torch.full((L.N, L.K // 32), 127, device=dev, dtype=torch.uint8).view(torch.float8_e8m0fnu)
        fl = 2.0 * M * L.N * L.K
        cases = {
            "bf16_linear": lambda i: torch.nn.functional.linear(a16, w16[i % len(w16)]),
            "fp8_scaled_mm_fp32_out": lambda i: torch._scaled_mm(a8, w8[i % len(w8)].t(), scale_a=one, scale_b=one,
                                                                 out_dtype=torch.float32),
            "mxfp8_scaled_mm_bf16_out": lambda i: torch._scaled_mm(a8, w8[i % len(w8)].t(), scale_a=sa, scale_b=sb,
                                                                   out_dtype=torch.bfloat16),
        }
        res = {}
        for name, f in cases.items():
            try:
                f(0)
                torch.cuda.synchronize()
                gr = torch.cuda.CUDAGraph()
                side = torch.cuda.Stream()
                side.wait_stream(torch.cuda.current_stream())
                with torch.cuda.stream(side):
                    f(1)
                torch.cuda.current_stream().wait_stream(side)
                with torch.cuda.graph(gr):
                    for i in range(n):
                        f(i)
                gr.replay()
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                gr.replay()
                e1.record()
                torch.cuda.synchronize()
                us = e0.elapsed_time(e1) * 1e3 / n
                res[name] = {"us": round(us, 3), "tflops": round(fl / (us * 1e-6) / 1e12, 1)}
            except Exception as e:  # a shape or dtype the library does not take
                res[name] = {"error": repr(e)[:160]}
        out[key] = res
        del w16, w8
    return out


def cpu_baseline(Ws, Xs, fmt, M, seconds, sfmt_i="", qv=0):
    """The oracle as it stands, on this host, over a bounded sample of the
    workload: its decomposition and quantization (pack) of the first rows of
    every layer, timed once, then its activation quantization and fp64
    decomposed product of those rows for at most 64 tokens, repeated for about
    `seconds`."""
    from oracle import sdq as S
    try:
        from threadpoolctl import threadpool_info
        threads = max([d.get("num_threads", 1) for d in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count()
    cfg_o = S.config_from(fmt, sfmt_i=sfmt_i, qv=qv)
    ms = min(M, 64)
    rows = 1024
    t0 = time.perf_counter()
    packs = [S.pack_logical(W[:rows], cfg_o) for W in Ws]
    t_pack = time.perf_counter() - t0
    n_w = sum(min(rows, W.shape[0]) * W.shape[1] for W in Ws)
    reps, t, flops = 0, 0.0, 0.0
    while t < seconds or reps == 0:
        t0 = time.perf_counter()
        for X, Lg in zip(Xs, packs):
            if cfg_o.family == "dual":
                S.gemm_fp64_dual(*S.quantize_act_dual(X[:ms]), Lg)
            else:
                Xq, s_a = S.quantize_act(X[:ms], cfg_o)
                S.gemm_fp64(Xq, s_a, Lg)
            flops += 2.0 * ms * Lg["N"] * Lg["K"]
        t += time.perf_counter() - t0
        reps += 1
    model, blas = host_description()
    return {"value": round(flops / t / 1e12, 8), "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{reps} repetitions of numpy quantize_act + fp64 gemm over the first {rows} rows of "
                      f"{len(Ws)} layer(s) at {ms} token(s), {t:.1f} s",
            "oracle_pack_s": round(t_pack, 2),
            "oracle_pack_weights_per_s": round(n_w / t_pack, 1),
            "cpu_model": model, "blas": blas}


if __name__ == "__main__":
    main()
