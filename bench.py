"""Throughput of the FP8 linear layer's hot path on one MI355X.

A step is one pass of the whole path at the Qwen2-1.5B QKV-projection shape
(M = 8192 tokens, K = 1536, N = 2048; per-tensor scales, X and W in E4M3, dY
in E5M2): amax and quantisation of X and W, the Fprop GEMM, amax and
quantisation of dY, the Dgrad and Wgrad GEMMs (puro_linear_fwd then
puro_linear_bwd). Inputs are seeded synthetic tensors resident in HBM before
the timed region.

Prints one JSON line: the metric (TFLOP/s of fwd + dgrad + wgrad GEMM work per
step time), a per-call breakdown and a roofline entry for the dominant kernel
(each call timed with HIP events on its stream around back-to-back launches),
and the CPU oracle timed on a sample of the same workload.
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

FP8_PEAK_TFLOPS = 5000.0   # MI355X dense FP8 MFMA
HBM_PEAK_GBS = 8000.0      # MI355X HBM3E
METRIC = "FP8 linear fwd+dgrad+wgrad TFLOP/s at Qwen2-1.5B shapes; % FP8 MFMA peak"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--tokens", type=int, default=8192)
    ap.add_argument("--cpu-tokens", type=int, default=8192,
                    help="tokens of the workload the CPU oracle is timed on (0: skip)")
    ap.add_argument("--cpu-reps", type=int, default=4, help="repetitions of the CPU oracle sample")
    ap.add_argument("--graph", action="store_true",
                    help="replay the step captured in a HIP graph instead of launching its kernels one by one "
                         "(measured no faster: the launches are not host-bound)")
    ap.add_argument("--only", choices=("step",) + CALLS + ("copy",),
                    help="run just this call (or a whole step) warmup + steps times and print its average "
                         "time, for profilers; 'copy' is a plain 256 MiB device copy that calibrates "
                         "the HBM byte counters")
    return ap.parse_args()


def cpu_baseline(tokens, reps):
    """The oracle (test infrastructure, unmodified) on the first `tokens`
    tokens of the same workload, `reps` times over: quantisation of X, W, dY
    and the three FP64 GEMMs; reported as TFLOP/s of the sampled GEMM work."""
    from oracle import linear
    from paper_2608_27370_amd import inputs
    d = inputs.qkv(M=tokens)
    rc = linear.recipe("tensor")
    t0 = time.perf_counter()
    for _ in range(reps):
        _, _, saved = linear.linear_fwd(d["X"], d["W"], rc)
        linear.linear_bwd(d["dY"], saved, rc)
    dt = time.perf_counter() - t0
    flops = reps * 3 * 2.0 * tokens * inputs.QKV_OUT * inputs.HIDDEN
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "seconds": round(dt, 2),
            "sample": "oracle linear fwd+bwd on %d of the 8192 tokens (X[%d,1536], W[2048,1536], dY[%d,2048]), "
                      "%d times; FP64 GEMMs on %d OpenMP threads" % (tokens, tokens, tokens, reps, threads)}


CALLS = ("quantize_x", "quantize_w", "fprop", "quantize_dy", "dgrad", "wgrad")


def calls(torch, puro, dev, M, N, K, X, W, dY, Y, dX, dW, saved):
    """The step's calls one at a time, on buffers of their own, as
    (key, label, fn, flops, algorithmic bytes, kernel launches) rows."""
    xq = torch.empty(M, K, dtype=torch.uint8, device=dev)
    wq = torch.empty(N, K, dtype=torch.uint8, device=dev)
    dyq = torch.empty(M, N, dtype=torch.uint8, device=dev)
    dyqT = torch.empty(N, M, dtype=torch.uint8, device=dev)
    sx = torch.empty(1, dtype=torch.float32, device=dev)
    sw = torch.empty(1, dtype=torch.float32, device=dev)
    sdy = torch.empty(1, dtype=torch.float32, device=dev)
    qws = torch.empty(max(1, puro.lib().puro_quantize_workspace_size(M, N)), dtype=torch.uint8, device=dev)
    gws = torch.empty(max(1, max(puro.fp8_gemm_workspace_size(M, N, K, 0), puro.fp8_gemm_workspace_size(M, K, N, 0),
                                 puro.fp8_gemm_workspace_size(N, K, M, 1))), dtype=torch.uint8, device=dev)
    A_f = puro.operand(xq, puro.E4M3, puro.SCALE_TENSOR, sx)
    B_f = puro.operand(wq, puro.E4M3, puro.SCALE_TENSOR, sw)
    A_d = puro.operand(dyq, puro.E5M2, puro.SCALE_TENSOR, sdy)
    B_d = puro.operand(saved["wq_t"], puro.E4M3, puro.SCALE_TENSOR, sw)
    A_w = puro.operand(dyqT, puro.E5M2, puro.SCALE_TENSOR, sdy)
    B_w = puro.operand(saved["xq_t"], puro.E4M3, puro.SCALE_TENSOR, sx)
    # quantisation moves 2 B read + 1 B (q) + 1 B (qT) written per element
    return [
        ("quantize_x", "quantize X (amax + encode, q and qT)", lambda: puro.quantize_fp8(
            X, puro.E4M3, out=dict(q=xq, scale=sx, qT=saved["xq_t"]), want_qT=True, ws=qws), None,
         M * K * 4.0, 2),
        ("quantize_w", "quantize W (amax + encode, q and qT)", lambda: puro.quantize_fp8(
            W, puro.E4M3, out=dict(q=wq, scale=sw, qT=saved["wq_t"]), want_qT=True, ws=qws), None,
         N * K * 4.0, 2),
        ("fprop", "fprop GEMM %dx%dx%d" % (M, N, K),
         lambda: puro.fp8_gemm(A_f, M, B_f, N, K, puro.OUT_BF16, D=Y, ws=gws), 2.0 * M * N * K, None,
         puro.fp8_gemm_plan(M, N, K)["launches"]),
        ("quantize_dy", "quantize dY (amax + encode, q and qT)", lambda: puro.quantize_fp8(
            dY, puro.E5M2, out=dict(q=dyq, scale=sdy, qT=dyqT), want_qT=True, ws=qws), None, M * N * 4.0, 2),
        ("dgrad", "dgrad GEMM %dx%dx%d" % (M, K, N),
         lambda: puro.fp8_gemm(A_d, M, B_d, K, N, puro.OUT_BF16, D=dX, ws=gws), 2.0 * M * N * K, None,
         puro.fp8_gemm_plan(M, K, N)["launches"]),
        ("wgrad", "wgrad GEMM %dx%dx%d" % (N, K, M),
         lambda: puro.fp8_gemm(A_w, N, B_w, K, M, puro.OUT_FP32, D=dW, ws=gws), 2.0 * M * N * K, None,
         puro.fp8_gemm_plan(N, K, M)["launches"]),
    ]


COPY_BYTES = 256 << 20
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "hbm_bytes_qkv.md")


def profiled_traffic(call):
    """HBM-side bytes per launch of `call` at the 8192-token workload, from the
    committed rocprofv3 FETCH_SIZE / WRITE_SIZE summary (scaled by its copy
    calibration); None when that summary is missing or any source it was
    measured on has changed since."""
    try:
        text = open(TRAFFIC_PROFILE).read()
        d = json.loads(text.split("```json", 1)[1].split("```", 1)[0])
        for path, digest in d["sources"].items():
            if hashlib.sha256(open(os.path.join(ROOT, path), "rb").read()).hexdigest() != digest:
                return None
        return d["calls"][call]["bytes"]
    except (OSError, IndexError, KeyError, ValueError):
        return None


def run_only(args, torch, stream, step, make_calls):
    """Profiling mode: one call (or the whole step) warmup + steps times."""
    if args.only == "copy":
        src = torch.empty(COPY_BYTES // 4, dtype=torch.float32, device=stream.device).fill_(1.0)
        dst = torch.empty_like(src)
        fn, label = (lambda: dst.copy_(src)), "plain device copy of %d bytes" % COPY_BYTES
    elif args.only == "step":
        fn, label = step, "linear fwd + bwd step"
    else:
        row = [r for r in make_calls() if r[0] == args.only][0]
        fn, label = row[2], row[1]
    for _ in range(args.warmup):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    print(json.dumps({"only": args.only, "call": label, "launches": args.steps,
                      "us_per_call": round(e0.elapsed_time(e1) / max(1, args.steps) * 1e3, 2)}))


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: this build measures the single-GPU share of the data-"
              "parallel path (every rank runs the same layer on its own tokens); --gpus %d is not "
              "supported" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_27370_amd import inputs, puro

    puro.lib()
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    M, K, N = args.tokens, inputs.HIDDEN, inputs.QKV_OUT
    d = inputs.qkv(M=M)

    def up(bits):
        import numpy as np
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)

    X, W, dY = up(d["X"]), up(d["W"]), up(d["dY"])
    rc = puro.LinearRecipe(puro.E4M3, puro.E4M3, puro.E5M2, 0, puro.SCALE_FP32)
    saved = puro.linear_saved(M, N, K, rc, dev)
    Y = torch.empty(M, N, dtype=torch.bfloat16, device=dev)
    dX = torch.empty(M, K, dtype=torch.bfloat16, device=dev)
    dW = torch.empty(N, K, dtype=torch.float32, device=dev)
    wsf = torch.empty(max(1, puro.linear_fwd_workspace_size(M, N, K, rc)), dtype=torch.uint8, device=dev)
    wsb = torch.empty(max(1, puro.linear_bwd_workspace_size(M, N, K, rc)), dtype=torch.uint8, device=dev)

    def step():
        puro.linear_fwd(X, W, rc, Y=Y, saved=saved, ws=wsf)
        puro.linear_bwd(dY, saved, rc, K, dX=dX, dW=dW, ws=wsb)

    stream = torch.cuda.current_stream()
    if args.only:
        run_only(args, torch, stream, step, lambda: calls(torch, puro, dev, M, N, K, X, W, dY, Y, dX, dW, saved))
        return
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    run = step
    if args.graph:
        # the step's launches captured once in a HIP graph and replayed: the
        # same kernels on the same buffers, without per-launch host overhead
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            step()
        stream.wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        run = graph.replay
        for _ in range(args.warmup):
            run()
        torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for _ in range(args.steps):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = e0.elapsed_time(e1) / args.steps
    gemm_flops = 3 * 2.0 * M * N * K
    value = gemm_flops / (ms_per_step * 1e-3) / 1e12

    # each call on its own, timed over back-to-back launches between two
    # events on the stream they run on (so that host launch latency hides
    # behind the queue, as in the step)
    kernels = calls(torch, puro, dev, M, N, K, X, W, dY, Y, dX, dW, saved)
    reps = max(20, args.steps // 2)
    breakdown = []
    for _, name, fn, flops, nbytes, launches in kernels:
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / reps * 1e3
        row = {"call": name, "us": round(us, 2), "launches": launches}
        if flops:
            row["tflops"] = round(flops / (us * 1e-6) / 1e12, 1)
        if nbytes:
            row["gbs_algorithmic"] = round(nbytes / (us * 1e-6) / 1e9, 1)
        breakdown.append(row)
    gemm_rows = [r for r in breakdown if "tflops" in r]
    gemm_us = sum(r["us"] for r in gemm_rows)
    # dominant kernel: the slowest call that is a single kernel launch
    single = [(r, k) for r, k in zip(breakdown, kernels) if k[5] == 1]
    dom, dom_k = max(single, key=lambda rk: rk[0]["us"])
    traffic = profiled_traffic(dom_k[0]) if M == 8192 else None
    if "tflops" in dom:
        roofline = {"bound": "mfma", "kernel": dom["call"], "achieved": dom["tflops"], "peak": FP8_PEAK_TFLOPS,
                    "unit": "TFLOP/s", "frac": round(dom["tflops"] / FP8_PEAK_TFLOPS, 4),
                    "algorithmic_flops_per_launch": dom_k[3]}
    else:
        roofline = {"bound": "hbm", "kernel": dom["call"], "achieved": dom["gbs_algorithmic"], "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": round(dom["gbs_algorithmic"] / HBM_PEAK_GBS, 4),
                    "algorithmic_bytes_per_launch": dom_k[4]}
    roofline["us_per_launch"] = dom["us"]
    roofline["traffic"] = traffic
    roofline["traffic_unit"] = "HBM-side bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)"

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp8",
        "data": "synthetic",
        "config": {"workload": "qkv_projection_fwd_dgrad_wgrad", "M": M, "K": K, "N": N,
                   "recipe": "per-tensor scales, X/W E4M3, dY E5M2, BF16 Y/dX, FP32 dW",
                   "launch": "hip_graph" if args.graph else "eager"},
        "pct_fp8_peak": round(100 * value / FP8_PEAK_TFLOPS, 2),
        "gemm_only_tflops": round(gemm_flops / (gemm_us * 1e-6) / 1e12, 1),
        "breakdown": breakdown,
        "roofline": roofline,
        "wall_s_timed": round(wall, 3),
    }
    if args.cpu_tokens > 0:
        out["cpu_baseline"] = cpu_baseline(args.cpu_tokens, args.cpu_reps)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
