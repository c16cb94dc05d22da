"""Throughput of the FP8 linear layer's hot path on one MI355X.

A step is one pass of the whole path at the Qwen2-1.5B QKV-projection shape
(M = 8192 tokens, K = 1536, N = 2048; per-tensor scales, X and W in E4M3, dY
in E5M2): amax and quantisation of X and W, the Fprop GEMM, amax and
quantisation of dY, the Dgrad and Wgrad GEMMs (puro_linear_fwd then
puro_linear_bwd). Inputs are seeded synthetic tensors resident in HBM before
the timed region.

Prints one JSON line: the metric (TFLOP/s of fwd + dgrad + wgrad GEMM work per
step time), a per-call breakdown and a roofline entry for the dominant kernel
(each call timed with HIP events on its stream around back-to-back launches;
also per launch, as median, p10 and p90, and with --cold after a fill that
evicts the caches), and the CPU oracle timed on a sample of the same workload.
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
    ap.add_argument("--cold", action="store_true",
                    help="also time every call after a 512 MiB fill that evicts the MALL and the L2s "
                         "(kept out of the default run, whose kernel trace profiles warm launches)")
    ap.add_argument("--graph", action="store_true",
                    help="replay the step captured in a HIP graph instead of launching its kernels one by one "
                         "(measured no faster: the launches are not host-bound)")
    ap.add_argument("--suite", action="store_true",
                    help="instead of the headline step, time every workload (the five Qwen2-1.5B-shaped ones "
                         "and the paper's own 1.7B shapes under both power-of-two scale rules) next to the "
                         "same GEMMs in BF16, and report the FP8 errors of the two rules; one JSON line each")
    ap.add_argument("--only", choices=("step",) + CALLS + ("copy",) + SWIGLU_CALLS + RMSNORM_CALLS,
                    help="run just this call (or a whole step) warmup + steps times and print its average "
                         "time, for profilers; 'copy' is a plain 256 MiB device copy that calibrates "
                         "the HBM byte counters; swiglu_* and rmsnorm_* are the fused SwiGLU / RMSNorm + "
                         "quantise calls of the 8192-token MLP and QKV input")
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
SWIGLU_CALLS = ("swiglu_tensor", "swiglu_groups", "swiglu_bwd_groups")
RMSNORM_CALLS = ("rmsnorm_tensor", "rmsnorm_groups")


def rmsnorm_workload(torch, puro, M=8192, d=1536):
    """The fused RMSNorm + quantise of the QKV projection's input: x [M, d]
    drawn on the device (N(0,1), 1% of the channels x20), gamma ~ N(1, 0.1^2),
    eps 1e-6, E4M3 with q and qT, per-tensor and 1x128 + 128x1 groups.
    Returns {name: (fused call, unfused call, algorithmic bytes)}; unfused is
    torch's BF16 RMSNorm, then puro_quantize_fp8 of its output. Algorithmic
    bytes: x read once (2 B) and q, qT written (2 B) per element."""
    dev = torch.device("cuda", 0)
    g = torch.Generator(device=dev)
    g.manual_seed(1)
    x = torch.randn(M, d, generator=g, device=dev)
    x[:, torch.randperm(d, generator=g, device=dev)[:d // 100]] *= 20.0
    x = x.to(torch.bfloat16)
    gamma = (1.0 + 0.1 * torch.randn(d, generator=g, device=dev)).to(torch.bfloat16)
    E4 = puro.E4M3
    outs = {"q": torch.empty(M, d, dtype=torch.uint8, device=dev), "qT": torch.empty(d, M, dtype=torch.uint8, device=dev),
            "rstd": torch.empty(M, dtype=torch.float32, device=dev)}
    ts = dict(outs, scale=torch.empty(1, dtype=torch.float32, device=dev))
    gs = dict(outs, scale=torch.empty(M, d // 128, dtype=torch.float32, device=dev),
              scaleT=torch.empty(d, M // 128, dtype=torch.float32, device=dev))
    ws = torch.empty(max(puro.lib().puro_rmsnorm_quantize_workspace_size(M, d),
                         puro.lib().puro_quantize_workspace_size(M, d)), dtype=torch.uint8, device=dev)

    def unfused(mode, rnd, out):
        def fn():
            y = torch.nn.functional.rms_norm(x, (d,), gamma, 1e-6)
            puro.quantize_fp8(y, E4, mode=mode, rnd=rnd, want_qT=True, out=out, ws=ws)
        return fn
    nbytes = M * d * 4.0
    return {
        "rmsnorm_tensor": (lambda: puro.rmsnorm_quantize_fp8(x, gamma, 1e-6, E4, puro.SCALE_TENSOR, puro.SCALE_FP32,
                                                             want_qT=True, out=ts, ws=ws),
                           unfused(puro.SCALE_TENSOR, puro.SCALE_FP32, ts), nbytes),
        "rmsnorm_groups": (lambda: puro.rmsnorm_quantize_fp8(x, gamma, 1e-6, E4, puro.SCALE_ROW_1x128, puro.SCALE_POW2,
                                                             want_qT=True, out=gs, ws=ws),
                           unfused(puro.SCALE_ROW_1x128, puro.SCALE_POW2, gs), nbytes),
    }


def swiglu_workload(torch, puro, M=8192):
    """The fused SwiGLU + quantise of the 8192-token MLP: H [M, 8960] from
    a device-drawn gate/up output [M, 17920] ~ N(0, 1.7^2) (the spread of the
    MLP's gate/up GEMM output), E4M3, per-tensor (q and qT) and 1x128 +
    128x1 power-of-two groups. Returns {name: (fused call, unfused call,
    algorithmic bytes)}; unfused is torch's BF16 silu and multiply, then
    puro_quantize_fp8 of the BF16 H. Algorithmic bytes: gate and up read
    once (4 B per H element) and one byte per element for each of q and qT.
    Also the backward (swiglu_bwd_groups): dgu [M, 17920] from dH [M, 8960]
    and the gate/up output, 1x128 + 128x1 groups; unfused is torch's binary32
    arithmetic of the same formulas into a BF16 dgu, then puro_quantize_fp8.
    Its algorithmic bytes: dH, g and u read once (6 B per dH element) and q,
    qT of both halves written (4 B)."""
    from paper_2608_27370_amd import inputs
    F = inputs.MLP
    dev = torch.device("cuda", 0)
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    gu = (torch.randn(M, 2 * F, generator=g, device=dev) * 1.7).to(torch.bfloat16)
    E4 = puro.E4M3
    outs = {"q": torch.empty(M, F, dtype=torch.uint8, device=dev), "qT": torch.empty(F, M, dtype=torch.uint8, device=dev)}
    ts = dict(outs, scale=torch.empty(1, dtype=torch.float32, device=dev))
    gs = dict(outs, scale=torch.empty(M, F // 128, dtype=torch.float32, device=dev),
              scaleT=torch.empty(F, M // 128, dtype=torch.float32, device=dev))
    ws = torch.empty(max(1, puro.lib().puro_swiglu_quantize_workspace_size(M, F)), dtype=torch.uint8, device=dev)
    Hbuf = torch.empty(M, F, dtype=torch.bfloat16, device=dev)

    def unfused(mode, rnd, out):
        def fn():
            torch.mul(torch.nn.functional.silu(gu[:, :F]), gu[:, F:], out=Hbuf)
            puro.quantize_fp8(Hbuf, E4, mode=mode, rnd=rnd, want_qT=True, out=out, ws=ws)
        return fn
    nbytes = M * F * 6.0
    dh = (torch.randn(M, F, generator=g, device=dev) * 1e-3).to(torch.bfloat16)
    dgu = torch.empty(M, 2 * F, dtype=torch.bfloat16, device=dev)
    bs = {"q": torch.empty(M, 2 * F, dtype=torch.uint8, device=dev),
          "qT": torch.empty(2 * F, M, dtype=torch.uint8, device=dev),
          "scale": torch.empty(M, 2 * F // 128, dtype=torch.float32, device=dev),
          "scaleT": torch.empty(2 * F, M // 128, dtype=torch.float32, device=dev)}
    wsb = torch.empty(max(1, puro.lib().puro_swiglu_bwd_quantize_workspace_size(M, F),
                          puro.lib().puro_quantize_workspace_size(M, 2 * F)), dtype=torch.uint8, device=dev)

    def unfused_bwd():
        gg, uu = gu[:, :F].float(), gu[:, F:].float()
        sg = torch.sigmoid(gg)
        dhf = dh.float()
        dgu[:, :F] = dhf * uu * (sg * (1.0 + gg * (1.0 - sg)))
        dgu[:, F:] = dhf * gg * sg
        puro.quantize_fp8(dgu, E4, mode=puro.SCALE_ROW_1x128, rnd=puro.SCALE_POW2, want_qT=True, out=bs, ws=wsb)
    return {
        "swiglu_bwd_groups": (lambda: puro.swiglu_bwd_quantize_fp8(dh, gu, E4, puro.SCALE_ROW_1x128, puro.SCALE_POW2,
                                                                   want_qT=True, out=bs, ws=wsb),
                              unfused_bwd, M * F * 10.0),
        "swiglu_tensor": (lambda: puro.swiglu_quantize_fp8(gu, F, E4, puro.SCALE_TENSOR, puro.SCALE_FP32,
                                                           want_qT=True, out=ts, ws=ws),
                          unfused(puro.SCALE_TENSOR, puro.SCALE_FP32, ts), nbytes),
        "swiglu_groups": (lambda: puro.swiglu_quantize_fp8(gu, F, E4, puro.SCALE_ROW_1x128, puro.SCALE_POW2,
                                                           want_qT=True, out=gs, ws=ws),
                          unfused(puro.SCALE_ROW_1x128, puro.SCALE_POW2, gs), nbytes),
    }


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
    if args.only in SWIGLU_CALLS:
        from paper_2608_27370_amd import puro
        fn, label = swiglu_workload(torch, puro)[args.only][0], "fused SwiGLU + quantise (%s)" % args.only
    elif args.only in RMSNORM_CALLS:
        from paper_2608_27370_amd import puro
        fn, label = rmsnorm_workload(torch, puro)[args.only][0], "fused RMSNorm + quantise (%s)" % args.only
    elif args.only == "copy":
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


class Suite:
    """Workloads for the comparison mode: device-drawn seeded inputs with the
    distributions of the parity inputs, each FP8 pass timed next to the same
    three GEMMs in BF16 (hipBLASLt through torch.mm)."""

    def __init__(self, torch, puro):
        self.torch, self.puro = torch, puro
        self.dev = torch.device("cuda", 0)
        self.stream = torch.cuda.current_stream()
        self.gen = torch.Generator(device=self.dev)
        self.gen.manual_seed(0)
        self.e0 = torch.cuda.Event(enable_timing=True)
        self.e1 = torch.cuda.Event(enable_timing=True)

    def normal(self, shape, std=1.0):
        t = self.torch
        return (t.randn(shape, generator=self.gen, device=self.dev) * std).to(t.bfloat16)

    def outliers(self, shape):
        """N(0,1) with 1% of the columns (input channels) scaled by 20."""
        t = self.torch
        x = t.randn(shape, generator=self.gen, device=self.dev)
        cols = t.randperm(shape[1], generator=self.gen, device=self.dev)[:max(1, shape[1] // 100)]
        x[:, cols] *= 20.0
        return x.to(t.bfloat16)

    def student_t3(self, shape):
        """Student-t with 3 degrees of freedom: z / sqrt(chi2_3 / 3)."""
        t = self.torch
        z = t.randn(shape, generator=self.gen, device=self.dev)
        c = sum(t.randn(shape, generator=self.gen, device=self.dev) ** 2 for _ in range(3))
        return (z / t.sqrt(c / 3.0)).to(t.bfloat16)

    def time_us(self, fn, reps):
        for _ in range(2):
            fn()
        self.torch.cuda.synchronize()
        self.e0.record(self.stream)
        for _ in range(reps):
            fn()
        self.e1.record(self.stream)
        self.torch.cuda.synchronize()
        return self.e0.elapsed_time(self.e1) / reps * 1e3

    def fp8_layers(self, layers, recipe):
        """Forward of every linear in order, then backward in reverse order,
        as a training step runs them. layers: list of (X, W, dY)."""
        t, P = self.torch, self.puro
        state, wsf, wsb = [], 1, 1
        for X, W, dY in layers:
            M, K = X.shape
            N = W.shape[0]
            wsf = max(wsf, P.linear_fwd_workspace_size(M, N, K, recipe))
            wsb = max(wsb, P.linear_bwd_workspace_size(M, N, K, recipe))
        wsf = t.empty(wsf, dtype=t.uint8, device=self.dev)
        wsb = t.empty(wsb, dtype=t.uint8, device=self.dev)
        outs = {}
        for X, W, dY in layers:
            M, K = X.shape
            N = W.shape[0]
            key = (M, N, K)
            if key not in outs:   # outputs of equal shapes share buffers (overwritten)
                outs[key] = (t.empty(M, N, dtype=t.bfloat16, device=self.dev),
                             t.empty(M, K, dtype=t.bfloat16, device=self.dev),
                             t.empty(N, K, dtype=t.float32, device=self.dev))
            state.append((X, W, dY, K, P.linear_saved(M, N, K, recipe, self.dev)) + outs[key])

        def run():
            for X, W, dY, K, saved, Y, dX, dW in state:
                P.linear_fwd(X, W, recipe, Y=Y, saved=saved, ws=wsf)
            for X, W, dY, K, saved, Y, dX, dW in reversed(state):
                P.linear_bwd(dY, saved, recipe, K, dX=dX, dW=dW, ws=wsb)
        return run, state

    def bf16_layers(self, layers):
        """The same GEMMs in BF16: Y = X W^T, dX = dY W, dW = dY^T X."""
        t = self.torch
        outs, state = {}, []
        for X, W, dY in layers:
            M, K = X.shape
            N = W.shape[0]
            key = (M, N, K)
            if key not in outs:
                outs[key] = (t.empty(M, N, dtype=t.bfloat16, device=self.dev),
                             t.empty(M, K, dtype=t.bfloat16, device=self.dev),
                             t.empty(N, K, dtype=t.bfloat16, device=self.dev))
            state.append((X, W, dY) + outs[key])

        def run():
            for X, W, dY, Y, dX, dW in state:
                t.mm(X, W.t(), out=Y)
            for X, W, dY, Y, dX, dW in reversed(state):
                t.mm(dY, W, out=dX)
                t.mm(dY.t(), X, out=dW)
        return run

    def compare(self, name, layers, recipe, reps, extra=None):
        flops = sum(3 * 2.0 * X.shape[0] * X.shape[1] * W.shape[0] for X, W, _ in layers)
        fp8, _ = self.fp8_layers(layers, recipe)
        us8 = self.time_us(fp8, reps)
        us16 = self.time_us(self.bf16_layers(layers), reps)
        row = {"workload": name, "gemms": [list(X.shape) + [W.shape[0]] for X, W, _ in layers[:4]],
               "linears": len(layers), "fp8_us": round(us8, 1), "bf16_us": round(us16, 1),
               "fp8_tflops": round(flops / us8 / 1e6, 1), "bf16_tflops": round(flops / us16 / 1e6, 1),
               "fp8_over_bf16": round(us16 / us8, 3)}
        row.update(extra or {})
        print(json.dumps(row), flush=True)
        return row

    def errors(self, X, W, dY, recipe):
        """Relative Frobenius errors of the FP8 Y, dX, dW (and, for scale,
        of the BF16 GEMMs) against FP32 products of the same BF16 inputs, and
        the relative RMS error of X after quantisation and dequantisation in
        1x128 groups."""
        t, P = self.torch, self.puro
        run, state = self.fp8_layers([(X, W, dY)], recipe)
        run()
        _, _, _, _, saved, Y, dX, dW = state[0]
        Xf, Wf, dYf = X.float(), W.float(), dY.float()
        ref = (t.mm(Xf, Wf.t()), t.mm(dYf, Wf), t.mm(dYf.t(), Xf))
        bf = (t.mm(X, W.t()), t.mm(dY, W), t.mm(dY.t(), X))

        def rel(a, b):
            return float(t.linalg.vector_norm(a.float() - b) / t.linalg.vector_norm(b))
        q = P.quantize_fp8(X, P.E4M3, mode=P.SCALE_ROW_1x128, rnd=recipe.rnd)
        table = t.arange(256, dtype=t.uint8).view(t.float8_e4m3fn).float().to(self.dev)
        xd = table[q["q"].long()] * q["scale"].repeat_interleave(128, dim=1)
        out = {"rel_err_" + k: round(rel(a, b), 6) for k, a, b in zip(("Y", "dX", "dW"), (Y, dX, dW), ref)}
        out.update({"bf16_rel_err_" + k: round(rel(a, b), 6) for k, a, b in zip(("Y", "dX", "dW"), bf, ref)})
        out["x_rel_rms_1x128"] = round(rel(xd, Xf), 6)
        return out


def run_suite(args):
    import torch
    from paper_2608_27370_amd import inputs, puro

    puro.lib()
    torch.cuda.set_device(0)
    S = Suite(torch, puro)
    reps = max(3, min(args.steps, 20))
    E4, E5 = puro.E4M3, puro.E5M2
    tensor = puro.LinearRecipe(E4, E4, E5, 0, puro.SCALE_FP32)
    H, Q, F, V = inputs.HIDDEN, inputs.QKV_OUT, inputs.MLP, inputs.VOCAB

    # single FP8 linear forward, 256 x 1536 x 1536
    X, W = S.normal((256, H)), S.normal((H, H), 0.02)
    y = torch.empty(256, H, dtype=torch.bfloat16, device=S.dev)
    sv = puro.linear_saved(256, H, H, tensor, S.dev)
    us8 = S.time_us(lambda: puro.linear_fwd(X, W, tensor, Y=y, saved=sv), 200)
    us16 = S.time_us(lambda: torch.mm(X, W.t(), out=y), 200)
    f = 2.0 * 256 * H * H
    print(json.dumps({"workload": "single_fwd_256x1536x1536", "fp8_us": round(us8, 2), "bf16_us": round(us16, 2),
                      "fp8_tflops": round(f / us8 / 1e6, 2), "bf16_tflops": round(f / us16 / 1e6, 2),
                      "fp8_over_bf16": round(us16 / us8, 3)}), flush=True)
    # QKV projection, M 8192
    S.compare("qkv_m8192", [(S.normal((8192, H)), S.normal((Q, H), 0.02), S.normal((8192, Q), 1e-3))], tensor, reps)
    # MLP: gate/up then down, outlier-channel activations
    S.compare("mlp_m8192", [(S.outliers((8192, H)), S.normal((2 * F, H), 0.02), S.normal((8192, 2 * F), 1e-3)),
                            (S.outliers((8192, F)), S.normal((H, F), 0.02), S.normal((8192, H), 1e-3))],
              tensor, reps)
    # LM head: Student-t(3) hidden states, dY = softmax(X W^T) - onehot(target)
    X, W = S.student_t3((8192, H)), S.normal((V, H), 0.02)
    tgt = torch.randint(0, V, (8192,), generator=S.gen, device=S.dev)
    dY = torch.empty(8192, V, dtype=torch.bfloat16, device=S.dev)
    Wf = W.float()
    for r0 in range(0, 8192, 1024):
        p = torch.softmax(torch.mm(X[r0:r0 + 1024].float(), Wf.t()), dim=1)
        p[torch.arange(p.shape[0], device=S.dev), tgt[r0:r0 + 1024]] -= 1.0
        dY[r0:r0 + 1024] = p.to(torch.bfloat16)
    del Wf, p
    S.compare("lm_head_m8192", [(X, W, dY)], tensor, reps)
    del X, W, dY
    torch.cuda.empty_cache()
    # 28 layers x (qkv, o, gate/up, down) at M 16384, blockwise E4M3 (one
    # weight set per layer; activations and gradients shared per linear kind)
    block = puro.LinearRecipe(E4, E4, E4, 1, puro.SCALE_POW2)
    acts = [(S.normal((16384, K)), S.normal((16384, N), 1e-3)) for _, N, K in inputs.LAYER_LINEARS]
    layers = [(acts[j][0], S.normal((N, K), 0.02), acts[j][1])
              for _ in range(inputs.LAYERS) for j, (_, N, K) in enumerate(inputs.LAYER_LINEARS)]
    S.compare("layers28_blockwise_m16384", layers, block, max(2, reps // 4))
    del layers, acts
    torch.cuda.empty_cache()
    # the paper's 1.7B shapes at M 8192, blockwise E4M3, both scale rules
    paper = [(S.outliers((8192, K)), S.normal((N, K), 0.02), S.normal((8192, N), 1e-3))
             for _, N, K in inputs.PAPER_LINEARS]
    for rnd, rule in ((puro.SCALE_POW2, "ceil"), (puro.SCALE_POW2_FLOOR, "floor_ocp_mx")):
        rc = puro.LinearRecipe(E4, E4, E4, 1, rnd)
        for (name, _, _), lin in zip(inputs.PAPER_LINEARS, paper):
            S.compare("paper_%s_m8192_%s" % (name, rule), [lin], rc, reps, S.errors(*lin, rc))
        S.compare("paper_layer_m8192_%s" % rule, paper, rc, reps)
    del paper
    torch.cuda.empty_cache()
    # the MLP's SwiGLU fused with the down projection's input quantisation,
    # and the RMSNorm fused with the QKV projection's
    # the BF16 epilogues: QKV's bias, the O projection's residual add (in place)
    for name, (M, N, K), bias, resid in (("qkv_fprop_bias_m8192", (8192, Q, H), True, False),
                                         ("o_fprop_residual_m8192", (8192, H, H), False, True)):
        xq = S.normal((M, K)).view(torch.uint8)[:, :K].contiguous() & 0x77      # finite E4M3 codes
        wq = S.normal((N, K)).view(torch.uint8)[:, :K].contiguous() & 0x77
        one = torch.ones(1, dtype=torch.float32, device=S.dev)
        A, B = puro.operand(xq, E4, puro.SCALE_TENSOR, one), puro.operand(wq, E4, puro.SCALE_TENSOR, one)
        b = S.normal((N,)) if bias else None
        r = S.normal((M, N)) if resid else None
        D = torch.empty(M, N, dtype=torch.bfloat16, device=S.dev)
        ws = torch.empty(max(1, puro.fp8_gemm_workspace_size(M, N, K, puro.OUT_BF16)), dtype=torch.uint8, device=S.dev)
        if resid:
            fused = lambda: puro.fp8_gemm_epilogue(A, M, B, N, K, residual=r, D=r, ws=ws)
            unfused = lambda: r.add_(puro.fp8_gemm(A, M, B, N, K, puro.OUT_BF16, D=D, ws=ws))
        else:
            fused = lambda: puro.fp8_gemm_epilogue(A, M, B, N, K, bias=b, D=D, ws=ws)
            unfused = lambda: puro.fp8_gemm(A, M, B, N, K, puro.OUT_BF16, D=D, ws=ws).add_(b)
        us_f, us_u = S.time_us(fused, 50), S.time_us(unfused, 50)
        print(json.dumps({"workload": name, "fused_us": round(us_f, 2), "unfused_us": round(us_u, 2),
                          "fused_over_unfused": round(us_u / us_f, 3),
                          "fused_tflops": round(2.0 * M * N * K / us_f / 1e6, 1)}), flush=True)
    work = dict(("mlp_%s_m8192" % k, v) for k, v in swiglu_workload(torch, puro).items())
    work.update(("qkv_input_%s_m8192" % k, v) for k, v in rmsnorm_workload(torch, puro).items())
    for name, (fused, unfused, nbytes) in work.items():
        us_f, us_u = S.time_us(fused, 50), S.time_us(unfused, 50)
        print(json.dumps({"workload": name, "fused_us": round(us_f, 2), "unfused_us": round(us_u, 2),
                          "fused_over_unfused": round(us_u / us_f, 3), "algorithmic_bytes": nbytes,
                          "fused_gbs": round(nbytes / us_f / 1e3, 1),
                          "fused_frac_hbm": round(nbytes / us_f / 1e3 / HBM_PEAK_GBS, 4)}), flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: this build measures the single-GPU share of the data-"
              "parallel path (every rank runs the same layer on its own tokens); --gpus %d is not "
              "supported" % args.gpus, file=sys.stderr)
        sys.exit(2)

    if args.suite:
        run_suite(args)
        return
    import numpy as np
    import torch
    from paper_2608_27370_amd import inputs, puro

    puro.lib()
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    M, K, N = args.tokens, inputs.HIDDEN, inputs.QKV_OUT
    d = inputs.qkv(M=M)

    def up(bits):
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
    # per-launch samples: each call bracketed by its own pair of events
    # (median, p10, p90), warm (back to back) and, with --cold, after a
    # 512 MiB fill that evicts the 256 MB MALL and the L2s
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev) if args.cold else None

    def sampled(fn, cold):
        for a, b in pairs:
            if cold:
                flush.zero_()
            a.record(stream)
            fn()
            b.record(stream)
        torch.cuda.synchronize()
        us = np.sort([a.elapsed_time(b) * 1e3 for a, b in pairs])
        return {k: round(float(np.percentile(us, q)), 2) for k, q in (("p10", 10), ("median", 50), ("p90", 90))}

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
        row = {"call": name, "us": round(us, 2), "launches": launches, "per_launch_us": sampled(fn, False)}
        if args.cold:
            row["cold_per_launch_us"] = sampled(fn, True)
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
