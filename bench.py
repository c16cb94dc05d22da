"""Throughput of the FP8 linear layers' hot path on one MI355X.

The default workload is one training step's linear layers of a 28-layer
Qwen2-1.5B-shaped transformer at M = 16384 tokens (one GPU's share: two of
the paper's 8192-token micro-batches): for every layer the QKV (2048 x
1536), O (1536 x 1536), fused gate/up (17920 x 1536) and down (1536 x 8960)
projections, forward in layer order and backward in reverse, with the
paper's blockwise recipe (Section 3.2): X and dY in 1x128 groups along each
GEMM's reduction dimension, W in 128x128 blocks, power-of-two scales, E4M3
throughout. A step is puro_linear_fwd for the 112 linears, then
puro_linear_bwd for them in reverse: amax and quantisation of every operand
and the Fprop, Dgrad and Wgrad GEMMs. Every layer has its own seeded
synthetic weights, activations and gradients (drawn on the device; weights
~N(0, 0.02^2), activations ~N(0, 1), gradients ~N(0, (1e-3)^2)), resident in
HBM before the timed region. ``--workload qkv`` times the per-tensor QKV
projection step (M 8192) instead; ``lm_head_bf16`` / ``lm_head_fp8`` the fused
LM head with its cross-entropy loss, forward and backward, at M 8192, V
151936, K 1536 (BF16 as the paper runs it, or the blockwise FP8 recipe);
``muonh28`` one MuonH optimiser step of the 28 layers' QKV, O, gate/up and down
matrices (Section 3.3), one call per kind.

Prints one JSON line: the metric (TFLOP/s of fwd + dgrad + wgrad GEMM work
per step time), the GEMM-only rate, a per-call breakdown (each kernel call
of one layer timed with HIP events on its stream over back-to-back launches,
and per launch as median / p10 / p90), a roofline entry for the dominant
kernel, the shader clock sampled during the timed region, and the CPU
oracle timed on a sample of the same workload.
"""

import argparse
import hashlib
import json
import os
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

FP8_PEAK_TFLOPS = 5000.0   # MI355X dense FP8 MFMA (256 CUs x 8192 FLOP/clk x 2.4 GHz)
PEAK_CLOCK_GHZ = 2.4
HBM_PEAK_GBS = 8000.0      # MI355X HBM3E
METRIC = "FP8 linear fwd+dgrad+wgrad TFLOP/s at Qwen2-1.5B shapes; % FP8 MFMA peak"
# the paper's mixed-precision MFU denominator (Section 3.1.3): 72% of the
# tensor-core work in FP8 at 419 TFLOP/s and 28% in BF16 at 209.5 on RTX 5090
PAPER_FP8_SHARE, PAPER_FP8_PEAK, PAPER_BF16_PEAK = 0.72, 419.0, 209.5
BF16_PEAK_TFLOPS = 2500.0  # MI355X dense BF16 MFMA


def p_eff(fp8_share, fp8_peak, bf16_peak):
    """Effective peak of a mixed FP8/BF16 workload (Section 3.1.3): the
    harmonic mix (fp8_share / fp8_peak + (1 - fp8_share) / bf16_peak)^-1,
    the rate at which that work would run with each part at its own peak."""
    return 1.0 / (fp8_share / fp8_peak + (1.0 - fp8_share) / bf16_peak)


WORKLOADS = ("layers28", "qkv", "lm_head_bf16", "lm_head_fp8", "muonh28")
DEFAULTS = {"layers28": (20, 3), "qkv": (1000, 50), "lm_head_bf16": (20, 3), "lm_head_fp8": (20, 3),
            "muonh28": (10, 2)}   # (steps, warmup)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--workload", choices=WORKLOADS, default="layers28",
                    help="layers28: the 28-layer blockwise step at M 16384 (default); "
                         "qkv: the per-tensor QKV projection step at M 8192; lm_head_bf16 / lm_head_fp8: the "
                         "fused LM head + cross-entropy at M 8192, V 151936; muonh28: one MuonH step of the "
                         "28 layers' matrices")
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=None)
    ap.add_argument("--cpu-tokens", type=int, default=None,
                    help="tokens per linear of the CPU oracle sample (0: skip)")
    ap.add_argument("--cold", action="store_true",
                    help="also time every call after a 512 MiB fill that evicts the MALL and the L2s "
                         "(kept out of the default run, whose kernel trace profiles warm launches)")
    ap.add_argument("--graph", action="store_true",
                    help="replay the step captured in a HIP graph instead of launching its kernels one by one")
    ap.add_argument("--suite", action="store_true",
                    help="instead of the headline step, time every workload (the five Qwen2-1.5B-shaped ones "
                         "and the paper's own 1.7B shapes under both power-of-two scale rules) next to the "
                         "same GEMMs in BF16, and report the FP8 errors of the two rules; one JSON line each")
    ap.add_argument("--only", default=None,
                    help="run just this call of the workload's breakdown (its key, e.g. gate_up.fprop), "
                         "'step', 'copy' (a plain 256 MiB device copy that calibrates the HBM byte counters) "
                         "or a fused call (%s) warmup + steps times and print its average time, for profilers"
                         % ", ".join(SWIGLU_CALLS + RMSNORM_CALLS))
    a = ap.parse_args()
    st, wu = DEFAULTS[a.workload]
    a.steps = st if a.steps is None else a.steps
    a.warmup = wu if a.warmup is None else a.warmup
    if a.cpu_tokens is None:
        a.cpu_tokens = {"layers28": 256, "qkv": 8192}.get(a.workload, 0)
    return a


def cpu_info():
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return model, os.cpu_count()


def cpu_baseline(workload, tokens):
    """The oracle (test infrastructure, unmodified) timed on a bounded sample
    of the workload: the linear layer's quantisation and its three FP64 GEMMs
    on the first `tokens` tokens; reported as TFLOP/s of the sampled GEMM
    work (the rate the oracle would sustain on the whole step)."""
    from oracle import linear
    from paper_2608_27370_amd import inputs
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    model, ncpu = cpu_info()
    flops = 0.0
    if workload == "layers28":
        rc = linear.recipe("block", dy_fmt="e4m3")
        data = [inputs.layer_linear(0, j, M=tokens) for j in range(len(inputs.LAYER_LINEARS))]
        t0 = time.perf_counter()
        for d in data:
            _, _, saved = linear.linear_fwd(d["X"], d["W"], rc)
            linear.linear_bwd(d["dY"], saved, rc)
            flops += 3 * 2.0 * tokens * d["W"].shape[0] * d["W"].shape[1]
        dt = time.perf_counter() - t0
        sample = ("oracle blockwise linear fwd+bwd of layer 0's four linears (qkv, o, gate/up, down) on the first "
                  "%d of the 16384 tokens: quantisation and FP64 GEMMs; the rate applies to the whole 28-layer "
                  "step, whose 128.8 TFLOP would take %.0f h at it" % (tokens, 0))
    else:
        d = inputs.qkv(M=tokens)
        rc = linear.recipe("tensor")
        t0 = time.perf_counter()
        _, _, saved = linear.linear_fwd(d["X"], d["W"], rc)
        linear.linear_bwd(d["dY"], saved, rc)
        dt = time.perf_counter() - t0
        flops = 3 * 2.0 * tokens * inputs.QKV_OUT * inputs.HIDDEN
        sample = "oracle per-tensor linear fwd+bwd on %d of the 8192 tokens of the QKV projection" % tokens
    value = flops / dt / 1e12
    if workload == "layers28":
        sample = sample.replace("take 0 h", "take %.0f h" % (128.8 / value / 3600.0))
    return {"value": value, "unit": "TFLOP/s", "cores": threads, "kind": "oracle", "seconds": round(dt, 2),
            "cpu_model": model, "nproc": ncpu, "sample": sample + "; FP64 GEMMs on %d OpenMP threads" % threads}


class ClockSampler:
    """The GFX clock sampled through amdsmi every few milliseconds while
    running: the mean over the XCDs of the metrics table's current GFX
    clocks, or (where the table has none) the clock-info reading; None when
    amdsmi is unavailable. The socket power is sampled beside it."""

    def __init__(self, period_s=0.005):
        self.samples, self.period, self._stop = [], period_s, threading.Event()
        self.power = []
        self.handle, self.source = None, None
        try:
            import amdsmi
            amdsmi.amdsmi_init()
            self.amdsmi = amdsmi
            self.handle = amdsmi.amdsmi_get_processor_handles()[0]
            self.read()
        except Exception:
            self.handle = None

    def read(self):
        try:
            m = self.amdsmi.amdsmi_get_gpu_metrics_info(self.handle)
            v = m.get("current_gfxclks")
            vals = [float(x) for x in v if isinstance(x, (int, float)) and 0 < x < 65535] if isinstance(v, list) else []
            if vals:
                self.source = "amdsmi metrics current_gfxclks, mean over %d XCDs" % len(vals)
                return sum(vals) / len(vals)
        except Exception:
            pass
        info = self.amdsmi.amdsmi_get_clock_info(self.handle, self.amdsmi.AmdSmiClkType.GFX)
        self.source = "amdsmi clock info GFX"
        return float(info["clk"])

    def read_power(self):
        try:
            info = self.amdsmi.amdsmi_get_power_info(self.handle)
            for k in ("current_socket_power", "average_socket_power", "socket_power"):
                v = info.get(k)
                if isinstance(v, (int, float)) and 0 < v < 65535:
                    return float(v)
        except Exception:
            pass
        return None

    def _run(self):
        while not self._stop.is_set():
            try:
                self.samples.append(self.read())
            except Exception:
                return
            w = self.read_power()
            if w is not None:
                self.power.append(w)
            time.sleep(self.period)

    def __enter__(self):
        if self.handle is not None:
            self.thread = threading.Thread(target=self._run, daemon=True)
            self.thread.start()
        return self

    def __exit__(self, *exc):
        if self.handle is not None:
            self._stop.set()
            self.thread.join()

    def summary(self):
        import numpy as np
        if not self.samples:
            return None
        s = np.array(self.samples)
        out = {"median_mhz": float(np.median(s)), "p10_mhz": float(np.percentile(s, 10)),
               "p90_mhz": float(np.percentile(s, 90)), "samples": int(s.size), "source": self.source}
        if self.power:
            out["median_socket_power_w"] = float(np.median(self.power))
        return out


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


class Call:
    """One kernel call of a step's breakdown: `count` times per step; `peak`
    is the MFMA peak its FLOPs are priced against."""

    def __init__(self, key, label, fn, flops=None, nbytes=None, launches=1, count=1, peak=FP8_PEAK_TFLOPS):
        self.key, self.label, self.fn = key, label, fn
        self.flops, self.nbytes, self.launches, self.count = flops, nbytes, launches, count
        self.peak = peak


class Layers28:
    """The 28-layer blockwise step at M = 16384 (see the module docstring)."""

    name = "layers28_blockwise_m16384"
    M = 16384

    def __init__(self, torch, puro, layers=None):
        from paper_2608_27370_amd import inputs
        self.torch, self.P, self.inputs = torch, puro, inputs
        nl = inputs.LAYERS if layers is None else layers
        P, M = puro, self.M
        dev = torch.device("cuda", 0)
        self.dev = dev
        self.rc = P.LinearRecipe(P.E4M3, P.E4M3, P.E4M3, 1, P.SCALE_POW2)
        gen = torch.Generator(device=dev)
        gen.manual_seed(4)

        def normal(shape, std):
            return (torch.randn(shape, generator=gen, device=dev) * std).to(torch.bfloat16)
        self.kinds = inputs.LAYER_LINEARS
        self.layers = []
        for _ in range(nl):
            row = []
            for name, N, K in self.kinds:
                row.append(dict(X=normal((M, K), 1.0), W=normal((N, K), 0.02), dY=normal((M, N), 1e-3),
                                saved=P.linear_saved(M, N, K, self.rc, dev)))
            self.layers.append(row)
        # outputs of one kind share their buffers across layers (overwritten)
        self.outs = [dict(Y=torch.empty(M, N, dtype=torch.bfloat16, device=dev),
                          dX=torch.empty(M, K, dtype=torch.bfloat16, device=dev),
                          dW=torch.empty(N, K, dtype=torch.float32, device=dev)) for _, N, K in self.kinds]
        self.wsf = torch.empty(max(P.linear_fwd_workspace_size(M, N, K, self.rc) for _, N, K in self.kinds),
                               dtype=torch.uint8, device=dev)
        self.wsb = torch.empty(max(P.linear_bwd_workspace_size(M, N, K, self.rc) for _, N, K in self.kinds),
                               dtype=torch.uint8, device=dev)
        self.gemm_flops = sum(3 * 2.0 * M * N * K for _, N, K in self.kinds) * nl
        # the dominant call, the gate/up Fprop, timed live inside the timed
        # steps: its layers' forward issues linear_fwd's own calls (the two
        # quantisations, then the GEMM on their operands) with events around
        # each GEMM
        self.live_key, self.live_kind = "gate_up.fprop", 2
        _, Nl, Kl = self.kinds[self.live_kind]
        E4, KM = P.E4M3, P.SCALE_KMAJOR
        self.ROW, self.BLK = P.SCALE_ROW_1x128 | KM, P.SCALE_BLOCK_128x128 | KM
        u8 = lambda *s: torch.empty(*s, dtype=torch.uint8, device=dev)
        f32 = lambda *s: torch.empty(*s, dtype=torch.float32, device=dev)
        self.lxq, self.lxs, self.lwq, self.lwb = u8(M, Kl), f32(Kl // 128, M), u8(Nl, Kl), f32(Kl // 128, Nl // 128)
        self.lgws = torch.empty(max(1, P.fp8_gemm_workspace_size(M, Nl, Kl, 0)), dtype=torch.uint8, device=dev)
        self.lqws = torch.empty(max(1, P.lib().puro_quantize_workspace_size(M, Kl),
                                    P.lib().puro_quantize_workspace_size(Nl, Kl)), dtype=torch.uint8, device=dev)
        self.live_flops = 2.0 * M * Nl * Kl
        self.config = {"workload": self.name, "layers": nl, "tokens": M,
                       "linears": {n: [N, K] for n, N, K in self.kinds},
                       "recipe": "blockwise: X, dY 1x128 groups along each GEMM's reduction dim, W 128x128 blocks, "
                                 "power-of-two scales, E4M3 throughout; BF16 Y/dX, FP32 dW"}

    def _live_fwd(self, lin, Y, ev):
        """The gate/up Fprop as puro_linear_fwd runs it (blockwise): X in 1x128
        rows with the 128x1 copy kept for Wgrad, W in 128x128 blocks with the
        transposed copy kept for Dgrad, then the GEMM, bracketed by `ev`."""
        P, sv = self.P, lin["saved"]
        _, N, K = self.kinds[self.live_kind]
        P.quantize_fp8(lin["X"], P.E4M3, self.ROW, P.SCALE_POW2, want_qT=True, ws=self.lqws,
                       out=dict(q=self.lxq, scale=self.lxs, qT=sv["xq_t"], scaleT=sv["x_scale"]))
        P.quantize_fp8(lin["W"], P.E4M3, self.BLK, P.SCALE_POW2, want_qT=True, ws=self.lqws,
                       out=dict(q=self.lwq, scale=self.lwb, qT=sv["wq_t"], scaleT=sv["w_scale"]))
        A = P.operand(self.lxq, P.E4M3, self.ROW, self.lxs)
        Bo = P.operand(self.lwq, P.E4M3, self.BLK, self.lwb)
        stream = self.torch.cuda.current_stream()
        ev[0].record(stream)
        P.fp8_gemm(A, self.M, Bo, N, K, P.OUT_BF16, D=Y, ws=self.lgws)
        ev[1].record(stream)

    def step(self, live=None):
        """One step; with `live` (a list of event pairs, one per layer) the
        gate/up Fprop GEMMs are bracketed by those events."""
        P = self.P
        for li, row in enumerate(self.layers):
            for j, lin in enumerate(row):
                if live is not None and j == self.live_kind:
                    self._live_fwd(lin, self.outs[j]["Y"], live[li])
                else:
                    P.linear_fwd(lin["X"], lin["W"], self.rc, Y=self.outs[j]["Y"], saved=lin["saved"], ws=self.wsf)
        for row in reversed(self.layers):
            for j in reversed(range(len(row))):
                lin, o = row[j], self.outs[j]
                P.linear_bwd(lin["dY"], lin["saved"], self.rc, lin["X"].shape[1], dX=o["dX"], dW=o["dW"],
                             ws=self.wsb)

    def calls(self):
        """The kernels of each linear kind (layer 0's tensors), called as the
        linear layer calls them: the same quantisers and GEMMs with the same
        k-block-major scale layouts; each occurs 28 times per step."""
        torch, P, M = self.torch, self.P, self.M
        E4, KM = P.E4M3, P.SCALE_KMAJOR
        ROW, BLK = P.SCALE_ROW_1x128 | KM, P.SCALE_BLOCK_128x128 | KM
        L = self.inputs.LAYERS       # each kind's calls occur once per layer of the step
        out = []
        for j, (name, N, K) in enumerate(self.kinds):
            lin, o = self.layers[0][j], self.outs[j]
            sv, dev = lin["saved"], self.dev
            u8 = lambda *s: torch.empty(*s, dtype=torch.uint8, device=dev)
            f32 = lambda *s: torch.empty(*s, dtype=torch.float32, device=dev)
            xq, xs = u8(M, K), f32(K // 128, M)
            wq, wb = u8(N, K), f32(K // 128, N // 128)
            dyq, dys, dyqT, dysT = u8(M, N), f32(N // 128, M), u8(N, M), f32(M // 128, N)
            gws = torch.empty(max(1, P.fp8_gemm_workspace_size(M, N, K, 0), P.fp8_gemm_workspace_size(M, K, N, 0),
                                  P.fp8_gemm_workspace_size(N, K, M, 1)), dtype=torch.uint8, device=dev)
            A_f, B_f = P.operand(xq, E4, ROW, xs), P.operand(wq, E4, BLK, wb)
            A_d, B_d = P.operand(dyq, E4, ROW, dys), P.operand(sv["wq_t"], E4, BLK, sv["w_scale"])
            A_w, B_w = P.operand(dyqT, E4, ROW, dysT), P.operand(sv["xq_t"], E4, ROW, sv["x_scale"])
            X, W, dY = lin["X"], lin["W"], lin["dY"]
            grp = 2.0 * 4 / 128          # two scale arrays of 4 B per 128 elements
            fl = 2.0 * M * N * K

            def q(x, mode, o_):
                return lambda: P.quantize_fp8(x, E4, mode, P.SCALE_POW2, want_qT=True, out=o_)

            def gemm(A, m, B, n, k, kind, D, w):
                return lambda: P.fp8_gemm(A, m, B, n, k, kind, D=D, ws=w)
            plan = lambda m, n, k: P.fp8_gemm_plan(m, n, k, P.SCALE_ROW_1x128, P.SCALE_BLOCK_128x128)["launches"]
            planw = lambda m, n, k: P.fp8_gemm_plan(m, n, k, P.SCALE_ROW_1x128, P.SCALE_ROW_1x128)["launches"]
            out += [
                Call(name + ".quantize_x", "%s: quantize X [%d,%d] (1x128 rows + 128x1 columns, one read)" % (name, M, K),
                     q(X, ROW, dict(q=xq, scale=xs, qT=sv["xq_t"], scaleT=sv["x_scale"])),
                     nbytes=M * K * (4.0 + grp), count=L),
                Call(name + ".quantize_w", "%s: quantize W [%d,%d] (128x128 blocks + transposed copy)" % (name, N, K),
                     q(W, BLK, dict(q=wq, scale=wb, qT=sv["wq_t"], scaleT=sv["w_scale"])),
                     nbytes=N * K * 4.0, count=L),
                Call(name + ".fprop", "%s: fprop GEMM %dx%dx%d" % (name, M, N, K),
                     gemm(A_f, M, B_f, N, K, P.OUT_BF16, o["Y"], gws),
                     flops=fl, launches=plan(M, N, K), count=L),
                Call(name + ".quantize_dy", "%s: quantize dY [%d,%d] (1x128 rows + 128x1 columns, one read)" % (name, M, N),
                     q(dY, ROW, dict(q=dyq, scale=dys, qT=dyqT, scaleT=dysT)), nbytes=M * N * (4.0 + grp), count=L),
                Call(name + ".dgrad", "%s: dgrad GEMM %dx%dx%d" % (name, M, K, N),
                     gemm(A_d, M, B_d, K, N, P.OUT_BF16, o["dX"], gws),
                     flops=fl, launches=plan(M, K, N), count=L),
                Call(name + ".wgrad", "%s: wgrad GEMM %dx%dx%d" % (name, N, K, M),
                     gemm(A_w, N, B_w, K, M, P.OUT_FP32, o["dW"], gws),
                     flops=fl, launches=planw(N, K, M), count=L),
            ]
        return out


class Qkv:
    """The per-tensor QKV projection step at M = 8192 (X, W E4M3; dY E5M2)."""

    name = "qkv_projection_fwd_dgrad_wgrad"

    def __init__(self, torch, puro, M=8192):
        import numpy as np
        from paper_2608_27370_amd import inputs
        self.torch, self.P = torch, puro
        dev = torch.device("cuda", 0)
        self.dev = dev
        self.M, self.K, self.N = M, inputs.HIDDEN, inputs.QKV_OUT
        d = inputs.qkv(M=M)

        def up(bits):
            return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)
        self.X, self.W, self.dY = up(d["X"]), up(d["W"]), up(d["dY"])
        P, M, K, N = puro, self.M, self.K, self.N
        self.rc = P.LinearRecipe(P.E4M3, P.E4M3, P.E5M2, 0, P.SCALE_FP32)
        self.saved = P.linear_saved(M, N, K, self.rc, dev)
        self.Y = torch.empty(M, N, dtype=torch.bfloat16, device=dev)
        self.dX = torch.empty(M, K, dtype=torch.bfloat16, device=dev)
        self.dW = torch.empty(N, K, dtype=torch.float32, device=dev)
        self.wsf = torch.empty(max(1, P.linear_fwd_workspace_size(M, N, K, self.rc)), dtype=torch.uint8, device=dev)
        self.wsb = torch.empty(max(1, P.linear_bwd_workspace_size(M, N, K, self.rc)), dtype=torch.uint8, device=dev)
        self.gemm_flops = 3 * 2.0 * M * N * K
        self.config = {"workload": self.name, "M": M, "K": K, "N": N,
                       "recipe": "per-tensor scales, X/W E4M3, dY E5M2, BF16 Y/dX, FP32 dW"}

    def step(self):
        P = self.P
        P.linear_fwd(self.X, self.W, self.rc, Y=self.Y, saved=self.saved, ws=self.wsf)
        P.linear_bwd(self.dY, self.saved, self.rc, self.K, dX=self.dX, dW=self.dW, ws=self.wsb)

    def calls(self):
        torch, P, M, N, K, dev = self.torch, self.P, self.M, self.N, self.K, self.dev
        xq = torch.empty(M, K, dtype=torch.uint8, device=dev)
        wq = torch.empty(N, K, dtype=torch.uint8, device=dev)
        dyq = torch.empty(M, N, dtype=torch.uint8, device=dev)
        dyqT = torch.empty(N, M, dtype=torch.uint8, device=dev)
        sx, sw, sdy = (torch.empty(1, dtype=torch.float32, device=dev) for _ in range(3))
        qws = torch.empty(max(1, P.lib().puro_quantize_workspace_size(M, N)), dtype=torch.uint8, device=dev)
        gws = torch.empty(max(1, P.fp8_gemm_workspace_size(M, N, K, 0), P.fp8_gemm_workspace_size(M, K, N, 0),
                              P.fp8_gemm_workspace_size(N, K, M, 1)), dtype=torch.uint8, device=dev)
        sv = self.saved
        A_f, B_f = P.operand(xq, P.E4M3, P.SCALE_TENSOR, sx), P.operand(wq, P.E4M3, P.SCALE_TENSOR, sw)
        A_d, B_d = P.operand(dyq, P.E5M2, P.SCALE_TENSOR, sdy), P.operand(sv["wq_t"], P.E4M3, P.SCALE_TENSOR, sw)
        A_w, B_w = P.operand(dyqT, P.E5M2, P.SCALE_TENSOR, sdy), P.operand(sv["xq_t"], P.E4M3, P.SCALE_TENSOR, sx)
        fl = 2.0 * M * N * K
        # quantisation moves 2 B read + 1 B (q) + 1 B (qT) written per element
        return [
            Call("quantize_x", "quantize X (amax + encode, q and qT)", lambda: P.quantize_fp8(
                self.X, P.E4M3, out=dict(q=xq, scale=sx, qT=sv["xq_t"]), want_qT=True, ws=qws),
                nbytes=M * K * 4.0, launches=2),
            Call("quantize_w", "quantize W (amax + encode, q and qT)", lambda: P.quantize_fp8(
                self.W, P.E4M3, out=dict(q=wq, scale=sw, qT=sv["wq_t"]), want_qT=True, ws=qws),
                nbytes=N * K * 4.0, launches=2),
            Call("fprop", "fprop GEMM %dx%dx%d" % (M, N, K),
                 lambda: P.fp8_gemm(A_f, M, B_f, N, K, P.OUT_BF16, D=self.Y, ws=gws), flops=fl,
                 launches=P.fp8_gemm_plan(M, N, K)["launches"]),
            Call("quantize_dy", "quantize dY (amax + encode, q and qT)", lambda: P.quantize_fp8(
                self.dY, P.E5M2, out=dict(q=dyq, scale=sdy, qT=dyqT), want_qT=True, ws=qws),
                nbytes=M * N * 4.0, launches=2),
            Call("dgrad", "dgrad GEMM %dx%dx%d" % (M, K, N),
                 lambda: P.fp8_gemm(A_d, M, B_d, K, N, P.OUT_BF16, D=self.dX, ws=gws), flops=fl,
                 launches=P.fp8_gemm_plan(M, K, N)["launches"]),
            Call("wgrad", "wgrad GEMM %dx%dx%d" % (N, K, M),
                 lambda: P.fp8_gemm(A_w, N, B_w, K, M, P.OUT_FP32, D=self.dW, ws=gws), flops=fl,
                 launches=P.fp8_gemm_plan(N, K, M)["launches"]),
        ]


class LmHead:
    """The fused LM head + cross-entropy at M 8192 tokens, V 151936, K 1536:
    forward (lse and loss) then backward (dX, dW) per step. X ~ Student-t(3),
    W ~ N(0, 0.02^2), targets uniform, drawn on the device. The algorithmic
    work is the three GEMMs' 6 M V K; the backward recomputes the logits (2 M V
    K more), which the rate does not count."""

    def __init__(self, torch, puro, recipe, M=8192):
        from paper_2608_27370_amd import inputs
        self.torch, self.P = torch, puro
        dev = torch.device("cuda", 0)
        self.dev = dev
        self.M, self.V, self.K = M, inputs.VOCAB, inputs.HIDDEN
        self.recipe = recipe
        gen = torch.Generator(device=dev)
        gen.manual_seed(5)
        M, V, K = self.M, self.V, self.K
        chi = torch.randn(M, K, 3, generator=gen, device=dev).square().sum(-1) / 3.0
        self.X = (torch.randn(M, K, generator=gen, device=dev) / chi.sqrt()).to(torch.bfloat16)
        self.W = (torch.randn(V, K, generator=gen, device=dev) * 0.02).to(torch.bfloat16)
        self.t = torch.randint(0, V, (M,), generator=gen, device=dev, dtype=torch.int32)
        self.lse = torch.empty(M, dtype=torch.float32, device=dev)
        self.loss = torch.empty(M, dtype=torch.float32, device=dev)
        self.dX = torch.empty(M, K, dtype=torch.bfloat16, device=dev)
        self.dW = torch.empty(V, K, dtype=torch.float32, device=dev)
        self.wsf = torch.empty(puro.lm_head_ce_workspace_size(M, V, K, recipe, False), dtype=torch.uint8, device=dev)
        self.wsb = torch.empty(puro.lm_head_ce_workspace_size(M, V, K, recipe, True), dtype=torch.uint8, device=dev)
        fp8 = recipe == puro.LM_HEAD_FP8
        self.name = "lm_head_ce_%s_m%d_v%d" % ("fp8" if fp8 else "bf16", M, V)
        self.flops = 6.0 * M * V * K
        self.peak = FP8_PEAK_TFLOPS if fp8 else BF16_PEAK_TFLOPS
        self.dtype = "fp8" if fp8 else "bf16"
        self.metric = "LM head + cross-entropy fwd+bwd TFLOP/s (6 M V K per step) at Qwen2-1.5B shapes"
        self.config = {"workload": self.name, "tokens": M, "vocab": V, "hidden": K,
                       "recipe": ("blockwise FP8: X 1x128 rows / 128x1 columns, W 128x128 blocks, dz BF16 then "
                                  "1x128 + 128x1, E4M3, power-of-two scales" if fp8 else
                                  "BF16 operands, binary32 accumulation, dz BF16"),
                       "logits": "never stored: forward reduces them to (max, sum exp) per 128-column block in "
                                 "the GEMM epilogue; backward recomputes them per 8192-column chunk"}

    def step(self):
        P = self.P
        P.lm_head_ce_fwd(self.X, self.W, self.t, self.recipe, lse=self.lse, loss=self.loss, ws=self.wsf)
        P.lm_head_ce_bwd(self.X, self.W, self.t, self.lse, self.recipe, grad_scale=1.0 / self.M, dX=self.dX,
                         dW=self.dW, ws=self.wsb)

    def calls(self):
        P, M, V, K = self.P, self.M, self.V, self.K
        fl = 2.0 * M * V * K
        return [
            Call("fwd", "forward: logits GEMM with the (max, sum exp) epilogue, lse per row%s" %
                 (", X and W quantised" if self.dtype == "fp8" else ""),
                 lambda: P.lm_head_ce_fwd(self.X, self.W, self.t, self.recipe, lse=self.lse, loss=self.loss,
                                          ws=self.wsf), flops=fl, launches=0, peak=self.peak),
            Call("bwd", "backward: per 8192-column chunk the logits GEMM with the softmax-gradient epilogue, "
                 "then dX and dW GEMMs (4 M V K executed, 4 M V K counted)",
                 lambda: P.lm_head_ce_bwd(self.X, self.W, self.t, self.lse, self.recipe, grad_scale=1.0 / M,
                                          dX=self.dX, dW=self.dW, ws=self.wsb), flops=2 * fl, launches=0,
                 peak=self.peak),
        ]


class MuonH28:
    """One MuonH step (Section 3.3) of the 28 layers' wrapped matrices: per
    kind (QKV 2048x1536, O 1536x1536, gate/up 17920x1536, down 1536x8960) one
    call on the 28 matrices stored back to back (FP32 W, G, momentum; W ~
    N(0, 0.02^2), G and momentum ~ N(0, (1e-3)^2), drawn on the device). The
    algorithmic work is the Newton-Schulz products counted dense: per matrix
    and step (r <= c its oriented shape) 2 r^2 c for X X^T, 2 r^3 for A A^T,
    2 r^2 c for B X, five steps. The two symmetric products compute only the
    tiles on or above the diagonal; the executed work is reported beside."""

    name = "muonh_28_layers_qwen2_1p5b"

    def __init__(self, torch, puro):
        from paper_2608_27370_amd import inputs
        self.torch, self.P = torch, puro
        dev = torch.device("cuda", 0)
        self.dev = dev
        gen = torch.Generator(device=dev)
        gen.manual_seed(7)
        L = inputs.LAYERS
        self.kinds = inputs.LAYER_LINEARS
        self.mats = []
        self.flops = 0.0
        for name, rows, cols in self.kinds:
            W = torch.randn(L, rows, cols, generator=gen, device=dev) * 0.02
            G = torch.randn(L, rows, cols, generator=gen, device=dev) * 1e-3
            buf = torch.randn(L, rows, cols, generator=gen, device=dev) * 1e-3
            R = torch.linalg.vector_norm(W.double(), dim=(1, 2)).float()
            wb = torch.empty(L, rows, cols, dtype=torch.bfloat16, device=dev)
            ws = torch.empty(puro.lib().puro_muonh_workspace_size(L, rows, cols), dtype=torch.uint8, device=dev)
            r, c = min(rows, cols), max(rows, cols)
            fl = L * 5 * (4.0 * r * r * c + 2.0 * r ** 3)
            self.flops += fl
            t = -(-r // 256)                     # 256-wide tiles of the symmetric products
            sym = t * (t + 1) / 2.0 / (t * t)    # the share of their tiles computed
            self.executed_flops = getattr(self, "executed_flops", 0.0) + L * 5 * (
                2.0 * r * r * c * sym + 2.0 * r ** 3 * sym + 2.0 * r * r * c)
            self.mats.append(dict(name=name, W=W, G=G, buf=buf, R=R, wb=wb, ws=ws, flops=fl, shape=(rows, cols)))
        self.peak = BF16_PEAK_TFLOPS
        self.dtype = "bf16"
        self.metric = ("MuonH optimiser step: Newton-Schulz TFLOP/s over the 28 layers' matrices, dense-equivalent "
                       "(BF16 MFMA)")
        self.config = {"workload": self.name, "layers": L, "matrices": {n: [r, c] for n, r, c in self.kinds},
                       "newton_schulz": "5 quintic steps in BF16, (a, b, c) = (3.4445, -4.7750, 2.0315)",
                       "state": "FP32 W, G, momentum (mu 0.95, Nesterov); BF16 copy of W' written",
                       "flops_counted_per_step": self.flops, "flops_executed_per_step": self.executed_flops,
                       "symmetric_products": "X X^T and b A + c A A^T: only the tiles on or above the diagonal, "
                                             "then mirrored"}

    def _call(self, m):
        P = self.P
        return lambda: P.muonh_step(m["W"], m["G"], m["buf"], m["R"], 1e-3, w_bf16=m["wb"], ws=m["ws"])

    def step(self):
        for m in self.mats:
            self._call(m)()

    def calls(self):
        out = []
        for m in self.mats:
            rows, cols = m["shape"]
            out.append(Call(m["name"], "%s: MuonH step of 28 [%d,%d] matrices (momentum, 5 Newton-Schulz steps of "
                            "3 batched BF16 GEMMs + transpose, hyperball)" % (m["name"], rows, cols),
                            self._call(m), flops=m["flops"], launches=0, peak=BF16_PEAK_TFLOPS))
        return out


COPY_BYTES = 256 << 20


def profiled(workload, key, field):
    """A per-launch figure (`field`: "bytes" = HBM-side bytes from rocprofv3
    FETCH_SIZE / WRITE_SIZE scaled by the copy calibration) of call `key`,
    from the committed summary profiles/hbm_bytes_<workload>.md; None when it
    is missing or any source it was measured on has changed since."""
    try:
        text = open(os.path.join(ROOT, "profiles", "hbm_bytes_%s.md" % workload)).read()
        d = json.loads(text.split("```json", 1)[1].split("```", 1)[0])
        for path, digest in d["sources"].items():
            if hashlib.sha256(open(os.path.join(ROOT, path), "rb").read()).hexdigest() != digest:
                return None
        return d["calls"][key][field]
    except (OSError, IndexError, KeyError, ValueError):
        return None


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


def run_only(args, torch, W):
    """Profiling mode: one call (or the whole step) warmup + steps times."""
    stream = torch.cuda.current_stream()
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
        fn, label = W.step, "%s step" % W.name
    else:
        rows = [c for c in W.calls() if c.key == args.only]
        if not rows:
            sys.exit("unknown --only %r; calls of %s: %s" % (args.only, W.name,
                                                             ", ".join(c.key for c in W.calls())))
        fn, label = rows[0].fn, rows[0].label
        # the call's operands are what the kind's earlier calls write (its
        # quantisations): run every call of the kind once, in order, first
        kind = args.only.split(".")[0]
        for c in W.calls():
            if c.key.split(".")[0] == kind:
                c.fn()
    for _ in range(args.warmup):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with ClockSampler() as clock:
        e0.record(stream)
        for _ in range(args.steps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
    print(json.dumps({"only": args.only, "call": label, "launches": args.steps,
                      "us_per_call": round(e0.elapsed_time(e1) / max(1, args.steps) * 1e3, 2),
                      "clock": clock.summary()}), flush=True)


def breakdown(args, torch, W, stream):
    """Each call of the workload timed on the stream it runs on: back-to-back
    launches between two events (the mean), and each launch bracketed by its
    own events (median, p10, p90), warm and with --cold after a 512 MiB fill
    that evicts the 256 MB MALL and the L2s."""
    import numpy as np
    calls = W.calls()
    reps = 20
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=W.dev) if args.cold else None

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
    rows = []
    for c in calls:
        for _ in range(3):
            c.fn()
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(reps):
            c.fn()
        e1.record(stream)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / reps * 1e3
        row = {"call": c.label, "key": c.key, "us": round(us, 2), "per_step": c.count,
               "launches": c.launches, "per_launch_us": sampled(c.fn, False)}
        if args.cold:
            row["cold_per_launch_us"] = sampled(c.fn, True)
        if c.flops:
            row["tflops"] = round(c.flops / (us * 1e-6) / 1e12, 1)
            row["frac_%s_peak" % ("fp8" if c.peak == FP8_PEAK_TFLOPS else "bf16")] = round(
                c.flops / (us * 1e-6) / 1e12 / c.peak, 4)
        if c.nbytes:
            row["gbs_algorithmic"] = round(c.nbytes / (us * 1e-6) / 1e9, 1)
            row["frac_hbm_peak"] = round(c.nbytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)
        rows.append(row)
    return calls, rows


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: it measures the single-GPU share of the data-"
              "parallel path (every rank runs the same layers on its own tokens); --gpus %d is not "
              "supported" % args.gpus, file=sys.stderr)
        sys.exit(2)
    if args.suite:
        run_suite(args)
        return
    import torch
    from paper_2608_27370_amd import puro

    puro.lib()
    torch.cuda.set_device(0)
    if args.workload == "layers28":
        # a single call profiles layer 0's tensors; a step needs every layer
        W = Layers28(torch, puro, layers=1 if args.only and args.only != "step" else None)
    elif args.workload == "qkv":
        W = Qkv(torch, puro)
    elif args.workload.startswith("lm_head"):
        W = LmHead(torch, puro, puro.LM_HEAD_FP8 if args.workload == "lm_head_fp8" else puro.LM_HEAD_BF16)
    else:
        W = MuonH28(torch, puro)
    flops = getattr(W, "flops", None) or W.gemm_flops
    peak = getattr(W, "peak", FP8_PEAK_TFLOPS)
    dtype = getattr(W, "dtype", "fp8")
    if args.only:
        run_only(args, torch, W)
        return
    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        W.step()
    torch.cuda.synchronize()
    run = W.step
    if args.graph:
        # the step's launches captured once in a HIP graph and replayed
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            W.step()
        stream.wait_stream(side)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            W.step()
        run = graph.replay
        for _ in range(args.warmup):
            run()
        torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    live = None
    if hasattr(W, "live_key") and not args.graph:
        mk = lambda: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
        live = [[mk() for _ in W.layers] for _ in range(args.steps)]
    with ClockSampler() as clock:
        t0 = time.perf_counter()
        e0.record(stream)
        for si in range(args.steps):
            if live is not None:
                W.step(live[si])
            else:
                run()
        e1.record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
    ms_per_step = e0.elapsed_time(e1) / args.steps
    value = flops / (ms_per_step * 1e-3) / 1e12

    calls, rows = breakdown(args, torch, W, stream)
    gemm_us = sum(r["us"] * r["per_step"] for r in rows if "tflops" in r)
    sum_us = sum(r["us"] * r["per_step"] for r in rows)
    # dominant kernel: the single-launch call with the largest share of a step
    # (workloads whose calls are entry points of several kernels: the call)
    single = [(r, c) for r, c in zip(rows, calls) if c.launches == 1] or list(zip(rows, calls))
    dom, dom_c = max(single, key=lambda rc: rc[0]["us"] * rc[0]["per_step"])
    if "tflops" in dom:
        roofline = {"bound": "mfma", "kernel": dom["call"], "achieved": dom["tflops"], "peak": dom_c.peak,
                    "unit": "TFLOP/s", "frac": round(dom["tflops"] / dom_c.peak, 4),
                    "algorithmic_flops_per_launch": dom_c.flops}
        if dom_c.launches != 1:
            roofline["note"] = "an entry point of several kernels; its kernels' own times are in the profiles"
    else:
        roofline = {"bound": "hbm", "kernel": dom["call"], "achieved": dom["gbs_algorithmic"], "peak": HBM_PEAK_GBS,
                    "unit": "GB/s", "frac": round(dom["gbs_algorithmic"] / HBM_PEAK_GBS, 4),
                    "algorithmic_bytes_per_launch": dom_c.nbytes}
    roofline["us_per_launch"] = dom["us"]
    if live is not None and dom_c.key == W.live_key:
        # the dominant kernel's own launches inside the timed steps
        import numpy as np
        us = np.array([a.elapsed_time(b) * 1e3 for st in live for a, b in st])
        ach = W.live_flops / (us.mean() * 1e-6) / 1e12
        roofline.update({"achieved": round(ach, 1), "frac": round(ach / dom_c.peak, 4),
                         "us_per_launch": round(float(us.mean()), 2),
                         "timing": "HIP events around each of the call's %d launches inside the timed steps "
                                   "(median %.2f us, p10 %.2f, p90 %.2f); the breakdown's back-to-back figure is "
                                   "%.2f us" % (us.size, np.median(us), np.percentile(us, 10), np.percentile(us, 90),
                                                dom["us"])})
    roofline["share_of_step"] = round(roofline["us_per_launch"] * dom["per_step"] / (ms_per_step * 1e3), 4)
    roofline["traffic"] = profiled(args.workload, dom_c.key, "bytes")
    roofline["traffic_unit"] = "HBM-side bytes per launch (rocprofv3 FETCH_SIZE + WRITE_SIZE, copy-calibrated)"
    clk = clock.summary()
    out = {
        "metric": getattr(W, "metric", METRIC),
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dtype,
        "data": "synthetic",
        "config": dict(W.config, launch="hip_graph" if args.graph else "eager"),
        "pct_%s_peak" % dtype: round(100 * value / peak, 2),
        "gemm_only_tflops": round(flops / (gemm_us * 1e-6) / 1e12, 1),
        "gemm_only_pct_%s_peak" % dtype: round(100 * flops / (gemm_us * 1e-6) / 1e12 / peak, 2),
        "breakdown_sum_ms": round(sum_us / 1e3, 3),
        "breakdown": rows,
        "roofline": roofline,
        "clock": clk,
        "wall_s_timed": round(wall, 3),
        "mfu_context": {"paper_p_eff_tflops": round(p_eff(PAPER_FP8_SHARE, PAPER_FP8_PEAK, PAPER_BF16_PEAK), 2),
                        "mi355x_p_eff_tflops_at_paper_mix": round(p_eff(PAPER_FP8_SHARE, FP8_PEAK_TFLOPS,
                                                                        BF16_PEAK_TFLOPS), 1),
                        "fp8_share_of_this_step": 1.0 if dtype == "fp8" else 0.0},
    }
    if clk:
        ghz = clk["median_mhz"] / 1e3
        out["pct_%s_peak_at_measured_clock" % dtype] = round(100 * value / (peak * ghz / PEAK_CLOCK_GHZ), 2)
    if args.cpu_tokens > 0:
        out["cpu_baseline"] = cpu_baseline(args.workload, args.cpu_tokens)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
