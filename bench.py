"""Benchmark of the DynamicPTQ quantized linear layer on one MI355X.

Headline workload (one "step"): every linear of the LLaMA-2-70B stack, 80
layers x (fused QKV 8192 -> 10240, o 8192 -> 8192, gate/up 8192 -> 57344,
down 28672 -> 8192 with the 28 x 1024 Hadamard), at M = 4096 prefill tokens.
The per-layer activation precision comes from the policy (Eq. 21, Algorithm 1
step 2) under a seeded mixed mask (4 of 80 layers at 8 bits).  Each linear
runs rotate+quantize then the GEMM with its dequant epilogue: a 4-bit layer
on the FP6 matrix cores (codes written straight into the FP6 operand layout,
weights pre-packed into it once), an 8-bit layer on the int8 matrix cores
(weights pre-packed into the 8-bit activation order once).  Both return the
oracle's results bit for bit.  Weights are N(0, 0.02) fp32 drawn on the device
(seeded), quantized to 4 bits per output channel by the library and resident
in HBM (34 GB of packed codes, 85 GB with the device-native layouts); each
linear's activations are the seeded fp16 input of that linear in the stack
(N(0,1) with outlier channels; Student-t(3) for the down projection).

    python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--extended]

Prints one JSON line.  value = total integer ops (2 M N K per linear) of a
step / wall time per step, in TOPS.  The other workloads (the tiny layer, the
LLaMA-2-7B QKV layer, the LLaMA-3-8B down projection at decode and prefill
sizes, the LLaMA-2-7B 32-layer stack, the 70B stack at M = 8 decode) are
reported under "configs", timed by graph-replayed launches.
"""

import argparse
import json
import os
import sys
import threading
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_INT8_TOPS = 5000.0      # MI355X dense int8 MFMA, T ops/s
PEAK_FP6_TOPS = 10100.0      # MI355X dense fp6 / fp4 MFMA, T ops/s
PEAK_HBM_GBS = 8000.0        # MI355X HBM3E, GB/s
# fp32 vector issue without packed instructions (the kernels are built without
# them): 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz lane-operations per second.
PEAK_LANE_OPS = 256 * 4 * 16 * 2.4e9
METRIC = "W4A4/W4A8 qlinear TOPS (rotate+quant+GEMM), % int8 MFMA peak; decode GB/s"
HEADLINE = "llama2_70b_layer"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_qgemm_fp6_llama2_70b_stack.txt")
TRAFFIC_SOURCE = os.path.join(ROOT, "paper_2606_12487_amd", "csrc", "qgemm_fp6.hip")
DECODE_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_qgemm_decode_llama2_70b_M8.txt")
DECODE_TRAFFIC_SOURCE = os.path.join(ROOT, "paper_2606_12487_amd", "csrc", "qgemm.hip")


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-workers", type=int, default=0,
                   help="worker processes of the CPU oracle baseline (0: affinity count, at most 16)")
    p.add_argument("--no-configs", action="store_true",
                   help="time only the headline stack (no other workloads)")
    p.add_argument("--extended", action="store_true",
                   help="also time the fused decode paths, the range quantizer, calibration and KV4")
    p.add_argument("--only", choices=["rq6", "gemm6", "rq8", "gemm8", "copy", "decode"],
                   help="launch one kernel family of the headline step --steps times at every "
                        "linear shape, nothing timed (for counter runs); copy: a 256 MiB device copy")
    return p.parse_args()


# ---------------------------------------------------------------------------
# helpers
# ---------------------------------------------------------------------------
def progress(msg):
    """One line on stderr per finished phase (the JSON line alone goes to stdout)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def source_digest(path):
    import hashlib
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def measured_traffic(path=None, source=None, key="hbm_bytes_per_launch"):
    """A figure of a committed counter summary (by default the mean HBM bytes
    per launch of the headline's FP6 GEMM), or None when the file is missing or
    was taken on other sources of the kernel."""
    path = path or TRAFFIC_FILE
    source = source or TRAFFIC_SOURCE
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("source_sha256_16") != source_digest(source):
        return None
    try:
        return float(kv[key]) if key == "traffic_over_algorithmic" else int(float(kv[key]))
    except (KeyError, ValueError):
        return None


class ClockSampler:
    """sclk / mclk read from the GPU's metrics table every ~20 ms on a thread
    while the timed steps run (MHz)."""

    def __init__(self):
        self.samples, self.error = [], None
        self._stop = threading.Event()
        self._t = None

    def __enter__(self):
        self._t = threading.Thread(target=self._run, daemon=True)
        self._t.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        self._t.join(timeout=5)

    def _run(self):
        try:
            import amdsmi
            amdsmi.amdsmi_init()
            try:
                h = amdsmi.amdsmi_get_processor_handles()[0]
                while not self._stop.is_set():
                    m = amdsmi.amdsmi_get_gpu_metrics_info(h)
                    self.samples.append((m.get("current_gfxclk"), m.get("average_gfxclk_frequency"),
                                         m.get("current_uclk")))
                    time.sleep(0.02)
            finally:
                amdsmi.amdsmi_shut_down()
        except Exception as e:  # no metrics on this machine: reported, not fatal
            self.error = repr(e)[:200]

    def summary(self):
        def col(i):
            v = [s[i] for s in self.samples if isinstance(s[i], (int, float))]
            return {"mean": round(sum(v) / len(v), 1), "min": min(v), "max": max(v)} if v else None
        return {"samples": len(self.samples), "sclk_current_mhz": col(0),
                "sclk_average_mhz": col(1), "mclk_mhz": col(2), "error": self.error}


def graph_time(torch, fns, reps=5):
    """Microseconds per call of a sequence of launches, captured once in a HIP
    graph and replayed `reps` times between two HIP events on the launch
    stream (no host launch gaps)."""
    for f in fns:
        f()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    with torch.cuda.graph(g, stream=s):
        for f in fns:
            f()
    g.replay()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / (reps * len(fns))
    del g
    return us


def k1_essential_ops(h, fp6=False):
    """Vector lane-operations per element rotate+quantize cannot avoid: log2 of
    the power-of-two factor in butterflies, 27 additions of the 28-point stage
    when h = 28 * 2^j (its pinned sequential order), 6 for widening, absmax,
    the corrected quotient (multiply, two FMAs), rounding and packing, and 2
    more for the FP6 operand (c / 2 and its fp16 conversion)."""
    f28 = h % 28 == 0
    p = h // 28 if f28 else h
    return p.bit_length() - 1 + (27 if f28 else 0) + 6 + (2 if fp6 else 0)


def k1_bytes(M, K, bits):
    """Algorithmic bytes of rotate+quantize: fp16 rows in, codes and scales out."""
    return 2 * M * K + M * K * bits // 8 + 4 * M


def gemm_bytes(M, K, N, bits):
    """Algorithmic bytes of the GEMM: codes, 4-bit weights, scales and fp16 y."""
    return M * K * bits // 8 + N * K // 2 + 4 * (M + N) + 2 * M * N


# ---------------------------------------------------------------------------
# the headline stack
# ---------------------------------------------------------------------------
class Stack:
    """Every linear of a layer stack with its own weights on the device.

    Weights: N(0, 0.02) fp32 drawn on the device per (layer, linear) with a
    seeded generator, quantized by dptq.prepare_weights (Eq. 5, per-channel
    4-bit) and pre-packed into the layout of the GEMM that runs the layer's
    bits: FP6 for a 4-bit layer, the 8-bit activation order for an 8-bit one.
    `fp6_all` / `a8_all` pack every layer into that layout as well (to run
    other policies on the same weights); `decode` also keeps every layer's codes
    in the decode layout (for decode batches)."""

    def __init__(self, torch, dptq, name, M, bits, fp6_all=False, a8_all=False, decode=False):
        import workloads
        self.torch, self.dptq = torch, dptq
        dev = torch.device("cuda:0")
        cfg = workloads.CONFIGS[name]
        self.name, self.M, self.L, self.lins = name, M, cfg["L"], cfg["linears"]
        self.bits = list(bits)
        gen = torch.Generator(device=dev)
        self.fp6, self.a8, self.dec, self.ws = [], [], [], []
        for l in range(self.L):
            f6, a8, dec, wsl = [], [], [], []
            for i, (_, K, N, h) in enumerate(self.lins):
                gen.manual_seed(cfg["seed"] * 1000003 + l * 16 + i)
                w = torch.randn((N, K), device=dev, generator=gen, dtype=torch.float32)
                w.mul_(0.02)
                wp, ws = dptq.prepare_weights(w, h)
                del w
                b = self.bits[l]
                f6.append(dptq.prepack_weights(wp, dptq.WEIGHTS_FP6) if fp6_all or b == 4 else None)
                a8.append(dptq.prepack_weights(wp, dptq.WEIGHTS_A8_ORDER).view(N, K // 2)
                          if a8_all or b == 8 else None)
                dec.append(dptq.prepack_weights(wp, dptq.WEIGHTS_DECODE) if decode else None)
                wsl.append(ws)
                del wp
            self.fp6.append(f6)
            self.a8.append(a8)
            self.dec.append(dec)
            self.ws.append(wsl)
        self.X = [torch.from_numpy(workloads.stack_layer_input(name, self.L // 2, n, M=M)).to(dev)
                  for n, *_ in self.lins]
        Kmax = max(K for _, K, _, _ in self.lins)
        Nmax = max(N for _, _, N, _ in self.lins)
        self.cbuf = torch.empty(M * Kmax, dtype=torch.int8, device=dev)
        self.a6buf = torch.empty(dptq.fp6_bytes(M, Kmax), dtype=torch.uint8, device=dev)
        self.sbuf = torch.empty(M, dtype=torch.float32, device=dev)
        self.ybuf = torch.empty(M * Nmax, dtype=torch.float16, device=dev)
        self.f6bytes = {K: dptq.fp6_bytes(M, K) for _, K, _, _ in self.lins}
        torch.cuda.synchronize()

    def ops(self):
        return 2.0 * self.M * sum(K * N for _, K, N, _ in self.lins) * self.L

    def weight_bytes(self):
        return sum(N * K // 2 + 4 * N for _, K, N, _ in self.lins) * self.L

    def launches(self, bits, events=None):
        """One pass over every linear: rotate+quantize then GEMM per linear.
        With `events`, a HIP event pair is recorded around every launch and
        (kernel, linear, start, end) appended."""
        dptq, M = self.dptq, self.M
        for l in range(self.L):
            b = bits[l]
            for i, (lin, K, N, h) in enumerate(self.lins):
                y = self.ybuf[: M * N].view(M, N)
                if b == 4:
                    a6 = self.a6buf[: self.f6bytes[K]]
                    k1 = lambda: dptq.rotate_quant_fp6(self.X[i], h, a6, self.sbuf)
                    g = lambda: dptq.qlinear_fp6(a6, self.sbuf, self.fp6[l][i], self.ws[l][i], M, K, N, y)
                    names = ("rq_fp6_a4", "gemm_fp6_a4")
                else:
                    codes = self.cbuf[: M * K].view(M, K)
                    k1 = lambda: dptq.rotate_quant(self.X[i], h, 8, codes, self.sbuf)
                    g = lambda: dptq.qlinear_a8(codes, self.sbuf, self.a8[l][i], self.ws[l][i], y)
                    names = ("rq_a8", "gemm_a8")
                for kname, f in zip(names, (k1, g)):
                    if events is None:
                        f()
                    else:
                        e0 = self.torch.cuda.Event(enable_timing=True)
                        e1 = self.torch.cuda.Event(enable_timing=True)
                        e0.record()
                        f()
                        e1.record()
                        events.append((kname, lin, e0, e1))

    def decode_launches(self, bits, X):
        """One pass at decode size: every linear from fp16 x, rotate+quantize
        then the decode GEMM on the decode weight layout."""
        dptq = self.dptq
        M = X[0].shape[0]
        for l in range(self.L):
            b = bits[l]
            for i, (_, K, N, h) in enumerate(self.lins):
                dt = self.torch.uint8 if b == 4 else self.torch.int8
                codes = self.cbuf[: M * K * b // 8].view(dt).view(M, K * b // 8)
                y = self.ybuf[: M * N].view(M, N)
                dptq.rotate_quant(X[i], h, b, codes, self.sbuf[:M])
                dptq.qlinear_decode_native(codes, self.sbuf[:M], b, self.dec[l][i], self.ws[l][i], y)


def time_headline(torch, dptq, args):
    import workloads
    cfg = workloads.CONFIGS[HEADLINE]
    L, M = cfg["L"], cfg["M"]
    mask = workloads.layer_mask(L, 4, cfg["mask_seed"])
    policy = lambda: dptq.layer_policy(L, mask)          # a1: host lookup, every step
    t0 = time.perf_counter()
    st = Stack(torch, dptq, HEADLINE, M, policy(), fp6_all=True, decode=True)
    setup_s = time.perf_counter() - t0
    progress(f"headline stack ready ({setup_s:.1f} s)")

    for _ in range(args.warmup):
        st.launches(policy())
    torch.cuda.synchronize()
    with ClockSampler() as clocks:
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        e0.record()
        for _ in range(args.steps):
            st.launches(policy())
        e1.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
    gpu_ms = e0.elapsed_time(e1) / args.steps
    progress(f"headline: {args.steps} steps, {wall * 1e3 / args.steps:.2f} ms per step")

    # One more step with an event pair around every launch: per-kernel
    # durations in the step's own order and cache state.
    events = []
    st.launches(policy(), events)
    torch.cuda.synchronize()
    per = {}
    for kname, lin, a, b in events:
        per.setdefault((kname, lin), []).append(a.elapsed_time(b) * 1e3)

    # The same stack with every layer at 4 bits, for the policy's cost.
    all4 = [4] * L
    st.launches(all4)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(3):
        st.launches(all4)
    torch.cuda.synchronize()
    all4_ms = (time.perf_counter() - t0) * 1e3 / 3
    return st, dict(wall=wall, gpu_ms=gpu_ms, per=per, clocks=clocks.summary(), setup_s=setup_s,
                    all4_ms=all4_ms, mask=[int(v) for v in mask], bits=policy())


def headline_record(st, r, args):
    M, L = st.M, st.L
    ops = st.ops()
    ms = r["wall"] * 1e3 / args.steps
    value = ops / (ms * 1e-3) / 1e12
    lin = {n: (K, N, h) for n, K, N, h in st.lins}
    bits = r["bits"]
    n8 = sum(1 for b in bits if b == 8)
    # per kernel family: launches and time per step, algorithmic work
    fam = {}
    kernels = {}
    for (kname, ln), us in sorted(r["per"].items()):
        K, N, h = lin[ln]
        b = 8 if kname.endswith("a8") else 4
        avg = sum(us) / len(us)
        ent = {"us": round(avg, 2), "launches_per_step": len(us)}
        if kname.startswith("gemm"):
            work = 2.0 * M * N * K
            ent["TOPS"] = round(work / (avg * 1e-6) / 1e12, 1)
            ent["frac_of_int8_peak"] = round(ent["TOPS"] / PEAK_INT8_TOPS, 4)
            if "fp6" in kname:
                ent["frac_of_fp6_peak"] = round(ent["TOPS"] / PEAK_FP6_TOPS, 4)
        else:
            work = k1_bytes(M, K, b)
            ent["GB/s"] = round(work / (avg * 1e-6) / 1e9, 1)
            ent["frac_of_hbm_peak"] = round(ent["GB/s"] / PEAK_HBM_GBS, 4)
            lane_ops = k1_essential_ops(h, fp6="fp6" in kname) * M * K
            ent["frac_of_alu_roof"] = round(lane_ops / (avg * 1e-6) / PEAK_LANE_OPS, 4)
        kernels[f"{kname}/{ln}"] = ent
        f = fam.setdefault(kname, {"us": 0.0, "n": 0, "work": 0.0})
        f["us"] += sum(us)
        f["n"] += len(us)
        f["work"] += work * len(us)
    dominant = max(fam, key=lambda k: fam[k]["us"])
    d = fam[dominant]
    kernel_names = {"gemm_fp6_a4": ("qgemm_fp6<false, false>", PEAK_FP6_TOPS),
                    "gemm_a8": ("qgemm_prefill_wide<8, false, true, false>", PEAK_INT8_TOPS)}
    if dominant.startswith("gemm"):
        kname, peak = kernel_names[dominant]
        achieved = d["work"] / (d["us"] * 1e-6) / 1e12
        traffic = measured_traffic() if dominant == "gemm_fp6_a4" else None
        roof = {"bound": "mfma", "kernel": kname, "achieved": round(achieved, 1), "peak": peak,
                "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                "frac_of_int8_peak": round(achieved / PEAK_INT8_TOPS, 4),
                "avg_launch_us": round(d["us"] / d["n"], 2), "launches_per_step": d["n"],
                "traffic": traffic,
                "algorithmic_bytes_per_launch": int(sum(
                    gemm_bytes(M, K, N, 4) for K, N, _ in lin.values()) / len(lin)),
                "share_of_step": round(d["us"] / 1e3 / ms, 3)}
    else:
        achieved = d["work"] / (d["us"] * 1e-6) / 1e9
        roof = {"bound": "hbm", "kernel": dominant, "achieved": round(achieved, 1),
                "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4),
                "traffic": None}
    gemm_us = sum(f["us"] for k, f in fam.items() if k.startswith("gemm"))
    k1_us = sum(f["us"] for k, f in fam.items() if not k.startswith("gemm"))
    return value, ms, roof, kernels, {
        "gemm_ms_per_step": round(gemm_us / 1e3, 3), "rotate_quant_ms_per_step": round(k1_us / 1e3, 3),
        "gemm_TOPS": round(ops / (gemm_us * 1e-6) / 1e12, 1),
        "layers_a8": n8, "mask_seed": 5,
        "all_a4_ms_per_step": round(r["all4_ms"], 3),
        "mixed_over_all_a4": round(ms / r["all4_ms"], 4),
    }


# ---------------------------------------------------------------------------
# other workloads (graph-replayed)
# ---------------------------------------------------------------------------
def single_linear(torch, dptq, name, M, copies_bytes=300 << 20):
    """K1 and GEMM of one linear at 4 bits (FP6 path and int8 path) and at 8
    bits (8-bit-order weights), inputs and weights cycling through copies
    beyond the last-level cache."""
    import numpy as np
    import workloads
    dev = torch.device("cuda:0")
    cfg = workloads.CONFIGS[name]
    K, N, h = cfg["K"], cfg["N"], cfg["h"]
    x = torch.from_numpy(workloads.activations_for(name, M=M)).to(dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(cfg["seed"] + 17)
    w = torch.randn((N, K), device=dev, generator=gen) * 0.02
    wp, ws = dptq.prepare_weights(w, h)
    del w
    R = int(max(2, min(16, copies_bytes // max(1, N * K // 2 + 2 * M * K))))
    xs = [x.clone() for _ in range(R)]
    wps = [wp.clone() for _ in range(R)]
    w6s = [dptq.prepack_weights(wp, dptq.WEIGHTS_FP6) for _ in range(R)] \
        if K % 128 == 0 and M > 16 else None
    w8s = [dptq.prepack_weights(wp, dptq.WEIGHTS_A8_ORDER).view(N, K // 2) for _ in range(R)] \
        if K % 128 == 0 else None
    wds = [dptq.prepack_weights(wp, dptq.WEIGHTS_DECODE) for _ in range(R)] \
        if K % 128 == 0 and M <= 16 else None
    y = torch.empty((M, N), dtype=torch.float16, device=dev)
    out = {"M": M, "K": K, "N": N, "had_size": h}
    n = 24
    ops = 2.0 * M * N * K

    def rec(k1_us, g_us, bits, path):
        r = {"rotate_quant_us": round(k1_us, 2), "gemm_us": round(g_us, 2),
             "rotate_quant_GB/s": round(k1_bytes(M, K, bits) / (k1_us * 1e-6) / 1e9, 1),
             "rotate_quant_frac_of_alu_roof": round(
                 k1_essential_ops(h, path == "fp6") * M * K / (k1_us * 1e-6) / PEAK_LANE_OPS, 4),
             "qlinear_TOPS": round(ops / ((k1_us + g_us) * 1e-6) / 1e12, 2),
             "gemm_TOPS": round(ops / (g_us * 1e-6) / 1e12, 2),
             "gemm_frac_of_int8_peak": round(ops / (g_us * 1e-6) / 1e12 / PEAK_INT8_TOPS, 4)}
        if path == "fp6":
            r["gemm_frac_of_fp6_peak"] = round(ops / (g_us * 1e-6) / 1e12 / PEAK_FP6_TOPS, 4)
        if M <= 16:
            r["gemm_GB/s"] = round(gemm_bytes(M, K, N, bits) / (g_us * 1e-6) / 1e9, 1)
            r["gemm_frac_of_hbm_peak"] = round(r["gemm_GB/s"] / PEAK_HBM_GBS, 4)
        return r

    for bits in (4, 8):
        codes, scales = dptq.rotate_quant(x, h, bits)
        k1 = graph_time(torch, [(lambda i: (lambda: dptq.rotate_quant(xs[i % R], h, bits, codes, scales)))(i)
                                for i in range(n)])
        g = graph_time(torch, [(lambda i: (lambda: dptq.qlinear(codes, scales, bits, wps[i % R], ws, y)))(i)
                               for i in range(n)])
        out[f"a{bits}_int8"] = rec(k1, g, bits, "int8")
        if wds is not None:   # decode batches: the decode weight layout, GEMM and from fp16 x
            gd = graph_time(torch, [(lambda i: (lambda: dptq.qlinear_decode_native(
                codes, scales, bits, wds[i % R], ws, y)))(i) for i in range(n)])
            out[f"a{bits}_decode_layout"] = rec(k1, gd, bits, "int8")
            xd = graph_time(torch, [(lambda i: (lambda: (
                dptq.rotate_quant(xs[i % R], h, bits, codes, scales),
                dptq.qlinear_decode_native(codes, scales, bits, wds[i % R], ws, y))))(i)
                for i in range(n)])
            out[f"a{bits}_decode_layout_from_x_us"] = round(xd, 2)
        if bits == 8 and w8s is not None:
            g8 = graph_time(torch, [(lambda i: (lambda: dptq.qlinear_a8(codes, scales, w8s[i % R], ws, y)))(i)
                                    for i in range(n)])
            out["a8_int8_a8order"] = rec(k1, g8, 8, "int8")
        if bits == 4 and w6s is not None and M > 16:   # the FP6 path serves prefill sizes
            a6, s6 = dptq.rotate_quant_fp6(x, h)
            k16 = graph_time(torch, [(lambda i: (lambda: dptq.rotate_quant_fp6(xs[i % R], h, a6, s6)))(i)
                                     for i in range(n)])
            g6 = graph_time(torch, [(lambda i: (lambda: dptq.qlinear_fp6(a6, s6, w6s[i % R], ws, M, K, N, y)))(i)
                                    for i in range(n)])
            out["a4_fp6"] = rec(k16, g6, 4, "fp6")
            # the FP6 layout's output bytes are 0.75 per code; GB/s above counts
            # the algorithmic 0.5
        if M <= 16:
            d = graph_time(torch, [(lambda i: (lambda: dptq.qlinear_decode_fused(
                x, h, bits, wps[i % R], ws, y, codes, scales, mode=dptq.DECODE_AUTO)))(i) for i in range(n)])
            out[f"a{bits}_decode_from_x_us"] = round(d, 2)
    del xs, wps, w6s, w8s
    torch.cuda.empty_cache()
    return out


def stack_7b(torch, dptq):
    """The LLaMA-2-7B 32-layer linear stack at M = 2048: the seeded 4-of-32
    mask, the paper's default set and all-4-bit, each one graph replay."""
    import workloads
    cfg = workloads.CONFIGS["llama2_7b_stack"]
    L, M = cfg["L"], cfg["M"]
    pol = {"seeded_mask": dptq.layer_policy(L, workloads.layer_mask(L, 4, cfg["mask_seed"])),
           "paper_default": dptq.layer_policy(L), "all_a4": [4] * L}
    st = Stack(torch, dptq, "llama2_7b_stack", M, pol["seeded_mask"], fp6_all=True, a8_all=True)
    out = {"M": M, "layers": L, "weights_GB": round(st.weight_bytes() / 1e9, 2)}
    res = {p: graph_time(torch, [lambda bits=bits: st.launches(bits)], reps=2) / 1e3
           for p, bits in pol.items()}
    ops = st.ops()
    for p, ms in res.items():
        out[f"{p}_ms"] = round(ms, 3)
        out[f"{p}_TOPS"] = round(ops / (ms * 1e-3) / 1e12, 1)
    out["seeded_mask_over_all_a4"] = round(res["seeded_mask"] / res["all_a4"], 4)
    out["paper_default_over_all_a4"] = round(res["paper_default"] / res["all_a4"], 4)
    del st
    torch.cuda.empty_cache()
    return out


def decode_70b(torch, st, bits):
    """The headline stack at M = 8 decode (every linear from fp16 x:
    rotate+quantize, then the decode GEMM on the decode weight layout), one
    graph replay per pass."""
    import workloads
    dev = torch.device("cuda:0")
    X = [torch.from_numpy(workloads.stack_layer_input(HEADLINE, st.L // 2, n, M=8)).to(dev)
         for n, *_ in st.lins]
    ms = graph_time(torch, [lambda: st.decode_launches(bits, X)], reps=3) / 1e3
    return {"M": 8, "layers": st.L, "ms": round(ms, 3),
            "weight_GB/s": round(st.weight_bytes() / (ms * 1e-3) / 1e9, 1),
            "frac_of_hbm_peak": round(st.weight_bytes() / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
            # HBM bytes of the decode GEMM over its algorithmic bytes, from the
            # committed counter summary of `bench.py --only decode` (None when
            # that summary was taken on other sources of the kernel)
            "gemm_traffic_over_algorithmic": measured_traffic(
                DECODE_TRAFFIC_FILE, DECODE_TRAFFIC_SOURCE, "traffic_over_algorithmic")}


def time_extended(torch, dptq):
    """Variants outside the headline: the range quantizer, calibration, KV4."""
    import numpy as np
    import workloads
    dev = torch.device("cuda:0")
    out = {}
    M, K, N, h = 2048, 4096, 12288, 4096
    rng = np.random.default_rng(7)
    x = torch.from_numpy(workloads.gauss_outliers(rng, M, K)).to(dev)
    wp = torch.from_numpy(workloads.random_weight_bytes(rng, N, K)).to(dev)
    ws = torch.full((N,), 1e-5, device=dev)
    sums = dptq.weight_sums(wp)
    y = torch.empty((M, N), dtype=torch.float16, device=dev)
    for bits in (4, 8):
        cr, sr, zr = dptq.rotate_quant_range(x, h, bits)
        out[f"range_a{bits}"] = {
            "rotate_quant_range_us": round(graph_time(
                torch, [lambda: dptq.rotate_quant_range(x, h, bits, cr, sr, zr)] * 24), 2),
            "qlinear_range_us": round(graph_time(
                torch, [lambda: dptq.qlinear_range(cr, sr, zr, bits, wp, ws, sums, y)] * 24), 2)}
    T = 2048
    xs, dxs = workloads.residual_stream(np.random.default_rng(11), 2, T, K)[0]
    xd, dxd = torch.from_numpy(xs).to(dev), torch.from_numpy(dxs).to(dev)
    jr = torch.empty(T, dtype=torch.float32, device=dev)
    snr = torch.empty(T, dtype=torch.float32, device=dev)
    means = torch.empty(2, dtype=torch.float64, device=dev)
    for bits in (4, 8):
        us = graph_time(torch, [lambda: dptq.residual_dynamics(xd, dxd, h, bits, jr=jr, snr=snr,
                                                               means=means)] * 24)
        out[f"calibration_a{bits}"] = {"us": round(us, 2),
                                       "GB/s": round((4 * T * K + 8 * T) / (us * 1e-6) / 1e9, 1)}
    T, D, g = 32 * 2048, 1024, 128
    gen = torch.Generator(device=dev)
    gen.manual_seed(8)
    kv = [torch.randn((T, D), device=dev, generator=gen).half() for _ in range(4)]
    outs = [dptq.kv_quant(t, g) for t in kv]
    rec = [torch.empty((T, D), dtype=torch.float16, device=dev) for _ in range(4)]
    nb = 2 * T * D + T * D // 2 + 8 * T * (D // g)
    q = graph_time(torch, [(lambda i: (lambda: dptq.kv_quant(kv[i % 4], g, *outs[i % 4])))(i) for i in range(8)])
    d = graph_time(torch, [(lambda i: (lambda: dptq.kv_dequant(*outs[i % 4], g, out=rec[i % 4])))(i)
                           for i in range(8)])
    out["kv4"] = {"tokens": T, "row": D, "group": g, "quant_us": round(q, 2),
                  "quant_GB/s": round(nb / (q * 1e-6) / 1e9, 1), "dequant_us": round(d, 2),
                  "dequant_GB/s": round(nb / (d * 1e-6) / 1e9, 1)}
    return out


# ---------------------------------------------------------------------------
# counter runs
# ---------------------------------------------------------------------------
def run_only(torch, dptq, args):
    """One kernel family of the headline step at each of its four linear
    shapes, --steps launches per shape, nothing timed (rocprofv3 --pmc)."""
    dev = torch.device("cuda:0")
    if args.only == "copy":
        n = 256 << 20
        src = torch.ones(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"only": "copy", "bytes_per_launch": n}))
        return
    if args.only == "decode":
        run_only_decode(torch, dptq, args)
        return
    import workloads
    cfg = workloads.CONFIGS[HEADLINE]
    M = cfg["M"]
    bits = 4 if args.only.endswith("6") else 8
    lins = cfg["linears"]
    gen = torch.Generator(device=dev)
    gen.manual_seed(1)
    X = [torch.from_numpy(workloads.stack_layer_input(HEADLINE, 40, n, M=M)).to(dev) for n, *_ in lins]
    W = []
    for _, K, N, _ in lins:
        wp = torch.randint(0, 256, (N, K // 2), dtype=torch.uint8, device=dev, generator=gen)
        layout = dptq.WEIGHTS_FP6 if bits == 4 else dptq.WEIGHTS_A8_ORDER
        W.append((dptq.prepack_weights(wp, layout), torch.full((N,), 1e-5, device=dev)))
        del wp
    Kmax = max(K for _, K, _, _ in lins)
    Nmax = max(N for _, _, N, _ in lins)
    a6 = torch.empty(dptq.fp6_bytes(M, Kmax), dtype=torch.uint8, device=dev)
    c8 = torch.empty(M * Kmax, dtype=torch.int8, device=dev)
    s = torch.empty(M, dtype=torch.float32, device=dev)
    yb = torch.empty(M * Nmax, dtype=torch.float16, device=dev)
    # valid operands in the shared buffers: the largest linear's codes
    iK = max(range(len(lins)), key=lambda i: lins[i][1])
    if bits == 4:
        dptq.rotate_quant_fp6(X[iK], lins[iK][3], a6[: dptq.fp6_bytes(M, lins[iK][1])], s)
    else:
        dptq.rotate_quant(X[iK], lins[iK][3], 8, c8[: M * lins[iK][1]].view(M, -1), s)
    torch.cuda.synchronize()
    for _ in range(args.steps):
        for i, (_, K, N, h) in enumerate(lins):
            y = yb[: M * N].view(M, N)
            if bits == 4:
                a = a6[: dptq.fp6_bytes(M, K)]
                if args.only == "rq6":
                    dptq.rotate_quant_fp6(X[i], h, a, s)
                else:
                    dptq.qlinear_fp6(a, s, W[i][0], W[i][1], M, K, N, y)
            else:
                c = c8[: M * K].view(M, K)
                if args.only == "rq8":
                    dptq.rotate_quant(X[i], h, 8, c, s)
                else:
                    dptq.qlinear_a8(c, s, W[i][0].view(N, K // 2), W[i][1], y)
    torch.cuda.synchronize()
    print(json.dumps({"only": args.only, "launches_per_shape": args.steps,
                      "shapes": [[M, K, N] for _, K, N, _ in lins]}))


def run_only_decode(torch, dptq, args):
    """The headline stack's four linears at M = 8 decode, A4: rotate+quantize
    from fp16 x, then the decode GEMM on the decode weight layout, --steps
    times in a fixed cycle over the four shapes, each shape's weights cycling
    through copies beyond the Infinity Cache (rocprofv3 kernel trace and
    counter passes; nothing timed here)."""
    import workloads
    dev = torch.device("cuda:0")
    cfg = workloads.CONFIGS[HEADLINE]
    lins, M, bits = cfg["linears"], 8, 4
    gen = torch.Generator(device=dev)
    gen.manual_seed(2)
    X = [torch.from_numpy(workloads.stack_layer_input(HEADLINE, 40, n, M=M)).to(dev) for n, *_ in lins]
    W = []
    for _, K, N, _ in lins:
        copies = max(2, -(-(600 << 20) // (N * K // 2)))
        ws = []
        for _ in range(copies):
            wp = torch.randint(0, 256, (N, K // 2), dtype=torch.uint8, device=dev, generator=gen)
            ws.append(dptq.prepack_weights(wp, dptq.WEIGHTS_DECODE))
            del wp
        W.append((ws, torch.full((N,), 1e-5, device=dev)))
    codes = [torch.empty((M, K // 2), dtype=torch.uint8, device=dev) for _, K, _, _ in lins]
    s = torch.empty(M, dtype=torch.float32, device=dev)
    ys = [torch.empty((M, N), dtype=torch.float16, device=dev) for _, _, N, _ in lins]
    torch.cuda.synchronize()
    for step in range(args.steps):
        for i, (_, K, N, h) in enumerate(lins):
            dptq.rotate_quant(X[i], h, bits, codes[i], s)
            wcopies, wsc = W[i]
            dptq.qlinear_decode_native(codes[i], s, bits, wcopies[step % len(wcopies)], wsc, ys[i])
    torch.cuda.synchronize()
    print(json.dumps({"only": "decode", "launches_per_shape": args.steps, "M": M, "bits": bits,
                      "shapes": [[M, K, N] for _, K, N, _ in lins],
                      "gemm_algorithmic_bytes": [N * K // 2 + 4 * N + M * K * bits // 8 + 4 * M + 2 * M * N
                                                 for _, K, N, _ in lins]}))


# ---------------------------------------------------------------------------
# CPU oracle baseline (runs before the GPU is touched)
# ---------------------------------------------------------------------------
_JOB = None


def _one_thread():
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(1)
    except Exception:
        pass


def _rotate_chunk(rows):
    """The oracle's rotate+quantize on token rows [rows[0], rows[1]) of the job."""
    from oracle import rotate_quant_ref
    x, h, bits = _JOB[:3]
    return rotate_quant_ref(x[rows[0]:rows[1]], h, bits)


def _gemm_chunk(cols):
    """The oracle's exact GEMM and epilogue for output channels [cols[0], cols[1])."""
    from oracle import qlinear_ref
    codes, scales, bits, wq, ws = _JOB
    return qlinear_ref(codes, scales, bits, wq[cols[0]:cols[1]], ws[cols[0]:cols[1]])


def _split(n, parts):
    k = max(1, min(n, parts))
    return [(n * i // k, n * (i + 1) // k) for i in range(k) if n * (i + 1) // k > n * i // k]


def _oracle_job(P, x, h, bits, wq, ws):
    """Seconds of the oracle on every row of x over P forked single-threaded
    workers: rotate+quantize split by token rows, then the exact GEMM and
    epilogue split by output channels.  Returns (rotate s, GEMM s)."""
    import multiprocessing as mp
    import numpy as np
    global _JOB
    ctx = mp.get_context("fork")
    _JOB = (x, h, bits)
    with ctx.Pool(P, initializer=_one_thread) as pool:
        t0 = time.perf_counter()
        parts = pool.map(_rotate_chunk, _split(x.shape[0], P))
        t_rot = time.perf_counter() - t0
    codes = np.concatenate([c for c, _ in parts])
    scales = np.concatenate([s for _, s in parts])
    _JOB = (codes, scales, bits, wq, ws)
    with ctx.Pool(P, initializer=_one_thread) as pool:
        t0 = time.perf_counter()
        pool.map(_gemm_chunk, _split(wq.shape[0], P))
        t_gemm = time.perf_counter() - t0
    _JOB = None
    return t_rot, t_gemm


def cpu_baseline(P):
    """The oracle timed on the host's cores (Section 4.9 workloads stand-ins):
    the single linears (tiny, LLaMA-2-7B QKV, LLaMA-3-8B down at every M) in
    full, the two stacks on 256 seeded rows per linear at each bit width,
    extrapolated linearly in M and over the layers of the mask."""
    import numpy as np
    import workloads
    cores = os.cpu_count()
    aff = len(os.sched_getaffinity(0))
    P = P or max(1, min(16, aff))
    rng = np.random.default_rng(123)

    def weights_for(x, K, N):
        wq = workloads.random_weight_bytes(rng, N, K)
        l1 = float(np.max(np.sum(np.abs(x.astype(np.float32)), axis=1))) or 1.0
        ws = (rng.uniform(0.5, 1.0, N) * 3e4 / (8 * K * l1)).astype(np.float32)
        return wq, ws

    out = {"cores": cores, "affinity": aff, "workers": P, "configs": {}}
    t_all = time.perf_counter()
    singles = [("tiny", 16), ("llama2_7b_qkv", 2048), ("llama3_8b_down", 1), ("llama3_8b_down", 4),
               ("llama3_8b_down", 16), ("llama3_8b_down", 2048)]
    for name, M in singles:
        cfg = workloads.CONFIGS[name]
        K, N, h = cfg["K"], cfg["N"], cfg["h"]
        x = workloads.activations_for(name, M=M)
        wq, ws = weights_for(x, K, N)
        ent = {}
        for bits in (4, 8):
            tr, tg = _oracle_job(P, x, h, bits, wq, ws)
            ent[f"a{bits}"] = {"rotate_quant_s": round(tr, 3), "gemm_s": round(tg, 3),
                               "TOPS": round(2.0 * M * N * K / (tr + tg) / 1e12, 6)}
        out["configs"][f"{name}_M{M}"] = ent
        progress(f"cpu baseline: {name} M={M} done")
    for name, mask_seed in (("llama2_7b_stack", 3), (HEADLINE, 5)):
        cfg = workloads.CONFIGS[name]
        L, M = cfg["L"], cfg["M"]
        mask = workloads.layer_mask(L, 4, mask_seed)
        n8 = int(mask.sum())
        per_bits = {4: 0.0, 8: 0.0}
        rows = 256
        for lin, K, N, h in cfg["linears"]:
            x = workloads.stack_layer_input(name, L // 2, lin, M=rows)
            wq, ws = weights_for(x, K, N)
            for bits in (4, 8):
                tr, tg = _oracle_job(P, x, h, bits, wq, ws)
                per_bits[bits] += (tr + tg) * M / rows    # one layer's linears at M tokens
                progress(f"cpu baseline: {name}/{lin} A{bits} {tr + tg:.1f} s")
        est = per_bits[4] * (L - n8) + per_bits[8] * n8
        ops = 2.0 * M * sum(K * N for _, K, N, _ in cfg["linears"]) * L
        progress(f"cpu baseline: {name} sampled rows done")
        out["configs"][name] = {"M": M, "layers": L, "sampled_rows_per_linear": rows,
                                "extrapolated": True, "s": round(est, 1),
                                "TOPS": round(ops / est / 1e12, 6)}
    out["total_s"] = round(time.perf_counter() - t_all, 1)
    head = out["configs"][HEADLINE]
    return {"value": head["TOPS"], "unit": "TOPS", "cores": P, "kind": "oracle",
            "sample": (f"{head['sampled_rows_per_linear']} seeded token rows per linear of the "
                       f"LLaMA-2-70B stack at each bit width (rotation, quantization, exact GEMM, "
                       f"epilogue), extrapolated to M = {head['M']} and the 80-layer mixed mask; "
                       f"{P} worker processes, one thread each"),
            "host": {"cpu_count": cores, "affinity": aff, "workers": P}, "per_config": out["configs"],
            "total_s": out["total_s"]}


# ---------------------------------------------------------------------------
def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU (asked for --gpus {args.gpus}): the sharded path is a "
              "design only, and every figure here is one GPU's", file=sys.stderr)
        sys.exit(2)
    cpu = None
    if not args.no_cpu_baseline and not args.only:
        cpu = cpu_baseline(args.cpu_workers)      # before anything touches the GPU
    import torch
    import paper_2606_12487_amd as dptq
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dptq.lib()
    if args.only:
        run_only(torch, dptq, args)
        return

    st, r = time_headline(torch, dptq, args)
    value, ms, roof, kernels, extra = headline_record(st, r, args)
    cfg_h = __import__("workloads").CONFIGS[HEADLINE]
    rec = {
        "metric": METRIC, "value": round(value, 2), "unit": "TOPS", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int4 x int4 on fp6 MFMA, int8 x int4 on int8 MFMA, exact int32 sums",
        "data": "synthetic",
        "config": {"workload": "llama2-70b 80-layer linear stack (qkv 8192->10240, o 8192->8192, "
                               "gate/up 8192->57344, down 28672->8192 at h=28x1024), M=4096 prefill, "
                               "seeded mixed A4/A8 mask (4 of 80 layers at 8 bits)",
                   "M": cfg_h["M"], "layers": cfg_h["L"], "mask": r["mask"], "parallelism": "none"},
        "frac_of_int8_peak": round(value / PEAK_INT8_TOPS, 4),
        "gpu_ms_per_step": round(r["gpu_ms"], 3),
        "roofline": roof,
        "clocks": r["clocks"],
        "headline": extra,
        "kernels": kernels,
        "setup_s": round(r["setup_s"], 1),
    }
    configs = {}
    if not args.no_configs:
        configs["llama2_70b_M8_decode"] = decode_70b(torch, st, r["bits"])
    del st
    torch.cuda.empty_cache()
    if not args.no_configs:
        progress("70B decode stack done")
        configs["tiny"] = single_linear(torch, dptq, "tiny", 16)
        configs["llama2_7b_qkv"] = single_linear(torch, dptq, "llama2_7b_qkv", 2048)
        for M in (1, 4, 16, 2048):
            configs[f"llama3_8b_down_M{M}"] = single_linear(torch, dptq, "llama3_8b_down", M)
        progress("single linears done")
        configs["llama2_7b_stack"] = stack_7b(torch, dptq)
        progress("7B stack done")
        rec["configs"] = configs
    if args.extended:
        rec["extended"] = time_extended(torch, dptq)
    if cpu is not None:
        rec["cpu_baseline"] = cpu
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
