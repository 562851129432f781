"""Benchmark of the DynamicPTQ quantized linear layer on one MI355X.

Workload (one "step"): the LLaMA-2-7B fused QKV projection, M = 2048 prefill
tokens, K = 4096, N = 12288, Hadamard 4096, with synthetic seeded fp16
activations (N(0,1) plus 4 outlier channels x50-x200) and N(0, 0.02) weights
quantized to 4 bits per output channel.  The layer policy (Eq. 21) is looked
up for a 32-layer model, and the step runs the layer as a non-sensitive layer
(A4) and then as a sensitive layer (A8): per precision one rotate+quantize
launch and one GEMM launch, all on one stream.  The A4 layer runs on the FP6
matrix cores (rotate+quantize writing the FP6 operand layout, then the FP6
GEMM against the same weights pre-packed once); the A8 layer on the int8
matrix cores.  Both return the oracle's results bit for bit.  Inputs are resident in HBM
before timing; the step cycles through enough copies of activations and
weights (> 256 MiB) that the Infinity Cache cannot hold them.  The timed
steps launch every kernel from the host on one stream; the same steps
replayed from captured HIP graphs are reported under "graph".

    python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--extended]

Prints one JSON line.  value = total integer ops (2 M N K per GEMM) / time.
"""

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_INT8_TOPS = 5000.0      # MI355X dense int8 MFMA, T ops/s
PEAK_HBM_GBS = 8000.0        # MI355X HBM3E, GB/s
METRIC = "W4A4/W4A8 qlinear TOPS (rotate+quant+GEMM), % int8 MFMA peak; decode GB/s"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--copies", type=int, default=12,
                   help="distinct activation/weight copies cycled per step")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-rows", type=int, default=160,
                   help="token rows of the workload the CPU oracle is timed on")
    p.add_argument("--extended", action="store_true",
                   help="also time the decode shapes, the fused decode, the range quantizer, "
                        "calibration, KV4 and whole stacks")
    p.add_argument("--only", choices=["rq4", "gemm4", "rq6", "gemm6", "rq8", "gemm8", "copy"],
                   help="run one kernel of the step --steps times (for counter runs) "
                        "or, with copy, a plain device copy of 256 MiB (counter calibration)")
    return p.parse_args()


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_qgemm_prefill_a8_llama2_7b_qkv.txt")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2606_12487_amd", "csrc", "qgemm.hip")
PEAK_FP6_TOPS = 10100.0      # MI355X dense fp6 / fp4 MFMA, T ops/s


def source_digest(path):
    import hashlib
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def measured_traffic():
    """HBM bytes per launch of the A8 int8 GEMM from the committed counter summary,
    or None when it is missing or was taken on a different kernel source."""
    if not os.path.exists(TRAFFIC_FILE):
        return None
    kv = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("source_sha256_16") != source_digest(KERNEL_SOURCE):
        return None
    try:
        return int(float(kv["hbm_bytes_per_launch"]))
    except (KeyError, ValueError):
        return None


def run_only(torch, dptq, cfg, args):
    """One kernel, repeated; nothing timed.  Used under rocprofv3 --pmc."""
    import numpy as np
    import workloads
    dev = torch.device("cuda:0")
    if args.only == "copy":
        n = 256 << 20
        src = torch.ones(n, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"only": "copy", "bytes_read_per_launch": n, "bytes_written_per_launch": n}))
        return
    M, K, N, h = cfg["M"], cfg["K"], cfg["N"], cfg["h"]
    rng = np.random.default_rng(cfg["seed"])
    x = torch.from_numpy(workloads.gauss_outliers(rng, M, K)).to(dev)
    w = torch.from_numpy(workloads.weights(rng, N, K)).to(dev)
    wp, ws = dptq.prepare_weights(w, h)
    del w
    y = torch.empty((M, N), dtype=torch.float16, device=dev)
    if args.only.endswith("6"):
        a6, s6 = dptq.rotate_quant_fp6(x, h)
        w6 = dptq.pack_fp6(wp)
        torch.cuda.synchronize()
        for _ in range(args.steps):
            if args.only.startswith("rq"):
                dptq.rotate_quant_fp6(x, h, a6, s6)
            else:
                dptq.qlinear_fp6(a6, s6, w6, ws, M, K, N, y)
        torch.cuda.synchronize()
        print(json.dumps({"only": args.only, "launches": args.steps}))
        return
    bits = 4 if args.only.endswith("4") else 8
    codes, scales = dptq.rotate_quant(x, h, bits)
    w8 = dptq.pack_w4_a8(wp) if bits == 8 else None
    torch.cuda.synchronize()
    for _ in range(args.steps):
        if args.only.startswith("rq"):
            dptq.rotate_quant(x, h, bits, codes, scales)
        elif bits == 8:
            dptq.qlinear_a8(codes, scales, w8, ws, y)     # the step's A8 GEMM
        else:
            dptq.qlinear(codes, scales, bits, wp, ws, y)
    torch.cuda.synchronize()
    print(json.dumps({"only": args.only, "launches": args.steps}))


def _events(torch, n):
    return [torch.cuda.Event(enable_timing=True) for _ in range(n)]


def time_layer(torch, dptq, cfg, args):
    import numpy as np
    import workloads
    dev = torch.device("cuda:0")
    M, K, N, h = cfg["M"], cfg["K"], cfg["N"], cfg["h"]
    rng = np.random.default_rng(cfg["seed"])
    x = torch.from_numpy(workloads.gauss_outliers(rng, M, K)).to(dev)
    w = torch.from_numpy(workloads.weights(rng, N, K)).to(dev)
    wp, ws = dptq.prepare_weights(w, h)
    del w
    R = max(1, args.copies)
    xs = [x.clone() for _ in range(R)]
    wps = [wp.clone() for _ in range(R)]
    w6s = [dptq.pack_fp6(wp) for _ in range(R)]      # the same weights, FP6 operand layout
    w8s = [dptq.pack_w4_a8(wp) for _ in range(R)]    # the same weights, 8-bit activation order
    wss = [ws.clone() for _ in range(R)]
    codes8 = torch.empty((M, K), dtype=torch.int8, device=dev)
    a6 = torch.empty((dptq.fp6_bytes(M, K),), dtype=torch.uint8, device=dev)
    scales = torch.empty((M,), dtype=torch.float32, device=dev)
    y = torch.empty((M, N), dtype=torch.float16, device=dev)
    torch.cuda.synchronize()

    n_layers = 32
    def layers(r, seq):
        for bits in seq:
            if bits == 4:
                dptq.rotate_quant_fp6(xs[r], h, a6, scales)
                dptq.qlinear_fp6(a6, scales, w6s[r], wss[r], M, K, N, y)
            else:
                dptq.rotate_quant(xs[r], h, bits, codes8, scales)
                dptq.qlinear_a8(codes8, scales, w8s[r], wss[r], y)

    def policy():
        bits_all = dptq.layer_policy(n_layers)
        return (bits_all[n_layers // 2], bits_all[0])     # a non-sensitive, a sensitive layer

    # The timed steps: every kernel launched from the host on one stream.
    seq = policy()
    for i in range(args.warmup):
        layers(i % R, policy())
    torch.cuda.synchronize()
    e0, e1 = _events(torch, 2)
    t0 = time.perf_counter()
    e0.record()
    for i in range(args.steps):
        layers(i % R, policy())
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = e0.elapsed_time(e1)

    # The same steps replayed from captured HIP graphs (one per input copy;
    # the policy lookup stays on the host), for reference.  A replay must
    # reproduce the eager result bit for bit.
    s_cap = torch.cuda.Stream()
    graphs = []
    for r in range(R):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s_cap):
            layers(r, seq)
        graphs.append(g)
    layers(0, seq)
    torch.cuda.synchronize()
    y_eager = y.clone()
    y.zero_()
    graphs[0].replay()
    torch.cuda.synchronize()
    if not torch.equal(y.view(torch.int16), y_eager.view(torch.int16)):
        raise RuntimeError("graph replay of the step differs from its eager launches")
    for i in range(args.warmup):
        graphs[i % R].replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        policy()
        graphs[i % R].replay()
    torch.cuda.synchronize()
    wall_graph = time.perf_counter() - t0
    del graphs
    return wall, gpu_ms, seq, wall_graph


def time_kernels(torch, dptq, cfg, args, seq, reps=24):
    """Average duration (ms) of each kernel of the step, from `reps`
    back-to-back launches captured in a HIP graph and replayed between two HIP
    events on the launch stream (no host launch gaps, no events between the
    launches).  Inputs cycle over the same copies as the step."""
    import numpy as np
    import workloads
    dev = torch.device("cuda:0")
    M, K, N, h = cfg["M"], cfg["K"], cfg["N"], cfg["h"]
    rng = np.random.default_rng(cfg["seed"] + 7)
    x = torch.from_numpy(workloads.gauss_outliers(rng, M, K)).to(dev)
    w = torch.from_numpy(workloads.weights(rng, N, K)).to(dev)
    wp, ws = dptq.prepare_weights(w, h)
    del w
    R = max(1, args.copies)
    xs = [x.clone() for _ in range(R)]
    wps = [wp.clone() for _ in range(R)]
    w6s = [dptq.pack_fp6(wp) for _ in range(R)]
    w8s = [dptq.pack_w4_a8(wp) for _ in range(R)]
    y = torch.empty((M, N), dtype=torch.float16, device=dev)
    out = {}
    # the step's kernels: FP6 A4 layer, int8 A8 layer
    a6, s6 = dptq.rotate_quant_fp6(x, h)
    out["rotate_quant_fp6_a4"] = _graph_time(torch, [
        (lambda i: (lambda: dptq.rotate_quant_fp6(xs[i % R], h, a6, s6)))(i) for i in range(reps)]) / 1e3
    out["gemm_fp6_a4"] = _graph_time(torch, [
        (lambda i: (lambda: dptq.qlinear_fp6(a6, s6, w6s[i % R], ws, M, K, N, y)))(i)
        for i in range(reps)]) / 1e3
    # the int8 matrix-core kernels for both precisions: the step's A8 GEMM on
    # weights in the 8-bit activation order, and for comparison the A8 and A4
    # GEMMs on the canonical nibble order
    for bits in (8, 4):
        codes, scales = dptq.rotate_quant(x, h, bits)
        if bits == 8:
            out["gemm_a8"] = _graph_time(torch, [
                (lambda i: (lambda: dptq.qlinear_a8(codes, scales, w8s[i % R], ws, y)))(i)
                for i in range(reps)]) / 1e3
        out[f"gemm_a{bits}_canonical_order"] = _graph_time(torch, [
            (lambda i: (lambda: dptq.qlinear(codes, scales, bits, wps[i % R], ws, y)))(i)
            for i in range(reps)]) / 1e3
        out[f"rotate_quant_a{bits}"] = _graph_time(torch, [
            (lambda i: (lambda: dptq.rotate_quant(xs[i % R], h, bits, codes, scales)))(i)
            for i in range(reps)]) / 1e3
    return out


def _graph_time(torch, fns, reps=5):
    """Microseconds per call of a sequence of launches, captured once in a HIP
    graph and replayed (no host launch gaps)."""
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
    e0, e1 = _events(torch, 2)
    e0.record()
    for _ in range(reps):
        g.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / (reps * len(fns))


def time_decode(torch, dptq, args):
    """Decode shapes of the LLaMA-3-8B down projection (K = 14336, N = 4096,
    h = 28 x 512): GEMM GB/s and rotate+quantize latency, each as graph-replayed
    back-to-back launches cycling 12 weight copies (more than the 256 MiB
    last-level cache holds)."""
    import numpy as np
    import workloads
    dev = torch.device("cuda:0")
    K, N, h = 14336, 4096, 28 * 512
    rng = np.random.default_rng(2)
    w = torch.from_numpy(workloads.weights(rng, N, K)).to(dev)
    wp, ws = dptq.prepare_weights(w, h)
    del w
    R = 12
    wps = [wp.clone() for _ in range(R)]
    out = {}
    for M in (1, 4, 16):
        x = torch.from_numpy(workloads.student_t(rng, M, K)).to(dev)
        for bits in (4, 8):
            codes, scales = dptq.rotate_quant(x, h, bits)
            y = torch.empty((M, N), dtype=torch.float16, device=dev)
            us = _graph_time(torch, [
                (lambda i: (lambda: dptq.qlinear(codes, scales, bits, wps[i % R], ws, y)))(i)
                for i in range(24)])
            nbytes = N * K // 2 + 4 * N + M * K * bits // 8 + 4 * M + 2 * M * N
            out[f"decode_M{M}_a{bits}"] = {"us": round(us, 2), "GB/s": round(nbytes / us / 1e3, 1)}
            us_rq = _graph_time(torch, [lambda: dptq.rotate_quant(x, h, bits, codes, scales)] * 24)
            out[f"rotate_quant_M{M}_a{bits}_us"] = round(us_rq, 2)
    return out


def time_decode_fused(torch, dptq):
    """Decode from fp16 x (rotate + quantize + GEMM) on both paths of the
    fused entry point and on its automatic choice, at LLaMA decode shapes:
    graph-replayed launches cycling weight copies beyond the last-level cache.
    GB/s counts the weights, their scales, x, the codes written and y."""
    import numpy as np
    import workloads
    dev = torch.device("cuda:0")
    shapes = [("llama2_7b_qkv", 1, 4096, 12288, 4096), ("llama2_7b_qkv", 2, 4096, 12288, 4096),
              ("llama2_7b_o", 1, 4096, 4096, 4096), ("llama2_7b_down", 1, 11008, 4096, 256),
              ("llama3_8b_down", 1, 14336, 4096, 28 * 512), ("llama3_8b_down", 4, 14336, 4096, 28 * 512),
              ("llama3_8b_down", 16, 14336, 4096, 28 * 512), ("llama2_70b_qkv", 8, 8192, 10240, 8192)]
    modes = {"auto": dptq.DECODE_AUTO, "one_launch": dptq.DECODE_ONE_LAUNCH,
             "two_launches": dptq.DECODE_TWO_LAUNCHES}
    rng = np.random.default_rng(6)
    out = {}
    for name, M, K, N, h in shapes:
        R = max(2, (300 << 20) // (N * K // 2))
        gen = torch.Generator(device=dev)
        gen.manual_seed(M + K + N)
        wps = [torch.randint(0, 256, (N, K // 2), dtype=torch.uint8, device=dev, generator=gen)
               for _ in range(R)]
        ws = torch.from_numpy(workloads.random_scales(rng, N)).to(dev)
        x = torch.from_numpy(workloads.student_t(rng, M, K)).to(dev)
        y = torch.empty((M, N), dtype=torch.float16, device=dev)
        for bits in (4, 8):
            codes, scales = dptq.rotate_quant(x, h, bits)
            nbytes = N * K // 2 + 4 * N + 2 * M * K + M * K * bits // 8 + 4 * M + 2 * M * N
            rec = {}
            for mname, mode in modes.items():
                try:
                    us = _graph_time(torch, [
                        (lambda i, mode=mode: (lambda: dptq.qlinear_decode_fused(
                            x, h, bits, wps[i % R], ws, y, codes, scales, mode=mode)))(i)
                        for i in range(24)])
                except dptq.DptqError:
                    continue          # the rows do not fit on chip for one launch
                rec[mname] = {"us": round(us, 2), "GB/s": round(nbytes / us / 1e3, 1)}
            out[f"{name}_M{M}_a{bits}"] = rec
        del wps
        torch.cuda.empty_cache()
    return out


def time_range(torch, dptq, cfg):
    """The range quantizer variant (Eq. 1 with a zero point) at the step's
    shape, next to the symmetric path: rotate + quantize, and the linear (the
    zero-point correction in the GEMM epilogue), each timed over 24
    graph-replayed launches."""
    import numpy as np
    import workloads
    dev = torch.device("cuda:0")
    M, K, N, h = cfg["M"], cfg["K"], cfg["N"], cfg["h"]
    rng = np.random.default_rng(7)
    x = torch.from_numpy(workloads.gauss_outliers(rng, M, K)).to(dev)
    wp = torch.from_numpy(workloads.random_weight_bytes(rng, N, K)).to(dev)
    ws = torch.from_numpy(workloads.random_scales(rng, N)).to(dev)
    sums = dptq.weight_sums(wp)
    y = torch.empty((M, N), dtype=torch.float16, device=dev)
    out = {"weight_sums_us": round(_graph_time(torch, [lambda: dptq.weight_sums(wp, sums)] * 24), 2)}
    for bits in (4, 8):
        c, s = dptq.rotate_quant(x, h, bits)
        cr, sr, zr = dptq.rotate_quant_range(x, h, bits)
        out[f"a{bits}"] = {
            "rotate_quant_us": round(_graph_time(torch, [lambda: dptq.rotate_quant(x, h, bits, c, s)] * 24), 2),
            "rotate_quant_range_us": round(_graph_time(
                torch, [lambda: dptq.rotate_quant_range(x, h, bits, cr, sr, zr)] * 24), 2),
            "qlinear_us": round(_graph_time(torch, [lambda: dptq.qlinear(c, s, bits, wp, ws, y)] * 24), 2),
            "qlinear_range_us": round(_graph_time(
                torch, [lambda: dptq.qlinear_range(cr, sr, zr, bits, wp, ws, sums, y)] * 24), 2),
        }
    return out


def time_calibration(torch, dptq):
    """Residual-dynamics calibration (Eq. 8-11) of one 4096-wide layer over a
    2048-token batch: per-token JR and SNR plus the layer means, graph-replayed
    over 12 input copies; GB/s counts reading x and dx once and writing the
    statistics."""
    import numpy as np
    import workloads
    dev = torch.device("cuda:0")
    T, K, h = 2048, 4096, 4096
    x, dx = workloads.residual_stream(np.random.default_rng(11), 2, T, K)[0]
    R = 12
    xs = [torch.from_numpy(x).to(dev) for _ in range(R)]
    dxs = [torch.from_numpy(dx).to(dev) for _ in range(R)]
    jr = torch.empty(T, dtype=torch.float32, device=dev)
    snr = torch.empty(T, dtype=torch.float32, device=dev)
    means = torch.empty(2, dtype=torch.float64, device=dev)
    out = {}
    for bits in (4, 8):
        us = _graph_time(torch, [
            (lambda i: (lambda: dptq.residual_dynamics(xs[i % R], dxs[i % R], h, bits,
                                                       jr=jr, snr=snr, means=means)))(i)
            for i in range(24)])
        nbytes = 2 * 2 * T * K + 8 * T + 16
        out[f"residual_dynamics_a{bits}"] = {"us": round(us, 2), "GB/s": round(nbytes / us / 1e3, 1)}
    return out


def time_kv(torch, dptq):
    """Group-wise KV4 codec on one layer's keys of a 32-sequence x 2048-token
    prefill for LLaMA-3-8B (8 KV heads x 128 = 1024 per token, group 128):
    quantize and reconstruct, graph-replayed over 4 distinct caches (> 256 MiB
    each way).  Algorithmic bytes: 2 B in, 0.5 B of codes and 8 B of (s, m)
    per 128-element group out, and the reverse for the reconstruction."""
    import numpy as np
    dev = torch.device("cuda:0")
    T, D, g = 32 * 2048, 1024, 128
    gen = torch.Generator(device=dev)
    gen.manual_seed(8)
    R = 4
    xs = [torch.randn((T, D), device=dev, generator=gen).half() for _ in range(R)]
    outs = [dptq.kv_quant(x, g) for x in xs]
    rec = [torch.empty((T, D), dtype=torch.float16, device=dev) for _ in range(R)]
    nbytes = 2 * T * D + T * D // 2 + 8 * T * (D // g)
    q_us = _graph_time(torch, [
        (lambda i: (lambda: dptq.kv_quant(xs[i % R], g, *outs[i % R])))(i) for i in range(8)])
    d_us = _graph_time(torch, [
        (lambda i: (lambda: dptq.kv_dequant(*outs[i % R], g, out=rec[i % R])))(i) for i in range(8)])
    del xs, outs, rec
    torch.cuda.empty_cache()
    return {"tokens": T, "row": D, "group": g,
            "quant_us": round(q_us, 2), "quant_GB/s": round(nbytes / q_us / 1e3, 1),
            "dequant_us": round(d_us, 2), "dequant_GB/s": round(nbytes / d_us / 1e3, 1)}


def time_stack(torch, dptq, name, Ms, reps=3):
    """End-to-end time of every linear of a whole layer stack (rotate+quantize
    and GEMM per linear, layer bits from the policy), captured as one HIP graph
    per policy and replayed.  Each layer has its own weights (random packed
    code bytes drawn on the device: the time does not depend on their values);
    each linear's input is the seeded stack input of a mid-stack layer.  At
    decode sizes (M <= 16) each linear is one call of the decode entry point,
    which picks one launch or two.
    Returns ms per stack for all-4-bit, the paper's default set, a seeded
    4-layer mask and all-8-bit activations, and the mixed/all-4-bit ratios.
    At prefill sizes the same policies run again with the 4-bit layers on the
    FP6 path (rotate+quantize into the FP6 layout, FP6 GEMM against weights
    packed once into it) and the 8-bit layers on the int8 path against weights
    packed once into the 8-bit activation order: the "_fp6" entries."""
    import workloads
    dev = torch.device("cuda:0")
    cfg = workloads.CONFIGS[name]
    L, lins = cfg["L"], cfg["linears"]
    gen = torch.Generator(device=dev)
    gen.manual_seed(cfg["seed"])
    W = [[(torch.randint(0, 256, (N, K // 2), dtype=torch.uint8, device=dev, generator=gen),
           torch.rand(N, device=dev, generator=gen) * 1e-3 + 1e-4)
          for _, K, N, _ in lins] for _ in range(L)]
    wbytes = sum(N * K // 2 + 4 * N for _, K, N, _ in lins) * L
    policies = {"all_a4": [4] * L, "default": dptq.layer_policy(L),
                "seeded_mask": dptq.layer_policy(L, workloads.layer_mask(L, 4, cfg["mask_seed"])),
                "all_a8": [8] * L}
    out = {"weights_GB": round(wbytes / 1e9, 2)}
    W6 = W8 = None
    if any(M > 16 for M in Ms):
        W6 = [[dptq.pack_fp6(W[l][i][0]) for i in range(len(lins))] for l in range(L)]
        W8 = [[dptq.pack_w4_a8(W[l][i][0]) for i in range(len(lins))] for l in range(L)]
    for M in Ms:
        X = [torch.from_numpy(workloads.stack_layer_input(name, L // 2, n, M=M)).to(dev)
             for n, *_ in lins]
        Kmax = max(K for _, K, _, _ in lins)
        Nmax = max(N for _, _, N, _ in lins)
        cbuf = torch.empty(M * Kmax, dtype=torch.uint8, device=dev)
        sbuf = torch.empty(M, dtype=torch.float32, device=dev)
        ybuf = torch.empty(M * Nmax, dtype=torch.float16, device=dev)
        res = {}
        for pname, bits in policies.items():
            def run(bits=bits):
                for l in range(L):
                    b = bits[l]
                    for i, (_, K, N, h) in enumerate(lins):
                        dt = torch.uint8 if b == 4 else torch.int8
                        codes = cbuf[: M * K * b // 8].view(dt).view(M, K * b // 8)
                        y = ybuf[: M * N].view(M, N)
                        if M <= 16:   # the decode entry point's own choice of path
                            dptq.qlinear_decode_fused(X[i], h, b, W[l][i][0], W[l][i][1], y, codes,
                                                      sbuf, mode=dptq.DECODE_AUTO)
                        else:
                            dptq.rotate_quant(X[i], h, b, codes, sbuf)
                            dptq.qlinear(codes, sbuf, b, W[l][i][0], W[l][i][1], y)
            res[pname] = _graph_time(torch, [run], reps=reps) / 1e3
        if M > 16:
            a6buf = torch.empty(max(dptq.fp6_bytes(M, K) for _, K, _, _ in lins), dtype=torch.uint8,
                                device=dev)
            for pname in ("all_a4", "default", "seeded_mask"):
                bits = policies[pname]

                def run6(bits=bits):
                    for l in range(L):
                        b = bits[l]
                        for i, (_, K, N, h) in enumerate(lins):
                            y = ybuf[: M * N].view(M, N)
                            if b == 4:
                                a6 = a6buf[: dptq.fp6_bytes(M, K)]
                                dptq.rotate_quant_fp6(X[i], h, a6, sbuf)
                                dptq.qlinear_fp6(a6, sbuf, W6[l][i], W[l][i][1], M, K, N, y)
                            else:
                                codes = cbuf[: M * K].view(torch.int8).view(M, K)
                                dptq.rotate_quant(X[i], h, 8, codes, sbuf)
                                dptq.qlinear_a8(codes, sbuf, W8[l][i], W[l][i][1], y)
                res[pname + "_fp6"] = _graph_time(torch, [run6], reps=reps) / 1e3
            del a6buf
        ops = 2.0 * M * sum(K * N for _, K, N, _ in lins) * L
        ent = {f"{p}_ms": round(v, 3) for p, v in res.items()}
        ent["default_over_all_a4"] = round(res["default"] / res["all_a4"], 4)
        ent["seeded_mask_over_all_a4"] = round(res["seeded_mask"] / res["all_a4"], 4)
        ent["all_a4_TOPS"] = round(ops / (res["all_a4"] * 1e-3) / 1e12, 1)
        ent["all_a4_weight_GB/s"] = round(wbytes / (res["all_a4"] * 1e-3) / 1e9, 1)
        if "all_a4_fp6" in res:
            ent["default_fp6_over_all_a4_fp6"] = round(res["default_fp6"] / res["all_a4_fp6"], 4)
            ent["seeded_mask_fp6_over_all_a4_fp6"] = round(res["seeded_mask_fp6"] / res["all_a4_fp6"], 4)
            ent["all_a4_fp6_TOPS"] = round(ops / (res["all_a4_fp6"] * 1e-3) / 1e12, 1)
        out[f"M{M}"] = ent
        del X, cbuf, ybuf
    del W, W6, W8
    torch.cuda.empty_cache()
    return out


def cpu_baseline(cfg, rows, seed=123):
    """Time the CPU oracle on a bounded sample: `rows` token rows of the same
    layer, both precisions (rotation + quantization + exact GEMM + epilogue)."""
    import numpy as np
    import workloads
    from oracle import rotate_quant_ref, qlinear_ref
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([d.get("num_threads", 1) for d in threadpool_info()] or [1])
    except Exception:
        blas_threads = 1
    M, K, N, h = cfg["M"], cfg["K"], cfg["N"], cfg["h"]
    rng = np.random.default_rng(seed)
    x = workloads.gauss_outliers(rng, rows, K)
    wp = workloads.random_weight_bytes(rng, N, K)
    ws = workloads.random_scales(rng, N)
    t0 = time.perf_counter()
    for bits in (4, 8):
        c, s = rotate_quant_ref(x, h, bits)
        qlinear_ref(c, s, bits, wp, ws)
    dt = time.perf_counter() - t0
    ops = 2 * (2.0 * rows * N * K)
    return {"value": round(ops / dt / 1e12, 6), "unit": "TOPS", "cores": int(blas_threads),
            "kind": "oracle",
            "sample": f"{rows} of {M} token rows, A4 and A8, K={K}, N={N}, h={h}: "
                      f"rotation, quantization, exact GEMM and epilogue; {dt:.1f} s"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); "
              "the library has no multi-GPU path (the sharding plan is documented, not built)", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2606_12487_amd as dptq
    import workloads
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dptq.lib()
    cfg = workloads.CONFIGS["llama2_7b_qkv"]
    M, K, N = cfg["M"], cfg["K"], cfg["N"]
    if args.only:
        run_only(torch, dptq, cfg, args)
        return

    wall, gpu_ms, seq, wall_graph = time_layer(torch, dptq, cfg, args)
    ops_gemm = 2.0 * M * N * K
    ops_step = ops_gemm * len(seq)
    value = ops_step * args.steps / wall / 1e12
    ms_step = wall * 1e3 / args.steps

    per = time_kernels(torch, dptq, cfg, args, seq)
    step_kernels = {"rotate_quant_fp6_a4": "rq_pow2_kernel<__half, 4, false, 12, false, true>",
                    "gemm_fp6_a4": "qgemm_fp6<false, false>",
                    "rotate_quant_a8": "rq_pow2_kernel<__half, 8, false, 12, false, false>",
                    "gemm_a8": "qgemm_prefill_wide<8, false, true>"}
    dominant = max(step_kernels, key=lambda k: per[k])
    dom_ms = per[dominant]
    fp6_ms = per["gemm_fp6_a4"]
    k1_bytes = 2 * M * K + dptq.fp6_bytes(M, K) + 4 * M
    rq6_ms = per["rotate_quant_fp6_a4"]
    is_fp6 = dominant == "gemm_fp6_a4"
    dom_peak = PEAK_FP6_TOPS if is_fp6 else PEAK_INT8_TOPS
    dom_achieved = ops_gemm / (dom_ms * 1e-3) / 1e12
    rec = {
        "metric": METRIC, "value": round(value, 3), "unit": "TOPS", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": "llama2-7b fused qkv qlinear, rotate+quant+GEMM at A4 (fp6 matrix "
                               "cores) then A8 (int8 matrix cores)",
                   "M": M, "K": K, "N": N, "had_size": cfg["h"], "bits": list(seq),
                   "parallelism": "none"},
        "roofline": {"bound": "mfma", "kernel": step_kernels[dominant],
                     "achieved": round(dom_achieved, 2), "peak": dom_peak,
                     "unit": "TFLOP/s", "frac": round(dom_achieved / dom_peak, 4),
                     "traffic": None if is_fp6 else measured_traffic()},
        "roofline_fp6_gemm": {"bound": "mfma", "kernel": step_kernels["gemm_fp6_a4"],
                              "achieved": round(ops_gemm / (fp6_ms * 1e-3) / 1e12, 2),
                              "peak": PEAK_FP6_TOPS, "unit": "TFLOP/s",
                              "frac": round(ops_gemm / (fp6_ms * 1e-3) / 1e12 / PEAK_FP6_TOPS, 4),
                              "frac_of_int8_peak": round(ops_gemm / (fp6_ms * 1e-3) / 1e12 / PEAK_INT8_TOPS, 4)},
        "gpu_ms_per_step": round(gpu_ms / args.steps, 4),
        "graph": {"value": round(ops_step * args.steps / wall_graph / 1e12, 3),
                  "ms_per_step": round(wall_graph * 1e3 / args.steps, 4),
                  "note": "the same steps replayed from captured HIP graphs"},
        "kernels_ms": {k: round(v, 4) for k, v in per.items()},
        "rotate_quant_fp6_a4": {"bound": "alu", "GB/s": round(k1_bytes / (rq6_ms * 1e-3) / 1e9, 1),
                                "frac_of_hbm_peak": round(k1_bytes / (rq6_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)},
    }
    # Decode GB/s (the metric's second half): config 3's down projection at
    # M = 1, 4, 16, a few seconds.
    rec["decode"] = time_decode(torch, dptq, args)
    if args.extended:
        rec["decode_fused"] = time_decode_fused(torch, dptq)
        rec["range_quantizer"] = time_range(torch, dptq, cfg)
        rec["calibration"] = time_calibration(torch, dptq)
        rec["kv4"] = time_kv(torch, dptq)
        rec["stacks"] = {"llama2_7b_32_layers": time_stack(torch, dptq, "llama2_7b_stack", (2048, 8, 1)),
                         "llama2_70b_80_layers": time_stack(torch, dptq, "llama2_70b_layer", (4096, 8, 1))}
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(cfg, args.cpu_rows)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
