"""Seeded synthetic workloads for the quantized linear layer.

Shared by the tests and the benchmark.  This module only draws inputs: it holds
none of the method's arithmetic (no rotation, no quantization, no GEMM).

The paper's own activations (LLaMA residual streams on WikiText-2 calibration
text) and weights are not available; these generators stand in for their
shapes and value structure:

* Gaussian tokens with a few massive channels (the massive activations of
  Section 2 that dominate the per-token range);
* heavy-tailed Student-t(3) inputs for the MLP down projection;
* residual-stream inputs whose massive channels switch on and off across
  seeded depth phases (the three-phase pattern of Section 2 and Eq. 6-7);
* weights ~ N(0, 0.02) in fp32, quantized offline by the library.
"""

import numpy as np

__all__ = ["CONFIGS", "gauss_massive", "gauss_outliers", "student_t",
           "residual_phase", "residual_stream", "weights", "layer_mask", "activations_for",
           "stack_layer_input", "stack_weights"]

# name -> description.  Linear tuples are (name, K, N, had_size).
CONFIGS = {
    "tiny": dict(M=16, K=256, N=512, h=256, seed=0, kind="gauss_massive",
                 bits=(4, 8)),
    "llama2_7b_qkv": dict(M=2048, K=4096, N=12288, h=4096, seed=1,
                          kind="gauss_outliers", bits=(4, 8)),
    "llama3_8b_down": dict(Ms=(1, 4, 16, 2048), K=14336, N=4096, h=28 * 512,
                           seed=2, kind="student_t", bits=(4, 8)),
    "llama2_7b_stack": dict(L=32, M=2048, seed=4, mask_seed=3,
                            linears=[("qkv", 4096, 12288, 4096),
                                     ("o", 4096, 4096, 4096),
                                     ("gate_up", 4096, 22016, 4096),
                                     ("down", 11008, 4096, 256)]),
    "llama2_70b_layer": dict(L=80, M=4096, Ms=(4096, 8), seed=5, mask_seed=5,
                             linears=[("qkv", 8192, 10240, 8192),
                                      ("o", 8192, 8192, 8192),
                                      ("gate_up", 8192, 57344, 8192),
                                      ("down", 28672, 8192, 28 * 1024)]),
}

_F16_MAX = 65504.0


def _to_f16(x):
    return np.clip(x, -_F16_MAX, _F16_MAX).astype(np.float16)


def gauss_massive(rng, M, K, n_channels=2, factor=100.0):
    """N(0,1) tokens with n_channels seeded channels scaled by `factor`."""
    x = rng.standard_normal((M, K), dtype=np.float32)
    cols = rng.choice(K, n_channels, replace=False)
    x[:, cols] *= np.float32(factor)
    return _to_f16(x)


def gauss_outliers(rng, M, K, n_channels=4, lo=50.0, hi=200.0):
    """N(0,1) tokens with n_channels seeded channels scaled by U[lo, hi] each."""
    x = rng.standard_normal((M, K), dtype=np.float32)
    cols = rng.choice(K, n_channels, replace=False)
    x[:, cols] *= rng.uniform(lo, hi, n_channels).astype(np.float32)
    return _to_f16(x)


def student_t(rng, M, K, nu=3.0):
    """Heavy-tailed Student-t(nu) tokens (SwiGLU-output-like), fp16."""
    return _to_f16(rng.standard_t(nu, size=(M, K)).astype(np.float32))


def residual_phase(rng, M, K, layer, phase, channels, factors):
    """Residual-stream input of one layer: N(0,1) plus massive channels that are
    switched on only for layers inside the seeded phase window [p1, p2].

    channels: the massive channel indices; factors: (first-token, other-token)
    multipliers per channel.  Token 0 plays the role of the BOS token.
    """
    x = rng.standard_normal((M, K), dtype=np.float32)
    p1, p2 = phase
    if p1 <= layer <= p2:
        for c, (f0, f1) in zip(channels, factors):
            x[0, c] *= np.float32(f0)
            x[1:, c] *= np.float32(f1)
    return _to_f16(x)


def residual_phase_plan(rng, K, L):
    """Seeded phase window and massive channels for a layer stack."""
    p1 = int(rng.integers(2, 5))
    p2 = int(rng.integers(L - 4, L))
    n = int(rng.integers(2, 5))
    channels = rng.choice(K, n, replace=False)
    factors = [(float(rng.uniform(100, 1000)), float(rng.uniform(10, 50)))
               for _ in range(n)]
    return (p1, p2), channels, factors


def residual_stream(rng, L, T, d, n_massive=3, early=3):
    """Per-layer (x, dx) pairs, fp16 [T, d] each, of a synthetic residual stream
    x^(l+1) = x^(l) + dx^(l) with the three-phase depth pattern of Section 2:
    in the first `early` layers massive activations emerge (large updates on a
    few seeded channels, largest on token 0, plus updates of the stream's own
    size); in the middle layers the updates are small relative to the stream;
    the last layer redistributes the massive channels with another large
    update.  The states are kept in fp32 and handed out rounded to fp16."""
    x = (0.5 * rng.standard_normal((T, d))).astype(np.float32)
    channels = rng.choice(d, n_massive, replace=False)
    out = []
    for layer in range(L):
        scale = float(np.sqrt(np.mean(x.astype(np.float64) ** 2)))
        if layer < early:
            dx = (2.0 * scale) * rng.standard_normal((T, d))
            dx[:, channels] += rng.uniform(20, 60, size=n_massive) * scale
            dx[0, channels] += rng.uniform(100, 300, size=n_massive) * scale
        elif layer == L - 1:
            dx = (2.0 * scale) * rng.standard_normal((T, d))
            dx[:, channels] -= 0.9 * x[:, channels]
        else:
            dx = (0.05 * scale) * rng.standard_normal((T, d))
        dx = dx.astype(np.float32)
        out.append((_to_f16(x), _to_f16(dx)))
        x = x + dx
    return out


def weights(rng, N, K, std=0.02):
    """Full-precision weights ~ N(0, std^2), fp32 [N, K] (out x in)."""
    w = rng.standard_normal((N, K), dtype=np.float32)
    w *= np.float32(std)
    return w


def layer_mask(L, n_sensitive=4, seed=3):
    """Seeded mask marking n_sensitive of L layers for 8-bit activations."""
    rng = np.random.default_rng(seed)
    mask = np.zeros(L, dtype=np.uint8)
    mask[rng.choice(L, n_sensitive, replace=False)] = 1
    return mask


def activations_for(name, M=None, seed=None):
    """Activations of one of the single-linear configs, as the config describes."""
    cfg = CONFIGS[name]
    rng = np.random.default_rng(cfg["seed"] if seed is None else seed)
    M = cfg.get("M") if M is None else M
    K = cfg["K"]
    kind = cfg["kind"]
    if kind == "gauss_massive":
        return gauss_massive(rng, M, K)
    if kind == "gauss_outliers":
        return gauss_outliers(rng, M, K)
    if kind == "student_t":
        return student_t(rng, M, K)
    raise ValueError(kind)


def random_code_bytes(rng, M, K, bits):
    """Seeded activation code buffers for GEMM tests: 4-bit -> uint8 [M, K/2]
    (every byte is a valid pair of nibbles), 8-bit -> int8 [M, K] in [-127, 127]."""
    if bits == 4:
        return rng.integers(0, 256, size=(M, K // 2), dtype=np.uint8)
    return rng.integers(-127, 128, size=(M, K), dtype=np.int8)


def random_weight_bytes(rng, N, K):
    """Seeded packed 4-bit weight buffer uint8 [N, K/2]."""
    return rng.integers(0, 256, size=(N, K // 2), dtype=np.uint8)


def random_sign_bits(rng, K):
    """Seeded random signs for the randomized rotation, as the bitmask the
    library takes: uint8 [ceil(K/8)], bit (k & 7) of byte k >> 3 set = -1."""
    return rng.integers(0, 256, size=((K + 7) // 8,), dtype=np.uint8)


def random_scales(rng, n, lo=1e-4, hi=1e-1):
    """Seeded positive fp32 scales."""
    return rng.uniform(lo, hi, n).astype(np.float32)


def stack_layer_input(name, layer, linear, M=None):
    """Input of one linear of one layer of a stack config, fp16 [M, K].

    llama2_7b_stack: the qkv and gate_up inputs follow the residual model
    (massive channels switched on inside the stack's seeded phase window),
    o inputs are N(0,1) and down inputs Student-t(3).  llama2_70b_layer: the
    qkv, o and gate_up inputs are N(0,1) with outlier channels as in the
    7B QKV config, down inputs Student-t(3).  Every (layer, linear) pair has
    its own seed."""
    cfg = CONFIGS[name]
    lin = {n: (K, N, h) for n, K, N, h in cfg["linears"]}
    K = lin[linear][0]
    M = cfg["M"] if M is None else M
    order = [n for n, *_ in cfg["linears"]].index(linear)
    rng = np.random.default_rng([cfg["seed"], layer, order])
    if linear == "down":
        return student_t(rng, M, K)
    if name == "llama2_7b_stack":
        if linear == "o":
            return _to_f16(rng.standard_normal((M, K), dtype=np.float32))
        plan = residual_phase_plan(np.random.default_rng(cfg["seed"]), K, cfg["L"])
        return residual_phase(rng, M, K, layer, *plan)
    return gauss_outliers(rng, M, K)


def stack_weights(name, layer, linear):
    """fp32 weights [N, K] of one linear of one layer of a stack config."""
    cfg = CONFIGS[name]
    names = [n for n, *_ in cfg["linears"]]
    _, K, N, _ = cfg["linears"][names.index(linear)]
    return weights(np.random.default_rng([cfg["seed"], layer, names.index(linear), 1]), N, K)
