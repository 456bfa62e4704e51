"""Seeded synthetic inputs for the Q4NX projection path, shared by the oracle
side (tests, CPU baseline) and the HIP side (tests, benchmark).

This module only *draws* inputs. It holds none of the method's arithmetic:
no packing, no dequantization (Eq. 3) and no projection (Eq. 14/15).  The
only rounding it does is the float32 -> bfloat16 conversion of freshly drawn
values, and for that it calls torch's own conversion, so it shares no code
with the oracle's bit-level bf16 helpers.

Shapes are the Gemma3 projections (N = output features, K = input features).
The paper fixes the 4B attention geometry (model dimension 2560, 8 heads,
4 KV groups, head dimension 256, 34 layers; Sec. 2.2, caption of the Gemma3-4B
layer figure); the FFN widths, the 1B and 27B models and the vocabulary size
are the public Gemma3 configurations.

Random streams (one per (seed, layer, projection)):
    weights:     PCG64(SeedSequence([seed, layer, proj]))
    activations: PCG64(SeedSequence([seed, layer, proj, 1]))
Draw order for the weights:
    1. codes   : N*K/16 raw 64-bit words; word w supplies codes 16w..16w+15
                 (row-major over [N][K]), 4 bits each from the least
                 significant end, so every code is uniform on 0..15.
    2. scales  : bf16(|standard_normal(N, K/32)| * 0.02)
    3. offsets : mode "zp"      -> z ~ U{0..15}; bf16(-f32(scale) * z)
                 mode "literal" -> bf16(uniform(0, 15))
Activations: bf16(standard_normal(shape)).
"""
from __future__ import annotations

import numpy as np

PROJ_IDS = {"q": 0, "k": 1, "v": 2, "o": 3, "gate": 4, "up": 5, "down": 6, "lm_head": 7}

# (name, N, K) per projection, in the order a layer applies them.
MODELS = {
    "1b": {
        "layers": 26,
        "proj": [("q", 1024, 1152), ("k", 256, 1152), ("v", 256, 1152), ("o", 1152, 1024),
                 ("gate", 6912, 1152), ("up", 6912, 1152), ("down", 1152, 6912)],
        "lm_head": None,
    },
    "4b": {
        "layers": 34,
        "proj": [("q", 2048, 2560), ("k", 1024, 2560), ("v", 1024, 2560), ("o", 2560, 2048),
                 ("gate", 10240, 2560), ("up", 10240, 2560), ("down", 2560, 10240)],
        "lm_head": ("lm_head", 262144, 2560),
    },
    "27b": {
        "layers": 62,
        "proj": [("q", 4096, 5376), ("k", 2048, 5376), ("v", 2048, 5376), ("o", 5376, 4096),
                 ("gate", 21504, 5376), ("up", 21504, 5376), ("down", 5376, 21504)],
        "lm_head": None,
    },
}

# Attention geometry (query heads H, KV groups G, head dimension d) and the
# layer pattern: 5 sliding-window layers (window 1024) per global layer,
# starting with a sliding-window layer (Sec. 2.2).  The 4B geometry is the
# paper's; the 1B and 27B ones are the public Gemma3 configurations.
ATTENTION = {
    "1b": {"H": 4, "G": 1, "d": 256},
    "4b": {"H": 8, "G": 4, "d": 256},
    "27b": {"H": 32, "G": 16, "d": 128},
}
SWA_WINDOW = 1024
GLOBAL_EVERY = 6


def is_global_layer(layer: int) -> bool:
    return (layer + 1) % GLOBAL_EVERY == 0


# The five workloads: model, token rows M, whether lm_head runs once per step.
CONFIGS = {
    0: {"name": "gemma3-1b q_proj GEMV 1024x1152", "model": "1b", "M": [1], "single": ("q", 1024, 1152)},
    1: {"name": "gemma3-1b decode step, 26 layers", "model": "1b", "M": [1]},
    2: {"name": "gemma3-4b decode step, 34 layers + lm_head", "model": "4b", "M": [1], "lm_head": True},
    3: {"name": "gemma3-4b prefill chunk, M=2048, 34 layers", "model": "4b", "M": [2048]},
    4: {"name": "gemma3-27b, 62 layers, M=1 decode and M=4096 prefill", "model": "27b", "M": [1, 4096]},
}

SCALE_STD = np.float32(0.02)
# Smallest non-zero magnitude the format accepts for a scale or offset: 2^-100.
_MIN_MAG_BITS = 27 << 7


def _to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """float32 array -> bf16 bit patterns (uint16), rounded by torch (RNE)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy()


def _bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    import torch
    t = torch.from_numpy(np.ascontiguousarray(b).view(np.int16))
    return t.view(torch.bfloat16).to(torch.float32).numpy()


def _clamp_tiny(bits: np.ndarray) -> np.ndarray:
    """Raise non-zero magnitudes below 2^-100 to 2^-100, keeping the sign."""
    mag = bits & 0x7FFF
    tiny = (mag != 0) & (mag < _MIN_MAG_BITS)
    if tiny.any():
        bits = bits.copy()
        bits[tiny] = (bits[tiny] & 0x8000) | _MIN_MAG_BITS
    return bits


def weight_rng(seed: int, layer: int, proj: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, layer, proj])))


def act_rng(seed: int, layer: int, proj: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, layer, proj, 1])))


def draw_codes(rng: np.random.Generator, N: int, K: int) -> np.ndarray:
    """Uniform 4-bit codes u8[N][K] in 0..15 (16 codes per raw 64-bit draw)."""
    n = N * K
    if n % 16:
        raise ValueError("N*K must be a multiple of 16")
    words = rng.bit_generator.random_raw(n // 16).astype(np.uint64)
    byts = words.view(np.uint8)          # little-endian: byte b of word w
    codes = np.empty(n, dtype=np.uint8)
    codes[0::2] = byts & 0x0F
    codes[1::2] = byts >> 4
    return codes.reshape(N, K)


def gen_weights(N: int, K: int, seed: int = 0, layer: int = 0, proj: int = 0,
                offset_mode: str = "zp"):
    """Codes u8[N][K], scales u16[N][K/32], offsets u16[N][K/32] (bf16 bits)."""
    if K % 32:
        raise ValueError("K must be a multiple of 32")
    rng = weight_rng(seed, layer, proj)
    codes = draw_codes(rng, N, K)
    G = K // 32
    s32 = np.abs(rng.standard_normal((N, G), dtype=np.float32)) * SCALE_STD
    scales = _clamp_tiny(_to_bf16_bits(s32))
    if offset_mode == "zp":
        z = rng.integers(0, 16, size=(N, G), dtype=np.int64).astype(np.float32)
        offsets = _to_bf16_bits(-_bf16_bits_to_f32(scales) * z)
    elif offset_mode == "literal":
        offsets = _to_bf16_bits(rng.uniform(0.0, 15.0, size=(N, G)).astype(np.float32))
    else:
        raise ValueError(f"unknown offset_mode {offset_mode!r}")
    offsets = _clamp_tiny(offsets)
    return codes, scales, offsets


def gen_activations(shape, seed: int = 0, layer: int = 0, proj: int = 0) -> np.ndarray:
    """bf16 bits of standard-normal activations (x[K] or X[M][K])."""
    rng = act_rng(seed, layer, proj)
    return _to_bf16_bits(rng.standard_normal(shape, dtype=np.float32))


def gen_edge_weights(N: int, K: int, seed: int = 0):
    """Weights that exercise the format's corner values: every code 0..15,
    zero scales, negative scales, +0/-0 offsets and magnitudes at both ends
    of the accepted range (2^-100 and just below 2^101)."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 999])))
    codes = draw_codes(rng, N, K)
    G = K // 32
    choices_s = np.array([0x0000, 0x8000, 0x3F80, 0xBF80, 0x3C00, 0xBCA3, 0x0D80, 0x8D80,
                          0x71FF, 0xF1FF, 0x3E4C, 0x4170], dtype=np.uint16)
    choices_m = np.array([0x0000, 0x8000, 0x3F80, 0xC0A0, 0x0D80, 0x8D80, 0x71FF, 0xF1FF,
                          0x3DCD, 0xBE00, 0x42F6, 0x4000], dtype=np.uint16)
    scales = choices_s[rng.integers(0, len(choices_s), size=(N, G))]
    offsets = choices_m[rng.integers(0, len(choices_m), size=(N, G))]
    return codes, scales, offsets


def gen_mx_weights(N: int, K: int, seed: int = 0, layer: int = 0, proj: int = 0, mode: str = "model"):
    """MXFP4-variant weights: FP4 E2M1 codes u8[N][K] (uniform 0..15) and E8M0
    scale bytes u8[N][K/32].  "model": scale exponents 2^-8..2^-5, the range a
    weight matrix of standard deviation ~0.02 gets (largest FP4 magnitude 6);
    "edge": scale bytes over the whole accepted range 27..227, both ends and
    1 (byte 127) included."""
    if K % 32:
        raise ValueError("K must be a multiple of 32")
    rng = weight_rng(seed, layer, proj + 100)
    codes = draw_codes(rng, N, K)
    G = K // 32
    if mode == "model":
        scales = rng.integers(119, 123, size=(N, G), dtype=np.int64).astype(np.uint8)
    elif mode == "edge":
        pick = np.array([27, 28, 60, 100, 126, 127, 128, 150, 200, 226, 227], dtype=np.uint8)
        scales = pick[rng.integers(0, len(pick), size=(N, G))]
    else:
        raise ValueError(f"unknown mode {mode!r}")
    return codes, scales


def device_act_seed(seed: int, layer: int, proj: int) -> int:
    """64-bit seed of the on-device activation stream of (seed, layer, proj)."""
    st = np.random.SeedSequence([seed, layer, proj, 2]).generate_state(2, dtype=np.uint32)
    return int(st[0]) | (int(st[1]) << 32)


def gen_activations_device(shape, seed: int = 0, layer: int = 0, proj: int = 0, device="cuda"):
    """bf16 standard-normal activations drawn directly on the GPU with torch's
    seeded generator (for large prefill inputs of the benchmark)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(device_act_seed(seed, layer, proj) & ((1 << 63) - 1))
    return torch.randn(shape, generator=g, device=device, dtype=torch.float32).to(torch.bfloat16)
