"""Counter-based seeded generators with bit-identical numpy and torch backends.

Every synthetic tensor is a pure function of (seed, tensor name, element
index).  Element i of a stream draws one 64-bit word from the SplitMix64
sequence (Steele, Lea and Flood, "Fast splittable pseudorandom number
generators", OOPSLA 2014): the state advances by the golden-ratio increment
and the word is the state passed through SplitMix64's published finaliser.
The stream key is the finaliser applied to seed * increment XOR FNV-1a-64 of
the tensor name.

Weights use an approximately normal value: the sum of the word's four 16-bit
fields (an Irwin-Hall(4) variable), centred and scaled to the requested
standard deviation.  Every step is integer arithmetic or a single float32
multiply, so the numpy and torch backends (any device) produce the same float32
value, and the same bf16 value after round-to-nearest-even.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

MASK64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15
MIX1 = 0xBF58476D1CE4E5B9
MIX2 = 0x94D049BB133111EB
# standard deviation of the sum of four independent uniform integers on [0, 65535]
IH4_STD = math.sqrt((65536.0 ** 2 - 1.0) / 3.0)
IH4_MEAN = 4 * 65535 // 2  # = 131070, the exact mean of the four-field sum


@dataclass(frozen=True)
class ModelShape:
    """Shape of a bidirectional masked-diffusion transformer."""
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    d_ffn: int
    vocab: int
    rope_base: float = 10000.0
    rms_eps: float = 1e-5

    @property
    def mask_id(self) -> int:
        # the last vocabulary entry is the [MASK] token
        return self.vocab - 1

    def n_params(self) -> int:
        d, f, v = self.d_model, self.d_ffn, self.vocab
        per_layer = 3 * d * d + d * d + 2 * f * d + d * f
        return self.n_layers * per_layer + 2 * v * d


# 2-layer fp32 parity model and the 8B-class bf16 model
TINY = ModelShape(n_layers=2, d_model=256, n_heads=4, head_dim=64, d_ffn=1024, vocab=1024)
B8 = ModelShape(n_layers=32, d_model=4096, n_heads=32, head_dim=128, d_ffn=12288, vocab=126464)


def fnv1a64(name: str) -> int:
    """FNV-1a 64-bit hash of a UTF-8 string (offset basis 0xcbf29ce484222325)."""
    h = 0xCBF29CE484222325
    for byte in name.encode("utf-8"):
        h ^= byte
        h = (h * 0x100000001B3) & MASK64
    return h


def _mix_int(z: int) -> int:
    z &= MASK64
    z = ((z ^ (z >> 30)) * MIX1) & MASK64
    z = ((z ^ (z >> 27)) * MIX2) & MASK64
    return z ^ (z >> 31)


def stream_key(seed: int, name: str) -> int:
    return _mix_int(((seed * GAMMA) & MASK64) ^ fnv1a64(name))


# ---------------------------------------------------------------- numpy backend

def _mix_np(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * np.uint64(MIX1)
    z = (z ^ (z >> np.uint64(27))) * np.uint64(MIX2)
    return z ^ (z >> np.uint64(31))


def counter_u64_np(key: int, start: int, n: int) -> np.ndarray:
    """Words start .. start+n-1 of the stream with the given key (uint64)."""
    idx = np.arange(start, start + n, dtype=np.uint64) + np.uint64(1)
    with np.errstate(over="ignore"):
        return _mix_np(idx * np.uint64(GAMMA) + np.uint64(key))


def _ih4_np(r: np.ndarray) -> np.ndarray:
    m = np.uint64(0xFFFF)
    s = (r & m) + ((r >> np.uint64(16)) & m) + ((r >> np.uint64(32)) & m) + (r >> np.uint64(48))
    return (s.astype(np.int64) - IH4_MEAN).astype(np.float32)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bits."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def weight_np(seed: int, name: str, shape, std: float = 0.02, dtype: str = "bf16") -> np.ndarray:
    """Approximately N(0, std^2) weights as float32 (bf16-representable if dtype='bf16')."""
    n = int(np.prod(shape))
    with np.errstate(over="ignore"):
        x = _ih4_np(counter_u64_np(stream_key(seed, name), 0, n)) * np.float32(std / IH4_STD)
    if dtype == "bf16":
        x = bf16_bits_to_f32(f32_to_bf16_bits(x))
    elif dtype != "f32":
        raise ValueError(dtype)
    return x.reshape(shape)


def tokens_np(seed: int, name: str, n: int, n_values: int) -> np.ndarray:
    """n integers uniform on [0, n_values) (int32)."""
    r = counter_u64_np(stream_key(seed, name), 0, n)
    return ((r >> np.uint64(33)) % np.uint64(n_values)).astype(np.int32)


def uniform01_np(seed: int, name: str, n: int) -> np.ndarray:
    """n float64 values uniform on [0, 1) from the top 53 bits of each word."""
    r = counter_u64_np(stream_key(seed, name), 0, n)
    return (r >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)


def hidden_np(seed: int, name: str, shape, dtype: str = "bf16") -> np.ndarray:
    """Synthetic final hidden states with unit variance per element."""
    return weight_np(seed, name, shape, std=1.0, dtype=dtype)


# ---------------------------------------------------------------- torch backend

def _signed(c: int) -> int:
    return c - (1 << 64) if c >= (1 << 63) else c


def _lsr(t, k: int):
    # logical right shift of int64 bits
    return (t >> k) & ((1 << (64 - k)) - 1)


def _mix_torch(z):
    z = (z ^ _lsr(z, 30)) * _signed(MIX1)
    z = (z ^ _lsr(z, 27)) * _signed(MIX2)
    return z ^ _lsr(z, 31)


def counter_u64_torch(key: int, start: int, n: int, device="cpu"):
    import torch
    idx = torch.arange(start + 1, start + n + 1, dtype=torch.int64, device=device)
    return _mix_torch(idx * _signed(GAMMA) + _signed(key))


def weight_torch(seed: int, name: str, shape, std: float = 0.02, dtype: str = "bf16",
                 device="cpu", chunk: int = 1 << 25):
    """Same values as weight_np, generated on a torch device."""
    import torch
    n = int(np.prod(shape))
    out_dtype = torch.bfloat16 if dtype == "bf16" else torch.float32
    out = torch.empty(n, dtype=out_dtype, device=device)
    key = stream_key(seed, name)
    scale = float(np.float32(std / IH4_STD))
    for s in range(0, n, chunk):
        m = min(chunk, n - s)
        r = counter_u64_torch(key, s, m, device)
        tot = (r & 0xFFFF) + ((r >> 16) & 0xFFFF) + ((r >> 32) & 0xFFFF) + ((r >> 48) & 0xFFFF)
        x = (tot - IH4_MEAN).to(torch.float32) * scale
        out[s:s + m] = x.to(out_dtype)
        del r, tot, x
    return out.view(*shape)


def tokens_torch(seed: int, name: str, n: int, n_values: int, device="cpu"):
    import torch
    r = counter_u64_torch(stream_key(seed, name), 0, n, device)
    return ((_lsr(r, 33)) % n_values).to(torch.int32)


# ---------------------------------------------------------------- model weights

WEIGHT_NAMES = ("wqkv", "wo", "wgu", "wdown")


def _weight_shapes(shape: ModelShape):
    d, f, v = shape.d_model, shape.d_ffn, shape.vocab
    per_layer = {"wqkv": (3 * d, d), "wo": (d, d), "wgu": (2 * f, d), "wdown": (d, f)}
    return {"emb": (v, d), "lm_head": (v, d)}, per_layer


def model_weights_np(shape: ModelShape, seed: int = 0, dtype: str = "bf16", layers=None) -> dict:
    """Weights as float32 numpy arrays.  Keys: emb, lm_head, layers.{l}.{name}."""
    top, per_layer = _weight_shapes(shape)
    w = {k: weight_np(seed, k, s, dtype=dtype) for k, s in top.items()}
    for l in (range(shape.n_layers) if layers is None else layers):
        for k, s in per_layer.items():
            w[f"layers.{l}.{k}"] = weight_np(seed, f"layers.{l}.{k}", s, dtype=dtype)
    return w


def model_weights_torch(shape: ModelShape, seed: int = 0, dtype: str = "bf16", device="cpu",
                        layers=None) -> dict:
    top, per_layer = _weight_shapes(shape)
    w = {k: weight_torch(seed, k, s, dtype=dtype, device=device) for k, s in top.items()}
    for l in (range(shape.n_layers) if layers is None else layers):
        for k, s in per_layer.items():
            w[f"layers.{l}.{k}"] = weight_torch(seed, f"layers.{l}.{k}", s, dtype=dtype, device=device)
    return w


def position_scales_np(seed: int, positions, s_lo: float, s_hi: float) -> np.ndarray:
    """Per-position logit scales, log-uniform on [s_lo, s_hi), fixed by absolute position.

    Returned as float32: the same values are handed to the GPU and the oracle.
    """
    positions = np.asarray(positions, dtype=np.int64)
    n = int(positions.max()) + 1 if positions.size else 0
    u = uniform01_np(seed, "position_scale", n)[positions]
    return np.exp(np.log(s_lo) + u * np.log(s_hi / s_lo)).astype(np.float32)
