"""Seeded synthetic inputs for the block-hybrid attention workloads.

This module only draws random numbers and rounds them to the input dtype; it
holds none of the layer's arithmetic.  The tests feed the same arrays to the
HIP library and to the CPU oracle, and the benchmark draws its inputs here.

Shapes follow the paper's serving setting (one 32-token active block per
request, a committed prefix of P tokens, Section 3.1 and the kernel benchmark
of Appendix A) with 16 query / 4 KV heads, head_dim 128 and feature
dimension f = 2F = 128.  The paper's prompt pools and trained weights are not
available; Gaussian activations and N(0, 0.02) feature-map weights stand in.
"""
from __future__ import annotations

from dataclasses import dataclass, replace

import numpy as np


@dataclass(frozen=True)
class Dims:
    B: int          # requests
    Hq: int         # query heads
    Hkv: int        # KV heads (divides Hq)
    d: int          # head_dim
    L: int          # active-block tokens
    F: int          # columns of W_h; the state has f = 2F rows
    dtype: str      # "f32" or "bf16": q, k, v, W, out, KV cache

    @property
    def f(self) -> int:
        return 2 * self.F

    def with_(self, **kw) -> "Dims":
        return replace(self, **kw)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), kept as float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32)


def to_dtype(x: np.ndarray, dtype: str) -> np.ndarray:
    x = np.asarray(x, dtype=np.float32)
    return round_bf16(x) if dtype == "bf16" else x


def gaussian(seed: int, shape, std: float = 1.0) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(shape) * std).astype(np.float32)


def device_gaussian(shape, seed: int, std: float = 1.0, dtype: str = "bf16",
                    device: str = "cuda", chunk_rows: int = 1 << 14):
    """Seeded N(0, std^2) tensor drawn on the device with torch's generator, in
    the activation dtype (bf16 values are rounded once, on creation).  Used for
    inputs too large to draw on the host; a test hands the same tensor to the
    library and copies the rows it checks to the host for the oracle.  Drawn
    in slices along the first axis so that no full-size fp32 copy exists."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    out = torch.empty(shape, dtype=tdt, device=device)
    flat = out.view(shape[0], -1)
    step = max(1, chunk_rows // max(1, flat.shape[1] // 4096 + 1))
    for r0 in range(0, shape[0], step):
        r1 = min(shape[0], r0 + step)
        x = torch.randn((r1 - r0, flat.shape[1]), generator=gen, device=device) * std
        flat[r0:r1] = x.to(tdt)
    return out


def block_qkv(dims: Dims, seed: int, scale: float = 1.0):
    """Active-block q [B][L][Hq][d], k, v [B][L][Hkv][d] ~ N(0, scale^2)."""
    rng = np.random.default_rng(seed)
    B, L, Hq, Hkv, d = dims.B, dims.L, dims.Hq, dims.Hkv, dims.d
    q = rng.standard_normal((B, L, Hq, d)) * scale
    k = rng.standard_normal((B, L, Hkv, d)) * scale
    v = rng.standard_normal((B, L, Hkv, d)) * scale
    return tuple(to_dtype(a, dims.dtype) for a in (q, k, v))


def feature_weights(dims: Dims, seed_w: int, seed_a: int, w_std: float = 0.02):
    """Wt [Hq][F][d] (row j is column j of W_h) ~ N(0, w_std^2); alpha [Hq] ~ N(0, 1)."""
    Wt = to_dtype(gaussian(seed_w, (dims.Hq, dims.F, dims.d), w_std), dims.dtype)
    alpha = gaussian(seed_a, (dims.Hq,), 1.0)
    return Wt, alpha


def sequence_qkv(dims: Dims, T: int, seed: int, scale: float = 1.0):
    """Training-sequence q [B][T][Hq][d], k, v [B][T][Hkv][d] ~ N(0, scale^2)."""
    return block_qkv(dims.with_(L=T), seed, scale)


def upstream(dims: Dims, T: int, seed: int, std: float = 1.0) -> np.ndarray:
    """An upstream gradient or a teacher output [B][T][Hq][d] ~ N(0, std^2)."""
    return to_dtype(gaussian(seed, (dims.B, T, dims.Hq, dims.d), std), dims.dtype)


def prefix_kv(B: int, P: int, Hkv: int, d: int, seed: int, scale: float, dtype: str):
    """Committed-prefix keys and values [B][P][Hkv][d] ~ N(0, scale^2)."""
    rng = np.random.default_rng(seed)
    kp = rng.standard_normal((B, P, Hkv, d)) * scale
    vp = rng.standard_normal((B, P, Hkv, d)) * scale
    return to_dtype(kp, dtype), to_dtype(vp, dtype)


def serve_prefix_lengths(B: int, seed: int = 3, L: int = 32, lo: int = 1024,
                         hi: int = 32768) -> np.ndarray:
    """Per-request committed prefix lengths, whole blocks, uniform in [lo, hi]."""
    rng = np.random.default_rng(seed)
    return (L * rng.integers(lo // L, hi // L + 1, size=B)).astype(np.int32)


# Named workloads: the shapes the parity tests and the benchmark use.
TINY = Dims(B=1, Hq=1, Hkv=1, d=64, L=8, F=32, dtype="f32")
DECODE1 = Dims(B=1, Hq=16, Hkv=4, d=128, L=32, F=64, dtype="bf16")
SERVE64 = Dims(B=64, Hq=16, Hkv=4, d=128, L=32, F=64, dtype="bf16")
PREFILL8 = Dims(B=8, Hq=16, Hkv=4, d=128, L=32, F=64, dtype="bf16")
MIX128 = Dims(B=128, Hq=16, Hkv=4, d=128, L=32, F=64, dtype="bf16")
# Stage-1 attention transfer: 8 sequences of 2048 tokens (training examples
# are truncated to 2048 tokens), one linearised layer.
TRAIN8 = Dims(B=8, Hq=16, Hkv=4, d=128, L=32, F=64, dtype="bf16")
TRAIN8_T = 2048

TINY_PREFIX = 32            # 4 committed blocks of 8 tokens
DECODE1_PREFIX = 4096
PREFILL8_T = 8192
MIX128_PREFIX = 32768
SERVE64_STEPS_PER_BLOCK = 8
