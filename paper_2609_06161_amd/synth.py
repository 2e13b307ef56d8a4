"""Seeded synthetic inputs for the AF1 factorized linear layer.

This module draws inputs only.  It holds none of the layer's arithmetic: the
sign factors are drawn already packed (uniform words are fair +-1 signs), the
scales and activations are drawn in float32/float64 and rounded once to their
16-bit storage types.  Both the HIP path and the CPU oracle are fed from here;
neither is imported by it.

Recipe (stands in for the LLaMA/Qwen/Gemma layers the paper quantises, whose
trained weights and calibration data are not available):
  1. Bv words, then Bu words: i.i.d. uniform uint32 (fair signs, packed
     row-major, column j of a row = bit j mod 32 of word j div 32; bit 1
     means -1).
  2. s_in, s_mid, s_out: lognormal(mean 0, sigma 0.5), rounded RNE to fp16.
  3. Outlier channels: round(0.01 n) distinct input channels (none when
     outliers are off).
  4. x: float32 N(0, 1) of shape [batch, n]; outlier channels scaled by 20 in
     float32; the whole tensor rounded once, RNE, to bfloat16.
  5. For the scale-only reconstruction (gradients with the signs frozen):
     the upstream gradient dy, float32 N(0, 1) times 2^-10 of shape
     [batch, m] (from its own seed), rounded once, RNE, to bfloat16.
"""
from dataclasses import dataclass

import numpy as np


# Named layer shapes (d_out, d_in, budget rank).  The rank is the largest
# multiple of 32 whose signs plus three fp16 scale vectors fit d_out * d_in
# bits; tests check every entry against the oracle's budget rule.
SHAPES = {
    "sq1024": (1024, 1024, 480),
    "attn4096": (4096, 4096, 2016),
    "kv1024x4096": (1024, 4096, 800),
    "mlp_up14336x4096": (14336, 4096, 3136),
    "mlp_down4096x14336": (4096, 14336, 3136),
    "sq8192": (8192, 8192, 4064),
    "mlp_up28672x8192": (28672, 8192, 6336),
    "mlp_down8192x28672": (8192, 28672, 6336),
}


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round to nearest, ties to even); finite
    inputs only.  Returns uint16 bit patterns."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return r.astype(np.uint16)


def f32_to_f16_bits(a: np.ndarray) -> np.ndarray:
    """Round to IEEE binary16 (numpy's RNE cast).  Returns uint16 patterns."""
    return np.ascontiguousarray(a).astype(np.float16).view(np.uint16)


def random_words(rng: np.random.Generator, rows: int, cols: int) -> np.ndarray:
    """rows x cols fair random signs, already packed (rows x cols/32 uint32)."""
    assert cols % 32 == 0
    w = rng.integers(0, 1 << 32, size=(rows, cols // 32), dtype=np.uint64)
    return w.astype(np.uint32)


def lognormal_f16(rng: np.random.Generator, size: int, sigma: float = 0.5) -> np.ndarray:
    return f32_to_f16_bits(rng.lognormal(mean=0.0, sigma=sigma, size=size).astype(np.float32))


def activations_bf16(rng: np.random.Generator, batch: int, n: int,
                     outlier_idx=None, outlier_scale: float = 20.0) -> np.ndarray:
    x = rng.standard_normal(size=(batch, n), dtype=np.float32)
    if outlier_idx is not None and len(outlier_idx):
        x[:, outlier_idx] *= np.float32(outlier_scale)
    return f32_to_bf16_bits(x)


@dataclass
class Linear:
    """One factorized layer plus an activation batch, as host arrays."""
    m: int
    n: int
    r: int
    Bu: np.ndarray      # [m, r/32] uint32
    Bv: np.ndarray      # [r, n/32] uint32
    s_out: np.ndarray   # [m] uint16 fp16 bits
    s_mid: np.ndarray   # [r] uint16 fp16 bits
    s_in: np.ndarray    # [n] uint16 fp16 bits
    x: np.ndarray       # [batch, n] uint16 bf16 bits
    outliers: np.ndarray

    @property
    def batch(self) -> int:
        return self.x.shape[0]


def make_linear(seed: int, m: int, n: int, r: int, batch: int,
                outliers: bool = True) -> Linear:
    """Draw one layer and its activations in the fixed order of the recipe."""
    rng = np.random.default_rng(seed)
    Bv = random_words(rng, r, n)
    Bu = random_words(rng, m, r)
    s_in = lognormal_f16(rng, n)
    s_mid = lognormal_f16(rng, r)
    s_out = lognormal_f16(rng, m)
    k = int(round(0.01 * n)) if outliers else 0
    idx = np.sort(rng.choice(n, size=k, replace=False)) if k else np.zeros(0, np.int64)
    x = activations_bf16(rng, batch, n, idx)
    return Linear(m, n, r, Bu, Bv, s_out, s_mid, s_in, x, idx)


def make_activations(seed: int, batch: int, n: int, outliers: bool = True) -> np.ndarray:
    rng = np.random.default_rng(seed)
    k = int(round(0.01 * n)) if outliers else 0
    idx = np.sort(rng.choice(n, size=k, replace=False)) if k else None
    return activations_bf16(rng, batch, n, idx)


def make_output_grad(seed: int, batch: int, m: int, scale: float = 2.0 ** -10) -> np.ndarray:
    """Upstream gradient of one linear's output for the scale-only
    reconstruction: float32 N(0, 1) times `scale` (a power of two, so the
    scaling is exact), shape [batch, m], rounded once, RNE, to bfloat16."""
    rng = np.random.default_rng(seed)
    g = rng.standard_normal(size=(batch, m), dtype=np.float32) * np.float32(scale)
    return f32_to_bf16_bits(g)


def random_sign_source(seed: int, rows: int, cols: int, dtype: str) -> np.ndarray:
    """A dense matrix whose signs are to be packed: float32/float16/int8
    values, or bfloat16 patterns ("bf16"), including signed zeros."""
    rng = np.random.default_rng(seed)
    v = rng.standard_normal(size=(rows, cols)).astype(np.float32)
    z = rng.random(size=(rows, cols)) < 0.02       # sprinkle +0 and -0
    v[z] = 0.0
    neg0 = z & (rng.random(size=(rows, cols)) < 0.5)
    v[neg0] = -0.0
    if dtype == "f32":
        return v
    if dtype == "f16":
        return v.astype(np.float16)
    if dtype == "bf16":
        return f32_to_bf16_bits(v)
    if dtype == "i8":
        q = rng.integers(-128, 128, size=(rows, cols), dtype=np.int64)
        return q.astype(np.int8)
    raise ValueError(dtype)


def draw_stack_ranks(seed: int, layers: int, linears, storage_bits):
    """Heterogeneous per-linear ranks for a decoder stack.

    ``linears`` is a list of (name, d_out, d_in, r0).  Each rank is drawn as
    32 * floor(u * r0 / 32) with u ~ U[0.75, 1.25] (at least 32); then, while
    the summed storage exceeds the summed dense weight count, the linear with
    the largest r / r0 (lowest index on ties) gives up 32.  The caller passes
    ``storage_bits(m, n, r)``, so this module carries no storage formula."""
    rng = np.random.default_rng(seed)
    entries = []
    for _ in range(layers):
        for name, m, n, r0 in linears:
            u = rng.uniform(0.75, 1.25)
            r = max(32, 32 * int(np.floor(u * r0 / 32)))
            entries.append([name, m, n, r0, r])
    total_w = sum(e[1] * e[2] for e in entries)

    def total_bits():
        return sum(storage_bits(e[1], e[2], e[4]) for e in entries)

    bits = total_bits()
    while bits > total_w:
        best = max(range(len(entries)), key=lambda i: (entries[i][4] / entries[i][3], -i))
        e = entries[best]
        bits -= storage_bits(e[1], e[2], e[4]) - storage_bits(e[1], e[2], e[4] - 32)
        e[4] -= 32
    return [tuple(e) for e in entries]
