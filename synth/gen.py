"""Workload table and seeded generators (see package docstring)."""
from __future__ import annotations

import dataclasses
import numpy as np

# Per-tensor stream ids: fixed so that a tensor's values do not depend on the
# order in which a caller draws them.
STREAMS = {"X": 1, "W": 2, "U": 3, "V": 4, "dY": 5, "W2": 6, "U2": 7, "V2": 8,
           "Q": 11, "K": 12, "Vt": 13, "dO": 14}


def bf16_bits_from_f32(a: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.reshape(-1).view(np.uint32)
    # u + 0x7FFF + (bit 16 of u), in 32-bit arithmetic: a sum past 2^32
    # (negative NaNs only) wraps to below 0x8000, and so gives the same top
    # half (0) as the exact sum truncated to 16 bits.
    r = (u >> 16) & 1
    r += 0x7FFF
    r += u
    r >>= 16
    return r.astype(np.uint16).reshape(a.shape)


def f32_from_bf16_bits(h: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> float32 (exact)."""
    h = np.ascontiguousarray(h, dtype=np.uint16)
    return (h.astype(np.uint32) << 16).view(np.float32)


def draw(shape, std: float, seed: int, stream: int, dtype: str, values: bool = True):
    """One N(0, std^2) tensor.

    Returns ``(values_f64, raw)`` where ``raw`` is what the GPU consumes:
    uint16 bf16 bits for ``dtype == "bf16"``, float32 for ``"fp32"``; and
    ``values_f64`` is exactly that tensor upcast to float64 (None when
    ``values`` is False).
    """
    rng = np.random.default_rng([seed, stream])
    a = rng.standard_normal(size=shape, dtype=np.float32)
    a *= np.float32(std)
    if dtype == "bf16":
        raw = bf16_bits_from_f32(a)
        return (f32_from_bf16_bits(raw).astype(np.float64) if values else None), raw
    if dtype == "fp32":
        return (a.astype(np.float64) if values else None), a
    raise ValueError(dtype)


def draw_int(shape, lo: int, hi: int, seed: int, stream: int, dtype: str):
    """Integer-valued tensor in [lo, hi] (exact in bf16 and fp32)."""
    rng = np.random.default_rng([seed, stream, 7])
    a = rng.integers(lo, hi + 1, size=shape).astype(np.float32)
    if dtype == "bf16":
        raw = bf16_bits_from_f32(a)
        return a.astype(np.float64), raw
    return a.astype(np.float64), a


@dataclasses.dataclass(frozen=True)
class Workload:
    """A named synthetic workload: a sparse+low-rank linear layer (or a pair
    of them with GELU between), or block-sparse attention."""
    name: str
    kind: str                 # "linear" | "mlp_pair" | "attention"
    dtype: str                # "bf16" | "fp32"
    T: int = 0                # tokens
    K: int = 0                # in-features
    N: int = 0                # out-features (hidden width for mlp_pair)
    b: int = 32               # block size
    max_stride: int = 1       # in blocks
    r: int = 0                # low-rank
    std_x: float = 0.02
    std_w: float = 0.02
    std_uv: float = 0.02
    std_dy: float = 0.02
    B: int = 0                # attention batch
    H: int = 0                # attention heads
    S: int = 0                # attention sequence length
    d: int = 0                # attention head dim
    global_blocks: int = 0    # attention: width of the global stripes, in blocks
    seed: int = 0


WORKLOADS = {
    # 256 tokens through a 1024x1024 layer, 32x32 blocks, strides < 32 blocks
    # (6 kept blocks per block row), rank 32, fp32 I/O.
    "linear_fp32_1024": Workload(
        "linear_fp32_1024", "linear", "fp32", T=256, K=1024, N=1024, b=32,
        max_stride=32, r=32, std_x=1.0, std_w=1.0 / np.sqrt(6 * 32),
        std_uv=1.0 / np.sqrt(1024), std_dy=1.0),
    # MLP fc1 of a 768-wide transformer: 4096 tokens, 768 -> 3072, 32x32
    # blocks, strides < 16 blocks on the 24x24 square, tiled 4x on the output.
    "mlp_fc1_768x3072": Workload(
        "mlp_fc1_768x3072", "linear", "bf16", T=4096, K=768, N=3072, b=32,
        max_stride=16, r=96),
    # MLP pair 1024 -> 4096 -> GELU -> 1024, 8192 tokens, 64x64 blocks.
    "mlp_pair_1024x4096": Workload(
        "mlp_pair_1024x4096", "mlp_pair", "bf16", T=8192, K=1024, N=4096,
        b=64, max_stride=16, r=128),
    # Block-sparse attention: batch 8, 12 heads, 4096 tokens, head dim 64,
    # 64x64 score blocks, strides < 64 blocks (7 kept blocks per block row).
    "attn_8x12x4096x64": Workload(
        "attn_8x12x4096x64", "attention", "bf16", B=8, H=12, S=4096, d=64,
        b=64, max_stride=64, std_x=1.0, std_dy=1.0),
    # The same attention with the global component: the first 64 queries
    # attend to every key and every query attends to the first 64 keys.
    "attn_global_8x12x4096x64": Workload(
        "attn_global_8x12x4096x64", "attention", "bf16", B=8, H=12, S=4096, d=64,
        b=64, max_stride=64, std_x=1.0, std_dy=1.0, global_blocks=1),
    # Pattern microbenchmark (appendix on microbenchmarking): forward product
    # of a 4096 x 4096 weight over 4096 tokens for random p x p block patterns
    # of 10% expected density and the flat block butterfly + low-rank layer
    # selected for a 10% budget, on the 32 x 32 block cover of each pattern.
    "patterns_4096x4096": Workload(
        "patterns_4096x4096", "patterns", "bf16", T=4096, K=4096, N=4096, b=32),
    # Flat butterfly vs its product form (appendix on benchmarking the
    # butterfly multiply): 1024 x 1024, 32 x 32 blocks, batch 2048, maximum
    # stride swept 2 .. 32; the timed step is the flat layer at stride 32.
    "butterfly_1024_b32": Workload(
        "butterfly_1024_b32", "butterfly", "bf16", T=2048, K=1024, N=1024, b=32,
        max_stride=32, std_x=1.0, std_dy=1.0),
    # Large layer 4096 -> 16384, 16384 tokens, 128x128 blocks, strides < 32.
    "linear_16384x4096_b128": Workload(
        "linear_16384x4096_b128", "linear", "bf16", T=16384, K=4096, N=16384,
        b=128, max_stride=32, r=256),
    "linear_16384x4096_b64": Workload(
        "linear_16384x4096_b64", "linear", "bf16", T=16384, K=4096, N=16384,
        b=64, max_stride=32, r=256),
    "linear_16384x4096_b32": Workload(
        "linear_16384x4096_b32", "linear", "bf16", T=16384, K=4096, N=16384,
        b=32, max_stride=32, r=256),
}


def random_block_mask(n_out: int, n_in: int, p: int, density: float, seed: int) -> np.ndarray:
    """Random sparsity pattern of the paper's pattern microbenchmark: the
    n_out x n_in matrix is split into p x p blocks and each block is kept
    independently with probability `density` (the expected density).
    Element mask, bool.  numpy PCG64 seeded with [seed, 101]."""
    assert n_out % p == 0 and n_in % p == 0
    rng = np.random.Generator(np.random.PCG64([seed, 101]))
    keep = rng.random((n_out // p, n_in // p)) < density
    return np.kron(keep.astype(np.int8), np.ones((p, p), np.int8)).astype(bool)
