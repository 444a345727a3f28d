"""Helpers for the GPU parity tests: move seeded synthetic inputs to the
device, read results back as float64, compare with the oracle."""
import numpy as np

import synth


def torch_cuda():
    import torch
    if not torch.cuda.is_available():
        import pytest
        pytest.skip("no GPU")
    return torch


def to_dev(raw: np.ndarray):
    """uint16 bf16 bits or float32 host array -> device tensor (bf16 / fp32)."""
    torch = torch_cuda()
    if raw.dtype == np.uint16:
        return torch.from_numpy(raw.view(np.int16).copy()).to("cuda").view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(raw, dtype=np.float32)).to("cuda")


def empty(shape, dtype: str):
    torch = torch_cuda()
    return torch.empty(shape, dtype=torch.bfloat16 if dtype == "bf16" else torch.float32,
                       device="cuda")


def to_host(t) -> np.ndarray:
    """Device tensor -> float64 numpy (exact upcast)."""
    import torch
    t = t.detach()
    if t.dtype == torch.bfloat16:
        raw = t.view(torch.int16).cpu().numpy().view(np.uint16)
        return synth.f32_from_bf16_bits(raw).astype(np.float64)
    return t.float().cpu().numpy().astype(np.float64)


def rel_fro(got: np.ndarray, ref: np.ndarray) -> float:
    den = np.linalg.norm(ref)
    return float(np.linalg.norm(got - ref) / (den if den > 0 else 1.0))


def bf16_round(x: np.ndarray) -> np.ndarray:
    """float64 -> nearest bf16 value (via float32; exact for the integer
    values the exactness tests use)."""
    return synth.f32_from_bf16_bits(synth.bf16_bits_from_f32(x.astype(np.float32))).astype(np.float64)


TOL = {"bf16": 2e-2, "fp32": 1e-5}
