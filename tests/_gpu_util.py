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


def max_rel_rows(got: np.ndarray, ref: np.ndarray, floor: float = 1e-3) -> float:
    """Largest relative error of any one row (first axis; a packed block
    [b][b] of dW counts as one row).  A row whose reference norm is below
    `floor` times the RMS row norm is measured against that floor instead,
    so an all-zero reference row cannot divide by zero."""
    g = np.asarray(got, np.float64).reshape(got.shape[0], -1)
    r = np.asarray(ref, np.float64).reshape(ref.shape[0], -1)
    if g.shape[0] == 0:
        return 0.0
    num = np.linalg.norm(g - r, axis=1)
    den = np.linalg.norm(r, axis=1)
    fl = floor * float(np.sqrt(np.mean(den ** 2)))
    den = np.maximum(den, fl if fl > 0 else 1.0)
    return float((num / den).max())


TOL = {"bf16": 2e-2, "fp32": 1e-5}
# Per-row (per-block) bound: a wholly wrong token row of a 4096-row output
# moves the Frobenius ratio by only ~1.6 %, so each row is checked too.
# Observed bf16 row errors are ~2e-3-5e-3, fp32 ~2e-6.
ROW_TOL = {"bf16": 1e-2, "fp32": 1e-5}


def check_close(name: str, got: np.ndarray, ref: np.ndarray, dtype: str,
                row_floor: float = 1e-3) -> None:
    """Relative Frobenius error of the whole tensor and of every row (every
    packed block) against the oracle.  row_floor: see max_rel_rows (1.0
    measures each row's error against at least the RMS row norm, for
    outputs whose rows can be far smaller than their rounding error, e.g.
    attention gradients of keys that receive little attention)."""
    e, m = rel_fro(got, ref), max_rel_rows(got, ref, row_floor)
    print(f"  {name}: rel_fro={e:.3e} max_row={m:.3e}", flush=True)
    assert e <= TOL[dtype], (name, "rel_fro", e)
    assert m <= ROW_TOL[dtype], (name, "max_row", m)
