"""Helpers for the GPU parity tests: uploads of generator bits, downloads to
float64, and the tolerance metric.

Tolerance: err = max_i |g_i - r_i| / max(|r_i|, rms(r)), i.e. the error of
each element relative to its own magnitude, floored at the tensor's RMS so
that near-zero entries do not blow up the ratio.  The bars are 2e-2 for
bf16 storage and 1e-5 for fp32.
"""

import numpy as np
import torch

TOL = {"bf16": 2e-2, "f32": 1e-5}


def up(bits: np.ndarray, dtype: str, device="cuda") -> torch.Tensor:
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(bits, dtype=np.float32)).to(device)


def up_i32(a, device="cuda") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(np.asarray(a), dtype=np.int32)).to(device)


def down(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu", torch.float64).numpy()


def down_bits(t: torch.Tensor) -> np.ndarray:
    """Storage bits of a device tensor (uint16 for bf16, float32 otherwise)."""
    c = t.detach().cpu().contiguous()
    if c.dtype == torch.bfloat16:
        return c.view(torch.int16).numpy().view(np.uint16)
    return c.numpy()


def rel_err(g: np.ndarray, r: np.ndarray) -> float:
    g = np.asarray(g, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    if r.size == 0:
        return 0.0
    rms = np.sqrt(np.mean(r * r))
    den = np.maximum(np.abs(r), rms)
    den = np.where(den == 0, 1.0, den)
    return float(np.max(np.abs(g - r) / den))


def assert_close(g, r, dtype: str, what: str = "", tol: float = None):
    e = rel_err(g, r)
    bar = TOL[dtype] if tol is None else tol
    assert np.all(np.isfinite(g)), f"{what}: non-finite output"
    assert e <= bar, f"{what}: max relative error {e:.3e} > {bar:.1e}"
    return e
