"""Helpers for the GPU parity tests: uploads of generator bits, downloads to
float64, and the tolerance metric.

Tolerance ("max relative error"): err = max_i |g_i - r_i| / max_i |r_i|, the
max-norm relative error of the tensor, <= 2e-2 for bf16 storage and <= 1e-5
for fp32.  A second bar guards against widespread small deviations:
rms(g - r) / rms(r) <= half of the first bar.  The element-wise ratio
max_i |g_i - r_i| / max(|r_i|, rms(r)) is returned for reporting.
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


def errors(g: np.ndarray, r: np.ndarray) -> dict:
    g = np.asarray(g, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    if r.size == 0:
        return dict(max_rel=0.0, rms_rel=0.0, elem_rel=0.0)
    e = np.abs(g - r)
    rmax = np.max(np.abs(r))
    rms = np.sqrt(np.mean(r * r))
    den = np.maximum(np.abs(r), rms)
    return dict(max_rel=float(e.max() / rmax) if rmax > 0 else float(e.max()),
                rms_rel=float(np.sqrt(np.mean(e * e)) / rms) if rms > 0 else float(np.sqrt(np.mean(e * e))),
                elem_rel=float(np.max(e / np.where(den == 0, 1.0, den))))


def rel_err(g, r) -> float:
    return errors(g, r)["max_rel"]


def assert_close(g, r, dtype: str, what: str = "", tol: float = None):
    bar = TOL[dtype] if tol is None else tol
    assert np.all(np.isfinite(g)), f"{what}: non-finite output"
    e = errors(g, r)
    assert e["max_rel"] <= bar, f"{what}: max relative error {e['max_rel']:.3e} > {bar:.1e} ({e})"
    assert e["rms_rel"] <= bar / 2, f"{what}: rms relative error {e['rms_rel']:.3e} > {bar / 2:.1e} ({e})"
    return e
