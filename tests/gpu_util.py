"""Helpers for the GPU parity tests: uploads of generator bits, downloads to
float64, and the tolerance gates.

The stated bar is a maximum relative error of 2e-2 for bf16 storage and
1e-5 for fp32, read tensor-wise (tests/test_bf16_reading.py pins why: with
bf16 storage even exact arithmetic exceeds a per-element 2e-2):
  max_rel  = max_i |g_i - r_i| / max_i |r_i|            <= bar
  rms_rel  = rms(g - r) / rms(r)                        <= bar / 2
  elem_rel = max_i |g_i - r_i| / max(|r_i|, rms(r))    <= max(bar, 8 rms_rel)
The last gate holds every element to the bar relative to its own magnitude
(floored at the tensor's RMS), except that an element may reach 8x the
tensor's RMS error: rounding noise spreads that far over millions of
elements, while a wrong element (an index, a dropped term) stands out far
beyond it.  Every comparison prints one line with these numbers and the
largest absolute error (which the anchor checks use to size their tie band).
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
        return dict(max_rel=0.0, rms_rel=0.0, elem_rel=0.0, max_abs=0.0)
    e = np.abs(g - r)
    rmax = np.max(np.abs(r))
    rms = np.sqrt(np.mean(r * r))
    den = np.maximum(np.abs(r), rms)
    return dict(max_rel=float(e.max() / rmax) if rmax > 0 else float(e.max()),
                rms_rel=float(np.sqrt(np.mean(e * e)) / rms) if rms > 0 else float(np.sqrt(np.mean(e * e))),
                elem_rel=float(np.max(e / np.where(den == 0, 1.0, den))), max_abs=float(e.max()))


def rel_err(g, r) -> float:
    return errors(g, r)["max_rel"]


def assert_close(g, r, dtype: str, what: str = "", tol: float = None):
    bar = TOL[dtype] if tol is None else tol
    assert np.all(np.isfinite(g)), f"{what}: non-finite output"
    e = errors(g, r)
    elem_bar = max(bar, 8.0 * e["rms_rel"])
    print(f"[parity] {what}: max_rel {e['max_rel']:.3e} (bar {bar:.0e})  rms_rel {e['rms_rel']:.3e}  "
          f"elem_rel {e['elem_rel']:.3e} (bar {elem_bar:.2e})  max_abs {e['max_abs']:.3e}", flush=True)
    assert e["max_rel"] <= bar, f"{what}: max relative error {e['max_rel']:.3e} > {bar:.1e} ({e})"
    assert e["rms_rel"] <= bar / 2, f"{what}: rms relative error {e['rms_rel']:.3e} > {bar / 2:.1e} ({e})"
    assert e["elem_rel"] <= elem_bar, (
        f"{what}: element-wise relative error {e['elem_rel']:.3e} > max(bar, 8 x rms) = {elem_bar:.2e} ({e})")
    return e
