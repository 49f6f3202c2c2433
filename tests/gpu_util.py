"""Shared helpers of the GPU parity tests (not collected by pytest itself).

Tolerances (floating point, HIP path vs the float64 oracle on identical inputs):
  bf16 outputs   max-abs <= 2e-2 and relative L2 <= 5e-3   (the workloads' bar)
  f32 outputs    max-abs <= 1e-5 and relative L2 <= 1e-5
  lse (float32)  max-abs <= 2e-4 for bf16 inputs, 1e-5 for f32 inputs: scores
                 of bf16 inputs are exact products summed in float32 (relative
                 error ~ D * 2^-24 on terms of size ~1), and lse does not see
                 the bf16 rounding of P or O.
Integer outputs (layout, compaction) are compared bit for bit.
"""

from __future__ import annotations

import sys

import numpy as np
import torch

DEV = torch.device("cuda:0")

TOL = {"bf16": (2e-2, 5e-3, 2e-4), "f32": (1e-5, 1e-5, 1e-5)}


def announce(msg: str):
    """Name the case on stdout before GPU work, so a crash still shows it."""
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def to64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def rel_l2(got, ref) -> float:
    den = float(np.linalg.norm(ref))
    return float(np.linalg.norm(got - ref)) / (den if den > 0 else 1.0)


def assert_parity(got, ref, dtype: str, what: str, lse_got=None, lse_ref=None):
    max_abs, rl2, lse_tol = TOL[dtype]
    err = float(np.abs(got - ref).max()) if got.size else 0.0
    r = rel_l2(got, ref)
    assert err <= max_abs and r <= rl2, f"{what}: max-abs {err:.3e} (<= {max_abs}), rel-L2 {r:.3e} (<= {rl2})"
    if lse_got is not None:
        e = float(np.abs(lse_got - lse_ref).max()) if lse_got.size else 0.0
        assert e <= lse_tol, f"{what}: lse max-abs {e:.3e} (<= {lse_tol})"
    return err, r


def torch_dtype(name: str):
    return {"bf16": torch.bfloat16, "f32": torch.float32}[name]


def gather_rows(t: torch.Tensor, idx: np.ndarray) -> np.ndarray:
    """Rows idx of a device tensor, as float64 on the host (a plain copy)."""
    if len(idx) == 0:
        return np.zeros((0,) + tuple(t.shape[1:]), np.float64)
    return to64(t[torch.as_tensor(np.asarray(idx, np.int64), device=t.device)])
