"""Shared test helpers: host<->device transfer and the parity measure."""
from __future__ import annotations

import numpy as np

import synth

# tolerance of the per-tensor max relative error: max|gpu - ref| / max|ref|
TOL = {"f32": 1e-4, "bf16": 2e-2}


def dev(a: np.ndarray, dtype: str, device="cuda"):
    """float32 host array (bf16-exact values when dtype == 'bf16') -> device tensor."""
    import torch
    a = np.ascontiguousarray(a, dtype=np.float32)
    if dtype == "bf16":
        bits = synth.bf16_bits(a).view(np.int16)
        return torch.from_numpy(bits.copy()).to(device).view(torch.bfloat16)
    return torch.from_numpy(a.copy()).to(device)


def host(t) -> np.ndarray:
    """device tensor -> float64 host array."""
    import torch
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def rel_err(got, ref) -> float:
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    den = np.abs(ref).max()
    num = np.abs(got - ref).max()
    if den == 0.0:
        return float(num)
    return float(num / den)


# Per-tensor errors of the current test, reported at the end of the session
# (tests/conftest.py prints the worst tensor of every test, so the errors are
# visible in a quiet run's tail).
RESULTS: list = []


def record(name: str, err: float, tol: float) -> None:
    import os
    RESULTS.append((os.environ.get("PYTEST_CURRENT_TEST", "?").split(" ")[0], name, float(err), float(tol)))


def check(name, got, ref, tol, floor_ref=None):
    """Per-tensor relative error <= tol. For tensors that vanish in the
    reference, compare max|got| against tol * max|floor_ref| (a sibling tensor)."""
    ref = np.asarray(ref, np.float64)
    # a reference that vanishes analytically (shift-invariance of softmax: key
    # biases and the key-LayerNorm shift) is only zero up to fp64 rounding
    if floor_ref is not None and np.abs(ref).max() <= 1e-9 * np.abs(floor_ref).max():
        e = float(np.abs(np.asarray(got, np.float64)).max() / max(np.abs(floor_ref).max(), 1e-30))
    else:
        e = rel_err(got, ref)
    assert np.all(np.isfinite(np.asarray(got, np.float64))), f"{name}: non-finite values"
    record(name, e, tol)
    assert e <= tol, f"{name}: max relative error {e:.3e} > {tol:.1e}"
    return e


def f32_params(d: dict) -> dict:
    return {k: (None if v is None else np.asarray(v, np.float64)) for k, v in d.items()}
