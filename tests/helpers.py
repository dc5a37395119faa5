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


def rounder(dtype: str):
    """Storage rounding of the GPU path's intermediates: bf16 (RNE) or float32."""
    if dtype == "bf16":
        return lambda a: synth.bf16_round(np.asarray(a, np.float32)).astype(np.float64)
    return lambda a: np.asarray(a, np.float32).astype(np.float64)


# The bound of a tensor is max(TOL, FLOOR_FACTOR * floor), where floor is how far
# the same oracle moves when its stored intermediates are rounded to the GPU's
# storage precision (the unavoidable error of any implementation that stores
# them so). Where the synthetic model makes a result ill-conditioned (tokens
# that differ by a few percent amplify every rounding of the shared part),
# floor exceeds TOL; elsewhere the bound is TOL itself.
FLOOR_FACTOR = 3.0


def _err(got, ref, floor_ref):
    ref = np.asarray(ref, np.float64)
    if floor_ref is not None and np.abs(ref).max() <= 1e-9 * np.abs(floor_ref).max():
        return float(np.abs(np.asarray(got, np.float64)).max() / max(np.abs(floor_ref).max(), 1e-30))
    return rel_err(got, ref)


def compare(name, got, ref, ref_stored, tol, floor_ref=None):
    """check() with the bound raised to FLOOR_FACTOR x the storage-precision floor."""
    floor = _err(ref_stored, ref, floor_ref)
    e = _err(got, ref, floor_ref)
    bound = max(tol, FLOOR_FACTOR * floor)
    assert np.all(np.isfinite(np.asarray(got, np.float64))), f"{name}: non-finite values"
    assert e <= bound, f"{name}: max relative error {e:.3e} > bound {bound:.1e} (tol {tol:.0e}, floor {floor:.2e})"
    return e, floor


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
    assert e <= tol, f"{name}: max relative error {e:.3e} > {tol:.1e}"
    return e


def f32_params(d: dict) -> dict:
    return {k: (None if v is None else np.asarray(v, np.float64)) for k, v in d.items()}
