"""Shared helpers for the GPU parity tests (comparison arithmetic only)."""
import numpy as np
import torch

# Bars: fp32 within 1e-5 and bf16 within 2e-2, both as max-norm relative error.
TOL = {"f32": 1e-5, "bf16": 2e-2}


def to64(t) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def maxnorm_rel(got: np.ndarray, ref: np.ndarray) -> float:
    scale = float(np.abs(ref).max()) if ref.size else 0.0
    if scale == 0.0:
        return float(np.abs(got).max()) if got.size else 0.0
    return float(np.abs(got - ref).max() / scale)


def assert_close(got, ref, dtype: str, what: str = ""):
    """Max-norm relative bar, plus an elementwise bound from the arithmetic.

    bf16: the result is an fp32 value rounded once to bf16 (half an ulp is at
    most 2^-8 relative); fp32 accumulation error adds far less than 2^-10 of
    the max-norm for the sums here.  fp32: accumulation only.
    """
    g = to64(got) if isinstance(got, torch.Tensor) else np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert g.shape == ref.shape, (what, g.shape, ref.shape)
    assert np.isfinite(g).all(), f"{what}: non-finite output"
    err = maxnorm_rel(g, ref)
    assert err <= TOL[dtype], f"{what}: max-norm relative error {err:.3e} > {TOL[dtype]}"
    scale = float(np.abs(ref).max()) if ref.size else 0.0
    if dtype == "bf16":
        bound = 2.0 ** -8 * np.abs(ref) + 2.0 ** -10 * scale
    else:
        bound = 1e-6 * np.abs(ref) + 2e-6 * scale
    bad = np.abs(g - ref) > bound
    assert not bad.any(), (f"{what}: {int(bad.sum())} elements outside the elementwise bound; "
                           f"first at {np.argwhere(bad)[0].tolist()}")
    return err
