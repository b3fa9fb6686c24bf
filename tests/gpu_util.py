"""Helpers shared by the GPU tests: device copies, the elementwise bar, NaN-
poisoned output buffers."""
import numpy as np
import torch

DEV = "cuda:0"
TOL = 1e-4


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def f64(a):
    """fp32-rounded copy in fp64: what the GPU actually sees."""
    return np.asarray(a, dtype=np.float32).astype(np.float64)


def host(t):
    return t.detach().cpu().numpy().astype(np.float64)


def assert_close(g, r, what, tol=TOL, scale=None):
    """|g - r| <= tol max(1, |r|) elementwise.  scale (same shape, optional):
    the root sum of squares of the terms each entry sums, which replaces |r|
    where it is larger -- an fp32 sum of many terms carries rounding error in
    proportion to the terms' size, not to a result that cancels to near 0."""
    err = np.abs(g - r)
    ref = np.maximum(1.0, np.abs(r))
    if scale is not None:
        ref = np.maximum(ref, scale)
    bad = err > tol * ref
    assert not np.isnan(g).any(), f"{what}: NaN in GPU output"
    assert not bad.any(), (f"{what}: {bad.sum()} elements out of tolerance, max abs err "
                           f"{err.max():.3e}, max rel {np.max(err / ref):.3e}")


def assert_round_trip(xr, x, what, tol=TOL):
    err = float(np.max(np.abs(xr - x))) if np.size(x) else 0.0
    assert err <= tol, f"{what}: round trip max abs err {err:.3e} > {tol:.0e}"


def poisoned(shape):
    return torch.full(shape, float("nan"), dtype=torch.float32, device=DEV)
