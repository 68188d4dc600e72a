"""Helpers for the GPU parity tests: device copies, dtype rounding and the
normwise tolerance used throughout.

Tolerance (normwise relative, per output tensor):
    ||gpu - oracle||_inf / ||oracle||_inf  <=  1e-10 (fp64)  or  1e-4 (fp32)
An all-zero oracle tensor requires an all-zero GPU tensor.  fp32 mode feeds the
oracle the fp32-rounded inputs (converted exactly to float64).
"""
import numpy as np
import torch

TOL = {"f64": 1e-10, "f32": 1e-4}
TORCH_DT = {"f64": torch.float64, "f32": torch.float32}


def rounded(a, dt):
    """The mode's storage values of a float64 draw, returned as float64 for the oracle."""
    if dt == "f32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    return np.ascontiguousarray(a, dtype=np.float64)


def dev(a, dt):
    if a is None:
        return None
    return torch.from_numpy(np.ascontiguousarray(a)).to(device="cuda", dtype=TORCH_DT[dt])


def host(t):
    return t.detach().to("cpu", torch.float64).numpy()


def rel_err(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    den = np.max(np.abs(ref)) if ref.size else 0.0
    num = np.max(np.abs(got - ref)) if ref.size else 0.0
    if den == 0.0:
        return 0.0 if num == 0.0 else np.inf
    return num / den


def assert_close(got, ref, dt, what=""):
    e = rel_err(got, ref)
    assert np.isfinite(np.asarray(got, dtype=np.float64)).all(), f"{what}: non-finite values"
    assert e <= TOL[dt], f"{what}: normwise relative error {e:.3e} > {TOL[dt]:.0e}"
    return e
