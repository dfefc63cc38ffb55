"""Error measures for the GPU product against the oracle (float64 y, A).

The gate for the matrix-vector product is tolerance-based: several float32
results are correct (any summation order), and a literal elementwise relative
error cannot serve where y cancels to near zero. Two measures, both <= 2e-3:
  (i)  max over outputs of |y - y_ref| / A, with A = sum_k |w_k * x_k|;
  (ii) per token column, max |y - y_ref| / max |y_ref|.
Also reported: NMSE = sum (y - y_ref)^2 / sum y_ref^2 (the paper's validation
measure, Sec. 3.2), and the largest elementwise relative error.
"""
import numpy as np

TOL = 2e-3


def measures(y, y_ref, A):
    y = np.asarray(y, np.float64).reshape(y_ref.shape)
    y_ref = np.asarray(y_ref, np.float64)
    A = np.asarray(A, np.float64).reshape(y_ref.shape)
    d = np.abs(y - y_ref)
    zeroA = A == 0
    if zeroA.any():
        assert (y[zeroA] == 0).all(), "an output whose terms are all zero must be exactly 0"
    scaled = float((d[~zeroA] / A[~zeroA]).max()) if (~zeroA).any() else 0.0
    if y_ref.ndim == 2:
        den = np.abs(y_ref).max(axis=1)
        den[den == 0] = 1.0
        normwise = float((d.max(axis=1) / den).max())
    else:
        normwise = float(d.max() / max(np.abs(y_ref).max(), 1e-300))
    nmse = float((d ** 2).sum() / max((y_ref ** 2).sum(), 1e-300))
    with np.errstate(divide="ignore", invalid="ignore"):
        elem = np.where(y_ref != 0, d / np.abs(y_ref), 0.0)
    return {"scaled": scaled, "normwise": normwise, "nmse": nmse, "elem_max": float(elem.max()),
            "n_over": int((elem > TOL).sum())}


def check(y, y_ref, A, tol=TOL, f32_bound=None, what=""):
    m = measures(y, y_ref, A)
    assert m["scaled"] <= tol, (what, m)
    assert m["normwise"] <= tol, (what, m)
    if f32_bound is not None:
        assert m["scaled"] <= f32_bound, (what, "exceeds float32-accumulation bound", m)
    return m
