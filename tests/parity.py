"""Tolerance rule shared by the GPU parity tests, smoke() and the bench.

Outputs are fp32 accumulations of exact products, so they differ from the
double-precision oracle only by rounding.  A row passes when
    |y_n - y*_n| <= tol * max(|y*_n|, ||w_hat_n * x||_2)
and the whole vector passes when additionally ||y - y*||_2 <= tol * ||y*||_2,
with tol = 2e-3.  The row magnitude ||w_hat_n * x||_2 is the natural scale of
rounding error in a dot product; relative error alone is meaningless for rows
whose exact value is near zero, and the vector criterion keeps a systematic
error from hiding under the per-row bound.
"""

import numpy as np

TOL = 2e-3


def check(y, ystar, rowmag, tol=TOL, what=""):
    y = np.asarray(y, dtype=np.float64)
    ystar = np.asarray(ystar, dtype=np.float64)
    rowmag = np.asarray(rowmag, dtype=np.float64)
    if y.shape != ystar.shape:
        raise AssertionError(f"{what}: shape {y.shape} != {ystar.shape}")
    if not np.all(np.isfinite(y)):
        raise AssertionError(f"{what}: non-finite output")
    err = np.abs(y - ystar)
    scale = np.maximum(np.abs(ystar), rowmag)
    rel = err / np.where(scale > 0, scale, 1.0)
    worst = int(np.argmax(rel)) if rel.size else 0
    if rel.size and rel.flat[worst] > tol:
        raise AssertionError(f"{what}: element {worst} error {err.flat[worst]:.3e} > {tol} * {scale.flat[worst]:.3e}")
    nrm = np.linalg.norm(ystar)
    if np.linalg.norm(y - ystar) > tol * nrm:
        raise AssertionError(f"{what}: ||y - y*|| = {np.linalg.norm(y - ystar):.3e} > {tol} * {nrm:.3e}")
    return float(rel.max()) if rel.size else 0.0
