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
U32 = 2.0 ** -24  # unit roundoff of float32


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


def fp32_bound(q, s_bits, bits, x, rows_per_block=4096):
    """Per row n, a bound on |y_n - y*_n| derived from float32 arithmetic alone.

    The kernels never round a product: an fp16 activation times a code of at
    most 8 bits times a power of two fits in float32's 24-bit significand.  So
    y_n is a float32 evaluation of a sum of exact terms: per group g of width b
    with scale s, the code terms c*u_i*x_i (u the stored offset code, c = 2 for
    b = 1, else 1) and the offset terms -o*x_i (o = 1 for b = 1, 2^(b-1) else),
    summed within the group, multiplied by s and summed over the groups (or the
    levels q_i = c*u_i - o taken directly).  Whatever the order and grouping,
    each term passes through at most D roundings of relative size u = 2^-24,
    so |y_n - y*_n| <= D * u * A_n, with
        A_n = sum_g s_g * (c * sum_i |u_i x_i| + o * sum_i |x_i|)
    bounding every partial sum.  D counts, for the deepest term: two roundings
    per two-term dot product along a chain of at most 32 (64), the merge of up
    to 5 accumulators (5), the offset and the scale (2), the 64-term group sum
    of x plus its 3 cross-lane adds (67), and the sum over the row's G groups
    (G): D = 138 + G.
    """
    q = np.asarray(q)
    bits = np.asarray(bits)
    x = np.abs(np.asarray(x, dtype=np.float64))
    N, K = q.shape
    Gc = K // 64
    xg = x.reshape(Gc, 64)
    sx = xg.sum(axis=1)                                     # sum_i |x_i| per group column
    s = np.asarray(s_bits, dtype=np.uint16).view(np.float16).astype(np.float64)
    A = np.empty(N, dtype=np.float64)
    for r0 in range(0, N, rows_per_block):
        r1 = min(N, r0 + rows_per_block)
        b = bits[r0:r1].astype(np.float64)
        one = bits[r0:r1] == 1
        o = np.where(one, 1.0, 2.0 ** (b - 1.0))
        c = np.where(one, 2.0, 1.0)
        qb = q[r0:r1].reshape(r1 - r0, Gc, 64).astype(np.float64)
        u = (qb + o[:, :, None]) / c[:, :, None]              # stored offset code
        ux = np.einsum("ngi,gi->ng", np.abs(u), xg)
        A[r0:r1] = np.sum(s[r0:r1] * (c * ux + o * sx[None, :]), axis=1)
    return (138 + Gc) * U32 * A


def check_bound(y, ystar, bound, what=""):
    """Every row within its float32 bound; returns the largest error / bound."""
    y = np.asarray(y, dtype=np.float64)
    err = np.abs(y - np.asarray(ystar, dtype=np.float64))
    bad = err > bound
    if np.any(bad):
        i = int(np.nonzero(bad)[0][0])
        raise AssertionError(f"{what}: row {i} error {err[i]:.3e} above its float32 bound {bound[i]:.3e} "
                             f"({int(bad.sum())} rows)")
    ratio = err / np.where(bound > 0, bound, 1.0)
    return float(ratio.max()) if ratio.size else 0.0
