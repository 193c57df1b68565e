"""Dequantization and the products the fused kernels compute (test infrastructure only).

Paper section 6: the fused kernels expand each group's packed codes with the
group scale and accumulate the matrix-vector product; they are exact up to the
order of floating-point summation, so the reference is the plain definition:

    w_hat[n][k] = s[n][k // 64] * q[n][k]                      (section 3.1)
    y[n]        = sum_k w_hat[n][k] * x[k]                     (GEMV, M = 1)
    Y[m][n]     = sum_k w_hat[n][k] * X[m][k]                  (small GEMM)

All arithmetic is in double: an fp16 scale times a level of at most 8 bits is
exact in double (and in float32), and fp16 activations are exact in double.
The matrix product is numpy's double matmul (a library primitive).
"""

import numpy as np

G = 64


def scales_f64(s_bits):
    """fp16 bit patterns -> exact doubles."""
    return np.asarray(s_bits, dtype=np.uint16).view(np.float16).astype(np.float64)


def dequant(q, s_bits):
    """w_hat = s * q in double, shape [N][K]."""
    q = np.asarray(q, dtype=np.float64)
    N, K = q.shape
    s = scales_f64(s_bits)
    return (q.reshape(N, K // G, G) * s[:, :, None]).reshape(N, K)


def gemv(q, s_bits, x):
    """y = w_hat @ x in double; x is fp16 (or any float) of length K."""
    x = np.asarray(x).astype(np.float64)
    return dequant(q, s_bits) @ x


def gemm(q, s_bits, X):
    """Y = X @ w_hat^T in double; X is [M][K]."""
    X = np.asarray(X).astype(np.float64)
    return X @ dequant(q, s_bits).T


def row_magnitude(q, s_bits, x):
    """||w_hat[n] * x||_2 per row: the scale of the rounding error of row n."""
    x = np.asarray(x).astype(np.float64)
    P = dequant(q, s_bits) * x[None, :]
    return np.sqrt(np.sum(P * P, axis=1))


def gemv_rows(q_rows, s_rows, x):
    """GEMV restricted to a sample of rows (q_rows [n][K], s_rows [n][K/64])."""
    return gemv(q_rows, s_rows, x)
