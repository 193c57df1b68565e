"""Differentiable bit selection in double precision (test infrastructure only).

Paper section 3.2 ("Differentiable bit selection") and Algorithm 1:
  * every group g of 64 weights carries logits l_g over the candidate widths
    B = (1, 2, 4, 8);
  * the selection path draws pi_g = softmax((l_g + e_g) / tau), with Gumbel
    noise e_g and temperature tau;
  * the soft-quantized weight is the convex combination
        w_soft_i = sum_k pi_{g,k} * w_hat^(B_k)_i ,
    where w_hat^(b) is the per-group quantizer of section 3.1 (Eq. (1) for
    b >= 2, sign/absmean for b = 1) applied at width b to every group;
  * the expected bit cost is bbar = (1/n) sum_g sum_k pi_{g,k} B_k;
  * Algorithm 1 returns the hardened widths b_g = B[argmax_k l_{g,k}].

Logit step of Algorithm 1 (section 3.3, "Gradient isolation"): the candidate
reconstructions are held constant (stop-gradient), so the only path from the
loss L = L_CE + lambda * bbar to l_g runs through pi_g.  With G_i = dL_CE /
dw_soft_i (supplied by the caller: it is the back-propagated gradient of the
network's loss), the chain rule gives
    a_{g,k}       = sum_{i in g} G_i * w_hat^(B_k)_i + lambda * B_k / n
    dL/dl_{g,k}   = (pi_{g,k} / tau) * (a_{g,k} - sum_j pi_{g,j} a_{g,j}).

Readings (the paper is silent on these):
  * the candidates use exactly the quantizer of ``quant`` (fp16-rounded scale,
    codes against the stored scale, round-half-to-even, sign(0) = +1,
    sequential double absmean), so that a one-hot pi reproduces the packed,
    deployed weights;
  * n in bbar is the number of groups, so bbar is the mean bits per weight;
  * the noise e is an input (drawn by the caller);
  * argmax takes the first of equal maxima;
  * the softmax subtracts the group's largest (l + e)/tau before exp, which is
    the same function and keeps exp in range.

Parity status: pinned by CPU tests against a hand-computed group (Eq. (1) at
all four widths, mixed with pi = (0.1, 0.2, 0.3, 0.4)), closed forms of the
softmax (uniform logits, a single raised logit), the convex-combination and
shift invariances, the tau -> 0 limit, and central finite differences of the
scalar objective for the logit gradient.
"""

import numpy as np

from . import quant

CANDIDATES = (1, 2, 4, 8)


def candidates(W):
    """w_hat^(B_k) for k = 0..3: double array [4, N, K] (section 3.1 at each width)."""
    W = np.asarray(W, dtype=np.float64)
    N, K = W.shape
    out = np.empty((len(CANDIDATES), N, K), dtype=np.float64)
    for k, b in enumerate(CANDIDATES):
        bits = np.full((N, K // quant.G), b, dtype=np.uint8)
        q, s16 = quant.quantize(W, bits)
        s = s16.view(np.float16).astype(np.float64)  # [N, K/64]
        levels = q.astype(np.float64).reshape(N, K // quant.G, quant.G)
        out[k] = (levels * s[:, :, None]).reshape(N, K)
    return out


def gumbel_softmax(logits, noise, tau):
    """pi = softmax((l + e) / tau) over the last axis, in double."""
    z = (np.asarray(logits, dtype=np.float64) + np.asarray(noise, dtype=np.float64)) / float(tau)
    z = z - np.max(z, axis=-1, keepdims=True)
    p = np.exp(z)
    return p / np.sum(p, axis=-1, keepdims=True)


def harden(logits):
    """Algorithm 1's result: B[argmax_k l_{g,k}] per group (first maximum), uint8."""
    idx = np.argmax(np.asarray(logits, dtype=np.float64), axis=-1)
    return np.asarray(CANDIDATES, dtype=np.uint8)[idx]


def forward(W, logits, noise, tau):
    """One forward pass of the selection path over a matrix W[N, K].

    logits and noise are [N, K/64, 4] (candidate order 1, 2, 4, 8); noise may be
    None (no noise).  Returns a dict with
      w_soft [N, K], pi [N, K/64, 4], bbar (float), hard_bits uint8 [N, K/64].
    """
    W = np.asarray(W, dtype=np.float64)
    N, K = W.shape
    Gc = K // quant.G
    logits = np.asarray(logits, dtype=np.float64)
    if logits.shape != (N, Gc, len(CANDIDATES)):
        raise ValueError("logits must be [N, K/64, 4]")
    noise = np.zeros_like(logits) if noise is None else np.asarray(noise, dtype=np.float64)
    if noise.shape != logits.shape:
        raise ValueError("noise must match logits")
    if not (tau > 0.0 and np.isfinite(tau)):
        raise ValueError("tau must be positive and finite")
    cand = candidates(W).reshape(len(CANDIDATES), N, Gc, quant.G)
    pi = gumbel_softmax(logits, noise, tau)
    w_soft = np.zeros((N, Gc, quant.G), dtype=np.float64)
    for k in range(len(CANDIDATES)):
        w_soft += pi[:, :, k, None] * cand[k]
    widths = np.asarray(CANDIDATES, dtype=np.float64)
    bbar = float(np.sum(pi * widths) / (N * Gc))
    return {"w_soft": w_soft.reshape(N, K), "pi": pi, "bbar": bbar, "hard_bits": harden(logits)}


def logit_grad(W, grad_w_soft, pi, tau, lam, n_groups=None):
    """dL/dl for the logit step (section 3.3): [N, K/64, 4] in double.

    grad_w_soft is G = dL_CE/dw_soft [N, K]; pi the forward's pi; lam the bit
    penalty lambda; n_groups the n of bbar (defaults to this matrix's groups,
    N*K/64; a network-wide bbar passes the network's total).
    """
    W = np.asarray(W, dtype=np.float64)
    N, K = W.shape
    Gc = K // quant.G
    pi = np.asarray(pi, dtype=np.float64)
    n = N * Gc if n_groups is None else int(n_groups)
    cand = candidates(W).reshape(len(CANDIDATES), N, Gc, quant.G)
    Gr = np.asarray(grad_w_soft, dtype=np.float64).reshape(N, Gc, quant.G)
    a = np.empty((N, Gc, len(CANDIDATES)), dtype=np.float64)
    for k, b in enumerate(CANDIDATES):
        a[:, :, k] = np.sum(Gr * cand[k], axis=-1) + lam * b / n
    mean_a = np.sum(pi * a, axis=-1, keepdims=True)
    return pi / float(tau) * (a - mean_a)
