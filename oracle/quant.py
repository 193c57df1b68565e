"""Per-group quantizer of VBQ in double precision (test infrastructure only).

Paper section 3.1: a weight matrix is partitioned into contiguous groups of
G = 64 weights, each with a scale s_g and a bit-width b_g.
  * b >= 2, Eq. (1): s = max_i |w_i| / (2^(b-1) - 1),
                     w_hat_i = s * clip(round(w_i / s), -(2^(b-1)-1), 2^(b-1)-1).
  * b = 1 (text following Eq. (1)): w_hat_i = sign(w_i) * mean_j |w_j|.

Readings (the paper is silent on these):
  * round is round-half-to-even (numpy.rint);
  * s is stored as IEEE fp16, rounded once from the double value, and the codes
    are computed against that stored s;
  * if the stored s is 0 (all-zero group, or underflow) every q is 0 for b >= 2;
  * sign(w) is +1 for w >= 0, including -0.0, so that a 1-bit group is a pure
    +/-1 code;
  * the 1-bit mean is the sequential double-precision sum of |w_i| over
    i = 0..63, divided by 64;
  * a scale whose fp16 rounding is infinite (max|w| / qmax, or the 1-bit mean,
    at or beyond 65520) is an error at every width: OverflowError.
"""

import numpy as np

G = 64
WIDTHS = (1, 2, 4, 8)


def qmax(b):
    """Largest level magnitude of width b: 2^(b-1) - 1 for b >= 2, 1 for b = 1."""
    if b not in WIDTHS:
        raise ValueError(f"bit-width {b} not in {{1,2,4,8}}")
    return 1 if b == 1 else (1 << (b - 1)) - 1


def fp16_bits(value):
    """Round a double to IEEE fp16 (round-to-nearest-even) and return its bits."""
    return int(np.array([value], dtype=np.float64).astype(np.float16).view(np.uint16)[0])


def fp16_value(bits):
    """The exact double value of an fp16 bit pattern."""
    return float(np.array([bits], dtype=np.uint16).view(np.float16).astype(np.float64)[0])


def round_half_even(v):
    """round() of Eq. (1): ties go to the even integer."""
    return float(np.rint(v))


def one_bit_sign(v):
    """sign() of the 1-bit rule, as a storable code: +1 for v >= 0 (incl. -0.0)."""
    return 1 if (v > 0.0 or v == 0.0) else -1


def quantize_group(w, b, group=G, exact_scale=False):
    """Quantize one group of `group` weights at width b.

    Returns (q, s_bits): q is a list of Python ints (the levels), s_bits the
    fp16 bit pattern of the stored scale.  Plain loops, in the order of section
    3.1.  `group` and `exact_scale` (keep s in double, no fp16 rounding) exist
    only to check the paper's G = 1 statement; with exact_scale the double
    scale is returned in place of the fp16 bits.
    """
    w = [float(v) for v in w]
    if len(w) != group:
        raise ValueError(f"a group has {group} weights")
    for v in w:
        if not np.isfinite(v):
            raise ValueError("non-finite weight")
    if b == 1:
        total = 0.0
        for v in w:  # sequential double sum
            total += abs(v)
        s_exact = total / group
        s_out = s_exact if exact_scale else fp16_bits(s_exact)
        if not exact_scale and not np.isfinite(fp16_value(s_out)):
            raise OverflowError("scale overflows fp16")  # the stored scale must be a finite fp16 value
        return [one_bit_sign(v) for v in w], s_out
    m = qmax(b)
    amax = 0.0
    for v in w:
        amax = max(amax, abs(v))
    if exact_scale:
        s = amax / m
        s_out = s
    else:
        s_out = fp16_bits(amax / m)
        s = fp16_value(s_out)
    if not np.isfinite(s):
        raise OverflowError("scale overflows fp16")
    if s == 0.0:
        return [0] * group, s_out
    q = []
    for v in w:
        r = round_half_even(v / s)
        q.append(int(min(max(r, -m), m)))
    return q, s_out


def quantize(W, bits):
    """Quantize a matrix W[N][K] (any float dtype) with bit map bits[N][K/64].

    Returns q int8[N][K] and s uint16[N][K/64] (fp16 bit patterns).
    Vectorised over groups of one width at a time; each step is the same as in
    quantize_group.
    """
    W = np.asarray(W, dtype=np.float64)
    bits = np.asarray(bits)
    N, K = W.shape
    if K % G:
        raise ValueError("K must be a multiple of 64")
    if not np.all(np.isfinite(W)):
        raise ValueError("non-finite weight")
    if bits.shape != (N, K // G) or not np.all(np.isin(bits, WIDTHS)):
        raise ValueError("bits must be [N, K/64] with values in {1,2,4,8}")
    Wg = W.reshape(N, K // G, G)
    q = np.zeros((N, K // G, G), dtype=np.int64)
    s16 = np.zeros((N, K // G), dtype=np.float16)
    for b in WIDTHS:
        sel = bits == b
        if not np.any(sel):
            continue
        wg = Wg[sel]  # [n, 64]
        if b == 1:
            total = np.zeros(wg.shape[0], dtype=np.float64)
            for i in range(G):  # sequential double sum, i = 0..63
                total = total + np.abs(wg[:, i])
            s = (total / G).astype(np.float16)
            if not np.all(np.isfinite(s)):
                raise OverflowError("scale overflows fp16")
            s16[sel] = s
            q[sel] = np.where(wg >= 0.0, 1, -1)
        else:
            m = qmax(b)
            s = (np.max(np.abs(wg), axis=1) / m).astype(np.float16)
            if not np.all(np.isfinite(s)):
                raise OverflowError("scale overflows fp16")
            s16[sel] = s
            sd = s.astype(np.float64)[:, None]
            with np.errstate(divide="ignore", invalid="ignore"):
                r = np.rint(wg / sd)
            r = np.clip(r, -m, m)
            r[np.broadcast_to(sd == 0.0, r.shape)] = 0.0
            q[sel] = r.astype(np.int64)
    return q.reshape(N, K).astype(np.int8), s16.view(np.uint16).copy()


def level_set(b):
    """All levels the quantizer can produce at width b."""
    if b == 1:
        return [-1, 1]
    m = qmax(b)
    return list(range(-m, m + 1))


def offset_code(q, b):
    """Offset-binary storage code of level q at width b (u = q + 2^(b-1); 1-bit: (q+1)/2)."""
    return (q + 1) // 2 if b == 1 else q + (1 << (b - 1))


def level_from_code(u, b):
    """Inverse of offset_code."""
    return 2 * u - 1 if b == 1 else u - (1 << (b - 1))
