"""CPU checks of the float32 error bound the GPU parity tests apply row by row.

The bound (tests/parity.py fp32_bound) is derived from float32 arithmetic; here
it is checked against float32 evaluations in two different orders (a dense
float32 matrix product, and per-group sums added group by group), and shown to
flag a single wrong code in most rows, where the 2e-3 tolerance rule alone
flags far fewer.
"""

import numpy as np

from oracle import matmul as omatmul
from paper_2607_02893_amd import synth
from tests import parity


def _case(N=600, K=4096, seed=5):
    spec = synth.MatrixSpec("t", 0, 0, N, K)
    bits, q, s = synth.make_matrix(spec, seed)
    x = synth.make_x(spec, seed)[0]
    return bits, q, s, x


def test_float32_evaluations_stay_inside_the_bound():
    bits, q, s, x = _case()
    ystar = omatmul.gemv(q, s, x)
    bound = parity.fp32_bound(q, s, bits, x)
    W32 = omatmul.dequant(q, s).astype(np.float32)
    x32 = x.astype(np.float32)
    y_dense = (W32 @ x32).astype(np.float64)
    assert parity.check_bound(y_dense, ystar, bound) < 0.05
    # per-group float32 sums, then the groups added in order (the kernels' shape)
    Gc = q.shape[1] // 64
    part = np.einsum("ngi,gi->ng", W32.reshape(-1, Gc, 64), x32.reshape(Gc, 64)).astype(np.float32)
    y_grp = np.zeros(q.shape[0], dtype=np.float32)
    for j in range(Gc):
        y_grp = (y_grp + part[:, j]).astype(np.float32)
    assert parity.check_bound(y_grp.astype(np.float64), ystar, bound) < 0.05


def test_bound_flags_a_single_wrong_code():
    bits, q, s, x = _case()
    ystar = omatmul.gemv(q, s, x)
    bound = parity.fp32_bound(q, s, bits, x)
    q2 = q.copy()
    for n in range(q.shape[0]):  # flip one 1-bit weight per row
        j = int(np.nonzero(bits[n] == 1)[0][0])
        q2[n, 64 * j + 5] = -q2[n, 64 * j + 5]
    y_wrong = omatmul.gemv(q2, s, x)
    flagged = np.abs(y_wrong - ystar) > bound
    assert flagged.mean() > 0.75
    # the relative tolerance alone sees far fewer of them
    rel = np.abs(y_wrong - ystar) / np.maximum(np.abs(ystar), omatmul.row_magnitude(q, s, x))
    assert (rel > parity.TOL).mean() < flagged.mean() - 0.3
