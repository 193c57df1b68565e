"""Exact probes and every-row checks through each kernel variant, at the 9B-class shapes.

For every way the library can run a product (the kernel it picks depends on the
widths, the grid and the number of activation rows), on full-size matrices:
  * one-hot probes x = e_k: y is column k of w_hat, bit for bit, on every row;
  * group-sum probes x = 1 on group column j, 0 elsewhere: y_n = s_nj * sum_i q_nji
    exactly (every partial result is a small integer times a power of two, and
    the final product has at most 24 significant bits), so one wrong code in the
    column shows;
  * a random x: EVERY row within the 2e-3 rule and within the float32 bound of
    tests/parity.py, which one wrong code exceeds;
  * fp16 output (VBQ_Y_F16): the float32 result rounded to nearest even, bit for bit.
Expected values come from oracle/ only (numpy, in row blocks on the host).
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import matmul as omatmul  # noqa: E402
from paper_2607_02893_amd import synth  # noqa: E402
from tests import parity  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def vbq():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a GPU")
    from paper_2607_02893_amd import vbq as v
    return v


def _say(msg):
    print(msg, flush=True)


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _oracle_rows(q, s, x, block=8192):
    y = np.empty(q.shape[0], dtype=np.float64)
    for r0 in range(0, q.shape[0], block):
        y[r0:r0 + block] = omatmul.gemv(q[r0:r0 + block], s[r0:r0 + block], x)
    return y


def _probe_columns(K):
    return sorted(k for k in {0, 1, 63, 64, K // 2 + 17, K - 65, K - 1} if 0 <= k < K)


def _probe_groups(Gc):
    return sorted({0, Gc // 2, Gc - 1})


def _column(q, s, k):
    return omatmul.scales_f64(s[:, k // 64]) * q[:, k].astype(np.float64)


def _group_sum(q, s, j):
    return omatmul.scales_f64(s[:, j]) * q[:, 64 * j:64 * j + 64].astype(np.int64).sum(axis=1).astype(np.float64)


def _suite(call, q, s, bits, K, what, seed, y16_call=None):
    """call(x fp16 [K]) -> y (numpy, N).  Exact probes, then a random x on every row."""
    for k in _probe_columns(K):
        e = np.zeros(K, dtype=np.float16)
        e[k] = 1.0
        y = call(e).astype(np.float64)
        want = _column(q, s, k)
        assert np.array_equal(y, want), f"{what}: one-hot column {k}, {int(np.sum(y != want))} rows differ"
    for j in _probe_groups(K // 64):
        e = np.zeros(K, dtype=np.float16)
        e[64 * j:64 * j + 64] = 1.0
        y = call(e).astype(np.float64)
        want = _group_sum(q, s, j)
        assert np.array_equal(y, want), f"{what}: group-sum column {j}, {int(np.sum(y != want))} rows differ"
    x = synth.draw_x(synth.rng_for(seed, 31), 1, K)[0]
    y = call(x)
    ystar = _oracle_rows(q, s, x)
    rel = parity.check(y, ystar, _row_mag(q, s, x), what=what)
    ratio = parity.check_bound(y, ystar, parity.fp32_bound(q, s, bits, x), what=what)
    if y16_call is not None:
        y16 = y16_call(x)
        assert y16.dtype == np.float16
        assert np.array_equal(y16.view(np.uint16), y.astype(np.float16).view(np.uint16)), f"{what}: fp16 output"
    _say(f"{what}: exact probes ok; every row: max rel err {rel:.2e}, max err / float32 bound {ratio:.3f}")


def _row_mag(q, s, x, block=8192):
    out = np.empty(q.shape[0], dtype=np.float64)
    for r0 in range(0, q.shape[0], block):
        out[r0:r0 + block] = omatmul.row_magnitude(q[r0:r0 + block], s[r0:r0 + block], x)
    return out


def _gemv_calls(Wp, one_wave=False):
    def call(x):
        return Wp.gemv(_dev(x), one_wave_per_unit=one_wave).cpu().numpy()

    def call16(x):
        return Wp.gemv(_dev(x), y_dtype=torch.float16, one_wave_per_unit=one_wave).cpu().numpy()
    return call, call16


# 9B-class matrices of the mixed-width step and the kernel each one takes
MIXED = [
    ("qkv", 0, "pair kernel, 8 waves (384 tiles x 4 units)"),
    ("o", 0, "pair kernel, 8 waves (256 tiles x 4 units)"),
    ("gate_up", 0, "pair kernel, 8 waves (448 tiles of 64 rows x 4 units)"),
    ("down", 0, "pair kernel, 16 waves (256 tiles x 8 units)"),
    ("down", 1, "one wave per unit (VBQ_ONE_WAVE_PER_UNIT)"),
    ("qkv", 1, "one wave per unit (VBQ_ONE_WAVE_PER_UNIT)"),
    ("head", 0, "one wave per unit (8016 units)"),
]


def _spec(wl, name):
    return next(m for m in wl.matrices if m.name == name)


@pytest.mark.parametrize("name,one_wave,kernel", MIXED)
def test_exact_probes_9b_mixed(vbq, name, one_wave, kernel):
    wl = synth.workload(3)
    spec = _spec(wl, name) if name != "head" else wl.matrices[-1]
    _say(f"9B {name} {spec.N}x{spec.K}: {kernel}")
    bits, q, s = synth.make_matrix(spec, wl.seed)
    blob, d = vbq.pack_codes(q, s, bits)
    Wp = vbq.PackedMatrix(blob, d)
    call, call16 = _gemv_calls(Wp, bool(one_wave))
    _suite(call, q, s, bits, spec.K, f"9B {name} [{kernel}]", 101, call16)


# one-width matrices (the uniform kernel, one template per width) and the bucketed head
UNIFORM = [
    ("recipe gate_up L1 (2-bit)", "recipe", "gate_up", 1),
    ("recipe down L0 (4-bit)", "recipe", "down", 0),
    ("uniform 8-bit o (1.46B-class)", "u8", "o", 0),
    ("uniform 1-bit qkv (1.46B-class)", "u1", "qkv", 0),
    ("uniform 1-bit head (1.46B-class, 64-row tiles: lookup-table decode)", "u1", "head", 32),
]


@pytest.mark.parametrize("what,kind,name,layer", UNIFORM)
def test_exact_probes_uniform_kernels(vbq, what, kind, name, layer):
    wl = synth.workload(3, recipe=True) if kind == "recipe" else synth.workload(4, uniform_bits=int(kind[1:]))
    spec = next(m for m in wl.matrices if m.name == name and m.layer == layer)
    _say(f"{what}: {spec.N}x{spec.K}")
    bits, q, s = synth.make_matrix(spec, wl.seed)
    assert np.unique(bits).size == 1
    blob, d = vbq.pack_codes(q, s, bits)
    Wp = vbq.PackedMatrix(blob, d)
    call, call16 = _gemv_calls(Wp)
    _suite(call, q, s, bits, spec.K, what, 103, call16)


@pytest.mark.parametrize("N,K,R", [(1000, 4096, 64), (700, 2048, 128), (1300, 1024, 256), (64, 64, 64)])
def test_exact_probes_lut_decode_tile_heights(vbq, N, K, R):
    """The 1-bit lookup-table decode (full tiles of one-width 1-bit matrices
    with R >= 64: a table per group column, rebuilt every R/64 slots), with a
    ragged last tile on the two-term dot-product path, every row exact."""
    spec = synth.MatrixSpec("u", 0, 1, N, K, uniform_bits=1)
    bits, q, s = synth.make_matrix(spec, 151)
    blob, d = vbq.pack_codes(q, s, bits, tile_rows=R)
    Wp = vbq.PackedMatrix(blob, d)
    assert vbq.kernel_name(d).startswith("vbq_mv_kernel<1,") and vbq.kernel_name(d).endswith(",0>")
    call, call16 = _gemv_calls(Wp)
    _suite(call, q, s, bits, K, f"1-bit lookup tables N={N} K={K} R={R}", 157, call16)


def test_exact_probes_bucketed_head(vbq):
    """The 9B recipe head (128256 x 4096, rows at 8/4/2/1 bits by frequency tier)
    as four one-width row buckets written through vbq_gemv_rows, every row."""
    wl = synth.workload(3, recipe=True)
    head = wl.matrices[-1]
    bits, q, s = synth.make_matrix(head, wl.seed)
    Wb = vbq.BucketedMatrix(vbq.pack_row_buckets(q, s, bits), head.N, head.K)
    _say(f"recipe head {head.N}x{head.K}: {[(b, p.N) for b, p, _ in Wb.parts]}")

    def call(x):
        return Wb.gemv(_dev(x)).cpu().numpy()

    def call16(x):
        y = torch.empty(head.N, dtype=torch.float16, device="cuda")
        return Wb.gemv(_dev(x), y).cpu().numpy()
    _suite(call, q, s, bits, head.K, "recipe head, 4 row buckets", 107, call16)


# several activation rows: X rows are probes and random rows, every row of Y checked
BATCH = [
    ("o", 2, "pair kernel, two rows (256 tiles x 4 units)", False),
    ("qkv", 2, "pair kernel, two rows (1536 units)", False),
    ("qkv", 2, "one wave per unit, two rows (1536 units)", True),
    ("gate_up", 4, "matrix cores, 64-row tiles", False),
    ("down", 16, "matrix cores, 16-row tiles, 8 units", False),
]


@pytest.mark.parametrize("name,M,kernel,one_wave", BATCH)
def test_exact_probes_9b_batch(vbq, name, M, kernel, one_wave):
    wl = synth.workload(3)
    spec = _spec(wl, name)
    _say(f"9B {name} {spec.N}x{spec.K} M={M}: {kernel}")
    bits, q, s = synth.make_matrix(spec, wl.seed)
    blob, d = vbq.pack_codes(q, s, bits)
    Wp = vbq.PackedMatrix(blob, d)
    K = spec.K
    rng = synth.rng_for(109, M)
    X = synth.draw_x(rng, M, K)
    k0, j0 = K - 1, (K // 64) // 2
    X[0] = 0
    X[0, k0] = 1.0                        # row 0: one-hot
    X[1] = 0
    X[1, 64 * j0:64 * j0 + 64] = 1.0      # row 1: group sum
    if M == 2:
        want = "vbq_mv_kernel<2,4>" if one_wave else "vbq_mv_pair_kernel<8,2>"
        assert vbq.kernel_name(Wp.call_desc(one_wave_per_unit=one_wave), M) == want
    Y = Wp.gemm_small(_dev(X), one_wave_per_unit=one_wave).cpu().numpy()
    assert np.array_equal(Y[0].astype(np.float64), _column(q, s, k0)), "one-hot row"
    assert np.array_equal(Y[1].astype(np.float64), _group_sum(q, s, j0)), "group-sum row"
    worst_rel, worst_b = 0.0, 0.0
    for m in range(2, M):
        ystar = _oracle_rows(q, s, X[m])
        worst_rel = max(worst_rel, parity.check(Y[m], ystar, _row_mag(q, s, X[m]), what=f"{name} M={M} row {m}"))
        worst_b = max(worst_b, parity.check_bound(Y[m], ystar, parity.fp32_bound(q, s, bits, X[m]),
                                                  what=f"{name} M={M} row {m}"))
    Y16 = Wp.gemm_small(_dev(X), y_dtype=torch.float16, one_wave_per_unit=one_wave).cpu().numpy()
    assert np.array_equal(Y16.view(np.uint16), Y.astype(np.float16).view(np.uint16)), "fp16 output"
    _say(f"9B {name} M={M}: exact rows ok; max rel err {worst_rel:.2e}, max err / float32 bound {worst_b:.3f}")


def test_padded_two_row_product_on_the_pair_kernel(vbq):
    """Two activation rows with padded strides (ldx > K, ldy > N) on a geometry
    the two-row pair kernel takes; nothing is written past N in a row."""
    spec = synth.MatrixSpec("t", 0, 0, 1000, 4096)
    bits, q, s = synth.make_matrix(spec, 113)
    blob, d = vbq.pack_codes(q, s, bits)
    Wp = vbq.PackedMatrix(blob, d)
    assert d.n_chunks == 4 and d.n_tiles * d.n_chunks <= 1024  # the two-row pair kernel's range
    X = synth.make_x(spec, 113, M=2)
    X[1] = 0
    X[1, 4095] = 1.0
    Xpad = torch.zeros((2, 4096 + 72), dtype=torch.float16, device="cuda")
    Xpad[:, :4096] = _dev(X)
    Ypad = torch.full((2, 1000 + 24), -3.0, dtype=torch.float32, device="cuda")
    Wp.gemm_small(Xpad[:, :4096], Ypad[:, :1000])
    Y = Ypad.cpu().numpy()
    assert np.all(Y[:, 1000:] == -3.0)
    parity.check(Y[0, :1000], omatmul.gemv(q, s, X[0]), omatmul.row_magnitude(q, s, X[0]), what="padded row 0")
    assert np.array_equal(Y[1, :1000].astype(np.float64), _column(q, s, 4095))
