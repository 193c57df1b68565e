"""GPU parity: the HIP path (through the C ABI) against the double-precision oracle.

Bars:
  * dequantized weights: bit-exact (s*q is exact in float32);
  * one-hot probe x = e_k through vbq_gemv: column k of w_hat, bit-exact;
  * outputs: tests/parity.py rule, tol 2e-3 (fp32 accumulation);
  * repeated calls: bitwise identical (fixed summation order).
Inputs come from paper_2607_02893_amd.synth (seeded); expected values come
from oracle/ only.
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import layout as olayout  # noqa: E402
from oracle import matmul as omatmul  # noqa: E402
from oracle import quant as oquant  # noqa: E402
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


def _packed(vbq, q, s, bits, R=0, C=0):
    blob, d = vbq.pack_codes(q, s, bits, tile_rows=R, chunk_groups=C)
    return vbq.PackedMatrix(blob, d)


def _x_dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).cuda()


GEOMS = [(512, 512, 0, 0), (1, 64, 16, 1), (37, 320, 16, 2), (100, 768, 64, 12), (130, 1024, 32, 5),
         (300, 640, 256, 3), (17, 896, 16, 7), (1000, 4096, 64, 64), (96, 14336, 16, 112)]


@pytest.mark.parametrize("N,K,R,C", GEOMS)
def test_dequant_bit_exact(vbq, N, K, R, C):
    _say(f"dequant N={N} K={K} R={R} C={C}")
    bits, q, s = synth.make_matrix(synth.MatrixSpec("t", N, K, N, K), 41)
    Wp = _packed(vbq, q, s, bits, R, C)
    W = Wp.dequant().cpu().numpy()
    want = omatmul.dequant(q, s)
    assert np.array_equal(W.astype(np.float64), want)


@pytest.mark.parametrize("N,K,R,C", GEOMS)
def test_gemv_matches_oracle(vbq, N, K, R, C):
    _say(f"gemv N={N} K={K} R={R} C={C}")
    spec = synth.MatrixSpec("t", N, K, N, K)
    bits, q, s = synth.make_matrix(spec, 43)
    x = synth.make_x(spec, 43)[0]
    Wp = _packed(vbq, q, s, bits, R, C)
    y = Wp.gemv(_x_dev(x)).cpu().numpy()
    rel = parity.check(y, omatmul.gemv(q, s, x), omatmul.row_magnitude(q, s, x), what=f"gemv {N}x{K}")
    _say(f"  max rel err {rel:.2e}")


# geometries the two-waves-per-unit kernel takes (mixed widths, 2..8 units
# of at most 32 columns per tile, a small grid), with ragged tiles and units;
# units per tile 2 (pairs of adjacent waves), 3-4 (eight waves) and 5-8
# (sixteen waves), so both ways of pairing waves, with and without idle pairs
PAIR_GEOMS = [(6144, 4096, 0, 0), (4096, 14336, 0, 0), (1000, 4096, 0, 0), (37, 320, 0, 0), (17, 896, 0, 0),
              (300, 640, 256, 3), (130, 1024, 32, 5), (77, 2048, 64, 11), (200, 2048, 16, 16),
              (150, 640, 16, 2), (90, 768, 32, 2), (50, 448, 16, 1)]


@pytest.mark.parametrize("N,K,R,C", PAIR_GEOMS)
def test_pair_kernel_matches_one_wave_per_unit(vbq, N, K, R, C):
    """Both kernels match the oracle; where one wave per unit also takes whole
    units (four or more units per tile) the two add the same per-unit row
    sums in the same order, so their outputs are bitwise equal."""
    _say(f"pair vs single N={N} K={K} R={R} C={C}")
    spec = synth.MatrixSpec("t", N, K, N, K)
    bits, q, s = synth.make_matrix(spec, 47)
    x = synth.make_x(spec, 47)[0]
    Wp = _packed(vbq, q, s, bits, R, C)
    xd = _x_dev(x)
    y_pair = Wp.gemv(xd).cpu().numpy()
    y_one = Wp.gemv(xd, one_wave_per_unit=True).cpu().numpy()
    if Wp.desc.n_chunks >= 4:
        assert np.array_equal(y_pair, y_one)
    want, mag = omatmul.gemv(q, s, x), omatmul.row_magnitude(q, s, x)
    parity.check(y_pair, want, mag, what=f"pair gemv {N}x{K}")
    parity.check(y_one, want, mag, what=f"one-wave gemv {N}x{K}")
    # two activation rows (the pair kernel takes up to four units per tile)
    X = synth.make_x(spec, 47, M=2)
    Xd = torch.from_numpy(np.ascontiguousarray(X)).to("cuda")
    Y_pair = Wp.gemm_small(Xd).cpu().numpy()
    Y_one = Wp.gemm_small(Xd, one_wave_per_unit=True).cpu().numpy()
    if Wp.desc.n_chunks >= 4:
        assert np.array_equal(Y_pair, Y_one)
    for m in range(2):
        parity.check(Y_pair[m], omatmul.gemv(q, s, X[m]), omatmul.row_magnitude(q, s, X[m]),
                     what=f"pair gemm_small {N}x{K} m={m}")


def test_one_hot_probe_is_exact(vbq):
    spec = synth.MatrixSpec("t", 0, 0, 300, 1024)
    bits, q, s = synth.make_matrix(spec, 47)
    Wp = _packed(vbq, q, s, bits, 32, 5)
    W = omatmul.dequant(q, s)
    for k in (0, 1, 62, 63, 64, 333, 1023):
        e = np.zeros(1024, dtype=np.float16)
        e[k] = 1.0
        y = Wp.gemv(_x_dev(e)).cpu().numpy()
        assert np.array_equal(y.astype(np.float64), W[:, k]), k
        e[k] = -2.0
        y = Wp.gemv(_x_dev(e)).cpu().numpy()
        assert np.array_equal(y.astype(np.float64), -2.0 * W[:, k]), k


def test_gemv_bitwise_repeatable(vbq):
    spec = synth.MatrixSpec("t", 0, 0, 2048, 4096)
    bits, q, s = synth.make_matrix(spec, 53)
    Wp = _packed(vbq, q, s, bits)
    x = _x_dev(synth.make_x(spec, 53)[0])
    y0 = Wp.gemv(x).cpu().numpy()
    for _ in range(3):
        assert np.array_equal(Wp.gemv(x).cpu().numpy(), y0)


@pytest.mark.parametrize("bits_u", [1, 2, 4, 8])
def test_uniform_width_vs_dense_float32(vbq, bits_u):
    """Uniform-width matrices against a plain PyTorch float32 dense product of
    the dequantized weights, and the oracle."""
    spec = synth.MatrixSpec("u", 0, bits_u, 768, 2048, uniform_bits=bits_u)
    bits, q, s = synth.make_matrix(spec, 59)
    x = synth.make_x(spec, 59)[0]
    Wp = _packed(vbq, q, s, bits)
    xd = _x_dev(x)
    y = Wp.gemv(xd)
    dense = torch.from_numpy(omatmul.dequant(q, s).astype(np.float32)).cuda()
    yref32 = (dense @ xd.float()).cpu().numpy()
    ystar = omatmul.gemv(q, s, x)
    rm = omatmul.row_magnitude(q, s, x)
    parity.check(y.cpu().numpy(), ystar, rm, what=f"uniform {bits_u}")
    parity.check(yref32, ystar, rm, what="torch fp32 dense")


@pytest.mark.parametrize("bits_u", [1, 2, 4, 8])
@pytest.mark.parametrize("N,K,R,C", GEOMS)
def test_uniform_width_gemv_all_geometries(vbq, bits_u, N, K, R, C):
    """One-width matrices take the uniform kernel (no width map, positions from
    ranks), including ragged tiles whose columns hold fewer than R rows."""
    spec = synth.MatrixSpec("t", N % 5, bits_u, N, K, uniform_bits=bits_u)
    bits, q, s = synth.make_matrix(spec, 103)
    x = synth.make_x(spec, 103)[0]
    y = _packed(vbq, q, s, bits, R, C).gemv(_x_dev(x)).cpu().numpy()
    parity.check(y, omatmul.gemv(q, s, x), omatmul.row_magnitude(q, s, x), what=f"uniform {bits_u}")


@pytest.mark.parametrize("M", [1, 2, 3, 4, 8, 11, 16])
@pytest.mark.parametrize("N,K,R,C", [(257, 768, 16, 12), (130, 4096, 64, 64), (64, 14336, 16, 112)])
def test_gemm_small_matches_oracle(vbq, M, N, K, R, C):
    _say(f"gemm_small M={M} N={N} K={K}")
    spec = synth.MatrixSpec("t", 1, 2, N, K)
    bits, q, s = synth.make_matrix(spec, 61)
    X = synth.make_x(spec, 61, M=M)
    Wp = _packed(vbq, q, s, bits, R, C)
    Y = Wp.gemm_small(_x_dev(X)).cpu().numpy()
    Ystar = omatmul.gemm(q, s, X)
    for m in range(M):
        parity.check(Y[m], Ystar[m], omatmul.row_magnitude(q, s, X[m]), what=f"gemm m={m}")


@pytest.mark.parametrize("M", [3, 16])
@pytest.mark.parametrize("N,K,R,C", GEOMS)
def test_gemm_small_all_geometries(vbq, M, N, K, R, C):
    """Matrix-core path (M >= 3) on every tile height (row groups of 16/32/64
    rows, several groups per tile for R = 128/256), ragged tiles and chunks."""
    _say(f"gemm_small geometry M={M} N={N} K={K} R={R} C={C}")
    spec = synth.MatrixSpec("t", N % 7, K % 5, N, K)
    bits, q, s = synth.make_matrix(spec, 83)
    X = synth.make_x(spec, 83, M=M)
    Y = _packed(vbq, q, s, bits, R, C).gemm_small(_x_dev(X)).cpu().numpy()
    Ystar = omatmul.gemm(q, s, X)
    for m in range(M):
        parity.check(Y[m], Ystar[m], omatmul.row_magnitude(q, s, X[m]), what=f"gemm m={m}")


@pytest.mark.parametrize("M", [2, 4, 16])
def test_gemm_small_one_hot_rows_are_exact(vbq, M):
    """Row m of X = e_{k_m}: row m of Y is column k_m of w_hat, bit for bit
    (levels are exact in fp16 and s * q is exact in fp32)."""
    spec = synth.MatrixSpec("t", 3, 1, 300, 1024)
    bits, q, s = synth.make_matrix(spec, 89)
    W = omatmul.dequant(q, s)
    ks = [(37 * m + 5) % 1024 for m in range(M)]
    X = np.zeros((M, 1024), dtype=np.float16)
    for m, k in enumerate(ks):
        X[m, k] = 1.0
    Y = _packed(vbq, q, s, bits, 64, 16).gemm_small(_x_dev(X)).cpu().numpy().astype(np.float64)
    for m, k in enumerate(ks):
        assert np.array_equal(Y[m], W[:, k]), (m, k)


@pytest.mark.parametrize("bits_u", [1, 2, 4, 8])
def test_gemm_small_uniform_widths(vbq, bits_u):
    spec = synth.MatrixSpec("t", 1, 4, 160, 2048, uniform_bits=bits_u)
    bits, q, s = synth.make_matrix(spec, 97)
    X = synth.make_x(spec, 97, M=8)
    Y = _packed(vbq, q, s, bits).gemm_small(_x_dev(X)).cpu().numpy()
    Ystar = omatmul.gemm(q, s, X)
    for m in range(8):
        parity.check(Y[m], Ystar[m], omatmul.row_magnitude(q, s, X[m]), what=f"uniform {bits_u} m={m}")


def test_gemm_small_bitwise_repeatable(vbq):
    spec = synth.MatrixSpec("t", 2, 5, 1000, 4096)
    bits, q, s = synth.make_matrix(spec, 101)
    Wp = _packed(vbq, q, s, bits)
    X = _x_dev(synth.make_x(spec, 101, M=16))
    y0 = Wp.gemm_small(X).cpu().numpy()
    for _ in range(3):
        assert np.array_equal(Wp.gemm_small(X).cpu().numpy(), y0)


def test_gemm_small_strided_and_empty(vbq):
    spec = synth.MatrixSpec("t", 1, 3, 200, 512)
    bits, q, s = synth.make_matrix(spec, 67)
    X = synth.make_x(spec, 67, M=5)
    Wp = _packed(vbq, q, s, bits)
    Xpad = torch.zeros((5, 512 + 64), dtype=torch.float16, device="cuda")
    Xpad[:, :512] = _x_dev(X)
    Ypad = torch.full((5, 256), 7.0, dtype=torch.float32, device="cuda")
    Wp.gemm_small(Xpad[:, :512], Ypad[:, :200])
    Yh = Ypad.cpu().numpy()
    Ystar = omatmul.gemm(q, s, X)
    for m in range(5):
        parity.check(Yh[m, :200], Ystar[m], omatmul.row_magnitude(q, s, X[m]))
    assert np.all(Yh[:, 200:] == 7.0)  # nothing written past N
    Wp.gemm_small(Xpad[:0, :512], Ypad[:0, :200])  # M = 0 is a no-op


def test_quantizer_path_bit_exact(vbq):
    """vbq_pack (C++ quantizer) -> device dequant equals oracle quantize -> dequant."""
    rng = synth.rng_for(71)
    W = synth.draw_weights(rng, 333, 1024, std=0.05)
    bits = synth.draw_bits(rng, 333, 16, synth.MIX_PILOT)
    blob, d = vbq.pack(W, bits)
    Wp = vbq.PackedMatrix(blob, d)
    q, s = oquant.quantize(W, bits)
    assert np.array_equal(Wp.dequant().cpu().numpy().astype(np.float64), omatmul.dequant(q, s))


def test_blob_roundtrip_through_device(vbq):
    spec = synth.MatrixSpec("t", 2, 2, 77, 640)
    bits, q, s = synth.make_matrix(spec, 73)
    Wp = _packed(vbq, q, s, bits, 16, 3)
    back = Wp.blob.cpu().numpy()
    q2, s2, b2 = olayout.unpack(back, Wp.desc.info())
    assert np.array_equal(q2, q) and np.array_equal(s2, s) and np.array_equal(b2, bits)


# ------------------------------------------------------------------ full-size workloads (sampled rows)

def _sampled_check(vbq, spec, seed, M=1, n_rows=192):
    bits, q, s = synth.make_matrix(spec, seed)
    X = synth.make_x(spec, seed, M=M)
    Wp = _packed(vbq, q, s, bits)
    if M == 1:
        Y = Wp.gemv(_x_dev(X[0])).cpu().numpy()[None, :]
    else:
        Y = Wp.gemm_small(_x_dev(X)).cpu().numpy()
    rows = np.unique(np.concatenate([np.arange(min(16, spec.N)), np.arange(max(0, spec.N - 16), spec.N),
                                     synth.rng_for(seed, 9).choice(spec.N, size=min(n_rows, spec.N), replace=False)]))
    worst = 0.0
    for m in range(M):
        ystar = omatmul.gemv(q[rows], s[rows], X[m])
        worst = max(worst, parity.check(Y[m, rows], ystar, omatmul.row_magnitude(q[rows], s[rows], X[m]),
                                        what=f"{spec.name} L{spec.layer} m={m}"))
    assert np.all(np.isfinite(Y))
    return worst


@pytest.mark.parametrize("cfg", [0, 1, 2, 3, 4])
def test_workload_matrices_full_size(vbq, cfg):
    wl = synth.workload(cfg)
    mats = wl.matrices if cfg == 0 else [m for m in wl.matrices if m.layer in (0, 1) and m.proj in (0, 3)] + \
        [m for m in wl.matrices if m.layer == 0 and m.proj in (1, 2)] + [wl.matrices[-1]]
    for spec in mats:
        for M in ((1, 2, 4, 8, 16) if cfg == 4 else (1,)):  # every batch size bench.py times
            w = _sampled_check(vbq, spec, wl.seed, M=M)
            _say(f"cfg{cfg} {spec.name} L{spec.layer} {spec.N}x{spec.K} M={M}: max rel err {w:.2e}")


@pytest.mark.parametrize("ub", [1, 2, 4, 8])
def test_workload4_uniform_variants(vbq, ub):
    wl = synth.workload(4, uniform_bits=ub)
    for spec in (wl.matrices[2], wl.matrices[-1]):
        w = _sampled_check(vbq, spec, wl.seed)
        _say(f"cfg4 u{ub} {spec.name} {spec.N}x{spec.K}: max rel err {w:.2e}")


# ------------------------------------------------------------------ recipe mode

def test_gemv_rows_index_map(vbq):
    """vbq_gemv_rows writes row n to y[rows[n]] with the same value vbq_gemv
    gives (same kernel, same order: bitwise), skips indices outside y and
    leaves every other entry of y alone."""
    spec = synth.MatrixSpec("t", 0, 0, 500, 1024)
    bits, q, s = synth.make_matrix(spec, 79)
    Wp = _packed(vbq, q, s, bits)
    xd = _x_dev(synth.make_x(spec, 79)[0])
    y_ref = Wp.gemv(xd).cpu().numpy()
    ylen = 1200
    rows = synth.rng_for(79, 3).permutation(ylen)[:spec.N].astype(np.int32)
    rows[[3, 77, 499]] = [-1, ylen, 1 << 30]  # not written
    y = torch.full((ylen,), -7.0, dtype=torch.float32, device="cuda")
    Wp.gemv_rows(xd, y, torch.from_numpy(rows).cuda())
    y = y.cpu().numpy()
    ok = (rows >= 0) & (rows < ylen)
    assert np.array_equal(y[rows[ok]], y_ref[ok])
    untouched = np.ones(ylen, dtype=bool)
    untouched[rows[ok]] = False
    assert np.all(y[untouched] == -7.0)


def test_gemv_rows_repeated_indices_and_empty_output(vbq):
    """Rows sharing an index write one of their own values there (which one is
    not defined); with y_len = 0 every index is outside y and nothing is
    written."""
    spec = synth.MatrixSpec("t", 0, 0, 300, 640)
    bits, q, s = synth.make_matrix(spec, 83)
    Wp = _packed(vbq, q, s, bits)
    xd = _x_dev(synth.make_x(spec, 83)[0])
    y_ref = Wp.gemv(xd).cpu().numpy()
    ylen = 40
    rows = (np.arange(spec.N) % ylen).astype(np.int32)  # every index shared by 7 or 8 rows
    y = torch.full((ylen,), -7.0, dtype=torch.float32, device="cuda")
    Wp.gemv_rows(xd, y, torch.from_numpy(rows).cuda())
    y = y.cpu().numpy()
    for i in range(ylen):
        assert y[i] in set(y_ref[rows == i].tolist()), i
    y0 = torch.full((8,), -7.0, dtype=torch.float32, device="cuda")
    rows_d = torch.from_numpy(rows).cuda()
    st = vbq.raw_gemv_rows(Wp.desc, Wp.blob.data_ptr(), xd.data_ptr(), y0.data_ptr(), 0, rows_d.data_ptr(),
                           torch.cuda.current_stream().cuda_stream)
    assert st == 0
    torch.cuda.synchronize()
    assert np.all(y0.cpu().numpy() == -7.0)


@pytest.mark.parametrize("N,K", [(3000, 1024), (700, 4096), (100, 640)])
def test_row_buckets_match_oracle(vbq, N, K):
    """A frequency-tiered head (the recipe's 8/4/2/1-bit rows) packed as four
    one-width row buckets: the bucketed product matches the oracle, and the
    same matrix packed whole (width map, mixed-width kernel) within the same
    tolerance."""
    _say(f"row buckets N={N} K={K}")
    spec = synth.MatrixSpec("h", 0, 4, N, K, row_tiers=synth.RECIPE_HEAD_TIERS)
    bits, q, s = synth.make_matrix(spec, 83)
    x = synth.make_x(spec, 83)[0]
    xd = _x_dev(x)
    Wb = vbq.BucketedMatrix(vbq.pack_row_buckets(q, s, bits), N, K)
    y_b = Wb.gemv(xd).cpu().numpy()
    y_w = _packed(vbq, q, s, bits).gemv(xd).cpu().numpy()
    want, mag = omatmul.gemv(q, s, x), omatmul.row_magnitude(q, s, x)
    rel = parity.check(y_b, want, mag, what=f"bucketed {N}x{K}")
    parity.check(y_w, want, mag, what=f"whole {N}x{K}")
    _say(f"  max rel err {rel:.2e}")


@pytest.mark.parametrize("N,K,tiers", [(3000, 1024, None), (100, 640, None), (128256, 4096, None),
                                        (700, 4096, ((0.5, 1), (0.5, 8))), (5000, 2048, ((0.9, 2), (0.1, 4)))])
def test_buckets_one_launch_bitwise_per_bucket(vbq, N, K, tiers):
    """vbq_gemv_buckets runs every row bucket in one launch (vbq_buckets_kernel<4>):
    bit for bit the per-bucket vbq_gemv_rows launches, fp32 and fp16 outputs,
    including buckets of a single partial tile (100 rows over four widths)."""
    spec = synth.MatrixSpec("h", 0, 4, N, K, row_tiers=tiers or synth.RECIPE_HEAD_TIERS)
    bits, q, s = synth.make_matrix(spec, 211)
    x = _x_dev(synth.make_x(spec, 211)[0])
    rb = vbq.pack_row_buckets(q, s, bits)
    one = vbq.BucketedMatrix(rb, N, K)
    each = vbq.BucketedMatrix(list(rb), N, K)
    assert one.kernel_name() == "vbq_buckets_kernel<4>" and each.kernel_name() == "per bucket"
    _say(f"buckets N={N} K={K}: {[(b, p.N, p.desc.tile_rows) for b, p, _ in one.parts]}")
    for dt in (torch.float32, torch.float16):
        y1 = torch.full((N,), float("nan"), dtype=dt, device="cuda")
        y2 = torch.full((N,), float("nan"), dtype=dt, device="cuda")
        one.gemv(x, y1)
        each.gemv(x, y2)
        torch.cuda.synchronize()
        assert torch.isfinite(y1.float()).all(), dt
        assert torch.equal(y1, y2), dt
    if N <= 5000:
        y = one.gemv(x).cpu().numpy()
        xh = synth.make_x(spec, 211)[0]
        parity.check(y, omatmul.gemv(q, s, xh), omatmul.row_magnitude(q, s, xh), what=f"one-launch buckets {N}x{K}")


def test_buckets_one_launch_short_y(vbq):
    """Rows whose output index is past y_len are skipped in the one-launch path
    as in vbq_gemv_rows (a y of the first 1000 rows of a 3000-row head)."""
    N, K = 3000, 1024
    spec = synth.MatrixSpec("h", 0, 4, N, K, row_tiers=synth.RECIPE_HEAD_TIERS)
    bits, q, s = synth.make_matrix(spec, 223)
    x = _x_dev(synth.make_x(spec, 223)[0])
    one = vbq.BucketedMatrix(vbq.pack_row_buckets(q, s, bits), N, K)
    full = one.gemv(x)
    y = torch.full((1008,), -5.0, dtype=torch.float32, device="cuda")
    st = vbq.raw_gemv_buckets(one.call_table(torch.float32), one.n_buckets, one.blob.data_ptr(),
                              one.row_index.data_ptr(), x.data_ptr(), y.data_ptr(), 1000, 0)
    assert st == 0
    torch.cuda.synchronize()
    assert torch.equal(y[:1000], full[:1000])
    assert torch.all(y[1000:] == -5.0)


def test_recipe_workload_full_size(vbq):
    """The 9B-class recipe step at full size: uniform 2- and 4-bit projections
    (the one-width kernel) and the tiered LM head as row buckets, sampled rows
    against the oracle."""
    wl = synth.workload(3, recipe=True)
    picks = [m for m in wl.matrices if m.layer == 0] + [m for m in wl.matrices if m.layer == 1 and m.proj == 3]
    for spec in picks:
        w = _sampled_check(vbq, spec, wl.seed)
        _say(f"recipe {spec.name} L{spec.layer} {spec.N}x{spec.K}: max rel err {w:.2e}")
    head = wl.matrices[-1]
    bits, q, s = synth.make_matrix(head, wl.seed)
    x = synth.make_x(head, wl.seed)[0]
    Wb = vbq.BucketedMatrix(vbq.pack_row_buckets(q, s, bits), head.N, head.K)
    y = Wb.gemv(_x_dev(x)).cpu().numpy()
    w = bits[:, 0]
    rows = np.unique(np.concatenate([np.nonzero(w == b)[0][:24] for b in (1, 2, 4, 8)] +
                                    [synth.rng_for(wl.seed, 9).choice(head.N, size=160, replace=False)]))
    rel = parity.check(y[rows], omatmul.gemv(q[rows], s[rows], x), omatmul.row_magnitude(q[rows], s[rows], x),
                       what="recipe head")
    assert np.all(np.isfinite(y))
    _say(f"recipe head {head.N}x{head.K} (4 buckets): max rel err {rel:.2e}")


@pytest.mark.parametrize("N,K", [(33, 1 << 20), ((1 << 20) + 3, 64)])
def test_extreme_aspect_ratios(vbq, N, K):
    # a very wide matrix (16384 group columns, a ragged 33-row tile) and a very tall one
    # (one group column, 2^20 + 3 rows): every row checked against the oracle, GEMV and M = 4
    _say(f"extreme shape N={N} K={K}")
    spec = synth.MatrixSpec("t", 0, 0, N, K)
    bits, q, s = synth.make_matrix(spec, 53)
    Wp = _packed(vbq, q, s, bits)
    X = synth.make_x(spec, 53, M=4)
    y = Wp.gemv(_x_dev(X[0])).cpu().numpy()
    parity.check(y, omatmul.gemv(q, s, X[0]), omatmul.row_magnitude(q, s, X[0]), what=f"gemv {N}x{K}")
    Y = Wp.gemm_small(_x_dev(X)).cpu().numpy()
    for m in range(4):
        parity.check(Y[m], omatmul.gemv(q, s, X[m]), omatmul.row_magnitude(q, s, X[m]), what=f"M=4 row {m}")
    if N < 64:  # one-hot columns of the wide matrix, including the last group column
        W = omatmul.dequant(q, s)
        for k in (0, 64 * 8191 + 5, K - 1):
            e = np.zeros(K, dtype=np.float16)
            e[k] = 1.0
            assert np.array_equal(Wp.gemv(_x_dev(e)).cpu().numpy().astype(np.float64), W[:, k]), k
