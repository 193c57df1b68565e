"""Host-side checks of libvbq that need no GPU.

* the library loads and exports every entry point include/vbq.h declares;
* vbq_pack_codes writes exactly the bytes of the oracle's independent packer
  (bit-exact, several geometries, ragged tiles and chunks);
* vbq_pack (C++ quantizer) matches the oracle quantizer + packer byte for byte,
  including rounding ties, stored-scale rounding, sign(0), zero groups and
  subnormal scales;
* every documented error path returns its status code.
"""

import ctypes
import json
import os
import re

import numpy as np
import pytest

from oracle import layout as olayout
from oracle import quant as oquant
from paper_2607_02893_amd import synth
from paper_2607_02893_amd import vbq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_exports_every_declared_symbol():
    with open(os.path.join(ROOT, "include", "vbq.h")) as f:
        hdr = f.read()
    declared = set(re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\*?\s+\*?(vbq_[a-z_0-9]+)\s*\(", hdr, re.M))
    assert declared == set(vbq.EXPORTS), declared ^ set(vbq.EXPORTS)
    lib = vbq.lib()
    for name in declared:
        assert hasattr(lib, name), name
    assert vbq.layout_version() == vbq.LAYOUT_VERSION == 1
    assert ctypes.sizeof(vbq.VbqDesc) == 272
    for s in range(11):
        assert vbq.status_string(s)


def _random_codes(rng, N, K, mix=synth.MIX_PILOT):
    bits = synth.draw_bits(rng, N, K // 64, mix)
    return bits, synth.draw_levels(rng, bits), synth.draw_scales(rng, N, K // 64)


@pytest.mark.parametrize("N,K,R,C", [(1, 64, 16, 1), (37, 320, 16, 2), (100, 768, 64, 12), (130, 1024, 32, 5),
                                     (64, 4096, 64, 64), (300, 640, 256, 3), (513, 512, 0, 0), (17, 896, 16, 7)])
def test_pack_codes_bytes_match_oracle(N, K, R, C):
    rng = synth.rng_for(5, N, K)
    bits, q, s = _random_codes(rng, N, K)
    blob, d = vbq.pack_codes(q, s, bits, tile_rows=R, chunk_groups=C)
    assert vbq.desc_check(d) == 0
    info = d.info()
    oblob, oinfo = olayout.pack(q, s, bits, info["R"], info["C"])
    for key in ("T", "U", "units", "n_entries", "section_off", "section_len", "total_bytes"):
        assert info[key] == oinfo[key], key
    assert np.array_equal(np.asarray(blob), oblob)


def test_pack_codes_hand_fixture(golden_dir):
    with open(os.path.join(golden_dir, "layout_tiny.json")) as f:
        fx = json.load(f)
    N, K = fx["N"], fx["K"]
    q = np.zeros((N, K), dtype=np.int8)
    s = np.zeros((N, K // 64), dtype=np.uint16)
    for r in range(N):
        for j in range(K // 64):
            g = fx["groups"][f"r{r}j{j}"]
            qq = [g["default_q"]] * 64
            for k, v in g["q_overrides"].items():
                qq[int(k)] = v
            q[r, 64 * j:64 * j + 64] = qq
            s[r, j] = int(g["s_bits"], 16)
    blob, d = vbq.pack_codes(q, s, np.array(fx["bits"], dtype=np.uint8), tile_rows=fx["R"], chunk_groups=fx["C"])
    ex = fx["expected"]
    assert list(d.section_off) == ex["section_off"] and list(d.section_len) == ex["section_len"]
    assert d.total_bytes == ex["total_bytes"]
    b = np.asarray(blob)
    wmap = np.frombuffer(b[256:272].tobytes(), dtype=np.uint64)
    assert [int(w) for w in wmap] == [int(w, 16) for w in ex["wmap"]]
    codes8 = np.frombuffer(b[1024:1088].tobytes(), dtype=np.uint32)
    assert [int(w) for w in codes8] == [int(w, 16) for w in fx["groups"]["r1j0"]["words"]]


def _quant_inputs(rng, N, K):
    W = synth.draw_weights(rng, N, K, std=1.0)
    bits = synth.draw_bits(rng, N, K // 64, {1: .25, 2: .25, 4: .25, 8: .25})
    W = W * rng.uniform(1e-3, 10, (N, 1)).astype(np.float32)
    # special groups: zeros, ties, negative zero, tiny (subnormal scales), large
    W[0, :64] = 0.0
    W[1, :64] = np.array([7, -3.5, 0.5, -0.49, 2.5, 1.5, -7, 0] * 8, dtype=np.float32)
    bits[1, 0] = 4
    W[2, :64] = -0.0
    bits[2, 0] = 1
    W[3, :64] = rng.standard_normal(64).astype(np.float32) * 1e-6
    W[4, :64] = rng.standard_normal(64).astype(np.float32) * 3000
    W[5, 64:128] = np.array([0.3, -0.2, 0.15002, -0.1] * 16, dtype=np.float32)
    bits[5, 1] = 2
    return W, bits


@pytest.mark.parametrize("N,K,R,C", [(40, 512, 16, 0), (97, 768, 32, 5), (8, 128, 16, 1)])
def test_pack_quantizer_matches_oracle(N, K, R, C):
    rng = synth.rng_for(9, N, K)
    W, bits = _quant_inputs(rng, N, K)
    blob, d = vbq.pack(W, bits, tile_rows=R, chunk_groups=C)
    q, s = oquant.quantize(W, bits)
    oblob, _ = olayout.pack(q, s, bits, d.tile_rows, d.chunk_groups)
    assert np.array_equal(np.asarray(blob), oblob)
    q2, s2, b2 = olayout.unpack(np.asarray(blob), d.info())
    assert np.array_equal(q2, q) and np.array_equal(s2, s) and np.array_equal(b2, bits)


def test_auto_geometry_is_valid():
    for N, K in [(512, 512), (768, 3072), (4096, 14336), (28672, 4096), (128256, 4096), (1, 64)]:
        nbytes, d = vbq.pack_size(np.ones((N, K // 64), dtype=np.uint8), K)
        assert vbq.desc_check(d) == 0 and nbytes == d.total_bytes
        assert d.tile_rows in (16, 32, 64) and 1 <= d.chunk_groups <= 128
        assert d.tile_rows * d.chunk_groups <= 8192


# ------------------------------------------------------------------ error paths

def _status(fn):
    with pytest.raises(vbq.VbqError) as ei:
        fn()
    return vbq.STATUS[ei.value.status]


def test_error_paths():
    rng = synth.rng_for(3)
    bits, q, s = _random_codes(rng, 8, 256)
    assert _status(lambda: vbq.pack_codes(q[:, :200], s, bits)) in ("VBQ_ERR_SHAPE", "VBQ_ERR_BITS")
    bad = bits.copy()
    bad[3, 2] = 3
    assert _status(lambda: vbq.pack_codes(q, s, bad)) == "VBQ_ERR_BITS"
    qq = q.copy()
    bits2 = bits.copy()
    bits2[0, 0] = 2
    qq[0, :64] = 0
    qq[0, 5] = -2  # the code for -2^(b-1) is outside the level set
    assert _status(lambda: vbq.pack_codes(qq, s, bits2)) == "VBQ_ERR_CODE_RANGE"
    bits1 = bits.copy()
    bits1[0, 0] = 1
    qq[0, :64] = 1
    qq[0, 7] = 0  # 1-bit levels are +-1 only
    assert _status(lambda: vbq.pack_codes(qq, s, bits1)) == "VBQ_ERR_CODE_RANGE"
    ss = s.copy()
    ss[1, 1] = 0x7C00  # +inf
    assert _status(lambda: vbq.pack_codes(q, ss, bits)) == "VBQ_ERR_NONFINITE"
    ss[1, 1] = 0xBC00  # -1.0
    assert _status(lambda: vbq.pack_codes(q, ss, bits)) == "VBQ_ERR_SCALE_RANGE"
    W = np.zeros((4, 128), dtype=np.float32)
    b4 = np.full((4, 2), 2, dtype=np.uint8)
    W[1, 3] = np.nan
    assert _status(lambda: vbq.pack(W, b4)) == "VBQ_ERR_NONFINITE"
    W[1, 3] = np.inf
    assert _status(lambda: vbq.pack(W, b4)) == "VBQ_ERR_NONFINITE"
    W[1, 3] = 1e6  # max|w|/1 overflows fp16
    assert _status(lambda: vbq.pack(W, b4)) == "VBQ_ERR_SCALE_RANGE"
    W[1, 3] = 0.0
    # 1 bit: a mean |w| at or beyond 65520 rounds to +inf, like the oracle's OverflowError
    b1 = np.ones((4, 2), dtype=np.uint8)
    W1 = np.zeros((4, 128), dtype=np.float32)
    W1[2, :64] = 1e6
    assert _status(lambda: vbq.pack(W1, b1)) == "VBQ_ERR_SCALE_RANGE"
    W1[2, :64] = -65520.0
    assert _status(lambda: vbq.pack(W1, b1)) == "VBQ_ERR_SCALE_RANGE"
    W1[2, :64] = 65519.99  # rounds to 65504, the largest fp16: packs
    blob1, d1 = vbq.pack(W1, b1)
    q1, s1, _ = olayout.unpack(np.asarray(blob1), d1.info())
    assert int(s1[2, 0]) == 0x7BFF
    assert _status(lambda: vbq.pack(W, b4, tile_rows=24)) == "VBQ_ERR_UNSUPPORTED"
    assert _status(lambda: vbq.pack(W, b4, tile_rows=64, chunk_groups=200)) == "VBQ_ERR_UNSUPPORTED"
    assert _status(lambda: vbq.pack_size(np.ones((4, 2), np.uint8), 100)) == "VBQ_ERR_SHAPE"
    assert _status(lambda: vbq.pack_size(np.ones((4, 0), np.uint8), 0)) == "VBQ_ERR_SHAPE"


def test_null_and_buffer_errors():
    lib = vbq.lib()
    bits = np.ones((2, 2), dtype=np.uint8)
    nbytes = ctypes.c_size_t(0)
    assert lib.vbq_pack_size(2, 128, None, None, ctypes.byref(nbytes), None) == 1
    q = np.ones((2, 128), dtype=np.int8)
    s = np.full((2, 2), 0x3C00, dtype=np.uint16)
    d = vbq.VbqDesc()
    assert lib.vbq_pack_size(2, 128, bits.ctypes.data_as(ctypes.c_void_p), None, ctypes.byref(nbytes), None) == 0
    small = np.zeros((int(nbytes.value) - 256) // 8, dtype=np.uint64)
    assert lib.vbq_pack_codes(2, 128, q.ctypes.data_as(ctypes.c_void_p), s.ctypes.data_as(ctypes.c_void_p),
                              bits.ctypes.data_as(ctypes.c_void_p), None, small.ctypes.data_as(ctypes.c_void_p),
                              small.nbytes, ctypes.byref(d)) == 7
    assert lib.vbq_pack_codes(2, 128, None, s.ctypes.data_as(ctypes.c_void_p), bits.ctypes.data_as(ctypes.c_void_p),
                              None, small.ctypes.data_as(ctypes.c_void_p), small.nbytes, ctypes.byref(d)) == 1
    # device entry points reject bad descriptors before touching the GPU
    assert lib.vbq_gemv(None, None, None, None, None) == 1
    bad = vbq.VbqDesc()
    assert lib.vbq_gemv(ctypes.byref(bad), ctypes.c_void_p(256), ctypes.c_void_p(256), ctypes.c_void_p(256),
                        None) == 8
    _, good = vbq.pack_codes(q, s, bits)
    assert vbq.desc_check(good) == 0
    good.version = 2
    assert vbq.desc_check(good) == 8
    good.version = 1
    good.section_len[3] += 1
    assert vbq.desc_check(good) == 8
    good.section_len[3] -= 1
    assert lib.vbq_gemm_small(ctypes.byref(good), ctypes.c_void_p(256), 17, None, 128, None, 2, None) == 2
    assert lib.vbq_gemm_small(ctypes.byref(good), ctypes.c_void_p(256), 0, None, 128, None, 2, None) == 0
    assert lib.vbq_gemv(ctypes.byref(good), ctypes.c_void_p(100), ctypes.c_void_p(256), ctypes.c_void_p(256),
                        None) == 7


def test_call_flags_are_checked_before_any_launch():
    """Descriptor call options: unknown bits are refused, VBQ_Y_F16 needs only
    2-byte alignment of y; all of it before anything touches the GPU."""
    lib = vbq.lib()
    rng = synth.rng_for(4)
    bits, q, s = _random_codes(rng, 8, 256)
    _, d = vbq.pack_codes(q, s, bits)
    A = 1 << 20  # aligned stand-in addresses, never dereferenced on this path
    d.flags = 4
    assert lib.vbq_gemv(ctypes.byref(d), ctypes.c_void_p(A), ctypes.c_void_p(A), ctypes.c_void_p(A), None) == 10
    assert lib.vbq_gemm_small(ctypes.byref(d), ctypes.c_void_p(A), 3, ctypes.c_void_p(A), 256,
                              ctypes.c_void_p(A), 8, None) == 10
    assert lib.vbq_gemv_rows(ctypes.byref(d), ctypes.c_void_p(A), ctypes.c_void_p(A), ctypes.c_void_p(A), 8,
                             ctypes.c_void_p(A), None) == 10
    d.flags = 0  # float y must be 4-byte aligned
    assert lib.vbq_gemv(ctypes.byref(d), ctypes.c_void_p(A), ctypes.c_void_p(A), ctypes.c_void_p(A + 2), None) == 7
    d.flags = vbq.Y_F16  # fp16 y: 2-byte alignment, an odd address is refused
    assert lib.vbq_gemv(ctypes.byref(d), ctypes.c_void_p(A), ctypes.c_void_p(A), ctypes.c_void_p(A + 1), None) == 7
    assert lib.vbq_gemm_small(ctypes.byref(d), ctypes.c_void_p(A), 4, ctypes.c_void_p(A), 256,
                              ctypes.c_void_p(A + 1), 8, None) == 7
    d.flags = vbq.Y_F16 | vbq.ONE_WAVE_PER_UNIT
    assert vbq.desc_check(d) == 0  # the options are not part of the layout


def test_pack_row_buckets_c_abi():
    """vbq_pack_row_buckets: every bucket's bytes are the oracle packer's bytes
    for that width's rows, at a 256-byte aligned offset; row_index lists the
    rows bucket by bucket; the size call agrees."""
    spec = synth.MatrixSpec("h", 0, 4, 513, 768, row_tiers=synth.RECIPE_HEAD_TIERS)
    bits, q, s = synth.make_matrix(spec, 75)
    w = bits[:, 0]
    blob, bk, row_index = vbq.pack_row_buckets_raw(q, s, w, tile_rows=32)
    assert [b.bits for b in bk] == sorted(set(int(v) for v in w))
    assert sorted(row_index.tolist()) == list(range(spec.N))
    end = 0
    for b in bk:
        assert b.blob_offset % 256 == 0 and b.blob_offset >= end and b.reserved == 0
        rows = row_index[b.row_begin:b.row_begin + b.n_rows]
        assert np.all(np.diff(rows) > 0) and np.all(w[rows] == b.bits) and b.desc.N == b.n_rows
        ob, _ = olayout.pack(q[rows], s[rows], bits[rows], b.desc.tile_rows, b.desc.chunk_groups)
        got = np.asarray(blob)[b.blob_offset:b.blob_offset + b.desc.total_bytes]
        assert np.array_equal(got, np.asarray(ob))
        end = b.blob_offset + b.desc.total_bytes
    lib = vbq.lib()
    nbytes, nb = ctypes.c_size_t(0), ctypes.c_int32(0)
    wb = np.ascontiguousarray(w)
    o32 = vbq.VbqPackOpts(32, 0, 0, 0)
    assert lib.vbq_pack_row_buckets_size(spec.N, spec.K, wb.ctypes.data_as(ctypes.c_void_p), ctypes.byref(o32),
                                         ctypes.byref(nbytes), ctypes.byref(nb)) == 0
    assert nb.value == len(bk) and nbytes.value == end
    # errors: a width outside {1,2,4,8}, NULL, a buffer too small, a level outside its width's set
    bad = wb.copy()
    bad[7] = 3
    assert _status(lambda: vbq.pack_row_buckets_raw(q, s, bad)) == "VBQ_ERR_BITS"
    assert lib.vbq_pack_row_buckets_size(spec.N, spec.K, None, None, ctypes.byref(nbytes), ctypes.byref(nb)) == 1
    small = np.zeros(64, dtype=np.uint64)
    out = (vbq.VbqBucket * vbq.MAX_BUCKETS)()
    ri = np.zeros(spec.N, dtype=np.int32)
    assert lib.vbq_pack_row_buckets(spec.N, spec.K, q.ctypes.data_as(ctypes.c_void_p),
                                    s.ctypes.data_as(ctypes.c_void_p), wb.ctypes.data_as(ctypes.c_void_p), None,
                                    small.ctypes.data_as(ctypes.c_void_p), small.nbytes, out, ctypes.byref(nb),
                                    ri.ctypes.data_as(ctypes.c_void_p)) == 7
    qq = np.array(q)
    r1 = int(np.nonzero(w == 1)[0][0])
    qq[r1, 0] = 0  # 1-bit levels are +-1
    assert _status(lambda: vbq.pack_row_buckets_raw(qq, s, w)) == "VBQ_ERR_CODE_RANGE"
    # vbq_gemv_buckets: bucket count checked first, none is a no-op
    assert lib.vbq_gemv_buckets(out, 5, None, None, None, None, 0, None) == 2
    assert lib.vbq_gemv_buckets(out, -1, None, None, None, None, 0, None) == 2
    assert lib.vbq_gemv_buckets(out, 0, None, None, None, None, 0, None) == 0
    assert lib.vbq_gemv_buckets(out, 1, None, None, None, None, 0, None) == 1


def test_buckets_kernel_choice():
    """vbq_gemv_buckets_kernel_name (descriptors only): a tiered head's buckets
    take one launch; one bucket, buckets whose one-width kernel would use more
    than four waves (K = 16384: eight units per tile), or buckets with unequal
    flags take one vbq_gemv_rows each; no bucket is "none"."""
    spec = synth.MatrixSpec("h", 0, 4, 3000, 1024, row_tiers=synth.RECIPE_HEAD_TIERS)
    bits, q, s = synth.make_matrix(spec, 61)
    rb = vbq.pack_row_buckets(q, s, bits)
    assert len(rb.buckets) == 4
    assert vbq.buckets_kernel_name(rb.buckets) == "vbq_buckets_kernel<4>"
    assert vbq.buckets_kernel_name(rb.buckets[:2]) == "vbq_buckets_kernel<4>"
    assert vbq.buckets_kernel_name(rb.buckets[:1]) == "per bucket"
    assert vbq.buckets_kernel_name([]) == "none"
    mixed = [vbq.VbqBucket.from_buffer_copy(b) for b in rb.buckets]
    mixed[1].desc.flags = vbq.Y_F16
    assert vbq.buckets_kernel_name(mixed) == "per bucket"
    wide = synth.MatrixSpec("w", 0, 4, 200, 16384, row_tiers=((0.5, 1), (0.5, 2)))
    bits, q, s = synth.make_matrix(wide, 67)
    assert vbq.buckets_kernel_name(vbq.pack_row_buckets(q, s, bits).buckets) == "per bucket"


def test_step_plan_argument_errors():
    """vbq_step_plan / _bytes / _run check everything on the host first."""
    lib = vbq.lib()
    nb = ctypes.c_size_t(0)
    assert lib.vbq_step_plan_bytes(0, ctypes.byref(nb)) == 2
    assert lib.vbq_step_plan_bytes(1, None) == 1
    assert lib.vbq_step_plan_bytes(3, ctypes.byref(nb)) == 0 and nb.value > 0
    per = nb.value // 3
    assert lib.vbq_step_workspace_bytes(3, ctypes.byref(nb)) == 0 and nb.value == 4 * (8 * 32 * 3 + 1)
    rng = synth.rng_for(6)
    bits, q, s = _random_codes(rng, 40, 1024)
    _, d = vbq.pack_codes(q, s, bits)
    A = 1 << 20
    plan = np.zeros(4 * per, dtype=np.uint8)

    def plan_of(desc, x=A, y=A, rows=None, y_len=0, n=1, buf=plan):
        g = (vbq.VbqStepGemv * 1)(vbq.VbqStepGemv(ctypes.pointer(desc), A, x, y, rows, y_len))
        return lib.vbq_step_plan(g, n, buf.ctypes.data_as(ctypes.c_void_p), buf.nbytes)
    assert plan_of(d) == 0
    assert plan_of(d, n=0) == 2
    assert plan_of(d, x=A + 8) == 7                 # x misaligned
    assert plan_of(d, y=A + 2) == 7                 # float y misaligned
    assert plan_of(d, x=0) == 1
    small = np.zeros(per - 8, dtype=np.uint8)
    assert plan_of(d, buf=small) == 7               # plan buffer too small
    assert plan_of(d, rows=A + 2, y_len=40) == 7    # row map misaligned
    assert plan_of(d, rows=A, y_len=-1) == 2
    d.flags = vbq.ONE_WAVE_PER_UNIT
    assert plan_of(d) == 10
    d.flags = 0
    _, dwide = vbq.pack_codes(q, s, bits, chunk_groups=1)  # 16 units per tile: beyond the pair body
    assert plan_of(dwide) == 10
    bad = vbq.VbqDesc()
    assert plan_of(bad) == 8
    assert lib.vbq_step_run(None, 1, ctypes.c_void_p(A), 64, 0, None) == 1
    assert lib.vbq_step_run(ctypes.c_void_p(A), 2, ctypes.c_void_p(A), 4 * 8 * 32, 0, None) == 7  # workspace too small
    assert lib.vbq_step_run(ctypes.c_void_p(A), 0, ctypes.c_void_p(A), 64, 0, None) == 2


def test_single_hip_runtime():
    """libvbq must share torch's HIP runtime: one libamdhip64 in the process."""
    assert len(vbq.hip_runtimes()) == 1


# ------------------------------------------------------------------ recipe mode

def test_recipe_workload_widths():
    """The recipe variant (paper section 4): layer-0 MLP at 4 bits, every other
    projection at 2 bits, the head tiered 0.5 / 1.5 / 10 / 88 % of rows at
    8 / 4 / 2 / 1 bits (mean 1.18 bits per weight)."""
    wl = synth.workload(4, recipe=True)
    for spec in wl.matrices[:-1]:
        bits, _ = synth.make_bits(spec, wl.seed)
        want = 4 if (spec.layer == 0 and spec.name in ("gate_up", "down")) else 2
        assert np.all(bits == want), (spec.name, spec.layer)
    head = wl.matrices[-1]
    bits, _ = synth.make_bits(head, wl.seed)
    w = bits[:, 0]
    assert np.all(bits == w[:, None])
    N = head.N
    counts = {b: int(np.count_nonzero(w == b)) for b in (1, 2, 4, 8)}
    assert counts[8] == round(0.005 * N) and counts[4] == round(0.015 * N) and counts[2] == round(0.10 * N)
    assert sum(counts.values()) == N
    assert abs(w.mean() - 1.18) < 0.005
    # the tiers are not contiguous row ranges (a frequency rank is not the row order)
    assert np.any(np.diff(np.nonzero(w == 8)[0]) > 1)


def test_pack_row_buckets_partition_and_bytes():
    """One packed matrix per width: the buckets partition the rows in order,
    each bucket has one width (no width-map words beyond its geometry's zero
    planes) and its bytes equal the oracle's packer on the same rows."""
    spec = synth.MatrixSpec("h", 0, 4, 777, 640, row_tiers=synth.RECIPE_HEAD_TIERS)
    bits, q, s = synth.make_matrix(spec, 71)
    bk = vbq.pack_row_buckets(q, s, bits)
    rows_all = np.sort(np.concatenate([r for _, r, _, _ in bk]))
    assert np.array_equal(rows_all, np.arange(spec.N))
    for b, rows, blob, d in bk:
        assert rows.dtype == np.int32 and np.all(np.diff(rows) > 0)
        assert np.all(bits[rows] == b)
        c = {1: 0, 2: 1, 4: 2, 8: 3}[b]
        assert d.n_entries[c] == len(rows) * (spec.K // 64) and sum(d.n_entries) == d.n_entries[c]
        ob, _ = olayout.pack(q[rows], s[rows], bits[rows], d.tile_rows, d.chunk_groups)
        assert np.array_equal(np.asarray(ob), np.asarray(blob))


def test_pack_row_buckets_rejects_mixed_rows():
    spec = synth.MatrixSpec("t", 0, 0, 40, 256)
    bits, q, s = synth.make_matrix(spec, 73)  # per-group widths
    with pytest.raises(ValueError):
        vbq.pack_row_buckets(q, s, bits)


# ------------------------------------------------- differentiable bit selection

def test_qat_workspace_size():
    assert vbq.qat_workspace_size(0) == 0
    assert vbq.qat_workspace_size(1) == 8
    assert vbq.qat_workspace_size(64) == 8
    assert vbq.qat_workspace_size(65) == 16
    big = vbq.qat_workspace_size(10 ** 9)
    assert big % 8 == 0 and 8 <= big <= 64 * 1024  # bounded by the launch, not by the size
    lib = vbq.lib()
    nb = ctypes.c_size_t(0)
    assert lib.vbq_qat_workspace_size(-1, ctypes.byref(nb)) == 2
    assert lib.vbq_qat_workspace_size(vbq.QAT_MAX_GROUPS + 1, ctypes.byref(nb)) == 2
    assert lib.vbq_qat_workspace_size(5, None) == 1


def test_qat_forward_argument_errors():
    # every case is rejected before anything is launched (fake, aligned addresses)
    A = 1 << 20  # a 16-byte aligned stand-in address, never dereferenced
    f = vbq.raw_qat_forward
    assert f(0, A, A, 0, 1.0, A, 0, 0, 0, 0, 0, 0) == 0            # n_groups == 0: nothing to do
    assert f(0, 0, 0, 0, 1.0, 0, 0, 0, A, 0, 0, 0) == 0            # ... and pointers may be NULL
    assert f(0, A, A, 0, 0.0, A, 0, 0, 0, 0, 0, 0) == 10           # tau is checked first
    assert f(4, 0, A, 0, 1.0, A, 0, 0, 0, 0, 0, 0) == 1            # W NULL
    assert f(4, A, 0, 0, 1.0, A, 0, 0, 0, 0, 0, 0) == 1            # logits NULL
    assert f(4, A, A, 0, 1.0, 0, 0, 0, 0, 0, 0, 0) == 1            # w_soft NULL
    assert f(-1, A, A, 0, 1.0, A, 0, 0, 0, 0, 0, 0) == 2           # n_groups < 0
    assert f(vbq.QAT_MAX_GROUPS + 1, A, A, 0, 1.0, A, 0, 0, 0, 0, 0, 0) == 2
    assert f(4, A, A, 0, float("nan"), A, 0, 0, 0, 0, 0, 0) == 5   # tau NaN
    assert f(4, A, A, 0, float("inf"), A, 0, 0, 0, 0, 0, 0) == 5   # tau Inf
    assert f(4, A, A, 0, 0.0, A, 0, 0, 0, 0, 0, 0) == 10           # tau == 0
    assert f(4, A, A, 0, -0.5, A, 0, 0, 0, 0, 0, 0) == 10          # tau < 0
    assert f(4, A, A, 0, 1e-39, A, 0, 0, 0, 0, 0, 0) == 10         # subnormal tau
    assert f(0, A, A, 0, 1.2e-38, A, 0, 0, 0, 0, 0, 0) == 0        # the smallest normal tau is accepted
    assert f(4, A + 4, A, 0, 1.0, A, 0, 0, 0, 0, 0, 0) == 7        # W misaligned
    assert f(4, A, A + 8, 0, 1.0, A, 0, 0, 0, 0, 0, 0) == 7        # logits misaligned
    assert f(4, A, A, A + 4, 1.0, A, 0, 0, 0, 0, 0, 0) == 7        # noise misaligned
    assert f(4, A, A, 0, 1.0, A + 4, 0, 0, 0, 0, 0, 0) == 7        # w_soft misaligned
    assert f(4, A, A, 0, 1.0, A, A + 4, 0, 0, 0, 0, 0) == 7        # pi misaligned
    assert f(4, A, A, 0, 1.0, A, 0, 0, A, 0, 0, 0) == 1            # bbar without workspace
    assert f(4, A, A, 0, 1.0, A, 0, 0, A + 4, A, 8, 0) == 7        # bbar misaligned
    assert f(4, A, A, 0, 1.0, A, 0, 0, A, A + 4, 8, 0) == 7        # workspace misaligned
    assert f(100, A, A, 0, 1.0, A, 0, 0, A, A, 8, 0) == 7          # workspace too small (needs 16)
    assert f(0, A, A, 0, 1.0, A, 0, 0, A, A, 0, 0) == 0            # empty: workspace of 0 bytes is enough
    assert f(4, A, A, 0, 1.0, A, 0, 0, 0, 0, 0, 0, flags=2) == 10  # unknown flag
    assert f(4, A, A, 0, 1.0, A + 8, 0, 0, 0, 0, 0, 0, flags=1) == 7  # bf16 w_soft misaligned


def test_qat_logit_grad_argument_errors():
    A = 1 << 20
    f = vbq.raw_qat_logit_grad
    assert f(0, 0, 0, 0, 1.0, 0.5, 1, 0, 0) == 0                   # nothing to do
    assert f(-1, A, A, A, 1.0, 0.5, 1, A, 0) == 2                  # n_groups < 0
    assert f(4, A, A, A, 1.0, 0.5, 0, A, 0) == 2                   # n_bbar < 1
    assert f(4, A, A, A, float("nan"), 0.5, 4, A, 0) == 5          # tau NaN
    assert f(4, A, A, A, 1.0, float("inf"), 4, A, 0) == 5          # lambda Inf
    assert f(4, A, A, A, -1.0, 0.5, 4, A, 0) == 10                 # tau < 0
    assert f(4, A, A, A, 1e-39, 0.5, 4, A, 0) == 10                # subnormal tau
    assert f(4, 0, A, A, 1.0, 0.5, 4, A, 0) == 1                   # W NULL
    assert f(4, A, 0, A, 1.0, 0.5, 4, A, 0) == 1                   # grad NULL
    assert f(4, A, A, 0, 1.0, 0.5, 4, A, 0) == 1                   # pi NULL
    assert f(4, A, A, A, 1.0, 0.5, 4, 0, 0) == 1                   # dlogits NULL
    assert f(4, A + 4, A, A, 1.0, 0.5, 4, A, 0) == 7               # misaligned
    assert f(4, A, A, A + 8, 1.0, 0.5, 4, A, 0) == 7
    assert f(4, A, A, A, 1.0, 0.5, 4, A + 4, 0) == 7


def test_binding_rejects_host_tensors_and_wrong_outputs():
    # a host pointer in a kernel would fault: the binding refuses before any call
    torch = pytest.importorskip("torch")
    W = torch.zeros(128)
    l = torch.zeros(8)
    with pytest.raises(ValueError, match="GPU tensor"):
        vbq.qat_forward(W, l, None, 1.0)
    with pytest.raises(ValueError, match="GPU tensor"):
        vbq.qat_logit_grad(W, torch.zeros(128), torch.zeros(8), 1.0, 0.1)
    with pytest.raises(ValueError):
        vbq._need(torch.zeros(3, dtype=torch.float16), "x", torch.float16, 3)
