"""CPU pins of the oracle against what the paper and the mathematics fix.

The oracle must be right before it can judge the kernels.  Each test here
checks it against something other than itself: hand-computed groups from
Eq. (1) (tests/golden), exact rational arithmetic, closed forms and
invariants.  The mutation tests at the end plant plausible mistakes in the
oracle's own steps and check that a pin catches each of them.
"""

import json
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import layout, matmul, quant, storage


def _load(golden_dir, name):
    with open(os.path.join(golden_dir, name)) as f:
        return json.load(f)


def _group_weights(g):
    if g["name"] == "ex3_1bit_sign_zero":
        return [1.0] * 32 + [-0.5] * 31 + [0.0]
    w = list(g["w_head"]) + [0.0] * (64 - len(g["w_head"]))
    return w


# ---------------------------------------------------------------- fp16 rounding

def _fp16_rne_exact(v):
    """Round a double onto the fp16 grid by exact rational arithmetic (RNE)."""
    f = Fraction(v)
    sign = -1 if f < 0 else 1
    a = abs(f)
    if a == 0:
        return 0.0
    # fp16: ulp is 2^(e-10) for normals with exponent e >= -14, 2^-24 below
    e = max(a.numerator.bit_length() - a.denominator.bit_length(), -14)
    while Fraction(2) ** e > a and e > -14:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    e = max(e, -14)
    ulp = Fraction(2) ** (e - 10)
    n = a / ulp
    lo = n.numerator // n.denominator
    rem = n - lo
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and lo % 2 == 1):
        lo += 1
    r = lo * ulp
    if r >= 65520:  # rounds past the largest finite fp16
        return sign * float("inf")
    return float(sign * r)


def test_fp16_rounding_matches_exact_rational_rne():
    rng = np.random.default_rng(7)
    vals = list(rng.uniform(-3, 3, 3000)) + list(rng.uniform(0, 1e-4, 500)) + \
        list(10.0 ** rng.uniform(-9, 4.8, 2000)) + [0.3, 1 / 127, 47.5 / 64, 65504.0, 65519.9, 2.0 ** -25,
                                                   3 * 2.0 ** -26, 1 + 2.0 ** -11, 1 + 3 * 2.0 ** -11]
    for v in vals:
        got = quant.fp16_value(quant.fp16_bits(v))
        want = _fp16_rne_exact(v)
        assert got == want or (np.isinf(got) and np.isinf(want)), (v, got, want)


# ---------------------------------------------------------------- quantizer pins

def test_hand_computed_groups(golden_dir):
    gold = _load(golden_dir, "quantizer_groups.json")
    for g in gold["groups"]:
        w = _group_weights(g)
        q, s_bits = quant.quantize_group(w, g["b"])
        assert s_bits == int(g["s_bits"], 16), g["name"]
        if "q_head" in g:
            n = len(g["q_head"])
            assert q[:n] == g["q_head"], g["name"]
            assert layout.offset_codes(q[:n], g["b"]) == g["u_head"], g["name"]
        if g["name"] == "ex3_1bit_sign_zero":
            assert q == [1] * 32 + [-1] * 31 + [1]
            assert quant.fp16_value(s_bits) == 0.7421875
        if "w_hat_0" in g:
            w_hat0 = quant.fp16_value(s_bits) * q[0]
            assert w_hat0 == g["w_hat_0"]
            assert float(np.float32(w_hat0)) == w_hat0          # exact in float32
            assert float(np.float16(w_hat0)) != w_hat0          # not in fp16


def test_vectorised_quantize_matches_group_quantizer(golden_dir):
    gold = _load(golden_dir, "quantizer_groups.json")
    rows = [_group_weights(g) for g in gold["groups"]]
    bits = [g["b"] for g in gold["groups"]]
    W = np.array([sum(rows, [])])                       # one row, 5 groups
    q, s = quant.quantize(W, np.array([bits]))
    for i, (w, b) in enumerate(zip(rows, bits)):
        qg, sg = quant.quantize_group(w, b)
        assert list(q[0, 64 * i:64 * i + 64]) == qg
        assert int(s[0, i]) == sg
    rng = np.random.default_rng(3)
    W = rng.standard_normal((9, 64 * 7)) * rng.uniform(0.01, 10, (9, 1))
    B = rng.choice([1, 2, 4, 8], size=(9, 7))
    q, s = quant.quantize(W, B)
    for r in range(9):
        for j in range(7):
            qg, sg = quant.quantize_group(W[r, 64 * j:64 * j + 64], int(B[r, j]))
            assert list(q[r, 64 * j:64 * j + 64]) == qg and int(s[r, j]) == sg


def test_tiny_gemv_examples(golden_dir):
    gold = _load(golden_dir, "quantizer_groups.json")
    byname = {g["name"]: g for g in gold["groups"]}
    for ex in gold["gemv"]:
        g = byname[ex["group"]]
        q, s_bits = quant.quantize_group(_group_weights(g), g["b"])
        x = np.zeros(64, dtype=np.float16)
        x[:len(ex["x_head"])] = ex["x_head"]
        y = matmul.gemv(np.array([q]), np.array([[s_bits]], dtype=np.uint16), x)
        assert y[0] == ex["y"]


@pytest.mark.parametrize("b", [2, 4, 8])
def test_idempotent_and_full_range(b):
    """Q(D(Q(w))) = Q(w) with the stored fp16 scale, and max|q| reaches qmax."""
    rng = np.random.default_rng(b)
    m = quant.qmax(b)
    for _ in range(400):
        w = rng.standard_normal(64) * 10.0 ** rng.uniform(-3, 2)
        q, sb = quant.quantize_group(w, b)
        s = quant.fp16_value(sb)
        assert max(abs(v) for v in q) == m
        assert all(-m <= v <= m for v in q)
        q2, sb2 = quant.quantize_group([s * v for v in q], b)
        assert q2 == q and sb2 == sb


def test_one_bit_idempotent_and_codes():
    rng = np.random.default_rng(11)
    for _ in range(400):
        w = rng.standard_normal(64) * 10.0 ** rng.uniform(-3, 2)
        q, sb = quant.quantize_group(w, 1)
        assert set(q) <= {-1, 1}
        s = quant.fp16_value(sb)
        q2, sb2 = quant.quantize_group([s * v for v in q], 1)
        assert q2 == q and sb2 == sb


def test_one_bit_is_binary_weight_rule_brute_force():
    """The 1-bit rule minimises ||w - a*sign(w)||^2 over a, at a = mean|w|
    (the classic binary-weight result); check the oracle's scale against a
    brute-force scan of a on the fp16 grid."""
    rng = np.random.default_rng(5)
    for _ in range(20):
        w = rng.standard_normal(64)
        q, sb = quant.quantize_group(w, 1)
        sgn = np.array(q, dtype=np.float64)
        grid = np.arange(0x3000, 0x3C00, dtype=np.uint16).view(np.float16).astype(np.float64)
        err = [np.sum((w - a * sgn) ** 2) for a in grid]
        best = grid[int(np.argmin(err))]
        assert abs(quant.fp16_value(sb) - best) <= 2 ** -11 * best + 1e-12


def test_zero_group_and_negative_zero():
    for b in (2, 4, 8):
        q, sb = quant.quantize_group([0.0] * 64, b)
        assert sb == 0 and q == [0] * 64
    q, sb = quant.quantize_group([-0.0] * 64, 1)
    assert sb == 0 and q == [1] * 64


@pytest.mark.filterwarnings("ignore:overflow encountered in cast")
def test_scale_overflow_raises():
    """A stored scale must be a finite fp16 value at every width (reading R3);
    the packer reports the same groups as VBQ_ERR_SCALE_RANGE."""
    with pytest.raises(OverflowError):
        quant.quantize_group([1e6] + [0.0] * 63, 2)
    with pytest.raises(OverflowError):
        quant.quantize(np.array([[1e6] + [0.0] * 63]), np.array([[4]]))
    # 1 bit: the mean |w| is the scale; 1e6 rounds to +inf in fp16
    with pytest.raises(OverflowError):
        quant.quantize_group([1e6] * 64, 1)
    with pytest.raises(OverflowError):
        quant.quantize(np.array([[1e6] * 64]), np.array([[1]]))
    # 65519.99 rounds down to 65504 (the largest fp16), 65520 rounds to +inf
    q, sb = quant.quantize_group([65519.99] * 64, 1)
    assert sb == 0x7BFF and q == [1] * 64
    with pytest.raises(OverflowError):
        quant.quantize_group([-65520.0] * 64, 1)
    qv, sv = quant.quantize(np.array([[65519.99] * 64]), np.array([[1]]))
    assert int(sv[0, 0]) == 0x7BFF


def test_group_size_one_is_degenerate():
    """Paper section 3.1 ("Why group size matters"): with G = 1 every width
    reproduces the weight, so there is nothing to choose.  Exact with a double
    scale; within fp16 rounding of the scale when it is stored in fp16."""
    rng = np.random.default_rng(13)
    for v in rng.standard_normal(300) * 3:
        outs = []
        for b in (1, 2, 4, 8):
            q, s = quant.quantize_group([v], b, group=1, exact_scale=True)
            assert abs(s * q[0] - v) <= 4 * np.finfo(np.float64).eps * abs(v)  # exact up to double rounding
            q, sb = quant.quantize_group([v], b, group=1)
            w_hat = quant.fp16_value(sb) * q[0]
            assert abs(w_hat - v) <= 2 ** -11 * abs(v)
            outs.append(w_hat)
    # with G = 64 the widths genuinely differ
    w = rng.standard_normal(64)
    recon = {b: matmul.dequant(np.array([quant.quantize_group(w, b)[0]]),
                               np.array([[quant.quantize_group(w, b)[1]]], dtype=np.uint16))[0]
             for b in (1, 2, 4, 8)}
    errs = [np.linalg.norm(recon[b] - w) for b in (1, 2, 4, 8)]
    assert errs[3] < errs[2] < errs[1]


def test_level_sets():
    assert quant.level_set(1) == [-1, 1]
    assert quant.level_set(2) == [-1, 0, 1]
    assert len(quant.level_set(4)) == 15 and len(quant.level_set(8)) == 255
    for b in (1, 2, 4, 8):
        for v in quant.level_set(b):
            u = quant.offset_code(v, b)
            assert 0 <= u < (1 << b) and quant.level_from_code(u, b) == v
        if b >= 2:
            assert quant.offset_code(-quant.qmax(b), b) == 1   # code 0 is never produced


# ---------------------------------------------------------------- dequant / products

def test_dequant_exact_in_float32():
    rng = np.random.default_rng(17)
    for b in (1, 2, 4, 8):
        q = np.array([rng.choice(quant.level_set(b), 64)])
        s = rng.uniform(0.0001, 60000, 1).astype(np.float16).view(np.uint16).reshape(1, 1)
        w = matmul.dequant(q, s)
        assert np.array_equal(w.astype(np.float32).astype(np.float64), w)


def _fraction_gemv(q, s_bits, x):
    s = matmul.scales_f64(s_bits)
    N, K = q.shape
    y = []
    for n in range(N):
        acc = Fraction(0)
        for k in range(K):
            acc += Fraction(float(s[n, k // 64])) * int(q[n, k]) * Fraction(float(x[k]))
        y.append(acc)
    return y


def test_gemv_against_exact_rational_brute_force():
    rng = np.random.default_rng(19)
    N, K = 5, 128
    bits = rng.choice([1, 2, 4, 8], size=(N, K // 64))
    q = np.zeros((N, K), dtype=np.int64)
    for n in range(N):
        for j in range(K // 64):
            q[n, 64 * j:64 * j + 64] = rng.choice(quant.level_set(int(bits[n, j])), 64)
    s = rng.uniform(0.01, 0.1, (N, K // 64)).astype(np.float16).view(np.uint16)
    x = rng.standard_normal(K).astype(np.float16)
    y = matmul.gemv(q, s, x)
    exact = _fraction_gemv(q, s, x)
    for n in range(N):
        assert abs(Fraction(y[n]) - exact[n]) <= Fraction(1, 10 ** 12) * (abs(exact[n]) + 1)
    X = rng.standard_normal((3, K)).astype(np.float16)
    Y = matmul.gemm(q, s, X)
    for m in range(3):
        ex = _fraction_gemv(q, s, X[m])
        for n in range(N):
            assert abs(Fraction(Y[m, n]) - ex[n]) <= Fraction(1, 10 ** 12) * (abs(ex[n]) + 1)


def test_one_hot_and_ones_closed_forms():
    rng = np.random.default_rng(23)
    N, K = 6, 192
    q = rng.integers(-7, 8, (N, K))
    s = rng.uniform(0.01, 0.1, (N, 3)).astype(np.float16).view(np.uint16)
    W = matmul.dequant(q, s)
    for k in (0, 63, 64, 191):
        e = np.zeros(K, dtype=np.float16)
        e[k] = 1
        assert np.array_equal(matmul.gemv(q, s, e), W[:, k])
    ones = np.ones(K, dtype=np.float16)
    sf = matmul.scales_f64(s)
    rowsum = [sum(sf[n, j] * int(np.sum(q[n, 64 * j:64 * j + 64])) for j in range(3)) for n in range(N)]
    assert np.allclose(matmul.gemv(q, s, ones), rowsum, rtol=0, atol=1e-12)


# ---------------------------------------------------------------- packed layout pins

def _tiny_inputs(fx):
    N, K = fx["N"], fx["K"]
    q = np.zeros((N, K), dtype=np.int64)
    s = np.zeros((N, K // 64), dtype=np.uint16)
    for r in range(N):
        for j in range(K // 64):
            g = fx["groups"][f"r{r}j{j}"]
            qq = [g["default_q"]] * 64
            for k, v in g["q_overrides"].items():
                qq[int(k)] = v
            q[r, 64 * j:64 * j + 64] = qq
            s[r, j] = int(g["s_bits"], 16)
    return q, s, np.array(fx["bits"], dtype=np.uint8)


def test_hand_packed_layout(golden_dir):
    fx = _load(golden_dir, "layout_tiny.json")
    q, s, bits = _tiny_inputs(fx)
    for name, g in fx["groups"].items():
        r, j = int(name[1]), int(name[3])
        u = layout.offset_codes(list(q[r, 64 * j:64 * j + 64]), g["b"])
        assert layout.encode_record(u, g["b"]) == [int(w, 16) for w in g["words"]], name
    blob, info = layout.pack(q, s, bits, fx["R"], fx["C"])
    ex = fx["expected"]
    assert info["section_off"] == ex["section_off"]
    assert info["section_len"] == ex["section_len"]
    assert info["total_bytes"] == ex["total_bytes"] == len(blob)
    off = info["section_off"]
    units = np.frombuffer(blob[off[0]:off[0] + 64].tobytes(), dtype=np.uint32).reshape(2, 8)
    assert units.tolist() == ex["unit_table"]
    wmap = np.frombuffer(blob[off[1]:off[1] + 16].tobytes(), dtype=np.uint64)
    assert [int(w) for w in wmap] == [int(w, 16) for w in ex["wmap"]]
    for c, names in ex["class_order"].items():
        c = int(c)
        b = (1, 2, 4, 8)[c]
        words = np.frombuffer(blob[off[2 + c]:off[2 + c] + info["section_len"][2 + c]].tobytes(), dtype=np.uint32)
        want = sum(([int(w, 16) for w in fx["groups"][n]["words"]] for n in names), [])
        assert [int(w) for w in words] == want
        sc = np.frombuffer(blob[off[6 + c]:off[6 + c] + 2 * len(names)].tobytes(), dtype=np.uint16)
        assert [int(v) for v in sc] == [int(fx["groups"][n]["s_bits"], 16) for n in names]
        assert len(words) == 2 * b * len(names)
    # every byte outside the sections is zero
    mask = np.ones(len(blob), dtype=bool)
    for o, ln in zip(info["section_off"], info["section_len"]):
        mask[o:o + ln] = False
    assert not blob[mask].any()


@pytest.mark.parametrize("N,K,R,C", [(1, 64, 16, 1), (37, 320, 16, 2), (100, 768, 64, 12),
                                     (130, 1024, 32, 5), (64, 4096, 64, 64), (300, 640, 256, 3)])
def test_pack_unpack_roundtrip(N, K, R, C):
    rng = np.random.default_rng(N * 31 + K)
    bits = rng.choice([1, 2, 4, 8], size=(N, K // 64), p=[0.69, 0.15, 0.12, 0.04])
    q = np.zeros((N, K), dtype=np.int64)
    for b in (1, 2, 4, 8):
        sel = np.repeat(bits == b, 64, axis=1)
        q[sel] = rng.choice(quant.level_set(b), int(sel.sum()))
    s = rng.uniform(0.01, 0.1, (N, K // 64)).astype(np.float16).view(np.uint16)
    blob, info = layout.pack(q, s, bits, R, C)
    q2, s2, b2 = layout.unpack(blob, info)
    assert np.array_equal(q2, q) and np.array_equal(s2, s) and np.array_equal(b2, bits)
    assert sum(info["section_len"][2:6]) == layout.code_bytes(bits)
    assert info["section_len"][6:10] == [2 * n for n in info["n_entries"]]
    assert sum(info["n_entries"]) == N * K // 64


def test_record_roundtrip_all_widths():
    rng = np.random.default_rng(29)
    for b in (1, 2, 4, 8):
        for _ in range(50):
            u = list(rng.integers(0, 1 << b, 64))
            assert layout.decode_record(layout.encode_record(u, b), b) == u


# ---------------------------------------------------------------- storage accounting

def test_table1_storage(golden_dir):
    gold = _load(golden_dir, "storage_table1.json")
    for row in gold["rows"]:
        got = storage.packed_bytes(row["params"], row["mean_bits"])
        if row["unit"] == "MB":
            assert abs(got / 1e6 - row["printed"]) <= 1.0, row
        else:
            assert abs(got / 1e9 - row["printed"]) <= 0.01, row
    rh = gold["recipe_head"]
    assert round(storage.mean_bits({int(k): v for k, v in rh["fractions"].items()}), 6) == rh["mean"]


def test_code_bytes_equal_params_times_mean_bits():
    rng = np.random.default_rng(31)
    bits = rng.choice([1, 2, 4, 8], size=(200, 12))
    counts = {b: int(np.sum(bits == b)) for b in (1, 2, 4, 8)}
    params = bits.size * 64
    assert layout.code_bytes(bits) == storage.packed_bytes(params, storage.mean_bits(counts))


# ---------------------------------------------------------------- planted mistakes

@pytest.mark.parametrize("mutation", ["round_half_away", "exact_scale_codes", "sign_zero_negative",
                                      "qmax_pow2", "sum_order_abs_missing"])
def test_pins_catch_planted_mistakes(golden_dir, monkeypatch, mutation):
    """Plant a plausible mistake in the oracle (on the CPU) and check that the
    hand-computed groups no longer pass."""
    if mutation == "round_half_away":
        monkeypatch.setattr(quant, "round_half_even",
                            lambda v: float(np.sign(v) * np.floor(abs(v) + 0.5)))
    elif mutation == "exact_scale_codes":
        monkeypatch.setattr(quant, "fp16_value", lambda bits: _last_exact[0])
    elif mutation == "sign_zero_negative":
        monkeypatch.setattr(quant, "one_bit_sign", lambda v: 1 if v > 0 else -1)
    elif mutation == "qmax_pow2":
        monkeypatch.setattr(quant, "qmax", lambda b: 1 if b == 1 else (1 << (b - 1)))
    elif mutation == "sum_order_abs_missing":
        orig = quant.quantize_group

        def wrong(w, b, **kw):
            if b == 1:
                s = sum(w) / 64
                return [quant.one_bit_sign(v) for v in w], quant.fp16_bits(abs(s))
            return orig(w, b, **kw)
        monkeypatch.setattr(quant, "quantize_group", wrong)
    if mutation == "exact_scale_codes":
        # codes computed against the double scale instead of the stored one
        orig_bits = quant.fp16_bits

        def record(v):
            _last_exact[0] = v
            return orig_bits(v)
        monkeypatch.setattr(quant, "fp16_bits", record)
    with pytest.raises(AssertionError):
        test_hand_computed_groups(golden_dir)


def test_pins_catch_unchecked_one_bit_overflow(monkeypatch):
    """Plant the mistake of returning the fp16 bits of +inf for a 1-bit group
    whose mean |w| overflows (the b >= 2 check alone): the overflow pin fails."""
    orig = quant.quantize_group

    def unchecked(w, b, **kw):
        if b == 1:
            total = 0.0
            for v in w:
                total += abs(float(v))
            return [quant.one_bit_sign(float(v)) for v in w], quant.fp16_bits(total / 64)
        return orig(w, b, **kw)
    monkeypatch.setattr(quant, "quantize_group", unchecked)
    with pytest.raises(BaseException) as err:
        with np.errstate(over="ignore"):
            test_scale_overflow_raises()
    assert "DID NOT RAISE" in str(err.value)


_last_exact = [0.0]
