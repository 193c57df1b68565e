"""GPU parity of the selection path (vbq_qat_forward, vbq_qat_logit_grad) against the oracle.

Bars:
  * candidate reconstructions: exact.  A one-hot pi (logit margins so wide
    that exp underflows to 0 in fp32) makes w_soft one candidate, which must
    equal the oracle's w_hat^(b) value for value, and equal vbq_dequant of
    vbq_pack at the hardened widths;
  * hardened widths: exact (argmax of the same fp32 logits on both sides);
  * pi, w_soft, bbar: the fp32 arithmetic bound below;
  * dL/dlogits of the logit step: the bound derived at _check_grad.

Tolerance (derived from the fp32 arithmetic, u = 2^-24).  The kernel forms
v_k = l_k + e_k, subtracts the group's largest v_m and divides by tau.  With
z_k = v_k/tau and Z = max_k |z_k| for the group: the sums put u|z_k| on each
z, the subtraction adds u|z_k - z_m| and the division u|z_k - z_m|, so the
exponent (z_k - z_m) is off by at most 3u(|z_k| + |z_m|); exp contributes at
most 2u relative plus that absolute error; the normalising sum 3u and the
division u.  So every pi_k is
within eps_g = u(12 Z + 8) relative of the exact value; the tests allow
u(16 Z + 16).  The mix folds pi_k * s_k (one rounding) and adds the four
terms with FMAs (three roundings), so |w_soft - w*| <= (eps_g + 8u) *
sum_k pi_k |w_hat_k|.  Values below the fp32 normal range add an absolute
1e-37 (pi) or 1e-37 * sum_k |w_hat_k| (w_soft).  bbar is a mean of per-group
sums_k pi_k B_k, each within eps_g + 4u, summed in double: relative
max_g eps_g + 8u.
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import qat as oqat  # noqa: E402
from paper_2607_02893_amd import synth  # noqa: E402

pytestmark = pytest.mark.gpu

U = 2.0 ** -24
WIDTHS = np.array([1, 2, 4, 8], dtype=np.float64)


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


def _run(vbq, W, logits, noise, tau, **kw):
    out = vbq.qat_forward(_dev(W), _dev(logits), None if noise is None else _dev(noise), tau, **kw)
    torch.cuda.synchronize()
    return [None if t is None else t.cpu().numpy() for t in out]


def _eps(logits, noise, tau):
    z = (logits.astype(np.float64) + (0.0 if noise is None else noise.astype(np.float64))) / tau
    Z = np.max(np.abs(z), axis=-1)
    return U * (16.0 * Z + 16.0)


def _check_mix(W, logits, noise, tau, got_w, got_pi, got_bbar, what):
    """Compare against the oracle with the derived bound; returns the worst ratio err/bound."""
    n = logits.shape[0]
    ref = oqat.forward(W.reshape(n, 64).astype(np.float64), logits.reshape(n, 1, 4),
                       None if noise is None else noise.reshape(n, 1, 4), tau)
    pi_ref = ref["pi"].reshape(n, 4)
    eps = _eps(logits, noise, tau)
    worst = 0.0
    if got_pi is not None:
        err = np.abs(got_pi.reshape(n, 4).astype(np.float64) - pi_ref)
        bound = eps[:, None] * pi_ref + 1e-37
        bad = err > bound
        assert not bad.any(), f"{what}: pi off at groups {np.nonzero(bad.any(axis=1))[0][:8]}"
        worst = max(worst, float(np.max(err / bound)))
    cand = oqat.candidates(W.reshape(n, 64).astype(np.float64)).reshape(4, n, 64)
    A = np.einsum("gk,kgi->gi", pi_ref, np.abs(cand))
    B = np.abs(cand).sum(axis=0)
    err = np.abs(got_w.reshape(n, 64).astype(np.float64) - ref["w_soft"].reshape(n, 64))
    bound = (eps[:, None] + 8 * U) * A + 1e-37 * B
    bad = err > bound
    assert not bad.any(), f"{what}: w_soft off at groups {np.nonzero(bad.any(axis=1))[0][:8]}"
    worst = max(worst, float(np.max(np.where(bound > 0, err / np.maximum(bound, 1e-300), 0.0))))
    if got_bbar is not None:
        tol = (float(eps.max()) + 8 * U) * ref["bbar"]
        assert abs(float(got_bbar[0]) - ref["bbar"]) <= tol, f"{what}: bbar {got_bbar[0]} vs {ref['bbar']}"
    return ref


SIZES = [1, 63, 64, 65, 1000, 4097, 2 * 64 * 2048 + 77]


@pytest.mark.parametrize("tau", [5.0, 0.5])
@pytest.mark.parametrize("n", SIZES)
def test_forward_matches_oracle(vbq, n, tau):
    _say(f"qat forward n_groups={n} tau={tau}")
    W, logits, noise = synth.selection_inputs(n, part=n)
    w_soft, pi, hard, bbar = _run(vbq, W, logits, noise, tau)
    ref = _check_mix(W, logits, noise, tau, w_soft, pi, bbar, f"n={n} tau={tau}")
    np.testing.assert_array_equal(hard, ref["hard_bits"].reshape(n))


def test_golden_group(vbq, golden_dir):
    import json
    import os
    with open(os.path.join(golden_dir, "qat_group.json")) as f:
        g = json.load(f)
    W = np.zeros(64, dtype=np.float32)
    W[: len(g["w_head"])] = g["w_head"]
    mix = g["mix"]
    noise = np.asarray(mix["noise"], dtype=np.float32).reshape(1, 4)
    logits = (2.0 * np.log([1.0, 2.0, 3.0, 4.0]) - np.asarray(mix["noise"])).astype(np.float32).reshape(1, 4)
    w_soft, pi, hard, bbar = _run(vbq, W, logits, noise, mix["tau"])
    # fp32 logits: pi is (0.1, 0.2, 0.3, 0.4) to about 1e-7
    np.testing.assert_allclose(pi[0], mix["pi"], rtol=2e-6)
    want = np.full(64, mix["w_soft_tail"])
    want[: len(mix["w_soft_head"])] = mix["w_soft_head"]
    np.testing.assert_allclose(w_soft, want, rtol=2e-6, atol=1e-7)
    assert abs(float(bbar[0]) - mix["bbar"]) < 1e-5
    assert int(hard[0]) == mix["hard_bits"]


def _one_hot_logits(widx):
    l = np.full((widx.size, 4), -1.0e4, dtype=np.float32)
    l[np.arange(widx.size), widx] = 0.0
    return l


def _check_one_hot(vbq, W, widx, what, noise=None):
    n = widx.size
    logits = _one_hot_logits(widx)
    w_soft, pi, hard, bbar = _run(vbq, W, logits, noise, 0.5)
    np.testing.assert_array_equal(pi, np.eye(4, dtype=np.float32)[widx])
    cand = oqat.candidates(W.reshape(n, 64).astype(np.float64)).reshape(4, n, 64)
    want = cand[widx, np.arange(n)]
    got = w_soft.reshape(n, 64).astype(np.float64)
    bad = got != want
    assert not bad.any(), f"{what}: {int(bad.sum())} weights differ, first at group {np.nonzero(bad.any(axis=1))[0][0]}"
    np.testing.assert_array_equal(hard, WIDTHS[widx].astype(np.uint8))
    assert float(bbar[0]) == pytest.approx(WIDTHS[widx].mean(), rel=1e-12)
    return w_soft, hard


@pytest.mark.parametrize("n", [1, 64, 3000, 64 * 2048 + 5])
def test_one_hot_candidates_exact(vbq, n):
    _say(f"qat one-hot n_groups={n}")
    W, _, _ = synth.selection_inputs(n, part=10_000 + n)
    widx = synth.rng_for(synth.SELECTION_SEED, 3001, n).integers(0, 4, size=n)
    _check_one_hot(vbq, W, widx, f"one-hot n={n}")


def test_one_hot_matches_packed_weights(vbq):
    # the deployed path: vbq_pack at the hardened widths, then vbq_dequant
    N, K = 96, 1024
    W, _, _ = synth.selection_inputs(N * K // 64, part=20_000)
    widx = synth.rng_for(synth.SELECTION_SEED, 3002).integers(0, 4, size=N * K // 64)
    w_soft, hard = _check_one_hot(vbq, W, widx, "one-hot vs pack")
    blob, d = vbq.pack(W.reshape(N, K), hard.reshape(N, K // 64))
    deq = vbq.PackedMatrix(blob, d).dequant().cpu().numpy()
    assert np.array_equal(deq, w_soft.reshape(N, K))


def _tie_groups():
    """Groups whose weights sit exactly on, or one float32 ulp either side of,
    the rounding midpoints (q + 1/2) * s of the 2-, 4- and 8-bit candidates."""
    groups = []
    for m in (1.0, 0.3, 7.0, 1.0e-3, 3.0e-6, 6.0e4):
        s = {b: float(np.float16(m / q)) for b, q in ((2, 1), (4, 7), (8, 127))}
        for b in (2, 4, 8):
            qm = {2: 1, 4: 7, 8: 127}[b]
            ks = np.arange(-qm, qm)  # midpoints between k and k + 1
            mids = ((ks + 0.5) * s[b]).astype(np.float32)
            pts = np.concatenate([mids, np.nextafter(mids, np.float32(np.inf)), np.nextafter(mids, np.float32(-np.inf))])
            pts = pts[np.abs(pts) < m]
            for i in range(0, len(pts), 63):
                g = np.zeros(64, dtype=np.float32)
                chunk = pts[i:i + 63]
                g[: len(chunk)] = chunk
                g[63] = np.float32(m) if i % 2 == 0 else -np.float32(m)
                groups.append(g)
    return np.stack(groups)


@pytest.mark.parametrize("width_index", [0, 1, 2, 3])
def test_rounding_ties_exact(vbq, width_index):
    G = _tie_groups()
    _say(f"qat ties: {G.shape[0]} groups at width {int(WIDTHS[width_index])}")
    widx = np.full(G.shape[0], width_index)
    _check_one_hot(vbq, G.reshape(-1), widx, f"ties width {int(WIDTHS[width_index])}")


def test_edge_groups_exact(vbq):
    rows = [np.zeros(64, dtype=np.float32),                              # all zero
            np.full(64, -0.0, dtype=np.float32),                         # negative zeros
            np.where(np.arange(64) % 2 == 0, 1e-9, -1e-9).astype(np.float32),  # scales underflow fp16
            np.where(np.arange(64) % 3 == 0, 3e-7, -2e-7).astype(np.float32),  # subnormal fp16 scales
            np.linspace(-6.0e4, 6.0e4, 64, dtype=np.float32),            # near the top of fp16
            np.full(64, 0.25, dtype=np.float32),                         # one repeated value
            np.array([1.0] + [0.0] * 63, dtype=np.float32)]              # one non-zero weight
    G = np.stack(rows)
    for k in range(4):
        _check_one_hot(vbq, G.reshape(-1), np.full(G.shape[0], k), f"edge groups width {int(WIDTHS[k])}")


def test_optional_outputs_and_no_noise(vbq):
    n = 777
    W, logits, noise = synth.selection_inputs(n, part=30_000)
    full = _run(vbq, W, logits, None, 1.3)
    _check_mix(W, logits, None, 1.3, full[0], full[1], full[3], "no noise")
    only = _run(vbq, W, logits, None, 1.3, pi=False, hard_bits=False, bbar=False)
    assert only[1] is None and only[2] is None and only[3] is None
    assert np.array_equal(only[0], full[0])


def test_bitwise_repeatable(vbq):
    n = 64 * 2048 + 999
    W, logits, noise = synth.selection_inputs(n, part=40_000)
    a = _run(vbq, W, logits, noise, 0.7)
    b = _run(vbq, W, logits, noise, 0.7)
    for x, y in zip(a, b):
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8))


def test_empty_and_errors(vbq):
    W = torch.zeros(64, dtype=torch.float32, device="cuda")
    l = torch.zeros(4, dtype=torch.float32, device="cuda")
    out = vbq.qat_forward(W[:0], l[:0], None, 1.0)
    torch.cuda.synchronize()
    assert out[0].numel() == 0
    with pytest.raises(vbq.VbqError):
        vbq.qat_forward(W, l, None, 0.0)
    with pytest.raises(vbq.VbqError):
        vbq.qat_forward(W, l, None, float("nan"))


def test_training_step_full_size(vbq):
    # the 131M-class model's linear weights end to end, one launch
    name, mats, n = synth.selection_workload(1)
    _say(f"qat full size: {name} {n} groups")
    W, logits, noise = synth.selection_inputs(n, part=1)
    tau = 0.5
    w_soft, pi, hard, bbar = _run(vbq, W, logits, noise, tau)
    # hardened widths and bbar over every group (pi from the oracle's softmax)
    np.testing.assert_array_equal(hard, oqat.harden(logits.reshape(n, 1, 4)).reshape(n))
    pi_ref = oqat.gumbel_softmax(logits, noise, tau)
    eps = _eps(logits, noise, tau)
    assert np.all(np.abs(pi.astype(np.float64) - pi_ref) <= eps[:, None] * pi_ref + 1e-37)
    bbar_ref = float(np.sum(pi_ref * WIDTHS) / n)
    assert abs(float(bbar[0]) - bbar_ref) <= (float(eps.max()) + 8 * U) * bbar_ref
    # w_soft on sampled groups: first, last, every matrix boundary, and random ones
    bounds = np.cumsum([0] + [N * K // 64 for _, N, K in mats])
    rng = synth.rng_for(synth.SELECTION_SEED, 3003)
    idx = np.unique(np.concatenate([[0, n - 1], bounds[:-1], bounds[1:] - 1, rng.integers(0, n, size=4000)]))
    Wg = W.reshape(n, 64)[idx]
    _check_mix(Wg.reshape(-1), logits[idx], noise[idx], tau, w_soft.reshape(n, 64)[idx], pi[idx], None,
               "full size sampled")


# ------------------------------------------------------------------ logit step

def _grad_inputs(n, part, tau):
    """Weights, dL/dw_soft and pi for the logit step.  pi is the oracle's softmax
    of the seeded logits and noise, rounded to float32 (no input comes from the
    kernels)."""
    W, logits, noise = synth.selection_inputs(n, part=part)
    G = synth.rng_for(synth.SELECTION_SEED, 3004, part).standard_normal(n * 64, dtype=np.float32)
    pi = oqat.gumbel_softmax(logits, noise, tau).astype(np.float32)
    return W, G, pi


def _check_grad(W, G, pi, tau, lam, n_bbar, got, what):
    """Bound (fp32, u = 2^-24): each a_k is a 64-term FMA sum scaled once and
    offset once, within 67u (sum_i |G_i w_hat_k,i| + |lambda| B_k / n); the
    pi-weighted mean, the difference and the scaling by pi_k / tau add a few u
    of the same magnitudes.  Allowed: (pi_k / tau) * 96u * (A_k + sum_j pi_j A_j)."""
    n = pi.shape[0]
    Wg = W.reshape(n, 64).astype(np.float64)
    want = oqat.logit_grad(Wg, G.reshape(n, 64), pi.reshape(n, 1, 4), tau, lam, n_groups=n_bbar).reshape(n, 4)
    cand = oqat.candidates(Wg).reshape(4, n, 64)
    A = np.einsum("gi,kgi->gk", np.abs(G.reshape(n, 64).astype(np.float64)), np.abs(cand)) + abs(lam) * WIDTHS / n_bbar
    p = pi.astype(np.float64)
    bound = p / tau * 96 * U * (A + np.sum(p * A, axis=-1, keepdims=True)) + 1e-37
    err = np.abs(got.reshape(n, 4).astype(np.float64) - want)
    bad = err > bound
    assert not bad.any(), f"{what}: dlogits off at groups {np.nonzero(bad.any(axis=1))[0][:8]}"


@pytest.mark.parametrize("lam", [0.0, 2.5])
@pytest.mark.parametrize("tau", [5.0, 0.5])
@pytest.mark.parametrize("n", [1, 65, 4097, 2 * 64 * 2048 + 77])
def test_logit_grad_matches_oracle(vbq, n, tau, lam):
    _say(f"qat logit grad n_groups={n} tau={tau} lambda={lam}")
    W, G, pi = _grad_inputs(n, 50_000 + n, tau)
    d = vbq.qat_logit_grad(_dev(W), _dev(G), _dev(pi), tau, lam)
    torch.cuda.synchronize()
    _check_grad(W, G, pi, tau, lam, n, d.cpu().numpy(), f"n={n} tau={tau} lambda={lam}")


def test_logit_grad_golden(vbq, golden_dir):
    import json
    import os
    with open(os.path.join(golden_dir, "qat_group.json")) as f:
        g = json.load(f)
    W = np.zeros(64, dtype=np.float32)
    W[: len(g["w_head"])] = g["w_head"]
    G = np.zeros(64, dtype=np.float32)
    G[0] = g["logit_grad"]["grad_entry0"]
    pi = np.asarray(g["mix"]["pi"], dtype=np.float32).reshape(1, 4)
    d = vbq.qat_logit_grad(_dev(W), _dev(G), _dev(pi), g["mix"]["tau"], g["logit_grad"]["lambda"]).cpu().numpy()
    # pi = (0.1, 0.2, 0.3, 0.4) rounded to float32: agreement to about 1e-7
    np.testing.assert_allclose(d[0], g["logit_grad"]["dlogits"], rtol=1e-6, atol=1e-7)


def test_logit_grad_rows_sum_to_zero_and_network_n(vbq):
    # softmax gradient: each group's dlogits sum to 0; n_bbar only scales the penalty
    n = 3000
    W, G, pi = _grad_inputs(n, 60_000, 1.0)
    d_local = vbq.qat_logit_grad(_dev(W), _dev(G), _dev(pi), 1.0, 3.0).cpu().numpy()
    d_net = vbq.qat_logit_grad(_dev(W), _dev(G), _dev(pi), 1.0, 3.0, n_bbar=10 * n).cpu().numpy()
    _check_grad(W, G, pi, 1.0, 3.0, 10 * n, d_net, "network n")
    # sum_k dlogits_k = (1/tau)(sum_k pi_k a_k - mean * sum_k pi_k): zero up to the
    # rounding of the a_k, which scales with their magnitudes A_k (not with |dlogits|)
    Wg = W.reshape(n, 64).astype(np.float64)
    cand = oqat.candidates(Wg).reshape(4, n, 64)
    A = np.einsum("gi,kgi->gk", np.abs(G.reshape(n, 64).astype(np.float64)), np.abs(cand)) + 3.0 * WIDTHS / n
    p = pi.astype(np.float64)
    assert np.all(np.abs(d_local.astype(np.float64).sum(axis=1)) <= 2 * 96 * U * np.sum(p * A, axis=1) + 1e-37)
    assert not np.array_equal(d_local, d_net)


def test_logit_grad_full_size(vbq):
    name, mats, n = synth.selection_workload(1)
    _say(f"qat logit grad full size: {name} {n} groups")
    tau, lam = 0.5, 0.05
    W, G, pi = _grad_inputs(n, 2, tau)
    d = vbq.qat_logit_grad(_dev(W), _dev(G), _dev(pi), tau, lam).cpu().numpy()
    rng = synth.rng_for(synth.SELECTION_SEED, 3005)
    bounds = np.cumsum([0] + [N * K // 64 for _, N, K in mats])
    idx = np.unique(np.concatenate([[0, n - 1], bounds[:-1], bounds[1:] - 1, rng.integers(0, n, size=4000)]))
    Wg = W.reshape(n, 64)[idx].reshape(-1)
    Gg = G.reshape(n, 64)[idx].reshape(-1)
    _check_grad(Wg, Gg, pi[idx], tau, lam, n, d[idx], "full size sampled")
    assert np.all(np.isfinite(d))


# ------------------------------------------------------------ beyond 4 GiB

BIG = (1 << 24) + (1 << 20) + 37  # 1.14G weights: every fp32 weight array passes the 4 GiB mark


def _big_sample(n):
    """Groups to check at full size: both sides of the 4 GiB byte offset, the ragged tail,
    and random ones."""
    edge = (1 << 32) // 256  # first group whose weights start at byte 2^32
    rng = synth.rng_for(synth.SELECTION_SEED, 3006)
    idx = np.concatenate([np.arange(edge - 70, edge + 70), np.arange(n - 100, n), rng.integers(0, n, size=3000)])
    return np.unique(idx[(idx >= 0) & (idx < n)])


def test_forward_beyond_4gib(vbq):
    _say(f"qat forward n_groups={BIG} ({BIG * 256 / 2**30:.2f} GiB of weights)")
    W, logits, noise = synth.selection_inputs(BIG, part=70_000)
    tau = 0.7
    w_soft, pi, hard, bbar = _run(vbq, W, logits, noise, tau)
    idx = _big_sample(BIG)
    _check_mix(W.reshape(BIG, 64)[idx].reshape(-1), logits[idx], noise[idx], tau, w_soft.reshape(BIG, 64)[idx],
               pi[idx], None, "beyond 4 GiB sampled")
    np.testing.assert_array_equal(hard, oqat.harden(logits.reshape(BIG, 1, 4)).reshape(BIG))
    pi_ref = oqat.gumbel_softmax(logits, noise, tau)
    bbar_ref = float(np.sum(pi_ref * WIDTHS) / BIG)
    assert abs(float(bbar[0]) - bbar_ref) <= (float(_eps(logits, noise, tau).max()) + 8 * U) * bbar_ref


def test_logit_grad_beyond_4gib(vbq):
    _say(f"qat logit grad n_groups={BIG}")
    tau, lam = 0.7, 0.01
    W, G, pi = _grad_inputs(BIG, 71_000, tau)
    d = vbq.qat_logit_grad(_dev(W), _dev(G), _dev(pi), tau, lam).cpu().numpy()
    idx = _big_sample(BIG)
    _check_grad(W.reshape(BIG, 64)[idx].reshape(-1), G.reshape(BIG, 64)[idx].reshape(-1), pi[idx], tau, lam, BIG,
                d[idx], "beyond 4 GiB sampled")
    assert np.all(np.isfinite(d))


# ------------------------------------------------------------- bf16 w_soft

@pytest.mark.parametrize("n", [1, 65, 4097, 2 * 64 * 2048 + 77])
def test_bf16_w_soft_is_the_rounded_fp32_result(vbq, n):
    # the bf16 output is the fp32 result rounded to nearest even (torch's CPU conversion
    # is the reference rounding), and so within the fp32 bound plus half a bf16 ulp
    _say(f"qat forward bf16 n_groups={n}")
    W, logits, noise = synth.selection_inputs(n, part=80_000 + n)
    tau = 0.5
    w32 = _run(vbq, W, logits, noise, tau)[0]
    out = vbq.qat_forward(_dev(W), _dev(logits), _dev(noise), tau, w_soft_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    w16 = out[0]
    assert w16.dtype == torch.bfloat16
    want = torch.from_numpy(w32).to(torch.bfloat16)
    assert torch.equal(w16.cpu().view(torch.int16), want.view(torch.int16))
    ref = oqat.forward(W.reshape(n, 64).astype(np.float64), logits.reshape(n, 1, 4), noise.reshape(n, 1, 4), tau)
    cand = oqat.candidates(W.reshape(n, 64).astype(np.float64)).reshape(4, n, 64)
    A = np.einsum("gk,kgi->gi", ref["pi"].reshape(n, 4), np.abs(cand))
    eps = _eps(logits, noise, tau)
    got = w16.float().cpu().numpy().reshape(n, 64).astype(np.float64)
    exact = ref["w_soft"].reshape(n, 64)
    bound = (eps[:, None] + 8 * U) * A * (1 + 2.0 ** -8) + 2.0 ** -8 * np.abs(exact) + 1e-37 * cand.__abs__().sum(0)
    assert np.all(np.abs(got - exact) <= bound)


def test_bf16_one_hot_is_the_rounded_candidate(vbq):
    n = 5000
    W, _, _ = synth.selection_inputs(n, part=90_000)
    widx = synth.rng_for(synth.SELECTION_SEED, 3007).integers(0, 4, size=n)
    out = vbq.qat_forward(_dev(W), _dev(_one_hot_logits(widx)), None, 0.5, w_soft_dtype=torch.bfloat16, pi=False,
                          hard_bits=False, bbar=False)
    cand = oqat.candidates(W.reshape(n, 64).astype(np.float64)).reshape(4, n, 64)[widx, np.arange(n)]
    want = torch.from_numpy(cand.astype(np.float32)).to(torch.bfloat16)  # exact in fp32, then rounded once
    # values compared (a zero candidate of a negative weight may come out as -0.0)
    assert torch.equal(out[0].cpu().reshape(n, 64), want)


@pytest.mark.parametrize("tau", [1.17549435e-38, 1e-30])
def test_tiny_tau_is_one_hot_on_the_noisy_argmax(vbq, tau):
    # the largest l + e is subtracted before dividing by tau: no inf - inf, pi is exactly
    # one-hot on argmax(l + e) (every other exponent underflows), as in the oracle
    n = 4096 + 3
    W, logits, noise = synth.selection_inputs(n, part=100_000)
    w_soft, pi, hard, bbar = _run(vbq, W, logits, noise, tau)
    ref = oqat.forward(W.reshape(n, 64).astype(np.float64), logits.reshape(n, 1, 4), noise.reshape(n, 1, 4), tau)
    k = np.argmax(logits.astype(np.float32) + noise.astype(np.float32), axis=1)
    np.testing.assert_array_equal(pi, np.eye(4, dtype=np.float32)[k])
    np.testing.assert_array_equal(ref["pi"].reshape(n, 4), np.eye(4)[k])
    cand = oqat.candidates(W.reshape(n, 64).astype(np.float64)).reshape(4, n, 64)
    assert np.array_equal(w_soft.reshape(n, 64).astype(np.float64), cand[k, np.arange(n)])
    assert float(bbar[0]) == pytest.approx(WIDTHS[k].mean(), rel=1e-12)
