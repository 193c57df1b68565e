"""CPU pins of the selection-path oracle (paper section 3.2, section 3.3, Algorithm 1).

Each test checks ``oracle.qat`` against something other than itself: a group
computed by hand at all four widths (tests/golden/qat_group.json), closed
forms of the softmax, the convex-combination and shift invariances, the
tau -> 0 limit, and central finite differences of the scalar objective for the
logit gradient.  The mutation tests at the end plant plausible mistakes in the
oracle and check that one of these pins catches each.
"""

import json
import os

import numpy as np
import pytest

from oracle import qat, quant


def _golden(golden_dir):
    with open(os.path.join(golden_dir, "qat_group.json")) as f:
        return json.load(f)


def _golden_inputs(g):
    w = np.zeros((1, 64))
    w[0, : len(g["w_head"])] = g["w_head"]
    mix = g["mix"]
    noise = np.asarray(mix["noise"], dtype=np.float64).reshape(1, 1, 4)
    logits = (2.0 * np.log([1.0, 2.0, 3.0, 4.0])).reshape(1, 1, 4) - noise
    return w, logits, noise, mix["tau"]


def _expand(head, tail):
    out = np.full(64, float(tail))
    out[: len(head)] = head
    return out


# ------------------------------------------------------------- hand-computed group

def test_golden_candidates(golden_dir):
    g = _golden(golden_dir)
    w, _, _, _ = _golden_inputs(g)
    cand = qat.candidates(w)
    for k, b in enumerate((1, 2, 4, 8)):  # the candidate order of section 3.2
        c = g["candidates"][str(b)]
        np.testing.assert_array_equal(cand[k, 0], _expand(c["w_hat_head"], c["w_hat_tail"]))


def test_golden_mix(golden_dir):
    g = _golden(golden_dir)
    w, logits, noise, tau = _golden_inputs(g)
    out = qat.forward(w, logits, noise, tau)
    mix = g["mix"]
    np.testing.assert_allclose(out["pi"][0, 0], mix["pi"], rtol=1e-12)
    np.testing.assert_allclose(out["w_soft"][0], _expand(mix["w_soft_head"], mix["w_soft_tail"]),
                               rtol=1e-12, atol=1e-15)
    assert out["bbar"] == pytest.approx(mix["bbar"], rel=1e-12)
    assert int(out["hard_bits"][0, 0]) == mix["hard_bits"]


def test_golden_logit_grad(golden_dir):
    g = _golden(golden_dir)
    w, logits, noise, tau = _golden_inputs(g)
    pi = qat.forward(w, logits, noise, tau)["pi"]
    G = np.zeros((1, 64))
    G[0, 0] = g["logit_grad"]["grad_entry0"]
    d = qat.logit_grad(w, G, pi, tau, g["logit_grad"]["lambda"])
    np.testing.assert_allclose(d[0, 0], g["logit_grad"]["dlogits"], rtol=1e-11, atol=1e-15)


# ------------------------------------------------------------- softmax closed forms

def test_uniform_logits_give_uniform_pi_and_mean_width():
    rng = np.random.default_rng(1)
    W = rng.standard_normal((3, 128))
    logits = np.zeros((3, 2, 4))
    out = qat.forward(W, logits, None, 0.7)
    np.testing.assert_array_equal(out["pi"], np.full((3, 2, 4), 0.25))
    assert out["bbar"] == 3.75  # (1 + 2 + 4 + 8) / 4
    cand = qat.candidates(W)
    np.testing.assert_allclose(out["w_soft"], cand.mean(axis=0), rtol=1e-15, atol=1e-300)


def test_single_raised_logit_closed_form():
    # l = (0, 0, 0, ln 3), tau = 1: pi = (1, 1, 1, 3)/6.
    W = np.random.default_rng(2).standard_normal((1, 64))
    logits = np.array([0.0, 0.0, 0.0, np.log(3.0)]).reshape(1, 1, 4)
    out = qat.forward(W, logits, None, 1.0)
    np.testing.assert_allclose(out["pi"][0, 0], [1 / 6, 1 / 6, 1 / 6, 1 / 2], rtol=1e-14)
    # tau = 2 halves the log-odds: pi = (1, 1, 1, sqrt 3)/(3 + sqrt 3).
    out2 = qat.forward(W, logits, None, 2.0)
    r3 = np.sqrt(3.0)
    np.testing.assert_allclose(out2["pi"][0, 0], np.array([1, 1, 1, r3]) / (3 + r3), rtol=1e-14)


def test_noise_is_added_to_logits():
    # softmax((l + e)/tau) depends on l + e only: moving mass from l to e changes nothing.
    rng = np.random.default_rng(3)
    W = rng.standard_normal((2, 192))
    l = rng.standard_normal((2, 3, 4))
    e = rng.gumbel(size=(2, 3, 4))
    a = qat.forward(W, l, e, 0.9)
    b = qat.forward(W, l + e, None, 0.9)
    np.testing.assert_allclose(a["pi"], b["pi"], rtol=1e-14)
    np.testing.assert_allclose(a["w_soft"], b["w_soft"], rtol=1e-13, atol=1e-300)
    # ... but the hardened widths read l alone.
    np.testing.assert_array_equal(a["hard_bits"], qat.harden(l))


def test_shift_invariance():
    rng = np.random.default_rng(4)
    W = rng.standard_normal((2, 128))
    l = rng.standard_normal((2, 2, 4))
    a = qat.forward(W, l, None, 0.5)
    b = qat.forward(W, l + 17.25, None, 0.5)
    np.testing.assert_allclose(a["pi"], b["pi"], rtol=1e-13)


# ------------------------------------------------------------------ invariants

def test_convex_combination_bounds_and_pi_simplex():
    rng = np.random.default_rng(5)
    W = (rng.standard_normal((6, 320)) * rng.uniform(0.01, 3, size=(6, 1)))
    l = rng.standard_normal((6, 5, 4)) * 2
    e = rng.gumbel(size=(6, 5, 4))
    out = qat.forward(W, l, e, 0.8)
    pi = out["pi"]
    assert np.all(pi >= 0) and np.allclose(pi.sum(axis=-1), 1.0, rtol=0, atol=1e-15)
    cand = qat.candidates(W)
    lo, hi = cand.min(axis=0), cand.max(axis=0)
    slack = 1e-15 * np.abs(cand).max(axis=0)
    assert np.all(out["w_soft"] >= lo - slack) and np.all(out["w_soft"] <= hi + slack)
    eb = (pi * np.array([1, 2, 4, 8])).sum(axis=-1)
    assert np.all(eb >= 1) and np.all(eb <= 8)
    assert out["bbar"] == pytest.approx(eb.mean(), rel=1e-14)


def test_low_temperature_limit_is_one_hot_on_noisy_argmax():
    # tau -> 0: pi concentrates on argmax (l + e), and w_soft is that candidate exactly.
    rng = np.random.default_rng(6)
    W = rng.standard_normal((4, 256))
    z = rng.permutation(np.tile(np.array([0.0, 3.0, 6.0, 9.0]), (4 * 4, 1)).T).T.reshape(4, 4, 4)
    l = z - 1.0
    e = np.ones_like(z)
    out = qat.forward(W, l, e, 1e-3)
    k = np.argmax(z, axis=-1)
    np.testing.assert_array_equal(out["pi"], np.eye(4)[k])
    cand = qat.candidates(W).reshape(4, 4, 4, 64)
    want = np.take_along_axis(cand, k[None, :, :, None], axis=0)[0].reshape(4, 256)
    np.testing.assert_array_equal(out["w_soft"], want)
    assert out["bbar"] == pytest.approx(np.array([1, 2, 4, 8])[k].mean(), rel=1e-15)


def test_harden_first_maximum():
    l = np.array([[[1.0, 3.0, 3.0, 2.0], [5.0, 5.0, 5.0, 5.0], [-1.0, -2.0, -3.0, -0.5]]])
    np.testing.assert_array_equal(qat.harden(l), [[2, 1, 8]])


def test_candidates_match_a_uniform_width_pack():
    # A one-width bit map through the packing quantizer gives the same reconstructions.
    rng = np.random.default_rng(7)
    W = rng.standard_normal((5, 192)).astype(np.float32).astype(np.float64)
    cand = qat.candidates(W)
    for k, b in enumerate(qat.CANDIDATES):
        q, s16 = quant.quantize(W, np.full((5, 3), b, dtype=np.uint8))
        s = s16.view(np.float16).astype(np.float64)
        for n in range(5):
            for j in range(3):
                want = [qi * s[n, j] for qi in q[n, 64 * j:64 * j + 64]]
                assert list(cand[k, n, 64 * j:64 * j + 64]) == want


# ------------------------------------------------------------- logit gradient

def _objective(W, G, l, e, tau, lam):
    out = qat.forward(W, l, e, tau)
    return float(np.sum(G * out["w_soft"])) + lam * out["bbar"]


def test_logit_grad_matches_central_differences():
    rng = np.random.default_rng(8)
    W = rng.standard_normal((3, 192))
    G = rng.standard_normal((3, 192))
    l = rng.standard_normal((3, 3, 4))
    e = rng.gumbel(size=(3, 3, 4))
    tau, lam = 0.7, 2.5
    pi = qat.forward(W, l, e, tau)["pi"]
    d = qat.logit_grad(W, G, pi, tau, lam)
    h = 1e-6
    fd = np.zeros_like(l)
    for idx in np.ndindex(*l.shape):
        lp, lm = l.copy(), l.copy()
        lp[idx] += h
        lm[idx] -= h
        fd[idx] = (_objective(W, G, lp, e, tau, lam) - _objective(W, G, lm, e, tau, lam)) / (2 * h)
    np.testing.assert_allclose(d, fd, rtol=1e-6, atol=1e-8)
    np.testing.assert_allclose(d.sum(axis=-1), 0.0, atol=1e-12)


def test_logit_grad_without_cross_entropy_is_the_penalty_gradient():
    """With G = 0 (the reading of section 3.3 (i) in which cross-entropy does
    not reach the logits) the gradient is that of lambda * bbar alone, in closed
    form: d(lambda bbar)/dl_k = (lambda / n) (pi_k / tau) (B_k - sum_j pi_j B_j)."""
    rng = np.random.default_rng(21)
    W = rng.standard_normal((2, 256))
    l = rng.standard_normal((2, 4, 4))
    e = rng.gumbel(size=(2, 4, 4))
    tau, lam, n = 0.9, 3.0, 8
    pi = qat.forward(W, l, e, tau)["pi"]
    d = qat.logit_grad(W, np.zeros_like(W), pi, tau, lam, n_groups=n)
    B = np.array([1.0, 2.0, 4.0, 8.0])
    expect = (lam / n) * (pi / tau) * (B - np.sum(pi * B, axis=-1, keepdims=True))
    np.testing.assert_allclose(d, expect, rtol=1e-13, atol=1e-15)


# ------------------------------------------------------------------ mutations

def _mutant_softmax_times_tau(logits, noise, tau):
    z = (np.asarray(logits, dtype=np.float64) + np.asarray(noise, dtype=np.float64)) * float(tau)
    z = z - np.max(z, axis=-1, keepdims=True)
    p = np.exp(z)
    return p / np.sum(p, axis=-1, keepdims=True)


def _mutant_softmax_noise_subtracted(logits, noise, tau):
    z = (np.asarray(logits, dtype=np.float64) - np.asarray(noise, dtype=np.float64)) / float(tau)
    z = z - np.max(z, axis=-1, keepdims=True)
    p = np.exp(z)
    return p / np.sum(p, axis=-1, keepdims=True)


@pytest.mark.parametrize("name,attr,mutant", [
    ("tau multiplies", "gumbel_softmax", _mutant_softmax_times_tau),
    ("noise subtracted", "gumbel_softmax", _mutant_softmax_noise_subtracted),
])
def test_golden_catches_planted_mistakes(golden_dir, monkeypatch, name, attr, mutant):
    monkeypatch.setattr(qat, attr, mutant)
    with pytest.raises(AssertionError):
        test_golden_mix(golden_dir)


def test_golden_catches_swapped_candidate_order(golden_dir, monkeypatch):
    monkeypatch.setattr(qat, "CANDIDATES", (1, 2, 8, 4))
    with pytest.raises(AssertionError):
        test_golden_candidates(golden_dir)
    with pytest.raises(AssertionError):
        test_golden_mix(golden_dir)


def test_golden_catches_hardening_on_the_noisy_sample(golden_dir, monkeypatch):
    real_forward = qat.forward

    def mutant(W, logits, noise, tau):
        out = real_forward(W, logits, noise, tau)
        out["hard_bits"] = qat.harden(np.asarray(logits) + np.asarray(noise))
        return out
    monkeypatch.setattr(qat, "forward", mutant)
    with pytest.raises(AssertionError):
        test_golden_mix(golden_dir)


def test_golden_catches_dropped_mean_subtraction(golden_dir, monkeypatch):
    def mutant(W, grad_w_soft, pi, tau, lam, n_groups=None):
        W = np.asarray(W, dtype=np.float64)
        N, K = W.shape
        cand = qat.candidates(W).reshape(4, N, K // 64, 64)
        Gr = np.asarray(grad_w_soft, dtype=np.float64).reshape(N, K // 64, 64)
        a = np.stack([np.sum(Gr * cand[k], axis=-1) + lam * b / (N * K // 64)
                      for k, b in enumerate(qat.CANDIDATES)], axis=-1)
        return pi / tau * a
    monkeypatch.setattr(qat, "logit_grad", mutant)
    with pytest.raises(AssertionError):
        test_golden_logit_grad(golden_dir)
