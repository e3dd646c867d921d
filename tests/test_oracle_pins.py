"""Pins of the CPU oracle against hand-derived cases, closed forms, invariants
and an independent bfloat16 conversion.  CPU only."""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle as O

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "hand_2x2.json")))


def A(x):
    return np.asarray(x, np.float64)


# ------------------------------------------------------------ hand cases

def test_hand_linear_backward():
    c = GOLD["linear_backward"]
    x, W, b, dY = A(c["x"]), A(c["W"]), A(c["b"]), A(c["dY"])
    assert np.array_equal(O.linear_fwd(x, W, b), A(c["y"]))
    dW, db, dX = O.linear_bwd(dY, x, W)
    assert np.array_equal(dW, A(c["dW"]))
    assert np.array_equal(db, A(c["db"]))
    assert np.array_equal(dX, A(c["dX"]))


def test_hand_sgd_momentum_then_mix():
    c = GOLD["sgd_momentum_then_mix"]
    p1, m1 = O.sgd_momentum(A(c["p"]), A(c["g"]), A(c["m0"]), c["lr"], c["momentum"],
                            c["weight_decay"])
    assert np.array_equal(m1, A(c["m1"]))
    assert np.array_equal(p1, A(c["p_local"]))
    assert np.array_equal(O.mix(p1, A(c["q"]), c["alpha"]), A(c["p_mixed"]))
    hp = dict(optim="sgd", lr=c["lr"], momentum=c["momentum"], weight_decay=0.0)
    p2, m2, v2, dis = O.update_mix(A(c["p"]), A(c["g"]), A(c["m0"]), None, A(c["q"]), hp,
                                   c["alpha"], 1)
    assert np.array_equal(p2, A(c["p_mixed"])) and v2 is None
    assert dis == float(np.sum((A(c["p_local"]) - 1.0) ** 2))


def test_hand_adamw_first_step():
    c = GOLD["adamw_first_step"]
    p1, m1, v1 = O.adamw(A(c["p"]), A(c["g"]), np.zeros((2, 2)), np.zeros((2, 2)), c["lr"],
                         c["beta1"], c["beta2"], c["eps"], c["weight_decay"], c["t"])
    assert np.array_equal(p1, A(c["p_local"]))


def test_adamw_first_step_closed_form_random():
    """t=1: m_hat = g, v_hat = g^2, so p1 = p(1 - lr wd) - lr g / (|g| + eps)."""
    rng = np.random.default_rng(5)
    p, g = rng.standard_normal(1000), rng.standard_normal(1000) * 1e-3
    lr, wd, eps = 1e-3, 0.1, 1e-8
    p1, _, _ = O.adamw(p, g, 0 * p, 0 * p, lr, 0.9, 0.95, eps, wd, 1, store=O.ident)
    ref = p * (1 - lr * wd) - lr * g / (np.abs(g) + eps)
    np.testing.assert_allclose(p1, ref, rtol=1e-12, atol=1e-15)


def test_adamw_constant_gradient_converges_to_sign_step():
    """With a constant gradient the bias-corrected ratio is g/|g| at every t."""
    p, g = A([1.0, -2.0]), A([0.3, -0.7])
    m = v = np.zeros(2)
    for t in range(1, 6):
        pn, m, v = O.adamw(p, g, m, v, 0.01, 0.9, 0.95, 0.0, 0.0, t, store=O.ident)
        np.testing.assert_allclose(pn, p - 0.01 * np.sign(g), rtol=1e-13)
        p = pn


def test_hand_push_sum():
    c = GOLD["push_sum_exchange"]
    w, alpha = O.push_sum_round(c["w"], c["sender"], c["receiver"])
    assert math.isclose(alpha, c["alpha"], rel_tol=1e-15)
    assert w == c["w_after"]
    xs, xr = A(c["x_sender"]), A(c["x_receiver"])
    before = c["w"][0] * xs + c["w"][1] * xr
    xr_new = O.mix(xr, xs, alpha)
    after = w[0] * xs + w[1] * xr_new
    np.testing.assert_allclose(before, A(c["mass"]), rtol=0, atol=1e-15)
    np.testing.assert_allclose(after, A(c["mass"]), rtol=0, atol=1e-15)


def test_push_sum_mass_and_expected_weight():
    """Push-sum conserves the total weight and, at lr 0, the weighted sum of the
    replicas; with uniformly random peers every weight averages to 1/M."""
    rng = np.random.default_rng(7)
    M = 4
    w = [1.0 / M] * M
    x = [rng.standard_normal(3) for _ in range(M)]
    mass0 = sum(wi * xi for wi, xi in zip(w, x))
    acc = np.zeros(M)
    n = 20000
    for it in range(n):
        i = int(rng.integers(M))
        j = int((i + 1 + rng.integers(M - 1)) % M)
        w, alpha = O.push_sum_round(w, i, j)
        x[j] = O.mix(x[j], x[i], alpha)
        acc += np.asarray(w)
        assert abs(sum(w) - 1.0) < 1e-12
    mass = sum(wi * xi for wi, xi in zip(w, x))
    np.testing.assert_allclose(mass, mass0, rtol=1e-9, atol=1e-12)
    np.testing.assert_allclose(acc / n, np.full(M, 1.0 / M), atol=0.01)


# ------------------------------------------------------------ invariants

@pytest.mark.parametrize("optim", ["sgd", "adamw"])
def test_mix_invariants(optim):
    from paper_2410_05985_amd import synthetic as S
    p, g, m, v, q = S.update_mix_inputs(4099, 11, optim)
    hp = dict(optim=optim, lr=1e-2, momentum=0.9, weight_decay=0.1, beta1=0.9, beta2=0.95,
              eps=1e-8)
    # alpha = 0: the pure local step
    p0, m0, v0, _ = O.update_mix(p, g, m, v, q, hp, 0.0, 3)
    if optim == "sgd":
        ref, _ = O.sgd_momentum(p, g, m, hp["lr"], 0.9, 0.1)
    else:
        ref, _, _ = O.adamw(p, g, m, v, hp["lr"], 0.9, 0.95, 1e-8, 0.1, 3)
    assert np.array_equal(p0, O.f32(ref))
    # identical peer: mixing is the identity (0.5 p + 0.5 p is exact)
    pl = O.f32(ref)
    assert np.array_equal(O.f32(O.mix(pl, pl, 0.5)), pl)
    # lr = 0 and no decay: pure averaging
    hp0 = dict(hp, lr=0.0, weight_decay=0.0)
    pz, _, _, _ = O.update_mix(p, g, m, v, q, hp0, 0.5, 3)
    assert np.array_equal(pz, O.f32(0.5 * A(p) + 0.5 * A(q)))
    # symmetric pair keeps the mean exactly
    a_, b_ = O.mix(p, q, 0.5), O.mix(q, p, 0.5)
    assert np.array_equal(a_, b_)
    assert np.array_equal(a_ + b_, A(p) + A(q))


def test_unit_order_and_units():
    assert O.reverse_unit_order(4) == [3, 2, 1, 0]
    units = O.gpt_units(12)
    assert len(units) == 14 and units[0] == ["wte", "wpe"] and units[-1] == ["lnf.g", "lnf.b"]
    assert sum(len(u) for u in units) == 2 + 12 * 12 + 2


# ------------------------------------------------------------ bfloat16

def test_bf16_matches_torch_cast_on_float32():
    rng = np.random.default_rng(3)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * s
                        for s in (1e-30, 1e-3, 1.0, 1e5, 1e30)])
    # exact ties: values halfway between two bfloat16 numbers
    base = torch.tensor(rng.standard_normal(1000), dtype=torch.float32).to(torch.bfloat16)
    bits = base.float().numpy().view(np.uint32) | np.uint32(0x8000)
    x = np.concatenate([x, bits.view(np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = O.bf16(x.astype(np.float64))
    assert np.array_equal(got, ref)


def test_bf16_special_values():
    vals = A([0.0, -0.0, 1.0, -1.0, np.inf, -np.inf, 1 + 2 ** -8, 1 + 3 * 2 ** -8,
              2.0 ** -133, 3 * 2.0 ** -134])
    got = O.bf16(vals)
    assert got[0] == 0 and got[1] == 0 and got[2] == 1 and got[3] == -1
    assert got[4] == np.inf and got[5] == -np.inf
    assert got[6] == 1.0                      # tie rounds to even
    assert got[7] == 1 + 4 * 2 ** -8          # tie rounds to even (upwards)
    assert got[8] == 2.0 ** -133              # smallest subnormal
    assert got[9] == 2.0 ** -132              # tie between 1 and 2 ulps -> even
    assert np.isnan(O.bf16(A([np.nan]))[0])
    # no double rounding: a float64 just above a bfloat16 tie rounds up
    x = 1 + 2 ** -8 + 2 ** -40
    assert O.bf16(A([x]))[0] == 1 + 2 ** -7


def _bf16_nearest_exact(x: float) -> float:
    """Plain definition on one value: enumerate the bfloat16 grid around x
    (8 significant bits; spacing 2**-133 below 2**-126) and take the
    nearest value in exact rational arithmetic, ties to the even
    significand; past the largest finite value the result is infinite."""
    from fractions import Fraction
    if x == 0:
        return x
    ax = Fraction(abs(x))
    e = max(math.frexp(abs(x))[1] - 8, -133)          # grid spacing 2**e
    lo = (ax / Fraction(2) ** e).__floor__()
    cands = [lo, lo + 1]
    best = min(cands, key=lambda k: (abs(Fraction(k) * Fraction(2) ** e - ax), k % 2))
    val = float(Fraction(best) * Fraction(2) ** e)
    if val >= 2.0 ** 128:
        val = math.inf
    return math.copysign(val, x)


def test_bf16_float64_brute_force():
    """float64 inputs with bits far below the bfloat16 grid (no double
    rounding), near ties, across the subnormal and overflow boundaries, in
    a 2-D array (shape kept), against the exact nearest-even definition."""
    rng = np.random.default_rng(5)
    x = rng.standard_normal(3000) * 10.0 ** rng.integers(-42, 39, 3000)
    k = rng.integers(0, 256, 600).astype(np.float64) + 0.5
    e = rng.integers(-141, 121, 600).astype(np.float64)
    ties = k * 2.0 ** e
    x = np.concatenate([x, ties, np.nextafter(ties, 0), np.nextafter(ties, np.inf), -ties,
                        [(2 - 2 ** -8) * 2.0 ** 127, (2 - 2 ** -9) * 2.0 ** 127,
                         np.nextafter((2 - 2 ** -9) * 2.0 ** 127, 0), 2.0 ** -126, 2.0 ** -127,
                         np.nextafter(2.0 ** -126, 0), 2.0 ** -134, np.nextafter(2.0 ** -134, 1), 5e-324,
                         0.0, -0.0, 1.0]])
    x = x.reshape(-1, 2)
    got = O.bf16(x)
    assert got.shape == x.shape
    want = np.array([_bf16_nearest_exact(float(v)) for v in x.reshape(-1)]).reshape(x.shape)
    assert np.array_equal(got, want)


def test_causal_logsumexp_brute_force_and_softmax():
    """The causal log-sum-exp (the softmax normaliser the fused attention
    stores) against a plain loop with math.fsum, and exp(s - lse) against the
    causal softmax on and below the diagonal; a row whose scores are all
    equal has lse = s + log(i + 1)."""
    rng = np.random.default_rng(11)
    s = rng.normal(0.0, 3.0, (2, 5, 5))
    lse = O.causal_logsumexp(s)
    for b in range(2):
        for i in range(5):
            want = math.log(math.fsum(math.exp(s[b, i, j]) for j in range(i + 1)))
            assert abs(lse[b, i] - want) <= 1e-12 * max(1.0, abs(want))
    p = O.causal_softmax(s)
    low = np.tril(np.ones((5, 5), dtype=bool))
    assert np.allclose(np.exp(s - lse[..., None])[:, low], p[:, low], rtol=1e-12, atol=0)
    flat = np.full((1, 4, 4), 0.7)
    assert np.allclose(O.causal_logsumexp(flat)[0], 0.7 + np.log(np.arange(1, 5)), rtol=0, atol=1e-14)
