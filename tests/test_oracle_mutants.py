"""Planted mistakes: each case swaps one oracle function for a copy with one
plausible error (a dropped term, a wrong sign, a transposed operand, a wrong
axis, an off-by-one mask, a coupled instead of decoupled decay) and checks
that the oracle's own pins -- hand-derived cases, closed forms, invariants,
finite differences, brute force -- reject it.  The mistake lives only in the
oracle, on the CPU, for the duration of one case (monkeypatch).  CPU only."""
import math

import numpy as np
import pytest

import oracle as O
import oracle.layup_ref as R
from tests import test_oracle_fd as FD
from tests import test_oracle_pins as PIN


def _linear_bwd_dx_transposed(dy, x, w, need_dx=True):
    # dX with the weight transposed (dy W^T instead of dy W)
    return dy.T @ x, dy.sum(axis=0), (dy @ w.T if need_dx else None)


def _linear_bwd_db_wrong_axis(dy, x, w, need_dx=True):
    # bias gradient summed over the features instead of the rows
    return dy.T @ x, dy.sum(axis=1), (dy @ w if need_dx else None)


def _layernorm_bwd_no_mean_term(dy, x, g, eps=1e-5):
    # the mean(dxh) term of the LayerNorm backward dropped
    mu = x.mean(axis=-1, keepdims=True)
    r = 1.0 / np.sqrt(((x - mu) ** 2).mean(axis=-1, keepdims=True) + eps)
    xh = (x - mu) * r
    dxh = dy * g
    dx = r * (dxh - xh * (dxh * xh).mean(axis=-1, keepdims=True))
    return dx, (dy * xh).sum(axis=0), dy.sum(axis=0)


def _layernorm_bwd_sign(dy, x, g, eps=1e-5):
    # wrong sign of the xh * mean(dxh * xh) term
    mu = x.mean(axis=-1, keepdims=True)
    r = 1.0 / np.sqrt(((x - mu) ** 2).mean(axis=-1, keepdims=True) + eps)
    xh = (x - mu) * r
    dxh = dy * g
    dx = r * (dxh - dxh.mean(axis=-1, keepdims=True) + xh * (dxh * xh).mean(axis=-1, keepdims=True))
    return dx, (dy * xh).sum(axis=0), dy.sum(axis=0)


def _gelu_grad_no_cubic(x):
    # derivative with the 3 * 0.044715 x^2 factor of the inner polynomial dropped
    c = math.sqrt(2.0 / math.pi)
    t = np.tanh(c * (x + 0.044715 * x ** 3))
    return 0.5 * (1.0 + t) + 0.5 * x * (1.0 - t * t) * c


def _softmax_bwd_sign(p, dp):
    return p * (dp + (dp * p).sum(axis=-1, keepdims=True))


def _causal_lse_strict(s):
    # mask that also drops the diagonal (k = 0 instead of k = 1)
    t = s.shape[-1]
    mask = np.triu(np.ones((t, t), dtype=bool), k=0)
    z = np.where(mask, -np.inf, s)
    with np.errstate(invalid="ignore", divide="ignore"):
        mx = np.max(z, axis=-1, keepdims=True)
        return (mx + np.log(np.exp(z - mx).sum(axis=-1, keepdims=True)))[..., 0]


def _cross_entropy_no_mean(z, y):
    # gradient of the summed loss (the 1/rows of the mean dropped)
    n = z.shape[0]
    zm = z.max(axis=-1, keepdims=True)
    e = np.exp(z - zm)
    s = e.sum(axis=-1, keepdims=True)
    loss = float(np.mean(np.log(s)[:, 0] + zm[:, 0] - z[np.arange(n), y]))
    dz = e / s
    dz[np.arange(n), y] -= 1.0
    return loss, dz


def _sgd_dampened(p, g, m, lr, momentum, weight_decay, wd_on=True, store=O.f32):
    # momentum with dampening (1 - mu) g, which the LibTorch default does not have
    p = np.asarray(p, np.float64)
    gg = np.asarray(g, np.float64) + (weight_decay * p if wd_on else 0.0)
    m_new = momentum * np.asarray(m, np.float64) + (1.0 - momentum) * gg
    return p - lr * m_new, store(m_new)


def _adamw_no_bias_correction(p, g, m, v, lr, beta1, beta2, eps, weight_decay, t, wd_on=True,
                              store=O.f32):
    p = np.asarray(p, np.float64)
    g = np.asarray(g, np.float64)
    if wd_on and weight_decay != 0.0:
        p = p * (1.0 - lr * weight_decay)
    m_new = beta1 * np.asarray(m, np.float64) + (1.0 - beta1) * g
    v_new = beta2 * np.asarray(v, np.float64) + (1.0 - beta2) * g * g
    return p - lr * m_new / (np.sqrt(v_new) + eps), store(m_new), store(v_new)


def _adamw_coupled_decay(p, g, m, v, lr, beta1, beta2, eps, weight_decay, t, wd_on=True,
                         store=O.f32):
    # L2 decay folded into the gradient (Adam + L2) instead of decoupled
    p = np.asarray(p, np.float64)
    g = np.asarray(g, np.float64) + (weight_decay * p if wd_on else 0.0)
    m_new = beta1 * np.asarray(m, np.float64) + (1.0 - beta1) * g
    v_new = beta2 * np.asarray(v, np.float64) + (1.0 - beta2) * g * g
    bc1, bc2 = 1.0 - beta1 ** t, 1.0 - beta2 ** t
    return (p - (lr / bc1) * m_new / (np.sqrt(v_new) / math.sqrt(bc2) + eps), store(m_new),
            store(v_new))


def _mix_swapped(p, q, alpha):
    # the receiving copy keeps alpha instead of 1 - alpha
    return alpha * np.asarray(p, np.float64) + (1.0 - alpha) * np.asarray(q, np.float64)


def _push_sum_alpha_inverted(w_self, w_sender):
    return w_self / (w_self + w_sender)


MUTANTS = [
    ("linear_bwd", _linear_bwd_dx_transposed, [PIN.test_hand_linear_backward, FD.test_fd_linear]),
    ("linear_bwd", _linear_bwd_db_wrong_axis, [PIN.test_hand_linear_backward, FD.test_fd_linear]),
    ("layernorm_bwd", _layernorm_bwd_no_mean_term, [FD.test_fd_layernorm]),
    ("layernorm_bwd", _layernorm_bwd_sign, [FD.test_fd_layernorm]),
    ("gelu_tanh_grad", _gelu_grad_no_cubic, [FD.test_fd_gelu_and_relu]),
    ("softmax_bwd", _softmax_bwd_sign, [FD.test_fd_causal_attention_core]),
    ("causal_logsumexp", _causal_lse_strict, [PIN.test_causal_logsumexp_brute_force_and_softmax]),
    ("cross_entropy", _cross_entropy_no_mean, [FD.test_fd_cross_entropy]),
    ("sgd_momentum", _sgd_dampened, [PIN.test_hand_sgd_momentum_then_mix]),
    ("adamw", _adamw_no_bias_correction, [PIN.test_hand_adamw_first_step,
                                          PIN.test_adamw_first_step_closed_form_random]),
    ("adamw", _adamw_coupled_decay, [PIN.test_adamw_first_step_closed_form_random]),
    ("mix", _mix_swapped, [PIN.test_hand_push_sum]),
    ("push_sum_alpha", _push_sum_alpha_inverted, [PIN.test_hand_push_sum]),
]


@pytest.mark.parametrize("name,fn,pins", MUTANTS, ids=[m[1].__name__.lstrip("_") for m in MUTANTS])
def test_pins_reject_planted_mistake(name, fn, pins, monkeypatch):
    for pin in pins:  # each pin passes on the unmodified oracle
        pin()
    monkeypatch.setattr(R, name, fn)
    monkeypatch.setattr(O, name, fn)
    for pin in pins:
        with pytest.raises((AssertionError, ValueError)):
            pin()
