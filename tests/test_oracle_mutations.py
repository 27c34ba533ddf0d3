"""The oracle's pins catch plausible mistakes.

Each case plants one mistake in a copy of an oracle function (on the CPU, via
monkeypatch) and checks that at least one pin of ``test_oracle_elbo`` fails:
a dropped 1/t, a missing max shift, a swapped bound branch, a wrong
derivative of the bound, a sign flip in the backward, a transposed or
mis-indexed operand.
"""
import numpy as np
import pytest
import torch

from oracle import elbo
import test_oracle_elbo as pins


@pytest.fixture(autouse=True)
def _float64_default():
    """The pins' torch autograd references run in float64 (as in their own
    module); the default is restored afterwards."""
    prev = torch.get_default_dtype()
    torch.set_default_dtype(torch.float64)
    yield
    torch.set_default_dtype(prev)

ALL_PINS = [
    pins.check_log_softmax,
    pins.check_t1_cross_entropy,
    pins.check_brute_force_expectation,
    pins.check_finite_differences,
    lambda: pins.check_autograd(on_policy=False),
    lambda: pins.check_autograd(on_policy=True),
    pins.check_on_policy_equivalence,
    pins.check_bound_equality_cases,
    pins.check_linearity,
    pins.check_bf16_widening,
]


def _any_pin_fails():
    for pin in ALL_PINS:
        try:
            with np.errstate(all="ignore"):
                pin()
        except (AssertionError, ValueError, IndexError, FloatingPointError):
            return True
    return False


def _orig(name):
    return getattr(elbo, name)


def mut_no_inv_t(H_b, W, y_b, mask_b, t, _f=_orig("ell_of_mask")):
    ell, rows, lsm = _f(H_b, W, y_b, mask_b, t)
    return ell * t, rows, lsm


def mut_no_max_shift(z):
    return z - np.log(np.exp(z).sum(axis=1, keepdims=True))


def mut_no_normaliser(z):
    return z - z.max(axis=1, keepdims=True)


def mut_bf16_shift_before_widening(bits):
    # the shift done in 16 bits drops every bit of the pattern
    u = (np.asarray(bits, dtype=np.uint16) << np.uint16(16)).astype(np.uint32)
    return u.view(np.float32).astype(np.float64)


def mut_bf16_low_half(bits):
    # the pattern placed in the low half of the float32 word
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32)
    return u.view(np.float32).astype(np.float64)


def mut_swap_branches(d, A, n_t, *rest):
    if A < 0:
        return (1.0 + d) * A / n_t, A / n_t
    e = np.exp(d)
    return e * A / n_t, e * A / n_t


def mut_taylor_everywhere(d, A, n_t, *rest):
    return (1.0 + d) * A / n_t, A / n_t


def mut_bound_derivative_missing_nt(d, A, n_t, *rest, _f=_orig("bound_term")):
    g, dg = _f(d, A, n_t, *rest)
    return g, dg * n_t


def mut_jensen_derivative_missing_exp(d, A, n_t, *rest, _f=_orig("bound_term")):
    g, dg = _f(d, A, n_t, *rest)
    return g, (A / n_t if A < 0 else dg)


def mut_backprop_sign(H_rows, W, y_rows, lsm, s, _f=_orig("backprop_rows")):
    gx, gw = _f(H_rows, W, y_rows, lsm, s)
    return -gx, -gw


def mut_backprop_no_onehot(H_rows, W, y_rows, lsm, s):
    dZ = s * np.exp(lsm)
    return dZ @ W.T, H_rows.T @ dZ


def mut_backprop_wrong_target(H_rows, W, y_rows, lsm, s):
    y = (np.asarray(y_rows).astype(np.int64) + 1) % W.shape[1]
    dZ = s * np.exp(lsm)
    dZ[np.arange(y.size), y] -= s
    return dZ @ W.T, H_rows.T @ dZ


def mut_backprop_rows_reversed(H_rows, W, y_rows, lsm, s, _f=_orig("backprop_rows")):
    gx, gw = _f(H_rows[::-1], W, y_rows, lsm, s)
    return gx, gw


def mut_dx_without_transpose(H_rows, W, y_rows, lsm, s):
    y = np.asarray(y_rows).astype(np.int64)
    dZ = s * np.exp(lsm)
    dZ[np.arange(y.size), y] -= s
    gx = (dZ[:, :W.shape[0]] if dZ.shape[1] >= W.shape[0] else dZ) @ W[:, :W.shape[0]]
    return gx, H_rows.T @ dZ


MUTATIONS = [
    ("ell_of_mask", mut_no_inv_t),
    ("log_softmax_rows", mut_no_max_shift),
    ("log_softmax_rows", mut_no_normaliser),
    ("bound_term", mut_swap_branches),
    ("bound_term", mut_taylor_everywhere),
    ("bound_term", mut_bound_derivative_missing_nt),
    ("bound_term", mut_jensen_derivative_missing_exp),
    ("backprop_rows", mut_backprop_sign),
    ("backprop_rows", mut_backprop_no_onehot),
    ("backprop_rows", mut_backprop_wrong_target),
    ("backprop_rows", mut_backprop_rows_reversed),
    ("backprop_rows", mut_dx_without_transpose),
    ("bf16_to_f64", mut_bf16_shift_before_widening),
    ("bf16_to_f64", mut_bf16_low_half),
]


def test_pins_pass_unmutated():
    assert not _any_pin_fails()


@pytest.mark.parametrize("name,fn", MUTATIONS, ids=[f.__name__ for _, f in MUTATIONS])
def test_mutation_is_caught(monkeypatch, name, fn):
    monkeypatch.setattr(elbo, name, fn)
    assert _any_pin_fails(), f"planted mistake {fn.__name__} in {name} passed every pin"


# ---------------------------------------------------------------- final RMSNorm

import test_oracle_rmsnorm as norm_pins
from oracle import rmsnorm as _rmsnorm

NORM_PINS = [
    norm_pins.check_round_to_bf16,
    norm_pins.check_rmsnorm_forward,
    norm_pins.check_rmsnorm_backward,
    lambda: norm_pins.test_per_sample_gradients_match_autograd(True),
]


def mut_norm_no_eps(x, gamma, eps):
    x = np.asarray(x, dtype=np.float64)
    r = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True))
    return x * r * gamma, r


def mut_norm_sum_not_mean(x, gamma, eps):
    x = np.asarray(x, dtype=np.float64)
    r = 1.0 / np.sqrt(np.sum(x * x, axis=-1, keepdims=True) + eps)
    return x * r * gamma, r


def mut_norm_bwd_no_projection(x, gamma, eps, dh):
    _, r = _rmsnorm.rmsnorm(x, gamma, eps)
    return r * gamma * dh, np.sum((dh * x * r).reshape(-1, x.shape[-1]), axis=0)


def mut_norm_bwd_r_squared(x, gamma, eps, dh):
    d = x.shape[-1]
    _, r = _rmsnorm.rmsnorm(x, gamma, eps)
    proj = np.sum(gamma * dh * x, axis=-1, keepdims=True)
    return r * gamma * dh - (r ** 2 / d) * x * proj, np.sum((dh * x * r).reshape(-1, d), axis=0)


def mut_norm_dgamma_without_r(x, gamma, eps, dh, _f=_rmsnorm.rmsnorm_backward):
    dx, _ = _f(x, gamma, eps, dh)
    return dx, np.sum((dh * x).reshape(-1, x.shape[-1]), axis=0)


def mut_round_truncates(v):
    v = np.asarray(v, dtype=np.float64)
    m, e = np.frexp(v)
    return np.ldexp(np.trunc(m * 256.0) / 256.0, e)


def mut_round_half_away(v):
    v = np.asarray(v, dtype=np.float64)
    m, e = np.frexp(v)
    return np.ldexp(np.sign(m) * np.floor(np.abs(m) * 256.0 + 0.5) / 256.0, e)


NORM_MUTATIONS = [
    ("round_to_bf16", mut_round_truncates),
    ("round_to_bf16", mut_round_half_away),
    ("rmsnorm", mut_norm_no_eps),
    ("rmsnorm", mut_norm_sum_not_mean),
    ("rmsnorm_backward", mut_norm_bwd_no_projection),
    ("rmsnorm_backward", mut_norm_bwd_r_squared),
    ("rmsnorm_backward", mut_norm_dgamma_without_r),
]


def _any_norm_pin_fails():
    for pin in NORM_PINS:
        try:
            with np.errstate(all="ignore"):
                pin()
        except (AssertionError, ValueError, IndexError, FloatingPointError):
            return True
    return False


def test_norm_pins_pass_unmutated():
    assert not _any_norm_pin_fails()


@pytest.mark.parametrize("name,fn", NORM_MUTATIONS, ids=[f.__name__ for _, f in NORM_MUTATIONS])
def test_norm_mutation_is_caught(monkeypatch, name, fn):
    monkeypatch.setattr(_rmsnorm, name, fn)
    assert _any_norm_pin_fails(), f"planted mistake {fn.__name__} in {name} passed every pin"
