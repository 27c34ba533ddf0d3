"""Pins for the per-sample form of the ELBO head and the final RMSNorm.

* RMSNorm forward equals torch.nn.functional.rms_norm (float64, CPU); its
  backward equals torch autograd of that routine and central finite
  differences;
* the per-sample literal loop with all samples sharing their activations
  equals the shared-hidden literal loop (and, per sample, sums to it);
* the accumulated gradients of the whole objective with per-sample
  activations and the norm equal torch autograd of an independently written
  expression (log_softmax, gather, both bound branches, off-policy);
* splitting the sample range splits the per-sample results exactly.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import elbo, rmsnorm
from test_oracle_elbo import _rand_problem

EPS = 1e-6


def check_rmsnorm_forward(fn=None):
    fn = fn or rmsnorm.rmsnorm
    rng = np.random.default_rng(11)
    for scale in (1e-3, 1.0, 40.0):
        x = rng.standard_normal((5, 7, 96)) * scale
        gam = rng.standard_normal(96)
        ref = F.rms_norm(torch.from_numpy(x), (96,), torch.from_numpy(gam), EPS).numpy()
        h, _ = fn(x, gam, EPS)
        assert np.allclose(h, ref, rtol=1e-12, atol=1e-14)


def check_rmsnorm_backward(fn=None):
    fn = fn or rmsnorm.rmsnorm_backward
    rng = np.random.default_rng(12)
    x = rng.standard_normal((6, 48)) * 0.7
    gam = rng.standard_normal(48)
    dh = rng.standard_normal((6, 48))
    xt = torch.from_numpy(x.copy()).requires_grad_(True)
    gt = torch.from_numpy(gam.copy()).requires_grad_(True)
    (F.rms_norm(xt, (48,), gt, EPS) * torch.from_numpy(dh)).sum().backward()
    dx, dg = fn(x, gam, EPS, dh)
    assert np.allclose(dx, xt.grad.numpy(), rtol=1e-11, atol=1e-13)
    assert np.allclose(dg, gt.grad.numpy(), rtol=1e-11, atol=1e-13)
    # central differences of <dh, rmsnorm(x)> in a few coordinates
    f = lambda xx: float(np.sum(dh * rmsnorm.rmsnorm(xx, gam, EPS)[0]))
    for (r, c) in ((0, 0), (3, 17), (5, 47)):
        e = np.zeros_like(x)
        e[r, c] = 1e-6
        fd = (f(x + e) - f(x - e)) / 2e-6
        assert abs(fd - dx[r, c]) <= 1e-6 * max(1.0, abs(fd))


def check_round_to_bf16(fn=None):
    """Against torch's float32 -> bfloat16 conversion (round to nearest even) on
    float32-representable values, plus exact ties."""
    fn = fn or rmsnorm.round_to_bf16
    rng = np.random.default_rng(13)
    v = (rng.standard_normal(20000) * np.exp(rng.uniform(-20, 20, 20000))).astype(np.float32)
    ref = torch.from_numpy(v).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(fn(v.astype(np.float64)), ref)
    # ties: 1 + 2^-8 lies halfway between 1 and 1 + 2^-7 -> even (1); 1 + 3 * 2^-8 -> 1 + 2^-6
    t = np.array([1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8, -(1 + 2.0 ** -8), 3 * 2.0 ** -9])
    assert np.array_equal(fn(t), [1.0, 1 + 2.0 ** -6, -1.0, 3 * 2.0 ** -9])


def test_round_to_bf16_matches_torch_and_ties():
    check_round_to_bf16()


def test_rmsnorm_forward_matches_torch():
    check_rmsnorm_forward()


def test_rmsnorm_backward_matches_autograd_and_differences():
    check_rmsnorm_backward()


def test_shared_activations_reduce_to_the_shared_loop():
    p, H, W, y, resp, adv = _rand_problem(31, B=2, L=6, d=5, V=9, n_t=3)
    ell_old = np.random.default_rng(1).standard_normal((p.B, p.n_t)) * 0.3 - 6
    ref = elbo.elbo_literal_f64(p, H, W, y, resp, adv, ell_old=ell_old, loss_scale=0.4)
    sh = elbo.elbo_per_sample(p, H, W, y, resp, adv, ell_old=ell_old, loss_scale=0.4, per_sample=False)
    rep = elbo.elbo_per_sample(p, np.stack([H] * p.n_t), W, y, resp, adv, ell_old=ell_old,
                               loss_scale=0.4, per_sample=True)
    for o in (sh, rep):
        assert np.allclose(o.ell, ref.ell, rtol=1e-14) and np.allclose(o.g, ref.g, rtol=1e-14)
        assert abs(o.loss - ref.loss) <= 1e-14 * abs(ref.loss)
        assert np.allclose(o.dW, ref.dW, rtol=1e-13, atol=1e-16)
    assert np.allclose(sh.dX, ref.dX, rtol=1e-13, atol=1e-16)
    assert np.allclose(rep.dX.sum(axis=0), ref.dX, rtol=1e-12, atol=1e-15)


def _torch_objective(p, X, gam, W, y, resp, adv, ell_old, scale):
    """-scale * sum_{b,j} g_{b,j} with h = rms_norm(X[q]) for sample q, written
    with torch ops from Eq. per_step_loss and Eq. g."""
    total = torch.zeros((), dtype=torch.float64)
    for q, j in enumerate(p.js):
        T, t, m, _ = elbo.sample_masks(p, resp, j)
        H = X[q] if gam is None else F.rms_norm(X[q], (p.d,), gam, EPS)
        for b in range(p.B):
            sel = torch.from_numpy(np.flatnonzero(m[b]))
            if sel.numel() == 0:
                ell = torch.zeros((), dtype=torch.float64)       # empty sum
            else:
                lp = torch.log_softmax(H[b, sel] @ W, dim=-1)
                tg = torch.from_numpy(y[b][sel.numpy()].astype(np.int64))
                ell = lp.gather(1, tg[:, None]).sum() / float(t[b])
            dj = ell - float(ell_old[b, j])
            A = float(adv[b])
            gj = (1 + dj) * A / p.n_t if A >= 0 else torch.exp(dj) * A / p.n_t
            total = total - scale * gj
    return total


@pytest.mark.parametrize("with_norm", [True, False])
def test_per_sample_gradients_match_autograd(with_norm):
    p, H, W, y, resp, adv = _rand_problem(32, B=2, L=6, d=6, V=10, n_t=3)
    rng = np.random.default_rng(2)
    X = rng.standard_normal((p.n_t, p.B, p.L, p.d)) * 1.3
    gam = 1.0 + 0.3 * rng.standard_normal(p.d)
    ell_old = elbo.elbo_per_sample(p, X, W, y, resp, adv, backward=False,
                                   gamma=gam if with_norm else None).ell
    ell_old = ell_old + rng.normal(0, 0.5, ell_old.shape)
    res = elbo.elbo_per_sample(p, X, W, y, resp, adv, ell_old=ell_old, loss_scale=0.3,
                               gamma=gam if with_norm else None, eps=EPS)
    Xt = torch.from_numpy(X.copy()).requires_grad_(True)
    Wt = torch.from_numpy(W.copy()).requires_grad_(True)
    gt = torch.from_numpy(gam.copy()).requires_grad_(True)
    if with_norm:
        obj = _torch_objective(p, Xt, gt, Wt, y, resp, adv, ell_old, 0.3)
    else:
        obj = _torch_objective(p, Xt, None, Wt, y, resp, adv, ell_old, 0.3)
    obj.backward()
    assert abs(res.loss - obj.item()) <= 1e-12 * abs(obj.item())
    assert np.allclose(res.dX, Xt.grad.numpy(), rtol=1e-10, atol=1e-13)
    assert np.allclose(res.dW, Wt.grad.numpy(), rtol=1e-10, atol=1e-13)
    if with_norm:
        assert np.allclose(res.dgamma, gt.grad.numpy(), rtol=1e-10, atol=1e-13)


def test_split_sample_range_with_per_sample_activations():
    p, H, W, y, resp, adv = _rand_problem(33, B=2, L=6, d=5, V=8, n_t=4)
    X = np.random.default_rng(4).standard_normal((4, p.B, p.L, p.d))
    gam = np.linspace(0.5, 1.5, p.d)
    full = elbo.elbo_per_sample(p, X, W, y, resp, adv, gamma=gam)
    import dataclasses
    a = elbo.elbo_per_sample(dataclasses.replace(p, j_begin=0, j_count=1), X[:1], W, y, resp, adv, gamma=gam)
    b = elbo.elbo_per_sample(dataclasses.replace(p, j_begin=1, j_count=3), X[1:], W, y, resp, adv, gamma=gam)
    assert np.allclose(np.concatenate([a.dX, b.dX]), full.dX, rtol=1e-13, atol=1e-16)
    assert np.allclose(a.dW + b.dW, full.dW, rtol=1e-12, atol=1e-15)
    assert np.allclose(a.dgamma + b.dgamma, full.dgamma, rtol=1e-12, atol=1e-15)
    assert abs(a.loss + b.loss - full.loss) <= 1e-13 * abs(full.loss)
