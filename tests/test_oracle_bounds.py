"""Pins for the objective modes beyond the paper's Eq. g: the Taylor-only and
Jensen-only ablations (Table 3) and the exact objective exp(B_theta - B_old) A
(Eq. elbo_ratio), whose gradient couples all n_t samples.

* direction of each bound (Lemma 1: e^x >= 1 + x; Lemma 2: Jensen's
  inequality): for A >= 0 the Taylor term is a lower bound and the Jensen term
  an upper bound of R = exp(mean d) A; for A < 0 the roles swap;
* the exact mode's terms sum to R, and its accumulated gradient equals
  torch.autograd of -scale exp(B_theta - B_old) A off-policy;
* on-policy every mode has value A and the same gradient (Section 3.2);
* the exact mode refuses a partial sample range.
"""
import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

from oracle import elbo
from test_oracle_elbo import _rand_problem



@pytest.fixture(autouse=True)
def _float64_default():
    """torch's autograd pins in this module run in float64; the default is
    restored afterwards, so that other modules (collected in the same
    process) keep float32."""
    prev = torch.get_default_dtype()
    torch.set_default_dtype(torch.float64)
    yield
    torch.set_default_dtype(prev)
MODES = (elbo.BOUND_PAPER, elbo.BOUND_TAYLOR, elbo.BOUND_JENSEN, elbo.BOUND_EXACT)


def _with_mode(p, mode):
    import dataclasses
    return dataclasses.replace(p, bound=mode)


@settings(max_examples=20, deadline=None)
@given(seed=st.integers(0, 10_000), eps=st.floats(1e-3, 0.5), a0=st.floats(0.01, 3), a1=st.floats(-3, -0.01))
def test_bound_directions(seed, eps, a0, a1):
    p, H, W, y, resp, adv = _rand_problem(seed, B=2, L=5, d=3, V=7, n_t=4)
    adv = np.array([a0, a1])
    Wold = W + eps * np.random.default_rng(seed + 1).standard_normal(W.shape)
    old = elbo.elbo_literal_f64(p, H, Wold, y, resp, adv, backward=False).ell
    res = {m: elbo.elbo_literal_f64(_with_mode(p, m), H, W, y, resp, adv, ell_old=old,
                                    backward=False) for m in MODES}
    R = np.exp((res[0].ell - old).mean(axis=1)) * adv
    tol = 1e-12 * (1 + np.abs(R))
    tay = res[elbo.BOUND_TAYLOR].g.sum(axis=1)
    jen = res[elbo.BOUND_JENSEN].g.sum(axis=1)
    assert tay[0] <= R[0] + tol[0] and jen[0] >= R[0] - tol[0]      # A >= 0
    assert tay[1] >= R[1] - tol[1] and jen[1] <= R[1] + tol[1]      # A < 0
    assert np.allclose(res[elbo.BOUND_EXACT].g.sum(axis=1), R, rtol=1e-12, atol=1e-15)
    # the paper's choice is the lower bound of the two in each sign
    assert np.allclose(res[elbo.BOUND_PAPER].g.sum(axis=1), [tay[0], jen[1]], rtol=1e-13)


def test_exact_gradient_matches_autograd_off_policy():
    p, H, W, y, resp, adv = _rand_problem(21, B=2, L=6, d=4, V=9, n_t=5)
    adv = np.array([0.8, -1.4])
    scale = 0.3
    ell_old = np.random.default_rng(3).standard_normal((p.B, p.n_t)) * 0.4 - 7.0
    res = elbo.elbo_literal_f64(_with_mode(p, elbo.BOUND_EXACT), H, W, y, resp, adv,
                                ell_old=ell_old, loss_scale=scale)
    Ht = torch.tensor(H, requires_grad=True)
    Wt = torch.tensor(W, requires_grad=True)
    total = torch.zeros(())
    for b in range(p.B):
        ells = []
        for j in p.js:
            T, t, m, _ = elbo.sample_masks(p, resp, j)
            sel = torch.from_numpy(np.flatnonzero(m[b]))
            tgt = torch.from_numpy(y[b][sel.numpy()].astype(np.int64))
            lp = torch.log_softmax(Ht[b, sel] @ Wt, dim=-1).gather(1, tgt[:, None]).sum()
            ells.append(lp / float(t[b]))
        Bhat = torch.stack(ells).mean()
        total = total - scale * torch.exp(Bhat - float(ell_old[b].mean())) * float(adv[b])
    total.backward()
    assert abs(res.loss - total.item()) <= 1e-12 * abs(total.item())
    assert np.allclose(res.dX, Ht.grad.numpy(), rtol=1e-10, atol=1e-13)
    assert np.allclose(res.dW, Wt.grad.numpy(), rtol=1e-10, atol=1e-13)


def test_all_modes_agree_on_policy():
    p, H, W, y, resp, adv = _rand_problem(5, B=2, L=6, d=4, V=8, n_t=4)
    fwd = elbo.elbo_literal_f64(p, H, W, y, resp, adv, backward=False)
    outs = [elbo.elbo_literal_f64(_with_mode(p, m), H, W, y, resp, adv, ell_old=fwd.ell)
            for m in MODES]
    for o in outs:
        assert np.allclose(o.g.sum(axis=1), adv, rtol=1e-14, atol=1e-15)
        assert np.allclose(o.dX, outs[0].dX, rtol=1e-13, atol=1e-16)
        assert np.allclose(o.dW, outs[0].dW, rtol=1e-13, atol=1e-16)


def test_collapsed_matches_literal_every_mode():
    p, H, W, y, resp, adv = _rand_problem(6, B=2, L=6, d=4, V=8, n_t=3)
    import workloads
    w = workloads.TINY.replace(B=3, n_t=3, lengths=(40, 64), adv="normal")
    x = workloads.generate(w)
    q = elbo.Problem(w.B, w.L, w.d, w.V, w.n_t, seed=w.philox_seed)
    ell_old = elbo.elbo_literal(q, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                                backward=False).ell + 0.2
    for m in MODES:
        qm = _with_mode(q, m)
        a = elbo.elbo_literal(qm, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"], ell_old=ell_old)
        c = elbo.elbo_collapsed(qm, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"], ell_old=ell_old)
        assert np.allclose(a.g, c.g, rtol=1e-12) and abs(a.loss - c.loss) <= 1e-12 * abs(a.loss)
        assert np.abs(a.dW - c.dW).max() <= 1e-11 * np.abs(a.dW).max()


def test_exact_mode_needs_full_range():
    p, H, W, y, resp, adv = _rand_problem(7, n_t=4)
    q = elbo.Problem(p.B, p.L, p.d, p.V, p.n_t, j_begin=1, j_count=2, seed=p.seed, bound=elbo.BOUND_EXACT)
    with pytest.raises(ValueError):
        elbo.elbo_literal_f64(q, H, W, y, resp, adv)
