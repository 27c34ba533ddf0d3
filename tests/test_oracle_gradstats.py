"""Pins for the gradient statistics against n_t (Section 4, "Effect of
Increasing MC Sample Sizes").

* the per-sample gradient is an unbiased estimate of the gradient of the full
  log-likelihood at every t: brute force over all 2^L masks with their exact
  probabilities (the gradient form of the closed form E[l | t] = sum_i log p_i),
  so the bias against a large-n_t reference can only come from Monte-Carlo
  noise;
* the summary statistics equal closed forms on constructed estimates
  (two repeats: sample std |a - b| / sqrt 2, mean (a + b) / 2);
* on a small workload the standard deviation falls as n_t grows, close to
  1 / sqrt(n_t) (the estimates for different samples are independent).
"""
import itertools

import numpy as np
import torch

import workloads
from oracle import elbo, gradstats


def test_per_sample_gradient_is_unbiased_at_every_t():
    rng = np.random.default_rng(21)
    L, d, V = 9, 5, 11
    H = rng.standard_normal((L, d))
    W = rng.standard_normal((d, V))
    y = rng.integers(0, V, size=L)
    Ht = torch.from_numpy(H.copy()).requires_grad_(True)
    Wt = torch.from_numpy(W.copy()).requires_grad_(True)
    full = torch.log_softmax(Ht @ Wt, dim=1)[torch.arange(L), torch.from_numpy(y)].sum()
    (-full).backward()                      # gradient of -sum log p (s = 1 per unit t)
    for t in (0.07, 0.5, 0.91):
        eX, eW = np.zeros_like(H), np.zeros_like(W)
        for bits in itertools.product((0, 1), repeat=L):
            m = np.array(bits, dtype=bool)
            k = int(m.sum())
            if k == 0:
                continue
            prob = t ** k * (1 - t) ** (L - k)
            _, rows, lsm = elbo.ell_of_mask(H, W, y, m, t)
            gx, gw = elbo.backprop_rows(H[rows], W, y[rows], lsm, 1.0 / t)
            eX[rows] += prob * gx
            eW += prob * gw
        assert np.allclose(eX, Ht.grad.numpy(), rtol=1e-11, atol=1e-13)
        assert np.allclose(eW, Wt.grad.numpy(), rtol=1e-11, atol=1e-13)


def test_summary_closed_forms():
    rng = np.random.default_rng(22)
    a, b = rng.standard_normal((2, 7, 5))
    ref = rng.standard_normal((7, 5))
    std, bias, scale = gradstats.moments_summary(np.stack([a, b]), ref)
    assert abs(std - np.mean(np.abs(a - b) / np.sqrt(2))) <= 1e-14
    assert abs(bias - np.mean(np.abs((a + b) / 2 - ref))) <= 1e-14
    assert abs(scale - np.mean(np.abs(ref))) <= 1e-14
    # one repeat: no spread, bias against itself zero
    std1, bias1, _ = gradstats.moments_summary(a[None], a)
    assert std1 == 0.0 and bias1 == 0.0


def test_std_falls_with_n_t_on_a_small_workload():
    w = workloads.TINY.replace(t_mode=1)     # stratified t keeps the estimates well-behaved
    res = gradstats.run(w, workloads.generate(w), (1, 4, 16), repeats=8, golden_n_t=64)
    s = [r["dW"]["std"] for r in res["rows"]]
    assert s[0] > s[1] > s[2]
    assert 1.3 < s[0] / s[1] < 3.5 and 1.3 < s[1] / s[2] < 3.5     # ~ sqrt(4) = 2
