"""Gradient statistics against n_t on the GPU (library moment kernels and the
experiment driver) vs float64 numpy / the oracle.

* bgpo_moments_update (Welford) and bgpo_moments_summary against two-pass
  numpy statistics on random data, sizes with a ragged tail;
* the whole experiment (on-policy gradients for several n_t, repeats,
  n_t = 16 reference) on the MID shape against ``oracle.gradstats``: every
  mean standard deviation and mean bias within 2e-2 relative (the bar of the
  gradients themselves).
"""
import numpy as np
import pytest
import torch

import workloads
from oracle import gradstats as ogs

pytestmark = pytest.mark.gpu

MID = workloads.Workload("mid_B4_L200_d576_V4288_nt3", B=4, L=200, d=576, V=4288, n_t=3,
                         lengths=(120, 200), group=4, data_seed=2001, philox_seed=0xB6B10001)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.mark.parametrize("n,count", [(1003, 1), (1003, 5), ((1 << 20) + 3, 4)])
def test_moments_kernels_match_numpy(n, count):
    from paper_2510_11683_amd import bgpo
    rng = np.random.default_rng(n + count)
    G = (rng.standard_normal((count, n)) * np.exp(rng.uniform(-3, 3, n))).astype(np.float32)
    ref = rng.standard_normal(n).astype(np.float32)
    mean = torch.zeros(n, dtype=torch.float32, device="cuda")
    m2 = torch.zeros_like(mean)
    for r in range(count):
        bgpo.bgpo_moments_update(torch.from_numpy(G[r]).cuda(), mean, m2, r)
    out = torch.zeros(3, dtype=torch.float64, device="cuda")
    bgpo.bgpo_moments_summary(mean, m2, torch.from_numpy(ref).cuda(), count, out, bgpo.moments_workspace())
    G64 = G.astype(np.float64)
    np.testing.assert_allclose(mean.cpu().numpy(), G64.mean(axis=0), rtol=1e-5, atol=1e-6 * np.abs(G64).max())
    m2_ref = ((G64 - G64.mean(axis=0)) ** 2).sum(axis=0)
    np.testing.assert_allclose(m2.cpu().numpy(), m2_ref, rtol=1e-4, atol=1e-6 * m2_ref.max())
    std, bias, scale = ogs.moments_summary(G64, ref.astype(np.float64))
    o = out.cpu().numpy()
    assert abs(o[0] - std) <= 1e-4 * max(std, 1e-30) + (1e-12 if count == 1 else 0)
    assert abs(o[1] - bias) <= 1e-5 * bias
    assert abs(o[2] - scale) <= 1e-12 * scale
    # without a reference
    bgpo.bgpo_moments_summary(mean, m2, None, count, out, bgpo.moments_workspace())
    o = out.cpu().numpy()
    assert o[1] == 0.0 and o[2] == 0.0


def test_experiment_matches_oracle_on_mid_shape():
    from paper_2510_11683_amd import gradstats
    w = MID
    x = workloads.generate(w)
    kw = dict(n_t_list=(1, 4), repeats=4, golden_n_t=16)
    gpu = gradstats.run(w, x, **kw)
    ref = ogs.run(w, x, **kw)
    for rg, rr in zip(gpu["rows"], ref["rows"]):
        assert rg["n_t"] == rr["n_t"]
        for k in ("dW", "dX"):
            for s in ("std", "bias", "ref"):
                assert abs(rg[k][s] - rr[k][s]) <= 2e-2 * rr[k][s], (rg["n_t"], k, s, rg[k][s], rr[k][s])
    assert gpu["rows"][1]["dW"]["std"] < gpu["rows"][0]["dW"]["std"]
