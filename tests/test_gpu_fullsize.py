"""Full-size parity: the LLaDA-8B head shape (d = 4096, V = 126464) in the launch
configuration that bench.py times, checked against the float64 oracle.

Compared on every case: every count and timestep, every l_{b,j} and g_{b,j},
the loss, dW on every vocabulary column that is the target of a masked row
(those carry the one-hot term and the largest entries) plus 2048 random
columns, and dX

* in full for B=8, L=256, n_t=16, for B=8, L=512, n_t=64 (the benchmark
  workload) and for B=8, L=512 with ragged lengths, n_t=16, off-policy
  (l_old = the oracle's l + N(0, 1) noise, both advantage signs: both branches
  of Eq. g with d != 0 through the multi-unit, batched-dW path);
* on sampled positions for B=16, L=1024, stratified t (the largest
  workload, all 32 samples).

The benchmark workload also runs under workspace budgets: 2 GiB (the
recompute backward, vocabulary chunks, nothing of size rows x V kept) and
8 GiB (the stored backward with smaller units), against the same oracle
result.  The oracle's collapsed form runs the log-softmax once per masked
position in float64, so these tests take tens of seconds of host time; its
results are computed once per workload.
"""
import numpy as np
import pytest
import torch

import workloads
from oracle import elbo
from gpu_util import Runner, rel_maxnorm

pytestmark = pytest.mark.gpu

ELL_RTOL = 1e-3
GRAD_RTOL = 2e-2
GiB = 1 << 30


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _oracle_problem(w):
    return elbo.Problem(w.B, w.L, w.d, w.V, w.n_t, seed=w.philox_seed,
                        seq_id_base=w.seq_id_base, t_mode=w.t_mode)


_CACHE = {}


def _case(w, off_policy=False, full_dx=True, seqs=(3, 12)):
    """Inputs, comparison set and oracle result of one workload (cached)."""
    key = (w.name, off_policy, full_dx)
    if key in _CACHE:
        return _CACHE[key]
    x = workloads.generate(w)
    op = _oracle_problem(w)
    rng = np.random.default_rng(7)
    used = np.zeros((w.B, w.L), dtype=bool)
    for j in op.js:
        used |= elbo.sample_masks(op, x["resp_mask"], j)[2]
    # dW columns: every target of a masked position, plus 2048 random ones
    tg = x["targets"][used]
    cols = np.unique(np.concatenate([tg, rng.choice(w.V, size=2048, replace=False)])).astype(np.int64)
    rows = None
    if not full_dx:
        rows = []
        for b in seqs:
            cand = np.flatnonzero(used[b])
            rows += list(b * w.L + rng.choice(cand, size=min(6, cand.size), replace=False))
        rows = np.array(rows, dtype=np.int64)
    ell_old = None
    if off_policy:
        ell_old = elbo.elbo_collapsed(op, x["hidden"], x["W"], x["targets"], x["resp_mask"],
                                      x["adv"], backward=False).ell
        ell_old = ell_old + np.random.default_rng(11).normal(0.0, 1.0, ell_old.shape)
    ref = elbo.elbo_collapsed(op, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                              ell_old=ell_old, dx_rows=rows, dw_cols=cols)
    _CACHE[key] = (x, cols, rows, ell_old, ref)
    return _CACHE[key]


def _run_and_compare(w, off_policy=False, full_dx=True, seqs=(3, 12), **kw):
    x, cols, rows, ell_old, ref = _case(w, off_policy, full_dx, seqs)
    r = Runner(w, x, **kw)
    r.bwd(ell_old=ell_old)
    torch.cuda.synchronize()
    js = list(range(w.n_t))
    nm, tt = r.nm.cpu().numpy(), r.t.cpu().numpy()
    ell, g = r.ell.cpu().numpy(), r.g.cpu().numpy()
    loss, flags = float(r.loss.item()), int(r.flags.item())
    if rows is None:
        dX = r.dX.cpu().numpy()
    else:
        dX = r.dX.reshape(w.B * w.L, w.d)[torch.from_numpy(rows).cuda()].cpu().numpy()
    dW = r.dW[:, torch.from_numpy(cols).cuda()].cpu().numpy()
    del r
    torch.cuda.empty_cache()

    assert flags == 0
    assert np.array_equal(nm, ref.n_masked)
    assert np.array_equal(tt.astype(np.float64), ref.t)
    np.testing.assert_allclose(ell, ref.ell, rtol=ELL_RTOL, atol=0)
    adv = x["adv"].astype(np.float64)
    old = ell if ell_old is None else ell_old
    g_of_ell = np.array([[elbo.bound_term(ell[b, j] - old[b, j], float(adv[b]), w.n_t)[0]
                          for j in js] for b in range(w.B)])
    np.testing.assert_allclose(g, g_of_ell, rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(g, ref.g, rtol=ELL_RTOL, atol=ELL_RTOL * np.abs(ref.g).max())
    if ell_old is None:
        np.testing.assert_allclose(g, ref.g, rtol=1e-12, atol=1e-15)     # on-policy: A / n_t
    assert abs(loss - (-g_of_ell.sum() / 8)) <= 1e-12 * np.abs(g_of_ell).sum()
    assert abs(loss - ref.loss) <= ELL_RTOL * np.abs(ref.g).sum() / 8
    assert np.abs(dX).max() > 0 and np.abs(dW).max() > 0
    assert rel_maxnorm(dX, ref.dX) <= GRAD_RTOL, rel_maxnorm(dX, ref.dX)
    assert rel_maxnorm(dW, ref.dW) <= GRAD_RTOL, rel_maxnorm(dW, ref.dW)
    return int(nm.sum())


def test_llada_head_B8_L512_nt64_all_samples():
    n = _run_and_compare(workloads.LLADA_L512_NT64)
    assert n > 100_000


@pytest.mark.parametrize("budget", [2 * GiB, 8 * GiB, 48 * GiB],
                         ids=["budget_2GiB_recompute", "budget_8GiB_stored", "budget_48GiB_dw_batch_4"])
def test_llada_head_B8_L512_nt64_under_budget(budget):
    from paper_2510_11683_amd import bgpo
    w = workloads.LLADA_L512_NT64
    plan = bgpo.bgpo_workspace_plan(bgpo.Problem(w.B, w.L, w.d, w.V, w.n_t, ws_budget=budget))
    assert plan["workspace_bytes"] <= budget
    assert plan["mode"] == ("recompute" if budget == 2 * GiB else "stored")
    if budget == 48 * GiB:
        assert plan["dw_batch"] == 4
    n = _run_and_compare(w, ws_budget=budget)
    assert n > 100_000


def test_llada_head_B8_L256_nt16_all_samples():
    assert _run_and_compare(workloads.LLADA_L256) > 0


def test_llada_head_B8_L512_ragged_nt16_off_policy():
    w = workloads.LLADA_L512_RAGGED
    x, *_ = _case(w, off_policy=True)
    assert (x["adv"] > 0).any() and (x["adv"] < 0).any()      # both branches of Eq. g
    assert _run_and_compare(w, off_policy=True) > 0


def test_largest_workload_B16_L1024_stratified_all_samples():
    w = workloads.STRESS_L1024
    assert _run_and_compare(w, full_dx=False, seqs=(3, 12)) > 0
