"""Full-size parity: the LLaDA-8B head shape (d = 4096, V = 126464) in the launch
configuration that bench.py times, checked against the float64 oracle on
sampled outputs.

* B=8, L=512, n_t=64 (the benchmark workload): every count and timestep, every
  l_{b,j} and g_{b,j}, the loss, dX on sampled positions and dW on sampled
  vocabulary columns (random ones plus the most frequent target tokens, whose
  columns carry the one-hot term and the largest entries).
* B=8, L=256, n_t=16 and B=8, L=512 with ragged lengths, n_t=16: the same
  checks over all samples.
* B=16, L=1024, stratified t (the largest workload), all 32 samples: the same
  checks.
The oracle's collapsed form runs the log-softmax once per masked position in
float64, so these tests take tens of seconds of host time.
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


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _sample_rows_cols(w, x, rng, used, n_rows_per_seq=6, seqs=(0, 5), n_cols=768, n_top=256):
    """dX rows: positions of responses `seqs` masked in some sample of the range."""
    rows = []
    for b in seqs:
        cand = np.flatnonzero(used[b])
        rows += list(b * w.L + rng.choice(cand, size=min(n_rows_per_seq, cand.size), replace=False))
    tg = x["targets"].reshape(-1)[x["resp_mask"].reshape(-1) != 0]
    vals, counts = np.unique(tg, return_counts=True)
    top = vals[np.argsort(-counts)[:n_top]]
    cols = np.unique(np.concatenate([top, rng.choice(w.V, size=n_cols, replace=False)]))
    return np.array(rows, dtype=np.int64), cols.astype(np.int64)


def _run_and_compare(w, j_begin, j_count, seqs):
    x = workloads.generate(w)
    rng = np.random.default_rng(7)
    op = elbo.Problem(w.B, w.L, w.d, w.V, w.n_t, j_begin=j_begin, j_count=j_count,
                      seed=w.philox_seed, seq_id_base=w.seq_id_base, t_mode=w.t_mode)
    used = np.zeros((w.B, w.L), dtype=bool)
    for j in op.js:
        used |= elbo.sample_masks(op, x["resp_mask"], j)[2]
    rows, cols = _sample_rows_cols(w, x, rng, used, seqs=seqs)
    r = Runner(w, x)
    r.bwd(j_begin=j_begin, j_count=j_count)
    torch.cuda.synchronize()
    js = list(range(j_begin, j_begin + j_count))
    nm = r.nm.cpu().numpy()
    tt = r.t.cpu().numpy()
    ell = r.ell.cpu().numpy()
    g = r.g.cpu().numpy()
    loss = float(r.loss.item())
    flags = int(r.flags.item())
    dX = r.dX.reshape(w.B * w.L, w.d)[torch.from_numpy(rows).cuda()].cpu().numpy()
    dW = r.dW[:, torch.from_numpy(cols).cuda()].cpu().numpy()
    del r
    torch.cuda.empty_cache()

    ref = elbo.elbo_collapsed(op, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                              dx_rows=rows, dw_cols=cols)
    assert flags == 0
    assert np.array_equal(nm[:, js], ref.n_masked[:, js])
    assert np.array_equal(tt[:, js].astype(np.float64), ref.t[:, js])
    np.testing.assert_allclose(ell[:, js], ref.ell[:, js], rtol=ELL_RTOL, atol=0)
    np.testing.assert_allclose(g[:, js], ref.g[:, js], rtol=1e-12, atol=1e-15)   # on-policy: A / n_t
    assert abs(loss - ref.loss) <= 1e-9 * max(abs(ref.loss), 1e-12)
    assert np.abs(dX).max() > 0 and np.abs(dW).max() > 0
    assert rel_maxnorm(dX, ref.dX) <= GRAD_RTOL, rel_maxnorm(dX, ref.dX)
    assert rel_maxnorm(dW, ref.dW) <= GRAD_RTOL, rel_maxnorm(dW, ref.dW)
    return nm[:, js].sum()


def test_llada_head_B8_L512_nt64_all_samples():
    n = _run_and_compare(workloads.LLADA_L512_NT64, 0, 64, seqs=(0, 5))
    assert n > 100_000


@pytest.mark.parametrize("w", [workloads.LLADA_L256, workloads.LLADA_L512_RAGGED], ids=lambda w: w.name)
def test_llada_head_nt16_all_samples(w):
    n = _run_and_compare(w, 0, w.n_t, seqs=(2, 7))
    assert n > 0


def test_largest_workload_B16_L1024_stratified_all_samples():
    w = workloads.STRESS_L1024
    n = _run_and_compare(w, 0, w.n_t, seqs=(3, 12))
    assert n > 0
