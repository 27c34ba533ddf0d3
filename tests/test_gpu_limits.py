"""Parity at the edges of the supported shape set, through the C ABI.

* B*L = 2^20 positions with B = 4096 (both at their maximum), ragged lengths:
  every count, timestep, l_{b,j}, the whole dX and the whole dW.
* V = 2^20 (the largest vocabulary): the same, dW on sampled vocabulary
  columns (every target, both ends of the vocabulary, 4096 random ones).
* d = 65536 (the largest hidden size) with B*L*d > 2^31 elements in the hidden
  states and dX (responses of 48 to 64 tokens in rows of 1024 positions, so the
  last response's rows sit past 2^31 elements; the hidden states of padding
  positions are zeros): element offsets past 32 bits in the gather and the dX
  scatter; dX on sampled positions, the whole dW.
* d*V > 2^31 elements in W, W^T and dW (d = 2112, V = 2^20).  W and the hidden
  states are zero outside the hidden units [0, 64) and [2048, 2112), whose
  W rows lie past 2^31 elements.  Zero units add exact zeros to every logit and
  have exactly zero dX columns and dW rows, so the problem equals the one over
  those 128 units: the oracle runs that one, the GPU the full one, and the other
  units must come out exactly zero.
Bars as in the other parity tests: counts and t bit-exact, l within 1e-3
relative, dX and dW within 2e-2 relative max-norm.  The oracle widens only the
hidden rows it reads (masked in some sample, or a compared dX row) to float64.
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

BASE = workloads.TINY.replace(hidden="normal", targets="uniform", adv="normal")
# name -> (workload, sampled dX rows, sampled dW columns, input layout)
CASES = {
    "positions_max_B4096_L256_d64_V128_nt2":
        (BASE.replace(B=4096, L=256, d=64, V=128, n_t=2, lengths=(1, 256), data_seed=2301,
                      philox_seed=0xB6B20001), False, False, "plain"),
    "vocab_max_B2_L64_d64_V1048576_nt3":
        (BASE.replace(B=2, L=64, d=64, V=1 << 20, n_t=3, data_seed=2302, philox_seed=0xB6B20002),
         False, True, "plain"),
    "hidden_over_2p31_B33_L1024_d65536_V64_nt2":
        (BASE.replace(B=33, L=1024, d=65536, V=64, n_t=2, lengths=(48, 64), hidden="rmsnorm",
                      data_seed=2303, philox_seed=0xB6B20003), True, False, "zero_padding"),
    "weight_over_2p31_B2_L64_d2112_V1048576_nt2":
        (BASE.replace(B=2, L=64, d=2112, V=1 << 20, n_t=2, data_seed=2304,
                      philox_seed=0xB6B20004), False, True, "units_0_64_2048_2112"),
}
UNITS = np.r_[0:64, 2048:2112]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _inputs(w, layout):
    """(inputs of the GPU run, workload and inputs of the oracle run)."""
    if layout == "plain":
        x = workloads.generate(w)
        return x, w, x
    if layout == "zero_padding":
        # hidden states drawn for the first lengths[1] positions of each
        # response (as a workload of that length), zero beyond: pages of the
        # host array that are never written
        x = workloads.generate(w, with_hidden=False)
        head = workloads.generate(w.replace(L=w.lengths[1]), with_weights=False)["hidden"]
        assert (x["lengths"] <= head.shape[1]).all()
        x["hidden"] = np.zeros((w.B, w.L, w.d), dtype=np.uint16)
        x["hidden"][:, :head.shape[1]] = head
        return x, w, x
    # the problem over UNITS embedded in the full hidden size
    ws = w.replace(d=UNITS.size)
    xs = workloads.generate(ws)
    x = dict(xs)
    x["hidden"] = np.zeros((w.B, w.L, w.d), dtype=np.uint16)
    x["hidden"][:, :, UNITS] = xs["hidden"]
    x["W"] = np.zeros((w.d, w.V), dtype=np.uint16)
    x["W"][UNITS] = xs["W"]
    assert (w.d - 1) * w.V >= 1 << 31 and UNITS[-1] == w.d - 1
    return x, ws, xs


def _sampled(w, x, op, sample_rows, sample_cols):
    """dX positions / dW columns to compare (None: all of them), and the
    positions masked in some sample."""
    rng = np.random.default_rng(11)
    rows = cols = None
    used = np.zeros(w.B * w.L, dtype=bool)
    for j in op.js:
        used |= elbo.sample_masks(op, x["resp_mask"], j)[2].reshape(-1)
    if sample_rows:
        cand = np.flatnonzero(used)
        # the last masked positions sit past 2^31 elements of hidden / dX
        rows = np.unique(np.concatenate([cand[-8:], rng.choice(cand, size=24, replace=False)]))
        assert rows[-1] * w.d >= 1 << 31
    if sample_cols:
        tg = x["targets"].reshape(-1)[x["resp_mask"].reshape(-1) != 0]
        cols = np.unique(np.concatenate([tg, np.arange(64), np.arange(w.V - 64, w.V),
                                         rng.choice(w.V, size=4096, replace=False)]))
    return rows, cols, used


def _oracle(w, x, op, rows, cols, used):
    # the oracle reads hidden rows only where some sample masks the position
    # or a dX row is asked for; those rows are widened exactly, the rest of the
    # float64 array is never touched
    read = used.copy()
    if rows is not None:
        read[rows] = True
    hf = np.zeros((w.B * w.L, w.d))
    hb = x["hidden"].reshape(w.B * w.L, w.d)
    pos = np.flatnonzero(read)
    for c0 in range(0, pos.size, 4096):
        hf[pos[c0:c0 + 4096]] = elbo.bf16_to_f64(hb[pos[c0:c0 + 4096]])
    return elbo.elbo_collapsed(op, None, x["W"], x["targets"], x["resp_mask"], x["adv"],
                               dx_rows=rows, dw_cols=cols, hidden_f64=hf.reshape(w.B, w.L, w.d),
                               row_chunk=64 if w.V >= 1 << 20 else 256)


@pytest.mark.parametrize("name", list(CASES))
def test_shape_limits(name):
    w, sample_rows, sample_cols, layout = CASES[name]
    assert w.B * w.L <= 1 << 20 and w.B <= 4096 and w.d <= 65536 and w.V <= 1 << 20
    x, wo, xo = _inputs(w, layout)
    op = elbo.Problem(wo.B, wo.L, wo.d, wo.V, wo.n_t, seed=wo.philox_seed,
                      seq_id_base=wo.seq_id_base, t_mode=wo.t_mode)
    rows, cols, used = _sampled(wo, xo, op, sample_rows, sample_cols)
    if layout.startswith("units"):
        # the last compared dW column's offset in the last W row is past 2^31
        assert (w.d - 1) * w.V + cols[-1] >= 1 << 31

    r = Runner(w, x)
    del x
    r.bwd()
    torch.cuda.synchronize()
    nm, tt = r.nm.cpu().numpy(), r.t.cpu().numpy()
    ell, g = r.ell.cpu().numpy(), r.g.cpu().numpy()
    loss, flags = float(r.loss.item()), int(r.flags.item())
    dX = r.dX.reshape(w.B * w.L, w.d)
    dX = (dX if rows is None else dX[torch.from_numpy(rows).cuda()]).cpu().numpy()
    dW = (r.dW if cols is None else r.dW[:, torch.from_numpy(cols).cuda()]).cpu().numpy()
    del r
    torch.cuda.empty_cache()
    if layout.startswith("units"):
        off = np.setdiff1d(np.arange(w.d), UNITS)
        assert not dX[:, off].any() and not dW[off].any()
        dX, dW = dX[:, UNITS], dW[UNITS]

    ref = _oracle(wo, xo, op, rows, cols, used)
    del xo
    ref_dX = ref.dX.reshape(-1, wo.d)
    assert flags == 0
    assert np.array_equal(nm, ref.n_masked)
    assert np.array_equal(tt.astype(np.float64), ref.t)
    assert nm.sum() > 0
    np.testing.assert_allclose(ell, ref.ell, rtol=ELL_RTOL, atol=0)
    np.testing.assert_allclose(g, ref.g, rtol=1e-12, atol=1e-15)      # on-policy: A / n_t
    assert abs(loss - ref.loss) <= 1e-9 * max(abs(ref.loss), 1e-12)
    assert np.abs(dX).max() > 0 and np.abs(dW).max() > 0
    assert rel_maxnorm(dX, ref_dX) <= GRAD_RTOL, rel_maxnorm(dX, ref_dX)
    assert rel_maxnorm(dW, ref.dW) <= GRAD_RTOL, rel_maxnorm(dW, ref.dW)
