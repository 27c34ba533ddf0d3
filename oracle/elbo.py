"""Float64 CPU oracle of the BGPO per-Monte-Carlo-sample ELBO head.

TEST INFRASTRUCTURE: this package is the oracle.  Only the test suite, the
smoke check and the benchmark's CPU-baseline leg may import it; the product
path never does.  It shares no code with the HIP path.

What is computed, per response b and Monte-Carlo sample j (Algorithm 1, inner
loops; Section 2.2 and Section 3):

  t_{b,j}      timestep on the 24-bit grid (see ``oracle.philox``)
  m_{b,j,i}    forward masking process: each response position masked with
               probability t (Section 2.1)
  log p_i      log-softmax of the LM-head logits z_i = h_i W at the target
               token y_i (the mask predictor's log-probability, Eq. per_step_loss)
  l_{b,j}      = (1/t) * sum_i m_{b,j,i} log p_i                (Eq. per_step_loss)
  d_{b,j}      = l_theta - l_old on the same masked sample      (Section 3.1)
  g_{b,j}      = (1 + d) A / n_t  if A >= 0  (first-order Taylor, Lemma 1)
               = e^d A / n_t      if A <  0  (Jensen, Lemma 2)  (Eq. g)
               (also: Taylor-only / Jensen-only ablations of Table 3, and the
               exact objective exp(mean_j d_j) A of Eq. elbo_ratio)
  loss        += -loss_scale * g_{b,j}    (Algorithm 1 sets L_j = -g_j / G)
  gradients    of the loss w.r.t. the hidden states and the head weights,
               accumulated over every (b, j) (Algorithm 1, gradient
               accumulation; Eq. lower_bound_def makes the objective a sum).

Chain rule used for the gradients: dg/dl = A/n_t (Taylor) or e^d A/n_t
(Jensen), d l / d z_{i,v} = (1/t) m_i ([v = y_i] - softmax(z_i)_v), hence
d loss / d z_{i,v} = s_{b,j} m_i (softmax(z_i)_v - [v = y_i]) with
s_{b,j} = loss_scale * (dg/dl) / t.

Inputs are the bf16 bit patterns produced by the workload generator; they are
widened to float64 exactly, so input rounding is not part of any error.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

from . import philox
from . import rmsnorm as _rms


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns (uint16) to float64."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def log_softmax_rows(z: np.ndarray) -> np.ndarray:
    """Row-wise log-softmax, shifted by the row maximum."""
    m = z.max(axis=1, keepdims=True)
    return z - (m + np.log(np.exp(z - m).sum(axis=1, keepdims=True)))


BOUND_PAPER, BOUND_TAYLOR, BOUND_JENSEN, BOUND_EXACT = 0, 1, 2, 3


def bound_term(d: float, A: float, n_t: int, mode: int = BOUND_PAPER, dbar: float = 0.0):
    """Per-sample objective term and its derivative w.r.t. l_j: (g_j, dg_j/dl_j).

    BOUND_PAPER  Eq. g: A >= 0 (including -0.0) takes the first-order Taylor
                 term (1 + d) A / n_t (Lemma 1), A < 0 the Jensen term
                 e^d A / n_t (Lemma 2)
    BOUND_TAYLOR the Taylor term for every A (ablation of Table 3)
    BOUND_JENSEN the Jensen term for every A (ablation of Table 3)
    BOUND_EXACT  the exact objective R = exp(dbar) A of Eq. elbo_ratio, dbar =
                 mean_j d_j over all n_t samples; g_j = R / n_t is sample j's
                 share of its value and dR/dl_j = exp(dbar) A / n_t"""
    if mode == BOUND_EXACT:
        e = np.exp(dbar)
        return e * A / n_t, e * A / n_t
    if mode == BOUND_TAYLOR or (mode == BOUND_PAPER and A >= 0):
        return (1.0 + d) * A / n_t, A / n_t
    e = np.exp(d)
    return e * A / n_t, e * A / n_t


@dataclasses.dataclass
class Problem:
    """Sizes and sampling parameters; mirrors the C-ABI problem struct."""
    B: int
    L: int
    d: int
    V: int
    n_t: int
    j_begin: int = 0
    j_count: Optional[int] = None
    seed: int = 0
    seq_id_base: int = 0
    t_mode: int = 0                 # 0 = i.i.d. U(0,1), 1 = stratified
    bound: int = 0                  # BOUND_PAPER / _TAYLOR / _JENSEN / _EXACT

    @property
    def js(self):
        jc = self.n_t - self.j_begin if self.j_count is None else self.j_count
        return range(self.j_begin, self.j_begin + jc)


def sample_masks(p: Problem, resp_mask: np.ndarray, j: int):
    """Timesteps and masks of every response in sample j.

    Returns (T24 int64 [B], t float64 [B], mask bool [B, L], idx int64 [N]) where
    idx lists the masked flat positions b*L + i in ascending order."""
    T = np.array([philox.t24(p.seed, p.seq_id_base + b, j, p.n_t, p.t_mode) for b in range(p.B)],
                 dtype=np.int64)
    m = np.stack([philox.mask_row(p.seed, p.seq_id_base + b, j, int(T[b]), resp_mask[b])
                  for b in range(p.B)])
    idx = np.flatnonzero(m.reshape(-1))
    return T, T.astype(np.float64) / float(1 << 24), m, idx


@dataclasses.dataclass
class Result:
    ell: np.ndarray            # [B, n_t] float64 (only the j range filled)
    g: np.ndarray              # [B, n_t]
    n_masked: np.ndarray       # [B, n_t] int64
    t: np.ndarray              # [B, n_t] float64
    loss: float
    dX: Optional[np.ndarray]   # [B, L, d] float64
    dW: Optional[np.ndarray]   # [d, V] float64
    idx: dict                  # j -> ascending masked flat positions


def ell_of_mask(H_b, W, y_b, mask_b, t):
    """Eq. per_step_loss for one response and one explicit mask.

    H_b [L, d] and W [d, V] float64, y_b [L] targets, mask_b [L] bool, t > 0.
    Returns (l, rows, log_softmax of the masked rows)."""
    rows = np.flatnonzero(mask_b)
    if rows.size == 0:
        return 0.0, rows, np.zeros((0, W.shape[1]))
    lsm = log_softmax_rows(H_b[rows] @ W)
    lp = lsm[np.arange(rows.size), np.asarray(y_b)[rows].astype(np.int64)]
    return lp.sum() / t, rows, lsm


def backprop_rows(H_rows, W, y_rows, lsm, s):
    """Backward of s * (-sum_i log p_i) through the head for the masked rows:
    dZ = s (softmax - onehot(y)), dX_rows = dZ W^T, dW = H_rows^T dZ."""
    y = np.asarray(y_rows).astype(np.int64)
    dZ = s * np.exp(lsm)
    dZ[np.arange(y.size), y] -= s
    return dZ @ W.T, H_rows.T @ dZ


def elbo_literal(p: Problem, hidden_bits, W_bits, targets, resp_mask, adv,
                 ell_old=None, loss_scale=1.0 / 8, backward=True) -> Result:
    """Algorithm 1's inner loops taken literally on bf16 inputs (widened exactly)."""
    return elbo_literal_f64(p, bf16_to_f64(hidden_bits).reshape(p.B, p.L, p.d),
                            bf16_to_f64(W_bits).reshape(p.d, p.V), targets, resp_mask, adv,
                            ell_old=ell_old, loss_scale=loss_scale, backward=backward)


def elbo_literal_f64(p: Problem, H, W, targets, resp_mask, adv,
                     ell_old=None, loss_scale=1.0 / 8, backward=True) -> Result:
    """Algorithm 1's inner loops taken literally: for every (j, b) draw the mask,
    run the head on the masked rows, form l, d, g and the loss term, and
    back-propagate it, accumulating dX and dW.  H [B, L, d] and W [d, V] are
    float64.  Slow; meant for small sizes."""
    ell = np.zeros((p.B, p.n_t))
    g = np.zeros((p.B, p.n_t))
    nm = np.zeros((p.B, p.n_t), dtype=np.int64)
    tt = np.zeros((p.B, p.n_t))
    dX = np.zeros((p.B, p.L, p.d)) if backward else None
    dW = np.zeros((p.d, p.V)) if backward else None
    loss = 0.0
    idx_all = {}
    dbar = np.zeros(p.B)
    if p.bound == BOUND_EXACT:
        # the exact objective couples the samples through mean_j d_j: a first
        # pass over all n_t samples gives it (Eq. elbo_ratio)
        if list(p.js) != list(range(p.n_t)):
            raise ValueError("the exact objective needs the full sample range")
        first = elbo_literal_f64(dataclasses.replace(p, bound=BOUND_PAPER), H, W, targets,
                                 resp_mask, adv, ell_old=ell_old, backward=False)
        d_all = first.ell - (0.0 if ell_old is None else np.asarray(ell_old, dtype=np.float64))
        dbar = d_all.mean(axis=1)
    for j in p.js:
        T, t, m, idx = sample_masks(p, resp_mask, j)
        idx_all[j] = idx
        for b in range(p.B):
            tt[b, j] = t[b]
            ell[b, j], rows, lsm = ell_of_mask(H[b], W, targets[b], m[b], t[b])
            nm[b, j] = rows.size
            dj = 0.0 if ell_old is None else ell[b, j] - float(ell_old[b, j])
            g[b, j], dg = bound_term(dj, float(adv[b]), p.n_t, p.bound, float(dbar[b]))
            loss += -loss_scale * g[b, j]
            if backward and rows.size:
                s = loss_scale * dg / t[b]
                gx, gw = backprop_rows(H[b, rows], W, np.asarray(targets[b])[rows], lsm, s)
                dX[b, rows] += gx
                dW += gw
    return Result(ell, g, nm, tt, loss, dX, dW, idx_all)


@dataclasses.dataclass
class SampleResult(Result):
    dgamma: Optional[np.ndarray] = None   # [d] float64 (with the final norm)


def elbo_per_sample(p: Problem, X, W, targets, resp_mask, adv, ell_old=None,
                    loss_scale=1.0 / 8, backward=True, gamma=None, eps=1e-6,
                    per_sample=True, head_bf16=False) -> SampleResult:
    """Algorithm 1's inner step with the mask predictor's output taken per
    sample: sample j (q = j - j_begin) has its own activations X[q] [B, L, d]
    (per_sample) or all samples share X [B, L, d].  With ``gamma`` the head
    input is the final RMSNorm of X (see ``oracle.rmsnorm``) and the gradients
    are those w.r.t. the norm's input and weight; ``head_bf16`` rounds the
    norm's output to bfloat16 before the head (the head's operand precision),
    the rounding passed through unchanged in the backward.  dX has the layout
    of X.  Float64 inputs; literal loops, small sizes only."""
    js = list(p.js)
    X = np.asarray(X, dtype=np.float64)
    Xq = (lambda q: X[q]) if per_sample else (lambda q: X)
    if gamma is None:
        Hq = Xq
    elif head_bf16:
        Hq = lambda q: _rms.round_to_bf16(_rms.rmsnorm(Xq(q), gamma, eps)[0])
    else:
        Hq = lambda q: _rms.rmsnorm(Xq(q), gamma, eps)[0]
    ell = np.zeros((p.B, p.n_t))
    g = np.zeros((p.B, p.n_t))
    nm = np.zeros((p.B, p.n_t), dtype=np.int64)
    tt = np.zeros((p.B, p.n_t))
    dX = np.zeros_like(X) if backward else None
    dW = np.zeros((p.d, p.V)) if backward else None
    dgamma = np.zeros(p.d) if (backward and gamma is not None) else None
    loss = 0.0
    idx_all = {}
    dbar = np.zeros(p.B)
    masks = {j: sample_masks(p, resp_mask, j) for j in js}
    if p.bound == BOUND_EXACT:
        # mean_j d_j over all samples first (Eq. elbo_ratio)
        if js != list(range(p.n_t)):
            raise ValueError("the exact objective needs the full sample range")
        for q, j in enumerate(js):
            for b in range(p.B):
                ell[b, j] = ell_of_mask(Hq(q)[b], W, targets[b], masks[j][2][b], masks[j][1][b])[0]
        dbar = (ell - (0.0 if ell_old is None else np.asarray(ell_old, dtype=np.float64))).mean(axis=1)
    for q, j in enumerate(js):
        T, t, m, idx = masks[j]
        idx_all[j] = idx
        H = Hq(q)
        dH = np.zeros_like(H) if backward else None
        for b in range(p.B):
            tt[b, j] = t[b]
            ell[b, j], rows, lsm = ell_of_mask(H[b], W, targets[b], m[b], t[b])
            nm[b, j] = rows.size
            dj = 0.0 if ell_old is None else ell[b, j] - float(ell_old[b, j])
            g[b, j], dg = bound_term(dj, float(adv[b]), p.n_t, p.bound, float(dbar[b]))
            loss += -loss_scale * g[b, j]
            if backward and rows.size:
                s = loss_scale * dg / t[b]
                gx, gw = backprop_rows(H[b, rows], W, np.asarray(targets[b])[rows], lsm, s)
                dH[b, rows] += gx
                dW += gw
        if backward:
            if gamma is not None:
                gx, gg = _rms.rmsnorm_backward(Xq(q), gamma, eps, dH)
                dgamma += gg
            else:
                gx = dH
            if per_sample:
                dX[q] += gx
            else:
                dX += gx
    return SampleResult(ell, g, nm, tt, loss, dX, dW, idx_all, dgamma)


def elbo_collapsed(p: Problem, hidden_bits, W_bits, targets, resp_mask, adv,
                   ell_old=None, loss_scale=1.0 / 8, backward=True,
                   dx_rows=None, dw_cols=None, row_chunk=256, hidden_f64=None) -> Result:
    """Same result for hidden states shared by all samples (the head-only slice).

    The log-softmax is computed once per response position; l_{b,j} is then the
    masked, 1/t-weighted sum of those values, and by linearity the accumulated
    backward is one pass with per-position weight w_{b,i} = sum_j s_{b,j} m_{b,j,i}.
    ``dx_rows`` (flat positions) and ``dw_cols`` (vocabulary ids) restrict the
    gradients to a subset, which is what makes full-size problems tractable:
    dX is returned as [len(dx_rows), d] and dW as [d, len(dw_cols)].
    ``hidden_f64`` [B, L, d] replaces the bf16 hidden states (e.g. the float64
    output of the final RMSNorm); dX is then the gradient w.r.t. it."""
    H = (bf16_to_f64(hidden_bits) if hidden_f64 is None else np.asarray(hidden_f64, dtype=np.float64)
         ).reshape(p.B * p.L, p.d)
    tg = targets.reshape(-1).astype(np.int64)
    resp = resp_mask.reshape(-1) != 0

    # masks of every sample first: only positions masked in at least one sample
    # of the range enter l or the gradients, so only those need a log-softmax
    masks = {}
    for j in p.js:
        masks[j] = sample_masks(p, resp_mask, j)
    used = np.zeros(p.B * p.L, dtype=bool)
    for j in p.js:
        used |= masks[j][2].reshape(-1)
    if dx_rows is not None:
        used[np.asarray(dx_rows, dtype=np.int64)] |= resp[np.asarray(dx_rows, dtype=np.int64)]
    pos = np.flatnonzero(used)

    W = bf16_to_f64(W_bits).reshape(p.d, p.V)
    lse = np.zeros(p.B * p.L)
    lp = np.zeros(p.B * p.L)
    for c0 in range(0, pos.size, row_chunk):
        rows = pos[c0:c0 + row_chunk]
        z = H[rows] @ W
        mx = z.max(axis=1)
        lse[rows] = mx + np.log(np.exp(z - mx[:, None]).sum(axis=1))
        lp[rows] = z[np.arange(rows.size), tg[rows]] - lse[rows]
    del W

    ell = np.zeros((p.B, p.n_t))
    g = np.zeros((p.B, p.n_t))
    nm = np.zeros((p.B, p.n_t), dtype=np.int64)
    tt = np.zeros((p.B, p.n_t))
    wpos = np.zeros(p.B * p.L)
    loss = 0.0
    idx_all = {}
    lp2 = lp.reshape(p.B, p.L)
    for j in p.js:
        T, t, m, idx = masks[j]
        idx_all[j] = idx
        for b in range(p.B):
            tt[b, j] = t[b]
            nm[b, j] = int(m[b].sum())
            ell[b, j] = lp2[b][m[b]].sum() / t[b]
    dbar = np.zeros(p.B)
    if p.bound == BOUND_EXACT:
        if list(p.js) != list(range(p.n_t)):
            raise ValueError("the exact objective needs the full sample range")
        dbar = (ell - (0.0 if ell_old is None else np.asarray(ell_old, dtype=np.float64))).mean(axis=1)
    for j in p.js:
        T, t, m, idx = masks[j]
        for b in range(p.B):
            dj = 0.0 if ell_old is None else ell[b, j] - float(ell_old[b, j])
            g[b, j], dg = bound_term(dj, float(adv[b]), p.n_t, p.bound, float(dbar[b]))
            loss += -loss_scale * g[b, j]
            wpos[b * p.L:(b + 1) * p.L] += (loss_scale * dg / t[b]) * m[b]

    dX = dW = None
    if backward:
        W = bf16_to_f64(W_bits).reshape(p.d, p.V)
        xr = pos if dx_rows is None else np.asarray(dx_rows, dtype=np.int64)
        dX = np.zeros((xr.size, p.d))
        for c0 in range(0, xr.size, row_chunk):
            rows = xr[c0:c0 + row_chunk]
            z = H[rows] @ W
            dZ = wpos[rows, None] * np.exp(z - lse[rows, None])
            dZ[np.arange(rows.size), tg[rows]] -= wpos[rows]
            dX[c0:c0 + rows.size] = dZ @ W.T
        if dx_rows is None:
            full = np.zeros((p.B * p.L, p.d))
            full[xr] = dX
            dX = full.reshape(p.B, p.L, p.d)
        cols = np.arange(p.V) if dw_cols is None else np.asarray(dw_cols, dtype=np.int64)
        act = pos[wpos[pos] != 0.0]
        Wc = W[:, cols]
        del W
        dW = np.zeros((p.d, cols.size))
        for c0 in range(0, act.size, 4 * row_chunk):
            rows = act[c0:c0 + 4 * row_chunk]
            z = H[rows] @ Wc
            dZ = wpos[rows, None] * np.exp(z - lse[rows, None])
            hit = tg[rows, None] == cols[None, :]
            dZ -= wpos[rows, None] * hit
            dW += H[rows].T @ dZ
    return Result(ell, g, nm, tt, loss, dX, dW, idx_all)
