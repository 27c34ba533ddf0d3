"""Float64 reference of the gradient statistics against n_t (Section 4
"Effect of Increasing MC Sample Sizes", Figure grad_time left and middle).

TEST INFRASTRUCTURE: part of the oracle; see ``oracle/__init__.py``.

For every n_t: the batch's gradient with Monte-Carlo seeds base + r, r <
repeats; per parameter the sample standard deviation over the repeats
(ddof = 1) and |mean over the repeats - reference|, the reference being the
gradient with n_t = golden_n_t and seed base + 10000; both averaged over all
parameters.  On-policy (ell_old absent).
"""
from __future__ import annotations

import dataclasses

import numpy as np

from . import elbo


def moments_summary(G: np.ndarray, ref: np.ndarray):
    """G [repeats, ...] estimates, ref [...]: (mean std, mean |bias|, mean |ref|)."""
    G = np.asarray(G, dtype=np.float64)
    std = np.std(G, axis=0, ddof=1) if G.shape[0] > 1 else np.zeros(G.shape[1:])
    return float(std.mean()), float(np.abs(G.mean(axis=0) - ref).mean()), float(np.abs(ref).mean())


def gradient(p: elbo.Problem, x: dict, loss_scale=1.0 / 8):
    r = elbo.elbo_collapsed(p, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                            loss_scale=loss_scale)
    return r.dW, r.dX


def run(w, x, n_t_list, repeats, golden_n_t, loss_scale=1.0 / 8):
    base = elbo.Problem(w.B, w.L, w.d, w.V, 1, seed=w.philox_seed, seq_id_base=w.seq_id_base,
                        t_mode=w.t_mode)
    gW, gX = gradient(dataclasses.replace(base, n_t=golden_n_t, seed=w.philox_seed + 10_000), x,
                      loss_scale)
    rows = []
    for n_t in n_t_list:
        Ws, Xs = [], []
        for r in range(repeats):
            dW, dX = gradient(dataclasses.replace(base, n_t=n_t, seed=w.philox_seed + r), x, loss_scale)
            Ws.append(dW)
            Xs.append(dX)
        rows.append({"n_t": n_t,
                     "dW": dict(zip(("std", "bias", "ref"), moments_summary(np.stack(Ws), gW))),
                     "dX": dict(zip(("std", "bias", "ref"), moments_summary(np.stack(Xs), gX)))})
    return {"golden_n_t": golden_n_t, "repeats": repeats, "rows": rows}
