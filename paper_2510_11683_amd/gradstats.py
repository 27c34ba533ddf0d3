"""Gradient standard deviation and bias against the Monte-Carlo sample size.

The procedure of Section 4 "Effect of Increasing MC Sample Sizes" (Figure
grad_time, left and middle), on the ELBO head: for every n_t the gradient of
one batch is computed `repeats` times with independent Monte-Carlo samples
(Philox seeds base + r); the per-parameter sample standard deviation across
the repeats and the absolute deviation of the repeats' mean from a reference
gradient computed with n_t = 256 (another seed) are averaged over the
parameters.  On-policy, as in the paper (the loss value itself is zero there).
Parameters: the LM-head weights (dW) and, as the gradient passed back into the
mask predictor, the hidden states (dX).

Every gradient comes from bgpo_elbo_bwd_accumulate and every statistic from
the library's moment kernels; this module only sequences the calls.

    python -m paper_2510_11683_amd.gradstats --workload llada_head_B8_L512_nt64
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import torch

from . import bgpo

N_T_LIST = (1, 2, 4, 8, 16, 32, 64)
REPEATS = 8
GOLDEN_N_T = 256
GOLDEN_SEED_OFFSET = 10_000


def run(w, x, n_t_list=N_T_LIST, repeats=REPEATS, golden_n_t=GOLDEN_N_T, loss_scale=1.0 / 8):
    """Returns {"golden_n_t", "repeats", "rows": [{n_t, dW: {std, bias, ref}, dX: {...}}], "seconds"}."""
    dev = bgpo.device_inputs(x)
    B, L, d, V = w.B, w.L, w.d, w.V

    def prob(n_t, seed):
        return bgpo.Problem(B, L, d, V, n_t, seed=seed, seq_id_base=w.seq_id_base, t_mode=w.t_mode)

    ws = bgpo.alloc_workspace(prob(1, 0))            # workspace does not depend on n_t
    mws = bgpo.moments_workspace()
    grads = {"dW": torch.zeros(d, V, dtype=torch.float32, device="cuda"),
             "dX": torch.zeros(B, L, d, dtype=torch.float32, device="cuda")}
    loss = torch.zeros(1, dtype=torch.float64, device="cuda")
    flags = torch.zeros(1, dtype=torch.int32, device="cuda")

    def gradient(n_t, seed):
        for gr in grads.values():
            gr.zero_()
        ell = torch.zeros(B, n_t, dtype=torch.float64, device="cuda")
        g = torch.zeros_like(ell)
        nm = torch.zeros(B, n_t, dtype=torch.int32, device="cuda")
        bgpo.bgpo_elbo_bwd_accumulate(prob(n_t, seed), dev["hidden"], dev["W"], dev["targets"],
                                      dev["resp_mask"], dev["adv"], None, loss_scale, grads["dX"],
                                      grads["dW"], ell, g, loss, nm, None, flags, ws)

    t0 = time.perf_counter()
    gradient(golden_n_t, w.philox_seed + GOLDEN_SEED_OFFSET)
    golden = {k: v.clone() for k, v in grads.items()}
    mom = {k: (torch.zeros_like(v), torch.zeros_like(v)) for k, v in grads.items()}
    out = torch.zeros(3, dtype=torch.float64, device="cuda")
    rows = []
    for n_t in n_t_list:
        for mean, m2 in mom.values():
            mean.zero_()
            m2.zero_()
        for r in range(repeats):
            gradient(n_t, w.philox_seed + r)
            for k, (mean, m2) in mom.items():
                bgpo.bgpo_moments_update(grads[k], mean, m2, r)
        row = {"n_t": n_t}
        for k, (mean, m2) in mom.items():
            bgpo.bgpo_moments_summary(mean, m2, golden[k], repeats, out, mws)
            std, bias, ref = (float(v) for v in out.cpu())
            row[k] = {"std": std, "bias": bias, "ref": ref}
        rows.append(row)
    torch.cuda.synchronize()
    if int(flags.item()):
        raise RuntimeError("non-finite values flagged during the gradient runs")
    return {"golden_n_t": golden_n_t, "repeats": repeats, "rows": rows,
            "seconds": time.perf_counter() - t0}


def main():
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    sys.path.insert(0, root)
    import workloads
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default=workloads.LLADA_L512_NT64.name,
                    choices=sorted(w.name for w in workloads.CONFIGS))
    ap.add_argument("--repeats", type=int, default=REPEATS)
    ap.add_argument("--golden-n-t", type=int, default=GOLDEN_N_T)
    args = ap.parse_args()
    w = {c.name: c for c in workloads.CONFIGS}[args.workload]
    res = run(w, workloads.generate(w), repeats=args.repeats, golden_n_t=args.golden_n_t)
    res["workload"] = w.name
    print(json.dumps(res))


if __name__ == "__main__":
    main()
