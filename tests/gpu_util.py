"""Helpers for the GPU parity tests: run the HIP path through the C ABI on
workload inputs and bring the outputs back as numpy arrays."""
import numpy as np
import torch

import workloads


def lib():
    from paper_2510_11683_amd import bgpo
    return bgpo


def problem(w: workloads.Workload, j_begin=0, j_count=None, n_t=None, bound=0, **kw):
    """The C-ABI problem of workload w; kw sets further fields (in_dtype,
    vocab_chunk, ws_budget, ...)."""
    b = lib()
    return b.Problem(w.B, w.L, w.d, w.V, w.n_t if n_t is None else n_t, j_begin=j_begin,
                     j_count=j_count, seed=w.philox_seed, seq_id_base=w.seq_id_base,
                     t_mode=w.t_mode, bound=bound, **kw)


class Runner:
    """Device buffers for one workload; calls accumulate into dX / dW / loss.
    ``kw`` are problem fields used by every call (e.g. vocab_chunk,
    ws_budget, in_dtype; with in_dtype = BGPO_F32 the fp32 arrays
    ``hidden_f32`` / ``W_f32`` of x are passed)."""

    def __init__(self, w: workloads.Workload, x: dict, device="cuda", **kw):
        b = lib()
        self.w = w
        self.kw = kw
        self.dev = b.device_inputs(x, device)
        if kw.get("in_dtype", 0) == b.BGPO_F32:
            self.dev["hidden"] = torch.from_numpy(x["hidden_f32"]).to(device)
            self.dev["W"] = torch.from_numpy(x["W_f32"]).to(device)
        self.ws = b.alloc_workspace(problem(w, **kw), device)
        B, L, d, V, nt = w.B, w.L, w.d, w.V, w.n_t
        self.dX = torch.zeros(B, L, d, dtype=torch.float32, device=device)
        self.dW = torch.zeros(d, V, dtype=torch.float32, device=device)
        self.ell = torch.zeros(B, nt, dtype=torch.float64, device=device)
        self.g = torch.zeros(B, nt, dtype=torch.float64, device=device)
        self.loss = torch.zeros(1, dtype=torch.float64, device=device)
        self.nm = torch.zeros(B, nt, dtype=torch.int32, device=device)
        self.t = torch.zeros(B, nt, dtype=torch.float32, device=device)
        self.flags = torch.zeros(1, dtype=torch.int32, device=device)

    def zero_grads(self):
        self.dX.zero_()
        self.dW.zero_()
        self.loss.zero_()

    def fwd(self, j_begin=0, j_count=None, timing=None):
        b = lib()
        d = self.dev
        b.bgpo_elbo_fwd(problem(self.w, j_begin, j_count, **self.kw), d["hidden"], d["W"], d["targets"],
                        d["resp_mask"], self.ell, self.nm, self.t, self.ws, timing=timing)

    def bwd(self, j_begin=0, j_count=None, ell_old=None, loss_scale=1.0 / 8, timing=None, bound=0):
        b = lib()
        d = self.dev
        eo = None if ell_old is None else torch.as_tensor(ell_old, dtype=torch.float64).cuda().contiguous()
        b.bgpo_elbo_bwd_accumulate(problem(self.w, j_begin, j_count, bound=bound, **self.kw),
                                   d["hidden"], d["W"],
                                   d["targets"], d["resp_mask"], d["adv"], eo, loss_scale,
                                   self.dX, self.dW, self.ell, self.g, self.loss, self.nm, self.t,
                                   self.flags, self.ws, timing=timing)

    def out(self):
        torch.cuda.synchronize()
        return dict(ell=self.ell.cpu().numpy(), g=self.g.cpu().numpy(), loss=float(self.loss.item()),
                    nm=self.nm.cpu().numpy(), t=self.t.cpu().numpy(),
                    dX=self.dX.cpu().numpy(), dW=self.dW.cpu().numpy(),
                    flags=int(self.flags.item()))


def rel_maxnorm(a, ref):
    """max |a - ref| / max |ref| (the relative max-norm error)."""
    den = float(np.abs(ref).max())
    return float(np.abs(np.asarray(a, dtype=np.float64) - ref).max()) / (den if den > 0 else 1.0)
