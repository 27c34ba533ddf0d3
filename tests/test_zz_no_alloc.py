"""The allocation-free backward (bgpo_elbo_bwd_accumulate_noalloc) against the
workspace entry point with the same layout: two calls in a row on the shared
static scratch, the second with a smaller problem, each bit-identical to the
workspace call; problems whose layout exceeds the scratch are refused before
anything runs (tested on the CPU in test_abi)."""
import numpy as np
import pytest
import torch

import workloads
from gpu_util import lib, problem

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lib()


def _buffers(w, x):
    b = lib()
    dev = b.device_inputs(x)
    f = dict(device="cuda")
    out = dict(dX=torch.zeros(w.B, w.L, w.d, dtype=torch.float32, **f),
               dW=torch.zeros(w.d, w.V, dtype=torch.float32, **f),
               ell=torch.zeros(w.B, w.n_t, dtype=torch.float64, **f),
               g=torch.zeros(w.B, w.n_t, dtype=torch.float64, **f),
               loss=torch.zeros(1, dtype=torch.float64, **f),
               nm=torch.zeros(w.B, w.n_t, dtype=torch.int32, **f),
               t=torch.zeros(w.B, w.n_t, dtype=torch.float32, **f),
               flags=torch.zeros(1, dtype=torch.int32, **f))
    return dev, out


def _run(w, x, ell_old, noalloc):
    b = lib()
    scratch = b.bgpo_noalloc_scratch_bytes()
    p = problem(w, ws_budget=scratch)
    dev, o = _buffers(w, x)
    eo = torch.from_numpy(ell_old).cuda()
    args = (dev["hidden"], dev["W"], dev["targets"], dev["resp_mask"], dev["adv"], eo, 0.25,
            o["dX"], o["dW"], o["ell"], o["g"], o["loss"], o["nm"], o["t"], o["flags"])
    for _ in range(2):                                    # accumulates twice
        if noalloc:
            b.bgpo_elbo_bwd_accumulate_noalloc(p, *args)
        else:
            ws = b.alloc_workspace(p)
            assert ws.numel() <= scratch
            b.bgpo_elbo_bwd_accumulate(p, *args, ws)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in o.items()}


def test_noalloc_matches_workspace_entry_point_twice_then_smaller():
    from test_gpu_parity import MID
    cases = [MID.replace(n_t=4), workloads.TINY.replace(n_t=5)]   # the second is smaller
    rng = np.random.default_rng(51)
    for w in cases:
        x = workloads.generate(w)
        ell_old = rng.normal(-400.0, 30.0, (w.B, w.n_t))       # off-policy, both branches
        ref = _run(w, x, ell_old, noalloc=False)
        got = _run(w, x, ell_old, noalloc=True)
        for k in ref:
            assert np.array_equal(got[k], ref[k]), (w.name, k)
        assert np.abs(got["dW"]).max() > 0 and got["flags"][0] == 0


def test_noalloc_under_graph_capture():
    """The allocation-free backward under HIP graph capture (the callers it is
    for): captured after one eager call, replayed twice with eager zeroing in
    between; every replay gives the workspace entry point's bits."""
    from test_gpu_parity import MID
    b = lib()
    w = MID.replace(n_t=3)
    x = workloads.generate(w)
    ell_old = np.random.default_rng(52).normal(-400.0, 30.0, (w.B, w.n_t))
    ref = _run(w, x, ell_old, noalloc=False)
    p = problem(w, ws_budget=b.bgpo_noalloc_scratch_bytes())
    dev, o = _buffers(w, x)
    eo = torch.from_numpy(ell_old).cuda()
    args = (dev["hidden"], dev["W"], dev["targets"], dev["resp_mask"], dev["adv"], eo, 0.25,
            o["dX"], o["dW"], o["ell"], o["g"], o["loss"], o["nm"], o["t"], o["flags"])
    b.bgpo_elbo_bwd_accumulate_noalloc(p, *args)          # the device's scratch address, once
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        b.bgpo_elbo_bwd_accumulate_noalloc(p, *args)
        b.bgpo_elbo_bwd_accumulate_noalloc(p, *args)       # accumulates twice, as _run does
    for _ in range(2):
        for k in ("dX", "dW", "loss", "ell", "g", "nm", "t", "flags"):
            o[k].zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = {k: v.cpu().numpy() for k, v in o.items()}
        for k in ref:
            assert np.array_equal(got[k], ref[k]), k
