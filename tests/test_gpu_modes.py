"""Parity of the input-type and backward modes of the C ABI.

* fp32 inputs (in_dtype = BGPO_F32): the device rounds hidden / x and W_head
  to bf16 (nearest even) as it reads them, so every output is bit-identical
  to a bf16 call on the host-rounded inputs (the tiny workload is drawn in
  fp32), with and without the final RMSNorm, and matches the oracle on the
  rounded values.
* The recompute backward (vocabulary chunks; chosen by a small workspace
  budget or forced with vocab_chunk): the float64 oracle off-policy with both
  bound branches, ragged last chunks, chunks wider than the vocabulary, the
  exact objective, per-sample inputs through the norm; l bit-identical to the
  stored backward (same forward), dX and dW close to it; deterministic reruns
  and linear in the sample range.
"""
import dataclasses

import numpy as np
import pytest
import torch

import workloads
from oracle import elbo
from gpu_util import Runner, lib, problem, rel_maxnorm
from test_gpu_parity import MID, _check_against_oracle, _oracle_problem

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lib()


def _off_policy_ell_old(w, x, seed, scale=1.0, bound=0):
    op = dataclasses.replace(_oracle_problem(w), bound=bound)
    ell = elbo.elbo_literal(op, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                            backward=False).ell
    return ell + np.random.default_rng(seed).normal(0, scale, ell.shape)


# ---------------------------------------------------------------- fp32 inputs

def test_fp32_inputs_tiny_bit_identical_to_host_rounding():
    w = workloads.TINY
    x = workloads.generate(w, keep_f32=True)
    b = lib()
    ell_old = _off_policy_ell_old(w, x, 21, 0.5)
    outs = []
    for kw in ({}, {"in_dtype": b.BGPO_F32}):
        r = Runner(w, x, **kw)
        r.fwd()
        f = r.out()
        r.bwd(ell_old=ell_old)
        outs.append((f, r.out()))
    (f16, b16), (f32, b32) = outs
    for k in ("ell", "nm", "t"):
        assert np.array_equal(f16[k], f32[k]), k
    for k in ("ell", "g", "nm", "t", "dX", "dW"):
        assert np.array_equal(b16[k], b32[k]), k
    assert b16["loss"] == b32["loss"]
    ref = elbo.elbo_literal(_oracle_problem(w), x["hidden"], x["W"], x["targets"], x["resp_mask"],
                            x["adv"], ell_old=ell_old)
    _check_against_oracle(w, b32, ref, range(w.n_t), x["adv"], ell_old)


def test_fp32_inputs_rmsnorm_bit_identical_to_host_rounding():
    """fp32 pre-norm activations and head weights through the fused final
    RMSNorm (per-sample activations, off-policy): dx, dgamma, dW, l, g
    bit-identical to the bf16 call on the rounded values."""
    b = lib()
    w = MID.replace(n_t=3)
    x = workloads.generate(w, keep_f32=True)
    rng = np.random.default_rng(31)
    x32 = (rng.standard_normal((w.n_t, w.B, w.L, w.d)) *
           np.exp(rng.uniform(-1, 1, (w.n_t, w.B, w.L, 1)))).astype(np.float32)
    x16 = workloads.f32_to_bf16_bits(x32).reshape(x32.shape)
    gamma = torch.from_numpy(workloads.norm_weight(w)).cuda()
    ell_old = torch.from_numpy(np.random.default_rng(32).normal(-900.0, 50.0, (w.B, w.n_t))).cuda()
    res = []
    for f32 in (False, True):
        p = problem(w, sample_stride=w.B * w.L * w.d, in_dtype=b.BGPO_F32 if f32 else b.BGPO_BF16)
        ws = b.alloc_workspace(p)
        xs = (torch.from_numpy(x32) if f32 else torch.from_numpy(x16.view(np.int16)).view(torch.bfloat16)).cuda()
        W = (torch.from_numpy(x["W_f32"]) if f32 else
             torch.from_numpy(x["W"].view(np.int16)).view(torch.bfloat16)).cuda()
        dev = b.device_inputs(x)
        dx = torch.zeros(w.n_t, w.B, w.L, w.d, dtype=torch.float32, device="cuda")
        dgam = torch.zeros(w.d, dtype=torch.float32, device="cuda")
        dW = torch.zeros(w.d, w.V, dtype=torch.float32, device="cuda")
        ell = torch.zeros(w.B, w.n_t, dtype=torch.float64, device="cuda")
        g = torch.zeros_like(ell)
        loss = torch.zeros(1, dtype=torch.float64, device="cuda")
        nm = torch.zeros(w.B, w.n_t, dtype=torch.int32, device="cuda")
        b.bgpo_elbo_bwd_accumulate_rmsnorm(p, xs, gamma, W, dev["targets"], dev["resp_mask"],
                                           dev["adv"], ell_old, 0.25, dx, dgam, dW, ell, g, loss,
                                           nm, None, None, ws)
        torch.cuda.synchronize()
        res.append([t.cpu().numpy() for t in (dx, dgam, dW, ell, g, loss, nm)])
    for a, c in zip(*res):
        assert np.array_equal(a, c)
    assert np.abs(res[0][0]).max() > 0


def test_fp32_inputs_recompute_bit_identical_to_bf16():
    """The recompute mode's dX GEMM reads a bf16 W_head in place (row-major)
    and an fp32 one from its slab-major bf16 copy: the same products in the
    same order, so dX and dW agree bit for bit (MID, chunks of 1024: 4 full
    and a last one of 192 ids)."""
    b = lib()
    w = MID
    x = workloads.generate(w, keep_f32=True)
    ell_old = _off_policy_ell_old(w, x, 43, 2.0)
    outs = []
    for kw in ({}, {"in_dtype": b.BGPO_F32}):
        assert b.bgpo_workspace_plan(problem(w, vocab_chunk=1024, **kw))["mode"] == "recompute"
        r = Runner(w, x, vocab_chunk=1024, **kw)
        r.bwd(ell_old=ell_old)
        outs.append(r.out())
    for k in ("ell", "g", "nm", "t", "dX", "dW"):
        assert np.array_equal(outs[0][k], outs[1][k]), k
    assert np.abs(outs[0]["dW"]).max() > 0


def test_stored_without_the_w_copy_bit_identical():
    """A budget just below the default layout keeps its units, dW batch and
    split capacity and drops the slab-major copy of W (the dX GEMM then reads
    W_head row-major): the same products in the same order, so every output
    is bit-identical to the default layout's (tiny, off-policy)."""
    b = lib()
    w = workloads.TINY
    x = workloads.generate(w)
    dflt = b.bgpo_workspace_plan(problem(w))
    tight = b.bgpo_workspace_plan(problem(w, ws_budget=dflt["workspace_bytes"] - 1))
    assert dflt["w_copy"] == 1 and tight["w_copy"] == 0
    for k in ("samples_per_unit", "dw_batch", "dx_splits", "vocab_chunk"):
        assert tight[k] == dflt[k], k
    ell_old = _off_policy_ell_old(w, x, 45, 0.5)
    outs = []
    for kw in ({}, {"ws_budget": dflt["workspace_bytes"] - 1}):
        r = Runner(w, x, **kw)
        r.bwd(ell_old=ell_old)
        outs.append(r.out())
    for k in ("ell", "g", "nm", "t", "dX", "dW"):
        assert np.array_equal(outs[0][k], outs[1][k]), k
    assert outs[0]["loss"] == outs[1]["loss"]


# ---------------------------------------------------------------- recompute backward

@pytest.mark.parametrize("chunk", [256, 1024, 4096, 8192], ids=lambda c: f"chunk{c}")
def test_recompute_mid_off_policy_both_branches(chunk):
    """MID: V = 4288 in chunks of 256 (17 chunks, last of 192), 1024 (4 + 192),
    4096 (1 + 192) and 8192 (one chunk wider than the vocabulary)."""
    w = MID
    x = workloads.generate(w)
    ell_old = _off_policy_ell_old(w, x, 41, 2.0)
    ref = elbo.elbo_literal(_oracle_problem(w), x["hidden"], x["W"], x["targets"],
                            x["resp_mask"], x["adv"], ell_old=ell_old, loss_scale=0.25)
    r = Runner(w, x, vocab_chunk=chunk)
    assert lib().bgpo_workspace_plan(problem(w, vocab_chunk=chunk))["mode"] == "recompute"
    r.bwd(ell_old=ell_old, loss_scale=0.25)
    rec = r.out()
    _check_against_oracle(w, rec, ref, range(w.n_t), x["adv"], ell_old, 0.25)
    s = Runner(w, x)
    s.bwd(ell_old=ell_old, loss_scale=0.25)
    sto = s.out()
    for k in ("ell", "g", "nm", "t"):
        assert np.array_equal(rec[k], sto[k]), k          # same forward, same l
    assert rel_maxnorm(rec["dX"], sto["dX"]) <= 1e-2
    assert rel_maxnorm(rec["dW"], sto["dW"]) <= 1e-2


def test_recompute_chosen_by_budget_tiny_and_exact_objective():
    """A budget below every stored layout picks the recompute backward; the
    exact objective (its forward pass over all samples first) matches the
    oracle there too."""
    b = lib()
    w = workloads.TINY.replace(n_t=6)
    x = workloads.generate(w)
    stored_min = b.bgpo_workspace_plan(problem(w, ws_budget=1 << 40))["workspace_bytes"]
    budget = None
    for cand in range(stored_min, 0, -(1 << 14)):
        try:
            plan = b.bgpo_workspace_plan(problem(w, ws_budget=cand))
        except b.BgpoError:
            break
        if plan["mode"] == "recompute":
            budget = cand
            break
    assert budget is not None
    ell_old = _off_policy_ell_old(w, x, 43, 1.0, bound=3)
    op = dataclasses.replace(_oracle_problem(w), bound=3)
    ref = elbo.elbo_literal(op, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                            ell_old=ell_old, loss_scale=0.25)
    r = Runner(w, x, ws_budget=budget)
    assert r.ws.numel() <= budget
    r.bwd(ell_old=ell_old, loss_scale=0.25, bound=3)
    _check_against_oracle(w, r.out(), ref, range(w.n_t), x["adv"], ell_old, 0.25, 3)


@pytest.mark.parametrize("B,L,d,V,n_t", [(1, 1, 64, 64, 3), (2, 70, 128, 320, 2)],
                         ids=["B1_L1_d64_V64", "B2_L70_d128_V320"])
def test_recompute_smallest_shapes(B, L, d, V, n_t):
    w = workloads.TINY.replace(B=B, L=L, d=d, V=V, n_t=n_t, adv="normal", data_seed=2200 + B * L)
    x = workloads.generate(w)
    ell_old = _off_policy_ell_old(w, x, 44, 0.5)
    ref = elbo.elbo_literal(_oracle_problem(w), x["hidden"], x["W"], x["targets"],
                            x["resp_mask"], x["adv"], ell_old=ell_old, loss_scale=0.25)
    r = Runner(w, x, vocab_chunk=256)
    r.bwd(ell_old=ell_old, loss_scale=0.25)
    _check_against_oracle(w, r.out(), ref, range(w.n_t), x["adv"], ell_old, 0.25)


def test_recompute_linearity_and_determinism():
    w = MID.replace(n_t=4)
    x = workloads.generate(w)
    r = Runner(w, x, vocab_chunk=1024)
    r.bwd()
    full = r.out()
    r.zero_grads()
    r.bwd()
    again = r.out()
    for k in ("dX", "dW", "ell", "g"):
        assert np.array_equal(full[k], again[k]), k
    assert full["loss"] == again["loss"]
    r.zero_grads()
    for jb, jc in ((0, 1), (1, 2), (3, 1)):
        r.bwd(j_begin=jb, j_count=jc)
    split = r.out()
    assert np.array_equal(split["ell"], full["ell"])
    assert rel_maxnorm(split["dX"], full["dX"]) <= 1e-5
    assert rel_maxnorm(split["dW"], full["dW"]) <= 1e-5


def test_recompute_per_sample_rmsnorm_matches_stored():
    """Per-sample pre-norm activations through the norm, off-policy: the
    recompute backward gives the stored backward's l, g bit for bit and its
    dx, dgamma, dW within 1e-2 (the stored one is checked against the oracle
    in the per-sample tests)."""
    b = lib()
    w = MID.replace(n_t=3)
    x = workloads.generate(w)
    xs = torch.from_numpy(workloads.pre_norm_activations(w, w.n_t).view(np.int16)).cuda().view(torch.bfloat16)
    gamma = torch.from_numpy(workloads.norm_weight(w)).cuda()
    ell_old = torch.from_numpy(np.random.default_rng(45).normal(-900.0, 50.0, (w.B, w.n_t))).cuda()
    dev = b.device_inputs(x)
    res = []
    for kw in ({}, {"vocab_chunk": 1024}):
        p = problem(w, sample_stride=w.B * w.L * w.d, **kw)
        ws = b.alloc_workspace(p)
        dx = torch.zeros(w.n_t, w.B, w.L, w.d, dtype=torch.float32, device="cuda")
        dgam = torch.zeros(w.d, dtype=torch.float32, device="cuda")
        dW = torch.zeros(w.d, w.V, dtype=torch.float32, device="cuda")
        ell = torch.zeros(w.B, w.n_t, dtype=torch.float64, device="cuda")
        g = torch.zeros_like(ell)
        loss = torch.zeros(1, dtype=torch.float64, device="cuda")
        nm = torch.zeros(w.B, w.n_t, dtype=torch.int32, device="cuda")
        b.bgpo_elbo_bwd_accumulate_rmsnorm(p, xs, gamma, dev["W"], dev["targets"], dev["resp_mask"],
                                           dev["adv"], ell_old, 0.25, dx, dgam, dW, ell, g, loss,
                                           nm, None, None, ws)
        torch.cuda.synchronize()
        res.append({k: t.cpu().numpy() for k, t in
                    dict(dx=dx, dgam=dgam, dW=dW, ell=ell, g=g, nm=nm).items()})
    sto, rec = res
    for k in ("ell", "g", "nm"):
        assert np.array_equal(sto[k], rec[k]), k
    for k in ("dx", "dgam", "dW"):
        assert rel_maxnorm(rec[k], sto[k]) <= 1e-2, k


def test_recompute_graph_capture_replays_match_eager():
    """The recompute backward only enqueues kernels too: captured in a HIP
    graph and replayed three times (eager zeroing and a host synchronisation
    between replays), every replay gives the eager call's bits."""
    w = MID.replace(n_t=4)
    x = workloads.generate(w)
    r = Runner(w, x, vocab_chunk=1024)
    r.bwd()
    eager = r.out()
    b, d = lib(), r.dev
    prob = problem(w, vocab_chunk=1024)
    graph = torch.cuda.CUDAGraph()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        b.bgpo_elbo_bwd_accumulate(prob, d["hidden"], d["W"], d["targets"], d["resp_mask"],
                                   d["adv"], None, 1.0 / 8, r.dX, r.dW, r.ell, r.g, r.loss, r.nm,
                                   r.t, r.flags, r.ws)
    for _ in range(3):
        r.zero_grads()
        for t in (r.ell, r.g, r.nm, r.t):
            t.zero_()
        torch.cuda.synchronize()
        graph.replay()
        o = r.out()
        for k in ("ell", "g", "nm", "t", "dX", "dW"):
            assert np.array_equal(o[k], eager[k]), k
        assert o["loss"] == eager["loss"] and o["flags"] == 0


def test_retained_rmsnorm_per_sample_bit_identical_to_two_pass():
    """The exact objective off-policy through the final RMSNorm with per-sample
    activations (MID, 12 samples: two units of one dW batch), with every
    sample's state retained and in two passes: the same kernels on the same
    units, so dx, dgamma, dW, l, g and the loss agree bit for bit (the
    two-pass path is checked against the oracle in the row-f1 tests)."""
    b = lib()
    w = MID.replace(n_t=12)
    x = workloads.generate(w)
    rng = np.random.default_rng(61)
    xs = workloads.f32_to_bf16_bits(
        (rng.standard_normal((w.n_t, w.B, w.L, w.d)) *
         np.exp(rng.uniform(-1, 1, (w.n_t, w.B, w.L, 1)))).astype(np.float32))
    xs = torch.from_numpy(xs.reshape(w.n_t, w.B, w.L, w.d).view(np.int16)).view(torch.bfloat16).cuda()
    gamma = torch.from_numpy(workloads.norm_weight(w)).cuda()
    dev = b.device_inputs(x)
    # l_old near l (an input both runs share): the forward entry point's l
    # plus N(0, 1), so that the exact objective's exp(mean log-ratio) is finite
    p0 = problem(w, sample_stride=w.B * w.L * w.d)
    ell0 = torch.zeros(w.B, w.n_t, dtype=torch.float64, device="cuda")
    nm0 = torch.zeros(w.B, w.n_t, dtype=torch.int32, device="cuda")
    b.bgpo_elbo_fwd_rmsnorm(p0, xs, gamma, dev["W"], dev["targets"], dev["resp_mask"], ell0, nm0,
                            None, b.alloc_workspace(p0))
    torch.cuda.synchronize()
    ell_old = ell0 + torch.from_numpy(np.random.default_rng(62).normal(0.0, 1.0, (w.B, w.n_t))).cuda()
    res = []
    for retain in (0, 1):
        p = dataclasses.replace(problem(w, sample_stride=w.B * w.L * w.d, bound=3),
                                retain_samples=retain)
        ws = b.alloc_workspace(p)
        dx = torch.zeros(w.n_t, w.B, w.L, w.d, dtype=torch.float32, device="cuda")
        dgam = torch.zeros(w.d, dtype=torch.float32, device="cuda")
        dW = torch.zeros(w.d, w.V, dtype=torch.float32, device="cuda")
        ell = torch.zeros(w.B, w.n_t, dtype=torch.float64, device="cuda")
        g = torch.zeros_like(ell)
        loss = torch.zeros(1, dtype=torch.float64, device="cuda")
        nm = torch.zeros(w.B, w.n_t, dtype=torch.int32, device="cuda")
        b.bgpo_elbo_bwd_accumulate_rmsnorm(p, xs, gamma, dev["W"], dev["targets"],
                                           dev["resp_mask"], dev["adv"], ell_old, 0.25, dx, dgam,
                                           dW, ell, g, loss, nm, None, None, ws)
        torch.cuda.synchronize()
        res.append([t.cpu().numpy() for t in (dx, dgam, dW, ell, g, loss, nm)])
    for name, a, c in zip(("dx", "dgamma", "dW", "ell", "g", "loss", "nm"), *res):
        assert np.array_equal(a, c), name
    assert np.abs(res[0][2]).max() > 0 and np.abs(res[0][0]).max() > 0


def test_dw_batches_of_four_with_a_ragged_last_batch():
    """A budget above the default layout raises the dW batch to four units:
    40 samples in units of 8 then give one dW GEMM over four units and one
    over the last unit alone.  Against the oracle (off-policy, both bound
    branches), and l, g, the loss and dX bit-identical to the default batches
    of two (the dW batching changes only dW's fp32 accumulation order)."""
    b = lib()
    w = MID.replace(n_t=40)
    x = workloads.generate(w)
    plan = b.bgpo_workspace_plan(problem(w, ws_budget=1 << 40))
    assert (plan["samples_per_unit"], plan["dw_batch"], plan["mode"]) == (8, 4, "stored")
    ell_old = _off_policy_ell_old(w, x, 47, 1.0)
    ref = elbo.elbo_literal(_oracle_problem(w), x["hidden"], x["W"], x["targets"],
                            x["resp_mask"], x["adv"], ell_old=ell_old)
    outs = []
    for kw in ({}, {"ws_budget": 1 << 40}):
        r = Runner(w, x, **kw)
        r.bwd(ell_old=ell_old)
        outs.append(r.out())
    _check_against_oracle(w, outs[1], ref, range(w.n_t), x["adv"], ell_old)
    for k in ("ell", "g", "nm", "t", "dX"):
        assert np.array_equal(outs[0][k], outs[1][k]), k
    assert outs[0]["loss"] == outs[1]["loss"]
    assert rel_maxnorm(outs[1]["dW"], outs[0]["dW"]) <= 1e-5
