"""Parity of the HIP path (through the C ABI) with the float64 oracle.

Bars: masks, compacted indices, counts and timesteps bit-exact; l_{b,j}
within 1e-3 relative; accumulated dX and dW within 2e-2 relative max-norm
(bf16 inputs, fp32 accumulation, bf16 dZ).
"""
import dataclasses

import numpy as np
import pytest
import torch

import workloads
from oracle import elbo
from gpu_util import Runner, lib, problem, rel_maxnorm

pytestmark = pytest.mark.gpu

ELL_RTOL = 1e-3
GRAD_RTOL = 2e-2

# several 256-wide tiles in every GEMM dimension with ragged tails: rows
# (masked positions), vocabulary (4288 = 16.75 tiles) and hidden size (576)
MID = workloads.Workload("mid_B4_L200_d576_V4288_nt3", B=4, L=200, d=576, V=4288, n_t=3,
                         lengths=(120, 200), group=4, data_seed=2001, philox_seed=0xB6B10001)


def _oracle_problem(w, j_begin=0, j_count=None):
    return elbo.Problem(w.B, w.L, w.d, w.V, w.n_t, j_begin=j_begin, j_count=j_count,
                        seed=w.philox_seed, seq_id_base=w.seq_id_base, t_mode=w.t_mode)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lib()


# ---------------------------------------------------------------- GEMM core

def _slab_major(X):
    """[R, K] -> the K-slab-major operand layout [K/64, R, 64]."""
    R, K = X.shape
    return X.reshape(R, K // 64, 64).permute(1, 0, 2).contiguous()


@pytest.mark.parametrize("M,N,K", [(300, 200, 192), (512, 768, 1024), (257, 1000, 64)])
def test_gemm_core_matches_fp32_reference(M, N, K):
    """The GEMM core of the production kernels (bgpo_test_gemm_nt) against
    exact products of the bf16 operands: ragged tiles in M and N, one slab."""
    g = torch.Generator().manual_seed(M * 7 + N)
    A = torch.randn(M, K, generator=g).to(torch.bfloat16)
    Bm = torch.randn(N, K, generator=g).to(torch.bfloat16)
    ref = A.double() @ Bm.double().T                      # exact products of bf16 values
    C = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    lib().bgpo_test_gemm_nt(_slab_major(A).cuda(), Bm.cuda(), C)
    torch.cuda.synchronize()
    err = (C.cpu().double() - ref).abs().max().item()
    assert err <= 1e-5 * (K ** 0.5) * ref.abs().max().item() + 1e-5, err


@pytest.mark.parametrize("M,N,K", [(320, 200, 192), (512, 768, 1024), (64, 1000, 64),
                                   (4288, 576, 256), (256, 256, 8192), (128, 1, 128)])
def test_gemm_core_transposed_a_matches_fp32_reference(M, N, K):
    """The dW GEMM's kernel (bgpo_test_gemm_tn): A read with its indices
    swapped through the transposing LDS reads, accumulated into C. Ragged
    tiles in M (by 64-wide slabs) and N, one slab of K and 128; twice in a
    row from a nonzero C, so both the read-modify-write of partial tiles and
    the accumulator preload of full tiles are checked against exact products
    of the bf16 operands."""
    g = torch.Generator().manual_seed(M * 5 + N + K)
    A = torch.randn(M, K, generator=g).to(torch.bfloat16)
    Bm = torch.randn(N, K, generator=g).to(torch.bfloat16)
    C0 = torch.randn(N, M, generator=g, dtype=torch.float32)
    prod = Bm.double() @ A.double().T                     # [N, M], exact products of bf16 values
    A_l = A.reshape(M // 64, 64, K).permute(0, 2, 1).contiguous()      # [M/64, K, 64]
    C = C0.clone().cuda()
    for rep in (1, 2):
        lib().bgpo_test_gemm_tn(A_l.cuda(), _slab_major(Bm).cuda(), C)
        torch.cuda.synchronize()
        ref = C0.double() + rep * prod
        err = (C.cpu().double() - ref).abs().max().item()
        assert err <= 2e-5 * (K ** 0.5) * prod.abs().max().item() + 1e-4, (rep, err)


@pytest.mark.parametrize("M,N,K,n_split", [(300, 200, 640, 4), (257, 520, 192, 3), (64, 64, 64, 4),
                                           (512, 256, 4096, 7)])
def test_gemm_core_split_k(M, N, K, n_split):
    """Split-K as the dX GEMM uses it: slices of a multiple of 64, empty
    trailing slices included (K = 64 in 4 slices, stored as zeros); the
    slices sum to the exact product."""
    g = torch.Generator().manual_seed(M + 3 * N + K)
    A = torch.randn(M, K, generator=g).to(torch.bfloat16)
    Bm = torch.randn(N, K, generator=g).to(torch.bfloat16)
    ref = A.double() @ Bm.double().T
    C = torch.full((n_split, M, N), float("nan"), dtype=torch.float32, device="cuda")
    lib().bgpo_test_gemm_split(_slab_major(A).cuda(), Bm.cuda(), C, n_split)
    torch.cuda.synchronize()
    got = C.cpu().double()
    ks = ((K + n_split - 1) // n_split + 63) // 64 * 64
    for s in range(n_split):
        if s * ks >= K:
            assert not got[s].any()                        # an empty slice stores zeros
    err = (got.sum(0) - ref).abs().max().item()
    assert err <= 1e-5 * (K ** 0.5) * ref.abs().max().item() + 1e-5, err


# ---------------------------------------------------------------- masks

# MID with the responses' global ids offset (seq = seq_id_base + b enters the
# Philox counters of t and of the masks), iid and stratified
MID_SEQ = MID.replace(name="mid_seq_id_base_1000003", seq_id_base=1000003)
MID_SEQ_STRAT = MID_SEQ.replace(name="mid_seq_id_base_1000003_stratified", t_mode=1)


@pytest.mark.parametrize("w", workloads.CONFIGS + (MID, MID_SEQ, MID_SEQ_STRAT),
                         ids=lambda w: w.name)
def test_masks_bit_exact(w):
    x = workloads.generate(w, with_weights=False, with_hidden=False)
    resp = torch.from_numpy(x["resp_mask"]).cuda()
    p = problem(w)
    op = _oracle_problem(w)
    idx = torch.full((w.B * w.L,), -7, dtype=torch.int32, device="cuda")
    nm = torch.zeros(w.B, dtype=torch.int32, device="cuda")
    t = torch.zeros(w.B, dtype=torch.float32, device="cuda")
    for j in sorted({0, 1, w.n_t - 1}):
        idx.fill_(-7)
        lib().bgpo_sample_masks(p, resp, j, idx, nm, t)
        T, tt, m, oidx = elbo.sample_masks(op, x["resp_mask"], j)
        torch.cuda.synchronize()
        n = int(nm.sum())
        assert n == oidx.size
        assert np.array_equal(idx[:n].cpu().numpy(), oidx)
        assert np.array_equal(nm.cpu().numpy(), m.sum(axis=1))
        assert np.array_equal(t.cpu().numpy().astype(np.float64), tt)   # exact multiples of 2^-24
        assert (idx[n:].cpu().numpy() == -7).all()                       # untouched tail


@pytest.mark.parametrize("B,L,lengths,j", [
    (2, 64, None, 0), (8, 512, None, 3), (3, 5000, (1, 5000), 1), (37, 1, None, 0),
    (4096, 256, (1, 256), 0), (4096, 256, None, 1), (1, 1 << 20, None, 2), (2048, 512, (300, 512), 5)],
    ids=["B2_L64", "B8_L512", "B3_L5000_ragged", "B37_L1", "B4096_L256_ragged", "B4096_L256",
         "B1_L2p20", "B2048_L512_ragged"])
def test_mask_multiblock_bit_exact(B, L, lengths, j):
    """The multi-block mask passes (used above 65536 positions, forced here at
    every size) give the oracle's compacted positions, counts and timesteps
    bit for bit, up to B*L = 2^20 positions (several blocks, ragged responses,
    single-position responses, one response spanning every block)."""
    w = workloads.TINY.replace(B=B, L=L, n_t=8, lengths=lengths, data_seed=2300 + B,
                               philox_seed=0xB6B0C000 + B * 7 + L)
    x = workloads.generate(w, with_weights=False, with_hidden=False)
    resp = torch.from_numpy(x["resp_mask"]).cuda()
    p = problem(w)
    op = _oracle_problem(w)
    idx = torch.full((B * L,), -7, dtype=torch.int32, device="cuda")
    nm = torch.zeros(B, dtype=torch.int32, device="cuda")
    t = torch.zeros(B, dtype=torch.float32, device="cuda")
    lib().bgpo_test_mask_multiblock(p, resp, j, idx, nm, t)
    T, tt, m, oidx = elbo.sample_masks(op, x["resp_mask"], j)
    torch.cuda.synchronize()
    n = int(nm.sum())
    assert n == oidx.size
    assert np.array_equal(idx[:n].cpu().numpy(), oidx)
    assert np.array_equal(nm.cpu().numpy(), m.sum(axis=1))
    assert np.array_equal(t.cpu().numpy().astype(np.float64), tt)
    assert (idx[n:].cpu().numpy() == -7).all()
    if B * L <= 65536:    # the single-workgroup kernel gives the same
        idx2 = torch.full((B * L,), -7, dtype=torch.int32, device="cuda")
        lib().bgpo_sample_masks(p, resp, j, idx2, nm, t)
        torch.cuda.synchronize()
        assert torch.equal(idx, idx2)


# ---------------------------------------------------------------- ELBO head

def _check_against_oracle(w, out, ref, js, adv, ell_old=None, loss_scale=1.0 / 8, bound=0):
    """Counts and t bit-exact, l within ELL_RTOL; g and the loss are functions of l,
    so they are checked tightly against the oracle's bound applied to the HIP
    path's own l (a 1e-3 error in l can be a large relative error in (1 + d) A
    when 1 + d is near 0); the gradients within GRAD_RTOL."""
    for j in js:
        assert np.array_equal(out["nm"][:, j], ref.n_masked[:, j])
        assert np.array_equal(out["t"][:, j].astype(np.float64), ref.t[:, j])
        np.testing.assert_allclose(out["ell"][:, j], ref.ell[:, j], rtol=ELL_RTOL, atol=0)
    old = out["ell"] if ell_old is None else ell_old          # NULL ell_old: on-policy, d = 0
    dbar = (out["ell"] - old).mean(axis=1)
    g_of_ell = np.array([[elbo.bound_term(out["ell"][b, j] - old[b, j], float(adv[b]), w.n_t, bound,
                                          dbar[b])[0] for j in range(w.n_t)] for b in range(w.B)])
    for j in js:
        np.testing.assert_allclose(out["g"][:, j], g_of_ell[:, j], rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(out["g"][:, j], ref.g[:, j], rtol=ELL_RTOL, atol=ELL_RTOL * np.abs(ref.g).max())
    js = list(js)
    expect_loss = -loss_scale * g_of_ell[:, js].sum()
    assert abs(out["loss"] - expect_loss) <= 1e-12 * loss_scale * np.abs(g_of_ell).sum()
    assert abs(out["loss"] - ref.loss) <= ELL_RTOL * loss_scale * np.abs(ref.g).sum()
    assert rel_maxnorm(out["dX"], ref.dX) <= GRAD_RTOL
    assert rel_maxnorm(out["dW"], ref.dW) <= GRAD_RTOL
    assert out["flags"] == 0


def test_tiny_parity_fwd_and_bwd():
    w = workloads.TINY
    x = workloads.generate(w)
    r = Runner(w, x)
    ref = elbo.elbo_literal(_oracle_problem(w), x["hidden"], x["W"], x["targets"],
                            x["resp_mask"], x["adv"])
    r.fwd()
    f = r.out()
    np.testing.assert_allclose(f["ell"], ref.ell, rtol=ELL_RTOL, atol=0)
    assert np.array_equal(f["nm"], ref.n_masked)
    r.bwd()
    _check_against_oracle(w, r.out(), ref, range(w.n_t), x["adv"])


def test_mid_parity_off_policy_both_branches():
    w = MID
    x = workloads.generate(w)
    assert (x["adv"] > 0).any() and (x["adv"] < 0).any()
    op = _oracle_problem(w)
    ell_old = elbo.elbo_literal(op, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                                backward=False).ell
    ell_old = ell_old + np.random.default_rng(5).normal(0, 2.0, ell_old.shape)
    ref = elbo.elbo_literal(op, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                            ell_old=ell_old, loss_scale=0.25)
    r = Runner(w, x)
    r.bwd(ell_old=ell_old, loss_scale=0.25)
    _check_against_oracle(w, r.out(), ref, range(w.n_t), x["adv"], ell_old, 0.25)


@pytest.mark.parametrize("bound", [1, 2, 3], ids=["taylor_only", "jensen_only", "exact"])
def test_mid_parity_off_policy_bound_modes(bound):
    """Table 3's single-bound ablations and the exact objective of Eq. elbo_ratio,
    off-policy with both advantage signs, against the oracle in the same mode."""
    w = MID
    x = workloads.generate(w)
    op = dataclasses.replace(_oracle_problem(w), bound=bound)
    ell_old = elbo.elbo_literal(op, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                                backward=False).ell
    ell_old = ell_old + np.random.default_rng(6).normal(0, 1.0, ell_old.shape)
    ref = elbo.elbo_literal(op, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                            ell_old=ell_old, loss_scale=0.25)
    r = Runner(w, x)
    r.bwd(ell_old=ell_old, loss_scale=0.25, bound=bound)
    _check_against_oracle(w, r.out(), ref, range(w.n_t), x["adv"], ell_old, 0.25, bound)


def test_every_bound_mode_identical_on_policy():
    """On-policy all objective modes have the same gradient scale A / n_t, so the
    HIP path gives bit-identical outputs for each (Section 3.2)."""
    w = MID
    x = workloads.generate(w)
    r = Runner(w, x)
    r.fwd()
    ell_fwd = r.out()["ell"].copy()
    outs = []
    for bound in (0, 1, 2, 3):
        r.zero_grads()
        r.bwd(ell_old=ell_fwd, bound=bound)
        outs.append(r.out())
    for o in outs[1:]:
        for k in ("ell", "g", "dX", "dW"):
            assert np.array_equal(o[k], outs[0][k]), k
        assert o["loss"] == outs[0]["loss"]


@pytest.mark.parametrize("n_t", [3, 12], ids=["one_unit", "two_units"])
def test_retained_exact_mode_matches_oracle_and_two_pass_mode(n_t):
    """retain_samples = 1 keeps every sample's state instead of running the
    forward twice: same oracle parity, and the same l, g, loss and dX as the
    two-pass mode bit for bit (identical kernels in the same order), dW
    included.  With two units (n_t = 12,
    units of 8 and 4 in one dW batch) the second unit's H_c^T columns start
    where the first unit's rows end, rounded up to 64, inside the first unit's
    256-row padding, and they hold the second unit's rows before the first
    unit's columns are scaled: the scaling must stop where they start."""
    from paper_2510_11683_amd import bgpo
    w = MID.replace(n_t=n_t)
    x = workloads.generate(w)
    op = dataclasses.replace(_oracle_problem(w), bound=3)
    ell_old = elbo.elbo_literal(op, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                                backward=False).ell
    ell_old = ell_old + np.random.default_rng(7).normal(0, 1.0, ell_old.shape)
    ref = elbo.elbo_literal(op, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                            ell_old=ell_old, loss_scale=0.25)
    outs = []
    for retain in (0, 1):
        r = Runner(w, x)
        pr = dataclasses.replace(problem(w, bound=3), retain_samples=retain)
        r.ws = bgpo.alloc_workspace(pr)
        d = r.dev
        eo = torch.as_tensor(ell_old, dtype=torch.float64).cuda()
        bgpo.bgpo_elbo_bwd_accumulate(pr, d["hidden"], d["W"], d["targets"], d["resp_mask"],
                                      d["adv"], eo, 0.25, r.dX, r.dW, r.ell, r.g, r.loss, r.nm,
                                      r.t, r.flags, r.ws)
        outs.append(r.out())
    two, ret = outs
    _check_against_oracle(w, ret, ref, range(w.n_t), x["adv"], ell_old, 0.25, 3)
    for k in ("ell", "g", "nm", "t", "dX", "dW"):
        assert np.array_equal(two[k], ret[k]), k
    assert two["loss"] == ret["loss"]


def test_exact_mode_partial_range_refused():
    w = MID
    x = workloads.generate(w, with_weights=True)
    r = Runner(w, x)
    from paper_2510_11683_amd import bgpo
    with pytest.raises(bgpo.BgpoError):
        r.bwd(j_begin=1, j_count=1, bound=3)


@pytest.mark.parametrize("w_std", [0.2, 0.5], ids=["logit_std_4.8", "logit_std_12"])
def test_mid_parity_peaky_logits(w_std):
    """Trained heads give far peakier softmaxes than N(0, 0.02) weights: with
    W ~ N(0, w_std^2) the logits have std w_std * sqrt(d), most of the
    probability sits on a few tokens and the stored exponentials of the others
    are far below the row's reference; off-policy, both bound branches."""
    w = MID.replace(w_std=w_std)
    x = workloads.generate(w)
    op = _oracle_problem(w)
    ell_old = elbo.elbo_literal(op, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                                backward=False).ell
    ell_old = ell_old + np.random.default_rng(9).normal(0, 1.0, ell_old.shape)
    ref = elbo.elbo_literal(op, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                            ell_old=ell_old, loss_scale=0.25)
    r = Runner(w, x)
    r.bwd(ell_old=ell_old, loss_scale=0.25)
    _check_against_oracle(w, r.out(), ref, range(w.n_t), x["adv"], ell_old, 0.25)


@pytest.mark.parametrize("n_t", [3, 12], ids=["one_unit", "two_units_one_dw_batch"])
def test_mid_parity_rows_outside_exponent_range(n_t):
    """The stored backward keeps a row's exponentials against its target
    logit plus 60 (log2 units); rows whose log2-sum-exp exceeds that by more
    than 64 (target log-probability below about -86) are recomputed after the
    forward.  With W ~ N(0, 1) (logit std 24) about half of the rows are such
    rows (counted here from float64 logits), off-policy, both bound branches.
    With 12 samples the second unit's rows sit after the first's in the dZ
    of their shared dW batch, so its recomputed rows are written there too."""
    w = MID.replace(w_std=1.0, n_t=n_t)
    if n_t == 12:
        plan = lib().bgpo_workspace_plan(problem(w))
        assert plan["samples_per_unit"] == 8 and plan["dw_batch"] == 2 and plan["mode"] == "stored"
    x = workloads.generate(w)
    H = elbo.bf16_to_f64(x["hidden"]).reshape(-1, w.d)
    z = H @ elbo.bf16_to_f64(x["W"])
    lse = z.max(1) + np.log(np.exp(z - z.max(1, keepdims=True)).sum(1))
    gap2 = (lse - z[np.arange(z.shape[0]), x["targets"].reshape(-1)]) / np.log(2.0)
    far = gap2[x["resp_mask"].reshape(-1).astype(bool)] > 124
    assert 0.2 < far.mean() < 0.8
    op = _oracle_problem(w)
    ell_old = elbo.elbo_literal(op, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                                backward=False).ell
    ell_old = ell_old + np.random.default_rng(12).normal(0, 1.0, ell_old.shape)
    ref = elbo.elbo_literal(op, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                            ell_old=ell_old, loss_scale=0.25)
    r = Runner(w, x)
    r.bwd(ell_old=ell_old, loss_scale=0.25)
    _check_against_oracle(w, r.out(), ref, range(w.n_t), x["adv"], ell_old, 0.25)


@pytest.mark.parametrize("B,L,d,V,n_t", [(1, 1, 64, 64, 3), (3, 3, 64, 192, 5), (2, 70, 128, 64, 2)],
                         ids=["B1_L1_d64_V64", "B3_L3_d64_V192", "B2_L70_d128_V64"])
def test_smallest_shapes(B, L, d, V, n_t):
    """The smallest supported sizes: one partial tile in every GEMM dimension,
    a vocabulary of one 64-wide half slice, single-position responses."""
    w = workloads.TINY.replace(B=B, L=L, d=d, V=V, n_t=n_t, adv="normal", data_seed=2100 + B * L)
    x = workloads.generate(w)
    op = _oracle_problem(w)
    ell_old = elbo.elbo_literal(op, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                                backward=False).ell
    ell_old = ell_old + np.random.default_rng(10).normal(0, 0.5, ell_old.shape)
    ref = elbo.elbo_literal(op, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                            ell_old=ell_old, loss_scale=0.25)
    r = Runner(w, x)
    r.bwd(ell_old=ell_old, loss_scale=0.25)
    _check_against_oracle(w, r.out(), ref, range(w.n_t), x["adv"], ell_old, 0.25)


def test_on_policy_d_is_exactly_zero():
    """ell from the forward entry point fed back as ell_old gives d == 0 bit-exactly,
    so g = A / n_t exactly (the equivalence case)."""
    w = MID
    x = workloads.generate(w)
    r = Runner(w, x)
    r.fwd()
    ell_fwd = r.out()["ell"].copy()
    r.bwd(ell_old=ell_fwd)
    o = r.out()
    assert np.array_equal(o["ell"], ell_fwd)
    adv = x["adv"].astype(np.float64)
    expect = np.repeat((adv / w.n_t)[:, None], w.n_t, axis=1)
    assert np.array_equal(o["g"], expect)


def test_linearity_and_determinism():
    w = MID.replace(n_t=4)
    x = workloads.generate(w)
    r = Runner(w, x)
    r.bwd()
    full = r.out()
    r.zero_grads()
    r.bwd()
    again = r.out()
    assert np.array_equal(full["dX"], again["dX"]) and np.array_equal(full["dW"], again["dW"])
    assert np.array_equal(full["ell"], again["ell"]) and full["loss"] == again["loss"]
    r.zero_grads()
    for jb, jc in ((0, 1), (1, 2), (3, 1)):
        r.bwd(j_begin=jb, j_count=jc)
    split = r.out()
    assert np.array_equal(split["ell"], full["ell"])
    assert abs(split["loss"] - full["loss"]) <= 1e-12 * abs(full["loss"])
    assert rel_maxnorm(split["dX"], full["dX"]) <= 1e-5
    assert rel_maxnorm(split["dW"], full["dW"]) <= 1e-5


def test_timing_record_counts_kernel_launches():
    """The optional timing record adds, per kernel class, the elapsed time and
    the number of kernel launches: 10 samples in units of 8 give 2 units; per
    unit one forward and dX GEMM launch, the three row-factor kernels of the
    gradient (row factors and target entries, H_c^T scaling, recomputed
    rows; class BGPO_K_SOFTMAX_GRAD), one
    gather, the three row reductions (target logit, log-sum-exp, per-response
    terms), and one mask and one dX reduction per sample; one dW GEMM for the
    batch of both units; the W transpose once per call."""
    w = workloads.TINY.replace(n_t=10)
    r = Runner(w, workloads.generate(w))
    t = lib().Timing()
    r.bwd(timing=t)
    torch.cuda.synchronize()
    got = {k: n for k, (ms, n) in t.as_dict().items()}
    assert got == {"transpose_w": 1, "mask": 10, "gather": 2, "fwd": 2, "ell": 6,
                   "softmax_grad": 6, "dx": 2, "dx_reduce": 10, "dw": 1, "recompute": 0}
    assert all(ms > 0 for ms, n in t.as_dict().values() if n)
    r.fwd(timing=t)                                     # forward only: no gradient classes
    got2 = {k: n for k, (ms, n) in t.as_dict().items()}
    assert got2 == {**got, "transpose_w": 2, "mask": 20, "gather": 4, "fwd": 4, "ell": 12}


def test_concurrent_streams_match_sequential():
    """Two problems, each with its own workspace, run on two streams at the
    same time give the same bits as one after the other: the entry points
    keep no state between calls, and every reduction has a fixed order."""
    wa = MID.replace(n_t=3)
    wb = MID.replace(n_t=5, data_seed=2002, philox_seed=0xB6B10002)
    xa, xb = workloads.generate(wa), workloads.generate(wb)
    r = Runner(wb, xb)
    r.fwd()
    old_b = r.out()["ell"] + np.random.default_rng(12).normal(0, 0.5, (wb.B, wb.n_t))  # off-policy
    del r
    seq = []
    for w, x, eo in ((wa, xa, None), (wb, xb, old_b)):
        r = Runner(w, x)
        r.bwd(ell_old=eo)
        r.bwd(ell_old=eo)                 # the second call accumulates onto the first
        seq.append(r.out())
        del r
    ra, rb = Runner(wa, xa), Runner(wb, xb)
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    cur = torch.cuda.current_stream()
    sa.wait_stream(cur)
    sb.wait_stream(cur)
    for _ in range(2):
        with torch.cuda.stream(sa):
            ra.bwd()
        with torch.cuda.stream(sb):
            rb.bwd(ell_old=old_b)
    cur.wait_stream(sa)
    cur.wait_stream(sb)
    for o, e in ((ra.out(), seq[0]), (rb.out(), seq[1])):
        for k in ("ell", "g", "nm", "t", "dX", "dW"):
            assert np.array_equal(o[k], e[k]), k
        assert o["loss"] == e["loss"] and o["flags"] == e["flags"] == 0
        assert np.abs(o["dX"]).max() > 0


def test_graph_capture_replays_match_eager():
    """A whole backward call captured in a HIP graph (the library allocates
    nothing, sets no memory and does not synchronise without a timing record,
    so every launch records) and replayed three times, with eager zeroing and
    a host synchronisation between replays: every replay gives the eager
    call's bits."""
    w = MID.replace(n_t=4)
    x = workloads.generate(w)
    r = Runner(w, x)
    r.bwd()
    eager = r.out()
    b, d = lib(), r.dev
    prob = problem(w)
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


def test_empty_range_and_empty_masks():
    w = MID
    x = workloads.generate(w)
    r = Runner(w, x)
    r.bwd(j_begin=1, j_count=0)
    o = r.out()
    assert not o["dX"].any() and not o["dW"].any() and o["loss"] == 0.0
    # a response-mask of all zeros: nothing is ever masked
    x0 = dict(x)
    x0["resp_mask"] = np.zeros_like(x["resp_mask"])
    r0 = Runner(w, x0)
    r0.bwd()
    o0 = r0.out()
    assert not o0["nm"].any() and not o0["ell"].any()
    assert not o0["dX"].any() and not o0["dW"].any()
    expect_g = np.where(x["adv"] >= 0, x["adv"].astype(np.float64), np.exp(0.0) * x["adv"]) / w.n_t
    np.testing.assert_allclose(o0["g"], np.repeat(expect_g[:, None], w.n_t, 1), rtol=1e-15)


def test_nonfinite_flag_raised_not_clamped():
    w = MID
    x = workloads.generate(w)
    x = dict(x)
    x["adv"] = -np.abs(x["adv"]) - 0.1            # Jensen branch everywhere
    r = Runner(w, x)
    ell_old = np.full((w.B, w.n_t), -1e6)         # d = l - l_old ~ +1e6 -> e^d overflows
    r.bwd(ell_old=ell_old, j_count=1)
    o = r.out()
    assert o["flags"] & lib().BGPO_FLAG_NONFINITE
    assert np.isinf(o["g"][:, 0]).all()


def test_memory_constant_in_n_t():
    """Peak device memory of a full bwd call is the same for n_t = 1, 4, 16 (the
    [B, n_t] outputs round to the same 512-byte allocation blocks here)."""
    w = MID
    x = workloads.generate(w)
    peaks = []
    for nt in (1, 4, 16):
        wn = w.replace(n_t=nt)
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        torch.cuda.reset_peak_memory_stats()
        free0 = torch.cuda.mem_get_info()[0]
        r = Runner(wn, x)
        r.bwd()
        torch.cuda.synchronize()
        peaks.append((torch.cuda.max_memory_allocated(), free0 - torch.cuda.mem_get_info()[0]))
        del r
    assert len({p[0] for p in peaks}) == 1, peaks
    assert len({p[1] for p in peaks}) == 1, peaks


@pytest.mark.parametrize("w", [MID_SEQ, MID_SEQ_STRAT], ids=lambda w: w.name)
def test_mid_parity_with_seq_id_base(w):
    """The full backward with the responses' global ids offset: masks, t, l,
    g and the gradients against the oracle (off-policy)."""
    w = w.replace(n_t=3)
    x = workloads.generate(w)
    op = _oracle_problem(w)
    ell_old = elbo.elbo_literal(op, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                                backward=False).ell
    ell_old = ell_old + np.random.default_rng(17).normal(0, 1.0, ell_old.shape)
    ref = elbo.elbo_literal(op, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                            ell_old=ell_old)
    r = Runner(w, x)
    r.bwd(ell_old=ell_old)
    _check_against_oracle(w, r.out(), ref, range(w.n_t), x["adv"], ell_old)
