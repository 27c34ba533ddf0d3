"""Pins for the float64 ELBO / lower-bound oracle.

Each check compares the oracle with something other than itself:

* log-softmax:    scipy.special.logsumexp and torch.log_softmax (float64)
* t = 1:          every response position is masked and l = -cross-entropy
                  (torch.nn.functional.cross_entropy, reduction 'sum')
* closed form:    brute force over all 2^L masks of one response at fixed t;
                  E[l | t] = sum_i log p_i for every t (Eq. per_step_loss with
                  the forward process of Section 2.1)
* gradients:      central finite differences of the oracle's own loss value,
                  and torch.autograd on an independently written expression
* equivalence:    on-policy, the bound's value equals A and its gradient equals
                  the gradient of exp(B_theta - B_old) A (Section 3.2)
* Lemmas 1 and 2: off-policy, sum_j g_j <= exp(mean_j d_j) A per response,
                  with equality exactly where the lemmas say
* linearity:      any split of the sample range accumulates to the same result
                  (Eq. lower_bound_def)
* literal form == collapsed form.

The ``check_*`` helpers raise AssertionError on a mismatch; the mutation
tests re-run them against deliberately broken copies of the oracle.
"""
import itertools

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st
from scipy.special import logsumexp

import workloads
from oracle import elbo



@pytest.fixture(autouse=True)
def _float64_default():
    """torch's autograd pins in this module run in float64; the default is
    restored afterwards, so that other modules (collected in the same
    process) keep float32."""
    prev = torch.get_default_dtype()
    torch.set_default_dtype(torch.float64)
    yield
    torch.set_default_dtype(prev)


def _rand_problem(seed, B=2, L=6, d=4, V=8, n_t=3, w_scale=0.5):
    rng = np.random.default_rng(seed)
    H = rng.standard_normal((B, L, d))
    W = rng.standard_normal((d, V)) * w_scale
    y = rng.integers(0, V, size=(B, L)).astype(np.int32)
    resp = np.ones((B, L), dtype=np.uint8)
    resp[-1, L - 2:] = 0
    adv = np.array([0.7, -1.3][:B] + [0.2] * max(0, B - 2), dtype=np.float64)
    p = elbo.Problem(B, L, d, V, n_t, seed=0xABCD0000 + seed)
    return p, H, W, y, resp, adv


# ---------------------------------------------------------------- log-softmax

def check_log_softmax(fn=None):
    fn = fn or elbo.log_softmax_rows
    rng = np.random.default_rng(3)
    for scale in (1.0, 12.8, 300.0):
        z = rng.standard_normal((7, 513)) * scale
        ref = z - logsumexp(z, axis=1, keepdims=True)
        tref = torch.log_softmax(torch.from_numpy(z), dim=1).numpy()
        out = fn(z)
        assert np.allclose(out, ref, rtol=0, atol=1e-10 * max(1.0, scale))
        assert np.allclose(out, tref, rtol=0, atol=1e-10 * max(1.0, scale))


def test_log_softmax_matches_libraries():
    check_log_softmax()


# ---------------------------------------------------------------- t = 1 case

def check_t1_cross_entropy(ell_fn=None):
    ell_fn = ell_fn or elbo.ell_of_mask
    rng = np.random.default_rng(5)
    L, d, V = 9, 16, 50
    H = rng.standard_normal((L, d))
    W = rng.standard_normal((d, V)) * 0.3
    y = rng.integers(0, V, size=L)
    ell, rows, _ = ell_fn(H, W, y, np.ones(L, dtype=bool), 1.0)
    ce = torch.nn.functional.cross_entropy(torch.from_numpy(H @ W), torch.from_numpy(y),
                                           reduction="sum").item()
    assert rows.size == L
    assert abs(ell - (-ce)) <= 1e-10 * abs(ce)


def test_t1_is_negative_cross_entropy():
    check_t1_cross_entropy()


# ---------------------------------------------------------------- brute force

def check_brute_force_expectation(ell_fn=None):
    """E over the forward process of l(y_t, t) equals sum_i log p_i at any t."""
    ell_fn = ell_fn or elbo.ell_of_mask
    rng = np.random.default_rng(11)
    L, d, V = 10, 6, 12
    H = rng.standard_normal((L, d))
    W = rng.standard_normal((d, V))
    y = rng.integers(0, V, size=L)
    full = torch.log_softmax(torch.from_numpy(H @ W), dim=1).numpy()[np.arange(L), y].sum()
    for t in (0.05, 0.37, 0.5, 0.93):
        acc = 0.0
        for bits in itertools.product((0, 1), repeat=L):
            m = np.array(bits, dtype=bool)
            k = int(m.sum())
            prob = t ** k * (1 - t) ** (L - k)
            acc += prob * ell_fn(H, W, y, m, t)[0]
        assert abs(acc - full) <= 1e-11 * abs(full), (t, acc, full)


def test_brute_force_expectation_equals_loglik():
    check_brute_force_expectation()


def test_brute_force_padding_never_counts():
    rng = np.random.default_rng(12)
    L, d, V = 8, 4, 6
    H = rng.standard_normal((L, d))
    W = rng.standard_normal((d, V))
    y = rng.integers(0, V, size=L)
    resp = np.array([1, 1, 1, 1, 1, 0, 0, 0], dtype=np.uint8)
    p = elbo.Problem(1, L, d, V, 64, seed=77)
    for j in range(64):
        T, t, m, idx = elbo.sample_masks(p, resp[None], j)
        assert not m[0, 5:].any()
        assert np.array_equal(idx, np.flatnonzero(m.reshape(-1)))


# ---------------------------------------------------------------- gradients

def _loss_value(p, H, W, y, resp, adv, ell_old, scale):
    return elbo.elbo_literal_f64(p, H, W, y, resp, adv, ell_old=ell_old,
                                 loss_scale=scale, backward=False).loss


def check_finite_differences(literal=None, seed=1):
    literal = literal or elbo.elbo_literal_f64
    p, H, W, y, resp, adv = _rand_problem(seed)
    scale = 0.125
    ell_old = np.random.default_rng(seed + 100).standard_normal((p.B, p.n_t)) * 0.5 - 8.0
    res = literal(p, H, W, y, resp, adv, ell_old=ell_old, loss_scale=scale)
    h = 1e-6
    rng = np.random.default_rng(seed + 200)
    for _ in range(12):
        b, i, k = rng.integers(p.B), rng.integers(p.L), rng.integers(p.d)
        Hp, Hm = H.copy(), H.copy()
        Hp[b, i, k] += h
        Hm[b, i, k] -= h
        fd = (_loss_value(p, Hp, W, y, resp, adv, ell_old, scale)
              - _loss_value(p, Hm, W, y, resp, adv, ell_old, scale)) / (2 * h)
        assert abs(fd - res.dX[b, i, k]) <= 1e-6 * max(1.0, abs(fd)), ("dX", b, i, k, fd, res.dX[b, i, k])
    for _ in range(12):
        k, v = rng.integers(p.d), rng.integers(p.V)
        Wp, Wm = W.copy(), W.copy()
        Wp[k, v] += h
        Wm[k, v] -= h
        fd = (_loss_value(p, H, Wp, y, resp, adv, ell_old, scale)
              - _loss_value(p, H, Wm, y, resp, adv, ell_old, scale)) / (2 * h)
        assert abs(fd - res.dW[k, v]) <= 1e-6 * max(1.0, abs(fd)), ("dW", k, v, fd, res.dW[k, v])


def test_gradient_finite_differences():
    check_finite_differences()


def _torch_bound_loss(p, H, W, y, resp, adv, ell_old, scale):
    """Independent torch expression of the accumulated loss sum_{b,j} -scale*g_{b,j}."""
    Ht = torch.tensor(H, requires_grad=True)
    Wt = torch.tensor(W, requires_grad=True)
    total = torch.zeros(())
    ells = torch.zeros(p.B, p.n_t)
    for j in p.js:
        T, t, m, _ = elbo.sample_masks(p, resp, j)
        for b in range(p.B):
            sel = torch.from_numpy(np.flatnonzero(m[b]))
            logits = Ht[b, sel] @ Wt
            tgt = torch.from_numpy(y[b][sel.numpy()].astype(np.int64))
            lp = torch.log_softmax(logits, dim=-1).gather(1, tgt[:, None]).sum()
            ell = lp / float(t[b])
            ells[b, j] = ell.detach()
            dlt = ell - (ell.detach() if ell_old is None else float(ell_old[b, j]))
            A = float(adv[b])
            gj = (1 + dlt) * A / p.n_t if A >= 0 else torch.exp(dlt) * A / p.n_t
            total = total - scale * gj
    total.backward()
    return total.item(), Ht.grad.numpy(), Wt.grad.numpy(), ells.numpy()


def check_autograd(literal=None, seed=2, on_policy=False):
    literal = literal or elbo.elbo_literal_f64
    p, H, W, y, resp, adv = _rand_problem(seed, B=3, L=7, d=5, V=11, n_t=4)
    adv = np.array([1.1, -0.6, -0.0])
    scale = 1 / 8
    ell_old = None if on_policy else np.random.default_rng(seed).standard_normal((p.B, p.n_t)) - 9.0
    val, gH, gW, ells = _torch_bound_loss(p, H, W, y, resp, adv, ell_old, scale)
    res = literal(p, H, W, y, resp, adv, ell_old=ell_old, loss_scale=scale)
    assert abs(res.loss - val) <= 1e-12 * max(1.0, abs(val))
    assert np.allclose(res.ell, ells, rtol=1e-12, atol=1e-12)
    assert np.allclose(res.dX, gH, rtol=1e-10, atol=1e-13)
    assert np.allclose(res.dW, gW, rtol=1e-10, atol=1e-13)


@pytest.mark.parametrize("on_policy", [False, True])
def test_gradient_autograd(on_policy):
    check_autograd(on_policy=on_policy)


# ---------------------------------------------------------------- equivalence

def check_on_policy_equivalence(literal=None, seed=4):
    """On-policy (theta_old = theta): R_lb = R = A in value; and the accumulated
    gradient of sum_j -scale g_j equals the gradient of -scale exp(B - B_old) A."""
    literal = literal or elbo.elbo_literal_f64
    p, H, W, y, resp, adv = _rand_problem(seed, B=2, L=6, d=4, V=9, n_t=5)
    scale = 0.25
    fwd = literal(p, H, W, y, resp, adv, loss_scale=scale, backward=False)
    res = literal(p, H, W, y, resp, adv, ell_old=fwd.ell, loss_scale=scale)
    # value: sum_j g_j = A exactly (every d_j is zero)
    assert np.array_equal(res.ell, fwd.ell)
    for b in range(p.B):
        assert abs(res.g[b].sum() - adv[b]) <= 1e-14 * max(1.0, abs(adv[b]))
    # gradient of the exact (non-linear) objective, all n_t graphs kept at once
    Ht = torch.tensor(H, requires_grad=True)
    Wt = torch.tensor(W, requires_grad=True)
    total = torch.zeros(())
    for b in range(p.B):
        ells = []
        for j in p.js:
            T, t, m, _ = elbo.sample_masks(p, resp, j)
            sel = torch.from_numpy(np.flatnonzero(m[b]))
            tgt = torch.from_numpy(y[b][sel.numpy()].astype(np.int64))
            lp = torch.log_softmax(Ht[b, sel] @ Wt, dim=-1).gather(1, tgt[:, None]).sum()
            ells.append(lp / float(t[b]))
        Bhat = torch.stack(ells).mean()
        R = torch.exp(Bhat - Bhat.detach()) * float(adv[b])
        assert abs(R.item() - adv[b]) <= 1e-14
        total = total - scale * R
    total.backward()
    assert np.allclose(res.dX, Ht.grad.numpy(), rtol=1e-10, atol=1e-13)
    assert np.allclose(res.dW, Wt.grad.numpy(), rtol=1e-10, atol=1e-13)


def test_on_policy_equivalence():
    check_on_policy_equivalence()


# ---------------------------------------------------------------- Lemmas 1, 2

def _R_and_Rlb(p, H, W, Wold, y, resp, adv, literal):
    old = literal(p, H, Wold, y, resp, adv, backward=False)
    new = literal(p, H, W, y, resp, adv, ell_old=old.ell, backward=False)
    dmean = (new.ell - old.ell).mean(axis=1)
    return np.exp(dmean) * adv, new.g.sum(axis=1), new.ell - old.ell


@settings(max_examples=25, deadline=None)
@given(seed=st.integers(0, 10_000), eps=st.floats(1e-3, 0.5),
       a0=st.floats(-3, 3), a1=st.floats(-3, 3))
def test_lower_bound_lemmas(seed, eps, a0, a1):
    p, H, W, y, resp, adv = _rand_problem(seed, B=2, L=5, d=3, V=7, n_t=4)
    adv = np.array([a0, a1])
    Wold = W + eps * np.random.default_rng(seed + 1).standard_normal(W.shape)
    R, Rlb, dd = _R_and_Rlb(p, H, W, Wold, y, resp, adv, elbo.elbo_literal_f64)
    assert np.all(Rlb <= R + 1e-12 * (1 + np.abs(R)))


def check_bound_equality_cases(literal=None):
    """Jensen is tight iff all d_j are equal; Taylor is tight iff mean d = 0."""
    literal = literal or elbo.elbo_literal_f64
    p, H, W, y, resp, adv = _rand_problem(8, B=2, L=6, d=4, V=8, n_t=4)
    adv = np.array([0.9, -1.7])
    base = literal(p, H, W, y, resp, adv, backward=False).ell
    # constant shift c: d_j = c for all j -> Jensen branch exact, Taylor strict
    c = 0.3
    res = literal(p, H, W, y, resp, adv, ell_old=base - c, backward=False)
    R = np.exp(c) * adv
    assert abs(res.g[1].sum() - R[1]) <= 1e-13 * abs(R[1])
    assert res.g[0].sum() < R[0] - 1e-3
    assert abs(res.g[0].sum() - (1 + c) * adv[0]) <= 1e-13
    # zero-mean, unequal d: Taylor exact, Jensen strict
    off = np.array([0.4, -0.4, 0.1, -0.1])
    res = literal(p, H, W, y, resp, adv, ell_old=base - off[None, :], backward=False)
    assert abs(res.g[0].sum() - adv[0]) <= 1e-13
    assert res.g[1].sum() < adv[1] - 1e-4


def test_bound_equality_cases():
    check_bound_equality_cases()


# ---------------------------------------------------------------- linearity

def check_linearity(literal=None):
    literal = literal or elbo.elbo_literal_f64
    p, H, W, y, resp, adv = _rand_problem(9, B=2, L=8, d=4, V=10, n_t=6)
    ell_old = np.random.default_rng(1).standard_normal((p.B, p.n_t)) - 10
    full = literal(p, H, W, y, resp, adv, ell_old=ell_old)
    parts = []
    for jb, jc in ((0, 1), (1, 3), (4, 2)):
        q = elbo.Problem(p.B, p.L, p.d, p.V, p.n_t, j_begin=jb, j_count=jc, seed=p.seed)
        parts.append(literal(q, H, W, y, resp, adv, ell_old=ell_old))
    assert abs(sum(r.loss for r in parts) - full.loss) <= 1e-13 * max(1, abs(full.loss))
    assert np.allclose(sum(r.dX for r in parts), full.dX, rtol=1e-12, atol=1e-14)
    assert np.allclose(sum(r.dW for r in parts), full.dW, rtol=1e-12, atol=1e-14)
    assert np.array_equal(sum(r.ell for r in parts), full.ell)


def test_linearity_over_sample_ranges():
    check_linearity()


# ---------------------------------------------------------------- literal == collapsed

@pytest.mark.parametrize("off_policy", [False, True])
def test_literal_equals_collapsed(off_policy):
    w = workloads.TINY.replace(lengths=(40, 64), B=4, adv="normal")
    x = workloads.generate(w)
    p = elbo.Problem(w.B, w.L, w.d, w.V, w.n_t, seed=w.philox_seed)
    ell_old = None
    if off_policy:
        ell_old = elbo.elbo_literal(p, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                                    backward=False).ell + 0.37
    a = elbo.elbo_literal(p, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"], ell_old=ell_old)
    c = elbo.elbo_collapsed(p, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"], ell_old=ell_old)
    assert np.array_equal(a.n_masked, c.n_masked)
    for j in p.js:
        assert np.array_equal(a.idx[j], c.idx[j])
    assert np.allclose(a.ell, c.ell, rtol=1e-12)
    assert np.allclose(a.g, c.g, rtol=1e-12)
    assert abs(a.loss - c.loss) <= 1e-12 * abs(a.loss)
    assert np.abs(a.dX - c.dX).max() <= 1e-11 * np.abs(a.dX).max()
    assert np.abs(a.dW - c.dW).max() <= 1e-11 * np.abs(a.dW).max()
    # restricted gradients equal the corresponding slices of the full ones
    rows = np.array([3, 70, 130, 200])
    cols = np.array([0, 5, 511, 1023])
    r = elbo.elbo_collapsed(p, x["hidden"], x["W"], x["targets"], x["resp_mask"], x["adv"],
                            ell_old=ell_old, dx_rows=rows, dw_cols=cols)
    assert np.allclose(r.dX, c.dX.reshape(-1, w.d)[rows], rtol=1e-12, atol=1e-15)
    assert np.allclose(r.dW, c.dW[:, cols], rtol=1e-12, atol=1e-15)


def test_zero_std_edge_cases():
    """Empty masks contribute l = 0 and no gradient; A = -0.0 takes the Taylor branch."""
    g, dg = elbo.bound_term(0.0, -0.0, 4)
    assert g == 0.0 and dg == 0.0 and np.signbit(dg)
    H = np.zeros((3, 2))
    W = np.zeros((2, 4))
    ell, rows, lsm = elbo.ell_of_mask(H, W, np.zeros(3, int), np.zeros(3, bool), 0.5)
    assert ell == 0.0 and rows.size == 0


# ---------------------------------------------------------------- bf16 widening

def check_bf16_widening(fn=None):
    """Every one of the 65536 bfloat16 bit patterns widened to float64 equals
    torch's own bfloat16 -> float64 conversion (NaN patterns give NaN, the
    two zeros keep their signs), and known values sit at their patterns."""
    fn = fn or elbo.bf16_to_f64
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    with np.errstate(invalid="ignore"):       # signalling-NaN patterns
        got = np.asarray(fn(bits), dtype=np.float64)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    assert got.shape == ref.shape
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))
    # 1.0 = 0x3F80, -2.0 = 0xC000, the smallest subnormal 2^-133 = 0x0001
    assert fn(np.array([0x3F80, 0xC000, 0x0001], dtype=np.uint16)).tolist() == [1.0, -2.0, 2.0 ** -133]
    # a 2-D array keeps its shape
    with np.errstate(invalid="ignore"):
        assert np.asarray(fn(bits.reshape(256, 256))).shape == (256, 256)


def test_bf16_widening_matches_torch_on_every_pattern():
    check_bf16_widening()
