"""Pins for the oracle's Philox4x32-10 stream and the timestep / mask draws.

* Known-answer vectors published with the generator (tests/golden).
* The integer contract of the timestep grid: i.i.d. T24 in [1, 2^24);
  stratified T24 inside stratum j, i.e. t in [j/n_t, (j+1)/n_t).
* Statistics: the masking rate equals t (Section 2.1: each response token is
  masked with probability t), and output bytes are uniform.
"""
import os

import numpy as np
import pytest
from scipy import stats

from oracle import philox

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.txt")


def _kat():
    rows = []
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        w = [int(x, 16) for x in line.split()]
        rows.append((w[0:4], w[4:6], w[6:10]))
    return rows


@pytest.mark.parametrize("ctr,key,expect", _kat())
def test_known_answer_vectors(ctr, key, expect):
    assert [int(x) for x in philox.philox4x32_10(ctr, key)] == expect


def test_vectorised_equals_scalar():
    key = philox.seed_key(0x123456789ABCDEF0)
    ctrs = np.array([[i, 7, 3, 0] for i in range(16)], dtype=np.uint64)
    batch = philox.philox4x32_10(ctrs, key)
    for i in range(16):
        assert list(batch[i]) == list(philox.philox4x32_10(ctrs[i], key))


def test_t_grid_iid_range():
    Ts = [philox.t24_iid(0xB6B00004, s, j) for s in range(64) for j in range(64)]
    assert min(Ts) >= 1 and max(Ts) < (1 << 24)
    u = np.array(Ts) / 2.0 ** 24
    # uniform on (0,1): Kolmogorov-Smirnov
    assert stats.kstest(u, "uniform").pvalue > 1e-4


@pytest.mark.parametrize("n_t", [1, 3, 32, 64])
def test_t_grid_stratified_in_stratum(n_t):
    for s in range(16):
        u24 = philox.u24_stratified(0xB6B00005, s)
        for j in range(n_t):
            T = philox.t24_stratified(0xB6B00005, s, j, n_t)
            assert 1 <= T < (1 << 24)
            # t_j = (j + u)/n_t exactly floored on the 24-bit grid
            assert T == max(((j << 24) + u24) // n_t, 1)
            assert j * (1 << 24) <= T * n_t + n_t - 1 or T == 1
            assert T * n_t < (j + 1) * (1 << 24)


def test_mask_rate_matches_t():
    seed = 0xB6B00002
    L = 512
    resp = np.ones(L, dtype=np.uint8)
    resp[400:] = 0
    tot_m, tot_exp, var = 0, 0.0, 0.0
    for s in range(8):
        for j in range(32):
            T = philox.t24_iid(seed, s, j)
            t = T / 2.0 ** 24
            m = philox.mask_row(seed, s, j, T, resp)
            assert not m[400:].any()              # padding is never masked
            tot_m += int(m.sum())
            tot_exp += 400 * t
            var += 400 * t * (1 - t)
    z = (tot_m - tot_exp) / np.sqrt(var)
    assert abs(z) < 5.0


def test_mask_extremes():
    resp = np.ones(257, dtype=np.uint8)
    assert not philox.mask_row(1, 0, 0, 1, resp)[:8].all()
    # T24 = 2^24 would mask every position (used only as a test hook)
    assert philox.mask_row(1, 0, 0, 1 << 24, resp).all()


def test_output_bytes_uniform():
    ctr = np.zeros((4096, 4), dtype=np.uint64)
    ctr[:, 0] = np.arange(4096)
    ctr[:, 1] = 5
    w = philox.philox4x32_10(ctr, philox.seed_key(99)).reshape(-1)
    by = w.view(np.uint8)
    counts = np.bincount(by, minlength=256)
    assert stats.chisquare(counts).pvalue > 1e-4


def test_keys_and_counters_decorrelate():
    a = philox.mask_words(7, 0, 0, 1024)
    b = philox.mask_words(7, 1, 0, 1024)
    c = philox.mask_words(7, 0, 1, 1024)
    d = philox.mask_words(8, 0, 0, 1024)
    for x in (b, c, d):
        assert (a != x).mean() > 0.99
