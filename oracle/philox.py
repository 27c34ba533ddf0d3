"""Philox4x32-10 counter-based generator and the BGPO timestep / mask draws.

TEST INFRASTRUCTURE: this package is the float64 CPU oracle.  Only the test
suite, the smoke check and the benchmark's CPU-baseline leg may import it.

Philox4x32-10 follows its published definition (Salmon, Moraes, Dror, Shaw,
"Parallel random numbers: as easy as 1, 2, 3", SC'11): a 4 x 32-bit counter
and a 2 x 32-bit key; each of the 10 rounds multiplies counter words 0 and 2
by the two round multipliers, keeps the 64-bit products' high and low halves,
and mixes the high halves with the other two counter words and the key; the
key is advanced by two Weyl constants between rounds.  This implementation is
vectorised numpy on uint64 lanes.

How the method's random numbers are drawn from it (the paper states only the
distributions, so the counter layout is a reading):
  * key = (seed mod 2^32, seed div 2^32)
  * timestep t of response ``seq`` in Monte-Carlo sample ``j`` (Eq. mcs_elbo,
    t ~ U[0,1], one per sample and per response as in Algorithm 1):
      counter (0, seq, j, 1), word 0, T24 = max(word >> 8, 1), t = T24 * 2^-24
    so t lies on the exact 24-bit grid (0, 1) and 1/t is always finite;
  * stratified timesteps t_k = (k + u)/n_t with one u per response:
      counter (0, seq, 0, 2), word 0, U24 = word >> 8,
      T24 = max(floor((j * 2^24 + U24) / n_t), 1);
  * the forward masking process (Section 2.1: each response token is masked
    independently with probability t): position i of response ``seq`` in
    sample ``j`` is masked iff it is a response position and
      (word (i mod 4) of Philox(counter (i div 4, seq, j, 0))) >> 8 < T24,
    an integer comparison whose probability is exactly T24 * 2^-24 = t.
"""
from __future__ import annotations

import numpy as np

PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85
ROUNDS = 10
_MASK32 = np.uint64(0xFFFFFFFF)


def philox4x32_10(counter, key):
    """Philox4x32-10 of ``counter`` (array [..., 4] of uint32-valued ints) under
    ``key`` (two uint32 words).  Returns uint32 array [..., 4]."""
    c = np.asarray(counter, dtype=np.uint64) & _MASK32
    c0, c1, c2, c3 = (c[..., 0].copy(), c[..., 1].copy(), c[..., 2].copy(), c[..., 3].copy())
    k0 = np.uint64(int(key[0]) & 0xFFFFFFFF)
    k1 = np.uint64(int(key[1]) & 0xFFFFFFFF)
    m0 = np.uint64(PHILOX_M0)
    m1 = np.uint64(PHILOX_M1)
    for r in range(ROUNDS):
        if r:
            k0 = (k0 + np.uint64(PHILOX_W0)) & _MASK32
            k1 = (k1 + np.uint64(PHILOX_W1)) & _MASK32
        p0 = m0 * c0            # < 2^64, exact in uint64
        p1 = m1 * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & _MASK32
        hi1, lo1 = p1 >> np.uint64(32), p1 & _MASK32
        c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return np.stack([c0, c1, c2, c3], axis=-1).astype(np.uint32)


def seed_key(seed: int):
    seed = int(seed) & 0xFFFFFFFFFFFFFFFF
    return (seed & 0xFFFFFFFF, seed >> 32)


def t24_iid(seed: int, seq_id: int, j: int) -> int:
    """Integer timestep T24 in [1, 2^24) for i.i.d. t ~ U(0,1)."""
    w = philox4x32_10([0, seq_id & 0xFFFFFFFF, j, 1], seed_key(seed))[0]
    return max(int(w) >> 8, 1)


def u24_stratified(seed: int, seq_id: int) -> int:
    w = philox4x32_10([0, seq_id & 0xFFFFFFFF, 0, 2], seed_key(seed))[0]
    return int(w) >> 8


def t24_stratified(seed: int, seq_id: int, j: int, n_t: int) -> int:
    """Integer timestep for the stratified grid t_j = (j + u)/n_t, u shared by a response."""
    u24 = u24_stratified(seed, seq_id)
    return max(((j << 24) + u24) // n_t, 1)


def t24(seed: int, seq_id: int, j: int, n_t: int, t_mode: int) -> int:
    return t24_iid(seed, seq_id, j) if t_mode == 0 else t24_stratified(seed, seq_id, j, n_t)


def mask_words(seed: int, seq_id: int, j: int, L: int) -> np.ndarray:
    """The 32-bit Philox word that decides each of the L positions (uint32 [L])."""
    nblk = (L + 3) // 4
    ctr = np.zeros((nblk, 4), dtype=np.uint64)
    ctr[:, 0] = np.arange(nblk, dtype=np.uint64)
    ctr[:, 1] = seq_id & 0xFFFFFFFF
    ctr[:, 2] = j
    ctr[:, 3] = 0
    words = philox4x32_10(ctr, seed_key(seed)).reshape(-1)
    return words[:L]


def mask_row(seed: int, seq_id: int, j: int, T24: int, resp_row: np.ndarray) -> np.ndarray:
    """Boolean mask of one response in one sample: response position and (word>>8) < T24."""
    resp_row = np.asarray(resp_row)
    words = mask_words(seed, seq_id, j, resp_row.shape[0])
    return (resp_row != 0) & ((words >> np.uint32(8)) < np.uint32(T24))
