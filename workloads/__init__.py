"""Seeded synthetic inputs for the BGPO masked-diffusion ELBO head.

This module draws the *inputs* only: hidden states, LM-head weights, target
tokens, response-length masks and per-response advantages.  It holds none of
the method's arithmetic (no timestep draw, no masking, no log-softmax, no
bound); those live separately in the float64 oracle and in the HIP path,
which both consume the arrays produced here.

The paper trains LLaDA-8B-Instruct with response length 512 (math, code) or
256 (planning), G = 8 responses per prompt and n_t = 16 or 32 Monte-Carlo
samples (Section 4.1 and Table 5).  Its datasets and trained weights are not
used; the workloads below stand in for them with the LLaDA head shape
d = 4096, V = 126464, uniform response lengths, Zipf(1.1) target tokens and
N(0, 0.02^2) head weights.

Rounding to bfloat16 is round-to-nearest-even on the float32 bit pattern, so
both consumers see exactly the same bf16 values.
"""
from __future__ import annotations

import dataclasses
from typing import Optional, Tuple

import numpy as np

T_IID = 0
T_STRATIFIED = 1


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and value distributions of one synthetic ELBO-head problem."""

    name: str
    B: int                      # responses in the batch (G per prompt)
    L: int                      # padded response length
    d: int                      # hidden size
    V: int                      # vocabulary size
    n_t: int                    # Monte-Carlo samples per response
    t_mode: int = T_IID         # T_IID: t ~ U(0,1); T_STRATIFIED: t_k = (k+u)/n_t
    hidden: str = "rmsnorm"     # "normal": N(0,1); "rmsnorm": N(0,1) then per-row RMS normalisation
    targets: str = "zipf"       # "uniform" over V or "zipf" (exponent 1.1)
    lengths: Optional[Tuple[int, int]] = None   # inclusive uniform response length; None = all L
    adv: str = "group"          # "normal": N(0,1) per response; "group": group-normalised over G
    group: int = 8              # G for group-normalised advantages
    w_std: float = 0.02         # head weight standard deviation
    data_seed: int = 1000       # numpy PCG64 seed
    philox_seed: int = 0xB6B00000
    seq_id_base: int = 0

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five problem sizes used throughout: a tiny correctness case, the
# LLaDA-8B head shape at response length 256 and 512 (uniform and ragged
# lengths), the large-MC regime n_t = 64, and a long-response stress case
# with stratified timesteps.
TINY = Workload("tiny_B2_L64_d128_V1024_nt4", B=2, L=64, d=128, V=1024, n_t=4,
                hidden="normal", targets="uniform", adv="normal",
                data_seed=1001, philox_seed=0xB6B00001)
LLADA_L256 = Workload("llada_head_B8_L256_nt16", B=8, L=256, d=4096, V=126464, n_t=16,
                      data_seed=1002, philox_seed=0xB6B00002)
LLADA_L512_RAGGED = Workload("llada_head_B8_L512_ragged_nt16", B=8, L=512, d=4096, V=126464,
                             n_t=16, lengths=(128, 512), data_seed=1003,
                             philox_seed=0xB6B00003)
LLADA_L512_NT64 = Workload("llada_head_B8_L512_nt64", B=8, L=512, d=4096, V=126464, n_t=64,
                           data_seed=1004, philox_seed=0xB6B00004)
STRESS_L1024 = Workload("llada_head_B16_L1024_ragged_nt32_stratified", B=16, L=1024, d=4096,
                        V=126464, n_t=32, t_mode=T_STRATIFIED, lengths=(256, 1024),
                        adv="normal", data_seed=1005, philox_seed=0xB6B00005)

CONFIGS = (TINY, LLADA_L256, LLADA_L512_RAGGED, LLADA_L512_NT64, STRESS_L1024)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest, ties to even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounded = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns to float32 (exact)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _zipf_tokens(rng: np.random.Generator, V: int, n: int, exponent: float = 1.1) -> np.ndarray:
    """Zipf(exponent) over V ranks by inverse CDF, then a seeded permutation of token ids."""
    ranks = np.arange(1, V + 1, dtype=np.float64)
    cdf = np.cumsum(ranks ** (-exponent))
    cdf /= cdf[-1]
    u = rng.random(n)
    r = np.minimum(np.searchsorted(cdf, u, side="right"), V - 1)
    perm = rng.permutation(V)
    return perm[r].astype(np.int32)


_CHUNK_ROWS = 1024


def _chunked(seed_seq, n_rows, fill, rows=_CHUNK_ROWS):
    """Fill rows [0, n_rows) in fixed chunks of ``rows``, chunk c drawing from
    its own stream spawned from ``seed_seq``; threads only change the speed."""
    import concurrent.futures as cf
    import os
    starts = list(range(0, n_rows, rows))
    seqs = seed_seq.spawn(len(starts))
    jobs = [(c, np.random.Generator(np.random.PCG64(q))) for c, q in zip(starts, seqs)]
    workers = max(1, min(16, len(os.sched_getaffinity(0))))
    with cf.ThreadPoolExecutor(workers) as ex:
        list(ex.map(lambda a: fill(*a), jobs))


def generate(w: Workload, *, with_weights: bool = True, with_hidden: bool = True,
             keep_f32: bool = False) -> dict:
    """Draw every input of workload ``w`` from numpy PCG64 streams spawned from
    ``w.data_seed`` (one stream per input, so W or hidden can be skipped).

    Returns a dict of numpy arrays:
      hidden    uint16 [B, L, d]  bf16 bits, row-major
      W         uint16 [d, V]     bf16 bits, row-major (V contiguous)
      targets   int32  [B, L]     target token per position (defined on padding too)
      resp_mask uint8  [B, L]     1 on response positions, 0 on padding
      adv       float32 [B]       per-response advantage
    plus ``lengths`` (int32 [B]).  ``keep_f32`` also returns the float32
    values before rounding as ``hidden_f32`` [B, L, d] and ``W_f32`` [d, V]
    (the rounded bits are those values rounded to nearest even).
    """
    # independent streams per input, so that any subset can be drawn alone
    ss = np.random.SeedSequence(w.data_seed).spawn(5)
    r_h, r_w, r_y, r_len, r_adv = (np.random.Generator(np.random.PCG64(s)) for s in ss)
    B, L, d, V = w.B, w.L, w.d, w.V

    hidden = None
    hidden_f32 = np.empty((B * L, d), dtype=np.float32) if (with_hidden and keep_f32) else None
    W_f32 = np.empty((d, V), dtype=np.float32) if (with_weights and keep_f32) else None
    if with_hidden:
        hidden = np.empty((B * L, d), dtype=np.uint16)

        def fill_h(c, rng):
            h = rng.standard_normal((min(B * L, c + _CHUNK_ROWS) - c, d), dtype=np.float32)
            if w.hidden == "rmsnorm":
                rms = np.sqrt(np.mean(h.astype(np.float64) ** 2, axis=-1, keepdims=True) + 1e-6)
                h = (h / rms).astype(np.float32)
            hidden[c:c + h.shape[0]] = f32_to_bf16_bits(h).reshape(h.shape)
            if hidden_f32 is not None:
                hidden_f32[c:c + h.shape[0]] = h

        _chunked(ss[0], B * L, fill_h)
        hidden = hidden.reshape(B, L, d)

    W = None
    if with_weights:
        W = np.empty((d, V), dtype=np.uint16)
        rows = max(1, (_CHUNK_ROWS * 512) // V)

        def fill_w(c, rng):
            n = min(d, c + rows) - c
            chunk = rng.standard_normal((n, V), dtype=np.float32) * np.float32(w.w_std)
            W[c:c + n] = f32_to_bf16_bits(chunk).reshape(n, V)
            if W_f32 is not None:
                W_f32[c:c + n] = chunk

        _chunked(ss[1], d, fill_w, rows)

    if w.targets == "uniform":
        targets = r_y.integers(0, V, size=(B, L), dtype=np.int64).astype(np.int32)
    else:
        targets = _zipf_tokens(r_y, V, B * L).reshape(B, L)

    if w.lengths is None:
        lengths = np.full(B, L, dtype=np.int32)
    else:
        lo, hi = w.lengths
        lengths = r_len.integers(lo, hi + 1, size=B, dtype=np.int64).astype(np.int32)
    resp_mask = (np.arange(L)[None, :] < lengths[:, None]).astype(np.uint8)

    r = r_adv.standard_normal(B)
    if w.adv == "group":
        G = w.group
        adv = np.empty(B, dtype=np.float64)
        for g0 in range(0, B, G):
            rg = r[g0:g0 + G]
            adv[g0:g0 + G] = (rg - rg.mean()) / (rg.std() + 1e-6)   # population std
        adv = adv.astype(np.float32)
    else:
        adv = r.astype(np.float32)

    out = dict(hidden=hidden, W=W, targets=targets, resp_mask=resp_mask, adv=adv,
               lengths=lengths)
    if keep_f32:
        out["hidden_f32"] = None if hidden_f32 is None else hidden_f32.reshape(B, L, d)
        out["W_f32"] = W_f32
    return out


def pre_norm_activations(w: Workload, n_samples: int = 0) -> np.ndarray:
    """Activations x in front of the final RMSNorm, as bf16 bits: N(0, 1)
    entries times a per-row scale drawn log-uniformly from [1/4, 4] (so the
    norm's 1/rms varies across rows).  ``n_samples`` = 0 gives one tensor
    [B, L, d] shared by all samples, n > 0 gives [n, B, L, d], sample q from
    its own stream."""
    B, L, d = w.B, w.L, w.d
    base = np.random.SeedSequence(w.data_seed).spawn(7)[5]
    n = max(1, n_samples)
    out = np.empty((n, B * L, d), dtype=np.uint16)
    for q, sq in enumerate(base.spawn(n)):
        def fill(c, rng, q=q):
            rows = min(B * L, c + _CHUNK_ROWS) - c
            scale = np.exp(rng.uniform(np.log(0.25), np.log(4.0), size=(rows, 1))).astype(np.float32)
            x = rng.standard_normal((rows, d), dtype=np.float32) * scale
            out[q, c:c + rows] = f32_to_bf16_bits(x).reshape(rows, d)
        _chunked(sq, B * L, fill)
    out = out.reshape(n, B, L, d)
    return out[0] if n_samples == 0 else out


def norm_weight(w: Workload) -> np.ndarray:
    """Final-RMSNorm weight, float32 [d]: 1 + 0.1 N(0, 1)."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(w.data_seed).spawn(7)[6]))
    return (1.0 + 0.1 * rng.standard_normal(w.d)).astype(np.float32)
