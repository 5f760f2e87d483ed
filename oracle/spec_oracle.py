"""Plain CPU oracle of stochastic speculative verification (test infrastructure).

This file is test infrastructure, like the rest of ``oracle/``: only the test
suite, the smoke check and the benchmark's CPU-baseline leg may use it, and
it imports nothing from the library.

Section 3.3: a proposal x_i drawn from the proposal law pi_i over the
candidate set is accepted with probability min{1, p_i(x_i) / pi_i(x_i)},
where p_i is the frozen causal verifier distribution (here the softmax of the
verifier's full-vocabulary logits at temperature T); on rejection a token is
drawn from the normalised positive part [p_i - pi_i]_+, which leaves the
committed token distributed exactly as p_i.  The block stops at its first
rejection (Algorithm 1(b) verify and commit).

Random numbers.  The accept test takes a uniform u_i per position as an
input.  The residual draw uses the Gumbel-max form
    y_i = argmax_v [ log w_i(v) + G_{i,v} ],  w_i = [p_i - pi_i]_+ ,
with one Gumbel variate per (row, token) from the Philox4x32-10 counter-based
generator (Salmon, Moraes, Dror and Shaw, SC'11), which both sides implement
from its published definition: ten rounds of two 32x32->64-bit products with
the multipliers 0xD2511F53 and 0xCD9E8D57 and a Weyl key schedule with
increments 0x9E3779B9 and 0xBB67AE85.  Token v of row i uses output word
v mod 4 of the block counter (v div 4, i, 0, 0) under the key (seed low
word, seed high word); the word u maps to U = (floor(u / 512) + 1/2) / 2^23,
a value strictly inside (0, 1) that single precision holds exactly, and
G = -log(-log U).

Readings (also in the design notes): R21 p_i is the verifier softmax at
temperature T over the whole vocabulary; R22 pi_i is given as probabilities
over the position's candidate ids (a token outside the candidates has
pi = 0); when none are given, the proposer is the greedy selection of
Section 3.3, whose law is the point mass at x_i (if x_i is a candidate);
R23 accept when u_i < min{1, p_i(x_i) / pi_i(x_i)}; R24 a fully accepted
block has no correction (-1), as in the greedy rule.

Parity pins: the committed token's distribution equals p_i (chi-square over
many seeded trials, for a one-hot and a spread proposal law); acceptance
frequencies match sum_v min{p_v, pi_v}; the generator's words are uniform
(chi-square) and the Gumbel maximum reproduces the softmax.
"""
from __future__ import annotations

from typing import Dict, Tuple

import numpy as np

__all__ = ["philox4x32_10", "gumbel_for", "verifier_log_probs", "spec_rows", "spec_verify"]

_M0, _M1 = np.uint64(0xD2511F53), np.uint64(0xCD9E8D57)
_W0, _W1 = np.uint32(0x9E3779B9), np.uint32(0xBB67AE85)
_MASK = np.uint64(0xFFFFFFFF)


def philox4x32_10(ctr: np.ndarray, key: Tuple[int, int]) -> np.ndarray:
    """Philox4x32-10 of counters ``ctr`` [..., 4] uint32 under ``key``."""
    c = np.asarray(ctr, dtype=np.uint32).copy()
    k0 = np.uint32(key[0] & 0xFFFFFFFF)
    k1 = np.uint32(key[1] & 0xFFFFFFFF)
    with np.errstate(over="ignore"):
        for _ in range(10):
            p0 = _M0 * c[..., 0].astype(np.uint64)
            p1 = _M1 * c[..., 2].astype(np.uint64)
            hi0, lo0 = (p0 >> np.uint64(32)).astype(np.uint32), (p0 & _MASK).astype(np.uint32)
            hi1, lo1 = (p1 >> np.uint64(32)).astype(np.uint32), (p1 & _MASK).astype(np.uint32)
            c = np.stack([hi1 ^ c[..., 1] ^ k0, lo1, hi0 ^ c[..., 3] ^ k1, lo0], axis=-1)
            k0 = np.uint32(k0 + _W0)
            k1 = np.uint32(k1 + _W1)
    return c


def gumbel_for(rows: np.ndarray, V: int, seed: int) -> np.ndarray:
    """G[row, v] for the given row indices and every token v < V (float64)."""
    rows = np.asarray(rows, dtype=np.uint32)
    nb = (V + 3) // 4
    ctr = np.zeros((len(rows), nb, 4), dtype=np.uint32)
    ctr[..., 0] = np.arange(nb, dtype=np.uint32)[None, :]
    ctr[..., 1] = rows[:, None]
    words = philox4x32_10(ctr, (seed & 0xFFFFFFFF, seed >> 32)).reshape(len(rows), nb * 4)[:, :V]
    U = ((words >> np.uint32(9)).astype(np.float64) + 0.5) / float(1 << 23)
    return -np.log(-np.log(U))


def verifier_log_probs(logits: np.ndarray, T: float) -> np.ndarray:
    """log p_i(v): log-softmax of logits / T over the vocabulary (float64)."""
    s = np.asarray(logits, dtype=np.float64) / T
    m = s.max(axis=1, keepdims=True)
    return s - m - np.log(np.exp(s - m).sum(axis=1, keepdims=True))


def spec_rows(logits: np.ndarray, T: float, x: np.ndarray, cand_id: np.ndarray, cand_prob: np.ndarray,
              u: np.ndarray, seed: int, row_ids: np.ndarray = None) -> Dict[str, np.ndarray]:
    """Per position: accept decision for x_i and the residual draw y_i.

    ``logits`` [rows, V] are the verifier's logits (float32 values), ``x``
    [rows] the proposals, ``cand_id`` / ``cand_prob`` [rows, K] the proposal
    law (``cand_prob=None``: point mass at x among the candidates), ``u``
    [rows] the accept uniforms.  ``row_ids`` are the generator row indices
    (default 0..rows-1).
    """
    rows, V = logits.shape
    logp = verifier_log_probs(logits, T)
    p = np.exp(logp)
    pi = np.zeros((rows, V), dtype=np.float64)
    K = cand_id.shape[1]
    ar = np.arange(rows)
    if cand_prob is None:
        cand_prob = (cand_id == np.asarray(x)[:, None]).astype(np.float64)
    np.add.at(pi, (np.repeat(ar, K), cand_id.reshape(-1)),
              np.asarray(cand_prob, dtype=np.float64).reshape(-1))
    px, pix = p[ar, x], pi[ar, x]
    ratio = np.where(pix > 0, px / np.where(pix > 0, pix, 1.0), np.inf)
    accept = u < np.minimum(1.0, ratio)
    w = np.maximum(p - pi, 0.0)
    with np.errstate(divide="ignore"):
        score = np.log(w) + gumbel_for(ar if row_ids is None else row_ids, V, seed)
    resample = np.argmax(score, axis=1).astype(np.int32)
    return dict(accept=accept, resample=resample, p_x=px, pi_x=pix, p=p, pi=pi)


def spec_verify(logits: np.ndarray, T: float, proposal: np.ndarray, cand_id: np.ndarray,
                cand_prob: np.ndarray, u: np.ndarray, seed: int) -> Dict[str, np.ndarray]:
    """Blocks [B, L]: accepted-prefix length and the token committed at the
    first rejection (-1 when every position is accepted)."""
    B, L = proposal.shape
    rs = spec_rows(logits, T, proposal.reshape(-1), cand_id, cand_prob, u.reshape(-1), seed)
    acc_rows = rs["accept"].reshape(B, L)
    accept = np.full(B, L, np.int32)
    correction = np.full(B, -1, np.int32)
    for b in range(B):
        for i in range(L):
            if not acc_rows[b, i]:
                accept[b] = i
                correction[b] = rs["resample"][b * L + i]
                break
    return dict(accept_len=accept, correction=correction, row_accept=rs["accept"],
                row_resample=rs["resample"])
