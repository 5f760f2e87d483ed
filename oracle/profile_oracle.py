"""Plain CPU oracle of the acceptance-profile statistics (test infrastructure).

This file is test infrastructure, like the rest of ``oracle/``: only the test
suite, the smoke check and the benchmark's CPU-baseline leg may use it, and
it imports nothing from the library.

It computes, in float64 and in the paper's order, what the decoder's
acceptance profile implies for decoding efficiency and for the position
weights of the proposal objective:

1. the acceptance profile a_i from observed accepted-prefix lengths: one
   minus the rejection rate at position i among the blocks whose
   verification reaches position i (Appendix "Brisk Backbone", the estimate
   used for Eq. idlm_tpf_instantiation; Section 3.2);
2. survival A_k = prod_{j<=k} a_j and the accepted-prefix law
   Pr(L = k) = A_k (1 - a_{k+1}) for k < M, A_M for k = M (Eq. nonuniform_tpf);
3. tokens per forward, TPF = sum_k Pr(L=k) g_k / sum_k Pr(L=k) c_k, and
   FPT = 1 / TPF (Eq. nonuniform_tpf), with the ISD instantiation
   TPF = (2 + sum_{k=1}^{M-1} A_k) / (2 - A_M), M = N - 1
   (Eq. idlm_tpf_instantiation) and its uniform-rejection special case
   TPF_N(r) (the stride equation of Section 2.2);
4. the risk-reward position weights w_i^raw = -dFPT/dz_i with the log-odds
   z_i = log(a_i / (1 - a_i)), and their mean-one normalisation
   w_i = M w_i^raw / (sum_j w_j^raw + eps) (Eq. brisk_weighting).

Readings (also in the design notes): R18 a position that no block reaches
has a_i = 1 (no rejection observed; it only matters when no block was
observed at all); R19 accepted-prefix lengths outside [0, M] are clamped
into it; R20 the derivative in item 4 is taken of the ISD FPT, as the paper
does in all its experiments.

Parity pins: the printed values of the stride equation (TPF 8, 4.09, 3.29,
2.77 at N = 8 and r = 0, 0.10, 0.15, 0.20); the stated reduction of the
general form to the ISD instantiation and to 1 + sum_k A_k; E[L] = sum_k A_k;
exact recovery of a rational profile from constructed counts; central finite
differences of FPT in z for the weights.
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence

import numpy as np

__all__ = [
    "accept_profile", "survival", "prefix_law", "tpf_general", "tpf_isd", "tpf_stride",
    "fpt_isd", "risk_reward_weights", "profile_summary",
]


def accept_profile(accept_len: Sequence[int], M: int) -> Dict[str, np.ndarray]:
    """Position-wise acceptance from accepted-prefix lengths L_b in [0, M].

    Block b reaches positions 1..min(L_b + 1, M) and is rejected at position
    L_b + 1 when L_b < M.  a_i = 1 - rejected_i / reached_i.
    """
    L = np.clip(np.asarray(accept_len, dtype=np.int64), 0, M)
    reach = np.zeros(M, dtype=np.int64)
    rej = np.zeros(M, dtype=np.int64)
    for i in range(1, M + 1):              # position i (1-based)
        reach[i - 1] = np.count_nonzero(L >= i - 1)
        rej[i - 1] = np.count_nonzero(L == i - 1)
    a = np.ones(M, dtype=np.float64)
    seen = reach > 0
    a[seen] = 1.0 - rej[seen] / reach[seen]
    return dict(a=a, reach=reach, rej=rej)


def survival(a: np.ndarray) -> np.ndarray:
    """A_k for k = 0..M (A_0 = 1)."""
    A = np.ones(len(a) + 1, dtype=np.float64)
    for k in range(1, len(a) + 1):
        A[k] = A[k - 1] * a[k - 1]
    return A


def prefix_law(a: np.ndarray) -> np.ndarray:
    """Pr(L = k), k = 0..M."""
    M = len(a)
    A = survival(a)
    p = np.empty(M + 1, dtype=np.float64)
    for k in range(M):
        p[k] = A[k] * (1.0 - a[k])
    p[M] = A[M]
    return p


def tpf_general(a: np.ndarray, g: np.ndarray, c: np.ndarray) -> float:
    """Renewal-reward tokens per forward with committed tokens g_k and cost c_k."""
    p = prefix_law(a)
    return float(np.dot(p, g) / np.dot(p, c))


def tpf_isd(a: np.ndarray) -> float:
    """ISD instantiation: (2 + sum_{k=1}^{M-1} A_k) / (2 - A_M)."""
    A = survival(a)
    M = len(a)
    return float((2.0 + A[1:M].sum()) / (2.0 - A[M]))


def fpt_isd(a: np.ndarray) -> float:
    return 1.0 / tpf_isd(a)


def tpf_stride(N: int, r: float) -> float:
    """Stride-N tokens per forward under a uniform rejection rate r."""
    s = 1.0 - r
    num = 2.0 + sum(s ** i for i in range(1, N - 1))
    return num / (2.0 - s ** (N - 1))


def risk_reward_weights(a: np.ndarray, eps: float = 0.0) -> Dict[str, np.ndarray]:
    """w^raw_i = -dFPT/dz_i of the ISD FPT and the mean-one weights.

    With Num = 2 + sum_{k=1}^{M-1} A_k and Den = 2 - A_M, FPT = Den / Num.
    dA_k/da_i = A_k / a_i for k >= i, so dNum/da_i = S_i / a_i with
    S_i = sum_{k=i}^{M-1} A_k and dDen/da_i = -A_M / a_i; da_i/dz_i =
    a_i (1 - a_i).  The factors of a_i cancel:
    w^raw_i = (1 - a_i) (A_M Num + Den S_i) / Num^2.
    """
    a = np.asarray(a, dtype=np.float64)
    M = len(a)
    A = survival(a)
    num = 2.0 + A[1:M].sum()
    den = 2.0 - A[M]
    raw = np.empty(M, dtype=np.float64)
    for i in range(1, M + 1):
        S_i = A[i:M].sum()                      # k = i..M-1
        raw[i - 1] = (1.0 - a[i - 1]) * (A[M] * num + den * S_i) / (num * num)
    w = M * raw / (raw.sum() + eps)
    return dict(raw=raw, w=w)


def profile_summary(accept_len: Sequence[int], M: int, eps: float = 0.0) -> Dict[str, np.ndarray]:
    """Everything the GPU statistics call reports, from accepted-prefix lengths."""
    prof = accept_profile(accept_len, M)
    rw = risk_reward_weights(prof["a"], eps)
    tpf = tpf_isd(prof["a"])
    return dict(a=prof["a"], reach=prof["reach"], rej=prof["rej"], raw=rw["raw"], w=rw["w"],
                tpf=tpf, fpt=1.0 / tpf)
