"""Pins of the stochastic speculative-verification oracle (CPU only): the
committed token must be distributed as the verifier's p, whatever the
proposal law (Section 3.3), checked by chi-square over seeded trials."""
import numpy as np
import pytest
from scipy import stats

import oracle

CHI_P = 1e-4   # reject only on overwhelming evidence; the seeds are fixed


def _chi2(counts, probs):
    n = counts.sum()
    keep = probs * n >= 5
    exp = probs[keep] * n
    obs = counts[keep]
    rest_e = n - exp.sum()
    rest_o = n - obs.sum()
    if rest_e >= 5:
        exp = np.append(exp, rest_e)
        obs = np.append(obs, rest_o)
    return stats.chisquare(obs, exp * obs.sum() / exp.sum()).pvalue


def test_philox_words_are_uniform():
    ctr = np.zeros((1 << 16, 4), dtype=np.uint32)
    ctr[:, 0] = np.arange(1 << 16)
    ctr[:, 1] = 7
    w = oracle.philox4x32_10(ctr, (12345, 678)).reshape(-1)
    counts = np.bincount(w >> np.uint32(24), minlength=256)
    assert stats.chisquare(counts).pvalue > CHI_P
    # distinct counters give distinct words (no trivial cycling)
    assert len(np.unique(w)) > 0.999 * len(w)


def test_gumbel_max_reproduces_softmax():
    rng = np.random.default_rng(0)
    logits = rng.standard_normal(10) * 2
    p = np.exp(logits - logits.max())
    p /= p.sum()
    rows = np.arange(100_000)
    G = oracle.gumbel_for(rows, 10, seed=99)
    draws = np.argmax(np.log(p)[None, :] + G, axis=1)
    assert _chi2(np.bincount(draws, minlength=10), p) > CHI_P


def _trial(logits, T, cand, prob, x_law_rng, n, seed):
    V = len(logits)
    K = len(cand)
    L = np.repeat(logits[None, :].astype(np.float32), n, axis=0)
    x = cand[x_law_rng.choice(K, size=n, p=prob)].astype(np.int32)
    u = x_law_rng.random(n)
    cid = np.repeat(cand[None, :], n, axis=0).astype(np.int32)
    cpr = np.repeat(prob[None, :], n, axis=0)
    out = oracle.spec_verify(L, T, x.reshape(n, 1), cid, cpr, u.reshape(n, 1), seed)
    committed = np.where(out["accept_len"] == 1, x, out["correction"])
    return committed, out, x


@pytest.mark.parametrize("T", [1.0, 0.7])
@pytest.mark.parametrize("law", ["spread", "onehot", "mismatched"])
def test_committed_token_is_distributed_as_p(T, law):
    rng = np.random.default_rng(5)
    V = 12
    logits = rng.standard_normal(V) * 1.5
    cand = np.array([3, 7, 1, 10])
    if law == "spread":
        prob = np.array([0.4, 0.3, 0.2, 0.1])
    elif law == "onehot":
        prob = np.array([1.0, 0.0, 0.0, 0.0])
    else:  # mass on tokens the verifier finds unlikely
        prob = np.array([0.05, 0.05, 0.1, 0.8])
    n = 200_000
    committed, out, x = _trial(logits, T, cand, prob, rng, n, seed=2024 + int(T * 10))
    p = np.exp(oracle.verifier_log_probs(logits[None, :].astype(np.float32), T)[0])
    assert _chi2(np.bincount(committed, minlength=V), p) > CHI_P
    # acceptance rate of the first position is sum_v min(p_v, pi_v)
    pi = np.zeros(V)
    pi[cand] = prob
    rate = np.minimum(p, pi).sum()
    acc = (out["accept_len"] == 1).mean()
    assert abs(acc - rate) < 5 * np.sqrt(rate * (1 - rate) / n) + 1e-12


def test_block_stops_at_first_rejection():
    rng = np.random.default_rng(8)
    B, L, V, K = 50, 6, 9, 3
    logits = rng.standard_normal((B * L, V)).astype(np.float32)
    cid = np.stack([rng.choice(V, K, replace=False) for _ in range(B * L)]).astype(np.int32)
    cpr = np.full((B * L, K), 1.0 / K)
    x = cid[np.arange(B * L), rng.integers(0, K, B * L)].reshape(B, L)
    u = rng.random((B, L))
    out = oracle.spec_verify(logits, 1.0, x, cid, cpr, u, seed=3)
    rows = oracle.spec_rows(logits, 1.0, x.reshape(-1), cid, cpr, u.reshape(-1), 3)
    for b in range(B):
        acc = rows["accept"][b * L:(b + 1) * L]
        a = int(np.argmin(acc)) if not acc.all() else L
        assert out["accept_len"][b] == a
        assert out["correction"][b] == (rows["resample"][b * L + a] if a < L else -1)


@pytest.mark.parametrize("T", [1.0, 2.5])
def test_greedy_proposer_point_mass(T):
    # no proposal probabilities: the proposer is the greedy selection, its law
    # the point mass at x; acceptance happens with probability p(x) and the
    # committed token is still distributed as p
    rng = np.random.default_rng(12)
    V, n = 10, 200_000
    logits = rng.standard_normal(V) * 1.2
    cand = np.array([4, 0, 8])
    x = np.full((n, 1), cand[1], np.int32)
    u = rng.random((n, 1))
    L = np.repeat(logits[None, :].astype(np.float32), n, axis=0)
    cid = np.repeat(cand[None, :], n, axis=0).astype(np.int32)
    out = oracle.spec_verify(L, T, x, cid, None, u, seed=77)
    committed = np.where(out["accept_len"] == 1, x[:, 0], out["correction"])
    p = np.exp(oracle.verifier_log_probs(logits[None, :].astype(np.float32), T)[0])
    assert _chi2(np.bincount(committed, minlength=V), p) > CHI_P
    rate = p[cand[1]]
    acc = (out["accept_len"] == 1).mean()
    assert abs(acc - rate) < 5 * np.sqrt(rate * (1 - rate) / n)
    # a rejected position never commits the proposal again
    assert not np.any(out["correction"][out["accept_len"] == 0] == cand[1])


def test_greedy_mode_equals_explicit_point_mass():
    rng = np.random.default_rng(13)
    rows, V, K = 64, 30, 5
    logits = rng.standard_normal((rows, V)).astype(np.float32) * 2
    cid = np.stack([rng.choice(V, K, replace=False) for _ in range(rows)]).astype(np.int32)
    x = cid[np.arange(rows), rng.integers(0, K, rows)]
    u = rng.random(rows)
    a = oracle.spec_rows(logits, 1.3, x, cid, None, u, 5)
    b = oracle.spec_rows(logits, 1.3, x, cid, (cid == x[:, None]).astype(np.float64), u, 5)
    assert np.array_equal(a["accept"], b["accept"]) and np.array_equal(a["resample"], b["resample"])
