"""GPU checks of stochastic speculative verification (brisk_spec_verify):
decision parity with the CPU oracle on the same inputs and random numbers,
and the distribution of the committed token (it must be the verifier's p)."""
import numpy as np
import pytest
import torch
from scipy import stats

import oracle
import synth

pytestmark = pytest.mark.gpu

brisk = pytest.importorskip("paper_2609_33390_amd")

CHI_P = 1e-4


def _softmax(x, axis=-1):
    e = np.exp(x - x.max(axis=axis, keepdims=True))
    return e / e.sum(axis=axis, keepdims=True)


RAGGED = synth.Workload("ragged-d200-v1003", B=4, L=16, d=200, V=1003, K=5, r=32,
                        sigma=0.3, flat_frac=0.0, seed=7)
# the largest K, with a single token outside the candidates
EDGE = synth.Workload("edge-k64-v65", B=3, L=8, d=64, V=65, K=64, r=32,
                      sigma=0.3, flat_frac=0.0, seed=8)


def _workload(name):
    return {RAGGED.name: RAGGED, EDGE.name: EDGE}.get(name) or synth.WORKLOADS[name]


def _setup(wl, T, seed, law="candidates", mix=0.3):
    """Proposal law over the proposer's top-K: the softmax of its logits at
    temperature T mixed with the uniform law (weight ``mix``), or uniform;
    x drawn from it, u ~ U(0, 1), verifier rows bf16(H + 0.3 N(0, 1))."""
    blk = synth.make_block(wl, "cuda")
    rows = wl.rows
    cl, ci = brisk.propose_block(blk.H, blk.W, wl.K)
    g = torch.Generator(device="cuda").manual_seed(seed)
    Hv = (blk.H.float() + 0.3 * torch.randn(blk.H.shape, generator=g, device="cuda")).to(torch.bfloat16)
    rng = np.random.default_rng(seed)
    cln, cin = cl.cpu().numpy().astype(np.float64), ci.cpu().numpy()
    if law == "candidates":
        prob = (1.0 - mix) * _softmax(cln / T) + mix / wl.K
    else:
        prob = np.full(cln.shape, 1.0 / wl.K)
    pick = np.array([rng.choice(wl.K, p=prob[r] / prob[r].sum()) for r in range(rows)])
    x = cin[np.arange(rows), pick].reshape(wl.B, wl.L).astype(np.int32)
    u = rng.random(rows).astype(np.float32)
    return blk, Hv, cin, prob.astype(np.float32), x, u


# Bound on |log p_gpu - log p_oracle|: fp32 logits (accumulation order) and
# an fp32 log-sum-exp over the vocabulary.  The measured error is ~1e-6 at
# d = 64 and ~1e-5 at d = 4096; the bound leaves an order of magnitude.
LOGP_ERR = 2e-4
G_ERR = 1e-4  # fp32 Gumbel variates against the float64 ones


def _oracle_margins(logits, T, cid, prob, x, u, seed, row_ids):
    """Oracle decisions plus which of them are well conditioned.

    Accept: u must be farther from min{1, p/pi} than the error p carries.
    Residual: where p and pi nearly cancel, w = [p - pi]_+ is not determined
    by fp32 inputs, so each token's score is taken as an interval over
    log p +- LOGP_ERR (and G +- G_ERR); a row is sure when the oracle's winner
    beats every other token over the whole interval.
    """
    pr = None if prob is None else prob.astype(np.float64)
    rs = oracle.spec_rows(logits, T, x, cid, pr, u.astype(np.float64), seed, row_ids)
    ratio = np.where(rs["pi_x"] > 0, rs["p_x"] / np.maximum(rs["pi_x"], 1e-300), np.inf)
    lim = np.minimum(1.0, ratio)
    sure_a = np.abs(u - lim) > 2 * LOGP_ERR * np.where(np.isfinite(lim), lim, 1.0) + 1e-6
    lp = np.log(rs["p"])
    G = oracle.gumbel_for(row_ids, logits.shape[1], seed)
    with np.errstate(divide="ignore"):
        # p <= 1 exactly, on both sides, so pi = 1 leaves no weight at all
        lo = np.log(np.maximum(np.minimum(np.exp(lp - LOGP_ERR), 1.0) - rs["pi"], 0.0)) + G - G_ERR
        hi = np.log(np.maximum(np.minimum(np.exp(lp + LOGP_ERR), 1.0) - rs["pi"], 0.0)) + G + G_ERR
    ar = np.arange(len(x))
    win = rs["resample"]
    hi_other = hi.copy()
    hi_other[ar, win] = -np.inf
    sure_r = lo[ar, win] > hi_other.max(axis=1)
    return rs, sure_a, sure_r


@pytest.mark.parametrize("name,T,law,n_sample", [
    ("tiny-d64-v512", 1.0, "candidates", 0),     # draws land on candidates
    ("tiny-d64-v512", 0.6, "uniform", 0),
    ("tiny-d64-v512", 4.0, "uniform", 0),        # draws land off the candidates
    ("ragged-d200-v1003", 2.0, "candidates", 0),  # ragged d and V, K + 1 = 6
    ("ragged-d200-v1003", 6.0, "uniform", 0),     # ... with draws off the candidates
    ("edge-k64-v65", 8.0, "uniform", 0),          # K = 64, one non-candidate token
    ("llada8b-b1-l32", 1.0, "candidates", 0),
    ("llada8b-b1-l32", 3.0, "uniform", 0),
    ("dream7b-b16-l32", 1.0, "candidates", 40),  # K + 1 = 17, flat rows; sampled rows
    # the batched shapes the benchmark times: 8 and 16 row tiles of the
    # large-row tile; sampled rows plus the first and last of every row tile
    pytest.param("llada8b-b64-l32", 1.0, "candidates", 32, marks=pytest.mark.slow),
    pytest.param("llada8b-b256-l16", 2.0, "uniform", 16, marks=pytest.mark.slow),
])
def test_spec_decisions_match_oracle(name, T, law, n_sample):
    wl = _workload(name)
    seed = 1234567 + int(T * 10)
    blk, Hv, cid, prob, x, u = _setup(wl, T, 11, law)
    out = brisk.spec_verify(Hv, blk.W, torch.from_numpy(x).cuda(), torch.from_numpy(cid).cuda(),
                            torch.from_numpy(prob).cuda(), torch.from_numpy(u).cuda(), seed, T)
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in out.items()}
    if n_sample == 0:
        sel = np.arange(wl.rows)
    else:  # random rows, and the first and last row of every 256-row tile
        edges = {t for t0 in range(0, wl.rows, 256) for t in (t0, min(t0 + 255, wl.rows - 1))}
        picked = np.random.default_rng(5).choice(wl.rows, n_sample, replace=False).tolist()
        sel = np.array(sorted(edges | set(picked)))
    print(f"[spec] {name} T={T} law={law}: oracle on {len(sel)} of {wl.rows} rows", flush=True)
    Hb = synth.bf16_bits(Hv)[sel]
    logits = oracle.lm_logits(oracle.bf16_to_f64(Hb), synth.bf16_bits(blk.W))
    rs, sure_a, sure_r = _oracle_margins(logits, T, cid[sel], prob[sel], x.reshape(-1)[sel], u[sel], seed, sel)
    assert sure_a.mean() > 0.9 and sure_r.mean() > 0.5, (sure_a.mean(), sure_r.mean())
    assert np.array_equal(g["row_accept"][sel][sure_a].astype(bool), rs["accept"][sure_a])
    assert np.array_equal(g["row_resample"][sel][sure_r], rs["resample"][sure_r])
    # block outcome from the GPU's own row decisions
    acc_rows = g["row_accept"].reshape(wl.B, wl.L).astype(bool)
    for b in range(wl.B):
        a = int(np.argmin(acc_rows[b])) if not acc_rows[b].all() else wl.L
        assert g["accept_len"][b] == a
        assert g["correction"][b] == (g["row_resample"][b * wl.L + a] if a < wl.L else -1)


@pytest.mark.parametrize("name,T", [("tiny-d64-v512", 2.0), ("ragged-d200-v1003", 4.0), ("llada8b-b1-l32", 1.0)])
def test_spec_greedy_proposer(name, T):
    # cand_prob = NULL: the greedy proposer, pi = point mass at x; the result
    # must equal an explicit one-hot law bit for bit, and the oracle
    wl = _workload(name)
    seed = 4242
    blk, Hv, cid, _, _, u = _setup(wl, T, 17, "uniform")
    x = cid[:, 0].reshape(wl.B, wl.L).astype(np.int32).copy()  # the top candidate
    onehot = (cid == x.reshape(-1)[:, None]).astype(np.float32)
    args = (Hv, blk.W, torch.from_numpy(x).cuda(), torch.from_numpy(cid).cuda())
    ug = torch.from_numpy(u).cuda()
    a = brisk.spec_verify(*args, None, ug, seed, T)
    b = brisk.spec_verify(*args, torch.from_numpy(onehot).cuda(), ug, seed, T)
    torch.cuda.synchronize()
    for k in a:
        assert torch.equal(a[k], b[k]), k
    g = {k: v.cpu().numpy() for k, v in a.items()}
    logits = oracle.lm_logits(oracle.bf16_to_f64(synth.bf16_bits(Hv)), synth.bf16_bits(blk.W))
    sel = np.arange(wl.rows)
    rs, sure_a, sure_r = _oracle_margins(logits, T, cid, None, x.reshape(-1), u, seed, sel)
    assert sure_a.mean() > 0.9 and sure_r.mean() > 0.5, (sure_a.mean(), sure_r.mean())
    assert np.array_equal(g["row_accept"][sure_a].astype(bool), rs["accept"][sure_a])
    assert np.array_equal(g["row_resample"][sure_r], rs["resample"][sure_r])
    # a rejected proposal is never drawn again at its own position
    rej = g["row_accept"] == 0
    assert not np.any(g["row_resample"][rej] == x.reshape(-1)[rej])


def _chi2(counts, probs):
    n = counts.sum()
    keep = probs * n >= 5
    exp, obs = probs[keep] * n, counts[keep]
    if n - exp.sum() >= 5:
        exp, obs = np.append(exp, n - exp.sum()), np.append(obs, n - obs.sum())
    return stats.chisquare(obs, exp * obs.sum() / exp.sum()).pvalue


@pytest.mark.parametrize("law", ["spread", "onehot", "mismatched"])
def test_committed_token_follows_the_verifier_distribution(law):
    # one verifier row repeated n times: every trial is one block of length 1
    n, V, d, K, T = 200_000, 24, 64, 4, 0.8
    rng = np.random.default_rng(3)
    h = torch.from_numpy(rng.standard_normal(d).astype(np.float32)).to(torch.bfloat16)
    W = torch.from_numpy((rng.standard_normal((V, d)) * 0.3).astype(np.float32)).to(torch.bfloat16)
    Hv = h[None, :].repeat(n, 1).contiguous().cuda()
    Wd = W.contiguous().cuda()
    cand = np.array([5, 9, 2, 17], np.int32)
    prob = {"spread": [0.4, 0.3, 0.2, 0.1], "onehot": [1.0, 0, 0, 0], "mismatched": [0.05, 0.05, 0.1, 0.8]}[law]
    prob = np.array(prob, np.float32)
    x = cand[rng.choice(K, size=n, p=prob / prob.sum())].reshape(n, 1)
    u = rng.random(n).astype(np.float32)
    cid = np.repeat(cand[None, :], n, axis=0)
    cpr = np.repeat(prob[None, :], n, axis=0)
    out = brisk.spec_verify(Hv, Wd, torch.from_numpy(x).cuda(), torch.from_numpy(cid).cuda(),
                            torch.from_numpy(cpr).cuda(), torch.from_numpy(u).cuda(), 99, T)
    torch.cuda.synchronize()
    acc = out["accept_len"].cpu().numpy()
    cor = out["correction"].cpu().numpy()
    committed = np.where(acc == 1, x[:, 0], cor)
    logits = oracle.lm_logits(oracle.bf16_to_f64(synth.bf16_bits(Hv[:1].cpu())), synth.bf16_bits(W))
    p = np.exp(oracle.verifier_log_probs(logits, T)[0])
    assert _chi2(np.bincount(committed, minlength=V), p) > CHI_P
    pi = np.zeros(V)
    pi[cand] = prob
    rate = np.minimum(p, pi).sum()
    assert abs((acc == 1).mean() - rate) < 5 * np.sqrt(rate * (1 - rate) / n) + 1e-9


def test_spec_deterministic_and_seed_sensitive():
    # a flat verifier law (T = 6) so the residual draws depend on the seed
    wl = RAGGED
    blk, Hv, cid, prob, x, u = _setup(wl, 6.0, 5, "uniform")
    args = (Hv, blk.W, torch.from_numpy(x).cuda(), torch.from_numpy(cid).cuda(), torch.from_numpy(prob).cuda(),
            torch.zeros(wl.rows, device="cuda"))
    a = brisk.spec_verify(*args, 7, 6.0)
    b = brisk.spec_verify(*args, 7, 6.0)
    c = brisk.spec_verify(*args, 8, 6.0)
    torch.cuda.synchronize()
    assert torch.equal(a["row_resample"], b["row_resample"])
    assert not torch.equal(a["row_resample"], c["row_resample"])
