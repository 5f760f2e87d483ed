"""Tie-aware comparison of GPU outputs with the oracle.

Floating-point tolerance: scores agree within 1e-2 absolute (bf16 inputs, fp32
accumulation); integer decisions (candidate ids, selected tokens, accept
lengths) must be identical wherever the oracle's relevant margin exceeds that
tolerance, and elsewhere the GPU's choice must be one the oracle scores within
the tolerance of the best.
"""
import numpy as np

SCORE_TOL = 1e-2


def check_gpu_order(cl, ci):
    """The GPU's own list is sorted by (logit desc, id asc) and has no repeats."""
    for r in range(cl.shape[0]):
        for k in range(cl.shape[1] - 1):
            a, b = cl[r, k], cl[r, k + 1]
            assert a > b or (a == b and ci[r, k] < ci[r, k + 1]), (r, k, a, b, ci[r, k], ci[r, k + 1])
        assert len(set(ci[r].tolist())) == cl.shape[1], r


def check_candidates(cl, ci, ol, tol=SCORE_TOL):
    """Compare GPU candidates (cl, ci) [n, K] with full oracle logit rows ol [n, V]."""
    n, K = ci.shape
    V = ol.shape[1]
    assert np.all((ci >= 0) & (ci < V))
    check_gpu_order(cl, ci)
    order = np.argsort(-ol, axis=1, kind="stable")[:, :K + 1]
    ov = np.take_along_axis(ol, order, axis=1).astype(np.float64)
    for r in range(n):
        got = ol[r, ci[r]].astype(np.float64)
        # the GPU's logit of each chosen token matches the oracle's logit of it
        assert np.max(np.abs(got - cl[r])) <= tol, (r, np.max(np.abs(got - cl[r])))
        # set: nothing chosen below the oracle's K-th value by more than tol,
        # and exact equality when the K / K+1 boundary is not a near-tie
        assert got.min() >= ov[r, K - 1] - tol, r
        if K < V and ov[r, K - 1] - ov[r, K] > tol:
            assert set(ci[r].tolist()) == set(order[r, :K].tolist()), r
        # order: exact wherever the oracle's neighbours are separated by > tol
        for k in range(K):
            left = k == 0 or ov[r, k - 1] - ov[r, k] > tol
            right = (k + 1 > K - 1 and (K >= V or ov[r, k] - ov[r, k + 1] > tol)) or \
                    (k + 1 <= K - 1 and ov[r, k] - ov[r, k + 1] > tol)
            if left and right:
                assert ci[r, k] == order[r, k], (r, k)


def check_rerank(gpu, orc, tol=SCORE_TOL, rel=0.0):
    """Conditional check: ``orc`` is the oracle run on the GPU's candidates with
    the GPU's selected prefix forced.  ``rel`` adds a relative part to the
    score bound: tol + rel * |gamma * d| per score (for corrector weights far
    beyond the workloads', where fp32 cannot reach the absolute bound)."""
    allowed = tol + rel * np.abs(orc["gamma"][:, None].astype(np.float64) * orc["resid"])
    r_err = np.abs(gpu["refined"].astype(np.float64) - orc["refined"])
    assert np.all(r_err <= allowed), (r_err.max(), np.max(np.abs(orc["refined"])))
    g_err = np.abs(gpu["gamma"].astype(np.float64) - orc["gamma"])
    assert np.all(g_err <= 1e-3 * np.abs(orc["gamma"]) + 1e-6), g_err.max()
    dmax = np.max(np.abs(orc["resid"]), axis=1, keepdims=True)
    d_err = np.abs(gpu["resid"].astype(np.float64) - orc["resid"])
    assert np.all(d_err <= 1e-3 * dmax + 1e-6), d_err.max()
    sel_g = gpu["selected"].ravel()
    sel_o = orc["selected"].ravel()
    sure = orc["margin"] > np.max(allowed, axis=1)
    assert np.array_equal(sel_g[sure], sel_o[sure])
    # near-ties: the GPU's pick scores within tol of the oracle's best
    return int((~sure).sum())


def rerank_pick_ok(gpu_sel, orc, cand_id, tol=SCORE_TOL, rel=0.0):
    """Every GPU pick is a candidate whose oracle refined score is within the
    score bound (tol, plus rel * max |gamma * d| of the row) of the best."""
    rows, K = cand_id.shape
    sel = gpu_sel.ravel()
    slack = tol + rel * np.max(np.abs(orc["gamma"][:, None].astype(np.float64) * orc["resid"]), axis=1)
    for r in range(rows):
        k = np.nonzero(cand_id[r] == sel[r])[0]
        assert k.size == 1, r
        assert orc["refined"][r, k[0]] >= orc["refined"][r].max() - slack[r], r
