"""GPU parity of the combined rerank + verification entry point.

``rerank_verify`` must return exactly what ``rerank`` followed by
``verify_accept`` returns: the same selections and scores bit for bit, and the
accept length and correction token of the first disagreement with the
verifier (Algorithm 1(b)), which the oracle recomputes from the selections.
The verifier rows are planted from the oracle's own selection so that accept
lengths cover every position of long blocks, across the 64-position chunks the
single-wavefront scan compares at once.  Shapes cover that scan (d_state <=
256, K <= 16) and the multi-wavefront scan followed by the verification kernel.

Corrector weights have std 0.1.  The score tolerance is absolute (1e-2), and
at std 0.3 with d_state 320 over 70 positions the residuals reach about 4e3
logits: the gate's fp32 dot product, whose terms cancel, then carries a
relative error near 1e-5, which puts refined scores about 1e-2 off.
"""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import synth
from oracle_io import oracle_inputs
from parity import SCORE_TOL, check_rerank, rerank_pick_ok

pytestmark = pytest.mark.gpu

brisk = pytest.importorskip("paper_2609_33390_amd")
DEV = "cuda"

CASES = [  # B, L, K, d, V, r (= d_state)
    (1, 8, 4, 64, 512, 32),         # tiny
    (3, 7, 5, 72, 1003, 32),        # ragged
    (4, 64, 8, 64, 700, 64),        # exactly one chunk
    (3, 65, 8, 64, 700, 64),        # one position past a chunk
    (5, 200, 8, 64, 900, 128),      # several chunks and a ragged tail
    (2, 130, 16, 64, 800, 256),     # largest single-wavefront shape
    (3, 70, 16, 64, 800, 320),      # d_state > 256: multi-wavefront scan
    (2, 40, 32, 64, 800, 64),       # K > 16: multi-wavefront scan
    (4, 1, 8, 64, 512, 64),         # one position per block
    (70, 3, 4, 64, 600, 32),        # many sequences, the smallest K
]


def _plant(sel, L, rng):
    """Verifier rows equal to ``sel`` except at one chosen position per row
    (or none), which covers chunk edges, the tail and full acceptance."""
    ver = sel.copy()
    picks = [0, 1, 62, 63, 64, 65, 127, 128, L // 2, L - 1, -1]
    for b in range(sel.shape[0]):
        pos = picks[(b + rng.integers(0, len(picks))) % len(picks)]
        if 0 <= pos < L:
            ver[b, pos] = (ver[b, pos] + 1 + rng.integers(0, 5)) % 100000
    return ver


def _to(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


@pytest.mark.parametrize("B,L,K,d,V,r", CASES)
def test_rerank_verify_matches_rerank_then_verify(B, L, K, d, V, r):
    print(f"[rerank_verify] B={B} L={L} K={K} d={d} V={V} d_state={r}", flush=True)
    wl = synth.Workload("rv", B=B, L=L, d=d, V=V, K=K, r=r, sigma=0.3, flat_frac=0.3, seed=7 * B + L + K)
    blk = synth.make_block(wl, "cpu", psi_std=0.1)
    io = oracle_inputs(blk)
    cl, ci = oracle.propose_block(io["H_bits"], io["W_bits"], K)
    free = oracle.rerank(io["psi"], io["alpha"], io["b_g"], io["H"], io["h_c"], io["x0"], io["W_bits"],
                         io["E_bits"], cl, ci, B, L)
    rng = np.random.default_rng(B * 1000 + L)
    ver = _plant(free["selected"].astype(np.int32), L, rng)

    dev = {k: blk.__dict__[k].to(DEV) for k in ("H", "W", "E", "h_c", "x0")}
    corr = brisk.Corrector({k: v.to(DEV) for k, v in blk.psi.items()}, blk.alpha, blk.b_g)
    gcl, gci = brisk.propose_block(dev["H"], dev["W"], K)
    args = (corr, dev["H"], dev["h_c"], dev["x0"], dev["W"], dev["E"], gcl, gci)
    sep = brisk.rerank(*args, B, L, want_scores=True)
    acc_s, cor_s = brisk.verify_accept(sep["selected"], _to(ver))
    fused = brisk.rerank_verify(*args, _to(ver), B, L, want_scores=True)
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in fused.items()}
    s = {k: v.cpu().numpy() for k, v in sep.items()}
    for k in ("selected", "refined", "gamma", "resid"):
        assert np.array_equal(g[k], s[k]), k
    assert np.array_equal(g["accept_len"], acc_s.cpu().numpy())
    assert np.array_equal(g["correction"], cor_s.cpu().numpy())

    # the oracle: the corrector on the GPU's candidates and prefix, then verification
    g["cand_logit"], g["cand_id"] = gcl.cpu().numpy(), gci.cpu().numpy()
    orc = oracle.rerank(io["psi"], io["alpha"], io["b_g"], io["H"], io["h_c"], io["x0"], io["W_bits"],
                        io["E_bits"], g["cand_logit"], g["cand_id"], B, L, prefix=g["selected"])
    check_rerank(g, orc)
    rerank_pick_ok(g["selected"], orc, g["cand_id"])
    oa, oc = oracle.verify_accept(g["selected"], ver)
    assert np.array_equal(oa, g["accept_len"]) and np.array_equal(oc, g["correction"])
    # where the oracle's own choice is clear of ties everywhere, the planted
    # positions are the accept lengths
    if free["margin"].min() > SCORE_TOL and np.array_equal(g["cand_id"], ci):
        want, _ = oracle.verify_accept(free["selected"], ver)
        assert np.array_equal(want, g["accept_len"])
    n_changed = int((g["selected"].ravel() != g["cand_id"][:, 0]).sum())
    print(f"  ok: accept lengths {sorted(set(g['accept_len'].tolist()))}, max |resid| "
          f"{np.abs(orc['resid']).max():.3g}, picks other than the top proposal {n_changed}", flush=True)


def test_rerank_verify_without_correction_output():
    B, L, K, d, V, r = 3, 90, 8, 64, 600, 64
    wl = synth.Workload("rv", B=B, L=L, d=d, V=V, K=K, r=r, sigma=0.3, flat_frac=0.3, seed=5)
    blk = synth.make_block(wl, DEV, psi_std=0.1)
    corr = brisk.Corrector(blk.psi, blk.alpha, blk.b_g)
    gcl, gci = brisk.propose_block(blk.H, blk.W, K)
    args = (corr, blk.H, blk.h_c, blk.x0, blk.W, blk.E, gcl, gci)
    sep = brisk.rerank(*args, B, L)
    acc_s, _ = brisk.verify_accept(sep["selected"], blk.verifier)
    acc = torch.full((B,), -7, dtype=torch.int32, device=DEV)
    sel = torch.empty(B, L, dtype=torch.int32, device=DEV)
    nws = brisk.rerank_workspace_size(corr, B, L, K)
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=DEV)
    st = brisk.lib().brisk_rerank_verify(
        ctypes.byref(corr.c_struct),
        blk.H.data_ptr(), blk.h_c.data_ptr(), blk.x0.data_ptr(), blk.W.data_ptr(), blk.E.data_ptr(),
        gcl.data_ptr(), gci.data_ptr(), blk.verifier.data_ptr(), B, L, K, d, V,
        sel.data_ptr(), None, None, None, acc.data_ptr(), None, ws.data_ptr(), nws,
        torch.cuda.current_stream().cuda_stream)
    assert st == 0
    torch.cuda.synchronize()
    assert torch.equal(acc, acc_s)
    assert torch.equal(sel, sep["selected"])
