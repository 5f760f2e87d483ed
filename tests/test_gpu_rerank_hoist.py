"""GPU: the rerank split at the candidates.

``rerank_hoist`` (the work that reads no candidate: projections of the hidden
states, the context and the anchors, their lifts) followed by
``rerank_finish`` must return bit for bit what ``rerank`` / ``rerank_verify``
return, with and without the per-token tables, on the single-wavefront and
the multi-wavefront scans.  The split workspace starts filled with NaN bytes,
so a finishing read of anything the hoist did not write shows up.  The last
tests run the hoist on a second stream while the LM-head pass that makes the
candidates streams (the order a decoding step uses), eagerly and captured in
a graph.
"""
import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

brisk = pytest.importorskip("paper_2609_33390_amd")
DEV = "cuda"

CASES = [  # B, L, K, d, V, r (= d_state), tables
    (1, 8, 4, 64, 512, 32, False),
    (3, 7, 5, 72, 1003, 32, False),     # ragged d and V
    (3, 7, 5, 72, 1003, 32, True),
    (5, 200, 8, 64, 900, 128, True),    # long blocks
    (2, 40, 32, 64, 800, 64, False),    # K > 16: multi-wavefront scan, then the verify kernel
    (3, 70, 16, 64, 800, 320, True),    # d_state > 256: multi-wavefront scan
    (70, 3, 4, 64, 600, 32, True),      # many sequences, the smallest K
]
KEYS = ("selected", "refined", "gamma", "resid")


def _nan_ws(corr, B, L, K):
    n = brisk.rerank_workspace_size(corr, B, L, K)
    return torch.full((max(n, 1),), 0xFF, dtype=torch.uint8, device=DEV)


def _same(a, b, keys):
    for k in keys:
        x, y = a[k].cpu().numpy(), b[k].cpu().numpy()
        assert np.array_equal(x.view(np.uint32) if x.dtype == np.float32 else x,
                              y.view(np.uint32) if y.dtype == np.float32 else y), k


@pytest.mark.parametrize("verify", [False, True])
@pytest.mark.parametrize("B,L,K,d,V,r,tables", CASES)
def test_split_rerank_matches_single_call(B, L, K, d, V, r, tables, verify):
    print(f"[rerank split] B={B} L={L} K={K} d={d} V={V} d_state={r} tables={tables} verify={verify}", flush=True)
    wl = synth.Workload("rh", B=B, L=L, d=d, V=V, K=K, r=r, sigma=0.3, flat_frac=0.3, seed=3 * B + L + K)
    blk = synth.make_block(wl, DEV, psi_std=0.1)
    corr = brisk.Corrector(blk.psi, blk.alpha, blk.b_g)
    if tables:
        corr.prepare(blk.W, blk.E)
    cl, ci = brisk.propose_block(blk.H, blk.W, K)
    args = (corr, blk.H, blk.h_c, blk.x0, blk.W, blk.E, cl, ci)
    if verify:
        one = brisk.rerank_verify(*args, blk.verifier, B, L, want_scores=True, workspace=_nan_ws(corr, B, L, K))
    else:
        one = brisk.rerank(*args, B, L, want_scores=True, workspace=_nan_ws(corr, B, L, K))
    ws = _nan_ws(corr, B, L, K)
    brisk.rerank_hoist(corr, blk.H, blk.h_c, blk.x0, blk.E, B, L, K, ws)
    two = brisk.rerank_finish(*args, B, L, ws, verifier=blk.verifier if verify else None, want_scores=True)
    torch.cuda.synchronize()
    _same(one, two, KEYS + (("accept_len", "correction") if verify else ()))
    assert np.isfinite(two["refined"].cpu().numpy()).all()


def _c1(tables=True):
    wl = synth.WORKLOADS["llada8b-b1-l32"]
    blk = synth.make_block(wl, DEV)
    corr = brisk.Corrector(blk.psi, blk.alpha, blk.b_g)
    if tables:
        corr.prepare(blk.W, blk.E)
    return wl, blk, corr


class _Step:
    """One decoding step with the hoist on a second stream beside the
    LM-head pass: fork, hoist | LM-head pass + merge, join, finish."""

    def __init__(self, wl, blk, corr):
        rows, K = wl.B * wl.L, wl.K
        self.wl, self.blk, self.corr = wl, blk, corr
        self.ws_p = torch.empty(brisk.propose_workspace_size(rows, wl.d, wl.V, K), dtype=torch.uint8, device=DEV)
        self.ws_r = _nan_ws(corr, wl.B, wl.L, K)
        self.cl = torch.empty(rows, K, dtype=torch.float32, device=DEV)
        self.ci = torch.empty(rows, K, dtype=torch.int32, device=DEV)
        self.out = {"selected": torch.empty(wl.B, wl.L, dtype=torch.int32, device=DEV),
                    "refined": torch.empty(rows, K, dtype=torch.float32, device=DEV),
                    "gamma": torch.empty(rows, dtype=torch.float32, device=DEV),
                    "resid": torch.empty(rows, K, dtype=torch.float32, device=DEV),
                    "accept_len": torch.empty(wl.B, dtype=torch.int32, device=DEV),
                    "correction": torch.empty(wl.B, dtype=torch.int32, device=DEV)}
        self.side = torch.cuda.Stream()

    def __call__(self):
        wl, b, c, o = self.wl, self.blk, self.corr, self.out
        main = torch.cuda.current_stream()
        self.side.wait_stream(main)
        brisk.rerank_hoist(c, b.H, b.h_c, b.x0, b.E, wl.B, wl.L, wl.K, self.ws_r, stream=self.side)
        brisk.propose_lmhead(b.H, b.W, wl.K, self.ws_p, stream=main)
        brisk.propose_merge(wl.B * wl.L, wl.V, wl.K, self.ws_p, self.cl, self.ci, stream=main)
        main.wait_stream(self.side)
        brisk.rerank_finish(c, b.H, b.h_c, b.x0, b.W, b.E, self.cl, self.ci, wl.B, wl.L, self.ws_r,
                            verifier=b.verifier, stream=main, **o)


def _reference(wl, blk, corr):
    cl, ci = brisk.propose_block(blk.H, blk.W, wl.K)
    ref = brisk.rerank_verify(corr, blk.H, blk.h_c, blk.x0, blk.W, blk.E, cl, ci, blk.verifier, wl.B, wl.L,
                              want_scores=True)
    ref["cand_logit"], ref["cand_id"] = cl, ci
    return ref


@pytest.mark.parametrize("tables", [True, False])
def test_hoist_beside_the_lmhead_pass(tables):
    print(f"[rerank split] two streams, llada8b-b1-l32, tables={tables}", flush=True)
    wl, blk, corr = _c1(tables)
    ref = _reference(wl, blk, corr)
    step = _Step(wl, blk, corr)
    for _ in range(3):
        step()
        torch.cuda.synchronize()
        _same(ref, step.out, KEYS + ("accept_len", "correction"))
        _same(ref, {"cand_logit": step.cl, "cand_id": step.ci}, ("cand_logit", "cand_id"))


def test_two_stream_step_in_a_graph():
    print("[rerank split] two streams captured in a graph, llada8b-b1-l32", flush=True)
    wl, blk, corr = _c1(True)
    ref = _reference(wl, blk, corr)
    step = _Step(wl, blk, corr)
    step()                                    # warm up outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        with torch.cuda.graph(g, stream=cap):
            step()
    torch.cuda.synchronize()
    for rep in range(4):
        for t in step.out.values():           # eager work between replays
            t.fill_(-1)
        step.cl.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        _same(ref, step.out, KEYS + ("accept_len", "correction"))
        _same(ref, {"cand_logit": step.cl, "cand_id": step.ci}, ("cand_logit", "cand_id"))
        print(f"  replay {rep} ok", flush=True)
