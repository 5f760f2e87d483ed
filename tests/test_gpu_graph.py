"""GPU checks of the launch structure: the LM-head pass and the merge called
separately equal brisk_propose_block, and a hipGraph capture of the whole step
(propose, rerank, verify; the last two also as the single rerank_verify call,
with and without the corrector's per-token tables) reproduces the eager
results on every replay."""
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

brisk = pytest.importorskip("paper_2609_33390_amd")


@pytest.mark.parametrize("name", ["tiny-d64-v512", "llada8b-b1-l32", "llada8b-b64-l32"])
def test_split_launches_equal_the_composed_call(name):
    wl = synth.WORKLOADS[name]
    blk = synth.make_block(wl, "cuda")
    rows = wl.rows
    cl, ci = brisk.propose_block(blk.H, blk.W, wl.K)
    ws = torch.empty(brisk.propose_workspace_size(rows, wl.d, wl.V, wl.K), dtype=torch.uint8, device="cuda")
    cl2 = torch.empty_like(cl)
    ci2 = torch.empty_like(ci)
    brisk.propose_lmhead(blk.H, blk.W, wl.K, ws)
    brisk.propose_merge(rows, wl.V, wl.K, ws, cl2, ci2)
    torch.cuda.synchronize()
    assert torch.equal(cl, cl2) and torch.equal(ci, ci2)


@pytest.mark.parametrize("name,fused,tables", [
    ("tiny-d64-v512", False, False), ("tiny-d64-v512", True, False),
    ("llada8b-b1-l32", False, False), ("llada8b-b1-l32", True, False),
    # with the corrector's per-token tables: the step blocks filled from them,
    # and (64 sequences) the scan gathering the table rows itself
    ("tiny-d64-v512", True, True), ("llada8b-b1-l32", True, True), ("llada8b-b64-l32", True, True)])
def test_graph_replay_matches_eager(name, fused, tables):
    wl = synth.WORKLOADS[name]
    blk = synth.make_block(wl, "cuda")
    corr = brisk.Corrector(blk.psi, blk.alpha, blk.b_g)
    if tables:
        corr.prepare(blk.W, blk.E)
    rows, K = wl.rows, wl.K
    dev = torch.device("cuda")
    cl = torch.empty(rows, K, dtype=torch.float32, device=dev)
    ci = torch.empty(rows, K, dtype=torch.int32, device=dev)
    sel = torch.empty(wl.B, wl.L, dtype=torch.int32, device=dev)
    acc = torch.empty(wl.B, dtype=torch.int32, device=dev)
    cor = torch.empty(wl.B, dtype=torch.int32, device=dev)
    ws_p = torch.empty(brisk.propose_workspace_size(rows, wl.d, wl.V, K), dtype=torch.uint8, device=dev)
    ws_r = torch.empty(brisk.rerank_workspace_size(corr, wl.B, wl.L, K), dtype=torch.uint8, device=dev)

    def step():
        brisk.propose_lmhead(blk.H, blk.W, K, ws_p)
        brisk.propose_merge(rows, wl.V, K, ws_p, cl, ci)
        if fused:
            brisk.rerank_verify(corr, blk.H, blk.h_c, blk.x0, blk.W, blk.E, cl, ci, blk.verifier, wl.B, wl.L,
                                selected=sel, accept_len=acc, correction=cor, workspace=ws_r)
            return
        brisk.rerank(corr, blk.H, blk.h_c, blk.x0, blk.W, blk.E, cl, ci, wl.B, wl.L, selected=sel,
                     workspace=ws_r)
        brisk.verify_accept(sel, blk.verifier, accept_len=acc, correction=cor)

    step()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (cl, ci, sel, acc, cor)]
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            step()
    torch.cuda.synchronize()
    for rep in range(4):
        for t in (cl, ci, sel, acc, cor):
            t.fill_(-7)                      # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(ref, (cl, ci, sel, acc, cor)):
            assert torch.equal(a, b), rep
