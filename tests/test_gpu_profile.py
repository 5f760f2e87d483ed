"""GPU parity of the acceptance-profile statistics (brisk_accept_profile)
against the CPU oracle on the same accepted-prefix lengths."""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

brisk = pytest.importorskip("paper_2609_33390_amd")


def _lengths(n, M, a, seed):
    """Accepted-prefix lengths of n blocks drawn from the profile a (first
    rejection at position i with probability 1 - a_i)."""
    rng = np.random.default_rng(seed)
    u = rng.random((n, M))
    rejected = u >= np.asarray(a)[None, :]
    first = np.where(rejected.any(axis=1), rejected.argmax(axis=1), M)
    return first.astype(np.int32)


def _compare(lens, M, eps):
    g = brisk.accept_profile(torch.from_numpy(lens).cuda(), M, eps=eps)
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in g.items()}
    o = oracle.profile_summary(lens, M, eps)
    np.testing.assert_allclose(g["a"], o["a"], rtol=0, atol=1e-15)
    np.testing.assert_allclose(g["w_raw"], o["raw"], rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(g["w"], o["w"], rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(g["tpf_fpt"], [o["tpf"], o["fpt"]], rtol=1e-13)
    return g


@pytest.mark.parametrize("n,M,seed", [(1, 7, 0), (1000, 7, 1), (100_000, 31, 2), (4097, 15, 3),
                                      (20_000, 1024, 4)])
def test_profile_matches_oracle(n, M, seed):
    rng = np.random.default_rng(seed)
    a = rng.uniform(0.6, 1.0, M)
    _compare(_lengths(n, M, a, seed), M, 1e-12)


def test_profile_of_the_decoding_path():
    # accepted lengths produced by the path itself on a small block batch
    import synth
    wl = synth.Workload("prof", B=64, L=16, d=64, V=512, K=4, r=32, sigma=0.3, flat_frac=0.5, seed=5)
    blk = synth.make_block(wl, "cuda")
    cl, ci = brisk.propose_block(blk.H, blk.W, wl.K)
    corr = brisk.Corrector(blk.psi, blk.alpha, blk.b_g)
    rr = brisk.rerank(corr, blk.H, blk.h_c, blk.x0, blk.W, blk.E, cl, ci, wl.B, wl.L)
    acc, _ = brisk.verify_accept(rr["selected"], blk.verifier)
    torch.cuda.synchronize()
    _compare(acc.cpu().numpy(), wl.L, 1e-12)


def test_profile_edge_cases():
    M = 8
    # no blocks: every position unreached, a = 1, TPF = M + 1, weights 0
    g = _compare(np.zeros(0, np.int32), M, 1e-12)
    assert np.all(g["a"] == 1.0) and g["tpf_fpt"][0] == M + 1 and np.all(g["w"] == 0.0)
    # every block rejected at position 1: a_1 = 0, TPF = 1
    g = _compare(np.zeros(50, np.int32), M, 1e-12)
    assert g["a"][0] == 0.0 and g["tpf_fpt"][0] == 1.0
    # out-of-range lengths are clamped into [0, M]
    lens = np.array([-5, 0, 3, 8, 9, 1000, 2], np.int32)
    g = brisk.accept_profile(torch.from_numpy(lens).cuda(), M, eps=1e-12)
    ref = brisk.accept_profile(torch.from_numpy(np.clip(lens, 0, M)).cuda(), M, eps=1e-12)
    torch.cuda.synchronize()
    for k in g:
        assert torch.equal(g[k], ref[k])
    # a single position
    _compare(np.array([0, 1, 1, 0, 1], np.int32), 1, 0.0)


def test_profile_deterministic_repeat():
    lens = _lengths(200_000, 31, np.full(31, 0.9), 7)
    t = torch.from_numpy(lens).cuda()
    g1 = brisk.accept_profile(t, 31)
    g2 = brisk.accept_profile(t, 31)
    torch.cuda.synchronize()
    for k in g1:
        assert torch.equal(g1[k], g2[k])
