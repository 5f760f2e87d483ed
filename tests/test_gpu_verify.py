"""GPU parity of the fused proposal + verifier LM-head pass
(brisk_propose_verify) and of the commit (brisk_verify_commit) against the
CPU oracle on the same inputs."""
import numpy as np
import pytest
import torch

import oracle
import synth
from parity import SCORE_TOL, check_candidates, check_gpu_order

pytestmark = pytest.mark.gpu

brisk = pytest.importorskip("paper_2609_33390_amd")


def _say(*a):
    print(*a, flush=True)


def _verifier_rows(blk, sigma, seed):
    """Verifier hidden states of the block under verification: the proposal
    rows plus seeded Gaussian noise, rounded to bf16."""
    g = torch.Generator(device=blk.H.device).manual_seed(seed)
    n = torch.randn(blk.H.shape, generator=g, device=blk.H.device, dtype=torch.float32)
    return (blk.H.float() + sigma * n).to(torch.bfloat16)


def _check_argmax(ver_token, Hv_bits, W_bits, rows):
    logits = oracle.lm_logits(oracle.bf16_to_f64(Hv_bits[rows]), W_bits)
    top2 = np.sort(logits, axis=1)[:, -2:]
    ref = oracle.verifier_argmax(Hv_bits[rows], W_bits)
    sure = (top2[:, 1] - top2[:, 0]) > SCORE_TOL
    assert np.array_equal(ver_token[rows][sure], ref[sure])
    # near ties: the GPU token's logit is within the tolerance of the maximum
    got = logits[np.arange(len(rows)), ver_token[rows]]
    assert np.all(got >= top2[:, 1] - SCORE_TOL)
    return int((~sure).sum())


@pytest.mark.parametrize("wl_name,sample", [("tiny-d64-v512", None), ("llada8b-b1-l32", 16)])
def test_fused_pass_matches_separate_pass_and_oracle(wl_name, sample):
    wl = synth.WORKLOADS[wl_name]
    blk = synth.make_block(wl, "cuda")
    Hv = _verifier_rows(blk, 0.3, 7)
    hidden = torch.cat([blk.H, Hv], dim=0).contiguous()
    rows = wl.rows
    cl, ci, vt = brisk.propose_verify(hidden, blk.W, rows, wl.K)
    cl_s, ci_s = brisk.propose_block(blk.H, blk.W, wl.K)
    torch.cuda.synchronize()
    # the proposal rows are exactly what the separate proposal pass gives
    assert torch.equal(ci, ci_s) and torch.equal(cl, cl_s)
    W_bits = synth.bf16_bits(blk.W)
    Hv_bits = synth.bf16_bits(Hv)
    rs = np.arange(rows) if sample is None else np.linspace(0, rows - 1, sample).astype(int)
    _say(f"  [{wl_name}] oracle argmax on {len(rs)} verifier rows")
    near = _check_argmax(vt.cpu().numpy(), Hv_bits, W_bits, rs)
    H_bits = synth.bf16_bits(blk.H)
    ol = oracle.lm_logits(oracle.bf16_to_f64(H_bits[rs]), W_bits)
    check_candidates(cl.cpu().numpy()[rs], ci.cpu().numpy()[rs], ol)
    check_gpu_order(cl.cpu().numpy(), ci.cpu().numpy())
    _say(f"  [{wl_name}] near-tie verifier rows: {near}")


@pytest.mark.slow
@pytest.mark.parametrize("wl_name", ["llada8b-b64-l32", "llada8b-b256-l16"])
def test_fused_pass_batched_shape(wl_name):
    """The fused pass at the shapes the benchmark times: 2048 (4096) proposal
    rows and as many verifier rows in one launch, 16 (32) row tiles of the
    large-row tile.  Checked on the first and last row of every 256-row tile
    of both halves, plus random rows."""
    _say(f"[fused pass] {wl_name}")
    wl = synth.WORKLOADS[wl_name]
    blk = synth.make_block(wl, "cuda")
    Hv = _verifier_rows(blk, 0.3, 11)
    hidden = torch.cat([blk.H, Hv], dim=0).contiguous()
    rows = wl.rows
    cl, ci, vt = brisk.propose_verify(hidden, blk.W, rows, wl.K)
    cl_s, ci_s = brisk.propose_block(blk.H, blk.W, wl.K)
    torch.cuda.synchronize()
    assert torch.equal(ci, ci_s) and torch.equal(cl, cl_s)
    rng = np.random.default_rng(5)
    edges = sorted({t for t0 in range(0, rows, 256) for t in (t0, t0 + 255)})
    rs = np.array(sorted(set(edges) | set(rng.choice(rows, 32, replace=False).tolist())))
    W_bits, Hv_bits, H_bits = synth.bf16_bits(blk.W), synth.bf16_bits(Hv), synth.bf16_bits(blk.H)
    _say(f"  oracle on {len(rs)} proposal and {len(rs)} verifier rows")
    near = _check_argmax(vt.cpu().numpy(), Hv_bits, W_bits, rs)
    ol = oracle.lm_logits(oracle.bf16_to_f64(H_bits[rs]), W_bits)
    check_candidates(cl.cpu().numpy()[rs], ci.cpu().numpy()[rs], ol)
    _say(f"  near-tie verifier rows: {near}")


# (100, 300, 16): 400 rows on the large-row tile with 16-key lists, whose
# epilogue filters survivors
@pytest.mark.parametrize("rows_prop,rows_ver,K", [(0, 40, 5), (40, 0, 5), (1, 1, 5), (100, 300, 5),
                                                  (100, 300, 16)])
def test_fused_pass_ragged(rows_prop, rows_ver, K):
    wl = synth.Workload("rg", B=1, L=rows_prop + rows_ver, d=136, V=1000, K=K, r=32, sigma=0.3,
                        flat_frac=0.5, seed=rows_prop * 7 + rows_ver)
    blk = synth.make_block(wl, "cuda")
    cl, ci, vt = brisk.propose_verify(blk.H, blk.W, rows_prop, wl.K)
    torch.cuda.synchronize()
    H_bits, W_bits = synth.bf16_bits(blk.H), synth.bf16_bits(blk.W)
    if rows_prop:
        ol = oracle.lm_logits(oracle.bf16_to_f64(H_bits[:rows_prop]), W_bits)
        check_candidates(cl.cpu().numpy(), ci.cpu().numpy(), ol)
    if rows_ver:
        _check_argmax(vt.cpu().numpy(), H_bits[rows_prop:], W_bits, np.arange(rows_ver))


def test_fused_pass_duplicate_rows_tie_to_lower_id():
    wl = synth.Workload("dup", B=1, L=24, d=64, V=700, K=4, r=32, sigma=0.3, flat_frac=0.0, seed=9)
    blk = synth.make_block(wl, "cuda", dup_top=True)
    _, _, vt = brisk.propose_verify(blk.H, blk.W, 0, wl.K)
    torch.cuda.synchronize()
    ref = oracle.verifier_argmax(synth.bf16_bits(blk.H), synth.bf16_bits(blk.W))
    assert np.array_equal(vt.cpu().numpy(), ref)


@pytest.mark.parametrize("B,L", [(1, 8), (7, 32), (64, 32), (5, 200), (300, 3)])
def test_verify_commit_matches_oracle(B, L):
    rng = np.random.default_rng(B * 1000 + L)
    ver = rng.integers(0, 50, (B, L)).astype(np.int32)
    prop = ver.copy()
    # forced first mismatches: none, the first, the middle, the last position
    for b in range(B):
        kind = b % 4
        if kind == 1:
            prop[b, 0] += 1
        elif kind == 2:
            prop[b, L // 2] += 1
        elif kind == 3:
            prop[b, L - 1] += 1
            if L > 2:
                prop[b, L - 2] = rng.integers(0, 50)
    acc, com, n = brisk.verify_commit(torch.from_numpy(prop).cuda(), torch.from_numpy(ver).cuda())
    torch.cuda.synchronize()
    oa, oc, on = oracle.verify_commit(prop, ver)
    assert np.array_equal(acc.cpu().numpy(), oa)
    assert np.array_equal(com.cpu().numpy(), oc)
    assert np.array_equal(n.cpu().numpy(), on)
