"""The binding refuses caller buffers of the wrong shape, dtype or device.

Every call below fails its checks before any pointer reaches the library, so
nothing is launched; the tensors live on the GPU so that only the shape,
dtype or size check can be what refuses them.
"""
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

brisk = pytest.importorskip("paper_2609_33390_amd")


@pytest.fixture(scope="module")
def tiny():
    blk = synth.make_block("tiny-d64-v512", "cuda")
    wl = blk.wl
    corr = brisk.Corrector(blk.psi, blk.alpha, blk.b_g)
    cl, ci = brisk.propose_block(blk.H, blk.W, wl.K)
    torch.cuda.synchronize()
    return blk, corr, cl, ci


def _i32(*s):
    return torch.zeros(*s, dtype=torch.int32, device="cuda")


def _f32(*s):
    return torch.zeros(*s, dtype=torch.float32, device="cuda")


def test_rerank_output_buffers(tiny):
    blk, corr, cl, ci = tiny
    B, L, K = blk.wl.B, blk.wl.L, blk.wl.K
    args = (corr, blk.H, blk.h_c, blk.x0, blk.W, blk.E, cl, ci, B, L)
    for kw in (dict(selected=_i32(B, L + 1)), dict(refined=_f32(B * L, K - 1)), dict(gamma=_f32(B * L + 1)),
               dict(resid=_f32(B * L * K)), dict(workspace=torch.zeros(16, dtype=torch.uint8, device="cuda"))):
        with pytest.raises(ValueError):
            brisk.rerank(*args, **kw)
    with pytest.raises(TypeError):
        brisk.rerank(*args, selected=torch.zeros(B, L, dtype=torch.int64, device="cuda"))
    with pytest.raises(ValueError):
        brisk.rerank(*args, workspace=torch.zeros(1 << 24, dtype=torch.uint8))       # host memory
    with pytest.raises(ValueError):
        brisk.rerank_verify(*args[:8], blk.verifier, B, L, accept_len=_i32(B + 1))
    with pytest.raises(ValueError):
        brisk.rerank_verify(*args[:8], blk.verifier[:, :-1].contiguous(), B, L)


def test_rerank_inputs_against_the_corrector(tiny):
    blk, corr, cl, ci = tiny
    B, L = blk.wl.B, blk.wl.L
    with pytest.raises(ValueError, match="corrector was built"):
        brisk.rerank(corr, blk.H[:, :56].contiguous(), blk.h_c, blk.x0, blk.W, blk.E, cl, ci, B, L)
    with pytest.raises(ValueError):
        brisk.rerank(corr, blk.H, blk.h_c, blk.x0, blk.W, blk.E[:-1].contiguous(), cl, ci, B, L)
    with pytest.raises(ValueError):
        brisk.rerank(corr, blk.H, blk.h_c, blk.x0, blk.W, blk.E, cl[:, :-1].contiguous(), ci, B, L)


def test_other_entry_points(tiny):
    blk, corr, cl, ci = tiny
    B, L, K = blk.wl.B, blk.wl.L, blk.wl.K
    sel = _i32(B, L)
    with pytest.raises(ValueError):
        brisk.verify_accept(sel, _i32(B, L), accept_len=_i32(B + 2))
    with pytest.raises(ValueError):
        brisk.verify_accept(sel, _i32(B, L + 1))
    with pytest.raises(ValueError):
        brisk.propose_block(blk.H, blk.W, K, cand_logit=_f32(B * L, K + 1))
    with pytest.raises(ValueError):
        brisk.propose_verify(blk.H, blk.W, 4, K, ver_token=_i32(3))
    with pytest.raises(ValueError):
        brisk.propose_lmhead(blk.H, blk.W, K, torch.zeros(8, dtype=torch.uint8, device="cuda"))
    with pytest.raises(ValueError):
        brisk.corrector_loss(blk.H, blk.W, ci, cl, _f32(B * L, K), _i32(B + 1), B, L)
    with pytest.raises(ValueError):
        brisk.spec_verify(blk.H, blk.W, sel, ci, _f32(B * L, K), _f32(B * L - 1), 7, 1.0)
