"""The propose call that allocates nothing against brisk_propose_block.

brisk_propose_block_noalloc keeps its key lists in the library's fixed
per-device scratch instead of a caller's workspace; its candidates must equal
those of brisk_propose_block bit for bit (same kernels, same order of work).
Two calls in a row, the second with a smaller input, check that nothing the
first call left in the shared scratch leaks into the second.
"""
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

brisk = pytest.importorskip("paper_2609_33390_amd")


def _block(rows, d, V, seed):
    wl = synth.Workload(f"noalloc-{rows}x{d}x{V}", B=1, L=rows, d=d, V=V, K=8, r=32,
                        sigma=0.3, flat_frac=0.5, seed=seed)
    return synth.make_block(wl, "cuda")


@pytest.mark.parametrize("first,second", [
    # large-row tile (two row tiles, ragged V), then the small-batch tile
    ((300, 1024, 70001, 8), (20, 512, 20000, 4)),
    # 16-key lists on the mid tile, then a single row with 8 keys
    ((64, 768, 40000, 16), (1, 256, 5003, 8)),
])
def test_noalloc_matches_workspace_call(first, second):
    for rows, d, V, K in (first, second):
        print(f"noalloc case rows={rows} d={d} V={V} K={K}", flush=True)
        blk = _block(rows, d, V, seed=rows + d)
        cl_ref, ci_ref = brisk.propose_block(blk.H, blk.W, K)
        cl = torch.full((rows, K), float("nan"), dtype=torch.float32, device="cuda")
        ci = torch.full((rows, K), -7, dtype=torch.int32, device="cuda")
        brisk.propose_block_noalloc(blk.H, blk.W, K, cl, ci)
        torch.cuda.synchronize()
        assert torch.equal(ci, ci_ref)
        assert torch.equal(cl.view(torch.int32), cl_ref.view(torch.int32))


def test_noalloc_refuses_a_shape_beyond_its_scratch():
    """64 rows with 64-key lists need 32 MiB of key lists: refused, outputs untouched."""
    H = torch.zeros(64, 256, dtype=torch.bfloat16, device="cuda")
    W = torch.zeros(40000, 256, dtype=torch.bfloat16, device="cuda")
    cl = torch.full((64, 64), 3.0, dtype=torch.float32, device="cuda")
    ci = torch.full((64, 64), 5, dtype=torch.int32, device="cuda")
    with pytest.raises(brisk.BriskError) as e:
        brisk.propose_block_noalloc(H, W, 64, cl, ci)
    assert e.value.status == -6
    torch.cuda.synchronize()
    assert bool((cl == 3.0).all()) and bool((ci == 5).all())
