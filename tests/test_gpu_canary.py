"""GPU checks that no entry point writes outside the buffers it is given:
every output, workspace and table is a view into a larger byte buffer whose
guard bands (4 KiB on each side, filled with 0xA5) must be unchanged after the
call.  Shapes include ragged tails and the large-row tile."""
import ctypes

import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu

brisk = pytest.importorskip("paper_2609_33390_amd")
DEV = "cuda"
GUARD = 4096
PATTERN = 0xA5


class Guarded:
    """A typed view of ``nbytes`` inside guard bands."""

    def __init__(self, shape, dtype):
        n = int(np.prod(shape)) if len(shape) else 1
        self.nbytes = n * torch.empty((), dtype=dtype).element_size()
        self.buf = torch.full((self.nbytes + 2 * GUARD,), PATTERN, dtype=torch.uint8, device=DEV)
        self.t = self.buf[GUARD:GUARD + self.nbytes].view(dtype).view(*shape)

    def intact(self):
        torch.cuda.synchronize()
        return bool((self.buf[:GUARD] == PATTERN).all()) and bool((self.buf[GUARD + self.nbytes:] == PATTERN).all())


def _ws(nbytes):
    return Guarded((max(int(nbytes), 1),), torch.uint8)


def _check(*gs):
    for g in gs:
        assert g.intact(), "a guard band was overwritten"


SHAPES = [  # name, B, L, d, V, K
    ("ragged", 3, 7, 72, 1003, 5),
    ("mid", 2, 30, 136, 2049, 8),
    ("large", 5, 60, 64, 3000, 8),     # 300 rows: the large-row tile
    ("k64", 2, 9, 64, 700, 64),
    ("unsplit", 70, 30, 72, 700, 8),  # 16800 candidates: projections with d unsplit, 128-wide tiles
]


def _block(B, L, d, V, K, seed):
    wl = synth.Workload("canary", B=B, L=L, d=d, V=V, K=K, r=32, sigma=0.3, flat_frac=0.5, seed=seed)
    return wl, synth.make_block(wl, DEV)


@pytest.mark.parametrize("name,B,L,d,V,K", SHAPES)
def test_step_entry_points_stay_in_bounds(name, B, L, d, V, K):
    wl, blk = _block(B, L, d, V, K, 11)
    rows = B * L
    cl, ci = Guarded((rows, K), torch.float32), Guarded((rows, K), torch.int32)
    wsp = _ws(brisk.propose_workspace_size(rows, d, V, K))
    brisk.propose_block(blk.H, blk.W, K, cand_logit=cl.t, cand_id=ci.t, workspace=wsp.t)
    _check(cl, ci, wsp)

    corr = brisk.Corrector(blk.psi, blk.alpha, blk.b_g)
    sel = Guarded((B, L), torch.int32)
    ref, res = Guarded((rows, K), torch.float32), Guarded((rows, K), torch.float32)
    gam = Guarded((rows,), torch.float32)
    wsr = _ws(brisk.rerank_workspace_size(corr, B, L, K))
    brisk.rerank(corr, blk.H, blk.h_c, blk.x0, blk.W, blk.E, cl.t, ci.t, B, L, selected=sel.t,
                 refined=ref.t, gamma=gam.t, resid=res.t, workspace=wsr.t)
    _check(sel, ref, res, gam, wsr)

    acc, cor = Guarded((B,), torch.int32), Guarded((B,), torch.int32)
    brisk.verify_accept(sel.t, blk.verifier, accept_len=acc.t, correction=cor.t)
    _check(acc, cor)

    sel2, gam2 = Guarded((B, L), torch.int32), Guarded((rows,), torch.float32)
    ref2, res2 = Guarded((rows, K), torch.float32), Guarded((rows, K), torch.float32)
    acc3, cor3, wsr2 = Guarded((B,), torch.int32), Guarded((B,), torch.int32), _ws(wsr.nbytes)
    brisk.rerank_verify(corr, blk.H, blk.h_c, blk.x0, blk.W, blk.E, cl.t, ci.t, blk.verifier, B, L,
                        selected=sel2.t, refined=ref2.t, gamma=gam2.t, resid=res2.t, accept_len=acc3.t,
                        correction=cor3.t, workspace=wsr2.t)
    _check(sel2, ref2, res2, gam2, acc3, cor3, wsr2)
    assert torch.equal(acc3.t, acc.t) and torch.equal(cor3.t, cor.t)

    L_ = brisk.lib()
    acc2, com, ncom = Guarded((B,), torch.int32), Guarded((B, L + 1), torch.int32), Guarded((B,), torch.int32)
    st = L_.brisk_verify_commit(sel.t.data_ptr(), blk.verifier.data_ptr(), B, L, acc2.t.data_ptr(),
                                com.t.data_ptr(), ncom.t.data_ptr(), None)
    assert st == 0
    _check(acc2, com, ncom)


@pytest.mark.parametrize("name,B,L,d,V,K", SHAPES)
def test_tables_split_and_noalloc_entry_points_stay_in_bounds(name, B, L, d, V, K):
    """The no-alloc propose, the per-token tables (brisk_corrector_prepare),
    the rerank that reads them (on the 70-sequence shape the scan gathers the
    table rows itself; with 64 keys the multi-wave scan runs) and the rerank
    split at the candidates, each into guarded buffers."""
    print(f"[canary] tables, split and no-alloc entries: {name} B={B} L={L} d={d} V={V} K={K}", flush=True)
    wl, blk = _block(B, L, d, V, K, 13)
    rows = B * L
    L_ = brisk.lib()
    cl, ci = Guarded((rows, K), torch.float32), Guarded((rows, K), torch.int32)
    brisk.propose_block_noalloc(blk.H, blk.W, K, cl.t, ci.t)
    _check(cl, ci)

    corr = brisk.Corrector(blk.psi, blk.alpha, blk.b_g)
    tb, wb = ctypes.c_size_t(0), ctypes.c_size_t(0)
    assert L_.brisk_corrector_tables_size(ctypes.byref(corr.c_struct), V, ctypes.byref(tb), ctypes.byref(wb)) == 0
    tab, wst = Guarded((tb.value // 4,), torch.float32), _ws(wb.value)
    st = L_.brisk_corrector_prepare(ctypes.byref(corr.c_struct), blk.W.data_ptr(), blk.E.data_ptr(), V, d,
                                    tab.t.data_ptr(), tb.value, wst.t.data_ptr(), wst.nbytes, None)
    assert st == 0
    _check(tab, wst)
    corr.tables = tab.t
    corr.c_struct.tables = tab.t.data_ptr()
    corr.c_struct.tables_V = V

    def outs():
        return {"selected": Guarded((B, L), torch.int32), "refined": Guarded((rows, K), torch.float32),
                "gamma": Guarded((rows,), torch.float32), "resid": Guarded((rows, K), torch.float32),
                "accept_len": Guarded((B,), torch.int32), "correction": Guarded((B,), torch.int32)}

    one, ws1 = outs(), _ws(brisk.rerank_workspace_size(corr, B, L, K))
    brisk.rerank_verify(corr, blk.H, blk.h_c, blk.x0, blk.W, blk.E, cl.t, ci.t, blk.verifier, B, L,
                        workspace=ws1.t, **{k: g.t for k, g in one.items()})
    _check(ws1, *one.values())

    two, ws2 = outs(), _ws(ws1.nbytes)
    brisk.rerank_hoist(corr, blk.H, blk.h_c, blk.x0, blk.E, B, L, K, ws2.t)
    _check(ws2)
    brisk.rerank_finish(corr, blk.H, blk.h_c, blk.x0, blk.W, blk.E, cl.t, ci.t, B, L, ws2.t,
                        verifier=blk.verifier, **{k: g.t for k, g in two.items()})
    _check(ws2, *two.values())
    for k in one:
        assert torch.equal(one[k].t, two[k].t), k


@pytest.mark.parametrize("name,B,L,d,V,K", SHAPES)
def test_verifier_side_entry_points_stay_in_bounds(name, B, L, d, V, K):
    wl, blk = _block(B, L, d, V, K, 12)
    rows = B * L
    g = torch.Generator(device=DEV).manual_seed(4)
    Hv = (blk.H.float() + 0.3 * torch.randn(blk.H.shape, generator=g, device=DEV)).to(torch.bfloat16)
    both = torch.cat([blk.H, Hv], dim=0).contiguous()
    cl, ci = Guarded((rows, K), torch.float32), Guarded((rows, K), torch.int32)
    vt = Guarded((rows,), torch.int32)
    wsv = _ws(_pv_ws(rows, rows, d, V, K))
    brisk.propose_verify(both, blk.W, rows, K, cand_logit=cl.t, cand_id=ci.t, ver_token=vt.t, workspace=wsv.t)
    _check(cl, ci, vt, wsv)

    L_ = brisk.lib()
    # stochastic verification: proposals are the top candidates, a spread law
    prob = torch.softmax(cl.t, dim=1).contiguous()
    x = ci.t[:, 0].reshape(B, L).contiguous()
    u = torch.rand(rows, generator=g, device=DEV)
    nb = ctypes.c_size_t(0)
    assert L_.brisk_spec_verify_workspace_size(B, L, V, K, ctypes.byref(nb)) == 0
    wss = _ws(nb.value)
    sacc, scor = Guarded((B,), torch.int32), Guarded((B,), torch.int32)
    racc, rres = Guarded((rows,), torch.int32), Guarded((rows,), torch.int32)
    st = L_.brisk_spec_verify(Hv.data_ptr(), blk.W.data_ptr(), x.data_ptr(), ci.t.data_ptr(), prob.data_ptr(),
                              u.data_ptr(), 77, 1.5, B, L, K, d, V, sacc.t.data_ptr(), scor.t.data_ptr(),
                              racc.t.data_ptr(), rres.t.data_ptr(), wss.t.data_ptr(), wss.nbytes, None)
    assert st == 0
    _check(sacc, scor, racc, rres, wss)

    # corrector loss on the candidates, with the proposal logits as refined logits
    lp, ce, kl, lm = (Guarded((rows,), torch.float32), Guarded((rows,), torch.float32),
                      Guarded((rows,), torch.float32), Guarded((2,), torch.float32))
    accl = torch.randint(0, L + 1, (B,), generator=g, device=DEV, dtype=torch.int32)
    st = L_.brisk_corrector_loss(Hv.data_ptr(), blk.W.data_ptr(), ci.t.data_ptr(), cl.t.data_ptr(),
                                 cl.t.data_ptr(), accl.data_ptr(), B, L, K, d, V, 0.01, lp.t.data_ptr(),
                                 ce.t.data_ptr(), kl.t.data_ptr(), lm.t.data_ptr(), None)
    assert st == 0
    _check(lp, ce, kl, lm)


def _pv_ws(rows_prop, rows_ver, d, V, K):
    nb = ctypes.c_size_t(0)
    assert brisk.lib().brisk_propose_verify_workspace_size(rows_prop, rows_ver, d, V, K, ctypes.byref(nb)) == 0
    return nb.value


@pytest.mark.parametrize("n,M", [(1, 1), (1000, 7), (300_000, 63), (5000, 64), (20_000, 1024)])
def test_accept_profile_stays_in_bounds(n, M):
    L_ = brisk.lib()
    g = torch.Generator(device=DEV).manual_seed(n + M)
    lens = torch.randint(0, M + 1, (n,), generator=g, device=DEV, dtype=torch.int32)
    nb = ctypes.c_size_t(0)
    assert L_.brisk_accept_profile_workspace_size(n, M, ctypes.byref(nb)) == 0
    ws = _ws(nb.value)
    a, wr, w, tf = (Guarded((M,), torch.float64), Guarded((M,), torch.float64), Guarded((M,), torch.float64),
                    Guarded((2,), torch.float64))
    st = L_.brisk_accept_profile(lens.data_ptr(), n, M, 0.0, a.t.data_ptr(), wr.t.data_ptr(), w.t.data_ptr(),
                                 tf.t.data_ptr(), ws.t.data_ptr(), ws.nbytes, None)
    assert st == 0
    _check(a, wr, w, tf, ws)
