"""Host-side checks of the C ABI that need no GPU.

The library must load and export every function ``include/brisk.h`` declares,
and every invalid call must be rejected by host validation before any HIP call.
Each call below is built to fail validation, so none of them launches work.
"""
import ctypes
import os
import re

import pytest

import paper_2609_33390_amd as brisk

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "brisk.h")

OK, ENULL, ESHAPE, EUNSUP, EWS = 0, -1, -2, -3, -4
FAKE = 0x10000          # an aligned non-null address that is never dereferenced
MISALIGNED = 0x10002


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(brisk_\w+)\s*\(", text)))


def test_header_declares_the_bound_symbols():
    assert _declared() == sorted(brisk.ABI_SYMBOLS)


def test_library_exports_every_declared_symbol():
    L = brisk.lib()
    for name in _declared():
        assert hasattr(L, name), name


def test_status_strings_and_version():
    L = brisk.lib()
    assert L.brisk_abi_version() == 10
    for st in (OK, ENULL, ESHAPE, EUNSUP, EWS, -5, -6):
        assert L.brisk_status_str(st).decode() != "unknown status"
        assert L.brisk_status_str(st).decode()
    assert L.brisk_status_str(123).decode() == "unknown status"


def _propose(**kw):
    a = dict(hidden=FAKE, lm_head=FAKE, rows=32, d=4096, V=126464, K=8, cl=FAKE, ci=FAKE,
             ws=FAKE, ws_bytes=0, stream=None)
    a.update(kw)
    return brisk.lib().brisk_propose_block(a["hidden"], a["lm_head"], a["rows"], a["d"], a["V"],
                                           a["K"], a["cl"], a["ci"], a["ws"], a["ws_bytes"], a["stream"])


@pytest.mark.parametrize("kw,want", [
    (dict(hidden=None), ENULL), (dict(lm_head=None), ENULL), (dict(cl=None), ENULL),
    (dict(ci=None), ENULL),
    (dict(rows=0), ESHAPE), (dict(rows=-3), ESHAPE), (dict(d=0), ESHAPE), (dict(K=0), ESHAPE),
    (dict(K=65), ESHAPE), (dict(V=4, K=8), ESHAPE), (dict(d=1 << 20), ESHAPE),
    (dict(d=4100), EUNSUP), (dict(hidden=MISALIGNED), EUNSUP), (dict(lm_head=MISALIGNED), EUNSUP),
    (dict(ws_bytes=0), EWS), (dict(ws=None, ws_bytes=1 << 40), EWS),
])
def test_propose_validation(kw, want):
    assert _propose(**kw) == want


@pytest.mark.parametrize("kw,want", [
    (dict(hidden=None), ENULL), (dict(lm_head=None), ENULL), (dict(rows=0), ESHAPE), (dict(K=65), ESHAPE),
    (dict(V=4, K=8), ESHAPE), (dict(d=4100), EUNSUP), (dict(hidden=MISALIGNED), EUNSUP),
    (dict(ws_bytes=0), EWS), (dict(ws=None, ws_bytes=1 << 40), EWS), (dict(ws=MISALIGNED), EUNSUP),
])
def test_propose_lmhead_validation(kw, want):
    a = dict(hidden=FAKE, lm_head=FAKE, rows=32, d=4096, V=126464, K=8, ws=FAKE, ws_bytes=1 << 30)
    a.update(kw)
    assert brisk.lib().brisk_propose_lmhead(a["hidden"], a["lm_head"], a["rows"], a["d"], a["V"], a["K"],
                                            a["ws"], a["ws_bytes"], None) == want


@pytest.mark.parametrize("kw,want", [
    (dict(cl=None), ENULL), (dict(ci=None), ENULL), (dict(rows=0), ESHAPE), (dict(K=0), ESHAPE),
    (dict(V=4, K=8), ESHAPE), (dict(ci=MISALIGNED), EUNSUP), (dict(ws_bytes=0), EWS),
    (dict(ws=MISALIGNED), EUNSUP),
])
def test_propose_merge_validation(kw, want):
    a = dict(rows=32, V=126464, K=8, cl=FAKE, ci=FAKE, ws=FAKE, ws_bytes=1 << 30)
    a.update(kw)
    assert brisk.lib().brisk_propose_merge(a["rows"], a["V"], a["K"], a["cl"], a["ci"], a["ws"],
                                           a["ws_bytes"], None) == want


def test_propose_workspace_size_query():
    n = brisk.propose_workspace_size(32, 4096, 126464, 8)
    assert n > 0
    assert _propose(ws_bytes=n - 1) == EWS
    with pytest.raises(brisk.BriskError):
        brisk.propose_workspace_size(0, 4096, 126464, 8)


def _corr(**kw):
    dims = dict(d_state=256, d_hproj=128, d_tproj=128, d_pos=32, d_feat=32, rank=128, max_L=32)
    ptrs = {n: FAKE for n in brisk.PSI_FIELDS}
    for k, v in kw.items():
        if k in dims:
            dims[k] = v
        else:
            ptrs[k] = v
    return brisk._CorrectorC(**dims, **ptrs, alpha=0.0, b_g=0.0)


def _rerank(c=None, **kw):
    a = dict(hidden=FAKE, ctx=FAKE, anchor=FAKE, W=FAKE, E=FAKE, cl=FAKE, ci=FAKE, B=1, L=32, K=8,
             d=4096, V=126464, sel=FAKE, ref=None, gam=None, res=None, ws=FAKE, ws_bytes=0)
    a.update(kw)
    c = _corr() if c is None else c
    return brisk.lib().brisk_rerank(ctypes.byref(c), a["hidden"], a["ctx"], a["anchor"], a["W"], a["E"],
                                    a["cl"], a["ci"], a["B"], a["L"], a["K"], a["d"], a["V"], a["sel"],
                                    a["ref"], a["gam"], a["res"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("ckw,kw,want", [
    (dict(W_c=None), {}, ENULL), (dict(A_h=None), {}, ENULL), ({}, dict(sel=None), ENULL),
    ({}, dict(anchor=None), ENULL),
    (dict(d_state=0), {}, ESHAPE), (dict(d_state=513), {}, ESHAPE), (dict(rank=300), {}, ESHAPE),
    ({}, dict(K=3), ESHAPE), ({}, dict(K=65), ESHAPE), ({}, dict(L=33), ESHAPE), ({}, dict(B=0), ESHAPE),
    ({}, dict(V=4), ESHAPE),
    ({}, dict(d=4092), EUNSUP), (dict(W_c=MISALIGNED), {}, EUNSUP), ({}, dict(E=MISALIGNED), EUNSUP),
    ({}, dict(ws_bytes=16), EWS),
])
def test_rerank_validation(ckw, kw, want):
    assert _rerank(_corr(**ckw), **kw) == want


def _rerank_verify(c=None, **kw):
    a = dict(hidden=FAKE, ctx=FAKE, anchor=FAKE, W=FAKE, E=FAKE, cl=FAKE, ci=FAKE, ver=FAKE, B=1, L=32, K=8,
             d=4096, V=126464, sel=FAKE, ref=None, gam=None, res=None, acc=FAKE, cor=None, ws=FAKE, ws_bytes=0)
    a.update(kw)
    c = _corr() if c is None else c
    return brisk.lib().brisk_rerank_verify(ctypes.byref(c), a["hidden"], a["ctx"], a["anchor"], a["W"], a["E"],
                                           a["cl"], a["ci"], a["ver"], a["B"], a["L"], a["K"], a["d"], a["V"],
                                           a["sel"], a["ref"], a["gam"], a["res"], a["acc"], a["cor"], a["ws"],
                                           a["ws_bytes"], None)


@pytest.mark.parametrize("ckw,kw,want", [
    ({}, dict(ver=None), ENULL), ({}, dict(acc=None), ENULL), ({}, dict(sel=None), ENULL),
    (dict(W_z=None), {}, ENULL),
    ({}, dict(ver=MISALIGNED), EUNSUP), ({}, dict(acc=MISALIGNED), EUNSUP), ({}, dict(cor=MISALIGNED), EUNSUP),
    ({}, dict(K=65), ESHAPE), ({}, dict(L=33), ESHAPE), (dict(d_state=513), {}, ESHAPE),
    ({}, dict(ws_bytes=16), EWS), ({}, dict(cor=FAKE, ws_bytes=16), EWS),
])
def test_rerank_verify_validation(ckw, kw, want):
    assert _rerank_verify(_corr(**ckw), **kw) == want


def _rerank_hoist(c=None, **kw):
    a = dict(hidden=FAKE, ctx=FAKE, anchor=FAKE, E=FAKE, B=1, L=32, K=8, d=4096, V=126464, ws=FAKE, ws_bytes=0)
    a.update(kw)
    c = _corr() if c is None else c
    return brisk.lib().brisk_rerank_hoist(ctypes.byref(c), a["hidden"], a["ctx"], a["anchor"], a["E"], a["B"],
                                          a["L"], a["K"], a["d"], a["V"], a["ws"], a["ws_bytes"], None)


@pytest.mark.parametrize("ckw,kw,want", [
    (dict(A_h=None), {}, ENULL), ({}, dict(hidden=None), ENULL), ({}, dict(ctx=None), ENULL),
    ({}, dict(anchor=None), ENULL), ({}, dict(E=None), ENULL),
    ({}, dict(K=3), ESHAPE), ({}, dict(L=33), ESHAPE), ({}, dict(B=0), ESHAPE), (dict(d_state=513), {}, ESHAPE),
    ({}, dict(d=4092), EUNSUP), ({}, dict(E=MISALIGNED), EUNSUP), ({}, dict(ws=MISALIGNED, ws_bytes=1 << 40), EUNSUP),
    ({}, dict(ws_bytes=16), EWS), ({}, dict(ws=None, ws_bytes=1 << 40), EWS),
])
def test_rerank_hoist_validation(ckw, kw, want):
    # the hoisted part reads no LM head or candidates: the call gets none
    assert _rerank_hoist(_corr(**ckw), **kw) == want


def _rerank_finish(c=None, **kw):
    a = dict(hidden=FAKE, ctx=FAKE, anchor=FAKE, W=FAKE, E=FAKE, cl=FAKE, ci=FAKE, ver=None, B=1, L=32, K=8,
             d=4096, V=126464, sel=FAKE, ref=None, gam=None, res=None, acc=None, cor=None, ws=FAKE, ws_bytes=0)
    a.update(kw)
    c = _corr() if c is None else c
    return brisk.lib().brisk_rerank_finish(ctypes.byref(c), a["hidden"], a["ctx"], a["anchor"], a["W"], a["E"],
                                           a["cl"], a["ci"], a["ver"], a["B"], a["L"], a["K"], a["d"], a["V"],
                                           a["sel"], a["ref"], a["gam"], a["res"], a["acc"], a["cor"], a["ws"],
                                           a["ws_bytes"], None)


@pytest.mark.parametrize("ckw,kw,want", [
    ({}, dict(W=None), ENULL), ({}, dict(cl=None), ENULL), ({}, dict(ci=None), ENULL), ({}, dict(sel=None), ENULL),
    ({}, dict(ver=FAKE), ENULL),                      # a verifier needs accept_len
    (dict(W_s=None), {}, ENULL),
    ({}, dict(ver=FAKE, acc=MISALIGNED), EUNSUP), ({}, dict(cor=MISALIGNED), EUNSUP),
    ({}, dict(K=65), ESHAPE), ({}, dict(L=33), ESHAPE),
    ({}, dict(ws_bytes=16), EWS), ({}, dict(ver=FAKE, acc=FAKE, ws_bytes=16), EWS),
])
def test_rerank_finish_validation(ckw, kw, want):
    assert _rerank_finish(_corr(**ckw), **kw) == want


def test_rerank_workspace_size_query():
    c = _corr()
    out = ctypes.c_size_t()
    assert brisk.lib().brisk_rerank_workspace_size(ctypes.byref(c), 64, 32, 8, ctypes.byref(out)) == OK
    assert out.value > 64 * 32 * 8 * 256 * 4
    assert brisk.lib().brisk_rerank_workspace_size(ctypes.byref(c), 64, 32, 2, ctypes.byref(out)) == ESHAPE


@pytest.mark.parametrize("args,want", [
    ((None, FAKE, 4, 8, FAKE, None), ENULL), ((FAKE, FAKE, 4, 8, None, None), ENULL),
    ((FAKE, FAKE, 0, 8, FAKE, None), ESHAPE), ((FAKE, FAKE, 4, 0, FAKE, None), ESHAPE),
    ((MISALIGNED, FAKE, 4, 8, FAKE, None), EUNSUP),
])
def test_verify_validation(args, want):
    assert brisk.lib().brisk_verify_accept(*args, None) == want


def test_python_binding_refuses_host_tensors():
    import torch
    h = torch.zeros(4, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="HIP device"):
        brisk.propose_block(h, h, 4)
    with pytest.raises(ValueError, match="HIP device"):
        brisk.verify_accept(torch.zeros(2, 3, dtype=torch.int32), torch.zeros(2, 3, dtype=torch.int32))


@pytest.mark.parametrize("args,want", [
    ((None, 4, 8, 0.0, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20), ENULL),
    ((FAKE, 4, 8, 0.0, None, FAKE, FAKE, FAKE, FAKE, 1 << 20), ENULL),
    ((FAKE, 4, 8, 0.0, FAKE, FAKE, FAKE, None, FAKE, 1 << 20), ENULL),
    ((FAKE, 4, 0, 0.0, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20), ESHAPE),
    ((FAKE, 4, 1025, 0.0, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20), ESHAPE),
    ((FAKE, -1, 8, 0.0, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20), ESHAPE),
    ((MISALIGNED, 4, 8, 0.0, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 20), EUNSUP),
    ((FAKE, 4, 8, 0.0, 0x10004, FAKE, FAKE, FAKE, FAKE, 1 << 20), EUNSUP),
    ((FAKE, 4, 8, 0.0, FAKE, FAKE, FAKE, FAKE, FAKE, 0), EWS),
    ((FAKE, 4, 8, 0.0, FAKE, FAKE, FAKE, FAKE, None, 1 << 20), EWS),
])
def test_accept_profile_validation(args, want):
    assert brisk.lib().brisk_accept_profile(*args, None) == want


def test_accept_profile_workspace_size_query():
    L = brisk.lib()
    n = ctypes.c_size_t(0)
    assert L.brisk_accept_profile_workspace_size(100000, 31, ctypes.byref(n)) == OK and n.value > 0
    assert L.brisk_accept_profile_workspace_size(0, 31, ctypes.byref(n)) == OK and n.value > 0
    assert L.brisk_accept_profile_workspace_size(10, 0, ctypes.byref(n)) == ESHAPE
    assert L.brisk_accept_profile_workspace_size(10, 8, None) == ENULL


@pytest.mark.parametrize("kw,want", [
    (dict(), OK), (dict(hidden=None), ENULL), (dict(ver=None), ENULL), (dict(cl=None), ENULL),
    (dict(rp=0, cl=None, ci=None), OK), (dict(rv=0, ver=None), OK), (dict(rp=0, rv=0), ESHAPE),
    (dict(rp=-1), ESHAPE), (dict(K=0), ESHAPE), (dict(d=4100), EUNSUP), (dict(ver=0x10002), EUNSUP),
    (dict(ws_bytes=0), EWS),
])
def test_propose_verify_validation(kw, want):
    a = dict(hidden=FAKE, W=FAKE, rp=32, rv=32, d=4096, V=126464, K=8, cl=FAKE, ci=FAKE, ver=FAKE,
             ws=FAKE, ws_bytes=1 << 30)
    a.update(kw)
    if want == OK:
        # valid arguments would launch: only check the size query agrees
        n = ctypes.c_size_t(0)
        assert brisk.lib().brisk_propose_verify_workspace_size(a["rp"], a["rv"], a["d"], a["V"], a["K"],
                                                               ctypes.byref(n)) == OK
        return
    st = brisk.lib().brisk_propose_verify(a["hidden"], a["W"], a["rp"], a["rv"], a["d"], a["V"], a["K"],
                                          a["cl"], a["ci"], a["ver"], a["ws"], a["ws_bytes"], None)
    assert st == want


@pytest.mark.parametrize("args,want", [
    ((None, FAKE, 4, 8, FAKE, FAKE, FAKE), ENULL), ((FAKE, FAKE, 4, 8, None, None, FAKE), ENULL),
    ((FAKE, FAKE, 4, 8, None, FAKE, None), ENULL), ((FAKE, FAKE, 0, 8, None, FAKE, FAKE), ESHAPE),
    ((FAKE, FAKE, 4, 0, None, FAKE, FAKE), ESHAPE), ((FAKE, MISALIGNED, 4, 8, None, FAKE, FAKE), EUNSUP),
])
def test_verify_commit_validation(args, want):
    assert brisk.lib().brisk_verify_commit(*args, None) == want


@pytest.mark.parametrize("kw,want", [
    (dict(hv=None), ENULL), (dict(acc=None), ENULL), (dict(lm=None), ENULL), (dict(B=0), ESHAPE),
    (dict(K=0), ESHAPE), (dict(K=65), ESHAPE), (dict(d=4100), EUNSUP), (dict(hv=MISALIGNED), EUNSUP),
    (dict(ce=MISALIGNED), EUNSUP),
])
def test_corrector_loss_validation(kw, want):
    a = dict(hv=FAKE, W=FAKE, ids=FAKE, cl=FAKE, ref=FAKE, acc=FAKE, B=2, L=8, K=8, d=4096, V=126464,
             beta=0.01, lp=FAKE, ce=None, kl=None, mean=FAKE, lm=FAKE)
    a.update(kw)
    st = brisk.lib().brisk_corrector_loss(a["hv"], a["lm"], a["ids"], a["cl"], a["ref"], a["acc"], a["B"],
                                          a["L"], a["K"], a["d"], a["V"], a["beta"], a["lp"], a["ce"],
                                          a["kl"], a["mean"], None)
    assert st == want


@pytest.mark.parametrize("kw,want", [
    (dict(prop=None), ENULL), (dict(u=None), ENULL), (dict(acc=None), ENULL), (dict(hv=None), ENULL),
    (dict(K=0), ESHAPE), (dict(K=65), ESHAPE), (dict(T=0.0), ESHAPE), (dict(T=float("nan")), ESHAPE),
    (dict(V=8, K=8), ESHAPE), (dict(d=4100), EUNSUP), (dict(cpr=MISALIGNED), EUNSUP),
    (dict(ws_bytes=0), EWS),
])
def test_spec_verify_validation(kw, want):
    a = dict(hv=FAKE, W=FAKE, prop=FAKE, cid=FAKE, cpr=FAKE, u=FAKE, seed=1, T=1.0, B=2, L=8, K=8,
             d=4096, V=126464, acc=FAKE, cor=None, ra=None, rr=None, ws=FAKE, ws_bytes=1 << 20)
    a.update(kw)
    st = brisk.lib().brisk_spec_verify(a["hv"], a["W"], a["prop"], a["cid"], a["cpr"], a["u"], a["seed"],
                                       a["T"], a["B"], a["L"], a["K"], a["d"], a["V"], a["acc"], a["cor"],
                                       a["ra"], a["rr"], a["ws"], a["ws_bytes"], None)
    assert st == want


@pytest.mark.parametrize("K,L,want", [(16, 41943, EWS), (16, 41944, EUNSUP)])
def test_rerank_scan_offset_limit_uses_padded_vectors(K, L, want):
    """With d_state = 32 each step vector is still padded to 256 floats, so one
    sequence's step blocks take L*(2+3K)*256*4 bytes: 41943 positions at K = 16
    fit below 2^31 (the call reaches the workspace check), 41944 do not."""
    c = _corr(d_state=32, max_L=1 << 16)
    assert _rerank(c, B=1, L=L, K=K) == want


def _psi_cpu(d=64, ds=32, dh=16, dt=16, dp=4, df=4, rk=16, max_L=8, **override):
    import torch
    d_in = dh + dt + dp + df
    shp = {"A_h": (ds, d), "A_e": (ds, d), "P_h": (dh, d), "P_e": (dt, d), "pos_emb": (max_L, dp),
           "P_phi": (df, 5), "W_z": (ds, d_in), "W_h": (ds, d_in), "W_s": (rk, ds), "W_c": (rk, d),
           "w_g": (ds + 5,)}
    shp.update(override)
    return {n: torch.zeros(s, dtype=torch.bfloat16) for n, s in shp.items()}


@pytest.mark.parametrize("field,bad", [
    ("A_e", (32, 72)), ("P_h", (16, 72)), ("P_e", (16, 8)), ("P_phi", (4, 6)), ("W_z", (32, 41)),
    ("W_h", (31, 40)), ("W_s", (16, 33)), ("W_c", (16, 72)), ("w_g", (36,)),
])
def test_corrector_refuses_inconsistent_parameter_shapes(field, bad):
    """Each psi tensor's shape follows from A_h [d_state, d] and the widths the
    other tensors declare; a mismatch would make a kernel read past a buffer."""
    with pytest.raises(ValueError, match="must have shape"):
        brisk.Corrector(_psi_cpu(**{field: bad}), 0.0, 0.0)
    with pytest.raises(ValueError, match="HIP device"):     # consistent shapes reach the device check
        brisk.Corrector(_psi_cpu(), 0.0, 0.0)


def test_binding_tensor_checks():
    """The binding's buffer check reports dtype, exact shape and layout errors
    before the device (the entry points' own uses run on the GPU)."""
    import torch
    chk = brisk._dev_tensor
    with pytest.raises(ValueError, match="must have shape"):
        chk(torch.zeros(2, 3, dtype=torch.int32), "x", torch.int32, shape=(2, 4))
    with pytest.raises(TypeError, match="int32"):
        chk(torch.zeros(2, 3, dtype=torch.int64), "x", torch.int32, shape=(2, 3))
    with pytest.raises(ValueError, match="contiguous"):
        chk(torch.zeros(3, 2, dtype=torch.int32).t(), "x", torch.int32, shape=(2, 3))
    with pytest.raises(ValueError, match="HIP device"):
        chk(torch.zeros(2, 3, dtype=torch.int32), "x", torch.int32, shape=(2, 3))
    with pytest.raises(TypeError, match="Tensor"):
        brisk._ws_bytes(bytearray(16), torch.device("cpu"), 0)
    with pytest.raises(ValueError, match="HIP device"):
        brisk._ws_bytes(torch.zeros(16, dtype=torch.uint8), torch.device("cpu"), 0)


@pytest.mark.parametrize("kw,want", [
    (dict(hidden=None), ENULL), (dict(cl=None), ENULL), (dict(rows=0), ESHAPE), (dict(K=65), ESHAPE),
    (dict(d=4092), EUNSUP), (dict(hidden=MISALIGNED), EUNSUP),
    # 64 rows with 64-key lists: 1024 parts of 64 keys per row, 32 MiB > the 16 MiB scratch
    (dict(rows=64, K=64), -6),
])
def test_propose_noalloc_validation(kw, want):
    """Every rejection happens on the host before any HIP call, the scratch
    limit included (the call never looks the scratch up for such a shape)."""
    a = dict(hidden=FAKE, lm_head=FAKE, rows=32, d=4096, V=126464, K=8, cl=FAKE, ci=FAKE)
    a.update(kw)
    need = ctypes.c_size_t()
    if want == -6:
        assert brisk.lib().brisk_propose_workspace_size(a["rows"], a["d"], a["V"], a["K"],
                                                        ctypes.byref(need)) == OK
        assert need.value > (16 << 20)
    assert brisk.lib().brisk_propose_block_noalloc(a["hidden"], a["lm_head"], a["rows"], a["d"], a["V"], a["K"],
                                                   a["cl"], a["ci"], None) == want


def test_noalloc_scratch_covers_the_decoding_workloads():
    """The five decoding workloads fit the fixed scratch of the no-alloc call."""
    import synth
    out = ctypes.c_size_t()
    for wl in synth.WORKLOADS.values():
        assert brisk.lib().brisk_propose_workspace_size(wl.B * wl.L, wl.d, wl.V, wl.K, ctypes.byref(out)) == OK
        assert out.value <= (16 << 20), wl.name


def test_corrector_tables_size_and_prepare_validation():
    """The per-token tables: sizes, and every rejection before any HIP call."""
    L = brisk.lib()
    c = _corr()
    tb, wb = ctypes.c_size_t(), ctypes.c_size_t()
    assert L.brisk_corrector_tables_size(ctypes.byref(c), 126464, ctypes.byref(tb), ctypes.byref(wb)) == OK
    assert tb.value == 3 * 126464 * 256 * 4                   # [EH; TZ; TH], rows of 256 floats
    assert wb.value == 126464 * (128 + 128) * 4               # P_e E and W_c E_out for every token
    assert L.brisk_corrector_tables_size(ctypes.byref(c), 0, ctypes.byref(tb), ctypes.byref(wb)) == ESHAPE
    assert L.brisk_corrector_tables_size(ctypes.byref(c), 10, None, ctypes.byref(wb)) == ENULL
    big = _corr(d_state=320)
    assert L.brisk_corrector_tables_size(ctypes.byref(big), 10, ctypes.byref(tb), ctypes.byref(wb)) == OK
    assert tb.value == 3 * 10 * 320 * 4                       # rows of d_state floats beyond 256

    def prep(**kw):
        a = dict(W=FAKE, E=FAKE, V=1000, d=4096, tab=FAKE, tab_bytes=1 << 40, ws=FAKE, ws_bytes=1 << 40)
        a.update(kw)
        return L.brisk_corrector_prepare(ctypes.byref(c), a["W"], a["E"], a["V"], a["d"], a["tab"],
                                         a["tab_bytes"], a["ws"], a["ws_bytes"], None)
    assert prep(W=None) == ENULL and prep(tab=None) == ENULL
    assert prep(V=0) == ESHAPE and prep(d=4) == ESHAPE
    assert prep(d=4092) == EUNSUP and prep(tab=MISALIGNED) == EUNSUP
    assert prep(tab_bytes=16) == EWS and prep(ws_bytes=16) == EWS and prep(ws=None) == EWS


def test_rerank_refuses_tables_of_another_vocabulary():
    c = _corr(tables=FAKE, tables_V=1000)
    assert _rerank(c, V=126464) == ESHAPE
    c = _corr(tables=MISALIGNED, tables_V=126464)
    assert _rerank(c, V=126464) == EUNSUP
    c = _corr(tables=FAKE, tables_V=126464)
    assert _rerank(c, V=126464) == EWS                        # passes the table checks
