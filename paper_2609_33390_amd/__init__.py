"""BRISK-DLM decoding hot path on MI355X (gfx950).

Thin Python binding of ``libbrisk.so``: it checks tensor metadata, allocates
outputs and workspaces with torch, and passes raw device pointers and the
current HIP stream to the C ABI declared in ``include/brisk.h``.  Every step of
the computation runs in the library's HIP kernels; there is no CPU fallback,
and a missing or unloadable library raises.

Entry points (same names as the C ABI):

* :func:`propose_block` - LM-head logits and ordered top-K candidates;
* :func:`rerank` - the prefix-conditioned corrector over the candidates;
* :func:`verify_accept` - greedy verification: accept length and correction;
* :func:`rerank_verify` - :func:`rerank` and :func:`verify_accept` in one call;
* :func:`propose_verify` - one LM-head pass for proposal rows (top-K) and
  verifier rows (argmax);
* :func:`verify_commit` - greedy verification and the committed tokens;
* :func:`corrector_loss` - the corrector's training loss on reached positions;
* :func:`spec_verify` - stochastic speculative verification with residual draws;
* :func:`accept_profile` - acceptance profile, tokens per forward and the
  risk-reward position weights from many blocks' accept lengths.
"""
from __future__ import annotations

import ctypes
import os
import threading
from typing import Dict, Optional, Tuple

import torch

__all__ = ["BriskError", "Corrector", "propose_block", "propose_block_noalloc", "propose_lmhead", "propose_merge", "rerank", "rerank_verify", "rerank_hoist", "rerank_finish", "verify_accept", "accept_profile",
           "propose_verify", "verify_commit", "corrector_loss", "spec_verify",
           "lib", "LIB_PATH", "ABI_SYMBOLS", "propose_workspace_size", "rerank_workspace_size"]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libbrisk.so")
ABI_SYMBOLS = ("brisk_status_str", "brisk_abi_version", "brisk_propose_workspace_size",
               "brisk_propose_block", "brisk_propose_block_noalloc", "brisk_propose_lmhead",
               "brisk_propose_merge",
               "brisk_rerank_workspace_size", "brisk_rerank", "brisk_rerank_verify",
               "brisk_rerank_hoist", "brisk_rerank_finish",
               "brisk_verify_accept", "brisk_propose_verify_workspace_size", "brisk_propose_verify",
               "brisk_verify_commit", "brisk_spec_verify_workspace_size", "brisk_spec_verify",
               "brisk_corrector_loss", "brisk_accept_profile_workspace_size",
               "brisk_accept_profile", "brisk_corrector_tables_size", "brisk_corrector_prepare")
PSI_FIELDS = ("A_h", "A_e", "P_h", "P_e", "pos_emb", "P_phi", "W_z", "W_h", "W_s", "W_c", "w_g")

_p = ctypes.c_void_p
_i32 = ctypes.c_int32
_sz = ctypes.c_size_t


class BriskError(RuntimeError):
    """A non-zero status returned by the library."""

    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: status {status} ({_status_str(status)})")


class _CorrectorC(ctypes.Structure):
    _fields_ = ([(n, _i32) for n in ("d_state", "d_hproj", "d_tproj", "d_pos", "d_feat", "rank", "max_L")]
                + [(n, _p) for n in PSI_FIELDS]
                + [("alpha", ctypes.c_float), ("b_g", ctypes.c_float), ("tables", _p), ("tables_V", _i32)])


_lib = None
_lib_lock = threading.Lock()


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    with _lib_lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                                   "`python -m paper_2609_33390_amd.build`")
            L = ctypes.CDLL(LIB_PATH)
            L.brisk_status_str.restype = ctypes.c_char_p
            L.brisk_status_str.argtypes = [ctypes.c_int]
            L.brisk_abi_version.restype = ctypes.c_int
            L.brisk_abi_version.argtypes = []
            L.brisk_propose_workspace_size.restype = ctypes.c_int
            L.brisk_propose_workspace_size.argtypes = [_i32, _i32, _i32, _i32, ctypes.POINTER(_sz)]
            L.brisk_propose_block.restype = ctypes.c_int
            L.brisk_propose_block.argtypes = [_p, _p, _i32, _i32, _i32, _i32, _p, _p, _p, _sz, _p]
            L.brisk_propose_block_noalloc.restype = ctypes.c_int
            L.brisk_propose_block_noalloc.argtypes = [_p, _p, _i32, _i32, _i32, _i32, _p, _p, _p]
            L.brisk_propose_lmhead.restype = ctypes.c_int
            L.brisk_propose_lmhead.argtypes = [_p, _p, _i32, _i32, _i32, _i32, _p, _sz, _p]
            L.brisk_propose_merge.restype = ctypes.c_int
            L.brisk_propose_merge.argtypes = [_i32, _i32, _i32, _p, _p, _p, _sz, _p]
            L.brisk_rerank_workspace_size.restype = ctypes.c_int
            L.brisk_rerank_workspace_size.argtypes = [ctypes.POINTER(_CorrectorC), _i32, _i32, _i32,
                                                      ctypes.POINTER(_sz)]
            L.brisk_rerank.restype = ctypes.c_int
            L.brisk_rerank.argtypes = [ctypes.POINTER(_CorrectorC), _p, _p, _p, _p, _p, _p, _p,
                                       _i32, _i32, _i32, _i32, _i32, _p, _p, _p, _p, _p, _sz, _p]
            L.brisk_rerank_verify.restype = ctypes.c_int
            L.brisk_rerank_verify.argtypes = [ctypes.POINTER(_CorrectorC), _p, _p, _p, _p, _p, _p, _p, _p,
                                              _i32, _i32, _i32, _i32, _i32, _p, _p, _p, _p, _p, _p,
                                              _p, _sz, _p]
            L.brisk_rerank_hoist.restype = ctypes.c_int
            L.brisk_rerank_hoist.argtypes = [ctypes.POINTER(_CorrectorC), _p, _p, _p, _p,
                                             _i32, _i32, _i32, _i32, _i32, _p, _sz, _p]
            L.brisk_rerank_finish.restype = ctypes.c_int
            L.brisk_rerank_finish.argtypes = L.brisk_rerank_verify.argtypes
            L.brisk_verify_accept.restype = ctypes.c_int
            L.brisk_verify_accept.argtypes = [_p, _p, _i32, _i32, _p, _p, _p]
            L.brisk_propose_verify_workspace_size.restype = ctypes.c_int
            L.brisk_propose_verify_workspace_size.argtypes = [_i32, _i32, _i32, _i32, _i32,
                                                              ctypes.POINTER(_sz)]
            L.brisk_propose_verify.restype = ctypes.c_int
            L.brisk_propose_verify.argtypes = [_p, _p, _i32, _i32, _i32, _i32, _i32, _p, _p, _p, _p,
                                               _sz, _p]
            L.brisk_verify_commit.restype = ctypes.c_int
            L.brisk_verify_commit.argtypes = [_p, _p, _i32, _i32, _p, _p, _p, _p]
            L.brisk_spec_verify_workspace_size.restype = ctypes.c_int
            L.brisk_spec_verify_workspace_size.argtypes = [_i32, _i32, _i32, _i32, ctypes.POINTER(_sz)]
            L.brisk_spec_verify.restype = ctypes.c_int
            L.brisk_spec_verify.argtypes = [_p, _p, _p, _p, _p, _p, ctypes.c_uint64, ctypes.c_float,
                                            _i32, _i32, _i32, _i32, _i32, _p, _p, _p, _p, _p, _sz, _p]
            L.brisk_corrector_loss.restype = ctypes.c_int
            L.brisk_corrector_loss.argtypes = [_p, _p, _p, _p, _p, _p, _i32, _i32, _i32, _i32, _i32,
                                               ctypes.c_float, _p, _p, _p, _p, _p]
            L.brisk_accept_profile_workspace_size.restype = ctypes.c_int
            L.brisk_accept_profile_workspace_size.argtypes = [_i32, _i32, ctypes.POINTER(_sz)]
            L.brisk_accept_profile.restype = ctypes.c_int
            L.brisk_accept_profile.argtypes = [_p, _i32, _i32, ctypes.c_double, _p, _p, _p, _p, _p,
                                               _sz, _p]
            L.brisk_corrector_tables_size.restype = ctypes.c_int
            L.brisk_corrector_tables_size.argtypes = [ctypes.POINTER(_CorrectorC), _i32, ctypes.POINTER(_sz),
                                                      ctypes.POINTER(_sz)]
            L.brisk_corrector_prepare.restype = ctypes.c_int
            L.brisk_corrector_prepare.argtypes = [ctypes.POINTER(_CorrectorC), _p, _p, _i32, _i32, _p, _sz, _p,
                                                  _sz, _p]
            _lib = L
        return _lib


def _status_str(status: int) -> str:
    try:
        return lib().brisk_status_str(status).decode()
    except Exception:  # pragma: no cover - message only
        return "?"


def _check(status: int, where: str) -> None:
    if status != 0:
        raise BriskError(status, where)


def _dev_tensor(t: torch.Tensor, name: str, dtype: torch.dtype, ndim: Optional[int] = None, *,
                shape: Optional[Tuple[int, ...]] = None, device: Optional[torch.device] = None) -> None:
    """Checks a tensor before its pointer goes to the library: type, dtype,
    dimension count or exact shape, contiguity, a HIP device, and (when
    ``device`` is given) the same device as the call's other tensors.  A
    wrong shape would otherwise let a kernel read or write past the buffer."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None:
        if tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    elif ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims, got shape {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must live on a HIP device, got {t.device}")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, the call's other tensors on {device}")


def _ws_bytes(ws: torch.Tensor, device: torch.device, need: int, name: str = "workspace") -> int:
    """Size in bytes of a caller's workspace, after checking that it is a
    contiguous tensor on the call's device and holds at least ``need`` bytes."""
    if not isinstance(ws, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not ws.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if ws.device.type != "cuda":
        raise ValueError(f"{name} must live on a HIP device, got {ws.device}")
    if ws.device != device:
        raise ValueError(f"{name} is on {ws.device}, the call's other tensors on {device}")
    nbytes = ws.numel() * ws.element_size()
    if nbytes < need:
        raise ValueError(f"{name} holds {nbytes} bytes, the call needs {need}")
    return nbytes


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream_ptr(device: torch.device, stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


_ws: Dict[Tuple[int, str], torch.Tensor] = {}


def _workspace(device: torch.device, nbytes: int, tag: str) -> torch.Tensor:
    """Per-device cached scratch buffer (grown on demand).  Callers that run the
    same entry point concurrently on several streams must pass their own."""
    key = (device.index if device.index is not None else torch.cuda.current_device(), tag)
    buf = _ws.get(key)
    if buf is None or buf.numel() < nbytes:
        buf = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
        _ws[key] = buf
    return buf


# ----------------------------------------------------------------- propose
def _lmhead_operands(hidden: torch.Tensor, lm_head: torch.Tensor):
    """(rows, d, V, device) of a hidden-state block and an LM head, checked."""
    _dev_tensor(hidden, "hidden", torch.bfloat16, 2)
    dev = hidden.device
    _dev_tensor(lm_head, "lm_head", torch.bfloat16, 2, device=dev)
    rows, d = hidden.shape
    if lm_head.shape[1] != d:
        raise ValueError("hidden and lm_head disagree on d")
    return rows, d, lm_head.shape[0], dev


def propose_workspace_size(rows: int, d: int, V: int, K: int) -> int:
    out = _sz()
    _check(lib().brisk_propose_workspace_size(rows, d, V, K, ctypes.byref(out)),
           "brisk_propose_workspace_size")
    return out.value


def propose_block(hidden: torch.Tensor, lm_head: torch.Tensor, K: int, *,
                  cand_logit: Optional[torch.Tensor] = None, cand_id: Optional[torch.Tensor] = None,
                  workspace: Optional[torch.Tensor] = None, stream=None
                  ) -> Tuple[torch.Tensor, torch.Tensor]:
    """Ordered top-K candidates of every row: (cand_logit [rows,K] fp32, cand_id [rows,K] int32)."""
    rows, d, V, dev = _lmhead_operands(hidden, lm_head)
    if cand_logit is None:
        cand_logit = torch.empty(rows, K, dtype=torch.float32, device=dev)
    if cand_id is None:
        cand_id = torch.empty(rows, K, dtype=torch.int32, device=dev)
    _dev_tensor(cand_logit, "cand_logit", torch.float32, shape=(rows, K), device=dev)
    _dev_tensor(cand_id, "cand_id", torch.int32, shape=(rows, K), device=dev)
    need = propose_workspace_size(rows, d, V, K)
    ws = workspace if workspace is not None else _workspace(dev, need, "propose")
    st = lib().brisk_propose_block(_ptr(hidden), _ptr(lm_head), rows, d, V, K, _ptr(cand_logit),
                                   _ptr(cand_id), _ptr(ws), _ws_bytes(ws, dev, need),
                                   _stream_ptr(dev, stream))
    _check(st, "brisk_propose_block")
    return cand_logit, cand_id


def propose_block_noalloc(hidden: torch.Tensor, lm_head: torch.Tensor, K: int, cand_logit: torch.Tensor,
                          cand_id: torch.Tensor, *, stream=None) -> None:
    """:func:`propose_block` on the library's fixed per-device scratch: the
    library allocates nothing; the caller passes the [rows, K] outputs.  Calls
    that overlap in time on one GPU race (they share the scratch)."""
    rows, d, V, dev = _lmhead_operands(hidden, lm_head)
    _dev_tensor(cand_logit, "cand_logit", torch.float32, shape=(rows, K), device=dev)
    _dev_tensor(cand_id, "cand_id", torch.int32, shape=(rows, K), device=dev)
    st = lib().brisk_propose_block_noalloc(_ptr(hidden), _ptr(lm_head), rows, d, V, K, _ptr(cand_logit),
                                           _ptr(cand_id), _stream_ptr(dev, stream))
    _check(st, "brisk_propose_block_noalloc")


def propose_lmhead(hidden: torch.Tensor, lm_head: torch.Tensor, K: int, workspace: torch.Tensor, *,
                   stream=None) -> None:
    """The LM-head pass of propose_block alone: per-share ordered keys into ``workspace``."""
    rows, d, V, dev = _lmhead_operands(hidden, lm_head)
    need = propose_workspace_size(rows, d, V, K)
    st = lib().brisk_propose_lmhead(_ptr(hidden), _ptr(lm_head), rows, d, V, K, _ptr(workspace),
                                    _ws_bytes(workspace, dev, need), _stream_ptr(dev, stream))
    _check(st, "brisk_propose_lmhead")


def propose_merge(rows: int, V: int, K: int, workspace: torch.Tensor, cand_logit: torch.Tensor,
                  cand_id: torch.Tensor, *, stream=None) -> None:
    """The merge of propose_block alone: candidates from the keys a propose_lmhead left."""
    _dev_tensor(cand_logit, "cand_logit", torch.float32, shape=(rows, K))
    dev = cand_logit.device
    _dev_tensor(cand_id, "cand_id", torch.int32, shape=(rows, K), device=dev)
    need = propose_workspace_size(rows, 8, V, K)   # the key layout does not depend on d
    st = lib().brisk_propose_merge(rows, V, K, _ptr(cand_logit), _ptr(cand_id), _ptr(workspace),
                                   _ws_bytes(workspace, dev, need), _stream_ptr(dev, stream))
    _check(st, "brisk_propose_merge")


# ----------------------------------------------------------------- rerank
class Corrector:
    """Corrector parameters psi: bf16 device tensors plus the two gate scalars."""

    def __init__(self, tensors: Dict[str, torch.Tensor], alpha: float, b_g: float):
        missing = [n for n in PSI_FIELDS if n not in tensors]
        if missing:
            raise ValueError(f"missing corrector tensors: {missing}")
        for n in PSI_FIELDS:
            v = tensors[n]
            if not isinstance(v, torch.Tensor) or v.dim() != (1 if n == "w_g" else 2):
                raise ValueError(f"{n} must be a {1 if n == 'w_g' else 2}-d tensor")
        self.t = {n: tensors[n].contiguous() for n in PSI_FIELDS}
        self.alpha, self.b_g = float(alpha), float(b_g)
        t = self.t
        ds, self.d = t["A_h"].shape
        self.device = t["A_h"].device
        self.dims = dict(d_state=ds, d_hproj=t["P_h"].shape[0], d_tproj=t["P_e"].shape[0],
                         d_pos=t["pos_emb"].shape[1], d_feat=t["P_phi"].shape[0],
                         rank=t["W_s"].shape[0], max_L=t["pos_emb"].shape[0])
        dm = self.dims
        d_in = dm["d_hproj"] + dm["d_tproj"] + dm["d_pos"] + dm["d_feat"]
        want = {"A_h": (ds, self.d), "A_e": (ds, self.d), "P_h": (dm["d_hproj"], self.d),
                "P_e": (dm["d_tproj"], self.d), "pos_emb": (dm["max_L"], dm["d_pos"]),
                "P_phi": (dm["d_feat"], 5), "W_z": (ds, d_in), "W_h": (ds, d_in),
                "W_s": (dm["rank"], ds), "W_c": (dm["rank"], self.d), "w_g": (ds + 5,)}
        for n in PSI_FIELDS:        # every shape first, then dtypes and devices
            if tuple(t[n].shape) != want[n]:
                raise ValueError(f"{n} must have shape {want[n]}, got {tuple(t[n].shape)}")
        for n in PSI_FIELDS:
            _dev_tensor(t[n], n, torch.bfloat16, shape=want[n], device=self.device)
        self._c = _CorrectorC(**self.dims, **{n: _ptr(self.t[n]) for n in PSI_FIELDS},
                              alpha=self.alpha, b_g=self.b_g, tables=None, tables_V=0)
        self.tables: Optional[torch.Tensor] = None

    @property
    def c_struct(self) -> _CorrectorC:
        return self._c

    def prepare(self, lm_head: torch.Tensor, tok_embed: torch.Tensor, *, stream=None) -> torch.Tensor:
        """Compute the per-token tables (brisk_corrector_prepare) for this LM
        head and input embedding; later rerank calls read the candidates' and
        anchors' lifts from them.  Returns the [3, V, max(256, d_state)] fp32
        tables, which the corrector keeps."""
        _dev_tensor(lm_head, "lm_head", torch.bfloat16, 2, device=self.device)
        V, d = lm_head.shape
        if d != self.d:
            raise ValueError(f"lm_head has d = {d}, the corrector d = {self.d}")
        _dev_tensor(tok_embed, "tok_embed", torch.bfloat16, shape=(V, d), device=self.device)
        tb, wb = _sz(), _sz()
        _check(lib().brisk_corrector_tables_size(ctypes.byref(self._c), V, ctypes.byref(tb), ctypes.byref(wb)),
               "brisk_corrector_tables_size")
        vs = max(256, self.dims["d_state"])
        tables = torch.empty(3, V, vs, dtype=torch.float32, device=self.device)
        ws = torch.empty(wb.value, dtype=torch.uint8, device=self.device)
        _check(lib().brisk_corrector_prepare(ctypes.byref(self._c), _ptr(lm_head), _ptr(tok_embed), V, d,
                                             _ptr(tables), tables.numel() * 4, _ptr(ws), wb.value,
                                             _stream_ptr(self.device, stream)),
               "brisk_corrector_prepare")
        self.tables = tables
        self._c.tables = _ptr(tables)
        self._c.tables_V = V
        return tables

    def drop_tables(self) -> None:
        """Forget the per-token tables: rerank projects the embedding rows again."""
        self.tables = None
        self._c.tables = None
        self._c.tables_V = 0


def rerank_workspace_size(corr: Corrector, B: int, L: int, K: int) -> int:
    out = _sz()
    _check(lib().brisk_rerank_workspace_size(ctypes.byref(corr.c_struct), B, L, K, ctypes.byref(out)),
           "brisk_rerank_workspace_size")
    return out.value


def _rerank_args(corr, hidden, ctx_hidden, anchor_tok, lm_head, tok_embed, cand_logit, cand_id, B, L,
                 want_scores, selected, refined, gamma, resid, workspace):
    rows = B * L
    _dev_tensor(hidden, "hidden", torch.bfloat16, 2)
    dev = hidden.device
    if hidden.shape[0] != rows:
        raise ValueError(f"hidden has {hidden.shape[0]} rows, B*L = {rows}")
    d = hidden.shape[1]
    if d != corr.d or corr.device != dev:
        raise ValueError(f"the corrector was built for d = {corr.d} on {corr.device}, "
                         f"the hidden states have d = {d} on {dev}")
    _dev_tensor(ctx_hidden, "ctx_hidden", torch.bfloat16, shape=(B, d), device=dev)
    _dev_tensor(anchor_tok, "anchor_tok", torch.int32, shape=(B,), device=dev)
    _dev_tensor(lm_head, "lm_head", torch.bfloat16, 2, device=dev)
    V = lm_head.shape[0]
    if lm_head.shape[1] != d:
        raise ValueError("hidden and lm_head disagree on d")
    _dev_tensor(tok_embed, "tok_embed", torch.bfloat16, shape=(V, d), device=dev)
    _dev_tensor(cand_id, "cand_id", torch.int32, 2, device=dev)
    K = cand_id.shape[1]
    _dev_tensor(cand_id, "cand_id", torch.int32, shape=(rows, K), device=dev)
    _dev_tensor(cand_logit, "cand_logit", torch.float32, shape=(rows, K), device=dev)
    if selected is None:
        selected = torch.empty(B, L, dtype=torch.int32, device=dev)
    if want_scores:
        if refined is None:
            refined = torch.empty(rows, K, dtype=torch.float32, device=dev)
        if gamma is None:
            gamma = torch.empty(rows, dtype=torch.float32, device=dev)
        if resid is None:
            resid = torch.empty(rows, K, dtype=torch.float32, device=dev)
    _dev_tensor(selected, "selected", torch.int32, shape=(B, L), device=dev)
    for name, t, shp in (("refined", refined, (rows, K)), ("gamma", gamma, (rows,)), ("resid", resid, (rows, K))):
        if t is not None:
            _dev_tensor(t, name, torch.float32, shape=shp, device=dev)
    need = rerank_workspace_size(corr, B, L, K)
    ws = workspace if workspace is not None else _workspace(dev, need, "rerank")
    ws_n = _ws_bytes(ws, dev, need)
    out = {"selected": selected}
    for k, v in (("refined", refined), ("gamma", gamma), ("resid", resid)):
        if v is not None:
            out[k] = v
    return K, d, V, dev, ws, ws_n, out


def rerank(corr: Corrector, hidden: torch.Tensor, ctx_hidden: torch.Tensor, anchor_tok: torch.Tensor,
           lm_head: torch.Tensor, tok_embed: torch.Tensor, cand_logit: torch.Tensor,
           cand_id: torch.Tensor, B: int, L: int, *, want_scores: bool = False,
           selected: Optional[torch.Tensor] = None, refined: Optional[torch.Tensor] = None,
           gamma: Optional[torch.Tensor] = None, resid: Optional[torch.Tensor] = None,
           workspace: Optional[torch.Tensor] = None, stream=None) -> Dict[str, torch.Tensor]:
    """Run the corrector; returns {"selected": [B,L] int32} plus "refined", "gamma",
    "resid" when ``want_scores`` (or when the caller passes those buffers)."""
    K, d, V, dev, ws, ws_n, out = _rerank_args(corr, hidden, ctx_hidden, anchor_tok, lm_head, tok_embed,
                                               cand_logit, cand_id, B, L, want_scores, selected, refined,
                                               gamma, resid, workspace)
    st = lib().brisk_rerank(ctypes.byref(corr.c_struct), _ptr(hidden), _ptr(ctx_hidden),
                            _ptr(anchor_tok), _ptr(lm_head), _ptr(tok_embed), _ptr(cand_logit),
                            _ptr(cand_id), B, L, K, d, V, _ptr(out["selected"]), _ptr(out.get("refined")),
                            _ptr(out.get("gamma")), _ptr(out.get("resid")), _ptr(ws), ws_n,
                            _stream_ptr(dev, stream))
    _check(st, "brisk_rerank")
    return out


def rerank_verify(corr: Corrector, hidden: torch.Tensor, ctx_hidden: torch.Tensor, anchor_tok: torch.Tensor,
                  lm_head: torch.Tensor, tok_embed: torch.Tensor, cand_logit: torch.Tensor,
                  cand_id: torch.Tensor, verifier: torch.Tensor, B: int, L: int, *,
                  want_scores: bool = False, selected: Optional[torch.Tensor] = None,
                  refined: Optional[torch.Tensor] = None, gamma: Optional[torch.Tensor] = None,
                  resid: Optional[torch.Tensor] = None, accept_len: Optional[torch.Tensor] = None,
                  correction: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                  stream=None) -> Dict[str, torch.Tensor]:
    """:func:`rerank` then :func:`verify_accept` on its selections, in one call.
    Returns the rerank outputs plus "accept_len" and "correction" [B] int32."""
    K, d, V, dev, ws, ws_n, out = _rerank_args(corr, hidden, ctx_hidden, anchor_tok, lm_head, tok_embed,
                                               cand_logit, cand_id, B, L, want_scores, selected, refined,
                                               gamma, resid, workspace)
    _dev_tensor(verifier, "verifier", torch.int32, shape=(B, L), device=dev)
    if accept_len is None:
        accept_len = torch.empty(B, dtype=torch.int32, device=dev)
    if correction is None:
        correction = torch.empty(B, dtype=torch.int32, device=dev)
    _dev_tensor(accept_len, "accept_len", torch.int32, shape=(B,), device=dev)
    _dev_tensor(correction, "correction", torch.int32, shape=(B,), device=dev)
    st = lib().brisk_rerank_verify(ctypes.byref(corr.c_struct), _ptr(hidden), _ptr(ctx_hidden),
                                   _ptr(anchor_tok), _ptr(lm_head), _ptr(tok_embed), _ptr(cand_logit),
                                   _ptr(cand_id), _ptr(verifier), B, L, K, d, V, _ptr(out["selected"]),
                                   _ptr(out.get("refined")), _ptr(out.get("gamma")), _ptr(out.get("resid")),
                                   _ptr(accept_len), _ptr(correction), _ptr(ws), ws_n,
                                   _stream_ptr(dev, stream))
    _check(st, "brisk_rerank_verify")
    out["accept_len"] = accept_len
    out["correction"] = correction
    return out


def rerank_hoist(corr: Corrector, hidden: torch.Tensor, ctx_hidden: torch.Tensor, anchor_tok: torch.Tensor,
                 tok_embed: torch.Tensor, B: int, L: int, K: int, workspace: torch.Tensor, *,
                 stream=None) -> None:
    """The part of :func:`rerank` that does not read the candidates, queued on
    ``stream`` into ``workspace`` (which :func:`rerank_finish` then completes);
    it may run while the LM-head pass that makes the candidates streams."""
    _dev_tensor(hidden, "hidden", torch.bfloat16, 2)
    dev = hidden.device
    rows, d = hidden.shape
    if rows != B * L:
        raise ValueError(f"hidden has {rows} rows, B*L = {B * L}")
    if d != corr.d or corr.device != dev:
        raise ValueError(f"the corrector was built for d = {corr.d} on {corr.device}, "
                         f"the hidden states have d = {d} on {dev}")
    _dev_tensor(ctx_hidden, "ctx_hidden", torch.bfloat16, shape=(B, d), device=dev)
    _dev_tensor(anchor_tok, "anchor_tok", torch.int32, shape=(B,), device=dev)
    _dev_tensor(tok_embed, "tok_embed", torch.bfloat16, 2, device=dev)
    if tok_embed.shape[1] != d:
        raise ValueError("hidden and tok_embed disagree on d")
    V = tok_embed.shape[0]
    need = rerank_workspace_size(corr, B, L, K)
    st = lib().brisk_rerank_hoist(ctypes.byref(corr.c_struct), _ptr(hidden), _ptr(ctx_hidden),
                                  _ptr(anchor_tok), _ptr(tok_embed), B, L, K, d, V, _ptr(workspace),
                                  _ws_bytes(workspace, dev, need), _stream_ptr(dev, stream))
    _check(st, "brisk_rerank_hoist")


def rerank_finish(corr: Corrector, hidden: torch.Tensor, ctx_hidden: torch.Tensor, anchor_tok: torch.Tensor,
                  lm_head: torch.Tensor, tok_embed: torch.Tensor, cand_logit: torch.Tensor,
                  cand_id: torch.Tensor, B: int, L: int, workspace: torch.Tensor, *,
                  verifier: Optional[torch.Tensor] = None, want_scores: bool = False,
                  selected: Optional[torch.Tensor] = None, refined: Optional[torch.Tensor] = None,
                  gamma: Optional[torch.Tensor] = None, resid: Optional[torch.Tensor] = None,
                  accept_len: Optional[torch.Tensor] = None, correction: Optional[torch.Tensor] = None,
                  stream=None) -> Dict[str, torch.Tensor]:
    """The rest of :func:`rerank` (``verifier`` None) or :func:`rerank_verify`
    on a ``workspace`` that :func:`rerank_hoist` filled with the same inputs;
    returns what that call returns."""
    K, d, V, dev, ws, ws_n, out = _rerank_args(corr, hidden, ctx_hidden, anchor_tok, lm_head, tok_embed,
                                               cand_logit, cand_id, B, L, want_scores, selected, refined,
                                               gamma, resid, workspace)
    if verifier is not None:
        _dev_tensor(verifier, "verifier", torch.int32, shape=(B, L), device=dev)
        if accept_len is None:
            accept_len = torch.empty(B, dtype=torch.int32, device=dev)
        if correction is None:
            correction = torch.empty(B, dtype=torch.int32, device=dev)
        _dev_tensor(accept_len, "accept_len", torch.int32, shape=(B,), device=dev)
        _dev_tensor(correction, "correction", torch.int32, shape=(B,), device=dev)
    st = lib().brisk_rerank_finish(ctypes.byref(corr.c_struct), _ptr(hidden), _ptr(ctx_hidden),
                                   _ptr(anchor_tok), _ptr(lm_head), _ptr(tok_embed), _ptr(cand_logit),
                                   _ptr(cand_id), _ptr(verifier), B, L, K, d, V, _ptr(out["selected"]),
                                   _ptr(out.get("refined")), _ptr(out.get("gamma")), _ptr(out.get("resid")),
                                   _ptr(accept_len), _ptr(correction), _ptr(ws), ws_n,
                                   _stream_ptr(dev, stream))
    _check(st, "brisk_rerank_finish")
    if verifier is not None:
        out["accept_len"] = accept_len
        out["correction"] = correction
    return out


# ----------------------------------------------------------------- verify
def verify_accept(proposal: torch.Tensor, verifier: torch.Tensor, *,
                  accept_len: Optional[torch.Tensor] = None, correction: Optional[torch.Tensor] = None,
                  stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """(accept_len [B] int32, correction [B] int32; -1 where the block is fully accepted)."""
    _dev_tensor(proposal, "proposal", torch.int32, 2)
    B, L = proposal.shape
    dev = proposal.device
    _dev_tensor(verifier, "verifier", torch.int32, shape=(B, L), device=dev)
    if accept_len is None:
        accept_len = torch.empty(B, dtype=torch.int32, device=dev)
    if correction is None:
        correction = torch.empty(B, dtype=torch.int32, device=dev)
    _dev_tensor(accept_len, "accept_len", torch.int32, shape=(B,), device=dev)
    _dev_tensor(correction, "correction", torch.int32, shape=(B,), device=dev)
    st = lib().brisk_verify_accept(_ptr(proposal), _ptr(verifier), B, L, _ptr(accept_len),
                                   _ptr(correction), _stream_ptr(dev, stream))
    _check(st, "brisk_verify_accept")
    return accept_len, correction


def accept_profile(accept_len: torch.Tensor, M: int, *, eps: float = 0.0,
                   workspace: Optional[torch.Tensor] = None, stream=None) -> Dict[str, torch.Tensor]:
    """Acceptance profile of verified blocks: ``a``, ``w_raw``, ``w`` [M] and
    ``tpf_fpt`` [2], all float64 on the device of ``accept_len``."""
    _dev_tensor(accept_len, "accept_len", torch.int32, 1)
    n = accept_len.shape[0]
    dev = accept_len.device
    nbytes = _sz(0)
    _check(lib().brisk_accept_profile_workspace_size(n, M, ctypes.byref(nbytes)),
           "brisk_accept_profile_workspace_size")
    if workspace is None:
        workspace = _workspace(dev, nbytes.value, "profile")
    ws_n = _ws_bytes(workspace, dev, nbytes.value)
    out = {k: torch.empty(M, dtype=torch.float64, device=dev) for k in ("a", "w_raw", "w")}
    out["tpf_fpt"] = torch.empty(2, dtype=torch.float64, device=dev)
    st = lib().brisk_accept_profile(_ptr(accept_len) if n > 0 else None, n, M, float(eps),
                                    _ptr(out["a"]), _ptr(out["w_raw"]), _ptr(out["w"]),
                                    _ptr(out["tpf_fpt"]), _ptr(workspace), ws_n,
                                    _stream_ptr(dev, stream))
    _check(st, "brisk_accept_profile")
    return out


def propose_verify(hidden: torch.Tensor, lm_head: torch.Tensor, rows_prop: int, K: int, *,
                   cand_logit: Optional[torch.Tensor] = None, cand_id: Optional[torch.Tensor] = None,
                   ver_token: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                   stream=None) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """One LM-head pass: the first ``rows_prop`` rows of ``hidden`` get ordered
    top-K candidates, the remaining rows their argmax token.
    Returns (cand_logit [rows_prop, K], cand_id [rows_prop, K], ver_token [rows_ver])."""
    rows, d, V, dev = _lmhead_operands(hidden, lm_head)
    rows_ver = rows - rows_prop
    if rows_prop < 0 or rows_ver < 0:
        raise ValueError("rows_prop must lie in [0, hidden rows]")
    if cand_logit is None:
        cand_logit = torch.empty(rows_prop, K, dtype=torch.float32, device=dev)
    if cand_id is None:
        cand_id = torch.empty(rows_prop, K, dtype=torch.int32, device=dev)
    if ver_token is None:
        ver_token = torch.empty(rows_ver, dtype=torch.int32, device=dev)
    _dev_tensor(cand_logit, "cand_logit", torch.float32, shape=(rows_prop, K), device=dev)
    _dev_tensor(cand_id, "cand_id", torch.int32, shape=(rows_prop, K), device=dev)
    _dev_tensor(ver_token, "ver_token", torch.int32, shape=(rows_ver,), device=dev)
    nbytes = _sz(0)
    _check(lib().brisk_propose_verify_workspace_size(rows_prop, rows_ver, d, V, K, ctypes.byref(nbytes)),
           "brisk_propose_verify_workspace_size")
    ws = workspace if workspace is not None else _workspace(dev, nbytes.value, "propose")
    st = lib().brisk_propose_verify(_ptr(hidden), _ptr(lm_head), rows_prop, rows_ver, d, V, K,
                                    _ptr(cand_logit) if rows_prop else None,
                                    _ptr(cand_id) if rows_prop else None,
                                    _ptr(ver_token) if rows_ver else None, _ptr(ws),
                                    _ws_bytes(ws, dev, nbytes.value), _stream_ptr(dev, stream))
    _check(st, "brisk_propose_verify")
    return cand_logit, cand_id, ver_token


def verify_commit(proposal: torch.Tensor, verifier: torch.Tensor, *, stream=None
                  ) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """(accept_len [B], committed [B, L + 1] padded with -1, n_committed [B])."""
    _dev_tensor(proposal, "proposal", torch.int32, 2)
    B, L = proposal.shape
    dev = proposal.device
    _dev_tensor(verifier, "verifier", torch.int32, shape=(B, L), device=dev)
    acc = torch.empty(B, dtype=torch.int32, device=dev)
    committed = torch.empty(B, L + 1, dtype=torch.int32, device=dev)
    n = torch.empty(B, dtype=torch.int32, device=dev)
    st = lib().brisk_verify_commit(_ptr(proposal), _ptr(verifier), B, L, _ptr(acc), _ptr(committed),
                                   _ptr(n), _stream_ptr(dev, stream))
    _check(st, "brisk_verify_commit")
    return acc, committed, n


def corrector_loss(ver_hidden: torch.Tensor, lm_head: torch.Tensor, cand_id: torch.Tensor,
                   cand_logit: torch.Tensor, refined: torch.Tensor, accept_len: torch.Tensor,
                   B: int, L: int, *, beta: float = 0.01, stream=None) -> Dict[str, torch.Tensor]:
    """Per-position losses ``loss_pos``, ``ce``, ``kl`` [B*L] and ``loss_mean``
    [2] = (mean over reached positions, their count)."""
    rows = B * L
    nrows, d, V, dev = _lmhead_operands(ver_hidden, lm_head)
    if nrows != rows:
        raise ValueError(f"ver_hidden has {nrows} rows, B*L = {rows}")
    _dev_tensor(cand_id, "cand_id", torch.int32, 2, device=dev)
    K = cand_id.shape[1]
    _dev_tensor(cand_id, "cand_id", torch.int32, shape=(rows, K), device=dev)
    _dev_tensor(cand_logit, "cand_logit", torch.float32, shape=(rows, K), device=dev)
    _dev_tensor(refined, "refined", torch.float32, shape=(rows, K), device=dev)
    _dev_tensor(accept_len, "accept_len", torch.int32, shape=(B,), device=dev)
    out = {k: torch.empty(rows, dtype=torch.float32, device=dev) for k in ("loss_pos", "ce", "kl")}
    out["loss_mean"] = torch.empty(2, dtype=torch.float32, device=dev)
    st = lib().brisk_corrector_loss(_ptr(ver_hidden), _ptr(lm_head), _ptr(cand_id), _ptr(cand_logit),
                                    _ptr(refined), _ptr(accept_len), B, L, K, d, V, float(beta),
                                    _ptr(out["loss_pos"]), _ptr(out["ce"]), _ptr(out["kl"]),
                                    _ptr(out["loss_mean"]), _stream_ptr(dev, stream))
    _check(st, "brisk_corrector_loss")
    return out


def spec_verify(ver_hidden: torch.Tensor, lm_head: torch.Tensor, proposal: torch.Tensor,
                cand_id: torch.Tensor, cand_prob: Optional[torch.Tensor], u_accept: torch.Tensor, seed: int,
                temperature: float = 1.0, *, workspace: Optional[torch.Tensor] = None,
                stream=None) -> Dict[str, torch.Tensor]:
    """Stochastic verification: ``accept_len``, ``correction`` [B] and the
    per-position ``row_accept``, ``row_resample`` [B*L].  ``cand_prob=None``
    is the greedy proposer (pi = point mass at the proposal)."""
    rows, d, V, dev = _lmhead_operands(ver_hidden, lm_head)
    _dev_tensor(proposal, "proposal", torch.int32, 2, device=dev)
    B, L = proposal.shape
    if B * L != rows:
        raise ValueError(f"proposal is [{B}, {L}], ver_hidden has {rows} rows")
    _dev_tensor(cand_id, "cand_id", torch.int32, 2, device=dev)
    K = cand_id.shape[1]
    _dev_tensor(cand_id, "cand_id", torch.int32, shape=(rows, K), device=dev)
    if cand_prob is not None:
        _dev_tensor(cand_prob, "cand_prob", torch.float32, shape=(rows, K), device=dev)
    _dev_tensor(u_accept, "u_accept", torch.float32, shape=(rows,), device=dev)
    nbytes = _sz(0)
    _check(lib().brisk_spec_verify_workspace_size(B, L, V, K, ctypes.byref(nbytes)),
           "brisk_spec_verify_workspace_size")
    ws = workspace if workspace is not None else _workspace(dev, nbytes.value, "spec")
    ws_n = _ws_bytes(ws, dev, nbytes.value)
    out = {"accept_len": torch.empty(B, dtype=torch.int32, device=dev),
           "correction": torch.empty(B, dtype=torch.int32, device=dev),
           "row_accept": torch.empty(B * L, dtype=torch.int32, device=dev),
           "row_resample": torch.empty(B * L, dtype=torch.int32, device=dev)}
    st = lib().brisk_spec_verify(_ptr(ver_hidden), _ptr(lm_head), _ptr(proposal), _ptr(cand_id),
                                 _ptr(cand_prob), _ptr(u_accept), int(seed) & ((1 << 64) - 1),
                                 float(temperature), B, L, K, d, V, _ptr(out["accept_len"]),
                                 _ptr(out["correction"]), _ptr(out["row_accept"]),
                                 _ptr(out["row_resample"]), _ptr(ws), ws_n, _stream_ptr(dev, stream))
    _check(st, "brisk_spec_verify")
    return out
