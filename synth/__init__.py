"""Seeded synthetic inputs for one BRISK-DLM decoding step.

This module only *draws* inputs: hidden states of the masked block positions,
the frozen LM head and input embedding, the context state and anchor token,
the corrector parameters, and the verifier's argmax tokens.  It holds none of
the method's arithmetic (no logits of the proposal path, no top-K, no
corrector, no acceptance scan).  Both the HIP path and the CPU oracle read the
same tensors produced here; neither is imported by this module.

The verifier tokens stand in for the output of the causal verifier pass that
the paper runs on the same backbone (Section 3.3, Algorithm 1(b)): the argmax
of the LM head applied to a noisy copy of each hidden state.  That argmax is a
property of the synthetic workload, not of the method, so it is computed here
with plain torch arithmetic in float32.

Values are drawn with ``torch.Generator`` on the device the caller names.  The
CPU and GPU generators produce different streams for the same seed, so a test
that compares the two paths always generates once and hands the very same
tensors to both.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional, Tuple, Union

import numpy as np
import torch

__all__ = [
    "Workload", "WORKLOADS", "corrector_dims", "Block", "make_block",
    "bf16_bits", "PSI_FIELDS",
]


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and value recipe of one synthetic decoding step.

    ``sigma`` is the verifier noise scale: one float for every sequence, or a
    ``(lo, hi)`` pair from which each sequence draws its own value uniformly.
    ``flat_frac`` is the fraction of rows that get no planted target (their
    logits stay flat, which produces near-ties in top-K and in the rerank).
    """
    name: str
    B: int
    L: int
    d: int
    V: int
    K: int
    r: int
    sigma: Union[float, Tuple[float, float]]
    flat_frac: float
    seed: int

    @property
    def rows(self) -> int:
        return self.B * self.L


# The five decoding workloads.  Shapes follow the LLaDA-8B backbone
# (hidden 4096, vocab 126464) and the Dream-7B backbone (hidden 3584, vocab
# 152064); the tiny one is small enough for exhaustive CPU checks.
WORKLOADS: Dict[str, Workload] = {
    w.name: w for w in [
        Workload("tiny-d64-v512", B=1, L=8, d=64, V=512, K=4, r=32,
                 sigma=0.3, flat_frac=0.0, seed=0),
        Workload("llada8b-b1-l32", B=1, L=32, d=4096, V=126464, K=8, r=256,
                 sigma=0.3, flat_frac=0.0, seed=1),
        Workload("llada8b-b64-l32", B=64, L=32, d=4096, V=126464, K=8, r=256,
                 sigma=(0.1, 0.6), flat_frac=0.0, seed=2),
        Workload("dream7b-b16-l32", B=16, L=32, d=3584, V=152064, K=16, r=256,
                 sigma=0.3, flat_frac=0.5, seed=3),
        Workload("llada8b-b256-l16", B=256, L=16, d=4096, V=126464, K=8, r=256,
                 sigma=0.3, flat_frac=0.0, seed=4),
    ]
}


def corrector_dims(r: int, max_L: int) -> Dict[str, int]:
    """Corrector widths for a given state width ``r``.

    The paper's head (Appendix, head configuration table) has a 128-wide state,
    64-wide hidden and token projections, 16-wide position and feature
    projections and a rank-64 residual.  A different ``r`` keeps those ratios.
    """
    return dict(d_state=r, d_hproj=r // 2, d_tproj=r // 2, d_pos=r // 8,
                d_feat=r // 8, rank=r // 2, max_L=max_L)


# Corrector parameter tensors, in the order the C structure lists them.
PSI_FIELDS = ("A_h", "A_e", "P_h", "P_e", "pos_emb", "P_phi", "W_z", "W_h",
              "W_s", "W_c", "w_g")


def psi_shapes(dims: Dict[str, int], d: int) -> Dict[str, Tuple[int, ...]]:
    ds, dh, dt = dims["d_state"], dims["d_hproj"], dims["d_tproj"]
    dp, df, rk = dims["d_pos"], dims["d_feat"], dims["rank"]
    d_in = dh + dt + dp + df
    return {
        "A_h": (ds, d), "A_e": (ds, d), "P_h": (dh, d), "P_e": (dt, d),
        "pos_emb": (dims["max_L"], dp), "P_phi": (df, 5),
        "W_z": (ds, d_in), "W_h": (ds, d_in), "W_s": (rk, ds), "W_c": (rk, d),
        "w_g": (ds + 5,),
    }


@dataclasses.dataclass
class Block:
    """All inputs of one decoding step (bf16 tensors unless noted)."""
    wl: Workload
    dims: Dict[str, int]
    H: torch.Tensor          # [B*L, d]  hidden state m_i of every masked position
    W: torch.Tensor          # [V, d]    LM head rows (also the output embedding)
    E: torch.Tensor          # [V, d]    input token embedding
    h_c: torch.Tensor        # [B, d]    context representation
    x0: torch.Tensor         # [B] int32 token preceding the block
    verifier: torch.Tensor   # [B, L] int32 verifier argmax tokens
    targets: torch.Tensor    # [B*L] int64 planted target id, -1 on flat rows
    psi: Dict[str, torch.Tensor]
    alpha: float
    b_g: float
    sigma: torch.Tensor      # [B] float32 verifier noise scale per sequence


def _child_gens(seed: int, n: int, device) -> list:
    gens = []
    for child in np.random.SeedSequence(seed).spawn(n):
        g = torch.Generator(device=device)
        g.manual_seed(int(child.generate_state(1, dtype=np.uint64)[0]) & ((1 << 63) - 1))
        gens.append(g)
    return gens


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """Host uint16 array with the bit patterns of a bfloat16 tensor."""
    assert t.dtype == torch.bfloat16
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def make_block(wl: Union[Workload, str], device: Union[str, torch.device] = "cpu", *,
               plant_scale: float = 3.0, psi_std: float = 0.02,
               flat_all: bool = False, dup_top: bool = False,
               seed: Optional[int] = None, verifier_chunk: int = 16384) -> Block:
    """Draw one decoding step's inputs on ``device``.

    Recipe (every rounding to bf16 is round-to-nearest-even, done once):

    * ``H ~ N(0, 1)``, ``h_c ~ N(0, 1)``, ``x0 ~ U{0..V-1}``.
    * ``E ~ N(0, 0.02^2)``; ``W ~ N(0, 0.02^2)`` in fp32, then every non-flat
      row ``r`` gets a target ``t_r ~ U{0..V-1}`` whose row is increased by
      ``plant_scale * H_r / |H_r|`` (``H_r`` already bf16-rounded; collisions
      add up), and W is rounded to bf16 at the end.
    * ``dup_top``: each planted target row is copied onto a second random id,
      so the two tokens have bitwise-equal logits (exercises the id tie-break).
    * Corrector tensors and the two gate scalars ``~ N(0, psi_std^2)``, bf16.
    * Verifier token of row ``r``: argmax over the vocabulary of the fp32
      product of the bf16 W with ``H_r + sigma_b * n_r``, ``n_r ~ N(0, 1)``,
      lowest id on ties.
    """
    if isinstance(wl, str):
        wl = WORKLOADS[wl]
    device = torch.device(device)
    B, L, d, V, r = wl.B, wl.L, wl.d, wl.V, wl.r
    rows = B * L
    dims = corrector_dims(r, L)
    shapes = psi_shapes(dims, d)
    gens = _child_gens(wl.seed if seed is None else seed, 16 + len(PSI_FIELDS) + 2, device)
    (gH, gW, gT, gF, gE, gC, gX, gN, gS, gD) = gens[:10]
    gpsi = gens[16:]

    f32 = dict(dtype=torch.float32, device=device)
    H = torch.randn(rows, d, generator=gH, **f32).to(torch.bfloat16)
    W32 = torch.randn(V, d, generator=gW, **f32).mul_(0.02)
    targets = torch.randint(0, V, (rows,), generator=gT, device=device)
    if flat_all:
        flat = torch.ones(rows, dtype=torch.bool, device=device)
    else:
        n_flat = int(np.floor(rows * wl.flat_frac))
        perm = torch.randperm(rows, generator=gF, device=device)
        flat = torch.zeros(rows, dtype=torch.bool, device=device)
        flat[perm[:n_flat]] = True
    targets = torch.where(flat, torch.full_like(targets, -1), targets)
    planted = (~flat).nonzero().flatten()
    if planted.numel():
        Hp = H[planted].float()
        boost = plant_scale * Hp / Hp.norm(dim=1, keepdim=True)
        W32.index_add_(0, targets[planted], boost)
    W = W32.to(torch.bfloat16)
    del W32
    if dup_top and planted.numel():
        partner = torch.randint(0, V, (planted.numel(),), generator=gD, device=device)
        src = targets[planted]
        keep = partner != src
        W[partner[keep]] = W[src[keep]]

    E = torch.randn(V, d, generator=gE, **f32).mul_(0.02).to(torch.bfloat16)
    h_c = torch.randn(B, d, generator=gC, **f32).to(torch.bfloat16)
    x0 = torch.randint(0, V, (B,), generator=gX, device=device).to(torch.int32)

    if isinstance(wl.sigma, tuple):
        lo, hi = wl.sigma
        sigma = lo + (hi - lo) * torch.rand(B, generator=gS, **f32)
    else:
        sigma = torch.full((B,), float(wl.sigma), **f32)
    noise = torch.randn(rows, d, generator=gN, **f32)
    Hn = H.float() + sigma.repeat_interleave(L)[:, None] * noise
    best = torch.full((rows,), -float("inf"), **f32)
    best_id = torch.zeros(rows, dtype=torch.int64, device=device)
    for v0 in range(0, V, verifier_chunk):
        lg = W[v0:v0 + verifier_chunk].float() @ Hn.T          # [chunk, rows]
        m, a = lg.max(dim=0)                                    # first max in chunk
        upd = m > best                                          # strict: earlier chunk wins ties
        best = torch.where(upd, m, best)
        best_id = torch.where(upd, a + v0, best_id)
    verifier = best_id.to(torch.int32).view(B, L)

    psi = {}
    for name, g in zip(PSI_FIELDS, gpsi):
        psi[name] = torch.randn(shapes[name], generator=g, **f32).mul_(psi_std).to(torch.bfloat16)
    ab = torch.randn(2, generator=gpsi[len(PSI_FIELDS)], **f32).mul_(psi_std).to(torch.bfloat16)
    alpha, b_g = (float(v) for v in ab.float().cpu())
    return Block(wl=wl, dims=dims, H=H, W=W, E=E, h_c=h_c, x0=x0, verifier=verifier,
                 targets=targets, psi=psi, alpha=alpha, b_g=b_g, sigma=sigma)
