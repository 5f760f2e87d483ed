"""Plain CPU oracle of one BRISK-DLM decoding step (test infrastructure).

This file is test infrastructure.  Only the test suite, the smoke check and
the benchmark's CPU-baseline leg may import it; the library under
``paper_2609_33390_amd`` never does, and this file imports nothing from it.

It computes, slowly and in the paper's order, what the GPU path computes:

1. proposal logits of every masked position (Section 3.3 "Rejection-aware
   candidate selection"; Algorithm 1(b), first step): the plain matrix product
   of the hidden states with the LM head;
2. the ordered candidate set C_i = TopK(q_i, K) (Section 3.3; Appendix
   "Candidate-Refinement Head Details"): a full stable sort;
3. the prefix-conditioned corrector (Eq. inference_head_state and
   Eq. candidate_residual in Section 3.3; Eq. head_residual_logits and the
   head configuration table in the Appendix; Algorithm 1(b) loop): the
   recurrence stepped left to right, every candidate scored exhaustively;
4. greedy verification (Section 2.2 accepted prefix; Section 3.3
   speculative acceptance at temperature zero; Algorithm 1(b) verify/commit):
   a linear scan for the first mismatch.

Arithmetic is float64 on the exact values of the bf16 inputs.  Where a float
decides an integer (the top-K order, the argmax of the refined scores) the
value is first rounded to float32, the precision the GPU kernels decide in.

Readings of points the paper leaves open (each is also listed in the design
notes): R1 corrector widths from one state width; R2 bias-free minGRU cell;
R3 Init = tanh of two bias-free maps; R4 h_c enters only through u_0;
R5 bias-free projections concatenated in the listed order; R6 feature order
and meaning; R7 0-based position embedding; R8 gate takes the raw features;
R9 E_out is the LM head; R10 base logit = raw logit; R11 greedy selection;
R12 ties in top-K go to the lower token id; R13 greedy acceptance.

Parity pins: top-K and verification are pinned by brute force; the logits by
exact rational arithmetic and one-hot special cases; the corrector by
closed-form special cases, the zero-weight reduction, candidate membership,
the paper's parameter count and a brute force over all candidate paths.  The
corrector has no worked numeric example in the paper, so its *values* beyond
those special cases are pinned only through them.
"""
from __future__ import annotations

from typing import Dict, Optional, Tuple

import numpy as np

__all__ = [
    "bf16_to_f64", "lm_logits", "topk", "propose_block", "corrector_init",
    "confidence_features", "rerank", "verify_accept", "corrector_param_count", "verifier_argmax",
    "verify_commit", "reached_mask", "corrector_loss",
]


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact value of bfloat16 bit patterns (the upper half of an IEEE binary32)."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _f32(x: np.ndarray) -> np.ndarray:
    return np.asarray(x, dtype=np.float64).astype(np.float32)


def lm_logits(H: np.ndarray, W_bits: np.ndarray, chunk: int = 8192) -> np.ndarray:
    """Proposal logits l^q[r, v] = <H[r], W[v]> rounded to float32.

    ``H`` is [rows, d] float64 (exact bf16 values); ``W_bits`` the [V, d] LM
    head as bf16 bits.  Each logit is one full-length float64 dot product; the
    vocabulary is visited in slices only to bound memory.
    """
    V = W_bits.shape[0]
    out = np.empty((H.shape[0], V), dtype=np.float32)
    for v0 in range(0, V, chunk):
        Wc = bf16_to_f64(W_bits[v0:v0 + chunk])
        out[:, v0:v0 + chunk] = _f32(H @ Wc.T)
    return out


def topk(logits: np.ndarray, K: int) -> Tuple[np.ndarray, np.ndarray]:
    """Ordered top-K of each row: logit descending, lower token id first on ties.

    A stable sort of the negated float32 logits keeps equal logits in id
    order, so the first K entries are exactly that order.
    """
    order = np.argsort(-logits, axis=1, kind="stable")[:, :K]
    vals = np.take_along_axis(logits, order, axis=1)
    return vals.astype(np.float32), order.astype(np.int32)


def propose_block(H_bits: np.ndarray, W_bits: np.ndarray, K: int) -> Tuple[np.ndarray, np.ndarray]:
    """Candidate logits and ids [rows, K] of every masked position."""
    return topk(lm_logits(bf16_to_f64(H_bits), W_bits), K)


def _sigmoid(x):
    """Logistic function; exp overflow for very negative inputs yields exactly 0."""
    with np.errstate(over="ignore"):
        return 1.0 / (1.0 + np.exp(-x))


def corrector_param_count(d_state, d_hproj, d_tproj, d_pos, d_feat, rank, max_L, d) -> int:
    """Trainable parameters of the corrector under readings R1-R5 and R8."""
    d_in = d_hproj + d_tproj + d_pos + d_feat
    return (2 * d_state * d            # Init: A_h, A_e
            + d_hproj * d + d_tproj * d  # P_h, P_e
            + max_L * d_pos + d_feat * 5  # position table, P_phi
            + 2 * d_state * d_in       # minGRU: W_z, W_h
            + rank * d_state + rank * d  # W_s, W_c
            + d_state + 5 + 2)         # w_g, b_g, alpha


def corrector_init(psi: Dict[str, np.ndarray], h_c: np.ndarray, E_x0: np.ndarray) -> np.ndarray:
    """u_0 = Init_psi(h_c, E(x_0)) = tanh(A_h h_c + A_e E(x_0))  (reading R3)."""
    return np.tanh(h_c @ psi["A_h"].T + E_x0 @ psi["A_e"].T)


def confidence_features(cand_logit: np.ndarray, cand_id: np.ndarray,
                        prev: np.ndarray, prev_logit: np.ndarray) -> np.ndarray:
    """The five base-proposal confidence features of each row (reading R6).

    [top1 - top2, top1 - top4, 1[prev is top1], 1[prev in top4],
    top1 - logit of prev at this position].  Inputs are per-row arrays:
    ``cand_logit``/``cand_id`` [n, K] in candidate order, ``prev``/``prev_logit`` [n].
    """
    c = cand_logit.astype(np.float64)
    is_top1 = (cand_id[:, 0] == prev).astype(np.float64)
    in_top4 = (cand_id[:, :4] == prev[:, None]).any(axis=1).astype(np.float64)
    return np.stack([c[:, 0] - c[:, 1], c[:, 0] - c[:, 3], is_top1, in_top4,
                     c[:, 0] - prev_logit.astype(np.float64)], axis=1)


def rerank(psi: Dict[str, np.ndarray], alpha: float, b_g: float,
           H: np.ndarray, h_c: np.ndarray, x0: np.ndarray,
           W_bits: np.ndarray, E_bits: np.ndarray,
           cand_logit: np.ndarray, cand_id: np.ndarray, B: int, L: int,
           prefix: Optional[np.ndarray] = None) -> Dict[str, np.ndarray]:
    """Run the corrector over every block, left to right.

    ``psi`` maps field names to float64 arrays (exact bf16 values); ``H``
    [B*L, d] and ``h_c`` [B, d] are float64; ``W_bits``/``E_bits`` are the LM
    head and the input embedding as bf16 bits (rows are gathered and decoded
    as needed).  ``cand_logit``/``cand_id`` [B*L, K] are the candidate sets.

    With ``prefix`` [B, L] given, the token fed to step i+1 is ``prefix[:, i]``
    instead of the oracle's own selection (teacher forcing); every other
    output is still computed.  Returns float32 ``refined``/``resid`` [B*L, K],
    ``gamma``/``margin`` [B*L], ``phi`` [B*L, 5] and int32 ``selected`` [B, L].
    """
    K = cand_id.shape[1]
    sig_a = _sigmoid(float(alpha))
    rows = B * L
    refined = np.zeros((rows, K), np.float32)
    resid = np.zeros((rows, K), np.float32)
    gamma = np.zeros(rows, np.float32)
    margin = np.zeros(rows, np.float32)
    phi_out = np.zeros((rows, 5), np.float32)
    selected = np.zeros((B, L), np.int32)

    u = corrector_init(psi, h_c, bf16_to_f64(E_bits[x0]))       # [B, d_state]
    prev = np.asarray(x0, dtype=np.int64)
    for i in range(L):
        r = np.arange(B) * L + i
        m = H[r]                                                  # m_i
        ids = cand_id[r]
        base = cand_logit[r]
        # full-vocabulary logit of the previous token at this position
        prev_logit = _f32(np.einsum("bd,bd->b", bf16_to_f64(W_bits[prev]), m))
        phi = confidence_features(base, ids, prev, prev_logit)
        x_hat = np.concatenate([m @ psi["P_h"].T,
                                bf16_to_f64(E_bits[prev]) @ psi["P_e"].T,
                                np.broadcast_to(psi["pos_emb"][i], (B, psi["pos_emb"].shape[1])),
                                phi @ psi["P_phi"].T], axis=1)
        z = _sigmoid(x_hat @ psi["W_z"].T)
        h_tilde = x_hat @ psi["W_h"].T
        u = (1.0 - z) * u + z * h_tilde
        g = sig_a * _sigmoid(np.concatenate([u, phi], axis=1) @ psi["w_g"] + b_g)
        s = u @ psi["W_s"].T                                      # W_s u_i   [B, rank]
        Eo = bf16_to_f64(W_bits[ids])                             # E_out(v)  [B, K, d]
        c = Eo @ psi["W_c"].T                                     # W_c E_out(v) [B, K, rank]
        dres = np.einsum("br,bkr->bk", s, c)
        lt = base.astype(np.float64) + g[:, None] * dres
        lt32 = _f32(lt)
        kstar = np.argmax(lt32, axis=1)                           # first maximum
        srt = np.sort(lt32.astype(np.float64), axis=1)
        refined[r] = lt32
        resid[r] = _f32(dres)
        gamma[r] = _f32(g)
        margin[r] = _f32(srt[:, -1] - srt[:, -2])
        phi_out[r] = _f32(phi)
        selected[:, i] = ids[np.arange(B), kstar]
        prev = (prefix[:, i] if prefix is not None else selected[:, i]).astype(np.int64)
    return dict(selected=selected, refined=refined, resid=resid, gamma=gamma,
                margin=margin, phi=phi_out)


def verify_accept(proposal: np.ndarray, verifier: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Accepted-prefix length and correction token of each block (reading R13).

    accept_b = number of leading positions where the proposal equals the
    verifier's argmax token; correction_b = the verifier's token at the first
    mismatch, or -1 when the whole block is accepted.
    """
    B, L = proposal.shape
    accept = np.full(B, L, np.int32)
    correction = np.full(B, -1, np.int32)
    for b in range(B):
        for i in range(L):
            if proposal[b, i] != verifier[b, i]:
                accept[b] = i
                correction[b] = verifier[b, i]
                break
    return accept, correction


def verifier_argmax(H_bits: np.ndarray, W_bits: np.ndarray) -> np.ndarray:
    """The verifier's greedy token of each row: the largest float32 logit, the
    lower token id among equal ones (the first entry of the ordered top-K)."""
    _, ids = topk(lm_logits(bf16_to_f64(H_bits), W_bits), 1)
    return ids[:, 0]


def verify_commit(proposal: np.ndarray, verifier: np.ndarray) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Committed tokens of each block (Algorithm 1(b) verify and commit): the
    accepted prefix, then the verifier's token at the first mismatch; the
    L + 1 slots are padded with -1.  Returns (accept, committed, n_committed)."""
    B, L = proposal.shape
    accept, correction = verify_accept(proposal, verifier)
    committed = np.full((B, L + 1), -1, np.int32)
    n = np.zeros(B, np.int32)
    for b in range(B):
        a = int(accept[b])
        committed[b, :a] = proposal[b, :a]
        n[b] = a
        if a < L:
            committed[b, a] = correction[b]
            n[b] = a + 1
    return accept, committed, n


def reached_mask(accept: np.ndarray, L: int) -> np.ndarray:
    """Positions whose verification decision is reached (Appendix head
    details): the accepted prefix and the first rejected position; every
    position of a fully accepted block.  [B, L] bool."""
    B = len(accept)
    m = np.zeros((B, L), dtype=bool)
    for b in range(B):
        m[b, :min(int(accept[b]) + 1, L)] = True
    return m


def _log_softmax(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    m = x.max(axis=-1, keepdims=True)
    return x - m - np.log(np.exp(x - m).sum(axis=-1, keepdims=True))


def corrector_loss(ver_H: np.ndarray, W_bits: np.ndarray, cand_id: np.ndarray,
                   cand_logit: np.ndarray, refined: np.ndarray, accept: np.ndarray, L: int,
                   beta: float = 0.01) -> Dict[str, np.ndarray]:
    """Corrector training loss on one batch of blocks (Appendix head details,
    Eq. head_training_loss).

    At position j with candidate set S_j: p_S = the verifier distribution
    restricted to S_j and renormalised (softmax of the verifier logits
    <E_out[v], h_j> at the candidate ids), q_S = the base distribution
    restricted to S_j (softmax of the candidate logits), r = softmax of the
    refined logits.  l_j = CE(p_S, r) + beta KL(q_S || r); the loss is the
    mean of l_j over the reached positions.  ``ver_H`` is [B*L, d] float64.
    """
    rows, K = cand_id.shape
    W = bf16_to_f64(W_bits)
    lp = np.einsum("rkd,rd->rk", W[cand_id.astype(np.int64)], ver_H)
    log_p = _log_softmax(lp)
    log_q = _log_softmax(cand_logit)
    log_r = _log_softmax(refined)
    p, q = np.exp(log_p), np.exp(log_q)
    ce = -(p * log_r).sum(axis=1)
    kl = (q * (log_q - log_r)).sum(axis=1)
    per = ce + beta * kl
    mask = reached_mask(accept, L).reshape(rows)
    loss_pos = np.where(mask, per, 0.0)
    return dict(loss_pos=loss_pos, ce=ce, kl=kl, mask=mask,
                mean=float(loss_pos.sum() / mask.sum()), count=int(mask.sum()))
