"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each test names what it pins: exact rational arithmetic, brute force on tiny
inputs, closed-form special cases of the corrector, the paper's printed
parameter count, and invariants the paper states.
"""
import itertools
from fractions import Fraction

import numpy as np
import pytest

import fixtures
import oracle
import synth
from oracle_io import f64_to_bf16_bits, oracle_inputs


# ---------------------------------------------------------------- bf16 format
def test_bf16_decode_known_patterns():
    bits = np.array([0x3F80, 0xC000, 0x0000, 0x8000, 0x3E80, 0x7F7F, 0x0001], np.uint16)
    want = [1.0, -2.0, 0.0, -0.0, 0.25, 3.3895313892515355e38, 9.183549615799121e-41]
    got = oracle.bf16_to_f64(bits)
    assert np.array_equal(got, np.array(want))


# ---------------------------------------------------------------- logits
def _rand_bf16(rng, shape, scale=1.0):
    f = (rng.standard_normal(shape) * scale).astype(np.float32)
    return (f.view(np.uint32) >> 16).astype(np.uint16)      # truncation: still valid bf16 values


def test_logits_match_exact_rational_sum():
    """Each logit is the float32 rounding of the exact dot product."""
    rng = np.random.default_rng(11)
    Hb, Wb = _rand_bf16(rng, (3, 16)), _rand_bf16(rng, (20, 16), 0.05)
    got = oracle.lm_logits(oracle.bf16_to_f64(Hb), Wb)
    Hf, Wf = oracle.bf16_to_f64(Hb), oracle.bf16_to_f64(Wb)
    for r in range(3):
        for v in range(20):
            exact = sum(Fraction(float(a)) * Fraction(float(b)) for a, b in zip(Hf[r], Wf[v]))
            ref = np.float32(float(exact))
            ulp = np.spacing(np.float32(abs(ref)))
            assert abs(Fraction(float(got[r, v])) - exact) <= Fraction(float(ulp)) / 2 * (1 + Fraction(1, 10**6))


def test_logits_one_hot_rows_pick_coordinates():
    """With W[v] the one-hot vector e_(v mod d), logit[r, v] is H[r, v mod d]."""
    rng = np.random.default_rng(3)
    d, V = 8, 24
    Hb = _rand_bf16(rng, (4, d))
    Wf = np.zeros((V, d))
    Wf[np.arange(V), np.arange(V) % d] = 1.0
    got = oracle.lm_logits(oracle.bf16_to_f64(Hb), f64_to_bf16_bits(Wf))
    H = oracle.bf16_to_f64(Hb)
    assert np.array_equal(got, H[:, np.arange(V) % d].astype(np.float32))


# ---------------------------------------------------------------- top-K
def _topk_bruteforce(row, K):
    """K passes of 'largest remaining value, smallest id among equals'."""
    taken, ids = set(), []
    for _ in range(K):
        best = None
        for v, x in enumerate(row):
            if v in taken:
                continue
            if best is None or x > row[best]:
                best = v
        taken.add(best)
        ids.append(best)
    return ids


@pytest.mark.parametrize("K", [1, 4, 8, 16])
def test_topk_against_bruteforce_with_ties(K):
    rng = np.random.default_rng(K)
    lg = rng.integers(-6, 6, size=(5, 40)).astype(np.float32) / 4   # many exact ties
    vals, ids = oracle.topk(lg, K)
    for r in range(5):
        want = _topk_bruteforce(list(lg[r]), K)
        assert list(ids[r]) == want
        assert np.array_equal(vals[r], lg[r, want])


def test_topk_tie_goes_to_lower_id():
    lg = np.array([[1.0, 3.0, 2.0, 3.0, 3.0, 0.5]], np.float32)
    vals, ids = oracle.topk(lg, 4)
    assert ids.tolist() == [[1, 3, 4, 2]]
    assert vals.tolist() == [[3.0, 3.0, 3.0, 2.0]]


def test_planted_target_is_top1_on_tiny_block():
    blk = synth.make_block("tiny-d64-v512", "cpu")
    io = oracle_inputs(blk)
    _, ids = oracle.propose_block(io["H_bits"], io["W_bits"], blk.wl.K)
    assert np.array_equal(ids[:, 0], blk.targets.numpy())


# ---------------------------------------------------------------- verification
def test_verify_bruteforce_all_mismatch_patterns():
    L = 6
    rng = np.random.default_rng(5)
    ver = rng.integers(0, 100, size=(1, L)).astype(np.int32)
    for pattern in itertools.product([0, 1], repeat=L):
        prop = ver.copy()
        for i, bad in enumerate(pattern):
            if bad:
                prop[0, i] = ver[0, i] + 1 + i
        acc, corr = oracle.verify_accept(prop, ver)
        lead = next((i for i, bad in enumerate(pattern) if bad), L)
        assert acc[0] == lead
        assert corr[0] == (ver[0, lead] if lead < L else -1)


def test_verify_invariants():
    rng = np.random.default_rng(6)
    B, L = 50, 9
    ver = rng.integers(0, 5, size=(B, L)).astype(np.int32)
    prop = np.where(rng.random((B, L)) < 0.8, ver, rng.integers(0, 5, size=(B, L))).astype(np.int32)
    acc, corr = oracle.verify_accept(prop, ver)
    assert np.all((acc >= 0) & (acc <= L))
    assert np.array_equal(acc == L, np.all(prop == ver, axis=1))
    assert np.array_equal(corr == -1, acc == L)
    acc2, corr2 = oracle.verify_accept(ver, ver)
    assert np.all(acc2 == L) and np.all(corr2 == -1)


# ---------------------------------------------------------------- corrector structure
def test_loss_kl_coefficient_is_the_tables():
    """The loss's anchor KL coefficient is the one the head configuration
    table prints (Appendix, Table head_implementation_details)."""
    import inspect
    g = fixtures.table("head_config.txt")
    assert inspect.signature(oracle.corrector_loss).parameters["beta"].default == g["anchor_kl_coefficient"]


def test_param_count_matches_paper():
    """Head configuration table: 128 state, 64/64 projections, 16/16, rank 64,
    7 positions; 1.89M trainable parameters at the 8B hidden size 4096; the
    step input is 160 wide."""
    g = fixtures.table("head_config.txt")
    dims = dict(d_state=int(g["state_dim"]), d_hproj=int(g["hidden_proj_dim"]), d_tproj=int(g["token_proj_dim"]),
                d_pos=int(g["position_proj_dim"]), d_feat=int(g["feature_proj_dim"]), rank=int(g["residual_rank"]),
                max_L=int(g["proposal_positions"]))
    n = oracle.corrector_param_count(d=4096, **dims)
    assert n == 1_884_487
    # the table prints 1.89M; this reading counts 0.29% fewer
    assert abs(n - g["trainable_params"]) / g["trainable_params"] < 0.003
    assert dims["d_hproj"] + dims["d_tproj"] + dims["d_pos"] + dims["d_feat"] == 160
    assert synth.corrector_dims(128, 7) == dims


# ---------------------------------------------------------------- corrector special cases
def _zero_psi(ds, dh, dt, dp, df, rk, max_L, d):
    d_in = dh + dt + dp + df
    return {"A_h": np.zeros((ds, d)), "A_e": np.zeros((ds, d)), "P_h": np.zeros((dh, d)),
            "P_e": np.zeros((dt, d)), "pos_emb": np.zeros((max_L, dp)), "P_phi": np.zeros((df, 5)),
            "W_z": np.zeros((ds, d_in)), "W_h": np.zeros((ds, d_in)), "W_s": np.zeros((rk, ds)),
            "W_c": np.zeros((rk, d)), "w_g": np.zeros(ds + 5)}


class Tiny:
    """Hand-built block: d=8, V=6, one sequence of 2 positions, K=4, state 2,
    projection widths 1 (hidden), 1 (token), 2 (position), 1 (feature), rank 2.
    x_hat = [P_h m (slot 0), P_e E(prev) (slot 1), pos (slots 2-3), P_phi phi (slot 4)]."""
    d, V, B, L, K = 8, 6, 1, 2, 4

    def __init__(self):
        self.psi = _zero_psi(2, 1, 1, 2, 1, 2, 2, self.d)
        self.psi["W_s"] = np.eye(2)
        self.psi["W_c"][0, 0] = 1.0          # W_c E_out(v) = (W[v,0], W[v,1])
        self.psi["W_c"][1, 1] = 1.0
        self.Wf = np.zeros((self.V, self.d))
        self.Ef = np.zeros((self.V, self.d))
        self.H = np.zeros((2, self.d))
        self.h_c = np.zeros((1, self.d))
        self.x0 = np.array([5])
        self.cand_id = np.array([[0, 1, 2, 3], [0, 1, 2, 3]], np.int32)
        self.cand_logit = np.array([[3.0, 2.875, 2.75, 2.5], [3.0, 2.875, 2.75, 2.5]], np.float32)
        self.alpha, self.b_g = 0.0, 0.0

    def run(self, prefix=None):
        return oracle.rerank(self.psi, self.alpha, self.b_g, self.H, self.h_c, self.x0,
                             f64_to_bf16_bits(self.Wf), f64_to_bf16_bits(self.Ef),
                             self.cand_logit, self.cand_id, self.B, self.L, prefix=prefix)


def test_zero_weights_reduce_to_top1():
    """All-zero corrector: residual 0, refined = base logits, x_i = top-1 and
    gamma = sigmoid(0) * sigmoid(0) = 1/4."""
    blk = synth.make_block("tiny-d64-v512", "cpu", psi_std=0.0)
    io = oracle_inputs(blk)
    cl, ci = oracle.propose_block(io["H_bits"], io["W_bits"], blk.wl.K)
    out = oracle.rerank(io["psi"], 0.0, 0.0, io["H"], io["h_c"], io["x0"], io["W_bits"],
                        io["E_bits"], cl, ci, blk.wl.B, blk.wl.L)
    assert np.array_equal(out["selected"].ravel(), ci[:, 0])
    assert np.array_equal(out["refined"], cl)
    assert np.all(out["resid"] == 0) and np.all(out["gamma"] == np.float32(0.25))


def test_closed_gate_reduces_to_top1():
    blk = synth.make_block("tiny-d64-v512", "cpu", psi_std=2.0)
    io = oracle_inputs(blk)
    cl, ci = oracle.propose_block(io["H_bits"], io["W_bits"], blk.wl.K)
    out = oracle.rerank(io["psi"], -200.0, 0.0, io["H"], io["h_c"], io["x0"], io["W_bits"],
                        io["E_bits"], cl, ci, blk.wl.B, blk.wl.L)
    assert np.array_equal(out["selected"].ravel(), ci[:, 0])


def test_selection_stays_in_candidate_set():
    """The head only reranks the candidates, never adds one."""
    for std in (0.02, 0.5, 3.0):
        blk = synth.make_block("tiny-d64-v512", "cpu", psi_std=std, flat_all=True)
        io = oracle_inputs(blk)
        cl, ci = oracle.propose_block(io["H_bits"], io["W_bits"], blk.wl.K)
        out = oracle.rerank(io["psi"], io["alpha"], io["b_g"], io["H"], io["h_c"], io["x0"],
                            io["W_bits"], io["E_bits"], cl, ci, blk.wl.B, blk.wl.L)
        for r, x in enumerate(out["selected"].ravel()):
            assert x in ci[r]


def test_residual_sign_and_gate_closed_form():
    """z = 0 keeps u_i = u_0 = tanh(A_h h_c); W_s = I and W_c reading the first
    two coordinates give d_k = u_0 . (W[v_k,0], W[v_k,1]); a saturated gate
    gives gamma = sigmoid(alpha) = 1/2.  Candidate 1 gets +2*tanh(2)/2 and wins."""
    t = Tiny()
    t.h_c[0, 0] = 1.0
    t.psi["A_h"][0, 0] = 2.0                         # u_0 = (tanh 2, 0)
    t.psi["pos_emb"][:, 0] = 1.0
    t.psi["W_z"][:, 2] = -80.0                       # z = sigmoid(-80) -> 0
    t.b_g = 60.0                                     # sigmoid(60) -> 1
    t.Wf[1, 0] = 2.0
    t.Wf[3, 0] = -1.0
    out = t.run()
    u0 = np.tanh(2.0)
    assert np.allclose(out["resid"][0], [0.0, 2 * u0, 0.0, -u0], atol=1e-12)
    assert np.allclose(out["gamma"], 0.5, atol=1e-12)
    assert np.allclose(out["refined"][0], [3.0, 2.875 + u0, 2.75, 2.5 - 0.5 * u0], atol=1e-6)
    assert out["selected"].tolist() == [[1, 1]]


def test_update_limits_and_position_index():
    """z = 1 gives u_i = W_h x_hat_i: with only the position slot nonzero,
    u_i = W_h[:, pos] pos_emb[i-1] (0-based table row).  The two table rows
    map to opposite states, so the residual flips sign between the positions."""
    t = Tiny()
    t.psi["pos_emb"][:] = np.eye(2)                  # row 0 -> slot 2, row 1 -> slot 3
    t.psi["W_z"][:, 2:4] = 80.0                      # z -> 1 at both steps
    t.psi["W_h"][:, 2] = [1.0, 0.0]
    t.psi["W_h"][:, 3] = [-1.0, 0.0]
    t.b_g = 60.0
    t.alpha = 60.0                                   # gamma -> 1
    t.Wf[1, 0] = 0.5                                 # helps id 1 at step 1
    t.Wf[2, 0] = -0.5                                # helps id 2 at step 2
    out = t.run()
    assert np.allclose(out["resid"][0], [0, 0.5, -0.5, 0], atol=1e-12)
    assert np.allclose(out["resid"][1], [0, -0.5, 0.5, 0], atol=1e-12)
    assert out["selected"].tolist() == [[1, 2]]


def test_update_blend_half_gate():
    """W_z = 0 gives z = 1/2: u_1 = (u_0 + h~_1)/2 and u_2 = (u_1 + h~_2)/2."""
    t = Tiny()
    t.h_c[0, 0] = 1.0
    t.psi["A_h"][0, 0] = 0.5
    t.psi["pos_emb"][:, 0] = [1.0, 2.0]
    t.psi["W_h"][:, 2] = [0.25, 0.0]
    t.Wf[:4, 0] = [1.0, 0.0, 0.0, 0.0]
    t.alpha, t.b_g = 60.0, 60.0
    out = t.run()
    u0 = np.tanh(0.5)
    u1 = 0.5 * u0 + 0.5 * 0.25
    u2 = 0.5 * u1 + 0.5 * 0.5
    assert np.isclose(out["resid"][0, 0], u1, atol=1e-7)
    assert np.isclose(out["resid"][1, 0], u2, atol=1e-7)


def test_previous_selected_token_feeds_next_step():
    """E(x_{i-1}) enters through P_e.  Token 1's embedding pushes step 2
    towards id 3, token 0's towards id 2; forcing either prefix shows it."""
    t = Tiny()
    t.psi["pos_emb"][:, 0] = 1.0
    t.psi["W_z"][:, 2] = 80.0                        # z -> 1
    t.psi["P_e"][0, 0] = 1.0                         # tproj = E(prev)[0]
    t.psi["W_h"][:, 1] = [1.0, 0.0]                  # u_i = (E(prev)[0], 0)
    t.Ef[0, 0], t.Ef[1, 0], t.Ef[5, 0] = -1.0, 1.0, 0.0
    t.Wf[2, 0], t.Wf[3, 0] = -1.0, 1.0
    t.alpha, t.b_g = 60.0, 60.0
    f0 = t.run(prefix=np.array([[0, 0]]))
    f1 = t.run(prefix=np.array([[1, 0]]))
    assert f0["selected"][0, 1] == 2 and f1["selected"][0, 1] == 3
    assert np.allclose(f0["resid"][1], [0, 0, 1, -1], atol=1e-12)
    assert np.allclose(f1["resid"][1], [0, 0, -1, 1], atol=1e-12)
    free = t.run()
    assert free["selected"][0, 0] == 0 and free["selected"][0, 1] == 2


def test_features_hand_worked():
    cl = np.array([[5.0, 4.0, 3.0, 2.0, 1.0]] * 3)
    ci = np.array([[10, 11, 12, 13, 14]] * 3)
    prev = np.array([10, 12, 99])
    prev_logit = np.array([5.0, 3.0, 0.5])
    phi = oracle.confidence_features(cl, ci, prev, prev_logit)
    assert phi.tolist() == [[1, 3, 1, 1, 0], [1, 3, 0, 1, 2], [1, 3, 0, 0, 4.5]]


def test_feature5_uses_full_vocab_logit_and_gate_uses_raw_features():
    """phi_5 = top1 - <W[prev], m_i> even when prev is not a candidate; with
    only the phi_1 coefficient of w_g set to 1, gamma = sigmoid(phi_1)."""
    t = Tiny()
    t.H[0, :2] = [1.0, 2.0]
    t.Wf[5, :2] = [0.5, 0.25]                        # x0 = 5, not a candidate
    t.psi["w_g"][2] = 1.0                            # index d_state + 0 -> phi_1
    t.alpha = 60.0
    out = t.run()
    assert np.isclose(out["phi"][0, 4], 3.0 - (0.5 + 0.5))
    assert np.isclose(out["phi"][0, 0], 0.125)
    assert np.isclose(out["gamma"][0], 1 / (1 + np.exp(-0.125)), atol=1e-7)


def test_init_reads_anchor_embedding_through_A_e():
    """u_0 = tanh(A_h h_c + A_e E(x_0)) (Init, reading R3) with h_c = 0 and only
    A_e[1, 1] = 1 gives u_0 = (0, tanh E[x_0, 1]) = (0, tanh 1.5).  z = 0 keeps
    u_i = u_0 at both steps; W_s = I and W_c reading the first two coordinates
    give d_k = tanh(1.5) * W[v_k, 1], so candidate 2 (W[2, 1] = 1) wins.

    Mutations this fails under: dropping the A_e term (u_0 = 0, residual 0);
    applying A_e to the LM-head row W[x_0] instead of the input embedding
    E[x_0] (W[x_0, 1] = -2, so the residual flips sign and top-1 stays)."""
    t = Tiny()
    t.psi["A_e"][1, 1] = 1.0
    t.Ef[5, 1] = 1.5                                 # x_0 = 5
    t.Wf[5, 1] = -2.0                                # a different value in E_out's row of x_0
    t.psi["pos_emb"][:, 0] = 1.0
    t.psi["W_z"][:, 2] = -80.0                       # z -> 0: u_i = u_0
    t.b_g = 60.0                                     # gamma = sigmoid(0) * 1 = 1/2
    t.Wf[2, 1] = 1.0
    out = t.run()
    u0 = np.tanh(1.5)
    for i in range(2):
        assert np.allclose(out["resid"][i], [0.0, 0.0, u0, 0.0], atol=1e-12)
    assert np.allclose(out["refined"][0], [3.0, 2.875, 2.75 + 0.5 * u0, 2.5], atol=1e-6)
    assert out["selected"].tolist() == [[2, 2]]


def test_hidden_projection_reads_the_current_row():
    """Slot 0 of x_hat is P_h m_i (reading R5).  With P_h reading coordinate 0,
    z = 1 and W_h copying slot 0 into the first state element, u_i = (m_i[0], 0)
    and d_k = m_i[0] * W[v_k, 0].  The two rows differ (m_1[0] = 1,
    m_2[0] = -2): residuals (0, 0.5, -0.5, 0) then (0, -1, 1, 0), selections 1
    then 2.

    Mutations this fails under: feeding m_{i-1} or m_{i+1} instead of m_i
    (the rows swap, at step 1 through numpy's wrap-around), or leaving the
    slot out (residual 0, top-1 at both steps)."""
    t = Tiny()
    t.H[0, 0], t.H[1, 0] = 1.0, -2.0
    t.psi["P_h"][0, 0] = 1.0
    t.psi["pos_emb"][:, 0] = 1.0
    t.psi["W_z"][:, 2] = 80.0                        # z -> 1
    t.psi["W_h"][:, 0] = [1.0, 0.0]                  # u_i = (x_hat_0, 0)
    t.Wf[1, 0], t.Wf[2, 0] = 0.5, -0.5
    t.b_g = 60.0                                     # gamma = 1/2
    out = t.run()
    assert np.allclose(out["resid"][0], [0.0, 0.5, -0.5, 0.0], atol=1e-12)
    assert np.allclose(out["resid"][1], [0.0, -1.0, 1.0, 0.0], atol=1e-12)
    assert np.allclose(out["refined"][1], [3.0, 2.375, 3.25, 2.5], atol=1e-6)
    assert out["selected"].tolist() == [[1, 2]]


def test_feature_projection_slot():
    """Slot 4 of x_hat is P_phi phi_i (readings R5, R6).  P_phi = [1, -1, 1/2,
    1/4, 1/4] and W_h copying slot 4 into the first state element give
    u_i = (P_phi phi_i, 0) at z = 1, and d_k = u_i[0] * W[v_k, 0] with only
    W[1, 0] = 1.  Step 1: phi = (1/8, 1/2, 0, 0, 3) (x_0 = 5 is no candidate,
    its logit is 0), P_phi phi = 3/8.  Step 2: x_1 = 1 is in the top 4 but not
    top 1, phi = (1/8, 1/2, 0, 1, 3), P_phi phi = 5/8.

    Mutations this fails under: leaving the slot out (residual 0, top-1
    selected), any reordering of the five features before P_phi (for example
    swapping the two indicator features gives 7/8 at step 2, reversing them
    gives other values at both steps), or gating the projection instead of the
    raw features."""
    t = Tiny()
    t.psi["P_phi"][0] = [1.0, -1.0, 0.5, 0.25, 0.25]
    t.psi["pos_emb"][:, 0] = 1.0
    t.psi["W_z"][:, 2] = 80.0                        # z -> 1
    t.psi["W_h"][:, 4] = [1.0, 0.0]                  # u_i = (P_phi phi_i, 0)
    t.Wf[1, 0] = 1.0
    t.b_g = 60.0                                     # gamma = 1/2
    out = t.run()
    assert np.allclose(out["phi"][0], [0.125, 0.5, 0.0, 0.0, 3.0], atol=1e-7)
    assert np.allclose(out["phi"][1], [0.125, 0.5, 0.0, 1.0, 3.0], atol=1e-7)
    assert np.allclose(out["resid"][0], [0.0, 0.375, 0.0, 0.0], atol=1e-12)
    assert np.allclose(out["resid"][1], [0.0, 0.625, 0.0, 0.0], atol=1e-12)
    assert np.allclose(out["gamma"], 0.5, atol=1e-12)
    assert out["selected"].tolist() == [[1, 1]]


def test_unique_self_consistent_path_is_the_greedy_one():
    """Brute force over all K^L candidate paths of a small block: run the
    corrector teacher-forced on each path; exactly one path chooses itself at
    every step, and it is the free-running result."""
    wl = synth.Workload("path-brute", B=1, L=6, d=64, V=512, K=4, r=32,
                        sigma=0.3, flat_frac=1.0, seed=9)
    blk = synth.make_block(wl, "cpu", psi_std=0.6)
    io = oracle_inputs(blk)
    cl, ci = oracle.propose_block(io["H_bits"], io["W_bits"], wl.K)
    free = oracle.rerank(io["psi"], io["alpha"], io["b_g"], io["H"], io["h_c"], io["x0"],
                         io["W_bits"], io["E_bits"], cl, ci, 1, wl.L)
    paths = np.array(list(itertools.product(range(wl.K), repeat=wl.L)))     # candidate slots
    P = len(paths)
    tok = ci[np.arange(wl.L)[None, :], paths]                                # [P, L]
    rep = lambda a: np.repeat(a, P, axis=0)
    out = oracle.rerank(io["psi"], io["alpha"], io["b_g"], np.tile(io["H"], (P, 1)), rep(io["h_c"]),
                        rep(io["x0"]), io["W_bits"], io["E_bits"], np.tile(cl, (P, 1)),
                        np.tile(ci, (P, 1)), P, wl.L, prefix=tok)
    consistent = np.all(out["selected"] == tok, axis=1)
    assert consistent.sum() == 1
    assert np.array_equal(tok[consistent][0], free["selected"][0])
    # the corrector changed at least one choice, so the check is not vacuous
    assert not np.array_equal(free["selected"][0], ci[:, 0])


def test_verify_commit_brute_force_and_invariants():
    rng = np.random.default_rng(11)
    for L in (1, 2, 5, 9):
        for _ in range(40):
            prop = rng.integers(0, 3, (3, L)).astype(np.int32)
            ver = rng.integers(0, 3, (3, L)).astype(np.int32)
            acc, com, n = oracle.verify_commit(prop, ver)
            for b in range(3):
                a = next((i for i in range(L) if prop[b, i] != ver[b, i]), L)
                want = list(prop[b, :a]) + ([int(ver[b, a])] if a < L else [])
                assert acc[b] == a and n[b] == len(want)
                assert list(com[b, :n[b]]) == want and np.all(com[b, n[b]:] == -1)
                # every committed token is what the verifier would emit at its position
                assert np.array_equal(com[b, :n[b]], ver[b, :n[b]])


def test_verifier_argmax_ties_and_planted_row():
    H = np.zeros((2, 8), np.float32)
    H[:, 0] = 1.0
    W = np.zeros((6, 8), np.float32)
    W[2, 0] = 2.0
    W[4, 0] = 2.0            # exact tie with row 2: the lower id wins
    W[5, 0] = -3.0
    bits = lambda x: (np.asarray(x, np.float32).view(np.uint32) >> 16).astype(np.uint16)
    assert list(oracle.verifier_argmax(bits(H), bits(W))) == [2, 2]
    H[1, 0] = -1.0           # now row 5 (-3 * -1 = 3) is the largest
    assert list(oracle.verifier_argmax(bits(H), bits(W))) == [2, 5]


def _softmax(x):
    e = np.exp(x - np.max(x))
    return e / e.sum()


def _loss_case(seed, K=5, B=2, L=3, d=8, V=11):
    rng = np.random.default_rng(seed)
    H = rng.standard_normal((B * L, d))
    W = rng.standard_normal((V, d)).astype(np.float32)
    W_bits = (W.view(np.uint32) >> 16).astype(np.uint16)
    ids = np.stack([rng.choice(V, K, replace=False) for _ in range(B * L)]).astype(np.int32)
    cl = rng.standard_normal((B * L, K))
    ref = rng.standard_normal((B * L, K))
    return H, W_bits, ids, cl, ref


def test_corrector_loss_hand_formula():
    H, W_bits, ids, cl, ref = _loss_case(0)
    acc = np.array([3, 0])
    out = oracle.corrector_loss(H, W_bits, ids, cl, ref, acc, 3, beta=0.25)
    W = oracle.bf16_to_f64(W_bits)
    for r in range(6):
        lp = np.array([W[v] @ H[r] for v in ids[r]])
        p, q, rr = _softmax(lp), _softmax(cl[r]), _softmax(ref[r])
        want = -np.sum(p * np.log(rr)) + 0.25 * np.sum(q * np.log(q / rr))
        assert out["ce"][r] + 0.25 * out["kl"][r] == pytest.approx(want, rel=1e-12)
    # block 0 fully accepted: all 3 positions; block 1 rejected at position 1: only it
    assert list(out["mask"]) == [True, True, True, True, False, False]
    assert out["count"] == 4
    assert out["mean"] == pytest.approx(out["loss_pos"].sum() / 4, rel=1e-15)


def test_corrector_loss_special_cases():
    H, W_bits, ids, cl, ref = _loss_case(1)
    acc = np.array([3, 3])
    # refined equal to the base logits: the KL term vanishes
    out = oracle.corrector_loss(H, W_bits, ids, cl, cl, acc, 3)
    assert np.allclose(out["kl"], 0.0, atol=1e-14)
    # refined logits that reproduce the verifier distribution: CE = its entropy (the minimum)
    W = oracle.bf16_to_f64(W_bits)
    lp = np.stack([[W[v] @ H[r] for v in ids[r]] for r in range(6)])
    out2 = oracle.corrector_loss(H, W_bits, ids, cl, lp + 3.0, acc, 3)
    ent = np.array([-np.sum(_softmax(x) * np.log(_softmax(x))) for x in lp])
    assert np.allclose(out2["ce"], ent, rtol=1e-12)
    out3 = oracle.corrector_loss(H, W_bits, ids, cl, ref, acc, 3)
    assert np.all(out3["ce"] >= ent - 1e-12) and np.all(out3["kl"] >= -1e-14)


def test_reached_mask_brute_force():
    for L in (1, 4, 7):
        for a in range(L + 1):
            m = oracle.reached_mask(np.array([a]), L)[0]
            assert list(m) == [j <= a for j in range(L)]
