"""CPU checks of the benchmark's roofline arithmetic: the algorithmic bytes
and flops of one step (LM head once, hidden and context states, corrector
parameters, gathered candidate and previous-token rows, outputs; LM-head
product plus the corrector per position and Init per sequence) and the
roofline time they give on MI355X (8 TB/s HBM3E, 2516.6 TFLOP/s dense bf16).
The expected figures are written out from those terms, not taken from the
code under test."""
import pytest

import bench
import synth


def test_decode_step_bytes_term_by_term():
    # llada8b-b1-l32: B = 1, L = 32, d = 4096, V = 126464, K = 8, r = 256
    # (d_state 256; projections and rank 128; position and feature widths 32)
    d, V, rows, B, K = 4096, 126464, 32, 1, 8
    psi = (2 * 256 * d          # A_h, A_e
           + 128 * d + 128 * d  # P_h, P_e
           + 32 * 32            # position table, L x d_pos
           + 32 * 5             # P_phi
           + 2 * 256 * 320      # W_z, W_h over the 320-wide step input
           + 128 * 256          # W_s
           + 128 * d            # W_c
           + 256 + 5)           # gate weights on u and the five features
    assert psi == 3_868_069
    expected = (2 * V * d                 # lm_head, read once
                + 2 * rows * d            # hidden states
                + 2 * B * d               # context state
                + 2 * psi                 # corrector parameters, bf16
                + rows * (K + 1) * 2 * d  # candidate rows and previous-token row
                + rows * K * 8            # candidates out
                + rows * 4 + B * 8)       # selections, accept length and correction
    assert expected == 1_046_361_042
    b, _ = bench.step_work(synth.WORKLOADS["llada8b-b1-l32"])
    assert b == expected


@pytest.mark.parametrize("name,gflop,t_roof_us", [
    ("llada8b-b1-l32", 33.5, 130.8),      # HBM-bound: 1.0464 GB / 8 TB/s
    ("llada8b-b64-l32", 2144.3, 852.1),   # MFMA-bound
    ("dream7b-b16-l32", 566.8, 225.2),
    ("llada8b-b256-l16", 4289.1, 1704.3),
])
def test_step_flops_and_roofline_time(name, gflop, t_roof_us):
    wl = synth.WORKLOADS[name]
    b, f = bench.step_work(wl)
    assert f / 1e9 == pytest.approx(gflop, rel=2e-3)
    assert bench.t_roof(b, f) * 1e6 == pytest.approx(t_roof_us, rel=1e-3)
    # the LM-head product dominates; the corrector adds about 11 MFLOP per
    # position at d = 4096, K = 8 (17 at the Dream shape's K = 16)
    rows = wl.B * wl.L
    per_pos = (f - 2 * rows * wl.d * wl.V) / rows
    assert per_pos / 1e6 == pytest.approx(17.0 if wl.K == 16 else 11.0, rel=0.06)


def test_lmhead_pass_work_and_bound():
    wl = synth.WORKLOADS["llada8b-b1-l32"]
    b, f = bench.lmhead_work(wl)
    assert b == 2 * 126464 * 4096 + 2 * 32 * 4096
    assert f == 2 * 32 * 4096 * 126464
    assert not bench.is_mfma_bound(b, f)   # intensity 32 flop/B against a ridge of 315
    wl = synth.WORKLOADS["llada8b-b256-l16"]
    assert bench.is_mfma_bound(*bench.lmhead_work(wl))
