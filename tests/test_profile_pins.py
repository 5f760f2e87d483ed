"""Pins of the acceptance-profile oracle against what the paper and the
mathematics fix (CPU only)."""
import itertools
from fractions import Fraction

import numpy as np
import pytest

import fixtures
import oracle


@pytest.mark.parametrize("N,r,printed", [tuple(float(x) for x in row) for row in fixtures.rows("tpf_stride8.txt")])
def test_stride_equation_printed_values(N, r, printed):
    # Section 2.2 prints TPF at stride N = 8 for these rejection rates, to two
    # decimals (tests/golden/tpf_stride8.txt)
    assert abs(oracle.tpf_stride(int(N), r) - printed) <= 0.005


@pytest.mark.parametrize("N", [2, 3, 8, 17])
@pytest.mark.parametrize("r", [0.0, 0.05, 0.3, 1.0])
def test_isd_instantiation_reduces_to_stride_equation(N, r):
    a = np.full(N - 1, 1.0 - r)
    assert oracle.tpf_isd(a) == pytest.approx(oracle.tpf_stride(N, r), rel=1e-12)


def test_general_form_with_isd_rewards_and_costs():
    rng = np.random.default_rng(1)
    for M in (1, 2, 5, 31):
        a = rng.uniform(0.0, 1.0, M)
        k = np.arange(M + 1)
        g = 2.0 + np.minimum(k, M - 1)
        c = np.where(k < M, 2.0, 1.0)
        assert oracle.tpf_general(a, g, c) == pytest.approx(oracle.tpf_isd(a), rel=1e-12)


def test_general_form_unit_cost_reduces_to_one_plus_survival_sum():
    # conventional speculative decoding: one guaranteed token, unit cost
    rng = np.random.default_rng(2)
    a = rng.uniform(0.2, 1.0, 12)
    k = np.arange(13)
    A = oracle.survival(a)
    assert oracle.tpf_general(a, k + 1.0, np.ones(13)) == pytest.approx(1.0 + A[1:].sum(), rel=1e-12)


def test_expected_prefix_length_identity_and_law_sums_to_one():
    rng = np.random.default_rng(3)
    a = rng.uniform(0.0, 1.0, 9)
    p = oracle.prefix_law(a)
    assert p.sum() == pytest.approx(1.0, abs=1e-14)
    assert np.all(p >= 0)
    assert np.dot(np.arange(10), p) == pytest.approx(oracle.survival(a)[1:].sum(), rel=1e-12)


def test_profile_recovers_rational_profile_exactly():
    # counts built from the prefix law of a rational profile reproduce it
    a_true = [Fraction(3, 4), Fraction(2, 3), Fraction(1, 2), Fraction(4, 5)]
    M = len(a_true)
    n = 2 ** 4 * 3 * 5 * 7
    counts = []
    A = Fraction(1)
    for k in range(M):
        counts.append(n * A * (1 - a_true[k]))
        A *= a_true[k]
    counts.append(n * A)
    assert all(c.denominator == 1 for c in counts)
    lens = np.repeat(np.arange(M + 1), [int(c) for c in counts])
    prof = oracle.accept_profile(lens, M)
    assert np.allclose(prof["a"], [float(x) for x in a_true], atol=1e-15)


def test_profile_brute_force_small():
    # every multiset of 3 blocks with M = 3, checked against direct counting
    M = 3
    for lens in itertools.product(range(M + 1), repeat=3):
        prof = oracle.accept_profile(lens, M)
        for i in range(1, M + 1):
            reach = sum(1 for L in lens if L + 1 >= i)
            rej = sum(1 for L in lens if L + 1 == i)
            assert prof["reach"][i - 1] == reach and prof["rej"][i - 1] == rej
            want = 1.0 if reach == 0 else 1.0 - rej / reach
            assert prof["a"][i - 1] == pytest.approx(want, abs=0)


def test_profile_clamps_out_of_range_lengths():
    prof = oracle.accept_profile([-3, 0, 7, 4], 4)
    ref = oracle.accept_profile([0, 0, 4, 4], 4)
    assert np.array_equal(prof["a"], ref["a"])


def _fpt_of_z(z):
    return oracle.fpt_isd(1.0 / (1.0 + np.exp(-z)))


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_weights_match_finite_differences_of_fpt(seed):
    rng = np.random.default_rng(seed)
    M = 7
    a = rng.uniform(0.05, 0.95, M)
    z = np.log(a / (1 - a))
    raw = oracle.risk_reward_weights(a)["raw"]
    h = 1e-6
    for i in range(M):
        zp, zm = z.copy(), z.copy()
        zp[i] += h
        zm[i] -= h
        fd = -(_fpt_of_z(zp) - _fpt_of_z(zm)) / (2 * h)
        assert raw[i] == pytest.approx(fd, rel=1e-6, abs=1e-12)


def test_weights_normalisation_and_sign():
    rng = np.random.default_rng(4)
    a = rng.uniform(0.3, 0.99, 15)
    rw = oracle.risk_reward_weights(a)
    assert np.all(rw["raw"] >= 0)
    assert rw["w"].mean() == pytest.approx(1.0, rel=1e-12)


def test_weights_emphasise_early_positions_for_a_uniform_profile():
    # Section 3.2: with a uniform unreliable profile the first positions
    # constrain block progress most
    rw = oracle.risk_reward_weights(np.full(7, 0.8))
    assert np.all(np.diff(rw["raw"]) < 0)


def test_weights_of_a_perfect_position_vanish():
    # a_i = 1 cannot be improved: its log-odds derivative is zero
    a = np.array([0.9, 1.0, 0.7])
    assert oracle.risk_reward_weights(a)["raw"][1] == 0.0
