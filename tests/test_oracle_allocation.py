"""Pins for the oracle's similarity statistic (Eq. 4) and retention allocation (Eqs. 5-8, K_i)."""
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import adadsf_oracle as O


# --------------------------------------------------------------------------- Eq. 4

def _rows(seed, n, d):
    return np.random.default_rng(seed).standard_normal((n, d))


def test_cosine_identity_layer_is_one():
    a = _rows(0, 50, 96)
    np.testing.assert_allclose(O.token_cosine(a, a), 1.0, rtol=0, atol=1e-15)
    tot, n = O.similarity_accumulate(a, a)
    assert n == 50 and abs(O.layer_similarity(tot, n) - 1.0) < 1e-15


@pytest.mark.parametrize("alpha", [3.5, -0.25])
def test_cosine_of_scaled_rows_is_sign(alpha):
    a = _rows(1, 20, 64)
    np.testing.assert_allclose(O.token_cosine(a, alpha * a), math.copysign(1.0, alpha), atol=1e-15)


def test_cosine_orthogonal_rows_are_zero():
    q, _ = np.linalg.qr(_rows(2, 64, 64))          # orthonormal columns
    a, c = q[:, 0:10].T, q[:, 10:20].T              # row i of a is orthogonal to row i of c
    np.testing.assert_allclose(O.token_cosine(a, c), 0.0, atol=1e-14)


def test_cosine_zero_row_is_zero_and_bounded():
    a = _rows(3, 30, 32)
    c = _rows(4, 30, 32)
    a[5] = 0.0
    cos = O.token_cosine(a, c)
    assert cos[5] == 0.0
    assert np.all(np.abs(cos) <= 1.0)


def test_cosine_matches_torch_library_routine():
    a = _rows(5, 40, 128)
    c = a + 0.3 * _rows(6, 40, 128)
    ref = torch.nn.functional.cosine_similarity(torch.from_numpy(a), torch.from_numpy(c), dim=-1)
    np.testing.assert_allclose(O.token_cosine(a, c), ref.numpy(), rtol=1e-14, atol=0)


def test_cosine_is_per_token_mean_not_flattened():
    # Two tokens with very different norms: the per-token mean weighs them equally.
    a = np.array([[1.0, 0.0], [100.0, 0.0]])
    c = np.array([[1.0, 0.0], [0.0, 100.0]])
    tot, n = O.similarity_accumulate(a, c)
    assert O.layer_similarity(tot, n) == pytest.approx(0.5, abs=1e-15)


# --------------------------------------------------------------------------- Eqs. 5-8

@pytest.mark.parametrize("tau", [0.25, 0.1, 0.05])
def test_uniform_similarity_gives_target(tau):
    r = O.retention_from_similarity([0.7] * 9, 0.6, tau)
    np.testing.assert_allclose(r, 0.6, rtol=0, atol=1e-15)


@pytest.mark.parametrize("seed", range(5))
@pytest.mark.parametrize("tau", [1.0, 0.25, 0.1, 0.05])
def test_budget_and_monotonicity(seed, tau):
    rng = np.random.default_rng(seed)
    L = int(rng.integers(2, 30))
    s = rng.uniform(0.2, 0.99, L)
    t = float(rng.uniform(0.2, 0.7))
    r = O.retention_from_similarity(s, t, tau, clip="none")
    assert abs(r.sum() - t * L) < 1e-12                 # constraint of Eq. 8
    order = np.argsort(s)
    assert np.all(np.diff(r[order]) <= 1e-15)            # more similar layer -> fewer tokens
    # r_i / r_j = r'_i / r'_j with r' in (0.05, 0.95)
    assert r.max() / r.min() < 0.95 / 0.05


def test_two_layer_closed_form():
    # For L = 2 the weights reduce to a logistic of the similarity gap:
    # w_1 = 1 / (1 + exp((s_2 - s_1) / tau)), z_2 = -z_1, and r'_1 + r'_2 = 1.
    s1, s2, tau, t, beta = 0.0, 1.0, 1.0, 0.5, 10.0
    w1 = 1.0 / (1.0 + math.exp((s2 - s1) / tau))
    z1 = beta * (0.5 - w1)
    rp1 = 0.05 + 0.9 / (1.0 + math.exp(-z1))
    expect = [2 * t * rp1, 2 * t * (1.0 - rp1)]
    r = O.retention_from_similarity([s1, s2], t, tau)
    np.testing.assert_allclose(r, expect, rtol=1e-14)
    np.testing.assert_allclose(r, [0.868775, 0.131225], atol=5e-7)


def test_shift_invariance_and_large_temperature():
    s = np.array([0.2, 0.4, 0.9, 0.55])
    np.testing.assert_allclose(O.retention_from_similarity(s + 0.3, 0.5, 0.1),
                               O.retention_from_similarity(s, 0.5, 0.1), rtol=1e-13)
    np.testing.assert_allclose(O.retention_from_similarity(s, 0.5, 1e9), 0.5, atol=1e-8)


def test_single_layer_and_no_temperature():
    assert O.retention_from_similarity([0.8], 0.7, 0.05)[0] == pytest.approx(0.7, abs=1e-15)
    np.testing.assert_array_equal(O.retention_from_similarity([0.1, 0.9, 0.5], 0.8, None), 0.8)


def test_budget_clip_worked_case():
    # Three very similar layers and nine dissimilar ones at t = 0.9: Eq. 8 alone
    # gives r > 1 for the nine. The budget clip caps them at 1 and gives the
    # remaining 10.8 - 9 = 1.8 to the three equal layers: 0.6 each.
    s = [0.9] * 3 + [0.3] * 9
    raw = O.retention_from_similarity(s, 0.9, 0.05, clip="none")
    assert raw[3:].min() > 1.0
    r = O.retention_from_similarity(s, 0.9, 0.05, clip="budget")
    np.testing.assert_allclose(r, [0.6] * 3 + [1.0] * 9, rtol=1e-13)
    assert abs(r.sum() - 0.9 * 12) < 1e-12
    np.testing.assert_array_equal(O.retention_from_similarity(s, 0.9, 0.05, clip="plain"),
                                  np.minimum(raw, 1.0))


def test_workload_profiles():
    # neox160m: similarities linspace(0.3, 0.9, 12), t = 0.6, tau = 0.25.
    r = O.retention_from_similarity(np.linspace(0.3, 0.9, 12), 0.6, 0.25)
    assert 0.29 < r.min() and r.max() < 0.77 and abs(r.mean() - 0.6) < 1e-12
    ks = [O.k_from_retention(x, 2048) for x in r]
    assert ks[0] == 1563 and ks[-1] == 600 and sum(ks) == 14741


# --------------------------------------------------------------------------- K_i = floor(r_i s)

def test_k_edges():
    assert O.k_from_retention(1.0, 2048) == 2048
    assert O.k_from_retention(0.0, 2048) == 0
    assert O.k_from_retention(0.5, 64) == 32
    assert O.k_from_retention(0.5, 64, "ceil") == 32
    assert O.k_from_retention(0.29, 100) == 29          # fp64 gives 28.999999999999996
    assert O.k_from_retention(0.57, 100) == 57
    assert O.k_from_retention(0.291, 100) == 29
    assert O.k_from_retention(0.291, 100, "ceil") == 30
    assert O.k_from_retention(1.2, 10) == 10             # clamped


def test_k_matches_exact_rational_floor():
    rng = np.random.default_rng(7)
    for _ in range(3000):
        milli = int(rng.integers(0, 1001))
        T = int(rng.integers(1, 8193))
        exact = Fraction(milli, 1000) * T
        r = float(Fraction(milli, 1000))
        assert O.k_from_retention(r, T) == math.floor(exact)
        assert O.k_from_retention(r, T, "ceil") == math.ceil(exact)
