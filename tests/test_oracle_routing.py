"""Pins for the oracle's router, Top-K selection, gather/scatter and bf16 rounding (Section 3.4)."""
import numpy as np
import pytest
import torch

import synthetic as S
from oracle import adadsf_oracle as O


def test_router_matches_torch_mlp():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((2, 33, 48))
    w1, b1, w2 = rng.standard_normal((16, 48)), rng.standard_normal(16), rng.standard_normal(16)
    mlp = torch.nn.Sequential(torch.nn.Linear(48, 16), torch.nn.ReLU(), torch.nn.Linear(16, 1)).double()
    with torch.no_grad():
        mlp[0].weight.copy_(torch.from_numpy(w1)); mlp[0].bias.copy_(torch.from_numpy(b1))
        mlp[2].weight.copy_(torch.from_numpy(w2)[None]); mlp[2].bias.fill_(0.75)
        ref = mlp(torch.from_numpy(x))[..., 0].numpy()
    np.testing.assert_allclose(O.router_scores(x, w1, b1, w2, 0.75), ref, rtol=1e-13, atol=1e-13)


def _check_topk(scores, k, idx):
    """Properties that define the selection uniquely."""
    B, T = scores.shape
    assert idx.shape == (B, k)
    for b in range(B):
        row = idx[b]
        assert np.all(np.diff(row) > 0)                  # unique, strictly ascending
        assert row.size == 0 or (row[0] >= 0 and row[-1] < T)
        kept = np.zeros(T, dtype=bool)
        kept[row] = True
        if 0 < k < T:
            lo = scores[b][kept].min()
            hi = scores[b][~kept].max()
            assert lo >= hi                              # every kept score >= every skipped score
            # at the threshold, the lowest positions win
            tie = np.flatnonzero(scores[b] == lo)
            n_above = np.count_nonzero(scores[b] > lo)
            np.testing.assert_array_equal(np.flatnonzero(kept & (scores[b] == lo)), tie[:k - n_above])


@pytest.mark.parametrize("T,k", [(1, 0), (1, 1), (7, 3), (64, 32), (100, 1), (257, 200), (2048, 1563)])
def test_topk_random(T, k):
    sc = S.random_scores(3, T, seed=T + k).numpy()
    _check_topk(sc, k, O.topk_select(sc, k))


@pytest.mark.parametrize("levels", [1, 2, 4, 8])
def test_topk_tie_heavy(levels):
    sc = S.router_scores_with_ties(4, 300, levels, seed=levels).numpy()
    for k in (0, 1, 37, 150, 299, 300):
        _check_topk(sc, k, O.topk_select(sc, k))


def test_topk_extremes_and_signed_zero():
    sc = np.array([[0.0, -0.0, 1.0, -np.inf, np.nan, np.inf, -0.0, 0.0]])
    assert O.topk_select(sc, 8).tolist() == [list(range(8))]
    assert O.topk_select(sc, 0).shape == (1, 0)
    # +inf, 1, then the four zeros by position, then -inf, then NaN last
    assert O.topk_select(sc, 3).tolist() == [[0, 2, 5]]
    assert O.topk_select(sc, 5).tolist() == [[0, 1, 2, 5, 6]]
    assert O.topk_select(sc, 7).tolist() == [[0, 1, 2, 3, 5, 6, 7]]


def test_topk_brute_force_small():
    # For tiny T, enumerate all k-subsets; the selection is the subset whose
    # scores sorted descending are lexicographically largest, ties -> smallest positions.
    import itertools
    rng = np.random.default_rng(3)
    for _ in range(200):
        T = int(rng.integers(1, 8))
        k = int(rng.integers(0, T + 1))
        sc = rng.integers(0, 3, (1, T)).astype(float)
        best = max(itertools.combinations(range(T), k),
                   key=lambda c: (sorted((sc[0, i] for i in c), reverse=True), [-i for i in c]))
        assert O.topk_select(sc, k)[0].tolist() == list(best)


def test_gather_equals_masked_selection():
    x = np.random.default_rng(1).standard_normal((2, 10, 4))
    idx = np.array([[1, 4, 9], [0, 2, 3]])
    m = np.zeros((2, 10), dtype=bool)
    for b in range(2):
        m[b, idx[b]] = True
    got = O.gather_rows(x, idx)
    for b in range(2):
        np.testing.assert_array_equal(got[b], x[b][m[b]])


def test_scatter_bypass_and_rounding():
    x = S.hidden_states(S.WORKLOADS["neox160m"], batch=2, seq=40).float().numpy()[..., :16]
    x = O.round_bf16(x)
    idx = np.array([[0, 5, 39], [3, 4, 20]])
    delta = O.round_bf16(np.random.default_rng(2).standard_normal((2, 3, 16)))
    y = O.scatter_residual(x, delta, idx, "bf16")
    kept = np.zeros((2, 40), dtype=bool)
    for b in range(2):
        kept[b, idx[b]] = True
        np.testing.assert_array_equal(y[b][~kept[b]], x[b][~kept[b]])     # bypass untouched
    # The kept rows: one rounding of the exact sum, checked against torch's fp32->bf16.
    exact = np.stack([x[b, idx[b]] + delta[b] for b in range(2)])
    ref = torch.from_numpy(exact.astype(np.float32)).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(np.stack([y[b, idx[b]] for b in range(2)]), ref)
    # k = 0 is the identity
    np.testing.assert_array_equal(O.scatter_residual(x, np.zeros((2, 0, 16)), np.zeros((2, 0), int), "bf16"), x)


def test_round_bf16_matches_torch_on_fp32_values():
    rng = np.random.default_rng(11)
    v = (rng.standard_normal(20000) * np.exp(rng.uniform(-20, 20, 20000))).astype(np.float32)
    # exact midpoints between neighbouring bf16 values exercise ties-to-even
    base = torch.from_numpy(v).to(torch.bfloat16).float().numpy()
    mids = (base.astype(np.float64) * (1 + 2.0 ** -9)).astype(np.float32)
    for arr in (v, mids):
        ref = torch.from_numpy(arr).to(torch.bfloat16).double().numpy()
        np.testing.assert_array_equal(O.round_bf16(arr.astype(np.float64)), ref)
    assert O.round_bf16(np.array([0.0]))[0] == 0.0
