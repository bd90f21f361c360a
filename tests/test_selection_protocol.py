"""The selection check of the GPU parity protocol (tests/gpu_util.py), run on
the CPU with planted score vectors: identical selections pass, a swap of two
near-tied tokens passes, and a swap that the score tolerance cannot explain
fails."""
import numpy as np
import pytest

from gpu_util import check_selection
from oracle import adadsf_oracle as O


def _case(seed=0, B=3, T=50, k=20):
    rng = np.random.default_rng(seed)
    ref = rng.standard_normal((B, T))
    bound = np.full((B, T), 1e-6)
    return ref, bound, k


def test_identical_scores_pass():
    ref, bound, k = _case()
    check_selection(ref, bound, ref.astype(np.float32).astype(np.float64), O.topk_select(ref, k), k)


def test_near_tie_swap_passes():
    ref, bound, k = _case(1)
    gpu = ref.copy()
    b = 1
    order = np.argsort(-ref[b], kind="stable")
    kth, nxt = order[k - 1], order[k]
    ref[b, nxt] = ref[b, kth] - 0.5e-6      # the oracle's (k+1)-th sits within the tolerance of its k-th
    gpu[b] = ref[b]
    gpu[b, nxt] = ref[b, kth] + 0.25e-6     # the GPU's rounding lifts it over the k-th
    gpu[b, kth] = ref[b, kth] - 0.5e-6
    idx = O.topk_select(gpu, k)
    assert not np.array_equal(idx, O.topk_select(ref, k))
    check_selection(ref, bound, gpu, idx, k)


def test_far_swap_fails():
    ref, bound, k = _case(2)
    gpu = ref.copy()
    b = 0
    order = np.argsort(-ref[b], kind="stable")
    worst = order[-1]
    gpu[b, worst] = ref[b, order[0]] + 1.0   # a GPU score far outside its bound
    with pytest.raises(AssertionError):
        check_selection(ref, bound, gpu, O.topk_select(gpu, k), k)
    # scores within bound but indices not the Top-K of the GPU's scores
    idx = O.topk_select(ref, k).copy()
    idx[b, 0] = worst
    idx[b].sort()
    with pytest.raises(AssertionError):
        check_selection(ref, bound, ref.copy(), idx, k)


def test_storage_half_ulp_bounds_rounding():
    """half_ulp is the largest error of rounding to bf16 / fp32 (torch's
    round-to-nearest-even): never exceeded, and reached at a tie."""
    import torch

    from gpu_util import storage_half_ulp, update_err
    rng = np.random.default_rng(3)
    v = rng.standard_normal(20000) * 10.0 ** rng.uniform(-3, 3, 20000)
    for dtype, tdt in (("bf16", torch.bfloat16), ("f32", torch.float32)):
        r = torch.from_numpy(v).to(tdt).double().numpy()
        assert np.all(np.abs(r - v) <= storage_half_ulp(r, dtype))
    tie = np.array([1.0 + 2.0 ** -8])   # halfway between two bf16 values (1 and 1 + 2^-7)
    r = torch.from_numpy(tie).to(torch.bfloat16).double().numpy()
    assert np.abs(r - tie)[0] == storage_half_ulp(r, "bf16")[0] == 2.0 ** -8
    # an update seen through a rounded output: exact update -> 0 excess
    x = np.array([10.0, -12.0])
    d = np.array([0.3, -0.01])
    y = torch.from_numpy(x + d).to(torch.bfloat16).double().numpy()
    assert update_err(y, x, d, "bf16") == 0.0
    assert update_err(y, x, d * 1.5, "bf16") > 0.0
