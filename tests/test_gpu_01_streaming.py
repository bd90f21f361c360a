"""GPU parity of the streaming kernels against the oracle, through the C ABI:
similarity statistic (Eq. 4), router, Top-K, gather and scatter (Section 3.4).

Tolerances:
  * similarity: products and sums in fp64 on both sides, so only summation
    order differs: 1e-12 relative;
  * router: a rounding-error bound of fp32 accumulation (gpu_util.router_bound);
  * Top-K, gather, scatter: bit-exact (integer / copy work; the scatter add of
    two bf16 or fp32 values rounds once in both implementations).
"""
import numpy as np
import pytest
import torch

import paper_2607_21291_amd as P
import synthetic as S
from oracle import adadsf_oracle as O

from gpu_util import announce, router_bound, to_np

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("n,d", [(1, 8), (3, 64), (1001, 768), (4096, 896), (777, 3584)])
def test_sim_stats(dev, dtype, n, d):
    announce(f"sim_stats dtype={dtype} n={n} d={d}")
    g = torch.Generator().manual_seed(n + d)
    a = torch.randn(n, d, generator=g).to(dtype)
    c = (a.float() + 0.7 * torch.randn(n, d, generator=g)).to(dtype)
    if n > 2:
        a[1] = 0                      # zero row -> cosine 0
        c[2] = a[2]                   # identical row -> cosine 1
    da, dc = a.to(dev), c.to(dev)
    accum = torch.zeros(2, dtype=torch.float64, device=dev)
    per = torch.empty(n, dtype=torch.float32, device=dev)
    P.sim_stats(da, dc, accum, per_token_cos=per)
    P.sim_stats(da, dc, accum)                         # accumulates a second time
    torch.cuda.synchronize()
    ref = O.token_cosine(to_np(a), to_np(c))
    got = accum.cpu().numpy()
    assert got[1] == 2 * n
    assert abs(got[0] - 2 * ref.sum()) <= 1e-12 * max(1.0, np.abs(ref).sum() * 2)
    np.testing.assert_allclose(per.cpu().numpy(), ref, rtol=1e-6, atol=1e-7)  # stored as fp32
    if n > 2:
        assert per[1].item() == 0.0 and abs(per[2].item() - 1.0) < 1e-7
    s = P.sim_finalize(accum)
    assert abs(s[0] - ref.mean()) < 1e-12
    # deterministic: identical inputs give a bitwise-identical sum
    acc2 = torch.zeros(2, dtype=torch.float64, device=dev)
    P.sim_stats(da, dc, acc2)
    P.sim_stats(da, dc, acc2)
    assert torch.equal(acc2, accum)


@pytest.mark.parametrize("name", ["tiny_neox_f32", "neox160m", "qwen05b", "qwen7b"])
@pytest.mark.parametrize("dr", [32, 64])
def test_router_scores(dev, name, dr):
    w = S.WORKLOADS[name].replace(d_router=dr)
    announce(f"router {name} d_r={dr}")
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w, batch=2, seq=333)
    scores = torch.empty(2, 333, dtype=torch.float32, device=dev)
    P.router_score(x.to(dev), W["router_w1"].to(dev), W["router_b1"].to(dev), W["router_w2"].to(dev), 0.125,
                   scores)
    torch.cuda.synchronize()
    W["router_b2"] = 0.125
    ref = O.router_scores(x, W["router_w1"], W["router_b1"], W["router_w2"], 0.125)
    err = np.abs(scores.cpu().numpy() - ref)
    assert np.all(err <= router_bound(to_np(x), W, w.dtype)), err.max()


def _check_topk(dev, scores: torch.Tensor, k: int):
    B, T = scores.shape
    idx = torch.full((B, max(k, 1)), -7, dtype=torch.int32, device=dev)
    P.topk_select(scores.to(dev), k, idx[:, :k] if k > 0 else idx[:, :0].contiguous())
    torch.cuda.synchronize()
    ref = O.topk_select(scores.numpy(), k)
    np.testing.assert_array_equal(idx[:, :k].cpu().numpy(), ref)


@pytest.mark.parametrize("B,T", [(1, 1), (3, 64), (2, 1000), (8, 2048), (4, 8192), (1, 12345), (2, 20000)])
def test_topk_random(dev, B, T):
    sc = S.random_scores(B, T, seed=B * T)
    for k in sorted({0, 1, T // 3, T // 2, T - 1, T}):
        announce(f"topk random B={B} T={T} k={k}")
        if k == 0:
            continue
        _check_topk(dev, sc, k)


@pytest.mark.parametrize("levels", [1, 2, 3, 8])
def test_topk_ties(dev, levels):
    sc = S.router_scores_with_ties(4, 3000, levels, seed=levels)
    for k in (1, 17, 1499, 1500, 2999, 3000):
        announce(f"topk ties levels={levels} k={k}")
        _check_topk(dev, sc, k)


def test_topk_special_values(dev):
    announce("topk special values")
    row = torch.tensor([0.0, -0.0, 1.0, -float("inf"), float("nan"), float("inf"), -0.0, 0.0, -1e-38, 1e-38,
                        -3.0, float("nan"), 3.0, 1e30, -1e30, 0.0], dtype=torch.float32)
    sc = torch.stack([row, row.flip(0)])
    for k in range(17):
        if k:
            _check_topk(dev, sc, k)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("B,T,d,k", [(1, 1, 8, 1), (2, 64, 128, 32), (3, 1000, 768, 577), (2, 4096, 896, 2362)])
def test_gather_scatter_bit_exact(dev, dtype, B, T, d, k):
    announce(f"gather/scatter dtype={dtype} B={B} T={T} d={d} k={k}")
    g = torch.Generator().manual_seed(T + k)
    x = torch.randn(B, T, d, generator=g).to(dtype)
    delta = torch.randn(B, k, d, generator=g).to(dtype)
    idx = torch.stack([torch.sort(torch.randperm(T, generator=g)[:k])[0] for _ in range(B)]).to(torch.int32)
    dx, di = x.to(dev), idx.to(dev)
    out = torch.empty(B, k, d, dtype=dtype, device=dev)
    P.gather_rows(dx, di, out)
    P.scatter_residual(dx, delta.to(dev), di)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(to_np(out), O.gather_rows(to_np(x), idx.numpy()))
    kind = "bf16" if dtype == torch.bfloat16 else "f32"
    np.testing.assert_array_equal(to_np(dx), O.scatter_residual(to_np(x), to_np(delta), idx.numpy(), kind))
