"""Pins of the oracle's router-score pathway (Section 3.4, training side):
score-gated layer, the gradient of a loss with respect to the kept tokens'
scores, and the router MLP's backward.

Independent references: torch autograd in float64 (a separate implementation
of the chain rule) and central finite differences of the oracle's own
forward, which check the derivative rather than retype its formula.
"""
import numpy as np
import torch

import synthetic as S
from oracle import adadsf_oracle as O


def _router_case(seed, n=64, d=48, dr=16):
    g = np.random.default_rng(seed)
    x = g.normal(size=(n, d))
    w1 = g.normal(size=(dr, d)) * 0.3
    b1 = g.normal(size=dr) * 0.1
    w2 = g.normal(size=dr)
    ds = g.normal(size=n)
    return x, w1, b1, w2, ds


def test_router_backward_matches_autograd():
    for seed in range(3):
        x, w1, b1, w2, ds = _router_case(seed)
        tx, tw1, tb1, tw2 = (torch.tensor(a, dtype=torch.float64, requires_grad=True) for a in (x, w1, b1, w2))
        tb2 = torch.tensor(0.37, dtype=torch.float64, requires_grad=True)
        score = torch.relu(tx @ tw1.T + tb1) @ tw2 + tb2
        (score * torch.tensor(ds)).sum().backward()
        r = O.router_backward(x, w1, b1, w2, ds)
        np.testing.assert_allclose(r["dw1"], tw1.grad.numpy(), rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(r["db1"], tb1.grad.numpy(), rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(r["dw2"], tw2.grad.numpy(), rtol=1e-12, atol=1e-12)
        assert abs(r["db2"] - tb2.grad.item()) < 1e-12
        np.testing.assert_allclose(r["dx"], tx.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_router_backward_finite_differences():
    x, w1, b1, w2, ds = _router_case(7)
    r = O.router_backward(x, w1, b1, w2, ds)

    def loss(x_, w1_, b1_, w2_):
        return float(np.dot(ds, O.router_scores(x_[None], w1_, b1_, w2_, 0.0)[0]))

    z = x @ w1.T + b1
    eps = 1e-6
    g = np.random.default_rng(1)
    for _ in range(12):  # entries of W1 whose perturbation crosses no ReLU kink
        i, j = g.integers(w1.shape[0]), g.integers(w1.shape[1])
        if np.min(np.abs(z[:, i])) < 1e-3:
            continue
        wp, wm = w1.copy(), w1.copy()
        wp[i, j] += eps
        wm[i, j] -= eps
        fd = (loss(x, wp, b1, w2) - loss(x, wm, b1, w2)) / (2 * eps)
        assert abs(fd - r["dw1"][i, j]) < 1e-6 * max(1.0, abs(fd))
    for _ in range(12):  # input entries
        t, c = g.integers(x.shape[0]), g.integers(x.shape[1])
        if np.min(np.abs(z[t])) < 1e-3:
            continue
        xp, xm = x.copy(), x.copy()
        xp[t, c] += eps
        xm[t, c] -= eps
        fd = (loss(xp, w1, b1, w2) - loss(xm, w1, b1, w2)) / (2 * eps)
        assert abs(fd - r["dx"][t, c]) < 1e-6 * max(1.0, abs(fd))
    # bias gradients: the score is linear in b2 and in w2 given the hidden units
    assert abs(r["db2"] - ds.sum()) < 1e-12
    np.testing.assert_allclose(r["dw2"], np.maximum(z, 0).T @ ds, rtol=1e-12)


def test_gate_score_grad_finite_differences():
    g = np.random.default_rng(3)
    B, T, d, k = 2, 12, 8, 5
    x = g.normal(size=(B, T, d))
    delta = g.normal(size=(B, k, d))
    dy = g.normal(size=(B, T, d))
    scores = g.normal(size=(B, T)) * 2
    idx = np.stack([np.sort(g.permutation(T)[:k]) for _ in range(B)])

    def output(sc):
        gk = O.sigmoid(np.stack([sc[b, idx[b]] for b in range(B)]))
        return O.scatter_residual(x, gk[..., None] * delta, idx)

    y = output(scores)
    grad = O.gate_score_grad(dy, x, y, scores, idx)
    eps = 1e-6
    for b in range(B):
        for t in range(T):
            sp, sm = scores.copy(), scores.copy()
            sp[b, t] += eps
            sm[b, t] -= eps
            fd = (np.sum(dy * output(sp)) - np.sum(dy * output(sm))) / (2 * eps)
            assert abs(fd - grad[b, t]) < 1e-7 * max(1.0, abs(fd))
            if t not in idx[b]:
                assert grad[b, t] == 0.0


def test_gate_score_grad_matches_autograd():
    g = np.random.default_rng(4)
    B, T, d, k = 3, 10, 6, 4
    x = g.normal(size=(B, T, d))
    delta = g.normal(size=(B, k, d))
    dy = g.normal(size=(B, T, d))
    idx = np.stack([np.sort(g.permutation(T)[:k]) for _ in range(B)])
    ts = torch.tensor(g.normal(size=(B, T)), dtype=torch.float64, requires_grad=True)
    y = torch.tensor(x).clone()
    for b in range(B):
        p = torch.tensor(idx[b])
        y[b, p] = y[b, p] + torch.sigmoid(ts[b, p])[:, None] * torch.tensor(delta[b])
    (y * torch.tensor(dy)).sum().backward()
    grad = O.gate_score_grad(dy, x, y.detach().numpy(), ts.detach().numpy(), idx)
    np.testing.assert_allclose(grad, ts.grad.numpy(), rtol=1e-12, atol=1e-13)


def test_gated_layer_definition_and_limit():
    w = S.WORKLOADS["tiny_neox_f32"]
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w)
    desc = dict(block=w.block, n_heads=w.n_heads, n_kv_heads=w.n_kv_heads, head_dim=w.head_dim, d_ff=w.d_ff,
                rotary_dims=w.rotary_dims, rope_theta=w.rope_theta, norm_eps=w.norm_eps)
    k = 20
    res_g = O.routed_layer(desc, W, x, k, gate=True)
    res = O.routed_layer(desc, W, x, k, idx=res_g["idx"])
    np.testing.assert_array_equal(res["delta"], res_g["delta"])  # the gate does not change the block
    xs = O.f64(x)
    for b in range(x.shape[0]):
        p = res_g["idx"][b]
        g = O.sigmoid(res_g["scores"][b, p])
        np.testing.assert_allclose(res_g["y"][b, p] - xs[b, p], g[:, None] * res_g["delta"][b], rtol=1e-12,
                                   atol=1e-15)
        skipped = np.setdiff1d(np.arange(x.shape[1]), p)
        np.testing.assert_array_equal(res_g["y"][b, skipped], xs[b, skipped])
    # very large router bias: sigmoid -> 1, the gated layer becomes the plain one
    W2 = dict(W, router_b2=60.0)
    res_big = O.routed_layer(desc, W2, x, k, idx=res_g["idx"], gate=True)
    np.testing.assert_allclose(res_big["y"], res["y"], rtol=0, atol=1e-20)
