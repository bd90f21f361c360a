"""Pins of the oracle's routed-layer backward (training side of Section 3.4).

1. torch autograd in float64 on an independently written layer: library
   layer norm, RoPE as multiplication of the (i, i + R/2) pairs by e^{i angle}
   as complex numbers, scaled_dot_product_attention (causal) with the kv
   heads repeated for GQA, library GELU / SiLU. Gradients of
   L = sum(y * dy) with respect to x and every weight must equal the
   oracle's (both block families, gated and plain, with skipped rows).
2. Central finite differences of the oracle's own forward (routed_layer,
   teacher-forced selection) for sampled weight and input coordinates.
3. block_forward_cache reproduces block_delta exactly.
"""
import math

import numpy as np
import pytest
import torch

from oracle import adadsf_oracle as O

NEOX = dict(block=O.NEOX, n_heads=4, n_kv_heads=4, head_dim=8, d_ff=48, rotary_dims=4, rope_theta=10000.0,
            norm_eps=1e-5)
QWEN = dict(block=O.QWEN, n_heads=4, n_kv_heads=2, head_dim=8, d_ff=40, rotary_dims=8, rope_theta=1e6,
            norm_eps=1e-6)
D = 32


def weights(desc, seed):
    rng = np.random.default_rng(seed)
    Hq, Hkv, hd, f = desc["n_heads"], desc["n_kv_heads"], desc["head_dim"], desc["d_ff"]
    neox = desc["block"] == O.NEOX
    n = lambda *s: rng.standard_normal(s) * 0.2
    W = {"norm1_w": 1 + n(D), "norm1_b": n(D) if neox else None, "norm2_w": 1 + n(D),
         "norm2_b": n(D) if neox else None, "w_qkv": n((Hq + 2 * Hkv) * hd, D), "b_qkv": n((Hq + 2 * Hkv) * hd),
         "w_o": n(D, Hq * hd), "b_o": n(D) if neox else None, "w_up": n(f if neox else 2 * f, D),
         "b_up": n(f) if neox else None, "w_down": n(D, f), "b_down": n(D) if neox else None,
         "router_w1": n(8, D), "router_b1": n(8), "router_w2": n(8), "router_b2": 0.0}
    return W


def torch_layer(desc, W, x, idx, gate):
    """The routed layer written independently in torch (float64)."""
    Hq, Hkv, hd, f = desc["n_heads"], desc["n_kv_heads"], desc["head_dim"], desc["d_ff"]
    R, th, eps = desc["rotary_dims"], desc["rope_theta"], desc["norm_eps"]
    neox = desc["block"] == O.NEOX
    F = torch.nn.functional
    B = x.shape[0]

    def rms(v, w):
        return v * torch.rsqrt((v * v).mean(-1, keepdim=True) + eps) * w

    def rot(t, pos):  # t [n, H, hd]
        half = R // 2
        ang = pos[:, None].double() * th ** (-(2.0 * torch.arange(half, dtype=torch.float64)) / R)
        z = torch.complex(t[..., :half], t[..., half:R]) * torch.polar(torch.ones_like(ang), ang)[:, None, :]
        return torch.cat([z.real, z.imag, t[..., R:]], dim=-1)

    h1 = torch.relu(x @ W["router_w1"].T + W["router_b1"])
    scores = h1 @ W["router_w2"]
    rows = []
    for b in range(B):
        p = torch.as_tensor(idx[b])
        xc = x[b, p]
        n = xc.shape[0]
        a = F.layer_norm(xc, (D,), W["norm1_w"], W["norm1_b"], eps) if neox else rms(xc, W["norm1_w"])
        qkv = a @ W["w_qkv"].T + W["b_qkv"]
        q = rot(qkv[:, :Hq * hd].reshape(n, Hq, hd), p)
        k = rot(qkv[:, Hq * hd:(Hq + Hkv) * hd].reshape(n, Hkv, hd), p)
        v = qkv[:, (Hq + Hkv) * hd:].reshape(n, Hkv, hd)
        rep = Hq // Hkv
        k = k.repeat_interleave(rep, dim=1)
        v = v.repeat_interleave(rep, dim=1)
        att = F.scaled_dot_product_attention(q.transpose(0, 1), k.transpose(0, 1), v.transpose(0, 1),
                                             is_causal=True).transpose(0, 1).reshape(n, Hq * hd)
        ao = att @ W["w_o"].T + (W["b_o"] if neox else 0.0)
        if neox:
            m = F.layer_norm(xc, (D,), W["norm2_w"], W["norm2_b"], eps)
            mo = F.gelu(m @ W["w_up"].T + W["b_up"]) @ W["w_down"].T + W["b_down"]
        else:
            m = rms(xc + ao, W["norm2_w"])
            gu = m @ W["w_up"].T
            mo = (F.silu(gu[:, :f]) * gu[:, f:]) @ W["w_down"].T
        g = torch.sigmoid(scores[b, p])[:, None] if gate else 1.0
        rows.append((b, p, xc + g * (ao + mo)))
    y = x.clone()
    for b, p, r in rows:
        y[b, p] = r
    return y


@pytest.mark.parametrize("gate", [False, True])
@pytest.mark.parametrize("desc", [NEOX, QWEN], ids=["neox", "qwen"])
def test_backward_matches_torch_autograd(desc, gate):
    W = weights(desc, 7 if gate else 3)
    rng = np.random.default_rng(11)
    B, T, k = 2, 9, 5
    x = rng.standard_normal((B, T, D))
    dy = rng.standard_normal((B, T, D))
    idx = np.stack([np.sort(rng.choice(T, k, replace=False)) for _ in range(B)])
    ref = O.routed_layer_backward(desc, W, x, dy, idx, gate=gate)
    dx = ref["dx"]
    router = ["router_w1", "router_b1", "router_w2"]
    if gate:
        # the router's share: the score gradient through the gate, then the router MLP's backward
        fwd = O.routed_layer(desc, W, x, k, idx=idx, gate=True)
        dscore = O.gate_score_grad(dy, x, fwd["y"], fwd["scores"], idx)
        rb = O.router_backward(x, W["router_w1"], W["router_b1"], W["router_w2"], dscore)
        dx = dx + rb["dx"]
    Wt = {key: (torch.tensor(v, requires_grad=key in O.GRAD_NAMES or key in router)
                if isinstance(v, np.ndarray) else v) for key, v in W.items()}
    xt = torch.tensor(x, requires_grad=True)
    y = torch_layer(desc, Wt, xt, idx, gate)
    (y * torch.tensor(dy)).sum().backward()
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-9, atol=1e-11)
    if gate:
        for name, key in (("router_w1", "dw1"), ("router_b1", "db1"), ("router_w2", "dw2")):
            np.testing.assert_allclose(rb[key], Wt[name].grad.numpy(), rtol=1e-9, atol=1e-11, err_msg=name)
    for name in O.GRAD_NAMES:
        if W[name] is None:
            assert ref["grads"][name] is None
            continue
        np.testing.assert_allclose(ref["grads"][name], Wt[name].grad.numpy(), rtol=1e-9, atol=1e-11,
                                   err_msg=name)
    # the forward of the independent layer agrees with the oracle's forward too
    np.testing.assert_allclose(y.detach().numpy(), O.routed_layer(desc, W, x, k, idx=idx, gate=gate)["y"],
                               rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("desc", [NEOX, QWEN], ids=["neox", "qwen"])
def test_backward_matches_finite_differences(desc):
    W = weights(desc, 5)
    rng = np.random.default_rng(4)
    B, T, k = 2, 8, 6
    x = rng.standard_normal((B, T, D))
    dy = rng.standard_normal((B, T, D))
    idx = np.stack([np.sort(rng.choice(T, k, replace=False)) for _ in range(B)])
    ref = O.routed_layer_backward(desc, W, x, dy, idx)

    def loss(Wv, xv):
        return float(np.sum(O.routed_layer(desc, Wv, xv, k, idx=idx)["y"] * dy))

    h = 1e-6
    for name in ["w_qkv", "w_o", "w_up", "w_down", "norm1_w", "norm2_w", "b_qkv"]:
        for _ in range(3):
            at = tuple(int(rng.integers(s)) for s in W[name].shape)
            Wp = {kk: (v.copy() if isinstance(v, np.ndarray) else v) for kk, v in W.items()}
            Wm = {kk: (v.copy() if isinstance(v, np.ndarray) else v) for kk, v in W.items()}
            Wp[name][at] += h
            Wm[name][at] -= h
            num = (loss(Wp, x) - loss(Wm, x)) / (2 * h)
            assert abs(num - ref["grads"][name][at]) <= 1e-6 * max(1.0, abs(num)), (name, at)
    for _ in range(6):
        b, t, c = int(rng.integers(B)), int(rng.integers(T)), int(rng.integers(D))
        xp, xm = x.copy(), x.copy()
        xp[b, t, c] += h
        xm[b, t, c] -= h
        num = (loss(W, xp) - loss(W, xm)) / (2 * h)
        assert abs(num - ref["dx"][b, t, c]) <= 1e-6 * max(1.0, abs(num))


@pytest.mark.parametrize("desc", [NEOX, QWEN], ids=["neox", "qwen"])
def test_forward_cache_reproduces_block_delta(desc):
    W = weights(desc, 9)
    rng = np.random.default_rng(2)
    xc = rng.standard_normal((6, D))
    pos = np.array([0, 2, 3, 7, 8, 12])
    delta, _ = O.block_forward_cache(desc, W, xc, pos)
    np.testing.assert_array_equal(delta, O.block_delta(desc, W, xc, pos))
