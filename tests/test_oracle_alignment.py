"""Pins of the oracle's alignment objective (Section 3.5, Eqs. 9-11).

Independent references: torch's softmax / log_softmax / kl_div / norm in
float64, closed forms for two classes, worked values, and invariants
(identity, shift invariance, Gibbs' inequality, full retention).
"""
import math

import numpy as np
import torch

import synthetic as S
from oracle import adadsf_oracle as O


def _t(a):
    return torch.tensor(a, dtype=torch.float64)


def test_softmax_rows_matches_torch_and_is_stable():
    g = np.random.default_rng(0)
    h = g.normal(size=(5, 7, 33)) * 3
    np.testing.assert_allclose(O.softmax_rows(h), torch.softmax(_t(h), dim=-1).numpy(), rtol=1e-13, atol=1e-16)
    big = np.array([[1000.0, 999.0, -1000.0], [-1e4, -1e4 + 1, -1e4 + 2]])
    p = O.softmax_rows(big)
    assert np.all(np.isfinite(p))
    np.testing.assert_allclose(p.sum(-1), 1.0, rtol=1e-15)
    np.testing.assert_allclose(p, torch.softmax(_t(big), dim=-1).numpy(), rtol=1e-13)
    np.testing.assert_allclose(O.softmax_rows(h + g.normal(size=(5, 7, 1)) * 50), O.softmax_rows(h), rtol=1e-10)


def test_hidden_align_identity_shift_and_two_class_closed_form():
    g = np.random.default_rng(1)
    h = g.normal(size=(3, 9, 16))
    assert np.all(O.hidden_align_sq(h, h) == 0.0)
    # a per-token constant added to every feature does not change the softmax
    np.testing.assert_allclose(O.hidden_align_sq(h + g.normal(size=(3, 9, 1)) * 5, h), 0.0, atol=1e-28)
    # d = 2: Softmax([a1, a2]) = (sig(a1 - a2), sig(a2 - a1))
    a, b = g.normal(size=(20, 2)) * 2, g.normal(size=(20, 2)) * 2
    sig = lambda v: 1.0 / (1.0 + math.exp(-v))
    for i in range(20):
        p = sig(a[i, 0] - a[i, 1])
        q = sig(b[i, 0] - b[i, 1])
        assert abs(O.hidden_align_sq(a[i], b[i]) - 2 * (p - q) ** 2) < 1e-15
    # disjoint one-hot limits: distance 2
    assert abs(O.hidden_align_sq(np.array([200.0, 0, 0]), np.array([0, 200.0, 0])) - 2.0) < 1e-15


def test_hidden_align_loss_is_the_entrywise_norm():
    g = np.random.default_rng(2)
    hs, hd = g.normal(size=(2, 11, 24)), g.normal(size=(2, 11, 24))
    ref = torch.linalg.norm((torch.softmax(_t(hs), -1) - torch.softmax(_t(hd), -1)).reshape(-1)).item()
    assert abs(O.hidden_align_loss(hs, hd) - ref) < 1e-14 * max(1.0, ref)


def test_kl_align_matches_torch_and_worked_values():
    g = np.random.default_rng(3)
    ld, ls = g.normal(size=(6, 101)) * 2, g.normal(size=(6, 101)) * 2
    ref = torch.nn.functional.kl_div(torch.log_softmax(_t(ls), -1), torch.log_softmax(_t(ld), -1),
                                     reduction="none", log_target=True).sum(-1).numpy()
    np.testing.assert_allclose(O.kl_align(ld, ls), ref, rtol=1e-12, atol=1e-15)
    # P = (1/2, 1/2), Q = (3/4, 1/4): KL(P || Q) = ln(4/3) / 2, and the other direction differs
    v = O.kl_align(np.array([0.0, 0.0]), np.array([math.log(3.0), 0.0]))
    assert abs(v - 0.5 * math.log(4.0 / 3.0)) < 1e-15
    w = O.kl_align(np.array([math.log(3.0), 0.0]), np.array([0.0, 0.0]))
    assert abs(w - (0.75 * math.log(1.5) + 0.25 * math.log(0.5))) < 1e-15
    # two classes: p log(p/q) + (1-p) log((1-p)/(1-q)) with p, q logistic of the logit gaps
    for i in range(10):
        a, b = g.normal(size=2) * 3, g.normal(size=2) * 3
        p = 1.0 / (1.0 + math.exp(-(a[0] - a[1])))
        q = 1.0 / (1.0 + math.exp(-(b[0] - b[1])))
        cf = p * math.log(p / q) + (1 - p) * math.log((1 - p) / (1 - q))
        assert abs(O.kl_align(a, b) - cf) < 1e-13


def test_kl_align_invariants():
    g = np.random.default_rng(4)
    ld = g.normal(size=(50, 64)) * 4
    ls = g.normal(size=(50, 64)) * 4
    assert np.all(np.abs(O.kl_align(ld, ld)) < 1e-14)
    kl = O.kl_align(ld, ls)
    assert np.all(kl > 0)  # Gibbs' inequality, distinct distributions
    shifted = O.kl_align(ld + g.normal(size=(50, 1)) * 100, ls - g.normal(size=(50, 1)) * 100)
    np.testing.assert_allclose(shifted, kl, rtol=1e-9)
    big = O.kl_align(np.array([[1e3, 0.0, -1e3]]), np.array([[0.0, 1e3, 0.0]]))
    assert np.isfinite(big[0]) and abs(big[0] - 1e3) < 1e-9  # P one-hot on class 0, Q puts e^-1000 there


def test_total_objective():
    assert O.total_objective(0.5, [1.0, 2.0, 6.0]) == 0.5 + 3.0


def test_align_stack_full_and_zero_retention():
    w = S.WORKLOADS["tiny_qwen_f32"].replace(n_layers=2)
    desc = dict(block=w.block, n_heads=w.n_heads, n_kv_heads=w.n_kv_heads, head_dim=w.head_dim, d_ff=w.d_ff,
                rotary_dims=w.rotary_dims, rope_theta=w.rope_theta, norm_eps=w.norm_eps)
    Ws = S.stack_weights(w)
    x = S.hidden_states(w)
    T = w.seq
    # full retention: the student is the teacher, bit for bit
    sums, xs, xd = O.align_stack(desc, Ws, x, [T, T])
    assert np.all(sums == 0.0) and np.array_equal(xs, xd)
    # no retention: the student keeps its input, the teacher runs the dense stack
    sums0, xs0, xd0 = O.align_stack(desc, Ws, x, [0, 0])
    np.testing.assert_array_equal(xs0, O.f64(x))
    d1 = O.dense_layer(desc, Ws[0], x)
    assert abs(sums0[0] - O.hidden_align_sq(O.f64(x), d1).sum()) < 1e-15
    assert sums0[1] > 0
