"""Pins of the oracle's incremental decoding (decode_stack, kept_set_stack).

The paper does not treat decoding; the reading (threshold routing of each new
token, per-layer kept sets) is stated in the oracle's header. These tests pin
it to properties that hold whatever the weights:

* causality: decoding token by token with the Top-K selections of the whole
  sequence forced reproduces the routed stack over the whole sequence
  (stack_forward, itself pinned against the transformers layers);
* thresholds of -inf keep every token: the dense stack;
* thresholds of +inf keep none: the input passes through;
* threshold routing keeps exactly the tokens whose own score reaches the
  threshold, and kept_set_stack over those decisions gives the same states;
* kept_set_layer over Top-K sets equals routed_layer.
"""
import numpy as np

import synthetic as S
from oracle import adadsf_oracle as O


def _desc(w):
    return dict(block=w.block, n_heads=w.n_heads, n_kv_heads=w.n_kv_heads, head_dim=w.head_dim, d_ff=w.d_ff,
                rotary_dims=w.rotary_dims, rope_theta=w.rope_theta, norm_eps=w.norm_eps)


def _setup(name, L=2, B=2, T=10, seed=0):
    w = S.WORKLOADS[name].replace(n_layers=L)
    Ws = S.stack_weights(w)
    x = S.hidden_states(w, seed_offset=seed, batch=B, seq=T)
    return w, _desc(w), Ws, x


def test_forced_topk_decode_equals_full_sequence_stack():
    for name in ("tiny_neox_f32", "tiny_qwen_f32"):
        w, desc, Ws, x = _setup(name, T=12)
        ks = [7, 4]
        y_full, idxs = O.stack_forward(desc, Ws, x, ks)
        B, T = x.shape[0], x.shape[1]
        force = np.zeros((len(Ws), B, T), dtype=bool)
        for l, idx in enumerate(idxs):
            for b in range(B):
                force[l, b, idx[b]] = True
        y_dec, keep, _ = O.decode_stack(desc, Ws, x, force=force)
        assert np.array_equal(keep, force)
        np.testing.assert_allclose(y_dec, y_full, rtol=0, atol=1e-12)


def test_thresholds_at_the_extremes():
    w, desc, Ws, x = _setup("tiny_neox_f32", T=6)
    L, B = len(Ws), x.shape[0]
    y_all, keep_all, _ = O.decode_stack(desc, Ws, x, thr=np.full((L, B), -np.inf))
    assert keep_all.all()
    dense = O.f64(x)
    for W in Ws:
        dense = O.dense_layer(desc, W, dense)
    np.testing.assert_allclose(y_all, dense, rtol=0, atol=1e-12)
    y_none, keep_none, _ = O.decode_stack(desc, Ws, x, thr=np.full((L, B), np.inf))
    assert not keep_none.any()
    np.testing.assert_array_equal(y_none, O.f64(x))


def test_threshold_routing_decisions_and_kept_sets():
    for name in ("tiny_neox_f32", "tiny_qwen_f32"):
        w, desc, Ws, x = _setup(name, T=9, seed=3)
        L, B, T = len(Ws), x.shape[0], x.shape[1]
        # thresholds from a first pass that keeps everything: the median score of each (layer, sequence)
        _, _, s_all = O.decode_stack(desc, Ws, x, thr=np.full((L, B), -np.inf))
        thr = np.median(s_all, axis=2)
        y, keep, scores = O.decode_stack(desc, Ws, x, thr=thr)
        np.testing.assert_array_equal(keep, scores >= thr[:, :, None])
        assert keep.any() and not keep.all()
        keeps = [[np.nonzero(keep[l, b])[0] for b in range(B)] for l in range(L)]
        np.testing.assert_allclose(O.kept_set_stack(desc, Ws, x, keeps), y, rtol=0, atol=1e-12)
        # a skipped token leaves that layer's state unchanged: its row only moves where it was kept
        never = ~keep.any(axis=0)
        np.testing.assert_array_equal(y[never], O.f64(x)[never])


def test_kept_set_layer_matches_routed_layer():
    w, desc, Ws, x = _setup("tiny_qwen_f32", L=1, T=11, seed=5)
    res = O.routed_layer(desc, Ws[0], x, 5)
    keeps = [list(res["idx"][b]) for b in range(x.shape[0])]
    np.testing.assert_allclose(O.kept_set_layer(desc, Ws[0], x, keeps), res["y"], rtol=0, atol=1e-13)
    # sets of different sizes per sequence, including an empty one
    y = O.kept_set_layer(desc, Ws[0], x, [[0, 3, 10], []])
    np.testing.assert_array_equal(y[1], O.f64(x)[1])
    d = O.block_delta(desc, Ws[0], O.f64(x)[0, [0, 3, 10]], np.array([0, 3, 10]))
    np.testing.assert_allclose(y[0, [0, 3, 10]], O.f64(x)[0, [0, 3, 10]] + d, rtol=0, atol=1e-13)
