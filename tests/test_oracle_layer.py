"""Pins for the oracle's decoder block, routed layer and stack (Eqs. 1-2, Section 3.4).

The dense block is cross-checked against the transformers library's own
GPT-NeoX and Qwen2 decoder layers in float64, with our weights loaded into
them. The routed layer is checked through the equivalence it must satisfy:
the kept rows equal the library layer applied to the kept subsequence at the
original positions, and the skipped rows are unchanged.
"""
import math
import warnings

import numpy as np
import pytest
import torch

import synthetic as S
from oracle import adadsf_oracle as O

warnings.filterwarnings("ignore")


def desc_of(w: S.Workload):
    return dict(block=w.block, n_heads=w.n_heads, n_kv_heads=w.n_kv_heads, head_dim=w.head_dim,
                d_ff=w.d_ff, rotary_dims=w.rotary_dims, rope_theta=w.rope_theta, norm_eps=w.norm_eps)


def t64(a):
    return a.detach().to(torch.float64)


def hf_layer(w: S.Workload, W):
    """A transformers decoder layer of the workload's family holding weights W (float64)."""
    from transformers import GPTNeoXConfig, Qwen2Config
    from transformers.models.gpt_neox.modeling_gpt_neox import GPTNeoXLayer
    from transformers.models.qwen2.modeling_qwen2 import Qwen2DecoderLayer
    d, H, Hkv, hd = w.d_model, w.n_heads, w.n_kv_heads, w.head_dim
    if w.block == S.NEOX:
        cfg = GPTNeoXConfig(hidden_size=d, num_attention_heads=H, intermediate_size=w.d_ff,
                            use_parallel_residual=True, hidden_act="gelu", layer_norm_eps=w.norm_eps,
                            attention_bias=True)
        cfg._attn_implementation = "eager"
        L = GPTNeoXLayer(cfg, 0).double().eval()
        # our Q|K|V block order -> the library's per-head [q | k | v] interleave
        perm = [which * H * hd + h * hd + j for h in range(H) for which in range(3) for j in range(hd)]
        with torch.no_grad():
            L.input_layernorm.weight.copy_(t64(W["norm1_w"])); L.input_layernorm.bias.copy_(t64(W["norm1_b"]))
            L.post_attention_layernorm.weight.copy_(t64(W["norm2_w"]))
            L.post_attention_layernorm.bias.copy_(t64(W["norm2_b"]))
            L.attention.query_key_value.weight.copy_(t64(W["w_qkv"])[perm])
            L.attention.query_key_value.bias.copy_(t64(W["b_qkv"])[perm])
            L.attention.dense.weight.copy_(t64(W["w_o"])); L.attention.dense.bias.copy_(t64(W["b_o"]))
            L.mlp.dense_h_to_4h.weight.copy_(t64(W["w_up"])); L.mlp.dense_h_to_4h.bias.copy_(t64(W["b_up"]))
            L.mlp.dense_4h_to_h.weight.copy_(t64(W["w_down"])); L.mlp.dense_4h_to_h.bias.copy_(t64(W["b_down"]))
        return L
    cfg = Qwen2Config(hidden_size=d, num_attention_heads=H, num_key_value_heads=Hkv,
                      intermediate_size=w.d_ff, rms_norm_eps=w.norm_eps, hidden_act="silu")
    cfg._attn_implementation = "eager"
    L = Qwen2DecoderLayer(cfg, 0).double().eval()
    wq = t64(W["w_qkv"]); bq = t64(W["b_qkv"])
    a, b = H * hd, (H + Hkv) * hd
    with torch.no_grad():
        L.input_layernorm.weight.copy_(t64(W["norm1_w"]))
        L.post_attention_layernorm.weight.copy_(t64(W["norm2_w"]))
        L.self_attn.q_proj.weight.copy_(wq[:a]); L.self_attn.q_proj.bias.copy_(bq[:a])
        L.self_attn.k_proj.weight.copy_(wq[a:b]); L.self_attn.k_proj.bias.copy_(bq[a:b])
        L.self_attn.v_proj.weight.copy_(wq[b:]); L.self_attn.v_proj.bias.copy_(bq[b:])
        L.self_attn.o_proj.weight.copy_(t64(W["w_o"]))
        f = w.d_ff
        L.mlp.gate_proj.weight.copy_(t64(W["w_up"])[:f]); L.mlp.up_proj.weight.copy_(t64(W["w_up"])[f:])
        L.mlp.down_proj.weight.copy_(t64(W["w_down"]))
    return L


def hf_forward(w: S.Workload, layer, x: np.ndarray, pos: np.ndarray) -> np.ndarray:
    """Run the library layer on rows x [n, d] at positions pos, causal among those rows."""
    n = x.shape[0]
    R = w.rotary_dims
    inv_freq = 1.0 / (w.rope_theta ** (torch.arange(0, R, 2, dtype=torch.float64) / R))
    freqs = torch.from_numpy(pos.astype(np.float64))[:, None] * inv_freq[None, :]
    emb = torch.cat((freqs, freqs), dim=-1)[None]
    mask = torch.full((n, n), float("-inf"), dtype=torch.float64).triu(1)[None, None]
    with torch.no_grad():
        out = layer(torch.from_numpy(x)[None], attention_mask=mask,
                    position_ids=torch.from_numpy(pos)[None],
                    position_embeddings=(emb.cos(), emb.sin()))
    if isinstance(out, tuple):
        out = out[0]
    return out[0].numpy()


# The library layers take a few steps in fp32 even on float64 inputs (the eager
# softmax, and Qwen2's RMSNorm), so the cross-check is bounded by fp32 rounding.
# A wrong term, sign, index or transposed operand gives errors of order 1e-2 or more.
TOL = {S.NEOX: 2e-6, S.QWEN: 2e-6}


@pytest.mark.parametrize("name", ["tiny_neox_f32", "tiny_qwen_f32"])
def test_dense_block_matches_library_layer(name):
    w = S.WORKLOADS[name]
    W = S.layer_weights(w, 0)
    x = O.f64(S.hidden_states(w))
    ours = O.dense_layer(desc_of(w), W, x)
    L = hf_layer(w, W)
    pos = np.arange(w.seq)
    for b in range(w.batch):
        ref = hf_forward(w, L, x[b], pos)
        err = np.max(np.abs(ours[b] - ref)) / np.max(np.abs(ref))
        assert err < TOL[w.block], err


@pytest.mark.parametrize("name", ["tiny_neox_f32", "tiny_qwen_f32"])
@pytest.mark.parametrize("k", [1, 5, 32, 63, 64])
def test_routed_layer_is_library_layer_on_kept_subsequence(name, k):
    w = S.WORKLOADS[name]
    W = S.layer_weights(w, 0)
    x = O.f64(S.hidden_states(w))
    res = O.routed_layer(desc_of(w), W, x, k)
    L = hf_layer(w, W)
    for b in range(w.batch):
        idx = res["idx"][b]
        kept = np.zeros(w.seq, dtype=bool)
        kept[idx] = True
        np.testing.assert_array_equal(res["y"][b][~kept], x[b][~kept])
        ref = hf_forward(w, L, x[b][idx], idx)
        err = np.max(np.abs(res["y"][b][idx] - ref)) / np.max(np.abs(ref))
        assert err < TOL[w.block], err


@pytest.mark.parametrize("name", ["tiny_neox_f32", "tiny_qwen_f32"])
def test_full_and_zero_retention(name):
    w = S.WORKLOADS[name]
    W = S.layer_weights(w, 0)
    x = O.f64(S.hidden_states(w))
    d = desc_of(w)
    full = O.routed_layer(d, W, x, w.seq)
    np.testing.assert_array_equal(full["idx"], np.tile(np.arange(w.seq), (w.batch, 1)))
    np.testing.assert_array_equal(full["y"], O.dense_layer(d, W, x))
    np.testing.assert_array_equal(O.routed_layer(d, W, x, 0)["y"], x)


def test_attention_matches_sdpa_and_single_token():
    rng = np.random.default_rng(4)
    n, Hq, Hkv, hd = 37, 6, 2, 16
    q, k, v = rng.standard_normal((n, Hq, hd)), rng.standard_normal((n, Hkv, hd)), rng.standard_normal((n, Hkv, hd))
    ours = O.causal_attention(q, k, v)
    tq = torch.from_numpy(q).transpose(0, 1)
    tk = torch.from_numpy(k).transpose(0, 1).repeat_interleave(Hq // Hkv, 0)
    tv = torch.from_numpy(v).transpose(0, 1).repeat_interleave(Hq // Hkv, 0)
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True)
    np.testing.assert_allclose(ours, ref.transpose(0, 1).reshape(n, -1).numpy(), rtol=1e-12, atol=1e-12)
    # one kept token attends only to itself
    one = O.causal_attention(q[:1], k[:1], v[:1]).reshape(Hq, hd)
    np.testing.assert_allclose(one, np.repeat(v[0], Hq // Hkv, axis=0), rtol=0, atol=1e-15)


@pytest.mark.parametrize("name", ["tiny_neox_f32", "tiny_qwen_f32"])
def test_rope_shift_invariance(name):
    # Attention depends only on position differences: shifting every kept
    # position by the same amount leaves the block output unchanged.
    w = S.WORKLOADS[name]
    W = S.layer_weights(w, 0)
    xc = O.f64(S.hidden_states(w))[0, :20]
    pos = np.sort(np.random.default_rng(5).choice(64, 20, replace=False))
    a = O.block_delta(desc_of(w), W, xc, pos)
    b = O.block_delta(desc_of(w), W, xc, pos + 1000)
    assert np.max(np.abs(a - b)) / np.max(np.abs(a)) < 1e-11


def test_rope_rotation_is_norm_preserving_and_matches_complex_form():
    rng = np.random.default_rng(6)
    x = rng.standard_normal((5, 3, 16))
    pos = np.array([0, 1, 7, 100, 2047])
    y = O.rope(x, pos, 8, 10000.0)
    np.testing.assert_array_equal(y[..., 8:], x[..., 8:])           # pass-through dims
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-14)
    # pair (i, i + 4) rotates as the complex number x_i + j x_{i+4} times exp(j pos theta_i)
    for i in range(4):
        z = (x[..., i] + 1j * x[..., i + 4]) * np.exp(1j * pos[:, None] * 10000.0 ** (-2 * i / 8))
        np.testing.assert_allclose(y[..., i], z.real, rtol=1e-13, atol=1e-13)
        np.testing.assert_allclose(y[..., i + 4], z.imag, rtol=1e-13, atol=1e-13)
    np.testing.assert_array_equal(O.rope(x, np.zeros(5), 8, 10000.0), x)


def test_norms_and_activations_match_torch():
    rng = np.random.default_rng(8)
    x, g, b = rng.standard_normal((7, 40)), rng.standard_normal(40), rng.standard_normal(40)
    tx = torch.from_numpy(x)
    np.testing.assert_allclose(O.layer_norm(x, g, b, 1e-5),
                               torch.nn.functional.layer_norm(tx, (40,), torch.from_numpy(g), torch.from_numpy(b), 1e-5).numpy(),
                               rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(O.rms_norm(x, g, 1e-6),
                               torch.nn.functional.rms_norm(tx, (40,), torch.from_numpy(g), 1e-6).numpy(),
                               rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(O.gelu(x), torch.nn.functional.gelu(tx).numpy(), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(O.silu(x), torch.nn.functional.silu(tx).numpy(), rtol=1e-13, atol=1e-15)


def test_stack_composition_and_calibration():
    w = S.WORKLOADS["tiny_neox_f32"].replace(n_layers=3)
    Ws = S.stack_weights(w)
    x = O.f64(S.hidden_states(w))
    d = desc_of(w)
    # all r = 1: the dense stack, i.e. three library layers in a row
    y, _ = O.stack_forward(d, Ws, x, [w.seq] * 3)
    ref = x.copy()
    for W in Ws:
        L = hf_layer(w, W)
        ref = np.stack([hf_forward(w, L, ref[b], np.arange(w.seq)) for b in range(w.batch)])
    assert np.max(np.abs(y - ref)) / np.max(np.abs(ref)) < TOL[w.block]
    # all r = 0: identity
    y0, _ = O.stack_forward(d, Ws, x, [0] * 3)
    np.testing.assert_array_equal(y0, x)
    # calibration: a layer whose output projections are zero is an identity layer -> s = 1
    Wz = dict(Ws[1])
    for key in ("w_o", "b_o", "w_down", "b_down"):
        Wz[key] = torch.zeros_like(Wz[key])
    s = O.calibrate_similarity(d, [Ws[0], Wz, Ws[2]], x)
    assert abs(s[1] - 1.0) < 1e-14 and s[0] < 1.0 and s[2] < 1.0
    assert math.isfinite(s.sum())
