"""GPU parity of incremental decoding with kept-token KV caches.

The paper treats prefill only; the decode reading (threshold routing of each
new token, per-layer caches of the kept tokens' keys and values) is stated in
the oracle's header, where the CPU tests pin it. Here:

1. decoding token by token from empty caches with forced keep decisions
   (thresholds of -inf / +inf) equals the oracle's stack over the whole
   sequence with the same kept sets (kept_set_stack, rounded to the storage
   format after each layer), within the layer tolerance; tokens skipped by
   every layer come out bitwise unchanged, and the cache lengths count the
   kept tokens;
2. dsf_stack_prefill equals the layer-by-layer stack bitwise, fills the
   caches' lengths and returns the lowest kept score of each sequence; the
   decode steps that follow route by those thresholds (each decision equals
   score >= threshold) and the whole sequence then matches the oracle over
   the prefill's selections plus the decode decisions;
3. a kept token meeting a full cache is skipped (reported as 2) and passes
   through bitwise; repeated steps are deterministic;
4. at the bench's decode shape (neox160m layer 0, 8 sequences, 2048-token
   prompt): a forced-kept token matches the oracle's block over the prompt's
   kept rows plus itself, and every routing decision, skipped row and cache
   length holds.
"""
import numpy as np
import pytest
import torch

import paper_2607_21291_amd as P
import synthetic as S
from oracle import adadsf_oracle as O

from gpu_util import TOL, announce, desc_dict, dtype_code, make_desc, rel_inf, to_np, workload, workspace

pytestmark = pytest.mark.gpu


class Caches:
    def __init__(self, w, B, cap, L, dev):
        dt = w.torch_dtype
        self.k = [torch.zeros(B, w.n_kv_heads, cap, w.head_dim, dtype=dt, device=dev) for _ in range(L)]
        self.v = [torch.zeros(B, w.n_kv_heads, cap, w.head_dim, dtype=dt, device=dev) for _ in range(L)]
        self.len = torch.zeros(L, B, dtype=torch.int32, device=dev)


def _decode(dev, w, dls, x_tok, t_pos, thr, caches, ws, max_pos, keep_out=None, scores_out=None):
    """One step: x_tok [B, d] (CPU) at position t_pos; returns the new states (CPU)."""
    xt = x_tok.to(dev).contiguous()
    B = xt.shape[0]
    pos = torch.full((B,), t_pos, dtype=torch.int32, device=dev)
    P.decode_step(make_desc(w), [dl.weights for dl in dls], xt, pos, max_pos, thr, caches.k, caches.v, caches.len,
                  ws, scores_out=scores_out, keep_out=keep_out)
    torch.cuda.synchronize()
    return xt.cpu()


def _delta_check(w, x, y, y_ref):
    assert rel_inf(to_np(y) - to_np(x), np.asarray(y_ref) - to_np(x)) < TOL[w.dtype]


@pytest.mark.parametrize("name,T,B", [("tiny_neox_f32", 40, 2), ("tiny_qwen_f32", 33, 2), ("neox_bf16_small", 300, 2),
                                      ("qwen_bf16_small", 48, 2), ("neox_bf16_hd128", 40, 2),
                                      ("qwen_bf16_hd128", 37, 2), ("neox_bf16_small", 24, 20),
                                      ("qwen_bf16_small", 20, 17)])
def test_decode_with_forced_keeps_matches_full_sequence(dev, name, T, B):
    """B <= 16 runs the projections on the few-row split-K GEMM, B > 16 on the tile GEMMs."""
    w = workload(name).replace(n_layers=2)
    L = 2
    Ws = S.stack_weights(w)
    dls = [P.DeviceLayer(W, dev) for W in Ws]
    x = S.hidden_states(w, batch=B, seq=T)
    g = np.random.default_rng(T)
    # kept sets of different sizes per (layer, sequence); token 0 skipped by every layer of sequence 1
    keeps = [[np.sort(g.choice(np.arange(1 if b else 0, T), size=max(1, int(T * frac) - b % 3), replace=False))
              for b in range(B)] for frac in (0.6, 0.35)]
    caches = Caches(w, B, T, L, dev)
    ws = torch.empty(P.decode_workspace_size(make_desc(w), dtype_code(w), B, T, T), dtype=torch.uint8, device=dev)
    y = torch.empty_like(x)
    keep_out = torch.empty(L, B, dtype=torch.int32, device=dev)
    announce(f"decode forced {name} T={T} B={B}")
    for t in range(T):
        forced = np.array([[t in set(keeps[l][b].tolist()) for b in range(B)] for l in range(L)])
        thr = torch.tensor(np.where(forced, -np.inf, np.inf), dtype=torch.float32, device=dev)
        y[:, t] = _decode(dev, w, dls, x[:, t], t, thr, caches, ws, T, keep_out=keep_out)
        assert np.array_equal(keep_out.cpu().numpy(), forced.astype(np.int32)), t
    y_ref = O.kept_set_stack(desc_dict(w), Ws, x, keeps, out_dtype=w.dtype)
    _delta_check(w, x, y, y_ref)
    assert torch.equal(y[1, 0], x[1, 0])  # skipped by every layer: bitwise unchanged
    lens = np.array([[len(keeps[l][b]) for b in range(B)] for l in range(L)])
    np.testing.assert_array_equal(caches.len.cpu().numpy(), lens)


@pytest.mark.parametrize("name", ["tiny_neox_f32", "qwen_bf16_small", "neox_bf16_small"])
def test_prefill_then_threshold_decode(dev, name):
    w = workload(name).replace(n_layers=2)
    L, B, T0, T1 = 2, 2, 64, 24
    T = T0 + T1
    ks = [40, 24]
    Ws = S.stack_weights(w)
    dls = [P.DeviceLayer(W, dev) for W in Ws]
    desc = make_desc(w)
    x = S.hidden_states(w, batch=B, seq=T, seed_offset=7)
    caches = Caches(w, B, T, L, dev)
    thr = torch.full((L, B), float("nan"), dtype=torch.float32, device=dev)
    xp = x[:, :T0].to(dev).contiguous()
    announce(f"prefill {name} T0={T0}")
    P.stack_prefill(desc, [dl.weights for dl in dls], ks, xp, caches.k, caches.v, caches.len,
                    workspace(w, B, T0, max(ks), dev), thr_out=thr)
    torch.cuda.synchronize()
    # the same layers one by one through the single-layer entry point: same kernels, same decisions
    xs = x[:, :T0].to(dev).contiguous()
    idxs, thr_ref = [], np.zeros((L, B), dtype=np.float32)
    for l, k in enumerate(ks):
        sc = torch.empty(B, T0, dtype=torch.float32, device=dev)
        idx = torch.empty(B, k, dtype=torch.int32, device=dev)
        P.sparse_block_forward(desc, dls[l].weights, xs, k, workspace(w, B, T0, k, dev), scores_out=sc, idx_out=idx)
        torch.cuda.synchronize()
        idxs.append(idx.cpu().numpy())
        scn = sc.cpu().numpy()
        thr_ref[l] = [scn[b, idxs[l][b]].min() for b in range(B)]
    assert torch.equal(xs, xp)
    np.testing.assert_array_equal(thr.cpu().numpy(), thr_ref)
    np.testing.assert_array_equal(caches.len.cpu().numpy(), np.array([[k] * B for k in ks]))
    # decode with the prefill's thresholds
    ws = torch.empty(P.decode_workspace_size(desc, dtype_code(w), B, T, T), dtype=torch.uint8, device=dev)
    ko = torch.empty(T1, L, B, dtype=torch.int32, device=dev)
    so = torch.empty(T1, L, B, dtype=torch.float32, device=dev)
    yd = torch.empty(B, T1, w.d_model, dtype=x.dtype)
    announce(f"threshold decode {name} T1={T1}")
    for t in range(T1):
        yd[:, t] = _decode(dev, w, dls, x[:, T0 + t], T0 + t, thr, caches, ws, T, keep_out=ko[t], scores_out=so[t])
    kon, son = ko.cpu().numpy(), so.cpu().numpy()
    np.testing.assert_array_equal(kon, (son >= thr.cpu().numpy()[None]).astype(np.int32))
    assert kon.any() and not kon.all()
    np.testing.assert_array_equal(caches.len.cpu().numpy(), np.array(ks)[:, None] + kon.sum(axis=0))
    keeps = [[np.concatenate([idxs[l][b], T0 + np.nonzero(kon[:, l, b])[0]]) for b in range(B)] for l in range(L)]
    y_ref = O.kept_set_stack(desc_dict(w), Ws, x, keeps, out_dtype=w.dtype)
    _delta_check(w, x[:, :T0], xp.cpu(), y_ref[:, :T0])
    _delta_check(w, x[:, T0:], yd, y_ref[:, T0:])


def test_full_cache_and_determinism(dev):
    w = workload("tiny_neox_f32").replace(n_layers=1)
    Ws = S.stack_weights(w)
    dls = [P.DeviceLayer(W, dev) for W in Ws]
    B, cap = 1, 2
    x = S.hidden_states(w, batch=B, seq=3, seed_offset=11)
    caches = Caches(w, B, cap, 1, dev)
    ws = torch.empty(P.decode_workspace_size(make_desc(w), dtype_code(w), B, 8, cap), dtype=torch.uint8, device=dev)
    thr = torch.full((1, B), -float("inf"), dtype=torch.float32, device=dev)
    ko = torch.empty(1, B, dtype=torch.int32, device=dev)
    announce("decode full cache")
    outs = []
    for t in range(3):
        outs.append(_decode(dev, w, dls, x[:, t], t, thr, caches, ws, 8, keep_out=ko))
        assert ko.item() == (1 if t < 2 else 2)
    assert torch.equal(outs[2], x[:, 2])
    assert caches.len.item() == 2
    # the same step from the same state twice: identical
    c2 = Caches(w, B, cap, 1, dev)
    a = _decode(dev, w, dls, x[:, 0], 0, thr, c2, ws, 8)
    c2.len.zero_()
    b = _decode(dev, w, dls, x[:, 0], 0, thr, c2, ws, 8)
    assert torch.equal(a, b) and torch.equal(a, outs[0])


def test_neox160m_decode_full_size(dev):
    """The bench's decode shape on layer 0 of the neox160m stack: prefill of
    B = 8 sequences of 2048 tokens keeping k_0 = 1563, then one decode step at
    position 2048. Sequence 0 is forced to keep its token: its output must
    equal the oracle's block over the prompt's kept rows plus the new token,
    at their positions (the new row last). The other sequences route by the
    prefill's thresholds: each decision is score >= threshold, skipped rows
    are bitwise unchanged, kept rows grow their cache by one."""
    w = S.WORKLOADS["neox160m"].replace(n_layers=1)
    B, T = w.batch, w.seq
    k0 = 1563
    W = S.layer_weights(w, 0)
    dl = P.DeviceLayer(W, dev)
    desc = make_desc(w)
    x = S.hidden_states(w)
    caches = Caches(w, B, T + 1, 1, dev)
    thr = torch.empty(1, B, dtype=torch.float32, device=dev)
    xp = x.to(dev).contiguous()
    announce(f"full-size decode neox160m prefill k={k0}")
    P.stack_prefill(desc, [dl.weights], [k0], xp, caches.k, caches.v, caches.len, workspace(w, B, T, k0, dev),
                    thr_out=thr)
    # the prefill's selection, by the single-layer entry point on the same input
    idx = torch.empty(B, k0, dtype=torch.int32, device=dev)
    xs = x.to(dev).contiguous()
    P.sparse_block_forward(desc, dl.weights, xs, k0, workspace(w, B, T, k0, dev), idx_out=idx)
    torch.cuda.synchronize()
    assert torch.equal(xs, xp)
    idx0 = idx[0].cpu().numpy()
    g = torch.Generator().manual_seed(2048)
    xn = (torch.randn(B, w.d_model, generator=g) * 0.02).to(w.torch_dtype)
    thr_step = thr.clone()
    thr_step[0, 0] = -float("inf")
    ko = torch.empty(1, B, dtype=torch.int32, device=dev)
    so = torch.empty(1, B, dtype=torch.float32, device=dev)
    ws = torch.empty(P.decode_workspace_size(desc, dtype_code(w), B, T + 1, T + 1), dtype=torch.uint8, device=dev)
    announce("full-size decode neox160m step")
    y = _decode(dev, w, [dl], xn, T, thr_step, caches, ws, T + 1, keep_out=ko, scores_out=so)
    kon, son, thn = ko.cpu().numpy()[0], so.cpu().numpy()[0], thr_step.cpu().numpy()[0]
    np.testing.assert_array_equal(kon, (son >= thn).astype(np.int32))
    assert kon[0] == 1
    lens = caches.len.cpu().numpy()[0]
    np.testing.assert_array_equal(lens, k0 + kon)
    for b in range(B):
        if not kon[b]:
            assert torch.equal(y[b], xn[b])
    rows = np.concatenate([O.f64(x[0])[idx0], O.f64(xn[0:1])])
    pos = np.concatenate([idx0, [T]])
    ref = O.f64(xn[0]) + O.block_delta(desc_dict(w), W, rows, pos)[-1]
    assert rel_inf(to_np(y[0]) - O.f64(xn[0]), ref - O.f64(xn[0])) < TOL[w.dtype]
