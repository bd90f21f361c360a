"""GPU parity of the routed layer's backward (training side of Section 3.4)
against the oracle's routed_layer_backward (pinned on the CPU against torch
autograd in float64 and finite differences).

For the given kept positions idx and output gradient dy: dx equals dy
bitwise at skipped rows; at kept rows the block's share dx - dy is held to
2e-2 of its infinity norm, on top of half a bf16 ulp of the stored dx; each
weight gradient (fp32) is held to 2e-2 of its infinity norm. Both block
families, plain and score-gated (the gate uses the GPU router's scores on
the GPU side and the oracle's own on the CPU), small ragged shapes and full
model shapes. Repeated calls are bitwise equal; k = 0 copies dy.
"""
import numpy as np
import pytest
import torch

import paper_2607_21291_amd as P
import synthetic as S
from oracle import adadsf_oracle as O

from gpu_util import TOL, announce, desc_dict, make_desc, rel_inf, to_np, update_err, workload, workspace

pytestmark = pytest.mark.gpu


def _grads(w, dev):
    qwen = w.block == S.QWEN
    shapes = {"w_qkv": (w.d_qkv, w.d_model), "b_qkv": (w.d_qkv,), "w_o": (w.d_model, w.d_attn),
              "w_up": (w.d_up, w.d_model), "w_down": (w.d_model, w.d_ff), "norm1_w": (w.d_model,),
              "norm2_w": (w.d_model,)}
    if not qwen:
        shapes.update(b_o=(w.d_model,), b_up=(w.d_ff,), b_down=(w.d_model,), norm1_b=(w.d_model,),
                      norm2_b=(w.d_model,))
    return {name: torch.full(shape, float("nan"), device=dev) for name, shape in shapes.items()}


def run_backward(dev, w, W, x, dy, idx, gate, scores=None):
    B, T, _ = x.shape
    dl = P.DeviceLayer(W, dev)
    k = idx.shape[1]
    desc = make_desc(w)
    xd, dyd = x.to(dev).contiguous(), dy.to(dev).contiguous()
    idd = torch.as_tensor(idx, dtype=torch.int32).to(dev).contiguous()
    dx = torch.full_like(xd, float("nan"))
    g = _grads(w, dev)
    ws = torch.empty(P.backward_workspace_size(desc, P.BF16, B, T, k), dtype=torch.uint8, device=dev)
    P.sparse_block_backward(desc, dl.weights, xd, dyd, idd, dx, g, ws, scores=scores,
                            flags=P.FLAG_GATE if gate else 0)
    torch.cuda.synchronize()
    assert P.workspace_status(ws) == 0, "a stream-K wait gave up"
    return dx, g


def gpu_scores(dev, w, W, x):
    B, T, _ = x.shape
    dl = P.DeviceLayer(W, dev)
    sc = torch.empty(B, T, dtype=torch.float32, device=dev)
    desc = make_desc(w)
    xd = x.to(dev).contiguous()
    ws = workspace(w, B, T, T, dev)
    idx = torch.empty(B, T, dtype=torch.int32, device=dev)
    P.sparse_block_forward(desc, dl.weights, xd, T, ws, scores_out=sc, idx_out=idx)
    torch.cuda.synchronize()
    return sc


def check_backward(w, W, x, dy, idx, gate, dx, g, seqs=None):
    ref = O.routed_layer_backward(desc_dict(w), W, x, dy, idx, gate=gate)
    dxg, dyn = to_np(dx), to_np(dy)
    B, T, _ = dyn.shape
    kept = np.zeros((B, T), dtype=bool)
    for b in range(B):
        kept[b, idx[b]] = True
    np.testing.assert_array_equal(dxg[~kept], dyn[~kept])
    errs = {"dx": update_err(dxg[kept], dyn[kept], ref["dx"][kept] - dyn[kept], w.dtype)}
    for name, t in g.items():
        got = t.double().cpu().numpy()
        assert np.all(np.isfinite(got)), name
        errs[name] = rel_inf(got, ref["grads"][name])
    print("[errors] " + " ".join(f"{n}={e:.1e}" for n, e in errs.items()), flush=True)
    for name, err in errs.items():
        assert err < TOL[w.dtype], (name, err)


CASES = [("neox_bf16_small", 150), ("qwen_bf16_small", 299), ("neox_bf16_hd128", 97), ("qwen_bf16_hd128", 129),
         ("neox_bf16_small", 1)]


@pytest.mark.parametrize("gate", [False, True])
@pytest.mark.parametrize("name,k", CASES)
def test_backward_matches_oracle(dev, name, k, gate):
    w = workload(name)
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w)
    B, T = x.shape[0], x.shape[1]
    g = torch.Generator().manual_seed(k + 17)
    dy = torch.randn(B, T, w.d_model, generator=g).to(torch.bfloat16)
    idx = np.stack([np.sort(torch.randperm(T, generator=g)[:k].numpy()) for _ in range(B)])
    sc = gpu_scores(torch.device("cuda:0"), w, W, x) if gate else None
    announce(f"backward {name} k={k} gate={gate}")
    dx, gr = run_backward(dev, w, W, x, dy, idx, gate, sc)
    check_backward(w, W, x, dy, idx, gate, dx, gr)


def test_backward_deterministic_and_empty(dev):
    w = workload("qwen_bf16_small")
    W = S.layer_weights(w, 1)
    x = S.hidden_states(w, seed_offset=2)
    B, T = x.shape[0], x.shape[1]
    g = torch.Generator().manual_seed(3)
    dy = torch.randn(B, T, w.d_model, generator=g).to(torch.bfloat16)
    idx = np.stack([np.sort(torch.randperm(T, generator=g)[:100].numpy()) for _ in range(B)])
    announce("backward determinism")
    dx1, g1 = run_backward(dev, w, W, x, dy, idx, False)
    dx2, g2 = run_backward(dev, w, W, x, dy, idx, False)
    assert torch.equal(dx1, dx2)
    for name in g1:
        assert torch.equal(g1[name], g2[name]), name
    dx0, _ = run_backward(dev, w, W, x, dy, np.zeros((B, 0), dtype=np.int64), False)
    assert torch.equal(dx0.cpu(), dy)


@pytest.mark.parametrize("name,B,T,k,gate", [("neox160m", 2, 2048, 1563, False), ("qwen05b", 1, 4096, 2362, True),
                                             ("qwen7b", 1, 2048, 1024, False)])
def test_backward_full_shapes(dev, name, B, T, k, gate):
    """Full model widths (NeoX-160M; Qwen2.5-0.5B with GQA 7:1 at head dim 64;
    Qwen2.5-7B with GQA 7:1 at head dim 128 and 18944-wide SwiGLU, where the
    projections take the 256 x 256 tiles) at full or long sequence lengths."""
    w = S.WORKLOADS[name].replace(batch=B, seq=T)
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w)
    g = torch.Generator().manual_seed(T + k)
    dy = (torch.randn(B, T, w.d_model, generator=g) * 0.02).to(torch.bfloat16)
    idx = np.stack([np.sort(torch.randperm(T, generator=g)[:k].numpy()) for _ in range(B)])
    sc = gpu_scores(torch.device("cuda:0"), w, W, x) if gate else None
    announce(f"backward full shape {name} B={B} T={T} k={k} gate={gate}")
    dx, gr = run_backward(dev, w, W, x, dy, idx, gate, sc)
    check_backward(w, W, x, dy, idx, gate, dx, gr)


def test_backward_streamk_wait_timeout_is_reported(dev, monkeypatch):
    """The weight gradients of a full-width NeoX-160M layer (B 2, k 1563 of
    2048: 3126 kept rows) take the stream-K grid. DSF_SK_SPIN_LIMIT=0 makes
    every wait for an earlier piece give up at once (every kernel still exits
    normally); the status word reports it, and the next normal call clears it
    and is correct again."""
    w = S.WORKLOADS["neox160m"].replace(batch=2, seq=2048)
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w)
    g = torch.Generator().manual_seed(17)
    dy = (torch.randn(2, 2048, w.d_model, generator=g) * 0.02).to(torch.bfloat16)
    idx = np.stack([np.sort(torch.randperm(2048, generator=g)[:1563].numpy()) for _ in range(2)])
    dl = P.DeviceLayer(W, dev)
    desc = make_desc(w)
    xd, dyd = x.to(dev).contiguous(), dy.to(dev).contiguous()
    idd = torch.as_tensor(idx, dtype=torch.int32).to(dev).contiguous()
    dx = torch.empty_like(xd)
    gr = _grads(w, dev)
    ws = torch.empty(P.backward_workspace_size(desc, P.BF16, 2, 2048, 1563), dtype=torch.uint8, device=dev)
    announce("backward stream-K give-up reported")
    monkeypatch.setenv("DSF_SK_SPIN_LIMIT", "0")
    P.sparse_block_backward(desc, dl.weights, xd, dyd, idd, dx, gr, ws)
    torch.cuda.synchronize()
    assert P.workspace_status(ws) == P.WS_STATUS_SK_TIMEOUT
    monkeypatch.delenv("DSF_SK_SPIN_LIMIT")
    dx, gr = run_backward(dev, w, W, x, dy, idx, False)
    check_backward(w, W, x, dy, idx, False, dx, gr)
