"""Full-size parity of the larger stacks, in the launch configuration the
benchmark times.

* Qwen2.5-0.5B shape (24 x 896, 14 / 2 heads of 64, SwiGLU 4864), B 8 x
  T 4096, k per layer from its similarity profile (Eqs. 5-8).
* Qwen2.5-7B shape (28 x 3584, 28 / 4 heads of 128, SwiGLU 18944), B 4 x
  T 8192, k per layer from similarities measured by the GPU calibration pass
  on the same stack, as the benchmark does.
* GPT-NeoX-1.4B shape (24 x 2048, 16 heads of 128, FFN 8192), B 4 x T 2048,
  layer 0 at r = 1 (equal, bitwise, to the dense path) and r = 0.25.
* Qwen2.5-1.5B shape (28 x 1536, 12 / 2 heads of 128, SwiGLU 8960), B 8 x
  T 2048, layer 0 at r = 0.8.

For every layer and every sequence of a stack: the stack call equals the
single-layer calls chained, bitwise; router scores lie within the fp32
bound; the GPU's indices are the oracle's Top-K of the GPU's scores; any
difference from the oracle's own selection is a near-tie; skipped rows are
bitwise unchanged. The oracle checks the kept rows teacher-forced, on one
sequence of layers 0, L/2 and L-1 (it needs from seconds to about half a
minute per sequence and layer at these shapes).
"""
import numpy as np
import pytest
import torch

import paper_2607_21291_amd as P
import synthetic as S

from gpu_util import (TOL, announce, check_layer, check_selection, desc_dict, make_desc, rel_inf, router_bound,
                      run_layer, to_np, workspace)
from oracle import adadsf_oracle as O

pytestmark = pytest.mark.gpu


class Stack:
    """A workload's layers on the device, its input and its k per layer."""

    def __init__(self, w, dev, ks):
        self.w, self.dev, self.ks = w, dev, ks
        self.layers = [P.DeviceLayer(S.layer_weights(w, l), dev) for l in range(w.n_layers)]
        self.x = S.hidden_states(w)
        self.desc = make_desc(w)

    def layer_input(self, l):
        """The GPU stack's hidden states entering layer l (device)."""
        xd = self.x.to(self.dev)
        if l > 0:
            ws = workspace(self.w, self.w.batch, self.w.seq, max(self.ks[:l]), self.dev)
            P.stack_forward(self.desc, [dl.weights for dl in self.layers[:l]], self.ks[:l], xd, ws)
            torch.cuda.synchronize()
        return xd

    def run_layer(self, l, xd):
        """Layer l in place on xd; returns (scores, idx) on the device."""
        w, k = self.w, self.ks[l]
        B, T = w.batch, w.seq
        scores = torch.empty(B, T, dtype=torch.float32, device=self.dev)
        idx = torch.empty(B, k, dtype=torch.int32, device=self.dev)
        ws = workspace(w, B, T, k, self.dev)
        P.sparse_block_forward(self.desc, self.layers[l].weights, xd, k, ws, scores_out=scores, idx_out=idx)
        torch.cuda.synchronize()
        assert P.workspace_status(ws) == 0
        return scores, idx


def calibrated_ks(w, st_layers, dev):
    """k per layer as the benchmark derives it: dense stack + Eq. 4 on the GPU,
    then Eqs. 5-8 and K = floor(r T)."""
    B, T, L = w.batch, w.seq, w.n_layers
    desc = make_desc(w)
    ws = workspace(w, B, T, T, dev, with_sim=True)
    accum = torch.zeros(L, 2, dtype=torch.float64, device=dev)
    xc = S.hidden_states(w).to(dev)
    P.stack_forward(desc, [dl.weights for dl in st_layers], [T] * L, xc, ws, flags=P.FLAG_DENSE, sim_accum=accum)
    s = P.sim_finalize(accum)
    r = P.retention_from_similarity(s, w.target, w.tau)
    return [P.k_from_retention(v, T) for v in r]


def profile_ks(w):
    r = P.retention_from_similarity(list(w.similarity), w.target, w.tau)
    return [P.k_from_retention(v, w.seq) for v in r]


_cache = {}


def stack_for(name, dev):
    if name not in _cache:
        _cache.clear()  # one large stack on the device at a time
        torch.cuda.empty_cache()
        w = S.WORKLOADS[name]
        announce(f"uploading {name} ({w.n_layers} layers)")
        if w.similarity is not None:
            st = Stack(w, dev, profile_ks(w))
        else:
            st = Stack(w, dev, [w.seq] * w.n_layers)
            st.ks = calibrated_ks(w, st.layers, dev)
        _cache[name] = st
    return _cache[name]


def check_stack_layerwise(st):
    """One stack call equals the chained single-layer calls, bitwise; every
    layer's selection and skipped rows checked for every sequence."""
    w = st.w
    B, T, L = w.batch, w.seq, w.n_layers
    xs = st.x.to(st.dev)
    ws = workspace(w, B, T, max(st.ks), st.dev)
    P.stack_forward(st.desc, [dl.weights for dl in st.layers], st.ks, xs, ws)
    torch.cuda.synchronize()
    assert P.workspace_status(ws) == 0
    del ws
    cur = st.x.to(st.dev)
    for l in range(L):
        announce(f"{w.name} layer {l} k={st.ks[l]}")
        xin = cur.clone()
        scores, idx = st.run_layer(l, cur)
        W = S.layer_weights(w, l)
        xin_np = to_np(xin)
        ref_scores = O.router_scores(xin_np, W["router_w1"], W["router_b1"], W["router_w2"], W["router_b2"])
        idx_np = idx.cpu().numpy().astype(np.int64)
        check_selection(ref_scores, router_bound(xin_np, W, w.dtype), scores.cpu().numpy(), idx_np, st.ks[l])
        kept = torch.zeros(B, T, dtype=torch.bool, device=st.dev)
        kept.scatter_(1, idx.long(), True)
        assert torch.equal(cur[~kept], xin[~kept])
        del xin
    assert torch.equal(xs, cur)


def check_layer_oracle(st, l, seq):
    w = st.w
    xd = st.layer_input(l)
    x_in = xd.cpu()
    announce(f"{w.name} layer {l} k={st.ks[l]}: oracle on sequence {seq}")
    scores, idx = st.run_layer(l, xd)
    check_layer(w, S.layer_weights(w, l), x_in, xd, scores, idx, st.ks[l], sample=[seq])


def test_qwen05b_stack_full_size(dev):
    st = stack_for("qwen05b", dev)
    assert st.ks[0] == 2362 and st.ks[-1] == 401
    check_stack_layerwise(st)


@pytest.mark.parametrize("l,seq", [(0, 2), (12, 5), (23, 7)])
def test_qwen05b_layer_oracle(dev, l, seq):
    check_layer_oracle(stack_for("qwen05b", dev), l, seq)


def test_qwen7b_stack_full_size(dev):
    st = stack_for("qwen7b", dev)
    announce(f"qwen7b calibrated k per layer {st.ks}")
    assert all(0 < k < st.w.seq for k in st.ks)
    assert abs(sum(st.ks) / (st.w.n_layers * st.w.seq) - st.w.target) < 2e-3  # sum r = t L (Eq. 8)
    check_stack_layerwise(st)


@pytest.mark.parametrize("l,seq", [(0, 0), (14, 1), (27, 3)])
def test_qwen7b_layer_oracle(dev, l, seq):
    check_layer_oracle(stack_for("qwen7b", dev), l, seq)


def test_neox14b_full_retention_is_dense(dev):
    w = S.WORKLOADS["neox14b"]
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w)
    T = w.seq
    announce("neox14b layer 0: k = T against DSF_FLAG_DENSE")
    y_full, scores, idx = run_layer(dev, w, W, x, T)
    assert torch.equal(idx.cpu(), torch.arange(T, dtype=torch.int32).expand(w.batch, T))
    y_dense, _, _ = run_layer(dev, w, W, x, T, flags=P.FLAG_DENSE)
    assert torch.equal(y_full, y_dense)
    check_layer(w, W, x, y_full, scores, idx, T, sample=[1])


def test_neox14b_quarter_retention(dev):
    w = S.WORKLOADS["neox14b"]
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w)
    k = P.k_from_retention(0.25, w.seq)
    assert k == 512
    announce(f"neox14b layer 0 k={k}")
    y, scores, idx = run_layer(dev, w, W, x, k)
    check_layer(w, W, x, y, scores, idx, k, sample=[0, 3])


def test_qwen15b_layer_full_size(dev):
    w = S.WORKLOADS["qwen15b"]
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w)
    k = P.k_from_retention(w.retention[0], w.seq)
    announce(f"qwen15b (12 q / 2 kv heads of 128) layer 0 k={k}")
    y, scores, idx = run_layer(dev, w, W, x, k)
    check_layer(w, W, x, y, scores, idx, k, sample=[0, 6])
