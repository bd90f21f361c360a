"""Router and Top-K in one launch (the last-arriving workgroup of each sequence
selects), against the oracle and against the two-launch path.

Sequence lengths are multiples of 64, where the layer takes the one-launch
path; DSF_UNFUSED_ROUTING=1 forces the router and Top-K kernels. Both paths
run the same router arithmetic and the same selection, so scores, indices and
layer outputs must agree bit for bit; the layer protocol of the other parity
tests (scores within the rounding bound, the oracle's Top-K of the GPU's
scores equal to the GPU's indices, outputs within 2e-2 of the oracle
teacher-forced with them) is applied to the one-launch path.
"""
import numpy as np
import pytest
import torch

import paper_2607_21291_amd as P
import synthetic as S
from oracle import adadsf_oracle as O

from gpu_util import announce, check_layer, make_desc, run_layer, workload, workspace

pytestmark = pytest.mark.gpu

CASES = [("neox_bf16_small", 3, 320, 1), ("neox_bf16_small", 3, 320, 107), ("neox_bf16_small", 3, 320, 319),
         ("neox_bf16_small", 3, 320, 320), ("qwen_bf16_small", 2, 256, 128), ("qwen_bf16_small", 2, 256, 255),
         ("neox_bf16_small", 5, 64, 17), ("qwen_bf16_hd128", 2, 448, 200)]


@pytest.mark.parametrize("name,B,T,k", CASES)
def test_one_launch_routing_matches_oracle_and_two_launches(dev, monkeypatch, name, B, T, k):
    w = workload(name).replace(batch=B, seq=T)
    announce(f"fused routing {name} B={B} T={T} k={k}")
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w)
    y, scores, idx = run_layer(dev, w, W, x, k)
    check_layer(w, W, x, y, scores, idx, k)
    monkeypatch.setenv("DSF_UNFUSED_ROUTING", "1")
    y2, scores2, idx2 = run_layer(dev, w, W, x, k)
    assert torch.equal(scores, scores2)
    assert torch.equal(idx, idx2)
    assert torch.equal(y, y2)


def test_one_launch_routing_ties_keep_lowest_positions(dev):
    # W1 = 0 and b1 = 0: every hidden unit is 0, every score is b2, and the
    # k kept tokens of every sequence are positions 0 .. k-1
    w = workload("neox_bf16_small").replace(batch=4, seq=192)
    announce("fused routing, all scores tied")
    W = dict(S.layer_weights(w, 2))
    W["router_w1"] = torch.zeros_like(W["router_w1"])
    W["router_b1"] = torch.zeros_like(W["router_b1"])
    x = S.hidden_states(w)
    for k in (1, 77, 191):
        y, scores, idx = run_layer(dev, w, W, x, k)
        assert torch.all(scores == scores[0, 0])
        assert torch.equal(idx.cpu(), torch.arange(k, dtype=torch.int32).expand(w.batch, k))
        check_layer(w, W, x, y, scores, idx, k)


def test_one_launch_routing_stack_repeats(dev, monkeypatch):
    # the per-sequence counters are left zero by every launch: a stack of
    # layers with different k, called twice, gives the same bits, and the same
    # bits as the two-launch path
    w = workload("neox_bf16_small").replace(n_layers=4, batch=3, seq=256)
    announce("fused routing stack, repeated")
    Ws = S.stack_weights(w)
    x = S.hidden_states(w)
    ks = [128, 255, 1, 64]
    dls = [P.DeviceLayer(W, dev) for W in Ws]
    ws = workspace(w, w.batch, w.seq, max(ks), dev)
    outs = []
    for env in (None, None, "1"):
        if env:
            monkeypatch.setenv("DSF_UNFUSED_ROUTING", env)
        xd = x.to(dev)
        P.stack_forward(make_desc(w), [dl.weights for dl in dls], ks, xd, ws)
        torch.cuda.synchronize()
        outs.append(xd.cpu())
    assert torch.equal(outs[0], outs[1])
    assert torch.equal(outs[0], outs[2])
