"""Parity at full benchmark size, in the launch configuration the benchmark
times: the 12-layer NeoX-160M-shaped stack (d 768, 12 x 64 heads, d_ff 3072)
on B = 8 sequences of T = 2048 tokens, one stack call with the per-layer k
that Eqs. 5-8 give for its similarity profile; and one Qwen-0.5B-shaped layer
(d 896, 14 / 2 heads, SwiGLU 4864) on B = 8, T = 4096.

The two larger shapes get one layer each: GPT-NeoX-1.4B (d 2048, 16 x 128
heads, d_ff 8192, B 4, T 2048) at its fixed r = 0.5, and Qwen2.5-7B (d 3584,
28 / 4 heads of 128, SwiGLU 18944, B 4, T 8192) at r = 0.5.

The oracle needs from 2 s to about a minute per sequence per layer here, so it checks
sampled (layer, sequence) pairs, teacher-forced with the GPU's indices; the
rest is covered by properties that hold at any size, for every sequence of
every layer: router scores within the fp32 bound, the GPU's indices equal to
the oracle's Top-K of the GPU's scores, skipped rows bitwise unchanged, and
the stack call equal, bitwise, to the single-layer calls chained.
"""
import pytest
import torch

import paper_2607_21291_amd as P
import synthetic as S

from gpu_util import announce, check_layer, make_desc, run_layer, workspace

pytestmark = pytest.mark.gpu


def profile_ks(w):
    r = P.retention_from_similarity(list(w.similarity), w.target, w.tau)
    return [P.k_from_retention(v, w.seq) for v in r]


def test_neox160m_stack_full_size(dev):
    w = S.WORKLOADS["neox160m"]
    ks = profile_ks(w)
    assert ks[0] == 1563 and ks[-1] == 600 and sum(ks) == 14741
    announce(f"full-size stack neox160m B={w.batch} T={w.seq} ks={ks}")
    Ws = S.stack_weights(w)
    x = S.hidden_states(w)
    dls = [P.DeviceLayer(W, dev) for W in Ws]
    xd = x.to(dev)
    ws = workspace(w, w.batch, w.seq, max(ks), dev)
    P.stack_forward(make_desc(w), [dl.weights for dl in dls], ks, xd, ws)
    torch.cuda.synchronize()
    cur = x
    for l, (W, k) in enumerate(zip(Ws, ks)):
        announce(f"full-size neox160m layer {l} k={k}")
        y, scores, idx = run_layer(dev, w, W, cur, k)
        sample = [(3 * l) % w.batch] if l in (0, 5, 11) else []
        check_layer(w, W, cur, y, scores, idx, k, sample=sample)
        cur = y.cpu()
    assert torch.equal(xd.cpu(), cur)


def test_qwen05b_layer_full_size(dev):
    w = S.WORKLOADS["qwen05b"]
    k = profile_ks(w)[0]
    announce(f"full-size layer qwen05b B={w.batch} T={w.seq} k={k}")
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w)
    y, scores, idx = run_layer(dev, w, W, x, k)
    check_layer(w, W, x, y, scores, idx, k, sample=[0, 5])


def test_neox14b_layer_full_size(dev):
    w = S.WORKLOADS["neox14b"]
    k = P.k_from_retention(w.retention[0], w.seq)
    announce(f"full-size layer neox14b B={w.batch} T={w.seq} k={k}")
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w)
    y, scores, idx = run_layer(dev, w, W, x, k)
    check_layer(w, W, x, y, scores, idx, k, sample=[3])


def test_qwen7b_layer_full_size(dev):
    w = S.WORKLOADS["qwen7b"]
    k = P.k_from_retention(w.target, w.seq)
    announce(f"full-size layer qwen7b B={w.batch} T={w.seq} k={k}")
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w)
    y, scores, idx = run_layer(dev, w, W, x, k)
    check_layer(w, W, x, y, scores, idx, k, sample=[1])

