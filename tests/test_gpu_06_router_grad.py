"""GPU parity of the router-score pathway (Section 3.4, training side).

1. The score-gated layer (DSF_FLAG_GATE): x + sigmoid(score) * delta at the
   kept rows, checked with the layer protocol of the ungated layer against the
   oracle's gated layer (teacher-forced with the GPU's indices); with the
   gate saturated at 1 the NeoX layer equals the ungated one bitwise; the
   gated stack equals the gated layers chained, bitwise.
2. dsf_gate_score_grad on seeded synthetic rows against the oracle, within
   the fp32 rounding bound of a d-term dot product; skipped positions exactly
   zero.
3. dsf_router_backward against the oracle's router backward, at small ragged
   sizes and at full benchmark size. The ReLU decision of a hidden unit whose
   pre-activation lies within the fp32 rounding bound of zero may go either
   way; each such unit adds what its flip can change to the allowance of the
   outputs it feeds (in practice no unit is that close).
"""
import numpy as np
import pytest
import torch

import paper_2607_21291_amd as P
import synthetic as S
from oracle import adadsf_oracle as O

from gpu_util import (TOL, U32, announce, check_layer, make_desc, rel_inf, run_layer, to_np, workload,
                      workspace)

pytestmark = pytest.mark.gpu

GATED = [("tiny_neox_f32", 32), ("tiny_qwen_f32", 63), ("neox_bf16_small", 150), ("qwen_bf16_small", 299),
         ("neox_bf16_hd128", 97), ("qwen_bf16_hd128", 129), ("neox_bf16_small", 1)]


def gamma(n: int) -> float:
    return n * U32 / (1 - n * U32)


# ------------------------------------------------------------ gated layer

@pytest.mark.parametrize("name,k", GATED)
def test_gated_layer_matches_oracle(dev, name, k):
    w = workload(name)
    announce(f"gated layer {name} k={k}")
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w)
    y, scores, idx = run_layer(dev, w, W, x, k, flags=P.FLAG_GATE)
    check_layer(w, W, x, y, scores, idx, k, gate=True)
    y2, _, _ = run_layer(dev, w, W, x, k, flags=P.FLAG_GATE)
    assert torch.equal(y, y2)


@pytest.mark.parametrize("schedule", ["streamk", "persistent"])
def test_gated_layer_persistent_schedules(dev, monkeypatch, schedule):
    w = workload("qwen_bf16_small")
    W = S.layer_weights(w, 1)
    x = S.hidden_states(w, seed_offset=1)
    monkeypatch.setenv("DSF_GEMM_SCHEDULE", schedule)
    announce(f"gated layer qwen_bf16_small {schedule}")
    y, scores, idx = run_layer(dev, w, W, x, 211, flags=P.FLAG_GATE)
    check_layer(w, W, x, y, scores, idx, 211, gate=True)


@pytest.mark.parametrize("name", ["neox_bf16_small", "qwen_bf16_small", "tiny_neox_f32"])
def test_saturated_gate_is_the_plain_layer(dev, name):
    # with a router bias of 200 every score exceeds 100, sigmoid rounds to 1
    # in fp32, and the gated update is the plain one
    w = workload(name)
    W = dict(S.layer_weights(w, 0), router_b2=200.0)
    x = S.hidden_states(w)
    k = w.seq // 2
    announce(f"saturated gate {name}")
    yg, sg, ig = run_layer(dev, w, W, x, k, flags=P.FLAG_GATE)
    yp, sp, ip = run_layer(dev, w, W, x, k)
    assert torch.equal(ig, ip) and torch.equal(sg, sp)
    assert float(sg.min()) > 100.0
    if w.block == "neox_parallel":
        # x + 1 * (C + b) rounds exactly as (C + b) + x
        assert torch.equal(yg, yp)
    else:
        assert rel_inf(to_np(yg) - to_np(x), to_np(yp) - to_np(x)) < TOL[w.dtype]


@pytest.mark.parametrize("name", ["neox_bf16_small", "qwen_bf16_small"])
def test_gated_stack_matches_layerwise(dev, name):
    w = workload(name).replace(n_layers=3)
    announce(f"gated stack {name}")
    Ws = S.stack_weights(w)
    x = S.hidden_states(w)
    T = w.seq
    ks = [T // 2, T - 3, max(1, T // 5)]
    dls = [P.DeviceLayer(W, dev) for W in Ws]
    xd = x.to(dev)
    ws = workspace(w, w.batch, T, max(ks), dev)
    P.stack_forward(make_desc(w), [dl.weights for dl in dls], ks, xd, ws, flags=P.FLAG_GATE)
    cur = x
    for W, k in zip(Ws, ks):
        y, _, _ = run_layer(dev, w, W, cur, k, flags=P.FLAG_GATE)
        cur = y.cpu()
    torch.cuda.synchronize()
    assert torch.equal(xd.cpu(), cur)


def test_gated_layer_full_size(dev):
    # neox160m layer 0 at B = 8, T = 2048, k = 1563: the down projection takes
    # the stream-K schedule, so the gate runs in its split-tile epilogue
    w = S.WORKLOADS["neox160m"]
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w)
    k = 1563
    announce(f"full-size gated layer neox160m k={k}")
    y, scores, idx = run_layer(dev, w, W, x, k, flags=P.FLAG_GATE)
    check_layer(w, W, x, y, scores, idx, k, sample=[6], gate=True)


# ------------------------------------------------------ gate score gradient

def _torch_dtype(dtype: str):
    return torch.float32 if dtype == "f32" else torch.bfloat16


def _gate_inputs(B, T, d, k, dtype, seed):
    g = np.random.default_rng(seed)
    tdt = _torch_dtype(dtype)
    x_in = torch.tensor(g.normal(size=(B, T, d)), dtype=tdt)
    x_out = torch.tensor(g.normal(size=(B, T, d)) * 0.3, dtype=tdt) + x_in
    dy = torch.tensor(g.normal(size=(B, T, d)), dtype=tdt)
    scores = torch.tensor(g.normal(size=(B, T)) * 3.0, dtype=torch.float32)
    idx = np.stack([np.sort(g.permutation(T)[:k]) for _ in range(B)]).astype(np.int32) if k > 0 \
        else np.zeros((B, 0), dtype=np.int32)
    return dy, x_in, x_out, scores, idx


@pytest.mark.parametrize("B,T,d,k,dtype", [(2, 64, 128, 20, "f32"), (3, 333, 768, 250, "bf16"),
                                           (2, 97, 3584, 1, "bf16"), (4, 2048, 768, 1563, "bf16"),
                                           (2, 50, 896, 50, "bf16")])
def test_gate_score_grad_matches_oracle(dev, B, T, d, k, dtype):
    announce(f"gate score grad B={B} T={T} d={d} k={k} {dtype}")
    dy, x_in, x_out, scores, idx = _gate_inputs(B, T, d, k, dtype, seed=B * 1000 + k)
    out = torch.full((B, T), float("nan"), dtype=torch.float32, device=dev)
    P.gate_score_grad(dy.to(dev), x_in.to(dev), x_out.to(dev), scores.to(dev), torch.tensor(idx).to(dev), out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    ref = O.gate_score_grad(to_np(dy), to_np(x_in), to_np(x_out), scores.numpy(), idx)
    kept = np.zeros((B, T), dtype=bool)
    for b in range(B):
        kept[b, idx[b]] = True
    assert np.all(got[~kept] == 0.0)
    mag = np.sum(np.abs(to_np(dy)) * np.abs(to_np(x_out) - to_np(x_in)), axis=-1) * (1 - O.sigmoid(scores.numpy()))
    bound = gamma(d + 8) * mag + 1e-30
    assert np.all(np.abs(got - ref)[kept] <= bound[kept]), np.max(np.abs(got - ref) - bound)


def test_gate_score_grad_edge_cases(dev):
    B, T, d = 2, 40, 64
    dy, x_in, x_out, scores, idx = _gate_inputs(B, T, d, 5, "bf16", seed=5)
    args = [t.to(dev) for t in (dy, x_in, x_out, scores)]
    announce("gate score grad: k = 0 and out-of-range positions")
    out = torch.full((B, T), float("nan"), dtype=torch.float32, device=dev)
    P.gate_score_grad(*args, torch.zeros(B, 0, dtype=torch.int32, device=dev), out)
    torch.cuda.synchronize()
    assert torch.all(out == 0)
    bad = idx.copy()
    bad[0, 1] = T        # ignored
    bad[1, 3] = -1       # ignored
    P.gate_score_grad(*args, torch.tensor(bad).to(dev), out)
    torch.cuda.synchronize()
    ref = O.gate_score_grad(to_np(dy), to_np(x_in), to_np(x_out), scores.numpy(), idx)
    got = out.cpu().numpy()
    assert got[0, idx[0, 1]] == 0.0 and got[1, idx[1, 3]] == 0.0
    keep = [(0, p) for j, p in enumerate(idx[0]) if j != 1] + [(1, p) for j, p in enumerate(idx[1]) if j != 3]
    for b, p in keep:
        assert abs(got[b, p] - ref[b, p]) <= 1e-4 * max(1.0, abs(ref[b, p]))


# ----------------------------------------------------------- router backward

def _allowance(x, w1, b1, w2, ds):
    """What the ReLU decisions that fp32 may take either way can change."""
    xs = x.reshape(-1, x.shape[-1])
    ax, aw1 = np.abs(xs), np.abs(w1)
    z = xs @ w1.T + (b1 if b1 is not None else 0.0)
    zb = gamma(xs.shape[1] + 4) * (ax @ aw1.T + (np.abs(b1) if b1 is not None else 0.0))
    amb = np.abs(z) <= zb
    flip = amb * np.abs(ds)[:, None] * np.abs(w2)[None, :]
    return {"dw1": flip.T @ ax, "db1": flip.sum(0), "dw2": (amb * np.abs(ds)[:, None] * (np.abs(z) + zb)).sum(0),
            "db2": 0.0, "dx": flip @ aw1, "n_ambiguous": int(amb.sum())}


def _run_router_backward(dev, x, W, ds, with_b1=True, dx0=None):
    d = x.shape[-1]
    n = x.numel() // d
    dr = W["router_w1"].shape[0]
    xd = x.to(dev).contiguous()
    w1, w2 = W["router_w1"].to(dev), W["router_w2"].to(dev)
    b1 = W["router_b1"].to(dev) if with_b1 else None
    f = dict(device=dev, dtype=torch.float32)
    out = {"dw1": torch.full((dr, d), float("nan"), **f), "dw2": torch.full((dr,), float("nan"), **f),
           "db2": torch.full((1,), float("nan"), **f),
           "db1": torch.full((dr,), float("nan"), **f) if with_b1 else None}
    dx = None if dx0 is None else dx0.to(dev).clone()
    P.router_backward(xd, w1, b1, w2, torch.tensor(ds, dtype=torch.float32, device=dev), out["dw1"], out["db1"],
                      out["dw2"], out["db2"], dx=dx)
    torch.cuda.synchronize()
    res = {k: (None if v is None else v.cpu().numpy().astype(np.float64)) for k, v in out.items()}
    res["db2"] = float(res["db2"][0])
    res["dx"] = None if dx is None else to_np(dx)
    return res


def _check_router_backward(w, W, x, ds, got, with_b1=True, dx0=None):
    xs = to_np(x)
    d = xs.shape[-1]
    w1, w2 = to_np(W["router_w1"]), to_np(W["router_w2"])
    b1 = to_np(W["router_b1"]) if with_b1 else None
    ref = O.router_backward(xs.reshape(-1, d), w1, b1, w2, ds)
    allow = _allowance(xs, w1, b1, w2, ds)
    tol = TOL[w.dtype]
    names = ["dw1", "dw2", "db2"] + (["db1"] if with_b1 else [])
    for name in names:
        r = np.asarray(ref[name], dtype=np.float64)
        g = np.asarray(got[name], dtype=np.float64)
        err = np.abs(g - r)
        lim = tol * max(np.max(np.abs(r)), 1e-30) + allow[name]
        assert np.all(err <= lim), (name, float(np.max(err - lim)))
    if dx0 is not None:
        rdx = ref["dx"]
        base = to_np(dx0).reshape(-1, d)
        gdx = got["dx"].reshape(-1, d)
        u = 2.0 ** -8 if w.dtype == "bf16" else U32  # rounding of the accumulated result
        lim = u * np.abs(base + rdx) + tol * np.max(np.abs(rdx)) + allow["dx"]
        assert np.all(np.abs(gdx - (base + rdx)) <= lim), float(np.max(np.abs(gdx - (base + rdx)) - lim))
    return allow["n_ambiguous"]


ROUTER_CASES = [("tiny_neox_f32", 32, 2, 64), ("tiny_qwen_f32", 16, 2, 63), ("neox160m", 32, 2, 333),
                ("neox160m", 16, 1, 100), ("neox160m", 48, 3, 77), ("neox160m", 64, 2, 257),
                ("qwen7b", 32, 1, 300), ("qwen05b", 64, 1, 1)]


@pytest.mark.parametrize("name,dr,B,T", ROUTER_CASES)
def test_router_backward_matches_oracle(dev, name, dr, B, T):
    w = S.WORKLOADS[name].replace(d_router=dr)
    announce(f"router backward {name} d_r={dr} B={B} T={T}")
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w, batch=B, seq=T)
    ds = np.random.default_rng(B * T + dr).normal(size=B * T)
    # dx starts at zero, then accumulates onto a random gradient
    dx0 = torch.zeros_like(x)
    got = _run_router_backward(dev, x, W, ds, dx0=dx0)
    _check_router_backward(w, W, x, ds, got, dx0=dx0)
    dx1 = torch.tensor(np.random.default_rng(7).normal(size=tuple(x.shape)), dtype=x.dtype)
    got1 = _run_router_backward(dev, x, W, ds, dx0=dx1)
    _check_router_backward(w, W, x, ds, got1, dx0=dx1)
    for key in ("dw1", "db1", "dw2"):
        assert np.array_equal(got[key], got1[key])  # the same fixed-order sums
    assert got["db2"] == got1["db2"]


def test_router_backward_without_b1_and_without_dx(dev):
    w = S.WORKLOADS["neox160m"]
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w, batch=2, seq=200)
    ds = np.random.default_rng(3).normal(size=400)
    announce("router backward without b1 / dx")
    Wn = dict(W, router_b1=None)
    got = _run_router_backward(dev, x, Wn, ds, with_b1=False)
    assert got["db1"] is None and got["dx"] is None
    _check_router_backward(w, Wn, x, ds, got, with_b1=False)


def test_router_backward_empty_writes_zeros(dev):
    w = S.WORKLOADS["neox160m"]
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w, batch=1, seq=8)[:, :0].contiguous()
    announce("router backward n = 0")
    got = _run_router_backward(dev, x, W, np.zeros(0))
    assert np.all(got["dw1"] == 0) and np.all(got["db1"] == 0) and np.all(got["dw2"] == 0) and got["db2"] == 0


@pytest.mark.parametrize("name", ["neox160m", "qwen05b"])
def test_router_backward_full_size(dev, name):
    w = S.WORKLOADS[name]
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w)
    n = w.batch * w.seq
    ds = np.random.default_rng(11).normal(size=n) * 1e-3
    announce(f"full-size router backward {name} n={n}")
    dx0 = torch.zeros_like(x)
    got = _run_router_backward(dev, x, W, ds, dx0=dx0)
    amb = _check_router_backward(w, W, x, ds, got, dx0=dx0)
    print(f"ambiguous hidden units: {amb}", flush=True)
