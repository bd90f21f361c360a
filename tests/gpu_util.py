"""Helpers shared by the GPU parity tests (no method arithmetic here)."""
import sys

import numpy as np
import torch

import paper_2607_21291_amd as P
import synthetic as S
from oracle import adadsf_oracle as O

U32 = 2.0 ** -24  # unit roundoff of fp32


def announce(msg: str):
    """Name the case on stdout before a GPU step, so a fault names what ran."""
    print(f"\n[gpu case] {msg}", flush=True)
    sys.stdout.flush()


def to_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().to(torch.float64).cpu().numpy()


def rel_inf(a, b) -> float:
    """max|a - b| / max|b| (infinity-norm relative error)."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.max(np.abs(b))
    return float(np.max(np.abs(a - b)) / (den if den > 0 else 1.0))


def desc_dict(w: S.Workload) -> dict:
    return dict(block=w.block, n_heads=w.n_heads, n_kv_heads=w.n_kv_heads, head_dim=w.head_dim, d_ff=w.d_ff,
                rotary_dims=w.rotary_dims, rope_theta=w.rope_theta, norm_eps=w.norm_eps)


def make_desc(w: S.Workload) -> P.LayerDesc:
    return P.make_desc(w.block, w.d_model, w.n_heads, w.n_kv_heads, w.head_dim, w.d_ff, w.rotary_dims,
                       w.d_router, w.norm_eps, w.rope_theta)


def dtype_code(w: S.Workload) -> int:
    return P.F32 if w.dtype == "f32" else P.BF16


def workspace(w: S.Workload, B: int, T: int, k_max: int, dev, with_sim=False) -> torch.Tensor:
    n = P.workspace_size(make_desc(w), dtype_code(w), B, T, k_max, with_sim)
    assert n > 0
    return torch.empty(n, dtype=torch.uint8, device=dev)


def router_bound(x, W, dtype: str) -> np.ndarray:
    """Rounding-error bound for the router score computed in fp32.

    The hidden units are d-term fp32 dot products (exact products for bf16
    inputs), the score a d_r-term fp32 sum: for any summation order,
    |err| <= gamma_{d+d_r+4} * (|w2| . (|W1| |x| + |b1|) + |b2|), gamma_n = n u / (1 - n u).
    """
    x = np.abs(np.asarray(x, dtype=np.float64))
    w1 = np.abs(to_np(W["router_w1"]))
    b1 = np.abs(to_np(W["router_b1"])) if W.get("router_b1") is not None else 0.0
    w2 = np.abs(to_np(W["router_w2"]))
    n = x.shape[-1] + w1.shape[0] + 4
    gamma = n * U32 / (1 - n * U32)
    return gamma * ((x @ w1.T + b1) @ w2 + abs(W.get("router_b2", 0.0))) + 1e-30


# ---------------------------------------------------------------- layers

TOL = {"f32": 1e-4, "bf16": 2e-2}

# Small bf16 shapes that still span several GEMM tiles and ragged tails.
SMALL = {
    "neox_bf16_small": S.WORKLOADS["neox160m"].replace(
        name="neox_bf16_small", n_layers=2, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64, d_ff=1024,
        rotary_dims=16, batch=2, seq=300),
    "qwen_bf16_small": S.WORKLOADS["qwen05b"].replace(
        name="qwen_bf16_small", n_layers=2, d_model=256, n_heads=4, n_kv_heads=2, head_dim=64, d_ff=512,
        rotary_dims=64, batch=2, seq=300),
    "neox_bf16_hd128": S.WORKLOADS["neox14b"].replace(
        name="neox_bf16_hd128", n_layers=2, d_model=512, n_heads=4, n_kv_heads=4, head_dim=128, d_ff=1024,
        rotary_dims=32, batch=2, seq=200),
    "qwen_bf16_hd128": S.WORKLOADS["qwen7b"].replace(
        name="qwen_bf16_hd128", n_layers=2, d_model=512, n_heads=8, n_kv_heads=2, head_dim=128, d_ff=768,
        rotary_dims=128, batch=1, seq=257),
}


def workload(name):
    return S.WORKLOADS[name] if name in S.WORKLOADS else SMALL[name]


def run_layer(dev, w, W, x, k, flags=0, idx_in=None):
    B, T = x.shape[0], x.shape[1]
    dl = P.DeviceLayer(W, dev)
    xd = x.to(dev).contiguous()
    scores = torch.empty(B, T, dtype=torch.float32, device=dev)
    idx = torch.empty(B, max(k, 1), dtype=torch.int32, device=dev)
    ws = workspace(w, B, T, k, dev)
    dense = flags & P.FLAG_DENSE
    P.sparse_block_forward(make_desc(w), dl.weights, xd, k, ws, flags=flags,
                           scores_out=None if dense else scores,
                           idx_out=None if (dense or k == 0) else idx[:, :k],
                           idx_in=None if idx_in is None else idx_in.to(dev))
    torch.cuda.synchronize()
    if k > 0:  # a call that launches nothing leaves the status word as it was
        assert P.workspace_status(ws) == 0, "a stream-K wait gave up"
    return xd, scores, idx[:, :k]


def check_selection(ref_scores, bound, sc_gpu, idx_gpu, k):
    """Selection steps of the parity protocol, for every sequence.

    GPU scores within the fp32 bound of the oracle's; the oracle's Top-K of
    the GPU's scores equal to the GPU's indices; and, where the oracle's own
    scores select differently, every token in the difference has an oracle
    score within the score tolerance of the oracle's k-th score (its own
    bound plus the largest bound of the sequence), so only near-ties can
    change places."""
    assert np.all(np.abs(sc_gpu - ref_scores) <= bound)
    np.testing.assert_array_equal(idx_gpu, O.topk_select(sc_gpu, k))
    if k == 0:
        return
    idx_ref = O.topk_select(ref_scores, k)
    for b in range(ref_scores.shape[0]):
        diff = np.setxor1d(idx_ref[b], idx_gpu[b])
        if diff.size == 0:
            continue
        kth = np.min(ref_scores[b, idx_ref[b]])
        tol = bound[b, diff] + np.max(bound[b])
        assert np.all(np.abs(ref_scores[b, diff] - kth) <= tol), (b, diff)


def check_layer(w, W, x, y_gpu, scores_gpu, idx_gpu, k, sample=None, gate=False):
    """Layer protocol: router scores within the fp32 bound, the oracle's Top-K
    of the GPU's scores equal to the GPU's indices and any difference from
    the oracle's own selection confined to near-ties (every sequence),
    skipped rows bitwise unchanged (every sequence), and the kept rows
    against the oracle teacher-forced with the GPU's indices, for the
    sequences in `sample` (None: all of them). gate: the score-gated layer."""
    xs = to_np(x)
    sc = scores_gpu.cpu().numpy()
    ref_scores = O.router_scores(x, W["router_w1"], W["router_b1"], W["router_w2"], W["router_b2"])
    idx = idx_gpu.cpu().numpy().astype(np.int64)
    check_selection(ref_scores, router_bound(xs, W, w.dtype), sc, idx, k)
    y = to_np(y_gpu)
    B, T, _ = xs.shape
    kept = np.zeros((B, T), dtype=bool)
    for b in range(B):
        kept[b, idx[b]] = True
        np.testing.assert_array_equal(y[b][~kept[b]], xs[b][~kept[b]])
    for b in (range(B) if sample is None else sample):
        res = O.routed_layer(desc_dict(w), W, xs[b:b + 1], k, idx=idx[b:b + 1], gate=gate)
        upd = res["y"][0][kept[b]] - xs[b][kept[b]]
        assert update_err(y[b][kept[b]], xs[b][kept[b]], upd, w.dtype) < TOL[w.dtype]
        assert rel_inf(y[b], res["y"][0]) < TOL[w.dtype]


def storage_half_ulp(v, dtype: str) -> np.ndarray:
    """Half a unit in the last place of each value in the storage format (the
    largest error of rounding it to nearest): bf16 keeps 8 significant bits,
    fp32 24."""
    bits = 8 if dtype == "bf16" else 24
    v = np.abs(np.asarray(v, dtype=np.float64))
    e = np.floor(np.log2(np.where(v > 0, v, 1.0)))
    return np.where(v > 0, 2.0 ** (e - bits), 0.0)


def update_err(y, x, upd_ref, dtype: str) -> float:
    """Relative error of a layer's update as observed through its stored
    output: the GPU stores y = x + delta rounded to the storage format, so
    y - x carries that rounding (half an ulp of y) on top of the kernel's own
    error. Returns max(|(y - x) - delta_ref| - half_ulp(y), 0) / max|delta_ref|."""
    y, x, upd_ref = (np.asarray(a, dtype=np.float64) for a in (y, x, upd_ref))
    excess = np.maximum(np.abs((y - x) - upd_ref) - storage_half_ulp(y, dtype), 0.0)
    den = np.max(np.abs(upd_ref))
    return float(np.max(excess) / (den if den > 0 else 1.0)) if excess.size else 0.0
