"""Helpers shared by the GPU parity tests (no method arithmetic here)."""
import sys

import numpy as np
import torch

import paper_2607_21291_amd as P
import synthetic as S

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
