"""Analytic work model of the depth-sparse stack: the FLOPs and bytes the
method must compute or move, used for roofline fractions and the FLOP ratio.

Only the layer stack is counted (no embedding, no LM head): the normalized
FLOPs of the paper's tables (sparse over dense) are layer-stack savings.
A layer keeping k of T tokens per sequence costs
  projections: 2 B k [d (Hq + 2 Hkv) hd + Hq hd d + m d f], m = 2 (GELU) or 3 (SwiGLU);
  attention:   4 hd Hq B k (k + 1) / 2 (causal, diagonal included);
  router:      2 B T (d d_r + d_r) (sparse layers only).
"""
from __future__ import annotations

from typing import Sequence

NEOX = "neox_parallel"


def proj_flops(w, B: int, k: int) -> float:
    m = 2 if w.block == NEOX else 3
    d, hd = w.d_model, w.head_dim
    per_token = d * (w.n_heads + 2 * w.n_kv_heads) * hd + w.n_heads * hd * d + m * d * w.d_ff
    return 2.0 * B * k * per_token


def attn_flops(w, B: int, k: int) -> float:
    return 4.0 * w.head_dim * w.n_heads * B * k * (k + 1) / 2.0


def router_flops(w, B: int, T: int) -> float:
    return 2.0 * B * T * (w.d_model * w.d_router + w.d_router)


def layer_flops(w, B: int, T: int, k: int, sparse: bool = True) -> float:
    f = proj_flops(w, B, k) + attn_flops(w, B, k)
    return f + (router_flops(w, B, T) if sparse else 0.0)


def stack_flops(w, B: int, T: int, ks: Sequence[int], sparse: bool = True) -> float:
    return sum(layer_flops(w, B, T, k, sparse) for k in ks)


def normalized_flops(w, T: int, ks: Sequence[int]) -> float:
    """Sparse stack FLOPs over dense stack FLOPs (the paper's cost metric)."""
    return stack_flops(w, 1, T, ks, True) / stack_flops(w, 1, T, [T] * len(ks), False)


# ---- per-launch algorithmic work of the individual kernels (one layer) ----

def gemm_down_flops(w, B: int, k: int) -> float:
    """The last GEMM of a layer: [attn | act] . [W_o | W_down]^T (NeoX, fused) or act . W_down^T (Qwen)."""
    d, f = w.d_model, w.d_ff
    K = w.n_heads * w.head_dim + f if w.block == NEOX else f
    return 2.0 * B * k * d * K


def router_bytes(w, B: int, T: int) -> float:
    eb = 4 if w.dtype == "f32" else 2
    return eb * B * T * w.d_model + 4.0 * B * T


def sim_bytes(w, B: int, T: int) -> float:
    eb = 4 if w.dtype == "f32" else 2
    return 2.0 * eb * B * T * w.d_model


def topk_bytes(w, B: int, T: int, k: int) -> float:
    """Scores read, kept positions written."""
    return 4.0 * B * T + 4.0 * B * k


def norm_bytes(w, B: int, k: int) -> float:
    """Gather + normalisation kernels of one layer: NeoX reads each kept row once
    and writes LN1 and LN2 of it; Qwen writes RMS1 of the kept row, then reads h
    and writes RMS2(h). Plus the kept positions."""
    eb = 4 if w.dtype == "f32" else 2
    rows = eb * B * k * w.d_model
    return (3.0 if w.block == NEOX else 4.0) * rows + 4.0 * B * k


def gate_grad_bytes(w, B: int, T: int, k: int) -> float:
    """Gate score gradient: dy, x_in and x_out rows of the kept tokens and
    their scores and positions read; the [B, T] score gradient written."""
    eb = 4 if w.dtype == "f32" else 2
    return 3.0 * eb * B * k * w.d_model + 8.0 * B * k + 4.0 * B * T


def router_bwd_bytes(w, n: int) -> float:
    """Router backward over n tokens: x and dscore read, dx read and written
    (accumulated), W1 and w2 read, the fp32 weight gradients written."""
    eb = 4 if w.dtype == "f32" else 2
    d, dr = w.d_model, w.d_router
    return eb * n * d + 4.0 * n + 2.0 * eb * n * d + eb * dr * (d + 2) + 4.0 * (dr * d + 2 * dr + 1)


def router_bwd_flops(w, n: int) -> float:
    """Three n x d x d_r contractions: the hidden units recomputed, dW1, dx."""
    return 6.0 * n * w.d_model * w.d_router


def align_hidden_bytes(w, n: int) -> float:
    """Eq. 9 summand over n tokens: both hidden rows read."""
    eb = 4 if w.dtype == "f32" else 2
    return 2.0 * eb * n * w.d_model


def kl_align_bytes(eb: int, rows: int, classes: int) -> float:
    """Eq. 10 over rows of logits: both logit rows read, one float written."""
    return 2.0 * eb * rows * classes + 4.0 * rows


def layer_weight_bytes(w) -> float:
    """One layer's weights in the workload's storage format (projections,
    router, norms and biases)."""
    eb = 4 if w.dtype == "f32" else 2
    m = 2 if w.block == NEOX else 3
    d, hd = w.d_model, w.head_dim
    proj = d * (w.n_heads + 2 * w.n_kv_heads) * hd + w.n_heads * hd * d + m * d * w.d_ff
    router = w.d_router * d + 2 * w.d_router
    norms = (4 if w.block == NEOX else 2) * d
    qkv_bias = (w.n_heads + 2 * w.n_kv_heads) * hd  # both families bias the QKV projection
    biases = qkv_bias + (2 * d + w.d_ff if w.block == NEOX else 0)
    return float(eb * (proj + router + norms + biases))


def decode_step_bytes(w, B: int, cache_lens) -> float:
    """HBM bytes one decode step must move: every layer's weights once, the
    keys and values of every cached kept token (cache_lens: [L][B] lengths
    read by the step), and the B new rows in and out of each layer."""
    eb = 4 if w.dtype == "f32" else 2
    kv = sum(sum(lb) for lb in cache_lens) * 2.0 * w.n_kv_heads * w.head_dim * eb
    rows = len(cache_lens) * 2.0 * B * w.d_model * eb
    return len(cache_lens) * layer_weight_bytes(w) + kv + rows


def kind_work(w, kind: str, B: int, T: int, k: int):
    """(work, unit) of one layer's launches of a kernel kind: flops for the
    MFMA kernels, bytes for the streaming ones; None for kinds not modelled."""
    d, hd, f = w.d_model, w.head_dim, w.d_ff
    dq, dkv = w.n_heads * hd, w.n_kv_heads * hd
    M = B * k
    if kind == "gemm_qkv":
        return 2.0 * M * d * (dq + 2 * dkv), "flop"
    if kind == "gemm_up":
        return 2.0 * M * d * f * (1 if w.block == NEOX else 2), "flop"
    if kind == "gemm_o":
        return 2.0 * M * dq * d, "flop"
    if kind == "gemm_down":
        return gemm_down_flops(w, B, k), "flop"
    if kind == "attn":
        return attn_flops(w, B, k), "flop"
    if kind == "router":
        return router_bytes(w, B, T), "byte"
    if kind == "topk":
        return topk_bytes(w, B, T, k), "byte"
    if kind == "norm":
        return norm_bytes(w, B, k), "byte"
    if kind == "sim":
        return sim_bytes(w, B, T), "byte"
    return None
