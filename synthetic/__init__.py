"""Seeded synthetic workloads for the depth-sparse layer stack.

This module only draws numbers and describes shapes. It holds none of the
method's arithmetic (no similarity, allocation, routing or layer maths), so the
CPU oracle and the HIP path can both be fed from it without sharing code.

Every tensor is drawn on the CPU from ``torch.Generator`` seeds so that the
values are identical on any machine. Floating-point values are drawn in fp32
and then rounded once to the workload dtype; the oracle widens those exact
values to fp64.

Value distributions (the paper releases no weights or calibration data):

* hidden states x ~ N(0, 0.02);
* every weight matrix and bias ~ N(0, 0.02);
* norm gains 1 + N(0, 0.02), LayerNorm shifts N(0, 0.02);
* router: W1 [d_r, d] and b1 [d_r] ~ N(0, 0.02), w2 [d_r] ~ N(0, 0.02), b2 = 0.

Seeds: x uses 1234 (+ an offset for extra batches); layer l's block weights use
1000 + l; layer l's router uses 2000 + l.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional

import numpy as np
import torch

NEOX = "neox_parallel"
QWEN = "qwen_seq"

X_SEED = 1234
LAYER_SEED = 1000
ROUTER_SEED = 2000
STD = 0.02


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape and routing settings of one synthetic stack."""

    name: str
    block: str            # NEOX (parallel residual, LayerNorm, GELU) or QWEN (sequential, RMSNorm, SwiGLU)
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    d_ff: int
    rotary_dims: int
    rope_theta: float
    norm_eps: float
    d_router: int
    batch: int
    seq: int
    dtype: str            # "f32" or "bf16"
    # Retention source: either fixed ratios, or a similarity profile plus the
    # allocator's target mean t and temperature tau.
    retention: Optional[tuple] = None
    similarity: Optional[tuple] = None
    target: Optional[float] = None
    tau: Optional[float] = None

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    @property
    def d_qkv(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def d_attn(self) -> int:
        return self.n_heads * self.head_dim

    @property
    def d_up(self) -> int:
        """Rows of the up projection: f for GELU, 2f (gate rows first) for SwiGLU."""
        return self.d_ff if self.block == NEOX else 2 * self.d_ff

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


def _linspace(a, b, n):
    return tuple(float(v) for v in np.linspace(a, b, n))


# The workloads. Shapes follow the public configurations of the model
# families the paper evaluates (GPT-NeoX, Qwen2.5); weights are random.
WORKLOADS: Dict[str, Workload] = {
    # Tiny single routed layer, fp32, NeoX-style block at d=128.
    "tiny_neox_f32": Workload(
        "tiny_neox_f32", NEOX, 1, 128, 4, 4, 32, 512, 8, 10000.0, 1e-5, 32,
        2, 64, "f32", retention=(0.5,)),
    # The same tiny size with a Qwen-style block (GQA 2:1, RMSNorm, SwiGLU, full rotary).
    "tiny_qwen_f32": Workload(
        "tiny_qwen_f32", QWEN, 1, 128, 4, 2, 32, 512, 32, 1e6, 1e-6, 32,
        2, 64, "f32", retention=(0.5,)),
    # GPT-NeoX-160M shape: 12 x 768, 12 heads of 64, FFN 3072, rotary 25 %.
    "neox160m": Workload(
        "neox160m", NEOX, 12, 768, 12, 12, 64, 3072, 16, 10000.0, 1e-5, 32,
        8, 2048, "bf16", similarity=_linspace(0.3, 0.9, 12), target=0.6, tau=0.25),
    # Qwen2.5-0.5B shape: 24 x 896, 14 q / 2 kv heads of 64, SwiGLU 4864.
    "qwen05b": Workload(
        "qwen05b", QWEN, 24, 896, 14, 2, 64, 4864, 64, 1e6, 1e-6, 32,
        8, 4096, "bf16", similarity=_linspace(0.5, 0.95, 24), target=0.5, tau=0.05),
    # GPT-NeoX-1.4B shape: 24 x 2048, 16 heads of 128, FFN 8192, rotary 25 %.
    "neox14b": Workload(
        "neox14b", NEOX, 24, 2048, 16, 16, 128, 8192, 32, 10000.0, 1e-5, 32,
        4, 2048, "bf16", retention=(0.5,) * 24),
    # The paper's own evaluation models at uniform retention (Tables 1-2):
    # GPT-NeoX-130M (its shape is not given; the 12 x 768 GPT-NeoX shape is
    # used) on 16 sequences of 1024 tokens, and Qwen2.5-1.5B (28 x 1536,
    # 12 q / 2 kv heads of 128, SwiGLU 8960) on 8 sequences of 2048.
    "neox130m": Workload(
        "neox130m", NEOX, 12, 768, 12, 12, 64, 3072, 16, 10000.0, 1e-5, 32,
        16, 1024, "bf16", retention=(0.8,) * 12),
    "qwen15b": Workload(
        "qwen15b", QWEN, 28, 1536, 12, 2, 128, 8960, 128, 1e6, 1e-6, 32,
        8, 2048, "bf16", retention=(0.8,) * 28),
    # Qwen2.5-7B shape: 28 x 3584, 28 q / 4 kv heads of 128, SwiGLU 18944.
    # Retention comes from similarities measured on the stack itself.
    "qwen7b": Workload(
        "qwen7b", QWEN, 28, 3584, 28, 4, 128, 18944, 128, 1e6, 1e-6, 32,
        4, 8192, "bf16", target=0.5, tau=0.05),
}


def _normal(gen: torch.Generator, shape, std=STD, mean=0.0) -> torch.Tensor:
    return torch.randn(*shape, generator=gen, dtype=torch.float32) * std + mean


def hidden_states(w: Workload, seed_offset: int = 0, batch: Optional[int] = None,
                  seq: Optional[int] = None) -> torch.Tensor:
    """x [B, T, d] ~ N(0, 0.02), rounded to the workload dtype (CPU tensor)."""
    g = torch.Generator().manual_seed(X_SEED + seed_offset)
    b = w.batch if batch is None else batch
    t = w.seq if seq is None else seq
    return _normal(g, (b, t, w.d_model)).to(w.torch_dtype)


def layer_weights(w: Workload, layer: int) -> Dict[str, Optional[torch.Tensor]]:
    """Block and router weights of one layer (CPU tensors in the workload dtype).

    Layouts (row-major, ``[out, in]``):
      w_qkv [(Hq + 2 Hkv) hd, d] in Q | K | V block order, b_qkv [(Hq + 2 Hkv) hd];
      w_o [d, Hq hd], b_o [d] (NeoX only);
      w_up [f, d] with b_up (NeoX), or [2f, d] gate rows then up rows (Qwen);
      w_down [d, f] with b_down (NeoX only);
      norm1_w/norm2_w [d], norm1_b/norm2_b [d] (LayerNorm only);
      router_w1 [d_r, d], router_b1 [d_r], router_w2 [d_r]; router_b2 is a float.
    """
    g = torch.Generator().manual_seed(LAYER_SEED + layer)
    d, f = w.d_model, w.d_ff
    neox = w.block == NEOX
    out: Dict[str, Optional[torch.Tensor]] = {}
    out["norm1_w"] = _normal(g, (d,), mean=1.0)
    out["norm1_b"] = _normal(g, (d,)) if neox else None
    out["norm2_w"] = _normal(g, (d,), mean=1.0)
    out["norm2_b"] = _normal(g, (d,)) if neox else None
    out["w_qkv"] = _normal(g, (w.d_qkv, d))
    out["b_qkv"] = _normal(g, (w.d_qkv,))
    out["w_o"] = _normal(g, (d, w.d_attn))
    out["b_o"] = _normal(g, (d,)) if neox else None
    out["w_up"] = _normal(g, (w.d_up, d))
    out["b_up"] = _normal(g, (f,)) if neox else None
    out["w_down"] = _normal(g, (d, f))
    out["b_down"] = _normal(g, (d,)) if neox else None
    gr = torch.Generator().manual_seed(ROUTER_SEED + layer)
    out["router_w1"] = _normal(gr, (w.d_router, d))
    out["router_b1"] = _normal(gr, (w.d_router,))
    out["router_w2"] = _normal(gr, (w.d_router,))
    for key, val in list(out.items()):
        if val is not None:
            out[key] = val.to(w.torch_dtype)
    out["router_b2"] = 0.0
    return out


def stack_weights(w: Workload, layers: Optional[List[int]] = None):
    ids = range(w.n_layers) if layers is None else layers
    return [layer_weights(w, l) for l in ids]


def router_scores_with_ties(batch: int, seq: int, levels: int, seed: int) -> torch.Tensor:
    """fp32 scores drawn from `levels` distinct values, for tie-heavy top-k cases."""
    g = torch.Generator().manual_seed(seed)
    q = torch.randint(0, levels, (batch, seq), generator=g)
    return (q.to(torch.float32) - levels / 2) * 0.25


def random_scores(batch: int, seq: int, seed: int) -> torch.Tensor:
    g = torch.Generator().manual_seed(seed)
    return torch.randn(batch, seq, generator=g, dtype=torch.float32)


def fixed_retention(w: Workload) -> Optional[List[float]]:
    return None if w.retention is None else list(w.retention)


def rows_per_sequence_bytes(w: Workload) -> int:
    """Bytes of one hidden row in the workload dtype."""
    return w.d_model * (4 if w.dtype == "f32" else 2)


def approx_param_bytes(w: Workload) -> int:
    eb = 4 if w.dtype == "f32" else 2
    per = (w.d_qkv * w.d_model + w.d_model * w.d_attn + w.d_up * w.d_model
           + w.d_model * w.d_ff)
    return per * w.n_layers * eb


__all__ = [
    "Workload", "WORKLOADS", "NEOX", "QWEN", "hidden_states", "layer_weights",
    "stack_weights", "router_scores_with_ties", "random_scores", "fixed_retention",
]
