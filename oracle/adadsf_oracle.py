"""CPU oracle for the AdaDSF depth-sparse layer stack.

TEST INFRASTRUCTURE. Only the test suite, the smoke check and the benchmark's
CPU-baseline leg may import this module. The product (the HIP library and its
Python binding) never calls it. The two share no code: both are fed by the
seeded generators in ``synthetic``, which hold no part of the method's
arithmetic.

Everything is computed in float64 with plain numpy; inputs that were rounded
to bf16 or fp32 are widened exactly. Matrix products use numpy's matmul as a
library primitive. There is no blocking, fusion or reordering beyond what each
definition states, so each function can be checked against the paper by eye.

Paper: "Adaptive Depth Sparse Framework: Similarity-Driven Resource Allocation
for Pre-Trained LLMs" (AdaDSF).

Readings taken where the paper is silent or ambiguous (each also in the design doc):

* Eq. 4 is applied per token over the hidden dimension, then averaged over the
  calibration tokens; a zero product of norms is guarded by 1e-8.
* Eq. 8 can give r_i > 1. The default clip sets such layers to 1 and hands the
  excess back to the other layers in proportion to r'_j, so sum(r) = tL still
  holds.
* K_i = floor(r_i T) (Section 3.4) is evaluated as floor(r_i T + 1e-6). This
  guard absorbs fp64 representation error, e.g. floor(0.29 * 100) = 28.
* Top-K ties go to the lower position; the kept positions are returned in
  ascending order. -0.0 equals +0.0, and NaN ranks below every number.
* Masked selection is read as compaction. The block runs on the kept rows
  only, at their original positions, and kept tokens attend causally among
  kept tokens. Skipped rows pass through unchanged, and the block output is
  not gated by the router score.
* The block is each model family's own pre-norm block. NeoX uses a parallel
  residual, LayerNorm, exact-erf GELU and partial rotary. Qwen uses a
  sequential residual, RMSNorm, SwiGLU, full rotary and GQA. Eq. 3 is a
  post-norm schematic that matches neither model.
* The router reads the raw residual-stream row: score = w2 . ReLU(W1 x + b1) + b2.
* Eq. 9's softmax runs over the hidden dimension of each token, and its
  2-norm is taken over the layer's whole hidden-state tensor. Eq. 10 is
  evaluated per row of logits, with the classes on the last axis.
* Decoding is not treated by the paper. Per-sequence Top-K needs the whole
  sequence, so at decode time a new token is kept by a layer when its router
  score is at least a per-(layer, sequence) threshold; a kept token joins the
  layer's kept set at its original position and attends causally over it.
  Every step of the layer is causal, so decoding token by token with given
  keep decisions equals the stack over the whole sequence with the same kept
  sets (decode_stack and kept_set_stack below; the CPU tests check this).

Parity status: every function here is pinned by the CPU tests (closed forms,
invariants, brute force, and library cross-checks against torch and the
transformers GPT-NeoX / Qwen2 layers). The values against the paper's own
trained models are unpinned, because the paper publishes no weights or worked
examples.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
from scipy.special import erf

NEOX = "neox_parallel"
QWEN = "qwen_seq"

COS_EPS = 1e-8
K_GUARD = 1e-6


def f64(a) -> np.ndarray:
    """Widen a numpy array or CPU torch tensor to float64 exactly."""
    if hasattr(a, "detach"):
        a = a.detach().to("cpu")
        import torch  # local: the oracle itself needs torch only for this conversion
        a = a.to(torch.float64).numpy()
    return np.asarray(a, dtype=np.float64)


# ---------------------------------------------------------------------------
# Rounding to the storage formats (used where a result is stored, e.g. scatter)
# ---------------------------------------------------------------------------

def round_bf16(v: np.ndarray) -> np.ndarray:
    """Round float64 values to bfloat16 (8 significant bits), ties to even.

    Written from the format's definition: mantissa in [0.5, 1) from frexp,
    scaled to 8 bits, rounded half-to-even (numpy's rint), scaled back.
    Valid for the normal range of bf16, which is fp32's exponent range.
    """
    v = np.asarray(v, dtype=np.float64)
    m, e = np.frexp(v)
    q = np.rint(m * 256.0)
    return np.ldexp(q, e - 8)


def round_f32(v: np.ndarray) -> np.ndarray:
    return np.asarray(v, dtype=np.float64).astype(np.float32).astype(np.float64)


def round_to(dtype: str, v: np.ndarray) -> np.ndarray:
    return round_bf16(v) if dtype == "bf16" else round_f32(v)


# ---------------------------------------------------------------------------
# Section 3.3, Eq. 4: cosine similarity between a layer's input and output
# ---------------------------------------------------------------------------

def token_cosine(x_in, x_out, eps: float = COS_EPS) -> np.ndarray:
    """Per-token cosine between input and output rows (Eq. 4 applied to one token).

    x_in, x_out: [..., d]. Returns [...]. A product of norms below eps is
    replaced by eps, so an all-zero row gives 0.
    """
    a = f64(x_in)
    c = f64(x_out)
    dot = np.sum(a * c, axis=-1)
    na = np.sqrt(np.sum(a * a, axis=-1))
    nc = np.sqrt(np.sum(c * c, axis=-1))
    return dot / np.maximum(na * nc, eps)


def similarity_accumulate(x_in, x_out) -> Tuple[float, int]:
    """(sum of per-token cosines, number of tokens) for one layer on one batch."""
    cos = token_cosine(x_in, x_out)
    return float(np.sum(cos)), int(cos.size)


def layer_similarity(sum_cos: float, n_tokens: int) -> float:
    """s_i: the mean per-token cosine over the calibration tokens (Eq. 4)."""
    return sum_cos / n_tokens


# ---------------------------------------------------------------------------
# Section 3.3, Eqs. 5-8: similarity -> layer-wise retention ratios
# ---------------------------------------------------------------------------

def retention_from_similarity(s: Sequence[float], t: float, tau: Optional[float],
                              beta: float = 10.0, clip: str = "budget") -> np.ndarray:
    """Retention ratio r_i per layer from similarities s_i.

    Step 1 (Eq. 5): w~_i = exp((s_i - max s) / tau), w_i = w~_i / sum_j w~_j.
    Step 2 (Eq. 6): z_i = beta * (mean_j w_j - w_i).
    Step 3 (Eq. 7): r'_i = 0.05 + 0.9 * sigmoid(z_i).
    Step 4 (Eq. 8): r_i = t L r'_i / sum_j r'_j, so sum_i r_i = t L.

    tau=None is the ablation without the similarity temperature: uniform r = t.
    clip="budget" caps r_i at 1 and hands the excess back to the other layers
    in proportion to r'_j until no layer exceeds 1. clip="plain" only caps at 1.
    clip="none" returns Eq. 8 as written.
    """
    s = f64(s)
    L = s.size
    if tau is None:
        return np.full(L, float(t))
    w_tilde = np.exp((s - np.max(s)) / tau)
    w = w_tilde / np.sum(w_tilde)
    z = beta * (np.mean(w) - w)
    r_prime = 0.05 + 0.9 * (1.0 / (1.0 + np.exp(-z)))
    r = (t * L / np.sum(r_prime)) * r_prime
    if clip == "none":
        return r
    if clip == "plain":
        return np.minimum(r, 1.0)
    if clip != "budget":
        raise ValueError(f"unknown clip mode {clip!r}")
    capped = np.zeros(L, dtype=bool)
    while np.any(r > 1.0):
        capped |= r > 1.0
        free = ~capped
        budget = t * L - np.count_nonzero(capped)
        r = np.where(capped, 1.0, 0.0)
        if np.any(free):
            r[free] = budget * r_prime[free] / np.sum(r_prime[free])
    return r


def k_from_retention(r: float, T: int, rounding: str = "floor") -> int:
    """Kept tokens per sequence: K = floor(r T) (Section 3.4), with a 1e-6 guard.

    rounding="ceil" gives ceil(r T - 1e-6) instead. The result is clamped to [0, T].
    """
    x = float(r) * T
    if rounding == "floor":
        k = math.floor(x + K_GUARD)
    elif rounding == "ceil":
        k = math.ceil(x - K_GUARD)
    else:
        raise ValueError(f"unknown rounding {rounding!r}")
    return int(min(max(k, 0), T))


# ---------------------------------------------------------------------------
# Section 3.4: router, Top-K selection, masked selection / residual bypass
# ---------------------------------------------------------------------------

def router_scores(x, w1, b1, w2, b2: float = 0.0) -> np.ndarray:
    """Token importance of a two-layer MLP router: w2 . ReLU(W1 x + b1) + b2.

    x: [B, T, d]; w1: [d_r, d]; b1: [d_r] or None; w2: [d_r]. Returns [B, T].
    """
    x = f64(x)
    hid = x @ f64(w1).T
    if b1 is not None:
        hid = hid + f64(b1)
    hid = np.maximum(hid, 0.0)
    return hid @ f64(w2) + float(b2)


def topk_select(scores, k: int) -> np.ndarray:
    """Top-K_i positions of each sequence, returned in ascending position order.

    Order of preference: larger score first, then lower position. Returns
    int64 [B, k]. Uses a lexicographic sort (library primitive) on
    (-score, position); numpy treats -0.0 == +0.0 and sorts NaN last.
    """
    sc = f64(scores)
    B, T = sc.shape
    if not 0 <= k <= T:
        raise ValueError("k out of range")
    out = np.empty((B, k), dtype=np.int64)
    pos = np.arange(T)
    for b in range(B):
        order = np.lexsort((pos, -sc[b]))
        out[b] = np.sort(order[:k])
    return out


def gather_rows(x, idx) -> np.ndarray:
    """x^ = the kept rows x[b, idx[b, j]] (masked selection as compaction)."""
    x = f64(x)
    idx = np.asarray(idx)
    return np.stack([x[b, idx[b]] for b in range(x.shape[0])])


def scatter_residual(x, delta, idx, dtype: Optional[str] = None) -> np.ndarray:
    """y = x, with y[b, idx[b, j]] = x[b, idx[b, j]] + delta[b, j].

    Skipped rows are untouched. With dtype given, the kept rows are rounded
    to that storage format (bf16 or f32) after the exact add.
    """
    y = f64(x).copy()
    delta = f64(delta)
    idx = np.asarray(idx)
    for b in range(y.shape[0]):
        v = y[b, idx[b]] + delta[b]
        y[b, idx[b]] = v if dtype is None else round_to(dtype, v)
    return y


# ---------------------------------------------------------------------------
# Section 3.1, Eqs. 1-2: the decoder block run on the kept tokens
# ---------------------------------------------------------------------------

def layer_norm(x, w, b, eps: float) -> np.ndarray:
    x = f64(x)
    mu = np.mean(x, axis=-1, keepdims=True)
    var = np.mean((x - mu) ** 2, axis=-1, keepdims=True)
    y = (x - mu) / np.sqrt(var + eps) * f64(w)
    return y if b is None else y + f64(b)


def rms_norm(x, w, eps: float) -> np.ndarray:
    x = f64(x)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * f64(w)


def gelu(x) -> np.ndarray:
    """Exact GELU: x * Phi(x), Phi the standard normal CDF."""
    x = f64(x)
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def silu(x) -> np.ndarray:
    x = f64(x)
    return x / (1.0 + np.exp(-x))


def rope(x, pos, rotary_dims: int, theta: float) -> np.ndarray:
    """Rotary position embedding (rotate-half form) on the first rotary_dims dims.

    x: [n, H, hd]; pos: [n] original token positions. For i < R/2 the pair
    (x_i, x_{i+R/2}) is rotated by the angle pos * theta^(-2i/R).
    """
    x = f64(x)
    R = rotary_dims
    half = R // 2
    inv_freq = theta ** (-(2.0 * np.arange(half)) / R)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]
    cos = np.cos(ang)[:, None, :]
    sin = np.sin(ang)[:, None, :]
    out = x.copy()
    x1 = x[..., :half]
    x2 = x[..., half:R]
    out[..., :half] = x1 * cos - x2 * sin
    out[..., half:R] = x2 * cos + x1 * sin
    return out


def causal_attention(q, k, v) -> np.ndarray:
    """Eq. 1 with a causal mask over the given (kept) tokens.

    q: [n, Hq, hd]; k, v: [n, Hkv, hd]; q head h reads kv head h // (Hq / Hkv).
    Token j attends to tokens j' <= j. Returns [n, Hq * hd].
    """
    q, k, v = f64(q), f64(k), f64(v)
    n, Hq, hd = q.shape
    Hkv = k.shape[1]
    group = Hq // Hkv
    out = np.zeros((n, Hq, hd))
    mask = np.triu(np.ones((n, n), dtype=bool), 1)
    for h in range(Hq):
        kh = h // group
        s = (q[:, h, :] @ k[:, kh, :].T) / math.sqrt(hd)
        s[mask] = -np.inf
        s = s - np.max(s, axis=1, keepdims=True)
        p = np.exp(s)
        p = p / np.sum(p, axis=1, keepdims=True)
        out[:, h, :] = p @ v[:, kh, :]
    return out.reshape(n, Hq * hd)


def block_delta(desc: Dict, W: Dict, xc, pos) -> np.ndarray:
    """Residual update produced by one decoder block on one sequence's kept rows.

    xc: [n, d] kept rows in position order; pos: [n] their original positions.
    Returns delta [n, d] such that the block's output rows are xc + delta.
    desc keys: block, n_heads, n_kv_heads, head_dim, d_ff, rotary_dims,
    rope_theta, norm_eps.
    """
    xc = f64(xc)
    n = xc.shape[0]
    Hq, Hkv, hd = desc["n_heads"], desc["n_kv_heads"], desc["head_dim"]
    f = desc["d_ff"]
    eps = desc["norm_eps"]
    neox = desc["block"] == NEOX

    def linear(inp, wname, bname=None):
        y = inp @ f64(W[wname]).T
        b = W.get(bname) if bname else None
        return y if b is None else y + f64(b)

    a = layer_norm(xc, W["norm1_w"], W["norm1_b"], eps) if neox else rms_norm(xc, W["norm1_w"], eps)
    qkv = linear(a, "w_qkv", "b_qkv")
    q = qkv[:, :Hq * hd].reshape(n, Hq, hd)
    k = qkv[:, Hq * hd:(Hq + Hkv) * hd].reshape(n, Hkv, hd)
    v = qkv[:, (Hq + Hkv) * hd:].reshape(n, Hkv, hd)
    q = rope(q, pos, desc["rotary_dims"], desc["rope_theta"])
    k = rope(k, pos, desc["rotary_dims"], desc["rope_theta"])
    attn = causal_attention(q, k, v)
    ao = linear(attn, "w_o", "b_o")
    if neox:
        m = layer_norm(xc, W["norm2_w"], W["norm2_b"], eps)
        mo = linear(gelu(linear(m, "w_up", "b_up")), "w_down", "b_down")
    else:
        h = xc + ao
        m = rms_norm(h, W["norm2_w"], eps)
        gu = linear(m, "w_up")
        mo = linear(silu(gu[:, :f]) * gu[:, f:], "w_down")
    return ao + mo


# ---------------------------------------------------------------------------
# Section 3.4: the sparse module (router -> Top-K -> block on kept rows -> bypass)
# ---------------------------------------------------------------------------

def routed_layer(desc: Dict, W: Dict, x, k: int, idx=None,
                 out_dtype: Optional[str] = None, gate: bool = False) -> Dict[str, np.ndarray]:
    """One sparse layer. Returns y, scores, idx and delta (kept rows, [B, k, d]).

    idx given: teacher-forced selection (the router still scores every token).
    out_dtype given: the kept rows of y are rounded to that storage format.
    gate: sigmoid(score) scales each kept token's update, so the loss reaches
    the router scores through a gradient (Section 3.4, read MoD-style);
    `delta` is then the ungated update.
    """
    x = f64(x)
    B, T, _ = x.shape
    scores = router_scores(x, W["router_w1"], W["router_b1"], W["router_w2"],
                           W.get("router_b2", 0.0))
    if idx is None:
        idx = topk_select(scores, k)
    idx = np.asarray(idx, dtype=np.int64)
    xc = gather_rows(x, idx)
    delta = np.stack([block_delta(desc, W, xc[b], idx[b]) for b in range(B)]) if k > 0 \
        else np.zeros((B, 0, x.shape[2]))
    if gate:
        g = sigmoid(np.stack([scores[b, idx[b]] for b in range(B)]))
        y = scatter_residual(x, g[..., None] * delta, idx, out_dtype)
    else:
        y = scatter_residual(x, delta, idx, out_dtype)
    return {"y": y, "scores": scores, "idx": idx, "delta": delta}


def dense_layer(desc: Dict, W: Dict, x) -> np.ndarray:
    """The unmodified layer on every token: x + block(x) at positions 0..T-1."""
    x = f64(x)
    B, T, _ = x.shape
    pos = np.arange(T)
    return np.stack([x[b] + block_delta(desc, W, x[b], pos) for b in range(B)])


def stack_forward(desc: Dict, Ws: List[Dict], x, ks: Sequence[int],
                  out_dtype: Optional[str] = None) -> Tuple[np.ndarray, List[np.ndarray]]:
    """Depth-sparse stack: x <- routed_layer_l(x, k_l) for l = 0..L-1.

    Returns the final hidden states and the kept positions of every layer.
    """
    x = f64(x)
    idxs = []
    for W, k in zip(Ws, ks):
        res = routed_layer(desc, W, x, int(k), out_dtype=out_dtype)
        x = res["y"]
        idxs.append(res["idx"])
    return x, idxs


def calibrate_similarity(desc: Dict, Ws: List[Dict], x) -> np.ndarray:
    """Dense calibration pass: s_l for every layer (Eq. 4 on the dense stack)."""
    x = f64(x)
    s = []
    for W in Ws:
        y = dense_layer(desc, W, x)
        tot, n = similarity_accumulate(x, y)
        s.append(layer_similarity(tot, n))
        x = y
    return np.asarray(s)


# ---------------------------------------------------------------------------
# Section 3.4, training side: gradients along the router-score pathway
# ---------------------------------------------------------------------------

def sigmoid(v) -> np.ndarray:
    """Logistic function 1 / (1 + e^-v)."""
    v = f64(v)
    return 1.0 / (1.0 + np.exp(-v))


def gate_score_grad(dy, x_in, x_out, scores, idx) -> np.ndarray:
    """dL/ds for every token of a gated routed layer (routed_layer(gate=True)).

    dy: gradient of the loss with respect to the layer output, [B, T, d];
    x_in, x_out: the layer's input and output; scores [B, T]; idx [B, k].
    A kept token p has y_p = x_p + sigmoid(s_p) delta_p, so
    dL/ds_p = sigmoid'(s_p) <dy_p, delta_p> = (1 - sigmoid(s_p)) <dy_p, y_p - x_p>.
    The selection itself is piecewise constant in the scores: skipped tokens
    get 0. Returns [B, T].
    """
    dy, x_in, x_out, sc = f64(dy), f64(x_in), f64(x_out), f64(scores)
    idx = np.asarray(idx)
    out = np.zeros(sc.shape)
    for b in range(sc.shape[0]):
        p = idx[b]
        out[b, p] = (1.0 - sigmoid(sc[b, p])) * np.sum(dy[b, p] * (x_out[b, p] - x_in[b, p]), axis=-1)
    return out


def router_backward(x, w1, b1, w2, dscore) -> Dict[str, np.ndarray]:
    """Gradients through score = w2 . ReLU(W1 x + b1) + b2 given dL/dscore.

    x: [..., d] tokens, dscore: [...] (same leading shape). Returns dw1 [d_r, d],
    db1 [d_r], dw2 [d_r], db2 (scalar) and dx [..., d] (the router's share of
    the input gradient). The ReLU's derivative at 0 is taken as 0.
    """
    x = f64(x)
    d = x.shape[-1]
    xt = x.reshape(-1, d)
    ds = f64(dscore).reshape(-1)
    w1, w2 = f64(w1), f64(w2)
    z = xt @ w1.T
    if b1 is not None:
        z = z + f64(b1)
    h = np.maximum(z, 0.0)
    dz = ds[:, None] * w2[None, :] * (z > 0.0)
    return {"dw1": dz.T @ xt, "db1": dz.sum(axis=0), "dw2": h.T @ ds, "db2": float(ds.sum()),
            "dx": (dz @ w1).reshape(x.shape)}



# ---------------------------------------------------------------------------
# Section 3.5: feature-preserving alignment (Eqs. 9-11)
# ---------------------------------------------------------------------------

def softmax_rows(h) -> np.ndarray:
    """Softmax over the last axis, shifted by the row maximum."""
    h = f64(h)
    e = np.exp(h - h.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def hidden_align_sq(h_sparse, h_dense) -> np.ndarray:
    """Per-token squared distance of Eq. 9: sum over the hidden dimension of
    (Softmax(h_sparse) - Softmax(h_dense))^2, the softmax taken over the
    hidden dimension of each token. Returns the leading shape of the inputs."""
    d = softmax_rows(h_sparse) - softmax_rows(h_dense)
    return np.sum(d * d, axis=-1)


def hidden_align_loss(h_sparse, h_dense) -> float:
    """Eq. 9 for one layer: the 2-norm of the difference of the per-token
    softmaxes, over the whole [B, T, d] hidden-state tensor (the entrywise
    norm of the matrix difference)."""
    return float(math.sqrt(np.sum(hidden_align_sq(h_sparse, h_dense))))


def log_softmax_rows(z) -> np.ndarray:
    """log Softmax over the last axis: z - max - log sum exp(z - max)."""
    z = f64(z)
    m = z.max(axis=-1, keepdims=True)
    return z - m - np.log(np.sum(np.exp(z - m), axis=-1, keepdims=True))


def kl_align(logits_dense, logits_sparse) -> np.ndarray:
    """Eq. 10 per row: sum_c P_dense(c) log(P_dense(c) / P_sparse(c)) with
    P = Softmax(logits) over the classes (last axis)."""
    lp = log_softmax_rows(logits_dense)
    lq = log_softmax_rows(logits_sparse)
    return np.sum(np.exp(lp) * (lp - lq), axis=-1)


def total_objective(l_align: float, l_hid: Sequence[float]) -> float:
    """Eq. 11: L_align + (1 / L) sum_l L_hid^(l)."""
    return float(l_align + np.mean(np.asarray(l_hid, dtype=np.float64)))


def align_stack(desc: Dict, Ws: List[Dict], x, ks: Sequence[int]) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Dense-teacher / sparse-student forward (Section 3.5): both stacks start
    from the same input; after layer l, Eq. 9 compares the student's hidden
    states (routed layers) with the teacher's (dense layers).

    Returns (per-layer sums of the per-token squared distances, the student's
    final hidden states, the teacher's). L_hid^(l) is the square root of the
    l-th sum.
    """
    xs = f64(x)
    xd = f64(x)
    sums = []
    for W, k in zip(Ws, ks):
        xd = dense_layer(desc, W, xd)
        xs = routed_layer(desc, W, xs, int(k))["y"] if k > 0 else xs
        sums.append(float(np.sum(hidden_align_sq(xs, xd))))
    return np.asarray(sums), xs, xd


# ---------------------------------------------------------------------------
# Incremental decoding (not treated by the paper; see the reading in the
# header): threshold routing of each new token and per-layer kept sets.
# ---------------------------------------------------------------------------

def keep_by_threshold(scores, thr) -> np.ndarray:
    """A new token is kept iff its router score >= the threshold (NaN: not kept)."""
    return np.asarray(scores, dtype=np.float64) >= np.asarray(thr, dtype=np.float64)


def kept_set_layer(desc: Dict, W: Dict, x, keeps: Sequence[Sequence[int]],
                   out_dtype: Optional[str] = None) -> np.ndarray:
    """One layer with explicit kept positions per sequence (the sets may differ
    in size): the block runs on each sequence's kept rows at their positions,
    the other rows pass through unchanged (Section 3.4 with a given selection).
    """
    x = f64(x)
    y = x.copy()
    for b in range(x.shape[0]):
        pos = np.asarray(sorted(keeps[b]), dtype=np.int64)
        if pos.size == 0:
            continue
        rows = x[b, pos] + block_delta(desc, W, x[b, pos], pos)
        y[b, pos] = rows if out_dtype is None else round_to(out_dtype, rows)
    return y


def kept_set_stack(desc: Dict, Ws: List[Dict], x, keeps_per_layer,
                   out_dtype: Optional[str] = None) -> np.ndarray:
    """kept_set_layer for l = 0..L-1; keeps_per_layer[l][b] = kept positions."""
    x = f64(x)
    for W, keeps in zip(Ws, keeps_per_layer):
        x = kept_set_layer(desc, W, x, keeps, out_dtype)
    return x


def decode_stack(desc: Dict, Ws: List[Dict], x, thr=None, force=None,
                 out_dtype: Optional[str] = None) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
    """Tokens t = 0..T-1 of every sequence processed one at a time.

    At layer l, token t's router score is taken on its current hidden state;
    the token is kept iff score >= thr[l][b] (or force[l][b][t] when force is
    given). A kept token's output is its row plus the block's update computed
    over the layer's kept rows so far (their layer inputs at their positions),
    itself last; a skipped token passes through. Returns (y [B, T, d],
    keep [L, B, T] bool, scores [L, B, T]).
    """
    x = f64(x)
    B, T, _ = x.shape
    L = len(Ws)
    y = x.copy()
    keep = np.zeros((L, B, T), dtype=bool)
    scores = np.zeros((L, B, T))
    kept_in = [[[] for _ in range(B)] for _ in range(L)]  # layer inputs of the kept rows
    kept_pos = [[[] for _ in range(B)] for _ in range(L)]
    for t in range(T):
        for b in range(B):
            row = y[b, t].copy()
            for l, W in enumerate(Ws):
                s = router_scores(row[None, None, :], W["router_w1"], W["router_b1"], W["router_w2"],
                                  W.get("router_b2", 0.0))[0, 0]
                scores[l, b, t] = s
                kl = bool(force[l][b][t]) if force is not None else bool(keep_by_threshold(s, thr[l][b]))
                keep[l, b, t] = kl
                if not kl:
                    continue
                kept_in[l][b].append(row)
                kept_pos[l][b].append(t)
                rows = np.stack(kept_in[l][b])
                delta = block_delta(desc, W, rows, np.asarray(kept_pos[l][b]))[-1]
                row = row + delta
                if out_dtype is not None:
                    row = round_to(out_dtype, row)
            y[b, t] = row
    return y, keep, scores


# ---------------------------------------------------------------------------
# Section 3.4, training side: the backward of the routed layer (the block's
# adjoint on the kept rows, and the adjoints of the gather and the scatter)
# ---------------------------------------------------------------------------

def gelu_grad(x) -> np.ndarray:
    """d/dx of x Phi(x): Phi(x) + x phi(x)."""
    x = f64(x)
    return 0.5 * (1.0 + erf(x / math.sqrt(2.0))) + x * np.exp(-0.5 * x * x) / math.sqrt(2.0 * math.pi)


def silu_grad(x) -> np.ndarray:
    """d/dx of x sigmoid(x): s (1 + x (1 - s)), s = sigmoid(x)."""
    x = f64(x)
    s = sigmoid(x)
    return s * (1.0 + x * (1.0 - s))


def layer_norm_backward(dy, x, w, eps: float):
    """Adjoint of y = (x - mu) / sigma * w + b over the last axis (biased
    variance, sigma = sqrt(var + eps)). Returns (dx, dw, db); dw and db are
    summed over the rows."""
    x, dy, w = f64(x), f64(dy), f64(w)
    mu = np.mean(x, axis=-1, keepdims=True)
    sig = np.sqrt(np.mean((x - mu) ** 2, axis=-1, keepdims=True) + eps)
    xh = (x - mu) / sig
    g = dy * w
    dx = (g - np.mean(g, axis=-1, keepdims=True) - xh * np.mean(g * xh, axis=-1, keepdims=True)) / sig
    return dx, np.sum(dy * xh, axis=0), np.sum(dy, axis=0)


def rms_norm_backward(dy, x, w, eps: float):
    """Adjoint of y = x / r * w, r = sqrt(mean(x^2) + eps). Returns (dx, dw)."""
    x, dy, w = f64(x), f64(dy), f64(w)
    r = np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    xh = x / r
    g = dy * w
    dx = (g - xh * np.mean(g * xh, axis=-1, keepdims=True)) / r
    return dx, np.sum(dy * xh, axis=0)


def rope_backward(dout, pos, rotary_dims: int, theta: float) -> np.ndarray:
    """Adjoint of rope(): each pair (i, i + R/2) was rotated by the angle
    pos * theta^(-2i/R), so its gradient is rotated back by the same angle."""
    d = f64(dout)
    R = rotary_dims
    half = R // 2
    inv_freq = theta ** (-(2.0 * np.arange(half)) / R)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]
    cos = np.cos(ang)[:, None, :]
    sin = np.sin(ang)[:, None, :]
    out = d.copy()
    d1 = d[..., :half]
    d2 = d[..., half:R]
    out[..., :half] = d1 * cos + d2 * sin
    out[..., half:R] = d2 * cos - d1 * sin
    return out


def causal_attention_backward(q, k, v, dout):
    """Adjoint of causal_attention(q, k, v) (Eq. 1 over the kept tokens).

    q [n, Hq, hd], k and v [n, Hkv, hd], dout [n, Hq * hd]. Per query head h
    on kv head h // (Hq / Hkv): P = softmax(q k^T / sqrt(hd)) causal,
    dV = P^T dO, dP = dO V^T, dS = P (dP - rowsum(P dP)), dQ = dS K / sqrt(hd),
    dK = dS^T Q / sqrt(hd); the kv gradients add up over the query heads of a
    group. Returns (dq, dk, dv) in the input layouts."""
    q, k, v = f64(q), f64(k), f64(v)
    n, Hq, hd = q.shape
    Hkv = k.shape[1]
    group = Hq // Hkv
    do = f64(dout).reshape(n, Hq, hd)
    dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    mask = np.triu(np.ones((n, n), dtype=bool), 1)
    sc = 1.0 / math.sqrt(hd)
    for h in range(Hq):
        kh = h // group
        s = (q[:, h, :] @ k[:, kh, :].T) * sc
        s[mask] = -np.inf
        p = np.exp(s - np.max(s, axis=1, keepdims=True))
        p = p / np.sum(p, axis=1, keepdims=True)
        dov = do[:, h, :]
        dv[:, kh, :] += p.T @ dov
        dp = dov @ v[:, kh, :].T
        ds = p * (dp - np.sum(p * dp, axis=1, keepdims=True))
        dq[:, h, :] = (ds @ k[:, kh, :]) * sc
        dk[:, kh, :] += (ds.T @ q[:, h, :]) * sc
    return dq, dk, dv


def block_forward_cache(desc: Dict, W: Dict, xc, pos):
    """block_delta with its intermediate values kept for the backward.
    Returns (delta, cache)."""
    xc = f64(xc)
    n = xc.shape[0]
    Hq, Hkv, hd = desc["n_heads"], desc["n_kv_heads"], desc["head_dim"]
    f = desc["d_ff"]
    eps = desc["norm_eps"]
    neox = desc["block"] == NEOX

    def linear(inp, wname, bname=None):
        y = inp @ f64(W[wname]).T
        b = W.get(bname) if bname else None
        return y if b is None else y + f64(b)

    c = {"xc": xc, "pos": np.asarray(pos)}
    c["a"] = layer_norm(xc, W["norm1_w"], W["norm1_b"], eps) if neox else rms_norm(xc, W["norm1_w"], eps)
    qkv = linear(c["a"], "w_qkv", "b_qkv")
    q = qkv[:, :Hq * hd].reshape(n, Hq, hd)
    k = qkv[:, Hq * hd:(Hq + Hkv) * hd].reshape(n, Hkv, hd)
    c["v"] = qkv[:, (Hq + Hkv) * hd:].reshape(n, Hkv, hd)
    c["q"] = rope(q, pos, desc["rotary_dims"], desc["rope_theta"])
    c["k"] = rope(k, pos, desc["rotary_dims"], desc["rope_theta"])
    c["attn"] = causal_attention(c["q"], c["k"], c["v"])
    ao = linear(c["attn"], "w_o", "b_o")
    if neox:
        c["m"] = layer_norm(xc, W["norm2_w"], W["norm2_b"], eps)
        c["u"] = linear(c["m"], "w_up", "b_up")
        c["act"] = gelu(c["u"])
    else:
        c["h"] = xc + ao
        c["m"] = rms_norm(c["h"], W["norm2_w"], eps)
        c["u"] = linear(c["m"], "w_up")
        c["act"] = silu(c["u"][:, :f]) * c["u"][:, f:]
    mo = linear(c["act"], "w_down", "b_down")
    return ao + mo, c


def block_backward(desc: Dict, W: Dict, cache: Dict, ddelta):
    """Adjoint of delta = block(xc): given ddelta = dL/d delta [n, d], returns
    (dL/dxc through the block, dict of weight gradients) for the cache of
    block_forward_cache. Weight gradients have the weights' layouts; the
    entries of absent biases are None."""
    dd = f64(ddelta)
    Hq, Hkv, hd = desc["n_heads"], desc["n_kv_heads"], desc["head_dim"]
    f = desc["d_ff"]
    eps = desc["norm_eps"]
    neox = desc["block"] == NEOX
    c = cache
    n = dd.shape[0]
    g = {}
    # FFN: mo = act W_down^T + b_down
    dact = dd @ f64(W["w_down"])
    g["w_down"] = dd.T @ c["act"]
    g["b_down"] = dd.sum(axis=0) if neox else None
    if neox:
        du = dact * gelu_grad(c["u"])
    else:
        gt, up = c["u"][:, :f], c["u"][:, f:]
        du = np.concatenate([dact * up * silu_grad(gt), dact * silu(gt)], axis=1)
    g["w_up"] = du.T @ c["m"]
    g["b_up"] = du.sum(axis=0) if neox else None
    dm = du @ f64(W["w_up"])
    if neox:
        dx_m, g["norm2_w"], g["norm2_b"] = layer_norm_backward(dm, c["xc"], W["norm2_w"], eps)
        dao = dd
        dx_h = 0.0
    else:
        dh, g["norm2_w"] = rms_norm_backward(dm, c["h"], W["norm2_w"], eps)
        g["norm2_b"] = None
        dao = dd + dh
        dx_m, dx_h = 0.0, dh
    # attention output projection: ao = attn W_o^T + b_o
    dattn = dao @ f64(W["w_o"])
    g["w_o"] = dao.T @ c["attn"]
    g["b_o"] = dao.sum(axis=0) if neox else None
    dqr, dkr, dv = causal_attention_backward(c["q"], c["k"], c["v"], dattn)
    dq = rope_backward(dqr, c["pos"], desc["rotary_dims"], desc["rope_theta"])
    dk = rope_backward(dkr, c["pos"], desc["rotary_dims"], desc["rope_theta"])
    dqkv = np.concatenate([dq.reshape(n, Hq * hd), dk.reshape(n, Hkv * hd), dv.reshape(n, Hkv * hd)], axis=1)
    g["w_qkv"] = dqkv.T @ c["a"]
    g["b_qkv"] = dqkv.sum(axis=0)
    da = dqkv @ f64(W["w_qkv"])
    if neox:
        dx_a, g["norm1_w"], g["norm1_b"] = layer_norm_backward(da, c["xc"], W["norm1_w"], eps)
    else:
        dx_a, g["norm1_w"] = rms_norm_backward(da, c["xc"], W["norm1_w"], eps)
        g["norm1_b"] = None
    return dx_a + dx_m + dx_h, g


GRAD_NAMES = ["w_qkv", "b_qkv", "w_o", "b_o", "w_up", "b_up", "w_down", "b_down",
              "norm1_w", "norm1_b", "norm2_w", "norm2_b"]


def routed_layer_backward(desc: Dict, W: Dict, x, dy, idx, gate: bool = False) -> Dict:
    """Backward of routed_layer(desc, W, x, k, idx=idx, gate=gate).

    The kept rows xc = x[b, idx[b]] produce y = xc + g delta (g = 1, or
    sigmoid of the router score with gate); skipped rows pass through, so
    dx = dy there. At a kept row dx = dy + (dL/dxc through delta), with
    dL/d delta = g dy. Weight gradients are summed over the sequences. The
    router's share (through the gated scores) is not included: it is
    gate_score_grad followed by router_backward.
    Returns {"dx": [B, T, d], "grads": {name: array or None}}.
    """
    x, dy = f64(x), f64(dy)
    idx = np.asarray(idx, dtype=np.int64)
    B = x.shape[0]
    dx = dy.copy()
    tot = {name: None for name in GRAD_NAMES}
    scores = router_scores(x, W["router_w1"], W["router_b1"], W["router_w2"], W.get("router_b2", 0.0))
    for b in range(B):
        p = idx[b]
        if p.size == 0:
            continue
        _, cache = block_forward_cache(desc, W, x[b, p], p)
        g = sigmoid(scores[b, p])[:, None] if gate else 1.0
        dxc, grads = block_backward(desc, W, cache, g * dy[b, p])
        dx[b, p] = dy[b, p] + dxc
        for name, val in grads.items():
            if val is not None:
                tot[name] = val if tot[name] is None else tot[name] + val
    return {"dx": dx, "grads": tot}
