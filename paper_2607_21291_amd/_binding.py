"""ctypes binding of libadadsf.so: the C ABI in include/adadsf.h, one Python
function per entry point, same names without the ``dsf_`` prefix.

Argument marshalling only. Tensors are torch tensors on the GPU (torch owns
device memory and streams); every computation runs in the library's HIP
kernels. A missing library raises immediately: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import torch  # loads the HIP runtime that the library binds to

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libadadsf.so")

F32, BF16 = 0, 1
BLOCK_NEOX_PARALLEL, BLOCK_QWEN_SEQ = 0, 1
FLAG_DENSE, FLAG_GATE = 1, 2
CLIP = {"none": 0, "plain": 1, "budget": 2}
ROUNDING = {"floor": 0, "ceil": 1}
KINDS = ["sim", "router", "topk", "norm", "gemm_qkv", "attn", "gemm_o", "gemm_up", "gemm_down",
         "gather", "scatter", "other", "backward", "align"]

STATUS = {0: "DSF_OK", 1: "DSF_EINVAL", 2: "DSF_EUNSUPPORTED", 3: "DSF_EWORKSPACE", 4: "DSF_EHIP",
          5: "DSF_ENODEVICE"}

EXPORTS = [
    "dsf_version", "dsf_last_error", "dsf_sim_workspace_size", "dsf_sim_stats", "dsf_sim_finalize",
    "dsf_retention_from_similarity", "dsf_k_from_retention", "dsf_router_score", "dsf_topk_select",
    "dsf_gather_rows", "dsf_scatter_residual", "dsf_attention_forward", "dsf_workspace_size",
    "dsf_sparse_block_forward", "dsf_stack_forward", "dsf_timing_enable", "dsf_timing_read",
    "dsf_gate_score_grad", "dsf_router_backward_workspace_size", "dsf_router_backward",
    "dsf_align_workspace_size", "dsf_align_hidden", "dsf_kl_align", "dsf_align_stack_workspace_size",
    "dsf_align_stack_forward", "dsf_decode_workspace_size", "dsf_decode_step", "dsf_stack_prefill",
    "dsf_workspace_status", "dsf_decode_static_scratch_bytes", "dsf_decode_step_static",
    "dsf_backward_workspace_size", "dsf_sparse_block_backward",
]
WS_STATUS_SK_TIMEOUT = 1


class DsfError(RuntimeError):
    def __init__(self, fn: str, code: int, msg: str):
        super().__init__(f"{fn} -> {STATUS.get(code, code)}: {msg}")
        self.code = code


class LayerDesc(ctypes.Structure):
    _fields_ = [("block", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("d_ff", ctypes.c_int32),
                ("rotary_dims", ctypes.c_int32), ("d_router", ctypes.c_int32), ("norm_eps", ctypes.c_float),
                ("reserved", ctypes.c_float), ("rope_theta", ctypes.c_double)]


_WEIGHT_FIELDS = ["router_w1", "router_b1", "router_w2", "router_b2", "reserved", "norm1_w", "norm1_b",
                  "norm2_w", "norm2_b", "w_qkv", "b_qkv", "w_o", "b_o", "w_up", "b_up", "w_down", "b_down"]


GRAD_FIELDS = ["w_qkv", "b_qkv", "w_o", "b_o", "w_up", "b_up", "w_down", "b_down", "norm1_w", "norm1_b",
               "norm2_w", "norm2_b"]


class LayerGrads(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in GRAD_FIELDS]


class LayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_float if n in ("router_b2", "reserved") else ctypes.c_void_p)
                for n in _WEIGHT_FIELDS]


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                           "(python -m paper_2607_21291_amd.build_lib)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, sz, f32, f64 = (ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t,
                                  ctypes.c_float, ctypes.c_double)
    sig = {
        "dsf_version": ([], i32),
        "dsf_last_error": ([], ctypes.c_char_p),
        "dsf_sim_workspace_size": ([i64], sz),
        "dsf_sim_stats": ([vp, vp, i32, i64, i32, vp, vp, vp, sz, vp], i32),
        "dsf_sim_finalize": ([vp, i32, vp, vp], i32),
        "dsf_retention_from_similarity": ([vp, i32, f64, f64, f64, i32, vp], i32),
        "dsf_k_from_retention": ([f64, i32, i32], i32),
        "dsf_router_score": ([vp, i32, i64, i32, i32, vp, vp, vp, f32, vp, vp], i32),
        "dsf_topk_select": ([vp, i32, i32, i32, vp, vp], i32),
        "dsf_gather_rows": ([vp, i32, i32, i32, i32, vp, i32, vp, vp], i32),
        "dsf_scatter_residual": ([vp, vp, i32, i32, i32, i32, vp, i32, vp], i32),
        "dsf_attention_forward": ([vp, vp, vp, i32, i32, i32, i32, i32, i32, vp, vp], i32),
        "dsf_workspace_size": ([vp, i32, i32, i32, i32, i32], sz),
        "dsf_workspace_status": ([vp, vp, vp], i32),
        "dsf_sparse_block_forward": ([vp, vp, i32, vp, i32, i32, i32, i32, vp, vp, vp, vp, sz, vp], i32),
        "dsf_stack_forward": ([vp, vp, i32, i32, vp, vp, i32, i32, i32, vp, vp, sz, vp], i32),
        "dsf_timing_enable": ([i32, ctypes.c_uint32], i32),
        "dsf_timing_read": ([i32, vp, vp], i32),
        "dsf_gate_score_grad": ([vp, vp, vp, i32, vp, vp, i32, i32, i32, i32, vp, vp], i32),
        "dsf_router_backward_workspace_size": ([i64, i32, i32], sz),
        "dsf_router_backward": ([vp, i32, i64, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp], i32),
        "dsf_align_workspace_size": ([i64], sz),
        "dsf_align_hidden": ([vp, vp, i32, i64, i32, vp, vp, vp, sz, vp], i32),
        "dsf_kl_align": ([vp, vp, i32, i64, i32, vp, vp, vp, sz, vp], i32),
        "dsf_align_stack_workspace_size": ([vp, i32, i32, i32], sz),
        "dsf_align_stack_forward": ([vp, vp, i32, i32, vp, vp, vp, i32, i32, i32, vp, vp, sz, vp], i32),
        "dsf_decode_workspace_size": ([vp, i32, i32, i32, i32], sz),
        "dsf_decode_step": ([vp, vp, i32, i32, vp, i32, vp, i32, vp, vp, vp, vp, vp, vp, i32, vp, sz, vp], i32),
        "dsf_stack_prefill": ([vp, vp, i32, i32, vp, vp, i32, i32, vp, vp, vp, i32, vp, vp, sz, vp], i32),
        "dsf_decode_static_scratch_bytes": ([], sz),
        "dsf_backward_workspace_size": ([vp, i32, i32, i32, i32], sz),
        "dsf_sparse_block_backward": ([vp, vp, i32, vp, vp, i32, i32, i32, vp, vp, i32, vp, vp, vp, sz, vp], i32),
        "dsf_decode_step_static": ([vp, vp, i32, i32, vp, i32, vp, i32, vp, vp, vp, vp, vp, vp, i32, vp], i32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    _lib = L
    return L


def _check(fn: str, rc: int):
    if rc != 0:
        raise DsfError(fn, rc, lib().dsf_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensors passed to the library must be contiguous")
    return t.data_ptr()


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise ValueError(f"unsupported dtype {t.dtype}")


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


# --------------------------------------------------------------- entry points

def version() -> int:
    return lib().dsf_version()


def last_error() -> str:
    return lib().dsf_last_error().decode()


def sim_workspace_size(n_tokens: int) -> int:
    return lib().dsf_sim_workspace_size(n_tokens)


def sim_stats(x_in, x_out, accum, per_token_cos=None, workspace=None, stream=None):
    d = x_in.shape[-1]
    n = x_in.numel() // d
    if workspace is None:
        workspace = torch.empty(max(sim_workspace_size(n), 256), dtype=torch.uint8, device=x_in.device)
    _check("dsf_sim_stats", lib().dsf_sim_stats(_ptr(x_in), _ptr(x_out), _dtype_code(x_in), n, d,
                                                _ptr(per_token_cos), _ptr(accum), _ptr(workspace),
                                                workspace.numel(), _stream(stream)))


def sim_finalize(accum, stream=None):
    L = accum.numel() // 2
    out = (ctypes.c_double * max(L, 1))()
    _check("dsf_sim_finalize", lib().dsf_sim_finalize(_ptr(accum), L, ctypes.addressof(out), _stream(stream)))
    return [out[i] for i in range(L)]


def retention_from_similarity(s: Sequence[float], t: float, tau: Optional[float], beta: float = 10.0,
                              clip: str = "budget"):
    L = len(s)
    sin = (ctypes.c_double * max(L, 1))(*s)
    rout = (ctypes.c_double * max(L, 1))()
    _check("dsf_retention_from_similarity",
           lib().dsf_retention_from_similarity(ctypes.addressof(sin), L, t, -1.0 if tau is None else tau, beta,
                                               CLIP[clip], ctypes.addressof(rout)))
    return [rout[i] for i in range(L)]


def k_from_retention(r: float, T: int, rounding: str = "floor") -> int:
    k = lib().dsf_k_from_retention(r, T, ROUNDING[rounding])
    if k < 0:
        raise DsfError("dsf_k_from_retention", 1, last_error())
    return k


def router_score(x, w1, b1, w2, b2: float, scores, stream=None):
    d = x.shape[-1]
    _check("dsf_router_score", lib().dsf_router_score(_ptr(x), _dtype_code(x), x.numel() // d, d, w1.shape[0],
                                                      _ptr(w1), _ptr(b1), _ptr(w2), float(b2), _ptr(scores),
                                                      _stream(stream)))


def gate_score_grad(dy, x_in, x_out, scores, idx, dscore, stream=None):
    B, T, d = dy.shape
    _check("dsf_gate_score_grad",
           lib().dsf_gate_score_grad(_ptr(dy), _ptr(x_in), _ptr(x_out), _dtype_code(dy), _ptr(scores), _ptr(idx),
                                     B, T, idx.shape[1], d, _ptr(dscore), _stream(stream)))


def router_backward_workspace_size(n_tokens: int, d: int, d_r: int) -> int:
    return lib().dsf_router_backward_workspace_size(n_tokens, d, d_r)


def router_backward(x, w1, b1, w2, dscore, dw1, db1, dw2, db2, dx=None, workspace=None, stream=None):
    d = x.shape[-1]
    n = x.numel() // d
    d_r = w1.shape[0]
    if workspace is None:
        workspace = torch.empty(max(router_backward_workspace_size(n, d, d_r), 256), dtype=torch.uint8,
                                device=x.device)
    _check("dsf_router_backward",
           lib().dsf_router_backward(_ptr(x), _dtype_code(x), n, d, d_r, _ptr(w1), _ptr(b1), _ptr(w2), _ptr(dscore),
                                     _ptr(dw1), _ptr(db1), _ptr(dw2), _ptr(db2), _ptr(dx), _ptr(workspace),
                                     workspace.numel(), _stream(stream)))


def topk_select(scores, k: int, idx, stream=None):
    B, T = scores.shape
    _check("dsf_topk_select", lib().dsf_topk_select(_ptr(scores), B, T, k, _ptr(idx), _stream(stream)))


def gather_rows(x, idx, out, stream=None):
    B, T, d = x.shape
    _check("dsf_gather_rows", lib().dsf_gather_rows(_ptr(x), _dtype_code(x), B, T, d, _ptr(idx), idx.shape[1],
                                                    _ptr(out), _stream(stream)))


def scatter_residual(x, delta, idx, stream=None):
    B, T, d = x.shape
    _check("dsf_scatter_residual", lib().dsf_scatter_residual(_ptr(x), _ptr(delta), _dtype_code(x), B, T, d,
                                                              _ptr(idx), idx.shape[1], _stream(stream)))


def attention_forward(q, k, v, out, stream=None):
    B, Hq, n, hd = q.shape
    _check("dsf_attention_forward", lib().dsf_attention_forward(_ptr(q), _ptr(k), _ptr(v), _dtype_code(q), B, Hq,
                                                                k.shape[1], n, hd, _ptr(out), _stream(stream)))


def workspace_size(desc: LayerDesc, dtype: int, B: int, T: int, k_max: int, with_similarity: bool = False) -> int:
    return lib().dsf_workspace_size(ctypes.addressof(desc), dtype, B, T, k_max, int(with_similarity))


def workspace_status(workspace, stream=None) -> int:
    """Status word of the last layer/stack call on this workspace (waits for the stream)."""
    out = ctypes.c_uint32(0)
    _check("dsf_workspace_status", lib().dsf_workspace_status(_ptr(workspace), ctypes.byref(out), _stream(stream)))
    return int(out.value)


def backward_workspace_size(desc: LayerDesc, dtype: int, B: int, T: int, k: int) -> int:
    return lib().dsf_backward_workspace_size(ctypes.addressof(desc), dtype, B, T, k)


def sparse_block_backward(desc: LayerDesc, weights: LayerWeights, x, dy, idx, dx, grads: dict, workspace,
                          scores=None, flags: int = 0, stream=None):
    """grads: name -> fp32 device tensor (or None) for the names in GRAD_FIELDS."""
    B, T, _ = x.shape
    k = idx.shape[1] if idx is not None else 0
    gs = LayerGrads(*[_ptr(grads.get(n)) for n in GRAD_FIELDS])
    _check("dsf_sparse_block_backward",
           lib().dsf_sparse_block_backward(ctypes.addressof(desc), ctypes.addressof(weights), _dtype_code(x),
                                           _ptr(x), _ptr(dy), B, T, k, _ptr(idx), _ptr(scores), flags, _ptr(dx),
                                           ctypes.addressof(gs), _ptr(workspace), workspace.numel(),
                                           _stream(stream)))


def sparse_block_forward(desc: LayerDesc, weights: LayerWeights, x, k: int, workspace, flags: int = 0,
                         scores_out=None, idx_out=None, idx_in=None, stream=None):
    B, T, _ = x.shape
    _check("dsf_sparse_block_forward",
           lib().dsf_sparse_block_forward(ctypes.addressof(desc), ctypes.addressof(weights), _dtype_code(x),
                                          _ptr(x), B, T, k, flags, _ptr(scores_out), _ptr(idx_out), _ptr(idx_in),
                                          _ptr(workspace), workspace.numel(), _stream(stream)))


def stack_forward(desc: LayerDesc, weights: Sequence[LayerWeights], ks: Sequence[int], x, workspace,
                  flags: int = 0, sim_accum=None, stream=None):
    B, T, _ = x.shape
    L = len(weights)
    arr = (LayerWeights * max(L, 1))(*weights)
    karr = (ctypes.c_int * max(L, 1))(*[int(k) for k in ks])
    _check("dsf_stack_forward",
           lib().dsf_stack_forward(ctypes.addressof(desc), ctypes.addressof(arr), L, _dtype_code(x),
                                   ctypes.addressof(karr), _ptr(x), B, T, flags, _ptr(sim_accum), _ptr(workspace),
                                   workspace.numel(), _stream(stream)))


def align_workspace_size(n_rows: int) -> int:
    return lib().dsf_align_workspace_size(n_rows)


def align_hidden(h_sparse, h_dense, accum, per_token_sq=None, workspace=None, stream=None):
    d = h_sparse.shape[-1]
    n = h_sparse.numel() // d
    if workspace is None:
        workspace = torch.empty(align_workspace_size(n), dtype=torch.uint8, device=h_sparse.device)
    _check("dsf_align_hidden", lib().dsf_align_hidden(_ptr(h_sparse), _ptr(h_dense), _dtype_code(h_sparse), n, d,
                                                      _ptr(per_token_sq), _ptr(accum), _ptr(workspace),
                                                      workspace.numel(), _stream(stream)))


def kl_align(logits_dense, logits_sparse, accum, per_row_kl=None, workspace=None, stream=None):
    C = logits_dense.shape[-1]
    n = logits_dense.numel() // C
    if workspace is None:
        workspace = torch.empty(align_workspace_size(n), dtype=torch.uint8, device=logits_dense.device)
    _check("dsf_kl_align", lib().dsf_kl_align(_ptr(logits_dense), _ptr(logits_sparse), _dtype_code(logits_dense), n,
                                              C, _ptr(per_row_kl), _ptr(accum), _ptr(workspace), workspace.numel(),
                                              _stream(stream)))


def align_stack_workspace_size(desc: LayerDesc, dtype: int, B: int, T: int) -> int:
    return lib().dsf_align_stack_workspace_size(ctypes.addressof(desc), dtype, B, T)


def align_stack_forward(desc: LayerDesc, weights: Sequence[LayerWeights], ks: Sequence[int], x_sparse, x_dense,
                        hid_accum, workspace, flags: int = 0, stream=None):
    B, T, _ = x_sparse.shape
    L = len(weights)
    arr = (LayerWeights * max(L, 1))(*weights)
    karr = (ctypes.c_int * max(L, 1))(*[int(k) for k in ks])
    _check("dsf_align_stack_forward",
           lib().dsf_align_stack_forward(ctypes.addressof(desc), ctypes.addressof(arr), L, _dtype_code(x_sparse),
                                         ctypes.addressof(karr), _ptr(x_sparse), _ptr(x_dense), B, T, flags,
                                         _ptr(hid_accum), _ptr(workspace), workspace.numel(), _stream(stream)))


def decode_workspace_size(desc: LayerDesc, dtype: int, B: int, max_pos: int, cap: int) -> int:
    return lib().dsf_decode_workspace_size(ctypes.addressof(desc), dtype, B, max_pos, cap)


def _ptr_array(tensors):
    return (ctypes.c_void_p * max(len(tensors), 1))(*[_ptr(t) for t in tensors])


def decode_step(desc: LayerDesc, weights: Sequence[LayerWeights], x, pos, max_pos: int, thr, cache_k, cache_v,
                cache_len, workspace, scores_out=None, keep_out=None, stream=None):
    """x [B, d]; pos int32 [B]; thr float [L, B]; cache_k / cache_v: L tensors [B, Hkv, cap, hd];
    cache_len int32 [L, B]."""
    B = x.shape[0]
    L = len(weights)
    cap = cache_k[0].shape[2] if L else 1
    arr = (LayerWeights * max(L, 1))(*weights)
    ck, cv = _ptr_array(cache_k), _ptr_array(cache_v)
    _check("dsf_decode_step",
           lib().dsf_decode_step(ctypes.addressof(desc), ctypes.addressof(arr), L, _dtype_code(x), _ptr(x), B,
                                 _ptr(pos), max_pos, _ptr(thr), _ptr(scores_out), _ptr(keep_out),
                                 ctypes.addressof(ck), ctypes.addressof(cv), _ptr(cache_len), cap, _ptr(workspace),
                                 workspace.numel(), _stream(stream)))


def decode_static_scratch_bytes() -> int:
    return lib().dsf_decode_static_scratch_bytes()


def decode_step_static(desc: LayerDesc, weights: Sequence[LayerWeights], x, pos, max_pos: int, thr, cache_k,
                       cache_v, cache_len, scores_out=None, keep_out=None, stream=None):
    """dsf_decode_step on the library's static device scratch (no workspace, no allocation)."""
    B = x.shape[0]
    L = len(weights)
    cap = cache_k[0].shape[2] if L else 1
    arr = (LayerWeights * max(L, 1))(*weights)
    ck, cv = _ptr_array(cache_k), _ptr_array(cache_v)
    _check("dsf_decode_step_static",
           lib().dsf_decode_step_static(ctypes.addressof(desc), ctypes.addressof(arr), L, _dtype_code(x), _ptr(x), B,
                                        _ptr(pos), max_pos, _ptr(thr), _ptr(scores_out), _ptr(keep_out),
                                        ctypes.addressof(ck), ctypes.addressof(cv), _ptr(cache_len), cap,
                                        _stream(stream)))


def stack_prefill(desc: LayerDesc, weights: Sequence[LayerWeights], ks: Sequence[int], x, cache_k, cache_v,
                  cache_len, workspace, thr_out=None, stream=None):
    """dsf_stack_forward over x [B, T, d] that also fills the decode caches."""
    B, T, _ = x.shape
    L = len(weights)
    cap = cache_k[0].shape[2] if L else 1
    arr = (LayerWeights * max(L, 1))(*weights)
    karr = (ctypes.c_int * max(L, 1))(*[int(k) for k in ks])
    ck, cv = _ptr_array(cache_k), _ptr_array(cache_v)
    _check("dsf_stack_prefill",
           lib().dsf_stack_prefill(ctypes.addressof(desc), ctypes.addressof(arr), L, _dtype_code(x),
                                   ctypes.addressof(karr), _ptr(x), B, T, ctypes.addressof(ck), ctypes.addressof(cv),
                                   _ptr(cache_len), cap, _ptr(thr_out), _ptr(workspace), workspace.numel(),
                                   _stream(stream)))


def timing_enable(max_records: int, kinds: Optional[Sequence[str]] = None):
    """Arm per-launch event timing for the named kernel classes (all if None)."""
    mask = (1 << len(KINDS)) - 1 if kinds is None else sum(1 << KINDS.index(k) for k in kinds)
    _check("dsf_timing_enable", lib().dsf_timing_enable(max_records, mask))


def timing_read(kind: str):
    n = ctypes.c_int(0)
    ms = ctypes.c_double(0.0)
    _check("dsf_timing_read", lib().dsf_timing_read(KINDS.index(kind), ctypes.addressof(n), ctypes.addressof(ms)))
    return n.value, ms.value


# ------------------------------------------------------ marshalling helpers

def make_desc(block: str, d_model: int, n_heads: int, n_kv_heads: int, head_dim: int, d_ff: int,
              rotary_dims: int, d_router: int, norm_eps: float, rope_theta: float) -> LayerDesc:
    code = {"neox_parallel": BLOCK_NEOX_PARALLEL, "qwen_seq": BLOCK_QWEN_SEQ}[block]
    return LayerDesc(code, d_model, n_heads, n_kv_heads, head_dim, d_ff, rotary_dims, d_router, norm_eps, 0.0,
                     rope_theta)


class DeviceLayer:
    """Keeps one layer's device tensors alive and exposes them as LayerWeights."""

    def __init__(self, tensors: dict, device):
        self.tensors = {}
        for name in _WEIGHT_FIELDS:
            if name in ("router_b2", "reserved"):
                continue
            t = tensors.get(name)
            self.tensors[name] = None if t is None else t.to(device).contiguous()
        self.router_b2 = float(tensors.get("router_b2", 0.0))
        kw = {n: _ptr(t) for n, t in self.tensors.items()}
        self.weights = LayerWeights(router_b2=self.router_b2, reserved=0.0, **kw)
