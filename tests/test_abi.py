"""C-ABI checks that need no GPU: exports, struct layout, host-side allocation
(Eqs. 5-8 and K) against the oracle, and argument-error paths.

Nothing here launches a kernel. The one call that passes argument checks
with placeholder pointers is skipped when a GPU is visible.
"""
import ctypes
import math
import os
import re
import subprocess

import numpy as np
import pytest

import paper_2607_21291_amd as P
from oracle import adadsf_oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "adadsf.h")


def _gpu():
    import torch
    return torch.cuda.is_available()


def test_library_exports_every_declared_symbol():
    text = open(HEADER).read()
    declared = set(re.findall(r"\b(dsf_[a-z0-9_]+)\s*\(", text))
    assert declared == set(P.EXPORTS)
    L = P.lib()
    for name in declared:
        assert getattr(L, name) is not None
    assert P.version() == 10000


def test_struct_layout_matches_c_header(tmp_path):
    src = tmp_path / "layout.cpp"
    src.write_text(
        '#include <cstdio>\n#include <cstddef>\n#include "adadsf.h"\n'
        "int main(){\n"
        ' std::printf("%zu %zu %zu %zu\\n", sizeof(dsf_layer_desc), offsetof(dsf_layer_desc, rope_theta),'
        " sizeof(dsf_layer_weights), offsetof(dsf_layer_weights, norm1_w));\n"
        ' std::printf("%zu %zu\\n", offsetof(dsf_layer_weights, w_down), offsetof(dsf_layer_weights, router_b2));\n'
        "}\n")
    exe = tmp_path / "layout"
    res = subprocess.run(["g++", "-std=c++17", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
                          "-I", "/opt/rocm/include", str(src), "-o", str(exe)], capture_output=True, text=True)
    if res.returncode != 0:
        pytest.skip("cannot compile against the HIP headers here: " + res.stderr[:200])
    out = subprocess.run([str(exe)], capture_output=True, text=True).stdout.split()
    got = [int(v) for v in out]
    assert got == [ctypes.sizeof(P.LayerDesc), P.LayerDesc.rope_theta.offset, ctypes.sizeof(P.LayerWeights),
                   P.LayerWeights.norm1_w.offset, P.LayerWeights.w_down.offset, P.LayerWeights.router_b2.offset]


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("tau", [None, 1.0, 0.25, 0.1, 0.05])
@pytest.mark.parametrize("clip", ["none", "plain", "budget"])
def test_host_allocation_matches_oracle(seed, tau, clip):
    rng = np.random.default_rng(seed)
    L = int(rng.integers(1, 40))
    s = rng.uniform(0.1, 0.99, L)
    t = float(rng.uniform(0.2, 0.95))
    ours = np.array(P.retention_from_similarity(list(s), t, tau, clip=clip))
    ref = O.retention_from_similarity(s, t, tau, clip=clip)
    np.testing.assert_allclose(ours, ref, rtol=1e-13, atol=1e-15)


def test_host_allocation_clip_case_and_workload_profiles():
    s = [0.9] * 3 + [0.3] * 9
    np.testing.assert_allclose(P.retention_from_similarity(s, 0.9, 0.05), [0.6] * 3 + [1.0] * 9, rtol=1e-13)
    r = P.retention_from_similarity(list(np.linspace(0.3, 0.9, 12)), 0.6, 0.25)
    assert [P.k_from_retention(x, 2048) for x in r] == [O.k_from_retention(x, 2048) for x in r]


def test_k_from_retention_matches_oracle():
    rng = np.random.default_rng(3)
    for _ in range(5000):
        r = float(rng.choice([rng.uniform(0, 1), round(rng.uniform(0, 1), 3), rng.integers(0, 101) / 100]))
        T = int(rng.integers(0, 9000))
        for mode in ("floor", "ceil"):
            assert P.k_from_retention(r, T, mode) == O.k_from_retention(r, T, mode)
    assert P.k_from_retention(0.29, 100) == 29
    with pytest.raises(P.DsfError):
        P.k_from_retention(float("nan"), 10)


def _desc(**kw):
    base = dict(block="neox_parallel", d_model=128, n_heads=4, n_kv_heads=4, head_dim=32, d_ff=512,
                rotary_dims=8, d_router=32, norm_eps=1e-5, rope_theta=1e4)
    base.update(kw)
    return P.make_desc(**base)


FAKE = 0x100000  # a 256-byte aligned placeholder address; never dereferenced by these tests


def _weights():
    kw = {n: FAKE for n in ("router_w1", "router_w2", "norm1_w", "norm2_w", "w_qkv", "w_o", "w_up", "w_down")}
    return P.LayerWeights(router_b2=0.0, reserved=0.0, **kw)


def _call_block(desc, weights, x=FAKE, B=2, T=64, k=32, flags=0, ws=FAKE, ws_bytes=None, dtype=P.F32):
    L = P.lib()
    if ws_bytes is None:
        ws_bytes = P.workspace_size(desc, dtype, B, T, k) if desc is not None else 1 << 30
    return L.dsf_sparse_block_forward(ctypes.addressof(desc) if desc is not None else None,
                                      ctypes.addressof(weights) if weights is not None else None, dtype, x, B,
                                      T, k, flags, None, None, None, ws, ws_bytes, None)


def test_error_paths_launch_nothing():
    d, w = _desc(), _weights()
    cases = [
        (dict(desc=None), 1),
        (dict(desc=_desc(head_dim=48)), 2),
        (dict(desc=_desc(n_kv_heads=3)), 1),
        (dict(desc=_desc(d_model=100)), 2),
        (dict(desc=_desc(d_ff=500)), 2),
        (dict(desc=_desc(rotary_dims=7)), 1),
        (dict(desc=_desc(d_router=40)), 2),
        (dict(k=65), 1),
        (dict(k=-1), 1),
        (dict(flags=1, k=32), 1),
        (dict(flags=4), 1),
        (dict(flags=3, k=64), 1),  # gating needs the router: not with DSF_FLAG_DENSE
        (dict(dtype=7), 2),
        (dict(ws_bytes=1024), 3),
        (dict(x=FAKE + 4), 1),
        (dict(x=None), 1),
        (dict(weights=None), 1),
    ]
    for kw, code in cases:
        args = dict(desc=d, weights=w)
        args.update(kw)
        rc = _call_block(**args)
        assert rc == code, (kw, rc, P.last_error())
        assert P.last_error()
    wq = _weights()
    wq.norm1_b = FAKE
    assert _call_block(_desc(block="qwen_seq", n_kv_heads=2), wq) == 1
    wn = _weights()
    wn.w_qkv = None
    assert _call_block(d, wn) == 1
    assert P.workspace_size(_desc(head_dim=48), P.F32, 2, 64, 32) == 0
    assert P.workspace_size(d, P.F32, 2, 64, 65) == 0


def test_error_paths_of_the_kernel_calls():
    L = P.lib()
    assert L.dsf_topk_select(FAKE, 2, 10, 11, FAKE, None) == 1
    assert L.dsf_gather_rows(FAKE, 1, 2, 10, 12, FAKE, 3, FAKE, None) == 2          # d % 8
    assert L.dsf_scatter_residual(FAKE, FAKE, 1, 2, 10, 16, FAKE, 11, None) == 1    # k > T
    assert L.dsf_router_score(FAKE, 1, 10, 64, 20, FAKE, None, FAKE, 0.0, FAKE, None) == 2
    assert L.dsf_attention_forward(FAKE, FAKE, FAKE, 1, 1, 6, 4, 8, 64, FAKE, None) == 1
    assert L.dsf_attention_forward(FAKE, FAKE, FAKE, 1, 1, 4, 4, 8, 96, FAKE, None) == 2
    assert L.dsf_sim_stats(FAKE, FAKE, 1, 100, 64, None, FAKE, FAKE, 0, None) == 3
    arr = (ctypes.c_double * 2)()
    assert L.dsf_retention_from_similarity(ctypes.addressof(arr), 2, 1.5, 0.1, 10.0, 2, ctypes.addressof(arr)) == 1
    # router-score pathway
    assert L.dsf_gate_score_grad(FAKE, FAKE, FAKE, 1, FAKE, FAKE, 2, 10, 3, 12, FAKE, None) == 2   # d % 8
    assert L.dsf_gate_score_grad(FAKE, FAKE, FAKE, 1, FAKE, FAKE, 2, 10, 11, 16, FAKE, None) == 1  # k > T
    assert L.dsf_gate_score_grad(FAKE + 4, FAKE, FAKE, 1, FAKE, FAKE, 2, 10, 3, 16, FAKE, None) == 1
    assert L.dsf_gate_score_grad(FAKE, FAKE, FAKE, 1, FAKE, FAKE, 2, 10, 3, 16, None, None) == 1
    assert L.dsf_router_backward_workspace_size(100, 64, 40) == 0
    assert L.dsf_router_backward_workspace_size(100, 60, 32) == 0
    assert L.dsf_router_backward_workspace_size(-1, 64, 32) == 0
    ws = L.dsf_router_backward_workspace_size(1000, 64, 32)
    assert ws >= 4 * (1000 * 32 + 16 * 65 + 32 * 64) and ws % 256 == 0
    rb = L.dsf_router_backward
    assert rb(FAKE, 1, 1000, 64, 40, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, ws, None) == 2
    assert rb(FAKE, 1, 1000, 64, 32, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, ws, None) == 1
    assert rb(FAKE, 1, 1000, 64, 32, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, ws - 4,
              None) == 3
    assert rb(FAKE, 1, 1000, 64, 32, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE + 16, ws,
              None) == 1
    assert rb(FAKE, 1, 1000, 64, 32, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE + 8, FAKE, ws,
              None) == 1
    assert rb(FAKE, 1, 1000, 64, 32, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, None, FAKE, ws, None) == 1
    # alignment objective
    assert L.dsf_align_workspace_size(-1) == 0 and L.dsf_align_workspace_size(1000) >= 8000
    assert L.dsf_align_hidden(FAKE, FAKE, 1, 100, 12, None, FAKE, FAKE, 1 << 20, None) == 2      # d % 8
    assert L.dsf_align_hidden(FAKE, FAKE, 1, 100, 8200, None, FAKE, FAKE, 1 << 20, None) == 2    # d > 8192
    assert L.dsf_align_hidden(FAKE, FAKE, 0, 100, 4104, None, FAKE, FAKE, 1 << 20, None) == 2    # fp32 d > 4096
    assert L.dsf_align_hidden(FAKE, FAKE, 1, 100, 64, None, FAKE, FAKE, 16, None) == 3           # workspace
    assert L.dsf_align_hidden(FAKE, FAKE, 1, 100, 64, None, None, FAKE, 1 << 20, None) == 1      # accum
    assert L.dsf_kl_align(FAKE, FAKE, 1, 10, 50257, None, FAKE, FAKE, 1 << 20, None) == 2        # C % 8
    assert L.dsf_kl_align(FAKE + 8, FAKE, 1, 10, 64, None, FAKE, FAKE, 1 << 20, None) == 1       # alignment
    assert L.dsf_align_hidden(None, None, 1, 0, 64, None, None, None, 0, None) == 0              # empty
    d = _desc()
    ks = (ctypes.c_int * 2)(32, 16)
    aws = L.dsf_align_stack_workspace_size(ctypes.addressof(d), P.F32, 2, 64)
    assert aws >= P.workspace_size(d, P.F32, 2, 64, 64)
    wts = (P.LayerWeights * 2)(_weights(), _weights())
    assert L.dsf_align_stack_forward(ctypes.addressof(d), ctypes.addressof(wts), 2, P.F32, ctypes.addressof(ks),
                                     FAKE, FAKE, 2, 64, 1, FAKE, FAKE, aws, None) == 1           # DENSE student
    assert L.dsf_align_stack_forward(ctypes.addressof(d), ctypes.addressof(wts), 2, P.F32, ctypes.addressof(ks),
                                     FAKE, FAKE, 2, 64, 0, FAKE, FAKE, aws - 256, None) == 3     # workspace
    assert L.dsf_align_stack_forward(ctypes.addressof(d), ctypes.addressof(wts), 2, P.F32, ctypes.addressof(ks),
                                     FAKE, FAKE, 2, 64, 0, None, FAKE, aws, None) == 1           # hid_accum
    # incremental decoding
    dws = L.dsf_decode_workspace_size(ctypes.addressof(d), P.F32, 4, 128, 64)
    assert dws > 0 and dws % 256 == 0
    assert L.dsf_decode_workspace_size(ctypes.addressof(d), P.F32, 4, 0, 64) == 0         # max_pos
    assert L.dsf_decode_workspace_size(ctypes.addressof(d), P.F32, 4, 128, 0) == 0        # cap
    assert L.dsf_decode_workspace_size(ctypes.addressof(d), P.F32, 4, 128, 65537) == 0    # cap above the limit
    assert L.dsf_decode_workspace_size(ctypes.addressof(_desc(head_dim=48)), P.F32, 4, 128, 64) == 0
    caches = (ctypes.c_void_p * 2)(FAKE, FAKE)
    bad = (ctypes.c_void_p * 2)(FAKE, FAKE + 8)
    ds = L.dsf_decode_step
    dargs = lambda **kw: [kw.get(n, v) for n, v in [
        ("desc", ctypes.addressof(d)), ("w", ctypes.addressof(wts)), ("L", 2), ("dtype", P.F32), ("x", FAKE),
        ("B", 4), ("pos", FAKE), ("max_pos", 128), ("thr", FAKE), ("sc", None), ("keep", None),
        ("ck", ctypes.addressof(caches)), ("cv", ctypes.addressof(caches)), ("len", FAKE), ("cap", 64),
        ("ws", FAKE), ("wsb", dws), ("s", None)]]
    assert ds(*dargs(ws=FAKE, wsb=dws - 256)) == 3                                         # workspace
    assert ds(*dargs(cv=ctypes.addressof(bad))) == 1                                       # cache alignment
    assert ds(*dargs(pos=None)) == 1
    assert ds(*dargs(thr=None)) == 1
    assert ds(*dargs(cap=0)) == 1
    assert ds(*dargs(cap=65537)) == 2
    assert ds(*dargs(x=FAKE + 4)) == 1
    assert ds(*dargs(dtype=7)) == 2
    assert ds(*dargs(B=0, x=None, pos=None, thr=None)) == 0                                # empty
    pws = P.workspace_size(d, P.F32, 2, 64, 32)
    sp = L.dsf_stack_prefill
    assert sp(ctypes.addressof(d), ctypes.addressof(wts), 2, P.F32, ctypes.addressof(ks), FAKE, 2, 64,
              ctypes.addressof(caches), ctypes.addressof(caches), FAKE, 16, None, FAKE, pws, None) == 1  # k > cap
    assert sp(ctypes.addressof(d), ctypes.addressof(wts), 2, P.F32, ctypes.addressof(ks), FAKE, 2, 64,
              ctypes.addressof(caches), ctypes.addressof(caches), None, 64, None, FAKE, pws, None) == 1  # cache_len
    assert sp(ctypes.addressof(d), ctypes.addressof(wts), 2, P.F32, ctypes.addressof(ks), FAKE, 2, 64,
              ctypes.addressof(caches), ctypes.addressof(caches), FAKE, 64, None, FAKE, pws - 256, None) == 3
    # empty problems are valid no-ops
    assert L.dsf_topk_select(None, 0, 10, 3, None, None) == 0
    assert L.dsf_gather_rows(None, 1, 2, 10, 16, None, 0, None, None) == 0
    assert _call_block(_desc(), _weights(), k=0) == 0


@pytest.mark.skipif(_gpu(), reason="placeholder pointers must never reach a real GPU")
def test_valid_arguments_without_gpu_report_no_device():
    assert _call_block(_desc(), _weights()) == 5
    assert "GPU" in P.last_error()


def test_workspace_status_rejects_null_pointers():
    L = P.lib()
    out = ctypes.c_uint32(7)
    assert L.dsf_workspace_status(None, ctypes.byref(out), None) == 1
    assert "null" in P.last_error()
    assert L.dsf_workspace_status(ctypes.c_void_p(256), None, None) == 1
    assert out.value == 7  # nothing written on an argument error


def test_backward_argument_errors():
    L = P.lib()
    d = _desc()
    assert L.dsf_backward_workspace_size(ctypes.addressof(d), P.F32, 2, 64, 32) == 0
    assert L.dsf_backward_workspace_size(ctypes.addressof(d), P.BF16, 2, 64, 65) == 0
    assert L.dsf_backward_workspace_size(ctypes.addressof(d), P.BF16, 2, 64, 32) > 0
    w = _weights()
    g = P.LayerGrads()
    args = lambda dtype, x, flags, scores: (ctypes.addressof(d), ctypes.addressof(w), dtype, x, x, 2, 64, 32,
                                            ctypes.c_void_p(256), scores, flags, x, ctypes.addressof(g),
                                            ctypes.c_void_p(256), 1 << 30, None)
    assert L.dsf_sparse_block_backward(*args(P.F32, ctypes.c_void_p(256), 0, None)) == 2
    assert L.dsf_sparse_block_backward(*args(P.BF16, None, 0, None)) == 1
    assert L.dsf_sparse_block_backward(*args(P.BF16, ctypes.c_void_p(256), P.FLAG_GATE, None)) == 1
    assert "scores" in P.last_error()
    assert L.dsf_sparse_block_backward(*args(P.BF16, ctypes.c_void_p(256), P.FLAG_DENSE, None)) == 1
