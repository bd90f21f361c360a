"""A decode step captured into a HIP graph (torch.cuda.CUDAGraph) and
replayed: every replay must equal the same step run eagerly, bit for bit.

dsf_decode_step launches kernels only, on the caller's stream (no memset,
copy, synchronisation or second stream), so a caller may capture it. The
graph is replayed several times with eager work between the replays (the
next token and its position are copied into the captured input buffers, the
outputs copied out) and each replay is checked against an eager twin that
started from the same prefill: the hidden states, the keep decisions, the
cache lengths and, at the end, the caches.
"""
import pytest
import torch

import paper_2607_21291_amd as P
import synthetic as S

from gpu_util import announce, dtype_code, make_desc, workload, workspace

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["neox_bf16_small", "qwen_bf16_small"])
def test_captured_decode_step_replays_match_eager(dev, name):
    w = workload(name).replace(n_layers=3)
    L, B, T0, N = 3, 3, 64, 6
    ks = [40, 24, 50]
    cap = T0 + N + 1
    Ws = S.stack_weights(w)
    dls = [P.DeviceLayer(W, dev) for W in Ws]
    desc = make_desc(w)
    weights = [dl.weights for dl in dls]
    x = S.hidden_states(w, batch=B, seq=T0 + N, seed_offset=11)
    dt = w.torch_dtype
    ck = [torch.zeros(B, w.n_kv_heads, cap, w.head_dim, dtype=dt, device=dev) for _ in range(L)]
    cv = [torch.zeros(B, w.n_kv_heads, cap, w.head_dim, dtype=dt, device=dev) for _ in range(L)]
    clen = torch.zeros(L, B, dtype=torch.int32, device=dev)
    thr = torch.empty(L, B, dtype=torch.float32, device=dev)
    announce(f"decode graph {name}: prefill")
    P.stack_prefill(desc, weights, ks, x[:, :T0].to(dev).contiguous(), ck, cv, clen, workspace(w, B, T0, max(ks), dev),
                    thr_out=thr)
    torch.cuda.synchronize()
    # eager twin and graph state start from the same prefill
    ck2, cv2, clen2 = [t.clone() for t in ck], [t.clone() for t in cv], clen.clone()
    ws = torch.empty(P.decode_workspace_size(desc, dtype_code(w), B, cap, cap), dtype=torch.uint8, device=dev)
    ws2 = torch.empty_like(ws)
    toks = [x[:, T0 + t].to(dev).contiguous() for t in range(N)]
    # step 0 eagerly on both states (it also settles any first-call setup)
    keep_e = torch.zeros(L, B, dtype=torch.int32, device=dev)
    xe = toks[0].clone()
    P.decode_step(desc, weights, xe, torch.full((B,), T0, dtype=torch.int32, device=dev), cap, thr, ck, cv, clen, ws,
                  keep_out=keep_e)
    xs = toks[0].clone()
    pos_s = torch.full((B,), T0, dtype=torch.int32, device=dev)
    keep_s = torch.zeros(L, B, dtype=torch.int32, device=dev)
    P.decode_step(desc, weights, xs, pos_s, cap, thr, ck2, cv2, clen2, ws2, keep_out=keep_s)
    torch.cuda.synchronize()
    assert torch.equal(xs, xe) and torch.equal(keep_s, keep_e) and torch.equal(clen2, clen)
    announce(f"decode graph {name}: capture")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        P.decode_step(desc, weights, xs, pos_s, cap, thr, ck2, cv2, clen2, ws2, keep_out=keep_s)
    for t in range(1, N):
        announce(f"decode graph {name}: replay {t}")
        xe = toks[t].clone()
        P.decode_step(desc, weights, xe, torch.full((B,), T0 + t, dtype=torch.int32, device=dev), cap, thr, ck, cv, clen,
                      ws, keep_out=keep_e)
        xs.copy_(toks[t])
        pos_s.fill_(T0 + t)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(xs, xe), f"replay {t}: hidden states"
        assert torch.equal(keep_s, keep_e), f"replay {t}: keep decisions"
        assert torch.equal(clen2, clen), f"replay {t}: cache lengths"
    for l in range(L):
        assert torch.equal(ck2[l], ck[l]) and torch.equal(cv2[l], cv[l])
    assert keep_e.any() or clen.sum() > sum(ks) * B
