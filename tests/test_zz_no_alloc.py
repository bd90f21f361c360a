"""dsf_decode_step_static, the decode step that allocates nothing (its scratch
is the library's static device array), against dsf_decode_step with a
workspace: same prompt caches, same tokens, bitwise-equal hidden states,
scores, keep decisions, caches and cache lengths. Two calls in a row, the
second with fewer sequences than the first, on both block families; and a
step too large for the static array is refused before anything runs."""
import pytest
import torch

import paper_2607_21291_amd as P
import synthetic as S

from gpu_util import announce, dtype_code, make_desc, workload, workspace

pytestmark = pytest.mark.gpu


def _state(w, dls, B, T0, ks, cap, dev):
    desc = make_desc(w)
    L = len(dls)
    ck = [torch.zeros(B, w.n_kv_heads, cap, w.head_dim, dtype=w.torch_dtype, device=dev) for _ in range(L)]
    cv = [torch.zeros_like(c) for c in ck]
    clen = torch.zeros(L, B, dtype=torch.int32, device=dev)
    thr = torch.empty(L, B, dtype=torch.float32, device=dev)
    xp = S.hidden_states(w, batch=B, seq=T0, seed_offset=3).to(dev).contiguous()
    P.stack_prefill(desc, [dl.weights for dl in dls], ks, xp, ck, cv, clen, workspace(w, B, T0, max(ks), dev),
                    thr_out=thr)
    torch.cuda.synchronize()
    return ck, cv, clen, thr


def _clone(st):
    ck, cv, clen, thr = st
    return [c.clone() for c in ck], [c.clone() for c in cv], clen.clone(), thr.clone()


@pytest.mark.parametrize("name", ["neox_bf16_small", "qwen_bf16_small"])
def test_static_decode_step_equals_workspace_step(dev, name):
    w = workload(name).replace(n_layers=2)
    L, T0, cap = 2, 64, 80
    ks = [40, 24]
    desc = make_desc(w)
    dls = [P.DeviceLayer(S.layer_weights(w, l), dev) for l in range(L)]
    weights = [dl.weights for dl in dls]
    for call, B in enumerate((4, 2)):  # the second call with a smaller batch
        ref = _state(w, dls, B, T0, ks, cap, dev)
        got = _clone(ref)
        g = torch.Generator().manual_seed(100 + call)
        tok = (torch.randn(B, w.d_model, generator=g) * 0.02).to(w.torch_dtype).to(dev)
        pos = torch.full((B,), T0, dtype=torch.int32, device=dev)
        thr = ref[3].clone()
        thr[:, 0] = -float("inf")  # sequence 0 keeps its token in every layer
        x_ref, x_got = tok.clone(), tok.clone()
        sc_ref, sc_got = (torch.full((L, B), float("nan"), device=dev) for _ in range(2))
        ko_ref, ko_got = (torch.full((L, B), -1, dtype=torch.int32, device=dev) for _ in range(2))
        ws = torch.empty(P.decode_workspace_size(desc, dtype_code(w), B, cap, cap), dtype=torch.uint8, device=dev)
        announce(f"decode step with workspace {name} B={B}")
        P.decode_step(desc, weights, x_ref, pos, cap, thr, ref[0], ref[1], ref[2], ws, scores_out=sc_ref,
                      keep_out=ko_ref)
        torch.cuda.synchronize()
        announce(f"decode step on static scratch {name} B={B} (call {call + 1})")
        P.decode_step_static(desc, weights, x_got, pos, cap, thr, got[0], got[1], got[2], scores_out=sc_got,
                             keep_out=ko_got)
        torch.cuda.synchronize()
        assert ko_ref[:, 0].eq(1).all()
        assert torch.equal(x_ref, x_got)
        assert torch.equal(sc_ref, sc_got) and torch.equal(ko_ref, ko_got)
        assert torch.equal(ref[2], got[2])
        for l in range(L):
            assert torch.equal(ref[0][l], got[0][l]) and torch.equal(ref[1][l], got[1][l])


def test_static_decode_step_refuses_oversized_steps(dev):
    w = workload("qwen_bf16_small").replace(n_layers=1)
    desc = make_desc(w)
    dl = P.DeviceLayer(S.layer_weights(w, 0), dev)
    B, cap = 2, 16
    big_pos = 1 << 20  # a RoPE table of 2^20 positions alone exceeds the static scratch
    assert P.decode_workspace_size(desc, dtype_code(w), B, big_pos, cap) > P.decode_static_scratch_bytes()
    assert P.decode_static_scratch_bytes() == 32 << 20
    ck = [torch.zeros(B, w.n_kv_heads, cap, w.head_dim, dtype=w.torch_dtype, device=dev)]
    cv = [torch.zeros_like(ck[0])]
    clen = torch.zeros(1, B, dtype=torch.int32, device=dev)
    thr = torch.zeros(1, B, device=dev)
    x = torch.zeros(B, w.d_model, dtype=w.torch_dtype, device=dev)
    pos = torch.zeros(B, dtype=torch.int32, device=dev)
    announce("static decode step: oversized request")
    with pytest.raises(P.DsfError) as e:
        P.decode_step_static(desc, [dl.weights], x, pos, big_pos, thr, ck, cv, clen)
    assert e.value.code == 3
    torch.cuda.synchronize()
    assert clen.eq(0).all() and x.eq(0).all()
