"""The per-kind launch timing that the bench's breakdown reads: every kernel
class of a routed layer records its launches, each timed by its own
dispatch, and nothing is recorded while timing is off."""
import pytest
import torch

import paper_2607_21291_amd as P
import synthetic as S

from gpu_util import announce, make_desc, workload, workspace

pytestmark = pytest.mark.gpu

# launches per layer of each kind besides the routing (the NeoX norm launch
# writes LN1 and LN2; the Qwen block normalises twice); every call also
# builds its RoPE table ("other")
EXPECTED = {
    "neox_bf16_small": {"router": 1, "norm": 1, "gemm_qkv": 1, "attn": 1, "gemm_up": 1, "gemm_down": 1},
    "qwen_bf16_small": {"router": 1, "norm": 2, "gemm_qkv": 1, "attn": 1, "gemm_o": 1, "gemm_up": 1,
                        "gemm_down": 1},
}


@pytest.mark.parametrize("name,T", [("neox_bf16_small", 300), ("neox_bf16_small", 256), ("qwen_bf16_small", 300)])
def test_layer_kinds_are_timed(dev, name, T):
    """Router and Top-K are one launch for sequences of a multiple of 64
    tokens up to 4096 and two launches otherwise."""
    announce(f"timing {name} T={T}")
    w = workload(name).replace(seq=T)
    expected = dict(EXPECTED[name], other=1)
    if T % 64 or T > 4096:
        expected["topk"] = 1
    W = S.layer_weights(w, 0)
    dl = P.DeviceLayer(W, dev)
    k = w.seq // 2
    xd = S.hidden_states(w).to(dev)
    ws = workspace(w, w.batch, w.seq, k, dev)
    reps = 3
    P.timing_enable(64 * reps)
    try:
        for _ in range(reps):
            P.sparse_block_forward(make_desc(w), dl.weights, xd, k, ws)
        torch.cuda.synchronize()
        seen = {}
        for kind in P.KINDS:
            n, ms = P.timing_read(kind)
            if n:
                seen[kind] = (n, ms)
    finally:
        P.timing_enable(0)
    assert {kk: v[0] for kk, v in seen.items()} == {kk: reps * v for kk, v in expected.items()}
    for kind, (n, ms) in seen.items():
        assert 0.0 < ms / n < 50.0, f"{kind}: {ms / n} ms per launch"
    # disarmed: nothing more is recorded
    P.sparse_block_forward(make_desc(w), dl.weights, xd, k, ws)
    torch.cuda.synchronize()
    assert all(P.timing_read(kind)[0] == 0 for kind in P.KINDS)
