"""The schedules of the bf16 projection GEMMs give the layer the oracle
computes: one tile per workgroup; a persistent grid taking whole tiles; and
stream-K (a persistent grid whose workgroups split the k-iterations of the
last tiles and add partial sums in a fixed order). DSF_GEMM_SCHEDULE forces
one of them. On these small shapes the forced persistent grids leave most
workgroups no tile or a short or empty piece, so those paths all run, as do
the partial sums with many contributors per tile.

Stream-K adds the partials in an order fixed by the shape, so repeated runs
are bitwise equal. Whole tiles round exactly as one tile per workgroup. The
split schedule rounds differently, and every schedule is held to the oracle
at the bf16 tolerance.
"""
import pytest
import torch

import paper_2607_21291_amd as P
import synthetic as S

from gpu_util import TOL, announce, check_layer, make_desc, rel_inf, run_layer, to_np, workload, workspace

pytestmark = pytest.mark.gpu

CASES = [("neox_bf16_small", 150), ("qwen_bf16_small", 299), ("neox_bf16_hd128", 97), ("qwen_bf16_hd128", 129),
         ("neox_bf16_small", 1)]


@pytest.mark.parametrize("schedule", ["streamk", "persistent"])
@pytest.mark.parametrize("name,k", CASES)
def test_persistent_schedules_match_oracle(dev, monkeypatch, name, k, schedule):
    w = workload(name)
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w)
    monkeypatch.setenv("DSF_GEMM_SCHEDULE", schedule)
    announce(f"{schedule} layer {name} k={k}")
    y, scores, idx = run_layer(dev, w, W, x, k)
    check_layer(w, W, x, y, scores, idx, k)
    y2, _, _ = run_layer(dev, w, W, x, k)
    assert torch.equal(y, y2)
    monkeypatch.setenv("DSF_GEMM_SCHEDULE", "classic")
    announce(f"classic layer {name} k={k}")
    yc, _, idxc = run_layer(dev, w, W, x, k)
    assert torch.equal(idx, idxc)
    if schedule == "persistent":
        assert torch.equal(y, yc)  # whole tiles: the same arithmetic as one tile per workgroup
    assert rel_inf(to_np(y) - to_np(x), to_np(yc) - to_np(x)) < TOL[w.dtype]


@pytest.mark.parametrize("schedule", ["streamk", "persistent"])
@pytest.mark.parametrize("name", ["neox_bf16_small", "qwen_bf16_small"])
def test_persistent_stack_matches_layerwise(dev, monkeypatch, name, schedule):
    w = workload(name).replace(n_layers=3)
    monkeypatch.setenv("DSF_GEMM_SCHEDULE", schedule)
    announce(f"{schedule} stack {name}")
    Ws = S.stack_weights(w)
    x = S.hidden_states(w)
    T = w.seq
    ks = [T // 2, T - 3, max(1, T // 5)]
    dls = [P.DeviceLayer(W, dev) for W in Ws]
    xd = x.to(dev)
    ws = workspace(w, w.batch, T, max(ks), dev)
    P.stack_forward(make_desc(w), [dl.weights for dl in dls], ks, xd, ws)
    cur = x
    for W, k in zip(Ws, ks):
        y, _, _ = run_layer(dev, w, W, cur, k)
        cur = y.cpu()
    torch.cuda.synchronize()
    assert torch.equal(xd.cpu(), cur)


def test_full_size_schedules_agree(dev, monkeypatch):
    # in the first neox160m layer (M = 8 x 1563 rows) the automatic choice
    # takes stream-K for the down projection (588 tiles)
    w = S.WORKLOADS["neox160m"]
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w)
    k = 1563
    announce("full-size neox160m layer 0: auto vs classic schedule")
    ya, _, idxa = run_layer(dev, w, W, x, k)
    monkeypatch.setenv("DSF_GEMM_SCHEDULE", "classic")
    yc, _, idxc = run_layer(dev, w, W, x, k)
    assert torch.equal(idxa, idxc)
    assert rel_inf(to_np(ya) - to_np(x), to_np(yc) - to_np(x)) < TOL[w.dtype]


@pytest.mark.parametrize("name", ["neox_bf16_small", "tiny_neox_f32"])
def test_second_stream_matches_one_stream(dev, monkeypatch, name):
    # the NeoX up projection runs on the library's second stream beside QKV
    # and attention; the same kernels on the same inputs give the same bits
    w = workload(name).replace(n_layers=3)
    Ws = S.stack_weights(w)
    x = S.hidden_states(w)
    T = w.seq
    ks = [T // 2, T - 3, max(1, T // 5)]
    dls = [P.DeviceLayer(W, dev) for W in Ws]
    ws = workspace(w, w.batch, T, max(ks), dev)
    announce(f"two streams vs one: {name}")
    x2 = x.to(dev)
    P.stack_forward(make_desc(w), [dl.weights for dl in dls], ks, x2, ws)
    monkeypatch.setenv("DSF_SINGLE_STREAM", "1")
    x1 = x.to(dev)
    P.stack_forward(make_desc(w), [dl.weights for dl in dls], ks, x1, ws)
    torch.cuda.synchronize()
    assert torch.equal(x1, x2)


@pytest.mark.parametrize("name,k", [("neox_bf16_small", 150), ("qwen_bf16_small", 299)])
def test_streamk_wait_timeout_is_reported(dev, monkeypatch, name, k):
    # The stream-K finisher waits for earlier pieces' partial sums with a
    # bounded spin. DSF_SK_SPIN_LIMIT=0 makes every such wait give up at once
    # (nothing waits, every kernel exits normally): the tile is then written
    # without the missing partials and the call's status word says so. With
    # the default limit the same call reports nothing and matches the oracle.
    w = workload(name)
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w)
    B, T = x.shape[0], x.shape[1]
    dl = P.DeviceLayer(W, dev)
    ws = workspace(w, B, T, k, dev)
    monkeypatch.setenv("DSF_GEMM_SCHEDULE", "streamk")
    monkeypatch.setenv("DSF_SK_SPIN_LIMIT", "0")
    announce(f"stream-K give-up report {name} k={k}")
    xg = x.to(dev)
    P.sparse_block_forward(make_desc(w), dl.weights, xg, k, ws)
    assert P.workspace_status(ws) & P.WS_STATUS_SK_TIMEOUT
    monkeypatch.delenv("DSF_SK_SPIN_LIMIT")
    announce(f"stream-K default wait {name} k={k}")
    xd = x.to(dev)
    scores = torch.empty(B, T, dtype=torch.float32, device=dev)
    idx = torch.empty(B, k, dtype=torch.int32, device=dev)
    P.sparse_block_forward(make_desc(w), dl.weights, xd, k, ws, scores_out=scores, idx_out=idx)
    assert P.workspace_status(ws) == 0
    check_layer(w, W, x, xd, scores, idx, k)
    # the same stack call clears the word at its start
    P.stack_forward(make_desc(w), [dl.weights], [k], x.to(dev), ws)
    assert P.workspace_status(ws) == 0


@pytest.mark.parametrize("name,k", CASES)
def test_large_tiles_match_oracle(dev, monkeypatch, name, k):
    """256 x 256 tiles (eight 64 x 128 waves) forced onto the small shapes:
    every tile is ragged in M, most in N, and the SwiGLU grids hold whole
    128-unit tiles; the layer must match the oracle and repeat bitwise, and
    agree with the 128 x 128 tiles within tolerance."""
    w = workload(name)
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w)
    monkeypatch.setenv("DSF_GEMM_TILE", "large")
    announce(f"large tiles layer {name} k={k}")
    y, scores, idx = run_layer(dev, w, W, x, k)
    check_layer(w, W, x, y, scores, idx, k)
    y2, _, _ = run_layer(dev, w, W, x, k)
    assert torch.equal(y, y2)
    monkeypatch.setenv("DSF_GEMM_TILE", "small")
    monkeypatch.setenv("DSF_GEMM_SCHEDULE", "classic")
    ys, _, idxs = run_layer(dev, w, W, x, k)
    assert torch.equal(idx, idxs)
    assert rel_inf(to_np(y) - to_np(x), to_np(ys) - to_np(x)) < TOL[w.dtype]


@pytest.mark.parametrize("name", ["neox_bf16_small", "qwen_bf16_hd128"])
def test_large_tile_stack_matches_layerwise(dev, monkeypatch, name):
    w = workload(name).replace(n_layers=3)
    monkeypatch.setenv("DSF_GEMM_TILE", "large")
    announce(f"large tiles stack {name}")
    Ws = S.stack_weights(w)
    x = S.hidden_states(w)
    T = w.seq
    ks = [T // 2, T - 3, max(1, T // 5)]
    dls = [P.DeviceLayer(W, dev) for W in Ws]
    xd = x.to(dev)
    ws = workspace(w, w.batch, T, max(ks), dev)
    P.stack_forward(make_desc(w), [dl.weights for dl in dls], ks, xd, ws)
    cur = x
    for W, k in zip(Ws, ks):
        y, _, _ = run_layer(dev, w, W, cur, k)
        cur = y.cpu()
    torch.cuda.synchronize()
    assert torch.equal(xd.cpu(), cur)


# Shapes whose large-tile grids leave a ragged last round when 8 workgroups
# are taken as resident (DSF_GEMM_TAIL=force), with K deep enough to cut:
# NeoX (2200 kept rows, 9 tile rows): QKV 108 tiles and the fused O + down
# projection 36 tiles, each 4 tiles in 2 pieces; Qwen (2 x 600 kept rows, 5
# tile rows): QKV 35 tiles, 3 in 2 pieces; O 25 tiles, 1 in 2 pieces; down
# (K 2560) 25 tiles, 1 in 4 pieces. The up projections (16 x 9 tiles; the
# SwiGLU launch) are never split.
TAIL = {
    "neox_bf16_tail": (S.WORKLOADS["neox14b"].replace(
        name="neox_bf16_tail", n_layers=1, d_model=1024, n_heads=8, n_kv_heads=8, head_dim=128, d_ff=4096,
        rotary_dims=32, batch=1, seq=2400), 2200, {"gemm_qkv": 2, "gemm_up": 1, "gemm_down": 2}),
    "qwen_bf16_tail": (S.WORKLOADS["qwen7b"].replace(
        name="qwen_bf16_tail", n_layers=1, d_model=1280, n_heads=10, n_kv_heads=2, head_dim=128, d_ff=2560,
        rotary_dims=128, batch=2, seq=700), 600, {"gemm_qkv": 2, "gemm_o": 2, "gemm_up": 1, "gemm_down": 2}),
}


@pytest.mark.slow
@pytest.mark.parametrize("name", list(TAIL))
def test_split_last_round_matches_oracle(dev, monkeypatch, name):
    """The last round of large tiles cut along K into 2 or 4 pieces (a second
    launch whose finishers add the others' partial sums in piece order): the
    layer matches the oracle, repeats bitwise, and agrees with the unsplit
    grid within tolerance; the timing records show two launches for each
    split projection."""
    w, k, launches = TAIL[name]
    W = S.layer_weights(w, 0)
    x = S.hidden_states(w)
    monkeypatch.setenv("DSF_GEMM_TILE", "large")
    monkeypatch.setenv("DSF_GEMM_TAIL", "force")
    announce(f"split last round {name} k={k}")
    P.timing_enable(64)
    try:
        y, scores, idx = run_layer(dev, w, W, x, k)
        seen = {kind: P.timing_read(kind)[0] for kind in launches}
    finally:
        P.timing_enable(0)
    assert seen == launches
    check_layer(w, W, x, y, scores, idx, k)
    y2, _, _ = run_layer(dev, w, W, x, k)
    assert torch.equal(y, y2)
    monkeypatch.setenv("DSF_GEMM_TAIL", "0")
    y0, _, idx0 = run_layer(dev, w, W, x, k)
    assert torch.equal(idx, idx0)
    assert rel_inf(to_np(y) - to_np(x), to_np(y0) - to_np(x)) < TOL[w.dtype]


@pytest.mark.slow
def test_split_last_round_repeats_bitwise_at_full_size(dev):
    """GPT-NeoX-1.4B layer shape (4 x 1024 kept rows, QKV 16 x 24 large tiles
    on 256 resident workgroups: the last 128 tiles cut in 2), in the default
    launch configuration: the split runs, and repeated calls give the same
    bits. Every partial tile moves through 32 stores per lane, so a partial
    whose data registers were overwritten while being stored shows here."""
    w = S.WORKLOADS["neox14b"].replace(n_layers=1)
    k = 1024
    W = S.layer_weights(w, 0)
    dl = P.DeviceLayer(W, dev)
    x0 = S.hidden_states(w).to(dev)
    ws = workspace(w, w.batch, w.seq, k, dev)
    announce(f"split last round repeat neox14b k={k}")
    outs = []
    P.timing_enable(64)
    try:
        for i in range(4):
            x = x0.clone()
            P.stack_forward(make_desc(w), [dl.weights], [k], x, ws)
            torch.cuda.synchronize()
            assert P.workspace_status(ws) == 0
            if i == 0:
                assert P.timing_read("gemm_qkv")[0] == 2  # the split ran
            outs.append(x)
    finally:
        P.timing_enable(0)
    for y in outs[1:]:
        assert torch.equal(y, outs[0])


def test_host_threads_get_their_own_second_streams(dev):
    # each host thread gets its own second stream (destroyed when the thread
    # exits); threads on their own caller streams and workspaces give the
    # single-threaded result bitwise, and a later call on the main thread
    # still works after the worker threads have gone
    import threading
    w = workload("neox_bf16_small").replace(n_layers=2)
    Ws = S.stack_weights(w)
    x = S.hidden_states(w)
    ks = [w.seq // 2, w.seq // 3]
    dls = [P.DeviceLayer(W, dev) for W in Ws]
    weights = [dl.weights for dl in dls]
    announce("second streams of several host threads")
    ref = x.to(dev)
    ws0 = workspace(w, w.batch, w.seq, max(ks), dev)
    P.stack_forward(make_desc(w), weights, ks, ref, ws0)
    torch.cuda.synchronize()
    n = 4
    xdev = x.to(dev)
    outs = [torch.empty_like(xdev) for _ in range(n)]
    wss = [workspace(w, w.batch, w.seq, max(ks), dev) for _ in range(n)]
    streams = [torch.cuda.Stream(dev) for _ in range(n)]
    torch.cuda.synchronize()
    errors = []

    def work(i):
        try:
            with torch.cuda.stream(streams[i]):  # the copy and the stack on one stream
                for _ in range(3):
                    outs[i].copy_(xdev)
                    P.stack_forward(make_desc(w), weights, ks, outs[i], wss[i])
            streams[i].synchronize()
        except Exception as e:  # reported below, on the test's thread
            errors.append(e)

    threads = [threading.Thread(target=work, args=(i,)) for i in range(n)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    for i in range(n):
        assert torch.equal(outs[i], ref), i
    again = x.to(dev)
    P.stack_forward(make_desc(w), weights, ks, again, ws0)
    torch.cuda.synchronize()
    assert torch.equal(again, ref)
