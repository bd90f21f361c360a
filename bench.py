#!/usr/bin/env python3
"""Depth-sparse stack throughput on one MI355X.

One step is one forward pass of the whole depth-sparse stack (router, Top-K,
gather + norm, QKV + RoPE, attention over kept tokens, output and FFN
projections, residual scatter, for every layer) over one batch of synthetic
hidden states at fixed per-layer retention. The retention ratios come from
the allocation of Eqs. 5-8 (run by the library's host code) on the
workload's similarity profile, or on similarities measured by the GPU
calibration pass (similarity statistic of Eq. 4 on the dense stack), which is
timed separately and reported as `calibration_ms`.

Inputs are resident in HBM before the timed region: every timed step runs on
its own pristine copy of the hidden states, prepared beforehand.

Prints one JSON line. `roofline` is for the dominant kernel (the last GEMM
of each layer, which for GPT-NeoX fuses the attention-output and FFN-down
projections along K), timed with HIP events around each of its launches
inside the timed region. `cpu_baseline` times the CPU oracle on a bounded
sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "depth-sparse stack tokens/sec at fixed r_l; MFMA util % and HBM GB/s % of peak"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


# HBM traffic of the dominant kernel, from two rocprofv3 passes (FETCH_SIZE,
# then WRITE_SIZE, per dispatch) scaled by what the same counters read for the
# library's plain copy kernel of known size. It holds only for the workload
# and the GEMM source it was measured on (SHA-256 of kernels_gemm.hip); for
# anything else `traffic` is null.
TRAFFIC_MEASURED = {"workload": "neox160m", "bytes_per_launch": 2.081e+08,
                    "gemm_source_sha256": "4cfa901f97fd6118d3472e7a082a1b59925dfe53fabfeb111c792a6825a9b490",
                    "profile": "profiles/gemm_down_neox160m.md"}


def gemm_source_sha256():
    import hashlib
    path = os.path.join(ROOT, "paper_2607_21291_amd", "csrc", "kernels_gemm.hip")
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(workload):
    t = TRAFFIC_MEASURED
    if not t or t["workload"] != workload or t["gemm_source_sha256"] != gemm_source_sha256():
        return None
    return t["bytes_per_launch"]


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def retention(P, w, calib_s=None):
    if w.retention is not None:
        return list(w.retention)
    s = calib_s if w.similarity is None else list(w.similarity)
    return P.retention_from_similarity(s, w.target, w.tau)


def streaming_rates(P, C, w, k, dev, weights0, reps=3):
    """The HBM-bound entry points standalone, against HBM peak: router, Top-K,
    gather, scatter and the similarity statistic, on one layer's shapes
    (B, T, d, k). "cold": each launch reads its own input buffer, cycling
    through copies that together exceed 1 GiB (more than the 256 MB MALL),
    so reads come from HBM; "hot": every launch on the same buffer."""
    import torch
    B, T, d = w.batch, w.seq, w.d_model
    eb = 4 if w.dtype == "f32" else 2
    xbytes = B * T * d * eb
    R = max(4, -(-(1 << 30) // xbytes) + 1)
    xs = [torch.randn(B, T, d, device=dev).mul_(0.02).to(w.torch_dtype) for _ in range(R)]
    scs = [torch.randn(B, T, device=dev) for _ in range(R)]
    idx = torch.stack([torch.sort(torch.randperm(T, device=dev)[:k])[0] for _ in range(B)]).to(torch.int32)
    delta = torch.randn(B, k, d, device=dev).mul_(0.02).to(w.torch_dtype)
    gout = torch.empty(B, k, d, device=dev, dtype=w.torch_dtype)
    scores = torch.empty(B, T, device=dev)
    idx_out = torch.empty(B, k, dtype=torch.int32, device=dev)
    accum = torch.zeros(2, dtype=torch.float64, device=dev)
    simws = torch.empty(max(P.sim_workspace_size(B * T), 256), dtype=torch.uint8, device=dev)
    W = {key: (v.to(dev) if hasattr(v, "to") else v) for key, v in weights0.items()
         if key.startswith("router_")}
    ops = {
        "router": (lambda i: P.router_score(xs[i], W["router_w1"], W["router_b1"], W["router_w2"],
                                            float(W["router_b2"]), scores), C.router_bytes(w, B, T)),
        "topk": (lambda i: P.topk_select(scs[i], k, idx_out), C.topk_bytes(w, B, T, k)),
        "gather": (lambda i: P.gather_rows(xs[i], idx, gout), 2.0 * eb * B * k * d + 4.0 * B * k),
        "scatter": (lambda i: P.scatter_residual(xs[i], delta, idx), 3.0 * eb * B * k * d + 4.0 * B * k),
        "sim": (lambda i: P.sim_stats(xs[i], xs[(i + 1) % R], accum, workspace=simws), C.sim_bytes(w, B, T)),
    }
    out = {}
    for name, (fn, nbytes) in ops.items():
        res = {"bytes_per_launch": nbytes}
        for mode in ("cold", "hot"):
            for i in range(min(R, 4)):
                fn(i if mode == "cold" else 0)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            n = R * reps
            torch.cuda.synchronize()
            e0.record()
            for i in range(n):
                fn(i % R if mode == "cold" else 0)
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / n
            gbs = nbytes / (us * 1e-6) / 1e9
            res[mode] = {"us": us, "GB/s": gbs, "frac_of_hbm_peak": gbs / PEAK_HBM_GBS}
        out[name] = res
    del xs, scs
    torch.cuda.empty_cache()
    return out


def _timed(fn, n_calls, reps_of):
    """Mean microseconds per call of fn(i) over n_calls calls (torch events)."""
    import torch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for i in range(n_calls):
        fn(reps_of(i))
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / n_calls


def router_pathway(P, C, w, ks, dev, desc, weights, x0, ws, ms_plain, steps, weights0):
    """The training-side router-score pathway (Section 3.4): the score-gated
    stack against the plain one, and the gate score gradient and the router
    backward standalone on one layer's shapes, cold (inputs cycled through
    more than 1 GiB of copies) and hot."""
    import torch
    B, T, d = w.batch, w.seq, w.d_model
    eb = 4 if w.dtype == "f32" else 2
    out = {}
    # gated stack, same k per layer
    xg = [x0.clone() for _ in range(steps)]
    xw = x0.clone()
    P.stack_forward(desc, weights, ks, xw, ws, flags=P.FLAG_GATE)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        P.stack_forward(desc, weights, ks, xg[i], ws, flags=P.FLAG_GATE)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    out["gated_stack"] = {"ms_per_step": ms, "tokens_per_s": B * T / (ms / 1e3), "vs_plain": ms / ms_plain}
    del xg, xw
    # gate score gradient at the mean k
    k = int(round(sum(ks) / len(ks)))
    rows = B * T * d * eb
    R = max(4, -(-(1 << 30) // (3 * rows)) + 1)
    dys = [torch.randn(B, T, d, device=dev).to(w.torch_dtype) for _ in range(R)]
    xis = [torch.randn(B, T, d, device=dev).to(w.torch_dtype) for _ in range(R)]
    xos = [torch.randn(B, T, d, device=dev).to(w.torch_dtype) for _ in range(R)]
    sc = torch.randn(B, T, device=dev)
    idx = torch.stack([torch.sort(torch.randperm(T, device=dev)[:k])[0] for _ in range(B)]).to(torch.int32)
    dsc = torch.empty(B, T, device=dev)
    fn = lambda i: P.gate_score_grad(dys[i], xis[i], xos[i], sc, idx, dsc)
    nbytes = C.gate_grad_bytes(w, B, T, k)
    res = {"k": k, "bytes_per_call": nbytes}
    for mode in ("cold", "hot"):
        fn(0)
        us = _timed(fn, 3 * R, (lambda i: i % R) if mode == "cold" else (lambda i: 0))
        res[mode] = {"us": us, "GB/s": nbytes / (us * 1e-6) / 1e9, "frac_of_hbm_peak": nbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS}
    out["gate_score_grad"] = res
    del dys, xis, xos
    # router backward over every token of the batch
    n = B * T
    W = {key: v.to(dev) for key, v in weights0.items() if key.startswith("router_") and hasattr(v, "to")}
    R = max(4, -(-(1 << 30) // (2 * rows)) + 1)
    xr = [torch.randn(B, T, d, device=dev).mul_(0.02).to(w.torch_dtype) for _ in range(R)]
    dxr = [torch.zeros(B, T, d, device=dev, dtype=w.torch_dtype) for _ in range(R)]
    dsr = torch.randn(n, device=dev)
    g = {name: torch.empty(shape, device=dev) for name, shape in
         (("dw1", (w.d_router, d)), ("db1", (w.d_router,)), ("dw2", (w.d_router,)), ("db2", (1,)))}
    rws = torch.empty(P.router_backward_workspace_size(n, d, w.d_router), dtype=torch.uint8, device=dev)
    fn = lambda i: P.router_backward(xr[i], W["router_w1"], W["router_b1"], W["router_w2"], dsr, g["dw1"], g["db1"],
                                     g["dw2"], g["db2"], dx=dxr[i], workspace=rws)
    nbytes, nflops = C.router_bwd_bytes(w, n), C.router_bwd_flops(w, n)
    res = {"n_tokens": n, "bytes_per_call": nbytes, "flops_per_call": nflops}
    for mode in ("cold", "hot"):
        fn(0)
        us = _timed(fn, 3 * R, (lambda i: i % R) if mode == "cold" else (lambda i: 0))
        res[mode] = {"us": us, "GB/s": nbytes / (us * 1e-6) / 1e9, "frac_of_hbm_peak": nbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS,
                     "TFLOP/s": nflops / (us * 1e-6) / 1e12}
    # the three launches of one call, on the library's event timing
    P.timing_enable(64, ["backward"])
    for i in range(8):
        fn(i % R)
    torch.cuda.synchronize()
    nb, msb = P.timing_read("backward")
    P.timing_enable(0)
    res["timed_calls"] = {"calls": nb, "us_per_call": msb * 1e3 / max(nb, 1)}
    out["router_backward"] = res
    del xr, dxr
    torch.cuda.empty_cache()
    return out


# vocabulary sizes of the two model families (logit rows of Eq. 10)
VOCAB = {"neox_parallel": 50304, "qwen_seq": 151936}


def alignment_objective(P, C, w, ks, dev, desc, weights, x0, ms_plain, steps):
    """Section 3.5: the dense-teacher / sparse-student stack with Eq. 9 per
    layer, against the sparse stack alone; and the Eq. 9 and Eq. 10 kernels
    standalone (Eq. 10 on synthetic logits of the model family's vocabulary
    for every token of the batch)."""
    import torch
    B, T, d = w.batch, w.seq, w.d_model
    eb = 4 if w.dtype == "f32" else 2
    dcode = P.F32 if w.dtype == "f32" else P.BF16
    out = {}
    ws = torch.empty(P.align_stack_workspace_size(desc, dcode, B, T), dtype=torch.uint8, device=dev)
    hid = torch.zeros(w.n_layers, dtype=torch.float64, device=dev)
    xs, xt = x0.clone(), x0.clone()
    P.align_stack_forward(desc, weights, ks, xs, xt, hid, ws)
    n_steps = max(2, steps)
    pairs = [(x0.clone(), x0.clone()) for _ in range(n_steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for a, b in pairs:
        P.align_stack_forward(desc, weights, ks, a, b, hid, ws)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / n_steps
    out["align_stack"] = {"ms_per_step": ms, "tokens_per_s": B * T / (ms / 1e3), "vs_sparse_stack": ms / ms_plain,
                          "note": "dense teacher + sparse student + Eq. 9 per layer"}
    del pairs, ws
    # Eq. 9 kernel standalone, cold (inputs cycled through > 1 GiB) and hot
    n = B * T
    nbytes = C.align_hidden_bytes(w, n)
    R = max(4, -(-(1 << 30) // int(nbytes)) + 1)
    hs = [torch.randn(B, T, d, device=dev).to(w.torch_dtype) for _ in range(R)]
    hd = [torch.randn(B, T, d, device=dev).to(w.torch_dtype) for _ in range(R)]
    acc = torch.zeros(1, dtype=torch.float64, device=dev)
    aws = torch.empty(P.align_workspace_size(n), dtype=torch.uint8, device=dev)
    fn = lambda i: P.align_hidden(hs[i], hd[i], acc, workspace=aws)
    res = {"bytes_per_call": nbytes}
    for mode in ("cold", "hot"):
        fn(0)
        us = _timed(fn, 3 * R, (lambda i: i % R) if mode == "cold" else (lambda i: 0))
        res[mode] = {"us": us, "GB/s": nbytes / (us * 1e-6) / 1e9, "frac_of_hbm_peak": nbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS}
    out["align_hidden"] = res
    del hs, hd
    # Eq. 10 over B*T rows of the family's vocabulary (each call streams far more than the MALL)
    V = VOCAB[w.block]
    ld = torch.randn(n, V, device=dev).mul_(3.0).to(w.torch_dtype)
    ls = (ld.float() + torch.randn(n, V, device=dev).mul_(0.5)).to(w.torch_dtype)
    kws = torch.empty(P.align_workspace_size(n), dtype=torch.uint8, device=dev)
    fn = lambda i: P.kl_align(ld, ls, acc, workspace=kws)
    nbytes = C.kl_align_bytes(eb, n, V)
    fn(0)
    us = _timed(fn, 3, lambda i: 0)
    out["kl_align"] = {"rows": n, "classes": V, "bytes_per_call": nbytes, "us": us,
                       "GB/s": nbytes / (us * 1e-6) / 1e9, "frac_of_hbm_peak": nbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS}
    del ld, ls
    torch.cuda.empty_cache()
    return out


def decode_leg(P, C, w, ks, dev, desc, weights, x0, steps):
    """Incremental decoding (the paper treats prefill only): the stack is
    prefilled over the batch's T tokens into per-layer caches of the kept
    tokens' keys and values, with thresholds = the lowest kept score of each
    (layer, sequence); then decode steps of one new synthetic token per
    sequence, routed by those thresholds on the device. Bytes per step: every
    layer's weights once plus the cached keys and values the step reads."""
    import torch
    B, T, L = w.batch, w.seq, w.n_layers
    dcode = P.F32 if w.dtype == "f32" else P.BF16
    warm = 3
    n = warm + steps
    cap = T + n + steps + 1  # eager steps, then as many replays of a captured step
    ck = [torch.empty(B, w.n_kv_heads, cap, w.head_dim, dtype=w.torch_dtype, device=dev) for _ in range(L)]
    cv = [torch.empty(B, w.n_kv_heads, cap, w.head_dim, dtype=w.torch_dtype, device=dev) for _ in range(L)]
    clen = torch.zeros(L, B, dtype=torch.int32, device=dev)
    thr = torch.empty(L, B, dtype=torch.float32, device=dev)
    x = x0.clone()
    wsp = torch.empty(P.workspace_size(desc, dcode, B, T, max(ks)), dtype=torch.uint8, device=dev)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    P.stack_prefill(desc, weights, ks, x, ck, cv, clen, wsp, thr_out=thr)
    torch.cuda.synchronize()
    prefill_ms = (time.perf_counter() - t0) * 1e3
    del wsp
    lens0 = clen.cpu().numpy()
    ws = torch.empty(P.decode_workspace_size(desc, dcode, B, cap, cap), dtype=torch.uint8, device=dev)
    g = torch.Generator().manual_seed(1234)
    toks = [(torch.randn(B, w.d_model, generator=g) * 0.02).to(w.torch_dtype).to(dev) for _ in range(n)]
    pos = [torch.full((B,), T + i, dtype=torch.int32, device=dev) for i in range(n)]
    keep = torch.zeros(n, L, B, dtype=torch.int32, device=dev)
    for i in range(warm):
        P.decode_step(desc, weights, toks[i], pos[i], cap, thr, ck, cv, clen, ws, keep_out=keep[i])
    lens_start = clen.cpu().numpy()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for i in range(warm, n):
        P.decode_step(desc, weights, toks[i], pos[i], cap, thr, ck, cv, clen, ws, keep_out=keep[i])
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    lens_end = clen.cpu().numpy()
    mean_lens = ((lens_start + lens_end) / 2.0).tolist()
    nbytes = C.decode_step_bytes(w, B, mean_lens)
    gbs = nbytes / (ms * 1e-3) / 1e9
    kept = keep[warm:].float().mean().item()
    # the same step captured into a HIP graph and replayed, the next token
    # and its position copied into the captured buffers before each replay
    xg, posg, keepg = toks[0].clone(), pos[0].clone(), torch.zeros(L, B, dtype=torch.int32, device=dev)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        P.decode_step(desc, weights, xg, posg, cap, thr, ck, cv, clen, ws, keep_out=keepg)
    torch.cuda.synchronize()
    e0.record()
    for i in range(steps):
        xg.copy_(toks[i % n])
        posg.fill_(T + n + i)
        graph.replay()
    e1.record()
    torch.cuda.synchronize()
    ms_graph = e0.elapsed_time(e1) / steps
    del graph
    del ck, cv, toks, ws
    torch.cuda.empty_cache()
    return {"tokens_per_s": B / (ms / 1e3), "ms_per_step": ms, "batch": B, "prefill_tokens": T,
            "graph": {"ms_per_step": ms_graph, "tokens_per_s": B / (ms_graph / 1e3),
                      "note": "one captured decode step replayed; each replay preceded by two small copies"},
            "prefill_ms": prefill_ms, "steps": steps, "cache_capacity": cap,
            "cache_len_after_prefill_mean": float(lens0.mean()), "kept_fraction_decode": kept,
            "roofline": {"bound": "hbm", "bytes_per_step": nbytes, "achieved": gbs, "peak": PEAK_HBM_GBS,
                         "unit": "GB/s", "frac": gbs / PEAK_HBM_GBS},
            "note": "routing rule at decode time (not in the paper): keep iff score >= the prefill's lowest kept "
                    "score of that (layer, sequence)"}


def cpu_baseline(w, ks, layers, min_seconds=10.0):
    """The oracle, as it stands, on whole sequences through `layers` layers.

    Sequences 0, 1, ... are run one after another until at least
    `min_seconds` have elapsed or the batch is exhausted, which bounds the
    sample to roughly 10-30 s of CPU work on any host.
    """
    from threadpoolctl import threadpool_info

    import synthetic as S
    from oracle import adadsf_oracle as O

    desc = dict(block=w.block, n_heads=w.n_heads, n_kv_heads=w.n_kv_heads, head_dim=w.head_dim, d_ff=w.d_ff,
                rotary_dims=w.rotary_dims, rope_theta=w.rope_theta, norm_eps=w.norm_eps)
    Ws = [{k: (O.f64(v) if hasattr(v, "detach") else v) for k, v in S.layer_weights(w, l).items()}
          for l in range(layers)]
    xall = S.hidden_states(w)
    dt, nseq = 0.0, 0
    while nseq < w.batch and dt < min_seconds:
        x = O.f64(xall[nseq:nseq + 1])
        t0 = time.perf_counter()
        for l in range(layers):
            x = O.routed_layer(desc, Ws[l], x, ks[l])["y"]
        dt += time.perf_counter() - t0
        nseq += 1
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    tokens = nseq * w.seq * layers / w.n_layers        # stack-equivalent tokens
    return {"value": tokens / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"sequences 0..{nseq - 1} of {w.batch} ({w.seq} tokens each) through layers 0..{layers - 1} "
                      f"of {w.n_layers}, run until >= {min_seconds:.0f} s; {dt:.1f} s for {tokens:.0f} "
                      f"stack-equivalent tokens",
            "seconds": dt, "cpu_count": os.cpu_count()}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="neox160m")
    ap.add_argument("--retention", type=float, default=None,
                    help="uniform retention r for every layer (skips the allocation and the calibration pass)")
    ap.add_argument("--batch", type=int, default=None, help="override the workload's batch")
    ap.add_argument("--seq", type=int, default=None, help="override the workload's sequence length")
    ap.add_argument("--cpu-layers", type=int, default=None, help="layers of the CPU oracle sample (default all)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-dense", action="store_true", help="skip the dense-stack comparison run")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the standalone sections (streaming entry points, router-score pathway, alignment "
                         "objective); used for the counter passes")
    ap.add_argument("--only-sparse", action="store_true",
                    help="launch only the sparse stack (warmup + timed steps): no calibration pass when the "
                         "workload fixes its similarity profile, no dense run, no breakdown pass, no CPU "
                         "baseline; used under rocprofv3 so every launch it sees is a timed-shape launch")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the depth-sparse stack is data-parallel over sequences with no "
              "exchange in the forward pass, so this build runs and reports the single-GPU shard "
              "(--gpus 1).", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2607_21291_amd as P
    import synthetic as S
    from paper_2607_21291_amd import costs as C

    dev = torch.device("cuda:0")
    w = S.WORKLOADS[args.workload]
    if args.batch or args.seq:
        w = w.replace(batch=args.batch or w.batch, seq=args.seq or w.seq)
        w = w.replace(name=f"{w.name}_B{w.batch}_T{w.seq}")
    if args.retention is not None:
        if not 0.0 < args.retention <= 1.0:
            ap.error("--retention must be in (0, 1]")
        w = w.replace(name=f"{w.name}_r{args.retention:g}", retention=(args.retention,) * w.n_layers,
                      similarity=None)
    B, T, L = w.batch, w.seq, w.n_layers
    dt = w.torch_dtype
    dcode = P.F32 if w.dtype == "f32" else P.BF16
    desc = P.make_desc(w.block, w.d_model, w.n_heads, w.n_kv_heads, w.head_dim, w.d_ff, w.rotary_dims,
                       w.d_router, w.norm_eps, w.rope_theta)
    log(f"workload {w.name}: L={L} d={w.d_model} B={B} T={T} dtype={w.dtype}")
    layers = [P.DeviceLayer(S.layer_weights(w, l), dev) for l in range(L)]
    weights = [dl.weights for dl in layers]
    x0 = S.hidden_states(w).to(dev)
    stream = torch.cuda.current_stream()

    if args.only_sparse:
        args.no_dense = args.no_cpu_baseline = True
    # calibration pass: dense stack + on-GPU similarity statistic (Eq. 4), allocation (Eqs. 5-8)
    s_meas, t_cal, sim_rate = None, None, None
    if args.retention is None and not (args.only_sparse and w.similarity is not None):
        ws_cal = torch.empty(P.workspace_size(desc, dcode, B, T, T, True), dtype=torch.uint8, device=dev)
        accum = torch.zeros(L, 2, dtype=torch.float64, device=dev)
        xc = x0.clone()
        P.stack_forward(desc, weights, [T] * L, xc, ws_cal, flags=P.FLAG_DENSE, sim_accum=accum)  # warm
        accum.zero_()
        xc.copy_(x0)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        P.stack_forward(desc, weights, [T] * L, xc, ws_cal, flags=P.FLAG_DENSE, sim_accum=accum)
        s_meas = P.sim_finalize(accum)
        t_cal = time.perf_counter() - t0
        # the similarity statistic's own kernels, in a second calibration pass
        P.timing_enable(4 * L + 8, ["sim"])
        accum.zero_()
        xc.copy_(x0)
        P.stack_forward(desc, weights, [T] * L, xc, ws_cal, flags=P.FLAG_DENSE, sim_accum=accum)
        torch.cuda.synchronize()
        n_sim, ms_sim = P.timing_read("sim")
        P.timing_enable(0)
        sim_rate = {"ms_per_layer": ms_sim / max(n_sim, 1), "launches": n_sim,
                    "achieved": C.sim_bytes(w, B, T) * n_sim / (ms_sim / 1e3) / 1e9 if ms_sim > 0 else None,
                    "unit": "GB/s", "peak": PEAK_HBM_GBS}
        if sim_rate["achieved"]:
            sim_rate["frac"] = sim_rate["achieved"] / PEAK_HBM_GBS
        del ws_cal, xc
        log(f"calibration pass {t_cal * 1e3:.2f} ms; measured similarity {[round(v, 4) for v in s_meas]}")
    r = retention(P, w, s_meas)
    ks = [P.k_from_retention(v, T) for v in r]
    log(f"k per layer {ks}")

    ws = torch.empty(P.workspace_size(desc, dcode, B, T, max(ks)), dtype=torch.uint8, device=dev)
    xs = [x0.clone() for _ in range(args.steps)]
    xw = x0.clone()
    for _ in range(args.warmup):
        xw.copy_(x0)
        P.stack_forward(desc, weights, ks, xw, ws)
    torch.cuda.synchronize()

    # timed region: K steps, dominant-kernel launches bracketed by HIP events,
    # and an event between consecutive steps (per-step median and minimum)
    P.timing_enable(args.steps * L + 8, ["gemm_down"])
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        marks[i].record(stream)
        P.stack_forward(desc, weights, ks, xs[i], ws)
    marks[-1].record(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    per_step = sorted(marks[i].elapsed_time(marks[i + 1]) for i in range(args.steps))
    n_dom, ms_dom = P.timing_read("gemm_down")
    P.timing_enable(0)
    ms_step = elapsed * 1e3 / args.steps
    tokens_per_s = B * T / (ms_step / 1e3)
    log(f"sparse stack {ms_step:.3f} ms/step, {tokens_per_s / 1e6:.3f} M tokens/s")

    # roofline of the dominant kernel: algorithmic FLOPs per launch / its average duration
    flops_dom = sum(C.gemm_down_flops(w, B, k) for k in ks if k > 0) * args.steps
    avg_ms = ms_dom / max(n_dom, 1)
    achieved = flops_dom / (ms_dom / 1e3) / 1e12 if ms_dom > 0 else 0.0
    roofline = {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": achieved / PEAK_BF16_TFLOPS, "traffic": measured_traffic(w.name),
                "kernel": "down projection: gemm_bf16_dma_kernel<4, 128, 128, 64, 64, 2, 64> (one tile per "
                          "workgroup) or gemm_bf16_sk_kernel<4, 128, 128, 64, 64, 2, 64> (stream-K, on layers "
                          "whose tiles leave a short last round); residual-scatter epilogue",
                "launches": n_dom, "avg_launch_us": avg_ms * 1e3,
                "flops_per_launch": flops_dom / max(n_dom, 1)}

    # per-kernel breakdown (a separate instrumented pass, every launch bracketed)
    breakdown = {}
    if not args.only_sparse:
        nb = min(args.steps, 10)
        P.timing_enable(nb * L * 16 + 64)
        for i in range(nb):
            xw.copy_(x0)
            P.stack_forward(desc, weights, ks, xw, ws)
        torch.cuda.synchronize()
        for kind in P.KINDS:
            n, ms = P.timing_read(kind)
            if n:
                breakdown[kind] = {"ms_per_step": ms / nb, "launches_per_step": n / nb}
        P.timing_enable(0)

    # work and achieved rates of the whole step
    sparse_flops = C.stack_flops(w, B, T, ks, True)
    gemm_flops = sum(C.proj_flops(w, B, k) for k in ks)
    attn_flops = sum(C.attn_flops(w, B, k) for k in ks)
    gemm_ms = sum(v["ms_per_step"] for k, v in breakdown.items() if k.startswith("gemm"))
    attn_ms = breakdown.get("attn", {}).get("ms_per_step", 0.0)
    router_ms = breakdown.get("router", {}).get("ms_per_step", 0.0)
    # every kernel kind against its own roofline (in-situ: the inputs of a layer
    # were written by the layer before, so reads may be served by the MALL)
    for kind, v in breakdown.items():
        wk = [C.kind_work(w, kind, B, T, k) for k in ks if k > 0]
        if not wk or wk[0] is None:
            continue
        total, unit = sum(x[0] for x in wk), wk[0][1]
        secs = v["ms_per_step"] / 1e3
        if unit == "flop":
            v.update(achieved=total / secs / 1e12, unit="TFLOP/s", peak=PEAK_BF16_TFLOPS,
                     frac=total / secs / 1e12 / PEAK_BF16_TFLOPS)
        else:
            v.update(achieved=total / secs / 1e9, unit="GB/s", peak=PEAK_HBM_GBS,
                     frac=total / secs / 1e9 / PEAK_HBM_GBS)
    rates = {
        "step_tflops": sparse_flops / (ms_step / 1e3) / 1e12,
        "gemm_tflops": gemm_flops / (gemm_ms / 1e3) / 1e12 if gemm_ms else None,
        "attn_tflops": attn_flops / (attn_ms / 1e3) / 1e12 if attn_ms else None,
        "router_gbs": sum(C.router_bytes(w, B, T) for k in ks if k > 0) / (router_ms / 1e3) / 1e9 if router_ms else None,
    }

    dense = None
    if not args.no_dense:
        xd = x0.clone()
        wsd = torch.empty(P.workspace_size(desc, dcode, B, T, T), dtype=torch.uint8, device=dev)
        P.stack_forward(desc, weights, [T] * L, xd, wsd, flags=P.FLAG_DENSE)
        nd = max(3, args.steps // 3)
        xds = [x0.clone() for _ in range(nd)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(nd):
            P.stack_forward(desc, weights, [T] * L, xds[i], wsd, flags=P.FLAG_DENSE)
        torch.cuda.synchronize()
        dense_ms = (time.perf_counter() - t0) * 1e3 / nd
        dense = {"ms_per_step": dense_ms, "speedup_sparse_vs_dense": dense_ms / ms_step,
                 "flop_ratio_sparse_over_dense": C.stack_flops(w, B, T, ks, True) / C.stack_flops(w, B, T, [T] * L, False)}
        log(f"dense stack {dense_ms:.3f} ms/step, speedup {dense_ms / ms_step:.2f}x")
        del xds, wsd, xd

    out = {
        "metric": METRIC,
        "value": tokens_per_s,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "ms_per_step_median": per_step[len(per_step) // 2],
        "ms_per_step_min": per_step[0],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded N(0, 0.02) hidden states and random-init weights of the stated shape)",
        "config": {"workload": f"{w.name}: {L}-layer {w.block} stack, d={w.d_model}, heads {w.n_heads}/{w.n_kv_heads}"
                               f"x{w.head_dim}, FFN {w.d_ff}, batch {B} x seq {T}",
                   "global_batch": B, "seq_len": T, "layers": L, "parallelism": "single GPU",
                   "mean_retention": sum(r) / L, "k_per_layer": ks},
        "roofline": roofline,
        "cpu_baseline": None,
        "kernel_breakdown": breakdown,
        "rates": rates,
        "dense": dense,
        "calibration_ms": None if t_cal is None else t_cal * 1e3,
        "similarity_kernel": sim_rate,
        "similarity_measured": s_meas,
        "hip_runtime": torch.version.hip,
    }
    if not (args.only_sparse or args.no_extras):
        kmean = int(round(sum(ks) / len(ks)))
        log(f"streaming entry points standalone (B={B}, T={T}, k={kmean}), cold and hot inputs")
        out["streaming_kernels"] = streaming_rates(P, C, w, kmean, dev, S.layer_weights(w, 0))
    if not (args.only_sparse or args.no_extras):
        log("router-score pathway: gated stack, gate score gradient, router backward")
        out["router_score_pathway"] = router_pathway(P, C, w, ks, dev, desc, weights, x0, ws, ms_step,
                                                     max(3, args.steps // 3), S.layer_weights(w, 0))
    if not (args.only_sparse or args.no_extras):
        log("alignment objective: teacher/student stack, Eq. 9 and Eq. 10 kernels")
        out["alignment_objective"] = alignment_objective(P, C, w, ks, dev, desc, weights, x0, ms_step,
                                                         max(3, args.steps // 3))
    if not (args.only_sparse or args.no_extras):
        log("incremental decoding: prefill into kept-token caches, then threshold-routed decode steps")
        out["decode"] = decode_leg(P, C, w, ks, dev, desc, weights, x0, max(10, args.steps))
    if not args.no_cpu_baseline:
        layers_cpu = L if args.cpu_layers is None else min(args.cpu_layers, L)
        log(f"cpu oracle baseline over {layers_cpu} layers of one sequence")
        out["cpu_baseline"] = cpu_baseline(w, ks, layers_cpu)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
