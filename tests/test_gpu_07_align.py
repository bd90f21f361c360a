"""GPU parity of the alignment objective (Section 3.5, Eqs. 9-11).

1. dsf_align_hidden (Eq. 9 summand) on seeded rows against the oracle, per
   token within a rounding bound derived from fp32 exponentials (relative
   error of each probability at most e_c = 8u + 2u |h_c - max h|, u = 2^-24,
   plus the normaliser's share) and fp64 sums; identical rows give exactly 0.
2. dsf_kl_align (Eq. 10) on seeded logits against the oracle, per row within
   4 e (sum_c P_c |ld_c - ls_c| + 1) with e the largest e_c of the row;
   identical rows give exactly 0; the sum lands in accum.
3. dsf_align_stack_forward: the dense-teacher / sparse-student stack equals
   the dense and sparse layers chained through the single-layer entry point
   (bitwise), each layer of which is checked against the oracle (teacher-
   forced, as the layer tests do), and its per-layer sums equal
   dsf_align_hidden on the chained states (bitwise) and the oracle's Eq. 9
   on them (within the bound of 1.).
"""
import numpy as np
import pytest
import torch

import paper_2607_21291_amd as P
import synthetic as S
from oracle import adadsf_oracle as O

from gpu_util import TOL, announce, check_layer, desc_dict, make_desc, rel_inf, run_layer, to_np, workload

pytestmark = pytest.mark.gpu

U = 2.0 ** -24


def _rows(n, d, dtype, seed, scale=2.0, noise=0.5):
    g = np.random.default_rng(seed)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    a = torch.tensor(g.normal(size=(n, d)) * scale, dtype=tdt)
    b = torch.tensor(to_np(a) + g.normal(size=(n, d)) * noise, dtype=tdt)
    return a, b


def _prob_err(h):
    """Per-element relative error bound e_c of the GPU's probabilities."""
    h = np.asarray(h, dtype=np.float64)
    e = 8 * U + 2 * U * np.abs(h - h.max(-1, keepdims=True))
    p = O.softmax_rows(h)
    return p, e + np.sum(p * e, -1, keepdims=True)


def _align_bound(hs, hd):
    p, ep = _prob_err(hs)
    q, eq = _prob_err(hd)
    dp, dq = p * ep, q * eq
    return np.sum(2 * np.abs(p - q) * (dp + dq) + (dp + dq) ** 2, -1) * 2 + 1e-300


@pytest.mark.parametrize("n,d,dtype", [(1000, 768, "bf16"), (333, 128, "f32"), (77, 3584, "bf16"),
                                       (50, 4096, "f32"), (5, 8192, "bf16"), (130, 896, "bf16")])
def test_align_hidden_matches_oracle(dev, n, d, dtype):
    announce(f"align hidden n={n} d={d} {dtype}")
    hs, hd = _rows(n, d, dtype, seed=n + d)
    hs[3] = hd[3]  # an identical row
    per = torch.full((n,), float("nan"), device=dev)
    accum = torch.full((1,), 1.5, dtype=torch.float64, device=dev)
    P.align_hidden(hs.to(dev), hd.to(dev), accum, per_token_sq=per)
    torch.cuda.synchronize()
    ref = O.hidden_align_sq(to_np(hs), to_np(hd))
    bound = _align_bound(to_np(hs), to_np(hd))
    got = per.cpu().numpy().astype(np.float64)
    # per-token values are stored as fp32
    assert np.all(np.abs(got - ref) <= bound + 2 * U * np.abs(ref)), np.max(np.abs(got - ref) - bound)
    assert got[3] == 0.0
    tot = accum.item() - 1.5
    assert abs(tot - ref.sum()) <= bound.sum() + 1e-15 * ref.sum()
    # deterministic
    acc2 = torch.zeros(1, dtype=torch.float64, device=dev)
    acc3 = torch.zeros(1, dtype=torch.float64, device=dev)
    P.align_hidden(hs.to(dev), hd.to(dev), acc2)
    P.align_hidden(hs.to(dev), hd.to(dev), acc3)
    torch.cuda.synchronize()
    assert acc2.item() == acc3.item()


def _kl_bound(ld, ls):
    ld, ls = np.asarray(ld, np.float64), np.asarray(ls, np.float64)
    e = 8 * U + 2 * U * np.maximum(np.abs(ld - ld.max(-1, keepdims=True)).max(-1),
                                   np.abs(ls - ls.max(-1, keepdims=True)).max(-1))
    p = O.softmax_rows(ld)
    return 4 * e * (np.sum(p * np.abs(ld - ls), -1) + 1) + 1e-12


@pytest.mark.parametrize("rows,C,dtype", [(64, 50304, "bf16"), (300, 1000, "f32"), (7, 151936, "bf16"),
                                          (3, 8, "f32"), (33, 2048, "bf16")])
def test_kl_align_matches_oracle(dev, rows, C, dtype):
    announce(f"kl align rows={rows} C={C} {dtype}")
    ld, ls = _rows(rows, C, dtype, seed=rows + C, scale=3.0, noise=0.7)
    ld[1] = ls[1]
    per = torch.full((rows,), float("nan"), device=dev)
    accum = torch.full((1,), -2.0, dtype=torch.float64, device=dev)
    P.kl_align(ld.to(dev), ls.to(dev), accum, per_row_kl=per)
    torch.cuda.synchronize()
    ref = O.kl_align(to_np(ld), to_np(ls))
    bound = _kl_bound(to_np(ld), to_np(ls))
    got = per.cpu().numpy().astype(np.float64)
    assert np.all(np.abs(got - ref) <= bound + 2 * U * np.abs(ref)), np.max(np.abs(got - ref) - bound)
    assert got[1] == 0.0
    assert abs((accum.item() + 2.0) - ref.sum()) <= bound.sum()


def test_align_empty_inputs(dev):
    accum = torch.full((1,), 3.0, dtype=torch.float64, device=dev)
    e = torch.empty(0, 64, dtype=torch.bfloat16, device=dev)
    announce("align: empty inputs")
    P.align_hidden(e, e, accum)
    P.kl_align(e, e, accum)
    torch.cuda.synchronize()
    assert accum.item() == 3.0


@pytest.mark.parametrize("name,gate", [("tiny_neox_f32", False), ("qwen_bf16_small", False),
                                       ("neox_bf16_small", True)])
def test_align_stack_matches_chained_layers(dev, name, gate):
    w = workload(name).replace(n_layers=3)
    announce(f"align stack {name} gate={gate}")
    Ws = S.stack_weights(w)
    x = S.hidden_states(w)
    T = w.seq
    ks = [T // 2, 0, max(1, T // 5)]
    dls = [P.DeviceLayer(W, dev) for W in Ws]
    xs, xt = x.to(dev), x.to(dev)
    hid = torch.zeros(3, dtype=torch.float64, device=dev)
    desc = make_desc(w)
    ws = torch.empty(P.align_stack_workspace_size(desc, P.F32 if w.dtype == "f32" else P.BF16, w.batch, T),
                     dtype=torch.uint8, device=dev)
    flags = P.FLAG_GATE if gate else 0
    P.align_stack_forward(desc, [dl.weights for dl in dls], ks, xs, xt, hid, ws, flags=flags)
    torch.cuda.synchronize()
    cur_s, cur_t = x, x
    for l, (W, k) in enumerate(zip(Ws, ks)):
        yt, _, _ = run_layer(dev, w, W, cur_t, T, flags=P.FLAG_DENSE)
        ref_t = O.dense_layer(desc_dict(w), W, to_np(cur_t))
        assert rel_inf(to_np(yt) - to_np(cur_t), ref_t - to_np(cur_t)) < TOL[w.dtype]
        if k > 0:
            ys, sc, idx = run_layer(dev, w, W, cur_s, k, flags=flags)
            check_layer(w, W, cur_s, ys, sc, idx, k, gate=gate)
        else:
            ys = cur_s.to(dev)
        one = torch.zeros(1, dtype=torch.float64, device=dev)
        P.align_hidden(ys, yt, one)
        torch.cuda.synchronize()
        assert one.item() == hid[l].item()
        a, b = to_np(ys), to_np(yt)
        ref = O.hidden_align_sq(a, b).sum()
        assert abs(hid[l].item() - ref) <= _align_bound(a, b).sum() + 1e-15 * ref
        cur_s, cur_t = ys.cpu(), yt.cpu()
    assert torch.equal(xs.cpu(), cur_s) and torch.equal(xt.cpu(), cur_t)
    assert hid[1].item() > 0  # the student skipped layer 1 entirely
