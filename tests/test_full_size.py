"""GPU parity at the full sizes of the evaluation workloads, in the launch
configuration the benchmark uses (``decode_step``, the plan's split length).

* Workloads 1 and 2 fit the oracle whole: everything is compared with the
  oracle's full compression pass and its fp64 attention.
* Workloads 3, 4 and 5 are too large for the oracle's assignment of every
  token.  The oracle runs the steps it can afford on the full inputs (the
  observation pass and the anchor selection of every head), then samples
  tokens.  For each sampled token it computes the nearest anchor, gamma,
  residual codes and utilities, which must match bit for bit or sit on the
  right side of the pooled budget cut.
* Decode at those sizes is checked by a property that holds at any size: it
  equals fp64 softmax attention over the dense reconstruction of the same
  cache.  That reconstruction is itself bit-exact against the oracle at the
  sizes the oracle covers.
"""
from __future__ import annotations

import math

import numpy as np
import pytest
import torch

import paper_2608_02901_amd as akv
import synth
from oracle import akvref as R
from paper_2608_02901_amd import _native as N
from parity_util import (assert_request_parity, gpu_encode, make_cfg, oracle_encode, plan_k,
                         selection_gap_ok)

pytestmark = pytest.mark.gpu


# Inside the fp32 error band the selection cut is decided on fp64 scores
# (exact fp64 logits, fp64 row sums of the observation pass): the two sides
# agree unless the oracle's n_top-th and (n_top+1)-th pooled scores are within
# ~1e-8 (relative).
SEL_GAP = 1e-7


def _export(plan, cache, b, n_app=0):
    return akv.export(plan, cache.cpu().numpy(), b, n_app)


def _header_flags(cache):
    """Anomaly bits the kernels raise in the cache header (0 = none)."""
    return int(cache[8:12].view(torch.int32).item())


def _np_attention(Kt, Vt, q):
    """Plain fp64 softmax attention (numpy, not the oracle): Kt, Vt [H][T][D], q [Hq][D]."""
    H, T, D = Kt.shape
    g = q.shape[0] // H
    out = np.empty((q.shape[0], D))
    for h in range(H):
        K = Kt[h].astype(np.float64)
        lg = K @ q[h * g:(h + 1) * g].astype(np.float64).T / math.sqrt(D)  # [T][g]
        p = np.exp(lg - lg.max(axis=0))
        out[h * g:(h + 1) * g] = (p.T @ Vt[h].astype(np.float64)) / p.sum(axis=0)[:, None]
    return out


def _layer_on_gpu(wl, steps=1):
    lay = synth.make_layer(wl, device="cuda", steps=steps)
    torch.cuda.synchronize()
    return lay


@pytest.mark.parametrize("wi", [1, 2])
def test_small_workloads_whole_against_oracle(wi):
    wl = synth.workload(wi)
    print(f"[full] workload {wi} {wl.name} lens={wl.seq_lens}", flush=True)
    lay = synth.make_layer(wl)
    cfg = make_cfg(wl)
    plan = N.Plan(cfg, wl.seq_lens)
    cache, ws, dws = gpu_encode(plan, lay)
    enc = oracle_encode(cfg, lay, 0)
    exp = _export(plan, cache, 0)
    assert _header_flags(cache) == 0
    ri = plan.requests[0]
    for h in range(wl.H):
        assert selection_gap_ok(enc["pooled"][h], ri.n_top, SEL_GAP), "near-tie at the selection cut"
    mism = assert_request_parity(exp, enc, cfg)
    print(f"[full] workload {wi}: fixup rows {exp['stats'][:2]}, budget bands {exp['stats'][4:6]}", flush=True)
    out = torch.empty(1, wl.Hq, wl.D, dtype=torch.float32, device="cuda")
    akv.decode_attn(plan, cache, lay.q[0].cuda(), out, dws)
    torch.cuda.synchronize()
    G = wl.G
    Kh = R.reconstruct(lay.K[0].float().numpy(), enc, "K", G, cfg.seed)
    Vh = R.reconstruct(lay.V[0].float().numpy(), enc, "V", G, cfg.seed)
    ref = R.attention(Kh, Vh, lay.q[0, 0].float().numpy())
    err = np.abs(out[0].cpu().numpy() - ref).max()
    print(f"[full] workload {wi}: decode max|err| {err:.3g}", flush=True)
    assert err <= (1e-4 if wl.dtype == "f32" else 2e-3)


def _sampled_request_check(cfg, lay, b, exp, ntok, rng):
    """Oracle on the full inputs of request b for the observation pass and the
    anchor sets, then on ntok sampled non-anchor tokens per head."""
    K = lay.K[b].float().cpu().numpy()
    V = lay.V[b].float().cpu().numpy()
    Q = lay.Qobs[b].float().cpu().numpy()
    H, S, D = K.shape
    g = Q.shape[0] // H
    W, k = cfg.window, plan_k(cfg, S)
    G = cfg.quant_group or D
    bf16 = cfg.dtype == N.BF16
    u_sel = {"K": [], "V": []}
    u_non = {"K": [], "V": []}
    n_checked = 0
    for h in range(H):
        Qg = np.ascontiguousarray(Q[h * g:(h + 1) * g])
        M, Z, Y = R.obs_head(K[h], V[h], Qg)
        _, pooled = R.selector_scores(K[h], Qg, M, Z, cfg.kappa)
        assert selection_gap_ok(pooled, R.n_top(k, W, cfg.rho), SEL_GAP), "near-tie at the selection cut"
        anc = R.select_anchors(pooled, S, W, k, cfg.rho, cfg.seed, h)
        np.testing.assert_array_equal(exp["anchors"][h], anc)
        free = np.setdiff1d(np.arange(S), anc)
        toks = np.sort(rng.choice(free, size=min(ntok, free.size), replace=False)).astype(np.int32)
        aK, gK, rK = R.assign_tokens(K[h], anc, bf16, toks)
        aV, gV, rV = R.assign_tokens(V[h], anc, bf16, toks)
        np.testing.assert_array_equal(exp["a_k"][h][toks], aK)
        np.testing.assert_array_equal(exp["a_v"][h][toks], aV)
        np.testing.assert_array_equal(exp["gamma_k"][h][toks], gK.astype(np.float32))
        np.testing.assert_array_equal(exp["gamma_v"][h][toks], gV.astype(np.float32))
        uK, uV = R.utilities(K[h], V[h], Qg, M, Z, Y, toks, rK, rV)
        for side, u, r in (("K", uK, rK), ("V", uV, rV)):
            sel = exp["sel_" + side.lower()][h][toks].astype(bool)
            u_sel[side].append(u[sel])
            u_non[side].append(u[~sel])
            for i in np.flatnonzero(sel):
                codes, scales = R.codec_encode(r[i], G, cfg.scale_mode, cfg.seed)
                np.testing.assert_array_equal(exp["codes_" + side.lower()][h][toks[i]], codes)
                np.testing.assert_array_equal(exp["scales_" + side.lower()][h][toks[i]], scales)
                n_checked += 1
    # The pooled cut: every selected sample outranks every unselected one.
    for side in "KV":
        s = np.concatenate(u_sel[side])
        n = np.concatenate(u_non[side])
        if s.size and n.size:
            assert s.min() >= n.max(), (side, s.min(), n.max())
    return n_checked


def _decode_property(plan, cache, dws, lay, b_list, steps, append):
    """decode_step / decode_attn output equals fp64 attention over the dense
    reconstruction of the same cache (tail tokens included)."""
    B = len(plan.seq_lens)
    Hq, D = plan.cfg.num_q_heads, plan.cfg.head_dim
    out = torch.empty(B, Hq, D, dtype=torch.float32, device="cuda")
    worst = 0.0
    for s in range(steps):
        if append:
            akv.decode_step(plan, cache, s, lay.k_new[s], lay.v_new[s], lay.q[s], out, dws)
        else:
            akv.decode_attn(plan, cache, lay.q[s], out, dws)
        torch.cuda.synchronize()
        n_app = s + 1 if append else 0
        for b in b_list:
            Kd = akv.reconstruct(plan, cache, b, 0, n_appended=n_app).cpu().numpy()
            Vd = akv.reconstruct(plan, cache, b, 1, n_appended=n_app).cpu().numpy()
            ref = _np_attention(Kd, Vd, lay.q[s, b].float().cpu().numpy())
            worst = max(worst, float(np.abs(out[b].cpu().numpy() - ref).max()))
    return worst


def test_workload3_128k_sampled_and_decode_steps():
    wl = synth.workload(3)
    print(f"[full] workload 3 {wl.name}", flush=True)
    lay = _layer_on_gpu(wl, steps=4)
    cfg = make_cfg(wl, max_append=64)
    plan = N.Plan(cfg, wl.seq_lens)
    cache, ws, dws = plan.alloc("cuda")
    keep = akv.encode(plan, lay.K[0], lay.V[0], lay.Qobs[0], cache, ws)
    torch.cuda.synchronize()
    del keep
    assert _header_flags(cache) == 0
    exp = _export(plan, cache, 0)
    print(f"[full] workload 3: fixup rows {exp['stats'][:2]}, budget bands {exp['stats'][4:6]}", flush=True)
    n = _sampled_request_check(cfg, lay, 0, exp, 256, np.random.default_rng(30))
    print(f"[full] workload 3: sampled codes checked {n}", flush=True)
    err = _decode_property(plan, cache, dws, lay, [0], steps=4, append=True)
    print(f"[full] workload 3: decode_step vs dense fp64 attention max|err| {err:.3g}", flush=True)
    assert err <= 2e-3
    # Appended tokens: the oracle's nearest anchor and gamma against its own anchor set.
    ex4 = _export(plan, cache, 0, 4)
    K = lay.K[0].float().cpu().numpy()
    V = lay.V[0].float().cpu().numpy()
    for h in range(wl.H):
        anc = ex4["anchors"][h]
        for X, new, side in ((K, lay.k_new, "k"), (V, lay.v_new, "v")):
            a, gm = R.assign_vectors(new[:4, 0, h].float().cpu().numpy(), X[h][anc], bf16=True)
            np.testing.assert_array_equal(ex4["tail_a_" + side][h], a)
            np.testing.assert_array_equal(ex4["tail_gamma_" + side][h], gm.astype(np.float32))


def test_workload4_70b_batch8():
    wl = synth.workload(4)
    print(f"[full] workload 4 {wl.name}", flush=True)
    lay = _layer_on_gpu(wl)
    cfg = make_cfg(wl)
    plan = N.Plan(cfg, wl.seq_lens)
    cache, ws, dws = plan.alloc("cuda")
    keep = akv.encode(plan, lay.K, lay.V, lay.Qobs, cache, ws)
    torch.cuda.synchronize()
    del keep
    assert _header_flags(cache) == 0
    rng = np.random.default_rng(40)
    for b in (0, 7):
        exp = _export(plan, cache, b)
        n = _sampled_request_check(cfg, lay, b, exp, 128, rng)
        print(f"[full] workload 4 request {b}: sampled codes checked {n}", flush=True)
    err = _decode_property(plan, cache, dws, lay, [0, 3, 7], steps=1, append=False)
    print(f"[full] workload 4: decode vs dense fp64 attention max|err| {err:.3g}", flush=True)
    assert err <= 2e-3


def test_workload5_ragged16():
    wl = synth.workload(5)
    print(f"[full] workload 5 {wl.name} lens={wl.seq_lens}", flush=True)
    lay = _layer_on_gpu(wl)
    cfg = make_cfg(wl)
    plan = N.Plan(cfg, wl.seq_lens)
    cache, ws, dws = plan.alloc("cuda")
    keep = akv.encode(plan, lay.K, lay.V, lay.Qobs, cache, ws)
    torch.cuda.synchronize()
    del keep
    assert _header_flags(cache) == 0
    order = np.argsort(wl.seq_lens)
    picks = [int(order[0]), int(order[len(order) // 2])]
    rng = np.random.default_rng(50)
    for b in picks:
        exp = _export(plan, cache, b)
        n = _sampled_request_check(cfg, lay, b, exp, 128, rng)
        print(f"[full] workload 5 request {b} (S={wl.seq_lens[b]}): sampled codes checked {n}", flush=True)
    err = _decode_property(plan, cache, dws, lay, picks + [int(order[-1])], steps=1, append=False)
    print(f"[full] workload 5: decode vs dense fp64 attention max|err| {err:.3g}", flush=True)
    assert err <= 2e-3


def test_long_sequence_more_than_256_splits():
    """One request of 540000 tokens: 264 splits of 2048 slots plus the tail
    record, so the merge takes its second round of records (more than one per
    thread).  decode_step over two appended tokens equals fp64 attention over
    the dense reconstruction."""
    wl = synth.Workload("long-540K", H=1, Hq=4, D=128, seq_lens=[540000], dtype="bf16", anchor_frac=0.02,
                        budget=0.05, n_centers=256, steps=2, append=True, seed=12)
    print(f"[full] {wl.name}", flush=True)
    lay = _layer_on_gpu(wl, steps=2)
    cfg = make_cfg(wl, max_append=2)
    plan = N.Plan(cfg, wl.seq_lens)
    assert math.ceil(wl.seq_lens[0] / 2048) + 1 > 256
    cache, ws, dws = plan.alloc("cuda")
    keep = akv.encode(plan, lay.K[0], lay.V[0], lay.Qobs[0], cache, ws)
    torch.cuda.synchronize()
    del keep
    assert _header_flags(cache) == 0
    err = _decode_property(plan, cache, dws, lay, [0], steps=2, append=True)
    print(f"[full] {wl.name}: decode_step vs dense fp64 attention max|err| {err:.3g}", flush=True)
    assert err <= 2e-3
