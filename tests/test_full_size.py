"""GPU parity at the full sizes of the evaluation workloads, in the launch
configuration the benchmark uses (``decode_step``, the plan's split length).

* Workloads 1 and 2: the whole compression pass against the oracle's, and
  the decode output against the oracle's fp64 attention over its own
  reconstruction.
* Workload 3 (the 128K layer): the same for all 8 heads, then the benchmark's
  64 appended tokens (every tail record against the oracle's nearest anchor
  and coefficient) and the decode outputs of steps 1 and 64 against the
  oracle's attention over its reconstruction plus the appended tokens.
* Workload 4 (70B shape, 8 requests): every request, encode and decode.
* Workload 5 (16 ragged requests): the shortest, the median and the longest.
* The paper's operating point (8B layer at 32K, k = S/128, theta = 0.05 from
  the byte budget, i.e. 20x): the residual count of the worked example and the
  whole request against the oracle, encode and decode.
* One 540000-token request (265 split records per query head, the merge's
  second round): decode_step against fp64 attention over the dense
  reconstruction of the same cache, a property that holds at any size (the
  reconstruction is itself bit-exact against the oracle wherever compared).
The oracle's wall time is printed with each comparison.
"""
from __future__ import annotations

import math
import time

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


def _oracle_whole_request(cfg, lay, b, exp, tag):
    """The oracle's full compression pass of request b; every exported stream
    must match it bit for bit (residual sets included)."""
    t0 = time.time()
    print(f"[full] {tag}: oracle encode of request {b} (S={lay.K[b].shape[1]}) ...", flush=True)
    enc = oracle_encode(cfg, _cpu_layer(lay), b)
    print(f"[full] {tag}: oracle encode took {time.time() - t0:.1f} s on {R.num_threads()} threads; "
          f"fixup rows {exp['stats'][:2]}, budget bands {exp['stats'][4:6]}", flush=True)
    S = lay.K[b].shape[1]
    n_top = R.n_top(plan_k(cfg, S), cfg.window, cfg.rho)
    for h in range(enc["anchors"].shape[0]):
        assert selection_gap_ok(enc["pooled"][h], n_top, SEL_GAP), "near-tie at the selection cut"
    assert_request_parity(exp, enc, cfg)
    return enc


class _CpuLayer:
    def __init__(self, lay):
        self.K = [t.cpu() for t in lay.K]
        self.V = [t.cpu() for t in lay.V]
        self.Qobs = [t.cpu() for t in lay.Qobs]


_cpu_cache = {}


def _cpu_layer(lay):
    key = id(lay)
    if key not in _cpu_cache:
        _cpu_cache.clear()
        _cpu_cache[key] = _CpuLayer(lay)
    return _cpu_cache[key]


def _oracle_decode_check(cfg, lay, b, enc, q, got, tails=None, tag="", cs=None):
    """Decode output of request b against the oracle's fp64 attention over its
    own dense reconstruction (and the appended tokens, encoded by the oracle
    against its anchors: fp32(gamma) * anchor, no residual)."""
    cl = _cpu_layer(lay)
    K = cl.K[b].float().numpy()
    V = cl.V[b].float().numpy()
    G = cfg.quant_group or K.shape[2]
    Kh = R.reconstruct(K, enc, "K", G, cfg.seed)
    Vh = R.reconstruct(V, enc, "V", G, cfg.seed)
    if tails is not None:
        kt, vt = tails  # [n][H][D] each
        H = K.shape[0]
        bf16 = cfg.dtype == N.BF16
        addK, addV = [], []
        for h in range(H):
            anc = enc["anchors"][h]
            rows = []
            for X, new in ((K, kt), (V, vt)):
                A = X[h][anc]
                a, gm = R.assign_vectors(new[:, h], A, bf16=bf16)
                rows.append(np.float32(gm)[:, None] * A[a].astype(np.float32))
            addK.append(rows[0])
            addV.append(rows[1])
        Kh = np.concatenate([Kh, np.stack(addK)], axis=1)
        Vh = np.concatenate([Vh, np.stack(addV)], axis=1)
    ref = R.attention(Kh, Vh, q, cs=None if cs is None else cs[: Kh.shape[1]])
    err = float(np.abs(got - ref).max())
    print(f"[full] {tag}: decode vs oracle attention max|err| {err:.3g}", flush=True)
    assert err <= 2e-3, err
    return err


def test_paper_operating_point_theta_20x():
    """App. A.1 worked example at full size: S = 32768, H = 8, D = 128, W = 32,
    k = S/128 = 256 and theta = 0.05 give N = 91,056 residuals (Eq.
    byte-budget), split N_K = floor(N/2), N_V = N - N_K; the compression pass
    at that budget matches the oracle's bit for bit and decode matches its
    attention."""
    S = 32768
    wl = synth.Workload("llama8b-32K-theta0.05", H=8, Hq=32, D=128, seq_lens=[S], dtype="bf16",
                        anchor_count=S // 128, n_centers=512, steps=2, seed=5)
    cfg = make_cfg(wl, budget_mode=N.BUDGET_THETA, budget=0.05)
    plan = N.Plan(cfg, wl.seq_lens)
    ri = plan.requests[0]
    n = R.theta_budget(S, 8, 128, 32, 256, 128, float(np.float32(0.05)))
    assert abs(n - 91056) <= 1  # the fp32 rounding of theta may move the floor by one
    assert (ri.residuals_k, ri.residuals_v) == (n // 2, n - n // 2)
    print(f"[full] operating point: k={ri.anchors} N_K={ri.residuals_k} N_V={ri.residuals_v} "
          f"cache {plan.cache_bytes / 1e6:.2f} MB vs dense {2 * S * 8 * 128 * 2 / 1e6:.1f} MB", flush=True)
    lay = _layer_on_gpu(wl, steps=2)
    cache, ws, dws = gpu_encode(plan, lay)
    assert _header_flags(cache) == 0
    exp = _export(plan, cache, 0)
    enc = _oracle_whole_request(cfg, lay, 0, exp, "operating point")
    assert int(exp["sel_k"].sum()) == ri.residuals_k and int(exp["sel_v"].sum()) == ri.residuals_v
    for s in range(2):
        out = torch.empty(1, wl.Hq, wl.D, dtype=torch.float32, device="cuda")
        akv.decode_attn(plan, cache, lay.q[s], out, dws)
        torch.cuda.synchronize()
        _oracle_decode_check(cfg, lay, 0, enc, lay.q[s, 0].float().cpu().numpy(), out[0].cpu().numpy(),
                             tag=f"operating point step {s}")


def test_workload3_128k_whole_with_64_appends():
    """The 128K layer against the oracle's whole compression pass (all 8
    heads), then the 64 generated tokens of the benchmark: every tail record
    against the oracle's nearest anchor and coefficient, and the decode
    outputs of steps 1 and 64 against the oracle's attention over its own
    reconstruction plus the appended tokens."""
    wl = synth.workload(3)
    NS = 64
    print(f"[full] workload 3 {wl.name}", flush=True)
    lay = _layer_on_gpu(wl, steps=NS)
    cfg = make_cfg(wl, max_append=NS)
    plan = N.Plan(cfg, wl.seq_lens)
    cache, ws, dws = plan.alloc("cuda")
    keep = akv.encode(plan, lay.K[0], lay.V[0], lay.Qobs[0], cache, ws)
    torch.cuda.synchronize()
    del keep
    assert _header_flags(cache) == 0
    exp = _export(plan, cache, 0)
    enc = _oracle_whole_request(cfg, lay, 0, exp, "workload 3")
    out = torch.empty(1, wl.Hq, wl.D, dtype=torch.float32, device="cuda")
    outs = {}
    for s in range(NS):
        akv.decode_step(plan, cache, s, lay.k_new[s], lay.v_new[s], lay.q[s], out, dws)
        if s in (0, NS - 1):
            torch.cuda.synchronize()
            outs[s] = out[0].cpu().numpy().copy()
    torch.cuda.synchronize()
    ex = _export(plan, cache, 0, NS)
    kt = lay.k_new[:, 0].float().cpu().numpy()
    vt = lay.v_new[:, 0].float().cpu().numpy()
    cl = _cpu_layer(lay)
    K = cl.K[0].float().numpy()
    V = cl.V[0].float().numpy()
    for h in range(wl.H):
        anc = enc["anchors"][h]
        for X, new, side in ((K, kt, "k"), (V, vt, "v")):
            a, gm = R.assign_vectors(new[:, h], X[h][anc], bf16=True)
            np.testing.assert_array_equal(ex["tail_a_" + side][h], a)
            np.testing.assert_array_equal(ex["tail_gamma_" + side][h], gm.astype(np.float32))
    for s, got in outs.items():
        _oracle_decode_check(cfg, lay, 0, enc, lay.q[s, 0].float().cpu().numpy(), got,
                             tails=(kt[:s + 1], vt[:s + 1]), tag=f"workload 3 step {s + 1}")


def test_workload3_128k_rope_whole_with_appends():
    """The 128K layer with keys given before RoPE and Llama-3.1's rotary
    frequencies (Sec. 3.2): the whole compression pass against the oracle's
    (anchors scored with the rotated keys, residuals ranked with R_t r), then
    8 generated tokens through decode_step, whose outputs at steps 1 and 8
    match the oracle's attention with every key rotated at its position."""
    wl = synth.workload(3)
    NS = 8
    freq = synth.llama31_inv_freq(wl.D)
    print(f"[full] workload 3 with RoPE {wl.name}", flush=True)
    lay = _layer_on_gpu(wl, steps=NS)
    cfg = make_cfg(wl, max_append=NS, rope_inv_freq=freq)
    plan = N.Plan(cfg, wl.seq_lens)
    cache, ws, dws = plan.alloc("cuda")
    keep = akv.encode(plan, lay.K[0], lay.V[0], lay.Qobs[0], cache, ws)
    torch.cuda.synchronize()
    del keep
    assert _header_flags(cache) == 0
    exp = _export(plan, cache, 0)
    enc = _oracle_whole_request(cfg, lay, 0, exp, "workload 3 RoPE")
    out = torch.empty(1, wl.Hq, wl.D, dtype=torch.float32, device="cuda")
    outs = {}
    for s in range(NS):
        akv.decode_step(plan, cache, s, lay.k_new[s], lay.v_new[s], lay.q[s], out, dws)
        if s in (0, NS - 1):
            torch.cuda.synchronize()
            outs[s] = out[0].cpu().numpy().copy()
    torch.cuda.synchronize()
    kt = lay.k_new[:, 0].float().cpu().numpy()
    vt = lay.v_new[:, 0].float().cpu().numpy()
    cs = R.rope_table(freq, wl.D, wl.seq_lens[0] + NS)
    for s, got in outs.items():
        _oracle_decode_check(cfg, lay, 0, enc, lay.q[s, 0].float().cpu().numpy(), got,
                             tails=(kt[:s + 1], vt[:s + 1]), tag=f"workload 3 RoPE step {s + 1}", cs=cs)


def test_workload4_70b_batch8_whole():
    """All 8 requests of the 70B-shaped batch against the oracle's whole
    compression pass, and the batched decode step of every request against
    the oracle's attention over its reconstruction."""
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
    out = torch.empty(wl.batch, wl.Hq, wl.D, dtype=torch.float32, device="cuda")
    akv.decode_attn(plan, cache, lay.q[0], out, dws)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    host = cache.cpu().numpy()
    for b in range(wl.batch):
        exp = akv.export(plan, host, b, 0)
        enc = _oracle_whole_request(cfg, lay, b, exp, f"workload 4 request {b}")
        _oracle_decode_check(cfg, lay, b, enc, lay.q[0, b].float().cpu().numpy(), got[b],
                             tag=f"workload 4 request {b}")


def test_workload5_ragged16_short_median_long():
    """The ragged batch of 16: the shortest, the median and the longest
    request against the oracle's whole compression pass, and their decode
    outputs against the oracle's attention over its reconstruction."""
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
    out = torch.empty(wl.batch, wl.Hq, wl.D, dtype=torch.float32, device="cuda")
    akv.decode_attn(plan, cache, lay.q[0], out, dws)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    host = cache.cpu().numpy()
    order = np.argsort(wl.seq_lens)
    for b in (int(order[0]), int(order[len(order) // 2]), int(order[-1])):
        exp = akv.export(plan, host, b, 0)
        tag = f"workload 5 request {b} (S={wl.seq_lens[b]})"
        enc = _oracle_whole_request(cfg, lay, b, exp, tag)
        _oracle_decode_check(cfg, lay, b, enc, lay.q[0, b].float().cpu().numpy(), got[b], tag=tag)


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
