"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Bit-exact: anchor sets, anchor indices, stored coefficients, residual codes
and scales (where both sides store a residual), dense reconstructions.
Residual sets: equal except candidates whose utility ties with the cut within
the fp32/fp64 difference of the utilities.  Attention outputs: within 1e-4
(fp32 cache) or 2e-2 (bf16 output) max-abs of the oracle's fp64 attention over
its own reconstruction."""
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


def _small(name, **kw):
    base = dict(name=name, H=2, Hq=8, D=128, seq_lens=[1000], dtype="bf16", anchor_frac=0.04, budget=0.05,
                n_centers=48, seed=11)
    base.update(kw)
    return synth.Workload(**base)


CASES = {
    "bf16_ragged": _small("bf16_ragged"),
    "bf16_gqa8": _small("bf16_gqa8", Hq=16, seq_lens=[1500], seed=12),
    "bf16_batch3": _small("bf16_batch3", seq_lens=[700, 1500, 2300], Hq=4, seed=13),
    "f32_group32": _small("f32_group32", H=1, Hq=1, dtype="f32", seq_lens=[1200], anchor_count=64, anchor_frac=0.0,
                          quant_group=32, n_outlier=0, seed=14),
}


def _export(plan, cache, b, n_app=0):
    return akv.export(plan, cache.cpu().numpy(), b, n_app)


@pytest.mark.parametrize("case", list(CASES))
def test_encode_matches_oracle(case):
    wl = CASES[case]
    print(f"[parity] encode {case} lens={wl.seq_lens}", flush=True)
    layer = synth.make_layer(wl)
    cfg = make_cfg(wl)
    plan = N.Plan(cfg, wl.seq_lens)
    cache, ws, dws = gpu_encode(plan, layer)
    for b in range(wl.batch):
        enc = oracle_encode(cfg, layer, b)
        exp = _export(plan, cache, b)
        ri = plan.requests[b]
        for h in range(wl.H):
            assert selection_gap_ok(enc["pooled"][h], ri.n_top), "near-tie at the selection cut"
        mism = assert_request_parity(exp, enc, cfg)
        print(f"[parity] {case} b={b} fixup rows K/V = {exp['stats'][0]}/{exp['stats'][1]} "
              f"set ties = {mism}", flush=True)


@pytest.mark.parametrize("case", ["bf16_ragged", "f32_group32"])
def test_override_anchors_downstream_bit_exact(case):
    wl = CASES[case]
    layer = synth.make_layer(wl, seed=wl.seed + 100)
    cfg = make_cfg(wl)
    plan = N.Plan(cfg, wl.seq_lens)
    S = wl.seq_lens[0]
    k = plan_k(cfg, S)
    rng = np.random.default_rng(0)
    ov = np.stack([np.sort(np.r_[rng.choice(S - wl.window, k - wl.window, replace=False),
                                 np.arange(S - wl.window, S)]) for _ in range(wl.H)]).astype(np.int32)
    cache, ws, dws = gpu_encode(plan, layer, override=ov)
    enc = oracle_encode(cfg, layer, 0, anchor_override=ov)
    exp = _export(plan, cache, 0)
    assert_request_parity(exp, enc, cfg)


@pytest.mark.parametrize("mode", [N.SCALE_ABSMAX_LITERAL, N.SCALE_RMS])
def test_codec_scale_readings(mode):
    wl = CASES["bf16_ragged"]
    layer = synth.make_layer(wl)
    cfg = make_cfg(wl, scale_mode=mode, quant_group=32)
    plan = N.Plan(cfg, wl.seq_lens)
    cache, ws, dws = gpu_encode(plan, layer)
    enc = oracle_encode(cfg, layer, 0)
    assert_request_parity(_export(plan, cache, 0), enc, cfg)


def _oracle_dense(cfg, layer, b, enc, side):
    X = (layer.K if side == "K" else layer.V)[b].float().numpy()
    return R.reconstruct(X, enc, side, cfg.quant_group or 128, cfg.seed)


@pytest.mark.parametrize("case", list(CASES))
def test_reconstruct_bit_exact(case):
    wl = CASES[case]
    layer = synth.make_layer(wl)
    cfg = make_cfg(wl)
    plan = N.Plan(cfg, wl.seq_lens)
    cache, ws, dws = gpu_encode(plan, layer)
    for b in range(wl.batch):
        enc = oracle_encode(cfg, layer, b)
        exp = _export(plan, cache, b)
        same = all((exp["sel_" + s].astype(bool) == enc["sel" + s.upper()].astype(bool)).all() for s in "kv")
        for side, si in (("K", 0), ("V", 1)):
            got = akv.reconstruct(plan, cache, b, si).cpu().numpy()
            ref = _oracle_dense(cfg, layer, b, enc, side)
            if same:
                np.testing.assert_array_equal(got, ref)
            else:
                sel = exp["sel_" + side.lower()].astype(bool) == enc["sel" + side].astype(bool)
                np.testing.assert_array_equal(got[sel], ref[sel])


@pytest.mark.parametrize("case", list(CASES))
def test_decode_matches_oracle_attention(case):
    wl = CASES[case]
    layer = synth.make_layer(wl, steps=2)
    cfg = make_cfg(wl)
    plan = N.Plan(cfg, wl.seq_lens)
    cache, ws, dws = gpu_encode(plan, layer)
    f32 = wl.dtype == "f32"
    for step in range(2):
        q = layer.q[step]
        out = torch.empty(wl.batch, wl.Hq, wl.D, dtype=torch.float32, device="cuda")
        akv.decode_attn(plan, cache, q.cuda(), out, dws)
        torch.cuda.synchronize()
        for b in range(wl.batch):
            enc = oracle_encode(cfg, layer, b)
            Kh = _oracle_dense(cfg, layer, b, enc, "K")
            Vh = _oracle_dense(cfg, layer, b, enc, "V")
            ref = R.attention(Kh, Vh, q[b].float().numpy())
            err = np.abs(out[b].cpu().numpy() - ref).max()
            print(f"[parity] decode {case} step={step} b={b} max|err|={err:.3g}", flush=True)
            assert err <= (1e-4 if f32 else 2e-3), err
        if not f32:
            outb = torch.empty(wl.batch, wl.Hq, wl.D, dtype=torch.bfloat16, device="cuda")
            akv.decode_attn(plan, cache, q.cuda(), outb, dws)
            torch.cuda.synchronize()
            for b in range(wl.batch):
                enc = oracle_encode(cfg, layer, b)
                ref = R.attention(_oracle_dense(cfg, layer, b, enc, "K"), _oracle_dense(cfg, layer, b, enc, "V"),
                                  q[b].float().numpy())
                assert np.abs(outb[b].float().cpu().numpy() - ref).max() <= 2e-2


@pytest.mark.parametrize("fused", [False, True], ids=["append_then_attn", "decode_step"])
def test_append_then_decode(fused):
    wl = _small("append", seq_lens=[1300], steps=6, append=True, seed=21)
    layer = synth.make_layer(wl)
    cfg = make_cfg(wl)
    plan = N.Plan(cfg, wl.seq_lens)
    cache, ws, dws = gpu_encode(plan, layer)
    enc = oracle_encode(cfg, layer, 0)
    Kh = _oracle_dense(cfg, layer, 0, enc, "K")
    Vh = _oracle_dense(cfg, layer, 0, enc, "V")
    Kx = layer.K[0].float().numpy()
    Vx = layer.V[0].float().numpy()
    tails_k, tails_v = [], []
    for n in range(wl.steps):
        out = torch.empty(1, wl.Hq, wl.D, dtype=torch.float32, device="cuda")
        if fused:
            akv.decode_step(plan, cache, n, layer.k_new[n].cuda(), layer.v_new[n].cuda(), layer.q[n].cuda(), out, dws)
        else:
            akv.append(plan, cache, n, layer.k_new[n].cuda(), layer.v_new[n].cuda(), dws)
            akv.decode_attn(plan, cache, layer.q[n].cuda(), out, dws, n_appended=n + 1)
        torch.cuda.synchronize()
        tk, tv = [], []
        for h in range(wl.H):
            anc = enc["anchors"][h]
            for X, new, tl in ((Kx, layer.k_new, tk), (Vx, layer.v_new, tv)):
                a, g = R.assign_vectors(new[n, 0, h:h + 1].float().numpy(), X[h][anc], bf16=True)
                tl.append((X[h][anc[a[0]]].astype(np.float32) * np.float32(g[0])).astype(np.float32))
        tails_k.append(np.stack(tk))
        tails_v.append(np.stack(tv))
        Kt = np.concatenate([Kh, np.stack(tails_k, 1)], 1)
        Vt = np.concatenate([Vh, np.stack(tails_v, 1)], 1)
        ref = R.attention(Kt, Vt, layer.q[n, 0].float().numpy())
        err = np.abs(out[0].cpu().numpy() - ref).max()
        assert err <= 2e-3, (n, err)
    exp = _export(plan, cache, 0, wl.steps)
    for h in range(wl.H):
        anc = enc["anchors"][h]
        for X, new, side in ((Kx, layer.k_new, "k"), (Vx, layer.v_new, "v")):
            a, g = R.assign_vectors(new[:, 0, h].float().numpy(), X[h][anc], bf16=True)
            np.testing.assert_array_equal(exp["tail_a_" + side][h], a)
            np.testing.assert_array_equal(exp["tail_gamma_" + side][h], g.astype(np.float32))
    dense = akv.reconstruct(plan, cache, 0, 0, n_appended=wl.steps).cpu().numpy()
    np.testing.assert_array_equal(dense[:, :wl.seq_lens[0]], Kh)
    np.testing.assert_array_equal(dense[:, wl.seq_lens[0]:], np.stack(tails_k, 1))


def test_all_anchor_cache_decodes_dense_attention():
    wl = _small("dense", seq_lens=[600], anchor_count=600, anchor_frac=0.0, seed=31)
    layer = synth.make_layer(wl)
    cfg = make_cfg(wl)
    plan = N.Plan(cfg, wl.seq_lens)
    cache, ws, dws = gpu_encode(plan, layer)
    out = torch.empty(1, wl.Hq, wl.D, dtype=torch.float32, device="cuda")
    akv.decode_attn(plan, cache, layer.q[0].cuda(), out, dws)
    torch.cuda.synchronize()
    K = layer.K[0].float().numpy().astype(np.float32)
    V = layer.V[0].float().numpy().astype(np.float32)
    ref = R.attention(K, V, layer.q[0, 0].float().numpy())
    assert np.abs(out[0].cpu().numpy() - ref).max() <= 2e-3


def test_encode_is_deterministic():
    wl = CASES["bf16_batch3"]
    layer = synth.make_layer(wl)
    plan = N.Plan(make_cfg(wl), wl.seq_lens)
    c1, _, _ = gpu_encode(plan, layer)
    c2, _, _ = gpu_encode(plan, layer)
    assert torch.equal(c1, c2)


def test_repeated_steps_share_one_workspace():
    """Twenty decode calls in a row on one decode workspace, each with its own
    queries and every other one appending: nothing one call leaves in the
    workspace leaks into the next, so every output matches the oracle's
    attention over the tokens appended so far."""
    wl = _small("repeat", seq_lens=[1600], steps=20, append=True, seed=51)
    layer = synth.make_layer(wl)
    cfg = make_cfg(wl)
    plan = N.Plan(cfg, wl.seq_lens)
    cache, ws, dws = gpu_encode(plan, layer)
    enc = oracle_encode(cfg, layer, 0)
    Kh = _oracle_dense(cfg, layer, 0, enc, "K")
    Vh = _oracle_dense(cfg, layer, 0, enc, "V")
    Kx, Vx = layer.K[0].float().numpy(), layer.V[0].float().numpy()
    tk, tv = [], []
    n_app = 0
    for s in range(wl.steps):
        out = torch.empty(1, wl.Hq, wl.D, dtype=torch.float32, device="cuda")
        if s % 2:
            akv.decode_step(plan, cache, n_app, layer.k_new[s].cuda(), layer.v_new[s].cuda(), layer.q[s].cuda(), out,
                            dws)
            rows_k, rows_v = [], []
            for h in range(wl.H):
                anc = enc["anchors"][h]
                for X, new, rows in ((Kx, layer.k_new, rows_k), (Vx, layer.v_new, rows_v)):
                    a, g = R.assign_vectors(new[s, 0, h:h + 1].float().numpy(), X[h][anc], bf16=True)
                    rows.append((X[h][anc[a[0]]].astype(np.float32) * np.float32(g[0])).astype(np.float32))
            tk.append(np.stack(rows_k))
            tv.append(np.stack(rows_v))
            n_app += 1
        else:
            akv.decode_attn(plan, cache, layer.q[s].cuda(), out, dws, n_appended=n_app)
        torch.cuda.synchronize()
        Kt = np.concatenate([Kh] + ([np.stack(tk, 1)] if tk else []), 1)
        Vt = np.concatenate([Vh] + ([np.stack(tv, 1)] if tv else []), 1)
        ref = R.attention(Kt, Vt, layer.q[s, 0].float().numpy())
        err = np.abs(out[0].cpu().numpy() - ref).max()
        assert np.isfinite(out.cpu().numpy()).all() and err <= 2e-3, (s, err)
