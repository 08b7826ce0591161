"""Keys stored before RoPE and rotated at decoding (Sec. 3.2 "RoPE"; Sec. 3.3
Eq. utilities with R_t; App. E "Implementation"), GPU against the oracle.

The compression pass takes the unrotated keys and Llama-3.1's rotary
frequencies: the anchors (scored with the rotated keys), the assignment,
coefficients, residual sets (ranked with q . R_t r) and codes must equal the
oracle's bit for bit.  Decode attention rotates every stored key at its
position; it must match the oracle's fp64 attention over its reconstruction
with the keys rotated, for prompt tokens, ENCODED and DENSE appended tokens,
within 2e-3 (bf16 cache, fp32 output) or 1e-4 (fp32 cache)."""
import numpy as np
import pytest
import torch

import paper_2608_02901_amd as akv
import synth
from oracle import akvref as R
from paper_2608_02901_amd import _native as N
from parity_util import assert_request_parity, gpu_encode, make_cfg, oracle_encode, rope_freqs, selection_gap_ok

pytestmark = pytest.mark.gpu

FREQ = synth.llama31_inv_freq(128)


def _wl(name, **kw):
    base = dict(name=name, H=2, Hq=8, D=128, seq_lens=[1000], dtype="bf16", anchor_frac=0.04, budget=0.05,
                n_centers=48, seed=41)
    base.update(kw)
    return synth.Workload(**base)


CASES = {
    "bf16_batch2": _wl("rope-bf16", seq_lens=[1100, 2300], seed=41),
    "bf16_gqa8": _wl("rope-gqa8", Hq=16, seq_lens=[1500], seed=42),
    "f32_group32": _wl("rope-f32", H=1, Hq=2, dtype="f32", seq_lens=[1200], anchor_count=64, anchor_frac=0.0,
                       quant_group=32, n_outlier=0, seed=43),
}


def _dense(cfg, layer, b, enc, side):
    X = (layer.K if side == "K" else layer.V)[b].float().numpy()
    return R.reconstruct(X, enc, side, cfg.quant_group or 128, cfg.seed)


@pytest.mark.parametrize("case", list(CASES))
def test_rope_encode_and_decode_match_oracle(case):
    wl = CASES[case]
    print(f"[rope] {case} lens={wl.seq_lens}", flush=True)
    layer = synth.make_layer(wl, steps=2)
    cfg = make_cfg(wl, rope_inv_freq=FREQ)
    plan = N.Plan(cfg, wl.seq_lens)
    cache, ws, dws = gpu_encode(plan, layer)
    f32 = wl.dtype == "f32"
    encs = []
    for b in range(wl.batch):
        enc = oracle_encode(cfg, layer, b)
        encs.append(enc)
        exp = akv.export(plan, cache.cpu().numpy(), b, 0)
        for h in range(wl.H):
            assert selection_gap_ok(enc["pooled"][h], plan.requests[b].n_top), "near-tie at the selection cut"
        assert_request_parity(exp, enc, cfg)
        # the stored keys are the unrotated ones
        for side, si in (("K", 0), ("V", 1)):
            np.testing.assert_array_equal(akv.reconstruct(plan, cache, b, si).cpu().numpy(),
                                          _dense(cfg, layer, b, enc, side))
    for step in range(2):
        q = layer.q[step]
        out = torch.empty(wl.batch, wl.Hq, wl.D, dtype=torch.float32, device="cuda")
        akv.decode_attn(plan, cache, q.cuda(), out, dws)
        torch.cuda.synchronize()
        for b in range(wl.batch):
            S = wl.seq_lens[b]
            cs = R.rope_table(FREQ, wl.D, S)
            ref = R.attention(_dense(cfg, layer, b, encs[b], "K"), _dense(cfg, layer, b, encs[b], "V"),
                              q[b].float().numpy(), cs=cs)
            err = np.abs(out[b].cpu().numpy() - ref).max()
            print(f"[rope] decode {case} step={step} b={b} max|err|={err:.3g}", flush=True)
            assert err <= (1e-4 if f32 else 2e-3), err


def test_rope_changes_what_attention_sees():
    """The same cache decoded with and without positions differs (the
    rotation reaches the logits), and the rotated decode is the oracle's."""
    wl = CASES["bf16_batch2"]
    layer = synth.make_layer(wl)
    q = layer.q[0].cuda()
    outs = []
    for freq in (None, FREQ):
        cfg = make_cfg(wl, rope_inv_freq=freq)
        plan = N.Plan(cfg, wl.seq_lens)
        cache, ws, dws = gpu_encode(plan, layer)
        out = torch.empty(wl.batch, wl.Hq, wl.D, dtype=torch.float32, device="cuda")
        akv.decode_attn(plan, cache, q, out, dws)
        torch.cuda.synchronize()
        outs.append(out.cpu().numpy())
    assert np.abs(outs[0] - outs[1]).max() > 1e-2


@pytest.mark.parametrize("mode", ["encoded", "dense"])
def test_rope_appended_tokens_rotate_at_their_positions(mode):
    wl = _wl("rope-append", seq_lens=[900, 1400], steps=5, append=True, seed=44)
    layer = synth.make_layer(wl)
    cfg = make_cfg(wl, rope_inv_freq=FREQ,
                   append_mode=N.APPEND_DENSE if mode == "dense" else N.APPEND_ENCODED)
    plan = N.Plan(cfg, wl.seq_lens)
    cache, ws, dws = gpu_encode(plan, layer)
    pref = []
    for b in range(wl.batch):
        enc = oracle_encode(cfg, layer, b)
        pref.append((enc, _dense(cfg, layer, b, enc, "K"), _dense(cfg, layer, b, enc, "V")))
    tails = [([], []) for _ in range(wl.batch)]
    for n in range(wl.steps):
        out = torch.empty(wl.batch, wl.Hq, wl.D, dtype=torch.float32, device="cuda")
        akv.decode_step(plan, cache, n, layer.k_new[n].cuda(), layer.v_new[n].cuda(), layer.q[n].cuda(), out, dws)
        torch.cuda.synchronize()
        for b in range(wl.batch):
            enc, Kh, Vh = pref[b]
            Kx, Vx = layer.K[b].float().numpy(), layer.V[b].float().numpy()
            tk, tv = [], []
            for h in range(wl.H):
                if mode == "dense":
                    tk.append(layer.k_new[n, b, h].float().numpy())
                    tv.append(layer.v_new[n, b, h].float().numpy())
                    continue
                anc = enc["anchors"][h]
                for X, new, tl in ((Kx, layer.k_new, tk), (Vx, layer.v_new, tv)):
                    a, g = R.assign_vectors(new[n, b, h:h + 1].float().numpy(), X[h][anc], bf16=True)
                    tl.append((X[h][anc[a[0]]].astype(np.float32) * np.float32(g[0])).astype(np.float32))
            tails[b][0].append(np.stack(tk))
            tails[b][1].append(np.stack(tv))
            Kt = np.concatenate([Kh, np.stack(tails[b][0], 1)], 1).astype(np.float32)
            Vt = np.concatenate([Vh, np.stack(tails[b][1], 1)], 1).astype(np.float32)
            cs = R.rope_table(FREQ, wl.D, Kt.shape[1])
            ref = R.attention(Kt, Vt, layer.q[n, b].float().numpy(), cs=cs)
            err = np.abs(out[b].cpu().numpy() - ref).max()
            assert err <= 2e-3, (mode, n, b, err)


def test_rope_all_anchor_cache_is_dense_rotated_attention():
    wl = _wl("rope-dense", seq_lens=[700], anchor_count=700, anchor_frac=0.0, seed=45)
    layer = synth.make_layer(wl)
    cfg = make_cfg(wl, rope_inv_freq=FREQ)
    plan = N.Plan(cfg, wl.seq_lens)
    cache, ws, dws = gpu_encode(plan, layer)
    out = torch.empty(1, wl.Hq, wl.D, dtype=torch.float32, device="cuda")
    akv.decode_attn(plan, cache, layer.q[0].cuda(), out, dws)
    torch.cuda.synchronize()
    K = layer.K[0].float().numpy().astype(np.float32)
    V = layer.V[0].float().numpy().astype(np.float32)
    ref = R.attention(K, V, layer.q[0, 0].float().numpy(), cs=R.rope_table(FREQ, wl.D, 700))
    assert np.abs(out[0].cpu().numpy() - ref).max() <= 2e-3
