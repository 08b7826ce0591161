"""Generated tokens stored exactly (App. E "Generated Tokens"; DENSE append
mode): every appended key and value joins the attention unchanged, so the
decode output after n appends is the oracle's attention over its
reconstruction of the compressed prefix plus the n exact tokens, and the
reconstruction returns those tokens bit for bit.  Batch of ragged requests,
fused decode_step and append-then-attention, bf16 and fp32."""
import numpy as np
import pytest
import torch

import paper_2608_02901_amd as akv
import synth
from oracle import akvref as R
from paper_2608_02901_amd import _native as N
from parity_util import assert_request_parity, gpu_encode, make_cfg, oracle_encode

pytestmark = pytest.mark.gpu

WLS = {
    "bf16_batch2": synth.Workload("dense-bf16", H=2, Hq=8, D=128, seq_lens=[900, 1700], dtype="bf16",
                                  anchor_frac=0.04, budget=0.05, n_centers=48, steps=5, append=True, seed=31),
    "f32": synth.Workload("dense-f32", H=1, Hq=2, D=128, seq_lens=[1100], dtype="f32", anchor_count=64,
                          budget=0.05, quant_group=32, n_centers=48, n_outlier=0, steps=5, append=True, seed=32),
}


@pytest.mark.parametrize("fused", [False, True], ids=["append_then_attn", "decode_step"])
@pytest.mark.parametrize("wl", list(WLS))
def test_dense_append_decodes_exact_tokens(wl, fused):
    w = WLS[wl]
    print(f"[dense-append] {wl} fused={fused}", flush=True)
    layer = synth.make_layer(w)
    cfg = make_cfg(w, append_mode=N.APPEND_DENSE)
    plan = N.Plan(cfg, w.seq_lens)
    cache, ws, dws = gpu_encode(plan, layer)
    f32 = w.dtype == "f32"
    G = cfg.quant_group or w.D
    ref_prefix = []
    for b in range(w.batch):
        enc = oracle_encode(cfg, layer, b)
        assert_request_parity(akv.export(plan, cache.cpu().numpy(), b, 0), enc, cfg)
        ref_prefix.append(tuple(R.reconstruct((layer.K if s == "K" else layer.V)[b].float().numpy(), enc, s, G,
                                              cfg.seed) for s in "KV"))
    for n in range(w.steps):
        out = torch.empty(w.batch, w.Hq, w.D, dtype=torch.float32, device="cuda")
        kn, vn, q = layer.k_new[n].cuda(), layer.v_new[n].cuda(), layer.q[n].cuda()
        if fused:
            akv.decode_step(plan, cache, n, kn, vn, q, out, dws)
        else:
            akv.append(plan, cache, n, kn, vn, dws)
            akv.decode_attn(plan, cache, q, out, dws, n_appended=n + 1)
        torch.cuda.synchronize()
        for b in range(w.batch):
            Kh, Vh = ref_prefix[b]
            Kt = np.concatenate([Kh, layer.k_new[:n + 1, b].float().numpy().transpose(1, 0, 2)], 1)
            Vt = np.concatenate([Vh, layer.v_new[:n + 1, b].float().numpy().transpose(1, 0, 2)], 1)
            ref = R.attention(Kt, Vt, layer.q[n, b].float().numpy())
            err = np.abs(out[b].cpu().numpy() - ref).max()
            assert err <= (1e-4 if f32 else 2e-3), (n, b, err)
    for b in range(w.batch):
        S = w.seq_lens[b]
        exp = akv.export(plan, cache.cpu().numpy(), b, w.steps)
        assert (exp["tail_a_k"] == -1).all() and (exp["tail_gamma_v"] == 0).all()
        for side, si, new in (("K", 0, layer.k_new), ("V", 1, layer.v_new)):
            dense = akv.reconstruct(plan, cache, b, si, n_appended=w.steps).cpu().numpy()
            np.testing.assert_array_equal(dense[:, :S], ref_prefix[b][si])
            np.testing.assert_array_equal(dense[:, S:], new[:, b].float().numpy().transpose(1, 0, 2))

