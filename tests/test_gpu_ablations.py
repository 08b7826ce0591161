"""GPU parity of the ablation variants of Sec. 4.3 against the oracle.

Residual ranking by cosine to the nearest anchor, residual norm, attention
score and at random; equal per-head residual budgets instead of the budget
pooled over heads; 2-bit quantization without the Hadamard rotation and the
Lloyd-Max codebook.  Every variant keeps the bit-exact bar of the method:
anchors, assignments, coefficients, residual sets (the exact top-N of the
oracle's fp64 keys), codes and scales; reconstructions bit-exact; decode
within the attention tolerance."""
import numpy as np
import pytest
import torch

import paper_2608_02901_amd as akv
import synth
from oracle import akvref as R
from paper_2608_02901_amd import _native as N
from parity_util import assert_request_parity, gpu_encode, make_cfg, oracle_encode

pytestmark = pytest.mark.gpu


def _wl(name, **kw):
    base = dict(name=name, H=2, Hq=8, D=128, seq_lens=[1000], dtype="bf16", anchor_frac=0.04, budget=0.05,
                n_centers=48, seed=21)
    base.update(kw)
    return synth.Workload(**base)


WLS = {
    "bf16": _wl("bf16"),
    "bf16_batch3": _wl("bf16_batch3", H=4, Hq=8, seq_lens=[700, 1500, 2300], seed=22),
    "f32_group32": _wl("f32_group32", H=1, Hq=1, dtype="f32", seq_lens=[1200], anchor_count=64, anchor_frac=0.0,
                       quant_group=32, n_outlier=0, seed=23),
}
RANKS = {"cosine": N.RANK_COSINE, "resnorm": N.RANK_RESNORM, "attention": N.RANK_ATTENTION,
         "random": N.RANK_RANDOM}


def _run(wl, **kw):
    layer = synth.make_layer(wl)
    cfg = make_cfg(wl, **kw)
    plan = N.Plan(cfg, wl.seq_lens)
    cache, ws, dws = gpu_encode(plan, layer)
    out = []
    for b in range(wl.batch):
        enc = oracle_encode(cfg, layer, b)
        exp = akv.export(plan, cache.cpu().numpy(), b, 0)
        assert_request_parity(exp, enc, cfg)
        out.append((exp, enc))
    return layer, cfg, plan, cache, dws, out


@pytest.mark.parametrize("wl", list(WLS))
@pytest.mark.parametrize("rank", list(RANKS))
def test_rank_ablation_matches_oracle(rank, wl):
    print(f"[ablation] rank={rank} wl={wl}", flush=True)
    *_, out = _run(WLS[wl], rank_mode=RANKS[rank])
    for exp, enc in out:
        for side in ("k", "v"):
            assert exp["sel_" + side].sum() == enc["nsel"][0 if side == "k" else 1]


@pytest.mark.parametrize("rank", ["utility", "resnorm"])
@pytest.mark.parametrize("wl", ["bf16", "bf16_batch3"])
def test_equal_per_head_budget_matches_oracle(wl, rank):
    print(f"[ablation] per-head budget rank={rank} wl={wl}", flush=True)
    w = WLS[wl]
    mode = N.RANK_UTILITY if rank == "utility" else RANKS[rank]
    layer, cfg, plan, *_, out = _run(w, rank_mode=mode, head_budget=1)
    for b, (exp, enc) in enumerate(out):
        ri = plan.requests[b]
        for side, n in (("k", ri.residuals_k), ("v", ri.residuals_v)):
            per_head = exp["sel_" + side].reshape(w.H, -1).sum(1)
            assert (per_head == n // w.H).all(), per_head  # every head holds exactly floor(N / H)


@pytest.mark.parametrize("wl", ["bf16", "f32_group32"])
def test_naive_codec_matches_oracle(wl):
    print(f"[ablation] naive codec wl={wl}", flush=True)
    w = WLS[wl]
    layer, cfg, plan, cache, dws, out = _run(w, scale_mode=N.SCALE_NAIVE)
    G = cfg.quant_group or 128
    q = synth.make_layer(w, steps=1).q[0]
    res = torch.empty(w.batch, w.Hq, w.D, dtype=torch.float32, device="cuda")
    akv.decode_attn(plan, cache, q.cuda(), res, dws)
    torch.cuda.synchronize()
    for b, (exp, enc) in enumerate(out):
        dense = {}
        for side, si in (("K", 0), ("V", 1)):
            X = (layer.K if side == "K" else layer.V)[b].float().numpy()
            ref = R.reconstruct(X, enc, side, G, cfg.seed)
            got = akv.reconstruct(plan, cache, b, si).cpu().numpy()
            np.testing.assert_array_equal(got, ref)
            dense[side] = ref
        ref = R.attention(dense["K"], dense["V"], q[b].float().numpy())
        err = np.abs(res[b].cpu().numpy() - ref).max()
        print(f"[ablation] naive decode b={b} max|err|={err:.3g}", flush=True)
        assert err <= (1e-4 if w.dtype == "f32" else 2e-3), err
