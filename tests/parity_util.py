"""Shared helpers of the GPU parity tests: run the HIP path and the CPU oracle
on the same seeded inputs and compare what must be identical."""
from __future__ import annotations

import math

import numpy as np
import torch

import paper_2608_02901_amd as akv
from paper_2608_02901_amd import _native as N
from oracle import akvref as R



def make_cfg(wl, **kw):
    base = dict(num_kv_heads=wl.H, num_q_heads=wl.Hq, head_dim=wl.D, window=wl.window,
                anchor_count=wl.anchor_count, anchor_frac=wl.anchor_frac, rho=0.7, kappa=7,
                budget_mode=N.BUDGET_FRACTION, budget=wl.budget, quant_group=wl.quant_group,
                scale_mode=N.SCALE_ABSMAX_OUTER, dtype=N.F32 if wl.dtype == "f32" else N.BF16,
                max_append=wl.steps if wl.append else 0, seed=wl.seed)
    base.update(kw)
    return N.Config.make(**base)


def gpu_encode(plan, layer, override=None):
    cache, ws, dws = plan.alloc("cuda")
    cache.zero_()  # padding between arrays stays defined, so whole blobs compare
    K = [t.cuda() for t in layer.K]
    V = [t.cuda() for t in layer.V]
    Q = [t.cuda() for t in layer.Qobs]
    ov = None if override is None else torch.from_numpy(np.ascontiguousarray(override, np.int32)).cuda()
    keep = akv.encode(plan, K, V, Q, cache, ws, anchor_override=ov)
    torch.cuda.synchronize()
    del keep
    return cache, ws, dws


def rope_freqs(cfg):
    """The rotary frequencies of a config, or None without positions."""
    if not cfg.rope:
        return None
    return np.array(cfg.rope_inv_freq[: cfg.head_dim // 2], np.float32)


def oracle_encode(cfg, layer, b, anchor_override=None):
    K = layer.K[b].float().numpy()
    V = layer.V[b].float().numpy()
    Q = layer.Qobs[b].float().numpy()
    H, S, D = K.shape
    k = plan_k(cfg, S)
    G = cfg.quant_group or D
    return R.encode(K, V, Q, W=cfg.window, k=k, rho=float(np.float32(cfg.rho)), kappa=cfg.kappa,
                    bf16=cfg.dtype == N.BF16, seed=cfg.seed, budget_mode=cfg.budget_mode,
                    budget=float(np.float32(cfg.budget)), budget_count=cfg.budget_count, G=G,
                    scale_mode=cfg.scale_mode, anchor_override=anchor_override, rank_mode=cfg.rank_mode,
                    head_budget=cfg.head_budget, inv_freq=rope_freqs(cfg))


def plan_k(cfg, S):
    if cfg.anchor_count > 0:
        return min(cfg.anchor_count, S)
    return min(S, max(cfg.window, int(math.floor(float(np.float32(cfg.anchor_frac)) * S))))


def selection_gap_ok(pooled, n_top, rel=1e-4):
    """True when the n_top-th and (n_top+1)-th pooled scores are clearly apart."""
    if n_top <= 0 or n_top >= pooled.shape[0]:
        return True
    srt = np.sort(pooled)[::-1]
    a, b = srt[n_top - 1], srt[n_top]
    return a - b > rel * max(a, 1e-30)


def compare_sets(gsel, osel, u, nsel):
    """Residual sets: identical (the pooled top-N of the oracle's fp64
    utilities, ties to the lower head, then the lower position); on a
    mismatch the message gives the mismatched utilities relative to the cut."""
    assert int(gsel.sum()) == int(osel.sum()) == int(nsel)
    diff = gsel != osel
    if diff.any():
        cand = u[u >= 0]
        cut = np.sort(cand)[::-1][nsel - 1] if 0 < nsel <= cand.size else float("nan")
        rel = np.abs(u[diff] - cut) / cut
        raise AssertionError(f"{int(diff.sum())} residual-set mismatches; oracle utilities at relative distance "
                             f"{np.sort(rel)[:6]} from the cut {cut:.6g}")
    return 0


def assert_request_parity(exp, enc, cfg, check_sets=True):
    """Bit-exact integer and coefficient streams of one request."""
    np.testing.assert_array_equal(exp["anchors"], enc["anchors"])
    np.testing.assert_array_equal(exp["a_k"], enc["aK"])
    np.testing.assert_array_equal(exp["a_v"], enc["aV"])
    np.testing.assert_array_equal(exp["gamma_k"], enc["gK"].astype(np.float32))
    np.testing.assert_array_equal(exp["gamma_v"], enc["gV"].astype(np.float32))
    mism = 0
    for side in ("k", "v"):
        gsel = exp["sel_" + side].astype(bool)
        osel = enc["sel" + side.upper()].astype(bool)
        u = enc["u" + side.upper()]
        n = int(enc["nsel"][0 if side == "k" else 1])
        if check_sets:
            mism += compare_sets(gsel, osel, u, n)
        both = gsel & osel
        np.testing.assert_array_equal(exp["codes_" + side][both], enc["codes" + side.upper()][both])
        np.testing.assert_array_equal(exp["scales_" + side][both], enc["scales" + side.upper()][both])
    return mism
