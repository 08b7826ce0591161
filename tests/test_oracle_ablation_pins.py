"""Pins of the oracle's ablation variants (Sec. 4.3 "Ablations and
Analysis") against numpy/scipy written from their definitions: the residual
rankings by cosine, residual norm, attention and at random; equal per-head
budgets; and the 2-bit quantizer without rotation or Lloyd-Max codebook.
No GPU."""
import math

import numpy as np
import pytest
import scipy.special

from oracle import akvref as R


def _bf16(x):
    x = np.asarray(x, np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def _problem(seed=0, H=2, Hq=4, S=150, D=16, W=6):
    rng = np.random.default_rng(seed)
    K = _bf16(rng.standard_normal((H, S, D)) * 1.2)
    V = _bf16(rng.standard_normal((H, S, D)))
    Q = _bf16(rng.standard_normal((Hq, W, D)))
    return K, V, Q


def _top(keys, N, per_head=False):
    """numpy top-N over (key desc, head asc, position asc); keys < 0 never."""
    H, S = keys.shape
    sel = np.zeros((H, S), bool)
    groups = [(h,) for h in range(H)] if per_head else [tuple(range(H))]
    n_each = N // H if per_head else N
    for hs in groups:
        cand = [(-keys[h, t], h, t) for h in hs for t in range(S) if keys[h, t] >= 0]
        cand.sort()
        for _, h, t in cand[:n_each]:
            sel[h, t] = True
    return sel


def _numpy_keys(mode, K, V, Q, enc):
    H, S, D = K.shape
    W = Q.shape[1]
    g = Q.shape[0] // H
    out = {}
    for side, X in (("K", K), ("V", V)):
        keys = np.full((H, S), -1.0)
        for h in range(H):
            anc = enc["anchors"][h]
            Qg = Q[h * g:(h + 1) * g].reshape(-1, D)
            # raw selector score: mean causal softmax of the observation rows
            A = np.zeros((g * W, S))
            for w in range(g * W):
                last = S - W + w % W
                A[w, : last + 1] = scipy.special.softmax(Qg[w] @ K[h, : last + 1].T / math.sqrt(D))
            sc = A.mean(0)
            for t in range(S):
                if t in anc:
                    continue
                a = X[h][anc[enc["a" + side][h, t]]]
                x = X[h, t]
                if mode == R.RANK_COSINE:
                    keys[h, t] = 1 - abs(x @ a) / math.sqrt((x @ x) * (a @ a))
                elif mode == R.RANK_RESNORM:
                    gm = np.float32(enc["g" + side][h, t])
                    r = x.astype(np.float32) - gm * a.astype(np.float32)
                    keys[h, t] = float(r.astype(np.float64) @ r.astype(np.float64))
                elif mode == R.RANK_ATTENTION:
                    keys[h, t] = sc[t]
        out[side] = keys
    return out


@pytest.mark.parametrize("mode", [R.RANK_COSINE, R.RANK_RESNORM, R.RANK_ATTENTION])
def test_residual_ranking_alternatives_match_numpy(mode):
    """Sec. 4.3 "Residual Ranking" (i)-(iii): the residual sets are the
    pooled top-N of the alternative key, computed here from its definition."""
    K, V, Q = _problem(1)
    enc = R.encode(K, V, Q, W=6, k=20, bf16=True, budget=0.1, G=16, rank_mode=mode)
    keys = _numpy_keys(mode, K, V, Q, enc)
    N = int(enc["nsel"][0])
    for side in "KV":
        np.testing.assert_allclose(enc["u" + side][enc["u" + side] >= 0], keys[side][keys[side] >= 0],
                                   rtol=1e-9, atol=1e-15)
        np.testing.assert_array_equal(enc["sel" + side].astype(bool), _top(keys[side], N))


def test_random_ranking_is_uniform_and_seeded():
    """Sec. 4.3 "Residual Ranking" (iv): every candidate is equally likely to
    get a residual (chi-square over many seeds), and the draw follows the seed."""
    K, V, Q = _problem(2, H=1, Hq=1, S=60)
    k, N = 12, 10
    counts = np.zeros(60)
    base = None
    for seed in range(400):
        enc = R.encode(K, V, Q, W=6, k=k, bf16=True, budget_mode=R.BUDGET_COUNT, budget_count=N, G=16,
                       rank_mode=R.RANK_RANDOM, seed=seed, anchor_override=np.r_[np.arange(0, 36, 6), 54 + np.arange(6)][None])
        counts += enc["selK"][0]
        if seed == 0:
            base = enc["selK"].copy()
    free = np.setdiff1d(np.arange(60), np.r_[np.arange(0, 36, 6), 54 + np.arange(6)])
    assert counts.sum() == 400 * N and np.all(counts[np.setdiff1d(np.arange(60), free)] == 0)
    import scipy.stats
    exp = 400 * N / free.size
    chi2 = float(np.sum((counts[free] - exp) ** 2 / exp))
    assert scipy.stats.chi2.sf(chi2, df=free.size - 1) > 1e-4
    again = R.encode(K, V, Q, W=6, k=k, bf16=True, budget_mode=R.BUDGET_COUNT, budget_count=N, G=16,
                     rank_mode=R.RANK_RANDOM, seed=0, anchor_override=np.r_[np.arange(0, 36, 6), 54 + np.arange(6)][None])
    np.testing.assert_array_equal(again["selK"], base)


def test_equal_per_head_budgets():
    """Sec. 4.3 "Component Removal" (ii): every head takes floor(N / H) of its
    own highest utilities instead of a share of the pooled top-N."""
    K, V, Q = _problem(3, H=3, Hq=6)
    enc = R.encode(K, V, Q, W=6, k=20, bf16=True, budget_mode=R.BUDGET_COUNT, budget_count=40, G=16, head_budget=1)
    for side in "KV":
        sel = enc["sel" + side].astype(bool)
        assert sel.sum(axis=1).tolist() == [13, 13, 13]
        np.testing.assert_array_equal(sel, _top(enc["u" + side], 40, per_head=True))
    pooled = R.encode(K, V, Q, W=6, k=20, bf16=True, budget_mode=R.BUDGET_COUNT, budget_count=40, G=16)
    assert pooled["selK"].sum() == 40 and sorted(pooled["selK"].sum(axis=1)) != [13, 13, 14]


def test_naive_codec_is_the_uniform_quantizer_without_rotation():
    """Sec. 4.3 "Component Removal" (iv): no rotation, uniform 4 levels on
    [-A, A] (A = group absmax, levels +-A/4, +-3A/4): codes equal numpy's
    uniform quantizer of the raw residual, and the error is at most A/4 per
    coordinate (the cell half-width)."""
    rng = np.random.default_rng(4)
    D, G = 32, 8
    for _ in range(50):
        r = rng.standard_normal(D).astype(np.float32)
        codes, scales = R.codec_encode(r, G, R.SCALE_NAIVE, 7)
        got = np.array([(codes[j // 4] >> (2 * (j % 4))) & 3 for j in range(D)])
        A = np.abs(r.reshape(-1, G)).max(axis=1).repeat(G)
        want = np.where(r < 0, np.where(np.abs(r) > A / 2, 0, 1), np.where(np.abs(r) > A / 2, 3, 2))
        np.testing.assert_array_equal(got, want)
        np.testing.assert_array_equal(scales, np.abs(r.reshape(-1, G)).max(axis=1).astype(np.float32) * np.float32(0.25))
        rt = R.codec_decode(codes, scales, D, G, 7, R.SCALE_NAIVE)
        assert np.all(np.abs(rt - r) <= A / 4 * (1 + 1e-6))
