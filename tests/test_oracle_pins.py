"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: a value the
paper prints, a published constant, a library routine, a closed form, an
invariant or a theorem, or exhaustive search on tiny inputs.  No GPU needed.
"""
import json
import math
import os

import numpy as np
import pytest
import scipy.linalg
import scipy.special
import scipy.stats

from oracle import akvref as R

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _bf16(x):
    """Round fp32 values to bf16 (RNE), returned as float64."""
    x = np.asarray(x, np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


# --------------------------------------------------------------------------- hashing

def test_splitmix64_published_output():
    # Reference implementation of SplitMix64 (Steele, Lea & Flood 2014): the
    # first output of a generator seeded with 0 is 0xE220A8397B1DCDAF.
    assert R.splitmix64(0) == 0xE220A8397B1DCDAF


def test_signs_are_balanced_and_seeded():
    s0 = R.hadamard_signs(0, 4096)
    s1 = R.hadamard_signs(1, 4096)
    assert set(np.unique(s0)) == {-1.0, 1.0}
    assert abs(s0.mean()) < 0.06
    assert (s0 != s1).mean() > 0.4


# --------------------------------------------------------------------------- rotation (App. A.1)

@pytest.mark.parametrize("D", [4, 8, 64, 128])
def test_fwht_equals_dense_sylvester_product(D):
    rng = np.random.default_rng(D)
    z = rng.integers(-50, 50, size=D).astype(np.float32)
    H = scipy.linalg.hadamard(D)  # Sylvester construction
    np.testing.assert_array_equal(R.fwht(z), (H @ z.astype(np.float64)).astype(np.float32))


def test_rotation_is_orthogonal():
    D = 128
    s = R.hadamard_signs(7, D).astype(np.float64)
    U = scipy.linalg.hadamard(D) * s[None, :] / math.sqrt(D)
    np.testing.assert_allclose(U.T @ U, np.eye(D), atol=1e-12)
    # The oracle's codec applies FWHT(s * r); U r equals that divided by sqrt(D).
    rng = np.random.default_rng(0)
    r = rng.standard_normal(D).astype(np.float32)
    z = R.fwht(s.astype(np.float32) * r)
    np.testing.assert_allclose(z / math.sqrt(D), U @ r.astype(np.float64), rtol=1e-5, atol=1e-5)


# --------------------------------------------------------------------------- codebook (Sec. 3.1)

def _lloyd_max_gaussian(levels=4, iters=2000):
    """Lloyd's algorithm on N(0,1): alternate centroid and midpoint conditions."""
    y = np.linspace(-1.5, 1.5, levels)
    for _ in range(iters):
        t = np.concatenate([[-np.inf], 0.5 * (y[1:] + y[:-1]), [np.inf]])
        pdf = scipy.stats.norm.pdf(t)
        cdf = scipy.stats.norm.cdf(t)
        y = (pdf[:-1] - pdf[1:]) / (cdf[1:] - cdf[:-1])
    t = 0.5 * (y[1:] + y[:-1])
    mse = 0.0
    edges = np.concatenate([[-np.inf], t, [np.inf]])
    for i in range(levels):
        a, b = edges[i], edges[i + 1]
        # E[(x - y_i)^2 ; a < x < b]
        m0 = scipy.stats.norm.cdf(b) - scipy.stats.norm.cdf(a)
        m1 = scipy.stats.norm.pdf(a) - scipy.stats.norm.pdf(b)
        pa = 0.0 if np.isinf(a) else a * scipy.stats.norm.pdf(a)
        pb = 0.0 if np.isinf(b) else b * scipy.stats.norm.pdf(b)
        m2 = m0 + pa - pb
        mse += m2 - 2 * y[i] * m1 + y[i] ** 2 * m0
    return y, t, mse


def test_codebook_constants_match_lloyd_iteration():
    y, t, mse = _lloyd_max_gaussian()
    # Decode of codes 0..3 at scale 1 gives the oracle's levels; read them back
    # through the codec with D = 4 (FWHT of a 1-hot pattern is exact).
    D = 4
    s = R.hadamard_signs(0, D)
    got = []
    for c in range(4):
        codes = np.array([c | (c << 2) | (c << 4) | (c << 6)], np.uint8)
        rt = R.codec_decode(codes, np.array([1.0], np.float32), D, D, 0)
        # all-equal codes -> zhat = level * ones; FWHT(ones) = D e_0; r~ = s * e_0 * level
        got.append(rt[0] * s[0])
    np.testing.assert_allclose(got, y, atol=2e-7)
    assert abs(t[2] - 0.9815988) < 2e-7
    assert abs(mse - 0.1174818) < 1e-6


def test_codec_planted_codes_roundtrip():
    D, G = 128, 32
    rng = np.random.default_rng(3)
    y, t, _ = _lloyd_max_gaussian()
    s = R.hadamard_signs(11, D).astype(np.float64)
    codes_true = rng.integers(0, 4, size=D)
    sigma = np.array([0.5, 1.0, 2.0, 4.0])
    zhat = np.repeat(sigma, G) * y[codes_true]
    # The RMS reading recovers sigma only approximately; LITERAL / OUTER take the
    # absmax, which on a planted grid that contains +-L1 in every group is L1*sigma.
    for g in range(4):
        zhat[g * G] = sigma[g] * y[3]
        codes_true[g * G] = 3
    r = (s * (scipy.linalg.hadamard(D) @ zhat) / D).astype(np.float32)
    codes, scales = R.codec_encode(r, G, R.SCALE_ABSMAX_OUTER, 11)
    unpacked = np.array([(codes[j // 4] >> (2 * (j % 4))) & 3 for j in range(D)])
    np.testing.assert_array_equal(unpacked, codes_true)
    np.testing.assert_allclose(scales, sigma, rtol=1e-5)
    rt = R.codec_decode(codes, scales, D, G, 11)
    np.testing.assert_allclose(rt, r, rtol=1e-4, atol=1e-5)


@pytest.mark.parametrize("mode,lo,hi", [(R.SCALE_RMS, 0.110, 0.128), (R.SCALE_ABSMAX_OUTER, 0.2, 0.4),
                                        (R.SCALE_ABSMAX_LITERAL, 0.45, 0.75)])
def test_codec_distortion_eta(mode, lo, hi):
    # Eq. eta: relative squared distortion of the codec.  For a Gaussian residual
    # the RMS reading approaches the Lloyd-Max MSE 0.1175; a dropped 1/D or a
    # wrong sign pattern in decode would push every mode far above 1.
    D = 128
    rng = np.random.default_rng(5)
    num = den = 0.0
    for _ in range(200):
        r = rng.standard_normal(D).astype(np.float32)
        c, sc = R.codec_encode(r, D, mode, 9)
        rt = R.codec_decode(c, sc, D, D, 9)
        num += float(np.sum((r.astype(np.float64) - rt) ** 2))
        den += float(np.sum(r.astype(np.float64) ** 2))
    eta = num / den
    assert lo < eta < hi, eta


def test_codec_zero_residual():
    D = 128
    codes, scales = R.codec_encode(np.zeros(D, np.float32), D, R.SCALE_ABSMAX_OUTER, 0)
    assert np.all(codes == 0b10101010) and np.all(scales == 0)
    np.testing.assert_array_equal(R.codec_decode(codes, scales, D, D, 0), np.zeros(D, np.float32))


# --------------------------------------------------------------------------- byte budget (Sec. 3.4, App. A.1)

def test_byte_budget_worked_example():
    with open(os.path.join(GOLDEN, "worked_example.json")) as f:
        ex = json.load(f)
    S, H, D, W, k, theta = ex["S"], ex["H"], ex["D"], ex["W"], ex["k"], ex["theta"]
    mbase = R.base_bytes(S, H, D, W, k)
    assert round(mbase / 1e6, 2) == ex["M_base_MB"]
    assert round(mbase / (4 * S * H * D) * 100, 1) == ex["M_base_percent"]
    assert round((theta * 4 * S * H * D - mbase) / 1e6, 2) == ex["left_MB"]
    assert round(4 * S * H * D / 1e6, 1) == ex["M_full_MB"]
    assert R.theta_budget(S, H, D, W, k, D, theta) == ex["N"]
    assert 2 * H * (S - W) == ex["token_sides"]


def test_byte_budget_is_zero_when_base_exceeds_target():
    assert R.theta_budget(4096, 8, 128, 32, 2048, 128, 0.01) == 0


# --------------------------------------------------------------------------- assignment (Sec. 3.1)

def _rand_bf16(rng, *shape):
    return _bf16(rng.standard_normal(shape))


def test_assignment_matches_exhaustive_cosine_search():
    rng = np.random.default_rng(0)
    S, D, k = 64, 16, 6
    X = _rand_bf16(rng, S, D)
    anchors = np.sort(rng.choice(S, k, replace=False)).astype(np.int32)
    a, g, r = R.assign_tokens(X, anchors, bf16=True)
    A = X[anchors]
    for t in range(S):
        if t in anchors:
            assert a[t] == list(anchors).index(t) and g[t] == 1.0
            assert np.all(r[t] == 0)
            continue
        cos = np.abs(A @ X[t]) / (np.linalg.norm(A, axis=1) * np.linalg.norm(X[t]))
        assert a[t] == int(np.argmax(cos))
        gam = float(X[t] @ A[a[t]] / (A[a[t]] @ A[a[t]]))
        assert g[t] == _bf16(np.float32(gam))
        np.testing.assert_array_equal(r[t], (X[t].astype(np.float32) -
                                              np.float32(g[t]) * A[a[t]].astype(np.float32)))


def test_assignment_special_cases():
    D = 8
    A = np.zeros((4, D))
    A[0, 0] = 2.0          # e0 * 2
    A[1, 1] = 1.0          # e1
    A[2, 0] = -4.0         # antiparallel to anchor 0
    A[3, 2] = 0.0          # zero anchor
    xs = np.zeros((4, D))
    xs[0, 1] = 3.0         # exactly 3 * anchor 1
    xs[1, 0] = 1.0         # parallel to anchors 0 and 2: tie -> lowest index 0
    xs[2, 3] = 5.0         # orthogonal to every anchor: all scores 0 -> index 0
    xs[3] = 0.0            # zero token
    a, g = R.assign_vectors(xs, A, bf16=False)
    assert list(a) == [1, 0, 0, 0]
    assert g[0] == 3.0 and g[1] == 0.5 and g[2] == 0.0 and g[3] == 0.0
    # antiparallel: a token along -e0 picks anchor 0 with negative gamma
    a2, g2 = R.assign_vectors(-xs[1:2], A, bf16=False)
    assert a2[0] == 0 and g2[0] == -0.5


def test_projection_closed_forms_fp32():
    rng = np.random.default_rng(1)
    S, D, k = 200, 128, 10
    X = rng.standard_normal((S, D)).astype(np.float32).astype(np.float64)
    anchors = np.arange(0, S, S // k)[:k].astype(np.int32)
    a, g, r = R.assign_tokens(X, anchors, bf16=False)
    for t in range(S):
        if t in anchors:
            continue
        an = X[anchors[a[t]]]
        gam = X[t] @ an / (an @ an)
        assert abs(g[t] - gam) <= 1e-7 * abs(gam) + 1e-30
        # residual is orthogonal to its anchor up to fp32 rounding
        assert abs(r[t].astype(np.float64) @ an) < 1e-5 * np.linalg.norm(X[t]) * np.linalg.norm(an)
        # ||r||^2 = ||x||^2 (1 - cos^2)  (Sec. 4.3, pre-RoPE paragraph)
        c = X[t] @ an / (np.linalg.norm(X[t]) * np.linalg.norm(an))
        np.testing.assert_allclose(r[t].astype(np.float64) @ r[t], (X[t] @ X[t]) * (1 - c * c), rtol=1e-4)


# --------------------------------------------------------------------------- selection (Sec. 3.2, App. A.2)

def test_selector_picks_planted_attention_sink_and_window():
    rng = np.random.default_rng(2)
    S, D, W, g, k, kappa = 96, 16, 8, 2, 20, 3
    K = _rand_bf16(rng, S, D) * 0.1
    Q = _rand_bf16(rng, g, W, D)
    # Position 17 aligns with the mean observation query: it must be a top anchor.
    K[17] = _bf16(4.0 * Q.reshape(-1, D).mean(0) / np.linalg.norm(Q.reshape(-1, D).mean(0)) * 3)
    V = _rand_bf16(rng, S, D)
    M, Z, Y = R.obs_head(K, V, Q)
    sc, pooled = R.selector_scores(K, Q, M, Z, kappa)
    assert int(np.argmax(sc)) == 17
    anchors = R.select_anchors(pooled, S, W, k, 0.7, 0, 0)
    assert len(anchors) == k and np.all(np.diff(anchors) > 0)
    assert set(range(S - W, S)) <= set(anchors.tolist())
    assert 17 in anchors
    # n_top = floor(0.7 * 12) = 8 best pooled scores are all anchors
    top = np.argsort(-pooled, kind="stable")[:R.n_top(k, W, 0.7)]
    assert set(top.tolist()) <= set(anchors.tolist())


def test_selector_scores_are_causal_softmax_averages():
    # Every observation row is a probability distribution over t <= its own
    # position, so the raw scores summed over all positions (including the
    # window, reconstructed from M and Z) equal 1 per row, averaged over rows.
    rng = np.random.default_rng(4)
    S, D, W, g = 40, 8, 4, 3
    K = _rand_bf16(rng, S, D)
    V = _rand_bf16(rng, S, D)
    Q = _rand_bf16(rng, g, W, D)
    M, Z, Y = R.obs_head(K, V, Q)
    # scipy softmax row by row with the causal mask, as a library check
    Qr = Q.reshape(g * W, D)
    logits = Qr @ K.T / math.sqrt(D)
    for w in range(g * W):
        last = S - W + (w % W)
        p = scipy.special.softmax(logits[w, : last + 1])
        np.testing.assert_allclose(Y[w], p @ V[: last + 1], rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(M[w], logits[w, : last + 1].max(), rtol=1e-14)
    sc, pooled = R.selector_scores(K, Q, M, Z, 1)
    np.testing.assert_allclose(pooled, sc)


def test_selector_ties_go_to_lower_positions():
    S, W, k = 50, 5, 15
    pooled = np.ones(S - W)
    anchors = R.select_anchors(pooled, S, W, k, 1.0, 0, 0)  # rho = 1: all by score
    np.testing.assert_array_equal(anchors, np.r_[np.arange(10), np.arange(S - W, S)])


def test_random_share_is_uniform_without_replacement():
    S, W, k = 40, 4, 14
    pooled = np.zeros(S - W)
    pooled[:3] = 1.0
    counts = np.zeros(S - W)
    for seed in range(3000):
        anc = R.select_anchors(pooled, S, W, k, 0.3, seed, 0)  # n_top = 3 -> 7 random
        assert len(set(anc.tolist())) == k
        counts[anc[anc < S - W]] += 1
    assert np.all(counts[:3] == 3000)
    rest = counts[3:]
    expected = 3000 * 7 / 33
    chi2 = float(np.sum((rest - expected) ** 2 / expected))
    assert scipy.stats.chi2.sf(chi2, df=32) > 1e-4


# --------------------------------------------------------------------------- budget (Sec. 3.4)

def test_budget_pools_heads_and_breaks_ties():
    u = np.array([[0.5, -1.0, 0.2, 0.2], [0.9, 0.2, -1.0, 0.1]])
    sel, n = R.budget_select(u, 3)
    assert n == 3
    np.testing.assert_array_equal(sel, [[1, 0, 1, 0], [1, 0, 0, 0]])
    sel, n = R.budget_select(u, 100)
    assert n == 6 and sel.sum() == 6 and sel[0, 1] == 0 and sel[1, 2] == 0


# --------------------------------------------------------------------------- utilities (Sec. 3.3, App. A.3)

def test_utilities_match_finite_difference_of_attention_output():
    """u^K and u^V are the squared first-order output change of dropping one
    token's residual (Eq. channels), for a single observation query."""
    rng = np.random.default_rng(6)
    S, D = 30, 16
    K = rng.standard_normal((S, D)) * 0.7
    V = rng.standard_normal((S, D))
    q = rng.standard_normal((1, 1, D))
    M, Z, Y = R.obs_head(K, V, q)
    t = 7
    rK = rng.standard_normal((1, D)).astype(np.float32)
    rV = rng.standard_normal((1, D)).astype(np.float32)
    uK, uV = R.utilities(K, V, q, M, Z, Y, np.array([t]), rK, rV)

    def out(Kx, Vx):
        p = scipy.special.softmax(Kx @ q[0, 0] / math.sqrt(D))
        return p @ Vx, p

    y0, p0 = out(K, V)
    errs = []
    for eps in (1e-4, 1e-5):
        K1 = K.copy()
        K1[t] -= eps * rK[0]
        dy = (out(K1, V)[0] - y0) / eps
        # First order, one perturbed token: the centring term of the K channel
        # vanishes (sum_t alpha_t (V_t - y) = 0), leaving alpha_t ds_t (V_t - y)
        # with ds_t = -q.r/sqrt(D), whose squared norm is the utility summand.
        rel = abs(float(dy @ dy) / uK[0] - 1.0)
        assert rel < 20 * eps, rel
        errs.append(rel)
        V1 = V.copy()
        V1[t] -= eps * rV[0]
        dyv = (out(K, V1)[0] - y0) / eps
        np.testing.assert_allclose(float(dyv @ dyv), uV[0], rtol=1e-6)
    assert errs[1] < errs[0] / 5  # the remainder is second order


# --------------------------------------------------------------------------- decode attention (Eq. exact-attention)

def test_all_anchor_encoding_reconstructs_exactly_and_attends_densely():
    rng = np.random.default_rng(8)
    H, Hq, S, D, W = 2, 4, 48, 16, 8
    K = _rand_bf16(rng, H, S, D)
    V = _rand_bf16(rng, H, S, D)
    Q = _rand_bf16(rng, Hq, W, D)
    enc = R.encode(K, V, Q, W=W, k=S, bf16=True, G=D)
    assert np.all(enc["selK"] == 0) and enc["nsel"].tolist() == [0, 0]
    Kh = R.reconstruct(K, enc, "K", D, 0)
    Vh = R.reconstruct(V, enc, "V", D, 0)
    np.testing.assert_array_equal(Kh, K.astype(np.float32))
    np.testing.assert_array_equal(Vh, V.astype(np.float32))
    q = rng.standard_normal((Hq, D))
    y = R.attention(Kh, Vh, q)
    for j in range(Hq):
        h = j // (Hq // H)
        p = scipy.special.softmax(K[h] @ q[j] / math.sqrt(D))
        np.testing.assert_allclose(y[j], p @ V[h], rtol=1e-12, atol=1e-13)


def test_output_error_theorem_holds_on_compressed_cache():
    """App. A.4: ||y - y^|| <= sum_t a^_t ||V_t - V^_t|| + 2 Vmax tanh(mu)."""
    rng = np.random.default_rng(9)
    H, Hq, S, D, W, k = 2, 4, 160, 32, 8, 24
    K = _rand_bf16(rng, H, S, D)
    V = _rand_bf16(rng, H, S, D)
    Q = _rand_bf16(rng, Hq, W, D)
    enc = R.encode(K, V, Q, W=W, k=k, bf16=True, budget=0.1, G=D)
    Kh = R.reconstruct(K, enc, "K", D, 0).astype(np.float64)
    Vh = R.reconstruct(V, enc, "V", D, 0).astype(np.float64)
    for _ in range(5):
        q = rng.standard_normal((Hq, D)) * 2
        y = R.attention(K.astype(np.float32), V.astype(np.float32), q)
        yh = R.attention(Kh.astype(np.float32), Vh.astype(np.float32), q)
        for j in range(Hq):
            h = j // (Hq // H)
            ah = scipy.special.softmax(Kh[h] @ q[j] / math.sqrt(D))
            ev = float(np.sum(ah * np.linalg.norm(V[h] - Vh[h], axis=1)))
            mu = np.linalg.norm(q[j]) * np.max(np.linalg.norm(K[h] - Kh[h], axis=1)) / math.sqrt(D)
            bound = ev + 2 * np.max(np.linalg.norm(V[h], axis=1)) * math.tanh(mu)
            err = np.linalg.norm(y[j] - yh[j])
            assert err <= bound * (1 + 1e-9), (err, bound)
            assert err > 0


def test_anchors_reconstruct_exactly_and_budget_counts():
    rng = np.random.default_rng(10)
    H, Hq, S, D, W, k = 2, 2, 200, 32, 8, 20
    K = _rand_bf16(rng, H, S, D)
    V = _rand_bf16(rng, H, S, D)
    Q = _rand_bf16(rng, Hq, W, D)
    enc = R.encode(K, V, Q, W=W, k=k, bf16=True, budget=0.05, G=8)
    N = int(math.floor(np.float32(0.05) * H * S))
    assert enc["nsel"].tolist() == [N, N]
    assert enc["selK"].sum() == N and enc["selV"].sum() == N
    Kh = R.reconstruct(K, enc, "K", 8, 0)
    for h in range(H):
        anc = enc["anchors"][h]
        np.testing.assert_array_equal(Kh[h][anc], K[h][anc].astype(np.float32))
        assert np.all(enc["uK"][h][anc] == -1) and np.all(enc["selK"][h][anc] == 0)
        assert np.all(enc["gK"][h][anc] == 1.0)
    # selected residuals reduce the reconstruction error of their token
    for h in range(H):
        sel = enc["selK"][h].astype(bool)
        a = enc["aK"][h]
        proj = enc["gK"][h][:, None] * K[h][enc["anchors"][h][a]]
        e_proj = np.linalg.norm(K[h] - proj, axis=1)
        e_rec = np.linalg.norm(K[h] - Kh[h], axis=1)
        assert np.all(e_rec[sel] < e_proj[sel])
