"""Pins of the oracle's observation-window steps against plain numpy/scipy
brute force: the selector score and its average pooling (App. A.2 Eq.
selector-score) and the multi-row utilities (Sec. 3.3 Eq. utilities).

Each brute force is written from the formula with library primitives only
(scipy's softmax, numpy's convolution and matrix products), so a dropped
term, a wrong row-to-query mapping or an off-centre pool in the oracle fails
here.  The mutation tests plant such mistakes in a private copy of the
oracle's source and check that the pins catch every one of them.  No GPU.
"""
import ctypes
import math
import os
import subprocess

import numpy as np
import pytest
import scipy.special

from oracle import akvref as R

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE_SRC = os.path.join(ROOT, "oracle", "akvref.c")


def _bf16(x):
    x = np.asarray(x, np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def _problem(seed, S=41, D=8, W=3, g=2):
    rng = np.random.default_rng(seed)
    K = _bf16(rng.standard_normal((S, D)) * 1.3)
    V = _bf16(rng.standard_normal((S, D)))
    Q = _bf16(rng.standard_normal((g, W, D)))
    return K, V, Q


def _causal_alpha(K, Q):
    """alpha[w, t] for the m = g*W observation rows in (query head, window
    offset) order: row w = jj*W + i is query head jj at position S-W+i and
    attends to t <= S-W+i (scipy softmax of the scaled logits)."""
    S, D = K.shape
    g, W, _ = Q.shape
    A = np.zeros((g * W, S))
    for jj in range(g):
        for i in range(W):
            last = S - W + i
            lg = K[: last + 1] @ Q[jj, i] / math.sqrt(D)
            A[jj * W + i, : last + 1] = scipy.special.softmax(lg)
    return A


def _brute_selector(K, Q, kappa):
    S = K.shape[0]
    W = Q.shape[1]
    A = _causal_alpha(K, Q)
    sc = A[:, : S - W].mean(axis=0)                        # column means over the m rows
    pooled = np.convolve(sc, np.ones(kappa) / kappa, "same")  # centred, zero padded, / kappa
    return sc, pooled


def _brute_utilities(K, V, Q, toks, rK, rV):
    D = K.shape[1]
    A = _causal_alpha(K, Q)
    Y = A @ V                                 # y_w, one row per observation row
    Qr = Q.reshape(-1, D)
    uK, uV = [], []
    for i, t in enumerate(toks):
        a2 = A[:, t] ** 2
        qr = Qr @ rK[i].astype(np.float64)
        vy = np.sum((V[t][None, :] - Y) ** 2, axis=1)
        uK.append(np.mean(a2 * qr ** 2 / D * vy))
        uV.append(np.mean(a2 * float(rV[i].astype(np.float64) @ rV[i].astype(np.float64))))
    return np.array(uK), np.array(uV)


def _oracle_selector(lib_mod, K, Q, kappa):
    M, Z, _ = lib_mod.obs_head(K, np.zeros_like(K), Q)
    return lib_mod.selector_scores(K, Q, M, Z, kappa)


def _oracle_utilities(lib_mod, K, V, Q, toks, rK, rV):
    M, Z, Y = lib_mod.obs_head(K, V, Q)
    return lib_mod.utilities(K, V, Q, M, Z, Y, toks, rK, rV)


def _selector_pin(lib_mod, seed=0):
    K, V, Q = _problem(seed)
    for kappa in (1, 3, 7, 9):
        sc, pooled = _oracle_selector(lib_mod, K, Q, kappa)
        bsc, bpooled = _brute_selector(K, Q, kappa)
        np.testing.assert_allclose(sc, bsc, rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(pooled, bpooled, rtol=1e-12, atol=1e-15)


def _utility_pin(lib_mod, seed=1):
    K, V, Q = _problem(seed)
    S, D = K.shape
    W = Q.shape[1]
    rng = np.random.default_rng(seed + 100)
    toks = np.array([0, 5, 17, S - W - 1], np.int32)
    rK = rng.standard_normal((toks.size, D)).astype(np.float32)
    rV = rng.standard_normal((toks.size, D)).astype(np.float32)
    uK, uV = _oracle_utilities(lib_mod, K, V, Q, toks, rK, rV)
    bK, bV = _brute_utilities(K, V, Q, toks, rK, rV)
    np.testing.assert_allclose(uK, bK, rtol=1e-11)
    np.testing.assert_allclose(uV, bV, rtol=1e-11)


def test_selector_score_is_column_mean_of_causal_softmax_then_centred_pool():
    """App. A.2 Eq. selector-score at kappa = 1, 3, 7, 9 with g = 2, W = 3:
    both edges of the pool (zero padding, division by kappa) included."""
    _selector_pin(R)


def test_selector_pool_edges_by_hand():
    # A raw score of 1 at position 0 only: the kappa = 7 pool spreads 1/7 over
    # positions 0..3 (centred window, zero padding, no renormalisation).
    sc = np.zeros(12)
    sc[0] = 1.0
    pooled = np.convolve(sc, np.ones(7) / 7, "same")
    np.testing.assert_allclose(pooled[:4], 1 / 7)
    assert np.all(pooled[4:] == 0)


def test_utilities_sum_every_observation_row():
    """Sec. 3.3 Eq. utilities with m = g W = 6 rows, each with its own causal
    softmax and its own y_w, against the brute force."""
    _utility_pin(R)


def test_utilities_single_row_reduce_to_the_two_channel_terms():
    # m = 1: u^K = alpha^2 (q.r)^2 / D ||v - y||^2 and u^V = alpha^2 ||r_V||^2.
    K, V, Q = _problem(3, g=1, W=1)
    D = K.shape[1]
    toks = np.array([4], np.int32)
    rK = np.ones((1, D), np.float32)
    rV = np.full((1, D), 0.5, np.float32)
    uK, uV = _oracle_utilities(R, K, V, Q, toks, rK, rV)
    a = _causal_alpha(K, Q)[0]
    y = a @ V
    np.testing.assert_allclose(uK[0], a[4] ** 2 * (Q[0, 0].sum()) ** 2 / D * np.sum((V[4] - y) ** 2), rtol=1e-12)
    np.testing.assert_allclose(uV[0], a[4] ** 2 * 0.25 * D, rtol=1e-12)


# --------------------------------------------------------------------------- planted mistakes

MUTANTS = {
    # the pool window shifted by one position
    "offcentre_pool": ("int u = t + d;", "int u = t + d + 1;", _selector_pin),
    # the pool renormalised at the edges instead of divided by kappa
    "edge_renormalised_pool": ("pooled[t] = s / kappa;",
                               "pooled[t] = s / (double)(((t + half < P - 1) ? t + half : P - 1) - "
                               "((t - half > 0) ? t - half : 0) + 1);", _selector_pin),
    # raw score summed, not averaged, over the rows
    "score_not_averaged": ("sc[t] = s / m;", "sc[t] = s;", _selector_pin),
    # utilities from the first observation row only
    "single_row_utilities": ("for (int w = 0; w < m; ++w) {\n      double a = obs_alpha",
                             "for (int w = 0; w < 1; ++w) {\n      double a = obs_alpha", _utility_pin),
    # observation rows read as if stored offset-major (w = i*g + jj)
    "row_mapping": ("int i = w % W;\n    int last = S - W + i;", "int i = w / g;\n    int last = S - W + i;",
                    _utility_pin),
    # alpha instead of alpha^2 in the key utility
    "alpha_not_squared": ("double a2 = a * a;", "double a2 = a;", _utility_pin),
}


class _Mutant:
    """The oracle's Python wrapper bound to a mutated build of its source."""

    def __init__(self, so_path):
        L = ctypes.CDLL(so_path)
        R._declare(L)
        self._L = L

    def __getattr__(self, name):
        fn = getattr(R, name)

        def call(*a, **k):
            saved = R._lib
            R._lib = self._L
            try:
                return fn(*a, **k)
            finally:
                R._lib = saved
        return call


@pytest.mark.parametrize("name", list(MUTANTS))
def test_pins_catch_planted_oracle_mistakes(name, tmp_path):
    old, new, pin = MUTANTS[name]
    src = open(ORACLE_SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    mutated = src.replace(old, new)
    c = tmp_path / "mut.c"
    c.write_text(mutated)
    so = tmp_path / "libmut.so"
    subprocess.check_call(["gcc", "-O1", "-ffp-contract=off", "-fPIC", "-shared", "-o", str(so), str(c), "-lm"])
    pin(R)  # the real oracle passes
    with pytest.raises(AssertionError):
        pin(_Mutant(str(so)))
