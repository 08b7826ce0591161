"""Pins of the oracle's positional-rotation path (Sec. 3.2: keys are projected
before RoPE, anchors are scored with the rotated keys, the stored keys are
rotated at decoding; Sec. 3.3 Eq. utilities with R_t; App. E
"Implementation").

The brute forces are numpy written from the definitions: the rotation of a
rotate-half pair as a complex multiplication, softmax attention over
explicitly rotated keys, the utilities with explicitly rotated residuals.
Special cases tie the new path to the pinned one: zero frequencies make R_t
the identity, so the rotated compression pass must equal the plain one bit
for bit.  Planted mistakes in a private copy of the oracle (rotation sign,
unrotated observation keys, unrotated key residuals, shifted positions) must
fail these pins.  No GPU.
"""
import ctypes
import math
import os
import subprocess

import numpy as np
import pytest
import scipy.special

import synth
from oracle import akvref as R

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE_SRC = os.path.join(ROOT, "oracle", "akvref.c")


def _bf16(x):
    x = np.asarray(x, np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def _np_rotate(cs_t, x):
    """R_t x as the complex product (x_f + i x_{f+F}) (c_f + i s_f)."""
    F = x.shape[-1] // 2
    z = x[..., :F] + 1j * x[..., F:]
    w = cs_t[..., 0].astype(np.float64) + 1j * cs_t[..., 1].astype(np.float64)
    p = z * w
    return np.concatenate([p.real, p.imag], axis=-1)


def _freqs(D=8, base=10.0):
    return (1.0 / base ** (np.arange(0, D, 2) / D)).astype(np.float32)


# --------------------------------------------------------------------------- rotation itself

def _table_pin(lib_mod):
    inv = synth.llama31_inv_freq(128)
    pos = np.array([0, 1, 2, 17, 4095, 32767, 131071, 131135])
    cs = lib_mod.rope_table(inv, 128, int(pos.max()) + 1)[pos]
    ang = pos[:, None].astype(np.float64) * inv[None, :].astype(np.float64)
    want = np.stack([np.cos(ang), np.sin(ang)], axis=-1).astype(np.float32)
    # fp32 roundings of the fp64 cos and sin: libm and numpy agree to within
    # one fp32 unit in the last place (almost always exactly)
    ulp = np.spacing(np.abs(want))
    assert np.all(np.abs(cs - want) <= ulp)
    assert np.mean(cs == want) > 0.999


def _rotate_pin(lib_mod):
    rng = np.random.default_rng(5)
    D = 16
    cs = lib_mod.rope_table(_freqs(D), D, 40)
    for t in (0, 1, 7, 39):
        x = _bf16(rng.standard_normal(D) * 3)
        got = lib_mod.rope_rotate(cs[t], x)
        np.testing.assert_allclose(got, _np_rotate(cs[t], x), rtol=0, atol=1e-15)


def test_rope_table_is_fp32_cos_sin_of_position_times_frequency():
    """Llama-3.1 frequencies at prompt and generation positions up to 128K."""
    _table_pin(R)


def test_rope_rotation_is_complex_multiplication_of_rotate_half_pairs():
    _rotate_pin(R)


def test_rope_rotation_by_hand():
    # Unit vectors of pair 0 at t = 1 with inv_freq[0] = 1 turn by one radian:
    # e_0 -> (cos 1) e_0 + (sin 1) e_F and e_F -> -(sin 1) e_0 + (cos 1) e_F,
    # the convention of rotate_half: x * cos + rotate_half(x) * sin.
    D, F = 8, 4
    inv = np.array([1.0, 0.5, 0.25, 0.125], np.float32)
    cs = R.rope_table(inv, D, 2)
    c1, s1 = np.float32(math.cos(1.0)), np.float32(math.sin(1.0))
    e0 = np.zeros(D); e0[0] = 1.0
    eF = np.zeros(D); eF[F] = 1.0
    np.testing.assert_array_equal(R.rope_rotate(cs[1], e0), [c1, 0, 0, 0, s1, 0, 0, 0])
    np.testing.assert_array_equal(R.rope_rotate(cs[1], eF), [-s1, 0, 0, 0, c1, 0, 0, 0])
    # position 0 is the identity
    x = np.arange(D, dtype=np.float64)
    np.testing.assert_array_equal(R.rope_rotate(cs[0], x), x)


def test_rope_preserves_norms_and_depends_on_relative_position():
    rng = np.random.default_rng(9)
    D = 128
    inv = synth.llama31_inv_freq(D)
    cs = R.rope_table(inv, D, 3000)
    for s, t in ((5, 17), (100, 2999), (2000, 2001)):
        q = _bf16(rng.standard_normal(D))
        k = _bf16(rng.standard_normal(D))
        rq, rk = R.rope_rotate(cs[s], q), R.rope_rotate(cs[t], k)
        np.testing.assert_allclose(np.linalg.norm(rk), np.linalg.norm(k), rtol=2e-7)
        # (R_s q).(R_t k) = q.(R_{t-s} k): the rotation encodes the offset
        # (up to the fp32 rounding of the table entries)
        np.testing.assert_allclose(rq @ rk, q @ R.rope_rotate(cs[t - s], k), rtol=0, atol=2e-5 * D)


def test_rope_keys_are_the_rotation_rounded_to_the_cache_dtype():
    rng = np.random.default_rng(2)
    S, D = 30, 16
    K = _bf16(rng.standard_normal((S, D)) * 2)
    cs = R.rope_table(_freqs(D, 100.0), D, S)
    for bf16 in (False, True):
        got = R.rope_keys(K, cs, bf16)
        want = _np_rotate(cs, K).astype(np.float32)
        want = _bf16(want) if bf16 else want.astype(np.float64)
        np.testing.assert_array_equal(got, want)


# --------------------------------------------------------------------------- the compression pass

def _problem(seed, H=2, S=96, D=16, W=4, g=2):
    rng = np.random.default_rng(seed)
    K = _bf16(rng.standard_normal((H, S, D)) * 1.5)
    V = _bf16(rng.standard_normal((H, S, D)))
    Q = _bf16(rng.standard_normal((H * g, W, D)) * 0.8)
    return K, V, Q


def _causal_alpha(K, Q):
    S, D = K.shape
    g, W, _ = Q.shape
    A = np.zeros((g * W, S))
    for jj in range(g):
        for i in range(W):
            last = S - W + i
            A[jj * W + i, : last + 1] = scipy.special.softmax(K[: last + 1] @ Q[jj, i] / math.sqrt(D))
    return A


def _selector_rope_pin(lib_mod):
    """The selector scores of the rotated pass are the column means of the
    causal softmax over the RoPE-rotated (bf16-rounded) keys, then pooled."""
    K, V, Q = _problem(4)
    H, S, D = K.shape
    W, g = Q.shape[1], Q.shape[0] // H
    inv = _freqs(D, 50.0)
    cs = lib_mod.rope_table(inv, D, S)
    enc = lib_mod.encode(K, V, Q, W=W, k=24, kappa=3, seed=3, inv_freq=inv)
    for h in range(H):
        Kr = _bf16(_np_rotate(cs, K[h]).astype(np.float32))
        A = _causal_alpha(Kr, Q[h * g:(h + 1) * g])
        sc = A[:, : S - W].mean(axis=0)
        pooled = np.convolve(sc, np.ones(3) / 3, "same")
        np.testing.assert_allclose(enc["pooled"][h], pooled, rtol=1e-11, atol=1e-15)


def _utilities_rope_pin(lib_mod):
    """u^K with R_t r^K_t (Sec. 3.3 Eq. utilities) and alpha, y_w from the
    rotated keys, against numpy; u^V is unchanged by the rotation."""
    K, V, Q = _problem(6, H=1, S=41, D=8, W=3, g=2)
    Kh, Vh = K[0], V[0]
    S, D = Kh.shape
    inv = _freqs(D, 10.0)
    cs = lib_mod.rope_table(inv, D, S)
    Kr = lib_mod.rope_keys(Kh, cs, True)
    rng = np.random.default_rng(60)
    toks = np.array([0, 5, 17, 36], np.int32)
    rK = rng.standard_normal((toks.size, D)).astype(np.float32)
    rV = rng.standard_normal((toks.size, D)).astype(np.float32)
    M, Z, Y = lib_mod.obs_head(Kr, Vh, Q)
    uK, uV = lib_mod.utilities(Kr, Vh, Q, M, Z, Y, toks, rK, rV, cs=cs)
    A = _causal_alpha(_bf16(_np_rotate(cs, Kh).astype(np.float32)), Q)
    Yb = A @ Vh
    Qr = Q.reshape(-1, D)
    for i, t in enumerate(toks):
        a2 = A[:, t] ** 2
        qr = Qr @ _np_rotate(cs[t], rK[i].astype(np.float64))
        vy = np.sum((Vh[t][None, :] - Yb) ** 2, axis=1)
        np.testing.assert_allclose(uK[i], np.mean(a2 * qr ** 2 / D * vy), rtol=1e-10)
        np.testing.assert_allclose(uV[i], np.mean(a2 * float(rV[i].astype(np.float64) @ rV[i])), rtol=1e-10)


def _attention_rope_pin(lib_mod):
    rng = np.random.default_rng(8)
    H, T, D, Hq = 2, 50, 16, 4
    Kt = rng.standard_normal((H, T, D)).astype(np.float32)
    Vt = rng.standard_normal((H, T, D)).astype(np.float32)
    q = rng.standard_normal((Hq, D))
    cs = lib_mod.rope_table(_freqs(D, 30.0), D, T)
    out = lib_mod.attention(Kt, Vt, q, cs=cs)
    for j in range(Hq):
        h = j // (Hq // H)
        Kr = _np_rotate(cs, Kt[h].astype(np.float64))
        p = scipy.special.softmax(Kr @ q[j] / math.sqrt(D))
        np.testing.assert_allclose(out[j], p @ Vt[h].astype(np.float64), rtol=1e-10, atol=1e-13)


def test_rotated_pass_scores_anchors_with_rotated_keys():
    _selector_rope_pin(R)


def test_rotated_utilities_against_numpy():
    _utilities_rope_pin(R)


def test_rotated_attention_against_numpy():
    _attention_rope_pin(R)


def test_zero_frequencies_reduce_to_the_unrotated_pass():
    """inv_freq = 0 makes every R_t the identity: the rotated compression pass
    and attention equal the plain ones bit for bit."""
    K, V, Q = _problem(11)
    H, S, D = K.shape
    kw = dict(W=Q.shape[1], k=20, kappa=7, seed=5, budget=0.1)
    a = R.encode(K, V, Q, **kw)
    b = R.encode(K, V, Q, inv_freq=np.zeros(D // 2, np.float32), **kw)
    for key in ("anchors", "aK", "gK", "aV", "gV", "uK", "uV", "selK", "selV", "codesK", "scalesK", "codesV",
                "scalesV", "pooled", "nsel"):
        np.testing.assert_array_equal(a[key], b[key], err_msg=key)
    cs = R.rope_table(np.zeros(D // 2, np.float32), D, S)
    Kt = R.reconstruct(K, a, "K", D, 5)
    Vt = R.reconstruct(V, a, "V", D, 5)
    q = np.random.default_rng(1).standard_normal((Q.shape[0], D))
    np.testing.assert_array_equal(R.attention(Kt, Vt, q), R.attention(Kt, Vt, q, cs=cs))


def test_rotation_changes_the_selection_but_not_the_projection():
    """With real frequencies the anchors follow the rotated keys while the
    stored representation is that of the unrotated keys: an anchor override
    makes the assignment, coefficients and residual codes independent of the
    rotation, while the selector scores (and, in general, the utilities)
    change."""
    K, V, Q = _problem(12)
    H, S, D = K.shape
    inv = _freqs(D, 20.0)
    anc = np.stack([np.sort(np.r_[np.arange(0, 60, 4)[:16], np.arange(S - 4, S)]) for _ in range(H)])
    kw = dict(W=Q.shape[1], k=anc.shape[1], kappa=7, seed=5, budget=1.0, anchor_override=anc)
    a = R.encode(K, V, Q, **kw)
    b = R.encode(K, V, Q, inv_freq=inv, **kw)
    for key in ("aK", "gK", "aV", "gV", "selK", "codesK", "scalesK", "codesV", "scalesV"):
        np.testing.assert_array_equal(a[key], b[key], err_msg=key)
    assert not np.array_equal(a["uK"], b["uK"])
    c = R.encode(K, V, Q, W=Q.shape[1], k=24, kappa=7, seed=5, inv_freq=inv)
    d = R.encode(K, V, Q, W=Q.shape[1], k=24, kappa=7, seed=5)
    assert not np.array_equal(c["pooled"], d["pooled"])


def test_all_anchor_cache_with_rope_equals_dense_rotated_attention():
    """k = S stores every key exactly (unrotated); decode attention with the
    keys rotated at their positions equals dense attention over the rotated
    keys (Sec. 3.2: R_t distributes over the decomposition)."""
    K, V, Q = _problem(13, S=40)
    H, S, D = K.shape
    inv = _freqs(D, 10.0)
    enc = R.encode(K, V, Q, W=Q.shape[1], k=S, seed=1, inv_freq=inv)
    Kt = R.reconstruct(K, enc, "K", D, 1)
    Vt = R.reconstruct(V, enc, "V", D, 1)
    np.testing.assert_array_equal(Kt, K.astype(np.float32))
    cs = R.rope_table(inv, D, S)
    q = np.random.default_rng(3).standard_normal((Q.shape[0], D))
    got = R.attention(Kt, Vt, q, cs=cs)
    g = Q.shape[0] // H
    for j in range(Q.shape[0]):
        Kr = _np_rotate(cs, K[j // g])
        p = scipy.special.softmax(Kr @ q[j] / math.sqrt(D))
        np.testing.assert_allclose(got[j], p @ V[j // g], rtol=1e-10, atol=1e-13)


def test_decomposed_rotated_logits_equal_rotated_reconstruction():
    """q . R_t x^_t = gamma_t (q . R_t abar_a(t)) + q . R_t r~_t: the anchor
    term and the residual term rotate separately (what a decode kernel that
    never rebuilds the dense key computes)."""
    K, V, Q = _problem(14, H=1, S=64)
    H, S, D = K.shape
    inv = _freqs(D, 10.0)
    enc = R.encode(K, V, Q, W=Q.shape[1], k=12, seed=2, budget=0.3, inv_freq=inv)
    cs = R.rope_table(inv, D, S)
    Kt = R.reconstruct(K, enc, "K", D, 2)[0].astype(np.float64)
    q = np.random.default_rng(4).standard_normal(D)
    anc = enc["anchors"][0]
    for t in range(S):
        a = enc["aK"][0, t]
        gm = enc["gK"][0, t]
        abar = K[0, anc[a]]
        rt = Kt[t] - (np.float32(gm) * abar.astype(np.float32)).astype(np.float64)
        lhs = q @ R.rope_rotate(cs[t], Kt[t])
        rhs = gm * (q @ _np_rotate(cs[t], abar)) + q @ _np_rotate(cs[t], rt)
        np.testing.assert_allclose(lhs, rhs, rtol=1e-9, atol=1e-9)


# --------------------------------------------------------------------------- planted mistakes

MUTANTS = {
    # the rotation turned the other way (R_{-t})
    "rotation_sign": ("out[f] = c * a - s * b;\n    out[f + F] = s * a + c * b;",
                      "out[f] = c * a + s * b;\n    out[f + F] = -s * a + c * b;", _rotate_pin),
    # anchors scored with the unrotated keys
    "unrotated_observation": ("Ko = Krot;", "Ko = Kh;", _selector_rope_pin),
    # u^K without R_t on the key residual
    "unrotated_key_residual": ("if (cs) {\n      akvref_rope_rotate(cs + (size_t)t * D, rk, D, dv);",
                               "if (0) {\n      akvref_rope_rotate(cs + (size_t)t * D, rk, D, dv);",
                               _utilities_rope_pin),
    # decode keys rotated at the mirrored positions
    "shifted_positions": ("akvref_rope_rotate(cs + (size_t)t * D, kk, D, kr);",
                          "akvref_rope_rotate(cs + (size_t)(T - 1 - t) * D, kk, D, kr);", _attention_rope_pin),
    # frequencies halved in the table
    "table_frequency": ("double ang = (double)t * (double)inv_freq[f];",
                        "double ang = (double)t * (double)inv_freq[f] * 0.5;", _table_pin),
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
def test_rope_pins_catch_planted_oracle_mistakes(name, tmp_path):
    old, new, pin = MUTANTS[name]
    src = open(ORACLE_SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    c = tmp_path / "mut.c"
    c.write_text(src.replace(old, new))
    so = tmp_path / "libmut.so"
    subprocess.check_call(["gcc", "-O1", "-ffp-contract=off", "-fPIC", "-shared", "-o", str(so), str(c), "-lm"])
    pin(R)
    with pytest.raises(AssertionError):
        pin(_Mutant(str(so)))
