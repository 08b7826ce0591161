"""ctypes wrapper of the AnchorKV CPU oracle (``oracle/akvref.c``).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, by the smoke check and by the
benchmark's CPU-baseline leg.  The product library never imports it.

Every function takes numpy arrays.  Floating-point inputs are passed as float64
holding values that are exactly representable in the cache dtype (fp32 or
bf16), so the conversion is exact.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "akvref.c")
_LIB = os.path.join(_HERE, "libakvref.so")

SCALE_ABSMAX_OUTER, SCALE_ABSMAX_LITERAL, SCALE_RMS, SCALE_NAIVE = 0, 1, 2, 3
RANK_UTILITY, RANK_COSINE, RANK_RESNORM, RANK_ATTENTION, RANK_RANDOM = 0, 1, 2, 3, 4
BUDGET_FRACTION, BUDGET_THETA, BUDGET_COUNT = 0, 1, 2


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (fp64, no contraction, OpenMP)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
                               "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        _lib = ctypes.CDLL(build())
        _declare(_lib)
    return _lib


_d = ctypes.POINTER(ctypes.c_double)
_f = ctypes.POINTER(ctypes.c_float)
_i = ctypes.POINTER(ctypes.c_int)
_u8 = ctypes.POINTER(ctypes.c_uint8)
_i64 = ctypes.POINTER(ctypes.c_int64)
_c_int, _c_u64, _c_i64, _c_dbl, _c_flt = ctypes.c_int, ctypes.c_uint64, ctypes.c_int64, ctypes.c_double, ctypes.c_float


def _declare(L):
    L.akvref_splitmix64.restype = _c_u64
    L.akvref_splitmix64.argtypes = [_c_u64]
    L.akvref_hadamard_signs.argtypes = [_c_u64, _c_int, _f]
    L.akvref_fwht.argtypes = [_f, _c_int]
    L.akvref_codec_encode.argtypes = [_f, _c_int, _c_int, _c_int, _c_u64, _u8, _f]
    L.akvref_codec_decode.argtypes = [_u8, _f, _c_int, _c_int, _c_u64, _c_int, _f]
    L.akvref_base_bytes.restype = _c_dbl
    L.akvref_base_bytes.argtypes = [_c_int] * 7
    L.akvref_theta_budget.restype = _c_i64
    L.akvref_theta_budget.argtypes = [_c_int] * 8 + [_c_dbl]
    L.akvref_obs_head.argtypes = [_d, _d, _d, _c_int, _c_int, _c_int, _c_int, _d, _d, _d]
    L.akvref_selector_scores.argtypes = [_d, _d, _d, _d, _c_int, _c_int, _c_int, _c_int, _c_int, _d, _d]
    L.akvref_n_top.restype = _c_int
    L.akvref_n_top.argtypes = [_c_int, _c_int, _c_flt]
    L.akvref_select_anchors.argtypes = [_d, _c_int, _c_int, _c_int, _c_flt, _c_u64, _c_int, _i]
    L.akvref_assign_tokens.argtypes = [_d, _c_int, _c_int, _i, _c_int, _c_int, _i, _c_int, _i, _d, _f]
    L.akvref_assign_vectors.argtypes = [_d, _c_int, _d, _c_int, _c_int, _c_int, _i, _d]
    L.akvref_utilities.argtypes = [_d, _d, _d, _d, _d, _d, _c_int, _c_int, _c_int, _c_int,
                                   _i, _c_int, _f, _f, _d, _d]
    L.akvref_budget_select.restype = _c_i64
    L.akvref_budget_select.argtypes = [_d, _c_int, _c_int, _c_i64, _u8]
    L.akvref_budget_select_per_head.restype = _c_i64
    L.akvref_budget_select_per_head.argtypes = [_d, _c_int, _c_int, _c_i64, _u8]
    L.akvref_rank_key.restype = _c_dbl
    L.akvref_rank_key.argtypes = [_c_int, _c_int, _c_int, _c_int, _d, _d, _c_int, _f, _c_dbl, _c_u64]
    L.akvref_encode.restype = _c_int
    L.akvref_encode.argtypes = ([_c_int] * 6 + [_c_flt, _c_int, _c_int, _c_u64, _c_int, _c_dbl, _c_i64,
                                                _c_int, _c_int, _c_int, _c_int, _d, _d, _d, _i, _i, _i, _d, _i, _d,
                                                _d, _d, _u8, _u8, _u8, _f, _u8, _f, _d, _i64])
    L.akvref_reconstruct.argtypes = [_d, _c_int, _c_int, _c_int, _c_u64, _c_int, _i, _c_int, _i, _d, _u8, _u8, _f,
                                     _f]
    L.akvref_attention.argtypes = [_f, _f, _c_int, _c_int, _c_int, _d, _c_int, _c_dbl, _d]
    L.akvref_attention_rope.argtypes = [_f, _f, _c_int, _c_int, _c_int, _d, _c_int, _c_dbl, _f, _d]
    L.akvref_rope_table.argtypes = [_f, _c_int, _c_int, _f]
    L.akvref_rope_rotate.argtypes = [_f, _d, _c_int, _d]
    L.akvref_rope_keys.argtypes = [_d, _c_int, _c_int, _f, _c_int, _d]
    L.akvref_utilities_rope.argtypes = [_d, _d, _d, _d, _d, _d, _c_int, _c_int, _c_int, _c_int,
                                        _i, _c_int, _f, _f, _f, _d, _d]
    L.akvref_encode_rope.restype = _c_int
    L.akvref_encode_rope.argtypes = ([_c_int] * 6 + [_c_flt, _c_int, _c_int, _c_u64, _c_int, _c_dbl, _c_i64,
                                                     _c_int, _c_int, _c_int, _c_int, _d, _d, _d, _i, _f, _i, _i,
                                                     _d, _i, _d, _d, _d, _u8, _u8, _u8, _f, _u8, _f, _d, _i64])
    L.akvref_num_threads.restype = _c_int
    L.akvref_set_threads.argtypes = [_c_int]


def _p(a, t):
    return a.ctypes.data_as(t)


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


# ----------------------------------------------------------------------------- primitives

def splitmix64(x: int) -> int:
    return int(lib().akvref_splitmix64(x))


def hadamard_signs(seed: int, D: int) -> np.ndarray:
    s = np.empty(D, np.float32)
    lib().akvref_hadamard_signs(seed, D, _p(s, _f))
    return s


def fwht(z) -> np.ndarray:
    z = _f32(z).copy()
    lib().akvref_fwht(_p(z, _f), z.shape[-1])
    return z


def codec_encode(r, G: int, mode: int, seed: int):
    r = _f32(r)
    D = r.shape[-1]
    codes = np.zeros(D // 4, np.uint8)
    scales = np.zeros(D // G, np.float32)
    lib().akvref_codec_encode(_p(r, _f), D, G, mode, seed, _p(codes, _u8), _p(scales, _f))
    return codes, scales


def codec_decode(codes, scales, D: int, G: int, seed: int, mode: int = SCALE_ABSMAX_OUTER) -> np.ndarray:
    codes = np.ascontiguousarray(codes, np.uint8)
    scales = _f32(scales)
    rt = np.empty(D, np.float32)
    lib().akvref_codec_decode(_p(codes, _u8), _p(scales, _f), D, G, seed, mode, _p(rt, _f))
    return rt


def base_bytes(S, H, D, W, k, elem_bytes=2, b_gamma=2) -> float:
    return float(lib().akvref_base_bytes(S, H, D, W, k, elem_bytes, b_gamma))


def theta_budget(S, H, D, W, k, G, theta, elem_bytes=2, b_gamma=2) -> int:
    return int(lib().akvref_theta_budget(S, H, D, W, k, G, elem_bytes, b_gamma, theta))


def rope_table(inv_freq, D: int, npos: int) -> np.ndarray:
    """fp32 cosines and sines [npos][D/2][2] of the rotation R_t (rotate-half pairs)."""
    inv_freq = _f32(inv_freq)
    cs = np.empty((npos, D // 2, 2), np.float32)
    lib().akvref_rope_table(_p(inv_freq, _f), D, npos, _p(cs, _f))
    return cs


def rope_rotate(cs_t, x) -> np.ndarray:
    """R_t x in fp64 for one position (cs_t: [D/2][2])."""
    cs_t, x = _f32(cs_t), _f64(x)
    out = np.empty_like(x)
    lib().akvref_rope_rotate(_p(cs_t, _f), _p(x, _d), x.shape[-1], _p(out, _d))
    return out


def rope_keys(Kh, cs, bf16: bool) -> np.ndarray:
    """Rotated keys of one head [S][D], rounded to the cache dtype."""
    Kh, cs = _f64(Kh), _f32(cs)
    S, D = Kh.shape
    out = np.empty((S, D))
    lib().akvref_rope_keys(_p(Kh, _d), S, D, _p(cs, _f), int(bf16), _p(out, _d))
    return out


def n_top(k, W, rho) -> int:
    return int(lib().akvref_n_top(k, W, rho))


# ----------------------------------------------------------------------------- per-head steps

def obs_head(Kh, Vh, Qg):
    """Observation-window attention of one KV head; Qg is [g][W][D]."""
    Kh, Vh, Qg = _f64(Kh), _f64(Vh), _f64(Qg)
    S, D = Kh.shape
    g, W, _ = Qg.shape
    m = g * W
    M, Z, Y = np.empty(m), np.empty(m), np.empty((m, D))
    lib().akvref_obs_head(_p(Kh, _d), _p(Vh, _d), _p(Qg, _d), S, D, W, g, _p(M, _d), _p(Z, _d), _p(Y, _d))
    return M, Z, Y


def selector_scores(Kh, Qg, M, Z, kappa):
    Kh, Qg, M, Z = _f64(Kh), _f64(Qg), _f64(M), _f64(Z)
    S, D = Kh.shape
    g, W, _ = Qg.shape
    P = S - W
    sc, pooled = np.empty(max(P, 1)), np.empty(max(P, 1))
    lib().akvref_selector_scores(_p(Kh, _d), _p(Qg, _d), _p(M, _d), _p(Z, _d), S, D, W, g, kappa,
                                 _p(sc, _d), _p(pooled, _d))
    return sc[:P], pooled[:P]


def select_anchors(pooled, S, W, k, rho, seed, h) -> np.ndarray:
    pooled = _f64(pooled)
    anchors = np.empty(k, np.int32)
    lib().akvref_select_anchors(_p(pooled, _d), S, W, k, rho, seed, h, _p(anchors, _i))
    return anchors


def assign_tokens(X, anchors, bf16: bool, toks=None, want_residual=True):
    X = _f64(X)
    S, D = X.shape
    anchors = _i32(anchors)
    toks = np.arange(S, dtype=np.int32) if toks is None else _i32(toks)
    n = toks.shape[0]
    a = np.empty(n, np.int32)
    g = np.empty(n, np.float64)
    r = np.empty((n, D), np.float32) if want_residual else None
    lib().akvref_assign_tokens(_p(X, _d), S, D, _p(anchors, _i), anchors.shape[0], int(bf16), _p(toks, _i), n,
                               _p(a, _i), _p(g, _d), _p(r, _f) if r is not None else None)
    return a, g, r


def assign_vectors(xs, A, bf16: bool):
    xs, A = _f64(xs), _f64(A)
    n, D = xs.shape
    a = np.empty(n, np.int32)
    g = np.empty(n, np.float64)
    lib().akvref_assign_vectors(_p(xs, _d), n, _p(A, _d), A.shape[0], D, int(bf16), _p(a, _i), _p(g, _d))
    return a, g


def utilities(Kh, Vh, Qg, M, Z, Y, toks, rK, rV, cs=None):
    """Eq. utilities; with a rotation table cs, Kh are the rotated keys and
    u^K uses R_t r^K_t."""
    Kh, Vh, Qg, M, Z, Y = map(_f64, (Kh, Vh, Qg, M, Z, Y))
    S, D = Kh.shape
    g, W, _ = Qg.shape
    toks = _i32(toks)
    rK, rV = _f32(rK), _f32(rV)
    n = toks.shape[0]
    uK, uV = np.empty(n), np.empty(n)
    if cs is None:
        lib().akvref_utilities(_p(Kh, _d), _p(Vh, _d), _p(Qg, _d), _p(M, _d), _p(Z, _d), _p(Y, _d), S, D, W, g,
                               _p(toks, _i), n, _p(rK, _f), _p(rV, _f), _p(uK, _d), _p(uV, _d))
    else:
        cs = _f32(cs)
        lib().akvref_utilities_rope(_p(Kh, _d), _p(Vh, _d), _p(Qg, _d), _p(M, _d), _p(Z, _d), _p(Y, _d), S, D, W,
                                    g, _p(toks, _i), n, _p(rK, _f), _p(rV, _f), _p(cs, _f), _p(uK, _d),
                                    _p(uV, _d))
    return uK, uV


def budget_select(u, N, per_head=False):
    u = _f64(u)
    H, S = u.shape
    sel = np.zeros((H, S), np.uint8)
    fn = lib().akvref_budget_select_per_head if per_head else lib().akvref_budget_select
    n = fn(_p(u, _d), H, S, N, _p(sel, _u8))
    return sel, int(n)


# ----------------------------------------------------------------------------- whole request

def encode(K, V, Qobs, *, W, k, rho=0.7, kappa=7, bf16=True, seed=0, budget_mode=BUDGET_FRACTION,
           budget=0.05, budget_count=0, G=None, scale_mode=SCALE_ABSMAX_OUTER, anchor_override=None,
           rank_mode=RANK_UTILITY, head_budget=0, inv_freq=None):
    """Algorithm 1 for one request.  K, V: [H][S][D]; Qobs: [Hq][W][D].  With
    inv_freq ([D/2] rotation frequencies) K holds the unrotated keys and the
    pass encodes positions as the paper does (Sec. 3.2)."""
    K, V, Qobs = _f64(K), _f64(V), _f64(Qobs)
    H, S, D = K.shape
    Hq = Qobs.shape[0]
    G = D if G is None else G
    out = dict(
        anchors=np.empty((H, k), np.int32), aK=np.empty((H, S), np.int32), gK=np.empty((H, S)),
        aV=np.empty((H, S), np.int32), gV=np.empty((H, S)), uK=np.empty((H, S)), uV=np.empty((H, S)),
        selK=np.empty((H, S), np.uint8), selV=np.empty((H, S), np.uint8),
        codesK=np.empty((H, S, D // 4), np.uint8), scalesK=np.empty((H, S, D // G), np.float32),
        codesV=np.empty((H, S, D // 4), np.uint8), scalesV=np.empty((H, S, D // G), np.float32),
        pooled=np.zeros((H, max(S - W, 1))), nsel=np.zeros(2, np.int64))
    ov = None if anchor_override is None else _i32(anchor_override)
    head = (H, Hq, D, S, W, k, rho, kappa, int(bf16), seed, budget_mode, budget, budget_count, G, scale_mode,
            rank_mode, int(head_budget), _p(K, _d), _p(V, _d), _p(Qobs, _d),
            _p(ov, _i) if ov is not None else None)
    if inv_freq is None:
        fn = lib().akvref_encode
    else:
        invf = _f32(inv_freq)
        head = head + (_p(invf, _f),)
        fn = lib().akvref_encode_rope
    rc = fn(
        *head, _p(out["anchors"], _i), _p(out["aK"], _i), _p(out["gK"], _d), _p(out["aV"], _i), _p(out["gV"], _d),
        _p(out["uK"], _d), _p(out["uV"], _d), _p(out["selK"], _u8), _p(out["selV"], _u8),
        _p(out["codesK"], _u8), _p(out["scalesK"], _f), _p(out["codesV"], _u8), _p(out["scalesV"], _f),
        _p(out["pooled"], _d), _p(out["nsel"], _i64))
    if rc != 0:
        raise ValueError("oracle rejected the configuration")
    out["pooled"] = out["pooled"][:, : S - W]
    out["scale_mode"] = scale_mode
    return out


def reconstruct(X, enc, side: str, G, seed):
    """Dense fp32 reconstruction [H][S][D] of side 'K' or 'V' from oracle outputs."""
    X = _f64(X)
    H, S, D = X.shape
    k = enc["anchors"].shape[1]
    out = np.empty((H, S, D), np.float32)
    for h in range(H):
        Xh = np.ascontiguousarray(X[h])
        anc = _i32(enc["anchors"][h])
        a = _i32(enc["a" + side][h])
        g = _f64(enc["g" + side][h])
        sel = np.ascontiguousarray(enc["sel" + side][h], np.uint8)
        codes = np.ascontiguousarray(enc["codes" + side][h], np.uint8)
        scales = _f32(enc["scales" + side][h])
        o = np.empty((S, D), np.float32)
        lib().akvref_reconstruct(_p(Xh, _d), S, D, G, seed, int(enc.get("scale_mode", 0)), _p(anc, _i), k,
                                 _p(a, _i), _p(g, _d), _p(sel, _u8), _p(codes, _u8), _p(scales, _f), _p(o, _f))
        out[h] = o
    return out


def attention(Kt, Vt, q, scale=None, cs=None):
    """Softmax attention in fp64 over dense entries Kt, Vt [H][T][D]; q [Hq][D].
    With a rotation table cs ([>= T][D/2][2]) entry t sits at position t and
    its key is rotated by R_t."""
    Kt, Vt, q = _f32(Kt), _f32(Vt), _f64(q)
    H, T, D = Kt.shape
    Hq = q.shape[0]
    scale = 1.0 / np.sqrt(D) if scale is None else float(scale)
    out = np.empty((Hq, D))
    if cs is None:
        lib().akvref_attention(_p(Kt, _f), _p(Vt, _f), H, T, D, _p(q, _d), Hq, scale, _p(out, _d))
    else:
        cs = _f32(cs)
        assert cs.shape[0] >= T
        lib().akvref_attention_rope(_p(Kt, _f), _p(Vt, _f), H, T, D, _p(q, _d), Hq, scale, _p(cs, _f), _p(out, _d))
    return out


def num_threads() -> int:
    return int(lib().akvref_num_threads())


def set_threads(n: int) -> None:
    """Threads of the oracle's parallel loops (timing only)."""
    lib().akvref_set_threads(int(n))
