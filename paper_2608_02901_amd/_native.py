"""ctypes binding of libanchorkv.so (the C ABI in include/anchorkv.h).

Argument marshalling only: tensors are passed as raw device pointers and the
caller's current HIP stream; every step of the compression and of decode
attention runs in the library's kernels.  Importing this module never builds
anything; when the library is missing the calls raise.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "lib", "libanchorkv.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_CAPACITY, ERR_CORRUPT_CACHE, ERR_HIP, ERR_BUFFER_TOO_SMALL = range(7)
F32, BF16 = 0, 1
SCALE_ABSMAX_OUTER, SCALE_ABSMAX_LITERAL, SCALE_RMS, SCALE_NAIVE = 0, 1, 2, 3
RANK_UTILITY, RANK_COSINE, RANK_RESNORM, RANK_ATTENTION, RANK_RANDOM = 0, 1, 2, 3, 4
APPEND_ENCODED, APPEND_DENSE = 0, 1
BUDGET_FRACTION, BUDGET_THETA, BUDGET_COUNT = 0, 1, 2

EXPORTED = ["anchorkv_plan_create", "anchorkv_plan_destroy", "anchorkv_cache_bytes", "anchorkv_encode_workspace_bytes",
            "anchorkv_decode_workspace_bytes", "anchorkv_plan_request", "anchorkv_encode", "anchorkv_append",
            "anchorkv_decode_attn", "anchorkv_decode_step", "anchorkv_decode_step_noalloc", "anchorkv_reconstruct",
            "anchorkv_export", "anchorkv_profile_enable", "anchorkv_profile_read", "anchorkv_profile_disable",
            "anchorkv_status_string", "anchorkv_last_error"]


class AnchorKVError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"anchorkv status {status}: {msg}")
        self.status = status


class Config(ctypes.Structure):
    _fields_ = [("num_kv_heads", ctypes.c_int32), ("num_q_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("window", ctypes.c_int32), ("anchor_count", ctypes.c_int32), ("anchor_frac", ctypes.c_float),
                ("rho", ctypes.c_float), ("kappa", ctypes.c_int32), ("budget_mode", ctypes.c_int32),
                ("budget", ctypes.c_float), ("budget_count", ctypes.c_int64), ("quant_group", ctypes.c_int32),
                ("scale_mode", ctypes.c_int32), ("dtype", ctypes.c_int32), ("max_append", ctypes.c_int32),
                ("rank_mode", ctypes.c_int32), ("head_budget", ctypes.c_int32), ("append_mode", ctypes.c_int32),
                ("seed", ctypes.c_uint64), ("rope", ctypes.c_int32), ("rope_inv_freq", ctypes.c_float * 64)]

    @classmethod
    def make(cls, *, num_kv_heads, num_q_heads, head_dim=128, window=32, anchor_count=0, anchor_frac=0.0,
             rho=0.7, kappa=7, budget_mode=BUDGET_FRACTION, budget=0.05, budget_count=0, quant_group=0,
             scale_mode=SCALE_ABSMAX_OUTER, dtype=BF16, max_append=0, rank_mode=RANK_UTILITY, head_budget=0,
             append_mode=APPEND_ENCODED, seed=0, rope_inv_freq=None):
        """rope_inv_freq: None (keys used as given) or the D/2 rotary
        frequencies; then K and k_new are the keys before the rotation."""
        freqs = (ctypes.c_float * 64)()
        if rope_inv_freq is not None:
            vals = [float(v) for v in rope_inv_freq]
            if len(vals) != head_dim // 2:
                raise ValueError("rope_inv_freq needs head_dim / 2 values")
            for i, v in enumerate(vals):
                freqs[i] = v
        return cls(num_kv_heads, num_q_heads, head_dim, window, anchor_count, anchor_frac, rho, kappa, budget_mode,
                   budget, budget_count, quant_group, scale_mode, dtype, max_append, rank_mode, head_budget,
                   append_mode, seed, 1 if rope_inv_freq is not None else 0, freqs)


class RequestInfo(ctypes.Structure):
    _fields_ = [("seq_len", ctypes.c_int32), ("anchors", ctypes.c_int32), ("n_top", ctypes.c_int32),
                ("n_rand", ctypes.c_int32), ("residuals_k", ctypes.c_int64), ("residuals_v", ctypes.c_int64)]


class ExportArrays(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("anchors", "a_k", "gamma_k", "sel_k", "codes_k", "scales_k", "a_v", "gamma_v", "sel_v", "codes_v",
                 "scales_v", "tail_a_k", "tail_gamma_k", "tail_a_v", "tail_gamma_v", "stats")]


_lib = None


def lib():
    """Loads libanchorkv.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"AnchorKV HIP library not built ({LIB_PATH}); run python -m paper_2608_02901_amd.build")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
        L.anchorkv_plan_create.restype = i32
        L.anchorkv_plan_create.argtypes = [ctypes.POINTER(Config), i32, ctypes.POINTER(i32), ctypes.POINTER(vp)]
        L.anchorkv_plan_destroy.argtypes = [vp]
        for n in ("anchorkv_cache_bytes", "anchorkv_encode_workspace_bytes", "anchorkv_decode_workspace_bytes"):
            getattr(L, n).restype = ctypes.c_size_t
            getattr(L, n).argtypes = [vp]
        L.anchorkv_plan_request.restype = i32
        L.anchorkv_plan_request.argtypes = [vp, i32, ctypes.POINTER(RequestInfo)]
        sz = ctypes.c_size_t
        L.anchorkv_encode.restype = i32
        L.anchorkv_encode.argtypes = [vp, vp, vp, sz, vp, sz, vp, sz, vp, sz, vp, sz, vp]
        L.anchorkv_append.restype = i32
        L.anchorkv_append.argtypes = [vp, vp, sz, i32, vp, vp, sz, vp, sz, vp]
        L.anchorkv_decode_attn.restype = i32
        L.anchorkv_decode_attn.argtypes = [vp, vp, sz, i32, vp, sz, vp, sz, i32, f32, vp, sz, vp]
        L.anchorkv_decode_step.restype = i32
        L.anchorkv_decode_step.argtypes = [vp, vp, sz, i32, vp, vp, sz, vp, sz, vp, sz, i32, f32, vp, sz, vp]
        L.anchorkv_decode_step_noalloc.restype = i32
        L.anchorkv_decode_step_noalloc.argtypes = [vp, vp, sz, i32, vp, vp, sz, vp, sz, vp, sz, i32, f32, vp]
        L.anchorkv_reconstruct.restype = i32
        L.anchorkv_reconstruct.argtypes = [vp, vp, sz, i32, i32, i32, vp, sz, vp]
        L.anchorkv_export.restype = i32
        L.anchorkv_export.argtypes = [vp, vp, sz, i32, i32, ctypes.POINTER(ExportArrays)]
        L.anchorkv_profile_enable.restype = i32
        L.anchorkv_profile_enable.argtypes = [ctypes.c_char_p, i32]
        L.anchorkv_profile_read.restype = i32
        L.anchorkv_profile_read.argtypes = [ctypes.c_char_p, ctypes.POINTER(f32), ctypes.POINTER(i32)]
        L.anchorkv_profile_disable.restype = i32
        L.anchorkv_profile_disable.argtypes = []
        L.anchorkv_status_string.restype = ctypes.c_char_p
        L.anchorkv_status_string.argtypes = [i32]
        L.anchorkv_last_error.restype = ctypes.c_char_p
        L.anchorkv_last_error.argtypes = []
        _lib = L
    return _lib


def last_error() -> str:
    return lib().anchorkv_last_error().decode()


def check(status: int):
    if status != OK:
        raise AnchorKVError(status, last_error())


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    return t.data_ptr()


def _nbytes(t) -> int:
    return 0 if t is None else t.numel() * t.element_size()


def _dev(t, what, dtype=None, shape=None):
    """Checks that a tensor handed to a device entry point lives on the GPU,
    is contiguous and, when given, has the dtype and shape the plan implies
    (the library also checks the byte sizes)."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{what} must be a GPU tensor (got {t.device})")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{what} must be {dtype} (got {t.dtype})")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{what} must have shape {tuple(shape)} (got {tuple(t.shape)})")
    return t


def _tdtype(code):
    import torch
    return torch.float32 if code == F32 else torch.bfloat16


def _stream(stream) -> Optional[int]:
    if stream is not None:
        return int(stream)
    import torch
    return torch.cuda.current_stream().cuda_stream


class Plan:
    """Host plan of one layer's compression for a batch of sequence lengths."""

    def __init__(self, cfg: Config, seq_lens: Sequence[int]):
        self.cfg = cfg
        self.seq_lens = [int(s) for s in seq_lens]
        arr = (ctypes.c_int32 * len(self.seq_lens))(*self.seq_lens)
        h = ctypes.c_void_p()
        check(lib().anchorkv_plan_create(ctypes.byref(cfg), len(self.seq_lens), arr, ctypes.byref(h)))
        self._h = h
        L = lib()
        self.cache_bytes = int(L.anchorkv_cache_bytes(h))
        self.encode_ws_bytes = int(L.anchorkv_encode_workspace_bytes(h))
        self.decode_ws_bytes = int(L.anchorkv_decode_workspace_bytes(h))
        self.requests: List[RequestInfo] = []
        for b in range(len(self.seq_lens)):
            ri = RequestInfo()
            check(L.anchorkv_plan_request(h, b, ctypes.byref(ri)))
            self.requests.append(ri)

    @property
    def handle(self):
        return self._h

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and _lib is not None:
            _lib.anchorkv_plan_destroy(h)
            self._h = None

    def alloc(self, device="cuda"):
        """Allocates (cache, encode workspace, decode workspace) as uint8 tensors."""
        import torch
        return (torch.empty(self.cache_bytes, dtype=torch.uint8, device=device),
                torch.empty(self.encode_ws_bytes, dtype=torch.uint8, device=device),
                torch.empty(self.decode_ws_bytes, dtype=torch.uint8, device=device))


def _packed(x):
    import torch
    if isinstance(x, (list, tuple)):
        return torch.cat([t.reshape(-1) for t in x]).contiguous()
    return x.contiguous()


def encode(plan: Plan, K, V, Qobs, cache, workspace, anchor_override=None, stream=None):
    import torch
    K, V, Qobs = _packed(K), _packed(V), _packed(Qobs)
    ov = None if anchor_override is None else _packed(anchor_override)
    dt = _tdtype(plan.cfg.dtype)
    for t, n in ((K, "K"), (V, "V"), (Qobs, "Q_obs")):
        _dev(t, n, dt)
    _dev(ov, "anchor_override", torch.int32)
    _dev(cache, "cache", torch.uint8)
    _dev(workspace, "workspace", torch.uint8)
    if _nbytes(K) != _nbytes(V):
        raise ValueError("K and V must have the same size")
    check(lib().anchorkv_encode(plan.handle, _ptr(K), _ptr(V), _nbytes(K), _ptr(Qobs), _nbytes(Qobs), _ptr(ov),
                                _nbytes(ov), _ptr(cache), _nbytes(cache), _ptr(workspace), _nbytes(workspace),
                                _stream(stream)))
    return K, V, Qobs, ov  # keep packed copies alive until the stream has consumed them


def _new_shape(plan):
    return (len(plan.seq_lens), plan.cfg.num_kv_heads, plan.cfg.head_dim)


def _q_shape(plan):
    return (len(plan.seq_lens), plan.cfg.num_q_heads, plan.cfg.head_dim)


def append(plan: Plan, cache, n_appended: int, k_new, v_new, workspace, stream=None):
    import torch
    k_new, v_new = k_new.contiguous(), v_new.contiguous()
    dt = _tdtype(plan.cfg.dtype)
    _dev(k_new, "k_new", dt, _new_shape(plan))
    _dev(v_new, "v_new", dt, _new_shape(plan))
    _dev(cache, "cache", torch.uint8)
    _dev(workspace, "workspace", torch.uint8)
    check(lib().anchorkv_append(plan.handle, _ptr(cache), _nbytes(cache), n_appended, _ptr(k_new), _ptr(v_new),
                                _nbytes(k_new), _ptr(workspace), _nbytes(workspace), _stream(stream)))
    return k_new, v_new


def decode_step(plan: Plan, cache, n_appended: int, k_new, v_new, q, out, workspace, out_dtype: Optional[int] = None,
                softmax_scale: float = 0.0, stream=None):
    import torch
    k_new, v_new, q = k_new.contiguous(), v_new.contiguous(), q.contiguous()
    if out_dtype is None:
        out_dtype = F32 if out.dtype == torch.float32 else BF16
    dt = _tdtype(plan.cfg.dtype)
    _dev(k_new, "k_new", dt, _new_shape(plan))
    _dev(v_new, "v_new", dt, _new_shape(plan))
    _dev(q, "q", dt, _q_shape(plan))
    _dev(out, "out", _tdtype(out_dtype), _q_shape(plan))
    _dev(cache, "cache", torch.uint8)
    _dev(workspace, "workspace", torch.uint8)
    check(lib().anchorkv_decode_step(plan.handle, _ptr(cache), _nbytes(cache), n_appended, _ptr(k_new), _ptr(v_new),
                                     _nbytes(k_new), _ptr(q), _nbytes(q), _ptr(out), _nbytes(out), out_dtype,
                                     softmax_scale, _ptr(workspace), _nbytes(workspace), _stream(stream)))
    return out


def decode_step_noalloc(plan: Plan, cache, n_appended: int, k_new, v_new, q, out, out_dtype: Optional[int] = None,
                        softmax_scale: float = 0.0, stream=None):
    """decode_step with the library's static per-GPU scratch instead of a
    caller workspace (the entry point allocates nothing)."""
    import torch
    k_new, v_new, q = k_new.contiguous(), v_new.contiguous(), q.contiguous()
    if out_dtype is None:
        out_dtype = F32 if out.dtype == torch.float32 else BF16
    dt = _tdtype(plan.cfg.dtype)
    _dev(k_new, "k_new", dt, _new_shape(plan))
    _dev(v_new, "v_new", dt, _new_shape(plan))
    _dev(q, "q", dt, _q_shape(plan))
    _dev(out, "out", _tdtype(out_dtype), _q_shape(plan))
    _dev(cache, "cache", torch.uint8)
    check(lib().anchorkv_decode_step_noalloc(plan.handle, _ptr(cache), _nbytes(cache), n_appended, _ptr(k_new),
                                             _ptr(v_new), _nbytes(k_new), _ptr(q), _nbytes(q), _ptr(out),
                                             _nbytes(out), out_dtype, softmax_scale, _stream(stream)))
    return out


def decode_attn(plan: Plan, cache, q, out, workspace, n_appended: int = 0, out_dtype: Optional[int] = None,
                softmax_scale: float = 0.0, stream=None):
    import torch
    q = q.contiguous()
    if out_dtype is None:
        out_dtype = F32 if out.dtype == torch.float32 else BF16
    _dev(q, "q", _tdtype(plan.cfg.dtype), _q_shape(plan))
    _dev(out, "out", _tdtype(out_dtype), _q_shape(plan))
    _dev(cache, "cache", torch.uint8)
    _dev(workspace, "workspace", torch.uint8)
    check(lib().anchorkv_decode_attn(plan.handle, _ptr(cache), _nbytes(cache), n_appended, _ptr(q), _nbytes(q),
                                     _ptr(out), _nbytes(out), out_dtype, softmax_scale, _ptr(workspace),
                                     _nbytes(workspace), _stream(stream)))
    return out


def reconstruct(plan: Plan, cache, request: int, side: int, n_appended: int = 0, out=None, stream=None):
    import torch
    H, D = plan.cfg.num_kv_heads, plan.cfg.head_dim
    rows = plan.seq_lens[request] + n_appended
    if out is None:
        out = torch.empty(H, rows, D, dtype=torch.float32, device=cache.device)
    _dev(out, "out", torch.float32, (H, rows, D))
    _dev(cache, "cache", torch.uint8)
    check(lib().anchorkv_reconstruct(plan.handle, _ptr(cache), _nbytes(cache), n_appended, request, side, _ptr(out),
                                     _nbytes(out), _stream(stream)))
    return out


class KernelTimer:
    """Times every launch of the named library kernels with HIP events
    recorded on each kernel's own stream (anchorkv_profile_*)."""

    def __init__(self, kernels, max_launches: int = 4096):
        self.kernels = [kernels] if isinstance(kernels, str) else list(kernels)
        check(lib().anchorkv_profile_enable(",".join(self.kernels).encode(), max_launches))

    def read(self, kernel: str):
        """(summed milliseconds, number of timed launches) of one kernel."""
        ms = ctypes.c_float()
        n = ctypes.c_int32()
        check(lib().anchorkv_profile_read(kernel.encode(), ctypes.byref(ms), ctypes.byref(n)))
        return float(ms.value), int(n.value)

    def close(self):
        check(lib().anchorkv_profile_disable())


def export(plan: Plan, cache_host: np.ndarray, request: int, n_appended: int = 0) -> dict:
    """Logical content of one request in position order, from a host copy."""
    cfg = plan.cfg
    H, D = cfg.num_kv_heads, cfg.head_dim
    G = cfg.quant_group or D
    ri = plan.requests[request]
    S, k = ri.seq_len, ri.anchors
    out = dict(
        anchors=np.zeros((H, k), np.int32), a_k=np.zeros((H, S), np.int32), gamma_k=np.zeros((H, S), np.float32),
        sel_k=np.zeros((H, S), np.uint8), codes_k=np.zeros((H, S, D // 4), np.uint8),
        scales_k=np.zeros((H, S, D // G), np.float32), a_v=np.zeros((H, S), np.int32),
        gamma_v=np.zeros((H, S), np.float32), sel_v=np.zeros((H, S), np.uint8),
        codes_v=np.zeros((H, S, D // 4), np.uint8), scales_v=np.zeros((H, S, D // G), np.float32),
        tail_a_k=np.zeros((H, max(n_appended, 1)), np.int32), tail_gamma_k=np.zeros((H, max(n_appended, 1)), np.float32),
        tail_a_v=np.zeros((H, max(n_appended, 1)), np.int32), tail_gamma_v=np.zeros((H, max(n_appended, 1)), np.float32),
        stats=np.zeros(6, np.int64))
    ea = ExportArrays(*[out[n].ctypes.data for n, _ in ExportArrays._fields_])
    host = np.ascontiguousarray(cache_host, dtype=np.uint8)
    check(lib().anchorkv_export(plan.handle, host.ctypes.data, host.nbytes, request, n_appended, ctypes.byref(ea)))
    for n in ("tail_a_k", "tail_gamma_k", "tail_a_v", "tail_gamma_v"):
        out[n] = out[n][:, :n_appended]
    return out
