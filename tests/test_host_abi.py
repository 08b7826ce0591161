"""Host-side checks of the C ABI: the library loads, exports every entry
point the header declares, validates arguments before touching the GPU, and
its plan arithmetic (anchor counts, score/random split, residual budgets)
agrees with the paper's formulas as the oracle computes them.  No GPU."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

import paper_2608_02901_amd as akv
from paper_2608_02901_amd import _native as N
from oracle import akvref as R

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _lib_or_skip():
    if not os.path.exists(N.LIB_PATH):
        pytest.skip("library not built")
    return N.lib()


def _header_functions():
    with open(os.path.join(ROOT, "include", "anchorkv.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(anchorkv_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_entry_point():
    L = _lib_or_skip()
    declared = _header_functions()
    assert len(declared) >= 13
    for name in declared:
        assert hasattr(L, name), name
    assert sorted(N.EXPORTED) == declared


def _cfg(**kw):
    base = dict(num_kv_heads=8, num_q_heads=32, head_dim=128, window=32, anchor_frac=0.02, rho=0.7, kappa=7,
                budget=0.05, dtype=N.BF16)
    base.update(kw)
    return N.Config.make(**base)


@pytest.mark.parametrize("kw,status", [
    (dict(num_q_heads=30), N.ERR_INVALID_ARG),
    (dict(num_q_heads=24), N.ERR_UNSUPPORTED),       # g = 3
    (dict(head_dim=96), N.ERR_INVALID_ARG),
    (dict(head_dim=64), N.ERR_UNSUPPORTED),
    (dict(kappa=6), N.ERR_INVALID_ARG),
    (dict(kappa=257), N.ERR_INVALID_ARG),
    (dict(quant_group=48), N.ERR_INVALID_ARG),
    (dict(quant_group=16), N.ERR_UNSUPPORTED),
    (dict(rho=1.5), N.ERR_INVALID_ARG),
    (dict(budget=-0.1), N.ERR_INVALID_ARG),
    (dict(anchor_frac=0.0), N.ERR_INVALID_ARG),
    (dict(anchor_count=20000, anchor_frac=0.0, seq=32768), N.ERR_UNSUPPORTED),
    (dict(anchor_count=16, anchor_frac=0.0), N.ERR_INVALID_ARG),  # k < W
    (dict(window=64, num_q_heads=64), N.ERR_UNSUPPORTED),         # m = 512
    (dict(dtype=7), N.ERR_INVALID_ARG),
])
def test_plan_rejects_bad_configs(kw, status):
    _lib_or_skip()
    kw = dict(kw)
    seq = kw.pop("seq", 4096)
    with pytest.raises(N.AnchorKVError) as e:
        N.Plan(_cfg(**kw), [seq])
    assert e.value.status == status
    assert N.last_error()


def test_plan_rejects_bad_batches():
    _lib_or_skip()
    for lens in ([], [32], [4096] * 65):
        with pytest.raises(N.AnchorKVError):
            N.Plan(_cfg(), lens)


@pytest.mark.parametrize("S", [4096, 32768, 131072, 7777])
def test_plan_counts_follow_the_paper(S):
    _lib_or_skip()
    p = N.Plan(_cfg(), [S])
    ri = p.requests[0]
    k = max(32, int(math.floor(np.float32(0.02) * S)))
    assert ri.anchors == k
    assert ri.n_top == R.n_top(k, 32, 0.7)
    assert ri.n_rand == k - 32 - ri.n_top
    n = int(math.floor(float(np.float32(0.05)) * 8 * S))
    assert ri.residuals_k == ri.residuals_v == min(n, 8 * (S - k))


def test_theta_budget_matches_worked_example_plan():
    _lib_or_skip()
    cfg = _cfg(anchor_count=256, anchor_frac=0.0, budget_mode=N.BUDGET_THETA, budget=0.05)
    p = N.Plan(cfg, [32768])
    ri = p.requests[0]
    theta = float(np.float32(0.05))
    n = R.theta_budget(32768, 8, 128, 32, 256, 128, theta)
    assert ri.residuals_k == n // 2 and ri.residuals_v == n - n // 2
    assert abs(n - 91056) <= 1  # fp32 rounding of theta may move the floor by one


def test_budget_caps_at_candidate_count():
    _lib_or_skip()
    p = N.Plan(_cfg(budget_mode=N.BUDGET_COUNT, budget_count=10 ** 9), [1000])
    ri = p.requests[0]
    assert ri.residuals_k == 8 * (1000 - ri.anchors)


def test_buffer_sizes_grow_with_batch():
    _lib_or_skip()
    p1 = N.Plan(_cfg(), [8192])
    p2 = N.Plan(_cfg(), [8192, 8192])
    assert p2.cache_bytes > p1.cache_bytes and p2.encode_ws_bytes > p1.encode_ws_bytes
    assert p1.cache_bytes < 8 * 8192 * 128 * 2 * 2 / 5  # well under the dense layer


def test_entry_points_validate_before_touching_the_gpu():
    L = _lib_or_skip()
    p = N.Plan(_cfg(max_append=4), [4096])
    assert L.anchorkv_encode(p.handle, None, None, None, None, None, None, None) == N.ERR_INVALID_ARG
    assert L.anchorkv_append(p.handle, 1, 4, 1, 1, 1, None) == N.ERR_CAPACITY
    assert L.anchorkv_append(p.handle, 1, -1, 1, 1, 1, None) == N.ERR_INVALID_ARG
    assert L.anchorkv_append(p.handle, 1, 0, 1, 1, None, None) == N.ERR_INVALID_ARG
    assert L.anchorkv_decode_step(p.handle, 1, 4, 1, 1, 1, 1, 0, 0.0, 1, None) == N.ERR_CAPACITY
    assert L.anchorkv_decode_step(p.handle, 1, 0, 1, 1, 1, 1, 7, 0.0, 1, None) == N.ERR_INVALID_ARG
    assert L.anchorkv_decode_step(p.handle, 1, 0, 1, 1, None, 1, 0, 0.0, 1, None) == N.ERR_INVALID_ARG
    assert L.anchorkv_decode_attn(p.handle, 1, 5, 1, 1, 0, 0.0, 1, None) == N.ERR_INVALID_ARG
    assert L.anchorkv_decode_attn(p.handle, 1, 0, 1, 1, 9, 0.0, 1, None) == N.ERR_INVALID_ARG
    assert L.anchorkv_reconstruct(p.handle, 1, 0, 3, 0, 1, None) == N.ERR_INVALID_ARG
    assert L.anchorkv_reconstruct(p.handle, 1, 0, 0, 2, 1, None) == N.ERR_INVALID_ARG
    assert L.anchorkv_status_string(N.ERR_HIP).decode() == "HIP runtime error"


def test_export_rejects_a_foreign_blob():
    _lib_or_skip()
    p = N.Plan(_cfg(), [4096])
    junk = np.zeros(p.cache_bytes, np.uint8)
    with pytest.raises(N.AnchorKVError) as e:
        N.export(p, junk, 0)
    assert e.value.status == N.ERR_CORRUPT_CACHE
