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
    (dict(scale_mode=4), N.ERR_INVALID_ARG),
    (dict(rank_mode=5), N.ERR_INVALID_ARG),
    (dict(rank_mode=-1), N.ERR_INVALID_ARG),
    (dict(head_budget=2), N.ERR_INVALID_ARG),
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


def test_equal_per_head_budgets_in_the_plan():
    """Equal per-head budgets (Sec. 4.3 ablation): every head gets floor(N / H)
    of the pooled count, so the request holds H * floor(N / H) per side; the
    per-(request, head) budget lists are limited to 64."""
    _lib_or_skip()
    pooled = N.Plan(_cfg(), [5000]).requests[0]
    per = N.Plan(_cfg(head_budget=1), [5000]).requests[0]
    assert per.residuals_k == pooled.residuals_k // 8 * 8 and per.residuals_v == pooled.residuals_v // 8 * 8
    N.Plan(_cfg(head_budget=1), [4096] * 8)  # 64 lists
    with pytest.raises(N.AnchorKVError) as e:
        N.Plan(_cfg(head_budget=1), [4096] * 9)
    assert e.value.status == N.ERR_UNSUPPORTED
    for mode in (N.RANK_COSINE, N.RANK_RESNORM, N.RANK_ATTENTION, N.RANK_RANDOM):
        assert N.Plan(_cfg(rank_mode=mode), [5000]).requests[0].residuals_k == pooled.residuals_k


def test_dense_tail_cache_bytes():
    """DENSE append mode (App. E "Generated Tokens"): the exact tail costs
    2 * H * D * element bytes per appended token and request on top of the
    same compressed prefix."""
    _lib_or_skip()
    lens, cap = [900, 1700], 5
    enc = N.Plan(_cfg(max_append=cap), lens)
    dense = N.Plan(_cfg(max_append=cap, append_mode=N.APPEND_DENSE), lens)
    extra = dense.cache_bytes - enc.cache_bytes
    need = len(lens) * 2 * 8 * cap * 128 * 2
    assert need <= extra <= need + 2 * 256  # two more arrays, each 256-byte aligned
    with pytest.raises(N.AnchorKVError):
        N.Plan(_cfg(append_mode=2), lens)


def test_buffer_sizes_grow_with_batch():
    _lib_or_skip()
    p1 = N.Plan(_cfg(), [8192])
    p2 = N.Plan(_cfg(), [8192, 8192])
    assert p2.cache_bytes > p1.cache_bytes and p2.encode_ws_bytes > p1.encode_ws_bytes
    assert p1.cache_bytes < 8 * 8192 * 128 * 2 * 2 / 5  # well under the dense layer


def _sizes(p):
    """Bytes the plan needs for each device buffer of the 4096-token 8B plan."""
    esz = 2
    H, Hq, D, W = 8, 32, 128, 32
    S = sum(p.seq_lens)
    B = len(p.seq_lens)
    return dict(kv=H * S * D * esz, qobs=B * Hq * W * D * esz, new=B * H * D * esz, q=B * Hq * D * esz,
                out32=B * Hq * D * 4, cache=p.cache_bytes, ws=p.encode_ws_bytes, dws=p.decode_ws_bytes)


def test_entry_points_validate_before_touching_the_gpu():
    L = _lib_or_skip()
    p = N.Plan(_cfg(max_append=4), [4096])
    z = _sizes(p)
    assert L.anchorkv_encode(p.handle, None, None, 0, None, 0, None, 0, None, 0, None, 0, None) == N.ERR_INVALID_ARG
    assert L.anchorkv_append(p.handle, 1, z["cache"], 4, 1, 1, z["new"], 1, z["dws"], None) == N.ERR_CAPACITY
    assert L.anchorkv_append(p.handle, 1, z["cache"], -1, 1, 1, z["new"], 1, z["dws"], None) == N.ERR_INVALID_ARG
    assert L.anchorkv_append(p.handle, 1, z["cache"], 0, 1, 1, z["new"], None, z["dws"], None) == N.ERR_INVALID_ARG
    step = lambda n, od, ws: L.anchorkv_decode_step(p.handle, 1, z["cache"], n, 1, 1, z["new"], 1, z["q"], 1,
                                                   z["out32"], od, 0.0, ws, z["dws"], None)
    assert step(4, 0, 1) == N.ERR_CAPACITY
    assert step(0, 7, 1) == N.ERR_INVALID_ARG
    assert step(0, 0, None) == N.ERR_INVALID_ARG
    attn = lambda n, od: L.anchorkv_decode_attn(p.handle, 1, z["cache"], n, 1, z["q"], 1, z["out32"], od, 0.0, 1,
                                               z["dws"], None)
    assert attn(5, 0) == N.ERR_INVALID_ARG
    assert attn(0, 9) == N.ERR_INVALID_ARG
    rec_bytes = 8 * 4096 * 128 * 4
    assert L.anchorkv_reconstruct(p.handle, 1, z["cache"], 0, 3, 0, 1, rec_bytes, None) == N.ERR_INVALID_ARG
    assert L.anchorkv_reconstruct(p.handle, 1, z["cache"], 0, 0, 2, 1, rec_bytes, None) == N.ERR_INVALID_ARG
    assert L.anchorkv_status_string(N.ERR_HIP).decode() == "HIP runtime error"
    assert L.anchorkv_status_string(N.ERR_BUFFER_TOO_SMALL).decode() == "buffer too small"


def test_undersized_buffers_are_rejected_before_any_launch():
    """Each device buffer one byte short of what the plan needs returns
    ANCHORKV_ERR_BUFFER_TOO_SMALL and names the buffer (no GPU is touched:
    the checks come before anything is enqueued)."""
    L = _lib_or_skip()
    p = N.Plan(_cfg(max_append=4), [4096])
    z = _sizes(p)

    def enc(**kw):
        a = dict(kv=z["kv"], qobs=z["qobs"], ov=0, cache=z["cache"], ws=z["ws"], ovp=None)
        a.update(kw)
        return L.anchorkv_encode(p.handle, 1, 1, a["kv"], 1, a["qobs"], a["ovp"], a["ov"], 1, a["cache"], 1, a["ws"],
                                 None)

    cases = [
        (lambda: enc(kv=z["kv"] - 1), "K / V"),
        (lambda: enc(qobs=z["qobs"] - 1), "Q_obs"),
        (lambda: enc(ovp=1, ov=4 * 8 * p.requests[0].anchors - 1), "anchor override"),
        (lambda: enc(cache=z["cache"] - 1), "cache"),
        (lambda: enc(ws=z["ws"] - 1), "encode workspace"),
        (lambda: L.anchorkv_append(p.handle, 1, z["cache"], 0, 1, 1, z["new"] - 1, 1, z["dws"], None),
         "k_new / v_new"),
        (lambda: L.anchorkv_append(p.handle, 1, z["cache"], 0, 1, 1, z["new"], 1, z["dws"] - 1, None),
         "decode workspace"),
        (lambda: L.anchorkv_decode_attn(p.handle, 1, z["cache"] - 1, 0, 1, z["q"], 1, z["out32"], 0, 0.0, 1,
                                        z["dws"], None), "cache"),
        (lambda: L.anchorkv_decode_attn(p.handle, 1, z["cache"], 0, 1, z["q"] - 1, 1, z["out32"], 0, 0.0, 1,
                                        z["dws"], None), "q"),
        (lambda: L.anchorkv_decode_attn(p.handle, 1, z["cache"], 0, 1, z["q"], 1, z["out32"] - 1, 0, 0.0, 1,
                                        z["dws"], None), "out"),
        (lambda: L.anchorkv_decode_attn(p.handle, 1, z["cache"], 0, 1, z["q"], 1, z["out32"] // 2 - 1, 1, 0.0, 1,
                                        z["dws"], None), "out"),
        (lambda: L.anchorkv_decode_step(p.handle, 1, z["cache"], 0, 1, 1, z["new"], 1, z["q"], 1, z["out32"], 0,
                                        0.0, 1, z["dws"] - 1, None), "decode workspace"),
        (lambda: L.anchorkv_reconstruct(p.handle, 1, z["cache"], 2, 0, 0, 1, 8 * 4098 * 128 * 4 - 1, None), "out"),
    ]
    for call, what in cases:
        assert call() == N.ERR_BUFFER_TOO_SMALL, what
        assert N.last_error().startswith(what + ":"), (what, N.last_error())
    host = np.zeros(p.cache_bytes - 1, np.uint8)
    ea = N.ExportArrays()
    assert L.anchorkv_export(p.handle, host.ctypes.data, host.nbytes, 0, 0, ctypes.byref(ea)) == N.ERR_BUFFER_TOO_SMALL


def test_plan_rejects_offsets_beyond_int32():
    """64 requests of 2^22 tokens with 16384 anchors per head: the counting
    sort's per-chunk anchor tables would pass 2^31 entries; the plan refuses
    it instead of wrapping its int32 offsets."""
    _lib_or_skip()
    cfg = _cfg(num_kv_heads=1, num_q_heads=1, anchor_count=16384, anchor_frac=0.0)
    with pytest.raises(N.AnchorKVError) as e:
        N.Plan(cfg, [1 << 22] * 64)
    assert e.value.status in (N.ERR_UNSUPPORTED,)


def test_fault_injection_stops_the_call_before_its_first_kernel(monkeypatch):
    """ANCHORKV_FAULT_INJECT=k_init: the encode reaches its first kernel and
    enqueues nothing from there on (the pointers here are not device memory:
    a launch would be an error), returning ANCHORKV_ERR_HIP with the kernel
    named; without the variable the plan's validation still passes."""
    L = _lib_or_skip()
    p = N.Plan(_cfg(), [4096])
    z = _sizes(p)
    monkeypatch.setenv("ANCHORKV_FAULT_INJECT", "k_init")
    st = L.anchorkv_encode(p.handle, 8, 8, z["kv"], 8, z["qobs"], None, 0, 8, z["cache"], 8, z["ws"], None)
    assert st == N.ERR_HIP
    assert "fault injected at kernel k_init" in N.last_error()


def test_export_rejects_a_foreign_blob():
    _lib_or_skip()
    p = N.Plan(_cfg(), [4096])
    junk = np.zeros(p.cache_bytes, np.uint8)
    with pytest.raises(N.AnchorKVError) as e:
        N.export(p, junk, 0)
    assert e.value.status == N.ERR_CORRUPT_CACHE


def test_noalloc_decode_step_rejects_a_plan_beyond_its_static_scratch():
    """The no-allocation decode step serves plans whose decode workspace fits
    its 32 MiB static scratch; 64 ragged 8B requests need about 77 MiB and are
    refused before anything touches the GPU."""
    L = _lib_or_skip()
    import synth
    wl = synth.workload(5)
    plan = N.Plan(_cfg(max_append=1), wl.seq_lens * 4)
    assert plan.decode_ws_bytes > 32 << 20
    big = 1 << 30
    st = L.anchorkv_decode_step_noalloc(plan.handle, 1, plan.cache_bytes, 0, 1, 1, big, 1, big, 1, big, 0, 0.0, None)
    assert st == N.ERR_BUFFER_TOO_SMALL and "static decode scratch" in N.last_error()
