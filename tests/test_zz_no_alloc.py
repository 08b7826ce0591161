"""The no-allocation decode step (anchorkv_decode_step_noalloc, the library's
static per-GPU scratch instead of a caller workspace) against
anchorkv_decode_step: two calls in a row through the C ABI, the second with a
smaller input, each giving the same attention output and the same appended
tail records as the workspace entry point on a copy of the same cache."""
import numpy as np
import pytest
import torch

import paper_2608_02901_amd as akv
import synth
from paper_2608_02901_amd import _native as N
from parity_util import gpu_encode, make_cfg

pytestmark = pytest.mark.gpu


def _one(wl, steps):
    print(f"[noalloc] {wl.name} lens={wl.seq_lens} steps={steps}", flush=True)
    layer = synth.make_layer(wl, steps=steps)
    cfg = make_cfg(wl, max_append=steps)
    plan = N.Plan(cfg, wl.seq_lens)
    assert plan.decode_ws_bytes <= 32 << 20
    cache_a, ws, dws = gpu_encode(plan, layer)
    cache_b = cache_a.clone()
    out_a = torch.empty(wl.batch, wl.Hq, wl.D, dtype=torch.float32, device="cuda")
    out_b = torch.empty_like(out_a)
    for s in range(steps):
        kn, vn, q = layer.k_new[s].cuda(), layer.v_new[s].cuda(), layer.q[s].cuda()
        akv.decode_step(plan, cache_a, s, kn, vn, q, out_a, dws)
        akv.decode_step_noalloc(plan, cache_b, s, kn, vn, q, out_b)
        torch.cuda.synchronize()
        assert torch.equal(out_a, out_b), (s, float((out_a - out_b).abs().max()))
    assert torch.equal(cache_a, cache_b)
    return plan


def test_noalloc_decode_step_matches_workspace_entry_point_twice():
    big = synth.Workload("noalloc-big", H=2, Hq=8, D=128, seq_lens=[6000, 3100], dtype="bf16", anchor_frac=0.03,
                         budget=0.05, n_centers=48, steps=3, append=True, seed=71)
    small = synth.Workload("noalloc-small", H=2, Hq=8, D=128, seq_lens=[1500], dtype="bf16", anchor_frac=0.03,
                           budget=0.05, n_centers=48, steps=2, append=True, seed=72)
    pb = _one(big, 3)
    ps = _one(small, 2)
    assert ps.decode_ws_bytes < pb.decode_ws_bytes and ps.cache_bytes < pb.cache_bytes

