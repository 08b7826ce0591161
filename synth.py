"""Seeded synthetic inputs for AnchorKV workloads.

Shared by the tests, the benchmark and the smoke check; it holds none of the
method's arithmetic, only the input recipe: clustered keys and values shaped
like one attention layer of Llama-3.1-8B / 70B (the paper's models, whose
activations are not available here).

Recipe per KV head and side: ``n_centers`` centres drawn from N(0, I_D); every
token picks a centre uniformly and adds N(0, sigma^2 I_D) noise.  Keys get
``n_outlier`` distinct outlier channels per head, scaled by ``outlier_scale``
after sampling.  Observation queries (the last W positions' queries) and
decode queries are N(0, I_D).  Values are drawn in fp32 and rounded to the
cache dtype (round-to-nearest-even for bf16).  Generation uses a
``torch.Generator`` on the requested device, so big layers are generated in
place on the GPU; both implementations always receive the same tensors.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional

import torch


@dataclasses.dataclass
class Workload:
    name: str
    H: int                    # KV heads
    Hq: int                   # query heads
    D: int                    # head dim
    seq_lens: List[int]       # per request
    dtype: str                # "f32" | "bf16"
    anchor_count: int = 0     # fixed k when > 0
    anchor_frac: float = 0.0  # else k = floor(frac * S)
    budget: float = 0.05      # residual fraction per side: N_side = floor(budget * H * S)
    quant_group: int = 0      # 0 -> D
    n_centers: int = 512
    sigma: float = 0.3
    n_outlier: int = 4
    outlier_scale: float = 8.0
    window: int = 32
    steps: int = 1            # decode steps
    append: bool = False      # append one token per step (encoded against the anchors)
    seed: int = 0

    @property
    def batch(self) -> int:
        return len(self.seq_lens)

    @property
    def G(self) -> int:
        return self.quant_group or self.D

    def k_of(self, S: int) -> int:
        if self.anchor_count > 0:
            return min(self.anchor_count, S)
        return min(S, max(self.window, int(math.floor(self.anchor_frac * S))))

    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16


def ragged_lengths(n: int, lo: int, hi: int, seed: int) -> List[int]:
    g = torch.Generator().manual_seed(seed)
    return [int(x) for x in torch.randint(lo, hi + 1, (n,), generator=g)]


def workload(i: int, seq_scale: float = 1.0) -> Workload:
    """The five evaluation workloads (1-based).  ``seq_scale`` < 1 shrinks the
    sequence lengths (for tests that must finish on a CPU)."""
    def s(n):
        return max(64, int(n * seq_scale))

    if i == 1:
        return Workload("1head-4K-f32", H=1, Hq=1, D=128, seq_lens=[s(4096)], dtype="f32", anchor_count=128,
                        budget=0.05, quant_group=32, n_centers=64, n_outlier=0, seed=0)
    if i == 2:
        return Workload("llama8b-32K-bf16", H=8, Hq=32, D=128, seq_lens=[s(32768)], dtype="bf16",
                        anchor_frac=0.02, budget=0.05, n_centers=512, seed=1)
    if i == 3:
        return Workload("llama8b-128K-bf16-append64", H=8, Hq=32, D=128, seq_lens=[s(131072)], dtype="bf16",
                        anchor_frac=0.02, budget=0.05, n_centers=512, steps=64, append=True, seed=2)
    if i == 4:
        return Workload("llama70b-32K-bf16-b8", H=8, Hq=64, D=128, seq_lens=[s(32768)] * 8, dtype="bf16",
                        anchor_frac=0.015, budget=0.04, n_centers=1024, seed=3)
    if i == 5:
        lens = [s(x) for x in ragged_lengths(16, 4096, 131072, seed=4)]
        return Workload("llama8b-ragged16-bf16", H=8, Hq=32, D=128, seq_lens=lens, dtype="bf16",
                        anchor_frac=0.02, budget=0.05, n_centers=512, seed=4)
    raise ValueError(i)


def _gen(device, seed):
    return torch.Generator(device=device).manual_seed(int(seed))


@dataclasses.dataclass
class Layer:
    """One layer's inputs.  K, V: per request [H][S_b][D]; Qobs: per request
    [Hq][W][D]; q: [steps][batch][Hq][D]; k_new/v_new: [steps][batch][H][D]
    (appended tokens), all on ``device`` in the workload dtype."""
    K: List[torch.Tensor]
    V: List[torch.Tensor]
    Qobs: List[torch.Tensor]
    q: torch.Tensor
    k_new: Optional[torch.Tensor]
    v_new: Optional[torch.Tensor]


def make_layer(wl: Workload, device="cpu", seed: Optional[int] = None, steps: Optional[int] = None) -> Layer:
    seed = wl.seed if seed is None else seed
    steps = wl.steps if steps is None else steps
    gen = _gen(device, seed)
    dt = wl.torch_dtype()
    K, V, Q = [], [], []
    # Centres and outlier channels are per head; appended tokens reuse them.
    heads = []
    for b, S in enumerate(wl.seq_lens):
        kb = torch.empty(wl.H, S, wl.D, device=device, dtype=dt)
        vb = torch.empty(wl.H, S, wl.D, device=device, dtype=dt)
        hb = []
        for h in range(wl.H):
            ck = torch.randn(wl.n_centers, wl.D, generator=gen, device=device)
            cv = torch.randn(wl.n_centers, wl.D, generator=gen, device=device)
            ch = torch.randperm(wl.D, generator=gen, device=device)[:wl.n_outlier]
            pick = torch.randint(0, wl.n_centers, (S,), generator=gen, device=device)
            x = ck[pick] + wl.sigma * torch.randn(S, wl.D, generator=gen, device=device)
            if wl.n_outlier:
                x[:, ch] *= wl.outlier_scale
            kb[h] = x.to(dt)
            pick = torch.randint(0, wl.n_centers, (S,), generator=gen, device=device)
            kb_v = cv[pick] + wl.sigma * torch.randn(S, wl.D, generator=gen, device=device)
            vb[h] = kb_v.to(dt)
            hb.append((ck, cv, ch))
        K.append(kb)
        V.append(vb)
        Q.append(torch.randn(wl.Hq, wl.window, wl.D, generator=gen, device=device).to(dt))
        heads.append(hb)
    q = torch.randn(steps, wl.batch, wl.Hq, wl.D, generator=gen, device=device).to(dt)
    k_new = v_new = None
    if wl.append:
        k_new = torch.empty(steps, wl.batch, wl.H, wl.D, device=device, dtype=dt)
        v_new = torch.empty(steps, wl.batch, wl.H, wl.D, device=device, dtype=dt)
        for b in range(wl.batch):
            for h in range(wl.H):
                ck, cv, ch = heads[b][h]
                pick = torch.randint(0, wl.n_centers, (steps,), generator=gen, device=device)
                x = ck[pick] + wl.sigma * torch.randn(steps, wl.D, generator=gen, device=device)
                if wl.n_outlier:
                    x[:, ch] *= wl.outlier_scale
                k_new[:, b, h] = x.to(dt)
                pick = torch.randint(0, wl.n_centers, (steps,), generator=gen, device=device)
                v_new[:, b, h] = (cv[pick] + wl.sigma * torch.randn(steps, wl.D, generator=gen,
                                                                     device=device)).to(dt)
    return Layer(K, V, Q, q, k_new, v_new)


def focused_queries(wl: Workload, K: List[torch.Tensor], steps: int, n_focus: int = 8, tau: float = 0.4,
                    noise: float = 0.3, seed: int = 0):
    """Observation and decode queries that attend to a few tokens, as a model's
    queries attend to what the context is about: per request and KV head,
    n_focus positions before the window are drawn; every query row is
    tau * sqrt(D) * (a focus key / its norm) + N(0, noise^2 I), observation row
    (j, i) of query head j using focus (i + j) mod n_focus and decode step s
    focus (s + j) mod n_focus, so the window's queries foreshadow the decode
    queries.  Returns (Qobs per request [Hq][W][D], q [steps][batch][Hq][D]) in
    the workload dtype, on K's device."""
    device = K[0].device
    gen = _gen(device, seed)
    dt = wl.torch_dtype()
    g = wl.Hq // wl.H
    Qs = []
    q = torch.empty(steps, wl.batch, wl.Hq, wl.D, device=device, dtype=dt)
    for b, S in enumerate(wl.seq_lens):
        Qb = torch.empty(wl.Hq, wl.window, wl.D, device=device, dtype=dt)
        for h in range(wl.H):
            pos = torch.randint(0, S - wl.window, (n_focus,), generator=gen, device=device)
            f = K[b][h, pos].float()
            f = f / f.norm(dim=1, keepdim=True).clamp_min(1e-30) * (tau * math.sqrt(wl.D))
            for jj in range(g):
                j = h * g + jj
                rows = f[(torch.arange(wl.window, device=device) + jj) % n_focus]
                Qb[j] = (rows + noise * torch.randn(wl.window, wl.D, generator=gen, device=device)).to(dt)
                rows = f[(torch.arange(steps, device=device) + jj) % n_focus]
                q[:, b, j] = (rows + noise * torch.randn(steps, wl.D, generator=gen, device=device)).to(dt)
        Qs.append(Qb)
    return Qs, q


def llama31_inv_freq(D: int = 128, base: float = 500000.0, factor: float = 8.0, low_freq_factor: float = 1.0,
                     high_freq_factor: float = 4.0, original_context: int = 8192):
    """Rotary frequencies of Llama-3.1 (rope_theta 500000 with the model's
    long-context rescaling of the low frequencies), as fp32 numpy values
    [D/2].  This is the model's positional encoding, an input of the
    compression pass when keys are given before the rotation."""
    import numpy as np
    inv = 1.0 / (base ** (np.arange(0, D, 2, dtype=np.float64) / D))
    wavelen = 2.0 * math.pi / inv
    low_wl = original_context / low_freq_factor
    high_wl = original_context / high_freq_factor
    out = np.where(wavelen > low_wl, inv / factor, inv)
    smooth = (original_context / wavelen - low_freq_factor) / (high_freq_factor - low_freq_factor)
    smoothed = (1.0 - smooth) * out / factor + smooth * out
    medium = (wavelen >= high_wl) & (wavelen <= low_wl)
    out = np.where(medium, smoothed, out)
    return out.astype(np.float32)
