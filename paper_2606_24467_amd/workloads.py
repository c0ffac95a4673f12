"""Seeded synthetic inputs for the CompressKV eviction path.

This module builds inputs only: it holds none of the method's arithmetic and
imports nothing else from this package, so the fp64 oracle and the HIP path
can both be fed from it.

The five workloads mirror the shapes the paper evaluates (section 4: Llama-3.1
8B and Qwen2.5 GQA models, contexts up to 128K, per-layer budgets 128-2048,
needle-in-a-haystack retrieval) with random data:

  tiny     1 layer,  batch 1, 8 q / 2 kv heads, D=64,  L=1024,   W=16, fp32
  llama1   1 layer,  batch 1, 32 q / 8 kv heads, D=128, L=32768, W=32, bf16
  llama32  32 layers of llama1's shape, Dirichlet per-layer budgets, 1-3 SRHs
  qwen128k 28 layers, 28 q / 4 kv heads, D=128, L=131072, W=64, bf16
  ragged8  32 layers, batch 8, lengths U[4096, 16384], 32 q / 8 kv, W=32, bf16
  paper    the paper's own setting (section 4) on llama32's shape: W=8, max
           pooling 5, the top 4 SRHs of each layer (any groups; groups
           without one are allowed), the layer-shared index set, Dirichlet
           per-layer budgets of 512 on average within [32, 3 x 512]

Recipe (per layer and sequence):
  * Q window, K and V are N(0, 1), drawn in fp32 and rounded to bf16
    (round to nearest even) for the bf16 workloads;
  * SRH mask: n_g heads of each group chosen without replacement (paper:
    4 heads of the layer chosen without replacement);
  * sinks: positions 0 .. n_sink-1 hold 3*sqrt(D) times the unit mean
    direction of all the group's window queries;
  * needles: n_needle positions in [n_sink + 2k, P - 2k), at least 2k apart,
    hold 3*sqrt(D) times the unit mean direction of the group's SRH window
    queries (k = pooling kernel, P = L - W);
  * per-layer budgets: a Dirichlet(1) split of the total above a per-layer
    minimum, rounded down, remainder to the largest fractional parts; with a
    per-layer maximum, the excess of capped layers is split again over the
    others in proportion to their shares until none exceeds it.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field, replace

import numpy as np

F32 = 0
BF16 = 1


@dataclass(frozen=True)
class Workload:
    name: str
    cid: int                     # index used in the seed path
    n_layers: int
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    seq_len: int                 # fixed length (ragged workloads: upper bound)
    window: int
    dtype: int
    pool_kernel: int = 7
    pool_type: int = 0           # 0 max, 1 avg
    n_sink: int = 4
    n_needle: int = 16
    budget: int = 0              # fixed per-layer budget (0: Dirichlet split)
    budget_total_per_layer: int = 0
    budget_min: int = 0
    srh_per_group: tuple = (2,)  # one value, or a range (lo, hi) drawn uniformly
    ragged: tuple = ()           # (lo, hi) inclusive lengths when ragged
    srh_per_layer: int = 0       # > 0: that many SRHs over all of the layer's heads
    index_layer: bool = False    # one index set per layer (layer-shared)
    budget_max: int = 0          # > 0: per-layer budget cap of the Dirichlet split


WORKLOADS = {
    "tiny": Workload("tiny", 0, 1, 1, 8, 2, 64, 1024, 16, F32, n_sink=2,
                     n_needle=4, budget=64, srh_per_group=(1,)),
    "llama1": Workload("llama1", 1, 1, 1, 32, 8, 128, 32768, 32, BF16,
                       n_sink=4, n_needle=16, budget=1024, srh_per_group=(2,)),
    "llama32": Workload("llama32", 2, 32, 1, 32, 8, 128, 32768, 32, BF16,
                        n_sink=4, n_needle=16, budget_total_per_layer=256,
                        budget_min=64, srh_per_group=(1, 3)),
    "qwen128k": Workload("qwen128k", 3, 28, 1, 28, 4, 128, 131072, 64, BF16,
                         n_sink=4, n_needle=32, budget_total_per_layer=3932,
                         budget_min=128, srh_per_group=(2,)),
    "ragged8": Workload("ragged8", 4, 32, 8, 32, 8, 128, 16384, 32, BF16,
                        n_sink=4, n_needle=16, budget=256, srh_per_group=(2,),
                        ragged=(4096, 16384)),
    "paper": Workload("paper", 5, 32, 1, 32, 8, 128, 32768, 8, BF16, pool_kernel=5,
                      n_sink=4, n_needle=16, budget_total_per_layer=512, budget_min=32,
                      budget_max=3 * 512, srh_per_layer=4, index_layer=True),
}


def get(name: str, **overrides) -> Workload:
    """A named workload, optionally with fields replaced (smaller L, fewer layers)."""
    return replace(WORKLOADS[name], **overrides)


def _rng(seed: int, *path: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([int(seed)] + [int(p) for p in path]))


# ----------------------------------------------------------------- bf16 bits
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    rounding = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + rounding) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# ------------------------------------------------------------- layer shapes
def seq_lengths(w: Workload, seed: int = 0) -> np.ndarray:
    if w.ragged:
        lo, hi = w.ragged
        return _rng(seed, w.cid, 2).integers(lo, hi, size=w.batch, endpoint=True).astype(np.int64)
    return np.full(w.batch, w.seq_len, dtype=np.int64)


def cu_seqlens(lengths: np.ndarray) -> np.ndarray:
    return np.concatenate([[0], np.cumsum(lengths)]).astype(np.int32)


def layer_budgets(w: Workload, seed: int = 0) -> np.ndarray:
    """Per-layer budget vector (the same for every group of a layer)."""
    if w.budget:
        return np.full(w.n_layers, w.budget, dtype=np.int64)
    n = w.n_layers
    total = w.budget_total_per_layer * n
    rest = total - n * w.budget_min
    p = _rng(seed, w.cid, 3).dirichlet(np.ones(n))
    raw = p * rest
    if w.budget_max:
        cap = float(w.budget_max - w.budget_min)
        capped = np.zeros(n, dtype=bool)
        while True:
            over = ~capped & (raw > cap)
            if not over.any():
                break
            capped |= over
            excess = float(np.sum(raw[capped] - cap))
            raw[capped] = cap
            free = ~capped
            raw[free] += excess * p[free] / p[free].sum()
    b = w.budget_min + np.floor(raw).astype(np.int64)
    frac = raw - np.floor(raw)
    short = int(total - b.sum())
    order = np.lexsort((np.arange(n), -frac))   # largest fraction, then lowest layer
    b[order[:short]] += 1
    return b


def srh_mask(w: Workload, layer: int, seed: int = 0) -> np.ndarray:
    """uint8 [Hq]: 1 for the layer's Semantic Retrieval Heads."""
    G = w.n_q_heads // w.n_kv_heads
    rng = _rng(seed, w.cid, 1, layer)
    mask = np.zeros(w.n_q_heads, dtype=np.uint8)
    if w.srh_per_layer:
        mask[rng.choice(w.n_q_heads, w.srh_per_layer, replace=False)] = 1
        return mask
    for g in range(w.n_kv_heads):
        if len(w.srh_per_group) == 1:
            n = w.srh_per_group[0]
        else:
            n = int(rng.integers(w.srh_per_group[0], w.srh_per_group[1], endpoint=True))
        for h in rng.choice(G, n, replace=False):
            mask[g * G + int(h)] = 1
    return mask


def _unit(x: np.ndarray) -> np.ndarray:
    n = float(np.linalg.norm(x))
    return x / n if n > 0 else x


def _needle_positions(rng, n, lo, hi, gap):
    """n positions in [lo, hi), pairwise >= gap apart (rejection sampling)."""
    if n == 0 or hi - lo < 1:
        return np.zeros(0, dtype=np.int64)
    chosen = []
    tries = 0
    while len(chosen) < n and tries < 100000:
        p = int(rng.integers(lo, hi))
        tries += 1
        if all(abs(p - c) >= gap for c in chosen):
            chosen.append(p)
    return np.sort(np.array(chosen, dtype=np.int64))


@dataclass
class LayerInputs:
    """One layer's inputs.  Float arrays hold the values the kernels see
    (bf16-rounded where the workload is bf16); *_bits hold raw bf16 bits."""
    workload: Workload
    layer: int
    cu_seqlens: np.ndarray          # int32 [batch+1]
    srh_mask: np.ndarray            # uint8 [Hq]
    budget: int
    q_win: np.ndarray               # float32 [batch, W, Hq, D]
    k: np.ndarray                   # float32 [T, Hkv, D]
    v: np.ndarray                   # float32 [T, Hkv, D]
    needles: dict = field(default_factory=dict)   # (b, g) -> positions

    @property
    def dtype(self) -> int:
        return self.workload.dtype

    def bits(self, name: str) -> np.ndarray:
        """Raw storage of q_win/k/v: uint16 bf16 bits, or the fp32 array."""
        a = getattr(self, name)
        return f32_to_bf16_bits(a) if self.dtype == BF16 else a


def make_layer(w: Workload, layer: int = 0, seed: int = 0,
               lengths: np.ndarray | None = None, budget: int | None = None) -> LayerInputs:
    """Inputs of one layer of workload ``w`` (all sequences packed)."""
    W, Hq, Hkv, D = w.window, w.n_q_heads, w.n_kv_heads, w.head_dim
    G = Hq // Hkv
    lens = seq_lengths(w, seed) if lengths is None else np.asarray(lengths, dtype=np.int64)
    cu = cu_seqlens(lens)
    T = int(cu[-1])
    mask = srh_mask(w, layer, seed)
    if budget is None:
        budget = int(layer_budgets(w, seed)[layer])
    rnd = (lambda a: bf16_bits_to_f32(f32_to_bf16_bits(a))) if w.dtype == BF16 else (lambda a: a)
    q = np.empty((w.batch, W, Hq, D), dtype=np.float32)
    k = np.empty((T, Hkv, D), dtype=np.float32)
    v = np.empty((T, Hkv, D), dtype=np.float32)
    needles = {}
    for b in range(w.batch):
        L = int(lens[b])
        s0 = int(cu[b])
        rng = _rng(seed, w.cid, 0, layer, b)
        q[b] = rnd(rng.standard_normal((W, Hq, D), dtype=np.float32))
        kb = rng.standard_normal((L, Hkv, D), dtype=np.float32)
        v[s0:s0 + L] = rnd(rng.standard_normal((L, Hkv, D), dtype=np.float32))
        P = L - W
        for g in range(Hkv):
            heads = list(range(g * G, (g + 1) * G))
            srh = [h for h in heads if mask[h]] or heads
            sink_dir = _unit(np.mean(q[b][:, heads, :].astype(np.float64), axis=(0, 1)))
            needle_dir = _unit(np.mean(q[b][:, srh, :].astype(np.float64), axis=(0, 1)))
            n_sink = min(w.n_sink, max(P, 0))
            kb[:n_sink, g, :] = (3.0 * math.sqrt(D) * sink_dir).astype(np.float32)
            lo = n_sink + 2 * w.pool_kernel
            hi = P - 2 * w.pool_kernel
            pos = _needle_positions(rng, w.n_needle, lo, hi, 2 * w.pool_kernel) if hi > lo else \
                np.zeros(0, dtype=np.int64)
            kb[pos, g, :] = (3.0 * math.sqrt(D) * needle_dir).astype(np.float32)
            needles[(b, g)] = pos
        k[s0:s0 + L] = rnd(kb)
    return LayerInputs(workload=w, layer=layer, cu_seqlens=cu, srh_mask=mask,
                       budget=int(budget), q_win=q, k=k, v=v, needles=needles)


def make_layer_device(w: Workload, layer: int, seed: int, device, lengths=None,
                      budget: int | None = None):
    """The same recipe drawn with torch's generator on ``device`` (fast for the
    multi-GiB benchmark stacks).  Returns a dict of device tensors plus the
    host-side cu_seqlens, SRH mask and budget.  Values differ from make_layer's
    (another random stream) but follow the same distributions and structure."""
    import torch

    W, Hq, Hkv, D = w.window, w.n_q_heads, w.n_kv_heads, w.head_dim
    G = Hq // Hkv
    lens = seq_lengths(w, seed) if lengths is None else np.asarray(lengths, dtype=np.int64)
    cu = cu_seqlens(lens)
    T = int(cu[-1])
    mask = srh_mask(w, layer, seed)
    if budget is None:
        budget = int(layer_budgets(w, seed)[layer])
    dt = torch.bfloat16 if w.dtype == BF16 else torch.float32
    gen = torch.Generator(device=device)
    gen.manual_seed(int(np.random.SeedSequence([seed, w.cid, 7, layer]).generate_state(1)[0]))
    q = torch.randn((w.batch, W, Hq, D), generator=gen, device=device).to(dt)
    k32 = torch.randn((T, Hkv, D), generator=gen, device=device)
    v = torch.randn((T, Hkv, D), generator=gen, device=device).to(dt)
    needles = {}
    for b in range(w.batch):
        L = int(lens[b])
        s0 = int(cu[b])
        P = L - W
        rng = _rng(seed, w.cid, 8, layer, b)
        qb = q[b].float()
        for g in range(Hkv):
            heads = list(range(g * G, (g + 1) * G))
            srh = [h for h in heads if mask[h]] or heads
            sink_dir = qb[:, heads, :].mean(dim=(0, 1))
            needle_dir = qb[:, srh, :].mean(dim=(0, 1))
            sink_dir = sink_dir / sink_dir.norm().clamp_min(1e-30)
            needle_dir = needle_dir / needle_dir.norm().clamp_min(1e-30)
            n_sink = min(w.n_sink, max(P, 0))
            if n_sink:
                k32[s0:s0 + n_sink, g, :] = 3.0 * math.sqrt(D) * sink_dir
            lo, hi = n_sink + 2 * w.pool_kernel, P - 2 * w.pool_kernel
            pos = _needle_positions(rng, w.n_needle, lo, hi, 2 * w.pool_kernel) if hi > lo \
                else np.zeros(0, dtype=np.int64)
            if pos.size:
                k32[s0 + torch.from_numpy(pos).to(device), g, :] = 3.0 * math.sqrt(D) * needle_dir
            needles[(b, g)] = pos
    k = k32.to(dt)
    del k32
    cu_dev = torch.from_numpy(cu.astype(np.int32)).to(device)
    return dict(q_win=q, k=k, v=v, cu_seqlens=cu_dev, cu_seqlens_host=cu, srh_mask=mask,
                budget=int(budget), needles=needles)
