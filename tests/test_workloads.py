"""The seeded generator: determinism, structure, budgets, and that injected
needle keys survive the oracle's selection when the budget can hold them."""
import numpy as np
import pytest

import oracle as O
from paper_2606_24467_amd import workloads as wl


def test_same_seed_same_bytes_and_seed_changes_data():
    w = wl.get("tiny")
    a = wl.make_layer(w, 0, seed=3)
    b = wl.make_layer(w, 0, seed=3)
    c = wl.make_layer(w, 0, seed=4)
    for name in ("q_win", "k", "v"):
        assert np.array_equal(getattr(a, name), getattr(b, name))
        assert not np.array_equal(getattr(a, name), getattr(c, name))
    assert np.array_equal(a.srh_mask, b.srh_mask)


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.00390625, 1.005859375, 1.0078125, -2.5, 3.3e-20], dtype=np.float32)
    bits = wl.f32_to_bf16_bits(x)
    back = wl.bf16_bits_to_f32(bits)
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: ties to the even mantissa (1.0)
    assert back[1] == 1.0
    assert back[2] == np.float32(1.0078125)
    assert back[3] == np.float32(1.0078125)
    assert back[4] == -2.5
    import torch
    ref = torch.from_numpy(x).to(torch.bfloat16).float().numpy()
    np.testing.assert_array_equal(back, ref)


def test_bf16_workload_values_are_representable():
    w = wl.get("llama1", seq_len=512, n_needle=2)
    x = wl.make_layer(w, 0)
    for name in ("q_win", "k", "v"):
        a = getattr(x, name)
        np.testing.assert_array_equal(wl.bf16_bits_to_f32(wl.f32_to_bf16_bits(a)), a)


@pytest.mark.parametrize("name", ["llama32", "qwen128k", "paper"])
def test_dirichlet_budgets(name):
    w = wl.get(name)
    b = wl.layer_budgets(w)
    assert b.sum() == w.budget_total_per_layer * w.n_layers
    assert b.min() >= w.budget_min
    assert np.array_equal(b, wl.layer_budgets(w))
    assert b.max() <= (w.budget_max or w.seq_len)


def test_budget_cap_redistributes_in_proportion():
    """The paper's [m, M] constraint (section 4: m = 32, M = 3 x the average):
    with a cap that binds, no layer exceeds it, the total is kept, and every
    uncapped layer receives at least its uncapped share."""
    w = wl.get("paper")
    capped = wl.layer_budgets(w)
    free = wl.layer_budgets(wl.get("paper", budget_max=0))
    assert free.max() > w.budget_max            # the cap binds for this seed
    assert capped.max() == w.budget_max
    assert capped.sum() == free.sum()
    below = free < w.budget_max
    assert np.all(capped[below] >= free[below] - 1)


def test_paper_srh_masks_are_four_heads_of_the_layer():
    w = wl.get("paper")
    G = w.n_q_heads // w.n_kv_heads
    empty_groups = 0
    for layer in range(w.n_layers):
        m = wl.srh_mask(w, layer)
        assert m.sum() == 4
        empty_groups += int((m.reshape(w.n_kv_heads, G).sum(1) == 0).sum())
    assert empty_groups > 0                     # groups without an SRH occur


def test_srh_counts_and_lengths():
    w = wl.get("llama32")
    G = w.n_q_heads // w.n_kv_heads
    counts = set()
    for layer in range(w.n_layers):
        m = wl.srh_mask(w, layer).reshape(w.n_kv_heads, G).sum(1)
        assert m.min() >= 1 and m.max() <= 3
        counts |= set(m.tolist())
    assert counts == {1, 2, 3}
    lens = wl.seq_lengths(wl.get("ragged8"))
    assert lens.shape == (8,) and lens.min() >= 4096 and lens.max() <= 16384
    cu = wl.cu_seqlens(lens)
    assert cu[0] == 0 and np.all(np.diff(cu) == lens)


def test_sinks_and_needles_placed():
    w = wl.get("tiny")
    x = wl.make_layer(w, 0, seed=1)
    G = w.n_q_heads // w.n_kv_heads
    for (b, g), pos in x.needles.items():
        assert len(pos) == w.n_needle
        assert np.all(np.diff(pos) >= 2 * w.pool_kernel)
        assert pos.min() >= w.n_sink + 2 * w.pool_kernel
        assert pos.max() < w.seq_len - w.window - 2 * w.pool_kernel
        srh = [h for h in range(g * G, (g + 1) * G) if x.srh_mask[h]]
        u = x.q_win[b][:, srh, :].astype(np.float64).mean(axis=(0, 1))
        kn = x.k[pos[0], g].astype(np.float64)
        cos = kn @ u / np.linalg.norm(kn) / np.linalg.norm(u)
        assert cos > 0.999
        assert np.allclose(x.k[0, g], x.k[1, g])   # sinks share one key


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_needles_retained_by_oracle_on_tiny(seed):
    """Invariant: injected high-affinity needles are kept (budget - W = 48
    >= n_sink + r + n_needle * k = 2 + 3 + 4 * 7)."""
    w = wl.get("tiny")
    x = wl.make_layer(w, 0, seed=seed)
    r = O.compress_layer(x.q_win, x.k, x.v, x.cu_seqlens, x.srh_mask, x.budget,
                         w.pool_kernel, w.pool_type)
    for (b, g), pos in x.needles.items():
        kept = set(r.idx[b, g].tolist())
        assert set(pos.tolist()) <= kept, (g, pos, sorted(kept))
        assert set(range(w.seq_len - w.window, w.seq_len)) <= kept
