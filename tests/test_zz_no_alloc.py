"""The allocation-free entry point (compresskv_compress_layer_noalloc) against
compresskv_compress_layer with a workspace: bit-identical outputs on two calls
in a row, the second with a smaller input, through the C ABI."""
import sys

import numpy as np
import pytest
import torch

from paper_2606_24467_amd import compresskv as C
from paper_2606_24467_amd import workloads as wl
from tests import parity_helpers as H


def _outputs(x, budget, dev):
    shape = (x.workload.batch, x.workload.n_kv_heads, budget)
    dt = torch.bfloat16 if x.dtype == wl.BF16 else torch.float32
    idx = torch.full(shape, -7, dtype=torch.int32, device=dev)
    ko = torch.full(shape + (x.workload.head_dim,), 3.0, dtype=dt, device=dev)
    vo = torch.full_like(ko, 5.0)
    sc = torch.full((x.workload.n_kv_heads, int(x.cu_seqlens[-1])), -1.0, device=dev)
    return idx, ko, vo, sc


@pytest.mark.gpu
@pytest.mark.parametrize("scoring", [C.SCORE_TWO_PASS, C.SCORE_ONE_PASS])
def test_noalloc_matches_workspace_entry_point(gpu, scoring):
    cases = [
        (wl.get("ragged8", batch=4, ragged=(3000, 9000), n_needle=4), 21, 300),
        (wl.get("llama1", seq_len=2000 + 7, n_needle=4), 22, 128),   # smaller second call
    ]
    for w, seed, budget in cases:
        x = wl.make_layer(w, 0, seed=seed)
        print(f"case {w.name} L={np.diff(x.cu_seqlens).tolist()} budget={budget} "
              f"scoring={scoring}", file=sys.stderr, flush=True)
        q, k, v, cu = H.device_tensors(x, gpu)
        p = C.Problem(q, k, v, cu, cu_seqlens_host=x.cu_seqlens, scoring=scoring)
        ws = C.workspace(p, x.srh_mask, budget, gpu)
        ref = _outputs(x, budget, gpu)
        got = _outputs(x, budget, gpu)
        C.compresskv_compress_layer(p, q, k, v, x.srh_mask, budget, *ref, ws)
        C.compresskv_compress_layer_noalloc(p, q, k, v, x.srh_mask, budget, *got)
        torch.cuda.synchronize()
        for a, b in zip(ref, got):
            assert torch.equal(a, b)
        ora = H.run_oracle(x, budget)
        H.check_indices(got[0].cpu().numpy(), ora, x.cu_seqlens, w.window, budget)


def test_noalloc_rejects_problems_beyond_its_scratch():
    """A problem whose workspace exceeds the fixed scratch is refused before
    anything touches a device (so this runs without a GPU)."""
    w = wl.get("llama1", seq_len=64)
    x = wl.make_layer(w, 0, seed=23)
    q = torch.zeros((1, w.window, w.n_q_heads, w.head_dim), dtype=torch.bfloat16)
    k = torch.zeros((64, w.n_kv_heads, w.head_dim), dtype=torch.bfloat16)
    big = np.array([0, 2_000_000], dtype=np.int32)     # 8 heads x 2M tokens of scores: 64 MiB
    p = C.Problem(q, k, k, torch.from_numpy(big), cu_seqlens_host=big)
    assert C.compresskv_workspace_bytes(p, x.srh_mask, 128) > 32 << 20
    with pytest.raises(C.CompressKVError) as e:
        C.compresskv_compress_layer_noalloc(p, q, k, k, x.srh_mask, 128, k, k, k, None,
                                            stream=0)
    assert e.value.status == C.WORKSPACE_TOO_SMALL
    assert "allocation-free" in str(e.value)
