"""The offline entry points (include/compresskv_offline.h) without a GPU:
every invalid call is rejected on the host before any HIP call."""
import ctypes

import numpy as np
import pytest

from paper_2606_24467_amd import build as B
from paper_2606_24467_amd import compresskv as C

FAKE = 0x10000000  # aligned, never dereferenced: every call below fails validation first


@pytest.fixture(scope="module")
def L():
    import os
    if not os.path.exists(B.lib_path()):
        B.build()
    return C.lib()


def _srh(S=2, N=3, H=8, Lc=50, spans=((1, 4), (10, 3))):
    spans_np = np.ascontiguousarray(np.array(spans, dtype=np.int32))
    p = C.CkvSrhProblem(n_samples=S, n_steps=N, n_heads=H, ctx_len=Lc,
                        spans_host=spans_np.ctypes.data)
    return p, spans_np


def _call(L, p, attn=FAKE, gen=FAKE, ctx=FAKE, spans=FAKE, scores=FAKE):
    return L.compresskv_srh_scores(ctypes.byref(p), attn, gen, ctx, spans, scores, None)


def test_srh_scores_validation(L):
    p, keep = _srh()
    assert L.compresskv_srh_scores(None, FAKE, FAKE, FAKE, FAKE, FAKE, None) == C.INVALID_ARGUMENT
    for field in ("n_samples", "n_steps", "n_heads", "ctx_len"):
        q, keep2 = _srh()
        setattr(q, field, 0)
        assert _call(L, q) == C.INVALID_ARGUMENT, field
    for spans in (((-1, 4), (10, 3)), ((1, 0), (10, 3)), ((1, 4), (48, 3))):
        q, keep3 = _srh(spans=spans)
        assert _call(L, q) == C.INVALID_ARGUMENT, spans
        assert "span" in L.compresskv_last_error().decode()
    q, keep4 = _srh()
    q.spans_host = None
    assert _call(L, q) == C.INVALID_ARGUMENT
    for arg in ("attn", "gen", "ctx", "spans", "scores"):
        assert _call(L, p, **{arg: 0}) == C.INVALID_ARGUMENT, arg
        assert _call(L, p, **{arg: FAKE + 2}) == C.UNSUPPORTED, arg


def test_select_srh_validation(L):
    f = L.compresskv_select_srh
    assert f(0, 32, FAKE, 4, FAKE, None) == C.INVALID_ARGUMENT
    assert f(32, 0, FAKE, 4, FAKE, None) == C.UNSUPPORTED
    assert f(32, 1025, FAKE, 4, FAKE, None) == C.UNSUPPORTED
    assert f(32, 32, FAKE, 0, FAKE, None) == C.INVALID_ARGUMENT
    assert f(32, 32, FAKE, 33, FAKE, None) == C.INVALID_ARGUMENT
    assert f(32, 32, None, 4, FAKE, None) == C.INVALID_ARGUMENT
    assert f(32, 32, FAKE, 4, None, None) == C.INVALID_ARGUMENT
    assert f(32, 32, FAKE + 2, 4, FAKE, None) == C.UNSUPPORTED
