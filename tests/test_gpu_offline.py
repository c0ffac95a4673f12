"""GPU parity of the offline analyses against the fp64 oracle
(oracle/offline_oracle.py): the SRH score of equation 1 and each layer's
top-k SRH set."""
import os
import sys
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import offline_oracle as OO
from paper_2606_24467_amd import compresskv as C

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

SRH_RTOL = 1e-5   # fp32 sums per step over at most a few hundred weights, fp64 over steps


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _calibration(seed, S, N, H, Lc, max_span=40):
    """Synthetic calibration run: softmax attention rows with a few peaked
    heads, random token ids, answer spans, and decoding steps of which about
    half generate an answer token."""
    rng = np.random.default_rng(seed)
    logits = rng.standard_normal((S, N, H, Lc)).astype(np.float32)
    spans = np.stack([rng.integers(0, Lc - max_span, size=S),
                      rng.integers(1, max_span + 1, size=S)], 1).astype(np.int32)
    for s in range(S):   # every 7th head attends to the span
        a0, n = spans[s]
        logits[s, :, ::7, a0:a0 + n] += 4.0
    attn = np.exp(logits - logits.max(-1, keepdims=True))
    attn /= attn.sum(-1, keepdims=True)
    ctx = rng.integers(0, 1000, size=(S, Lc)).astype(np.int32)
    gen = rng.integers(1000, 2000, size=(S, N)).astype(np.int32)
    for s in range(S):
        a0, n = spans[s]
        hits = rng.random(N) < 0.5
        gen[s, hits] = ctx[s, a0 + rng.integers(0, n, size=hits.sum())]
    return attn.astype(np.float32), gen, ctx, spans


def _run(gpu, attn, gen, ctx, spans):
    at = torch.from_numpy(attn).to(gpu)
    return C.srh_scores(at, torch.from_numpy(gen).to(gpu), torch.from_numpy(ctx).to(gpu),
                        spans).cpu().numpy()


def test_srh_scores_hand_worked(gpu):
    rows = {}
    for line in open(os.path.join(GOLDEN, "srh_worked.txt")):
        line = line.strip()
        if line and not line.startswith("#"):
            k, *v = line.split()
            rows.setdefault(k, []).append(v)
    attn = np.zeros((1, 3, 2, 5), dtype=np.float32)
    for r in rows["attn"]:
        attn[0, int(r[0]), int(r[1])] = [float(Fraction(x)) for x in r[2:]]
    ctx = np.array([[int(x) for x in rows["ctx"][0]]], dtype=np.int32)
    gen = np.array([[int(x) for x in rows["gen"][0]]], dtype=np.int32)
    spans = np.array([[int(x) for x in rows["span"][0]]], dtype=np.int32)
    got = _run(gpu, attn, gen, ctx, spans)
    np.testing.assert_allclose(got, [float(Fraction(x)) for x in rows["scores"][0]], rtol=1e-6)
    mask = C.select_srh(torch.from_numpy(got).to(gpu), 1, 1).cpu().numpy()
    assert mask[0].tolist() == [1, 0]


@pytest.mark.parametrize("S,N,H,Lc", [(3, 20, 64, 300), (2, 9, 1024, 700), (1, 1, 5, 41)])
def test_srh_scores_match_oracle(gpu, S, N, H, Lc):
    _say(f"case srh S={S} N={N} H={H} L={Lc}")
    attn, gen, ctx, spans = _calibration(S * 100 + H, S, N, H, Lc, max_span=min(40, Lc - 1))
    got = _run(gpu, attn, gen, ctx, spans)
    want = OO.srh_scores(attn, gen, ctx, spans)
    np.testing.assert_allclose(got, want, rtol=SRH_RTOL, atol=1e-6)


def test_select_srh_matches_oracle_with_ties(gpu):
    rng = np.random.default_rng(5)
    n_layers, hp = 32, 32
    scores = rng.integers(0, 6, size=n_layers * hp).astype(np.float32)   # many ties
    for k in (1, 4, 31, 32):
        got = C.select_srh(torch.from_numpy(scores).to(gpu), n_layers, k).cpu().numpy()
        assert np.array_equal(got, OO.select_srh(scores, n_layers, k)), k


def test_calibration_to_layer_masks(gpu):
    """The scores of a 32-layer x 32-head calibration, ranked per layer, give
    the same SRH masks as the oracle's scores (a mask differs only where two
    oracle scores tie within the tolerance)."""
    S, N, H, Lc = 2, 16, 32 * 32, 512
    attn, gen, ctx, spans = _calibration(9, S, N, H, Lc)
    got = _run(gpu, attn, gen, ctx, spans)
    want = OO.srh_scores(attn, gen, ctx, spans)
    m_gpu = C.select_srh(torch.from_numpy(got).to(gpu), 32, 4).cpu().numpy()
    m_ora = OO.select_srh(want, 32, 4)
    for l in range(32):
        if np.array_equal(m_gpu[l], m_ora[l]):
            continue
        w = want[l * 32:(l + 1) * 32]
        kth = np.sort(w)[::-1][3]
        diff = np.flatnonzero(m_gpu[l] != m_ora[l])
        assert np.all(np.abs(w[diff] - kth) <= SRH_RTOL * kth), (l, diff)
