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


@pytest.mark.parametrize("S,N,H,Lc", [(3, 20, 64, 300), (2, 9, 1024, 700), (1, 1, 5, 41),
                                      (3, 800, 6, 48)])   # last: more pairs than one LDS block
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


# ------------------------------------------------------------ equations 2 - 4
ERR_RTOL = 2e-3   # fp32 attention and projection (exp2, fixed-order sums) against fp64


def _error_case(seed, lens, Hq, Hkv, D, T, B, d_model, dtype):
    """Full caches, decoding queries, W_O and a synthetic compact cache (a
    random sorted subset of min(L, B) positions per sequence and group, its
    K/V rows copied on the host), with the values the kernels read."""
    rng = np.random.default_rng(seed)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    tt = torch.bfloat16 if dtype == C.BF16 else torch.float32
    def rnd(*shape, s=1.0):
        return torch.from_numpy((rng.standard_normal(shape) * s).astype(np.float32)).to(tt)
    k = rnd(int(cu[-1]), Hkv, D)
    v = rnd(int(cu[-1]), Hkv, D)
    q = rnd(len(lens), T, Hq, D, s=2.0)
    w_o = rnd(d_model, Hq * D, s=1.0 / np.sqrt(Hq * D))
    batch = len(lens)
    idx = np.full((batch, Hkv, B), -1, dtype=np.int64)
    k_out = torch.zeros((batch, Hkv, B, D), dtype=tt)
    v_out = torch.zeros((batch, Hkv, B, D), dtype=tt)
    for b, L in enumerate(lens):
        n = min(L, B)
        for g in range(Hkv):
            keep = np.sort(rng.choice(L, size=n, replace=False))
            idx[b, g, :n] = keep
            k_out[b, g, :n] = k[cu[b] + keep, g]
            v_out[b, g, :n] = v[cu[b] + keep, g]
    return dict(cu=cu, k=k, v=v, q=q, w_o=w_o, idx=idx, k_out=k_out, v_out=v_out)


def _gpu_error(c, gpu, eps=1e-6):
    k, v, q = c["k"].to(gpu), c["v"].to(gpu), c["q"].to(gpu)
    cu = torch.from_numpy(c["cu"]).to(gpu)
    qw = torch.zeros((q.shape[0], 1, q.shape[2], q.shape[3]), dtype=q.dtype, device=gpu)
    p = C.Problem(qw, k, v, cu, cu_seqlens_host=c["cu"], pool_kernel=1)
    return C.layer_error(p, q, k, v, c["k_out"].to(gpu), c["v_out"].to(gpu), c["w_o"].to(gpu),
                         eps=eps).item()


def _oracle_error(c, eps=1e-6):
    f = lambda t: t.float().numpy().astype(np.float64)
    return OO.layer_error(f(c["q"]), f(c["k"]), f(c["v"]), c["cu"], c["idx"], f(c["w_o"]), eps=eps)


@pytest.mark.parametrize("name,kw", [
    ("bf16 D128 ragged", dict(lens=(3000, 1700), Hq=32, Hkv=8, D=128, T=8, B=256, d_model=512,
                              dtype=C.BF16)),
    ("bf16 64 rows", dict(lens=(2500,), Hq=32, Hkv=8, D=128, T=16, B=300, d_model=256,
                          dtype=C.BF16)),
    ("fp32 D64", dict(lens=(700, 1300, 90), Hq=8, Hkv=2, D=64, T=5, B=100, d_model=200,
                      dtype=C.F32)),
    ("bf16 one step", dict(lens=(1025,), Hq=8, Hkv=8, D=128, T=1, B=17, d_model=64,
                           dtype=C.BF16)),
    # more steps and sequences than one block of the kernels holds
    ("bf16 64 steps G=4 batch 2", dict(lens=(3000, 2200), Hq=32, Hkv=8, D=128, T=64, B=256,
                                       d_model=512, dtype=C.BF16)),
    ("bf16 20 steps G=7", dict(lens=(2600,), Hq=28, Hkv=4, D=128, T=20, B=128, d_model=256,
                               dtype=C.BF16)),
    ("fp32 40 sequences x 3 steps", dict(lens=tuple(range(100, 900, 20)), Hq=8, Hkv=2, D=64, T=3,
                                         B=64, d_model=128, dtype=C.F32)),
])
def test_layer_error_matches_oracle(gpu, name, kw):
    _say(f"case layer error {name}")
    c = _error_case(11, **kw)
    got = _gpu_error(c, gpu)
    want = _oracle_error(c)
    assert want > 0
    np.testing.assert_allclose(got, want, rtol=ERR_RTOL)


def test_layer_error_is_zero_when_every_position_is_kept(gpu):
    """B >= L: the compact cache holds every row in order, so both attentions
    see the same keys in the same chunks and the error is exactly 0."""
    c = _error_case(12, lens=(900, 400), Hq=16, Hkv=4, D=128, T=4, B=1024, d_model=128,
                    dtype=C.BF16)
    for b, L in enumerate((900, 400)):
        for g in range(4):
            assert np.array_equal(c["idx"][b, g, :L], np.arange(L))
    assert _gpu_error(c, gpu) == 0.0


def test_errors_to_layer_budgets(gpu):
    """Four layers: GPU errors, then the library's allocation, against the
    oracle's errors and allocation (the paper's m = 32, M = 3 x average)."""
    errs_gpu, errs_ora = [], []
    for l, B in enumerate((40, 120, 300, 80)):
        c = _error_case(20 + l, lens=(2000,), Hq=32, Hkv=8, D=128, T=8, B=B, d_model=256,
                        dtype=C.BF16)
        errs_gpu.append(_gpu_error(c, gpu))
        errs_ora.append(_oracle_error(c))
    np.testing.assert_allclose(errs_gpu, errs_ora, rtol=ERR_RTOL)
    per = 128
    got = C.allocate_budgets(np.array(errs_gpu, dtype=np.float32), 4 * per, 32, 3 * per)
    want = OO.allocate_budgets(OO.normalize_errors(np.array(errs_ora)), 4 * per, 32, 3 * per)
    assert got.sum() == 4 * per
    assert np.all(np.abs(got - want) <= 1)   # equal up to the rounding of nearly equal shares


def test_offline_kernels_are_deterministic(gpu):
    """Every sum of the SRH score and of the eviction error runs in a fixed
    order, so repeated calls give the same bits (here with several span
    lengths, answer steps spread over the waves of a head, and a ragged
    error case)."""
    attn, gen, ctx, spans = _calibration(21, 3, 40, 70, 600, max_span=150)
    first = _run(gpu, attn, gen, ctx, spans)
    for _ in range(3):
        assert np.array_equal(_run(gpu, attn, gen, ctx, spans), first)
    c = _error_case(12, lens=(2100, 900), Hq=16, Hkv=4, D=128, T=4, B=200, d_model=256,
                    dtype=C.BF16)
    e0 = _gpu_error(c, gpu)
    for _ in range(3):
        assert _gpu_error(c, gpu) == e0
