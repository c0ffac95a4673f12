"""The C ABI without a GPU: the library loads, exports every symbol the header
declares, sizes workspaces, and rejects invalid arguments on the host before
any HIP call (so no device is touched).  Only invalid calls are made here."""
import ctypes
import subprocess

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


def test_every_header_symbol_is_exported(L):
    names = C.exported_names()
    assert {"compresskv_score", "compresskv_select", "compresskv_gather",
            "compresskv_compress_layer", "compresskv_workspace_bytes",
            "compresskv_status_string", "compresskv_last_error"} <= set(names)
    out = subprocess.run(["nm", "-D", "--defined-only", B.lib_path()], capture_output=True,
                         text=True).stdout
    defined = {line.split()[-1] for line in out.splitlines() if line.strip()}
    for n in names:
        assert n in defined, n
        assert hasattr(L, n)


def test_status_strings(L):
    for s, text in [(0, "ok"), (1, "invalid argument"), (2, "unsupported"),
                    (3, "workspace too small"), (4, "HIP error")]:
        assert L.compresskv_status_string(s).decode() == text


class Case:
    """A valid problem description plus host arrays kept alive for the call."""

    def __init__(self, lens=(100, 200), Hq=8, Hkv=2, D=128, W=16, dtype=C.BF16):
        self.cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        self.mask = np.zeros(Hq, dtype=np.uint8)
        G = Hq // Hkv
        self.mask[::G] = 1
        self.p = C.CkvProblem(batch=len(lens), n_q_heads=Hq, n_kv_heads=Hkv, head_dim=D,
                              window=W, dtype=dtype, pool_type=C.POOL_MAX, pool_kernel=7,
                              reduce_order=C.POOL_THEN_MEAN, scale=0.0, cu_seqlens=FAKE,
                              cu_seqlens_host=self.cu.ctypes.data, k_stride_tok=Hkv * D,
                              k_stride_head=D, v_stride_tok=Hkv * D, v_stride_head=D)

    def ws_bytes(self, L, budget=64):
        return L.compresskv_workspace_bytes(ctypes.byref(self.p), self.mask.ctypes.data, budget)

    def score(self, L, q=FAKE, k=FAKE, scores=FAKE, ws=FAKE, ws_bytes=1 << 40):
        return L.compresskv_score(ctypes.byref(self.p), q, k, self.mask.ctypes.data, scores, ws,
                                  ws_bytes, None)

    def compress(self, L, budget=64, ws_bytes=1 << 40, ws=FAKE, k_out=FAKE):
        return L.compresskv_compress_layer(ctypes.byref(self.p), FAKE, FAKE, FAKE,
                                           self.mask.ctypes.data, budget, FAKE, k_out, FAKE, None,
                                           ws, ws_bytes, None)

    def select(self, L, budget=64):
        return L.compresskv_select(ctypes.byref(self.p), FAKE, budget, FAKE, None, 0, None)

    def gather(self, L, budget=64, idx=FAKE):
        return L.compresskv_gather(ctypes.byref(self.p), FAKE, FAKE, idx, budget, FAKE, FAKE,
                                   None)


def test_workspace_bytes_layout(L):
    c = Case()
    n = c.ws_bytes(L)
    assert n > 0 and n % 256 == 0
    T = int(c.cu[-1])
    scores = -(-2 * T * 4 // 256) * 256
    assert n >= scores + 2 * 2 * 16 * 8          # scores + one chunk of row stats per group
    assert L.compresskv_last_error().decode() == ""


def _mutate(case, **fields):
    for k, v in fields.items():
        setattr(case.p, k, v)
    return case


INVALID = [
    ("batch", dict(batch=0), C.INVALID_ARGUMENT),
    ("heads", dict(n_q_heads=7), C.INVALID_ARGUMENT),
    ("head_dim", dict(head_dim=96), C.UNSUPPORTED),
    ("dtype", dict(dtype=7), C.UNSUPPORTED),
    ("window", dict(window=0), C.INVALID_ARGUMENT),
    ("even pool", dict(pool_kernel=4), C.INVALID_ARGUMENT),
    ("big pool", dict(pool_kernel=33), C.INVALID_ARGUMENT),
    ("pool type", dict(pool_type=2), C.INVALID_ARGUMENT),
    ("order", dict(reduce_order=2), C.INVALID_ARGUMENT),
    ("cu null", dict(cu_seqlens=None), C.INVALID_ARGUMENT),
    ("cu misaligned", dict(cu_seqlens=FAKE + 2), C.UNSUPPORTED),
    ("stride not 16-byte multiple", dict(k_stride_tok=2 * 128 + 4), C.UNSUPPORTED),
    ("stride zero", dict(v_stride_head=0), C.INVALID_ARGUMENT),
    ("head stride below head_dim", dict(k_stride_head=120), C.INVALID_ARGUMENT),
    ("token stride below head_dim", dict(v_stride_tok=64), C.INVALID_ARGUMENT),
    ("scoring", dict(scoring=4), C.INVALID_ARGUMENT),
    ("too many kv heads", dict(n_kv_heads=256, n_q_heads=256), C.UNSUPPORTED),
    ("index mode", dict(index_mode=2), C.INVALID_ARGUMENT),
    ("reserved", dict(reserved=1), C.INVALID_ARGUMENT),
    ("layer set, mean then pool", dict(index_mode=C.INDEX_LAYER, reduce_order=C.MEAN_THEN_POOL),
     C.UNSUPPORTED),
]


@pytest.mark.parametrize("name,fields,status", INVALID, ids=[c[0] for c in INVALID])
def test_invalid_problem_is_rejected_everywhere(L, name, fields, status):
    for call in ("score", "compress", "select", "gather"):
        c = _mutate(Case(), **fields)
        st = getattr(c, call)(L)
        assert st == status, (call, st, L.compresskv_last_error())
        assert L.compresskv_last_error().decode() != ""
    c = _mutate(Case(), **fields)
    assert c.ws_bytes(L) == 0


@pytest.mark.parametrize("cu,status", [
    ([0, 100, 90], C.INVALID_ARGUMENT),     # decreasing
    ([0, 10, 200], C.INVALID_ARGUMENT),     # a sequence shorter than the window
    ([5, 100, 300], C.INVALID_ARGUMENT),    # cu[0] != 0
])
def test_bad_cu_seqlens(L, cu, status):
    c = Case()
    c.cu[:] = cu
    assert c.score(L) == status
    assert c.compress(L) == status


def test_mask_rules(L):
    c = Case()
    c.mask[:] = 0
    c.mask[0] = 1                      # group 1 has no SRH
    assert c.score(L) == C.INVALID_ARGUMENT
    assert "no Semantic Retrieval Head" in L.compresskv_last_error().decode()
    c = Case(W=64, Hq=32, Hkv=4)
    c.mask[:] = 1                      # 8 SRHs x 4 row tiles = 32 > 16
    assert c.score(L) == C.UNSUPPORTED


def test_row_tile_limits(L):
    """Up to 16 row tiles per group (W = 64 with 4 SRHs in one group); 12
    for fp32 queries at head_dim 128, whose 16 tiles would not fit the LDS.
    Only the workspace query runs: it plans the call without touching a
    device."""
    def case(dtype, D, n_srh):
        c = Case(W=64, Hq=32, Hkv=4, D=D, dtype=dtype)
        c.mask[:] = 0
        c.mask[:n_srh] = 1             # n_srh SRHs in group 0, 4 row tiles each
        c.mask[8::8] = 1               # one in every other group
        return c
    assert case(C.BF16, 128, 4).ws_bytes(L) > 0
    assert case(C.F32, 64, 4).ws_bytes(L) > 0
    assert case(C.F32, 128, 3).ws_bytes(L) > 0
    assert case(C.F32, 128, 4).ws_bytes(L) == 0
    assert "must be <= 12" in L.compresskv_last_error().decode()
    assert case(C.BF16, 128, 5).ws_bytes(L) == 0
    assert "must be <= 16" in L.compresskv_last_error().decode()


def test_mask_rules_of_the_layer_shared_set(L):
    c = _mutate(Case(), index_mode=C.INDEX_LAYER)
    c.mask[:] = 0
    c.mask[0] = 1                      # group 1 has no SRH: allowed for a layer-wide set
    assert c.ws_bytes(L) > 0
    assert L.compresskv_last_error().decode() == ""
    c.mask[:] = 0                      # but the layer needs one
    assert c.score(L) == C.INVALID_ARGUMENT
    assert "no Semantic Retrieval Head" in L.compresskv_last_error().decode()
    assert c.ws_bytes(L) == 0
    m = _mutate(LayersCase(n_layers=3), index_mode=C.INDEX_LAYER)
    m.masks[1, :] = 0
    m.masks[1, 0] = 1
    assert m.ws_bytes(L) > 0
    m.masks[2, :] = 0
    assert m.compress_layers(L) == C.INVALID_ARGUMENT
    assert "layer 2" in L.compresskv_last_error().decode()


def test_budget_pointer_and_workspace_rules(L):
    c = Case()
    assert c.compress(L, budget=15) == C.INVALID_ARGUMENT          # budget < W
    assert c.select(L, budget=15) == C.INVALID_ARGUMENT
    assert c.gather(L, budget=0) == C.INVALID_ARGUMENT
    assert c.score(L, q=0) == C.INVALID_ARGUMENT
    assert c.score(L, k=FAKE + 8) == C.UNSUPPORTED                 # 16-byte alignment
    assert c.gather(L, idx=FAKE + 2) == C.UNSUPPORTED
    assert c.compress(L, k_out=0) == C.INVALID_ARGUMENT
    need = c.ws_bytes(L)
    assert c.compress(L, ws_bytes=need - 1) == C.WORKSPACE_TOO_SMALL
    assert c.score(L, ws_bytes=need - 1) == C.WORKSPACE_TOO_SMALL
    assert c.compress(L, ws=FAKE + 16) == C.UNSUPPORTED            # 256-byte alignment


class LayersCase(Case):
    """A valid multi-layer call: n_layers copies of the problem's operands."""

    def __init__(self, n_layers=3, **kw):
        super().__init__(**kw)
        self.n = n_layers
        self.masks = np.ascontiguousarray(np.tile(self.mask, (n_layers, 1)))
        self.budgets = np.full(n_layers, 64, dtype=np.int32)
        self.arrays = {name: (ctypes.c_void_p * n_layers)(*([FAKE] * n_layers))
                       for name in ("q", "k", "v", "idx", "k_out", "v_out")}

    def addr(self, name):
        return ctypes.cast(self.arrays[name], ctypes.c_void_p).value

    def ws_bytes(self, L, budget=64):
        return L.compresskv_layers_workspace_bytes(ctypes.byref(self.p), self.n,
                                                   self.masks.ctypes.data)

    def compress_layers(self, L, ws_bytes=1 << 40, ws=FAKE, n=None):
        return L.compresskv_compress_layers(
            ctypes.byref(self.p), self.n if n is None else n, self.addr("q"), self.addr("k"),
            self.addr("v"), self.masks.ctypes.data, self.budgets.ctypes.data, self.addr("idx"),
            self.addr("k_out"), self.addr("v_out"), None, ws, ws_bytes, None)

    def score_layers(self, L, scores=FAKE, ws_bytes=1 << 40):
        return L.compresskv_score_layers(ctypes.byref(self.p), self.n, self.addr("q"),
                                         self.addr("k"), self.masks.ctypes.data, scores, FAKE,
                                         ws_bytes, None)


@pytest.mark.parametrize("name,fields,status", INVALID, ids=[c[0] for c in INVALID])
def test_invalid_problem_is_rejected_by_multi_layer_calls(L, name, fields, status):
    c = _mutate(LayersCase(), **fields)
    assert c.compress_layers(L) == status, L.compresskv_last_error()
    c = _mutate(LayersCase(), **fields)
    assert c.score_layers(L) == status, L.compresskv_last_error()
    c = _mutate(LayersCase(), **fields)
    assert c.ws_bytes(L) == 0


def test_multi_layer_workspace_grows_with_layers(L):
    one, four = LayersCase(n_layers=1), LayersCase(n_layers=4)
    n1, n4 = one.ws_bytes(L), four.ws_bytes(L)
    assert n1 > 0 and n4 > 0 and n1 % 256 == 0 and n4 % 256 == 0
    T = int(one.cu[-1])
    assert n4 - n1 >= 3 * 2 * T * 4                # three more layers of scores at least
    assert n4 < 4 * n1 + 4 * 1024


def test_multi_layer_rules_name_the_layer(L):
    c = LayersCase(n_layers=4)
    c.masks[2, :] = 0
    c.masks[2, 0] = 1                               # layer 2, group 1: no SRH
    assert c.compress_layers(L) == C.INVALID_ARGUMENT
    assert "layer 2" in L.compresskv_last_error().decode()
    c = LayersCase(n_layers=4)
    c.budgets[1] = 15                               # < W
    assert c.compress_layers(L) == C.INVALID_ARGUMENT
    assert "layer 1" in L.compresskv_last_error().decode()
    c = LayersCase(n_layers=4)
    c.arrays["k_out"][3] = None
    assert c.compress_layers(L) == C.INVALID_ARGUMENT
    assert "layer 3: k_out" in L.compresskv_last_error().decode()
    c = LayersCase(n_layers=4)
    c.arrays["v"][0] = FAKE + 8                     # 16-byte alignment
    assert c.compress_layers(L) == C.UNSUPPORTED
    c = LayersCase(n_layers=4)
    assert c.compress_layers(L, n=0) == C.INVALID_ARGUMENT
    need = c.ws_bytes(L)
    assert c.compress_layers(L, ws_bytes=need - 1) == C.WORKSPACE_TOO_SMALL
    assert c.compress_layers(L, ws=FAKE + 16) == C.UNSUPPORTED
    assert c.score_layers(L, scores=0) == C.INVALID_ARGUMENT
    assert c.score_layers(L, ws_bytes=need - 1) == C.WORKSPACE_TOO_SMALL


def test_multi_layer_row_tile_limit_uses_the_largest_layer(L):
    c = LayersCase(n_layers=2, W=64, Hq=32, Hkv=4)
    c.masks[1, :] = 1                               # layer 1: 8 SRHs x 4 row tiles > 16
    assert c.compress_layers(L) == C.UNSUPPORTED
    assert c.ws_bytes(L) == 0


def test_group_budget_rules(L):
    c = Case()                                   # Hkv = 2, W = 16
    gb = np.array([64, 32], dtype=np.int32)
    f_sel = lambda b, p=c.p: L.compresskv_select_heads(ctypes.byref(p), FAKE, b, FAKE, None)
    f_gat = lambda b, p=c.p: L.compresskv_gather_heads(ctypes.byref(p), FAKE, FAKE, FAKE, b,
                                                       FAKE, FAKE, None)
    f_all = lambda b, p=c.p, ws=1 << 40: L.compresskv_compress_layer_heads(
        ctypes.byref(p), FAKE, FAKE, FAKE, c.mask.ctypes.data, b, FAKE, FAKE, FAKE, None, FAKE,
        ws, None)
    for f in (f_sel, f_gat, f_all):
        assert f(None) == C.INVALID_ARGUMENT
        low = np.array([64, 15], dtype=np.int32)          # group 1 below W
        assert f(low.ctypes.data) == C.INVALID_ARGUMENT
        assert "group 1" in L.compresskv_last_error().decode()
    layer = _mutate(Case(), index_mode=C.INDEX_LAYER)
    assert L.compresskv_select_heads(ctypes.byref(layer.p), FAKE, gb.ctypes.data, FAKE,
                                     None) == C.UNSUPPORTED
    need = c.ws_bytes(L, budget=64)
    assert f_all(gb.ctypes.data, ws=need - 1) == C.WORKSPACE_TOO_SMALL
    assert L.compresskv_gather_heads(ctypes.byref(c.p), FAKE, FAKE, FAKE + 2, gb.ctypes.data,
                                     FAKE, FAKE, None) == C.UNSUPPORTED


@pytest.mark.parametrize("name,fields,mask_heads", [
    ("fp32 inputs", dict(dtype=C.F32), None),
    ("layer-shared index set", dict(index_mode=C.INDEX_LAYER), None),
    ("more than 6 row tiles per group", dict(n_q_heads=8, n_kv_heads=1, window=16), 7),
])
def test_forced_single_pass_where_it_does_not_apply(L, name, fields, mask_heads):
    """CKV_SCORE_ONE_PASS on a problem the single pass does not cover is
    refused on the host with CKV_UNSUPPORTED (nothing is enqueued); the
    workspace size does not depend on the scoring field."""
    c = Case()
    if "n_q_heads" in fields:
        c = Case(Hq=8, Hkv=1)
    _mutate(c, **fields)
    if mask_heads:
        c.mask[:] = 0
        c.mask[:mask_heads] = 1
    n_auto = c.ws_bytes(L)
    _mutate(c, scoring=C.SCORE_ONE_PASS)
    assert c.ws_bytes(L) == n_auto > 0
    for call in ("score", "compress"):
        st = getattr(c, call)(L)
        assert st == C.UNSUPPORTED, (call, st, L.compresskv_last_error())
        assert "single-pass" in L.compresskv_last_error().decode()


# (lengths, window, SRHs per group, dtype) -> path of CKV_SCORE_AUTO, _TWO_PASS,
# _TWO_LAUNCHES (1 single pass, 2 two launches, 3 one launch).  Statistics
# chunks are 512 keys up to 8k-key sequences of 8 groups and 1024 at 32k; the
# library's own choice takes one launch for bf16, at most 6 row tiles
# (ceil(W/16) x SRHs) and at least 16 chunks in every sequence.
PATH_CASES = [
    ("32k, 2 row tiles", (32768,), 32, 1, C.BF16, (3, 3, 2)),
    ("8192 keys: 16 chunks of 512", (8192,), 32, 1, C.BF16, (3, 3, 2)),
    ("8000 keys: under 16 chunks", (8000,), 32, 1, C.BF16, (2, 3, 2)),
    ("ragged 4k and 16k", (4096, 16384), 32, 1, C.BF16, (2, 3, 2)),
    ("6 row tiles", (32768,), 48, 2, C.BF16, (3, 3, 2)),
    ("8 row tiles", (32768,), 64, 2, C.BF16, (2, 3, 2)),
    ("12 row tiles", (32768,), 64, 3, C.BF16, (2, 2, 2)),
    ("fp32", (32768,), 32, 1, C.F32, (2, 2, 2)),
]


@pytest.mark.parametrize("name,lens,W,n_srh,dtype,expect", PATH_CASES,
                         ids=[c[0] for c in PATH_CASES])
def test_scoring_path_choice_on_the_host(L, name, lens, W, n_srh, dtype, expect):
    """compresskv_scoring_path needs no GPU for the two-pass forms; each
    scoring field gets the form the header documents."""
    L.compresskv_scoring_path.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    L.compresskv_scoring_path.restype = ctypes.c_int
    c = Case(lens=lens, Hq=32, Hkv=8, W=W, dtype=dtype)
    c.mask[:] = 0
    for g in range(8):
        c.mask[4 * g:4 * g + n_srh] = 1
    for scoring, want in zip((C.SCORE_AUTO, C.SCORE_TWO_PASS, C.SCORE_TWO_LAUNCHES), expect):
        _mutate(c, scoring=scoring)
        got = L.compresskv_scoring_path(ctypes.byref(c.p), c.mask.ctypes.data)
        assert got == want, (name, scoring, got, L.compresskv_last_error())
