#!/usr/bin/env python
"""Benchmark of the CompressKV prefill-time eviction path on one MI355X.

A step compresses every layer of the workload once (one compresskv_compress_layers
call: score -> select -> gather for all layers) with inputs already resident in HBM;
--mode per-layer instead calls compresskv_compress_layer per layer over --streams streams.
The reported value is prompt tokens compressed per second per layer:
sum_b L_b * n_layers / step_time.

Default workload: 32 layers of the Llama-3-8B shape (32 query / 8 KV heads,
head_dim 128, bf16) at a 32768-token prompt, window 32, max pooling 7,
per-layer budgets from a Dirichlet split of 32 x 256 tokens per group (>= 64)
and 1-3 SRHs per group and layer.

Rank 0 prints one JSON line (see the contract in the repository's design notes),
including a roofline object for the dominant kernel phase (HIP events on the
launch stream) and the fp64 CPU oracle timed on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "prompt tokens compressed/sec per layer (1 GPU); % HBM roofline; MFMA util"
HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}   # dense, MI355X

# HBM bytes moved by one score phase (its kernels: fused_fill_kernel +
# fused_kernel + fused_catchup_kernel in one launch, or stats_kernel +
# colsum_kernel), measured with rocprofv3: FETCH_SIZE x 2 (the factor a plain
# copy of known size gives on this GPU) + WRITE_SIZE, in KiB per dispatch, in
# separate runs (profiles/).  A figure is valid only for the kernel sources it
# was taken with: keyed by their hash.  Single-layer workloads: one layer's
# score phase.
def _traffic(**kernels):
    """kernel name -> (FETCH_SIZE KiB, WRITE_SIZE KiB) per dispatch."""
    return sum(2 * f + w for f, w in kernels.values()) * 1024


MEASURED_TRAFFIC = {
    ("llama32", 32, "7f9fea8574bc8c35"): _traffic(
        fused_fill_kernel=(11.07, 8385.03),
        fused_kernel=(2286840.01, 37992.78),
        fused_catchup_kernel=(11.5, 0.0)),
    ("paper", 32, "7f9fea8574bc8c35"): _traffic(
        fused_fill_kernel=(11.03, 4161.03),
        fused_kernel=(959899.58, 15118.56),
        fused_catchup_kernel=(10.5, 0.0)),
    ("llama1", 1, "7f9fea8574bc8c35"): _traffic(
        fused_fill_kernel=(11.01, 196.06),
        fused_kernel=(63444.26, 1184.08),
        fused_catchup_kernel=(18.0, 0.0)),
    ("qwen128k", 28, "7f9fea8574bc8c35"): _traffic(
        stats_kernel=(1852714.58, 8064.0),
        colsum_kernel=(1947639.95, 57591.34)),
    ("ragged8", 32, "7f9fea8574bc8c35"): _traffic(
        stats_kernel=(2673161.67, 22016.0),
        colsum_kernel=(2843577.0, 82242.56)),
    ("tiny", 1, "7f9fea8574bc8c35"): _traffic(
        stats_kernel=(297.42, 16.5),
        colsum_kernel=(334.25, 8.42)),
}

# MFMA work the score phase executes, from rocprofv3 on the same sources:
# SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 FLOP summed over its kernels, and each
# kernel's SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / 8 XCDs x 1024 SIMDs).
def _mfma(**kernels):
    """kernel name -> (MFMA_MOPS_BF16, MFMA busy cycles, GRBM_GUI_ACTIVE) per dispatch."""
    return {"executed_flops_per_launch": sum(m for m, _, _ in kernels.values()) * 512,
            "busy_frac": {k: b / (g / 8 * 1024) for k, (_, b, g) in kernels.items()}}


MEASURED_MFMA = {
    ("llama32", 32, "7f9fea8574bc8c35"): _mfma(
        fused_kernel=(581683200.0, 290841600.0, 14110831.91)),
    ("paper", 32, "7f9fea8574bc8c35"): _mfma(
        fused_kernel=(70909952.0, 35454976.0, 6371246.21)),
    ("llama1", 1, "7f9fea8574bc8c35"): _mfma(
        fused_kernel=(17727488.0, 8863744.0, 805205.82)),
    ("qwen128k", 28, "7f9fea8574bc8c35"): _mfma(
        stats_kernel=(939524096.0, 469762048.0, 10013512.88),
        colsum_kernel=(987693056.0, 493846528.0, 14205209.47)),
    ("ragged8", 32, "7f9fea8574bc8c35"): _mfma(
        stats_kernel=(738197504.0, 369098752.0, 18793655.91),
        colsum_kernel=(731906048.0, 365953024.0, 21214593.44)),
}


# The sources that decide what the score phase reads and writes: its kernels,
# their device building blocks and the host plan (chunking, workspace).
SCORE_PHASE_SOURCES = ("ckv_device.h", "score_common.h", "score_kernels.h", "score_layers.hip",
                       "api.hip")


def kernel_source_hash() -> str:
    import hashlib
    root = os.path.join(ROOT, "paper_2606_24467_amd", "csrc")
    h = hashlib.sha256()
    for f in SCORE_PHASE_SOURCES:
        h.update(f.encode())
        with open(os.path.join(root, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def algorithmic_bytes(lens, Hkv, D, es, W, n_srh_total, budget, scored_groups):
    """Bytes the method must move for one layer: K once for every KV group that
    has an SRH (with the layer-shared index set a group without one adds
    nothing to the layer score), the SRH window queries, the kept K/V rows of
    every group read and written, and the int32 indices."""
    k_bytes = sum(lens) * scored_groups * D * es
    q_bytes = len(lens) * W * n_srh_total * D * es
    kept = sum(min(budget, L) for L in lens)
    gather = 4 * kept * Hkv * D * es + 4 * kept * Hkv
    return k_bytes + q_bytes, gather


def cpu_baseline(layers, w, seconds):
    """The fp64 oracle on (layer, sequence, KV group) units, layer after layer,
    until about `seconds` of CPU time, scaled to tokens per second per layer.
    With the layer-shared index set a unit is a (layer, sequence) with all of
    its groups."""
    import numpy as np
    import oracle as O

    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()
                       if i.get("user_api") == "blas"] or [1])
    except Exception:
        threads = 1
    G = w.n_q_heads // w.n_kv_heads
    cu = layers[0]["cu_seqlens_host"]
    tokens_layer = int(cu[-1])
    done_tokens = 0          # group-tokens: a (sequence, group) unit of length L counts L
    t_total = 0.0
    n = 0
    for lay in layers:
        q_all = lay["q_win"].float().cpu().numpy()
        for b in range(w.batch):
            s0, s1 = int(cu[b]), int(cu[b + 1])
            if w.index_layer:
                q = q_all[b:b + 1]
                k = lay["k"][s0:s1].float().cpu().numpy()
                v = lay["v"][s0:s1].float().cpu().numpy()
                t0 = time.perf_counter()
                O.compress_layer(q, k, v, np.array([0, s1 - s0]), lay["srh_mask"], lay["budget"],
                                 w.pool_kernel, w.pool_type, index_mode=O.LAYER_SHARED)
                t_total += time.perf_counter() - t0
                done_tokens += (s1 - s0) * w.n_kv_heads
                n += 1
                if t_total >= seconds:
                    break
                continue
            for g in range(w.n_kv_heads):
                q = q_all[b:b + 1, :, g * G:(g + 1) * G, :]
                k = lay["k"][s0:s1, g:g + 1, :].float().cpu().numpy()
                v = lay["v"][s0:s1, g:g + 1, :].float().cpu().numpy()
                mask = lay["srh_mask"][g * G:(g + 1) * G]
                t0 = time.perf_counter()
                O.compress_layer(q, k, v, np.array([0, s1 - s0]), mask, lay["budget"],
                                 w.pool_kernel, w.pool_type)
                t_total += time.perf_counter() - t0
                done_tokens += s1 - s0
                n += 1
                if t_total >= seconds:
                    break
            if t_total >= seconds:
                break
        if t_total >= seconds:
            break
    group_tokens_layer = tokens_layer * w.n_kv_heads
    t_layer = t_total * group_tokens_layer / done_tokens
    cpu_model = ""
    try:
        info = {}
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ":" in ln:
                    k, v = ln.split(":", 1)
                    info.setdefault(k.strip(), v.strip())
                if not ln.strip() and info:
                    break
        cpu_model = (f"{info.get('model name', '')} ({info.get('vendor_id', '')} family "
                     f"{info.get('cpu family', '?')} model {info.get('model', '?')} stepping "
                     f"{info.get('stepping', '?')}, {os.cpu_count()} logical CPUs)")
    except OSError:
        pass
    return {"value": tokens_layer / t_layer, "unit": "tokens/s/layer", "cores": int(threads),
            "kind": "oracle", "blas_threads": int(threads), "host_cpus": os.cpu_count(),
            "cpu_model": cpu_model,
            "note": "numpy fp64; its element-wise exp and max run on one thread",
            "sample": f"{n} (layer, sequence{'' if w.index_layer else ', KV group'}) units "
                      f"from layer 0 on "
                      f"({done_tokens} group-tokens, {done_tokens / group_tokens_layer:.2f} "
                      f"layers' worth), {t_total:.1f} s of oracle time, scaled to one layer"}


def _time_ms(torch, fn, reps=5):
    """Mean HIP-event time of fn() on the current stream (after one warm-up)."""
    fn()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(reps)]
    for e0, e1 in ev:
        e0.record()
        fn()
        e1.record()
    torch.cuda.synchronize()
    return float(sum(e0.elapsed_time(e1) for e0, e1 in ev) / reps)


def bench_offline(dev, C, wl, torch, np):
    """The offline analyses at the sizes of the Llama-3-8B setting, synthetic
    inputs: one JSON line per measurement with its algorithmic bytes."""
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    # SRH score (equation 1): 4 samples x 32 decoding steps, 32 layers x 32 heads,
    # 8192-token contexts, 32-token answer spans, every other step an answer token
    S, N, H, Lc, span = 4, 32, 1024, 8192, 32
    attn = torch.rand((S, N, H, Lc), generator=g, device=dev, dtype=torch.float32)
    ctx = torch.randint(0, 30000, (S, Lc), generator=g, device=dev, dtype=torch.int32)
    spans = np.array([[100 + 1000 * s, span] for s in range(S)], dtype=np.int32)
    gen = torch.full((S, N), 40000, device=dev, dtype=torch.int32)
    for s in range(S):
        gen[s, ::2] = ctx[s, spans[s, 0]]
    # inputs resident on the device before the timed calls (the convenience
    # wrapper would copy the spans from the host on every call)
    sp, spans_np = C.srh_problem(attn, spans)
    spans_dev = torch.from_numpy(spans_np).to(dev)
    srh_out = torch.empty(H, dtype=torch.float32, device=dev)
    ms = _time_ms(torch, lambda: C.compresskv_srh_scores(sp, attn, gen, ctx, spans_dev, srh_out))
    hit_bytes = S * (N // 2) * H * span * 4
    print(json.dumps({"metric": "SRH score (equation 1)", "workload":
                      f"{S} samples x {N} steps, {H} heads, context {Lc}, span {span}",
                      "ms": ms, "algorithmic_bytes": hit_bytes,
                      "achieved_GBs": hit_bytes / ms / 1e6, "bound": "latency"}), flush=True)
    del attn
    # layer eviction error (equations 2-4) at one Llama-3-8B layer: L = 32768,
    # 32 query / 8 KV heads, D = 128, bf16, 8 decoding steps, budget 256,
    # W_O 4096 x 4096
    L, Hq, Hkv, D, T, B, dm = 32768, 32, 8, 128, 8, 256, 4096
    bf = torch.bfloat16
    k = torch.randn((L, Hkv, D), generator=g, device=dev).to(bf)
    v = torch.randn((L, Hkv, D), generator=g, device=dev).to(bf)
    k_out = k[:B].permute(1, 0, 2).contiguous()[None]
    v_out = v[:B].permute(1, 0, 2).contiguous()[None]
    q_dec = torch.randn((1, T, Hq, D), generator=g, device=dev).to(bf)
    w_o = (torch.randn((dm, Hq * D), generator=g, device=dev) / 64).to(bf)
    cu_host = np.array([0, L], dtype=np.int32)
    cu = torch.from_numpy(cu_host).to(dev)
    p = C.Problem(torch.zeros((1, 1, Hq, D), dtype=bf, device=dev), k, v, cu,
                  cu_seqlens_host=cu_host, pool_kernel=1)
    e = C.CkvErrorProblem(n_steps=T, d_model=dm, budget=B, eps=1e-6)
    err_ws = torch.empty(C.compresskv_layer_error_workspace_bytes(p, e), dtype=torch.uint8,
                         device=dev)
    err = torch.empty(1, dtype=torch.float32, device=dev)
    ms = _time_ms(torch, lambda: C.compresskv_layer_error(p, e, q_dec, k, v, k_out, v_out, w_o,
                                                          err, err_ws))
    nbytes = 2 * L * Hkv * D * 2 + 2 * Hkv * B * D * 2 + dm * Hq * D * 2 + T * Hq * D * 2
    print(json.dumps({"metric": "layer eviction error (equations 2-4)", "workload":
                      f"L={L}, {Hq}q/{Hkv}kv heads, D={D}, bf16, {T} steps, budget {B}, "
                      f"W_O {dm}x{Hq * D}", "ms": ms, "algorithmic_bytes": nbytes,
                      "achieved_GBs": nbytes / ms / 1e6, "peak_GBs": 8000.0,
                      "frac": nbytes / ms / 1e6 / 8000.0, "bound": "hbm"}), flush=True)
    # per-group budgets against one fixed budget at the same total, one
    # Llama-3-8B layer at 32768 tokens
    w = wl.get("llama1")
    lay = wl.make_layer_device(w, 0, 0, dev)
    p1 = C.Problem(lay["q_win"], lay["k"], lay["v"], lay["cu_seqlens"],
                   cu_seqlens_host=lay["cu_seqlens_host"], pool_kernel=w.pool_kernel,
                   pool_type=w.pool_type)
    budgets = [64, 128, 256, 512, 1024, 1536, 2048, 2624]           # sum 8192 = 8 x 1024
    ws = C.workspace(p1, lay["srh_mask"], max(budgets), dev)
    ms_h = _time_ms(torch, lambda: C.compress_layer_heads(p1, lay["q_win"], lay["k"], lay["v"],
                                                          lay["srh_mask"], budgets, ws=ws))
    ms_f = _time_ms(torch, lambda: C.compress_layer(p1, lay["q_win"], lay["k"], lay["v"],
                                                    lay["srh_mask"], 1024, ws=ws))
    print(json.dumps({"metric": "per-group budgets (compress_layer_heads)", "workload":
                      "llama1: L=32768, 32q/8kv, D=128, bf16; budgets 64..2624 per group, "
                      "sum 8192", "ms": ms_h, "fixed_budget_1024_ms": ms_f}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=30)
    ap.add_argument("--workload", default="llama32",
                    help="tiny | llama1 | llama32 | qwen128k | ragged8 | paper")
    ap.add_argument("--sets", type=int, default=0,
                    help="single-layer workloads: input sets the steps rotate over (0: enough "
                         "for 512 MiB of K and V, at least 5, so no step finds its inputs in "
                         "the 256 MB last-level cache)")
    ap.add_argument("--layers", type=int, default=0, help="limit the layer count (0: all)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--mode", default="layers", choices=["layers", "per-layer"],
                    help="layers: one compresskv_compress_layers call per step (default); "
                         "per-layer: one compresskv_compress_layer call per layer")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--streams", type=int, default=2,
                    help="per-layer mode: alternate the layers over this many streams")
    ap.add_argument("--offline", action="store_true",
                    help="only time the offline analyses (SRH scores, layer eviction error) "
                         "and the per-group-budget path, one JSON line each")
    ap.add_argument("--scoring", default="auto", choices=["auto", "two", "one", "two-launches"],
                    help="scoring implementation (ckv_problem.scoring): the library's choice, "
                         "two passes over K (one launch where the shape allows), the single "
                         "pass, or two passes in two launches")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain elementwise copy of MIB MiB (3 times): the "
                         "reference point that scales the HBM byte counters")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: this path has no multi-GPU mode "
              f"(asked for --gpus {args.gpus}); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2606_24467_amd import build as B
    from paper_2606_24467_amd import compresskv as C
    from paper_2606_24467_amd import workloads as wl

    if not os.path.exists(B.lib_path()):
        B.build()
    dev = torch.device("cuda:0")
    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.ones(n // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)      # one kernel: reads n bytes, writes n bytes
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": n, "copy_calibration_bytes_written": n,
                          "launches": 3, "kernel": "torch neg (elementwise, fp32)"}), flush=True)
        return
    if args.offline:
        bench_offline(dev, C, wl, torch, np)
        return
    w = wl.get(args.workload)
    n_layers = args.layers or w.n_layers
    es = 2 if w.dtype == wl.BF16 else 4
    single = n_layers == 1
    mode = C.INDEX_LAYER if w.index_layer else C.INDEX_PER_GROUP
    if single:
        # one layer per step, rotating over input sets (distinct K, V, Q, SRH
        # masks) so that each step reads its inputs from HBM
        set_bytes = 2 * sum(int(x) for x in wl.seq_lengths(w, args.seed)) * w.n_kv_heads \
            * w.head_dim * es
        n_sets = args.sets or min(1024, max(5, -(-(512 << 20) // set_bytes)))
        budget0 = int(wl.layer_budgets(w, args.seed)[0])
        log(f"bench: workload {w.name}, one layer per step over {n_sets} input sets")
        layers = [wl.make_layer_device(w, r, args.seed, dev, budget=budget0)
                  for r in range(n_sets)]
    else:
        n_sets = 1
        log(f"bench: workload {w.name}, {n_layers} layers, generating inputs on the GPU")
        layers = [wl.make_layer_device(w, l, args.seed, dev) for l in range(n_layers)]
    torch.cuda.synchronize()
    lens = [int(x) for x in np.diff(layers[0]["cu_seqlens_host"])]
    budgets = [lay["budget"] for lay in layers]
    log(f"bench: inputs ready, lengths {lens[:8]}, budgets {budgets[:8]}...")

    scoring = {"auto": C.SCORE_AUTO, "two": C.SCORE_TWO_PASS, "one": C.SCORE_ONE_PASS,
               "two-launches": C.SCORE_TWO_LAUNCHES}[args.scoring]
    probs, outs = [], []
    score_bytes_total = 0
    alg_bytes_total = 0
    score_flops_total = 0   # one pass of window-row x key dot products
    for lay in layers:
        p = C.Problem(lay["q_win"], lay["k"], lay["v"], lay["cu_seqlens"],
                      cu_seqlens_host=lay["cu_seqlens_host"], pool_kernel=w.pool_kernel,
                      pool_type=w.pool_type, index_mode=mode, scoring=scoring)
        probs.append(p)
        B_l = lay["budget"]
        shape = (w.batch, w.n_kv_heads, B_l, w.head_dim)
        outs.append((torch.empty((w.batch, w.n_kv_heads, B_l), dtype=torch.int32, device=dev),
                     torch.empty(shape, dtype=lay["k"].dtype, device=dev),
                     torch.empty(shape, dtype=lay["v"].dtype, device=dev)))
        n_srh = int(lay["srh_mask"].sum())
        G = w.n_q_heads // w.n_kv_heads
        scored = int((lay["srh_mask"].reshape(w.n_kv_heads, G).sum(1) > 0).sum())
        sb, gb = algorithmic_bytes(lens, w.n_kv_heads, w.head_dim, es, w.window, n_srh, B_l,
                                   scored)
        score_flops_total += 2 * w.window * n_srh * w.head_dim * sum(lens)
        score_bytes_total += sb
        alg_bytes_total += sb + gb
    q_l = [lay["q_win"] for lay in layers]
    k_l = [lay["k"] for lay in layers]
    v_l = [lay["v"] for lay in layers]
    masks = np.stack([lay["srh_mask"] for lay in layers])
    main = torch.cuda.current_stream()

    if single:
        ws1 = torch.empty(max(C.compresskv_workspace_bytes(p, lay["srh_mask"], lay["budget"])
                              for p, lay in zip(probs, layers)), dtype=torch.uint8, device=dev)
        step_no = [0]

        def step():
            r = step_no[0] % n_sets
            step_no[0] += 1
            lay, (idx, k_out, v_out) = layers[r], outs[r]
            C.compresskv_compress_layer(probs[r], lay["q_win"], lay["k"], lay["v"],
                                        lay["srh_mask"], lay["budget"], idx, k_out, v_out, None,
                                        ws1, main)
        n_streams = 1
    elif args.mode == "layers":
        ws_layers = C.layers_workspace(probs[0], masks, dev)
        call = C.LayersCall(probs[0], q_l, k_l, v_l, masks, budgets, [o[0] for o in outs],
                            [o[1] for o in outs], [o[2] for o in outs], None, ws_layers)

        def step():
            call(main)
        n_streams = 1
    else:
        # One workspace per stream; every stream keeps the default priority.
        n_streams = max(1, args.streams)
        streams = [main] + [torch.cuda.Stream() for _ in range(n_streams - 1)]
        ws_need = max(C.compresskv_workspace_bytes(p, lay["srh_mask"], lay["budget"])
                      for p, lay in zip(probs, layers))
        ws = [torch.empty(ws_need, dtype=torch.uint8, device=dev) for _ in streams]

        def step():
            fork = torch.cuda.Event()
            fork.record(main)
            for st in streams[1:]:
                st.wait_event(fork)
            for li, (lay, p, (idx, k_out, v_out)) in enumerate(zip(layers, probs, outs)):
                si = li % n_streams
                C.compresskv_compress_layer(p, lay["q_win"], lay["k"], lay["v"],
                                            lay["srh_mask"], lay["budget"], idx, k_out, v_out,
                                            None, ws[si], streams[si])
            for st in streams[1:]:
                ev = torch.cuda.Event()
                ev.record(st)
                main.wait_event(ev)

    # Score phase alone (the two kernels that stream K), bracketed by events on
    # the stream it runs on: every layer in one multi-layer call, or (single
    # layer) one compresskv_score call per input set in turn.  It runs before
    # the warm-up steps (its first `pre` calls untimed), so the GPU's clocks
    # have settled when both this and the timed steps are measured.
    reps = max(3, args.steps)
    pre = 30
    sev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(reps + pre)]
    if single:
        scores1 = torch.empty((w.n_kv_heads, probs[0].total_tokens), dtype=torch.float32,
                              device=dev)
        for r in range(reps + pre):      # the first `pre` repetitions are a warm-up
            lay = layers[(r + 1) % n_sets]
            sev[r][0].record(main)
            C.compresskv_score(probs[(r + 1) % n_sets], lay["q_win"], lay["k"], lay["srh_mask"],
                               scores1, ws1, main)
            sev[r][1].record(main)
        # per step: the one layer's score bytes, not the sum over the sets
        score_bytes_total //= n_sets
        alg_bytes_total //= n_sets
        score_flops_total //= n_sets
    else:
        scores_all = torch.empty((n_layers, w.n_kv_heads, probs[0].total_tokens),
                                 dtype=torch.float32, device=dev)
        ws_s = C.layers_workspace(probs[0], masks, dev)
        for r in range(reps + pre):      # the first `pre` repetitions are a warm-up
            sev[r][0].record(main)
            C.compresskv_score_layers(probs[0], q_l, k_l, masks, scores_all, ws_s, main)
            sev[r][1].record(main)
    torch.cuda.synchronize()
    score_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in sev[pre:]]))
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"bench: {args.warmup} warmup steps done")
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    log(f"bench: {args.steps} timed steps in {elapsed * 1e3:.2f} ms")

    ms_per_step = elapsed * 1e3 / args.steps
    tokens = sum(lens)
    value = tokens * n_layers / (ms_per_step / 1e3)
    achieved = score_bytes_total / (score_ms / 1e3) / 1e9
    e2e_gbs = alg_bytes_total / (ms_per_step / 1e3) / 1e9
    path_id = C.compresskv_scoring_path(probs[0], layers[0]["srh_mask"])
    path_name = {1: "single pass", 2: "two passes, two launches",
                 3: "two passes, one launch"}[path_id]
    score_kernels = {1: "onepass_kernel (+ catch-up and boundary kernels)",
                     2: "stats_kernel + colsum_kernel",
                     3: "fused_kernel (+ its fill and catch-up kernels)"}[path_id]
    src_key = (w.name, n_layers, kernel_source_hash())
    traffic = MEASURED_TRAFFIC.get(src_key)
    counted = MEASURED_MFMA.get(src_key)
    dt = "bf16" if w.dtype == wl.BF16 else "f32"
    mfma_tflops = score_flops_total / (score_ms / 1e3) / 1e12

    result = {
        "metric": METRIC, "value": value, "unit": "tokens/s/layer", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": dt, "data": "synthetic",
        "config": {"workload": f"{w.name}: {n_layers} layers, batch {w.batch}, "
                               f"{w.n_q_heads}q/{w.n_kv_heads}kv heads, D={w.head_dim}, "
                               f"L={'ragged ' + str(w.ragged) if w.ragged else w.seq_len}, "
                               f"W={w.window}, maxpool {w.pool_kernel}" +
                   (f", top {w.srh_per_layer} SRHs per layer, layer-shared index set"
                    if w.index_layer else ""),
                   "layers": n_layers, "batch": w.batch, "seq_lens": lens[:16],
                   "budgets": budgets[:n_layers] if not single else budgets[:1],
                   "index_set": "layer-shared" if w.index_layer else "per KV group",
                   "mode": "one layer per step" if single else args.mode,
                   "input_sets": n_sets, "streams": n_streams,
                   "scoring": path_name},
        "roofline": {"bound": "hbm",
                     "kernel": (f"score phase: {score_kernels} of one layer "
                                "(compresskv_score, input sets in turn)") if single else
                               (f"score phase: {score_kernels} over {n_layers} "
                                f"layers (one compresskv_score_layers call)"),
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "avg_ms": score_ms, "bytes_per_launch": score_bytes_total,
                     "launches_timed": reps, "launches_untimed": pre,
                     "when": "before the warm-up steps"},
        "mfma": {"flops_per_launch": score_flops_total, "achieved": mfma_tflops,
                 "peak": MFMA_PEAK_TFLOPS[dt], "unit": "TFLOP/s",
                 "frac": mfma_tflops / MFMA_PEAK_TFLOPS[dt],
                 "note": "algorithmic Q.K^T FLOPs of the score phase (one pass)",
                 "counters": None if counted is None else {
                     "executed_flops_per_launch": counted["executed_flops_per_launch"],
                     "executed_frac": counted["executed_flops_per_launch"] / (score_ms / 1e3)
                                      / 1e12 / MFMA_PEAK_TFLOPS[dt],
                     "busy_frac": counted["busy_frac"],
                     "note": "both passes' MFMA FLOPs from SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 "
                             "over the same HIP-event time; MFMA busy cycles per kernel"}},
        "end_to_end": {"algorithmic_bytes_per_step": alg_bytes_total, "achieved_gbs": e2e_gbs,
                       "frac": e2e_gbs / HBM_PEAK_GBS},
    }
    if not args.no_cpu_baseline:
        log("bench: timing the fp64 oracle on a bounded sample")
        result["cpu_baseline"] = cpu_baseline(layers, w, args.cpu_seconds)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
