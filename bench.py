#!/usr/bin/env python3
"""Benchmark of the sparse block-decode hot path on one MI355X.

A step is one block of the two-stream pipeline (herald_decode_block) on the
8B-class layer workload (bf16, 16 sequences x 32768 cached tokens, 32 query /
8 KV heads, d=128, B=32, T=32, 5% budget): the next block's selection
(representative query, scoring scan, GQA importance, top-k, gather) on the
retrieval stream overlapped with T=32 denoising steps of block attention on
the main stream, then the join, the append of the completed block and the
pool swap. Inputs are seeded synthetic tensors resident in HBM before timing.

Prints one JSON line. `value` is denoise steps/s of the whole pipeline
(T steps per block / block time). The roofline object is for the dominant
kernel (block attention: HBM-bound, its K/V bytes over the launch time),
timed with HIP events on its stream; the
selection scan's HBM figures and the CPU oracle's rate are reported beside it.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0
FP32_VECTOR_PEAK_TFLOPS = 157.3


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="layer32k",
                    choices=["layer32k", "long128k", "tiny", "ragged", "pipeline36",
                             "xq-sweep"])
    ap.add_argument("--blocks", type=int, default=3,
                    help="timed blocks of the 36-layer pipeline workload")
    ap.add_argument("--dense-layers", type=int, default=0,
                    help="36-layer workload: how many first layers keep exact attention")
    ap.add_argument("--drafts", action="store_true",
                    help="36-layer workload: draft lookahead (draft group at step 1, the next "
                         "selection after it with the draft KV as normalisation tail)")
    ap.add_argument("--select-x", type=int, default=0, choices=[0, 1],
                    help="36-layer workload: next-block representative query, 0 the mean of "
                         "the block's queries, 1 its centre row")
    ap.add_argument("--graph", action="store_true",
                    help="8B-class layer: replay the pipelined block from HIP graphs (one per "
                         "pool parity, captured after the warm-up)")
    ap.add_argument("--serial", action="store_true",
                    help="one stream: the next block's selection and gather run on the main "
                         "stream ahead of the denoising steps instead of beside them")
    ap.add_argument("--dense", action="store_true",
                    help="denoise over the full cache (GPU-only dense baseline)")
    ap.add_argument("--reps", type=int, default=30, help="isolated kernel timing reps")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seqs", type=int, default=0,
                    help="sequences in the CPU oracle sample (0: the whole batch)")
    ap.add_argument("--cpu-steps", type=int, default=0,
                    help="attention steps per sampled sequence (0: all T)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain copy of MIB MiB (counter calibration)")
    ap.add_argument("--read-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain read (sum) of MIB MiB (counter calibration)")
    return ap.parse_args()


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: the hot path is measured on a single "
              "MI355X, and the library has no multi-GPU path (each GPU would take its own "
              "sequences or KV heads with no exchange).", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_21633_amd import herald as H
    from paper_2606_21633_amd import synth

    dev = "cuda:0"
    torch.cuda.set_device(0)
    if args.copy_calibration:
        return copy_calibration(args.copy_calibration)
    if args.read_calibration:
        return read_calibration(args.read_calibration)
    if args.workload == "ragged":
        return bench_ragged(args)
    if args.workload == "pipeline36":
        return bench_pipeline36(args)
    if args.workload == "xq-sweep":
        return bench_xq_sweep(args)
    wl = {"layer32k": synth.LAYER_32K, "long128k": synth.LONG_128K,
          "tiny": synth.TINY_F32}[args.workload]
    b, B, T = wl.batch, wl.block, wl.steps
    Hq, Hkv, d = wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    elt = 2 if wl.dtype == "bf16" else 4
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    print(f"[bench] generating {wl.name}", file=sys.stderr, flush=True)
    inp = synth.make_host(wl)

    def dv(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    S = int(inp["seq_lens"][0])
    hd = H.heads(Hq, Hkv, d, wl.dtype)
    k_b = H.budget_tokens(S, *wl.budget)
    k_max = k_b
    cap = S + B
    # full cache with room for the appended block
    cache_k = torch.zeros((b, Hkv, cap, d), dtype=tdt, device=dev)
    cache_v = torch.zeros_like(cache_k)
    cache_k[:, :, :S] = dv(inp["k"])
    cache_v[:, :, :S] = dv(inp["v"])
    lens0 = dv(inp["seq_lens"])
    lens = lens0.clone()
    kps = torch.full((b,), k_b, dtype=torch.int32, device=dev)
    pools = [[torch.zeros((b, Hkv, k_max + B, d), dtype=tdt, device=dev) for _ in range(2)]
             for _ in range(2)]                       # [active/idle][k, v]
    n_pool = [torch.full((b,), k_b, dtype=torch.int32, device=dev),
              torch.zeros((b,), dtype=torch.int32, device=dev)]
    q_sel, q_next = dv(inp["q_sel"]), dv(inp["q_next"])
    q_steps, blk_k, blk_v = dv(inp["q"]), dv(inp["blk_k"]), dv(inp["blk_v"])
    done_k, done_v = dv(inp["done_k"]), dv(inp["done_v"])
    out = torch.empty((b, B, Hq, d), dtype=tdt, device=dev)

    # initial selection (the prefill-time top-k) into the first active pool
    kv_cache = H.kv_view(cache_k, cache_v, lens, S)
    ws_sel = H.workspace(H.select_workspace(hd, b, S), dev)
    idx = torch.empty((b, Hkv, k_max), dtype=torch.int32, device=dev)
    H.select(hd, b, B, q_sel, kv_cache, kps, k_max, idx, ws_sel)
    H.gather(hd, b, kv_cache, idx, kps, k_max, H.pool_view(*pools[0]))
    torch.cuda.synchronize()

    s_main = torch.cuda.Stream(device=dev)
    s_retr = s_main if args.serial else torch.cuda.Stream(device=dev)
    ws = H.workspace(H.decode_block_workspace(hd, b, B, S, k_max), dev)
    state = {"a": 0}

    def step():
        a = state["a"]
        i = 1 - a
        with torch.cuda.stream(s_main):
            lens.copy_(lens0)          # every block sees the same S (one batch)
        cache = H.pool_view(cache_k, cache_v)
        layer = H.Layer(cache, H.pool_view(*pools[a]), H.pool_view(*pools[i]),
                        q_steps.data_ptr(), blk_k.data_ptr(), blk_v.data_ptr(),
                        done_k.data_ptr(), done_v.data_ptr(), q_next.data_ptr(),
                        out.data_ptr(), 0)
        H.decode_block(hd, [layer], b, B, T, lens, S, n_pool[a], k_max + B, n_pool[i], kps,
                       k_max, args.dense, ws, s_main, s_retr)
        state["a"] = i

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    if args.graph:
        # the whole block (lengths reset, both streams, join, append) as one
        # graph per pool parity; the timed loop replays them alternately
        graphs = []
        for _ in range(2):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=s_main):
                step()
            graphs.append(g)
        torch.cuda.synchronize()

        def step():   # noqa: F811 (the replaying step replaces the eager one)
            with torch.cuda.stream(s_main):   # the timing events are on s_main
                graphs[state["a"]].replay()
            state["a"] = 1 - state["a"]
        for _ in range(2):
            step()
        torch.cuda.synchronize()
    print(f"[bench] timing {args.steps} pipelined blocks", file=sys.stderr, flush=True)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(s_main)
    for _ in range(args.steps):
        step()
    ev1.record(s_main)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_block = ev0.elapsed_time(ev1) / args.steps
    ms_block_wall = wall * 1e3 / args.steps

    # ---- isolated kernels, HIP events on the stream they run on --------------
    def timed(fn, reps, stream):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        for _ in range(min(3, reps)):
            fn()
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    a = state["a"]
    n_ctx = int(n_pool[a][0].item())
    pool_kv = H.kv_view(pools[a][0], pools[a][1], n_pool[a], k_max + B)
    ctx_kv = kv_cache if args.dense else pool_kv
    ctx_rows = S if args.dense else n_ctx
    max_ctx = S if args.dense else k_max + B
    ws_att = H.workspace(H.block_attn_workspace(hd, b, B, max_ctx), dev)
    lens.copy_(lens0)
    torch.cuda.synchronize()
    # the denoising phase alone: steps x T launches back to back on s_main,
    # each step's own queries and block KV
    n_att = args.steps * T

    def denoise_phase():
        for j in range(n_att):
            t = j % T
            H.block_attn(hd, b, B, q_steps[t], ctx_kv, blk_k[t], blk_v[t], out, ws_att,
                         stream=s_main)
    with torch.cuda.stream(s_main):
        ms_attn = timed(denoise_phase, 1, s_main) / n_att
        # per-launch spread: an event between consecutive launches
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(min(n_att, 256) + 1)]
        evs[0].record(s_main)
        for j in range(len(evs) - 1):
            t = j % T
            H.block_attn(hd, b, B, q_steps[t], ctx_kv, blk_k[t], blk_v[t], out, ws_att,
                         stream=s_main)
            evs[j + 1].record(s_main)
        torch.cuda.synchronize()
        per = np.array([evs[j].elapsed_time(evs[j + 1]) for j in range(len(evs) - 1)])
        # cold: one launch right after reading 512 MiB of other data, so that
        # neither L2 nor the last-level cache holds the pool (a read leaves no
        # dirty lines whose write-back the timed launch would pay for)
        flush = torch.ones(512 << 20, dtype=torch.uint8, device=dev)
        cold = []
        for j in range(10):
            flush.max()
            c0 = torch.cuda.Event(enable_timing=True)
            c1 = torch.cuda.Event(enable_timing=True)
            c0.record(s_main)
            H.block_attn(hd, b, B, q_steps[j % T], ctx_kv, blk_k[j % T], blk_v[j % T], out,
                         ws_att, stream=s_main)
            c1.record(s_main)
            torch.cuda.synchronize()
            cold.append(c0.elapsed_time(c1))
        del flush
        ms_sel = timed(lambda: H.select(hd, b, B, q_next, kv_cache, kps, k_max, idx, ws_sel,
                                        stream=s_main), max(5, args.reps // 3), s_main)
        ms_gat = timed(lambda: H.gather(hd, b, kv_cache, idx, kps, k_max,
                                        H.pool_view(*pools[1 - a]), stream=s_main),
                       args.reps, s_main)

    keys = ctx_rows + B
    attn_flops = 4.0 * (Hq // Hkv) * B * d * keys * b * Hkv
    # K and V rows of context + block, plus the queries read and outputs written
    attn_bytes = 2.0 * d * elt * keys * b * Hkv + 2.0 * b * B * Hq * d * elt
    attn_tflops = attn_flops / (ms_attn * 1e-3) / 1e12
    attn_gbps = attn_bytes / (ms_attn * 1e-3) / 1e9
    sel_bytes = float(S) * d * elt * b * Hkv
    sel_gbps = sel_bytes / (ms_sel * 1e-3) / 1e9
    gat_bytes = 4.0 * d * elt * k_b * b * Hkv
    gat_gbps = gat_bytes / (ms_gat * 1e-3) / 1e9
    steps_per_s = T / (ms_block * 1e-3)
    peak = BF16_MFMA_PEAK_TFLOPS if wl.dtype == "bf16" else FP32_VECTOR_PEAK_TFLOPS

    res = {
        "metric": "denoise steps/s (sparse block attn) + selection scan HBM GB/s, % of roofline",
        "value": round(steps_per_s, 3),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_block, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "f32",
        "data": "synthetic (seeded N(0,1) with planted heavy hitters and sinks)",
        "config": {"workload": wl.name, "batch": b, "seq_len": S, "block": B, "steps": T,
                   "q_heads": Hq, "kv_heads": Hkv, "head_dim": d, "budget_tokens": k_b,
                   "layers": 1, "mode": "dense" if args.dense else "sparse",
                   "graph": bool(args.graph), "streams": 1 if args.serial else 2,
                   "step": ("one block on one stream: next-block selection, T denoising "
                            "steps, append, swap" if args.serial else
                            "one pipelined block: next-block selection on a second stream "
                            "overlapped with T denoising steps, join, append, swap")},
        # B*G query rows per KV head give 4*B*G*d flops per 4*d bytes of bf16 K+V
        # (B*G = 128: 128 flop/B, below the 2.5 PFLOP/s / 8 TB/s ridge of 312):
        # the kernel is bound by HBM, and its MFMA rate is reported beside.
        "roofline": {"bound": "hbm", "achieved": round(attn_gbps, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(attn_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": profiled_traffic(wl, args.dense),
                     "kernel": "herald_block_attn (attention + split combine)",
                     "ms": round(ms_attn, 5), "launches_timed": n_att,
                     "bytes_per_launch": attn_bytes,
                     "flops_per_launch": attn_flops, "TFLOPs": round(attn_tflops, 2),
                     "mfma_frac": round(attn_tflops / peak, 4),
                     "ms_p10_p50_p90": [round(float(np.percentile(per, x)), 5)
                                        for x in (10, 50, 90)],
                     "cold_ms_p50": round(float(np.median(cold)), 5),
                     "cold_frac": round(attn_bytes / (np.median(cold) * 1e-3) / 1e9
                                        / HBM_PEAK_GBPS, 4)},
        "selection": {"ms": round(ms_sel, 5), "k_bytes": sel_bytes,
                      "scan_GBps": round(sel_gbps, 1),
                      "frac_hbm": round(sel_gbps / HBM_PEAK_GBPS, 4)},
        "gather": {"ms": round(ms_gat, 5), "bytes": gat_bytes,
                   "GBps": round(gat_gbps, 1)},
        "pipeline": {"ms_per_block_events": round(ms_block, 4),
                     "ms_per_block_wall": round(ms_block_wall, 4),
                     "tokens_per_s": round(b * B / (ms_block * 1e-3), 1),
                     "attention_only_ms": round(T * ms_attn, 4)},
        "device": torch.cuda.get_device_name(0),
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(wl, inp, k_b, args.cpu_seqs or b,
                                           args.cpu_steps or T, args.dense)
    print(json.dumps(res), flush=True)


PROFILES = os.path.join(ROOT, "profiles")


def kernel_source_digest() -> str:
    """sha256 of the attention kernel's source files (a traffic figure taken
    from hardware counters holds only for the source it was measured on)."""
    import hashlib
    h = hashlib.sha256()
    for f in ("attn.hip", "common.h"):
        with open(os.path.join(ROOT, "paper_2606_21633_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def profiled_traffic(wl, dense):
    """HBM bytes per attention launch from the committed counter summary of
    this workload (FETCH_SIZE + WRITE_SIZE, calibrated on a plain copy), or
    None when there is none or the kernel source changed since."""
    if dense or wl.name != "8B-layer bf16 16x(32q,8kv) d128 S32768 B32 T32":
        return None
    path = os.path.join(PROFILES, "block_attn_layer32k_traffic.txt")
    try:
        kv = {}
        with open(path) as fh:
            for line in fh:
                if line.startswith("traffic:"):
                    for tok in line.split()[1:]:
                        k, _, v = tok.partition("=")
                        kv[k] = v
        if kv.get("source_sha256") != kernel_source_digest():
            return None
        return float(kv["bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def copy_calibration(mib: int):
    """A plain streaming copy of known size (dst = src * 1, fp32, 5 times) for
    scaling the FETCH_SIZE / WRITE_SIZE counters to bytes."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(5):
        torch.mul(src, 1.0, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration": True, "bytes_read_per_launch": n * 4,
                      "bytes_written_per_launch": n * 4, "launches": 5}), flush=True)


def read_calibration(mib: int):
    """A plain streaming read of known size (a sum over fp32, 5 times): the
    FETCH_SIZE of a kernel that only reads, beside the copy's."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    for _ in range(5):
        src.sum()
    torch.cuda.synchronize()
    print(json.dumps({"read_calibration": True, "bytes_read_per_launch": n * 4,
                      "launches": 5}), flush=True)


def _timed(fn, reps, stream):
    import torch
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    for _ in range(3):
        fn()
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def bench_ragged(args):
    """Ragged paged serving batch (64 sequences, 8K-64K tokens, 16-token pages
    in shuffled order, B=16, T=16, 5% budget per sequence). A step: paged
    selection and gather of every sequence's pool, then T denoising steps."""
    import torch
    from paper_2606_21633_amd import herald as H
    from paper_2606_21633_amd import synth
    dev = "cuda:0"
    wl = synth.RAGGED_PAGED
    b, B, T = wl.batch, wl.block, wl.steps
    Hq, Hkv, d = wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    print(f"[bench] generating {wl.name}", file=sys.stderr, flush=True)
    inp = synth.make_host(wl)

    def dv(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    lens_h = inp["seq_lens"]
    S_max = int(lens_h.max())
    kps_h = np.array([H.budget_tokens(int(x), *wl.budget) for x in lens_h], np.int32)
    k_max = int(kps_h.max())
    hd = H.heads(Hq, Hkv, d, "bf16")
    pk_, pv_, pt = dv(inp["pages_k"]), dv(inp["pages_v"]), dv(inp["page_table"])
    lens, kps = dv(lens_h), dv(kps_h)
    kv = H.kv_view(pk_, pv_, lens, S_max, page_table=pt)
    q_sel, q_steps = dv(inp["q_sel"]), dv(inp["q"])
    blk_k, blk_v = dv(inp["blk_k"]), dv(inp["blk_v"])
    idx = torch.empty((b, Hkv, k_max), dtype=torch.int32, device=dev)
    pool_k = torch.zeros((b, Hkv, k_max, d), dtype=torch.bfloat16, device=dev)
    pool_v = torch.zeros_like(pool_k)
    pool = H.kv_view(pool_k, pool_v, kps, k_max)
    out = torch.empty((b, B, Hq, d), dtype=torch.bfloat16, device=dev)
    ws_sel = H.workspace(H.select_workspace(hd, b, S_max), dev)
    ws_att = H.workspace(H.block_attn_workspace(hd, b, B, k_max), dev)
    s = torch.cuda.current_stream()

    def step():
        H.select(hd, b, B, q_sel, kv, kps, k_max, idx, ws_sel)
        H.gather(hd, b, kv, idx, kps, k_max, H.pool_view(pool_k, pool_v))
        for t in range(T):
            H.block_attn(hd, b, B, q_steps[t], pool, blk_k[t], blk_v[t], out, ws_att)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ms_step = _timed(step, args.steps, s)
    ms_sel = _timed(lambda: H.select(hd, b, B, q_sel, kv, kps, k_max, idx, ws_sel), 10, s)
    ms_gat = _timed(lambda: H.gather(hd, b, kv, idx, kps, k_max, H.pool_view(pool_k, pool_v)),
                    20, s)
    ms_att = _timed(lambda: H.block_attn(hd, b, B, q_steps[0], pool, blk_k[0], blk_v[0], out,
                                         ws_att), 30, s)
    keys = float(np.sum(kps_h + B))
    flops = 4.0 * (Hq // Hkv) * B * d * keys * Hkv
    abytes = 2.0 * d * 2 * keys * Hkv + 2.0 * b * B * Hq * d * 2
    agbps = abytes / (ms_att * 1e-3) / 1e9
    kbytes = float(np.sum(lens_h)) * Hkv * d * 2
    res = {"metric": "denoise steps/s (sparse block attn) + selection scan HBM GB/s, % of roofline",
           "value": round(T / (ms_step * 1e-3), 3), "unit": "steps/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic (seeded N(0,1) with planted heavy hitters and sinks)",
           "config": {"workload": wl.name, "batch": b, "seq_len_total": int(np.sum(lens_h)),
                      "seq_len_range": [int(lens_h.min()), S_max], "block": B, "steps": T,
                      "page_size": wl.page_size, "step": "paged selection + gather, then T "
                      "denoising steps (same stream)"},
           "roofline": {"bound": "hbm", "achieved": round(agbps, 1), "peak": HBM_PEAK_GBPS,
                        "unit": "GB/s", "frac": round(agbps / HBM_PEAK_GBPS, 4),
                        "bytes_per_launch": abytes,
                        "traffic": None, "kernel": "herald_block_attn", "ms": round(ms_att, 5),
                        "TFLOPs": round(flops / (ms_att * 1e-3) / 1e12, 2)},
           "selection": {"ms": round(ms_sel, 5), "k_bytes": kbytes,
                         "scan_GBps": round(kbytes / (ms_sel * 1e-3) / 1e9, 1),
                         "frac_hbm": round(kbytes / (ms_sel * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4)},
           "gather": {"ms": round(ms_gat, 5)}, "device": torch.cuda.get_device_name(0)}
    print(json.dumps(res), flush=True)


def bench_xq_sweep(args):
    """Selection cost against the number x of query rows (the query-count
    trade-off of sec. IV-A.2), on the 8B-class layer: herald_select (mean of
    the B queries) and herald_select_xq for x = 1 (centre query) ... 32 (every
    block query). Each call scores all 16 x 8 x 32768 cached rows in fp64."""
    import torch
    from paper_2606_21633_amd import herald as H
    from paper_2606_21633_amd import synth
    dev = "cuda:0"
    wl = synth.LAYER_32K
    b, B = wl.batch, wl.block
    Hq, Hkv, d = wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    G = Hq // Hkv
    print(f"[bench] generating {wl.name}", file=sys.stderr, flush=True)
    inp = synth.make_host(wl)

    def dv(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    S = int(inp["seq_lens"][0])
    hd = H.heads(Hq, Hkv, d, wl.dtype)
    k_b = H.budget_tokens(S, *wl.budget)
    kk, vv, lens = dv(inp["k"]), dv(inp["v"]), dv(inp["seq_lens"])
    kv = H.kv_view(kk, vv, lens, S)
    q_sel = dv(inp["q_sel"])
    kps = torch.full((b,), k_b, dtype=torch.int32, device=dev)
    idx = torch.empty((b, Hkv, k_b), dtype=torch.int32, device=dev)
    s = torch.cuda.current_stream()
    kbytes = float(S) * d * 2 * b * Hkv
    rows = []
    ws = H.workspace(H.select_workspace(hd, b, S), dev)
    ms = _timed(lambda: H.select(hd, b, B, q_sel, kv, kps, k_b, idx, ws), args.reps, s)
    rows.append({"x": "mean", "ms": round(ms, 4), "scan_GBps": round(kbytes / ms / 1e6, 1)})
    del ws
    per_x = {}
    for x in (1, 2, 4, 8, 16, 32):
        ws = H.workspace(H.select_xq_workspace(hd, b, x, S), dev)
        reps = max(3, args.reps // x)
        ms = _timed(lambda: H.select_xq(hd, b, B, x, q_sel, kv, kps, k_b, idx, ws), reps, s)
        flops = 2.0 * x * G * d * S * b * Hkv
        per_x[x] = ms
        rows.append({"x": x, "ms": round(ms, 4), "scan_GBps": round(kbytes / ms / 1e6, 1),
                     "fp64_TFLOPs": round(flops / ms / 1e9, 2),
                     "workspace_GB": round(ws.numel() / 1e9, 3)})
        del ws
        torch.cuda.empty_cache()
    # the paper's selection: centre query, block n's draft KV as normalisation
    # tail, plus the attention output handed to the FFN
    ws = H.workspace(H.select_xq_workspace(hd, b, 1, S), dev)
    dk = torch.randn((b, B, Hkv, d), device=dev).to(torch.bfloat16)
    dvv = torch.randn((b, B, Hkv, d), device=dev).to(torch.bfloat16)
    o = torch.empty((b, 1, Hq, d), dtype=torch.bfloat16, device=dev)
    ms_d = _timed(lambda: H.select_draft(hd, b, B, 1, q_sel, kv, dk, B, kps, k_b, idx, ws),
                  args.reps, s)
    ms_o = _timed(lambda: H.select_attn(hd, b, B, 1, q_sel, kv, dk, dvv, B, kps, k_b, idx, o, ws),
                  args.reps, s)
    rows.append({"x": "1 + draft tail", "ms": round(ms_d, 4),
                 "scan_GBps": round(kbytes / ms_d / 1e6, 1)})
    rows.append({"x": "1 + draft tail + attention output", "ms": round(ms_o, 4),
                 "scan_GBps": round(kbytes / ms_o / 1e6, 1),
                 "kv_bytes_GBps": round(2 * kbytes / ms_o / 1e6, 1)})
    del ws
    for r in rows:
        if isinstance(r["x"], int):
            r["speedup_vs_x32"] = round(per_x[32] / r["ms"], 2)
    res = {"metric": "selection throughput vs query count x (x = 1 over x = 32)",
           "value": round(per_x[32] / per_x[1], 3), "unit": "x", "n_gpus": 1,
           "steps": args.reps, "warmup": 3, "ms_per_step": round(per_x[1], 4),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f64",
           "data": "synthetic (seeded N(0,1) with planted heavy hitters and sinks)",
           "config": {"workload": wl.name + " selection", "batch": b, "seq_len": S,
                      "block": B, "q_heads": Hq, "kv_heads": Hkv, "head_dim": d,
                      "budget_tokens": k_b},
           "sweep": rows, "device": torch.cuda.get_device_name(0)}
    print(json.dumps(res), flush=True)


def bench_pipeline36(args):
    """Full pipelined block decode over 36 layers (bf16, 8 sequences x 65536
    tokens, 32 query / 8 KV heads, B=32, T=32, 5% budget), caches generated on
    the device. Reports decode tokens/s of the two-stream sparse pipeline next
    to dense attention (100% budget, the same kernels over the full cache) on
    the same inputs."""
    import torch
    from paper_2606_21633_amd import herald as H
    from paper_2606_21633_amd import synth
    dev = "cuda:0"
    wl = synth.PIPELINE_36L
    L, b, B, T = wl.layers, wl.batch, wl.block, wl.steps
    Hq, Hkv, d, S0 = wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.seq_len
    nblk = args.warmup + args.blocks
    cap = S0 + (2 * nblk + 1) * B
    nd = max(0, min(args.dense_layers, L))
    print(f"[bench] generating {wl.name} on the device", file=sys.stderr, flush=True)
    data = synth.make_device_layers(wl, dev, capacity=cap)
    gen = data["gen"]
    hd = H.heads(Hq, Hkv, d, "bf16")
    k_hi = H.budget_tokens(cap, *wl.budget)
    pcap = k_hi + B
    layers = []
    for l in range(L):
        u = data["u"][l]
        layers.append(dict(
            k=data["k"][l], v=data["v"][l],
            pools=[[torch.zeros((b, Hkv, pcap, d), dtype=torch.bfloat16, device=dev)
                    for _ in range(2)] for _ in range(2)],
            q=synth.device_queries(wl, u, gen, (T,), dev),
            bk=synth.device_normal(wl, gen, (T, b, B, Hkv, d), dev),
            bv=synth.device_normal(wl, gen, (T, b, B, Hkv, d), dev),
            dk=synth.device_normal(wl, gen, (b, B, Hkv, d), dev),
            dvv=synth.device_normal(wl, gen, (b, B, Hkv, d), dev),
            qn=synth.device_queries(wl, u, gen, (), dev),
            out=torch.empty((b, B, Hq, d), dtype=torch.bfloat16, device=dev)))
        if args.drafts:
            layers[-1].update(
                qd=synth.device_queries(wl, u, gen, (), dev),
                ddk=synth.device_normal(wl, gen, (b, B, Hkv, d), dev),
                ddv=synth.device_normal(wl, gen, (b, B, Hkv, d), dev),
                od=torch.empty((b, B, Hq, d), dtype=torch.bfloat16, device=dev))
    torch.cuda.synchronize()
    s_main = torch.cuda.Stream(device=dev)
    s_retr = s_main if args.serial else torch.cuda.Stream(device=dev)

    def run(dense):
        lens_h = np.full(b, S0, np.int32)
        lens = torch.from_numpy(lens_h.copy()).to(dev)
        n_pool = [torch.zeros(b, dtype=torch.int32, device=dev) for _ in range(2)]
        ws = H.workspace(H.decode_block_workspace(hd, b, B, cap, k_hi), dev)
        if not dense:   # initial selection (prefill-time top-k) into pool 0
            k0 = H.budget_tokens(S0, *wl.budget)
            kps0 = torch.full((b,), k0, dtype=torch.int32, device=dev)
            idx = torch.empty((b, Hkv, k0), dtype=torch.int32, device=dev)
            wsel = H.workspace(H.select_workspace(hd, b, S0), dev)
            for Ly in layers[nd:]:
                kv = H.kv_view(Ly["k"], Ly["v"], lens, S0)
                H.select(hd, b, B, Ly["qn"], kv, kps0, k0, idx, wsel)
                H.gather(hd, b, kv, idx, kps0, k0, H.pool_view(*Ly["pools"][0]))
            n_pool[0].fill_(k0)
        torch.cuda.synchronize()
        a, times = 0, []
        kn = torch.zeros((b,), dtype=torch.int32, device=dev)
        graphs = {}
        for n in range(nblk):
            S = int(lens_h[0])
            kn_h = H.budget_tokens(S, *wl.budget)
            kn.fill_(kn_h)
            lay = [H.Layer(H.pool_view(Ly["k"], Ly["v"]), H.pool_view(*Ly["pools"][a]),
                           H.pool_view(*Ly["pools"][1 - a]), Ly["q"].data_ptr(),
                           Ly["bk"].data_ptr(), Ly["bv"].data_ptr(), Ly["dk"].data_ptr(),
                           Ly["dvv"].data_ptr(), Ly["qn"].data_ptr(), Ly["out"].data_ptr(), 0,
                           int(l < nd)) for l, Ly in enumerate(layers)]
            for Lr, Ly in zip(lay, layers):
                Lr.select_x = args.select_x
                if args.drafts:
                    Lr.q_draft, Lr.draft_k = Ly["qd"].data_ptr(), Ly["ddk"].data_ptr()
                    Lr.draft_v, Lr.out_draft = Ly["ddv"].data_ptr(), Ly["od"].data_ptr()
            torch.cuda.synchronize()
            if args.graph and n >= args.warmup and a not in graphs:
                # one graph per pool parity, host bounds set to the run's maxima
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g, stream=s_main):
                    H.decode_block(hd, lay, b, B, T, lens, cap - B, n_pool[a], pcap,
                                   n_pool[1 - a], kn, k_hi, dense, ws, s_main, s_retr)
                graphs[a] = (g, lay)
                torch.cuda.synchronize()
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(s_main)
            if a in graphs:
                with torch.cuda.stream(s_main):
                    graphs[a][0].replay()
            else:
                H.decode_block(hd, lay, b, B, T, lens, S, n_pool[a], pcap, n_pool[1 - a], kn,
                               kn_h, dense, ws, s_main, s_retr)
            e1.record(s_main)
            torch.cuda.synchronize()
            print(f"[bench] {'dense' if dense else 'sparse'} block {n}: "
                  f"{e0.elapsed_time(e1):.2f} ms", file=sys.stderr, flush=True)
            if n >= args.warmup:
                times.append(e0.elapsed_time(e1))
            lens_h += B
            a = 1 - a
        return float(np.mean(times))

    ms_sparse = run(False)
    ms_dense = run(True)
    tok = b * B
    res = {"metric": "decode tokens/s (36-layer pipelined block decode)",
           "value": round(tok / (ms_sparse * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1,
           "steps": args.blocks, "warmup": args.warmup, "ms_per_step": round(ms_sparse, 3),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic, generated on the device (seeded torch generator)",
           "config": {"workload": wl.name, "layers": L, "batch": b, "seq_len": S0, "block": B,
                      "steps": T, "budget": "5%", "dense_layers": nd,
                      "drafts": bool(args.drafts), "select_x": args.select_x,
                      "graph": bool(args.graph), "streams": 1 if args.serial else 2,
                      "step": "one block: next-block selection of "
                      "all layers on the retrieval stream, T x L denoising steps on the main "
                      "stream, join, append, swap"},
           "dense": {"ms_per_block": round(ms_dense, 3),
                     "tokens_per_s": round(tok / (ms_dense * 1e-3), 1)},
           "speedup_vs_dense": round(ms_dense / ms_sparse, 3),
           "device": torch.cuda.get_device_name(0)}
    print(json.dumps(res), flush=True)


def cpu_baseline(wl, inp, k_b, nseq, nsteps, dense):
    """The oracle, as it stands, on the same step: for `nseq` sequences the
    selection + gather of the next pool and `nsteps` denoising steps, scaled
    to one block of the whole batch (batch x (selection + T attention
    steps)) and reported in denoise steps/s. By default the sample is the
    whole block, so nothing is extrapolated."""
    import oracle
    S = int(inp["seq_lens"][0])
    t_sel = t_att = 0.0
    for s in range(nseq):
        K = inp["k"][s, :, :S]
        V = inp["v"][s, :, :S]
        t0 = time.perf_counter()
        if dense:
            pk, pv = K, V
        else:
            idx, _, _, _ = oracle.select(inp["q_next"][s], K, k_b)
            pk, pv = oracle.gather(K, idx), oracle.gather(V, idx)
        t1 = time.perf_counter()
        for t in range(nsteps):
            oracle.attn(inp["q"][t][s], pk, pv, inp["blk_k"][t][s], inp["blk_v"][t][s])
        t2 = time.perf_counter()
        t_sel += t1 - t0
        t_att += t2 - t1
    block_s = (t_sel / nseq + t_att / (nseq * nsteps) * wl.steps) * wl.batch
    res = {"value": round(wl.steps / block_s, 6), "unit": "steps/s",
           "cores": oracle.threads(), "kind": "oracle",
           "sample": f"{nseq} of {wl.batch} sequences x (selection+gather and {nsteps} of "
                     f"{wl.steps} attention steps), scaled to one block of the batch",
           "seconds": round(t_sel + t_att, 2)}
    # the same oracle on one core: one sequence, its selection + gather and eight
    # attention steps, scaled the same way
    n_all = oracle.threads()
    oracle.set_threads(1)
    try:
        K, V = inp["k"][0, :, :S], inp["v"][0, :, :S]
        t0 = time.perf_counter()
        if dense:
            pk, pv = K, V
        else:
            idx, _, _, _ = oracle.select(inp["q_next"][0], K, k_b)
            pk, pv = oracle.gather(K, idx), oracle.gather(V, idx)
        t1 = time.perf_counter()
        n1 = min(8, wl.steps)
        for t in range(n1):
            oracle.attn(inp["q"][t][0], pk, pv, inp["blk_k"][t][0], inp["blk_v"][t][0])
        t2 = time.perf_counter()
    finally:
        oracle.set_threads(n_all)
    block1 = ((t1 - t0) + (t2 - t1) / n1 * wl.steps) * wl.batch
    res["single_core"] = {"value": round(wl.steps / block1, 6), "unit": "steps/s", "cores": 1,
                          "sample": f"1 of {wl.batch} sequences x (selection+gather and {n1} "
                                    f"of {wl.steps} attention steps), scaled to one block of "
                                    f"the batch", "seconds": round(t2 - t0, 2)}
    return res


if __name__ == "__main__":
    main()
