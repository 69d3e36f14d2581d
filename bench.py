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
kernel (block attention, bf16 MFMA), timed with HIP events on its stream; the
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
                    choices=["layer32k", "long128k", "tiny"])
    ap.add_argument("--dense", action="store_true",
                    help="denoise over the full cache (GPU-only dense baseline)")
    ap.add_argument("--reps", type=int, default=30, help="isolated kernel timing reps")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seqs", type=int, default=0,
                    help="sequences in the CPU oracle sample (0: the whole batch)")
    ap.add_argument("--cpu-steps", type=int, default=0,
                    help="attention steps per sampled sequence (0: all T)")
    return ap.parse_args()


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on one GPU only: the hot path is measured on a single "
              "MI355X and this build has no multi-GPU path (see DESIGN.md, sharding).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_21633_amd import herald as H
    from paper_2606_21633_amd import synth

    dev = "cuda:0"
    torch.cuda.set_device(0)
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
    s_retr = torch.cuda.Stream(device=dev)
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
        for _ in range(3):
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
    with torch.cuda.stream(s_main):
        ms_attn = timed(lambda: H.block_attn(hd, b, B, q_steps[0], ctx_kv, blk_k[0],
                                             blk_v[0], out, ws_att, stream=s_main),
                        args.reps, s_main)
        ms_sel = timed(lambda: H.select(hd, b, B, q_next, kv_cache, kps, k_max, idx, ws_sel,
                                        stream=s_main), max(5, args.reps // 3), s_main)
        ms_gat = timed(lambda: H.gather(hd, b, kv_cache, idx, kps, k_max,
                                        H.pool_view(*pools[1 - a]), stream=s_main),
                       args.reps, s_main)

    keys = ctx_rows + B
    attn_flops = 4.0 * (Hq // Hkv) * B * d * keys * b * Hkv
    attn_bytes = 2.0 * d * elt * keys * b * Hkv
    attn_tflops = attn_flops / (ms_attn * 1e-3) / 1e12
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
                   "step": "one pipelined block: next-block selection on a second stream "
                           "overlapped with T denoising steps, join, append, swap"},
        "roofline": {"bound": "mfma", "achieved": round(attn_tflops, 2), "peak": peak,
                     "unit": "TFLOP/s", "frac": round(attn_tflops / peak, 4),
                     "traffic": None, "kernel": "herald_block_attn (attention + split "
                     "combine)", "ms": round(ms_attn, 5), "flops_per_launch": attn_flops,
                     "kv_bytes_per_launch": attn_bytes,
                     "kv_GBps": round(attn_bytes / (ms_attn * 1e-3) / 1e9, 1)},
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
    return {"value": round(wl.steps / block_s, 6), "unit": "steps/s",
            "cores": oracle.threads(), "kind": "oracle",
            "sample": f"{nseq} of {wl.batch} sequences x (selection+gather and {nsteps} of "
                      f"{wl.steps} attention steps), scaled to one block of the batch",
            "seconds": round(t_sel + t_att, 2)}


if __name__ == "__main__":
    main()
