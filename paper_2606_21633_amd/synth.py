"""Seeded synthetic inputs for the sparse block-decode hot path.

This module holds the workload shapes and the random input recipe only; it
contains none of the method's arithmetic (no scoring, budget or attention),
so that the GPU library and the CPU oracle can both be fed from it.

Recipe (stand-in for the paper's LongBench prompts and model activations):

* Every tensor is i.i.d. N(0, 1) in float32. The slice of each tensor that
  belongs to sequence b (selection queries, per-step block queries, K cache,
  V cache, per-step block K/V, completed block K/V, next-block selection
  queries) and the planting draws of sequence b come from their own PCG64
  stream ``numpy.random.default_rng([seed, tensor, b])``. Device-resident
  workloads too large for host memory use a seeded ``torch.Generator`` on
  the device instead.
* Heavy hitters: for every (sequence, KV head) a random unit vector u (from
  N(0, I_d), normalised) is drawn. 3u is added to a random 5% of the cached
  keys (round half-up of 0.05 S positions, drawn without replacement from
  [4, S)) and to every query row of the query heads of that KV head; 6u is
  added to positions 0..3 (attention sinks). The ``spans`` recipe instead
  puts the 3u bias on 8 non-overlapping contiguous spans of random length
  64..512. V and the block's own K/V are left unbiased.
* Biases are added in float32; bfloat16 workloads are then rounded to
  nearest-even bfloat16.
* Ragged workloads draw each sequence length uniformly from [S_lo, S_hi];
  paged ones store the cache as ``[page][Hkv][page_size][d]`` with the
  physical page order a seeded random permutation.
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str            # "f32" or "bf16"
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    seq_len: int          # S (or S_hi for ragged workloads)
    block: int            # B
    steps: int            # T
    budget: tuple = (1, 20)   # fraction num/den of the prefix kept per KV head
    planting: str = "uniform"  # "uniform" (5% of keys) or "spans"
    seq_len_lo: int = 0   # >0: ragged lengths uniform in [seq_len_lo, seq_len]
    page_size: int = 0    # >0: paged cache with this many tokens per page
    layers: int = 1
    seed: int = 0

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five workloads the hot path is measured and checked on.
TINY_F32 = Workload("tiny-fp32 1x(8q,2kv) d64 S4096 B4 T4", "f32", 1, 8, 2, 64,
                    4096, 4, 4, seed=1)
LAYER_32K = Workload("8B-layer bf16 16x(32q,8kv) d128 S32768 B32 T32", "bf16", 16,
                     32, 8, 128, 32768, 32, 32, seed=2)
LONG_128K = Workload("long bf16 4x(32q,8kv) d128 S131072 B32 T16 spans", "bf16", 4,
                     32, 8, 128, 131072, 32, 16, planting="spans", seed=3)
RAGGED_PAGED = Workload("ragged-paged bf16 64x(32q,8kv) d128 S8K-64K B16 T16 p16",
                        "bf16", 64, 32, 8, 128, 65536, 16, 16, seq_len_lo=8192,
                        page_size=16, seed=4)
PIPELINE_36L = Workload("pipelined 36L bf16 8x(32q,8kv) d128 S65536 B32 T32", "bf16",
                        8, 32, 8, 128, 65536, 32, 32, layers=36, seed=5)

WORKLOADS = {w.name: w for w in (TINY_F32, LAYER_32K, LONG_128K, RAGGED_PAGED,
                                 PIPELINE_36L)}


def _planted_count(S: int) -> int:
    """Number of heavy-hitter positions: 5% of S, rounded half-up."""
    return (S + 10) // 20


def seq_lens(wl: Workload, rng: np.random.Generator) -> np.ndarray:
    if wl.seq_len_lo > 0:
        return rng.integers(wl.seq_len_lo, wl.seq_len, size=wl.batch,
                            endpoint=True).astype(np.int32)
    return np.full(wl.batch, wl.seq_len, np.int32)


def _unit(rng, d):
    u = rng.standard_normal(d)
    return (u / np.linalg.norm(u)).astype(np.float32)


def _spans(rng, S, count=8, lo=64, hi=512):
    """Non-overlapping spans inside [4, S) by rejection."""
    taken = np.zeros(S, bool)
    taken[:4] = True
    out = []
    tries = 0
    while len(out) < count and tries < 10000:
        tries += 1
        ln = int(rng.integers(lo, hi, endpoint=True))
        if ln >= S - 4:
            continue
        st = int(rng.integers(4, S - ln + 1))
        if taken[st:st + ln].any():
            continue
        taken[st:st + ln] = True
        out.append((st, ln))
    return out


def _to_dtype(x: np.ndarray, dtype: str):
    """float32 array -> float32 array, or bfloat16 bits (uint16) by RNE."""
    if dtype == "f32":
        return np.ascontiguousarray(x, np.float32)
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


_TAGS = dict(q_sel=0, q=1, k=2, v=3, blk_k=4, blk_v=5, done_k=6, done_v=7, q_next=8,
             plant=9, lens=10, pages=11)


def _child(seed: int, tag: str, b: int = 0) -> np.random.Generator:
    """Independent PCG64 stream keyed by (seed, tensor, sequence)."""
    return np.random.default_rng([seed, _TAGS[tag], b])


def _plant_plan(wl: Workload, seed: int, i: int, S: int):
    """Heavy-hitter draws of sequence i: per KV head a unit vector u and the
    key positions that get +3u (positions 0..3 get +6u)."""
    rng = _child(seed, "plant", i)
    us, rows = [], []
    for _ in range(wl.num_kv_heads):
        u = _unit(rng, wl.head_dim)
        if wl.planting == "spans":
            pos = np.concatenate([np.arange(st, st + ln) for st, ln in _spans(rng, S)]
                                 or [np.zeros(0, np.int64)])
        elif S > 4:
            n = _planted_count(S)
            pos = rng.choice(S - 4, size=min(n, S - 4), replace=False) + 4
        else:
            pos = np.zeros(0, np.int64)
        us.append(u)
        rows.append(pos)
    return np.stack(us), rows


def make_host(wl: Workload, seed: int | None = None, threads: int = 8) -> dict:
    """Host (numpy) inputs for one layer of ``wl``.

    Every tensor slice of sequence b is drawn from its own PCG64 stream keyed
    by (seed, tensor, b), so the draws run on several threads and are still
    reproducible. Returns a dict with
      seq_lens [b] int32,
      q_sel [b][B][Hq][d], q [T][b][B][Hq][d],
      k, v: contiguous [b][Hkv][S_max][d] (zero rows beyond each length), or,
            for paged workloads, pages_k/pages_v [n_pages][Hkv][P][d] and
            page_table [b][max_pages] int32,
      blk_k, blk_v [T][b][B][Hkv][d], done_k, done_v [b][B][Hkv][d],
      q_next [b][B][Hq][d] (the following block's selection queries).
    Float arrays are float32, or uint16 holding bfloat16 bits.
    """
    import concurrent.futures as cf
    seed = wl.seed if seed is None else seed
    b, B, T = wl.batch, wl.block, wl.steps
    Hq, Hkv, d, G = wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.group
    lens = seq_lens(wl, _child(seed, "lens"))
    S_max = int(lens.max())
    et = np.float32 if wl.dtype == "f32" else np.uint16
    plans = [_plant_plan(wl, seed, i, int(lens[i])) for i in range(b)]
    out = dict(seq_lens=lens,
               q_sel=np.empty((b, B, Hq, d), et), q=np.empty((T, b, B, Hq, d), et),
               blk_k=np.empty((T, b, B, Hkv, d), et), blk_v=np.empty((T, b, B, Hkv, d), et),
               done_k=np.empty((b, B, Hkv, d), et), done_v=np.empty((b, B, Hkv, d), et),
               q_next=np.empty((b, B, Hq, d), et))
    P = wl.page_size
    if P > 0:
        npg = [(int(s) + P - 1) // P for s in lens]
        total = int(sum(npg))
        perm = _child(seed, "pages").permutation(total).astype(np.int32)
        table = np.zeros((b, max(npg)), np.int32)
        starts = np.concatenate([[0], np.cumsum(npg)])
        for i in range(b):
            table[i, :npg[i]] = perm[starts[i]:starts[i + 1]]
        out["pages_k"] = np.zeros((total, Hkv, P, d), et)
        out["pages_v"] = np.zeros((total, Hkv, P, d), et)
        out["page_table"] = table
    else:
        out["k"] = np.zeros((b, Hkv, S_max, d), et)
        out["v"] = np.zeros((b, Hkv, S_max, d), et)

    def fill(task):
        name, i = task
        rng = _child(seed, name, i)
        u, rows = plans[i]
        S = int(lens[i])
        if name in ("k", "v"):
            x = rng.standard_normal((Hkv, S, d), dtype=np.float32)
            if name == "k":
                for h in range(Hkv):
                    x[h, rows[h]] += 3 * u[h]
                    x[h, :min(4, S)] += 6 * u[h]
            x = _to_dtype(x, wl.dtype)
            if P > 0:
                pad = np.zeros((Hkv, npg[i] * P, d), et)
                pad[:, :S] = x
                pages = np.ascontiguousarray(pad.reshape(Hkv, npg[i], P, d).transpose(1, 0, 2, 3))
                out["pages_" + name][table[i, :npg[i]]] = pages
            else:
                out[name][i, :, :S] = x
            return
        tgt = out[name]
        sl = (slice(None), i) if name in ("q", "blk_k", "blk_v") else (i,)
        x = rng.standard_normal(tgt[sl].shape, dtype=np.float32)
        if name in ("q_sel", "q", "q_next"):
            x += 3 * np.repeat(u, G, axis=0)          # [Hq][d], broadcast over rows
        tgt[sl] = _to_dtype(x, wl.dtype)

    names = ("q_sel", "q", "k", "v", "blk_k", "blk_v", "done_k", "done_v", "q_next")
    tasks = [(n, i) for n in names for i in range(b)]
    with cf.ThreadPoolExecutor(threads) as ex:
        list(ex.map(fill, tasks))
    return out


def make_device_layers(wl: Workload, device, seed: int | None = None,
                       capacity: int | None = None):
    """Device-resident inputs for a multi-layer workload (too large for host
    memory), drawn with a seeded torch generator on ``device``.

    The same recipe as ``make_host`` (N(0,1), 3u heavy hitters on 5% of keys
    and on all queries of the group, 6u sinks, bfloat16 RNE), layer by layer.
    Returns a dict of lists (one entry per layer): k, v caches
    [b][Hkv][capacity][d] (rows beyond seq_len are zero), q_sel, and the
    per-layer biases u [b][Hkv][d] so that per-step queries drawn later get the
    same heavy-hitter direction.
    """
    import torch
    seed = wl.seed if seed is None else seed
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    b, Hkv, d, G, S = wl.batch, wl.num_kv_heads, wl.head_dim, wl.group, wl.seq_len
    cap = capacity or S
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    n_plant = _planted_count(S)
    out = dict(k=[], v=[], u=[])
    for _ in range(wl.layers):
        k = torch.zeros((b, Hkv, cap, d), dtype=dt, device=device)
        v = torch.zeros((b, Hkv, cap, d), dtype=dt, device=device)
        u = torch.randn((b, Hkv, d), generator=gen, device=device)
        u = u / u.norm(dim=-1, keepdim=True)
        for i in range(b):
            kk = torch.randn((Hkv, S, d), generator=gen, device=device)
            # 5% heavy hitters per head in [4, S), then the sinks
            pos = torch.argsort(torch.rand((Hkv, S - 4), generator=gen, device=device),
                                dim=1)[:, :n_plant] + 4
            bias = torch.zeros((Hkv, S), device=device)
            bias.scatter_(1, pos, 3.0)
            bias[:, :4] = 6.0
            kk += bias[:, :, None] * u[i][:, None, :]
            k[i, :, :S] = kk.to(dt)
            v[i, :, :S] = torch.randn((Hkv, S, d), generator=gen, device=device).to(dt)
            del kk, bias, pos
        out["k"].append(k)
        out["v"].append(v)
        out["u"].append(u)
    out["gen"] = gen
    return out


def device_queries(wl: Workload, u, gen, shape_prefix, device):
    """Queries [*shape_prefix][b][B][Hq][d] with the 3u bias of each group."""
    import torch
    b, B, Hq, d, G = wl.batch, wl.block, wl.num_q_heads, wl.head_dim, wl.group
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    q = torch.randn((*shape_prefix, b, B, Hq, d), generator=gen, device=device)
    q += 3.0 * u.repeat_interleave(G, dim=1)[:, None, :, :]
    return q.to(dt)


def device_normal(wl: Workload, gen, shape, device):
    import torch
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    return torch.randn(shape, generator=gen, device=device).to(dt)
