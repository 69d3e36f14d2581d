"""GPU parity of herald_gather (bit-exact) and herald_block_attn (fp32:
1e-5 abs; bf16: 2e-2 abs after rounding the GPU output to bf16) against the
fp64 oracle on the same seeded inputs."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_21633_amd import herald as H
from paper_2606_21633_amd import synth
from tests.gpu_util import (DEV, Staged, budgets, f64, seq_kv_host, to_dev, to_host)

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}


@pytest.mark.parametrize("paged", [False, True])
@pytest.mark.parametrize("row0", [0, 5])
def test_gather_is_bitwise_row_copy(paged, row0):
    wl = synth.Workload("gather", "bf16", 4, 8, 2, 128, 3000, 4, 1, seq_len_lo=40,
                        page_size=16 if paged else 0, seed=3)
    inp = synth.make_host(wl)
    st = Staged(wl, inp)
    kps_h = budgets(inp["seq_lens"], 1, 10)
    k_max = int(kps_h.max())
    idx, kps = st.select(kps_h, k_max)
    cap = k_max + row0 + 3
    pk = torch.zeros((wl.batch, wl.num_kv_heads, cap, wl.head_dim), dtype=torch.bfloat16,
                     device=DEV)
    pv = torch.zeros_like(pk)
    H.gather(st.hd, wl.batch, st.kv, to_dev(idx), kps, k_max, H.pool_view(pk, pv), row0)
    torch.cuda.synchronize()
    pk_h, pv_h = to_host(pk), to_host(pv)
    for b in range(wl.batch):
        kh, vh = seq_kv_host(inp, b)
        k = int(kps_h[b])
        want_k = oracle.gather(kh, idx[b, :, :k])
        want_v = oracle.gather(vh, idx[b, :, :k])
        assert pk_h[b, :, row0:row0 + k].tobytes() == want_k.tobytes()
        assert pv_h[b, :, row0:row0 + k].tobytes() == want_v.tobytes()
        assert not pk_h[b, :, :row0].any() and not pk_h[b, :, row0 + k:].any()


def run_attn(dtype, batch, Hq, Hkv, d, block, n_ctx, seed=0, seqs=None, paged=False):
    """Random context (ragged n_ctx per sequence), block KV and queries;
    GPU block attention vs oracle.attn per sequence."""
    rng = np.random.default_rng(seed)
    n_ctx = np.asarray(n_ctx, np.int32)
    cap = max(1, int(n_ctx.max()))

    def rnd(shape):
        x = rng.standard_normal(shape).astype(np.float32)
        return synth._to_dtype(x, dtype)
    q = rnd((batch, block, Hq, d))
    ck = rnd((batch, Hkv, cap, d))
    cv = rnd((batch, Hkv, cap, d))
    bk = rnd((batch, block, Hkv, d))
    bv = rnd((batch, block, Hkv, d))
    hd = H.heads(Hq, Hkv, d, dtype)
    lens = to_dev(n_ctx)
    tq, tbk, tbv = map(to_dev, (q, bk, bv))
    if paged:
        # the same context rows in pages of `paged` rows, physical pages in a
        # seeded order: pages [n_pages][Hkv][P][d], page_table [batch][max_pages]
        P = int(paged)
        max_pages = (cap + P - 1) // P
        perm = rng.permutation(batch * max_pages).astype(np.int32)
        pt = perm.reshape(batch, max_pages)
        pk = np.zeros((batch * max_pages, Hkv, P, d), dtype=ck.dtype)
        pv = np.zeros_like(pk)
        for b in range(batch):
            for j in range(max_pages):
                rows = slice(j * P, min((j + 1) * P, cap))
                n = rows.stop - rows.start
                pk[pt[b, j], :, :n] = ck[b, :, rows]
                pv[pt[b, j], :, :n] = cv[b, :, rows]
        tpk, tpv, tpt = map(to_dev, (pk, pv, pt))
        ctx = H.kv_view(tpk, tpv, lens, int(n_ctx.max()), page_table=tpt)
    else:
        tck, tcv = map(to_dev, (ck, cv))
        ctx = H.kv_view(tck, tcv, lens, int(n_ctx.max()))
    out = torch.zeros_like(tq)
    ws = H.workspace(H.block_attn_workspace(hd, batch, block, int(n_ctx.max())), DEV)
    H.block_attn(hd, batch, block, tq, ctx, tbk, tbv, out, ws)
    torch.cuda.synchronize()
    got = f64(to_host(out))
    worst = 0.0
    for b in (range(batch) if seqs is None else seqs):
        n = int(n_ctx[b])
        want = oracle.attn(q[b], ck[b, :, :n], cv[b, :, :n], bk[b], bv[b])
        err = float(np.abs(got[b] - want).max())
        worst = max(worst, err)
        assert err <= TOL[dtype], f"seq {b} (n_ctx={n}): max abs err {err}"
    print(f"[attn] {dtype} b={batch} G={Hq // Hkv} d={d} B={block}: max abs err {worst:.3g}")
    return worst


def test_attn_fp32_tiny_workload_shape():
    run_attn("f32", 1, 8, 2, 64, 4, [209], seed=1)


@pytest.mark.parametrize("n_ctx", [[0, 1, 63, 64, 65, 700], [1638] * 2])
def test_attn_fp32_ragged(n_ctx):
    run_attn("f32", len(n_ctx), 8, 2, 64, 4, n_ctx, seed=2)


@pytest.mark.parametrize("G,block,d", [(4, 32, 128), (4, 16, 128), (4, 4, 128), (8, 32, 128),
                                       (1, 32, 128), (2, 8, 64), (4, 32, 64), (1, 1, 64),
                                       (4, 64, 128), (2, 64, 64), (8, 64, 128)])
def test_attn_bf16_shapes(G, block, d):
    run_attn("bf16", 3, 2 * G, 2, d, block, [0, 97, 1300], seed=G * 100 + block + d)


@pytest.mark.parametrize("n_ctx", [[1], [64], [63, 65, 127, 129], [5000, 3, 4096]])
def test_attn_bf16_ragged_tiles(n_ctx):
    run_attn("bf16", len(n_ctx), 32, 8, 128, 32, n_ctx, seed=len(n_ctx))


@pytest.mark.parametrize("block,paged", [(32, False), (16, 16)])
def test_attn_bf16_ragged_more_groups_than_cus(block, paged):
    """40 sequences of seeded ragged lengths (equal lengths and empty contexts
    among them): more workgroups than CUs, so the kernel takes the sequences
    longest context first; every output must still land on its own sequence."""
    rng = np.random.default_rng(41)
    n_ctx = rng.integers(0, 3000, size=40)
    n_ctx[[3, 17]] = 0
    n_ctx[[5, 6, 30]] = 1234
    run_attn("bf16", 40, 32, 8, 128, block, n_ctx.tolist(), seed=42, paged=paged)


def test_attn_bf16_ragged_most_ordered_groups():
    """256 sequences, the most the kernel orders by context length (its LDS
    table of lengths full), ragged contexts up to 1200 rows."""
    rng = np.random.default_rng(45)
    n_ctx = rng.integers(0, 1200, size=256)
    n_ctx[[0, 255]] = 1199
    run_attn("bf16", 256, 8, 2, 128, 16, n_ctx.tolist(), seed=46)


def test_attn_bf16_many_key_splits():
    """One sequence and one KV head over 20000 context rows: the plan splits
    the keys 128 ways, so the combine merges its partials in 16 groups."""
    run_attn("bf16", 1, 4, 1, 128, 32, [20000], seed=12)


def test_attn_bf16_layer_32k_pool_shape():
    """The denoising step of the 8B-class 32K layer: 16 sequences, 1638 pool
    rows + 32 block rows per KV head; 4 sequences checked by the oracle."""
    run_attn("bf16", 16, 32, 8, 128, 32, [1638] * 16, seed=9, seqs=[0, 5, 10, 15])


@pytest.mark.parametrize("dtype,d,P,n_ctx", [("bf16", 128, 16, [0, 1, 700, 5000]),
                                             ("bf16", 64, 8, [33, 2048, 4100]),
                                             ("f32", 64, 16, [17, 300, 1000])])
def test_attn_paged_context(dtype, d, P, n_ctx):
    """Context rows read through a page table (pages of P rows in a seeded
    physical order), e.g. dense attention over a paged cache."""
    run_attn(dtype, len(n_ctx), 16, 4, d, 32 if dtype == "bf16" else 4, n_ctx,
             seed=P + d, paged=P)


def test_attn_bf16_long_128k_pool_shape():
    """The denoising step of the 128K-context layer: 4 sequences, 6554 pool
    rows + 32 block rows per KV head, keys split 4 ways and combined; two
    sequences checked by the oracle."""
    run_attn("bf16", 4, 32, 8, 128, 32, [6554] * 4, seed=13, seqs=[0, 3])


def test_attn_bf16_dense_over_full_cache_shape():
    """Dense attention (the 100%-budget baseline) over 65536 cached rows."""
    run_attn("bf16", 2, 32, 8, 128, 32, [65536, 40000], seed=10)


def run_attn_groups(dtype, batch, groups, Hq, Hkv, d, block, n_ctx, seed=0, seqs=None):
    """groups query groups per sequence over one shared context, each with its
    own block KV: GPU herald_block_attn_groups vs oracle.attn_groups."""
    rng = np.random.default_rng(seed)
    n_ctx = np.asarray(n_ctx, np.int32)
    cap = max(1, int(n_ctx.max()))

    def rnd(shape):
        x = rng.standard_normal(shape).astype(np.float32)
        return synth._to_dtype(x, dtype)
    nb = groups * block
    q = rnd((batch, nb, Hq, d))
    ck = rnd((batch, Hkv, cap, d))
    cv = rnd((batch, Hkv, cap, d))
    bk = rnd((batch, nb, Hkv, d))
    bv = rnd((batch, nb, Hkv, d))
    hd = H.heads(Hq, Hkv, d, dtype)
    tq, tck, tcv, tbk, tbv = map(to_dev, (q, ck, cv, bk, bv))
    lens = to_dev(n_ctx)  # the view holds its device pointer: keep it alive
    ctx = H.kv_view(tck, tcv, lens, int(n_ctx.max()))
    out = torch.zeros_like(tq)
    ws = H.workspace(H.block_attn_workspace(hd, batch * groups, block, int(n_ctx.max())), DEV)
    H.block_attn_groups(hd, batch, block, groups, tq, ctx, tbk, tbv, out, ws)
    torch.cuda.synchronize()
    got = f64(to_host(out))
    worst = 0.0
    for b in (range(batch) if seqs is None else seqs):
        n = int(n_ctx[b])
        want = oracle.attn_groups(q[b], ck[b, :, :n], cv[b, :, :n], bk[b], bv[b], groups)
        err = float(np.abs(got[b] - want).max())
        worst = max(worst, err)
        assert err <= TOL[dtype], f"seq {b} (n_ctx={n}): max abs err {err}"
    print(f"[attn groups] {dtype} b={batch} groups={groups} d={d} B={block}: max abs err {worst:.3g}")
    return worst


@pytest.mark.parametrize("dtype,groups,block,n_ctx", [
    ("bf16", 2, 32, [1638, 0, 700]), ("bf16", 3, 16, [5000, 64, 1]), ("bf16", 2, 4, [300, 31]),
    ("f32", 2, 4, [209, 0]), ("f32", 3, 8, [700, 65, 1])])
def test_attn_groups_share_the_context_not_each_other(dtype, groups, block, n_ctx):
    d = 128 if dtype == "bf16" else 64
    run_attn_groups(dtype, len(n_ctx), groups, 8, 2, d, block, n_ctx, seed=groups * 10 + block)


def test_attn_groups_ragged_more_groups_than_cus():
    """24 sequences of ragged lengths, 2 query groups each (48 query groups
    over 8 KV heads, two row blocks each): the kernel runs the query groups
    longest context first, each group still attending to its own sequence's
    context and its own block rows."""
    rng = np.random.default_rng(43)
    n_ctx = rng.integers(0, 2500, size=24)
    n_ctx[[2, 11]] = 0
    n_ctx[[4, 5]] = 1500
    run_attn_groups("bf16", 24, 2, 32, 8, 128, 32, n_ctx.tolist(), seed=44)


def test_attn_groups_layer_32k_draft_step_shape():
    """The 2B-token step of the 8B-class layer: denoising and draft groups of
    32 queries over the 1638-row pool; 3 sequences checked by the oracle."""
    run_attn_groups("bf16", 16, 2, 32, 8, 128, 32, [1638] * 16, seed=12, seqs=[0, 7, 15])
