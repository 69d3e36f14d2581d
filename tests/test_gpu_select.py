"""GPU parity of herald_select against the fp64 oracle: selected indices must
be identical (ascending, -1 padded), on seeded inputs that span several
scoring chunks with ragged tails, contiguous and paged caches, every
supported group size and head dim, budget edge cases and exact ties."""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_21633_amd import herald as H
from paper_2606_21633_amd import synth
from tests.gpu_util import (DEV, Staged, assert_same_selection, boundary_gap, budgets, f64,
                            seq_kv_host, to_dev, to_host)

pytestmark = pytest.mark.gpu


def check_select(wl, inp=None, kps_h=None, k_max=None, seqs=None):
    inp = synth.make_host(wl) if inp is None else inp
    st = Staged(wl, inp)
    lens = inp["seq_lens"]
    kps_h = budgets(lens, *wl.budget) if kps_h is None else np.asarray(kps_h, np.int32)
    if k_max is None:
        k_max = int(max(1, min(kps_h.max(), lens.max())))
    got, _ = st.select(kps_h, k_max)
    near, gaps = 0, []
    for b in (range(wl.batch) if seqs is None else seqs):
        S = int(lens[b])
        k = int(min(max(kps_h[b], 0), S, k_max))
        assert (got[b, :, k:] == -1).all()
        if k == 0:
            continue
        kh, _ = seq_kv_host(inp, b)
        idx_o, shat, _, _ = oracle.select(inp["q_sel"][b], kh, k)
        for h in range(wl.num_kv_heads):
            near += assert_same_selection(got[b, h, :k], idx_o[h], shat[h], k)
            gaps.append(boundary_gap(shat[h], k))
    print(f"[select] {wl.name}: near-ties={near} min rel gap={min(gaps) if gaps else None}")
    return near


SMALL = synth.Workload("small bf16 ragged", "bf16", 3, 8, 2, 128, 5000, 4, 1,
                       seq_len_lo=700, seed=11)


def test_select_tiny_fp32_workload():
    assert check_select(synth.TINY_F32) == 0


@pytest.mark.parametrize("G,d,dtype", [(1, 64, "bf16"), (2, 128, "bf16"), (4, 128, "bf16"),
                                       (8, 64, "bf16"), (4, 64, "f32"), (2, 128, "f32")])
def test_select_group_and_dims(G, d, dtype):
    wl = SMALL.replace(name=f"G{G} d{d} {dtype}", num_q_heads=2 * G, dtype=dtype,
                       head_dim=d, seed=20 + G + d)
    assert check_select(wl) == 0


def test_select_ragged_paged():
    wl = SMALL.replace(name="paged ragged", batch=5, page_size=16, seq_len=3000,
                       seq_len_lo=17, seed=31)
    assert check_select(wl) == 0


@pytest.mark.parametrize("page_size,G", [(8, 4), (64, 8), (4096, 4), (4096, 8), (8, 1)])
def test_select_paged_page_sizes(page_size, G):
    # the page-table slice of each scoring chunk is staged per workgroup: pages
    # of 8 rows (256 per chunk), 64, and pages longer than a chunk (one entry);
    # G = 8 takes the FMA scoring kernel, G <= 4 the MFMA one
    wl = SMALL.replace(name=f"paged P{page_size} G{G}", batch=4, num_q_heads=2 * G,
                       page_size=page_size, seq_len=9000 if page_size > 2048 else 5000,
                       seq_len_lo=17, seed=40 + page_size % 97 + G)
    assert check_select(wl) == 0


@pytest.mark.parametrize("kps,k_max", [([1, 1, 1], 1), ([0, 5, 2000], 2000),
                                        ([10 ** 6, 3, 7], 4000), ([-3, 700, 699], 700),
                                        ([5000, 5000, 5000], 5000)])
def test_select_budget_edges(kps, k_max):
    inp = synth.make_host(SMALL)
    k_max = min(k_max, int(inp["seq_lens"].max()))
    assert check_select(SMALL, inp, np.array(kps), k_max) == 0


def test_select_single_row_and_tiny_sequences():
    wl = SMALL.replace(name="tiny seqs", batch=4, seq_len=3, seq_len_lo=1, seed=5)
    assert check_select(wl, kps_h=np.array([1, 1, 2, 3])) == 0


def _tie_inputs(S=3000, d=128):
    rng = np.random.default_rng(77)
    wl = synth.Workload("ties", "bf16", 2, 4, 1, d, S, 4, 1, seed=77)
    inp = synth.make_host(wl)
    k = inp["k"]
    # sequence 0: every key identical -> the lowest k indices
    k[0, 0, :] = k[0, 0, 123]
    # sequence 1: three distinct key rows repeated across every scoring chunk
    rows = k[1, 0, [10, 20, 30]].copy()
    k[1, 0, :] = rows[rng.integers(0, 3, S)]
    return wl, inp


@pytest.mark.parametrize("kk", [1, 7, 1023, 1024, 1500, 2999])
def test_select_exact_ties_go_to_lower_index(kk):
    wl, inp = _tie_inputs()
    assert check_select(wl, inp, np.array([kk, kk]), kk) == 0
    st = Staged(wl, inp)
    got, _ = st.select(np.array([kk, kk], np.int32), kk)
    np.testing.assert_array_equal(got[0, 0], np.arange(kk))


@pytest.mark.parametrize("kk", [1, 9999, 19999])
def test_select_exact_ties_beyond_lds_candidates(kk):
    # 20000 identical keys: the boundary bucket exceeds the 16384 candidates
    # the top-k kernel holds in LDS, so every digit is resolved by passes over
    # the keys in global memory, down to the exact tie
    wl, inp = _tie_inputs(S=20000)
    assert check_select(wl, inp, np.array([kk, kk]), kk) == 0
    st = Staged(wl, inp)
    got, _ = st.select(np.array([kk, kk], np.int32), kk)
    np.testing.assert_array_equal(got[0, 0], np.arange(kk))


@pytest.mark.parametrize("pos", [0, 3, 63, 64, 1023, 1024, 2047, 4095, 4096, 4999])
def test_select_dominant_key_found_anywhere(pos):
    wl = SMALL.replace(name="dominant", batch=1, seq_len=5000, seq_len_lo=0, seed=pos)
    inp = synth.make_host(wl)
    qbar = (inp["q_sel"][0].astype(np.uint32) << 16).view(np.float32).mean(0)[0]
    row = (40 * qbar / np.linalg.norm(qbar)).astype(np.float32)
    import torch as _t
    inp["k"][0, 0, pos] = _t.from_numpy(row).to(_t.bfloat16).view(_t.int16).numpy().view(np.uint16)
    st = Staged(wl, inp)
    got, _ = st.select(np.array([1], np.int32), 1)
    assert got[0, 0, 0] == pos
    assert check_select(wl, inp, np.array([1]), 1) == 0


# ---------------------------------------------------------------- x query rows


def check_select_xq(wl, x, inp=None, kps_h=None, k_max=None, seqs=None):
    inp = synth.make_host(wl) if inp is None else inp
    st = Staged(wl, inp)
    lens = inp["seq_lens"]
    kps_h = budgets(lens, *wl.budget) if kps_h is None else np.asarray(kps_h, np.int32)
    if k_max is None:
        k_max = int(max(1, min(kps_h.max(), lens.max())))
    got = st.select_xq(x, kps_h, k_max)
    near = 0
    for b in (range(wl.batch) if seqs is None else seqs):
        S = int(lens[b])
        k = int(min(max(kps_h[b], 0), S, k_max))
        assert (got[b, :, k:] == -1).all()
        if k == 0:
            continue
        kh, _ = seq_kv_host(inp, b)
        idx_o, shat = oracle.select_xq(inp["q_sel"][b], kh, k, x)
        for h in range(wl.num_kv_heads):
            near += assert_same_selection(got[b, h, :k], idx_o[h], shat[h], k)
    print(f"[select_xq] {wl.name} x={x}: near-ties={near}")
    return near


XQ = SMALL.replace(name="xq", block=32, seq_len=4500, seq_len_lo=900, seed=13)


@pytest.mark.parametrize("x", [1, 2, 3, 4, 5, 8, 32])
def test_select_xq_rows_g4(x):
    # score rows x * 4: 4 (matrix-core scan with the rows as heads), 8, 12,
    # 16, 20, 32, 128 (score-row scan, 1 to 8 groups of 16)
    wl = XQ.replace(name=f"xq x{x}", num_q_heads=8, seed=50 + x)
    assert check_select_xq(wl, x) == 0


@pytest.mark.parametrize("G,d,dtype,x", [(1, 64, "bf16", 1), (1, 64, "bf16", 3), (2, 128, "bf16", 2),
                                         (2, 64, "f32", 5), (4, 128, "f32", 4), (8, 64, "bf16", 7),
                                         (1, 128, "bf16", 16)])
def test_select_xq_group_and_dims(G, d, dtype, x):
    wl = XQ.replace(name=f"xq G{G} d{d} {dtype} x{x}", num_q_heads=2 * G, dtype=dtype,
                    head_dim=d, seed=60 + G + d + x)
    assert check_select_xq(wl, x) == 0


@pytest.mark.parametrize("x,page_size", [(1, 16), (6, 16), (6, 8), (6, 4096), (1, 4096)])
def test_select_xq_paged_ragged(x, page_size):
    # pages of 8 rows (the smallest), 16, and pages longer than a scoring chunk
    wl = XQ.replace(name=f"xq paged P{page_size}", batch=5, page_size=page_size,
                    seq_len=9000 if page_size > 2048 else 5000, seq_len_lo=17, num_q_heads=8,
                    seed=31 + x + page_size % 89)
    assert check_select_xq(wl, x) == 0


@pytest.mark.parametrize("G,x", [(4, 64), (8, 64), (8, 1)])
def test_select_largest_block(G, x):
    """Blocks of 64 rows (the largest): the mean over 64 query rows, and the
    x-row selection up to every row of the block (x G = 512 score rows per KV
    head, the largest the library takes)."""
    wl = XQ.replace(name=f"B64 G{G} x{x}", block=64, num_q_heads=2 * G, seq_len=3000,
                    seq_len_lo=700, seed=70 + G + x)
    assert check_select(wl) == 0
    assert check_select_xq(wl, x) == 0


def test_select_xq_budget_edges_and_ties():
    inp = synth.make_host(XQ.replace(num_q_heads=8))
    wl = XQ.replace(num_q_heads=8)
    assert check_select_xq(wl, 4, inp, np.array([1, 10 ** 6, 700]),
                           int(inp["seq_lens"].max())) == 0
    # every cached row identical: all importances equal, the lowest k indices
    inp["k"][0, :, :] = inp["k"][0, :, 77:78]
    st = Staged(wl, inp)
    got = st.select_xq(8, np.array([300, 5, 5], np.int32), 300)
    for h in range(wl.num_kv_heads):
        np.testing.assert_array_equal(got[0, h], np.arange(300))


def test_select_xq_one_row_differs_from_the_mean():
    # the centre query and the mean of the block queries are different
    # representatives: on random queries their selections differ
    wl = XQ.replace(name="xq vs mean", batch=1, seq_len=4000, seq_len_lo=0, num_q_heads=8, seed=3)
    inp = synth.make_host(wl)
    st = Staged(wl, inp)
    kps = budgets(inp["seq_lens"], *wl.budget)
    a = st.select_xq(1, kps)
    m, _ = st.select(kps)
    assert (a != m).any()


@pytest.mark.parametrize("x,seqs", [(1, [0, 15]), (8, [7]), (32, [3])])
def test_select_xq_layer_32k_sampled(x, seqs):
    """The 8B-class 32K layer as the x sweep runs it (all 16 sequences on the
    GPU in one call), sampled sequences checked by the oracle."""
    assert check_select_xq(synth.LAYER_32K, x, seqs=seqs) == 0


# ---------------------------------------------------------------- draft tail


def check_select_draft(wl, x, n_draft, scale=2.0, seqs=None, seed=5):
    inp = synth.make_host(wl)
    rng = np.random.default_rng(seed)
    st = Staged(wl, inp)
    lens = inp["seq_lens"]
    kps_h = budgets(lens, *wl.budget)
    k_max = int(max(1, min(kps_h.max(), lens.max())))
    d = wl.head_dim
    draft = synth._to_dtype((rng.standard_normal((wl.batch, max(n_draft, 1), wl.num_kv_heads, d))
                             * scale).astype(np.float32), wl.dtype)
    kps = to_dev(kps_h)
    idx = torch.full((wl.batch, wl.num_kv_heads, k_max), -7, dtype=torch.int32, device=DEV)
    ws = H.workspace(H.select_xq_workspace(st.hd, wl.batch, max(x, 1), st.S_max), DEV)
    tdraft = to_dev(draft)
    H.select_draft(st.hd, wl.batch, wl.block, x, st.q_sel, st.kv, tdraft, n_draft, kps,
                   k_max, idx, ws)
    torch.cuda.synchronize()
    got = idx.cpu().numpy()
    near = 0
    for b in (range(wl.batch) if seqs is None else seqs):
        S = int(lens[b])
        k = int(min(max(kps_h[b], 0), S, k_max))
        assert (got[b, :, k:] == -1).all()
        kh, _ = seq_kv_host(inp, b)
        tail = draft[b, :n_draft] if n_draft > 0 else None
        idx_o, shat = oracle.select_draft(inp["q_sel"][b], kh, tail, k, x)
        for h in range(wl.num_kv_heads):
            near += assert_same_selection(got[b, h, :k], idx_o[h], shat[h], k)
    print(f"[select_draft] {wl.name} x={x} n_draft={n_draft}: near-ties={near}")
    return near, got


@pytest.mark.parametrize("x,n_draft", [(0, 32), (1, 32), (0, 0), (1, 1), (3, 64), (8, 32)])
def test_select_draft_tail(x, n_draft):
    wl = XQ.replace(name=f"draft x{x}", num_q_heads=8, seed=80 + x + n_draft)
    assert check_select_draft(wl, x, n_draft)[0] == 0


@pytest.mark.parametrize("G,d,dtype", [(1, 64, "f32"), (8, 128, "bf16"), (2, 64, "bf16")])
def test_select_draft_group_and_dims(G, d, dtype):
    wl = XQ.replace(name=f"draft G{G} d{d} {dtype}", num_q_heads=2 * G, head_dim=d, dtype=dtype,
                    seed=90 + G + d)
    assert check_select_draft(wl, 0, 16)[0] == 0


def test_select_draft_paged_and_strong_draft_changes_selection():
    wl = XQ.replace(name="draft paged", batch=4, page_size=16, seq_len=3000, seq_len_lo=17,
                    num_q_heads=8, seed=33)
    near, with_d = check_select_draft(wl, 1, 32, scale=8.0)
    assert near == 0
    _, without = check_select_draft(wl, 1, 0)
    assert (with_d != without).any()


# ---------------------------------------------------------------- attention output

OUT_TOL = {"bf16": 2e-2, "f32": 1e-5}


def check_select_attn(wl, x, n_draft, seqs=None, seed=6):
    inp = synth.make_host(wl)
    rng = np.random.default_rng(seed)
    st = Staged(wl, inp)
    lens = inp["seq_lens"]
    kps_h = budgets(lens, *wl.budget)
    k_max = int(max(1, min(kps_h.max(), lens.max())))
    d, Hkv, Hq = wl.head_dim, wl.num_kv_heads, wl.num_q_heads
    dk = synth._to_dtype((rng.standard_normal((wl.batch, max(n_draft, 1), Hkv, d)) * 2.0)
                         .astype(np.float32), wl.dtype)
    dv = synth._to_dtype(rng.standard_normal((wl.batch, max(n_draft, 1), Hkv, d))
                         .astype(np.float32), wl.dtype)
    tdk, tdv, kps = to_dev(dk), to_dev(dv), to_dev(kps_h)
    nrow = max(x, 1)
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    o = torch.zeros((wl.batch, nrow, Hq, d), dtype=tdt, device=DEV)
    idx = torch.full((wl.batch, Hkv, k_max), -7, dtype=torch.int32, device=DEV)
    ws = H.workspace(H.select_xq_workspace(st.hd, wl.batch, nrow, st.S_max), DEV)
    H.select_attn(st.hd, wl.batch, wl.block, x, st.q_sel, st.kv, tdk, tdv, n_draft, kps, k_max,
                  idx, o, ws)
    torch.cuda.synchronize()
    got, got_o = idx.cpu().numpy(), f64(to_host(o))
    near, worst = 0, 0.0
    for b in (range(wl.batch) if seqs is None else seqs):
        S = int(lens[b])
        k = int(min(max(kps_h[b], 0), S, k_max))
        kh, vh = seq_kv_host(inp, b)
        tk, tv = (dk[b, :n_draft], dv[b, :n_draft]) if n_draft else (None, None)
        idx_o, shat, o_o = oracle.select_draft(inp["q_sel"][b], kh, tk, k, x, V=vh, tail_v=tv)
        for h in range(Hkv):
            near += assert_same_selection(got[b, h, :k], idx_o[h], shat[h], k)
        err = float(np.abs(got_o[b] - o_o).max())
        worst = max(worst, err)
        assert err <= OUT_TOL[wl.dtype], f"seq {b}: attention output max abs err {err}"
    print(f"[select_attn] {wl.name} x={x} n_draft={n_draft}: near-ties={near} "
          f"max abs err {worst:.3g}")
    return near


@pytest.mark.parametrize("x,n_draft", [(0, 0), (0, 32), (1, 32), (3, 5), (8, 0)])
def test_select_attention_output(x, n_draft):
    wl = XQ.replace(name=f"attn out x{x}", num_q_heads=8, seed=120 + x + n_draft)
    assert check_select_attn(wl, x, n_draft) == 0


@pytest.mark.parametrize("G,d,dtype,x", [(1, 64, "f32", 0), (2, 128, "f32", 2), (8, 64, "bf16", 1),
                                         (4, 64, "bf16", 32)])
def test_select_attention_output_group_and_dims(G, d, dtype, x):
    wl = XQ.replace(name=f"attn out G{G} d{d} {dtype}", num_q_heads=2 * G, head_dim=d,
                    dtype=dtype, seed=130 + G + d + x)
    assert check_select_attn(wl, x, 16) == 0


def test_select_attention_output_paged():
    wl = XQ.replace(name="attn out paged", batch=4, page_size=16, seq_len=3000, seq_len_lo=17,
                    num_q_heads=8, seed=34)
    assert check_select_attn(wl, 1, 32) == 0


def test_select_attention_output_layer_32k_sampled():
    assert check_select_attn(synth.LAYER_32K, 1, 32, seqs=[0, 9]) == 0


def test_select_layer_32k_workload_full():
    """All 16 sequences x 8 KV heads of the 8B-class 32K layer."""
    assert check_select(synth.LAYER_32K) == 0


def test_select_long_128k_workload_full():
    """All 4 sequences x 8 KV heads at 131072 cached tokens (spans)."""
    assert check_select(synth.LONG_128K) == 0


def test_select_ragged_paged_workload_sampled():
    """The 64-sequence ragged paged layer, computed on the GPU in one call;
    12 sequences (shortest, longest and 10 seeded picks) checked by the oracle."""
    wl = synth.RAGGED_PAGED
    inp = synth.make_host(wl)
    lens = inp["seq_lens"]
    pick = set(np.random.default_rng(0).choice(wl.batch, 10, replace=False).tolist())
    pick |= {int(np.argmin(lens)), int(np.argmax(lens))}
    assert check_select(wl, inp, seqs=sorted(pick)) == 0
