"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these checks re-run the oracle's own formula: they compare it with
high-precision brute force (mpmath, 50 digits), with textbook library routines
(torch's scaled_dot_product_attention in float64, numpy sorting), with
invariants and closed forms, and with special cases whose answer is known.
"""
import json
import os

import mpmath
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))


def _rand(rng, shape, dtype):
    x = rng.standard_normal(shape).astype(np.float32)
    if dtype == "f32":
        return x
    if dtype == "f64":
        return x.astype(np.float64)
    t = torch.from_numpy(x).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def _f64(a):
    """exact fp64 value of an oracle input array (float32/float64/bf16 bits)"""
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


# ---------------------------------------------------------------- budget


def test_budget_matches_workload_table():
    g = json.load(open(os.path.join(HERE, "golden", "budget_5pct.json")))
    num, den = g["fraction"]
    for S, k in g["cases"]:
        assert oracle.budget(S, num, den) == k


@pytest.mark.parametrize("S,num,den,k", [
    (1, 1, 20, 1),        # never below one token
    (9, 1, 20, 1),        # 0.45 -> 0 -> clamped to 1
    (10, 1, 20, 1),       # 0.5 rounds half up
    (30, 1, 20, 2),       # 1.5 rounds half up
    (49, 1, 20, 2),       # 2.45 rounds down
    (100, 1, 1, 100),     # full budget keeps everything
    (100, 3, 2, 100),     # never above S
    (65536, 1, 20, 3277),
])
def test_budget_rounding(S, num, den, k):
    assert oracle.budget(S, num, den) == k


# ---------------------------------------------------------------- selection


def _mp_select(q_sel, K, k):
    """50-digit brute force of the selection: mean query, scores, per-head
    softmax, GQA sum, exact sort by (importance desc, index asc)."""
    mpmath.mp.dps = 50
    q = _f64(q_sel)
    kk = _f64(K)
    B, Hq, d = q.shape
    Hkv, S, _ = kk.shape
    G = Hq // Hkv
    scale = 1 / mpmath.sqrt(d)
    shat = [[mpmath.mpf(0)] * S for _ in range(Hkv)]
    for hq in range(Hq):
        h = hq // G
        qbar = [mpmath.fsum(mpmath.mpf(float(q[i, hq, e])) for i in range(B)) / B
                for e in range(d)]
        z = [scale * mpmath.fsum(qbar[e] * mpmath.mpf(float(kk[h, s, e]))
                                 for e in range(d)) for s in range(S)]
        den = mpmath.fsum(mpmath.exp(x) for x in z)
        for s in range(S):
            shat[h][s] += mpmath.exp(z[s]) / den
    idx = []
    for h in range(Hkv):
        order = sorted(range(S), key=lambda s: (-shat[h][s], s))
        idx.append(sorted(order[:k]))
    return np.array(idx, np.int32), shat


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("B,Hq,Hkv,d,S,k", [
    (1, 1, 1, 8, 17, 5),
    (4, 4, 1, 8, 40, 7),
    (4, 8, 2, 16, 64, 9),
    (3, 2, 2, 8, 33, 33),
])
def test_select_matches_50_digit_bruteforce(dtype, B, Hq, Hkv, d, S, k):
    rng = np.random.default_rng(100 + S + B + Hq)
    q_sel = _rand(rng, (B, Hq, d), dtype)
    K = _rand(rng, (Hkv, S, d), dtype)
    idx, shat, m, l = oracle.select(q_sel, K, k)
    ref_idx, ref_shat = _mp_select(q_sel, K, k)
    np.testing.assert_array_equal(idx, ref_idx)
    for h in range(Hkv):
        for s in range(S):
            assert abs(shat[h, s] - float(ref_shat[h][s])) <= 1e-14 * float(ref_shat[h][s])


@pytest.mark.parametrize("G", [1, 2, 4])
def test_importance_reproduces_sdpa_outputs(G):
    """sum_s s_hat[h,s] v_s equals the sum over the group of the attention
    outputs of the representative queries: pins the 1/sqrt(d) scale, the
    per-head softmax normalisation, the G-sum and the head grouping."""
    rng = np.random.default_rng(7 + G)
    B, Hkv, d, S = 4, 2, 16, 50
    Hq = G * Hkv
    q_sel = _rand(rng, (B, Hq, d), "f64")
    K = _rand(rng, (Hkv, S, d), "f64")
    V = rng.standard_normal((Hkv, S, d))
    _, shat, _, _ = oracle.select(q_sel, K, 5)
    qbar = torch.from_numpy(q_sel).mean(0)                     # [Hq][d]
    kt = torch.from_numpy(K).repeat_interleave(G, 0)           # [Hq][S][d]
    vt = torch.from_numpy(V).repeat_interleave(G, 0)
    o = F.scaled_dot_product_attention(qbar[:, None, :], kt, vt)[:, 0]  # [Hq][d]
    want = o.reshape(Hkv, G, d).sum(1).numpy()
    got = np.einsum("hs,hsd->hd", shat, V)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


def test_importance_sums_to_group_size():
    rng = np.random.default_rng(3)
    for G in (1, 3, 4, 8):
        q_sel = _rand(rng, (5, 2 * G, 32), "bf16")
        K = _rand(rng, (2, 300, 32), "bf16")
        _, shat, _, _ = oracle.select(q_sel, K, 10)
        np.testing.assert_allclose(shat.sum(1), G, rtol=1e-13)


def test_topk_is_textbook_ranking_of_importance():
    """The selected set is the first k under numpy's stable ordering of
    (-importance, index), returned ascending."""
    rng = np.random.default_rng(11)
    q_sel = _rand(rng, (8, 8, 64), "bf16")
    K = _rand(rng, (2, 1000, 64), "bf16")
    for k in (1, 37, 500, 999, 1000):
        idx, shat, _, _ = oracle.select(q_sel, K, k)
        for h in range(2):
            order = np.argsort(-shat[h], kind="stable")
            np.testing.assert_array_equal(idx[h], np.sort(order[:k]))


def test_single_query_single_head_is_topk_of_dot_products():
    """G = 1, B = 1: the softmax is monotone, so the selection is the top-k
    of the raw dot products q . k_s."""
    rng = np.random.default_rng(5)
    q = rng.standard_normal((1, 1, 32))
    K = rng.standard_normal((1, 2000, 32))
    dots = K[0] @ q[0, 0]
    assert len(np.unique(dots)) == dots.size
    for k in (1, 10, 100, 1999):
        idx, _, _, _ = oracle.select(q, K, k)
        np.testing.assert_array_equal(idx[0], np.sort(np.argsort(-dots)[:k]))


def test_representative_query_is_the_mean():
    """B queries q+a, q-a, q, ..., q (exact in fp64) select exactly what the
    single query q selects, and with identical importance values."""
    rng = np.random.default_rng(9)
    d, S = 16, 200
    q = np.round(rng.standard_normal((1, 4, d)) * 64) / 64
    a = np.round(rng.standard_normal((1, 4, d)) * 64) / 64
    K = rng.standard_normal((2, S, d))
    rows = np.concatenate([q + a, q - a, q, q], axis=0)       # B = 4, mean = q
    idx1, s1, _, _ = oracle.select(q, K, 20)
    idx4, s4, _, _ = oracle.select(rows, K, 20)
    np.testing.assert_array_equal(idx1, idx4)
    np.testing.assert_allclose(s4, s1, rtol=1e-14)
    # the sum (not the mean) of the rows would change the ranking key
    idx_sum, s_sum, _, _ = oracle.select(4 * q, K, 20)
    assert not np.allclose(s_sum, s1, rtol=1e-6)


def test_ties_go_to_lower_index():
    d, S = 8, 40
    q = np.ones((1, 1, d))
    K = np.zeros((1, S, d))
    K[0, 1::2] = 0.5                        # odd positions: equal, higher score
    idx, shat, _, _ = oracle.select(q, K, S // 2 + 3)
    assert len(np.unique(shat[0, 1::2])) == 1 and len(np.unique(shat[0, 0::2])) == 1
    want = np.sort(np.concatenate([np.arange(1, S, 2), [0, 2, 4]]))
    np.testing.assert_array_equal(idx[0], want)
    # all-equal keys: the lowest k indices
    idx, _, _, _ = oracle.select(q, np.zeros((1, S, d)), 7)
    np.testing.assert_array_equal(idx[0], np.arange(7))


# ---------------------------------------------------------------- x query rows


def _mp_select_xq(q_sel, K, k, rows):
    """50-digit brute force of the x-row selection over the given block rows:
    per (row, head) scores and softmax, summed over rows and the group."""
    mpmath.mp.dps = 50
    q = _f64(q_sel)
    kk = _f64(K)
    _, Hq, d = q.shape
    Hkv, S, _ = kk.shape
    G = Hq // Hkv
    scale = 1 / mpmath.sqrt(d)
    shat = [[mpmath.mpf(0)] * S for _ in range(Hkv)]
    for i in rows:
        for hq in range(Hq):
            h = hq // G
            z = [scale * mpmath.fsum(mpmath.mpf(float(q[i, hq, e])) * mpmath.mpf(float(kk[h, s, e]))
                                     for e in range(d)) for s in range(S)]
            den = mpmath.fsum(mpmath.exp(x) for x in z)
            for s in range(S):
                shat[h][s] += mpmath.exp(z[s]) / den
    idx = []
    for h in range(Hkv):
        order = sorted(range(S), key=lambda s: (-shat[h][s], s))
        idx.append(sorted(order[:k]))
    return np.array(idx, np.int32), shat


@pytest.mark.parametrize("B,x,rows", [(4, 1, [1]), (5, 1, [2]), (4, 2, [1, 2]), (4, 3, [0, 1, 2]),
                                      (5, 3, [1, 2, 3]), (4, 4, [0, 1, 2, 3])])
def test_select_xq_matches_50_digit_bruteforce_on_the_centred_rows(B, x, rows):
    """x rows centred in the block (the lower middle row for even B, as the
    centre [MASK] position of Eq. 2 ties there), each with its own softmax,
    importance summed over rows and heads."""
    rng = np.random.default_rng(40 + 10 * B + x)
    q_sel = _rand(rng, (B, 4, 8), "bf16")
    K = _rand(rng, (2, 23, 8), "bf16")
    idx, shat = oracle.select_xq(q_sel, K, 6, x)
    ref_idx, ref_shat = _mp_select_xq(q_sel, K, 6, rows)
    np.testing.assert_array_equal(idx, ref_idx)
    for h in range(2):
        for s in range(23):
            assert abs(shat[h, s] - float(ref_shat[h][s])) <= 1e-14 * float(ref_shat[h][s])


def test_select_xq_one_row_is_the_mean_selection_of_that_row():
    """x = 1 scores with the centre row alone: exactly what the mean
    selection computes when every block row equals that row."""
    rng = np.random.default_rng(21)
    for B in (1, 4, 7, 32):
        q_sel = _rand(rng, (B, 8, 32), "bf16")
        K = _rand(rng, (2, 500, 32), "bf16")
        c = (B - 1) // 2
        same = np.repeat(q_sel[c:c + 1], B, axis=0)
        idx1, s1 = oracle.select_xq(q_sel, K, 25, 1)
        idx0, s0, _, _ = oracle.select(same, K, 25)
        np.testing.assert_array_equal(idx1, idx0)
        np.testing.assert_array_equal(s1, s0)


@pytest.mark.parametrize("B,x", [(8, 2), (8, 5), (8, 8), (6, 3)])
def test_select_xq_is_the_sum_of_single_row_importances(B, x):
    rng = np.random.default_rng(B * 10 + x)
    q_sel = _rand(rng, (B, 4, 16), "f32")
    K = _rand(rng, (2, 300, 16), "f32")
    _, sx = oracle.select_xq(q_sel, K, 10, x)
    c0 = (B - x) // 2
    want = np.zeros_like(sx)
    for i in range(c0, c0 + x):
        _, si, _, _ = oracle.select(np.repeat(q_sel[i:i + 1], B, axis=0), K, 10)
        want += si
    np.testing.assert_allclose(sx, want, rtol=1e-13)
    np.testing.assert_allclose(sx.sum(1), x * 2, rtol=1e-13)   # x rows x G = 2 heads


def test_select_xq_importance_reproduces_sdpa_outputs():
    """sum_s s_hat[h,s] v_s is the sum of the attention outputs of the x
    window rows over the heads of the group."""
    rng = np.random.default_rng(77)
    B, x, G, Hkv, d, S = 6, 4, 2, 2, 16, 60
    q_sel = _rand(rng, (B, G * Hkv, d), "f64")
    K = _rand(rng, (Hkv, S, d), "f64")
    V = rng.standard_normal((Hkv, S, d))
    _, shat = oracle.select_xq(q_sel, K, 5, x)
    c0 = (B - x) // 2
    q = torch.from_numpy(q_sel[c0:c0 + x]).permute(1, 0, 2)          # [Hq][x][d]
    kt = torch.from_numpy(K).repeat_interleave(G, 0)
    vt = torch.from_numpy(V).repeat_interleave(G, 0)
    o = F.scaled_dot_product_attention(q, kt, vt)                    # [Hq][x][d]
    want = o.sum(1).reshape(Hkv, G, d).sum(1).numpy()
    got = np.einsum("hs,hsd->hd", shat, V)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


def test_select_xq_ties_go_to_lower_index():
    q = np.ones((3, 1, 8))
    idx, _ = oracle.select_xq(q, np.zeros((1, 40, 8)), 7, 2)
    np.testing.assert_array_equal(idx[0], np.arange(7))


@pytest.mark.parametrize("pos", [0, 1, 63, 64, 127, 128, 500, 998, 999])
def test_planted_key_anywhere_is_selected(pos):
    """Every prefix entry is scored: a dominant key is found at any position."""
    rng = np.random.default_rng(pos)
    q_sel = rng.standard_normal((4, 4, 32))
    K = rng.standard_normal((1, 1000, 32))
    K[0, pos] = 20 * q_sel.mean(0)[0] / np.linalg.norm(q_sel.mean(0)[0])
    idx, _, _, _ = oracle.select(q_sel, K, 1)
    assert idx[0, 0] == pos


def test_full_budget_selects_everything():
    rng = np.random.default_rng(1)
    K = _rand(rng, (3, 77, 16), "bf16")
    idx, _, _, _ = oracle.select(_rand(rng, (2, 6, 16), "bf16"), K, 77)
    np.testing.assert_array_equal(idx, np.tile(np.arange(77), (3, 1)))


# ---------------------------------------------------------------- gather


def test_gather_copies_rows_bitwise():
    rng = np.random.default_rng(2)
    for dt in ("f32", "bf16"):
        K = _rand(rng, (2, 90, 16), dt)
        idx = np.sort(rng.choice(90, (2, 13), replace=True), axis=1).astype(np.int32)
        pool = oracle.gather(K, idx, cap=20)
        for h in range(2):
            assert pool[h, :13].tobytes() == K[h, idx[h]].tobytes()
            assert not pool[h, 13:].any()
        full = oracle.gather(K, np.tile(np.arange(90, dtype=np.int32), (2, 1)))
        assert full.tobytes() == K.tobytes()


# ---------------------------------------------------------------- attention


def _sdpa(q, keys, vals, mask=None):
    """q [B][Hq][d], keys/vals [Hkv][n][d] (float64) -> [B][Hq][d]"""
    Hq, Hkv = q.shape[1], keys.shape[0]
    G = Hq // Hkv
    qt = torch.from_numpy(q).transpose(0, 1)                   # [Hq][B][d]
    kt = torch.from_numpy(keys).repeat_interleave(G, 0)
    vt = torch.from_numpy(vals).repeat_interleave(G, 0)
    m = None if mask is None else torch.from_numpy(mask).repeat_interleave(G, 0)[:, None, :]
    return F.scaled_dot_product_attention(qt, kt, vt, attn_mask=m).transpose(0, 1).numpy()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_attention_over_full_prefix_is_dense_sdpa(dtype):
    rng = np.random.default_rng(21)
    B, Hq, Hkv, d, n = 4, 8, 2, 32, 150
    q = _rand(rng, (B, Hq, d), dtype)
    ck, cv = _rand(rng, (Hkv, n, d), dtype), _rand(rng, (Hkv, n, d), dtype)
    bk, bv = _rand(rng, (B, Hkv, d), dtype), _rand(rng, (B, Hkv, d), dtype)
    out = oracle.attn(q, ck, cv, bk, bv)
    keys = np.concatenate([_f64(ck), _f64(bk).transpose(1, 0, 2)], axis=1)
    vals = np.concatenate([_f64(cv), _f64(bv).transpose(1, 0, 2)], axis=1)
    np.testing.assert_allclose(out, _sdpa(_f64(q), keys, vals), rtol=1e-12, atol=1e-13)


def test_sparse_attention_is_masked_dense_attention():
    """Selection + gather + attention equals dense attention over the whole
    prefix with every unselected prefix entry masked out."""
    rng = np.random.default_rng(22)
    B, Hq, Hkv, d, S, k = 4, 8, 2, 16, 120, 17
    q_sel, q = _rand(rng, (B, Hq, d), "bf16"), _rand(rng, (B, Hq, d), "bf16")
    K, V = _rand(rng, (Hkv, S, d), "bf16"), _rand(rng, (Hkv, S, d), "bf16")
    bk, bv = _rand(rng, (B, Hkv, d), "bf16"), _rand(rng, (B, Hkv, d), "bf16")
    idx, _, _, _ = oracle.select(q_sel, K, k)
    out = oracle.attn(q, oracle.gather(K, idx), oracle.gather(V, idx), bk, bv)
    mask = np.zeros((Hkv, S + B), bool)
    for h in range(Hkv):
        mask[h, idx[h]] = True
    mask[:, S:] = True
    keys = np.concatenate([_f64(K), _f64(bk).transpose(1, 0, 2)], axis=1)
    vals = np.concatenate([_f64(V), _f64(bv).transpose(1, 0, 2)], axis=1)
    np.testing.assert_allclose(out, _sdpa(_f64(q), keys, vals, mask), rtol=1e-12,
                               atol=1e-13)


def test_attention_rows_are_convex_combinations():
    rng = np.random.default_rng(23)
    B, Hq, Hkv, d, n = 3, 4, 4, 8, 30
    q = rng.standard_normal((B, Hq, d)) * 5
    ck = rng.standard_normal((Hkv, n, d))
    bk = rng.standard_normal((B, Hkv, d))
    out = oracle.attn(q, ck, np.full((Hkv, n, d), 2.5), bk, np.full((B, Hkv, d), 2.5))
    np.testing.assert_allclose(out, 2.5, rtol=1e-14)
    # an empty context leaves attention over the block alone
    out0 = oracle.attn(q, np.zeros((Hkv, 0, d)), np.zeros((Hkv, 0, d)), bk,
                       np.broadcast_to(np.arange(d, dtype=float), (B, Hkv, d)).copy())
    np.testing.assert_allclose(out0, np.broadcast_to(np.arange(d, dtype=float), out0.shape),
                               rtol=1e-13)


# ---------------------------------------------------------------- block schedule


def test_full_budget_schedule_is_dense_decoding():
    """At a 100% budget the pool of every block is the whole prefix, block n
    included once completed: each step equals dense attention over the
    growing cache plus the block's own KV."""
    rng = np.random.default_rng(31)
    B, T, Hq, Hkv, d, S0 = 4, 2, 4, 2, 16, 40
    K0, V0 = _rand(rng, (Hkv, S0, d), "f64"), _rand(rng, (Hkv, S0, d), "f64")
    blocks = []
    for _ in range(3):
        blocks.append(dict(
            q_steps=_rand(rng, (T, B, Hq, d), "f64"),
            k_steps=_rand(rng, (T, B, Hkv, d), "f64"),
            v_steps=_rand(rng, (T, B, Hkv, d), "f64"),
            k_done=_rand(rng, (B, Hkv, d), "f64"),
            v_done=_rand(rng, (B, Hkv, d), "f64"),
            q_next=_rand(rng, (B, Hq, d), "f64")))
    idx0 = np.tile(np.arange(S0, dtype=np.int32), (Hkv, 1))
    outs = oracle.decode_blocks(K0, V0, idx0, blocks, num=1, den=1)
    Kc, Vc = K0, V0
    for n, blk in enumerate(blocks):
        for t in range(T):
            keys = np.concatenate([Kc, blk["k_steps"][t].transpose(1, 0, 2)], axis=1)
            vals = np.concatenate([Vc, blk["v_steps"][t].transpose(1, 0, 2)], axis=1)
            np.testing.assert_allclose(outs[n][t], _sdpa(blk["q_steps"][t], keys, vals),
                                       rtol=1e-12, atol=1e-13)
        Kc = np.concatenate([Kc, blk["k_done"].transpose(1, 0, 2)], axis=1)
        Vc = np.concatenate([Vc, blk["v_done"].transpose(1, 0, 2)], axis=1)


def test_schedule_selects_from_prefix_before_current_block():
    """Block n+1's pool: top-k over the prefix before block n, then block n's
    completed KV unconditionally (the draft-lookahead schedule)."""
    rng = np.random.default_rng(32)
    B, T, Hq, Hkv, d, S0 = 2, 1, 2, 1, 8, 60
    K0, V0 = _rand(rng, (Hkv, S0, d), "f64"), _rand(rng, (Hkv, S0, d), "f64")
    mk = lambda: dict(q_steps=_rand(rng, (T, B, Hq, d), "f64"),
                      k_steps=_rand(rng, (T, B, Hkv, d), "f64"),
                      v_steps=_rand(rng, (T, B, Hkv, d), "f64"),
                      k_done=_rand(rng, (B, Hkv, d), "f64"),
                      v_done=_rand(rng, (B, Hkv, d), "f64"),
                      q_next=_rand(rng, (B, Hq, d), "f64"))
    blocks = [mk(), mk()]
    idx0, _, _, _ = oracle.select(_rand(rng, (B, Hq, d), "f64"), K0, 3)
    outs = oracle.decode_blocks(K0, V0, idx0, blocks, num=1, den=20)
    k1 = oracle.budget(S0, 1, 20)
    idx1, _, _, _ = oracle.select(blocks[0]["q_next"], K0, k1)
    pool_k = np.concatenate([K0[:, idx1[0]], blocks[0]["k_done"].transpose(1, 0, 2)], 1)
    pool_v = np.concatenate([V0[:, idx1[0]], blocks[0]["v_done"].transpose(1, 0, 2)], 1)
    want = _sdpa(blocks[1]["q_steps"][0],
                 np.concatenate([pool_k, blocks[1]["k_steps"][0].transpose(1, 0, 2)], 1),
                 np.concatenate([pool_v, blocks[1]["v_steps"][0].transpose(1, 0, 2)], 1))
    np.testing.assert_allclose(outs[1][0], want, rtol=1e-12, atol=1e-13)


# ---------------------------------------------------------------- draft lookahead


@pytest.mark.parametrize("x", [0, 1, 3])
def test_select_draft_without_tail_is_the_plain_selection(x):
    rng = np.random.default_rng(60 + x)
    q_sel = _rand(rng, (6, 8, 16), "bf16")
    K = _rand(rng, (2, 400, 16), "bf16")
    idx, s = oracle.select_draft(q_sel, K, None, 30, x)
    if x == 0:
        idx0, s0, _, _ = oracle.select(q_sel, K, 30)
    else:
        idx0, s0 = oracle.select_xq(q_sel, K, 30, x)
    np.testing.assert_array_equal(idx, idx0)
    np.testing.assert_array_equal(s, s0)


@pytest.mark.parametrize("x", [0, 1, 2])
def test_select_draft_tail_enters_the_normalisers_only(x):
    """The draft rows are scored and normalised with the cache (the same
    importance as a selection over cache + draft) but never selected: the
    result is the top-k of the cache rows' importances alone."""
    rng = np.random.default_rng(70 + x)
    B, Hq, Hkv, d, S, n = 4, 8, 2, 16, 300, 4
    q_sel = _rand(rng, (B, Hq, d), "f64")
    K = _rand(rng, (Hkv, S, d), "f64")
    tail = _rand(rng, (n, Hkv, d), "f64") * 3.0                 # strong draft keys
    idx, s = oracle.select_draft(q_sel, K, tail, 25, x)
    Kx = np.concatenate([K, tail.transpose(1, 0, 2)], axis=1)
    if x == 0:
        _, sx, _, _ = oracle.select(q_sel, Kx, 25)
    else:
        _, sx = oracle.select_xq(q_sel, Kx, 25, x)
    np.testing.assert_array_equal(s, sx[:, :S])
    for h in range(Hkv):
        np.testing.assert_array_equal(idx[h], np.sort(np.argsort(-sx[h, :S], kind="stable")[:25]))
    assert (s.sum(1) < (1 if x == 0 else x) * (Hq // Hkv) - 1e-3).all()   # draft mass excluded


def test_select_draft_tail_shifts_the_ranking_between_heads():
    """A draft row aligned with head 0's query dominates head 0's normaliser,
    so the cache ranking follows head 1: the selection becomes head 1's
    top-k of its scores."""
    d, S = 8, 200
    rng = np.random.default_rng(5)
    q0 = np.zeros(d); q0[0] = 1.0
    q1 = np.zeros(d); q1[1] = 1.0
    q_sel = np.stack([q0, q1])[None] * 2.0                         # B = 1, Hq = 2, Hkv = 1
    K = rng.standard_normal((1, S, d))
    tail = np.zeros((1, 1, d)); tail[0, 0, 0] = 60.0               # exp(~42) swamps head 0
    idx, _ = oracle.select_draft(q_sel, K, tail, 10)
    by_h1 = np.sort(np.argsort(-K[0, :, 1], kind="stable")[:10])
    np.testing.assert_array_equal(idx[0], by_h1)
    idx0, _, _, _ = oracle.select(q_sel, K, 10)
    assert not np.array_equal(idx0[0], by_h1)


def test_attention_groups_are_masked_dense_attention():
    """Two groups of B queries over one context: group j sees the context and
    its own B block rows, not the other group's (block-diagonal mask)."""
    rng = np.random.default_rng(88)
    B, Hq, Hkv, d, n = 4, 4, 2, 16, 30
    q = _rand(rng, (2 * B, Hq, d), "f64")
    ck, cv = _rand(rng, (Hkv, n, d), "f64"), _rand(rng, (Hkv, n, d), "f64")
    bk, bv = _rand(rng, (2 * B, Hkv, d), "f64"), _rand(rng, (2 * B, Hkv, d), "f64")
    got = oracle.attn_groups(q, ck, cv, bk, bv, 2)
    keys = np.concatenate([ck, bk.transpose(1, 0, 2)], axis=1)
    vals = np.concatenate([cv, bv.transpose(1, 0, 2)], axis=1)
    for j in range(2):
        mask = np.zeros((Hkv, n + 2 * B), bool)
        mask[:, :n] = True
        mask[:, n + j * B:n + (j + 1) * B] = True
        want = _sdpa(q[j * B:(j + 1) * B], keys, vals, mask)
        np.testing.assert_allclose(got[j * B:(j + 1) * B], want, rtol=1e-12, atol=1e-13)
    np.testing.assert_array_equal(oracle.attn_groups(q[:B], ck, cv, bk[:B], bv[:B], 1),
                                  oracle.attn(q[:B], ck, cv, bk[:B], bv[:B]))


@pytest.mark.parametrize("x", [0, 1])
def test_full_budget_schedule_with_drafts_is_dense_decoding(x):
    """At a 100% budget the draft changes no selection (everything is
    selected): outputs equal those of the schedule without drafts."""
    rng = np.random.default_rng(41)
    B, T, Hq, Hkv, d, S0 = 4, 2, 4, 2, 16, 40
    K0, V0 = _rand(rng, (Hkv, S0, d), "f64"), _rand(rng, (Hkv, S0, d), "f64")
    blocks = []
    for _ in range(3):
        blocks.append(dict(
            q_steps=_rand(rng, (T, B, Hq, d), "f64"),
            k_steps=_rand(rng, (T, B, Hkv, d), "f64"),
            v_steps=_rand(rng, (T, B, Hkv, d), "f64"),
            k_done=_rand(rng, (B, Hkv, d), "f64"),
            v_done=_rand(rng, (B, Hkv, d), "f64"),
            k_draft=_rand(rng, (B, Hkv, d), "f64") * 4.0,
            q_next=_rand(rng, (B, Hq, d), "f64")))
    for blk in blocks:
        blk["q_draft"] = _rand(rng, (B, Hq, d), "f64")
        blk["v_draft"] = _rand(rng, (B, Hkv, d), "f64")
    idx0 = np.tile(np.arange(S0, dtype=np.int32), (Hkv, 1))
    douts = []
    with_d = oracle.decode_blocks(K0, V0, idx0, blocks, num=1, den=1, x=x, draft_outs=douts)
    without = oracle.decode_blocks(K0, V0, idx0, [{k: v for k, v in b.items() if k != "k_draft"}
                                                  for b in blocks], num=1, den=1)
    for a, b in zip(with_d, without):
        np.testing.assert_array_equal(a, b)
    # the draft group: dense attention over the prefix before its block plus
    # the draft's own KV (at 100% the pool is the whole prefix)
    Kc, Vc = K0, V0
    for n, blk in enumerate(blocks):
        keys = np.concatenate([Kc, blk["k_draft"].transpose(1, 0, 2)], axis=1)
        vals = np.concatenate([Vc, blk["v_draft"].transpose(1, 0, 2)], axis=1)
        np.testing.assert_allclose(douts[n], _sdpa(blk["q_draft"], keys, vals),
                                   rtol=1e-12, atol=1e-13)
        Kc = np.concatenate([Kc, blk["k_done"].transpose(1, 0, 2)], axis=1)
        Vc = np.concatenate([Vc, blk["v_done"].transpose(1, 0, 2)], axis=1)


def test_schedule_with_draft_selects_with_the_draft_as_tail():
    """At 5% the draft KV of block n shapes block n+1's selection through the
    normalisers: pool(n+1) = select_draft top-k of the prefix before block n,
    then block n's completed KV."""
    rng = np.random.default_rng(33)
    B, T, Hq, Hkv, d, S0 = 2, 1, 4, 1, 8, 80
    K0, V0 = _rand(rng, (Hkv, S0, d), "f64"), _rand(rng, (Hkv, S0, d), "f64")
    mk = lambda: dict(q_steps=_rand(rng, (T, B, Hq, d), "f64"),
                      k_steps=_rand(rng, (T, B, Hkv, d), "f64"),
                      v_steps=_rand(rng, (T, B, Hkv, d), "f64"),
                      k_done=_rand(rng, (B, Hkv, d), "f64"),
                      v_done=_rand(rng, (B, Hkv, d), "f64"),
                      k_draft=_rand(rng, (B, Hkv, d), "f64") * 5.0,
                      q_next=_rand(rng, (B, Hq, d), "f64"))
    blocks = [mk(), mk()]
    idx0, _, _, _ = oracle.select(_rand(rng, (B, Hq, d), "f64"), K0, 4)
    outs = oracle.decode_blocks(K0, V0, idx0, blocks, num=1, den=20, x=1)
    k1 = oracle.budget(S0, 1, 20)
    c = (B - 1) // 2
    Kx = np.concatenate([K0, blocks[0]["k_draft"].transpose(1, 0, 2)], axis=1)
    _, sx = oracle.select_xq(np.repeat(blocks[0]["q_next"][c:c + 1], B, axis=0), Kx, k1, 1)
    sel = np.sort(np.argsort(-sx[0, :S0], kind="stable")[:k1])
    pool_k = np.concatenate([K0[:, sel], blocks[0]["k_done"].transpose(1, 0, 2)], 1)
    pool_v = np.concatenate([V0[:, sel], blocks[0]["v_done"].transpose(1, 0, 2)], 1)
    want = _sdpa(blocks[1]["q_steps"][0],
                 np.concatenate([pool_k, blocks[1]["k_steps"][0].transpose(1, 0, 2)], 1),
                 np.concatenate([pool_v, blocks[1]["v_steps"][0].transpose(1, 0, 2)], 1))
    np.testing.assert_allclose(outs[1][0], want, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("x,n", [(0, 0), (0, 3), (1, 3), (3, 2)])
def test_selection_output_is_sdpa_of_the_representative_rows(x, n):
    """The attention output kept beside the ranking is exact attention of
    each representative row over the cache plus the draft (fp64 SDPA)."""
    rng = np.random.default_rng(200 + 10 * x + n)
    B, Hq, Hkv, d, S = 5, 8, 2, 16, 120
    q_sel = _rand(rng, (B, Hq, d), "f64")
    K, V = _rand(rng, (Hkv, S, d), "f64"), _rand(rng, (Hkv, S, d), "f64")
    tk = _rand(rng, (n, Hkv, d), "f64") if n else None
    tv = _rand(rng, (n, Hkv, d), "f64") if n else None
    idx, s, o = oracle.select_draft(q_sel, K, tk, 9, x, V=V, tail_v=tv)
    idx0, s0 = oracle.select_draft(q_sel, K, tk, 9, x)
    np.testing.assert_array_equal(idx, idx0)
    np.testing.assert_array_equal(s, s0)
    keys = K if not n else np.concatenate([K, tk.transpose(1, 0, 2)], axis=1)
    vals = V if not n else np.concatenate([V, tv.transpose(1, 0, 2)], axis=1)
    if x == 0:
        rows = q_sel.mean(0, keepdims=True)
    else:
        c0 = (B - x) // 2
        rows = q_sel[c0:c0 + x]
    np.testing.assert_allclose(o, _sdpa(rows, keys, vals), rtol=1e-12, atol=1e-13)
