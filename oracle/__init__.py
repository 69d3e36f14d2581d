"""HERALD reference oracle (CPU, fp64). TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package; the product library never does, and
the two share no code. Inputs are numpy arrays (float32, float64, or uint16
holding bfloat16 bit patterns) or torch CPU tensors of those types; every
element is decoded exactly to fp64 inside the C code (``herald_oracle.c``).

Functions and the passages of the paper they follow:

* ``budget``      per-KV-head selection budget k (sec. IV-B.4: k is the
                  per-KV-head budget; the 5% operating point of sec. VI).
                  Rounding half-up is a reading (the paper gives none).
* ``select``      representative-query selection, one sequence: mean of the
                  block's B queries per head (the representative query of
                  sec. IV-A.2, mean variant), full-prefix scoring, softmax
                  statistics per query head, GQA importance
                  s_hat_h[s] = sum_g exp(s[g,s]-m_g)/l_g and one top-k per
                  KV head (sec. IV-B.4). Ties: lower index; output ascending.
* ``select_xq``   selection with x query rows used as they are: the x rows
                  centred in the block (rows floor((B-x)/2) ...), softmax
                  statistics per (row, head) and the importance summed over
                  all x*G softmax-normalised score rows (the G-sum of
                  sec. IV-B.4 extended over rows, a reading). x = 1 is the
                  centre [MASK] query of sec. IV-A.2 (Eq. 2; lower middle
                  row for even B); x = B every query of the block.
* ``select_draft`` block n+1's selection with block n's draft KV appended
                  for normalisation (sec. IV-B.2, steps 7-8): representative
                  = mean (x = 0) or the x centred rows; the draft rows enter
                  every softmax normaliser (m, l) but are never candidates
                  (a reading: the completed block replaces them).
* ``attn_groups`` the 2B-token step of sec. IV-B.2 (step 3): groups of B
                  queries that attend to the same context, each to its own
                  block KV and not to the other groups (custom masks).
* ``gather``      copy of the selected rows into the sparse pool (sec. IV-B.3).
* ``attn``        B-query GQA attention over a context plus the block's own
                  KV, unmasked (sec. II-A: bidirectional inside the block,
                  causal to the completed prefix, which the context is).
* ``decode_blocks`` the dual-stream block schedule written sequentially
                  (sec. IV-A.1 and IV-B.2): block n+1's pool is the top-k of
                  the prefix before block n plus block n's completed KV.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "herald_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

F32, BF16, F64 = 0, 1, 2


def build(force: bool = True) -> str:
    """Compile the C oracle with gcc (strict IEEE fp64, OpenMP)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        cmd = ["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp",
               "-shared", "-fPIC", "-std=c11", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build(force=True)
    lib = ctypes.CDLL(_LIB_PATH)
    i64, i32, p, d = ctypes.c_int64, ctypes.c_int, ctypes.c_void_p, ctypes.c_double
    lib.herald_oracle_threads.restype = i32
    lib.herald_oracle_threads.argtypes = []
    lib.herald_oracle_set_threads.restype = None
    lib.herald_oracle_set_threads.argtypes = [i32]
    lib.herald_oracle_budget.restype = i64
    lib.herald_oracle_budget.argtypes = [i64, i64, i64]
    lib.herald_oracle_select.restype = i32
    lib.herald_oracle_select.argtypes = [i32, i32, i32, i32, i64, p, i32, p, i32,
                                         i64, p, p, p, p]
    lib.herald_oracle_select_xq.restype = i32
    lib.herald_oracle_select_xq.argtypes = [i32, i32, i32, i32, i32, i64, p, i32, p, i32,
                                            i64, p, p]
    lib.herald_oracle_select_draft.restype = i32
    lib.herald_oracle_select_draft.argtypes = [i32, i32, i32, i32, i32, i64, p, i32, p, i32,
                                               p, i32, i64, i64, p, p, p, p, p]
    lib.herald_oracle_gather.restype = i32
    lib.herald_oracle_gather.argtypes = [i32, i32, i64, p, i32, p, i64, i64, p]
    lib.herald_oracle_attn.restype = i32
    lib.herald_oracle_attn.argtypes = [i32, i32, i32, i32, i64, i64, p, i32, p, p,
                                       i32, p, p, i32, p]
    _lib = lib
    return lib


def _as_np(x):
    """numpy view of an input, plus its oracle element-type code."""
    try:
        import torch
        if isinstance(x, torch.Tensor):
            x = x.detach().cpu().contiguous()
            if x.dtype == torch.bfloat16:
                return x.view(torch.int16).numpy().view(np.uint16), BF16
            x = x.numpy()
    except ImportError:  # pragma: no cover
        pass
    x = np.ascontiguousarray(x)
    if x.dtype == np.float32:
        return x, F32
    if x.dtype == np.float64:
        return x, F64
    if x.dtype == np.uint16:
        return x, BF16
    raise TypeError(f"oracle input dtype {x.dtype} not supported")


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def threads() -> int:
    """OpenMP threads the oracle's loops use."""
    return int(_load().herald_oracle_threads())


def set_threads(n: int) -> None:
    """Sets the OpenMP threads of the oracle's loops (at least 1)."""
    _load().herald_oracle_set_threads(int(n))


def budget(S: int, num: int = 1, den: int = 20) -> int:
    """k = clamp(floor(S*num/den + 1/2), 1, S)."""
    return int(_load().herald_oracle_budget(int(S), int(num), int(den)))


def select(q_sel, K, k: int):
    """One sequence. q_sel [B][Hq][d], K [Hkv][S][d].

    Returns (idx int32 [Hkv][k] ascending, s_hat float64 [Hkv][S],
    m float64 [Hq], l float64 [Hq]).
    """
    q, qt = _as_np(q_sel)
    kk, kt = _as_np(K)
    B, Hq, d = q.shape
    Hkv, S, d2 = kk.shape
    assert d == d2 and Hq % Hkv == 0
    idx = np.empty((Hkv, k), np.int32)
    s_hat = np.empty((Hkv, S), np.float64)
    m = np.empty(Hq, np.float64)
    l = np.empty(Hq, np.float64)
    rc = _load().herald_oracle_select(B, Hq, Hkv, d, S, _ptr(q), qt, _ptr(kk), kt,
                                      int(k), _ptr(s_hat), _ptr(m), _ptr(l), _ptr(idx))
    if rc != 0:
        raise ValueError("herald_oracle_select: bad arguments")
    return idx, s_hat, m, l


def select_xq(q_sel, K, k: int, x: int):
    """One sequence, x query rows. q_sel [B][Hq][d], K [Hkv][S][d].

    Returns (idx int32 [Hkv][k] ascending, s_hat float64 [Hkv][S]).
    """
    q, qt = _as_np(q_sel)
    kk, kt = _as_np(K)
    B, Hq, d = q.shape
    Hkv, S, d2 = kk.shape
    assert d == d2 and Hq % Hkv == 0
    idx = np.empty((Hkv, k), np.int32)
    s_hat = np.empty((Hkv, S), np.float64)
    rc = _load().herald_oracle_select_xq(B, int(x), Hq, Hkv, d, S, _ptr(q), qt, _ptr(kk), kt,
                                         int(k), _ptr(s_hat), _ptr(idx))
    if rc != 0:
        raise ValueError("herald_oracle_select_xq: bad arguments")
    return idx, s_hat


def select_draft(q_sel, K, tail, k: int, x: int = 0, V=None, tail_v=None):
    """One sequence. q_sel [B][Hq][d], K [Hkv][S][d], tail [n][Hkv][d] (or
    None). Returns (idx int32 [Hkv][k] ascending, s_hat float64 [Hkv][S]);
    with V [Hkv][S][d] (and tail_v like tail) also the attention output of
    every representative row, float64 [max(x,1)][Hq][d]."""
    q, qt = _as_np(q_sel)
    kk, kt = _as_np(K)
    B, Hq, d = q.shape
    Hkv, S, d2 = kk.shape
    assert d == d2 and Hq % Hkv == 0
    if tail is None:
        tt, ttype, n = np.zeros((1, Hkv, d), np.float64), F64, 0
    else:
        tt, ttype = _as_np(tail)
        assert tt.shape[1:] == (Hkv, d)
        n = tt.shape[0]
    idx = np.empty((Hkv, k), np.int32)
    s_hat = np.empty((Hkv, S), np.float64)
    o = vv = tv = None
    if V is not None:
        vv, vt = _as_np(V)
        assert vt == kt and vv.shape == kk.shape
        if tail_v is not None:
            tv, tvt = _as_np(tail_v)
            assert tvt == ttype and tv.shape == tt.shape
        elif n:
            raise ValueError("tail_v is needed with a tail")
        o = np.empty((max(int(x), 1), Hq, d), np.float64)
    rc = _load().herald_oracle_select_draft(B, int(x), Hq, Hkv, d, S, _ptr(q), qt, _ptr(kk),
                                            kt, _ptr(tt), ttype, n, int(k), _ptr(s_hat),
                                            _ptr(idx), None if vv is None else _ptr(vv),
                                            None if tv is None else _ptr(tv),
                                            None if o is None else _ptr(o))
    if rc != 0:
        raise ValueError("herald_oracle_select_draft: bad arguments")
    return (idx, s_hat) if o is None else (idx, s_hat, o)


def attn_groups(q, ctx_k, ctx_v, blk_k, blk_v, groups: int):
    """One sequence, `groups` groups of B queries. q [groups*B][Hq][d];
    blk_k/blk_v [groups*B][Hkv][d]; group j's queries attend to the context
    and to block rows j*B .. j*B+B-1 only. Returns float64 [groups*B][Hq][d]."""
    qq, _ = _as_np(q)
    bk, _ = _as_np(blk_k)
    bv, _ = _as_np(blk_v)
    n = qq.shape[0]
    assert n % groups == 0 and bk.shape[0] == n and bv.shape[0] == n
    B = n // groups
    return np.concatenate([attn(qq[j * B:(j + 1) * B], ctx_k, ctx_v, bk[j * B:(j + 1) * B],
                                bv[j * B:(j + 1) * B]) for j in range(groups)], axis=0)


def gather(K, idx, cap: int | None = None):
    """pool[h][j] = K[h][idx[h][j]] (bit copy). K [Hkv][S][d], idx [Hkv][k]."""
    kk, kt = _as_np(K)
    ii = np.ascontiguousarray(idx, dtype=np.int32)
    Hkv, S, d = kk.shape
    k = ii.shape[1]
    cap = k if cap is None else cap
    pool = np.zeros((Hkv, cap, d), kk.dtype)
    rc = _load().herald_oracle_gather(Hkv, d, S, _ptr(kk), kt, _ptr(ii), k, cap,
                                      _ptr(pool))
    if rc != 0:
        raise ValueError("herald_oracle_gather: bad arguments")
    return pool


def attn(q, ctx_k, ctx_v, blk_k, blk_v):
    """One sequence. q [B][Hq][d]; ctx_k/ctx_v [Hkv][n][d]; blk_k/blk_v
    [B][Hkv][d]. Returns float64 [B][Hq][d]."""
    qq, qt = _as_np(q)
    ck, ckt = _as_np(ctx_k)
    cv, cvt = _as_np(ctx_v)
    bk, bkt = _as_np(blk_k)
    bv, bvt = _as_np(blk_v)
    assert ckt == cvt and bkt == bvt
    B, Hq, d = qq.shape
    Hkv, n, _ = ck.shape
    out = np.empty((B, Hq, d), np.float64)
    rc = _load().herald_oracle_attn(B, Hq, Hkv, d, n, n, _ptr(qq), qt, _ptr(ck),
                                    _ptr(cv), ckt, _ptr(bk), _ptr(bv), bkt, _ptr(out))
    if rc != 0:
        raise ValueError("herald_oracle_attn: bad arguments")
    return out


def decode_blocks(K0, V0, pool_idx0, blocks, num: int = 1, den: int = 20, x: int = 0,
                  draft_outs: list | None = None):
    """Sequential schedule of consecutive blocks of one sequence, one layer.

    K0, V0 [Hkv][S0][d]: the prefix cache before the first block.
    pool_idx0 [Hkv][k0]: the initial selection (the prefill-time top-k).
    blocks: list of dicts, one per block n, with
        q_steps  [T][B][Hq][d]  the block's denoising queries,
        k_steps, v_steps [T][B][Hkv][d]  the block's own KV per step,
        k_done, v_done [B][Hkv][d]  the completed block's KV,
        q_next [B][Hq][d]  block n+1's selection queries.
    Optional per block: k_draft [B][Hkv][d], block n's draft KV, which block
    n+1's selection appends for normalisation (sec. IV-B.2, steps 7-8);
    x = 0 selects with the mean of q_next, x >= 1 with its x centred rows.
    With q_draft [B][Hq][d] and v_draft as well, the draft group of the
    2B-token step attends to pool(n) and its own draft KV; its output is
    appended to draft_outs (None for blocks without a draft) if given.
    Block n is denoised over pool(n); block n+1's selection runs over the
    prefix before block n; pool(n+1) = that top-k followed by block n's
    completed KV; then the cache grows by block n's completed KV.
    Returns the list of per-block outputs [T][B][Hq][d] (fp64).
    """
    Kc, kt = _as_np(K0)
    Vc, _ = _as_np(V0)
    pool_k = gather(Kc, pool_idx0)
    pool_v = gather(Vc, pool_idx0)
    outs = []
    for blk in blocks:
        T = len(blk["q_steps"])
        outs.append(np.stack([attn(blk["q_steps"][t], pool_k, pool_v,
                                   blk["k_steps"][t], blk["v_steps"][t])
                              for t in range(T)]))
        if draft_outs is not None:
            draft_outs.append(attn(blk["q_draft"], pool_k, pool_v, blk["k_draft"], blk["v_draft"])
                              if blk.get("q_draft") is not None else None)
        S = Kc.shape[1]
        k = budget(S, num, den)
        if x == 0 and blk.get("k_draft") is None:
            idx, _, _, _ = select(blk["q_next"], Kc, k)
        else:
            idx, _ = select_draft(blk["q_next"], Kc, blk.get("k_draft"), k, x)
        kd, _ = _as_np(blk["k_done"])
        vd, _ = _as_np(blk["v_done"])
        kd = np.ascontiguousarray(kd.transpose(1, 0, 2))
        vd = np.ascontiguousarray(vd.transpose(1, 0, 2))
        pool_k = np.concatenate([gather(Kc, idx), kd], axis=1)
        pool_v = np.concatenate([gather(Vc, idx), vd], axis=1)
        Kc = np.concatenate([Kc, kd], axis=1)
        Vc = np.concatenate([Vc, vd], axis=1)
    return outs
