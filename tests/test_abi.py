"""C-ABI checks that need no GPU: the library loads, exports every symbol
that include/herald.h declares, and rejects bad arguments with the
documented status codes before enqueuing anything (all calls below fail
host-side validation, so no kernel is launched)."""
import ctypes
import os
import re

import pytest

import oracle
from paper_2606_21633_amd import herald as H

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "herald.h")

pytestmark = pytest.mark.skipif(not os.path.exists(H.LIB_PATH),
                                reason="libherald.so not built")

FAKE = 0x10000  # 16-byte aligned, never dereferenced: validation fails first


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(herald_\w+)\s*\(", src)))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for fn in ("herald_select", "herald_gather", "herald_block_attn",
               "herald_decode_block"):
        assert fn in names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(H.LIB_PATH)
    for fn in declared_functions():
        assert hasattr(lib, fn), fn
    assert set(declared_functions()) == set(H.EXPORTS)


def test_status_strings():
    for st in range(5):
        assert H.lib().herald_status_string(st)


@pytest.mark.parametrize("S,num,den", [(1, 1, 20), (9, 1, 20), (10, 1, 20), (4096, 1, 20),
                                       (32768, 1, 20), (131072, 1, 20), (65536, 1, 20),
                                       (12345, 7, 100), (100, 1, 1), (100, 3, 2),
                                       (0, 1, 20), (5, 1, 0), (5, -1, 3)])
def test_budget_agrees_with_oracle(S, num, den):
    assert H.budget_tokens(S, num, den) == oracle.budget(S, num, den)


def _kv(**kw):
    kv = H.KV(k=FAKE, v=FAKE, stride_b=8 * 1024 * 128, stride_h=1024 * 128, stride_s=128,
              page_table=None, page_size=0, max_pages=0, stride_page=0, seq_lens=FAKE,
              max_seq_len=1024)
    for a, b in kw.items():
        setattr(kv, a, b)
    return kv


def _select(hd=None, batch=2, block=4, q=FAKE, kv=None, kps=FAKE, k_max=52, idx=FAKE,
            ws=FAKE * 256, ws_bytes=None):
    hd = hd or H.heads(32, 8, 128, "bf16")
    kv = kv or _kv()
    if ws_bytes is None:
        ws_bytes = H.select_workspace(hd, batch, kv.max_seq_len) - 1  # one byte short
    return H.lib().herald_select(ctypes.byref(hd), batch, block, q, ctypes.byref(kv), kps,
                                 k_max, idx, ws, ws_bytes, None)


def test_select_validation():
    assert _select() == H.ERR_WORKSPACE                       # one byte short
    assert _select(ws=None, ws_bytes=1 << 40) == H.ERR_WORKSPACE
    assert _select(ws=FAKE + 16, ws_bytes=1 << 40) == H.ERR_WORKSPACE  # not 256-aligned
    assert _select(q=None) == H.ERR_INVALID_ARG
    assert _select(q=FAKE + 2) == H.ERR_INVALID_ARG            # misaligned rows
    assert _select(kps=None) == H.ERR_INVALID_ARG
    assert _select(idx=None) == H.ERR_INVALID_ARG
    assert _select(batch=0) == H.ERR_INVALID_ARG
    assert _select(block=0) == H.ERR_INVALID_ARG
    assert _select(block=65) == H.ERR_UNSUPPORTED
    assert _select(k_max=0) == H.ERR_INVALID_ARG
    assert _select(k_max=1025) == H.ERR_INVALID_ARG            # k_max > max_seq_len
    assert _select(hd=H.heads(32, 8, 96, "bf16")) == H.ERR_UNSUPPORTED
    assert _select(hd=H.heads(30, 8, 128, "bf16")) == H.ERR_INVALID_ARG  # H_q % H_kv
    assert _select(hd=H.heads(48, 3, 128, "bf16")) == H.ERR_UNSUPPORTED  # G = 16
    assert _select(hd=H.Heads(32, 8, 128, 7)) == H.ERR_INVALID_ARG       # dtype
    assert _select(kv=_kv(k=None)) == H.ERR_INVALID_ARG
    assert _select(kv=_kv(seq_lens=None)) == H.ERR_INVALID_ARG
    assert _select(kv=_kv(max_seq_len=0)) == H.ERR_INVALID_ARG
    assert _select(kv=_kv(stride_s=100)) == H.ERR_INVALID_ARG            # < head_dim
    assert _select(kv=_kv(stride_s=132)) == H.ERR_INVALID_ARG            # rows not 16B
    assert _select(kv=_kv(page_table=FAKE, page_size=12, max_pages=100,
                          stride_page=8 * 16 * 128)) == H.ERR_INVALID_ARG  # not 2^n
    assert _select(kv=_kv(page_table=FAKE, page_size=16, max_pages=10,
                          stride_page=8 * 16 * 128)) == H.ERR_INVALID_ARG  # too few pages


def _select_xq(hd=None, batch=2, block=4, x=2, q=FAKE, kv=None, kps=FAKE, k_max=52, idx=FAKE,
               ws=FAKE * 256, ws_bytes=None):
    hd = hd or H.heads(32, 8, 128, "bf16")
    kv = kv or _kv()
    if ws_bytes is None:
        ws_bytes = H.select_xq_workspace(hd, batch, x, kv.max_seq_len) - 1  # one byte short
    return H.lib().herald_select_xq(ctypes.byref(hd), batch, block, x, q, ctypes.byref(kv),
                                    kps, k_max, idx, ws, ws_bytes, None)


def test_select_xq_validation():
    assert _select_xq() == H.ERR_WORKSPACE                    # one byte short
    assert _select_xq(ws_bytes=H.select_workspace(H.heads(32, 8, 128, "bf16"), 2, 1024)) \
        == H.ERR_WORKSPACE                                     # the x = 1 size is too small
    assert _select_xq(x=0) == H.ERR_INVALID_ARG
    assert _select_xq(x=5, ws_bytes=1 << 40) == H.ERR_INVALID_ARG   # x > block
    assert _select_xq(q=None) == H.ERR_INVALID_ARG
    assert _select_xq(q=FAKE + 2) == H.ERR_INVALID_ARG
    assert _select_xq(kps=None) == H.ERR_INVALID_ARG
    assert _select_xq(idx=None) == H.ERR_INVALID_ARG
    assert _select_xq(block=65) == H.ERR_UNSUPPORTED
    assert _select_xq(k_max=1025) == H.ERR_INVALID_ARG
    assert _select_xq(kv=_kv(k=None)) == H.ERR_INVALID_ARG
    assert _select_xq(hd=H.heads(32, 8, 96, "bf16")) == H.ERR_UNSUPPORTED


def _select_draft(x=0, draft=FAKE, n_draft=32, batch=2, block=32, ws_bytes=None, **kw):
    hd = H.heads(32, 8, 128, "bf16")
    kv = _kv()
    if ws_bytes is None:
        ws_bytes = H.select_xq_workspace(hd, batch, max(x, 1), kv.max_seq_len) - 1
    return H.lib().herald_select_draft(ctypes.byref(hd), batch, block, x, FAKE,
                                       ctypes.byref(kv), draft, n_draft, FAKE, 52, FAKE,
                                       FAKE * 256, ws_bytes, None)


def test_select_draft_validation():
    assert _select_draft() == H.ERR_WORKSPACE                     # one byte short
    assert _select_draft(x=2) == H.ERR_WORKSPACE
    assert _select_draft(x=-1, ws_bytes=1 << 40) == H.ERR_INVALID_ARG
    assert _select_draft(x=33, ws_bytes=1 << 40) == H.ERR_INVALID_ARG   # x > block
    assert _select_draft(n_draft=-1, ws_bytes=1 << 40) == H.ERR_INVALID_ARG
    assert _select_draft(n_draft=65, ws_bytes=1 << 40) == H.ERR_INVALID_ARG
    assert _select_draft(draft=None, ws_bytes=1 << 40) == H.ERR_INVALID_ARG
    assert _select_draft(draft=FAKE + 4, ws_bytes=1 << 40) == H.ERR_INVALID_ARG
    assert _select_draft(draft=None, n_draft=0) == H.ERR_WORKSPACE  # no draft: fine to here


def test_select_attn_validation():
    hd = H.heads(32, 8, 128, "bf16")

    def call(o=FAKE, dv=FAKE, n=32, v=FAKE, wsb=10):
        kv = _kv(v=v)
        return H.lib().herald_select_attn(ctypes.byref(hd), 2, 32, 1, FAKE, ctypes.byref(kv),
                                          FAKE, dv, n, FAKE, 52, FAKE, o, FAKE * 256, wsb, None)
    assert call() == H.ERR_WORKSPACE                  # valid up to the workspace
    assert call(o=None) == H.ERR_INVALID_ARG
    assert call(o=FAKE + 8) == H.ERR_INVALID_ARG
    assert call(dv=None) == H.ERR_INVALID_ARG         # the draft's V is read
    assert call(dv=None, n=0) == H.ERR_WORKSPACE
    assert call(v=None) == H.ERR_INVALID_ARG          # the cache's V is read


def test_block_attn_groups_validation():
    hd = H.heads(32, 8, 128, "bf16")
    kv = _kv(max_seq_len=1638)

    def call(groups, ws=None, ws_bytes=0, q=FAKE, batch=16):
        return H.lib().herald_block_attn_groups(ctypes.byref(hd), batch, 32, groups, q,
                                                ctypes.byref(kv), FAKE, FAKE, FAKE, ws,
                                                ws_bytes, None)
    assert call(0) == H.ERR_INVALID_ARG
    assert call(-2) == H.ERR_INVALID_ARG
    assert call(2, q=FAKE + 8) == H.ERR_INVALID_ARG
    # one sequence, two groups: the key range is split, and the partials are
    # sized for batch * groups = 2 blocks, more than for one block
    need = H.block_attn_workspace(hd, 2, 32, 1638)
    small = H.block_attn_workspace(hd, 1, 32, 1638)
    assert need > small > 256                     # so the call below fails the size check
    assert call(2, ws=FAKE * 256, ws_bytes=small, batch=1) == H.ERR_WORKSPACE
    assert call(2, ws=None, ws_bytes=1 << 40, batch=1) == H.ERR_WORKSPACE


def test_select_xq_workspace_grows_with_x():
    hd = H.heads(32, 8, 128, "bf16")
    w = [H.select_xq_workspace(hd, 16, x, 32768) for x in (1, 2, 4, 8, 16, 32)]
    assert all(a < b for a, b in zip(w, w[1:]))
    # the fp64 scores of x * G score rows per cached row dominate
    assert w[-1] >= 16 * 8 * 32768 * 32 * 4 * 8
    assert w[0] == H.select_workspace(hd, 16, 32768)
    assert H.select_xq_workspace(hd, 16, 0, 32768) == 0
    assert H.select_xq_workspace(H.heads(64, 8, 128, "bf16"), 1, 64, 100) > 0    # x G = 512
    assert H.select_xq_workspace(H.heads(64, 8, 128, "bf16"), 1, 65, 100) == 0   # x G = 520


def test_workspace_queries():
    hd = H.heads(32, 8, 128, "bf16")
    assert H.select_workspace(hd, 16, 32768) > 16 * 8 * 32768 * 8
    assert H.select_workspace(hd, 0, 32768) == 0
    assert H.select_workspace(H.heads(32, 8, 96, "bf16"), 1, 10) == 0
    assert H.block_attn_workspace(hd, 16, 32, 1670) >= 256
    assert H.block_attn_workspace(hd, 16, 0, 1670) == 0
    assert H.decode_block_workspace(hd, 8, 32, 65536, 3277) > H.select_workspace(hd, 8, 65536)


def test_gather_and_attn_validation():
    hd = H.heads(32, 8, 128, "bf16")
    kv = _kv()
    pool = H.Pool(FAKE, FAKE, 8 * 100 * 128, 100 * 128, 128, 100)
    L = H.lib()
    st = L.herald_gather(ctypes.byref(hd), 2, ctypes.byref(kv), FAKE, FAKE, 101,
                         ctypes.byref(pool), 0, None)
    assert st == H.ERR_INVALID_ARG                  # k_max beyond pool capacity
    st = L.herald_gather(ctypes.byref(hd), 2, ctypes.byref(kv), FAKE, FAKE, 50,
                         ctypes.byref(pool), 51, None)
    assert st == H.ERR_INVALID_ARG                  # dst_row0 + k_max > capacity
    st = L.herald_gather(ctypes.byref(hd), 2, ctypes.byref(_kv(v=None)), FAKE, FAKE, 50,
                         ctypes.byref(pool), 0, None)
    assert st == H.ERR_INVALID_ARG                  # gather needs V
    ctx = _kv(max_seq_len=100000)
    need = H.block_attn_workspace(hd, 2, 32, 100000)
    st = L.herald_block_attn(ctypes.byref(hd), 2, 32, FAKE, ctypes.byref(ctx), FAKE, FAKE,
                             FAKE, FAKE * 256, need - 1, None)
    assert need > 256 and st == H.ERR_WORKSPACE
    st = L.herald_block_attn(ctypes.byref(hd), 2, 32, None, ctypes.byref(ctx), FAKE, FAKE,
                             FAKE, FAKE * 256, need, None)
    assert st == H.ERR_INVALID_ARG


def test_decode_block_validation():
    hd = H.heads(32, 8, 128, "bf16")
    L = H.lib()
    cache = H.Pool(FAKE, FAKE, 8 * 2048 * 128, 2048 * 128, 128, 2048)
    pool = H.Pool(FAKE, FAKE, 8 * 200 * 128, 200 * 128, 128, 200)
    lay = H.Layer(cache, pool, pool, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0)
    arr = (H.Layer * 1)(lay)
    args = lambda **kw: dict(dict(nl=1, batch=2, block=32, steps=4, seq=FAKE, maxs=2000,
                                  na=FAKE, maxa=150, ni=FAKE, kn=FAKE, kmax=100, dense=0,
                                  ws=FAKE * 256, wsb=1 << 40), **kw)

    def call(a):
        return L.herald_decode_block(ctypes.byref(hd), a["nl"], a["batch"], a["block"],
                                     a["steps"], arr, a["seq"], a["maxs"], a["na"], a["maxa"],
                                     a["ni"], a["kn"], a["kmax"], a["dense"], a["ws"],
                                     a["wsb"], None, None)
    assert call(args(maxs=2017)) == H.ERR_INVALID_ARG   # cache capacity < S + block
    assert call(args(kmax=169)) == H.ERR_INVALID_ARG    # idle capacity < k_max + block
    assert call(args(maxa=201)) == H.ERR_INVALID_ARG    # active capacity
    assert call(args(steps=0)) == H.ERR_INVALID_ARG
    assert call(args(kn=None)) == H.ERR_INVALID_ARG
    assert call(args(wsb=10)) == H.ERR_WORKSPACE
    assert call(args(ws=FAKE * 256 + 16)) == H.ERR_WORKSPACE


def test_decode_block_draft_fields_are_validated():
    hd = H.heads(32, 8, 128, "bf16")
    cache = H.Pool(FAKE, FAKE, 8 * 2048 * 128, 2048 * 128, 128, 2048)
    pool = H.Pool(FAKE, FAKE, 8 * 200 * 128, 200 * 128, 128, 200)

    def call(steps=4, wsb=10, **fields):
        lay = H.Layer(cache, pool, pool, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0)
        for k, v in fields.items():
            setattr(lay, k, v)
        arr = (H.Layer * 1)(lay)
        return H.lib().herald_decode_block(ctypes.byref(hd), 1, 2, 32, steps, arr, FAKE, 2000,
                                           FAKE, 150, FAKE, FAKE, 100, 0, FAKE * 256, wsb,
                                           None, None)
    full = dict(q_draft=FAKE, draft_k=FAKE, draft_v=FAKE, out_draft=FAKE)
    assert call(**full) == H.ERR_WORKSPACE                      # valid up to the workspace
    assert call(select_x=1) == H.ERR_WORKSPACE
    assert call(select_x=2) == H.ERR_INVALID_ARG                # 0 or 1 only
    assert call(select_x=-1) == H.ERR_INVALID_ARG
    assert call(steps=1, **full) == H.ERR_INVALID_ARG           # the draft runs with step 1
    for missing in ("draft_k", "draft_v", "out_draft"):
        assert call(**dict(full, **{missing: None})) == H.ERR_INVALID_ARG
    assert call(**dict(full, draft_k=FAKE + 4)) == H.ERR_INVALID_ARG


def test_decode_block_dense_layers_need_no_pools():
    """A layer flagged dense keeps no pools: its null pool views pass the
    checks, while the sparse layers beside it are still checked."""
    hd = H.heads(32, 8, 128, "bf16")
    L = H.lib()
    cache = H.Pool(FAKE, FAKE, 8 * 2048 * 128, 2048 * 128, 128, 2048)
    pool = H.Pool(FAKE, FAKE, 8 * 200 * 128, 200 * 128, 128, 200)
    small = H.Pool(FAKE, FAKE, 8 * 100 * 128, 100 * 128, 128, 100)
    none = H.Pool(None, None, 0, 0, 0, 0)
    dense = H.Layer(cache, none, none, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, 0, 1)

    def call(layers):
        arr = (H.Layer * len(layers))(*layers)
        return L.herald_decode_block(ctypes.byref(hd), len(layers), 2, 32, 4, arr, FAKE, 2000,
                                     FAKE, 150, FAKE, FAKE, 100, 0, FAKE * 256, 1 << 40,
                                     None, None)
    bad = H.Layer(cache, pool, small, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0, 0)
    good = H.Layer(cache, pool, pool, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0, 0)
    assert call([dense, bad]) == H.ERR_INVALID_ARG   # idle pool of the sparse layer too small
    undense = H.Layer(cache, none, none, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, 0, 0)
    assert call([undense, good]) == H.ERR_INVALID_ARG  # same layer without the flag
    # all checks pass; without a GPU the first HIP call then fails
    assert call([dense, good]) not in (H.ERR_INVALID_ARG, H.ERR_WORKSPACE)
