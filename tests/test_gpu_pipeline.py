"""GPU parity of herald_decode_block, the two-stream block pipeline:

* every denoising step of every layer and block matches the oracle's
  sequential schedule (oracle.decode_blocks) within the bf16 tolerance;
* the pipelined run (selection on a second stream) is bit-identical to the
  same calls issued on one stream, also when the main stream is delayed so
  that the two streams interleave differently;
* the dense mode (no selection, attention over the whole cache) matches the
  oracle at a 100% budget;
* the appended block lands in the cache and at the tail of the next pool.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_21633_amd import herald as H
from paper_2606_21633_amd import synth
from tests.gpu_util import DEV, f64, to_dev, to_host

pytestmark = pytest.mark.gpu

TOL = 2e-2


def make_case(b=2, Hq=8, Hkv=2, d=128, B=8, T=2, L=2, nblocks=3, S_lo=900, S_hi=1500,
              seed=1, dtype="bf16", drafts=False):
    rng = np.random.default_rng(seed)
    lens = rng.integers(S_lo, S_hi, size=b, endpoint=True).astype(np.int32)
    cap = int(lens.max()) + nblocks * B

    def rnd(shape):
        return synth._to_dtype(rng.standard_normal(shape).astype(np.float32), dtype)
    layers = []
    for _ in range(L):
        k = np.zeros((b, Hkv, cap, d), np.uint16)
        v = np.zeros((b, Hkv, cap, d), np.uint16)
        for i in range(b):
            k[i, :, :lens[i]] = rnd((Hkv, int(lens[i]), d))
            v[i, :, :lens[i]] = rnd((Hkv, int(lens[i]), d))
        blocks = [dict(q=rnd((T, b, B, Hq, d)), bk=rnd((T, b, B, Hkv, d)),
                       bv=rnd((T, b, B, Hkv, d)), dk=rnd((b, B, Hkv, d)),
                       dvv=rnd((b, B, Hkv, d)), qn=rnd((b, B, Hq, d)))
                  for _ in range(nblocks)]
        if drafts:
            for blk in blocks:   # strong draft keys, so that the tail matters
                blk.update(qd=rnd((b, B, Hq, d)), ddk=synth._to_dtype(
                    3.0 * rng.standard_normal((b, B, Hkv, d)).astype(np.float32), dtype),
                    ddv=rnd((b, B, Hkv, d)))
        layers.append(dict(k=k, v=v, q_sel0=rnd((b, B, Hq, d)), blocks=blocks))
    return dict(b=b, Hq=Hq, Hkv=Hkv, d=d, B=B, T=T, L=L, nblocks=nblocks, lens=lens,
                cap=cap, layers=layers)


def run_gpu(case, dense=False, one_stream=False, delay_main=0, num=1, den=20, dense_layers=(),
            draft_layers=(), select_x=0, graphs=False):
    b, Hq, Hkv, d, B, T, L = (case[x] for x in ("b", "Hq", "Hkv", "d", "B", "T", "L"))
    hd = H.heads(Hq, Hkv, d, "bf16")
    lens_h = case["lens"].copy()
    lens = to_dev(lens_h)
    S_bound = int(lens_h.max()) + case["nblocks"] * B
    k_hi = max(H.budget_tokens(int(s), num, den) for s in lens_h + case["nblocks"] * B)
    k_hi = max(k_hi, 1)
    pcap = k_hi + B
    dl = []
    for lay in case["layers"]:
        L_ = dict(k=to_dev(lay["k"]), v=to_dev(lay["v"]))
        L_["pools"] = [[torch.zeros((b, Hkv, pcap, d), dtype=torch.bfloat16, device=DEV)
                        for _ in range(2)] for _ in range(2)]
        L_["out"] = torch.zeros((T, b, B, Hq, d), dtype=torch.bfloat16, device=DEV)
        L_["out_draft"] = torch.zeros((b, B, Hq, d), dtype=torch.bfloat16, device=DEV)
        L_["blocks"] = [{n: to_dev(a) for n, a in blk.items()} for blk in lay["blocks"]]
        # a graph keeps the input pointers it was captured with: fixed buffers
        # that every block's inputs are copied into
        L_["stage"] = {n: torch.empty_like(t) for n, t in L_["blocks"][0].items()}
        dl.append(L_)
    n_pool = [torch.zeros(b, dtype=torch.int32, device=DEV) for _ in range(2)]
    # initial selection per layer (prefill-time top-k) into pool 0
    k0 = np.array([H.budget_tokens(int(s), num, den) for s in lens_h], np.int32)
    kmax0 = int(k0.max())
    kps0 = to_dev(k0)
    if not dense:
        ws = H.workspace(H.select_workspace(hd, b, int(lens_h.max())), DEV)
        idx = torch.empty((b, Hkv, kmax0), dtype=torch.int32, device=DEV)
        for l, (lay, L_) in enumerate(zip(case["layers"], dl)):
            if l in dense_layers:
                continue
            kv = H.kv_view(L_["k"], L_["v"], lens, int(lens_h.max()))
            H.select(hd, b, B, to_dev(lay["q_sel0"]), kv, kps0, kmax0, idx, ws)
            H.gather(hd, b, kv, idx, kps0, kmax0, H.pool_view(*L_["pools"][0]))
        n_pool[0].copy_(kps0)
    torch.cuda.synchronize()
    s_main = torch.cuda.Stream(device=DEV)
    s_retr = s_main if one_stream else torch.cuda.Stream(device=DEV)
    ws = H.workspace(H.decode_block_workspace(hd, b, B, S_bound, k_hi), DEV)
    outs = []
    a = 0
    kn = torch.zeros(b, dtype=torch.int32, device=DEV)   # updated in place every block
    graph = [None, None]
    for n in range(case["nblocks"]):
        kn_h = np.array([H.budget_tokens(int(s), num, den) for s in lens_h], np.int32)
        kn.copy_(torch.from_numpy(kn_h))
        layers = []
        for l, L_ in enumerate(dl):
            blk = L_["blocks"][n]
            if graphs:
                for name, t in blk.items():
                    L_["stage"][name].copy_(t)
                blk = L_["stage"]
            layer = H.Layer(
                H.pool_view(L_["k"], L_["v"]), H.pool_view(*L_["pools"][a]),
                H.pool_view(*L_["pools"][1 - a]), blk["q"].data_ptr(), blk["bk"].data_ptr(),
                blk["bv"].data_ptr(), blk["dk"].data_ptr(), blk["dvv"].data_ptr(),
                blk["qn"].data_ptr(), L_["out"].data_ptr(), b * B * Hq * d,
                int(l in dense_layers))
            layer.select_x = select_x
            if l in draft_layers:
                layer.q_draft, layer.draft_k = blk["qd"].data_ptr(), blk["ddk"].data_ptr()
                layer.draft_v, layer.out_draft = blk["ddv"].data_ptr(), L_["out_draft"].data_ptr()
            layers.append(layer)
        torch.cuda.synchronize()
        if delay_main:
            with torch.cuda.stream(s_main):
                torch.cuda._sleep(delay_main)
        # host-side arguments that a graph fixes: the largest S and k of the run
        S_arg = int(lens_h.max()) if not graphs else S_bound - B
        k_arg = int(kn_h.max()) if not graphs else k_hi
        call = lambda: H.decode_block(hd, layers, b, B, T, lens, S_arg, n_pool[a], pcap,
                                      n_pool[1 - a], kn, k_arg, dense, ws, s_main, s_retr)
        if not graphs:
            call()
        elif graph[a] is None:
            # capture this parity's block (the capture itself runs nothing),
            # then replay it
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=s_main):
                call()
            graph[a] = (g, layers)
            torch.cuda.synchronize()
            g.replay()
        else:
            graph[a][0].replay()
        torch.cuda.synchronize()
        if graphs:   # eager work between replays
            x = torch.randn(256, 256, device=DEV)
            (x @ x).sum().item()
        outs.append([to_host(L_["out"]).copy() for L_ in dl])
        if draft_layers:
            outs[-1].append([to_host(L_["out_draft"]).copy() for L_ in dl])
        lens_h = lens_h + B
        assert np.array_equal(lens.cpu().numpy(), lens_h)
        if not dense:
            assert np.array_equal(n_pool[1 - a].cpu().numpy(), kn_h + B)
        a = 1 - a
    caches = [(to_host(L_["k"]), to_host(L_["v"])) for L_ in dl]
    return outs, caches


def oracle_outs(case, num=1, den=20, dense_layers=(), draft_layers=(), select_x=0):
    """Per layer, per sequence: oracle.decode_blocks -> [block][layer][T][b]...
    A dense layer is the same schedule at a 100% budget. Draft layers carry
    their draft KV (the next selection's normalisation tail) and draft group
    (whose outputs go to res[("draft", l, i)])."""
    res = {}
    for l, lay in enumerate(case["layers"]):
        nm, dn = (1, 1) if l in dense_layers else (num, den)
        for i in range(case["b"]):
            S = int(case["lens"][i])
            K0, V0 = lay["k"][i, :, :S], lay["v"][i, :, :S]
            k0 = oracle.budget(S, nm, dn)
            idx0, _, _, _ = oracle.select(lay["q_sel0"][i], K0, k0)
            blocks = [dict(q_steps=blk["q"][:, i], k_steps=blk["bk"][:, i],
                           v_steps=blk["bv"][:, i], k_done=blk["dk"][i], v_done=blk["dvv"][i],
                           q_next=blk["qn"][i]) for blk in lay["blocks"]]
            if l in draft_layers:
                for blk, src in zip(blocks, lay["blocks"]):
                    blk.update(q_draft=src["qd"][i], k_draft=src["ddk"][i],
                               v_draft=src["ddv"][i])
            douts = []
            x = select_x if l not in dense_layers else 0
            res[(l, i)] = oracle.decode_blocks(K0, V0, idx0, blocks, nm, dn, x=x,
                                               draft_outs=douts)
            res[("draft", l, i)] = douts
    return res


def check_against_oracle(case, outs, num=1, den=20, dense_layers=(), draft_layers=(),
                         select_x=0):
    ref = oracle_outs(case, num, den, dense_layers, draft_layers, select_x)
    worst = 0.0
    for n in range(case["nblocks"]):
        for l in range(case["L"]):
            got = f64(outs[n][l])                         # [T][b][B][Hq][d]
            for i in range(case["b"]):
                err = float(np.abs(got[:, i] - ref[(l, i)][n]).max())
                worst = max(worst, err)
                assert err <= TOL, f"block {n} layer {l} seq {i}: {err}"
                if l in draft_layers:
                    gd = f64(outs[n][case["L"]][l])[i]
                    err = float(np.abs(gd - ref[("draft", l, i)][n]).max())
                    worst = max(worst, err)
                    assert err <= TOL, f"draft group, block {n} layer {l} seq {i}: {err}"
    print(f"[pipeline] max abs err {worst:.3g}")


def test_pipeline_matches_oracle_schedule():
    case = make_case()
    outs, caches = run_gpu(case)
    check_against_oracle(case, outs)
    # the completed blocks were appended to the cache
    for l, lay in enumerate(case["layers"]):
        for i in range(case["b"]):
            S = int(case["lens"][i])
            for n, blk in enumerate(lay["blocks"]):
                rows = caches[l][0][i, :, S + n * case["B"]:S + (n + 1) * case["B"]]
                assert rows.tobytes() == np.ascontiguousarray(
                    blk["dk"][i].transpose(1, 0, 2)).tobytes()


def test_pipelined_equals_single_stream_bitwise():
    case = make_case(seed=2)
    ref, _ = run_gpu(case, one_stream=True)
    for delay in (0, 2_000_000):
        got, _ = run_gpu(case, delay_main=delay)
        for n in range(case["nblocks"]):
            for l in range(case["L"]):
                assert got[n][l].tobytes() == ref[n][l].tobytes(), (delay, n, l)


def test_dense_mode_matches_full_budget_oracle():
    case = make_case(seed=3, nblocks=2)
    outs, _ = run_gpu(case, dense=True)
    check_against_oracle(case, outs, num=1, den=1)


def test_pipeline_with_dense_first_layers():
    """Layers flagged dense keep exact attention over the growing cache (the
    oracle's schedule at a 100% budget) while the sparse layers beside them
    follow the 5% schedule; layer 0 dense, layers 1-2 sparse."""
    case = make_case(seed=5, L=3)
    outs, _ = run_gpu(case, dense_layers=(0,))
    check_against_oracle(case, outs, dense_layers=(0,))


@pytest.mark.parametrize("select_x", [0, 1])
def test_pipeline_with_drafts(select_x):
    """Draft lookahead: layers 0 and 2 run their draft group at step 1 and
    select the next block with the draft KV as normalisation tail (layer 1
    has no draft); every denoising output, every draft-group output and so
    every pool matches the oracle's schedule with drafts."""
    case = make_case(seed=7, L=3, T=3, drafts=True)
    outs, _ = run_gpu(case, draft_layers=(0, 2), select_x=select_x)
    check_against_oracle(case, outs, draft_layers=(0, 2), select_x=select_x)


def test_pipeline_with_drafts_and_a_dense_layer_bitwise_single_stream():
    case = make_case(seed=8, L=2, T=2, drafts=True)
    ref, _ = run_gpu(case, one_stream=True, draft_layers=(0, 1), dense_layers=(0,))
    got, _ = run_gpu(case, delay_main=1_000_000, draft_layers=(0, 1), dense_layers=(0,))
    for n in range(case["nblocks"]):
        for l in range(case["L"] + 1):
            a, b = got[n][l], ref[n][l]
            if isinstance(a, list):
                for x, y in zip(a, b):
                    assert x.tobytes() == y.tobytes(), (n, l)
            else:
                assert a.tobytes() == b.tobytes(), (n, l)
    check_against_oracle(case, got, dense_layers=(0,), draft_layers=(0, 1))


def test_pipeline_layer32k_shapes_one_block():
    """One pipelined block at the 8B-class layer's head layout and budget
    (2 sequences x 8192 tokens, B=32, T=2) against the oracle."""
    case = make_case(b=2, Hq=32, Hkv=8, d=128, B=32, T=2, L=1, nblocks=2, S_lo=8192,
                     S_hi=8192, seed=4)
    outs, _ = run_gpu(case)
    check_against_oracle(case, outs)


def test_pipeline_36_layer_workload_shape_sampled():
    """The 36-layer workload's per-layer shape (8 sequences x 65536 tokens,
    32 query / 8 KV heads, B=32, 5% budget) with its device-side generator,
    two layers and T=2 steps per block, two pipelined blocks; sequences 0 and
    5 of both layers are checked against the oracle's sequential schedule."""
    import dataclasses
    wl = dataclasses.replace(synth.PIPELINE_36L, layers=2, steps=2)
    b, B, T, L = wl.batch, wl.block, wl.steps, wl.layers
    Hq, Hkv, d, S0 = wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.seq_len
    nblocks = 2
    cap = S0 + (nblocks + 1) * B
    data = synth.make_device_layers(wl, DEV, capacity=cap)
    gen = data["gen"]
    hd = H.heads(Hq, Hkv, d, "bf16")
    k_hi = H.budget_tokens(cap, *wl.budget)
    pcap = k_hi + B
    lay = []
    for l in range(L):
        u = data["u"][l]
        lay.append(dict(
            k=data["k"][l], v=data["v"][l], q_sel0=synth.device_queries(wl, u, gen, (), DEV),
            pools=[[torch.zeros((b, Hkv, pcap, d), dtype=torch.bfloat16, device=DEV)
                    for _ in range(2)] for _ in range(2)],
            out=torch.zeros((T, b, B, Hq, d), dtype=torch.bfloat16, device=DEV),
            blocks=[dict(q=synth.device_queries(wl, u, gen, (T,), DEV),
                         bk=synth.device_normal(wl, gen, (T, b, B, Hkv, d), DEV),
                         bv=synth.device_normal(wl, gen, (T, b, B, Hkv, d), DEV),
                         dk=synth.device_normal(wl, gen, (b, B, Hkv, d), DEV),
                         dvv=synth.device_normal(wl, gen, (b, B, Hkv, d), DEV),
                         qn=synth.device_queries(wl, u, gen, (), DEV))
                    for _ in range(nblocks)]))
    samp = (0, 5)
    # host copies for the oracle, taken before the pipeline appends blocks
    host = {(l, i): (to_host(lay[l]["k"][i, :, :S0]), to_host(lay[l]["v"][i, :, :S0]))
            for l in range(L) for i in samp}
    lens = torch.full((b,), S0, dtype=torch.int32, device=DEV)
    k0 = H.budget_tokens(S0, *wl.budget)
    kps0 = torch.full((b,), k0, dtype=torch.int32, device=DEV)
    idx = torch.empty((b, Hkv, k0), dtype=torch.int32, device=DEV)
    wsel = H.workspace(H.select_workspace(hd, b, S0), DEV)
    for Ly in lay:
        kv = H.kv_view(Ly["k"], Ly["v"], lens, S0)
        H.select(hd, b, B, Ly["q_sel0"], kv, kps0, k0, idx, wsel)
        H.gather(hd, b, kv, idx, kps0, k0, H.pool_view(*Ly["pools"][0]))
    n_pool = [kps0.clone(), torch.zeros(b, dtype=torch.int32, device=DEV)]
    s_main, s_retr = torch.cuda.Stream(device=DEV), torch.cuda.Stream(device=DEV)
    ws = H.workspace(H.decode_block_workspace(hd, b, B, cap, k_hi), DEV)
    outs, a, S = [], 0, S0
    for n in range(nblocks):
        kn_h = H.budget_tokens(S, *wl.budget)
        kn = torch.full((b,), kn_h, dtype=torch.int32, device=DEV)
        layers = [H.Layer(H.pool_view(Ly["k"], Ly["v"]), H.pool_view(*Ly["pools"][a]),
                          H.pool_view(*Ly["pools"][1 - a]), Ly["blocks"][n]["q"].data_ptr(),
                          Ly["blocks"][n]["bk"].data_ptr(), Ly["blocks"][n]["bv"].data_ptr(),
                          Ly["blocks"][n]["dk"].data_ptr(), Ly["blocks"][n]["dvv"].data_ptr(),
                          Ly["blocks"][n]["qn"].data_ptr(), Ly["out"].data_ptr(),
                          b * B * Hq * d) for Ly in lay]
        torch.cuda.synchronize()
        H.decode_block(hd, layers, b, B, T, lens, S, n_pool[a], pcap, n_pool[1 - a], kn, kn_h,
                       False, ws, s_main, s_retr)
        torch.cuda.synchronize()
        outs.append([to_host(Ly["out"]).copy() for Ly in lay])
        S += B
        a = 1 - a
    assert int(lens[0].item()) == S0 + nblocks * B
    worst = 0.0
    for l in range(L):
        q0 = to_host(lay[l]["q_sel0"])
        blocks_h = [{k: to_host(t) for k, t in blk.items()} for blk in lay[l]["blocks"]]
        for i in samp:
            K0, V0 = host[(l, i)]
            idx0, _, _, _ = oracle.select(q0[i], K0, oracle.budget(S0, *wl.budget))
            ref = oracle.decode_blocks(
                K0, V0, idx0,
                [dict(q_steps=bh["q"][:, i], k_steps=bh["bk"][:, i], v_steps=bh["bv"][:, i],
                      k_done=bh["dk"][i], v_done=bh["dvv"][i], q_next=bh["qn"][i])
                 for bh in blocks_h], *wl.budget)
            for n in range(nblocks):
                err = float(np.abs(f64(outs[n][l][:, i]) - ref[n]).max())
                worst = max(worst, err)
                assert err <= TOL, f"layer {l} seq {i} block {n}: {err}"
    print(f"[pipeline 36L shape] max abs err {worst:.3g}")


def test_pipeline_replayed_from_hip_graphs_matches_eager():
    """One captured graph per pool parity (the active/idle pointers alternate),
    replayed block after block with eager work (a matmul and a copy) between
    replays: every replayed block's outputs, caches and pool lengths equal
    those of the eager run bit for bit."""
    case = make_case(seed=9, L=2, T=3, nblocks=4, drafts=True)
    ref, ref_caches = run_gpu(case, draft_layers=(1,), select_x=1)
    got, got_caches = run_gpu(case, draft_layers=(1,), select_x=1, graphs=True)
    for n in range(case["nblocks"]):
        for l in range(case["L"] + 1):
            a, b = got[n][l], ref[n][l]
            if isinstance(a, list):
                for x, y in zip(a, b):
                    assert x.tobytes() == y.tobytes(), (n, l)
            else:
                assert a.tobytes() == b.tobytes(), (n, l)
    for (ka, va), (kb, vb) in zip(got_caches, ref_caches):
        assert ka.tobytes() == kb.tobytes() and va.tobytes() == vb.tobytes()
