"""Helpers shared by the GPU parity tests: device staging of the seeded
synthetic inputs, calls through the C ABI, and comparison with the oracle."""
from __future__ import annotations

import numpy as np
import torch

import oracle
from paper_2606_21633_amd import herald as H
from paper_2606_21633_amd import synth

DEV = "cuda:0"


def to_dev(a: np.ndarray):
    """numpy (float32, uint16 = bf16 bits, int32) -> device tensor."""
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(DEV)
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def to_host(t):
    """device tensor -> numpy (bf16 -> uint16 bits)."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def f64(a: np.ndarray) -> np.ndarray:
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def budgets(lens, num=1, den=20):
    return np.array([H.budget_tokens(int(s), num, den) for s in lens], np.int32)


def seq_kv_host(inp: dict, b: int):
    """Logical [Hkv][S_b][d] K and V of sequence b (de-paged if needed)."""
    S = int(inp["seq_lens"][b])
    if "k" in inp:
        return inp["k"][b, :, :S], inp["v"][b, :, :S]
    P = inp["pages_k"].shape[2]
    pages = inp["page_table"][b, : (S + P - 1) // P]
    k = inp["pages_k"][pages].transpose(1, 0, 2, 3).reshape(inp["pages_k"].shape[1], -1,
                                                           inp["pages_k"].shape[3])
    v = inp["pages_v"][pages].transpose(1, 0, 2, 3).reshape(k.shape)
    return np.ascontiguousarray(k[:, :S]), np.ascontiguousarray(v[:, :S])


class Staged:
    """Device copies of one layer's inputs plus the C-ABI views."""

    def __init__(self, wl: synth.Workload, inp: dict):
        self.wl, self.inp = wl, inp
        self.hd = H.heads(wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.dtype)
        self.lens_h = inp["seq_lens"]
        self.lens = to_dev(self.lens_h)
        self.S_max = int(self.lens_h.max())
        self.q_sel = to_dev(inp["q_sel"])
        if "k" in inp:
            self.k, self.v = to_dev(inp["k"]), to_dev(inp["v"])
            self.kv = H.kv_view(self.k, self.v, self.lens, self.S_max)
        else:
            self.k, self.v = to_dev(inp["pages_k"]), to_dev(inp["pages_v"])
            self.pt = to_dev(inp["page_table"])
            self.kv = H.kv_view(self.k, self.v, self.lens, self.S_max, page_table=self.pt)

    def select(self, kps_h: np.ndarray, k_max: int | None = None, q_sel=None):
        wl = self.wl
        k_max = int(kps_h.max()) if k_max is None else k_max
        kps = to_dev(kps_h.astype(np.int32))
        idx = torch.full((wl.batch, wl.num_kv_heads, k_max), -7, dtype=torch.int32,
                         device=DEV)
        ws = H.workspace(H.select_workspace(self.hd, wl.batch, self.S_max), DEV)
        H.select(self.hd, wl.batch, wl.block, self.q_sel if q_sel is None else q_sel,
                 self.kv, kps, k_max, idx, ws)
        torch.cuda.synchronize()
        return idx.cpu().numpy(), kps

    def select_xq(self, x: int, kps_h: np.ndarray, k_max: int | None = None):
        wl = self.wl
        k_max = int(kps_h.max()) if k_max is None else k_max
        kps = to_dev(kps_h.astype(np.int32))
        idx = torch.full((wl.batch, wl.num_kv_heads, k_max), -7, dtype=torch.int32,
                         device=DEV)
        ws = H.workspace(H.select_xq_workspace(self.hd, wl.batch, x, self.S_max), DEV)
        H.select_xq(self.hd, wl.batch, wl.block, x, self.q_sel, self.kv, kps, k_max, idx, ws)
        torch.cuda.synchronize()
        return idx.cpu().numpy()


def assert_same_selection(got: np.ndarray, want: np.ndarray, s_hat: np.ndarray, k: int,
                          band: float = 1e-12) -> int:
    """Indices must be identical; the only tolerated difference is a swap
    among entries whose oracle importance lies within a relative `band` of
    the k-th largest (a certified near-tie, reported by the return value)."""
    if np.array_equal(got, want):
        return 0
    assert got.shape == want.shape
    g, w = set(got.tolist()), set(want.tolist())
    assert len(g) == len(got), "duplicate indices"
    diff = g ^ w
    kth = np.sort(s_hat)[::-1][k - 1]
    for s in diff:
        assert 0 <= s < s_hat.size and abs(s_hat[s] - kth) <= band * kth, (
            f"index {s} differs: s_hat={s_hat[s]!r}, k-th={kth!r}")
    assert np.array_equal(np.sort(got), got), "not ascending"
    return len(diff)


def boundary_gap(s_hat: np.ndarray, k: int) -> float:
    """Relative gap between the k-th and (k+1)-th largest importance."""
    if k >= s_hat.size:
        return float("inf")
    srt = np.sort(s_hat)[::-1]
    return float((srt[k - 1] - srt[k]) / srt[k - 1])
