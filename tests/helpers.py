"""Shared pieces of the GPU parity tests: running the library, asking the
oracle the same question, and the comparison rules.

Comparison rules (the library's contract):
  * index sets: identical to the oracle's, except for swaps among entries
    whose oracle (fp64) scores differ by less than TIE_REL relative to the
    oracle's m-th score; the GPU set must be duplicate-free, in range,
    ascending and padded with -1;
  * attention outputs: within ATOL_OUT max-abs of the oracle's attention over
    the GPU's own index set (and of the oracle pipeline when the sets agree);
  * gathers: bit-exact.
"""
from __future__ import annotations

import math
from typing import Optional

import numpy as np
import torch

import oracle
import paper_2607_26475_amd as ckv
import synth

SCALE = float(np.float32(1.0 / math.sqrt(128.0)))
ATOL_OUT = 2e-3
TIE_REL = 1e-5
# fp32 dot product over 128 products plus the final scaling: |err| <= this
# factor times scale * sum_c |q_c k_c| (sequential-sum worst case).
SCORE_REL = 130 * 2.0 ** -24


def device() -> torch.device:
    assert torch.cuda.is_available(), "GPU tests need a visible MI355X"
    return torch.device("cuda:0")


def u16(t: torch.Tensor) -> np.ndarray:
    return synth.to_u16(t)


def bf2f(u: np.ndarray) -> np.ndarray:
    return (np.asarray(u, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def orc() -> oracle.Oracle:
    return oracle.get()


# Running totals of the index-set comparisons of this test session, printed
# in pytest's terminal summary (tests/conftest.py): units compared, units
# whose sets differ by tolerated near-tie swaps, the most entries swapped in
# one unit and the largest gap found, relative to |tau|.
SWAP_STATS = {"units": 0, "swapped_units": 0, "max_entries": 0, "max_gap_rel": 0.0}


def check_index_sets(gpu_idx, gpu_nsel, orc_idx, orc_nsel, S, lens, units=None):
    """Compare GPU and oracle index sets unit by unit under the near-tie rule.

    gpu_idx/orc_idx [B][Hkv][k], S the oracle's fp64 scores [B][Hkv][>=n].
    Returns the number of units whose sets differ (by tolerated swaps)."""
    B, Hkv, k = gpu_idx.shape
    if units is None:
        units = [(b, h) for b in range(B) for h in range(Hkv)]
    swaps = 0
    for b, h in units:
        n = int(lens[b])
        m = min(k, n)
        assert gpu_nsel[b, h] == m, (b, h, gpu_nsel[b, h], m)
        assert orc_nsel[b, h] == m
        P = gpu_idx[b, h, :m].astype(np.int64)
        assert np.all(gpu_idx[b, h, m:] == -1), (b, h)
        if m:
            assert P[0] >= 0 and P[-1] < n, (b, h, P[0], P[-1], n)
            assert np.all(np.diff(P) > 0), (b, h, "not ascending / duplicates")
        O = orc_idx[b, h, :m].astype(np.int64)
        SWAP_STATS["units"] += 1
        if np.array_equal(P, O):
            continue
        swaps += 1
        Su = S[b, h]
        missing = np.setdiff1d(O, P)
        extra = np.setdiff1d(P, O)
        assert len(missing) == len(extra)
        tau = Su[O].min()
        gap = Su[missing].max() - Su[extra].min()
        assert gap <= TIE_REL * abs(tau), (b, h, len(missing), gap, tau)
        SWAP_STATS["swapped_units"] += 1
        SWAP_STATS["max_entries"] = max(SWAP_STATS["max_entries"], len(missing))
        if tau != 0:
            SWAP_STATS["max_gap_rel"] = max(SWAP_STATS["max_gap_rel"], float(gap / abs(tau)))
    return swaps


def check_scores(gpu_scores, orc_scores, q_sel_u16, keys_u16, lens, G):
    """GPU fp32 scores within the fp32 dot-product bound of the oracle's;
    positions >= n_b exactly -inf."""
    B, Hkv, nmax = gpu_scores.shape
    qf = np.abs(bf2f(q_sel_u16).astype(np.float64))
    for b in range(B):
        for h in range(Hkv):
            n = int(lens[b])
            assert np.all(gpu_scores[b, h, n:] == -np.inf), (b, h)
            if n == 0:
                continue
            kf = np.abs(bf2f(keys_u16[b, h, :n]).astype(np.float64))
            mag = (qf[b, h * G:(h + 1) * G] @ kf.T).max(axis=0) * SCALE
            err = np.abs(gpu_scores[b, h, :n].astype(np.float64) - orc_scores[b, h, :n])
            assert np.all(err <= SCORE_REL * mag + 1e-30), (b, h, err.max())


def oracle_attn_over(shape_o, q_att, k_src, v_src, idx, n_sel, k):
    """Oracle attention of q_att over the rows idx of the given sources."""
    B, Hkv = shape_o.batch, shape_o.num_kv_heads
    d = shape_o.head_dim
    kb = np.zeros((B, Hkv, k, d), np.uint16)
    vb = np.zeros((B, Hkv, k, d), np.uint16)
    o = orc()
    o.gather_kv(shape_o, k_src.reshape(-1), v_src.reshape(-1), idx, n_sel, k, kb, vb)
    return o.sparse_decode_attn(shape_o, q_att, kb, vb, n_sel, k, SCALE, nthreads=8)


def make_prediction(kind, S_att, S_sel, lens, k, max_ctx, rng):
    """Host-made predicted sets [B][Hkv][k] (ascending, -1 padded) and counts."""
    B, Hkv = S_att.shape[:2]
    idx = np.full((B, Hkv, k), -1, np.int32)
    cnt = np.zeros((B, Hkv), np.int32)
    o = orc()
    for b in range(B):
        n = int(lens[b])
        m = min(k, n)
        for h in range(Hkv):
            if kind == "speculative":
                sel, mm = o.unit_select(S_sel[b, h, :n], k)
                p = sel[:mm]
            elif kind == "exact":
                sel, mm = o.unit_select(S_att[b, h, :n], k)
                p = sel[:mm]
            elif kind == "disjoint":  # the lowest-scoring positions
                p = np.sort(np.argsort(S_att[b, h, :n], kind="stable")[:m])
            elif kind == "half":  # every other selected row replaced by an unselected one
                sel, mm = o.unit_select(S_att[b, h, :n], k)
                keep = sel[:mm][::2]
                others = np.setdiff1d(np.arange(n), sel[:mm])
                extra = rng.choice(others, size=min(mm - len(keep), len(others)), replace=False)
                p = np.sort(np.concatenate([keep, extra]))
            elif kind == "empty":
                p = np.zeros(0, np.int64)
            elif kind == "beyond":  # k distinct positions anywhere in the stored rows
                p = np.sort(rng.choice(max_ctx, size=k, replace=False))
            else:
                raise KeyError(kind)
            idx[b, h, :len(p)] = p
            cnt[b, h] = len(p)
    return idx, cnt


def oracle_lowrank_buffers(shape_o, K, V, rank, u_fac, w_fac, idx_true, n_true, idx_pred,
                           n_pred, k):
    """The rows a layer with key reconstruction attends over, in idx_true
    order: for a row of idx_true also in idx_pred (a hit) its stored key, for
    a miss the key the oracle rebuilds from the factors; the stored value
    either way.  Returns bf16 bit buffers kb, vb [B][Hkv][k][d]."""
    B, Hkv, d = shape_o.batch, shape_o.num_kv_heads, shape_o.head_dim
    rec = orc().reconstruct_keys(shape_o, rank, u_fac, w_fac, idx_true, n_true, k, fill=0)
    kb = np.zeros((B, Hkv, k, d), np.uint16)
    vb = np.zeros((B, Hkv, k, d), np.uint16)
    for b in range(B):
        for h in range(Hkv):
            m = int(n_true[b, h])
            rows = idx_true[b, h, :m]
            hit = np.isin(rows, idx_pred[b, h, :max(0, min(int(n_pred[b, h]), k))])
            kb[b, h, :m] = np.where(hit[:, None], K[b, h, rows], rec[b, h, :m])
            vb[b, h, :m] = V[b, h, rows]
    return kb, vb


class Run:
    """Device buffers and one call of the fused entry point."""

    def __init__(self, w: synth.Workload, lens: torch.Tensor, dev):
        self.w = w
        B, Hq, Hkv, d, k = w.batch, w.q_heads, w.kv_heads, w.head_dim, w.k
        self.idx = torch.full((B, Hkv, k), -9, dtype=torch.int32, device=dev)
        self.n_sel = torch.full((B, Hkv), -9, dtype=torch.int32, device=dev)
        self.out = torch.full((B, Hq, d), float("nan"), dtype=torch.float32, device=dev)
        self.lens = lens

    def same_step(self, q_att, q_sel, k_score, k_src, v_src, src_kind, key_stride=None,
                  kv_stride=None):
        w = self.w
        s = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx,
                          key_row_stride=key_stride, kv_row_stride=kv_stride)
        ws = ckv.workspace(s, w.k, ckv.ENTRY_CRITICAL_KV_ATTN)
        ckv.critical_kv_attn(s, q_att, q_sel, k_score, self.lens, w.k, SCALE, k_src, v_src,
                             src_kind, None, None, None, self.idx, self.n_sel, self.out, ws)
        torch.cuda.synchronize()
        return s

    def pipelined(self, q_att, q_sel, k_score, k_buf, v_buf, n_sel_in, key_stride=None):
        w = self.w
        s = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx,
                          key_row_stride=key_stride)
        ws = ckv.workspace(s, w.k, ckv.ENTRY_CRITICAL_KV_ATTN)
        ckv.critical_kv_attn(s, q_att, q_sel, k_score, self.lens, w.k, SCALE, None, None,
                             0, k_buf, v_buf, n_sel_in, self.idx, self.n_sel, self.out, ws)
        torch.cuda.synchronize()
        return s

    def in_place(self, q_att, q_sel, k_score, k_src, v_src, src_kind, idx_in, n_sel_in,
                 kv_stride=None):
        """Pipelined over the rows idx_in of k_src/v_src, read where they are."""
        w = self.w
        s = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx, kv_row_stride=kv_stride)
        ws = ckv.workspace(s, w.k, ckv.ENTRY_CRITICAL_KV_ATTN)
        ckv.critical_kv_attn(s, q_att, q_sel, k_score, self.lens, w.k, SCALE, k_src, v_src,
                             src_kind, None, None, n_sel_in, self.idx, self.n_sel, self.out,
                             ws, idx_in=idx_in)
        torch.cuda.synchronize()
        return s

    def host(self):
        return (self.idx.cpu().numpy(), self.n_sel.cpu().numpy(), self.out.cpu().numpy())
