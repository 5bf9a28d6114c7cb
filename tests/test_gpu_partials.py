"""Per-workgroup histograms of the scoring pass (MI355X only).

With many (request, KV head) units and contexts the fused selection handles,
the scoring pass stores one first-digit histogram per (unit, workgroup) and
the selection sums the few that cover its unit, so a call clears nothing.
These cases put 128 units on short, ragged contexts (empty, below k, equal to
k, one above, full) so that unit boundaries fall inside workgroup ranges, and
check every entry that scores with a histogram against the oracle.  The
kernel profile tells which histogram mode ran: no clearing kernel here, and
the clearing kernel for a small batch, where summing slots would cost more.
"""
from __future__ import annotations

import dataclasses

import numpy as np
import pytest
import torch

import paper_2607_26475_amd as ckv
import synth
from helpers import (ATOL_OUT, SCALE, check_index_sets, device, make_prediction,
                     oracle_attn_over, orc, u16)

pytestmark = pytest.mark.gpu


def _log(*a):
    print(*a, flush=True)


def _workload(B=16, max_ctx=3000, k=256):
    return dataclasses.replace(synth.WORKLOADS["llama8b_s"], name=f"partials{B}x{max_ctx}",
                               batch=B, max_ctx=max_ctx, ctx_min=1, k=k, layers=1)


def _layer(w, dev, seed=21):
    t = synth.make_layer(w, seed=seed, device=dev)
    lens = t["ctx_lens"].cpu()
    if w.batch >= 6:  # the edge lengths
        for b, n in enumerate([0, 100, w.k, w.k + 1, w.max_ctx]):
            lens[b] = n
    t["ctx_lens"] = lens.to(dev)
    return t


def _kernels(fn):
    ckv.profile_begin()
    fn()
    return ckv.profile_end()


def _oracle_sets(w, q, K, lens):
    o = orc()
    so = o.shape(w.batch, w.q_heads, w.kv_heads, w.head_dim, w.max_ctx)
    S = o.score_keys(so, q, K, lens, SCALE, nthreads=8)
    idx, nsel = o.select_topk(so, S, lens, w.k, nthreads=8)
    return so, S, idx, nsel


@pytest.mark.parametrize("B,max_ctx,k", [(16, 3000, 256), (32, 1500, 128), (16, 20000, 1024)])
def test_same_step_partials(B, max_ctx, k):
    _log("same-step partials", B, max_ctx, k)
    dev = device()
    w = _workload(B, max_ctx, k)
    t = _layer(w, dev)
    s = ckv.shape_for(B, w.q_heads, w.kv_heads, max_ctx)
    ws = ckv.workspace(s, k, ckv.ENTRY_CRITICAL_KV_ATTN)
    ws.fill_(0xA5)
    i32 = dict(dtype=torch.int32, device=dev)
    idx, nsel = torch.full((B, w.kv_heads, k), -9, **i32), torch.full((B, w.kv_heads), -9, **i32)
    out = torch.full((B, w.q_heads, w.head_dim), float("nan"), device=dev)

    def call():
        ckv.critical_kv_attn(s, t["q"], None, t["k"], t["ctx_lens"], k, SCALE, t["k"], t["v"],
                             ckv.SRC_DEVICE, None, None, None, idx, nsel, out, ws)

    stats = _kernels(call)
    assert "zero" not in stats, stats
    torch.cuda.synchronize()
    lens = t["ctx_lens"].cpu().numpy()
    q, K, V = u16(t["q"]), u16(t["k"]), u16(t["v"])
    so, S, r_idx, r_nsel = _oracle_sets(w, q, K, lens)
    g_idx, g_nsel = idx.cpu().numpy(), nsel.cpu().numpy()
    swaps = check_index_sets(g_idx, g_nsel, r_idx, r_nsel, S, lens)
    ref = oracle_attn_over(so, q, K, V, g_idx, g_nsel, k)
    err = np.abs(out.cpu().numpy() - ref).max()
    _log(f"  swaps {swaps}, max abs err {err:.2e}")
    assert err <= ATOL_OUT
    # a second call on the same workspace (nothing cleared in between)
    idx.fill_(-9)
    call()
    torch.cuda.synchronize()
    np.testing.assert_array_equal(idx.cpu().numpy(), g_idx)


def test_small_batch_clears_and_adds():
    _log("small batch: added histograms")
    dev = device()
    w = synth.WORKLOADS["dual64_s"]
    t = synth.make_layer(w, seed=3, device=dev)
    s = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx)
    ws = ckv.workspace(s, w.k, ckv.ENTRY_CRITICAL_KV_ATTN)
    i32 = dict(dtype=torch.int32, device=dev)
    idx, nsel = torch.empty((w.batch, w.kv_heads, w.k), **i32), torch.empty((w.batch, w.kv_heads), **i32)
    out = torch.empty((w.batch, w.q_heads, w.head_dim), device=dev)
    stats = _kernels(lambda: ckv.critical_kv_attn(
        s, t["q"], t["q_sel"], t["k"], t["ctx_lens"], w.k, SCALE, t["k"], t["v"],
        ckv.SRC_DEVICE, None, None, None, idx, nsel, out, ws))
    assert stats.get("zero", (0,))[0] == 1, stats


def test_pipelined_and_corrected_partials():
    """The dual kernel's scoring role stores slots too: pipelined selection
    from q_sel and both selections of the corrected entry."""
    _log("pipelined + corrected partials")
    dev = device()
    w = _workload(16, 3000, 256)
    t = _layer(w, dev, seed=22)
    B, Hq, Hkv, d, k, n = w.batch, w.q_heads, w.kv_heads, w.head_dim, w.k, w.max_ctx
    g = synth.generator(w.name, 22, 0, "qsel", dev)
    q_sel = (0.8 * t["q"].float() + 0.6 * torch.randn(t["q"].shape, generator=g, device=dev)
             ).to(torch.bfloat16)
    lens = t["ctx_lens"].cpu().numpy()
    q, qs, K, V = u16(t["q"]), u16(q_sel), u16(t["k"]), u16(t["v"])
    so, S_att, r_att, r_natt = _oracle_sets(w, q, K, lens)
    _, S_sel, r_sel, r_nsel = _oracle_sets(w, qs, K, lens)
    s = ckv.shape_for(B, Hq, Hkv, n)
    i32 = dict(dtype=torch.int32, device=dev)

    # pipelined: attention over a prefetched buffer, selection from q_sel
    pred, npred = make_prediction("speculative", S_att, S_sel, lens, k, n,
                                  np.random.default_rng(5))
    idx_pred, n_pred = torch.from_numpy(pred).to(dev), torch.from_numpy(npred).to(dev)
    k_buf = torch.zeros((B, Hkv, k, d), dtype=torch.bfloat16, device=dev)
    v_buf = torch.zeros_like(k_buf)
    ckv.gather_kv(s, t["k"], t["v"], ckv.SRC_DEVICE, idx_pred, n_pred, k, k_buf, v_buf)
    ws = ckv.workspace(s, k, ckv.ENTRY_CRITICAL_KV_ATTN)
    ws.fill_(0x5A)
    idx, nsel = torch.full((B, Hkv, k), -9, **i32), torch.full((B, Hkv), -9, **i32)
    out = torch.full((B, Hq, d), float("nan"), device=dev)
    stats = _kernels(lambda: ckv.critical_kv_attn(
        s, t["q"], q_sel, t["k"], t["ctx_lens"], k, SCALE, None, None, 0, k_buf, v_buf,
        n_pred, idx, nsel, out, ws))
    assert "zero" not in stats, stats
    torch.cuda.synchronize()
    check_index_sets(idx.cpu().numpy(), nsel.cpu().numpy(), r_sel, r_nsel, S_sel, lens)
    ref = orc().sparse_decode_attn(so, q, u16(k_buf), u16(v_buf), npred, k, SCALE, nthreads=8)
    assert np.abs(out.cpu().numpy() - ref).max() <= ATOL_OUT

    # corrected: the current query's own set, then the next step's from q_sel
    wsc = ckv.workspace(s, k, ckv.ENTRY_CORRECTED_ATTN)
    wsc.fill_(0x5A)
    idx_true, idx_next = torch.full((B, Hkv, k), -9, **i32), torch.full((B, Hkv, k), -9, **i32)
    n_true, n_next, hits = (torch.full((B, Hkv), -9, **i32) for _ in range(3))
    stats = _kernels(lambda: ckv.corrected_attn(
        s, t["q"], q_sel, t["k"], t["ctx_lens"], k, SCALE, t["k"], t["v"], ckv.SRC_DEVICE,
        idx_pred, n_pred, k_buf, v_buf, idx_true, n_true, hits, idx_next, n_next, out, wsc))
    assert "zero" not in stats, stats
    torch.cuda.synchronize()
    g_true, g_nt = idx_true.cpu().numpy(), n_true.cpu().numpy()
    check_index_sets(g_true, g_nt, r_att, r_natt, S_att, lens)
    check_index_sets(idx_next.cpu().numpy(), n_next.cpu().numpy(), r_sel, r_nsel, S_sel, lens)
    ref = oracle_attn_over(so, q, K, V, g_true, g_nt, k)
    assert np.abs(out.cpu().numpy() - ref).max() <= ATOL_OUT


def test_chunk_selection_partials():
    _log("chunk selection partials")
    dev = device()
    w = _workload(16, 6000, 256)
    t = _layer(w, dev, seed=23)
    B, Hq, Hkv, d, k, n = w.batch, w.q_heads, w.kv_heads, w.head_dim, w.k, w.max_ctx
    chunk = 4
    s = ckv.shape_for(B, Hq, Hkv, n)
    cmax = (n + chunk - 1) // chunk
    lm = torch.empty((B, Hkv, cmax, d), dtype=torch.bfloat16, device=dev)
    ckv.chunk_landmarks(s, chunk, t["k"], t["ctx_lens"], lm)
    ws = ckv.workspace(s, k, ckv.ENTRY_CRITICAL_KV_ATTN)
    ws.fill_(0x33)
    i32 = dict(dtype=torch.int32, device=dev)
    cidx, nch = torch.full((B, Hkv, k // chunk), -9, **i32), torch.full((B, Hkv), -9, **i32)
    rows, nrows = torch.full((B, Hkv, k), -9, **i32), torch.full((B, Hkv), -9, **i32)
    stats = _kernels(lambda: ckv.select_chunks(s, chunk, t["q"], lm, t["ctx_lens"], k, SCALE,
                                               cidx, nch, rows, nrows, ws))
    assert "zero" not in stats, stats
    torch.cuda.synchronize()
    lens = t["ctx_lens"].cpu().numpy()
    o = orc()
    so = o.shape(B, Hq, Hkv, d, n)
    r_cidx, r_nch, _, _ = o.select_chunks(so, chunk, u16(t["q"]), u16(lm), lens, k, SCALE,
                                          nthreads=8)
    # the landmark scores decide near-ties, as for positions
    clens = (lens + chunk - 1) // chunk
    sc = o.shape(B, Hq, Hkv, d, cmax)
    S = o.score_keys(sc, u16(t["q"]), u16(lm), clens, SCALE, nthreads=8)
    g_c, g_nc = cidx.cpu().numpy(), nch.cpu().numpy()
    check_index_sets(g_c, g_nc, r_cidx, r_nch, S, clens)
    g_r, g_nr = rows.cpu().numpy(), nrows.cpu().numpy()
    for b in range(B):  # the rows are the expansion of the GPU's chunks
        for h in range(Hkv):
            want, nr = o.expand_chunks(chunk, g_c[b, h, :g_nc[b, h]], int(lens[b]), k)
            assert g_nr[b, h] == nr and np.array_equal(g_r[b, h], want), (b, h)
