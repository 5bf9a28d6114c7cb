"""Chunk landmarks and chunk selection against the oracle (MI355X only).

Sec. 2.2 / Sec. 4.1: chunks of adjacent rows carry fixed landmarks (here the
mean key, rounded once to bf16); the query selects chunks and the selected
chunks' rows are retrieved.  Landmarks and row lists are checked bit-exactly,
chunk sets under the near-tie rule on the oracle's chunk scores, outputs
against the oracle's attention over the GPU's rows.
"""
from __future__ import annotations

import dataclasses

import numpy as np
import pytest
import torch

import paper_2607_26475_amd as ckv
import synth
from helpers import (ATOL_OUT, SCALE, check_index_sets, device, oracle_attn_over, orc, u16)

pytestmark = pytest.mark.gpu
FILL = 0x7777


def _log(*a):
    print(*a, flush=True)


def _landmarks(s, chunk, keys, lens, dev):
    B, Hkv, n = s.batch, s.num_kv_heads, s.max_ctx
    cmax = (n + chunk - 1) // chunk
    lm = torch.full((B, Hkv, cmax, 128), FILL, dtype=torch.int16, device=dev)
    ckv.chunk_landmarks(s, chunk, keys, lens, lm)
    torch.cuda.synchronize()
    return lm


@pytest.mark.parametrize("wl,chunk,interleaved", [
    ("tiny", 1, False), ("tiny", 16, False), ("llama8b_s", 4, True),
    ("llama8b_s", 7, False), ("dual64_s", 64, True)])
def test_landmarks_exact(wl, chunk, interleaved):
    _log("landmarks", wl, chunk, interleaved)
    dev = device()
    w = synth.WORKLOADS[wl]
    t = synth.make_layer(w, seed=4, device=dev)
    d = w.head_dim
    if interleaved:
        kv = synth.interleave_kv(t["k"], t["v"])
        keys, stride = kv, 2 * d
        keys_h = u16(t["k"])
    else:
        keys, stride = t["k"], d
        keys_h = u16(t["k"])
    s = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx, key_row_stride=stride)
    lm = _landmarks(s, chunk, keys, t["ctx_lens"], dev).cpu().numpy().view(np.uint16)
    o = orc()
    so = o.shape(w.batch, w.q_heads, w.kv_heads, d, w.max_ctx)
    ref = o.chunk_landmarks(so, chunk, keys_h, t["ctx_lens"].cpu().numpy(), fill=FILL)
    assert np.array_equal(lm, ref)


# contexts of 700..1500 rows: at k 2048 every chunk of every unit is selected
# and the last chunk is partial in most units
EXTRA = {"short_s": dataclasses.replace(synth.WORKLOADS["llama8b_s"], name="short_s",
                                        max_ctx=1500, ctx_min=700),
         # group sizes 8 and 2
         "g8_s": dataclasses.replace(synth.WORKLOADS["llama8b_s"], name="g8_s", q_heads=64),
         "g2_s": dataclasses.replace(synth.WORKLOADS["llama8b_s"], name="g2_s", q_heads=16)}


def _workload(wl):
    return EXTRA[wl] if wl in EXTRA else synth.WORKLOADS[wl]


def _fused(w, chunk, k, dev):
    """Whether the call selects, expands and attends in one launch."""
    G = w.q_heads // w.kv_heads
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    return (chunk > 1 and G % 2 == 0 and G <= 8 and 512 <= k <= 2048 and k // chunk <= 1024
            and 2 * w.batch * w.kv_heads <= cus)


def _chunk_case(wl, chunk, k, seed, dev, lens=None):
    w = _workload(wl)
    t = synth.make_layer(w, seed=seed, device=dev)
    if lens is not None:  # context lengths of the batch's requests, replaced
        t["ctx_lens"] = torch.tensor(lens, dtype=torch.int32, device=dev)
    s = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx)
    lm = _landmarks(s, chunk, t["k"], t["ctx_lens"], dev)
    return w, t, s, lm


def _oracle_chunk_scores(w, chunk, q_sel_h, lm_h, lens_h):
    o = orc()
    cmax = lm_h.shape[2]
    sc = o.shape(w.batch, w.q_heads, w.kv_heads, w.head_dim, cmax)
    clens = np.array([(int(n) + chunk - 1) // chunk for n in lens_h], np.int32)
    return o.score_keys(sc, q_sel_h, lm_h, clens, SCALE, nthreads=8), clens


@pytest.mark.parametrize("wl,chunk,k,lens", [
    ("tiny", 16, 256, None), ("llama8b_s", 4, 256, None), ("llama8b_s", 7, 252, None),
    ("dual64_s", 8, 256, None), ("llama8b_s", 8, 256, (0, 5)),
    # one launch selects, expands and attends (head halves)
    ("llama8b_s", 8, 512, None), ("llama8b_s", 4, 2048, None), ("llama8b_s", 7, 700, None),
    ("long128k_s", 16, 1024, None), ("short_s", 8, 2048, None), ("dual64_s", 2, 2048, None),
    # empty contexts, one partial chunk, a partial last chunk
    ("llama8b_s", 8, 512, (0, 5)), ("llama8b_s", 8, 512, (13, 4999)),
    ("g8_s", 8, 1024, None), ("g2_s", 4, 1024, None)])
def test_chunked_kv_attn(wl, chunk, k, lens):
    """Same-step chunked decode: chunk set, rows and output, through the
    separate selection, expansion and attention kernels for small budgets and
    through the one-launch form for the others."""
    _log("chunked", wl, chunk, k, lens)
    dev = device()
    w, t, s, lm = _chunk_case(wl, chunk, k, 5, dev, lens)
    B, Hq, Hkv, d = w.batch, w.q_heads, w.kv_heads, w.head_dim
    kc = k // chunk
    i32 = dict(dtype=torch.int32, device=dev)
    cidx, rows = torch.full((B, Hkv, kc), -9, **i32), torch.full((B, Hkv, k), -9, **i32)
    nch, nrows = torch.full((B, Hkv), -9, **i32), torch.full((B, Hkv), -9, **i32)
    out = torch.full((B, Hq, d), float("nan"), device=dev)
    ws = ckv.workspace(s, k, ckv.ENTRY_CRITICAL_KV_ATTN)
    ws.fill_(0xA5)
    ckv.profile_begin()
    ckv.chunked_kv_attn(s, chunk, t["q"], t["q_sel"], lm, t["ctx_lens"], k, SCALE, t["k"],
                        t["v"], ckv.SRC_DEVICE, cidx, nch, rows, nrows, out, ws)
    kernels = ckv.profile_end()
    torch.cuda.synchronize()
    fused = _fused(w, chunk, k, dev)
    assert ("select_attn" in kernels) == fused and ("expand" in kernels) != fused, kernels
    lens_h = t["ctx_lens"].cpu().numpy()
    lm_h = lm.cpu().numpy().view(np.uint16)
    q_sel_h, q_att_h, K, V = u16(t["q_sel"]), u16(t["q"]), u16(t["k"]), u16(t["v"])
    S, clens = _oracle_chunk_scores(w, chunk, q_sel_h, lm_h, lens_h)
    o = orc()
    g_c, g_nc = cidx.cpu().numpy(), nch.cpu().numpy()
    g_r, g_nr = rows.cpu().numpy(), nrows.cpu().numpy()
    so = o.shape(B, Hq, Hkv, d, w.max_ctx)
    r_c, r_nc, r_r, r_nr = o.select_chunks(so, chunk, q_sel_h, lm_h, lens_h, k, SCALE,
                                           nthreads=8)
    swaps = check_index_sets(g_c, g_nc, r_c, r_nc, S, clens)
    for b in range(B):  # the rows are exactly the expansion of the GPU's chunks
        for h in range(Hkv):
            want, nr = o.expand_chunks(chunk, g_c[b, h, :g_nc[b, h]], int(lens_h[b]), k)
            assert g_nr[b, h] == nr and np.array_equal(g_r[b, h], want), (b, h)
    ref = oracle_attn_over(so, q_att_h, K, V, g_r, g_nr, k)
    err = np.abs(out.cpu().numpy() - ref).max()
    _log(f"  swaps {swaps}, max abs err {err:.2e}")
    assert err <= ATOL_OUT
    if swaps == 0:
        assert np.array_equal(g_r, r_r)


def test_chunk_rows_gather_from_host():
    """Pipelined flavour: the selected chunks' rows gathered from pinned host
    memory as contiguous blocks, bit-exact."""
    dev = device()
    chunk, k = 8, 256
    w, t, s, lm = _chunk_case("long128k_s", chunk, k, 6, dev)
    B, Hkv, d = w.batch, w.kv_heads, w.head_dim
    i32 = dict(dtype=torch.int32, device=dev)
    cidx, rows = torch.empty((B, Hkv, k // chunk), **i32), torch.empty((B, Hkv, k), **i32)
    nch, nrows = torch.empty((B, Hkv), **i32), torch.empty((B, Hkv), **i32)
    ws = ckv.workspace(s, k, ckv.ENTRY_CRITICAL_KV_ATTN)
    ckv.select_chunks(s, chunk, t["q_sel"], lm, t["ctx_lens"], k, SCALE, cidx, nch, rows, nrows,
                      ws)
    kv = synth.host_kv(t["k"], t["v"])
    sk = ckv.shape_for(B, w.q_heads, Hkv, w.max_ctx, kv_row_stride=2 * d)
    k_buf = torch.zeros((B, Hkv, k, d), dtype=torch.bfloat16, device=dev)
    v_buf = torch.zeros_like(k_buf)
    ckv.gather_kv(sk, kv.data_ptr(), kv.data_ptr() + 2 * d, ckv.SRC_HOST_PINNED, rows, nrows, k,
                  k_buf, v_buf)
    torch.cuda.synchronize()
    r, nr = rows.cpu().numpy(), nrows.cpu().numpy()
    kb = k_buf.cpu().view(torch.int16).numpy()
    vb = v_buf.cpu().view(torch.int16).numpy()
    K = t["k"].cpu().view(torch.int16).numpy()
    V = t["v"].cpu().view(torch.int16).numpy()
    for b in range(B):
        for h in range(Hkv):
            m = int(nr[b, h])
            # whole chunks fill the budget, but a selected last chunk may be partial
            assert min(k, int(t["ctx_lens"][b])) - chunk < m <= min(k, int(t["ctx_lens"][b]))
            assert np.array_equal(kb[b, h, :m], K[b, h, r[b, h, :m]])
            assert np.array_equal(vb[b, h, :m], V[b, h, r[b, h, :m]])
