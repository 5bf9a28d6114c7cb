"""GPU parity of each C-ABI entry point against the oracle (MI355X only)."""
from __future__ import annotations

import zlib

import numpy as np
import pytest
import torch

import paper_2607_26475_amd as ckv
import synth
from helpers import (ATOL_OUT, SCALE, bf2f, check_index_sets, check_scores, device, orc,
                     u16)

pytestmark = pytest.mark.gpu


def _log(*a):
    print(*a, flush=True)


# ---- score_keys ---------------------------------------------------------------
@pytest.mark.parametrize("wl", ["tiny", "llama8b_s", "dual64_s"])
def test_score_keys(wl):
    _log("score_keys", wl)
    dev = device()
    w = synth.WORKLOADS[wl]
    t = synth.make_layer(w, seed=3, device=dev)
    s = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx)
    scores = torch.full((w.batch, w.kv_heads, w.max_ctx), 7.0, device=dev)
    ckv.score_keys(s, t["q_sel"], t["k"], t["ctx_lens"], SCALE, scores)
    torch.cuda.synchronize()
    lens = t["ctx_lens"].cpu().numpy()
    q_sel, keys = u16(t["q_sel"]), u16(t["k"])
    o = orc()
    so = o.shape(w.batch, w.q_heads, w.kv_heads, w.head_dim, w.max_ctx)
    ref = o.score_keys(so, q_sel, keys, lens, SCALE, nthreads=8)
    check_scores(scores.cpu().numpy(), ref, q_sel, keys, lens, w.group)


def test_score_keys_strided_rows():
    """Key rows at stride 2d (K|V interleaved): the V half is never read."""
    _log("score_keys strided")
    dev = device()
    g = torch.Generator(device="cpu").manual_seed(11)
    B, Hq, Hkv, n, d = 2, 16, 4, 777, 128
    kv = torch.randn((B, Hkv, n, 2, d), generator=g).to(torch.bfloat16)
    kv[:, :, :, 1] = float("nan")
    q = torch.randn((B, Hq, d), generator=g).to(torch.bfloat16)
    lens = torch.tensor([777, 300], dtype=torch.int32)
    s = ckv.shape_for(B, Hq, Hkv, n, key_row_stride=2 * d)
    scores = torch.zeros((B, Hkv, n), device=dev)
    kv_d, q_d, lens_d = kv.to(dev), q.to(dev), lens.to(dev)
    ckv.score_keys(s, q_d, kv_d, lens_d, SCALE, scores)
    torch.cuda.synchronize()
    o = orc()
    so = o.shape(B, Hq, Hkv, d, n, key_row_stride=2 * d)
    ref = o.score_keys(so, u16(q), u16(kv).reshape(-1), lens.numpy(), SCALE)
    keys = u16(kv[:, :, :, 0].contiguous())
    check_scores(scores.cpu().numpy(), ref, u16(q), keys, lens.numpy(), Hq // Hkv)


# ---- select_topk ----------------------------------------------------------------
def _select_case(name):
    g = np.random.default_rng(zlib.crc32(name.encode()))
    if name == "continuous":
        B, Hkv, n, k, lens = 1, 2, 4096, 256, [4096]
        S = g.standard_normal((B, Hkv, n)).astype(np.float32)
    elif name == "ragged":
        B, Hkv, n, k, lens = 4, 2, 5000, 300, [0, 17, 4999, 301]
        S = (g.standard_normal((B, Hkv, n)) * 30).astype(np.float32)
    elif name == "ties":
        B, Hkv, n, k, lens = 2, 3, 20000, 1000, [20000, 12345]
        S = g.integers(-3, 4, size=(B, Hkv, n)).astype(np.float32) * 0.5
    elif name == "all_equal":
        B, Hkv, n, k, lens = 1, 2, 50000, 777, [50000]
        S = np.full((B, Hkv, n), 1.25, np.float32)
    elif name == "signed_zero":
        B, Hkv, n, k, lens = 1, 1, 3000, 100, [3000]
        S = np.where(g.random((B, Hkv, n)) < 0.5, -0.0, 0.0).astype(np.float32)
        S[0, 0, ::97] = -1.0
    elif name == "negative":
        B, Hkv, n, k, lens = 2, 2, 6000, 500, [6000, 4321]
        S = (-np.abs(g.standard_normal((B, Hkv, n))) - 1e-3).astype(np.float32)
    elif name == "bin_edges":
        # every unit's scores sit within a few order-key steps of the lower
        # edge of one first-digit bin (11 bits of the monotone key, both
        # signs, zeros and subnormals included), so that the bin and
        # above-bin decisions meet exact edge values and heavy ties
        bins = [5, 6, 100, 1000, 1023, 1024, 1025, 1026, 1900, 2043]
        B, Hkv, n, k = len(bins), 1, 5000, 1500
        lens = [5000, 4999, 3001, 5000, 2000, 5000, 4097, 5000, 1501, 5000]
        S = np.empty((B, Hkv, n), np.float32)
        for b, c in enumerate(bins):
            keys = np.arange((c << 21) - 3, (c << 21) + 4, dtype=np.int64)
            keys = keys[keys != 0x7FFFFFFF]  # no float has this key (-0 is +0)
            bits = np.where(keys >= 0x80000000, keys ^ 0x80000000, ~keys & 0xFFFFFFFF)
            vals = bits.astype(np.uint32).view(np.float32)
            if c == 1024:
                vals = np.append(vals, np.float32(-0.0))
            assert np.all(np.isfinite(vals))
            S[b, 0] = g.choice(vals, size=n)
    elif name == "infinities":
        # -inf scores (fp32 overflow of finite inputs) and +inf ones; in two
        # units the k-th largest score is -inf itself
        B, Hkv, n, k, lens = 2, 2, 5000, 1500, [5000, 3000]
        S = np.full((B, Hkv, n), -np.inf, np.float32)
        fin = g.permutation(n)[:1000]
        S[0, 0, fin] = g.standard_normal(1000)
        S[0, 1] = g.standard_normal(n)
        S[0, 1, g.permutation(n)[:20]] = np.inf
        mix = g.permutation(3000)
        S[1, 1, mix[:700]] = g.standard_normal(700)
        S[1, 1, mix[700:800]] = np.inf
    elif name == "budget_ge_context":
        B, Hkv, n, k, lens = 3, 2, 100, 128, [100, 64, 1]
        S = g.standard_normal((B, Hkv, n)).astype(np.float32)
    elif name == "dense_cluster":
        # the cut falls inside a block of values one ulp apart
        B, Hkv, n, k, lens = 1, 4, 70000, 1024, [70000]
        base = np.float32(150.0)
        S = g.standard_normal((B, Hkv, n)).astype(np.float32) * 10
        steps = g.integers(0, 4000, size=(B, Hkv, n // 10))
        S[:, :, : n // 10] = np.nextafter(base, np.float32(np.inf)) + steps.astype(
            np.float32) * np.spacing(base)
    elif name == "over_bitmap":
        B, Hkv, n, k, lens = 1, 1, 1100000, 8192, [1100000]
        S = g.standard_normal((B, Hkv, n)).astype(np.float32)
    else:
        raise KeyError(name)
    lens = np.array(lens, np.int32)
    for b in range(B):  # garbage beyond the context must be ignored
        S[b, :, lens[b]:] = np.nan
    return B, Hkv, n, k, lens, S


@pytest.mark.parametrize("name", ["continuous", "ragged", "ties", "all_equal",
                                  "signed_zero", "negative", "bin_edges", "infinities",
                                  "budget_ge_context", "dense_cluster", "over_bitmap"])
def test_select_topk_exact(name):
    """Same fp32 scores on both sides: the index sets must be identical."""
    _log("select_topk", name)
    dev = device()
    B, Hkv, n, k, lens, S = _select_case(name)
    s = ckv.shape_for(B, Hkv, Hkv, n)
    ws = ckv.workspace(s, k, ckv.ENTRY_SELECT_TOPK)
    ws.fill_(0xA5)  # contents on entry must not matter
    idx = torch.full((B, Hkv, k), -9, dtype=torch.int32, device=dev)
    n_sel = torch.full((B, Hkv), -9, dtype=torch.int32, device=dev)
    ckv.select_topk(s, torch.from_numpy(S).to(dev), torch.from_numpy(lens).to(dev), k, idx,
                    n_sel, ws)
    torch.cuda.synchronize()
    o = orc()
    so = o.shape(B, Hkv, Hkv, 128, n)
    ref_idx, ref_n = o.select_topk(so, S.astype(np.float64), lens, k, nthreads=8)
    np.testing.assert_array_equal(n_sel.cpu().numpy(), ref_n)
    np.testing.assert_array_equal(idx.cpu().numpy(), ref_idx)


def test_select_topk_nan_stays_in_bounds():
    """NaN scores are outside the contract (the set is then unspecified), but
    the selection must still write only inside its rows: n_sel <= m,
    ascending in-range positions before it, -1 after, nothing past idx."""
    _log("select_topk NaN scores")
    dev = device()
    g = np.random.default_rng(77)
    B, Hkv, n, k = 2, 2, 20000, 1000
    lens = np.array([20000, 7000], np.int32)
    S = g.standard_normal((B, Hkv, n)).astype(np.float32)
    S[g.random(S.shape) < 0.1] = np.nan
    S[1, 1, :] = np.nan  # a unit of NaN only
    s = ckv.shape_for(B, Hkv, Hkv, n)
    ws = ckv.workspace(s, k, ckv.ENTRY_SELECT_TOPK)
    canary = 4096
    flat = torch.full((B * Hkv * k + canary,), -7, dtype=torch.int32, device=dev)
    idx = flat[: B * Hkv * k].view(B, Hkv, k)
    n_sel = torch.full((B, Hkv), -9, dtype=torch.int32, device=dev)
    ckv.select_topk(s, torch.from_numpy(S).to(dev), torch.from_numpy(lens).to(dev), k, idx,
                    n_sel, ws)
    torch.cuda.synchronize()
    f = flat.cpu().numpy()
    assert np.all(f[B * Hkv * k:] == -7)
    I, N = idx.cpu().numpy(), n_sel.cpu().numpy()
    for b in range(B):
        for h in range(Hkv):
            m = min(k, int(lens[b]))
            ns = int(N[b, h])
            assert 0 <= ns <= m, (b, h, ns)
            row = I[b, h]
            assert np.all(np.diff(row[:ns]) > 0) and np.all(row[:ns] >= 0)
            assert np.all(row[:ns] < lens[b]) and np.all(row[ns:] == -1)


# ---- gather_kv ---------------------------------------------------------------------
@pytest.mark.parametrize("src_kind", [ckv.SRC_DEVICE, ckv.SRC_HOST_PINNED])
def test_gather_kv_exact(src_kind):
    _log("gather_kv", src_kind)
    dev = device()
    rng = np.random.default_rng(5)
    B, Hkv, n, k, d = 2, 8, 3000, 256, 128
    src = rng.integers(0, 65536, size=(B, Hkv, n, 2, d), dtype=np.uint16)
    idx = np.full((B, Hkv, k), -1, np.int32)
    n_sel = rng.integers(0, k + 1, size=(B, Hkv)).astype(np.int32)
    n_sel[0, 0], n_sel[0, 1], n_sel[1, 7] = 0, k, 1
    for b in range(B):
        for h in range(Hkv):
            idx[b, h, :n_sel[b, h]] = np.sort(rng.choice(n, n_sel[b, h], replace=False))
    src_t = torch.from_numpy(src.view(np.int16))
    if src_kind == ckv.SRC_HOST_PINNED:
        src_t = src_t.pin_memory()
    else:
        src_t = src_t.to(dev)
    k_ptr = src_t.data_ptr()
    v_ptr = k_ptr + d * 2
    s = ckv.shape_for(B, Hkv, Hkv, n, kv_row_stride=2 * d)
    kd = torch.full((B, Hkv, k, d), 0x5BCD, dtype=torch.int16, device=dev)
    vd = torch.full((B, Hkv, k, d), 0x5BCD, dtype=torch.int16, device=dev)
    ckv.gather_kv(s, k_ptr, v_ptr, src_kind, torch.from_numpy(idx).to(dev),
                  torch.from_numpy(n_sel).to(dev), k, kd, vd)
    torch.cuda.synchronize()
    o = orc()
    so = o.shape(B, Hkv, Hkv, d, n, kv_row_stride=2 * d)
    rk = np.full((B, Hkv, k, d), 0x5BCD, np.uint16)
    rv = np.full((B, Hkv, k, d), 0x5BCD, np.uint16)
    flat = src.reshape(-1)
    o.gather_kv(so, flat, flat[d:], idx, n_sel, k, rk, rv)
    np.testing.assert_array_equal(kd.cpu().numpy().view(np.uint16), rk)
    np.testing.assert_array_equal(vd.cpu().numpy().view(np.uint16), rv)


# ---- sparse_decode_attn --------------------------------------------------------------
@pytest.mark.parametrize("Hq,Hkv", [(32, 8), (8, 8), (16, 8), (64, 8), (32, 2)])
def test_sparse_decode_attn(Hq, Hkv):
    _log("sparse_decode_attn", Hq, Hkv)
    dev = device()
    g = torch.Generator(device="cpu").manual_seed(Hq * 100 + Hkv)
    B, k, d = 3, 300, 128
    q = (torch.randn((B, Hq, d), generator=g) * 2.5).to(torch.bfloat16)
    kb = torch.randn((B, Hkv, k, d), generator=g).to(torch.bfloat16)
    vb = torch.randn((B, Hkv, k, d), generator=g).to(torch.bfloat16)
    choices = [0, 1, 127, 128, 129, 256, 299, 300]
    n_sel = torch.tensor([[choices[(b * Hkv + h) % len(choices)] for h in range(Hkv)]
                          for b in range(B)], dtype=torch.int32)
    s = ckv.shape_for(B, Hq, Hkv, 4096)
    ws = ckv.workspace(s, k, ckv.ENTRY_SPARSE_DECODE_ATTN)
    out = torch.full((B, Hq, d), float("nan"), device=dev)
    ckv.sparse_decode_attn(s, q.to(dev), kb.to(dev), vb.to(dev), n_sel.to(dev), k, SCALE,
                           out, ws)
    torch.cuda.synchronize()
    o = orc()
    so = o.shape(B, Hq, Hkv, d, 4096)
    ref = o.sparse_decode_attn(so, u16(q), u16(kb), u16(vb), n_sel.numpy(), k, SCALE,
                               nthreads=8)
    got = out.cpu().numpy()
    assert np.all(np.isfinite(got))
    err = np.abs(got - ref).max()
    _log("  max abs err", err)
    assert err <= ATOL_OUT
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hkv):
            if n_sel[b, h] == 0:
                assert np.all(got[b, h * G:(h + 1) * G] == 0.0)
