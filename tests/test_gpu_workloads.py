"""GPU parity of whole decode steps on the workloads' inputs (MI355X only).

Reduced workloads are checked on every unit; full-size layers are checked on a
seeded sample of (request, KV head) units, which are independent end to end,
so a sampled unit is a complete check of that unit.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import paper_2607_26475_amd as ckv
import synth
from helpers import (ATOL_OUT, SCALE, Run, check_index_sets, device, make_prediction,
                     oracle_attn_over, orc, u16)

pytestmark = pytest.mark.gpu


def _log(*a):
    print(*a, flush=True)


def _oracle_full(w, t, q_att, q_sel, keys, k_src, v_src, lens):
    o = orc()
    so = o.shape(w.batch, w.q_heads, w.kv_heads, w.head_dim, w.max_ctx)
    S = o.score_keys(so, q_sel, keys, lens, SCALE, nthreads=8)
    idx, n_sel = o.select_topk(so, S, lens, w.k, nthreads=8)
    return so, S, idx, n_sel


@pytest.mark.parametrize("wl", ["tiny", "llama8b_s", "dual64_s"])
def test_same_step_hbm(wl):
    """Fused same-step entry, K/V in HBM (the dual workload selects with q2)."""
    _log("same-step", wl)
    dev = device()
    w = synth.WORKLOADS[wl]
    t = synth.make_layer(w, seed=1, device=dev)
    run = Run(w, t["ctx_lens"], dev)
    run.same_step(t["q"], t["q_sel"], t["k"], t["k"], t["v"], ckv.SRC_DEVICE)
    g_idx, g_nsel, g_out = run.host()
    lens = t["ctx_lens"].cpu().numpy()
    q_att, q_sel, K, V = u16(t["q"]), u16(t["q_sel"]), u16(t["k"]), u16(t["v"])
    so, S, r_idx, r_nsel = _oracle_full(w, t, q_att, q_sel, K, K, V, lens)
    swaps = check_index_sets(g_idx, g_nsel, r_idx, r_nsel, S, lens)
    _log("  units with tolerated swaps:", swaps)
    ref_gpu_set = oracle_attn_over(so, q_att, K, V, g_idx, g_nsel, w.k)
    err = np.abs(g_out - ref_gpu_set).max()
    _log("  max abs err vs oracle over GPU set:", err)
    assert err <= ATOL_OUT
    if swaps == 0:
        _, _, r_out = orc().critical_kv_attn(so, q_att, q_sel, K, K, V, lens, w.k, SCALE,
                                             nthreads=8)
        assert np.abs(g_out - r_out).max() <= ATOL_OUT
    if w.keys == "planted":
        marked = t["marked"].cpu().numpy()
        for b in range(w.batch):
            for h in range(w.kv_heads):
                planted = set(np.nonzero(marked[b, h])[0].tolist())
                assert planted <= set(g_idx[b, h, :g_nsel[b, h]].tolist())


@pytest.mark.parametrize("wl", ["long128k_s", "dual64_s", "million_s"])
def test_pipelined_host_pinned(wl):
    """Two steps of the pipelined flow with K/V in pinned host memory:
    step t-1 selects (q_sel) -> gather from host into the layer buffer ->
    step t attends (q_att) over the buffer while selecting again."""
    _log("pipelined", wl)
    dev = device()
    w = synth.WORKLOADS[wl]
    t = synth.make_layer(w, seed=2, device=dev)
    kv_host = synth.host_kv(t["k"], t["v"])
    d = w.head_dim
    lens = t["ctx_lens"]
    # step t-1: selection only matters; attention reads the host rows in place
    prev = Run(w, lens, dev)
    prev.same_step(t["q"], t["q_sel"], t["k"], kv_host.data_ptr(),
                   kv_host.data_ptr() + 2 * d, ckv.SRC_HOST_PINNED, kv_stride=2 * d)
    # assemble the buffer from host memory
    s_kv = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx, kv_row_stride=2 * d)
    k_buf = torch.empty((w.batch, w.kv_heads, w.k, d), dtype=torch.bfloat16, device=dev)
    v_buf = torch.empty_like(k_buf)
    ckv.gather_kv(s_kv, kv_host.data_ptr(), kv_host.data_ptr() + 2 * d, ckv.SRC_HOST_PINNED,
                  prev.idx, prev.n_sel, w.k, k_buf, v_buf)
    # step t
    cur = Run(w, lens, dev)
    cur.pipelined(t["q"], t["q_sel"], t["k"], k_buf, v_buf, prev.n_sel)
    p_idx, p_nsel, p_out = prev.host()
    c_idx, c_nsel, c_out = cur.host()
    lens_h = lens.cpu().numpy()
    q_att, q_sel, K, V = u16(t["q"]), u16(t["q_sel"]), u16(t["k"]), u16(t["v"])
    so, S, r_idx, r_nsel = _oracle_full(w, t, q_att, q_sel, K, K, V, lens_h)
    for g_idx, g_nsel in ((p_idx, p_nsel), (c_idx, c_nsel)):
        swaps = check_index_sets(g_idx, g_nsel, r_idx, r_nsel, S, lens_h)
        _log("  units with tolerated swaps:", swaps)
    # step-invariant queries: the set selected at t equals the one used at t
    np.testing.assert_array_equal(c_idx, p_idx)
    ref = oracle_attn_over(so, q_att, K, V, p_idx, p_nsel, w.k)
    for out in (p_out, c_out):
        err = np.abs(out - ref).max()
        _log("  max abs err:", err)
        assert err <= ATOL_OUT
    # the assembled buffer is a bit-exact copy of the selected rows
    kb = k_buf.cpu()
    for b in range(w.batch):
        for h in range(w.kv_heads):
            m = int(p_nsel[b, h])
            rows = torch.from_numpy(p_idx[b, h, :m].astype(np.int64))
            assert torch.equal(kb[b, h, :m].view(torch.int16),
                               t["k"][b, h].cpu()[rows].view(torch.int16))


IN_PLACE_CASES = [
    ("tiny", "speculative", "separate"),
    ("llama8b_s", "half", "interleaved"),
    ("dual64_s", "beyond", "separate"),
    ("dual64_s", "empty", "interleaved"),
    ("long128k_s", "speculative", "host"),
]


@pytest.mark.parametrize("wl,kind,layout", IN_PLACE_CASES)
def test_pipelined_in_place(wl, kind, layout):
    """Pipelined entry over a set selected one step earlier and read in place
    through idx_in (no assembled buffer): out is the attention of q_att over
    exactly the rows idx_in, idx_out the selection of q_sel for the next
    step.  The earlier sets are forced from the host: the speculative query's
    own selection, half of the current query's set replaced, distinct
    positions anywhere in the stored rows (past short contexts too), none."""
    _log("pipelined in place", wl, kind, layout)
    dev = device()
    w = synth.WORKLOADS[wl]
    B, Hq, Hkv, d, k, n = w.batch, w.q_heads, w.kv_heads, w.head_dim, w.k, w.max_ctx
    t = synth.make_layer(w, seed=4, device=dev)
    lens = t["ctx_lens"]
    lens_h = lens.cpu().numpy()
    q_att, q_sel, K, V = u16(t["q"]), u16(t["q_sel"]), u16(t["k"]), u16(t["v"])
    o = orc()
    so = o.shape(B, Hq, Hkv, d, n)
    S_att = o.score_keys(so, q_att, K, lens_h, SCALE, nthreads=8)
    S_sel = o.score_keys(so, q_sel, K, lens_h, SCALE, nthreads=8)
    pred, npred = make_prediction(kind, S_att, S_sel, lens_h, k, n, np.random.default_rng(11))
    keep = None
    if layout == "host":
        keep = synth.host_kv(t["k"], t["v"])
        k_src, v_src, stride, kind_src = keep.data_ptr(), keep.data_ptr() + 2 * d, 2 * d, \
            ckv.SRC_HOST_PINNED
    elif layout == "interleaved":
        keep = synth.interleave_kv(t["k"], t["v"])
        k_src, v_src, stride, kind_src = keep.data_ptr(), keep.data_ptr() + 2 * d, 2 * d, \
            ckv.SRC_DEVICE
    else:
        k_src, v_src, stride, kind_src = t["k"], t["v"], None, ckv.SRC_DEVICE
    idx_in = torch.from_numpy(pred).to(dev)
    n_in = torch.from_numpy(npred).to(dev)
    run = Run(w, lens, dev)
    run.in_place(t["q"], t["q_sel"], t["k"], k_src, v_src, kind_src, idx_in, n_in,
                 kv_stride=stride)
    g_idx, g_nsel, g_out = run.host()
    r_idx, r_nsel = o.select_topk(so, S_sel, lens_h, k, nthreads=8)
    swaps = check_index_sets(g_idx, g_nsel, r_idx, r_nsel, S_sel, lens_h)
    _log("  units with tolerated swaps:", swaps)
    ref = oracle_attn_over(so, q_att, K, V, pred, npred, k)
    err = np.abs(g_out - ref).max()
    _log("  max abs err vs oracle over idx_in:", err)
    assert err <= ATOL_OUT
    if kind == "empty":
        assert not g_out.any()
    # the earlier set was read, not written
    np.testing.assert_array_equal(idx_in.cpu().numpy(), pred)
    del keep


@pytest.mark.parametrize("Hq,Hkv", [(8, 8), (16, 8), (64, 8), (32, 2)])
def test_fused_modes_group_sizes(Hq, Hkv):
    """The fused entry for group sizes 1, 2, 8 and 16 in both modes: same-step
    (selection then attention over the rows read in place) and pipelined in
    place (attention over the same-step call's set, selection from a second
    query).  Ragged contexts, some shorter than k."""
    _log("fused modes", Hq, Hkv)
    dev = device()
    w = synth.Workload(f"groups_{Hq}_{Hkv}", 3, Hq, Hkv, 128, 3000, 200, 512, 1, "hbm",
                       True, "normal")
    t = synth.make_layer(w, seed=7, device=dev)
    lens = torch.tensor([300, 3000, 1777], dtype=torch.int32, device=dev)  # one below k
    lens_h = lens.cpu().numpy()
    q_att, q_sel, K, V = u16(t["q"]), u16(t["q_sel"]), u16(t["k"]), u16(t["v"])
    o = orc()
    so = o.shape(w.batch, Hq, Hkv, w.head_dim, w.max_ctx)
    S_att = o.score_keys(so, q_att, K, lens_h, SCALE, nthreads=8)
    S_sel = o.score_keys(so, q_sel, K, lens_h, SCALE, nthreads=8)
    first = Run(w, lens, dev)  # selects with q_att
    first.same_step(t["q"], t["q"], t["k"], t["k"], t["v"], ckv.SRC_DEVICE)
    f_idx, f_nsel, f_out = first.host()
    r_idx, r_nsel = o.select_topk(so, S_att, lens_h, w.k, nthreads=8)
    check_index_sets(f_idx, f_nsel, r_idx, r_nsel, S_att, lens_h)
    err = np.abs(f_out - oracle_attn_over(so, q_att, K, V, f_idx, f_nsel, w.k)).max()
    _log("  same-step max abs err:", err)
    assert err <= ATOL_OUT
    second = Run(w, lens, dev)  # attends over the first set, selects with q_sel
    second.in_place(t["q"], t["q_sel"], t["k"], t["k"], t["v"], ckv.SRC_DEVICE, first.idx,
                    first.n_sel)
    s_idx, s_nsel, s_out = second.host()
    r_idx, r_nsel = o.select_topk(so, S_sel, lens_h, w.k, nthreads=8)
    check_index_sets(s_idx, s_nsel, r_idx, r_nsel, S_sel, lens_h)
    err = np.abs(s_out - oracle_attn_over(so, q_att, K, V, f_idx, f_nsel, w.k)).max()
    _log("  pipelined in place max abs err:", err)
    assert err <= ATOL_OUT


def _sampled_units(w, count, seed):
    rng = np.random.default_rng(seed)
    units = [(b, h) for b in range(w.batch) for h in range(w.kv_heads)]
    pick = rng.choice(len(units), size=min(count, len(units)), replace=False)
    return [units[i] for i in sorted(pick)]


def _check_units(w, t, g_idx, g_nsel, g_out, units, k_rows, v_rows):
    """Oracle per unit on the sampled units (independent of all others)."""
    o = orc()
    G, d = w.group, w.head_dim
    lens = t["ctx_lens"].cpu().numpy()
    q_att = u16(t["q"])
    q_sel = u16(t["q_sel"])
    for b, h in units:
        n = int(lens[b])
        keys = u16(t["k"][b, h, :n])
        S = o.unit_scores(q_sel[b, h * G:(h + 1) * G], keys, SCALE)
        r_idx, m = o.unit_select(S, w.k)
        Sfull = np.full((1, 1, n), np.nan)
        Sfull[0, 0] = S
        check_index_sets(g_idx[b:b + 1, h:h + 1], g_nsel[b:b + 1, h:h + 1],
                         r_idx[None, None], np.array([[m]]), Sfull, np.array([n]))
        sel = g_idx[b, h, :m].astype(np.int64)
        kr = u16(k_rows(b, h, sel))
        vr = u16(v_rows(b, h, sel))
        ref, _ = o.unit_attn(q_att[b, h * G:(h + 1) * G], kr, vr, SCALE)
        err = np.abs(g_out[b, h * G:(h + 1) * G] - ref).max()
        assert err <= ATOL_OUT, (b, h, err)
    _log("  checked units:", units)


@pytest.mark.parametrize("layout", ["separate", "interleaved"])
def test_full_llama8b_layer_sampled(layout):
    """One full-size Llama-8B-shaped layer (B16, 32/8 heads, n 32768, k 2048)
    through the fused same-step entry with K/V in HBM, in either layout the
    benchmark runs (separate K and V caches, or K|V interleaved per position)."""
    _log("full llama8b layer", layout)
    dev = device()
    w = synth.WORKLOADS["llama8b"]
    t = synth.make_layer(w, seed=0, layer=0, device=dev)
    d = w.head_dim
    run = Run(w, t["ctx_lens"], dev)
    if layout == "interleaved":
        kv = synth.interleave_kv(t["k"], t["v"])
        run.same_step(t["q"], t["q_sel"], kv.data_ptr(), kv.data_ptr(),
                      kv.data_ptr() + 2 * d, ckv.SRC_DEVICE, key_stride=2 * d,
                      kv_stride=2 * d)
        del kv
    else:
        run.same_step(t["q"], t["q_sel"], t["k"], t["k"], t["v"], ckv.SRC_DEVICE)
    g_idx, g_nsel, g_out = run.host()
    assert np.all(np.isfinite(g_out))
    units = _sampled_units(w, 8, seed=0)
    _check_units(w, t, g_idx, g_nsel, g_out, units,
                 lambda b, h, s: t["k"][b, h][torch.from_numpy(s).to(dev)],
                 lambda b, h, s: t["v"][b, h][torch.from_numpy(s).to(dev)])


def test_full_llama8b_pipelined_in_place_sampled():
    """One full-size Llama-8B-shaped layer in the pipelined form the benchmark
    also times: step t-1 selects from a speculative query (same-step call),
    step t attends with the current query over that set read in place from
    HBM while selecting again from the next speculative query.  Sampled units:
    the new set against the oracle's selection, the output against the
    oracle's attention over the earlier set."""
    _log("full llama8b pipelined in place")
    dev = device()
    w = synth.WORKLOADS["llama8b"]
    t = synth.make_layer(w, seed=0, layer=1, device=dev)
    G, d = w.group, w.head_dim
    g = synth.generator(w.name, 0, 1, "spec", dev)
    spec = [(0.8 * t["q"].float() + 0.6 * torch.randn(t["q"].shape, generator=g, device=dev))
            .to(torch.bfloat16) for _ in range(2)]
    prev = Run(w, t["ctx_lens"], dev)
    prev.same_step(t["q"], spec[0], t["k"], t["k"], t["v"], ckv.SRC_DEVICE)
    cur = Run(w, t["ctx_lens"], dev)
    cur.in_place(t["q"], spec[1], t["k"], t["k"], t["v"], ckv.SRC_DEVICE, prev.idx, prev.n_sel)
    p_idx, p_nsel, _ = prev.host()
    g_idx, g_nsel, g_out = cur.host()
    assert np.all(np.isfinite(g_out))
    o = orc()
    lens = t["ctx_lens"].cpu().numpy()
    q_att, q_sel = u16(t["q"]), u16(spec[1])
    units = _sampled_units(w, 8, seed=1)
    for b, h in units:
        n = int(lens[b])
        keys = u16(t["k"][b, h, :n])
        S = o.unit_scores(q_sel[b, h * G:(h + 1) * G], keys, SCALE)
        r_idx, m = o.unit_select(S, w.k)
        Sfull = np.full((1, 1, n), np.nan)
        Sfull[0, 0] = S
        check_index_sets(g_idx[b:b + 1, h:h + 1], g_nsel[b:b + 1, h:h + 1],
                         r_idx[None, None], np.array([[m]]), Sfull, np.array([n]))
        mp = int(p_nsel[b, h])
        rows = torch.from_numpy(p_idx[b, h, :mp].astype(np.int64)).to(dev)
        ref, _ = o.unit_attn(q_att[b, h * G:(h + 1) * G], u16(t["k"][b, h][rows]),
                             u16(t["v"][b, h][rows]), SCALE)
        err = np.abs(g_out[b, h * G:(h + 1) * G] - ref).max()
        assert err <= ATOL_OUT, (b, h, err)
    _log("  checked units:", units)


def test_full_million_layer_sampled():
    """One full-size million-token layer (B1, n 1048576, k 8192) with K/V in
    pinned host memory: select, gather over the host link, attend."""
    _log("full million layer")
    dev = device()
    w = synth.WORKLOADS["million"]
    t = synth.make_layer(w, seed=0, layer=0, device=dev)
    kv_host = synth.host_kv(t["k"], t["v"])
    del t["v"]
    torch.cuda.empty_cache()
    d = w.head_dim
    lens = t["ctx_lens"]
    sel = Run(w, lens, dev)
    s = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx)
    scores = torch.empty((w.batch, w.kv_heads, w.max_ctx), device=dev)
    ckv.score_keys(s, t["q_sel"], t["k"], lens, SCALE, scores)
    ws = ckv.workspace(s, w.k, ckv.ENTRY_SELECT_TOPK)
    ckv.select_topk(s, scores, lens, w.k, sel.idx, sel.n_sel, ws)
    s_kv = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx, kv_row_stride=2 * d)
    k_buf = torch.empty((w.batch, w.kv_heads, w.k, d), dtype=torch.bfloat16, device=dev)
    v_buf = torch.empty_like(k_buf)
    ckv.gather_kv(s_kv, kv_host.data_ptr(), kv_host.data_ptr() + 2 * d, ckv.SRC_HOST_PINNED,
                  sel.idx, sel.n_sel, w.k, k_buf, v_buf)
    ws_a = ckv.workspace(s, w.k, ckv.ENTRY_SPARSE_DECODE_ATTN)
    ckv.sparse_decode_attn(s, t["q"], k_buf, v_buf, sel.n_sel, w.k, SCALE, sel.out, ws_a)
    torch.cuda.synchronize()
    g_idx, g_nsel, g_out = sel.host()
    # every selected row sits in the cluster (1 % of positions, far above the rest)
    marked = t["marked"].cpu().numpy()
    for h in range(w.kv_heads):
        assert marked[0, h, g_idx[0, h, :g_nsel[0, h]]].all()
    units = _sampled_units(w, 2, seed=1)
    _check_units(w, t, g_idx, g_nsel, g_out, units,
                 lambda b, h, s_: kv_host[b, h, torch.from_numpy(s_), 0],
                 lambda b, h, s_: kv_host[b, h, torch.from_numpy(s_), 1])


def test_full_dual64_pipelined_sampled():
    """The full-size dual-token workload (B64, n_b ~ U{16384..65536}, k 2048,
    K|V host-pinned) through the pipelined fused entry, as a serving step
    runs it: the set selected from q2 one step earlier is gathered over the
    host link, then one launch attends with q1 over it while scoring q2 for
    the next step.  Sampled units against the oracle."""
    _log("full dual64 pipelined")
    dev = device()
    w = synth.WORKLOADS["dual64"]
    t = synth.make_layer(w, seed=0, layer=0, device=dev)
    kv_host = synth.host_kv(t["k"], t["v"])
    del t["v"]
    torch.cuda.empty_cache()
    d = w.head_dim
    lens = t["ctx_lens"]
    s = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx)
    # step t-1: the selection from q2
    prev = Run(w, lens, dev)
    scores = torch.empty((w.batch, w.kv_heads, w.max_ctx), device=dev)
    ckv.score_keys(s, t["q_sel"], t["k"], lens, SCALE, scores)
    ws = ckv.workspace(s, w.k, ckv.ENTRY_SELECT_TOPK)
    ckv.select_topk(s, scores, lens, w.k, prev.idx, prev.n_sel, ws)
    del scores, ws
    s_kv = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx, kv_row_stride=2 * d)
    k_buf = torch.empty((w.batch, w.kv_heads, w.k, d), dtype=torch.bfloat16, device=dev)
    v_buf = torch.empty_like(k_buf)
    ckv.gather_kv(s_kv, kv_host.data_ptr(), kv_host.data_ptr() + 2 * d, ckv.SRC_HOST_PINNED,
                  prev.idx, prev.n_sel, w.k, k_buf, v_buf)
    # step t: attention (q1) over the buffer and scoring (q2) in one launch
    cur = Run(w, lens, dev)
    cur.pipelined(t["q"], t["q_sel"], t["k"], k_buf, v_buf, prev.n_sel)
    p_idx, p_nsel, _ = prev.host()
    c_idx, c_nsel, c_out = cur.host()
    np.testing.assert_array_equal(c_idx, p_idx)  # step-invariant queries
    np.testing.assert_array_equal(c_nsel, p_nsel)
    assert np.all(np.isfinite(c_out))
    units = _sampled_units(w, 6, seed=3)
    _check_units(w, t, c_idx, c_nsel, c_out, units,
                 lambda b, h, s_: kv_host[b, h, torch.from_numpy(s_), 0],
                 lambda b, h, s_: kv_host[b, h, torch.from_numpy(s_), 1])


def test_full_long128k_decode_step_sampled():
    """The full-size long-context workload (B8, n 131072, k 4096, K|V
    host-pinned) through the two-buffer decode loop over two layers, the
    launch configuration of the benchmark's pipeline: each layer attends with
    this step's query over the set its speculative query selected a step
    earlier, gathered on the copy stream.  Sampled units against the oracle."""
    from test_gpu_pipeline import Loop

    _log("full long128k decode step")
    dev = device()
    w = synth.WORKLOADS["long128k"]
    lp = Loop(w, 2, steps=1, seed=4, dev=dev)
    lp.bootstrap()
    boot = [i.cpu().numpy() for i in lp.idx[0]], [n.cpu().numpy() for n in lp.nsel[0]]
    pipe = ckv.Pipeline()
    hist = lp.run(1, pipe)
    pipe.close()
    g_idx, g_nsel, g_out = hist[0][:3]
    o = orc()
    G = w.group
    lens = lp.lens.cpu().numpy()
    for l in range(2):
        q_att = u16(lp.q_att[1][l])
        q_sel = u16(lp.q_sel[1][l])
        for b, h in _sampled_units(w, 3, seed=5 + l):
            n = int(lens[b])
            keys = u16(lp.t[l]["k"][b, h, :n])
            # this step's selection, from its speculative query
            S = o.unit_scores(q_sel[b, h * G:(h + 1) * G], keys, SCALE)
            r_idx, m = o.unit_select(S, w.k)
            Sfull = np.full((1, 1, n), np.nan)
            Sfull[0, 0] = S
            check_index_sets(g_idx[l][b:b + 1, h:h + 1], g_nsel[l][b:b + 1, h:h + 1],
                             r_idx[None, None], np.array([[m]]), Sfull, np.array([n]))
            # this step's attention, over the set selected before it
            mp = int(boot[1][l][b, h])
            rows = torch.from_numpy(boot[0][l][b, h, :mp].astype(np.int64))
            kv = lp.kv_host[l]
            ref, _ = o.unit_attn(q_att[b, h * G:(h + 1) * G], u16(kv[b, h, rows, 0]),
                                 u16(kv[b, h, rows, 1]), SCALE)
            err = np.abs(g_out[l][b, h * G:(h + 1) * G] - ref).max()
            assert err <= ATOL_OUT, (l, b, h, err)
    _log("  checked 3 units in each of 2 layers")


def test_full_million_decode_step_sampled():
    """The full-size million-token request (B1, n 1048576, k 8192, K|V
    host-pinned) through the two-buffer decode loop over two layers, as the
    benchmark runs it: the attend-and-score launch at n = 2^20, the
    many-workgroup selection, refills of 80 workgroups, and the second layer
    reusing the histograms the first layer's selection left clear.  The
    queries are the workload's own (the 1 % cluster lies along them, so the
    cut falls inside the cluster, among near ties).  Sampled units against
    the oracle."""
    from test_gpu_pipeline import Loop

    _log("full million decode step")
    dev = device()
    w = synth.WORKLOADS["million"]
    lp = Loop(w, 2, steps=1, seed=0, dev=dev)
    for st in range(2):
        for l in range(2):
            lp.q_att[st][l] = lp.t[l]["q"]
            lp.q_sel[st][l] = lp.t[l]["q"]
    lp.bootstrap()
    boot = [i.cpu().numpy() for i in lp.idx[0]], [n.cpu().numpy() for n in lp.nsel[0]]
    pipe = ckv.Pipeline()
    ckv.profile_begin()
    hist = lp.run(1, pipe)
    kernels = ckv.profile_end()
    pipe.close()
    assert kernels["zero"][0] == 1, kernels  # the second layer found the histograms clear
    g_idx, g_nsel, g_out = hist[0][:3]
    o = orc()
    G = w.group
    lens = lp.lens.cpu().numpy()
    swaps = 0
    for l in range(2):
        q = u16(lp.t[l]["q"])
        for b, h in _sampled_units(w, 3, seed=7 + l):
            n = int(lens[b])
            keys = u16(lp.t[l]["k"][b, h, :n])
            S = o.unit_scores(q[b, h * G:(h + 1) * G], keys, SCALE)
            r_idx, m = o.unit_select(S, w.k)
            Sfull = np.full((1, 1, n), np.nan)
            Sfull[0, 0] = S
            swaps += check_index_sets(g_idx[l][b:b + 1, h:h + 1], g_nsel[l][b:b + 1, h:h + 1],
                                      r_idx[None, None], np.array([[m]]), Sfull, np.array([n]))
            mp = int(boot[1][l][b, h])
            rows = torch.from_numpy(boot[0][l][b, h, :mp].astype(np.int64))
            kv = lp.kv_host[l]
            ref, _ = o.unit_attn(q[b, h * G:(h + 1) * G], u16(kv[b, h, rows, 0]),
                                 u16(kv[b, h, rows, 1]), SCALE)
            err = np.abs(g_out[l][b, h * G:(h + 1) * G] - ref).max()
            assert err <= ATOL_OUT, (l, b, h, err)
    _log(f"  checked 3 units in each of 2 layers; units with near-tie swaps: {swaps}")
