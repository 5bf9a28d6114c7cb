"""Miss correction, ckv_corrected_attn, against the oracle (MI355X only).

Sec. 5.3 (prioritized missing KV transfer) and Sec. 5.4 (deferred reordering):
whatever the predicted set already in the buffer, the layer's output must be
the attention of the current query over its own top-k, and the buffer must
end up holding every row of that set.  The predictions here are forced from
the host: the speculative query's set (the pipeline's), the exact set, a
disjoint set (every row a miss), half of the set replaced, no prediction at
all, and a prediction reaching past short contexts.
"""
from __future__ import annotations

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


CASES = [
    ("dual64_s", "speculative", ckv.SRC_HOST_PINNED),
    ("dual64_s", "exact", ckv.SRC_DEVICE),
    ("dual64_s", "disjoint", ckv.SRC_DEVICE),
    ("llama8b_s", "half", ckv.SRC_HOST_PINNED),
    ("tiny", "empty", ckv.SRC_DEVICE),
    ("dual64_s", "beyond", ckv.SRC_DEVICE),
]


@pytest.mark.parametrize("wl,kind,src_kind", CASES)
def test_corrected_attn(wl, kind, src_kind):
    _log("corrected", wl, kind, src_kind)
    dev = device()
    w = synth.WORKLOADS[wl]
    B, Hq, Hkv, d, k, n = w.batch, w.q_heads, w.kv_heads, w.head_dim, w.k, w.max_ctx
    t = synth.make_layer(w, seed=3, device=dev)
    lens = t["ctx_lens"]
    lens_h = lens.cpu().numpy()
    q_att, q_sel, K, V = u16(t["q"]), u16(t["q_sel"]), u16(t["k"]), u16(t["v"])
    o = orc()
    so = o.shape(B, Hq, Hkv, d, n)
    S_att = o.score_keys(so, q_att, K, lens_h, SCALE, nthreads=8)
    S_sel = o.score_keys(so, q_sel, K, lens_h, SCALE, nthreads=8)
    pred, npred = make_prediction(kind, S_att, S_sel, lens_h, k, n, np.random.default_rng(7))

    if src_kind == ckv.SRC_HOST_PINNED:
        kv = synth.host_kv(t["k"], t["v"])
        k_src, v_src, stride = kv.data_ptr(), kv.data_ptr() + 2 * d, 2 * d
    else:
        k_src, v_src, stride = t["k"], t["v"], d
    s = ckv.shape_for(B, Hq, Hkv, n, kv_row_stride=stride)
    idx_pred = torch.from_numpy(pred).to(dev)
    n_pred = torch.from_numpy(npred).to(dev)
    k_buf = torch.zeros((B, Hkv, k, d), dtype=torch.bfloat16, device=dev)
    v_buf = torch.zeros_like(k_buf)
    ckv.gather_kv(s, k_src, v_src, src_kind, idx_pred, n_pred, k, k_buf, v_buf)  # the prefetch
    i32 = dict(dtype=torch.int32, device=dev)
    idx_true, idx_next = torch.full((B, Hkv, k), -9, **i32), torch.full((B, Hkv, k), -9, **i32)
    n_true, n_next, hits = (torch.full((B, Hkv), -9, **i32) for _ in range(3))
    out = torch.full((B, Hq, d), float("nan"), device=dev)
    ws = ckv.workspace(s, k, ckv.ENTRY_CORRECTED_ATTN)
    ws.fill_(0xA5)
    ckv.corrected_attn(s, t["q"], t["q_sel"], t["k"], lens, k, SCALE, k_src, v_src, src_kind,
                       idx_pred, n_pred, k_buf, v_buf, idx_true, n_true, hits, idx_next,
                       n_next, out, ws)
    torch.cuda.synchronize()
    g_true, g_nt = idx_true.cpu().numpy(), n_true.cpu().numpy()
    g_next, g_nn = idx_next.cpu().numpy(), n_next.cpu().numpy()
    g_hits, g_out = hits.cpu().numpy(), out.cpu().numpy()

    r_true, r_nt = o.select_topk(so, S_att, lens_h, k, nthreads=8)
    swaps = check_index_sets(g_true, g_nt, r_true, r_nt, S_att, lens_h)
    r_next, r_nn = o.select_topk(so, S_sel, lens_h, k, nthreads=8)
    check_index_sets(g_next, g_nn, r_next, r_nn, S_sel, lens_h)
    total = found = 0
    for b in range(B):
        for h in range(Hkv):
            want = len(np.intersect1d(g_true[b, h, :g_nt[b, h]], pred[b, h, :npred[b, h]]))
            assert g_hits[b, h] == want, (b, h, g_hits[b, h], want)
            total += g_nt[b, h]
            found += want
    if kind == "exact":
        assert found == total
    if kind in ("empty",):
        assert found == 0
    # the output is the current query's attention over its own set
    ref = oracle_attn_over(so, q_att, K, V, g_true, g_nt, k)
    err = np.abs(g_out - ref).max()
    _log(f"  hit rate {found / max(total, 1):.3f}, swaps {swaps}, max abs err {err:.2e}")
    assert err <= ATOL_OUT
    if swaps == 0:
        _, _, r_out = o.critical_kv_attn(so, q_att, q_att, K, K, V, lens_h, k, SCALE,
                                         nthreads=8)
        assert np.abs(g_out - r_out).max() <= ATOL_OUT
    # the buffer holds every selected row (each selected K row is in some slot)
    kb = k_buf.cpu().view(torch.int16).numpy()
    for b in range(B):
        for h in range(Hkv):
            m = int(g_nt[b, h])
            rows = {kb[b, h, s_].tobytes() for s_ in range(k)}
            for p in g_true[b, h, :m]:
                assert K[b, h, p].view(np.int16).tobytes() in rows, (b, h, p)
