"""Debug mode (MI355X only): entries check their device-side inputs on the
device before launching and every launch synchronises.  Valid calls give the
same bits as outside debug mode; each violated precondition (a context
length past max_ctx, a count above k, an index entry at or past its unit's
context length) is refused with CKV_EINVAL naming it, before any of the
entry's own kernels runs; -1 entries are accepted."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import paper_2607_26475_amd as ckv
import synth
from helpers import SCALE, device

pytestmark = pytest.mark.gpu


@pytest.fixture
def debug_mode():
    ckv.set_debug(True)
    try:
        yield
    finally:
        ckv.set_debug(False)


def _tiny():
    dev = device()
    w = synth.WORKLOADS["tiny"]
    t = synth.make_layer(w, seed=2, device=dev)
    s = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx)
    return dev, w, t, s


def _same_step(dev, w, t, s, lens):
    i32 = dict(dtype=torch.int32, device=dev)
    idx = torch.full((w.batch, w.kv_heads, w.k), -9, **i32)
    nsel = torch.full((w.batch, w.kv_heads), -9, **i32)
    out = torch.full((w.batch, w.q_heads, w.head_dim), float("nan"), device=dev)
    ws = ckv.workspace(s, w.k, ckv.ENTRY_CRITICAL_KV_ATTN)
    ckv.critical_kv_attn(s, t["q"], None, t["k"], lens, w.k, SCALE, t["k"], t["v"],
                         ckv.SRC_DEVICE, None, None, None, idx, nsel, out, ws)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), nsel.cpu().numpy(), out.cpu().numpy()


def test_debug_mode_gives_the_same_bits():
    dev, w, t, s = _tiny()
    ref = _same_step(dev, w, t, s, t["ctx_lens"])
    ckv.set_debug(True)
    try:
        got = _same_step(dev, w, t, s, t["ctx_lens"])
    finally:
        ckv.set_debug(False)
    for a, b in zip(ref, got):
        np.testing.assert_array_equal(a, b)


def _refused(fn, what):
    with pytest.raises(ckv.CkvError) as e:
        fn()
    assert e.value.status == 1 and what in str(e.value), str(e.value)  # CKV_EINVAL


def test_context_length_past_max_ctx(debug_mode):
    dev, w, t, s = _tiny()
    bad = torch.tensor([w.max_ctx + 1], dtype=torch.int32, device=dev)
    _refused(lambda: _same_step(dev, w, t, s, bad), "ctx_lens[0]")
    scores = torch.empty((w.batch, w.kv_heads, w.max_ctx), device=dev)
    _refused(lambda: ckv.score_keys(s, t["q"], t["k"], bad, SCALE, scores), "ctx_lens[0]")


def test_gather_index_and_count(debug_mode):
    dev, w, t, s = _tiny()
    U, k, d = w.units, 64, w.head_dim
    rng = np.random.default_rng(1)
    idx = np.stack([np.sort(rng.choice(w.max_ctx, k, replace=False)) for _ in range(U)])
    idx = idx.astype(np.int32).reshape(w.batch, w.kv_heads, k)
    nsel = np.full((w.batch, w.kv_heads), k, np.int32)
    kb = torch.empty((w.batch, w.kv_heads, k, d), dtype=torch.bfloat16, device=dev)
    vb = torch.empty_like(kb)

    def gather(ix, ns):
        ckv.gather_kv(s, t["k"], t["v"], ckv.SRC_DEVICE, torch.from_numpy(ix).to(dev),
                      torch.from_numpy(ns).to(dev), k, kb, vb)
        torch.cuda.synchronize()

    ok = idx.copy()
    ok[0, 1, -3:] = -1  # padding inside the count is accepted
    gather(ok, nsel)
    bad = idx.copy()
    bad[0, 1, 5] = w.max_ctx  # no context length given: the bound is max_ctx
    _refused(lambda: gather(bad, nsel), "index entry 5 of unit 1")
    past = idx.copy()
    past[0, 0, 7] = w.max_ctx + 100
    ns = nsel.copy()
    ns[0, 0] = 7  # entries past the count are not checked
    gather(past, ns)
    big = nsel.copy()
    big[0, 1] = k + 1
    _refused(lambda: gather(idx, big), "n_sel of unit 1")


def test_in_place_index_past_the_context(debug_mode):
    dev, w, t, s = _tiny()
    i32 = dict(dtype=torch.int32, device=dev)
    n = int(t["ctx_lens"][0])
    k = w.k
    idx_in = torch.arange(k, **i32).view(1, 1, k).repeat(w.batch, w.kv_heads, 1).contiguous()
    n_in = torch.full((w.batch, w.kv_heads), k, **i32)
    idx = torch.empty((w.batch, w.kv_heads, k), **i32)
    nsel = torch.empty((w.batch, w.kv_heads), **i32)
    out = torch.empty((w.batch, w.q_heads, w.head_dim), device=dev)
    ws = ckv.workspace(s, k, ckv.ENTRY_CRITICAL_KV_ATTN)
    lens = torch.tensor([k + 10], **i32)  # a context of k + 10 positions

    def call(ix):
        ckv.critical_kv_attn(s, t["q"], t["q_sel"], t["k"], lens, k, SCALE, t["k"], t["v"],
                             ckv.SRC_DEVICE, None, None, n_in, idx, nsel, out, ws, idx_in=ix)
        torch.cuda.synchronize()

    call(idx_in)
    bad = idx_in.clone()
    bad[0, 1, 3] = k + 10  # at the context length: not a position of the context
    assert k + 10 <= n
    _refused(lambda: call(bad), "index entry 3 of unit 1")
