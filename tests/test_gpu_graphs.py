"""The fused entries captured into a HIP graph and replayed (MI355X only).

A serving loop captures a layer once and replays it every step.  Every entry
here launches kernels only (no memsets, no allocation, no host
synchronisation), so its launches can be captured.  Each test captures one
call with static buffers, then replays it several times.  Before each replay
it writes new queries into the captured buffers and runs other eager work.
It checks every replay bit for bit against the same call made eagerly.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import paper_2607_26475_amd as ckv
import synth
from helpers import SCALE, device, make_prediction, orc, u16

pytestmark = pytest.mark.gpu

REPLAYS = 4


def _log(*a):
    print(*a, flush=True)


def _queries(w, dev, step):
    g = synth.generator(w.name, 31, 0, f"graphq{step}", dev)
    q = torch.randn((w.batch, w.q_heads, w.head_dim), generator=g, device=dev).to(torch.bfloat16)
    q2 = (0.8 * q.float() + 0.6 * torch.randn(q.shape, generator=g, device=dev)).to(torch.bfloat16)
    return q, q2


def _busy(dev):
    """Unrelated eager work between replays."""
    a = torch.randn((1 << 22,), device=dev)
    return (a * 2 + 1).sum().item()


@pytest.mark.parametrize("wl", ["llama8b_s", "dual64_s"])
def test_same_step_graph(wl):
    _log("graph same-step", wl)
    dev = device()
    w = synth.WORKLOADS[wl]
    t = synth.make_layer(w, seed=9, device=dev)
    B, Hq, Hkv, d, k, n = w.batch, w.q_heads, w.kv_heads, w.head_dim, w.k, w.max_ctx
    s = ckv.shape_for(B, Hq, Hkv, n)
    ws = ckv.workspace(s, k, ckv.ENTRY_CRITICAL_KV_ATTN)
    q, q2 = (torch.empty((B, Hq, d), dtype=torch.bfloat16, device=dev) for _ in range(2))
    i32 = dict(dtype=torch.int32, device=dev)
    idx, nsel = torch.empty((B, Hkv, k), **i32), torch.empty((B, Hkv), **i32)
    out = torch.empty((B, Hq, d), device=dev)

    def call(q_att, q_sel, idx_, nsel_, out_, ws_):
        ckv.critical_kv_attn(s, q_att, q_sel, t["k"], t["ctx_lens"], k, SCALE, t["k"], t["v"],
                             ckv.SRC_DEVICE, None, None, None, idx_, nsel_, out_, ws_)

    q0, q20 = _queries(w, dev, 0)
    q.copy_(q0)
    q2.copy_(q20)
    side = torch.cuda.Stream(device=dev)
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up before capture, as torch asks
        call(q, q2, idx, nsel, out, ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        call(q, q2, idx, nsel, out, ws)
    torch.cuda.synchronize()
    # eager reference buffers of their own
    ws_e = ckv.workspace(s, k, ckv.ENTRY_CRITICAL_KV_ATTN)
    idx_e, nsel_e = torch.empty_like(idx), torch.empty_like(nsel)
    out_e = torch.empty_like(out)
    for step in range(1, REPLAYS + 1):
        qa, qs = _queries(w, dev, step)
        q.copy_(qa)
        q2.copy_(qs)
        _busy(dev)
        graph.replay()
        torch.cuda.synchronize()
        call(qa, qs, idx_e, nsel_e, out_e, ws_e)
        torch.cuda.synchronize()
        assert torch.equal(idx, idx_e), step
        assert torch.equal(nsel, nsel_e), step
        assert torch.equal(out, out_e), step
    _log(f"  {REPLAYS} replays identical to eager calls")


def test_corrected_graph():
    """The corrected entry: selection, miss gather into the buffer, attention
    with the next step's scoring, combine; the buffer is refilled from the
    prediction before every replay."""
    _log("graph corrected")
    dev = device()
    w = synth.WORKLOADS["dual64_s"]
    t = synth.make_layer(w, seed=10, device=dev)
    B, Hq, Hkv, d, k, n = w.batch, w.q_heads, w.kv_heads, w.head_dim, w.k, w.max_ctx
    kv = synth.host_kv(t["k"], t["v"])
    s = ckv.shape_for(B, Hq, Hkv, n, kv_row_stride=2 * d)
    k_src, v_src = kv.data_ptr(), kv.data_ptr() + 2 * d
    lens_h = t["ctx_lens"].cpu().numpy()
    o = orc()
    so = o.shape(B, Hq, Hkv, d, n)
    K = u16(t["k"])
    i32 = dict(dtype=torch.int32, device=dev)
    q, q2 = (torch.empty((B, Hq, d), dtype=torch.bfloat16, device=dev) for _ in range(2))
    bufs = {}

    def fresh(tag):
        bufs[tag] = dict(
            k_buf=torch.zeros((B, Hkv, k, d), dtype=torch.bfloat16, device=dev),
            v_buf=torch.zeros((B, Hkv, k, d), dtype=torch.bfloat16, device=dev),
            idx_true=torch.empty((B, Hkv, k), **i32), n_true=torch.empty((B, Hkv), **i32),
            hits=torch.empty((B, Hkv), **i32), idx_next=torch.empty((B, Hkv, k), **i32),
            n_next=torch.empty((B, Hkv), **i32), out=torch.empty((B, Hq, d), device=dev),
            ws=ckv.workspace(s, k, ckv.ENTRY_CORRECTED_ATTN))
        return bufs[tag]

    g, e = fresh("graph"), fresh("eager")
    # a fixed prediction: the speculative selection of the first queries
    qa0, qs0 = _queries(w, dev, 0)
    S_att = o.score_keys(so, u16(qa0), K, lens_h, SCALE, nthreads=8)
    S_sel = o.score_keys(so, u16(qs0), K, lens_h, SCALE, nthreads=8)
    pred, npred = make_prediction("speculative", S_att, S_sel, lens_h, k, n,
                                  np.random.default_rng(1))
    idx_pred, n_pred = torch.from_numpy(pred).to(dev), torch.from_numpy(npred).to(dev)

    def prefetch(b):
        ckv.gather_kv(s, k_src, v_src, ckv.SRC_HOST_PINNED, idx_pred, n_pred, k, b["k_buf"],
                      b["v_buf"])

    def call(q_att, q_sel, b):
        ckv.corrected_attn(s, q_att, q_sel, t["k"], t["ctx_lens"], k, SCALE, k_src, v_src,
                           ckv.SRC_HOST_PINNED, idx_pred, n_pred, b["k_buf"], b["v_buf"],
                           b["idx_true"], b["n_true"], b["hits"], b["idx_next"], b["n_next"],
                           b["out"], b["ws"])

    q.copy_(qa0)
    q2.copy_(qs0)
    side = torch.cuda.Stream(device=dev)
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        prefetch(g)
        call(q, q2, g)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        call(q, q2, g)
    torch.cuda.synchronize()
    for step in range(1, REPLAYS + 1):
        qa, qs = _queries(w, dev, step)
        q.copy_(qa)
        q2.copy_(qs)
        prefetch(g)  # the misses of the previous replay overwrote slots
        _busy(dev)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        prefetch(e)
        call(qa, qs, e)
        torch.cuda.synchronize()
        for name in ("idx_true", "n_true", "hits", "idx_next", "n_next", "out", "k_buf",
                     "v_buf"):
            assert torch.equal(g[name], e[name]), (step, name)
    _log(f"  {REPLAYS} replays identical to eager calls")


def test_decode_loop_graph():
    """Two whole pipelined decode steps (every layer's attention and next-step
    selection on the compute stream, the host gathers on the copy stream,
    the fill and release events between them) captured as one graph: each
    replay must match two eager steps of an identical loop."""
    from test_gpu_pipeline import Loop

    _log("graph decode loop")
    dev = device()
    w = synth.WORKLOADS["long128k_s"]
    layers = 4  # a captured two-buffer step needs an even number of layers
    lg = Loop(w, layers, steps=2, seed=12, dev=dev)
    le = Loop(w, layers, steps=2, seed=12, dev=dev)
    pipes = {}
    for name, lp in (("graph", lg), ("eager", le)):
        lp.bootstrap()
        pipes[name] = ckv.Pipeline()
        lp.copy.wait_stream(lp.compute)
        pipes[name].prime(lp.shape, w.k, lp.layer_io(1, 0), ckv.SRC_HOST_PINNED, lp.k_buf,
                          lp.v_buf, lp.copy)
    torch.cuda.synchronize()

    def two_steps(lp, pipe, cs):
        lp.copy.wait_stream(cs)
        for st, cur in ((1, 0), (2, 1)):
            pipe.step(lp.shape, lp.layer_io(st, cur), lp.lens, w.k, SCALE, ckv.SRC_HOST_PINNED,
                      lp.k_buf, lp.v_buf, lp.ws, cs, lp.copy)
        cs.wait_stream(lp.copy)

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        two_steps(lg, pipes["graph"], torch.cuda.current_stream())
    torch.cuda.synchronize()
    for rep in range(3):
        _busy(dev)
        # the graph does not wait for fills recorded outside it (the prime)
        torch.cuda.current_stream().wait_stream(lg.copy)
        graph.replay()
        torch.cuda.synchronize()
        two_steps(le, pipes["eager"], le.compute)
        torch.cuda.synchronize()
        for l in range(layers):
            assert torch.equal(lg.out[l], le.out[l]), (rep, l)
            for par in range(2):
                assert torch.equal(lg.idx[par][l], le.idx[par][l]), (rep, l, par)
                assert torch.equal(lg.nsel[par][l], le.nsel[par][l]), (rep, l, par)
    for p in pipes.values():
        p.close()
    _log("  3 replays of two steps identical to eager steps")


def test_decode_loop_graph_refuses_odd_layers():
    """A graph fixes each layer's buffer at capture time, so a captured
    two-buffer step over an odd number of layers would attend over another
    layer's rows at its next launch: the call is refused (CKV_EINVAL) and
    enqueues nothing."""
    from test_gpu_pipeline import Loop

    _log("graph decode loop, odd layer count")
    dev = device()
    w = synth.WORKLOADS["long128k_s"]
    lp = Loop(w, 3, steps=1, seed=13, dev=dev)
    lp.bootstrap()
    pipe = ckv.Pipeline()
    lp.copy.wait_stream(lp.compute)
    pipe.prime(lp.shape, w.k, lp.layer_io(1, 0), ckv.SRC_HOST_PINNED, lp.k_buf, lp.v_buf,
               lp.copy)
    torch.cuda.synchronize()
    raised = []
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        cs = torch.cuda.current_stream()
        lp.copy.wait_stream(cs)
        try:
            pipe.step(lp.shape, lp.layer_io(1, 0), lp.lens, w.k, SCALE, ckv.SRC_HOST_PINNED,
                      lp.k_buf, lp.v_buf, lp.ws, cs, lp.copy)
        except ckv.CkvError as e:
            raised.append(e)
        cs.wait_stream(lp.copy)
    torch.cuda.synchronize()
    pipe.close()
    assert raised and raised[0].status == 1, raised
    assert "even number of layers" in str(raised[0])
