"""The two-buffer decode loop (ckv_decode_step) against the oracle, and its
stream ordering under injected delays (MI355X only).

Semantics checked, per layer l and step t (Sec. 4.1, Sec. 5.3, Sec. 5.4):
  out_t[l]  = attention of q_att_t[l] over the rows selected at step t-1
  idx_t[l]  = top-k of the scores of q_sel_t[l]
with the selection before the first step made from a bootstrap query (the
pre-decoding step).  Queries change from step to step, so a buffer holding
the wrong layer's or the wrong step's rows shows up in the outputs.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import paper_2607_26475_amd as ckv
import synth
from helpers import (ATOL_OUT, SCALE, check_index_sets, device, oracle_attn_over,
                     oracle_lowrank_buffers, orc, u16)

pytestmark = pytest.mark.gpu


def _log(*a):
    print(*a, flush=True)


class Loop:
    """Inputs and state of a pipelined decode over L layers of one workload."""

    def __init__(self, w, layers, steps, seed, dev):
        self.w, self.L, self.dev = w, layers, dev
        d = w.head_dim
        B, Hq, Hkv, k = w.batch, w.q_heads, w.kv_heads, w.k
        self.t = [synth.make_layer(w, seed=seed, layer=l, device=dev) for l in range(layers)]
        self.lens = self.t[0]["ctx_lens"]
        for t in self.t:
            assert torch.equal(t["ctx_lens"], self.lens)
        self.kv_host = [synth.host_kv(t["k"], t["v"]) for t in self.t]
        # per step (0 = bootstrap selection) the attending and selecting queries
        self.q_att, self.q_sel = [], []
        for s in range(steps + 1):
            qa, qs = [], []
            for l in range(layers):
                g = synth.generator(w.name, seed, l, f"step{s}", dev)
                a = torch.randn((B, Hq, d), generator=g, device=dev).to(torch.bfloat16)
                b = (0.8 * a.float() + 0.6 * torch.randn((B, Hq, d), generator=g, device=dev)
                     ).to(torch.bfloat16)
                qa.append(a)
                qs.append(b)
            self.q_att.append(qa)
            self.q_sel.append(qs)
        mk = lambda: [torch.full((B, Hkv, k), -9, dtype=torch.int32, device=dev)
                      for _ in range(layers)]
        mn = lambda: [torch.full((B, Hkv), -9, dtype=torch.int32, device=dev)
                      for _ in range(layers)]
        self.idx = [mk(), mk()]
        self.nsel = [mn(), mn()]
        self.out = [torch.full((B, Hq, d), float("nan"), device=dev) for _ in range(layers)]
        self.corrected = False
        self.lowrank = {}  # layer -> (rank, u_fac, w_fac): misses' keys rebuilt
        self.idx_true = mk()
        self.n_true = mn()
        self.hits = mn()
        self.k_buf = [torch.empty((B, Hkv, k, d), dtype=torch.bfloat16, device=dev)
                      for _ in range(2)]
        self.v_buf = [torch.empty_like(self.k_buf[0]) for _ in range(2)]
        self.shape = ckv.shape_for(B, Hq, Hkv, w.max_ctx, kv_row_stride=2 * d)
        self.ws = ckv.workspace(self.shape, k, ckv.ENTRY_DECODE_STEP)
        self.chunk, self.lms = 1, None      # chunked layers: set_chunked()
        self.chunk_layers = None            # the chunked layers (None: all of them)
        self.two, self.local = False, None  # two-token layers: set_two_tokens()
        self.two_layers = None              # the two-token layers (None: all of them)
        self.out_spec = [torch.full((B, Hq, d), float("nan"), device=dev) for _ in range(layers)]
        self.in_place = False               # rows read from the device caches, no buffers
        self.copy = torch.cuda.Stream(device=dev)
        self.compute = torch.cuda.current_stream(dev)

    def layer_io(self, step, cur):
        d = self.w.head_dim
        nxt = 1 - cur
        return [{"q_att": self.q_att[step][l], "q_sel": self.q_sel[step][l],
                 "k_score": self.t[l]["k"], "k_src": self.kv_host[l].data_ptr(),
                 "v_src": self.kv_host[l].data_ptr() + 2 * d,
                 "idx_prev": self.idx[cur][l], "n_sel_prev": self.nsel[cur][l],
                 "idx_next": self.idx[nxt][l], "n_sel_next": self.nsel[nxt][l],
                 "out": self.out[l],
                 "idx_true": self.idx_true[l] if self.corrected else None,
                 "n_true": self.n_true[l] if self.corrected else None,
                 "hits": self.hits[l] if self.corrected else None,
                 "lr_rank": self.lowrank[l][0] if l in self.lowrank else 0,
                 "lr_u": self.lowrank[l][1] if l in self.lowrank else None,
                 "lr_w": self.lowrank[l][2] if l in self.lowrank else None,
                 "chunk": self.chunk if self.chunked(l) else 1,
                 "landmarks": self.lms[l] if self.chunked(l) else None,
                 "k_local": self.local[step][l][0] if self.two_token(l) else None,
                 "v_local": self.local[step][l][1] if self.two_token(l) else None,
                 "out_spec": self.out_spec[l] if self.two_token(l) else None}
                for l in range(self.L)]

    def two_token(self, l):
        return self.two and (self.two_layers is None or l in self.two_layers)

    def chunked(self, l):
        return self.chunk > 1 and (self.chunk_layers is None or l in self.chunk_layers)

    def set_chunked(self, chunk):
        """Chunked layers: landmarks of `chunk` rows of every layer's keys."""
        w, dev = self.w, self.dev
        s = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx)
        cmax = (w.max_ctx + chunk - 1) // chunk
        self.chunk = chunk
        self.lms = []
        for l in range(self.L):
            lm = torch.empty((w.batch, w.kv_heads, cmax, w.head_dim), dtype=torch.bfloat16,
                             device=dev)
            ckv.chunk_landmarks(s, chunk, self.t[l]["k"], self.lens, lm)
            self.lms.append(lm)
        torch.cuda.synchronize()

    def set_two_tokens(self, steps):
        """Two-token layers: the current and the speculative token's own K/V
        rows per (step, layer), [B][Hkv][2][d]."""
        w, dev = self.w, self.dev
        self.two = True
        self.local = []
        for st in range(steps + 1):
            row = []
            for l in range(self.L):
                g = synth.generator(w.name, 99, l, f"local{st}", dev)
                shp = (w.batch, w.kv_heads, 2, w.head_dim)
                row.append((torch.randn(shp, generator=g, device=dev).to(torch.bfloat16),
                            torch.randn(shp, generator=g, device=dev).to(torch.bfloat16)))
            self.local.append(row)

    def bootstrap(self):
        """Selection before the first step (the pre-decoding step), into set 0."""
        w = self.w
        s = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx)
        if self.chunk > 1:
            ws = ckv.workspace(s, w.k, ckv.ENTRY_CRITICAL_KV_ATTN)
            i32 = dict(dtype=torch.int32, device=self.dev)
            cidx = torch.empty((w.batch, w.kv_heads, w.k // self.chunk), **i32)
            nch = torch.empty((w.batch, w.kv_heads), **i32)
            for l in range(self.L):
                ckv.select_chunks(s, self.chunk, self.q_sel[0][l], self.lms[l], self.lens, w.k,
                                  SCALE, cidx, nch, self.idx[0][l], self.nsel[0][l], ws)
            torch.cuda.synchronize()
            return
        scores = torch.empty((w.batch, w.kv_heads, w.max_ctx), device=self.dev)
        ws = ckv.workspace(s, w.k, ckv.ENTRY_SELECT_TOPK)
        for l in range(self.L):
            ckv.score_keys(s, self.q_sel[0][l], self.t[l]["k"], self.lens, SCALE, scores)
            ckv.select_topk(s, scores, self.lens, w.k, self.idx[0][l], self.nsel[0][l], ws)
        torch.cuda.synchronize()

    def run(self, steps, pipe, delay=None):
        """steps decode steps; returns host copies of (idx, nsel, out) per step."""
        if self.in_place:  # caches in device memory: rows read in place
            shape = ckv.shape_for(self.w.batch, self.w.q_heads, self.w.kv_heads,
                                  self.w.max_ctx)
        else:
            shape = self.shape
            self.copy.wait_stream(self.compute)
            pipe.prime(self.shape, self.w.k, self.layer_io(1, 0), ckv.SRC_HOST_PINNED,
                       self.k_buf, self.v_buf, self.copy)
        cur, hist = 0, []
        for st in range(1, steps + 1):
            if delay is not None:
                delay(self.copy if delay.stream == "copy" else self.compute)
            if self.in_place:
                io = self.layer_io(st, cur)
                for l in range(self.L):
                    io[l]["k_src"], io[l]["v_src"] = self.t[l]["k"], self.t[l]["v"]
                pipe.step(shape, io, self.lens, self.w.k, SCALE, ckv.SRC_DEVICE, None, None,
                          self.ws, self.compute, None)
            else:
                pipe.step(shape, self.layer_io(st, cur), self.lens, self.w.k, SCALE,
                          ckv.SRC_HOST_PINNED, self.k_buf, self.v_buf, self.ws, self.compute,
                          self.copy)
            self.compute.wait_stream(self.copy)
            torch.cuda.synchronize()
            nxt = 1 - cur
            hist.append(([i.cpu().numpy() for i in self.idx[nxt]],
                         [n.cpu().numpy() for n in self.nsel[nxt]],
                         [o.cpu().numpy() for o in self.out],
                         [i.cpu().numpy() for i in self.idx_true],
                         [n.cpu().numpy() for n in self.n_true],
                         [h.cpu().numpy() for h in self.hits],
                         [o.cpu().numpy() for o in self.out_spec]))
            cur = nxt
        return hist


@pytest.mark.parametrize("wl,layers", [("long128k_s", 3), ("dual64_s", 2)])
def test_pipeline_matches_oracle(wl, layers):
    _log("pipeline", wl, layers)
    dev = device()
    w = synth.WORKLOADS[wl]
    lp = Loop(w, layers, steps=2, seed=5, dev=dev)
    lp.bootstrap()
    boot = ([i.cpu().numpy() for i in lp.idx[0]], [n.cpu().numpy() for n in lp.nsel[0]])
    pipe = ckv.Pipeline()
    hist = lp.run(2, pipe)
    pipe.close()
    o = orc()
    lens = lp.lens.cpu().numpy()
    so = o.shape(w.batch, w.q_heads, w.kv_heads, w.head_dim, w.max_ctx)
    prev_sets = boot
    for st in range(1, 3):
        g_idx, g_nsel, g_out = hist[st - 1][:3]
        for l in range(layers):
            K, V = u16(lp.t[l]["k"]), u16(lp.t[l]["v"])
            # selection at this step from this step's speculative query
            S = o.score_keys(so, u16(lp.q_sel[st][l]), K, lens, SCALE, nthreads=8)
            r_idx, r_nsel = o.select_topk(so, S, lens, w.k, nthreads=8)
            swaps = check_index_sets(g_idx[l], g_nsel[l], r_idx, r_nsel, S, lens)
            # attention of this step's query over the set selected one step earlier
            ref = oracle_attn_over(so, u16(lp.q_att[st][l]), K, V, prev_sets[0][l],
                                   prev_sets[1][l], w.k)
            err = np.abs(g_out[l] - ref).max()
            _log(f"  step {st} layer {l}: swaps {swaps}, max abs err {err:.2e}")
            assert err <= ATOL_OUT
        prev_sets = (g_idx, g_nsel)


def test_pipeline_gather_width_bit_identical():
    """The refill grid changes how many workgroups move the rows, not which:
    the loop at 16 and 4096 workgroups and at the width it picks by shape
    gives the same index sets and outputs bit for bit."""
    _log("pipeline gather widths")
    dev = device()
    w = synth.WORKLOADS["long128k_s"]
    results = []
    for width in (0, 16, 4096):
        lp = Loop(w, 2, steps=2, seed=8, dev=dev)
        lp.bootstrap()
        pipe = ckv.Pipeline()
        pipe.set_gather_width(width)
        results.append(lp.run(2, pipe))
        pipe.close()
    with pytest.raises(ckv.CkvError):
        ckv.Pipeline().set_gather_width(4097)
    for other in results[1:]:
        for st in range(2):
            for a, b in zip(results[0][st][:3], other[st][:3]):
                for x, y in zip(a, b):
                    np.testing.assert_array_equal(x, y)


@pytest.mark.parametrize("wl,layers", [("llama8b_s", 2), ("dual64_s", 3)])
def test_pipeline_in_place_matches_oracle(wl, layers):
    """The loop without buffers (cache in device memory): every layer attends
    over the rows of last step's set read in place and selects the next set."""
    _log("pipeline in place", wl, layers)
    dev = device()
    w = synth.WORKLOADS[wl]
    lp = Loop(w, layers, steps=2, seed=6, dev=dev)
    lp.bootstrap()
    boot = ([i.cpu().numpy() for i in lp.idx[0]], [n.cpu().numpy() for n in lp.nsel[0]])
    shape = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx)
    ws = ckv.workspace(shape, w.k, ckv.ENTRY_CRITICAL_KV_ATTN)
    pipe = ckv.Pipeline()
    cur, hist = 0, []
    for st in range(1, 3):
        io = lp.layer_io(st, cur)
        for l in range(layers):
            io[l]["k_src"], io[l]["v_src"] = lp.t[l]["k"], lp.t[l]["v"]
        pipe.step(shape, io, lp.lens, w.k, SCALE, ckv.SRC_DEVICE, None, None, ws, lp.compute,
                  None)
        torch.cuda.synchronize()
        nxt = 1 - cur
        hist.append(([i.cpu().numpy() for i in lp.idx[nxt]],
                     [n.cpu().numpy() for n in lp.nsel[nxt]],
                     [o.cpu().numpy() for o in lp.out]))
        cur = nxt
    pipe.close()
    o = orc()
    lens = lp.lens.cpu().numpy()
    so = o.shape(w.batch, w.q_heads, w.kv_heads, w.head_dim, w.max_ctx)
    prev_sets = boot
    for st in range(1, 3):
        g_idx, g_nsel, g_out = hist[st - 1]
        for l in range(layers):
            K, V = u16(lp.t[l]["k"]), u16(lp.t[l]["v"])
            S = o.score_keys(so, u16(lp.q_sel[st][l]), K, lens, SCALE, nthreads=8)
            r_idx, r_nsel = o.select_topk(so, S, lens, w.k, nthreads=8)
            swaps = check_index_sets(g_idx[l], g_nsel[l], r_idx, r_nsel, S, lens)
            ref = oracle_attn_over(so, u16(lp.q_att[st][l]), K, V, prev_sets[0][l],
                                   prev_sets[1][l], w.k)
            err = np.abs(g_out[l] - ref).max()
            _log(f"  step {st} layer {l}: swaps {swaps}, max abs err {err:.2e}")
            assert err <= ATOL_OUT
        prev_sets = (g_idx, g_nsel)


class _Delay:
    """Keeps one stream busy (device copies) before each step."""

    def __init__(self, stream_name, dev):
        self.stream = stream_name
        self.a = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
        self.b = torch.empty_like(self.a)

    def __call__(self, stream):
        with torch.cuda.stream(stream):
            for _ in range(40):
                self.b.copy_(self.a)


@pytest.mark.parametrize("stream_name", ["copy", "compute"])
def test_pipeline_ordering_under_delay(stream_name):
    """A busy copy stream (gathers land late: read-after-write) or a busy
    compute stream (buffers released late: write-after-read) must not change
    a single output bit."""
    _log("pipeline delay", stream_name)
    dev = device()
    w = synth.WORKLOADS["long128k_s"]
    lp = Loop(w, 3, steps=2, seed=7, dev=dev)
    lp.bootstrap()
    pipe = ckv.Pipeline()
    ref = lp.run(2, pipe)
    lp.bootstrap()
    got = lp.run(2, pipe, delay=_Delay(stream_name, dev))
    pipe.close()
    for (ri, rn, ro, *_), (gi, gn, go, *_) in zip(ref, got):
        for l in range(3):
            np.testing.assert_array_equal(ri[l], gi[l])
            np.testing.assert_array_equal(rn[l], gn[l])
            np.testing.assert_array_equal(ro[l], go[l])


@pytest.mark.parametrize("wl,layers,lowrank", [("dual64_s", 3, ()), ("long128k_s", 2, ()),
                                               ("dual64_s", 3, (1,))])
def test_pipeline_corrected_matches_oracle(wl, layers, lowrank):
    """Corrected layers in the decode loop: whatever was prefetched from the
    previous step's speculative selection, each layer's output is the current
    query's attention over its own top-k (the same-step result), the misses
    against the prefetched set are counted in hits, and the speculative
    selection for the next step is made as before.  Layers in `lowrank`
    rebuild their misses' keys (Sec. 5.3, adaptive key reconstruction): they
    attend over the prefetched keys of the hits and the rebuilt keys of the
    misses."""
    _log("pipeline corrected", wl, layers, lowrank)
    dev = device()
    w = synth.WORKLOADS[wl]
    lp = Loop(w, layers, steps=2, seed=11, dev=dev)
    lp.corrected = True
    rank = 32
    for l in lowrank:
        lp.lowrank[l] = (rank,) + synth.low_rank_factors(w, rank, seed=11, layer=l, device=dev)
    lp.bootstrap()
    boot = [i.cpu().numpy() for i in lp.idx[0]], [n.cpu().numpy() for n in lp.nsel[0]]
    pipe = ckv.Pipeline()
    hist = lp.run(2, pipe)
    pipe.close()
    o = orc()
    lens = lp.lens.cpu().numpy()
    so = o.shape(w.batch, w.q_heads, w.kv_heads, w.head_dim, w.max_ctx)
    prev_pred = boot
    for st in range(1, 3):
        g_idx, g_nsel, g_out, g_true, g_ntrue, g_hits = hist[st - 1][:6]
        for l in range(layers):
            K, V = u16(lp.t[l]["k"]), u16(lp.t[l]["v"])
            q_att = u16(lp.q_att[st][l])
            S = o.score_keys(so, q_att, K, lens, SCALE, nthreads=8)
            r_true, r_nt = o.select_topk(so, S, lens, w.k, nthreads=8)
            check_index_sets(g_true[l], g_ntrue[l], r_true, r_nt, S, lens)
            S2 = o.score_keys(so, u16(lp.q_sel[st][l]), K, lens, SCALE, nthreads=8)
            r_next, r_nn = o.select_topk(so, S2, lens, w.k, nthreads=8)
            check_index_sets(g_idx[l], g_nsel[l], r_next, r_nn, S2, lens)
            total = found = 0
            for b in range(w.batch):
                for h in range(w.kv_heads):
                    t_ = g_true[l][b, h, :g_ntrue[l][b, h]]
                    p_ = prev_pred[0][l][b, h, :prev_pred[1][l][b, h]]
                    want = len(np.intersect1d(t_, p_))
                    assert g_hits[l][b, h] == want, (st, l, b, h)
                    total += len(t_)
                    found += want
            if l in lp.lowrank:
                kb, vb = oracle_lowrank_buffers(so, K, V, rank, u16(lp.lowrank[l][1]),
                                                u16(lp.lowrank[l][2]), g_true[l], g_ntrue[l],
                                                prev_pred[0][l], prev_pred[1][l], w.k)
                ref = o.sparse_decode_attn(so, q_att, kb, vb, g_ntrue[l], w.k, SCALE,
                                           nthreads=8)
            else:
                ref = oracle_attn_over(so, q_att, K, V, g_true[l], g_ntrue[l], w.k)
            err = np.abs(g_out[l] - ref).max()
            _log(f"  step {st} layer {l}: hit rate {found / max(total, 1):.3f}, "
                 f"max abs err {err:.2e}")
            assert err <= ATOL_OUT
        prev_pred = (g_idx, g_nsel)


def _concurrent_stream(compute, dev, tries=8):
    """A new stream whose work runs beside `compute`.  Streams share the
    device's few hardware queues round-robin, and two streams on one queue
    run in submission order, where a missing wait cannot show.  A stream
    qualifies if a tiny kernel on it completes while `compute` is still busy
    with a long run of copies."""
    import time
    a = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
    b = torch.empty_like(a)
    for _ in range(tries):
        st = torch.cuda.Stream(device=dev)
        torch.cuda.synchronize()
        with torch.cuda.stream(compute):
            for _ in range(60):
                b.copy_(a)
            busy = torch.cuda.Event()
            busy.record(compute)
        with torch.cuda.stream(st):
            torch.zeros(1, device=dev)
            mark = torch.cuda.Event()
            mark.record(st)
        t0 = time.time()
        while not mark.query() and time.time() - t0 < 10:
            time.sleep(1e-4)
        concurrent = mark.query() and not busy.query()
        torch.cuda.synchronize()
        if concurrent:
            return st
    return None


@pytest.mark.parametrize("flags,stream_name", [
    (ckv.Pipeline.CHECK_NO_FILL_WAIT | ckv.Pipeline.CHECK_POISON, "copy"),
    (ckv.Pipeline.CHECK_NO_RELEASE_WAIT, "compute"),
    (ckv.Pipeline.CHECK_NO_RELEASE_WAIT | ckv.Pipeline.CHECK_POISON, "compute"),
], ids=["no_fill_wait+poison/busy_copy", "no_release_wait/busy_compute",
        "no_release_wait+poison/busy_compute"])
def test_pipeline_hazard_tests_see_a_missing_wait(flags, stream_name):
    """Detection power of test_pipeline_ordering_under_delay: with the fill
    wait removed and the copy stream held back, a layer attends over a
    buffer still holding another layer's rows (or poison); with the release
    wait removed and the compute stream held back, a buffer is refilled
    before the attention that needs its old rows.  Either way the outputs
    must differ from the reference, while the loop with its waits, held back
    the same way, stays bit-identical to it."""
    _log("pipeline hazard control", flags, stream_name)
    dev = device()
    w = synth.WORKLOADS["long128k_s"]
    lp = Loop(w, 3, steps=2, seed=7, dev=dev)
    lp.copy = _concurrent_stream(lp.compute, dev)
    if lp.copy is None:
        pytest.skip("no stream runs beside the compute stream: the waits cannot matter")
    lp.bootstrap()
    pipe = ckv.Pipeline()
    ref = lp.run(2, pipe)
    lp.bootstrap()
    same = lp.run(2, pipe, delay=_Delay(stream_name, dev))
    lp.bootstrap()
    pipe.set_checks(flags)
    broken = lp.run(2, pipe, delay=_Delay(stream_name, dev))
    pipe.set_checks(0)
    pipe.close()
    for (ri, rn, ro, *_), (gi, gn, go, *_) in zip(ref, same):
        for l in range(3):
            np.testing.assert_array_equal(ro[l], go[l])
            np.testing.assert_array_equal(ri[l], gi[l])
    differing = [(st, l) for st, ((_, _, ro, *_), (_, _, bo, *_)) in enumerate(zip(ref, broken))
                 for l in range(3) if not np.array_equal(ro[l], bo[l], equal_nan=False)]
    _log(f"  outputs that differ without the wait: {differing}")
    assert differing, "removing a wait changed nothing: the delay test could not see it"



def _gpu_chunk_sets(rows, nrows, chunk, kc):
    """The chunk set behind expanded rows: ascending chunk numbers, -1 padded."""
    B, Hkv, _ = rows.shape
    cidx = np.full((B, Hkv, kc), -1, np.int32)
    nch = np.zeros((B, Hkv), np.int32)
    for b in range(B):
        for h in range(Hkv):
            c = np.unique(rows[b, h, :nrows[b, h]] // chunk)
            cidx[b, h, :len(c)] = c
            nch[b, h] = len(c)
    return cidx, nch


@pytest.mark.parametrize("wl,layers,chunk,in_place", [
    ("long128k_s", 3, 8, False), ("dual64_s", 2, 4, False), ("llama8b_s", 2, 8, True)])
def test_pipeline_chunked_matches_oracle(wl, layers, chunk, in_place):
    """Chunked layers in the decode loop (Sec. 2.2 chunk landmarks): each step
    selects the k/chunk chunks whose landmarks score best against the
    speculative query, expands them to rows and prefetches those rows for
    the next step (as contiguous blocks from pinned memory, or read in place
    from the device caches); the current query attends over the rows chosen
    one step earlier.  Chunk sets under the near-tie rule on the oracle's
    landmark scores, rows exactly the expansion of the GPU's chunks, outputs
    against the oracle's attention over the earlier rows."""
    _log("pipeline chunked", wl, layers, chunk, "in place" if in_place else "two buffers")
    dev = device()
    w = synth.WORKLOADS[wl]
    lp = Loop(w, layers, steps=2, seed=17, dev=dev)
    lp.in_place = in_place
    lp.set_chunked(chunk)
    lp.bootstrap()
    boot = ([i.cpu().numpy() for i in lp.idx[0]], [n.cpu().numpy() for n in lp.nsel[0]])
    pipe = ckv.Pipeline()
    hist = lp.run(2, pipe)
    pipe.close()
    o = orc()
    lens = lp.lens.cpu().numpy()
    so = o.shape(w.batch, w.q_heads, w.kv_heads, w.head_dim, w.max_ctx)
    cmax = (w.max_ctx + chunk - 1) // chunk
    sc = o.shape(w.batch, w.q_heads, w.kv_heads, w.head_dim, cmax)
    clens = np.array([(int(n) + chunk - 1) // chunk for n in lens], np.int32)
    kc = w.k // chunk
    prev = boot
    for st in range(1, 3):
        g_idx, g_nsel, g_out = hist[st - 1][:3]
        for l in range(layers):
            K, V = u16(lp.t[l]["k"]), u16(lp.t[l]["v"])
            lm = o.chunk_landmarks(so, chunk, K, lens)
            g_lm = u16(lp.lms[l])
            for b in range(w.batch):  # landmarks past a request's chunks are not written
                assert np.array_equal(lm[b, :, :clens[b]], g_lm[b, :, :clens[b]]), "landmarks"
            q_sel = u16(lp.q_sel[st][l])
            S = o.score_keys(sc, q_sel, lm, clens, SCALE, nthreads=8)
            r_c, r_nc, _, _ = o.select_chunks(so, chunk, q_sel, lm, lens, w.k, SCALE,
                                              nthreads=8)
            g_c, g_nc = _gpu_chunk_sets(g_idx[l], g_nsel[l], chunk, kc)
            swaps = check_index_sets(g_c, g_nc, r_c, r_nc, S, clens)
            for b in range(w.batch):
                for h in range(w.kv_heads):
                    want, nr = o.expand_chunks(chunk, g_c[b, h, :g_nc[b, h]], int(lens[b]), w.k)
                    assert g_nsel[l][b, h] == nr, (st, l, b, h)
                    assert np.array_equal(g_idx[l][b, h], want), (st, l, b, h)
            ref = oracle_attn_over(so, u16(lp.q_att[st][l]), K, V, prev[0][l], prev[1][l],
                                   w.k)
            err = np.abs(g_out[l] - ref).max()
            _log(f"  step {st} layer {l}: chunk swaps {swaps}, max abs err {err:.2e}")
            assert err <= ATOL_OUT
        prev = (g_idx, g_nsel)


@pytest.mark.parametrize("wl,layers,in_place", [
    ("dual64_s", 3, False), ("long128k_s", 2, False), ("llama8b_s", 2, True)])
def test_pipeline_two_tokens_matches_oracle(wl, layers, in_place):
    """Two-token layers in the decode loop (Sec. 5.2): one launch attends with
    the current token and the speculative token over the rows selected one
    step earlier, each also over the tokens' own rows under the causal mask,
    and scores with the speculative query for the next step's selection."""
    _log("pipeline two tokens", wl, layers, "in place" if in_place else "two buffers")
    dev = device()
    w = synth.WORKLOADS[wl]
    lp = Loop(w, layers, steps=2, seed=19, dev=dev)
    lp.in_place = in_place
    lp.set_two_tokens(2)
    lp.bootstrap()
    boot = ([i.cpu().numpy() for i in lp.idx[0]], [n.cpu().numpy() for n in lp.nsel[0]])
    pipe = ckv.Pipeline()
    hist = lp.run(2, pipe)
    pipe.close()
    o = orc()
    lens = lp.lens.cpu().numpy()
    so = o.shape(w.batch, w.q_heads, w.kv_heads, w.head_dim, w.max_ctx)
    B, Hkv, k, d = w.batch, w.kv_heads, w.k, w.head_dim
    prev = boot
    for st in range(1, 3):
        g_idx, g_nsel, g_out = hist[st - 1][:3]
        g_spec = hist[st - 1][6]
        for l in range(layers):
            K, V = u16(lp.t[l]["k"]), u16(lp.t[l]["v"])
            q_att, q_sel = u16(lp.q_att[st][l]), u16(lp.q_sel[st][l])
            S = o.score_keys(so, q_sel, K, lens, SCALE, nthreads=8)
            r_idx, r_nsel = o.select_topk(so, S, lens, k, nthreads=8)
            swaps = check_index_sets(g_idx[l], g_nsel[l], r_idx, r_nsel, S, lens)
            kb = np.zeros((B, Hkv, k, d), np.uint16)
            vb = np.zeros_like(kb)
            o.gather_kv(so, K.reshape(-1), V.reshape(-1), prev[0][l], prev[1][l], k, kb, vb)
            kl, vl = lp.local[st][l]
            r_cur, r_spec = o.dual_token_attn(so, q_att, q_sel, kb, vb, prev[1][l], u16(kl),
                                              u16(vl), k, SCALE, nthreads=8)
            e1 = np.abs(g_out[l] - r_cur).max()
            e2 = np.abs(g_spec[l] - r_spec).max()
            _log(f"  step {st} layer {l}: swaps {swaps}, max abs err {e1:.2e} / {e2:.2e}")
            assert e1 <= ATOL_OUT and e2 <= ATOL_OUT
        prev = (g_idx, g_nsel)
