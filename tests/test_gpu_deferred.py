"""Deferred selections in the decode loop without buffers (MI355X only).

With the decode step's workspace, a plain layer followed by a plain layer,
or a two-token layer followed by a two-token layer, leaves its selection
(its sets for the next step) to the next layer's attend-and-score launch,
which runs it as a third role with 256-thread workgroups; the layer's
attention partials are merged by the merge launch.
The selection is exact and the merge takes the same order of operations
either way, so every index set, count and output must equal, bit for bit,
those of the same loop with every selection in its own layer's call
(CHECK_NO_DEFER).  Cases: all layers plain (the selection of layers 0 .. L-2
deferred, the last one's run at the end of the call), a chunked layer in the
middle (the pending selection runs before it), all layers two-token, plain
and two-token layers mixed (a pending selection runs when the kind changes),
a single layer, ragged contexts, three seeded random sequences of the three
kinds; two steps each, and the first step's plain layers also against the
oracle.
Deferral needs the per-workgroup histogram slots (at most 8 per unit, so at
least about 74 units beside 512 scoring workgroups): the batches here have
80 and 96 units.
"""
from __future__ import annotations

import dataclasses

import numpy as np
import pytest
import torch

import paper_2607_26475_amd as ckv
import synth
from helpers import ATOL_OUT, SCALE, check_index_sets, device, oracle_attn_over, orc, u16
from test_gpu_pipeline import Loop

pytestmark = pytest.mark.gpu


def _log(*a):
    print(*a, flush=True)


def _run(w, layers, chunk_layers, two_layers, no_defer, dev, steps=2):
    lp = Loop(w, layers, steps=steps, seed=17, dev=dev)
    lp.in_place = True
    if chunk_layers:
        lp.chunk_layers = set(chunk_layers)
        lp.set_chunked(8)
    if two_layers:
        lp.two_layers = None if two_layers == "all" else set(two_layers)
        lp.set_two_tokens(steps)
    lp.bootstrap()
    boot = ([i.cpu().numpy() for i in lp.idx[0]], [n.cpu().numpy() for n in lp.nsel[0]])
    pipe = ckv.Pipeline()
    if no_defer:
        pipe.set_checks(ckv.Pipeline.CHECK_NO_DEFER)
    ckv.profile_begin()
    hist = lp.run(steps, pipe)
    kernels = ckv.profile_end()
    pipe.close()
    return lp, boot, hist, kernels


WL = {"llama80": dataclasses.replace(synth.WORKLOADS["llama8b_s"], name="llama80", batch=10),
      "dual96": dataclasses.replace(synth.WORKLOADS["dual64_s"], name="dual96", batch=12),
      # group sizes 8 and 2 (the 2G = 16 head rows of two tokens at G = 8)
      "g8": dataclasses.replace(synth.WORKLOADS["llama8b_s"], name="g8", batch=10, q_heads=64),
      "g2": dataclasses.replace(synth.WORKLOADS["llama8b_s"], name="g2", batch=10, q_heads=16)}


def _random_kinds(count=3, layers=6, seed=0):
    """Seeded sequences of plain, two-token and chunked layers."""
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(count):
        kinds = rng.integers(0, 3, size=layers)
        chunk = tuple(int(l) for l in np.nonzero(kinds == 2)[0]) or None
        two = tuple(int(l) for l in np.nonzero(kinds == 1)[0]) or None
        out.append(("llama80", layers, chunk, two))
    return out


@pytest.mark.parametrize("wl,layers,chunk_layers,two_layers", [
    ("llama80", 4, None, None), ("llama80", 4, (2,), None), ("llama80", 1, None, None),
    ("dual96", 3, None, None), ("llama80", 4, None, "all"), ("llama80", 5, None, (1, 2, 4)),
    ("g8", 3, None, None), ("g8", 3, None, "all"), ("g2", 3, None, (1, 2))] + _random_kinds())
def test_deferred_selection_matches_undeferred(wl, layers, chunk_layers, two_layers):
    _log("deferred", wl, layers, chunk_layers, two_layers)
    dev = device()
    w = WL[wl]
    lp, boot, hist, kernels = _run(w, layers, chunk_layers, two_layers, False, dev)
    _, _, ref, ref_kernels = _run(w, layers, chunk_layers, two_layers, True, dev)
    _log("  kernels", {k: v[0] for k, v in kernels.items()},
         "undeferred", {k: v[0] for k, v in ref_kernels.items()})
    def kind(l):
        if chunk_layers and l in chunk_layers:
            return 2
        return 1 if two_layers and (two_layers == "all" or l in two_layers) else 0

    plain = [l for l in range(layers) if kind(l) == 0]
    # layers followed by a layer of their kind (plain or two-token) defer their
    # selection; plain ones merge their partials in a merge launch instead
    deferred = [l for l in range(layers)
                if kind(l) != 2 and l + 1 < layers and kind(l + 1) == kind(l)]
    merges = [l for l in deferred if kind(l) == 0] + [l for l in range(layers) if kind(l) == 1]
    assert "zero" not in kernels, kernels  # per-workgroup histogram slots
    assert kernels.get("combine", (0,))[0] == 2 * len(merges), kernels
    assert kernels["finish"][0] == ref_kernels["finish"][0] - 2 * len(deferred), kernels
    for st in range(2):
        for part in (0, 1, 2, 6):  # idx, n_sel, outputs, speculative outputs of every layer
            for l in range(layers):
                np.testing.assert_array_equal(hist[st][part][l], ref[st][part][l],
                                              err_msg=f"step {st + 1} layer {l} part {part}")
    # the first step's plain layers against the oracle
    o = orc()
    lens = lp.lens.cpu().numpy()
    so = o.shape(w.batch, w.q_heads, w.kv_heads, w.head_dim, w.max_ctx)
    g_idx, g_nsel, g_out = hist[0][:3]
    for l in plain:
        K, V = u16(lp.t[l]["k"]), u16(lp.t[l]["v"])
        S = o.score_keys(so, u16(lp.q_sel[1][l]), K, lens, SCALE, nthreads=8)
        r_idx, r_nsel = o.select_topk(so, S, lens, w.k, nthreads=8)
        swaps = check_index_sets(g_idx[l], g_nsel[l], r_idx, r_nsel, S, lens)
        att = oracle_attn_over(so, u16(lp.q_att[1][l]), K, V, boot[0][l], boot[1][l], w.k)
        err = np.abs(g_out[l] - att).max()
        _log(f"  layer {l}: swaps {swaps}, max abs err {err:.2e}")
        assert err <= ATOL_OUT


def test_full_llama8b_decode_step_deferred():
    """Three full-size Llama-8B-shaped layers (B16, 32 / 8 heads, n 32768, k
    2048) through one decode step without buffers, with the deferred
    selections (five histogram slots per unit) and without: every set, count
    and output bit for bit, and two sampled units of the middle layer's new
    set against the oracle's selection."""
    _log("full llama8b decode step, deferred")
    dev = device()
    w = synth.WORKLOADS["llama8b"]
    L, G, k = 3, w.group, w.k
    ts = [synth.make_layer(w, seed=0, layer=l, device=dev) for l in range(L)]
    lens = ts[0]["ctx_lens"]
    shape = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx)
    i32 = dict(dtype=torch.int32, device=dev)
    B, Hq, Hkv, d = w.batch, w.q_heads, w.kv_heads, w.head_dim
    spec = []
    for l, t in enumerate(ts):
        g = synth.generator(w.name, 0, l, "spec", dev)
        spec.append((0.8 * t["q"].float() + 0.6 * torch.randn(t["q"].shape, generator=g,
                                                               device=dev)).to(torch.bfloat16))
    ws = ckv.workspace(shape, k, ckv.ENTRY_DECODE_STEP)
    idx0 = [torch.empty((B, Hkv, k), **i32) for _ in range(L)]
    n0 = [torch.empty((B, Hkv), **i32) for _ in range(L)]
    boot_out = torch.empty((B, Hq, d), device=dev)
    for l, t in enumerate(ts):  # the pre-decoding selection
        ckv.critical_kv_attn(shape, t["q"], spec[l], t["k"], lens, k, SCALE, t["k"], t["v"],
                             ckv.SRC_DEVICE, None, None, None, idx0[l], n0[l], boot_out, ws)
    res = []
    for no_defer in (False, True):
        idx1 = [torch.full((B, Hkv, k), -9, **i32) for _ in range(L)]
        n1 = [torch.full((B, Hkv), -9, **i32) for _ in range(L)]
        out = [torch.full((B, Hq, d), float("nan"), device=dev) for _ in range(L)]
        io = [{"q_att": t["q"], "q_sel": spec[l], "k_score": t["k"], "k_src": t["k"],
               "v_src": t["v"], "idx_prev": idx0[l], "n_sel_prev": n0[l], "idx_next": idx1[l],
               "n_sel_next": n1[l], "out": out[l]} for l, t in enumerate(ts)]
        pipe = ckv.Pipeline()
        if no_defer:
            pipe.set_checks(ckv.Pipeline.CHECK_NO_DEFER)
        ckv.profile_begin()
        pipe.step(shape, io, lens, k, SCALE, ckv.SRC_DEVICE, None, None, ws, None, None)
        kernels = ckv.profile_end()
        torch.cuda.synchronize()
        pipe.close()
        _log("  no_defer", no_defer, {n: v[0] for n, v in kernels.items()})
        res.append(([i.cpu().numpy() for i in idx1], [n.cpu().numpy() for n in n1],
                    [o.cpu().numpy() for o in out], kernels))
    assert res[0][3]["finish"][0] == 1 and res[1][3]["finish"][0] == L, (res[0][3], res[1][3])
    for part in range(3):
        for l in range(L):
            np.testing.assert_array_equal(res[0][part][l], res[1][part][l],
                                          err_msg=f"layer {l} part {part}")
    o = orc()
    lens_h = lens.cpu().numpy()
    q_sel = u16(spec[1])
    for b, h in ((3, 5), (11, 2)):
        n = int(lens_h[b])
        S = o.unit_scores(q_sel[b, h * G:(h + 1) * G], u16(ts[1]["k"][b, h, :n]), SCALE)
        r_idx, m = o.unit_select(S, k)
        Sfull = np.full((1, 1, n), np.nan)
        Sfull[0, 0] = S
        check_index_sets(res[0][0][1][b:b + 1, h:h + 1], res[0][1][1][b:b + 1, h:h + 1],
                         r_idx[None, None], np.array([[m]]), Sfull, np.array([n]))
