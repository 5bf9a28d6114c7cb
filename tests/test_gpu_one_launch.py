"""The same-step layer in one launch (k_critical) on an MI355X.

Where it applies (even group size up to 8, a multiple of 8 units with the
per-workgroup histogram slots, two workgroups per unit on the device, 512 <=
k <= 2048), a same-step call scores, selects and attends in one launch, each
unit's selection starting once its scores are handed over.  The selection
is exact, so every index set and count must equal, bit for bit, those of the
same call in two launches (scoring launch, then the selection and attention
launch); the kernel profile shows which form ran.  By default both forms
attend with row halves (each of a unit's two workgroups over half the rows
with all heads, the second merging the first's partial inside the launch)
in the same code, so the outputs must be equal too.  With head halves asked
for, the one launch attends over the whole set with half the heads per
workgroup: the same terms added in another order, so its outputs must agree
with the row halves' within fp32 rounding (FORM_TOL) and repeat bit for bit.  The one-launch
results are also checked against the oracle (Sec. 2.2 selection, Sec.
5.3-5.4 attention).  The hand-over flags live in the workspace: a workspace
filled with garbage, calls of other shapes in between, and graph replays
(one tag for every replay) must all leave the results unchanged.
"""
from __future__ import annotations

import dataclasses

import numpy as np
import pytest
import torch

import paper_2607_26475_amd as ckv
import synth
from helpers import ATOL_OUT, SCALE, check_index_sets, device, oracle_attn_over, orc, u16

pytestmark = pytest.mark.gpu

# Outputs of the row-halves and head-halves forms: fp32 weighted means of
# bf16 values of magnitude below about 4, summed in different orders (per
# wave, then per half or per head group), differ by a few units in the last
# place; 4e-6 is about 30 ulp at 1.0, far below the 2e-3 parity tolerance.
FORM_TOL = 4e-6
ROWS, HEADS, OFF = ckv.ONE_LAUNCH_ROW_HALVES, ckv.ONE_LAUNCH_HEAD_HALVES, ckv.ONE_LAUNCH_OFF

BASE = synth.WORKLOADS["llama8b_s"]
CASES = {
    # units, group size, stored context (ragged, not a multiple of 32 or odd), k
    "u40_g4": dataclasses.replace(BASE, name="u40_g4", batch=5, q_heads=32, kv_heads=8,
                                  max_ctx=5000, ctx_min=5000, k=1024),
    "u48_g2": dataclasses.replace(BASE, name="u48_g2", batch=6, q_heads=16, kv_heads=8,
                                  max_ctx=4099, ctx_min=4099, k=512),
    "u64_g8": dataclasses.replace(BASE, name="u64_g8", batch=8, q_heads=64, kv_heads=8,
                                  max_ctx=3001, ctx_min=3001, k=2048),
    "u80_dual": dataclasses.replace(BASE, name="u80_dual", batch=10, q_heads=32, kv_heads=8,
                                    max_ctx=6000, ctx_min=6000, k=2000, dual=True),
    "u48_h4": dataclasses.replace(BASE, name="u48_h4", batch=12, q_heads=16, kv_heads=4,
                                  max_ctx=7000, ctx_min=7000, k=700),
}


def _lens(w, seed):
    rng = np.random.default_rng(seed)
    lens = rng.integers(0, w.max_ctx + 1, size=w.batch)
    lens[0] = w.max_ctx
    lens[1] = 0
    lens[2] = min(w.k - 1, w.max_ctx)  # every position selected
    lens[3] = 10  # row halves: the first takes all 10 rows, the second none
    return torch.tensor(lens, dtype=torch.int32)


def _call(w, t, lens, ws, interleaved, mode, stream=None):
    dev = t["q"].device
    d = w.head_dim
    if interleaved:
        kv = t["kv"]
        keys, k_src, v_src = kv, kv.data_ptr(), kv.data_ptr() + 2 * d
        s = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx, key_row_stride=2 * d,
                          kv_row_stride=2 * d)
    else:
        keys, k_src, v_src = t["k"], t["k"], t["v"]
        s = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx)
    idx = torch.full((w.batch, w.kv_heads, w.k), -9, dtype=torch.int32, device=dev)
    nsel = torch.full((w.batch, w.kv_heads), -9, dtype=torch.int32, device=dev)
    out = torch.full((w.batch, w.q_heads, d), float("nan"), device=dev)
    ckv.set_one_launch_same_step(mode)
    try:
        ckv.profile_begin()
        ckv.critical_kv_attn(s, t["q"], t["q_sel"], keys, lens, w.k, SCALE, k_src, v_src,
                             ckv.SRC_DEVICE, None, None, None, idx, nsel, out, ws, stream)
        kernels = ckv.profile_end()
    finally:
        ckv.set_one_launch_same_step(ROWS)
    torch.cuda.synchronize()
    return idx, nsel, out, kernels


def _setup(name, interleaved, seed=3):
    dev = device()
    w = CASES[name]
    t = synth.make_layer(w, seed=seed, device=dev)
    if interleaved:
        t["kv"] = synth.interleave_kv(t["k"], t["v"])
    lens = _lens(w, seed).to(dev)
    s = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx)
    ws = ckv.workspace(s, w.k, ckv.ENTRY_CRITICAL_KV_ATTN)
    ws.fill_(0xA5)  # garbage where the hand-over flags live
    return dev, w, t, lens, ws


def _same_sets_close_outputs(a, b):
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
    diff = (a[2] - b[2]).abs().max().item() if a[2].numel() else 0.0
    assert diff <= FORM_TOL, diff
    return diff


@pytest.mark.parametrize("name,interleaved", [("u40_g4", False), ("u48_g2", False),
                                              ("u64_g8", False), ("u80_dual", False),
                                              ("u48_h4", False), ("u40_g4", True)])
def test_one_launch_matches_two_launches_and_oracle(name, interleaved):
    print("one launch", name, "interleaved" if interleaved else "separate", flush=True)
    dev, w, t, lens, ws = _setup(name, interleaved)
    one = _call(w, t, lens, ws, interleaved, ROWS)
    heads = _call(w, t, lens, ws, interleaved, HEADS)
    two = _call(w, t, lens, ws, interleaved, OFF)
    print("  kernels", {k: v[0] for k, v in one[3].items()}, "/",
          {k: v[0] for k, v in two[3].items()}, flush=True)
    assert set(one[3]) == {"critical"}, one[3]
    assert set(heads[3]) == {"critical"}, heads[3]
    assert "critical" not in two[3] and "select_attn" in two[3] and "combine" not in two[3], two[3]
    for a, b in zip(one[:3], two[:3]):
        assert torch.equal(a, b)
    diff = _same_sets_close_outputs(heads, two)
    again = _call(w, t, lens, ws, interleaved, ROWS)  # the flags were left clear
    for a, b in zip(one[:3], again[:3]):
        assert torch.equal(a, b)
    print(f"  head halves against row halves: sets equal, outputs within {diff:.2e}", flush=True)
    o = orc()
    so = o.shape(w.batch, w.q_heads, w.kv_heads, w.head_dim, w.max_ctx)
    lens_h = lens.cpu().numpy()
    K, V = u16(t["k"]), u16(t["v"])
    S = o.score_keys(so, u16(t["q_sel"]), K, lens_h, SCALE, nthreads=8)
    r_idx, r_nsel = o.select_topk(so, S, lens_h, w.k, nthreads=8)
    g_idx, g_nsel, g_out = (x.cpu().numpy() for x in one[:3])
    swaps = check_index_sets(g_idx, g_nsel, r_idx, r_nsel, S, lens_h)
    err = np.abs(g_out - oracle_attn_over(so, u16(t["q"]), K, V, g_idx, g_nsel, w.k)).max()
    print(f"  tolerated swaps {swaps}, max abs err {err:.2e}", flush=True)
    assert err <= ATOL_OUT


def test_one_launch_between_other_shapes():
    """One workspace for calls of two shapes in turn (the second reaches
    further into it); each call's results stay those of its first call."""
    dev, w1, t1, lens1, ws = _setup("u40_g4", False, seed=5)
    w2 = CASES["u80_dual"]
    t2 = synth.make_layer(w2, seed=6, device=dev)
    lens2 = _lens(w2, 6).to(dev)
    s2 = ckv.shape_for(w2.batch, w2.q_heads, w2.kv_heads, w2.max_ctx)
    ws2 = ckv.workspace(s2, w2.k, ckv.ENTRY_CRITICAL_KV_ATTN)
    big = ws if ws.numel() >= ws2.numel() else ws2
    first1 = _call(w1, t1, lens1, big, False, ROWS)
    first2 = _call(w2, t2, lens2, big, False, ROWS)
    for _ in range(2):
        r1 = _call(w1, t1, lens1, big, False, ROWS)
        r2 = _call(w2, t2, lens2, big, False, ROWS)
        for a, b in zip(first1[:3] + first2[:3], r1[:3] + r2[:3]):
            assert torch.equal(a, b)


def test_one_launch_graph_replays():
    """Captured once, replayed three times with eager calls of the same entry
    between the replays: every replay equals the eager call bit for bit (the
    tag is the same in every replay, so each launch must leave its flags
    clear)."""
    dev, w, t, lens, ws = _setup("u48_g2", False, seed=9)
    ref = _call(w, t, lens, ws, False, ROWS)
    s = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx)
    idx = torch.full_like(ref[0], -9)
    nsel = torch.full_like(ref[1], -9)
    out = torch.full_like(ref[2], float("nan"))
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        ckv.critical_kv_attn(s, t["q"], t["q_sel"], t["k"], lens, w.k, SCALE, t["k"], t["v"],
                             ckv.SRC_DEVICE, None, None, None, idx, nsel, out, ws)
    for rep in range(3):
        idx.fill_(-9)
        nsel.fill_(-9)
        out.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip((idx, nsel, out), ref[:3]):
            assert torch.equal(a, b), rep
        eager = _call(w, t, lens, ws, False, ROWS)
        for a, b in zip(eager[:3], ref[:3]):
            assert torch.equal(a, b), rep


def test_one_launch_full_size_repeated():
    """Four Llama-8B layers (B16, 32 q / 8 KV heads, n 32768, k 2048) called
    in turn 25 times through one workspace in each one-launch form: the row
    halves bit-identical to the two-launch form of the same layer, the head
    halves with its index sets and within FORM_TOL of its outputs, and every
    repeat bit-identical to the form's first call."""
    dev = device()
    w = dataclasses.replace(synth.WORKLOADS["llama8b"], layers=4)
    s = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx)
    ws = ckv.workspace(s, w.k, ckv.ENTRY_CRITICAL_KV_ATTN)
    layers = [synth.make_layer(w, seed=0, layer=l, device=dev) for l in range(w.layers)]
    ref = [_call(w, t, t["ctx_lens"], ws, False, OFF)[:3] for t in layers]
    first = [_call(w, t, t["ctx_lens"], ws, False, HEADS)[:3] for t in layers]
    for l in range(w.layers):
        _same_sets_close_outputs(first[l], ref[l])
    for it in range(25):
        for l, t in enumerate(layers):
            for mode, want in ((ROWS, ref[l]), (HEADS, first[l])):
                got = _call(w, t, t["ctx_lens"], ws, False, mode)
                assert set(got[3]) == {"critical"}, got[3]
                for a, b in zip(got[:3], want):
                    assert torch.equal(a, b), (it, l, mode)
    print("  200 one-launch calls bit-identical to their references", flush=True)
