"""ckv_critical_kv_attn_noalloc (the fused step on the library's fixed
per-device scratch) against ckv_critical_kv_attn with a caller workspace, on
the same inputs (MI355X only).

Calls in a row go through the fixed scratch: a batch whose same-step layer
runs as one launch (its hand-over flags in the scratch) twice, then two
smaller shapes, each finding the previous call's contents in the scratch;
a last call runs the pipelined form (rows read in place) on another shape.
Both entries run the same kernels, so index sets, counts and outputs must be
bit-identical.  A shape whose workspace exceeds the scratch is refused.
"""
from __future__ import annotations

import dataclasses

import numpy as np
import pytest
import torch

import paper_2607_26475_amd as ckv
import synth
from helpers import SCALE, device

pytestmark = pytest.mark.gpu


def _log(*a):
    print(*a, flush=True)


def _outputs(w, dev):
    B, Hq, Hkv, d, k = w.batch, w.q_heads, w.kv_heads, w.head_dim, w.k
    return (torch.full((B, Hkv, k), -9, dtype=torch.int32, device=dev),
            torch.full((B, Hkv), -9, dtype=torch.int32, device=dev),
            torch.full((B, Hq, d), float("nan"), dtype=torch.float32, device=dev))


def _same(a, b, what):
    for x, y, name in zip(a, b, ("idx", "n_sel", "out")):
        assert torch.equal(x, y), (what, name)


# 40 units: the same-step call runs as one launch, its hand-over flags in the scratch
ONE_LAUNCH = dataclasses.replace(synth.WORKLOADS["llama8b_s"], name="u40", batch=5, max_ctx=5000,
                                 ctx_min=3000, k=1024)


def _same_step_pair(wl, seed, dev):
    w = wl if isinstance(wl, synth.Workload) else synth.WORKLOADS[wl]
    t = synth.make_layer(w, seed=seed, device=dev)
    s = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx)
    assert ckv.workspace_bytes(s, w.k, ckv.ENTRY_CRITICAL_KV_ATTN) <= ckv.NOALLOC_SCRATCH_BYTES
    ws = ckv.workspace(s, w.k, ckv.ENTRY_CRITICAL_KV_ATTN)
    ref, got = _outputs(w, dev), _outputs(w, dev)
    ckv.critical_kv_attn(s, t["q"], t["q_sel"], t["k"], t["ctx_lens"], w.k, SCALE, t["k"],
                         t["v"], ckv.SRC_DEVICE, None, None, None, *ref, ws)
    ckv.profile_begin()
    ckv.critical_kv_attn_noalloc(s, t["q"], t["q_sel"], t["k"], t["ctx_lens"], w.k, SCALE,
                                 t["k"], t["v"], ckv.SRC_DEVICE, None, None, None, *got)
    kernels = ckv.profile_end()
    torch.cuda.synchronize()
    assert torch.isfinite(got[2]).all()
    _same(ref, got, w.name)
    assert ("critical" in kernels) == (w is ONE_LAUNCH), kernels
    return w, t, got


def test_noalloc_matches_workspace_entry():
    dev = device()
    # 1. the layer in one launch (hand-over flags in the scratch), twice, then
    # 2. a smaller shape and 3. a smaller one again on the same (now stale) scratch
    _log("no-alloc: same-step u40 (one launch) twice, llama8b_s, then tiny")
    _same_step_pair(ONE_LAUNCH, 20, dev)
    _same_step_pair(ONE_LAUNCH, 19, dev)
    _same_step_pair("llama8b_s", 21, dev)
    _same_step_pair("tiny", 22, dev)
    # 3. the pipelined form over rows read in place, selected one step earlier
    _log("no-alloc: pipelined in place, dual64_s")
    w, t, prev = _same_step_pair("dual64_s", 23, dev)
    s = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx)
    ws = ckv.workspace(s, w.k, ckv.ENTRY_CRITICAL_KV_ATTN)
    g = synth.generator(w.name, 23, 0, "next", dev)
    q_next = torch.randn(t["q"].shape, generator=g, device=dev).to(torch.bfloat16)
    ref, got = _outputs(w, dev), _outputs(w, dev)
    ckv.critical_kv_attn(s, q_next, t["q_sel"], t["k"], t["ctx_lens"], w.k, SCALE, t["k"],
                         t["v"], ckv.SRC_DEVICE, None, None, prev[1], *ref, ws, idx_in=prev[0])
    ckv.critical_kv_attn_noalloc(s, q_next, t["q_sel"], t["k"], t["ctx_lens"], w.k, SCALE,
                                 t["k"], t["v"], ckv.SRC_DEVICE, None, None, prev[1], *got,
                                 idx_in=prev[0])
    torch.cuda.synchronize()
    _same(ref, got, "dual64_s pipelined")
    _log("  all three calls bit-identical to the workspace entry")


def test_noalloc_refuses_a_shape_beyond_the_scratch():
    dev = device()
    w = synth.WORKLOADS["long128k"]
    s = ckv.shape_for(w.batch, w.q_heads, w.kv_heads, w.max_ctx)
    assert ckv.workspace_bytes(s, w.k, ckv.ENTRY_CRITICAL_KV_ATTN) > ckv.NOALLOC_SCRATCH_BYTES
    x = torch.empty(16, dtype=torch.int32, device=dev)
    with pytest.raises(ckv.CkvError) as e:
        ckv.critical_kv_attn_noalloc(s, x, None, x, x, w.k, SCALE, x, x, ckv.SRC_DEVICE, None,
                                     None, None, x, x, x)
    assert e.value.status == 4 and "fixed scratch" in str(e.value)
