"""Same-step decode through the one-launch selection and attention (MI355X
only): every workgroup selects its unit's set, then either attends over its
share of the rows with all the group's heads, or, for an even group size with
k <= 2048 when head halves are asked for, over the whole set with half the
heads, writing its outputs directly.  Two shares (two workgroups per unit,
the default wherever head halves would apply) merge inside the launch; more
shares are merged by the merge kernel.
Checked against the oracle: index sets under the near-tie rule, outputs
within 2e-3 of the oracle's attention over the GPU's own set (and of the
oracle's whole step when the sets agree), for head halves, 1, 2 and 4 row
shares, group sizes 1, 2, 4 and 8, ragged contexts, a context shorter than k
and an empty one.  The kernel profile confirms which launches ran.
"""
from __future__ import annotations

import dataclasses

import numpy as np
import pytest
import torch

import paper_2607_26475_amd as ckv
import synth
from helpers import (ATOL_OUT, SCALE, Run, check_index_sets, device, oracle_attn_over, orc,
                     u16)

pytestmark = pytest.mark.gpu


def _log(*a):
    print(*a, flush=True)


BASE = synth.WORKLOADS["llama8b_s"]
# (name, workload changes, context lengths or None for the drawn ones, row
# shares: 0 for the split by heads, whether head halves are asked for)
CASES = [
    ("k1024_rows", dict(k=1024), None, 2, False),
    ("k1024_heads", dict(k=1024), None, 0, True),
    ("k2048_rows", dict(k=2048, max_ctx=8000, ctx_min=5000), None, 2, False),
    ("k2048_heads", dict(k=2048, max_ctx=8000, ctx_min=5000), None, 0, True),
    ("k4096_2shares", dict(k=4096, max_ctx=20000, ctx_min=15000), None, 2, False),
    ("k8192_4shares", dict(k=8192, max_ctx=40000, ctx_min=30000, batch=1), None, 4, False),
    ("short_and_empty", dict(k=1024, batch=3), [5000, 700, 0], 2, False),
    ("short_and_empty_heads", dict(k=1024, batch=3), [5000, 700, 0], 0, True),
    ("tiny_share", dict(k=1024, batch=3), [5000, 10, 0], 2, False),
    ("g8", dict(k=1024, q_heads=64), None, 2, False),
    ("g8_heads", dict(k=1024, q_heads=64), None, 0, True),
    ("g2", dict(k=1024, q_heads=16), None, 2, False),
    ("g1", dict(k=1024, q_heads=8), None, 2, False),
    ("one_share", dict(k=256), None, 1, False),
]


@pytest.mark.parametrize("name,changes,lens,shares,heads", CASES, ids=[c[0] for c in CASES])
def test_select_attn_matches_oracle(name, changes, lens, shares, heads):
    _log("select+attention", name)
    dev = device()
    w = dataclasses.replace(BASE, name=f"selattn_{name}", **changes)
    t = synth.make_layer(w, seed=31, device=dev)
    if lens is not None:
        t["ctx_lens"] = torch.tensor(lens, dtype=torch.int32, device=dev)
    run = Run(w, t["ctx_lens"], dev)
    ckv.set_one_launch_same_step(ckv.ONE_LAUNCH_HEAD_HALVES if heads else ckv.ONE_LAUNCH_ROW_HALVES)
    try:
        ckv.profile_begin()
        run.same_step(t["q"], t["q_sel"], t["k"], t["k"], t["v"], ckv.SRC_DEVICE)
        kernels = ckv.profile_end()
    finally:
        ckv.set_one_launch_same_step(ckv.ONE_LAUNCH_ROW_HALVES)
    assert "select_attn" in kernels and "attn" not in kernels, kernels
    assert ("combine" in kernels) == (shares > 2), kernels
    g_idx, g_nsel, g_out = run.host()
    lens_np = t["ctx_lens"].cpu().numpy()
    q_att, q_sel, K, V = u16(t["q"]), u16(t["q_sel"]), u16(t["k"]), u16(t["v"])
    o = orc()
    so = o.shape(w.batch, w.q_heads, w.kv_heads, w.head_dim, w.max_ctx)
    S = o.score_keys(so, q_sel, K, lens_np, SCALE, nthreads=8)
    r_idx, r_nsel = o.select_topk(so, S, lens_np, w.k, nthreads=8)
    swaps = check_index_sets(g_idx, g_nsel, r_idx, r_nsel, S, lens_np)
    ref = oracle_attn_over(so, q_att, K, V, g_idx, g_nsel, w.k)
    err = float(np.abs(g_out - ref).max())
    _log(f"  units with swaps {swaps}, max abs err {err:.2e}")
    assert err <= ATOL_OUT
    if swaps == 0:
        _, _, r_out = o.critical_kv_attn(so, q_att, q_sel, K, K, V, lens_np, w.k, SCALE,
                                         nthreads=8)
        assert np.abs(g_out - r_out).max() <= ATOL_OUT
    for b in range(w.batch):
        if lens_np[b] == 0:
            assert np.all(g_out[b] == 0.0), b
