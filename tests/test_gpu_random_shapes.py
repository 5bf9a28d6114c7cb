"""Seeded random shapes through the fused entry against the oracle (MI355X only).

Batch, KV heads, group size, stored context, budget and every request's
context length are drawn from a fixed seed.  So the fused entry's paths and
their launch shapes meet cases that no fixed case names: ragged last groups and
tiles, contexts shorter than the budget or empty, budgets of a single row,
contexts past the one-workgroup selection's limit.  The paths are the
one-launch selection and attention in both of its forms, the three-kernel
path, and the many-workgroup selection.  Each case checks the same-step call
(Sec. 2.2 selection, Sec. 5.3-5.4 attention).  Its index sets are compared
with the oracle's under the near-tie rule, and its output with the oracle's
attention over the GPU's set.  Then the case checks the pipelined call that
attends over that set in place and selects with a second query.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import paper_2607_26475_amd as ckv
import synth
from helpers import ATOL_OUT, SCALE, Run, check_index_sets, device, oracle_attn_over, orc, u16

pytestmark = pytest.mark.gpu


def _cases(count=40, seed=20261202):
    rng = np.random.default_rng(seed)
    cases = []
    for i in range(count):
        hkv = int(rng.choice([1, 2, 4, 8]))
        g = int(rng.choice([1, 2, 4, 8, 16]))
        b = int(rng.integers(1, 8))
        band = i % 4  # context bands: tiny, short, medium, past 65536
        lo, hi = [(1, 300), (300, 5000), (5000, 24000), (65537, 70000)][band]
        if band == 3:  # keep the oracle's work small at the longest contexts
            b, hkv = min(b, 2), min(hkv, 2)
        n = int(rng.integers(lo, hi + 1))
        k = int(rng.integers(1, min(2048, n + 64) + 1))
        lens = rng.integers(0, n + 1, size=b)
        if i % 3 == 0:
            lens[0] = n  # a full context
        if i % 5 == 1:
            lens[-1] = 0  # an empty one
        dual = bool(rng.integers(0, 2))
        keys = "lognormal" if rng.integers(0, 2) else "normal"
        cases.append((f"r{i:02d}_b{b}_h{hkv}x{g}_n{n}_k{k}", b, g * hkv, hkv, n, k,
                      [int(x) for x in lens], dual, keys))
    return cases


CASES = _cases()


@pytest.mark.parametrize("name,B,Hq,Hkv,n,k,lens,dual,keys", CASES, ids=[c[0] for c in CASES])
def test_random_shape_fused_entry(name, B, Hq, Hkv, n, k, lens, dual, keys):
    print("random shape", name, "lens", lens, "dual", dual, keys, flush=True)
    dev = device()
    w = synth.Workload(name, B, Hq, Hkv, 128, n, n, k, 1, "hbm", dual, keys)
    t = synth.make_layer(w, seed=11, device=dev)
    lens_d = torch.tensor(lens, dtype=torch.int32, device=dev)
    lens_h = np.array(lens, dtype=np.int32)
    q_att, q_sel, K, V = u16(t["q"]), u16(t["q_sel"]), u16(t["k"]), u16(t["v"])
    o = orc()
    so = o.shape(B, Hq, Hkv, w.head_dim, n)
    # same-step: the attending query selects
    first = Run(w, lens_d, dev)
    first.same_step(t["q"], t["q"], t["k"], t["k"], t["v"], ckv.SRC_DEVICE)
    f_idx, f_nsel, f_out = first.host()
    S_att = o.score_keys(so, q_att, K, lens_h, SCALE, nthreads=8)
    r_idx, r_nsel = o.select_topk(so, S_att, lens_h, k, nthreads=8)
    swaps = check_index_sets(f_idx, f_nsel, r_idx, r_nsel, S_att, lens_h)
    err = np.abs(f_out - oracle_attn_over(so, q_att, K, V, f_idx, f_nsel, k)).max()
    print(f"  same-step: tolerated swaps {swaps}, max abs err {err:.2e}", flush=True)
    assert err <= ATOL_OUT
    # pipelined in place: attend over that set, select with the second query
    second = Run(w, lens_d, dev)
    second.in_place(t["q"], t["q_sel"], t["k"], t["k"], t["v"], ckv.SRC_DEVICE, first.idx,
                    first.n_sel)
    s_idx, s_nsel, s_out = second.host()
    S_sel = S_att if not dual else o.score_keys(so, q_sel, K, lens_h, SCALE, nthreads=8)
    r_idx, r_nsel = o.select_topk(so, S_sel, lens_h, k, nthreads=8)
    swaps = check_index_sets(s_idx, s_nsel, r_idx, r_nsel, S_sel, lens_h)
    err = np.abs(s_out - oracle_attn_over(so, q_att, K, V, f_idx, f_nsel, k)).max()
    print(f"  pipelined in place: tolerated swaps {swaps}, max abs err {err:.2e}", flush=True)
    assert err <= ATOL_OUT
