"""Claims in the pipelined scoring pass (MI355X only).

A pipelined attend-and-score launch whose scoring adds its first-digit
histograms (contexts above 65536 positions) takes its work as claims of 64
groups of 32 positions from a counter when the pass has at least four claims
per scoring workgroup; the workgroup that takes the last claim resets the
counter.  These cases are the smallest shapes that take claims on the device
(16 units of 2^18 positions: 2048 claims for 512 resident workgroups), with
ragged contexts (claims that end inside or lie past n_b) and, in one case, a
row count that is not a multiple of 4 (the scores' unaligned store path).
Two layers, and in one case two steps, run through the decode step on one
workspace with one clear, so every later pass starts from the counter the
previous pass reset.  Every unit is checked against the oracle.
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


def _workload(max_ctx):
    return dataclasses.replace(synth.WORKLOADS["long128k_s"], name=f"claims{max_ctx}",
                               batch=2, max_ctx=max_ctx, ctx_min=150001, k=512, layers=2)


def _claims_per_wg(w, dev):
    # the attend-and-score kernel keeps two scoring workgroups per CU resident
    # (its LDS allows two); claims of 64 groups of 32 positions per unit
    nwg = 2 * torch.cuda.get_device_properties(dev).multi_processor_count
    groups = (w.max_ctx + 31) // 32
    return w.units * ((groups + 63) // 64) / min(nwg, w.units * groups)


@pytest.mark.parametrize("max_ctx,in_place,steps", [(262144, True, 2), (262144, False, 1),
                                                    (262147, True, 1)])
def test_claims_decode_step_matches_oracle(max_ctx, in_place, steps):
    dev = device()
    w = _workload(max_ctx)
    cpw = _claims_per_wg(w, dev)
    _log(f"claims: max_ctx {max_ctx}, in place {in_place}, steps {steps}, "
         f"{cpw:.2f} claims per workgroup")
    assert cpw >= 4, "the shape no longer reaches the claim path"
    layers = 2
    lp = Loop(w, layers, steps=steps, seed=31, dev=dev)
    lp.in_place = in_place
    lp.bootstrap()
    boot = ([i.cpu().numpy() for i in lp.idx[0]], [n.cpu().numpy() for n in lp.nsel[0]])
    pipe = ckv.Pipeline()
    ckv.profile_begin()
    hist = lp.run(steps, pipe)
    kernels = ckv.profile_end()
    pipe.close()
    # one clear per call: every later pass found the counter and histograms clear
    assert kernels["zero"][0] == steps, kernels
    o = orc()
    lens = lp.lens.cpu().numpy()
    so = o.shape(w.batch, w.q_heads, w.kv_heads, w.head_dim, w.max_ctx)
    prev = boot
    for st in range(1, steps + 1):
        g_idx, g_nsel, g_out = hist[st - 1][:3]
        for l in range(layers):
            K, V = u16(lp.t[l]["k"]), u16(lp.t[l]["v"])
            S = o.score_keys(so, u16(lp.q_sel[st][l]), K, lens, SCALE, nthreads=8)
            r_idx, r_nsel = o.select_topk(so, S, lens, w.k, nthreads=8)
            swaps = check_index_sets(g_idx[l], g_nsel[l], r_idx, r_nsel, S, lens)
            ref = oracle_attn_over(so, u16(lp.q_att[st][l]), K, V, prev[0][l], prev[1][l], w.k)
            err = np.abs(g_out[l] - ref).max()
            _log(f"  step {st} layer {l}: swaps {swaps}, max abs err {err:.2e}")
            assert err <= ATOL_OUT
        prev = (g_idx, g_nsel)
