"""Co-batched dual-token attention, ckv_dual_token_attn, against the oracle
(MI355X only).  Sec. 5.2: the current and the speculative token attend over
the same selected rows in one launch, each also over its own new rows under
the causal mask."""
from __future__ import annotations

import numpy as np
import pytest
import torch

import paper_2607_26475_amd as ckv
from helpers import ATOL_OUT, SCALE, device, orc

pytestmark = pytest.mark.gpu


# k >= 512 (two workgroups per unit fit): a workgroup per token over all rows,
# the own rows merged in the same launch; smaller k: 2G head rows per chunk
# workgroup and the merge launch
@pytest.mark.parametrize("Hq,Hkv,k", [(32, 8, 300), (8, 8, 256), (16, 8, 512), (64, 8, 2048),
                                      (16, 2, 1000), (32, 8, 1024), (8, 8, 600)])
def test_dual_token_attn(Hq, Hkv, k):
    print("dual token", Hq, Hkv, k, flush=True)
    dev = device()
    g = torch.Generator(device=dev)
    g.manual_seed(Hq * 1000 + k)
    B, d = 3, 128
    bf = lambda *shape, sc=1.0: (torch.randn(shape, generator=g, device=dev) * sc).to(
        torch.bfloat16)
    q_cur = bf(B, Hq, d)
    q_spec = (0.8 * q_cur.float() + 0.6 * torch.randn((B, Hq, d), generator=g, device=dev)).to(
        torch.bfloat16)
    k_buf, v_buf = bf(B, Hkv, k, d), bf(B, Hkv, k, d)
    k_loc, v_loc = bf(B, Hkv, 2, d, sc=2.0), bf(B, Hkv, 2, d)
    pattern = [k, 0, 1, k - 3, 17, k // 2, 250, 7]
    ns = np.array([[pattern[(b * Hkv + h) % 8] for h in range(Hkv)] for b in range(B)],
                  np.int32)
    n_sel = torch.from_numpy(ns).to(dev)
    s = ckv.shape_for(B, Hq, Hkv, 4096)
    ws = ckv.workspace(s, k, ckv.ENTRY_DUAL_TOKEN_ATTN)
    out_c = torch.full((B, Hq, d), float("nan"), device=dev)
    out_s = torch.full_like(out_c, float("nan"))
    ckv.profile_begin()
    ckv.dual_token_attn(s, q_cur, q_spec, k_buf, v_buf, n_sel, k_loc, v_loc, k, SCALE, out_c,
                        out_s, ws)
    kernels = ckv.profile_end()
    torch.cuda.synchronize()
    assert ("combine" in kernels) == (k < 512), kernels
    u = lambda t: t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    o = orc()
    so = o.shape(B, Hq, Hkv, d, 4096)
    rc, rs = o.dual_token_attn(so, u(q_cur), u(q_spec), u(k_buf), u(v_buf), ns, u(k_loc),
                               u(v_loc), k, SCALE, nthreads=8)
    ec = np.abs(out_c.cpu().numpy() - rc).max()
    es = np.abs(out_s.cpu().numpy() - rs).max()
    print(f"  max abs err current {ec:.2e}, speculative {es:.2e}", flush=True)
    assert ec <= ATOL_OUT and es <= ATOL_OUT
