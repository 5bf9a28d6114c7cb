"""The read-rate probe (MI355X only).

The probe's duration stands for what the memory system gives an attention
launch's access pattern, so it must read exactly the rows of that pattern.
Each thread writes the XOR of the 16-byte K and V pieces it loads; the test
recomputes every thread's checksum on the CPU from the pattern the header
states (the grid of each form, each wave's run of 16-row blocks, 4 rows per
load, the lane's 16 bytes of a row, clamped positions) and compares them word
for word, for the three forms, separate and interleaved K|V, a ragged budget,
-1 padding and a position past max_ctx.
"""
from __future__ import annotations

import numpy as np
import pytest
import torch

import paper_2607_26475_amd as ckv
from helpers import device

pytestmark = pytest.mark.gpu

B, HQ, HKV, D, N = 2, 32, 8, 128, 3000


def _words(t: torch.Tensor) -> np.ndarray:
    """[B][Hkv][N][row] bf16 -> uint32 [U][N][row / 2]."""
    a = t.contiguous().view(torch.int16).cpu().numpy().view(np.uint32)
    return a.reshape(B * HKV, N, -1)


def _lane_xor(Kw, Vw, u, p, vo):
    """XOR of lane l's 16-byte pieces of rows p[l] (K at word 0, V at word vo)."""
    lch = np.arange(64) & 15
    cols = 4 * lch[:, None] + np.arange(4)[None, :]
    kx = np.bitwise_xor.reduce(Kw[u, p[:, None], cols], axis=1)
    vx = np.bitwise_xor.reduce(Vw[u, p[:, None], vo + cols], axis=1)
    return kx ^ vx


def _wave(Kw, Vw, u, pos, i0, i1, vo):
    """The checksums of one wave reading positions pos[i0 .. i1]."""
    lrow = np.arange(64) >> 4
    acc = np.zeros(64, np.uint32)
    for b in range(i0, i1 + 1, 16):
        for it in range(4):
            i = np.minimum(b + 4 * it + lrow, i1)
            p = np.clip(pos[i], 0, N - 1)
            acc ^= _lane_xor(Kw, Vw, u, p, vo)
    return acc


def _expected(mode, Kw, Vw, idx, k, vo):
    U = B * HKV
    if mode == ckv.PROBE_STANDALONE:
        chunks = (k + 255) // 256
        out = np.zeros((U * chunks, 256), np.uint32)
        for u in range(U):
            for c in range(chunks):
                for w in range(4):
                    i0 = c * 256 + 64 * w
                    i1 = min(i0 + 64, k) - 1
                    if i0 <= i1:
                        out[u * chunks + c, 64 * w:64 * w + 64] = _wave(Kw, Vw, u, idx[u], i0,
                                                                        i1, vo)
        return out.ravel()
    blocks = (U + 7) // 8 * 8 * 2
    out = np.zeros((blocks, 1024), np.uint32)
    for blk in range(blocks):
        grp, r = blk // 16, blk % 16
        part, u = r >> 3, grp * 8 + (r & 7)
        if u >= U:
            continue
        lo, hi = 0, k
        if mode == ckv.PROBE_ROW_HALVES:
            per = ((k + 1) // 2 + 15) & ~15
            lo = min(part * per, k)
            hi = min(lo + per, k)
        pos = idx[u, lo:hi]
        nblk = (hi - lo + 15) // 16
        for w in range(16):
            b0, b1 = w * nblk // 16, (w + 1) * nblk // 16
            if b0 < b1:
                out[blk, 64 * w:64 * w + 64] = _wave(Kw, Vw, u, pos, 16 * b0,
                                                     min(16 * b1, hi - lo) - 1, vo)
    return out.ravel()


@pytest.mark.parametrize("mode", [ckv.PROBE_STANDALONE, ckv.PROBE_ROW_HALVES,
                                  ckv.PROBE_HEAD_HALVES])
@pytest.mark.parametrize("interleaved", [False, True])
@pytest.mark.parametrize("k", [256, 200])
def test_probe_reads_the_pattern(mode, interleaved, k):
    print("probe", mode, interleaved, k, flush=True)
    dev = device()
    g = torch.Generator(device="cpu").manual_seed(7 + k)
    if interleaved:
        kv = torch.randn((B, HKV, N, 2 * D), generator=g).to(torch.bfloat16).to(dev)
        k_rows, v_rows, vo = kv, kv[..., D:], D // 2
        shape = ckv.shape_for(B, HQ, HKV, N, kv_row_stride=2 * D)
        Kw = Vw = _words(kv)
    else:
        K = torch.randn((B, HKV, N, D), generator=g).to(torch.bfloat16).to(dev)
        V = torch.randn((B, HKV, N, D), generator=g).to(torch.bfloat16).to(dev)
        k_rows, v_rows, vo = K, V, 0
        shape = ckv.shape_for(B, HQ, HKV, N)
        Kw, Vw = _words(K), _words(V)
    rng = np.random.default_rng(k)
    idx = np.stack([np.sort(rng.choice(N, k, replace=False)) for _ in range(B * HKV)])
    idx = idx.astype(np.int32)
    idx[0, -9:] = -1         # padding reads row 0
    idx[1, 3] = N + 5        # past max_ctx: row N - 1
    idx_t = torch.from_numpy(idx).to(dev)
    words = ckv.probe_sink_words(shape, k, mode)
    assert words > 0
    sink = torch.full((words,), -1, dtype=torch.int32, device=dev)
    ckv.probe_read_rows(shape, k_rows, v_rows if not interleaved else kv.data_ptr() + 2 * D,
                        idx_t, k, mode, sink)
    torch.cuda.synchronize()
    got = sink.cpu().numpy().view(np.uint32)
    want = _expected(mode, Kw, Vw, idx, k, vo)
    assert got.shape == want.shape
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, (bad[:8], got[bad[:8]], want[bad[:8]])
