"""Seeded synthetic inputs for critical-KV decode workloads.

This module only draws inputs: queries, keys, values and context lengths in
bf16 with the shapes and value distributions of the workloads below.  It holds
none of the method's arithmetic (no scoring, selection or attention), so that
the HIP library and the CPU oracle can share it without sharing computation.

Every tensor is drawn from its own ``torch.Generator`` whose seed is a stable
hash of (workload name, seed, layer, tensor tag); the same call on the same
device always gives the same bits.  fp32 draws are rounded to bf16 with
round-to-nearest-even (``Tensor.to(torch.bfloat16)``).

Workloads (Llama-shaped decode, head_dim 128):
  tiny      B1,  8/2 heads, n 4096, k 256, 1 layer; 16 planted keys per KV
            head equal to bf16(4 * mean of the group's query vectors)
  llama8b   B16, 32/8, n 32768, k 2048, 32 layers; keys N(0,1) times a
            per-(layer, KV head) channel scale ~ LogNormal(0, 0.5)
  long128k  B8,  32/8, n 131072, k 4096, 32 layers; K/V host-pinned
  dual64    B64, 32/8, n_b ~ U{16384..65536}, k 2048, 32 layers; two queries,
            q2 = bf16(0.8 q1 + 0.6 eps); K/V host-pinned
  million   B1,  32/8, n 1048576, k 8192, 32 layers; 1 % of the positions of
            each (request, KV head) drawn from a high-norm cluster along the
            group's mean query direction; K/V host-pinned
Reduced variants (suffix ``_s``) keep head layout and distributions with
shorter contexts, ragged lengths and one or two layers.
"""
from __future__ import annotations

import dataclasses
import math
import zlib
from typing import Dict, Optional

import numpy as np
import torch

__all__ = ["Workload", "WORKLOADS", "make_layer", "to_u16", "generator",
           "interleave_kv", "host_kv", "low_rank_factors"]


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    q_heads: int
    kv_heads: int
    head_dim: int
    max_ctx: int          # rows stored per (request, KV head)
    ctx_min: int          # n_b ~ U{ctx_min..max_ctx}; == max_ctx => fixed
    k: int                # sparse budget per KV head
    layers: int
    placement: str        # "hbm": K/V in device memory; "host": host-pinned
    dual: bool            # a second (speculative) query selects
    keys: str             # "normal" | "planted" | "lognormal" | "cluster"

    @property
    def group(self) -> int:
        return self.q_heads // self.kv_heads

    @property
    def units(self) -> int:
        return self.batch * self.kv_heads


def _w(name, B, hq, hkv, n, k, L, place, dual=False, keys="normal", nmin=None):
    return Workload(name, B, hq, hkv, 128, n, n if nmin is None else nmin, k, L,
                    place, dual, keys)


WORKLOADS: Dict[str, Workload] = {w.name: w for w in [
    _w("tiny", 1, 8, 2, 4096, 256, 1, "hbm", keys="planted"),
    _w("llama8b", 16, 32, 8, 32768, 2048, 32, "hbm", keys="lognormal"),
    _w("long128k", 8, 32, 8, 131072, 4096, 32, "host"),
    _w("dual64", 64, 32, 8, 65536, 2048, 32, "host", dual=True, nmin=16384),
    _w("million", 1, 32, 8, 1048576, 8192, 32, "host", keys="cluster"),
    # reduced variants: same head layout and distributions, ragged lengths
    _w("llama8b_s", 2, 32, 8, 5000, 256, 2, "hbm", keys="lognormal", nmin=3001),
    _w("long128k_s", 2, 32, 8, 16384, 512, 2, "host", nmin=12007),
    _w("dual64_s", 4, 32, 8, 6000, 256, 2, "host", dual=True, nmin=1500),
    _w("million_s", 1, 32, 8, 70000, 1024, 1, "host", keys="cluster"),
]}


def generator(wl: str, seed: int, layer: int, tag: str, device) -> torch.Generator:
    """A generator seeded by a stable hash of (workload, seed, layer, tag)."""
    h = zlib.crc32(f"{wl}/{seed}/{layer}/{tag}".encode())
    g = torch.Generator(device=device)
    g.manual_seed(h)
    return g


def to_u16(t: torch.Tensor) -> np.ndarray:
    """bf16 tensor -> numpy uint16 array of its bit patterns (host copy)."""
    assert t.dtype == torch.bfloat16
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def _randn(shape, g, device) -> torch.Tensor:
    return torch.randn(shape, generator=g, device=device, dtype=torch.float32)


def _fill_normal_bf16(out: torch.Tensor, g: torch.Generator, scale=None) -> None:
    """out[b] <- bf16(N(0,1) [* scale]) slice by slice (bounded fp32 temp)."""
    for b in range(out.shape[0]):
        z = torch.randn(out.shape[1:], generator=g, device=out.device,
                        dtype=torch.float32)
        if scale is not None:
            z.mul_(scale)
        out[b].copy_(z.to(torch.bfloat16))
        del z


def make_layer(w: Workload, seed: int = 0, layer: int = 0,
               device: str | torch.device = "cpu",
               ctx_override: Optional[int] = None) -> Dict[str, torch.Tensor]:
    """Draw one layer of inputs for workload ``w`` on ``device``.

    Returns bf16 tensors ``q`` (attending query, [B][Hq][d]), ``q_sel``
    (selecting query; the same tensor unless ``w.dual``), ``k`` and ``v``
    ([B][Hkv][max_ctx][d], rows >= n_b hold draws too and must be ignored),
    int32 ``ctx_lens`` [B] and ``marked``, a bool [B][Hkv][max_ctx] mask of the
    planted or cluster positions (all False for plain normal keys).  All live
    on ``device``; host placement is arranged by the caller (``host_kv``).
    """
    dev = torch.device(device)
    B, Hq, Hkv, d, n = w.batch, w.q_heads, w.kv_heads, w.head_dim, w.max_ctx
    G = w.group
    gq = generator(w.name, seed, layer, "q", dev)
    q = _randn((B, Hq, d), gq, dev).to(torch.bfloat16)
    if w.dual:
        ge = generator(w.name, seed, layer, "q2", dev)
        eps = _randn((B, Hq, d), ge, dev)
        q_sel = (0.8 * q.float() + 0.6 * eps).to(torch.bfloat16)
    else:
        q_sel = q
    if ctx_override is not None:
        lens = torch.full((B,), int(ctx_override), dtype=torch.int32)
    elif w.ctx_min < n:
        # a request's context length is the same in every layer
        gl = generator(w.name, seed, 0, "len", "cpu")
        lens = torch.randint(w.ctx_min, n + 1, (B,), generator=gl,
                             dtype=torch.int64).to(torch.int32)
    else:
        lens = torch.full((B,), n, dtype=torch.int32)
    lens = lens.to(dev)

    k = torch.empty((B, Hkv, n, d), dtype=torch.bfloat16, device=dev)
    v = torch.empty((B, Hkv, n, d), dtype=torch.bfloat16, device=dev)
    chan = None
    if w.keys == "lognormal":
        gs = generator(w.name, seed, layer, "chan", dev)
        chan = torch.exp(0.5 * _randn((Hkv, 1, d), gs, dev))
    _fill_normal_bf16(k, generator(w.name, seed, layer, "k", dev), chan)
    _fill_normal_bf16(v, generator(w.name, seed, layer, "v", dev))

    marked = torch.zeros((B, Hkv, n), dtype=torch.bool, device=dev)
    if w.keys in ("planted", "cluster"):
        gp = generator(w.name, seed, layer, "pos", dev)
        qbar = q.float().view(B, Hkv, G, d).mean(dim=2)          # [B][Hkv][d]
        for b in range(B):
            for h in range(Hkv):
                if w.keys == "planted":
                    cnt = 16
                else:
                    cnt = int(round(0.01 * n))
                pos = torch.randperm(n, generator=gp, device=dev)[:cnt]
                marked[b, h, pos] = True
                if w.keys == "planted":
                    row = (4.0 * qbar[b, h]).to(torch.bfloat16)
                    k[b, h, pos] = row.expand(cnt, d)
                else:
                    u = qbar[b, h] / qbar[b, h].norm()
                    z = _randn((cnt, d), gp, dev)
                    rows = 2.0 * math.sqrt(d) * u + 0.5 * z
                    k[b, h, pos] = rows.to(torch.bfloat16)
    return {"q": q, "q_sel": q_sel, "k": k, "v": v, "ctx_lens": lens,
            "marked": marked}


def low_rank_factors(w: Workload, rank: int, seed: int = 0, layer: int = 0,
                     device: str | torch.device = "cpu"):
    """Low-rank key-cache factors of one layer: ``u`` [B][Hkv][max_ctx][rank]
    with bf16(N(0,1)) entries and ``w`` [B][Hkv][rank][d] with
    bf16(N(0,1) / sqrt(rank)) entries, so that a rebuilt key entry has about
    unit variance like the drawn keys.  The factors are drawn independently of
    the layer's keys: the rebuilt keys are not approximations of them, which
    keeps a key that was rebuilt apart from one that was fetched."""
    dev = torch.device(device)
    B, Hkv, n, d = w.batch, w.kv_heads, w.max_ctx, w.head_dim
    u = torch.empty((B, Hkv, n, rank), dtype=torch.bfloat16, device=dev)
    wf = torch.empty((B, Hkv, rank, d), dtype=torch.bfloat16, device=dev)
    _fill_normal_bf16(u, generator(w.name, seed, layer, f"lr_u{rank}", dev))
    _fill_normal_bf16(wf, generator(w.name, seed, layer, f"lr_w{rank}", dev),
                      1.0 / math.sqrt(rank))
    return u, wf


def interleave_kv(k: torch.Tensor, v: torch.Tensor) -> torch.Tensor:
    """K and V interleaved per row on k's device: [B][Hkv][n][2][d].

    Row j of (b, h) holds its key then its value (2*d contiguous bf16), so a
    selected position is one 512-byte read; keys are rows at stride 2*d from
    the start, values the same from element d.
    """
    B, Hkv, n, d = k.shape
    out = torch.empty((B, Hkv, n, 2, d), dtype=torch.bfloat16, device=k.device)
    for b in range(B):
        out[b, :, :, 0].copy_(k[b])
        out[b, :, :, 1].copy_(v[b])
    return out


def host_kv(k: torch.Tensor, v: torch.Tensor) -> torch.Tensor:
    """K and V interleaved per row in pinned host memory: [B][Hkv][n][2][d].

    Row j of (b, h) then holds its key and value as 2*d contiguous bf16
    values; K rows are at stride 2*d from the tensor's start and V rows at
    the same stride from element d.
    """
    B, Hkv, n, d = k.shape
    out = torch.empty((B, Hkv, n, 2, d), dtype=torch.bfloat16, pin_memory=True)
    for b in range(B):
        out[b, :, :, 0].copy_(k[b])
        out[b, :, :, 1].copy_(v[b])
    return out
