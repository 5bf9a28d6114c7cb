"""CPU oracle for critical-KV selection and sparse decode attention.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg may import this package; the library and its binding never
do.  The arithmetic lives in ``ckv_oracle.c`` (plain C, fp64); this module
builds it with gcc and marshals numpy arrays through ctypes.

Functions pinned by the CPU test suite: scores, selection, gather,
attention and their composition.  The paper prints no worked example, so no
function is pinned to a value printed in the paper; the pins are closed forms,
brute force on tiny inputs, library special cases and invariants.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "ckv_oracle.c")
# CKV_ORACLE_LIB names another build of the same source (the sanitizer run
# of the pin suite loads one built with -fsanitize=address,undefined)
DEFAULT_LIB = os.path.join(HERE, "libckv_oracle.so")
LIB = os.environ.get("CKV_ORACLE_LIB") or DEFAULT_LIB


def build(src: str = SRC, out: str = DEFAULT_LIB, extra=()) -> str:
    """Compile the oracle with gcc (-O2, C11) into a shared library."""
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-shared", "-fPIC", *extra,
           f"-I{HERE}", "-o", out, src, "-lm", "-lpthread"]
    subprocess.run(cmd, check=True)
    return out


class _Shape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("max_ctx", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("key_row_stride", ctypes.c_int64),
                ("kv_row_stride", ctypes.c_int64)]


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _u16(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    assert a.dtype == np.uint16, a.dtype
    return a


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


class Oracle:
    """ctypes handle on one build of the oracle library."""

    def __init__(self, path: str = LIB):
        if path == DEFAULT_LIB and not os.path.exists(DEFAULT_LIB):
            build()
        self.path = path
        lib = ctypes.CDLL(path)
        vp, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_float
        lib.ckvref_bf16_to_f64.restype = ctypes.c_double
        lib.ckvref_bf16_to_f64.argtypes = [ctypes.c_uint16]
        lib.ckvref_unit_scores.restype = None
        lib.ckvref_unit_scores.argtypes = [i32, i32, i32, vp, vp, i64, f32, vp]
        lib.ckvref_unit_select.restype = i32
        lib.ckvref_unit_select.argtypes = [i32, vp, i32, vp]
        lib.ckvref_unit_attn.restype = None
        lib.ckvref_unit_attn.argtypes = [i32, i32, i32, vp, vp, vp, f32, vp, vp]
        sp = ctypes.POINTER(_Shape)
        lib.ckvref_score_keys.argtypes = [sp, vp, vp, vp, f32, vp, i32]
        lib.ckvref_select_topk.argtypes = [sp, vp, vp, i32, vp, vp, i32]
        lib.ckvref_gather_kv.argtypes = [sp, vp, vp, vp, vp, i32, vp, vp]
        lib.ckvref_sparse_decode_attn.argtypes = [sp, vp, vp, vp, vp, i32, f32, vp, i32]
        lib.ckvref_critical_kv_attn.argtypes = [sp, vp, vp, vp, vp, vp, vp, i32, f32,
                                                vp, vp, vp, i32]
        lib.ckvref_f64_to_bf16.restype = ctypes.c_uint16
        lib.ckvref_f64_to_bf16.argtypes = [ctypes.c_double]
        lib.ckvref_chunk_landmarks.argtypes = [sp, i32, vp, vp, vp]
        lib.ckvref_expand_chunks.argtypes = [i32, i32, vp, i32, i32, vp]
        lib.ckvref_select_chunks.argtypes = [sp, i32, vp, vp, vp, i32, f32, vp, vp, vp, vp,
                                             i32]
        lib.ckvref_reconstruct_keys.argtypes = [sp, i32, vp, vp, vp, vp, i32, vp]
        lib.ckvref_reconstruct_keys.restype = ctypes.c_int
        lib.ckvref_dual_token_attn.argtypes = [sp, vp, vp, vp, vp, vp, vp, vp, i32, f32, vp,
                                               vp, i32]
        for f in ("ckvref_dual_token_attn", "ckvref_score_keys", "ckvref_select_topk",
                  "ckvref_gather_kv",
                  "ckvref_sparse_decode_attn", "ckvref_critical_kv_attn",
                  "ckvref_chunk_landmarks", "ckvref_expand_chunks", "ckvref_select_chunks"):
            getattr(lib, f).restype = ctypes.c_int
        self.lib = lib

    # ---- single unit ----------------------------------------------------
    def bf16_to_f64(self, bits: int) -> float:
        return self.lib.ckvref_bf16_to_f64(int(bits))

    def unit_scores(self, q: np.ndarray, keys: np.ndarray, scale: float,
                    n: Optional[int] = None) -> np.ndarray:
        """q [G][d] uint16; keys [n][stride] uint16 (first d columns used)."""
        q, keys = _u16(q), _u16(keys)
        G, d = q.shape
        n = keys.shape[0] if n is None else n
        S = np.full(max(n, 1), np.nan)
        self.lib.ckvref_unit_scores(G, d, n, _p(q), _p(keys), keys.shape[1],
                                    scale, _p(S))
        return S[:n]

    def unit_select(self, S: np.ndarray, k: int) -> Tuple[np.ndarray, int]:
        S = np.ascontiguousarray(S, dtype=np.float64)
        idx = np.full(k, -7, dtype=np.int32)
        m = self.lib.ckvref_unit_select(len(S), _p(S), k, _p(idx))
        return idx, m

    def unit_attn(self, q: np.ndarray, k_rows: np.ndarray, v_rows: np.ndarray,
                  scale: float) -> Tuple[np.ndarray, np.ndarray]:
        q, k_rows, v_rows = _u16(q), _u16(k_rows), _u16(v_rows)
        G, d = q.shape
        m = k_rows.shape[0]
        out = np.full((G, d), np.nan)
        p = np.full((G, max(m, 1)), np.nan)
        self.lib.ckvref_unit_attn(G, d, m, _p(q), _p(k_rows), _p(v_rows), scale,
                                  _p(out), _p(p))
        return out, p[:, :m]

    # ---- whole batch, one function per library entry point --------------
    @staticmethod
    def shape(B, Hq, Hkv, d, max_ctx, key_row_stride=None, kv_row_stride=None):
        return _Shape(B, Hq, Hkv, d, max_ctx, 0,
                      d if key_row_stride is None else key_row_stride,
                      d if kv_row_stride is None else kv_row_stride)

    def score_keys(self, s: _Shape, q, k_score, ctx_lens, scale, nthreads=1):
        q, k_score, lens = _u16(q), _u16(k_score), _i32(ctx_lens)
        scores = np.full((s.batch, s.num_kv_heads, s.max_ctx), np.nan)
        rc = self.lib.ckvref_score_keys(ctypes.byref(s), _p(q), _p(k_score), _p(lens),
                                        scale, _p(scores), nthreads)
        assert rc == 0
        return scores

    def select_topk(self, s: _Shape, scores, ctx_lens, k, nthreads=1):
        scores = np.ascontiguousarray(scores, dtype=np.float64)
        lens = _i32(ctx_lens)
        idx = np.full((s.batch, s.num_kv_heads, k), -7, dtype=np.int32)
        n_sel = np.full((s.batch, s.num_kv_heads), -7, dtype=np.int32)
        rc = self.lib.ckvref_select_topk(ctypes.byref(s), _p(scores), _p(lens), k,
                                         _p(idx), _p(n_sel), nthreads)
        assert rc == 0
        return idx, n_sel

    def gather_kv(self, s: _Shape, k_src, v_src, idx, n_sel, k, k_dst, v_dst):
        """k_src/v_src: flat uint16 views whose row stride is kv_row_stride."""
        k_src, v_src = _u16(k_src), _u16(v_src)
        idx, n_sel = _i32(idx), _i32(n_sel)
        assert k_dst.flags.c_contiguous and v_dst.flags.c_contiguous
        rc = self.lib.ckvref_gather_kv(ctypes.byref(s), _p(k_src), _p(v_src), _p(idx),
                                       _p(n_sel), k, _p(k_dst), _p(v_dst))
        assert rc == 0

    def sparse_decode_attn(self, s: _Shape, q_att, k_buf, v_buf, n_sel, k, scale,
                           nthreads=1):
        q_att, k_buf, v_buf, n_sel = _u16(q_att), _u16(k_buf), _u16(v_buf), _i32(n_sel)
        out = np.full((s.batch, s.num_q_heads, s.head_dim), np.nan)
        rc = self.lib.ckvref_sparse_decode_attn(ctypes.byref(s), _p(q_att), _p(k_buf),
                                                _p(v_buf), _p(n_sel), k, scale,
                                                _p(out), nthreads)
        assert rc == 0
        return out

    def critical_kv_attn(self, s: _Shape, q_att, q_sel, k_score, k_src, v_src,
                         ctx_lens, k, scale, nthreads=1):
        q_att, k_score = _u16(q_att), _u16(k_score)
        q_sel = None if q_sel is None else _u16(q_sel)
        k_src, v_src, lens = _u16(k_src), _u16(v_src), _i32(ctx_lens)
        idx = np.full((s.batch, s.num_kv_heads, k), -7, dtype=np.int32)
        n_sel = np.full((s.batch, s.num_kv_heads), -7, dtype=np.int32)
        out = np.full((s.batch, s.num_q_heads, s.head_dim), np.nan)
        rc = self.lib.ckvref_critical_kv_attn(ctypes.byref(s), _p(q_att), _p(q_sel),
                                              _p(k_score), _p(k_src), _p(v_src),
                                              _p(lens), k, scale, _p(idx), _p(n_sel),
                                              _p(out), nthreads)
        assert rc == 0
        return idx, n_sel, out


    # ---- chunk landmarks --------------------------------------------------
    def f64_to_bf16(self, x: float) -> int:
        return self.lib.ckvref_f64_to_bf16(float(x))

    def chunk_landmarks(self, s: _Shape, chunk: int, keys, ctx_lens, fill=0xFFFF):
        """[B][Hkv][ceil(max_ctx/chunk)][d] uint16; unwritten rows keep `fill`."""
        keys, lens = _u16(keys), _i32(ctx_lens)
        cmax = (s.max_ctx + chunk - 1) // chunk
        out = np.full((s.batch, s.num_kv_heads, cmax, s.head_dim), fill, dtype=np.uint16)
        rc = self.lib.ckvref_chunk_landmarks(ctypes.byref(s), chunk, _p(keys), _p(lens),
                                             _p(out))
        assert rc == 0
        return out

    def expand_chunks(self, chunk: int, chunk_idx, n: int, k: int) -> Tuple[np.ndarray, int]:
        ci = _i32(chunk_idx)
        rows = np.full(k, -7, dtype=np.int32)
        r = self.lib.ckvref_expand_chunks(chunk, len(ci), _p(ci), n, k, _p(rows))
        return rows, r

    def select_chunks(self, s: _Shape, chunk: int, q_sel, landmarks, ctx_lens, k, scale,
                      nthreads=1):
        q_sel, lm, lens = _u16(q_sel), _u16(landmarks), _i32(ctx_lens)
        kc = k // chunk
        U = (s.batch, s.num_kv_heads)
        cidx = np.full(U + (kc,), -7, dtype=np.int32)
        nch = np.full(U, -7, dtype=np.int32)
        rows = np.full(U + (k,), -7, dtype=np.int32)
        nrows = np.full(U, -7, dtype=np.int32)
        rc = self.lib.ckvref_select_chunks(ctypes.byref(s), chunk, _p(q_sel), _p(lm), _p(lens),
                                           k, scale, _p(cidx), _p(nch), _p(rows), _p(nrows),
                                           nthreads)
        assert rc == 0
        return cidx, nch, rows, nrows


    # ---- dual-token attention ------------------------------------------------
    def dual_token_attn(self, s: _Shape, q_cur, q_spec, k_buf, v_buf, n_sel, k_local,
                        v_local, k, scale, nthreads=1):
        q_cur, q_spec, k_buf, v_buf = _u16(q_cur), _u16(q_spec), _u16(k_buf), _u16(v_buf)
        k_local, v_local, n_sel = _u16(k_local), _u16(v_local), _i32(n_sel)
        shp = (s.batch, s.num_q_heads, s.head_dim)
        out_cur, out_spec = np.full(shp, np.nan), np.full(shp, np.nan)
        rc = self.lib.ckvref_dual_token_attn(ctypes.byref(s), _p(q_cur), _p(q_spec), _p(k_buf),
                                             _p(v_buf), _p(n_sel), _p(k_local), _p(v_local), k,
                                             scale, _p(out_cur), _p(out_spec), nthreads)
        assert rc == 0
        return out_cur, out_spec


    # ---- low-rank key reconstruction ----------------------------------------
    def reconstruct_keys(self, s: _Shape, rank: int, u_fac, w_fac, idx, n_sel, k,
                         fill=0x7777):
        u_fac, w_fac, idx, n_sel = _u16(u_fac), _u16(w_fac), _i32(idx), _i32(n_sel)
        out = np.full((s.batch, s.num_kv_heads, k, s.head_dim), fill, dtype=np.uint16)
        rc = self.lib.ckvref_reconstruct_keys(ctypes.byref(s), rank, _p(u_fac), _p(w_fac),
                                              _p(idx), _p(n_sel), k, _p(out))
        assert rc == 0
        return out


_default: Optional[Oracle] = None


def get() -> Oracle:
    """The oracle built from this directory's source (built on first use)."""
    global _default
    if _default is None:
        _default = Oracle()
    return _default
