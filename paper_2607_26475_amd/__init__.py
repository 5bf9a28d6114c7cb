"""Python binding of libckv (critical-KV selection and sparse decode attention
on MI355X).

Argument marshalling only: every function passes raw pointers, sizes and the
current HIP stream to the C ABI declared in ``include/ckv.h`` and raises
``CkvError`` on a non-zero status.  All computation happens in the HIP
kernels of ``libckv.so``; there is no fallback.  torch is used for device
memory, pinned host memory and streams.

The library must have been built first (``python paper_2607_26475_amd/build.py``
or ``__graft_entry__.build()``); importing this package without it raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

__all__ = [
    "CkvError", "Shape", "shape_for", "workspace_bytes", "workspace",
    "score_keys", "select_topk", "gather_kv", "sparse_decode_attn",
    "critical_kv_attn", "critical_kv_attn_noalloc", "NOALLOC_SCRATCH_BYTES", "corrected_attn", "chunk_landmarks", "select_chunks",
    "chunked_kv_attn", "dual_token_attn", "reconstruct_keys", "corrected_attn_lowrank",
    "MAX_RANK", "ABI_VERSION", "profile_begin", "profile_end", "abi_version",
    "Layer", "layer_array", "Pipeline", "status_str", "LIB_PATH",
    "SRC_DEVICE", "SRC_HOST_PINNED", "ENTRY_SELECT_TOPK",
    "ENTRY_SPARSE_DECODE_ATTN", "ENTRY_CRITICAL_KV_ATTN", "ENTRY_CORRECTED_ATTN", "ENTRY_DUAL_TOKEN_ATTN", "ENTRY_DECODE_STEP",
    "EXPORTS", "probe_read_rows", "probe_sink_words", "PROBE_STANDALONE", "PROBE_ROW_HALVES",
    "PROBE_HEAD_HALVES", "set_debug", "set_one_launch_same_step", "ONE_LAUNCH_OFF",
    "ONE_LAUNCH_ROW_HALVES", "ONE_LAUNCH_HEAD_HALVES",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libckv.so")

SRC_DEVICE, SRC_HOST_PINNED = 0, 1
ENTRY_SELECT_TOPK, ENTRY_SPARSE_DECODE_ATTN, ENTRY_CRITICAL_KV_ATTN = 1, 2, 3
ENTRY_CORRECTED_ATTN, ENTRY_DUAL_TOKEN_ATTN, ENTRY_DECODE_STEP = 4, 5, 6
PROBE_STANDALONE, PROBE_ROW_HALVES, PROBE_HEAD_HALVES = 0, 1, 2
EXPORTS = ("ckv_abi_version", "ckv_status_str", "ckv_last_error_detail",
           "ckv_workspace_bytes", "ckv_score_keys", "ckv_select_topk",
           "ckv_gather_kv", "ckv_sparse_decode_attn", "ckv_critical_kv_attn",
           "ckv_critical_kv_attn_noalloc",
           "ckv_corrected_attn", "ckv_chunk_landmarks", "ckv_select_chunks",
           "ckv_chunked_kv_attn", "ckv_dual_token_attn", "ckv_reconstruct_keys",
           "ckv_corrected_attn_lowrank",
           "ckv_kernel_name", "ckv_profile_begin", "ckv_profile_begin_sampled",
           "ckv_profile_end",
           "ckv_pipeline_create", "ckv_pipeline_destroy", "ckv_pipeline_set_gather_width",
           "ckv_pipeline_set_checks",
           "ckv_pipeline_prime",
           "ckv_decode_step", "ckv_probe_read_rows", "ckv_probe_sink_words", "ckv_set_debug",
           "ckv_set_one_launch_same_step")
KERNEL_COUNT = 16
MAX_RANK = 4096
ABI_VERSION = 9  # CKV_ABI_VERSION of include/ckv.h that this binding marshals for


class CkvError(RuntimeError):
    def __init__(self, fn: str, status: int, detail: str):
        super().__init__(f"{fn}: {status_str(status)} ({status}): {detail}")
        self.status = status


class KernelStats(ctypes.Structure):
    """Mirror of ``ckv_kernel_stats``."""
    _fields_ = [("launches", ctypes.c_int64), ("total_ms", ctypes.c_double),
                ("max_ms", ctypes.c_double)]


class Layer(ctypes.Structure):
    """Mirror of ``ckv_layer``."""
    _fields_ = [(name, ctypes.c_void_p) for name in (
        "q_att", "q_sel", "k_score", "k_src", "v_src", "idx_prev", "n_sel_prev",
        "idx_next", "n_sel_next", "out", "idx_true", "n_true", "hits")] + [
        ("lr_rank", ctypes.c_int32), ("lr_u", ctypes.c_void_p), ("lr_w", ctypes.c_void_p),
        ("chunk", ctypes.c_int32), ("landmarks", ctypes.c_void_p),
        ("k_local", ctypes.c_void_p), ("v_local", ctypes.c_void_p),
        ("out_spec", ctypes.c_void_p)]


class Shape(ctypes.Structure):
    """Mirror of ``ckv_shape``."""
    _fields_ = [("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("max_ctx", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("key_row_stride", ctypes.c_int64),
                ("kv_row_stride", ctypes.c_int64)]


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run "
                          "`python paper_2607_26475_amd/build.py` first")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    sp = ctypes.POINTER(Shape)
    sig = {
        "ckv_abi_version": (ctypes.c_int, []),
        "ckv_status_str": (ctypes.c_char_p, [ctypes.c_int]),
        "ckv_last_error_detail": (ctypes.c_char_p, []),
        "ckv_workspace_bytes": (ctypes.c_int, [sp, i32, ctypes.c_int, ctypes.POINTER(sz)]),
        "ckv_score_keys": (ctypes.c_int, [sp, vp, vp, vp, ctypes.c_float, vp, vp]),
        "ckv_select_topk": (ctypes.c_int, [sp, vp, vp, i32, vp, vp, vp, sz, vp]),
        "ckv_gather_kv": (ctypes.c_int, [sp, vp, vp, ctypes.c_int, vp, vp, i32, vp, vp, vp]),
        "ckv_sparse_decode_attn": (ctypes.c_int, [sp, vp, vp, vp, vp, i32, ctypes.c_float,
                                                  vp, vp, sz, vp]),
        "ckv_critical_kv_attn": (ctypes.c_int, [sp, vp, vp, vp, vp, i32, ctypes.c_float,
                                                vp, vp, ctypes.c_int, vp, vp, vp, vp, vp,
                                                vp, vp, vp, sz, vp]),
        "ckv_critical_kv_attn_noalloc": (ctypes.c_int, [sp, vp, vp, vp, vp, i32,
                                                        ctypes.c_float, vp, vp, ctypes.c_int,
                                                        vp, vp, vp, vp, vp, vp, vp, vp]),
        "ckv_corrected_attn": (ctypes.c_int, [sp, vp, vp, vp, vp, i32, ctypes.c_float,
                                              vp, vp, ctypes.c_int, vp, vp, vp, vp, vp, vp,
                                              vp, vp, vp, vp, vp, sz, vp]),
        "ckv_chunk_landmarks": (ctypes.c_int, [sp, i32, vp, vp, vp, vp]),
        "ckv_select_chunks": (ctypes.c_int, [sp, i32, vp, vp, vp, i32, ctypes.c_float, vp, vp,
                                             vp, vp, vp, sz, vp]),
        "ckv_chunked_kv_attn": (ctypes.c_int, [sp, i32, vp, vp, vp, vp, i32, ctypes.c_float,
                                               vp, vp, ctypes.c_int, vp, vp, vp, vp, vp, vp,
                                               sz, vp]),
        "ckv_dual_token_attn": (ctypes.c_int, [sp, vp, vp, vp, vp, vp, vp, vp, i32,
                                               ctypes.c_float, vp, vp, vp, sz, vp]),
        "ckv_reconstruct_keys": (ctypes.c_int, [sp, i32, vp, vp, vp, vp, i32, vp, vp]),
        "ckv_corrected_attn_lowrank": (ctypes.c_int, [sp, vp, vp, vp, vp, i32, ctypes.c_float,
                                                      vp, vp, ctypes.c_int, i32, vp, vp, vp,
                                                      vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                                      vp, sz, vp]),
        "ckv_kernel_name": (ctypes.c_char_p, [ctypes.c_int]),
        "ckv_profile_begin": (ctypes.c_int, [ctypes.c_uint32]),
        "ckv_profile_begin_sampled": (ctypes.c_int, [ctypes.c_uint32, ctypes.c_uint32]),
        "ckv_profile_end": (ctypes.c_int, [ctypes.POINTER(KernelStats)]),
        "ckv_probe_read_rows": (ctypes.c_int, [sp, vp, vp, vp, i32, ctypes.c_int, vp, sz, vp]),
        "ckv_probe_sink_words": (sz, [sp, i32, ctypes.c_int]),
        "ckv_set_debug": (ctypes.c_int, [ctypes.c_int]),
        "ckv_set_one_launch_same_step": (ctypes.c_int, [ctypes.c_int]),
        "ckv_pipeline_create": (ctypes.c_int, [ctypes.POINTER(vp)]),
        "ckv_pipeline_destroy": (ctypes.c_int, [vp]),
        "ckv_pipeline_set_gather_width": (ctypes.c_int, [vp, ctypes.c_int]),
        "ckv_pipeline_set_checks": (ctypes.c_int, [vp, ctypes.c_uint]),
        "ckv_pipeline_prime": (ctypes.c_int, [vp, sp, i32, ctypes.POINTER(Layer), ctypes.c_int,
                                              ctypes.c_int, ctypes.POINTER(vp),
                                              ctypes.POINTER(vp), vp]),
        "ckv_decode_step": (ctypes.c_int, [vp, sp, ctypes.c_int, ctypes.POINTER(Layer), vp,
                                           i32, ctypes.c_float, ctypes.c_int,
                                           ctypes.POINTER(vp), ctypes.POINTER(vp), vp, sz, vp,
                                           vp]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


_lib = _load()
if _lib.ckv_abi_version() != ABI_VERSION:
    raise ImportError(f"{LIB_PATH} has ABI {_lib.ckv_abi_version()}, the binding expects "
                      f"{ABI_VERSION}; rebuild it")


def abi_version() -> int:
    return _lib.ckv_abi_version()


def status_str(status: int) -> str:
    return _lib.ckv_status_str(status).decode()


def _check(fn: str, status: int) -> None:
    if status != 0:
        raise CkvError(fn, status, _lib.ckv_last_error_detail().decode())


def shape_for(batch: int, num_q_heads: int, num_kv_heads: int, max_ctx: int,
              head_dim: int = 128, key_row_stride: Optional[int] = None,
              kv_row_stride: Optional[int] = None) -> Shape:
    return Shape(batch, num_q_heads, num_kv_heads, head_dim, max_ctx, 0,
                 head_dim if key_row_stride is None else key_row_stride,
                 head_dim if kv_row_stride is None else kv_row_stride)


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def workspace_bytes(shape: Shape, k: int, entry: int) -> int:
    n = ctypes.c_size_t(0)
    _check("ckv_workspace_bytes",
           _lib.ckv_workspace_bytes(ctypes.byref(shape), k, entry, ctypes.byref(n)))
    return n.value


def workspace(shape: Shape, k: int, entry: int, device="cuda") -> torch.Tensor:
    """A device byte tensor large enough for `entry` (torch allocations are
    256-byte aligned)."""
    return torch.empty(max(workspace_bytes(shape, k, entry), 1), dtype=torch.uint8,
                       device=device)


def score_keys(shape: Shape, q, k_score, ctx_lens, scale: float, scores,
               stream=None) -> None:
    _check("ckv_score_keys", _lib.ckv_score_keys(
        ctypes.byref(shape), _ptr(q), _ptr(k_score), _ptr(ctx_lens), scale,
        _ptr(scores), _stream(stream)))


def select_topk(shape: Shape, scores, ctx_lens, k: int, idx, n_sel, ws,
                stream=None) -> None:
    _check("ckv_select_topk", _lib.ckv_select_topk(
        ctypes.byref(shape), _ptr(scores), _ptr(ctx_lens), k, _ptr(idx), _ptr(n_sel),
        _ptr(ws), ws.numel() if ws is not None else 0, _stream(stream)))


def gather_kv(shape: Shape, k_src, v_src, src_kind: int, idx, n_sel, k: int,
              k_dst, v_dst, stream=None) -> None:
    _check("ckv_gather_kv", _lib.ckv_gather_kv(
        ctypes.byref(shape), _ptr(k_src), _ptr(v_src), src_kind, _ptr(idx), _ptr(n_sel),
        k, _ptr(k_dst), _ptr(v_dst), _stream(stream)))


def sparse_decode_attn(shape: Shape, q_att, k_buf, v_buf, n_sel, k: int,
                       scale: float, out, ws, stream=None) -> None:
    _check("ckv_sparse_decode_attn", _lib.ckv_sparse_decode_attn(
        ctypes.byref(shape), _ptr(q_att), _ptr(k_buf), _ptr(v_buf), _ptr(n_sel), k, scale,
        _ptr(out), _ptr(ws), ws.numel() if ws is not None else 0, _stream(stream)))


def critical_kv_attn(shape: Shape, q_att, q_sel, k_score, ctx_lens, k: int,
                     scale: float, k_src, v_src, src_kind: int, k_buf, v_buf,
                     n_sel_in, idx_out, n_sel_out, out, ws, stream=None,
                     idx_in=None) -> None:
    """Same-step (k_buf and idx_in None), pipelined over an assembled buffer
    (k_buf), or pipelined over the rows idx_in read in place."""
    _check("ckv_critical_kv_attn", _lib.ckv_critical_kv_attn(
        ctypes.byref(shape), _ptr(q_att), _ptr(q_sel), _ptr(k_score), _ptr(ctx_lens), k,
        scale, _ptr(k_src), _ptr(v_src), src_kind, _ptr(idx_in), _ptr(k_buf), _ptr(v_buf),
        _ptr(n_sel_in), _ptr(idx_out), _ptr(n_sel_out), _ptr(out), _ptr(ws),
        ws.numel() if ws is not None else 0, _stream(stream)))


NOALLOC_SCRATCH_BYTES = 64 << 20  # CKV_NOALLOC_SCRATCH_BYTES


def critical_kv_attn_noalloc(shape: Shape, q_att, q_sel, k_score, ctx_lens, k: int,
                             scale: float, k_src, v_src, src_kind: int, k_buf, v_buf,
                             n_sel_in, idx_out, n_sel_out, out, stream=None,
                             idx_in=None) -> None:
    """critical_kv_attn with the library's fixed per-device scratch instead of
    a workspace (the call allocates nothing)."""
    _check("ckv_critical_kv_attn_noalloc", _lib.ckv_critical_kv_attn_noalloc(
        ctypes.byref(shape), _ptr(q_att), _ptr(q_sel), _ptr(k_score), _ptr(ctx_lens), k,
        scale, _ptr(k_src), _ptr(v_src), src_kind, _ptr(idx_in), _ptr(k_buf), _ptr(v_buf),
        _ptr(n_sel_in), _ptr(idx_out), _ptr(n_sel_out), _ptr(out), _stream(stream)))


def corrected_attn(shape: Shape, q_att, q_sel, k_score, ctx_lens, k: int, scale: float,
                   k_src, v_src, src_kind: int, idx_pred, n_pred, k_buf, v_buf, idx_true,
                   n_true, hits, idx_next, n_next, out, ws, stream=None) -> None:
    _check("ckv_corrected_attn", _lib.ckv_corrected_attn(
        ctypes.byref(shape), _ptr(q_att), _ptr(q_sel), _ptr(k_score), _ptr(ctx_lens), k,
        scale, _ptr(k_src), _ptr(v_src), src_kind, _ptr(idx_pred), _ptr(n_pred),
        _ptr(k_buf), _ptr(v_buf), _ptr(idx_true), _ptr(n_true), _ptr(hits), _ptr(idx_next),
        _ptr(n_next), _ptr(out), _ptr(ws), ws.numel() if ws is not None else 0,
        _stream(stream)))


def corrected_attn_lowrank(shape: Shape, q_att, q_sel, k_score, ctx_lens, k: int,
                           scale: float, k_src, v_src, src_kind: int, rank: int, u_fac, w_fac,
                           idx_pred, n_pred, k_buf, v_buf, idx_true, n_true, hits, idx_next,
                           n_next, out, ws, stream=None) -> None:
    _check("ckv_corrected_attn_lowrank", _lib.ckv_corrected_attn_lowrank(
        ctypes.byref(shape), _ptr(q_att), _ptr(q_sel), _ptr(k_score), _ptr(ctx_lens), k,
        scale, _ptr(k_src), _ptr(v_src), src_kind, rank, _ptr(u_fac), _ptr(w_fac),
        _ptr(idx_pred), _ptr(n_pred), _ptr(k_buf), _ptr(v_buf), _ptr(idx_true), _ptr(n_true),
        _ptr(hits), _ptr(idx_next), _ptr(n_next), _ptr(out), _ptr(ws),
        ws.numel() if ws is not None else 0, _stream(stream)))


def reconstruct_keys(shape: Shape, rank: int, u_fac, w_fac, idx, n_sel, k: int, k_dst,
                     stream=None) -> None:
    _check("ckv_reconstruct_keys", _lib.ckv_reconstruct_keys(
        ctypes.byref(shape), rank, _ptr(u_fac), _ptr(w_fac), _ptr(idx), _ptr(n_sel), k,
        _ptr(k_dst), _stream(stream)))


def dual_token_attn(shape: Shape, q_cur, q_spec, k_buf, v_buf, n_sel, k_local, v_local,
                    k: int, scale: float, out_cur, out_spec, ws, stream=None) -> None:
    _check("ckv_dual_token_attn", _lib.ckv_dual_token_attn(
        ctypes.byref(shape), _ptr(q_cur), _ptr(q_spec), _ptr(k_buf), _ptr(v_buf), _ptr(n_sel),
        _ptr(k_local), _ptr(v_local), k, scale, _ptr(out_cur), _ptr(out_spec), _ptr(ws),
        ws.numel() if ws is not None else 0, _stream(stream)))


def chunk_landmarks(shape: Shape, chunk: int, keys, ctx_lens, landmarks,
                    stream=None) -> None:
    _check("ckv_chunk_landmarks", _lib.ckv_chunk_landmarks(
        ctypes.byref(shape), chunk, _ptr(keys), _ptr(ctx_lens), _ptr(landmarks),
        _stream(stream)))


def select_chunks(shape: Shape, chunk: int, q_sel, landmarks, ctx_lens, k: int,
                  scale: float, chunk_idx, n_chunks, rows, n_rows, ws, stream=None) -> None:
    _check("ckv_select_chunks", _lib.ckv_select_chunks(
        ctypes.byref(shape), chunk, _ptr(q_sel), _ptr(landmarks), _ptr(ctx_lens), k, scale,
        _ptr(chunk_idx), _ptr(n_chunks), _ptr(rows), _ptr(n_rows), _ptr(ws),
        ws.numel() if ws is not None else 0, _stream(stream)))


def chunked_kv_attn(shape: Shape, chunk: int, q_att, q_sel, landmarks, ctx_lens, k: int,
                    scale: float, k_src, v_src, src_kind: int, chunk_idx, n_chunks, rows,
                    n_rows, out, ws, stream=None) -> None:
    _check("ckv_chunked_kv_attn", _lib.ckv_chunked_kv_attn(
        ctypes.byref(shape), chunk, _ptr(q_att), _ptr(q_sel), _ptr(landmarks),
        _ptr(ctx_lens), k, scale, _ptr(k_src), _ptr(v_src), src_kind, _ptr(chunk_idx),
        _ptr(n_chunks), _ptr(rows), _ptr(n_rows), _ptr(out), _ptr(ws),
        ws.numel() if ws is not None else 0, _stream(stream)))


KERNEL_IDS = {"zero": 0, "score": 1, "hist": 2, "filter": 3, "finish": 4, "attn": 5,
              "combine": 6, "dual": 7, "gather": 8, "miss": 9, "landmarks": 10,
              "expand": 11, "reconstruct": 12, "select_attn": 13, "probe": 14,
              "critical": 15}


def profile_begin(kernels=None, every: int = 1) -> None:
    """Start stamping library kernels with dispatch start/end events: all of
    them, or only the named kernel classes; with every > 1 only launches 0,
    every, 2*every, ... of each class."""
    mask = (1 << KERNEL_COUNT) - 1
    if kernels is not None:
        mask = 0
        for name in kernels:
            mask |= 1 << KERNEL_IDS[name]
    _check("ckv_profile_begin_sampled", _lib.ckv_profile_begin_sampled(mask, every))


def profile_end() -> dict:
    """Stop recording; {kernel name: (launches, total_ms, max_ms)} for every
    kernel class that ran (waits for the recorded kernels)."""
    arr = (KernelStats * KERNEL_COUNT)()
    _check("ckv_profile_end", _lib.ckv_profile_end(arr))
    return {_lib.ckv_kernel_name(i).decode(): (arr[i].launches, arr[i].total_ms, arr[i].max_ms)
            for i in range(KERNEL_COUNT) if arr[i].launches}


def set_debug(on: bool) -> None:
    """Debug mode (process-wide): entries check their device-side inputs
    (context lengths, input counts and index sets) on the device and every
    launch synchronises; a violation raises CkvError (CKV_EINVAL)."""
    _check("ckv_set_debug", _lib.ckv_set_debug(1 if on else 0))


ONE_LAUNCH_OFF, ONE_LAUNCH_ROW_HALVES, ONE_LAUNCH_HEAD_HALVES = 0, 1, 2


def set_one_launch_same_step(on) -> None:
    """Whether same-step calls run as one launch where that form applies
    (process-wide).  True / ONE_LAUNCH_ROW_HALVES (the default): one launch
    whose two workgroups per unit attend over half the rows each and merge in
    the launch.  False / ONE_LAUNCH_OFF: the scoring launch, then the
    selection and attention launch, attending the same way (the same bits).
    ONE_LAUNCH_HEAD_HALVES: two workgroups per unit attending over the whole
    set with half the heads each, in one launch where that applies; the same
    index sets, outputs within fp32 rounding of the other forms."""
    _check("ckv_set_one_launch_same_step", _lib.ckv_set_one_launch_same_step(int(on)))


def probe_sink_words(shape: Shape, k: int, mode: int) -> int:
    """uint32 words of sink that probe_read_rows needs (0: shape, k or mode
    invalid)."""
    return int(_lib.ckv_probe_sink_words(ctypes.byref(shape), k, mode))


def probe_read_rows(shape: Shape, k_rows, v_rows, idx, k: int, mode: int, sink,
                    stream=None) -> None:
    """Read-rate probe (measurement only): reads the rows idx selects with the
    access pattern of one attention launch (PROBE_*) and no arithmetic; sink
    is a device tensor of at least probe_sink_words() int32/uint32 words."""
    _check("ckv_probe_read_rows", _lib.ckv_probe_read_rows(
        ctypes.byref(shape), _ptr(k_rows), _ptr(v_rows), _ptr(idx), k, mode, _ptr(sink),
        sink.numel() if sink is not None else 0, _stream(stream)))


def layer_array(layers) -> "ctypes.Array":
    """dicts with the ckv_layer field names (tensors, ints or None) -> the
    ckv_layer array the decode loop takes; an array is returned as it is, so
    a loop can build its per-parity arrays once."""
    if isinstance(layers, ctypes.Array):
        return layers
    arr = (Layer * len(layers))()
    for i, d in enumerate(layers):
        for name, typ in Layer._fields_:
            if typ is ctypes.c_int32:
                setattr(arr[i], name, int(d.get(name) or 0))
            else:
                setattr(arr[i], name, _ptr(d.get(name)))
    return arr


class Pipeline:
    """The decode loop of ``ckv_decode_step`` (owns its events): two buffers
    refilled on a copy stream, or, with ``k_buf`` and ``v_buf`` None, rows
    read in place from a cache in device memory."""

    def __init__(self):
        h = ctypes.c_void_p()
        _check("ckv_pipeline_create", _lib.ckv_pipeline_create(ctypes.byref(h)))
        self._h = h

    def close(self) -> None:
        if self._h:
            _lib.ckv_pipeline_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    CHECK_NO_FILL_WAIT, CHECK_NO_RELEASE_WAIT, CHECK_POISON, CHECK_NO_DEFER = 1, 2, 4, 8

    def set_checks(self, flags: int) -> None:
        """Tests of the event protocol only: skip the fill or release waits,
        or poison released buffers; or run every selection in its own layer's
        call (CHECK_NO_DEFER; see ckv_pipeline_set_checks)."""
        _check("ckv_pipeline_set_checks", _lib.ckv_pipeline_set_checks(self._h, flags))

    def set_gather_width(self, workgroups: int) -> None:
        _check("ckv_pipeline_set_gather_width",
               _lib.ckv_pipeline_set_gather_width(self._h, workgroups))

    @staticmethod
    def _bufs(k_buf, v_buf):
        """ctypes arrays of the two buffers; (None, None) for the in-place loop."""
        if k_buf is None and v_buf is None:
            return None, None
        kb = (ctypes.c_void_p * 2)(_ptr(k_buf[0]), _ptr(k_buf[1]))
        vb = (ctypes.c_void_p * 2)(_ptr(v_buf[0]), _ptr(v_buf[1]))
        return kb, vb

    def prime(self, shape: Shape, k: int, layers, src_kind: int, k_buf, v_buf,
              copy_stream) -> None:
        arr = layer_array(layers)
        kb, vb = self._bufs(k_buf, v_buf)
        _check("ckv_pipeline_prime", _lib.ckv_pipeline_prime(
            self._h, ctypes.byref(shape), k, arr, len(layers), src_kind, kb, vb,
            _stream(copy_stream)))

    def step(self, shape: Shape, layers, ctx_lens, k: int, scale: float, src_kind: int,
             k_buf, v_buf, ws, compute_stream, copy_stream) -> None:
        """One decode step over ``layers`` (dicts or a ``layer_array``)."""
        arr = layer_array(layers)
        kb, vb = self._bufs(k_buf, v_buf)
        _check("ckv_decode_step", _lib.ckv_decode_step(
            self._h, ctypes.byref(shape), len(layers), arr, _ptr(ctx_lens), k, scale,
            src_kind, kb, vb, _ptr(ws), ws.numel(), _stream(compute_stream),
            _stream(copy_stream)))
