"""The C ABI without a GPU: the library loads, exports every symbol the header
declares, and rejects bad arguments on the host before touching the device."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2607_26475_amd as ckv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ckv.h")
FAKE = 0x100000          # 16-byte aligned, never dereferenced by these calls
STATUS = {"OK": 0, "EINVAL": 1, "ESHAPE": 2, "EUNSUPPORTED": 3, "EWORKSPACE": 4,
          "EHIP": 5}


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\w[\w\s\*]*?\b(ckv_\w+)\(", text, re.M)))


def test_header_functions_are_exported():
    declared = declared_functions()
    assert set(declared) == set(ckv.EXPORTS), declared
    out = subprocess.run(["nm", "-D", "--defined-only", ckv.LIB_PATH],
                         capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (ckv_\w+)$", out, re.M))
    for name in declared:
        assert name in exported, name
        assert hasattr(ckv._lib, name)


def test_abi_version_and_status_text():
    assert ckv.abi_version() == ckv.ABI_VERSION == 9
    texts = {ckv.status_str(v) for v in STATUS.values()}
    assert len(texts) == len(STATUS)
    assert ckv.status_str(99) == "unknown status"


def call_score(shape, q=FAKE, k=FAKE, lens=FAKE, scale=0.088, out=FAKE):
    return ckv._lib.ckv_score_keys(ctypes.byref(shape), q, k, lens, scale, out, 0)


def good_shape(**kw):
    args = dict(batch=2, num_q_heads=8, num_kv_heads=2, max_ctx=64)
    args.update(kw)
    return ckv.shape_for(**args)


@pytest.mark.parametrize("kw,status", [
    (dict(num_q_heads=6, num_kv_heads=4), "ESHAPE"),
    (dict(head_dim=64), "EUNSUPPORTED"),
    (dict(num_q_heads=6, num_kv_heads=2), "EUNSUPPORTED"),
    (dict(num_q_heads=64, num_kv_heads=2), "EUNSUPPORTED"),
    (dict(max_ctx=0), "ESHAPE"),
    (dict(key_row_stride=100), "ESHAPE"),
    (dict(kv_row_stride=132), "ESHAPE"),
    (dict(num_kv_heads=0), "ESHAPE"),
])
def test_shape_validation(kw, status):
    assert call_score(good_shape(**kw)) == STATUS[status]
    assert ckv._lib.ckv_last_error_detail().decode() != ""


def test_pointer_and_value_validation():
    s = good_shape()
    assert call_score(s, q=None) == STATUS["EINVAL"]
    assert call_score(s, out=FAKE + 4) == STATUS["EINVAL"]        # misaligned
    assert call_score(s, scale=0.0) == STATUS["EINVAL"]
    assert call_score(s, scale=-1.0) == STATUS["EINVAL"]
    assert call_score(s, scale=float("nan")) == STATUS["EINVAL"]
    s.reserved = 1
    assert call_score(s) == STATUS["EINVAL"]
    assert ckv._lib.ckv_score_keys(None, FAKE, FAKE, FAKE, 0.1, FAKE, 0) == STATUS["EINVAL"]


def test_budget_and_workspace_validation():
    s = good_shape()
    lib = ckv._lib
    # k < 1
    assert lib.ckv_select_topk(ctypes.byref(s), FAKE, FAKE, 0, FAKE, FAKE, FAKE, 1 << 20,
                               0) == STATUS["ESHAPE"]
    need = ckv.workspace_bytes(s, 16, ckv.ENTRY_SELECT_TOPK)
    assert need > 0
    # workspace missing / too small / misaligned
    assert lib.ckv_select_topk(ctypes.byref(s), FAKE, FAKE, 16, FAKE, FAKE, None, need,
                               0) == STATUS["EWORKSPACE"]
    assert lib.ckv_select_topk(ctypes.byref(s), FAKE, FAKE, 16, FAKE, FAKE, FAKE, need - 1,
                               0) == STATUS["EWORKSPACE"]
    assert lib.ckv_select_topk(ctypes.byref(s), FAKE, FAKE, 16, FAKE, FAKE, FAKE + 16, need,
                               0) == STATUS["EWORKSPACE"]
    # bad src kind is rejected before any device call
    assert lib.ckv_gather_kv(ctypes.byref(s), FAKE, FAKE, 7, FAKE, FAKE, 16, FAKE, FAKE,
                             0) == STATUS["EINVAL"]
    with pytest.raises(ckv.CkvError):
        ckv.workspace_bytes(s, 16, 42)


def test_workspace_sizes_grow_with_shape():
    small = good_shape(max_ctx=1000)
    big = good_shape(max_ctx=100000)
    for e in (ckv.ENTRY_SELECT_TOPK, ckv.ENTRY_SPARSE_DECODE_ATTN,
              ckv.ENTRY_CRITICAL_KV_ATTN):
        a = ckv.workspace_bytes(small, 256, e)
        assert a % 256 == 0 and a > 0
        assert ckv.workspace_bytes(small, 1024, e) >= a
        if e != ckv.ENTRY_SPARSE_DECODE_ATTN:
            assert ckv.workspace_bytes(big, 256, e) > a
    crit = ckv.workspace_bytes(small, 256, ckv.ENTRY_CRITICAL_KV_ATTN)
    assert crit >= ckv.workspace_bytes(small, 256, ckv.ENTRY_SELECT_TOPK)


def test_pipeline_argument_checks():
    lib = ckv._lib
    s = good_shape()
    bufs = (ctypes.c_void_p * 2)(FAKE, FAKE)
    assert lib.ckv_pipeline_create(None) == STATUS["EINVAL"]
    assert lib.ckv_pipeline_destroy(None) == STATUS["OK"]
    assert lib.ckv_pipeline_set_gather_width(None, 64) == STATUS["EINVAL"]
    assert lib.ckv_pipeline_set_checks(None, 1) == STATUS["EINVAL"]
    layers = (ckv.Layer * 2)()
    assert lib.ckv_pipeline_prime(None, ctypes.byref(s), 16, layers, 2, 0, bufs, bufs,
                                  None) == STATUS["EINVAL"]
    # the in-place loop (no buffers) has no room for misses: refused before any launch
    lay = (ckv.Layer * 1)()
    lay[0].idx_true = FAKE
    assert lib.ckv_decode_step(FAKE, ctypes.byref(s), 1, lay, FAKE, 16, 0.1, 0, None, None,
                               FAKE, 1 << 20, None, None) == STATUS["EINVAL"]
    assert "buffers" in lib.ckv_last_error_detail().decode()
    assert lib.ckv_decode_step(None, ctypes.byref(s), 2, layers, FAKE, 16, 0.1, 0, bufs,
                               bufs, FAKE, 1 << 20, None, None) == STATUS["EINVAL"]


def test_corrected_attn_argument_checks():
    lib = ckv._lib
    s = good_shape()
    need = ckv.workspace_bytes(s, 16, ckv.ENTRY_CORRECTED_ATTN)
    assert need >= ckv.workspace_bytes(s, 16, ckv.ENTRY_CRITICAL_KV_ATTN)
    # larger budgets than the LDS miss lists hold need a free-slot list too
    assert (ckv.workspace_bytes(good_shape(max_ctx=20000), 9000, ckv.ENTRY_CORRECTED_ATTN) >
            ckv.workspace_bytes(good_shape(max_ctx=20000), 9000, ckv.ENTRY_CRITICAL_KV_ATTN))

    def call(**kw):
        args = dict(q_att=FAKE, q_sel=None, k_score=FAKE, lens=FAKE, k=16, scale=0.1,
                    k_src=FAKE, v_src=FAKE, kind=0, idx_pred=FAKE, n_pred=FAKE, k_buf=FAKE,
                    v_buf=FAKE, idx_true=FAKE, n_true=FAKE, hits=FAKE, idx_next=FAKE,
                    n_next=FAKE, out=FAKE, ws=FAKE, ws_bytes=need)
        args.update(kw)
        return lib.ckv_corrected_attn(ctypes.byref(s), *args.values(), None)

    assert call(idx_pred=None) == STATUS["EINVAL"]
    assert call(hits=None) == STATUS["EINVAL"]
    assert call(k_buf=FAKE + 8) == STATUS["EINVAL"]
    assert call(kind=5) == STATUS["EINVAL"]
    assert call(k=0) == STATUS["ESHAPE"]
    assert call(ws_bytes=need - 1) == STATUS["EWORKSPACE"]
    assert call(ws=None) == STATUS["EWORKSPACE"]


def test_chunk_entries_argument_checks():
    lib = ckv._lib
    s = good_shape()
    need = ckv.workspace_bytes(s, 16, ckv.ENTRY_CRITICAL_KV_ATTN)
    assert lib.ckv_chunk_landmarks(ctypes.byref(s), 0, FAKE, FAKE, FAKE, None) == STATUS["ESHAPE"]
    assert lib.ckv_chunk_landmarks(ctypes.byref(s), 4, None, FAKE, FAKE, None) == STATUS["EINVAL"]

    def sel(chunk=4, k=16, ws=FAKE, ws_bytes=need, rows=FAKE):
        return lib.ckv_select_chunks(ctypes.byref(s), chunk, FAKE, FAKE, FAKE, k, 0.1, FAKE,
                                     FAKE, rows, FAKE, ws, ws_bytes, None)

    assert sel(k=18) == STATUS["ESHAPE"]       # k not a multiple of the chunk
    assert sel(chunk=0) == STATUS["ESHAPE"]
    assert sel(rows=None) == STATUS["EINVAL"]
    assert sel(ws_bytes=need - 1) == STATUS["EWORKSPACE"]
    assert lib.ckv_chunked_kv_attn(ctypes.byref(s), 4, FAKE, None, FAKE, FAKE, 16, 0.1, FAKE,
                                   FAKE, 3, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, need,
                                   None) == STATUS["EINVAL"]  # bad src kind


def test_dual_token_argument_checks():
    lib = ckv._lib
    s = good_shape()
    need = ckv.workspace_bytes(s, 16, ckv.ENTRY_DUAL_TOKEN_ATTN)
    assert need > ckv.workspace_bytes(s, 16, ckv.ENTRY_SPARSE_DECODE_ATTN)  # 2G head rows

    def call(shape=s, q_spec=FAKE, ws_bytes=need):
        return lib.ckv_dual_token_attn(ctypes.byref(shape), FAKE, q_spec, FAKE, FAKE, FAKE,
                                       FAKE, FAKE, 16, 0.1, FAKE, FAKE, FAKE, ws_bytes, None)

    assert call(q_spec=None) == STATUS["EINVAL"]
    assert call(ws_bytes=need - 1) == STATUS["EWORKSPACE"]
    assert call(shape=good_shape(num_q_heads=32, num_kv_heads=2)) == STATUS["EUNSUPPORTED"]


def test_reconstruct_argument_checks():
    lib = ckv._lib
    s = good_shape()

    def rec(rank=8, u=FAKE, w=FAKE, k=16, dst=FAKE):
        return lib.ckv_reconstruct_keys(ctypes.byref(s), rank, u, w, FAKE, FAKE, k, dst, None)

    assert rec(rank=0) == STATUS["ESHAPE"]
    assert rec(rank=ckv.MAX_RANK + 1) == STATUS["ESHAPE"]
    assert rec(u=None) == STATUS["EINVAL"]
    assert rec(w=FAKE + 2) == STATUS["EINVAL"]
    assert rec(dst=None) == STATUS["EINVAL"]
    assert rec(k=0) == STATUS["ESHAPE"]
    need = ckv.workspace_bytes(s, 16, ckv.ENTRY_CORRECTED_ATTN)

    def call(**kw):
        args = dict(q_att=FAKE, q_sel=None, k_score=FAKE, lens=FAKE, k=16, scale=0.1,
                    k_src=FAKE, v_src=FAKE, kind=0, rank=8, u=FAKE, w=FAKE, idx_pred=FAKE,
                    n_pred=FAKE, k_buf=FAKE, v_buf=FAKE, idx_true=FAKE, n_true=FAKE,
                    hits=FAKE, idx_next=FAKE, n_next=FAKE, out=FAKE, ws=FAKE, ws_bytes=need)
        args.update(kw)
        return lib.ckv_corrected_attn_lowrank(ctypes.byref(s), *args.values(), None)

    assert call(rank=0) == STATUS["ESHAPE"]
    assert call(u=None) == STATUS["EINVAL"]
    assert call(w=None) == STATUS["EINVAL"]
    assert call(v_src=None) == STATUS["EINVAL"]
    # keys are rebuilt, so k_src may be NULL: the call gets as far as the workspace check
    assert call(k_src=None, ws_bytes=need - 1) == STATUS["EWORKSPACE"]


def test_layer_struct_layout(tmp_path):
    """The ctypes mirror of ckv_layer has the C compiler's offsets."""
    names = [n for n, _ in ckv.Layer._fields_]
    src = tmp_path / "layout.c"
    src.write_text('#include <stddef.h>\n#include <stdio.h>\n#include "ckv.h"\n'
                   "int main(void) {\n" +
                   "".join(f'  printf("%zu\\n", offsetof(ckv_layer, {n}));\n' for n in names) +
                   '  printf("%zu\\n", sizeof(ckv_layer));\n  return 0;\n}\n')
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)], check=True)
    got = [int(x) for x in subprocess.run([str(exe)], capture_output=True, text=True,
                                          check=True).stdout.split()]
    assert got == [getattr(ckv.Layer, n).offset for n in names] + [ctypes.sizeof(ckv.Layer)]


def test_critical_kv_attn_mode_checks():
    """idx_in (rows in place) and k_buf (assembled rows) are exclusive; each
    pipelined mode needs n_sel_in."""
    lib = ckv._lib
    s = good_shape()
    need = ckv.workspace_bytes(s, 16, ckv.ENTRY_CRITICAL_KV_ATTN)

    def call(idx_in=None, k_buf=None, v_buf=None, n_in=None, k_src=FAKE, v_src=FAKE):
        return lib.ckv_critical_kv_attn(ctypes.byref(s), FAKE, None, FAKE, FAKE, 16, 0.1,
                                        k_src, v_src, 0, idx_in, k_buf, v_buf, n_in, FAKE,
                                        FAKE, FAKE, FAKE, need, 0)

    assert call(idx_in=FAKE, k_buf=FAKE, v_buf=FAKE, n_in=FAKE) == STATUS["EINVAL"]
    assert call(idx_in=FAKE) == STATUS["EINVAL"]             # no n_sel_in
    assert call(idx_in=FAKE, n_in=FAKE, k_src=None) == STATUS["EINVAL"]
    assert call(k_buf=FAKE, v_buf=FAKE) == STATUS["EINVAL"]  # no n_sel_in
    assert "exclusive" in (lib.ckv_critical_kv_attn(
        ctypes.byref(s), FAKE, None, FAKE, FAKE, 16, 0.1, FAKE, FAKE, 0, FAKE, FAKE, FAKE,
        FAKE, FAKE, FAKE, FAKE, FAKE, need, 0), ckv._lib.ckv_last_error_detail().decode())[1]


def test_noalloc_entry_refuses_oversized_shapes():
    """The fixed-scratch entry checks the shape's workspace against
    CKV_NOALLOC_SCRATCH_BYTES before any runtime call (so also without a GPU)."""
    lib = ckv._lib
    big = good_shape(batch=8, num_q_heads=32, num_kv_heads=8, max_ctx=131072)
    assert ckv.workspace_bytes(big, 4096, ckv.ENTRY_CRITICAL_KV_ATTN) > ckv.NOALLOC_SCRATCH_BYTES
    rc = lib.ckv_critical_kv_attn_noalloc(ctypes.byref(big), FAKE, None, FAKE, FAKE, 4096, 0.1,
                                          FAKE, FAKE, 0, None, None, None, None, FAKE, FAKE,
                                          FAKE, 0)
    assert rc == STATUS["EWORKSPACE"]
    assert "fixed scratch" in lib.ckv_last_error_detail().decode()
    # argument errors come first too
    assert lib.ckv_critical_kv_attn_noalloc(ctypes.byref(big), FAKE, None, FAKE, FAKE, 0, 0.1,
                                            FAKE, FAKE, 0, None, None, None, None, FAKE, FAKE,
                                            FAKE, 0) == STATUS["ESHAPE"]
    # the Llama-8B layer fits
    llama = good_shape(batch=16, num_q_heads=32, num_kv_heads=8, max_ctx=32768)
    assert ckv.workspace_bytes(llama, 2048, ckv.ENTRY_CRITICAL_KV_ATTN) <= \
        ckv.NOALLOC_SCRATCH_BYTES


def test_probe_sizes_and_refusals():
    s = good_shape(batch=16, num_q_heads=32, num_kv_heads=8, max_ctx=32768)
    assert ckv.probe_sink_words(s, 2048, ckv.PROBE_STANDALONE) == 128 * 8 * 256
    assert ckv.probe_sink_words(s, 2048, ckv.PROBE_ROW_HALVES) == 256 * 1024
    assert ckv.probe_sink_words(s, 2048, ckv.PROBE_HEAD_HALVES) == 256 * 1024
    assert ckv.probe_sink_words(s, 4096, ckv.PROBE_HEAD_HALVES) == 0   # halves: k <= 2048
    assert ckv.probe_sink_words(s, 2048, 3) == 0
    assert ckv.probe_sink_words(good_shape(batch=3, num_kv_heads=2), 256,
                                ckv.PROBE_ROW_HALVES) == 16 * 1024  # 6 units -> 8 per XCD round
    call = ckv._lib.ckv_probe_read_rows
    assert call(ctypes.byref(s), FAKE, FAKE, FAKE, 2048, 3, FAKE, 1 << 20, None) == STATUS["EINVAL"]
    assert call(ctypes.byref(s), FAKE, FAKE, FAKE, 4096, ckv.PROBE_ROW_HALVES, FAKE, 1 << 20,
                None) == STATUS["ESHAPE"]
    assert call(ctypes.byref(s), FAKE, FAKE, FAKE, 2048, ckv.PROBE_STANDALONE, FAKE, 1000,
                None) == STATUS["EINVAL"]   # sink smaller than needed
    assert call(ctypes.byref(s), None, FAKE, FAKE, 2048, ckv.PROBE_STANDALONE, FAKE, 1 << 20,
                None) == STATUS["EINVAL"]
    assert call(ctypes.byref(s), FAKE, FAKE, FAKE + 4, 2048, ckv.PROBE_STANDALONE, FAKE,
                1 << 20, None) == STATUS["EINVAL"]   # misaligned
    empty = good_shape(batch=0, num_q_heads=32, num_kv_heads=8, max_ctx=32768)
    for mode in (ckv.PROBE_STANDALONE, ckv.PROBE_ROW_HALVES, ckv.PROBE_HEAD_HALVES):
        assert call(ctypes.byref(empty), FAKE, FAKE, FAKE, 2048, mode, FAKE, 0, None) == 0


def test_debug_mode_switch_without_a_gpu():
    """Debug mode checks device-side inputs only when a unit exists: host-side
    refusals are unchanged, and empty batches still return before any launch."""
    assert ckv._lib.ckv_set_debug(1) == 0
    try:
        s = good_shape()
        assert call_score(s, q=None) == STATUS["EINVAL"]
        empty = good_shape(batch=0)
        assert call_score(empty) == 0
    finally:
        assert ckv._lib.ckv_set_debug(0) == 0


def test_one_launch_modes_match_the_header():
    """The one-launch setting's modes: the binding's constants are the
    header's enum values, and every mode (and any other nonzero value, which
    means row halves) is accepted without a GPU."""
    text = open(os.path.join(os.path.dirname(__file__), "..", "include", "ckv.h")).read()
    vals = dict(re.findall(r"(CKV_ONE_LAUNCH_\w+) = (\d+)", text))
    assert vals == {"CKV_ONE_LAUNCH_OFF": "0", "CKV_ONE_LAUNCH_ROW_HALVES": "1",
                    "CKV_ONE_LAUNCH_HEAD_HALVES": "2"}, vals
    assert (ckv.ONE_LAUNCH_OFF, ckv.ONE_LAUNCH_ROW_HALVES, ckv.ONE_LAUNCH_HEAD_HALVES) == (0, 1, 2)
    try:
        for mode in (ckv.ONE_LAUNCH_OFF, ckv.ONE_LAUNCH_HEAD_HALVES, 7, False, True):
            ckv.set_one_launch_same_step(mode)
    finally:
        ckv.set_one_launch_same_step(ckv.ONE_LAUNCH_ROW_HALVES)
