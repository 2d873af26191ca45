"""Python binding of libkvlink.so, the gfx950 KVLink hot path (arXiv 2502.16002).

Argument marshalling only: every step of the path runs in the library (host
layout code and HIP kernels).  torch supplies device memory and streams.  The
functions carry the names of the C entry points declared in include/kvlink.h
and raise :class:`KVLinkError` on a non-OK status.  There is no fallback: if
the library is not built, importing the binding raises.
"""
import ctypes
import os

import numpy as np
# torch first: libkvlink.so then binds to the HIP runtime torch has loaded
# (loading the library first would bring in a second HIP runtime beside
# torch's, and the two do not share devices)
import torch  # noqa: F401

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libkvlink.so")

KVLINK_F32, KVLINK_BF16 = 0, 1
KVLINK_STAGE_ROPE, KVLINK_STAGE_SPLIT, KVLINK_STAGE_COMBINE = 1, 2, 4
KVLINK_STAGE_ALL = 7
KVLINK_PLAN_XCD = 1
KVLINK_PLAN_COMBINE = 4
KVLINK_PLAN_IN_LAUNCH = 8
STATUS = {0: "OK", 1: "ERR_INVALID_ARG", 2: "ERR_UNSUPPORTED", 3: "ERR_LAYOUT",
          4: "ERR_WORKSPACE", 5: "ERR_HIP"}


class KVLinkError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


class kvlink_kv_view(ctypes.Structure):
    _fields_ = [("base", ctypes.c_void_p),
                ("layer_stride", ctypes.c_int64),
                ("head_stride", ctypes.c_int64),
                ("row_stride", ctypes.c_int64),
                ("seq_stride", ctypes.c_int64),
                ("page_stride", ctypes.c_int64),
                ("block_table", ctypes.c_void_p),
                ("page_size", ctypes.c_int32),
                ("max_pages", ctypes.c_int32)]


class kvlink_span(ctypes.Structure):
    _fields_ = [("src_seq", ctypes.c_int32), ("src_row", ctypes.c_int32),
                ("dst_seq", ctypes.c_int32), ("dst_row", ctypes.c_int32),
                ("len", ctypes.c_int32), ("delta", ctypes.c_int32)]


SPAN_FIELDS = 6   # int32 fields of kvlink_span, in declaration order


class kvlink_attend_plan(ctypes.Structure):
    _fields_ = [("table", ctypes.c_void_p),
                ("table_len", ctypes.c_int32),
                ("n_workgroups", ctypes.c_int32),
                ("n_units", ctypes.c_int32),
                ("n_segments", ctypes.c_int32),
                ("row_block", ctypes.c_int32),
                ("n_seqs", ctypes.c_int32),
                ("n_split_units", ctypes.c_int32),
                ("flags", ctypes.c_uint32),
                ("rope_table", ctypes.c_void_p)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                          "(there is no CPU fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    i32, i64, f64, f32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double, ctypes.c_float
    vp, sz = ctypes.c_void_p, ctypes.c_size_t
    lib.kvlink_build_layout.argtypes = [i32] + [vp] * 16
    lib.kvlink_build_layout.restype = ctypes.c_int
    lib.kvlink_reencode_keys.argtypes = [ctypes.c_int, i32, i32, i32, f64, i32, vp, i32,
                                         kvlink_kv_view, kvlink_kv_view, vp]
    lib.kvlink_reencode_keys.restype = ctypes.c_int
    lib.kvlink_encode_keys_at_positions.argtypes = lib.kvlink_reencode_keys.argtypes
    lib.kvlink_encode_keys_at_positions.restype = ctypes.c_int
    lib.kvlink_reencode_keys_mapped.argtypes = [ctypes.c_int, i32, i32, i32, f64, i32, vp, i32,
                                                vp, ctypes.c_int64, kvlink_kv_view,
                                                kvlink_kv_view, vp]
    lib.kvlink_reencode_keys_mapped.restype = ctypes.c_int
    lib.kvlink_group_spans.argtypes = [i32, vp, i32, vp, vp, ctypes.POINTER(i32)]
    lib.kvlink_group_spans.restype = ctypes.c_int
    lib.kvlink_reencode_keys_shared.argtypes = [ctypes.c_int, i32, i32, i32, f64, i32, vp, vp, i32,
                                                kvlink_kv_view, kvlink_kv_view, vp]
    lib.kvlink_reencode_keys_shared.restype = ctypes.c_int
    lib.kvlink_load_stage_bytes.argtypes = [ctypes.c_int, i32, i32, i32, i32]
    lib.kvlink_load_stage_bytes.restype = sz
    lib.kvlink_load_and_reencode.argtypes = [ctypes.c_int, i32, i32, i32, f64, i32, vp, i32, vp, vp,
                                             i32, vp, sz, kvlink_kv_view, kvlink_kv_view, i32, vp,
                                             vp]
    lib.kvlink_load_and_reencode.restype = ctypes.c_int
    lib.kvlink_attend_make_plan.argtypes = [ctypes.c_int, i32, i32, i32, i32, vp, vp, vp, i32,
                                            i32, i32, ctypes.c_uint32, vp, i64,
                                            ctypes.POINTER(kvlink_attend_plan)]
    lib.kvlink_attend_make_plan.restype = ctypes.c_int
    lib.kvlink_attend_workspace_bytes.argtypes = [ctypes.c_int, i32, i32, i32, i32,
                                                  ctypes.POINTER(kvlink_attend_plan)]
    lib.kvlink_attend_workspace_bytes.restype = sz
    lib.kvlink_attend_new_tokens.argtypes = [
        ctypes.c_int, i32, i32, i32, f64, f32, i32, i32, i32, i32,
        vp, vp, vp, vp, vp, vp, vp, kvlink_kv_view, kvlink_kv_view, i32, vp, vp,
        kvlink_attend_plan, vp, sz, vp]
    lib.kvlink_attend_new_tokens.restype = ctypes.c_int
    lib.kvlink_attend_new_tokens_noalloc.argtypes = lib.kvlink_attend_new_tokens.argtypes[:-3] + [vp]
    lib.kvlink_attend_new_tokens_noalloc.restype = ctypes.c_int
    lib.kvlink_attend_new_tokens_fused.argtypes = (lib.kvlink_attend_new_tokens.argtypes[:-3] +
                                                   [vp, vp, i32, vp, sz, vp])
    lib.kvlink_attend_new_tokens_fused.restype = ctypes.c_int
    lib.kvlink_attend_stages.argtypes = lib.kvlink_attend_new_tokens.argtypes + [ctypes.c_uint32]
    lib.kvlink_attend_stages.restype = ctypes.c_int
    lib.kvlink_attend_rope_table.argtypes = [i32, f64, i32, vp, vp, vp]
    lib.kvlink_attend_rope_table.restype = ctypes.c_int
    lib.kvlink_last_error.restype = ctypes.c_char_p
    lib.kvlink_version.restype = ctypes.c_char_p
    return lib


_lib = _load()


def kvlink_last_error():
    return _lib.kvlink_last_error().decode()


def kvlink_version():
    return _lib.kvlink_version().decode()


def _check(status):
    if status != 0:
        raise KVLinkError(status, kvlink_last_error())


def _ptr(x):
    """Device or host address of a torch tensor / numpy array, or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    return x.data_ptr()


def _stream(stream):
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def kv_view(tensor, layer_stride, head_stride, row_stride, seq_stride=0, page_stride=0,
            block_table=None, page_size=0, max_pages=0):
    """A kvlink_kv_view over a device tensor (strides in elements)."""
    return kvlink_kv_view(_ptr(tensor), int(layer_stride), int(head_stride), int(row_stride),
                          int(seq_stride), int(page_stride), _ptr(block_table), int(page_size),
                          int(max_pages))


# ------------------------------------------------------------------ entry points


def kvlink_build_layout(seq_doc_ptr, doc_len, link_count, n_query, doc_src_seq=None,
                        doc_src_row=None, doc_src_pos0=None):
    """Host index maps of a request batch; returns a dict of numpy arrays.

    Keys: spans [n_docs, 6] int32 (kvlink_span fields), doc_pos0, seq_cached,
    seq_new_ptr, new_pos, new_visible, new_doc, new_slot and totals
    (n_docs, n_new, max_doc_len, max_cached, max_new, max_total).
    """
    def arr(a):
        return None if a is None else np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    sdp, dl, lc, nq = arr(seq_doc_ptr), arr(doc_len), arr(link_count), arr(n_query)
    src_seq, src_row, src_pos0 = arr(doc_src_seq), arr(doc_src_row), arr(doc_src_pos0)
    n_seqs = len(nq)
    if len(sdp) != n_seqs + 1:
        raise ValueError("seq_doc_ptr must have n_seqs + 1 entries")
    totals = np.zeros(6, np.int64)
    _check(_lib.kvlink_build_layout(n_seqs, _ptr(sdp), _ptr(dl), _ptr(lc), _ptr(nq),
                                    _ptr(src_seq), _ptr(src_row), _ptr(src_pos0),
                                    None, None, None, None, None, None, None, None,
                                    _ptr(totals)))
    n_docs, n_new = int(totals[0]), int(totals[1])
    out = {
        "spans": np.zeros((n_docs, SPAN_FIELDS), np.int32),
        "doc_pos0": np.zeros(n_docs, np.int32),
        "seq_cached": np.zeros(n_seqs, np.int32),
        "seq_new_ptr": np.zeros(n_seqs + 1, np.int32),
        "new_pos": np.zeros(n_new, np.int32),
        "new_visible": np.zeros(n_new, np.int32),
        "new_doc": np.zeros(n_new, np.int32),
        "new_slot": np.zeros(n_new, np.int32),
        "totals": totals,
    }
    _check(_lib.kvlink_build_layout(n_seqs, _ptr(sdp), _ptr(dl), _ptr(lc), _ptr(nq),
                                    _ptr(src_seq), _ptr(src_row), _ptr(src_pos0),
                                    _ptr(out["spans"]), _ptr(out["doc_pos0"]),
                                    _ptr(out["seq_cached"]), _ptr(out["seq_new_ptr"]),
                                    _ptr(out["new_pos"]), _ptr(out["new_visible"]),
                                    _ptr(out["new_doc"]), _ptr(out["new_slot"]),
                                    _ptr(totals)))
    return out


def kvlink_reencode_keys(dtype, n_layers, n_kv_heads, head_dim, rope_theta, n_spans, d_spans,
                         max_span_len, src, dst, stream=None):
    _check(_lib.kvlink_reencode_keys(int(dtype), int(n_layers), int(n_kv_heads), int(head_dim),
                                     float(rope_theta), int(n_spans), _ptr(d_spans),
                                     int(max_span_len), src, dst, _stream(stream)))


def kvlink_encode_keys_at_positions(dtype, n_layers, n_kv_heads, head_dim, rope_theta, n_spans,
                                    d_spans, max_span_len, src, dst, stream=None):
    _check(_lib.kvlink_encode_keys_at_positions(int(dtype), int(n_layers), int(n_kv_heads),
                                                int(head_dim), float(rope_theta), int(n_spans),
                                                _ptr(d_spans), int(max_span_len), src, dst,
                                                _stream(stream)))


def kvlink_reencode_keys_mapped(dtype, n_layers, n_kv_heads, head_dim, rope_theta, n_spans,
                                d_spans, max_span_len, d_stored_pos, stored_pos_stride, src, dst,
                                stream=None):
    _check(_lib.kvlink_reencode_keys_mapped(int(dtype), int(n_layers), int(n_kv_heads),
                                            int(head_dim), float(rope_theta), int(n_spans),
                                            _ptr(d_spans), int(max_span_len), _ptr(d_stored_pos),
                                            int(stored_pos_stride), src, dst, _stream(stream)))


def kvlink_group_spans(spans, max_group=0):
    """Group spans [n, 6] int32 (kvlink_span fields) that read the same stored
    rows, runs longer than max_group (> 0) cut into near-equal groups:
    returns (order, group_ptr) int32 arrays."""
    sp = np.ascontiguousarray(np.asarray(spans, dtype=np.int32).reshape(-1, SPAN_FIELDS))
    n = len(sp)
    order = np.zeros(max(n, 1), np.int32)
    gptr = np.zeros(n + 1, np.int32)
    ng = ctypes.c_int32(0)
    _check(_lib.kvlink_group_spans(n, _ptr(sp), int(max_group), _ptr(order), _ptr(gptr),
                                   ctypes.byref(ng)))
    return order[:n], gptr[:ng.value + 1]


def kvlink_reencode_keys_shared(dtype, n_layers, n_kv_heads, head_dim, rope_theta, n_groups,
                                d_group_ptr, d_spans, max_span_len, src, dst, stream=None):
    _check(_lib.kvlink_reencode_keys_shared(int(dtype), int(n_layers), int(n_kv_heads),
                                            int(head_dim), float(rope_theta), int(n_groups),
                                            _ptr(d_group_ptr), _ptr(d_spans), int(max_span_len),
                                            src, dst, _stream(stream)))


def kvlink_load_stage_bytes(dtype, n_kv_heads, head_dim, stored_rows, n_slots=2):
    return int(_lib.kvlink_load_stage_bytes(int(dtype), int(n_kv_heads), int(head_dim),
                                            int(stored_rows), int(n_slots)))


def kvlink_load_and_reencode(dtype, n_layers, n_kv_heads, head_dim, rope_theta, n_spans, d_spans,
                             max_span_len, h_k, h_v, stored_rows, d_stage, stage_bytes, k_dst,
                             v_dst, literal=0, copy_stream=None, compute_stream=None):
    _check(_lib.kvlink_load_and_reencode(int(dtype), int(n_layers), int(n_kv_heads),
                                         int(head_dim), float(rope_theta), int(n_spans),
                                         _ptr(d_spans), int(max_span_len), _ptr(h_k), _ptr(h_v),
                                         int(stored_rows), _ptr(d_stage), int(stage_bytes),
                                         k_dst, v_dst, int(literal), _stream(copy_stream),
                                         _stream(compute_stream)))


def kvlink_attend_make_plan(dtype, n_q_heads, n_kv_heads, head_dim, seq_new_ptr, seq_cached,
                            new_visible, n_compute_units, n_workgroups=0, row_block=0, flags=0):
    """Host-built split-K schedule: returns (plan, table) with table an int32
    numpy array; plan.table is None until the caller sets it to the address
    of a device copy of the table."""
    snp = np.ascontiguousarray(np.asarray(seq_new_ptr, dtype=np.int32))
    sc = np.ascontiguousarray(np.asarray(seq_cached, dtype=np.int32))
    vis = np.ascontiguousarray(np.asarray(new_visible, dtype=np.int32))
    if len(sc) != len(snp) - 1:
        raise ValueError("seq_cached must have n_seqs entries")
    plan = kvlink_attend_plan()
    args = (int(dtype), int(n_q_heads), int(n_kv_heads), int(head_dim), len(snp) - 1, _ptr(snp),
            _ptr(sc), _ptr(vis), int(n_compute_units), int(n_workgroups), int(row_block),
            int(flags))
    _check(_lib.kvlink_attend_make_plan(*args, None, 0, ctypes.byref(plan)))
    table = np.zeros(max(plan.table_len, 1), np.int32)
    _check(_lib.kvlink_attend_make_plan(*args, _ptr(table), len(table), ctypes.byref(plan)))
    return plan, table[:plan.table_len]


def kvlink_attend_rope_table(head_dim, rope_theta, n_new_total, d_new_pos, d_table, stream=None):
    _check(_lib.kvlink_attend_rope_table(int(head_dim), float(rope_theta), int(n_new_total),
                                         _ptr(d_new_pos), _ptr(d_table), _stream(stream)))


def kvlink_attend_workspace_bytes(dtype, n_q_heads, n_kv_heads, head_dim, n_new_total, plan):
    return int(_lib.kvlink_attend_workspace_bytes(int(dtype), int(n_q_heads), int(n_kv_heads),
                                                  int(head_dim), int(n_new_total),
                                                  ctypes.byref(plan)))


def kvlink_attend_new_tokens(dtype, n_q_heads, n_kv_heads, head_dim, rope_theta, softmax_scale,
                             n_seqs, n_new_total, max_new, max_cached, d_seq_new_ptr,
                             d_seq_cached, d_new_pos, d_new_visible, q_new, k_new, v_new,
                             k_cache, v_cache, layer, out, lse, plan, workspace,
                             workspace_bytes, stream=None):
    _check(_lib.kvlink_attend_new_tokens(
        int(dtype), int(n_q_heads), int(n_kv_heads), int(head_dim), float(rope_theta),
        float(softmax_scale), int(n_seqs), int(n_new_total), int(max_new), int(max_cached),
        _ptr(d_seq_new_ptr), _ptr(d_seq_cached), _ptr(d_new_pos), _ptr(d_new_visible),
        _ptr(q_new), _ptr(k_new), _ptr(v_new), k_cache, v_cache, int(layer), _ptr(out),
        _ptr(lse), plan, _ptr(workspace), int(workspace_bytes), _stream(stream)))


KVLINK_NOALLOC_SCRATCH_BYTES = 32 << 20   # as include/kvlink.h
KVLINK_FUSED_MAX_SPANS = 48                # as include/kvlink.h


def kvlink_attend_new_tokens_fused(dtype, n_q_heads, n_kv_heads, head_dim, rope_theta,
                                   softmax_scale, n_seqs, n_new_total, max_new, max_cached,
                                   d_seq_new_ptr, d_seq_cached, d_new_pos, d_new_visible, q_new,
                                   k_new, v_new, k_cache, v_cache, layer, out, lse, plan, d_spans,
                                   d_seq_span_ptr, max_spans_per_seq, workspace, workspace_bytes,
                                   stream=None):
    _check(_lib.kvlink_attend_new_tokens_fused(
        int(dtype), int(n_q_heads), int(n_kv_heads), int(head_dim), float(rope_theta),
        float(softmax_scale), int(n_seqs), int(n_new_total), int(max_new), int(max_cached),
        _ptr(d_seq_new_ptr), _ptr(d_seq_cached), _ptr(d_new_pos), _ptr(d_new_visible),
        _ptr(q_new), _ptr(k_new), _ptr(v_new), k_cache, v_cache, int(layer), _ptr(out),
        _ptr(lse), plan, _ptr(d_spans), _ptr(d_seq_span_ptr), int(max_spans_per_seq),
        _ptr(workspace), int(workspace_bytes), _stream(stream)))


def kvlink_attend_new_tokens_noalloc(dtype, n_q_heads, n_kv_heads, head_dim, rope_theta,
                                     softmax_scale, n_seqs, n_new_total, max_new, max_cached,
                                     d_seq_new_ptr, d_seq_cached, d_new_pos, d_new_visible, q_new,
                                     k_new, v_new, k_cache, v_cache, layer, out, lse, plan,
                                     stream=None):
    _check(_lib.kvlink_attend_new_tokens_noalloc(
        int(dtype), int(n_q_heads), int(n_kv_heads), int(head_dim), float(rope_theta),
        float(softmax_scale), int(n_seqs), int(n_new_total), int(max_new), int(max_cached),
        _ptr(d_seq_new_ptr), _ptr(d_seq_cached), _ptr(d_new_pos), _ptr(d_new_visible),
        _ptr(q_new), _ptr(k_new), _ptr(v_new), k_cache, v_cache, int(layer), _ptr(out),
        _ptr(lse), plan, _stream(stream)))


def kvlink_attend_stages(dtype, n_q_heads, n_kv_heads, head_dim, rope_theta, softmax_scale,
                         n_seqs, n_new_total, max_new, max_cached, d_seq_new_ptr, d_seq_cached,
                         d_new_pos, d_new_visible, q_new, k_new, v_new, k_cache, v_cache, layer,
                         out, lse, plan, workspace, workspace_bytes, stream=None,
                         stages=KVLINK_STAGE_ALL):
    _check(_lib.kvlink_attend_stages(
        int(dtype), int(n_q_heads), int(n_kv_heads), int(head_dim), float(rope_theta),
        float(softmax_scale), int(n_seqs), int(n_new_total), int(max_new), int(max_cached),
        _ptr(d_seq_new_ptr), _ptr(d_seq_cached), _ptr(d_new_pos), _ptr(d_new_visible),
        _ptr(q_new), _ptr(k_new), _ptr(v_new), k_cache, v_cache, int(layer), _ptr(out),
        _ptr(lse), plan, _ptr(workspace), int(workspace_bytes), _stream(stream),
        int(stages)))
