"""Device-side request batches for the KVLink hot path.

A batch owns the device buffers of one request batch: the uploaded index maps
from ``kvlink_build_layout``, the destination K/V caches (contiguous or paged)
and the attention workspace.  Running the path is two library calls:
``reencode`` (all layers, one launch) and ``attend`` (one layer).  Everything
here is buffer management and argument marshalling; the work runs in
libkvlink.so.

Storage layouts used here (all elements of the workload dtype, head_dim
innermost):

* contiguous stored caches:  [n_layers][H_kv][R][d], documents back to back;
* contiguous request caches: [n_layers][H_kv][n_seqs][cap][d] with
  cap >= max over requests of (cached rows + new tokens);
* paged caches: [n_layers][n_pages][H_kv][page][d]: one page holds all KV
  heads of `page` consecutive rows; a block table per sequence maps logical
  pages to physical pages.
"""
import numpy as np
import torch

from . import (KVLINK_BF16, KVLINK_F32, KVLINK_PLAN_XCD,
               KVLINK_STAGE_ALL, SPAN_FIELDS, kv_view,
               kvlink_attend_make_plan, kvlink_attend_new_tokens, kvlink_attend_rope_table,
               kvlink_attend_stages, kvlink_group_spans, kvlink_reencode_keys_shared,
               kvlink_attend_new_tokens_fused,
               kvlink_attend_workspace_bytes, kvlink_build_layout,
               kvlink_encode_keys_at_positions, kvlink_load_and_reencode,
               kvlink_load_stage_bytes, kvlink_reencode_keys, kvlink_reencode_keys_mapped)

TORCH_DTYPE = {KVLINK_F32: torch.float32, KVLINK_BF16: torch.bfloat16}

# schedule options used unless a caller names others
DEFAULT_PLAN_FLAGS = KVLINK_PLAN_XCD
# destinations per group of the document-major re-encode: a document reused
# by more spans is read once per group of at most this many, which bounds the
# work of one workgroup (a document serving hundreds of requests would
# otherwise set the launch's duration alone).  Cutting smaller groups costs
# more than it balances: on the 16-request pool (up to 9 uses per document)
# groups of at most 2, 3, 4 or 6 all measured slower than whole documents.
SHARED_MAX_GROUP = 16


def dtype_code(name):
    return {"f32": KVLINK_F32, "bf16": KVLINK_BF16}[name]


def contiguous_view(t, n_kv_heads, n_seqs, cap, d):
    """View of a [L][H][S][cap][d] tensor."""
    return kv_view(t, n_kv_heads * n_seqs * cap * d, n_seqs * cap * d, d, seq_stride=cap * d)


def paged_view(t, n_pages, n_kv_heads, page, d, block_table, max_pages):
    """View of a [L][n_pages][H][page][d] tensor through a block table."""
    return kv_view(t, n_pages * n_kv_heads * page * d, page * d, d, page_stride=n_kv_heads * page * d,
                   block_table=block_table, page_size=page, max_pages=max_pages)


class Batch:
    """Index maps and workspace of one request batch on the device."""

    def __init__(self, dtype, n_layers, n_q_heads, n_kv_heads, head_dim, rope_theta, softmax_scale,
                 seq_doc_ptr, doc_len, link_count, n_query, doc_src_seq=None, doc_src_row=None,
                 doc_src_pos0=None, n_workgroups=0, device="cuda", fused_rope=True, row_block=0,
                 plan_flags=None):
        self.dtype = dtype
        self.torch_dtype = TORCH_DTYPE[dtype]
        self.n_layers, self.n_q_heads, self.n_kv_heads = n_layers, n_q_heads, n_kv_heads
        self.head_dim, self.rope_theta, self.softmax_scale = head_dim, rope_theta, softmax_scale
        self.device = device
        self.seq_doc_ptr = np.asarray(seq_doc_ptr, dtype=np.int32)
        self.layout = kvlink_build_layout(seq_doc_ptr, doc_len, link_count, n_query, doc_src_seq,
                                          doc_src_row, doc_src_pos0)
        t = self.layout["totals"]
        self.n_docs, self.n_new = int(t[0]), int(t[1])
        self.max_doc_len, self.max_cached = int(t[2]), int(t[3])
        self.max_new, self.max_total = int(t[4]), int(t[5])
        self.n_seqs = len(n_query)

        def up(a):
            return torch.from_numpy(np.ascontiguousarray(a)).to(device)
        self.d_spans = up(self.layout["spans"].reshape(-1, SPAN_FIELDS))
        # each request's spans (documents), for the re-encode fused into the
        # attention
        self.d_seq_span_ptr = up(self.seq_doc_ptr)
        self.max_spans_per_seq = int(np.max(np.diff(self.seq_doc_ptr))) if self.n_seqs else 0
        # documents reused within the batch: their stored rows are re-encoded
        # document-major (read once per group of at most SHARED_MAX_GROUP of
        # their spans)
        _, gptr = kvlink_group_spans(self.layout["spans"])
        self.shared_docs = len(gptr) - 1 < self.n_docs
        order, gptr = kvlink_group_spans(self.layout["spans"], SHARED_MAX_GROUP)
        self.n_groups = len(gptr) - 1
        if self.shared_docs:
            self.d_spans_grouped = up(self.layout["spans"].reshape(-1, SPAN_FIELDS)[order])
            self.d_group_ptr = up(gptr)
        self.d_seq_new_ptr = up(self.layout["seq_new_ptr"])
        self.d_seq_cached = up(self.layout["seq_cached"])
        self.d_new_pos = up(self.layout["new_pos"])
        self.d_new_visible = up(self.layout["new_visible"])
        # bf16 batches rotate their new tokens inside the split-attention
        # launch, from a per-batch cos/sin table; fp32 keeps the RoPE launch
        self.rope_table = None
        if fused_rope and dtype == KVLINK_BF16:
            self.rope_table = torch.empty((max(self.n_new, 1), head_dim // 2, 2),
                                          dtype=torch.float32, device=device)
            self.build_rope_table()
        self.set_schedule(n_workgroups, row_block, plan_flags)

    def build_rope_table(self, stream=None):
        """(Re)compute the batch's RoPE table (one launch)."""
        if self.rope_table is not None:
            kvlink_attend_rope_table(self.head_dim, self.rope_theta, self.n_new, self.d_new_pos,
                                     self.rope_table, stream)

    def set_schedule(self, n_workgroups=0, row_block=0, flags=None):
        """Build the split-K schedule (n_workgroups and row_block 0: the
        library's cost model for this device; flags: kvlink_attend_make_plan
        flags, None for DEFAULT_PLAN_FLAGS),
        upload its table and allocate the workspace (zeroed: its merge
        counters must start at zero; every call leaves them zero)."""
        cus = torch.cuda.get_device_properties(torch.device(self.device)).multi_processor_count
        if flags is None:
            flags = DEFAULT_PLAN_FLAGS
        self.plan, table = kvlink_attend_make_plan(self.dtype, self.n_q_heads, self.n_kv_heads,
                                                   self.head_dim, self.layout["seq_new_ptr"],
                                                   self.layout["seq_cached"],
                                                   self.layout["new_visible"], cus, n_workgroups,
                                                   row_block, flags)
        self.plan_table = torch.from_numpy(np.ascontiguousarray(table)).to(self.device)
        self.plan.table = self.plan_table.data_ptr()
        if self.rope_table is not None:
            self.plan.rope_table = self.rope_table.data_ptr()
        self.n_workgroups = self.plan.n_workgroups
        self.ws_bytes = kvlink_attend_workspace_bytes(self.dtype, self.n_q_heads, self.n_kv_heads,
                                                      self.head_dim, self.n_new, self.plan)
        if self.ws_bytes == 0:
            raise ValueError("invalid attention sizes")
        self.workspace = torch.zeros(self.ws_bytes, dtype=torch.uint8, device=self.device)

    def reencode(self, src_view, dst_view, stream=None, shared=None):
        """Re-encode every cached key of the batch, all layers (one launch);
        document-major when some document serves several spans (shared None:
        then; True / False force either form; the document-major form needs
        distinct source and destination buffers)."""
        if shared is None:
            shared = self.shared_docs
        if shared:
            gp = self.d_group_ptr if self.shared_docs else None
            if gp is None:
                order, gptr = kvlink_group_spans(self.layout["spans"], SHARED_MAX_GROUP)
                self.d_spans_grouped = torch.from_numpy(np.ascontiguousarray(
                    self.layout["spans"].reshape(-1, SPAN_FIELDS)[order])).to(self.device)
                self.d_group_ptr = gp = torch.from_numpy(gptr).to(self.device)
            kvlink_reencode_keys_shared(self.dtype, self.n_layers, self.n_kv_heads, self.head_dim,
                                        self.rope_theta, self.n_groups, gp,
                                        self.d_spans_grouped, self.max_doc_len, src_view,
                                        dst_view, stream)
        else:
            kvlink_reencode_keys(self.dtype, self.n_layers, self.n_kv_heads, self.head_dim,
                                 self.rope_theta, self.n_docs, self.d_spans, self.max_doc_len,
                                 src_view, dst_view, stream)

    def encode_at_positions(self, src_view, dst_view, stream=None):
        """Rotate keys stored without RoPE to their global positions, all
        layers (one launch)."""
        kvlink_encode_keys_at_positions(self.dtype, self.n_layers, self.n_kv_heads, self.head_dim,
                                        self.rope_theta, self.n_docs, self.d_spans,
                                        self.max_doc_len, src_view, dst_view, stream)

    def reencode_mapped(self, src_view, dst_view, d_stored_pos, stored_pos_stride, stream=None):
        """Re-encode a compressed cache: every stored row with its own stored
        position (d_stored_pos, device int32, indexed (src_seq, row))."""
        kvlink_reencode_keys_mapped(self.dtype, self.n_layers, self.n_kv_heads, self.head_dim,
                                    self.rope_theta, self.n_docs, self.d_spans, self.max_doc_len,
                                    d_stored_pos, stored_pos_stride, src_view, dst_view, stream)

    def load_stage_bytes(self, stored_rows, n_slots=None):
        """Bytes of a staging area of n_slots layers (default: every layer,
        so the load runs as two large chunks; two slots make every layer a
        chunk, several times slower)."""
        return kvlink_load_stage_bytes(self.dtype, self.n_kv_heads, self.head_dim, stored_rows,
                                       self.n_layers if n_slots is None else n_slots)

    def load_and_reencode(self, h_k, h_v, stored_rows, stage, k_view, v_view, literal=False,
                          copy_stream=None, compute_stream=None):
        """Stored caches in pinned host memory, [n_layers][H_kv][stored_rows][d]:
        with stage None the kernels read them directly (one re-encode and one
        value-gather launch for all layers); with a staging tensor they are
        copied in chunks of consecutive layers (a ring over the layers it
        holds) on copy_stream while compute_stream (torch's current stream
        when None) re-encodes the chunks already copied."""
        kvlink_load_and_reencode(self.dtype, self.n_layers, self.n_kv_heads, self.head_dim,
                                 self.rope_theta, self.n_docs, self.d_spans, self.max_doc_len,
                                 h_k, h_v, stored_rows, stage,
                                 0 if stage is None else stage.numel() * stage.element_size(),
                                 k_view, v_view, int(bool(literal)), copy_stream, compute_stream)

    def attend(self, layer, q_new, k_new, v_new, k_view, v_view, out, lse=None, stream=None,
               stages=KVLINK_STAGE_ALL, workspace=None, fused_reencode=False):
        """RoPE + append of the new tokens and their attention, one layer
        (all stages, or the ones named by the stage mask).  `workspace`
        replaces the batch's own (at least ws_bytes, 256-byte aligned, zeroed
        before its first use).  fused_reencode: k_view's cached rows hold the
        keys as stored, re-encoded inside the split launch (all stages, wide
        bf16 kernel only)."""
        ws = self.workspace if workspace is None else workspace
        if ws.numel() * ws.element_size() < self.ws_bytes:
            raise ValueError("workspace smaller than ws_bytes")
        args = (self.dtype, self.n_q_heads, self.n_kv_heads, self.head_dim, self.rope_theta,
                self.softmax_scale, self.n_seqs, self.n_new, self.max_new, self.max_cached,
                self.d_seq_new_ptr, self.d_seq_cached, self.d_new_pos, self.d_new_visible, q_new,
                k_new, v_new, k_view, v_view, layer, out, lse, self.plan, ws,
                self.ws_bytes, stream)
        if fused_reencode:
            if stages != KVLINK_STAGE_ALL:
                raise ValueError("the fused re-encode runs all stages in one call")
            kvlink_attend_new_tokens_fused(*args[:23], self.d_spans, self.d_seq_span_ptr,
                                           self.max_spans_per_seq, ws, self.ws_bytes, stream)
        elif stages == KVLINK_STAGE_ALL:
            kvlink_attend_new_tokens(*args)
        else:
            kvlink_attend_stages(*args, stages=stages)

    def new_out(self):
        return torch.empty((self.n_new, self.n_q_heads, self.head_dim), dtype=self.torch_dtype,
                           device=self.device)

    def new_lse(self):
        return torch.empty((self.n_new, self.n_q_heads), dtype=torch.float32, device=self.device)
