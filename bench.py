#!/usr/bin/env python3
"""Benchmark of the KVLink hot path on one MI355X.

One step is one pass of the whole path over one request batch: the index maps
of the batch are already on the device; the step re-encodes the cached keys
of every layer (one launch) and then, layer by layer, rotates and appends the
new tokens and runs their attention over the concatenated cache.  Inputs are
resident in HBM before the timed region starts.

Every timed region cycles through enough copies of the caches (at least
512 MB of distinct K and V) that back-to-back steps do not find their data in
the 256 MB last-level cache.

Prints one JSON line.  The metric is microseconds per layer of the path
(re-encode + new-token attention) at the Llama-3.1-8B attention shape, with
the algorithmic HBM GB/s, TFLOP/s and the roofline fraction of the dominant
kernel, and the CPU oracle timed on a bounded sample as a reported baseline.
The headline workload is the 10-document batch; the same line carries the
40-document long-context batch, its decoding step and the shared-pool batch
of 16 requests under "workloads".
"""
import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0            # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2500.0    # MI355X dense bf16
VALU_F32_PEAK_TFLOPS = 157.3
LLC_DEFEAT_BYTES = 512 << 20      # distinct cache bytes a timed region cycles through

METRIC = "µs/layer and HBM GB/s for re-encode+new-token attention at 8B shape; % roofline"
HEADLINE = "llama8b-32layer-10doc"
EXTRAS = ["llama8b-32layer-40x512", "llama8b-decode-40x512", "llama8b-paged-16req"]

CSRC = os.path.join(ROOT, "paper_2502_16002_amd", "csrc")
# sources that decide each kernel's memory traffic (hashed to tell whether
# the committed counter figures still describe the kernel that runs)
KERNEL_SOURCES = {
    "attend_mfma_kernel": ["attend_mfma.hip", "merge_launch.h", "mfma_ops.h", "attend_common.h",
                           "kvlink_internal.h"],
    "attend_decode_kernel": ["attend_decode.hip", "merge_launch.h", "mfma_ops.h", "attend_common.h",
                             "kvlink_internal.h"],
    "reencode_kernel": ["reencode.hip", "kvlink_internal.h"],
    "reencode_shared_kernel": ["reencode.hip", "kvlink_internal.h"],
}
# split-attention kernel by (dtype, the schedule's row block)
SPLIT_KERNEL = {("bf16", 256): "attend_mfma_kernel", ("bf16", 128): "attend_mfma_kernel",
                ("bf16", 64): "attend_mfma_kernel", ("bf16", 16): "attend_decode_kernel",
                ("f32", 16): "attend_valu_kernel"}
# committed counter summaries, one per workload
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_{workload}.md")
PLAN_IN_LAUNCH = 8                # kvlink_attend_make_plan: split units merged in the launch


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=HEADLINE)
    ap.add_argument("--no-extras", action="store_true",
                    help="measure the named workload only (no long-context, decode and pool "
                         "entries)")
    ap.add_argument("--workgroups", type=int, default=0,
                    help="workgroups of the split attention (0: the library's schedule)")
    ap.add_argument("--row-block", type=int, default=0,
                    help="rows per unit of the split attention (0: the library's schedule)")
    ap.add_argument("--plan-flags", type=int, default=None,
                    help="kvlink_attend_make_plan flags (default: the runtime's)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-host-load", action="store_true")
    ap.add_argument("--host-load-only", action="store_true",
                    help="only the host-to-device load of the workload's stored caches "
                         "(copies, direct and staged forms), for a trace")
    ap.add_argument("--kernel-iters", type=int, default=20)
    ap.add_argument("--eager", action="store_true",
                    help="time steps launched from Python instead of a captured HIP graph")
    ap.add_argument("--separate-rope", action="store_true",
                    help="run the new tokens' RoPE as its own launch instead of inside the "
                         "split attention (bf16)")
    return ap.parse_args()


def to_torch(w, x, device):
    import torch
    if w.dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(device)


def copies_for(bytes_per_copy):
    """Cache copies a timed region cycles through: at least two, and enough
    for LLC_DEFEAT_BYTES of distinct data."""
    return max(2, math.ceil(LLC_DEFEAT_BYTES / max(bytes_per_copy, 1)))


class Setup:
    """Device buffers of a single-request workload (documents stored back to
    back, concatenated cache with room for the new tokens), in n_copies
    copies (stored keys, re-encoded keys, values) used in turn."""

    def __init__(self, w, n_workgroups, device="cuda", fused_rope=True, row_block=0, flags=None):
        import torch
        import workloads
        from paper_2502_16002_amd.runtime import Batch, contiguous_view, dtype_code
        self.w = w
        L, H, d = w.n_layers, w.n_kv_heads, w.head_dim
        row0 = workloads.doc_row0(w)
        docs = w.docs[0]
        self.batch = b = Batch(dtype_code(w.dtype), L, w.n_q_heads, H, d, w.rope_theta, w.scale,
                               [0, len(docs)], w.doc_len(0), w.link_count[0], w.n_query,
                               doc_src_row=[int(row0[j]) for j in docs], n_workgroups=n_workgroups,
                               device=device, fused_rope=fused_rope, row_block=row_block,
                               plan_flags=flags)
        R = int(sum(w.doc_table_len))
        self.R = R
        self.cap = cap = b.max_total
        es = 2 if w.dtype == "bf16" else 4
        self.n_copies = copies_for(L * H * (R + 2 * cap) * d * es)
        ksrc = torch.empty((L, H, R, d), dtype=b.torch_dtype, device=device)
        vdst = torch.zeros((L, H, 1, cap, d), dtype=b.torch_dtype, device=device)
        self.q, self.kn, self.vn = [], [], []
        for l in range(L):
            ld = workloads.layer_data(w, l)
            ksrc[l] = to_torch(w, ld.k_store, device)
            kc, vc = workloads.request_cache(w, ld, 0)
            vdst[l, :, 0, :kc.shape[1]] = to_torch(w, vc, device)
            self.q.append(to_torch(w, ld.q_new, device))
            self.kn.append(to_torch(w, ld.k_new, device))
            self.vn.append(to_torch(w, ld.v_new, device))
        self.k_src = [ksrc] + [ksrc.clone() for _ in range(self.n_copies - 1)]
        self.v_dst = [vdst] + [vdst.clone() for _ in range(self.n_copies - 1)]
        self.k_dst = [torch.zeros((L, H, 1, cap, d), dtype=b.torch_dtype, device=device)
                      for _ in range(self.n_copies)]
        self.src_views = [contiguous_view(t, H, 1, R, d) for t in self.k_src]
        self.dst_views = [contiguous_view(t, H, 1, cap, d) for t in self.k_dst]
        self.v_views = [contiguous_view(t, H, 1, cap, d) for t in self.v_dst]
        self.out = b.new_out()
        self.lse = b.new_lse()

    def reencode(self, i=0):
        self.batch.reencode(self.src_views[i], self.dst_views[i])

    def encode_at_positions(self, i=0):
        self.batch.encode_at_positions(self.src_views[i], self.dst_views[i])

    def attend(self, l, i=0, stages=7, workspace=None):
        self.batch.attend(l, self.q[l], self.kn[l], self.vn[l], self.dst_views[i],
                          self.v_views[i], self.out, self.lse, stages=stages, workspace=workspace)

    def time_fused_reencode(self, iters):
        """The re-encode folded into the split attention: each copy's cache
        gets the stored keys at the request's rows (its re-encoded rows
        overwritten), and every layer's attention re-encodes them as its
        tiles are staged.  Microseconds per layer, the attention of every
        layer over every copy captured in one HIP graph, as the separate
        path's attention is timed."""
        import torch
        L, C = self.w.n_layers, self.n_copies
        for i in range(C):
            self.k_dst[i][:, :, 0, :self.R] = self.k_src[i]

        def attend_fused(l, i):
            self.batch.attend(l, self.q[l], self.kn[l], self.vn[l], self.dst_views[i],
                              self.v_views[i], self.out, self.lse, fused_reencode=True)
        g = capture(lambda: [attend_fused(l, i) for i in range(C) for l in range(L)])
        g.replay()
        torch.cuda.synchronize()
        return time_region(lambda i: g.replay(), max(1, iters // C)) / (L * C) * 1000.0

    def step(self, i=0):
        # the batch's RoPE table (one launch; a no-op with the separate RoPE)
        self.batch.build_rope_table()
        # a decoding step attends over a cache re-encoded at prefill
        if not self.w.decode:
            self.reencode(i)
        for l in range(self.w.n_layers):
            self.attend(l, i)

    def time_stages(self, iters):
        """Average duration of one launch of each attention stage.  Every
        layer gets its own workspace, so the RoPE stages of all layers, the
        split attentions of all layers and the combines of all layers, over
        every cache copy, can each be captured as one HIP graph (torch's
        capture records the library's launches; a workload of few layers
        repeats them, so that a replay holds at least 32 launches); each graph
        is replayed `iters` times between two events on the replay stream, so
        the events bracket back-to-back device execution with no host gaps."""
        import torch
        L, C = self.w.n_layers, self.n_copies
        if not hasattr(self, "ws_layers"):
            self.ws_layers = [torch.zeros_like(self.batch.workspace) for _ in range(L)]
        reps = max(1, 32 // (L * C))    # at least 32 launches per replay

        def group(stage):
            return lambda: [self.attend(l, i, stages=stage, workspace=self.ws_layers[l])
                            for _ in range(reps) for i in range(C) for l in range(L)]
        # every layer's partials and outputs exist before the stages run apart
        for l in range(L):
            self.attend(l, workspace=self.ws_layers[l])
        out = {"rope": None}
        # with the fused RoPE the RoPE stage launches nothing
        names = [("split", 2)]
        plan = self.batch.plan
        if plan.n_split_units > 0 and not (plan.flags & PLAN_IN_LAUNCH):
            names.append(("combine", 4))    # else the combine stage launches nothing
        else:
            out["combine"] = 0.0
        if self.batch.rope_table is None:
            names.insert(0, ("rope", 1))
        for name, stage in names:
            g = capture(group(stage))
            g.replay()
            torch.cuda.synchronize()
            s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            s.record()
            for _ in range(iters):
                g.replay()
            e.record()
            torch.cuda.synchronize()
            out[name] = s.elapsed_time(e) / (iters * L * C * reps)
        return out


def capture(fn):
    """fn's launches captured in a HIP graph (after one run on a side stream,
    as torch's capture requires)."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    return g


class PagedSetup(Setup):
    """Device buffers of the shared-pool workload: the stored document caches
    live once in a paged pool (16-token pages, placed by the workload's page
    permutation); every request gets re-encoded K copies in pages of its own
    (shuffled), and reads V straight from the pool pages of its documents
    through its V block table, with fresh pages after them for its new
    tokens.  Pool, per-request keys and values come in n_copies copies."""

    def __init__(self, w, n_workgroups, device="cuda", seed=11, fused_rope=True, row_block=0,
                 flags=None):
        import torch
        import workloads
        from paper_2502_16002_amd.runtime import Batch, dtype_code, paged_view
        self.w = w
        L, H, d, P = w.n_layers, w.n_kv_heads, w.head_dim, w.page_size
        rng = np.random.default_rng(seed)
        doc_pages = [(n + P - 1) // P for n in w.doc_table_len]
        n_pool = sum(doc_pages)
        first = np.concatenate([[0], np.cumsum(doc_pages)[:-1]])
        pool_table = np.zeros((len(doc_pages), max(doc_pages)), np.int32)
        for j, (f, npg) in enumerate(zip(first, doc_pages)):
            pool_table[j, :npg] = w.pool_page_perm[f:f + npg]
        sdp = np.concatenate([[0], np.cumsum([len(x) for x in w.docs])]).astype(np.int32)
        dl = [w.doc_table_len[j] for s in range(w.n_seqs) for j in w.docs[s]]
        lc = [k for s in range(w.n_seqs) for k in w.link_count[s]]
        src_seq = [j for s in range(w.n_seqs) for j in w.docs[s]]
        self.batch = b = Batch(dtype_code(w.dtype), L, w.n_q_heads, H, d, w.rope_theta, w.scale,
                               sdp, dl, lc, w.n_query, doc_src_seq=src_seq,
                               doc_src_row=[0] * len(dl), n_workgroups=n_workgroups,
                               device=device, fused_rope=fused_rope, row_block=row_block,
                               plan_flags=flags)
        td = b.torch_dtype
        max_new_pages = (b.max_new + P - 1) // P
        n_fresh = w.n_seqs * max_new_pages
        seq_cached = b.layout["seq_cached"]
        max_pages = max(int((seq_cached[s] + w.n_new(s) + P - 1) // P) for s in range(w.n_seqs))
        page_bytes = H * P * d * 2
        self.n_copies = copies_for(L * page_bytes * (2 * n_pool + n_fresh + w.n_seqs * max_pages))
        self.pool_table = torch.from_numpy(pool_table).to(device)
        k_pool = torch.zeros((L, n_pool, H, P, d), dtype=td, device=device)
        v_all = torch.zeros((L, n_pool + n_fresh, H, P, d), dtype=td, device=device)
        row0 = workloads.doc_row0(w)
        self.q, self.kn, self.vn = [], [], []
        for l in range(L):
            ld = workloads.layer_data(w, l)
            for j, n in enumerate(w.doc_table_len):
                k = to_torch(w, ld.k_store[:, row0[j]:row0[j] + n], device)
                v = to_torch(w, ld.v_store[:, row0[j]:row0[j] + n], device)
                for pg in range(doc_pages[j]):
                    phys = int(pool_table[j, pg])
                    k_pool[l, phys] = k[:, pg * P:(pg + 1) * P]
                    v_all[l, phys] = v[:, pg * P:(pg + 1) * P]
            self.q.append(to_torch(w, ld.q_new, device))
            self.kn.append(to_torch(w, ld.k_new, device))
            self.vn.append(to_torch(w, ld.v_new, device))
        k_table = rng.permutation(w.n_seqs * max_pages).astype(np.int32).reshape(w.n_seqs, -1)
        v_table = np.zeros((w.n_seqs, max_pages), np.int32)
        for s in range(w.n_seqs):
            pages = [int(pool_table[j, pg]) for j in w.docs[s] for pg in range(doc_pages[j])]
            fresh = n_pool + s * max_new_pages + np.arange(max_pages - len(pages))
            v_table[s] = np.concatenate([pages, fresh]).astype(np.int32)
        self.k_table = torch.from_numpy(k_table).to(device)
        self.v_table = torch.from_numpy(v_table).to(device)
        C = self.n_copies
        self.k_src = [k_pool] + [k_pool.clone() for _ in range(C - 1)]
        self.v_dst = [v_all] + [v_all.clone() for _ in range(C - 1)]
        self.k_dst = [torch.zeros((L, w.n_seqs * max_pages, H, P, d), dtype=td, device=device)
                      for _ in range(C)]
        self.src_views = [paged_view(t, n_pool, H, P, d, self.pool_table, max(doc_pages))
                          for t in self.k_src]
        self.dst_views = [paged_view(t, w.n_seqs * max_pages, H, P, d, self.k_table, max_pages)
                          for t in self.k_dst]
        self.v_views = [paged_view(t, n_pool + n_fresh, H, P, d, self.v_table, max_pages)
                        for t in self.v_dst]
        self.out = b.new_out()
        self.lse = b.new_lse()


def host_load(st, iters=3):
    """The stored caches in pinned host memory, loaded to the device with the
    keys re-encoded (the first steps of the time-to-first-token path): the
    plain copies alone, the kernels reading host memory directly, and the
    staged copies through a ring of slots with the re-encodes on a second
    stream (two slots, and one slot per layer), or on the copy stream itself.
    Milliseconds per load of all layers."""
    import torch
    b, w = st.batch, st.w
    h_k = st.k_src[0].cpu().pin_memory()
    h_v = st.k_src[1].cpu().pin_memory()       # any stored-shape data serves as values
    R = h_k.shape[2]
    stage2 = torch.empty(b.load_stage_bytes(R, 2), dtype=torch.uint8, device="cuda")
    stage_all = torch.empty(b.load_stage_bytes(R, w.n_layers), dtype=torch.uint8, device="cuda")
    k_dst = torch.empty_like(st.k_dst[0])
    v_dst = torch.empty_like(st.v_dst[0])
    from paper_2502_16002_amd.runtime import contiguous_view
    H, d = w.n_kv_heads, w.head_dim
    kv_k = contiguous_view(k_dst, H, 1, st.cap, d)
    kv_v = contiguous_view(v_dst, H, 1, st.cap, d)
    dev_k = torch.empty_like(st.k_src[0])
    dev_v = torch.empty_like(st.k_src[0])
    copy = torch.cuda.Stream()
    cur = torch.cuda.current_stream()

    def timed(fn):
        torch.cuda.synchronize()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        copy.wait_stream(cur)
        for _ in range(iters):
            fn()
        cur.wait_stream(copy)
        e.record()
        torch.cuda.synchronize()
        return s.elapsed_time(e) / iters

    def copies():
        with torch.cuda.stream(copy):
            dev_k.copy_(h_k, non_blocking=True)
            dev_v.copy_(h_v, non_blocking=True)
    direct = lambda: b.load_and_reencode(h_k, h_v, R, None, kv_k, kv_v, compute_stream=cur)
    ring2 = lambda: b.load_and_reencode(h_k, h_v, R, stage2, kv_k, kv_v, copy_stream=copy,
                                        compute_stream=cur)
    ring_all = lambda: b.load_and_reencode(h_k, h_v, R, stage_all, kv_k, kv_v, copy_stream=copy,
                                           compute_stream=cur)
    serial = lambda: b.load_and_reencode(h_k, h_v, R, stage2, kv_k, kv_v, copy_stream=cur,
                                         compute_stream=cur)
    for fn in (direct, ring2, ring_all, serial):
        fn()
    copy_ms, dir_ms = timed(copies), timed(direct)
    r2_ms, rall_ms, ser_ms = timed(ring2), timed(ring_all), timed(serial)
    nbytes = 2 * h_k.numel() * h_k.element_size()
    return {"bytes": nbytes, "copy_only_ms": round(copy_ms, 3),
            "copy_gbps": round(nbytes / (copy_ms * 1e-3) / 1e9, 1),
            "load_reencode_direct_ms": round(dir_ms, 3),
            "direct_gbps": round(nbytes / (dir_ms * 1e-3) / 1e9, 1),
            "load_reencode_staged_two_streams_2_slots_ms": round(r2_ms, 3),
            f"load_reencode_staged_two_streams_{w.n_layers}_slots_ms": round(rall_ms, 3),
            "load_reencode_staged_one_stream_ms": round(ser_ms, 3)}


def device_copy_gbps(nbytes=1 << 30, iters=10):
    """A plain device-to-device copy of nbytes (larger than the 256 MB last
    level cache), read + written bytes per second: the practical HBM ceiling
    on this machine, as a sanity anchor for the nominal 8 TB/s."""
    import torch
    src = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(iters):
        dst.copy_(src)
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / iters
    del src, dst
    return round(2 * nbytes / (ms * 1e-3) / 1e9, 1)


def algorithmic(w, batch):
    """Bytes and flops the method itself moves (per the closed forms)."""
    es = 2 if w.dtype == "bf16" else 4
    Tc = int(batch.layout["seq_cached"].astype(np.int64).sum())
    n_new = batch.n_new
    H, Hq, d = w.n_kv_heads, w.n_q_heads, w.head_dim
    # re-encode: every destination row written, every stored row read once
    # (a document reused by several spans is read once for all of them)
    from paper_2502_16002_amd import kvlink_group_spans
    spans = batch.layout["spans"]
    order, gptr = kvlink_group_spans(spans)
    stored_rows = int(sum(int(spans[order[gptr[g]], 4]) for g in range(len(gptr) - 1)))
    re_bytes = w.n_layers * H * (Tc + stored_rows) * d * es
    pairs = int((batch.layout["new_pos"].astype(np.int64) + 1).sum())
    at_bytes = (2 * H * Tc * d + n_new * (Hq + 2 * H) * d + n_new * Hq * d) * es
    at_flops = 4 * d * Hq * pairs
    return dict(reencode_bytes=re_bytes, attend_bytes=at_bytes, attend_flops=at_flops,
                pairs_per_qhead=pairs, cached_tokens=Tc, new_tokens=n_new)


def source_hash(kernel):
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel, workload):
    """HBM bytes per launch from the committed counter summary: rows
    `| kernel | workload | source hash | fetch bytes | write bytes |`.  None when
    there is no row for this kernel and workload, or the kernel's sources
    changed since the counters were taken."""
    path = TRAFFIC_FILE.format(workload=workload)
    if kernel not in KERNEL_SOURCES or not os.path.exists(path):
        return None
    want = source_hash(kernel)
    for line in open(path):
        cells = [c.strip().strip("`") for c in line.strip().strip("|").split("|")]
        if len(cells) == 5 and cells[0] == kernel and cells[1] == workload and cells[2] == want:
            return int(cells[3]) + int(cells[4])
    return None


def time_region(fn, iters):
    """Average device time of fn over iters calls, between two events on the
    current stream."""
    import torch
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for i in range(iters):
        fn(i)
    e.record()
    torch.cuda.synchronize()
    return s.elapsed_time(e) / iters


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo)."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or platform.machine()


def cpu_baseline(w, alg, budget_s=15.0):
    """The oracle, untouched, on the same workload: per request, the
    re-encode of every document and the attention of every new token and
    head; whole layers (single-request workloads) or whole requests (the
    pool batch), in order, until about budget_s seconds have run, scaled to
    microseconds per layer of the whole batch."""
    import oracle
    import workloads
    f = lambda x: workloads.as_f64(w, x)
    total, done = 0.0, 0
    units = [(l, s) for l in range(w.n_layers) for s in range(w.n_seqs)]
    for l, s in units:
        ld = workloads.layer_data(w, l)
        kc, vc = workloads.request_cache(w, ld, s)
        q, kn, vn = workloads.request_new(w, ld, s)
        kc, vc, q, kn, vn = f(kc), f(vc), f(q), f(kn), f(vn)
        t0 = time.perf_counter()
        r0, g = 0, 0
        for j, L in enumerate([] if w.decode else w.doc_len(s)):
            oracle.reencode(kc[:, r0:r0 + L], g, w.rope_theta)
            r0 += L
            g += L + w.link_count[s][j]
        oracle.attend(w.doc_len(s), w.link_count[s], w.n_query[s], q, kn, vn, kc, vc,
                      w.rope_theta, w.scale)
        total += time.perf_counter() - t0
        done += 1
        if total >= budget_s:
            break
    per_layer = total / done * w.n_seqs
    what = (f"{done} of {w.n_layers} layers" if w.n_seqs == 1 else
            f"{done} of {w.n_seqs} requests of layer 0, scaled to all {w.n_seqs}")
    return {"value": round(per_layer * 1e6, 1), "unit": "us/layer",
            "cores": oracle.num_threads(), "kind": "oracle",
            "sample": f"{what} in full (" + ("" if w.decode else "re-encode of every document + ")
                      + "attention of every new token and head), "
                      f"{total:.1f} s of oracle time",
            "cpu": cpu_model()}


def measure(w, args, headline):
    """Everything the bench line reports for one workload."""
    import torch
    st = (PagedSetup if w.pool else Setup)(w, args.workgroups, fused_rope=not args.separate_rope,
                                           row_block=args.row_block, flags=args.plan_flags)
    b = st.batch
    alg = algorithmic(w, b)
    C = st.n_copies
    print(f"# setup done: {w.name} cached={alg['cached_tokens']} new={alg['new_tokens']} "
          f"workgroups={b.n_workgroups} segments={b.plan.n_segments} row_block={b.plan.row_block} "
          f"copies={C}", file=sys.stderr, flush=True)

    for _ in range(args.warmup):
        st.step(0)
    torch.cuda.synchronize()
    # the last layer's output of a step, to check that every later replay
    # reproduces it bit for bit (the schedule's merge order is fixed)
    first_out = st.out.clone()
    # steps over the cache copies in turn
    ms_step_eager = time_region(lambda i: st.step(i % C), args.steps)
    # the same steps captured once in a HIP graph (torch's capture records
    # the library's launches on the capture stream) and replayed: the device
    # work is identical, without the host's per-launch cost
    graph = capture(lambda: [st.step(i) for i in range(C)])
    for _ in range(max(1, args.warmup // C)):
        graph.replay()
    torch.cuda.synchronize()
    reps = max(1, args.steps // C)
    ms_step_graph = time_region(lambda i: graph.replay(), reps) / C
    ms_step = ms_step_eager if args.eager else ms_step_graph
    torch.cuda.synchronize()
    assert torch.equal(st.out.view(torch.int16), first_out.view(torch.int16)), \
        "a replayed step changed the output"

    # isolated kernels, each group captured in a HIP graph and replayed on
    # torch's current stream (the stream the library launches on): the
    # re-encode and the literal form over the cache copies in turn, the
    # attention of every layer in one call each, and each attention stage
    # over all layers
    it = args.kernel_iters
    L = w.n_layers
    n_re = max(16, C)
    re_ms = lit_ms = None
    if not w.decode:
        g_re = capture(lambda: [st.reencode(i % C) for i in range(n_re)])
        g_re.replay()
        re_ms = time_region(lambda i: g_re.replay(), max(1, it // 4)) / n_re
        if not w.pool:
            g_lit = capture(lambda: [st.encode_at_positions(i % C) for i in range(n_re)])
            g_lit.replay()
            lit_ms = time_region(lambda i: g_lit.replay(), max(1, it // 4)) / n_re
    g_at = capture(lambda: [st.attend(l, i) for i in range(C) for l in range(L)])
    g_at.replay()
    at_ms = time_region(lambda i: g_at.replay(), max(1, it // C)) / (L * C)
    stage_ms = st.time_stages(max(1, it // 4))

    us_layer = ms_step * 1000.0 / L
    step_bytes = (0 if w.decode else alg["reencode_bytes"]) + L * alg["attend_bytes"]
    step_flops = L * alg["attend_flops"]
    peak_flops = MFMA_BF16_PEAK_TFLOPS if w.dtype == "bf16" else VALU_F32_PEAK_TFLOPS
    ai = alg["attend_flops"] / alg["attend_bytes"]
    at_bound = "mfma" if ai > peak_flops * 1e12 / (HBM_PEAK_GBPS * 1e9) else "hbm"

    re_roof = None
    if re_ms is not None:
        re_gbps = alg["reencode_bytes"] / (re_ms * 1e-3) / 1e9
        # document-major when the batch reuses a document (the library's choice)
        re_kernel = "reencode_shared_kernel" if b.shared_docs else "reencode_kernel"
        re_roof = {"kernel": re_kernel, "bound": "hbm", "achieved": round(re_gbps, 1),
                   "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                   "frac": round(re_gbps / HBM_PEAK_GBPS, 4),
                   "traffic": measured_traffic(re_kernel, w.name),
                   "us_per_launch": round(re_ms * 1000, 2),
                   "bytes_per_launch": alg["reencode_bytes"]}

    # the attention of a layer: the split kernel, plus the combine launch
    # when the schedule merges split units there (its duration is then part
    # of the attention's)
    split_kernel = SPLIT_KERNEL[(w.dtype, b.plan.row_block)]   # the library's own choice
    combine_runs = b.plan.n_split_units > 0 and not (b.plan.flags & PLAN_IN_LAUNCH)
    att_ms = stage_ms["split"] + (stage_ms["combine"] if combine_runs else 0.0)
    gbps = alg["attend_bytes"] / (att_ms * 1e-3) / 1e9
    tflops = alg["attend_flops"] / (att_ms * 1e-3) / 1e12
    at_kernel = split_kernel + (" + combine_kernel" if combine_runs else "")
    if at_bound == "hbm":
        at_roof = {"kernel": at_kernel, "bound": "hbm", "achieved": round(gbps, 1),
                   "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": round(gbps / HBM_PEAK_GBPS, 4)}
    else:
        at_roof = {"kernel": at_kernel, "bound": "mfma", "achieved": round(tflops, 2),
                   "peak": peak_flops, "unit": "TFLOP/s", "frac": round(tflops / peak_flops, 4)}
    split_gbps = alg["attend_bytes"] / (stage_ms["split"] * 1e-3) / 1e9
    split_tflops = alg["attend_flops"] / (stage_ms["split"] * 1e-3) / 1e12
    at_roof.update({
        "traffic": None if combine_runs else measured_traffic(split_kernel, w.name),
        "us_per_launch": round(att_ms * 1000, 2),
        "split_only_us": round(stage_ms["split"] * 1000, 2),
        "split_only_frac": round(split_gbps / HBM_PEAK_GBPS if at_bound == "hbm"
                                 else split_tflops / peak_flops, 4),
        "split_traffic": measured_traffic(split_kernel, w.name),
        "bytes_per_launch": alg["attend_bytes"], "flops_per_launch": alg["attend_flops"],
        "hbm_gbps": round(gbps, 1), "tflops": round(tflops, 2),
        "hbm_frac": round(gbps / HBM_PEAK_GBPS, 4), "mfma_frac": round(tflops / peak_flops, 4)})
    fused = b.rope_table is not None
    stages = {"rope": "inside the split attention" if fused else "own launch",
              "rope_new_us": None if fused else round(stage_ms["rope"] * 1000, 2),
              "split_attention_us": round(stage_ms["split"] * 1000, 2),
              "combine_us": round(stage_ms["combine"] * 1000, 2) if combine_runs else 0.0,
              "merge": "combine launch" if combine_runs else
                       ("inside the split launch" if b.plan.n_split_units else "none needed"),
              "all_stages_one_call_us": round(at_ms * 1000, 2),
              "reencode_us_per_layer": None if re_ms is None else round(re_ms * 1000 / L, 2)}
    dominant_attend = re_ms is None or L * att_ms > re_ms
    config = {"workload": w.name, "launch": "eager" if args.eager else "hip_graph",
              "requests": w.n_seqs, "n_layers": L, "n_q_heads": w.n_q_heads,
              "n_kv_heads": w.n_kv_heads, "head_dim": w.head_dim, "rope_theta": w.rope_theta,
              "documents": sum(len(x) for x in w.docs),
              "link_tokens_per_doc": max(max(x) if x else 0 for x in w.link_count),
              "query_tokens": int(sum(w.n_query)), "cached_tokens": alg["cached_tokens"],
              "new_tokens": alg["new_tokens"], "attention_workgroups": b.n_workgroups,
              "attention_segments": b.plan.n_segments,
              "attention_row_block": b.plan.row_block,
              "attention_plan_flags": b.plan.flags,
              "cache_copies_cycled": C,
              "step": "decode: attention only" if w.decode else "re-encode + attention"}
    res = {
        "value": round(us_layer, 3),
        "ms_per_step": round(ms_step, 4),
        "config": config,
        "hbm_gbps": round(step_bytes / (ms_step * 1e-3) / 1e9, 1),
        "tflops": round(step_flops / (ms_step * 1e-3) / 1e12, 3),
        "roofline": at_roof if dominant_attend else re_roof,
        "roofline_other": re_roof if dominant_attend else at_roof,
        "per_layer_kernels": stages,
        "us_per_layer_eager_launch": round(ms_step_eager * 1000.0 / L, 3),
        "us_per_layer_graph_launch": round(ms_step_graph * 1000.0 / L, 3),
    }
    if lit_ms is not None:
        res["literal_encode"] = {
            "us_per_launch": round(lit_ms * 1000, 2),
            "gbps": round(alg["reencode_bytes"] / (lit_ms * 1e-3) / 1e9, 1),
            "frac": round(alg["reencode_bytes"] / (lit_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4)}
    # the re-encode folded into the attention (wide bf16 kernel), against the
    # separate re-encode plus attention, per layer
    from paper_2502_16002_amd import KVLINK_FUSED_MAX_SPANS
    if (not w.pool and not w.decode and w.dtype == "bf16" and b.plan.row_block in (256, 128, 64)
            and b.max_spans_per_seq <= KVLINK_FUSED_MAX_SPANS):
        fused_us = st.time_fused_reencode(it)
        sep_us = re_ms * 1000 / L + at_ms * 1000
        res["fused_reencode"] = {
            "us_per_layer_fused_attention": round(fused_us, 2),
            "us_per_layer_separate": round(sep_us, 2),
            "separate_parts": "re-encode per layer + attention (all stages, one call)",
            "selected": "fused" if fused_us < sep_us else "separate"}
    if headline and not w.pool and not w.decode and not args.no_host_load:
        res["host_load"] = host_load(st)
    if not args.no_cpu_baseline and (headline or w.pool):
        res["cpu_baseline"] = cpu_baseline(w, alg)
    del st, graph, g_at
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the path is single-GPU; see the sharding notes)", file=sys.stderr)
        sys.exit(2)
    import torch
    import workloads
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    w = workloads.get(args.workload)
    if args.host_load_only:
        st = Setup(w, args.workgroups)
        print(json.dumps({"workload": w.name, "host_load": host_load(st)}), flush=True)
        return
    head = measure(w, args, headline=True)
    res = {
        "metric": METRIC,
        "value": head["value"],
        "unit": "us/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded, Llama-shaped caches; no weights or datasets)",
    }
    res.update({k: v for k, v in head.items() if k not in ("value", "ms_per_step")})
    res["device_copy_gbps"] = device_copy_gbps()
    if not args.no_extras and args.workload == HEADLINE:
        res["workloads"] = {}
        for name in EXTRAS:
            r = measure(workloads.get(name), args, headline=False)
            res["workloads"][name] = r
            print(f"# {name}: {r['value']} us/layer", file=sys.stderr, flush=True)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
