"""Test helpers: move a synthetic workload onto the device, run the library's
path on it, and compare against the oracle.

Comparison bars (from the tolerances of the workloads):
  * fp32: max |gpu - oracle| <= 1e-5 per element;
  * bf16: per output row (a key vector, or one token and head of the
    attention output), max |gpu - oracle| <= 2e-2 * max |oracle row|.
    The re-encode is also held to a bf16 rounding bar: every element within
    2^-8 |oracle| + 1e-6 * max |oracle row| (half an ulp plus float noise).
  * index maps: bit-exact.
"""
import numpy as np

import workloads

F32_ATOL = 1e-5
BF16_ROW_REL = 2e-2


def to_torch(w, x, device="cuda"):
    import torch
    if w.dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(device)


def to_f64(t):
    import torch
    return t.detach().to(torch.float64).cpu().numpy()


def check_close(w, got, ref, what=""):
    """Apply the workload's bar; rows are the last axis.  Returns the worst
    metric (abs error for f32, row-relative error for bf16)."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), what + ": non-finite output"
    if w.dtype == "f32":
        err = float(np.max(np.abs(got - ref))) if got.size else 0.0
        assert err <= F32_ATOL, f"{what}: max abs err {err:.3e} > {F32_ATOL}"
        return err
    rowmax = np.maximum(np.max(np.abs(ref), axis=-1), 1e-30)
    rel = np.max(np.abs(got - ref), axis=-1) / rowmax
    worst = float(np.max(rel)) if rel.size else 0.0
    assert worst <= BF16_ROW_REL, f"{what}: row-relative err {worst:.3e} > {BF16_ROW_REL}"
    return worst


def check_bf16_rounding(got, ref, what=""):
    """Every element within half a bf16 ulp of the exact value, plus noise."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    rowmax = np.max(np.abs(ref), axis=-1, keepdims=True)
    bound = 2.0 ** -8 * np.abs(ref) + 1e-6 * rowmax
    bad = np.abs(got - ref) > bound
    assert not bad.any(), f"{what}: {int(bad.sum())} elements beyond half an ulp"


# ------------------------------------------------------------- contiguous


class ContiguousRun:
    """A single-request workload whose stored caches are the request's
    documents back to back (the tiny, 1B and 8B workloads)."""

    def __init__(self, w, layers, n_workgroups=0, device="cuda", fused_rope=True, row_block=0,
                 plan_flags=None):
        import torch
        from paper_2502_16002_amd.runtime import Batch, contiguous_view, dtype_code
        assert w.n_seqs == 1 and not w.pool
        self.w, self.layers = w, layers
        L, H, d = w.n_layers, w.n_kv_heads, w.head_dim
        self.lds = [workloads.layer_data(w, l) for l in range(L)]
        row0 = workloads.doc_row0(w)
        docs = w.docs[0]
        self.batch = Batch(dtype_code(w.dtype), L, w.n_q_heads, H, d, w.rope_theta, w.scale,
                           [0, len(docs)], w.doc_len(0), w.link_count[0], w.n_query,
                           doc_src_row=[int(row0[j]) for j in docs], n_workgroups=n_workgroups,
                           device=device, fused_rope=fused_rope, row_block=row_block,
                           plan_flags=plan_flags)
        b = self.batch
        R = int(sum(w.doc_table_len))
        self.cap = max(b.max_total, 1)
        self.R = R
        self.k_src = to_torch(w, np.stack([ld.k_store for ld in self.lds]), device)   # [L][H][R][d]
        self.k_dst = torch.zeros((L, H, 1, self.cap, d), dtype=b.torch_dtype, device=device)
        self.v_dst = torch.zeros((L, H, 1, self.cap, d), dtype=b.torch_dtype, device=device)
        kc_rows = []
        for l, ld in enumerate(self.lds):
            kc, vc = workloads.request_cache(w, ld, 0)
            self.v_dst[l, :, 0, :kc.shape[1]] = to_torch(w, vc, device)
            kc_rows.append(kc)
        self.src_view = contiguous_view(self.k_src, H, 1, R, d)
        self.k_view = contiguous_view(self.k_dst, H, 1, self.cap, d)
        self.v_view = contiguous_view(self.v_dst, H, 1, self.cap, d)
        self.q = [to_torch(w, ld.q_new, device) for ld in self.lds]
        self.kn = [to_torch(w, ld.k_new, device) for ld in self.lds]
        self.vn = [to_torch(w, ld.v_new, device) for ld in self.lds]
        self.out = {l: b.new_out() for l in layers}
        self.lse = {l: b.new_lse() for l in layers}

    def run(self):
        import torch
        self.batch.reencode(self.src_view, self.k_view)
        for l in self.layers:
            self.batch.attend(l, self.q[l], self.kn[l], self.vn[l], self.k_view, self.v_view,
                              self.out[l], self.lse[l])
        torch.cuda.synchronize()

    # oracle-side inputs of one layer (float64)
    def oracle_inputs(self, l):
        w, ld = self.w, self.lds[l]
        kc, vc = workloads.request_cache(w, ld, 0)
        q, kn, vn = workloads.request_new(w, ld, 0)
        f = lambda x: workloads.as_f64(w, x)
        return f(kc), f(vc), f(q), f(kn), f(vn)


# ------------------------------------------------------------------- paged


class PagedRun:
    """The shared-pool workload: stored document caches live once in a paged
    pool (pages placed by the workload's permutation); every request gets
    re-encoded K copies in its own pages, and reads V straight from the pool
    pages of its documents through its V block table (values are never
    rewritten), with fresh pages after them for its new tokens."""

    def __init__(self, w, n_workgroups=0, device="cuda", seed=11, fused_rope=True, row_block=0,
                 plan_flags=None):
        import torch
        from paper_2502_16002_amd.runtime import Batch, dtype_code, paged_view
        assert w.pool
        self.w = w
        L, H, d, P = w.n_layers, w.n_kv_heads, w.head_dim, w.page_size
        rng = np.random.default_rng(seed)
        self.lds = [workloads.layer_data(w, l) for l in range(L)]
        doc_pages = [(n + P - 1) // P for n in w.doc_table_len]
        assert all(n % P == 0 for n in w.doc_table_len)
        n_pool_pages = sum(doc_pages)
        perm = w.pool_page_perm
        first = np.concatenate([[0], np.cumsum(doc_pages)[:-1]])
        max_doc_pages = max(doc_pages)
        pool_table = np.zeros((len(w.doc_table_len), max_doc_pages), np.int32)
        for j, (f, npg) in enumerate(zip(first, doc_pages)):
            pool_table[j, :npg] = perm[f:f + npg]
        self.pool_table = torch.from_numpy(pool_table).to(device)

        sdp = np.concatenate([[0], np.cumsum([len(x) for x in w.docs])]).astype(np.int32)
        dl = [w.doc_table_len[j] for s in range(w.n_seqs) for j in w.docs[s]]
        lc = [k for s in range(w.n_seqs) for k in w.link_count[s]]
        src_seq = [j for s in range(w.n_seqs) for j in w.docs[s]]
        self.batch = Batch(dtype_code(w.dtype), L, w.n_q_heads, H, d, w.rope_theta, w.scale,
                           sdp, dl, lc, w.n_query, doc_src_seq=src_seq,
                           doc_src_row=[0] * len(dl), n_workgroups=n_workgroups, device=device,
                           fused_rope=fused_rope, row_block=row_block, plan_flags=plan_flags)
        b = self.batch
        td = b.torch_dtype
        # pool tensors [L][page][H][P][d]; V gets extra fresh pages for new tokens
        max_new_pages = (b.max_new + P - 1) // P
        n_fresh = w.n_seqs * max_new_pages
        self.k_pool = torch.zeros((L, n_pool_pages, H, P, d), dtype=td, device=device)
        self.v_all = torch.zeros((L, n_pool_pages + n_fresh, H, P, d), dtype=td, device=device)
        row0 = workloads.doc_row0(w)
        for l, ld in enumerate(self.lds):
            for j, n in enumerate(w.doc_table_len):
                k = to_torch(w, ld.k_store[:, row0[j]:row0[j] + n], device)   # [H][n][d]
                v = to_torch(w, ld.v_store[:, row0[j]:row0[j] + n], device)
                for pg in range(doc_pages[j]):
                    phys = int(pool_table[j, pg])
                    self.k_pool[l, phys] = k[:, pg * P:(pg + 1) * P]
                    self.v_all[l, phys] = v[:, pg * P:(pg + 1) * P]
        # per-request K pages (shuffled) and V tables (pool pages, then fresh)
        seq_cached = b.layout["seq_cached"]
        self.max_pages = max(int((seq_cached[s] + w.n_new(s) + P - 1) // P) for s in range(w.n_seqs))
        k_table = rng.permutation(w.n_seqs * self.max_pages).astype(np.int32).reshape(w.n_seqs, -1)
        v_table = np.zeros((w.n_seqs, self.max_pages), np.int32)
        for s in range(w.n_seqs):
            pages = [int(pool_table[j, pg]) for j in w.docs[s] for pg in range(doc_pages[j])]
            assert len(pages) * P == seq_cached[s]
            fresh = n_pool_pages + s * max_new_pages + np.arange(self.max_pages - len(pages))
            v_table[s] = np.concatenate([pages, fresh]).astype(np.int32)
        self.k_table_np, self.v_table_np = k_table, v_table
        self.k_table = torch.from_numpy(k_table).to(device)
        self.v_table = torch.from_numpy(v_table).to(device)
        self.k_dst = torch.zeros((L, w.n_seqs * self.max_pages, H, P, d), dtype=td, device=device)
        self.src_view = paged_view(self.k_pool, n_pool_pages, H, P, d, self.pool_table, max_doc_pages)
        self.k_view = paged_view(self.k_dst, w.n_seqs * self.max_pages, H, P, d, self.k_table,
                                 self.max_pages)
        self.v_view = paged_view(self.v_all, n_pool_pages + n_fresh, H, P, d, self.v_table,
                                 self.max_pages)
        self.q = [to_torch(w, ld.q_new, device) for ld in self.lds]
        self.kn = [to_torch(w, ld.k_new, device) for ld in self.lds]
        self.vn = [to_torch(w, ld.v_new, device) for ld in self.lds]
        self.out = [b.new_out() for _ in range(L)]
        self.lse = [b.new_lse() for _ in range(L)]

    def run(self):
        import torch
        self.batch.reencode(self.src_view, self.k_view)
        for l in range(self.w.n_layers):
            self.batch.attend(l, self.q[l], self.kn[l], self.vn[l], self.k_view, self.v_view,
                              self.out[l], self.lse[l])
        torch.cuda.synchronize()

    def request_rows(self, table, s, rows):
        """(page, slot) of logical rows of request s under a block table."""
        P = self.w.page_size
        rows = np.asarray(rows)
        return table[s, rows // P], rows % P

    def oracle_inputs(self, l, s):
        w, ld = self.w, self.lds[l]
        kc, vc = workloads.request_cache(w, ld, s)
        q, kn, vn = workloads.request_new(w, ld, s)
        f = lambda x: workloads.as_f64(w, x)
        return f(kc), f(vc), f(q), f(kn), f(vn)
