"""Seeded synthetic inputs shaped like the KVLink workloads (arXiv 2502.16002).

This module only draws random numbers and arranges them; it holds none of the
method's arithmetic (no rotation, no masking, no softmax).  Both the oracle
side (tests) and the GPU side (tests, benchmark) take their inputs from here.

The paper measures on public QA datasets and real Llama weights that are not
available here; these seeded tensors stand in for them, with the shapes of the
paper's setups: Llama-3.2-1B / Llama-3.1-8B attention shapes (Sec. 3.1), ten
retrieved documents of a few hundred tokens (Sec. 3.3), and K link tokens per
document (KVLink5, Sec. 3.1).

Recipe (all draws from numpy PCG64):
  * layout randomness (document lengths, query length, document picks) comes
    from ``default_rng([seed, 0])``;
  * the tensors of layer l come from ``default_rng([seed, 1, l])``, drawn in
    the fixed order k_cached, v_cached, q_new, k_new, v_new;
  * f32 workloads draw every tensor from N(0, 1);
  * bf16 workloads draw cached and new keys and values from N(0, 1)/sqrt(d)
    and queries from N(0, 1), then round to bfloat16 (round to nearest even);
  * cached keys are taken as already carrying RoPE at their local positions
    0..L-1 (a rotated Gaussian vector is again Gaussian).
"""
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

# ---------------------------------------------------------------- bfloat16 bits


def f32_to_bf16_bits(x):
    """Round float32 values to bfloat16 (nearest even); return the uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    u = u + (((u >> 16) & 1) + np.uint32(0x7FFF))
    return (u >> 16).astype(np.uint16)


def bf16_bits_to_f32(b):
    """Exact widening of bfloat16 bits to float32."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# ------------------------------------------------------------------- workloads


@dataclass
class Workload:
    """Shape and layout of one synthetic workload.

    A request holds ``docs[s]`` (indices into the document table, in retrieval
    order), ``link_count[s]`` (K link tokens after each of those documents)
    and ``n_query[s]`` query tokens.  ``doc_table_len[j]`` is the length of
    stored document j.  With ``pool`` set, the stored documents form one shared
    pool (paged with ``page_size``-token pages) that requests pick from;
    otherwise each request stores its own documents back to back.
    """
    name: str
    dtype: str                      # "f32" or "bf16"
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    rope_theta: float
    seed: int
    doc_table_len: List[int]
    docs: List[List[int]]
    link_count: List[List[int]]
    n_query: List[int]
    pool: bool = False
    page_size: int = 0
    pool_page_perm: Optional[np.ndarray] = None
    description: str = ""
    decode: bool = False            # a decoding step: the cache is already re-encoded
    extra: dict = field(default_factory=dict)

    @property
    def n_seqs(self):
        return len(self.docs)

    def doc_len(self, s):
        return [self.doc_table_len[j] for j in self.docs[s]]

    def cached_rows(self, s):
        return sum(self.doc_len(s))

    def n_new(self, s):
        return sum(self.link_count[s]) + self.n_query[s]

    def total_positions(self, s):
        return self.cached_rows(s) + self.n_new(s)

    @property
    def scale(self):
        return 1.0 / float(np.sqrt(self.head_dim))


def _make(name, dtype, n_layers, hq, hkv, d, theta, seed, lens, links, nq, desc, decode=False):
    return Workload(name=name, dtype=dtype, n_layers=n_layers, n_q_heads=hq, n_kv_heads=hkv,
                    head_dim=d, rope_theta=theta, seed=seed,
                    doc_table_len=list(lens), docs=[list(range(len(lens)))],
                    link_count=[[links] * len(lens)], n_query=[nq], description=desc,
                    decode=decode)


def tiny_f32(seed=2502):
    """3 documents of 32 tokens, 2 link tokens each, 16 query tokens: 118
    positions; 4 query heads over 2 KV heads, head_dim 64, theta 1e4, fp32."""
    return _make("tiny-f32-3x32", "f32", 1, 4, 2, 64, 1e4, seed, [32] * 3, 2, 16,
                 "tiny fp32 case, 1 layer")


def llama1b_layer(seed=2503):
    """Llama-3.2-1B attention shape (32/8 heads, head_dim 64, theta 5e5), one
    layer, 10 documents of U{150..250} tokens, 5 link tokens each, 64 queries."""
    rng = np.random.default_rng([seed, 0])
    lens = rng.integers(150, 250, size=10, endpoint=True).tolist()
    return _make("llama1b-1layer-10doc", "bf16", 1, 32, 8, 64, 5e5, seed, lens, 5, 64,
                 "Llama-3.2-1B shape, 1 layer, 10 docs of 150-250 tokens")


def llama8b_10doc(seed=2504, n_layers=32):
    """Llama-3.1-8B attention shape (32/8 heads, head_dim 128, theta 5e5), 32
    layers, 10 documents of U{100..300} tokens, 5 link tokens each, 64 queries."""
    rng = np.random.default_rng([seed, 0])
    lens = rng.integers(100, 300, size=10, endpoint=True).tolist()
    return _make("llama8b-32layer-10doc", "bf16", n_layers, 32, 8, 128, 5e5, seed, lens, 5,
                 64, "Llama-3.1-8B shape, 32 layers, 10 docs of 100-300 tokens")


def llama8b_long(seed=2505, n_layers=32):
    """Llama-3.1-8B attention shape, 32 layers, 40 documents of 512 tokens,
    5 link tokens each, 128 queries (20,480 cached tokens, 20,808 positions)."""
    return _make("llama8b-32layer-40x512", "bf16", n_layers, 32, 8, 128, 5e5, seed,
                 [512] * 40, 5, 128, "Llama-3.1-8B shape, 32 layers, 40 docs of 512 tokens")


def llama8b_paged(seed=2506, n_layers=1):
    """Llama-3.1-8B attention shape; a pool of 64 stored documents of 256
    tokens in 16-token pages; 16 requests, each picking 20 distinct documents
    in random order (documents repeat across requests), 5 link tokens each and
    U{32..128} query tokens."""
    rng = np.random.default_rng([seed, 0])
    n_pool, pool_len, page = 64, 256, 16
    docs = [rng.choice(n_pool, size=20, replace=False).tolist() for _ in range(16)]
    nq = rng.integers(32, 128, size=16, endpoint=True).tolist()
    n_pages = n_pool * pool_len // page
    perm = rng.permutation(n_pages).astype(np.int32)   # physical page of logical pool page
    return Workload(name="llama8b-paged-16req", dtype="bf16", n_layers=n_layers,
                    n_q_heads=32, n_kv_heads=8, head_dim=128, rope_theta=5e5, seed=seed,
                    doc_table_len=[pool_len] * n_pool, docs=docs,
                    link_count=[[5] * 20 for _ in range(16)], n_query=nq, pool=True,
                    page_size=page, pool_page_perm=perm,
                    description="Llama-3.1-8B shape, shared 64x256-token paged pool, 16 requests")


def llama8b_long_decode(seed=2505, n_layers=32):
    """One decoding step after the long-context prefill: the 40 x 512-token
    cache of the long workload (already re-encoded) and a single new query
    token per layer, 4 GQA rows per KV head."""
    return _make("llama8b-decode-40x512", "bf16", n_layers, 32, 8, 128, 5e5, seed,
                 [512] * 40, 0, 1, "Llama-3.1-8B shape, decode step over 40 docs of 512 tokens",
                 decode=True)


def llama8b_paged_decode(seed=2506, n_layers=1):
    """One decoding step of the 16 shared-pool requests: each request's 20
    documents read through its page tables and one new query token."""
    w = llama8b_paged(seed, n_layers)
    w.name = "llama8b-paged-decode-16req"
    w.link_count = [[0] * len(d) for d in w.docs]
    w.n_query = [1] * w.n_seqs
    w.decode = True
    w.description = "Llama-3.1-8B shape, decode step of 16 requests over the shared paged pool"
    return w


WORKLOADS = {
    "tiny-f32-3x32": tiny_f32,
    "llama1b-1layer-10doc": llama1b_layer,
    "llama8b-32layer-10doc": llama8b_10doc,
    "llama8b-32layer-40x512": llama8b_long,
    "llama8b-paged-16req": llama8b_paged,
    "llama8b-decode-40x512": llama8b_long_decode,
    "llama8b-paged-decode-16req": llama8b_paged_decode,
}


def get(name, **kw):
    return WORKLOADS[name](**kw)


def custom(doc_len, link_count, n_query, n_q_heads=4, n_kv_heads=2, head_dim=64,
           rope_theta=1e4, dtype="f32", seed=7, n_layers=1, name="custom"):
    """A single-request workload with explicit lengths (edge cases, small tests)."""
    lc = link_count if isinstance(link_count, (list, tuple)) else [link_count] * len(doc_len)
    return Workload(name=name, dtype=dtype, n_layers=n_layers, n_q_heads=n_q_heads,
                    n_kv_heads=n_kv_heads, head_dim=head_dim, rope_theta=rope_theta, seed=seed,
                    doc_table_len=list(doc_len), docs=[list(range(len(doc_len)))],
                    link_count=[list(lc)], n_query=[n_query])


# ------------------------------------------------------------------- tensors


def _draw(rng, shape, std, dtype):
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    if dtype == "bf16":
        return f32_to_bf16_bits(x)
    return x


@dataclass
class LayerData:
    """Tensors of one layer.  bf16 workloads hold uint16 bit patterns, f32
    workloads hold float32.  Shapes:

    * k_store, v_store: [H_kv, R, d], the stored document caches; R is the sum
      of the table's document lengths, document j at rows doc_row0[j]..
    * q_new: [N, H_q, d]; k_new, v_new: [N, H_kv, d], new tokens of every
      request back to back (request s at rows new_row0[s]..), in increasing
      global position within each request, keys and queries before RoPE.
    """
    k_store: np.ndarray
    v_store: np.ndarray
    q_new: np.ndarray
    k_new: np.ndarray
    v_new: np.ndarray


def doc_row0(w: Workload):
    return np.concatenate([[0], np.cumsum(w.doc_table_len)[:-1]]).astype(np.int64) \
        if w.doc_table_len else np.zeros(0, np.int64)


def new_row0(w: Workload):
    n = [w.n_new(s) for s in range(w.n_seqs)]
    return np.concatenate([[0], np.cumsum(n)]).astype(np.int64)


def layer_data(w: Workload, layer: int) -> LayerData:
    rng = np.random.default_rng([w.seed, 1, layer])
    d, hkv, hq = w.head_dim, w.n_kv_heads, w.n_q_heads
    R = int(sum(w.doc_table_len))
    N = int(new_row0(w)[-1])
    kv_std = 1.0 if w.dtype == "f32" else 1.0 / np.sqrt(d)
    k_store = _draw(rng, (hkv, R, d), kv_std, w.dtype)
    v_store = _draw(rng, (hkv, R, d), kv_std, w.dtype)
    q_new = _draw(rng, (N, hq, d), 1.0, w.dtype)
    k_new = _draw(rng, (N, hkv, d), kv_std, w.dtype)
    v_new = _draw(rng, (N, hkv, d), kv_std, w.dtype)
    return LayerData(k_store, v_store, q_new, k_new, v_new)


def as_f64(w: Workload, x):
    """Exact widening of a workload tensor to float64."""
    if w.dtype == "bf16":
        return bf16_bits_to_f32(x).astype(np.float64)
    return np.asarray(x, dtype=np.float64)


def request_cache(w: Workload, ld: LayerData, s: int):
    """Stored caches of request s's documents back to back in retrieval order,
    [H_kv, T_c, d] each (a gather of stored rows; no arithmetic)."""
    r0 = doc_row0(w)
    rows = np.concatenate([np.arange(r0[j], r0[j] + w.doc_table_len[j]) for j in w.docs[s]]) \
        if w.docs[s] else np.zeros(0, np.int64)
    return ld.k_store[:, rows, :], ld.v_store[:, rows, :]


def request_new(w: Workload, ld: LayerData, s: int):
    n0 = new_row0(w)
    sl = slice(int(n0[s]), int(n0[s + 1]))
    return ld.q_new[sl], ld.k_new[sl], ld.v_new[sl]
