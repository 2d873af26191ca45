"""CPU tests of the C-ABI library: it loads, exports every declared symbol,
rejects bad arguments before any HIP call, and its host layout maps equal the
ones derived from the oracle's sequence layout, bit for bit."""
import ctypes
import os
import re

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle
import workloads
from conftest import ROOT

HEADER = os.path.join(ROOT, "include", "kvlink.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kvlink_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def kv():
    import paper_2502_16002_amd as kv
    return kv


def test_library_exports_every_declared_symbol(kv):
    names = _declared_functions()
    assert {"kvlink_build_layout", "kvlink_reencode_keys", "kvlink_attend_new_tokens",
            "kvlink_attend_workspace_bytes", "kvlink_last_error"} <= set(names)
    lib = ctypes.CDLL(kv.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
        assert hasattr(kv, n), "binding lacks " + n
    assert kv.kvlink_version().startswith("kvlink")


def _kernel_metadata(so_path):
    """(name, private segment bytes, spilled VGPRs) of every gfx950 kernel in
    the library: its offload bundles (one per source file) unbundled and their
    AMDGPU metadata notes read with the ROCm LLVM tools."""
    import shutil
    import subprocess
    import tempfile
    import yaml
    llvm = "/opt/rocm/llvm/bin"
    tools = [os.path.join(llvm, t) for t in ("llvm-objcopy", "clang-offload-bundler", "llvm-readobj")]
    if not all(os.path.exists(t) for t in tools):
        pytest.skip("ROCm LLVM tools not found")
    out = []
    with tempfile.TemporaryDirectory() as d:
        fat = os.path.join(d, "fatbin")
        subprocess.run([tools[0], "--dump-section", ".hip_fatbin=" + fat, so_path], check=True)
        data = open(fat, "rb").read()
        magic = b"__CLANG_OFFLOAD_BUNDLE__"
        starts = [m.start() for m in re.finditer(re.escape(magic), data)] + [len(data)]
        for k in range(len(starts) - 1):
            b, co = os.path.join(d, f"b{k}"), os.path.join(d, f"c{k}")
            open(b, "wb").write(data[starts[k]:starts[k + 1]])
            subprocess.run([tools[1], "--unbundle", "--type=o",
                            "--targets=hipv4-amdgcn-amd-amdhsa--gfx950", "--input=" + b,
                            "--output=" + co], check=True)
            notes = subprocess.run([tools[2], "--notes", co], check=True, capture_output=True,
                                   text=True).stdout
            if "amdhsa.kernels:" not in notes:
                continue
            text = notes[notes.index("amdhsa.kernels:"):]
            text = text[:text.index("\n...")] if "\n..." in text else text
            for kern in yaml.safe_load(text)["amdhsa.kernels"]:
                out.append((kern[".name"], kern[".private_segment_fixed_size"],
                            kern[".vgpr_spill_count"]))
    return out


def test_hot_path_kernels_use_no_scratch(kv):
    """A kernel with a private (scratch) segment pays for it at every launch
    (a 64-byte stack array cost the split attention 5 to 17 us per layer), so
    every kernel the default path launches stays free of one.  Exempt: the
    fused re-encode's instances and the 128-row units, which the schedule
    does not pick by default."""
    kernels = _kernel_metadata(kv.LIB_PATH)
    assert len(kernels) > 50
    names = [n for n, _, _ in kernels]
    for k in ["reencode_kernel", "reencode_shared_kernel", "attend_mfma_kernel",
              "attend_decode_kernel", "combine_kernel", "rope_table_kernel"]:
        assert any(k in n for n in names), k

    def exempt(n):
        return "attend_mfma_kernel" in n and (re.search(r"ShapeILi\dELi\dEEELb1E", n) is not None
                                              or "ShapeILi2ELi2E" in n)

    bad = [(n, p) for n, p, _ in kernels if p > 0 and not exempt(n)]
    assert not bad, bad


def test_struct_sizes_match_header(kv):
    assert ctypes.sizeof(kv.kvlink_span) == 24
    assert ctypes.sizeof(kv.kvlink_kv_view) == 64
    assert ctypes.sizeof(kv.kvlink_attend_plan) == 48


# --------------------------------------------------------------- layout maps


def _oracle_maps(doc_len, link_count, n_query):
    """Index maps derived from the oracle's per-position layout and map."""
    kind, seg, idx = oracle.layout(doc_len, link_count, n_query)
    is_doc = kind == oracle.KIND_DOC
    newp = np.nonzero(~is_doc)[0]
    doc_cum = np.cumsum(is_doc)
    if len(kind) <= 600:
        mask = oracle.full_mask(kind, seg)
        visible = np.array([int(mask[a][is_doc].sum()) for a in newp], np.int64)
    else:  # new rows see every position at or before their own (pinned on small cases)
        visible = doc_cum[newp]
    g = np.array([int(np.argmax(is_doc & (seg == i))) for i in range(len(doc_len))], np.int64)
    return dict(doc_pos0=g, new_pos=newp, new_visible=visible, new_doc=seg[newp],
                new_slot=idx[newp], seq_cached=int(is_doc.sum()), T=len(kind))


CASES = [
    ([32, 32, 32], [2, 2, 2], 16),
    ([2, 2, 1], [1, 1, 1], 1),             # Fig. 2
    ([5], [0], 7),                          # K = 0
    ([1, 1, 1, 1], [3, 0, 2, 1], 0),        # ragged, no queries
    ([], [], 9),                            # no documents
    ([512] * 40, [5] * 40, 128),            # long context
]


@pytest.mark.parametrize("doc_len,link_count,n_query", CASES)
def test_layout_bit_exact_vs_oracle(kv, doc_len, link_count, n_query):
    L = kv.kvlink_build_layout([0, len(doc_len)], doc_len, link_count, [n_query])
    o = _oracle_maps(doc_len, link_count, n_query)
    assert np.array_equal(L["doc_pos0"], o["doc_pos0"])
    assert np.array_equal(L["new_pos"], o["new_pos"])
    assert np.array_equal(L["new_visible"], o["new_visible"])
    assert np.array_equal(L["new_doc"], o["new_doc"])
    assert np.array_equal(L["new_slot"], o["new_slot"])
    assert L["seq_cached"].tolist() == [o["seq_cached"]]
    assert L["seq_new_ptr"].tolist() == [0, len(o["new_pos"])]
    t = L["totals"]
    assert t[0] == len(doc_len) and t[1] == len(o["new_pos"]) and t[5] == o["T"]
    # re-encode spans: delta = g_i (stored at 0), rows back to back
    sp = L["spans"]
    rows = np.concatenate([[0], np.cumsum(doc_len)[:-1]]) if doc_len else np.zeros(0)
    assert np.array_equal(sp[:, 5], o["doc_pos0"])
    assert np.array_equal(sp[:, 3], rows) and np.array_equal(sp[:, 1], rows)
    assert np.array_equal(sp[:, 4], doc_len)


def test_layout_paged_batch_vs_oracle(kv):
    w = workloads.llama8b_paged()
    sdp = np.concatenate([[0], np.cumsum([len(d) for d in w.docs])])
    dl = [w.doc_table_len[j] for s in range(w.n_seqs) for j in w.docs[s]]
    lc = [k for s in range(w.n_seqs) for k in w.link_count[s]]
    src_seq = [j for s in range(w.n_seqs) for j in w.docs[s]]
    L = kv.kvlink_build_layout(sdp, dl, lc, w.n_query, doc_src_seq=src_seq,
                               doc_src_row=[0] * len(dl), doc_src_pos0=[3] * len(dl))
    for s in range(w.n_seqs):
        o = _oracle_maps(w.doc_len(s), w.link_count[s], w.n_query[s])
        a, b = L["seq_new_ptr"][s], L["seq_new_ptr"][s + 1]
        assert np.array_equal(L["new_pos"][a:b], o["new_pos"])
        assert np.array_equal(L["new_visible"][a:b], o["new_visible"])
        d0, d1 = sdp[s], sdp[s + 1]
        assert np.array_equal(L["doc_pos0"][d0:d1], o["doc_pos0"])
        assert np.array_equal(L["spans"][d0:d1, 5], o["doc_pos0"] - 3)
        assert np.array_equal(L["spans"][d0:d1, 0], w.docs[s])
        assert np.all(L["spans"][d0:d1, 2] == s)
        assert L["seq_cached"][s] == o["seq_cached"]


def test_layout_link_ids_follow_document_index(kv):
    """Appendix A.2: the link tokens of the n-th document are link_n-1..link_n-K."""
    L = kv.kvlink_build_layout([0, 3], [4, 4, 4], [2, 2, 2], [1])
    assert L["new_doc"].tolist() == [0, 0, 1, 1, 2, 2, -1]
    assert L["new_slot"].tolist() == [0, 1, 0, 1, 0, 1, 0]


@pytest.mark.parametrize("args,status", [
    (([0, 2], [3, 0], [1, 1], [2]), 3),        # empty document
    (([0, 2], [3, 3], [1, -1], [2]), 3),       # negative link count
    (([0, 1], [3], [1], [-2]), 3),             # negative query count
    (([1, 1], [3], [1], [2]), 3),              # seq_doc_ptr[0] != 0
    (([0, 2, 1], [3, 3], [1, 1], [2, 2]), 3),  # decreasing seq_doc_ptr
])
def test_layout_rejects_invalid(kv, args, status):
    with pytest.raises(kv.KVLinkError) as e:
        kv.kvlink_build_layout(*args)
    assert e.value.status == status


# ------------------------------------------------- validation before any HIP


def _view(kv, base=4096, **kw):
    return kv.kvlink_kv_view(base, kw.get("ls", 1024), kw.get("hs", 256), kw.get("rs", 64),
                             kw.get("ss", 0), kw.get("ps", 0), kw.get("bt", None),
                             kw.get("pg", 0), kw.get("mp", 0))


@pytest.mark.parametrize("change,status", [
    (dict(head_dim=96), 2),
    (dict(dtype=7), 2),
    (dict(n_layers=0), 1),
    (dict(theta=0.0), 1),
    (dict(theta=float("nan")), 1),
    (dict(src_base=0), 1),
    (dict(src_base=4100), 1),              # not 16-byte aligned
    (dict(rs=65), 1),                      # stride not a multiple of 16 bytes
    (dict(spans=None), 1),
])
@pytest.mark.parametrize("fn", ["kvlink_reencode_keys", "kvlink_encode_keys_at_positions"])
def test_reencode_validation(kv, change, status, fn):
    a = dict(dtype=kv.KVLINK_BF16, n_layers=2, n_kv_heads=2, head_dim=64, theta=1e4, n_spans=1,
             spans=8192, max_len=4, src_base=4096, rs=64)
    a.update(change)
    src = _view(kv, a["src_base"], rs=a["rs"])
    dst = _view(kv, 8192)
    with pytest.raises(kv.KVLinkError) as e:
        getattr(kv, fn)(a["dtype"], a["n_layers"], a["n_kv_heads"], a["head_dim"], a["theta"],
                        a["n_spans"], a["spans"], a["max_len"], src, dst, stream=0)
    assert e.value.status == status


@pytest.mark.parametrize("fn", ["kvlink_reencode_keys", "kvlink_encode_keys_at_positions"])
def test_reencode_empty_is_a_no_op(kv, fn):
    getattr(kv, fn)(kv.KVLINK_BF16, 1, 1, 64, 1e4, 0, None, 0, _view(kv), _view(kv), stream=0)


@pytest.mark.parametrize("pos,stride", [(None, 0), (8192, -1)])
def test_reencode_mapped_validation(kv, pos, stride):
    with pytest.raises(kv.KVLinkError) as e:
        kv.kvlink_reencode_keys_mapped(kv.KVLINK_BF16, 2, 2, 64, 1e4, 1, 8192, 4, pos, stride,
                                       _view(kv), _view(kv, 8192), stream=0)
    assert e.value.status == 1


@pytest.mark.parametrize("change,status", [
    (dict(head_dim=96), 2),
    (dict(dtype=7), 2),
    (dict(n_layers=0), 1),
    (dict(n_groups=-1), 1),
    (dict(theta=0.0), 1),
    (dict(gptr=None), 1),
    (dict(spans=None), 1),
    (dict(src_base=8192), 1),          # src and dst are one buffer
    (dict(src_base=0), 1),
    (dict(rs=63), 1),
])
def test_reencode_shared_validation(kv, change, status):
    a = dict(dtype=kv.KVLINK_BF16, n_layers=2, n_kv_heads=2, head_dim=64, theta=1e4, n_groups=1,
             gptr=12288, spans=8192, max_len=4, src_base=4096, rs=64)
    a.update(change)
    src = _view(kv, a["src_base"], rs=a["rs"])
    dst = _view(kv, 8192)
    with pytest.raises(kv.KVLinkError) as e:
        kv.kvlink_reencode_keys_shared(a["dtype"], a["n_layers"], a["n_kv_heads"], a["head_dim"],
                                       a["theta"], a["n_groups"], a["gptr"], a["spans"],
                                       a["max_len"], src, dst, stream=0)
    assert e.value.status == status


def test_reencode_shared_empty_is_a_no_op(kv):
    kv.kvlink_reencode_keys_shared(kv.KVLINK_BF16, 2, 2, 64, 1e4, 0, None, None, 4, _view(kv),
                                   _view(kv, 8192), stream=0)


def test_group_spans(kv):
    """Spans reading the same stored rows (same source sequence, row and
    length) form one group, each group in span order; every span appears
    once."""
    rng = np.random.default_rng(5)
    for n in [0, 1, 7, 200]:
        src = rng.integers(0, 4, size=(n, 3))     # few distinct sources
        spans = np.zeros((n, 6), np.int32)
        spans[:, 0] = src[:, 0] % 2
        spans[:, 1] = src[:, 1] * 100
        spans[:, 4] = 1 + src[:, 2] % 2
        spans[:, 2] = np.arange(n)
        spans[:, 3] = rng.integers(0, 1000, size=n)
        spans[:, 5] = rng.integers(0, 5000, size=n)
        order, gptr = kv.kvlink_group_spans(spans)
        assert sorted(order.tolist()) == list(range(n))
        assert gptr[0] == 0 and gptr[-1] == n and np.all(np.diff(gptr) >= 1)
        keys = [tuple(spans[i, [0, 1, 4]]) for i in order]
        for g in range(len(gptr) - 1):
            grp = order[gptr[g]:gptr[g + 1]]
            assert len({keys[i] for i in range(gptr[g], gptr[g + 1])}) == 1
            assert list(grp) == sorted(grp)
            if g:
                assert keys[gptr[g]] > keys[gptr[g] - 1]
        assert len(gptr) - 1 == len({tuple(r) for r in spans[:, [0, 1, 4]]})


def test_group_spans_max_group(kv):
    """With max_group > 0 a run of n spans reading the same rows is cut into
    ceil(n / max_group) consecutive groups of near-equal size, in the same
    order as the uncut grouping; max_group < 0 is refused."""
    rng = np.random.default_rng(6)
    n = 300
    spans = np.zeros((n, 6), np.int32)
    spans[:, 0] = rng.integers(0, 7, size=n)
    spans[:, 4] = 16
    spans[:, 2] = np.arange(n)
    full_order, full_ptr = kv.kvlink_group_spans(spans)
    for mg in [1, 2, 3, 4, 10, 1000]:
        order, gptr = kv.kvlink_group_spans(spans, max_group=mg)
        assert np.array_equal(order, full_order)
        assert set(full_ptr.tolist()) <= set(gptr.tolist())
        for g in range(len(full_ptr) - 1):
            a, b = full_ptr[g], full_ptr[g + 1]
            cuts = [c for c in gptr.tolist() if a <= c <= b]
            sizes = np.diff(cuts)
            assert len(sizes) == -(-(b - a) // mg)
            assert sizes.max() <= mg and sizes.max() - sizes.min() <= 1
    with pytest.raises(kv.KVLinkError):
        kv.kvlink_group_spans(spans, max_group=-1)


def test_load_stage_bytes(kv):
    assert kv.kvlink_load_stage_bytes(kv.KVLINK_BF16, 8, 128, 1000) == 4 * 8 * 1000 * 128 * 2
    assert kv.kvlink_load_stage_bytes(kv.KVLINK_F32, 2, 64, 10) == 4 * 2 * 10 * 64 * 4
    assert kv.kvlink_load_stage_bytes(kv.KVLINK_BF16, 8, 128, 1000, 6) == 12 * 8 * 1000 * 128 * 2
    assert kv.kvlink_load_stage_bytes(kv.KVLINK_BF16, 8, 128, 0) == 0
    assert kv.kvlink_load_stage_bytes(kv.KVLINK_BF16, 8, 128, 1000, 1) == 0


@pytest.mark.parametrize("change,status", [
    (dict(h_k=None), 1),
    (dict(stored_rows=0), 1),
    (dict(literal=2), 1),
    (dict(head_dim=96), 2),
    (dict(h_k=4096 + 8), 1),                # not 16-byte aligned
    (dict(stage=4096 + 16), 4),             # not 256-byte aligned
    (dict(stage_bytes=1024), 4),
    (dict(spans=None), 1),
])
def test_load_and_reencode_validation(kv, change, status):
    a = dict(dtype=kv.KVLINK_BF16, head_dim=64, h_k=4096, h_v=4096, stored_rows=8, literal=0,
             stage=8192, stage_bytes=1 << 20, spans=8192)
    a.update(change)
    with pytest.raises(kv.KVLinkError) as e:
        kv.kvlink_load_and_reencode(a["dtype"], 2, 2, a["head_dim"], 1e4, 1, a["spans"], 4,
                                    a["h_k"], a["h_v"], a["stored_rows"], a["stage"],
                                    a["stage_bytes"], _view(kv), _view(kv), a["literal"],
                                    copy_stream=0, compute_stream=0)
    assert e.value.status == status


def _plan(kv, dtype=None, hq=8, hkv=2, d=128, snp=(0, 10), vis=(100,) * 10, n_wg=0):
    dtype = kv.KVLINK_BF16 if dtype is None else dtype
    tc = [max(vis)] * (len(snp) - 1)
    plan, _ = kv.kvlink_attend_make_plan(dtype, hq, hkv, d, list(snp), tc, list(vis), 256, n_wg)
    plan.table = 4096          # a fake, aligned device address: nothing is launched
    return plan


def _attend_args(kv, **change):
    a = dict(dtype=kv.KVLINK_BF16, hq=8, hkv=2, d=128, theta=5e5, scale=0.088, n_seqs=1,
             n_new=10, max_new=10, max_cached=100, snp=16, sc=16, pos=16, vis=16, q=4096,
             k=4096, v=4096, kview=_view(kv), vview=_view(kv), layer=0, out=4096, lse=None,
             plan=None, ws=1 << 20, ws_bytes=1 << 30)
    a.update(change)
    if a["plan"] is None:
        a["plan"] = _plan(kv)
    return a


def _call_attend(kv, a, stages=None):
    args = (a["dtype"], a["hq"], a["hkv"], a["d"], a["theta"], a["scale"], a["n_seqs"],
            a["n_new"], a["max_new"], a["max_cached"], a["snp"], a["sc"], a["pos"], a["vis"],
            a["q"], a["k"], a["v"], a["kview"], a["vview"], a["layer"], a["out"], a["lse"],
            a["plan"], a["ws"], a["ws_bytes"])
    if stages is None:
        kv.kvlink_attend_new_tokens(*args, stream=0)
    else:
        kv.kvlink_attend_stages(*args, stream=0, stages=stages)


def _bad_plan(kv, **fields):
    p = _plan(kv)
    for k, v in fields.items():
        setattr(p, k, v)
    return p


@pytest.mark.parametrize("change,status", [
    (dict(d=80), 2),
    (dict(hq=6, hkv=4), 1),                # not a multiple
    (dict(hq=48, hkv=3), 2),               # group 16
    (dict(n_seqs=0), 1),
    (dict(max_new=0), 1),
    (dict(max_new=11), 1),
    (dict(theta=-1.0), 1),
    (dict(scale=float("inf")), 1),
    (dict(scale=0.0), 1),
    (dict(scale=-0.1), 1),
    (dict(snp=None), 1),
    (dict(q=None), 1),
    (dict(out=None), 1),
    (dict(ws=None), 4),
    (dict(ws=1000), 4),                    # misaligned
    (dict(ws_bytes=16), 4),
    (dict(layer=-1), 1),
    (dict(q=4100), 1),                     # misaligned new-token inputs
    (dict(v=4104), 1),
    ("table", 1),                          # plan without a device table
    ("rope_misaligned", 1),
    ("table_misaligned", 1),
    ("row_block", 1),                      # plan of the other path
    ("n_seqs", 1),
    ("table_len", 1),
    ("other_dtype", 1),                    # bf16 (matrix-core) plan for an fp32 call
])
def test_attend_validation(kv, change, status):
    if isinstance(change, str):
        plan = {"table": lambda: _bad_plan(kv, table=None),
                "table_misaligned": lambda: _bad_plan(kv, table=4100),
                "rope_misaligned": lambda: _bad_plan(kv, rope_table=4100),
                "row_block": lambda: _bad_plan(kv, row_block=16),
                "n_seqs": lambda: _bad_plan(kv, n_seqs=2),
                "table_len": lambda: _bad_plan(kv, table_len=3),
                "other_dtype": lambda: _plan(kv)}[change]()
        change = dict(plan=plan, dtype=kv.KVLINK_F32) if change == "other_dtype" else dict(plan=plan)
    with pytest.raises(kv.KVLinkError) as e:
        _call_attend(kv, _attend_args(kv, **change))
    assert e.value.status == status
    assert kv.kvlink_last_error()


@pytest.mark.parametrize("args,status", [
    ((80, 5e5, 4, 4096, 4096), 2),          # head_dim
    ((128, 0.0, 4, 4096, 4096), 1),         # theta
    ((128, float("nan"), 4, 4096, 4096), 1),
    ((128, 5e5, -1, 4096, 4096), 1),
    ((128, 5e5, 4, None, 4096), 1),
    ((128, 5e5, 4, 4096, None), 1),
    ((128, 5e5, 4, 4096, 4100), 1),         # misaligned table
])
def test_rope_table_validation(kv, args, status):
    with pytest.raises(kv.KVLinkError) as e:
        kv.kvlink_attend_rope_table(*args, stream=0)
    assert e.value.status == status


def test_rope_table_empty_is_a_no_op(kv):
    kv.kvlink_attend_rope_table(128, 5e5, 0, None, None, stream=0)


@pytest.mark.parametrize("stages", [0, 8, 15])
def test_attend_stages_rejects_bad_masks(kv, stages):
    with pytest.raises(kv.KVLinkError) as e:
        _call_attend(kv, _attend_args(kv), stages=stages)
    assert e.value.status == 1


def test_attend_no_new_tokens_is_a_no_op(kv):
    _call_attend(kv, _attend_args(kv, n_new=0, max_new=0))


def test_workspace_bytes(kv):
    f = kv.kvlink_attend_workspace_bytes
    bf, f32 = kv.KVLINK_BF16, kv.KVLINK_F32
    counters = 64 * 1024                      # the merge counters come first
    one = _plan(kv, n_wg=1)                   # one segment per unit: no partials
    assert one.n_segments == one.n_units
    assert f(bf, 8, 2, 128, 10, one) == counters + _align(10 * 8 * 128 * 2)
    assert f(bf, 8, 2, 96, 10, one) == 0
    many = _plan(kv, n_wg=1 << 20)            # one tile per segment
    assert many.n_segments > many.n_units
    rb = many.row_block
    assert f(bf, 8, 2, 128, 10, many) == (counters + _align(10 * 8 * 128 * 2) +
                                           _align(many.n_segments * rb * 128 * 2) +
                                           _align(many.n_segments * rb * 2 * 4))
    thin = _plan(kv, f32, 4, 2, 64, (0, 22), [200] * 22, n_wg=12)
    assert thin.row_block == 16 and thin.n_segments > thin.n_units
    assert f(f32, 4, 2, 64, 22, thin) > f(f32, 4, 2, 64, 22, _plan(kv, f32, 4, 2, 64, (0, 22),
                                                                     [200] * 22, n_wg=1))


def _align(x):
    return (x + 255) // 256 * 256


REC = 16   # int32 fields of a segment record


def _decode(plan, table, n_seqs):
    """Split a schedule table into its sections (layout in include/kvlink.h)."""
    t = np.asarray(table)
    n_seg, n_u, n_sp = plan.n_segments, plan.n_units, plan.n_split_units
    recs = t[:REC * n_seg].reshape(n_seg, REC)
    o = REC * n_seg
    unit_recs = t[o:o + 8 * n_u].reshape(n_u, 8)
    split = t[o + 8 * n_u:o + 8 * n_u + n_sp]
    assert len(t) == o + 8 * n_u + n_sp == plan.table_len
    return recs, unit_recs, split


def _expected_units(L, G, hkv, rb):
    """(s, h, rho0, rows, n0, T_c, cmax, nvirt, tiles) of every unit, from
    the layout and the attention map of Sec. 2.3: the block's last token sees
    new_visible cached rows and the new rows up to its own."""
    snp, vis, sc = L["seq_new_ptr"], L["new_visible"], L["seq_cached"]
    out, seq_unit = [], []
    for s in range(len(snp) - 1):
        seq_unit.append(len(out))
        n0 = int(snp[s])
        rows_s = int(snp[s + 1] - snp[s]) * G
        for h in range(hkv):
            for rho0 in range(0, rows_s, rb):
                rows = min(rb, rows_s - rho0)
                r_last = (rho0 + rows - 1) // G
                cmax = int(vis[n0 + r_last])
                nvirt = cmax + r_last + 1
                out.append((s, h, rho0, rows, n0, int(sc[s]), cmax, nvirt, -(-nvirt // 64)))
    seq_unit.append(len(out))
    return np.array(out, np.int64).reshape(-1, 9), np.array(seq_unit)


def _check_schedule(kv, w, n_wg_req, row_block=0, flags=0):
    sdp = np.concatenate([[0], np.cumsum([len(d) for d in w.docs])])
    dl = [w.doc_table_len[j] for s in range(w.n_seqs) for j in w.docs[s]]
    lc = [k for s in range(w.n_seqs) for k in w.link_count[s]]
    L = kv.kvlink_build_layout(sdp, dl, lc, w.n_query)
    dt = kv.KVLINK_F32 if w.dtype == "f32" else kv.KVLINK_BF16
    plan, table = kv.kvlink_attend_make_plan(dt, w.n_q_heads, w.n_kv_heads, w.head_dim,
                                             L["seq_new_ptr"], L["seq_cached"], L["new_visible"],
                                             256, n_wg_req, row_block, flags)
    G = w.n_q_heads // w.n_kv_heads
    max_new = int(np.max(np.diff(L["seq_new_ptr"])))
    mfma = w.dtype == "bf16" and max_new * G > 16
    assert plan.row_block in ((256, 128, 64) if mfma else (16,))
    if row_block:
        assert plan.row_block == row_block
    recs, unit_recs, split = _decode(plan, table, w.n_seqs)
    units, _ = _expected_units(L, G, w.n_kv_heads, plan.row_block)
    assert plan.n_units == len(units)
    T = int(units[:, 8].sum())
    n = plan.n_workgroups
    assert 1 <= n <= T <= 10 ** 7 and plan.n_segments >= n
    if n_wg_req:
        assert n == min(n_wg_req, T)
    # every workgroup's chain starts at its own record, only moves forward,
    # and together the chains visit every record once
    seen = np.zeros(len(recs), bool)
    chain_of = np.full(len(recs), -1)
    for w_i in range(n):
        g = w_i
        while g >= 0:
            assert not seen[g]
            seen[g] = True
            chain_of[g] = w_i
            nxt = int(recs[g, 13])
            assert nxt < 0 or nxt > g
            g = nxt
    assert seen.all()
    # per unit: its segments cover its tiles once, in order of their index,
    # and every record carries its unit's fields, segment count and first
    # segment in unit order; the unit records and the split list agree
    nseg = np.array([np.sum(recs[:, 14] == u) for u in range(len(units))])
    unit_seg = np.concatenate([[0], np.cumsum(nseg)])
    assert np.all(nseg >= 1) and unit_seg[-1] == len(recs)
    assert np.array_equal(unit_recs[:, :5], units[:, [0, 1, 2, 3, 4]])
    assert np.array_equal(unit_recs[:, 5], unit_seg[:-1]) and np.array_equal(unit_recs[:, 6], nseg)
    assert np.all(unit_recs[:, 7] == 0)
    assert list(split) == [u for u in range(len(units)) if nseg[u] > 1]
    for u in range(len(units)):
        mine = recs[recs[:, 14] == u]
        mine = mine[np.argsort(mine[:, 7])]
        assert list(mine[:, 7]) == list(range(len(mine)))
        assert mine[0, 4] == 0 and mine[-1, 5] == units[u, 8]
        assert np.array_equal(mine[1:, 4], mine[:-1, 5]) and np.all(mine[:, 5] > mine[:, 4])
        for r in mine:
            assert tuple(r[[0, 1, 2, 3, 8, 9, 10, 11]]) == tuple(units[u, :8])
            assert r[6] == len(mine) and r[12] == unit_seg[u] and r[15] == 0
    # the wide kernel's 256-row units write the new values once: a segment
    # copies the tokens whose first GQA row lies in its unit's block, every
    # nseg-th from its own index on; over all segments that is every new
    # token of every (request, KV head) exactly once
    copies = {}
    for r in recs:
        s_, h_, rho0, rows, nseg_r, loc = (int(x) for x in r[[0, 1, 2, 3, 6, 7]])
        t0, t1 = -(-rho0 // G), (rho0 + rows - 1) // G + 1
        for t in range(t0 + loc, t1, nseg_r):
            copies[(s_, h_, t)] = copies.get((s_, h_, t), 0) + 1
    snp = L["seq_new_ptr"]
    want = {(s_, h_, t) for s_ in range(len(snp) - 1) for h_ in range(w.n_kv_heads)
            for t in range(int(snp[s_ + 1] - snp[s_]))}
    assert set(copies) == want and all(c == 1 for c in copies.values())
    return plan


@pytest.mark.parametrize("name", ["tiny-f32-3x32", "llama1b-1layer-10doc",
                                  "llama8b-32layer-10doc", "llama8b-32layer-40x512",
                                  "llama8b-paged-16req", "llama8b-decode-40x512",
                                  "llama8b-paged-decode-16req"])
def test_attend_schedule(kv, name):
    """Every schedule, chosen by the cost model or forced, deals every tile of
    every unit out exactly once, in contiguous segments with consistent
    numbering and forward chains per workgroup."""
    w = workloads.get(name)
    chosen = _check_schedule(kv, w, 0)
    for n in [1, 3, 64, 1 << 20]:
        _check_schedule(kv, w, n)
    rows = max(w.n_new(s) for s in range(w.n_seqs)) * (w.n_q_heads // w.n_kv_heads)
    wide = w.dtype == "bf16" and rows > 16
    for rb in ((256, 128, 64) if wide else (16,)):
        for flags in (0, kv.KVLINK_PLAN_XCD):
            _check_schedule(kv, w, 0, rb, flags)
            _check_schedule(kv, w, 7, rb, flags)
    # the long-context workload's tile count keeps the whole chip busy
    if name == "llama8b-32layer-40x512":
        assert chosen.n_workgroups >= 200
    # near ties of the estimate go to the cut with the most workgroups: the
    # 10-document workload fills every compute unit (measured faster than
    # the 208 workgroups of the lowest estimate), a decoding step takes one
    # workgroup per compute unit
    if name in ("llama8b-32layer-10doc", "llama8b-paged-16req", "llama8b-decode-40x512"):
        assert chosen.n_workgroups == 256
    # split units of a decoding step: 32 segments each over the long cache
    # merge faster in the combine launch, the pool's two each in the launch
    if name == "llama8b-decode-40x512":
        assert chosen.flags & kv.KVLINK_PLAN_COMBINE
    if name == "llama8b-paged-decode-16req":
        assert chosen.flags & kv.KVLINK_PLAN_IN_LAUNCH
    # the kernel: 16-row units for bf16 batches of at most 16 rows per KV
    # head (decoding steps), 256-row units for the other bf16 batches
    if w.dtype == "bf16":
        assert chosen.row_block in ((256, 128, 64) if wide else (16,))
    if w.decode:
        assert chosen.n_workgroups >= 256     # every compute unit busy


@settings(max_examples=80, deadline=None)
@given(st.data())
def test_attend_schedule_random_batches(kv, data):
    """The schedule invariants over random batches: 1-4 requests of 0-5
    documents (1-400 tokens, documents shared between requests), 0-5 link
    tokens each, 0-40 queries (at least one new token per request), GQA
    groups 1-8, both dtypes, chosen and forced workgroup counts."""
    n_seqs = data.draw(st.integers(1, 4))
    table = data.draw(st.lists(st.integers(1, 400), min_size=1, max_size=6))
    docs, links, nq = [], [], []
    for _ in range(n_seqs):
        d = data.draw(st.lists(st.integers(0, len(table) - 1), min_size=0, max_size=5))
        lc = data.draw(st.lists(st.integers(0, 5), min_size=len(d), max_size=len(d)))
        q = data.draw(st.integers(0 if sum(lc) else 1, 40))
        docs.append(d)
        links.append(lc)
        nq.append(q)
    hkv = data.draw(st.sampled_from([1, 2, 8]))
    g = data.draw(st.sampled_from([1, 2, 4, 8]))
    dtype = data.draw(st.sampled_from(["bf16", "f32"]))
    w = workloads.Workload(name="random", dtype=dtype, n_layers=1, n_q_heads=hkv * g,
                           n_kv_heads=hkv, head_dim=data.draw(st.sampled_from([64, 128])),
                           rope_theta=1e4, seed=1, doc_table_len=table, docs=docs,
                           link_count=links, n_query=nq)
    rows = max(w.n_new(s) for s in range(w.n_seqs)) * g
    rb = data.draw(st.sampled_from([0, 256, 128, 64])) if dtype == "bf16" and rows > 16 else 0
    _check_schedule(kv, w, data.draw(st.sampled_from([0, 0, 1, 2, 7, 300])), rb,
                    data.draw(st.sampled_from([0, kv.KVLINK_PLAN_XCD])))


def test_attend_schedule_errors(kv):
    mk = kv.kvlink_attend_make_plan
    bf = kv.KVLINK_BF16
    with pytest.raises(kv.KVLinkError) as e:
        mk(bf, 32, 8, 96, [0, 4], [10], [1, 2, 3, 4], 256)
    assert e.value.status == 2
    for args, status in [((bf, 32, 8, 128, [0, 4], [10], [1, 2, 3, 4], 0), 1),
                         ((bf, 32, 8, 128, [0, 4], [10], [1, 2, 3, 4], 256, -1), 1),
                         ((bf, 32, 8, 128, [1, 4], [10], [1, 2, 3, 4], 256), 3),
                         ((bf, 32, 8, 128, [0, 4, 3], [10, 10], [1, 2, 3, 4], 256), 3),
                         ((bf, 32, 8, 128, [0, 4], [10], [1, -2, 3, 4], 256), 3),
                         ((bf, 32, 8, 128, [0, 4], [-1], [1, 2, 3, 4], 256), 3),
                         ((bf, 32, 6, 128, [0, 4], [10], [1, 2, 3, 4], 256), 1)]:
        with pytest.raises(kv.KVLinkError) as e:
            mk(*args)
        assert e.value.status == status, args


def _call_noalloc(kv, a):
    kv.kvlink_attend_new_tokens_noalloc(
        a["dtype"], a["hq"], a["hkv"], a["d"], a["theta"], a["scale"], a["n_seqs"], a["n_new"],
        a["max_new"], a["max_cached"], a["snp"], a["sc"], a["pos"], a["vis"], a["q"], a["k"],
        a["v"], a["kview"], a["vview"], a["layer"], a["out"], a["lse"], a["plan"], stream=0)


@pytest.mark.parametrize("change,status", [
    (dict(d=80), 2),
    (dict(n_seqs=0), 1),
    (dict(scale=0.0), 1),
    (dict(q=None), 1),
    ("table", 1),
])
def test_attend_noalloc_validation(kv, change, status):
    """The allocation-free entry point validates like the workspace one,
    before any HIP call (the scratch lookup included)."""
    if change == "table":
        change = dict(plan=_bad_plan(kv, table=None))
    with pytest.raises(kv.KVLinkError) as e:
        _call_noalloc(kv, _attend_args(kv, **change))
    assert e.value.status == status


def test_attend_noalloc_refuses_calls_beyond_its_scratch(kv):
    """A schedule whose split partials need more than the library's scratch
    (one 64-key tile per segment over a 100,000-row cache) is refused with
    KVLINK_ERR_WORKSPACE before any HIP call."""
    plan = _plan(kv, snp=(0, 64), vis=(100000,) * 64, n_wg=1 << 20)
    need = kv.kvlink_attend_workspace_bytes(kv.KVLINK_BF16, 8, 2, 128, 64, plan)
    assert need > kv.KVLINK_NOALLOC_SCRATCH_BYTES
    with pytest.raises(kv.KVLinkError) as e:
        _call_noalloc(kv, _attend_args(kv, plan=plan, n_new=64, max_new=64, max_cached=100000))
    assert e.value.status == 4
    assert "scratch" in kv.kvlink_last_error()


def test_attend_noalloc_no_new_tokens_is_a_no_op(kv):
    _call_noalloc(kv, _attend_args(kv, n_new=0, max_new=0))


# ------------------------------------------------ re-encode fused into attention


def _call_fused(kv, a, spans=4096, span_ptr=4096, max_spans=10):
    kv.kvlink_attend_new_tokens_fused(
        a["dtype"], a["hq"], a["hkv"], a["d"], a["theta"], a["scale"], a["n_seqs"], a["n_new"],
        a["max_new"], a["max_cached"], a["snp"], a["sc"], a["pos"], a["vis"], a["q"], a["k"],
        a["v"], a["kview"], a["vview"], a["layer"], a["out"], a["lse"], a["plan"], spans,
        span_ptr, max_spans, a["ws"], a["ws_bytes"], stream=0)


@pytest.mark.parametrize("case,status", [
    ("too_many_spans", 2),      # more spans per request than the LDS tables hold
    ("negative_spans", 1),
    ("no_spans", 1),
    ("no_span_ptr", 1),
    ("decode_plan", 2),         # 16-row units: the decode kernel has no fused form
    ("f32", 2),
])
def test_attend_fused_validation(kv, case, status):
    """The fused entry point refuses, before any HIP call, what the wide bf16
    kernel's fused re-encode cannot run."""
    a = _attend_args(kv)
    kw = {}
    if case == "too_many_spans":
        kw = dict(max_spans=kv.KVLINK_FUSED_MAX_SPANS + 1)
    elif case == "negative_spans":
        kw = dict(max_spans=-1)
    elif case == "no_spans":
        kw = dict(spans=None)
    elif case == "no_span_ptr":
        kw = dict(span_ptr=None)
    elif case == "decode_plan":
        a = _attend_args(kv, plan=_plan(kv, snp=(0, 2), vis=(100, 100)), n_new=2, max_new=2)
        assert a["plan"].row_block == 16
    elif case == "f32":
        a = _attend_args(kv, dtype=kv.KVLINK_F32)
    with pytest.raises(kv.KVLinkError) as e:
        _call_fused(kv, a, **kw)
    assert e.value.status == status
    assert kv.kvlink_last_error()
