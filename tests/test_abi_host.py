"""CPU tests of the C-ABI library: it loads, exports every declared symbol,
rejects bad arguments before any HIP call, and its host layout maps equal the
ones derived from the oracle's sequence layout, bit for bit."""
import ctypes
import os
import re

import numpy as np
import pytest

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


def test_struct_sizes_match_header(kv):
    assert ctypes.sizeof(kv.kvlink_span) == 24
    assert ctypes.sizeof(kv.kvlink_kv_view) == 64


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
def test_reencode_validation(kv, change, status):
    a = dict(dtype=kv.KVLINK_BF16, n_layers=2, n_kv_heads=2, head_dim=64, theta=1e4, n_spans=1,
             spans=8192, max_len=4, src_base=4096, rs=64)
    a.update(change)
    src = _view(kv, a["src_base"], rs=a["rs"])
    dst = _view(kv, 8192)
    with pytest.raises(kv.KVLinkError) as e:
        kv.kvlink_reencode_keys(a["dtype"], a["n_layers"], a["n_kv_heads"], a["head_dim"],
                                a["theta"], a["n_spans"], a["spans"], a["max_len"], src, dst,
                                stream=0)
    assert e.value.status == status


def test_reencode_empty_is_a_no_op(kv):
    kv.kvlink_reencode_keys(kv.KVLINK_BF16, 1, 1, 64, 1e4, 0, None, 0, _view(kv), _view(kv),
                            stream=0)


def _attend_args(kv, **change):
    a = dict(dtype=kv.KVLINK_BF16, hq=8, hkv=2, d=128, theta=5e5, scale=0.088, n_seqs=1,
             n_new=10, max_new=10, max_cached=100, snp=16, sc=16, pos=16, vis=16, q=4096,
             k=4096, v=4096, kview=_view(kv), vview=_view(kv), layer=0, out=4096, lse=None,
             split=0, ws=1 << 20, ws_bytes=1 << 30)
    a.update(change)
    return a


def _call_attend(kv, a):
    kv.kvlink_attend_new_tokens(a["dtype"], a["hq"], a["hkv"], a["d"], a["theta"], a["scale"],
                                a["n_seqs"], a["n_new"], a["max_new"], a["max_cached"], a["snp"],
                                a["sc"], a["pos"], a["vis"], a["q"], a["k"], a["v"], a["kview"],
                                a["vview"], a["layer"], a["out"], a["lse"], a["split"], a["ws"],
                                a["ws_bytes"], stream=0)


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
    (dict(split=100), 1),
    (dict(snp=None), 1),
    (dict(q=None), 1),
    (dict(out=None), 1),
    (dict(ws=None), 4),
    (dict(ws=1000), 4),                    # misaligned
    (dict(ws_bytes=16), 4),
    (dict(layer=-1), 1),
])
def test_attend_validation(kv, change, status):
    with pytest.raises(kv.KVLinkError) as e:
        _call_attend(kv, _attend_args(kv, **change))
    assert e.value.status == status
    assert kv.kvlink_last_error()


@pytest.mark.parametrize("stages", [0, 8, 15])
def test_attend_stages_rejects_bad_masks(kv, stages):
    a = _attend_args(kv)
    with pytest.raises(kv.KVLinkError) as e:
        kv.kvlink_attend_stages(a["dtype"], a["hq"], a["hkv"], a["d"], a["theta"], a["scale"],
                                a["n_seqs"], a["n_new"], a["max_new"], a["max_cached"], a["snp"],
                                a["sc"], a["pos"], a["vis"], a["q"], a["k"], a["v"], a["kview"],
                                a["vview"], a["layer"], a["out"], a["lse"], a["split"], a["ws"],
                                a["ws_bytes"], stream=0, stages=stages)
    assert e.value.status == 1


def test_attend_no_new_tokens_is_a_no_op(kv):
    _call_attend(kv, _attend_args(kv, n_new=0, max_new=0))


def test_workspace_bytes(kv):
    f = kv.kvlink_attend_workspace_bytes
    assert f(kv.KVLINK_BF16, 32, 8, 128, 1, 114, 114, 2000, 0) > 114 * 32 * 128 * 2
    assert f(kv.KVLINK_BF16, 32, 8, 96, 1, 114, 114, 2000, 0) == 0
    assert f(kv.KVLINK_BF16, 32, 8, 128, 1, 114, 114, 2000, 100) == 0
    # more splits need more partial storage
    assert f(kv.KVLINK_F32, 4, 2, 64, 1, 22, 22, 96, 128) >= f(kv.KVLINK_F32, 4, 2, 64, 1, 22, 22, 96, 1024)


def test_split_planner(kv):
    """The host split planner returns a positive multiple of 128 for valid
    layouts, no more than the longest row block needs, and 0 on bad input."""
    for name in ["tiny-f32-3x32", "llama8b-32layer-10doc", "llama8b-32layer-40x512",
                 "llama8b-paged-16req"]:
        w = workloads.get(name)
        sdp = np.concatenate([[0], np.cumsum([len(d) for d in w.docs])])
        dl = [w.doc_table_len[j] for s in range(w.n_seqs) for j in w.docs[s]]
        lc = [k for s in range(w.n_seqs) for k in w.link_count[s]]
        L = kv.kvlink_build_layout(sdp, dl, lc, w.n_query)
        dt = kv.KVLINK_F32 if w.dtype == "f32" else kv.KVLINK_BF16
        sk = kv.kvlink_attend_split_keys(dt, w.n_q_heads, w.n_kv_heads, w.head_dim,
                                         L["seq_new_ptr"], L["new_visible"], 256)
        assert sk > 0 and sk % 128 == 0
        assert sk < int(L["totals"][5]) + 128
    assert kv.kvlink_attend_split_keys(kv.KVLINK_BF16, 32, 8, 96, [0, 4], [1, 2, 3, 4], 256) == 0
    assert kv.kvlink_attend_split_keys(kv.KVLINK_BF16, 32, 8, 128, [0, 4], [1, 2, 3, 4], 0) == 0
