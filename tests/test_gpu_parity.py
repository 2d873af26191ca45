"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the
same seeded inputs, at the workload sizes the benchmark uses, plus the
invariants of the method (delta = 0 is a copy, values untouched, schedule
invariance, in-place = out-of-place, run-to-run determinism)."""
import numpy as np
import pytest

import oracle
import workloads
from harness import ContiguousRun, check_bf16_rounding, check_close, to_f64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    import paper_2502_16002_amd  # noqa: F401  (raises if the library is missing)


def _print(*a):
    print(*a, flush=True)


# ------------------------------------------------------------------ re-encode


def _check_reencode(run, layers, rows_sample=None):
    w = run.w
    k_dst = run.k_dst
    b = run.batch
    spans = b.layout["spans"]
    worst = 0.0
    for l in layers:
        kc, _ = workloads.request_cache(w, run.lds[l], 0)
        kc = workloads.as_f64(w, kc)                              # [H][T_c][d]
        got = to_f64(k_dst[l, :, 0, :kc.shape[1]])
        for i, sp in enumerate(spans):
            r0, n, delta = int(sp[3]), int(sp[4]), int(sp[5])
            rows = np.arange(r0, r0 + n) if rows_sample is None else \
                np.unique(np.clip(r0 + rows_sample % n, r0, r0 + n - 1))
            ref = oracle.reencode(kc[:, rows], delta, w.rope_theta)
            worst = max(worst, check_close(w, got[:, rows], ref, f"re-encode layer {l} doc {i}"))
            if w.dtype == "bf16":
                check_bf16_rounding(got[:, rows], ref, f"re-encode layer {l} doc {i}")
    return worst


def test_reencode_tiny_f32():
    w = workloads.tiny_f32()
    run = ContiguousRun(w, layers=[])
    run.batch.reencode(run.src_view, run.k_view)
    _print("tiny re-encode worst", _check_reencode(run, [0]))


def test_reencode_llama1b():
    w = workloads.llama1b_layer()
    run = ContiguousRun(w, layers=[])
    run.batch.reencode(run.src_view, run.k_view)
    _print("1b re-encode worst", _check_reencode(run, [0]))


def test_reencode_llama8b_all_layers():
    w = workloads.llama8b_10doc()
    run = ContiguousRun(w, layers=[])
    run.batch.reencode(run.src_view, run.k_view)
    _print("8b re-encode worst", _check_reencode(run, range(w.n_layers)))


@pytest.fixture(scope="module")
def long_run():
    """The 40 x 512-token workload, all 32 layers re-encoded and attended
    once (shared by the re-encode and attention checks below)."""
    w = workloads.llama8b_long()
    run = ContiguousRun(w, layers=list(range(w.n_layers)))
    run.run()
    return run


def _long_token_sample(n_new, seed):
    """About 5% of the new tokens (seeded) plus the first and last token of
    every 16-token block (at group 4 the smallest unit of the wide kernel,
    64 rows; a 128- or 256-row unit is two or four such blocks)."""
    rng = np.random.default_rng(seed)
    edges = [t for b in range(0, n_new, 16) for t in (b, min(b + 15, n_new - 1))]
    pick = rng.choice(n_new, size=max(1, round(0.05 * n_new)), replace=False)
    return np.unique(np.concatenate([edges, pick]))


def test_reencode_long(long_run):
    """Every key of layers 0, 15 and 31; on every other layer about 5% of
    each document's rows (seeded) plus its first and last row."""
    run = long_run
    worst = _check_reencode(run, [0, 15, 31])
    rng = np.random.default_rng(5)
    for l in range(run.w.n_layers):
        if l in (0, 15, 31):
            continue
        rows = np.concatenate([[0, 511], rng.integers(0, 512, 26)])
        worst = max(worst, _check_reencode(run, [l], rows_sample=rows))
    _print("long re-encode worst", worst)


def test_reencode_first_document_is_bitwise_copy_and_in_place_matches():
    import torch
    from paper_2502_16002_amd.runtime import contiguous_view
    w = workloads.llama1b_layer()
    run = ContiguousRun(w, layers=[])
    run.batch.reencode(run.src_view, run.k_view)
    sp = run.batch.layout["spans"]
    assert sp[0][5] == 0
    n0 = int(sp[0][4])
    torch.cuda.synchronize()
    assert torch.equal(run.k_dst[0, :, 0, :n0].view(torch.int16),
                       run.k_src[0, :, :n0].view(torch.int16))
    # in place: load the stored keys into the concatenated buffer, rotate there
    inplace = torch.zeros_like(run.k_dst)
    inplace[:, :, 0, :run.R] = run.k_src
    view = contiguous_view(inplace, w.n_kv_heads, 1, run.cap, w.head_dim)
    run.batch.reencode(view, view)
    torch.cuda.synchronize()
    assert torch.equal(inplace.view(torch.int16), run.k_dst.view(torch.int16))


# ------------------------------------------- keys stored without rotation


def _check_encode_at_positions(run, layers, rows_sample=None):
    """Keys of the stored caches taken as un-rotated (the paper's literal
    storage form): key t of document i must come out as R(g_i + t) k."""
    w = run.w
    spans = run.batch.layout["spans"]
    worst = 0.0
    for l in layers:
        kc, _ = workloads.request_cache(w, run.lds[l], 0)
        kc = workloads.as_f64(w, kc)                              # [H][T_c][d]
        got = to_f64(run.k_dst[l, :, 0, :kc.shape[1]])
        for i, sp in enumerate(spans):
            r0, n, delta = int(sp[3]), int(sp[4]), int(sp[5])
            ts = np.arange(n) if rows_sample is None else np.unique(rows_sample % n)
            ref = np.stack([oracle.reencode(kc[:, r0 + t], delta + int(t), w.rope_theta)
                            for t in ts], axis=1)                 # [H][len(ts)][d]
            worst = max(worst, check_close(w, got[:, r0 + ts], ref, f"literal layer {l} doc {i}"))
            if w.dtype == "bf16":
                check_bf16_rounding(got[:, r0 + ts], ref, f"literal layer {l} doc {i}")
    return worst


def test_encode_at_positions_tiny_f32():
    w = workloads.tiny_f32()
    run = ContiguousRun(w, layers=[])
    run.batch.encode_at_positions(run.src_view, run.k_view)
    _print("tiny literal worst", _check_encode_at_positions(run, [0]))


def test_encode_at_positions_llama8b_all_layers():
    w = workloads.llama8b_10doc()
    run = ContiguousRun(w, layers=[])
    run.batch.encode_at_positions(run.src_view, run.k_view)
    worst = _check_encode_at_positions(run, [0, 31])
    rng = np.random.default_rng(6)
    worst = max(worst, _check_encode_at_positions(run, [4, 17], rows_sample=rng.integers(0, 300, 24)))
    _print("8b literal worst", worst)


def test_encode_at_positions_equals_reencode_of_locally_rotated_keys():
    """R(g + t) k = R(g) R(t) k: the literal form of raw keys equals the
    delta form of the same keys rotated at local positions 0.. (the local
    rotation done by the oracle and rounded to the workload dtype)."""
    import torch
    from harness import to_torch
    w = workloads.llama1b_layer()
    run = ContiguousRun(w, layers=[])
    run.batch.encode_at_positions(run.src_view, run.k_view)
    literal = to_f64(run.k_dst[0, :, 0, :run.R])
    # the stored keys rotated at their local positions, as a cache would hold them
    ks = workloads.as_f64(w, run.lds[0].k_store)                 # [H][R][d]
    row0 = workloads.doc_row0(w)
    local = np.empty_like(ks)
    for j, n in enumerate(w.doc_table_len):
        for t in range(n):
            local[:, row0[j] + t] = oracle.reencode(ks[:, row0[j] + t], t, w.rope_theta)
    bits = workloads.f32_to_bf16_bits(local.astype(np.float32))
    run.k_src[0] = to_torch(w, bits)
    run.k_dst.zero_()
    run.batch.reencode(run.src_view, run.k_view)
    torch.cuda.synchronize()
    delta_form = to_f64(run.k_dst[0, :, 0, :run.R])
    # the delta path rounds the locally rotated keys to bf16 before the
    # second rotation, which spreads that rounding over each rotation pair:
    # the two results agree within a bf16 ulp of the pair's norm
    h = literal.shape[-1] // 2
    pair = np.sqrt(literal[..., :h] ** 2 + literal[..., h:] ** 2)
    pair = np.concatenate([pair, pair], axis=-1)
    assert np.all(np.abs(literal - delta_form) <= 2.0 ** -7 * pair + 1e-6)


# ------------------------------------------------------ compressed caches


def test_compressed_cache_reencode_and_attention():
    """A compressed cache (Sec. 2.4): each document keeps about a quarter of
    its tokens, cached with RoPE at their original positions p_t; the kept
    keys are re-encoded to contiguous global positions, R(g_i + t - p_t), and
    the new tokens attend over them with the kept-token counts as document
    lengths."""
    import torch
    rng = np.random.default_rng(29)
    orig = rng.integers(300, 600, size=10, endpoint=True)
    kept = [np.sort(rng.choice(n, size=n // 4, replace=False)) for n in orig]
    w = workloads.custom([len(k) for k in kept], 5, 64, n_q_heads=32, n_kv_heads=8,
                         head_dim=128, dtype="bf16", rope_theta=5e5, seed=31, n_layers=2)
    run = ContiguousRun(w, layers=[0, 1])
    b = run.batch
    stored_pos = np.concatenate(kept).astype(np.int32)            # by stored row
    d_pos = torch.from_numpy(stored_pos).cuda()
    b.reencode_mapped(run.src_view, run.k_view, d_pos, 0)
    for l in [0, 1]:
        b.attend(l, run.q[l], run.kn[l], run.vn[l], run.k_view, run.v_view, run.out[l],
                 run.lse[l])
    torch.cuda.synchronize()
    g = b.layout["doc_pos0"]
    row0 = workloads.doc_row0(w)
    for l in [0, 1]:
        kc, vc, q, kn, vn = run.oracle_inputs(l)                  # stored keys as cached
        enc = np.empty_like(kc)
        for i, p in enumerate(kept):
            for t, pt in enumerate(p):
                r = int(row0[i]) + t
                enc[:, r] = oracle.reencode(kc[:, r], int(g[i]) + t - int(pt), w.rope_theta)
        got = to_f64(run.k_dst[l, :, 0, :kc.shape[1]])
        check_close(w, got, enc, f"compressed re-encode layer {l}")
        check_bf16_rounding(got, enc, f"compressed re-encode layer {l}")
        # attention over the re-encoded keys: the oracle takes them as cached
        # at their global positions (no further rotation)
        ref, ref_lse = oracle.attend(w.doc_len(0), w.link_count[0], w.n_query[0], q, kn, vn, enc,
                                     vc, w.rope_theta, w.scale, src_pos0=[int(x) for x in g])
        check_close(w, to_f64(run.out[l]), ref, f"compressed attention layer {l}")
        assert float(np.max(np.abs(to_f64(run.lse[l]) - ref_lse))) <= 2e-2


# ------------------------------------------- caches loaded from host memory


def _load_setup(w):
    import torch
    from harness import to_torch
    run = ContiguousRun(w, layers=[])
    h_k = run.k_src.cpu().pin_memory()                         # [L][H][R][d]
    h_v = to_torch(w, np.stack([ld.v_store for ld in run.lds]), "cpu").pin_memory()
    return run, h_k, h_v


def _load(run, h_k, h_v, way, literal, n_slots=2, k2=None, v2=None, copy=None):
    import torch
    from paper_2502_16002_amd.runtime import contiguous_view
    w, b = run.w, run.batch
    stage = None if way == "direct" else \
        torch.empty(b.load_stage_bytes(run.R, n_slots), dtype=torch.uint8, device="cuda")
    k2 = torch.zeros_like(run.k_dst) if k2 is None else k2
    v2 = torch.zeros_like(run.v_dst) if v2 is None else v2
    H, d = w.n_kv_heads, w.head_dim
    if copy is None:
        copy = torch.cuda.Stream() if way == "staged" else torch.cuda.current_stream()
    b.load_and_reencode(h_k, h_v, run.R, stage, contiguous_view(k2, H, 1, run.cap, d),
                        contiguous_view(v2, H, 1, run.cap, d), literal=literal,
                        copy_stream=copy, compute_stream=torch.cuda.current_stream())
    return k2, v2, stage


@pytest.mark.parametrize("literal,way,n_slots", [(0, "direct", 2), (1, "direct", 2),
                                                 (0, "staged", 2), (1, "staged", 2),
                                                 (0, "staged", 5), (0, "staged", 7),
                                                 (1, "staged", 32),
                                                 (0, "staged_one_stream", 2)])
def test_load_and_reencode_from_host(literal, way, n_slots):
    """All 32 layers of the 10-document workload loaded from pinned host
    memory, read directly by the kernels or copied through a staging ring
    (copies on one stream, re-encodes on another, or both on one; staging
    areas of 2, 5, 7 and 32 layers: chunks of 1, 2, 3 and 16 layers, the
    ring wrapping and the last chunk short for 7): the keys
    against the oracle (every key of four layers: R(delta_i), or R(g_i + t)
    for keys cached without rotation), bit for bit equal to the
    device-resident entry point on every layer; the values equal the stored
    ones."""
    import torch
    w = workloads.llama8b_10doc()
    run, h_k, h_v = _load_setup(w)
    k2, v2, _ = _load(run, h_k, h_v, way, literal, n_slots)
    torch.cuda.synchronize()
    check = _check_encode_at_positions if literal else _check_reencode
    run_k = run.k_dst
    run.k_dst = k2
    worst = check(run, [0, 9, 22, 31])
    run.k_dst = run_k
    _print(f"load {way} literal={literal} slots={n_slots}: oracle worst {worst:.3e}")
    if literal:
        run.batch.encode_at_positions(run.src_view, run.k_view)
    else:
        run.batch.reencode(run.src_view, run.k_view)
    torch.cuda.synchronize()
    assert torch.equal(k2.view(torch.int16), run.k_dst.view(torch.int16))
    assert torch.equal(v2[:, :, 0, :run.R].view(torch.int16),
                       run.v_dst[:, :, 0, :run.R].view(torch.int16))


def test_load_and_reencode_staged_back_to_back():
    """Two staged loads on two streams, one right after the other with no
    synchronisation, through the same two-slot staging area and with
    different stored caches: the second call's first copies must wait for
    the first call's last re-encodes, which still read those slots.  Both
    results equal the device-resident re-encode of their own inputs."""
    import torch
    w = workloads.llama8b_10doc()
    run, h_k, h_v = _load_setup(w)
    h_k2 = (h_k.float() * -0.5).to(h_k.dtype).pin_memory()     # other keys, same shape
    h_v2 = (h_v.float() * 2.0).to(h_v.dtype).pin_memory()
    copy = torch.cuda.Stream()
    ka, va, stage = _load(run, h_k, h_v, "staged", 0, copy=copy)
    from paper_2502_16002_amd.runtime import contiguous_view
    H, d = w.n_kv_heads, w.head_dim
    kb, vb = torch.zeros_like(run.k_dst), torch.zeros_like(run.v_dst)
    run.batch.load_and_reencode(h_k2, h_v2, run.R, stage, contiguous_view(kb, H, 1, run.cap, d),
                                contiguous_view(vb, H, 1, run.cap, d), copy_stream=copy,
                                compute_stream=torch.cuda.current_stream())
    torch.cuda.synchronize()
    for hk, hv, k_got, v_got in [(h_k, h_v, ka, va), (h_k2, h_v2, kb, vb)]:
        run.k_src.copy_(hk)
        run.k_dst.zero_()
        run.batch.reencode(run.src_view, run.k_view)
        torch.cuda.synchronize()
        assert torch.equal(k_got.view(torch.int16), run.k_dst.view(torch.int16))
        assert torch.equal(v_got[:, :, 0, :run.R].cpu().view(torch.int16),
                           hv.view(torch.int16)[:, :, :run.R])


def test_load_and_reencode_direct_refuses_unpinned_host_memory():
    """Reading host memory directly needs it pinned and mapped; a pageable
    array is refused before any launch."""
    import paper_2502_16002_amd as kv
    from paper_2502_16002_amd.runtime import contiguous_view
    import torch
    w = workloads.tiny_f32()
    run = ContiguousRun(w, layers=[])
    h = np.zeros(run.k_src.numel() + 64, np.float32)
    h = h[(-h.ctypes.data % 16) // 4:][:run.k_src.numel()]       # 16-byte aligned, pageable
    with pytest.raises(kv.KVLinkError) as e:
        run.batch.load_and_reencode(h, h, run.R, None, run.k_view, run.v_view)
    assert e.value.status == 1
    torch.cuda.synchronize()


# ------------------------------------------------------------------ attention


def _check_attend(run, l, rows=None, tag=""):
    w = run.w
    kc, vc, q, kn, vn = run.oracle_inputs(l)
    ref, ref_lse = oracle.attend(w.doc_len(0), w.link_count[0], w.n_query[0], q, kn, vn, kc, vc,
                                 w.rope_theta, w.scale, rows=rows)
    got = to_f64(run.out[l])
    lse = to_f64(run.lse[l])
    if rows is not None:
        got, lse = got[rows], lse[rows]
    worst = check_close(w, got, ref, f"{tag} attention layer {l}")
    lse_err = float(np.max(np.abs(lse - ref_lse)))
    assert lse_err <= (1e-5 if w.dtype == "f32" else 2e-2), f"{tag} lse err {lse_err}"
    return worst, lse_err


def _check_append(run, l):
    """The new tokens' keys (rotated at their positions) and values were
    appended after the cached rows."""
    w, b = run.w, run.batch
    Tc = int(b.layout["seq_cached"][0])
    _, _, _, kn, vn = run.oracle_inputs(l)
    pos = b.layout["new_pos"]
    got_k = to_f64(run.k_dst[l, :, 0, Tc:Tc + b.n_new])      # [H][n_new][d]
    got_v = to_f64(run.v_dst[l, :, 0, Tc:Tc + b.n_new])
    ref_k = np.stack([[oracle.rope(kn[r, h], int(pos[r]), w.rope_theta) for r in range(b.n_new)]
                      for h in range(w.n_kv_heads)])
    check_close(w, got_k, ref_k, "appended keys")
    assert np.array_equal(got_v, vn.transpose(1, 0, 2))


def test_attend_tiny_f32():
    w = workloads.tiny_f32()
    run = ContiguousRun(w, layers=[0])
    run.run()
    _print("tiny attend", _check_attend(run, 0, tag="tiny"))
    _check_append(run, 0)


def test_attend_llama1b():
    w = workloads.llama1b_layer()
    run = ContiguousRun(w, layers=[0])
    run.run()
    _print("1b attend", _check_attend(run, 0, tag="1b"))
    _check_append(run, 0)


def test_attend_llama8b_32_layers():
    """Every new token and head of every one of the 32 layers."""
    w = workloads.llama8b_10doc()
    run = ContiguousRun(w, layers=list(range(w.n_layers)))
    run.run()
    worst = (0.0, 0.0)
    for l in range(w.n_layers):
        e = _check_attend(run, l, tag="8b")
        worst = (max(worst[0], e[0]), max(worst[1], e[1]))
    _print("8b attend worst (row rel, lse abs) over 32 layers", worst)
    _check_append(run, 31)


def test_attend_long_full_layers(long_run):
    """Layers 0, 15 and 31 of the 20,808-position workload: all 328 new
    tokens x 32 heads, i.e. every row of the six row blocks of every KV
    head; and the appended rows of layer 31."""
    for l in [0, 15, 31]:
        _print("long attend layer", l, _check_attend(long_run, l, tag="long"))
    _check_append(long_run, 31)


def test_attend_long_other_layers_sampled(long_run):
    """The other 29 layers: about 5% of the new tokens of each (seeded, a
    new sample per layer) plus the first and last token of every row block."""
    run = long_run
    n_new = run.batch.n_new
    worst = (0.0, 0.0)
    for l in range(run.w.n_layers):
        if l in (0, 15, 31):
            continue
        rows = _long_token_sample(n_new, 100 + l)
        e = _check_attend(run, l, rows=rows, tag="long sampled")
        worst = (max(worst[0], e[0]), max(worst[1], e[1]))
    _print("long attend sampled layers worst (row rel, lse abs)", worst)


@pytest.mark.parametrize("n_wg", [1, 5, 64, 1 << 20])
def test_schedule_invariance(n_wg):
    """One workgroup for everything (all units direct, many segments per
    workgroup), ranges crossing units, and one tile per segment (the request
    is capped at the tile count) agree with the default schedule."""
    w = workloads.llama1b_layer()
    base = ContiguousRun(w, layers=[0])
    base.run()
    other = ContiguousRun(w, layers=[0], n_workgroups=n_wg)
    other.run()
    a, b = to_f64(base.out[0]), to_f64(other.out[0])
    rowmax = np.maximum(np.max(np.abs(a), axis=-1), 1e-30)
    # Two schedules round differently: their bf16 split partials (half an
    # ulp, 2^-9 of the row maximum, on each side), the bf16 weights P under
    # different running maxima, and the final bf16 rounding (one ulp apart,
    # up to 2^-7 of the row maximum).  They must agree within the bf16
    # tolerance each result meets against the oracle.
    diff = float(np.max(np.max(np.abs(a - b), axis=-1) / rowmax))
    _print("schedule", n_wg, "max diff / row max", diff)
    assert diff <= 2e-2
    _check_attend(other, 0, tag=f"n_wg {n_wg}")


@pytest.mark.parametrize("doc_len,link_count,n_query", [
    ([], [], 9),                            # no documents: plain causal queries
    ([37], [0], 20),                        # one document, K = 0
    ([1, 1, 3, 1], [3, 0, 2, 1], 0),        # ragged, no queries
    ([130, 5, 260], [5, 5, 5], 33),         # lengths crossing tile edges
])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_attend_edge_layouts(doc_len, link_count, n_query, dtype):
    w = workloads.custom(doc_len, link_count, n_query, n_q_heads=8, n_kv_heads=2,
                         head_dim=128 if dtype == "bf16" else 64, dtype=dtype,
                         rope_theta=5e5, seed=17)
    for n_wg in [0, 3]:
        run = ContiguousRun(w, layers=[0], n_workgroups=n_wg)
        run.run()
        _check_attend(run, 0, tag=f"edge{doc_len}/{n_wg}")
        if doc_len:
            _check_reencode(run, [0])


def test_run_twice_is_bitwise_identical():
    import torch
    w = workloads.llama1b_layer()
    run = ContiguousRun(w, layers=[0])
    run.run()
    first = run.out[0].clone()
    run.run()
    assert torch.equal(first.view(torch.int16), run.out[0].view(torch.int16))


@pytest.mark.parametrize("n_wg", [0, 7])
def test_stage_by_stage_matches_all_stages(n_wg):
    """The three stages launched one call at a time give the same bits as the
    single call."""
    import torch
    from paper_2502_16002_amd import (KVLINK_STAGE_COMBINE, KVLINK_STAGE_ROPE,
                                      KVLINK_STAGE_SPLIT)
    w = workloads.llama1b_layer()
    run = ContiguousRun(w, layers=[0], n_workgroups=n_wg)
    run.run()
    first, first_lse = run.out[0].clone(), run.lse[0].clone()
    run.out[0].zero_()
    run.lse[0].zero_()
    for st in [KVLINK_STAGE_ROPE, KVLINK_STAGE_SPLIT, KVLINK_STAGE_COMBINE]:
        run.batch.attend(0, run.q[0], run.kn[0], run.vn[0], run.k_view, run.v_view, run.out[0],
                         run.lse[0], stages=st)
    torch.cuda.synchronize()
    assert torch.equal(first.view(torch.int16), run.out[0].view(torch.int16))
    assert torch.equal(first_lse, run.lse[0])


def test_graph_replay_matches_eager():
    """The path captured in a HIP graph (torch's graph capture records the
    library's launches on the capture stream) gives the eager result on
    every replay, with eager work and synchronisations between replays."""
    import torch
    w = workloads.llama1b_layer()
    run = ContiguousRun(w, layers=[0])
    run.run()
    ref_out, ref_lse = run.out[0].clone(), run.lse[0].clone()
    ref_k = run.k_dst.clone()

    def step():
        run.batch.reencode(run.src_view, run.k_view)
        run.batch.attend(0, run.q[0], run.kn[0], run.vn[0], run.k_view, run.v_view, run.out[0],
                         run.lse[0])
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for i in range(3):
        run.out[0].zero_()
        run.lse[0].zero_()
        run.k_dst.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(run.out[0].view(torch.int16), ref_out.view(torch.int16)), i
        assert torch.equal(run.lse[0], ref_lse), i
        assert torch.equal(run.k_dst.view(torch.int16), ref_k.view(torch.int16)), i
        run.run()                                  # eager work between replays
        assert torch.equal(run.out[0].view(torch.int16), ref_out.view(torch.int16)), i


# ------------------------------------------------------------ fused RoPE


def test_rope_table_matches_fp64_angles():
    """Every entry of the batch's RoPE table is cos/sin of the fp64 angle
    p_n * theta^(-2j/d) (Sec. 2.2), rounded to float."""
    import torch
    from paper_2502_16002_amd import kvlink_attend_rope_table
    for d, theta, top in [(128, 5e5, 20808), (64, 1e4, 118)]:
        pos = np.concatenate([np.arange(0, 40), np.arange(top - 40, top)]).astype(np.int32)
        d_pos = torch.from_numpy(pos).cuda()
        table = torch.empty((len(pos), d // 2, 2), dtype=torch.float32, device="cuda")
        kvlink_attend_rope_table(d, theta, len(pos), d_pos, table)
        torch.cuda.synchronize()
        got = table.cpu().numpy().astype(np.float64)
        ang = pos[:, None].astype(np.float64) * theta ** (-2.0 * np.arange(d // 2) / d)[None, :]
        err = max(float(np.max(np.abs(got[..., 0] - np.cos(ang)))),
                  float(np.max(np.abs(got[..., 1] - np.sin(ang)))))
        _print("rope table", d, theta, err)
        assert err <= 2.0 ** -24


def _fused_vs_separate(make, layers):
    """The same batch with the RoPE inside the split launch and as its own
    launch: identical bytes in the outputs, the lse and both caches."""
    import torch
    a, b = make(True), make(False)
    assert a.batch.plan.rope_table and not b.batch.plan.rope_table
    a.run()
    b.run()
    for l in layers:
        assert torch.equal(a.out[l].view(torch.int16), b.out[l].view(torch.int16)), l
        assert torch.equal(a.lse[l], b.lse[l]), l
    assert torch.equal(a.k_dst.view(torch.int16), b.k_dst.view(torch.int16))
    v_a = a.v_dst if hasattr(a, "v_dst") else a.v_all
    v_b = b.v_dst if hasattr(b, "v_dst") else b.v_all
    assert torch.equal(v_a.view(torch.int16), v_b.view(torch.int16))
    return a


@pytest.mark.parametrize("name,n_wg", [("llama1b", 0), ("llama1b", 1), ("llama1b", 7),
                                       ("llama1b", 1 << 20), ("8b-2layer", 0),
                                       ("decode-2layer", 0), ("decode-2layer", 1 << 20)])
def test_fused_rope_matches_separate_launch(name, n_wg):
    w = {"llama1b": lambda: workloads.llama1b_layer(),
         "8b-2layer": lambda: workloads.llama8b_10doc(n_layers=2),
         "decode-2layer": lambda: workloads.llama8b_long_decode(n_layers=2)}[name]()
    layers = list(range(w.n_layers))
    run = _fused_vs_separate(lambda f: ContiguousRun(w, layers, n_workgroups=n_wg, fused_rope=f),
                             layers)
    _check_attend(run, layers[-1], rows=np.arange(min(run.batch.n_new, 24)), tag=f"fused {name}")
    _check_append(run, layers[-1])


@pytest.mark.parametrize("doc_len,link_count,n_query,head_dim", [
    ([], [], 9, 128),                       # only new keys: tile 0 holds new rows
    ([1, 1, 3, 1], [3, 0, 2, 1], 0, 64),    # ragged, no queries
    ([130, 5, 260], [5, 5, 5], 33, 128),    # new rows across tile edges
    ([37], [0], 1, 64),                     # decode kernel: one token
    ([700, 2000], [0, 0], 1, 128),          # decode kernel: long cache, many segments
])
def test_fused_rope_edge_layouts(doc_len, link_count, n_query, head_dim):
    w = workloads.custom(doc_len, link_count, n_query, n_q_heads=8, n_kv_heads=2,
                         head_dim=head_dim, dtype="bf16", rope_theta=5e5, seed=29)
    for n_wg in [0, 3, 1 << 20]:
        run = _fused_vs_separate(lambda f: ContiguousRun(w, [0], n_workgroups=n_wg, fused_rope=f),
                                 [0])
        _check_attend(run, 0, tag=f"fused edge {doc_len}/{n_wg}")
        _check_append(run, 0)


def test_fused_rope_paged_pool():
    """Fused RoPE with the new rows written through per-request block tables
    (K into shuffled request pages, V into fresh pages after the pool's)."""
    from harness import PagedRun
    w = workloads.llama8b_paged()
    _fused_vs_separate(lambda f: PagedRun(w, fused_rope=f), [0])


# ------------------------------------------------- batches of several requests


class _BatchRun:
    """Several requests in one batch over contiguous caches: stored documents
    back to back in one source sequence, each request's re-encoded keys and
    its values in its own sequence of [layer][head][request][row][d] views."""

    def __init__(self, w, n_workgroups=0, fused_rope=True):
        import torch
        from harness import to_torch
        from paper_2502_16002_amd.runtime import Batch, contiguous_view, dtype_code
        self.w = w
        L, H, d = w.n_layers, w.n_kv_heads, w.head_dim
        self.ld = workloads.layer_data(w, 0)
        row0 = workloads.doc_row0(w)
        sdp = np.concatenate([[0], np.cumsum([len(x) for x in w.docs])]).astype(np.int32)
        dl = [w.doc_table_len[j] for x in w.docs for j in x]
        lc = [k for x in w.link_count for k in x]
        self.batch = b = Batch(dtype_code(w.dtype), L, w.n_q_heads, H, d, w.rope_theta, w.scale,
                               sdp, dl, lc, w.n_query, doc_src_seq=[0] * len(dl),
                               doc_src_row=[int(row0[j]) for x in w.docs for j in x],
                               n_workgroups=n_workgroups, fused_rope=fused_rope)
        R = max(int(sum(w.doc_table_len)), 1)
        S, cap = w.n_seqs, max(b.max_total, 1)
        self.k_src = torch.zeros((L, H, 1, R, d), dtype=b.torch_dtype, device="cuda")
        if sum(w.doc_table_len):
            self.k_src[0, :, 0] = to_torch(w, self.ld.k_store)
        self.k_dst = torch.zeros((L, H, S, cap, d), dtype=b.torch_dtype, device="cuda")
        self.v_dst = torch.zeros((L, H, S, cap, d), dtype=b.torch_dtype, device="cuda")
        for q in range(S):
            _, vc = workloads.request_cache(w, self.ld, q)
            if vc.shape[1]:
                self.v_dst[0, :, q, :vc.shape[1]] = to_torch(w, vc)
        self.src_view = contiguous_view(self.k_src, H, 1, R, d)
        self.k_view = contiguous_view(self.k_dst, H, S, cap, d)
        self.v_view = contiguous_view(self.v_dst, H, S, cap, d)
        self.q, self.kn, self.vn = (to_torch(w, x) for x in (self.ld.q_new, self.ld.k_new,
                                                             self.ld.v_new))
        self.out = {0: b.new_out()}
        self.lse = {0: b.new_lse()}

    def run(self):
        import torch
        self.batch.reencode(self.src_view, self.k_view)
        self.batch.attend(0, self.q, self.kn, self.vn, self.k_view, self.v_view, self.out[0],
                          self.lse[0])
        torch.cuda.synchronize()


def _check_batch(run, tag):
    w, b = run.w, run.batch
    got, lse = to_f64(run.out[0]), to_f64(run.lse[0])
    k_dst, v_dst = to_f64(run.k_dst[0]), to_f64(run.v_dst[0])
    for q in range(w.n_seqs):
        kc, vc = workloads.request_cache(w, run.ld, q)
        qn, kn, vn = workloads.request_new(w, run.ld, q)
        f = lambda x: workloads.as_f64(w, x)
        kc, vc, qn, kn, vn = f(kc), f(vc), f(qn), f(kn), f(vn)
        n0, n1 = int(b.layout["seq_new_ptr"][q]), int(b.layout["seq_new_ptr"][q + 1])
        Tc = int(b.layout["seq_cached"][q])
        assert Tc == kc.shape[1]
        if n1 > n0:
            ref, ref_lse = oracle.attend(w.doc_len(q), w.link_count[q], w.n_query[q], qn, kn, vn,
                                         kc, vc, w.rope_theta, w.scale)
            check_close(w, got[n0:n1], ref, f"{tag} request {q}")
            assert float(np.max(np.abs(lse[n0:n1] - ref_lse))) <= (1e-5 if w.dtype == "f32"
                                                                    else 2e-2)
            # the appended new rows, after the request's cached rows
            pos = b.layout["new_pos"][n0:n1]
            ref_k = np.stack([[oracle.rope(kn[r, h], int(pos[r]), w.rope_theta)
                               for r in range(n1 - n0)] for h in range(w.n_kv_heads)])
            check_close(w, k_dst[:, q, Tc:Tc + n1 - n0], ref_k, f"{tag} appended keys {q}")
            assert np.array_equal(v_dst[:, q, Tc:Tc + n1 - n0], vn.transpose(1, 0, 2))
        # the re-encoded documents of the request
        spans = b.layout["spans"][int(np.sum([len(x) for x in w.docs[:q]])):][:len(w.docs[q])]
        for sp in spans:
            rows = np.arange(int(sp[3]), int(sp[3]) + int(sp[4]))
            ref = oracle.reencode(kc[:, rows], int(sp[5]), w.rope_theta)
            check_close(w, k_dst[:, q, rows], ref, f"{tag} re-encode request {q}")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("kind", ["prefill", "decode"])
def test_batch_of_requests_contiguous(dtype, kind):
    """Four requests of different shapes in one batch over contiguous caches
    (a request without documents, one document, several, one reused by two
    requests): every request's output, LSE, appended rows and re-encoded keys
    against the oracle; for bf16 also the RoPE inside the split kernels
    against its separate launch, bit for bit."""
    table = [130, 7, 64, 300, 1, 45]
    docs = [[], [3], [0, 1, 2], [4, 5, 0]]
    if kind == "prefill":
        links = [[], [5], [2, 0, 3], [1, 1, 4]]
        nq = [9, 33, 1, 17]
    else:
        links = [[], [0], [0, 0, 0], [0, 0, 0]]
        nq = [1, 2, 1, 4]
    w = workloads.Workload(name="batch4", dtype=dtype, n_layers=1, n_q_heads=8, n_kv_heads=2,
                           head_dim=128 if dtype == "bf16" else 64, rope_theta=5e5, seed=37,
                           doc_table_len=table, docs=docs, link_count=links, n_query=nq)
    for n_wg in [0, 3]:
        if dtype == "bf16":
            a, b = _BatchRun(w, n_wg, True), _BatchRun(w, n_wg, False)
            a.run()
            b.run()
            import torch
            assert torch.equal(a.out[0].view(torch.int16), b.out[0].view(torch.int16))
            assert torch.equal(a.k_dst.view(torch.int16), b.k_dst.view(torch.int16))
            run = a
            assert run.batch.plan.row_block in ((16,) if kind == "decode" else (256, 128, 64))
        else:
            run = _BatchRun(w, n_wg)
            run.run()
        _check_batch(run, f"batch {dtype} {kind} {n_wg}")


@pytest.mark.parametrize("seed", range(8))
def test_random_batches(seed):
    """Seeded random batches: 1-4 requests of 0-5 documents (1-300 tokens,
    shared between requests), 0-5 link tokens each, 0-40 queries, GQA groups
    1-8, head_dim 64 or 128, both dtypes, a random workgroup count: every
    request against the oracle."""
    rng = np.random.default_rng(1000 + seed)
    table = [int(x) for x in rng.integers(1, 301, size=int(rng.integers(1, 7)))]
    docs, links, nq = [], [], []
    for _ in range(int(rng.integers(1, 5))):
        d = [int(x) for x in rng.integers(0, len(table), size=int(rng.integers(0, 6)))]
        lc = [int(x) for x in rng.integers(0, 6, size=len(d))]
        docs.append(d)
        links.append(lc)
        nq.append(int(rng.integers(0 if sum(lc) else 1, 41)))
    hkv = int(rng.choice([1, 2, 8]))
    g = int(rng.choice([1, 2, 4, 8]))
    dtype = ["bf16", "f32"][seed % 2]
    w = workloads.Workload(name=f"random{seed}", dtype=dtype, n_layers=1, n_q_heads=hkv * g,
                           n_kv_heads=hkv, head_dim=int(rng.choice([64, 128])),
                           rope_theta=float(rng.choice([1e4, 5e5])), seed=41 + seed,
                           doc_table_len=table, docs=docs, link_count=links, n_query=nq)
    n_wg = int(rng.choice([0, 1, 5, 300]))
    _print("random batch", seed, dtype, "heads", hkv * g, hkv, "d", w.head_dim, "docs", docs,
           "links", links, "queries", nq, "n_wg", n_wg)
    run = _BatchRun(w, n_wg)
    run.run()
    _check_batch(run, f"random {seed}")


# ------------------------------------------------------------- GQA groups


@pytest.mark.parametrize("hq,hkv", [(4, 4), (8, 4), (16, 2), (8, 8)])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("layout", ["prefill", "decode"])
def test_gqa_groups(hq, hkv, dtype, layout):
    """GQA groups 1, 2 and 8 (the workloads use 2 and 4): row packing
    (row = token x group + head), unit sizes and the path choice (the decode
    kernel when group x new tokens <= 16), against the oracle; for bf16 the
    RoPE inside the split kernels against its separate launch, bit for bit."""
    if layout == "prefill":
        doc_len, link_count, n_query = [45, 130, 7], [3, 2, 1], 21
    else:
        doc_len, link_count, n_query = [300, 520], [0, 0], 16 // (hq // hkv) if hq // hkv > 1 else 2
    w = workloads.custom(doc_len, link_count, n_query, n_q_heads=hq, n_kv_heads=hkv,
                         head_dim=128 if dtype == "bf16" else 64, dtype=dtype, rope_theta=5e5,
                         seed=31)
    for n_wg in [0, 5]:
        if dtype == "bf16":
            run = _fused_vs_separate(
                lambda f: ContiguousRun(w, [0], n_workgroups=n_wg, fused_rope=f), [0])
        else:
            run = ContiguousRun(w, [0], n_workgroups=n_wg)
            run.run()
        g = hq // hkv
        if dtype == "bf16":
            expect = (16,) if g * max(run.batch.max_new, 1) <= 16 else (256, 128, 64)
            assert run.batch.plan.row_block in expect
        _check_attend(run, 0, tag=f"gqa {hq}/{hkv} {dtype} {layout} {n_wg}")
        _check_append(run, 0)


# ---------------------------------------------------------------- decode step


def test_decode_step_long_cache():
    """One new query token (4 GQA rows per KV head) over the 20,480-token
    re-encoded cache of the long workload: every output row and the append."""
    w = workloads.llama8b_long_decode(n_layers=2)
    run = ContiguousRun(w, layers=[0, 1])
    run.run()
    assert run.batch.plan.row_block == 16           # the decode kernel
    for l in [0, 1]:
        _print("decode layer", l, _check_attend(run, l, tag="decode"))
    _check_append(run, 1)


@pytest.mark.parametrize("doc_len,link_count,n_query", [
    ([37], [0], 1),                         # one token, one short document
    ([130, 5, 260], [1, 0, 1], 2),          # 4 new tokens: 16 rows, tiles across documents
    ([1, 1, 3, 1], [1, 0, 1, 1], 0),        # ragged, link tokens only (12 rows)
    ([], [], 3),                            # no documents
    ([700, 2000], [0, 0], 1),               # a long cache cut into many segments
])
@pytest.mark.parametrize("head_dim", [64, 128])
def test_decode_kernel_layouts(doc_len, link_count, n_query, head_dim):
    """Units of at most 16 rows (group 4, up to 4 new tokens) on the decode
    kernel, for several workgroup counts, split units merged in the launch
    or by the combine launch, with the new rows' RoPE and append inside the
    split launch or before it."""
    import paper_2502_16002_amd as kv
    w = workloads.custom(doc_len, link_count, n_query, n_q_heads=8, n_kv_heads=2,
                         head_dim=head_dim, dtype="bf16", rope_theta=5e5, seed=23)
    for flags in [kv.KVLINK_PLAN_XCD | kv.KVLINK_PLAN_IN_LAUNCH, kv.KVLINK_PLAN_COMBINE]:
        for fused in [True, False]:
            for n_wg in [0, 1, 3, 1 << 20]:
                run = ContiguousRun(w, layers=[0], n_workgroups=n_wg, plan_flags=flags,
                                    fused_rope=fused)
                assert run.batch.plan.row_block == 16
                run.run()
                tag = f"decode{doc_len}/{head_dim}/{n_wg}/{flags}/{fused}"
                _check_attend(run, 0, tag=tag)
                _check_append(run, 0)
                _counters_zero(run)


def test_decode_step_paged_pool():
    """One new token for each of the 16 shared-pool requests, keys and values
    read through the block tables."""
    from harness import PagedRun
    w = workloads.llama8b_paged_decode()
    run = PagedRun(w)
    run.run()
    b = run.batch
    got_all, lse_all = to_f64(run.out[0]), to_f64(run.lse[0])
    for s in range(w.n_seqs):
        kc, vc, q, kn, vn = run.oracle_inputs(0, s)
        ref, ref_lse = oracle.attend(w.doc_len(s), w.link_count[s], w.n_query[s], q, kn, vn, kc,
                                     vc, w.rope_theta, w.scale)
        n0 = int(b.layout["seq_new_ptr"][s])
        check_close(w, got_all[n0:n0 + 1], ref, f"paged decode request {s}")
        assert float(np.max(np.abs(lse_all[n0:n0 + 1] - ref_lse))) <= 2e-2


# ------------------------------------------------- document-major re-encode


def test_shared_reencode_equals_per_span_pool():
    """The shared pool (every document used by about five of the sixteen
    requests): the document-major re-encode writes the same bytes as the
    per-span one, and is what the batch runs by default."""
    import torch
    import paper_2502_16002_amd as kv
    from harness import PagedRun
    w = workloads.llama8b_paged()
    run = PagedRun(w)
    b = run.batch
    assert b.shared_docs and len(w.doc_table_len) <= b.n_groups < b.n_docs
    run.k_dst.zero_()
    b.reencode(run.src_view, run.k_view, shared=False)
    per_span = run.k_dst.clone()
    run.k_dst.zero_()
    b.reencode(run.src_view, run.k_view)
    torch.cuda.synchronize()
    assert torch.equal(per_span.view(torch.int16), run.k_dst.view(torch.int16))
    # every cut of the documents' runs of spans (one group per document, one
    # span per group, groups of up to 2 or 3) writes the same bytes
    spans = b.layout["spans"].reshape(-1, 6)
    for mg in [0, 1, 2, 3]:
        order, gptr = kv.kvlink_group_spans(spans, mg)
        d_sp = torch.from_numpy(np.ascontiguousarray(spans[order])).cuda()
        d_gp = torch.from_numpy(gptr).cuda()
        run.k_dst.zero_()
        kv.kvlink_reencode_keys_shared(b.dtype, b.n_layers, b.n_kv_heads, b.head_dim,
                                       b.rope_theta, len(gptr) - 1, d_gp, d_sp, b.max_doc_len,
                                       run.src_view, run.k_view)
        torch.cuda.synchronize()
        assert torch.equal(per_span.view(torch.int16), run.k_dst.view(torch.int16)), mg


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_shared_reencode_equals_per_span_batch(dtype):
    """A contiguous batch where one document serves three spans and another
    two (one of them twice in one request), both dtypes and head_dims."""
    import torch
    for d in [64, 128]:
        w = workloads.Workload(name="shared", dtype=dtype, n_layers=3, n_q_heads=8, n_kv_heads=2,
                               head_dim=d, rope_theta=5e5, seed=43, doc_table_len=[70, 1, 300],
                               docs=[[0, 2], [2, 0, 2], [0, 1]], link_count=[[1, 2], [0, 0, 3],
                                                                              [2, 2]],
                               n_query=[5, 9, 1])
        run = _BatchRun(w)
        assert run.batch.shared_docs
        run.batch.reencode(run.src_view, run.k_view, shared=False)
        per_span = run.k_dst.clone()
        run.k_dst.zero_()
        run.batch.reencode(run.src_view, run.k_view, shared=True)
        torch.cuda.synchronize()
        assert torch.equal(per_span, run.k_dst)
        run.run()                                  # the default path, then the attention
        _check_batch(run, f"shared {dtype} {d}")


# ---------------------------------------------------------------- paged pool


def test_paged_pool_reencode_and_attention():
    """Shared 64-document pool in 16-token pages, 16 requests: per-request
    re-encoded K copies in shuffled pages, V read from the pool pages.  Every
    request: the re-encoded keys of all 20 of its spans, and the output and
    LSE of all of its new tokens and heads."""
    from harness import PagedRun
    w = workloads.llama8b_paged()
    run = PagedRun(w)
    run.run()
    b = run.batch
    k_dst = to_f64(run.k_dst[0])                       # [pages][H][P][d]
    out_all, lse_all = to_f64(run.out[0]), to_f64(run.lse[0])
    worst_k, worst_o, worst_lse = 0.0, 0.0, 0.0
    d0 = 0
    for s in range(w.n_seqs):
        kc, vc, q, kn, vn = run.oracle_inputs(0, s)
        spans = b.layout["spans"][d0:d0 + len(w.docs[s])]
        d0 += len(w.docs[s])
        for i, sp in enumerate(spans):
            rows = np.arange(sp[3], sp[3] + sp[4])
            pg, slot = run.request_rows(run.k_table_np, s, rows)
            got = k_dst[pg, :, slot, :].transpose(1, 0, 2)      # [H][n][d]
            ref = oracle.reencode(kc[:, rows], int(sp[5]), w.rope_theta)
            worst_k = max(worst_k, check_close(w, got, ref, f"paged re-encode request {s} span {i}"))
            check_bf16_rounding(got, ref, f"paged re-encode request {s} span {i}")
        n0, n1 = int(b.layout["seq_new_ptr"][s]), int(b.layout["seq_new_ptr"][s + 1])
        ref, ref_lse = oracle.attend(w.doc_len(s), w.link_count[s], w.n_query[s], q, kn, vn, kc,
                                     vc, w.rope_theta, w.scale)
        worst_o = max(worst_o, check_close(w, out_all[n0:n1], ref, f"paged attention request {s}"))
        lse_err = float(np.max(np.abs(lse_all[n0:n1] - ref_lse)))
        assert lse_err <= 2e-2, f"paged lse request {s}: {lse_err}"
        worst_lse = max(worst_lse, lse_err)
    _print("paged pool worst: re-encode", worst_k, "attention", worst_o, "lse", worst_lse)
    # values in the pool pages are untouched
    ld = run.lds[0]
    assert np.array_equal(to_f64(run.v_all[0, int(run.pool_table[3, 2])]),
                          workloads.as_f64(w, ld.v_store[:, 3 * 256 + 32:3 * 256 + 48]).reshape(8, 16, 128))


# ------------------------------------- wide-kernel unit shapes and the merge


def _counters_zero(run):
    import torch
    torch.cuda.synchronize()
    assert int(run.batch.workspace[:64 * 1024].count_nonzero()) == 0, "merge counters not reset"


# plan flags: the cost model's merge; XCD numbering with the combine launch;
# XCD numbering with the merge in the launch; the merge in the launch alone
@pytest.mark.parametrize("flags", [0, 1 | 4, 1 | 8, 8])
@pytest.mark.parametrize("row_block", [256, 128, 64])
def test_wide_unit_shapes_against_oracle(row_block, flags):
    if row_block == 256 and flags & 8:
        pytest.skip("256-row units merge by the combine launch only")
    """Each unit shape of the wide kernel (256 rows on eight wavefronts; 128
    and 64 rows on two key groups of four wavefronts), with and without the
    XCD-aware numbering, split units merged by the combine
    launch or inside the split launch: the 10-document Llama-8B workload (two
    layers, every row) and the Llama-1B one (head_dim 64) under the
    schedule's own cut and under forced workgroup counts that split every
    unit into one-tile segments; the appended rows of every layer (the
    256-row units copy each new value once, dealt over a unit's segments);
    the merge counters are zero afterwards."""
    worst = 0.0
    for w, n_wgs in [(workloads.llama8b_10doc(n_layers=2), [0]),
                     (workloads.llama1b_layer(), [0, 1, 7, 1 << 20])]:
        for n_wg in n_wgs:
            run = ContiguousRun(w, layers=list(range(w.n_layers)), n_workgroups=n_wg,
                                row_block=row_block, plan_flags=flags)
            assert run.batch.plan.row_block == row_block
            run.run()
            for l in range(w.n_layers):
                worst = max(worst, _check_attend(run, l, tag=f"rb{row_block}/{n_wg}/{flags}")[0])
                _check_append(run, l)
            _counters_zero(run)
            if n_wg == 1 << 20:
                assert run.batch.plan.n_split_units == run.batch.plan.n_units
    _print(f"row block {row_block} flags {flags}: worst row rel {worst:.3e}")


@pytest.mark.parametrize("row_block", [256, 128, 64])
@pytest.mark.parametrize("doc_len,link_count,n_query", [
    ([5], [0], 7),                          # K = 0: causal queries
    ([1, 1, 1], [3, 3, 3], 0),              # 1-token documents, no queries
    ([63, 64, 65], [1, 2, 3], 5),           # lengths across tile edges
    ([], [], 40),                           # no documents
    ([300, 700], [5, 5], 64),               # a longer cache cut into segments
])
def test_wide_unit_shapes_edge_layouts(row_block, doc_len, link_count, n_query):
    w = workloads.custom(doc_len, link_count, n_query, n_q_heads=8, n_kv_heads=2, head_dim=128,
                         dtype="bf16", rope_theta=5e5, seed=17)
    for n_wg in [0, 3, 1 << 20]:
        run = ContiguousRun(w, layers=[0], n_workgroups=n_wg, row_block=row_block)
        run.run()
        _check_attend(run, 0, tag=f"edge rb{row_block}/{n_wg}")
        _check_append(run, 0)
        _counters_zero(run)


@pytest.mark.parametrize("row_block", [128, 64])
def test_wide_unit_shapes_paged_pool(row_block):
    """The 16-request shared pool through block tables with the smaller unit
    shapes and the XCD-aware numbering: every request's output and LSE."""
    from harness import PagedRun
    w = workloads.llama8b_paged()
    run = PagedRun(w, row_block=row_block, plan_flags=1 | 8)
    run.run()
    b = run.batch
    out_all, lse_all = to_f64(run.out[0]), to_f64(run.lse[0])
    worst = 0.0
    for s in range(w.n_seqs):
        kc, vc, q, kn, vn = run.oracle_inputs(0, s)
        ref, ref_lse = oracle.attend(w.doc_len(s), w.link_count[s], w.n_query[s], q, kn, vn, kc,
                                     vc, w.rope_theta, w.scale)
        n0, n1 = int(b.layout["seq_new_ptr"][s]), int(b.layout["seq_new_ptr"][s + 1])
        worst = max(worst, check_close(w, out_all[n0:n1], ref, f"paged rb{row_block} request {s}"))
        assert float(np.max(np.abs(lse_all[n0:n1] - ref_lse))) <= 2e-2
    _counters_zero(run)
    _print(f"paged pool row block {row_block}: worst {worst:.3e}")


# -------------------------------------------- re-encode fused into attention


def _fused_equals_separate(batch, layers, separate, fused, k_fused, stored_rows):
    """Run the separate path (re-encode, then every layer's attention) and
    the fused one (every layer's attention over the stored keys); the fused
    outputs and LSE must equal the separate ones bit for bit, the stored
    rows must be unchanged and the appended new rows equal.
    separate(): returns {layer: (out, lse)} and the separate cache;
    fused(): returns {layer: (out, lse)}; stored_rows(k) -> (stored part,
    new part) of a cache for comparison."""
    import torch
    ref, k_sep = separate()
    before = stored_rows(k_fused)[0].clone()
    got = fused()
    torch.cuda.synchronize()
    for l in layers:
        assert torch.equal(got[l][0].view(torch.int16), ref[l][0].view(torch.int16)), l
        assert torch.equal(got[l][1], ref[l][1]), l
    st_f, new_f = stored_rows(k_fused)
    assert torch.equal(st_f.view(torch.int16), before.view(torch.int16)), "stored rows written"
    assert torch.equal(new_f.view(torch.int16), stored_rows(k_sep)[1].view(torch.int16))


def _fused_contiguous(w, layers, **kw):
    import torch
    from paper_2502_16002_amd.runtime import contiguous_view
    run = ContiguousRun(w, layers, **kw)
    b = run.batch
    H, d = w.n_kv_heads, w.head_dim
    Tc = int(b.layout["seq_cached"][0])
    assert Tc == run.R                                # documents stored in request order
    k_f = torch.zeros_like(run.k_dst)
    k_f[:, :, 0, :run.R] = run.k_src
    view = contiguous_view(k_f, H, 1, run.cap, d)

    def separate():
        run.run()
        return {l: (run.out[l], run.lse[l]) for l in layers}, run.k_dst

    def fused():
        res = {}
        for l in layers:
            out, lse = b.new_out(), b.new_lse()
            b.attend(l, run.q[l], run.kn[l], run.vn[l], view, run.v_view, out, lse,
                     fused_reencode=True)
            res[l] = (out, lse)
        return res
    rows = lambda k: (k[:, :, 0, :Tc], k[layers][:, :, 0, Tc:Tc + b.n_new])
    _fused_equals_separate(b, layers, separate, fused, k_f, rows)
    return run


@pytest.mark.parametrize("row_block,flags", [(0, None), (256, 1 | 4), (128, 1 | 8), (128, 1 | 4),
                                             (64, 1 | 8), (64, 1 | 4)])
def test_fused_reencode_llama1b(row_block, flags):
    """head_dim 64, ten documents: the fused re-encode gives the separate
    path's bytes for every unit shape and merge, and several workgroup
    counts; the outputs against the oracle."""
    w = workloads.llama1b_layer()
    for n_wg in [0, 1, 7]:
        run = _fused_contiguous(w, [0], n_workgroups=n_wg, row_block=row_block, plan_flags=flags)
        _check_attend(run, 0, tag=f"fused 1b rb{row_block} {flags} {n_wg}")


def test_fused_reencode_llama8b_two_layers():
    """head_dim 128, the 10-document batch, two layers, the default plan."""
    w = workloads.llama8b_10doc(n_layers=2)
    run = _fused_contiguous(w, [0, 1])
    _check_attend(run, 1, tag="fused 8b")


def test_fused_reencode_long_context():
    """The 40-document, 20,480-row cache (40 spans per request), two layers:
    the fused bytes equal the separate path's on every output row."""
    w = workloads.llama8b_long(n_layers=2)
    _fused_contiguous(w, [0, 1])


@pytest.mark.parametrize("doc_len,link_count,n_query", [
    ([1, 1, 3, 1], [1, 0, 1, 1], 17),        # documents shorter than a key group
    ([63, 64, 65], [2, 2, 2], 30),            # documents ending around tile edges
    ([130, 5, 260], [1, 0, 1], 20),
    ([700, 2000], [0, 0], 9),                 # long documents, many tiles each
])
def test_fused_reencode_edge_layouts(doc_len, link_count, n_query):
    w = workloads.custom(doc_len, link_count, n_query, n_q_heads=8, n_kv_heads=2, head_dim=128,
                         dtype="bf16", rope_theta=5e5, seed=41)
    for n_wg in [0, 3]:
        run = _fused_contiguous(w, [0], n_workgroups=n_wg)
        assert run.batch.plan.row_block in (256, 128, 64)
        _check_attend(run, 0, tag=f"fused edge {doc_len} {n_wg}")


def test_fused_reencode_paged_pool():
    """The shared pool: the fused path reads every request's keys straight
    from the pool pages through the values' block table (no per-request key
    copies at all) and matches the per-request re-encoded copies bit for
    bit; every request against the oracle."""
    import torch
    from harness import PagedRun
    from paper_2502_16002_amd.runtime import paged_view
    w = workloads.llama8b_paged()
    run = PagedRun(w)
    b = run.batch
    L, H, d, P = w.n_layers, w.n_kv_heads, w.head_dim, w.page_size
    n_pool = run.k_pool.shape[1]
    k_all = torch.zeros_like(run.v_all)
    k_all[:, :n_pool] = run.k_pool
    view = paged_view(k_all, run.v_all.shape[1], H, P, d, run.v_table, run.max_pages)

    def separate():
        run.run()
        return {l: (run.out[l], run.lse[l]) for l in range(L)}, None

    def fused():
        res = {}
        for l in range(L):
            out, lse = b.new_out(), b.new_lse()
            b.attend(l, run.q[l], run.kn[l], run.vn[l], view, run.v_view, out, lse,
                     fused_reencode=True)
            res[l] = (out, lse)
        return res
    ref, _ = separate()
    pool_before = k_all[:, :n_pool].clone()
    got = fused()
    torch.cuda.synchronize()
    for l in range(L):
        assert torch.equal(got[l][0].view(torch.int16), ref[l][0].view(torch.int16)), l
        assert torch.equal(got[l][1], ref[l][1]), l
    assert torch.equal(k_all[:, :n_pool].view(torch.int16), pool_before.view(torch.int16))
    got_all = to_f64(got[0][0])
    for s in [0, 7, 15]:
        kc, vc, q, kn, vn = run.oracle_inputs(0, s)
        ref_o, _ = oracle.attend(w.doc_len(s), w.link_count[s], w.n_query[s], q, kn, vn, kc, vc,
                                 w.rope_theta, w.scale)
        n0 = int(b.layout["seq_new_ptr"][s])
        check_close(w, got_all[n0:n0 + w.n_new(s)], ref_o, f"fused paged request {s}")


def test_fused_reencode_batch_of_requests():
    """Four requests over one stored sequence (a document reused by two
    requests, one request without documents): each request's spans rotate
    its own rows; bytes equal to the separate path's."""
    import torch
    from paper_2502_16002_amd.runtime import contiguous_view
    table = [130, 7, 64, 300, 1, 45]
    w = workloads.Workload(name="batch4", dtype="bf16", n_layers=1, n_q_heads=8, n_kv_heads=2,
                           head_dim=128, rope_theta=5e5, seed=37, doc_table_len=table,
                           docs=[[], [3], [0, 1, 2], [4, 5, 0]],
                           link_count=[[], [5], [2, 0, 3], [1, 1, 4]], n_query=[9, 33, 1, 17])
    run = _BatchRun(w)
    b = run.batch
    H, d = w.n_kv_heads, w.head_dim
    k_f = torch.zeros_like(run.k_dst)
    for sp in b.layout["spans"].reshape(-1, 6):
        src_row, dst_seq, dst_row, n = int(sp[1]), int(sp[2]), int(sp[3]), int(sp[4])
        k_f[:, :, dst_seq, dst_row:dst_row + n] = run.k_src[:, :, 0, src_row:src_row + n]
    S, cap = w.n_seqs, k_f.shape[3]
    view = contiguous_view(k_f, H, S, cap, d)
    run.run()
    ref_out, ref_lse = run.out[0].clone(), run.lse[0].clone()
    out, lse = b.new_out(), b.new_lse()
    b.attend(0, run.q, run.kn, run.vn, view, run.v_view, out, lse, fused_reencode=True)
    torch.cuda.synchronize()
    assert b.plan.row_block in (256, 128, 64)
    assert torch.equal(out.view(torch.int16), ref_out.view(torch.int16))
    assert torch.equal(lse, ref_lse)
