"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: values the
paper gives for a worked example, closed forms, textbook and library special
cases, brute force on tiny inputs, and invariants.  They are chosen so that a
plausible mistake in the oracle (a dropped term, a wrong sign or index, a
swapped RoPE pairing, a wrong GQA mapping, a wrong mask) fails one of them.
"""
import math

import numpy as np
import pytest
import scipy.special
import torch

import oracle
import workloads
from conftest import golden_path

# ------------------------------------------------------------------ RoPE pins


def test_rope_d2_is_plain_rotation():
    """d = 2: the only frequency is theta^0 = 1, so R_p is the textbook 2-D
    rotation by p radians (positive direction), for any theta."""
    for p in [0, 1, 2, 3, 10, 100, 12345]:
        for theta in [1e4, 5e5]:
            for x in [(1.0, 0.0), (0.0, 1.0), (0.3, -1.7)]:
                c, s = math.cos(p), math.sin(p)
                want = (x[0] * c - x[1] * s, x[0] * s + x[1] * c)
                got = oracle.rope(np.array(x), p, theta)
                assert abs(got[0] - want[0]) < 1e-12 and abs(got[1] - want[1]) < 1e-12


@pytest.mark.parametrize("d,theta,j,omega", [
    # theta^(-2j/d) at points where it has a closed form
    (64, 1e4, 0, 1.0),
    (64, 1e4, 8, 0.1),            # 10^4^(-16/64) = 10^-1
    (64, 1e4, 16, 0.01),          # 10^4^(-32/64)
    (64, 1e4, 24, 0.001),         # 10^4^(-48/64)
    (128, 1e4, 32, 0.01),
    (128, 5e5, 32, 1.0 / math.sqrt(5e5)),
    (128, 5e5, 0, 1.0),
    (64, 5e5, 16, 1.0 / math.sqrt(5e5)),
])
def test_rope_pairing_and_frequency(d, theta, j, omega):
    """A unit vector on dimension j moves only within the pair (j, j + d/2),
    by the angle p * omega_j with omega_j = theta^(-2j/d) (half-split pairing)."""
    for p in [1, 7, 517, 20807]:
        e = np.zeros(d)
        e[j] = 1.0
        got = oracle.rope(e, p, theta)
        want = np.zeros(d)
        want[j] = math.cos(p * omega)
        want[j + d // 2] = math.sin(p * omega)
        # p*omega in double carries ~p*1e-16 rad of rounding; 1e-11 covers it
        np.testing.assert_allclose(got, want, atol=1e-11, rtol=0)


def test_rope_matches_complex_multiplication():
    """RoPE as complex multiplication (the RoFormer view): the pair
    (x_j, x_{j+d/2}) is the complex number x_j + i x_{j+d/2}, multiplied by
    exp(i p omega_j)."""
    rng = np.random.default_rng(11)
    for d in [2, 8, 64, 128]:
        for theta in [1e4, 5e5]:
            for p in [0, 3, 250, 20807]:
                x = rng.standard_normal(d)
                h = d // 2
                omega = np.array([float(theta) ** (-2.0 * j / d) for j in range(h)])
                z = (x[:h] + 1j * x[h:]) * np.exp(1j * p * omega)
                want = np.concatenate([z.real, z.imag])
                np.testing.assert_allclose(oracle.rope(x, p, theta), want, atol=1e-10, rtol=0)


def test_rope_composition_identity():
    """R_(p+delta) k == R_delta R_p k to 1e-12 over the positions of the
    workloads (the identity that lets the re-encode use one extra rotation)."""
    rng = np.random.default_rng(12)
    worst = 0.0
    for d in [64, 128]:
        for theta in [1e4, 5e5]:
            for _ in range(40):
                p, delta = (int(v) for v in rng.integers(0, 20809, size=2))
                k = rng.standard_normal(d)
                direct = oracle.rope(k, p + delta, theta)
                composed = oracle.rope(oracle.rope(k, p, theta), delta, theta)
                worst = max(worst, float(np.max(np.abs(direct - composed))))
    assert worst <= 1e-12, worst


def test_rope_preserves_pair_norms_and_relative_position():
    """Each pair is rotated (norm kept), and <R_a q, R_b k> depends on a - b only."""
    rng = np.random.default_rng(13)
    d, theta = 128, 5e5
    q, k = rng.standard_normal(d), rng.standard_normal(d)
    h = d // 2
    r = oracle.rope(k, 777, theta)
    np.testing.assert_allclose(r[:h] ** 2 + r[h:] ** 2, k[:h] ** 2 + k[h:] ** 2, rtol=1e-13)
    base = np.dot(oracle.rope(q, 900, theta), oracle.rope(k, 300, theta))
    for shift in [1, 55, 10000]:
        s = np.dot(oracle.rope(q, 900 + shift, theta), oracle.rope(k, 300 + shift, theta))
        assert abs(s - base) < 1e-10


def test_reencode_equals_rotation_at_global_positions():
    """Sec. 2.2: a key stored with RoPE at local position t and re-encoded by
    delta = g (the document's global offset) equals the un-rotated key rotated
    directly at its global position g + t."""
    rng = np.random.default_rng(14)
    d, theta, L = 128, 5e5, 40
    for g in [0, 34, 517, 20163]:
        x = rng.standard_normal((L, d))               # W_k x, no position yet
        stored = np.stack([oracle.rope(x[t], t, theta) for t in range(L)])
        got = oracle.reencode(stored, g, theta)
        want = np.stack([oracle.rope(x[t], g + t, theta) for t in range(L)])
        assert np.max(np.abs(got - want)) <= 1e-12
    # delta = 0 is the identity, bit for bit
    y = rng.standard_normal((3, 7, d))
    assert np.array_equal(oracle.reencode(y, 0, theta), y)


def test_reencode_rejects_bad_head_dim():
    with pytest.raises(ValueError):
        oracle.reencode(np.zeros((2, 3)), 1, 1e4)


# ---------------------------------------------------------------- layout pins


def test_layout_tiny_workload_positions():
    """3 documents of 32 tokens, 2 link tokens each, 16 query tokens: 118
    positions; documents start at 0, 34, 68; link tokens at 32-33, 66-67,
    100-101; queries at 102..117."""
    kind, seg, idx = oracle.layout([32, 32, 32], [2, 2, 2], 16)
    assert len(kind) == 118
    starts = [int(np.argmax((kind == oracle.KIND_DOC) & (seg == i))) for i in range(3)]
    assert starts == [0, 34, 68]
    links = np.nonzero(kind == oracle.KIND_LINK)[0].tolist()
    assert links == [32, 33, 66, 67, 100, 101]
    assert np.nonzero(kind == oracle.KIND_QUERY)[0].tolist() == list(range(102, 118))
    assert seg[links].tolist() == [0, 0, 1, 1, 2, 2] and idx[links].tolist() == [0, 1] * 3


def test_layout_sec22_position_example():
    """Sec. 2.2: with Doc_a before Doc_b, the second token of Doc_b sits at
    |Doc_a| + 2 in the paper's 1-based numbering (no link tokens)."""
    for la, lb in [(5, 3), (100, 7), (1, 2)]:
        kind, seg, idx = oracle.layout([la, lb], [0, 0], 0)
        pos = int(np.nonzero((seg == 1) & (idx == 1))[0][0])
        assert pos + 1 == la + 2


def test_layout_rejects_invalid():
    for args in [([0, 3], [1, 1], 2), ([3], [-1], 2), ([3], [1], -1)]:
        with pytest.raises(ValueError):
            oracle.layout(*args)


def _load_golden_map(name):
    rows = []
    with open(golden_path(name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append([int(v) for v in line.split()])
    return np.array(rows, dtype=bool)


def test_attention_map_fig2():
    """Sec. 2.3, Fig. 2: the 9x9 training map of the worked example, 33
    allowed entries; the rows of the link tokens and the user token (26
    entries) equal plain causal rows, the inference map of the caption."""
    want = _load_golden_map("fig2_attention_map.txt")
    kind, seg, _ = oracle.layout([2, 2, 1], [1, 1, 1], 1)
    got = oracle.full_mask(kind, seg)
    assert got.shape == (9, 9)
    assert np.array_equal(got, want)
    assert int(got.sum()) == 33
    new_rows = np.nonzero(kind != oracle.KIND_DOC)[0]
    assert new_rows.tolist() == [2, 5, 7, 8]
    causal = np.tril(np.ones((9, 9), dtype=bool))
    assert np.array_equal(got[new_rows], causal[new_rows])
    assert int(got[new_rows].sum()) == 26


def test_allowed_pairs_closed_form_tiny():
    """Every new token sees every position at or before its own, so the new
    rows of the tiny workload hold sum(p + 1) = 2173 allowed entries."""
    kind, seg, _ = oracle.layout([32, 32, 32], [2, 2, 2], 16)
    m = oracle.full_mask(kind, seg)
    assert int(m[kind != oracle.KIND_DOC].sum()) == 2173


def test_allowed_pairs_closed_form_long():
    """40 documents of 512 tokens, 5 link tokens each, 128 queries: 20,808
    positions, and sum over new positions of (p + 1) = 4,774,596."""
    kind, seg, _ = oracle.layout([512] * 40, [5] * 40, 128)
    assert len(kind) == 20808
    newp = np.nonzero(kind != oracle.KIND_DOC)[0]
    assert int((newp + 1).sum()) == 4774596
    # spot-check the map itself on a few rows
    for a in [newp[0], newp[4], newp[200], newp[-1]]:
        assert all(oracle.allowed(kind, seg, int(a), b) for b in range(0, int(a) + 1, 997))
        assert not oracle.allowed(kind, seg, int(a), int(a) + 1)


def test_doc_tokens_are_local_causal():
    kind, seg, _ = oracle.layout([4, 3], [2, 2], 2)
    m = oracle.full_mask(kind, seg)
    # token 1 of doc 1 (position 7) sees only positions 6, 7
    assert np.nonzero(m[7])[0].tolist() == [6, 7]
    # doc tokens never see link tokens
    assert not m[np.ix_(kind == oracle.KIND_DOC, kind == oracle.KIND_LINK)].any()


# ------------------------------------------------------------- attention pins


def _rope_np(x, p, theta):
    """Independent RoPE for the brute force: complex multiplication form."""
    d = x.shape[-1]
    h = d // 2
    omega = float(theta) ** (-2.0 * np.arange(h) / d)
    z = (x[..., :h] + 1j * x[..., h:]) * np.exp(1j * p * omega)
    return np.concatenate([z.real, z.imag], axis=-1)


def _tiny_inputs(seed=3, doc_len=(32, 32, 32), links=2, nq=16, hq=4, hkv=2, d=64):
    w = workloads.custom(list(doc_len), links, nq, n_q_heads=hq, n_kv_heads=hkv, head_dim=d,
                         seed=seed)
    ld = workloads.layer_data(w, 0)
    kc, vc = workloads.request_cache(w, ld, 0)
    q, kn, vn = workloads.request_new(w, ld, 0)
    return w, kc.astype(np.float64), vc.astype(np.float64), q.astype(np.float64), \
        kn.astype(np.float64), vn.astype(np.float64)


def _brute_force(w, kc, vc, q, kn, vn):
    """Full T x T masked softmax in numpy (scipy softmax) over the whole
    sequence, keys built with the complex-form RoPE: the softmax rows P[h] of
    the link and query tokens, their outputs and LSE."""
    theta, scale = w.rope_theta, w.scale
    dl, lc, nq = w.doc_len(0), w.link_count[0], w.n_query[0]
    kind, seg, idx = oracle.layout(dl, lc, nq)
    T = len(kind)
    mask = oracle.full_mask(kind, seg)
    hkv, d = kc.shape[0], kc.shape[2]
    hq = q.shape[1]
    # keys and values of every position, keys at their global positions
    K = np.zeros((T, hkv, d))
    V = np.zeros((T, hkv, d))
    Q = np.zeros((T, hq, d))
    row0 = np.concatenate([[0], np.cumsum(dl)])
    n = 0
    for p in range(T):
        if kind[p] == oracle.KIND_DOC:
            r = row0[seg[p]] + idx[p]
            g = p - idx[p]
            K[p] = _rope_np(kc[:, r, :], g, theta)    # stored at local t, moved by g
            V[p] = vc[:, r, :]
        else:
            K[p] = _rope_np(kn[n], p, theta)
            V[p] = vn[n]
            Q[p] = _rope_np(q[n], p, theta)
            n += 1
    new_rows = np.nonzero(kind != oracle.KIND_DOC)[0]
    out_bf = np.zeros((len(new_rows), hq, d))
    lse_bf = np.zeros((len(new_rows), hq))
    probs = np.zeros((hq, len(new_rows), T))
    group = hq // hkv
    for h in range(hq):
        S = scale * (Q[:, h, :] @ K[:, h // group, :].T)
        S = np.where(mask, S, -np.inf)
        P = scipy.special.softmax(S[new_rows], axis=1)
        probs[h] = P
        out_bf[:, h, :] = P @ V[:, h // group, :]
        lse_bf[:, h] = scipy.special.logsumexp(S[new_rows], axis=1)
    return new_rows, probs, out_bf, lse_bf


def test_attend_matches_brute_force_full_matrix():
    """The brute-force full-matrix masked softmax equals the oracle's
    streaming rows of the link and query tokens."""
    w, kc, vc, q, kn, vn = _tiny_inputs()
    _, _, out_bf, lse_bf = _brute_force(w, kc, vc, q, kn, vn)
    out, lse = oracle.attend(w.doc_len(0), w.link_count[0], w.n_query[0], q, kn, vn, kc, vc,
                             w.rope_theta, w.scale)
    assert np.max(np.abs(out - out_bf)) <= 1e-12
    assert np.max(np.abs(lse - lse_bf)) <= 1e-12


@pytest.mark.parametrize("hq,hkv", [(4, 2), (8, 2)])
def test_attend_probs_matches_brute_force_softmax_row(hq, hkv):
    """attend_probs, element by element, equals the brute-force softmax row
    (same token, same query head) for heads of every KV group, the last
    included (h // group = hkv - 1), on link tokens of the first and later
    documents and on query tokens."""
    w, kc, vc, q, kn, vn = _tiny_inputs(seed=13, hq=hq, hkv=hkv)
    new_rows, probs, _, _ = _brute_force(w, kc, vc, q, kn, vn)
    dl, lc, nq = w.doc_len(0), w.link_count[0], w.n_query[0]
    group = hq // hkv
    heads = [0, group - 1, group, hq - 1]       # KV groups 0, 0, 1 and the last
    for r in [0, 1, 2, 3, 5, len(new_rows) - 1]:
        for h in heads:
            p = oracle.attend_probs(dl, lc, nq, q, kn, kc, w.rope_theta, w.scale, r, h)
            assert p.shape == probs[h, r].shape
            assert np.max(np.abs(p - probs[h, r])) <= 1e-13, (r, h)


def test_attend_one_document_no_links_equals_torch_sdpa():
    """One document and K = 0 (the PromptCache-style layout) reduces the query
    rows to plain causal attention with an offset: torch's float64
    scaled_dot_product_attention with enable_gqa (query head h reads KV head
    h // group) on the same rotated inputs."""
    L, nq, hq, hkv, d, theta = 20, 9, 8, 2, 32, 1e4
    w, kc, vc, q, kn, vn = _tiny_inputs(seed=5, doc_len=(L,), links=0, nq=nq, hq=hq, hkv=hkv,
                                        d=d)
    scale = 0.37
    out, lse = oracle.attend([L], [0], nq, q, kn, vn, kc, vc, theta, scale)
    T = L + nq
    Kall = np.concatenate([kc.transpose(1, 0, 2),                       # doc at offset 0
                           np.stack([oracle.rope(kn[i, h], L + i, theta)
                                     for i in range(nq) for h in range(hkv)]).reshape(nq, hkv, d)])
    Vall = np.concatenate([vc.transpose(1, 0, 2), vn])
    Qr = np.stack([oracle.rope(q[i, h], L + i, theta)
                   for i in range(nq) for h in range(hq)]).reshape(nq, hq, d)
    mask = np.arange(T)[None, :] <= (L + np.arange(nq))[:, None]
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(Qr.transpose(1, 0, 2))[None], torch.from_numpy(Kall.transpose(1, 0, 2))[None],
        torch.from_numpy(Vall.transpose(1, 0, 2))[None], attn_mask=torch.from_numpy(mask),
        scale=scale, enable_gqa=True)[0].numpy().transpose(1, 0, 2)
    assert np.max(np.abs(out - ref)) <= 1e-12


def test_attend_rows_sum_to_one_and_respect_map():
    w, kc, vc, q, kn, vn = _tiny_inputs(seed=8)
    dl, lc, nq = w.doc_len(0), w.link_count[0], w.n_query[0]
    kind, seg, _ = oracle.layout(dl, lc, nq)
    new_rows = np.nonzero(kind != oracle.KIND_DOC)[0]
    for r in [0, 1, 3, 5, 21]:
        for h in [0, 3]:
            p = oracle.attend_probs(dl, lc, nq, q, kn, kc, w.rope_theta, w.scale, r, h)
            assert abs(math.fsum(p) - 1.0) <= 1e-12
            a = int(new_rows[r])
            assert np.all(p[a + 1:] == 0) and np.all(p[:a + 1] > 0)


def test_attend_uniform_values_and_single_key():
    rng = np.random.default_rng(21)
    hq, hkv, d = 4, 2, 16
    # uniform values: every allowed value equal -> output equals it
    dl, lc, nq = [5, 6], [2, 1], 4
    n_new = sum(lc) + nq
    vconst = rng.standard_normal(d)
    kc = rng.standard_normal((hkv, sum(dl), d))
    vc = np.broadcast_to(vconst, (hkv, sum(dl), d)).copy()
    q = rng.standard_normal((n_new, hq, d))
    kn = rng.standard_normal((n_new, hkv, d))
    vn = np.broadcast_to(vconst, (n_new, hkv, d)).copy()
    out, _ = oracle.attend(dl, lc, nq, q, kn, vn, kc, vc, 1e4, 0.25)
    assert np.max(np.abs(out - vconst)) <= 1e-13
    # no documents: the first query sees only itself (position 0, no rotation)
    nq = 3
    q = rng.standard_normal((nq, hq, d))
    kn = rng.standard_normal((nq, hkv, d))
    vn = rng.standard_normal((nq, hkv, d))
    out, lse = oracle.attend([], [], nq, q, kn, vn, np.zeros((hkv, 0, d)), np.zeros((hkv, 0, d)),
                             1e4, 0.25)
    for h in range(hq):
        np.testing.assert_array_equal(out[0, h], vn[0, h // 2])
        assert abs(lse[0, h] - 0.25 * np.dot(q[0, h], kn[0, h // 2])) <= 1e-14


def test_attend_row_subset_matches_full():
    w, kc, vc, q, kn, vn = _tiny_inputs(seed=9)
    dl, lc, nq = w.doc_len(0), w.link_count[0], w.n_query[0]
    full, lfull = oracle.attend(dl, lc, nq, q, kn, vn, kc, vc, w.rope_theta, w.scale)
    rows = [21, 0, 7]
    sub, lsub = oracle.attend(dl, lc, nq, q, kn, vn, kc, vc, w.rope_theta, w.scale, rows=rows)
    np.testing.assert_array_equal(sub, full[rows])
    np.testing.assert_array_equal(lsub, lfull[rows])


def test_attend_src_pos0_shift():
    """Keys stored at local positions s0 + t need delta = g - s0: storing them
    at shifted positions and passing src_pos0 gives the same attention."""
    rng = np.random.default_rng(31)
    hq, hkv, d, theta = 4, 2, 32, 1e4
    dl, lc, nq = [6, 5], [1, 1], 3
    x = rng.standard_normal((hkv, sum(dl), d))          # un-rotated keys
    local = np.concatenate([np.arange(6), np.arange(5)])
    s0 = [100, 3]
    shifted = np.concatenate([np.full(6, s0[0]), np.full(5, s0[1])])
    st0 = np.stack([[oracle.rope(x[h, r], local[r], theta) for r in range(11)] for h in range(hkv)])
    st1 = np.stack([[oracle.rope(x[h, r], local[r] + shifted[r], theta) for r in range(11)]
                    for h in range(hkv)])
    n_new = 5
    q = rng.standard_normal((n_new, hq, d))
    kn = rng.standard_normal((n_new, hkv, d))
    vn = rng.standard_normal((n_new, hkv, d))
    vc = rng.standard_normal((hkv, 11, d))
    a, _ = oracle.attend(dl, lc, nq, q, kn, vn, st0, vc, theta, 0.2)
    b, _ = oracle.attend(dl, lc, nq, q, kn, vn, st1, vc, theta, 0.2, src_pos0=s0)
    assert np.max(np.abs(a - b)) <= 1e-12
