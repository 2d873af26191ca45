// kvlink_api.cpp — the C ABI of include/kvlink.h: host-side layout, argument
// validation (before any HIP call) and the launches.
#include <algorithm>
#include <tuple>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <functional>
#include <mutex>
#include <string>
#include <vector>

#include "kvlink_internal.h"

namespace {

thread_local std::string g_error;

kvlink_status fail(kvlink_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_error = buf;
    return st;
}

kvlink_status ok() {
    g_error.clear();
    return KVLINK_OK;
}

size_t elem_size(kvlink_dtype dt) { return dt == KVLINK_BF16 ? 2 : 4; }

bool dtype_ok(kvlink_dtype dt) { return dt == KVLINK_F32 || dt == KVLINK_BF16; }

// A view must be usable with 16-byte vector accesses.
kvlink_status check_view(const kvlink_kv_view& v, kvlink_dtype dt, const char* name) {
    const size_t es = elem_size(dt);
    const int64_t q = (int64_t)(16 / es);
    if (!v.base) return fail(KVLINK_ERR_INVALID_ARG, "%s: base is NULL", name);
    if (reinterpret_cast<uintptr_t>(v.base) % 16)
        return fail(KVLINK_ERR_INVALID_ARG, "%s: base is not 16-byte aligned", name);
    if (v.layer_stride % q || v.head_stride % q || v.row_stride % q || v.seq_stride % q ||
        v.page_stride % q)
        return fail(KVLINK_ERR_INVALID_ARG, "%s: a stride is not a multiple of 16 bytes", name);
    if (v.layer_stride < 0 || v.head_stride < 0 || v.row_stride < 0 || v.seq_stride < 0 ||
        v.page_stride < 0)
        return fail(KVLINK_ERR_INVALID_ARG, "%s: negative stride", name);
    if (v.block_table && (v.page_size < 1 || v.max_pages < 1))
        return fail(KVLINK_ERR_INVALID_ARG, "%s: paged view needs page_size and max_pages >= 1",
                    name);
    return KVLINK_OK;
}

kvlink::View to_view(const kvlink_kv_view& v) {
    kvlink::View d;
    d.base = reinterpret_cast<char*>(v.base);
    d.layer_stride = v.layer_stride;
    d.head_stride = v.head_stride;
    d.row_stride = v.row_stride;
    d.seq_stride = v.seq_stride;
    d.page_stride = v.page_stride;
    d.block_table = v.block_table;
    d.page_size = v.block_table ? v.page_size : 1;
    d.max_pages = v.max_pages;
    return d;
}

}  // namespace

namespace kvlink {

RopeFreqs make_rope_freqs(double theta, int head_dim) {
    RopeFreqs f;
    for (int j = 0; j < 64; ++j)
        f.w[j] = j < head_dim / 2
                     ? (double)powl((long double)theta, -2.0L * j / (long double)head_dim)
                     : 0.0;
    // pi/2 = p0 + p1 + p2 with p0, p1 of 22 significant bits each
    const long double pio2 = acosl(0.0L);
    auto trunc22 = [](long double v) {
        int e;
        const long double m = frexpl(v, &e);
        return ldexpl(floorl(ldexpl(m, 22)), e - 22);
    };
    const long double p0 = trunc22(pio2);
    const long double p1 = trunc22(pio2 - p0);
    f.pio2[0] = (double)p0;
    f.pio2[1] = (double)p1;
    f.pio2[2] = (double)(pio2 - p0 - p1);
    return f;
}

}  // namespace kvlink

extern "C" {

kvlink_status kvlink_build_layout(int32_t n_seqs, const int32_t* seq_doc_ptr,
                                  const int32_t* doc_len, const int32_t* link_count,
                                  const int32_t* n_query, const int32_t* doc_src_seq,
                                  const int32_t* doc_src_row, const int32_t* doc_src_pos0,
                                  kvlink_span* spans, int32_t* doc_pos0, int32_t* seq_cached,
                                  int32_t* seq_new_ptr, int32_t* new_pos, int32_t* new_visible,
                                  int32_t* new_doc, int32_t* new_slot, int64_t* totals) {
    try {
        if (n_seqs < 1) return fail(KVLINK_ERR_INVALID_ARG, "n_seqs must be >= 1");
        if (!seq_doc_ptr || !n_query)
            return fail(KVLINK_ERR_INVALID_ARG, "seq_doc_ptr and n_query are required");
        if (seq_doc_ptr[0] != 0) return fail(KVLINK_ERR_LAYOUT, "seq_doc_ptr[0] must be 0");
        for (int s = 0; s < n_seqs; ++s)
            if (seq_doc_ptr[s + 1] < seq_doc_ptr[s])
                return fail(KVLINK_ERR_LAYOUT, "seq_doc_ptr decreases at request %d", s);
        const int64_t n_docs = seq_doc_ptr[n_seqs];
        if (n_docs > 0 && (!doc_len || !link_count))
            return fail(KVLINK_ERR_INVALID_ARG, "doc_len and link_count are required");
        for (int64_t i = 0; i < n_docs; ++i) {
            if (doc_len[i] < 1) return fail(KVLINK_ERR_LAYOUT, "doc_len[%lld] < 1", (long long)i);
            if (link_count[i] < 0)
                return fail(KVLINK_ERR_LAYOUT, "link_count[%lld] < 0", (long long)i);
        }
        int64_t n_new = 0, max_doc = 0, max_cached = 0, max_new_s = 0, max_total = 0;
        for (int s = 0; s < n_seqs; ++s) {
            if (n_query[s] < 0) return fail(KVLINK_ERR_LAYOUT, "n_query[%d] < 0", s);
            int64_t tc = 0, nn = n_query[s];
            for (int64_t i = seq_doc_ptr[s]; i < seq_doc_ptr[s + 1]; ++i) {
                tc += doc_len[i];
                nn += link_count[i];
                max_doc = std::max<int64_t>(max_doc, doc_len[i]);
            }
            if (tc + nn > INT32_MAX)
                return fail(KVLINK_ERR_LAYOUT, "request %d has more than 2^31-1 positions", s);
            n_new += nn;
            max_cached = std::max(max_cached, tc);
            max_new_s = std::max(max_new_s, nn);
            max_total = std::max(max_total, tc + nn);
        }
        if (n_new > INT32_MAX) return fail(KVLINK_ERR_LAYOUT, "more than 2^31-1 new tokens");

        // Sec. 2.3: each document is followed by its K link tokens; the query
        // tokens come after the last document (Sec. 2.1).
        int64_t nidx = 0;
        for (int s = 0; s < n_seqs; ++s) {
            if (seq_new_ptr) seq_new_ptr[s] = (int32_t)nidx;
            int64_t pos = 0, row = 0;
            const int64_t d0 = seq_doc_ptr[s], d1 = seq_doc_ptr[s + 1];
            for (int64_t i = d0; i < d1; ++i) {
                const int64_t g = pos;              // global offset of the document
                if (doc_pos0) doc_pos0[i] = (int32_t)g;
                if (spans) {
                    kvlink_span sp;
                    sp.src_seq = doc_src_seq ? doc_src_seq[i] : 0;
                    sp.src_row = doc_src_row ? doc_src_row[i] : (int32_t)row;
                    sp.dst_seq = s;
                    sp.dst_row = (int32_t)row;
                    sp.len = doc_len[i];
                    sp.delta = (int32_t)(g - (doc_src_pos0 ? doc_src_pos0[i] : 0));
                    spans[i] = sp;
                }
                pos += doc_len[i];
                row += doc_len[i];
                for (int k = 0; k < link_count[i]; ++k, ++pos, ++nidx) {
                    // a link token sees every cached row up to its own document
                    if (new_pos) new_pos[nidx] = (int32_t)pos;
                    if (new_visible) new_visible[nidx] = (int32_t)row;
                    if (new_doc) new_doc[nidx] = (int32_t)(i - d0);
                    if (new_slot) new_slot[nidx] = k;
                }
            }
            if (seq_cached) seq_cached[s] = (int32_t)row;
            for (int q = 0; q < n_query[s]; ++q, ++pos, ++nidx) {
                if (new_pos) new_pos[nidx] = (int32_t)pos;
                if (new_visible) new_visible[nidx] = (int32_t)row;
                if (new_doc) new_doc[nidx] = -1;
                if (new_slot) new_slot[nidx] = q;
            }
        }
        if (seq_new_ptr) seq_new_ptr[n_seqs] = (int32_t)nidx;
        if (totals) {
            totals[0] = n_docs;
            totals[1] = n_new;
            totals[2] = max_doc;
            totals[3] = max_cached;
            totals[4] = max_new_s;
            totals[5] = max_total;
        }
        return ok();
    } catch (...) {
        return fail(KVLINK_ERR_INVALID_ARG, "unexpected exception in kvlink_build_layout");
    }
}

namespace {
kvlink_status rotate_keys(const char* name, bool per_token, kvlink_dtype dtype, int32_t n_layers,
                          int32_t n_kv_heads, int32_t head_dim, double rope_theta, int32_t n_spans,
                          const kvlink_span* d_spans, int32_t max_span_len, kvlink_kv_view src,
                          kvlink_kv_view dst, void* stream, const int32_t* pos_map = nullptr,
                          int64_t pos_stride = 0) {
    try {
        if (!dtype_ok(dtype)) return fail(KVLINK_ERR_UNSUPPORTED, "unknown dtype %d", (int)dtype);
        if (head_dim != 64 && head_dim != 128)
            return fail(KVLINK_ERR_UNSUPPORTED, "head_dim %d (built: 64, 128)", head_dim);
        if (n_layers < 1 || n_kv_heads < 1)
            return fail(KVLINK_ERR_INVALID_ARG, "n_layers and n_kv_heads must be >= 1");
        if (n_spans < 0 || max_span_len < 0)
            return fail(KVLINK_ERR_INVALID_ARG, "n_spans and max_span_len must be >= 0");
        if (!(rope_theta > 0.0) || !std::isfinite(rope_theta))
            return fail(KVLINK_ERR_INVALID_ARG, "rope_theta must be positive and finite");
        if (n_spans > 65535) return fail(KVLINK_ERR_UNSUPPORTED, "more than 65535 spans");
        if ((int64_t)n_layers * n_kv_heads > (int64_t)8 * 65535)
            return fail(KVLINK_ERR_UNSUPPORTED, "too many layers x heads");
        if (n_spans == 0 || max_span_len == 0) return ok();
        if (!d_spans) return fail(KVLINK_ERR_INVALID_ARG, "d_spans is NULL");
        kvlink_status st = check_view(src, dtype, "src");
        if (st != KVLINK_OK) return st;
        if ((st = check_view(dst, dtype, "dst")) != KVLINK_OK) return st;
        hipError_t e = kvlink::launch_reencode(dtype, head_dim, n_layers, n_kv_heads,
                                               kvlink::make_rope_freqs(rope_theta, head_dim),
                                               n_spans, d_spans, max_span_len, to_view(src),
                                               to_view(dst),
                                               per_token ? kvlink::kReencodePerToken
                                                         : kvlink::kReencodeDelta,
                                               reinterpret_cast<hipStream_t>(stream), pos_map,
                                               pos_stride);
        if (e != hipSuccess) return fail(KVLINK_ERR_HIP, "%s launch: %s", name, hipGetErrorString(e));
        return ok();
    } catch (...) {
        return fail(KVLINK_ERR_HIP, "unexpected exception in %s", name);
    }
}
}  // namespace

kvlink_status kvlink_group_spans(int32_t n_spans, const kvlink_span* h_spans, int32_t max_group,
                                 int32_t* h_order, int32_t* h_group_ptr, int32_t* n_groups) {
    try {
        if (n_spans < 0) return fail(KVLINK_ERR_INVALID_ARG, "n_spans < 0");
        if (max_group < 0) return fail(KVLINK_ERR_INVALID_ARG, "max_group < 0");
        if (!n_groups || (n_spans > 0 && (!h_spans || !h_order || !h_group_ptr)))
            return fail(KVLINK_ERR_INVALID_ARG, "a required pointer is NULL");
        // stable order by (src_seq, src_row, len): spans reading the same
        // stored rows become neighbours, each group in span order
        std::vector<int32_t> order((size_t)n_spans);
        for (int32_t i = 0; i < n_spans; ++i) order[(size_t)i] = i;
        auto key = [&](int32_t i) {
            const kvlink_span& sp = h_spans[i];
            return std::make_tuple(sp.src_seq, sp.src_row, sp.len);
        };
        std::stable_sort(order.begin(), order.end(),
                         [&](int32_t a, int32_t b) { return key(a) < key(b); });
        for (int32_t i = 0; i < n_spans; ++i) h_order[i] = order[(size_t)i];
        // runs of equal keys, each cut into ceil(n / max_group) groups whose
        // sizes differ by at most one
        int32_t g = 0;
        if (h_group_ptr) h_group_ptr[0] = 0;
        for (int32_t i = 0; i < n_spans;) {
            int32_t j = i + 1;
            while (j < n_spans && key(order[(size_t)j]) == key(order[(size_t)i])) ++j;
            const int32_t n = j - i;
            const int32_t parts = max_group > 0 ? (n + max_group - 1) / max_group : 1;
            for (int32_t k = 1; k <= parts; ++k)
                h_group_ptr[++g] = i + (int32_t)((int64_t)n * k / parts);
            i = j;
        }
        *n_groups = g;
        return ok();
    } catch (...) {
        return fail(KVLINK_ERR_INVALID_ARG, "unexpected exception in kvlink_group_spans");
    }
}

kvlink_status kvlink_reencode_keys_shared(kvlink_dtype dtype, int32_t n_layers,
                                          int32_t n_kv_heads, int32_t head_dim, double rope_theta,
                                          int32_t n_groups, const int32_t* d_group_ptr,
                                          const kvlink_span* d_spans, int32_t max_span_len,
                                          kvlink_kv_view src, kvlink_kv_view dst, void* stream) {
    try {
        if (!dtype_ok(dtype)) return fail(KVLINK_ERR_UNSUPPORTED, "unknown dtype %d", (int)dtype);
        if (head_dim != 64 && head_dim != 128)
            return fail(KVLINK_ERR_UNSUPPORTED, "head_dim %d (built: 64, 128)", head_dim);
        if (n_layers < 1 || n_kv_heads < 1)
            return fail(KVLINK_ERR_INVALID_ARG, "n_layers and n_kv_heads must be >= 1");
        if (n_groups < 0 || max_span_len < 0)
            return fail(KVLINK_ERR_INVALID_ARG, "n_groups and max_span_len must be >= 0");
        if (!(rope_theta > 0.0) || !std::isfinite(rope_theta))
            return fail(KVLINK_ERR_INVALID_ARG, "rope_theta must be positive and finite");
        if (n_groups > 65535) return fail(KVLINK_ERR_UNSUPPORTED, "more than 65535 groups");
        if ((int64_t)n_layers * n_kv_heads > (int64_t)8 * 65535)
            return fail(KVLINK_ERR_UNSUPPORTED, "too many layers x heads");
        if (n_groups == 0 || max_span_len == 0) return ok();
        if (!d_spans || !d_group_ptr)
            return fail(KVLINK_ERR_INVALID_ARG, "d_spans and d_group_ptr are required");
        kvlink_status st = check_view(src, dtype, "src");
        if (st != KVLINK_OK) return st;
        if ((st = check_view(dst, dtype, "dst")) != KVLINK_OK) return st;
        if (src.base == dst.base)
            return fail(KVLINK_ERR_INVALID_ARG, "src and dst must be different buffers");
        hipError_t e = kvlink::launch_reencode_shared(
            dtype, head_dim, n_layers, n_kv_heads, kvlink::make_rope_freqs(rope_theta, head_dim),
            n_groups, d_group_ptr, d_spans, max_span_len, to_view(src), to_view(dst),
            reinterpret_cast<hipStream_t>(stream));
        if (e != hipSuccess)
            return fail(KVLINK_ERR_HIP, "kvlink_reencode_keys_shared launch: %s",
                        hipGetErrorString(e));
        return ok();
    } catch (...) {
        return fail(KVLINK_ERR_HIP, "unexpected exception in kvlink_reencode_keys_shared");
    }
}

kvlink_status kvlink_reencode_keys(kvlink_dtype dtype, int32_t n_layers, int32_t n_kv_heads,
                                   int32_t head_dim, double rope_theta, int32_t n_spans,
                                   const kvlink_span* d_spans, int32_t max_span_len,
                                   kvlink_kv_view src, kvlink_kv_view dst, void* stream) {
    return rotate_keys("kvlink_reencode_keys", false, dtype, n_layers, n_kv_heads, head_dim,
                       rope_theta, n_spans, d_spans, max_span_len, src, dst, stream);
}

kvlink_status kvlink_reencode_keys_mapped(kvlink_dtype dtype, int32_t n_layers,
                                          int32_t n_kv_heads, int32_t head_dim, double rope_theta,
                                          int32_t n_spans, const kvlink_span* d_spans,
                                          int32_t max_span_len, const int32_t* d_stored_pos,
                                          int64_t stored_pos_stride, kvlink_kv_view src,
                                          kvlink_kv_view dst, void* stream) {
    if (n_spans > 0 && max_span_len > 0 && !d_stored_pos)
        return fail(KVLINK_ERR_INVALID_ARG, "d_stored_pos is NULL");
    if (stored_pos_stride < 0)
        return fail(KVLINK_ERR_INVALID_ARG, "stored_pos_stride must be >= 0");
    return rotate_keys("kvlink_reencode_keys_mapped", true, dtype, n_layers, n_kv_heads, head_dim,
                       rope_theta, n_spans, d_spans, max_span_len, src, dst, stream, d_stored_pos,
                       stored_pos_stride);
}

kvlink_status kvlink_encode_keys_at_positions(kvlink_dtype dtype, int32_t n_layers,
                                              int32_t n_kv_heads, int32_t head_dim,
                                              double rope_theta, int32_t n_spans,
                                              const kvlink_span* d_spans, int32_t max_span_len,
                                              kvlink_kv_view src, kvlink_kv_view dst,
                                              void* stream) {
    return rotate_keys("kvlink_encode_keys_at_positions", true, dtype, n_layers, n_kv_heads,
                       head_dim, rope_theta, n_spans, d_spans, max_span_len, src, dst, stream);
}

size_t kvlink_load_stage_bytes(kvlink_dtype dtype, int32_t n_kv_heads, int32_t head_dim,
                               int32_t stored_rows, int32_t n_slots) {
    if (!dtype_ok(dtype) || n_kv_heads < 1 || head_dim < 1 || stored_rows < 1 || n_slots < 2)
        return 0;
    return (size_t)n_slots * 2 * n_kv_heads * stored_rows * head_dim * elem_size(dtype);
}

}  // extern "C"

namespace {

// HIP events of the staged load, created on first use and kept for the life
// of the calling thread, one set per device.  Re-recording an event is safe
// while earlier waits on it are pending: a wait takes the record that was
// current when it was enqueued.
struct StageEvents {
    int device = -1;
    std::vector<hipEvent_t> ev;   // [0]: entry; then loaded[k], freed[k] for each slot k
};

hipError_t stage_events(int n_slots, hipEvent_t** out) {
    thread_local std::vector<StageEvents> pools;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    StageEvents* pool = nullptr;
    for (StageEvents& p : pools)
        if (p.device == dev) pool = &p;
    if (!pool) {
        pools.push_back(StageEvents());
        pool = &pools.back();
        pool->device = dev;
    }
    const size_t need = 1 + 2 * (size_t)n_slots;
    while (pool->ev.size() < need) {
        hipEvent_t ev = nullptr;
        e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
        if (e != hipSuccess) return e;
        pool->ev.push_back(ev);
    }
    *out = pool->ev.data();
    return hipSuccess;
}

}  // namespace

extern "C" {

kvlink_status kvlink_load_and_reencode(kvlink_dtype dtype, int32_t n_layers, int32_t n_kv_heads,
                                       int32_t head_dim, double rope_theta, int32_t n_spans,
                                       const kvlink_span* d_spans, int32_t max_span_len,
                                       const void* h_k, const void* h_v, int32_t stored_rows,
                                       void* d_stage, size_t stage_bytes, kvlink_kv_view k_dst,
                                       kvlink_kv_view v_dst, int32_t literal, void* copy_stream,
                                       void* compute_stream) {
    try {
        if (!dtype_ok(dtype)) return fail(KVLINK_ERR_UNSUPPORTED, "unknown dtype %d", (int)dtype);
        if (head_dim != 64 && head_dim != 128)
            return fail(KVLINK_ERR_UNSUPPORTED, "head_dim %d (built: 64, 128)", head_dim);
        if (n_layers < 1 || n_kv_heads < 1 || stored_rows < 1)
            return fail(KVLINK_ERR_INVALID_ARG, "n_layers, n_kv_heads and stored_rows must be >= 1");
        if (n_spans < 0 || max_span_len < 0)
            return fail(KVLINK_ERR_INVALID_ARG, "n_spans and max_span_len must be >= 0");
        if (n_spans > 65535) return fail(KVLINK_ERR_UNSUPPORTED, "more than 65535 spans");
        if (n_kv_heads > 8 * 65535) return fail(KVLINK_ERR_UNSUPPORTED, "too many heads");
        if (!(rope_theta > 0.0) || !std::isfinite(rope_theta))
            return fail(KVLINK_ERR_INVALID_ARG, "rope_theta must be positive and finite");
        if (literal != 0 && literal != 1) return fail(KVLINK_ERR_INVALID_ARG, "literal must be 0 or 1");
        if (!h_k || !h_v) return fail(KVLINK_ERR_INVALID_ARG, "h_k or h_v is NULL");
        if (n_spans > 0 && max_span_len > 0 && !d_spans)
            return fail(KVLINK_ERR_INVALID_ARG, "d_spans is NULL");
        // a slot holds one layer's stored keys and values
        const size_t slot_bytes = kvlink_load_stage_bytes(dtype, n_kv_heads, head_dim, stored_rows, 2) / 2;
        if (d_stage && reinterpret_cast<uintptr_t>(d_stage) % 256)
            return fail(KVLINK_ERR_WORKSPACE, "d_stage is not 256-byte aligned");
        if (d_stage && stage_bytes < 2 * slot_bytes)
            return fail(KVLINK_ERR_WORKSPACE, "d_stage has %zu bytes, needs at least %zu (two slots)",
                        stage_bytes, 2 * slot_bytes);
        kvlink_status st = check_view(k_dst, dtype, "k_dst");
        if (st != KVLINK_OK) return st;
        if ((st = check_view(v_dst, dtype, "v_dst")) != KVLINK_OK) return st;
        if (reinterpret_cast<uintptr_t>(h_k) % 16 || reinterpret_cast<uintptr_t>(h_v) % 16)
            return fail(KVLINK_ERR_INVALID_ARG, "h_k or h_v is not 16-byte aligned");

        const size_t es = elem_size(dtype);
        const size_t layer_bytes = slot_bytes / 2;
        hipStream_t cs = reinterpret_cast<hipStream_t>(copy_stream);
        hipStream_t ks = reinterpret_cast<hipStream_t>(compute_stream);
        const kvlink::RopeFreqs freqs = kvlink::make_rope_freqs(rope_theta, head_dim);
        const bool work = n_spans > 0 && max_span_len > 0;
        const int rot = literal ? kvlink::kReencodePerToken : kvlink::kReencodeDelta;
        // the stored caches as a view: [layer][n_kv_heads][stored_rows][head_dim]
        auto stored_view = [&](const void* base, int64_t layer_stride) {
            kvlink::View v;
            v.base = reinterpret_cast<char*>(const_cast<void*>(base));
            v.layer_stride = layer_stride;
            v.head_stride = (int64_t)stored_rows * head_dim;
            v.row_stride = head_dim;
            v.seq_stride = 0;
            v.page_stride = 0;
            v.block_table = nullptr;
            v.page_size = 1;
            v.max_pages = 0;
            return v;
        };

        if (!d_stage) {
            // Direct: the kernels read the pinned host arrays over the bus
            // (their device mapping), all layers in one re-encode launch and
            // one value-gather launch on compute_stream.  Memory that is not
            // mapped for the device is refused before any launch.
            void* dk = nullptr;
            void* dv = nullptr;
            if (hipHostGetDevicePointer(&dk, const_cast<void*>(h_k), 0) != hipSuccess || !dk ||
                hipHostGetDevicePointer(&dv, const_cast<void*>(h_v), 0) != hipSuccess || !dv) {
                (void)hipGetLastError();
                return fail(KVLINK_ERR_INVALID_ARG,
                            "h_k or h_v is not pinned host memory mapped for the device "
                            "(allocate it with hipHostMalloc) and no staging area was given");
            }
            if (!work) return ok();
            const int64_t ls = (int64_t)n_kv_heads * stored_rows * head_dim;
            hipError_t e = kvlink::launch_reencode(dtype, head_dim, n_layers, n_kv_heads, freqs,
                                                   n_spans, d_spans, max_span_len,
                                                   stored_view(dk, ls), to_view(k_dst), rot, ks);
            if (e == hipSuccess)
                e = kvlink::launch_reencode(dtype, head_dim, n_layers, n_kv_heads, freqs, n_spans,
                                            d_spans, max_span_len, stored_view(dv, ls),
                                            to_view(v_dst), kvlink::kReencodeCopy, ks);
            if (e != hipSuccess)
                return fail(KVLINK_ERR_HIP, "kvlink_load_and_reencode: %s", hipGetErrorString(e));
            return ok();
        }

        // Staged: the staging area holds `cap` layers (at least two); they
        // form a ring of chunks of G consecutive layers, G as large as a
        // copy of at least kMinCopyBytes of keys needs while the ring keeps
        // at least two chunks.  Chunk c (layers [cG, cG + G)) goes to ring
        // entry c % n_ring as one keys copy and one values copy (the host
        // arrays are layer-major, so a chunk is contiguous in each); its
        // copy waits until the re-encode of chunk c - n_ring has released
        // the entry, and its re-encode (one launch for the chunk's layers)
        // waits for its copy.  Few large copies: each copy and each
        // cross-stream wait carries a fixed cost.
        constexpr size_t kMinCopyBytes = 64u << 20;
        const int cap = (int)std::min<size_t>((size_t)n_layers, stage_bytes / slot_bytes);
        const int G = std::max(1, std::min<int>(
                                      (int)((kMinCopyBytes + layer_bytes - 1) / layer_bytes),
                                      cap / 2));
        const int n_ring = cap / G;
        const size_t chunk_bytes = (size_t)G * layer_bytes;   // keys (or values) of a chunk
        const int64_t ls = (int64_t)n_kv_heads * stored_rows * head_dim;
        auto layer_of = [&](const kvlink_kv_view& v, int l) {
            kvlink::View d = to_view(v);
            d.base += (int64_t)l * v.layer_stride * (int64_t)es;
            return d;
        };
        const bool two = cs != ks;
        hipEvent_t* ev = nullptr;
        hipError_t e = two ? stage_events(n_ring, &ev) : hipSuccess;
        // the first copies reuse entries that the re-encodes of an earlier
        // call on compute_stream may still be reading
        if (two && e == hipSuccess) e = hipEventRecord(ev[0], ks);
        if (two && e == hipSuccess) e = hipStreamWaitEvent(cs, ev[0], 0);
        const int n_chunks = (n_layers + G - 1) / G;
        for (int c = 0; c < n_chunks && e == hipSuccess; ++c) {
            const int l0 = c * G, nl = std::min(G, n_layers - l0);
            const int slot = c % n_ring;
            hipEvent_t loaded = two ? ev[1 + 2 * slot] : nullptr;
            hipEvent_t freed = two ? ev[2 + 2 * slot] : nullptr;
            char* k_slot = reinterpret_cast<char*>(d_stage) + (size_t)slot * 2 * chunk_bytes;
            char* v_slot = k_slot + chunk_bytes;
            if (two && c >= n_ring) e = hipStreamWaitEvent(cs, freed, 0);
            if (e == hipSuccess)
                e = hipMemcpyAsync(k_slot, reinterpret_cast<const char*>(h_k) + l0 * layer_bytes,
                                   (size_t)nl * layer_bytes, hipMemcpyHostToDevice, cs);
            if (e == hipSuccess)
                e = hipMemcpyAsync(v_slot, reinterpret_cast<const char*>(h_v) + l0 * layer_bytes,
                                   (size_t)nl * layer_bytes, hipMemcpyHostToDevice, cs);
            if (two && e == hipSuccess) e = hipEventRecord(loaded, cs);
            if (two && e == hipSuccess) e = hipStreamWaitEvent(ks, loaded, 0);
            if (e == hipSuccess && work)
                e = kvlink::launch_reencode(dtype, head_dim, nl, n_kv_heads, freqs, n_spans,
                                            d_spans, max_span_len, stored_view(k_slot, ls),
                                            layer_of(k_dst, l0), rot, ks);
            if (e == hipSuccess && work)
                e = kvlink::launch_reencode(dtype, head_dim, nl, n_kv_heads, freqs, n_spans,
                                            d_spans, max_span_len, stored_view(v_slot, ls),
                                            layer_of(v_dst, l0), kvlink::kReencodeCopy, ks);
            if (two && e == hipSuccess) e = hipEventRecord(freed, ks);
        }
        if (e != hipSuccess)
            return fail(KVLINK_ERR_HIP, "kvlink_load_and_reencode: %s", hipGetErrorString(e));
        return ok();
    } catch (...) {
        return fail(KVLINK_ERR_HIP, "unexpected exception in kvlink_load_and_reencode");
    }
}

kvlink_status kvlink_attend_make_plan(kvlink_dtype dtype, int32_t n_q_heads, int32_t n_kv_heads,
                                      int32_t head_dim, int32_t n_seqs,
                                      const int32_t* seq_new_ptr, const int32_t* seq_cached,
                                      const int32_t* new_visible,
                                      int32_t n_compute_units, int32_t n_workgroups,
                                      int32_t row_block, uint32_t flags, int32_t* table,
                                      int64_t table_capacity, kvlink_attend_plan* plan) {
    try {
        if (!dtype_ok(dtype)) return fail(KVLINK_ERR_UNSUPPORTED, "unknown dtype %d", (int)dtype);
        if (head_dim != 64 && head_dim != 128)
            return fail(KVLINK_ERR_UNSUPPORTED, "head_dim %d (built: 64, 128)", head_dim);
        if (n_q_heads < 1 || n_kv_heads < 1 || n_q_heads % n_kv_heads)
            return fail(KVLINK_ERR_INVALID_ARG, "n_q_heads must be a positive multiple of n_kv_heads");
        const int group = n_q_heads / n_kv_heads;
        if (group != 1 && group != 2 && group != 4 && group != 8)
            return fail(KVLINK_ERR_UNSUPPORTED, "GQA group %d (built: 1, 2, 4, 8)", group);
        if (n_seqs < 1) return fail(KVLINK_ERR_INVALID_ARG, "n_seqs must be >= 1");
        if (!seq_new_ptr || !seq_cached || !new_visible || !plan)
            return fail(KVLINK_ERR_INVALID_ARG,
                        "seq_new_ptr, seq_cached, new_visible and plan are required");
        if (n_compute_units < 1) return fail(KVLINK_ERR_INVALID_ARG, "n_compute_units must be >= 1");
        if (n_workgroups < 0) return fail(KVLINK_ERR_INVALID_ARG, "n_workgroups must be >= 0");
        if (row_block < 0) return fail(KVLINK_ERR_INVALID_ARG, "row_block must be >= 0");
        if (flags & ~(uint32_t)(KVLINK_PLAN_XCD | KVLINK_PLAN_COMBINE | KVLINK_PLAN_IN_LAUNCH))
            return fail(KVLINK_ERR_INVALID_ARG, "unknown plan flags 0x%x", (unsigned)flags);
        if ((flags & KVLINK_PLAN_COMBINE) && (flags & KVLINK_PLAN_IN_LAUNCH))
            return fail(KVLINK_ERR_INVALID_ARG, "KVLINK_PLAN_COMBINE and KVLINK_PLAN_IN_LAUNCH exclude each other");
        std::vector<int32_t> tab;
        kvlink::PlanCounts c;
        const char* why = "";
        const int st = kvlink::build_attend_schedule(dtype, n_q_heads, n_kv_heads, head_dim, n_seqs,
                                                     seq_new_ptr, seq_cached, new_visible,
                                                     n_compute_units, n_workgroups, row_block,
                                                     flags, table ? &tab : nullptr, &c, &why);
        if (st != KVLINK_OK) return fail((kvlink_status)st, "%s", why);
        if (c.table_len > INT32_MAX) return fail(KVLINK_ERR_LAYOUT, "schedule table too large");
        if (table) {
            if (table_capacity < c.table_len)
                return fail(KVLINK_ERR_INVALID_ARG, "table holds %lld entries, needs %lld",
                            (long long)table_capacity, (long long)c.table_len);
            std::copy(tab.begin(), tab.end(), table);
        }
        plan->table = nullptr;
        plan->table_len = (int32_t)c.table_len;
        plan->n_workgroups = c.n_wg;
        plan->n_units = c.n_units;
        plan->n_segments = c.n_segments;
        plan->row_block = c.row_block;
        plan->n_seqs = n_seqs;
        plan->n_split_units = c.n_split;
        plan->flags = (flags & ~(uint32_t)(KVLINK_PLAN_COMBINE | KVLINK_PLAN_IN_LAUNCH)) |
                      (c.in_launch ? KVLINK_PLAN_IN_LAUNCH : KVLINK_PLAN_COMBINE);
        plan->rope_table = nullptr;
        return ok();
    } catch (...) {
        return fail(KVLINK_ERR_INVALID_ARG, "unexpected exception in kvlink_attend_make_plan");
    }
}

size_t kvlink_attend_workspace_bytes(kvlink_dtype dtype, int32_t n_q_heads, int32_t n_kv_heads,
                                     int32_t head_dim, int32_t n_new_total,
                                     const kvlink_attend_plan* plan) {
    if (!dtype_ok(dtype) || !plan) return 0;
    kvlink::AttendPlan p;
    if (!kvlink::make_attend_plan(dtype, n_q_heads, n_kv_heads, head_dim, n_new_total, *plan, &p))
        return 0;
    return p.total_bytes;
}

}  // extern "C"

namespace {

// ------------------------------------------------ allocation-free attention

// Device memory of kvlink_attend_new_tokens_noalloc: one copy per GPU, held
// from the library's load until the process ends.  In host code `scratch`
// names a host-side stand-in; the device address of each GPU's copy comes
// from hipGetSymbolAddress and is the only form passed to kernels.
__device__ __align__(256) unsigned char scratch[KVLINK_NOALLOC_SCRATCH_BYTES];

std::mutex g_scratch_mu;
std::vector<void*> g_scratch_dev;   // per device id: its copy of scratch, NULL until looked up

// The current device's copy of scratch, looked up on the first call on that
// device (with it current) and kept.
hipError_t current_scratch(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if ((int)g_scratch_dev.size() <= dev) g_scratch_dev.resize((size_t)dev + 1, nullptr);
    if (!g_scratch_dev[(size_t)dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        g_scratch_dev[(size_t)dev] = p;
    }
    *out = g_scratch_dev[(size_t)dev];
    return hipSuccess;
}

kvlink_status attend_impl(
    kvlink_dtype dtype, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
    double rope_theta, float softmax_scale, int32_t n_seqs, int32_t n_new_total,
    int32_t max_new, int32_t max_cached, const int32_t* d_seq_new_ptr,
    const int32_t* d_seq_cached, const int32_t* d_new_pos, const int32_t* d_new_visible,
    const void* q_new, const void* k_new, const void* v_new, kvlink_kv_view k_cache,
    kvlink_kv_view v_cache, int32_t layer, void* out, float* lse, kvlink_attend_plan sched,
    void* workspace, size_t workspace_bytes, void* stream, uint32_t stages, bool noalloc,
    const kvlink_span* fuse_spans = nullptr, const int32_t* fuse_span_ptr = nullptr) {
    try {
        const uint32_t all = KVLINK_STAGE_ROPE | KVLINK_STAGE_SPLIT | KVLINK_STAGE_COMBINE;
        if (stages == 0 || (stages & ~all))
            return fail(KVLINK_ERR_INVALID_ARG, "stage mask %u", (unsigned)stages);
        if (!dtype_ok(dtype)) return fail(KVLINK_ERR_UNSUPPORTED, "unknown dtype %d", (int)dtype);
        if (head_dim != 64 && head_dim != 128)
            return fail(KVLINK_ERR_UNSUPPORTED, "head_dim %d (built: 64, 128)", head_dim);
        if (n_q_heads < 1 || n_kv_heads < 1 || n_q_heads % n_kv_heads)
            return fail(KVLINK_ERR_INVALID_ARG, "n_q_heads must be a positive multiple of n_kv_heads");
        const int group = n_q_heads / n_kv_heads;
        if (group != 1 && group != 2 && group != 4 && group != 8)
            return fail(KVLINK_ERR_UNSUPPORTED, "GQA group %d (built: 1, 2, 4, 8)", group);
        if (n_seqs < 1 || n_new_total < 0 || max_new < 0 || max_cached < 0 || layer < 0)
            return fail(KVLINK_ERR_INVALID_ARG, "negative size or layer");
        if (n_new_total > 0 && max_new < 1)
            return fail(KVLINK_ERR_INVALID_ARG, "max_new must be >= 1 when there are new tokens");
        if ((int64_t)max_new > n_new_total)
            return fail(KVLINK_ERR_INVALID_ARG, "max_new exceeds n_new_total");
        if (!(rope_theta > 0.0) || !std::isfinite(rope_theta))
            return fail(KVLINK_ERR_INVALID_ARG, "rope_theta must be positive and finite");
        if (!(softmax_scale > 0.f) || !std::isfinite(softmax_scale))
            return fail(KVLINK_ERR_INVALID_ARG, "softmax_scale must be positive and finite");
        if (n_new_total == 0) return ok();
        if (!sched.table) return fail(KVLINK_ERR_INVALID_ARG, "plan.table is NULL");
        if (reinterpret_cast<uintptr_t>(sched.table) % 16)
            return fail(KVLINK_ERR_INVALID_ARG, "plan.table is not 16-byte aligned");
        if (sched.n_seqs != n_seqs)
            return fail(KVLINK_ERR_INVALID_ARG, "plan is for %d requests, call has %d", sched.n_seqs,
                        n_seqs);
        if (!kvlink::attend_row_block_ok(kvlink::attend_path(dtype, group, max_new), sched.row_block))
            return fail(KVLINK_ERR_INVALID_ARG, "plan row_block %d does not match this call's path",
                        sched.row_block);
        if (!d_seq_new_ptr || !d_seq_cached || !d_new_pos || !d_new_visible)
            return fail(KVLINK_ERR_INVALID_ARG, "a layout descriptor pointer is NULL");
        if (!q_new || !k_new || !v_new || !out)
            return fail(KVLINK_ERR_INVALID_ARG, "q_new, k_new, v_new and out are required");
        if ((reinterpret_cast<uintptr_t>(q_new) | reinterpret_cast<uintptr_t>(k_new) |
             reinterpret_cast<uintptr_t>(v_new)) % 16)
            return fail(KVLINK_ERR_INVALID_ARG, "q_new, k_new and v_new must be 16-byte aligned");
        if (reinterpret_cast<uintptr_t>(sched.rope_table) % 16)
            return fail(KVLINK_ERR_INVALID_ARG, "plan.rope_table is not 16-byte aligned");
        kvlink_status st = check_view(k_cache, dtype, "k_cache");
        if (st != KVLINK_OK) return st;
        if ((st = check_view(v_cache, dtype, "v_cache")) != KVLINK_OK) return st;
        kvlink::AttendPlan plan;
        if (!kvlink::make_attend_plan(dtype, n_q_heads, n_kv_heads, head_dim, n_new_total, sched,
                                      &plan))
            return fail(KVLINK_ERR_INVALID_ARG, "invalid attention sizes or plan counts");
        if (noalloc) {
            // the library's scratch instead of a workspace: refused before any
            // HIP call when the call needs more than it holds
            if (plan.total_bytes > (size_t)KVLINK_NOALLOC_SCRATCH_BYTES)
                return fail(KVLINK_ERR_WORKSPACE,
                            "the call needs %zu bytes of scratch; the allocation-free entry "
                            "point holds %zu (use kvlink_attend_new_tokens with a workspace)",
                            plan.total_bytes, (size_t)KVLINK_NOALLOC_SCRATCH_BYTES);
            hipError_t e = current_scratch(&workspace);
            if (e != hipSuccess)
                return fail(KVLINK_ERR_HIP, "scratch lookup: %s", hipGetErrorString(e));
            workspace_bytes = (size_t)KVLINK_NOALLOC_SCRATCH_BYTES;
        }
        if (!workspace) return fail(KVLINK_ERR_WORKSPACE, "workspace is NULL");
        if (reinterpret_cast<uintptr_t>(workspace) % 256)
            return fail(KVLINK_ERR_WORKSPACE, "workspace is not 256-byte aligned");
        if (workspace_bytes < plan.total_bytes)
            return fail(KVLINK_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", workspace_bytes,
                        plan.total_bytes);
        kvlink::AttendArgs a;
        a.q_new = q_new;
        a.k_new = k_new;
        a.v_new = v_new;
        a.k = to_view(k_cache);
        a.v = to_view(v_cache);
        a.layer = layer;
        a.seq_new_ptr = d_seq_new_ptr;
        a.seq_cached = d_seq_cached;
        a.new_pos = d_new_pos;
        a.new_visible = d_new_visible;
        a.freqs = kvlink::make_rope_freqs(rope_theta, head_dim);
        a.scale = softmax_scale;
        a.out = out;
        a.lse = lse;
        a.workspace = workspace;
        a.rope_table = sched.rope_table;
        a.fuse_spans = fuse_spans;
        a.fuse_span_ptr = fuse_span_ptr;
        hipError_t e =
            kvlink::launch_attend(dtype, plan, a, reinterpret_cast<hipStream_t>(stream), stages);
        if (e != hipSuccess) return fail(KVLINK_ERR_HIP, "attention launch: %s", hipGetErrorString(e));
        return ok();
    } catch (...) {
        return fail(KVLINK_ERR_HIP, "unexpected exception in kvlink_attend_stages");
    }
}

}  // namespace

extern "C" {

kvlink_status kvlink_attend_stages(
    kvlink_dtype dtype, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
    double rope_theta, float softmax_scale, int32_t n_seqs, int32_t n_new_total,
    int32_t max_new, int32_t max_cached, const int32_t* d_seq_new_ptr,
    const int32_t* d_seq_cached, const int32_t* d_new_pos, const int32_t* d_new_visible,
    const void* q_new, const void* k_new, const void* v_new, kvlink_kv_view k_cache,
    kvlink_kv_view v_cache, int32_t layer, void* out, float* lse, kvlink_attend_plan sched,
    void* workspace, size_t workspace_bytes, void* stream, uint32_t stages) {
    return attend_impl(dtype, n_q_heads, n_kv_heads, head_dim, rope_theta, softmax_scale, n_seqs,
                       n_new_total, max_new, max_cached, d_seq_new_ptr, d_seq_cached, d_new_pos,
                       d_new_visible, q_new, k_new, v_new, k_cache, v_cache, layer, out, lse,
                       sched, workspace, workspace_bytes, stream, stages, false);
}

kvlink_status kvlink_attend_new_tokens(
    kvlink_dtype dtype, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
    double rope_theta, float softmax_scale, int32_t n_seqs, int32_t n_new_total,
    int32_t max_new, int32_t max_cached, const int32_t* d_seq_new_ptr,
    const int32_t* d_seq_cached, const int32_t* d_new_pos, const int32_t* d_new_visible,
    const void* q_new, const void* k_new, const void* v_new, kvlink_kv_view k_cache,
    kvlink_kv_view v_cache, int32_t layer, void* out, float* lse, kvlink_attend_plan plan,
    void* workspace, size_t workspace_bytes, void* stream) {
    return kvlink_attend_stages(dtype, n_q_heads, n_kv_heads, head_dim, rope_theta, softmax_scale,
                                n_seqs, n_new_total, max_new, max_cached, d_seq_new_ptr,
                                d_seq_cached, d_new_pos, d_new_visible, q_new, k_new, v_new,
                                k_cache, v_cache, layer, out, lse, plan, workspace,
                                workspace_bytes, stream,
                                KVLINK_STAGE_ROPE | KVLINK_STAGE_SPLIT | KVLINK_STAGE_COMBINE);
}

kvlink_status kvlink_attend_new_tokens_noalloc(
    kvlink_dtype dtype, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
    double rope_theta, float softmax_scale, int32_t n_seqs, int32_t n_new_total,
    int32_t max_new, int32_t max_cached, const int32_t* d_seq_new_ptr,
    const int32_t* d_seq_cached, const int32_t* d_new_pos, const int32_t* d_new_visible,
    const void* q_new, const void* k_new, const void* v_new, kvlink_kv_view k_cache,
    kvlink_kv_view v_cache, int32_t layer, void* out, float* lse, kvlink_attend_plan plan,
    void* stream) {
    return attend_impl(dtype, n_q_heads, n_kv_heads, head_dim, rope_theta, softmax_scale, n_seqs,
                       n_new_total, max_new, max_cached, d_seq_new_ptr, d_seq_cached, d_new_pos,
                       d_new_visible, q_new, k_new, v_new, k_cache, v_cache, layer, out, lse,
                       plan, nullptr, 0, stream,
                       KVLINK_STAGE_ROPE | KVLINK_STAGE_SPLIT | KVLINK_STAGE_COMBINE, true);
}

kvlink_status kvlink_attend_new_tokens_fused(
    kvlink_dtype dtype, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
    double rope_theta, float softmax_scale, int32_t n_seqs, int32_t n_new_total,
    int32_t max_new, int32_t max_cached, const int32_t* d_seq_new_ptr,
    const int32_t* d_seq_cached, const int32_t* d_new_pos, const int32_t* d_new_visible,
    const void* q_new, const void* k_new, const void* v_new, kvlink_kv_view k_cache,
    kvlink_kv_view v_cache, int32_t layer, void* out, float* lse, kvlink_attend_plan plan,
    const kvlink_span* d_spans, const int32_t* d_seq_span_ptr, int32_t max_spans_per_seq,
    void* workspace, size_t workspace_bytes, void* stream) {
    if (max_spans_per_seq < 0) return fail(KVLINK_ERR_INVALID_ARG, "max_spans_per_seq < 0");
    if (max_spans_per_seq > KVLINK_FUSED_MAX_SPANS)
        return fail(KVLINK_ERR_UNSUPPORTED, "%d spans in a request (the fused re-encode holds %d)",
                    max_spans_per_seq, KVLINK_FUSED_MAX_SPANS);
    if (dtype != KVLINK_BF16 || !kvlink::attend_row_block_ok(kvlink::kPathWide, plan.row_block))
        return fail(KVLINK_ERR_UNSUPPORTED,
                    "the fused re-encode runs on the wide bf16 kernel (row_block 256, 128 or 64)");
    if (n_new_total > 0 && (!d_spans || !d_seq_span_ptr))
        return fail(KVLINK_ERR_INVALID_ARG, "d_spans and d_seq_span_ptr are required");
    return attend_impl(dtype, n_q_heads, n_kv_heads, head_dim, rope_theta, softmax_scale, n_seqs,
                       n_new_total, max_new, max_cached, d_seq_new_ptr, d_seq_cached, d_new_pos,
                       d_new_visible, q_new, k_new, v_new, k_cache, v_cache, layer, out, lse,
                       plan, workspace, workspace_bytes, stream,
                       KVLINK_STAGE_ROPE | KVLINK_STAGE_SPLIT | KVLINK_STAGE_COMBINE, false,
                       d_spans, d_seq_span_ptr);
}

kvlink_status kvlink_attend_rope_table(int32_t head_dim, double rope_theta, int32_t n_new_total,
                                       const int32_t* d_new_pos, float* d_table, void* stream) {
    try {
        if (head_dim != 64 && head_dim != 128)
            return fail(KVLINK_ERR_UNSUPPORTED, "head_dim %d (built: 64, 128)", head_dim);
        if (!(rope_theta > 0.0) || !std::isfinite(rope_theta))
            return fail(KVLINK_ERR_INVALID_ARG, "rope_theta must be positive and finite");
        if (n_new_total < 0) return fail(KVLINK_ERR_INVALID_ARG, "n_new_total < 0");
        if (n_new_total == 0) return ok();
        if (!d_new_pos || !d_table)
            return fail(KVLINK_ERR_INVALID_ARG, "d_new_pos and d_table are required");
        if (reinterpret_cast<uintptr_t>(d_table) % 16)
            return fail(KVLINK_ERR_INVALID_ARG, "d_table is not 16-byte aligned");
        hipError_t e = kvlink::launch_rope_table(head_dim, kvlink::make_rope_freqs(rope_theta, head_dim),
                                                 n_new_total, d_new_pos, d_table,
                                                 reinterpret_cast<hipStream_t>(stream));
        if (e != hipSuccess) return fail(KVLINK_ERR_HIP, "rope table launch: %s", hipGetErrorString(e));
        return ok();
    } catch (...) {
        return fail(KVLINK_ERR_HIP, "unexpected exception in kvlink_attend_rope_table");
    }
}

const char* kvlink_last_error(void) { return g_error.c_str(); }

const char* kvlink_version(void) { return "kvlink-gfx950 0.1"; }

}  // extern "C"
