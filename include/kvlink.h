/*
 * kvlink.h — C ABI of the MI355X (gfx950) KVLink inference hot path.
 *
 * KVLink (arXiv 2502.16002) precomputes the KV cache of every document on its
 * own, concatenates the caches of the retrieved documents at inference time,
 * moves their keys to their global positions (Sec. 2.2, positional
 * re-encoding) and runs one forward pass over the link tokens placed after
 * each document and the query tokens (Sec. 2.3).  This library implements the
 * per-layer parts of that path that touch the cache:
 *
 *   kvlink_build_layout       index maps of the concatenated sequence (host)
 *   kvlink_reencode_keys      K' = R(delta_i) K for every cached key (GPU)
 *   kvlink_encode_keys_at_positions
 *                             K' = R(g_i + t) K for keys cached without
 *                             rotation (the paper's literal form, GPU)
 *   kvlink_reencode_keys_mapped
 *                             K' = R(g_i + t - p_t) K for compressed caches
 *                             (kept tokens at original positions p_t, GPU)
 *   kvlink_load_and_reencode  the same, from caches held in host memory: read
 *                             by the kernels over the bus, or copied in
 *                             chunks of layers through a device staging
 *                             ring (GPU)
 *   kvlink_attend_make_plan   balanced split-K schedule of a batch (host)
 *   kvlink_attend_new_tokens  RoPE of the new tokens at their global positions,
 *                             append of their keys/values to the cache and
 *                             split-K GQA attention over the cache (GPU)
 *   kvlink_attend_new_tokens_fused
 *                             the same over the stored keys, re-encoded as
 *                             the attention stages them (GPU)
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  * Every function returns a kvlink_status, never aborts, and lets no C++
 *    exception cross the ABI.  On a non-OK status kvlink_last_error() returns a
 *    message (thread-local, valid until the next call on that thread).
 *  * Host-side validation happens before any HIP call: a call that returns
 *    KVLINK_ERR_INVALID_ARG, KVLINK_ERR_UNSUPPORTED, KVLINK_ERR_LAYOUT or
 *    KVLINK_ERR_WORKSPACE has launched nothing.  KVLINK_ERR_HIP means a launch
 *    failed; the message holds HIP's error string.
 *  * GPU calls are asynchronous on `stream` (a hipStream_t passed as void*;
 *    NULL means the null stream).  The library allocates no device memory and
 *    keeps no state between calls (except the HIP events that the staged
 *    kvlink_load_and_reencode keeps for reuse); the caller owns every
 *    buffer, including the workspace.  Host arrays are only read during the
 *    call.
 *  * Positions are 0-based.  RoPE (Sec. 2.2) rotates each pair
 *    (x_j, x_{j + d/2}), j < d/2, by pos * theta^(-2j/d): the half-split
 *    pairing of the Llama family the paper fine-tunes (Sec. 3.1).  Angles are
 *    formed in double precision on the device and the cos/sin values rounded
 *    to float before the rotation, which runs in float.
 *  * bf16 values are rounded from float with round-to-nearest-even.
 *  * Device descriptor arrays (d_* arguments) are not re-validated on the
 *    device; they must be the uploaded outputs of kvlink_build_layout for the
 *    same request batch.
 */
#ifndef KVLINK_H
#define KVLINK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    KVLINK_OK = 0,
    KVLINK_ERR_INVALID_ARG = 1, /* null pointer, bad scalar, misaligned buffer */
    KVLINK_ERR_UNSUPPORTED = 2, /* head_dim, dtype or GQA group not built      */
    KVLINK_ERR_LAYOUT = 3,      /* inconsistent lengths, counts or positions    */
    KVLINK_ERR_WORKSPACE = 4,   /* workspace missing or too small               */
    KVLINK_ERR_HIP = 5          /* a HIP launch failed                          */
} kvlink_status;

typedef enum { KVLINK_F32 = 0, KVLINK_BF16 = 1 } kvlink_dtype;

/*
 * A K or V tensor covering all layers, on the device.  Element j (0 <= j <
 * head_dim, always unit stride) of row `row` of KV head `head` of sequence
 * `seq` in layer `layer` is at
 *
 *   contiguous (block_table == NULL):
 *     base + layer*layer_stride + head*head_stride + seq*seq_stride
 *          + row*row_stride + j
 *   paged (block_table != NULL):
 *     base + layer*layer_stride + head*head_stride
 *          + block_table[seq*max_pages + row/page_size]*page_stride
 *          + (row % page_size)*row_stride + j
 *
 * Strides are in elements.  base must be 16-byte aligned and every stride a
 * multiple of 16 bytes.  The block table is a device array of int32 physical
 * page numbers.
 */
typedef struct {
    void* base;
    int64_t layer_stride;
    int64_t head_stride;
    int64_t row_stride;
    int64_t seq_stride;
    int64_t page_stride;
    const int32_t* block_table;
    int32_t page_size;
    int32_t max_pages;
} kvlink_kv_view;

/*
 * One stored document cache to re-encode (Sec. 2.2): `len` rows starting at
 * row src_row of sequence src_seq of the source view go, rotated by
 * R(delta), to rows dst_row.. of sequence dst_seq of the destination view.
 * delta = g_i - src_pos0_i, the document's global offset after
 * concatenation minus the position its keys were rotated at when cached.
 */
typedef struct {
    int32_t src_seq;
    int32_t src_row;
    int32_t dst_seq;
    int32_t dst_row;
    int32_t len;
    int32_t delta;
} kvlink_span;

/*
 * kvlink_build_layout — index maps of a batch of requests (host, integer,
 * bit-exact).  Follows the layout of Sec. 2.1 and Sec. 2.3: in request s the
 * retrieved documents come in retrieval order, each as
 * (c_1..c_L, link_1..link_K), and the query tokens follow.  The link tokens
 * of the n-th document are link_n-1..link_n-K (Appendix A.2).
 *
 * Inputs (host arrays):
 *   n_seqs                 number of requests (>= 1)
 *   seq_doc_ptr[n_seqs+1]  request s owns documents seq_doc_ptr[s]..seq_doc_ptr[s+1]-1
 *                          (non-decreasing, seq_doc_ptr[0] == 0)
 *   doc_len[n_docs]        L_i >= 1, rows of each document's stored cache
 *   link_count[n_docs]     K_i >= 0, link tokens after each document
 *   n_query[n_seqs]        query tokens of each request, >= 0
 *   doc_src_seq[n_docs]    source sequence of each stored cache (NULL: 0)
 *   doc_src_row[n_docs]    first row of it in that sequence (NULL: the
 *                          documents of each request stored back to back,
 *                          i.e. the same rows as in the destination)
 *   doc_src_pos0[n_docs]   position its keys were rotated at (NULL: 0)
 *
 * Outputs (host arrays sized by the caller; any may be NULL to skip it):
 *   spans[n_docs]          re-encode descriptors (dst_seq = s, dst_row = first
 *                          row of the document in the request's concatenated
 *                          cache, rows of a request's documents back to back
 *                          in retrieval order)
 *   doc_pos0[n_docs]       global position g_i of each document's first token
 *   seq_cached[n_seqs]     T_c: cached rows of each request
 *   seq_new_ptr[n_seqs+1]  request s owns new tokens seq_new_ptr[s]..seq_new_ptr[s+1]-1
 *   new_pos[n_new]         global position of each new token; within a
 *                          request the new tokens are the link tokens in
 *                          document order, then the query tokens, so the
 *                          positions increase
 *   new_visible[n_new]     cached rows visible to the new token: the rows of
 *                          every document at or before its own (all T_c for
 *                          query tokens); the token also sees the new tokens
 *                          of its request up to and including itself
 *   new_doc[n_new]         document index within the request, -1 for queries
 *   new_slot[n_new]        link index k (0-based) or query index
 *   totals[6]              n_docs, n_new, max doc_len, max T_c, max new
 *                          tokens per request, max total positions per request
 *
 * Errors: KVLINK_ERR_INVALID_ARG for a null required input or n_seqs < 1;
 * KVLINK_ERR_LAYOUT for a length < 1, a negative count, a non-monotone
 * seq_doc_ptr, or a position that would not fit in int32.
 */
kvlink_status kvlink_build_layout(int32_t n_seqs, const int32_t* seq_doc_ptr,
                                  const int32_t* doc_len, const int32_t* link_count,
                                  const int32_t* n_query, const int32_t* doc_src_seq,
                                  const int32_t* doc_src_row, const int32_t* doc_src_pos0,
                                  kvlink_span* spans, int32_t* doc_pos0, int32_t* seq_cached,
                                  int32_t* seq_new_ptr, int32_t* new_pos, int32_t* new_visible,
                                  int32_t* new_doc, int32_t* new_slot, int64_t* totals);

/*
 * kvlink_reencode_keys — positional re-encoding of cached keys (Sec. 2.2):
 * for every layer l < n_layers, KV head h < n_kv_heads, span i and row
 * t < len_i:
 *     dst(l, h, dst_seq_i, dst_row_i + t) = R(delta_i) src(l, h, src_seq_i, src_row_i + t)
 * Values are never touched.  One launch covers all layers (delta does not
 * depend on the layer).  src and dst may be the same view (in place) as long
 * as every span maps its rows onto themselves; otherwise they must not
 * overlap.
 *
 *   d_spans       device array of n_spans kvlink_span
 *   max_span_len  an upper bound of every span's len (sizes the grid)
 *   head_dim      64 or 128; dtype KVLINK_F32 or KVLINK_BF16
 *
 * Errors: KVLINK_ERR_INVALID_ARG (null pointers, n_layers/n_kv_heads < 1,
 * n_spans < 0, rope_theta <= 0, misaligned base or stride),
 * KVLINK_ERR_UNSUPPORTED (head_dim, dtype), KVLINK_ERR_HIP.
 * n_spans == 0 or max_span_len == 0 launches nothing and returns KVLINK_OK.
 */
kvlink_status kvlink_reencode_keys(kvlink_dtype dtype, int32_t n_layers, int32_t n_kv_heads,
                                   int32_t head_dim, double rope_theta, int32_t n_spans,
                                   const kvlink_span* d_spans, int32_t max_span_len,
                                   kvlink_kv_view src, kvlink_kv_view dst, void* stream);

/*
 * kvlink_encode_keys_at_positions — the paper's literal storage form
 * (Sec. 2.2): keys are cached without any positional rotation (K = W_k x)
 * and the global rotation is applied at inference, per token:
 *     dst(l, h, dst_seq_i, dst_row_i + t) = R(delta_i + t) src(l, h, src_seq_i, src_row_i + t)
 * With the spans of kvlink_build_layout and doc_src_pos0 = 0, delta_i = g_i,
 * so key t of document i lands at its global position g_i + t.  This equals
 * kvlink_reencode_keys applied to keys stored rotated at local positions
 * 0.. (rotations compose).  Arguments, layouts, aliasing rules and errors
 * are those of kvlink_reencode_keys.
 */
kvlink_status kvlink_encode_keys_at_positions(kvlink_dtype dtype, int32_t n_layers,
                                              int32_t n_kv_heads, int32_t head_dim,
                                              double rope_theta, int32_t n_spans,
                                              const kvlink_span* d_spans, int32_t max_span_len,
                                              kvlink_kv_view src, kvlink_kv_view dst,
                                              void* stream);

/*
 * kvlink_reencode_keys_mapped — re-encoding of compressed caches (Sec. 2.4:
 * only some tokens of a document are kept, e.g. its anchor tokens or the
 * tokens a compressor keeps, each cached with RoPE at its original position
 * p).  The kept keys take contiguous global positions after concatenation,
 * so the rotation differs per key:
 *     dst(l, h, dst_seq_i, dst_row_i + t) = R(delta_i + t - p) src(l, h, src_seq_i, src_row_i + t),
 *     p = d_stored_pos[src_seq_i * stored_pos_stride + src_row_i + t]
 * (p = t gives kvlink_reencode_keys, p = 0 kvlink_encode_keys_at_positions).
 * The layout comes from kvlink_build_layout with the kept-token counts as
 * document lengths; attention over the result needs nothing else.
 *
 *   d_stored_pos        device int32 array: the stored position of every
 *                       source row, indexed by (src_seq, row)
 *   stored_pos_stride   entries per source sequence in d_stored_pos
 * Other arguments, layouts and errors as kvlink_reencode_keys; also
 * KVLINK_ERR_INVALID_ARG for a NULL d_stored_pos or a negative stride.
 */
kvlink_status kvlink_reencode_keys_mapped(kvlink_dtype dtype, int32_t n_layers,
                                          int32_t n_kv_heads, int32_t head_dim, double rope_theta,
                                          int32_t n_spans, const kvlink_span* d_spans,
                                          int32_t max_span_len, const int32_t* d_stored_pos,
                                          int64_t stored_pos_stride, kvlink_kv_view src,
                                          kvlink_kv_view dst, void* stream);

/*
 * kvlink_group_spans — group the spans that read the same stored rows (host,
 * integer).  A document reused by several requests of a batch (the cache
 * reuse of Sec. 1 and Sec. 3.3: one precomputed cache per document, shared by
 * every request that retrieves it) appears in one span per use, all with the
 * same (src_seq, src_row, len) and each with its own destination and delta.
 *
 *   h_spans[n_spans]        host spans (e.g. kvlink_build_layout's)
 *   max_group               0: one group per distinct (src_seq, src_row,
 *                           len); > 0: such a run of n spans is cut into
 *                           ceil(n / max_group) consecutive groups whose
 *                           sizes differ by at most one (kvlink_reencode_keys_
 *                           shared then reads those stored rows once per
 *                           group, and a workgroup's work is bounded by
 *                           max_group destinations)
 *   h_order[n_spans]        out: span indices, grouped, each group in span
 *                           order, groups by (src_seq, src_row, len)
 *   h_group_ptr[n_spans+1]  out: group g is h_order[h_group_ptr[g] ..
 *                           h_group_ptr[g+1])
 *   n_groups                out
 * Errors: KVLINK_ERR_INVALID_ARG (n_spans < 0, max_group < 0, NULL pointers).
 */
kvlink_status kvlink_group_spans(int32_t n_spans, const kvlink_span* h_spans, int32_t max_group,
                                 int32_t* h_order, int32_t* h_group_ptr, int32_t* n_groups);

/*
 * kvlink_reencode_keys_shared — kvlink_reencode_keys, document-major: the
 * stored rows of each group of spans are read once and written, rotated by
 * each span's delta, to every span's destination (Sec. 2.2; the bytes moved
 * are the group's rows once plus every destination, instead of every span's
 * rows twice).  The result is the same, byte for byte, as
 * kvlink_reencode_keys over the same spans.
 *
 *   n_groups, d_group_ptr   device int32 [n_groups + 1]: group g's spans are
 *                           d_spans[d_group_ptr[g] .. d_group_ptr[g+1])
 *   d_spans                 device spans in group order (kvlink_group_spans'
 *                           h_order applied); all spans of a group must
 *                           share src_seq, src_row and len (the first span's
 *                           are used); max_span_len as kvlink_reencode_keys
 * src and dst must be different buffers (no in-place form).  Other
 * arguments, layouts and errors as kvlink_reencode_keys, with n_groups in
 * place of n_spans; also KVLINK_ERR_INVALID_ARG for src.base == dst.base.
 */
kvlink_status kvlink_reencode_keys_shared(kvlink_dtype dtype, int32_t n_layers,
                                          int32_t n_kv_heads, int32_t head_dim, double rope_theta,
                                          int32_t n_groups, const int32_t* d_group_ptr,
                                          const kvlink_span* d_spans, int32_t max_span_len,
                                          kvlink_kv_view src, kvlink_kv_view dst, void* stream);

/*
 * Bytes of a device staging area of n_slots slots for kvlink_load_and_reencode:
 * a slot holds one layer's stored keys and values (2 * n_kv_heads *
 * stored_rows * head_dim elements).  Returns 0 for invalid sizes or
 * n_slots < 2.
 */
size_t kvlink_load_stage_bytes(kvlink_dtype dtype, int32_t n_kv_heads, int32_t head_dim,
                               int32_t stored_rows, int32_t n_slots);

/*
 * kvlink_load_and_reencode — the first steps of the time-to-first-token path
 * (Sec. 3.3 times it from caches held in CPU memory): the stored document
 * caches of a batch are loaded from host memory, their keys re-encoded
 * (Sec. 2.2, as kvlink_reencode_keys, or kvlink_encode_keys_at_positions
 * with literal = 1) into k_dst and their values gathered into v_dst, both
 * through the spans.  Two ways:
 *   d_stage == NULL (direct): the kernels read the pinned host arrays over
 *     the bus through their device mapping: one re-encode launch and one
 *     value-gather launch for all layers on compute_stream (copy_stream is
 *     not used).  The arrays must be pinned and mapped for the device
 *     (hipHostMalloc with default flags); otherwise KVLINK_ERR_INVALID_ARG
 *     and nothing is launched.
 *   d_stage != NULL (staged): the staging area holds cap =
 *     min(n_layers, stage_bytes / slot) layers (slot as
 *     kvlink_load_stage_bytes: one layer's keys and values), used as a ring
 *     of floor(cap / G) chunks of G consecutive layers, G the fewest layers
 *     whose keys reach 64 MiB, at most cap / 2 (so the ring has two chunks
 *     or more).  Chunk c is copied (one copy for its keys, one for its
 *     values) to ring entry c % n_ring on copy_stream and re-encoded from it
 *     on compute_stream.  With two streams, events order them: the
 *     re-encode of a chunk waits for its copy, the copy waits for the
 *     re-encode that last read its entry, and the first copies wait for the
 *     work compute_stream held when the call was made (an earlier call's
 *     re-encodes may still read the entries).  With copy_stream ==
 *     compute_stream the stream itself orders everything.  Copies and
 *     cross-stream waits carry a fixed cost each; a staging area of many
 *     layers keeps them few (with two slots every layer is a chunk).
 *     The events are created on a thread's first staged call on a device
 *     and kept for reuse by later calls of that thread.
 * The call enqueues the work and returns.
 *
 *   h_k, h_v      host arrays [n_layers][n_kv_heads][stored_rows][head_dim],
 *                 16-byte aligned, the stored caches of the batch's documents
 *                 (span i's rows from src_row_i; src_seq is not used); they
 *                 must stay valid until compute_stream has finished
 *   d_stage, stage_bytes  NULL, or a device staging area of at least
 *                 kvlink_load_stage_bytes(..., 2) bytes, 256-byte aligned
 *   k_dst, v_dst  destination views (K and V rows of every span land at
 *                 dst_row_i.. of sequence dst_seq_i, layer l)
 *   literal       0: keys cached rotated at local positions (R(delta_i));
 *                 1: cached without rotation (R(delta_i + t))
 *   copy_stream, compute_stream  hipStream_t as void*
 *
 * Errors: those of kvlink_reencode_keys, and KVLINK_ERR_INVALID_ARG (null or
 * misaligned host arrays, unmapped host memory on the direct way,
 * stored_rows < 1, literal not 0 or 1), KVLINK_ERR_WORKSPACE (staging area
 * misaligned or smaller than two slots).
 */
kvlink_status kvlink_load_and_reencode(kvlink_dtype dtype, int32_t n_layers, int32_t n_kv_heads,
                                       int32_t head_dim, double rope_theta, int32_t n_spans,
                                       const kvlink_span* d_spans, int32_t max_span_len,
                                       const void* h_k, const void* h_v, int32_t stored_rows,
                                       void* d_stage, size_t stage_bytes, kvlink_kv_view k_dst,
                                       kvlink_kv_view v_dst, int32_t literal, void* copy_stream,
                                       void* compute_stream);

/*
 * Schedule of the split-K attention of a request batch (host-built once per
 * batch, reused for every layer).  The new-token rows of each request are
 * packed per KV head as row = token * group + head-in-group (group =
 * n_q_heads / n_kv_heads) and cut into row blocks of row_block rows; a
 * (request, KV head, row block) unit walks the keys its last token sees in
 * 64-key tiles.  The units' tiles are dealt out to n_workgroups persistent
 * workgroups in contiguous pieces (the split-K of flash-decoding, balanced
 * across units by a cost model): either each unit cut into pieces of equal
 * cost, one per workgroup, or equal-cost ranges over all units in order;
 * each piece of a unit that one workgroup covers is a segment.  A unit with
 * several segments has its partial results merged by a log-sum-exp merge:
 * by a combine launch, or (row blocks 128, 64 and 16, when the schedule
 * chooses it) inside the split launch by the unit's last-arriving workgroup.
 *
 * The table (int32, built on the host by kvlink_attend_make_plan, then
 * copied to the device by the caller) holds, in order:
 *   n_segments x 16    segment records {request, KV head, first row of the
 *                      block, rows in the block, first tile, end tile,
 *                      segments of the unit, index of this one among them,
 *                      first new token of the request, T_c of the request,
 *                      cached rows the block's last token sees, key count
 *                      of the unit, first segment of the unit in unit
 *                      order, next record of the same workgroup (-1: none),
 *                      unit, 0}; record w (w < n_workgroups) is workgroup
 *                      w's first segment
 *   n_units x 8        unit records {request, KV head, first row of the
 *                      block, rows in the block, first new token of the
 *                      request, first segment in unit order, segments, 0}
 *   n_split_units      the units with more than one segment (merged)
 * Like the layout arrays, the device copy is trusted: it must be the
 * unmodified table built for the same batch.
 */
typedef struct {
    const int32_t* table; /* device copy of the table (NULL in make_plan's output) */
    int32_t table_len;    /* int32 entries of the table */
    int32_t n_workgroups;
    int32_t n_units;
    int32_t n_segments;
    int32_t row_block;    /* rows per unit: 256, 128 or 64, or 16 (at most 16 rows per KV
                             head; fp32) */
    int32_t n_seqs;
    int32_t n_split_units; /* units with more than one segment */
    uint32_t flags;       /* the kvlink_attend_make_plan flags the schedule was built
                             with, with KVLINK_PLAN_COMBINE or KVLINK_PLAN_IN_LAUNCH
                             set to the merge it uses */
    /* device table of kvlink_attend_rope_table for the same batch, or NULL
     * (then the RoPE stage runs as its own launch) */
    const float* rope_table;
} kvlink_attend_plan;

/*
 * kvlink_attend_rope_table — the cos/sin values of every new token's
 * rotation (Sec. 2.2: the new tokens sit at their global positions), once per
 * batch: table[n][j] = (cos(pos_n w_j), sin(pos_n w_j)), w_j =
 * rope_theta^(-2j/head_dim), j < head_dim/2, angles in double precision
 * rounded to float (as the RoPE stage computes them).  With plan.rope_table
 * set to this table, kvlink_attend_new_tokens for bf16 batches rotates the
 * new tokens inside the split-attention launch: the RoPE stage launches
 * nothing, and the split stage rotates the queries it loads and appends the
 * rotated keys and the values to the cache rows T_c + r itself (every
 * workgroup whose keys include new rows writes the keys it reads, all with
 * identical bytes; values likewise, except that 256-row units read the new
 * values from v_new and write each one once).  The cache holds every new
 * row when the launch completes.  fp32 batches always use the separate RoPE
 * launch.
 *
 *   d_new_pos   device int32 [n_new_total] (the layout's new_pos)
 *   d_table     device float [n_new_total][head_dim / 2][2]
 * Errors: KVLINK_ERR_INVALID_ARG (null pointers, rope_theta <= 0,
 * n_new_total < 0), KVLINK_ERR_UNSUPPORTED (head_dim), KVLINK_ERR_HIP.
 */
kvlink_status kvlink_attend_rope_table(int32_t head_dim, double rope_theta, int32_t n_new_total,
                                       const int32_t* d_new_pos, float* d_table, void* stream);

/*
 * kvlink_attend_make_plan — build the schedule (pure host computation).
 *
 *   seq_new_ptr[n_seqs+1], seq_cached[n_seqs], new_visible[n_new]
 *                    host outputs of kvlink_build_layout for the batch
 *   n_compute_units  compute units of the device (sizes the schedule)
 *   n_workgroups     0: chosen by a cost model (a segment costs a set-up,
 *                    a tile its K/V stream plus the products of the steps
 *                    its wavefronts do not skip and, for new rows among
 *                    its keys, their RoPE and append as the fused form
 *                    does them; the launch is as long as its longest
 *                    workgroup, and split units add their merge; of the
 *                    cuts within 2% of the best estimate, the one with the
 *                    most workgroups is taken);
 *                    > 0: that many workgroups (capped at the tile count)
 *   row_block        0: chosen by the same cost model among the row blocks
 *                    of the batch's kernel (256, 128, 64 for batches with
 *                    more than 16 rows per request and KV head, else 16);
 *                    else that row block (KVLINK_ERR_UNSUPPORTED if it is
 *                    not one of them)
 *   flags            a combination of
 *                    KVLINK_PLAN_XCD: number the workgroups so that those
 *                      whose first segment shares a request and KV head run
 *                      on one XCD (workgroup w runs on XCD w % 8 on MI355X),
 *                      sharing one L2;
 *                    KVLINK_PLAN_COMBINE or KVLINK_PLAN_IN_LAUNCH (not
 *                      both): merge split units by the combine launch, or
 *                      inside the split launch (row blocks 128, 64 and 16;
 *                      IN_LAUNCH with row_block 256 is KVLINK_ERR_UNSUPPORTED);
 *                      without either the cost model chooses, and
 *                      plan->flags reports the choice;
 *                    none changes the result beyond float rounding order
 *   table, table_capacity  host array for the table; with table == NULL
 *                    only *plan is filled (to size the array)
 *   plan             out: counts and row_block; plan->table and
 *                    plan->rope_table are set to NULL (the caller stores
 *                    the table's device copy in table and, for the fused
 *                    RoPE, the batch's kvlink_attend_rope_table result in
 *                    rope_table)
 *
 * The result of the attention does not depend on the schedule beyond float
 * rounding order.  Errors: KVLINK_ERR_INVALID_ARG (null required pointer,
 * n_seqs < 1, n_compute_units < 1, n_workgroups < 0, row_block < 0, unknown
 * flags, table too small), KVLINK_ERR_UNSUPPORTED (head_dim, dtype, group,
 * row_block, more than 16384 units), KVLINK_ERR_LAYOUT (seq_new_ptr not
 * non-decreasing from 0, seq_cached or new_visible negative, a key range
 * beyond 2^30).
 */
enum {
    KVLINK_PLAN_XCD = 1,
    KVLINK_PLAN_COMBINE = 4,
    KVLINK_PLAN_IN_LAUNCH = 8
};

kvlink_status kvlink_attend_make_plan(kvlink_dtype dtype, int32_t n_q_heads, int32_t n_kv_heads,
                                      int32_t head_dim, int32_t n_seqs,
                                      const int32_t* seq_new_ptr, const int32_t* seq_cached,
                                      const int32_t* new_visible,
                                      int32_t n_compute_units, int32_t n_workgroups,
                                      int32_t row_block, uint32_t flags, int32_t* table,
                                      int64_t table_capacity, kvlink_attend_plan* plan);

/*
 * Workspace bytes kvlink_attend_new_tokens needs: 64 KiB of merge counters,
 * then the rotated queries and, when some unit has several segments, the
 * split partials.  Returns 0 for invalid sizes or a null plan.
 *
 * The counters (the workspace's first 64 KiB) must be zero before a
 * workspace is first used, with any plan: fill them with zeros once after
 * allocating it.  Every call that completes leaves them zero again, so a
 * workspace is reused without clearing.
 */
size_t kvlink_attend_workspace_bytes(kvlink_dtype dtype, int32_t n_q_heads, int32_t n_kv_heads,
                                     int32_t head_dim, int32_t n_new_total,
                                     const kvlink_attend_plan* plan);

/*
 * kvlink_attend_new_tokens — one layer of the forward pass over the new
 * tokens (Sec. 2.3, last paragraph: the link tokens are appended after the
 * reused caches and run with the customised attention map; Sec. 2.1: the
 * query follows).  For every request s and new token r of it, at global
 * position p_r:
 *
 *   1. q_r, k_r are rotated by R(p_r) (they arrive before RoPE);
 *   2. the rotated k_r and v_r are appended to the cache of `layer` at row
 *      seq_cached[s] + r (right after the request's cached rows);
 *   3. for every query head hq (KV head hk = hq / (n_q_heads / n_kv_heads)):
 *        out[r][hq] = sum_b softmax_b(scale * <q_r, k_b>) v_b
 *      over the keys b the attention map of Sec. 2.3 lets a link or query
 *      token see: every position at or before p_r, i.e. the first
 *      new_visible[r] cached rows and the new tokens 0..r of the request.
 *      lse[r][hq] (if lse != NULL) = log sum_b exp(scale * <q_r, k_b>).
 *
 * Arguments:
 *   n_seqs, n_new_total        requests and new tokens in the batch
 *   max_new, max_cached        max over requests of new tokens and of T_c
 *   d_seq_new_ptr[n_seqs+1], d_seq_cached[n_seqs], d_new_pos[n_new_total],
 *   d_new_visible[n_new_total] device copies of kvlink_build_layout outputs
 *   q_new  [n_new_total][n_q_heads][head_dim]   device, dtype, pre-RoPE
 *   k_new, v_new [n_new_total][n_kv_heads][head_dim]  device, dtype
 *                              (q_new, k_new, v_new 16-byte aligned)
 *   k_cache, v_cache           views (see kvlink_kv_view) whose rows
 *                              0..T_c-1 of request s hold its re-encoded keys
 *                              and its values, with room for the new rows
 *   out   [n_new_total][n_q_heads][head_dim]    device, dtype
 *   lse   [n_new_total][n_q_heads] float, or NULL
 *   plan                       schedule from kvlink_attend_make_plan for the
 *                              same batch, with plan.table pointing at the
 *                              device copy of its table (16-byte aligned).
 *                              Its row_block must match this call's path
 *                              (KVLINK_ERR_INVALID_ARG otherwise).  With
 *                              plan.rope_table set (16-byte aligned, the
 *                              batch's kvlink_attend_rope_table), a bf16
 *                              call does steps 1 and 2 inside the split
 *                              launch (same bytes as the separate launch)
 *   workspace, workspace_bytes at least kvlink_attend_workspace_bytes(...)
 *                              device bytes, 256-byte aligned, its first
 *                              64 KiB zero (see kvlink_attend_workspace_bytes)
 *
 * softmax_scale must be positive and finite (1/sqrt(head_dim) for the Llama
 * family).  Supported: head_dim 64 or 128; n_q_heads / n_kv_heads in {1, 2, 4, 8};
 * dtype KVLINK_F32 or KVLINK_BF16 (float accumulation and softmax either way).
 *
 * Errors: KVLINK_ERR_INVALID_ARG, KVLINK_ERR_UNSUPPORTED,
 * KVLINK_ERR_WORKSPACE, KVLINK_ERR_HIP, as listed above.  n_new_total == 0
 * launches nothing and returns KVLINK_OK.
 */
kvlink_status kvlink_attend_new_tokens(
    kvlink_dtype dtype, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
    double rope_theta, float softmax_scale, int32_t n_seqs, int32_t n_new_total,
    int32_t max_new, int32_t max_cached, const int32_t* d_seq_new_ptr,
    const int32_t* d_seq_cached, const int32_t* d_new_pos, const int32_t* d_new_visible,
    const void* q_new, const void* k_new, const void* v_new, kvlink_kv_view k_cache,
    kvlink_kv_view v_cache, int32_t layer, void* out, float* lse, kvlink_attend_plan plan,
    void* workspace, size_t workspace_bytes, void* stream);

/*
 * kvlink_attend_stages — kvlink_attend_new_tokens run stage by stage, with
 * identical arguments plus a bit mask of the stages to launch:
 *   KVLINK_STAGE_ROPE     steps 1 and 2 (RoPE of the new tokens, append of
 *                         their keys and values, rotated q to the workspace);
 *                         launches nothing when plan.rope_table is set for
 *                         a bf16 call, whose SPLIT stage then does both
 *   KVLINK_STAGE_SPLIT    step 3 over every segment of the plan (a unit
 *                         with one segment writes out and lse directly, the
 *                         others write split partials to the workspace)
 *   KVLINK_STAGE_COMBINE  log-sum-exp merge of the split partials into out
 *                         and lse (no launch when every unit has one segment)
 * Stages must run in this order, on the same stream, with the same workspace
 * and arguments; kvlink_attend_new_tokens is all three.  For callers that
 * time or overlap the stages separately.  Errors as kvlink_attend_new_tokens,
 * plus KVLINK_ERR_INVALID_ARG for an empty or unknown mask.
 */
enum { KVLINK_STAGE_ROPE = 1, KVLINK_STAGE_SPLIT = 2, KVLINK_STAGE_COMBINE = 4 };

kvlink_status kvlink_attend_stages(
    kvlink_dtype dtype, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
    double rope_theta, float softmax_scale, int32_t n_seqs, int32_t n_new_total,
    int32_t max_new, int32_t max_cached, const int32_t* d_seq_new_ptr,
    const int32_t* d_seq_cached, const int32_t* d_new_pos, const int32_t* d_new_visible,
    const void* q_new, const void* k_new, const void* v_new, kvlink_kv_view k_cache,
    kvlink_kv_view v_cache, int32_t layer, void* out, float* lse, kvlink_attend_plan plan,
    void* workspace, size_t workspace_bytes, void* stream, uint32_t stages);

/*
 * kvlink_attend_new_tokens_noalloc — kvlink_attend_new_tokens for callers
 * that cannot allocate device memory or own a workspace: code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation.  Same
 * arguments and result (the same kernels, the same schedule: the outputs are
 * bit for bit those of kvlink_attend_new_tokens), without the workspace.
 *
 * The rotated queries and split partials go to a scratch area inside the
 * library: a static device array of KVLINK_NOALLOC_SCRATCH_BYTES bytes, one
 * copy per GPU, held from the library's load until the process ends.  Its
 * address on a device is looked up once, on the first call with that device
 * current.  The call allocates nothing (no hipMalloc, no allocating library
 * routine).  Every call on one GPU uses that GPU's single copy: calls that
 * overlap on one GPU (different streams, or host threads without ordering)
 * race and give wrong results; calls ordered on one stream do not.  The
 * scratch needs no clearing: its merge counters (its first 64 KiB, as in a
 * workspace) are zero when the library is loaded and every completed call
 * leaves them zero; every other byte a call reads was written earlier in the
 * same call.
 *
 * Errors: those of kvlink_attend_new_tokens; KVLINK_ERR_WORKSPACE when the
 * call needs more than KVLINK_NOALLOC_SCRATCH_BYTES (kvlink_attend_workspace_bytes
 * of the same arguments), before any HIP call; KVLINK_ERR_HIP if the scratch
 * address cannot be looked up.
 */
#define KVLINK_NOALLOC_SCRATCH_BYTES (32u << 20)

kvlink_status kvlink_attend_new_tokens_noalloc(
    kvlink_dtype dtype, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
    double rope_theta, float softmax_scale, int32_t n_seqs, int32_t n_new_total,
    int32_t max_new, int32_t max_cached, const int32_t* d_seq_new_ptr,
    const int32_t* d_seq_cached, const int32_t* d_new_pos, const int32_t* d_new_visible,
    const void* q_new, const void* k_new, const void* v_new, kvlink_kv_view k_cache,
    kvlink_kv_view v_cache, int32_t layer, void* out, float* lse, kvlink_attend_plan plan,
    void* stream);

/*
 * kvlink_attend_new_tokens_fused — kvlink_attend_new_tokens with the
 * positional re-encode of the cached keys (Sec. 2.2) folded into the split
 * launch: k_cache holds, at every request's cached rows, the keys as stored
 * (rotated at their documents' own positions, not yet re-encoded), and the
 * kernel rotates each cached key of span i by R(delta_i) in LDS, once per
 * workgroup, as its 64-key tile arrives and before any product reads it.
 * The rotation uses the re-encode launch's routine and angles, so out and lse
 * equal, bit for bit, kvlink_reencode_keys over the same spans into a cache
 * of the same layout followed by kvlink_attend_new_tokens with the same plan.
 * The cached rows of k_cache are only read; the new tokens' rows are handled
 * (appended, with the RoPE inside the split launch when the plan has a rope
 * table) as by kvlink_attend_new_tokens.  The separate re-encode's write of
 * the re-encoded keys is skipped; every call rotates again.
 *
 *   d_spans, d_seq_span_ptr  device: request s's spans are d_spans[
 *                            d_seq_span_ptr[s] .. d_seq_span_ptr[s + 1]),
 *                            in increasing dst_row, not overlapping (as
 *                            kvlink_build_layout makes them); a cached row
 *                            of request s in none of them is used as stored.
 *                            dst_row, len and delta are read (dst rows are
 *                            request s's rows of k_cache)
 *   max_spans_per_seq        the most spans of any request, at most
 *                            KVLINK_FUSED_MAX_SPANS (the (cos, sin) tables of
 *                            a request's spans are held in LDS)
 * Other arguments, layouts and errors as kvlink_attend_new_tokens; also
 * KVLINK_ERR_UNSUPPORTED for a plan not on the wide bf16 kernel (row_block
 * 256, 128 or 64) or more than KVLINK_FUSED_MAX_SPANS spans per request,
 * and KVLINK_ERR_INVALID_ARG for NULL span arrays or a negative count.
 */
#define KVLINK_FUSED_MAX_SPANS 48

kvlink_status kvlink_attend_new_tokens_fused(
    kvlink_dtype dtype, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
    double rope_theta, float softmax_scale, int32_t n_seqs, int32_t n_new_total,
    int32_t max_new, int32_t max_cached, const int32_t* d_seq_new_ptr,
    const int32_t* d_seq_cached, const int32_t* d_new_pos, const int32_t* d_new_visible,
    const void* q_new, const void* k_new, const void* v_new, kvlink_kv_view k_cache,
    kvlink_kv_view v_cache, int32_t layer, void* out, float* lse, kvlink_attend_plan plan,
    const kvlink_span* d_spans, const int32_t* d_seq_span_ptr, int32_t max_spans_per_seq,
    void* workspace, size_t workspace_bytes, void* stream);

/* Message of the last non-OK status on the calling thread ("" if none). */
const char* kvlink_last_error(void);

/* Library version string. */
const char* kvlink_version(void);

#ifdef __cplusplus
}
#endif
#endif
