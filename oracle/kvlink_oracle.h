/*
 * kvlink_oracle.h — plain CPU reference for the KVLink inference hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  This library is the oracle that the GPU path is
 * checked against.  Only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark may load it.  It shares no code, header or table with
 * the GPU library and never calls it.
 *
 * Everything is computed in IEEE double precision, with RoPE angles formed and
 * evaluated in 80-bit long double before rounding to double.  Positions are
 * 0-based.  Paper references are to "KVLink: Accelerating Large Language
 * Models via Efficient KV Cache Reuse" (arXiv 2502.16002).
 *
 * Parity status of each function (what pins it is listed in the tests):
 *   kvo_layout, kvo_allowed, kvo_full_mask  pinned (Fig. 2 worked example,
 *                                           Sec. 2.2 position example, closed forms)
 *   kvo_rope, kvo_reencode                  pinned (unit-circle values, closed-form
 *                                           frequencies, complex-number form,
 *                                           composition identity)
 *   kvo_attend, kvo_attend_probs            pinned (brute-force masked softmax,
 *                                           library SDPA special case, invariants)
 */
#ifndef KVLINK_ORACLE_H
#define KVLINK_ORACLE_H

#ifdef __cplusplus
extern "C" {
#endif

/* Token kinds of the concatenated sequence (Sec. 2.3). */
enum { KVO_DOC = 0, KVO_LINK = 1, KVO_QUERY = 2 };

/* Number of OpenMP threads the oracle runs with. */
int kvo_num_threads(void);

/*
 * Sequence layout (Sec. 2.1 and the link-token equation of Sec. 2.3): the
 * retrieved documents in order, each c = (c_1..c_L, link_1..link_K), then the
 * query tokens.  For every global position p writes kind[p], seg[p] (document
 * index, -1 for query tokens) and idx[p] (token index inside the document,
 * link index k, or query index).  The output arrays may be NULL to only count.
 * Returns the total number of positions T, or -1 if an input is invalid
 * (n_docs < 0, n_query < 0, a length < 1, a link count < 0).
 */
int kvo_layout(int n_docs, const int* doc_len, const int* link_count, int n_query,
               int* kind, int* seg, int* idx);

/*
 * Training attention map (Sec. 2.3, Fig. 2): 1 if position a may attend to
 * position b.  Document tokens attend causally inside their own document; link
 * and query tokens attend to every position at or before their own.
 */
int kvo_allowed(const int* kind, const int* seg, int a, int b);

/* The full T x T map of kvo_allowed, row-major: mask[a*T + b]. */
void kvo_full_mask(int T, const int* kind, const int* seg, unsigned char* mask);

/*
 * RoPE rotation R_pos (Sec. 2.2): rotates each pair (x_j, x_{j+d/2}), j < d/2,
 * by the angle pos * theta^(-2j/d), in place.  d must be even.
 */
void kvo_rope(double* x, int d, long long pos, double theta);

/*
 * Positional re-encoding (Sec. 2.2): k_out[v] = R_delta k_in[v] for n_vec
 * vectors of length d.  In-place use (k_out == k_in) is allowed.  Returns 0,
 * or -1 if d is odd, below 2 or above 1024.
 */
int kvo_reencode(const double* k_in, double* k_out, long long n_vec, int d,
                 long long delta, double theta);

/*
 * Attention of the new tokens (link and query tokens) of one request over the
 * concatenated sequence (Sec. 2.2 and 2.3), one layer.
 *
 *   k_cached, v_cached : [n_kv_heads][T_c][d], the stored caches of the
 *                        documents back to back in retrieval order, T_c = sum
 *                        of doc_len.  Stored keys carry RoPE at positions
 *                        src_pos0[i] + t (src_pos0 NULL means all zero).
 *   q_new              : [n_new][n_q_heads][d] before RoPE
 *   k_new, v_new       : [n_new][n_kv_heads][d], keys before RoPE
 *                        (new tokens in increasing global position)
 *   rows               : indices of the new tokens to compute (n_rows of
 *                        them), or NULL for all n_new in order
 *   out                : [n_rows][n_q_heads][d], lse : [n_rows][n_q_heads]
 *                        (natural-log sum of exp of the scaled scores)
 *
 * Query head h reads KV head h / (n_q_heads / n_kv_heads).  Returns 0, or -1 on
 * invalid input.
 */
int kvo_attend(int n_docs, const int* doc_len, const int* link_count, int n_query,
               const long long* src_pos0,
               int n_q_heads, int n_kv_heads, int d, double theta, double scale,
               const double* k_cached, const double* v_cached,
               const double* q_new, const double* k_new, const double* v_new,
               int n_rows, const int* rows, double* out, double* lse);

/*
 * The softmax probabilities of one new token `row` and one query head over
 * all T positions of the sequence (0 where the map forbids), same inputs as
 * kvo_attend.  probs has T entries.  Returns T, or -1 on invalid input.
 */
int kvo_attend_probs(int n_docs, const int* doc_len, const int* link_count, int n_query,
                     const long long* src_pos0,
                     int n_q_heads, int n_kv_heads, int d, double theta, double scale,
                     const double* k_cached, const double* q_new, const double* k_new,
                     int row, int head, double* probs);

#ifdef __cplusplus
}
#endif
#endif
