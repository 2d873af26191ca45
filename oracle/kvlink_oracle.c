/*
 * kvlink_oracle.c — plain CPU reference for the KVLink inference hot path.
 *
 * TEST INFRASTRUCTURE ONLY (see kvlink_oracle.h).  Slow on purpose: each
 * function writes out the definition it follows, in double precision, with no
 * blocking, fusion or reordering.  Built with -ffp-contract=off so that no
 * multiply-add is fused behind the reader's back.
 */
#include "kvlink_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int kvo_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ---------------------------------------------------------------- layout */

/* Sec. 2.3: every document c = (c_1..c_L, c_link1..c_linkK); Sec. 2.1: the
 * documents are concatenated in retrieval order and the query follows. */
int kvo_layout(int n_docs, const int* doc_len, const int* link_count, int n_query,
               int* kind, int* seg, int* idx) {
    if (n_docs < 0 || n_query < 0) return -1;
    long long p = 0;
    for (int i = 0; i < n_docs; ++i) {
        if (doc_len[i] < 1 || link_count[i] < 0) return -1;
        for (int t = 0; t < doc_len[i]; ++t, ++p) {
            if (kind) { kind[p] = KVO_DOC; seg[p] = i; idx[p] = t; }
        }
        for (int k = 0; k < link_count[i]; ++k, ++p) {
            if (kind) { kind[p] = KVO_LINK; seg[p] = i; idx[p] = k; }
        }
    }
    for (int q = 0; q < n_query; ++q, ++p) {
        if (kind) { kind[p] = KVO_QUERY; seg[p] = -1; idx[p] = q; }
    }
    if (p > 0x7fffffffLL) return -1;
    return (int)p;
}

/* Sec. 2.3 and Fig. 2: document tokens keep local causal attention inside
 * their document; each link token attends to all preceding tokens (itself
 * included); the question and user tokens are standard causal. */
int kvo_allowed(const int* kind, const int* seg, int a, int b) {
    if (b > a) return 0;
    if (kind[a] == KVO_DOC) return kind[b] == KVO_DOC && seg[b] == seg[a];
    return 1;
}

void kvo_full_mask(int T, const int* kind, const int* seg, unsigned char* mask) {
    for (int a = 0; a < T; ++a)
        for (int b = 0; b < T; ++b)
            mask[(size_t)a * T + b] = (unsigned char)kvo_allowed(kind, seg, a, b);
}

/* ------------------------------------------------------------------ RoPE */

/* cos and sin of pos * theta^(-2j/d) for j < d/2, angles in long double. */
static void rope_angles(int d, long long pos, double theta, double* c, double* s) {
    for (int j = 0; j < d / 2; ++j) {
        long double w = powl((long double)theta, -2.0L * (long double)j / (long double)d);
        long double ang = (long double)pos * w;
        c[j] = (double)cosl(ang);
        s[j] = (double)sinl(ang);
    }
}

/* Apply a rotation given by its cos/sin table to one vector. */
static void rope_apply(const double* x, double* y, int d, const double* c, const double* s) {
    int h = d / 2;
    for (int j = 0; j < h; ++j) {
        double a = x[j], b = x[j + h];
        y[j]     = a * c[j] - b * s[j];
        y[j + h] = a * s[j] + b * c[j];
    }
}

void kvo_rope(double* x, int d, long long pos, double theta) {
    double* c = (double*)malloc(sizeof(double) * (size_t)(d / 2 + 1));
    double* s = (double*)malloc(sizeof(double) * (size_t)(d / 2 + 1));
    rope_angles(d, pos, theta, c, s);
    rope_apply(x, x, d, c, s);
    free(c);
    free(s);
}

/* Sec. 2.2: keys stored with RoPE at their local positions are moved to their
 * global positions by one more rotation, R_delta (rotations compose:
 * R_delta R_t = R_(delta+t)).  Values are never touched. */
int kvo_reencode(const double* k_in, double* k_out, long long n_vec, int d,
                 long long delta, double theta) {
    if (d < 2 || d % 2 || d > 1024 || n_vec < 0) return -1;
    double* c = (double*)malloc(sizeof(double) * (size_t)(d / 2 + 1));
    double* s = (double*)malloc(sizeof(double) * (size_t)(d / 2 + 1));
    rope_angles(d, delta, theta, c, s);
    #pragma omp parallel for schedule(static)
    for (long long v = 0; v < n_vec; ++v) {
        double tmp[1024];
        rope_apply(k_in + v * d, tmp, d, c, s);
        memcpy(k_out + v * d, tmp, sizeof(double) * (size_t)d);
    }
    free(c);
    free(s);
    return 0;
}

/* ------------------------------------------------------------- attention */

/* Everything the attention of one request needs, formed in the paper's order:
 * layout, re-encoded document keys, RoPE'd new keys, values per position. */
typedef struct {
    int T, n_new, hkv, d;
    int* kind; int* seg; int* idx;
    int* new_pos;      /* [n_new] global position of the n-th new token */
    double* keys;      /* [T][hkv][d] keys at their global positions */
    const double* vsrc_cached; const double* vsrc_new; int T_c;
    int* row_of;       /* [T] row in the cached arrays (doc) or new index */
} seqctx;

static void ctx_free(seqctx* c) {
    free(c->kind); free(c->seg); free(c->idx); free(c->new_pos);
    free(c->keys); free(c->row_of);
}

static int ctx_build(seqctx* c, int n_docs, const int* doc_len, const int* link_count,
                     int n_query, const long long* src_pos0, int hkv, int d, double theta,
                     const double* k_cached, const double* v_cached,
                     const double* k_new, const double* v_new) {
    memset(c, 0, sizeof(*c));
    int T = kvo_layout(n_docs, doc_len, link_count, n_query, NULL, NULL, NULL);
    if (T < 0 || hkv < 1 || d < 2 || d % 2 || d > 1024) return -1;
    c->T = T; c->hkv = hkv; c->d = d;
    c->kind = (int*)malloc(sizeof(int) * (size_t)(T + 1));
    c->seg = (int*)malloc(sizeof(int) * (size_t)(T + 1));
    c->idx = (int*)malloc(sizeof(int) * (size_t)(T + 1));
    c->row_of = (int*)malloc(sizeof(int) * (size_t)(T + 1));
    kvo_layout(n_docs, doc_len, link_count, n_query, c->kind, c->seg, c->idx);

    /* rows of each document in the stored (back to back) cache arrays */
    int T_c = 0;
    for (int i = 0; i < n_docs; ++i) T_c += doc_len[i];
    c->T_c = T_c;
    int* doc_row0 = (int*)malloc(sizeof(int) * (size_t)(n_docs + 1));
    int acc = 0;
    for (int i = 0; i < n_docs; ++i) { doc_row0[i] = acc; acc += doc_len[i]; }

    int n_new = 0;
    for (int p = 0; p < T; ++p) if (c->kind[p] != KVO_DOC) ++n_new;
    c->n_new = n_new;
    c->new_pos = (int*)malloc(sizeof(int) * (size_t)(n_new + 1));
    for (int p = 0, n = 0; p < T; ++p) {
        if (c->kind[p] == KVO_DOC) {
            c->row_of[p] = doc_row0[c->seg[p]] + c->idx[p];
        } else {
            c->row_of[p] = n;
            c->new_pos[n++] = p;
        }
    }

    c->keys = (double*)malloc(sizeof(double) * (size_t)T * hkv * d + 8);
    c->vsrc_cached = v_cached; c->vsrc_new = v_new;
    #pragma omp parallel for schedule(dynamic, 16)
    for (int p = 0; p < T; ++p) {
        double cs[512], sn[512];
        long long rot;
        const double* src;
        long long src_stride;
        if (c->kind[p] == KVO_DOC) {
            /* document i starts at global position g_i = p - t; its keys were
             * stored with RoPE at src_pos0[i] + t, so delta = g_i - src_pos0[i] */
            int i = c->seg[p];
            long long g = (long long)p - c->idx[p];
            rot = g - (src_pos0 ? src_pos0[i] : 0);
            src = k_cached + (size_t)c->row_of[p] * d;
            src_stride = (long long)T_c * d;
        } else {
            /* a new token is rotated at its own global position */
            rot = p;
            src = k_new + (size_t)c->row_of[p] * hkv * d;
            src_stride = d;
        }
        rope_angles(d, rot, theta, cs, sn);
        for (int h = 0; h < hkv; ++h)
            rope_apply(src + h * src_stride, c->keys + ((size_t)p * hkv + h) * d, d, cs, sn);
    }
    free(doc_row0);
    return 0;
}

static const double* ctx_value(const seqctx* c, int p, int h) {
    if (c->kind[p] == KVO_DOC)
        return c->vsrc_cached + ((size_t)h * c->T_c + c->row_of[p]) * c->d;
    return c->vsrc_new + ((size_t)c->row_of[p] * c->hkv + h) * c->d;
}

/* Scaled scores of one query vector (already at its position) over every
 * allowed position; forbidden positions get -INFINITY.  Returns the max. */
static double row_scores(const seqctx* c, int a, int hk, const double* q, double scale,
                         double* sc) {
    double m = -INFINITY;
    for (int b = 0; b < c->T; ++b) {
        if (!kvo_allowed(c->kind, c->seg, a, b)) { sc[b] = -INFINITY; continue; }
        const double* k = c->keys + ((size_t)b * c->hkv + hk) * c->d;
        double dot = 0.0;
        for (int j = 0; j < c->d; ++j) dot += q[j] * k[j];
        sc[b] = scale * dot;
        if (sc[b] > m) m = sc[b];
    }
    return m;
}

int kvo_attend(int n_docs, const int* doc_len, const int* link_count, int n_query,
               const long long* src_pos0,
               int n_q_heads, int n_kv_heads, int d, double theta, double scale,
               const double* k_cached, const double* v_cached,
               const double* q_new, const double* k_new, const double* v_new,
               int n_rows, const int* rows, double* out, double* lse) {
    if (n_q_heads < 1 || n_kv_heads < 1 || n_q_heads % n_kv_heads) return -1;
    seqctx c;
    if (ctx_build(&c, n_docs, doc_len, link_count, n_query, src_pos0, n_kv_heads, d, theta,
                  k_cached, v_cached, k_new, v_new))
        return -1;
    int group = n_q_heads / n_kv_heads;
    int nr = rows ? n_rows : c.n_new;
    for (int r = 0; r < nr; ++r)
        if ((rows ? rows[r] : r) < 0 || (rows ? rows[r] : r) >= c.n_new) { ctx_free(&c); return -1; }

    #pragma omp parallel
    {
        double* sc = (double*)malloc(sizeof(double) * (size_t)(c.T + 1));
        double q[1024], cs[512], sn[512];
        #pragma omp for schedule(dynamic, 1)
        for (long long w = 0; w < (long long)nr * n_q_heads; ++w) {
            int r = (int)(w / n_q_heads), h = (int)(w % n_q_heads);
            int n = rows ? rows[r] : r;
            int a = c.new_pos[n];
            int hk = h / group;                              /* GQA */
            rope_angles(d, a, theta, cs, sn);                /* query at its position */
            rope_apply(q_new + ((size_t)n * n_q_heads + h) * d, q, d, cs, sn);
            double m = row_scores(&c, a, hk, q, scale, sc);
            long double z = 0.0L;
            long double o[1024];
            for (int j = 0; j < d; ++j) o[j] = 0.0L;
            for (int b = 0; b < c.T; ++b) {
                if (sc[b] == -INFINITY) continue;
                double p = exp(sc[b] - m);                   /* softmax, max-subtracted */
                z += p;
                const double* v = ctx_value(&c, b, hk);
                for (int j = 0; j < d; ++j) o[j] += (long double)p * v[j];
            }
            double* dst = out + ((size_t)r * n_q_heads + h) * d;
            for (int j = 0; j < d; ++j) dst[j] = (double)(o[j] / z);
            if (lse) lse[(size_t)r * n_q_heads + h] = m + (double)logl(z);
        }
        free(sc);
    }
    ctx_free(&c);
    return 0;
}

int kvo_attend_probs(int n_docs, const int* doc_len, const int* link_count, int n_query,
                     const long long* src_pos0,
                     int n_q_heads, int n_kv_heads, int d, double theta, double scale,
                     const double* k_cached, const double* q_new, const double* k_new,
                     int row, int head, double* probs) {
    if (n_q_heads < 1 || n_kv_heads < 1 || n_q_heads % n_kv_heads) return -1;
    if (head < 0 || head >= n_q_heads) return -1;
    seqctx c;
    if (ctx_build(&c, n_docs, doc_len, link_count, n_query, src_pos0, n_kv_heads, d, theta,
                  k_cached, NULL, k_new, NULL))
        return -1;
    if (row < 0 || row >= c.n_new) { ctx_free(&c); return -1; }
    double q[1024], cs[512], sn[512];
    int a = c.new_pos[row];
    rope_angles(d, a, theta, cs, sn);
    rope_apply(q_new + ((size_t)row * n_q_heads + head) * d, q, d, cs, sn);
    double m = row_scores(&c, a, head / (n_q_heads / n_kv_heads), q, scale, probs);
    long double z = 0.0L;
    for (int b = 0; b < c.T; ++b) if (probs[b] != -INFINITY) z += exp(probs[b] - m);
    for (int b = 0; b < c.T; ++b)
        probs[b] = probs[b] == -INFINITY ? 0.0 : (double)((long double)exp(probs[b] - m) / z);
    int T = c.T;
    ctx_free(&c);
    return T;
}
