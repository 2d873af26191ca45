// attend_common.h — definitions shared by the attention kernels.
#pragma once

#include "kvlink_internal.h"

namespace kvlink {
namespace attn {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
// Finite stand-in for "no score seen yet" in log2 units: any real score
// exceeds it, and masked scores (-inf) still give weight 0 without NaN.
constexpr float kNoMax = -1.0e30f;


// Request of global new token n (binary search over seq_new_ptr).
__device__ __forceinline__ int seq_of(const int32_t* seq_new_ptr, int n_seqs, int n) {
    int lo = 0, hi = n_seqs - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (seq_new_ptr[mid] <= n) lo = mid; else hi = mid - 1;
    }
    return lo;
}

// Eight (cos, sin) pairs of a rope table row from entry j (64 bytes).
__device__ __forceinline__ void rope_table8(const float2* row, int j, float* c, float* s) {
    const float4* t = reinterpret_cast<const float4*>(row + j);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float4 v = t[i];
        c[2 * i] = v.x;
        s[2 * i] = v.y;
        c[2 * i + 1] = v.z;
        s[2 * i + 1] = v.w;
    }
}

// Key range of a row block: cached rows seen by its last token (cmax) and
// the virtual key count cmax + (last token + 1).
struct BlockKeys {
    int cmax, nvirt, r_last;
};
__device__ __forceinline__ BlockKeys block_keys(const int32_t* new_visible, int n0, int rows_s,
                                                int rho0, int row_block, int group) {
    const int rho_end = min(rho0 + row_block, rows_s);
    BlockKeys b;
    b.r_last = (rho_end - 1) / group;
    b.cmax = new_visible[n0 + b.r_last];
    b.nvirt = b.cmax + b.r_last + 1;
    return b;
}

// Arguments of the split kernels and the combine.  The schedule table (see
// the schedule's description in the public header) is read through seg
// (n_segments records of kSegRecord int32, as 4 int4; record w is workgroup
// w's first segment), unit (n_units records of kUnitRecord int32, as 2 int4)
// and split_units (the n_split units with several segments).
struct KParams {
    const void* q_rot;
    View k, v;
    int layer, n_seqs, n_q_heads, n_kv_heads, group;
    const int32_t* seq_new_ptr;
    const int32_t* seq_cached;
    const int32_t* new_visible;
    float scale_log2;
    int row_block, n_units, n_segments;
    const int4* seg;
    const int4* unit;
    const int32_t* split_units;
    int n_split;
    void* part_o;     // split partials O / l, in the workload dtype
    float* part_ml;   // their (running max in log2 units, sum) pairs
    // arrival counters of the units whose segments the split kernel merges
    // in the same launch, one per unit; zero before the launch and after it
    uint32_t* counters;
    // wide kernel's 128- and 64-row units and the decode kernel: split units
    // merged in the launch by their last-arriving workgroup (1), or left to
    // the combine launch (0)
    int merge_in_launch;
    void* out;
    float* lse;
    // With rope (the batch's cos/sin table, [n_new][D/2] (cos, sin)), the
    // split kernels rotate the queries of q_new themselves and append the new
    // tokens' rotated keys (k_new) and values (v_new) to the cache rows they
    // read; q_rot is then unused.
    const float2* rope;
    const void* q_new;
    const void* k_new;
    const void* v_new;
    // With fuse_spans (wide kernel), the cached keys are read as stored and
    // re-encoded as their tiles are staged: request s's spans are
    // fuse_spans[fuse_span_ptr[s] .. fuse_span_ptr[s + 1]) (dst_row order,
    // at most kMaxFuseSpans used), and a cached key in span i is rotated by
    // R(delta_i) (angles from freqs); NULL: the keys are used as read.
    const kvlink_span* fuse_spans;
    const int32_t* fuse_span_ptr;
    RopeFreqs freqs;
};

// Spans of one request the fused re-encode holds (their cos/sin tables sit
// in LDS beside the wide kernel's ring).
constexpr int kMaxFuseSpans = KVLINK_FUSED_MAX_SPANS;

static_assert(kSegRecord == 16, "segment records are read as four int4");
static_assert(kUnitRecord == 8, "unit records are read as two int4");

// Record g of the schedule (uniform loads).
__device__ __forceinline__ void load_record(const KParams& p, int g, int4 (&rec)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) rec[i] = p.seg[4 * (int64_t)g + i];
}

// The record's indices fit the launch: request, head, rows of one block,
// segment numbering within the unit's partials, and a chain that only moves
// forward (so a workgroup's walk ends).
__device__ __forceinline__ bool record_ok(const KParams& p, const int4 (&rec)[4], int g) {
    const int nseg = rec[1].z, loc = rec[1].w, part = rec[3].x, next = rec[3].y, unit = rec[3].z;
    return rec[0].x >= 0 && rec[0].x < p.n_seqs && rec[0].y >= 0 && rec[0].y < p.n_kv_heads &&
           rec[0].w >= 0 && rec[0].w <= p.row_block && nseg >= 1 && loc >= 0 && loc < nseg &&
           part >= 0 && part + nseg <= p.n_segments && (next < 0 || next > g) && unit >= 0 &&
           unit < p.n_units;
}

// Wait until every memory access this wave issued has completed (stores
// included), as a compiler barrier too, so no access moves across it.  With a
// workgroup barrier after it, the stores are visible to the other waves.
__device__ __forceinline__ void wait_vm_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Fused RoPE: new rows [na, nb) of request token base n0 and KV head h are
// written to the cache rows Tc + r of the views, keys rotated from k_new by
// the table, values copied from v_new (bf16; a task is 16 bytes of each half
// of one row, NT threads).  Workgroups whose key ranges overlap write the
// same rows with the same bytes.  The caller makes the stores visible
// (wait_vm_all, then a workgroup barrier) before loading those rows.
// kV = false appends the keys only (for a kernel that reads the new values
// straight from v_new and copies them into the cache by itself).
template <int D, int NT, bool kV = true>
__device__ __forceinline__ void append_new_rows(const KParams& p, const RowPtr& kp,
                                                const RowPtr& vp, int h, int n0, int Tc, int na,
                                                int nb) {
    constexpr int Hh = D / 2, TPR = Hh / 8;   // tasks per row
    const bf16_t* kn = reinterpret_cast<const bf16_t*>(p.k_new);
    const bf16_t* vn = reinterpret_cast<const bf16_t*>(p.v_new);
    for (int i = threadIdx.x; i < (nb - na) * TPR; i += NT) {
        const int r = na + i / TPR, c = 8 * (i % TPR);
        const int64_t n = n0 + r;
        const int64_t src = (n * p.n_kv_heads + h) * D + c;
        const uint4 a = *reinterpret_cast<const uint4*>(kn + src);
        const uint4 b = *reinterpret_cast<const uint4*>(kn + src + Hh);
        uint4 va, vb;
        if constexpr (kV) {
            va = *reinterpret_cast<const uint4*>(vn + src);
            vb = *reinterpret_cast<const uint4*>(vn + src + Hh);
        }
        float cs[8], sn[8];
        rope_table8(p.rope + n * Hh, c, cs, sn);
        uint4 x, y;
        rope_rotate16<bf16_t>(a, b, cs, sn, x, y);
        char* kd = const_cast<char*>(kp.row(Tc + r)) + 2 * c;
        *reinterpret_cast<uint4*>(kd) = x;
        *reinterpret_cast<uint4*>(kd + 2 * Hh) = y;
        if constexpr (kV) {
            char* vd = const_cast<char*>(vp.row(Tc + r)) + 2 * c;
            *reinterpret_cast<uint4*>(vd) = va;
            *reinterpret_cast<uint4*>(vd + 2 * Hh) = vb;
        }
    }
}

// Queries of one GQA row as the B operand pieces a lane holds (dims
// 32ds + 8lg.. for each 32-dim step ds): from the rotated-query workspace,
// or, with the fused RoPE, from q_new rotated by the table (the pairs of a
// lane are steps ds and ds + D/64).  load() only issues the loads, get()
// rotates, so a caller can let their latency overlap other loads.
template <int D>
struct QRow {
    static constexpr int DS = D / 32;
    uint4 raw[DS];
    float4 tab[DS / 2][4];

    __device__ __forceinline__ void load(const KParams& p, int64_t n, int hq, int lg) {
        const int64_t off = (n * p.n_q_heads + hq) * D + 8 * lg;
        const bf16_t* src = reinterpret_cast<const bf16_t*>(p.rope ? p.q_new : p.q_rot) + off;
#pragma unroll
        for (int ds = 0; ds < DS; ++ds) raw[ds] = *reinterpret_cast<const uint4*>(src + 32 * ds);
        if (!p.rope) return;
#pragma unroll
        for (int ds = 0; ds < DS / 2; ++ds) {
            const float4* t = reinterpret_cast<const float4*>(p.rope + n * (D / 2) + 32 * ds + 8 * lg);
#pragma unroll
            for (int i = 0; i < 4; ++i) tab[ds][i] = t[i];
        }
    }

    __device__ __forceinline__ void get(const KParams& p, uint4 (&q)[DS]) const {
        if (!p.rope) {
#pragma unroll
            for (int ds = 0; ds < DS; ++ds) q[ds] = raw[ds];
            return;
        }
#pragma unroll
        for (int ds = 0; ds < DS / 2; ++ds) {
            float cs[8], sn[8];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                cs[2 * i] = tab[ds][i].x;
                sn[2 * i] = tab[ds][i].y;
                cs[2 * i + 1] = tab[ds][i].z;
                sn[2 * i + 1] = tab[ds][i].w;
            }
            rope_rotate16<bf16_t>(raw[ds], raw[ds + DS / 2], cs, sn, q[ds], q[ds + DS / 2]);
        }
    }
};

hipError_t launch_attend_mfma(int head_dim, const KParams& p, int n_wg, hipStream_t stream);
hipError_t launch_attend_decode(int head_dim, const KParams& p, int n_wg, hipStream_t stream);
// GQA rows per unit of the wide-block (256, 128 or 64) and decode kernels
bool attend_mfma_row_block_ok(int row_block);
int attend_decode_row_block();

}  // namespace attn
}  // namespace kvlink
