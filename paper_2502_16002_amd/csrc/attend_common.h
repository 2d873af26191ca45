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

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
    return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
    return x;
}

// Request of global new token n (binary search over seq_new_ptr).
__device__ __forceinline__ int seq_of(const int32_t* seq_new_ptr, int n_seqs, int n) {
    int lo = 0, hi = n_seqs - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (seq_new_ptr[mid] <= n) lo = mid; else hi = mid - 1;
    }
    return lo;
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
    void* out;
    float* lse;
};

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
    const int nseg = rec[1].z, loc = rec[1].w, part = rec[3].x, next = rec[3].y;
    return rec[0].x >= 0 && rec[0].x < p.n_seqs && rec[0].y >= 0 && rec[0].y < p.n_kv_heads &&
           rec[0].w >= 0 && rec[0].w <= p.row_block && nseg >= 1 && loc >= 0 && loc < nseg &&
           part >= 0 && part + nseg <= p.n_segments && (next < 0 || next > g);
}

hipError_t launch_attend_mfma(int head_dim, const KParams& p, int n_wg, hipStream_t stream);
hipError_t launch_attend_decode(int head_dim, const KParams& p, int n_wg, hipStream_t stream);
// GQA rows per unit of the wide-block and decode kernels
int attend_mfma_row_block();
int attend_decode_row_block();

}  // namespace attn
}  // namespace kvlink
