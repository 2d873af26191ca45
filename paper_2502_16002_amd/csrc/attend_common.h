// attend_common.h — definitions shared by the attention kernels.
#pragma once

#include "kvlink_internal.h"

namespace kvlink {
namespace attn {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

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

// Arguments of the split kernels and the combine.
struct KParams {
    const void* q_rot;
    View k, v;
    int layer, n_seqs, n_q_heads, n_kv_heads, group;
    const int32_t* seq_new_ptr;
    const int32_t* seq_cached;
    const int32_t* new_visible;
    float scale_log2;
    int split_keys, n_splits, row_block;
    float* part_o;
    float* part_ml;
    void* out;
    float* lse;
};


hipError_t launch_attend_mfma(int head_dim, const KParams& p, dim3 grid, hipStream_t stream);
// GQA rows per workgroup of the MFMA kernel
int attend_mfma_row_block();

}  // namespace attn
}  // namespace kvlink
