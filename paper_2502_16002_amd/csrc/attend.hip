// attend.hip — one layer of the forward pass over the new tokens of KVLink
// (Sec. 2.3, last paragraph): the link tokens placed after every document
// and the query tokens attend to the concatenated, re-encoded cache.
//
// Kernels, in launch order:
//   rope_new_kernel     rotates q and k of every new token at its global
//                       position, writes the rotated q to the workspace and
//                       appends the rotated k and the v to the cache rows
//                       T_c + r of the layer (the paper appends the link
//                       tokens after the reused caches);
//   attend_*_kernel     split-K (flash-decoding style) GQA attention: a
//                       workgroup owns one KV head, a block of GQA-packed rows
//                       (row = token * group + head-in-group, so the rows of a
//                       block share the KV head and nearly the same visible
//                       range) and one split of the block's key range;
//   combine_kernel      log-sum-exp merge of the splits (skipped when one
//                       split covers every block).
//
// The attention map of a link or query token reduces to "every position at or
// before mine" (Sec. 2.3).  In cache-row terms, token r of a request sees the
// first new_visible[r] cached rows and new rows 0..r.  A row block walks a
// virtual key range: first the cached rows its last token sees (cmax), then
// the new rows up to its last token; each key is masked per row.
#include <algorithm>

#include "kvlink_internal.h"

namespace kvlink {
namespace {

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

// --------------------------------------------------------------- prologue

template <typename T, int D>
__global__ __launch_bounds__(256) void rope_new_kernel(
    const T* __restrict__ q_new, const T* __restrict__ k_new, const T* __restrict__ v_new,
    T* __restrict__ q_rot, View k, View v, int layer, int n_seqs, int n_new_total, int n_q_heads,
    int n_kv_heads, const int32_t* __restrict__ seq_new_ptr,
    const int32_t* __restrict__ seq_cached, const int32_t* __restrict__ new_pos, double theta) {
    constexpr int H = D / 2;
    const int idx = blockIdx.x * 256 + threadIdx.x;
    if (idx >= n_new_total * H) return;
    const int n = idx / H, j = idx % H;
    const int s = seq_of(seq_new_ptr, n_seqs, n);
    const int r = n - seq_new_ptr[s];
    const int row = seq_cached[s] + r;
    float c, sn;
    rope_cos_sin(new_pos[n], j, D, theta, &c, &sn);
    for (int h = 0; h < n_q_heads; ++h) {
        const int64_t o = ((int64_t)n * n_q_heads + h) * D;
        const float a = to_f32(q_new[o + j]), b = to_f32(q_new[o + j + H]);
        q_rot[o + j] = from_f32<T>(a * c - b * sn);
        q_rot[o + j + H] = from_f32<T>(a * sn + b * c);
    }
    T* kb = reinterpret_cast<T*>(k.base);
    T* vb = reinterpret_cast<T*>(v.base);
    for (int h = 0; h < n_kv_heads; ++h) {
        const int64_t o = ((int64_t)n * n_kv_heads + h) * D;
        const float a = to_f32(k_new[o + j]), b = to_f32(k_new[o + j + H]);
        const int64_t ko = view_offset(k, layer, h, s, row);
        kb[ko + j] = from_f32<T>(a * c - b * sn);
        kb[ko + j + H] = from_f32<T>(a * sn + b * c);
        const int64_t vo = view_offset(v, layer, h, s, row);
        vb[vo + j] = v_new[o + j];
        vb[vo + j + H] = v_new[o + j + H];
    }
}

// ------------------------------------------------------ VALU split kernel
//
// Used for fp32 and as the plain reference schedule: 16 GQA rows per
// workgroup (4 per wavefront), 64-key tiles staged to LDS as float, one key
// per lane for the scores, one or two head-dim columns per lane for P.V.

template <typename T, int D>
__global__ __launch_bounds__(256) void attend_valu_kernel(KParams p) {
    constexpr int RB = 16, KT = 64, RPW = 4, DPL = D / 64;
    __shared__ float s_q[RB][D];
    __shared__ float s_k[KT][D + 1];
    __shared__ float s_v[KT][D];

    const int split = blockIdx.x;
    const int s = blockIdx.z / p.n_kv_heads, h = blockIdx.z % p.n_kv_heads;
    const int n0 = p.seq_new_ptr[s];
    const int rows_s = (p.seq_new_ptr[s + 1] - n0) * p.group;
    const int rho0 = blockIdx.y * RB;
    if (rho0 >= rows_s) return;
    const BlockKeys bk = block_keys(p.new_visible, n0, rows_s, rho0, RB, p.group);
    const int kbeg = split * p.split_keys;
    if (kbeg >= bk.nvirt) return;
    const int kend = min(kbeg + p.split_keys, bk.nvirt);
    const int Tc = p.seq_cached[s];

    const T* q_rot = reinterpret_cast<const T*>(p.q_rot);
    for (int i = threadIdx.x; i < RB * D; i += 256) {
        const int row = i / D, d = i % D;
        const int rho = rho0 + row;
        float x = 0.f;
        if (rho < rows_s) {
            const int r = rho / p.group, hq = h * p.group + rho % p.group;
            x = to_f32(q_rot[((int64_t)(n0 + r) * p.n_q_heads + hq) * D + d]);
        }
        s_q[row][d] = x;
    }

    const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
    float m[RPW], l[RPW], o[RPW][DPL];
    int vis[RPW], tok[RPW];
    bool valid[RPW];
#pragma unroll
    for (int i = 0; i < RPW; ++i) {
        const int rho = rho0 + wave * RPW + i;
        valid[i] = rho < rows_s;
        tok[i] = valid[i] ? rho / p.group : 0;
        vis[i] = valid[i] ? p.new_visible[n0 + tok[i]] : 0;
        m[i] = -INFINITY;
        l[i] = 0.f;
#pragma unroll
        for (int dd = 0; dd < DPL; ++dd) o[i][dd] = 0.f;
    }

    const T* kb = reinterpret_cast<const T*>(p.k.base);
    const T* vb = reinterpret_cast<const T*>(p.v.base);
    for (int t0 = kbeg; t0 < kend; t0 += KT) {
        __syncthreads();
        for (int i = threadIdx.x; i < KT * D; i += 256) {
            const int key = i / D, d = i % D;
            const int vk = t0 + key;
            float kx = 0.f, vx = 0.f;
            if (vk < kend) {
                const int row = vk < bk.cmax ? vk : Tc + (vk - bk.cmax);
                kx = to_f32(kb[view_offset(p.k, p.layer, h, s, row) + d]);
                vx = to_f32(vb[view_offset(p.v, p.layer, h, s, row) + d]);
            }
            s_k[key][d] = kx;
            s_v[key][d] = vx;
        }
        __syncthreads();
        const int vk = t0 + lane;
#pragma unroll
        for (int i = 0; i < RPW; ++i) {
            if (!valid[i]) continue;
            const int row = wave * RPW + i;
            float sc = 0.f;
#pragma unroll 8
            for (int d = 0; d < D; ++d) sc += s_q[row][d] * s_k[lane][d];
            const bool ok = vk < kend && (vk < bk.cmax ? vk < vis[i] : (vk - bk.cmax) <= tok[i]);
            sc = ok ? sc * p.scale_log2 : -INFINITY;
            const float m_new = fmaxf(m[i], wave_max(sc));
            if (m_new == -INFINITY) continue;
            const float alpha = exp2f(m[i] - m_new);
            const float pr = ok ? exp2f(sc - m_new) : 0.f;
            l[i] = l[i] * alpha + wave_sum(pr);
            m[i] = m_new;
#pragma unroll
            for (int dd = 0; dd < DPL; ++dd) o[i][dd] *= alpha;
#pragma unroll
            for (int j = 0; j < KT; ++j) {
                const float pj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(pr), j));
#pragma unroll
                for (int dd = 0; dd < DPL; ++dd) o[i][dd] += pj * s_v[j][lane + 64 * dd];
            }
        }
    }

#pragma unroll
    for (int i = 0; i < RPW; ++i) {
        if (!valid[i]) continue;
        const int rho = rho0 + wave * RPW + i;
        const int hq = h * p.group + rho % p.group;
        const int64_t orow = (int64_t)(n0 + tok[i]) * p.n_q_heads + hq;
        if (p.n_splits == 1) {
            T* out = reinterpret_cast<T*>(p.out);
            const float inv = 1.f / l[i];
#pragma unroll
            for (int dd = 0; dd < DPL; ++dd) out[orow * D + lane + 64 * dd] = from_f32<T>(o[i][dd] * inv);
            if (p.lse && lane == 0) p.lse[orow] = (m[i] + log2f(l[i])) * kLn2;
        } else {
            const int64_t pi = orow * p.n_splits + split;
#pragma unroll
            for (int dd = 0; dd < DPL; ++dd) p.part_o[pi * D + lane + 64 * dd] = o[i][dd];
            if (lane == 0) {
                p.part_ml[pi * 2] = m[i];
                p.part_ml[pi * 2 + 1] = l[i];
            }
        }
    }
}

// ------------------------------------------------------------- combine

template <typename T, int D>
__global__ __launch_bounds__(256) void combine_kernel(KParams p, int n_new_total) {
    constexpr int DPL = D / 64;
    const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
    const int64_t orow = (int64_t)blockIdx.x * 4 + wave;   // (n, hq) flattened
    if (orow >= (int64_t)n_new_total * p.n_q_heads) return;
    const int n = (int)(orow / p.n_q_heads), hq = (int)(orow % p.n_q_heads);
    const int s = seq_of(p.seq_new_ptr, p.n_seqs, n);
    const int n0 = p.seq_new_ptr[s];
    const int rows_s = (p.seq_new_ptr[s + 1] - n0) * p.group;
    const int rho = (n - n0) * p.group + hq % p.group;
    const int rho0 = rho / p.row_block * p.row_block;
    const BlockKeys bk = block_keys(p.new_visible, n0, rows_s, rho0, p.row_block, p.group);
    const int nsp = (bk.nvirt + p.split_keys - 1) / p.split_keys;

    float M = -INFINITY;
    for (int c = 0; c < nsp; ++c) M = fmaxf(M, p.part_ml[(orow * p.n_splits + c) * 2]);
    float L = 0.f, acc[DPL];
#pragma unroll
    for (int dd = 0; dd < DPL; ++dd) acc[dd] = 0.f;
    for (int c = 0; c < nsp; ++c) {
        const int64_t pi = orow * p.n_splits + c;
        const float mc = p.part_ml[pi * 2];
        if (mc == -INFINITY) continue;
        const float w = exp2f(mc - M);
        L += w * p.part_ml[pi * 2 + 1];
#pragma unroll
        for (int dd = 0; dd < DPL; ++dd) acc[dd] += w * p.part_o[pi * D + lane + 64 * dd];
    }
    T* out = reinterpret_cast<T*>(p.out);
    const float inv = 1.f / L;
#pragma unroll
    for (int dd = 0; dd < DPL; ++dd) out[orow * D + lane + 64 * dd] = from_f32<T>(acc[dd] * inv);
    if (p.lse && lane == 0) p.lse[orow] = (M + log2f(L)) * kLn2;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

template <typename T, int D>
hipError_t launch_typed(const AttendPlan& pl, const AttendArgs& a, hipStream_t stream) {
    char* ws = reinterpret_cast<char*>(a.workspace);
    T* q_rot = reinterpret_cast<T*>(ws);
    KParams p;
    p.q_rot = q_rot;
    p.k = a.k;
    p.v = a.v;
    p.layer = a.layer;
    p.n_seqs = pl.n_seqs;
    p.n_q_heads = pl.n_q_heads;
    p.n_kv_heads = pl.n_kv_heads;
    p.group = pl.group;
    p.seq_new_ptr = a.seq_new_ptr;
    p.seq_cached = a.seq_cached;
    p.new_visible = a.new_visible;
    p.scale_log2 = a.scale * kLog2e;
    p.split_keys = pl.split_keys;
    p.n_splits = pl.n_splits;
    p.row_block = pl.row_block;
    p.part_o = reinterpret_cast<float*>(ws + pl.q_rot_bytes);
    p.part_ml = reinterpret_cast<float*>(ws + pl.q_rot_bytes + pl.part_o_bytes);
    p.out = a.out;
    p.lse = a.lse;

    const int n_pairs = pl.n_new_total * (D / 2);
    hipLaunchKernelGGL((rope_new_kernel<T, D>), dim3((n_pairs + 255) / 256), dim3(256), 0, stream,
                       reinterpret_cast<const T*>(a.q_new), reinterpret_cast<const T*>(a.k_new),
                       reinterpret_cast<const T*>(a.v_new), q_rot, a.k, a.v, a.layer, pl.n_seqs,
                       pl.n_new_total, pl.n_q_heads, pl.n_kv_heads, a.seq_new_ptr, a.seq_cached,
                       a.new_pos, a.theta);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;

    const int n_rb = (pl.max_new * pl.group + pl.row_block - 1) / pl.row_block;
    dim3 grid(pl.n_splits, n_rb, pl.n_seqs * pl.n_kv_heads);
    hipLaunchKernelGGL((attend_valu_kernel<T, D>), grid, dim3(256), 0, stream, p);
    e = hipGetLastError();
    if (e != hipSuccess || pl.n_splits == 1) return e;

    const int64_t n_rows = (int64_t)pl.n_new_total * pl.n_q_heads;
    hipLaunchKernelGGL((combine_kernel<T, D>), dim3((unsigned)((n_rows + 3) / 4)), dim3(256), 0,
                       stream, p, pl.n_new_total);
    return hipGetLastError();
}

}  // namespace

bool make_attend_plan(kvlink_dtype dt, int n_q_heads, int n_kv_heads, int head_dim, int n_seqs,
                      int n_new_total, int max_new, int max_cached, int split_keys,
                      AttendPlan* p) {
    if (n_q_heads < 1 || n_kv_heads < 1 || n_q_heads % n_kv_heads) return false;
    if (head_dim != 64 && head_dim != 128) return false;
    if (n_seqs < 1 || n_new_total < 0 || max_new < 0 || max_cached < 0) return false;
    if (split_keys < 0 || split_keys % 128) return false;
    const size_t elem = dt == KVLINK_BF16 ? 2 : 4;
    p->n_q_heads = n_q_heads;
    p->n_kv_heads = n_kv_heads;
    p->group = n_q_heads / n_kv_heads;
    p->head_dim = head_dim;
    p->n_seqs = n_seqs;
    p->n_new_total = n_new_total;
    p->max_new = max_new;
    p->max_cached = max_cached;
    p->use_mfma = false;
    p->row_block = 16;
    const int64_t max_keys = (int64_t)max_cached + max_new;
    if (split_keys == 0) {
        // aim at about 1024 workgroups in total, splits of at least 256 keys
        const int64_t n_rb = (int64_t)n_seqs * n_kv_heads *
                             (((int64_t)max_new * p->group + p->row_block - 1) / p->row_block);
        const int64_t want_splits = n_rb > 0 ? (1024 + n_rb - 1) / n_rb : 1;
        int64_t sk = (max_keys + want_splits - 1) / std::max<int64_t>(want_splits, 1);
        sk = (sk + 127) / 128 * 128;
        split_keys = (int)std::max<int64_t>(256, sk);
    }
    p->split_keys = split_keys;
    p->n_splits = (int)std::max<int64_t>(1, (max_keys + split_keys - 1) / split_keys);
    const int64_t rows = (int64_t)n_new_total * n_q_heads;
    p->q_rot_bytes = align256((size_t)rows * head_dim * elem);
    if (p->n_splits > 1) {
        p->part_o_bytes = align256((size_t)rows * p->n_splits * head_dim * sizeof(float));
        p->part_ml_bytes = align256((size_t)rows * p->n_splits * 2 * sizeof(float));
    } else {
        p->part_o_bytes = p->part_ml_bytes = 0;
    }
    p->total_bytes = std::max<size_t>(256, p->q_rot_bytes + p->part_o_bytes + p->part_ml_bytes);
    return true;
}

hipError_t launch_attend(kvlink_dtype dt, const AttendPlan& p, const AttendArgs& a,
                         hipStream_t stream) {
    if (dt == KVLINK_BF16)
        return p.head_dim == 128 ? launch_typed<bf16_t, 128>(p, a, stream)
                                 : launch_typed<bf16_t, 64>(p, a, stream);
    return p.head_dim == 128 ? launch_typed<float, 128>(p, a, stream)
                             : launch_typed<float, 64>(p, a, stream);
}

}  // namespace kvlink
