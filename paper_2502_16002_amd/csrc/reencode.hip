// reencode.hip — positional re-encoding of cached keys (KVLink Sec. 2.2).
//
// Keys of a document were stored with RoPE at the positions they had when the
// document was encoded alone.  After concatenation the document starts at
// global offset g_i, so every stored key is rotated once more, by
// R(delta_i) with delta_i = g_i - (its stored start position); rotations
// compose, R(delta) R(t) = R(delta + t).  Values are not touched.
//
// The paper's literal storage form keeps keys without any rotation and
// applies the global rotation at inference: key t of document i is rotated
// by R(delta_i + t) (delta_i = g_i for keys stored from position 0).  The same
// kernel does this with a per-row cos/sin table (kPerToken).  A compressed
// cache (Sec. 2.4: only some tokens' keys kept, at their original positions
// p_t) is re-encoded to contiguous global positions with R(delta_i + t - p_t),
// p_t read from a per-row map of stored positions.
//
// The pass is bound by HBM bandwidth (about 1.5 flop per byte moved):
//   * one launch covers every layer and KV head, since delta does not depend
//     on them;
//   * a workgroup owns up to kRows rows of one document for lh_per_wg(D)
//     (layer, head) pairs (8 KiB of bf16 keys at head_dim 128, one 16-byte
//     vector pair per thread), so the document's cos/sin table is built once
//     (double-precision angles reduced and evaluated in registers, stored to
//     LDS) and then held in registers: each thread always handles the same
//     slice of the rotation pairs; the first loads are issued before the table
//     is built, so that its work overlaps their latency;
//   * each thread moves 16-byte vectors: the slice [j0, j0+E) and its partner
//     slice [j0+d/2, j0+d/2+E), consecutive threads cover one row, then the
//     next row, so a wavefront reads and writes whole contiguous rows;
//   * kUnroll vectors are loaded before any is stored, to keep enough bytes in
//     flight per wavefront;
//   * loads and stores are non-temporal (every byte is touched once), and a
//     workgroup covers 8 rows, so the many short documents of a request
//     spread evenly over the compute units;
//   * a grid of at least kLongGrid workgroups (a long-context batch: a
//     steady stream, ramp and tail negligible) runs with at most
//     kLongResident workgroups resident per CU, capped through their LDS
//     allocation: on MI355X fewer concurrent streams then sustain a higher
//     HBM rate (79-80% of peak against 76-77% at full residency, 40 x 512
//     tokens x 32 layers x 8 heads), while short grids keep full residency
//     (there ramp and tail dominate and the cap costs 3-15%).
#include "kvlink_internal.h"

namespace kvlink {
namespace {

constexpr int kThreads = 256;
constexpr int kRows = 8;
constexpr int kUnroll = 2;
constexpr int kLongGrid = 65536;
constexpr int kLongResident = 6;
constexpr int kLdsPerCu = 160 * 1024;

// (layer, head) pairs per workgroup of the per-span kernel: 32 rows of
// head_dim 128 (4 pairs x 8 rows), scaled so a workgroup always holds 32 x 128
// elements.
__host__ __device__ constexpr int lh_per_wg(int D) { return 4 * 128 / D; }

typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 load_stream(const void* p) {
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
    return uint4{v.x, v.y, v.z, v.w};
}

__device__ __forceinline__ void store_stream(const uint4& v, void* p) {
    __builtin_nontemporal_store(u32x4_t{v.x, v.y, v.z, v.w}, reinterpret_cast<u32x4_t*>(p));
}

// Rotation of one 16-byte slice pair (dims j.. and j + D/2..) by (c, s) and
// its non-temporal store at q (the slice) and q + D/2 (its partner); the
// per-span and the shared kernels both go through it, so they write the same
// bytes (and the same as the re-encode fused into the split attention).
template <typename T, int D>
__device__ __forceinline__ void rotate_store(const uint4& lo, const uint4& hi, const float* c,
                                             const float* s, T* q) {
    uint4 x, y;
    rope_rotate16<T>(lo, hi, c, s, x, y);
    store_stream(x, q);
    store_stream(y, q + D / 2);
}

// Modes: kDelta rotates every row of a span by R(delta); kPerToken rotates
// row t by R(delta + t) (keys stored without rotation); kCopy moves the rows
// unchanged (values gathered through the same spans).
enum { kDelta = 0, kPerToken = 1, kCopy = 2 };

// pos_map (kPerToken only, may be NULL): stored position of every source row,
// entry src_seq * pos_stride + row; the angle of row t is delta + t - pos.
template <typename T, int D, int kMode>
__global__ __launch_bounds__(kThreads) void reencode_kernel(View src, View dst,
                                                            const kvlink_span* __restrict__ spans,
                                                            int n_lh, int n_kv_heads,
                                                            RopeFreqs freqs,
                                                            const int32_t* __restrict__ pos_map,
                                                            int64_t pos_stride) {
    constexpr int H = D / 2;                 // rotation pairs per vector
    constexpr int E = 16 / (int)sizeof(T);   // elements per 16-byte access
    constexpr int TPV = H / E;               // threads per vector
    constexpr int VPP = kThreads / TPV;      // vectors per pass of the workgroup
    constexpr int TR = kMode == kPerToken ? kRows : 1;   // rows of the cos/sin table
    __shared__ float s_cos[TR][H], s_sin[TR][H];

    const kvlink_span sp = spans[blockIdx.y];
    const int r0 = blockIdx.x * kRows;
    if (r0 >= sp.len) return;
    const int rows = min(kRows, sp.len - r0);
    constexpr int kLH = lh_per_wg(D);
    const int lh0 = blockIdx.z * kLH;
    const int nlh = min(kLH, n_lh - lh0);

    const int sub = threadIdx.x % TPV;
    const int n_vec = rows * nlh;
    uint4 lo[kUnroll], hi[kUnroll];
    int64_t doff[kUnroll];
    auto load_round = [&](int v0) {
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int v = v0 + u * VPP;
            if (v < n_vec) {
                const int lh = lh0 + v / rows;
                const int row = v % rows;
                const int layer = lh / n_kv_heads, head = lh % n_kv_heads;
                const int64_t so =
                    view_offset(src, layer, head, sp.src_seq, sp.src_row + r0 + row) + sub * E;
                const T* p = reinterpret_cast<const T*>(src.base) + so;
                lo[u] = load_stream(p);
                hi[u] = load_stream(p + H);
                doff[u] = view_offset(dst, layer, head, sp.dst_seq, sp.dst_row + r0 + row) + sub * E;
            }
        }
    };
    // the first round of loads goes out before the cos/sin table is built,
    // so that the table's double-precision work overlaps their latency
    const int v_first = threadIdx.x / TPV;
    load_round(v_first);

    if constexpr (kMode != kCopy) {
        for (int i = threadIdx.x; i < TR * H; i += kThreads) {
            const int tr = i / H, j = i % H;
            int64_t pos = (int64_t)sp.delta;
            if constexpr (kMode == kPerToken) {
                pos += r0 + tr;
                if (pos_map && r0 + tr < sp.len)
                    pos -= pos_map[(int64_t)sp.src_seq * pos_stride + sp.src_row + r0 + tr];
            }
            rope_cos_sin(pos, j, freqs, &s_cos[tr][j], &s_sin[tr][j]);
        }
        __syncthreads();
    }

    float c[E], s[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        c[e] = kMode == kCopy ? 1.f : s_cos[0][sub * E + e];
        s[e] = kMode == kCopy ? 0.f : s_sin[0][sub * E + e];
    }

    for (int v0 = v_first; v0 < n_vec; v0 += VPP * kUnroll) {
        if (v0 != v_first) load_round(v0);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int v = v0 + u * VPP;
            if (v < n_vec) {
                T* q = reinterpret_cast<T*>(dst.base) + doff[u];
                if constexpr (kMode == kCopy) {
                    store_stream(lo[u], q);
                    store_stream(hi[u], q + H);
                    continue;
                }
                if constexpr (kMode == kPerToken) {
                    const int row = v % rows;
#pragma unroll
                    for (int e = 0; e < E; ++e) {
                        c[e] = s_cos[row][sub * E + e];
                        s[e] = s_sin[row][sub * E + e];
                    }
                }
                rotate_store<T, D>(lo[u], hi[u], c, s, q);
            }
        }
    }
}

// Document-major re-encode: the spans of group g (spans[group_ptr[g] ..
// group_ptr[g+1])) all read the same stored rows (one document reused by
// several requests, each at its own global offset).  A workgroup loads its
// kRowsS rows x kLHS (layer, head) pairs of the group's document once, then
// for each span rotates them by that span's delta and stores them at the
// span's destination: the stored rows are read once per group instead of
// once per span.  The cos/sin tables of up to kMaxDst spans are built per
// round (double-precision angles, in LDS), together with the destinations'
// span records and page offsets; the first round's table work overlaps the
// loads.
constexpr int kMaxDst = 32;
constexpr int kRowsS = 16;  // rows per workgroup of the shared kernel
constexpr int kLHS = 4;     // (layer, head) pairs per workgroup of the shared kernel

template <typename T, int D>
__global__ __launch_bounds__(kThreads) void reencode_shared_kernel(
    View src, View dst, const kvlink_span* __restrict__ spans,
    const int32_t* __restrict__ group_ptr, int n_lh, int n_kv_heads, RopeFreqs freqs) {
    constexpr int H = D / 2;
    constexpr int E = 16 / (int)sizeof(T);
    constexpr int TPV = H / E;
    constexpr int VPP = kThreads / TPV;
    constexpr int NB = (kRowsS * kLHS + VPP - 1) / VPP;  // vectors per thread
    __shared__ float s_cos[kMaxDst][H], s_sin[kMaxDst][H];
    __shared__ kvlink_span s_dst[kMaxDst];
    __shared__ int64_t s_base[kMaxDst];

    const int sp0 = group_ptr[blockIdx.y], sp1 = group_ptr[blockIdx.y + 1];
    if (sp1 <= sp0) return;
    const kvlink_span first = spans[sp0];
    const int r0 = blockIdx.x * kRowsS;
    if (r0 >= first.len) return;
    const int rows = min(kRowsS, first.len - r0);
    const int lh0 = blockIdx.z * kLHS;
    const int nlh = min(kLHS, n_lh - lh0);
    const int sub = threadIdx.x % TPV;
    const int n_vec = rows * nlh;

    uint4 lo[NB], hi[NB];
#pragma unroll
    for (int u = 0; u < NB; ++u) {
        const int v = threadIdx.x / TPV + u * VPP;
        if (v < n_vec) {
            const int lh = lh0 + v / rows, row = v % rows;
            const T* p = reinterpret_cast<const T*>(src.base) +
                         view_offset(src, lh / n_kv_heads, lh % n_kv_heads, first.src_seq,
                                     first.src_row + r0 + row) +
                         sub * E;
            lo[u] = load_stream(p);
            hi[u] = load_stream(p + H);
        }
    }

    for (int c0 = sp0; c0 < sp1; c0 += kMaxDst) {
        const int nd = min(kMaxDst, sp1 - c0);
        __syncthreads();   // the previous round's tables are no longer read
        // one thread per destination fetches its span record and, when its
        // rows lie in one page (or the view is contiguous), the element offset
        // of its first row from one block-table read: all destinations' reads
        // are in flight together, not one dependent chain per destination
        if (threadIdx.x < nd) {
            const kvlink_span sp = spans[c0 + threadIdx.x];
            const int drow0 = sp.dst_row + r0;
            int64_t base = -1;
            if (dst.block_table) {
                if (drow0 % dst.page_size + rows <= dst.page_size)
                    base = (int64_t)dst.block_table[(int64_t)sp.dst_seq * dst.max_pages +
                                                    drow0 / dst.page_size] * dst.page_stride +
                           (int64_t)(drow0 % dst.page_size) * dst.row_stride;
            } else {
                base = (int64_t)sp.dst_seq * dst.seq_stride + (int64_t)drow0 * dst.row_stride;
            }
            s_dst[threadIdx.x] = sp;
            s_base[threadIdx.x] = base;
        }
        for (int i = threadIdx.x; i < nd * H; i += kThreads) {
            const int k = i / H, j = i % H;
            rope_cos_sin((int64_t)spans[c0 + k].delta, j, freqs, &s_cos[k][j], &s_sin[k][j]);
        }
        __syncthreads();
        for (int k = 0; k < nd; ++k) {
            float c[E], s[E];
#pragma unroll
            for (int e = 0; e < E; ++e) {
                c[e] = s_cos[k][sub * E + e];
                s[e] = s_sin[k][sub * E + e];
            }
            const int64_t base = s_base[k];
#pragma unroll
            for (int u = 0; u < NB; ++u) {
                const int v = threadIdx.x / TPV + u * VPP;
                if (v < n_vec) {
                    const int lh = lh0 + v / rows, row = v % rows;
                    const int layer = lh / n_kv_heads, head = lh % n_kv_heads;
                    const int64_t off =
                        base >= 0 ? (int64_t)layer * dst.layer_stride +
                                        (int64_t)head * dst.head_stride + base +
                                        (int64_t)row * dst.row_stride
                                  : view_offset(dst, layer, head, s_dst[k].dst_seq,
                                                s_dst[k].dst_row + r0 + row);
                    rotate_store<T, D>(lo[u], hi[u], c, s,
                                       reinterpret_cast<T*>(dst.base) + off + sub * E);
                }
            }
        }
    }
}

template <typename T, int D>
hipError_t launch_shared(int n_layers, int n_kv_heads, const RopeFreqs& freqs, int n_groups,
                         const int32_t* group_ptr, const kvlink_span* spans, int max_span_len,
                         const View& src, const View& dst, hipStream_t stream) {
    const int n_lh = n_layers * n_kv_heads;
    dim3 grid((max_span_len + kRowsS - 1) / kRowsS, n_groups, (n_lh + kLHS - 1) / kLHS);
    hipLaunchKernelGGL((reencode_shared_kernel<T, D>), grid, dim3(kThreads), 0, stream, src, dst,
                       spans, group_ptr, n_lh, n_kv_heads, freqs);
    return hipGetLastError();
}

template <typename T, int D>
hipError_t launch(int n_layers, int n_kv_heads, const RopeFreqs& freqs, int n_spans,
                  const kvlink_span* spans, int max_span_len, const View& src, const View& dst,
                  int mode, const int32_t* pos_map, int64_t pos_stride, hipStream_t stream) {
    const int n_lh = n_layers * n_kv_heads;
    constexpr int kLH = lh_per_wg(D);
    dim3 grid((max_span_len + kRows - 1) / kRows, n_spans, (n_lh + kLH - 1) / kLH);
    // residency cap of long grids: dynamic LDS that, with the kernel's own
    // cos/sin table, fills kLdsPerCu / kLongResident per workgroup
    const unsigned table = 2u * (mode == kPerToken ? kRows : 1) * (D / 2) * (unsigned)sizeof(float);
    const unsigned lds = (int64_t)grid.x * grid.y * grid.z >= kLongGrid
                             ? kLdsPerCu / kLongResident - table
                             : 0u;
    if (mode == kPerToken)
        hipLaunchKernelGGL((reencode_kernel<T, D, kPerToken>), grid, dim3(kThreads), lds, stream,
                           src, dst, spans, n_lh, n_kv_heads, freqs, pos_map, pos_stride);
    else if (mode == kCopy)
        hipLaunchKernelGGL((reencode_kernel<T, D, kCopy>), grid, dim3(kThreads), lds, stream, src,
                           dst, spans, n_lh, n_kv_heads, freqs, nullptr, (int64_t)0);
    else
        hipLaunchKernelGGL((reencode_kernel<T, D, kDelta>), grid, dim3(kThreads), lds, stream, src,
                           dst, spans, n_lh, n_kv_heads, freqs, nullptr, (int64_t)0);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_reencode(kvlink_dtype dt, int head_dim, int n_layers, int n_kv_heads,
                           const RopeFreqs& freqs, int n_spans, const kvlink_span* spans,
                           int max_span_len, const View& src, const View& dst, int mode,
                           hipStream_t stream, const int32_t* pos_map, int64_t pos_stride) {
    if (dt == KVLINK_BF16) {
        if (head_dim == 128)
            return launch<bf16_t, 128>(n_layers, n_kv_heads, freqs, n_spans, spans, max_span_len,
                                       src, dst, mode, pos_map, pos_stride, stream);
        return launch<bf16_t, 64>(n_layers, n_kv_heads, freqs, n_spans, spans, max_span_len, src,
                                  dst, mode, pos_map, pos_stride, stream);
    }
    if (head_dim == 128)
        return launch<float, 128>(n_layers, n_kv_heads, freqs, n_spans, spans, max_span_len, src,
                                  dst, mode, pos_map, pos_stride, stream);
    return launch<float, 64>(n_layers, n_kv_heads, freqs, n_spans, spans, max_span_len, src, dst,
                             mode, pos_map, pos_stride, stream);
}

hipError_t launch_reencode_shared(kvlink_dtype dt, int head_dim, int n_layers, int n_kv_heads,
                                  const RopeFreqs& freqs, int n_groups, const int32_t* group_ptr,
                                  const kvlink_span* spans, int max_span_len, const View& src,
                                  const View& dst, hipStream_t stream) {
    if (dt == KVLINK_BF16) {
        if (head_dim == 128)
            return launch_shared<bf16_t, 128>(n_layers, n_kv_heads, freqs, n_groups, group_ptr,
                                              spans, max_span_len, src, dst, stream);
        return launch_shared<bf16_t, 64>(n_layers, n_kv_heads, freqs, n_groups, group_ptr, spans,
                                         max_span_len, src, dst, stream);
    }
    if (head_dim == 128)
        return launch_shared<float, 128>(n_layers, n_kv_heads, freqs, n_groups, group_ptr, spans,
                                         max_span_len, src, dst, stream);
    return launch_shared<float, 64>(n_layers, n_kv_heads, freqs, n_groups, group_ptr, spans,
                                    max_span_len, src, dst, stream);
}

}  // namespace kvlink
