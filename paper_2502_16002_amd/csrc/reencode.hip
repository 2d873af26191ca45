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
//   * a workgroup owns up to kRows rows of one document for kLH (layer, head)
//     pairs, so the document's cos/sin table is built once (double-precision
//     angles reduced and evaluated in registers, stored to LDS) and then held
//     in registers: each thread always handles the same slice of the rotation
//     pairs;
//   * each thread moves 16-byte vectors: the slice [j0, j0+E) and its partner
//     slice [j0+d/2, j0+d/2+E), consecutive threads cover one row, then the
//     next row, so a wavefront reads and writes whole contiguous rows;
//   * kUnroll vectors are loaded before any is stored, to keep enough bytes in
//     flight per wavefront;
//   * loads and stores are non-temporal (every byte is touched once), and a
//     workgroup covers 16 rows, so the many short documents of a request
//     spread evenly over the compute units.
#include "kvlink_internal.h"

namespace kvlink {
namespace {

constexpr int kThreads = 256;
constexpr int kRows = 16;
constexpr int kLH = 8;
constexpr int kUnroll = 4;

typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 load_stream(const void* p) {
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
    return uint4{v.x, v.y, v.z, v.w};
}

__device__ __forceinline__ void store_stream(const uint4& v, void* p) {
    __builtin_nontemporal_store(u32x4_t{v.x, v.y, v.z, v.w}, reinterpret_cast<u32x4_t*>(p));
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
    const int lh0 = blockIdx.z * kLH;
    const int nlh = min(kLH, n_lh - lh0);

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

    const int sub = threadIdx.x % TPV;
    float c[E], s[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        c[e] = kMode == kCopy ? 1.f : s_cos[0][sub * E + e];
        s[e] = kMode == kCopy ? 0.f : s_sin[0][sub * E + e];
    }

    const int n_vec = rows * nlh;
    for (int v0 = threadIdx.x / TPV; v0 < n_vec; v0 += VPP * kUnroll) {
        uint4 lo[kUnroll], hi[kUnroll];
        int64_t doff[kUnroll];
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
                float a[E], b[E], x[E], y[E];
                unpack16<T>(lo[u], a);
                unpack16<T>(hi[u], b);
                if constexpr (kMode == kPerToken) {
                    const int row = v % rows;
#pragma unroll
                    for (int e = 0; e < E; ++e) {
                        c[e] = s_cos[row][sub * E + e];
                        s[e] = s_sin[row][sub * E + e];
                    }
                }
#pragma unroll
                for (int e = 0; e < E; ++e) {
                    x[e] = a[e] * c[e] - b[e] * s[e];
                    y[e] = a[e] * s[e] + b[e] * c[e];
                }
                store_stream(pack16<T>(x), q);
                store_stream(pack16<T>(y), q + H);
            }
        }
    }
}

template <typename T, int D>
hipError_t launch(int n_layers, int n_kv_heads, const RopeFreqs& freqs, int n_spans,
                  const kvlink_span* spans, int max_span_len, const View& src, const View& dst,
                  int mode, const int32_t* pos_map, int64_t pos_stride, hipStream_t stream) {
    const int n_lh = n_layers * n_kv_heads;
    dim3 grid((max_span_len + kRows - 1) / kRows, n_spans, (n_lh + kLH - 1) / kLH);
    if (mode == kPerToken)
        hipLaunchKernelGGL((reencode_kernel<T, D, kPerToken>), grid, dim3(kThreads), 0, stream,
                           src, dst, spans, n_lh, n_kv_heads, freqs, pos_map, pos_stride);
    else if (mode == kCopy)
        hipLaunchKernelGGL((reencode_kernel<T, D, kCopy>), grid, dim3(kThreads), 0, stream, src,
                           dst, spans, n_lh, n_kv_heads, freqs, nullptr, (int64_t)0);
    else
        hipLaunchKernelGGL((reencode_kernel<T, D, kDelta>), grid, dim3(kThreads), 0, stream, src,
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

}  // namespace kvlink
