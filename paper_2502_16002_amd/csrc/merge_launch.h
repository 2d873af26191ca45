// merge_launch.h — merge of a split unit's partials inside the launch that
// computed them: agent-coherent partial stores, coherent reloads, and the
// last-arriving workgroup's merge of the segments' softmax partials (each
// segment's normalised output weighted by its sum and by 2^(its maximum - the
// overall maximum)), so no second launch is needed.
#pragma once

#include "attend_common.h"
#include "mfma_ops.h"

namespace kvlink {
namespace attn {
namespace {

// 8-byte stores coherent at agent scope (they bypass the non-coherent
// caches), for the partials one workgroup writes and another, possibly on
// another XCD, reads in the same launch.
__device__ __forceinline__ void store_agent(void* p, uint32_t lo, uint32_t hi) {
    __hip_atomic_store(reinterpret_cast<uint64_t*>(p), ((uint64_t)hi << 32) | lo,
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// 16-byte loads coherent at agent scope, through a buffer resource over the
// partials (sc1: they do not take stale lines from a non-coherent cache);
// plain loads to the compiler, so a batch of them goes out together.
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ __amdgpu_buffer_rsrc_t coherent_rsrc(const void* base) {
    // descriptor word 3 of gfx9 buffer resources (32-bit data format)
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, 0x7fffffff, 0x00020000);
}
__device__ __forceinline__ uint4 load_coherent16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
#if defined(__HIP_DEVICE_COMPILE__)
    const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 16);
    return uint4{v.x, v.y, v.z, v.w};
#else
    return uint4{0u, 0u, 0u, 0u};
#endif
}
typedef unsigned u32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint2 load_coherent8(__amdgpu_buffer_rsrc_t r, uint32_t off) {
#if defined(__HIP_DEVICE_COMPILE__)
    const u32x2_t v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 16);
    return uint2{v.x, v.y};
#else
    return uint2{0u, 0u};
#endif
}

// The last-arriving workgroup of a split unit merges its partials: rows
// [0, rows) of the unit, each with nseg partials from entry part * kRB +
// row * nseg on (O / l bf16, (m, l) float).  A row is handled by LPS = D / 8
// lanes, each holding 16 bytes (8 dims) of every partial vector; the
// workgroup's lane groups take RPP rows per pass, P passes.  The segments
// are taken in chunks of SC, each chunk's loads for every pass issued
// together (at most 32 vectors per lane in flight) before any is used; a
// row's state (running maximum M, sum L, 8 accumulators) carries across
// chunks.  out = sum_s w_s (O/l)_s / sum_s w_s, w_s = 2^(m_s - M) l_s; the
// running maximum starts finite, so a segment that saw no key of a row
// weighs 0.
template <int D, int kRB, int kThreads>
__device__ void merge_unit(const KParams& p, int part, int rows, int nseg, int h, int rho0,
                           int n0) {
    constexpr int LPS = D / 8;                     // lanes per row
    constexpr int RPP = kThreads / LPS;            // rows per pass of the workgroup
    constexpr int P = (kRB + RPP - 1) / RPP;       // passes
    constexpr int SC = (32 / P < LPS) ? 32 / P : LPS;   // segments per chunk
    static_assert(SC >= 1 && P * SC <= 32, "merge chunk");
    const int lane = threadIdx.x & 63;
    const int grp = threadIdx.x / LPS, gl = threadIdx.x % LPS;
    const int lane0 = lane & ~(LPS - 1);           // first lane of this row's group
    const __amdgpu_buffer_rsrc_t ro = coherent_rsrc(p.part_o);
    const __amdgpu_buffer_rsrc_t rm = coherent_rsrc(p.part_ml);
    float M[P], L[P], acc[P][8];
    int64_t base[P];
#pragma unroll
    for (int k = 0; k < P; ++k) {
        const int r = min(grp + RPP * k, rows - 1);   // in-bounds addresses for spare lanes
        base[k] = (int64_t)part * kRB + (int64_t)r * nseg;
        M[k] = kNoMax;
        L[k] = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[k][e] = 0.f;
    }
    for (int cb = 0; cb < nseg; cb += SC) {
        const int nb = min(SC, nseg - cb);
        uint4 v[P][SC];
        uint2 mine[P];
#pragma unroll
        for (int k = 0; k < P; ++k) {
            if (k * RPP >= rows) continue;            // uniform: no row of this pass
            mine[k] = load_coherent8(rm, (uint32_t)((base[k] + cb + min(gl, nb - 1)) * 8));
#pragma unroll
            for (int i = 0; i < SC; ++i)
                v[k][i] = i < nb ? load_coherent16(ro, (uint32_t)(((base[k] + cb + i) * D + 8 * gl) * 2))
                                 : uint4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int k = 0; k < P; ++k) {
            if (k * RPP >= rows) continue;
            const float mm = __uint_as_float(mine[k].x), ll = __uint_as_float(mine[k].y);
            float mb = gl < nb ? mm : kNoMax;
#pragma unroll
            for (int off = 1; off < LPS; off *= 2) mb = fmaxf(mb, __shfl_xor(mb, off));
            const float Mn = fmaxf(M[k], mb);
            const float a = __builtin_amdgcn_exp2f(M[k] - Mn);
            const float w_mine = gl < nb ? __builtin_amdgcn_exp2f(mm - Mn) * ll : 0.f;
            float ws = w_mine;
#pragma unroll
            for (int off = 1; off < LPS; off *= 2) ws += __shfl_xor(ws, off);
            L[k] = L[k] * a + ws;
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[k][e] *= a;
#pragma unroll
            for (int i = 0; i < SC; ++i) {
                if (i < nb) {                                 // uniform
                    const float w = __shfl(w_mine, lane0 + i);
                    float x[8];
                    unpack16<bf16_t>(v[k][i], x);
#pragma unroll
                    for (int e = 0; e < 8; ++e) acc[k][e] += w * x[e];
                }
            }
            M[k] = Mn;
        }
    }
#pragma unroll
    for (int k = 0; k < P; ++k) {
        const int r = grp + RPP * k;
        if (r >= rows) continue;
        const int rho = rho0 + r;
        const int64_t orow =
            (int64_t)(n0 + rho / p.group) * p.n_q_heads + h * p.group + rho % p.group;
        const float inv = 1.f / L[k];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[k][e] *= inv;
        *reinterpret_cast<uint4*>(reinterpret_cast<bf16_t*>(p.out) + orow * D + 8 * gl) =
            pack16<bf16_t>(acc[k]);
        if (p.lse && gl == 0) p.lse[orow] = (M[k] + log2f(L[k])) * kLn2;
    }
}

}  // namespace
}  // namespace attn
}  // namespace kvlink
