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
#include <type_traits>

#include "attend_common.h"

namespace kvlink {
namespace {

using namespace attn;

// --------------------------------------------------------------- prologue

// One workgroup per new token.  The token's q, k and v vectors are requested
// first (they do not depend on the layout), then the token's cos/sin table is
// built (double-precision angles, in registers, stored to LDS) while they are
// in flight; every q head and k head is rotated with 16-byte accesses (q to
// the workspace, k to the cache row T_c + r) and the v heads are copied to
// the same cache row.
template <typename T, int D>
__global__ __launch_bounds__(256) void rope_new_kernel(
    const T* __restrict__ q_new, const T* __restrict__ k_new, const T* __restrict__ v_new,
    T* __restrict__ q_rot, View k, View v, int layer, int n_seqs, int n_q_heads, int n_kv_heads,
    const int32_t* __restrict__ seq_new_ptr, const int32_t* __restrict__ seq_cached,
    const int32_t* __restrict__ new_pos, RopeFreqs freqs) {
    constexpr int H = D / 2;
    constexpr int E = 16 / (int)sizeof(T);
    constexpr int TPV = H / E;               // threads per head vector
    constexpr int HPP = 256 / TPV;           // head vectors per pass
    constexpr int kPre = 2;                  // passes whose loads are issued up front
    constexpr int VPH = D / E;               // 16-byte vectors per v head
    __shared__ float s_cos[H], s_sin[H];
    const int n = blockIdx.x;
    const int nh = n_q_heads + n_kv_heads;
    const int sub = threadIdx.x % TPV;
    auto src_of = [&](int hv) {
        return hv < n_q_heads ? q_new + ((int64_t)n * n_q_heads + hv) * D
                              : k_new + ((int64_t)n * n_kv_heads + (hv - n_q_heads)) * D;
    };
    uint4 lo[kPre], hi[kPre], vv = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int u = 0; u < kPre; ++u) {
        const int hv = threadIdx.x / TPV + u * HPP;
        if (hv < nh) {
            const T* src = src_of(hv);
            lo[u] = *reinterpret_cast<const uint4*>(src + sub * E);
            hi[u] = *reinterpret_cast<const uint4*>(src + H + sub * E);
        }
    }
    const bool has_v = threadIdx.x < n_kv_heads * VPH;
    if (has_v) {
        const int hk = threadIdx.x / VPH, cch = threadIdx.x % VPH;
        vv = *reinterpret_cast<const uint4*>(v_new + ((int64_t)n * n_kv_heads + hk) * D + cch * E);
    }

    const int s = seq_of(seq_new_ptr, n_seqs, n);
    const int row = seq_cached[s] + (n - seq_new_ptr[s]);
    const int pos = new_pos[n];
    for (int j = threadIdx.x; j < H; j += 256) rope_cos_sin(pos, j, freqs, &s_cos[j], &s_sin[j]);
    __syncthreads();
    float c[E], sn[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        c[e] = s_cos[sub * E + e];
        sn[e] = s_sin[sub * E + e];
    }
    T* kb = reinterpret_cast<T*>(k.base);
    T* vb = reinterpret_cast<T*>(v.base);
    auto rotate_store = [&](int hv, const uint4& l4, const uint4& h4) {
        T* dst = hv < n_q_heads ? q_rot + ((int64_t)n * n_q_heads + hv) * D
                                : kb + view_offset(k, layer, hv - n_q_heads, s, row);
        uint4 x, y;
        rope_rotate16<T>(l4, h4, c, sn, x, y);
        *reinterpret_cast<uint4*>(dst + sub * E) = x;
        *reinterpret_cast<uint4*>(dst + H + sub * E) = y;
    };
#pragma unroll
    for (int u = 0; u < kPre; ++u) {
        const int hv = threadIdx.x / TPV + u * HPP;
        if (hv < nh) rotate_store(hv, lo[u], hi[u]);
    }
    for (int hv = threadIdx.x / TPV + kPre * HPP; hv < nh; hv += HPP) {
        const T* src = src_of(hv);
        rotate_store(hv, *reinterpret_cast<const uint4*>(src + sub * E),
                     *reinterpret_cast<const uint4*>(src + H + sub * E));
    }
    if (has_v) {
        const int hk = threadIdx.x / VPH, cch = threadIdx.x % VPH;
        *reinterpret_cast<uint4*>(vb + view_offset(v, layer, hk, s, row) + cch * E) = vv;
    }
    for (int i = threadIdx.x + 256; i < n_kv_heads * VPH; i += 256) {
        const int hk = i / VPH, cch = i % VPH;
        *reinterpret_cast<uint4*>(vb + view_offset(v, layer, hk, s, row) + cch * E) =
            *reinterpret_cast<const uint4*>(v_new + ((int64_t)n * n_kv_heads + hk) * D + cch * E);
    }
}

// The batch's RoPE table: entry (n, j) = (cos, sin) of new token n's angle
// for pair j, by the same routine as the RoPE stage.
__global__ __launch_bounds__(64) void rope_table_kernel(const int32_t* __restrict__ new_pos,
                                                        int half, RopeFreqs freqs,
                                                        float2* __restrict__ table) {
    const int n = blockIdx.x;
    const int pos = new_pos[n];
    for (int j = threadIdx.x; j < half; j += 64) {
        float c, s;
        rope_cos_sin(pos, j, freqs, &c, &s);
        table[(int64_t)n * half + j] = make_float2(c, s);
    }
}

// ------------------------------------------------------ VALU split kernel
//
// Used for fp32 and as the plain reference schedule: 16 GQA rows per
// workgroup (4 per wavefront), 64-key tiles staged to LDS as float, one key
// per lane for the scores (each K element read once for the wavefront's four
// rows), then P V with one or two head-dim columns per lane.  The next tile's
// K and V are loaded into registers (16-byte loads) while the current one is
// used.

constexpr int kValuRB = 16, kValuKT = 64;

template <int D>
struct alignas(16) ValuSmem {
    float q[kValuRB][D];
    float k[kValuKT][D + 4];   // 16-byte aligned rows; float4 reads by key stay conflict-free
    float v[kValuKT][D];
};

// One segment: tiles [tile_a, tile_b) of KV head h's rows [rho0, rho0 + 16)
// of request s.  Early returns are uniform over the workgroup.
template <typename T, int D>
__device__ __forceinline__ void valu_segment(const KParams& p, ValuSmem<D>& sm, int s, int h,
                                             int rho0, int tile_a, int tile_b, int part, int nseg,
                                             int seg_local) {
    const bool direct = nseg == 1;
    constexpr int RB = kValuRB, KT = kValuKT, RPW = 4, DPL = D / 64;
    constexpr int E = 16 / (int)sizeof(T);          // elements per 16-byte chunk
    constexpr int CPR = D / E;                      // chunks per K or V row
    constexpr int U = KT * CPR / 256;               // chunks per thread per tile
    static_assert(U * 256 == KT * CPR, "tile chunks");
    auto& s_q = sm.q;
    auto& s_k = sm.k;
    auto& s_v = sm.v;

    const int n0 = p.seq_new_ptr[s];
    const int rows_s = (p.seq_new_ptr[s + 1] - n0) * p.group;
    if (rho0 < 0 || rho0 >= rows_s) return;
    const BlockKeys bk = block_keys(p.new_visible, n0, rows_s, rho0, RB, p.group);
    const int kbeg = tile_a * KT;
    if (kbeg >= bk.nvirt) return;
    const int kend = min(tile_b * KT, bk.nvirt);
    const int Tc = p.seq_cached[s];

    const T* kb = reinterpret_cast<const T*>(p.k.base);
    const T* vb = reinterpret_cast<const T*>(p.v.base);
    // this thread's chunks of the tile from t0 (keys past the segment end
    // read its last key; they are masked)
    uint4 kr[U], vr[U];
    auto fetch = [&](int t0) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int c = threadIdx.x + 256 * u, key = c / CPR, col = (c % CPR) * E;
            const int vk = min(t0 + key, kend - 1);
            const int row = vk < bk.cmax ? vk : Tc + (vk - bk.cmax);
            kr[u] = *reinterpret_cast<const uint4*>(kb + view_offset(p.k, p.layer, h, s, row) + col);
            vr[u] = *reinterpret_cast<const uint4*>(vb + view_offset(p.v, p.layer, h, s, row) + col);
        }
    };
    auto stage = [&]() {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int c = threadIdx.x + 256 * u, key = c / CPR, col = (c % CPR) * E;
            float fk[E], fv[E];
            unpack16<T>(kr[u], fk);
            unpack16<T>(vr[u], fv);
#pragma unroll
            for (int e = 0; e < E; ++e) {
                s_k[key][col + e] = fk[e];
                s_v[key][col + e] = fv[e];
            }
        }
    };
    fetch(kbeg);

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

    for (int t0 = kbeg; t0 < kend; t0 += KT) {
        __syncthreads();   // the previous tile's readers are done
        stage();
        __syncthreads();
        if (t0 + KT < kend) fetch(t0 + KT);
        const int vk = t0 + lane;
        // scores of the wavefront's rows for key vk
        float sc[RPW];
#pragma unroll
        for (int i = 0; i < RPW; ++i) sc[i] = 0.f;
#pragma unroll 4
        for (int d = 0; d < D; d += 4) {
            const float4 k4 = *reinterpret_cast<const float4*>(&s_k[lane][d]);
#pragma unroll
            for (int i = 0; i < RPW; ++i) {
                const float4 q4 = *reinterpret_cast<const float4*>(&s_q[wave * RPW + i][d]);
                sc[i] += q4.x * k4.x + q4.y * k4.y + q4.z * k4.z + q4.w * k4.w;
            }
        }
        // online softmax of the four rows, their cross-lane reductions
        // interleaved (independent chains of shuffles)
        float x[RPW], mx[RPW], pr[RPW], ps[RPW];
        bool ok[RPW];
#pragma unroll
        for (int i = 0; i < RPW; ++i) {
            ok[i] = valid[i] && vk < kend &&
                    (vk < bk.cmax ? vk < vis[i] : (vk - bk.cmax) <= tok[i]);
            x[i] = ok[i] ? sc[i] * p.scale_log2 : -INFINITY;
            mx[i] = x[i];
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1)
#pragma unroll
            for (int i = 0; i < RPW; ++i) mx[i] = fmaxf(mx[i], __shfl_xor(mx[i], off));
        float alpha[RPW];
        bool live[RPW];
#pragma unroll
        for (int i = 0; i < RPW; ++i) {
            const float m_new = fmaxf(m[i], mx[i]);
            live[i] = m_new != -INFINITY;   // some key of the row seen so far
            alpha[i] = live[i] ? exp2f(m[i] - m_new) : 1.f;
            pr[i] = ok[i] ? exp2f(x[i] - m_new) : 0.f;
            ps[i] = pr[i];
            if (live[i]) m[i] = m_new;
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1)
#pragma unroll
            for (int i = 0; i < RPW; ++i) ps[i] += __shfl_xor(ps[i], off);
#pragma unroll
        for (int i = 0; i < RPW; ++i) {
            if (!live[i]) continue;
            l[i] = l[i] * alpha[i] + ps[i];
#pragma unroll
            for (int dd = 0; dd < DPL; ++dd) o[i][dd] *= alpha[i];
        }
        // P V: each value read once for the four rows
#pragma unroll 8
        for (int j = 0; j < KT; ++j) {
            float vv[DPL];
#pragma unroll
            for (int dd = 0; dd < DPL; ++dd) vv[dd] = s_v[j][lane + 64 * dd];
#pragma unroll
            for (int i = 0; i < RPW; ++i) {
                const float pj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(pr[i]), j));
#pragma unroll
                for (int dd = 0; dd < DPL; ++dd) o[i][dd] += pj * vv[dd];
            }
        }
    }

#pragma unroll
    for (int i = 0; i < RPW; ++i) {
        if (!valid[i]) continue;
        const int rho = rho0 + wave * RPW + i;
        const int hq = h * p.group + rho % p.group;
        const int64_t orow = (int64_t)(n0 + tok[i]) * p.n_q_heads + hq;
        if (direct) {
            T* out = reinterpret_cast<T*>(p.out);
            const float inv = 1.f / l[i];
#pragma unroll
            for (int dd = 0; dd < DPL; ++dd) out[orow * D + lane + 64 * dd] = from_f32<T>(o[i][dd] * inv);
            if (p.lse && lane == 0) p.lse[orow] = (m[i] + log2f(l[i])) * kLn2;
        } else {
            // O / l in the workload dtype (0 for a row that saw no key here)
            const int64_t pi = (int64_t)part * RB + (int64_t)(rho - rho0) * nseg + seg_local;
            const float inv = l[i] > 0.f ? 1.f / l[i] : 0.f;
            T* po = reinterpret_cast<T*>(p.part_o) + pi * D;
#pragma unroll
            for (int dd = 0; dd < DPL; ++dd) po[lane + 64 * dd] = from_f32<T>(o[i][dd] * inv);
            if (lane == 0) {
                p.part_ml[pi * 2] = m[i];
                p.part_ml[pi * 2 + 1] = l[i];
            }
        }
    }
}

// Persistent workgroups over the schedule, as the matrix-core kernel.
template <typename T, int D>
__global__ __launch_bounds__(256) void attend_valu_kernel(KParams p) {
    __shared__ ValuSmem<D> sm;
    for (int g = blockIdx.x, first = 1; g >= 0 && g < p.n_segments; first = 0) {
        int4 rec[4];
        load_record(p, g, rec);
        if (!record_ok(p, rec, g)) break;
        if (!first) __syncthreads();
        valu_segment<T, D>(p, sm, rec[0].x, rec[0].y, rec[0].z, rec[1].x, rec[1].y, rec[3].x,
                           rec[1].z, rec[1].w);
        g = rec[3].y;
    }
}

// ------------------------------------------------------------- combine

// The rows of units with several segments (rows of single-segment units
// were written by the split kernel).  Workgroup (x, y) takes rows
// [x * RPB, (x+1) * RPB) of the y-th such unit, from its unit record; a row is
// handled by LPS lanes, each holding 16 bytes of every partial vector.  A
// unit's partials (O / l in the workload dtype, float (m, l)) are row-major
// over its segments, so a row's are one contiguous run; up to LPS segments
// are requested in one round, lane j of the row's group holding segment j's
// (m, l).  out = sum_s w_s (O/l)_s / sum_s w_s with w_s = 2^(m_s - M) l_s.
// With kShare (16-row units: a decoding step's few rows over many segments),
// when the block has fewer rows than lane groups and a row more than one run
// of segments, S groups share a row, each taking every S-th run of LPS
// segments, and merge their states through LDS.
// (Four workgroups per compute unit, i.e. at most 128 registers per lane:
// the partial loads in flight are what the kernel's speed depends on; two,
// at most 256, for the shared-row and fp32 forms, which would otherwise
// spill to scratch, whose setup costs a launch far more than the lower
// occupancy.)
template <typename T, int D, bool kShare>
__global__ __launch_bounds__(256, (kShare || sizeof(T) == 4) ? 2 : 4) void combine_kernel(KParams p) {
    constexpr int EPL = 16 / (int)sizeof(T);   // elements per 16-byte load
    constexpr int LPS = D / EPL;               // lanes per row
    constexpr int RPW = 64 / LPS;              // lane groups (rows) per wavefront
    constexpr int RPB = 4 * RPW;               // lane groups (rows) per workgroup
    constexpr int CAP = LPS;                   // segments per round of loads
    constexpr int SH = kShare ? RPB : 1;
    __shared__ float s_ml[SH][2];
    __shared__ float s_acc[SH][LPS][EPL];
    const int wave = threadIdx.x / 64, lane = threadIdx.x % 64;
    const int grp = lane / LPS, gl = lane % LPS;
    const int q = wave * RPW + grp;            // lane group of the workgroup
    for (int su = blockIdx.y; su < p.n_split; su += gridDim.y) {
        const int u = p.split_units[su];
        if (u < 0 || u >= p.n_units) continue;
        const int4 u0 = p.unit[2 * (int64_t)u], u1 = p.unit[2 * (int64_t)u + 1];
        const int s = u0.x, h = u0.y, rho0 = u0.z, rows = u0.w;
        const int n0 = u1.x, seg0 = u1.y, nseg = u1.z;
        if (s < 0 || s >= p.n_seqs || h < 0 || h >= p.n_kv_heads || rows < 1 ||
            rows > p.row_block || seg0 < 0 || nseg < 2 || seg0 + nseg > p.n_segments)
            continue;
        if (blockIdx.x * RPB >= rows) continue;
        const int here = min(RPB, rows - (int)blockIdx.x * RPB);
        int S = 1;                                  // lane groups per row
        if constexpr (kShare)
            while (2 * S * here <= RPB && S * CAP < nseg) S *= 2;
        const int r = blockIdx.x * RPB + q / S, phase = q % S;
        const bool valid = q / S < here;
        const int rr = valid ? r : rows - 1;   // in-bounds addresses for spare lanes
        const int64_t base = (int64_t)seg0 * p.row_block + (int64_t)rr * nseg;
        const float2* ml = reinterpret_cast<const float2*>(p.part_ml) + base;
        const uint4* po =
            reinterpret_cast<const uint4*>(reinterpret_cast<const T*>(p.part_o) + base * D);

        // the running maximum starts finite, so a segment that saw no key of
        // this row (maximum -inf or the finite floor, sum 0) weighs 0
        float M = kNoMax, L = 0.f, acc[EPL];
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[e] = 0.f;
        const int n_mine = valid ? nseg : 0;
        auto rounds = [&](auto cap_c) {
            constexpr int C = decltype(cap_c)::value;
            for (int cb = phase * C; cb < n_mine; cb += S * C) {
                const int nb = min(C, nseg - cb);
                const float2 mine = ml[cb + min(gl, nb - 1)];
                uint4 v[C];
#pragma unroll
                for (int i = 0; i < C; ++i) v[i] = po[(int64_t)(cb + min(i, nb - 1)) * LPS + gl];
                float mb = gl < nb ? mine.x : kNoMax;
#pragma unroll
                for (int off = 1; off < LPS; off *= 2) mb = fmaxf(mb, __shfl_xor(mb, off));
                const float Mn = fmaxf(M, mb);
                const float a = __builtin_amdgcn_exp2f(M - Mn);
                const float w_mine = gl < nb ? __builtin_amdgcn_exp2f(mine.x - Mn) * mine.y : 0.f;
                float ws = w_mine;
#pragma unroll
                for (int off = 1; off < LPS; off *= 2) ws += __shfl_xor(ws, off);
                L = L * a + ws;
#pragma unroll
                for (int e = 0; e < EPL; ++e) acc[e] *= a;
#pragma unroll
                for (int i = 0; i < C; ++i) {
                    const float w = __shfl(w_mine, grp * LPS + i);   // 0 past the last segment
                    float x[EPL];
                    unpack16<T>(v[i], x);
#pragma unroll
                    for (int e = 0; e < EPL; ++e) acc[e] += w * x[e];
                }
                M = Mn;
            }
        };
        // units of at most four or eight segments (the split units of a
        // prefill) take rounds of that many: a lane then issues four or eight
        // partial loads per round, not sixteen
        if (!kShare && nseg <= 4) rounds(std::integral_constant<int, 4>{});
        else if (!kShare && nseg <= 8) rounds(std::integral_constant<int, 8>{});
        else rounds(std::integral_constant<int, CAP>{});
        if constexpr (kShare) {
            if (S > 1) {   // uniform over the workgroup
                if (gl == 0) {
                    s_ml[q][0] = M;
                    s_ml[q][1] = L;
                }
#pragma unroll
                for (int e = 0; e < EPL; ++e) s_acc[q][gl][e] = acc[e];
                __syncthreads();
                if (valid && phase == 0) {
                    for (int k = 1; k < S; ++k) {
                        const float Mk = s_ml[q + k][0];
                        const float Mn = fmaxf(M, Mk);
                        const float a = __builtin_amdgcn_exp2f(M - Mn);
                        const float b = __builtin_amdgcn_exp2f(Mk - Mn);
                        L = L * a + s_ml[q + k][1] * b;
#pragma unroll
                        for (int e = 0; e < EPL; ++e) acc[e] = acc[e] * a + s_acc[q + k][gl][e] * b;
                        M = Mn;
                    }
                }
                __syncthreads();
            }
        }
        if (valid && phase == 0) {
            const int rho = rho0 + r;
            const int64_t orow =
                (int64_t)(n0 + rho / p.group) * p.n_q_heads + h * p.group + rho % p.group;
            const float inv = 1.f / L;
#pragma unroll
            for (int e = 0; e < EPL; ++e) acc[e] *= inv;
            *reinterpret_cast<uint4*>(reinterpret_cast<T*>(p.out) + orow * D + EPL * gl) =
                pack16<T>(acc);
            if (p.lse && gl == 0) p.lse[orow] = (M + log2f(L)) * kLn2;
        }
    }
}

template <typename T, int D>
constexpr int combine_rows_per_block() {
    return 4 * (64 / (D / (16 / (int)sizeof(T))));
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

template <typename T, int D>
hipError_t launch_typed(const AttendPlan& pl, const AttendArgs& a, hipStream_t stream,
                        unsigned stages) {
    char* ws = reinterpret_cast<char*>(a.workspace);
    T* q_rot = reinterpret_cast<T*>(ws + kCounterBytes);
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
    p.row_block = pl.row_block;
    p.n_units = pl.n_units;
    p.n_segments = pl.n_segments;
    p.seg = reinterpret_cast<const int4*>(pl.table);
    p.unit = reinterpret_cast<const int4*>(pl.table + (size_t)kSegRecord * pl.n_segments);
    p.split_units = pl.table + (size_t)kSegRecord * pl.n_segments + (size_t)kUnitRecord * pl.n_units;
    p.n_split = pl.n_split;
    p.counters = reinterpret_cast<uint32_t*>(ws);
    p.part_o = ws + kCounterBytes + pl.q_rot_bytes;
    p.part_ml = reinterpret_cast<float*>(ws + kCounterBytes + pl.q_rot_bytes + pl.part_o_bytes);
    p.out = a.out;
    p.lse = a.lse;
    // the matrix-core kernels take the RoPE over when the batch's table is given
    const bool fused = a.rope_table && pl.path != kPathValu;
    p.rope = fused ? reinterpret_cast<const float2*>(a.rope_table) : nullptr;
    p.merge_in_launch = pl.merge_in_launch ? 1 : 0;
    p.q_new = a.q_new;
    p.k_new = a.k_new;
    p.v_new = a.v_new;
    p.fuse_spans = pl.path == kPathWide ? a.fuse_spans : nullptr;
    p.fuse_span_ptr = a.fuse_span_ptr;
    p.freqs = a.freqs;

    hipError_t e = hipSuccess;
    if ((stages & KVLINK_STAGE_ROPE) && !fused) {
        hipLaunchKernelGGL((rope_new_kernel<T, D>), dim3(pl.n_new_total), dim3(256), 0, stream,
                           reinterpret_cast<const T*>(a.q_new), reinterpret_cast<const T*>(a.k_new),
                           reinterpret_cast<const T*>(a.v_new), q_rot, a.k, a.v, a.layer,
                           pl.n_seqs, pl.n_q_heads, pl.n_kv_heads, a.seq_new_ptr, a.seq_cached,
                           a.new_pos, a.freqs);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }

    if ((stages & KVLINK_STAGE_SPLIT) && pl.n_wg > 0) {
        if (pl.path == kPathWide) {
            e = launch_attend_mfma(D, p, pl.n_wg, stream);
        } else if (pl.path == kPathDecode) {
            e = launch_attend_decode(D, p, pl.n_wg, stream);
        } else {
            hipLaunchKernelGGL((attend_valu_kernel<T, D>), dim3(pl.n_wg), dim3(256), 0, stream, p);
            e = hipGetLastError();
        }
        if (e != hipSuccess) return e;
    }
    // the split kernel may merge its split units itself
    if (!(stages & KVLINK_STAGE_COMBINE) || !pl.partials || pl.merge_in_launch) return hipSuccess;

    constexpr int rpb = combine_rows_per_block<T, D>();
    const dim3 grid((pl.row_block + rpb - 1) / rpb, std::min(pl.n_split, 65535));
    if (pl.path != kPathWide)
        hipLaunchKernelGGL((combine_kernel<T, D, true>), grid, dim3(256), 0, stream, p);
    else
        hipLaunchKernelGGL((combine_kernel<T, D, false>), grid, dim3(256), 0, stream, p);
    return hipGetLastError();
}

}  // namespace

bool attend_row_block_ok(AttendPath path, int row_block) {
    if (path == kPathWide) return attn::attend_mfma_row_block_ok(row_block);
    return row_block == (path == kPathDecode ? attn::attend_decode_row_block() : kValuRB);
}

bool make_attend_plan(kvlink_dtype dt, int n_q_heads, int n_kv_heads, int head_dim,
                      int n_new_total, const kvlink_attend_plan& sched, AttendPlan* p) {
    if (n_q_heads < 1 || n_kv_heads < 1 || n_q_heads % n_kv_heads) return false;
    if (head_dim != 64 && head_dim != 128) return false;
    if (n_new_total < 0 || sched.n_seqs < 1) return false;
    // the kernel is fixed by the dtype and the schedule's row block
    int path = -1;
    if (dt == KVLINK_BF16 && attend_row_block_ok(kPathWide, sched.row_block)) path = kPathWide;
    if (dt == KVLINK_BF16 && attend_row_block_ok(kPathDecode, sched.row_block)) path = kPathDecode;
    if (dt == KVLINK_F32 && attend_row_block_ok(kPathValu, sched.row_block)) path = kPathValu;
    if (path < 0) return false;
    if (sched.n_units > kMaxUnits) return false;
    if (sched.n_workgroups < 0 || sched.n_units < 0 || sched.n_segments < sched.n_units)
        return false;
    if ((int64_t)sched.n_segments * kSegRecord > INT32_MAX) return false;
    if (sched.n_workgroups > 0 && (sched.n_units < 1 || sched.n_segments < 1)) return false;
    const int64_t want = (int64_t)kSegRecord * sched.n_segments +
                         (int64_t)kUnitRecord * sched.n_units + sched.n_split_units;
    if (sched.n_segments < sched.n_workgroups) return false;
    if (sched.n_split_units < 0 || sched.n_split_units > sched.n_units) return false;
    if ((sched.n_split_units > 0) != (sched.n_segments > sched.n_units)) return false;
    if (sched.table_len != want) return false;
    const size_t elem = dt == KVLINK_BF16 ? 2 : 4;
    p->n_q_heads = n_q_heads;
    p->n_kv_heads = n_kv_heads;
    p->group = n_q_heads / n_kv_heads;
    p->head_dim = head_dim;
    p->n_seqs = sched.n_seqs;
    p->n_new_total = n_new_total;
    p->row_block = sched.row_block;
    p->path = path;
    p->n_wg = sched.n_workgroups;
    p->n_units = sched.n_units;
    p->n_segments = sched.n_segments;
    p->table = sched.table;
    p->partials = sched.n_split_units > 0;
    p->merge_in_launch = path != kPathValu && (sched.flags & KVLINK_PLAN_IN_LAUNCH) != 0;
    if ((sched.flags & KVLINK_PLAN_IN_LAUNCH) && (sched.flags & KVLINK_PLAN_COMBINE)) return false;
    p->n_split = sched.n_split_units;
    const int64_t rows = (int64_t)n_new_total * n_q_heads;
    p->q_rot_bytes = align256((size_t)rows * head_dim * elem);
    if (p->partials) {
        const size_t prow = (size_t)sched.n_segments * sched.row_block;
        p->part_o_bytes = align256(prow * head_dim * elem);
        p->part_ml_bytes = align256(prow * 2 * sizeof(float));
        // the in-launch merge addresses the partials with 32-bit offsets
        if (p->part_o_bytes >= ((size_t)1 << 31)) return false;
    } else {
        p->part_o_bytes = p->part_ml_bytes = 0;
    }
    p->total_bytes = kCounterBytes + p->q_rot_bytes + p->part_o_bytes + p->part_ml_bytes;
    return true;
}

hipError_t launch_rope_table(int head_dim, const RopeFreqs& freqs, int n_new_total,
                             const int32_t* new_pos, float* table, hipStream_t stream) {
    if (n_new_total == 0) return hipSuccess;
    hipLaunchKernelGGL(rope_table_kernel, dim3(n_new_total), dim3(64), 0, stream, new_pos,
                       head_dim / 2, freqs, reinterpret_cast<float2*>(table));
    return hipGetLastError();
}

hipError_t launch_attend(kvlink_dtype dt, const AttendPlan& p, const AttendArgs& a,
                         hipStream_t stream, unsigned stages) {
    if (dt == KVLINK_BF16)
        return p.head_dim == 128 ? launch_typed<bf16_t, 128>(p, a, stream, stages)
                                 : launch_typed<bf16_t, 64>(p, a, stream, stages);
    return p.head_dim == 128 ? launch_typed<float, 128>(p, a, stream, stages)
                             : launch_typed<float, 64>(p, a, stream, stages);
}

}  // namespace kvlink
