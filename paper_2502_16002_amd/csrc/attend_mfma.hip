// attend_mfma.hip — bf16 split-K attention of the new tokens on gfx950 matrix
// cores (v_mfma_f32_16x16x32_bf16, float accumulation).
//
// A workgroup owns one KV head, 64 GQA-packed rows (16 tokens x 4 heads for
// a group of 4) and one split of the block's virtual key range.  Its eight
// wavefronts form two row groups of 32 rows times four key waves; each is an
// independent online-softmax worker over 32-key chunks (key wave w takes
// chunks w, w+4, ...) for its 32 rows.  The two waves that take the same
// chunk read it at about the same time, so the second read is served by the
// L1 cache.  Per-wave state fits two wavefronts per SIMD, so one wave's
// softmax overlaps the other's matrix products:
//
//   S^T = K Q^T     A = 16 keys x 32 dims of K, straight from global memory
//                   into registers (row-major K is already the A layout);
//                   B = Q^T, loaded once (rows x dims, again row-major).
//                   The accumulator holds, per lane, 4 keys of one row.
//   P   = exp2(S*scale*log2e - m)   in float, per lane, then packed to bf16:
//                   the 8 keys a lane holds for its row are exactly the 8
//                   k-elements the B operand of the next product needs, so
//                   P goes from accumulator to operand without a shuffle.
//   O^T += V^T P^T  A = V^T (16 dims x 32 keys): V is row-major in memory, so
//                   each wave transposes its 32 x d V chunk through a
//                   wave-private LDS tile (rows of 32 keys, 80-byte stride:
//                   the 8-byte operand reads are bank-conflict free).
//
// The key order inside the 32-key contraction is permuted the same way in
// both operands (lane group g holds keys 4g..4g+3 and 16+4g..16+4g+3), which
// leaves the sum unchanged.  The row max is reduced across the four lane
// groups that hold a row; the row sum stays per lane until the end.  After
// the loop the key waves of a row group merge their (m, l, O) in LDS and key
// wave 0 writes the group's result (final output, or a split partial for the
// combine).
#include <algorithm>

#include "attend_common.h"

namespace kvlink {
namespace attn {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

namespace {

constexpr int kRB = 64;         // GQA rows per workgroup
constexpr int kRG = 2;          // row groups (of kRB / kRG rows) per workgroup
constexpr int kKW = 4;          // key waves per row group
constexpr int kWaves = kRG * kKW;
constexpr int kRT = kRB / kRG / 16;   // 16-row tiles per wave
constexpr int kChunk = 32;      // keys per wave step
constexpr int kVtStride = 80;   // bytes per dim row of the transposed V tile

template <int D>
struct Smem {
    static constexpr int vt_wave = D * kVtStride;
    static constexpr int vt_all = kWaves * vt_wave;
    static constexpr int slot = (D / 16) * kRT * 4 * 64 * 4;   // one wave's O^T registers
    static constexpr int merge = kRG * 2 * slot;
    static constexpr int ml_off = vt_all > merge ? vt_all : merge;
    static constexpr int bytes = ml_off + 2 * kWaves * (kRB / kRG) * 4;
};

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4& v) {
    return __builtin_bit_cast(bf16x8, v);
}

__device__ __forceinline__ uint32_t pack_bf16(float a, float b) {
    return (uint32_t)from_f32<bf16_t>(a).bits | ((uint32_t)from_f32<bf16_t>(b).bits << 16);
}

__device__ __forceinline__ void wave_lds_fence() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Rescale threshold of the online softmax, in log2 units: the running row
// maximum m is only raised (and O, l rescaled) when a score exceeds it by
// more than kTau, so probabilities p = 2^(s - m) stay below 2^kTau (exact in
// float, representable in bf16) and the rescale is rare after the first
// chunks.
constexpr float kTau = 8.0f;
// Finite stand-in for "no score seen yet": any real score exceeds it by more
// than kTau, and masked scores (-inf) still give p = 0 without NaN.
constexpr float kNoMax = -1.0e30f;

template <int D>
__global__ __launch_bounds__(64 * kWaves, 1) void attend_mfma_kernel(KParams p) {
    constexpr int DT = D / 16;   // 16-dim tiles of O^T
    constexpr int DS = D / 32;   // 32-dim steps of S^T = K Q^T
    constexpr int VCH = D / 64;  // 16-byte V chunks a lane loads per key
    __shared__ __attribute__((aligned(16))) unsigned char smem[Smem<D>::bytes];

    const int split = blockIdx.x;
    const int s = blockIdx.z / p.n_kv_heads, h = blockIdx.z % p.n_kv_heads;
    const int G = p.group;
    const int n0 = p.seq_new_ptr[s];
    const int rows_s = (p.seq_new_ptr[s + 1] - n0) * G;
    const int rho0 = blockIdx.y * kRB;
    if (rho0 >= rows_s) return;
    const BlockKeys bk = block_keys(p.new_visible, n0, rows_s, rho0, kRB, G);
    const int kbeg = split * p.split_keys;
    if (kbeg >= bk.nvirt) return;
    const int kend = min(kbeg + p.split_keys, bk.nvirt);
    const int Tc = p.seq_cached[s];
    const int vis_min = p.new_visible[n0 + rho0 / G];
    const float c2 = p.scale_log2;   // > 0

    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int rg = wave / kKW, kw = wave % kKW;     // row group, key wave
    const int lr = lane & 15, lg = lane >> 4;
    const int rho_w = rho0 + rg * (kRB / kRG);      // first row of this wave

    // The rows of this lane (one per row tile).  Row r may see virtual
    // key v iff v < lo[rt] (cached rows up to its document, within the split)
    // or cmax <= v <= hi[rt] (new rows up to its own, within the split).
    int tok[kRT], lo[kRT], hi[kRT];
#pragma unroll
    for (int rt = 0; rt < kRT; ++rt) {
        const int rho = rho_w + 16 * rt + lr;
        tok[rt] = rho < rows_s ? rho / G : -1;
        const int vis = tok[rt] >= 0 ? p.new_visible[n0 + tok[rt]] : 0;
        lo[rt] = min(vis, kend);
        hi[rt] = tok[rt] >= 0 ? min(bk.cmax + tok[rt], kend - 1) : -1;
    }

    // Q^T operand, loaded once
    const bf16_t* q_rot = reinterpret_cast<const bf16_t*>(p.q_rot);
    bf16x8 qB[kRT][DS];
#pragma unroll
    for (int rt = 0; rt < kRT; ++rt) {
        const int rho = rho_w + 16 * rt + lr;
        const int tq = max(tok[rt], 0);
        const int64_t qrow = ((int64_t)(n0 + tq) * p.n_q_heads + h * G + rho % G) * D;
#pragma unroll
        for (int ds = 0; ds < DS; ++ds) {
            uint4 v = *reinterpret_cast<const uint4*>(q_rot + qrow + 32 * ds + 8 * lg);
            if (tok[rt] < 0) v = uint4{0u, 0u, 0u, 0u};
            qB[rt][ds] = as_bf16x8(v);
        }
    }

    floatx4 o[DT][kRT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
        for (int rt = 0; rt < kRT; ++rt) o[dt][rt] = floatx4{0.f, 0.f, 0.f, 0.f};
    float m[kRT], lsum[kRT];
#pragma unroll
    for (int rt = 0; rt < kRT; ++rt) {
        m[rt] = kNoMax;
        lsum[rt] = 0.f;
    }

    const RowPtr kp = row_ptr<bf16_t>(p.k, p.layer, h, s);
    const RowPtr vp = row_ptr<bf16_t>(p.v, p.layer, h, s);
    unsigned char* vt = smem + wave * Smem<D>::vt_wave;
    const int kg = lane & 7, cc = lane >> 3;      // V loader: keys 4kg..4kg+3, dims 8cc..
    const int n_chunks = (kend - kbeg + kChunk - 1) / kChunk;

    // virtual key -> cache row (clamped into the split so that every load is
    // of a real row; out-of-range keys are masked)
    auto key_row = [&](int v) {
        v = min(v, kend - 1);
        return v < bk.cmax ? v : Tc + (v - bk.cmax);
    };
    auto load_k = [&](int c, uint4 (&ka)[2][DS]) {
        const int v0 = kbeg + c * kChunk;
#pragma unroll
        for (int kt = 0; kt < 2; ++kt) {
            const char* kr = kp.row(key_row(v0 + 16 * kt + lr)) + 16 * lg;
#pragma unroll
            for (int ds = 0; ds < DS; ++ds) ka[kt][ds] = *reinterpret_cast<const uint4*>(kr + 64 * ds);
        }
    };
    auto load_v = [&](int c, uint4 (&va)[4][VCH]) {
        const int v0 = kbeg + c * kChunk;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const char* vr = vp.row(key_row(v0 + 4 * kg + i)) + 16 * cc;
#pragma unroll
            for (int j = 0; j < VCH; ++j) va[i][j] = *reinterpret_cast<const uint4*>(vr + 128 * j);
        }
    };

    // K of the next chunk is prefetched into registers one iteration ahead;
    // V of the current chunk is requested at the top of the iteration and
    // lands while the K Q^T products run
    uint4 ka[2][DS];
    if (kw < n_chunks) load_k(kw, ka);

    for (int c = kw; c < n_chunks; c += kKW) {
        const int v0 = kbeg + c * kChunk;
        uint4 va[4][VCH];
        load_v(c, va);
        uint4 kn[2][DS];
        const bool has_next = c + kKW < n_chunks;
        if (has_next) load_k(c + kKW, kn);

        // S^T = K Q^T
        floatx4 sacc[2][kRT];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int rt = 0; rt < kRT; ++rt) {
                floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ds = 0; ds < DS; ++ds)
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(ka[kt][ds]), qB[rt][ds],
                                                                  acc, 0, 0, 0);
                sacc[kt][rt] = acc;
            }

        // transpose V through the wave's LDS tile: row d holds the 32 keys of
        // dim d; a lane writes keys 4kg..4kg+3 of 8 dims.  The fence orders
        // these writes after the previous chunk's reads of the tile.
        wave_lds_fence();
#pragma unroll
        for (int j = 0; j < VCH; ++j) {
            const uint32_t w0[4] = {va[0][j].x, va[0][j].y, va[0][j].z, va[0][j].w};
            const uint32_t w1[4] = {va[1][j].x, va[1][j].y, va[1][j].z, va[1][j].w};
            const uint32_t w2[4] = {va[2][j].x, va[2][j].y, va[2][j].z, va[2][j].w};
            const uint32_t w3[4] = {va[3][j].x, va[3][j].y, va[3][j].z, va[3][j].w};
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int wi = e >> 1;
                uint32_t a, b;
                if (e & 1) {
                    a = __builtin_amdgcn_perm(w1[wi], w0[wi], 0x07060302u);
                    b = __builtin_amdgcn_perm(w3[wi], w2[wi], 0x07060302u);
                } else {
                    a = __builtin_amdgcn_perm(w1[wi], w0[wi], 0x05040100u);
                    b = __builtin_amdgcn_perm(w3[wi], w2[wi], 0x05040100u);
                }
                const int d = 8 * cc + 64 * j + e;
                *reinterpret_cast<uint2*>(vt + d * kVtStride + 8 * kg) = uint2{a, b};
            }
        }

        // mask (only chunks that reach past what every row of the block sees)
        if (v0 + kChunk > vis_min) {
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int v = v0 + 16 * kt + 4 * lg + i;
#pragma unroll
                    for (int rt = 0; rt < kRT; ++rt) {
                        const bool ok = v < lo[rt] || (v >= bk.cmax && v <= hi[rt]);
                        sacc[kt][rt][i] = ok ? sacc[kt][rt][i] : -INFINITY;
                    }
                }
        }

        // online softmax in base 2 with a lazily raised maximum
        float mx[kRT];
        bool over = false;
#pragma unroll
        for (int rt = 0; rt < kRT; ++rt) {
            mx[rt] = fmaxf(fmaxf(fmaxf(sacc[0][rt][0], sacc[0][rt][1]), fmaxf(sacc[0][rt][2], sacc[0][rt][3])),
                           fmaxf(fmaxf(sacc[1][rt][0], sacc[1][rt][1]), fmaxf(sacc[1][rt][2], sacc[1][rt][3])));
            over |= mx[rt] * c2 > m[rt] + kTau;
        }
        if (__builtin_amdgcn_ballot_w64(over)) {
#pragma unroll
            for (int rt = 0; rt < kRT; ++rt) {
                float r = mx[rt];
                r = fmaxf(r, __shfl_xor(r, 16));
                r = fmaxf(r, __shfl_xor(r, 32));
                const float m_new = fmaxf(m[rt], r * c2);
                const float alpha = __builtin_amdgcn_exp2f(m[rt] - m_new);
                m[rt] = m_new;
                lsum[rt] *= alpha;
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) o[dt][rt] *= alpha;
            }
        }
        uint32_t pk[kRT][4];
#pragma unroll
        for (int rt = 0; rt < kRT; ++rt) {
            float pr[2][4];
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    pr[kt][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kt][rt][i], c2, -m[rt]));
            lsum[rt] += ((pr[0][0] + pr[0][1]) + (pr[0][2] + pr[0][3])) +
                        ((pr[1][0] + pr[1][1]) + (pr[1][2] + pr[1][3]));
            pk[rt][0] = pack_bf16(pr[0][0], pr[0][1]);
            pk[rt][1] = pack_bf16(pr[0][2], pr[0][3]);
            pk[rt][2] = pack_bf16(pr[1][0], pr[1][1]);
            pk[rt][3] = pack_bf16(pr[1][2], pr[1][3]);
        }

        // O^T += V^T P^T
        wave_lds_fence();
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
            const unsigned char* row = vt + (16 * dt + lr) * kVtStride + 8 * lg;
            const uint2 lo8 = *reinterpret_cast<const uint2*>(row);
            const uint2 hi8 = *reinterpret_cast<const uint2*>(row + 32);
            const bf16x8 a = as_bf16x8(uint4{lo8.x, lo8.y, hi8.x, hi8.y});
#pragma unroll
            for (int rt = 0; rt < kRT; ++rt)
                o[dt][rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                    a, as_bf16x8(uint4{pk[rt][0], pk[rt][1], pk[rt][2], pk[rt][3]}), o[dt][rt],
                    0, 0, 0);
        }

        if (has_next) {
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int ds = 0; ds < DS; ++ds) ka[kt][ds] = kn[kt][ds];
        }
    }

    // row sums: add the four lane groups that hold each row
#pragma unroll
    for (int rt = 0; rt < kRT; ++rt) {
        lsum[rt] += __shfl_xor(lsum[rt], 16);
        lsum[rt] += __shfl_xor(lsum[rt], 32);
    }

    // merge the key waves of each row group
    constexpr int RW = kRB / kRG;                   // rows per row group
    float* s_m = reinterpret_cast<float*>(smem + Smem<D>::ml_off);
    float* s_l = s_m + kWaves * RW;
    __syncthreads();                                // every wave is done with its V^T tile
    if (lg == 0) {
#pragma unroll
        for (int rt = 0; rt < kRT; ++rt) {
            s_m[wave * RW + 16 * rt + lr] = m[rt];
            s_l[wave * RW + 16 * rt + lr] = lsum[rt];
        }
    }
    __syncthreads();
    float Mrow[kRT], Lrow[kRT];
#pragma unroll
    for (int rt = 0; rt < kRT; ++rt) {
        const int row = 16 * rt + lr;
        float M = kNoMax;
#pragma unroll
        for (int w = 0; w < kKW; ++w) M = fmaxf(M, s_m[(rg * kKW + w) * RW + row]);
        float L = 0.f;
#pragma unroll
        for (int w = 0; w < kKW; ++w)
            L += s_l[(rg * kKW + w) * RW + row] *
                 __builtin_amdgcn_exp2f(s_m[(rg * kKW + w) * RW + row] - M);
        const float f = __builtin_amdgcn_exp2f(m[rt] - M);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) o[dt][rt] *= f;
        Mrow[rt] = M;
        Lrow[rt] = L;
    }
    constexpr int SLOT = Smem<D>::slot / 4;         // floats
    float* slot = reinterpret_cast<float*>(smem) + rg * 2 * SLOT;
    auto store_slot = [&](float* sl) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int rt = 0; rt < kRT; ++rt)
                *reinterpret_cast<floatx4*>(sl + ((dt * kRT + rt) * 64 + lane) * 4) = o[dt][rt];
    };
    auto add_slot = [&](const float* sl) {
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
#pragma unroll
            for (int rt = 0; rt < kRT; ++rt)
                o[dt][rt] += *reinterpret_cast<const floatx4*>(sl + ((dt * kRT + rt) * 64 + lane) * 4);
    };
    if (kw >= 2) store_slot(slot + (kw - 2) * SLOT);
    __syncthreads();
    if (kw < 2) add_slot(slot + kw * SLOT);
    __syncthreads();
    if (kw == 1) store_slot(slot);
    __syncthreads();
    if (kw != 0) return;
    add_slot(slot);

    // key wave 0 of each row group writes the group's rows
#pragma unroll
    for (int rt = 0; rt < kRT; ++rt) {
        if (tok[rt] < 0) continue;
        const int rho = rho_w + 16 * rt + lr;
        const int64_t orow = (int64_t)(n0 + tok[rt]) * p.n_q_heads + h * G + rho % G;
        if (p.n_splits == 1) {
            bf16_t* out = reinterpret_cast<bf16_t*>(p.out) + orow * D;
            const float inv = 1.f / Lrow[rt];
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                const floatx4 v = o[dt][rt];
                *reinterpret_cast<uint2*>(out + 16 * dt + 4 * lg) =
                    uint2{pack_bf16(v[0] * inv, v[1] * inv), pack_bf16(v[2] * inv, v[3] * inv)};
            }
            if (p.lse && lg == 0) p.lse[orow] = (Mrow[rt] + log2f(Lrow[rt])) * kLn2;
        } else {
            const int64_t pi = orow * p.n_splits + split;
            float* po = p.part_o + pi * D;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
                *reinterpret_cast<floatx4*>(po + 16 * dt + 4 * lg) = o[dt][rt];
            if (lg == 0) {
                p.part_ml[pi * 2] = Mrow[rt];
                p.part_ml[pi * 2 + 1] = Lrow[rt];
            }
        }
    }
}

}  // namespace

hipError_t launch_attend_mfma(int head_dim, const KParams& p, dim3 grid, hipStream_t stream) {
    if (head_dim == 128)
        hipLaunchKernelGGL(attend_mfma_kernel<128>, grid, dim3(64 * kWaves), 0, stream, p);
    else
        hipLaunchKernelGGL(attend_mfma_kernel<64>, grid, dim3(64 * kWaves), 0, stream, p);
    return hipGetLastError();
}

}  // namespace attn
}  // namespace kvlink
