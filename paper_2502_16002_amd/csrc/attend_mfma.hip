// attend_mfma.hip — bf16 split-K attention of the new tokens on gfx950 matrix
// cores (v_mfma_f32_16x16x32_bf16, float accumulation).
//
// A workgroup owns one KV head, kRB = 256 GQA-packed rows (64 tokens x 4
// heads for a group of 4) and one split of the block's virtual key range.
// Each of its eight wavefronts owns 32 of the rows and walks every key of
// the split (two wavefronts per SIMD, so one's softmax overlaps the other's
// matrix products); K and V tiles of 64 keys are brought into LDS once per
// workgroup and shared by the eight waves:
//
//   * the tiles are loaded straight from global memory into a four-stage
//     LDS ring with 16-byte direct-to-LDS loads (each wave issues an eighth
//     of a tile), so the loads of the next three tiles are in flight while the
//     current one is used, at no register cost;
//   * K is stored in MFMA operand order (for each 16-key x 32-dim block,
//     lane l's 16 bytes at l*16): the A operand of S^T = K Q^T is one
//     conflict-free ds_read_b128 per lane;
//   * V is stored row-major with the 16-byte chunks of row k XOR-swizzled by
//     k, and read with ds_read_b64_tr_b16, which hands each lane four keys of
//     one dim: exactly the A operand of O^T = V^T P^T, with no transpose on
//     the vector ALUs.
//
// Per wave and 32-key sub-tile:
//   S^T = K Q^T     B = Q^T (32 rows, loaded once into registers); the
//                   accumulator holds, per lane, 4 keys of one row;
//   P   = 2^(S*scale*log2e - m)  per lane in float, packed to bf16: the 8
//                   keys a lane holds for its row are the 8 k-elements the B
//                   operand of the next product needs (lane group g holds
//                   keys 4g..4g+3 and 16+4g..16+4g+3; the A operand uses the
//                   same key order, which leaves the contraction unchanged);
//   O^T += V^T P^T
//
// The running row maximum is raised lazily (only when a score exceeds it by
// more than 2^kTau), so the rescale of O and l and the cross-lane reduction
// are off the common path.
#include <algorithm>
#include <type_traits>

#include "attend_common.h"

namespace kvlink {
namespace attn {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short shortx4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) shortx4 lds_shortx4;

namespace {

constexpr int kWaves = 8;
constexpr int kRT = 2;                    // 16-row tiles per wave
constexpr int kRB = kWaves * kRT * 16;    // GQA rows per workgroup
constexpr int kTile = 64;                 // keys per LDS stage
constexpr int kStages = 4;
// Rescale threshold of the online softmax, in log2 units: p = 2^(s - m)
// stays below 2^kTau (exact in float, representable in bf16).
constexpr float kTau = 8.0f;
// Finite stand-in for "no score seen yet": any real score exceeds it by more
// than kTau, and masked scores (-inf) still give p = 0 without NaN.
constexpr float kNoMax = -1.0e30f;

template <int D>
struct Smem {
    static constexpr int k_bytes = kTile * D * 2;
    static constexpr int v_bytes = kTile * D * 2;
    static constexpr int stage = k_bytes + v_bytes;
    // direct-to-LDS loads need a non-zero LDS address: keep the first bytes
    // of the allocation out of the ring
    static constexpr int base = 1024;
    static constexpr int bytes = base + kStages * stage;
};

__device__ __forceinline__ bf16x8 as_bf16x8(const uint4& v) {
    return __builtin_bit_cast(bf16x8, v);
}


// Transposed reads of the V^T operands of one 32-key sub-tile: r[dt][h] for
// dt < DT (16-dim tiles) and h in {0, 1} (keys 4g.. and 16+4g..).  a[dt] is
// the LDS byte address of tile dt's first read; the second half of the keys
// sits OFF bytes further (an immediate offset).  Issued as one block followed
// by a single wait on the LDS counter; the results are early-clobber outputs,
// since a read's data may return while later reads of the block still need
// their address registers.  The V tile was written by direct-to-LDS loads
// whose completion the caller has already waited for (vector-memory counter
// and a workgroup barrier), so no further wait on those loads is needed.
template <int DT, int OFF0, int OFF1>
__device__ __forceinline__ void read_vt(const uint32_t (&a)[DT], uint2 (&r)[DT][2]);

// (The host compilation pass sees only the declarations: the register
// constraints exist for the GPU target alone.)
#define KVLINK_TR_READ(o, i, off) "ds_read_b64_tr_b16 %" #o ", %" #i " offset:%" #off "\n\t"
template <int OFF0, int OFF1>
__device__ __forceinline__ void read_vt8(const uint32_t (&a)[8], uint2 (&r)[8][2]) {
#if defined(__HIP_DEVICE_COMPILE__)
    asm volatile(
        KVLINK_TR_READ(0, 16, 24) KVLINK_TR_READ(1, 16, 25)
        KVLINK_TR_READ(2, 17, 24) KVLINK_TR_READ(3, 17, 25)
        KVLINK_TR_READ(4, 18, 24) KVLINK_TR_READ(5, 18, 25)
        KVLINK_TR_READ(6, 19, 24) KVLINK_TR_READ(7, 19, 25)
        KVLINK_TR_READ(8, 20, 24) KVLINK_TR_READ(9, 20, 25)
        KVLINK_TR_READ(10, 21, 24) KVLINK_TR_READ(11, 21, 25)
        KVLINK_TR_READ(12, 22, 24) KVLINK_TR_READ(13, 22, 25)
        KVLINK_TR_READ(14, 23, 24) KVLINK_TR_READ(15, 23, 25)
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(r[0][0]), "=&v"(r[0][1]), "=&v"(r[1][0]), "=&v"(r[1][1]), "=&v"(r[2][0]),
          "=&v"(r[2][1]), "=&v"(r[3][0]), "=&v"(r[3][1]), "=&v"(r[4][0]), "=&v"(r[4][1]),
          "=&v"(r[5][0]), "=&v"(r[5][1]), "=&v"(r[6][0]), "=&v"(r[6][1]), "=&v"(r[7][0]),
          "=&v"(r[7][1])
        : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "v"(a[4]), "v"(a[5]), "v"(a[6]),
          "v"(a[7]), "i"(OFF0), "i"(OFF1)
        : "memory");
#endif
}

template <int OFF0, int OFF1>
__device__ __forceinline__ void read_vt4(const uint32_t (&a)[4], uint2 (&r)[4][2]) {
#if defined(__HIP_DEVICE_COMPILE__)
    asm volatile(
        KVLINK_TR_READ(0, 8, 12) KVLINK_TR_READ(1, 8, 13)
        KVLINK_TR_READ(2, 9, 12) KVLINK_TR_READ(3, 9, 13)
        KVLINK_TR_READ(4, 10, 12) KVLINK_TR_READ(5, 10, 13)
        KVLINK_TR_READ(6, 11, 12) KVLINK_TR_READ(7, 11, 13)
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(r[0][0]), "=&v"(r[0][1]), "=&v"(r[1][0]), "=&v"(r[1][1]), "=&v"(r[2][0]),
          "=&v"(r[2][1]), "=&v"(r[3][0]), "=&v"(r[3][1])
        : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "i"(OFF0), "i"(OFF1)
        : "memory");
#endif
}
#undef KVLINK_TR_READ

template <int DT, int OFF0, int OFF1>
__device__ __forceinline__ void read_vt(const uint32_t (&a)[DT], uint2 (&r)[DT][2]) {
    if constexpr (DT == 8) read_vt8<OFF0, OFF1>(a, r);
    else read_vt4<OFF0, OFF1>(a, r);
}

// bf16 pair (RNE) of two floats, low half first: one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack2(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(floatx2{a, b}, bf16x2));
}

// LDS byte address of a pointer into a __shared__ array (the low 32 bits of
// its generic address).
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return static_cast<uint32_t>(reinterpret_cast<uintptr_t>(p));
}

// 16-byte direct load from global memory into LDS: lane i's bytes land at
// lds + 16 i (lds must be wave-uniform and not LDS address 0).  Device pass
// only, like the register-constrained asm above.
__device__ __forceinline__ void load_lds16(const void* src, void* lds) {
#if defined(__HIP_DEVICE_COMPILE__)
    __builtin_amdgcn_global_load_lds(src, lds, 16, 0, 0);
#endif
}

// Wait until at most n of this wave's vector-memory loads are outstanding.
template <int n>
__device__ __forceinline__ void wait_vm() {
    static_assert(n >= 0 && n < 64, "vmcnt range");
    // vmcnt is split over bits [3:0] and [15:14]; expcnt (bits [6:4]) and
    // lgkmcnt (bits [11:8]) are left at their maxima, i.e. not waited on
    __builtin_amdgcn_s_waitcnt((n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

template <int D>
__global__ __launch_bounds__(64 * kWaves, 1) void attend_mfma_kernel(KParams p) {
    constexpr int DT = D / 16;         // 16-dim tiles of O^T
    constexpr int DS = D / 32;         // 32-dim steps of S^T = K Q^T
    constexpr int KB = 4 * DS;         // 1 KB operand blocks of a K tile
    constexpr int VI = kTile * D * 2 / 1024;   // 1 KB direct loads of a V tile
    constexpr int CH = D / 8;          // 16-byte chunks per V row
    constexpr int LPW = (KB + VI) / kWaves;    // direct loads per wave per tile
    static_assert((KB % kWaves) == 0 && (VI % kWaves) == 0, "tile split");
    __shared__ __attribute__((aligned(1024))) unsigned char smem[Smem<D>::bytes];

    const int split = blockIdx.x;
    const int s = blockIdx.z / p.n_kv_heads, h = blockIdx.z % p.n_kv_heads;
    const int G = p.group;
    // request descriptors (independent loads)
    const int n0 = p.seq_new_ptr[s];
    const int rows_s = (p.seq_new_ptr[s + 1] - n0) * G;
    const int Tc = p.seq_cached[s];
    const int rho0 = blockIdx.y * kRB;
    if (rho0 >= rows_s) return;

    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int lr = lane & 15, lg = lane >> 4;
    const int rho_w = rho0 + wave * kRT * 16;      // first row of this wave

    // Everything below depends on n0 only and is requested together before
    // the split's key range is known: the block's key bound, the visible
    // prefix of this wave's first token and of every row, and the Q operand.
    const int r_last = (min(rho0 + kRB, rows_s) - 1) / G;
    const int cmax = p.new_visible[n0 + r_last];
    const int wave_vis_min = p.new_visible[n0 + min(rho_w, rows_s - 1) / G];
    int tok[kRT], vis[kRT];
#pragma unroll
    for (int rt = 0; rt < kRT; ++rt) {
        const int rho = rho_w + 16 * rt + lr;
        tok[rt] = rho < rows_s ? rho / G : -1;
        vis[rt] = p.new_visible[n0 + max(tok[rt], 0)];
    }
    const bf16_t* q_rot = reinterpret_cast<const bf16_t*>(p.q_rot);
    uint4 qraw[kRT][DS];
#pragma unroll
    for (int rt = 0; rt < kRT; ++rt) {
        const int rho = rho_w + 16 * rt + lr;
        const int64_t qrow = ((int64_t)(n0 + max(tok[rt], 0)) * p.n_q_heads + h * G + rho % G) * D;
#pragma unroll
        for (int ds = 0; ds < DS; ++ds)
            qraw[rt][ds] = *reinterpret_cast<const uint4*>(q_rot + qrow + 32 * ds + 8 * lg);
    }

    // the block's virtual key range: cached rows its last token sees, then
    // the new rows up to its last token; this workgroup's split of it
    BlockKeys bk;
    bk.r_last = r_last;
    bk.cmax = cmax;
    bk.nvirt = cmax + r_last + 1;
    const int kbeg = split * p.split_keys;
    if (kbeg >= bk.nvirt) return;
    const int kend = min(kbeg + p.split_keys, bk.nvirt);
    const float c2 = p.scale_log2;   // > 0

    // Row r may see virtual key v iff v < lo (cached rows up to its document,
    // within the split) or cmax <= v <= hi (new rows up to its own, within
    // the split).
    int lo[kRT], hi[kRT];
#pragma unroll
    for (int rt = 0; rt < kRT; ++rt) {
        lo[rt] = tok[rt] >= 0 ? min(vis[rt], kend) : 0;
        hi[rt] = tok[rt] >= 0 ? min(bk.cmax + tok[rt], kend - 1) : -1;
    }
    bf16x8 qB[kRT][DS];
#pragma unroll
    for (int rt = 0; rt < kRT; ++rt)
#pragma unroll
        for (int ds = 0; ds < DS; ++ds)
            qB[rt][ds] = as_bf16x8(tok[rt] >= 0 ? qraw[rt][ds] : uint4{0u, 0u, 0u, 0u});

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
    const int n_tiles = (kend - kbeg + kTile - 1) / kTile;

    // virtual key -> cache row, clamped into the split so that every load
    // reads a real row (keys past the split end are masked)
    auto key_row = [&](int v) {
        v = min(v, kend - 1);
        return v < bk.cmax ? v : Tc + (v - bk.cmax);
    };
    // Per-lane parts of the direct-load addresses, fixed for the whole
    // split: this wave loads K blocks wave + kWaves*i and V slots
    // (wave + kWaves*i)*64 + lane of every tile.
    constexpr int KI = KB / kWaves, VJ = VI / kWaves;
    int k_key[KI], k_off[KI], v_key[VJ], v_off[VJ];
#pragma unroll
    for (int i = 0; i < KI; ++i) {
        const int b = wave + kWaves * i;                  // K block (sc, kt, ds)
        const int ds = b % DS, kt = (b / DS) % 2, sc = b / (2 * DS);
        k_key[i] = 32 * sc + 16 * kt + lr;
        k_off[i] = 64 * ds + 16 * lg;
    }
#pragma unroll
    for (int i = 0; i < VJ; ++i) {
        const int pos = (wave + kWaves * i) * 64 + lane;  // 16-byte slot of the V tile
        const int key = pos / CH, pc = pos % CH;
        v_key[i] = key;
        v_off[i] = 16 * (pc ^ (key & (CH - 1)));          // logical chunk stored at slot pc
    }
    // per-lane part of the V^T operand reads (see the product below): lane
    // (lg, lr) reads key 4lg + lr/4 (plus multiples of 16, which leave the
    // swizzle unchanged), logical chunk 2dt + (lr/2)%2, half lr%2
    uint32_t v_rel[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
        const int key = 4 * lg + (lr >> 2);
        const int c = 2 * dt + ((lr >> 1) & 1);
        v_rel[dt] = key * (2 * D) + 16 * (c ^ (key & (CH - 1))) + 8 * (lr & 1);
    }
    const bool contiguous = kp.table == nullptr && vp.table == nullptr;
    const int fast_end = min(kend, bk.cmax);              // rows here are the keys themselves

    // this wave's share of tile t, straight into LDS stage t % kStages
    auto issue_tile = [&](int t) {
        unsigned char* st = smem + Smem<D>::base + (t % kStages) * Smem<D>::stage;
        const int tb = kbeg + t * kTile;
        if (contiguous && tb + kTile <= fast_end) {
            // the whole tile is cached rows tb.., one 64-bit add per load
            const char* kt0 = kp.base + (int64_t)tb * kp.row_bytes;
            const char* vt0 = vp.base + (int64_t)tb * vp.row_bytes;
#pragma unroll
            for (int i = 0; i < KI; ++i)
                load_lds16(kt0 + k_key[i] * kp.row_bytes + k_off[i], st + (wave + kWaves * i) * 1024);
#pragma unroll
            for (int i = 0; i < VJ; ++i)
                load_lds16(vt0 + v_key[i] * vp.row_bytes + v_off[i],
                           st + Smem<D>::k_bytes + (wave + kWaves * i) * 1024);
        } else {
#pragma unroll
            for (int i = 0; i < KI; ++i)
                load_lds16(kp.row(key_row(tb + k_key[i])) + k_off[i], st + (wave + kWaves * i) * 1024);
#pragma unroll
            for (int i = 0; i < VJ; ++i)
                load_lds16(vp.row(key_row(tb + v_key[i])) + v_off[i],
                           st + Smem<D>::k_bytes + (wave + kWaves * i) * 1024);
        }
    };

#pragma unroll
    for (int t = 0; t < kStages - 1; ++t)
        if (t < n_tiles) issue_tile(t);

    for (int t = 0; t < n_tiles; ++t) {
        // this wave's loads of tile t are done when at most those of the
        // next kStages-2 tiles are still outstanding; the barrier makes every
        // wave's part visible and frees the stage of tile t-1 for tile
        // t+kStages-1
        const int ahead = min(kStages - 2, n_tiles - 1 - t);
        if (ahead >= 2) wait_vm<2 * LPW>(); else if (ahead == 1) wait_vm<LPW>(); else wait_vm<0>();
        __syncthreads();
        if (t + kStages - 1 < n_tiles) issue_tile(t + kStages - 1);

        const unsigned char* st = smem + Smem<D>::base + (t % kStages) * Smem<D>::stage;
        // V^T operand addresses of this stage (the sub-tile and key-half
        // parts are immediate offsets of the reads)
        uint32_t va[DT];
        const uint32_t vt = lds_addr(st + Smem<D>::k_bytes);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) va[dt] = vt + v_rel[dt];

        auto sub_tile = [&](auto sc_const) {
            constexpr int sc = decltype(sc_const)::value;
            const int v0 = kbeg + t * kTile + 32 * sc;

            // S^T = K Q^T
            floatx4 sacc[2][kRT];
#pragma unroll
            for (int kt = 0; kt < 2; ++kt) {
#pragma unroll
                for (int rt = 0; rt < kRT; ++rt) sacc[kt][rt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ds = 0; ds < DS; ++ds) {
                    const bf16x8 a = as_bf16x8(*reinterpret_cast<const uint4*>(
                        st + ((sc * 2 + kt) * DS + ds) * 1024 + lane * 16));
#pragma unroll
                    for (int rt = 0; rt < kRT; ++rt)
                        sacc[kt][rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qB[rt][ds],
                                                                               sacc[kt][rt], 0, 0, 0);
                }
            }

            // mask, by the kind of sub-tile (wave-uniform): keys below every
            // row's visible prefix need none; keys in the cached region need
            // v < lo; keys in the new-token region need v <= hi; a sub-tile
            // across cmax needs both tests.  Lane group g holds key offsets
            // 16kt + 4g + i of the sub-tile.
            const int vb = v0 + 4 * lg;
            if (v0 + 32 > wave_vis_min) {
                if (v0 + 32 <= bk.cmax) {
#pragma unroll
                    for (int rt = 0; rt < kRT; ++rt) {
                        const int t_lo = lo[rt] - vb;
#pragma unroll
                        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                            for (int i = 0; i < 4; ++i)
                                sacc[kt][rt][i] = 16 * kt + i < t_lo ? sacc[kt][rt][i] : -INFINITY;
                    }
                } else if (v0 >= bk.cmax) {
#pragma unroll
                    for (int rt = 0; rt < kRT; ++rt) {
                        const int t_hi = hi[rt] - vb;
#pragma unroll
                        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                            for (int i = 0; i < 4; ++i)
                                sacc[kt][rt][i] = 16 * kt + i <= t_hi ? sacc[kt][rt][i] : -INFINITY;
                    }
                } else {
#pragma unroll
                    for (int rt = 0; rt < kRT; ++rt) {
                        const int t_lo = lo[rt] - vb, t_c = bk.cmax - vb, t_hi = hi[rt] - vb;
#pragma unroll
                        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                            for (int i = 0; i < 4; ++i) {
                                const int o = 16 * kt + i;
                                const bool ok = o < t_lo || (o >= t_c && o <= t_hi);
                                sacc[kt][rt][i] = ok ? sacc[kt][rt][i] : -INFINITY;
                            }
                    }
                }
            }

            // online softmax in base 2 with a lazily raised maximum, on
            // x = s * scale_log2 - m: the slow path (cross-lane maximum,
            // rescale of O and l) runs only if some x exceeds kTau.  The
            // maximum is taken over x, the result of a fused multiply-add,
            // so no NaN-quieting is needed in front of it.
            float x[kRT][8];
            bool over = false;
#pragma unroll
            for (int rt = 0; rt < kRT; ++rt) {
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    x[rt][j] = __builtin_fmaf(sacc[j >> 2][rt][j & 3], c2, -m[rt]);
                const float mx = fmaxf(fmaxf(fmaxf(x[rt][0], x[rt][1]), fmaxf(x[rt][2], x[rt][3])),
                                       fmaxf(fmaxf(x[rt][4], x[rt][5]), fmaxf(x[rt][6], x[rt][7])));
                over |= mx > kTau;
            }
            if (__builtin_amdgcn_ballot_w64(over)) {
                // from the raw scores: x loses them while m is still kNoMax
#pragma unroll
                for (int rt = 0; rt < kRT; ++rt) {
                    float r = fmaxf(fmaxf(fmaxf(sacc[0][rt][0], sacc[0][rt][1]),
                                          fmaxf(sacc[0][rt][2], sacc[0][rt][3])),
                                    fmaxf(fmaxf(sacc[1][rt][0], sacc[1][rt][1]),
                                          fmaxf(sacc[1][rt][2], sacc[1][rt][3])));
                    r = fmaxf(r, __shfl_xor(r, 16));
                    r = fmaxf(r, __shfl_xor(r, 32));
                    const float m_new = fmaxf(m[rt], r * c2);
                    const float alpha = __builtin_amdgcn_exp2f(m[rt] - m_new);
                    m[rt] = m_new;
                    lsum[rt] *= alpha;
#pragma unroll
                    for (int dt = 0; dt < DT; ++dt) o[dt][rt] *= alpha;
#pragma unroll
                    for (int j = 0; j < 8; ++j)
                        x[rt][j] = __builtin_fmaf(sacc[j >> 2][rt][j & 3], c2, -m_new);
                }
            }
            // p = 2^x, packed to bf16 pairs; the row sum adds the rounded
            // pairs (the weights the product below uses) with dot products
            // against (1, 1)
            uint32_t pk[kRT][4];
            const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
            for (int rt = 0; rt < kRT; ++rt)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    pk[rt][j] = pack2(__builtin_amdgcn_exp2f(x[rt][2 * j]),
                                      __builtin_amdgcn_exp2f(x[rt][2 * j + 1]));
                    lsum[rt] = __builtin_amdgcn_fdot2_f32_bf16(
                        __builtin_bit_cast(bf16x2, pk[rt][j]), ones, lsum[rt], false);
                }

            // O^T += V^T P^T.  For a 16-lane block, the transpose read gives
            // lane i element i%4 of the 4-element rows supplied by lanes
            // 4k + i/4 (k = 0..3); lane j therefore supplies key
            // 32sc + 16h + 4lg + j/4, dims 16dt + 4(j%4).., so that lane i
            // receives keys 4lg+k (k = 0..3) of dim 16dt + i.
            uint2 vr[DT][2];
            read_vt<DT, 32 * sc * 2 * D, (32 * sc + 16) * 2 * D>(va, vr);
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                const uint2* half = vr[dt];
                const bf16x8 a = as_bf16x8(uint4{half[0].x, half[0].y, half[1].x, half[1].y});
#pragma unroll
                for (int rt = 0; rt < kRT; ++rt)
                    o[dt][rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        a, as_bf16x8(uint4{pk[rt][0], pk[rt][1], pk[rt][2], pk[rt][3]}), o[dt][rt],
                        0, 0, 0);
            }
        };
        sub_tile(std::integral_constant<int, 0>{});
        if (kbeg + t * kTile + 32 < kend) sub_tile(std::integral_constant<int, 1>{});
    }

    // row sums: add the four lane groups that hold each row
#pragma unroll
    for (int rt = 0; rt < kRT; ++rt) {
        lsum[rt] += __shfl_xor(lsum[rt], 16);
        lsum[rt] += __shfl_xor(lsum[rt], 32);
    }

    // each wave writes its own rows
#pragma unroll
    for (int rt = 0; rt < kRT; ++rt) {
        if (tok[rt] < 0) continue;
        const int rho = rho_w + 16 * rt + lr;
        const int64_t orow = (int64_t)(n0 + tok[rt]) * p.n_q_heads + h * G + rho % G;
        if (p.n_splits == 1) {
            bf16_t* out = reinterpret_cast<bf16_t*>(p.out) + orow * D;
            const float inv = 1.f / lsum[rt];
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                const floatx4 v = o[dt][rt];
                *reinterpret_cast<uint2*>(out + 16 * dt + 4 * lg) =
                    uint2{pack2(v[0] * inv, v[1] * inv), pack2(v[2] * inv, v[3] * inv)};
            }
            if (p.lse && lg == 0) p.lse[orow] = (m[rt] + log2f(lsum[rt])) * kLn2;
        } else {
            const int64_t pi = orow * p.n_splits + split;
            float* po = p.part_o + pi * D;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt)
                *reinterpret_cast<floatx4*>(po + 16 * dt + 4 * lg) = o[dt][rt];
            if (lg == 0) {
                p.part_ml[pi * 2] = m[rt];
                p.part_ml[pi * 2 + 1] = lsum[rt];
            }
        }
    }
}

}  // namespace

int attend_mfma_row_block() { return kRB; }

hipError_t launch_attend_mfma(int head_dim, const KParams& p, dim3 grid, hipStream_t stream) {
    if (head_dim == 128)
        hipLaunchKernelGGL(attend_mfma_kernel<128>, grid, dim3(64 * kWaves), 0, stream, p);
    else
        hipLaunchKernelGGL(attend_mfma_kernel<64>, grid, dim3(64 * kWaves), 0, stream, p);
    return hipGetLastError();
}

}  // namespace attn
}  // namespace kvlink
