// attend_mfma.hip — bf16 split-K attention of the new tokens on gfx950 matrix
// cores (v_mfma_f32_16x16x32_bf16, float accumulation).
//
// A unit is one KV head's GQA-packed rows of one request (a block of 256,
// 128 or 64 rows: 64, 32 or 16 tokens x 4 heads for a group of 4); its keys
// are walked in 64-key tiles.  The workgroups are persistent: each owns a
// contiguous range of the schedule's tiles, which may cover the end of one
// unit and the start of the next (one segment per unit touched).  The eight
// wavefronts (two per SIMD, so one's softmax can overlap the other's matrix
// products) split a unit two ways, by a template choice:
//
//   * 256-row units: each wavefront owns 32 rows and walks every key of the
//     segment;
//   * 128- and 64-row units: the wavefronts form two key groups of four; in
//     each group a wavefront owns 32 (or 16) rows, and group g takes the
//     32-key half g of every tile.  The two groups' online-softmax states of
//     a row are merged through LDS at the end of the segment.
//
// K and V tiles are brought into LDS once per workgroup and shared by the
// eight waves:
//
//   * the tiles are loaded straight from global memory into a four-stage
//     LDS ring with 16-byte direct-to-LDS loads (each wave issues an eighth
//     of a tile), at no register cost.  At the barrier of tile t each wave
//     has waited for its own loads of tile t+1 only (the loads of a wave
//     complete in issue order; a direct-to-LDS load counts as complete once
//     its bytes are in LDS), so tiles t+2 and t+3 stay in flight across it;
//     with the fused re-encode, which rewrites a tile in LDS after its
//     barrier, the barrier is a full one;
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
//
// A unit cut into several segments stores one partial result per segment
// (O / l in bf16, (m, l) in float).  The partials are merged either by the
// combine launch that follows, or, by the schedule's choice, inside the same
// launch: each segment then stores its partial with agent-coherent stores,
// waits for them, and increments the unit's arrival counter; the workgroup
// that arrives last reads every segment's partial back with agent-coherent
// loads and writes the unit's output and LSE.  The counter wraps to zero on
// the last arrival, so a counter array that starts at zero is left at zero
// by every launch.
#include <algorithm>
#include <type_traits>

#include "attend_common.h"
#include "merge_launch.h"
#include "mfma_ops.h"

namespace kvlink {
namespace attn {

namespace {

constexpr int kWaves = 8;
constexpr int kTile = 64;                 // keys per LDS stage
constexpr int kStages = 4;
// Rescale threshold of the online softmax, in log2 units: p = 2^(s - m)
// stays below 2^kTau (exact in float, representable in bf16).
constexpr float kTau = 8.0f;

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

// LDS of the fused re-encode, after the ring: the (cos, sin) table of every
// span of the request ([kMaxFuseSpans][D/2]) and the spans' first and end
// rows and deltas.
template <int D>
struct FuseSmem {
    static constexpr int cs = 0;
    static constexpr int start = cs + kMaxFuseSpans * (D / 2) * 8;
    static constexpr int end = start + kMaxFuseSpans * 4;
    static constexpr int delta = end + kMaxFuseSpans * 4;
    static constexpr int bytes = delta + kMaxFuseSpans * 4;
};

// Shape of a unit: kRT 16-row tiles per wavefront and kKG key groups; the
// wavefronts of a group own kRB rows between them.
template <int kRT_, int kKG_>
struct Shape {
    static constexpr int kRT = kRT_;
    static constexpr int kKG = kKG_;
    static constexpr int kRW = kWaves / kKG;        // wavefronts per key group
    static constexpr int kRB = kRW * kRT * 16;      // GQA rows per unit
    static constexpr bool kMergeInLaunch = kKG == 2;
    static_assert(kKG == 1 || kKG == 2, "one or two key groups");
    static_assert(kRT == 1 || kRT == 2, "one or two row tiles per wavefront");
};

// One segment of a unit: tiles [tile_a, tile_b) of the key range of KV head
// h's rows [rho0, rho0 + rows) of request s, from its schedule record.
// Every early return is uniform over the workgroup.
template <int D, class S, bool kFuse, bool kPaged>
__device__ __forceinline__ void attend_segment(const KParams& p, unsigned char* smem,
                                               const int4 (&rec)[4]) {
    constexpr int kRT = S::kRT, kKG = S::kKG, kRW = S::kRW, kRB = S::kRB;
    constexpr int DT = D / 16;         // 16-dim tiles of O^T
    constexpr int DS = D / 32;         // 32-dim steps of S^T = K Q^T
    constexpr int KB = 4 * DS;         // 1 KB operand blocks of a K tile
    constexpr int VI = kTile * D * 2 / 1024;   // 1 KB direct loads of a V tile
    constexpr int CH = D / 8;          // 16-byte chunks per V row
    constexpr int LPW = (KB + VI) / kWaves;    // direct loads per wave per tile
    static_assert((KB % kWaves) == 0 && (VI % kWaves) == 0, "tile split");

    const int s = rec[0].x, h = rec[0].y, rho0 = rec[0].z, rows = rec[0].w;
    const int tile_a = rec[1].x, tile_b = rec[1].y;
    const int nseg = rec[1].z, seg_local = rec[1].w, part = rec[3].x, unit = rec[3].z;
    const bool direct = nseg == 1;
    const int n0 = rec[2].x, Tc = rec[2].y;
    BlockKeys bk;
    bk.cmax = rec[2].z;
    bk.nvirt = rec[2].w;
    const int G = p.group;
    const int kbeg = tile_a * kTile;
    if (kbeg >= bk.nvirt || rows < 1) return;
    const int kend = min(tile_b * kTile, bk.nvirt);
    const int n_tiles = (kend - kbeg + kTile - 1) / kTile;
    const int rho_end = rho0 + rows;

    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    const int lr = lane & 15, lg = lane >> 4;
    const int rw = wave % kRW, kg = wave / kRW;    // row wave and key group
    const int rho_w = rho0 + rw * kRT * 16;        // first row of this wave

    // (contiguous caches: the launch picks kPaged = false only when neither
    // view has a block table, and the null tables below fold every paged
    // branch away)
    RowPtr kp = row_ptr<bf16_t>(p.k, p.layer, h, s);
    RowPtr vp = row_ptr<bf16_t>(p.v, p.layer, h, s);
    if constexpr (!kPaged) {
        kp.table = nullptr;
        vp.table = nullptr;
    }

    // virtual key -> cache row, clamped into the segment so that every load
    // reads a real row (keys past the segment end are masked)
    auto key_row = [&](int v) {
        v = min(v, kend - 1);
        return v < bk.cmax ? v : Tc + (v - bk.cmax);
    };
    // With the fused RoPE the tiles take the new rows' values straight from
    // v_new (new row r of the request, this KV head): only the keys go
    // through the cache, which the segment appends them to first.  256-row
    // units only: with many segments appending the same new rows it saves
    // 1.4% on the shared-pool batch; 64-row units measured no gain (and the
    // fused re-encode's instances have no register to spare).
    constexpr bool kVDirect = !kFuse && S::kRB == 256;
    const bool v_direct = kVDirect && p.rope != nullptr;
    auto v_new_row = [&](int r) {
        return reinterpret_cast<const char*>(p.v_new) +
               ((int64_t)(n0 + r) * p.n_kv_heads + h) * (D * (int64_t)sizeof(bf16_t));
    };
    // Per-lane parts of the direct-load addresses, fixed for the whole
    // segment: this wave loads K blocks wave + kWaves*i and V slots
    // (wave + kWaves*i)*64 + lane of every tile.
    constexpr int KI = KB / kWaves, VJ = VI / kWaves;
    static_assert(64 / CH <= 16, "a V load spans one 16-key group");
    int k_key[KI], k_off[KI], v_key[VJ], v_off[VJ];
    int k_key0[KI], v_key0[VJ];                           // first key of the load (uniform)
#pragma unroll
    for (int i = 0; i < KI; ++i) {
        const int b = wave + kWaves * i;                  // K block (sc, kt, ds)
        const int ds = b % DS, kt = (b / DS) % 2, sc = b / (2 * DS);
        k_key0[i] = 32 * sc + 16 * kt;
        k_key[i] = k_key0[i] + lr;
        k_off[i] = 64 * ds + 16 * lg;
    }
#pragma unroll
    for (int i = 0; i < VJ; ++i) {
        const int pos = (wave + kWaves * i) * 64 + lane;  // 16-byte slot of the V tile
        const int key = pos / CH, pc = pos % CH;
        v_key0[i] = (wave + kWaves * i) * 64 / CH;
        v_key[i] = key;
        v_off[i] = 16 * (pc ^ (key & (CH - 1)));          // logical chunk stored at slot pc
    }
    // rows below fast_end are the keys themselves; tiles there take their
    // rows by 16-row groups (one page each, when paged): a load's address is
    // its group's first row (the same in every lane, or the tile's first row
    // when contiguous) plus a 32-bit lane offset fixed for the segment
    const bool grouped = kp.groups_of_16() && vp.groups_of_16() &&
                         kp.row_bytes < (1 << 24) && vp.row_bytes < (1 << 24);
    const int fast_end = grouped ? min(kend, bk.cmax) : 0;
    uint32_t k_lane[KI], v_lane[VJ];
#pragma unroll
    for (int i = 0; i < KI; ++i) k_lane[i] = (uint32_t)(lr * kp.row_bytes + k_off[i]);
#pragma unroll
    for (int i = 0; i < VJ; ++i) v_lane[i] = (uint32_t)((v_key[i] & 15) * vp.row_bytes + v_off[i]);

    // this wave's share of tile t, straight into LDS stage t % kStages
    auto issue_tile = [&](int t) {
        unsigned char* st = smem + Smem<D>::base + (t % kStages) * Smem<D>::stage;
        const int tb = kbeg + t * kTile;
        if (!kPaged && tb + kTile <= fast_end) {
            // contiguous rows: one base per tile
            const char* kb = kp.base + (int64_t)tb * kp.row_bytes;
            const char* vb = vp.base + (int64_t)tb * vp.row_bytes;
#pragma unroll
            for (int i = 0; i < KI; ++i)
                load_lds16(kb + (k_lane[i] + (uint32_t)(k_key0[i] * kp.row_bytes)),
                           st + (wave + kWaves * i) * 1024);
#pragma unroll
            for (int i = 0; i < VJ; ++i)
                load_lds16(vb + (v_lane[i] + (uint32_t)((v_key0[i] & ~15) * vp.row_bytes)),
                           st + Smem<D>::k_bytes + (wave + kWaves * i) * 1024);
        } else if (tb + kTile <= fast_end) {
            // a K block covers keys g..g+15 and a V load keys within one
            // aligned 16-key group g, so one page per load; the page reads
            // of the tile go out together, ahead of the address arithmetic
            int kpg[KI] = {}, vpg[VJ] = {};
            if (kp.table) {
#pragma unroll
                for (int i = 0; i < KI; ++i) kpg[i] = kp.page_of(tb + k_key0[i]);
            }
            if (vp.table) {
#pragma unroll
                for (int i = 0; i < VJ; ++i) vpg[i] = vp.page_of(tb + (v_key0[i] & ~15));
            }
#pragma unroll
            for (int i = 0; i < KI; ++i)
                load_lds16(kp.in_page(kpg[i], tb + k_key0[i]) + k_lane[i],
                           st + (wave + kWaves * i) * 1024);
#pragma unroll
            for (int i = 0; i < VJ; ++i)
                load_lds16(vp.in_page(vpg[i], tb + (v_key0[i] & ~15)) + v_lane[i],
                           st + Smem<D>::k_bytes + (wave + kWaves * i) * 1024);
        } else {
#pragma unroll
            for (int i = 0; i < KI; ++i)
                load_lds16(kp.row(key_row(tb + k_key[i])) + k_off[i], st + (wave + kWaves * i) * 1024);
#pragma unroll
            for (int i = 0; i < VJ; ++i) {
                const int v = min(tb + v_key[i], kend - 1);
                const char* src = v_direct && v >= bk.cmax ? v_new_row(v - bk.cmax) : vp.row(key_row(v));
                load_lds16(src + v_off[i], st + Smem<D>::k_bytes + (wave + kWaves * i) * 1024);
            }
        }
    };

    // With the fused RoPE, the new rows among the segment's keys ([na, nb)
    // of the request's new tokens) are appended to the cache before any tile
    // holding them is loaded: ahead of tile 0 when it holds some, else while
    // tile 0 is in flight (the prologue's full wait and barrier below then
    // cover the stores before tiles 1.. go out).
    const int na = max(kbeg, bk.cmax) - bk.cmax, nb = kend - bk.cmax;
    const bool has_new = p.rope != nullptr && nb > na;
    const bool tile0_new = has_new && kbeg + kTile > bk.cmax;
    if (tile0_new) {
        append_new_rows<D, 64 * kWaves, !kVDirect>(p, kp, vp, h, n0, Tc, na, nb);
        wait_vm_all();
        __syncthreads();
    }

    // The queries go out first (they come from the L2: every segment of the
    // unit reads them), then tile 0, then the rows' visible prefixes; the
    // queries' rotation (fused RoPE) runs while tile 0 is in flight.  Tiles 1
    // and 2 follow once tile 0 has arrived and its first products are
    // issued, so that when every workgroup starts at once tile 0 is not
    // queued behind them (its products are what the loop waits for; issuing
    // tiles 1..3 with tile 0 measured no faster on any workload).
    // Fused re-encode: the request's spans are read first (one per thread),
    // so that waiting for them never waits for tile 0
    unsigned char* fsm = smem + Smem<D>::bytes;
    int f_n = 0;
    int4 f_sp = {0, 0, 0, 0};
    if constexpr (kFuse) {
        const int b0 = load_uniform(p.fuse_span_ptr + s);
        f_n = min(max(load_uniform(p.fuse_span_ptr + s + 1) - b0, 0), kMaxFuseSpans);
        if ((int)threadIdx.x < f_n) {
            const kvlink_span sp = p.fuse_spans[b0 + threadIdx.x];
            f_sp = int4{sp.dst_row, sp.dst_row + sp.len, sp.delta, 0};
        }
    }
    int tok[kRT];
    QRow<D> qrow[kRT];
#pragma unroll
    for (int rt = 0; rt < kRT; ++rt) {
        const int rho = rho_w + 16 * rt + lr;
        tok[rt] = rho < rho_end ? rho / G : -1;
        qrow[rt].load(p, n0 + max(tok[rt], 0), h * G + rho % G, lg);
    }
    issue_tile(0);
    // ... and their (cos, sin) tables built while tile 0 is in flight (the
    // previous segment's rotations are done with the area: its last tile's
    // rotation ended in a barrier)
    if constexpr (kFuse) {
        int* f_start = reinterpret_cast<int*>(fsm + FuseSmem<D>::start);
        int* f_end = reinterpret_cast<int*>(fsm + FuseSmem<D>::end);
        int* f_delta = reinterpret_cast<int*>(fsm + FuseSmem<D>::delta);
        if ((int)threadIdx.x < f_n) {
            f_start[threadIdx.x] = f_sp.x;
            f_end[threadIdx.x] = f_sp.y;
            f_delta[threadIdx.x] = f_sp.z;
        }
        __syncthreads();
        float2* f_cs = reinterpret_cast<float2*>(fsm + FuseSmem<D>::cs);
        for (int i = threadIdx.x; i < f_n * (D / 2); i += 64 * kWaves) {
            float c, sn;
            rope_cos_sin((int64_t)f_delta[i / (D / 2)], i % (D / 2), p.freqs, &c, &sn);
            f_cs[i] = float2{c, sn};
        }
    }
    int vis[kRT];
#pragma unroll
    for (int rt = 0; rt < kRT; ++rt) vis[rt] = p.new_visible[n0 + max(tok[rt], 0)];
    // this wave's rows: the first and last tokens, the visible prefix of the
    // last (prefixes grow with the token)
    // (scalar loads at clamped indices: a vector load here would make the
    // compiler wait for every load in flight, tile 0's included, before the
    // queries' rotation)
    const bool wave_active = rho_w < rho_end;
    const int tok_min = min(rho_w, rho_end - 1) / G;
    const int tok_max = (min(rho_w + kRT * 16, rho_end) - 1) / G;
    const int vis_lo = load_uniform(p.new_visible + n0 + tok_min);
    const int vis_hi = load_uniform(p.new_visible + n0 + tok_max);
    const int wave_vis_min = wave_active ? vis_lo : 0;
    const int wave_vis_max = wave_active ? vis_hi : 0;
    // the Q operand (rows past the block end hold the request's first
    // token's queries: finite values whose results are never written)
    bf16x8 qB[kRT][DS];
#pragma unroll
    for (int rt = 0; rt < kRT; ++rt) {
        uint4 q[DS];
        qrow[rt].get(p, q);
#pragma unroll
        for (int ds = 0; ds < DS; ++ds) qB[rt][ds] = as_bf16x8(q[ds]);
    }
    if (has_new && !tile0_new) append_new_rows<D, 64 * kWaves, !kVDirect>(p, kp, vp, h, n0, Tc, na, nb);

    const float c2 = p.scale_log2;   // > 0
    // Row r may see virtual key v iff v < lo (cached rows up to its document,
    // within the segment) or cmax <= v <= hi (new rows up to its own, within
    // the segment).
    int lo[kRT], hi[kRT];
#pragma unroll
    for (int rt = 0; rt < kRT; ++rt) {
        lo[rt] = tok[rt] >= 0 ? min(vis[rt], kend) : 0;
        hi[rt] = tok[rt] >= 0 ? min(bk.cmax + tok[rt], kend - 1) : -1;
    }
    // A 32-key sub-tile from v0 is dead for this wave when no row of it sees
    // any of its keys: all cached keys at or past the last row's prefix and
    // all new keys past the last row's token (always, for a wave without
    // rows).  It is live iff v0 < live_a (it starts below the segment end,
    // the cached region's end and the widest prefix) or live_b < v0 <= live_c
    // (it reaches past cmax and starts at or before the last row's new key
    // and the segment end): three scalar compares per test.
    const int live_a = wave_active ? min(min(wave_vis_max, bk.cmax), kend) : -1;
    const int live_b = bk.cmax - 32;
    const int live_c = wave_active ? min(bk.cmax + tok_max, kend - 1) : -1;
    auto dead = [&](int v0) { return !(v0 < live_a || (v0 > live_b && v0 <= live_c)); };

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

    // ---- pieces of a 32-key sub-tile.  A sub-tile is addressed by the
    // start of its K blocks (ks: half h of a stage's K area starts
    // h * 2 * DS KB in) and of its V rows (vs: half h starts 32 h rows into
    // the stage's V area).
    auto k_sub = [&](const unsigned char* st, int h) { return st + h * 2 * DS * 1024; };
    auto v_sub = [&](const unsigned char* st, int h) {
        return st + Smem<D>::k_bytes + h * 32 * 2 * D;
    };

    // one 16-key half kt of S^T = K Q^T
    auto qk_half = [&](const unsigned char* ks, auto kt_const, floatx4 (&sacc)[2][kRT]) {
        constexpr int kt = decltype(kt_const)::value;
#pragma unroll
        for (int rt = 0; rt < kRT; ++rt) sacc[kt][rt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ds = 0; ds < DS; ++ds) {
            const bf16x8 a = as_bf16x8(
                *reinterpret_cast<const uint4*>(ks + (kt * DS + ds) * 1024 + lane * 16));
#pragma unroll
            for (int rt = 0; rt < kRT; ++rt)
                sacc[kt][rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qB[rt][ds],
                                                                       sacc[kt][rt], 0, 0, 0);
        }
    };

    // keys below every row's visible prefix need no mask; keys in the cached
    // region need v < lo; keys in the new-token region need v <= hi; a
    // sub-tile across cmax needs both tests (the kind is wave-uniform).
    // Lane group g holds key offsets 16kt + 4g + i of the sub-tile.
    auto mask = [&](floatx4 (&sacc)[2][kRT], int v0) {
        const int vb = v0 + 4 * lg;
        if (v0 + 32 <= wave_vis_min) return;
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
    };

    // O^T += V^T P^T.  For a 16-lane block, the transpose read gives lane i
    // element i%4 of the 4-element rows supplied by lanes 4k + i/4 (k =
    // 0..3); lane j therefore supplies key 16e + 4lg + j/4 of the sub-tile
    // (e: key half), dims 16dt + 4(j%4).., so that lane i receives keys
    // 4lg+k (k = 0..3) of dim 16dt + i.  The key-half part of the addresses
    // is an immediate offset.
    auto v_issue = [&](const unsigned char* vs, uint2 (&vr)[DT][2]) {
        const uint32_t vt = lds_addr(vs);
        uint32_t va[DT];
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) va[dt] = vt + v_rel[dt];
        issue_vt<DT, 0, 16 * 2 * D>(va, vr);
    };
    // One step of the pipeline: the current sub-tile (S in s_cur, keys from
    // v0, values at vc) becomes P and is added to O, while the matrix cores
    // compute S of the next sub-tile (K at kn) into s_nxt.  The online
    // softmax works in base 2 on x = s * scale_log2 - m with a lazily raised
    // maximum: the slow path (cross-lane maximum, rescale of O and l) runs
    // only if some x exceeds kTau; the maximum is taken over x, the result of
    // a fused multiply-add, so no NaN-quieting is needed in front of it.  P
    // is packed to bf16 pairs; the row sum adds the rounded pairs (the
    // weights the product uses) with dot products against (1, 1).
    //
    // The vector work is written out in chunks, one per matrix product, each
    // chunk fenced by a scheduling barrier: a product occupies the matrix
    // core for 16 cycles, during which the wave issues the chunk's
    // independent vector instructions.
    auto step = [&](floatx4 (&s_cur)[2][kRT], floatx4 (&s_nxt)[2][kRT], int v0,
                    const unsigned char* vc, const unsigned char* kn) {
        mask(s_cur, v0);

        // K operands of the next sub-tile (both key halves)
        bf16x8 ka[2][DS];
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int ds = 0; ds < DS; ++ds)
                ka[kt][ds] = as_bf16x8(
                    *reinterpret_cast<const uint4*>(kn + (kt * DS + ds) * 1024 + lane * 16));
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
            for (int rt = 0; rt < kRT; ++rt) s_nxt[kt][rt] = floatx4{0.f, 0.f, 0.f, 0.f};

        // first half: products of key half 0, with x = s * c2 - m and the
        // maxima (8 fused multiply-adds per row tile over the products)
        float x[kRT][8];
        constexpr int NP = kRT * DS;               // products per key half
        constexpr int FPC = 8 / DS;                // multiply-adds per chunk
        static_assert(NP <= 8 && 8 % NP == 0, "chunking");
#pragma unroll
        for (int i = 0; i < NP; ++i) {
            const int ds = i / kRT, rt = i % kRT;
            s_nxt[0][rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[0][ds], qB[rt][ds],
                                                                   s_nxt[0][rt], 0, 0, 0);
#pragma unroll
            for (int f = 0; f < FPC; ++f) {
                const int idx = i * FPC + f, r = idx / 8, j = idx % 8;
                x[r][j] = __builtin_fmaf(s_cur[j >> 2][r][j & 3], c2, -m[r]);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        bool over = false;
#pragma unroll
        for (int rt = 0; rt < kRT; ++rt) {
            const float mx = fmaxf(fmaxf(fmaxf(x[rt][0], x[rt][1]), fmaxf(x[rt][2], x[rt][3])),
                                   fmaxf(fmaxf(x[rt][4], x[rt][5]), fmaxf(x[rt][6], x[rt][7])));
            over |= mx > kTau;
        }

        if (__builtin_amdgcn_ballot_w64(over)) {
            // from the raw scores: x loses them while m is still kNoMax
#pragma unroll
            for (int rt = 0; rt < kRT; ++rt) {
                float r = fmaxf(fmaxf(fmaxf(s_cur[0][rt][0], s_cur[0][rt][1]),
                                      fmaxf(s_cur[0][rt][2], s_cur[0][rt][3])),
                                fmaxf(fmaxf(s_cur[1][rt][0], s_cur[1][rt][1]),
                                      fmaxf(s_cur[1][rt][2], s_cur[1][rt][3])));
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
                    x[rt][j] = __builtin_fmaf(s_cur[j >> 2][rt][j & 3], c2, -m_new);
            }
        }

        // the V^T operands of this sub-tile go out now and are waited for just
        // before the P V products; the K operands still to be used must have
        // arrived first, or the compiler's own waits for them (which know
        // nothing of these reads) would also wait for the V reads
#if defined(__HIP_DEVICE_COMPILE__)
#pragma unroll
        for (int ds = 0; ds < DS; ++ds) asm volatile("" ::"v"(ka[1][ds]));
#endif
        uint2 vr[DT][2];
        v_issue(vc, vr);

        // second half: products of key half 1 with row tile 0's weights
        // (p = 2^x packed to bf16, and the row sums); then the P V products
        // of each row tile with the next row tile's weights.  Every product
        // is paired with about one exponential, the vector work one
        // product's 16 matrix-core cycles hide.
        uint32_t pk[kRT][4];
        const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
        float e[kRT][8];
        auto weights = [&](int r, int k) {   // weight k of row tile r; a pair when k is odd
            e[r][k] = __builtin_amdgcn_exp2f(x[r][k]);
            if (k & 1) {
                pk[r][k / 2] = pack2(e[r][k - 1], e[r][k]);
                lsum[r] = __builtin_amdgcn_fdot2_f32_bf16(
                    __builtin_bit_cast(bf16x2, pk[r][k / 2]), ones, lsum[r], false);
            }
        };
        constexpr int EB = 8 / NP;                 // row tile 0 weights per product
#pragma unroll
        for (int i = 0; i < NP; ++i) {
            const int ds = i / kRT, rt = i % kRT;
            s_nxt[1][rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka[1][ds], qB[rt][ds],
                                                                   s_nxt[1][rt], 0, 0, 0);
#pragma unroll
            for (int f = 0; f < EB; ++f) weights(0, i * EB + f);
            __builtin_amdgcn_sched_barrier(0);
        }

        // O^T += V^T P^T (operands as laid out by v_issue)
        wait_vt(vr);
        bf16x8 va_op[DT];
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
            va_op[dt] = as_bf16x8(uint4{vr[dt][0].x, vr[dt][0].y, vr[dt][1].x, vr[dt][1].y});
        constexpr int EC = 8 / DT;                 // next row tile's weights per product
#pragma unroll
        for (int rt = 0; rt < kRT; ++rt) {
            const bf16x8 pb = as_bf16x8(uint4{pk[rt][0], pk[rt][1], pk[rt][2], pk[rt][3]});
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) {
                o[dt][rt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va_op[dt], pb, o[dt][rt], 0,
                                                                    0, 0);
                if (rt + 1 < kRT) {
#pragma unroll
                    for (int f = 0; f < EC; ++f) weights(rt + 1, dt * EC + f);
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
        }
    };

    // ---- software pipeline over this wave's 32-key sub-tiles.  A step turns
    // S of one sub-tile into P V while the matrix cores compute S of the
    // wave's next sub-tile (for the last, a discarded product over the
    // current stage).  With one key group a wave takes both halves of every
    // tile (the barrier that makes tile t+1 visible sits before the step of
    // half 1 of tile t); with two, group g takes half g of every tile (the
    // barrier sits before the step of tile t).  After the barrier, the stage
    // of tile t-1, last read before it, receives tile t+3.  The prologue
    // issues tiles 0..2 (1 and 2 after tile 0's barrier).
    auto stage_of = [&](int t) { return smem + Smem<D>::base + (t % kStages) * Smem<D>::stage; };
    constexpr std::integral_constant<int, 0> K0{};
    constexpr std::integral_constant<int, 1> K1{};

    // Fused re-encode of tile t, resident and visible in its stage, before
    // any product reads it: each cached key of a span is rotated by
    // R(delta) of the span, through the same routine and (cos, sin) values
    // as the re-encode launch, so the stage then holds the re-encoded cache's
    // bytes.  Item (block pair, lane): the K blocks of dims 32d.. and
    // 32d + D/2.. of one 16-key group hold a pair's two halves in the same
    // lane slot (key 16 sckt + lane % 16, dims 8 (lane / 16)..).  A
    // barrier ends it.  f_cur: the last span starting at or before the
    // tile's first key (tiles come in key order).
    int f_cur = 0;
    auto rotate_tile = [&](int t) {
        if constexpr (kFuse) {
            constexpr int PAIRS = KB / 2;
            const int* f_start = reinterpret_cast<const int*>(fsm + FuseSmem<D>::start);
            const int* f_end = reinterpret_cast<const int*>(fsm + FuseSmem<D>::end);
            const float2* f_cs = reinterpret_cast<const float2*>(fsm + FuseSmem<D>::cs);
            const int tb = kbeg + t * kTile;
            while (f_cur + 1 < f_n && f_start[f_cur + 1] <= tb) ++f_cur;
            if ((int)threadIdx.x < PAIRS * 64) {
                const int pi = threadIdx.x >> 6, ln = threadIdx.x & 63;
                const int sckt = pi / (DS / 2), dlo = pi % (DS / 2);
                unsigned char* st = stage_of(t);
                uint4* plo = reinterpret_cast<uint4*>(st + (sckt * DS + dlo) * 1024 + ln * 16);
                uint4* phi =
                    reinterpret_cast<uint4*>(st + (sckt * DS + dlo + DS / 2) * 1024 + ln * 16);
                const int v = tb + 16 * sckt + (ln & 15);
                int k = f_cur;
                while (k + 1 < f_n && f_start[k + 1] <= v) ++k;
                if (f_n > 0 && v < bk.cmax && v < kend && v >= f_start[k] && v < f_end[k]) {
                    const float2* row = f_cs + k * (D / 2) + 32 * dlo + 8 * (ln >> 4);
                    float c[8], sn[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        c[e] = row[e].x;
                        sn[e] = row[e].y;
                    }
                    uint4 x, y;
                    rope_rotate16<bf16_t>(*plo, *phi, c, sn, x, y);
                    *plo = x;
                    *phi = y;
                }
            }
            __syncthreads();
        }
    };

    wait_vm_all();
    __syncthreads();
    rotate_tile(0);

    // a step whose current and next sub-tiles are both dead for the wave is
    // skipped; a step that runs on a dead sub-tile's never-computed S masks
    // all of it
    const int h0 = kKG == 2 ? kg : 0;      // this wave's first half
    floatx4 s_a[2][kRT], s_b[2][kRT];
    if (!dead(kbeg + 32 * h0)) {
        qk_half(k_sub(stage_of(0), h0), K0, s_a);
        qk_half(k_sub(stage_of(0), h0), K1, s_a);
    }
    if (n_tiles > 1) issue_tile(1);
    if (n_tiles > 2) issue_tile(2);
    // tile t+1 resident and visible, and the stage of tile t-1 refilled
    auto next_tile_barrier = [&](int t) {
        // this wave's loads of tile t+1 are done when at most those of
        // tile t+2 are outstanding
        if (t + 2 < n_tiles) wait_vm<LPW>(); else wait_vm<0>();
        if constexpr (kFuse) __syncthreads();
        else barrier_keep_loads();
        if (t + 3 < n_tiles) issue_tile(t + 3);
        rotate_tile(t + 1);
    };
    if constexpr (kKG == 1) {
        const int n_sub = (kend - kbeg + 31) / 32;
        for (int t = 0; t < n_tiles; ++t) {
            const unsigned char* st = stage_of(t);
            const int v0 = kbeg + 64 * t;
            // half 0 of tile t -> half 1, same stage
            if (!(dead(v0) && dead(v0 + 32))) step(s_a, s_b, v0, v_sub(st, 0), k_sub(st, 1));
            if (2 * t + 1 >= n_sub) break;
            // half 1 of tile t -> half 0 of tile t+1, behind its barrier
            const bool more = t + 1 < n_tiles;
            if (more) next_tile_barrier(t);
            if (!(dead(v0 + 32) && dead(v0 + 64)))
                step(s_b, s_a, v0 + 32, v_sub(st, 1), k_sub(more ? stage_of(t + 1) : st, 0));
        }
    } else {
        // half kg of tile t -> half kg of tile t+1, behind its barrier (every
        // wave takes every barrier, whether or not its steps run)
        auto tile_step = [&](int t, floatx4 (&cur)[2][kRT], floatx4 (&nxt)[2][kRT]) {
            const bool more = t + 1 < n_tiles;
            if (more) next_tile_barrier(t);
            const int v0 = kbeg + 64 * t + 32 * kg;
            if (!(dead(v0) && dead(v0 + 64)))
                step(cur, nxt, v0, v_sub(stage_of(t), kg),
                     k_sub(stage_of(more ? t + 1 : t), kg));
        };
        for (int t = 0; t < n_tiles; t += 2) {
            tile_step(t, s_a, s_b);
            if (t + 1 >= n_tiles) break;
            tile_step(t + 1, s_b, s_a);
        }
    }

    // row sums: add the four lane groups that hold each row
#pragma unroll
    for (int rt = 0; rt < kRT; ++rt) {
        lsum[rt] += __shfl_xor(lsum[rt], 16);
        lsum[rt] += __shfl_xor(lsum[rt], 32);
    }

    // two key groups: group 1 hands its (m, l, O) of every row to group 0
    // through LDS (in the ring, free once every wave has left the loop);
    // lane (lg, lr) holds dims 16dt + 4lg.. of row 16rt + lr in both groups
    if constexpr (kKG == 2) {
        constexpr int OS = D + 4;                               // floats per row (bank skew)
        float* xo = reinterpret_cast<float*>(smem + Smem<D>::base) + rw * kRT * 16 * OS;
        float* xml = reinterpret_cast<float*>(smem + Smem<D>::base) + kRW * kRT * 16 * OS +
                     rw * kRT * 16 * 2;
        static_assert(kRW * kRT * 16 * (OS + 2) * 4 <= kStages * Smem<D>::stage, "merge area");
        __syncthreads();
        if (kg == 1) {
#pragma unroll
            for (int rt = 0; rt < kRT; ++rt) {
#pragma unroll
                for (int dt = 0; dt < DT; ++dt)
                    *reinterpret_cast<floatx4*>(xo + (16 * rt + lr) * OS + 16 * dt + 4 * lg) =
                        o[dt][rt];
                if (lg == 0) {
                    xml[(16 * rt + lr) * 2] = m[rt];
                    xml[(16 * rt + lr) * 2 + 1] = lsum[rt];
                }
            }
        }
        __syncthreads();
        if (kg == 0) {
#pragma unroll
            for (int rt = 0; rt < kRT; ++rt) {
                const float m1 = xml[(16 * rt + lr) * 2], l1 = xml[(16 * rt + lr) * 2 + 1];
                const float M = fmaxf(m[rt], m1);
                const float a0 = __builtin_amdgcn_exp2f(m[rt] - M);
                const float a1 = __builtin_amdgcn_exp2f(m1 - M);
                m[rt] = M;
                lsum[rt] = lsum[rt] * a0 + l1 * a1;
#pragma unroll
                for (int dt = 0; dt < DT; ++dt)
                    o[dt][rt] = o[dt][rt] * a0 +
                                *reinterpret_cast<const floatx4*>(
                                    xo + (16 * rt + lr) * OS + 16 * dt + 4 * lg) * a1;
            }
        }
    }

    // the waves of key group 0 write their rows: the output, or this
    // segment's partial (O / l in bf16, 0 for a row that saw no key of the
    // segment, with (m, l) in float; a unit's partials are row-major over its
    // segments, so the merge reads one contiguous run per row)
    if (kg == 0) {
#pragma unroll
        for (int rt = 0; rt < kRT; ++rt) {
            if (tok[rt] < 0) continue;
            const int rho = rho_w + 16 * rt + lr;
            const int64_t orow = (int64_t)(n0 + tok[rt]) * p.n_q_heads + h * G + rho % G;
            const float inv = lsum[rt] > 0.f ? 1.f / lsum[rt] : 0.f;
            if (direct) {
                bf16_t* dst = reinterpret_cast<bf16_t*>(p.out) + orow * D;
#pragma unroll
                for (int dt = 0; dt < DT; ++dt) {
                    const floatx4 v = o[dt][rt];
                    *reinterpret_cast<uint2*>(dst + 16 * dt + 4 * lg) =
                        uint2{pack2(v[0] * inv, v[1] * inv), pack2(v[2] * inv, v[3] * inv)};
                }
                if (lg == 0 && p.lse) p.lse[orow] = (m[rt] + log2f(lsum[rt])) * kLn2;
            } else {
                const int64_t pi = (int64_t)part * kRB + (int64_t)(rho - rho0) * nseg + seg_local;
                bf16_t* dst = reinterpret_cast<bf16_t*>(p.part_o) + pi * D;
                if (S::kMergeInLaunch && p.merge_in_launch) {
#pragma unroll
                    for (int dt = 0; dt < DT; ++dt) {
                        const floatx4 v = o[dt][rt];
                        store_agent(dst + 16 * dt + 4 * lg, pack2(v[0] * inv, v[1] * inv),
                                    pack2(v[2] * inv, v[3] * inv));
                    }
                    if (lg == 0)
                        store_agent(p.part_ml + pi * 2, __float_as_uint(m[rt]),
                                    __float_as_uint(lsum[rt]));
                } else {
#pragma unroll
                    for (int dt = 0; dt < DT; ++dt) {
                        const floatx4 v = o[dt][rt];
                        *reinterpret_cast<uint2*>(dst + 16 * dt + 4 * lg) =
                            uint2{pack2(v[0] * inv, v[1] * inv), pack2(v[2] * inv, v[3] * inv)};
                    }
                    if (lg == 0) {
                        p.part_ml[pi * 2] = m[rt];
                        p.part_ml[pi * 2 + 1] = lsum[rt];
                    }
                }
            }
        }
    }
    // This segment's share of the new values for the cache: the tokens whose
    // first row is in the unit's block, dealt over the unit's segments, so
    // the request's new values are written once per head (no tile of this
    // launch reads them back), stored with the partials
    constexpr int VC_TPR = D / 8;
    const int vc_t0 = (rho0 + G - 1) / G, vc_t1 = (rho_end - 1) / G + 1;
    const int vc_n = v_direct && vc_t1 - vc_t0 > seg_local
                         ? (vc_t1 - vc_t0 - seg_local + nseg - 1) / nseg * VC_TPR
                         : 0;
    auto vc_token = [&](int i) { return vc_t0 + seg_local + (i / VC_TPR) * nseg; };
    auto vc_src = [&](int i) {
        return reinterpret_cast<const uint4*>(
            reinterpret_cast<const bf16_t*>(p.v_new) +
            ((int64_t)(n0 + vc_token(i)) * p.n_kv_heads + h) * D + 8 * (i % VC_TPR));
    };
    for (int i = threadIdx.x; i < vc_n; i += 64 * kWaves) {
        const uint4 x = *vc_src(i);
        *reinterpret_cast<uint4*>(const_cast<char*>(vp.row(Tc + vc_token(i))) +
                                  16 * (i % VC_TPR)) = x;
    }
    // (256-row units always leave their partials to the combine launch: the
    // merge's registers would crowd the eight-wavefront loop)
    if constexpr (!S::kMergeInLaunch) return;
    if (direct || !p.merge_in_launch) return;

    // arrival: every partial store of the workgroup has completed (each wave
    // waits for its own, then the barrier), then one increment of the unit's
    // counter; it wraps to 0 when the last segment arrives, which merges
    wait_vm_all();
    __syncthreads();
    int* flag = reinterpret_cast<int*>(smem);     // below the ring
    if (threadIdx.x == 0) {
        const unsigned old = __builtin_amdgcn_atomic_inc32(p.counters + unit, (unsigned)(nseg - 1),
                                                           __ATOMIC_RELAXED, "agent");
        *flag = old == (unsigned)(nseg - 1);
    }
    __syncthreads();
    const bool last = *flag != 0;
    if (last) merge_unit<D, kRB, 64 * kWaves>(p, part, rows, nseg, h, rho0, n0);
}

// A persistent workgroup runs its chain of segments of the schedule: record
// blockIdx.x first, then the records its `next` fields name.
template <int D, class S, bool kFuse, bool kPaged>
__global__ __launch_bounds__(64 * kWaves, 1) void attend_mfma_kernel(KParams p) {
    __shared__ __attribute__((aligned(1024)))
    unsigned char smem[Smem<D>::bytes + (kFuse ? FuseSmem<D>::bytes : 0)];
    for (int g = blockIdx.x, first = 1; g >= 0 && g < p.n_segments; first = 0) {
        int4 rec[4];
        load_record(p, g, rec);
        if (!record_ok(p, rec, g)) break;
        // the previous segment's waves are done with every LDS stage
        if (!first) __syncthreads();
        attend_segment<D, S, kFuse, kPaged>(p, smem, rec);
        g = rec[3].y;
    }
}

template <int D, bool kFuse, bool kPaged>
void launch_dfp(const KParams& p, int n_wg, hipStream_t stream) {
    const dim3 grid(n_wg), block(64 * kWaves);
    if (p.row_block == Shape<2, 1>::kRB)
        hipLaunchKernelGGL((attend_mfma_kernel<D, Shape<2, 1>, kFuse, kPaged>), grid, block, 0,
                           stream, p);
    else if (p.row_block == Shape<2, 2>::kRB)
        hipLaunchKernelGGL((attend_mfma_kernel<D, Shape<2, 2>, kFuse, kPaged>), grid, block, 0,
                           stream, p);
    else
        hipLaunchKernelGGL((attend_mfma_kernel<D, Shape<1, 2>, kFuse, kPaged>), grid, block, 0,
                           stream, p);
}

template <int D>
void launch_d(const KParams& p, int n_wg, hipStream_t stream) {
    const bool paged = p.k.block_table || p.v.block_table;
    if (p.fuse_spans)
        paged ? launch_dfp<D, true, true>(p, n_wg, stream) : launch_dfp<D, true, false>(p, n_wg, stream);
    else
        paged ? launch_dfp<D, false, true>(p, n_wg, stream)
              : launch_dfp<D, false, false>(p, n_wg, stream);
}

}  // namespace

bool attend_mfma_row_block_ok(int row_block) {
    return row_block == Shape<2, 1>::kRB || row_block == Shape<2, 2>::kRB ||
           row_block == Shape<1, 2>::kRB;
}

hipError_t launch_attend_mfma(int head_dim, const KParams& p, int n_wg, hipStream_t stream) {
    if (!attend_mfma_row_block_ok(p.row_block)) return hipErrorInvalidValue;
    if (head_dim == 128)
        launch_d<128>(p, n_wg, stream);
    else
        launch_d<64>(p, n_wg, stream);
    return hipGetLastError();
}

}  // namespace attn
}  // namespace kvlink
