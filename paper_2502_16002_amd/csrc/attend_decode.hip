// attend_decode.hip — bf16 split-K attention for units of at most 16 GQA
// rows: the query heads of a decoding step (one to a few new tokens per
// request and KV head).  With so few rows each K/V byte feeds only a few
// flops, and the pass is bound by streaming the cache from HBM; the kernel is
// built to keep many independent loads in flight per compute unit.
//
// A unit (request, KV head, at most 16 rows token * group + head) walks its
// keys in 32-key steps.  The four wavefronts of a workgroup take the steps of
// a segment round-robin, each keeping its own online-softmax state for all 16
// rows, and merge their four states through LDS at the end; a wavefront
// streams K and V on its own, with no workgroup barrier inside the key loop:
//
//   * K is loaded with 16-byte global loads straight into registers (two
//     register sets, a step ahead), in matrix-core operand order: for
//     S^T = K Q^T lane l holds key l%16 and dims 8(l/16).. of a 32-dim step,
//     which is the A operand;
//   * V goes by 16-byte direct-to-LDS loads into the wavefront's own
//     two-stage LDS ring (row-major, 16-byte chunks XOR-swizzled by key) and
//     is read back with ds_read_b64_tr_b16 as the A operand of
//     O^T = V^T P^T, exactly as in the wide-block kernel;
//   * the products run on 16-row tiles, padding a unit's rows (4 for one
//     token of a group of 4) with zero queries: the matrix cores have ample
//     slack here, and a padded 16x16x32 product takes far fewer issue cycles
//     than the same contraction as vector dot products.
//
// Scores, masks and the lazily raised running maximum follow the wide-block
// kernel: P = 2^(S * scale * log2e - m), with m raised only when a score
// exceeds it by more than 2^kTau.
#include <type_traits>

#include "attend_common.h"
#include "merge_launch.h"
#include "mfma_ops.h"

namespace kvlink {
namespace attn {
namespace {

constexpr int kDW = 4;       // wavefronts per workgroup
constexpr int kDR = 16;      // GQA rows per unit
constexpr int kStep = 32;    // keys per wavefront step
constexpr int kTile = 64;    // keys per schedule tile
constexpr float kTau = 8.0f;

// LDS: the (m, l) pairs of every wave and row for the merge, then each
// wave's area: two V stages, reused for its O in the merge.  Direct-to-LDS
// loads need a non-zero LDS address, which the (m, l) block in front gives.
template <int D>
struct DecodeSmem {
    static constexpr int v_bytes = kStep * D * 2;          // V of one step
    static constexpr int o_stride = D + 4;                 // floats per merge row (bank skew)
    static constexpr int o_bytes = kDR * o_stride * 4;     // one wave's O for the merge
    static constexpr int wave = 2 * v_bytes;
    static_assert(o_bytes <= wave, "merge area inside the wave's stages");
    static constexpr int ml = 0;
    static constexpr int flag = 1020;                      // the last-arrival flag
    static constexpr int base = 1024;
    static_assert(kDW * kDR * 2 * 4 <= flag, "(m, l) block");
    static constexpr int bytes = base + kDW * wave;
};

// K operands of one step (key half kh, 32-dim step ds).
template <int D>
struct StepRegs {
    uint4 k[2][D / 32];
};

// 16 bytes of K into registers, with the cache policy kPolicy.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
template <int kPolicy>
__device__ __forceinline__ uint4 load16(const char* p) {
    if constexpr (kPolicy == kStream) {
        const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
        return uint4{v[0], v[1], v[2], v[3]};
    } else {
        return *reinterpret_cast<const uint4*>(p);
    }
}

// One segment: tiles [tile_a, tile_b) of the keys of KV head h for rows
// [rho0, rho0 + rows) of request s, each wavefront taking every kDW-th
// 32-key step.  A split unit's segment stores its partial, either for the
// combine launch or, merged in this launch, with agent-coherent stores
// followed by its arrival on the unit's counter; the last arrival merges the
// unit's partials.  Every early return is uniform over the workgroup.
template <int D, int kPolK, int kPolV>
__device__ __forceinline__ void decode_segment(const KParams& p, unsigned char* smem,
                                               const int4 (&rec)[4]) {
    constexpr int DS = D / 32;         // 32-dim steps of S^T
    constexpr int DT = D / 16;         // 16-dim tiles of O^T
    constexpr int CH = D / 8;          // 16-byte chunks per row
    constexpr int VL = D / 16;         // 1 KB V loads per step
    static_assert(VL * 1024 == kStep * D * 2, "V step split");
    static_assert(64 / CH <= 16, "a V load stays inside one 16-key group");

    const int s = rec[0].x, h = rec[0].y, rho0 = rec[0].z, rows = rec[0].w;
    const int tile_a = rec[1].x, tile_b = rec[1].y;
    const int nseg = rec[1].z, seg_local = rec[1].w, part = rec[3].x, unit = rec[3].z;
    const bool direct = nseg == 1;
    const bool in_launch = !direct && p.merge_in_launch;
    const int n0 = rec[2].x, Tc = rec[2].y, cmax = rec[2].z, nvirt = rec[2].w;
    const int G = p.group;
    const int kbeg = tile_a * kTile;
    // (a split segment merged in the launch must still arrive)
    if (kbeg >= nvirt && !in_launch) return;
    const int kend = min(tile_b * kTile, nvirt);

    constexpr int LPS = 2 * DS + VL;   // loads per step
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    const int lr = lane & 15, lg = lane >> 4;
    unsigned char* vs = smem + DecodeSmem<D>::base + wave * DecodeSmem<D>::wave;

    // the wavefront's steps, as key offsets v0 (-1: none left)
    int stat_t = wave;
    auto next_step = [&]() -> int {
        const int v0 = kbeg + stat_t * kStep;
        stat_t += kDW;
        return v0 < kend ? v0 : -1;
    };

    // (the policies follow the views: a streamed view is contiguous, and its
    // null table folds the paged branches away)
    RowPtr kp = row_ptr<bf16_t>(p.k, p.layer, h, s);
    RowPtr vp = row_ptr<bf16_t>(p.v, p.layer, h, s);
    if constexpr (kPolK == kStream) kp.table = nullptr;
    if constexpr (kPolV == kStream) vp.table = nullptr;
    // below fast_end keys are cached rows taken by 16-row groups (one page
    // each when paged): a load's address is its group's first row (the same
    // in every lane; the step's first row when contiguous) plus a 32-bit
    // lane offset fixed for the segment; elsewhere each lane maps its key on
    // its own
    const bool grouped = kp.groups_of_16() && vp.groups_of_16() &&
                         kp.row_bytes < (1 << 24) && vp.row_bytes < (1 << 24);
    const int fast_end = grouped ? min(kend, cmax) : 0;
    auto key_row = [&](int v) {
        v = min(v, kend - 1);
        return v < cmax ? v : Tc + (v - cmax);
    };

    // V load i of a step fills LDS slot 64i + lane of the stage: key
    // (64i + lane) / CH, slot chunk lane % CH, which holds the row's logical
    // chunk (lane % CH) ^ (key % CH)
    auto v_key = [&](int i) { return (64 * i + lane) / CH; };
    auto v_off = [&](int i) { return 16 * ((lane % CH) ^ (v_key(i) & (CH - 1))); };
    const uint32_t k_lane = (uint32_t)(lr * kp.row_bytes + 16 * lg);
    uint32_t v_lane[VL];
#pragma unroll
    for (int i = 0; i < VL; ++i) v_lane[i] = (uint32_t)((v_key(i) & 15) * vp.row_bytes + v_off(i));

    // Loads of the step at v0: K into r, then V into LDS stage st, with the
    // cache policies the launch chose for the two views.
    auto issue_k_as = [&](int v0, StepRegs<D>& r, auto policy) {
        constexpr int pol = decltype(policy)::value;
        if (kPolK == kStream && v0 + kStep <= fast_end) {
            const char* b = kp.base + (int64_t)v0 * kp.row_bytes;
#pragma unroll
            for (int kh = 0; kh < 2; ++kh) {
                const char* g = b + (k_lane + (uint32_t)(16 * kh * kp.row_bytes));
#pragma unroll
                for (int ds = 0; ds < DS; ++ds) r.k[kh][ds] = load16<pol>(g + 64 * ds);
            }
        } else if (v0 + kStep <= fast_end) {
            int pg[2] = {0, 0};
            if (kp.table) {
                pg[0] = kp.page_of(v0);
                pg[1] = kp.page_of(v0 + 16);
            }
#pragma unroll
            for (int kh = 0; kh < 2; ++kh) {
                const char* g = kp.in_page(pg[kh], v0 + 16 * kh) + k_lane;
#pragma unroll
                for (int ds = 0; ds < DS; ++ds) r.k[kh][ds] = load16<pol>(g + 64 * ds);
            }
        } else {
#pragma unroll
            for (int kh = 0; kh < 2; ++kh) {
                const char* g = kp.row(key_row(v0 + 16 * kh + lr)) + 16 * lg;
#pragma unroll
                for (int ds = 0; ds < DS; ++ds) r.k[kh][ds] = load16<pol>(g + 64 * ds);
            }
        }
    };
    auto issue_v_as = [&](int v0, unsigned char* st, auto policy) {
        constexpr int pol = decltype(policy)::value;
        if (kPolV == kStream && v0 + kStep <= fast_end) {
            const char* b = vp.base + (int64_t)v0 * vp.row_bytes;
#pragma unroll
            for (int i = 0; i < VL; ++i) {
                const int kh = (64 * i / CH) >> 4;          // the load's 16-key group
                load_lds16<pol>(b + (v_lane[i] + (uint32_t)(16 * kh * vp.row_bytes)), st + i * 1024);
            }
        } else if (v0 + kStep <= fast_end) {
            int pg[2] = {0, 0};
            if (vp.table) {
                pg[0] = vp.page_of(v0);
                pg[1] = vp.page_of(v0 + 16);
            }
#pragma unroll
            for (int i = 0; i < VL; ++i) {
                const int kh = (64 * i / CH) >> 4;          // the load's 16-key group
                load_lds16<pol>(vp.in_page(pg[kh], v0 + 16 * kh) + v_lane[i], st + i * 1024);
            }
        } else {
#pragma unroll
            for (int i = 0; i < VL; ++i)
                load_lds16<pol>(vp.row(key_row(v0 + v_key(i))) + v_off(i), st + i * 1024);
        }
    };
    constexpr std::integral_constant<int, kPolK> pol_k{};
    constexpr std::integral_constant<int, kPolV> pol_v{};
    auto issue_k = [&](int v0, StepRegs<D>& r) { issue_k_as(v0, r, pol_k); };
    auto issue_v = [&](int v0, unsigned char* st) { issue_v_as(v0, st, pol_v); };
    auto stage = [&](int parity) { return vs + parity * DecodeSmem<D>::v_bytes; };

    // rows of the unit: lane row lr (padding rows past `rows` see no key)
    const int rho = rho0 + lr;
    const bool row_ok = lr < rows;
    const int tok = row_ok ? rho / G : 0;
    const int vis = p.new_visible[n0 + tok];
    const int lo = row_ok ? min(vis, kend) : 0;              // cached keys v < lo
    const int hi = row_ok ? min(cmax + tok, kend - 1) : -1;  // new keys cmax <= v <= hi
    const int tok_max = (rho0 + max(rows, 1) - 1) / G;
    const int vis_min = p.new_visible[n0 + rho0 / G];
    const int vis_max = p.new_visible[n0 + tok_max];
    // a step no row sees (only possible at a unit's ends)
    auto dead = [&](int v0) {
        const bool cached_seen = v0 < vis_max && v0 < cmax;
        const bool new_seen = v0 + kStep > cmax && max(v0, cmax) <= cmax + tok_max;
        return !cached_seen && !new_seen;
    };

    // With the fused RoPE, the new rows among the segment's keys ([na, nb)
    // of the request's new tokens) are appended to the cache, the stores
    // waited for and the workgroup synchronised before any load that may
    // read them: ahead of the prologue's loads when those reach the new
    // rows, else right after them (the key loop has no barrier of its own).
    const int na = max(kbeg, cmax) - cmax, nb = kend - cmax;
    const bool has_new = p.rope != nullptr && nb > na;
    const bool early_new = has_new && kbeg + 2 * kDW * kStep > cmax;
    if (early_new) {
        append_new_rows<D, 64 * kDW>(p, kp, vp, h, n0, Tc, na, nb);
        wait_vm_all();
        __syncthreads();
    }

    StepRegs<D> R0, R1;
    int va = next_step();
    if (va >= 0) {
        issue_k(va, R0);
        issue_v(va, stage(0));
    }
    // queries, B operand of S^T: row lr, dims 32ds + 8lg
    // (their rotation, with the fused RoPE, after the next step's loads
    // are issued)
    QRow<D> qrow;
    qrow.load(p, n0 + tok, h * G + rho % G, lg);
    int vb = va >= 0 ? next_step() : -1;
    if (vb >= 0) {
        issue_k(vb, R1);
        issue_v(vb, stage(1));
    }
    bf16x8 qB[DS];
    {
        uint4 q[DS];
        qrow.get(p, q);
#pragma unroll
        for (int ds = 0; ds < DS; ++ds) qB[ds] = as_bf16x8(row_ok ? q[ds] : uint4{0u, 0u, 0u, 0u});
    }
    if (has_new && !early_new) {
        append_new_rows<D, 64 * kDW>(p, kp, vp, h, n0, Tc, na, nb);
        wait_vm_all();
        __syncthreads();
    }

    const float c2 = p.scale_log2;
    floatx4 o[DT];
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
    float m = kNoMax, lsum = 0.f;

    // transposed-read addresses of the V^T operand in stage 0 (see the
    // wide-block kernel): lane (lg, lr) reads key 4lg + lr/4, chunk
    // 2dt + (lr/2)%2, half lr%2; the keys 16.. of the step sit 16 rows
    // further, stage 1 v_bytes further
    uint32_t va_lds[DT];
    {
        const uint32_t base = lds_addr(vs);
        const int key = 4 * lg + (lr >> 2);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
            const int c = 2 * dt + ((lr >> 1) & 1);
            va_lds[dt] = base + key * (2 * D) + 16 * (c ^ (key & (CH - 1))) + 8 * (lr & 1);
        }
    }

    // the step at v0 from registers r and LDS stage `parity`; `more`: the
    // wavefront's following step is in flight behind it.  The loads of the
    // step after that go into r once K has fed the products and into the
    // stage once its V has been read; returns its v0 (-1: none).
    auto run_step = [&](int v0, StepRegs<D>& r, auto parity, bool more) -> int {
        constexpr int par = decltype(parity)::value;
        // this step's loads are done when at most the next step's are
        // outstanding
        if (more) wait_vm<LPS>(); else wait_vm<0>();
        const int v_next = next_step();
        const bool live = !dead(v0);
        floatx4 sacc[2];
        if (live) {
#pragma unroll
            for (int kh = 0; kh < 2; ++kh) {
                sacc[kh] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ds = 0; ds < DS; ++ds)
                    sacc[kh] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(r.k[kh][ds]),
                                                                       qB[ds], sacc[kh], 0, 0, 0);
            }
        }
        const bool next_ok = v_next >= 0;
        if (next_ok) issue_k(v_next, r);
        if (!live) {
            if (next_ok) issue_v(v_next, stage(par));
            return v_next;
        }

        // mask: lane group lg holds keys 16kh + 4lg + i of the step
        const int vb4 = v0 + 4 * lg;
        if (v0 + kStep > vis_min || v0 + kStep > cmax) {
#pragma unroll
            for (int kh = 0; kh < 2; ++kh)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int v = vb4 + 16 * kh + i;
                    const bool ok = v < lo || (v >= cmax && v <= hi);
                    sacc[kh][i] = ok ? sacc[kh][i] : -INFINITY;
                }
        }
        float x[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) x[t] = __builtin_fmaf(sacc[t >> 2][t & 3], c2, -m);
        float mx = x[0];
#pragma unroll
        for (int t = 1; t < 8; ++t) mx = fmaxf(mx, x[t]);
        if (__builtin_amdgcn_ballot_w64(mx > kTau)) {
            // from the raw scores: x loses them while m is still kNoMax
            float rm = sacc[0][0];
#pragma unroll
            for (int t = 1; t < 8; ++t) rm = fmaxf(rm, sacc[t >> 2][t & 3]);
            rm = fmaxf(rm, __shfl_xor(rm, 16));
            rm = fmaxf(rm, __shfl_xor(rm, 32));
            const float m_new = fmaxf(m, rm * c2);
            const float alpha = __builtin_amdgcn_exp2f(m - m_new);
            m = m_new;
            lsum *= alpha;
#pragma unroll
            for (int dt = 0; dt < DT; ++dt) o[dt] *= alpha;
#pragma unroll
            for (int t = 0; t < 8; ++t) x[t] = __builtin_fmaf(sacc[t >> 2][t & 3], c2, -m);
        }
        uint32_t pk[4];
        const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            pk[t] = pack2(__builtin_amdgcn_exp2f(x[2 * t]), __builtin_amdgcn_exp2f(x[2 * t + 1]));
            lsum = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, pk[t]), ones, lsum,
                                                   false);
        }
        // O^T += V^T P^T; the stage is free for the next step once the reads
        // have returned
        uint2 vr[DT][2];
        issue_vt<DT, par * DecodeSmem<D>::v_bytes, par * DecodeSmem<D>::v_bytes + 16 * 2 * D>(va_lds,
                                                                                              vr);
        wait_vt(vr);
        if (next_ok) issue_v(v_next, stage(par));
        const bf16x8 b = as_bf16x8(uint4{pk[0], pk[1], pk[2], pk[3]});
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) {
            const bf16x8 a = as_bf16x8(uint4{vr[dt][0].x, vr[dt][0].y, vr[dt][1].x, vr[dt][1].y});
            o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, o[dt], 0, 0, 0);
        }
        return v_next;
    };

    constexpr std::integral_constant<int, 0> P0{};
    constexpr std::integral_constant<int, 1> P1{};
    while (va >= 0) {
        va = run_step(va, R0, P0, vb >= 0);
        if (vb < 0) break;
        vb = run_step(vb, R1, P1, va >= 0);
    }

    // this wave's state: row sums over the four lane groups, then O, m and l
    // into LDS for the merge
    lsum += __shfl_xor(lsum, 16);
    lsum += __shfl_xor(lsum, 32);
    {
        float* ow = reinterpret_cast<float*>(vs);
#pragma unroll
        for (int dt = 0; dt < DT; ++dt)
            *reinterpret_cast<floatx4*>(ow + lr * DecodeSmem<D>::o_stride + 16 * dt + 4 * lg) = o[dt];
        float* ml = reinterpret_cast<float*>(smem + DecodeSmem<D>::ml);
        if (lg == 0) {
            ml[(wave * kDR + lr) * 2] = m;
            ml[(wave * kDR + lr) * 2 + 1] = lsum;
        }
    }
    __syncthreads();

    // merge: thread (row r, four dims at 4c) weighs each wave's state by
    // 2^(m_w - M); a wave that saw no key of the row has l_w = 0 and O_w = 0
    const float* ml = reinterpret_cast<const float*>(smem + DecodeSmem<D>::ml);
    for (int idx = threadIdx.x; idx < rows * (D / 4); idx += 64 * kDW) {
        const int r = idx / (D / 4), c = idx % (D / 4);
        float M = kNoMax;
#pragma unroll
        for (int w = 0; w < kDW; ++w) M = fmaxf(M, ml[(w * kDR + r) * 2]);
        float L = 0.f;
        floatx4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int w = 0; w < kDW; ++w) {
            const float a = __builtin_amdgcn_exp2f(ml[(w * kDR + r) * 2] - M);
            L += a * ml[(w * kDR + r) * 2 + 1];
            const float* ow = reinterpret_cast<const float*>(smem + DecodeSmem<D>::base +
                                                             w * DecodeSmem<D>::wave);
            acc += a * *reinterpret_cast<const floatx4*>(ow + r * DecodeSmem<D>::o_stride + 4 * c);
        }
        const int rr = rho0 + r;
        const int64_t orow = (int64_t)(n0 + rr / G) * p.n_q_heads + h * G + rr % G;
        // the output, or this segment's partial: O / l in bf16 (0 for a row
        // that saw no key of the segment) with (m, l) in float, row-major over
        // the unit's segments; stored coherently when merged in this launch
        const float inv = L > 0.f ? 1.f / L : 0.f;
        const uint32_t o01 = pack2(acc[0] * inv, acc[1] * inv);
        const uint32_t o23 = pack2(acc[2] * inv, acc[3] * inv);
        const int64_t pi = (int64_t)part * kDR + (int64_t)r * nseg + seg_local;
        if (direct) {
            *reinterpret_cast<uint2*>(reinterpret_cast<bf16_t*>(p.out) + orow * D + 4 * c) =
                uint2{o01, o23};
            if (c == 0 && p.lse) p.lse[orow] = (M + log2f(L)) * kLn2;
        } else if (in_launch) {
            store_agent(reinterpret_cast<bf16_t*>(p.part_o) + pi * D + 4 * c, o01, o23);
            if (c == 0) store_agent(p.part_ml + pi * 2, __float_as_uint(M), __float_as_uint(L));
        } else {
            *reinterpret_cast<uint2*>(reinterpret_cast<bf16_t*>(p.part_o) + pi * D + 4 * c) =
                uint2{o01, o23};
            if (c == 0) {
                p.part_ml[pi * 2] = M;
                p.part_ml[pi * 2 + 1] = L;
            }
        }
    }
    if (!in_launch) return;

    // arrival: every partial store of the workgroup has completed (each wave
    // waits for its own, then the barrier), then one increment of the unit's
    // arrival counter, which wraps to 0 on the last arrival, which merges
    wait_vm_all();
    __syncthreads();
    int* flag = reinterpret_cast<int*>(smem + DecodeSmem<D>::flag);
    if (threadIdx.x == 0) {
        const unsigned old = __builtin_amdgcn_atomic_inc32(p.counters + unit, (unsigned)(nseg - 1),
                                                           __ATOMIC_RELAXED, "agent");
        *flag = old == (unsigned)(nseg - 1);
    }
    __syncthreads();
    if (*flag) merge_unit<D, kDR, 64 * kDW>(p, part, rows, nseg, h, rho0, n0);
}

// A persistent workgroup runs its chain of segments: record blockIdx.x
// first, then the records its `next` fields name.  kPolK and kPolV are the
// cache policies of the K and V loads: a contiguous cache is streamed
// (non-temporal: each byte is read once per call), a paged one is read
// through the caches, since its pages may be shared between requests (the
// values of a shared document pool).
template <int D, int kPolK, int kPolV>
__global__ __launch_bounds__(64 * kDW, 1) void attend_decode_kernel(KParams p) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[DecodeSmem<D>::bytes];
    for (int g = blockIdx.x, first = 1; g >= 0 && g < p.n_segments; first = 0) {
        int4 rec[4];
        load_record(p, g, rec);
        if (!record_ok(p, rec, g)) break;
        // the previous segment's merge is done with every wave's LDS area
        if (!first) __syncthreads();
        decode_segment<D, kPolK, kPolV>(p, smem, rec);
        g = rec[3].y;
    }
}

}  // namespace

int attend_decode_row_block() { return kDR; }

namespace {
template <int D>
void launch_decode_d(const KParams& p, int n_wg, hipStream_t stream) {
    const dim3 grid(n_wg), block(64 * kDW);
    const bool pk = p.k.block_table != nullptr, pv = p.v.block_table != nullptr;
    if (pk && pv)
        hipLaunchKernelGGL((attend_decode_kernel<D, kCached, kCached>), grid, block, 0, stream, p);
    else if (pk)
        hipLaunchKernelGGL((attend_decode_kernel<D, kCached, kStream>), grid, block, 0, stream, p);
    else if (pv)
        hipLaunchKernelGGL((attend_decode_kernel<D, kStream, kCached>), grid, block, 0, stream, p);
    else
        hipLaunchKernelGGL((attend_decode_kernel<D, kStream, kStream>), grid, block, 0, stream, p);
}
}  // namespace

hipError_t launch_attend_decode(int head_dim, const KParams& p, int n_wg, hipStream_t stream) {
    if (head_dim == 128)
        launch_decode_d<128>(p, n_wg, stream);
    else
        launch_decode_d<64>(p, n_wg, stream);
    return hipGetLastError();
}

}  // namespace attn
}  // namespace kvlink
