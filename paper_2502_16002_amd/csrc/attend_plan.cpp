// attend_plan.cpp — host-side schedule of the split-K attention.
//
// Work unit: (request s, KV head h, row block b).  The rows of request s for
// KV head h are its new tokens' query heads packed as row = token * group +
// head-in-group; block b holds rows [b * row_block, (b + 1) * row_block).  The
// unit's keys are the cached rows its last token sees (the attention map of
// Sec. 2.3: every position at or before the token's own) followed by the new
// rows up to that token; it walks them in 64-key tiles.
//
// A schedule gives every workgroup one or more segments (a contiguous tile
// range of one unit); a unit cut into several segments has its partial
// results merged by the combine.  Two ways of cutting are considered for
// each workgroup count n:
//
//   * unit-aligned: with n >= units, every workgroup gets one segment and
//     each unit k_u near-equal pieces, the k_u chosen greedily to minimise
//     the longest piece; with n < units, whole units are packed onto the
//     workgroups longest first;
//   * equal ranges: the tiles of all units, in order, cut into n contiguous
//     ranges of equal cost, crossing unit boundaries (perfect balance, but a
//     workgroup whose range crosses a boundary pays a second segment).
//
// Each cut is priced by a cost model fitted
// to MI355X timings of the Llama-8B-shaped workloads: a segment costs a
// fixed set-up (its record, the first key tiles and queries, the partial
// write); a tile costs its K/V stream plus the products of the (wavefront,
// step) pairs the kernel does not skip, more for steps that need the mask,
// plus, for the new rows among its keys, their RoPE and append (which the
// split launch does itself when the batch's RoPE table is given); the launch
// lasts as long as its longest workgroup; split units add the combine launch
// and the traffic of their partials.  Of the cuts priced within 2% of the
// cheapest, the one with the most workgroups is taken (the model leaves out
// costs that more workgroups do not shrink, and measured near ties favour
// filling the chip).
//
// Segment records are numbered so that record w is workgroup w's first
// segment; further segments of a workgroup follow the first n and are
// chained by the record's `next` field.  A workgroup therefore issues its
// first key-tile loads after one table read.  Unit records and the list of
// units with several segments drive the combine the same way.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdint>
#include <queue>
#include <vector>

#include "kvlink_internal.h"

namespace kvlink {
namespace {

constexpr int kTileKeys = 64;

struct Unit {
    int s, h, rho0, tiles, rows, n0, Tc, cmax, nvirt;
    std::vector<double> prefix;   // prefix[t]: cost of tiles [0, t), in us
    std::vector<float> live;      // live fraction of each tile
    double cost(int64_t t0, int64_t len) const { return prefix[t0 + len] - prefix[t0]; }
};

struct Seg {
    int w, u;
    int64_t t0, len;
};

struct CostModel {
    // a segment costs per_segment_us + first_us * (live fraction of its first
    // tile), plus split_us when its unit has several segments; a tile
    // tile_us + live_us * (live fraction) + mask_us * (masked fraction)
    double per_segment_us, first_us, tile_us, live_us, mask_us;
    double split_us;
    int slots_per_cu;
    // the RoPE and append of the new keys a segment reads (inside the split
    // launch), per 64 new rows
    double append_us;
    // split units merged in the launch (merge_bytes_per_us > 0): the slowest
    // last-arriving workgroup's merge follows, merge_us plus the unit's
    // partial bytes at merge_bytes_per_us; else by the combine launch:
    // combine_us plus all partial bytes, written and read, at
    // combine_bytes_per_us
    double merge_us, merge_bytes_per_us, combine_us, combine_bytes_per_us;
};

// Constants fitted to per-workgroup timelines (probe builds stamping each
// workgroup's phases with the 100 MHz real-time counter) of the Llama-8B
// workloads on MI355X.
//
// Wide kernel, 256-row units (fitted jointly on the 10- and 40-document
// workloads): a tile costs its stream of K and V (about 1.6 us at the share
// of HBM a workgroup gets while all stream) plus its products, which scale
// with the fraction of (wavefront, 32-key step) pairs that are live: a
// wavefront skips a step none of its rows sees (link tokens see only the
// documents before them), but the workgroup still streams the tile.  A live
// step that some row of the wavefront sees only in part (it runs the mask)
// costs about four times one seen whole.  A segment adds its record and, for
// its first tile, the products that wait for the tile's loads.  A segment
// whose keys include new rows first rotates and appends them, one round of
// loads and stores per 64 rows (about 0.9 us each).
//
// 128- and 64-row units: a segment's record and prologue (queries and the
// first tile) take about 5.1 and 3.6 us; a tile about 1.5 and 0.86 us, with
// little dependence on how many of its steps are live (a per-workgroup
// timeline fit over the 10-document workload: loop = 0.15 + 1.51 x tiles and
// 1.9 + 0.86 x tiles, residual sd 0.6 and 0.5 us).  A split segment merged in the launch adds its
// partial's coherent stores and the arrival (about 4.2 and 2.6 us; 3 us for
// 256 rows); the last arrival's merge reads the unit's partials at about
// 0.1 MB/us after 2 us.  Merged by the combine launch instead, a split
// segment's partial stores add about 1.5 us and the combine about 6 us plus
// the partial traffic at an effective ~6 TB/s.
//
// Decode kernel: one workgroup per compute unit (two would share its HBM
// stream and measured slower), a tile (64 keys of K and V) costing its bytes
// at a compute unit's share of ~6 TB/s, plus the start of a segment (its
// first loads' latency).  Split units: the combine launch costs about 3.4 us
// plus the partials' traffic; merged in the launch, a split segment's
// coherent stores and arrival add about 0.9 us and the last arrival's merge
// 1 us plus the unit's partials at ~0.013 MB/us (a 32-segment unit: 4.6 us in
// all, two segments: 2.1 us).  VALU kernel: fp32, a fixed cost per tile.
CostModel cost_model(AttendPath path, int head_dim, int row_block, bool in_launch) {
    const bool d128 = head_dim == 128;
    const double f = d128 ? 1.0 : 0.63;   // head_dim 64: fewer bytes and products per key
    CostModel cm;
    if (path == kPathWide) {
        if (row_block == 256)
            cm = {0.8, 3.67 * f, 1.61 * f, 0.65 * f, 1.97 * f, 0.0, 1, 0.9 * f, 0, 0, 0, 0};
        else if (row_block == 128)
            cm = {5.1, 0.0, 1.4 * f, 0.1 * f, 0.0, 0.0, 1, 0.9 * f, 0, 0, 0, 0};
        else
            cm = {3.6, 0.0, 0.8 * f, 0.06 * f, 0.0, 0.0, 1, 0.9 * f, 0, 0, 0, 0};
        if (in_launch) {
            cm.split_us = row_block == 256 ? 3.0 : row_block == 128 ? 4.2 : 2.6;
            cm.merge_us = 2.0;
            cm.merge_bytes_per_us = 1.0e5;
        } else {
            cm.split_us = row_block == 256 ? 0.0 : 1.5;
            cm.combine_us = 6.0;
            cm.combine_bytes_per_us = 6.0e6;
        }
        return cm;
    }
    if (path == kPathDecode) {
        if (in_launch)
            return {3.0, 0.0, d128 ? 2.8 : 1.5, 0.0, 0.0, 0.9, 1, 0.0, 1.0, 1.27e4, 0, 0};
        return {3.0, 0.0, d128 ? 2.8 : 1.5, 0.0, 0.0, 0.0, 1, 0.0, 0, 0, 3.4, 6.0e6};
    }
    return {4.0, 0.0, d128 ? 1.0 : 0.6, 0.0, 0.0, 0.0, d128 ? 2 : 4, 0.0, 0, 0, 4.0, 6.0e6};
}

// Live (wavefront, 32-key step) pairs of tile t of a wide-kernel unit, by the
// rule the kernel skips a step with.  The unit's rows are split over kRW row
// wavefronts of rpw rows (kRW * rpw = row block); with one key group a
// wavefront takes both 32-key halves of the tile and skips the step of half
// j when neither that half nor the next one it would compute is seen by any
// of its rows; with two, the wavefronts of group j take half j and the next
// half they compute is 64 keys on.  Returns the live pairs out of 2 * kRW;
// *masked counts the live ones whose half is not wholly below the
// wavefront's smallest visible prefix.
int live_pairs(const Unit& x, int t, int group, int row_block, const int32_t* new_visible,
               int* masked) {
    const int kg = row_block == 256 ? 1 : 2;
    const int rw_n = 8 / kg, rpw = row_block / rw_n;
    int cnt = 0;
    *masked = 0;
    for (int w = 0; w < rw_n; ++w) {
        const int rw = x.rho0 + rpw * w;
        if (rw >= x.rho0 + x.rows) continue;
        const int tok_max = (std::min(rw + rpw, x.rho0 + x.rows) - 1) / group;
        const int vis_max = new_visible[x.n0 + tok_max];
        const int vis_min = new_visible[x.n0 + rw / group];
        auto dead = [&](int64_t v0) {
            if (v0 >= x.nvirt) return true;
            const bool cached_seen = v0 < vis_max && v0 < x.cmax;
            const bool new_seen = v0 + 32 > x.cmax && std::max<int64_t>(v0, x.cmax) <= x.cmax + tok_max;
            return !cached_seen && !new_seen;
        };
        for (int j = 0; j < 2; ++j) {
            const int64_t v0 = (int64_t)kTileKeys * t + 32 * j;
            if (!(dead(v0) && dead(v0 + 32 * kg))) {
                ++cnt;
                if (v0 + 32 > vis_min) ++*masked;
            }
        }
    }
    return cnt;
}

// n contiguous ranges of equal cost over the units' tiles in order
void cut_equal_ranges(const std::vector<Unit>& units, int n, std::vector<Seg>* segs) {
    double W = 0.0;
    for (const Unit& x : units) W += x.prefix.back();
    size_t u = 0;
    int64_t t_in_u = 0;   // next tile of unit u to hand out
    double done = 0.0;    // cost handed out before tile t_in_u of unit u
    for (int w = 0; w < n; ++w) {
        const double end = w + 1 == n ? W : W * (w + 1) / n;
        while (u < units.size()) {
            const Unit& x = units[u];
            if (t_in_u >= x.tiles) {
                ++u;
                t_in_u = 0;
                continue;
            }
            if (done >= end - 1e-9 && w + 1 < n) break;
            // the tiles of unit u that start before `end`
            int64_t take = x.tiles - t_in_u;
            if (w + 1 < n) {
                const double target = x.prefix[t_in_u] + (end - done);
                const auto it = std::lower_bound(x.prefix.begin() + t_in_u + 1, x.prefix.end(),
                                                 target - 1e-9);
                take = std::min<int64_t>(take, (it - x.prefix.begin()) - t_in_u);
            }
            take = std::max<int64_t>(1, take);
            segs->push_back({w, (int)u, t_in_u, take});
            done += x.cost(t_in_u, take);
            t_in_u += take;
        }
    }
}

// [t0, t1) of unit x cut into k pieces of near-equal cost (piece i ends at the
// first tile boundary past i+1 k-ths of the cost, at least one tile each)
void cut_unit(const Unit& x, int k, std::vector<int64_t>* ends) {
    ends->clear();
    const double W = x.prefix.back();
    int64_t t = 0;
    for (int i = 0; i < k; ++i) {
        int64_t e = x.tiles;
        if (i + 1 < k) {
            const double target = W * (i + 1) / k;
            e = std::lower_bound(x.prefix.begin() + t + 1, x.prefix.end(), target - 1e-9) -
                x.prefix.begin();
            e = std::max<int64_t>(e, t + 1);
            e = std::min<int64_t>(e, x.tiles - (k - 1 - i));   // room for the pieces left
        }
        ends->push_back(e);
        t = e;
    }
}

// unit-aligned cut (see the file comment)
void cut_unit_aligned(const std::vector<Unit>& units, int n, std::vector<Seg>* segs) {
    const int nu = (int)units.size();
    if (n >= nu) {
        std::vector<int> k(nu, 1);
        std::vector<int64_t> ends;
        auto longest = [&](int u) {
            cut_unit(units[u], k[u], &ends);
            double m = 0.0;
            for (int i = 0, t = 0; i < k[u]; t = (int)ends[i], ++i)
                m = std::max(m, units[u].cost(t, ends[i] - t));
            return m;
        };
        std::priority_queue<std::pair<double, int>> pq;   // (longest piece, -unit)
        for (int u = 0; u < nu; ++u) pq.push({longest(u), -u});
        for (int extra = n - nu; extra > 0 && !pq.empty();) {
            const int u = -pq.top().second;
            pq.pop();
            if (k[u] >= units[u].tiles) continue;   // one tile per piece already
            ++k[u];
            --extra;
            pq.push({longest(u), -u});
        }
        int w = 0;
        for (int u = 0; u < nu; ++u) {
            cut_unit(units[u], k[u], &ends);
            for (int i = 0, t = 0; i < k[u]; t = (int)ends[i], ++i)
                segs->push_back({w++, u, t, ends[i] - t});
        }
        return;
    }
    // fewer workgroups than units: whole units, longest first onto the least
    // loaded workgroup
    std::vector<int> order(nu);
    for (int u = 0; u < nu; ++u) order[u] = u;
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) {
        return units[a].prefix.back() > units[b].prefix.back();
    });
    std::priority_queue<std::pair<double, int>> load;   // (-load, -workgroup)
    for (int w = 0; w < n; ++w) load.push({0.0, -w});
    std::vector<int> owner(nu);
    for (int u : order) {
        auto top = load.top();
        load.pop();
        owner[u] = -top.second;
        load.push({top.first - units[u].prefix.back(), top.second});
    }
    for (int u = 0; u < nu; ++u) segs->push_back({owner[u], u, 0, units[u].tiles});
}

// Renumbers the workgroups of a cut densely (a cut may leave some of the n
// workgroups without work: equal ranges narrower than a tile, or a unit that
// cannot be cut finer than one tile per piece) and returns their count.
int compact_workgroups(std::vector<Seg>* segs) {
    std::vector<int> id;
    for (Seg& g : *segs) {
        if (g.w >= (int)id.size()) id.resize(g.w + 1, -1);
    }
    int n = 0;
    for (const Seg& g : *segs)
        if (id[g.w] < 0) id[g.w] = n++;
    for (Seg& g : *segs) g.w = id[g.w];
    return n;
}

int used_workgroups(const std::vector<Seg>& segs) {
    int n = 0;
    for (const Seg& g : segs) n = std::max(n, g.w + 1);
    return n;
}

double estimate_us(const std::vector<Unit>& units, const std::vector<Seg>& segs,
                   const CostModel& cm, int head_dim, int elem) {
    std::vector<int> pieces(units.size(), 0);
    for (const Seg& g : segs) ++pieces[g.u];
    std::vector<double> wg(used_workgroups(segs), 0.0);
    for (const Seg& g : segs)
        wg[g.w] += cm.per_segment_us + cm.first_us * units[g.u].live[g.t0] +
                   units[g.u].cost(g.t0, g.len) + (pieces[g.u] > 1 ? cm.split_us : 0.0);
    double t = *std::max_element(wg.begin(), wg.end());
    const double row_bytes = head_dim * elem + 8.0;
    if (cm.merge_bytes_per_us > 0.0) {
        double merge = 0.0;
        for (size_t u = 0; u < units.size(); ++u)
            if (pieces[u] > 1)
                merge = std::max(merge, cm.merge_us + pieces[u] * units[u].rows * row_bytes /
                                                          cm.merge_bytes_per_us);
        return t + merge;
    }
    double bytes = 0.0;
    for (size_t u = 0; u < units.size(); ++u)
        if (pieces[u] > 1) bytes += 2.0 * pieces[u] * units[u].rows * row_bytes;   // write + read
    if (bytes > 0.0) t += cm.combine_us + bytes / cm.combine_bytes_per_us;
    return t;
}

// XCD-aware numbering: workgroup w of a launch runs on XCD w % kXcds on
// MI355X, and the XCDs have separate L2 caches.  Workgroups whose first
// segment belongs to the same (request, KV head) are given ids on one XCD
// where the ids allow, so that they share that KV head's keys and values and
// the unit's queries through one L2.
constexpr int kXcds = 8;
void number_by_xcd(const std::vector<Unit>& units, int n_kv_heads, std::vector<Seg>* segs) {
    const int n = used_workgroups(*segs);
    // the workgroup's first segment in (unit, tile) order decides
    std::vector<int> pref(n, 0);
    std::vector<int64_t> first_t(n, INT64_MAX);
    for (const Seg& g : *segs) {
        const int64_t key = (int64_t)g.u << 32 | g.t0;
        if (key < first_t[g.w]) {
            first_t[g.w] = key;
            pref[g.w] = (units[g.u].s * n_kv_heads + units[g.u].h) % kXcds;
        }
    }
    std::vector<std::vector<int>> free_ids(kXcds);
    for (int id = n - 1; id >= 0; --id) free_ids[id % kXcds].push_back(id);   // smallest last
    std::vector<int> new_id(n, -1), deferred;
    for (int w = 0; w < n; ++w) {
        auto& f = free_ids[pref[w]];
        if (!f.empty()) {
            new_id[w] = f.back();
            f.pop_back();
        } else {
            deferred.push_back(w);
        }
    }
    std::vector<int> rest;
    for (int x = 0; x < kXcds; ++x)
        for (int id : free_ids[x]) rest.push_back(id);
    std::sort(rest.begin(), rest.end());
    for (size_t i = 0; i < deferred.size(); ++i) new_id[deferred[i]] = rest[i];
    for (Seg& g : *segs) g.w = new_id[g.w];
}

}  // namespace

AttendPath attend_path(kvlink_dtype dt, int group, int max_new) {
    if (dt != KVLINK_BF16) return kPathValu;
    return (int64_t)group * max_new <= 16 ? kPathDecode : kPathWide;
}

int build_attend_schedule(kvlink_dtype dt, int n_q_heads, int n_kv_heads, int head_dim,
                          int n_seqs, const int32_t* seq_new_ptr, const int32_t* seq_cached,
                          const int32_t* new_visible, int n_compute_units, int n_workgroups,
                          int row_block, unsigned flags, std::vector<int32_t>* table,
                          PlanCounts* counts, const char** why) {
    const int group = n_q_heads / n_kv_heads;
    if (seq_new_ptr[0] != 0) {
        *why = "seq_new_ptr[0] must be 0";
        return KVLINK_ERR_LAYOUT;
    }
    int max_new = 0;
    for (int s = 0; s < n_seqs; ++s) {
        if (seq_new_ptr[s + 1] < seq_new_ptr[s]) {
            *why = "seq_new_ptr is not non-decreasing";
            return KVLINK_ERR_LAYOUT;
        }
        max_new = std::max(max_new, seq_new_ptr[s + 1] - seq_new_ptr[s]);
    }
    for (int n = 0; n < seq_new_ptr[n_seqs]; ++n)
        if (new_visible[n] < 0) {
            *why = "new_visible is negative";
            return KVLINK_ERR_LAYOUT;
        }
    for (int s = 0; s < n_seqs; ++s)
        if (seq_cached[s] < 0) {
            *why = "seq_cached is negative";
            return KVLINK_ERR_LAYOUT;
        }
    const AttendPath path = attend_path(dt, group, max_new);
    // row blocks to consider: the wide kernel's three unit shapes, or the
    // 16-row units of the decode and vector kernels
    std::vector<int> rbs;
    if (path == kPathWide) rbs = {256, 128, 64};
    else rbs = {16};
    if (row_block != 0) {
        if (!attend_row_block_ok(path, row_block)) {
            *why = "row_block is not one of this batch's kernel (wide: 256, 128, 64; else 16)";
            return KVLINK_ERR_UNSUPPORTED;
        }
        rbs = {row_block};
    }
    const int elem = dt == KVLINK_BF16 ? 2 : 4;
    // merge of split units: in the split launch (wide and decode kernels) or
    // by the combine launch; the flags may force one
    std::vector<bool> modes;
    if (path == kPathValu || (flags & KVLINK_PLAN_COMBINE)) modes = {false};
    else if (flags & KVLINK_PLAN_IN_LAUNCH) modes = {true};
    else modes = {true, false};
    if ((flags & KVLINK_PLAN_IN_LAUNCH) && row_block == 256) {
        *why = "256-row units merge by the combine launch only";
        return KVLINK_ERR_UNSUPPORTED;
    }

    std::vector<Unit> units;
    std::vector<Seg> segs;
    int rb = rbs[0];
    bool in_launch = false;
    double best_rb_est = 1e300;
    for (int cand_rb : rbs)
      for (bool mode : modes) {
        if (mode && cand_rb == 256) continue;   // 256-row units: combine launch only
        const CostModel cm = cost_model(path, head_dim, cand_rb, mode);
        std::vector<Unit> us;
        for (int s = 0; s < n_seqs; ++s) {
            const int n0 = seq_new_ptr[s];
            const int rows_s = (seq_new_ptr[s + 1] - n0) * group;
            for (int h = 0; h < n_kv_heads; ++h)
                for (int rho0 = 0; rho0 < rows_s; rho0 += cand_rb) {
                    const int rows = std::min(cand_rb, rows_s - rho0);
                    const int r_last = (rho0 + rows - 1) / group;
                    const int vis = new_visible[n0 + r_last];
                    const int64_t nvirt = (int64_t)vis + r_last + 1;
                    if (nvirt > INT32_MAX / 2) {
                        *why = "key range too long";
                        return KVLINK_ERR_LAYOUT;
                    }
                    us.push_back({s, h, rho0, (int)((nvirt + kTileKeys - 1) / kTileKeys), rows,
                                  n0, seq_cached[s], vis, (int)nvirt, {}});
                }
        }
        if ((int64_t)us.size() > kMaxUnits) continue;   // too many for the merge counters
        int64_t T = 0;
        for (const Unit& x : us) T += x.tiles;
        for (Unit& x : us) {
            x.prefix.assign((size_t)x.tiles + 1, 0.0);
            x.live.assign((size_t)x.tiles, 1.0f);
            const int pairs = path == kPathWide ? (cand_rb == 256 ? 16 : 8) : 16;
            for (int t = 0; t < x.tiles; ++t) {
                int masked = 0;
                const int live = path == kPathWide
                                     ? live_pairs(x, t, group, cand_rb, new_visible, &masked)
                                     : pairs;
                const double lf = (double)live / pairs, mf = (double)masked / pairs;
                x.live[t] = (float)lf;
                const int64_t new_rows =
                    std::max<int64_t>(0, std::min<int64_t>(x.nvirt, (int64_t)kTileKeys * (t + 1)) -
                                             std::max<int64_t>(x.cmax, (int64_t)kTileKeys * t));
                x.prefix[t + 1] = x.prefix[t] + cm.tile_us + cm.live_us * lf + cm.mask_us * mf +
                                  cm.append_us * new_rows / kTileKeys;
            }
        }

        std::vector<Seg> best_segs, cand;
        double best_est = 1e300;
        if (T > 0) {
            const int64_t max_n = std::min<int64_t>(T, (int64_t)cm.slots_per_cu * n_compute_units);
            // every cut's estimate, then the cut that keeps the most
            // workgroups busy among those within kNearTie of the best
            // estimate: the estimate leaves out the launch and prologue costs
            // that do not shrink with more workgroups, and measured near ties
            // favour filling every compute unit
            constexpr double kNearTie = 0.02;
            struct Est {
                double t;
                int c, way, used;
            };
            std::vector<Est> est;
            auto cut = [&](int c, int way) {
                cand.clear();
                if (way == 0) cut_unit_aligned(us, c, &cand);
                else cut_equal_ranges(us, c, &cand);
            };
            auto consider = [&](int c, bool any_cost) {
                for (int way = 0; way < 2; ++way) {
                    cut(c, way);
                    const int used = compact_workgroups(&cand);
                    // a forced count takes only cuts that use every workgroup
                    if (used < c && any_cost) continue;
                    est.push_back({estimate_us(us, cand, cm, head_dim, elem), c, way, used});
                }
            };
            if (n_workgroups > 0) {
                consider((int)std::min<int64_t>(n_workgroups, T), true);
            } else {
                for (int c = 1; c <= max_n; ++c) consider(c, false);
            }
            double best = 1e300;
            for (const Est& e : est) best = std::min(best, e.t);
            const Est* pick = nullptr;
            for (const Est& e : est)   // most workgroups, then lowest estimate, then unit-aligned
                if (e.t <= best * (1.0 + kNearTie) &&
                    (!pick || e.used > pick->used || (e.used == pick->used && e.t < pick->t)))
                    pick = &e;
            if (pick) {
                cut(pick->c, pick->way);
                compact_workgroups(&cand);
                best_segs = cand;
                best_est = pick->t;
            }
        } else {
            best_est = 0.0;
        }
        if (best_est < best_rb_est) {
            best_rb_est = best_est;
            rb = cand_rb;
            in_launch = mode;
            units = std::move(us);
            segs = std::move(best_segs);
        }
      }
    if (best_rb_est == 1e300) {
        *why = "more units than the merge counters hold";
        return KVLINK_ERR_UNSUPPORTED;
    }
    if ((flags & KVLINK_PLAN_XCD) && !segs.empty()) number_by_xcd(units, n_kv_heads, &segs);
    const int n = used_workgroups(segs);

    // segments per unit, in tile order, and the unit-order numbering used
    // for the partials and the combine
    const int n_seg = (int)segs.size();
    std::vector<std::vector<int>> of_unit(units.size());
    for (int i = 0; i < n_seg; ++i) of_unit[segs[i].u].push_back(i);
    std::vector<int32_t> unit_seg(units.size() + 1, 0);
    std::vector<int> local(n_seg);
    for (size_t u = 0; u < units.size(); ++u) {
        std::sort(of_unit[u].begin(), of_unit[u].end(),
                  [&](int a, int b) { return segs[a].t0 < segs[b].t0; });
        for (size_t j = 0; j < of_unit[u].size(); ++j) local[of_unit[u][j]] = (int)j;
        unit_seg[u + 1] = unit_seg[u] + (int32_t)of_unit[u].size();
    }
    // record ids: workgroup w's first segment is record w, the others follow
    // in order, chained by `next`
    std::vector<int> order(n_seg);
    for (int i = 0; i < n_seg; ++i) order[i] = i;
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return segs[a].w < segs[b].w; });
    std::vector<int> rec_id(n_seg), next(n_seg, -1), last(n, -1);
    int extra = n;
    for (int i : order) {
        const int w = segs[i].w;
        if (last[w] < 0) {
            rec_id[i] = w;
        } else {
            rec_id[i] = extra++;
            next[last[w]] = rec_id[i];
        }
        last[w] = i;
    }

    if (extra != n_seg) {   // every workgroup of a compacted cut has a segment
        *why = "internal error: schedule record numbering";
        return KVLINK_ERR_LAYOUT;
    }

    counts->n_wg = n;
    counts->n_units = (int)units.size();
    counts->n_segments = n_seg;
    counts->row_block = rb;
    counts->in_launch = in_launch;
    std::vector<int32_t> split;
    for (size_t u = 0; u < units.size(); ++u)
        if (unit_seg[u + 1] - unit_seg[u] > 1) split.push_back((int32_t)u);
    counts->n_split = (int)split.size();
    counts->table_len = (int64_t)kSegRecord * n_seg + (int64_t)kUnitRecord * units.size() +
                        (int64_t)split.size();
    if (table) {
        table->assign((size_t)counts->table_len, 0);
        int32_t* t = table->data();
        for (int i = 0; i < n_seg; ++i) {
            const Seg& g = segs[i];
            const Unit& x = units[g.u];
            int32_t* r = t + (int64_t)kSegRecord * rec_id[i];
            r[kSegS] = x.s;
            r[kSegH] = x.h;
            r[kSegRho0] = x.rho0;
            r[kSegRows] = x.rows;
            r[kSegTileA] = (int32_t)g.t0;
            r[kSegTileB] = (int32_t)(g.t0 + g.len);
            r[kSegNseg] = unit_seg[g.u + 1] - unit_seg[g.u];
            r[kSegLocal] = local[i];
            r[kSegN0] = x.n0;
            r[kSegTc] = x.Tc;
            r[kSegCmax] = x.cmax;
            r[kSegNvirt] = x.nvirt;
            r[kSegPart] = unit_seg[g.u];
            r[kSegNext] = next[i];
            r[kSegUnit] = g.u;
        }
        int32_t* ut = t + (int64_t)kSegRecord * n_seg;
        for (size_t u = 0; u < units.size(); ++u) {
            int32_t* r = ut + (int64_t)kUnitRecord * u;
            r[kUnitS] = units[u].s;
            r[kUnitH] = units[u].h;
            r[kUnitRho0] = units[u].rho0;
            r[kUnitRows] = units[u].rows;
            r[kUnitN0] = units[u].n0;
            r[kUnitSeg0] = unit_seg[u];
            r[kUnitNseg] = unit_seg[u + 1] - unit_seg[u];
        }
        std::copy(split.begin(), split.end(), ut + (int64_t)kUnitRecord * units.size());
    }
    return KVLINK_OK;
}

}  // namespace kvlink
