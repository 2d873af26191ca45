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
    // tile); a tile tile_us + live_us * (live fraction) + mask_us * (masked
    // fraction)
    double per_segment_us, first_us, tile_us, live_us, mask_us, combine_us, combine_bytes_per_us;
    int slots_per_cu;
    // the RoPE and append of the new keys a segment reads (inside the split
    // launch), per 64 new rows
    double append_us;
};

// Wide-block kernel: fitted jointly to per-workgroup timelines of the 10-
// and 40-document workloads.  A tile costs its stream of K and V (about
// 1.6 us at the share of HBM a workgroup gets while all stream) plus its
// products, which scale with the fraction of (wavefront, 32-key step) pairs
// that are live: a wavefront skips a step none of its rows sees (link tokens
// see only the documents before them), but the workgroup still streams the
// tile.  A live step that some row of the wavefront sees only in part (it
// runs the mask) costs about four times one seen whole.  A segment adds its
// record and, for its first tile, the products that wait for the tile's
// loads instead of overlapping them.  A segment whose keys include new rows
// first rotates and appends them, one round of loads and stores per 64 rows
// (about 0.9 us each).  The combine costs about 6 us plus its partial
// traffic, written and read back at an effective ~6 TB/s.  Decode kernel: two
// workgroups per compute unit sharing the unit's HBM stream, so a tile (64
// keys of K and V) costs its bytes at an eighth of a compute unit's share of
// ~6 TB/s, plus the start of a segment (its first loads' latency).  VALU
// kernel: fp32, a fixed cost per tile.
CostModel cost_model(AttendPath path, int head_dim) {
    const bool d128 = head_dim == 128;
    const double f = d128 ? 1.0 : 0.63;   // head_dim 64: fewer bytes and products per key
    if (path == kPathWide)
        return {0.8, 3.67 * f, 1.61 * f, 0.65 * f, 1.97 * f, 6.0, 6.0e6, 1, 0.9 * f};
    if (path == kPathDecode) return {3.0, 0.0, d128 ? 2.8 : 1.5, 0.0, 0.0, 6.0, 6.0e6, 2, 0.0};
    return {4.0, 0.0, d128 ? 1.0 : 0.6, 0.0, 0.0, 4.0, 6.0e6, d128 ? 2 : 4, 0.0};
}

// Live (wavefront, 32-key step) pairs of tile t of a wide-kernel unit, by the
// rule the kernel skips a step with: step j of wavefront w is dead when none
// of the wavefront's rows sees a key of sub-tiles j or j+1 (32 rows per
// wavefront, eight wavefronts); *masked counts the live pairs whose
// sub-tile is not wholly below the wavefront's smallest visible prefix.
int live_pairs(const Unit& x, int t, int group, const int32_t* new_visible, int* masked) {
    int cnt = 0;
    *masked = 0;
    for (int w = 0; w < 8; ++w) {
        const int rw = x.rho0 + 32 * w;
        if (rw >= x.rho0 + x.rows) continue;
        const int tok_max = (std::min(rw + 32, x.rho0 + x.rows) - 1) / group;
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
            if (!(dead(v0) && dead(v0 + 32))) {
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
    std::vector<double> wg(used_workgroups(segs), 0.0);
    std::vector<int> pieces(units.size(), 0);
    for (const Seg& g : segs) {
        wg[g.w] += cm.per_segment_us + cm.first_us * units[g.u].live[g.t0] +
                   units[g.u].cost(g.t0, g.len);
        ++pieces[g.u];
    }
    double t = *std::max_element(wg.begin(), wg.end());
    double bytes = 0.0;
    for (size_t u = 0; u < units.size(); ++u)
        if (pieces[u] > 1)
            bytes += 2.0 * pieces[u] * units[u].rows * (head_dim * elem + 8.0);   // write + read
    if (bytes > 0.0) t += cm.combine_us + bytes / cm.combine_bytes_per_us;
    return t;
}

}  // namespace

AttendPath attend_path(kvlink_dtype dt, int group, int max_new) {
    if (dt != KVLINK_BF16) return kPathValu;
    return (int64_t)group * max_new <= attend_row_block(kPathDecode) ? kPathDecode : kPathWide;
}

int build_attend_schedule(kvlink_dtype dt, int n_q_heads, int n_kv_heads, int head_dim,
                          int n_seqs, const int32_t* seq_new_ptr, const int32_t* seq_cached,
                          const int32_t* new_visible, int n_compute_units, int n_workgroups,
                          std::vector<int32_t>* table, PlanCounts* counts, const char** why) {
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
    const int rb = attend_row_block(path);

    std::vector<Unit> units;
    for (int s = 0; s < n_seqs; ++s) {
        const int n0 = seq_new_ptr[s];
        const int rows_s = (seq_new_ptr[s + 1] - n0) * group;
        for (int h = 0; h < n_kv_heads; ++h)
            for (int rho0 = 0; rho0 < rows_s; rho0 += rb) {
                const int rows = std::min(rb, rows_s - rho0);
                const int r_last = (rho0 + rows - 1) / group;
                const int vis = new_visible[n0 + r_last];
                const int64_t nvirt = (int64_t)vis + r_last + 1;
                if (nvirt > INT32_MAX / 2) {
                    *why = "key range too long";
                    return KVLINK_ERR_LAYOUT;
                }
                units.push_back({s, h, rho0, (int)((nvirt + kTileKeys - 1) / kTileKeys), rows, n0,
                                 seq_cached[s], vis, (int)nvirt, {}});
            }
    }
    int64_t T = 0;
    for (const Unit& x : units) T += x.tiles;
    const CostModel cm = cost_model(path, head_dim);
    for (Unit& x : units) {
        x.prefix.assign((size_t)x.tiles + 1, 0.0);
        x.live.assign((size_t)x.tiles, 1.0f);
        for (int t = 0; t < x.tiles; ++t) {
            int masked = 0;
            const int live = path == kPathWide ? live_pairs(x, t, group, new_visible, &masked) : 16;
            x.live[t] = (float)(live / 16.0);
            const int64_t new_rows =
                std::max<int64_t>(0, std::min<int64_t>(x.nvirt, (int64_t)kTileKeys * (t + 1)) -
                                         std::max<int64_t>(x.cmax, (int64_t)kTileKeys * t));
            x.prefix[t + 1] = x.prefix[t] + cm.tile_us + cm.live_us * live / 16.0 +
                              cm.mask_us * masked / 16.0 + cm.append_us * new_rows / kTileKeys;
        }
    }

    std::vector<Seg> segs, cand;
    if (T > 0) {
        const int64_t max_n = std::min<int64_t>(T, (int64_t)cm.slots_per_cu * n_compute_units);
        // every cut's estimate, then the cut that keeps the most workgroups
        // busy among those within kNearTie of the best estimate: the
        // estimate leaves out the launch and prologue costs that do not
        // shrink with more workgroups, and measured near ties favour filling
        // every compute unit
        constexpr double kNearTie = 0.02;
        struct Est {
            double t;
            int c, way, used;
        };
        std::vector<Est> est;
        auto cut = [&](int c, int way) {
            cand.clear();
            if (way == 0) cut_unit_aligned(units, c, &cand);
            else cut_equal_ranges(units, c, &cand);
        };
        auto consider = [&](int c, bool any_cost) {
            for (int way = 0; way < 2; ++way) {
                cut(c, way);
                const int used = compact_workgroups(&cand);
                // a forced count takes only cuts that use every workgroup
                if (used < c && any_cost) continue;
                est.push_back({estimate_us(units, cand, cm, head_dim, dt == KVLINK_BF16 ? 2 : 4), c,
                               way, used});
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
            segs = cand;
        }
    }
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
