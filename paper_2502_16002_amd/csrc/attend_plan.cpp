// attend_plan.cpp — host-side schedule of the split-K attention.
//
// Work unit: (request s, KV head h, row block b).  The rows of request s for
// KV head h are its new tokens' query heads packed as row = token * group +
// head-in-group; block b holds rows [b * row_block, (b + 1) * row_block).  The
// unit's keys are the cached rows its last token sees (the attention map of
// Sec. 2.3: every position at or before the token's own) followed by the new
// rows up to that token; it walks them in 64-key tiles.
//
// All tiles, units in (s, h, b) order, are dealt out to the workgroups as
// contiguous ranges of equal cost, so every workgroup gets the same work
// whatever the mix of long and short units (the row blocks of link tokens
// early in the context see few keys, those of the queries see all of them).
// A tile of a unit whose rows fill at most half the workgroup's wavefronts
// costs half (its other wavefronts sit idle and their SIMDs run one
// wavefront instead of two).  A workgroup's range crosses unit boundaries;
// each piece is a segment with its own partial result, merged by the combine
// when a unit has several.  Each segment gets a record with everything its
// workgroup needs to issue its first key-tile loads after a single table
// read.
//
// The number of workgroups comes from a cost model: a workgroup costs a fixed
// set-up per segment (loads of its rows' queries and the first key tiles)
// plus a per-tile cost; the launch lasts as long as its longest workgroup;
// units with several segments add the combine launch and the traffic of
// their partials.  Constants are fitted to MI355X timings of the Llama-8B
// shaped 10- and 40-document workloads.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdint>
#include <vector>

#include "kvlink_internal.h"

namespace kvlink {
namespace {

constexpr int kTileKeys = 64;

struct Unit {
    int s, h, rho0, tiles, rows, n0, Tc, cmax, nvirt;
    double weight;   // cost of one tile relative to a full row block
};

struct CostModel {
    double per_segment_us, per_tile_us;
    int slots_per_cu;
};

CostModel cost_model(bool mfma, int head_dim) {
    if (mfma) return {4.0, head_dim == 128 ? 2.1 : 1.3, 1};
    return {3.0, head_dim == 128 ? 1.0 : 0.6, head_dim == 128 ? 2 : 4};
}

// Pieces of n contiguous ranges of equal cost over the units' tiles (a
// tile of unit u costs units[u].weight).  Calls f(w, u, first tile, count)
// for every non-empty piece, in order.
template <typename F>
void for_each_piece(const std::vector<Unit>& units, const std::vector<double>& woff, int n, F&& f) {
    const double W = woff.back();
    size_t u = 0;
    int64_t t_in_u = 0;   // next tile of unit u to hand out
    for (int w = 0; w < n; ++w) {
        const double end = w + 1 == n ? W : W * (w + 1) / n;
        while (u < units.size()) {
            if (t_in_u >= units[u].tiles) {
                ++u;
                t_in_u = 0;
                continue;
            }
            // tiles of unit u whose start lies before `end`
            const double start_w = woff[u] + t_in_u * units[u].weight;
            if (start_w >= end - 1e-9 && w + 1 < n) break;
            int64_t take = w + 1 == n ? units[u].tiles - t_in_u
                                      : (int64_t)std::ceil((end - start_w) / units[u].weight - 1e-9);
            take = std::max<int64_t>(1, std::min<int64_t>(take, units[u].tiles - t_in_u));
            f(w, (int)u, t_in_u, take);
            t_in_u += take;
        }
    }
}

double estimate_us(const std::vector<Unit>& units, const std::vector<double>& woff, int n,
                   const CostModel& cm, int head_dim) {
    std::vector<double> wg(n, 0.0);
    std::vector<int> pieces(units.size(), 0);
    for_each_piece(units, woff, n, [&](int w, int u, int64_t, int64_t len) {
        wg[w] += cm.per_segment_us + cm.per_tile_us * units[u].weight * (double)len;
        ++pieces[u];
    });
    double t = *std::max_element(wg.begin(), wg.end());
    double bytes = 0.0;
    for (size_t u = 0; u < units.size(); ++u)
        if (pieces[u] > 1)
            bytes += 2.0 * pieces[u] * units[u].rows * (head_dim + 2) * 4.0;   // write + read
    if (bytes > 0.0) t += 3.0 + bytes / 4.0e6;   // combine launch, ~4 TB/s effective
    return t;
}

}  // namespace

bool attend_uses_mfma(kvlink_dtype dt, int group, int max_new) {
    return dt == KVLINK_BF16 && (int64_t)max_new * group >= 32;
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
        const int n = seq_new_ptr[s + 1] - seq_new_ptr[s];
        if (n < 0) {
            *why = "seq_new_ptr is not non-decreasing";
            return KVLINK_ERR_LAYOUT;
        }
        max_new = std::max(max_new, n);
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
    const bool mfma = attend_uses_mfma(dt, group, max_new);
    const int rb = attend_row_block(mfma);

    // rows per wavefront of the kernel the path selects (8 x 32 rows on the
    // matrix cores, 4 x 4 on the VALU path)
    const int rows_per_wave = rb / 8 > 0 && mfma ? rb / 8 : rb / 4;
    std::vector<Unit> units;
    std::vector<int32_t> seq_unit(n_seqs + 1);
    for (int s = 0; s < n_seqs; ++s) {
        seq_unit[s] = (int32_t)units.size();
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
                const int waves = (rows + rows_per_wave - 1) / rows_per_wave;
                const double weight = mfma && waves <= 4 ? 0.5 : 1.0;
                units.push_back({s, h, rho0, (int)((nvirt + kTileKeys - 1) / kTileKeys), rows, n0,
                                 seq_cached[s], vis, (int)nvirt, weight});
            }
    }
    seq_unit[n_seqs] = (int32_t)units.size();
    std::vector<double> woff(units.size() + 1, 0.0);
    int64_t T = 0;
    for (size_t u = 0; u < units.size(); ++u) {
        woff[u + 1] = woff[u] + units[u].tiles * units[u].weight;
        T += units[u].tiles;
    }

    int n = 0;
    if (T > 0) {
        const CostModel cm = cost_model(mfma, head_dim);
        const int64_t max_n = std::min<int64_t>(T, (int64_t)cm.slots_per_cu * n_compute_units);
        if (n_workgroups > 0) {
            n = (int)std::min<int64_t>(n_workgroups, T);
        } else {
            double best = 1e300;
            for (int c = 1; c <= max_n; ++c) {
                const double t = estimate_us(units, woff, c, cm, head_dim);
                if (t < best * 0.99) {   // fewer workgroups on near ties
                    best = t;
                    n = c;
                }
            }
        }
    }

    // segments in order; a workgroup owns a contiguous run of them
    struct Seg {
        int w, u;
        int64_t t0, len;
    };
    std::vector<Seg> segs;
    for_each_piece(units, woff, n, [&](int w, int u, int64_t t0, int64_t len) {
        segs.push_back({w, u, t0, len});
    });
    std::vector<int32_t> wg_seg(n + 1, 0);
    std::vector<int32_t> unit_seg(units.size() + 1, -1);
    std::vector<int> pieces(units.size(), 0);
    for (size_t i = 0; i < segs.size(); ++i) {
        ++wg_seg[segs[i].w + 1];
        if (unit_seg[segs[i].u] < 0) unit_seg[segs[i].u] = (int32_t)i;
        ++pieces[segs[i].u];
    }
    for (int w = 0; w < n; ++w) wg_seg[w + 1] += wg_seg[w];
    const int n_seg = (int)segs.size();
    unit_seg[units.size()] = n_seg;
    for (size_t u = units.size(); u-- > 0;)      // (only for T == 0: no pieces at all)
        if (unit_seg[u] < 0) unit_seg[u] = unit_seg[u + 1];

    counts->n_wg = n;
    counts->n_units = (int)units.size();
    counts->n_segments = n_seg;
    counts->row_block = rb;
    const int64_t rec0 = ((int64_t)n + 1 + 3) / 4 * 4;   // records start 16-byte aligned
    counts->table_len = rec0 + (int64_t)kSegRecord * n_seg + (int64_t)units.size() + 1 + n_seqs + 1;
    if (table) {
        table->assign((size_t)counts->table_len, 0);
        int32_t* t = table->data();
        std::copy(wg_seg.begin(), wg_seg.end(), t);
        for (int i = 0; i < n_seg; ++i) {
            const Seg& g = segs[i];
            const Unit& x = units[g.u];
            int32_t* r = t + rec0 + (int64_t)kSegRecord * i;
            r[kSegS] = x.s;
            r[kSegH] = x.h;
            r[kSegRho0] = x.rho0;
            r[kSegRows] = x.rows;
            r[kSegTileA] = (int32_t)g.t0;
            r[kSegTileB] = (int32_t)(g.t0 + g.len);
            r[kSegNseg] = pieces[g.u];
            r[kSegLocal] = i - unit_seg[g.u];
            r[kSegN0] = x.n0;
            r[kSegTc] = x.Tc;
            r[kSegCmax] = x.cmax;
            r[kSegNvirt] = x.nvirt;
        }
        int32_t* us = t + rec0 + (int64_t)kSegRecord * n_seg;
        std::copy(unit_seg.begin(), unit_seg.end(), us);
        std::copy(seq_unit.begin(), seq_unit.end(), us + units.size() + 1);
    }
    return KVLINK_OK;
}

}  // namespace kvlink
