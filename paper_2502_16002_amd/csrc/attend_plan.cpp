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
// equal contiguous ranges, so every workgroup gets the same number of tiles
// whatever the mix of long and short units (the row blocks of link tokens
// early in the context see few keys, those of the queries see all of them).
// A workgroup's range crosses unit boundaries; each piece is a segment with
// its own partial result, merged by the combine when a unit has several.
//
// The number of workgroups comes from a cost model: a workgroup costs a fixed
// set-up per segment (loads of its rows' queries and the first key tiles)
// plus a per-tile cost; the launch lasts as long as its longest workgroup;
// units with several segments add the combine launch and the traffic of
// their partials.  Constants are fitted to MI355X timings of the Llama-8B
// shaped 10- and 40-document workloads.
#include <algorithm>
#include <cstdint>
#include <vector>

#include "kvlink_internal.h"

namespace kvlink {
namespace {

constexpr int kTileKeys = 64;

struct Unit {
    int s, h, rho0, tiles, rows;
};

struct CostModel {
    double per_segment_us, per_tile_us;
    int slots_per_cu;
};

CostModel cost_model(bool mfma, int head_dim) {
    if (mfma) return {4.5, head_dim == 128 ? 1.9 : 1.2, 1};
    return {3.0, head_dim == 128 ? 1.0 : 0.6, head_dim == 128 ? 2 : 4};
}

// Piece boundaries of n equal ranges over units with prefix tile offsets
// `off` (off[u] = first global tile of unit u, off.back() = total).
template <typename F>
void for_each_piece(const std::vector<int64_t>& off, int n, F&& f) {
    const int64_t T = off.back();
    size_t u = 0;
    for (int w = 0; w < n; ++w) {
        const int64_t t0 = T * w / n, t1 = T * (w + 1) / n;
        while (off[u + 1] <= t0) ++u;
        for (int64_t t = t0; t < t1;) {
            while (off[u + 1] <= t) ++u;
            const int64_t e = std::min(t1, off[u + 1]);
            f(w, (int)u, t - off[u], e - t);
            t = e;
        }
    }
}

double estimate_us(const std::vector<Unit>& units, const std::vector<int64_t>& off, int n,
                   const CostModel& cm, int head_dim) {
    std::vector<double> wg(n, 0.0);
    std::vector<int> pieces(units.size(), 0);
    for_each_piece(off, n, [&](int w, int u, int64_t, int64_t len) {
        wg[w] += cm.per_segment_us + cm.per_tile_us * (double)len;
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
                          int n_seqs, const int32_t* seq_new_ptr, const int32_t* new_visible,
                          int n_compute_units, int n_workgroups, std::vector<int32_t>* table,
                          PlanCounts* counts, const char** why) {
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
    const bool mfma = attend_uses_mfma(dt, group, max_new);
    const int rb = attend_row_block(mfma);

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
                units.push_back({s, h, rho0, (int)((nvirt + kTileKeys - 1) / kTileKeys), rows});
            }
    }
    seq_unit[n_seqs] = (int32_t)units.size();
    std::vector<int64_t> off(units.size() + 1, 0);
    for (size_t u = 0; u < units.size(); ++u) off[u + 1] = off[u] + units[u].tiles;
    const int64_t T = off.back();

    int n = 0;
    if (T > 0) {
        const CostModel cm = cost_model(mfma, head_dim);
        const int64_t max_n = std::min<int64_t>(T, (int64_t)cm.slots_per_cu * n_compute_units);
        if (n_workgroups > 0) {
            n = (int)std::min<int64_t>(n_workgroups, T);
        } else {
            double best = 1e300;
            for (int c = 1; c <= max_n; ++c) {
                const double t = estimate_us(units, off, c, cm, head_dim);
                if (t < best * 0.99) {   // fewer workgroups on near ties
                    best = t;
                    n = c;
                }
            }
        }
    }

    // wg entries and segment numbering
    std::vector<int32_t> wg(4 * (size_t)n, 0);
    std::vector<int32_t> unit_seg(units.size() + 1, -1);
    int n_seg = 0;
    int last_w = -1;
    for_each_piece(off, n, [&](int w, int u, int64_t t0, int64_t len) {
        if (w != last_w) {
            wg[4 * w + 0] = u;
            wg[4 * w + 1] = (int32_t)t0;
            wg[4 * w + 3] = n_seg;
            last_w = w;
        }
        wg[4 * w + 2] += (int32_t)len;
        if (unit_seg[u] < 0) unit_seg[u] = n_seg;
        ++n_seg;
    });
    unit_seg[units.size()] = n_seg;
    for (size_t u = units.size(); u-- > 0;)      // (only for T == 0: no pieces at all)
        if (unit_seg[u] < 0) unit_seg[u] = unit_seg[u + 1];

    counts->n_wg = n;
    counts->n_units = (int)units.size();
    counts->n_segments = n_seg;
    counts->row_block = rb;
    counts->table_len = 4 * (int64_t)n + 4 * (int64_t)units.size() + (int64_t)units.size() + 1 +
                        n_seqs + 1;
    if (table) {
        table->clear();
        table->reserve((size_t)counts->table_len);
        table->insert(table->end(), wg.begin(), wg.end());
        for (const Unit& x : units) {
            table->push_back(x.s);
            table->push_back(x.h);
            table->push_back(x.rho0);
            table->push_back(x.tiles);
        }
        table->insert(table->end(), unit_seg.begin(), unit_seg.end());
        table->insert(table->end(), seq_unit.begin(), seq_unit.end());
    }
    return KVLINK_OK;
}

}  // namespace kvlink
