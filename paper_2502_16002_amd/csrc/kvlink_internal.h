// kvlink_internal.h — shared device helpers and launcher declarations of the
// gfx950 KVLink library.  Not part of the public ABI (see include/kvlink.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kvlink.h"

#include <vector>

namespace kvlink {

// ------------------------------------------------------------ element types

struct bf16_t {
    uint16_t bits;
};

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16_t x) { return __uint_as_float((uint32_t)x.bits << 16); }

template <typename T>
__device__ __forceinline__ T from_f32(float x);
template <>
__device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <>
__device__ __forceinline__ bf16_t from_f32<bf16_t>(float x) {
    // IEEE conversion: round to nearest even (v_cvt_pk_bf16_f32 on gfx950)
    __bf16 h = (__bf16)x;
    return bf16_t{__builtin_bit_cast(uint16_t, h)};
}

// 16 bytes of T <-> floats (8 bf16 or 4 f32 per 16-byte access)
template <typename T>
__device__ __forceinline__ void unpack16(const uint4& v, float* f);
template <>
__device__ __forceinline__ void unpack16<float>(const uint4& v, float* f) {
    f[0] = __uint_as_float(v.x);
    f[1] = __uint_as_float(v.y);
    f[2] = __uint_as_float(v.z);
    f[3] = __uint_as_float(v.w);
}
template <>
__device__ __forceinline__ void unpack16<bf16_t>(const uint4& v, float* f) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        f[2 * i] = __uint_as_float(w[i] << 16);
        f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
}

template <typename T>
__device__ __forceinline__ uint4 pack16(const float* f);
template <>
__device__ __forceinline__ uint4 pack16<float>(const float* f) {
    return uint4{__float_as_uint(f[0]), __float_as_uint(f[1]), __float_as_uint(f[2]),
                 __float_as_uint(f[3])};
}
// two floats to a packed bf16 pair, round to nearest even (one
// v_cvt_pk_bf16_f32 on gfx950)
typedef float f32x2_v __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_v{lo, hi}, bf16x2_v));
}
template <>
__device__ __forceinline__ uint4 pack16<bf16_t>(const float* f) {
    return uint4{pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]), pack_bf16x2(f[4], f[5]),
                 pack_bf16x2(f[6], f[7])};
}

// ------------------------------------------------------------------- views

// Device copy of kvlink_kv_view, with the base typed by the caller.
struct View {
    char* base;  // bytes
    int64_t layer_stride, head_stride, row_stride, seq_stride, page_stride;  // elements
    const int32_t* block_table;
    int32_t page_size, max_pages;
};

// Element offset of (layer, head, seq, row, 0) in a view.
__device__ __forceinline__ int64_t view_offset(const View& v, int layer, int head, int seq,
                                               int row) {
    int64_t off = (int64_t)layer * v.layer_stride + (int64_t)head * v.head_stride;
    if (v.block_table) {
        const int page = v.block_table[(int64_t)seq * v.max_pages + row / v.page_size];
        off += (int64_t)page * v.page_stride + (int64_t)(row % v.page_size) * v.row_stride;
    } else {
        off += (int64_t)seq * v.seq_stride + (int64_t)row * v.row_stride;
    }
    return off;
}

// Rows of one (layer, head, seq) slice of a view, with the slice's part of
// the address hoisted: the per-row cost is one multiply-add (contiguous) or a
// block-table lookup (paged).
// A wavefront-uniform int32 read through the scalar cache (the address must
// be the same in every lane and the memory not written during the kernel).
__device__ __forceinline__ int32_t load_uniform(const int32_t* p) {
    return *(const __attribute__((address_space(4))) int32_t*)p;
}

struct RowPtr {
    const char* base;          // bytes: contiguous: row 0 of the slice; paged: (layer, head)
    int64_t row_bytes;         // row stride in bytes
    const int32_t* table;      // paged: this sequence's block-table row, else NULL
    int64_t page_bytes;        // paged: page stride in bytes
    int32_t page_size;
    int32_t page_shift;        // log2(page_size) for a power of two, else -1
    __device__ __forceinline__ const char* row(int r) const {
        if (!table) return base + (int64_t)r * row_bytes;
        const int pg = table[r / page_size];
        return base + (int64_t)pg * page_bytes + (int64_t)(r % page_size) * row_bytes;
    }
    // True when every aligned group of 16 rows lies in one page.
    __device__ __forceinline__ bool groups_of_16() const { return !table || page_shift >= 4; }
    // Paged slices whose 16-row groups lie in one page: the page of row r
    // (the same in every lane), read through the scalar cache, so that the
    // wavefront's vector loads in flight do not delay it.
    __device__ __forceinline__ int page_of(int r) const {
        return load_uniform(table + (r >> page_shift));
    }
    // Row r of page pg (from page_of; ignored when contiguous); for r a
    // multiple of 16, rows r..r+15 follow it at row_bytes.
    __device__ __forceinline__ const char* in_page(int pg, int r) const {
        if (!table) return base + (int64_t)r * row_bytes;
        return base + (int64_t)pg * page_bytes + (int64_t)(r & (page_size - 1)) * row_bytes;
    }
};

template <typename T>
__device__ __forceinline__ RowPtr row_ptr(const View& v, int layer, int head, int seq) {
    RowPtr r;
    const int64_t es = sizeof(T);
    r.base = v.base + ((int64_t)layer * v.layer_stride + (int64_t)head * v.head_stride) * es;
    r.row_bytes = v.row_stride * es;
    if (v.block_table) {
        r.table = v.block_table + (int64_t)seq * v.max_pages;
        r.page_bytes = v.page_stride * es;
        r.page_size = v.page_size;
        r.page_shift = (v.page_size & (v.page_size - 1)) == 0 ? __builtin_ctz(v.page_size) : -1;
    } else {
        r.base += (int64_t)seq * v.seq_stride * es;
        r.table = nullptr;
        r.page_bytes = 0;
        r.page_size = 1;
        r.page_shift = 0;
    }
    return r;
}

// RoPE frequencies of one (theta, head_dim): w[j] = theta^(-2j/d) for
// j < d/2, and pi/2 split into three parts for the argument reduction
// (pio2[0] and pio2[1] carry 22 significant bits each, so n * pio2[k] is
// exact for |n| < 2^31; the sum matches pi/2 to about 64 bits).  Built on the
// host in long double (make_rope_freqs) and passed by value to the kernels.
struct RopeFreqs {
    double w[64];
    double pio2[3];
};

RopeFreqs make_rope_freqs(double theta, int head_dim);

// RoPE of 16 bytes of each half of a head vector (Sec. 2.2; dims j and
// j + D/2 form a pair): lo holds dims j.., hi dims j + D/2.., c and s the
// cos/sin of their angles.  Every kernel that rotates keys or queries goes
// through this one routine (the re-encode, the new tokens' RoPE, fused or
// not, and the re-encode fused into the split attention), so each pair of
// forms produces the same bytes.
template <typename T>
__device__ __forceinline__ void rope_rotate16(const uint4& lo, const uint4& hi, const float* c,
                                              const float* s, uint4& x_out, uint4& y_out) {
    constexpr int E = 16 / (int)sizeof(T);
    float a[E], b[E], x[E], y[E];
    unpack16<T>(lo, a);
    unpack16<T>(hi, b);
#pragma unroll
    for (int e = 0; e < E; ++e) {
        x[e] = __builtin_fmaf(a[e], c[e], -(b[e] * s[e]));
        y[e] = __builtin_fmaf(a[e], s[e], b[e] * c[e]);
    }
    x_out = pack16<T>(x);
    y_out = pack16<T>(y);
}

// cos and sin of the RoPE angle pos * w[j] (Sec. 2.2), computed in double
// precision in registers, then rounded to float: Cody-Waite reduction of the
// angle by pi/2, Taylor series of sin and cos on the reduced argument
// (|r| <= pi/4, truncation error below 1e-17), and the quadrant.
__device__ __forceinline__ void rope_cos_sin(int64_t pos, int j, const RopeFreqs& f, float* c,
                                             float* s) {
    const double x = (double)pos * f.w[j];
    const double n = rint(x * 0.63661977236758134308);   // x / (pi/2), rounded
    double r = fma(-n, f.pio2[0], x);
    r = fma(-n, f.pio2[1], r);
    r = fma(-n, f.pio2[2], r);
    const double r2 = r * r;
    // sin r = r - r^3/3! + ... + r^17/17!, cos r = 1 - r^2/2! + ... + r^16/16!
    double ps = 1.0 / 355687428096000.0;                  // 1/17!
    ps = fma(ps, r2, -1.0 / 1307674368000.0);             // 1/15!
    ps = fma(ps, r2, 1.0 / 6227020800.0);                 // 1/13!
    ps = fma(ps, r2, -1.0 / 39916800.0);                  // 1/11!
    ps = fma(ps, r2, 1.0 / 362880.0);                     // 1/9!
    ps = fma(ps, r2, -1.0 / 5040.0);                      // 1/7!
    ps = fma(ps, r2, 1.0 / 120.0);                        // 1/5!
    ps = fma(ps, r2, -1.0 / 6.0);                         // 1/3!
    const double sr = fma(ps * r2, r, r);
    double pc = 1.0 / 20922789888000.0;                   // 1/16!
    pc = fma(pc, r2, -1.0 / 87178291200.0);               // 1/14!
    pc = fma(pc, r2, 1.0 / 479001600.0);                  // 1/12!
    pc = fma(pc, r2, -1.0 / 3628800.0);                   // 1/10!
    pc = fma(pc, r2, 1.0 / 40320.0);                      // 1/8!
    pc = fma(pc, r2, -1.0 / 720.0);                       // 1/6!
    pc = fma(pc, r2, 1.0 / 24.0);                         // 1/4!
    pc = fma(pc, r2, -0.5);                               // 1/2!
    const double cr = fma(pc, r2, 1.0);
    const int q = (int)((long long)n & 3);
    const double sv = q == 0 ? sr : q == 1 ? cr : q == 2 ? -sr : -cr;
    const double cv = q == 0 ? cr : q == 1 ? -sr : q == 2 ? -cr : sr;
    *c = (float)cv;
    *s = (float)sv;
}

// ---------------------------------------------------------------- launchers

// mode: kReencodeDelta rotates every row of a span by R(delta);
// kReencodePerToken rotates row t by R(delta + t - p), p = 0 or, with
// pos_map, the row's stored position pos_map[src_seq * pos_stride + row]
// (keys stored without rotation, or a compressed cache); kReencodeCopy
// moves the rows unchanged (values).
enum { kReencodeDelta = 0, kReencodePerToken = 1, kReencodeCopy = 2 };
hipError_t launch_reencode(kvlink_dtype dt, int head_dim, int n_layers, int n_kv_heads,
                           const RopeFreqs& freqs, int n_spans, const kvlink_span* spans,
                           int max_span_len, const View& src, const View& dst, int mode,
                           hipStream_t stream, const int32_t* pos_map = nullptr,
                           int64_t pos_stride = 0);

// Document-major re-encode: group g's spans (spans[group_ptr[g] ..
// group_ptr[g+1])) share their stored rows, read once for all of them.
hipError_t launch_reencode_shared(kvlink_dtype dt, int head_dim, int n_layers, int n_kv_heads,
                                  const RopeFreqs& freqs, int n_groups, const int32_t* group_ptr,
                                  const kvlink_span* spans, int max_span_len, const View& src,
                                  const View& dst, hipStream_t stream);

// Sizes of one attention call, from the arguments and the schedule.
struct AttendPlan {
    int n_q_heads, n_kv_heads, group, head_dim;
    int n_seqs, n_new_total;
    int row_block;          // GQA rows per unit
    int path;               // AttendPath
    int n_wg, n_units, n_segments, n_split;
    const int32_t* table;   // device copy of the schedule table
    bool partials;          // some unit has several segments
    bool merge_in_launch;   // wide kernel: split units merged inside the split launch
    size_t q_rot_bytes, part_o_bytes, part_ml_bytes, total_bytes;
};

// The split kernel of a call.  bf16 runs on the matrix cores at every row
// count: units of more than 16 GQA rows (group * new tokens of the longest
// request) on the wide-block kernel (256-row units, K/V tiles shared by eight
// wavefronts), smaller ones, as in a decoding step, on the decode kernel
// (16-row units, each wavefront streaming its own keys), whose padded 16-row
// products still take far fewer issue cycles than vector dot products.  fp32
// runs on the VALU kernel (16-row units).
enum AttendPath { kPathWide = 0, kPathDecode = 1, kPathValu = 2 };
AttendPath attend_path(kvlink_dtype dt, int group, int max_new);
// whether a schedule's row block belongs to a path (wide: 256, 128 or 64;
// decode and vector: 16)
bool attend_row_block_ok(AttendPath path, int row_block);

// The workspace starts with the arrival counters of the units a split
// kernel (wide or decode) merges in its own launch (one uint32 per unit, at
// most kMaxUnits):
// they must be zero before a workspace's first use, and every completed call
// leaves them zero.  The rotated queries and the split partials follow.
constexpr size_t kCounterBytes = 64 * 1024;
constexpr int kMaxUnits = (int)(kCounterBytes / 4);

// Fills every field from the sizes and the schedule's counts; returns false
// on invalid sizes or counts.
bool make_attend_plan(kvlink_dtype dt, int n_q_heads, int n_kv_heads, int head_dim,
                      int n_new_total, const kvlink_attend_plan& sched, AttendPlan* p);

// Segment record of the schedule table: kSegRecord int32 fields.
enum {
    kSegS = 0, kSegH, kSegRho0, kSegRows, kSegTileA, kSegTileB, kSegNseg, kSegLocal,
    kSegN0, kSegTc, kSegCmax, kSegNvirt, kSegPart, kSegNext, kSegUnit, kSegSpare, kSegRecord
};

// Unit record of the schedule table: kUnitRecord int32 fields.
enum {
    kUnitS = 0, kUnitH, kUnitRho0, kUnitRows, kUnitN0, kUnitSeg0, kUnitNseg, kUnitSpare,
    kUnitRecord
};

// The schedule of kvlink_attend_make_plan (host).  Returns a kvlink_status
// and, on failure, a message in *why.
struct PlanCounts {
    int n_wg, n_units, n_segments, row_block, n_split;
    bool in_launch;   // split units merged inside the split launch
    int64_t table_len;
};
int build_attend_schedule(kvlink_dtype dt, int n_q_heads, int n_kv_heads, int head_dim,
                          int n_seqs, const int32_t* seq_new_ptr, const int32_t* seq_cached,
                          const int32_t* new_visible, int n_compute_units, int n_workgroups,
                          int row_block, unsigned flags, std::vector<int32_t>* table,
                          PlanCounts* counts, const char** why);

struct AttendArgs {
    const void* q_new;
    const void* k_new;
    const void* v_new;
    View k, v;
    int layer;
    const int32_t* seq_new_ptr;
    const int32_t* seq_cached;
    const int32_t* new_pos;
    const int32_t* new_visible;
    RopeFreqs freqs;
    float scale;
    void* out;
    float* lse;
    void* workspace;
    const float* rope_table;   // the batch's cos/sin table, or NULL
    // re-encode fused into the split launch (wide kernel): the requests'
    // spans and their offsets [n_seqs + 1], or NULL
    const kvlink_span* fuse_spans = nullptr;
    const int32_t* fuse_span_ptr = nullptr;
};

hipError_t launch_attend(kvlink_dtype dt, const AttendPlan& p, const AttendArgs& a,
                         hipStream_t stream, unsigned stages);
// (cos, sin) of every new token's angles, [n_new_total][head_dim / 2]
hipError_t launch_rope_table(int head_dim, const RopeFreqs& freqs, int n_new_total,
                             const int32_t* new_pos, float* table, hipStream_t stream);

}  // namespace kvlink
