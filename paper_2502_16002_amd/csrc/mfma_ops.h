// mfma_ops.h — register and LDS helpers shared by the matrix-core attention
// kernels: operand types, the transposed LDS reads of V^T operands, bf16
// packing and the direct-to-LDS loads with their waits.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace kvlink {
namespace attn {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short shortx4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) shortx4 lds_shortx4;

namespace {

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

// The same reads issued without the wait: the caller waits with wait_vt,
// whose in-out operands keep every use of r after the wait.  Only valid
// where the compiler issues no LDS access of its own in between (its own
// waits would then also cover these reads, which is correct but slower).
#define KVLINK_TR_ISSUE(o, i, off) "ds_read_b64_tr_b16 %" #o ", %" #i " offset:%" #off "\n\t"
template <int OFF0, int OFF1>
__device__ __forceinline__ void issue_vt8(const uint32_t (&a)[8], uint2 (&r)[8][2]) {
#if defined(__HIP_DEVICE_COMPILE__)
    asm volatile(
        KVLINK_TR_ISSUE(0, 16, 24) KVLINK_TR_ISSUE(1, 16, 25)
        KVLINK_TR_ISSUE(2, 17, 24) KVLINK_TR_ISSUE(3, 17, 25)
        KVLINK_TR_ISSUE(4, 18, 24) KVLINK_TR_ISSUE(5, 18, 25)
        KVLINK_TR_ISSUE(6, 19, 24) KVLINK_TR_ISSUE(7, 19, 25)
        KVLINK_TR_ISSUE(8, 20, 24) KVLINK_TR_ISSUE(9, 20, 25)
        KVLINK_TR_ISSUE(10, 21, 24) KVLINK_TR_ISSUE(11, 21, 25)
        KVLINK_TR_ISSUE(12, 22, 24) KVLINK_TR_ISSUE(13, 22, 25)
        KVLINK_TR_ISSUE(14, 23, 24) KVLINK_TR_ISSUE(15, 23, 25)
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
__device__ __forceinline__ void issue_vt4(const uint32_t (&a)[4], uint2 (&r)[4][2]) {
#if defined(__HIP_DEVICE_COMPILE__)
    asm volatile(
        KVLINK_TR_ISSUE(0, 8, 12) KVLINK_TR_ISSUE(1, 8, 13)
        KVLINK_TR_ISSUE(2, 9, 12) KVLINK_TR_ISSUE(3, 9, 13)
        KVLINK_TR_ISSUE(4, 10, 12) KVLINK_TR_ISSUE(5, 10, 13)
        KVLINK_TR_ISSUE(6, 11, 12) KVLINK_TR_ISSUE(7, 11, 13)
        : "=&v"(r[0][0]), "=&v"(r[0][1]), "=&v"(r[1][0]), "=&v"(r[1][1]), "=&v"(r[2][0]),
          "=&v"(r[2][1]), "=&v"(r[3][0]), "=&v"(r[3][1])
        : "v"(a[0]), "v"(a[1]), "v"(a[2]), "v"(a[3]), "i"(OFF0), "i"(OFF1)
        : "memory");
#endif
}
#undef KVLINK_TR_ISSUE

__device__ __forceinline__ void wait_vt(uint2 (&r)[8][2]) {
#if defined(__HIP_DEVICE_COMPILE__)
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(r[0][0]), "+v"(r[0][1]), "+v"(r[1][0]), "+v"(r[1][1]), "+v"(r[2][0]),
                   "+v"(r[2][1]), "+v"(r[3][0]), "+v"(r[3][1]), "+v"(r[4][0]), "+v"(r[4][1]),
                   "+v"(r[5][0]), "+v"(r[5][1]), "+v"(r[6][0]), "+v"(r[6][1]), "+v"(r[7][0]),
                   "+v"(r[7][1])
                 :
                 : "memory");
#endif
}

__device__ __forceinline__ void wait_vt(uint2 (&r)[4][2]) {
#if defined(__HIP_DEVICE_COMPILE__)
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(r[0][0]), "+v"(r[0][1]), "+v"(r[1][0]), "+v"(r[1][1]), "+v"(r[2][0]),
                   "+v"(r[2][1]), "+v"(r[3][0]), "+v"(r[3][1])
                 :
                 : "memory");
#endif
}

template <int DT, int OFF0, int OFF1>
__device__ __forceinline__ void issue_vt(const uint32_t (&a)[DT], uint2 (&r)[DT][2]) {
    if constexpr (DT == 8) issue_vt8<OFF0, OFF1>(a, r);
    else issue_vt4<OFF0, OFF1>(a, r);
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

// Cache-policy bits of a load: kStream marks data read once (non-temporal).
constexpr int kCached = 0, kStream = 2;

// 16-byte direct load from global memory into LDS: lane i's bytes land at
// lds + 16 i (lds must be wave-uniform and not LDS address 0).  Device pass
// only, like the register-constrained asm above.
template <int kPolicy = kCached>
__device__ __forceinline__ void load_lds16(const void* src, void* lds) {
#if defined(__HIP_DEVICE_COMPILE__)
    __builtin_amdgcn_global_load_lds(src, lds, 16, 0, kPolicy);
#endif
}

// Workgroup barrier that leaves this wave's vector-memory loads in flight
// (__syncthreads waits for all of them): the wave's LDS accesses complete
// first, and the compiler keeps memory accesses on their side of it.
__device__ __forceinline__ void barrier_keep_loads() {
#if defined(__HIP_DEVICE_COMPILE__)
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
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

}  // namespace
}  // namespace attn
}  // namespace kvlink
