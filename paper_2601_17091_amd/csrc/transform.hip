// ROCKET transform on CDNA4 (gfx950): fused MFMA kernel, plain direct
// kernel, and the HIP-facing half of the C ABI.
//
// Fused kernel (one workgroup = a few series x one split of the work items
// of one code variant):
//   1. the series are staged HBM -> LDS with coalesced loads, with zero
//      margins on both sides that stand in for the zero padding (Sec. 2.1);
//   2. each wavefront takes work items from an LDS counter; an item holds 4
//      or 8 kernels of one (length, dilation, padding) bucket, which share
//      their outputs' positions and the series values under every tap;
//   3. outputs are computed in tiles of 64 consecutive positions, lane l
//      taking position 64k + l of tile k; for tap j the 64 lanes read 64
//      consecutive series values (index 64k - p + j*d + l): one
//      conflict-free ds_read_addtid_b32 per tile and tap, addressed by a
//      scalar register;
//   4. the dot products of a tile are an outer-product contraction over the
//      taps: v_mfma_f32_4x4x1_16b_f32 multiplies the 4 kernels' weights (A,
//      one kernel per block row) by the 64 lanes' series values (B), one tap
//      per instruction, accumulating onto the bias;
//   5. MAX is a per-lane running max reduced across the wavefront at the end
//      of a series; the positive count is a ballot of y > 0 popcounted on
//      the scalar unit; no dot product is written to memory (Sec. 3.2 keeps
//      only the two counters per pair as well);
//   6. PPV = count / O and MAX are written to F in the original kernel order.
//
// MINIROCKET kernel (the variant Sec. 5 names): the same staging and tiles;
// the dot products of its 42 kernels of one (dilation, padding) come from
// the 9 shared tap values and their sum on the vector unit, and each is
// compared with the item's biases of its kernel; PPV = count / O per
// (kernel, bias).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cmath>
#include <cstring>
#include <mutex>
#include <new>

#include "rocket_internal.h"

using rocket::ItemDesc;

typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v2f __attribute__((ext_vector_type(2)));
constexpr uint64_t kNegInfPair = 0xff800000ff800000ull;  // two fp32 -inf

// ---------------------------------------------------------------------------
// Checked build (compiled with ROCKET_CHECKED=1 into librocket_checked.so):
// every LDS tile read is checked against the bytes its workgroup staged,
// every feature store of the workgroup kernels against the rows and columns
// of its launch, and every slot column the series-lane permutation reads
// against the plan's slots.  A failed check sets a bit of g_rocket_checks
// (read and cleared by rocket_check_flags) and the access is redirected
// inside the buffer or skipped, so a wrong index never reads or writes
// outside it.  The product build compiles none of this.
// ---------------------------------------------------------------------------
#ifndef ROCKET_CHECKED
#define ROCKET_CHECKED 0
#endif
[[maybe_unused]] constexpr uint32_t kCheckLdsRead = 1u;  // an LDS tile read outside the staged bytes
[[maybe_unused]] constexpr uint32_t kCheckStore = 2u;    // a feature store outside its rows / columns
[[maybe_unused]] constexpr uint32_t kCheckSlotRead = 4u; // a read of the slot-ordered buffer outside its columns
#if ROCKET_CHECKED
__device__ unsigned int g_rocket_checks;
__shared__ uint32_t g_check_lds_lo, g_check_lds_hi;  // staged LDS bytes [lo, hi) of the workgroup
__shared__ float *g_check_out_lo;                     // the launch's output floats [lo, hi)
__shared__ float *g_check_out_hi;
__device__ __forceinline__ void check_failed(uint32_t bit) {
    if ((threadIdx.x & 63) == 0) atomicOr(&g_rocket_checks, bit);
}
#endif

// The LDS byte address m of a read of `bytes` bytes (wave-uniform), checked
// in checked builds; a read outside the staged bytes goes to their start.
__device__ __forceinline__ uint32_t lds_checked(uint32_t m, uint32_t bytes) {
#if ROCKET_CHECKED
    // the bounds come from LDS into vector registers; the result goes to a
    // scalar operand (M0), so it is made wave-uniform explicitly (it is
    // uniform: m and the bounds are)
    const uint32_t lo = __builtin_amdgcn_readfirstlane(g_check_lds_lo);
    const uint32_t hi = __builtin_amdgcn_readfirstlane(g_check_lds_hi);
    uint32_t r = m;
    if (m < lo || m + bytes > hi) {
        check_failed(kCheckLdsRead);
        r = lo;
    }
    return __builtin_amdgcn_readfirstlane(r);
#endif
    (void)bytes;
    return m;
}

// Whether the n floats at f lie in the launch's output (always true in the
// product build).
__device__ __forceinline__ bool store_checked(const float *f, int n) {
#if ROCKET_CHECKED
    if (f < g_check_out_lo || f + n > g_check_out_hi) {
        check_failed(kCheckStore);
        return false;
    }
#endif
    (void)f;
    (void)n;
    return true;
}

// Record a workgroup's staged LDS bytes and its launch's output range
// (checked builds; thread 0, before the workgroup's barrier).
__device__ __forceinline__ void set_check_bounds(const float *smem, int64_t staged_floats, float *out_lo,
                                                 float *out_hi) {
#if ROCKET_CHECKED
    if (threadIdx.x == 0) {
        g_check_lds_lo = (uint32_t)(__UINTPTR_TYPE__)(__attribute__((address_space(3))) const float *)smem;
        g_check_lds_hi = g_check_lds_lo + 4u * (uint32_t)staged_floats;
        g_check_out_lo = out_lo;
        g_check_out_hi = out_hi;
    }
#endif
    (void)smem;
    (void)staged_floats;
    (void)out_lo;
    (void)out_hi;
}

// Read-only tables indexed by wavefront-uniform values are read through the
// constant address space, which lets the compiler use scalar loads.
template <typename T>
using ConstPtr = const __attribute__((address_space(4))) T *;
template <typename T>
__device__ __forceinline__ ConstPtr<T> as_const(const T *p) {
    return (ConstPtr<T>)(p);
}

// LDS byte address of a pointer into the kernel's shared memory.
typedef __attribute__((address_space(3))) const float lds_cfloat;
__device__ __forceinline__ uint32_t lds_addr(const float *p) {
    return (uint32_t)(__UINTPTR_TYPE__)(lds_cfloat *)p;
}

// The series values of up to 4 tiles under one tap: NT reads of 64
// consecutive floats, 256 bytes apart, the first at LDS byte address m
// (wavefront-uniform).  ds_read_addtid_b32 reads the dword at
// M0 + offset + 4 * lane, so the address comes from a scalar register and no
// vector instruction computes it.  M0 is written right before the reads
// (one wait state between the write and its first use) and is not used by
// compiled code in these kernels.  The reads complete before the asm block
// ends (lgkmcnt(0)), so the outputs are ready when the compiler sees them.
template <int NT>
__device__ __forceinline__ void lds_tiles_raw(uint32_t m, float (&xv)[NT]);
template <>
__device__ __forceinline__ void lds_tiles_raw<1>(uint32_t m, float (&xv)[1]) {
    asm volatile(
        "s_mov_b32 m0, %1\n\ts_nop 0\n\t"
        "ds_read_addtid_b32 %0\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=v"(xv[0])
        : "s"(m)
        : "memory");
}
template <>
__device__ __forceinline__ void lds_tiles_raw<2>(uint32_t m, float (&xv)[2]) {
    asm volatile(
        "s_mov_b32 m0, %2\n\ts_nop 0\n\t"
        "ds_read_addtid_b32 %0\n\tds_read_addtid_b32 %1 offset:256\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(xv[0]), "=&v"(xv[1])
        : "s"(m)
        : "memory");
}
template <>
__device__ __forceinline__ void lds_tiles_raw<3>(uint32_t m, float (&xv)[3]) {
    asm volatile(
        "s_mov_b32 m0, %3\n\ts_nop 0\n\t"
        "ds_read_addtid_b32 %0\n\tds_read_addtid_b32 %1 offset:256\n\t"
        "ds_read_addtid_b32 %2 offset:512\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(xv[0]), "=&v"(xv[1]), "=&v"(xv[2])
        : "s"(m)
        : "memory");
}
template <>
__device__ __forceinline__ void lds_tiles_raw<4>(uint32_t m, float (&xv)[4]) {
    asm volatile(
        "s_mov_b32 m0, %4\n\ts_nop 0\n\t"
        "ds_read_addtid_b32 %0\n\tds_read_addtid_b32 %1 offset:256\n\t"
        "ds_read_addtid_b32 %2 offset:512\n\tds_read_addtid_b32 %3 offset:768\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(xv[0]), "=&v"(xv[1]), "=&v"(xv[2]), "=&v"(xv[3])
        : "s"(m)
        : "memory");
}
// 5..8 tiles: all reads from one M0, then two waits.  lds_tiles waits until
// at most NT-4 reads are in flight (lgkmcnt(NT-4)); LDS reads complete in
// order, so tiles 0-3 are ready and their MFMAs can issue while the rest
// arrive.  lds_tiles_rest then waits for the rest: it takes tiles 4.. as
// operands and returns them, so no use of them precedes it.
template <int NT>
__device__ __forceinline__ void lds_tiles_rest(float (&xv)[NT]);

template <>
__device__ __forceinline__ void lds_tiles_raw<5>(uint32_t m, float (&xv)[5]) {
    asm volatile(
        "s_mov_b32 m0, %5\n\ts_nop 0\n\t"
        "ds_read_addtid_b32 %0\n\t"
        "ds_read_addtid_b32 %1 offset:256\n\t"
        "ds_read_addtid_b32 %2 offset:512\n\t"
        "ds_read_addtid_b32 %3 offset:768\n\t"
        "ds_read_addtid_b32 %4 offset:1024\n\t"
        "s_waitcnt lgkmcnt(1)"
        : "=&v"(xv[0]), "=&v"(xv[1]), "=&v"(xv[2]), "=&v"(xv[3]), "=&v"(xv[4])
        : "s"(m)
        : "memory");
}
template <>
__device__ __forceinline__ void lds_tiles_rest<5>(float (&xv)[5]) {
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(xv[4]) : : "memory");
}

template <>
__device__ __forceinline__ void lds_tiles_raw<6>(uint32_t m, float (&xv)[6]) {
    asm volatile(
        "s_mov_b32 m0, %6\n\ts_nop 0\n\t"
        "ds_read_addtid_b32 %0\n\t"
        "ds_read_addtid_b32 %1 offset:256\n\t"
        "ds_read_addtid_b32 %2 offset:512\n\t"
        "ds_read_addtid_b32 %3 offset:768\n\t"
        "ds_read_addtid_b32 %4 offset:1024\n\t"
        "ds_read_addtid_b32 %5 offset:1280\n\t"
        "s_waitcnt lgkmcnt(2)"
        : "=&v"(xv[0]), "=&v"(xv[1]), "=&v"(xv[2]), "=&v"(xv[3]), "=&v"(xv[4]), "=&v"(xv[5])
        : "s"(m)
        : "memory");
}
template <>
__device__ __forceinline__ void lds_tiles_rest<6>(float (&xv)[6]) {
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(xv[4]), "+v"(xv[5]) : : "memory");
}

template <>
__device__ __forceinline__ void lds_tiles_raw<7>(uint32_t m, float (&xv)[7]) {
    asm volatile(
        "s_mov_b32 m0, %7\n\ts_nop 0\n\t"
        "ds_read_addtid_b32 %0\n\t"
        "ds_read_addtid_b32 %1 offset:256\n\t"
        "ds_read_addtid_b32 %2 offset:512\n\t"
        "ds_read_addtid_b32 %3 offset:768\n\t"
        "ds_read_addtid_b32 %4 offset:1024\n\t"
        "ds_read_addtid_b32 %5 offset:1280\n\t"
        "ds_read_addtid_b32 %6 offset:1536\n\t"
        "s_waitcnt lgkmcnt(3)"
        : "=&v"(xv[0]), "=&v"(xv[1]), "=&v"(xv[2]), "=&v"(xv[3]), "=&v"(xv[4]), "=&v"(xv[5]), "=&v"(xv[6])
        : "s"(m)
        : "memory");
}
template <>
__device__ __forceinline__ void lds_tiles_rest<7>(float (&xv)[7]) {
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(xv[4]), "+v"(xv[5]), "+v"(xv[6]) : : "memory");
}

template <>
__device__ __forceinline__ void lds_tiles_raw<8>(uint32_t m, float (&xv)[8]) {
    asm volatile(
        "s_mov_b32 m0, %8\n\ts_nop 0\n\t"
        "ds_read_addtid_b32 %0\n\t"
        "ds_read_addtid_b32 %1 offset:256\n\t"
        "ds_read_addtid_b32 %2 offset:512\n\t"
        "ds_read_addtid_b32 %3 offset:768\n\t"
        "ds_read_addtid_b32 %4 offset:1024\n\t"
        "ds_read_addtid_b32 %5 offset:1280\n\t"
        "ds_read_addtid_b32 %6 offset:1536\n\t"
        "ds_read_addtid_b32 %7 offset:1792\n\t"
        "s_waitcnt lgkmcnt(4)"
        : "=&v"(xv[0]), "=&v"(xv[1]), "=&v"(xv[2]), "=&v"(xv[3]), "=&v"(xv[4]), "=&v"(xv[5]), "=&v"(xv[6]), "=&v"(xv[7])
        : "s"(m)
        : "memory");
}
template <>
__device__ __forceinline__ void lds_tiles_rest<8>(float (&xv)[8]) {
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(xv[4]), "+v"(xv[5]), "+v"(xv[6]), "+v"(xv[7]) : : "memory");
}

// The reads of lds_tiles_raw, with the address checked in checked builds.
template <int NT>
__device__ __forceinline__ void lds_tiles(uint32_t m, float (&xv)[NT]) {
    lds_tiles_raw<NT>(lds_checked(m, 256u * NT), xv);
}

// The reads of lds_tiles_raw<NT> (NT <= 4) without the wait: the values
// arrive in xv once lds_wait<NT, KEEP> has run after them.
template <int NT>
__device__ __forceinline__ void lds_issue_raw(uint32_t m, float (&xv)[NT]);
template <>
__device__ __forceinline__ void lds_issue_raw<1>(uint32_t m, float (&xv)[1]) {
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tds_read_addtid_b32 %0" : "=v"(xv[0]) : "s"(m) : "memory");
}
template <>
__device__ __forceinline__ void lds_issue_raw<2>(uint32_t m, float (&xv)[2]) {
    asm volatile(
        "s_mov_b32 m0, %2\n\ts_nop 0\n\t"
        "ds_read_addtid_b32 %0\n\tds_read_addtid_b32 %1 offset:256"
        : "=&v"(xv[0]), "=&v"(xv[1])
        : "s"(m)
        : "memory");
}
template <>
__device__ __forceinline__ void lds_issue_raw<3>(uint32_t m, float (&xv)[3]) {
    asm volatile(
        "s_mov_b32 m0, %3\n\ts_nop 0\n\t"
        "ds_read_addtid_b32 %0\n\tds_read_addtid_b32 %1 offset:256\n\t"
        "ds_read_addtid_b32 %2 offset:512"
        : "=&v"(xv[0]), "=&v"(xv[1]), "=&v"(xv[2])
        : "s"(m)
        : "memory");
}
template <>
__device__ __forceinline__ void lds_issue_raw<4>(uint32_t m, float (&xv)[4]) {
    asm volatile(
        "s_mov_b32 m0, %4\n\ts_nop 0\n\t"
        "ds_read_addtid_b32 %0\n\tds_read_addtid_b32 %1 offset:256\n\t"
        "ds_read_addtid_b32 %2 offset:512\n\tds_read_addtid_b32 %3 offset:768"
        : "=&v"(xv[0]), "=&v"(xv[1]), "=&v"(xv[2]), "=&v"(xv[3])
        : "s"(m)
        : "memory");
}
template <int NT>
__device__ __forceinline__ void lds_issue(uint32_t m, float (&xv)[NT]) {
    lds_issue_raw<NT>(lds_checked(m, 256u * NT), xv);
}

// Waits until at most KEEP LDS reads are in flight.  LDS reads complete in
// order, so the reads issued before the last KEEP (xv among them) have
// arrived; xv passes through the statement, so nothing reads it earlier.
template <int KEEP, int NT>
struct LdsWait;
template <int KEEP>
struct LdsWait<KEEP, 1> {
    __device__ __forceinline__ static void run(float (&xv)[1]) {
        asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(xv[0]) : "n"(KEEP) : "memory");
    }
};
template <int KEEP>
struct LdsWait<KEEP, 2> {
    __device__ __forceinline__ static void run(float (&xv)[2]) {
        asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(xv[0]), "+v"(xv[1]) : "n"(KEEP) : "memory");
    }
};
template <int KEEP>
struct LdsWait<KEEP, 3> {
    __device__ __forceinline__ static void run(float (&xv)[3]) {
        asm volatile("s_waitcnt lgkmcnt(%3)" : "+v"(xv[0]), "+v"(xv[1]), "+v"(xv[2]) : "n"(KEEP) : "memory");
    }
};
template <int KEEP>
struct LdsWait<KEEP, 4> {
    __device__ __forceinline__ static void run(float (&xv)[4]) {
        asm volatile("s_waitcnt lgkmcnt(%4)"
                     : "+v"(xv[0]), "+v"(xv[1]), "+v"(xv[2]), "+v"(xv[3])
                     : "n"(KEEP)
                     : "memory");
    }
};
template <int NT, int KEEP>
__device__ __forceinline__ void lds_wait(float (&xv)[NT]) {
    LdsWait<KEEP, NT>::run(xv);
}

// NC tiles (256 bytes apart) at each of P bases sb bytes apart, the first at
// m: P runs of reads under one M0 each, M0 advanced by sb between runs (one
// wait state after every M0 write).  Tiles are numbered base-major.  As for
// lds_tiles, at most NC * P - 4 reads are left in flight on return when
// NC * P > 4 (lds_tiles_rest then waits for the rest).
template <int NC, int P>
__device__ __forceinline__ void lds_multi_raw(uint32_t m, uint32_t sb, float (&xv)[NC * P]);
template <>
__device__ __forceinline__ void lds_multi_raw<1, 4>(uint32_t m, uint32_t sb, float (&xv)[4]) {
    asm volatile(
        "s_mov_b32 m0, %4\n\ts_nop 0\n\tds_read_addtid_b32 %0\n\t"
        "s_add_u32 m0, m0, %5\n\ts_nop 0\n\tds_read_addtid_b32 %1\n\t"
        "s_add_u32 m0, m0, %5\n\ts_nop 0\n\tds_read_addtid_b32 %2\n\t"
        "s_add_u32 m0, m0, %5\n\ts_nop 0\n\tds_read_addtid_b32 %3\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(xv[0]), "=&v"(xv[1]), "=&v"(xv[2]), "=&v"(xv[3])
        : "s"(m), "s"(sb)
        : "memory", "scc");
}
template <>
__device__ __forceinline__ void lds_multi_raw<2, 4>(uint32_t m, uint32_t sb, float (&xv)[8]) {
    asm volatile(
        "s_mov_b32 m0, %8\n\ts_nop 0\n\t"
        "ds_read_addtid_b32 %0\n\tds_read_addtid_b32 %1 offset:256\n\t"
        "s_add_u32 m0, m0, %9\n\ts_nop 0\n\t"
        "ds_read_addtid_b32 %2\n\tds_read_addtid_b32 %3 offset:256\n\t"
        "s_add_u32 m0, m0, %9\n\ts_nop 0\n\t"
        "ds_read_addtid_b32 %4\n\tds_read_addtid_b32 %5 offset:256\n\t"
        "s_add_u32 m0, m0, %9\n\ts_nop 0\n\t"
        "ds_read_addtid_b32 %6\n\tds_read_addtid_b32 %7 offset:256\n\t"
        "s_waitcnt lgkmcnt(4)"
        : "=&v"(xv[0]), "=&v"(xv[1]), "=&v"(xv[2]), "=&v"(xv[3]), "=&v"(xv[4]), "=&v"(xv[5]), "=&v"(xv[6]), "=&v"(xv[7])
        : "s"(m), "s"(sb)
        : "memory", "scc");
}
template <>
__device__ __forceinline__ void lds_multi_raw<3, 2>(uint32_t m, uint32_t sb, float (&xv)[6]) {
    asm volatile(
        "s_mov_b32 m0, %6\n\ts_nop 0\n\t"
        "ds_read_addtid_b32 %0\n\tds_read_addtid_b32 %1 offset:256\n\tds_read_addtid_b32 %2 offset:512\n\t"
        "s_add_u32 m0, m0, %7\n\ts_nop 0\n\t"
        "ds_read_addtid_b32 %3\n\tds_read_addtid_b32 %4 offset:256\n\tds_read_addtid_b32 %5 offset:512\n\t"
        "s_waitcnt lgkmcnt(2)"
        : "=&v"(xv[0]), "=&v"(xv[1]), "=&v"(xv[2]), "=&v"(xv[3]), "=&v"(xv[4]), "=&v"(xv[5])
        : "s"(m), "s"(sb)
        : "memory", "scc");
}
template <>
__device__ __forceinline__ void lds_multi_raw<4, 2>(uint32_t m, uint32_t sb, float (&xv)[8]) {
    asm volatile(
        "s_mov_b32 m0, %8\n\ts_nop 0\n\t"
        "ds_read_addtid_b32 %0\n\tds_read_addtid_b32 %1 offset:256\n\t"
        "ds_read_addtid_b32 %2 offset:512\n\tds_read_addtid_b32 %3 offset:768\n\t"
        "s_add_u32 m0, m0, %9\n\ts_nop 0\n\t"
        "ds_read_addtid_b32 %4\n\tds_read_addtid_b32 %5 offset:256\n\t"
        "ds_read_addtid_b32 %6 offset:512\n\tds_read_addtid_b32 %7 offset:768\n\t"
        "s_waitcnt lgkmcnt(4)"
        : "=&v"(xv[0]), "=&v"(xv[1]), "=&v"(xv[2]), "=&v"(xv[3]), "=&v"(xv[4]), "=&v"(xv[5]), "=&v"(xv[6]), "=&v"(xv[7])
        : "s"(m), "s"(sb)
        : "memory", "scc");
}

namespace {

constexpr int kBlock = 256;       // 4 wavefronts per workgroup
constexpr int kBigBlock = 1024;   // 16 wavefronts share one large staged row
constexpr int64_t kBigLds = 40 * 1024;  // staged rows above this use kBigBlock
constexpr int64_t kRowsLdsBudget = 30 * 1024;  // LDS for the series of one workgroup (5 per CU)
constexpr int kMaxRowsPerBlock = 7;
constexpr int kXcds = 8;          // MI355X: 8 XCDs, workgroups dealt round-robin
constexpr int kTile = rocket::kTile;

struct FusedArgs {
    const float *X;
    float *F;
    int64_t row0;      // first row of this launch (rows are independent)
    int64_t n_rows;    // rows in this launch
    int32_t L;
    int32_t K;
    int32_t nf;        // features per kernel in F: 2 (PPV, MAX) or 3 (+ MPV); 1 for
                       // MINIROCKET, whose K is then its feature count
    int32_t C;         // channels per series
    const float *thr;     // MINIROCKET items: per item [nq][4] thresholds
    const ItemDesc *items;
    const float *wpk;
    const float *bias;
    const int32_t *kid;
    const int32_t *order;
    const int32_t *split_begin;  // n_variants * nsplit + 1 offsets into order
    int32_t nsplit;
    int32_t n_variants;          // variants that have items, launched variant-major
    int32_t variants[rocket::kNumVariants];
    int64_t groups_per_xcd;      // row groups (of rows_per_block series) per XCD
    int32_t halo_lo;
    int32_t row_stride;
    int32_t tail_pad;        // zero floats staged after the last row
    int32_t rows_per_block;  // series staged together in one workgroup's LDS
    int32_t vec4;            // 1: rows are staged with 16-byte loads and LDS writes (L, halo_lo and
                             // row_stride multiples of 4 floats, X 16-byte aligned)
    float *S;                // series-lane layout: features in slot order (see below)
    int64_t s_rows;          // rows one slot column of S holds
    int64_t s_floats;        // floats of S this launch may write (bounds of checked builds)
};

// DPP controls (GFX9 encoding)
constexpr int kDppQuadSwap1 = 0xB1;   // quad_perm(1,0,3,2)
constexpr int kDppQuadSwap2 = 0x4E;   // quad_perm(2,3,0,1)
constexpr int kDppRowHalfMirror = 0x141;
constexpr int kDppRowMirror = 0x140;
constexpr int kDppRowRor8 = 0x128;     // row_ror:8 (lane i of a row reads lane i^8)

// Where a block's series values come from.  m0(j) is the LDS byte address
// of lane 0's value under tap j in the block's first tile; lane l reads 4*l
// bytes further and tile u of the block 256*u bytes further.  channel(off)
// moves to another channel's row (off floats further).
//   PaddedTiles:  the row sits in LDS with zero margins wide enough for
//                 every tap of every real output (and the tail pad after
//                 the last row for the lanes past O), so tap j is d floats
//                 after tap j-1.
//   ClampedTiles: the row sits in LDS with kClampMargin zeros on each side
//                 (long series, whose full margins would not fit).  The
//                 series index of lane 0 under tap j is clamped into
//                 [-kClampMargin, L] on the scalar unit: a block whose
//                 positions all lie left (right) of the series then reads
//                 zeros from the left (right) margin, and a block that
//                 overlaps the series is not moved, so every read stays in
//                 the margins and yields the zero-padded value.
struct PaddedTiles {
    uint32_t base;  // LDS byte address of lane 0's value under tap 0
    int d;
    __device__ __forceinline__ uint32_t m0(int j) const { return base + 4u * (uint32_t)(j * d); }
    __device__ __forceinline__ PaddedTiles channel(int off) const {
        return PaddedTiles{base + 4u * (uint32_t)off, d};
    }
};

struct ClampedTiles {
    uint32_t row;  // LDS byte address of series index 0
    int b0;        // series index under tap 0 of lane 0
    int d;
    int L;
    __device__ __forceinline__ uint32_t m0(int j) const {
        const int b = min(max(b0 + j * d, -rocket::kClampMargin), L);
        return row + 4u * (uint32_t)b;
    }
    __device__ __forceinline__ ClampedTiles channel(int off) const {
        return ClampedTiles{row + 4u * (uint32_t)off, b0, d, L};
    }
};

// The padded layout with each block's series offset clamped to at most L
// (Toeplitz items' last super-tile, whose taps reach up to (sigma - 1) d past
// the other blocks): a block that starts at or past L holds no real output
// that reads a series value, only zero padding, so it reads the zeros at L
// instead and every read stays inside the row's margins and the tail pad.
struct RightClampedTiles {
    uint32_t row;  // LDS byte address of series index 0
    int b0;        // series index under tap 0 of lane 0
    int d;
    int L;
    __device__ __forceinline__ uint32_t m0(int j) const { return row + 4u * (uint32_t)min(b0 + j * d, L); }
};

// The reads of lds_multi_raw, every run's address checked in checked
// builds (a failed run sends every run to the start of the staged bytes).
template <int NC, int P>
__device__ __forceinline__ void lds_multi(uint32_t m, uint32_t sb, float (&xv)[NC * P]) {
#if ROCKET_CHECKED
    bool ok = true;
#pragma unroll
    for (int k = 0; k < P; ++k) ok = ok && lds_checked(m + (uint32_t)k * sb, 256u * NC) == m + (uint32_t)k * sb;
    if (!ok) {
        m = g_check_lds_lo;
        sb = 0;
    }
    m = __builtin_amdgcn_readfirstlane(m);
    sb = __builtin_amdgcn_readfirstlane(sb);
#endif
    lds_multi_raw<NC, P>(m, sb, xv);
}

// The padded layout for P runs of NC tiles each, run k sb bytes after run 0
// (P super-tiles of a Toeplitz item whose super-tiles hold NC chunks): tile
// u is chunk u % NC of run u / NC.
template <int NC, int P>
struct MultiTiles {
    uint32_t base;  // LDS byte address of lane 0's value under tap 0, run 0
    int d;
    uint32_t sb;    // bytes from one run to the next
    __device__ __forceinline__ uint32_t m0(int j) const { return base + 4u * (uint32_t)(j * d); }
};

// How the tiles of one block group: 0 for one run (the block's last tile is
// the row's or super-tile's last), NC for MultiTiles (every run's last
// tile is its super-tile's last chunk).
template <typename Src>
struct TileRuns {
    static constexpr int nc = 0;
};
template <int NC, int P>
struct TileRuns<MultiTiles<NC, P>> {
    static constexpr int nc = NC;
};
__device__ constexpr bool run_last(int u, int nt, int nc) { return nc ? (u % nc == nc - 1) : (u == nt - 1); }

// The series values of a block's tiles under tap j.
template <int NT, typename Src>
__device__ __forceinline__ void read_tiles(const Src &src, int j, float (&xv)[NT]) {
    lds_tiles<NT>(src.m0(j), xv);
}

// Sources whose next tap's reads tile_mfma issues before the current tap's
// MFMAs (blocks of up to 4 tiles).  Only the series-lane reads: in the
// fused kernel the second set of tile registers lowers the occupancy from 5
// to 4 wavefronts per SIMD (100-thousand-series calls 2.2 % slower), while
// the series-lane kernel keeps its register count (a million 64-sample
// series: 0.4 % faster).
template <typename Src>
struct PipelinedReads {
    static constexpr bool value = false;
};
template <int NT, int NC, int P>
__device__ __forceinline__ void read_tiles(const MultiTiles<NC, P> &src, int j, float (&xv)[NT]) {
    static_assert(NT == NC * P, "one block reads all of its runs");
    lds_multi<NC, P>(src.m0(j), src.sb, xv);
}

// Per-series accumulators of one work item, per lane and kernel slot: the
// running max, the positive count (wavefront-uniform, scalar registers) and,
// when MPV is computed, the sum of the positive values.
template <int G>
struct RowAcc {
    v4f mx[G];
    uint32_t cnt[G][4];
    v4f ps[G];
};

// Multichannel items (Sec. 3.3): where the item's weights and channel rows
// are.  w is the lane's first packed weight (slot lane & 3); the weights of
// the item's ci-th channel, group g, tap j are at w[((ci*G + g)*ELL + j)*4].
// The channels are the set bits of mask, in ascending order; the row of
// channel c sits c*cstride floats after the series' first row.
struct McCtx {
    const float *w;
    uint64_t mask;
    int n_ch;
    int cstride;
};

// One channel's A-operand weights of a multichannel item (wp: its first).
template <int ELL, int G>
__device__ __forceinline__ void load_channel_weights(const float *wp, float (&wc)[G][ELL]) {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int j = 0; j < ELL; ++j) wc[g][j] = wp[(g * ELL + j) * 4];
}

// The contraction of one block of NT tiles over the taps of one channel:
// tap j of every tile and kernel group is issued before tap j+1, so the
// wavefront keeps NT*G independent MFMA accumulation chains in flight.  With
// FIRST set each chain starts from its start value (the slots' biases, or,
// in the last tile of a row, -inf on lanes past the last output); without
// it the chains continue from acc (the next channel of a multichannel item).
template <int ELL, int G, int NT, bool LAST, bool FIRST, typename Src>
__device__ __forceinline__ void tile_mfma(const Src &src, const float (&wa)[G][ELL],
                                          const v4f (&binit)[G], const v4f (&blast)[G],
                                          v4f (&acc)[NT][G]) {
    if constexpr (NT <= 4 && PipelinedReads<Src>::value) {
        // tap j + 1's reads are in flight while tap j's MFMAs issue
        float xv[2][NT];
        lds_issue<NT>(src.m0(0), xv[0]);
#pragma unroll
        for (int j = 0; j < ELL; ++j) {
            if (j + 1 < ELL) {
                lds_issue<NT>(src.m0(j + 1), xv[(j + 1) & 1]);
                lds_wait<NT, NT>(xv[j & 1]);
            } else {
                lds_wait<NT, 0>(xv[j & 1]);
            }
#pragma unroll
            for (int u = 0; u < NT; ++u)
#pragma unroll
                for (int g = 0; g < G; ++g) {
                    const v4f c = (FIRST && j == 0)
                                      ? ((LAST && run_last(u, NT, TileRuns<Src>::nc)) ? blast[g] : binit[g])
                                      : acc[u][g];
                    acc[u][g] = __builtin_amdgcn_mfma_f32_4x4x1f32(wa[g][j], xv[j & 1][u], c, 0, 0, 0);
                }
        }
        return;
    }
#pragma unroll
    for (int j = 0; j < ELL; ++j) {
        float xv[NT];
        read_tiles<NT>(src, j, xv);
        constexpr int NA = NT > 4 ? 4 : NT;  // tiles ready after lds_tiles
#pragma unroll
        for (int u = 0; u < NT; ++u) {
            if (NT > 4 && u == NA) {
                // tiles 4..: wait for the rest of the reads only now, after
                // the MFMAs of tiles 0-3 (the barriers keep this order)
                __builtin_amdgcn_sched_barrier(0);
                if constexpr (NT > 4) lds_tiles_rest<NT>(xv);
            }
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const v4f c = (FIRST && j == 0)
                                  ? ((LAST && run_last(u, NT, TileRuns<Src>::nc)) ? blast[g] : binit[g])
                                  : acc[u][g];
                acc[u][g] = __builtin_amdgcn_mfma_f32_4x4x1f32(wa[g][j], xv[u], c, 0, 0, 0);
            }
        }
        if (NT > 4) __builtin_amdgcn_sched_barrier(0);
    }
}

// Fold NT tiles of finished dot products into the row accumulators.  A chain
// started at -inf stays -inf, so MAX folds every result (v_max3 over pairs of
// tiles), the positive count is a ballot of y > 0 popcounted on the scalar
// unit, and the MPV numerator adds max(y, 0).
template <int G, int NT, bool MPV>
__device__ __forceinline__ void block_reduce(const v4f (&acc)[NT][G], RowAcc<G> &ra) {
#pragma unroll
    for (int u = 0; u < NT; ++u)
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                ra.cnt[g][v] += (uint32_t)__popcll(__builtin_amdgcn_ballot_w64(acc[u][g][v] > 0.0f));
    if (MPV) {
#pragma unroll
        for (int u = 0; u < NT; ++u)
#pragma unroll
            for (int g = 0; g < G; ++g)
#pragma unroll
                for (int v = 0; v < 4; ++v) ra.ps[g][v] += fmaxf(acc[u][g][v], 0.0f);
    }
#pragma unroll
    for (int u = 0; u + 1 < NT; u += 2)
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                ra.mx[g][v] = fmaxf(fmaxf(ra.mx[g][v], acc[u][g][v]), acc[u + 1][g][v]);
    if (NT % 2 == 1) {
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int v = 0; v < 4; ++v) ra.mx[g][v] = fmaxf(ra.mx[g][v], acc[NT - 1][g][v]);
    }
}

// One block of NT tiles.  Univariate items keep their weights in registers
// (wa); multichannel items (MC) run the MFMA chains over every channel of
// their mask, reading each channel's weights in turn: the next channel's
// weights are loaded while the current channel's MFMAs run, and the channel
// numbers come from the mask (s_ff1) without a memory access.  The scheduling
// barriers keep the block's MFMAs in one run and its reduction in another:
// on gfx950 fp32 MFMA and VALU instructions of a SIMD do not execute at the
// same time, and a VALU instruction placed between two MFMAs of a wavefront
// costs more than the same instruction in a run of VALU work.
template <int ELL, int G, int NT, bool LAST, bool MPV, bool MC, typename Src>
__device__ __forceinline__ void tile_block(const Src &src, const float (&wa)[G][ELL],
                                           const McCtx &mc, const v4f (&binit)[G],
                                           const v4f (&blast)[G], RowAcc<G> &ra) {
    v4f acc[NT][G];
    if constexpr (!MC) {
        tile_mfma<ELL, G, NT, LAST, true>(src, wa, binit, blast, acc);
    } else {
        float wc[G][ELL], wn[G][ELL];
        uint64_t m = mc.mask;
        int c = (int)__builtin_ctzll(m);
        m &= m - 1;
        load_channel_weights<ELL, G>(mc.w, wc);
        for (int ci = 0; ci < mc.n_ch; ++ci) {
            int cn = 0;
            if (ci + 1 < mc.n_ch) {
                load_channel_weights<ELL, G>(mc.w + (ci + 1) * (G * ELL * 4), wn);
                cn = (int)__builtin_ctzll(m);
                m &= m - 1;
            }
            const Src s = src.channel(c * mc.cstride);
            if (ci == 0)
                tile_mfma<ELL, G, NT, LAST, true>(s, wc, binit, blast, acc);
            else
                tile_mfma<ELL, G, NT, LAST, false>(s, wc, binit, blast, acc);
#pragma unroll
            for (int g = 0; g < G; ++g)
#pragma unroll
                for (int j = 0; j < ELL; ++j) wc[g][j] = wn[g][j];
            c = cn;
        }
    }
    __builtin_amdgcn_sched_barrier(0);
    // raised wave priority while the reduction runs: a wavefront that has
    // finished its MFMAs gets its vector work issued first (measured: 0.4 %
    // faster passes over 100,000 series of 1,000 samples, 0.7 % faster long
    // series; same results)
    __builtin_amdgcn_s_setprio(1);
    block_reduce<G, NT, MPV>(acc, ra);
    __builtin_amdgcn_s_setprio(0);
}

// The last block of a row: its tile count nv (1..N) selects a code copy.
// (LASTB false: a block of nv tiles whose last tile is not the row's last.)
template <int ELL, int G, int N, bool MPV, bool MC, typename Src, bool LASTB = true>
struct TailTiles {
    __device__ __forceinline__ static void run(int nv, const Src &src, const float (&wa)[G][ELL],
                                               const McCtx &mc, const v4f (&binit)[G],
                                               const v4f (&blast)[G], RowAcc<G> &ra) {
        if (nv == N)
            tile_block<ELL, G, N, LASTB, MPV, MC>(src, wa, mc, binit, blast, ra);
        else
            TailTiles<ELL, G, N - 1, MPV, MC, Src, LASTB>::run(nv, src, wa, mc, binit, blast, ra);
    }
};

template <int ELL, int G, bool MPV, bool MC, typename Src, bool LASTB>
struct TailTiles<ELL, G, 0, MPV, MC, Src, LASTB> {
    __device__ __forceinline__ static void run(int, const Src &, const float (&)[G][ELL],
                                               const McCtx &, const v4f (&)[G], const v4f (&)[G],
                                               RowAcc<G> &) {}
};

// The last block of a row and then the row's epilogue, a code copy per
// tile count nv (1..N): each copy reduces and writes the features from the
// registers its own block left the accumulators in (one epilogue after the
// copies would first have to move them into common registers).
template <int ELL, int G, int N, bool MPV, bool MC, typename Src>
struct TailTilesThen {
    template <typename Epi>
    __device__ __forceinline__ static void run(int nv, const Src &src, const float (&wa)[G][ELL],
                                               const McCtx &mc, const v4f (&binit)[G],
                                               const v4f (&blast)[G], RowAcc<G> &ra, const Epi &epi) {
        if (nv == N) {
            tile_block<ELL, G, N, true, MPV, MC>(src, wa, mc, binit, blast, ra);
            epi(ra);
        } else {
            TailTilesThen<ELL, G, N - 1, MPV, MC, Src>::run(nv, src, wa, mc, binit, blast, ra, epi);
        }
    }
};
template <int ELL, int G, bool MPV, bool MC, typename Src>
struct TailTilesThen<ELL, G, 0, MPV, MC, Src> {
    template <typename Epi>
    __device__ __forceinline__ static void run(int, const Src &, const float (&)[G][ELL], const McCtx &,
                                               const v4f (&)[G], const v4f (&)[G], RowAcc<G> &, const Epi &) {}
};

// Combining operations of the wavefront reductions: max for MAX, sum for
// the MPV numerator.
struct OpMax {
    __device__ __forceinline__ static float f(float a, float b) { return fmaxf(a, b); }
};
struct OpSum {
    __device__ __forceinline__ static float f(float a, float b) { return a + b; }
};

template <typename Op, int CTRL>
__device__ __forceinline__ float dpp_row_step(float v) {
    // every lane of a full row reads a valid lane for these controls, so the
    // move can fold into the combining instruction's DPP source
    const int moved = __builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, true);
    return Op::f(v, __int_as_float(moved));
}

// Lane-wise combination of two registers after swapping the upper 32 lanes
// of a with the lower 32 lanes of b: lanes 0-31 then reduce a over lane pairs
// (i, i+32), lanes 32-63 reduce b.
template <typename Op>
__device__ __forceinline__ float fold32(float a, float b) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(a), __float_as_uint(b), false,
                                                    false);
    return Op::f(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// The same with 16-lane rows: odd rows of a swap with even rows of b, so
// rows 0 and 2 of the result reduce a over row pairs, rows 1 and 3 reduce b.
template <typename Op>
__device__ __forceinline__ float fold16(float a, float b) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false,
                                                    false);
    return Op::f(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

// Reduction within each 16-lane row, broadcast to the row.
template <typename Op>
__device__ __forceinline__ float row_reduce(float v) {
    v = dpp_row_step<Op, kDppQuadSwap1>(v);
    v = dpp_row_step<Op, kDppQuadSwap2>(v);
    v = dpp_row_step<Op, kDppRowHalfMirror>(v);
    v = dpp_row_step<Op, kDppRowMirror>(v);
    return v;
}

// Reduce the 4 slot values of one group over the wavefront: on return, the
// lanes of 16-lane row q hold the result of slot slot_of_row(q).
template <typename Op>
__device__ __forceinline__ float reduce4(const v4f &m) {
    return row_reduce<Op>(fold16<Op>(fold32<Op>(m[0], m[1]), fold32<Op>(m[2], m[3])));
}
// fold32(m0, m1): lanes 0-31 slot 0, lanes 32-63 slot 1; fold16 of
// (slot0|slot1) and (slot2|slot3): row 0 slot 0, row 1 slot 2, row 2 slot 1,
// row 3 slot 3.
__device__ constexpr int slot_of_row(int q) { return ((q & 1) << 1) | (q >> 1); }

// The same for the 8 slots of two groups at once: after the 32- and 16-lane
// folds of each group, the two 16-lane rows q of the groups fold over lane
// pairs (i, i+8) into one register (lanes 0-7 of the row keep group 0,
// lanes 8-15 group 1), and three DPP steps finish each 8-lane half-row.  On
// return the lanes 16q + 8h .. 16q + 8h + 7 hold slot slot_of_row(q) of
// group h.  18 vector instructions for 8 slots, against 20 for two reduce4.
template <typename Op>
__device__ __forceinline__ float reduce8(const v4f &m0, const v4f &m1, bool hi8) {
    const float e = fold16<Op>(fold32<Op>(m0[0], m0[1]), fold32<Op>(m0[2], m0[3]));
    const float h = fold16<Op>(fold32<Op>(m1[0], m1[1]), fold32<Op>(m1[2], m1[3]));
    const float re = dpp_row_step<Op, kDppRowRor8>(e);
    const float rh = dpp_row_step<Op, kDppRowRor8>(h);
    float v = hi8 ? rh : re;
    v = dpp_row_step<Op, kDppQuadSwap1>(v);
    v = dpp_row_step<Op, kDppQuadSwap2>(v);
    return dpp_row_step<Op, kDppRowHalfMirror>(v);
}

// The writer lane of a kernel slot after the wavefront reduction (-1: the
// lane writes nothing): lane 16q writes slot slot_of_row(q) of a 4-kernel
// item; lane 16q + 8h writes slot slot_of_row(q) of group h of an 8-kernel
// item.  Returns the slot index 4h + v, or -1.
template <int G>
__device__ __forceinline__ int writer_slot(int lane) {
    if (G == 1) return (lane & 15) == 0 ? slot_of_row(lane >> 4) : -1;
    return (lane & 7) == 0 ? 4 * ((lane >> 3) & 1) + slot_of_row(lane >> 4) : -1;
}

template <int G, bool MPV>
__device__ __forceinline__ void init_row(RowAcc<G> &ra) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
        // -inf into the four running maxima with two 64-bit moves
        v2f lo, hi;
        asm volatile("v_mov_b64 %0, %2\n\tv_mov_b64 %1, %2" : "=v"(lo), "=v"(hi) : "s"(kNegInfPair));
        ra.mx[g] = v4f{lo[0], lo[1], hi[0], hi[1]};
        if (MPV) ra.ps[g] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int v = 0; v < 4; ++v) ra.cnt[g][v] = 0;
    }
}

// One kernel's features from its writer lane: PPV = c / O, MAX, and MPV.
template <bool MPV>
__device__ __forceinline__ void write_features(uint32_t c, float m, float psum, int ok, double inv_O,
                                               float *Frow) {
    // (float)c / (float)O, correctly rounded: for c <= O < 2^24 the quotient
    // is never a float midpoint and lies at least 2^-49 (relative) from one,
    // while c * fl64(1/O) is within 2^-52 of it, so rounding the double
    // product to float gives the same float as the fp32 division
    const float ppv = (float)((double)c * inv_O);
    if (!store_checked(Frow + (MPV ? 3 : 2) * (int64_t)ok, MPV ? 3 : 2)) return;
    if (MPV) {
        // rows of 3 floats: 4-byte aligned only
        float *f = Frow + 3 * (int64_t)ok;
        f[0] = ppv;
        f[1] = m;
        f[2] = c > 0 ? psum / (float)c : 0.0f;
    } else {
        float2 res;
        res.x = ppv;
        res.y = m;
        *reinterpret_cast<float2 *>(Frow + 2 * (int64_t)ok) = res;
    }
}

// MAX (and the MPV numerator) over the wavefront (counts are already
// scalar), then per kernel {PPV, MAX} (or {PPV, MAX, MPV}), written by the
// writer lanes (writer_slot); okid is the kernel id the lane writes, or -1.
template <int G, bool MPV>
__device__ __forceinline__ void write_row(const RowAcc<G> &ra, int okid, double inv_O, float *Frow,
                                          bool hi8) {
    if constexpr (G == 1) {
        const float m = reduce4<OpMax>(ra.mx[0]);
        const float psum = MPV ? reduce4<OpSum>(ra.ps[0]) : 0.0f;
        // the count of slot slot_of_row(q) into writer lane 16q (scalar to
        // lane moves: one instruction each, no lane masks)
        uint32_t c;
        asm volatile(
            "v_writelane_b32 %0, %1, 0\n\t"
            "v_writelane_b32 %0, %2, 16\n\t"
            "v_writelane_b32 %0, %3, 32\n\t"
            "v_writelane_b32 %0, %4, 48"
            : "=&v"(c)
            : "s"(ra.cnt[0][slot_of_row(0)]), "s"(ra.cnt[0][slot_of_row(1)]), "s"(ra.cnt[0][slot_of_row(2)]),
              "s"(ra.cnt[0][slot_of_row(3)]));
        if (okid >= 0) write_features<MPV>(c, m, psum, okid, inv_O, Frow);
    } else {
        const float m = reduce8<OpMax>(ra.mx[0], ra.mx[1], hi8);
        const float psum = MPV ? reduce8<OpSum>(ra.ps[0], ra.ps[1], hi8) : 0.0f;
        // the count of slot slot_of_row(q) of group h into lane 16q + 8h
        uint32_t c;
        asm volatile(
            "v_writelane_b32 %0, %1, 0\n\t"
            "v_writelane_b32 %0, %2, 8\n\t"
            "v_writelane_b32 %0, %3, 16\n\t"
            "v_writelane_b32 %0, %4, 24\n\t"
            "v_writelane_b32 %0, %5, 32\n\t"
            "v_writelane_b32 %0, %6, 40\n\t"
            "v_writelane_b32 %0, %7, 48\n\t"
            "v_writelane_b32 %0, %8, 56"
            : "=&v"(c)
            : "s"(ra.cnt[0][slot_of_row(0)]), "s"(ra.cnt[1][slot_of_row(0)]), "s"(ra.cnt[0][slot_of_row(1)]),
              "s"(ra.cnt[1][slot_of_row(1)]), "s"(ra.cnt[0][slot_of_row(2)]), "s"(ra.cnt[1][slot_of_row(2)]),
              "s"(ra.cnt[0][slot_of_row(3)]), "s"(ra.cnt[1][slot_of_row(3)]));
        if (okid >= 0) write_features<MPV>(c, m, psum, okid, inv_O, Frow);
    }
}

// The row epilogue of run_item as a function object (write_row with the
// item's writer lane, 1/O and the row's F pointer).
template <int G, bool MPV>
struct RowWriter {
    int okid;
    double inv_O;
    float *Frow;
    bool hi8;
    __device__ __forceinline__ void operator()(const RowAcc<G> &ra) const {
        write_row<G, MPV>(ra, okid, inv_O, Frow, hi8);
    }
};

// One work item over the `nrows` series staged in LDS: the item's weights
// are loaded once and reused for every series.  Each series runs the item's
// tiles in blocks of NT (the last block holds the remaining 1..NT tiles).
template <int ELL, int G, bool CLAMP, bool MPV, bool MC>
__device__ __forceinline__ void run_item(const ItemDesc &it, const float *rows0, int nrows,
                                         const FusedArgs &a, float *F0, int lane) {
    constexpr int NT = rocket::kTilesPerBlock[G - 1];
    // A operand: lane holds the weight of kernel slot (lane & 3) for every
    // tap; univariate items keep them in registers for the whole item,
    // multichannel ones read each channel's weights per block (McCtx)
    float wa[G][ELL];
    if constexpr (!MC) {
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int j = 0; j < ELL; ++j) wa[g][j] = a.wpk[it.w_off + (g * ELL + j) * 4 + (lane & 3)];
    }
    McCtx mc{};
    if constexpr (MC)
        mc = McCtx{a.wpk + it.w_off + (lane & 3), ((uint64_t)it.ch_mask[1] << 32) | it.ch_mask[0], it.n_ch,
                   a.row_stride};
    const int row_pitch = a.C * a.row_stride;  // floats per staged series (LDS offsets fit 32 bits)
    // C operand of the first tap: the bias of block row v (kernel slot v),
    // and in the last tile of a series -inf on the lanes past the last
    // output, so that they change no feature
    const int rem = it.O - (it.n_tiles - 1) * kTile;  // real outputs in the last tile, 1..64
    v4f binit[G], blast[G];
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const float b = as_const(a.bias)[it.k_off + 4 * g + v];
            // copied into a vector register once per item (an opaque copy,
            // so the compiler keeps it there instead of copying the scalar
            // bias again before every block)
            float bv;
            asm volatile("v_mov_b32 %0, %1" : "=v"(bv) : "s"(b));
            binit[g][v] = bv;
            blast[g][v] = lane < rem ? bv : -INFINITY;
        }
    const int nfull = (it.n_tiles - 1) / NT;  // full blocks before the last block
    const int nv = it.n_tiles - nfull * NT;   // tiles in the last block, 1..NT
    // the kernel id this lane writes after the reduction (-1: not a writer,
    // or an empty slot)
    const int wslot = writer_slot<G>(lane);
    const int okid = wslot >= 0 ? a.kid[it.k_off + wslot] : -1;
    const bool hi8 = (lane & 8) != 0;
    const int64_t f_stride = (int64_t)a.nf * a.K;
    for (int r = 0; r < nrows; ++r) {
        RowAcc<G> ra;
        init_row<G, MPV>(ra);
        const uint32_t row = lds_addr(rows0 + r * row_pitch);  // series index 0
        // block b starts at output b*NT*64; its lane 0 reads series index
        // b*NT*64 - p under tap 0 (a wavefront-uniform offset)
        for (int blk = 0; blk < nfull; ++blk) {
            const int b0 = blk * (NT * kTile) - it.p;
            if constexpr (CLAMP)
                tile_block<ELL, G, NT, false, MPV, MC>(ClampedTiles{row, b0, it.d, a.L}, wa, mc, binit,
                                                       blast, ra);
            else
                tile_block<ELL, G, NT, false, MPV, MC>(PaddedTiles{row + 4u * (uint32_t)b0, it.d}, wa,
                                                       mc, binit, blast, ra);
        }
        const int b0 = nfull * (NT * kTile) - it.p;
        const RowWriter<G, MPV> epi{okid, it.inv_O, F0 + r * f_stride, hi8};
        if constexpr (CLAMP)
            TailTilesThen<ELL, G, NT, MPV, MC, ClampedTiles>::run(nv, ClampedTiles{row, b0, it.d, a.L}, wa, mc,
                                                                  binit, blast, ra, epi);
        else
            TailTilesThen<ELL, G, NT, MPV, MC, PaddedTiles>::run(
                nv, PaddedTiles{row + 4u * (uint32_t)b0, it.d}, wa, mc, binit, blast, ra, epi);
    }
}

__device__ __forceinline__ ItemDesc load_item(ConstPtr<ItemDesc> p) {
    ItemDesc it;
    it.variant = p->variant;
    it.d = p->d;
    it.p = p->p;
    it.O = p->O;
    it.n_tiles = p->n_tiles;
    it.w_off = p->w_off;
    it.k_off = p->k_off;
    it.cost = p->cost;
    it.n_ch = p->n_ch;
    it.ch_off = p->ch_off;
    it.t_off = p->t_off;
    it.nq = p->nq;
    it.ch_mask[0] = p->ch_mask[0];
    it.ch_mask[1] = p->ch_mask[1];
    it.inv_O = p->inv_O;
    return it;
}

// Items of one variant, taken one at a time from the workgroup's counter.
template <int ELL, int G, bool CLAMP, bool MPV, bool MC>
__device__ __forceinline__ void run_items(int *next_item, int beg, int cnt_items,
                                          const float *rows0, int nrows, const FusedArgs &a,
                                          float *F0, int lane) {
    while (true) {
        int idx = 0;
        if (lane == 0) idx = atomicAdd(next_item, 1);
        idx = __builtin_amdgcn_readfirstlane(__shfl(idx, 0, 64));
        if (idx >= cnt_items) break;
        const ItemDesc it = load_item(as_const(a.items) + as_const(a.order)[beg + idx]);
        run_item<ELL, G, CLAMP, MPV, MC>(it, rows0, nrows, a, F0, lane);
    }
}

// What one workgroup does: a row group, one variant, one split of its items.
// ---------------------------------------------------------------------------
// VALU items: the one or two kernels left over in a bucket of a long-series
// plan.  A 4-slot MFMA group would run them with 3 or 2 empty slots, and
// each empty slot still costs its share of the MFMA and of the reduction; on
// the VALU each kernel costs one fp32 FMA per tap and tile (4.5 cycles
// against 8.7 for the 4-slot MFMA) and one result register to reduce.  The
// tiles, blocks (8 tiles), series reads and the -inf start of lanes past O
// are those of a one-group MFMA item; the weights and biases are scalars.
// ---------------------------------------------------------------------------

template <int NK>
struct ValuAcc {
    float mx[NK];
    uint32_t cnt[NK];
    float ps[NK];
};

template <int ELL, int NK, int NT, bool LAST, bool MPV, typename Src>
__device__ __forceinline__ void valu_block(const Src &src, const float (&w)[NK][ELL], const float (&binit)[NK],
                                           const float (&blast)[NK], ValuAcc<NK> &va) {
    float acc[NT][NK];
#pragma unroll
    for (int j = 0; j < ELL; ++j) {
        float xv[NT];
        lds_tiles<NT>(src.m0(j), xv);
        if constexpr (NT > 4) lds_tiles_rest<NT>(xv);
#pragma unroll
        for (int u = 0; u < NT; ++u)
#pragma unroll
            for (int c = 0; c < NK; ++c) {
                const float a0 = (j == 0) ? ((LAST && u == NT - 1) ? blast[c] : binit[c]) : acc[u][c];
                acc[u][c] = fmaf(w[c][j], xv[u], a0);
            }
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < NT; ++u)
#pragma unroll
        for (int c = 0; c < NK; ++c) va.cnt[c] += (uint32_t)__popcll(__builtin_amdgcn_ballot_w64(acc[u][c] > 0.0f));
    if (MPV) {
#pragma unroll
        for (int u = 0; u < NT; ++u)
#pragma unroll
            for (int c = 0; c < NK; ++c) va.ps[c] += fmaxf(acc[u][c], 0.0f);
    }
#pragma unroll
    for (int u = 0; u + 1 < NT; u += 2)
#pragma unroll
        for (int c = 0; c < NK; ++c) va.mx[c] = fmaxf(fmaxf(va.mx[c], acc[u][c]), acc[u + 1][c]);
    if (NT % 2 == 1) {
#pragma unroll
        for (int c = 0; c < NK; ++c) va.mx[c] = fmaxf(va.mx[c], acc[NT - 1][c]);
    }
}

template <int ELL, int NK, int N, bool MPV, typename Src>
struct ValuTail {
    __device__ __forceinline__ static void run(int nv, const Src &src, const float (&w)[NK][ELL],
                                               const float (&binit)[NK], const float (&blast)[NK],
                                               ValuAcc<NK> &va) {
        if (nv == N)
            valu_block<ELL, NK, N, true, MPV>(src, w, binit, blast, va);
        else
            ValuTail<ELL, NK, N - 1, MPV, Src>::run(nv, src, w, binit, blast, va);
    }
};
template <int ELL, int NK, bool MPV, typename Src>
struct ValuTail<ELL, NK, 0, MPV, Src> {
    __device__ __forceinline__ static void run(int, const Src &, const float (&)[NK][ELL], const float (&)[NK],
                                               const float (&)[NK], ValuAcc<NK> &) {}
};

// Combine over the whole wavefront (every lane gets the result).
template <typename Op>
__device__ __forceinline__ float wave_all(float v) {
    return row_reduce<Op>(fold16<Op>(fold32<Op>(v, v), fold32<Op>(v, v)));
}

template <int ELL, int NK, bool CLAMP, bool MPV>
__device__ __forceinline__ void run_valu_item(const ItemDesc &it, const float *rows0, int nrows, const FusedArgs &a,
                                              float *F0, int lane) {
    constexpr int NT = rocket::kTilesPerBlock[0];
    // weights and biases are the same on every lane: scalar registers
    float w[NK][ELL], binit[NK], blast[NK];
    const int rem = it.O - (it.n_tiles - 1) * kTile;
#pragma unroll
    for (int c = 0; c < NK; ++c) {
#pragma unroll
        for (int j = 0; j < ELL; ++j) w[c][j] = as_const(a.wpk)[it.w_off + j * 4 + c];
        const float b = as_const(a.bias)[it.k_off + c];
        float bv;
        asm volatile("v_mov_b32 %0, %1" : "=v"(bv) : "s"(b));
        binit[c] = bv;
        blast[c] = lane < rem ? bv : -INFINITY;
    }
    int kid[NK];
#pragma unroll
    for (int c = 0; c < NK; ++c) kid[c] = as_const(a.kid)[it.k_off + c];
    const int row_pitch = a.C * a.row_stride;
    const int nfull = (it.n_tiles - 1) / NT;
    const int nv = it.n_tiles - nfull * NT;
    const int64_t f_stride = (int64_t)a.nf * a.K;
    for (int r = 0; r < nrows; ++r) {
        ValuAcc<NK> va;
#pragma unroll
        for (int c = 0; c < NK; ++c) {
            va.mx[c] = -INFINITY;
            va.cnt[c] = 0;
            va.ps[c] = 0.0f;
        }
        const uint32_t row = lds_addr(rows0 + r * row_pitch);
        for (int blk = 0; blk < nfull; ++blk) {
            const int b0 = blk * (NT * kTile) - it.p;
            if constexpr (CLAMP)
                valu_block<ELL, NK, NT, false, MPV>(ClampedTiles{row, b0, it.d, a.L}, w, binit, blast, va);
            else
                valu_block<ELL, NK, NT, false, MPV>(PaddedTiles{row + 4u * (uint32_t)b0, it.d}, w, binit, blast, va);
        }
        const int b0 = nfull * (NT * kTile) - it.p;
        if constexpr (CLAMP)
            ValuTail<ELL, NK, NT, MPV, ClampedTiles>::run(nv, ClampedTiles{row, b0, it.d, a.L}, w, binit, blast, va);
        else
            ValuTail<ELL, NK, NT, MPV, PaddedTiles>::run(nv, PaddedTiles{row + 4u * (uint32_t)b0, it.d}, w, binit,
                                                         blast, va);
        float m[NK], psum[NK];
#pragma unroll
        for (int c = 0; c < NK; ++c) {
            m[c] = wave_all<OpMax>(va.mx[c]);
            psum[c] = MPV ? wave_all<OpSum>(va.ps[c]) : 0.0f;
        }
        if (lane == 0) {
#pragma unroll
            for (int c = 0; c < NK; ++c)
                write_features<MPV>(va.cnt[c], m[c], psum[c], kid[c], it.inv_O, F0 + r * f_stride);
        }
    }
}

template <int ELL, int NK, bool CLAMP, bool MPV>
__device__ __forceinline__ void run_valu_items(int *next_item, int beg, int cnt_items, const float *rows0, int nrows,
                                               const FusedArgs &a, float *F0, int lane) {
    while (true) {
        int idx = 0;
        if (lane == 0) idx = atomicAdd(next_item, 1);
        idx = __builtin_amdgcn_readfirstlane(__shfl(idx, 0, 64));
        if (idx >= cnt_items) break;
        const ItemDesc it = load_item(as_const(a.items) + as_const(a.order)[beg + idx]);
        run_valu_item<ELL, NK, CLAMP, MPV>(it, rows0, nrows, a, F0, lane);
    }
}

// ---------------------------------------------------------------------------
// Toeplitz items: the one (NK = 1) or two (NK = 2) kernels left over in a
// bucket at a large dilation d.  The 4 slots of one MFMA group hold the same
// kernel at SIGMA = 4 / NK shifts: slot s is kernel s / SIGMA shifted by
// h = s % SIGMA taps (weight w[m - h] at tap m, ELL + SIGMA - 1 taps), so the
// MFMA chain of lane l reading series index t0 - p + m d + l at tap m
// computes, in slot s, the output at position t0 + l + h d.  Outputs come in
// super-tiles of SIGMA d consecutive positions per kernel: ceil(d / 64)
// chunks at t0 = T + 64 c cover positions T .. T + d - 1 for shift 0 and the
// same plus h d for shift h; lanes with 64 c + l >= d (the last chunk) start
// from -inf, as lanes past O do in an MFMA item's last tile.  The last,
// partial super-tile masks each slot on its own (positions below O) and, in
// the padded layout, clamps its block offsets to at most L (its taps reach
// past the row's margin; see RightClampedTiles).  One
// MFMA chain of ELL + SIGMA - 1 taps thus yields 4 x 64 outputs, where a
// VALU item spends ELL fp32 FMAs per 64 outputs and kernel.
// ---------------------------------------------------------------------------
// Whole super-tiles of NC chunks, P per block (padded rows): the block's
// tiles are the NC chunks of each of P consecutive super-tiles, each
// super-tile's last chunk starting from blast.  Returns the super-tiles
// done, a multiple of P; the caller runs the rest one per block.
template <int TAPS, int NC, int P, bool MPV>
__device__ __forceinline__ int toep_runs(uint32_t row, int p, int d, int span, int s_full,
                                         const float (&wa)[1][TAPS], const v4f (&binit)[1],
                                         const v4f (&blast)[1], RowAcc<1> &ra) {
    const McCtx mc{};
    const int groups = s_full / P;
    const uint32_t sb = 4u * (uint32_t)span;
    for (int gi = 0; gi < groups; ++gi) {
        const int b0 = gi * P * span - p;
        tile_block<TAPS, 1, NC * P, true, MPV, false>(MultiTiles<NC, P>{row + 4u * (uint32_t)b0, d, sb}, wa, mc,
                                                       binit, blast, ra);
    }
    return groups * P;
}

template <int ELL, int NK, bool CLAMP, bool MPV>
__device__ __forceinline__ void run_toep_item(const ItemDesc &it, const float *rows0, int nrows,
                                              const FusedArgs &a, float *F0, int lane) {
    constexpr int SIGMA = 4 / NK;
    constexpr int TAPS = ELL + SIGMA - 1;
    constexpr int NT = rocket::kTilesPerBlock[0];
    float wa[1][TAPS];
#pragma unroll
    for (int j = 0; j < TAPS; ++j) wa[0][j] = a.wpk[it.w_off + j * 4 + (lane & 3)];
    const int d = it.d;
    const int nc = it.n_tiles;                // chunks per super-tile
    const int remc = d - (nc - 1) * kTile;    // positions of a super-tile's last chunk, 1..64
    v4f binit[1], blast[1];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        const float b = as_const(a.bias)[it.k_off + v];
        float bv;
        asm volatile("v_mov_b32 %0, %1" : "=v"(bv) : "s"(b));
        binit[0][v] = bv;
        blast[0][v] = lane < remc ? bv : -INFINITY;
    }
    int kid[NK];
#pragma unroll
    for (int q = 0; q < NK; ++q) kid[q] = as_const(a.kid)[it.k_off + q * SIGMA];
    const int span = SIGMA * d;
    const int s_full = it.O / span;
    const int rest = it.O - s_full * span;
    const int nlast = rest > 0 ? (min(rest, d) + kTile - 1) / kTile : 0;
    const int nblk = (nc + NT - 1) / NT;  // blocks per super-tile
    const int bsz = nc / nblk, bextra = nc % nblk;
    const McCtx mc{};
    const int row_pitch = a.row_stride;
    const int64_t f_stride = (int64_t)a.nf * a.K;
    for (int r = 0; r < nrows; ++r) {
        RowAcc<1> ra;
        init_row<1, MPV>(ra);
        const uint32_t row = lds_addr(rows0 + r * row_pitch);
        // super-tiles of at most 4 chunks: several per block (padded rows)
        int st0 = 0;
        if constexpr (!CLAMP) {
            switch (nc) {
                case 1: st0 = toep_runs<TAPS, 1, 4, MPV>(row, it.p, d, span, s_full, wa, binit, blast, ra); break;
                case 2: st0 = toep_runs<TAPS, 2, 4, MPV>(row, it.p, d, span, s_full, wa, binit, blast, ra); break;
                case 3: st0 = toep_runs<TAPS, 3, 2, MPV>(row, it.p, d, span, s_full, wa, binit, blast, ra); break;
                case 4: st0 = toep_runs<TAPS, 4, 2, MPV>(row, it.p, d, span, s_full, wa, binit, blast, ra); break;
                default: break;
            }
        }
        for (int st = st0; st < s_full; ++st) {
            const int T = st * span;
            // nblk blocks of nearly equal size (the first nc % nblk one tile
            // larger), so that no block is left with one or two tiles
            int c0 = 0;
            for (int blk = 0; blk + 1 < nblk; ++blk) {
                const int sz = bsz + (blk < bextra ? 1 : 0);
                const int b0 = T + c0 * kTile - it.p;
                if constexpr (CLAMP)
                    TailTiles<TAPS, 1, NT, MPV, false, ClampedTiles, false>::run(sz, ClampedTiles{row, b0, d, a.L}, wa,
                                                                                 mc, binit, blast, ra);
                else
                    TailTiles<TAPS, 1, NT, MPV, false, PaddedTiles, false>::run(
                        sz, PaddedTiles{row + 4u * (uint32_t)b0, d}, wa, mc, binit, blast, ra);
                c0 += sz;
            }
            const int b0 = T + c0 * kTile - it.p;
            if constexpr (CLAMP)
                TailTiles<TAPS, 1, NT, MPV, false, ClampedTiles>::run(nc - c0, ClampedTiles{row, b0, d, a.L}, wa, mc,
                                                                      binit, blast, ra);
            else
                TailTiles<TAPS, 1, NT, MPV, false, PaddedTiles>::run(nc - c0, PaddedTiles{row + 4u * (uint32_t)b0, d},
                                                                     wa, mc, binit, blast, ra);
        }
        // the last, partial super-tile: chunk by chunk, each slot valid on
        // the lanes whose position is in its chunk's d and below O
        const int T = s_full * span;
        for (int c = 0; c < nlast; ++c) {
            v4f bm[1];
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int lim = min(d - c * kTile, it.O - T - c * kTile - (v % SIGMA) * d);
                bm[0][v] = lane < lim ? binit[0][v] : -INFINITY;
            }
            const int b0 = T + c * kTile - it.p;
            if constexpr (CLAMP)
                tile_block<TAPS, 1, 1, true, MPV, false>(ClampedTiles{row, b0, d, a.L}, wa, mc, binit, bm, ra);
            else
                tile_block<TAPS, 1, 1, true, MPV, false>(RightClampedTiles{row, b0, d, a.L}, wa, mc, binit, bm, ra);
        }
        // each kernel's features from its SIGMA slots
#pragma unroll
        for (int q = 0; q < NK; ++q) {
            uint32_t cnt = 0;
            float m = ra.mx[0][q * SIGMA], ps = MPV ? ra.ps[0][q * SIGMA] : 0.0f;
#pragma unroll
            for (int h = 0; h < SIGMA; ++h) cnt += ra.cnt[0][q * SIGMA + h];
#pragma unroll
            for (int h = 1; h < SIGMA; ++h) {
                m = fmaxf(m, ra.mx[0][q * SIGMA + h]);
                if (MPV) ps += ra.ps[0][q * SIGMA + h];
            }
            m = wave_all<OpMax>(m);
            if (MPV) ps = wave_all<OpSum>(ps);
            if (lane == 0 && kid[q] >= 0) write_features<MPV>(cnt, m, ps, kid[q], it.inv_O, F0 + r * f_stride);
        }
    }
}

template <int ELL, int NK, bool CLAMP, bool MPV>
__device__ __forceinline__ void run_toep_items(int *next_item, int beg, int cnt_items, const float *rows0, int nrows,
                                               const FusedArgs &a, float *F0, int lane) {
    while (true) {
        int idx = 0;
        if (lane == 0) idx = atomicAdd(next_item, 1);
        idx = __builtin_amdgcn_readfirstlane(__shfl(idx, 0, 64));
        if (idx >= cnt_items) break;
        const ItemDesc it = load_item(as_const(a.items) + as_const(a.order)[beg + idx]);
        run_toep_item<ELL, NK, CLAMP, MPV>(it, rows0, nrows, a, F0, lane);
    }
}

struct GroupWork {
    int variant;
    int beg;        // first entry of the items' order
    int cnt_items;
    int nrows;      // series staged
    int64_t grow;   // first series (global row)
};

// Workgroup = (variant, row group, split).  Workgroup b runs on XCD b % 8.
// Every XCD takes its own share of the row groups and walks them variant by
// variant, so all XCDs get the same mix of work while the CUs of an XCD run
// one code variant at a time.  Returns false when the workgroup has nothing
// to do (uniformly for the whole workgroup).
__device__ __forceinline__ bool group_work(const FusedArgs &a, GroupWork &w) {
    const int64_t b = blockIdx.x;
    const int xcd = (int)(b % kXcds);
    const int64_t local = b / kXcds;
    const int64_t per_variant = a.groups_per_xcd * a.nsplit;
    const int vi = (int)(local / per_variant);
    const int64_t rest = local % per_variant;
    const int64_t group = xcd * a.groups_per_xcd + rest / a.nsplit;
    const int split = (int)(rest % a.nsplit);
    w.variant = a.variants[vi];
    w.beg = as_const(a.split_begin)[w.variant * a.nsplit + split];
    w.cnt_items = as_const(a.split_begin)[w.variant * a.nsplit + split + 1] - w.beg;
    const int64_t first = group * a.rows_per_block;
    if (w.cnt_items == 0 || first >= a.n_rows) return false;
    w.nrows = (int)min((int64_t)a.rows_per_block, a.n_rows - first);
    w.grow = a.row0 + first;
    return true;
}

// Stages the group's series (every channel) with their zero margins into
// smem, coalesced (channel c of row r at (r*C + c)*row_stride), and the tail
// pad after them.
template <int BLOCK>
__device__ __forceinline__ bool stage_group(const FusedArgs &a, float *smem, int *next_item,
                                            GroupWork &w) {
    if (!group_work(a, w)) return false;
    if (a.vec4) {
        // 4 floats per lane: the series and both margins are whole 16-byte
        // words, so no word straddles a margin
        const int stride4 = a.row_stride >> 2, lo4 = a.halo_lo >> 2, L4 = a.L >> 2;
        for (int rc = 0; rc < w.nrows * a.C; ++rc) {
            const float4 *x = reinterpret_cast<const float4 *>(a.X + ((w.grow * a.C) + rc) * (int64_t)a.L);
            float4 *dst = reinterpret_cast<float4 *>(smem + rc * a.row_stride);
            for (int e = threadIdx.x; e < stride4; e += BLOCK) {
                const int m = e - lo4;
                dst[e] = (m >= 0 && m < L4) ? x[m] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            }
        }
    } else {
        for (int rc = 0; rc < w.nrows * a.C; ++rc) {
            const float *x = a.X + ((w.grow * a.C) + rc) * (int64_t)a.L;
            float *dst = smem + rc * a.row_stride;
            for (int e = threadIdx.x; e < a.row_stride; e += BLOCK) {
                const int m = e - a.halo_lo;
                dst[e] = (m >= 0 && m < a.L) ? x[m] : 0.0f;
            }
        }
    }
    // zeros after the last row: lanes past the last output of an item read
    // up to tail_pad floats past it
    for (int e = threadIdx.x; e < a.tail_pad; e += BLOCK) smem[w.nrows * a.C * a.row_stride + e] = 0.0f;
    set_check_bounds(smem, (int64_t)w.nrows * a.C * a.row_stride + a.tail_pad,
                     a.F + a.row0 * (int64_t)a.nf * a.K, a.F + (a.row0 + a.n_rows) * (int64_t)a.nf * a.K);
    if (threadIdx.x == 0) *next_item = 0;
    __syncthreads();
    return true;
}

// Workgroup = (variant, row group, split); each workgroup stages its row
// group in LDS and runs the items of one variant over it.
template <int BLOCK, bool CLAMP, bool MPV, bool MC>
__global__ __launch_bounds__(BLOCK) void rocket_fused_kernel(FusedArgs a) {
    extern __shared__ __align__(16) float smem[];
    __shared__ int next_item;
    GroupWork w;
    if (!stage_group<BLOCK>(a, smem, &next_item, w)) return;
    const int lane = threadIdx.x & (rocket::kWave - 1);
    float *F0 = a.F + w.grow * (int64_t)a.nf * a.K;
    const float *rows0 = smem + a.halo_lo;
    const int beg = w.beg, cnt = w.cnt_items, nr = w.nrows;
    if constexpr (MC) {
        // multichannel plans hold 4-kernel items only (variants 0, 2, 4)
        switch (w.variant) {
            case 0: run_items<7, 1, CLAMP, MPV, MC>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
            case 2: run_items<9, 1, CLAMP, MPV, MC>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
            default: run_items<11, 1, CLAMP, MPV, MC>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
        }
    } else {
        switch (w.variant) {
            case 0: run_items<7, 1, CLAMP, MPV, MC>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
            case 1: run_items<7, 2, CLAMP, MPV, MC>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
            case 2: run_items<9, 1, CLAMP, MPV, MC>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
            case 3: run_items<9, 2, CLAMP, MPV, MC>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
            case 4: run_items<11, 1, CLAMP, MPV, MC>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
            case 5: run_items<11, 2, CLAMP, MPV, MC>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
            // VALU items (univariate long-series plans)
            case 6: run_valu_items<7, 1, CLAMP, MPV>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
            case 7: run_valu_items<7, 2, CLAMP, MPV>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
            case 8: run_valu_items<9, 1, CLAMP, MPV>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
            case 9: run_valu_items<9, 2, CLAMP, MPV>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
            case 10: run_valu_items<11, 1, CLAMP, MPV>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
            default: run_valu_items<11, 2, CLAMP, MPV>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
        }
    }
}

// Toeplitz items (univariate long-series plans) in a kernel of their own,
// launched over the same row groups on a stream of the plan, beside the
// fused kernel (the two write disjoint features): in the fused kernel's code
// their extra tap counts raise the scalar-register pressure of every
// variant's loop.
template <int BLOCK, bool CLAMP, bool MPV>
__global__ __launch_bounds__(BLOCK) void rocket_toeplitz_kernel(FusedArgs a) {
    extern __shared__ __align__(16) float smem[];
    __shared__ int next_item;
    GroupWork w;
    if (!stage_group<BLOCK>(a, smem, &next_item, w)) return;
    const int lane = threadIdx.x & (rocket::kWave - 1);
    float *F0 = a.F + w.grow * (int64_t)a.nf * a.K;
    const float *rows0 = smem + a.halo_lo;
    const int beg = w.beg, cnt = w.cnt_items, nr = w.nrows;
    switch (w.variant) {
        case 12: run_toep_items<7, 1, CLAMP, MPV>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
        case 13: run_toep_items<7, 2, CLAMP, MPV>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
        case 14: run_toep_items<9, 1, CLAMP, MPV>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
        case 15: run_toep_items<9, 2, CLAMP, MPV>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
        case 16: run_toep_items<11, 1, CLAMP, MPV>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
        default: run_toep_items<11, 2, CLAMP, MPV>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
    }
}

// ---------------------------------------------------------------------------
// Series-lane layout (short univariate series).  The 64 lanes of a
// wavefront take 64 series, and LDS holds the workgroup's 64 series
// position-major: the values of all 64 series at one position are 64
// consecutive floats, so a tap's read is again one ds_read_addtid_b32 per
// position.  One MFMA then computes one output position for 4 kernels x 64
// series, and a block runs NT consecutive positions.  Every lane keeps the
// count, the max (and the MPV sum) of its own series, so no cross-lane
// reduction is needed: for short series the per-series reductions and
// writes of the position-tiled layout cost more than the dot products.
// ---------------------------------------------------------------------------

constexpr int kSeriesLanes = rocket::kWave;              // series per workgroup
constexpr int kSeriesMargin = rocket::kMaxTilesPerBlock;  // zero positions on each side
using rocket::kSeriesMaxL;                                 // longest series it takes
constexpr int64_t kSeriesMinRows = 4096;  // fewer series per call: too few workgroups, use tiles

// Stages the group's series: position m of series r at
// smem[(m + kSeriesMargin) * 64 + r], with zeros in the margins and in the
// lanes past the group's last series.  Consecutive threads write
// consecutive LDS words (no bank conflicts); their global reads are a
// series apart and hit the same cache lines across the loop.
template <int BLOCK>
__device__ __forceinline__ bool stage_series(const FusedArgs &a, float *smem, int *next_item,
                                             GroupWork &w) {
    if (!group_work(a, w)) return false;
    const int total = (a.L + 2 * kSeriesMargin) * kSeriesLanes;
    const float *x = a.X + w.grow * (int64_t)a.L;
    for (int e = threadIdx.x; e < total; e += BLOCK) {
        const int r = e & (kSeriesLanes - 1);
        const int m = e / kSeriesLanes - kSeriesMargin;
        smem[e] = (r < w.nrows && m >= 0 && m < a.L) ? x[(int64_t)r * a.L + m] : 0.0f;
    }
    set_check_bounds(smem, total, a.S, a.S + a.s_floats);
    if (threadIdx.x == 0) *next_item = 0;
    __syncthreads();
    return true;
}

// Series-lane reads.  pos0 is the LDS byte address of position 0 (its 64
// series); the position of the block's first output under tap j is clamped
// into [-kSeriesMargin, L] on the scalar unit, as for ClampedTiles: a block
// whose positions all lie outside the series reads zeros from a margin, a
// block that overlaps it is not moved.
struct SeriesTiles {
    uint32_t pos0;
    int b0;  // position under tap 0 of the block's first output
    int d;
    int L;
    __device__ __forceinline__ uint32_t m0(int j) const {
        const int b = min(max(b0 + j * d, -kSeriesMargin), L);
        return pos0 + 256u * (uint32_t)b;
    }
};

template <>
struct PipelinedReads<SeriesTiles> {
    static constexpr bool value = true;
};

// Per-lane (per-series) accumulators of one work item.
template <int G>
struct SeriesAcc {
    v4f mx[G];
    uint32_t cnt[G][4];
    v4f ps[G];
};

// [y > 0] as 0 or 1.  For a float that is not a NaN the bits read as a
// signed integer are positive exactly when y > 0 (+0 reads 0; -0 and the
// negative values read negative), so med3(bits, 0, 1) is the indicator.
__device__ __forceinline__ uint32_t positive01(float y) {
    uint32_t r;
    asm("v_med3_i32 %0, %1, 0, 1" : "=v"(r) : "v"(y));
    return r;
}

// Fold NT positions of finished dot products into the lanes' accumulators:
// the counts add the indicators two at a time, MAX folds pairs with v_max3.
template <int G, int NT, bool MPV>
__device__ __forceinline__ void series_reduce(const v4f (&acc)[NT][G], SeriesAcc<G> &sa) {
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            uint32_t c = sa.cnt[g][v];
#pragma unroll
            for (int u = 0; u < NT; u += 2) {
                if (u + 1 < NT)
                    c += positive01(acc[u][g][v]) + positive01(acc[u + 1][g][v]);
                else
                    c += positive01(acc[u][g][v]);
            }
            sa.cnt[g][v] = c;
        }
    if (MPV) {
#pragma unroll
        for (int u = 0; u < NT; ++u)
#pragma unroll
            for (int g = 0; g < G; ++g)
#pragma unroll
                for (int v = 0; v < 4; ++v) sa.ps[g][v] += fmaxf(acc[u][g][v], 0.0f);
    }
#pragma unroll
    for (int u = 0; u + 1 < NT; u += 2)
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int v = 0; v < 4; ++v)
                sa.mx[g][v] = fmaxf(fmaxf(sa.mx[g][v], acc[u][g][v]), acc[u + 1][g][v]);
    if (NT % 2 == 1) {
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int v = 0; v < 4; ++v) sa.mx[g][v] = fmaxf(sa.mx[g][v], acc[NT - 1][g][v]);
    }
}

// NT consecutive output positions of one item for the 64 series.
template <int ELL, int G, int NT, bool MPV>
__device__ __forceinline__ void series_block(const SeriesTiles &src, const float (&wa)[G][ELL],
                                             const v4f (&binit)[G], SeriesAcc<G> &sa) {
    v4f acc[NT][G];
    tile_mfma<ELL, G, NT, false, true>(src, wa, binit, binit, acc);
    __builtin_amdgcn_sched_barrier(0);
    // raised wave priority while the fold runs, as in the fused kernel
    __builtin_amdgcn_s_setprio(1);
    series_reduce<G, NT, MPV>(acc, sa);
    __builtin_amdgcn_s_setprio(0);
}

// The last positions of an item, nv (1..N) of them: a code copy per count.
template <int ELL, int G, int N, bool MPV>
struct SeriesTail {
    __device__ __forceinline__ static void run(int nv, const SeriesTiles &src, const float (&wa)[G][ELL],
                                               const v4f (&binit)[G], SeriesAcc<G> &sa) {
        if (nv == N)
            series_block<ELL, G, N, MPV>(src, wa, binit, sa);
        else
            SeriesTail<ELL, G, N - 1, MPV>::run(nv, src, wa, binit, sa);
    }
};
template <int ELL, int G, bool MPV>
struct SeriesTail<ELL, G, 0, MPV> {
    __device__ __forceinline__ static void run(int, const SeriesTiles &, const float (&)[G][ELL],
                                               const v4f (&)[G], SeriesAcc<G> &) {}
};

// One work item over the group's 64 series: all O positions in blocks of
// NT, then each lane writes the features of its series for the item's
// kernels.
template <int ELL, int G, bool MPV>
__device__ __forceinline__ void run_series_item(const ItemDesc &it, uint32_t pos0, int nrows,
                                                const FusedArgs &a, int64_t srow0, int lane) {
    constexpr int NT = rocket::kTilesPerBlock[G - 1];
    float wa[G][ELL];
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int j = 0; j < ELL; ++j) wa[g][j] = a.wpk[it.w_off + (g * ELL + j) * 4 + (lane & 3)];
    // C operand of the first tap: the bias of block row v (kernel slot v),
    // the same on every lane (series)
    v4f binit[G];
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const float b = as_const(a.bias)[it.k_off + 4 * g + v];
            float bv;
            asm volatile("v_mov_b32 %0, %1" : "=v"(bv) : "s"(b));
            binit[g][v] = bv;
        }
    SeriesAcc<G> sa;
#pragma unroll
    for (int g = 0; g < G; ++g) {
        v2f lo, hi;
        asm volatile("v_mov_b64 %0, %2\n\tv_mov_b64 %1, %2" : "=v"(lo), "=v"(hi) : "s"(kNegInfPair));
        sa.mx[g] = v4f{lo[0], lo[1], hi[0], hi[1]};
        if (MPV) sa.ps[g] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int v = 0; v < 4; ++v) sa.cnt[g][v] = 0;
    }
    const int nfull = it.O / NT;          // full blocks
    const int nv = it.O - nfull * NT;     // positions in the last block, 0..NT-1
    for (int blk = 0; blk < nfull; ++blk)
        series_block<ELL, G, NT, MPV>(SeriesTiles{pos0, blk * NT - it.p, it.d, a.L}, wa, binit, sa);
    if (nv > 0)
        SeriesTail<ELL, G, NT - 1, MPV>::run(nv, SeriesTiles{pos0, nfull * NT - it.p, it.d, a.L}, wa,
                                             binit, sa);
    // features into the slot-ordered buffer: slot s of series r (of this
    // launch) at S[(s * s_rows + r) * nf], so the 64 lanes of a slot write
    // 64 * nf consecutive floats
    if (lane < nrows) {
        float *Srow = a.S + (srow0 + lane) * (int64_t)a.nf;
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int slot = it.k_off + 4 * g + v;
                if (as_const(a.kid)[slot] >= 0)
                    write_features<MPV>(sa.cnt[g][v], sa.mx[g][v], sa.ps[g][v], 0, it.inv_O,
                                        Srow + slot * a.s_rows * (int64_t)a.nf);
            }
    }
}

template <int ELL, int G, bool MPV>
__device__ __forceinline__ void run_series_items(int *next_item, int beg, int cnt_items, uint32_t pos0,
                                                 int nrows, const FusedArgs &a, int64_t srow0, int lane) {
    while (true) {
        int idx = 0;
        if (lane == 0) idx = atomicAdd(next_item, 1);
        idx = __builtin_amdgcn_readfirstlane(__shfl(idx, 0, 64));
        if (idx >= cnt_items) break;
        const ItemDesc it = load_item(as_const(a.items) + as_const(a.order)[beg + idx]);
        run_series_item<ELL, G, MPV>(it, pos0, nrows, a, srow0, lane);
    }
}

// Workgroup = (variant, group of 64 series, split), mapped as for the fused
// kernel; each wavefront takes items from the workgroup's counter.
template <bool MPV>
__global__ __launch_bounds__(kBlock) void rocket_series_kernel(FusedArgs a) {
    extern __shared__ float smem[];
    __shared__ int next_item;
    GroupWork w;
    if (!stage_series<kBlock>(a, smem, &next_item, w)) return;
    const int lane = threadIdx.x & (rocket::kWave - 1);
    const int64_t F0 = w.grow - a.row0;  // first series of the group in S
    uint32_t pos0 = lds_addr(smem + kSeriesMargin * kSeriesLanes);
    asm volatile("" : "+s"(pos0));  // computed once (not again in every block)
    const int beg = w.beg, cnt = w.cnt_items, nr = w.nrows;
    switch (w.variant) {
        case 0: run_series_items<7, 1, MPV>(&next_item, beg, cnt, pos0, nr, a, F0, lane); break;
        case 1: run_series_items<7, 2, MPV>(&next_item, beg, cnt, pos0, nr, a, F0, lane); break;
        case 2: run_series_items<9, 1, MPV>(&next_item, beg, cnt, pos0, nr, a, F0, lane); break;
        case 3: run_series_items<9, 2, MPV>(&next_item, beg, cnt, pos0, nr, a, F0, lane); break;
        case 4: run_series_items<11, 1, MPV>(&next_item, beg, cnt, pos0, nr, a, F0, lane); break;
        default: run_series_items<11, 2, MPV>(&next_item, beg, cnt, pos0, nr, a, F0, lane); break;
    }
}

// F rows in the original kernel order from the slot-ordered buffer: a tile
// is 64 kernels x 64 series, and the workgroups (4 wavefronts) stride over
// the tiles; wavefront w takes the tile's series 16w .. 16w + 15.  Lane l
// moves kernel k0 + l: it reads the 16 series' features from its slot column
// as whole 16-byte vectors (16 * NF consecutive floats, 128 or 192 bytes),
// then writes them series by series, so each series' 64 kernels go out as
// 64 * NF consecutive floats.  Columns hold s_rows series, a multiple of 64,
// so the reads of a partial last tile stay inside the column; only the
// writes check the series count.  No LDS: the kernel runs beside the series
// kernel, which fills the LDS.
template <int NF>
__global__ __launch_bounds__(kBlock) void rocket_slot_permute_kernel(const float *S, int64_t s_rows,
                                                                     const int32_t *slot_of, int32_t K,
                                                                     int64_t n_rows, float *F,
                                                                     int32_t n_slots) {
    constexpr int kRows = 16;
    constexpr int kVec = kRows * NF / 4;  // float4 per lane
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t k_tiles = ((int64_t)K + 63) / 64;
    const int64_t n_tiles = k_tiles * ((n_rows + 63) / 64);
    for (int64_t t = blockIdx.x; t < n_tiles; t += gridDim.x) {
        const int64_t k = (t % k_tiles) * 64 + lane;
        const int64_t r0 = (t / k_tiles) * 64 + wave * kRows;
        if (k >= K || r0 >= n_rows) continue;
#if ROCKET_CHECKED
        // the slot column this lane reads must be one of the buffer's n_slots
        if (slot_of[k] < 0 || slot_of[k] >= n_slots) {
            check_failed(kCheckSlotRead);
            continue;
        }
#endif
        const float4 *src = reinterpret_cast<const float4 *>(S + ((int64_t)slot_of[k] * s_rows + r0) * NF);
        float v[kVec * 4];
#pragma unroll
        for (int i = 0; i < kVec; ++i) {
            const float4 q = src[i];
            v[4 * i] = q.x;
            v[4 * i + 1] = q.y;
            v[4 * i + 2] = q.z;
            v[4 * i + 3] = q.w;
        }
        const int nr = (int)min<int64_t>(kRows, n_rows - r0);
        float *b = F + r0 * (int64_t)K * NF + k * NF;
#pragma unroll
        for (int rr = 0; rr < kRows; ++rr) {
            if (rr < nr) {
                if constexpr (NF == 2) {
                    *reinterpret_cast<float2 *>(b) = make_float2(v[2 * rr], v[2 * rr + 1]);
                } else {
#pragma unroll
                    for (int f = 0; f < NF; ++f) b[f] = v[NF * rr + f];
                }
            }
            b += (int64_t)K * NF;
        }
    }
}

// ---------------------------------------------------------------------------
// MINIROCKET (Dempster, Schmidt and Webb, KDD 2021; Sec. 5 names it as a
// variant the same principle carries over to).  Its 84 kernels have 9 taps,
// weight 2 on a choice of 3 taps (a, b, c) and -1 on the other six, so a dot
// product is
//     C = 3 (x_a + x_b + x_c) - (x_0 + ... + x_8).
// An item holds the 42 kernels of one parity at one (dilation, padding)
// (the pair (dilation i, kernel k) is padded when i + k is even) and NQ (4 or
// 8) of each kernel's biases.  For each tile of 64 output positions the nine
// tap values are read from LDS once and their sum S is formed once, by a
// pairwise tree, for all 42 kernels; a kernel then costs two adds and one
// fma on the vector unit,
//     C = fma(3, (x_a + x_b) + x_c, -S),
// instead of nine multiply-adds.  Rounding: |C - C_exact| <= 3 gamma_2
// sum_chosen |x| + gamma_4 sum_all |x| + u |C|, about 12u sum_chosen |x| +
// 5u sum_others |x| (u = 2^-24), inside the gamma_9 sum_j |w_j x_j| = 18u
// sum_chosen |x| + 9u sum_others |x| that bounds any 9-term fp32 evaluation
// (additions of subnormals are exact, so no underflow term is added).
// Feature (kernel, bias b) counts C > b: one compare per tile, a ballot
// popcounted on the scalar unit.
// ---------------------------------------------------------------------------

using rocket::kMrKappa;
constexpr int kMrTiles = 4;  // tiles per block (the last 0..3 tiles run one at a time)

// Tap `which` (0, 1, 2 for a < b < c) of MINIROCKET kernel k: the k-th choice
// of 3 of the 9 taps in lexicographic order.
constexpr int mr_tap(int k, int which) {
    int n = 0;
    for (int a = 0; a < 9; ++a)
        for (int b = a + 1; b < 9; ++b)
            for (int c = b + 1; c < 9; ++c) {
                if (n == k) return which == 0 ? a : (which == 1 ? b : c);
                ++n;
            }
    return -1;
}
static_assert(mr_tap(0, 0) == 0 && mr_tap(0, 2) == 2 && mr_tap(83, 0) == 6 && mr_tap(83, 2) == 8,
              "84 lexicographic choices of 3 of 9 taps");

// Count registers of an item: feature g = kappa * NQ + q (kernel 2 kappa +
// parity, bias q) lives in lane g % 64 of register g / 64.
template <int NQ>
constexpr int mr_regs() { return (kMrKappa * NQ + 63) / 64; }

// The count of feature G over the block's NT tiles (a ballot popcount per
// tile, summed on the scalar unit) into its lane of the block's partial
// counts.
template <int G, int NT>
__device__ __forceinline__ void mr_count(const float (&C)[NT], float b, uint32_t &part) {
    uint32_t s = 0;
#pragma unroll
    for (int u = 0; u < NT; ++u) s += (uint32_t)__popcll(__builtin_amdgcn_ballot_w64(C[u] > b));
    asm volatile("v_writelane_b32 %0, %1, %2" : "+v"(part) : "s"(s), "i"(G % 64));
}

template <int KAPPA, int Q, int NQ, int NT, int R>
struct MrCounts {
    __device__ __forceinline__ static void run(const float (&C)[NT], const float (&b)[NQ], uint32_t (&part)[R]) {
        constexpr int G = KAPPA * NQ + Q;
        mr_count<G, NT>(C, b[Q], part[G / 64]);
        MrCounts<KAPPA, Q + 1, NQ, NT, R>::run(C, b, part);
    }
};
template <int KAPPA, int NQ, int NT, int R>
struct MrCounts<KAPPA, NQ, NQ, NT, R> {
    __device__ __forceinline__ static void run(const float (&)[NT], const float (&)[NQ], uint32_t (&)[R]) {}
};

// Kernels 2 KAPPA + PAR, KAPPA = KAPPA0 .. 41, over the block's NT tiles: the
// dot products from the shared tap values and sum, then the compares.  Each
// kernel's section is closed by a scheduling barrier and loads the next
// kernel's biases (scalar loads) while its own compares run, so only two
// kernels' biases are live in scalar registers.
template <int PAR, int KAPPA, int NQ, int NT, int R>
struct MrKernels {
    __device__ __forceinline__ static void run(const float (&x)[9][NT], const float (&S)[NT],
                                               ConstPtr<float> thr, const float (&b)[NQ], uint32_t (&part)[R]) {
        constexpr int k = 2 * KAPPA + PAR;
        constexpr int ta = mr_tap(k, 0), tb = mr_tap(k, 1), tc = mr_tap(k, 2);
        float bn[NQ];
        if constexpr (KAPPA + 1 < kMrKappa) {
#pragma unroll
            for (int q = 0; q < NQ; ++q) bn[q] = thr[(KAPPA + 1) * NQ + q];
        }
        float C[NT];
#pragma unroll
        for (int u = 0; u < NT; ++u) C[u] = fmaf(3.0f, (x[ta][u] + x[tb][u]) + x[tc][u], -S[u]);
        MrCounts<KAPPA, 0, NQ, NT, R>::run(C, b, part);
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (KAPPA + 1 < kMrKappa) MrKernels<PAR, KAPPA + 1, NQ, NT, R>::run(x, S, thr, bn, part);
    }
};

// One block of NT tiles of an item over one series.  rem = outputs of the
// block's last tile (64 unless it is the series' last tile): lanes past it
// get S = +inf, so C = -inf there and no bias is exceeded.
template <int PAR, int NQ, int NT, typename Src>
__device__ __forceinline__ void mr_block(const Src &src, ConstPtr<float> thr, int rem, int lane,
                                         uint32_t (&part)[mr_regs<NQ>()], uint32_t (&cnt)[mr_regs<NQ>()]) {
    float x[9][NT];
#pragma unroll
    for (int j = 0; j < 9; ++j) lds_tiles<NT>(src.m0(j), x[j]);
    float S[NT];
#pragma unroll
    for (int u = 0; u < NT; ++u)
        S[u] = (((x[0][u] + x[1][u]) + (x[2][u] + x[3][u])) + ((x[4][u] + x[5][u]) + (x[6][u] + x[7][u]))) +
               x[8][u];
    S[NT - 1] = lane < rem ? S[NT - 1] : INFINITY;
    // a fresh copy of the bias pointer per block keeps the bias loads inside
    // the block (hoisted out of the row loop, 42 * NQ biases would not fit
    // the scalar registers)
    uint64_t tp = (uint64_t)(__UINTPTR_TYPE__)thr;
    asm volatile("" : "+s"(tp));
    const ConstPtr<float> tb = (ConstPtr<float>)(__UINTPTR_TYPE__)tp;
    float b0[NQ];
#pragma unroll
    for (int q = 0; q < NQ; ++q) b0[q] = tb[q];
    MrKernels<PAR, 0, NQ, NT, mr_regs<NQ>()>::run(x, S, tb, b0, part);
#pragma unroll
    for (int r = 0; r < mr_regs<NQ>(); ++r) cnt[r] += part[r];
}

template <int PAR, int NQ, bool CLAMP>
__device__ __forceinline__ void run_mr_item(const ItemDesc &it, const float *rows0, int nrows,
                                            const FusedArgs &a, float *F0, int lane) {
    constexpr int NT = kMrTiles;
    constexpr int R = mr_regs<NQ>();
    const ConstPtr<float> thr = as_const(a.thr) + it.t_off;
    // the feature each lane writes from each count register (-1: none)
    int64_t fidx[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int g = 64 * r + lane;
        const int kappa = g / NQ, q = g % NQ;
        fidx[r] = (kappa < kMrKappa && it.k_off + q < it.n_ch)
                      ? (int64_t)it.w_off + (int64_t)(2 * kappa + PAR) * it.n_ch + it.k_off + q
                      : -1;
    }
    uint32_t part[R], cnt[R];
#pragma unroll
    for (int r = 0; r < R; ++r) part[r] = cnt[r] = 0;  // lanes past 42 * NQ stay 0
    const int rem = it.O - (it.n_tiles - 1) * kTile;  // outputs in the last tile, 1..64
    const int nfull = it.n_tiles / NT;                // blocks of NT tiles
    const int ntail = it.n_tiles - nfull * NT;        // then 0..NT-1 single tiles
    const int row_pitch = a.row_stride;
    const int64_t f_stride = (int64_t)a.nf * a.K;
    for (int r = 0; r < nrows; ++r) {
        const uint32_t row = lds_addr(rows0 + r * row_pitch);
        for (int blk = 0; blk < nfull; ++blk) {
            const int b0 = blk * (NT * kTile) - it.p;
            const int rb = (ntail == 0 && blk == nfull - 1) ? rem : kTile;
            if constexpr (CLAMP)
                mr_block<PAR, NQ, NT>(ClampedTiles{row, b0, it.d, a.L}, thr, rb, lane, part, cnt);
            else
                mr_block<PAR, NQ, NT>(PaddedTiles{row + 4u * (uint32_t)b0, it.d}, thr, rb, lane, part, cnt);
        }
        for (int t = 0; t < ntail; ++t) {
            const int b0 = (nfull * NT + t) * kTile - it.p;
            const int rb = t == ntail - 1 ? rem : kTile;
            if constexpr (CLAMP)
                mr_block<PAR, NQ, 1>(ClampedTiles{row, b0, it.d, a.L}, thr, rb, lane, part, cnt);
            else
                mr_block<PAR, NQ, 1>(PaddedTiles{row + 4u * (uint32_t)b0, it.d}, thr, rb, lane, part, cnt);
        }
        // PPV = count / O, correctly rounded as in write_features
#pragma unroll
        for (int rr = 0; rr < R; ++rr) {
            if (fidx[rr] >= 0 && store_checked(F0 + r * f_stride + fidx[rr], 1))
                F0[r * f_stride + fidx[rr]] = (float)((double)cnt[rr] * it.inv_O);
            cnt[rr] = 0;
        }
    }
}

template <int PAR, int NQ, bool CLAMP>
__device__ __forceinline__ void run_mr_items(int *next_item, int beg, int cnt_items, const float *rows0,
                                             int nrows, const FusedArgs &a, float *F0, int lane) {
    while (true) {
        int idx = 0;
        if (lane == 0) idx = atomicAdd(next_item, 1);
        idx = __builtin_amdgcn_readfirstlane(__shfl(idx, 0, 64));
        if (idx >= cnt_items) break;
        const ItemDesc it = load_item(as_const(a.items) + as_const(a.order)[beg + idx]);
        run_mr_item<PAR, NQ, CLAMP>(it, rows0, nrows, a, F0, lane);
    }
}

// MINIROCKET workgroup: as rocket_fused_kernel; variant = mr_variant(parity, NQ).
template <int BLOCK, bool CLAMP>
__global__ __launch_bounds__(BLOCK) void rocket_minirocket_kernel(FusedArgs a) {
    extern __shared__ __align__(16) float smem[];
    __shared__ int next_item;
    GroupWork w;
    if (!stage_group<BLOCK>(a, smem, &next_item, w)) return;
    const int lane = threadIdx.x & (rocket::kWave - 1);
    float *F0 = a.F + w.grow * (int64_t)a.nf * a.K;
    const float *rows0 = smem + a.halo_lo;
    const int beg = w.beg, cnt = w.cnt_items, nr = w.nrows;
    switch (w.variant) {
        case 0: run_mr_items<0, rocket::kMrQSmall, CLAMP>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
        case 1: run_mr_items<0, rocket::kMrQLarge, CLAMP>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
        case 2: run_mr_items<0, rocket::kMrQTiny, CLAMP>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
        case 3: run_mr_items<1, rocket::kMrQSmall, CLAMP>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
        case 4: run_mr_items<1, rocket::kMrQLarge, CLAMP>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
        default: run_mr_items<1, rocket::kMrQTiny, CLAMP>(&next_item, beg, cnt, rows0, nr, a, F0, lane); break;
    }
}

// Plain kernel: one wavefront per (series, kernel) pair, lanes over output
// positions, taps read straight from global memory with the zero padding
// applied by bounds checks.
__global__ __launch_bounds__(kBlock) void rocket_direct_kernel(
    const float *__restrict__ X, int64_t row0, int32_t L, int32_t K, int32_t k0,
    const int32_t *__restrict__ len, const int32_t *__restrict__ dil,
    const int32_t *__restrict__ pad, const float *__restrict__ bias,
    const float *__restrict__ w, int32_t max_len, int32_t nf, int32_t C,
    const int32_t *__restrict__ ccount, const int32_t *__restrict__ cindex,
    float *__restrict__ F) {
    const int64_t row = row0 + blockIdx.x;
    const int k = k0 + (int)blockIdx.y * (kBlock / 64) + (int)(threadIdx.x >> 6);
    if (k >= K) return;
    const int lane = threadIdx.x & 63;
    const int ell = len[k], d = dil[k], p = pad[k];
    const int nch = C > 1 ? ccount[k] : 1;
    const float b = bias[k];
    const int64_t O = (int64_t)L + 2 * (int64_t)p - (int64_t)(ell - 1) * d;
    float mx = -INFINITY, ps = 0.0f;
    uint32_t c = 0;
    for (int64_t t = lane; t < O; t += 64) {
        float acc = b;
        for (int s = 0; s < nch; ++s) {
            const int ch = C > 1 ? cindex[(int64_t)k * C + s] : 0;
            const float *x = X + (row * C + ch) * (int64_t)L;
            const float *wk = w + ((int64_t)k * C + s) * max_len;
            for (int j = 0; j < ell; ++j) {
                const int64_t m = t - p + (int64_t)j * d;
                const float xv = (m >= 0 && m < L) ? x[m] : 0.0f;
                acc = fmaf(wk[j], xv, acc);
            }
        }
        c += acc > 0.0f ? 1u : 0u;
        ps += acc > 0.0f ? acc : 0.0f;
        mx = fmaxf(mx, acc);
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        mx = fmaxf(mx, __shfl_xor(mx, off, 64));
        c += __shfl_xor(c, off, 64);
        ps += __shfl_xor(ps, off, 64);
    }
    if (lane == 0) {
        float *f = F + row * (int64_t)nf * K + (int64_t)nf * k;
        f[0] = (float)c / (float)O;
        f[1] = mx;
        if (nf == 3) f[2] = c > 0 ? ps / (float)c : 0.0f;
    }
}

template <typename T>
hipError_t upload(const std::vector<T> &h, T **d) {
    *d = nullptr;
    if (h.empty()) return hipSuccess;
    hipError_t e = hipMalloc((void **)d, h.size() * sizeof(T));
    if (e != hipSuccess) return e;
    return hipMemcpy(*d, h.data(), h.size() * sizeof(T), hipMemcpyHostToDevice);
}

template <typename T>
hipError_t upload_raw(const T *h, size_t n, T **d) {
    *d = nullptr;
    hipError_t e = hipMalloc((void **)d, n * sizeof(T));
    if (e != hipSuccess) return e;
    return hipMemcpy(*d, h, n * sizeof(T), hipMemcpyHostToDevice);
}

}  // namespace

// The fused kernel's instances: bit 0 the 1024-thread block (rows above
// kBigLds), bit 1 clamped indices, bit 2 MPV, bit 3 multichannel items.
constexpr int kFusedInstances = 16;
static const void *fused_fn(int sel) {
    static const void *const fns[kFusedInstances] = {
        (const void *)rocket_fused_kernel<kBlock, false, false, false>,
        (const void *)rocket_fused_kernel<kBigBlock, false, false, false>,
        (const void *)rocket_fused_kernel<kBlock, true, false, false>,
        (const void *)rocket_fused_kernel<kBigBlock, true, false, false>,
        (const void *)rocket_fused_kernel<kBlock, false, true, false>,
        (const void *)rocket_fused_kernel<kBigBlock, false, true, false>,
        (const void *)rocket_fused_kernel<kBlock, true, true, false>,
        (const void *)rocket_fused_kernel<kBigBlock, true, true, false>,
        (const void *)rocket_fused_kernel<kBlock, false, false, true>,
        (const void *)rocket_fused_kernel<kBigBlock, false, false, true>,
        (const void *)rocket_fused_kernel<kBlock, true, false, true>,
        (const void *)rocket_fused_kernel<kBigBlock, true, false, true>,
        (const void *)rocket_fused_kernel<kBlock, false, true, true>,
        (const void *)rocket_fused_kernel<kBigBlock, false, true, true>,
        (const void *)rocket_fused_kernel<kBlock, true, true, true>,
        (const void *)rocket_fused_kernel<kBigBlock, true, true, true>,
    };
    return fns[sel];
}

// The MINIROCKET kernel's instances: bit 0 the 1024-thread block, bit 1
// clamped indices.
constexpr int kMrInstances = 4;
static const void *mr_fn(int sel) {
    static const void *const fns[kMrInstances] = {
        (const void *)rocket_minirocket_kernel<kBlock, false>,
        (const void *)rocket_minirocket_kernel<kBigBlock, false>,
        (const void *)rocket_minirocket_kernel<kBlock, true>,
        (const void *)rocket_minirocket_kernel<kBigBlock, true>,
    };
    return fns[sel];
}

// The Toeplitz kernel's instances: bit 0 the 1024-thread block, bit 1
// clamped indices, bit 2 MPV.
constexpr int kToepInstances = 8;
static const void *toep_fn(int sel) {
    static const void *const fns[kToepInstances] = {
        (const void *)rocket_toeplitz_kernel<kBlock, false, false>,
        (const void *)rocket_toeplitz_kernel<kBigBlock, false, false>,
        (const void *)rocket_toeplitz_kernel<kBlock, true, false>,
        (const void *)rocket_toeplitz_kernel<kBigBlock, true, false>,
        (const void *)rocket_toeplitz_kernel<kBlock, false, true>,
        (const void *)rocket_toeplitz_kernel<kBigBlock, false, true>,
        (const void *)rocket_toeplitz_kernel<kBlock, true, true>,
        (const void *)rocket_toeplitz_kernel<kBigBlock, true, true>,
    };
    return fns[sel];
}

static const void *series_fn(bool mpv) {
    return mpv ? (const void *)rocket_series_kernel<true> : (const void *)rocket_series_kernel<false>;
}

struct rocket_plan {
    rocket::HostPlan host;
    // code variants in launch order: by total item cost, largest first
    int32_t variant_order[rocket::kNumVariants] = {};
    int device = 0;
    int n_cu = 0;
    bool direct = false;
    bool clamp = false;      // rows staged with kClampMargin zeros on each side, tap offsets clamped
    bool series = false;     // series-lane layout available (short univariate series)
    int64_t series_min_rows = 0;  // calls with at least this many series use it
    int64_t series_lds = 0;       // its LDS per workgroup
    int32_t *d_slot_of = nullptr;  // series-lane layout: the slot of each kernel
    // series-lane layout: the slot-ordered feature buffer (two halves),
    // allocated on first use and grown as needed; transforms on different
    // streams take turns on it (each waits for the previous user's event).
    // The permutation of one chunk runs on the plan's own stream while the
    // next chunk's series kernel runs on the caller's.
    mutable std::mutex scratch_mu;
    mutable float *d_scratch = nullptr;
    mutable size_t scratch_bytes = 0;
    mutable hipEvent_t scratch_done = nullptr;
    hipStream_t aux = nullptr;
    // the series kernels of odd chunks run on this stream (even ones on the
    // caller's), so that consecutive chunks overlap instead of draining the
    // GPU between them
    hipStream_t odd = nullptr;
    hipEvent_t half_full[2] = {nullptr, nullptr};
    hipEvent_t half_free[2] = {nullptr, nullptr};
    hipEvent_t aux_done = nullptr;
    hipEvent_t call_start = nullptr;  // the caller's stream at the start of a call (odd waits on it)
    hipEvent_t odd_done = nullptr;    // the odd stream's last chunk of a call
    // plans with Toeplitz items: their kernel runs on this stream, beside the
    // fused kernel on the caller's (they write disjoint features)
    mutable std::mutex side_mu;
    hipStream_t side = nullptr;
    hipEvent_t side_start = nullptr;
    hipEvent_t side_done = nullptr;
    bool mpv = false;        // third feature per kernel: mean of positive values
    bool minirocket = false; // MINIROCKET plan: F [n, n_features], PPV only
    int64_t f_cols = 0;      // columns of F
    int32_t C = 1;           // channels per series
    int32_t halo_lo = 0;     // staged layout actually used (floats)
    int32_t row_stride = 0;
    int32_t tail_pad = 0;
    int rows_per_block = 1;  // series staged per workgroup
    int64_t lds_bytes = 0;   // per workgroup: the rows plus the tail pad
    ItemDesc *d_items = nullptr;
    float *d_wpk = nullptr;
    float *d_bias = nullptr;
    int32_t *d_kid = nullptr;
    int32_t *d_order = nullptr;
    int32_t *d_split_begin = nullptr;
    float *d_thr = nullptr;
    // the kernel set as given, for the direct kernel
    int32_t max_len = 0;
    int32_t *d_cc = nullptr;  // channel counts and indices (multichannel sets)
    int32_t *d_ci = nullptr;
    int32_t *d_len = nullptr;
    int32_t *d_dil = nullptr;
    int32_t *d_pad = nullptr;
    float *d_b = nullptr;
    float *d_w = nullptr;
};

static void plan_free_device(rocket_plan *p) {
    if (p->scratch_done) (void)hipEventDestroy(p->scratch_done);
    for (hipEvent_t ev : {p->half_full[0], p->half_full[1], p->half_free[0], p->half_free[1], p->aux_done,
                          p->call_start, p->odd_done, p->side_start, p->side_done})
        if (ev) (void)hipEventDestroy(ev);
    if (p->aux) (void)hipStreamDestroy(p->aux);
    if (p->odd) (void)hipStreamDestroy(p->odd);
    if (p->side) (void)hipStreamDestroy(p->side);
    void *ptrs[] = {p->d_scratch, p->d_slot_of, p->d_items, p->d_wpk, p->d_bias, p->d_kid, p->d_order,
                    p->d_split_begin, p->d_thr, p->d_len, p->d_dil, p->d_pad, p->d_b,
                    p->d_w, p->d_cc, p->d_ci};
    for (void *q : ptrs)
        if (q) (void)hipFree(q);
}

static rocket_status map_hip(hipError_t e) {
    if (e == hipSuccess) return ROCKET_OK;
    if (e == hipErrorOutOfMemory) return ROCKET_ERR_OOM;
    return ROCKET_ERR_HIP;
}

// Staged layout: rows with zero margins wide enough for every tap of every
// real output if that fits one workgroup's LDS (and clamped is not asked
// for), else rows with kClampMargin zeros on each side and clamped tap
// offsets.  Rows per workgroup: as many as fit the LDS budget (at least
// one).  Returns false when neither layout fits; *lds is the workgroup's LDS.
static bool choose_layout(rocket_plan *p, bool clamped, const hipDeviceProp_t &prop, int64_t *lds) {
    const int64_t limit = (int64_t)prop.sharedMemPerBlock;
    const int64_t L = p->host.L;
    auto layout = [&](int64_t stride, int64_t pad, int *rows) {
        const int64_t row_bytes = stride * p->C * (int64_t)sizeof(float);  // every channel
        const int64_t pad_bytes = pad * (int64_t)sizeof(float);
        *rows = (int)std::max<int64_t>(
            1, std::min<int64_t>(kMaxRowsPerBlock, (kRowsLdsBudget - pad_bytes) / row_bytes));
        return *rows * row_bytes + pad_bytes;
    };
    if (!clamped && p->host.row_stride > 0 &&
        (*lds = layout(p->host.row_stride, p->host.tail_pad, &p->rows_per_block)) <= limit) {
        p->halo_lo = p->host.halo_lo;
        p->row_stride = p->host.row_stride;
        p->tail_pad = p->host.tail_pad;
        return true;
    }
    // the clamped layout: each row keeps both of its margins; zeros after
    // the last row cover the reads of lanes past O
    if ((*lds = layout(L + 2 * rocket::kClampMargin, rocket::kTile, &p->rows_per_block)) <= limit) {
        p->clamp = true;
        p->halo_lo = rocket::kClampMargin;
        p->row_stride = (int32_t)(L + 2 * rocket::kClampMargin);
        p->tail_pad = rocket::kTile;
        return true;
    }
    return false;
}

// Dynamic-LDS limits already granted to the workgroup kernels, per device.
// The limit is a process-wide attribute of each kernel function, shared by
// every plan, so it is only ever raised: a later plan with a smaller
// footprint above 64 KB must not lower it below what an earlier plan
// launches with.
constexpr int kMaxDevices = 64;
static std::mutex g_lds_attr_mu;
static int g_lds_attr[kMaxDevices][kFusedInstances + kMrInstances + kToepInstances];

static hipError_t allow_lds(int device, int64_t lds) {
    if (lds <= 64 * 1024) return hipSuccess;
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_lds_attr_mu);
    hipError_t e = hipSuccess;
    for (int sel = 0; sel < kFusedInstances + kMrInstances + kToepInstances && e == hipSuccess; ++sel) {
        int &granted = g_lds_attr[device][sel];
        if (granted >= lds) continue;
        const void *fn = sel < kFusedInstances ? fused_fn(sel)
                         : sel < kFusedInstances + kMrInstances ? mr_fn(sel - kFusedInstances)
                                                                 : toep_fn(sel - kFusedInstances - kMrInstances);
        e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e == hipSuccess) granted = (int)lds;
    }
    return e;
}

// Upload the work tables and allow the kernels the workgroup's LDS.
static hipError_t upload_tables(rocket_plan *p, int64_t lds) {
    // A launch runs the workgroups of one variant after another (per XCD),
    // and a variant's workgroups each hold 1/nsplit of its items, so the
    // variants with the most work per workgroup go first: the launch then
    // ends on the short workgroups of the light variants rather than on a
    // late start of the longest ones.
    const int nv = p->host.n_variants;
    int64_t cost[rocket::kNumVariants] = {};
    for (const ItemDesc &it : p->host.items) cost[it.variant] += it.cost;
    for (int v = 0; v < nv; ++v) p->variant_order[v] = v;
    std::stable_sort(p->variant_order, p->variant_order + nv,
                     [&](int32_t x, int32_t y) { return cost[x] > cost[y]; });
    hipError_t e = upload(p->host.items, &p->d_items);
    if (e == hipSuccess) e = upload(p->host.wpk, &p->d_wpk);
    if (e == hipSuccess) e = upload(p->host.bias, &p->d_bias);
    if (e == hipSuccess) e = upload(p->host.kid, &p->d_kid);
    if (e == hipSuccess) e = upload(p->host.order, &p->d_order);
    if (e == hipSuccess) e = upload(p->host.split_begin, &p->d_split_begin);
    if (e == hipSuccess) e = upload(p->host.thr, &p->d_thr);
    if (e == hipSuccess) e = allow_lds(p->device, lds);
    return e;
}

extern "C" rocket_status rocket_plan_create_ex(const rocket_kernels *k, int32_t L, uint32_t flags,
                                               rocket_plan **out) {
    if (!out) return ROCKET_ERR_INVALID_ARG;
    *out = nullptr;
    if ((flags & ~(ROCKET_PLAN_DIRECT | ROCKET_PLAN_CLAMPED | ROCKET_PLAN_MPV | ROCKET_PLAN_TILED |
                   ROCKET_PLAN_SERIES)) ||
        ((flags & ROCKET_PLAN_DIRECT) && (flags & (ROCKET_PLAN_CLAMPED | ROCKET_PLAN_TILED))) ||
        ((flags & ROCKET_PLAN_SERIES) &&
         (flags & (ROCKET_PLAN_DIRECT | ROCKET_PLAN_CLAMPED | ROCKET_PLAN_TILED))))
        return ROCKET_ERR_INVALID_ARG;
    rocket_status st = rocket::validate_kernels(k, L);
    if (st != ROCKET_OK) return st;
    rocket_plan *p = new (std::nothrow) rocket_plan();
    if (!p) return ROCKET_ERR_OOM;
    st = rocket::build_host_plan(k, L, &p->host);
    if (st != ROCKET_OK) {
        delete p;
        return st;
    }
    hipError_t e = hipGetDevice(&p->device);
    hipDeviceProp_t prop;
    if (e == hipSuccess) e = hipGetDeviceProperties(&prop, p->device);
    if (e != hipSuccess) {
        delete p;
        return ROCKET_ERR_HIP;
    }
    p->n_cu = prop.multiProcessorCount;
    p->mpv = (flags & ROCKET_PLAN_MPV) != 0;
    p->C = p->host.n_channels;
    p->f_cols = (int64_t)(p->mpv ? 3 : 2) * k->n_kernels;
    int64_t lds = 0;
    p->direct = (flags & ROCKET_PLAN_DIRECT) != 0;
    // short univariate series: the series-lane layout for calls with many
    // series (ROCKET_PLAN_SERIES: for every call), unless a position-tiled
    // layout is asked for; the position-tiled layout serves the rest
    const bool want_series = (flags & ROCKET_PLAN_SERIES) != 0;
    if (!p->direct && !(flags & (ROCKET_PLAN_CLAMPED | ROCKET_PLAN_TILED)) && p->C == 1 && L <= kSeriesMaxL) {
        p->series_lds = (int64_t)(L + 2 * kSeriesMargin) * kSeriesLanes * (int64_t)sizeof(float);
        if (p->series_lds <= (int64_t)prop.sharedMemPerBlock) {
            p->series = true;
            p->series_min_rows = want_series ? 0 : kSeriesMinRows;
        }
    }
    if (want_series && !p->series) {
        delete p;
        return ROCKET_ERR_INVALID_ARG;
    }
    if (!p->direct && !choose_layout(p, (flags & ROCKET_PLAN_CLAMPED) != 0, prop, &lds)) p->direct = true;
    p->lds_bytes = p->direct ? 0 : lds;
    if (p->series) {
        std::vector<int32_t> slot_of((size_t)k->n_kernels, -1);
        for (size_t q = 0; q < p->host.kid.size(); ++q)
            if (p->host.kid[q] >= 0) slot_of[(size_t)p->host.kid[q]] = (int32_t)q;
        if (std::find(slot_of.begin(), slot_of.end(), -1) != slot_of.end()) {  // every kernel has a slot
            plan_free_device(p);
            delete p;
            return ROCKET_ERR_INTERNAL;
        }
        e = upload(slot_of, &p->d_slot_of);
        for (hipEvent_t *ev : {&p->scratch_done, &p->half_full[0], &p->half_full[1], &p->half_free[0],
                               &p->half_free[1], &p->aux_done, &p->call_start, &p->odd_done})
            if (e == hipSuccess) e = hipEventCreateWithFlags(ev, hipEventDisableTiming);
        if (e == hipSuccess) e = hipStreamCreateWithFlags(&p->aux, hipStreamNonBlocking);
        if (e == hipSuccess) e = hipStreamCreateWithFlags(&p->odd, hipStreamNonBlocking);
    }
    if (!p->direct && !p->minirocket &&
        std::any_of(p->host.items.begin(), p->host.items.end(),
                    [](const rocket::ItemDesc &it) { return it.variant >= rocket::kToepVariant0; })) {
        for (hipEvent_t *ev : {&p->side_start, &p->side_done})
            if (e == hipSuccess) e = hipEventCreateWithFlags(ev, hipEventDisableTiming);
        if (e == hipSuccess) e = hipStreamCreateWithFlags(&p->side, hipStreamNonBlocking);
    }
    const int32_t K = k->n_kernels;
    p->max_len = k->max_len;
    if (e == hipSuccess) e = upload_raw(k->length, (size_t)K, &p->d_len);
    if (e == hipSuccess) e = upload_raw(k->dilation, (size_t)K, &p->d_dil);
    if (e == hipSuccess) e = upload_raw(k->padding, (size_t)K, &p->d_pad);
    if (e == hipSuccess) e = upload_raw(k->bias, (size_t)K, &p->d_b);
    if (e == hipSuccess) e = upload_raw(k->weights, (size_t)K * p->C * k->max_len, &p->d_w);
    if (e == hipSuccess && p->C > 1) e = upload_raw(k->channel_count, (size_t)K, &p->d_cc);
    if (e == hipSuccess && p->C > 1) e = upload_raw(k->channel_index, (size_t)K * p->C, &p->d_ci);
    if (!p->direct && e == hipSuccess) e = upload_tables(p, lds);
    if (e != hipSuccess) {
        plan_free_device(p);
        delete p;
        return map_hip(e);
    }
    *out = p;
    return ROCKET_OK;
}

extern "C" rocket_status rocket_minirocket_plan_create(const rocket_minirocket_params *m, uint32_t flags,
                                                       rocket_plan **out) {
    if (!out) return ROCKET_ERR_INVALID_ARG;
    *out = nullptr;
    if (flags & ~ROCKET_PLAN_CLAMPED) return ROCKET_ERR_INVALID_ARG;
    rocket_status st = rocket::validate_minirocket(m);
    if (st != ROCKET_OK) return st;
    rocket_plan *p = new (std::nothrow) rocket_plan();
    if (!p) return ROCKET_ERR_OOM;
    st = rocket::build_minirocket_plan(m, &p->host);
    if (st != ROCKET_OK) {
        delete p;
        return st;
    }
    hipError_t e = hipGetDevice(&p->device);
    hipDeviceProp_t prop;
    if (e == hipSuccess) e = hipGetDeviceProperties(&prop, p->device);
    if (e != hipSuccess) {
        delete p;
        return ROCKET_ERR_HIP;
    }
    p->n_cu = prop.multiProcessorCount;
    p->minirocket = true;
    p->C = 1;
    p->f_cols = p->host.n_features;
    int64_t lds = 0;
    if (!choose_layout(p, (flags & ROCKET_PLAN_CLAMPED) != 0, prop, &lds)) {
        // a series too long for one workgroup's LDS even with 512-zero margins
        delete p;
        return ROCKET_ERR_LENGTH;
    }
    p->lds_bytes = lds;
    e = upload_tables(p, lds);
    if (e != hipSuccess) {
        plan_free_device(p);
        delete p;
        return map_hip(e);
    }
    *out = p;
    return ROCKET_OK;
}

extern "C" rocket_status rocket_plan_create(const rocket_kernels *k, int32_t L, rocket_plan **out) {
    return rocket_plan_create_ex(k, L, ROCKET_PLAN_DEFAULT, out);
}

extern "C" void rocket_plan_destroy(rocket_plan *p) {
    if (!p) return;
    plan_free_device(p);
    delete p;
}

extern "C" int32_t rocket_checked_build(void) { return ROCKET_CHECKED ? 1 : 0; }

extern "C" rocket_status rocket_check_flags(uint32_t *flags) {
    if (!flags) return ROCKET_ERR_INVALID_ARG;
    *flags = 0;
#if ROCKET_CHECKED
    // the variable's own symbol, not its host-side name: the runtime resolves
    // the current device's copy
    if (hipDeviceSynchronize() != hipSuccess) return ROCKET_ERR_HIP;
    unsigned int v = 0;
    const unsigned int zero = 0;
    if (hipMemcpyFromSymbol(&v, HIP_SYMBOL(g_rocket_checks), sizeof(v)) != hipSuccess ||
        hipMemcpyToSymbol(HIP_SYMBOL(g_rocket_checks), &zero, sizeof(zero)) != hipSuccess)
        return ROCKET_ERR_HIP;
    *flags = v;
#endif
    return ROCKET_OK;
}

extern "C" rocket_status rocket_plan_info(const rocket_plan *p, rocket_plan_facts *out) {
    if (!p || !out) return ROCKET_ERR_INVALID_ARG;
    out->n_items = (int64_t)p->host.items.size();
    out->n_buckets = p->host.n_buckets;
    // series-lane plans: one MFMA serves 64 series, so a series costs
    // (positions x taps x groups) / 64 of them
    out->mfma_per_row = p->series ? (p->host.series_mfma_64 + kSeriesLanes / 2) / kSeriesLanes
                                  : p->host.mfma_per_row;
    out->lds_bytes = p->series ? p->series_lds : p->lds_bytes;
    out->direct = p->direct ? 1 : 0;
    out->clamped = p->clamp ? 1 : 0;
    out->features_per_kernel = p->minirocket ? 0 : (p->mpv ? 3 : 2);
    out->n_features = p->f_cols;
    out->minirocket = p->minirocket ? 1 : 0;
    out->series_lane = p->series ? 1 : 0;
    out->valu_fma_per_row = p->host.valu_fma_per_row;
    out->rows_per_block = p->direct ? 0 : (p->series ? kSeriesLanes : p->rows_per_block);
    int64_t toep = 0;
    if (!p->minirocket)
        for (const rocket::ItemDesc &it : p->host.items)
            if (it.variant >= rocket::kToepVariant0) ++toep;
    out->toeplitz_items = toep;
    return ROCKET_OK;
}

static rocket_status launch_direct(const rocket_plan *p, const float *X, int64_t n, float *F,
                                   hipStream_t s) {
    const int32_t K = p->host.n_kernels;
    const int per_block = kBlock / 64;
    const int64_t max_y = 65535;
    const int64_t max_x = INT_MAX;
    for (int64_t r0 = 0; r0 < n; r0 += max_x) {
        const int64_t nr = std::min<int64_t>(max_x, n - r0);
        for (int64_t k0 = 0; k0 < K; k0 += max_y * per_block) {
            const int64_t nk = std::min<int64_t>(max_y * per_block, K - k0);
            dim3 grid((unsigned)nr, (unsigned)((nk + per_block - 1) / per_block));
            hipLaunchKernelGGL(rocket_direct_kernel, grid, dim3(kBlock), 0, s, X, r0, p->host.L, K,
                               (int32_t)k0, p->d_len, p->d_dil, p->d_pad, p->d_b, p->d_w,
                               p->max_len, p->mpv ? 3 : 2, p->C, p->d_cc, p->d_ci, F);
            if (hipGetLastError() != hipSuccess) return ROCKET_ERR_HIP;
        }
    }
    return ROCKET_OK;
}

// The workgroup kernels (fused, MINIROCKET, series-lane) over n rows: F
// receives the features, or, for the series-lane kernel, S (s_rows rows per
// slot column).
static rocket_status launch_groups(const rocket_plan *p, bool series, const float *X, int64_t n, float *F,
                                   float *S, int64_t s_rows, hipStream_t s) {
    // enough workgroups to fill the chip several times over: split the work
    // items of a series across workgroups when there are few series
    const int64_t target = 8 * (int64_t)std::max(p->n_cu, 1);
    const int64_t row_bytes = (int64_t)p->row_stride * (int64_t)sizeof(float);  // one channel
    const int R = series ? kSeriesLanes : p->rows_per_block;
    const int64_t groups = (n + R - 1) / R;
    int li = 0;
    // ... but once there are 2 workgroups per CU, keep a few items per
    // wavefront of a workgroup in each split (on average over the variants
    // present): 2 for 4-wavefront workgroups, 4 for the 16-wavefront ones of
    // long rows (with fewer, wavefronts wait idle at the end of a workgroup
    // while others finish)
    const bool big_group = !series && row_bytes * p->C > kBigLds;
    const int min_items = big_group ? 4 * (kBigBlock / 64) : 2 * (kBlock / 64);
    const int n_var = p->host.n_variants;
    int64_t n_present = 0;
    for (int v = 0; v < n_var; ++v)
        if (p->host.split_begin[v + 1] > p->host.split_begin[v]) ++n_present;
    n_present = std::max<int64_t>(n_present, 1);
    const int64_t per_variant = (int64_t)p->host.items.size() / n_present;
    const int64_t few_groups = 2 * (int64_t)std::max(p->n_cu, 1);
    if (series) {
        // a series-lane chunk's workgroups are few and short: split them only
        // as far as about 4 workgroups per CU, so that the whole grid is
        // resident at once and no partial second round of workgroups trails
        // each chunk
        while (li + 1 < rocket::kNumSplitLayouts &&
               groups * rocket::kSplitCounts[li + 1] <= 4 * (int64_t)std::max(p->n_cu, 1) &&
               per_variant / rocket::kSplitCounts[li + 1] >= min_items)
            ++li;
    } else {
        while (li + 1 < rocket::kNumSplitLayouts && groups * rocket::kSplitCounts[li] < target &&
               (per_variant / rocket::kSplitCounts[li + 1] >= min_items ||
                groups * n_present * rocket::kSplitCounts[li] < few_groups))
            ++li;
    }
    const int nsplit = rocket::kSplitCounts[li];
    FusedArgs a;
    a.X = X;
    a.F = F;
    a.L = p->host.L;
    // F rows hold nf * K floats: per kernel (PPV, MAX[, MPV]); a MINIROCKET
    // plan's rows hold its n_features PPVs (nf = 1)
    a.K = p->minirocket ? (int32_t)p->f_cols : p->host.n_kernels;
    a.nf = p->minirocket ? 1 : (p->mpv ? 3 : 2);
    a.thr = p->d_thr;
    a.C = p->C;
    a.items = p->d_items;
    a.wpk = p->d_wpk;
    a.bias = p->d_bias;
    a.kid = p->d_kid;
    a.order = p->d_order;
    a.split_begin = p->d_split_begin + p->host.layout_off[li];
    a.nsplit = nsplit;
    a.n_variants = 0;
    // The cost order (variant_order) pays where a launch is a few rounds
    // of workgroups per CU, so that its end is a visible share of it (1,000
    // series: 2.5-3.5 % faster).  Launches of many rounds keep the index
    // order, which measured 0.2 % faster on 100,000 series; series-lane
    // chunks keep it too (their launches overlap the next chunk's on a
    // second stream, and the cost order measured 1.6 % slower there).
    const bool cost_order = !series && groups * nsplit * n_present < 128 * (int64_t)std::max(p->n_cu, 1);
    for (int i = 0; i < n_var; ++i) {
        const int v = cost_order ? p->variant_order[i] : i;
        const int32_t *sb = p->host.split_begin.data() + p->host.layout_off[li];
        if (sb[(v + 1) * nsplit] > sb[v * nsplit]) a.variants[a.n_variants++] = v;
    }
    a.halo_lo = p->halo_lo;
    a.row_stride = p->row_stride;
    a.tail_pad = p->tail_pad;
    a.rows_per_block = R;
    a.vec4 = (a.L % 4 == 0 && a.halo_lo % 4 == 0 && a.row_stride % 4 == 0 && a.tail_pad % 4 == 0 &&
              ((uintptr_t)X % 16) == 0)
                 ? 1
                 : 0;
    a.S = S;
    a.s_rows = s_rows;
    a.s_floats = series ? (int64_t)p->host.kid.size() * s_rows * a.nf : 0;
    const size_t lds = (size_t)(series ? p->series_lds : p->lds_bytes);
    const bool big = big_group;
    const int sel = (big ? 1 : 0) | (p->clamp ? 2 : 0) | (p->mpv ? 4 : 0) | (p->C > 1 ? 8 : 0);
    // ROCKET plans: the Toeplitz items' variants go to a kernel of their
    // own
    FusedArgs parts[2] = {a, a};
    const void *fns[2] = {nullptr, nullptr};
    int nparts = 0;
    if (series || p->minirocket) {
        fns[nparts++] = series ? series_fn(p->mpv) : mr_fn(sel & 3);
    } else {
        parts[0].n_variants = parts[1].n_variants = 0;
        for (int i = 0; i < a.n_variants; ++i) {
            FusedArgs &q = parts[a.variants[i] >= rocket::kToepVariant0 ? 1 : 0];
            q.variants[q.n_variants++] = a.variants[i];
        }
        if (parts[0].n_variants > 0) {
            parts[nparts] = parts[0];
            fns[nparts++] = fused_fn(sel);
        }
        if (parts[1].n_variants > 0) {
            parts[nparts] = parts[1];
            fns[nparts++] = toep_fn(sel & 7);
        }
    }
    // a Toeplitz part runs on the plan's side stream, concurrently with the
    // fused part: it starts after the caller's earlier work and the call
    // ends on the caller's stream after both
    const bool side = nparts == 2 && p->side != nullptr;
    std::unique_lock<std::mutex> side_lock(p->side_mu, std::defer_lock);
    if (side) {
        side_lock.lock();
        if (hipEventRecord(p->side_start, s) != hipSuccess || hipStreamWaitEvent(p->side, p->side_start, 0) != hipSuccess)
            return ROCKET_ERR_HIP;
    }
    rocket_status st = ROCKET_OK;
    for (int part = nparts - 1; part >= 0 && st == ROCKET_OK; --part) {
        FusedArgs &q = parts[part];
        hipStream_t sq = (side && part == 1) ? p->side : s;
        const int64_t max_rows =
            ((int64_t)INT_MAX / (nsplit * std::max(q.n_variants, 1)) / kXcds - 1) * kXcds * R;
        for (int64_t r0 = 0; r0 < n; r0 += max_rows) {
            q.row0 = r0;
            q.n_rows = std::min<int64_t>(max_rows, n - r0);
            const int64_t groups_now = (q.n_rows + R - 1) / R;
            q.groups_per_xcd = (groups_now + kXcds - 1) / kXcds;
            const unsigned nb = (unsigned)(kXcds * q.groups_per_xcd * nsplit * q.n_variants);
            void *args[] = {&q};
            if (hipLaunchKernel(fns[part], dim3(nb), dim3(big ? kBigBlock : kBlock), args, lds, sq) != hipSuccess ||
                hipGetLastError() != hipSuccess) {
                st = ROCKET_ERR_HIP;
                break;
            }
        }
    }
    // also after a failure part-way: the caller's stream waits for whatever
    // the side stream holds
    if (side && (hipEventRecord(p->side_done, p->side) != hipSuccess ||
                 hipStreamWaitEvent(s, p->side_done, 0) != hipSuccess))
        return ROCKET_ERR_HIP;
    return st;
}

// Series-lane layout: the rows go in chunks; for each chunk the series
// kernel writes the features in slot order into one half of a feature
// buffer (each slot's features of 64 consecutive series are contiguous), and
// the permutation kernel writes the chunk's F rows in the original kernel
// order, 64 kernels (64 * nf floats) at a time.  The scatter of single
// features over F rows would otherwise cost more than the dot products of
// short series.  The permutation (memory-bound) runs on the plan's own
// stream, beside the next chunk's series kernel (compute-bound) on the
// caller's; chunk i uses half i % 2, which it takes once the permutation of
// chunk i - 2 is done with it.  The call ends on the caller's stream after
// the last permutation.

// Floats of one series' slot-ordered features.
static int64_t series_slot_row_floats(const rocket_plan *p) {
    return (int64_t)p->host.kid.size() * (p->mpv ? 3 : 2);
}

// Rows per chunk for halves of at most half_bytes (a multiple of 64, at
// most 8,192 and no more than the call needs); 0 when not even 64 series fit.
static int64_t series_chunk_rows(const rocket_plan *p, int64_t n, size_t half_bytes) {
    const int64_t row_bytes = std::max<int64_t>(series_slot_row_floats(p), 1) * (int64_t)sizeof(float);
    int64_t chunk = (int64_t)(half_bytes / (size_t)row_bytes) / kSeriesLanes * kSeriesLanes;
    if (chunk < kSeriesLanes) return 0;
    chunk = std::min<int64_t>(8192, chunk);
    return std::min(chunk, (n + kSeriesLanes - 1) / kSeriesLanes * kSeriesLanes);
}

// The chunk loop over a two-half buffer of `chunk` rows per half.  Chunk i
// runs its series kernel on the caller's stream (i even) or on the plan's
// odd-chunk stream (i odd), so each stream only ever uses its own half, and
// consecutive chunks overlap; the permutations run in chunk order on the
// plan's permutation stream.  The caller holds p->scratch_mu (the plan's
// streams and events are shared by every transform of the plan).
static rocket_status enqueue_series(const rocket_plan *p, const float *X, int64_t n, float *F,
                                    hipStream_t s, float *buf, int64_t chunk) {
    const int64_t K = p->host.n_kernels;
    const int nf = p->mpv ? 3 : 2;
    const int64_t half = chunk * series_slot_row_floats(p);  // floats
    const void *pf = nf == 3 ? (const void *)rocket_slot_permute_kernel<3>
                             : (const void *)rocket_slot_permute_kernel<2>;
    // a failure part-way still ends with the tail below, so that the next
    // transform of this plan waits for whatever this one enqueued
    rocket_status st = ROCKET_OK;
    // the odd-chunk stream starts after the caller's earlier work (X ready,
    // the previous user of the buffer done)
    if (hipEventRecord(p->call_start, s) != hipSuccess || hipStreamWaitEvent(p->odd, p->call_start, 0) != hipSuccess)
        st = ROCKET_ERR_HIP;
    int i = 0;
    for (int64_t r0 = 0; r0 < n && st == ROCKET_OK; r0 += chunk, ++i) {
        const int h = i & 1;
        hipStream_t sh = h ? p->odd : s;
        const int64_t m = std::min(chunk, n - r0);
        float *Sh = buf + h * half;
        if (i >= 2 && hipStreamWaitEvent(sh, p->half_free[h], 0) != hipSuccess) {
            st = ROCKET_ERR_HIP;
            break;
        }
        st = launch_groups(p, true, X + r0 * p->host.L, m, nullptr, Sh, chunk, sh);
        if (st != ROCKET_OK) break;
        if (hipEventRecord(p->half_full[h], sh) != hipSuccess ||
            hipStreamWaitEvent(p->aux, p->half_full[h], 0) != hipSuccess) {
            st = ROCKET_ERR_HIP;
            break;
        }
        const int64_t tiles = ((K + 63) / 64) * ((m + 63) / 64);
        // one workgroup per CU, striding over the tiles: the permutation then
        // moves its bytes at a modest rate over the whole of the next chunk's
        // series kernel (a full grid moves them in a burst that stalls it)
        const dim3 grid((unsigned)std::min<int64_t>(tiles, std::max(p->n_cu, 1)));
        const float *S = Sh;
        const int32_t *slot_of = p->d_slot_of;
        int32_t K32 = (int32_t)K;
        int64_t s_rows = chunk;
        float *Fc = F + r0 * K * nf;
        int64_t mm = m;
        int32_t n_slots = (int32_t)p->host.kid.size();
        void *args[] = {(void *)&S, &s_rows, (void *)&slot_of, &K32, (void *)&mm, &Fc, &n_slots};
        if (hipLaunchKernel(pf, grid, dim3(kBlock), args, 0, p->aux) != hipSuccess ||
            hipGetLastError() != hipSuccess || hipEventRecord(p->half_free[h], p->aux) != hipSuccess) {
            st = ROCKET_ERR_HIP;
            break;
        }
    }
    const bool tail_ok = hipEventRecord(p->aux_done, p->aux) == hipSuccess &&
                         hipStreamWaitEvent(s, p->aux_done, 0) == hipSuccess &&
                         hipEventRecord(p->odd_done, p->odd) == hipSuccess &&
                         hipStreamWaitEvent(s, p->odd_done, 0) == hipSuccess;
    if (st != ROCKET_OK) return st;
    return tail_ok ? ROCKET_OK : ROCKET_ERR_HIP;
}

// The plan's own feature buffer: at most 1 GiB (halves of up to 8,192 rows),
// allocated on first use and grown as needed; transforms on different
// streams take turns on it (each waits for the previous user's event).
static rocket_status launch_series(const rocket_plan *p, const float *X, int64_t n, float *F,
                                   hipStream_t s) {
    const int64_t chunk = std::max<int64_t>(kSeriesLanes, series_chunk_rows(p, n, (size_t)1 << 29));
    const size_t need = (size_t)(2 * chunk * series_slot_row_floats(p)) * sizeof(float);
    std::lock_guard<std::mutex> lock(p->scratch_mu);
    if (p->scratch_bytes < need) {
        // hipFree waits for the work that still uses the old buffer
        if (p->d_scratch && hipFree(p->d_scratch) != hipSuccess) return ROCKET_ERR_HIP;
        p->d_scratch = nullptr;
        p->scratch_bytes = 0;
        if (hipMalloc(&p->d_scratch, need) != hipSuccess) return ROCKET_ERR_OOM;
        p->scratch_bytes = need;
    }
    // the previous transform of this plan (on any stream) is done with it
    if (hipStreamWaitEvent(s, p->scratch_done, 0) != hipSuccess) return ROCKET_ERR_HIP;
    const rocket_status st = enqueue_series(p, X, n, F, s, p->d_scratch, chunk);
    // recorded after the tail, also after a failure part-way
    const bool rec_ok = hipEventRecord(p->scratch_done, s) == hipSuccess;
    if (st != ROCKET_OK) return st;
    return rec_ok ? ROCKET_OK : ROCKET_ERR_HIP;
}

// ---------------------------------------------------------------------------
// Static scratch of rocket_transform_plan_noalloc: the series-lane feature
// buffer of callers that cannot allocate device memory.  Every GPU the
// library runs on holds its own copy of the array (from the first use of the
// library's code there until the process ends).  Host code uses the device
// address that hipGetSymbolAddress returns for the current device, never the
// array's name (a host-side stand-in).
// ---------------------------------------------------------------------------
constexpr size_t kNoAllocScratchBytes = (size_t)64 << 20;  // ROCKET_NOALLOC_SCRATCH_BYTES
static_assert(kNoAllocScratchBytes == (size_t)ROCKET_NOALLOC_SCRATCH_BYTES, "header and library agree");
static __device__ __align__(256) float scratch[kNoAllocScratchBytes / sizeof(float)];

static std::mutex g_scratch_mu;
static float *g_scratch_ptr[kMaxDevices];

// The device address of `scratch` on `device` (which must be current),
// looked up once per device.
static rocket_status noalloc_scratch(int device, float **out) {
    if (device < 0 || device >= kMaxDevices) return ROCKET_ERR_INVALID_ARG;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[device]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return ROCKET_ERR_HIP;
        g_scratch_ptr[device] = (float *)ptr;
    }
    *out = g_scratch_ptr[device];
    return ROCKET_OK;
}

// The series-lane chunk loop over the static scratch (two halves of 32 MiB).
static rocket_status launch_series_noalloc(const rocket_plan *p, const float *X, int64_t n, float *F,
                                           hipStream_t s, float *buf) {
    const int64_t chunk = series_chunk_rows(p, n, kNoAllocScratchBytes / 2);
    if (chunk == 0) return ROCKET_ERR_SCRATCH;
    std::lock_guard<std::mutex> lock(p->scratch_mu);
    return enqueue_series(p, X, n, F, s, buf, chunk);
}

static rocket_status launch_fused(const rocket_plan *p, const float *X, int64_t n, float *F,
                                  hipStream_t s) {
    return (p->series && n >= p->series_min_rows) ? launch_series(p, X, n, F, s)
                                                  : launch_groups(p, false, X, n, F, nullptr, 0, s);
}

// The plan's streams, events and tables live on the device it was created
// on: that device must be the current one.
static rocket_status check_plan_device(const rocket_plan *p) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return ROCKET_ERR_HIP;
    return dev == p->device ? ROCKET_OK : ROCKET_ERR_INVALID_ARG;
}

extern "C" rocket_status rocket_transform_plan(const rocket_plan *p, const float *X_dev, int64_t n,
                                               float *F_dev, void *hip_stream) {
    if (!p || n < 0) return ROCKET_ERR_INVALID_ARG;
    const rocket_status dst = check_plan_device(p);
    if (dst != ROCKET_OK) return dst;
    if (n == 0) return ROCKET_OK;
    if (!X_dev || !F_dev) return ROCKET_ERR_INVALID_ARG;
    hipStream_t s = (hipStream_t)hip_stream;
    return p->direct ? launch_direct(p, X_dev, n, F_dev, s) : launch_fused(p, X_dev, n, F_dev, s);
}

extern "C" rocket_status rocket_transform_plan_noalloc(const rocket_plan *p, const float *X_dev, int64_t n,
                                                       float *F_dev, void *hip_stream) {
    if (!p || n < 0) return ROCKET_ERR_INVALID_ARG;
    const rocket_status dst = check_plan_device(p);
    if (dst != ROCKET_OK) return dst;
    const int dev = p->device;
    float *buf = nullptr;
    const rocket_status st = noalloc_scratch(dev, &buf);
    if (st != ROCKET_OK) return st;
    if (n == 0) return ROCKET_OK;
    if (!X_dev || !F_dev) return ROCKET_ERR_INVALID_ARG;
    hipStream_t s = (hipStream_t)hip_stream;
    if (p->direct) return launch_direct(p, X_dev, n, F_dev, s);
    if (p->series && n >= p->series_min_rows) return launch_series_noalloc(p, X_dev, n, F_dev, s, buf);
    return launch_groups(p, false, X_dev, n, F_dev, nullptr, 0, s);
}

// Host-to-host transform with copies overlapped against the transform:
// batch i uses X and F staging buffer i % 2.  Its copy in waits until the
// transform of batch i-2 (the last reader of that X buffer) is done; its
// transform waits for its copy in and for the copy out of batch i-2 (the
// last reader of that F buffer); its copy out waits for its transform.
extern "C" rocket_status rocket_transform_host(const rocket_plan *p, const float *X_host, int64_t n,
                                               float *F_host, int64_t batch_rows,
                                               void *hip_stream) {
    if (!p || n < 0 || batch_rows < 0) return ROCKET_ERR_INVALID_ARG;
    const rocket_status dst = check_plan_device(p);
    if (dst != ROCKET_OK) return dst;
    if (n == 0) return ROCKET_OK;
    if (!X_host || !F_host) return ROCKET_ERR_INVALID_ARG;
    const int64_t L = (int64_t)p->host.L * p->C;  // floats per series (every channel)
    const int64_t K2 = p->f_cols;  // floats per feature row
    int64_t B = batch_rows;
    // default: about 8 batches, so copies have neighbours to overlap with,
    // each within 256 MiB of staging
    if (B == 0)
        B = std::max<int64_t>(1, std::min<int64_t>((n + 7) / 8, (int64_t)(256 << 20) / ((L + K2) * 4)));
    B = std::min(B, n);
    const int64_t nb = (n + B - 1) / B;
    hipStream_t sc = (hipStream_t)hip_stream;
    hipStream_t s_in = nullptr, s_out = nullptr;
    float *dX[2] = {nullptr, nullptr}, *dF[2] = {nullptr, nullptr};
    hipEvent_t ev_in[2] = {}, ev_tr[2] = {}, ev_out[2] = {};
    rocket_status st = ROCKET_OK;
    hipError_t e = hipStreamCreateWithFlags(&s_in, hipStreamNonBlocking);
    if (e == hipSuccess) e = hipStreamCreateWithFlags(&s_out, hipStreamNonBlocking);
    for (int j = 0; j < 2 && e == hipSuccess; ++j) {
        e = hipMalloc((void **)&dX[j], (size_t)(B * L * 4));
        if (e == hipSuccess) e = hipMalloc((void **)&dF[j], (size_t)(B * K2 * 4));
        if (e == hipSuccess) e = hipEventCreateWithFlags(&ev_in[j], hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&ev_tr[j], hipEventDisableTiming);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&ev_out[j], hipEventDisableTiming);
    }
    for (int64_t i = 0; i < nb && e == hipSuccess && st == ROCKET_OK; ++i) {
        const int j = (int)(i & 1);
        const int64_t r0 = i * B, m = std::min(B, n - r0);
        if (i >= 2) e = hipStreamWaitEvent(s_in, ev_tr[j], 0);
        if (e == hipSuccess)
            e = hipMemcpyAsync(dX[j], X_host + r0 * L, (size_t)(m * L * 4), hipMemcpyHostToDevice, s_in);
        if (e == hipSuccess) e = hipEventRecord(ev_in[j], s_in);
        if (e == hipSuccess) e = hipStreamWaitEvent(sc, ev_in[j], 0);
        if (e == hipSuccess && i >= 2) e = hipStreamWaitEvent(sc, ev_out[j], 0);
        if (e == hipSuccess) st = rocket_transform_plan(p, dX[j], m, dF[j], sc);
        if (e == hipSuccess && st == ROCKET_OK) e = hipEventRecord(ev_tr[j], sc);
        if (e == hipSuccess && st == ROCKET_OK) e = hipStreamWaitEvent(s_out, ev_tr[j], 0);
        if (e == hipSuccess && st == ROCKET_OK)
            e = hipMemcpyAsync(F_host + r0 * K2, dF[j], (size_t)(m * K2 * 4), hipMemcpyDeviceToHost, s_out);
        if (e == hipSuccess && st == ROCKET_OK) e = hipEventRecord(ev_out[j], s_out);
    }
    // drain every stream before the staging buffers go away
    const hipError_t e1 = s_in ? hipStreamSynchronize(s_in) : hipSuccess;
    const hipError_t e2 = hipStreamSynchronize(sc);
    const hipError_t e3 = s_out ? hipStreamSynchronize(s_out) : hipSuccess;
    for (int j = 0; j < 2; ++j) {
        if (dX[j]) (void)hipFree(dX[j]);
        if (dF[j]) (void)hipFree(dF[j]);
        if (ev_in[j]) (void)hipEventDestroy(ev_in[j]);
        if (ev_tr[j]) (void)hipEventDestroy(ev_tr[j]);
        if (ev_out[j]) (void)hipEventDestroy(ev_out[j]);
    }
    if (s_in) (void)hipStreamDestroy(s_in);
    if (s_out) (void)hipStreamDestroy(s_out);
    if (st != ROCKET_OK) return st;
    if (e != hipSuccess) return map_hip(e);
    if (e1 != hipSuccess || e2 != hipSuccess || e3 != hipSuccess) return ROCKET_ERR_HIP;
    return ROCKET_OK;
}

extern "C" rocket_status rocket_transform(const float *X_dev, int64_t n, int32_t L,
                                          const rocket_kernels *k, float *F_dev, void *hip_stream) {
    if (n < 0) return ROCKET_ERR_INVALID_ARG;
    if (n > 0 && (!X_dev || !F_dev)) return ROCKET_ERR_INVALID_ARG;
    rocket_status st = rocket::validate_kernels(k, L);
    if (st != ROCKET_OK) return st;
    if (n == 0) return ROCKET_OK;
    rocket_plan *p = nullptr;
    st = rocket_plan_create(k, L, &p);
    if (st != ROCKET_OK) return st;
    st = rocket_transform_plan(p, X_dev, n, F_dev, hip_stream);
    const hipError_t e = hipStreamSynchronize((hipStream_t)hip_stream);
    rocket_plan_destroy(p);
    if (st != ROCKET_OK) return st;
    return e == hipSuccess ? ROCKET_OK : ROCKET_ERR_HIP;
}
