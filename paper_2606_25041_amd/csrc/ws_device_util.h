// Device helpers shared by the attention kernels (ws_kernels.hip) and the
// gradient kernels (ws_bwd.hip): vector types, wave-level reductions,
// uniform loads, multiply-shift division, key ends of a row, bf16 packing,
// explicit wait counts and barriers, the LDS tile swizzle and the
// direct-to-LDS loads.  Device code only; included inside no namespace.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ws_kernels.h"

namespace ws {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));


typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// max / sum of a value over lanes l and l^32 (same query column, other keys)
__device__ __forceinline__ float halves_max(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float halves_sum(float x) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Read-only metadata (page tables, cache lengths, block offsets) read at a
// wave-uniform index goes through the constant address space, so it becomes a
// scalar load: it does not count against the vector-memory counter that the
// tile pipeline waits on.
typedef const __attribute__((address_space(4))) int32_t cint32;
__device__ __forceinline__ int ld_uniform(const int32_t *p, int64_t i) { return ((const cint32 *)p)[i]; }

// n / d for n < 2^31 with the host-computed divider of d
__device__ __forceinline__ uint32_t fastdiv(uint32_t n, FastDiv f) {
    return (uint32_t)(((uint64_t)n * f.mul) >> f.shift);
}

// End (exclusive) of the keys token i of a prefill sees: the end of its
// block (the first offset > i), or, when the block ends in a token-causal
// segment starting at ts (text != nullptr, [nb] starts of this stream),
// max(ts, i + 1).  Non-decreasing in i.
template <bool UNIFORM>
__device__ __forceinline__ int row_key_end(const int32_t *off, const int32_t *text, int nb, int i) {
    auto at = [&](const int32_t *p, int k) { return UNIFORM ? ld_uniform(p, k) : p[k]; };
    int lo = 1, hi = nb;  // answer index in [1, nb]
    while (lo < hi) {
        int mid = (lo + hi) >> 1;
        if (at(off, mid) > i) hi = mid; else lo = mid + 1;
    }
    return text ? max(at(text, lo - 1), i + 1) : at(off, lo);
}

// Two floats rounded to bf16 (RNE), lo in the low half: one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    typedef __bf16 b16x2 __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){lo, hi}, b16x2));
}

// s_waitcnt with vector-memory count <= N and LDS/scalar count = 0 (the export
// count is not waited on).  gfx9 encoding: vmcnt[3:0], expcnt[6:4],
// lgkmcnt[11:8], vmcnt[5:4] in bits [15:14].
template <int N>
__device__ __forceinline__ void wait_vm_lgkm() {
    static_assert(N >= 0 && N < 64, "vmcnt has 6 bits");
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
}

// Work-group barrier without the memory fence of __syncthreads(): that fence
// also waits for every direct-to-LDS load in flight, and the pipeline keeps
// two tiles in flight across each barrier.  The explicit waits in front of
// each barrier make the LDS data it publishes complete.
__device__ __forceinline__ void wg_barrier() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// LDS layout of a key tile: rows of D bf16, no padding; 16-byte chunk c of
// key row r sits in slot c ^ swz(r) of that row.  With this swizzle the K
// reads of S^T (16 consecutive rows, one chunk) and the V transpose reads of
// O^T (4 rows x 4 chunks per 32 lanes) each touch 16 distinct 16-byte bank
// groups.
template <int D>
__device__ __forceinline__ int swz(int r) {
    if constexpr (D == 128) return 4 * (r & 3) + ((r >> 2) & 3);   // 256-byte rows
    else return 4 * ((r >> 1) & 1) + ((r >> 2) & 3);                // 128-byte rows, two per bank line
}

typedef __attribute__((address_space(3))) char lds_char;

// LDS byte address of a pointer into a __shared__ array.
__device__ __forceinline__ uint32_t lds_addr(const char *p) {
    return (uint32_t)(uintptr_t)(const lds_char *)p;
}

// 16 bytes per lane from global memory straight into LDS at lds + 16 * lane
// (lds wave-uniform, in M0).  Written as inline assembly on purpose: with the
// load-to-LDS builtin in a loop the compiler's wait-count model turns every
// later LDS-read wait into a full drain (lgkmcnt(0)), which serialises the
// MFMA blocks.  These loads are invisible to that model; the kernel waits
// for them itself (wait_vm_lgkm before each barrier that publishes a tile).
// M0 is written here; no other code in this file uses M0, so clobbering it
// is safe (clang warns because M0 is a reserved register).
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// Per-lane 64-bit address:
__device__ __forceinline__ void dma16(const char *g, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" :: "v"(g), "s"(lds) : "memory", "m0");
}
// Wave-uniform base + per-lane 32-bit byte offset:
__device__ __forceinline__ void dma16s(const char *base, uint32_t off, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" :: "v"(off), "s"(base), "s"(lds) : "memory", "m0");
}
#pragma clang diagnostic pop


}  // namespace
}  // namespace ws
