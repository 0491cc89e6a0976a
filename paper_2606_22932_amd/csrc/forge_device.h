// Device-side helpers shared by the HIP translation units of libforge (gfx950 only):
// vector types, LDS barrier, bf16 packing, non-temporal accesses and the XCD-aware
// workgroup-to-tile mapping.
#pragma once

#include "forge_internal.h"

namespace forge_impl {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef short v4i16_t __attribute__((ext_vector_type(4)));

// Buffer offset of a DMA piece that must read zero.  Tensors hold fewer than 2^31
// elements and d_in, d_out are multiples of 8, so a chunk spans at most 2^32 - 16 bytes:
// this offset is past the end of every chunk's buffer.
constexpr uint32_t OOR_OFFSET = 0xFFFFFFF0u;

// ------------------------------------------------------------------------ small helpers

__device__ __forceinline__ void lds_barrier()
{
    // Wait for this wave's LDS traffic only, then barrier: outstanding global loads (the
    // stream waves' prefetch) stay in flight across it.
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__device__ __forceinline__ float bf_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf_hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi)
{
    bf16x2_t r = {(__bf16)lo, (__bf16)hi};   // v_cvt_pk_bf16_f32: round to nearest even
    return __builtin_bit_cast(uint32_t, r);
}

template <typename T> __device__ __forceinline__ T ld_nt(const void *p)
{
    return __builtin_nontemporal_load(reinterpret_cast<const T *>(p));
}
template <typename T> __device__ __forceinline__ void st_nt(void *p, T v)
{
    __builtin_nontemporal_store(v, reinterpret_cast<T *>(p));
}

// Workgroups are dispatched round-robin over the 8 XCDs (each with its own L2): give
// each XCD a contiguous run of the ntiles tiles of a launch.
__device__ __forceinline__ int xcd_remap(int bid, int ntiles)
{
    const int k = ntiles >> 3, r = ntiles & 7;
    const int x = bid & 7, s = bid >> 3;
    return (x < r) ? x * (k + 1) + s : r * (k + 1) + (x - r) * k + s;
}

// Tile t of one matrix in groups of `group_p` tile rows, so that concurrently resident
// tiles share their dY row slabs and X column slabs.
__device__ __forceinline__ void raster(int t, int tiles_p, int tiles_q, int group_p, int &tp, int &tq)
{
    const int per_group = group_p * tiles_q;
    const int g = t / per_group;
    const int first = g * group_p;
    const int gsz = min(group_p, tiles_p - first);
    const int within = t - g * per_group;
    tp = first + within % gsz;
    tq = within / gsz;
}

__device__ __forceinline__ void tile_of(int bid, int ntiles, int tiles_p, int tiles_q,
                                        int group_p, int &tp, int &tq)
{
    raster(xcd_remap(bid, ntiles), tiles_p, tiles_q, group_p, tp, tq);
}

}  // namespace forge_impl
