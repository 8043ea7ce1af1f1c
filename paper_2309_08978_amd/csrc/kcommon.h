// Device-side helpers shared by the GEMM and GEMV kernel templates.
#pragma once

#include <hip/hip_runtime.h>
#include "internal.h"

namespace nnjit {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// Workgroups of one dispatch are handed to the 8 XCDs of the chip in turn
// (flat id 0 -> XCD 0, 1 -> XCD 1, ...), and each XCD has its own L2.  This
// renumbering makes ids that are consecutive in the new numbering run on the
// same XCD, so tiles that share operand rows or columns share an L2.  It is a
// bijection of [0, G) for any G.
__device__ __forceinline__ int xcd_remap(int flat, int G) {
    const int q = G >> 3, r = G & 7;
    const int xcd = flat & 7, local = flat >> 3;
    return (xcd < r) ? xcd * (q + 1) + local : r * (q + 1) + (xcd - r) * q + local;
}

// Tile of a GEMM launch from its index in the (XCD-renumbered) order: tiles
// run in groups of G tile rows, each group column by column (G rows of one
// tile column, then the next column), so that the run of consecutive tiles an
// XCD holds at once covers about G rows and (run / G) columns of tiles -- A
// rows and B columns that the XCD's L2 shares -- instead of one whole column
// of tiles, which makes every XCD read all of A.  G = tiles_m is the plain
// column-major order.  A bijection of [0, tiles_m * tiles_n).
__device__ __forceinline__ void tile_of(int tile, int tiles_m, int tiles_n, int G, int &tm, int &tn)
{
    const int span = G * tiles_n;
    const int g = tile / span, local = tile - g * span;
    const int rows = min(G, tiles_m - g * G);
    tm = g * G + local % rows;
    tn = local / rows;
}

// Wait until at most N vector memory operations of this wave are pending.
template <int N>
__device__ __forceinline__ void wait_vmcnt()
{
    static_assert(N >= 0 && N <= 63, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// 16 bytes per lane from global memory to LDS: lane l's bytes land at LDS
// address lds + 16 l (lds must be wave-uniform).  Issued as inline assembly
// so that the compiler does not treat the copy as an LDS store of unknown
// target and wait for every copy in flight before each LDS read; the kernel
// orders the copies against the reads itself (counted vmcnt waits plus a
// barrier).  Vector memory loads complete in issue order, so the compiler's
// own vmcnt waits stay correct with these extra loads in the queue.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"   // m0 is written on purpose
__device__ __forceinline__ void copy16_to_lds(const void *src, unsigned lds)
{
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(lds) : "memory", "m0");
}
#pragma clang diagnostic pop

// Workgroup barrier for the copy pipeline: this wave's LDS reads are complete
// and every wave has arrived.  Global memory ordering is not needed here (the
// copies are waited for by count), so unlike __syncthreads() it does not
// wait for all outstanding vector memory operations.
__device__ __forceinline__ void lds_barrier()
{
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

}  // namespace nnjit
