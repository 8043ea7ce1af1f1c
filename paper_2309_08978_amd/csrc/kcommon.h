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

}  // namespace nnjit
