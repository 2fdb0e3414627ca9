// Device helpers shared by the MFMA tile kernels (gram.hip, factor.hip,
// static.hip).
#pragma once

#include <hip/hip_runtime.h>

namespace mfac {
namespace {

typedef double v4d __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));

// Row, within a 16 x 16 MFMA output tile, of accumulator register r of lane l
// (the column is l % 16 for both). fp64 16x16x4: rows l/16 + 4r; fp32
// 16x16x4: rows 4(l/16) + r (four consecutive rows per lane).
__device__ __forceinline__ int mfma64_row(int lane, int r) { return (lane >> 4) + 4 * r; }
__device__ __forceinline__ int mfma32_row(int lane, int r) { return 4 * (lane >> 4) + r; }

// Work-groups are dispatched round-robin over the 8 XCDs (each with its own
// L2). Remap so that consecutive logical indices share an XCD: the tiles of
// one matrix then run on one XCD and share its L2 copy of the operands.
__device__ __forceinline__ int xcd_remap(int p, int n) {
    if (n % 8) return p;
    return (p % 8) * (n / 8) + p / 8;
}

// Component t (a compile-time constant after unrolling) of a float4.
__device__ __forceinline__ float f4_at(const float4& v, int t) { return t == 0 ? v.x : t == 1 ? v.y : t == 2 ? v.z : v.w; }

// v where ok, else zeros; element-wise so the value stays in registers.
__device__ __forceinline__ float4 keep4(bool ok, float4 v) {
    return make_float4(ok ? v.x : 0.f, ok ? v.y : 0.f, ok ? v.z : 0.f, ok ? v.w : 0.f);
}

}  // namespace
}  // namespace mfac
