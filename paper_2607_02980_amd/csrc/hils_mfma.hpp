// gfx950 MFMA helpers for the bf16 kernels.
//
// v_mfma_f32_16x16x32_bf16 (D = A*B + C, A 16x32, B 32x16, D 16x16), lane l:
//   A: 8 values A[m = l%16][k = (l/16)*8 + j]
//   B: 8 values B[k = (l/16)*8 + j][n = l%16]
//   D: 4 values D[m = (l/16)*4 + i][n = l%16]
// (layout checked on the hardware against a host product of random integers).
#pragma once

#include <hip/hip_runtime.h>

#include "hils_device.hpp"

namespace hils {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) float f32x4;

__device__ __forceinline__ f32x4 mfma16x16x32(const bf16x8& a, const bf16x8& b, const f32x4& c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 ld_bf16x8(const void* p) { return *reinterpret_cast<const bf16x8*>(p); }

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }

// Round 8 floats to bf16 (nearest-even) into one MFMA operand.
__device__ __forceinline__ bf16x8 pack_bf16x8(const float* x) {
    uint32_t w[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const uint32_t lo = from_f32<bf16>(x[2 * t]).bits, hi = from_f32<bf16>(x[2 * t + 1]).bits;
        w[t] = lo | (hi << 16);
    }
    return as_bf16x8(make_uint4(w[0], w[1], w[2], w[3]));
}

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// Block index remap so that consecutive logical blocks run on the same XCD
// (workgroups are dispatched round-robin over the 8 XCDs, each with its own
// L2): logical block = (physical % 8) * ceil(n/8) + physical / 8.
__device__ __forceinline__ int xcd_remap(int physical, int n) {
    const int per = (n + 7) / 8;
    const int x = physical % 8, r = physical / 8;
    const int full = n % 8 == 0 ? 8 : n % 8;  // XCDs that get `per` blocks
    int logical;
    if (x < full)
        logical = x * per + r;
    else
        logical = full * per + (x - full) * (per - 1) + r;
    return logical;
}

}  // namespace hils
