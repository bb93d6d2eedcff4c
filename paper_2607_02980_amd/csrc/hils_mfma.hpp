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

// 16-byte global load marked non-temporal (data streamed once: it is not kept in
// the caches at the expense of data that is reused).
__device__ __forceinline__ uint4 ld_stream16(const void* p) {
    typedef unsigned v4u __attribute__((ext_vector_type(4)));
    const v4u t = __builtin_nontemporal_load(reinterpret_cast<const v4u*>(p));
    return make_uint4(t[0], t[1], t[2], t[3]);
}
__device__ __forceinline__ bf16x8 ld_stream_bf16x8(const void* p) {
    typedef unsigned v4u __attribute__((ext_vector_type(4)));
    return __builtin_bit_cast(bf16x8, __builtin_nontemporal_load(reinterpret_cast<const v4u*>(p)));
}

// Round 8 floats to bf16 (nearest-even) into one MFMA operand.
__device__ __forceinline__ bf16x8 pack_bf16x8(const float* x) {
    bf16x8 r;
#pragma unroll
    for (int j = 0; j < 8; ++j) r[j] = static_cast<__bf16>(x[j]);
    return r;
}

// ds_read_b64_tr_b16 (gfx950 LDS transpose read).  In every 16-lane group,
// lane t receives element t%4 of the 8-byte words addressed by lanes 4j + t/4
// of its group, j = 0..3 (layout checked on the hardware).
typedef short v4i16 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ v4i16 lds_read_tr16(const void* p) {
    typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(p));
}

// MFMA operand from a row-major LDS tile X[k][n] (row stride ld elements, rows
// 8-byte aligned): lane l receives X[k0 + (l/16)*8 + j][n0 + l%16], j = 0..7,
// i.e. a B operand over (k, n), or an A operand over (m = n, k).
template <typename E>
__device__ __forceinline__ bf16x8 tr_operand(const E* X, int ld, int k0, int n0, int lane) {
    const int g = lane / 16, s = lane % 16;
    const E* p = X + (size_t)(k0 + g * 8 + s / 4) * ld + n0 + 4 * (s % 4);
    const v4i16 a = lds_read_tr16(p);
    const v4i16 b = lds_read_tr16(p + 4 * ld);
    typedef short v8i16 __attribute__((ext_vector_type(8)));
    const v8i16 c = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    return __builtin_bit_cast(bf16x8, c);
}

// The same over the 32 rows k0 + {4g..4g+3} U {16+4g..16+4g+3} (g = l/16): the
// key order in which a pair of 16x16 accumulator blocks holds 32 keys.
template <typename E>
__device__ __forceinline__ bf16x8 tr_operand_perm(const E* X, int ld, int k0, int n0, int lane) {
    const int g = lane / 16, s = lane % 16;
    const E* p = X + (size_t)(k0 + g * 4 + s / 4) * ld + n0 + 4 * (s % 4);
    const v4i16 a = lds_read_tr16(p);
    const v4i16 b = lds_read_tr16(p + 16 * ld);
    typedef short v8i16 __attribute__((ext_vector_type(8)));
    const v8i16 c = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    return __builtin_bit_cast(bf16x8, c);
}

// Staggered LDS tiles: rows of W = 64 or 128 bf16 at a stride of W + 16, rows with
// r % 8 >= 4 shifted by 8 more.  Relative to the 128-byte LDS bank cycle (32 banks
// of 4 bytes) rows r = 0..7 then start at 16-byte slots 0, 2, 4, 6, 1, 3, 5, 7, so
// that row-wise 16-byte operand reads (8 lanes = 8 rows per cycle) and transposing
// reads (16 lanes = 4 rows x 32 bytes per cycle) are both free of bank conflicts,
// which no uniform row padding gives (+8 suits the first, +16 the second); unlike
// an XOR swizzle, offsets along a row stay linear, so that the column steps of
// unrolled loops fold into the instruction offsets.
template <int W>
__device__ __forceinline__ int st_off(int r, int c) {
    return r * (W + 16) + 8 * ((r >> 2) & 1) + c;
}
template <int W>
constexpr int st_size(int rows) {
    return rows * (W + 16) + 8;
}
// row_operand / tr_operand of a staggered tile (r0, k0 multiples of 8: the shift of
// a row then depends on the lane alone, and the compiler keeps one address per lane)
template <int W>
__device__ __forceinline__ bf16x8 row_operand_st(const bf16* X, int r0, int k0, int lane) {
    return ld_bf16x8(X + (r0 + lane % 16) * (W + 16) + 8 * ((lane >> 2) & 1) + k0 + (lane / 16) * 8);
}
template <int W>
__device__ __forceinline__ bf16x8 tr_operand_st(const bf16* X, int k0, int n0, int lane) {
    const int g = lane / 16, s = lane % 16;
    // rows k0 + 8g + s/4 have r % 8 < 4; the second read's rows (+4) have r % 8 >= 4
    const bf16* p = X + (k0 + g * 8 + s / 4) * (W + 16) + n0 + 4 * (s % 4);
    const v4i16 a = lds_read_tr16(p);
    const v4i16 b = lds_read_tr16(p + 4 * (W + 16) + 8);
    typedef short v8i16 __attribute__((ext_vector_type(8)));
    const v8i16 v = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    return __builtin_bit_cast(bf16x8, v);
}
// tr_operand_perm of a staggered tile (k0 a multiple of 8)
template <int W>
__device__ __forceinline__ bf16x8 tr_operand_perm_st(const bf16* X, int k0, int n0, int lane) {
    const int g = lane / 16, s = lane % 16;
    // rows k0 + 4g + s/4: r % 8 >= 4 for odd g
    const bf16* p = X + (k0 + g * 4 + s / 4) * (W + 16) + 8 * (g & 1) + n0 + 4 * (s % 4);
    const v4i16 a = lds_read_tr16(p);
    const v4i16 b = lds_read_tr16(p + 16 * (W + 16));  // rows + 16: the same r % 8
    typedef short v8i16 __attribute__((ext_vector_type(8)));
    const v8i16 v = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    return __builtin_bit_cast(bf16x8, v);
}

// "Lane order" of a D-vector held as O^T accumulators (DB = D/16 blocks, lane
// group lg = l/16 holding d = 16 db + 4 lg + i): element d is stored at position
// 32 (db / 2) + 8 lg + 4 (db % 2) + i.  A lane moves its 32 values as D/32
// 16-byte pieces, and piece t of the four lanes of a row is one contiguous
// 64-byte span (positions 32 t .. 32 t + 31), so every access instruction covers
// whole 64-byte runs of each row.  Used for the per-slot partial vectors that
// one kernel writes and another reads in the same lane layout.
template <int D>
__device__ __forceinline__ void store_lane_order(bf16* row, const f32x4* o, int lg) {
    uint32_t w[D / 8];
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
        w[2 * db] = pack_bf16x2(o[db][0], o[db][1]);
        w[2 * db + 1] = pack_bf16x2(o[db][2], o[db][3]);
    }
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
#pragma unroll
    for (int t = 0; t < D / 32; ++t) {
        const u32x4 v = {w[4 * t], w[4 * t + 1], w[4 * t + 2], w[4 * t + 3]};
        *reinterpret_cast<u32x4*>(row + 32 * t + 8 * lg) = v;
    }
}

// Loads a lane-order vector; fma_lane_order adds wgt times it to acc (O^T layout).
template <int D>
__device__ __forceinline__ void load_lane_order(const bf16* row, int lg, uint4* x) {
#pragma unroll
    for (int t = 0; t < D / 32; ++t) x[t] = *reinterpret_cast<const uint4*>(row + 32 * t + 8 * lg);
}
// (ok = false adds nothing, whatever bits x holds.)
template <int D>
__device__ __forceinline__ void fma_lane_order(const uint4* x, float wgt, bool ok, f32x4* acc) {
#pragma unroll
    for (int t = 0; t < D / 32; ++t) {
        const uint32_t v[4] = {ok ? x[t].x : 0u, ok ? x[t].y : 0u, ok ? x[t].z : 0u, ok ? x[t].w : 0u};
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int db = 2 * t + h;
            acc[db][0] += wgt * __uint_as_float(v[2 * h] << 16);
            acc[db][1] += wgt * __uint_as_float(v[2 * h] & 0xffff0000u);
            acc[db][2] += wgt * __uint_as_float(v[2 * h + 1] << 16);
            acc[db][3] += wgt * __uint_as_float(v[2 * h + 1] & 0xffff0000u);
        }
    }
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
