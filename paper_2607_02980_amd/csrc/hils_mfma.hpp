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

// Swizzled LDS tiles ("st"), rows of W = 64 or 128 bf16.  On gfx950 the LDS
// serves 16-byte reads to four groups of 16 lanes (lanes 0-31 or 32-63, split by
// the parity of lane bits 2-4) and 8-byte (also transposing) reads to lanes 0-31
// and 32-63, each group over 64 banks of 4 bytes; 16-byte stores go 8 lanes at a
// time and 8-byte stores 16 lanes at a time, over 32 banks (measured with the
// bank-conflict counters).  The layouts below put the row-wise 16-byte operand
// reads (16 rows of one column piece), the transposing reads (4 rows x 32 bytes
// per 16 lanes, rows r and r + 4 or r + 16), the 16-byte stores of a row piece per
// lane and of whole rows on distinct banks:
//   W = 128: rows padded to 144, rows 8..15 of every 16 shifted by 64 more, 64
//     elements between groups of 16 rows, and the two 16-byte pieces of each
//     32-byte pair swapped in rows with r % 8 >= 4.  The swap only touches the
//     lowest bit of the piece index, so column offsets that are multiples of 16
//     stay linear and fold into the instructions' offsets.
//   W = 64: unpadded, the 16-byte pieces of row r permuted by XOR with
//     (r & 7) ^ 5 (r >> 3 & 1) (its 8-byte stores of one column still meet two
//     rows per bank).
template <int W>
__device__ __forceinline__ int st_off(int r, int c) {
    static_assert(W == 64 || W == 128, "swizzled tiles are 64 or 128 wide");
    if constexpr (W == 128)
        return (r >> 4) * (16 * (W + 16) + 64) + (r & 15) * (W + 16) + 64 * ((r >> 3) & 1) +
               8 * ((c >> 3) ^ ((r >> 2) & 1)) + (c & 7);
    else
        return r * W + 8 * ((c >> 3) ^ (r & 7) ^ (((r >> 3) & 1) * 5)) + (c & 7);
}
template <int W>
constexpr int st_size(int rows) {
    return W == 128 ? (rows + 15) / 16 * (16 * (W + 16) + 64) : rows * W;
}
// Elements per 16 rows of a swizzled tile: row r + 16 m is row r moved by m groups.
template <int W>
constexpr int st_group() {
    return W == 128 ? 16 * (W + 16) + 64 : 16 * W;
}
// Offset of (r, c0 + c) for a column offset c0 that the layout keeps linear (a
// multiple of 16 for W = 128; none for W = 64, whose XOR reaches bit 2 of the piece
// index): the lane-dependent part and the constant part apart, so that the latter
// folds into the instructions' offsets.
template <int W>
__device__ __forceinline__ int st_off_lin(int r, int c0, int c) {
    if constexpr (W == 128)
        return st_off<W>(r, c) + c0;
    else
        return st_off<W>(r, c0 + c);
}
// row_operand / tr_operand of a swizzled tile (r0 and k0 multiples of 16)
template <int W>
__device__ __forceinline__ bf16x8 row_operand_st(const bf16* X, int r0, int k0, int lane) {
    return ld_bf16x8(X + (r0 / 16) * st_group<W>() + st_off_lin<W>(lane % 16, k0, (lane / 16) * 8));
}
template <int W>
__device__ __forceinline__ bf16x8 tr_operand_st(const bf16* X, int k0, int n0, int lane) {
    const int g = lane / 16, s = lane % 16;
    const int r = g * 8 + s / 4, c = 4 * (s % 4);
    const bf16* base = X + (k0 / 16) * st_group<W>();
    const v4i16 a = lds_read_tr16(base + st_off_lin<W>(r, n0, c));
    const v4i16 b = lds_read_tr16(base + st_off_lin<W>(r + 4, n0, c));
    typedef short v8i16 __attribute__((ext_vector_type(8)));
    const v8i16 v = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    return __builtin_bit_cast(bf16x8, v);
}
// tr_operand_perm of a swizzled tile (k0 and n0 multiples of 16)
template <int W>
__device__ __forceinline__ bf16x8 tr_operand_perm_st(const bf16* X, int k0, int n0, int lane) {
    const int g = lane / 16, s = lane % 16;
    const int r = g * 4 + s / 4, c = 4 * (s % 4);
    const bf16* base = X + (k0 / 16) * st_group<W>();
    const v4i16 a = lds_read_tr16(base + st_off_lin<W>(r, n0, c));
    const v4i16 b = lds_read_tr16(base + st_group<W>() + st_off_lin<W>(r, n0, c));
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
