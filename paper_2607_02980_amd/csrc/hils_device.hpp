// Device-side helpers for the HiLS kernels (gfx950, 64-lane wavefronts).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hils {

constexpr int kWave = 64;
constexpr int kChunk = 64;  // S: the only chunk size with kernels

// Index of the calling wave in its workgroup, as a wave-uniform (scalar) value.
// Conditions built from it compile to scalar branches; this matters for MFMA,
// which does not honour the EXEC mask, so an MFMA under a lane-masked branch
// that the compiler cannot prove uniform still runs when every lane is off.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x / kWave); }

// ---- storage types -------------------------------------------------------

struct bf16 {
    uint16_t bits;
};

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return __uint_as_float((uint32_t)x.bits << 16); }

template <typename T>
__device__ __forceinline__ T from_f32(float x);
template <>
__device__ __forceinline__ float from_f32<float>(float x) { return x; }
// Round to nearest, ties to even, with the hardware conversion (v_cvt_pk_bf16_f32
// on gfx950; it agrees bit for bit with the integer rounding x + 0x7fff + lsb on
// finite inputs, denormals included, and keeps NaN a NaN).
template <>
__device__ __forceinline__ bf16 from_f32<bf16>(float x) {
    bf16 r;
    r.bits = __builtin_bit_cast(uint16_t, static_cast<__bf16>(x));
    return r;
}

// Two floats to a packed bf16 pair (lo in the low half).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2_t;
    bf16x2_t v;
    v[0] = static_cast<__bf16>(lo);
    v[1] = static_cast<__bf16>(hi);
    return __builtin_bit_cast(uint32_t, v);
}

// Load 8 consecutive elements (16 B for bf16, 32 B for f32) as floats.
__device__ __forceinline__ void load8(const bf16* p, float* o) {
    const uint4 w = *reinterpret_cast<const uint4*>(p);
    const uint32_t a[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        o[2 * t] = __uint_as_float(a[t] << 16);
        o[2 * t + 1] = __uint_as_float(a[t] & 0xffff0000u);
    }
}
__device__ __forceinline__ void load8(const float* p, float* o) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
    o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
}

// ---- wave reductions (all 64 lanes receive the result) --------------------

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, kWave);
    return x;
}
__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) x = fmaxf(x, __shfl_xor(x, m, kWave));
    return x;
}

// ---- DPP reductions inside groups of 8 / 16 / 32 lanes (no LDS round trip) --
template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}
// Sum over each aligned group of N lanes (N = 1, 2, 4, 8, 16, 32, 64); every
// lane of the group receives the group's sum.
template <int N>
__device__ __forceinline__ float group_sum(float x) {
    if constexpr (N >= 2) x += dpp<0xB1>(x);    // quad_perm [1,0,3,2]: lane ^ 1
    if constexpr (N >= 4) x += dpp<0x4E>(x);    // quad_perm [2,3,0,1]: lane ^ 2
    if constexpr (N >= 8) x += dpp<0x141>(x);   // row_half_mirror: the other quad of the 8
    if constexpr (N >= 16) x += dpp<0x140>(x);  // row_mirror: the other half of the 16-lane row
    if constexpr (N >= 32) x += __shfl_xor(x, 16, kWave);
    if constexpr (N >= 64) x += __shfl_xor(x, 32, kWave);
    return x;
}

// exp(x) for x <= 0 typically; exact -inf -> 0.
// Sum / max over the four lanes l % 16 + {0, 16, 32, 48} (the lane groups of an
// MFMA accumulator column), with the gfx950 lane swaps v_permlane16_swap and
// v_permlane32_swap (VALU, no LDS round trip).  permlane16_swap(x, x) leaves each
// lane with {x, x of lane l ^ 16} in its two results, permlane32_swap likewise for
// l ^ 32 (checked on the hardware); every lane ends with the same bits.
__device__ __forceinline__ float group4_sum(float x) {
    const uint32_t u = __float_as_uint(x);
    const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const uint32_t v = __float_as_uint(y);
    const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}
__device__ __forceinline__ float group4_max(float x) {
    const uint32_t u = __float_as_uint(x);
    const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const uint32_t v = __float_as_uint(y);
    const auto b = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// Every lane gets the value of lane l % 16 (lane group 0), with the same swaps.
__device__ __forceinline__ float group0_bcast(float x) {
    const uint32_t u = __float_as_uint(x);
    const uint32_t y = __builtin_amdgcn_permlane16_swap(u, u, false, false)[0];   // rows {0, 0, 2, 2}
    return __uint_as_float(__builtin_amdgcn_permlane32_swap(y, y, false, false)[0]);  // rows {0, 0, 0, 0}
}

__device__ __forceinline__ float fexp(float x) { return __expf(x); }
// 2^x with the hardware instruction (v_exp_f32); exp(x) = fexp2(x * kLog2e).
constexpr float kLog2e = 1.4426950408889634f;
__device__ __forceinline__ float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Order-preserving map float -> uint32 (larger float => larger key; -0 < +0).
__device__ __forceinline__ uint32_t ordered_key(float f) {
    uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ int popc64(uint64_t m) { return __popcll(m); }

// ---- chunk geometry (Sec. 2.1) ------------------------------------------

// |C_i| = l(i)/S for a query at position i, with l(i) clamped at 0.
__device__ __forceinline__ int n_candidates(int i, int W) {
    int t = i - W + 1;
    if (t < 0) return 0;
    return t / kChunk;
}

// ---- wave top-K selection ------------------------------------------------
//
// One wavefront selects the K best of n candidates (score sc[e], chunk id[e]),
// ordered by score descending and then id ascending (ties to the smaller
// chunk, Eq. (9) rank with that reading of ties).  sc/id live in LDS.  The
// chosen ids are written ascending to out_id[0..m) with their scores to
// out_sc, m = min(K, n) is returned (to every lane).
//
// Method: exact radix select.  T = the m-th largest 32-bit order key is built
// bit by bit with ballot counts; everything above T is kept, and among the
// entries equal to T the `need` smallest ids are kept (a second bitwise
// search, only when T is tied).  No sorting network and no data movement
// besides the final compaction.
__device__ __forceinline__ int wave_count_ge(const float* sc, int n, uint32_t t) {
    const int lane = __lane_id();
    int c = 0;
    for (int base = 0; base < n; base += kWave) {
        const int e = base + lane;
        const bool pr = e < n && ordered_key(sc[e]) >= t;
        c += popc64(__ballot(pr));
    }
    return c;
}

__device__ inline int wave_topk(const float* sc, const int* id, int n, int K, int* out_id, float* out_sc,
                                int* tmp_id, float* tmp_sc) {
    const int lane = __lane_id();
    const int m = n < K ? n : K;
    if (m <= 0) return 0;
    uint32_t T = 0;
    bool all = (n <= K);
    int cnt_gt = 0, need = 0;
    uint32_t id_thr = 0x7fffffffu;
    if (!all) {
        for (int bit = 31; bit >= 0; --bit) {
            const uint32_t t = T | (1u << bit);
            if (wave_count_ge(sc, n, t) >= m) T = t;
        }
        cnt_gt = (T == 0xffffffffu) ? 0 : wave_count_ge(sc, n, T + 1);
        need = m - cnt_gt;
        int ties = wave_count_ge(sc, n, T) - cnt_gt;
        if (ties > need) {
            // need-th smallest id among the entries with key == T
            uint32_t x = 0;
            for (int bit = 30; bit >= 0; --bit) {
                const uint32_t y = x | (1u << bit);
                int c = 0;
                for (int base = 0; base < n; base += kWave) {
                    const int e = base + lane;
                    const bool pr = e < n && ordered_key(sc[e]) == T && (uint32_t)id[e] < y;
                    c += popc64(__ballot(pr));
                }
                if (c < need) x = y;
            }
            id_thr = x;  // keep ties with id <= x
        }
    }
    // compact the chosen entries (any order) into tmp
    int w = 0;
    for (int base = 0; base < n; base += kWave) {
        const int e = base + lane;
        bool pr = false;
        if (e < n) {
            if (all) {
                pr = true;
            } else {
                const uint32_t k = ordered_key(sc[e]);
                pr = k > T || (k == T && (uint32_t)id[e] <= id_thr);
            }
        }
        const uint64_t bal = __ballot(pr);
        if (pr) {
            const int pos = w + popc64(bal & ((1ull << lane) - 1ull));
            tmp_id[pos] = id[e];
            tmp_sc[pos] = sc[e];
        }
        w += popc64(bal);
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    // rank by id (m <= 64: one entry per lane)
    if (lane < m) {
        const int my = tmp_id[lane];
        int r = 0;
        for (int t = 0; t < m; ++t) r += tmp_id[t] < my;
        out_id[r] = my;
        out_sc[r] = tmp_sc[lane];
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    return m;
}

// Register-resident variant: lane l holds candidates e = l + 64*r (r < E) with
// score sc[r], chunk id[r] and a valid flag; every pass of the radix select
// is compares and ballots on registers only.  Same order and outputs as
// wave_topk.
// FIRST: the order of the ids.  kTopkUnordered: any order (the survivors are
// ranked through LDS).  Otherwise the ids ascend over (register, lane) when
// register FIRST (if >= 0) is taken first and then registers 0, 1, ... in turn;
// the compaction position is then the ascending rank and out_* are written
// directly.
constexpr int kTopkUnordered = -2, kTopkNatural = -1;

// m-th largest value of one NB-bit key per lane (0 if fewer than m lanes hold
// a key >= 1): the bits of the threshold from the top, one ballot each.
template <int NB = 32>
__device__ __forceinline__ uint32_t wave_kth_key(uint32_t x, int m) {
    uint32_t T = 0;
    for (int bit = NB - 1; bit >= 0; --bit) {
        const uint32_t t = T | (1u << bit);
        if (popc64(__ballot(x >= t)) >= m) T = t;
    }
    return T;
}

template <int E, int FIRST = kTopkUnordered>
__device__ inline int wave_topk_reg(const float (&sc)[E], const int (&id)[E], const bool (&valid)[E], int K,
                                    int* out_id, float* out_sc, int* tmp_id, float* tmp_sc) {
    const int lane = __lane_id();
    // validity is folded into the key: invalid -> 0, valid -> >= 1 (only the
    // all-ones NaN pattern maps to 0 and is lifted to 1), so every threshold
    // t >= 1 below excludes invalid entries with a single compare
    uint32_t key[E];
    int n = 0;
#pragma unroll
    for (int r = 0; r < E; ++r) {
        const uint32_t k = ordered_key(sc[r]);
        key[r] = valid[r] ? (k ? k : 1u) : 0u;
        n += popc64(__ballot(valid[r]));
    }
    const int m = n < K ? n : K;
    if (m <= 0) return 0;
    auto count_ge = [&](uint32_t t) {
        int c = 0;
#pragma unroll
        for (int r = 0; r < E; ++r) c += popc64(__ballot(key[r] >= t));
        return c;
    };
    uint32_t T = 0, id_thr = 0x7fffffffu;
    const bool all = (n <= K);
    constexpr bool kOrdered = FIRST != kTopkUnordered;
    if (!all && E > 1) {
        // Fast path.  The m-th largest of the lane maxima is a lower bound of the
        // m-th largest key (m lanes hold a key at least as large), and so is T0,
        // that bound with its low 16 bits cleared (found in 16 ballot steps), so
        // the m best entries are among the survivors key >= T0.  When they fit one
        // per lane they are compacted in visiting order and selected with
        // one-register passes.
        uint32_t lmax = 0;
#pragma unroll
        for (int r = 0; r < E; ++r) lmax = key[r] > lmax ? key[r] : lmax;
        uint32_t T0 = wave_kth_key<16>(lmax >> 16, m) << 16;
        T0 = T0 ? T0 : 1u;
        const int c = count_ge(T0);
        if (c <= kWave) {
            int w = 0;
#pragma unroll
            for (int q = 0; q < E; ++q) {
                const int r = FIRST >= 0 ? (q == 0 ? FIRST : (q - 1 < FIRST ? q - 1 : q)) : q;
                const bool pr = key[r] >= T0;
                const uint64_t bal = __ballot(pr);
                if (pr) {
                    const int pos = w + popc64(bal & ((1ull << lane) - 1ull));
                    tmp_id[pos] = id[r];
                    tmp_sc[pos] = sc[r];
                }
                w += popc64(bal);
            }
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
            const bool have = lane < c;
            const int i1 = have ? tmp_id[lane] : 0;
            const float s1 = have ? tmp_sc[lane] : 0.f;
            uint32_t k1 = 0;
            if (have) {
                const uint32_t k = ordered_key(s1);
                k1 = k ? k : 1u;
            }
            const uint32_t T1 = wave_kth_key(k1, m);  // >= T0 >= 1
            const int cnt_gt = (T1 == 0xffffffffu) ? 0 : popc64(__ballot(k1 > T1));
            const int need = m - cnt_gt;
            const int ties = popc64(__ballot(k1 == T1));
            uint32_t thr = 0x7fffffffu;
            if (ties > need) {
                uint32_t x = 0;
                for (int bit = 30; bit >= 0; --bit) {
                    const uint32_t y = x | (1u << bit);
                    if (popc64(__ballot(k1 == T1 && (uint32_t)i1 < y)) < need) x = y;
                }
                thr = x;
            }
            const bool pr = k1 > T1 || (k1 == T1 && (uint32_t)i1 <= thr);
            const uint64_t bal = __ballot(pr);
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
            const int pos = popc64(bal & ((1ull << lane) - 1ull));
            if (kOrdered) {
                // survivors ascend by id over the lanes: the compaction is the order
                if (pr) {
                    out_id[pos] = i1;
                    out_sc[pos] = s1;
                }
            } else {
                if (pr) {
                    tmp_id[pos] = i1;
                    tmp_sc[pos] = s1;
                }
                __builtin_amdgcn_wave_barrier();
                __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
                if (lane < m) {
                    const int my = tmp_id[lane];
                    int rk = 0;
                    for (int t = 0; t < m; ++t) rk += tmp_id[t] < my;
                    out_id[rk] = my;
                    out_sc[rk] = tmp_sc[lane];
                }
            }
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
            return m;
        }
    }
    if (!all) {
        for (int bit = 31; bit >= 0; --bit) {
            const uint32_t t = T | (1u << bit);
            if (count_ge(t) >= m) T = t;
        }
        // T >= 1 here: m valid entries have keys >= 1
        const int cnt_gt = (T == 0xffffffffu) ? 0 : count_ge(T + 1);
        const int need = m - cnt_gt;
        const int ties = count_ge(T) - cnt_gt;
        if (ties > need) {
            uint32_t x = 0;
            for (int bit = 30; bit >= 0; --bit) {
                const uint32_t y = x | (1u << bit);
                int c = 0;
#pragma unroll
                for (int r = 0; r < E; ++r) c += popc64(__ballot(key[r] == T && (uint32_t)id[r] < y));
                if (c < need) x = y;
            }
            id_thr = x;
        }
    }
    int* dst_id = kOrdered ? out_id : tmp_id;
    float* dst_sc = kOrdered ? out_sc : tmp_sc;
    int w = 0;
#pragma unroll
    for (int q = 0; q < E; ++q) {
        // visiting order: FIRST, then the others ascending
        const int r = FIRST >= 0 ? (q == 0 ? FIRST : (q - 1 < FIRST ? q - 1 : q)) : q;
        const bool pr = key[r] != 0u && (all || key[r] > T || (key[r] == T && (uint32_t)id[r] <= id_thr));
        const uint64_t bal = __ballot(pr);
        if (pr) {
            const int pos = w + popc64(bal & ((1ull << lane) - 1ull));
            dst_id[pos] = id[r];
            dst_sc[pos] = sc[r];
        }
        w += popc64(bal);
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    if (kOrdered) return m;
    if (lane < m) {
        const int my = tmp_id[lane];
        int rk = 0;
        for (int t = 0; t < m; ++t) rk += tmp_id[t] < my;
        out_id[rk] = my;
        out_sc[rk] = tmp_sc[lane];
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    return m;
}

}  // namespace hils
