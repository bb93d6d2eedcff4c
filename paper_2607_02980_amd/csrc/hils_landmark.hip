// Landmark compression of Prop. 3.1 (forward and backward), gfx950.
//
// For landmark head hl of KV group g and chunk c with keys k_j (the chunk's S
// rows of the group's K) and landmark query q'_c:
//   s_j = scale * q'_c . k_j,  p = softmax(s),
//   k'_c = sum_j p_j k_j  (attention of q'_c over its chunk),
//   b'_c = -sum_j p_j log p_j = LSE(s) - sum_j p_j s_j  (entropy).
// Backward, for upstream dk'_c and db'_c:
//   dL/dp_j = dk'_c . k_j - db'_c (log p_j + 1),
//   ds_j    = p_j (dL/dp_j - sum_m p_m dL/dp_m),
//   dq'_c   = scale sum_j ds_j k_j,
//   dk_j    = sum over the group's landmark heads of p_j dk'_c + scale ds_j q'_c.
//
// One 256-thread block per (chunk, KV group, batch): the chunk's 64 keys are
// read once into LDS and serve every landmark head of the group (one per query
// head when Hl == Hq, one when Hl == Hkv), one wave per head.  The work is a
// single pass over K (16 KiB per chunk in bf16), so the kernels are organised
// around that read; the arithmetic is a few dot products per key.
//
// Shared-query variant (the landmark-token-free alternative of Sec. 4.1): one
// query per landmark head serves every chunk, lq is [Hl, D], and its gradient
// is the sum of the per-chunk gradients: k_lmk_bwd leaves them in fp32 in the
// workspace and k_lmk_dq_sum adds them up in a fixed order.
#include "hils_device.hpp"
#include "hils_dispatch.hpp"
#include "hils_internal.hpp"
#include "hils_mfma.hpp"

namespace hils {

namespace {

constexpr int kBlock = 256;
constexpr int kMaxLmkHeads = 8;  // landmark heads per KV group (Hl / Hkv <= G <= 8)

template <typename T, int D>
struct LmkSmem {
    float k[kChunk][D + 1];       // the chunk's keys
    float q[kMaxLmkHeads][D];     // landmark queries q'_c of the group's heads
    float dk[kMaxLmkHeads][D];    // upstream dk'_c (backward)
    float p[kMaxLmkHeads][kChunk];
    float ds[kMaxLmkHeads][kChunk];
    float db[kMaxLmkHeads];
};

// Stage the chunk's keys and, per landmark head of the group, one D-vector
// from each of up to two [B, Hl, L/S, D] tensors (x0 is [Hl, D] when
// x0_shared: the shared landmark query).
template <typename T, int D>
__device__ __forceinline__ void stage(const LmkArgs& a, LmkSmem<T, D>& sm, int b, int g, int c, int nlh,
                                      const void* x0, bool x0_shared, float (*s0)[D], const void* x1,
                                      float (*s1)[D]) {
    const int tid = threadIdx.x;
    const int nC = a.L / kChunk;
    const T* kb = as<T>(a.k) + (((size_t)b * a.Hkv + g) * a.L + (size_t)c * kChunk) * D;
    for (int e = tid; e < kChunk * D / 8; e += kBlock) {
        const int j = e / (D / 8), dd = (e % (D / 8)) * 8;
        float x[8];
        load8(kb + (size_t)j * D + dd, x);
#pragma unroll
        for (int t = 0; t < 8; ++t) sm.k[j][dd + t] = x[t];
    }
    for (int e = tid; e < nlh * D; e += kBlock) {
        const int hh = e / D, dd = e % D;
        const size_t row = ((size_t)b * a.Hl + g * nlh + hh) * nC + c;
        const size_t row0 = x0_shared ? (size_t)(g * nlh + hh) : row;
        if (x0) s0[hh][dd] = to_f32(as<T>(x0)[row0 * D + dd]);
        if (x1) s1[hh][dd] = to_f32(as<T>(x1)[row * D + dd]);
    }
}

// Lane j: s_j = scale * q . k_j for the head's query row in LDS.
template <int D>
__device__ __forceinline__ float key_dot(const float (*k)[D + 1], const float* q, int j) {
    float acc = 0.f;
#pragma unroll 8
    for (int dd = 0; dd < D; ++dd) acc += q[dd] * k[j][dd];
    return acc;
}

template <typename T, int D>
__global__ __launch_bounds__(kBlock) void k_lmk_fwd(LmkArgs a) {
    __shared__ LmkSmem<T, D> sm;
    __shared__ float s_bias[kMaxLmkHeads];
    const int c = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x, wave = wave_id(), lane = tid % kWave;
    const int nlh = a.Hl / a.Hkv, nC = a.L / kChunk;
    stage<T, D>(a, sm, b, g, c, nlh, a.lq, a.shared, sm.q, nullptr, nullptr);
    __syncthreads();
    for (int hh = wave; hh < nlh; hh += kBlock / kWave) {
        const float s = a.scale * key_dot<D>(sm.k, sm.q[hh], lane);  // lane = key (S = 64)
        const float m = wave_max(s);
        const float e = fexp(s - m);
        const float z = wave_sum(e);
        const float lse = m + __logf(z);
        const float p = e / z;
        sm.p[hh][lane] = p;
        const float ps = wave_sum(p * s);
        if (lane == 0) s_bias[hh] = lse - ps;  // -sum p log p with log p = s - lse
    }
    __syncthreads();
    for (int o = tid; o < nlh * D; o += kBlock) {
        const int hh = o / D, dd = o % D;
        float acc = 0.f;
#pragma unroll 16
        for (int j = 0; j < kChunk; ++j) acc += sm.p[hh][j] * sm.k[j][dd];
        const size_t row = ((size_t)b * a.Hl + g * nlh + hh) * nC + c;
        as_mut<T>(a.lmk)[row * D + dd] = from_f32<T>(acc);
        if (dd == 0) a.bias[row] = s_bias[hh];
    }
}

template <typename T, int D>
__global__ __launch_bounds__(kBlock) void k_lmk_bwd(LmkArgs a) {
    __shared__ LmkSmem<T, D> sm;
    const int c = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x, wave = wave_id(), lane = tid % kWave;
    const int nlh = a.Hl / a.Hkv, nC = a.L / kChunk;
    stage<T, D>(a, sm, b, g, c, nlh, a.lq, a.shared, sm.q, a.dlmk, sm.dk);
    if (tid < nlh) sm.db[tid] = a.dbias ? a.dbias[((size_t)b * a.Hl + g * nlh + tid) * nC + c] : 0.f;
    __syncthreads();
    for (int hh = wave; hh < nlh; hh += kBlock / kWave) {
        const float s = a.scale * key_dot<D>(sm.k, sm.q[hh], lane);
        const float m = wave_max(s);
        const float e = fexp(s - m);
        const float z = wave_sum(e);
        const float logp = s - (m + __logf(z));
        const float p = e / z;
        const float gp = key_dot<D>(sm.k, sm.dk[hh], lane) - sm.db[hh] * (logp + 1.f);
        const float mean = wave_sum(p * gp);
        sm.p[hh][lane] = p;
        sm.ds[hh][lane] = p * (gp - mean);
    }
    __syncthreads();
    // dq'_c per head (the shared query: the chunk's term, in fp32)
    for (int o = tid; o < nlh * D; o += kBlock) {
        const int hh = o / D, dd = o % D;
        float acc = 0.f;
#pragma unroll 16
        for (int j = 0; j < kChunk; ++j) acc += sm.ds[hh][j] * sm.k[j][dd];
        const size_t row = ((size_t)b * a.Hl + g * nlh + hh) * nC + c;
        if (a.shared)
            a.ws[row * D + dd] = a.scale * acc;
        else
            as_mut<T>(a.dlq)[row * D + dd] = from_f32<T>(a.scale * acc);
    }
    // dk of the chunk's keys, summed over the group's landmark heads
    T* dkb = as_mut<T>(a.dk) + (((size_t)b * a.Hkv + g) * a.L + (size_t)c * kChunk) * D;
    for (int o = tid; o < kChunk * D; o += kBlock) {
        const int j = o / D, dd = o % D;
        float acc = 0.f;
        for (int hh = 0; hh < nlh; ++hh) acc += sm.p[hh][j] * sm.dk[hh][dd] + a.scale * sm.ds[hh][j] * sm.q[hh][dd];
        dkb[(size_t)j * D + dd] = from_f32<T>(acc);
    }
}

// Shared query: dlq[hl] = sum over b, then c, of the chunk terms.  One block per
// landmark head; thread t adds rows t / D, t / D + 256 / D, ... of column t % D,
// then the 256 / D partial sums are added in thread order.
template <typename T, int D>
__global__ __launch_bounds__(kBlock) void k_lmk_dq_sum(LmkArgs a) {
    constexpr int R = kBlock / D;
    __shared__ float part[R][D];
    const int hl = blockIdx.x, tid = threadIdx.x, dd = tid % D, r0 = tid / D;
    const int nC = a.L / kChunk;
    float acc = 0.f;
    for (int b = 0; b < a.B; ++b) {
        const float* src = a.ws + ((size_t)b * a.Hl + hl) * nC * D;
        for (int c = r0; c < nC; c += R) acc += src[(size_t)c * D + dd];
    }
    part[r0][dd] = acc;
    __syncthreads();
    if (tid < D) {
        float t = 0.f;
#pragma unroll
        for (int r = 0; r < R; ++r) t += part[r][tid];
        as_mut<T>(a.dlq)[(size_t)hl * D + tid] = from_f32<T>(t);
    }
}

// ---- bf16 storage: one wavefront per (chunk, KV group, batch), on MFMA --------
// The group's landmark heads are the MFMA columns (lane l: head l % 16, nlh <= 8
// valid).  S^T = K Q'^T from K rows and q' read straight from HBM; the softmax,
// log-sum-exp and entropy per head across the four lane groups (permlane swaps);
// k' = K^T P^T with K^T from the wave's LDS copy of K (transposing reads) and P
// split into a bf16 head and residual, so that the product keeps P to ~fp32.
// Backward: dK'-scores GP^T = K dK'^T the same way, ds, dq' = scale K^T DS^T, and
// dK = [P | scale DS] [dK' ; q'] as one (keys x 32) by (32 x dims) product per
// tile, its A operand transposed through LDS.

template <int D>
struct LmkWaveSmem {
    bf16 k[kChunk * (D + 16)];  // the chunk's keys, row-major (K^T operands)
};
template <int D>
struct LmkWaveSmemB {
    bf16 k[kChunk * (D + 16)];
    bf16 t[kChunk * 40];        // [key][p hi | p lo | scale ds hi | scale ds lo] x 8 heads (+8 pad)
    bf16 r[32 * (D + 16)];      // [dk' ; dk' ; q' ; q'] x 8 heads, row-major (B operands of dK)
};

// operand pair of P^T in the permuted key order of two S^T blocks, split hi / lo
__device__ __forceinline__ void split_perm(const f32x4& e0, const f32x4& e1, bf16x8& hi, bf16x8& lo) {
    float x[8] = {e0[0], e0[1], e0[2], e0[3], e1[0], e1[1], e1[2], e1[3]};
    float y[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) y[t] = x[t] - to_f32(from_f32<bf16>(x[t]));
    hi = pack_bf16x8(x);
    lo = pack_bf16x8(y);
}

// Shared front of both passes: S^T, p, log-sum-exp, with K staged into `sk`.
// Returns per lane st[kb][i] = p of key 16 kb + 4 lg + i for head n16 (0 for
// heads >= nlh), and the head's lse (natural units) and sum p s.
template <int D>
__device__ __forceinline__ void lmk_softmax(const LmkArgs& a, const bf16* kg, const bf16* qrow, bool hv, bf16* sk,
                                            f32x4 (&st)[4], float& lse, float& ps) {
    constexpr int KS = D / 32, VROW = D + 16;
    const int lane = threadIdx.x % kWave, lg = lane / 16, n16 = lane % 16;
    bf16x8 kA[4][KS], qB[KS];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) kA[kb][ks] = ld_bf16x8(kg + (size_t)(kb * 16 + n16) * D + ks * 32 + lg * 8);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 qq = ld_bf16x8(qrow + ks * 32 + lg * 8);
        qB[ks] = hv ? qq : as_bf16x8(make_uint4(0, 0, 0, 0));
    }
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            *reinterpret_cast<bf16x8*>(sk + (kb * 16 + n16) * VROW + ks * 32 + lg * 8) = kA[kb][ks];
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
        st[kb] = zero4();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) st[kb] = mfma16x16x32(kA[kb][ks], qB[ks], st[kb]);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            st[kb][i] *= a.scale;  // s_j
            mx = fmaxf(mx, st[kb][i]);
        }
    }
    mx = group4_max(mx);
    float sum = 0.f, sw = 0.f;
    f32x4 e[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            e[kb][i] = fexp(st[kb][i] - mx);
            sum += e[kb][i];
            sw += e[kb][i] * st[kb][i];
        }
    sum = group4_sum(sum);
    sw = group4_sum(sw);
    const float inv = 1.f / sum;
    lse = mx + __logf(sum);
    ps = sw * inv;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) st[kb][i] = hv ? e[kb][i] * inv : 0.f;
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
}

// O^T[dim][head] = K^T X^T for X = st (probabilities or ds), hi/lo split.
template <int D>
__device__ __forceinline__ void lmk_kt_times(const bf16* sk, const f32x4 (&x)[4], f32x4 (&o)[D / 16]) {
    constexpr int DB = D / 16, VROW = D + 16;
    const int lane = threadIdx.x % kWave;
    bf16x8 h0, l0, h1, l1;
    split_perm(x[0], x[1], h0, l0);
    split_perm(x[2], x[3], h1, l1);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
        const bf16x8 a0 = tr_operand_perm(sk, VROW, 0, db * 16, lane);
        const bf16x8 a1 = tr_operand_perm(sk, VROW, 32, db * 16, lane);
        f32x4 acc = mfma16x16x32(a0, h0, zero4());
        acc = mfma16x16x32(a0, l0, acc);
        acc = mfma16x16x32(a1, h1, acc);
        o[db] = mfma16x16x32(a1, l1, acc);
    }
}

template <int D>
__global__ __launch_bounds__(kWave) void k_lmk_fwd_m(LmkArgs a) {
    constexpr int DB = D / 16;
    __shared__ __align__(16) LmkWaveSmem<D> sm;
    const int c = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
    const int lane = threadIdx.x, lg = lane / 16, n16 = lane % 16;
    const int nlh = a.Hl / a.Hkv, nC = a.L / kChunk;
    const bool hv = n16 < nlh;
    const int hl = g * nlh + min(n16, nlh - 1);
    const size_t row = ((size_t)b * a.Hl + hl) * nC + c;
    const bf16* kg = as<bf16>(a.k) + (((size_t)b * a.Hkv + g) * a.L + (size_t)c * kChunk) * D;
    const bf16* qrow = as<bf16>(a.lq) + (a.shared ? (size_t)hl : row) * D;
    f32x4 st[4];
    float lse, ps;
    lmk_softmax<D>(a, kg, qrow, hv, sm.k, st, lse, ps);
    f32x4 o[DB];
    lmk_kt_times<D>(sm.k, st, o);
    if (hv) {
        bf16* out = as_mut<bf16>(a.lmk) + row * D;
#pragma unroll
        for (int db = 0; db < DB; ++db)
            *reinterpret_cast<uint2*>(out + db * 16 + lg * 4) =
                make_uint2(pack_bf16x2(o[db][0], o[db][1]), pack_bf16x2(o[db][2], o[db][3]));
        if (lg == 0) a.bias[row] = lse - ps;  // -sum p log p with log p = s - lse
    }
}

template <int D>
__global__ __launch_bounds__(kWave) void k_lmk_bwd_m(LmkArgs a) {
    constexpr int KS = D / 32, DB = D / 16, VROW = D + 16, TROW = 40;
    __shared__ __align__(16) LmkWaveSmemB<D> sm;
    const int c = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
    const int lane = threadIdx.x, lg = lane / 16, n16 = lane % 16;
    const int nlh = a.Hl / a.Hkv, nC = a.L / kChunk;
    const bool hv = n16 < nlh;
    const int hl = g * nlh + min(n16, nlh - 1);
    const size_t row = ((size_t)b * a.Hl + hl) * nC + c;
    const bf16* kg = as<bf16>(a.k) + (((size_t)b * a.Hkv + g) * a.L + (size_t)c * kChunk) * D;
    const bf16* qrow = as<bf16>(a.lq) + (a.shared ? (size_t)hl : row) * D;
    const bf16* dkrow = as<bf16>(a.dlmk) + row * D;
    // B rows of the dK product: dk' of head m in rows m and 8 + m, q' in 16 + m and
    // 24 + m (zero for m >= nlh)
    for (int e = lane; e < 32 * D / 8; e += kWave) {
        const int rr = e / (D / 8), d8 = (e % (D / 8)) * 8, m = rr % 8;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (m < nlh) {
            const size_t rm = ((size_t)b * a.Hl + g * nlh + m) * nC + c;
            v = rr < 16 ? *reinterpret_cast<const uint4*>(as<bf16>(a.dlmk) + rm * D + d8)
                        : *reinterpret_cast<const uint4*>(as<bf16>(a.lq) + (a.shared ? (size_t)(g * nlh + m) : rm) * D + d8);
        }
        *reinterpret_cast<uint4*>(sm.r + rr * VROW + d8) = v;
    }
    f32x4 p[4];
    float lse, ps;
    lmk_softmax<D>(a, kg, qrow, hv, sm.k, p, lse, ps);
    // GP^T = K dK'^T (K operands again from HBM through L2), then
    // gp_j = dk'.k_j - db' (log p_j + 1), ds_j = p_j (gp_j - sum_m p_m gp_m)
    bf16x8 dB[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 x = ld_bf16x8(dkrow + ks * 32 + lg * 8);
        dB[ks] = hv ? x : as_bf16x8(make_uint4(0, 0, 0, 0));
    }
    const float db = (a.dbias && hv) ? a.dbias[row] : 0.f;
    f32x4 ds[4];
    float mean = 0.f;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
        f32x4 gp = zero4();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            gp = mfma16x16x32(ld_bf16x8(sm.k + (kb * 16 + n16) * VROW + ks * 32 + lg * 8), dB[ks], gp);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            // log p_j = s_j - lse, and s_j = lse + log p_j is not kept: recompute from p
            const float logp = p[kb][i] > 0.f ? __logf(p[kb][i]) : 0.f;
            ds[kb][i] = gp[i] - db * (logp + 1.f);
            mean += p[kb][i] * ds[kb][i];
        }
    }
    mean = group4_sum(mean);
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) ds[kb][i] = p[kb][i] * (ds[kb][i] - mean);
    // dq' = scale K^T DS^T
    f32x4 o[DB];
    lmk_kt_times<D>(sm.k, ds, o);
    if (hv) {
        if (a.shared) {
            float* dst = a.ws + row * D;
#pragma unroll
            for (int d = 0; d < DB; ++d) *reinterpret_cast<f32x4*>(dst + d * 16 + lg * 4) = o[d] * a.scale;
        } else {
            bf16* dst = as_mut<bf16>(a.dlq) + row * D;
#pragma unroll
            for (int d = 0; d < DB; ++d)
                *reinterpret_cast<uint2*>(dst + d * 16 + lg * 4) = make_uint2(
                    pack_bf16x2(a.scale * o[d][0], a.scale * o[d][1]), pack_bf16x2(a.scale * o[d][2], a.scale * o[d][3]));
        }
    }
    // T[key][..]: p hi, p lo, scale ds hi, scale ds lo of head n16 (lanes n16 < 8)
    if (n16 < 8) {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int key = kb * 16 + lg * 4 + i;
                const float pv = hv ? p[kb][i] : 0.f, dv = hv ? a.scale * ds[kb][i] : 0.f;
                const bf16 ph = from_f32<bf16>(pv), dh = from_f32<bf16>(dv);
                sm.t[key * TROW + n16] = ph;
                sm.t[key * TROW + 8 + n16] = from_f32<bf16>(pv - to_f32(ph));
                sm.t[key * TROW + 16 + n16] = dh;
                sm.t[key * TROW + 24 + n16] = from_f32<bf16>(dv - to_f32(dh));
            }
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    // dK[key][dim] = sum_m p_m,key dk'_m + scale ds_m,key q'_m (lane: keys 4 lg + i, dim n16)
    bf16* dkb = as_mut<bf16>(a.dk) + (((size_t)b * a.Hkv + g) * a.L + (size_t)c * kChunk) * D;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
        const bf16x8 aT = ld_bf16x8(sm.t + (kb * 16 + n16) * TROW + lg * 8);
#pragma unroll
        for (int d = 0; d < DB; ++d) {
            const f32x4 acc = mfma16x16x32(aT, tr_operand(sm.r, VROW, 0, d * 16, lane), zero4());
#pragma unroll
            for (int i = 0; i < 4; ++i) dkb[(size_t)(kb * 16 + lg * 4 + i) * D + d * 16 + n16] = from_f32<bf16>(acc[i]);
        }
    }
}

template <bool BWD>
struct LmkRun {
    template <typename T, int D, int G>
    static hipError_t run(const LmkArgs& a, hipStream_t s) {
        const dim3 grid(a.L / kChunk, a.Hkv, a.B);
        constexpr bool kMfma = sizeof(T) == 2;
        if (BWD) {
            if constexpr (kMfma)
                HILS_LAUNCH("k_lmk_bwd", (k_lmk_bwd_m<D>), grid, dim3(kWave), 0, s, a);
            else
                HILS_LAUNCH("k_lmk_bwd", (k_lmk_bwd<T, D>), grid, dim3(kBlock), 0, s, a);
            if (a.shared) HILS_LAUNCH("k_lmk_dq_sum", (k_lmk_dq_sum<T, D>), dim3(a.Hl), dim3(kBlock), 0, s, a);
        } else {
            if constexpr (kMfma)
                HILS_LAUNCH("k_lmk_fwd", (k_lmk_fwd_m<D>), grid, dim3(kWave), 0, s, a);
            else
                HILS_LAUNCH("k_lmk_fwd", (k_lmk_fwd<T, D>), grid, dim3(kBlock), 0, s, a);
        }
        return hipGetLastError();
    }
};

}  // namespace

size_t landmark_workspace_bytes(int B, int Hl, int nC, int d, bool shared) {
    return shared ? (size_t)B * Hl * nC * d * sizeof(float) : 0;
}

// The kernels depend on (T, D) only; G = 1 picks one instantiation.
hipError_t launch_landmark_fwd(const LmkArgs& a, hipStream_t s) { return dispatch<LmkRun<false>>(a.bf16, a.d, 1, a, s); }
hipError_t launch_landmark_bwd(const LmkArgs& a, hipStream_t s) { return dispatch<LmkRun<true>>(a.bf16, a.d, 1, a, s); }

}  // namespace hils
