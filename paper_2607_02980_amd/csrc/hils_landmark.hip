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

template <bool BWD>
struct LmkRun {
    template <typename T, int D, int G>
    static hipError_t run(const LmkArgs& a, hipStream_t s) {
        const dim3 grid(a.L / kChunk, a.Hkv, a.B);
        if (BWD) {
            HILS_LAUNCH("k_lmk_bwd", (k_lmk_bwd<T, D>), grid, dim3(kBlock), 0, s, a);
            if (a.shared) HILS_LAUNCH("k_lmk_dq_sum", (k_lmk_dq_sum<T, D>), dim3(a.Hl), dim3(kBlock), 0, s, a);
        } else
            HILS_LAUNCH("k_lmk_fwd", (k_lmk_fwd<T, D>), grid, dim3(kBlock), 0, s, a);
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
