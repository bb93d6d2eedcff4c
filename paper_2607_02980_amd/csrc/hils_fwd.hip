// HiLS attention prefill forward, fp32 storage, gfx950 (the bf16 path runs on
// MFMA in hils_prefill.hip).
//
// Row kernels: one wavefront scores and selects for one (b, KV group, query)
// row; one 256-thread workgroup computes the local-window term, the per-chunk
// terms and their fusion for one row.
#include "hils_device.hpp"
#include "hils_dispatch.hpp"
#include "hils_internal.hpp"

namespace hils {

constexpr int kBlock = 256;
constexpr int kSlice = 1024;  // candidates scored per selection round of one wave

__device__ __forceinline__ int query_position(const FwdArgs& a, int b, int n) {
    if (!a.decode) return n;
    int len = a.seqlens ? a.seqlens[b] : a.L;
    len = len < 1 ? 1 : (len > a.L ? a.L : len);
    return len - 1;
}

// ---------------------------------------------------------------------------
// Landmark scoring + group max + top-K (Eq. (9), Sec. 4.1 / App. C).
// Grid: ceil(rows / 4) blocks of 4 waves; wave w owns row blockIdx.x*4 + w,
// rows ordered (b, g, n).  The candidates C_i are scored in slices of kSlice;
// each slice is merged with the running top-K by an exact wave radix select.
// ---------------------------------------------------------------------------
template <typename T, int D, int G>
__global__ __launch_bounds__(kBlock) void k_score_topk_rows(FwdArgs a) {
    __shared__ float s_q[4][G][D];
    __shared__ float s_sc[4][kSlice + 64];
    __shared__ int s_id[4][kSlice + 64];
    __shared__ int s_bid[4][64];
    __shared__ float s_bsc[4][64];
    __shared__ int s_tid[4][64];
    __shared__ float s_tsc[4][64];

    const int wave = wave_id(), lane = threadIdx.x % kWave;
    const long row = (long)blockIdx.x * 4 + wave;
    if (row >= (long)a.B * a.Hkv * a.N) return;  // whole wave leaves; no block barriers below
    const int n = (int)(row % a.N);
    const int g = (int)((row / a.N) % a.Hkv);
    const int b = (int)(row / ((long)a.N * a.Hkv));
    const int pos = query_position(a, b, n);
    const int ncand = n_candidates(pos, a.W);
    const int nC = a.L / kChunk;

    const T* qr = as<T>(a.q_route ? a.q_route : a.q);
    for (int e = lane; e < G * D; e += kWave) {
        const int hh = e / D, dd = e % D;
        s_q[wave][hh][dd] = to_f32(qr[(((size_t)b * a.Hq + g * G + hh) * a.N + n) * D + dd]);
    }
    __builtin_amdgcn_wave_barrier();

    // s^ of head hh for chunk c (Eq. (9) with Eq. (11))
    auto score = [&](int hh, int c) {
        const int hl = (a.Hl == a.Hq) ? g * G + hh : g;
        const T* lr = as<T>(a.lmk) + (((size_t)b * a.Hl + hl) * nC + c) * D;
        float acc = 0.f;
#pragma unroll 4
        for (int dd = 0; dd < D; dd += 8) {
            float x[8];
            load8(lr + dd, x);
#pragma unroll
            for (int t = 0; t < 8; ++t) acc += s_q[wave][hh][dd + t] * x[t];
        }
        float sv = a.scale * acc;
        if (a.bias) sv += a.bias[((size_t)b * a.Hl + hl) * nC + c];
        return sv;
    };
    // per-head normalised ranking: each head's log-sum-exp over C_i first
    float lse[G];
#pragma unroll
    for (int hh = 0; hh < G; ++hh) lse[hh] = 0.f;
    if (a.head_norm && ncand > 0) {
#pragma unroll 1
        for (int hh = 0; hh < G; ++hh) {
            float m = -INFINITY, sum = 0.f;
            for (int c = lane; c < ncand; c += kWave) {
                const float sv = score(hh, c);
                const float nm = fmaxf(m, sv);
                sum = sum * fexp(m - nm) + fexp(sv - nm);
                m = nm;
            }
            const float M = wave_max(m);
            const float S = wave_sum(m == -INFINITY ? 0.f : sum * fexp(m - M));
            lse[hh] = M + __logf(S);
        }
    }

    int nbest = 0;
    for (int s0 = 0; s0 < ncand; s0 += kSlice) {
        const int len = min(kSlice, ncand - s0);
        for (int e = lane; e < len; e += kWave) {
            const int c = s0 + e;
            float best = -INFINITY;
#pragma unroll
            for (int hh = 0; hh < G; ++hh) best = fmaxf(best, score(hh, c) - lse[hh]);
            s_sc[wave][e] = best;
            s_id[wave][e] = c;
        }
        for (int t = lane; t < nbest; t += kWave) {
            s_sc[wave][len + t] = s_bsc[wave][t];
            s_id[wave][len + t] = s_bid[wave][t];
        }
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        nbest = wave_topk(s_sc[wave], s_id[wave], len + nbest, a.K, s_bid[wave], s_bsc[wave], s_tid[wave],
                          s_tsc[wave]);
    }
    int32_t* orow = a.idx + (((size_t)b * a.Hkv + g) * a.N + n) * a.K;
    for (int t = lane; t < a.K; t += kWave) orow[t] = t < nbest ? s_bid[wave][t] : -1;
}

// ---------------------------------------------------------------------------
// Local window + per-chunk softmax + fusion (Eqs. (1), (10)) for one row.
// Grid (N, Hkv, B), 256 threads.  Parts are 64-key blocks: the selected
// chunks, then the chunk-aligned pieces of the local window [l(i), i] (the
// last piece is cut at i).  Each part is staged in LDS; wave w computes the
// logits of heads w, w+4, ...; the G*D outputs are spread over the block.
// ---------------------------------------------------------------------------
template <typename T, int D, int G>
__global__ __launch_bounds__(kBlock) void k_attn_rows(FwdArgs a) {
    constexpr int R = (G * D + kBlock - 1) / kBlock;
    __shared__ float s_q[G][D];
    __shared__ float s_qr[G][D];
    __shared__ float s_k[kChunk][D + 1];
    __shared__ float s_v[kChunk][D];
    __shared__ float s_p[G][kChunk];
    __shared__ float s_m[G], s_l[G], s_sh[G];
    __shared__ int s_sel[64];
    __shared__ int s_nsel;

    const int tid = threadIdx.x, wave = wave_id(), lane = tid % kWave;
    const int n = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
    const int pos = query_position(a, b, n);
    const int ncand = n_candidates(pos, a.W);
    const int nC = a.L / kChunk;
    const T* q = as<T>(a.q);
    const T* qr = as<T>(a.q_route ? a.q_route : a.q);
    const T* kb = as<T>(a.k) + ((size_t)b * a.Hkv + g) * a.L * D;
    const T* vb = as<T>(a.v) + ((size_t)b * a.Hkv + g) * a.L * D;

    for (int e = tid; e < G * D; e += kBlock) {
        const int hh = e / D, dd = e % D;
        const size_t off = (((size_t)b * a.Hq + g * G + hh) * a.N + n) * D + dd;
        s_q[hh][dd] = to_f32(q[off]);
        s_qr[hh][dd] = to_f32(qr[off]);
    }
    if (tid == 0) {
        const int32_t* irow = a.idx + (((size_t)b * a.Hkv + g) * a.N + n) * a.K;
        int cnt = 0;
        for (int t = 0; t < a.K; ++t)
            if (idx_entry_valid(irow, t, ncand)) s_sel[cnt++] = irow[t];
        s_nsel = cnt;
    }
    __syncthreads();
    const int nsel = s_nsel;
    const int c_lo = ncand, c_hi = pos / kChunk;
    const int nparts = nsel + (c_hi - c_lo + 1);

    float accl[R], fus[R], m0[R], l0[R], Mf[R], Zf[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        accl[r] = 0.f; fus[r] = 0.f; m0[r] = -INFINITY; l0[r] = 0.f; Mf[r] = -INFINITY; Zf[r] = 0.f;
    }

    for (int part = 0; part < nparts; ++part) {
        const bool is_chunk = part < nsel;
        const int c = is_chunk ? s_sel[part] : c_lo + (part - nsel);
        const int j0 = c * kChunk;
        const int nk = is_chunk ? kChunk : min(kChunk, pos - j0 + 1);
        for (int e = tid; e < kChunk * D / 8; e += kBlock) {
            const int j = e / (D / 8), dd = (e % (D / 8)) * 8;
            float x[8], y[8];
            load8(kb + (size_t)(j0 + j) * D + dd, x);
            load8(vb + (size_t)(j0 + j) * D + dd, y);
#pragma unroll
            for (int t = 0; t < 8; ++t) {
                s_k[j][dd + t] = x[t];
                s_v[j][dd + t] = y[t];
            }
        }
        __syncthreads();
        for (int hh = wave; hh < G; hh += 4) {
            float s = -INFINITY;
            if (lane < nk) {
                float acc = 0.f;
#pragma unroll 16
                for (int dd = 0; dd < D; ++dd) acc += s_q[hh][dd] * s_k[lane][dd];
                s = a.scale * acc;
            }
            const float m = wave_max(s);
            const float p = lane < nk ? fexp(s - m) : 0.f;
            const float l = wave_sum(p);
            s_p[hh][lane] = p;
            float sh = 0.f;
            if (is_chunk) {
                const int hl = (a.Hl == a.Hq) ? g * G + hh : g;
                const T* lr = as<T>(a.lmk) + (((size_t)b * a.Hl + hl) * nC + c) * D;
                float acc = 0.f;
                for (int dd = lane; dd < D; dd += kWave) acc += s_qr[hh][dd] * to_f32(lr[dd]);
                acc = wave_sum(acc);
                sh = a.scale * acc + (a.bias ? a.bias[((size_t)b * a.Hl + hl) * nC + c] : 0.f);
            }
            if (lane == 0) {
                s_m[hh] = m;
                s_l[hh] = l;
                s_sh[hh] = sh;
            }
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int o = tid + r * kBlock;
            if (o < G * D) {
                const int hh = o / D, dd = o % D;
                float acc = 0.f;
                for (int j = 0; j < nk; ++j) acc += s_p[hh][j] * s_v[j][dd];
                const float m = s_m[hh], l = s_l[hh];
                if (is_chunk) {
                    // chunk term: log-mass s^_c, normalised intra-chunk output
                    const float oc = acc / l, z = s_sh[hh];
                    const float mn = fmaxf(Mf[r], z);
                    const float eo = fexp(Mf[r] - mn), ez = fexp(z - mn);
                    Zf[r] = Zf[r] * eo + ez;
                    fus[r] = fus[r] * eo + ez * oc;
                    Mf[r] = mn;
                } else {
                    // local window: online softmax across its pieces
                    const float mn = fmaxf(m0[r], m);
                    const float eo = fexp(m0[r] - mn), en = fexp(m - mn);
                    l0[r] = l0[r] * eo + l * en;
                    accl[r] = accl[r] * eo + acc * en;
                    m0[r] = mn;
                }
            }
        }
        __syncthreads();
    }

    T* out = as_mut<T>(a.out);
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int o = tid + r * kBlock;
        if (o < G * D) {
            const int hh = o / D, dd = o % D;
            const float lam0 = m0[r] + __logf(l0[r]);  // log Z_swa
            const float o0 = accl[r] / l0[r];
            const float mn = fmaxf(Mf[r], lam0);
            const float eo = fexp(Mf[r] - mn), ez = fexp(lam0 - mn);
            const float Z = Zf[r] * eo + ez;
            const float F = fus[r] * eo + ez * o0;
            const size_t row = ((size_t)b * a.Hq + g * G + hh) * a.N + n;
            out[row * D + dd] = from_f32<T>(F / Z);
            if (dd == 0) a.lse[row] = mn + __logf(Z);
        }
    }
}

struct FwdRun {
    template <typename T, int D, int G>
    static hipError_t run(const FwdArgs& a, hipStream_t s) {
        if (!a.given_idx) {
            const long rows = (long)a.B * a.Hkv * a.N;
            HILS_LAUNCH("k_score_topk_rows", (k_score_topk_rows<T, D, G>), dim3((unsigned)((rows + 3) / 4)), dim3(kBlock), 0, s, a);
        }
        HILS_LAUNCH("k_attn_rows", (k_attn_rows<T, D, G>), dim3(a.N, a.Hkv, a.B), dim3(kBlock), 0, s, a);
        return hipGetLastError();
    }
};

hipError_t launch_prefill_rows(const FwdArgs& a, hipStream_t s) {
    return dispatch<FwdRun>(a.bf16, a.d, a.Hq / a.Hkv, a, s);
}

}  // namespace hils
