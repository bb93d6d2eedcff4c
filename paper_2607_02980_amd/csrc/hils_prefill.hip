// HiLS attention prefill forward on MFMA (bf16 storage, fp32 accumulation), gfx950.
//
//   P1 k_pf_score    per 64-query tile: s^_hc = scale * q^_h . k'_c (+ b') on 16x16x32
//                    MFMA tiles, the group max over the G heads (App. C), and the
//                    top-K of every row (exact register radix select, Eq. (9)).  Also
//                    writes ref = the row's best group score (>= every selected s^_hc).
//   inverse index    rows that selected each (b, g, chunk)
//   P3 k_pf_chunks   chunk-major: K_c, V_c staged once in LDS, the selecting rows
//                    gathered 16 at a time; S^T = K_c Q^T, the intra-chunk softmax
//                    (Eq. (10)) and s^ of the (row, head, chunk).  Each (row, head,
//                    slot) gets its chunk output o_c (bf16 partial) and the weight
//                    exp(s^ - ref) (float).  A chunk's rows are scattered over the
//                    sequence, so per-slot partials replace atomics (float atomics on
//                    gfx950 sustain ~0.3 G-ops/ms, 7 ms for the 32K workload).
//   P2 k_pf_local    flash-style local window [l(i), i] (Eq. (1)) per 16*QB-query
//                    tile, then the fusion (Eq. (10)) with the row's slots summed in
//                    slot order: acc = sum_k w_k o_k, zsum = sum_k w_k, M = max(log Z_swa, ref),
//                    out = (e^{log Z_swa - M} o_swa + e^{ref - M} acc) / (e^{log Z_swa - M} + e^{ref - M} zsum),
//                    lse = M + log(denominator).
//
// MFMA orientation: attention tiles compute S^T = K Q^T (keys on the M side,
// queries on N).  The accumulator then holds, in lane l, 4 consecutive keys of
// query l%16, which is exactly the B-operand layout of O^T = V^T P^T when the
// keys of a 32-key step are taken in the order the accumulators hold them
// ({4g..4g+3} U {16+4g..16+4g+3} for lane group g = l/16); V^T is staged in
// LDS so the matching A-operand reads are two 8-byte loads.  Every O^T value a
// lane holds belongs to its own query, so softmax rescaling is lane-local.
#include "hils_device.hpp"
#include "hils_dispatch.hpp"
#include "hils_internal.hpp"
#include "hils_mfma.hpp"

namespace hils {

namespace {

constexpr int kBlock = 256;
constexpr int kSQ = 64;   // queries per score tile (4 waves x 16)
constexpr int kSL = 256;  // candidate chunks per score slice

struct PfLayout {
    size_t part, wgt, ref, inv_base;
    InvLayout inv;
    size_t total;
};

// part [B, Hq, N, K, d] bf16, wgt [B, Hq, N, K] f32, ref [B, Hkv, N] f32, inverse index
PfLayout pf_layout(int B, int Hq, int Hkv, int N, int L, int d, int K) {
    PfLayout w;
    w.part = 0;
    w.wgt = align256(w.part + (size_t)B * Hq * N * K * d * sizeof(uint16_t));
    w.ref = align256(w.wgt + (size_t)B * Hq * N * K * sizeof(float));
    w.inv_base = align256(w.ref + (size_t)B * Hkv * N * sizeof(float));
    w.inv = inv_layout(B, Hkv, N, L, K, w.inv_base);
    w.total = w.inv.end;
    return w;
}

template <int D>
struct Tiles {
    static constexpr int KS = D / 32;      // k-steps over the head dimension
    static constexpr int DB = D / 16;      // 16-wide blocks of the head dimension
    static constexpr int KROW = D + 8;     // bf16 per padded K row in LDS
    static constexpr int VROW = 64 + 8;    // bf16 per padded V^T row in LDS
};

// Stage one 64-key block: K rows (padded) and V transposed into LDS.
template <int D>
__device__ __forceinline__ void stage_kv(const bf16* kb, const bf16* vb, bf16* s_k, bf16* s_vt) {
    constexpr int KROW = Tiles<D>::KROW, VROW = Tiles<D>::VROW;
    constexpr int PPT = kChunk * D / 8 / kBlock;  // 16-byte pieces per thread
    const int tid = threadIdx.x;
    uint4 xk[PPT], xv[PPT];
#pragma unroll
    for (int u = 0; u < PPT; ++u) {
        const int e = tid + u * kBlock, j = e / (D / 8), d8 = (e % (D / 8)) * 8;
        xk[u] = *reinterpret_cast<const uint4*>(kb + (size_t)j * D + d8);
        xv[u] = *reinterpret_cast<const uint4*>(vb + (size_t)j * D + d8);
    }
#pragma unroll
    for (int u = 0; u < PPT; ++u) {
        const int e = tid + u * kBlock, j = e / (D / 8), d8 = (e % (D / 8)) * 8;
        *reinterpret_cast<uint4*>(s_k + j * KROW + d8) = xk[u];
        const uint32_t w[4] = {xv[u].x, xv[u].y, xv[u].z, xv[u].w};
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            s_vt[(d8 + 2 * t) * VROW + j].bits = (uint16_t)(w[t] & 0xffffu);
            s_vt[(d8 + 2 * t + 1) * VROW + j].bits = (uint16_t)(w[t] >> 16);
        }
    }
}

// A operand of S^T = K Q^T for key block kb (16 keys) and k-step ks.
template <int D>
__device__ __forceinline__ bf16x8 k_operand(const bf16* s_k, int kb, int ks, int lane) {
    return ld_bf16x8(s_k + (kb * 16 + lane % 16) * Tiles<D>::KROW + ks * 32 + (lane / 16) * 8);
}

// A operand of O^T = V^T P^T for dims block db and 32-key step t (permuted key order).
template <int D>
__device__ __forceinline__ bf16x8 vt_operand(const bf16* s_vt, int db, int t, int lane) {
    const bf16* row = s_vt + (db * 16 + lane % 16) * Tiles<D>::VROW + 32 * t + (lane / 16) * 4;
    const uint2 lo = *reinterpret_cast<const uint2*>(row);
    const uint2 hi = *reinterpret_cast<const uint2*>(row + 16);
    return as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y));
}

// B operand of O^T = V^T P^T from exponentiated S^T accumulators of key blocks 2t, 2t+1.
__device__ __forceinline__ bf16x8 p_operand(const float* e0, const float* e1) {
    float x[8] = {e0[0], e0[1], e0[2], e0[3], e1[0], e1[1], e1[2], e1[3]};
    return pack_bf16x8(x);
}

// ---------------------------------------------------------------------------
// P1: scores, group max, top-K
// ---------------------------------------------------------------------------
template <int D, int G>
__global__ __launch_bounds__(kBlock) void k_pf_score(FwdArgs a, float* ref_out) {
    constexpr int KS = Tiles<D>::KS;
    constexpr int NCB = kSL / 16;
    constexpr int E = kSL / kWave;
    __shared__ float s_sig[kSQ][kSL + 1];
    __shared__ int s_tid[4][64], s_oid[4][64];
    __shared__ float s_tsc[4][64], s_osc[4][64];
    const int tid = threadIdx.x, w = wave_id(), lane = tid % kWave;
    const int ntiles = (a.N + kSQ - 1) / kSQ;
    const int tile = xcd_remap(blockIdx.x, ntiles), g = blockIdx.y, b = blockIdx.z;
    const int q0 = tile * kSQ;
    const int qlast = min(q0 + kSQ - 1, a.N - 1);
    const int nct = n_candidates(qlast, a.W);
    const int nC = a.L / kChunk;
    const int qw0 = q0 + 16 * w;
    const bf16* qr = as<bf16>(a.q_route ? a.q_route : a.q);
    const bf16* lmk = as<bf16>(a.lmk);

    float bsc[16];
    int bid[16], nb[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        bsc[r] = 0.f;
        bid[r] = -1;
        nb[r] = 0;
    }
    for (int s0 = 0; s0 < nct; s0 += kSL) {
        const int len = min(kSL, nct - s0);
        const int ncb = (len + 15) / 16;
        f32x4 sig[NCB];
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) sig[cb] = f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
        for (int hh = 0; hh < G; ++hh) {
            const int h = g * G + hh, hl = (a.Hl == a.Hq) ? h : g;
            const int qa = min(qw0 + lane % 16, a.N - 1);
            bf16x8 aq[KS];
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                aq[ks] = ld_bf16x8(qr + (((size_t)b * a.Hq + h) * a.N + qa) * D + ks * 32 + (lane / 16) * 8);
            const bf16* lbase = lmk + ((size_t)b * a.Hl + hl) * nC * D;
            const float* bbase = a.bias ? a.bias + ((size_t)b * a.Hl + hl) * nC : nullptr;
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) {
                if (cb < ncb) {
                    const int c = min(s0 + cb * 16 + lane % 16, nC - 1);
                    bf16x8 bl[KS];
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) bl[ks] = ld_bf16x8(lbase + (size_t)c * D + ks * 32 + (lane / 16) * 8);
                    f32x4 acc4 = zero4();
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) acc4 = mfma16x16x32(aq[ks], bl[ks], acc4);
                    const float bv = bbase ? bbase[c] : 0.f;
#pragma unroll
                    for (int i = 0; i < 4; ++i) sig[cb][i] = fmaxf(sig[cb][i], a.scale * acc4[i] + bv);
                }
            }
        }
        // this wave's 16 rows -> LDS (row = 16w + (l/16)*4 + i, column = 16cb + l%16)
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
            if (cb < ncb) {
#pragma unroll
                for (int i = 0; i < 4; ++i) s_sig[16 * w + (lane / 16) * 4 + i][cb * 16 + lane % 16] = sig[cb][i];
            }
        }
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int n = qw0 + r;
            if (n >= a.N) break;
            const int lim = min(n_candidates(n, a.W), s0 + len) - s0;
            if (lim <= 0) continue;
            float sc[E + 1];
            int id[E + 1];
            bool ok[E + 1];
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const int col = e * kWave + lane;
                ok[e] = col < lim;
                sc[e] = ok[e] ? s_sig[16 * w + r][col] : 0.f;
                id[e] = s0 + col;
            }
            ok[E] = lane < nb[r];
            sc[E] = bsc[r];
            id[E] = bid[r];
            nb[r] = wave_topk_reg<E + 1>(sc, id, ok, a.K, s_oid[w], s_osc[w], s_tid[w], s_tsc[w]);
            bsc[r] = lane < nb[r] ? s_osc[w][lane] : 0.f;
            bid[r] = lane < nb[r] ? s_oid[w][lane] : -1;
        }
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int n = qw0 + r;
        if (n >= a.N) break;
        int32_t* orow = a.idx + (((size_t)b * a.Hkv + g) * a.N + n) * a.K;
        if (lane < a.K) orow[lane] = lane < nb[r] ? bid[r] : -1;
        const float top = wave_max(lane < nb[r] ? bsc[r] : -INFINITY);
        if (lane == 0) ref_out[((size_t)b * a.Hkv + g) * a.N + n] = top;
    }
}

// Forced selection: ref = the best group score among the given chunks.
// One wave per (n, g, b) row.
template <int D, int G>
__global__ __launch_bounds__(kWave) void k_pf_ref_given(FwdArgs a, float* ref_out) {
    const int n = blockIdx.x, g = blockIdx.y, b = blockIdx.z, lane = threadIdx.x;
    const int nC = a.L / kChunk;
    const int32_t* irow = a.idx + (((size_t)b * a.Hkv + g) * a.N + n) * a.K;
    const int ncand = n_candidates(n, a.W);
    float best = -INFINITY;
    if (lane < a.K && idx_entry_valid(irow, lane, ncand)) {
        const int c = irow[lane];
        const bf16* qr = as<bf16>(a.q_route ? a.q_route : a.q);
        for (int hh = 0; hh < G; ++hh) {
            const int h = g * G + hh, hl = (a.Hl == a.Hq) ? h : g;
            const bf16* qrow = qr + (((size_t)b * a.Hq + h) * a.N + n) * D;
            const bf16* lrow = as<bf16>(a.lmk) + (((size_t)b * a.Hl + hl) * nC + c) * D;
            float d0 = 0.f;
            for (int dd = 0; dd < D; dd += 8) {
                float x[8], y[8];
                load8(qrow + dd, x);
                load8(lrow + dd, y);
#pragma unroll
                for (int t = 0; t < 8; ++t) d0 += x[t] * y[t];
            }
            best = fmaxf(best, a.scale * d0 + (a.bias ? a.bias[((size_t)b * a.Hl + hl) * nC + c] : 0.f));
        }
    }
    best = wave_max(best);
    if (lane == 0) ref_out[((size_t)b * a.Hkv + g) * a.N + n] = best;
}

// ---------------------------------------------------------------------------
// P3: retrieved chunks, chunk-major
// ---------------------------------------------------------------------------
// One block per work item: kInvSeg consecutive entries of one (b, g, chunk) list.
template <int D, int G>
__global__ __launch_bounds__(kBlock) void k_pf_chunks(FwdArgs a, const int* offsets, const int* list,
                                                      const int4* work, const int* nwork, const float* ref,
                                                      bf16* part, float* wgt) {
    constexpr int KS = Tiles<D>::KS, DB = Tiles<D>::DB;
    __shared__ __align__(16) bf16 s_k[kChunk * Tiles<D>::KROW];
    __shared__ __align__(16) bf16 s_vt[D * Tiles<D>::VROW];
    const int tid = threadIdx.x, w = wave_id(), lane = tid % kWave;
    const int nC = a.L / kChunk;
    if ((int)blockIdx.x >= *nwork) return;
    const int4 wi = work[blockIdx.x];
    const int c = wi.y;
    const size_t bg = (size_t)wi.x;
    const int b = (int)(bg / a.Hkv), g = (int)(bg % a.Hkv);
    const int beg = offsets[bg * (nC + 1) + c] + wi.z * kInvSeg;
    const int len = min(kInvSeg, offsets[bg * (nC + 1) + c + 1] - beg);
    if (len <= 0) return;
    const int* seg = list + bg * a.N * a.K + beg;
    stage_kv<D>(as<bf16>(a.k) + (bg * a.L + (size_t)c * kChunk) * D, as<bf16>(a.v) + (bg * a.L + (size_t)c * kChunk) * D,
                s_k, s_vt);
    __syncthreads();
    const bf16* qbase = as<bf16>(a.q);
    const bf16* rbase = as<bf16>(a.q_route);
    for (int e0 = 0; e0 < len; e0 += 16) {
        const int e = e0 + lane % 16;
        const bool qv = e < len;
        const int ent = qv ? seg[e] : 0;
        const int n = ent >> 6, slot = ent & 63;
        const float rf = qv ? ref[bg * a.N + n] : 0.f;
        for (int hh = w; hh < G; hh += 4) {
            const int h = g * G + hh, hl = (a.Hl == a.Hq) ? h : g;
            const size_t qrow = ((size_t)b * a.Hq + h) * a.N + n;
            bf16x8 bq[KS];
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                bq[ks] = qv ? ld_bf16x8(qbase + qrow * D + ks * 32 + (lane / 16) * 8) : as_bf16x8(make_uint4(0, 0, 0, 0));
            // surrogate score s^ = q^ . k'_c: the landmark row is row 0 of the A tile
            f32x4 sh4 = zero4();
            const bf16* lrow = as<bf16>(a.lmk) + (((size_t)b * a.Hl + hl) * nC + c) * D;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const bf16x8 al = (lane % 16 == 0) ? ld_bf16x8(lrow + ks * 32 + (lane / 16) * 8)
                                                   : as_bf16x8(make_uint4(0, 0, 0, 0));
                const bf16x8 br = (rbase && qv) ? ld_bf16x8(rbase + qrow * D + ks * 32 + (lane / 16) * 8) : bq[ks];
                sh4 = mfma16x16x32(al, br, sh4);
            }
            float shat = __shfl(sh4[0], lane % 16, kWave);
            shat = a.scale * shat + (a.bias ? a.bias[((size_t)b * a.Hl + hl) * nC + c] : 0.f);
            // S^T = K_c Q^T
            f32x4 st[4];
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) {
                st[kb] = zero4();
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) st[kb] = mfma16x16x32(k_operand<D>(s_k, kb, ks, lane), bq[ks], st[kb]);
            }
            float mx = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    st[kb][i] *= a.scale;
                    mx = fmaxf(mx, st[kb][i]);
                }
            mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
            mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
            float sum = 0.f;
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) sum += fexp(st[kb][i] - mx);
            sum += __shfl_xor(sum, 16, kWave);
            sum += __shfl_xor(sum, 32, kWave);
            // intra-chunk softmax: p_j = exp(s_j - lse_c)
            const float off = qv ? -(mx + __logf(sum)) : -INFINITY;
            float ex[4][4];
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) ex[kb][i] = fexp(st[kb][i] + off);
            const bf16x8 pb0 = p_operand(ex[0], ex[1]);
            const bf16x8 pb1 = p_operand(ex[2], ex[3]);
            bf16* prow = part + (qrow * a.K + slot) * D;
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                f32x4 o = zero4();
                o = mfma16x16x32(vt_operand<D>(s_vt, db, 0, lane), pb0, o);
                o = mfma16x16x32(vt_operand<D>(s_vt, db, 1, lane), pb1, o);
                if (qv) {
                    const uint32_t lo = from_f32<bf16>(o[0]).bits | ((uint32_t)from_f32<bf16>(o[1]).bits << 16);
                    const uint32_t hi = from_f32<bf16>(o[2]).bits | ((uint32_t)from_f32<bf16>(o[3]).bits << 16);
                    *reinterpret_cast<uint2*>(prow + db * 16 + (lane / 16) * 4) = make_uint2(lo, hi);
                }
            }
            if (qv && lane < 16) wgt[qrow * a.K + slot] = fexp(shat - rf);
        }
    }
}

// ---------------------------------------------------------------------------
// P2: local window (flash style) + fusion epilogue
// ---------------------------------------------------------------------------
template <int G>
struct LocalCfg {
    static constexpr int QB = G >= 8 ? 1 : 8 / G;  // 16-query blocks per tile
    static constexpr int QT = 16 * QB;
    static constexpr int ITEMS = G * QB;           // (head, query block) items
    static constexpr int IPW = (ITEMS + 3) / 4;    // items per wave
};

template <int D, int G>
__global__ __launch_bounds__(kBlock) void k_pf_local(FwdArgs a, const float* ref, const bf16* part, const float* wgt) {
    using C = LocalCfg<G>;
    constexpr int KS = Tiles<D>::KS, DB = Tiles<D>::DB, IPW = C::IPW;
    __shared__ __align__(16) bf16 s_k[kChunk * Tiles<D>::KROW];
    __shared__ __align__(16) bf16 s_vt[D * Tiles<D>::VROW];
    const int tid = threadIdx.x, w = wave_id(), lane = tid % kWave;
    const int ntiles = (a.N + C::QT - 1) / C::QT;
    const int tile = xcd_remap(blockIdx.x, ntiles), g = blockIdx.y, b = blockIdx.z;
    const int q0 = tile * C::QT;
    const int qlast = min(q0 + C::QT - 1, a.N - 1);
    const int kbeg = n_candidates(q0, a.W) * kChunk;
    const size_t bg = (size_t)b * a.Hkv + g;
    const bf16* kbase = as<bf16>(a.k) + bg * a.L * D;
    const bf16* vbase = as<bf16>(a.v) + bg * a.L * D;

    bf16x8 bq[IPW][KS];
    f32x4 o[IPW][DB];
    float m[IPW], l[IPW];
#pragma unroll
    for (int it = 0; it < IPW; ++it) {
        const int item = w + 4 * it;
        m[it] = -INFINITY;
        l[it] = 0.f;
#pragma unroll
        for (int db = 0; db < DB; ++db) o[it][db] = zero4();
        if (item < C::ITEMS) {
            const int hh = item / C::QB, qb = item % C::QB;
            const int nq = min(q0 + qb * 16 + lane % 16, a.N - 1);
            const bf16* qrow = as<bf16>(a.q) + (((size_t)b * a.Hq + g * G + hh) * a.N + nq) * D;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) bq[it][ks] = ld_bf16x8(qrow + ks * 32 + (lane / 16) * 8);
        }
    }

    for (int j0 = kbeg; j0 <= qlast; j0 += kChunk) {
        __syncthreads();
        stage_kv<D>(kbase + (size_t)j0 * D, vbase + (size_t)j0 * D, s_k, s_vt);
        __syncthreads();
#pragma unroll
        for (int it = 0; it < IPW; ++it) {
            const int item = w + 4 * it;
            if (item >= C::ITEMS) continue;
            const int qb = item % C::QB;
            const int nq = q0 + qb * 16 + lane % 16;
            const int ell = n_candidates(nq, a.W) * kChunk;
            f32x4 st[4];
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) {
                st[kb] = zero4();
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) st[kb] = mfma16x16x32(k_operand<D>(s_k, kb, ks, lane), bq[it][ks], st[kb]);
            }
            float mx = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int j = j0 + kb * 16 + (lane / 16) * 4 + i;
                    const bool valid = nq < a.N && j <= nq && j >= ell;
                    st[kb][i] = valid ? a.scale * st[kb][i] : -INFINITY;
                    mx = fmaxf(mx, st[kb][i]);
                }
            mx = fmaxf(mx, __shfl_xor(mx, 16, kWave));
            mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
            const float mnew = fmaxf(m[it], mx);
            const float muse = mnew == -INFINITY ? 0.f : mnew;
            const float alpha = fexp(m[it] - muse);
            float ex[4][4], psum = 0.f;
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    ex[kb][i] = fexp(st[kb][i] - muse);
                    psum += ex[kb][i];
                }
            psum += __shfl_xor(psum, 16, kWave);
            psum += __shfl_xor(psum, 32, kWave);
            l[it] = l[it] * alpha + psum;
            m[it] = mnew;
            const bf16x8 pb0 = p_operand(ex[0], ex[1]);
            const bf16x8 pb1 = p_operand(ex[2], ex[3]);
#pragma unroll
            for (int db = 0; db < DB; ++db) {
#pragma unroll
                for (int i = 0; i < 4; ++i) o[it][db][i] *= alpha;
                o[it][db] = mfma16x16x32(vt_operand<D>(s_vt, db, 0, lane), pb0, o[it][db]);
                o[it][db] = mfma16x16x32(vt_operand<D>(s_vt, db, 1, lane), pb1, o[it][db]);
            }
        }
    }

    // fusion epilogue
    bf16* out = as_mut<bf16>(a.out);
#pragma unroll
    for (int it = 0; it < IPW; ++it) {
        const int item = w + 4 * it;
        if (item >= C::ITEMS) continue;
        const int hh = item / C::QB, qb = item % C::QB;
        const int nq = q0 + qb * 16 + lane % 16;
        if (nq >= a.N) continue;
        const size_t row = ((size_t)b * a.Hq + g * G + hh) * a.N + nq;
        const float lam0 = m[it] + __logf(l[it]);
        const float rf = ref[bg * a.N + nq];
        // the row's retrieved chunks: slots in idx order, valid entries only
        const int32_t* irow = a.idx + (bg * a.N + nq) * a.K;
        const int ncand = n_candidates(nq, a.W);
        float zs = 0.f;
        f32x4 av[DB];
#pragma unroll
        for (int db = 0; db < DB; ++db) av[db] = zero4();
        // slots in groups of SB, every load of a group issued before any use
        constexpr int SB = 4;
        for (int k0 = 0; k0 < a.K; k0 += SB) {
            float wk[SB];
            uint2 pv[SB][DB];
#pragma unroll
            for (int u = 0; u < SB; ++u) {
                const int k = k0 + u;
                const bool ok = k < a.K && idx_entry_valid(irow, k, ncand);
                wk[u] = ok ? wgt[row * a.K + k] : 0.f;
                const bf16* prow = part + (row * a.K + (ok ? k : 0)) * D;
#pragma unroll
                for (int db = 0; db < DB; ++db)
                    pv[u][db] = ok ? *reinterpret_cast<const uint2*>(prow + db * 16 + (lane / 16) * 4) : make_uint2(0, 0);
            }
#pragma unroll
            for (int u = 0; u < SB; ++u) {
                zs += wk[u];
#pragma unroll
                for (int db = 0; db < DB; ++db) {
                    av[db][0] += wk[u] * __uint_as_float(pv[u][db].x << 16);
                    av[db][1] += wk[u] * __uint_as_float(pv[u][db].x & 0xffff0000u);
                    av[db][2] += wk[u] * __uint_as_float(pv[u][db].y << 16);
                    av[db][3] += wk[u] * __uint_as_float(pv[u][db].y & 0xffff0000u);
                }
            }
        }
        const float M = fmaxf(lam0, rf);
        const float wl = fexp(lam0 - M) / l[it];
        const float wc = zs > 0.f ? fexp(rf - M) : 0.f;
        const float Z = fexp(lam0 - M) + wc * zs;
        const float inv = 1.f / Z;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
            const int d0 = db * 16 + (lane / 16) * 4;
            const float r0 = (wl * o[it][db][0] + wc * av[db][0]) * inv;
            const float r1 = (wl * o[it][db][1] + wc * av[db][1]) * inv;
            const float r2 = (wl * o[it][db][2] + wc * av[db][2]) * inv;
            const float r3 = (wl * o[it][db][3] + wc * av[db][3]) * inv;
            const uint32_t lo = from_f32<bf16>(r0).bits | ((uint32_t)from_f32<bf16>(r1).bits << 16);
            const uint32_t hi = from_f32<bf16>(r2).bits | ((uint32_t)from_f32<bf16>(r3).bits << 16);
            *reinterpret_cast<uint2*>(out + row * D + d0) = make_uint2(lo, hi);
        }
        if (lane < 16) a.lse[row] = M + __logf(Z);
    }
}

struct PfRun {
    template <typename T, int D, int G>
    static hipError_t run(const FwdArgs& a, hipStream_t s) {
        const PfLayout ly = pf_layout(a.B, a.Hq, a.Hkv, a.N, a.L, D, a.K);
        char* ws = static_cast<char*>(a.ws);
        bf16* part = reinterpret_cast<bf16*>(ws + ly.part);
        float* wgt = reinterpret_cast<float*>(ws + ly.wgt);
        float* ref = reinterpret_cast<float*>(ws + ly.ref);
        if (a.given_idx) {
            HILS_LAUNCH("k_pf_ref_given", (k_pf_ref_given<D, G>), dim3(a.N, a.Hkv, a.B), dim3(kWave), 0, s, a, ref);
        } else {
            HILS_LAUNCH("k_pf_score", (k_pf_score<D, G>), dim3((a.N + kSQ - 1) / kSQ, a.Hkv, a.B), dim3(kBlock), 0, s, a,
                               ref);
        }
        const InvArgs ia{a.idx, a.B, a.Hkv, a.N, a.K, a.W, a.L};
        launch_inverse_index(ia, ly.inv, a.ws, s);
        HILS_LAUNCH("k_pf_chunks", (k_pf_chunks<D, G>), dim3((unsigned)ly.inv.max_work), dim3(kBlock), 0, s, a,
                           reinterpret_cast<const int*>(ws + ly.inv.offsets), reinterpret_cast<const int*>(ws + ly.inv.list),
                           reinterpret_cast<const int4*>(ws + ly.inv.work), reinterpret_cast<const int*>(ws + ly.inv.nwork),
                           (const float*)ref, part, wgt);
        HILS_LAUNCH("k_pf_local", (k_pf_local<D, G>), dim3((a.N + LocalCfg<G>::QT - 1) / LocalCfg<G>::QT, a.Hkv, a.B),
                           dim3(kBlock), 0, s, a, (const float*)ref, (const bf16*)part, (const float*)wgt);
        return hipGetLastError();
    }
};

}  // namespace

size_t prefill_workspace_bytes(int B, int Hq, int Hkv, int N, int L, int d, int K, int bf16_storage) {
    if (!bf16_storage) return 0;  // the fp32 path needs no workspace
    return pf_layout(B, Hq, Hkv, N, L, d, K).total;
}

hipError_t launch_prefill_fwd(const FwdArgs& a, hipStream_t s) {
    if (!a.bf16) return launch_prefill_rows(a, s);
    return dispatch<PfRun>(1, a.d, a.Hq / a.Hkv, a, s);
}

}  // namespace hils
