// HiLS attention prefill forward on MFMA (bf16 storage, fp32 accumulation), gfx950.
//
//   P0 k_pf_lse      (per-head normalised ranking) LSE_h over C_i of every (row, head)
//   P1 k_pf_sigma    per 128 queries of a KV group: s^_hc = scale * q^_h . k'_c (+ b')
//      k_pf_select   on 16x16x32 MFMA tiles and the group max over the G heads (App.
//                    C) into the workspace, then the top-K of every row (exact
//                    register radix select, Eq. (9)), one wave per row.  With more
//                    than 1024 candidate chunks, when that array does not fit the
//                    records' area and under union packing, k_pf_score does both
//                    in one pass per 32-query tile.
//   inverse index    rows that selected each (b, g, chunk)
//   P3 k_pf_chunks   chunk-major: K_c, V_c staged once in LDS, the selecting rows
//                    gathered 16 at a time; S^T = K_c Q^T, the intra-chunk softmax
//                    (Eq. (10)) and s^ of the (row, head, chunk).  Each (row, head,
//                    slot) gets its chunk output o_c (bf16 partial) and its raw
//                    surrogate score s^ (float).  A chunk's rows are scattered over the
//                    sequence, so per-slot partials replace atomics (float atomics on
//                    gfx950 sustain ~0.3 G-ops/ms, 7 ms for the 32K workload).
//   P2 k_pf_local    flash-style local window [l(i), i] (Eq. (1)) per tile of 16*8/G
//                    queries x G heads (8 waves), then the fusion (Eq. (10)) of each
//                    (row, head) with its own stabiliser (App. C: the fusion weights
//                    are per head even though the selection is shared):
//                    M = max(log Z_swa, max_k s^_k),
//                    out = (e^{log Z_swa - M} o_swa + sum_k e^{s^_k - M} o_k)
//                          / (e^{log Z_swa - M} + sum_k e^{s^_k - M}),
//                    lse = M + log(denominator).
//
// MFMA orientation: attention tiles compute S^T = K Q^T (keys on the M side,
// queries on N).  The accumulator then holds, in lane l, 4 consecutive keys of
// query l%16, which is exactly the B-operand layout of O^T = V^T P^T when the
// keys of a 32-key step are taken in the order the accumulators hold them
// ({4g..4g+3} U {16+4g..16+4g+3} for lane group g = l/16); V stays row-major in
// LDS and the matching A operands come from transposing reads
// (ds_read_b64_tr_b16).  Every O^T value a lane holds belongs to its own query,
// so softmax rescaling is lane-local.  Per-slot partial vectors are stored in
// the accumulators' lane order (store_lane_order).
#include <atomic>

#include "hils_device.hpp"
#include "hils_dispatch.hpp"
#include "hils_internal.hpp"
#include "hils_mfma.hpp"

namespace hils {

namespace {

constexpr int kBlock = 256;
constexpr int kSQ = 32;   // queries per score tile (two 16-row MFMA tiles)
constexpr int kSL = 256;  // candidate chunks per score slice

struct PfLayout {
    size_t part, wgt, inv_base;
    InvLayout inv;
    size_t total;
};

// part [B, Hkv, N/QT, K, QT, G, d] bf16 with QT = 128 / G, the query tile of the
// local pass (each d-vector in lane order).  The G heads of a (row, slot) are
// adjacent, so the heads' chunk outputs, written by the waves of one workgroup,
// form one contiguous run; slot k of a whole query tile is one contiguous span
// (32 KiB), which the local pass reads while it sums slot k for all its rows
// (the row-major order [N, K, G, d] had it jump 16 KiB between rows: 3% slower
// here, and 4% slower writes).  wgt [B, Hkv, N/QT, K, QT, G] f32 (the raw s^ of
// each (row, slot, head)), inverse index; N rounded up to a multiple of QT.
// Element offset of the partial of (row n, slot, head hh) of KV group bg = b * Hkv + g
// (D = 1: of its weight).
__device__ __forceinline__ size_t part_offset(size_t bg, int N, int n, int K, int slot, int G, int hh, int D) {
    const int QT = 128 / G, nt = (N + QT - 1) / QT;
    return (((((bg * nt + n / QT) * K + slot) * QT + n % QT) * G) + hh) * (size_t)D;
}

// N: rows of one segment; row_end: the rows of every segment lie below it (-1: one
// segment from row 0)
PfLayout pf_layout(int B, int Hq, int Hkv, int N, int L, int d, int K, int row_end = -1) {
    PfLayout w;
    w.part = 0;
    const int QT = 128 / (Hq / Hkv);
    const size_t Np = (size_t)(N + QT - 1) / QT * QT;
    w.wgt = align256(w.part + (size_t)B * Hq * Np * K * d * sizeof(uint16_t));
    w.inv_base = align256(w.wgt + (size_t)B * Hq * Np * K * sizeof(float));
    w.inv = inv_layout(B, Hkv, N, L, K, w.inv_base, row_end);
    w.total = w.inv.end;
    return w;
}

template <int D>
struct Tiles {
    static constexpr int KS = D / 32;      // k-steps over the head dimension
    static constexpr int DB = D / 16;      // 16-wide blocks of the head dimension
    static constexpr int KROW = D + 8;     // bf16 per padded K / V row in LDS
    static constexpr int PPT = kChunk * D / 8 / kBlock;  // 16-byte pieces of a K or V block per thread
};

// One 64-key block of K or V in registers (PPT 16-byte pieces per thread), and its
// store into a padded row-major LDS tile.
template <int D>
struct KVRegs {
    uint4 x[Tiles<D>::PPT];
};
template <int D>
__device__ __forceinline__ KVRegs<D> load_block(const bf16* src) {
    KVRegs<D> r;
#pragma unroll
    for (int u = 0; u < Tiles<D>::PPT; ++u) {
        const int e = threadIdx.x + u * kBlock, j = e / (D / 8), d8 = (e % (D / 8)) * 8;
        r.x[u] = *reinterpret_cast<const uint4*>(src + (size_t)j * D + d8);
    }
    return r;
}
template <int D>
__device__ __forceinline__ void store_block(bf16* tile, const KVRegs<D>& r) {
#pragma unroll
    for (int u = 0; u < Tiles<D>::PPT; ++u) {
        const int e = threadIdx.x + u * kBlock, j = e / (D / 8), d8 = (e % (D / 8)) * 8;
        *reinterpret_cast<uint4*>(tile + j * Tiles<D>::KROW + d8) = r.x[u];
    }
}

// A operand of S^T = K Q^T for key block kb (16 keys) and k-step ks.
template <int D>
__device__ __forceinline__ bf16x8 k_operand(const bf16* s_k, int kb, int ks, int lane) {
    return ld_bf16x8(s_k + (kb * 16 + lane % 16) * Tiles<D>::KROW + ks * 32 + (lane / 16) * 8);
}

// A operand of O^T = V^T P^T for dims block db and 32-key step t (permuted key
// order), read from row-major V with transposing loads.
template <int D>
__device__ __forceinline__ bf16x8 vt_operand(const bf16* s_v, int db, int t, int lane) {
    return tr_operand_perm(s_v, Tiles<D>::KROW, 32 * t, db * 16, lane);
}

// B operand of O^T = V^T P^T from exponentiated S^T accumulators of key blocks 2t, 2t+1.
__device__ __forceinline__ bf16x8 p_operand(const f32x4& e0, const f32x4& e1) {
    float x[8] = {e0[0], e0[1], e0[2], e0[3], e1[0], e1[1], e1[2], e1[3]};
    return pack_bf16x8(x);
}

// ---------------------------------------------------------------------------
// P1: scores, group max, top-K
// ---------------------------------------------------------------------------
// (max, sum of exp) pairs merged over each aligned group of 16 lanes.
__device__ __forceinline__ void lse16_merge(float& m, float& s) {
    auto step = [&](float om, float os) {
        const float nm = fmaxf(m, om);
        s = (m == -INFINITY ? 0.f : s * fexp(m - nm)) + (om == -INFINITY ? 0.f : os * fexp(om - nm));
        m = nm;
    };
    step(dpp<0xB1>(m), dpp<0xB1>(s));
    step(dpp<0x4E>(m), dpp<0x4E>(s));
    step(dpp<0x141>(m), dpp<0x141>(s));
    step(dpp<0x140>(m), dpp<0x140>(s));
}

// NORM: rank by per-head normalised scores: k_pf_lse has left each (row, head)'s
// log-sum-exp over C_i in the lse output, and the scores here subtract it before
// the maximum over the group's heads.
//
// Four waves per 32-row tile: wave w scores chunk blocks w, w + 4, ... of each
// slice against all rows, then selects rows 8w .. 8w + 7 one after another.  Both
// phases are latency-bound (L2 loads, then chains of ballots), so the tile is kept
// small enough (33 KB of scores in LDS, <= 128 VGPRs) for four blocks per CU.  The
// rows' running best lists (K entries each) live in dynamic LDS, so the row loop
// is not unrolled: one copy of the selection code.
constexpr int kSW = 4;           // waves per score block
constexpr int kSR = kSQ / kSW;   // rows selected per wave
size_t score_dyn_lds(int K) { return (size_t)kSQ * K * (sizeof(float) + sizeof(int)) + kSQ * sizeof(int); }
template <int D, int G, bool NORM>
__global__ __launch_bounds__(kSW * kWave, NORM ? 3 : 4) void k_pf_score(FwdArgs a) {
    constexpr int KS = Tiles<D>::KS;
    constexpr int NCB = kSL / 16;
    constexpr int E = kSL / kWave;
    constexpr int NJ = NCB / kSW, NT = kSQ / 16;
    static_assert(NJ * kSW == NCB, "chunk blocks split evenly over the waves");
    __shared__ float s_sig[kSQ][kSL + 1];
    __shared__ int s_tid[kSW][64];
    __shared__ float s_tsc[kSW][64];
    __shared__ float s_lse[NORM ? G : 1][kSQ];
    extern __shared__ int s_dyn[];
    const int K = a.K;
    float* s_bsc = reinterpret_cast<float*>(s_dyn);          // [kSQ][K] running best scores
    int* s_bid = reinterpret_cast<int*>(s_bsc + kSQ * K);    // [kSQ][K] their chunks (ascending)
    int* s_nb = s_bid + kSQ * K;                             // [kSQ] list lengths
    const int tid = threadIdx.x, w = wave_id(), lane = tid % kWave;
    // 1-D grid, KV group fastest: workgroups are dealt round-robin to the 8 XCDs, so
    // with Hkv = 8 each XCD scores one group and keeps that group's landmarks in its
    // L2; tiles in descending order, the longest candidate lists first
    const int ntiles = (a.N + kSQ - 1) / kSQ;
    const int g = blockIdx.x % a.Hkv, rest = blockIdx.x / a.Hkv;
    const int tile = ntiles - 1 - rest % ntiles, b = rest / ntiles;
    const int q0 = tile * kSQ;
    const int qlast = min(q0 + kSQ - 1, a.N - 1);
    const int nct = n_candidates(qlast, a.W);
    const int nC = a.L / kChunk;
    const int qw0 = q0 + kSR * w;
    const bf16* qr = as<bf16>(a.q_route ? a.q_route : a.q);
    const bf16* lmk = as<bf16>(a.lmk);
    if (lane < kSR) s_nb[kSR * w + lane] = 0;  // a wave's rows are its own: no barrier needed

    if constexpr (NORM) {
        // the per-(row, head) log-sum-exps that k_pf_lse left in the lse output
        for (int e = tid; e < G * kSQ; e += kSW * kWave) {
            const int hh = e / kSQ, row = e % kSQ, n = min(q0 + row, a.N - 1);
            s_lse[hh][row] = a.lse[((size_t)b * a.Hq + g * G + hh) * a.N + n];
        }
        __syncthreads();
    }
    for (int s0 = 0; s0 < nct; s0 += kSL) {
        const int len = min(kSL, nct - s0);
        const int ncb = (len + 15) / 16;
        // Wave w scores chunk blocks cb = w + kSW j (j < NJ) against all kSQ rows of the
        // tile (4 row tiles), so each landmark operand it loads feeds 4 MFMAs; all of a
        // head's landmark loads are issued before its MFMAs.
        f32x4 sig[NT][NJ];
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int j = 0; j < NJ; ++j) sig[t][j] = f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
#pragma unroll 1
        for (int hh = 0; hh < G; ++hh) {
            const int h = g * G + hh, hl = (a.Hl == a.Hq) ? h : g;
            const bf16* lbase = lmk + ((size_t)b * a.Hl + hl) * nC * D;
            // the tile's query operands once per head, then the landmark blocks one
            // at a time, each feeding the NT row tiles
            bf16x8 aq[NT][KS];
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const int qa = min(q0 + 16 * t + lane % 16, a.N - 1);
#pragma unroll
                for (int ks = 0; ks < KS; ++ks)
                    aq[t][ks] = ld_bf16x8(qr + (((size_t)b * a.Hq + h) * a.N + qa) * D + ks * 32 + (lane / 16) * 8);
            }
            float sub[NT][4];
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int i = 0; i < 4; ++i) sub[t][i] = NORM ? s_lse[hh][16 * t + (lane / 16) * 4 + i] : 0.f;
#pragma unroll
            for (int j = 0; j < NJ; ++j) {
                const int c = min(s0 + (w + kSW * j) * 16 + lane % 16, nC - 1);
                bf16x8 bl[KS];
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) bl[ks] = ld_bf16x8(lbase + (size_t)c * D + ks * 32 + (lane / 16) * 8);
                const float bv = a.bias ? a.bias[((size_t)b * a.Hl + hl) * nC + c] : 0.f;
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    f32x4 acc4 = zero4();
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) acc4 = mfma16x16x32(aq[t][ks], bl[ks], acc4);
#pragma unroll
                    for (int i = 0; i < 4; ++i) sig[t][j][i] = fmaxf(sig[t][j][i], a.scale * acc4[i] + bv - sub[t][i]);
                }
            }
        }
        __syncthreads();  // the previous slice's rows are selected
        // all rows x this wave's chunk blocks -> LDS (row = 16t + (l/16)*4 + i, column = 16cb + l%16)
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int j = 0; j < NJ; ++j)
                if (w + kSW * j < ncb)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        s_sig[16 * t + (lane / 16) * 4 + i][(w + kSW * j) * 16 + lane % 16] = sig[t][j][i];
        __syncthreads();
#pragma unroll 1
        for (int r = 0; r < kSR; ++r) {
            const int n = qw0 + r, row = kSR * w + r;
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
                sc[e] = ok[e] ? s_sig[row][col] : 0.f;
                id[e] = s0 + col;
            }
            const int nb = s_nb[row];
            ok[E] = lane < nb;
            sc[E] = ok[E] ? s_bsc[row * K + lane] : 0.f;
            id[E] = ok[E] ? s_bid[row * K + lane] : -1;
            // ids ascend over (register E: the running best, all below s0; then
            // registers 0.. : s0 + e*64 + lane); the selection rewrites the row's list
            const int m = wave_topk_reg<E + 1, E>(sc, id, ok, K, s_bid + row * K, s_bsc + row * K, s_tid[w], s_tsc[w]);
            if (lane == 0) s_nb[row] = m;
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        }
    }
#pragma unroll 1
    for (int r = 0; r < kSR; ++r) {
        const int n = qw0 + r, row = kSR * w + r;
        if (n >= a.N) break;
        const int nb = s_nb[row];
        int32_t* orow = a.idx + (((size_t)b * a.Hkv + g) * a.N + n) * K;
        if (lane < K) orow[lane] = lane < nb ? s_bid[row * K + lane] : -1;
    }
}

// ---------------------------------------------------------------------------
// P0 (per-head normalised ranking only): the log-sum-exp over the candidate chunks
// of every (row, query head), LSE_h(i) = log sum_{c in C_i} exp(s^_hc) (Sec. 4.1),
// which the ranking subtracts before the group max.  One block of 8 waves per
// (128 rows, query head): wave w holds the q^ rows of its 16 queries as A operands,
// the candidates' landmark rows come through LDS 64 at a time (double-buffered:
// the next block is fetched into registers while the current one is used), and
// every lane keeps a running (max, sum of exp) for its 4 rows over the candidate
// columns it holds, merged over the 16 lanes of its group at the end.  The result
// goes to the prefill's lse output, which the fusion overwrites at the end of the
// call.
constexpr int kLseRows = 128;
constexpr int kLseCand = 64;
template <int D>
__global__ __launch_bounds__(8 * kWave) void k_pf_lse(FwdArgs a) {
    constexpr int KS = D / 32, NT = 8 * kWave;
    constexpr int PPT = kLseCand * D / 8 / NT;  // 16-byte pieces per thread of a landmark block
    static_assert(PPT >= 1 && PPT * NT == kLseCand * D / 8, "landmark blocks split evenly over the threads");
    __shared__ __align__(16) bf16 s_l[2][st_size<D>(kLseCand)];
    __shared__ float s_b[2][kLseCand];
    const int tid = threadIdx.x, w = wave_id(), lane = tid % kWave, lg = lane / 16;
    const int q0 = blockIdx.x * kLseRows, h = blockIdx.y, b = blockIdx.z;
    const int G = a.Hq / a.Hkv, hl = (a.Hl == a.Hq) ? h : h / G;
    const int nC = a.L / kChunk;
    const int qlast = min(q0 + kLseRows - 1, a.N - 1);
    const int nct = min(nC, n_candidates(qlast, a.W));
    const bf16* qr = as<bf16>(a.q_route ? a.q_route : a.q);
    const bf16* lbase = as<bf16>(a.lmk) + ((size_t)b * a.Hl + hl) * nC * D;
    const float* bbase = a.bias ? a.bias + ((size_t)b * a.Hl + hl) * nC : nullptr;
    // the wave's 16 q^ rows as A operands (row l%16, dims 32 ks + 8 (l/16) ...)
    bf16x8 aq[KS];
    {
        const int qa = min(q0 + 16 * w + lane % 16, a.N - 1);
        const bf16* qrow = qr + (((size_t)b * a.Hq + h) * a.N + qa) * D;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) aq[ks] = ld_bf16x8(qrow + ks * 32 + lg * 8);
    }
    struct LRegs {
        uint4 x[PPT];
        float bv;
    };
    auto fetch = [&](int c0) {
        LRegs r;
#pragma unroll
        for (int u = 0; u < PPT; ++u) {
            const int e = tid + u * NT, j = e / (D / 8), d8 = (e % (D / 8)) * 8;
            const int c = min(c0 + j, nC - 1);
            r.x[u] = *reinterpret_cast<const uint4*>(lbase + (size_t)c * D + d8);
        }
        r.bv = (bbase && tid < kLseCand) ? bbase[min(c0 + tid, nC - 1)] : 0.f;
        return r;
    };
    auto store = [&](int buf, const LRegs& r) {
#pragma unroll
        for (int u = 0; u < PPT; ++u) {
            const int e = tid + u * NT, j = e / (D / 8), d8 = (e % (D / 8)) * 8;
            *reinterpret_cast<uint4*>(&s_l[buf][st_off<D>(j, d8)]) = r.x[u];
        }
        if (tid < kLseCand) s_b[buf][tid] = r.bv;
    };
    // running (max, sum of exp) of rows q0 + 16 w + 4 lg + i over this lane's columns
    float rm[4], rs[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        rm[i] = -INFINITY;
        rs[i] = 0.f;
    }
    const int nblk = (nct + kLseCand - 1) / kLseCand;
    if (nblk > 0) {
        LRegs nx = fetch(0);
        store(0, nx);
        __syncthreads();
        for (int blk = 0; blk < nblk; ++blk) {
            const int buf = blk & 1;
            const bool more = blk + 1 < nblk;  // uniform over the block
            if (more) nx = fetch((blk + 1) * kLseCand);
            float x[4][4];
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) {
                f32x4 acc = zero4();
#pragma unroll
                for (int ks = 0; ks < KS; ++ks)
                    acc = mfma16x16x32(aq[ks], row_operand_st<D>(s_l[buf], nb * 16, ks * 32, lane), acc);
                const int j = nb * 16 + lane % 16, c = blk * kLseCand + j;
                const float bv = s_b[buf][j];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int n = q0 + 16 * w + 4 * lg + i;
                    x[nb][i] = (n < a.N && c < n_candidates(n, a.W)) ? a.scale * acc[i] + bv : -INFINITY;
                }
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float mx = fmaxf(fmaxf(x[0][i], x[1][i]), fmaxf(x[2][i], x[3][i]));
                if (mx == -INFINITY) continue;
                const float nm = fmaxf(rm[i], mx);
                float sum = rs[i] * fexp(rm[i] - nm);
#pragma unroll
                for (int nb = 0; nb < 4; ++nb) sum += fexp(x[nb][i] - nm);
                rm[i] = nm;
                rs[i] = sum;
            }
            if (more) store(buf ^ 1, nx);
            __syncthreads();
        }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        lse16_merge(rm[i], rs[i]);
        const int n = q0 + 16 * w + 4 * lg + i;
        if (lane % 16 == 0 && n < a.N)
            a.lse[((size_t)b * a.Hq + h) * a.N + n] = rm[i] == -INFINITY ? -INFINITY : rm[i] + __logf(rs[i]);
    }
}

// ---------------------------------------------------------------------------
// P1 split in two (up to 1024 candidate chunks): the group scores
// sigma_ic = max_h s^_hc (App. C) of every (row, KV group, candidate), then the
// top-K of each row from them.  k_pf_sigma takes 128 rows of one KV group per
// block of 8 waves: each wave holds the q^ rows of its 16 queries for the G heads
// as MFMA A operands, the candidates' landmark rows come through LDS 64 at a time
// (one tile per landmark head, double-buffered) and serve all 8 waves, and the
// max over the heads stays in registers until a block of 64 candidates is done
// and written out.  With 128 rows behind every landmark load the scoring runs at
// about three times the rate of the fused 32-row scorer, whose selection is then
// the only part left to it; k_pf_select ranks each row in one wave
// (wave_topk_reg over E registers of 64 candidates, ties to the smaller id, the
// same selection as the fused scorer makes).  sigma [B, Hkv, N, L/S] f32 lives in
// the records' area of the workspace, which the chunk pass fills only after the
// selection.  NORM (per-head normalised ranking): each head's scores less the
// (row, head) log-sum-exp that k_pf_lse left in lse, before the max over heads.
template <int D, int G, bool NORM>
__global__ __launch_bounds__(8 * kWave) void k_pf_sigma(FwdArgs a, float* sig) {
    constexpr int KS = D / 32, NT = 8 * kWave;
    constexpr int PPT = kLseCand * D / 8 / NT;  // 16-byte pieces per thread of a landmark block
    static_assert(PPT >= 1 && PPT * NT == kLseCand * D / 8, "landmark blocks split evenly over the threads");
    __shared__ __align__(16) bf16 s_l[2][st_size<D>(kLseCand)];
    __shared__ float s_b[2][kLseCand];
    const int tid = threadIdx.x, w = wave_id(), lane = tid % kWave, lg = lane / 16;
    const int q0 = blockIdx.x * kLseRows, g = blockIdx.y, b = blockIdx.z;
    const int nC = a.L / kChunk;
    const int qlast = min(q0 + kLseRows - 1, a.N - 1);
    const int nct = min(nC, n_candidates(qlast, a.W));
    const bool shared_lmk = a.Hl != a.Hq;  // one landmark head per KV group
    const int NH = shared_lmk ? 1 : G;     // landmark tiles per block of candidates
    const size_t bg = (size_t)b * a.Hkv + g;
    const bf16* qr = as<bf16>(a.q_route ? a.q_route : a.q);
    // the wave's 16 q^ rows of each head (row l%16, dims 32 ks + 8 (l/16) ...)
    bf16x8 aq[G][KS];
    {
        const int qa = min(q0 + 16 * w + lane % 16, a.N - 1);
#pragma unroll
        for (int hh = 0; hh < G; ++hh)
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                aq[hh][ks] = ld_bf16x8(qr + (((size_t)b * a.Hq + g * G + hh) * a.N + qa) * D + ks * 32 + lg * 8);
    }
    // NORM: the log-sum-exps of rows 16 w + 4 lg + i (k_pf_lse left them in lse)
    float sub[NORM ? G : 1][4];
#pragma unroll
    for (int hh = 0; hh < (NORM ? G : 1); ++hh)
#pragma unroll
        for (int i = 0; i < 4; ++i)
            sub[hh][i] = NORM ? a.lse[((size_t)b * a.Hq + g * G + hh) * a.N + min(q0 + 16 * w + 4 * lg + i, a.N - 1)]
                              : 0.f;
    struct LRegs {
        uint4 x[PPT];
        float bv;
    };
    // step t: candidate block t / NH, landmark head t % NH
    auto fetch = [&](int t) {
        const int hl = shared_lmk ? g : g * G + t % NH;
        const size_t lrow0 = ((size_t)b * a.Hl + hl) * nC;
        const int c0 = (t / NH) * kLseCand;
        LRegs r;
#pragma unroll
        for (int u = 0; u < PPT; ++u) {
            const int e = tid + u * NT, j = e / (D / 8), d8 = (e % (D / 8)) * 8;
            r.x[u] = *reinterpret_cast<const uint4*>(as<bf16>(a.lmk) + (lrow0 + min(c0 + j, nC - 1)) * D + d8);
        }
        r.bv = (a.bias && tid < kLseCand) ? a.bias[lrow0 + min(c0 + tid, nC - 1)] : 0.f;
        return r;
    };
    auto store = [&](int buf, const LRegs& r) {
#pragma unroll
        for (int u = 0; u < PPT; ++u) {
            const int e = tid + u * NT, j = e / (D / 8), d8 = (e % (D / 8)) * 8;
            *reinterpret_cast<uint4*>(&s_l[buf][st_off<D>(j, d8)]) = r.x[u];
        }
        if (tid < kLseCand) s_b[buf][tid] = r.bv;
    };
    const int nsteps = (nct + kLseCand - 1) / kLseCand * NH;
    if (nsteps == 0) return;  // uniform over the block: no row of the tile has candidates
    LRegs nx = fetch(0);
    store(0, nx);
    __syncthreads();
    f32x4 sg[4];  // sigma of rows 16 w + 4 lg + i, candidates 16 nb + l%16 of the block
    for (int t = 0; t < nsteps; ++t) {
        const int buf = t & 1, lh = t % NH;
        const bool more = t + 1 < nsteps;  // uniform over the block
        if (more) nx = fetch(t + 1);
        if (lh == 0)
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) sg[nb] = f32x4{-INFINITY, -INFINITY, -INFINITY, -INFINITY};
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
            if (!shared_lmk && hh != lh) continue;  // this tile is head lh's landmark rows
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) {
                f32x4 acc = zero4();
#pragma unroll
                for (int ks = 0; ks < KS; ++ks)
                    acc = mfma16x16x32(aq[hh][ks], row_operand_st<D>(s_l[buf], nb * 16, ks * 32, lane), acc);
                const float bv = s_b[buf][nb * 16 + lane % 16];
#pragma unroll
                for (int i = 0; i < 4; ++i) sg[nb][i] = fmaxf(sg[nb][i], a.scale * acc[i] + bv - sub[NORM ? hh : 0][i]);
            }
        }
        if (lh == NH - 1) {
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) {
                const int c = (t / NH) * kLseCand + nb * 16 + lane % 16;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int n = q0 + 16 * w + 4 * lg + i;
                    if (n < a.N && c < nC) sig[(bg * a.N + n) * nC + c] = sg[nb][i];
                }
            }
        }
        if (more) store(buf ^ 1, nx);
        __syncthreads();
    }
}

// One wave per (row, KV group): the K best of sigma over the row's candidates
// C_i (E registers of 64 candidates per lane, ids ascending over (register, lane)).
constexpr int kSelWaves = 4;
template <int E>
__global__ __launch_bounds__(kSelWaves * kWave) void k_pf_select(FwdArgs a, const float* sig) {
    __shared__ int s_tid[kSelWaves][kWave];
    __shared__ float s_tsc[kSelWaves][kWave];
    __shared__ int s_oid[kSelWaves][kWave];
    __shared__ float s_osc[kSelWaves][kWave];
    const int w = wave_id(), lane = threadIdx.x % kWave;
    const size_t r = (size_t)blockIdx.x * kSelWaves + w;  // (b, g, n) row
    if (r >= (size_t)a.B * a.Hkv * a.N) return;           // whole wave
    const int n = (int)(r % a.N);
    const int nC = a.L / kChunk, lim = min(nC, n_candidates(n, a.W));
    const float* row = sig + r * nC;
    float sc[E];
    int id[E];
    bool ok[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int c = e * kWave + lane;
        ok[e] = c < lim;
        sc[e] = ok[e] ? row[c] : 0.f;
        id[e] = c;
    }
    const int m = wave_topk_reg<E, kTopkNatural>(sc, id, ok, a.K, s_oid[w], s_osc[w], s_tid[w], s_tsc[w]);
    int32_t* orow = a.idx + r * a.K;
    if (lane < a.K) orow[lane] = lane < m ? s_oid[w][lane] : -1;
}

// ---------------------------------------------------------------------------
// P3: retrieved chunks, chunk-major
// ---------------------------------------------------------------------------
// One block per work item: up to kInvSeg entries of one (b, g, chunk) list that
// lie in one bucket of rows (2048, more for long sequences: see kInvBucketRows).
// The items of a (b, g) come bucket by bucket, so the query rows that the blocks
// in flight gather (2048 rows x G heads, 2 MiB at d = 128) stay in the L2s.
// Units of work are (16 entries, head) pairs; wave w takes units w, w + 4, ...,
// and the next unit's rows are fetched while the current one computes.  K and V
// of the chunk, and the landmark rows of the group's heads, stay in LDS and every
// unit reads its MFMA operands from there, so that a wave holds only one unit's
// state and the prefetched operands of the next: four waves per SIMD keep the
// gathers of many units in flight (the kernel waits on memory, not on the matrix
// cores).  K rows are padded by 8 elements, V rows by 16: on gfx950 both the
// 16-byte row reads and the transposing reads of these tiles meet two addresses
// per bank (the bank-conflict counters put that at about a third of the LDS
// cycles), but LDS waits are about 1 % of the wave cycles here, so the simpler
// padded layouts stay.
template <int D, int G, bool ROUTE>
__global__ __launch_bounds__(kBlock, ROUTE ? 2 : 4) void k_pf_chunks(FwdArgs a, const int* boff, int nR,
                                                                    const int* list, const int4* work,
                                                                    size_t max_work_bg, const int* nwork,
                                                                    bf16* part, float* wgt, int n0, int Ns) {
    constexpr int KS = Tiles<D>::KS, DB = Tiles<D>::DB;
    constexpr int KROW = Tiles<D>::KROW, VROW = D + 16;
    __shared__ __align__(16) bf16 s_k[kChunk * KROW];
    __shared__ __align__(16) bf16 s_v[kChunk * VROW];
    __shared__ __align__(16) bf16 s_l[G][D];
    __shared__ float s_bias[G];
    __shared__ int s_ent[kInvSeg];  // the segment's entries (row << 6 | slot)
    const int tid = threadIdx.x, w = wave_id(), lane = tid % kWave, lg = lane / 16;
    const int nC = a.L / kChunk;
    // logical blocks of (b, g) = bg are bg * max_work_bg + item, those past its item
    // count leave; each XCD takes one contiguous range of logical blocks (one (b, g)
    // and range of row buckets), so its L2 holds only the query rows of its buckets
    const int lb = xcd_remap((int)blockIdx.x, (int)gridDim.x);
    const size_t bg = (size_t)lb / max_work_bg;
    const int item = (int)((size_t)lb % max_work_bg);
    if (item >= nwork[bg]) return;
    const int4 wi = work[lb];
    const int c = wi.y;
    const int b = (int)(bg / a.Hkv), g = (int)(bg % a.Hkv);
    const int* bo = boff + bg * ((size_t)nC * nR + 1);
    const int jb = c * nR + wi.x;
    const int beg = bo[jb] + wi.z * kInvSeg;
    const int len = min(kInvSeg, bo[jb + 1] - beg);
    if (len <= 0) return;
    const int* seg = list + bg * (size_t)Ns * a.K + beg;
    static_assert(kInvSeg <= kBlock, "one entry per thread");
    if (tid < len) s_ent[tid] = seg[tid];
    {
        const KVRegs<D> kr = load_block<D>(as<bf16>(a.k) + (bg * a.L + (size_t)c * kChunk) * D);
        const KVRegs<D> vr = load_block<D>(as<bf16>(a.v) + (bg * a.L + (size_t)c * kChunk) * D);
        if (tid < G * D / 8) {
            const int hh = tid / (D / 8), d8 = (tid % (D / 8)) * 8;
            const int hl = (a.Hl == a.Hq) ? g * G + hh : g;
            const size_t lrow = ((size_t)b * a.Hl + hl) * nC + c;
            *reinterpret_cast<uint4*>(&s_l[hh][d8]) =
                *reinterpret_cast<const uint4*>(as<bf16>(a.lmk) + lrow * D + d8);
            if (d8 == 0) s_bias[hh] = a.bias ? a.bias[lrow] : 0.f;
        }
#pragma unroll
        for (int u = 0; u < Tiles<D>::PPT; ++u) {
            const int e = tid + u * kBlock, j = e / (D / 8), d8 = (e % (D / 8)) * 8;
            *reinterpret_cast<uint4*>(s_k + j * KROW + d8) = kr.x[u];
            *reinterpret_cast<uint4*>(s_v + j * VROW + d8) = vr.x[u];
        }
    }
    __syncthreads();
    const float c1 = a.scale * kLog2e;
    const bf16* qbase = as<bf16>(a.q);
    const bf16* rbase = as<bf16>(a.q_route);
    const int nunits = ((len + 15) / 16) * G;

    struct Ops {
        uint4 q[KS], qr[ROUTE ? KS : 1];
        int ent;
    };
    // branch-free loads: an entry past the end reads the last entry's row
    auto load_ops = [&](int u, Ops& x) {
        const int grp = u / G, hh = u % G;
        const int e = min(grp * 16 + lane % 16, len - 1);
        const int ent = s_ent[e];
        x.ent = (u < nunits && grp * 16 + lane % 16 < len) ? ent : -1;
        const size_t qrow = ((size_t)b * a.Hq + g * G + hh) * a.N + n0 + (ent >> 6);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            x.q[ks] = *reinterpret_cast<const uint4*>(qbase + qrow * D + ks * 32 + lg * 8);
            if constexpr (ROUTE) x.qr[ks] = *reinterpret_cast<const uint4*>(rbase + qrow * D + ks * 32 + lg * 8);
        }
    };
    // a wave's units are u = w, w + 4, ...; the operands of the next two are in flight
    auto unit = [&](int u, const Ops& cur, Ops& nxt) {
        load_ops(u + 8, nxt);
        const int hh = u % G;
        const bool qv = cur.ent >= 0;
        const int n = cur.ent >> 6, slot = cur.ent & 63;
        // surrogate score s^ = q^ . k'_c: the landmark row is row 0 of the A tile
        f32x4 sh4 = zero4();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const bf16x8 lrow = ld_bf16x8(&s_l[hh][ks * 32 + lg * 8]);
            const bf16x8 aL = (lane % 16 == 0) ? lrow : as_bf16x8(make_uint4(0, 0, 0, 0));
            if constexpr (ROUTE)
                sh4 = mfma16x16x32(aL, as_bf16x8(cur.qr[ks]), sh4);
            else
                sh4 = mfma16x16x32(aL, as_bf16x8(cur.q[ks]), sh4);
        }
        const float shat = a.scale * group0_bcast(sh4[0]) + s_bias[hh];
        // S^T = K_c Q^T and the intra-chunk softmax p_j = exp(s_j - lse_c)
        // (scheduling barriers keep the operand reads of one key block, or of two
        // dim blocks below, live at a time: that is what fits four waves per SIMD)
        f32x4 st[4];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
            st[kb] = zero4();
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                st[kb] = mfma16x16x32(k_operand<D>(s_k, kb, ks, lane), as_bf16x8(cur.q[ks]), st[kb]);
            __builtin_amdgcn_sched_barrier(0);
        }
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) mx = fmaxf(mx, fmaxf(fmaxf(st[kb][0], st[kb][1]), fmaxf(st[kb][2], st[kb][3])));
        mx = group4_max(mx);
        const float m2 = mx * c1;
        // unnormalised exp in (0, 1] as the P operand; 1/sum is applied to O^T
        float sum = 0.f;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                st[kb][i] = fexp2(fmaf(st[kb][i], c1, -m2));
                sum += st[kb][i];
            }
        const bf16x8 pb0 = p_operand(st[0], st[1]);
        const bf16x8 pb1 = p_operand(st[2], st[3]);
        sum = group4_sum(sum);
        const float inv = 1.f / sum;
        f32x4 o[DB];
#pragma unroll
        for (int db = 0; db < DB; ++db) {
            o[db] = mfma16x16x32(tr_operand_perm(s_v, VROW, 0, db * 16, lane), pb0, zero4());
            o[db] = mfma16x16x32(tr_operand_perm(s_v, VROW, 32, db * 16, lane), pb1, o[db]);
            if (db % 2 == 1) __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int i = 0; i < 4; ++i) o[db][i] *= inv;
        if (qv) {
            store_lane_order<D>(part + part_offset(bg, Ns, n, a.K, slot, G, hh, D), o, lg);
            if (lane < 16) wgt[part_offset(bg, Ns, n, a.K, slot, G, hh, 1)] = shat;
        }
    };
    Ops opa, opb, opc;
    load_ops(w, opa);
    load_ops(w + 4, opb);
    for (int u = w; u < nunits; u += 12) {
        unit(u, opa, opc);
        if (u + 4 >= nunits) break;
        unit(u + 4, opb, opa);
        if (u + 8 >= nunits) break;
        unit(u + 8, opc, opb);
    }
}

// ---------------------------------------------------------------------------
// P2: local window (flash style) + fusion epilogue
// ---------------------------------------------------------------------------
// One block of 8 waves per tile of QT = 16 * 8 / G queries of one KV group:
// wave w owns the item (head w / QB, 16-query block w % QB), i.e. 16 rows of
// one head (under UNION: queries 16/G w .. 16/G (w + 1) - 1, all G heads).  The 64-key blocks of K and V that the tile's windows cover are
// double-buffered in LDS: block j + 1 is fetched into registers while block j
// is used and stored into the other buffer afterwards, one barrier per block.
// After the window, the row's retrieved-chunk slots are added into the same
// accumulators (fusion, Eq. (10)), stabilised per (row, head) by
// M = max(log Z_swa, max_k s^_k):
//   out = (e^{log Z_swa - M} o_swa + sum_k e^{s^_k - M} o_k) / (e^{log Z_swa - M} + sum_k e^{s^_k - M}).
template <int G>
struct LocalCfg {
    static constexpr int QB = 8 / G;   // 16-query blocks per tile
    static constexpr int QT = 16 * QB;
    static constexpr int NT = 8 * kWave;
};

// UNION (the paper's one-load-multiple-compute, Sec. 4.2, on MFMA): instead of
// reading per-slot partials, the tile loads the union of its rows' selected
// chunks once each (ascending, double-buffered like the window) and computes
// every chunk for all of its rows; a row that did not select the chunk gets
// weight 0, and a wave none of whose rows selected it skips the chunk's MFMAs.
// With adjacent queries that retrieve overlapping chunks the union is small and
// no partials go through HBM.  The union is built in LDS from the rows' idx: a
// bitmap over the chunks, then the set bits in order (dynamic LDS: the bitmap,
// the rows' valid entries, the union list).
template <int D, int G, bool UNION, bool ROUTE>
__global__ __launch_bounds__(LocalCfg<G>::NT, 2) void k_pf_local(FwdArgs a, const bf16* part, const float* wgt, int n0,
                                                                 int Ns) {
    using C = LocalCfg<G>;
    constexpr int KS = Tiles<D>::KS, DB = Tiles<D>::DB;
    constexpr int KROW = Tiles<D>::KROW, VROW = D + 16;
    constexpr int PPT = kChunk * D / 8 / C::NT;  // 16-byte pieces per thread of a K or V block
    static_assert(C::QT == 128 / G, "part_offset tiles the partials by the local pass's query tile");
    static_assert(PPT >= 1 && kChunk * D / 8 == PPT * C::NT, "K/V blocks split evenly over the threads");
    __shared__ __align__(16) bf16 s_k[2][kChunk * KROW];
    __shared__ __align__(16) bf16 s_v[2][kChunk * VROW];
    const int tid = threadIdx.x, w = wave_id(), lane = tid % kWave, lg = lane / 16;
    // the tiles of rows n0 .. n0 + Ns - 1 (the partials are indexed from n0)
    const int ntiles = (Ns + C::QT - 1) / C::QT;
    const int tile = xcd_remap(blockIdx.x, ntiles), g = blockIdx.y, b = blockIdx.z;
    const int q0 = n0 + tile * C::QT;
    const int qlast = min(q0 + C::QT - 1, a.N - 1);
    const int kbeg = n_candidates(q0, a.W) * kChunk;
    const int kfull = n_candidates(qlast, a.W) * kChunk;  // keys >= kfull are in every row's window...
    const size_t bg = (size_t)b * a.Hkv + g;
    const bf16* kbase = as<bf16>(a.k) + bg * a.L * D;
    const bf16* vbase = as<bf16>(a.v) + bg * a.L * D;
    const float c1 = a.scale * kLog2e;
    // row of the tile and query head of this lane's MFMA column: 16 queries of
    // one head per wave, or under UNION the paper's packing (Sec. 4.2) of 16 / G
    // queries x the G heads, so that a wave's chunks are the union of only 16 / G
    // queries' selections (the heads share the selection)
    const int hh = UNION ? (lane % 16) % G : w / C::QB;
    const int trow = UNION ? w * (16 / G) + (lane % 16) / G : (w % C::QB) * 16 + lane % 16;
    const int nq_raw = q0 + trow;
    const int nq = min(nq_raw, a.N - 1);
    const size_t row = ((size_t)b * a.Hq + g * G + hh) * a.N + nq;

    // union of the tile's selections (UNION only)
    extern __shared__ int s_dyn[];
    __shared__ int s_nu;
    __shared__ __align__(16) bf16 s_lm[UNION ? 2 : 1][UNION ? G * D : 8];  // the chunk's landmark rows
    __shared__ float s_lb[UNION ? 2 : 1][UNION ? G : 1];                  // and biases
    const int nC = a.L / kChunk, nwords = (nC + 31) / 32;
    int* s_bits = s_dyn;
    int* s_idx = s_bits + nwords;              // [QT][K] the rows' valid entries, then INT_MAX
    int* s_list = s_idx + C::QT * a.K;         // the union, ascending
    if constexpr (UNION) {
        for (int i = tid; i < nwords; i += C::NT) s_bits[i] = 0;
        __syncthreads();
        for (int e = tid; e < C::QT * a.K; e += C::NT) {
            const int r = e / a.K, n = q0 + r;
            int v = INT_MAX;
            if (n < a.N) {
                const int raw = a.idx[(bg * a.N + n) * a.K + e % a.K];
                if (raw >= 0 && raw < n_candidates(n, a.W)) v = raw;
            }
            s_idx[e] = v;
            if (v != INT_MAX) atomicOr(reinterpret_cast<unsigned*>(&s_bits[v >> 5]), 1u << (v & 31));
        }
        __syncthreads();
        if (w == 0) {
            int base = 0;
            for (int w0 = 0; w0 < nwords; w0 += kWave) {
                unsigned word = w0 + lane < nwords ? (unsigned)s_bits[w0 + lane] : 0u;
                const int cnt = __popc(word);
                int incl = cnt;
#pragma unroll
                for (int o2 = 1; o2 < kWave; o2 <<= 1) {
                    const int y = __shfl_up(incl, o2, kWave);
                    if (lane >= o2) incl += y;
                }
                int pos = base + incl - cnt;
                while (word) {
                    s_list[pos++] = (w0 + lane) * 32 + __ffs(word) - 1;
                    word &= word - 1u;
                }
                base += __shfl(incl, kWave - 1, kWave);
            }
            if (lane == 0) s_nu = base;
        }
        // (the barrier before the window's first block orders these writes)
    }

    struct KV {
        uint4 k[PPT], v[PPT];
    };
    auto fetch = [&](int j0) {
        KV x;
#pragma unroll
        for (int u = 0; u < PPT; ++u) {
            const int e = tid + u * C::NT, j = e / (D / 8), d8 = (e % (D / 8)) * 8;
            x.k[u] = *reinterpret_cast<const uint4*>(kbase + (size_t)(j0 + j) * D + d8);
            x.v[u] = *reinterpret_cast<const uint4*>(vbase + (size_t)(j0 + j) * D + d8);
        }
        return x;
    };
    auto stage = [&](int buf, const KV& x) {
#pragma unroll
        for (int u = 0; u < PPT; ++u) {
            const int e = tid + u * C::NT, j = e / (D / 8), d8 = (e % (D / 8)) * 8;
            *reinterpret_cast<uint4*>(&s_k[buf][j * KROW + d8]) = x.k[u];
            *reinterpret_cast<uint4*>(&s_v[buf][j * VROW + d8]) = x.v[u];
        }
    };

    bf16x8 bq[KS];
    {
        const bf16* qrow = as<bf16>(a.q) + row * D;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) bq[ks] = ld_bf16x8(qrow + ks * 32 + lg * 8);
    }
    f32x4 o[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db] = zero4();
    float m = -INFINITY, l = 0.f;  // running max (log2 units) and sum
    const int ell = n_candidates(nq, a.W) * kChunk;

    KV nx = fetch(kbeg);
    stage(0, nx);
    __syncthreads();
    int buf = 0;
    for (int j0 = kbeg; j0 <= qlast; j0 += kChunk, buf ^= 1) {
        const bool more = j0 + kChunk <= qlast;  // uniform over the block
        if (more) nx = fetch(j0 + kChunk);
        const bf16* tk = s_k[buf];
        const bf16* tv = s_v[buf];
        // S^T for the wave's 16 rows (scheduling barriers keep one key block's
        // operands live at a time)
        f32x4 st[4];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
            st[kb] = zero4();
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                st[kb] = mfma16x16x32(ld_bf16x8(tk + (kb * 16 + lane % 16) * KROW + ks * 32 + lg * 8), bq[ks], st[kb]);
            __builtin_amdgcn_sched_barrier(0);
        }
        // ...and below every row of the tile: such blocks need no mask
        const bool full = j0 >= kfull && j0 + kChunk - 1 <= q0;
        float mx = -INFINITY;
        if (full) {
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    st[kb][i] *= c1;
                    mx = fmaxf(mx, st[kb][i]);
                }
        } else {
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int j = j0 + kb * 16 + lg * 4 + i;
                    const bool valid = nq_raw < a.N && j <= nq && j >= ell;
                    st[kb][i] = valid ? st[kb][i] * c1 : -INFINITY;
                    mx = fmaxf(mx, st[kb][i]);
                }
        }
        mx = group4_max(mx);
        const float mnew = fmaxf(m, mx);
        const float muse = mnew == -INFINITY ? 0.f : mnew;
        const float alpha = fexp2(m - muse);
        float psum = 0.f;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                st[kb][i] = fexp2(st[kb][i] - muse);
                psum += st[kb][i];
            }
        const bf16x8 pb0 = p_operand(st[0], st[1]);
        const bf16x8 pb1 = p_operand(st[2], st[3]);
        psum = group4_sum(psum);
        l = l * alpha + psum;
        m = mnew;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
            o[db] *= alpha;
            o[db] = mfma16x16x32(tr_operand_perm(tv, VROW, 0, db * 16, lane), pb0, o[db]);
            o[db] = mfma16x16x32(tr_operand_perm(tv, VROW, 32, db * 16, lane), pb1, o[db]);
            if (db % 2 == 1) __builtin_amdgcn_sched_barrier(0);
        }
        if (more) stage(buf ^ 1, nx);
        __syncthreads();
    }

    // fusion epilogue (lane: row l%16 of the item, dims 16 db + 4 lg + i)
    const float lam0 = (m + __log2f(l)) * (1.f / kLog2e);  // local log-sum-exp (l >= 1: key nq is in the window)
    // M: the (row, head)'s stabiliser, zs: the fusion denominator relative to e^M;
    // o holds the numerator relative to e^M
    float M = lam0, zs = 1.f;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db] *= 1.f / l;
    if constexpr (UNION) {
        // the union's chunks, each for all rows of the tile
        const int U = s_nu;
        bf16x8 bqr[ROUTE ? KS : 1];
        if constexpr (ROUTE) {
            const bf16* rrow = as<bf16>(a.q_route) + row * D;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) bqr[ks] = ld_bf16x8(rrow + ks * 32 + lg * 8);
        }
        const int* myidx = s_idx + trow * a.K;
        int ptr = 0;
        // Four union chunks in flight: chunk u is computed from LDS buffer u % 2 while
        // chunks u + 1 .. u + 3 wait in a ring of registers (named slots, the loop
        // unrolled four times, so that no register copy waits on a pending load) and
        // chunk u + 4 is fetched into the slot chunk u + 1 leaves when it is staged.
        // The chunk's G landmark rows and biases travel with its K/V (threads <
        // G * D / 8).  Past the union's end the fetches re-read the last chunk (in
        // bounds, never staged), so the loads are the same in every iteration.
        const bool lm_thread = tid < G * D / 8;
        const int lm_h = tid / (D / 8), lm_d8 = (tid % (D / 8)) * 8;
        const int lm_hl = (a.Hl == a.Hq) ? g * G + min(lm_h, G - 1) : g;
        const bf16* lm_base = as<bf16>(a.lmk) + ((size_t)b * a.Hl + lm_hl) * nC * D + lm_d8;
        struct Slot {
            KV kv;
            uint4 lm;
            float lb;
        };
        auto fetch_slot = [&](int u) {
            Slot x;
            const int cc = U > 0 ? s_list[min(u, U - 1)] : 0;
            x.kv = fetch(cc * kChunk);
            x.lm = lm_thread ? *reinterpret_cast<const uint4*>(lm_base + (size_t)cc * D) : make_uint4(0, 0, 0, 0);
            x.lb = (lm_thread && lm_d8 == 0 && a.bias) ? a.bias[((size_t)b * a.Hl + lm_hl) * nC + cc] : 0.f;
            return x;
        };
        auto stage_slot = [&](int bb, const Slot& x) {
            stage(bb, x.kv);
            if (lm_thread) {
                *reinterpret_cast<uint4*>(&s_lm[bb][lm_h * D + lm_d8]) = x.lm;
                if (lm_d8 == 0) s_lb[bb][lm_h] = x.lb;
            }
        };
        // chunk u from buffer u % 2: s^, the intra-chunk softmax and O^T for the rows
        // that selected it, folded into the row's online fusion
        auto compute = [&](int u) {
            const int bb = u & 1;
            const int c = s_list[u];
            const bool sel = nq_raw < a.N && myidx[min(ptr, a.K - 1)] == c && ptr < a.K;
            ptr += sel ? 1 : 0;
            if (__ballot(sel) == 0ull) return;
            const bf16* tk = s_k[bb];
            const bf16* tv = s_v[bb];
            // s^ of the rows for chunk c: the G heads' landmark rows are rows 0..G-1
            // of the A tile, so column p's own head hh sits in accumulator row hh,
            // held by lane group hh / 4 as element hh % 4
            f32x4 sh4 = zero4();
            const int ar = min(lane % 16, G - 1);
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const bf16x8 lrow = ld_bf16x8(&s_lm[bb][ar * D + ks * 32 + lg * 8]);
                const bf16x8 aL = (lane % 16 < G) ? lrow : as_bf16x8(make_uint4(0, 0, 0, 0));
                sh4 = mfma16x16x32(aL, ROUTE ? bqr[ks] : bq[ks], sh4);
            }
            const int hi = hh & 3;
            const float shv = hi == 0 ? sh4[0] : hi == 1 ? sh4[1] : hi == 2 ? sh4[2] : sh4[3];
            float shr;
            if constexpr (G <= 4)
                shr = group0_bcast(shv);
            else
                shr = __shfl(shv, (hh >> 2) * 16 + lane % 16, kWave);
            const float shat = a.scale * shr + s_lb[bb][hh];
            f32x4 st[4];
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) {
                st[kb] = zero4();
#pragma unroll
                for (int ks = 0; ks < KS; ++ks)
                    st[kb] = mfma16x16x32(ld_bf16x8(tk + (kb * 16 + lane % 16) * KROW + ks * 32 + lg * 8), bq[ks],
                                          st[kb]);
                __builtin_amdgcn_sched_barrier(0);
            }
            float mx = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) mx = fmaxf(mx, st[kb][i]);
            mx = group4_max(mx) * c1;
            float psum = 0.f;
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    st[kb][i] = fexp2(fmaf(st[kb][i], c1, -mx));
                    psum += st[kb][i];
                }
            const bf16x8 pb0 = p_operand(st[0], st[1]);
            const bf16x8 pb1 = p_operand(st[2], st[3]);
            psum = group4_sum(psum);
            // online fusion: a selected chunk whose s^ exceeds the row's M so far
            // rescales the numerator and denominator to the new maximum
            const float Mn = sel ? fmaxf(M, shat) : M;
            const float rs = fexp(M - Mn);
            zs *= rs;
            M = Mn;
            const float wk = sel ? fexp(shat - M) : 0.f;
            zs += wk;
            const float f = wk / psum;
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                f32x4 oc = mfma16x16x32(tr_operand_perm(tv, VROW, 0, db * 16, lane), pb0, zero4());
                oc = mfma16x16x32(tr_operand_perm(tv, VROW, 32, db * 16, lane), pb1, oc);
                o[db] = o[db] * rs + f * oc;
                if (db % 2 == 1) __builtin_amdgcn_sched_barrier(0);
            }
        };
        // one step: fetch chunk u + 4 into `ld`, compute chunk u, stage chunk u + 1
        // (held in `st`) into the other buffer
        auto step = [&](int u, Slot& st, Slot& ld) {
            ld = fetch_slot(u + 4);
            compute(u);
            if (u + 1 < U) stage_slot((u + 1) & 1, st);
            __syncthreads();
        };
        Slot r0, r1, r2, r3;
        if (U > 0) {
            stage_slot(0, fetch_slot(0));
            r1 = fetch_slot(1);
            r2 = fetch_slot(2);
            r3 = fetch_slot(3);
        }
        __syncthreads();
        for (int u = 0; u < U; u += 4) {
            step(u, r1, r0);
            if (u + 1 >= U) break;
            step(u + 1, r2, r1);
            if (u + 2 >= U) break;
            step(u + 2, r3, r2);
            if (u + 3 >= U) break;
            step(u + 3, r0, r3);
        }
    } else {
    // the row's retrieved chunks: slots in idx order, valid entries only
    constexpr int SB = D >= 128 ? 2 : 4;  // slots whose loads are in flight together
    const int32_t* irow = a.idx + (bg * a.N + nq) * a.K;
    const int ncand = n_candidates(nq, a.W);
    // online fusion over the slots: each group of SB slots may raise the
    // (row, head)'s maximum M, which rescales the numerator and denominator
    int prev = -1;
    for (int k0 = 0; k0 < a.K; k0 += SB) {
        float sv[SB];
        bool okk[SB];
        uint4 pv[SB][D / 32];
#pragma unroll
        for (int u = 0; u < SB; ++u) {
            const int k = min(k0 + u, a.K - 1);
            const int cc = irow[k];
            const bool ok = k0 + u < a.K && cc >= 0 && cc < ncand && cc > prev;
            prev = cc;  // idx_entry_valid compares with the previous entry as written
            sv[u] = wgt[part_offset(bg, Ns, nq - n0, a.K, k, G, hh, 1)];
            okk[u] = ok;
            // (address independent of idx, so these loads issue with the idx loads;
            // an invalid slot's bits are masked by fma_lane_order)
            load_lane_order<D>(part + part_offset(bg, Ns, nq - n0, a.K, k, G, hh, D), lg, pv[u]);
        }
        float Mn = M;
#pragma unroll
        for (int u = 0; u < SB; ++u) Mn = okk[u] ? fmaxf(Mn, sv[u]) : Mn;
        const float rs = fexp(M - Mn);
#pragma unroll
        for (int db = 0; db < DB; ++db) o[db] *= rs;
        zs *= rs;
        M = Mn;
#pragma unroll
        for (int u = 0; u < SB; ++u) {
            const float wk = okk[u] ? fexp(sv[u] - M) : 0.f;
            zs += wk;
            fma_lane_order<D>(pv[u], wk, okk[u], o);
        }
    }
    }
    const float Z = zs;
    const float inv = 1.f / Z;
    if (nq_raw < a.N) {
        bf16* out = as_mut<bf16>(a.out);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
            const int d0 = db * 16 + lg * 4;
            const f32x4 r = o[db] * inv;
            *reinterpret_cast<uint2*>(out + row * D + d0) = make_uint2(pack_bf16x2(r[0], r[1]), pack_bf16x2(r[2], r[3]));
        }
        if (lane < 16) a.lse[row] = M + __logf(Z);
    }
}

// Rows of one segment of the chunk-major pass.  The per-slot records of a row
// take B Hq K (2 d + 4) bytes (133 KB per row at 32 query heads, K = 16, d = 128):
// with many rows the inverse index, chunk pass and local pass run once per
// segment of rows over one workspace, so that the records stay under the cap
// (hils_prefill_record_cap, 16 GiB by default) whatever the sequence length (the
// paper's 512K-token prefill would otherwise need 69 GB).  Segments are multiples
// of kPfSegAlign rows (whole query tiles of the local pass).  Each row's terms are
// computed the same way in any segment, so the results do not depend on the cap;
// a segment costs its own inverse index and launch tails (a 32K prefill split in
// 4 segments: 3.47 -> 3.76 ms), so the default cap keeps the 32K and training
// shapes in one.
std::atomic<size_t> g_record_cap{size_t(16) << 30};
constexpr int kPfSegAlign = 2048;
int pf_segment_rows(int B, int Hq, int N, int d, int K) {
    const size_t cap = g_record_cap.load(std::memory_order_relaxed);
    const size_t per_row = (size_t)B * Hq * K * (2 * (size_t)d + 4);
    if ((size_t)N * per_row <= cap) return N;
    const size_t rows = cap / per_row / kPfSegAlign * kPfSegAlign;
    return (int)std::min((size_t)N, std::max((size_t)kPfSegAlign, rows));
}

struct PfRun {
    template <typename T, int D, int G>
    static hipError_t run(const FwdArgs& a, hipStream_t s) {
        const int seg = pf_segment_rows(a.B, a.Hq, a.N, D, a.K);
        const PfLayout ly = pf_layout(a.B, a.Hq, a.Hkv, seg, a.L, D, a.K, seg < a.N ? a.N : -1);
        char* ws = static_cast<char*>(a.ws);
        bf16* part = reinterpret_cast<bf16*>(ws + ly.part);
        float* wgt = reinterpret_cast<float*>(ws + ly.wgt);
        if (!a.given_idx) {
            const dim3 grid((unsigned)((a.N + kSQ - 1) / kSQ) * a.Hkv * a.B);
            const size_t dyn = score_dyn_lds(a.K);
            if (a.head_norm) {
                const dim3 lgr((unsigned)((a.N + kLseRows - 1) / kLseRows), a.Hq, a.B);
                HILS_LAUNCH("k_pf_lse", k_pf_lse<D>, lgr, dim3(8 * kWave), 0, s, a);
            }
            const int nC = a.L / kChunk;
            if (nC <= 16 * kWave && !a.union_pack &&
                (size_t)a.B * a.Hkv * a.N * nC * sizeof(float) <= ly.wgt - ly.part) {
                // the split scorer: sigma in the records' area (see k_pf_sigma)
                float* sigma = reinterpret_cast<float*>(ws + ly.part);
                const dim3 sgr((unsigned)((a.N + kLseRows - 1) / kLseRows), a.Hkv, a.B);
                if (a.head_norm)
                    HILS_LAUNCH("k_pf_sigma", (k_pf_sigma<D, G, true>), sgr, dim3(8 * kWave), 0, s, a, sigma);
                else
                    HILS_LAUNCH("k_pf_sigma", (k_pf_sigma<D, G, false>), sgr, dim3(8 * kWave), 0, s, a, sigma);
                const size_t rows = (size_t)a.B * a.Hkv * a.N;
                const dim3 rgr((unsigned)((rows + kSelWaves - 1) / kSelWaves));
                const dim3 rbl(kSelWaves * kWave);
                if (nC <= kWave)
                    HILS_LAUNCH("k_pf_select", k_pf_select<1>, rgr, rbl, 0, s, a, (const float*)sigma);
                else if (nC <= 2 * kWave)
                    HILS_LAUNCH("k_pf_select", k_pf_select<2>, rgr, rbl, 0, s, a, (const float*)sigma);
                else if (nC <= 4 * kWave)
                    HILS_LAUNCH("k_pf_select", k_pf_select<4>, rgr, rbl, 0, s, a, (const float*)sigma);
                else if (nC <= 8 * kWave)
                    HILS_LAUNCH("k_pf_select", k_pf_select<8>, rgr, rbl, 0, s, a, (const float*)sigma);
                else
                    HILS_LAUNCH("k_pf_select", k_pf_select<16>, rgr, rbl, 0, s, a, (const float*)sigma);
            } else if (a.head_norm) {
                HILS_LAUNCH("k_pf_score", (k_pf_score<D, G, true>), grid, dim3(kSW * kWave), dyn, s, a);
            } else {
                HILS_LAUNCH("k_pf_score", (k_pf_score<D, G, false>), grid, dim3(kSW * kWave), dyn, s, a);
            }
        }
        const dim3 lgrid((a.N + LocalCfg<G>::QT - 1) / LocalCfg<G>::QT, a.Hkv, a.B);
        if (a.union_pack) {
            // one-load-multiple-compute: no inverse index, no per-slot partials
            const int nC = a.L / kChunk;
            const int qk = LocalCfg<G>::QT * a.K;
            const size_t dyn = (size_t)((nC + 31) / 32 + qk + min(nC, qk)) * sizeof(int);
            if (a.q_route)
                HILS_LAUNCH("k_pf_union", (k_pf_local<D, G, true, true>), lgrid, dim3(LocalCfg<G>::NT), dyn, s, a,
                            (const bf16*)nullptr, (const float*)nullptr, 0, a.N);
            else
                HILS_LAUNCH("k_pf_union", (k_pf_local<D, G, true, false>), lgrid, dim3(LocalCfg<G>::NT), dyn, s, a,
                            (const bf16*)nullptr, (const float*)nullptr, 0, a.N);
            return hipGetLastError();
        }
        const int* boff = reinterpret_cast<const int*>(ws + ly.inv.boff);
        const int* list = reinterpret_cast<const int*>(ws + ly.inv.list);
        const int4* work = reinterpret_cast<const int4*>(ws + ly.inv.work);
        const int* nwork = reinterpret_cast<const int*>(ws + ly.inv.nwork);
        const dim3 cgrid((unsigned)(ly.inv.max_work_bg * a.B * a.Hkv));
        for (int n0 = 0; n0 < a.N; n0 += seg) {
            const int Ns = std::min(seg, a.N - n0);
            const InvArgs ia{a.idx, a.B, a.Hkv, Ns, a.K, a.W, a.L, n0, a.N};
            launch_inverse_index(ia, ly.inv, a.ws, s);
            if (a.q_route)
                HILS_LAUNCH("k_pf_chunks", (k_pf_chunks<D, G, true>), cgrid, dim3(kBlock), 0, s, a, boff, ly.inv.nR,
                            list, work, ly.inv.max_work_bg, nwork, part, wgt, n0, Ns);
            else
                HILS_LAUNCH("k_pf_chunks", (k_pf_chunks<D, G, false>), cgrid, dim3(kBlock), 0, s, a, boff, ly.inv.nR,
                            list, work, ly.inv.max_work_bg, nwork, part, wgt, n0, Ns);
            const dim3 sgrid((Ns + LocalCfg<G>::QT - 1) / LocalCfg<G>::QT, a.Hkv, a.B);
            HILS_LAUNCH("k_pf_local", (k_pf_local<D, G, false, false>), sgrid, dim3(LocalCfg<G>::NT), 0, s, a,
                        (const bf16*)part, (const float*)wgt, n0, Ns);
        }
        return hipGetLastError();
    }
};

}  // namespace

size_t prefill_record_cap(size_t bytes) {
    return bytes ? g_record_cap.exchange(bytes) : g_record_cap.load();
}

size_t prefill_workspace_bytes(int B, int Hq, int Hkv, int N, int L, int d, int K, int bf16_storage,
                               int union_pack) {
    if (!bf16_storage || union_pack) return 0;  // the fp32 and union paths need no workspace
    const int seg = pf_segment_rows(B, Hq, N, d, K);
    return pf_layout(B, Hq, Hkv, seg, L, d, K, seg < N ? N : -1).total;
}

hipError_t launch_prefill_fwd(const FwdArgs& a, hipStream_t s) {
    if (!a.bf16) return launch_prefill_rows(a, s);
    return dispatch<PfRun>(1, a.d, a.Hq / a.Hkv, a, s);
}

}  // namespace hils
