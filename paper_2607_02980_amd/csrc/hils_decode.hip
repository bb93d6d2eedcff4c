// HiLS attention decode forward, gfx950.  N >= 1 new queries per sequence (N > 1:
// drafted tokens verified together, each at its own position); the work is a
// stream over HBM (landmark scan, then K/V gathers), so the kernels are
// organised for coalesced, many-in-flight loads rather than for math.
//
// Every (sequence b, new query n) is a row of its own: grids run over the
// B * N rows, and workspace records, idx, out and lse are indexed by
// rg = (b * Hkv + g) * N + n (the [B, Hkv, N, K] order of idx).  The caches are
// contiguous ([B, Hkv, L, d] K/V, [B, Hl, L/S, d] landmarks, [B, Hl, L/S] bias)
// or paged: with a page table, chunk c of sequence b is page block_table[b, c]
// of pools [P, Hkv, S, d], [P, Hl, d] and [P, Hl] (a page holds one chunk).
//
//   A  k_dec_scan     grid (nslices, Hkv, B*N): scores SLICE candidate chunks of one
//                     KV group (s^_hc for the G heads, max over heads, Eq. (9) /
//                     App. C) and keeps the slice's top-K (exact wave radix select).
//                     Small LDS, so many slices stream per CU while others select.
//   B  merge          top-K over the slices' survivors -> idx: for bf16 at the start
//                     of C, in each workgroup of a row's retrieved chunks (no launch
//                     and no round trip through idx in between); fp32: k_dec_merge,
//                     grid (Hkv, B*N)
//   C  k_dec_parts    grid (K + nlocal, Hkv, B*N)
//        x <  K     : the intra-chunk softmax of selected chunk x (Eq. (10)) and
//                     its surrogate score s^_hc
//        x >= K     : one 64-key piece of the local window [l(i), i] (Eq. (1))
//                     (bf16: on MFMA, run_part_mfma)
//   A part (chunk or piece) leaves per head its max, sum and unnormalised P.V.
//   D  k_dec_combine  grid (Hkv, B*N): local pieces merged by online softmax,
//                     then the fusion softmax over {s^_hc} U {log Z_swa} -> out, lse
// Parts (local pieces and chunks) leave a record {m, l, s^, o[d]} per head.
#include <type_traits>

#include "hils_device.hpp"
#include "hils_dispatch.hpp"
#include "hils_internal.hpp"
#include "hils_mfma.hpp"

namespace hils {

namespace {

constexpr int kBlock = 256;
constexpr int kSlice = 256;       // candidate chunks per scan workgroup
constexpr int kMaxLocalPieces = 64;  // local window pieces per row (W <= 4032)
constexpr int kRowWaves = 8;         // waves of a k_dec_row workgroup
// The one-workgroup-per-row pass is used for kRowPassMinRows..(CUs of the device)
// rows (b, g, n): with fewer it would leave CUs idle, with more its workgroups run
// in rounds that each wait out a selection and a fusion; otherwise the parts
// spread over per-part workgroups.
constexpr int kRowPassMinRows = 128;
constexpr int kMqMaxUnion = 256;  // union chunks of a multi-query workgroup (larger: per-part path)

struct DecLayout {
    int nC, nslices, nlocal, nparts;  // nparts = K + nlocal records per (b, g)
    int mq_umax;                      // union chunks per multi-query workgroup (at most)
    int hn_words;                     // 4-byte words of one (row, slice) record of hn
    size_t cand, parts, lse, mq, hn, total;  // byte offsets
};

__host__ __device__ inline int local_pieces_max(int W) { return (W + 62) / 64 + 1; }

// R = B * N rows; with N > 1 also the records of the multi-query pass
// (k_dec_mq: per workgroup mq_umax union chunks x 16 tile rows); under the per-head
// normalised ranking (HN) also, per (row, slice), the union of the G heads' top-K
// chunks of the slice by raw score: its size, ids and G raw scores each.
__host__ __device__ inline DecLayout dec_layout(int B, int N, int Hkv, int G, int d, int L, int K, int W,
                                                int HN) {
    const int R = B * N;
    DecLayout o;
    o.nC = L / kChunk;
    o.nslices = (o.nC + kSlice - 1) / kSlice;
    o.nlocal = local_pieces_max(W);
    o.nparts = K + o.nlocal;
    const size_t bg = (size_t)R * Hkv;
    o.cand = 0;
    o.parts = ((bg * o.nslices * K * 8) + 255) & ~(size_t)255;
    // per-head (max, sum of exp) of each slice's scores, for the normalised ranking
    o.lse = o.parts + ((bg * o.nparts * G * (4 + d) * 4 + 255) & ~(size_t)255);
    o.mq = o.lse + ((bg * o.nslices * G * 2 * 4 + 255) & ~(size_t)255);
    const int nq = 16 / G < 8 ? 16 / G : 8;  // queries per multi-query workgroup
    o.mq_umax = nq * K + o.nlocal + 1;
    const size_t mq_groups = N > 1 ? (size_t)B * ((N + nq - 1) / nq) * Hkv : 0;
    o.hn = o.mq + ((mq_groups * o.mq_umax * 16 * (4 + d) * 4 + 255) & ~(size_t)255);
    o.hn_words = (1 + G * K * (1 + G) + 3) & ~3;
    o.total = o.hn + (HN ? ((bg * o.nslices * o.hn_words * 4 + 255) & ~(size_t)255) : 0);
    return o;
}

// Query n of sequence b sits at len - N + n, len = seqlens[b] clamped into [N, L].
__device__ __forceinline__ int decode_position(const FwdArgs& a, int b, int n) {
    int len = a.seqlens ? a.seqlens[b] : a.L;
    len = len < a.N ? a.N : (len > a.L ? a.L : len);
    return len - a.N + n;
}

// Page of chunk c of sequence b; entries outside [0, P) are clamped (memory
// safety only: such a table has no meaning).
__device__ __forceinline__ int page_of(const FwdArgs& a, int nC, int b, int c) {
    const int p = a.block_table[(size_t)b * nC + c];
    return p < 0 ? 0 : (p >= a.num_pages ? a.num_pages - 1 : p);
}

// Element offset of the first K (or V) row of chunk c of sequence b, KV head g.
__device__ __forceinline__ size_t kv_chunk_offset(const FwdArgs& a, int nC, int b, int g, int c, int D) {
    if (a.block_table) return ((size_t)page_of(a, nC, b, c) * a.Hkv + g) * kChunk * D;
    return (((size_t)b * a.Hkv + g) * a.L + (size_t)c * kChunk) * D;
}

// Row of chunk c's landmark of head hl (times D: its element offset); the bias
// of that landmark has the same index.
__device__ __forceinline__ size_t lmk_row(const FwdArgs& a, int nC, int b, int hl, int c) {
    if (a.block_table) return (size_t)page_of(a, nC, b, c) * a.Hl + hl;
    return ((size_t)b * a.Hl + hl) * nC + c;
}

// Row of query head h, new query n of sequence b in q / out [B, Hq, N, D] and lse.
__device__ __forceinline__ size_t q_row(const FwdArgs& a, int b, int h, int n) {
    return ((size_t)b * a.Hq + h) * a.N + n;
}

// Record of one part for one head: m, l, s^, (pad), o[D] (unnormalised).
template <int D>
__device__ __forceinline__ float* part_record(const FwdArgs& a, const DecLayout& ly, size_t rg, int part, int hh,
                                              int G) {
    float* base = reinterpret_cast<float*>(static_cast<char*>(a.ws) + ly.parts);
    return base + ((rg * ly.nparts + part) * G + hh) * (4 + D);
}

// Shared memory of a part: K and V of 64 keys (raw storage rows padded by 16 B), q, P.
template <typename T, int D, int G>
struct PartSmem {
    static constexpr int kRowBytes = D * (int)sizeof(T) + 16;
    unsigned char kv[2][kChunk * kRowBytes];
    float q[G][D];
    float p[G][kChunk];
};

// NQ: new queries of one sequence scored together (one landmark read for all).
template <int G, int NQ>
struct ScanSmem {
    float score[NQ][G][kSlice];
    float sig[NQ][kSlice];
    int id[kSlice];
    int oid[NQ][64], tid[NQ][64];
    float osc[NQ][64], tsc[NQ][64];
    unsigned hb[NQ][kSlice / 32];          // per query: the union of its heads' top-K (bitmap)
    int hw_id[4][64], hw_tid[4][64];       // per wave: one head's top-K (normalised ranking)
    float hw_sc[4][64], hw_tsc[4][64];
};

// 8 consecutive elements of an fp32 LDS row.
__device__ __forceinline__ void lds_load8(const unsigned char* p, float* o, float) {
    const float4 x = *reinterpret_cast<const float4*>(p);
    const float4 y = *reinterpret_cast<const float4*>(p + 16);
    o[0] = x.x; o[1] = x.y; o[2] = x.z; o[3] = x.w; o[4] = y.x; o[5] = y.y; o[6] = y.z; o[7] = y.w;
}
// 2 consecutive elements of an fp32 LDS row.
__device__ __forceinline__ float2 lds_load2(const unsigned char* p, float) {
    return *reinterpret_cast<const float2*>(p);
}

// One 64-key part (a local-window piece or a retrieved chunk) of row (b, g):
// per head m = max_j s_j, l = sum_j exp(s_j - m), o = sum_j exp(s_j - m) v_j.
template <typename T, int D, int G>
__device__ void run_part(const FwdArgs& a, const DecLayout& ly, PartSmem<T, D, G>& sm, int b, int n, int g,
                         size_t rg, int part, int c, int nk, bool is_chunk) {
    constexpr int RB = PartSmem<T, D, G>::kRowBytes;
    constexpr int PIECES = D * (int)sizeof(T) / 16;  // 16-byte pieces per row
    const int tid = threadIdx.x, wave = wave_id(), lane = tid % kWave;
    const size_t kv_off = kv_chunk_offset(a, ly.nC, b, g, c, D);
    const unsigned char* kg = reinterpret_cast<const unsigned char*>(as<T>(a.k) + kv_off);
    const unsigned char* vg = reinterpret_cast<const unsigned char*>(as<T>(a.v) + kv_off);
    // All 64 rows lie inside the cache or page (c < L/64), so every load is in bounds;
    // rows past the query position are loaded but never read back.
    constexpr int PPT = kChunk * PIECES / kBlock;  // pieces per thread per matrix
    uint4 xk[PPT], xv[PPT];
#pragma unroll
    for (int u = 0; u < PPT; ++u) {
        const int e = tid + u * kBlock, j = e / PIECES, pc = e % PIECES;
        xk[u] = *reinterpret_cast<const uint4*>(kg + (size_t)j * D * sizeof(T) + pc * 16);
        xv[u] = *reinterpret_cast<const uint4*>(vg + (size_t)j * D * sizeof(T) + pc * 16);
    }
    // retrieved chunk: its landmark rows and the routing queries, fetched with K/V
    // (lane pairs: elements 2*lane, 2*lane+1 of head `wave + 4*u`)
    constexpr int HPW = (G + 3) / 4;  // heads per wave
    float lm2[HPW][2], qr2[HPW][2];
#pragma unroll
    for (int u = 0; u < HPW; ++u) {
        lm2[u][0] = lm2[u][1] = qr2[u][0] = qr2[u][1] = 0.f;
        const int hh = wave + 4 * u;
        if (is_chunk && hh < G && 2 * lane < D) {
            const int hl = (a.Hl == a.Hq) ? g * G + hh : g;
            const T* qr = as<T>(a.q_route ? a.q_route : a.q) + q_row(a, b, g * G + hh, n) * D + 2 * lane;
            const T* lr = as<T>(a.lmk) + lmk_row(a, ly.nC, b, hl, c) * D + 2 * lane;
            qr2[u][0] = to_f32(qr[0]);
            qr2[u][1] = to_f32(qr[1]);
            lm2[u][0] = to_f32(lr[0]);
            lm2[u][1] = to_f32(lr[1]);
        }
    }
    constexpr int QV = G * D / 8;
    float qx[8];
    const int qe = tid * 8;
    if (tid < QV) load8(as<T>(a.q) + q_row(a, b, g * G + qe / D, n) * D + qe % D, qx);
#pragma unroll
    for (int u = 0; u < PPT; ++u) {
        const int e = tid + u * kBlock, j = e / PIECES, pc = e % PIECES;
        *reinterpret_cast<uint4*>(&sm.kv[0][j * RB + pc * 16]) = xk[u];
        *reinterpret_cast<uint4*>(&sm.kv[1][j * RB + pc * 16]) = xv[u];
    }
    if (tid < QV) {
#pragma unroll
        for (int t = 0; t < 8; ++t) sm.q[(qe + t) / D][(qe + t) % D] = qx[t];
    }
    __syncthreads();
    for (int hh = wave; hh < G; hh += kBlock / kWave) {
        float s = -INFINITY;
        if (lane < nk) {
            const unsigned char* kr = &sm.kv[0][lane * RB];
            float acc = 0.f;
#pragma unroll 4
            for (int dd = 0; dd < D; dd += 8) {
                float x[8];
                lds_load8(kr + dd * sizeof(T), x, T{});
                const float4 qa = *reinterpret_cast<const float4*>(&sm.q[hh][dd]);
                const float4 qb = *reinterpret_cast<const float4*>(&sm.q[hh][dd + 4]);
                acc += qa.x * x[0] + qa.y * x[1] + qa.z * x[2] + qa.w * x[3];
                acc += qb.x * x[4] + qb.y * x[5] + qb.z * x[6] + qb.w * x[7];
            }
            s = a.scale * acc;
        }
        const float m = wave_max(s);
        const float pj = lane < nk ? fexp(s - m) : 0.f;
        const float l = wave_sum(pj);
        sm.p[hh][lane] = pj;
        float sh = -INFINITY;
        if (is_chunk) {
            const int u = (hh - wave) / 4;
            const int hl = (a.Hl == a.Hq) ? g * G + hh : g;
            const float acc = wave_sum(qr2[u][0] * lm2[u][0] + qr2[u][1] * lm2[u][1]);
            sh = a.scale * acc + (a.bias ? a.bias[lmk_row(a, ly.nC, b, hl, c)] : 0.f);
        }
        if (lane == 0) {
            float* r = part_record<D>(a, ly, rg, part, hh, G);
            r[0] = m;
            r[1] = l;
            r[2] = sh;
        }
    }
    __syncthreads();
    for (int o = tid; o < G * D / 2; o += kBlock) {
        const int hh = (2 * o) / D, dd = (2 * o) % D;
        float acc0 = 0.f, acc1 = 0.f;
        if (nk == kChunk) {  // full part: every LDS read of the loop in flight together
#pragma unroll 16
            for (int j = 0; j < kChunk; ++j) {
                const float pj = sm.p[hh][j];
                const float2 v = lds_load2(&sm.kv[1][j * RB + dd * sizeof(T)], T{});
                acc0 += pj * v.x;
                acc1 += pj * v.y;
            }
        } else {
            for (int j = 0; j < nk; ++j) {
                const float pj = sm.p[hh][j];
                const float2 v = lds_load2(&sm.kv[1][j * RB + dd * sizeof(T)], T{});
                acc0 += pj * v.x;
                acc1 += pj * v.y;
            }
        }
        float* r = part_record<D>(a, ly, rg, part, hh, G);
        r[4 + dd] = acc0;
        r[5 + dd] = acc1;
    }
}

// The same part on MFMA for bf16 storage.  Wave w owns keys [16w, 16w + 16):
// S^T = K Q^T (16 keys x the G heads as MFMA columns) from K rows and q read
// straight from HBM; after the block-wide max and sum per head, O^T = V^T P^T
// (v_mfma 16x16x16) with P^T taken from the accumulators as they are and V^T
// from the wave's 16 V rows in LDS by one transposing read per 16 dims.  The
// four waves' O^T partials are summed through LDS.
template <int D, int G>
struct PartSmemM {
    bf16 v[kChunk * (D + 8)];
    float m[4][16], l[4][16];
    float o[4][G][D];
};

template <int D, int G>
__device__ void run_part_mfma(const FwdArgs& a, const DecLayout& ly, PartSmemM<D, G>& sm, int b, int n, int g,
                              size_t rg, int part, int c, int nk, bool is_chunk) {
    constexpr int KS = D / 32, DB = D / 16, VROW = D + 8;
    typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
    const int tid = threadIdx.x, w = wave_id(), lane = tid % kWave, lg = lane / 16, n16 = lane % 16;
    const size_t kv_off = kv_chunk_offset(a, ly.nC, b, g, c, D);
    const bf16* kg = as<bf16>(a.k) + kv_off;
    const bf16* vg = as<bf16>(a.v) + kv_off;
    // A operands: K rows 16w + l%16 (rows past the query position are loaded, in
    // bounds, and masked out of the softmax); B operands: q of head l%16 (< G)
    const int key = 16 * w + n16;
    bf16x8 kA[KS], qB[KS];
    const bf16* qrow = as<bf16>(a.q) + q_row(a, b, g * G + min(n16, G - 1), n) * D;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        kA[ks] = ld_bf16x8(kg + (size_t)key * D + ks * 32 + lg * 8);
        const bf16x8 qq = ld_bf16x8(qrow + ks * 32 + lg * 8);
        qB[ks] = n16 < G ? qq : as_bf16x8(make_uint4(0, 0, 0, 0));
    }
    // the wave's 16 V rows into LDS; rows at or past nk are zeroed
    {
        constexpr int PR = D / 8;  // 16-byte pieces per row
#pragma unroll
        for (int u = 0; u < 16 * PR / kWave; ++u) {
            const int e = lane + u * kWave, r = e / PR, pc = e % PR;
            const int j = 16 * w + r;
            const uint4 x = *reinterpret_cast<const uint4*>(vg + (size_t)j * D + pc * 8);
            *reinterpret_cast<uint4*>(sm.v + j * VROW + pc * 8) = j < nk ? x : make_uint4(0, 0, 0, 0);
        }
    }
    // retrieved chunk: s^ of head wave (+4) from q^ and the landmark row (lane pairs)
    constexpr int HPW = (G + 3) / 4;
    float sh[HPW];
#pragma unroll
    for (int u = 0; u < HPW; ++u) {
        sh[u] = -INFINITY;
        const int hh = w + 4 * u;
        if (is_chunk && hh < G) {
            float acc = 0.f;
            if (2 * lane < D) {
                const int hl = (a.Hl == a.Hq) ? g * G + hh : g;
                const bf16* qr = as<bf16>(a.q_route ? a.q_route : a.q) + q_row(a, b, g * G + hh, n) * D + 2 * lane;
                const bf16* lr = as<bf16>(a.lmk) + lmk_row(a, ly.nC, b, hl, c) * D + 2 * lane;
                acc = to_f32(qr[0]) * to_f32(lr[0]) + to_f32(qr[1]) * to_f32(lr[1]);
            }
            acc = wave_sum(acc);
            sh[u] = a.scale * acc +
                    (a.bias ? a.bias[lmk_row(a, ly.nC, b, (a.Hl == a.Hq) ? g * G + hh : g, c)] : 0.f);
        }
    }
    // S^T (lane: head l%16, keys 16w + 4(l/16) + i)
    f32x4 st = zero4();
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) st = mfma16x16x32(kA[ks], qB[ks], st);
    const float c1 = a.scale * kLog2e;
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        st[i] = 16 * w + 4 * lg + i < nk ? st[i] * c1 : -INFINITY;
        mx = fmaxf(mx, st[i]);
    }
    mx = group4_max(mx);
    if (lane < 16) sm.m[w][lane] = mx;
    __syncthreads();
    const float M = fmaxf(fmaxf(sm.m[0][n16], sm.m[1][n16]), fmaxf(sm.m[2][n16], sm.m[3][n16]));  // log2 units
    float p[4], ls = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        p[i] = fexp2(st[i] - M);
        ls += p[i];
    }
    ls = group4_sum(ls);
    if (lane < 16) sm.l[w][lane] = ls;
    bf16x4 pb;
#pragma unroll
    for (int i = 0; i < 4; ++i) pb[i] = static_cast<__bf16>(p[i]);
    // O^T partial over this wave's keys (lane: head l%16, dims 16db + 4(l/16) + i)
    const int g4 = lane / 16, s16 = lane % 16;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
        const bf16* src = sm.v + (16 * w + 4 * g4 + s16 / 4) * VROW + db * 16 + 4 * (s16 % 4);
        const v4i16 va = lds_read_tr16(src);
        const f32x4 o = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(bf16x4, va), pb, zero4(), 0, 0, 0);
        if (n16 < G) *reinterpret_cast<f32x4*>(&sm.o[w][n16][db * 16 + 4 * lg]) = o;
    }
    __syncthreads();
    for (int e = tid; e < G * D; e += kBlock) {
        const int hh = e / D, dd = e % D;
        float* r = part_record<D>(a, ly, rg, part, hh, G);
        r[4 + dd] = sm.o[0][hh][dd] + sm.o[1][hh][dd] + sm.o[2][hh][dd] + sm.o[3][hh][dd];
        if (dd == 0) {
            r[0] = (fmaxf(fmaxf(sm.m[0][hh], sm.m[1][hh]), fmaxf(sm.m[2][hh], sm.m[3][hh]))) * (1.f / kLog2e);
            r[1] = sm.l[0][hh] + sm.l[1][hh] + sm.l[2][hh] + sm.l[3][hh];
        }
    }
    // s^ of the wave's heads (lane 0 of the owning wave)
#pragma unroll
    for (int u = 0; u < HPW; ++u) {
        const int hh = w + 4 * u;
        if (hh < G && lane == 0) part_record<D>(a, ly, rg, part, hh, G)[2] = sh[u];
    }
}

// ---- B: merge the slices' survivors into the final top-K --------------------
// By a workgroup of NW waves for row rg.  Per round each wave selects the top-K of
// its 64*E survivors from registers (all loads in flight together); wave 0 then
// merges the NW lists with the running best.  E (8 or 16) is chosen so that one
// round covers all the slices' survivors where it can.  The result, ascending
// chunk ids, is left in ms.bid[0, ms.nbest).
template <int NW>
struct MergeSmem {
    int wid[NW][64], tid[NW][64], bid[64];
    float wsc[NW][64], tsc[NW][64], bsc[64];
    int wn[NW], nbest;
};
// (wave: the caller's wave index within the NW waves that share ms; every wave of
// the workgroup calls merge_row the same number of times: it holds block barriers)
template <int E, int NW>
__device__ void merge_row(const FwdArgs& a, const DecLayout& ly, size_t rg, MergeSmem<NW>& ms, int wave) {
    constexpr int NT = NW * kWave;
    constexpr int E2 = NW + 1;  // NW wave lists + running best, <= 64 each
    const int lane = threadIdx.x % kWave;
    const float* cand_sc = reinterpret_cast<const float*>(static_cast<const char*>(a.ws) + ly.cand);
    const int* cand_id = reinterpret_cast<const int*>(cand_sc + (size_t)a.B * a.N * a.Hkv * ly.nslices * a.K);
    const size_t base = rg * ly.nslices * a.K;
    const int total = ly.nslices * a.K;
    int nbest = 0;
    for (int r0 = 0; r0 < total; r0 += NT * E) {
        float sc[E];
        int id[E];
        bool ok[E];
#pragma unroll
        for (int r = 0; r < E; ++r) {
            const int e = r0 + (wave * E + r) * kWave + lane;
            id[r] = e < total ? cand_id[base + e] : -1;
            sc[r] = e < total ? cand_sc[base + e] : 0.f;
        }
#pragma unroll
        for (int r = 0; r < E; ++r) ok[r] = id[r] >= 0;
        const int nw = wave_topk_reg<E>(sc, id, ok, a.K, ms.wid[wave], ms.wsc[wave], ms.tid[wave], ms.tsc[wave]);
        if (lane == 0) ms.wn[wave] = nw;
        __syncthreads();
        if (wave == 0) {
            float sc2[E2];
            int id2[E2];
            bool ok2[E2];
#pragma unroll
            for (int r = 0; r < E2; ++r) {
                const int list = r;  // lane indexes the entry inside list r
                const int cnt = list < NW ? ms.wn[list] : nbest;
                ok2[r] = lane < cnt;
                id2[r] = ok2[r] ? (list < NW ? ms.wid[list][lane] : ms.bid[lane]) : -1;
                sc2[r] = ok2[r] ? (list < NW ? ms.wsc[list][lane] : ms.bsc[lane]) : 0.f;
            }
            __builtin_amdgcn_wave_barrier();
            nbest = wave_topk_reg<E2>(sc2, id2, ok2, a.K, ms.bid, ms.bsc, ms.tid[0], ms.tsc[0]);
        }
        __syncthreads();
    }
    if (wave == 0 && lane == 0) ms.nbest = nbest;
    __syncthreads();
}

// The same merge by one wave alone, without block barriers (the rest of the
// workgroup does other work meanwhile): rounds of 64*E survivors, each round's top-K
// merged with the running best.  The result is left in ms.bid[0, ms.nbest).
template <int E>
__device__ void merge_row_wave(const FwdArgs& a, const DecLayout& ly, size_t rg, MergeSmem<1>& ms) {
    const int lane = threadIdx.x % kWave;
    const float* cand_sc = reinterpret_cast<const float*>(static_cast<const char*>(a.ws) + ly.cand);
    const int* cand_id = reinterpret_cast<const int*>(cand_sc + (size_t)a.B * a.N * a.Hkv * ly.nslices * a.K);
    const size_t base = rg * ly.nslices * a.K;
    const int total = ly.nslices * a.K;
    int nbest = 0;
    for (int r0 = 0; r0 < total; r0 += kWave * E) {
        float sc[E];
        int id[E];
        bool ok[E];
#pragma unroll
        for (int r = 0; r < E; ++r) {
            const int e = r0 + r * kWave + lane;
            id[r] = e < total ? cand_id[base + e] : -1;
            sc[r] = e < total ? cand_sc[base + e] : 0.f;
        }
#pragma unroll
        for (int r = 0; r < E; ++r) ok[r] = id[r] >= 0;
        const int nw = wave_topk_reg<E>(sc, id, ok, a.K, ms.wid[0], ms.wsc[0], ms.tid[0], ms.tsc[0]);
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        float sc2[2];
        int id2[2];
        bool ok2[2];
        ok2[0] = lane < nw;
        id2[0] = ok2[0] ? ms.wid[0][lane] : -1;
        sc2[0] = ok2[0] ? ms.wsc[0][lane] : 0.f;
        ok2[1] = lane < nbest;
        id2[1] = ok2[1] ? ms.bid[lane] : -1;
        sc2[1] = ok2[1] ? ms.bsc[lane] : 0.f;
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        nbest = wave_topk_reg<2>(sc2, id2, ok2, a.K, ms.bid, ms.bsc, ms.tid[0], ms.tsc[0]);
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    }
    if (lane == 0) ms.nbest = nbest;
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
}

// One part per wavefront (bf16): no block barriers.  S^T = K Q^T for the 64 keys
// (K rows and q straight from HBM as MFMA operands), the softmax per head over the
// four lane groups with permlane swaps, and O^T = V^T P^T with V^T from the
// wave's own LDS tile (transposing reads); the record is written by the lanes
// that hold it.  Keys at or past nk are masked.
template <int D>
struct PartWaveSmem {
    static constexpr int VROW = D + 16;  // padded rows (transposing reads meet two addresses per bank)
    bf16 v[kChunk * VROW];
};

// B operand of O^T = V^T P^T from the exponentiated S^T blocks 2t, 2t + 1.
__device__ __forceinline__ bf16x8 pack_bf16x8_4x2(const f32x4& e0, const f32x4& e1) {
    const float x[8] = {e0[0], e0[1], e0[2], e0[3], e1[0], e1[1], e1[2], e1[3]};
    return pack_bf16x8(x);
}

template <int D, int G>
__device__ void run_part_wave(const FwdArgs& a, const DecLayout& ly, bf16* sv, int b, int n, int g, size_t rg,
                              int part, int c, int nk, bool is_chunk) {
    constexpr int KS = D / 32, DB = D / 16, VROW = PartWaveSmem<D>::VROW;
    const int lane = threadIdx.x % kWave, lg = lane / 16, n16 = lane % 16;
    const size_t kv_off = kv_chunk_offset(a, ly.nC, b, g, c, D);
    const bf16* kg = as<bf16>(a.k) + kv_off;
    const bf16* vg = as<bf16>(a.v) + kv_off;
    // V rows into the wave's tile (all 64 rows lie in the cache or page; rows at or
    // past nk are zeroed so that they add nothing)
    {
        constexpr int PR = D / 8;  // 16-byte pieces per row
        uint4 x[kChunk * PR / kWave];
#pragma unroll
        for (int u = 0; u < kChunk * PR / kWave; ++u) {
            const int e = lane + u * kWave, r = e / PR, pc = e % PR;
            x[u] = *reinterpret_cast<const uint4*>(vg + (size_t)r * D + pc * 8);
        }
        bf16x8 kA[4][KS];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) kA[kb][ks] = ld_bf16x8(kg + (size_t)(kb * 16 + n16) * D + ks * 32 + lg * 8);
        bf16x8 qB[KS];
        const bf16* qrow = as<bf16>(a.q) + q_row(a, b, g * G + min(n16, G - 1), n) * D;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const bf16x8 qq = ld_bf16x8(qrow + ks * 32 + lg * 8);
            qB[ks] = n16 < G ? qq : as_bf16x8(make_uint4(0, 0, 0, 0));
        }
        // s^ of the retrieved chunk for head n16: q^ . k' over the lane's 8 dims per
        // k-step, summed over the four lane groups
        float sh = -INFINITY;
        if (is_chunk) {
            const int hh = min(n16, G - 1);
            const int hl = (a.Hl == a.Hq) ? g * G + hh : g;
            const bf16* qr = as<bf16>(a.q_route ? a.q_route : a.q) + q_row(a, b, g * G + hh, n) * D;
            const bf16* lr = as<bf16>(a.lmk) + lmk_row(a, ly.nC, b, hl, c) * D;
            float acc = 0.f;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const bf16x8 x1 = ld_bf16x8(qr + ks * 32 + lg * 8), y1 = ld_bf16x8(lr + ks * 32 + lg * 8);
#pragma unroll
                for (int t = 0; t < 8; ++t) acc += (float)x1[t] * (float)y1[t];
            }
            sh = a.scale * group4_sum(acc) + (a.bias ? a.bias[lmk_row(a, ly.nC, b, hl, c)] : 0.f);
        }
#pragma unroll
        for (int u = 0; u < kChunk * PR / kWave; ++u) {
            const int e = lane + u * kWave, r = e / PR, pc = e % PR;
            *reinterpret_cast<uint4*>(sv + r * VROW + pc * 8) = r < nk ? x[u] : make_uint4(0, 0, 0, 0);
        }
        // S^T (lane: head n16, keys 16 kb + 4 lg + i), in log2 units
        const float c1 = a.scale * kLog2e;
        f32x4 st[4];
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
            st[kb] = zero4();
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) st[kb] = mfma16x16x32(kA[kb][ks], qB[ks], st[kb]);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                st[kb][i] = kb * 16 + lg * 4 + i < nk ? st[kb][i] * c1 : -INFINITY;
                mx = fmaxf(mx, st[kb][i]);
            }
        }
        mx = group4_max(mx);
        float ls = 0.f;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                st[kb][i] = fexp2(st[kb][i] - mx);
                ls += st[kb][i];
            }
        ls = group4_sum(ls);
        const bf16x8 pb0 = pack_bf16x8_4x2(st[0], st[1]);
        const bf16x8 pb1 = pack_bf16x8_4x2(st[2], st[3]);
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        // O^T (lane: head n16, dims 16 db + 4 lg + i), unnormalised
        if (n16 < G) {
            float* r = part_record<D>(a, ly, rg, part, n16, G);
            if (lg == 0) {
                r[0] = mx * (1.f / kLog2e);
                r[1] = ls;
                r[2] = sh;
            }
        }
#pragma unroll
        for (int db = 0; db < DB; ++db) {
            f32x4 o = mfma16x16x32(tr_operand_perm(sv, VROW, 0, db * 16, lane), pb0, zero4());
            o = mfma16x16x32(tr_operand_perm(sv, VROW, 32, db * 16, lane), pb1, o);
            if (n16 < G) *reinterpret_cast<f32x4*>(part_record<D>(a, ly, rg, part, n16, G) + 4 + db * 16 + lg * 4) = o;
        }
    }
}

// bf16, few rows: four parts per block, one per wave, the fusion a pass of its own.
// E > 0: the workgroups of a row's retrieved chunks first merge the scan's
// survivors themselves (the same result in each; the first writes the row of
// idx), so that no launch and no round trip through idx separate the selection
// from the gathers; E = 0: idx given.
template <int D, int G, int E>
__global__ __launch_bounds__(kBlock) void k_dec_parts_w(FwdArgs a) {
    constexpr int NW = kBlock / kWave;
    __shared__ __align__(16) PartWaveSmem<D> sm[NW];
    __shared__ MergeSmem<NW> ms;
    const int w = wave_id();
    const int part = blockIdx.x * NW + w, g = blockIdx.y, b = blockIdx.z / a.N, n = blockIdx.z % a.N;
    const size_t rg = ((size_t)b * a.Hkv + g) * a.N + n;
    const DecLayout ly = dec_layout(a.B, a.N, a.Hkv, G, D, a.L, a.K, a.W, a.head_norm);
    const int pos = decode_position(a, b, n);
    const int lane = threadIdx.x % kWave;
    int csel = -1;  // this wave's chunk if part < K
    if constexpr (E > 0) {
        if ((int)blockIdx.x * NW < a.K) {  // uniform over the workgroup
            merge_row<E, NW>(a, ly, rg, ms, w);
            const int nb = ms.nbest;
            if (blockIdx.x == 0)
                for (int t = threadIdx.x; t < a.K; t += kBlock) a.idx[rg * a.K + t] = t < nb ? ms.bid[t] : -1;
            if (part < a.K) csel = part < nb ? ms.bid[part] : -1;
        }
    } else {
        if (part < a.K) {
            const int32_t* irow = a.idx + rg * a.K;
            csel = idx_entry_valid(irow, part, n_candidates(pos, a.W)) ? irow[part] : -1;
        }
    }
    if (part >= ly.nparts) return;  // whole wave; no block barriers below
    int c = __builtin_amdgcn_readfirstlane(csel), nk = kChunk;
    if (part >= a.K) {
        c = n_candidates(pos, a.W) + (part - a.K);
        nk = min(kChunk, pos - c * kChunk + 1);
        if (c > pos / kChunk) c = -1;
    }
    if (c < 0) {
        if (lane < G) {
            float* r = part_record<D>(a, ly, rg, part, lane, G);
            r[0] = -INFINITY;
            r[1] = 0.f;
            r[2] = -INFINITY;
        }
        return;
    }
    run_part_wave<D, G>(a, ly, sm[w].v, b, n, g, rg, part, c, nk, part < a.K);
}

template <int D>
__device__ void empty_part(const FwdArgs& a, const DecLayout& ly, size_t rg, int part, int G) {
    for (int hh = threadIdx.x; hh < G; hh += kBlock) {
        float* r = part_record<D>(a, ly, rg, part, hh, G);
        r[0] = -INFINITY;
        r[1] = 0.f;
        r[2] = -INFINITY;
    }
}

// ---- A: landmark scan slices --------------------------------------------------
// Scores of head hh of the nq query rows (b, n0 + q) for the slice's chunks
// [c0, c0 + len) into s_score[q][hh].  LPR lanes read one landmark row (16 B
// each), RPS rows per wave load; each row read is scored against all nq queries.
// Contiguous landmarks are rows c0 + r of one [L/S, D] slab; paged ones are found
// through the slice's page ids (s_page).
template <typename T, int D, int G, int NQ, bool PAGED, bool STREAM>
__device__ __forceinline__ void scan_head(const FwdArgs& a, const DecLayout& ly, int b, int n0, int nq, int g,
                                          int hh, int c0, int len, const int* s_page, float (*s_score)[G][kSlice]) {
    constexpr int LPR = D * (int)sizeof(T) / 16;
    constexpr int EPL = 16 / (int)sizeof(T);  // elements per lane per load
    constexpr int RPS = kWave / LPR;
    const int lane = threadIdx.x % kWave, sub = lane / LPR, seg = lane % LPR;
    const int hl = (a.Hl == a.Hq) ? g * G + hh : g;
    float qv[NQ][EPL];
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
        const T* qr = as<T>(a.q_route ? a.q_route : a.q) + q_row(a, b, g * G + hh, n0 + min(q, nq - 1)) * D + seg * EPL;
#pragma unroll
        for (int t = 0; t < EPL; ++t) qv[q][t] = to_f32(qr[t]);
    }
    const T* lm = as<T>(a.lmk) + seg * EPL;
    const T* base = lm + (PAGED ? 0 : lmk_row(a, ly.nC, b, hl, c0) * D);
    // NB independent 16-byte loads per lane are issued before any math; rows
    // past the slice end re-read the last row (in bounds, result discarded).
    // STREAM (the sequence's new queries all in this workgroup): the landmarks
    // are read once per step, with non-temporal loads; otherwise other query
    // groups rescan them and find them in the caches.
    constexpr int NB = NQ == 1 ? 16 : 8;
    for (int r0 = 0; r0 < len; r0 += RPS * NB) {
        uint4 x[NB];
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            const int r = min(r0 + u * RPS + sub, len - 1);
            const T* src = PAGED ? lm + ((size_t)s_page[r] * a.Hl + hl) * D : base + (size_t)r * D;
            x[u] = STREAM ? ld_stream16(src) : *reinterpret_cast<const uint4*>(src);
        }
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            float xf[EPL];
            if constexpr (sizeof(T) == 2) {
                const uint32_t w[4] = {x[u].x, x[u].y, x[u].z, x[u].w};
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    xf[2 * t] = __uint_as_float(w[t] << 16);
                    xf[2 * t + 1] = __uint_as_float(w[t] & 0xffff0000u);
                }
            } else {
                xf[0] = __uint_as_float(x[u].x);
                xf[1] = __uint_as_float(x[u].y);
                xf[2] = __uint_as_float(x[u].z);
                xf[3] = __uint_as_float(x[u].w);
            }
            const int r = r0 + u * RPS + sub;
#pragma unroll
            for (int q = 0; q < NQ; ++q) {
                float part = 0.f;
#pragma unroll
                for (int t = 0; t < EPL; ++t) part += qv[q][t] * xf[t];
                part = group_sum<LPR>(part);
                if (seg == 0 && r < len) s_score[q][hh][r] = a.scale * part;
            }
        }
    }
}

// The same with one landmark head per KV group (Hl = Hkv): the G heads share each
// landmark row, so the waves split the slice's rows instead of the heads and score
// every row they load against all G heads' queries (each row read once).
template <typename T, int D, int G, int NQ, bool PAGED, bool STREAM>
__device__ __forceinline__ void scan_shared(const FwdArgs& a, const DecLayout& ly, int b, int n0, int nq, int g,
                                            int wv, int nw, int c0, int len, const int* s_page,
                                            float (*s_score)[G][kSlice]) {
    constexpr int LPR = D * (int)sizeof(T) / 16;
    constexpr int EPL = 16 / (int)sizeof(T);
    constexpr int RPS = kWave / LPR;
    const int lane = threadIdx.x % kWave, sub = lane / LPR, seg = lane % LPR;
    float qv[G][NQ][EPL];
#pragma unroll
    for (int hh = 0; hh < G; ++hh)
#pragma unroll
        for (int q = 0; q < NQ; ++q) {
            const T* qr =
                as<T>(a.q_route ? a.q_route : a.q) + q_row(a, b, g * G + hh, n0 + min(q, nq - 1)) * D + seg * EPL;
#pragma unroll
            for (int t = 0; t < EPL; ++t) qv[hh][q][t] = to_f32(qr[t]);
        }
    const T* lm = as<T>(a.lmk) + seg * EPL;
    const T* base = lm + (PAGED ? 0 : lmk_row(a, ly.nC, b, g, c0) * D);
    constexpr int NB = 16;
    for (int r0 = wv * RPS * NB; r0 < len; r0 += nw * RPS * NB) {
        uint4 x[NB];
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            const int r = min(r0 + u * RPS + sub, len - 1);
            const T* src = PAGED ? lm + ((size_t)s_page[r] * a.Hl + g) * D : base + (size_t)r * D;
            x[u] = STREAM ? ld_stream16(src) : *reinterpret_cast<const uint4*>(src);
        }
#pragma unroll
        for (int u = 0; u < NB; ++u) {
            float xf[EPL];
            if constexpr (sizeof(T) == 2) {
                const uint32_t w[4] = {x[u].x, x[u].y, x[u].z, x[u].w};
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    xf[2 * t] = __uint_as_float(w[t] << 16);
                    xf[2 * t + 1] = __uint_as_float(w[t] & 0xffff0000u);
                }
            } else {
                xf[0] = __uint_as_float(x[u].x);
                xf[1] = __uint_as_float(x[u].y);
                xf[2] = __uint_as_float(x[u].z);
                xf[3] = __uint_as_float(x[u].w);
            }
            const int r = r0 + u * RPS + sub;
#pragma unroll
            for (int hh = 0; hh < G; ++hh)
#pragma unroll
                for (int q = 0; q < NQ; ++q) {
                    float part = 0.f;
#pragma unroll
                    for (int t = 0; t < EPL; ++t) part += qv[hh][q][t] * xf[t];
                    part = group_sum<LPR>(part);
                    if (seg == 0 && r < len) s_score[q][hh][r] = a.scale * part;
                }
        }
    }
}

// PAGED is a kernel parameter so that the contiguous scan keeps its small
// register footprint (the paged loads need a 64-bit address per row).
// mode kScanSelect: group scores and the slice's top-K.  mode kScanNormKeep (the
// per-head normalised ranking, one pass over the landmarks): each head's (max, sum
// of exp) over the slice, and the union of the G heads' top-K of the slice by raw
// score with every member's G raw scores.  The group score max_h (s^_h - LSE_h)
// needs each head's log-sum-exp over all of C_i, known only after every slice; the
// union holds every chunk that can be among the row's K best by it (if a head's own
// top-K of the slice misses c, K chunks of the slice beat c in that head, and so in
// the normalised ranking wherever that head attains c's maximum), and k_dec_hnsel
// ranks the unions once the log-sum-exps are known.
// NQ new queries of one sequence share a workgroup (grid z = B x ceil(N / NQ)):
// the landmark rows are read once for all of them; wave q selects for query q.
// Each query row keeps its own candidate count (its own position).
constexpr int kScanSelect = 0, kScanNormKeep = 1;
template <typename T, int D, int G, int NQ, bool PAGED>
__global__ __launch_bounds__(kBlock) void k_dec_scan(FwdArgs a, int mode) {
    static_assert(NQ <= kBlock / kWave, "one selecting wave per query");
    const int ngrp = (a.N + NQ - 1) / NQ;
    const int b = blockIdx.z / ngrp, n0 = (blockIdx.z % ngrp) * NQ, g = blockIdx.y;
    const int nq = min(NQ, a.N - n0);
    const DecLayout ly = dec_layout(a.B, a.N, a.Hkv, G, D, a.L, a.K, a.W, a.head_norm);
    __shared__ ScanSmem<G, NQ> ss;
    const int tid = threadIdx.x, wave = wave_id(), lane = tid % kWave;
    const int c0 = blockIdx.x * kSlice;
    float* cand_sc = reinterpret_cast<float*>(static_cast<char*>(a.ws) + ly.cand);
    int* cand_id = reinterpret_cast<int*>(cand_sc + (size_t)a.B * a.N * a.Hkv * ly.nslices * a.K);
    // per query: its row, its slice length (0 if the slice is past its candidates)
    auto row_of = [&](int q) { return ((size_t)b * a.Hkv + g) * a.N + n0 + q; };
    auto len_of = [&](int q) {
        return q < nq ? max(0, min(kSlice, n_candidates(decode_position(a, b, n0 + q), a.W) - c0)) : 0;
    };
    int len = 0;  // the longest of the queries' slices (the last query's)
#pragma unroll
    for (int q = 0; q < NQ; ++q) len = max(len, len_of(q));
    // rows whose slice is empty: empty survivors (or lse partials and an empty union) now
    for (int q = 0; q < nq; ++q) {
        if (len_of(q) > 0) continue;
        const size_t rg = row_of(q);
        if (mode == kScanNormKeep) {
            float* lp = reinterpret_cast<float*>(static_cast<char*>(a.ws) + ly.lse) + (rg * ly.nslices) * G * 2;
            for (int t = tid; t < G; t += kBlock) {
                lp[(blockIdx.x * G + t) * 2] = -INFINITY;
                lp[(blockIdx.x * G + t) * 2 + 1] = 0.f;
            }
            int* rec = reinterpret_cast<int*>(static_cast<char*>(a.ws) + ly.hn) +
                       (rg * ly.nslices + blockIdx.x) * ly.hn_words;
            if (tid == 0) rec[0] = 0;
        } else {
            const size_t cbase = (rg * ly.nslices + blockIdx.x) * a.K;
            for (int t = tid; t < a.K; t += kBlock) {
                cand_sc[cbase + t] = -INFINITY;
                cand_id[cbase + t] = -1;
            }
        }
    }
    if (len <= 0) return;
    if constexpr (PAGED) {
        // the slice's page ids (s_id is free until the selection pass)
        for (int r = tid; r < len; r += kBlock) ss.id[r] = page_of(a, ly.nC, b, c0 + r);
        __syncthreads();
    }
    const bool stream = a.N <= NQ;
    bool shared_lmk = false;  // one landmark row per KV group: read once for the G heads
    if constexpr (G > 1 && G * NQ <= 4) shared_lmk = a.Hl != a.Hq;
    if (shared_lmk) {
        if constexpr (G > 1 && G * NQ <= 4) {
            if (stream)
                scan_shared<T, D, G, NQ, PAGED, true>(a, ly, b, n0, nq, g, wave, kBlock / kWave, c0, len, ss.id,
                                                      ss.score);
            else
                scan_shared<T, D, G, NQ, PAGED, false>(a, ly, b, n0, nq, g, wave, kBlock / kWave, c0, len, ss.id,
                                                       ss.score);
        }
    } else {
        for (int hh = wave; hh < G; hh += kBlock / kWave)
            if (stream)
                scan_head<T, D, G, NQ, PAGED, true>(a, ly, b, n0, nq, g, hh, c0, len, ss.id, ss.score);
            else
                scan_head<T, D, G, NQ, PAGED, false>(a, ly, b, n0, nq, g, hh, c0, len, ss.id, ss.score);
    }
    __syncthreads();
    if (a.bias) {
        for (int e = tid; e < G * len; e += kBlock) {
            const int hh = e / len, r = e % len;
            const int hl = (a.Hl == a.Hq) ? g * G + hh : g;
            const float bv = a.bias[PAGED ? (size_t)ss.id[r] * a.Hl + hl : lmk_row(a, ly.nC, b, hl, c0 + r)];
#pragma unroll
            for (int q = 0; q < NQ; ++q) ss.score[q][hh][r] += bv;
        }
        __syncthreads();
    }
    if (mode == kScanNormKeep) {
        for (int i = tid; i < NQ * (kSlice / 32); i += kBlock) (&ss.hb[0][0])[i] = 0u;
        for (int e = wave; e < nq * G; e += kBlock / kWave) {
            const int q = e / G, hh = e % G, lq = len_of(q);
            if (lq <= 0) continue;
            float m = -INFINITY;
            for (int r = lane; r < lq; r += kWave) m = fmaxf(m, ss.score[q][hh][r]);
            m = wave_max(m);
            float sum = 0.f;
            for (int r = lane; r < lq; r += kWave) sum += fexp(ss.score[q][hh][r] - m);
            sum = wave_sum(sum);
            if (lane == 0) {
                float* lp = reinterpret_cast<float*>(static_cast<char*>(a.ws) + ly.lse) + (row_of(q) * ly.nslices) * G * 2;
                lp[(blockIdx.x * G + hh) * 2] = m;
                lp[(blockIdx.x * G + hh) * 2 + 1] = sum;
            }
        }
        __syncthreads();  // the bitmaps are clear
        // each (query, head): its top-K of the slice by raw score, into the query's bitmap
        for (int e = wave; e < nq * G; e += kBlock / kWave) {
            const int q = e / G, hh = e % G, lq = len_of(q);
            if (lq <= 0) continue;
            constexpr int E = kSlice / kWave;
            float sc[E];
            int id[E];
            bool ok[E];
#pragma unroll
            for (int r = 0; r < E; ++r) {
                const int el = r * kWave + lane;
                ok[r] = el < lq;
                sc[r] = ok[r] ? ss.score[q][hh][el] : 0.f;
                id[r] = ok[r] ? el : -1;
            }
            const int m = wave_topk_reg<E, kTopkNatural>(sc, id, ok, a.K, ss.hw_id[wave], ss.hw_sc[wave],
                                                         ss.hw_tid[wave], ss.hw_tsc[wave]);
            for (int t = lane; t < m; t += kWave) {
                const int el = ss.hw_id[wave][t];
                atomicOr(&ss.hb[q][el >> 5], 1u << (el & 31));
            }
        }
        __syncthreads();
        // the union, ascending, with the G raw scores of each member
        if (wave < nq) {
            const int q = wave;
            int* rec = reinterpret_cast<int*>(static_cast<char*>(a.ws) + ly.hn) +
                       (row_of(q) * ly.nslices + blockIdx.x) * ly.hn_words;
            int* rid = rec + 1;
            float* rsc = reinterpret_cast<float*>(rec + 1 + G * a.K);
            constexpr int NWD = kSlice / 32;
            unsigned word = lane < NWD ? ss.hb[q][lane] : 0u;
            const int cnt = __popc(word);
            int incl = cnt;
#pragma unroll
            for (int o = 1; o < NWD; o <<= 1) {
                const int y = __shfl_up(incl, o, kWave);
                if (lane >= o) incl += y;
            }
            int pos = incl - cnt;
            while (word) {
                const int el = lane * 32 + __ffs(word) - 1;
                rid[pos] = c0 + el;
#pragma unroll
                for (int hh = 0; hh < G; ++hh) rsc[pos * G + hh] = ss.score[q][hh][el];
                ++pos;
                word &= word - 1u;
            }
            const int U = __shfl(incl, NWD - 1, kWave);
            if (lane == 0) rec[0] = U;
        }
        return;
    }
    for (int e = tid; e < NQ * len; e += kBlock) {
        const int q = e / len, r = e % len;
        float m = -INFINITY;
#pragma unroll
        for (int hh = 0; hh < G; ++hh)
            m = fmaxf(m, ss.score[q][hh][r]);
        ss.sig[q][r] = m;
    }
    __syncthreads();
    if (wave < nq) {
        const int q = wave, lq = len_of(q);
        if (lq > 0) {
            constexpr int E = kSlice / kWave;
            float sc[E];
            int id[E];
            bool ok[E];
#pragma unroll
            for (int r = 0; r < E; ++r) {
                const int e = r * kWave + lane;
                ok[r] = e < lq;
                sc[r] = ok[r] ? ss.sig[q][e] : 0.f;
                id[r] = ok[r] ? c0 + e : -1;
            }
            const int m = wave_topk_reg<E, kTopkNatural>(sc, id, ok, a.K, ss.oid[q], ss.osc[q], ss.tid[q],
                                                         ss.tsc[q]);  // ids c0 + e*64 + lane
            const size_t cbase = (row_of(q) * ly.nslices + blockIdx.x) * a.K;
            for (int t = lane; t < a.K; t += kWave) {
                cand_sc[cbase + t] = t < m ? ss.osc[q][t] : -INFINITY;
                cand_id[cbase + t] = t < m ? ss.oid[q][t] : -1;
            }
        }
    }
}

// Per-head normalised ranking, after the one-pass scan: one wave per (row, slice).
// The row's per-head log-sum-exps over all of C_i from the slices' (max, sum of
// exp) partials, then the slice's union ranked by max_h (s^_h - LSE_h) and its
// top-K written as the slice's survivors, which the merge then takes as usual.
// E: registers per lane for the union (G * K <= 64 E).
template <int E>
__global__ __launch_bounds__(kBlock) void k_dec_hnsel(FwdArgs a, int G, int D) {
    __shared__ int s_oid[kBlock / kWave][64], s_tid[kBlock / kWave][64];
    __shared__ float s_osc[kBlock / kWave][64], s_tsc[kBlock / kWave][64];
    const int w = wave_id(), lane = threadIdx.x % kWave;
    const int g = blockIdx.y, b = blockIdx.z / a.N, n = blockIdx.z % a.N;
    const size_t rg = ((size_t)b * a.Hkv + g) * a.N + n;
    const DecLayout ly = dec_layout(a.B, a.N, a.Hkv, G, D, a.L, a.K, a.W, a.head_norm);
    const int sl = blockIdx.x * (kBlock / kWave) + w;
    if (sl >= ly.nslices) return;  // the whole wave; no block barriers below
    // LSE of every head: lane l takes head l % G over slices l / G, l / G + 64 / G, ...
    // (G a power of two), then the lanes of one head merge their (max, sum of exp)
    const float* lp = reinterpret_cast<const float*>(static_cast<const char*>(a.ws) + ly.lse) +
                      (rg * ly.nslices) * G * 2;
    float mx = -INFINITY, sm = 0.f;
    for (int t = lane / G; t < ly.nslices; t += kWave / G) {
        const float pm = lp[(t * G + lane % G) * 2], ps = lp[(t * G + lane % G) * 2 + 1];
        if (ps > 0.f) {
            const float nm = fmaxf(mx, pm);
            sm = sm * fexp(mx - nm) + ps * fexp(pm - nm);
            mx = nm;
        }
    }
    for (int o = G; o < kWave; o <<= 1) {
        const float om = __shfl_xor(mx, o, kWave), os = __shfl_xor(sm, o, kWave);
        const float nm = fmaxf(mx, om);
        if (nm != -INFINITY) {
            sm = (mx == -INFINITY ? 0.f : sm * fexp(mx - nm)) + (om == -INFINITY ? 0.f : os * fexp(om - nm));
            mx = nm;
        }
    }
    const float lse = mx + __logf(sm);  // lanes h < G hold head h's
    float lh[8];
#pragma unroll
    for (int h = 0; h < 8; ++h) lh[h] = __shfl(lse, h, kWave);
    const int* rec = reinterpret_cast<const int*>(static_cast<const char*>(a.ws) + ly.hn) +
                     (rg * ly.nslices + sl) * ly.hn_words;
    const int U = min(rec[0], G * a.K);
    const int* rid = rec + 1;
    const float* rsc = reinterpret_cast<const float*>(rec + 1 + G * a.K);
    float sc[E];
    int id[E];
    bool ok[E];
#pragma unroll
    for (int r = 0; r < E; ++r) {
        const int e = r * kWave + lane;
        ok[r] = e < U;
        id[r] = ok[r] ? rid[e] : -1;
        float m = -INFINITY;
#pragma unroll
        for (int h = 0; h < 8; ++h)
            if (h < G && ok[r]) m = fmaxf(m, rsc[e * G + h] - lh[h]);
        sc[r] = ok[r] ? m : 0.f;
    }
    // the union's ids ascend over (register, lane)
    const int m = wave_topk_reg<E, kTopkNatural>(sc, id, ok, a.K, s_oid[w], s_osc[w], s_tid[w], s_tsc[w]);
    float* cand_sc = reinterpret_cast<float*>(static_cast<char*>(a.ws) + ly.cand);
    int* cand_id = reinterpret_cast<int*>(cand_sc + (size_t)a.B * a.N * a.Hkv * ly.nslices * a.K);
    const size_t cbase = (rg * ly.nslices + sl) * a.K;
    for (int t = lane; t < a.K; t += kWave) {
        cand_sc[cbase + t] = t < m ? s_osc[w][t] : -INFINITY;
        cand_id[cbase + t] = t < m ? s_oid[w][t] : -1;
    }
}

// fp32 path: the merge as its own pass (one workgroup per row) before k_dec_parts.
template <int E>
__global__ __launch_bounds__(kBlock) void k_dec_merge(FwdArgs a, int G, int D) {
    __shared__ MergeSmem<kBlock / kWave> ms;
    const int b = blockIdx.y / a.N, n = blockIdx.y % a.N, g = blockIdx.x;
    const size_t rg = ((size_t)b * a.Hkv + g) * a.N + n;
    const DecLayout ly = dec_layout(a.B, a.N, a.Hkv, G, D, a.L, a.K, a.W, a.head_norm);
    merge_row<E, kBlock / kWave>(a, ly, rg, ms, wave_id());
    for (int t = threadIdx.x; t < a.K; t += kBlock) a.idx[rg * a.K + t] = t < ms.nbest ? ms.bid[t] : -1;
}

// ---- C: one selected chunk or one local-window piece per workgroup -----------
template <typename T, int D, int G>
__global__ __launch_bounds__(kBlock) void k_dec_parts(FwdArgs a) {
    constexpr bool kMfma = sizeof(T) == 2;
    typedef typename std::conditional<kMfma, PartSmemM<D, G>, PartSmem<T, D, G>>::type Smem;
    __shared__ Smem sm;
    __shared__ int s_c;
    const int slot = blockIdx.x, g = blockIdx.y, b = blockIdx.z / a.N, n = blockIdx.z % a.N;
    const size_t rg = ((size_t)b * a.Hkv + g) * a.N + n;
    const DecLayout ly = dec_layout(a.B, a.N, a.Hkv, G, D, a.L, a.K, a.W, a.head_norm);
    const int pos = decode_position(a, b, n);
    auto run = [&](int part, int c, int nk, bool is_chunk) {
        if constexpr (kMfma)
            run_part_mfma<D, G>(a, ly, sm, b, n, g, rg, part, c, nk, is_chunk);
        else
            run_part<T, D, G>(a, ly, sm, b, n, g, rg, part, c, nk, is_chunk);
    };
    if (slot >= a.K) {
        const int piece = slot - a.K;
        const int c = n_candidates(pos, a.W) + piece;
        if (c > pos / kChunk) {
            empty_part<D>(a, ly, rg, slot, G);
            return;
        }
        run(slot, c, min(kChunk, pos - c * kChunk + 1), false);
        return;
    }
    if (threadIdx.x == 0) {
        const int32_t* irow = a.idx + rg * a.K;
        s_c = idx_entry_valid(irow, slot, n_candidates(pos, a.W)) ? irow[slot] : -1;
    }
    __syncthreads();
    const int c = s_c;
    if (c < 0) {
        empty_part<D>(a, ly, rg, slot, G);
        return;
    }
    run(slot, c, kChunk, true);
}

// ---- D: fusion -----------------------------------------------------------------
// Per head: local pieces merge into (lambda0 = log Z_swa, o0); then the fusion
// weights are exp(z_t - L) over z = {lambda0} U {s^_c}, L = LSE(z), and each
// retrieved chunk contributes exp(s^_c - L) * o_c with o_c its own softmax output.
// Run by all NT threads of a workgroup once row rg's part records are written.
constexpr int kMaxParts = 64 + kMaxLocalPieces;
template <int G>
struct CombineSmem {
    float w[G][kMaxParts];  // weight of each part's unnormalised o
    float lse[G];
};
template <typename T, int D, int G, int NT>
__device__ void combine_row(const FwdArgs& a, const DecLayout& ly, CombineSmem<G>& cs, int b, int n, int g,
                            size_t rg) {
    constexpr int NW = NT / kWave;
    constexpr int OPT = (G * D + NT - 1) / NT;  // outputs per thread (o = tid + t NT < G D)
    constexpr int CH = 48;                      // parts whose values are loaded ahead of the weights
    const int tid = threadIdx.x, wave = wave_id(), lane = tid % kWave;
    // the first CH parts' values of this thread's outputs, in flight with the headers below
    float v0[OPT][CH];
#pragma unroll
    for (int t = 0; t < OPT; ++t) {
        const int o = min(tid + t * NT, G * D - 1), hh = o / D, dd = o % D;
#pragma unroll
        for (int j = 0; j < CH; ++j) v0[t][j] = part_record<D>(a, ly, rg, min(j, ly.nparts - 1), hh, G)[4 + dd];
    }
    for (int hh = wave; hh < G; hh += NW) {
        // local pieces: lanes < nlocal
        float m = -INFINITY, l = 0.f;
        if (lane < ly.nlocal) {
            const float* r = part_record<D>(a, ly, rg, a.K + lane, hh, G);
            m = r[0];
            l = r[1];
        }
        const float m0 = wave_max(m);
        const float l0 = wave_sum(l > 0.f ? l * fexp(m - m0) : 0.f);
        const float lam0 = m0 + __logf(l0);
        // chunks: lanes < K
        float z = -INFINITY, lc = 0.f;
        if (lane < a.K) {
            const float* r = part_record<D>(a, ly, rg, lane, hh, G);
            lc = r[1];
            z = lc > 0.f ? r[2] : -INFINITY;
        }
        const float M = fmaxf(wave_max(z), lam0);
        const float Z = wave_sum(lc > 0.f ? fexp(z - M) : 0.f) + fexp(lam0 - M);
        const float L = M + __logf(Z);
        const float a0 = fexp(lam0 - L) / l0;  // applied to each piece as exp(m - m0)
        if (lane < ly.nlocal) cs.w[hh][a.K + lane] = l > 0.f ? a0 * fexp(m - m0) : 0.f;
        if (lane < a.K) cs.w[hh][lane] = lc > 0.f ? fexp(z - L) / lc : 0.f;
        if (lane == 0) cs.lse[hh] = L;
    }
    __syncthreads();
#pragma unroll
    for (int t = 0; t < OPT; ++t) {
        const int o = tid + t * NT, hh = o / D, dd = o % D;
        if (o >= G * D) break;
        float acc = 0.f;
#pragma unroll
        for (int j = 0; j < CH; ++j) {
            const float w = j < ly.nparts ? cs.w[hh][j] : 0.f;
            acc += w != 0.f ? w * v0[t][j] : 0.f;
        }
        for (int pt = CH; pt < ly.nparts; ++pt) {
            const float w = cs.w[hh][pt];
            const float v = part_record<D>(a, ly, rg, pt, hh, G)[4 + dd];
            acc += w != 0.f ? w * v : 0.f;
        }
        const size_t row = q_row(a, b, g * G + hh, n);
        as_mut<T>(a.out)[row * D + dd] = from_f32<T>(acc);
        if (dd == 0) a.lse[row] = cs.lse[hh];
    }
}

// fp32 path: the fusion as its own pass, one workgroup per row.
template <typename T, int D, int G>
__global__ __launch_bounds__(kBlock) void k_dec_combine(FwdArgs a) {
    __shared__ CombineSmem<G> cs;
    const int g = blockIdx.x, b = blockIdx.y / a.N, n = blockIdx.y % a.N;
    const size_t rg = ((size_t)b * a.Hkv + g) * a.N + n;
    const DecLayout ly = dec_layout(a.B, a.N, a.Hkv, G, D, a.L, a.K, a.W, a.head_norm);
    combine_row<T, D, G, kBlock>(a, ly, cs, b, n, g, rg);
}

// The parts of row rg taken by this wave (w, w + kRowWaves, ...), each as in
// run_part_wave, with the next part's K, V and landmark rows loaded while the
// current one computes: each operand's registers are refilled as soon as the
// current part is done with them (V once staged in LDS, the landmark rows once
// s^ is formed, K once S is).  The loads are the same in every iteration (past
// the wave's last part every lane reads one 16-byte piece), so that the
// compiler counts the outstanding loads exactly.  q and q^ of the row are loaded
// once; s^ is the diagonal of the landmark rows x q^ MFMA.
struct RowPart {
    int c, nk, chunk;  // chunk (c < 0: nothing to attend), its first nk keys, retrieved or local
};
// The wave takes entries j = j0, j0 + kRowWaves, ... < nj of a list of record slots,
// slot_of(j) (slot < K: retrieved chunk slot; K + p: window piece p).
template <int D, int G, bool ROUTE, typename SlotOf>
__device__ void row_parts(const FwdArgs& a, const DecLayout& ly, bf16* sv, const int* s_sel, int b, int n, int g,
                          size_t rg, int pos, int ncand, int j0, int nj, SlotOf&& slot_of) {
    constexpr int KS = D / 32, DB = D / 16, VROW = PartWaveSmem<D>::VROW, PV = kChunk * D / 8 / kWave;
    const int lane = threadIdx.x % kWave, lg = lane / 16, n16 = lane % 16;
    const float c1 = a.scale * kLog2e;
    const bf16x8 zero8 = as_bf16x8(make_uint4(0, 0, 0, 0));
    auto part_of = [&](int part) {
        RowPart r;
        if (part >= a.K) {
            r.c = ncand + (part - a.K);
            r.nk = min(kChunk, pos - r.c * kChunk + 1);
            r.chunk = 0;
            if (r.c > pos / kChunk) r.c = -1;
        } else {
            r.c = s_sel[part];
            r.nk = kChunk;
            r.chunk = 1;
        }
        return r;
    };
    // q and q^ of the row's G heads as B operands (head l%16; zero past G)
    bf16x8 qB[KS], qR[ROUTE ? KS : 1];
    {
        const int hh = min(n16, G - 1);
        const bf16* qrow = as<bf16>(a.q) + q_row(a, b, g * G + hh, n) * D;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const bf16x8 qq = ld_bf16x8(qrow + ks * 32 + lg * 8);
            qB[ks] = n16 < G ? qq : zero8;
        }
        if constexpr (ROUTE) {
            const bf16* rrow = as<bf16>(a.q_route) + q_row(a, b, g * G + hh, n) * D;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const bf16x8 qq = ld_bf16x8(rrow + ks * 32 + lg * 8);
                qR[ks] = n16 < G ? qq : zero8;
            }
        }
    }
    const int hl = (a.Hl == a.Hq) ? g * G + min(n16, G - 1) : g;  // landmark head of lane l%16
    struct KOp {
        bf16x8 k[4][KS];
    };
    struct VOp {
        bf16x8 v[PV];
    };
    struct LOp {
        bf16x8 l[KS];
    };
    auto load_k = [&](const RowPart& p, bool real) {
        KOp x;
        const bf16* kg = as<bf16>(a.k) + kv_chunk_offset(a, ly.nC, b, g, p.c < 0 ? 0 : p.c, D);
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                x.k[kb][ks] = ld_bf16x8(kg + (real ? (size_t)(kb * 16 + n16) * D + ks * 32 + lg * 8 : 0));
        return x;
    };
    auto load_v = [&](const RowPart& p, bool real) {
        VOp x;
        const bf16* vg = as<bf16>(a.v) + kv_chunk_offset(a, ly.nC, b, g, p.c < 0 ? 0 : p.c, D);
#pragma unroll
        for (int u = 0; u < PV; ++u) {
            const int e = lane + u * kWave, r = e / (D / 8), pc = e % (D / 8);
            x.v[u] = ld_bf16x8(vg + (real ? (size_t)r * D + pc * 8 : 0));
        }
        return x;
    };
    auto load_l = [&](const RowPart& p, bool real) {
        LOp x;
        const bf16* lr = as<bf16>(a.lmk) + lmk_row(a, ly.nC, b, hl, p.c < 0 ? 0 : p.c) * D;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) x.l[ks] = ld_bf16x8(lr + (real ? ks * 32 + lg * 8 : 0));
        return x;
    };
    RowPart p = part_of(slot_of(j0));
    VOp vx = load_v(p, true);
    LOp lx = load_l(p, true);
    KOp kx = load_k(p, true);
    for (int j = j0; j < nj; j += kRowWaves) {
        const int part = slot_of(j);
        const bool real = j + kRowWaves < nj;  // uniform over the wave
        const RowPart pn = part_of(slot_of(real ? j + kRowWaves : j));
        const int nk = p.nk;
        // V rows into the wave's tile (rows at or past nk zeroed); the next V
#pragma unroll
        for (int u = 0; u < PV; ++u) {
            const int e = lane + u * kWave, r = e / (D / 8), pc = e % (D / 8);
            *reinterpret_cast<bf16x8*>(sv + r * VROW + pc * 8) = r < nk ? vx.v[u] : zero8;
        }
        vx = load_v(pn, real);
        // s^ of a retrieved chunk for head n16: the diagonal (m = n = n16) of the
        // landmark rows (A, row m = head m) x q^ (B, column n = head n), held by lane
        // group n16 / 4; the next landmark rows
        f32x4 s4 = zero4();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) s4 = mfma16x16x32(lx.l[ks], ROUTE ? qR[ks] : qB[ks], s4);
        lx = load_l(pn, real);
        float dg = s4[0];
#pragma unroll
        for (int i = 1; i < 4; ++i)
            if (n16 % 4 == i) dg = s4[i];
        const float sdiag = __shfl(dg, n16 + 16 * (n16 / 4), kWave);
        // (branch-free: without a bias the load reads the landmark cache's first word)
        const float* bsrc = a.bias ? a.bias + lmk_row(a, ly.nC, b, hl, p.c < 0 ? 0 : p.c)
                                   : reinterpret_cast<const float*>(a.lmk);
        const float bv = *bsrc;
        const float sh = p.chunk && p.c >= 0 ? a.scale * sdiag + (a.bias ? bv : 0.f) : -INFINITY;
        // S^T (lane: head n16, keys 16 kb + 4 lg + i), in log2 units; the next K
        f32x4 st[4];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
            st[kb] = zero4();
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) st[kb] = mfma16x16x32(kx.k[kb][ks], qB[ks], st[kb]);
        }
        kx = load_k(pn, real);
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                st[kb][i] = kb * 16 + lg * 4 + i < nk ? st[kb][i] * c1 : -INFINITY;
                mx = fmaxf(mx, st[kb][i]);
            }
        mx = group4_max(mx);
        float ls = 0.f;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                st[kb][i] = fexp2(st[kb][i] - mx);
                ls += st[kb][i];
            }
        ls = group4_sum(ls);
        const bf16x8 pb0 = pack_bf16x8_4x2(st[0], st[1]);
        const bf16x8 pb1 = pack_bf16x8_4x2(st[2], st[3]);
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        // the record (an empty one when there is nothing to attend: l = 0, and the
        // fusion never reads its o); O^T (lane: head n16, dims 16 db + 4 lg + i)
        const bool empty = p.c < 0;
        if (n16 < G) {
            float* r = part_record<D>(a, ly, rg, part, n16, G);
            if (lg == 0) {
                r[0] = empty ? -INFINITY : mx * (1.f / kLog2e);
                r[1] = empty ? 0.f : ls;
                r[2] = empty ? -INFINITY : sh;
            }
        }
#pragma unroll
        for (int db = 0; db < DB; ++db) {
            f32x4 o = mfma16x16x32(tr_operand_perm(sv, VROW, 0, db * 16, lane), pb0, zero4());
            o = mfma16x16x32(tr_operand_perm(sv, VROW, 32, db * 16, lane), pb1, o);
            if (n16 < G) *reinterpret_cast<f32x4*>(part_record<D>(a, ly, rg, part, n16, G) + 4 + db * 16 + lg * 4) = o;
        }
        // the tile is rewritten by the next part: its reads above must be complete
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        p = pn;
    }
}

// ---- bf16: one workgroup of kRowWaves waves per row ----------------------------
// Two phases.  In the first, the last wave selects (E > 0: the merge of the scan's
// survivors, which also writes the row of idx; E = 0: idx given) while the other
// waves each take one piece of the local window, which does not depend on the
// selection.  After a barrier, the remaining window pieces and the K retrieved
// chunks are spread over all the waves (one part at a time per wave), and after a
// second barrier the fusion combines the row's records: one launch after the scan,
// and the records only cross between waves of one workgroup, never between
// workgroups.
template <int D, int G, int E, bool ROUTE>
__global__ __launch_bounds__(kRowWaves * kWave) void k_dec_row(FwdArgs a) {
    constexpr int NT = kRowWaves * kWave;
    constexpr int kTileBytes = (int)sizeof(PartWaveSmem<D>) * kRowWaves;
    static_assert(sizeof(MergeSmem<kRowWaves>) <= (size_t)kTileBytes, "the merge scratch fits in the part tiles");
    // the waves' part tiles; the merging wave's tile holds its scratch until the
    // parts of the selection start
    constexpr int kMergeWave = kRowWaves - 1;
    constexpr int kTileElems = (int)(sizeof(PartWaveSmem<D>) / sizeof(bf16));
    static_assert(sizeof(MergeSmem<1>) <= sizeof(PartWaveSmem<D>), "the merge scratch fits in one part tile");
    __shared__ __align__(16) unsigned char s_raw[kTileBytes];
    __shared__ CombineSmem<G> cs;
    __shared__ int s_sel[64];
    bf16* tiles = reinterpret_cast<bf16*>(s_raw);
    auto& ms = *reinterpret_cast<MergeSmem<1>*>(tiles + (size_t)kMergeWave * kTileElems);
    const int g = blockIdx.x, b = blockIdx.y / a.N, n = blockIdx.y % a.N;
    const size_t rg = ((size_t)b * a.Hkv + g) * a.N + n;
    const DecLayout ly = dec_layout(a.B, a.N, a.Hkv, G, D, a.L, a.K, a.W, a.head_norm);
    const int pos = decode_position(a, b, n);
    const int ncand = n_candidates(pos, a.W);
    const int tid = threadIdx.x, w = wave_id(), lane = tid % kWave;
    bf16* mytile = tiles + (size_t)w * kTileElems;
    // phase 1: the last wave selects (merging the scan's survivors) while the others
    // take the local window's first pieces, which do not depend on the selection
    const int nlA = min(ly.nlocal, kMergeWave);  // window pieces of phase 1
    if (w == kMergeWave) {
        if constexpr (E > 0) {
            merge_row_wave<E>(a, ly, rg, ms);
            for (int t = lane; t < a.K; t += kWave) {
                const int v = t < ms.nbest ? ms.bid[t] : -1;
                s_sel[t] = v;
                a.idx[rg * a.K + t] = v;
            }
        } else {
            for (int t = lane; t < a.K; t += kWave) {
                const int32_t* irow = a.idx + rg * a.K;
                s_sel[t] = idx_entry_valid(irow, t, ncand) ? irow[t] : -1;
            }
        }
    } else if (w < nlA) {
        row_parts<D, G, ROUTE>(a, ly, mytile, s_sel, b, n, g, rg, pos, ncand, w, w + 1,
                               [&](int j) { return a.K + j; });
    }
    __syncthreads();  // s_sel is set; the merge scratch is free
    // phase 2: the rest of the window's pieces, then the retrieved chunks
    const int nwB = ly.nlocal - nlA, nB = nwB + a.K;
    if (w < nB)
        row_parts<D, G, ROUTE>(a, ly, mytile, s_sel, b, n, g, rg, pos, ncand, w, nB,
                               [&](int j) { return j < nwB ? a.K + nlA + j : j - nwB; });
    __syncthreads();  // every record of the row is written
    combine_row<bf16, D, G, NT>(a, ly, cs, b, n, g, rg);
}

// ---- bf16, several new queries per sequence: one workgroup per query group -----
// The sequence's new queries are taken NQ = min(8, 16 / G) at a time, and the
// NQ x G (query, head) rows fill the 16 rows of one MFMA tile (row r: query r / G,
// head r % G).  Each workgroup selects for its queries (merge_row, 8 / NQ waves per
// query), builds the union of their chunks in LDS (the retrieved ones and the local
// windows' chunks, each flagged per query), computes every union chunk once for all
// 16 rows -- row r keeps the whole chunk if its query retrieved it, the keys up to
// its query's position if the chunk is in that query's window, nothing otherwise --
// and then fuses each row's parts.  A chunk that several of the queries use is read
// from HBM once; drafted tokens of one sequence share their window entirely.
template <int G>
struct MqCfg {
    static constexpr int NQ = 16 / G < 8 ? 16 / G : 8;  // queries per workgroup
    static constexpr int WPQ = kRowWaves / NQ;            // merge waves per query
};

template <int D, int G, int E, bool ROUTE>
__global__ __launch_bounds__(kRowWaves * kWave) void k_dec_mq(FwdArgs a) {
    using C = MqCfg<G>;
    constexpr int NQ = C::NQ, WPQ = C::WPQ, NT = kRowWaves * kWave;
    constexpr int KS = D / 32, DB = D / 16, VROW = PartWaveSmem<D>::VROW, PV = kChunk * D / 8 / kWave;
    constexpr int kTileBytes = (int)sizeof(PartWaveSmem<D>) * kRowWaves;
    constexpr int RECF = 4 + D;  // floats per record
    static_assert(NQ * sizeof(MergeSmem<WPQ>) <= (size_t)kTileBytes, "the merge scratch fits in the part tiles");
    static_assert(16 * kMqMaxUnion * sizeof(float) <= (size_t)kTileBytes, "the fusion weights fit in the part tiles");
    // part tiles; before the parts the merges' scratch and the union bitmap, after them
    // the fusion weights, in the same bytes
    __shared__ __align__(16) unsigned char s_raw[kTileBytes];
    __shared__ int s_sel[NQ][64];
    __shared__ int s_nsel[NQ];
    __shared__ int s_u[kMqMaxUnion];       // union chunk ids, ascending
    __shared__ unsigned s_flag[kMqMaxUnion];  // bit q: in query q's window; bit 16 + q: retrieved by query q
    __shared__ int s_nu;
    __shared__ float s_lse[16];
    const int ngrp = (a.N + NQ - 1) / NQ;
    const int g = blockIdx.x, b = blockIdx.y / ngrp, n0 = (blockIdx.y % ngrp) * NQ;
    const int nq = min(NQ, a.N - n0);
    const DecLayout ly = dec_layout(a.B, a.N, a.Hkv, G, D, a.L, a.K, a.W, a.head_norm);
    const int tid = threadIdx.x, w = wave_id(), lane = tid % kWave, lg = lane / 16, n16 = lane % 16;
    auto row_of = [&](int q) { return ((size_t)b * a.Hkv + g) * a.N + n0 + q; };

    // ---- selection for each query ----
    {
        const int q = w / WPQ, qc = min(q, nq - 1);
        if constexpr (E > 0) {
            MergeSmem<WPQ>& ms = reinterpret_cast<MergeSmem<WPQ>*>(s_raw)[q];
            merge_row<E, WPQ>(a, ly, row_of(qc), ms, w % WPQ);  // every wave: the same barriers
            if (w % WPQ == 0 && q < nq) {
                for (int t = lane; t < a.K; t += kWave) {
                    const int v = t < ms.nbest ? ms.bid[t] : -1;
                    if (t < 64) s_sel[q][t] = v;
                    a.idx[row_of(q) * a.K + t] = v;
                }
                if (lane == 0) s_nsel[q] = ms.nbest;
            }
        } else {
            if (w % WPQ == 0 && q < nq) {
                // the valid entries of the given row, in order
                const int32_t* irow = a.idx + row_of(q) * a.K;
                const int ncand = n_candidates(decode_position(a, b, n0 + q), a.W);
                const bool ok = lane < a.K && idx_entry_valid(irow, lane, ncand);
                const uint64_t bal = __ballot(ok);
                if (ok) s_sel[q][popc64(bal & ((1ull << lane) - 1ull))] = irow[lane];
                if (lane == 0) s_nsel[q] = popc64(bal);
            }
        }
    }
    __syncthreads();
    // ---- the union of the queries' chunks: a bitmap over the chunks, then its set bits ----
    unsigned* bits = reinterpret_cast<unsigned*>(s_raw);
    const int nwords = (ly.nC + 31) / 32;
    for (int i = tid; i < nwords; i += NT) bits[i] = 0u;
    __syncthreads();
    for (int e = tid; e < NQ * 64; e += NT) {
        const int q = e / 64, t = e % 64;
        if (q < nq && t < s_nsel[q]) {
            const int c = s_sel[q][t];
            atomicOr(&bits[c >> 5], 1u << (c & 31));
        }
    }
    for (int e = tid; e < NQ * kMaxLocalPieces; e += NT) {
        const int q = e / kMaxLocalPieces, piece = e % kMaxLocalPieces;
        if (q >= nq || piece >= ly.nlocal) continue;
        const int pos = decode_position(a, b, n0 + q);
        const int c = n_candidates(pos, a.W) + piece;
        if (c <= pos / kChunk) atomicOr(&bits[c >> 5], 1u << (c & 31));
    }
    __syncthreads();
    if (w == 0) {
        int base = 0;
        for (int w0 = 0; w0 < nwords; w0 += kWave) {
            unsigned word = w0 + lane < nwords ? bits[w0 + lane] : 0u;
            const int cnt = __popc(word);
            int incl = cnt;
#pragma unroll
            for (int o2 = 1; o2 < kWave; o2 <<= 1) {
                const int y = __shfl_up(incl, o2, kWave);
                if (lane >= o2) incl += y;
            }
            int pos = base + incl - cnt;
            while (word) {
                if (pos < kMqMaxUnion) s_u[pos] = (w0 + lane) * 32 + __ffs(word) - 1;
                ++pos;
                word &= word - 1u;
            }
            base += __shfl(incl, kWave - 1, kWave);
        }
        if (lane == 0) s_nu = min(base, kMqMaxUnion);  // the host keeps the union within kMqMaxUnion
    }
    __syncthreads();
    const int U = s_nu;
    for (int i = tid; i < U; i += NT) {
        const int c = s_u[i];
        unsigned f = 0u;
        for (int q = 0; q < nq; ++q) {
            const int pos = decode_position(a, b, n0 + q);
            if (c >= n_candidates(pos, a.W) && c <= pos / kChunk) f |= 1u << q;
        }
        s_flag[i] = f;
    }
    __syncthreads();
    for (int e = tid; e < NQ * 64; e += NT) {
        const int q = e / 64, t = e % 64;
        if (q < nq && t < s_nsel[q]) {
            const int c = s_sel[q][t];
            int lo = 0, hi = U - 1;  // c is in the union: binary search
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (s_u[mid] < c) lo = mid + 1;
                else hi = mid;
            }
            atomicOr(&s_flag[lo], 1u << (16 + q));
        }
    }
    __syncthreads();  // the union is set; the bitmap's bytes are free for the tiles

    // ---- the parts: union chunk u by wave u % 8, for all 16 rows ----
    float* recs = reinterpret_cast<float*>(static_cast<char*>(a.ws) + ly.mq) +
                  ((size_t)(blockIdx.y * gridDim.x + blockIdx.x) * ly.mq_umax) * 16 * RECF;
    {
        const int rq = n16 / G, rh = n16 % G;             // the lane's tile row: query, head
        const bool rvalid = rq < nq;
        const int rpos = decode_position(a, b, n0 + min(rq, nq - 1));
        bf16* sv = reinterpret_cast<bf16*>(s_raw) + (size_t)w * (sizeof(PartWaveSmem<D>) / sizeof(bf16));
        const float c1 = a.scale * kLog2e;
        const bf16x8 zero8 = as_bf16x8(make_uint4(0, 0, 0, 0));
        bf16x8 qB[KS], qR[ROUTE ? KS : 1];
        {
            const size_t qrow = q_row(a, b, g * G + rh, n0 + min(rq, nq - 1));
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const bf16x8 x = ld_bf16x8(as<bf16>(a.q) + qrow * D + ks * 32 + lg * 8);
                qB[ks] = rvalid ? x : zero8;
                if constexpr (ROUTE) {
                    const bf16x8 y = ld_bf16x8(as<bf16>(a.q_route) + qrow * D + ks * 32 + lg * 8);
                    qR[ks] = rvalid ? y : zero8;
                }
            }
        }
        const int hl = (a.Hl == a.Hq) ? g * G + rh : g;  // landmark head of the lane's row
        struct KOp {
            bf16x8 k[4][KS];
        };
        struct VOp {
            bf16x8 v[PV];
        };
        struct LOp {
            bf16x8 l[KS];
        };
        auto load_k = [&](int c, bool real) {
            KOp x;
            const bf16* kg = as<bf16>(a.k) + kv_chunk_offset(a, ly.nC, b, g, c, D);
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int ks = 0; ks < KS; ++ks)
                    x.k[kb][ks] = ld_bf16x8(kg + (real ? (size_t)(kb * 16 + n16) * D + ks * 32 + lg * 8 : 0));
            return x;
        };
        auto load_v = [&](int c, bool real) {
            VOp x;
            const bf16* vg = as<bf16>(a.v) + kv_chunk_offset(a, ly.nC, b, g, c, D);
#pragma unroll
            for (int u = 0; u < PV; ++u) {
                const int e = lane + u * kWave, r = e / (D / 8), pc = e % (D / 8);
                x.v[u] = ld_bf16x8(vg + (real ? (size_t)r * D + pc * 8 : 0));
            }
            return x;
        };
        auto load_l = [&](int c, bool real) {
            LOp x;
            const bf16* lr = as<bf16>(a.lmk) + lmk_row(a, ly.nC, b, hl, c) * D;
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) x.l[ks] = ld_bf16x8(lr + (real ? ks * 32 + lg * 8 : 0));
            return x;
        };
        if (w < U) {
            int c = s_u[w];
            VOp vx = load_v(c, true);
            LOp lx = load_l(c, true);
            KOp kx = load_k(c, true);
            for (int u = w; u < U; u += kRowWaves) {
                const bool real = u + kRowWaves < U;  // uniform over the wave
                const int cn = s_u[real ? u + kRowWaves : u];
                const unsigned f = s_flag[u];
                const bool loc = rvalid && ((f >> rq) & 1u), ret = rvalid && ((f >> (16 + rq)) & 1u);
                // keys of the chunk the lane's row attends to
                const int nk = ret ? kChunk : (loc ? min(kChunk, rpos - c * kChunk + 1) : 0);
                // V rows into the wave's tile; rows no tile row attends to are zeroed
                const int nkmax = (int)wave_max((float)nk);
#pragma unroll
                for (int uu = 0; uu < PV; ++uu) {
                    const int e = lane + uu * kWave, r = e / (D / 8), pc = e % (D / 8);
                    *reinterpret_cast<bf16x8*>(sv + r * VROW + pc * 8) = r < nkmax ? vx.v[uu] : zero8;
                }
                vx = load_v(cn, real);
                // s^ of the chunk for row n16 (diagonal of landmark rows x q^)
                f32x4 s4 = zero4();
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) s4 = mfma16x16x32(lx.l[ks], ROUTE ? qR[ks] : qB[ks], s4);
                lx = load_l(cn, real);
                float dg = s4[0];
#pragma unroll
                for (int i = 1; i < 4; ++i)
                    if (n16 % 4 == i) dg = s4[i];
                const float sdiag = __shfl(dg, n16 + 16 * (n16 / 4), kWave);
                const float* bsrc = a.bias ? a.bias + lmk_row(a, ly.nC, b, hl, c) : reinterpret_cast<const float*>(a.lmk);
                const float bv = *bsrc;
                const float sh = a.scale * sdiag + (a.bias ? bv : 0.f);
                // S^T (lane: row n16, keys 16 kb + 4 lg + i), in log2 units
                f32x4 st[4];
#pragma unroll
                for (int kb = 0; kb < 4; ++kb) {
                    st[kb] = zero4();
#pragma unroll
                    for (int ks = 0; ks < KS; ++ks) st[kb] = mfma16x16x32(kx.k[kb][ks], qB[ks], st[kb]);
                }
                kx = load_k(cn, real);
                float mx = -INFINITY;
#pragma unroll
                for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        st[kb][i] = kb * 16 + lg * 4 + i < nk ? st[kb][i] * c1 : -INFINITY;
                        mx = fmaxf(mx, st[kb][i]);
                    }
                mx = group4_max(mx);
                const float muse = mx == -INFINITY ? 0.f : mx;
                float ls = 0.f;
#pragma unroll
                for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        st[kb][i] = fexp2(st[kb][i] - muse);
                        ls += st[kb][i];
                    }
                ls = group4_sum(ls);
                const bf16x8 pb0 = pack_bf16x8_4x2(st[0], st[1]);
                const bf16x8 pb1 = pack_bf16x8_4x2(st[2], st[3]);
                __builtin_amdgcn_wave_barrier();
                __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
                // the record of (u, row n16): m, l (0: the row does not use the chunk), s^, o
                // (rows that do not use the chunk write nothing; the fusion reads only
                // the records its flags name)
                float* rec = recs + ((size_t)u * 16 + n16) * RECF;
                if (lg == 0 && nk > 0) {
                    rec[0] = mx * (1.f / kLog2e);
                    rec[1] = ls;
                    rec[2] = ret ? sh : -INFINITY;
                }
#pragma unroll
                for (int db = 0; db < DB; ++db) {
                    f32x4 o = mfma16x16x32(tr_operand_perm(sv, VROW, 0, db * 16, lane), pb0, zero4());
                    o = mfma16x16x32(tr_operand_perm(sv, VROW, 32, db * 16, lane), pb1, o);
                    if (nk > 0) *reinterpret_cast<f32x4*>(rec + 4 + db * 16 + lg * 4) = o;
                }
                __builtin_amdgcn_wave_barrier();
                __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
                c = cn;
            }
        }
    }
    __syncthreads();  // every record written; the tiles' bytes now hold the fusion weights

    // ---- fusion, per tile row r (query r / G, head r % G) ----
    // wave w takes rows w and w + 8: the headers {m, l, s^} of the row's parts (lane
    // l: union entries l, l + 64, ...; at most kMqMaxUnion / 64 per lane) are read once,
    // and the row's parts with a nonzero weight are listed in LDS (entry, weight)
    constexpr int UPL = kMqMaxUnion / kWave;
    float* s_wt = reinterpret_cast<float*>(s_raw);                   // [16][kMqMaxUnion]
    int* s_wu = reinterpret_cast<int*>(s_raw) + 16 * kMqMaxUnion;    // [16][kMqMaxUnion]
    __shared__ int s_wn[16];
    static_assert(2 * 16 * kMqMaxUnion * sizeof(float) <= (size_t)kTileBytes, "the part lists fit in the tiles");
    for (int r = w; r < 16; r += kRowWaves) {
        const int q = r / G;
        if (q >= nq) continue;
        float hm[UPL], hl_[UPL], hs[UPL];
        bool isl[UPL], isr[UPL];
#pragma unroll
        for (int t = 0; t < UPL; ++t) {
            const int u = lane + t * kWave;
            const unsigned f = u < U ? s_flag[u] : 0u;
            isl[t] = (f >> q) & 1u;
            isr[t] = (f >> (16 + q)) & 1u;
            const float* rc = recs + ((size_t)min(u, U - 1) * 16 + r) * RECF;
            hm[t] = rc[0];
            hl_[t] = rc[1];
            hs[t] = rc[2];
        }
        // local pieces (window chunks of query q) by online softmax, then the chunks it retrieved
        float m0 = -INFINITY;
#pragma unroll
        for (int t = 0; t < UPL; ++t)
            if (isl[t]) m0 = fmaxf(m0, hm[t]);
        m0 = wave_max(m0);
        float l0 = 0.f, zmax = -INFINITY;
#pragma unroll
        for (int t = 0; t < UPL; ++t) {
            if (isl[t] && hl_[t] > 0.f) l0 += hl_[t] * fexp(hm[t] - m0);
            if (isr[t] && hl_[t] > 0.f) zmax = fmaxf(zmax, hs[t]);
        }
        l0 = wave_sum(l0);
        const float lam0 = m0 + __logf(l0);
        const float M = fmaxf(wave_max(zmax), lam0);
        float Z = 0.f;
#pragma unroll
        for (int t = 0; t < UPL; ++t)
            if (isr[t] && hl_[t] > 0.f) Z += fexp(hs[t] - M);
        Z = wave_sum(Z) + fexp(lam0 - M);
        const float L = M + __logf(Z);
        const float a0 = fexp(lam0 - L) / l0;
        int base = 0;
#pragma unroll
        for (int t = 0; t < UPL; ++t) {
            float wt = 0.f;
            if (isl[t] && hl_[t] > 0.f) wt = a0 * fexp(hm[t] - m0);
            else if (isr[t] && hl_[t] > 0.f) wt = fexp(hs[t] - L) / hl_[t];
            const bool nz = wt != 0.f;
            const uint64_t bal = __ballot(nz);
            if (nz) {
                const int at = base + popc64(bal & ((1ull << lane) - 1ull));
                s_wt[r * kMqMaxUnion + at] = wt;
                s_wu[r * kMqMaxUnion + at] = lane + t * kWave;
            }
            base += popc64(bal);
        }
        if (lane == 0) {
            s_lse[r] = L;
            s_wn[r] = base;
        }
    }
    __syncthreads();
    // outputs: thread t -> row t / (D/4), dims 4 (t % (D/4)) ...; the row's listed
    // parts in batches of 16 loads in flight
    constexpr int TPR = D / 4;     // threads per row
    constexpr int RPP = NT / TPR;  // rows per pass
    for (int r = tid / TPR; r < 16; r += RPP) {
        const int q = r / G, d0 = (tid % TPR) * 4;
        if (q >= nq) continue;
        const int cnt = s_wn[r];
        f32x4 acc = zero4();
        for (int j0 = 0; j0 < cnt; j0 += 16) {
            f32x4 v[16];
            float wt[16];
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int jj = min(j0 + j, cnt - 1);
                wt[j] = j0 + j < cnt ? s_wt[r * kMqMaxUnion + jj] : 0.f;
                v[j] = *reinterpret_cast<const f32x4*>(recs + ((size_t)s_wu[r * kMqMaxUnion + jj] * 16 + r) * RECF + 4 + d0);
            }
#pragma unroll
            for (int j = 0; j < 16; ++j)
                if (wt[j] != 0.f) acc += wt[j] * v[j];
        }
        const size_t orow = q_row(a, b, g * G + r % G, n0 + q);
        *reinterpret_cast<uint2*>(as_mut<bf16>(a.out) + orow * D + d0) =
            make_uint2(pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]));
        if (d0 == 0) a.lse[orow] = s_lse[r];
    }
}

struct DecRun {
    template <typename T, int D, int G>
    static hipError_t run(const FwdArgs& a, hipStream_t s) {
        const int R = a.B * a.N;  // rows (sequence, new query); the host keeps R <= 65535
        const DecLayout ly = dec_layout(a.B, a.N, a.Hkv, G, D, a.L, a.K, a.W, a.head_norm);
        if (!a.given_idx) {
            // one new query per sequence: a workgroup per (slice, group, row); several:
            // the sequence's queries four at a time share each landmark read
            auto scan = [&](int mode) {
                if (a.N == 1) {
                    const dim3 grid(ly.nslices, a.Hkv, R);
                    if (a.block_table)
                        HILS_LAUNCH("k_dec_scan", (k_dec_scan<T, D, G, 1, true>), grid, dim3(kBlock), 0, s, a, mode);
                    else
                        HILS_LAUNCH("k_dec_scan", (k_dec_scan<T, D, G, 1, false>), grid, dim3(kBlock), 0, s, a, mode);
                } else {
                    const dim3 grid(ly.nslices, a.Hkv, a.B * ((a.N + 3) / 4));
                    if (a.block_table)
                        HILS_LAUNCH("k_dec_scan", (k_dec_scan<T, D, G, 4, true>), grid, dim3(kBlock), 0, s, a, mode);
                    else
                        HILS_LAUNCH("k_dec_scan", (k_dec_scan<T, D, G, 4, false>), grid, dim3(kBlock), 0, s, a, mode);
                }
            };
            if (a.head_norm) {
                scan(kScanNormKeep);
                const dim3 hgrid((ly.nslices + kBlock / kWave - 1) / (kBlock / kWave), a.Hkv, R);
                const int gk = G * a.K;
                if (gk <= 64)
                    HILS_LAUNCH("k_dec_hnsel", (k_dec_hnsel<1>), hgrid, dim3(kBlock), 0, s, a, G, D);
                else if (gk <= 128)
                    HILS_LAUNCH("k_dec_hnsel", (k_dec_hnsel<2>), hgrid, dim3(kBlock), 0, s, a, G, D);
                else if (gk <= 256)
                    HILS_LAUNCH("k_dec_hnsel", (k_dec_hnsel<4>), hgrid, dim3(kBlock), 0, s, a, G, D);
                else
                    HILS_LAUNCH("k_dec_hnsel", (k_dec_hnsel<8>), hgrid, dim3(kBlock), 0, s, a, G, D);
            } else {
                scan(kScanSelect);
            }
        }
        if constexpr (sizeof(T) == 2) {
            const int surv = ly.nslices * a.K;  // the scan's survivors per row
            const int rows = R * a.Hkv;
            constexpr int NQ = MqCfg<G>::NQ, WPQ = MqCfg<G>::WPQ;
            if (a.N > 1 && ly.mq_umax <= kMqMaxUnion) {
                // several new queries per sequence: a workgroup per group of NQ of them
                const dim3 mgrid(a.Hkv, a.B * ((a.N + NQ - 1) / NQ)), mblock(kRowWaves * kWave);
                auto mq = [&](auto e_tag) {
                    constexpr int EE = decltype(e_tag)::value;
                    if (a.q_route)
                        HILS_LAUNCH("k_dec_mq", (k_dec_mq<D, G, EE, true>), mgrid, mblock, 0, s, a);
                    else
                        HILS_LAUNCH("k_dec_mq", (k_dec_mq<D, G, EE, false>), mgrid, mblock, 0, s, a);
                };
                if (a.given_idx)
                    mq(std::integral_constant<int, 0>{});
                else if (surv <= WPQ * kWave * 4)
                    mq(std::integral_constant<int, 4>{});
                else if (surv <= WPQ * kWave * 8)
                    mq(std::integral_constant<int, 8>{});
                else
                    mq(std::integral_constant<int, 16>{});
            } else if (rows >= kRowPassMinRows && rows <= device_cus()) {
                // a workgroup per row; one merge round covers kRowWaves * 64 * E survivors
                const dim3 rgrid(a.Hkv, R), rblock(kRowWaves * kWave);
                auto row = [&](auto e_tag) {
                    constexpr int EE = decltype(e_tag)::value;
                    if (a.q_route)
                        HILS_LAUNCH("k_dec_row", (k_dec_row<D, G, EE, true>), rgrid, rblock, 0, s, a);
                    else
                        HILS_LAUNCH("k_dec_row", (k_dec_row<D, G, EE, false>), rgrid, rblock, 0, s, a);
                };
                if (a.given_idx)
                    row(std::integral_constant<int, 0>{});
                else if (surv <= kRowWaves * kWave * 4)
                    row(std::integral_constant<int, 4>{});
                else if (surv <= kRowWaves * kWave * 8)
                    row(std::integral_constant<int, 8>{});
                else
                    row(std::integral_constant<int, 16>{});
            } else {
                // few rows: a workgroup per four parts, then the fusion
                constexpr int WPB = kBlock / kWave;
                const dim3 pgrid((ly.nparts + WPB - 1) / WPB, a.Hkv, R);
                if (a.given_idx)
                    HILS_LAUNCH("k_dec_parts", (k_dec_parts_w<D, G, 0>), pgrid, dim3(kBlock), 0, s, a);
                else if (surv <= kBlock * 8)
                    HILS_LAUNCH("k_dec_parts", (k_dec_parts_w<D, G, 8>), pgrid, dim3(kBlock), 0, s, a);
                else
                    HILS_LAUNCH("k_dec_parts", (k_dec_parts_w<D, G, 16>), pgrid, dim3(kBlock), 0, s, a);
                HILS_LAUNCH("k_dec_combine", (k_dec_combine<T, D, G>), dim3(a.Hkv, R), dim3(kBlock), 0, s, a);
            }
        } else {
            if (!a.given_idx) {
                if (ly.nslices * a.K <= kBlock * 8)
                    HILS_LAUNCH("k_dec_merge", (k_dec_merge<8>), dim3(a.Hkv, R), dim3(kBlock), 0, s, a, G, D);
                else
                    HILS_LAUNCH("k_dec_merge", (k_dec_merge<16>), dim3(a.Hkv, R), dim3(kBlock), 0, s, a, G, D);
            }
            HILS_LAUNCH("k_dec_parts", (k_dec_parts<T, D, G>), dim3(a.K + ly.nlocal, a.Hkv, R), dim3(kBlock), 0, s, a);
            HILS_LAUNCH("k_dec_combine", (k_dec_combine<T, D, G>), dim3(a.Hkv, R), dim3(kBlock), 0, s, a);
        }
        return hipGetLastError();
    }
};

}  // namespace

// Compute units of the current device (a host-side attribute query; nothing cached).
int device_cus() {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
        return 256;
    return n;
}


size_t decode_workspace_bytes(int B, int N, int Hkv, int G, int d, int L, int K, int W, int head_norm) {
    return dec_layout(B, N, Hkv, G, d, L, K, W, head_norm).total;
}

hipError_t launch_decode_fwd(const FwdArgs& a, hipStream_t s) {
    return dispatch<DecRun>(a.bf16, a.d, a.Hq / a.Hkv, a, s);
}

}  // namespace hils
