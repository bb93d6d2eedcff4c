// HiLS attention backward on MFMA (bf16 storage, fp32 accumulation), gfx950.
//
// The gradient of Eq. (10) with the selection held fixed.  With g = dO_i,
// u = g . out_i and L = the forward's fusion log-sum-exp of a (row, head):
//   local key j:    w_j = exp(s_j - L);  dv_j += w_j g;  ds_j = w_j (g.v_j - u)
//   chunk c, key j: p_j = exp(s_j - lse_c), a_c = exp(s^_c - L), u_c = sum_j p_j g.v_j,
//                   dv_j += a_c p_j g;  ds_j = a_c p_j (g.v_j - u_c);  ds^_c = a_c (u_c - u)
//   dq += scale ds_j k_j;  dk_j += scale ds_j q;  dq^ += scale ds^_c k'_c;
//   dk'_c += scale ds^_c q^;  db'_c += ds^_c
//
// Kernels (one launch each, in this order):
//   k_bwd_u        u per (row, head)
//   inverse index  the rows that retrieved each (b, g, chunk); k_inv_sort puts every
//                  list in ascending row order so that the sums below have one order
//   k_bwd_keys     one block of 8 waves per (b, g, chunk c), 64 (row, head) pairs per
//                  step: first the rows whose local window covers keys of c, then the
//                  rows that retrieved c.  Phase 1, one 16-pair tile per two waves, each
//                  against half the chunk's keys (its K and V held in registers as A
//                  operands): S^T = K Q^T and GV^T = V dO^T on MFMA, the softmax terms
//                  (for retrieving rows the two halves' max / sum meet in LDS), ds; for
//                  retrieving rows also s^_c (one more MFMA against the landmark rows)
//                  and ds^_c.  Phase 2, 16 keys x half the head dim per wave: dK and dV
//                  as MFMA reductions over the step's 64 pairs, dk' as one more
//                  (heads x pairs) product, and for retrieving rows the chunk's share
//                  of dq (K^T ds^T / scale, a bf16 partial of the row's slot), with
//                  operands read back from row-major LDS tiles by transposing reads
//                  (ds_read_b64_tr_b16).  The q / dO tiles are double-buffered: the
//                  next step's rows are fetched and staged while the current step
//                  computes.  dk, dv, dk', db' of chunk c are written once (no atomics).
//   k_bwd_dq       query-major: dq over the local window (the forward's local tile with
//                  ds in place of p), plus the row's slot partials and scale ds^ k'.
#include "hils_device.hpp"
#include "hils_dispatch.hpp"
#include "hils_internal.hpp"
#include "hils_mfma.hpp"

namespace hils {

namespace {

constexpr int kBlock = 256;
constexpr int kPairs = 64;          // (row, head) pairs per step of k_bwd_keys
constexpr int kSortWin = 8192;      // rows per bitmap pass of k_inv_sort
constexpr int kSortWords = kSortWin / 32;
static_assert(kSortWords % kBlock == 0, "k_inv_sort scans whole runs of words per thread");

struct BwLayout {
    size_t u, dqp, dsh, sorted, inv_base;
    InvLayout inv;
    size_t total;
};

// u [B, Hq, N] f32 | dq partials [B, Hkv, N, K, G, d] bf16 | ds^ [B, Hkv, N, K, G] f32 |
// (the G heads of a (row, slot) adjacent: one workgroup's waves write them together)
// sorted lists [B, Hkv, N*K] i32 | inverse index
// Element offset of the per-slot value of (row n, slot, head hh) of KV group bg.
__device__ __forceinline__ size_t slot_offset(size_t bg, int N, int n, int K, int slot, int G, int hh, int D) {
    return (((bg * N + n) * K + slot) * G + hh) * (size_t)D;
}

BwLayout bw_layout(int B, int Hq, int Hkv, int N, int L, int d, int K) {
    BwLayout w;
    w.u = 0;
    w.dqp = align256(w.u + (size_t)B * Hq * N * sizeof(float));
    w.dsh = align256(w.dqp + (size_t)B * Hq * N * K * d * sizeof(uint16_t));
    w.sorted = align256(w.dsh + (size_t)B * Hq * N * K * sizeof(float));
    w.inv_base = align256(w.sorted + (size_t)B * Hkv * N * K * sizeof(int));
    w.inv = inv_layout(B, Hkv, N, L, K, w.inv_base);
    w.total = w.inv.end;
    return w;
}

template <int D>
struct BT {
    static constexpr int KS = D / 32;    // 32-wide k-steps over the head dim
    static constexpr int DB = D / 16;    // 16-wide blocks of the head dim
    static constexpr int KROW = D + 8;   // padded row of a [64][D] tile (bf16)
    static constexpr int PROW = 64 + 8;  // padded row of a [64 pairs][64 keys] tile
    static constexpr int HROW = 16 + 8;  // padded row of the [64 pairs][16 heads] tile
};

// The value, moved through a vector register: the compiler then treats it as
// per-lane and selects with it instead of branching.
__device__ __forceinline__ int in_vgpr(int x) {
    int y;
    asm volatile("v_mov_b32 %0, %1" : "=v"(y) : "v"(x));
    return y;
}

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Operand read from a padded row-major tile: rows r0 + l%16, the 8 consecutive
// columns k0 + (l/16)*8 ...
template <int ROW>
__device__ __forceinline__ bf16x8 row_operand(const bf16* base, int r0, int k0, int lane) {
    return ld_bf16x8(base + (r0 + lane % 16) * ROW + k0 + (lane / 16) * 8);
}

// B operand from two S^T accumulator blocks (keys 32t + (l/16)*4 + i, then +16).
__device__ __forceinline__ bf16x8 pack_perm(const float* e0, const float* e1) {
    const float x[8] = {e0[0], e0[1], e0[2], e0[3], e1[0], e1[1], e1[2], e1[3]};
    return pack_bf16x8(x);
}

// ---------------------------------------------------------------------------
// u = dO . out: D/8 lanes per (row, head), 16 bytes of each per lane
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(kBlock) void k_bwd_u(BwdArgs a, float* u) {
    constexpr int LPR = D / 8;  // lanes per row
    const size_t rows = (size_t)a.B * a.Hq * a.N;
    const size_t r = (size_t)blockIdx.x * (kBlock / LPR) + threadIdx.x / LPR;
    const int d0 = (threadIdx.x % LPR) * 8;
    const size_t rr = r < rows ? r : rows - 1;  // every lane reaches the group sum below
    const uint4 go = *reinterpret_cast<const uint4*>(as<bf16>(a.dout) + rr * D + d0);
    const uint4 oo = *reinterpret_cast<const uint4*>(as<bf16>(a.out) + rr * D + d0);
    float acc = bf_lo(go.x) * bf_lo(oo.x) + bf_hi(go.x) * bf_hi(oo.x);
    acc += bf_lo(go.y) * bf_lo(oo.y) + bf_hi(go.y) * bf_hi(oo.y);
    acc += bf_lo(go.z) * bf_lo(oo.z) + bf_hi(go.z) * bf_hi(oo.z);
    acc += bf_lo(go.w) * bf_lo(oo.w) + bf_hi(go.w) * bf_hi(oo.w);
    acc = group_sum<LPR>(acc);
    if (r < rows && d0 == 0) u[r] = acc;
}

// ---------------------------------------------------------------------------
// Ascending-row copy of every (b, g, chunk) list.  Rows in a list are distinct
// (a row names a chunk at most once), so a bitmap over rows gives each entry its
// rank; rows are taken in windows of kSortWin.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_inv_sort(const int* offsets, const int* list, int* sorted, int N, int K,
                                                     int nC, int W) {
    __shared__ uint32_t s_bits[kSortWords];
    __shared__ int s_pre[kSortWords];
    __shared__ int s_wave[kBlock / kWave];
    const int c = blockIdx.x, bg = blockIdx.y, tid = threadIdx.x, lane = tid % kWave, w = wave_id();
    const int beg = offsets[(size_t)bg * (nC + 1) + c];
    const int len = offsets[(size_t)bg * (nC + 1) + c + 1] - beg;
    if (len == 0) return;
    const int* src = list + (size_t)bg * N * K + beg;
    int* dst = sorted + (size_t)bg * N * K + beg;
    // the first row whose candidate set contains c
    const int row_lo = min(N, max(0, (c + 1) * kChunk + W - 1));
    int base = 0;
    for (int w0 = row_lo; w0 < N; w0 += kSortWin) {
        for (int i = tid; i < kSortWords; i += kBlock) s_bits[i] = 0u;
        __syncthreads();
        for (int e = tid; e < len; e += kBlock) {
            const int n = (src[e] >> 6) - w0;
            if (n >= 0 && n < kSortWin) atomicOr(&s_bits[n >> 5], 1u << (n & 31));
        }
        __syncthreads();
        // exclusive prefix of the word popcounts: each thread scans a run of words
        constexpr int PER = kSortWords / kBlock;
        int run = 0;
#pragma unroll
        for (int i = 0; i < PER; ++i) run += __popc(s_bits[tid * PER + i]);
        int incl = run;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const int y = __shfl_up(incl, o, kWave);
            if (lane >= o) incl += y;
        }
        if (lane == kWave - 1) s_wave[w] = incl;
        __syncthreads();
        int excl = incl - run;
        for (int i = 0; i < w; ++i) excl += s_wave[i];
#pragma unroll
        for (int i = 0; i < PER; ++i) {
            s_pre[tid * PER + i] = excl;
            excl += __popc(s_bits[tid * PER + i]);
        }
        int total = 0;
        for (int i = 0; i < kBlock / kWave; ++i) total += s_wave[i];
        __syncthreads();
        for (int e = tid; e < len; e += kBlock) {
            const int ent = src[e];
            const int n = (ent >> 6) - w0;
            if (n >= 0 && n < kSortWin) {
                const int wd = n >> 5;
                dst[base + s_pre[wd] + __popc(s_bits[wd] & ((1u << (n & 31)) - 1u))] = ent;
            }
        }
        base += total;
        __syncthreads();
    }
}

// ---------------------------------------------------------------------------
// Key-major pass: dK, dV, dK', db' of one chunk and the retrieved chunks' dq partials
// ---------------------------------------------------------------------------
// One block of 8 waves per (b, g, chunk c), two waves per SIMD.  A step takes 64
// (row, head) pairs, four tiles of 16.  Phase 1: wave w holds K and V of the key
// half 32 (w % 2) ... of the chunk in registers and works on pair tile w / 2, so
// that the two waves of a tile share its softmax terms through LDS (retrieved
// chunks: the max, sum and sum of p gv over each half).  Phase 2: wave w owns keys
// 16 (w % 4) ... x head-dim half w / 2 / 2 of dK and dV, head-dim block w of dK'
// and, for retrieving rows, head-dim half w % 2 of pair tile w / 2's dq partial.
constexpr int kKeyWaves = 8;
constexpr int kKeyThreads = kKeyWaves * kWave;

// Tiles k, q, g, qr, p, ds are swizzled (st_off), rows of D or 64 bf16.
template <int D, bool ROUTE>
struct KeySmem {
    static constexpr int KROW = BT<D>::KROW, TD = st_size<D>(64), TP = st_size<kChunk>(kPairs);
    bf16 k[TD];                       // K of the chunk [key][d] (K^T operands of dq)
    bf16 q[2][TD];                    // q of a step's pairs [pair][d], two steps in flight
    bf16 g[2][TD];                    // dO
    bf16 qr[ROUTE ? 2 : 1][ROUTE ? TD : 8];  // q^ (routing queries given)
    bf16 p[TP];                       // dV weights [pair][key]
    bf16 ds[TP];                      // ds [pair][key]
    bf16 h[kPairs * 16];                             // ds^_c in the columns of the pair's landmark head
    bf16 lm[8 * KROW];                               // landmark rows of the group's heads (or its one)
    float red[2][kPairs][3];                            // per key half: max, sum, sum of p gv of each pair
    float db[4][16];
};

// What a wave fetches for its pair tile's next step: q (key half 0) or dO (key
// half 1) rows, q^ (key half 0, routing queries given), and per pair the row entry
// (n << 6 | slot, or -1), L * log2(e) (+inf for an empty pair, which zeroes all of
// its weights) and u.
template <int KS, bool ROUTE>
struct PairOps {
    bf16x8 x[KS], y[ROUTE ? KS : 1];
    float L2, u;
    int ent;
};

// Head-dim half `half` (blocks half * D/32 ...) of a lane-order vector.
template <int D>
__device__ __forceinline__ void store_lane_order_half(bf16* row, const f32x4* o, int lg, int half) {
    typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
#pragma unroll
    for (int t = 0; t < D / 64; ++t) {
        const u32x4 v = {pack_bf16x2(o[2 * t][0], o[2 * t][1]), pack_bf16x2(o[2 * t][2], o[2 * t][3]),
                         pack_bf16x2(o[2 * t + 1][0], o[2 * t + 1][1]), pack_bf16x2(o[2 * t + 1][2], o[2 * t + 1][3])};
        *reinterpret_cast<u32x4*>(row + 32 * (half * (D / 64) + t) + 8 * lg) = v;
    }
}

template <int D, int G, bool ROUTE>
__global__ __launch_bounds__(kKeyThreads) void k_bwd_keys(BwdArgs a, const int* offsets, const int* sorted,
                                                          const float* u, bf16* dqp, float* dshat) {
    constexpr int KS = BT<D>::KS, DB = BT<D>::DB, KROW = BT<D>::KROW;
    constexpr int R = kPairs / G;  // rows per step
    constexpr int DH = DB / 2;     // phase 2: head-dim blocks per wave
    __shared__ __align__(16) KeySmem<D, ROUTE> sm;
    const int tid = threadIdx.x, w = wave_id(), lane = tid % kWave, lg = lane / 16;
    const int nC = a.L / kChunk;
    // Workgroups go round-robin over the 8 XCDs.  With nC a multiple of 32 the chunk
    // order below gives each XCD runs of 4 neighbouring chunks (whose local windows
    // overlap, so their rows meet in that XCD's L2), the runs spread over the whole
    // chunk range and dealt to the XCDs in alternating directions (early chunks are
    // retrieved by more rows: one contiguous range per XCD would load the XCDs
    // unevenly).
    int c = blockIdx.x;
    if (nC % 32 == 0) {
        const int x = c % 8, blk = c / 32;
        c = 4 * (blk % 2 ? 7 - x : x) + 32 * blk + (c / 8) % 4;
    }
    const int g = blockIdx.y, b = blockIdx.z;
    const size_t bg = (size_t)b * a.Hkv + g;
    const int j0 = c * kChunk;
    const bool per_head_lmk = (a.Hl == a.Hq);
    const int nLH = per_head_lmk ? G : 1;
    const bf16* qb = as<bf16>(a.q);
    const bf16* gob = as<bf16>(a.dout);
    const bf16* rb = as<bf16>(a.q_route);
    const float c1 = a.scale * kLog2e;
    const int kh = w % 2, pt = w / 2;   // phase 1: key half, pair tile
    const int kb2 = w % 4, dh = w / 4;  // phase 2: 16-key block, head-dim half of dK / dV

    // K and V of the key half as phase-1 A operands (lane: key 32 kh + 16 kb + l%16,
    // dims 32 ks + (l/16)*8 ...); waves of pair tiles 0 and 1 also store their first
    // or second 16 keys into LDS for the K^T operands of the dq partials
    bf16x8 kA[2][KS], vA[2][KS];
    {
        const bf16* kb0 = as<bf16>(a.k) + (bg * a.L + j0) * D;
        const bf16* vb0 = as<bf16>(a.v) + (bg * a.L + j0) * D;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const size_t off = (size_t)(32 * kh + kb * 16 + lane % 16) * D + ks * 32 + lg * 8;
                kA[kb][ks] = ld_bf16x8(kb0 + off);
                vA[kb][ks] = ld_bf16x8(vb0 + off);
            }
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
            if (kb == pt)
#pragma unroll
                for (int ks = 0; ks < KS; ++ks)
                    *reinterpret_cast<bf16x8*>(sm.k + st_off<D>(32 * kh + kb * 16 + lane % 16, ks * 32 + lg * 8)) =
                        kA[kb][ks];
        for (int e = tid; e < nLH * (D / 8); e += kKeyThreads) {
            const int m = e / (D / 8), d8 = (e % (D / 8)) * 8;
            const int hlm = per_head_lmk ? g * G + m : g;
            *reinterpret_cast<uint4*>(sm.lm + m * KROW + d8) =
                *reinterpret_cast<const uint4*>(as<bf16>(a.lmk) + (((size_t)b * a.Hl + hlm) * nC + c) * D + d8);
        }
    }

    // this lane's pair in phase 1
    const int pair = pt * 16 + lane % 16;
    const int hh = pair / R, r = pair % R;
    const int h = g * G + hh;
    const int hfirst = (pt * 16) / R;
    const int hl = per_head_lmk ? h : g;
    // row of the landmark tile in A-operand row m = l%16 of s^: head hfirst + m of the
    // tile (per-head landmarks; rows past the group's heads repeat its last one and
    // are not used) or the group's one landmark
    const int lrow = per_head_lmk ? min(hfirst + lane % 16, G - 1) : 0;
    const int hloc = per_head_lmk ? hh - hfirst : 0;
    const float bias_h = a.bias ? a.bias[((size_t)b * a.Hl + hl) * nC + c] : 0.f;

    f32x4 dk[DH], dv[DH], dkl = zero4();
#pragma unroll
    for (int dl = 0; dl < DH; ++dl) dk[dl] = dv[dl] = zero4();
    float dbl = 0.f;

    const int n_lo = j0, n_hi = min(a.N - 1, j0 + kChunk + a.W - 2);
    const int nlocal = max(0, n_hi - n_lo + 1);
    const int beg = offsets[bg * (nC + 1) + c];
    const int nret = offsets[bg * (nC + 1) + c + 1] - beg;
    const int* seg = sorted + bg * a.N * a.K + beg;
    const int nsl = (nlocal + R - 1) / R;
    const int nst = nsl + (nret + R - 1) / R;

    // Loads below are branch-free (indices clamped to a valid row, the result masked
    // afterwards) so that the compiler can count outstanding loads exactly and the
    // prefetch of the next step is not drained by a full wait at every step.
    auto entry_of = [&](int s) -> int {
        // `loc` goes through a vector register so that the choice below is a select,
        // not a scalar branch around the load
        const int loc = in_vgpr(s < nsl ? 1 : 0);
        const int e = loc ? s * R + r : (s - nsl) * R + r;
        const int lim = loc ? nlocal : nret;
        const int got = seg[min(max(e, 0), max(nret - 1, 0))];
        const int ent = loc ? (n_lo + e) << 6 : got;
        return (s < nst && e < lim) ? ent : -1;
    };
    // An empty pair (ent < 0) reads row 0 and gets L = +inf.
    const bf16* src = kh ? gob : qb;
    auto load_ops = [&](int ent) {
        PairOps<KS, ROUTE> x;
        x.ent = ent;
        const bool ok = ent >= 0;
        const size_t row = ((size_t)b * a.Hq + h) * a.N + (ok ? (ent >> 6) : 0);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const int d0 = ks * 32 + lg * 8;
            x.x[ks] = ld_bf16x8(src + row * D + d0);
            if constexpr (ROUTE) x.y[ks] = ld_bf16x8(rb + row * D + d0);
        }
        const float L = a.lse[row];
        x.L2 = ok ? L * kLog2e : INFINITY;
        x.u = u[row];
        return x;
    };
    auto stage_ops = [&](int buf, const PairOps<KS, ROUTE>& x) {
        bf16* dst = kh ? sm.g[buf] : sm.q[buf];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const int o = st_off<D>(pair, ks * 32 + lg * 8);
            *reinterpret_cast<bf16x8*>(dst + o) = x.x[ks];
            if constexpr (ROUTE)
                if (kh == 0) *reinterpret_cast<bf16x8*>(sm.qr[buf] + o) = x.y[ks];
        }
    };

    PairOps<KS, ROUTE> nxt = load_ops(entry_of(0));
    float curL2 = nxt.L2, curU = nxt.u;
    int curEnt = nxt.ent;
    stage_ops(0, nxt);
    nxt = load_ops(entry_of(1));
    int ent_next = entry_of(2);

    for (int st = 0; st < nst; ++st) {
        const int buf = st & 1;
        const bool retrieval = st >= nsl;
        const bool qv = curEnt >= 0;
        const int qn = curEnt >> 6, slot = curEnt & 63;
        __syncthreads();  // step st's tiles are staged; step st - 1's phase 2 is done

        // ---- phase 1: pair tile pt against the 32 keys of half kh ----
        bf16x8 bq[KS], bo[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            bq[ks] = row_operand_st<D>(sm.q[buf], pt * 16, ks * 32, lane);
            bo[ks] = row_operand_st<D>(sm.g[buf], pt * 16, ks * 32, lane);
        }
        f32x4 s4[2], gv4[2];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            s4[kb] = zero4();
            gv4[kb] = zero4();
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                s4[kb] = mfma16x16x32(kA[kb][ks], bq[ks], s4[kb]);
                gv4[kb] = mfma16x16x32(vA[kb][ks], bo[ks], gv4[kb]);
            }
        }
        float pw[2][4], ds[2][4];
        float dsh = 0.f;  // ds^_c of the lane's pair (retrieving rows)
        if (!retrieval) {
            // rows of the step below j0 + 63 see only part of the chunk (j <= n)
            const bool diag = st * R < kChunk - 1;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    float x = fmaf(s4[kb][i], c1, -curL2);
                    if (diag && j0 + 32 * kh + kb * 16 + lg * 4 + i > qn) x = -INFINITY;
                    const float wgt = fexp2(x);
                    pw[kb][i] = wgt;
                    ds[kb][i] = wgt * (gv4[kb][i] - curU);
                }
        } else {
            // s^_c of the pair: landmark rows (A) against the pair's q^ (B)
            f32x4 sh4 = zero4();
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const bf16x8 al = ld_bf16x8(sm.lm + lrow * KROW + ks * 32 + lg * 8);
                if constexpr (ROUTE)
                    sh4 = mfma16x16x32(al, row_operand_st<D>(sm.qr[buf], pt * 16, ks * 32, lane), sh4);
                else
                    sh4 = mfma16x16x32(al, bq[ks], sh4);
            }
            float mine = sh4[0];
#pragma unroll
            for (int i = 1; i < 4; ++i)
                if (hloc == i) mine = sh4[i];
            const float shat = a.scale * group0_bcast(mine) + bias_h;
            // softmax terms over this half's 32 keys
            float mx = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) mx = fmaxf(mx, fmaxf(fmaxf(s4[kb][0], s4[kb][1]), fmaxf(s4[kb][2], s4[kb][3])));
            mx = group4_max(mx);
            const float m2 = mx * c1;
            float sum = 0.f, ue = 0.f;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float e = fexp2(fmaf(s4[kb][i], c1, -m2));
                    pw[kb][i] = e;
                    sum += e;
                    ue = fmaf(e, gv4[kb][i], ue);
                }
            sum = group4_sum(sum);
            ue = group4_sum(ue);
            if (lg == 0) {
                sm.red[kh][pair][0] = mx;
                sm.red[kh][pair][1] = sum;
                sm.red[kh][pair][2] = ue;
            }
            __syncthreads();
            // both halves, combined in the same order by the two waves of the tile
            const float mo = sm.red[kh ^ 1][pair][0], so = sm.red[kh ^ 1][pair][1], uo = sm.red[kh ^ 1][pair][2];
            const float m0 = kh ? mo : mx, m1 = kh ? mx : mo;
            const float s0 = kh ? so : sum, s1 = kh ? sum : so;
            const float u0 = kh ? uo : ue, u1 = kh ? ue : uo;
            const float M = fmaxf(m0, m1);
            const float f0 = fexp2((m0 - M) * c1), f1 = fexp2((m1 - M) * c1);
            const float tot = s0 * f0 + s1 * f1;
            const float inv = 1.f / tot;
            const float uc = (u0 * f0 + u1 * f1) * inv;
            const float al = qv ? fexp2(fmaf(shat, kLog2e, -curL2)) : 0.f;
            const float f = al * inv * (kh ? f1 : f0);
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    pw[kb][i] *= f;
                    ds[kb][i] = pw[kb][i] * (gv4[kb][i] - uc);
                }
            dsh = al * (uc - curU);
            if (kh == 0) {
                if (ROUTE && qv && lane < 16) dshat[slot_offset(bg, a.N, qn, a.K, slot, G, hh, 1)] = dsh;
                // H row of the pair: ds^ split into a bf16 head and its bf16 residual, in
                // columns m and 8 + m of its landmark head m (the product then keeps ds^
                // to about fp32 accuracy)
                if (lane < 16) {
                    const int col = per_head_lmk ? hh : 0;
                    const float hi = to_f32(from_f32<bf16>(dsh)), lo = dsh - hi;
                    float hv[16];
#pragma unroll
                    for (int t = 0; t < 16; ++t) hv[t] = t == col ? hi : (t == col + 8 ? lo : 0.f);
                    uint32_t wds[8];
#pragma unroll
                    for (int t = 0; t < 8; ++t) wds[t] = pack_bf16x2(hv[2 * t], hv[2 * t + 1]);
                    *reinterpret_cast<uint4*>(sm.h + pair * 16) = make_uint4(wds[0], wds[1], wds[2], wds[3]);
                    *reinterpret_cast<uint4*>(sm.h + pair * 16 + 8) = make_uint4(wds[4], wds[5], wds[6], wds[7]);
                }
                // db': sum ds^ over the pairs of each head of the tile
                const float hs = (R >= 16) ? group_sum<16>(dsh) : group_sum<8>(dsh);
                if (lane < 16 && (lane % (R >= 16 ? 16 : 8)) == 0) dbl += hs;
            }
        }
        // dV weights and ds, row-major [pair][key]
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            const int key = 32 * kh + kb * 16 + lg * 4;
            *reinterpret_cast<uint2*>(sm.p + st_off<kChunk>(pair, key)) =
                make_uint2(pack_bf16x2(pw[kb][0], pw[kb][1]), pack_bf16x2(pw[kb][2], pw[kb][3]));
            *reinterpret_cast<uint2*>(sm.ds + st_off<kChunk>(pair, key)) =
                make_uint2(pack_bf16x2(ds[kb][0], ds[kb][1]), pack_bf16x2(ds[kb][2], ds[kb][3]));
        }
        // stage step st + 1 into the other buffers (read last by step st - 1's phase 2)
        // and fetch step st + 2
        const float nL2 = nxt.L2, nU = nxt.u;
        const int nEnt = nxt.ent;
        if (st + 1 < nst) stage_ops(buf ^ 1, nxt);
        const int ent_after = entry_of(st + 3);
        nxt = load_ops(ent_next);
        ent_next = ent_after;
        __syncthreads();

        // ---- phase 2: keys 16 kb2 ... x head-dim half dh, over the 64 pairs ----
        bf16x8 ads[2], ap[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            ads[t] = tr_operand_st<kChunk>(sm.ds, t * 32, kb2 * 16, lane);
            ap[t] = tr_operand_st<kChunk>(sm.p, t * 32, kb2 * 16, lane);
        }
#pragma unroll
        for (int dl = 0; dl < DH; ++dl) {
            const int db = dh * DH + dl;
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                dk[dl] = mfma16x16x32(ads[t], tr_operand_st<D>(sm.q[buf], t * 32, db * 16, lane), dk[dl]);
                dv[dl] = mfma16x16x32(ap[t], tr_operand_st<D>(sm.g[buf], t * 32, db * 16, lane), dv[dl]);
            }
        }
        if (retrieval) {
            // dk': the H tile against q^ (or q), head-dim block w
            if (w < DB)
#pragma unroll
                for (int t = 0; t < 2; ++t)
                    dkl = mfma16x16x32(tr_operand(sm.h, 16, t * 32, 0, lane),
                                       tr_operand_st<D>(ROUTE ? sm.qr[buf] : sm.q[buf], t * 32, w * 16, lane), dkl);
            // the chunk's share of dq / scale for pair tile pt, head-dim half kh: K^T ds^T,
            // and without routing queries also ds^_c k'_c (lane: dims 16 db + (l/16)*4 + i)
            const bf16x8 b0 = row_operand_st<kChunk>(sm.ds, pt * 16, 0, lane);
            const bf16x8 b1 = row_operand_st<kChunk>(sm.ds, pt * 16, 32, lane);
            f32x4 od[DB / 2];
#pragma unroll
            for (int dl = 0; dl < DB / 2; ++dl) {
                const int db = kh * (DB / 2) + dl;
                f32x4 o0 = zero4();
                if constexpr (!ROUTE) {
                    const uint2 lw = *reinterpret_cast<const uint2*>(sm.lm + (per_head_lmk ? hh : 0) * KROW + db * 16 + lg * 4);
                    o0 = f32x4{dsh * bf_lo(lw.x), dsh * bf_hi(lw.x), dsh * bf_lo(lw.y), dsh * bf_hi(lw.y)};
                }
                od[dl] = mfma16x16x32(tr_operand_st<D>(sm.k, 0, db * 16, lane), b0, o0);
                od[dl] = mfma16x16x32(tr_operand_st<D>(sm.k, 32, db * 16, lane), b1, od[dl]);
            }
            if (qv) store_lane_order_half<D>(dqp + slot_offset(bg, a.N, qn, a.K, slot, G, hh, D), od, lg, kh);
        }
        curL2 = nL2;
        curU = nU;
        curEnt = nEnt;
    }

    // ---- dK, dV of the chunk (lane: key 16 kb2 + (l/16)*4 + i, dim 16 db + l%16) ----
    bf16* dkp = as_mut<bf16>(a.dk) + (bg * a.L + j0) * D;
    bf16* dvp = as_mut<bf16>(a.dv) + (bg * a.L + j0) * D;
#pragma unroll
    for (int dl = 0; dl < DH; ++dl)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int key = kb2 * 16 + lg * 4 + i, d = (dh * DH + dl) * 16 + lane % 16;
            dkp[key * D + d] = from_f32<bf16>(a.scale * dk[dl][i]);
            dvp[key * D + d] = from_f32<bf16>(dv[dl][i]);
        }
    // ---- dK' (lane: rows (l/16)*4 + i = head m and its residual row m + 8 in lane
    // l ^ 32, dim 16 w + l%16) ----
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float v = dkl[i] + __shfl_xor(dkl[i], 32, kWave);
        const int m = lg * 4 + i, d = w * 16 + lane % 16;
        if (w < DB && lg < 2 && m < nLH) {
            const int hl_out = per_head_lmk ? g * G + m : g;
            as_mut<bf16>(a.dlmk)[(((size_t)b * a.Hl + hl_out) * nC + c) * D + d] = from_f32<bf16>(a.scale * v);
        }
    }
    // ---- db': per-lane head sums of the pair tiles ----
    if (a.dbias) {
        if (kh == 0 && lane < 16) sm.db[pt][lane] = dbl;
        __syncthreads();
        if (tid < nLH) {
            float v = 0.f;
            for (int tt = 0; tt < 4; ++tt)
                for (int l = 0; l < 16; ++l)
                    if (!per_head_lmk || (tt * 16 + l) / R == tid) v += sm.db[tt][l];
            const int hl_out = per_head_lmk ? g * G + tid : g;
            a.dbias[((size_t)b * a.Hl + hl_out) * nC + c] = v;
        }
    }
}

// ---------------------------------------------------------------------------
// Query-major dq: local window, then the row's retrieved-chunk partials
// ---------------------------------------------------------------------------
// One block of 8 waves per tile of 16 * 8 / G rows of one KV group; wave w owns
// the item (head w / QB, 16-row block w % QB).  The window's 64-key blocks of K
// and V are double-buffered in LDS (the next block is fetched into registers
// while the current one is used), one barrier per block.
template <int G>
struct DqCfg {
    static constexpr int QB = 8 / G;          // 16-row blocks per workgroup
    static constexpr int QT = 16 * QB;        // rows per workgroup
    static constexpr int NT = 8 * kWave;      // threads
};

template <int D>
struct DqSmem {
    static constexpr int KROW = BT<D>::KROW;
    bf16 k[2][st_size<D>(kChunk)];  // swizzled: row-wise and transposing reads
    bf16 v[2][kChunk * KROW];
};

// acc (O^T layout) += x * the bf16 row held as lv (dims 16 db + (l/16)*4 ...)
template <int DB>
__device__ __forceinline__ void fma_lmk(f32x4* acc, const uint2* lv, float x) {
#pragma unroll
    for (int db = 0; db < DB; ++db) {
        acc[db][0] += x * bf_lo(lv[db].x);
        acc[db][1] += x * bf_hi(lv[db].x);
        acc[db][2] += x * bf_lo(lv[db].y);
        acc[db][3] += x * bf_hi(lv[db].y);
    }
}

// ROUTE: routing queries given, so that scale ds^ k' goes to dq^ instead of dq.
template <int D, int G, bool ROUTE>
__global__ __launch_bounds__(DqCfg<G>::NT, 4) void k_bwd_dq(BwdArgs a, const float* u, const bf16* dqp,
                                                           const float* dshat) {
    using C = DqCfg<G>;
    constexpr int KS = BT<D>::KS, DB = BT<D>::DB, KROW = BT<D>::KROW;
    constexpr int PPT = kChunk * D / 8 / C::NT;  // 16-byte pieces per thread of a K or V block
    static_assert(PPT >= 1 && kChunk * D / 8 == PPT * C::NT, "K/V blocks split evenly over the threads");
    __shared__ __align__(16) DqSmem<D> sm;
    const int tid = threadIdx.x, w = wave_id(), lane = tid % kWave, lg = lane / 16;
    const int ntiles = (a.N + C::QT - 1) / C::QT;
    const int tile = xcd_remap(blockIdx.x, ntiles), g = blockIdx.y, b = blockIdx.z;
    const int q0 = tile * C::QT;
    const int qlast = min(q0 + C::QT - 1, a.N - 1);
    const int kbeg = n_candidates(q0, a.W) * kChunk;
    const size_t bg = (size_t)b * a.Hkv + g;
    const int nC = a.L / kChunk;
    const bf16* kbase = as<bf16>(a.k) + bg * a.L * D;
    const bf16* vbase = as<bf16>(a.v) + bg * a.L * D;
    const int hh = w / C::QB, qb = w % C::QB;
    const int nq_raw = q0 + qb * 16 + lane % 16;
    const int nq = min(nq_raw, a.N - 1);
    const int h = g * G + hh;
    const size_t qrow = ((size_t)b * a.Hq + h) * a.N + nq;

    struct KV {
        uint4 k[PPT], v[PPT];
    };
    auto fetch = [&](int j0) {
        KV x;
#pragma unroll
        for (int t = 0; t < PPT; ++t) {
            const int e = tid + t * C::NT, j = e / (D / 8), d8 = (e % (D / 8)) * 8;
            x.k[t] = *reinterpret_cast<const uint4*>(kbase + (size_t)(j0 + j) * D + d8);
            x.v[t] = *reinterpret_cast<const uint4*>(vbase + (size_t)(j0 + j) * D + d8);
        }
        return x;
    };
    auto stage = [&](int buf, const KV& x) {
#pragma unroll
        for (int t = 0; t < PPT; ++t) {
            const int e = tid + t * C::NT, j = e / (D / 8), d8 = (e % (D / 8)) * 8;
            *reinterpret_cast<uint4*>(&sm.k[buf][st_off<D>(j, d8)]) = x.k[t];
            *reinterpret_cast<uint4*>(&sm.v[buf][j * KROW + d8]) = x.v[t];
        }
    };

    bf16x8 bq[KS], bo[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        bq[ks] = ld_bf16x8(as<bf16>(a.q) + qrow * D + ks * 32 + lg * 8);
        bo[ks] = ld_bf16x8(as<bf16>(a.dout) + qrow * D + ks * 32 + lg * 8);
    }
    f32x4 dq[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) dq[db] = zero4();
    const float Lr = a.lse[qrow], ub = u[qrow];
    const int ell = n_candidates(nq, a.W) * kChunk;

    KV nx = fetch(kbeg);
    stage(0, nx);
    __syncthreads();
    int buf = 0;
    for (int j0 = kbeg; j0 <= qlast; j0 += kChunk, buf ^= 1) {
        const bool more = j0 + kChunk <= qlast;  // uniform over the block
        if (more) nx = fetch(j0 + kChunk);
        const bf16* tk = sm.k[buf];
        const bf16* tv = sm.v[buf];
        // keys in two halves of 32 (fewer live accumulators); dq takes the halves in order
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
            f32x4 s4[2], gv4[2];
#pragma unroll
            for (int k2 = 0; k2 < 2; ++k2) {
                const int kb = 2 * hf + k2;
                s4[k2] = zero4();
                gv4[k2] = zero4();
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    s4[k2] = mfma16x16x32(row_operand_st<D>(tk, kb * 16, ks * 32, lane), bq[ks], s4[k2]);
                    gv4[k2] = mfma16x16x32(row_operand<KROW>(tv, kb * 16, ks * 32, lane), bo[ks], gv4[k2]);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
            float ds[2][4];
#pragma unroll
            for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int j = j0 + (2 * hf + k2) * 16 + lg * 4 + i;
                    const bool valid = nq_raw < a.N && j <= nq && j >= ell;
                    const float wgt = valid ? fexp(a.scale * s4[k2][i] - Lr) : 0.f;
                    ds[k2][i] = wgt * (gv4[k2][i] - ub);
                }
            const bf16x8 bh = pack_perm(ds[0], ds[1]);
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                dq[db] = mfma16x16x32(tr_operand_perm_st<D>(tk, 32 * hf, db * 16, lane), bh, dq[db]);
                if (db % 4 == 3) __builtin_amdgcn_sched_barrier(0);
            }
        }
        if (more) stage(buf ^ 1, nx);
        __syncthreads();
    }
    // epilogue (lane: row l%16 of the item, dims 16db + (l/16)*4 + {0..3}): the row's
    // slot partials and scale ds^ k', one slot ahead in flight (the slot's chunk id,
    // which the landmark row's address needs, two ahead)
    if (nq_raw >= a.N) return;  // no barriers below
    const int hl = (a.Hl == a.Hq) ? h : g;
    const int32_t* irow = a.idx + (bg * a.N + nq) * a.K;
    const int ncand = n_candidates(nq, a.W);
    f32x4 accr[ROUTE ? DB : 1];
#pragma unroll
    for (int db = 0; db < (ROUTE ? DB : 1); ++db) accr[db] = zero4();
    // a slot's inputs: the lane-order partial (which, without routing queries, holds
    // ds^_c k'_c too) and, with routing queries, ds^ and the landmark row k'_c
    struct SlotIn {
        uint4 pv[D / 32];
        uint2 lv[ROUTE ? DB : 1];
        float x;
    };
    auto fetch_slot = [&](int k, int cc) {
        SlotIn r;
        load_lane_order<D>(dqp + slot_offset(bg, a.N, nq, a.K, k, G, hh, D), lg, r.pv);
        if constexpr (ROUTE) {
            const int ck = (cc >= 0 && cc < ncand) ? cc : 0;
            r.x = dshat[slot_offset(bg, a.N, nq, a.K, k, G, hh, 1)];
            const bf16* lrow = as<bf16>(a.lmk) + (((size_t)b * a.Hl + hl) * nC + ck) * D;
#pragma unroll
            for (int db = 0; db < DB; ++db) r.lv[db] = *reinterpret_cast<const uint2*>(lrow + db * 16 + lg * 4);
        }
        return r;
    };
    if (a.K > 0) {
        int c_prev = -1, c_cur = irow[0], c_nxt = irow[min(1, a.K - 1)];
        SlotIn cur = fetch_slot(0, c_cur);
        for (int k = 0; k < a.K; ++k) {
            const int c_after = irow[min(k + 2, a.K - 1)];
            const SlotIn nx = fetch_slot(min(k + 1, a.K - 1), c_nxt);
            // idx_entry_valid: a candidate chunk, above the previous entry as written
            const bool ok = c_cur >= 0 && c_cur < ncand && c_cur > c_prev;
            fma_lane_order<D>(cur.pv, 1.f, ok, dq);
            // ds^ unscaled: dq^ is scaled at the end
            if constexpr (ROUTE) fma_lmk<DB>(accr, cur.lv, ok ? cur.x : 0.f);
            c_prev = c_cur;
            c_cur = c_nxt;
            c_nxt = c_after;
            cur = nx;
        }
    }
    bf16* dqo = as_mut<bf16>(a.dq) + qrow * D;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
        const int d0 = db * 16 + lg * 4;
        const f32x4 x = dq[db] * a.scale;
        *reinterpret_cast<uint2*>(dqo + d0) = make_uint2(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]));
        if constexpr (ROUTE) {
            const f32x4 y = accr[db] * a.scale;
            *reinterpret_cast<uint2*>(as_mut<bf16>(a.dq_route) + qrow * D + d0) =
                make_uint2(pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3]));
        }
    }
}

struct BwRun {
    template <typename T, int D, int G>
    static hipError_t run(const BwdArgs& a, hipStream_t s) {
        const BwLayout ly = bw_layout(a.B, a.Hq, a.Hkv, a.N, a.L, D, a.K);
        char* ws = static_cast<char*>(a.ws);
        float* u = reinterpret_cast<float*>(ws + ly.u);
        bf16* dqp = reinterpret_cast<bf16*>(ws + ly.dqp);
        float* dsh = reinterpret_cast<float*>(ws + ly.dsh);
        int* sorted = reinterpret_cast<int*>(ws + ly.sorted);
        const int* offsets = reinterpret_cast<const int*>(ws + ly.inv.offsets);
        const int nC = a.L / kChunk;
        const size_t rows = (size_t)a.B * a.Hq * a.N;
        constexpr int upb = kBlock / (D / 8);  // rows per k_bwd_u block
        HILS_LAUNCH("k_bwd_u", (k_bwd_u<D>), dim3((unsigned)((rows + upb - 1) / upb)), dim3(kBlock), 0, s, a, u);
        const InvArgs ia{a.idx, a.B, a.Hkv, a.N, a.K, a.W, a.L, 0, a.N};
        launch_inverse_index(ia, ly.inv, a.ws, s, false);
        HILS_LAUNCH("k_inv_sort", k_inv_sort, dim3(nC, a.B * a.Hkv), dim3(kBlock), 0, s, offsets,
                    reinterpret_cast<const int*>(ws + ly.inv.list), sorted, a.N, a.K, nC, a.W);
        if (a.q_route)
            HILS_LAUNCH("k_bwd_keys", (k_bwd_keys<D, G, true>), dim3(nC, a.Hkv, a.B), dim3(kKeyThreads), 0, s, a, offsets,
                        (const int*)sorted, (const float*)u, dqp, dsh);
        else
            HILS_LAUNCH("k_bwd_keys", (k_bwd_keys<D, G, false>), dim3(nC, a.Hkv, a.B), dim3(kKeyThreads), 0, s, a, offsets,
                        (const int*)sorted, (const float*)u, dqp, dsh);
        const dim3 dgrid((a.N + DqCfg<G>::QT - 1) / DqCfg<G>::QT, a.Hkv, a.B);
        if (a.dq_route)
            HILS_LAUNCH("k_bwd_dq", (k_bwd_dq<D, G, true>), dgrid, dim3(DqCfg<G>::NT), 0, s, a, (const float*)u,
                        (const bf16*)dqp, (const float*)dsh);
        else
            HILS_LAUNCH("k_bwd_dq", (k_bwd_dq<D, G, false>), dgrid, dim3(DqCfg<G>::NT), 0, s, a, (const float*)u,
                        (const bf16*)dqp, (const float*)dsh);
        return hipGetLastError();
    }
};

}  // namespace

size_t bwd_mfma_workspace_bytes(int B, int Hq, int Hkv, int N, int L, int d, int K) {
    return bw_layout(B, Hq, Hkv, N, L, d, K).total;
}

hipError_t launch_bwd_mfma(const BwdArgs& a, hipStream_t s) { return dispatch<BwRun>(1, a.d, a.Hq / a.Hkv, a, s); }

}  // namespace hils
