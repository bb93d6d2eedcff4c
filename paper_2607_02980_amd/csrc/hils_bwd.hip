// HiLS attention backward for fp32 storage (VALU), and the inverse index that the
// bf16 backward (MFMA) and the bf16 prefill share, gfx950.
//
// With g = dO and u = g . out for a (row, head), and L its fusion LSE:
//   local key j:     w_j = exp(s_j - L);  dv_j += w_j g;  ds_j = w_j (g.v_j - u)
//   chunk c, key j:  p_j = exp(s_j - log Z_c), a_c = exp(s^_c - L), u_c = g . o_c
//                    dv_j += a_c p_j g;  ds_j = a_c p_j (g.v_j - u_c)
//   retrieval score: ds^_c = a_c (u_c - u)
//   dq += scale ds_j k_j;  dk_j += scale ds_j q;  dq^ += scale ds^_c k'_c;
//   dk'_c += scale ds^_c q^;  db'_c += ds^_c
// (Eq. (10) differentiated with the selection fixed; selection gets no gradient.)
//
// Kernels:
//   k_bwd_dq_rows      query-major: dq and dq^ of one (b, group, n) row
//   k_inv_*            inverse index: for each (b, group, chunk) the rows that selected it
//   k_bwd_dkdv_chunks  key-major: dk, dv of one chunk from the rows whose local window
//                      covers it and from the rows that retrieved it, plus dk', db'
// Everything is accumulated on chip and written once; no floating-point atomics.
#include <type_traits>

#include "hils_device.hpp"
#include "hils_dispatch.hpp"
#include "hils_internal.hpp"

namespace hils {

constexpr int kBlock = 256;
constexpr int kSortCap = 4096;  // retrieval lists up to this length are sorted (deterministic order)

BwdWorkspace bwd_workspace_layout(int B, int Hkv, int N, int L, int K) {
    const InvLayout iv = inv_layout(B, Hkv, N, L, K, 0);
    BwdWorkspace w;
    w.counts = iv.counts;
    w.offsets = iv.offsets;
    w.cursor = iv.cursor;
    w.list = iv.list;
    w.total = iv.end;
    return w;
}

// ---------------------------------------------------------------------------
// dq / dq^ : one workgroup per (n, g, b); parts as in the forward row kernel.
// ---------------------------------------------------------------------------
template <typename T, int D, int G>
__global__ __launch_bounds__(kBlock) void k_bwd_dq_rows(BwdArgs a) {
    constexpr int R = (G * D + kBlock - 1) / kBlock;
    __shared__ float s_q[G][D], s_qr[G][D], s_do[G][D];
    __shared__ float s_k[kChunk][D + 1];
    __shared__ float s_v[kChunk][D + 1];
    __shared__ float s_cs[G][kChunk];
    __shared__ float s_dsh[G], s_L[G], s_ub[G];
    __shared__ int s_sel[64];
    __shared__ int s_nsel;

    const int tid = threadIdx.x, wave = wave_id(), lane = tid % kWave;
    const int n = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
    const int pos = n;
    const int ncand = n_candidates(pos, a.W);
    const int nC = a.L / kChunk;
    const T* kb = as<T>(a.k) + ((size_t)b * a.Hkv + g) * a.L * D;
    const T* vb = as<T>(a.v) + ((size_t)b * a.Hkv + g) * a.L * D;
    const T* qr = as<T>(a.q_route ? a.q_route : a.q);

    for (int e = tid; e < G * D; e += kBlock) {
        const int hh = e / D, dd = e % D;
        const size_t off = (((size_t)b * a.Hq + g * G + hh) * a.N + n) * D + dd;
        s_q[hh][dd] = to_f32(as<T>(a.q)[off]);
        s_qr[hh][dd] = to_f32(qr[off]);
        s_do[hh][dd] = to_f32(as<T>(a.dout)[off]);
    }
    if (tid == 0) {
        const int32_t* irow = a.idx + (((size_t)b * a.Hkv + g) * a.N + n) * a.K;
        int cnt = 0;
        for (int t = 0; t < a.K; ++t)
            if (idx_entry_valid(irow, t, ncand)) s_sel[cnt++] = irow[t];
        s_nsel = cnt;
    }
    __syncthreads();
    for (int hh = wave; hh < G; hh += 4) {
        const size_t row = ((size_t)b * a.Hq + g * G + hh) * a.N + n;
        float acc = 0.f;
        for (int dd = lane; dd < D; dd += kWave) acc += s_do[hh][dd] * to_f32(as<T>(a.out)[row * D + dd]);
        acc = wave_sum(acc);
        if (lane == 0) {
            s_ub[hh] = acc;
            s_L[hh] = a.lse[row];
        }
    }
    const int nsel = s_nsel;
    const int c_lo = ncand, c_hi = pos / kChunk;
    const int nparts = nsel + (c_hi - c_lo + 1);
    float dq[R], dqh[R];
#pragma unroll
    for (int r = 0; r < R; ++r) dq[r] = dqh[r] = 0.f;

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
            const float L = s_L[hh], ub = s_ub[hh];
            float s = -INFINITY, gv = 0.f;
            if (lane < nk) {
                float acc = 0.f, acc2 = 0.f;
#pragma unroll 16
                for (int dd = 0; dd < D; ++dd) {
                    acc += s_q[hh][dd] * s_k[lane][dd];
                    acc2 += s_do[hh][dd] * s_v[lane][dd];
                }
                s = a.scale * acc;
                gv = acc2;
            }
            float ds;
            if (is_chunk) {
                const float m = wave_max(s);
                const float l = wave_sum(fexp(s - m));
                const float lsec = m + __logf(l);
                const float p = fexp(s - lsec);
                const float uc = wave_sum(p * gv);
                const int hl = (a.Hl == a.Hq) ? g * G + hh : g;
                const T* lr = as<T>(a.lmk) + (((size_t)b * a.Hl + hl) * nC + c) * D;
                float acc = 0.f;
                for (int dd = lane; dd < D; dd += kWave) acc += s_qr[hh][dd] * to_f32(lr[dd]);
                acc = wave_sum(acc);
                const float sh = a.scale * acc + (a.bias ? a.bias[((size_t)b * a.Hl + hl) * nC + c] : 0.f);
                const float al = fexp(sh - L);
                ds = al * p * (gv - uc);
                if (lane == 0) s_dsh[hh] = al * (uc - ub);
            } else {
                const float w = lane < nk ? fexp(s - L) : 0.f;
                ds = w * (gv - ub);
            }
            s_cs[hh][lane] = ds;
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int o = tid + r * kBlock;
            if (o < G * D) {
                const int hh = o / D, dd = o % D;
                float acc = 0.f;
                for (int j = 0; j < nk; ++j) acc += s_cs[hh][j] * s_k[j][dd];
                dq[r] += a.scale * acc;
                if (is_chunk) {
                    const int hl = (a.Hl == a.Hq) ? g * G + hh : g;
                    const T* lr = as<T>(a.lmk) + (((size_t)b * a.Hl + hl) * nC + c) * D;
                    dqh[r] += a.scale * s_dsh[hh] * to_f32(lr[dd]);
                }
            }
        }
        __syncthreads();
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int o = tid + r * kBlock;
        if (o < G * D) {
            const int hh = o / D, dd = o % D;
            const size_t off = (((size_t)b * a.Hq + g * G + hh) * a.N + n) * D + dd;
            if (a.q_route) {
                as_mut<T>(a.dq)[off] = from_f32<T>(dq[r]);
                as_mut<T>(a.dq_route)[off] = from_f32<T>(dqh[r]);
            } else {
                as_mut<T>(a.dq)[off] = from_f32<T>(dq[r] + dqh[r]);
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Inverse index: (b, g, c) -> rows n whose selection holds c.
// ---------------------------------------------------------------------------
__global__ void k_fill_i32(int* p, size_t n, int v) {
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = v;
}

// Entries are processed per (b, g) in blocks of kInvRows rows; a block first
// counts its entries per chunk in LDS and then touches each global counter
// once, so global atomics scale with (blocks x chunks touched), not entries.
// Counters are kept per (chunk, row bucket): every list is the concatenation of
// its buckets' sub-lists in bucket order, so a consumer can take the entries of
// one chunk that fall in one range of rows (the chunk pass walks the buckets in
// order, so the query rows it gathers stay in L2).
// List entries are (n << 6) | slot (slot < K <= 64).
constexpr int kInvRows = 256;
constexpr int kInvHist = 8192;  // chunks counted in LDS; larger L falls back to global atomics
static_assert(kInvBucketRows % kInvRows == 0, "a block of rows lies in one bucket");

// (n: the row relative to a.n0)
__device__ __forceinline__ bool entry_valid(const InvArgs& a, const int32_t* irow, int slot, int n, int* c) {
    if (!idx_entry_valid(irow, slot, n_candidates(a.n0 + n, a.W))) return false;
    *c = irow[slot];
    return true;
}

// grid (ceil(N / kInvRows), B*Hkv); counts [bg][nR][nC] (a block's counters are
// contiguous: one bucket)
__global__ __launch_bounds__(kBlock) void k_inv_count(InvArgs a, int nR, int brows, int* counts) {
    __shared__ int s_hist[kInvHist];
    const int bg = blockIdx.y, n0 = blockIdx.x * kInvRows, tid = threadIdx.x;
    const int nC = a.L / kChunk, R = n0 / brows;
    const bool lds = nC <= kInvHist;
    int* gcnt = counts + (size_t)bg * nC * nR;
    if (lds)
        for (int c = tid; c < nC; c += kBlock) s_hist[c] = 0;
    __syncthreads();
    const int rows = min(kInvRows, a.N - n0);
    for (int e = tid; e < rows * a.K; e += kBlock) {
        const int n = n0 + e / a.K, slot = e % a.K;
        const int32_t* irow = a.idx + ((size_t)bg * a.Nrow + a.n0 + n) * a.K;
        int c;
        if (!entry_valid(a, irow, slot, n, &c)) continue;
        if (lds)
            atomicAdd(&s_hist[c], 1);
        else
            atomicAdd(&gcnt[R * nC + c], 1);
    }
    __syncthreads();
    if (lds)
        for (int c = tid; c < nC; c += kBlock)
            if (s_hist[c]) atomicAdd(&gcnt[R * nC + c], s_hist[c]);
}

__global__ __launch_bounds__(kBlock) void k_inv_fill(InvArgs a, int nR, int brows, const int* boff, int* cursor,
                                                     int* list) {
    __shared__ int s_hist[kInvHist];
    const int bg = blockIdx.y, n0 = blockIdx.x * kInvRows, tid = threadIdx.x;
    const int nC = a.L / kChunk, R = n0 / brows;
    const bool lds = nC <= kInvHist;
    int* gcur = cursor + (size_t)bg * nC * nR;
    const int* off = boff + (size_t)bg * (nC * nR + 1);
    int* lst = list + (size_t)bg * a.N * a.K;
    const int rows = min(kInvRows, a.N - n0);
    if (lds) {
        for (int c = tid; c < nC; c += kBlock) s_hist[c] = 0;
        __syncthreads();
        for (int e = tid; e < rows * a.K; e += kBlock) {
            const int n = n0 + e / a.K, slot = e % a.K;
            int c;
            if (entry_valid(a, a.idx + ((size_t)bg * a.Nrow + a.n0 + n) * a.K, slot, n, &c)) atomicAdd(&s_hist[c], 1);
        }
        __syncthreads();
        // reserve this block's range of every chunk it touches; s_hist becomes the running position
        for (int c = tid; c < nC; c += kBlock)
            if (s_hist[c]) s_hist[c] = off[c * nR + R] + atomicAdd(&gcur[R * nC + c], s_hist[c]);
        __syncthreads();
    }
    for (int e = tid; e < rows * a.K; e += kBlock) {
        const int n = n0 + e / a.K, slot = e % a.K;
        int c;
        if (!entry_valid(a, a.idx + ((size_t)bg * a.Nrow + a.n0 + n) * a.K, slot, n, &c)) continue;
        const int pos = lds ? atomicAdd(&s_hist[c], 1) : off[c * nR + R] + atomicAdd(&gcur[R * nC + c], 1);
        lst[pos] = (n << 6) | slot;
    }
}

// Exclusive prefix sum of one int per thread over a kBlock-thread block (wave
// scans by shuffles, then the wave totals); every thread gets the block total.
// Contains barriers: called by every thread of the block.
__device__ __forceinline__ int block_exclusive_scan(int x, int* s_wave, int* total) {
    const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
    int incl = x;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const int y = __shfl_up(incl, o, kWave);
        if (lane >= o) incl += y;
    }
    if (lane == kWave - 1) s_wave[w] = incl;
    __syncthreads();
    int before = 0, all = 0;
#pragma unroll
    for (int i = 0; i < kBlock / kWave; ++i) {
        const int t = s_wave[i];
        before += i < w ? t : 0;
        all += t;
    }
    __syncthreads();  // s_wave may be reused by the caller
    *total = all;
    return before + incl - x;
}

// one block per (b, g): exclusive scan of the nR x nC counts in chunk-major order
// into boff[nC * nR + 1], and each chunk's whole list into offsets[nC + 1]
__global__ __launch_bounds__(kBlock) void k_inv_scan(const int* counts, int* boff, int* offsets, int nC, int nR) {
    __shared__ int s_part[kBlock / kWave];
    const int bg = blockIdx.x, tid = threadIdx.x;
    const int M = nC * nR;
    const int per = (M + kBlock - 1) / kBlock;
    const int lo = min(M, tid * per), hi = min(M, lo + per);
    const int* cnt = counts + (size_t)bg * M;
    int* bo = boff + (size_t)bg * (M + 1);
    int* off = offsets + (size_t)bg * (nC + 1);
    int sum = 0;
    auto count = [&](int i) { return cnt[(i % nR) * nC + i / nR]; };  // i = c * nR + R
    for (int i = lo; i < hi; ++i) sum += count(i);
    int total;
    int run = block_exclusive_scan(sum, s_part, &total);
    if (tid == 0) {
        bo[M] = total;
        off[nC] = total;
    }
    for (int i = lo; i < hi; ++i) {
        bo[i] = run;
        if (i % nR == 0) off[i / nR] = run;
        run += count(i);
    }
}

InvLayout inv_layout(int B, int Hkv, int N, int L, int K, size_t base, int row_end) {
    const size_t bg = (size_t)B * Hkv, nC = (size_t)L / kChunk;
    InvLayout w;
    w.brows = kInvBucketRows;
    while ((size_t)w.brows * K < 64 * nC && w.brows < N) w.brows *= 2;
    w.nR = (N + w.brows - 1) / w.brows;
    const size_t M = nC * (size_t)w.nR;
    w.counts = align256(base);
    w.offsets = align256(w.counts + bg * M * sizeof(int));
    w.boff = align256(w.offsets + bg * (nC + 1) * sizeof(int));
    w.cursor = align256(w.boff + bg * (M + 1) * sizeof(int));
    w.list = align256(w.cursor + bg * M * sizeof(int));
    // A (chunk, bucket) sub-list of len entries makes ceil(len / kInvSeg) <= len / kInvSeg
    // + 1 items, and only the chunks c < n / kChunk of a bucket's last row n can
    // have entries there (a candidate chunk ends before the query): at most
    // (R + 1) * brows / kChunk sub-lists of bucket R are not empty; for a segment of
    // rows that starts later, bucket R's rows lie below row_end, whose candidate
    // chunks number at most row_end / kChunk + 1.
    size_t subl = 0;
    for (int R = 0; R < w.nR; ++R)
        subl += row_end < 0 ? std::min(nC, (size_t)(R + 1) * (w.brows / kChunk))
                            : std::min(nC, (size_t)row_end / kChunk + 1);
    w.max_work_bg = (size_t)N * K / kInvSeg + subl;
    w.work = align256(w.list + bg * (size_t)N * K * sizeof(int));
    w.nwork = align256(w.work + bg * w.max_work_bg * sizeof(int4));
    w.end = align256(w.nwork + bg * sizeof(int));
    return w;
}

// Work items of one (b, g) (one block each): its (chunk, bucket) sub-lists cut into
// segments of kInvSeg entries, bucket-major, so that the items in flight together
// work on one range of rows.
__global__ __launch_bounds__(kBlock) void k_inv_work(const int* boff, int nC, int nR, size_t max_work_bg, int4* work,
                                                     int* nwork) {
    __shared__ int s_part[kBlock / kWave];
    const int bg = blockIdx.x, tid = threadIdx.x;
    const int M = nC * nR;
    const int* bo = boff + (size_t)bg * (M + 1);
    int4* wk = work + (size_t)bg * max_work_bg;
    const int per = (M + kBlock - 1) / kBlock;
    const int lo = min(M, tid * per), hi = min(M, lo + per);
    auto nseg = [&](int i) {  // i = R * nC + c
        const int j = (i % nC) * nR + i / nC;
        return (bo[j + 1] - bo[j] + kInvSeg - 1) / kInvSeg;
    };
    int sum = 0;
    for (int i = lo; i < hi; ++i) sum += nseg(i);
    int total;
    int run = block_exclusive_scan(sum, s_part, &total);
    if (tid == 0) nwork[bg] = total;
    for (int i = lo; i < hi; ++i) {
        const int ns = nseg(i);
        for (int sgi = 0; sgi < ns; ++sgi) wk[run + sgi] = make_int4(i / nC, i % nC, sgi, 0);
        run += ns;
    }
}

void launch_inverse_index(const InvArgs& a, const InvLayout& w, void* ws, hipStream_t s, bool work_list) {
    char* base = static_cast<char*>(ws);
    int* counts = reinterpret_cast<int*>(base + w.counts);
    int* offsets = reinterpret_cast<int*>(base + w.offsets);
    int* boff = reinterpret_cast<int*>(base + w.boff);
    int* cursor = reinterpret_cast<int*>(base + w.cursor);
    int* list = reinterpret_cast<int*>(base + w.list);
    const int nC = a.L / kChunk;
    const size_t ncnt = (size_t)a.B * a.Hkv * nC * w.nR;
    const unsigned gc = (unsigned)((ncnt + kBlock - 1) / kBlock);
    const dim3 grows((a.N + kInvRows - 1) / kInvRows, a.B * a.Hkv);
    HILS_LAUNCH("k_fill_i32", k_fill_i32, dim3(gc), dim3(kBlock), 0, s, counts, ncnt, 0);
    HILS_LAUNCH("k_fill_i32", k_fill_i32, dim3(gc), dim3(kBlock), 0, s, cursor, ncnt, 0);
    HILS_LAUNCH("k_inv_count", k_inv_count, grows, dim3(kBlock), 0, s, a, w.nR, w.brows, counts);
    HILS_LAUNCH("k_inv_scan", k_inv_scan, dim3(a.B * a.Hkv), dim3(kBlock), 0, s, (const int*)counts, boff, offsets,
                nC, w.nR);
    HILS_LAUNCH("k_inv_fill", k_inv_fill, grows, dim3(kBlock), 0, s, a, w.nR, w.brows, (const int*)boff, cursor,
                list);
    if (work_list)
        HILS_LAUNCH("k_inv_work", k_inv_work, dim3(a.B * a.Hkv), dim3(kBlock), 0, s, (const int*)boff, nC, w.nR,
                    w.max_work_bg, reinterpret_cast<int4*>(base + w.work), reinterpret_cast<int*>(base + w.nwork));
}

// ---------------------------------------------------------------------------
// dk, dv of chunk c (and dk', db' of its landmark heads): one workgroup per (c, g, b).
// Phase A: rows n in [cS, (c+1)S + W - 2] whose local window covers keys of c.
// Phase B: rows that retrieved c (sorted ascending when the list fits kSortCap).
// ---------------------------------------------------------------------------
template <typename T, int D, int G>
__global__ __launch_bounds__(kBlock) void k_bwd_dkdv_chunks(BwdArgs a, const int* offsets, const int* list) {
    constexpr int RK = kChunk * D / kBlock;
    constexpr int RL = (G * D + kBlock - 1) / kBlock;
    __shared__ float s_k[kChunk][D + 1];
    __shared__ float s_v[kChunk][D + 1];
    __shared__ float s_q[G][D], s_qr[G][D], s_do[G][D], s_lm[G][D];
    __shared__ float s_cv[G][kChunk], s_cs[G][kChunk];
    __shared__ float s_dsh[G], s_L[G], s_db[G];
    __shared__ int s_list[kSortCap];

    const int tid = threadIdx.x, wave = wave_id(), lane = tid % kWave;
    const int c = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
    const int nC = a.L / kChunk;
    const int j0 = c * kChunk;
    const bool per_head_lmk = (a.Hl == a.Hq);
    const int nLH = per_head_lmk ? G : 1;
    const T* kb = as<T>(a.k) + ((size_t)b * a.Hkv + g) * a.L * D;
    const T* vb = as<T>(a.v) + ((size_t)b * a.Hkv + g) * a.L * D;
    const T* qr_base = as<T>(a.q_route ? a.q_route : a.q);

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
    for (int e = tid; e < nLH * D; e += kBlock) {
        const int lh = e / D, dd = e % D;
        const int hl = per_head_lmk ? g * G + lh : g;
        s_lm[lh][dd] = to_f32(as<T>(a.lmk)[(((size_t)b * a.Hl + hl) * nC + c) * D + dd]);
    }
    if (tid < G) s_db[tid] = 0.f;

    float dk[RK], dv[RK], dl[RL];
#pragma unroll
    for (int r = 0; r < RK; ++r) dk[r] = dv[r] = 0.f;
#pragma unroll
    for (int r = 0; r < RL; ++r) dl[r] = 0.f;

    auto process_row = [&](int n, bool retrieval) {
        __syncthreads();  // previous row's LDS readers are done
        for (int e = tid; e < G * D; e += kBlock) {
            const int hh = e / D, dd = e % D;
            const size_t off = (((size_t)b * a.Hq + g * G + hh) * a.N + n) * D + dd;
            s_q[hh][dd] = to_f32(as<T>(a.q)[off]);
            s_do[hh][dd] = to_f32(as<T>(a.dout)[off]);
            if (retrieval) s_qr[hh][dd] = to_f32(qr_base[off]);
        }
        if (tid < G) s_L[tid] = a.lse[((size_t)b * a.Hq + g * G + tid) * a.N + n];
        __syncthreads();
        const int nk = retrieval ? kChunk : min(n, j0 + kChunk - 1) - j0 + 1;
        for (int hh = wave; hh < G; hh += 4) {
            const size_t row = ((size_t)b * a.Hq + g * G + hh) * a.N + n;
            float ub = 0.f;
            for (int dd = lane; dd < D; dd += kWave) ub += s_do[hh][dd] * to_f32(as<T>(a.out)[row * D + dd]);
            ub = wave_sum(ub);
            const float L = s_L[hh];
            float s = -INFINITY, gv = 0.f;
            if (lane < nk) {
                float acc = 0.f, acc2 = 0.f;
#pragma unroll 16
                for (int dd = 0; dd < D; ++dd) {
                    acc += s_q[hh][dd] * s_k[lane][dd];
                    acc2 += s_do[hh][dd] * s_v[lane][dd];
                }
                s = a.scale * acc;
                gv = acc2;
            }
            float cv, cs;
            if (retrieval) {
                const float m = wave_max(s);
                const float l = wave_sum(fexp(s - m));
                const float p = fexp(s - (m + __logf(l)));
                const float uc = wave_sum(p * gv);
                const int lh = per_head_lmk ? hh : 0;
                const int hl = per_head_lmk ? g * G + hh : g;
                float acc = 0.f;
                for (int dd = lane; dd < D; dd += kWave) acc += s_qr[hh][dd] * s_lm[lh][dd];
                acc = wave_sum(acc);
                const float sh = a.scale * acc + (a.bias ? a.bias[((size_t)b * a.Hl + hl) * nC + c] : 0.f);
                const float al = fexp(sh - L);
                cv = al * p;
                cs = al * p * (gv - uc);
                if (lane == 0) s_dsh[hh] = al * (uc - ub);
            } else {
                const float w = lane < nk ? fexp(s - L) : 0.f;
                cv = w;
                cs = w * (gv - ub);
            }
            s_cv[hh][lane] = cv;
            s_cs[hh][lane] = cs;
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < RK; ++r) {
            const int e = tid + r * kBlock;
            const int j = e / D, dd = e % D;
            float av = 0.f, ak = 0.f;
#pragma unroll
            for (int hh = 0; hh < G; ++hh) {
                av += s_cv[hh][j] * s_do[hh][dd];
                ak += s_cs[hh][j] * s_q[hh][dd];
            }
            dv[r] += av;
            dk[r] += a.scale * ak;
        }
        if (retrieval) {
#pragma unroll
            for (int r = 0; r < RL; ++r) {
                const int e = tid + r * kBlock;
                if (e < nLH * D) {
                    const int lh = e / D, dd = e % D;
                    float acc = 0.f;
                    if (per_head_lmk) {
                        acc = s_dsh[lh] * s_qr[lh][dd];
                    } else {
#pragma unroll
                        for (int hh = 0; hh < G; ++hh) acc += s_dsh[hh] * s_qr[hh][dd];
                    }
                    dl[r] += a.scale * acc;
                }
            }
            if (tid == 0) {
                for (int hh = 0; hh < G; ++hh) s_db[per_head_lmk ? hh : 0] += s_dsh[hh];
            }
        }
    };

    // phase A: local windows covering this chunk
    const int n_hi = min(a.N - 1, j0 + kChunk + a.W - 2);
    for (int n = j0; n <= n_hi; ++n) process_row(n, false);

    // phase B: retrievals of this chunk
    const size_t bg = (size_t)b * a.Hkv + g;
    const int beg = offsets[bg * (nC + 1) + c];
    const int len = offsets[bg * (nC + 1) + c + 1] - beg;
    const int* seg = list + bg * a.N * a.K + beg;
    if (len <= kSortCap) {
        __syncthreads();
        int P = 1;
        while (P < len) P <<= 1;
        for (int t = tid; t < P; t += kBlock) s_list[t] = t < len ? seg[t] : 0x7fffffff;
        __syncthreads();
        for (int kk = 2; kk <= P; kk <<= 1) {
            for (int jj = kk >> 1; jj > 0; jj >>= 1) {
                for (int t = tid; t < P; t += kBlock) {
                    const int u = t ^ jj;
                    if (u > t) {
                        const int x = s_list[t], y = s_list[u];
                        const bool up = (t & kk) == 0;
                        if ((x > y) == up) {
                            s_list[t] = y;
                            s_list[u] = x;
                        }
                    }
                }
                __syncthreads();
            }
        }
        for (int t = 0; t < len; ++t) process_row(s_list[t] >> 6, true);
    } else {
        for (int t = 0; t < len; ++t) process_row(seg[t] >> 6, true);
    }
    __syncthreads();

    T* dkp = as_mut<T>(a.dk) + (bg * a.L + j0) * D;
    T* dvp = as_mut<T>(a.dv) + (bg * a.L + j0) * D;
#pragma unroll
    for (int r = 0; r < RK; ++r) {
        const int e = tid + r * kBlock;
        dkp[e] = from_f32<T>(dk[r]);
        dvp[e] = from_f32<T>(dv[r]);
    }
#pragma unroll
    for (int r = 0; r < RL; ++r) {
        const int e = tid + r * kBlock;
        if (e < nLH * D) {
            const int lh = e / D, dd = e % D;
            const int hl = per_head_lmk ? g * G + lh : g;
            as_mut<T>(a.dlmk)[(((size_t)b * a.Hl + hl) * nC + c) * D + dd] = from_f32<T>(dl[r]);
        }
    }
    if (a.dbias && tid < nLH) {
        const int hl = per_head_lmk ? g * G + tid : g;
        a.dbias[((size_t)b * a.Hl + hl) * nC + c] = s_db[tid];
    }
}

struct BwdRun {
    template <typename T, int D, int G>
    static hipError_t run(const BwdArgs& a, hipStream_t s) {
        if constexpr (!std::is_same<T, float>::value) return hipErrorInvalidValue;  // bf16: launch_bwd_mfma
        const InvLayout w = inv_layout(a.B, a.Hkv, a.N, a.L, a.K, 0);
        char* ws = static_cast<char*>(a.ws);
        const int* offsets = reinterpret_cast<const int*>(ws + w.offsets);
        const int* list = reinterpret_cast<const int*>(ws + w.list);
        const int nC = a.L / kChunk;
        const InvArgs ia{a.idx, a.B, a.Hkv, a.N, a.K, a.W, a.L, 0, a.N};
        launch_inverse_index(ia, w, a.ws, s, false);
        HILS_LAUNCH("k_bwd_dq_rows", (k_bwd_dq_rows<T, D, G>), dim3(a.N, a.Hkv, a.B), dim3(kBlock), 0, s, a);
        HILS_LAUNCH("k_bwd_dkdv_chunks", (k_bwd_dkdv_chunks<T, D, G>), dim3(nC, a.Hkv, a.B), dim3(kBlock), 0, s, a,
                           offsets, list);
        return hipGetLastError();
    }
};

hipError_t launch_bwd(const BwdArgs& a, hipStream_t s) {
    if (a.bf16) return launch_bwd_mfma(a, s);
    return dispatch<BwdRun>(0, a.d, a.Hq / a.Hkv, a, s);
}

}  // namespace hils
