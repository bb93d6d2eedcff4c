// Host-side launch interface between the C-ABI layer and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace hils {

// Geometry and pointers of one forward call (prefill or decode).
struct FwdArgs {
    const void* q;
    const void* k;
    const void* v;
    const void* lmk;
    const float* bias;      // nullable
    const void* q_route;    // nullable: q^ = q
    const int32_t* seqlens; // decode only, nullable: L
    const int32_t* block_table; // decode only, nullable: contiguous caches; else [B, L/S] page ids
    int num_pages;              // pages in the pools when paged
    void* out;
    float* lse;
    int32_t* idx;
    int B, Hq, Hkv, Hl, N, L, d, K, W;
    float scale;
    int bf16;      // storage dtype
    int decode;    // 1: query n of sequence b sits at len_b - N + n (len_b = seqlens[b] in [N, L])
    int given_idx; // 1: consume idx
    int head_norm; // 1: rank by per-head normalised scores
    int union_pack; // 1: prefill chunk terms by the union of each tile's selections
    void* ws;
    size_t ws_bytes;
};

struct BwdArgs {
    const void* dout;
    const void* q;
    const void* k;
    const void* v;
    const void* lmk;
    const float* bias;
    const void* q_route;
    const void* out;
    const float* lse;
    const int32_t* idx;
    void* dq;
    void* dk;
    void* dv;
    void* dlmk;
    float* dbias;     // nullable
    void* dq_route;   // nullable: folded into dq
    int B, Hq, Hkv, Hl, N, L, d, K, W;
    float scale;
    int bf16;
    void* ws;
    size_t ws_bytes;
};

// Landmark compression (Prop. 3.1), forward and backward.
struct LmkArgs {
    const void* lq;      // landmark queries q'_c   [B, Hl, L/S, d] ([Hl, d] if shared)
    const void* k;       // keys                    [B, Hkv, L, d]
    void* lmk;           // fwd out: k'_c           [B, Hl, L/S, d]
    float* bias;         // fwd out: b'_c           [B, Hl, L/S]
    const void* dlmk;    // bwd in:  dL/dk'_c
    const float* dbias;  // bwd in:  dL/db'_c (nullable: 0)
    void* dlq;           // bwd out: dL/dq'_c       [B, Hl, L/S, d] ([Hl, d] if shared)
    void* dk;            // bwd out: dL/dk          [B, Hkv, L, d]
    float* ws;           // shared query: per-chunk dq' in fp32 [B, Hl, L/S, d]
    int B, Hkv, Hl, L, d;
    float scale;
    int bf16;
    int shared;          // one landmark query per head for every chunk (Sec. 4.1)
};

inline size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Optional per-kernel timing (hils_timing_enable): every launch is bracketed by
// HIP events on its stream when timing is on for the calling thread.
bool timing_on();
void timing_begin(const char* name, hipStream_t s);
void timing_end(hipStream_t s);

#define HILS_LAUNCH(NAME, KERNEL, GRID, BLOCK, LDS, STREAM, ...)              \
    do {                                                                       \
        const bool hils_timed_ = ::hils::timing_on();                          \
        if (hils_timed_) ::hils::timing_begin(NAME, STREAM);                   \
        hipLaunchKernelGGL(KERNEL, GRID, BLOCK, LDS, STREAM, __VA_ARGS__);     \
        if (hils_timed_) ::hils::timing_end(STREAM);                           \
    } while (0)

// Inverse index of a selection: for every (b, g, chunk) the rows n that chose it.
// The inverse index of rows n0 .. n0 + N - 1 of idx ([B, Hkv, Nrow, K]); list
// entries hold the row relative to n0.
struct InvArgs {
    const int32_t* idx;
    int B, Hkv, N, K, W, L;
    int n0, Nrow;
};
struct InvLayout {
    size_t counts, offsets, cursor, list;  // byte offsets from the workspace base
    size_t boff;    // [bg][nC * nR + 1]: start of the (chunk, row bucket) sub-lists
    size_t work;    // [bg][max_work_bg] work items (row bucket, chunk, segment, 0)
    size_t nwork;   // [bg] number of work items of each (b, g)
    size_t end;
    int nR;              // row buckets
    int brows;           // rows per bucket (a multiple of kInvBucketRows)
    size_t max_work_bg;  // upper bound of the work items of one (b, g)
};
constexpr int kInvSeg = 256;          // list entries per work item
// Rows per bucket, at least: a chunk's list is ordered by bucket.  Buckets grow
// (doubling) until a (chunk, bucket) sub-list holds about 64 entries on average
// (brows * K >= 64 * L/S), so that long sequences keep full work items.
constexpr int kInvBucketRows = 2048;
// row_end >= 0: the layout serves segments of up to N rows anywhere below row row_end
// (the work-item bound then allows every candidate chunk of those rows per bucket)
InvLayout inv_layout(int B, int Hkv, int N, int L, int K, size_t base, int row_end = -1);
// Every (b, g, chunk) list is sorted by row bucket (the sub-list of bucket R starts
// at boff[c * nR + R]); offsets[c] .. offsets[c + 1] bound the whole list.
// work_list = false skips the work items (consumers that walk whole lists do not
// read them).
void launch_inverse_index(const InvArgs& a, const InvLayout& w, void* ws, hipStream_t s, bool work_list = true);

// Workspace layout of the backward (byte offsets from ws).
struct BwdWorkspace {
    size_t counts, offsets, cursor, list, total;
};
BwdWorkspace bwd_workspace_layout(int B, int Hkv, int N, int L, int K);

// Compute units of the current device (a host-side attribute query; nothing cached).
int device_cus();

size_t decode_workspace_bytes(int B, int N, int Hkv, int G, int d, int L, int K, int W, int head_norm);

size_t prefill_workspace_bytes(int B, int Hq, int Hkv, int N, int L, int d, int K, int bf16, int union_pack);
// The chunk-major prefill's cap on the records of one segment of rows (bytes): set
// (bytes > 0) and read; returns the previous value.
size_t prefill_record_cap(size_t bytes);

hipError_t launch_prefill_fwd(const FwdArgs& a, hipStream_t s);
hipError_t launch_prefill_rows(const FwdArgs& a, hipStream_t s);  // fp32 storage
hipError_t launch_decode_fwd(const FwdArgs& a, hipStream_t s);
// The no-allocation decode's file-scope device array: its size, and its device
// address on the current device (looked up once per device).
size_t decode_noalloc_capacity();
hipError_t decode_noalloc_scratch(void** ptr);
hipError_t launch_landmark_fwd(const LmkArgs& a, hipStream_t s);
hipError_t launch_landmark_bwd(const LmkArgs& a, hipStream_t s);
size_t landmark_workspace_bytes(int B, int Hl, int nC, int d, bool shared);
hipError_t launch_bwd(const BwdArgs& a, hipStream_t s);       // fp32 storage
hipError_t launch_bwd_mfma(const BwdArgs& a, hipStream_t s);  // bf16 storage
size_t bwd_mfma_workspace_bytes(int B, int Hq, int Hkv, int N, int L, int d, int K);

}  // namespace hils
