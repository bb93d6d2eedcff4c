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
    void* out;
    float* lse;
    int32_t* idx;
    int B, Hq, Hkv, Hl, N, L, d, K, W;
    float scale;
    int bf16;      // storage dtype
    int decode;    // 1: query n = 0 of sequence b sits at seqlens[b]-1
    int given_idx; // 1: consume idx
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

// Workspace layout of the backward (byte offsets from ws).
struct BwdWorkspace {
    size_t counts, offsets, cursor, list, total;
};
BwdWorkspace bwd_workspace_layout(int B, int Hkv, int N, int L, int K);

size_t decode_workspace_bytes(int B, int Hkv, int G, int d, int L, int K, int W);

hipError_t launch_prefill_fwd(const FwdArgs& a, hipStream_t s);
hipError_t launch_decode_fwd(const FwdArgs& a, hipStream_t s);
hipError_t launch_bwd(const BwdArgs& a, hipStream_t s);

}  // namespace hils
