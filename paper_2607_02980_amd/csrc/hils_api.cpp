// C-ABI of libhils.so: argument validation, workspace sizing and dispatch.
// Every check runs on the host before any HIP call.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <string>
#include <vector>

#include "../../include/hils.h"
#include "hils_internal.hpp"

namespace {

thread_local std::string g_err;

struct TimedLaunch {
    const char* name;
    hipEvent_t e0, e1;
};
thread_local bool g_timing = false;
thread_local std::vector<TimedLaunch> g_launches;

void release_launches() {
    for (auto& t : g_launches) {
        (void)hipEventDestroy(t.e0);
        (void)hipEventDestroy(t.e1);
    }
    g_launches.clear();
}

int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int ok() {
    g_err.clear();
    return HILS_OK;
}

int check_params(const hils_params* p, int op) {
    if (!p) return fail(HILS_ERR_INVALID, "params is NULL");
    if (op != HILS_OP_PREFILL && op != HILS_OP_DECODE && op != HILS_OP_BWD && op != HILS_OP_LANDMARK)
        return fail(HILS_ERR_INVALID, "unknown op %d", op);
    if (p->B < 1 || p->Hq < 1 || p->Hkv < 1 || p->N < 1 || p->L < 1 || p->d < 1)
        return fail(HILS_ERR_INVALID, "B, Hq, Hkv, N, L and d must be >= 1 (B=%d Hq=%d Hkv=%d N=%d L=%d d=%d)",
                    p->B, p->Hq, p->Hkv, p->N, p->L, p->d);
    if (p->chunk < 1 || p->topk < 1 || p->window < 1)
        return fail(HILS_ERR_INVALID, "chunk, topk and window must be >= 1 (chunk=%d topk=%d window=%d)", p->chunk,
                    p->topk, p->window);
    if (p->Hq % p->Hkv) return fail(HILS_ERR_INVALID, "Hq=%d is not a multiple of Hkv=%d", p->Hq, p->Hkv);
    if (p->Hl != p->Hq && p->Hl != p->Hkv)
        return fail(HILS_ERR_INVALID, "Hl=%d must equal Hq=%d or Hkv=%d", p->Hl, p->Hq, p->Hkv);
    if (p->L % p->chunk) return fail(HILS_ERR_INVALID, "L=%d is not a multiple of chunk=%d", p->L, p->chunk);
    // the field's bits as an int: a C caller may store any value there, and loading
    // one outside the enumerators as the enum type is undefined in C++
    int dtype_raw = 0;
    static_assert(sizeof(p->dtype) == sizeof(int), "hils_dtype has the size of an int");
    memcpy(&dtype_raw, &p->dtype, sizeof dtype_raw);
    if (dtype_raw != HILS_F32 && dtype_raw != HILS_BF16) return fail(HILS_ERR_INVALID, "unknown dtype %d", dtype_raw);
    if (!isfinite(p->scale)) return fail(HILS_ERR_INVALID, "scale is not finite");
    if (p->flags & ~(HILS_FLAG_GIVEN_IDX | HILS_FLAG_SHARED_LMK_QUERY | HILS_FLAG_HEAD_NORM_SELECT |
                     HILS_FLAG_UNION_PACKING))
        return fail(HILS_ERR_INVALID, "unknown flags 0x%x", p->flags);
    if ((p->flags & HILS_FLAG_HEAD_NORM_SELECT) && op == HILS_OP_LANDMARK)
        return fail(HILS_ERR_INVALID, "HILS_FLAG_HEAD_NORM_SELECT does not apply to the landmark compression");
    if ((p->flags & HILS_FLAG_SHARED_LMK_QUERY) && op != HILS_OP_LANDMARK)
        return fail(HILS_ERR_INVALID, "HILS_FLAG_SHARED_LMK_QUERY applies to the landmark compression only");
    if ((p->flags & HILS_FLAG_GIVEN_IDX) && op == HILS_OP_LANDMARK)
        return fail(HILS_ERR_INVALID, "HILS_FLAG_GIVEN_IDX does not apply to the landmark compression");
    if (op == HILS_OP_DECODE && p->N > p->L)
        return fail(HILS_ERR_INVALID, "decode needs N <= L new queries per sequence (N=%d L=%d)", p->N, p->L);
    if (op == HILS_OP_DECODE && (long)p->B * p->N > 65535)
        return fail(HILS_ERR_INVALID, "decode needs B * N <= 65535 (B=%d N=%d)", p->B, p->N);
    if (op != HILS_OP_DECODE && op != HILS_OP_LANDMARK && p->N > p->L)
        return fail(HILS_ERR_INVALID, "prefill/backward need N <= L (N=%d L=%d)", p->N, p->L);
    if (p->B > 65535 || p->Hkv > 65535) return fail(HILS_ERR_INVALID, "B and Hkv must be <= 65535");
    if (op == HILS_OP_BWD && (p->flags & HILS_FLAG_GIVEN_IDX))
        return fail(HILS_ERR_INVALID, "HILS_FLAG_GIVEN_IDX is a forward flag (the backward always reads idx)");
    // kernel coverage
    if (p->chunk != 64) return fail(HILS_ERR_UNSUPPORTED, "chunk=%d: kernels exist for chunk 64 only", p->chunk);
    if (p->d != 64 && p->d != 128) return fail(HILS_ERR_UNSUPPORTED, "d=%d: kernels exist for d in {64, 128}", p->d);
    const int G = p->Hq / p->Hkv;
    if (G != 1 && G != 2 && G != 4 && G != 8)
        return fail(HILS_ERR_UNSUPPORTED, "group size G=%d: kernels exist for G in {1, 2, 4, 8}", G);
    if (p->topk > 64) return fail(HILS_ERR_UNSUPPORTED, "topk=%d: kernels exist for topk <= 64", p->topk);
    if (op == HILS_OP_DECODE && p->window > 4032)
        return fail(HILS_ERR_UNSUPPORTED, "window=%d: the decode kernels cover windows <= 4032", p->window);
    return HILS_OK;
}

size_t ws_bytes_for(const hils_params* p, int op) {
    switch (op) {
        case HILS_OP_LANDMARK:
            return hils::landmark_workspace_bytes(p->B, p->Hl, p->L / p->chunk, p->d,
                                                  (p->flags & HILS_FLAG_SHARED_LMK_QUERY) != 0);
        case HILS_OP_BWD:
            if (p->dtype == HILS_BF16)
                return hils::bwd_mfma_workspace_bytes(p->B, p->Hq, p->Hkv, p->N, p->L, p->d, p->topk);
            return hils::bwd_workspace_layout(p->B, p->Hkv, p->N, p->L, p->topk).total;
        case HILS_OP_DECODE:
            return hils::decode_workspace_bytes(p->B, p->N, p->Hkv, p->Hq / p->Hkv, p->d, p->L, p->topk, p->window,
                                                (p->flags & HILS_FLAG_HEAD_NORM_SELECT) != 0);
        default:
            return hils::prefill_workspace_bytes(p->B, p->Hq, p->Hkv, p->N, p->L, p->d, p->topk,
                                                 p->dtype == HILS_BF16,
                                                 (p->flags & HILS_FLAG_UNION_PACKING) != 0);
    }
}

int check_ws(const hils_params* p, int op, const void* ws, size_t bytes) {
    const size_t need = ws_bytes_for(p, op);
    if (need == 0) return HILS_OK;
    if (!ws) return fail(HILS_ERR_WORKSPACE, "workspace is NULL but %zu bytes are needed", need);
    if (bytes < need) return fail(HILS_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", bytes, need);
    return HILS_OK;
}

int hip_status(hipError_t e, const char* what) {
    if (e != hipSuccess) return fail(HILS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
    return ok();
}

#define REQUIRE(ptr) \
    if (!(ptr)) return fail(HILS_ERR_INVALID, "required pointer '%s' is NULL", #ptr)

hils::FwdArgs fwd_args(const hils_params* p, const void* q, const void* k, const void* v, const void* lmk,
                       const float* bias, const void* q_route, const int32_t* seqlens, void* out, float* lse,
                       int32_t* idx, void* ws, size_t ws_bytes, int decode) {
    hils::FwdArgs a;
    a.q = q; a.k = k; a.v = v; a.lmk = lmk; a.bias = bias; a.q_route = q_route; a.seqlens = seqlens;
    a.block_table = nullptr; a.num_pages = 0;
    a.out = out; a.lse = lse; a.idx = idx;
    a.B = p->B; a.Hq = p->Hq; a.Hkv = p->Hkv; a.Hl = p->Hl; a.N = p->N; a.L = p->L; a.d = p->d;
    a.K = p->topk; a.W = p->window; a.scale = p->scale;
    a.bf16 = p->dtype == HILS_BF16;
    a.decode = decode;
    a.given_idx = (p->flags & HILS_FLAG_GIVEN_IDX) ? 1 : 0;
    a.head_norm = (p->flags & HILS_FLAG_HEAD_NORM_SELECT) ? 1 : 0;
    a.union_pack = (p->flags & HILS_FLAG_UNION_PACKING) ? 1 : 0;
    a.ws = ws; a.ws_bytes = ws_bytes;
    return a;
}

}  // namespace

namespace hils {
bool timing_on() { return g_timing; }
void timing_begin(const char* name, hipStream_t s) {
    TimedLaunch t{name, nullptr, nullptr};
    if (hipEventCreate(&t.e0) != hipSuccess || hipEventCreate(&t.e1) != hipSuccess) return;
    (void)hipEventRecord(t.e0, s);
    g_launches.push_back(t);
}
void timing_end(hipStream_t s) {
    if (!g_launches.empty()) (void)hipEventRecord(g_launches.back().e1, s);
}
}  // namespace hils

extern "C" {

int hils_timing_enable(int on) {
    g_timing = on != 0;
    if (!g_timing) release_launches();
    return ok();
}

int hils_timing_read(char* names, size_t names_len, float* total_ms, int* launches, int max_kernels,
                     int* n_kernels) {
    if (!n_kernels) return fail(HILS_ERR_INVALID, "n_kernels is NULL");
    std::vector<std::string> order;
    std::vector<float> tot;
    std::vector<int> cnt;
    for (auto& t : g_launches) {
        float ms = 0.f;
        if (hipEventSynchronize(t.e1) != hipSuccess || hipEventElapsedTime(&ms, t.e0, t.e1) != hipSuccess) {
            release_launches();
            return fail(HILS_ERR_HIP, "reading kernel timing events failed");
        }
        size_t k = 0;
        while (k < order.size() && order[k] != t.name) ++k;
        if (k == order.size()) {
            order.push_back(t.name);
            tot.push_back(0.f);
            cnt.push_back(0);
        }
        tot[k] += ms;
        cnt[k] += 1;
    }
    release_launches();
    *n_kernels = (int)order.size();
    std::string joined;
    for (size_t k = 0; k < order.size() && (int)k < max_kernels; ++k) {
        if (total_ms) total_ms[k] = tot[k];
        if (launches) launches[k] = cnt[k];
        joined += order[k];
        joined += '\n';
    }
    if (names && names_len) {
        const size_t n = joined.size() < names_len - 1 ? joined.size() : names_len - 1;
        memcpy(names, joined.data(), n);
        names[n] = 0;
    }
    return ok();
}


int hils_version(void) { return 100; }

size_t hils_prefill_record_cap(size_t bytes) { return hils::prefill_record_cap(bytes); }

const char* hils_last_error(void) { return g_err.c_str(); }

int hils_workspace_size(const hils_params* p, int op, size_t* bytes) {
    int rc = check_params(p, op);
    if (rc) return rc;
    if (!bytes) return fail(HILS_ERR_INVALID, "bytes is NULL");
    *bytes = ws_bytes_for(p, op);
    return ok();
}

int hils_prefill_fwd(const hils_params* p, const void* q, const void* k, const void* v, const void* lmk,
                     const float* lmk_bias, const void* q_route, void* out, float* lse, int32_t* idx,
                     void* workspace, size_t ws_bytes, void* stream) {
    int rc = check_params(p, HILS_OP_PREFILL);
    if (rc) return rc;
    REQUIRE(q); REQUIRE(k); REQUIRE(v); REQUIRE(lmk); REQUIRE(out); REQUIRE(lse); REQUIRE(idx);
    rc = check_ws(p, HILS_OP_PREFILL, workspace, ws_bytes);
    if (rc) return rc;
    const hils::FwdArgs a = fwd_args(p, q, k, v, lmk, lmk_bias, q_route, nullptr, out, lse, idx, workspace,
                                     ws_bytes, 0);
    return hip_status(hils::launch_prefill_fwd(a, (hipStream_t)stream), "hils_prefill_fwd launch");
}

int hils_decode_fwd(const hils_params* p, const void* q, const void* k_cache, const void* v_cache,
                    const void* lmk_cache, const float* lmk_bias, const void* q_route, const int32_t* seqlens,
                    void* out, float* lse, int32_t* idx, void* workspace, size_t ws_bytes, void* stream) {
    int rc = check_params(p, HILS_OP_DECODE);
    if (rc) return rc;
    REQUIRE(q); REQUIRE(k_cache); REQUIRE(v_cache); REQUIRE(lmk_cache); REQUIRE(out); REQUIRE(lse); REQUIRE(idx);
    rc = check_ws(p, HILS_OP_DECODE, workspace, ws_bytes);
    if (rc) return rc;
    const hils::FwdArgs a = fwd_args(p, q, k_cache, v_cache, lmk_cache, lmk_bias, q_route, seqlens, out, lse, idx,
                                     workspace, ws_bytes, 1);
    return hip_status(hils::launch_decode_fwd(a, (hipStream_t)stream), "hils_decode_fwd launch");
}

int hils_decode_fwd_noalloc(const hils_params* p, const void* q, const void* k_cache, const void* v_cache,
                            const void* lmk_cache, const float* lmk_bias, const void* q_route,
                            const int32_t* seqlens, void* out, float* lse, int32_t* idx, void* stream) {
    int rc = check_params(p, HILS_OP_DECODE);
    if (rc) return rc;
    REQUIRE(q); REQUIRE(k_cache); REQUIRE(v_cache); REQUIRE(lmk_cache); REQUIRE(out); REQUIRE(lse); REQUIRE(idx);
    const size_t need = ws_bytes_for(p, HILS_OP_DECODE);
    const size_t cap = hils::decode_noalloc_capacity();
    if (need > cap)
        return fail(HILS_ERR_WORKSPACE,
                    "hils_decode_fwd_noalloc: this call needs %zu bytes of workspace, above the library's fixed "
                    "%zu-byte array (use hils_decode_fwd with a workspace, or fewer sequences/new tokens)",
                    need, cap);
    void* ws = nullptr;
    rc = hip_status(hils::decode_noalloc_scratch(&ws), "hils_decode_fwd_noalloc: device address of the array");
    if (rc) return rc;
    const hils::FwdArgs a = fwd_args(p, q, k_cache, v_cache, lmk_cache, lmk_bias, q_route, seqlens, out, lse, idx,
                                     ws, cap, 1);
    return hip_status(hils::launch_decode_fwd(a, (hipStream_t)stream), "hils_decode_fwd_noalloc launch");
}

int hils_decode_paged_fwd(const hils_params* p, const void* q, const void* k_pages, const void* v_pages,
                          const void* lmk_pages, const float* bias_pages, const void* q_route,
                          const int32_t* block_table, int num_pages, const int32_t* seqlens, void* out, float* lse,
                          int32_t* idx, void* workspace, size_t ws_bytes, void* stream) {
    int rc = check_params(p, HILS_OP_DECODE);
    if (rc) return rc;
    REQUIRE(q); REQUIRE(k_pages); REQUIRE(v_pages); REQUIRE(lmk_pages); REQUIRE(block_table);
    REQUIRE(out); REQUIRE(lse); REQUIRE(idx);
    if (num_pages < 1) return fail(HILS_ERR_INVALID, "num_pages must be >= 1 (got %d)", num_pages);
    rc = check_ws(p, HILS_OP_DECODE, workspace, ws_bytes);
    if (rc) return rc;
    hils::FwdArgs a = fwd_args(p, q, k_pages, v_pages, lmk_pages, bias_pages, q_route, seqlens, out, lse, idx,
                               workspace, ws_bytes, 1);
    a.block_table = block_table;
    a.num_pages = num_pages;
    return hip_status(hils::launch_decode_fwd(a, (hipStream_t)stream), "hils_decode_paged_fwd launch");
}

int hils_bwd(const hils_params* p, const void* dout, const void* q, const void* k, const void* v, const void* lmk,
             const float* lmk_bias, const void* q_route, const void* out, const float* lse, const int32_t* idx,
             void* dq, void* dk, void* dv, void* dlmk, float* dlmk_bias, void* dq_route, void* workspace,
             size_t ws_bytes, void* stream) {
    int rc = check_params(p, HILS_OP_BWD);
    if (rc) return rc;
    REQUIRE(dout); REQUIRE(q); REQUIRE(k); REQUIRE(v); REQUIRE(lmk); REQUIRE(out); REQUIRE(lse); REQUIRE(idx);
    REQUIRE(dq); REQUIRE(dk); REQUIRE(dv); REQUIRE(dlmk);
    if (q_route && !dq_route)
        return fail(HILS_ERR_INVALID, "q_route is given, so dq_route must be non-NULL");
    rc = check_ws(p, HILS_OP_BWD, workspace, ws_bytes);
    if (rc) return rc;
    hils::BwdArgs a;
    a.dout = dout; a.q = q; a.k = k; a.v = v; a.lmk = lmk; a.bias = lmk_bias; a.q_route = q_route;
    a.out = out; a.lse = lse; a.idx = idx;
    a.dq = dq; a.dk = dk; a.dv = dv; a.dlmk = dlmk; a.dbias = dlmk_bias; a.dq_route = q_route ? dq_route : nullptr;
    a.B = p->B; a.Hq = p->Hq; a.Hkv = p->Hkv; a.Hl = p->Hl; a.N = p->N; a.L = p->L; a.d = p->d;
    a.K = p->topk; a.W = p->window; a.scale = p->scale;
    a.bf16 = p->dtype == HILS_BF16;
    a.ws = workspace; a.ws_bytes = ws_bytes;
    return hip_status(hils::launch_bwd(a, (hipStream_t)stream), "hils_bwd launch");
}

static hils::LmkArgs lmk_args(const hils_params* p) {
    hils::LmkArgs a = {};
    a.B = p->B; a.Hkv = p->Hkv; a.Hl = p->Hl; a.L = p->L; a.d = p->d;
    a.scale = p->scale;
    a.bf16 = p->dtype == HILS_BF16;
    a.shared = (p->flags & HILS_FLAG_SHARED_LMK_QUERY) != 0;
    return a;
}

int hils_landmark_fwd(const hils_params* p, const void* lq, const void* k, void* lmk, float* lmk_bias,
                      void* stream) {
    int rc = check_params(p, HILS_OP_LANDMARK);
    if (rc) return rc;
    REQUIRE(lq); REQUIRE(k); REQUIRE(lmk); REQUIRE(lmk_bias);
    hils::LmkArgs a = lmk_args(p);
    a.lq = lq; a.k = k; a.lmk = lmk; a.bias = lmk_bias;
    return hip_status(hils::launch_landmark_fwd(a, (hipStream_t)stream), "hils_landmark_fwd launch");
}

int hils_landmark_bwd(const hils_params* p, const void* lq, const void* k, const void* dlmk,
                      const float* dlmk_bias, void* dlq, void* dk, void* workspace, size_t ws_bytes,
                      void* stream) {
    int rc = check_params(p, HILS_OP_LANDMARK);
    if (rc) return rc;
    REQUIRE(lq); REQUIRE(k); REQUIRE(dlmk); REQUIRE(dlq); REQUIRE(dk);
    rc = check_ws(p, HILS_OP_LANDMARK, workspace, ws_bytes);
    if (rc) return rc;
    hils::LmkArgs a = lmk_args(p);
    a.lq = lq; a.k = k; a.dlmk = dlmk; a.dbias = dlmk_bias; a.dlq = dlq; a.dk = dk;
    a.ws = static_cast<float*>(workspace);
    return hip_status(hils::launch_landmark_bwd(a, (hipStream_t)stream), "hils_landmark_bwd launch");
}

}  // extern "C"
