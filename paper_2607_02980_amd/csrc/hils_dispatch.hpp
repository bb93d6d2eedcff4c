// Compile-time dispatch over (storage type, head dim D, group size G).
#pragma once

#include <hip/hip_runtime.h>

#include "hils_device.hpp"

namespace hils {

// Calls F::template run<T, D, G>(args...) for the runtime (bf16, d, G); returns
// hipErrorInvalidValue for combinations without kernels (the host API rejects
// them earlier with HILS_ERR_UNSUPPORTED).
template <typename F, typename... A>
hipError_t dispatch(int bf16_storage, int d, int G, A&&... args) {
#define HILS_CASE(TT, DD, GG) \
    if (d == DD && G == GG) return F::template run<TT, DD, GG>(args...);
#define HILS_CASES(TT)                                                                        \
    HILS_CASE(TT, 64, 1) HILS_CASE(TT, 64, 2) HILS_CASE(TT, 64, 4) HILS_CASE(TT, 64, 8)       \
    HILS_CASE(TT, 128, 1) HILS_CASE(TT, 128, 2) HILS_CASE(TT, 128, 4) HILS_CASE(TT, 128, 8)
    if (bf16_storage) {
        HILS_CASES(bf16)
    } else {
        HILS_CASES(float)
    }
#undef HILS_CASES
#undef HILS_CASE
    return hipErrorInvalidValue;
}

template <typename T>
__device__ __forceinline__ const T* as(const void* p) {
    return reinterpret_cast<const T*>(p);
}
template <typename T>
__device__ __forceinline__ T* as_mut(void* p) {
    return reinterpret_cast<T*>(p);
}

// idx entry `slot` of a selection row is used iff it names a candidate chunk
// (0 <= c < |C_i|) and is larger than the previous entry (rows ascend).
__device__ __forceinline__ bool idx_entry_valid(const int32_t* row, int slot, int ncand) {
    const int c = row[slot];
    if (c < 0 || c >= ncand) return false;
    if (slot > 0 && c <= row[slot - 1]) return false;
    return true;
}

}  // namespace hils
