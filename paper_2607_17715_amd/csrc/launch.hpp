// Kernel launchers (defined in kernels.hip), called by the C ABI in api.cpp.
// Non-null events are stamped at the kernel's start and end.
#pragma once

#include <hip/hip_runtime.h>

#include "plan.hpp"

namespace c2kv {

enum SrcKind { kSrcPaged = 0, kSrcPool = 1, kSrcPoolI8 = 2 };

hipError_t launch_attention(const Plan& p, void* ws, int src_kind, const void* k, const void* v,
                            const float* k_scale, const float* v_scale, const void* q,
                            const void* k_suf, const void* v_suf, void* out, float* lse,
                            hipStream_t st, hipEvent_t e0, hipEvent_t e1);
hipError_t launch_merge(const Plan& p, void* ws, void* out, float* lse, hipStream_t st,
                        hipEvent_t e0, hipEvent_t e1);
// Device address of the current GPU's static scratch array (C2KV_STATIC_SCRATCH_BYTES),
// looked up once per device with that device current, then cached.
hipError_t static_scratch(void** ptr);

hipError_t launch_compose(const Plan& p, void* ws, int pool_dtype, const void* k, const void* v,
                          const float* k_scale, const float* v_scale, void* k_pages,
                          void* v_pages, int64_t* out_src_row, int32_t* out_pos,
                          hipStream_t st, hipEvent_t e0, hipEvent_t e1);

}  // namespace c2kv
