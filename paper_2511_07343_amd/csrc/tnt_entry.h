// Internal entry shared by the C ABI's forward calls.  Internal to the library.
#pragma once

#include <hip/hip_runtime.h>

#include "../../include/tnt.h"

namespace tnt {
// tnt_mem_fwd's validation and launch sequence.  `fork`: the global memory's
// chain may run on the library's helper stream (true) or stays on `stream`.
tnt_status forward_entry(const tnt_config* cfg, const void* q, const void* k, const void* v,
                         const float* lr, const float* mom, const float* decay,
                         const float* W1_init, const float* W2_init, void* o,
                         float* final_state, void* saved, size_t saved_bytes, void* workspace,
                         size_t ws_bytes, bool fork, hipStream_t stream);
}  // namespace tnt
