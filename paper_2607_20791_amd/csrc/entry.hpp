// Host routines shared by the C ABI's source files (internal).
#pragma once
#include <stdint.h>

#include "rgd.h"

namespace rgd {

// Sets the thread's last-error message and returns code.
int32_t set_error(int32_t code, const char* msg);

// min-p (pless false) or p-less draws on z [R][V] with a caller-provided
// device workspace of rgd_sampler_workspace_bytes(R, V) bytes, 256-byte
// aligned: the body of rgd_kernel_sample / rgd_kernel_sample_pless, which
// validates its arguments before any HIP call.
int32_t kernel_sample(const float* z, int32_t R, int32_t V, float T, float min_p, bool pless,
                      const uint64_t* seeds, uint32_t ctr, uint32_t stream0, int32_t draws, void* workspace,
                      int32_t* out, rgd_stream stream);

}  // namespace rgd
