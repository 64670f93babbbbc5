// Internal interface between the C-ABI front end (qx_api.cpp) and the kernel
// launchers. Descriptors reaching these functions are validated and supported.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/qx.h"

namespace qx {

int launch_dequant(const qx_desc* d, const void* packed, int out_kind, void* out, hipStream_t s);
int launch_gemv(const qx_desc* d, const void* packed, const uint16_t* x, uint16_t* y,
                hipStream_t s);
int launch_gemm(const qx_desc* d, const void* packed, int m, const uint16_t* X, uint16_t* Y,
                hipStream_t s);

}  // namespace qx
