// Internal interface between the C-ABI front end (qx_api.cpp) and the kernel
// launchers. Descriptors reaching these functions are validated and supported.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/qx.h"

namespace qx {

// Byte offsets of the Q4X regions after the 4-bit codes of an n x k matrix:
// binary16 scales per group of 64, ceil(G/16) uint32 selector words per row
// (2 bits per group), and the 64-entry binary16 codebook at a multiple of 16.
struct Q4xOffsets {
  size_t scales, selectors, codebook, total;
  int groups, words;
};
__host__ __device__ inline Q4xOffsets q4x_offsets(int n, int k) {
  Q4xOffsets o;
  o.groups = k / 64;
  o.words = (o.groups + 15) / 16;
  o.scales = (size_t)n * k / 2;
  o.selectors = o.scales + (size_t)n * o.groups * 2;
  o.codebook = (o.selectors + (size_t)n * o.words * 4 + 15) / 16 * 16;
  o.total = o.codebook + 128;
  return o;
}

int launch_dequant(const qx_desc* d, const void* packed, int out_kind, void* out, hipStream_t s);
int launch_gemv(const qx_desc* d, const void* packed, const uint16_t* x, uint16_t* y,
                hipStream_t s);
int launch_gemm(const qx_desc* d, const void* packed, int m, const uint16_t* X, uint16_t* Y,
                hipStream_t s);
int launch_gemv_a8(const qx_desc* d, const void* packed, const uint16_t* x, uint16_t* y,
                   hipStream_t s);

// W·A8 for many rows: per-row int8 activations and the integer-product GEMM
// (uniform descriptors).
int launch_quantize_a8(int m, int k, const uint16_t* X, int8_t* Xq, float* sx, hipStream_t s);
int launch_gemm_a8(const qx_desc* d, const void* packed, int m, const int8_t* Xq, const float* sx, uint16_t* Y,
                   hipStream_t s);
// The small-batch A8 kernel for 2 <= m <= 4 pre-quantized rows (any k).
int launch_gemv_a8_multi(const qx_desc* d, const void* packed, int m, const int8_t* Xq, const float* sx,
                         uint16_t* Y, hipStream_t s);
// The A8 GEMV of Q4X matrices (fp16 table entries times the integer xq; k <= 88*128).
int launch_gemv_lut_a8(const qx_desc* d, const void* packed, const uint16_t* x, uint16_t* y, hipStream_t s);
int launch_gemm_lut_a8(const qx_desc* d, const void* packed, int m, const int8_t* Xq, const float* sx,
                       uint16_t* Y, hipStream_t s);
// The A8 GEMV on one row already quantized (k <= 88*128).
int launch_gemv_a8q(const qx_desc* d, const void* packed, const int8_t* xq, const float* sx, uint16_t* y,
                    hipStream_t s);

// Products of at most QX_MULTI_MAX_M rows may run GEMV-style (gemv_multi_applies
// decides; launch_gemv_multi takes 2 <= m <= QX_MULTI_MAX_M, any k, every kind).
#ifndef QX_MULTI_MAX_M
#define QX_MULTI_MAX_M 4
#endif
bool gemv_multi_applies(const qx_desc* d, int m);
int launch_gemv_multi(const qx_desc* d, const void* packed, int m, const uint16_t* X, uint16_t* Y,
                      hipStream_t s);

// Products of 2 <= m <= QX_SKINNY_MAX_M rows on the matrix cores with the GEMV's
// chunk-per-lane loads (gemm_skinny.hip; gemm_skinny_applies picks it per shape and
// format); k up to 128 chunks.
#ifndef QX_SKINNY_MAX_M
#define QX_SKINNY_MAX_M 64
#endif
bool gemm_skinny_applies(const qx_desc* d, int m);

int launch_gemm_skinny(const qx_desc* d, const void* packed, int m, const uint16_t* X, uint16_t* Y,
                       hipStream_t s);

}  // namespace qx
