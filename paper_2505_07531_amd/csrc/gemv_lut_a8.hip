// GEMV with 8-bit activations for the table formats: per-group codebooks (QuantX's
// non-uniform groups, Section 2.2, in its W3A8 configurations, Table 1) and Q4X
// (the paper's own runtime configuration: Q4X with 8-bit round-to-nearest per-token
// activations, Table 2). The activation vector is quantized as in the uniform A8
// GEMV (amax = max |x|, xq = nearest integer to x * fp32(127/amax), s_x = amax/127)
// and, since table levels are fp16 entries rather than integers, the integers xq
// are staged as exact binary16 values and multiplied with the looked-up entries in
// fp32 like the fp16 GEMV of the same format:
//   codebook  y[n] = s_x * sum_k C[n, j(k)][q_k] * xq_k
//   Q4X       y[n] = s_x * sum_j s_j * sum_{k in group j} CB[t_j][q_k] * xq_k.
// One (row, 128-code chunk) item per lane; for k = 128*32 or 128*64 a row fills half
// or all of a wave and is summed in registers (the wave-kernel structure), other k
// up to 88 chunks use R rows per block with partials through LDS (the row kernel).
#include "gemv_common.h"

#include <algorithm>

namespace qx {
namespace {

__device__ __forceinline__ float wave_max_q(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// Nearest integer to x * inv (the product exact: one fused multiply-add with
// 1.5 * 2^23, whose rounding step is 1), as an fp32 value.
__device__ __forceinline__ float q8f(_Float16 v, float inv) {
  return __builtin_fmaf((float)v, inv, 12582912.0f) - 12582912.0f;
}

// Block-wide maximum magnitude of the staged x pieces (every thread gets it).
template <int XP>
__device__ __forceinline__ float block_amax(const u32x4 (&xr)[XP], float* red, int nthreads) {
  h2_t mh = {(_Float16)0, (_Float16)0};
#pragma unroll
  for (int i = 0; i < XP; ++i) {  // clamped duplicates of valid pieces leave the max unchanged
    const uint32_t w[4] = {xr[i].x, xr[i].y, xr[i].z, xr[i].w};
#pragma unroll
    for (int q = 0; q < 4; ++q)
      mh = __builtin_elementwise_max(mh, __builtin_elementwise_abs(__builtin_bit_cast(h2_t, w[q])));
  }
  const float m = wave_max_q(fmaxf((float)mh.x, (float)mh.y));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  float amax = 0.f;
  for (int i = 0; i < (nthreads >> 6); ++i) amax = fmaxf(amax, red[i]);
  return amax;
}

// The pieces as exact binary16 integers xq = nearest integer to x * inv.
template <int XP>
__device__ __forceinline__ void quantize_pieces(u32x4 (&xr)[XP], float inv) {
#pragma unroll
  for (int i = 0; i < XP; ++i) {
    uint32_t w[4] = {xr[i].x, xr[i].y, xr[i].z, xr[i].w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const h2_t h = __builtin_bit_cast(h2_t, w[q]);
      const h2_t o = {(_Float16)q8f(h.x, inv), (_Float16)q8f(h.y, inv)};
      w[q] = __builtin_bit_cast(uint32_t, o);
    }
    xr[i] = u32x4{w[0], w[1], w[2], w[3]};
  }
}

// k = 128*LPR with LPR in {32, 64}: as the fp16 wave kernel, a row's chunks fill LPR
// lanes of one wave and are summed with DPP; the block's WPB waves stage x once.
template <int BITS, int KIND, int G, int LPR, int WPB>
__global__ __launch_bounds__(64 * WPB) void gemv_lut_a8_wave_kernel(const char* __restrict__ packed,
                                                                    const uint16_t* __restrict__ x,
                                                                    uint16_t* __restrict__ y, int n) {
  constexpr int C = LPR, NT = 64 * WPB, RPW = 64 / LPR, RPB = WPB * RPW;
  constexpr int XP = (C * 16 + NT - 1) / NT;
  __shared__ __align__(16) char xs[C * kXBlock];
  __shared__ __align__(16) uint32_t q4lut[KIND == QX_Q4X ? 32 : 1];
  __shared__ float red[WPB];
  const int k = C * 128;
  const size_t meta_off = (size_t)n * k * BITS / 8;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c = lane & (LPR - 1);
  const int row = blockIdx.x * RPB + wave * RPW + lane / LPR;
  const DecodeConsts kc = decode_consts();

  u32x4 xr[XP];
  load_x<XP>(x, 0, C, xr, NT);
  Item<BITS, KIND, G> it;
  load_item<BITS, KIND, G>(it, packed, meta_off, min(row, n - 1), c, C, k / G);
  if constexpr (KIND == QX_Q4X) stage_q4x_lut(packed, n, k, q4lut);
  const float amax = block_amax<XP>(xr, red, NT);
  quantize_pieces<XP>(xr, amax > 0.f ? 127.f / amax : 0.f);
  store_x<BITS, KIND, G, XP, C * 16 % NT == 0>(xr, C, xs, nullptr, NT);
  __syncthreads();
  float v = chunk_dot<BITS, KIND, G>(it, xs + c * kXBlock, nullptr, kc, q4lut);
  v = (LPR == 32) ? half_wave_sum(v) : wave_sum(v);
  const float sx = amax > 0.f ? amax / 127.f : 0.f;
  if ((lane & (LPR - 1)) == LPR - 1 && row < n) y[row] = (uint16_t)float_to_half_bits(v * sx);
}

template <int BITS, int KIND, int G, int XP>
__global__ __launch_bounds__(1024) void gemv_lut_a8_row_kernel(const char* __restrict__ packed,
                                                               const uint16_t* __restrict__ x,
                                                               uint16_t* __restrict__ y, int n, int k, int R) {
  extern __shared__ __align__(16) char smem[];
  __shared__ __align__(16) uint32_t q4lut[KIND == QX_Q4X ? 32 : 1];
  __shared__ float red[16];
  const int C = k >> 7, G_row = k / G, nthreads = blockDim.x;
  const size_t meta_off = (size_t)n * k * BITS / 8;
  const int row0 = blockIdx.x * R;
  const int rows = min(R, n - row0);
  char* xs = smem;                                             // C * kXBlock bytes
  float* part = reinterpret_cast<float*>(smem + C * kXBlock);  // R * C floats
  const DecodeConsts kc = decode_consts();

  u32x4 xr[XP];
  load_x<XP>(x, 0, C, xr, nthreads);
  const int t = threadIdx.x, r = t / C, c = t - r * C;
  const bool valid = r < rows;
  Item<BITS, KIND, G> it;
  load_item<BITS, KIND, G>(it, packed, meta_off, row0 + min(r, rows - 1), c, C, G_row);
  if constexpr (KIND == QX_Q4X) stage_q4x_lut(packed, n, k, q4lut);

  // amax over the vector (every block gets the same maximum: a maximum is exact), then
  // the pieces as exact binary16 integers xq, staged in decoder order
  const float amax = block_amax<XP>(xr, red, nthreads);
  quantize_pieces<XP>(xr, amax > 0.f ? 127.f / amax : 0.f);
  store_x<BITS, KIND, G, XP>(xr, C, xs, nullptr, nthreads);
  __syncthreads();
  if (valid) part[t] = chunk_dot<BITS, KIND, G>(it, xs + c * kXBlock, nullptr, kc, q4lut);
  __syncthreads();
  const float sx = amax > 0.f ? amax / 127.f : 0.f;
  const int wave = t >> 6, lane = t & 63;
  for (int rr = wave; rr < rows; rr += nthreads >> 6) {
    float v = 0.f;
    for (int cc = lane; cc < C; cc += 64) v += part[rr * C + cc];
    v = wave_sum(v);
    if (lane == 63) y[row0 + rr] = (uint16_t)float_to_half_bits(v * sx);
  }
}

template <int BITS, int KIND, int G>
static int launch_lut_a8_t(const qx_desc* d, const void* packed, const uint16_t* x, uint16_t* y, hipStream_t s) {
  const int C = d->k / 128;
  if (C > kMaxTileChunks) return QX_E_UNSUPPORTED;
  const char* p = static_cast<const char*>(packed);
  if (C == 32 || C == 64) {
    constexpr int WPB = 4;
    const int rpb = WPB * 64 / C;
    const dim3 grid((unsigned)((d->n + rpb - 1) / rpb)), block(64 * WPB);
    if (C == 32)
      hipLaunchKernelGGL((gemv_lut_a8_wave_kernel<BITS, KIND, G, 32, WPB>), grid, block, 0, s, p, x, y, d->n);
    else
      hipLaunchKernelGGL((gemv_lut_a8_wave_kernel<BITS, KIND, G, 64, WPB>), grid, block, 0, s, p, x, y, d->n);
    return hipGetLastError() == hipSuccess ? QX_OK : QX_E_HIP;
  }
  int R, threads;
  gemv_row_shape(d->n, C, KIND == QX_CODEBOOK && BITS == 4 && G == 32, &R, &threads);
  const size_t lds = (size_t)C * kXBlock + (size_t)R * C * sizeof(float);
  const int xp = (C * 16 + threads - 1) / threads;
  const dim3 grid((unsigned)((d->n + R - 1) / R)), block(threads);
  if (xp <= 1)
    hipLaunchKernelGGL((gemv_lut_a8_row_kernel<BITS, KIND, G, 1>), grid, block, lds, s, p, x, y, d->n, d->k, R);
  else if (xp <= 2)
    hipLaunchKernelGGL((gemv_lut_a8_row_kernel<BITS, KIND, G, 2>), grid, block, lds, s, p, x, y, d->n, d->k, R);
  else  // long rows have blocks of >= 256 threads, so xp <= ceil(88*16/256) = 6
    hipLaunchKernelGGL((gemv_lut_a8_row_kernel<BITS, KIND, G, 6>), grid, block, lds, s, p, x, y, d->n, d->k, R);
  return hipGetLastError() == hipSuccess ? QX_OK : QX_E_HIP;
}

}  // namespace

// Codebook and Q4X descriptors with k <= 88 chunks (as the uniform A8 GEMV).
int launch_gemv_lut_a8(const qx_desc* d, const void* packed, const uint16_t* x, uint16_t* y, hipStream_t s) {
  if (d->kind == QX_Q4X) return launch_lut_a8_t<4, QX_Q4X, 64>(d, packed, x, y, s);
  if (d->kind != QX_CODEBOOK) return QX_E_UNSUPPORTED;
#define QX_LUT_A8_CASE(B, G) \
  if (d->bits == B && d->group == G) return launch_lut_a8_t<B, QX_CODEBOOK, G>(d, packed, x, y, s);
  QX_LUT_A8_CASE(3, 32) QX_LUT_A8_CASE(3, 64) QX_LUT_A8_CASE(3, 128)
  QX_LUT_A8_CASE(4, 32) QX_LUT_A8_CASE(4, 64) QX_LUT_A8_CASE(4, 128)
#undef QX_LUT_A8_CASE
  return QX_E_UNSUPPORTED;
}

}  // namespace qx
