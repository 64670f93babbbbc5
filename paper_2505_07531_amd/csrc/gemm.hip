// Batched quantized GEMM (prefill): Y[m][n] = sum_k X[m][k] W'[n][k].
//
// The product is a dense contraction once W' is dequantized, so it runs on the
// matrix cores: per 128-wide K step a block dequantizes a 64-row x 128 W' tile
// into LDS (fp16, natural K order; uniform W' = fp16(s*(q-z)) by one packed
// fp16 multiply of exact integers) next to the matching X tile, and each wave
// multiplies its 16 weight rows with every 16-row slice of X using
// v_mfma_f32_16x16x32_f16 (fp16 inputs, fp32 accumulators).
//
// Launch: 256 threads (4 waves); block (bx, by) owns weight rows
// [64 bx, 64 bx + 64) and activation rows [BM by, BM by + BM), BM = 16*MT.
#include "qx_device.h"
#include "qx_internal.h"

namespace qx {

constexpr int kGemmThreads = 256;
constexpr int kBN = 64;
constexpr int kRowBytes = 272;  // LDS row stride: 128 fp16 + 16 bytes of padding

// Natural-order 4-code selector of block t (codes 4t..4t+3) of a chunk.
template <int BITS, int T>
__device__ __forceinline__ uint32_t block_sel(const uint32_t (&d)[4 * BITS]) {
  if constexpr (BITS == 4) {
    constexpr int j = T / 2;
    const uint32_t lo = d[j] & 0x0F0F0F0Fu, hi = (d[j] >> 4) & 0x0F0F0F0Fu;
    return (T & 1) ? perm(hi, lo, 0x07030602u) : perm(hi, lo, 0x05010400u);
  } else if constexpr (T < 12) {
    return u3_sel_a(d[T]);
  } else if constexpr (T < 24) {
    return u3_sel_b(d[T - 12]);
  } else {
    return u3_sel_spare<T - 24>(d[T - 24], d[8 + ((T - 24) & 3)]);
  }
}

// Decode codes [32U, 32U + 32) of a chunk into 16 fp16 pairs.
template <int BITS, int KIND, int G, int U>
__device__ __forceinline__ void decode_quarter(const uint32_t (&d)[4 * BITS], const uint32_t* meta,
                                               uint32_t (&w)[16]) {
  constexpr int kMetaDw = KIND == QX_UNIFORM ? 1 : (1 << BITS) / 2;
#pragma unroll
  for (int v = 0; v < 8; ++v) {
    uint32_t Q;
    switch (v) {
      case 0: Q = block_sel<BITS, 8 * U + 0>(d); break;
      case 1: Q = block_sel<BITS, 8 * U + 1>(d); break;
      case 2: Q = block_sel<BITS, 8 * U + 2>(d); break;
      case 3: Q = block_sel<BITS, 8 * U + 3>(d); break;
      case 4: Q = block_sel<BITS, 8 * U + 4>(d); break;
      case 5: Q = block_sel<BITS, 8 * U + 5>(d); break;
      case 6: Q = block_sel<BITS, 8 * U + 6>(d); break;
      default: Q = block_sel<BITS, 8 * U + 7>(d); break;
    }
    const int g = (4 * (8 * U + v)) / G;
    block_weights<BITS, KIND>(Q, meta + g * kMetaDw, w[2 * v], w[2 * v + 1]);
  }
}

template <int BITS, int KIND, int G, int MT>
__global__ __launch_bounds__(kGemmThreads) void gemm_kernel(const char* __restrict__ packed,
                                                             const uint16_t* __restrict__ X,
                                                             uint16_t* __restrict__ Y, int n,
                                                             int k, int m) {
  constexpr int BM = 16 * MT;
  constexpr int kMetaDw = KIND == QX_UNIFORM ? 128 / G : (128 / G) * (1 << BITS) / 2;
  __shared__ __align__(16) char xs[BM * kRowBytes];
  __shared__ __align__(16) char ws[kBN * kRowBytes];
  const int C = k >> 7, G_row = k / G;
  const size_t meta_off = (size_t)n * k * BITS / 8;
  const int n0 = blockIdx.x * kBN, m0 = blockIdx.y * BM;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int wrow = n0 + lane;  // weight row this lane decodes
  const bool wvalid = wrow < n;

  f4_t acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f4_t{0.f, 0.f, 0.f, 0.f};

  for (int c = 0; c < C; ++c) {
    // X tile [BM][128]
    for (int p = threadIdx.x; p < BM * 16; p += kGemmThreads) {
      const int r = p >> 4, t = p & 15;
      u32x4 v = u32x4{0u, 0u, 0u, 0u};
      if (m0 + r < m)
        v = *reinterpret_cast<const u32x4*>(X + (size_t)(m0 + r) * k + (size_t)c * 128 + 8 * t);
      *reinterpret_cast<u32x4*>(xs + r * kRowBytes + 16 * t) = v;
    }
    // W' tile: lane -> weight row, wave -> quarter of the chunk
    if (wvalid) {
      const u32x4* code = reinterpret_cast<const u32x4*>(packed) + ((size_t)wrow * BITS * C + c);
      uint32_t d[4 * BITS];
#pragma unroll
      for (int s = 0; s < BITS; ++s) {
        const u32x4 v = code[(size_t)s * C];
        d[4 * s] = v.x; d[4 * s + 1] = v.y; d[4 * s + 2] = v.z; d[4 * s + 3] = v.w;
      }
      const size_t gidx = (size_t)wrow * G_row + (size_t)c * (128 / G);
      const uint32_t* mp = reinterpret_cast<const uint32_t*>(
          packed + meta_off + gidx * (KIND == QX_UNIFORM ? 4 : 2 * (1 << BITS)));
      uint32_t meta[kMetaDw];
#pragma unroll
      for (int i = 0; i < kMetaDw; ++i) meta[i] = mp[i];
      uint32_t w[16];
      switch (wave) {
        case 0: decode_quarter<BITS, KIND, G, 0>(d, meta, w); break;
        case 1: decode_quarter<BITS, KIND, G, 1>(d, meta, w); break;
        case 2: decode_quarter<BITS, KIND, G, 2>(d, meta, w); break;
        default: decode_quarter<BITS, KIND, G, 3>(d, meta, w); break;
      }
      u32x4* dst = reinterpret_cast<u32x4*>(ws + lane * kRowBytes + 64 * wave);
#pragma unroll
      for (int i = 0; i < 4; ++i) dst[i] = u32x4{w[4 * i], w[4 * i + 1], w[4 * i + 2], w[4 * i + 3]};
    }
    __syncthreads();
    // MFMA: wave -> weight rows [16 wave, 16 wave + 16)
    const int li = lane & 15, lq = lane >> 4;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const h8_t b = *reinterpret_cast<const h8_t*>(ws + (16 * wave + li) * kRowBytes + 64 * kk + 16 * lq);
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        const h8_t a = *reinterpret_cast<const h8_t*>(xs + (16 * t + li) * kRowBytes + 64 * kk + 16 * lq);
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, acc[t], 0, 0, 0);
      }
    }
    __syncthreads();
  }
  // D[i][j]: lane holds rows 4*(lane/16) + r, column lane % 16
  const int col = n0 + 16 * wave + (lane & 15);
  if (col < n) {
#pragma unroll
    for (int t = 0; t < MT; ++t) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + 16 * t + 4 * (lane >> 4) + r;
        if (row < m) Y[(size_t)row * n + col] = (uint16_t)float_to_half_bits(acc[t][r]);
      }
    }
  }
}

template <int BITS, int KIND, int G>
static int launch_gemm_t(const qx_desc* d, const void* packed, int m, const uint16_t* X,
                         uint16_t* Y, hipStream_t s) {
  const char* p = static_cast<const char*>(packed);
  const unsigned nb = (unsigned)((d->n + kBN - 1) / kBN);
  if (m <= 16) {
    hipLaunchKernelGGL((gemm_kernel<BITS, KIND, G, 1>), dim3(nb, (m + 15) / 16), dim3(kGemmThreads), 0, s, p, X, Y, d->n, d->k, m);
  } else if (m <= 32) {
    hipLaunchKernelGGL((gemm_kernel<BITS, KIND, G, 2>), dim3(nb, (m + 31) / 32), dim3(kGemmThreads), 0, s, p, X, Y, d->n, d->k, m);
  } else {
    hipLaunchKernelGGL((gemm_kernel<BITS, KIND, G, 4>), dim3(nb, (m + 63) / 64), dim3(kGemmThreads), 0, s, p, X, Y, d->n, d->k, m);
  }
  return hipGetLastError() == hipSuccess ? QX_OK : QX_E_HIP;
}

int launch_gemm(const qx_desc* d, const void* packed, int m, const uint16_t* X, uint16_t* Y,
                hipStream_t s) {
#define QX_GEMM_CASE(B, K, G) \
  if (d->bits == B && d->kind == K && d->group == G) return launch_gemm_t<B, K, G>(d, packed, m, X, Y, s);
  QX_GEMM_CASE(3, 0, 32) QX_GEMM_CASE(3, 0, 64) QX_GEMM_CASE(3, 0, 128)
  QX_GEMM_CASE(3, 1, 32) QX_GEMM_CASE(3, 1, 64) QX_GEMM_CASE(3, 1, 128)
  QX_GEMM_CASE(4, 0, 32) QX_GEMM_CASE(4, 0, 64) QX_GEMM_CASE(4, 0, 128)
  QX_GEMM_CASE(4, 1, 32) QX_GEMM_CASE(4, 1, 64) QX_GEMM_CASE(4, 1, 128)
#undef QX_GEMM_CASE
  return QX_E_UNSUPPORTED;
}

}  // namespace qx
