// Dequantization kernel: packed blob -> raw codes (uint8 [n][k]) or fp16 W'
// [n][k], bit-exact with the definitions (uniform W' = fp16_RNE(s*(q-z)): the
// exact integers q - z times s in one IEEE fp16 multiply; codebook W' = C[q], a
// byte copy through the v_perm tables; Q4X W' = fp16_RNE(s*CB[sel][q]), the
// table entry times s in one IEEE fp16 multiply). One lane per (row, 128-code
// chunk).
#include "qx_device.h"
#include "qx_internal.h"

namespace qx {

// 128 codes of a chunk as 32 dwords, four codes per dword in natural order.
template <int BITS>
__device__ __forceinline__ void chunk_codes(const uint32_t (&d)[4 * BITS], uint32_t (&q)[32]) {
  if constexpr (BITS == 4) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const uint32_t lo = d[j] & 0x0F0F0F0Fu;         // codes 0 2 4 6
      const uint32_t hi = (d[j] >> 4) & 0x0F0F0F0Fu;  // codes 1 3 5 7
      q[2 * j] = perm(hi, lo, 0x05010400u);
      q[2 * j + 1] = perm(hi, lo, 0x07030602u);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 12; ++i) {
      q[i] = u3_sel_a(d[i]);
      q[12 + i] = u3_sel_b(d[i]);
    }
    q[24] = u3_sel_spare<0>(d[0], d[8]);
    q[25] = u3_sel_spare<1>(d[1], d[9]);
    q[26] = u3_sel_spare<2>(d[2], d[10]);
    q[27] = u3_sel_spare<3>(d[3], d[11]);
    q[28] = u3_sel_spare<4>(d[4], d[8]);
    q[29] = u3_sel_spare<5>(d[5], d[9]);
    q[30] = u3_sel_spare<6>(d[6], d[10]);
    q[31] = u3_sel_spare<7>(d[7], d[11]);
  }
}

template <int BITS, int KIND, int G, int OUT>
__global__ __launch_bounds__(256) void dequant_kernel(const char* __restrict__ packed,
                                                       void* __restrict__ out, int n, int k) {
  const int C = k >> 7;
  const size_t item = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (item >= (size_t)n * C) return;
  const int row = (int)(item / C), c = (int)(item - (size_t)row * C);
  const u32x4* code = reinterpret_cast<const u32x4*>(packed) + ((size_t)row * BITS * C + c);
  uint32_t d[4 * BITS];
#pragma unroll
  for (int s = 0; s < BITS; ++s) {
    const u32x4 v = code[(size_t)s * C];
    d[4 * s] = v.x; d[4 * s + 1] = v.y; d[4 * s + 2] = v.z; d[4 * s + 3] = v.w;
  }
  uint32_t q[32];
  chunk_codes<BITS>(d, q);
  const size_t e0 = (size_t)row * k + (size_t)c * 128;  // first output element
  if constexpr (OUT == QX_OUT_CODES) {
    u32x4* o = reinterpret_cast<u32x4*>(static_cast<uint8_t*>(out) + e0);
#pragma unroll
    for (int i = 0; i < 8; ++i) o[i] = u32x4{q[4 * i], q[4 * i + 1], q[4 * i + 2], q[4 * i + 3]};
    return;
  } else if constexpr (KIND == QX_Q4X) {
    // groups 2c (codes 0-63) and 2c + 1 (64-127): the selected sub-codebook's entry
    // times the group's scale, one IEEE fp16 multiply of the two binary16 values
    const Q4xOffsets L = q4x_offsets(n, k);
    const uint32_t sw = *reinterpret_cast<const uint32_t*>(packed + L.scales + ((size_t)row * L.groups + 2 * c) * 2);
    const uint32_t selw = *reinterpret_cast<const uint32_t*>(packed + L.selectors + ((size_t)row * L.words + c / 8) * 4);
    const uint32_t* cb = reinterpret_cast<const uint32_t*>(packed + L.codebook);
    uint32_t w[64];  // fp16 pairs, natural order
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      const uint32_t* tab = cb + 8 * ((selw >> (4 * (c % 8) + 2 * g)) & 3u);
      const uint32_t sp = ((sw >> (16 * g)) & 0xFFFFu) * 0x00010001u;  // (s, s)
#pragma unroll
      for (int t = 16 * g; t < 16 * g + 16; ++t) {
        block_weights<4, QX_CODEBOOK>(q[t], tab, w[2 * t], w[2 * t + 1]);
        w[2 * t] = hmul2(w[2 * t], sp);
        w[2 * t + 1] = hmul2(w[2 * t + 1], sp);
      }
    }
    u32x4* o = reinterpret_cast<u32x4*>(static_cast<uint16_t*>(out) + e0);
#pragma unroll
    for (int i = 0; i < 16; ++i) o[i] = u32x4{w[4 * i], w[4 * i + 1], w[4 * i + 2], w[4 * i + 3]};
  } else {
    const size_t meta_off = (size_t)n * k * BITS / 8;
    const size_t g0 = (size_t)row * (k / G) + (size_t)c * (128 / G);
    uint32_t w[64];  // fp16 pairs, natural order
    constexpr int kDw = KIND == QX_UNIFORM ? 1 : (1 << BITS) / 2;  // dwords per group table
    const uint32_t* mp = reinterpret_cast<const uint32_t*>(packed + meta_off) + g0 * kDw;
#pragma unroll
    for (int t = 0; t < 32; ++t)
      block_weights<BITS, KIND>(q[t], mp + ((4 * t) / G) * kDw, w[2 * t], w[2 * t + 1]);
    u32x4* o = reinterpret_cast<u32x4*>(static_cast<uint16_t*>(out) + e0);
#pragma unroll
    for (int i = 0; i < 16; ++i) o[i] = u32x4{w[4 * i], w[4 * i + 1], w[4 * i + 2], w[4 * i + 3]};
  }
}

template <int BITS, int KIND, int G>
static int launch_dequant_t(const qx_desc* d, const void* packed, int out_kind, void* out,
                            hipStream_t s) {
  const size_t items = (size_t)d->n * (d->k / 128);
  const dim3 grid((unsigned)((items + 255) / 256)), block(256);
  const char* p = static_cast<const char*>(packed);
  if (out_kind == QX_OUT_CODES)
    hipLaunchKernelGGL((dequant_kernel<BITS, KIND, G, QX_OUT_CODES>), grid, block, 0, s, p, out, d->n, d->k);
  else
    hipLaunchKernelGGL((dequant_kernel<BITS, KIND, G, QX_OUT_F16>), grid, block, 0, s, p, out, d->n, d->k);
  return hipGetLastError() == hipSuccess ? QX_OK : QX_E_HIP;
}

int launch_dequant(const qx_desc* d, const void* packed, int out_kind, void* out, hipStream_t s) {
#define QX_DQ_CASE(B, K, G) \
  if (d->bits == B && d->kind == K && d->group == G) return launch_dequant_t<B, K, G>(d, packed, out_kind, out, s);
  QX_DQ_CASE(3, 0, 32) QX_DQ_CASE(3, 0, 64) QX_DQ_CASE(3, 0, 128)
  QX_DQ_CASE(3, 1, 32) QX_DQ_CASE(3, 1, 64) QX_DQ_CASE(3, 1, 128)
  QX_DQ_CASE(4, 0, 32) QX_DQ_CASE(4, 0, 64) QX_DQ_CASE(4, 0, 128)
  QX_DQ_CASE(4, 1, 32) QX_DQ_CASE(4, 1, 64) QX_DQ_CASE(4, 1, 128)
  QX_DQ_CASE(4, 2, 64)
#undef QX_DQ_CASE
  return QX_E_UNSUPPORTED;
}

}  // namespace qx
