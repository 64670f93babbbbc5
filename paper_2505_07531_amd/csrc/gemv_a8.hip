// Batch-1 GEMV with 8-bit activations: the paper keeps activations at 8 bits
// and not below (Section 2.4), and its W3A8 configurations (Table 1) and Table
// 2's runs quantize them per token by round-to-nearest. Here one activation
// vector gets one symmetric scale,
//   amax = max |x|, inv = 127 / amax (fp32), xq = nearest integer to x * inv
//   (the product exact), s_x = amax / 127 (fp32; amax = 0 gives xq = 0, y = 0),
// and uniform codes are multiplied with xq in exact integers:
//   y[n] = s_x * sum_j s_j * (sum_{k in j} q*xq - z_j * sum_{k in j} xq).
//
// Every block computes the same amax (a maximum is exact in any order) and
// quantizes its own copy of x while staging it in LDS; the integer products run
// on v_dot4_i32_i8 (four int8 products per lane and instruction), so a 4-bit
// code costs about a quarter of the VALU work of the fp16-activation path. The
// launch paths follow the fp16 GEMV: one 128-code chunk per lane, a wave per row
// pair for k = 128*32 or 128*64, rows of up to 88 chunks split over a block.
#include "gemv_common.h"  // also the row kernels' shape rule
#include "qx_internal.h"

#include <algorithm>

namespace qx {
namespace {

constexpr int kX8Block = 144;  // LDS bytes per chunk of int8 activations (128 + 16 pad)

template <int BITS, int G>
struct CodesA8 {
  uint32_t d[4 * BITS];  // the chunk's code slices
  uint32_t m[128 / G];   // scale | zero << 16 per group
};

template <int BITS, int G>
__device__ __forceinline__ void load_codes_a8(CodesA8<BITS, G>& it, const char* __restrict__ packed,
                                              size_t meta_off, int row, int c, int C, int G_row) {
  const u32x4* code = reinterpret_cast<const u32x4*>(packed) + ((size_t)row * BITS * C + c);
#pragma unroll
  for (int s = 0; s < BITS; ++s) {
    const u32x4 v = __builtin_nontemporal_load(code + (size_t)s * C);
    it.d[4 * s + 0] = v.x; it.d[4 * s + 1] = v.y; it.d[4 * s + 2] = v.z; it.d[4 * s + 3] = v.w;
  }
  const uint32_t* mp = reinterpret_cast<const uint32_t*>(packed + meta_off) + (size_t)row * G_row +
                       (size_t)c * (128 / G);
  if constexpr (128 / G == 4) {
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(mp));
    it.m[0] = v.x; it.m[1] = v.y; it.m[2] = v.z; it.m[3] = v.w;
  } else if constexpr (128 / G == 2) {
    const u32x2 v = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(mp));
    it.m[0] = v.x; it.m[1] = v.y;
  } else {
    it.m[0] = __builtin_nontemporal_load(mp);
  }
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// x * inv + 1.5 * 2^23 in one fused multiply-add (the fp16 x widened exactly): the
// sum lies in [2^23, 2^24), where fp32 steps by 1, so its single rounding is the
// nearest-even integer to the exact product, and the low byte of the result's bits
// is that integer as int8 (|x * inv| <= 127 since |x| <= amax).
__device__ __forceinline__ uint32_t q8_bits(_Float16 v, float inv) {
  return __builtin_bit_cast(uint32_t, __builtin_fmaf((float)v, inv, 12582912.0f));
}
// int8 bytes of four q8_bits values, in argument order
__device__ __forceinline__ uint32_t pack4(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  return perm(perm(d, c, 0x04000C0Cu), perm(b, a, 0x0C0C0400u), 0x07060100u);
}

// One piece of int8 activations (8 values, decoder order) to LDS, and the sum of
// xq over each group, whose pieces sit in consecutive lanes (every lane calls this).
template <int G>
__device__ __forceinline__ void store_x8(u32x2 o, int p, int C, char* xs, float* gs) {
  const bool valid = p < C * 16;
  if (valid) *reinterpret_cast<u32x2*>(xs + (p >> 4) * kX8Block + (p & 15) * 8) = o;
  constexpr int PPG = G / 8;  // pieces per group, consecutive lanes
  float s = (float)__builtin_amdgcn_sdot4((int)o.y, 0x01010101, __builtin_amdgcn_sdot4((int)o.x, 0x01010101, 0, false), false);
  if constexpr (PPG >= 4) {
    s = dpp_plus<0xB1, 0xF>(s);
    s = dpp_plus<0x4E, 0xF>(s);
    if constexpr (PPG >= 8) s = dpp_plus<0x141, 0xF>(s);
    if constexpr (PPG >= 16) s = dpp_plus<0x140, 0xF>(s);
  }
  if (valid && (p & (PPG - 1)) == 0) gs[p / PPG] = s;
}

// Quantize the staged pieces of x (XP 16-byte pieces per thread, piece p = chunk
// p/16, values 8*(p%16)..) with the block-wide scale, store them in LDS as int8 in
// the order the decoder consumes them (b = 4: per 8 codes the even then the odd
// positions; b = 3: natural), and the integer sum of xq per group in gs. Returns
// the vector's scale s_x. Contains one barrier.
template <int BITS, int G, int XP>
__device__ __forceinline__ float stage_x_a8(const u32x4 (&xr)[XP], int C, char* xs, float* gs,
                                            float* red, int nthreads) {
  h2_t mh = {(_Float16)0, (_Float16)0};
#pragma unroll
  for (int i = 0; i < XP; ++i) {  // clamped duplicates of valid pieces leave the max unchanged
    const uint32_t w[4] = {xr[i].x, xr[i].y, xr[i].z, xr[i].w};
#pragma unroll
    for (int t = 0; t < 4; ++t)
      mh = __builtin_elementwise_max(mh, __builtin_elementwise_abs(__builtin_bit_cast(h2_t, w[t])));
  }
  float m = fmaxf((float)mh.x, (float)mh.y);
  m = wave_max(m);
  const int wave = threadIdx.x >> 6, nwaves = nthreads >> 6;
  if ((threadIdx.x & 63) == 0) red[wave] = m;
  __syncthreads();
  float amax = 0.f;
  for (int i = 0; i < nwaves; ++i) amax = fmaxf(amax, red[i]);
  const float inv = amax > 0.f ? 127.f / amax : 0.f;
#pragma unroll
  for (int i = 0; i < XP; ++i) {
    const int p = threadIdx.x + i * nthreads;
    const uint32_t w[4] = {xr[i].x, xr[i].y, xr[i].z, xr[i].w};
    uint32_t q[8];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const h2_t h = __builtin_bit_cast(h2_t, w[t]);
      q[2 * t] = q8_bits(h.x, inv);
      q[2 * t + 1] = q8_bits(h.y, inv);
    }
    u32x2 o;
    if constexpr (BITS == 4) {
      o.x = pack4(q[0], q[2], q[4], q[6]);
      o.y = pack4(q[1], q[3], q[5], q[7]);
    } else {
      o.x = pack4(q[0], q[1], q[2], q[3]);
      o.y = pack4(q[4], q[5], q[6], q[7]);
    }
    store_x8<G>(o, p, C, xs, gs);
  }
  return amax > 0.f ? amax / 127.f : 0.f;
}

// Stage int8 activations already quantized (qx_quantize_a8: natural order, 8 bytes
// per piece) like stage_x_a8 stages its own: decoder order, group sums of xq.
template <int BITS, int G, int XP>
__device__ __forceinline__ void stage_xq_a8(const u32x2 (&xr)[XP], int C, char* xs, float* gs, int nthreads) {
#pragma unroll
  for (int i = 0; i < XP; ++i) {
    const int p = threadIdx.x + i * nthreads;
    u32x2 o = xr[i];
    if constexpr (BITS == 4) o = u32x2{perm(xr[i].y, xr[i].x, 0x06040200u), perm(xr[i].y, xr[i].x, 0x07050301u)};
    store_x8<G>(o, p, C, xs, gs);
  }
}

// sum_j s_j * (sum q*xq - z_j * sum xq) over the groups of one chunk.
template <int BITS, int G>
__device__ __forceinline__ float chunk_dot_a8(const CodesA8<BITS, G>& it, const char* xb, const float* gs) {
  constexpr int NG = 128 / G;
  const uint32_t* xd = reinterpret_cast<const uint32_t*>(xb);
  int acc[NG];
#pragma unroll
  for (int g = 0; g < NG; ++g) acc[g] = 0;
  if constexpr (BITS == 4) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {  // dword j: codes 8j..8j+7, group 8j / G
      const uint32_t D = it.d[j];
      const int g = (8 * j) / G;
      acc[g] = __builtin_amdgcn_sdot4((int)(D & 0x0F0F0F0Fu), (int)xd[2 * j], acc[g], false);
      acc[g] = __builtin_amdgcn_sdot4((int)((D >> 4) & 0x0F0F0F0Fu), (int)xd[2 * j + 1], acc[g], false);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 12; ++i) {  // A fields: codes 4i..; B fields: codes 48 + 4i..
      const uint32_t D = it.d[i];
      const int ga = (4 * i) / G, gb = (48 + 4 * i) / G;
      acc[ga] = __builtin_amdgcn_sdot4((int)u3_sel_a(D), (int)xd[i], acc[ga], false);
      acc[gb] = __builtin_amdgcn_sdot4((int)u3_sel_b(D), (int)xd[12 + i], acc[gb], false);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {  // spare codes 96 + 4i..
      uint32_t S;
      switch (i) {  // the bit-2 position depends on the dword index at compile time
        case 0: S = u3_sel_spare<0>(it.d[0], it.d[8]); break;
        case 1: S = u3_sel_spare<1>(it.d[1], it.d[9]); break;
        case 2: S = u3_sel_spare<2>(it.d[2], it.d[10]); break;
        case 3: S = u3_sel_spare<3>(it.d[3], it.d[11]); break;
        case 4: S = u3_sel_spare<4>(it.d[4], it.d[8]); break;
        case 5: S = u3_sel_spare<5>(it.d[5], it.d[9]); break;
        case 6: S = u3_sel_spare<6>(it.d[6], it.d[10]); break;
        default: S = u3_sel_spare<7>(it.d[7], it.d[11]); break;
      }
      const int gg = (96 + 4 * i) / G;
      acc[gg] = __builtin_amdgcn_sdot4((int)S, (int)xd[24 + i], acc[gg], false);
    }
  }
  float part = 0.f;
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const uint32_t word = it.m[g];
    const int z = (int)half_bits_to_float(word >> 16);
    part += half_bits_to_float(word & 0xFFFFu) * (float)(acc[g] - z * (int)gs[g]);
  }
  return part;
}

// k = 128*LPR with LPR in {32, 64}: as the fp16 wave kernel.
// PREQ: x is already int8 (qx_quantize_a8) with its scale at *sxp; else fp16.
template <int BITS, int G, int LPR, int WPB, bool PREQ>
__global__ __launch_bounds__(64 * WPB) void gemv_a8_wave_kernel(const char* __restrict__ packed,
                                                                const void* __restrict__ x,
                                                                const float* __restrict__ sxp,
                                                                uint16_t* __restrict__ y, int n) {
  constexpr int C = LPR, NT = 64 * WPB, RPW = 64 / LPR, RPB = WPB * RPW;
  constexpr int XP = (C * 16 + NT - 1) / NT;
  __shared__ __align__(16) char xs[C * kX8Block];
  __shared__ float gs[C * (128 / G)];
  __shared__ float red[WPB];
  const int k = C * 128;
  const size_t meta_off = (size_t)n * k * BITS / 8;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c = lane & (LPR - 1);
  const int row = blockIdx.x * RPB + wave * RPW + lane / LPR;

  float sx;
  CodesA8<BITS, G> it;
  if constexpr (PREQ) {
    u32x2 xr[XP];
    const u32x2* src = reinterpret_cast<const u32x2*>(x);
#pragma unroll
    for (int i = 0; i < XP; ++i) xr[i] = src[min((int)threadIdx.x + i * NT, C * 16 - 1)];
    load_codes_a8<BITS, G>(it, packed, meta_off, min(row, n - 1), c, C, k / G);
    stage_xq_a8<BITS, G, XP>(xr, C, xs, gs, NT);
    sx = *sxp;
  } else {
    u32x4 xr[XP];
    const u32x4* src = reinterpret_cast<const u32x4*>(x);
#pragma unroll
    for (int i = 0; i < XP; ++i) xr[i] = src[min((int)threadIdx.x + i * NT, C * 16 - 1)];
    load_codes_a8<BITS, G>(it, packed, meta_off, min(row, n - 1), c, C, k / G);
    sx = stage_x_a8<BITS, G, XP>(xr, C, xs, gs, red, NT);
  }
  __syncthreads();
  float v = chunk_dot_a8<BITS, G>(it, xs + c * kX8Block, gs + c * (128 / G));
  v = (LPR == 32) ? half_wave_sum(v) : wave_sum(v);
  if ((lane & (LPR - 1)) == LPR - 1 && row < n) y[row] = (uint16_t)float_to_half_bits(v * sx);
}

// Any k up to 88 chunks: one (row, chunk) item per lane, R rows per block, partials
// through LDS and one wave per row adding them in a fixed order (as the fp16 row kernel).
template <int BITS, int G, int XP, bool PREQ>
__global__ __launch_bounds__(1024) void gemv_a8_row_kernel(const char* __restrict__ packed,
                                                           const void* __restrict__ x,
                                                           const float* __restrict__ sxp,
                                                           uint16_t* __restrict__ y, int n, int k, int R) {
  extern __shared__ __align__(16) char smem[];
  __shared__ float red[16];
  const int C = k >> 7, G_row = k / G, nthreads = blockDim.x;
  const size_t meta_off = (size_t)n * k * BITS / 8;
  const int row0 = blockIdx.x * R;
  const int rows = min(R, n - row0);
  char* xs = smem;                                                   // C * kX8Block
  float* part = reinterpret_cast<float*>(smem + C * kX8Block);       // R * C
  float* gs = part + R * C;                                          // C * 128/G
  const int t = threadIdx.x, r = t / C, c = t - r * C;
  const bool valid = r < rows;
  float sx;
  CodesA8<BITS, G> it;
  if constexpr (PREQ) {
    u32x2 xr[XP];
    const u32x2* src = reinterpret_cast<const u32x2*>(x);
#pragma unroll
    for (int i = 0; i < XP; ++i) xr[i] = src[min((int)threadIdx.x + i * nthreads, C * 16 - 1)];
    load_codes_a8<BITS, G>(it, packed, meta_off, row0 + min(r, rows - 1), c, C, G_row);
    stage_xq_a8<BITS, G, XP>(xr, C, xs, gs, nthreads);
    sx = *sxp;
  } else {
    u32x4 xr[XP];
    const u32x4* src = reinterpret_cast<const u32x4*>(x);
#pragma unroll
    for (int i = 0; i < XP; ++i) xr[i] = src[min((int)threadIdx.x + i * nthreads, C * 16 - 1)];
    load_codes_a8<BITS, G>(it, packed, meta_off, row0 + min(r, rows - 1), c, C, G_row);
    sx = stage_x_a8<BITS, G, XP>(xr, C, xs, gs, red, nthreads);
  }
  __syncthreads();
  if (valid) part[t] = chunk_dot_a8<BITS, G>(it, xs + c * kX8Block, gs + c * (128 / G));
  __syncthreads();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int rr = wave; rr < rows; rr += nthreads >> 6) {
    float v = 0.f;
    for (int cc = lane; cc < C; cc += 64) v += part[rr * C + cc];
    v = wave_sum(v);
    if (lane == 63) y[row0 + rr] = (uint16_t)float_to_half_bits(v * sx);
  }
}

// 2 <= m <= M pre-quantized rows (qx_gemm_a8 with a few rows): the segmented
// small-batch structure of the fp16 kernel (R rows per block, k walked in
// segments of S chunks, one item per lane and segment) with the int8 products of
// the A8 GEMV, each chunk multiplied with the M staged rows. Vectors past m repeat
// row m - 1 and are not stored. LDS: M staged segments (S chunks of 144 bytes
// each), M*S*(128/G) group sums of xq, then R*S*M lane totals.
template <int BITS, int G, int M>
__global__ __launch_bounds__(512) void gemv_a8_multi_kernel(const char* __restrict__ packed,
                                                            const int8_t* __restrict__ Xq,
                                                            const float* __restrict__ sxp,
                                                            uint16_t* __restrict__ Y, int n, int k, int m,
                                                            int R, int S) {
  extern __shared__ __align__(16) char smem[];
  constexpr int NG = 128 / G;
  const int C = k >> 7, G_row = k / G, nthreads = blockDim.x;
  const size_t meta_off = (size_t)n * k * BITS / 8;
  const int row0 = blockIdx.x * R;
  const int rows = min(R, n - row0);
  const int xbytes = S * kX8Block;
  float* gs = reinterpret_cast<float*>(smem + M * xbytes);  // [M][S*NG]
  float* part = gs + M * S * NG;                             // [M][R*S]
  const int t = threadIdx.x, r = t / S, c = t - r * S;
  const int row = row0 + min(r, rows - 1);
  const int nseg = (C + S - 1) / S;

  float tot[M];
#pragma unroll
  for (int v = 0; v < M; ++v) tot[v] = 0.f;
  for (int seg = 0; seg < nseg; ++seg) {
    const int cs = min(S, C - seg * S);
    // every thread holds at most one 8-byte piece per row and segment (the launcher
    // makes blockDim.x >= 16*S)
    u32x2 xr[M][1];
#pragma unroll
    for (int v = 0; v < M; ++v) {
      const u32x2* src = reinterpret_cast<const u32x2*>(Xq + (size_t)min(v, m - 1) * k) + seg * S * 16;
      xr[v][0] = src[min(t, cs * 16 - 1)];
    }
    CodesA8<BITS, G> it;
    load_codes_a8<BITS, G>(it, packed, meta_off, row, seg * S + min(c, cs - 1), C, G_row);
    if (seg > 0) __syncthreads();  // the previous segment is no longer read
#pragma unroll
    for (int v = 0; v < M; ++v) stage_xq_a8<BITS, G, 1>(xr[v], cs, smem + v * xbytes, gs + v * S * NG, nthreads);
    __syncthreads();
    if (c < cs) {
#pragma unroll
      for (int v = 0; v < M; ++v)
        tot[v] += chunk_dot_a8<BITS, G>(it, smem + v * xbytes + c * kX8Block, gs + v * S * NG + c * NG);
    }
  }
  if (r < rows) {
#pragma unroll
    for (int v = 0; v < M; ++v) part[v * R * S + t] = tot[v];
  }
  __syncthreads();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int mm = min(m, M), items = rows * mm;
  for (int q = wave; q < items; q += nthreads >> 6) {
    const int rr = q / mm, v = q - rr * mm;
    float s = lane < S ? part[v * R * S + rr * S + lane] : 0.f;
    s = wave_sum(s);
    if (lane == 63) Y[(size_t)v * n + row0 + rr] = (uint16_t)float_to_half_bits(s * sxp[v]);
  }
}

template <int BITS, int G, bool PREQ>
int launch_gemv_a8_t(const qx_desc* d, const void* packed, const void* x, const float* sx, uint16_t* y,
                     hipStream_t s) {
  const char* p = static_cast<const char*>(packed);
  const int C = d->k / 128;
  constexpr int WPB = 4;
  if (C == 32 || C == 64) {
    const int rpb = WPB * 64 / C;
    const dim3 grid((unsigned)((d->n + rpb - 1) / rpb)), block(64 * WPB);
    if (C == 32)
      hipLaunchKernelGGL((gemv_a8_wave_kernel<BITS, G, 32, WPB, PREQ>), grid, block, 0, s, p, x, sx, y, d->n);
    else
      hipLaunchKernelGGL((gemv_a8_wave_kernel<BITS, G, 64, WPB, PREQ>), grid, block, 0, s, p, x, sx, y, d->n);
  } else if (C <= 88) {
    int R, threads;
    gemv_row_shape(d->n, C, false, &R, &threads);
    const size_t lds = (size_t)C * kX8Block + (size_t)(R * C + C * (128 / G)) * sizeof(float);
    const int xp = (C * 16 + threads - 1) / threads;
    const dim3 grid((unsigned)((d->n + R - 1) / R)), block(threads);
    if (xp <= 1)
      hipLaunchKernelGGL((gemv_a8_row_kernel<BITS, G, 1, PREQ>), grid, block, lds, s, p, x, sx, y, d->n, d->k, R);
    else if (xp <= 2)
      hipLaunchKernelGGL((gemv_a8_row_kernel<BITS, G, 2, PREQ>), grid, block, lds, s, p, x, sx, y, d->n, d->k, R);
    else
      hipLaunchKernelGGL((gemv_a8_row_kernel<BITS, G, 6, PREQ>), grid, block, lds, s, p, x, sx, y, d->n, d->k, R);
  } else {
    return QX_E_UNSUPPORTED;
  }
  return hipGetLastError() == hipSuccess ? QX_OK : QX_E_HIP;
}

}  // namespace

int launch_gemv_a8(const qx_desc* d, const void* packed, const uint16_t* x, uint16_t* y, hipStream_t s) {
  if (d->kind != QX_UNIFORM) return launch_gemv_lut_a8(d, packed, x, y, s);
#define QX_A8_CASE(B, G) \
  if (d->bits == B && d->group == G) return launch_gemv_a8_t<B, G, false>(d, packed, x, nullptr, y, s);
  QX_A8_CASE(3, 32) QX_A8_CASE(3, 64) QX_A8_CASE(3, 128)
  QX_A8_CASE(4, 32) QX_A8_CASE(4, 64) QX_A8_CASE(4, 128)
#undef QX_A8_CASE
  return QX_E_UNSUPPORTED;
}

int launch_gemv_a8_multi(const qx_desc* d, const void* packed, int m, const int8_t* Xq, const float* sx,
                         uint16_t* Y, hipStream_t s) {
  if (d->kind != QX_UNIFORM || m < 2 || m > 4) return QX_E_UNSUPPORTED;
  const int C = d->k / 128, S = std::min(C, 32);
  // R rows per block: R*S lanes fill blocks of at least 512 threads best (16 rows at S = 32)
  const int r_max = std::min(256, 512 / S);
  int R = r_max;
  double best_u = -1.0;
  for (int r = 1; r <= r_max; ++r) {
    const int th = 64 * ((r * S + 63) / 64);
    if (th < 512 && r < r_max) continue;
    const double u = (double)(r * S) / th;
    if (u > best_u + 1e-9) { best_u = u; R = r; }
  }
  const int threads = 64 * ((R * S + 63) / 64);
  if (threads < 16 * S || threads > 512) return QX_E_UNSUPPORTED;  // never with the shapes above
  const int M = m <= 2 ? 2 : 4, NG = 128 / d->group;
  const size_t lds = (size_t)M * S * kX8Block + (size_t)M * S * NG * 4 + (size_t)M * R * S * 4;
  const dim3 grid((unsigned)((d->n + R - 1) / R)), block(threads);
  const char* p = static_cast<const char*>(packed);
#define QX_A8M_CASE(B, G)                                                                                  \
  if (d->bits == B && d->group == G) {                                                                     \
    if (M == 2)                                                                                            \
      hipLaunchKernelGGL((gemv_a8_multi_kernel<B, G, 2>), grid, block, lds, s, p, Xq, sx, Y, d->n, d->k, m, R, S); \
    else                                                                                                   \
      hipLaunchKernelGGL((gemv_a8_multi_kernel<B, G, 4>), grid, block, lds, s, p, Xq, sx, Y, d->n, d->k, m, R, S); \
    return hipGetLastError() == hipSuccess ? QX_OK : QX_E_HIP;                                            \
  }
  QX_A8M_CASE(3, 32) QX_A8M_CASE(3, 64) QX_A8M_CASE(3, 128)
  QX_A8M_CASE(4, 32) QX_A8M_CASE(4, 64) QX_A8M_CASE(4, 128)
#undef QX_A8M_CASE
  return QX_E_UNSUPPORTED;
}

int launch_gemv_a8q(const qx_desc* d, const void* packed, const int8_t* xq, const float* sx, uint16_t* y,
                    hipStream_t s) {
  if (d->kind != QX_UNIFORM) return QX_E_UNSUPPORTED;
#define QX_A8_CASE(B, G) \
  if (d->bits == B && d->group == G) return launch_gemv_a8_t<B, G, true>(d, packed, xq, sx, y, s);
  QX_A8_CASE(3, 32) QX_A8_CASE(3, 64) QX_A8_CASE(3, 128)
  QX_A8_CASE(4, 32) QX_A8_CASE(4, 64) QX_A8_CASE(4, 128)
#undef QX_A8_CASE
  return QX_E_UNSUPPORTED;
}

}  // namespace qx
