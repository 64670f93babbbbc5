// W·A8 for many activation rows: per-token int8 activations (qx_quantize_a8) and
// the integer-product GEMM of uniform codes on the matrix cores (qx_gemm_a8).
//
// Per row r of X: amax = max |x|, inv = 127 / amax, xq = nearest integer to the
// exact x * inv, s_x = amax / 127 (all fp32, as the A8 GEMV). Then
//   Y[r][n] = s_x[r] * sum_j s[n][j] * sum_{k in group j} (q[n][k] - z[n][j]) * xq[r][k]
// with the group sums exact int32 from v_mfma_i32_16x16x32_i8: the B operand is
// q - z as int8 (one byte subtract per four codes, no borrow since q | 0x80 > z),
// the A operand xq, and each k-step of 32 codes lies in one group (g >= 32), so a
// group's int32 tile is scaled by its s and added to an fp32 tile when it ends.
//
// Work split: a block of W waves (4, or 8 for rows of more than 64 chunks) owns
// 16*(W/KS) weight rows (the MFMA columns; 16 per group of KS waves) and 16*MT
// activation rows (the MFMA rows), and walks k KS chunks at a
// time, wave ks of a group taking chunk ks: the chunks' activation tiles, codes and
// group words go to LDS, the next ones are loaded into registers meanwhile, and the
// KS partial tiles are added through LDS at the end. Lane group g (lane / 16) of
// k-step T takes the 8 consecutive codes of slot 4T + g; the slots are chosen so
// that the four lane groups decode one field kind per step (3-bit: bits 0-2, bits
// 3-5 or the spare codes), with per-lane byte offsets and shifts.
#include "qx_device.h"
#include "qx_internal.h"

namespace qx {
namespace {

constexpr int kA8Threads = 256;
#ifndef QX_A8_WIDE
// rows of more than 64 chunks take 8-wave blocks with twice the k split, the same weight
// rows per block (4096x11008 uniform-3 at m = 16 / 64 / 512: 19.9 / 33.1 / 94.9 ->
// 13.6 / 24.9 / 81.2 us; 11008x4096 unchanged); 0 keeps the 4-wave shapes
#define QX_A8_WIDE 1
#endif
typedef int32_t i4_t __attribute__((ext_vector_type(4)));

// x * inv + 1.5 * 2^23 in one fused multiply-add: its single rounding is the
// nearest-even integer to the exact product, whose low byte is the int8 code.
__device__ __forceinline__ uint32_t q8(_Float16 v, float inv) {
  return __builtin_bit_cast(uint32_t, __builtin_fmaf((float)v, inv, 12582912.0f));
}
__device__ __forceinline__ uint32_t pack4(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  return perm(perm(d, c, 0x04000C0Cu), perm(b, a, 0x0C0C0400u), 0x07060100u);
}

// One block per activation row: the row's maximum magnitude, then its int8 codes
// in natural order and its scale.
__global__ __launch_bounds__(kA8Threads) void quantize_a8_kernel(const uint16_t* __restrict__ X,
                                                                 int8_t* __restrict__ Xq,
                                                                 float* __restrict__ sx, int k) {
  __shared__ float red[kA8Threads / 64];
  const int row = blockIdx.x, np = k >> 3;
  const u32x4* src = reinterpret_cast<const u32x4*>(X + (size_t)row * k);
  h2_t mh = {(_Float16)0, (_Float16)0};
  for (int p = threadIdx.x; p < np; p += kA8Threads) {
    const u32x4 v = src[p];
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int t = 0; t < 4; ++t)
      mh = __builtin_elementwise_max(mh, __builtin_elementwise_abs(__builtin_bit_cast(h2_t, w[t])));
  }
  float m = fmaxf((float)mh.x, (float)mh.y);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  float amax = 0.f;
#pragma unroll
  for (int i = 0; i < kA8Threads / 64; ++i) amax = fmaxf(amax, red[i]);
  const float inv = amax > 0.f ? 127.f / amax : 0.f;
  u32x2* dst = reinterpret_cast<u32x2*>(Xq + (size_t)row * k);
  for (int p = threadIdx.x; p < np; p += kA8Threads) {
    const u32x4 v = src[p];
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    uint32_t q[8];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const h2_t h = __builtin_bit_cast(h2_t, w[t]);
      q[2 * t] = q8(h.x, inv);
      q[2 * t + 1] = q8(h.y, inv);
    }
    dst[p] = u32x2{pack4(q[0], q[1], q[2], q[3]), pack4(q[4], q[5], q[6], q[7])};
  }
  if (threadIdx.x == 0) sx[row] = amax > 0.f ? amax / 127.f : 0.f;
}

// q - z as int8 bytes of four codes q (bytes < 16) and z replicated in each byte.
__device__ __forceinline__ uint32_t minus_z(uint32_t q, uint32_t zz) {
  return ((q | 0x80808080u) - zz) ^ 0x80808080u;
}

// Codes of slot 4T + g (8 consecutive codes, natural order) from the 16*BITS bytes
// of one (row, chunk), as two dwords of bytes.
template <int BITS, int T>
__device__ __forceinline__ u32x2 slot_codes(const char* cb, int g) {
  if constexpr (BITS == 4) {
    const uint32_t D = *reinterpret_cast<const uint32_t*>(cb + 16 * T + 4 * g);
    const uint32_t lo = D & 0x0F0F0F0Fu, hi = (D >> 4) & 0x0F0F0F0Fu;
    return u32x2{perm(hi, lo, 0x05010400u), perm(hi, lo, 0x07030602u)};
  } else if constexpr (T < 3) {
    // T = 0: bits 0-2 of dwords 2g, 2g+1; T = 1: bits 0-2 of dwords 8+2g, 9+2g (g < 2)
    // or bits 3-5 of dwords 2(g-2), 2(g-2)+1; T = 2: bits 3-5 of dwords 4+2g, 5+2g
    const int off = T == 0 ? 8 * g : T == 1 ? (g < 2 ? 32 + 8 * g : 8 * (g - 2)) : 16 + 8 * g;
    const uint32_t sh = T == 0 ? 0u : T == 1 ? (g < 2 ? 0u : 3u) : 3u;
    const u32x2 D = *reinterpret_cast<const u32x2*>(cb + off);
    return u32x2{(D.x >> sh) & 0x07070707u, (D.y >> sh) & 0x07070707u};
  } else {
    // spare codes 96 + 8g' .. (g' = g): bits 0-1 in bits 6-7 of bytes 8g.., bit 2 in
    // bit 6 + g/2 of bytes 32 + 8(g%2) ..
    const u32x2 L = *reinterpret_cast<const u32x2*>(cb + 8 * g);
    const u32x2 H = *reinterpret_cast<const u32x2*>(cb + 32 + 8 * (g & 1));
    const uint32_t sh = 4u + (uint32_t)(g >> 1);
    return u32x2{((L.x >> 6) & 0x03030303u) | ((H.x >> sh) & 0x04040404u),
                 ((L.y >> 6) & 0x03030303u) | ((H.y >> sh) & 0x04040404u)};
  }
}

template <int BITS, int G, int MT, int KS, int W = 4>
__global__ __launch_bounds__(64 * W) void gemm_a8_kernel(const char* __restrict__ packed,
                                                             const int8_t* __restrict__ Xq,
                                                             const float* __restrict__ sx,
                                                             uint16_t* __restrict__ Y, int n, int k,
                                                             int m) {
  constexpr int NTH = 64 * W;
  constexpr int NW = W / KS;                // wave groups on different weight rows
  static_assert(W % KS == 0, "the k split divides the waves");
  constexpr int BM = 16 * MT, BN = 16 * NW, NG = 128 / G;
  constexpr int CS = 80;        // LDS bytes per weight row of the code tile (bank-spread rows)
  constexpr int XS = 144;       // LDS bytes per activation row of the activation tile
  constexpr int XPC = KS * BM * 8;   // 16-byte activation pieces per step (KS chunks)
  constexpr int XP = (XPC + NTH - 1) / NTH;
  constexpr int CPC = KS * BN * BITS;  // 16-byte code pieces per step
  constexpr int CP = (CPC + NTH - 1) / NTH;
  constexpr int MPC = KS * BN * NG;  // group words per step
  constexpr int MP = (MPC + NTH - 1) / NTH;
  static_assert((KS - 1) * NW * MT * 1024 <= KS * BM * XS, "the k-split reduction must fit the LDS tile");
  __shared__ __align__(16) char xs[KS * BM * XS];
  __shared__ __align__(16) char cs[KS * BN * CS];
  __shared__ uint32_t ms[KS * BN * NG];

  const int n0 = blockIdx.x * BN, m0 = blockIdx.y * BM;
  const int C = k >> 7, G_row = k / G;
  const size_t meta_off = (size_t)n * k * BITS / 8;
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63, g = lane >> 4, li = lane & 15;
  const int ks = wave % KS, wr = wave / KS;  // this wave's chunk within a step, weight-row group

  // chunks c0 .. c0 + KS - 1 of the tiles into registers (rows and chunks clamped in
  // bounds; clamped copies are never multiplied or stored)
  u32x4 xr[XP], cr[CP];
  uint32_t mr[MP];
  auto load = [&](int c0) {
#pragma unroll
    for (int i = 0; i < XP; ++i) {
      const int p = min(t + i * NTH, XPC - 1);
      const int q = p / (BM * 8), pr = p % (BM * 8);
      const int row = min(m0 + (pr >> 3), m - 1), c = min(c0 + q, C - 1);
      xr[i] = *reinterpret_cast<const u32x4*>(Xq + (size_t)row * k + (size_t)c * 128 + (pr & 7) * 16);
    }
#pragma unroll
    for (int i = 0; i < CP; ++i) {
      const int p = min(t + i * NTH, CPC - 1);
      const int q = p / (BN * BITS), pr = p % (BN * BITS);
      const int row = min(n0 + pr / BITS, n - 1), sl = pr % BITS, c = min(c0 + q, C - 1);
      cr[i] = *reinterpret_cast<const u32x4*>(packed + (((size_t)row * BITS + sl) * C + c) * 16);
    }
#pragma unroll
    for (int i = 0; i < MP; ++i) {
      const int p = min(t + i * NTH, MPC - 1);
      const int q = p / (BN * NG), pr = p % (BN * NG);
      const int row = min(n0 + pr / NG, n - 1), c = min(c0 + q, C - 1);
      mr[i] = *reinterpret_cast<const uint32_t*>(packed + meta_off + ((size_t)row * G_row + c * NG + pr % NG) * 4);
    }
  };
  auto store = [&]() {
#pragma unroll
    for (int i = 0; i < XP; ++i) {
      const int p = t + i * NTH;
      if (XPC % NTH == 0 || p < XPC) *reinterpret_cast<u32x4*>(xs + (p >> 3) * XS + (p & 7) * 16) = xr[i];
    }
#pragma unroll
    for (int i = 0; i < CP; ++i) {
      const int p = t + i * NTH;
      if (CPC % NTH == 0 || p < CPC) *reinterpret_cast<u32x4*>(cs + (p / BITS) * CS + (p % BITS) * 16) = cr[i];
    }
#pragma unroll
    for (int i = 0; i < MP; ++i) {
      const int p = t + i * NTH;
      if (MPC % NTH == 0 || p < MPC) ms[p] = mr[i];
    }
  };

  f4_t acc[MT];
  i4_t part[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    acc[mt] = f4_t{0.f, 0.f, 0.f, 0.f};
    part[mt] = i4_t{0, 0, 0, 0};
  }
  load(0);
  store();
  __syncthreads();
  // this wave's tiles: activation rows of chunk ks, weight row (MFMA column) li of group wr
  const char* xw = xs + ks * BM * XS;
  const char* crow = cs + (ks * BN + 16 * wr + li) * CS;
  const uint32_t* mrow = ms + (ks * BN + 16 * wr + li) * NG;
  for (int c0 = 0; c0 < C; c0 += KS) {
    if (c0 + KS < C) load(c0 + KS);
    if (c0 + ks < C) {
#define QX_A8_KSTEP(T)                                                                          \
  {                                                                                             \
    constexpr int grp = (32 * (T)) / G;                                                         \
    const uint32_t w = mrow[grp];                                                               \
    const uint32_t z = (uint32_t)(float)__builtin_bit_cast(_Float16, (uint16_t)(w >> 16));      \
    const uint32_t zz = z * 0x01010101u;                                                        \
    const u32x2 q = slot_codes<BITS, T>(crow, g);                                               \
    const long b = (long)(((uint64_t)minus_z(q.y, zz) << 32) | minus_z(q.x, zz));               \
    _Pragma("unroll") for (int mt = 0; mt < MT; ++mt) {                                         \
      const long a = *reinterpret_cast<const long*>(xw + (16 * mt + li) * XS + 32 * (T) + 8 * g); \
      part[mt] = __builtin_amdgcn_mfma_i32_16x16x32_i8(a, b, part[mt], 0, 0, 0);                \
    }                                                                                           \
    if constexpr ((32 * ((T) + 1)) % G == 0) { /* the group ends: scale and add */              \
      const float s = (float)__builtin_bit_cast(_Float16, (uint16_t)(w & 0xFFFFu));             \
      _Pragma("unroll") for (int mt = 0; mt < MT; ++mt) {                                       \
        _Pragma("unroll") for (int r = 0; r < 4; ++r) acc[mt][r] += s * (float)part[mt][r];     \
        part[mt] = i4_t{0, 0, 0, 0};                                                            \
      }                                                                                         \
    }                                                                                           \
  }
      QX_A8_KSTEP(0)
      QX_A8_KSTEP(1)
      QX_A8_KSTEP(2)
      QX_A8_KSTEP(3)
#undef QX_A8_KSTEP
    }
    __syncthreads();  // every wave is done with these chunks
    if (c0 + KS < C) {
      store();
      __syncthreads();
    }
  }

  // KS partial tiles -> one, in ks order, through LDS (every wave passed the last barrier)
  if constexpr (KS > 1) {
    float* red = reinterpret_cast<float*>(xs);
    if (ks > 0) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        *reinterpret_cast<f4_t*>(red + (((ks - 1) * NW + wr) * MT + mt) * 256 + 4 * lane) = acc[mt];
    }
    __syncthreads();
    if (ks > 0) return;
#pragma unroll
    for (int q = 1; q < KS; ++q)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        acc[mt] += *reinterpret_cast<const f4_t*>(red + (((q - 1) * NW + wr) * MT + mt) * 256 + 4 * lane);
  }

  // D of a 16x16 tile: lane holds activation rows 4g + r, weight row (column) li
  const int col = n0 + 16 * wr + li;
  if (col < n) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + 16 * mt + 4 * g + r;
        if (row < m) Y[(size_t)row * n + col] = (uint16_t)float_to_half_bits(sx[row] * acc[mt][r]);
      }
  }
}

template <int BITS, int G, int MT, int KS, int W = 4>
void launch_a8_cfg(const qx_desc* d, const char* p, int m, const int8_t* Xq, const float* sx, uint16_t* Y,
                   hipStream_t s) {
  constexpr int BN = 16 * (W / KS), BM = 16 * MT;
  const dim3 grid((unsigned)((d->n + BN - 1) / BN), (unsigned)((m + BM - 1) / BM));
  hipLaunchKernelGGL((gemm_a8_kernel<BITS, G, MT, KS, W>), grid, dim3(64 * W), 0, s, p, Xq, sx, Y, d->n, d->k, m);
}

// Tiles by m: few activation rows split each weight tile's chunks over the four
// waves (more blocks, k-split partials added through LDS); many rows give each
// wave 64 activation rows so that each decoded code feeds four MFMAs, and still
// split k when 64 x 64 tiles would leave fewer than 512 blocks (e.g. 4096 weight
// rows at m = 128: 128 blocks with the whole k, 512 with it split four ways).
template <int BITS, int G>
int launch_gemm_a8_t(const qx_desc* d, const char* p, int m, const int8_t* Xq, const float* sx, uint16_t* Y,
                     hipStream_t s) {
  const long tiles64 = (long)((d->n + 63) / 64) * ((m + 63) / 64);
  const bool wide = QX_A8_WIDE && d->k > 64 * 128;  // long rows: twice the waves, each walking half the chunks
  if (m <= 16) {
    if (wide) launch_a8_cfg<BITS, G, 1, 8, 8>(d, p, m, Xq, sx, Y, s);
    else launch_a8_cfg<BITS, G, 1, 4>(d, p, m, Xq, sx, Y, s);
  } else if (m <= 64) {
    if (wide) launch_a8_cfg<BITS, G, 2, 4, 8>(d, p, m, Xq, sx, Y, s);
    else launch_a8_cfg<BITS, G, 2, 2>(d, p, m, Xq, sx, Y, s);
  } else if (tiles64 < 256) {
    launch_a8_cfg<BITS, G, 4, 4>(d, p, m, Xq, sx, Y, s);
  } else if (tiles64 < 512) {
    if (wide) launch_a8_cfg<BITS, G, 4, 4, 8>(d, p, m, Xq, sx, Y, s);
    else launch_a8_cfg<BITS, G, 4, 2>(d, p, m, Xq, sx, Y, s);
  } else {
    if (wide) launch_a8_cfg<BITS, G, 4, 2, 8>(d, p, m, Xq, sx, Y, s);
    else launch_a8_cfg<BITS, G, 4, 1>(d, p, m, Xq, sx, Y, s);
  }
  return hipGetLastError() == hipSuccess ? QX_OK : QX_E_HIP;
}

}  // namespace

int launch_quantize_a8(int m, int k, const uint16_t* X, int8_t* Xq, float* sx, hipStream_t s) {
  hipLaunchKernelGGL(quantize_a8_kernel, dim3((unsigned)m), dim3(kA8Threads), 0, s, X, Xq, sx, k);
  return hipGetLastError() == hipSuccess ? QX_OK : QX_E_HIP;
}

int launch_gemm_a8(const qx_desc* d, const void* packed, int m, const int8_t* Xq, const float* sx, uint16_t* Y,
                   hipStream_t s) {
  const char* p = static_cast<const char*>(packed);
#define QX_A8G_CASE(B, G) \
  if (d->bits == B && d->group == G) return launch_gemm_a8_t<B, G>(d, p, m, Xq, sx, Y, s);
  QX_A8G_CASE(3, 32) QX_A8G_CASE(3, 64) QX_A8G_CASE(3, 128)
  QX_A8G_CASE(4, 32) QX_A8G_CASE(4, 64) QX_A8G_CASE(4, 128)
#undef QX_A8G_CASE
  return QX_E_UNSUPPORTED;
}

}  // namespace qx
