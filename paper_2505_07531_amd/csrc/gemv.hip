// Batch-1 quantized GEMV: y = W' x, W' dequantized on the fly from the packed
// layout. Decoding is memory-bound (Section 2.4 of the paper), so the kernel
// is built around streaming the packed bytes once at full HBM width:
//
//   * work item = (row, 128-code chunk); a lane reads its chunk as b 16-byte
//     loads from the slice planes, so each load instruction of a wave covers
//     contiguous 16-byte pieces of one plane;
//   * every load of a lane's items is issued before any is consumed;
//   * x is staged once per workgroup in LDS, permuted into the pair order the
//     decoders produce and padded so that lanes on consecutive chunks hit
//     different banks;
//   * codes are decoded in registers (qx_device.h) and multiplied with
//     v_dot2_f32_f16 (exact fp16 products, fp32 sums); uniform groups are
//     scaled once per group;
//   * per-chunk partial sums go through LDS and are reduced per row by one
//     wave with DPP/shuffles, in a fixed order (deterministic; no atomics).
//
// Launch: 256 threads; block b owns rows [R*b, R*b + R); items are the R x CT
// (row, chunk) pairs of a K tile of CT <= 88 chunks, dealt round-robin to the
// 256 lanes (ITEMS per lane). K longer than 88 chunks is walked in tiles of 64.
#include "qx_device.h"
#include "qx_internal.h"

namespace qx {

constexpr int kThreads = 256;
constexpr int kMaxTileChunks = 88;
constexpr int kLongTileChunks = 64;
constexpr int kXBlock = 272;  // bytes of LDS per chunk of x: 256 + 16 padding

// Stage x[k0 .. k0 + 128*ct) into LDS in decoder pair order.
template <int BITS>
__device__ __forceinline__ void stage_x(const uint16_t* __restrict__ x, int c0, int ct,
                                        char* xs) {
  const uint4* src = reinterpret_cast<const uint4*>(x) + (size_t)c0 * 16;
  for (int p = threadIdx.x; p < ct * 16; p += kThreads) {
    const uint4 v = src[p];
    uint4 o;
    if (BITS == 4) {  // [x0 x1][x2 x3][x4 x5][x6 x7] -> [x0 x4][x2 x6][x1 x5][x3 x7]
      o.x = perm(v.z, v.x, 0x05040100u);
      o.y = perm(v.w, v.y, 0x05040100u);
      o.z = perm(v.z, v.x, 0x07060302u);
      o.w = perm(v.w, v.y, 0x07060302u);
    } else {  // per 4: [x0 x1][x2 x3] -> [x0 x2][x1 x3]
      o.x = perm(v.y, v.x, 0x05040100u);
      o.y = perm(v.y, v.x, 0x07060302u);
      o.z = perm(v.w, v.z, 0x05040100u);
      o.w = perm(v.w, v.z, 0x07060302u);
    }
    *reinterpret_cast<uint4*>(xs + (p >> 4) * kXBlock + (p & 15) * 16) = o;
  }
}

// Raw bytes of one item: codes (4*BITS dwords) and its group tables.
template <int BITS, int KIND, int G>
struct Item {
  static constexpr int kGroups = 128 / G;
  static constexpr int kMetaDw = KIND == 0 ? kGroups : kGroups * (1 << BITS) / 2;
  uint32_t d[4 * BITS];
  uint32_t m[kMetaDw];
};

template <int BITS, int KIND, int G>
__device__ __forceinline__ void load_item(Item<BITS, KIND, G>& it, const char* __restrict__ packed,
                                          size_t meta_off, int row, int c, int C, int G_row) {
  const u32x4* code = reinterpret_cast<const u32x4*>(packed) + ((size_t)row * BITS * C + c);
#pragma unroll
  for (int s = 0; s < BITS; ++s) {
    const u32x4 v = __builtin_nontemporal_load(code + (size_t)s * C);
    it.d[4 * s + 0] = v.x; it.d[4 * s + 1] = v.y; it.d[4 * s + 2] = v.z; it.d[4 * s + 3] = v.w;
  }
  constexpr int kDw = Item<BITS, KIND, G>::kMetaDw;
  const size_t gidx = (size_t)row * G_row + (size_t)c * (128 / G);
  const size_t moff = meta_off + gidx * (KIND == 0 ? 4 : 2 * (1 << BITS));
  const uint32_t* mp = reinterpret_cast<const uint32_t*>(packed + moff);
  if constexpr (kDw % 4 == 0) {
#pragma unroll
    for (int i = 0; i < kDw / 4; ++i) {
      const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(mp) + i);
      it.m[4 * i + 0] = v.x; it.m[4 * i + 1] = v.y; it.m[4 * i + 2] = v.z; it.m[4 * i + 3] = v.w;
    }
  } else if constexpr (kDw == 2) {
    const u32x2 v = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(mp));
    it.m[0] = v.x; it.m[1] = v.y;
  } else {
    it.m[0] = __builtin_nontemporal_load(mp);
  }
}

// Partial dot product of one chunk with its x block (LDS, pair order).
template <int BITS, int KIND, int G>
__device__ __forceinline__ float chunk_dot(const Item<BITS, KIND, G>& it, const char* xb) {
  constexpr int NG = 128 / G;
  const uint4* xv = reinterpret_cast<const uint4*>(xb);
  if constexpr (BITS == 4 && KIND == 0) {
    float part = 0.f;
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const UniformGroup ug = uniform_group(it.m[g]);
      float acc = 0.f;
#pragma unroll
      for (int j = g * G / 8; j < (g + 1) * G / 8; ++j) {
        const uint4 x = xv[j];
        const uint32_t D = it.d[j];
        acc = dot2(hadd2((D & 0x000F000Fu) | kMagic1024, ug.z1024), x.x, acc);
        acc = dot2(hadd2(((D >> 8) & 0x000F000Fu) | kMagic1024, ug.z1024), x.y, acc);
        acc = dot2(hadd2(((D >> 4) & 0x000F000Fu) | kMagic1024, ug.z1024), x.z, acc);
        acc = dot2(hadd2(((D >> 12) & 0x000F000Fu) | kMagic1024, ug.z1024), x.w, acc);
      }
      part += ug.s * acc;
    }
    return part;
  } else if constexpr (BITS == 4 && KIND == 1) {
    float acc = 0.f;
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const LutGroup<4> t = lut_group<4>(&it.m[g * 8]);
#pragma unroll
      for (int j = g * G / 8; j < (g + 1) * G / 8; ++j) {
        const uint4 x = xv[j];
        const uint32_t D = it.d[j];
        uint32_t lo, hi;
        lut4_bytes(t, D & 0x0F0F0F0Fu, lo, hi);          // codes 0 2 4 6
        acc = dot2(perm(hi, lo, 0x06020400u), x.x, acc);  // (0, 4)
        acc = dot2(perm(hi, lo, 0x07030501u), x.y, acc);  // (2, 6)
        lut4_bytes(t, (D >> 4) & 0x0F0F0F0Fu, lo, hi);   // codes 1 3 5 7
        acc = dot2(perm(hi, lo, 0x06020400u), x.z, acc);  // (1, 5)
        acc = dot2(perm(hi, lo, 0x07030501u), x.w, acc);  // (3, 7)
      }
    }
    return acc;
  } else if constexpr (BITS == 3 && KIND == 0) {
    float acc[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) acc[g] = 0.f;
    UniformGroup ug[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) ug[g] = uniform_group(it.m[g]);
    // x dword index of code block t (codes 4t..4t+3) is 2t (pair 0,2) and 2t+1 (pair 1,3)
    const uint32_t* xd = reinterpret_cast<const uint32_t*>(xb);
#pragma unroll
    for (int i = 0; i < 12; ++i) {
      const uint32_t D = it.d[i];
      const U3Pairs p = u3_fields(D);
      const int ga = (4 * i) / G, gb = (48 + 4 * i) / G;
      const uint2 xa = *reinterpret_cast<const uint2*>(xd + 2 * i);
      const uint2 xb2 = *reinterpret_cast<const uint2*>(xd + 2 * (12 + i));
      acc[ga] = dot2(hadd2(p.a0, ug[ga].z1024), xa.x, acc[ga]);
      acc[ga] = dot2(hadd2(p.a1, ug[ga].z1024), xa.y, acc[ga]);
      acc[gb] = dot2(hadd2(p.b0, ug[gb].z128), xb2.x, acc[gb]);
      acc[gb] = dot2(hadd2(p.b1, ug[gb].z128), xb2.y, acc[gb]);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      uint32_t s0, s1;
      switch (i) {  // the bit-2 position depends on the dword index at compile time
        case 0: u3_spare<0>(it.d[0], it.d[8], s0, s1); break;
        case 1: u3_spare<1>(it.d[1], it.d[9], s0, s1); break;
        case 2: u3_spare<2>(it.d[2], it.d[10], s0, s1); break;
        case 3: u3_spare<3>(it.d[3], it.d[11], s0, s1); break;
        case 4: u3_spare<4>(it.d[4], it.d[8], s0, s1); break;
        case 5: u3_spare<5>(it.d[5], it.d[9], s0, s1); break;
        case 6: u3_spare<6>(it.d[6], it.d[10], s0, s1); break;
        default: u3_spare<7>(it.d[7], it.d[11], s0, s1); break;
      }
      const int gs = (96 + 4 * i) / G;
      const uint2 xs = *reinterpret_cast<const uint2*>(xd + 2 * (24 + i));
      acc[gs] = dot2(hadd2(s0, ug[gs].z16), xs.x, acc[gs]);
      acc[gs] = dot2(hadd2(s1, ug[gs].z16), xs.y, acc[gs]);
    }
    float part = 0.f;
#pragma unroll
    for (int g = 0; g < NG; ++g) part += ug[g].s * acc[g];
    return part;
  } else {  // BITS == 3, codebook
    LutGroup<3> t[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) t[g] = lut_group<3>(&it.m[g * 4]);
    const uint32_t* xd = reinterpret_cast<const uint32_t*>(xb);
    float acc = 0.f;
#pragma unroll
    for (int i = 0; i < 12; ++i) {
      const uint32_t D = it.d[i];
      const int ga = (4 * i) / G, gb = (48 + 4 * i) / G;
      uint32_t p02, p13;
      const uint2 xa = *reinterpret_cast<const uint2*>(xd + 2 * i);
      lut3_pairs(t[ga], u3_sel_a(D), p02, p13);
      acc = dot2(p02, xa.x, acc);
      acc = dot2(p13, xa.y, acc);
      const uint2 xb2 = *reinterpret_cast<const uint2*>(xd + 2 * (12 + i));
      lut3_pairs(t[gb], u3_sel_b(D), p02, p13);
      acc = dot2(p02, xb2.x, acc);
      acc = dot2(p13, xb2.y, acc);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      uint32_t S;
      switch (i) {
        case 0: S = u3_sel_spare<0>(it.d[0], it.d[8]); break;
        case 1: S = u3_sel_spare<1>(it.d[1], it.d[9]); break;
        case 2: S = u3_sel_spare<2>(it.d[2], it.d[10]); break;
        case 3: S = u3_sel_spare<3>(it.d[3], it.d[11]); break;
        case 4: S = u3_sel_spare<4>(it.d[4], it.d[8]); break;
        case 5: S = u3_sel_spare<5>(it.d[5], it.d[9]); break;
        case 6: S = u3_sel_spare<6>(it.d[6], it.d[10]); break;
        default: S = u3_sel_spare<7>(it.d[7], it.d[11]); break;
      }
      const int gs = (96 + 4 * i) / G;
      uint32_t p02, p13;
      lut3_pairs(t[gs], S, p02, p13);
      const uint2 xs = *reinterpret_cast<const uint2*>(xd + 2 * (24 + i));
      acc = dot2(p02, xs.x, acc);
      acc = dot2(p13, xs.y, acc);
    }
    return acc;
  }
}

template <int BITS, int KIND, int G, int ITEMS>
__global__ __launch_bounds__(kThreads) void gemv_kernel(const char* __restrict__ packed,
                                                         const uint16_t* __restrict__ x,
                                                         uint16_t* __restrict__ y, int n, int k,
                                                         int R) {
  extern __shared__ __align__(16) char smem[];
  const int C = k >> 7;
  const int G_row = k / G;
  const size_t meta_off = (size_t)n * k * BITS / 8;
  const int row0 = blockIdx.x * R;
  const int rows = min(R, n - row0);
  const int CT = C <= kMaxTileChunks ? C : kLongTileChunks;
  char* xs = smem;                                              // CT * kXBlock bytes
  float* part = reinterpret_cast<float*>(smem + CT * kXBlock);  // R * CT floats

  float acc[ITEMS];
#pragma unroll
  for (int j = 0; j < ITEMS; ++j) acc[j] = 0.f;

  for (int c0 = 0; c0 < C; c0 += CT) {
    const int ct = min(CT, C - c0);
    Item<BITS, KIND, G> it[ITEMS];
    bool valid[ITEMS];
    int cl[ITEMS];
#pragma unroll
    for (int j = 0; j < ITEMS; ++j) {
      const int i = threadIdx.x + j * kThreads;
      const int r = i / CT;
      cl[j] = i - r * CT;
      valid[j] = r < rows && cl[j] < ct;
      if (valid[j]) load_item<BITS, KIND, G>(it[j], packed, meta_off, row0 + r, c0 + cl[j], C, G_row);
    }
    if (c0 > 0) __syncthreads();  // previous tile's x no longer read
    stage_x<BITS>(x, c0, ct, xs);
    __syncthreads();
#pragma unroll
    for (int j = 0; j < ITEMS; ++j)
      if (valid[j]) acc[j] += chunk_dot<BITS, KIND, G>(it[j], xs + cl[j] * kXBlock);
  }

  // per-item partials -> LDS [R][CT], then one wave per row sums them in a fixed order
#pragma unroll
  for (int j = 0; j < ITEMS; ++j) {
    const int i = threadIdx.x + j * kThreads;
    if (i < R * CT) part[i] = acc[j];
  }
  __syncthreads();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int r = wave; r < rows; r += kThreads / 64) {
    float v = 0.f;
    for (int c = lane; c < CT; c += 64) v += part[r * CT + c];
    v = wave_sum(v);
    if (lane == 0) y[row0 + r] = (uint16_t)float_to_half_bits(v);
  }
}

// Rows per block and items per lane for an n x k matrix.
static void gemv_shape(int n, int k, int* R, int* items) {
  const int C = k / 128;
  const int CT = C <= kMaxTileChunks ? C : kLongTileChunks;
  int r = 8;
  while (r > 1 && (n + r - 1) / r < 512) r >>= 1;  // keep >= 512 blocks when n allows
  while (r > 1 && r * CT > 4 * kThreads) r >>= 1;
  *R = r;
  *items = (r * CT + kThreads - 1) / kThreads;
}

template <int BITS, int KIND, int G>
static int launch_gemv_t(const qx_desc* d, const void* packed, const uint16_t* x, uint16_t* y,
                         hipStream_t s) {
  int R, items;
  gemv_shape(d->n, d->k, &R, &items);
  const int C = d->k / 128;
  const int CT = C <= kMaxTileChunks ? C : kLongTileChunks;
  const size_t lds = (size_t)CT * kXBlock + (size_t)R * CT * sizeof(float);
  const dim3 grid((d->n + R - 1) / R), block(kThreads);
  const char* p = static_cast<const char*>(packed);
  switch (items) {
    case 1: hipLaunchKernelGGL((gemv_kernel<BITS, KIND, G, 1>), grid, block, lds, s, p, x, y, d->n, d->k, R); break;
    case 2: hipLaunchKernelGGL((gemv_kernel<BITS, KIND, G, 2>), grid, block, lds, s, p, x, y, d->n, d->k, R); break;
    case 3: hipLaunchKernelGGL((gemv_kernel<BITS, KIND, G, 3>), grid, block, lds, s, p, x, y, d->n, d->k, R); break;
    default: hipLaunchKernelGGL((gemv_kernel<BITS, KIND, G, 4>), grid, block, lds, s, p, x, y, d->n, d->k, R); break;
  }
  return hipGetLastError() == hipSuccess ? QX_OK : QX_E_HIP;
}

int launch_gemv(const qx_desc* d, const void* packed, const uint16_t* x, uint16_t* y,
                hipStream_t s) {
#define QX_GEMV_CASE(B, K, G) \
  if (d->bits == B && d->kind == K && d->group == G) return launch_gemv_t<B, K, G>(d, packed, x, y, s);
  QX_GEMV_CASE(3, 0, 32) QX_GEMV_CASE(3, 0, 64) QX_GEMV_CASE(3, 0, 128)
  QX_GEMV_CASE(3, 1, 32) QX_GEMV_CASE(3, 1, 64) QX_GEMV_CASE(3, 1, 128)
  QX_GEMV_CASE(4, 0, 32) QX_GEMV_CASE(4, 0, 64) QX_GEMV_CASE(4, 0, 128)
  QX_GEMV_CASE(4, 1, 32) QX_GEMV_CASE(4, 1, 64) QX_GEMV_CASE(4, 1, 128)
#undef QX_GEMV_CASE
  return QX_E_UNSUPPORTED;
}

}  // namespace qx
