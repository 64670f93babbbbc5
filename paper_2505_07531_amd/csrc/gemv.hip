// Batch-1 quantized GEMV: y = W' x, W' dequantized on the fly from the packed
// layout. Decoding is memory-bound (Section 2.4 of the paper), so the kernel
// is built around streaming the packed bytes once at full HBM width:
//
//   * work item = (row, 128-code chunk); a lane reads its chunk as b 16-byte
//     loads from the slice planes, so each load instruction of a wave covers
//     contiguous 16-byte pieces of one plane;
//   * x is loaded first (it is small and L2-resident), then every weight load
//     of the lane is issued before any is consumed; x is permuted into the pair
//     order of the decoders and staged once per workgroup in LDS, padded so
//     that lanes on consecutive chunks hit different banks;
//   * codes are decoded in registers (qx_device.h), one v_and_or_b32 per code
//     pair, and multiplied with v_dot2_f32_f16 (exact fp16 products, fp32
//     sums); uniform codes enter as M + q and the zero point is folded out
//     once per group with sums over x formed while x is staged, so no
//     instruction per pair subtracts it; groups are scaled once;
//   * partial sums are reduced per row in a fixed order with DPP (no atomics;
//     results are deterministic).
//
// Three launch paths, all with one 128-code chunk per lane (more resident
// waves measured faster than more chunks per lane):
//   wave kernel: K = 128*32 or 128*64, a row fills half or all of a wave and
//                is reduced in registers;
//   row kernel:  any other K up to 88 chunks, R rows per block sized to leave
//                few idle lanes, partials through LDS;
//   tile kernel: longer K, walked in tiles of 64 chunks.
#include "qx_device.h"
#include "qx_internal.h"

#include <algorithm>

namespace qx {

constexpr int kThreads = 256;
constexpr int kMaxTileChunks = 88;
constexpr int kLongTileChunks = 64;
constexpr int kXBlock = 272;                                   // LDS bytes per chunk of x

// x pieces [c0*16, (c0+ct)*16) of this thread, loaded into registers. Every load
// is issued (indices clamped in bounds) so the compiler can count outstanding
// loads and wait for x alone.
template <int XP>
__device__ __forceinline__ void load_x(const uint16_t* __restrict__ x, int c0, int ct,
                                       u32x4 (&xr)[XP], int stride = kThreads) {
  const u32x4* src = reinterpret_cast<const u32x4*>(x) + (size_t)c0 * 16;
#pragma unroll
  for (int i = 0; i < XP; ++i) {
    const int p = min((int)threadIdx.x + i * stride, ct * 16 - 1);
    xr[i] = src[p];
  }
}

// Sums over one 16-byte piece of x (8 natural-order values at chunk position
// 8*pc) for the folded zero point of uniform groups: sum x and sum M x, M the
// bias that the decoder adds to the code at each position (b = 4: 1024 at even,
// 64 at odd positions; b = 3: 1024 for codes 0-47, 128 for 48-95, 16 above).
// Products of fp16 values are exact in fp32.
template <int BITS>
__device__ __forceinline__ void piece_sums(const u32x4& v, int pc, float& sx, float& mx) {
  const uint32_t one = 0x3C003C00u;  // (1, 1)
  sx = dot2(v.w, one, dot2(v.z, one, dot2(v.y, one, dot2(v.x, one, 0.f))));
  if (BITS == 4) {
    const uint32_t m = 0x54006400u;  // (1024, 64)
    mx = dot2(v.w, m, dot2(v.z, m, dot2(v.y, m, dot2(v.x, m, 0.f))));
  } else {
    mx = (pc < 6 ? 1024.f : pc < 12 ? 128.f : 16.f) * sx;
  }
}

// Sum of v over aligned groups of N consecutive lanes (N = 4, 8, 16), in every lane.
template <int N>
__device__ __forceinline__ float lane_group_sum(float v) {
  v = dpp_plus<0xB1, 0xF>(v);                    // quad_perm [1,0,3,2]
  v = dpp_plus<0x4E, 0xF>(v);                    // quad_perm [2,3,0,1]
  if constexpr (N >= 8) v = dpp_plus<0x141, 0xF>(v);   // row_half_mirror
  if constexpr (N >= 16) v = dpp_plus<0x140, 0xF>(v);  // row_mirror
  return v;
}

// Permute the loaded pieces into decoder pair order and store them in LDS
// (piece p of the tile: chunk p / 16, values 8 (p % 16) ..). For uniform
// groups, also store (sum M x, sum x) per group of the tile in gs; the pieces
// of a group sit in consecutive lanes.
template <int BITS, int KIND, int G, int XP, bool EXACT = false>  // EXACT: every piece is in range
__device__ __forceinline__ void store_x(const u32x4 (&xr)[XP], int ct, char* xs, float2* gs,
                                        int stride = kThreads) {
#pragma unroll
  for (int i = 0; i < XP; ++i) {
    const int p = threadIdx.x + i * stride;
    const u32x4 v = xr[i];
    if (EXACT || p < ct * 16) {
      u32x4 o;
      if (BITS == 4) {  // [x0 x1][x2 x3][x4 x5][x6 x7] -> [x0 x4][x1 x5][x2 x6][x3 x7]
        o.x = perm(v.z, v.x, 0x05040100u);
        o.y = perm(v.z, v.x, 0x07060302u);
        o.z = perm(v.w, v.y, 0x05040100u);
        o.w = perm(v.w, v.y, 0x07060302u);
      } else {  // per 4: [x0 x1][x2 x3] -> [x0 x2][x1 x3]
        o.x = perm(v.y, v.x, 0x05040100u);
        o.y = perm(v.y, v.x, 0x07060302u);
        o.z = perm(v.w, v.z, 0x05040100u);
        o.w = perm(v.w, v.z, 0x07060302u);
      }
      *reinterpret_cast<u32x4*>(xs + (p >> 4) * kXBlock + (p & 15) * 16) = o;
    }
    if constexpr (KIND == QX_UNIFORM) {
      constexpr int PPG = G / 8;  // pieces per group
      float sx, mx;
      piece_sums<BITS>(v, p & 15, sx, mx);
      sx = lane_group_sum<PPG>(sx);
      mx = lane_group_sum<PPG>(mx);
      if ((p & (PPG - 1)) == 0 && (EXACT || p < ct * 16)) gs[p / PPG] = make_float2(mx, sx);
    }
  }
}

// Raw bytes of one item: codes (4*BITS dwords) and its group tables.
template <int BITS, int KIND, int G>
struct Item {
  static constexpr int kGroups = 128 / G;
  // Q4X: m[0] = the two groups' binary16 scales, m[1] = their selectors (bits 0-1, 2-3)
  static constexpr int kMetaDw = KIND == QX_Q4X ? 2 : KIND == 0 ? kGroups : kGroups * (1 << BITS) / 2;
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
  if constexpr (KIND == QX_Q4X) {  // groups 2c and 2c + 1 of the row
    const size_t sel_off = meta_off + meta_off / 16;  // after n*G binary16 scales (n*k/32 bytes)
    const int W = (G_row + 15) / 16;
    it.m[0] = __builtin_nontemporal_load(
        reinterpret_cast<const uint32_t*>(packed + meta_off + ((size_t)row * G_row + 2 * c) * 2));
    const uint32_t sw = __builtin_nontemporal_load(
        reinterpret_cast<const uint32_t*>(packed + sel_off + ((size_t)row * W + c / 8) * 4));
    it.m[1] = (sw >> (4 * (c % 8))) & 0xFu;
    return;
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

// Bit-2 source dword of spare codes of code dword I, and the two spare helpers
// dispatched on the compile-time index.
template <int I, int BITS, int KIND, int G>
__device__ __forceinline__ void spare_pairs(const Item<BITS, KIND, G>& it, const DecodeConsts& k,
                                            uint32_t& s0, uint32_t& s1) {
  u3_spare<I>(it.d[I], it.d[8 + (I & 3)], k, s0, s1);
}
template <int I, int BITS, int KIND, int G>
__device__ __forceinline__ uint32_t spare_sel(const Item<BITS, KIND, G>& it) {
  return u3_sel_spare<I>(it.d[I], it.d[8 + (I & 3)]);
}

// Scale and zero point of a uniform group word: s * (acc - sum M x - z sum x),
// with acc = sum (M + q) x over the group, is s * sum (q - z) x.
__device__ __forceinline__ float fold_group(uint32_t word, float acc, float2 gsum) {
  const float s = half_bits_to_float(word & 0xFFFFu), z = half_bits_to_float(word >> 16);
  return s * (acc - gsum.x - z * gsum.y);
}

// Partial dot product of one chunk with its x block (LDS, pair order). Uniform
// codes enter the products as M + q (no subtraction per pair); gs holds the
// chunk's (sum M x, sum x) per group and fold_group takes the zero point out.
template <int BITS, int KIND, int G>
__device__ __forceinline__ float chunk_dot(const Item<BITS, KIND, G>& it, const char* xb,
                                           const float2* gs, const DecodeConsts& k,
                                           const uint32_t* q4lut = nullptr) {
  constexpr int NG = 128 / G;
  const u32x4* xv = reinterpret_cast<const u32x4*>(xb);
  if constexpr (KIND == QX_Q4X) {
    // two groups of 64: the selected sub-codebook (lookup tables in LDS), the scale
    // applied once to each group's sum of table entries times x
    float part = 0.f;
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      const uint32_t* tp = q4lut + 8 * ((it.m[1] >> (2 * g)) & 3u);
      const u32x4 tl = *reinterpret_cast<const u32x4*>(tp), th = *reinterpret_cast<const u32x4*>(tp + 4);
      const LutGroup<4> t = {{tl.x, tl.y, tl.z, tl.w}, {th.x, th.y, th.z, th.w}};
      float acc = 0.f;
#pragma unroll
      for (int j = 8 * g; j < 8 * g + 8; ++j) {
        const u32x4 x = xv[j];
        const uint32_t D = it.d[j];
        uint32_t elo, ehi, olo, ohi;
        lut4_bytes(t, D & 0x0F0F0F0Fu, elo, ehi);         // codes 0 2 4 6
        lut4_bytes(t, (D >> 4) & 0x0F0F0F0Fu, olo, ohi);  // codes 1 3 5 7
        acc = dot2(perm(ehi, elo, 0x06020400u), x.x, acc);  // (0, 4)
        acc = dot2(perm(ohi, olo, 0x06020400u), x.y, acc);  // (1, 5)
        acc = dot2(perm(ehi, elo, 0x07030501u), x.z, acc);  // (2, 6)
        acc = dot2(perm(ohi, olo, 0x07030501u), x.w, acc);  // (3, 7)
      }
      part += half_bits_to_float((it.m[0] >> (16 * g)) & 0xFFFFu) * acc;
    }
    return part;
  } else if constexpr (BITS == 4 && KIND == 0) {
    float part = 0.f;
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      float acc = 0.f;
#pragma unroll
      for (int j = g * G / 8; j < (g + 1) * G / 8; ++j) {
        const u32x4 x = xv[j];
        const uint32_t D = it.d[j], Ds = D >> 8;
        acc = dot2((D & k.m000f) | k.mag1024, x.x, acc);   // (0, 4)
        acc = dot2((D & k.m00f0) | k.mag64, x.y, acc);     // (1, 5)
        acc = dot2((Ds & k.m000f) | k.mag1024, x.z, acc);  // (2, 6)
        acc = dot2((Ds & k.m00f0) | k.mag64, x.w, acc);    // (3, 7)
      }
      part += fold_group(it.m[g], acc, gs[g]);
    }
    return part;
  } else if constexpr (BITS == 4 && KIND == 1) {
    float acc = 0.f;
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const LutGroup<4> t = lut_group<4>(&it.m[g * 8]);
#pragma unroll
      for (int j = g * G / 8; j < (g + 1) * G / 8; ++j) {
        const u32x4 x = xv[j];
        const uint32_t D = it.d[j];
        uint32_t elo, ehi, olo, ohi;
        lut4_bytes(t, D & 0x0F0F0F0Fu, elo, ehi);         // codes 0 2 4 6
        lut4_bytes(t, (D >> 4) & 0x0F0F0F0Fu, olo, ohi);  // codes 1 3 5 7
        acc = dot2(perm(ehi, elo, 0x06020400u), x.x, acc);  // (0, 4)
        acc = dot2(perm(ohi, olo, 0x06020400u), x.y, acc);  // (1, 5)
        acc = dot2(perm(ehi, elo, 0x07030501u), x.z, acc);  // (2, 6)
        acc = dot2(perm(ohi, olo, 0x07030501u), x.w, acc);  // (3, 7)
      }
    }
    return acc;
  } else if constexpr (BITS == 3 && KIND == 0) {
    float acc[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) acc[g] = 0.f;
    // x dwords of code block t (codes 4t..4t+3): 2t = pair (0,2), 2t+1 = pair (1,3)
    const uint32_t* xd = reinterpret_cast<const uint32_t*>(xb);
#pragma unroll
    for (int i = 0; i < 12; ++i) {
      const U3Pairs p = u3_fields(it.d[i], k);
      const int ga = (4 * i) / G, gb = (48 + 4 * i) / G;
      const u32x2 xa = *reinterpret_cast<const u32x2*>(xd + 2 * i);
      const u32x2 xb2 = *reinterpret_cast<const u32x2*>(xd + 2 * (12 + i));
      acc[ga] = dot2(p.a0, xa.x, acc[ga]);
      acc[ga] = dot2(p.a1, xa.y, acc[ga]);
      acc[gb] = dot2(p.b0, xb2.x, acc[gb]);
      acc[gb] = dot2(p.b1, xb2.y, acc[gb]);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      uint32_t s0, s1;
      switch (i) {  // the bit-2 position depends on the dword index at compile time
        case 0: spare_pairs<0>(it, k, s0, s1); break;
        case 1: spare_pairs<1>(it, k, s0, s1); break;
        case 2: spare_pairs<2>(it, k, s0, s1); break;
        case 3: spare_pairs<3>(it, k, s0, s1); break;
        case 4: spare_pairs<4>(it, k, s0, s1); break;
        case 5: spare_pairs<5>(it, k, s0, s1); break;
        case 6: spare_pairs<6>(it, k, s0, s1); break;
        default: spare_pairs<7>(it, k, s0, s1); break;
      }
      const int gg = (96 + 4 * i) / G;
      const u32x2 xs = *reinterpret_cast<const u32x2*>(xd + 2 * (24 + i));
      acc[gg] = dot2(s0, xs.x, acc[gg]);
      acc[gg] = dot2(s1, xs.y, acc[gg]);
    }
    float part = 0.f;
#pragma unroll
    for (int g = 0; g < NG; ++g) part += fold_group(it.m[g], acc[g], gs[g]);
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
      const u32x2 xa = *reinterpret_cast<const u32x2*>(xd + 2 * i);
      lut3_pairs(t[ga], u3_sel_a(D), p02, p13);
      acc = dot2(p02, xa.x, acc);
      acc = dot2(p13, xa.y, acc);
      const u32x2 xb2 = *reinterpret_cast<const u32x2*>(xd + 2 * (12 + i));
      lut3_pairs(t[gb], u3_sel_b(D), p02, p13);
      acc = dot2(p02, xb2.x, acc);
      acc = dot2(p13, xb2.y, acc);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      uint32_t S;
      switch (i) {
        case 0: S = spare_sel<0>(it); break;
        case 1: S = spare_sel<1>(it); break;
        case 2: S = spare_sel<2>(it); break;
        case 3: S = spare_sel<3>(it); break;
        case 4: S = spare_sel<4>(it); break;
        case 5: S = spare_sel<5>(it); break;
        case 6: S = spare_sel<6>(it); break;
        default: S = spare_sel<7>(it); break;
      }
      const int gs = (96 + 4 * i) / G;
      uint32_t p02, p13;
      lut3_pairs(t[gs], S, p02, p13);
      const u32x2 xs = *reinterpret_cast<const u32x2*>(xd + 2 * (24 + i));
      acc = dot2(p02, xs.x, acc);
      acc = dot2(p13, xs.y, acc);
    }
    return acc;
  }
}

// Q4X: the matrix's 4 x 16 binary16 codebook as the v_perm lookup tables of
// lut4_bytes (per sub-codebook 4 dwords of low bytes, then 4 of high bytes),
// written to LDS by the first 16 threads of the block.
__device__ __forceinline__ void stage_q4x_lut(const char* __restrict__ packed, int n, int k,
                                              uint32_t* lut) {
  if (threadIdx.x < 16) {
    const int t = threadIdx.x >> 2, i = threadIdx.x & 3;
    const uint32_t* cb = reinterpret_cast<const uint32_t*>(packed + q4x_offsets(n, k).codebook) + 8 * t;
    const uint32_t w0 = cb[2 * i], w1 = cb[2 * i + 1];
    lut[8 * t + i] = perm(w1, w0, 0x06040200u);
    lut[8 * t + 4 + i] = perm(w1, w0, 0x07050301u);
  }
}

// K = 128*LPR with LPR in {32, 64}: a row's chunks fill LPR lanes of one wave, so
// each row is reduced in registers with DPP and stored by one lane; no LDS
// partials and no second barrier. A block has WPB waves and stages x once for
// its WPB*64/LPR rows.
template <int BITS, int KIND, int G, int LPR, int WPB>
__global__ __launch_bounds__(64 * WPB) void gemv_wave_kernel(const char* __restrict__ packed,
                                                             const uint16_t* __restrict__ x,
                                                             uint16_t* __restrict__ y, int n) {
  constexpr int C = LPR, NT = 64 * WPB, RPW = 64 / LPR, RPB = WPB * RPW;
  constexpr int XP = (C * 16 + NT - 1) / NT;
  __shared__ __align__(16) char xs[C * kXBlock];
  __shared__ float2 gs[KIND == QX_UNIFORM ? C * (128 / G) : 1];
  __shared__ __align__(16) uint32_t q4lut[KIND == QX_Q4X ? 32 : 1];
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
  store_x<BITS, KIND, G, XP, C * 16 % NT == 0>(xr, C, xs, gs, NT);
  __syncthreads();
  float v = chunk_dot<BITS, KIND, G>(it, xs + c * kXBlock, gs + c * (128 / G), kc, q4lut);
  v = (LPR == 32) ? half_wave_sum(v) : wave_sum(v);
  if ((lane & (LPR - 1)) == LPR - 1 && row < n) y[row] = (uint16_t)float_to_half_bits(v);
}

// Codebook 3-bit, group 128, k = 128*32, for matrices with few rows: two lanes
// per chunk, one row per wave, so that each wave carries half the decode work
// and a SIMD interleaves twice as many waves while the codes arrive. Lane l
// takes chunk l % 32; lanes 0-31 decode the fields in bits 0-2 (codes 0-47) and
// the spare codes of dwords 0-3, lanes 32-63 the fields in bits 3-5 (codes
// 48-95) and the spare codes of dwords 4-7. Both run the same instructions: the
// second half loads slice 1 into the registers the first half fills with slice
// 0 and vice versa, and the field shift, spare bit and x offsets are per lane.
template <int WPB>
__global__ __launch_bounds__(64 * WPB) void gemv_cb3_half_kernel(const char* __restrict__ packed,
                                                                 const uint16_t* __restrict__ x,
                                                                 uint16_t* __restrict__ y, int n) {
  constexpr int C = 32, NT = 64 * WPB, XP = (C * 16 + NT - 1) / NT;
  __shared__ __align__(16) char xs[C * kXBlock];
  float2* no_gs = nullptr;  // codebook groups need no sums over x
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int c = lane & 31, h = lane >> 5;
  const int row = blockIdx.x * WPB + wave;
  const size_t meta_off = (size_t)n * C * 128 * 3 / 8;

  u32x4 xr[XP];
  load_x<XP>(x, 0, C, xr, NT);
  const int r = min(row, n - 1);
  const u32x4* code = reinterpret_cast<const u32x4*>(packed) + ((size_t)r * 3 * C + c);
  const u32x4 s0 = __builtin_nontemporal_load(code + (size_t)h * C);        // slice h
  const u32x4 s1 = __builtin_nontemporal_load(code + (size_t)(1 - h) * C);  // slice 1 - h
  const u32x4 s2 = __builtin_nontemporal_load(code + (size_t)2 * C);
  const u32x4 tb = __builtin_nontemporal_load(
      reinterpret_cast<const u32x4*>(packed + meta_off + ((size_t)r * C + c) * 16));
  store_x<3, QX_CODEBOOK, 128, XP, C * 16 % NT == 0>(xr, C, xs, no_gs, NT);
  __syncthreads();

  const uint32_t m[4] = {tb.x, tb.y, tb.z, tb.w};
  const LutGroup<3> t = lut_group<3>(m);
  const uint32_t sh = 3u * h;                     // field: bits 0-2 or 3-5 of each byte
  const uint32_t ssh = 4u + h;                    // spare bit 2: bit 6 or 7 of H
  const char* xc = xs + c * kXBlock;
  // x blocks (4 codes, 8 bytes) of register group R0 / R1 / R2 and of the spare codes
  const int xo0 = h ? 8 * 16 : 0, xo1 = h ? 8 * 12 : 8 * 4, xo2 = h ? 8 * 20 : 8 * 8;
  const int xos = h ? 8 * 28 : 8 * 24;
  const uint32_t R[12] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w, s2.x, s2.y, s2.z, s2.w};
  float acc = 0.f;
#pragma unroll
  for (int i = 0; i < 12; ++i) {
    const int xo = (i < 4 ? xo0 : i < 8 ? xo1 : xo2) + 8 * (i & 3);
    uint32_t p02, p13;
    lut3_pairs(t, (R[i] >> sh) & 0x07070707u, p02, p13);
    const u32x2 xv = *reinterpret_cast<const u32x2*>(xc + xo);
    acc = dot2(p02, xv.x, acc);
    acc = dot2(p13, xv.y, acc);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {  // spare codes of the dword in R0[i]; bit 2 in R2[i]
    const uint32_t S = ((R[i] >> 6) & 0x03030303u) | ((R[8 + i] >> ssh) & 0x04040404u);
    uint32_t p02, p13;
    lut3_pairs(t, S, p02, p13);
    const u32x2 xv = *reinterpret_cast<const u32x2*>(xc + xos + 8 * i);
    acc = dot2(p02, xv.x, acc);
    acc = dot2(p13, xv.y, acc);
  }
  const float v = wave_sum(acc);
  if (lane == 63 && row < n) y[row] = (uint16_t)float_to_half_bits(v);
}

// Byte offset of the group sums after C chunks of x and n floats of partials.
__host__ __device__ constexpr int row_lds_gsum_offset(int C, int nfloats) {
  return C * kXBlock + (nfloats * 4 + 7) / 8 * 8;
}

// K up to 88 chunks, any count: one (row, chunk) item per lane. The block has
// 64*ceil(R*C/64) threads, with R picked so that few lanes idle (for C = 86,
// R = 8 rows fill 688 of 704 lanes); per-item partials go through LDS and one
// wave per row adds them in a fixed order.
template <int BITS, int KIND, int G, int XP>
__global__ __launch_bounds__(1024) void gemv_row_kernel(const char* __restrict__ packed,
                                                        const uint16_t* __restrict__ x,
                                                        uint16_t* __restrict__ y, int n, int k,
                                                        int R) {
  extern __shared__ __align__(16) char smem[];
  const int C = k >> 7, G_row = k / G, nthreads = blockDim.x;
  const size_t meta_off = (size_t)n * k * BITS / 8;
  const int row0 = blockIdx.x * R;
  const int rows = min(R, n - row0);
  char* xs = smem;                                             // C * kXBlock bytes
  float* part = reinterpret_cast<float*>(smem + C * kXBlock);  // R * C floats
  float2* gs = reinterpret_cast<float2*>(smem + row_lds_gsum_offset(C, R * C));  // C * 128/G
  __shared__ __align__(16) uint32_t q4lut[KIND == QX_Q4X ? 32 : 1];
  const DecodeConsts kc = decode_consts();

  u32x4 xr[XP];
  const u32x4* src = reinterpret_cast<const u32x4*>(x);
#pragma unroll
  for (int i = 0; i < XP; ++i) xr[i] = src[min((int)threadIdx.x + i * nthreads, C * 16 - 1)];
  const int t = threadIdx.x, r = t / C, c = t - r * C;
  const bool valid = r < rows;
  Item<BITS, KIND, G> it;
  load_item<BITS, KIND, G>(it, packed, meta_off, row0 + min(r, rows - 1), c, C, G_row);
  if constexpr (KIND == QX_Q4X) stage_q4x_lut(packed, n, k, q4lut);
  store_x<BITS, KIND, G, XP>(xr, C, xs, gs, nthreads);
  __syncthreads();
  if (valid) part[t] = chunk_dot<BITS, KIND, G>(it, xs + c * kXBlock, gs + c * (128 / G), kc, q4lut);
  __syncthreads();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  for (int rr = wave; rr < rows; rr += nthreads >> 6) {
    float v = 0.f;
    for (int cc = lane; cc < C; cc += 64) v += part[rr * C + cc];
    v = wave_sum(v);
    if (lane == 63) y[row0 + rr] = (uint16_t)float_to_half_bits(v);
  }
}

// Any K: items are the R x CT (row, chunk) pairs of a K tile of CT <= 88 chunks,
// dealt round-robin to the 256 lanes (ITEMS per lane); per-item partial sums go
// through LDS and one wave per row adds them in a fixed order. K longer than 88
// chunks is walked in tiles of 64 chunks.
template <int BITS, int KIND, int G, int ITEMS, int XP>
__global__ __launch_bounds__(kThreads) void gemv_tile_kernel(const char* __restrict__ packed,
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
  float2* gs = reinterpret_cast<float2*>(smem + row_lds_gsum_offset(CT, R * CT));  // CT * 128/G
  __shared__ __align__(16) uint32_t q4lut[KIND == QX_Q4X ? 32 : 1];
  const DecodeConsts kc = decode_consts();
  if constexpr (KIND == QX_Q4X) stage_q4x_lut(packed, n, k, q4lut);  // before the first barrier

  float acc[ITEMS];
#pragma unroll
  for (int j = 0; j < ITEMS; ++j) acc[j] = 0.f;

  for (int c0 = 0; c0 < C; c0 += CT) {
    const int ct = min(CT, C - c0);
    u32x4 xr[XP];
    load_x<XP>(x, c0, ct, xr);
    Item<BITS, KIND, G> it[ITEMS];
    bool valid[ITEMS];
    int cl[ITEMS];
#pragma unroll
    for (int j = 0; j < ITEMS; ++j) {
      const int i = threadIdx.x + j * kThreads;
      const int r = i / CT;
      cl[j] = i - r * CT;
      valid[j] = r < rows && cl[j] < ct;
      // invalid slots load an in-bounds chunk and are never consumed
      load_item<BITS, KIND, G>(it[j], packed, meta_off, row0 + min(r, rows - 1),
                               c0 + min(cl[j], ct - 1), C, G_row);
    }
    if (c0 > 0) __syncthreads();  // previous tile's x no longer read
    store_x<BITS, KIND, G, XP>(xr, ct, xs, gs);
    __syncthreads();
#pragma unroll
    for (int j = 0; j < ITEMS; ++j)
      if (valid[j]) acc[j] += chunk_dot<BITS, KIND, G>(it[j], xs + cl[j] * kXBlock, gs + cl[j] * (128 / G), kc, q4lut);
  }

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
    if (lane == 63) y[row0 + r] = (uint16_t)float_to_half_bits(v);
  }
}

#ifndef QX_GEMV_TILE_ROWS
#define QX_GEMV_TILE_ROWS 8
#endif
#ifndef QX_GEMV_HALF_MAX_N
#define QX_GEMV_HALF_MAX_N 8192  // rows up to which codebook-3 g128 rows of 32 chunks take two lanes per chunk
#endif
#ifndef QX_GEMV_WPB
#define QX_GEMV_WPB 4  // waves per block of the wave kernel
#endif

// Rows per block and block size of the row kernel for C chunks per row: among
// blocks of at least 256 threads (x is staged once per block), the R whose R*C
// items leave the fewest idle lanes in 64*ceil(R*C/64) threads; at most 8 rows
// when rows are long, so that large matrices still get many blocks.
static void gemv_row_shape(int C, int* R, int* threads) {
  const int r_max = C >= 32 ? std::min(8, 1024 / C) : std::min(256, 1024 / C);
  int best_r = 0;
  double best_u = -1.0;
  for (int pass = 0; pass < 2 && best_r == 0; ++pass) {
    for (int r = 1; r <= r_max; ++r) {
      const int t = 64 * ((r * C + 63) / 64);
      if (pass == 0 && t < 256) continue;
      const double u = (double)(r * C) / t;
      if (u > best_u + 1e-9) { best_u = u; best_r = r; }
    }
  }
  *R = best_r;
  *threads = 64 * ((best_r * C + 63) / 64);
}

static void gemv_tile_shape(int n, int k, int* R, int* items) {
  const int C = k / 128;
  const int CT = C <= kMaxTileChunks ? C : kLongTileChunks;
  int r = QX_GEMV_TILE_ROWS;
  while (r > 1 && (n + r - 1) / r < 512) r >>= 1;  // keep >= 512 blocks when n allows
  while (r > 1 && r * CT > 4 * kThreads) r >>= 1;
  *R = r;
  *items = (r * CT + kThreads - 1) / kThreads;
}

template <int BITS, int KIND, int G>
static void launch_gemv_tile(const qx_desc* d, const char* p, const uint16_t* x, uint16_t* y,
                             hipStream_t s) {
  int R, items;
  gemv_tile_shape(d->n, d->k, &R, &items);
  const int C = d->k / 128;
  const int CT = C <= kMaxTileChunks ? C : kLongTileChunks;
  const size_t lds = (size_t)row_lds_gsum_offset(CT, R * CT) + (size_t)CT * (128 / G) * sizeof(float2);
  const dim3 grid((d->n + R - 1) / R), block(kThreads);
  const int xp = (CT * 16 + kThreads - 1) / kThreads;  // x pieces per thread: 1..6
#define QX_GEMV_LAUNCH(I, XP) \
  hipLaunchKernelGGL((gemv_tile_kernel<BITS, KIND, G, I, XP>), grid, block, lds, s, p, x, y, d->n, d->k, R)
  if (xp <= 2) {
    switch (items) {
      case 1: QX_GEMV_LAUNCH(1, 2); break;
      case 2: QX_GEMV_LAUNCH(2, 2); break;
      default: QX_GEMV_LAUNCH(4, 2); break;
    }
  } else if (xp <= 4) {
    switch (items) {
      case 1: QX_GEMV_LAUNCH(1, 4); break;
      case 2: QX_GEMV_LAUNCH(2, 4); break;
      default: QX_GEMV_LAUNCH(4, 4); break;
    }
  } else {
    switch (items) {
      case 1: QX_GEMV_LAUNCH(1, 6); break;
      case 2: QX_GEMV_LAUNCH(2, 6); break;
      case 3: QX_GEMV_LAUNCH(3, 6); break;
      default: QX_GEMV_LAUNCH(4, 6); break;
    }
  }
#undef QX_GEMV_LAUNCH
}

template <int BITS, int KIND, int G>
static int launch_gemv_t(const qx_desc* d, const void* packed, const uint16_t* x, uint16_t* y,
                         hipStream_t s) {
  const char* p = static_cast<const char*>(packed);
  const int C = d->k / 128;
  if (C == 32 || C == 64) {
    // one (row, chunk) item per lane: more resident waves measured faster than more
    // items per lane at every decoder shape
    constexpr int WPB = QX_GEMV_WPB;
    const int rpb = WPB * 64 / C;
    const unsigned blocks = (unsigned)((d->n + rpb - 1) / rpb);
    if (BITS == 3 && KIND == QX_CODEBOOK && G == 128 && C == 32 && d->n <= QX_GEMV_HALF_MAX_N)
      hipLaunchKernelGGL((gemv_cb3_half_kernel<8>), dim3((d->n + 7) / 8), dim3(512), 0, s, p, x, y, d->n);
    else if (C == 32)
      hipLaunchKernelGGL((gemv_wave_kernel<BITS, KIND, G, 32, WPB>), dim3(blocks), dim3(64 * WPB), 0, s, p, x, y, d->n);
    else
      hipLaunchKernelGGL((gemv_wave_kernel<BITS, KIND, G, 64, WPB>), dim3(blocks), dim3(64 * WPB), 0, s, p, x, y, d->n);
  } else if (C <= kMaxTileChunks) {
    int R, threads;
    gemv_row_shape(C, &R, &threads);
    const unsigned blocks = (unsigned)((d->n + R - 1) / R);
    const size_t lds = (size_t)row_lds_gsum_offset(C, R * C) + (size_t)C * (128 / G) * sizeof(float2);
    const int xp = (C * 16 + threads - 1) / threads;
#define QX_ROW_LAUNCH(XP) \
  hipLaunchKernelGGL((gemv_row_kernel<BITS, KIND, G, XP>), dim3(blocks), dim3(threads), lds, s, p, x, y, d->n, d->k, R)
    // blocks have >= 256 threads or C < 32, so xp <= ceil(88*16/256) = 6 never
    // exceeds 4 in practice (C = 33..43 give 3); larger values take the tile kernel
    if (xp <= 1) QX_ROW_LAUNCH(1);
    else if (xp <= 2) QX_ROW_LAUNCH(2);
    else if (xp <= 4) QX_ROW_LAUNCH(4);
    else launch_gemv_tile<BITS, KIND, G>(d, p, x, y, s);
#undef QX_ROW_LAUNCH
  } else {
    launch_gemv_tile<BITS, KIND, G>(d, p, x, y, s);
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
  QX_GEMV_CASE(4, 2, 64)
#undef QX_GEMV_CASE
  return QX_E_UNSUPPORTED;
}

}  // namespace qx
