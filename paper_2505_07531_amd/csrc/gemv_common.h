// Device helpers shared by the GEMV kernels (gemv.hip, gemv_multi.hip): staging
// of activation vectors in LDS, the packed bytes of one (row, 128-code chunk)
// item, and the chunk dot products of every format.
#pragma once

#include "qx_device.h"
#include "qx_internal.h"

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

// Sum of one 16-byte piece of x (8 values) for the folded zero point of uniform
// groups (one dot2 chain with the pair (1, 1); products of binary16 values are
// exact in fp32).
__device__ __forceinline__ float piece_sum(const u32x4& v) {
  const uint32_t one = in_vgpr(0x3C003C00u);  // (1, 1)
  return dot2(v.w, one, dot2(v.z, one, dot2(v.y, one, dot2_0(v.x, one))));
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
// groups, also store sum x per group of the tile in gs; the pieces of a group
// sit in consecutive lanes.
template <int BITS, int KIND, int G, int XP, bool EXACT = false>  // EXACT: every piece is in range
__device__ __forceinline__ void store_x(const u32x4 (&xr)[XP], int ct, char* xs, float* gs,
                                        int stride = kThreads) {
#pragma unroll
  for (int i = 0; i < XP; ++i) {
    const int p = threadIdx.x + i * stride;
    const u32x4 v = xr[i];
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
    if (EXACT || p < ct * 16) *reinterpret_cast<u32x4*>(xs + (p >> 4) * kXBlock + (p & 15) * 16) = o;
    if constexpr (KIND == QX_UNIFORM) {
      constexpr int PPG = G / 8;  // pieces per group
      const float sx = lane_group_sum<PPG>(piece_sum(v));
      if ((p & (PPG - 1)) == 0 && (EXACT || p < ct * 16)) gs[p / PPG] = sx;
    }
  }
}

// Raw bytes of one item: codes (4*BITS dwords) and its group tables.
template <bool NT, typename T>
__device__ __forceinline__ T ld_nt(const T* p) {
  if constexpr (NT) return __builtin_nontemporal_load(p);
  else return *p;
}

template <int BITS, int KIND, int G>
struct Item {
  static constexpr int kGroups = 128 / G;
  // Q4X: m[0] = the two groups' binary16 scales, m[1] = their selectors (bits 0-1, 2-3)
  static constexpr int kMetaDw = KIND == QX_Q4X ? 2 : KIND == 0 ? kGroups : kGroups * (1 << BITS) / 2;
  uint32_t d[4 * BITS];
  uint32_t m[kMetaDw];
};

// Codes and tables of one (row, chunk) item. NT: non-temporal loads (streamed once);
// the small-batch kernel reads each 128-byte line as two halves from two items and
// keeps them cached when a lane has more than one item.
template <int BITS, int KIND, int G, bool NT = true>
__device__ __forceinline__ void load_item(Item<BITS, KIND, G>& it, const char* __restrict__ packed,
                                          size_t meta_off, int row, int c, int C, int G_row) {
  const u32x4* code = reinterpret_cast<const u32x4*>(packed) + ((size_t)row * BITS * C + c);
#pragma unroll
  for (int s = 0; s < BITS; ++s) {
    const u32x4 v = ld_nt<NT>(code + (size_t)s * C);
    it.d[4 * s + 0] = v.x; it.d[4 * s + 1] = v.y; it.d[4 * s + 2] = v.z; it.d[4 * s + 3] = v.w;
  }
  if constexpr (KIND == QX_Q4X) {  // groups 2c and 2c + 1 of the row
    const size_t sel_off = meta_off + meta_off / 16;  // after n*G binary16 scales (n*k/32 bytes)
    const int W = (G_row + 15) / 16;
    it.m[0] = ld_nt<NT>(
        reinterpret_cast<const uint32_t*>(packed + meta_off + ((size_t)row * G_row + 2 * c) * 2));
    const uint32_t sw = ld_nt<NT>(
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
      const u32x4 v = ld_nt<NT>(reinterpret_cast<const u32x4*>(mp) + i);
      it.m[4 * i + 0] = v.x; it.m[4 * i + 1] = v.y; it.m[4 * i + 2] = v.z; it.m[4 * i + 3] = v.w;
    }
  } else if constexpr (kDw == 2) {
    const u32x2 v = ld_nt<NT>(reinterpret_cast<const u32x2*>(mp));
    it.m[0] = v.x; it.m[1] = v.y;
  } else {
    it.m[0] = ld_nt<NT>(mp);
  }
}

// Bit-2 source dword of spare codes of code dword I, and the two spare helpers
// dispatched on the compile-time index.
template <int I, int BITS, int KIND, int G>
__device__ __forceinline__ void spare_raw(const Item<BITS, KIND, G>& it, const DecodeConsts& k,
                                          uint32_t& s0, uint32_t& s1) {
  u3_spare_raw<I>(it.d[I], it.d[8 + (I & 3)], k, s0, s1);
}
template <int I, int BITS, int KIND, int G>
__device__ __forceinline__ uint32_t spare_sel(const Item<BITS, KIND, G>& it) {
  return u3_sel_spare<I>(it.d[I], it.d[8 + (I & 3)]);
}

// Uniform codes enter the products unbiased, as binary16 subnormals: a code q in
// fraction bits [f, f + b) of a half reads as q * 2^(f - 24) (the GEMV masks its
// field out of the packed dword and nothing else). Products with x and their fp32
// sums are exact up to the rounding of the sums, there is no bias whose sum over x
// has to cancel, and a group whose codes are all 0 sums to exactly 0. Field kinds
// per half: b = 4: bits 0-3 and 4-7; b = 3: bits 0-2, 3-5, 6-8 (spare codes).
template <int BITS>
struct RawFields {
  static constexpr int kN = BITS == 4 ? 2 : 3;
};
// sum q x of one group from its per-field-kind accumulators f[0..kN)
template <int BITS>
__device__ __forceinline__ float raw_group_sum(const float* f) {
  if constexpr (BITS == 4) return fmaf(f[1], 0x1p20f, f[0] * 0x1p24f);
  else return fmaf(f[2], 0x1p18f, fmaf(f[1], 0x1p21f, f[0] * 0x1p24f));
}

// Scale and zero point of a uniform group word: s * (sum q x - z sum x) =
// s * sum (q - z) x over the group; the error of both sums scales with s.
__device__ __forceinline__ float fold_group(uint32_t word, float qx, float sx) {
  const float s = half_bits_to_float(word & 0xFFFFu), z = half_bits_to_float(word >> 16);
  return s * fmaf(-z, sx, qx);
}

// Partial dot product of one chunk with its x block (LDS, pair order). Uniform
// codes enter the products as subnormal integers (no subtraction per pair); gs
// holds the chunk's sum x per group and fold_group takes the zero point out.
template <int BITS, int KIND, int G>
__device__ __forceinline__ float chunk_dot(const Item<BITS, KIND, G>& it, const char* xb,
                                           const float* gs, const DecodeConsts& k,
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
      float f[2] = {0.f, 0.f};  // bits 0-3, bits 4-7
#pragma unroll
      for (int j = g * G / 8; j < (g + 1) * G / 8; ++j) {
        const u32x4 x = xv[j];
        const uint32_t D = it.d[j], Ds = D >> 8;
        f[0] = dot2(D & k.m000f, x.x, f[0]);   // (0, 4)
        f[1] = dot2(D & k.m00f0, x.y, f[1]);   // (1, 5)
        f[0] = dot2(Ds & k.m000f, x.z, f[0]);  // (2, 6)
        f[1] = dot2(Ds & k.m00f0, x.w, f[1]);  // (3, 7)
      }
      part += fold_group(it.m[g], raw_group_sum<4>(f), gs[g]);
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
    // 4-code block t (codes 4t..4t+3) feeds x dwords 2t (pair (0,2)) and 2t+1 (pair
    // (1,3)); blocks 0-11 are the bits 0-2 fields of code dwords 0-11, 12-23 their
    // bits 3-5 fields, 24-31 the spare codes. One accumulator per (group, field kind).
    float f[NG][3];
#pragma unroll
    for (int g = 0; g < NG; ++g) f[g][0] = f[g][1] = f[g][2] = 0.f;
#pragma unroll
    for (int i = 0; i < 12; i += 2) {
      const u32x4 xa = xv[i / 2], xb4 = xv[6 + i / 2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const U3Pairs p = u3_raw(it.d[i + h], k);
        const int ga = (4 * (i + h)) / G, gb = (48 + 4 * (i + h)) / G;
        f[ga][0] = dot2(p.a0, h ? xa.z : xa.x, f[ga][0]);
        f[ga][0] = dot2(p.a1, h ? xa.w : xa.y, f[ga][0]);
        f[gb][1] = dot2(p.b0, h ? xb4.z : xb4.x, f[gb][1]);
        f[gb][1] = dot2(p.b1, h ? xb4.w : xb4.y, f[gb][1]);
      }
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      uint32_t s0, s1;
      switch (i) {  // the bit-2 position depends on the dword index at compile time
        case 0: spare_raw<0>(it, k, s0, s1); break;
        case 1: spare_raw<1>(it, k, s0, s1); break;
        case 2: spare_raw<2>(it, k, s0, s1); break;
        case 3: spare_raw<3>(it, k, s0, s1); break;
        case 4: spare_raw<4>(it, k, s0, s1); break;
        case 5: spare_raw<5>(it, k, s0, s1); break;
        case 6: spare_raw<6>(it, k, s0, s1); break;
        default: spare_raw<7>(it, k, s0, s1); break;
      }
      const int gg = (96 + 4 * i) / G;
      const u32x4 xs4 = xv[12 + i / 2];
      f[gg][2] = dot2(s0, (i & 1) ? xs4.z : xs4.x, f[gg][2]);
      f[gg][2] = dot2(s1, (i & 1) ? xs4.w : xs4.y, f[gg][2]);
    }
    float part = 0.f;
#pragma unroll
    for (int g = 0; g < NG; ++g) part += fold_group(it.m[g], raw_group_sum<3>(f[g]), gs[g]);
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

// Q4X: the matrix's codebook tables in LDS (see stage_q4x_tables).
__device__ __forceinline__ void stage_q4x_lut(const char* __restrict__ packed, int n, int k,
                                              uint32_t* lut) {
  stage_q4x_tables(packed + q4x_offsets(n, k).codebook, lut);
}

// Rows per block R and block size of the row kernels (one (row, chunk) item per
// lane, x staged once per block) for n rows of C chunks: among blocks of at least
// 256 threads, the R whose R*C items leave the fewest idle lanes in 64*ceil(R*C/64)
// threads; at most 8 rows when rows are long. Short rows (< 32 chunks) take at most
// n / QX_ROW_MIN_BLOCKS rows, so that the grid has blocks for every compute unit
// where n allows (4096 rows of 4 chunks: 64 blocks of 64 rows 5.3 us, 512 blocks of 8
// rows 3.9 us; 4096 rows of 11 chunks 4.9 vs 3.6 us), but at least 4 above 16
// chunks, and x stays within 4 pieces per thread; heavy items (codebook-4 g32,
// measured slower) keep the rule without that cap.
#ifndef QX_ROW_MIN_BLOCKS
#define QX_ROW_MIN_BLOCKS 512
#endif
inline void gemv_row_shape(int n, int C, bool heavy_items, int* R, int* threads) {
  int r_max = C >= 32 ? (8 < 1024 / C ? 8 : 1024 / C) : (256 < 1024 / C ? 256 : 1024 / C);
  if (QX_ROW_MIN_BLOCKS > 0 && !heavy_items && C < 32) {
    const int floor_r = (C > 16 ? 4 : 1) < r_max ? (C > 16 ? 4 : 1) : r_max;
    const int cap = r_max < n / QX_ROW_MIN_BLOCKS ? r_max : n / QX_ROW_MIN_BLOCKS;
    r_max = floor_r > cap ? floor_r : cap;
  }
  int best_r = 0;
  double best_u = -1.0;
  for (int pass = 0; pass < 2 && best_r == 0; ++pass) {
    for (int r = 1; r <= r_max; ++r) {
      const int t = 64 * ((r * C + 63) / 64);
      if ((pass == 0 && t < 256) || (C < 32 && t < 4 * C)) continue;  // short rows: x in <= 4 pieces per thread
      const double u = (double)(r * C) / t;
      if (u > best_u + 1e-9) { best_u = u; best_r = r; }
    }
  }
  *R = best_r;
  *threads = 64 * ((best_r * C + 63) / 64);
}

// Byte offset of the group sums after C chunks of x and n floats of partials.
__host__ __device__ constexpr int row_lds_gsum_offset(int C, int nfloats) {
  return C * kXBlock + (nfloats * 4 + 7) / 8 * 8;
}

}  // namespace qx
