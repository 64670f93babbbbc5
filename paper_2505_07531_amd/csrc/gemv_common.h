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

// Sums over one 16-byte piece of x (8 values at chunk position 8*pc) for the
// folded zero point of uniform groups: sum x, and sum M x with M the bias that
// the decoder adds to the code at each position (b = 4: 1024 in bits 0-3, 64 in
// bits 4-7 of a half; b = 3: 1024 for codes 0-47, 128 for 48-95, 16 above).
// sum M x is formed exactly as chunk_dot forms the piece's sum of (M + q) x: one
// dot2 chain over the decoder-order pairs o.x .. o.w, from 0, with the pair
// (M, M) that the decoder yields for q = 0. So for a group whose codes are all
// zero the two sums are the same bits and the group contributes exactly 0
// (e.g. an all-zero group, which the quantizer stores with s = 1).
template <int BITS>
__device__ __forceinline__ void piece_sums(const u32x4& v, const u32x4& o, int pc, float& sx,
                                           float& mx) {
  const uint32_t one = 0x3C003C00u;  // (1, 1)
  if (BITS == 4) {
    sx = dot2(v.w, one, dot2(v.z, one, dot2(v.y, one, dot2_0(v.x, one))));
    const uint32_t m1024 = in_vgpr(kMagic1024), m64 = in_vgpr(0x54005400u);
    mx = dot2(m64, o.w, dot2(m1024, o.z, dot2(m64, o.y, dot2_0(m1024, o.x))));
  } else {
    // one M for the whole piece, a power of two: the chain of (M, M) pairs is M times
    // the chain of (1, 1) pairs bit for bit (sums of binary16 values are never fp32
    // subnormal, and M x cannot overflow)
    const uint32_t o1 = in_vgpr(one);
    sx = dot2(o1, o.w, dot2(o1, o.z, dot2(o1, o.y, dot2_0(o1, o.x))));
    mx = (pc < 6 ? 1024.f : pc < 12 ? 128.f : 16.f) * sx;
  }
}

// Sum of the N per-piece partial sums of one group in the balanced pairwise order
// of lane_group_sum (xor 1, xor 2, half-row mirror, row mirror; fp32 addition is
// commutative), the order in which the staged sum M x of the group was added.
template <int N>
__device__ __forceinline__ float piece_tree(const float* a) {
  if constexpr (N == 1) return a[0];
  else return piece_tree<N / 2>(a) + piece_tree<N / 2>(a + N / 2);
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
      float sx, mx;
      piece_sums<BITS>(v, o, p & 15, sx, mx);
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
// with acc = sum (M + q) x over the group, is s * sum (q - z) x. acc and sum M x
// are rounded in the same order (piece_sums, piece_tree): the difference is
// exactly 0 when every code of the group is 0, and otherwise carries the rounding
// of sums of (M + q) x, which s scales with the group's levels.
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
    // one dot2 chain per 8-code piece, the pieces of a group added in the order of the
    // staged sum M x (piece_sums, piece_tree)
    float a[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const u32x4 x = xv[j];
      const uint32_t D = it.d[j], Ds = D >> 8;
      float acc = dot2_0((D & k.m000f) | k.mag1024, x.x);  // (0, 4)
      acc = dot2((D & k.m00f0) | k.mag64, x.y, acc);          // (1, 5)
      acc = dot2((Ds & k.m000f) | k.mag1024, x.z, acc);       // (2, 6)
      a[j] = dot2((Ds & k.m00f0) | k.mag64, x.w, acc);        // (3, 7)
    }
    float part = 0.f;
#pragma unroll
    for (int g = 0; g < NG; ++g) part += fold_group(it.m[g], piece_tree<G / 8>(a + g * (G / 8)), gs[g]);
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
    // one dot2 chain per 8-code piece (x dwords 4p..4p+3): 4-code block t (codes
    // 4t..4t+3) feeds x dwords 2t (pair (0,2)) and 2t+1 (pair (1,3)), so piece p is
    // blocks 2p, 2p+1; pieces 0-5 are the bits 0-2 fields, 6-11 the bits 3-5 fields,
    // 12-15 the spare codes. The pieces of a group are added as in piece_tree.
    float a[16];
#pragma unroll
    for (int i = 0; i < 12; ++i) {
      const U3Pairs p = u3_fields(it.d[i], k);
      const int pa = i / 2, pb = 6 + i / 2;
      const u32x4 xa4 = xv[pa], xb4 = xv[pb];  // 16-byte pieces (one LDS read each per two i)
      const uint32_t xa0 = (i & 1) ? xa4.z : xa4.x, xa1 = (i & 1) ? xa4.w : xa4.y;
      const uint32_t xb0 = (i & 1) ? xb4.z : xb4.x, xb1 = (i & 1) ? xb4.w : xb4.y;
      a[pa] = (i & 1) ? dot2(p.a0, xa0, a[pa]) : dot2_0(p.a0, xa0);
      a[pa] = dot2(p.a1, xa1, a[pa]);
      a[pb] = (i & 1) ? dot2(p.b0, xb0, a[pb]) : dot2_0(p.b0, xb0);
      a[pb] = dot2(p.b1, xb1, a[pb]);
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
      const int ps = 12 + i / 2;
      const u32x4 xs4 = xv[ps];
      const uint32_t xs0 = (i & 1) ? xs4.z : xs4.x, xs1 = (i & 1) ? xs4.w : xs4.y;
      a[ps] = (i & 1) ? dot2(s0, xs0, a[ps]) : dot2_0(s0, xs0);
      a[ps] = dot2(s1, xs1, a[ps]);
    }
    float part = 0.f;
#pragma unroll
    for (int g = 0; g < NG; ++g) part += fold_group(it.m[g], piece_tree<G / 8>(a + g * (G / 8)), gs[g]);
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
