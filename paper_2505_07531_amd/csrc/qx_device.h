// Device helpers shared by the libqx kernels: in-register decoding of the
// packed layout (declared in include/qx.h) into fp16 pairs.
//
// Codes are turned into fp16 without conversion instructions: a code q placed
// in the fraction bits of an fp16 whose exponent makes one fraction step
// worth 1 reads as M + q (M = 1024 for bits 0-2/0-3, 128 for bits 3-5, 16 for
// bits 6-8 of a half); subtracting the pair (M + z, M + z) with one packed
// fp16 add leaves the exact integers q - z. The GEMVs skip the bias: the code
// field alone, masked out of its dword, is a binary16 subnormal q * 2^(f - 24)
// (f its lowest fraction bit), which v_dot2 multiplies exactly. Codebook entries are fetched with
// v_perm_b32, which picks bytes out of an 8-byte register table: the low and
// the high bytes of the 2^b fp16 entries sit in separate tables, four codes
// are looked up per instruction, and a final byte interleave rebuilds fp16
// pairs.
//
// Pair order. Every consumer reads activations in the order in which pairs
// come out of the decoders:
//   b = 4: code dword j (codes 8j..8j+7) yields (0,4) (2,6) (1,5) (3,7);
//   b = 3: each 4-code block (4t..4t+3) yields (0,2) (1,3).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/qx.h"

namespace qx {

typedef _Float16 h2_t __attribute__((ext_vector_type(2)));
typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef float f4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ h2_t as_h2(uint32_t u) { return __builtin_bit_cast(h2_t, u); }
__device__ __forceinline__ uint32_t as_u32(h2_t v) { return __builtin_bit_cast(uint32_t, v); }

// {hi, lo} byte select: selector byte e in 0..3 picks lo byte e, 4..7 picks hi byte e-4,
// 12 gives 0x00.
__device__ __forceinline__ uint32_t perm(uint32_t hi, uint32_t lo, uint32_t sel) {
  return __builtin_amdgcn_perm(hi, lo, sel);
}

// acc + a.x*b.x + a.y*b.y with exact fp16 products and an fp32 sum (v_dot2_f32_f16).
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float acc) {
  return __builtin_amdgcn_fdot2(as_h2(a), as_h2(b), acc, false);
}

// a.x*b.x + a.y*b.y from 0: the three-address v_dot2_f32_f16 with an inline 0
// (the compiler otherwise zeroes a register for the accumulating two-address form).
__device__ __forceinline__ float dot2_0(uint32_t a, uint32_t b) {
  float r;
  asm("v_dot2_f32_f16 %0, %1, %2, 0" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

__device__ __forceinline__ uint32_t hadd2(uint32_t a, uint32_t b) {
  return as_u32(as_h2(a) + as_h2(b));
}
__device__ __forceinline__ uint32_t hmul2(uint32_t a, uint32_t b) {
  return as_u32(as_h2(a) * as_h2(b));
}

__device__ __forceinline__ float half_bits_to_float(uint32_t h) {
  return (float)__builtin_bit_cast(_Float16, (uint16_t)h);
}
__device__ __forceinline__ uint32_t float_to_half_bits(float f) {  // round to nearest even
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)f);
}
__device__ __forceinline__ uint32_t splat_half(float f) {
  const uint32_t h = float_to_half_bits(f);
  return h | (h << 16);
}

// Bias magic numbers: binary16 1024 (fraction step 1), 128 (step 1/8), 16 (step 1/64).
constexpr uint32_t kMagic1024 = 0x64006400u;
constexpr uint32_t kMagic128 = 0x58005800u;
constexpr uint32_t kMagic16 = 0x4C004C00u;

// Register byte tables of one codebook group: lo[t] / hi[t] hold the low / high
// bytes of entries 4t..4t+3 (t < 2^b / 4).
template <int BITS>
struct LutGroup {
  uint32_t lo[(1 << BITS) / 4], hi[(1 << BITS) / 4];
};
template <int BITS>
__device__ __forceinline__ LutGroup<BITS> lut_group(const uint32_t* w) {  // 2^(b-1) dwords
  LutGroup<BITS> t;
#pragma unroll
  for (int i = 0; i < (1 << BITS) / 4; ++i) {
    t.lo[i] = perm(w[2 * i + 1], w[2 * i], 0x06040200u);
    t.hi[i] = perm(w[2 * i + 1], w[2 * i], 0x07050301u);
  }
  return t;
}

// Constants kept in VGPRs so that "(D & mask) | bias" is one v_and_or_b32 (VOP3 on
// this target encodes no 32-bit literal and reads at most one scalar register).
__device__ __forceinline__ uint32_t in_vgpr(uint32_t c) {
  asm volatile("" : "+v"(c));
  return c;
}
struct DecodeConsts {
  uint32_t m0007, m0038, m00c0, m0100, m000f, m00f0, mag1024, mag128, mag64, mag16;
};
__device__ __forceinline__ DecodeConsts decode_consts() {
  DecodeConsts k;
  k.m0007 = in_vgpr(0x00070007u);
  k.m0038 = in_vgpr(0x00380038u);
  k.m00c0 = in_vgpr(0x00C000C0u);
  k.m0100 = in_vgpr(0x01000100u);
  k.m000f = in_vgpr(0x000F000Fu);
  k.m00f0 = in_vgpr(0x00F000F0u);
  k.mag1024 = in_vgpr(0x64006400u);
  k.mag128 = in_vgpr(0x58005800u);
  k.mag64 = in_vgpr(0x54005400u);
  k.mag16 = in_vgpr(0x4C004C00u);
  return k;
}

// ----------------------------------------------------------------- b = 3
// "M + q" pairs of the A and B fields of code dword D (bytes b0..b3):
//   a0 = (A0, A2), a1 = (A1, A3) with M = 1024; b0 = (B0, B2), b1 = (B1, B3) with M = 128.
struct U3Pairs {
  uint32_t a0, a1, b0, b1;
};
__device__ __forceinline__ U3Pairs u3_fields(uint32_t D, const DecodeConsts& k) {
  const uint32_t Ds = D >> 8;
  U3Pairs p;
  p.a0 = (D & k.m0007) | k.mag1024;
  p.a1 = (Ds & k.m0007) | k.mag1024;
  p.b0 = (D & k.m0038) | k.mag128;
  p.b1 = (Ds & k.m0038) | k.mag128;
  return p;
}
// The same fields as binary16 subnormals (no bias): a = (A0, A2), (A1, A3) read as
// q * 2^-24, b = (B0, B2), (B1, B3) as q * 2^-21.
__device__ __forceinline__ U3Pairs u3_raw(uint32_t D, const DecodeConsts& k) {
  const uint32_t Ds = D >> 8;
  U3Pairs p;
  p.a0 = D & k.m0007;
  p.a1 = Ds & k.m0007;
  p.b0 = D & k.m0038;
  p.b1 = Ds & k.m0038;
  return p;
}
// Spare codes of code dword i (< 8): bits 0-1 in the spare fields of D, bit 2 in
// H = dword 8 + (i & 3), bit 6 (i < 4) or bit 7 (i >= 4) of the matching byte.
// Returns pairs for spare codes (0, 2) and (1, 3) of the dword in bits 6-8 of each
// half, i.e. binary16 subnormals q * 2^-18.
template <int I>
__device__ __forceinline__ void u3_spare_raw(uint32_t D, uint32_t H, const DecodeConsts& k,
                                             uint32_t& s0, uint32_t& s1) {
  constexpr int kUp = (I < 4) ? 2 : 1;    // bit 6 or 7 of bytes 0/2 -> bit 8 of each half
  constexpr int kDown = (I < 4) ? 6 : 7;  // bit 6 or 7 of bytes 1/3 -> bit 8 of each half
  s0 = (D & k.m00c0) | ((H << kUp) & k.m0100);
  s1 = ((D >> 8) & k.m00c0) | ((H >> kDown) & k.m0100);
}
// Byte selectors (4 codes, natural order) of the three fields of code dword D.
__device__ __forceinline__ uint32_t u3_sel_a(uint32_t D) { return D & 0x07070707u; }
__device__ __forceinline__ uint32_t u3_sel_b(uint32_t D) { return (D >> 3) & 0x07070707u; }
template <int I>
__device__ __forceinline__ uint32_t u3_sel_spare(uint32_t D, uint32_t H) {
  constexpr int kSh = (I < 4) ? 4 : 5;  // bit 6 or 7 of each byte -> bit 2
  return ((D >> 6) & 0x03030303u) | ((H >> kSh) & 0x04040404u);
}

// Codebook lookup of four 3-bit selectors: fp16 pairs (c0, c2) and (c1, c3).
__device__ __forceinline__ void lut3_pairs(const LutGroup<3>& t, uint32_t S, uint32_t& p02,
                                           uint32_t& p13) {
  const uint32_t lo = perm(t.lo[1], t.lo[0], S);
  const uint32_t hi = perm(t.hi[1], t.hi[0], S);
  p02 = perm(hi, lo, 0x06020400u);
  p13 = perm(hi, lo, 0x07030501u);
}
// Same, natural pairs (c0, c1) and (c2, c3).
__device__ __forceinline__ void lut3_pairs_nat(const LutGroup<3>& t, uint32_t S, uint32_t& p01,
                                               uint32_t& p23) {
  const uint32_t lo = perm(t.lo[1], t.lo[0], S);
  const uint32_t hi = perm(t.hi[1], t.hi[0], S);
  p01 = perm(hi, lo, 0x05010400u);
  p23 = perm(hi, lo, 0x07030602u);
}

// ----------------------------------------------------------------- b = 4
// Codebook lookup of four 4-bit selectors (bytes 0..15): entries 0-7 from tables
// [0..1], 8-15 from [2..3], merged with a byte mask built by v_perm.
__device__ __forceinline__ void lut4_bytes(const LutGroup<4>& t, uint32_t S, uint32_t& lo,
                                           uint32_t& hi) {
  const uint32_t sel = S & 0x07070707u;
  // selector byte 4 (bit 3 clear) -> 0xFF, 12 (bit 3 set) -> 0x00
  const uint32_t mask = perm(0x000000FFu, 0u, (S & 0x08080808u) | 0x04040404u);
  const uint32_t la = perm(t.lo[1], t.lo[0], sel), lb = perm(t.lo[3], t.lo[2], sel);
  const uint32_t ha = perm(t.hi[1], t.hi[0], sel), hb = perm(t.hi[3], t.hi[2], sel);
  lo = (la & mask) | (lb & ~mask);
  hi = (ha & mask) | (hb & ~mask);
}

// fp16 W' pairs (c0,c1), (c2,c3) of one 4-code block (natural-order selector Q).
// Uniform: the exact integers q - z (biased-exponent trick) times the scale pair
// in one packed fp16 multiply, i.e. fp16_RNE(s*(q-z)) with IEEE signed zeros.
// Codebook: the table entries, copied bytewise.
template <int BITS, int KIND>
__device__ __forceinline__ void block_weights(uint32_t Q, const uint32_t* meta, uint32_t& w01,
                                              uint32_t& w23) {
  if constexpr (KIND == QX_UNIFORM) {
    const uint32_t word = meta[0];
    const uint32_t sp = (word & 0xFFFFu) * 0x00010001u;  // (s, s)
    const uint32_t zc = splat_half(-(1024.0f + half_bits_to_float(word >> 16)));
    w01 = hmul2(hadd2(perm(Q, Q, 0x0C010C00u) | kMagic1024, zc), sp);
    w23 = hmul2(hadd2(perm(Q, Q, 0x0C030C02u) | kMagic1024, zc), sp);
  } else {
    const LutGroup<BITS> t = lut_group<BITS>(meta);
    uint32_t lo, hi;
    if constexpr (BITS == 3) {
      lo = perm(t.lo[1], t.lo[0], Q);
      hi = perm(t.hi[1], t.hi[0], Q);
    } else {
      lut4_bytes(t, Q, lo, hi);
    }
    w01 = perm(hi, lo, 0x05010400u);
    w23 = perm(hi, lo, 0x07030602u);
  }
}

// Dequantization constants of the uniform groups of one (row, chunk): the scale
// pair (s, s) and -(M + z) pairs for the bias magic numbers M of each field.
template <int BITS, int G>
struct GroupConsts {
  uint32_t sp[128 / G], z1024[128 / G], zb[128 / G], z16[128 / G];  // zb: M = 128 (b=3), 64 (b=4)
};
template <int BITS, int G>
__device__ __forceinline__ GroupConsts<BITS, G> group_consts(const uint32_t* m) {
  GroupConsts<BITS, G> gc;
#pragma unroll
  for (int i = 0; i < 128 / G; ++i) {
    const uint32_t w = m[i];
    // z is an integer-valued fp16 in [0, 2^b - 1]; -(M + z) is exact in fp16 and its bits
    // are those of -M plus z fraction steps
    const uint32_t z = (uint32_t)(unsigned short)__builtin_bit_cast(_Float16, (uint16_t)(w >> 16));
    gc.sp[i] = perm(w, w, 0x01000100u);
    gc.z1024[i] = (0xE400u + z) * 0x00010001u;
    gc.zb[i] = BITS == 3 ? (0xD800u + 8u * z) * 0x00010001u : (0xD400u + 16u * z) * 0x00010001u;
    gc.z16[i] = (0xCC00u + 64u * z) * 0x00010001u;
  }
  return gc;
}

__device__ __forceinline__ uint32_t deq(uint32_t mq, uint32_t zc, uint32_t sp) {
  return hmul2(hadd2(mq, zc), sp);  // fp16(s * (q - z)), q - z exact
}

__device__ __forceinline__ h8_t frag(uint32_t a, uint32_t b, uint32_t c, uint32_t d) {
  return __builtin_bit_cast(h8_t, u32x4{a, b, c, d});
}

// Cross-lane fp32 sums with DPP only (no LDS traffic). A DPP "row" is 16 lanes.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float dpp_plus(float v) {
  // lanes of rows outside ROW_MASK add 0 (the "old" operand)
  return v + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
                 0, __builtin_bit_cast(int, v), CTRL, ROW_MASK, 0xF, false));
}
// Every lane of each 16-lane row ends with that row's sum.
__device__ __forceinline__ float row16_sum(float v) {
  v = dpp_plus<0xB1, 0xF>(v);   // quad_perm [1,0,3,2]
  v = dpp_plus<0x4E, 0xF>(v);   // quad_perm [2,3,0,1]
  v = dpp_plus<0x141, 0xF>(v);  // row_half_mirror
  v = dpp_plus<0x140, 0xF>(v);  // row_mirror
  return v;
}
// Sum of lanes 0..31 in lane 31 and of lanes 32..63 in lane 63.
__device__ __forceinline__ float half_wave_sum(float v) {
  v = row16_sum(v);
  return dpp_plus<0x142, 0xA>(v);  // row_bcast:15 into rows 1 and 3
}
// Sum of all 64 lanes in lane 63.
__device__ __forceinline__ float wave_sum(float v) {
  v = half_wave_sum(v);
  return dpp_plus<0x143, 0xC>(v);  // row_bcast:31 into rows 2 and 3
}

// Q4X: a matrix's 4 x 16 binary16 codebook (128 bytes at `codebook`) as the
// v_perm lookup tables of lut4_bytes (per sub-codebook 4 dwords of low bytes, then
// 4 of high bytes), written to LDS by the first 16 threads of the block.
__device__ __forceinline__ void stage_q4x_tables(const char* __restrict__ codebook, uint32_t* lut) {
  if (threadIdx.x < 16) {
    const int t = threadIdx.x >> 2, i = threadIdx.x & 3;
    const uint32_t* cb = reinterpret_cast<const uint32_t*>(codebook) + 8 * t;
    const uint32_t w0 = cb[2 * i], w1 = cb[2 * i + 1];
    lut[8 * t + i] = perm(w1, w0, 0x06040200u);
    lut[8 * t + 4 + i] = perm(w1, w0, 0x07050301u);
  }
}

}  // namespace qx
