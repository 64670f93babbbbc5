// Batched quantized GEMM (prefill): Y[m][n] = sum_k X[m][k] W'[n][k].
//
// Once W' is dequantized the product is a dense contraction, so it runs on the
// matrix cores (v_mfma_f32_16x16x32_f16: fp16 operands, fp32 accumulators).
// The weights are the B operand and reach LDS only as packed codes: every lane
// dequantizes, in registers, exactly the eight weights that its B fragment
// holds, so the decode work of a weight is paid once per block of activation
// rows and no LDS bandwidth is spent on fp16 W'. The activations are staged in
// LDS once per block and chunk, in the order in which the decoders emit weight
// pairs.
//
// Fragments. A 128-code chunk of one weight row splits into 16 fragments of
// 8 codes; fragment f = 4t + g feeds k-step t (32 of the 128 k) of the MFMA
// from lane group g = lane / 16. The split is chosen so that, at a given
// k-step, all four lane groups decode the same kind of field with the same
// instructions (only the source dword differs, fetched by a per-lane address),
// and so that every field of one k-step lies in one quantization group whose
// index depends on t alone:
//   b = 4: fragment f is code dword f (codes 8f..8f+7), pairs (0,4) (1,5) (2,6) (3,7);
//   b = 3: f < 12 is code dword f: codes 4f..4f+3 from bits 0-2 of its bytes and
//          48+4f..48+4f+3 from bits 3-5, pairs (0,2) (1,3) of each; f >= 12 holds
//          the spare codes 96+8p..96+8p+7 (p = f - 12) of code dwords 2p, 2p+1.
// Uniform weights are dequantized exactly, fp16(s*(q-z)), by one packed add of
// exact integers and one packed multiply (the same arithmetic as qx_dequant);
// codebook weights are table entries fetched with v_perm_b32.
//
// Tiling. A block has W waves (4, or 8 / 16 for rows of more than 64 chunks): KS of
// them split the chunks of a row (round r gives wave ks chunk r*KS + ks) and W/KS
// take different weight rows.
// A wave owns 16*NT weight rows and 16*MT activation rows. Codes reach the
// waves through LDS: the codes and group tables of the block's rows for the next
// super-round (S rounds, S*KS chunks) are loaded in contiguous runs while the
// current one is multiplied and are written to LDS at its end; each lane then
// reads the dwords of its fragments from there. Activations are loaded DX
// rounds ahead into registers and written to one of two LDS buffers, in decoder
// pair order. One barrier per round, two per super-round. The KS partial tiles
// are added in a fixed order through LDS, so results are deterministic.
#include "qx_device.h"
#include "qx_internal.h"

namespace qx {

constexpr int kXRowBytes = 272;  // one activation row of one chunk (fragment order) + 16 B pad

// Codes and group tables of one (weight row, chunk) as one lane needs them.
template <int BITS, int KIND, int G>
struct LaneCodes {
  static constexpr int kDw = BITS == 4 ? 4 : 7;
  // Q4X: m[0] = the two groups' binary16 scales, m[1] = their selectors (bits 0-1, 2-3)
  static constexpr int kMetaDw = KIND == QX_UNIFORM ? 128 / G : KIND == QX_Q4X ? 2 : (128 / G) << (BITS - 1);
  uint32_t d[kDw];  // b = 3: d[0..2] code dwords g, 4+g, 8+g; d[3..4] dwords 2g, 2g+1;
                    //        d[5..6] dwords 8+2(g&1), 9+2(g&1) (bit 2 of the spare codes)
  uint32_t m[kMetaDw];
};

// LDS image of the codes and group tables of a block's weight rows for SC
// consecutive chunks (one super-round). Rows are padded so that the 16 rows read
// by one instruction start in different banks.
template <int BITS, int KIND, int G, int SC>
struct CodeTile {
  static constexpr int kRowBytes = BITS * SC * 16;
  static constexpr int kRowStride = kRowBytes + (272 - kRowBytes % 256) % 256;  // = 16 mod 256
  static constexpr int kMetaRow = KIND == QX_UNIFORM ? SC * (128 / G) * 4
                                  : KIND == QX_Q4X  ? SC * 8
                                                    : SC * (128 / G) * (2 << BITS);
  // padded by the width of a lane's table read (uniform: 4, 8 or 16 bytes for 1, 2 or 4
  // groups per chunk), so that every read is aligned to its width
  static constexpr int kMetaStride = kMetaRow + (KIND == QX_UNIFORM ? 4 * (128 / G) : KIND == QX_Q4X ? 8 : 16);
};

template <int BITS, int KIND, int G, int SC>
__device__ __forceinline__ void read_lane_codes(LaneCodes<BITS, KIND, G>& lc, const char* ct,
                                                const char* mt, int rl, int cl, int g) {
  using T = CodeTile<BITS, KIND, G, SC>;
  const char* row = ct + rl * T::kRowStride + cl * 16;
#pragma unroll
  for (int t = 0; t < (BITS == 4 ? 4 : 3); ++t)
    lc.d[t] = *reinterpret_cast<const uint32_t*>(row + t * SC * 16 + 4 * g);
  if constexpr (BITS == 3) {
    const u32x2 lo = *reinterpret_cast<const u32x2*>(row + (g >> 1) * SC * 16 + 8 * (g & 1));
    const u32x2 hi = *reinterpret_cast<const u32x2*>(row + 2 * SC * 16 + 8 * (g & 1));
    lc.d[3] = lo.x; lc.d[4] = lo.y; lc.d[5] = hi.x; lc.d[6] = hi.y;
  }
  constexpr int kDw = LaneCodes<BITS, KIND, G>::kMetaDw;
  const char* mp = mt + rl * T::kMetaStride + cl * kDw * 4;
  if constexpr (kDw == 1) {
    lc.m[0] = *reinterpret_cast<const uint32_t*>(mp);
  } else if constexpr (kDw == 2) {
    const u32x2 v = *reinterpret_cast<const u32x2*>(mp);
    lc.m[0] = v.x; lc.m[1] = v.y;
  } else {
#pragma unroll
    for (int i = 0; i < kDw / 4; ++i) {
      const u32x4 v = reinterpret_cast<const u32x4*>(mp)[i];
      lc.m[4 * i] = v.x; lc.m[4 * i + 1] = v.y; lc.m[4 * i + 2] = v.z; lc.m[4 * i + 3] = v.w;
    }
  }
}

// B fragment of k-step T for this lane (weights in register pair order). Q4X with
// SCALE = false: the sub-codebook entries alone (the group's scale applied to the sum).
template <int BITS, int KIND, int G, int T, bool SCALE = true>
__device__ __forceinline__ h8_t decode_frag(const LaneCodes<BITS, KIND, G>& lc,
                                            const GroupConsts<BITS, G>& gc,
                                            const LutGroup<BITS> (&lut)[128 / G],
                                            const DecodeConsts& k, uint32_t up, uint32_t dn,
                                            uint32_t ssh) {
  if constexpr (BITS == 4) {
    constexpr int gr = (32 * T) / G;
    const uint32_t D = lc.d[T], Ds = D >> 8;
    if constexpr (KIND == QX_UNIFORM) {
      return frag(deq((D & k.m000f) | k.mag1024, gc.z1024[gr], gc.sp[gr]),   // (0, 4)
                  deq((D & k.m00f0) | k.mag64, gc.zb[gr], gc.sp[gr]),       // (1, 5)
                  deq((Ds & k.m000f) | k.mag1024, gc.z1024[gr], gc.sp[gr]),  // (2, 6)
                  deq((Ds & k.m00f0) | k.mag64, gc.zb[gr], gc.sp[gr]));     // (3, 7)
    } else {
      uint32_t elo, ehi, olo, ohi;
      lut4_bytes(lut[gr], D & 0x0F0F0F0Fu, elo, ehi);         // codes 0 2 4 6
      lut4_bytes(lut[gr], (D >> 4) & 0x0F0F0F0Fu, olo, ohi);  // codes 1 3 5 7
      if constexpr (KIND == QX_Q4X && SCALE)  // fp16(s * CB[t][q]): one rounding, as qx_dequant
        return frag(hmul2(perm(ehi, elo, 0x06020400u), gc.sp[gr]), hmul2(perm(ohi, olo, 0x06020400u), gc.sp[gr]),
                    hmul2(perm(ehi, elo, 0x07030501u), gc.sp[gr]), hmul2(perm(ohi, olo, 0x07030501u), gc.sp[gr]));
      return frag(perm(ehi, elo, 0x06020400u), perm(ohi, olo, 0x06020400u),
                  perm(ehi, elo, 0x07030501u), perm(ohi, olo, 0x07030501u));
    }
  } else if constexpr (T < 3) {
    constexpr int ga = (16 * T) / G, gb = (48 + 16 * T) / G;
    const uint32_t D = lc.d[T];
    if constexpr (KIND == QX_UNIFORM) {
      const U3Pairs p = u3_fields(D, k);
      return frag(deq(p.a0, gc.z1024[ga], gc.sp[ga]), deq(p.a1, gc.z1024[ga], gc.sp[ga]),
                  deq(p.b0, gc.zb[gb], gc.sp[gb]), deq(p.b1, gc.zb[gb], gc.sp[gb]));
    } else {
      uint32_t a02, a13, b02, b13;
      lut3_pairs(lut[ga], u3_sel_a(D), a02, a13);
      lut3_pairs(lut[gb], u3_sel_b(D), b02, b13);
      return frag(a02, a13, b02, b13);
    }
  } else {
    constexpr int gs = 96 / G;
    uint32_t w[4];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint32_t L = lc.d[3 + h], H = lc.d[5 + h];
      if constexpr (KIND == QX_UNIFORM) {
        // bit 6 (spare dwords 0-3) or 7 (4-7) of bytes 0/2 and 1/3 of H -> bit 8 of each half
        const uint32_t t0 = ((H << up) & k.m0100) | k.mag16;
        const uint32_t t1 = ((H >> dn) & k.m0100) | k.mag16;
        w[2 * h] = deq((L & k.m00c0) | t0, gc.z16[gs], gc.sp[gs]);
        w[2 * h + 1] = deq(((L >> 8) & k.m00c0) | t1, gc.z16[gs], gc.sp[gs]);
      } else {
        const uint32_t S = ((L >> 6) & 0x03030303u) | ((H >> ssh) & 0x04040404u);
        lut3_pairs(lut[gs], S, w[2 * h], w[2 * h + 1]);
      }
    }
    return frag(w[0], w[1], w[2], w[3]);
  }
}

// Activation piece for fragment f of one row of one chunk: 16 bytes in the pair
// order of decode_frag. lo/hi are the two 8-byte halves read from X.
template <int BITS>
__device__ __forceinline__ void x_piece_offsets(int f, int& o1, int& o2) {  // in elements
  if (BITS == 4) {
    o1 = 8 * f; o2 = o1 + 4;
  } else {
    o1 = f < 12 ? 4 * f : 96 + 8 * (f - 12);
    o2 = f < 12 ? 48 + 4 * f : o1 + 4;
  }
}
template <int BITS>
__device__ __forceinline__ u32x4 x_piece(u32x2 lo, u32x2 hi) {
  u32x4 o;
  if (BITS == 4) {  // [x0 x1][x2 x3] [x4 x5][x6 x7] -> [x0 x4][x1 x5][x2 x6][x3 x7]
    o.x = perm(hi.x, lo.x, 0x05040100u);
    o.y = perm(hi.x, lo.x, 0x07060302u);
    o.z = perm(hi.y, lo.y, 0x05040100u);
    o.w = perm(hi.y, lo.y, 0x07060302u);
  } else {  // per four: [x0 x1][x2 x3] -> [x0 x2][x1 x3]
    o.x = perm(lo.y, lo.x, 0x05040100u);
    o.y = perm(lo.y, lo.x, 0x07060302u);
    o.z = perm(hi.y, hi.x, 0x05040100u);
    o.w = perm(hi.y, hi.x, 0x07060302u);
  }
  return o;
}

// Four int8 activation codes (the bytes of b) as exact binary16 pairs (v0, v1), (v2, v3):
// v + 128 in the fraction bits of 1024, minus 1152.
__device__ __forceinline__ u32x2 i8x4_to_h4(uint32_t b) {
  const uint32_t u = b ^ 0x80808080u;
  const uint32_t m1152 = 0xE480E480u;  // (-1152, -1152)
  return u32x2{hadd2(perm(0u, u, 0x0C010C00u) | kMagic1024, m1152),
               hadd2(perm(0u, u, 0x0C030C02u) | kMagic1024, m1152)};
}

// A8: X holds int8 activation codes [m][k] (qx_quantize_a8) and sx their per-row
// scales; the codes enter the products as exact binary16 integers and each output
// row is multiplied by its scale before rounding. Otherwise X is fp16 [m][k].
template <int BITS, int KIND, int G, int MT, int NT, int KS, int S, int DX, bool A8, int W = 4>
__global__ __launch_bounds__(64 * W) void gemm_kernel(const char* __restrict__ packed,
                                                             const void* __restrict__ Xv,
                                                             const float* __restrict__ sx,
                                                             uint16_t* __restrict__ Y, int n,
                                                             int k, int m, int nx, int my) {
  constexpr int NTH = 64 * W;   // threads per block
  constexpr int NG = W / KS;  // wave groups on different weight rows
  static_assert(W % KS == 0, "the k split divides the waves");
  constexpr int BM = 16 * MT, BN = 16 * NT * NG, SC = S * KS;
  using CT = CodeTile<BITS, KIND, G, SC>;
  constexpr int kXPieces = KS * BM * 16 / NTH;  // activation pieces per thread and round
  constexpr int kXBuf = KS * BM * kXRowBytes;
  constexpr int kCTotal = BN * BITS * SC;                                 // 16-byte code pieces
  constexpr int kCPieces = (kCTotal + NTH - 1) / NTH;  // per thread
  constexpr int kMetaUnit = KIND == QX_UNIFORM ? 4 : KIND == QX_Q4X ? 8 : 16;  // bytes per table load
  constexpr int kMPieces = (BN * CT::kMetaRow / kMetaUnit + NTH - 1) / NTH;
  static_assert(KS * BM * 16 % NTH == 0, "activation pieces must divide evenly");
  static_assert(S % DX == 0, "activation register sets must divide the super-round");
  static_assert((KS - 1) * NG * MT * NT * 1024 <= 2 * kXBuf, "reduction must fit the LDS buffers");
  __shared__ __align__(16) char xs[2 * kXBuf];
  __shared__ __align__(16) char cts[BN * CT::kRowStride];
  __shared__ __align__(16) char mts[BN * CT::kMetaStride];
  __shared__ __align__(16) uint32_t q4lut[KIND == QX_Q4X ? 32 : 1];

  // Block -> (weight tile bn, activation tile bm). With several activation tiles,
  // the tiles of one weight tile go to one XCD (workgroups are dealt to the 8 XCDs
  // round-robin), so its codes are fetched from HBM once and re-read from that L2.
  int bn, bm;
  if (my == 1) {
    bn = blockIdx.x; bm = 0;
  } else {
    const int q = blockIdx.x >> 3;
    bm = q % my;
    bn = (q / my) * 8 + (blockIdx.x & 7);
  }
  if (bn >= nx) return;  // padding blocks of the XCD mapping: whole block, before any barrier
  const int n0 = bn * BN, m0 = bm * BM;
  const int C = k >> 7, G_row = k / G, R = (C + KS - 1) / KS, NSR = (R + S - 1) / S;
  const size_t meta_off = (size_t)n * k * BITS / 8;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int ks = wave % KS, ng = wave / KS;
  const int g = lane >> 4, li = lane & 15;
  const DecodeConsts kc = decode_consts();
  const uint32_t up = g < 2 ? 2u : 1u, dn = g < 2 ? 6u : 7u, ssh = g < 2 ? 4u : 5u;

  // Codes of super-round j (chunks [j*SC, j*SC + SC)) of the block's rows: contiguous
  // runs of SC*16 bytes per (row, slice) and of the group tables per row, loaded
  // into registers at the start of super-round j - 1 (rows and chunks clamped in
  // bounds; the clamped copies are never multiplied) and written to LDS at its end.
  auto load_codes = [&](int j, u32x4 (&cr)[kCPieces], u32x4 (&mr)[kMPieces]) {
#pragma unroll
    for (int i = 0; i < kCPieces; ++i) {
      const int p = min((int)threadIdx.x + i * NTH, kCTotal - 1);
      const int cl = p % SC, sl = (p / SC) % BITS, rl = p / (SC * BITS);
      const int row = min(n0 + rl, n - 1), c = min(j * SC + cl, C - 1);
      cr[i] = *reinterpret_cast<const u32x4*>(packed + (((size_t)row * BITS + sl) * C + c) * 16);
    }
    constexpr int kUnits = CT::kMetaRow / kMetaUnit;  // per row
#pragma unroll
    for (int i = 0; i < kMPieces; ++i) {
      const int p = min((int)threadIdx.x + i * NTH, BN * kUnits - 1);
      const int ul = p % kUnits, rl = p / kUnits;
      const int row = min(n0 + rl, n - 1);
      if constexpr (KIND == QX_Q4X) {
        // chunk c of the row: the scales of groups 2c, 2c + 1 (one dword) and their
        // selectors (4 bits of the row's selector word for groups 16(c/8) ..)
        const int c = min(j * SC + ul, C - 1), sel_words = (G_row + 15) / 16;
        const uint32_t sc = *reinterpret_cast<const uint32_t*>(packed + meta_off + ((size_t)row * G_row + 2 * c) * 2);
        const uint32_t sw = *reinterpret_cast<const uint32_t*>(packed + meta_off + meta_off / 16 +
                                                               ((size_t)row * sel_words + c / 8) * 4);
        mr[i] = u32x4{sc, (sw >> (4 * (c % 8))) & 0xFu, 0u, 0u};
        continue;
      }
      // group index of this unit, clamped to the row's last group
      const int gi = min(j * SC * (128 / G) + ul * kMetaUnit / (KIND == QX_UNIFORM ? 4 : 2 << BITS),
                         G_row - 1);
      const char* src = packed + meta_off + ((size_t)row * G_row + gi) * (KIND == QX_UNIFORM ? 4 : 2 << BITS);
      if constexpr (KIND == QX_UNIFORM)
        mr[i] = u32x4{*reinterpret_cast<const uint32_t*>(src), 0u, 0u, 0u};
      else
        mr[i] = *reinterpret_cast<const u32x4*>(src + (ul * 16) % (2 << BITS));
    }
  };
  auto store_codes = [&](const u32x4 (&cr)[kCPieces], const u32x4 (&mr)[kMPieces]) {
#pragma unroll
    for (int i = 0; i < kCPieces; ++i) {
      const int p = threadIdx.x + i * NTH;
      const int cl = p % SC, sl = (p / SC) % BITS, rl = p / (SC * BITS);
      if (kCTotal % NTH == 0 || p < kCTotal)
        *reinterpret_cast<u32x4*>(cts + rl * CT::kRowStride + sl * SC * 16 + cl * 16) = cr[i];
    }
    constexpr int kUnits = CT::kMetaRow / kMetaUnit;
#pragma unroll
    for (int i = 0; i < kMPieces; ++i) {
      const int p = threadIdx.x + i * NTH;
      if (p < BN * kUnits) {
        const int ul = p % kUnits, rl = p / kUnits;
        char* dst = mts + rl * CT::kMetaStride + ul * kMetaUnit;
        if constexpr (KIND == QX_UNIFORM)
          *reinterpret_cast<uint32_t*>(dst) = mr[i].x;
        else if constexpr (KIND == QX_Q4X)
          *reinterpret_cast<u32x2*>(dst) = u32x2{mr[i].x, mr[i].y};
        else
          *reinterpret_cast<u32x4*>(dst) = mr[i];
      }
    }
  };
  // activation pieces of round r into registers (rows and chunks clamped in bounds;
  // rows past m are never stored, chunks past C are never multiplied)
  auto load_x = [&](int r, u32x2 (&lo)[kXPieces], u32x2 (&hi)[kXPieces]) {
#pragma unroll
    for (int i = 0; i < kXPieces; ++i) {
      const int p = threadIdx.x + i * NTH;
      const int f = p & 15, ml = (p >> 4) % BM, kq = p / (16 * BM);
      const int c = min(r * KS + kq, C - 1), row = min(m0 + ml, m - 1);
      int o1, o2;
      x_piece_offsets<BITS>(f, o1, o2);
      if constexpr (A8) {
        const int8_t* src = static_cast<const int8_t*>(Xv) + (size_t)row * k + (size_t)c * 128;
        lo[i] = i8x4_to_h4(*reinterpret_cast<const uint32_t*>(src + o1));
        hi[i] = i8x4_to_h4(*reinterpret_cast<const uint32_t*>(src + o2));
      } else {
        const uint16_t* src = static_cast<const uint16_t*>(Xv) + (size_t)row * k + (size_t)c * 128;
        lo[i] = *reinterpret_cast<const u32x2*>(src + o1);
        hi[i] = *reinterpret_cast<const u32x2*>(src + o2);
      }
    }
  };
  auto store_x = [&](int buf, const u32x2 (&lo)[kXPieces], const u32x2 (&hi)[kXPieces]) {
#pragma unroll
    for (int i = 0; i < kXPieces; ++i) {
      const int p = threadIdx.x + i * NTH;
      const int f = p & 15, ml = (p >> 4) % BM, kq = p / (16 * BM);
      *reinterpret_cast<u32x4*>(xs + buf * kXBuf + (kq * BM + ml) * kXRowBytes + 16 * f) =
          x_piece<BITS>(lo[i], hi[i]);
    }
  };

  f4_t acc[MT][NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = f4_t{0.f, 0.f, 0.f, 0.f};
  // Q4X with 8-bit activations: k-steps 0-1 / 2-3 of a chunk are its groups 0 / 1; their
  // sums of CB[t][q] * xq come from the matrix cores and are scaled by the group's s in
  // fp32 (the exact s * CB of qx_gemv_a8, not W' rounded to binary16)
  constexpr bool kQ4xGroupSums = A8 && KIND == QX_Q4X;
  f4_t gsum[kQ4xGroupSums ? MT : 1][kQ4xGroupSums ? NT : 1];

  u32x4 cr[kCPieces], mr[kMPieces];
  if constexpr (KIND == QX_Q4X) stage_q4x_tables(packed + q4x_offsets(n, k).codebook, q4lut);
  load_codes(0, cr, mr);
  store_codes(cr, mr);
  // Activations: round r + DX is loaded into register set r % DX during round r, and
  // round r + 1 (loaded DX - 1 rounds earlier) is written to LDS buffer (r + 1) & 1
  // at its end, so every load has DX rounds to arrive.
  u32x2 xlo[DX][kXPieces], xhi[DX][kXPieces];
  load_x(0, xlo[0], xhi[0]);
  store_x(0, xlo[0], xhi[0]);
#pragma unroll
  for (int i = 1; i < DX; ++i) load_x(i, xlo[i], xhi[i]);
  __syncthreads();

  // Every load is issued unconditionally (indices clamped in bounds) so that the
  // compiler waits for exactly the loads a step consumes; rounds past the last
  // chunk multiply nothing.
  for (int j = 0; j < NSR; ++j) {
    load_codes(j + 1, cr, mr);
#pragma unroll
    for (int u = 0; u < S; ++u) {
      const int r = j * S + u;
      load_x(r + DX, xlo[u % DX], xhi[u % DX]);
      if (r * KS + ks < C) {
        const char* xb = xs + (r & 1) * kXBuf + ks * BM * kXRowBytes;
        LaneCodes<BITS, KIND, G> cur[NT];
        GroupConsts<BITS, G> gc[NT];
        LutGroup<BITS> lut[NT][128 / G];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
          read_lane_codes<BITS, KIND, G, SC>(cur[nt], cts, mts, 16 * (ng * NT + nt) + li, u * KS + ks, g);
          if constexpr (KIND == QX_UNIFORM) {
            gc[nt] = group_consts<BITS, G>(cur[nt].m);
          } else if constexpr (KIND == QX_Q4X) {
#pragma unroll
            for (int i = 0; i < 2; ++i) {  // group i of the chunk: scale pair, sub-codebook tables
              gc[nt].sp[i] = perm(cur[nt].m[0], cur[nt].m[0], i == 0 ? 0x01000100u : 0x03020302u);
              const uint32_t* tp = q4lut + 8 * ((cur[nt].m[1] >> (2 * i)) & 3u);
              const u32x4 tl = *reinterpret_cast<const u32x4*>(tp), th = *reinterpret_cast<const u32x4*>(tp + 4);
              lut[nt][i] = LutGroup<4>{{tl.x, tl.y, tl.z, tl.w}, {th.x, th.y, th.z, th.w}};
            }
          } else {
#pragma unroll
            for (int i = 0; i < 128 / G; ++i) lut[nt][i] = lut_group<BITS>(&cur[nt].m[i << (BITS - 1)]);
          }
        }
#define QX_GEMM_KSTEP(T)                                                                      \
  {                                                                                           \
    h8_t a[MT];                                                                               \
    _Pragma("unroll") for (int mt = 0; mt < MT; ++mt) a[mt] = *reinterpret_cast<const h8_t*>( \
        xb + (16 * mt + li) * kXRowBytes + 64 * (T) + 16 * g);                                \
    _Pragma("unroll") for (int nt = 0; nt < NT; ++nt) {                                       \
      const h8_t b = decode_frag<BITS, KIND, G, T, !kQ4xGroupSums>(cur[nt], gc[nt], lut[nt], kc, up, dn, ssh); \
      _Pragma("unroll") for (int mt = 0; mt < MT; ++mt) {                                     \
        if constexpr (kQ4xGroupSums)                                                          \
          gsum[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(                             \
              a[mt], b, (T) % 2 == 0 ? f4_t{0.f, 0.f, 0.f, 0.f} : gsum[mt][nt], 0, 0, 0);     \
        else                                                                                  \
          acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[mt], b, acc[mt][nt], 0, 0, 0); \
      }                                                                                       \
    }                                                                                         \
    if constexpr (kQ4xGroupSums && (T) % 2 == 1) { /* the group's scale on its sum */         \
      _Pragma("unroll") for (int nt = 0; nt < NT; ++nt) {                                     \
        const float sg = half_bits_to_float((cur[nt].m[0] >> (8 * (T) - 8)) & 0xFFFFu);       \
        _Pragma("unroll") for (int mt = 0; mt < MT; ++mt) acc[mt][nt] += sg * gsum[mt][nt];   \
      }                                                                                       \
    }                                                                                         \
  }
        QX_GEMM_KSTEP(0)
        QX_GEMM_KSTEP(1)
        QX_GEMM_KSTEP(2)
        QX_GEMM_KSTEP(3)
#undef QX_GEMM_KSTEP
      }
      store_x((r + 1) & 1, xlo[(u + 1) % DX], xhi[(u + 1) % DX]);
      __syncthreads();
    }
    store_codes(cr, mr);  // every wave is past the super-round's last read of the tile
    __syncthreads();
  }

  // KS partial tiles -> one, in ks order, through LDS (every wave passed the last barrier)
  if constexpr (KS > 1) {
    float* red = reinterpret_cast<float*>(xs);
    if (ks > 0) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
          *reinterpret_cast<f4_t*>(red + ((((ks - 1) * NG + ng) * MT + mt) * NT + nt) * 256 + 4 * lane) =
              acc[mt][nt];
    }
    __syncthreads();
    if (ks > 0) return;
#pragma unroll
    for (int q = 1; q < KS; ++q)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
          acc[mt][nt] += *reinterpret_cast<const f4_t*>(
              red + ((((q - 1) * NG + ng) * MT + mt) * NT + nt) * 256 + 4 * lane);
  }

  // D[i][j] of a 16x16 tile: lane holds rows 4*(lane/16) + r, column lane % 16
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) {
    const int col = n0 + 16 * (ng * NT + nt) + li;
    if (col < n) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = m0 + 16 * mt + 4 * g + r;
          if (row < m)
            Y[(size_t)row * n + col] = (uint16_t)float_to_half_bits(A8 ? acc[mt][nt][r] * sx[row] : acc[mt][nt][r]);
        }
    }
  }
}

template <int BITS, int KIND, int G, int MT, int NT, int KS, int S, int DX, bool A8, int W = 4>
static void launch_gemm_cfg(const qx_desc* d, const char* p, int m, const void* X, const float* sx,
                            uint16_t* Y, hipStream_t s) {
  constexpr int BN = 16 * NT * (W / KS), BM = 16 * MT;
  const int nx = (d->n + BN - 1) / BN, my = (m + BM - 1) / BM;
  const unsigned blocks = my == 1 ? (unsigned)nx : (unsigned)((nx + 7) / 8) * 8u * (unsigned)my;
  hipLaunchKernelGGL((gemm_kernel<BITS, KIND, G, MT, NT, KS, S, DX, A8, W>), dim3(blocks), dim3(64 * W),
                     0, s, p, X, sx, Y, d->n, d->k, m, nx, my);
}

// Tile shape per activation row count (from a sweep of MT, NT, KS, S, DX on the
// 3-bit g64 MLP shapes at m = 16, 64, 512, and at m = 128-512 a split of k when
// the tiles are few: uniform 4096x11008 at m = 128 took 113 us whole and 57 us
// split four ways, codebook-3 78 and 55 us split two ways; at m = 32, 35 and 27 us
// with four waves instead of two on each 32 x 32 tile). Small m is bound by streaming the codes:
// one 16-row activation tile, 16 weight rows per block and the chunks of a row
// split over the four waves, so that the grid has enough blocks. Larger m gets
// larger activation tiles so that each decoded weight feeds more MFMAs; with
// m > 64 a wave owns 64 activation x 32 weight rows.
#ifndef QX_GEMM_CFG
#define QX_GEMM_CFG 0  // 0: by m; 1, 2, 4 force one shape
#endif
#ifndef QX_GEMM_MID_W
// rows of more than 64 chunks at 16 < m <= 64: the k split over 8 waves instead of 4
// (4096x11008 at m = 64: uniform-3 39.9 -> 33.4 us, uniform-4 37.1 -> 29.1, codebook-3
// 34.8 -> 31.3); 4 keeps the 4-wave shape
#define QX_GEMM_MID_W 8
#endif
#ifndef QX_GEMM_BIG_W
// m > 64, rows of more than 64 chunks, 129-256 tiles (one block of 8 waves per compute
// unit): k split over 2 of 8 waves instead of walked by one (4096x11008 at m = 512:
// uniform-3 122.7 -> 98.4 us, uniform-4 101.2 -> 84.4; codebook-3 at m = 256 78.6 ->
// 61.8, but 112.7 -> 120.3 at m = 512, 512 tiles); 4 keeps the 4-wave shapes
#define QX_GEMM_BIG_W 8
#endif
#ifndef QX_GEMM_BIG_S
#define QX_GEMM_BIG_S 4  // super-round (rounds per code load) of the 128 x 192 blocks
#endif
#ifndef QX_GEMM_BIG_DX
#define QX_GEMM_BIG_DX 1  // activation rounds in flight of the 128 x 192 blocks (11008x4096 u3g64 m = 512: 95.1 us with 2, 89.8 with 1)
#endif
#ifndef QX_GEMM_SMALL_W
#define QX_GEMM_SMALL_W 4  // 4: waves per block for m <= 16 by shape; 8, 16 force (sweeps)
#endif
template <int BITS, int KIND, int G, bool A8 = false>
static int launch_gemm_t(const qx_desc* d, const void* packed, int m, const void* X, const float* sx,
                         uint16_t* Y, hipStream_t s) {
  const char* p = static_cast<const char*>(packed);
  constexpr bool kUni = KIND == QX_UNIFORM;
  const int cfg = QX_GEMM_CFG > 0 ? QX_GEMM_CFG : m <= 16 ? 1 : m <= 64 ? 2 : 4;
  switch (cfg) {
    case 1: {
      // rows of more than 64 chunks: the k split over 8 waves (codebook, Q4X) or 16
      // (uniform, m <= 8), each walking fewer chunks; 4096x11008 at m = 16 took 24.7 us
      // (codebook-3) and 24.6 (Q4X) with 4 waves, 19.5 and 19.2 with 8, uniform-3 at
      // m = 8 18.2 and 16.1 with 16 (shorter rows were slower split wider)
      const int C = d->k / 128;
      const int w = QX_GEMM_SMALL_W != 4 ? QX_GEMM_SMALL_W
                    : C > 64 ? (!kUni ? 8 : m <= 8 ? 16 : 4) : 4;
      if constexpr (kUni) {
        if (w == 16) launch_gemm_cfg<BITS, KIND, G, 1, 1, 16, 1, 1, A8, 16>(d, p, m, X, sx, Y, s);
        else if (w == 8) launch_gemm_cfg<BITS, KIND, G, 1, 1, 8, 1, 1, A8, 8>(d, p, m, X, sx, Y, s);
        else launch_gemm_cfg<BITS, KIND, G, 1, 1, 4, 2, 2, A8>(d, p, m, X, sx, Y, s);
      } else {  // 16 waves do not fit the tables of the codebook formats in LDS
        if (w >= 8) launch_gemm_cfg<BITS, KIND, G, 1, 1, 8, 1, 1, A8, 8>(d, p, m, X, sx, Y, s);
        else launch_gemm_cfg<BITS, KIND, G, 1, 1, 4, 1, 1, A8>(d, p, m, X, sx, Y, s);
      }
      break;
    }
    case 2:
      if constexpr (kUni) {
        // at most 128 tiles of 32 x 32 (a 4096-row matrix at m <= 32): four waves per tile
        const long tiles = (long)((d->n + 31) / 32) * ((m + 31) / 32);
        if (QX_GEMM_CFG == 0 && tiles <= 128) launch_gemm_cfg<BITS, KIND, G, 2, 1, 4, 2, 1, A8>(d, p, m, X, sx, Y, s);
        else if (QX_GEMM_MID_W == 8 && d->k > 64 * 128) launch_gemm_cfg<BITS, KIND, G, 2, 1, 4, 2, 1, A8, 8>(d, p, m, X, sx, Y, s);
        else launch_gemm_cfg<BITS, KIND, G, 2, 1, 2, 2, 1, A8>(d, p, m, X, sx, Y, s);
      } else {
        if (QX_GEMM_MID_W == 8 && d->k > 64 * 128) launch_gemm_cfg<BITS, KIND, G, 2, 1, 4, 2, 2, A8, 8>(d, p, m, X, sx, Y, s);
        else launch_gemm_cfg<BITS, KIND, G, 2, 1, 2, 2, 2, A8>(d, p, m, X, sx, Y, s);
      }
      break;
    default:
      if constexpr (kUni) {
        // few 128 x 64 tiles (e.g. 4096 weight rows at m <= 256): split k over the waves
        const long tiles = (long)((d->n + 127) / 128) * ((m + 63) / 64);
        // many rows: 128 x 48 per wave (each decoded fragment feeds 8 products) in
        // 128 x 192 blocks, one per compute unit, where the last round of blocks keeps
        // most units busy (11008x4096 uniform-3 at m = 512: 110 -> 91 us, m = 1024 193
        // -> 165; 22016x4096 m = 512 183 -> 163; but 11008 rows at m = 768, two rounds
        // with 92 blocks in the second, 166 against 167). 128 x 32 per wave in 128 x 256
        // blocks of 8 waves (two per SIMD: about 30 % more work per compute unit in the
        // same time) where those take fewer rounds of blocks (11008x4096 uniform-3 g64 at
        // m = 2048: 298.7 -> 248.3 us, 12288x4096 299.6 -> 255.0, 22016x4096 at m = 1024
        // 297.5 -> 241.0; with as many rounds, e.g. 11008 rows at m = 512, 76.8 against
        // 79.3 for the 4-wave blocks). Not for 3-bit g32, whose 8-wave tile spills.
        const long mb = (m + 127) / 128;
        const long big = (long)((d->n + 191) / 192) * mb, big8 = (long)((d->n + 255) / 256) * mb;
        const long last = big % 256 == 0 ? 256 : big % 256;
        constexpr bool kBig8 = !(BITS == 3 && G == 32);
        if (kBig8 && QX_GEMM_CFG == 0 && m >= 384 && (big8 + 255) / 256 < (big + 255) / 256) {
          if constexpr (kBig8)
            launch_gemm_cfg<BITS, KIND, G, 8, 2, 1, QX_GEMM_BIG_S, QX_GEMM_BIG_DX, A8, 8>(d, p, m, X, sx, Y, s);
        } else if (QX_GEMM_CFG == 0 && m >= 384 && last >= 150)
          launch_gemm_cfg<BITS, KIND, G, 8, 3, 1, QX_GEMM_BIG_S, QX_GEMM_BIG_DX, A8>(d, p, m, X, sx, Y, s);
        else if (QX_GEMM_CFG == 0 && tiles <= 64) launch_gemm_cfg<BITS, KIND, G, 4, 2, 4, 1, 1, A8>(d, p, m, X, sx, Y, s);
        else if (QX_GEMM_CFG == 0 && tiles <= 128) launch_gemm_cfg<BITS, KIND, G, 4, 2, 2, 4, 2, A8>(d, p, m, X, sx, Y, s);
        else if (QX_GEMM_BIG_W == 8 && d->k > 64 * 128 && tiles <= 256)
          launch_gemm_cfg<BITS, KIND, G, 4, 2, 2, 4, 2, A8, 8>(d, p, m, X, sx, Y, s);
        else launch_gemm_cfg<BITS, KIND, G, 4, 2, 1, 4, 2, A8>(d, p, m, X, sx, Y, s);
      } else {
        // codebook and Q4X: 64 x 64 tiles; at most 128 of them split k over two waves
        const long tiles = (long)((d->n + 63) / 64) * ((m + 63) / 64);
        if (QX_GEMM_CFG == 0 && tiles <= 128) launch_gemm_cfg<BITS, KIND, G, 4, 1, 2, 4, 2, A8>(d, p, m, X, sx, Y, s);
        else if (QX_GEMM_BIG_W == 8 && d->k > 64 * 128 && tiles <= 256 && !(BITS == 4 && G == 32)) {
          if constexpr (!(BITS == 4 && G == 32))  // 32-code tables of 16 entries overflow LDS at 8 waves
            launch_gemm_cfg<BITS, KIND, G, 4, 1, 2, 4, 2, A8, 8>(d, p, m, X, sx, Y, s);
        } else {
          launch_gemm_cfg<BITS, KIND, G, 4, 1, 1, 4, 2, A8>(d, p, m, X, sx, Y, s);
        }
      }
      break;
  }
  return hipGetLastError() == hipSuccess ? QX_OK : QX_E_HIP;
}

int launch_gemm(const qx_desc* d, const void* packed, int m, const uint16_t* X, uint16_t* Y,
                hipStream_t s) {
#define QX_GEMM_CASE(B, K, G) \
  if (d->bits == B && d->kind == K && d->group == G) return launch_gemm_t<B, K, G>(d, packed, m, X, nullptr, Y, s);
  QX_GEMM_CASE(3, 0, 32) QX_GEMM_CASE(3, 0, 64) QX_GEMM_CASE(3, 0, 128)
  QX_GEMM_CASE(3, 1, 32) QX_GEMM_CASE(3, 1, 64) QX_GEMM_CASE(3, 1, 128)
  QX_GEMM_CASE(4, 0, 32) QX_GEMM_CASE(4, 0, 64) QX_GEMM_CASE(4, 0, 128)
  QX_GEMM_CASE(4, 1, 32) QX_GEMM_CASE(4, 1, 64) QX_GEMM_CASE(4, 1, 128)
  QX_GEMM_CASE(4, 2, 64)
#undef QX_GEMM_CASE
  return QX_E_UNSUPPORTED;
}

// Codebook and Q4X weights with int8 activation rows (qx_gemm_a8): the fp16 matrix-core
// GEMM above on the activation codes, scaled per row.
int launch_gemm_lut_a8(const qx_desc* d, const void* packed, int m, const int8_t* Xq, const float* sx,
                       uint16_t* Y, hipStream_t s) {
#define QX_GEMM_A8_CASE(B, K, G) \
  if (d->bits == B && d->kind == K && d->group == G) return launch_gemm_t<B, K, G, true>(d, packed, m, Xq, sx, Y, s);
  QX_GEMM_A8_CASE(3, 1, 32) QX_GEMM_A8_CASE(3, 1, 64) QX_GEMM_A8_CASE(3, 1, 128)
  QX_GEMM_A8_CASE(4, 1, 32) QX_GEMM_A8_CASE(4, 1, 64) QX_GEMM_A8_CASE(4, 1, 128)
  QX_GEMM_A8_CASE(4, 2, 64)
#undef QX_GEMM_A8_CASE
  return QX_E_UNSUPPORTED;
}

}  // namespace qx
