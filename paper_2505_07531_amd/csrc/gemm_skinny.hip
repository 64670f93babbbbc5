// Small-batch quantized GEMM on the matrix cores: Y[m][n] = sum_k X[m][k] W'[n][k]
// for 2 <= m <= 64 activation rows (decode of several sequences, short prefill chunks).
//
// With few activation rows the product is still bound by streaming the packed
// weights (decoding is memory-bound, Section 2.4 of the paper), so this kernel
// keeps the GEMV's access pattern and puts only the multiply on the matrix
// cores:
//
//   * a lane owns one (weight row, 128-code chunk) item, read with b 16-byte
//     loads from the slice planes, exactly as the GEMV reads it; no code byte
//     goes through LDS;
//   * the lane decodes its chunk into sixteen 8-weight pieces, each the B
//     fragment of one v_mfma_f32_16x16x32_f16: lane l holds k-slice l / 16 of
//     column l % 16, so the 16 lanes of a lane group are 16 weight rows on the
//     same chunk, and the four lane groups are four chunks whose products the
//     instruction adds;
//   * uniform weights are dequantized exactly, fp16(s (q - z)), by one packed add
//     of exact integers and one packed multiply (the arithmetic of qx_dequant),
//     codebook weights are table entries fetched with v_perm_b32, Q4X entries
//     times the group's scale;
//   * the A fragment of a piece is the 8 activations of the piece's positions in
//     the decoder's pair order; a wave stages up to 16 activation rows of its four
//     chunks in its own LDS rows with coalesced loads and reads the fragments
//     from there (rows past the tile repeat its last row and are not stored);
//     more than 16 rows are taken as 16-row tiles in turn, the codes decoded again
//     for each;
//   * the W waves of a block share its 16*RF weight rows and split the chunks
//     (wave w takes chunks 4(w + W j) .. + 3 for j < J); their 16x16 fp32 tiles are
//     added in wave order through LDS, so results are deterministic.
//
// RF weight-row fragments share each A fragment: tall matrices take three per
// wave, which puts one block on nearly every compute unit of an 11008-row matrix.
// That form loads all its codes before its first product, so each compute unit
// streams only until its one block has its data. Where a compute unit holds fewer rows
// in the pipelined form below (one block per compute unit, activations staged once, two
// 16-row groups in flight per wave while the previous one is multiplied), or four
// groups or more, rows of at most 32 chunks at m <= 16 take that form (22016x4096
// uniform-4 g128 at m = 2 / 16: 16.0 / 17.6 us -> 13.8 / 15.2; 16400x4096 uniform-3 g64
// 13.6 / 15.3 -> 10.8 / 12.2; 8192x4096 7.9 / 9.3 -> 7.0 / 8.5; 11008 and 12288 rows,
// 48 rows per compute unit in both forms: the one-shot form measured equal or faster,
// except for Q4X at m >= 3: 11008x4096 13.8 / 14.3 / 15.1 -> 12.6 / 12.5 / 13.3 at m = 4 /
// 8 / 16, 12288x4096 14.0 / 14.6 / 15.4 -> 12.5 / 12.7 / 13.6).
// qx_gemm routes m rows here where it measured faster (gemm_skinny_applies).
#include <atomic>
#include <utility>

#include "gemv_common.h"

namespace qx {
namespace {

// Activation pieces in the decoders' pair order: b = 4 (0,4) (1,5) (2,6) (3,7);
// b = 3 per four values (0,2) (1,3).
template <int BITS>
__device__ __forceinline__ h8_t x_frag(const u32x4 v) {
  if constexpr (BITS == 4)
    return frag(perm(v.z, v.x, 0x05040100u), perm(v.z, v.x, 0x07060302u), perm(v.w, v.y, 0x05040100u),
                perm(v.w, v.y, 0x07060302u));
  else
    return frag(perm(v.y, v.x, 0x05040100u), perm(v.y, v.x, 0x07060302u), perm(v.w, v.z, 0x05040100u),
                perm(v.w, v.z, 0x07060302u));
}

// Per-item decode tables: uniform scale / zero pairs, or the codebook (Q4X: the
// selected sub-codebooks and the scale pairs) of the item's groups.
template <int BITS, int KIND, int G>
struct ItemTables {
  static constexpr int NG = 128 / G;
  GroupConsts<BITS, G> gc;  // uniform; Q4X uses sp
  LutGroup<BITS> lut[KIND == QX_UNIFORM ? 1 : NG];
};

// valid = false (a chunk slot past the end of the row): tables whose every weight is
// +-0, so that the slot adds nothing to the lane group's sum.
template <int BITS, int KIND, int G>
__device__ __forceinline__ ItemTables<BITS, KIND, G> item_tables(const Item<BITS, KIND, G>& it,
                                                                 const uint32_t* q4lut, bool valid) {
  ItemTables<BITS, KIND, G> t;
  if constexpr (KIND == QX_UNIFORM) {
    t.gc = group_consts<BITS, G>(it.m);
#pragma unroll
    for (int g = 0; g < 128 / G; ++g) t.gc.sp[g] = valid ? t.gc.sp[g] : 0u;  // s (q - z) -> +-0
  } else if constexpr (KIND == QX_Q4X) {
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      t.gc.sp[g] = perm(it.m[0], it.m[0], g == 0 ? 0x01000100u : 0x03020302u);
      const uint32_t* tp = q4lut + 8 * ((it.m[1] >> (2 * g)) & 3u);
      const u32x4 tl = *reinterpret_cast<const u32x4*>(tp), th = *reinterpret_cast<const u32x4*>(tp + 4);
      t.lut[g] = LutGroup<4>{{tl.x, tl.y, tl.z, tl.w}, {th.x, th.y, th.z, th.w}};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        t.lut[g].lo[i] = valid ? t.lut[g].lo[i] : 0u;
        t.lut[g].hi[i] = valid ? t.lut[g].hi[i] : 0u;
      }
    }
  } else {
#pragma unroll
    for (int g = 0; g < 128 / G; ++g) {
      t.lut[g] = lut_group<BITS>(&it.m[g << (BITS - 1)]);
#pragma unroll
      for (int i = 0; i < (1 << BITS) / 4; ++i) {
        t.lut[g].lo[i] = valid ? t.lut[g].lo[i] : 0u;
        t.lut[g].hi[i] = valid ? t.lut[g].hi[i] : 0u;
      }
    }
  }
  return t;
}

// B fragment of piece P (codes 8P .. 8P + 7 of the chunk) in the decoder's pair order.
//   b = 4: code dword P;
//   b = 3: P < 6: bits 0-2 fields of code dwords 2P, 2P + 1; 6 <= P < 12: bits 3-5
//          fields of dwords 2(P - 6), 2(P - 6) + 1; P >= 12: spare codes of dwords
//          2(P - 12), 2(P - 12) + 1 (bit 2 in dword 8 + (i & 3)).
template <int BITS, int KIND, int G, int P>
__device__ __forceinline__ h8_t piece_frag(const Item<BITS, KIND, G>& it, const ItemTables<BITS, KIND, G>& t,
                                           const DecodeConsts& k) {
  constexpr int gr = (8 * P) / G;  // the piece's group within the chunk
  if constexpr (BITS == 4) {
    const uint32_t D = it.d[P], Ds = D >> 8;
    if constexpr (KIND == QX_UNIFORM) {
      const GroupConsts<4, G>& gc = t.gc;
      return frag(deq((D & k.m000f) | k.mag1024, gc.z1024[gr], gc.sp[gr]),   // (0, 4)
                  deq((D & k.m00f0) | k.mag64, gc.zb[gr], gc.sp[gr]),       // (1, 5)
                  deq((Ds & k.m000f) | k.mag1024, gc.z1024[gr], gc.sp[gr]),  // (2, 6)
                  deq((Ds & k.m00f0) | k.mag64, gc.zb[gr], gc.sp[gr]));     // (3, 7)
    } else {
      uint32_t elo, ehi, olo, ohi;
      lut4_bytes(t.lut[gr], D & 0x0F0F0F0Fu, elo, ehi);         // codes 0 2 4 6
      lut4_bytes(t.lut[gr], (D >> 4) & 0x0F0F0F0Fu, olo, ohi);  // codes 1 3 5 7
      const uint32_t p0 = perm(ehi, elo, 0x06020400u), p1 = perm(ohi, olo, 0x06020400u);
      const uint32_t p2 = perm(ehi, elo, 0x07030501u), p3 = perm(ohi, olo, 0x07030501u);
      if constexpr (KIND == QX_Q4X)  // fp16(s * CB[t][q]): one rounding, as qx_dequant
        return frag(hmul2(p0, t.gc.sp[gr]), hmul2(p1, t.gc.sp[gr]), hmul2(p2, t.gc.sp[gr]),
                    hmul2(p3, t.gc.sp[gr]));
      return frag(p0, p1, p2, p3);
    }
  } else if constexpr (P < 12) {
    constexpr bool kA = P < 6;
    constexpr int i0 = kA ? 2 * P : 2 * (P - 6);
    uint32_t w[4];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const uint32_t D = it.d[i0 + h];
      if constexpr (KIND == QX_UNIFORM) {
        const U3Pairs p = u3_fields(D, k);
        if constexpr (kA) {
          w[2 * h] = deq(p.a0, t.gc.z1024[gr], t.gc.sp[gr]);
          w[2 * h + 1] = deq(p.a1, t.gc.z1024[gr], t.gc.sp[gr]);
        } else {
          w[2 * h] = deq(p.b0, t.gc.zb[gr], t.gc.sp[gr]);
          w[2 * h + 1] = deq(p.b1, t.gc.zb[gr], t.gc.sp[gr]);
        }
      } else {
        lut3_pairs(t.lut[gr], kA ? u3_sel_a(D) : u3_sel_b(D), w[2 * h], w[2 * h + 1]);
      }
    }
    return frag(w[0], w[1], w[2], w[3]);
  } else {
    uint32_t w[4];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      constexpr int kI0 = 2 * (P - 12);
      const int i = kI0 + h;  // code dword of the spare codes; bit 2 in dword 8 + (i & 3)
      const uint32_t D = it.d[kI0 + h], H = it.d[8 + ((kI0 + h) & 3)];
      if constexpr (KIND == QX_UNIFORM) {
        // bit 6 (dwords 0-3) or 7 (4-7) of bytes 0/2 and 1/3 of H -> bit 8 of each half
        const uint32_t up = i < 4 ? 2u : 1u, dn = i < 4 ? 6u : 7u;
        const uint32_t t0 = ((H << up) & k.m0100) | k.mag16;
        const uint32_t t1 = ((H >> dn) & k.m0100) | k.mag16;
        w[2 * h] = deq((D & k.m00c0) | t0, t.gc.z16[gr], t.gc.sp[gr]);
        w[2 * h + 1] = deq(((D >> 8) & k.m00c0) | t1, t.gc.z16[gr], t.gc.sp[gr]);
      } else {
        const uint32_t ssh = i < 4 ? 4u : 5u;  // bit 6 or 7 of each byte -> bit 2
        const uint32_t S = ((D >> 6) & 0x03030303u) | ((H >> ssh) & 0x04040404u);
        lut3_pairs(t.lut[gr], S, w[2 * h], w[2 * h + 1]);
      }
    }
    return frag(w[0], w[1], w[2], w[3]);
  }
}

// One staged activation row of a wave's four chunks (1 KB) plus 16 bytes, so that
// the 16 rows that one lane group reads start in different banks.
constexpr int kXRow = 1024 + 16;

#ifndef QX_SKINNY_PIN
#define QX_SKINNY_PIN 1
#endif
#ifndef QX_SKINNY_AHEAD
#define QX_SKINNY_AHEAD 1  // items whose codes are requested before the first product
#endif

// Block: W = blockDim.x / 64 waves on weight rows n0 .. n0 + 16 RF - 1. Lane l of
// wave w: column (weight row) n0 + 16 f + l % 16 of fragment f, chunk
// 4 (w + W j) + l / 16 of item j, activation row 16 mt + l % 16 of tile mt (rows past
// the tile's last repeat it). Up to MT tiles of 16 activation rows are taken in turn;
// the codes stay in registers and are decoded again for each tile.
//
// Activations: the rows of an item's four chunks are contiguous 1 KB runs, so the
// wave loads each run with one fully coalesced 16-byte-per-lane load (lane l: chunk
// l / 16, piece l % 16), permutes it into the decoders' pair order and writes it to its
// own LDS rows; each lane then reads its 16 A fragments (row l % 16, chunk l / 16)
// from there. Reading the fragments straight from X would touch 64 cache lines per
// load instead of 8.
// Loads are issued in the order the products consume them: the first tile's
// activation rows of item 0, the first weight-row fragment of item 0, its other
// fragments and those of the next QX_SKINNY_AHEAD - 1 items. When an item's rows are
// staged, the next staged rows (next item, else next tile) are requested, then the codes
// of the item QX_SKINNY_AHEAD ahead: a wave's loads return in order, so rows requested
// behind all of its codes would wait for every one of them.
// LDS: W * min(m, 16) rows of kXRow bytes and the W * RF tiles of 16 x 16 fp32 that are
// added in wave order, past the rows where LDS allows (then one barrier per activation
// tile orders the tiles' writes after the previous sums, and a wave stages and multiplies
// the next tile meanwhile), else over them after each tile.
template <int BITS, int KIND, int G, int RF, int J, int LB, int MT>
__global__ __launch_bounds__(LB) void gemm_skinny_kernel(const char* __restrict__ packed,
                                                         const uint16_t* __restrict__ X,
                                                         uint16_t* __restrict__ Y, int n, int k, int m,
                                                         int red_off) {
  extern __shared__ __align__(16) char lds[];
  __shared__ __align__(16) uint32_t q4lut[KIND == QX_Q4X ? 32 : 1];
  const int C = k >> 7, G_row = k / G, W = blockDim.x >> 6;
  const size_t meta_off = (size_t)n * k * BITS / 8;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int g = lane >> 4, li = lane & 15;
  const int n0 = blockIdx.x * 16 * RF;
  const DecodeConsts kc = decode_consts();
  const int mtiles = (m + 15) >> 4, rows0 = min(m, 16);
  char* xs = lds + (size_t)wave * rows0 * kXRow;  // this wave's activation rows (one 16-row tile)
  // W * RF tiles of 16 x 16: past the staged rows (red_off > 0) where LDS allows, else over them
  float* red = reinterpret_cast<float*>(lds + red_off);

  Item<BITS, KIND, G> it[J][RF];
  auto load_frag = [&](int j, int f) {  // rows and chunks clamped in bounds
    load_item<BITS, KIND, G, J == 1>(it[j][f], packed, meta_off, min(n0 + 16 * f + li, n - 1),
                                     min(4 * (wave + W * j) + g, C - 1), C, G_row);
  };
  u32x4 xv[16];
  auto load_x = [&](int j, int mt) {  // chunks past C clamped to the last (their weights are zero)
    const uint16_t* src = X + (size_t)16 * mt * k + (size_t)min(4 * (wave + W * j) + g, C - 1) * 128 + 8 * li;
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (16 * mt + r < m) xv[r] = *reinterpret_cast<const u32x4*>(src + (size_t)r * k);
  };
  load_x(0, 0);  // small and L2-resident: first, so that staging waits for it alone
  if (QX_SKINNY_PIN) __builtin_amdgcn_sched_barrier(0);
  load_frag(0, 0);
  if (QX_SKINNY_PIN) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int j = 0; j < (J < QX_SKINNY_AHEAD ? J : QX_SKINNY_AHEAD); ++j)
#pragma unroll
    for (int f = j == 0 ? 1 : 0; f < RF; ++f) load_frag(j, f);
  if (QX_SKINNY_PIN) __builtin_amdgcn_sched_barrier(0);
  if constexpr (KIND == QX_Q4X) {
    stage_q4x_lut(packed, n, k, q4lut);
    __syncthreads();
  }

  // activation tiles of 16 rows in turn (at most MT), every code decoded again for each
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    if (mt >= mtiles) break;
    const int rows = min(16, m - 16 * mt);
    f4_t acc[RF];
#pragma unroll
    for (int f = 0; f < RF; ++f) acc[f] = f4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < J; ++j) {
      if (4 * (wave + W * j) >= C) break;  // the wave's chunks of this item are all past C
      // stage the item's rows; the LDS instructions of one wave execute in order, so the
      // reads below see these writes and the writes see the previous item's reads done
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (r < rows)
          *reinterpret_cast<u32x4*>(xs + r * kXRow + 16 * lane) = __builtin_bit_cast(u32x4, x_frag<BITS>(xv[r]));
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      h8_t a[16];
      {
        const char* src = xs + min(li, rows - 1) * kXRow + 256 * g;
#pragma unroll
        for (int P = 0; P < 16; ++P) a[P] = *reinterpret_cast<const h8_t*>(src + 16 * P);
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      // the next staged rows: this tile's next item, else the next tile's first; then the
      // codes QX_SKINNY_AHEAD items ahead, so that each item's rows wait in the wave's
      // in-order returns only behind the codes of the items before it
      if (j + 1 < J && 4 * (wave + W * (j + 1)) < C) load_x(j + 1, mt);
      else if (mt + 1 < MT && mt + 1 < mtiles) load_x(0, mt + 1);
      if (mt == 0 && j + QX_SKINNY_AHEAD < J) {
        if (QX_SKINNY_PIN) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int f = 0; f < RF; ++f) load_frag(j + QX_SKINNY_AHEAD, f);
      }
      if (QX_SKINNY_PIN) __builtin_amdgcn_sched_barrier(0);
      const bool valid = 4 * (wave + W * j) + g < C;  // false only in the last item of a row
#pragma unroll
      for (int f = 0; f < RF; ++f) {
        const ItemTables<BITS, KIND, G> tb = item_tables<BITS, KIND, G>(it[j][f], q4lut, valid);
#define QX_SKINNY_PIECE(P) \
  acc[f] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[P], piece_frag<BITS, KIND, G, P>(it[j][f], tb, kc), acc[f], 0, 0, 0);
        QX_SKINNY_PIECE(0) QX_SKINNY_PIECE(1) QX_SKINNY_PIECE(2) QX_SKINNY_PIECE(3)
        QX_SKINNY_PIECE(4) QX_SKINNY_PIECE(5) QX_SKINNY_PIECE(6) QX_SKINNY_PIECE(7)
        QX_SKINNY_PIECE(8) QX_SKINNY_PIECE(9) QX_SKINNY_PIECE(10) QX_SKINNY_PIECE(11)
        QX_SKINNY_PIECE(12) QX_SKINNY_PIECE(13) QX_SKINNY_PIECE(14) QX_SKINNY_PIECE(15)
#undef QX_SKINNY_PIECE
      }
    }

    // wave tiles -> LDS: red[(w * RF + f) * 256 + 4 * lane + r] holds D[4 g + r][li]. Over
    // the staged rows every wave must be past its reads of them; past them only past the
    // previous tile's sums (so a wave stages and multiplies the next tile meanwhile)
    if (red_off == 0 || mt > 0) __syncthreads();
#pragma unroll
    for (int f = 0; f < RF; ++f) *reinterpret_cast<f4_t*>(red + (wave * RF + f) * 256 + 4 * lane) = acc[f];
    __syncthreads();
    // output (row 16 mt + r of Y, column c) = tile f = c / 16, element D[r][c % 16]:
    // lane 16 (r / 4) + c % 16, register r % 4; waves added in order
    for (int o = threadIdx.x; o < 256 * RF; o += blockDim.x) {
      const int c = o % (16 * RF), r = o / (16 * RF);
      const int f = c >> 4;
      const int idx = f * 256 + 4 * (16 * (r >> 2) + (c & 15)) + (r & 3);
      float s = 0.f;
      for (int w = 0; w < W; ++w) s += red[w * RF * 256 + idx];
      if (r < rows && n0 + c < n) Y[(size_t)(16 * mt + r) * n + n0 + c] = (uint16_t)float_to_half_bits(s);
    }
    if (red_off == 0 && mt + 1 < mtiles) __syncthreads();  // the sums are read before the next tile is staged
  }
}

template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
// f(0), f(1), .., f(N - 1) with compile-time arguments
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Products of one group of RF weight-row fragments with the A fragments held in
// registers: acc[f] = sum over the lane's 16 pieces.
template <int BITS, int KIND, int G, int RF>
__device__ __forceinline__ void mul_group(const Item<BITS, KIND, G> (&it)[RF], const h8_t (&a)[16],
                                          const uint32_t* q4lut, bool valid, const DecodeConsts& kc,
                                          f4_t (&acc)[RF]) {
#pragma unroll
  for (int f = 0; f < RF; ++f) {
    acc[f] = f4_t{0.f, 0.f, 0.f, 0.f};
    const ItemTables<BITS, KIND, G> tb = item_tables<BITS, KIND, G>(it[f], q4lut, valid);
#define QX_SKINNY_PIECE(P) \
  acc[f] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[P], piece_frag<BITS, KIND, G, P>(it[f], tb, kc), acc[f], 0, 0, 0);
    QX_SKINNY_PIECE(0) QX_SKINNY_PIECE(1) QX_SKINNY_PIECE(2) QX_SKINNY_PIECE(3)
    QX_SKINNY_PIECE(4) QX_SKINNY_PIECE(5) QX_SKINNY_PIECE(6) QX_SKINNY_PIECE(7)
    QX_SKINNY_PIECE(8) QX_SKINNY_PIECE(9) QX_SKINNY_PIECE(10) QX_SKINNY_PIECE(11)
    QX_SKINNY_PIECE(12) QX_SKINNY_PIECE(13) QX_SKINNY_PIECE(14) QX_SKINNY_PIECE(15)
#undef QX_SKINNY_PIECE
  }
}

// Pipelined form for rows of 29-32 chunks (one item per lane, all 8 waves busy) and
// m <= 16, on matrices of at least NB groups of 16 RF weight rows per compute unit: one
// block of 8 waves per compute unit stages the activations once and keeps each lane's 16
// A fragments in registers, then takes groups blockIdx.x, blockIdx.x + gridDim.x, ... in
// turn (the chip reads one band of rows at a time). Each wave keeps the codes of NB
// groups in flight: those of group s + NB are requested once group s is multiplied, so
// the decode and products of one group overlap the arrival of the next. The waves do not
// wait for each other: each writes its fp32 tile of group s to its own LDS slot, and
// after one barrier the block adds the slots in wave order and stores its rows. Rows of
// the last group past n repeat row n - 1; no load reaches past the block's last group.
template <int BITS, int KIND, int G, int RF, int NB>
__global__ __launch_bounds__(512) void gemm_skinny_loop_kernel(const char* __restrict__ packed,
                                                               const uint16_t* __restrict__ X,
                                                               uint16_t* __restrict__ Y, int n, int k, int m,
                                                               int slot_off, int slot_stride) {
  constexpr int W = 8;
  extern __shared__ __align__(16) char lds[];
  __shared__ __align__(16) uint32_t q4lut[KIND == QX_Q4X ? 32 : 1];
  const int C = k >> 7, G_row = k / G;
  const size_t meta_off = (size_t)n * k * BITS / 8;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int g = lane >> 4, li = lane & 15;
  const int rows = min(m, 16);
  const int groups = (n + 16 * RF - 1) / (16 * RF);
  const int steps = (groups - (int)blockIdx.x + (int)gridDim.x - 1) / (int)gridDim.x;  // groups of this block
  const int c = min(4 * wave + g, C - 1);
  const bool valid = 4 * wave + g < C;
  const DecodeConsts kc = decode_consts();

  Item<BITS, KIND, G> it[NB][RF];
  auto load_grp = [&](Item<BITS, KIND, G>(&dst)[RF], int s) {  // group blockIdx.x + s gridDim.x
    const int n0 = ((int)blockIdx.x + s * (int)gridDim.x) * 16 * RF;
#pragma unroll
    for (int f = 0; f < RF; ++f)
      load_item<BITS, KIND, G, true>(dst[f], packed, meta_off, min(n0 + 16 * f + li, n - 1), c, C, G_row);
  };
  u32x4 xv[16];
  {
    const uint16_t* src = X + (size_t)c * 128 + 8 * li;
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (r < rows) xv[r] = *reinterpret_cast<const u32x4*>(src + (size_t)r * k);
  }
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    load_grp(it[b], b);
    __builtin_amdgcn_sched_barrier(0);
  }
  if constexpr (KIND == QX_Q4X) stage_q4x_lut(packed, n, k, q4lut);

  h8_t a[16];
  {
    char* xs = lds + (size_t)wave * rows * kXRow;
#pragma unroll
    for (int r = 0; r < 16; ++r)
      if (r < rows) *reinterpret_cast<u32x4*>(xs + r * kXRow + 16 * lane) = __builtin_bit_cast(u32x4, x_frag<BITS>(xv[r]));
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const char* src = xs + min(li, rows - 1) * kXRow + 256 * g;
#pragma unroll
    for (int P = 0; P < 16; ++P) a[P] = *reinterpret_cast<const h8_t*>(src + 16 * P);
  }
  // Wave tiles of group s at lds + slot_off + wave * slot_stride + s * RF KB: past the
  // staged rows, where no wave waits for another before its products (one barrier
  // precedes the sums); or, where LDS is short (m near 16), over the wave's own staged
  // rows, which it has read (one wave's LDS instructions execute in order), after a
  // barrier that keeps the waves in step as they start (measured faster there).
  if (KIND == QX_Q4X || slot_off == 0) __syncthreads();  // (the Q4X tables are staged)
  float* const myslots = reinterpret_cast<float*>(lds + slot_off + (size_t)wave * slot_stride);
  auto product = [&](const Item<BITS, KIND, G>(&cur)[RF], int st) {
    f4_t acc[RF];
    mul_group<BITS, KIND, G, RF>(cur, a, q4lut, valid, kc, acc);
    float* rd = myslots + st * RF * 256;
#pragma unroll
    for (int f = 0; f < RF; ++f) *reinterpret_cast<f4_t*>(rd + f * 256 + 4 * lane) = acc[f];
  };
  // Full rounds: group s0 + b, then the load of group s0 + b + NB into its registers.
  // The rest (NB + e groups, 0 <= e < NB) runs as straight-line code for each e, so that
  // every wait before a group's products leaves the later groups' loads in flight and no
  // load reaches past the block's last group.
  int s0 = 0;
  for (; s0 + 2 * NB <= steps; s0 += NB) {
    static_for<NB>([&](auto b) {
      product(it[b], s0 + b);
      __builtin_amdgcn_sched_barrier(0);
      load_grp(it[b], s0 + b + NB);
      __builtin_amdgcn_sched_barrier(0);
    });
  }
  const int e = steps - s0 - NB;  // 0 <= e < NB (the launch gives every block NB groups or more)
  static_for<NB>([&](auto E) {
    if (e == E) {
      static_for<NB>([&](auto b) {
        product(it[b], s0 + b);
        if constexpr (b < E) {
          __builtin_amdgcn_sched_barrier(0);
          load_grp(it[b], s0 + b + NB);
          __builtin_amdgcn_sched_barrier(0);
        }
      });
      static_for<E>([&](auto b) { product(it[b], s0 + NB + b); });
    }
  });
  __syncthreads();
  // output (row r of Y, column n0 + cc of group s) = tile f = cc / 16, element D[r][cc % 16]:
  // lane 16 (r / 4) + cc % 16, register r % 4; waves added in order
  for (int o = threadIdx.x; o < steps * 256 * RF; o += 64 * W) {
    const int st = o / (256 * RF), oo = o % (256 * RF);
    const int cc = oo % (16 * RF), r = oo / (16 * RF);
    const int f = cc >> 4;
    const int idx = f * 256 + 4 * (16 * (r >> 2) + (cc & 15)) + (r & 3);
    float sum = 0.f;
#pragma unroll
    for (int w = 0; w < W; ++w)
      sum += reinterpret_cast<const float*>(lds + slot_off + (size_t)w * slot_stride)[st * RF * 256 + idx];
    const int n0 = ((int)blockIdx.x + st * (int)gridDim.x) * 16 * RF;
    if (r < rows && n0 + cc < n) Y[(size_t)r * n + n0 + cc] = (uint16_t)float_to_half_bits(sum);
  }
}

#ifndef QX_SKINNY_LOOP
#define QX_SKINNY_LOOP 1  // 0: the one-shot form only
#endif


// Compute units of the current device (cached per device).
inline int compute_units() {
  static std::atomic<int> cus[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int v = cus[dev].load(std::memory_order_relaxed);
  if (v == 0) {
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
    cus[dev].store(v, std::memory_order_relaxed);
  }
  return v;
}

// LDS of the pipelined form for m rows and `tiles` group tiles per wave: each wave's
// tiles past the 8 waves' staged rows where that fits, else over the wave's own staged
// rows; 0 if neither fits.
inline size_t loop_lds(int m, int tiles, int* slot_off, int* slot_stride) {
  const int rows_bytes = std::min(m, 16) * kXRow, slots_bytes = tiles * 1024;
  if (8 * (rows_bytes + slots_bytes) <= 160 * 1024) {
    *slot_off = 8 * rows_bytes; *slot_stride = slots_bytes;
    return (size_t)8 * (rows_bytes + slots_bytes);
  }
  if (slots_bytes <= rows_bytes) {
    *slot_off = 0; *slot_stride = rows_bytes;
    return (size_t)8 * rows_bytes;
  }
  return 0;
}

template <int BITS, int KIND, int G, int RF, int NB>
int launch_loop(const qx_desc* d, const char* p, int m, const uint16_t* X, uint16_t* Y, hipStream_t s) {
  const int groups = (d->n + 16 * RF - 1) / (16 * RF), blocks = compute_units();
  const int steps = (groups + blocks - 1) / blocks;
  if (groups / blocks < NB || m > 16 || d->k / 128 > 32) return QX_E_UNSUPPORTED;  // every block holds NB groups
  int slot_off, slot_stride;
  const size_t lds = loop_lds(m, steps * RF, &slot_off, &slot_stride);
  if (lds == 0) return QX_E_UNSUPPORTED;
  if (lds > 160 * 1024) return QX_E_UNSUPPORTED;
  hipLaunchKernelGGL((gemm_skinny_loop_kernel<BITS, KIND, G, RF, NB>), dim3((unsigned)blocks), dim3(512), lds, s, p, X, Y,
                     d->n, d->k, m, slot_off, slot_stride);
  return hipGetLastError() == hipSuccess ? QX_OK : QX_E_HIP;
}

template <int BITS, int KIND, int G, int RF, int J, int LB>
int launch_cfg(const qx_desc* d, const char* p, int m, const uint16_t* X, uint16_t* Y, hipStream_t s) {
  const int C = d->k / 128;
  const int W = (C + 4 * J - 1) / (4 * J);
  if (W > LB / 64 || m > 64) return QX_E_UNSUPPORTED;
  const size_t rows_bytes = (size_t)W * std::min(m, 16) * kXRow, red_bytes = (size_t)W * RF * 256 * sizeof(float);
  const bool sep = rows_bytes + red_bytes <= 160 * 1024;  // reduction tiles past the staged rows
  const size_t lds = sep ? rows_bytes + red_bytes : std::max(rows_bytes, red_bytes);
  const int red_off = sep ? (int)rows_bytes : 0;
  const unsigned blocks = (unsigned)((d->n + 16 * RF - 1) / (16 * RF));
  if (m <= 16)
    hipLaunchKernelGGL((gemm_skinny_kernel<BITS, KIND, G, RF, J, LB, 1>), dim3(blocks), dim3(64 * W), lds, s, p, X,
                       Y, d->n, d->k, m, red_off);
  else
    hipLaunchKernelGGL((gemm_skinny_kernel<BITS, KIND, G, RF, J, LB, 4>), dim3(blocks), dim3(64 * W), lds, s, p, X,
                       Y, d->n, d->k, m, red_off);
  return hipGetLastError() == hipSuccess ? QX_OK : QX_E_HIP;
}

#ifndef QX_SKINNY_RF
#define QX_SKINNY_RF 0  // 0: by shape; 1, 2, 3 force the weight-row fragments per wave
#endif
#ifndef QX_SKINNY_RF6_ROWS
#define QX_SKINNY_RF6_ROWS 16384  // rows from which one-item lanes take six weight-row fragments
#endif
#ifndef QX_SKINNY_LB
#define QX_SKINNY_LB 512  // threads per block at most (8 waves: up to 256 VGPRs per lane)
#endif

template <int BITS, int KIND, int G>
int launch_t(const qx_desc* d, const void* packed, int m, const uint16_t* X, uint16_t* Y, hipStream_t s) {
  const char* p = static_cast<const char*>(packed);
  constexpr int LB = QX_SKINNY_LB, WMAX = LB / 64;
  const int C = d->k / 128;
  const int J = (C + 4 * WMAX - 1) / (4 * WMAX);  // items per lane
  // tall matrices: three weight-row fragments per wave with one item per lane, two with
  // two (the registers of three spill in some formats), one beyond
  const bool six = d->n >= QX_SKINNY_RF6_ROWS && J == 1 && m <= 16 &&
                   !(KIND == QX_CODEBOOK && BITS == 4 && G <= 64);  // their tables spill at six
  const int rf = QX_SKINNY_RF ? QX_SKINNY_RF : six ? 6 : d->n >= 8192 ? (J == 1 ? 3 : J == 2 ? 2 : 1) : 1;
  if (m < 1 || m > QX_SKINNY_MAX_M) return QX_E_UNSUPPORTED;
  if (QX_SKINNY_LOOP && J == 1 && m <= 16 && C > 28) {
    // pipelined form where it holds fewer rows per compute unit than a block of the
    // one-shot form, or four groups or more (measured; see the kernel's comment)
    const int groups = (d->n + 15) / 16, cus = compute_units();
    const int steps = (groups + cus - 1) / cus;
    int so, ss;
    const bool q4x3 = KIND == QX_Q4X && m >= 3;  // Q4X at m >= 3 whenever every unit holds two groups
    if (groups / cus >= 2 && (q4x3 || steps < rf || steps >= 4) && loop_lds(m, steps, &so, &ss) > 0)
      return launch_loop<BITS, KIND, G, 1, 2>(d, p, m, X, Y, s);
  }
#define QX_SKINNY_J(JJ)                                                                                   \
  case JJ:                                                                                                \
    return rf >= 6 && JJ == 1 ? launch_cfg<BITS, KIND, G, 6, 1, LB>(d, p, m, X, Y, s)                \
           : rf >= 3 ? launch_cfg<BITS, KIND, G, (JJ <= 2 ? 3 : 4 - JJ / 2), JJ, LB>(d, p, m, X, Y, s)   \
           : rf == 2 ? launch_cfg<BITS, KIND, G, (JJ <= 3 ? 2 : 1), JJ, LB>(d, p, m, X, Y, s)             \
                     : launch_cfg<BITS, KIND, G, 1, JJ, LB>(d, p, m, X, Y, s);
  switch (J) {
    QX_SKINNY_J(1) QX_SKINNY_J(2) QX_SKINNY_J(3) QX_SKINNY_J(4)
    default: return QX_E_UNSUPPORTED;
  }
#undef QX_SKINNY_J
}

}  // namespace

// Whether qx_gemm runs m rows on this kernel. Beyond 16 rows (several activation tiles,
// every code decoded again per tile) only rows of at most 32 chunks with one round of
// blocks (us at m = 24 / 32 / 48 / 64 against the matrix-core GEMM, weights rotated over
// four copies: 11008x4096 uniform-3 g64 16.8 / 17.5 / 23.7 / 29.4 vs 21.6 / 21.5 / 27.5 /
// 27.8; 12288x4096 codebook-3 15.0 / 15.8 / 20.6 / 25.5 vs 19.9 / 19.9 / 25.0 / 25.1;
// 4096x4096 codebook-3 8.9 / 9.1 / 11.5 / 14.0 vs 14.8 / 14.9 / 15.3 / 15.5; 22016 rows,
// two rounds: 28.5 / 30.2 / 40.2 / 49.7 vs 24.5 / 24.9 / 40.1 / 41.4; at m = 64 the tall
// matrices' GEMM gains came from the last-level cache: with the c5 MLP's weights streamed
// from HBM, 87.2 us per gate + up + down against 89.7 with them on the GEMM). Up to 16 rows: measured against the
// small-batch GEMV-style kernel (m <= 4) and the matrix-core GEMM in all thirteen formats
// (us, 3-bit uniform g64 at m = 2 / 8 / 16: 11008x4096 8.4 / 9.0 / 9.9 against 9.2 / 15.7 /
// 15.8; 4096x4096 4.9 / 5.5 / 6.2 against 5.5 / 8.7 / 8.7). Rows of more than 32 chunks
// (two to four items per lane, the next item's codes requested as each item is staged),
// at m = 2 / 3 / 4 / 5 / 8 / 16: 4096x11008 uniform-3 g64 9.1 at m = 2 against 10.9 for the
// GEMV-style kernel, 5120x13824 18.3 against 16.2 (uniform codes at m = 2 on four items
// stay there); 4-bit codebooks of 128 codes faster at every m (4096x11008 12.4 / 12.8 /
// 12.9 / 13.2 / 13.8 / 15.8 against 13.7 / 18.0 / 18.4 / 17.1 / 17.3 / 19.4; 5120x13824
// 24.2 / .. / 34.1 against 24.5 / .. / 40.9), of 64 codes on two items up to m = 5 and on
// three up to m = 3 (4096x8192 12.3 / 13.9 / 15.1 / 16.6 / 22.2 against 15.2 / 16.8 / 17.1
// / 19.5 / 19.6); Q4X on two items up to m = 8 (4096x8192 9.8 / 10.0 / 10.1 / 11.8 / 15.2
// against 10.1 / 12.0 / 12.4 / 17.6 / 17.5) and on three at m = 3, 4 (14.1 / 15.8 against
// 16.2 / 16.5); 4-bit codebooks of 32 codes nowhere (their tables spill registers).
bool gemm_skinny_applies(const qx_desc* d, int m) {
  const int C = d->k / 128, J = (C + 31) / 32;  // items per lane (8 waves of 4 chunks)
#ifdef QX_SKINNY_FORCE
  return m >= 2 && m <= QX_SKINNY_MAX_M && J <= 4;
#endif
  if (m < 2 || m > QX_SKINNY_MAX_M || J > 4) return false;
  const bool cb = d->kind == QX_CODEBOOK, q4x = d->kind == QX_Q4X;
  if (m > 16) {  // 16-row activation tiles in turn, every code decoded again for each
    const int rf = d->n >= 8192 ? 3 : 1;
    return J == 1 && (d->n + 16 * rf - 1) / (16 * rf) <= 256 && !q4x && !(cb && d->bits == 4 && d->group <= 64);
  }
  if (cb && d->bits == 4) {
    if (d->group == 128) return true;
    if (d->group == 64) return J == 1 || (J == 2 && m <= 5) || (J == 3 && m <= 3);
    return false;
  }
  if (q4x) return J == 1 ? (m >= 3 || d->n <= 4096) : J == 2 ? m <= 8 : J == 3 && m >= 3 && m <= 4;
  if (J == 4 && m == 2) return cb;  // uniform codes at m = 2 on rows of 97-128 chunks: GEMV-style
  return true;
}

int launch_gemm_skinny(const qx_desc* d, const void* packed, int m, const uint16_t* X, uint16_t* Y,
                       hipStream_t s) {
#define QX_SKINNY_CASE(B, K, G) \
  if (d->bits == B && d->kind == K && d->group == G) return launch_t<B, K, G>(d, packed, m, X, Y, s);
  QX_SKINNY_CASE(3, 0, 32) QX_SKINNY_CASE(3, 0, 64) QX_SKINNY_CASE(3, 0, 128)
  QX_SKINNY_CASE(3, 1, 32) QX_SKINNY_CASE(3, 1, 64) QX_SKINNY_CASE(3, 1, 128)
  QX_SKINNY_CASE(4, 0, 32) QX_SKINNY_CASE(4, 0, 64) QX_SKINNY_CASE(4, 0, 128)
  QX_SKINNY_CASE(4, 1, 32) QX_SKINNY_CASE(4, 1, 64) QX_SKINNY_CASE(4, 1, 128)
  QX_SKINNY_CASE(4, 2, 64)
#undef QX_SKINNY_CASE
  return QX_E_UNSUPPORTED;
}

}  // namespace qx
