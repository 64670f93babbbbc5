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
//   * codes are decoded in registers (qx_device.h), one or two VALU instructions
//     per code pair, and multiplied with v_dot2_f32_f16 (exact fp16 products, fp32
//     sums); uniform codes enter as subnormal integers (the masked field
//     alone) and the zero point is folded out once per group with the sum of
//     x formed while x is staged, so no instruction per pair subtracts it;
//     groups are scaled once;
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
#include "gemv_common.h"

#include <algorithm>

namespace qx {
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
  __shared__ float gs[KIND == QX_UNIFORM ? C * (128 / G) : 1];
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
  float* no_gs = nullptr;  // codebook groups need no sums over x
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


// 4-bit codebook with groups of 32, k = 128*C with C in {32, 64}: a chunk's 16-byte
// code slice s is group s, and each group brings a 32-byte table, so a whole chunk is
// 192 bytes -- too many registers for one lane. Here lane 4c + s of a row takes chunk c,
// group s (16 bytes of codes, 32 of table, 16 of its x per code dword); a row spans 4C
// lanes (2 or 4 waves), summed per wave with DPP and across its waves through LDS in a
// fixed order.
template <int C>
__global__ __launch_bounds__(256) void gemv_cb4g32_kernel(const char* __restrict__ packed,
                                                          const uint16_t* __restrict__ x,
                                                          uint16_t* __restrict__ y, int n) {
  constexpr int NT = 256, L = 4 * C, RPB = NT / L, WPR = L / 64, XP = (C * 16 + NT - 1) / NT;
  static_assert(RPB >= 1 && NT % L == 0, "whole rows per block");
  __shared__ __align__(16) char xs[C * kXBlock];
  __shared__ float red[NT / 64];
  const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
  const int idx = t % L, c = idx >> 2, s = idx & 3;
  const int r = min((int)blockIdx.x * RPB + t / L, n - 1);
  const size_t meta_off = (size_t)n * C * 64;  // n * k * 4 / 8

  u32x4 xr[XP];
  load_x<XP>(x, 0, C, xr, NT);
  const u32x4 D4 = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(packed) + (((size_t)r * 4 + s) * C + c));
  const u32x4* tp = reinterpret_cast<const u32x4*>(packed + meta_off + ((size_t)r * 4 * C + 4 * c + s) * 32);
  const u32x4 t0 = __builtin_nontemporal_load(tp), t1 = __builtin_nontemporal_load(tp + 1);
  store_x<4, QX_CODEBOOK, 32, XP, C * 16 % NT == 0>(xr, C, xs, nullptr, NT);
  __syncthreads();

  const uint32_t m[8] = {t0.x, t0.y, t0.z, t0.w, t1.x, t1.y, t1.z, t1.w};
  const LutGroup<4> tab = lut_group<4>(m);
  const u32x4* xv = reinterpret_cast<const u32x4*>(xs + c * kXBlock) + 4 * s;
  const uint32_t Dw[4] = {D4.x, D4.y, D4.z, D4.w};
  float acc = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {  // code dword 4s + j of the chunk: codes 8j..8j+7 of the group
    const u32x4 xj = xv[j];
    uint32_t elo, ehi, olo, ohi;
    lut4_bytes(tab, Dw[j] & 0x0F0F0F0Fu, elo, ehi);         // codes 0 2 4 6
    lut4_bytes(tab, (Dw[j] >> 4) & 0x0F0F0F0Fu, olo, ohi);  // codes 1 3 5 7
    acc = dot2(perm(ehi, elo, 0x06020400u), xj.x, acc);     // (0, 4)
    acc = dot2(perm(ohi, olo, 0x06020400u), xj.y, acc);     // (1, 5)
    acc = dot2(perm(ehi, elo, 0x07030501u), xj.z, acc);     // (2, 6)
    acc = dot2(perm(ohi, olo, 0x07030501u), xj.w, acc);     // (3, 7)
  }
  const float v = wave_sum(acc);
  if (lane == 63) red[wave] = v;
  __syncthreads();
  const int row = (int)blockIdx.x * RPB + t;
  if (t < RPB && row < n) {
    float sum = 0.f;
    for (int w = 0; w < WPR; ++w) sum += red[t * WPR + w];
    y[row] = (uint16_t)float_to_half_bits(sum);
  }
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
  float* gs = reinterpret_cast<float*>(smem + row_lds_gsum_offset(C, R * C));  // C * 128/G
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
  float* gs = reinterpret_cast<float*>(smem + row_lds_gsum_offset(CT, R * CT));  // CT * 128/G
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
  const size_t lds = (size_t)row_lds_gsum_offset(CT, R * CT) + (size_t)CT * (128 / G) * sizeof(float);
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
  if (BITS == 4 && KIND == QX_CODEBOOK && G == 32 && (C == 32 || C == 64)) {
    // one group per lane (11008x4096: 14.1 us against 30.8 with a chunk per lane)
    if (C == 32)
      hipLaunchKernelGGL((gemv_cb4g32_kernel<32>), dim3((unsigned)((d->n + 1) / 2)), dim3(256), 0, s, p, x, y, d->n);
    else
      hipLaunchKernelGGL((gemv_cb4g32_kernel<64>), dim3((unsigned)d->n), dim3(256), 0, s, p, x, y, d->n);
  } else if (C == 32 || C == 64) {
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
    gemv_row_shape(d->n, C, KIND == QX_CODEBOOK && BITS == 4 && G == 32, &R, &threads);
    const unsigned blocks = (unsigned)((d->n + R - 1) / R);
    const size_t lds = (size_t)row_lds_gsum_offset(C, R * C) + (size_t)C * (128 / G) * sizeof(float);
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
