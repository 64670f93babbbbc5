// Small-batch decode: Y = X W'^T for 2 to 4 activation rows, GEMV-style. Every
// code is decoded once per lane (as in the batch-1 GEMV) and its weight pairs are
// multiplied with each of the m activation vectors staged in LDS, so the decode
// work is shared by the batch and the matrix is still streamed once, where the
// matrix-core GEMM would multiply 16-row activation tiles that are mostly padding
// (gemv_multi_applies picks between the two per shape and format, from
// measurements). A block takes R rows and walks the reduction axis in segments of
// S 128-code chunks (one item per lane and segment), so the LDS it needs does not
// grow with k; lane totals go through LDS and one wave per (row, vector) adds them
// in a fixed order.
#include "gemv_common.h"

#include <algorithm>

namespace qx {
namespace {

// Calls emit(accumulator slot, fp16 weight pair, x dword index within the chunk's
// staged x block) for the 64 pairs of one item, in the decoders' pair order. Table
// formats: slot = group within the chunk. Uniform codes: binary16 subnormals (the
// masked field alone; the caller folds the zero point per group), slot = group *
// RawFields<BITS>::kN + field kind, each kind with its own power-of-two unit.
template <int BITS, int KIND, int G, typename F>
__device__ __forceinline__ void for_each_pair(const Item<BITS, KIND, G>& it, const DecodeConsts& k,
                                              const uint32_t* q4lut, F&& emit) {
  constexpr int NG = 128 / G;
  if constexpr (KIND == QX_Q4X) {  // two groups of 64: the selected sub-codebook's tables
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      const uint32_t* tp = q4lut + 8 * ((it.m[1] >> (2 * g)) & 3u);
      const u32x4 tl = *reinterpret_cast<const u32x4*>(tp), th = *reinterpret_cast<const u32x4*>(tp + 4);
      const LutGroup<4> t = {{tl.x, tl.y, tl.z, tl.w}, {th.x, th.y, th.z, th.w}};
#pragma unroll
      for (int j = 8 * g; j < 8 * g + 8; ++j) {
        const uint32_t D = it.d[j];
        uint32_t elo, ehi, olo, ohi;
        lut4_bytes(t, D & 0x0F0F0F0Fu, elo, ehi);
        lut4_bytes(t, (D >> 4) & 0x0F0F0F0Fu, olo, ohi);
        emit(g, perm(ehi, elo, 0x06020400u), 4 * j);
        emit(g, perm(ohi, olo, 0x06020400u), 4 * j + 1);
        emit(g, perm(ehi, elo, 0x07030501u), 4 * j + 2);
        emit(g, perm(ohi, olo, 0x07030501u), 4 * j + 3);
      }
    }
  } else if constexpr (BITS == 4 && KIND == QX_UNIFORM) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int g = (8 * j) / G;
      const uint32_t D = it.d[j], Ds = D >> 8;
      emit(2 * g, D & k.m000f, 4 * j);           // (0, 4)
      emit(2 * g + 1, D & k.m00f0, 4 * j + 1);   // (1, 5)
      emit(2 * g, Ds & k.m000f, 4 * j + 2);      // (2, 6)
      emit(2 * g + 1, Ds & k.m00f0, 4 * j + 3);  // (3, 7)
    }
  } else if constexpr (BITS == 4 && KIND == QX_CODEBOOK) {
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const LutGroup<4> t = lut_group<4>(&it.m[g * 8]);
#pragma unroll
      for (int j = g * G / 8; j < (g + 1) * G / 8; ++j) {
        const uint32_t D = it.d[j];
        uint32_t elo, ehi, olo, ohi;
        lut4_bytes(t, D & 0x0F0F0F0Fu, elo, ehi);
        lut4_bytes(t, (D >> 4) & 0x0F0F0F0Fu, olo, ohi);
        emit(g, perm(ehi, elo, 0x06020400u), 4 * j);
        emit(g, perm(ohi, olo, 0x06020400u), 4 * j + 1);
        emit(g, perm(ehi, elo, 0x07030501u), 4 * j + 2);
        emit(g, perm(ohi, olo, 0x07030501u), 4 * j + 3);
      }
    }
  } else if constexpr (BITS == 3 && KIND == QX_UNIFORM) {
#pragma unroll
    for (int i = 0; i < 12; ++i) {
      const U3Pairs p = u3_raw(it.d[i], k);
      const int ga = (4 * i) / G, gb = (48 + 4 * i) / G;
      emit(3 * ga, p.a0, 2 * i);
      emit(3 * ga, p.a1, 2 * i + 1);
      emit(3 * gb + 1, p.b0, 2 * (12 + i));
      emit(3 * gb + 1, p.b1, 2 * (12 + i) + 1);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      uint32_t s0, s1;
      switch (i) {
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
      emit(3 * gg + 2, s0, 2 * (24 + i));
      emit(3 * gg + 2, s1, 2 * (24 + i) + 1);
    }
  } else {  // BITS == 3, codebook
    LutGroup<3> t[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) t[g] = lut_group<3>(&it.m[g * 4]);
#pragma unroll
    for (int i = 0; i < 12; ++i) {
      const uint32_t D = it.d[i];
      const int ga = (4 * i) / G, gb = (48 + 4 * i) / G;
      uint32_t p02, p13;
      lut3_pairs(t[ga], u3_sel_a(D), p02, p13);
      emit(ga, p02, 2 * i);
      emit(ga, p13, 2 * i + 1);
      lut3_pairs(t[gb], u3_sel_b(D), p02, p13);
      emit(gb, p02, 2 * (12 + i));
      emit(gb, p13, 2 * (12 + i) + 1);
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
      emit(gs, p02, 2 * (24 + i));
      emit(gs, p13, 2 * (24 + i) + 1);
    }
  }
}

// M activation vectors (m <= M; vectors past m repeat vector m - 1 and are not
// stored). A block owns R rows and walks k in segments of S chunks: lane (r, c)
// takes chunk c of each segment of row r. Per segment the codes are loaded, the M
// x blocks of its chunks are staged in LDS, then every lane multiplies. LDS: M
// staged segments (S chunks each), then R*S*M lane totals, then M*S*(128/G) group
// sums of x (uniform). (Loading the next segment before multiplying the current
// one costs registers and measured no faster.)
template <int BITS, int KIND, int G, int M>
__global__ __launch_bounds__(512) void gemv_multi_kernel(const char* __restrict__ packed,
                                                          const uint16_t* __restrict__ X,
                                                          uint16_t* __restrict__ Y, int n, int k,
                                                          int m, int R, int S) {
  extern __shared__ __align__(16) char smem[];
  __shared__ __align__(16) uint32_t q4lut[KIND == QX_Q4X ? 32 : 1];
  constexpr int NG = 128 / G;
  const int C = k >> 7, G_row = k / G, nthreads = blockDim.x;
  const size_t meta_off = (size_t)n * k * BITS / 8;
  const int row0 = blockIdx.x * R;
  const int rows = min(R, n - row0);
  const int xbytes = S * kXBlock;
  float* part = reinterpret_cast<float*>(smem + M * xbytes);       // [M][R*S]
  float* gs = part + M * R * S;                                    // [M][S*NG] (uniform)
  const DecodeConsts kc = decode_consts();
  const int t = threadIdx.x, r = t / S, c = t - r * S;
  const int row = row0 + min(r, rows - 1);
  const int nseg = (C + S - 1) / S;

  // every thread holds at most one 16-byte x piece per vector and segment: the
  // launcher makes blockDim.x >= 16*S
  u32x4 xr[M];
  Item<BITS, KIND, G> it;
  auto load_segment = [&](int seg) {
    const int cs = min(S, C - seg * S);
#pragma unroll
    for (int v = 0; v < M; ++v) {
      const u32x4* src = reinterpret_cast<const u32x4*>(X + (size_t)min(v, m - 1) * k) + seg * S * 16;
      xr[v] = src[min(t, cs * 16 - 1)];
    }
    load_item<BITS, KIND, G>(it, packed, meta_off, row, seg * S + min(c, cs - 1), C, G_row);
  };
  if constexpr (KIND == QX_Q4X) stage_q4x_lut(packed, n, k, q4lut);  // read after the first barrier
  float tot[M];
#pragma unroll
  for (int v = 0; v < M; ++v) tot[v] = 0.f;
  const char* xb = smem + c * kXBlock;
  for (int seg = 0; seg < nseg; ++seg) {
    const int cs = min(S, C - seg * S);
    load_segment(seg);
    if (seg > 0) __syncthreads();  // the previous segment is no longer read
    u32x4 one[1];
#pragma unroll
    for (int v = 0; v < M; ++v) {
      one[0] = xr[v];
      store_x<BITS, KIND, G, 1>(one, cs, smem + v * xbytes, gs + v * S * NG, nthreads);
    }
    const Item<BITS, KIND, G>& cur = it;
    __syncthreads();

    // one accumulator per slot and vector (for_each_pair)
    constexpr int NF = KIND == QX_UNIFORM ? RawFields<BITS>::kN : 1;
    float acc[M][NG * NF];
#pragma unroll
    for (int v = 0; v < M; ++v)
#pragma unroll
      for (int g = 0; g < NG * NF; ++g) acc[v][g] = 0.f;
    for_each_pair<BITS, KIND, G>(cur, kc, q4lut, [&](int slot, uint32_t pair, int xdw) {
#pragma unroll
      for (int v = 0; v < M; ++v) {
        const uint32_t xv = reinterpret_cast<const uint32_t*>(xb + v * xbytes)[xdw];
        acc[v][slot] = dot2(pair, xv, acc[v][slot]);
      }
    });
    if (c < cs) {
#pragma unroll
      for (int v = 0; v < M; ++v) {
#pragma unroll
        for (int g = 0; g < NG; ++g) {
          if constexpr (KIND == QX_UNIFORM)
            tot[v] += fold_group(cur.m[g], raw_group_sum<BITS>(&acc[v][g * NF]), gs[v * S * NG + c * NG + g]);
          else if constexpr (KIND == QX_Q4X) tot[v] += half_bits_to_float((cur.m[0] >> (16 * g)) & 0xFFFFu) * acc[v][g];
          else tot[v] += acc[v][g];
        }
      }
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
    if (lane == 63) Y[(size_t)v * n + row0 + rr] = (uint16_t)float_to_half_bits(s);
  }
}

// Segment width S = min(C, 32) chunks; R rows per block such that R*S lanes fill
// blocks of at least 512 threads best (R = 16 when S = 32). Then every thread holds
// at most one 16-byte piece of each x segment (16*S <= blockDim.x).
void multi_shape(int C, int* R, int* S, int* threads) {
  const int s = std::min(C, 32);
  const int r_max = std::min(256, 512 / s);
  int best_r = r_max;
  double best_u = -1.0;
  for (int r = 1; r <= r_max; ++r) {
    const int th = 64 * ((r * s + 63) / 64);
    if (th < 512 && r < r_max) continue;
    const double u = (double)(r * s) / th;
    if (u > best_u + 1e-9) { best_u = u; best_r = r; }
  }
  *R = best_r;
  *S = s;
  *threads = 64 * ((best_r * s + 63) / 64);
}

template <int BITS, int KIND, int G, int M>
int launch_multi_m(const qx_desc* d, const char* p, int m, const uint16_t* X, uint16_t* Y, hipStream_t s) {
  const int C = d->k / 128;
  int R, S, threads;
  multi_shape(C, &R, &S, &threads);
  if (threads < 16 * S || threads > 512) return QX_E_UNSUPPORTED;  // never with the shapes above
  const size_t lds = (size_t)M * S * kXBlock + (size_t)M * R * S * sizeof(float) +
                     (KIND == QX_UNIFORM ? (size_t)M * S * (128 / G) * sizeof(float) : 0);
  const dim3 grid((unsigned)((d->n + R - 1) / R)), block(threads);
  hipLaunchKernelGGL((gemv_multi_kernel<BITS, KIND, G, M>), grid, block, lds, s, p, X, Y, d->n, d->k, m, R, S);
  return hipGetLastError() == hipSuccess ? QX_OK : QX_E_HIP;
}

template <int BITS, int KIND, int G>
int launch_multi_t(const qx_desc* d, const void* packed, int m, const uint16_t* X, uint16_t* Y, hipStream_t s) {
  const char* p = static_cast<const char*>(packed);
  if (m <= 2) return launch_multi_m<BITS, KIND, G, 2>(d, p, m, X, Y, s);
  return launch_multi_m<BITS, KIND, G, 4>(d, p, m, X, Y, s);
}

}  // namespace

// Whether a product of m <= 4 rows runs GEMV-style (m = 1: the batch-1 GEMV, else
// the kernel above) rather than on the matrix-core GEMM. Measured on 11008 x 4096
// and 4096 x 11008 matrices in all twelve formats: the GEMV-style kernels win at
// m = 1 and m = 2 and, when k > n, up to m = 4 (the GEMM then has few row tiles,
// each with a long k loop); at m = 3, 4 with k <= n the GEMM is as fast or faster.
// 4-bit codebooks of 32-code groups (a 32-byte table per 32 codes) decode faster
// into matrix-core fragments at every m, except one row of 32 or 64 chunks, where the
// group-per-lane GEMV is faster (11008x4096: 14.2 against 19.7 us); at m = 2 so do
// 4-bit 64-code groups when
// k <= n. Q4X (whose 16-entry lookups make the GEMM decode-bound) runs GEMV-style
// for every m <= 4.
bool gemv_multi_applies(const qx_desc* d, int m) {
  if (d->kind == QX_Q4X) return m >= 1 && m <= QX_MULTI_MAX_M;
  if (m < 1 || m > QX_MULTI_MAX_M) return false;
  const bool cb4 = d->kind == QX_CODEBOOK && d->bits == 4;
  if (cb4 && d->group == 32)  // one row of 32 or 64 chunks: the group-per-lane GEMV
    return m == 1 && (d->k == 32 * 128 || d->k == 64 * 128);
  if (m == 1 || d->k > d->n) return true;
  return m == 2 && !(cb4 && d->group == 64);
}

int launch_gemv_multi(const qx_desc* d, const void* packed, int m, const uint16_t* X, uint16_t* Y,
                      hipStream_t s) {
#define QX_MULTI_CASE(B, K, G) \
  if (d->bits == B && d->kind == K && d->group == G) return launch_multi_t<B, K, G>(d, packed, m, X, Y, s);
  QX_MULTI_CASE(3, 0, 32) QX_MULTI_CASE(3, 0, 64) QX_MULTI_CASE(3, 0, 128)
  QX_MULTI_CASE(3, 1, 32) QX_MULTI_CASE(3, 1, 64) QX_MULTI_CASE(3, 1, 128)
  QX_MULTI_CASE(4, 0, 32) QX_MULTI_CASE(4, 0, 64) QX_MULTI_CASE(4, 0, 128)
  QX_MULTI_CASE(4, 1, 32) QX_MULTI_CASE(4, 1, 64) QX_MULTI_CASE(4, 1, 128)
  QX_MULTI_CASE(4, 2, 64)
#undef QX_MULTI_CASE
  return QX_E_UNSUPPORTED;
}

}  // namespace qx
