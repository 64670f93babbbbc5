// C-ABI front end of libqx: descriptor and argument validation, the host
// packer of the packed layout, and dispatch to the kernel launchers.
#include <cmath>
#include <cstring>
#include <thread>
#include <vector>

#include "qx_internal.h"

namespace {

constexpr int kMaxK = 1 << 20;

// Well-formed: the fields make sense. Supported: a kernel instance exists.
int check_desc(const qx_desc* d) {
  if (d == nullptr) return QX_E_ARG;
  if (d->flags != 0 || d->n < 0 || d->k <= 0 || d->k % 128 != 0 || d->k > kMaxK) return QX_E_ARG;
  if (d->kind != QX_UNIFORM && d->kind != QX_CODEBOOK && d->kind != QX_Q4X) return QX_E_ARG;
  if (d->kind == QX_Q4X && (d->bits != 4 || d->group != 64)) return QX_E_ARG;  // fixed by the format
  if (d->bits < 1 || d->bits > 8 || d->group <= 0 || d->k % d->group != 0) return QX_E_ARG;
  if (d->bits != 3 && d->bits != 4) return QX_E_UNSUPPORTED;
  if (d->group != 32 && d->group != 64 && d->group != 128) return QX_E_UNSUPPORTED;
  return QX_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned2(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 1u) == 0; }

size_t meta_bytes_per_group(const qx_desc* d) {
  return d->kind == QX_UNIFORM ? 4 : 2u * (1u << d->bits);
}

size_t packed_bytes(const qx_desc* d) {
  if (d->kind == QX_Q4X) return qx::q4x_offsets(d->n, d->k).total;
  const size_t n = (size_t)d->n, k = (size_t)d->k;
  return n * k * d->bits / 8 + n * (k / d->group) * meta_bytes_per_group(d);
}

// binary16 helpers for validation only
bool half_finite(uint16_t h) { return ((h >> 10) & 31) != 31; }
double half_value(uint16_t h) {
  const int s = h >> 15, e = (h >> 10) & 31, f = h & 1023;
  const double v = e == 0 ? std::ldexp((double)f, -24) : std::ldexp((double)(f | 1024), e - 25);
  return s ? -v : v;
}

// One chunk (128 codes of one row) into its 16*b bytes, per the layout in qx.h.
void pack_chunk(const uint8_t* q, int bits, uint8_t* out) {
  if (bits == 4) {
    for (int j = 0; j < 64; ++j) out[j] = (uint8_t)(q[2 * j] | (q[2 * j + 1] << 4));
    return;
  }
  for (int j = 0; j < 48; ++j) out[j] = (uint8_t)(q[j] | (q[48 + j] << 3));
  for (int m = 0; m < 32; ++m) {
    const uint8_t v = q[96 + m];
    out[m] |= (uint8_t)((v & 3) << 6);
    out[32 + m % 16] |= (uint8_t)(((v >> 2) & 1) << (6 + m / 16));
  }
}

void pack_rows(const qx_desc* d, const uint8_t* codes, int r0, int r1, uint8_t* blob) {
  const int b = d->bits, C = d->k / 128;
  uint8_t chunk[64];
  for (int r = r0; r < r1; ++r) {
    for (int c = 0; c < C; ++c) {
      pack_chunk(codes + (size_t)r * d->k + (size_t)c * 128, b, chunk);
      for (int s = 0; s < b; ++s)
        std::memcpy(blob + (((size_t)r * b + s) * C + c) * 16, chunk + 16 * s, 16);
    }
  }
}

}  // namespace

extern "C" {

const char* qx_status_str(int st) {
  switch (st) {
    case QX_OK: return "ok";
    case QX_E_ARG: return "invalid argument";
    case QX_E_UNSUPPORTED: return "unsupported configuration";
    case QX_E_SIZE: return "output buffer too small";
    case QX_E_HIP: return "HIP launch error";
    default: return "unknown status";
  }
}

int qx_pack_layout(const qx_desc* d, const uint8_t* codes, const uint16_t* scales,
                   const uint16_t* zeros, const uint16_t* codebook, void* packed, size_t cap,
                   size_t* packed_size) {
  const int st = check_desc(d);
  if (st != QX_OK) return st;
  if (packed_size == nullptr || d->kind == QX_Q4X) return QX_E_ARG;
  const size_t total = packed_bytes(d);
  *packed_size = total;
  if (packed == nullptr) return QX_OK;
  if (cap < total) return QX_E_SIZE;
  const size_t n = (size_t)d->n, k = (size_t)d->k, G = k / d->group;
  if (n == 0) return QX_OK;
  if (codes == nullptr) return QX_E_ARG;
  if (d->kind == QX_UNIFORM && (scales == nullptr || zeros == nullptr)) return QX_E_ARG;
  if (d->kind == QX_CODEBOOK && codebook == nullptr) return QX_E_ARG;
  const uint8_t qmax = (uint8_t)((1u << d->bits) - 1);
  for (size_t i = 0; i < n * k; ++i)
    if (codes[i] > qmax) return QX_E_ARG;
  if (d->kind == QX_UNIFORM) {
    for (size_t i = 0; i < n * G; ++i) {
      if (!half_finite(scales[i]) || !half_finite(zeros[i])) return QX_E_ARG;
      const double z = half_value(zeros[i]);
      if (z != std::floor(z) || z < 0 || z > qmax) return QX_E_ARG;
    }
  }
  uint8_t* blob = static_cast<uint8_t*>(packed);
  // codes region, rows split across host threads
  const unsigned hw = std::thread::hardware_concurrency();
  const int nt = (int)std::max(1u, std::min(hw == 0 ? 1u : hw, (unsigned)((n + 255) / 256)));
  if (nt <= 1) {
    pack_rows(d, codes, 0, d->n, blob);
  } else {
    std::vector<std::thread> th;
    for (int t = 0; t < nt; ++t) {
      const int r0 = (int)(n * t / nt), r1 = (int)(n * (t + 1) / nt);
      th.emplace_back(pack_rows, d, codes, r0, r1, blob);
    }
    for (auto& x : th) x.join();
  }
  // metadata region
  uint8_t* meta = blob + n * k * d->bits / 8;
  if (d->kind == QX_UNIFORM) {
    for (size_t i = 0; i < n * G; ++i) {
      const uint32_t w = (uint32_t)scales[i] | ((uint32_t)zeros[i] << 16);
      meta[4 * i + 0] = (uint8_t)w;
      meta[4 * i + 1] = (uint8_t)(w >> 8);
      meta[4 * i + 2] = (uint8_t)(w >> 16);
      meta[4 * i + 3] = (uint8_t)(w >> 24);
    }
  } else {
    const size_t E = (size_t)1 << d->bits;
    for (size_t i = 0; i < n * G * E; ++i) {
      meta[2 * i] = (uint8_t)codebook[i];
      meta[2 * i + 1] = (uint8_t)(codebook[i] >> 8);
    }
  }
  return QX_OK;
}

int qx_pack_q4x(const qx_desc* d, const uint8_t* codes, const uint16_t* scales,
                const uint8_t* selectors, const uint16_t* codebook, void* packed, size_t cap,
                size_t* packed_size) {
  const int st = check_desc(d);
  if (st != QX_OK) return st;
  if (packed_size == nullptr || d->kind != QX_Q4X) return QX_E_ARG;
  const qx::Q4xOffsets L = qx::q4x_offsets(d->n, d->k);
  *packed_size = L.total;
  if (packed == nullptr) return QX_OK;
  if (cap < L.total) return QX_E_SIZE;
  const size_t n = (size_t)d->n, k = (size_t)d->k, G = (size_t)L.groups;
  if (codebook == nullptr) return QX_E_ARG;
  if (n > 0 && (codes == nullptr || scales == nullptr || selectors == nullptr)) return QX_E_ARG;
  for (size_t i = 0; i < n * k; ++i)
    if (codes[i] > 15) return QX_E_ARG;
  for (size_t i = 0; i < n * G; ++i)
    if (selectors[i] > 3) return QX_E_ARG;
  uint8_t* blob = static_cast<uint8_t*>(packed);
  std::memset(blob, 0, L.total);
  pack_rows(d, codes, 0, d->n, blob);
  for (size_t i = 0; i < n * G; ++i) {
    blob[L.scales + 2 * i] = (uint8_t)scales[i];
    blob[L.scales + 2 * i + 1] = (uint8_t)(scales[i] >> 8);
  }
  for (size_t r = 0; r < n; ++r)
    for (size_t j = 0; j < G; ++j) {
      const size_t byte = L.selectors + (r * L.words + j / 16) * 4 + (j % 16) / 4;
      blob[byte] |= (uint8_t)(selectors[r * G + j] << (2 * (j % 4)));
    }
  for (int e = 0; e < 64; ++e) {
    blob[L.codebook + 2 * e] = (uint8_t)codebook[e];
    blob[L.codebook + 2 * e + 1] = (uint8_t)(codebook[e] >> 8);
  }
  return QX_OK;
}

int qx_dequant(const qx_desc* d, const void* packed, int out_kind, void* out, hipStream_t stream) {
  const int st = check_desc(d);
  if (st != QX_OK) return st;
  if (out_kind != QX_OUT_F16 && out_kind != QX_OUT_CODES) return QX_E_ARG;
  if (d->n == 0) return QX_OK;
  if (packed == nullptr || out == nullptr || !aligned16(packed) || !aligned16(out)) return QX_E_ARG;
  return qx::launch_dequant(d, packed, out_kind, out, stream);
}

int qx_gemv(const qx_desc* d, const void* packed, const uint16_t* x, uint16_t* y,
            hipStream_t stream) {
  const int st = check_desc(d);
  if (st != QX_OK) return st;
  if (d->n == 0) return QX_OK;
  if (packed == nullptr || x == nullptr || y == nullptr) return QX_E_ARG;
  if (!aligned16(packed) || !aligned16(x) || !aligned2(y)) return QX_E_ARG;
  return qx::launch_gemv(d, packed, x, y, stream);
}

int qx_gemv_a8(const qx_desc* d, const void* packed, const uint16_t* x, uint16_t* y,
               hipStream_t stream) {
  const int st = check_desc(d);
  if (st != QX_OK) return st;
  if (d->k > 88 * 128) return QX_E_UNSUPPORTED;
  if (d->n == 0) return QX_OK;
  if (packed == nullptr || x == nullptr || y == nullptr) return QX_E_ARG;
  if (!aligned16(packed) || !aligned16(x) || !aligned2(y)) return QX_E_ARG;
  return qx::launch_gemv_a8(d, packed, x, y, stream);
}

int qx_quantize_a8(int32_t m, int32_t k, const uint16_t* X, int8_t* Xq, float* sx, hipStream_t stream) {
  if (m < 0 || m > 65536 || k <= 0 || k % 128 != 0 || k > kMaxK) return QX_E_ARG;
  if (m == 0) return QX_OK;
  if (X == nullptr || Xq == nullptr || sx == nullptr) return QX_E_ARG;
  if (!aligned16(X) || !aligned16(Xq) || (reinterpret_cast<uintptr_t>(sx) & 3u) != 0) return QX_E_ARG;
  return qx::launch_quantize_a8(m, k, X, Xq, sx, stream);
}

int qx_gemm_a8(const qx_desc* d, const void* packed, int32_t m, const int8_t* Xq, const float* sx,
               uint16_t* Y, hipStream_t stream) {
  const int st = check_desc(d);
  if (st != QX_OK) return st;
  if (m < 0 || m > 65536) return QX_E_ARG;
  if (m == 0 || d->n == 0) return QX_OK;
  if (packed == nullptr || Xq == nullptr || sx == nullptr || Y == nullptr) return QX_E_ARG;
  if (!aligned16(packed) || !aligned16(Xq) || (reinterpret_cast<uintptr_t>(sx) & 3u) != 0 || !aligned2(Y))
    return QX_E_ARG;
  if (d->kind != QX_UNIFORM)  // table levels are fp16: the fp16 matrix cores on the int8 codes
    return qx::launch_gemm_lut_a8(d, packed, m, Xq, sx, Y, stream);
  if (m == 1 && d->k <= 88 * 128)  // one row: the A8 GEMV (v_dot4 on its staged int8 row)
    return qx::launch_gemv_a8q(d, packed, Xq, sx, Y, stream);
  // a few rows: every code decoded once for all of them, where that measured faster
  // than the matrix cores (m = 2 on any shape; m = 3, 4 when k > n)
  if (m == 2 || (m >= 3 && m <= 4 && d->k > d->n))
    return qx::launch_gemv_a8_multi(d, packed, m, Xq, sx, Y, stream);
  return qx::launch_gemm_a8(d, packed, m, Xq, sx, Y, stream);
}

int qx_gemm(const qx_desc* d, const void* packed, int32_t m, const uint16_t* X, uint16_t* Y,
            hipStream_t stream) {
  const int st = check_desc(d);
  if (st != QX_OK) return st;
  if (m < 0 || m > 65536) return QX_E_ARG;
  if (m == 0 || d->n == 0) return QX_OK;
  if (packed == nullptr || X == nullptr || Y == nullptr) return QX_E_ARG;
  if (!aligned16(packed) || !aligned16(X) || !aligned2(Y)) return QX_E_ARG;
  if (m == 1 && qx::gemv_multi_applies(d, 1)) return qx::launch_gemv(d, packed, X, Y, stream);
  // a few rows: the GEMV's chunk-per-lane loads with the products on the matrix cores
  if (qx::gemm_skinny_applies(d, m)) return qx::launch_gemm_skinny(d, packed, m, X, Y, stream);
  if (qx::gemv_multi_applies(d, m))  // a few rows: decode every code once, GEMV-style
    return m == 1 ? qx::launch_gemv(d, packed, X, Y, stream)
                  : qx::launch_gemv_multi(d, packed, m, X, Y, stream);
  return qx::launch_gemm(d, packed, m, X, Y, stream);
}

}  // extern "C"
