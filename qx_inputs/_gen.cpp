// Seeded synthetic inputs for the group-wise quantized GEMV/GEMM workloads.
//
// This file is input preparation only. It draws weights and activations from
// a counter-based generator, and it turns fp32 weights into the integer codes
// and fp16 per-group tables that the library's packer takes as input. The
// quantized product path never quantizes, and the oracle never re-derives
// codes: both consume what this file writes.
//
// Random numbers: Philox4x64-10 (Salmon, Moraes, Dror and Shaw, "Parallel
// random numbers: as easy as 1, 2, 3", SC 2011). Element i of stream t under
// seed s is drawn from the block Philox(counter = (i, 0, 0, 0), key = (s, t)),
// so any row of any matrix can be regenerated without drawing the others.
//
// Quantizers (the paper distinguishes uniform quantization with equally spaced
// levels from non-uniform, PDF-driven per-group codebooks, Section 2.2 and the
// caption of Figure 2a):
//   uniform : per group, the range [min(w,0), max(w,0)] is split into 2^b-1
//             steps; the step is rounded UP to fp16, the zero-point is an
//             integer code, codes are round-to-nearest-even and clamped.
//   codebook: per group, 1-D k-means (Lloyd) started from the uniform levels,
//             centroids rounded to fp16, then each weight takes the nearest
//             stored entry (ties to the lower index).
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <vector>

#include <omp.h>

namespace {

// ---------------------------------------------------------------- Philox4x64
inline void mulhilo64(uint64_t a, uint64_t b, uint64_t* hi, uint64_t* lo) {
  const __uint128_t p = (__uint128_t)a * (__uint128_t)b;
  *hi = (uint64_t)(p >> 64);
  *lo = (uint64_t)p;
}

inline void philox4x64_10(const uint64_t in[4], const uint64_t key_in[2], uint64_t out[4]) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ULL, M1 = 0xCA5A826395121157ULL;
  const uint64_t W0 = 0x9E3779B97F4A7C15ULL, W1 = 0xBB67AE8584CAA73BULL;
  uint64_t c0 = in[0], c1 = in[1], c2 = in[2], c3 = in[3];
  uint64_t k0 = key_in[0], k1 = key_in[1];
  for (int r = 0; r < 10; ++r) {
    uint64_t hi0, lo0, hi1, lo1;
    mulhilo64(M0, c0, &hi0, &lo0);
    mulhilo64(M1, c2, &hi1, &lo1);
    const uint64_t n0 = hi1 ^ c1 ^ k0, n1 = lo1, n2 = hi0 ^ c3 ^ k1, n3 = lo0;
    c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    k0 += W0; k1 += W1;
  }
  out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

// Uniform double strictly inside (0, 1) from the top 53 bits.
inline double u01(uint64_t x) { return ((double)(x >> 11) + 0.5) * 0x1p-53; }

const double kTwoPi = 6.283185307179586476925286766559;

enum Dist { kNormal = 0, kLaplace = 1, kStudentT4 = 2 };

// One sample per Philox block, so that sample i depends only on i.
inline double draw(int dist, double p, uint64_t seed, uint64_t stream, uint64_t i) {
  const uint64_t ctr[4] = {i, 0, 0, 0};
  const uint64_t key[2] = {seed, stream};
  uint64_t r[4];
  philox4x64_10(ctr, key, r);
  switch (dist) {
    case kNormal: {  // Box-Muller, cosine branch; p = standard deviation
      const double z = std::sqrt(-2.0 * std::log(u01(r[0]))) * std::cos(kTwoPi * u01(r[1]));
      return p * z;
    }
    case kLaplace: {  // inverse CDF; p = scale b
      const double u = u01(r[0]) - 0.5;
      const double a = std::fabs(u);
      const double mag = -p * std::log(1.0 - 2.0 * a);
      return u < 0 ? -mag : mag;
    }
    case kStudentT4: {  // Z / sqrt(V/4), V ~ chi^2_4 = -2 ln(U1 U2); Var(t_4) = 2; p = target std
      const double z = std::sqrt(-2.0 * std::log(u01(r[0]))) * std::cos(kTwoPi * u01(r[1]));
      const double v = -2.0 * (std::log(u01(r[2])) + std::log(u01(r[3])));
      return (p / std::sqrt(2.0)) * z / std::sqrt(v / 4.0);
    }
  }
  return 0.0;
}

// ------------------------------------------------------------ binary16 helpers
// binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits.
inline double half_to_double(uint16_t h) {
  const int s = h >> 15, e = (h >> 10) & 31, f = h & 1023;
  double v;
  if (e == 0) v = std::ldexp((double)f, -24);
  else if (e == 31) v = f ? NAN : INFINITY;
  else v = std::ldexp((double)(f | 1024), e - 25);
  return s ? -v : v;
}

// Encode a non-negative value that is exactly representable in binary16.
inline uint16_t encode_half_mag(double v) {
  if (v == 0.0) return 0;
  if (std::isinf(v)) return 0x7C00;
  int ex;
  const double m = std::frexp(v, &ex);  // v = m * 2^ex, m in [0.5, 1)
  const int E = ex + 14;                // biased exponent of v = (2m) * 2^(ex-1)
  if (E <= 0) return (uint16_t)std::ldexp(v, 24);  // subnormal: v = f * 2^-24
  const uint16_t f = (uint16_t)((m * 2.0 - 1.0) * 1024.0);
  return (uint16_t)((E << 10) | f);
}

// mode 0: round to nearest, ties to even.  mode 1: round toward +infinity.
inline uint16_t double_to_half(double x, int mode) {
  if (std::isnan(x)) return 0x7E00;
  const bool neg = std::signbit(x);
  const double a = std::fabs(x);
  uint16_t mag;
  if (std::isinf(a)) {
    mag = 0x7C00;
  } else {
    int ex;
    std::frexp(a, &ex);  // a in [2^(ex-1), 2^ex)
    const double q = (a < 0x1p-14) ? 0x1p-24 : std::ldexp(1.0, ex - 11);  // spacing of binary16 near a
    const double m = a / q;  // exact: q is a power of two
    double r;
    if (mode == 0) r = std::nearbyint(m);
    else r = neg ? std::floor(m) : std::ceil(m);
    const double v = r * q;
    mag = (v > 65504.0) ? (uint16_t)0x7C00 : encode_half_mag(v);
  }
  return (uint16_t)((neg ? 0x8000 : 0) | mag);
}

// ---------------------------------------------------------------- quantizers
struct UniformParams {
  double s16;   // fp16 step (as a double)
  int z;        // integer zero-point
  bool ok;
};

inline UniformParams uniform_params(const float* w, int g, int bits) {
  double lo = 0.0, hi = 0.0;
  for (int i = 0; i < g; ++i) {
    lo = std::min(lo, (double)w[i]);
    hi = std::max(hi, (double)w[i]);
  }
  const int qmax = (1 << bits) - 1;
  UniformParams p{1.0, 0, true};
  if (hi == lo) return p;  // all-zero group: step 1, zero 0, every code 0
  const double s = (hi - lo) / (double)qmax;
  p.s16 = half_to_double(double_to_half(s, 1));
  if (!(p.s16 > 0.0) || std::isinf(p.s16)) { p.ok = false; return p; }
  double z = std::nearbyint(-lo / p.s16);
  z = std::min(std::max(z, 0.0), (double)qmax);
  p.z = (int)z;
  return p;
}

inline int uniform_code(double w, const UniformParams& p, int qmax) {
  double q = std::nearbyint(w / p.s16) + (double)p.z;
  q = std::min(std::max(q, 0.0), (double)qmax);
  return (int)q;
}

// Lloyd iterations on one sorted group. c[] holds E strictly increasing
// centroids on entry and on exit. Returns the number of iterations run.
int lloyd_sorted(const double* v, const double* prefix, int g, double* c, int E, int max_iter) {
  std::vector<int> split(E + 1), prev(E + 1, -1);
  int it = 0;
  for (; it < max_iter; ++it) {
    // split[e] = first index whose nearest centroid is >= e (ties go to the lower centroid).
    split[0] = 0;
    split[E] = g;
    for (int e = 1; e < E; ++e) {
      // smallest i with |v[i]-c[e]| < |v[i]-c[e-1]|; the predicate is monotone in i
      int lo = split[e - 1], hi = g;
      while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        const bool closer_up = std::fabs(v[mid] - c[e]) < std::fabs(v[mid] - c[e - 1]);
        if (closer_up) hi = mid; else lo = mid + 1;
      }
      split[e] = lo;
    }
    if (split == prev) break;
    prev = split;
    for (int e = 0; e < E; ++e) {
      const int a = split[e], b = split[e + 1];
      if (b > a) c[e] = (prefix[b] - prefix[a]) / (double)(b - a);
    }
  }
  return it;
}

}  // namespace

extern "C" {

// Raw Philox4x64-10 block, exposed for known-answer tests.
void qxi_philox4x64(const uint64_t* ctr, const uint64_t* key, uint64_t* out) {
  philox4x64_10(ctr, key, out);
}

// binary16 conversion, exposed so its rounding can be checked against numpy.
void qxi_double_to_half(const double* x, int64_t count, int mode, uint16_t* out) {
  for (int64_t i = 0; i < count; ++i) out[i] = double_to_half(x[i], mode);
}

// Fill out[0..count) with samples start..start+count-1 of (seed, stream).
// dist: 0 normal(0, p), 1 Laplace(0, p), 2 Student-t(4) scaled to std p.
int qxi_fill_f64(int dist, double p, uint64_t seed, uint64_t stream, uint64_t start, int64_t count,
                 double* out, int nthreads) {
  if (dist < 0 || dist > 2 || count < 0) return -1;
#pragma omp parallel for schedule(static) num_threads(nthreads > 0 ? nthreads : omp_get_max_threads())
  for (int64_t i = 0; i < count; ++i) out[i] = draw(dist, p, seed, stream, start + (uint64_t)i);
  return 0;
}

int qxi_fill_f32(int dist, double p, uint64_t seed, uint64_t stream, uint64_t start, int64_t count,
                 float* out, int nthreads) {
  if (dist < 0 || dist > 2 || count < 0) return -1;
#pragma omp parallel for schedule(static) num_threads(nthreads > 0 ? nthreads : omp_get_max_threads())
  for (int64_t i = 0; i < count; ++i) out[i] = (float)draw(dist, p, seed, stream, start + (uint64_t)i);
  return 0;
}

// Uniform group-wise quantization of w [n][k] (groups of g along k).
// codes [n][k] in [0, 2^bits); scales, zeros [n][k/g] as binary16 bit patterns.
int qxi_quantize_uniform(const float* w, int64_t n, int64_t k, int bits, int g, uint8_t* codes,
                         uint16_t* scales, uint16_t* zeros, int nthreads) {
  if (n < 0 || k <= 0 || g <= 0 || k % g != 0 || bits < 1 || bits > 8) return -1;
  const int64_t G = k / g, total = n * G;
  const int qmax = (1 << bits) - 1;
  int bad = 0;
#pragma omp parallel for schedule(static) reduction(| : bad) \
    num_threads(nthreads > 0 ? nthreads : omp_get_max_threads())
  for (int64_t t = 0; t < total; ++t) {
    const float* wg = w + t * g;
    const UniformParams p = uniform_params(wg, g, bits);
    if (!p.ok) { bad |= 1; continue; }
    for (int i = 0; i < g; ++i) codes[t * g + i] = (uint8_t)uniform_code((double)wg[i], p, qmax);
    scales[t] = double_to_half(p.s16, 0);
    zeros[t] = double_to_half((double)p.z, 0);
  }
  return bad ? -2 : 0;
}

// Per-group codebook quantization: 2^bits fp16 entries per group, fit by 1-D
// k-means started at the group's uniform levels. codebook [n][k/g][2^bits].
// raw (nullable) receives the converged centroids before fp16 rounding, and
// iters (nullable) the Lloyd iteration count of each group.
int qxi_quantize_codebook(const float* w, int64_t n, int64_t k, int bits, int g, int max_iter,
                          uint8_t* codes, uint16_t* codebook, double* raw, int32_t* iters,
                          int nthreads) {
  if (n < 0 || k <= 0 || g <= 0 || k % g != 0 || bits < 1 || bits > 8 || max_iter < 0) return -1;
  const int64_t G = k / g, total = n * G;
  const int E = 1 << bits;
  int bad = 0;
#pragma omp parallel num_threads(nthreads > 0 ? nthreads : omp_get_max_threads()) reduction(| : bad)
  {
    std::vector<double> v(g), prefix(g + 1), c(E), cb(E);
#pragma omp for schedule(static)
    for (int64_t t = 0; t < total; ++t) {
      const float* wg = w + t * g;
      const UniformParams p = uniform_params(wg, g, bits);
      if (!p.ok) { bad |= 1; continue; }
      for (int e = 0; e < E; ++e) c[e] = p.s16 * (double)(e - p.z);
      for (int i = 0; i < g; ++i) v[i] = (double)wg[i];
      std::sort(v.begin(), v.end());
      prefix[0] = 0.0;
      for (int i = 0; i < g; ++i) prefix[i + 1] = prefix[i] + v[i];
      const int it = lloyd_sorted(v.data(), prefix.data(), g, c.data(), E, max_iter);
      if (iters) iters[t] = it;
      if (raw) for (int e = 0; e < E; ++e) raw[t * E + e] = c[e];
      uint16_t* out = codebook + t * E;
      for (int e = 0; e < E; ++e) {
        out[e] = double_to_half(c[e], 0);
        cb[e] = half_to_double(out[e]);
      }
      // Lloyd keeps centroids sorted and fp16 rounding is monotone; the sort
      // below only guards the stored table's ascending order.
      std::vector<int> order(E);
      for (int e = 0; e < E; ++e) order[e] = e;
      std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return cb[a] < cb[b]; });
      uint16_t tmp[256];
      for (int e = 0; e < E; ++e) tmp[e] = out[order[e]];
      for (int e = 0; e < E; ++e) { out[e] = tmp[e]; cb[e] = half_to_double(tmp[e]); }
      for (int i = 0; i < g; ++i) {
        const double x = (double)wg[i];
        int best = 0;
        double bd = std::fabs(x - cb[0]);
        for (int e = 1; e < E; ++e) {
          const double d = std::fabs(x - cb[e]);
          if (d < bd) { bd = d; best = e; }
        }
        codes[t * g + i] = (uint8_t)best;
      }
    }
  }
  return bad ? -2 : 0;
}

// Q4X (groups of 64, a 4 x 16 binary16 codebook): per group, the 32-bin histogram
// over [-1, 1] of w / s16 (fractions), and, given the codebook, the nearest level
// fp16(s16 * CB[t][e]) of every weight for each sub-codebook t (ties to the lowest
// index) and the sub-codebook of least squared error (ties to the lowest t).
int qxi_q4x_histograms(const float* w, int64_t ngroups, const uint16_t* s16, double* hist,
                       int threads) {
#pragma omp parallel for num_threads(threads) schedule(static)
  for (int64_t g = 0; g < ngroups; ++g) {
    const double s = half_to_double(s16[g]);
    double* h = hist + g * 32;
    for (int b = 0; b < 32; ++b) h[b] = 0.0;
    for (int i = 0; i < 64; ++i) {
      const double u = (double)w[g * 64 + i] / s;
      int b = (int)std::floor((u + 1.0) * 16.0);
      b = b < 0 ? 0 : (b > 31 ? 31 : b);
      h[b] += 1.0 / 64.0;
    }
  }
  return 0;
}

int qxi_q4x_assign(const float* w, int64_t ngroups, const uint16_t* s16, const uint16_t* cb,
                   uint8_t* codes, uint8_t* sel, int threads) {
#pragma omp parallel for num_threads(threads) schedule(static)
  for (int64_t g = 0; g < ngroups; ++g) {
    const double s = half_to_double(s16[g]);
    double best_err = INFINITY;
    uint8_t best_q[64];
    int best_t = 0;
    for (int t = 0; t < 4; ++t) {
      double lv[16];
      for (int e = 0; e < 16; ++e) lv[e] = half_to_double(double_to_half(s * half_to_double(cb[16 * t + e]), 0));
      double err = 0.0;
      uint8_t q[64];
      for (int i = 0; i < 64; ++i) {
        const double x = (double)w[g * 64 + i];
        int best = 0;
        double bd = std::fabs(x - lv[0]);
        for (int e = 1; e < 16; ++e) {
          const double d = std::fabs(x - lv[e]);
          if (d < bd) { bd = d; best = e; }
        }
        q[i] = (uint8_t)best;
        err += bd * bd;
      }
      if (err < best_err) {
        best_err = err;
        best_t = t;
        for (int i = 0; i < 64; ++i) best_q[i] = q[i];
      }
    }
    sel[g] = (uint8_t)best_t;
    for (int i = 0; i < 64; ++i) codes[g * 64 + i] = best_q[i];
  }
  return 0;
}

}  // extern "C"
