/*
 * qx.h -- C ABI of libqx: group-wise low-bit quantized weights, dequantized
 * and multiplied by fp16 activations on an MI355X (gfx950) GPU.
 *
 * The method (QuantX, arXiv 2505.07531): a weight matrix is quantized
 * group-wise to b bits with group size g along the reduction axis -- the
 * paper's WbA16Gg notation, Table 1 -- either uniformly (equally spaced
 * levels) or with a non-uniform per-group codebook (Section 2.2; Figure 2a
 * shows one group mapped to its codebook). Decoding is memory-bound, so the
 * packing and the dequantization kernels decide the runtime (Section 2.4).
 * This library is that runtime side: it packs codes and tables into one blob
 * and runs the fused dequantize-and-multiply kernels on it.
 *
 * Conventions shared by every call
 *   - W is n x k with rows = output features (the nn.Linear orientation); k
 *     is the reduction axis and groups are g consecutive elements of a row.
 *   - fp16 means IEEE binary16, passed as its uint16_t bit pattern.
 *   - Host pointers are read synchronously. Device pointers must be 16-byte
 *     aligned and stay valid until the work queued on the stream has run.
 *   - Device calls enqueue work on `stream` (NULL = the null stream) and
 *     return without synchronizing. They allocate no memory, keep no global
 *     mutable state besides a per-device cache of the compute-unit count
 *     (filled on first use), and may be captured into a HIP graph. A launch
 *     is checked with hipGetLastError, so a HIP error that an earlier call on
 *     the thread left unread is reported as QX_E_HIP.
 *   - The caller owns every buffer and the stream.
 *   - Errors are negative status codes, listed below; QX_OK is 0. Argument
 *     errors are detected before anything is enqueued. An error raised by the
 *     GPU while the kernel runs surfaces at the caller's synchronization.
 *
 * Packed layout (version 1). The paper fixes no bit layout (its layout
 * figure, Figure 3b, is absent), so this library defines one:
 *   C = k / 128 chunks of 128 consecutive codes per row; G = k / g groups.
 *   Codes region, n*k*b/8 bytes at offset 0: chunk c of row n is 16*b bytes,
 *   split into b slices of 16 bytes; slice s (chunk bytes 16s..16s+15) is at
 *   byte offset ((n*b + s)*C + c)*16. Chunk bit p is bit p%8 of chunk byte
 *   p/8. Inside a chunk:
 *     b = 4: code i in chunk bits 4i..4i+3.
 *     b = 3: chunk byte j (0..47) = A field (bits 0-2) | B field (bits 3-5)
 *            | spare field (bits 6-7);
 *            code i < 48 is the A field of byte i; code 48+j is the B field
 *            of byte j; code 96+m (m < 32) keeps bits 0-1 in the spare field
 *            of byte m and bit 2 in bit 6 + m/16 of byte 32 + m%16.
 *   Metadata region at offset n*k*b/8:
 *     uniform : uint32 per (row, group) at (n*G + j)*4 = scale | zero << 16.
 *     codebook: 2^b fp16 entries per (row, group) at (n*G + j)*2^(b+1).
 *
 * Q4X (the paper's own 4-bit format, Section 3.2, Q4X item, and the Figure 3
 * captions): one codebook of 64 fp16 centroids per matrix, as 4 sub-codebooks
 * of 16; per group of g = 64 weights an fp16 scale s, a 2-bit selector t and
 * 64 4-bit indices q; W' = fp16_RNE(s * CB[t][q]); 4 + 18/64 bits per weight.
 * Blob (b = 4, W = ceil(G/16) selector words per row):
 *   codes     offset 0: the 4-bit codes region above, n*k/2 bytes;
 *   scales    offset S0 = n*k/2: fp16 per (row, group) at S0 + (n*G + j)*2;
 *   selectors offset L0 = S0 + n*G*2: uint32 words, t of group j in bits
 *             2*(j%16), 2*(j%16)+1 of word L0 + (n*W + j/16)*4; other bits 0;
 *   codebook  offset B0 = L0 + n*W*4 rounded up to a multiple of 16: entry e
 *             of sub-codebook t at B0 + (16*t + e)*2; total B0 + 128 bytes.
 */
#ifndef QX_H_
#define QX_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* HIP's stream handle (the same declaration as hip_runtime_api.h). */
typedef struct ihipStream_t* hipStream_t;

enum { QX_UNIFORM = 0, QX_CODEBOOK = 1, QX_Q4X = 2 };  /* qx_desc.kind */
enum { QX_OUT_F16 = 0, QX_OUT_CODES = 1 };   /* qx_dequant out_kind */

enum {
  QX_OK = 0,
  QX_E_ARG = -1,          /* null or misaligned pointer, malformed descriptor or table */
  QX_E_UNSUPPORTED = -2,  /* well-formed but not built (e.g. bits = 2, group = 256) */
  QX_E_SIZE = -3,         /* output capacity too small */
  QX_E_HIP = -4           /* the HIP runtime refused the launch */
};

/*
 * Descriptor of one quantized matrix.
 *   n     rows (output features), n >= 0
 *   k     reduction length, a positive multiple of 128 (at most 1 << 20)
 *   bits  code width b: 3 or 4 (4 for QX_Q4X)
 *   group g: 32, 64 or 128 (64 for QX_Q4X)
 *   kind  QX_UNIFORM, QX_CODEBOOK or QX_Q4X; a QX_Q4X descriptor with other
 *         bits or group is malformed (QX_E_ARG)
 *   flags must be 0
 */
typedef struct {
  int32_t n, k, bits, group, kind;
  uint32_t flags;
} qx_desc;

/*
 * qx_pack_layout -- write the packed blob of one quantized matrix (host).
 * Passage: group-wise b-bit codes with per-group metadata (Table 1's WbA16Gg
 * notation; uniform levels versus a per-group codebook, Section 2.2 and
 * Figure 2a).
 *   codes     uint8 [n][k] row-major, each < 2^bits.
 *   scales    fp16 [n][k/g] (uniform; NULL for codebook). Must be finite.
 *   zeros     fp16 [n][k/g] (uniform; NULL for codebook). Each must be an
 *             integer in [0, 2^bits - 1] (the levels are scale*(q - zero)).
 *   codebook  fp16 [n][k/g][2^bits] (codebook; NULL for uniform). Any values.
 *   packed    output, host memory of `cap` bytes; NULL = size query only.
 *   packed_size  receives the blob size (n*k*b/8 plus the tables); required.
 * All pointers are host pointers. Pure and synchronous; returns QX_E_ARG for
 * a bad descriptor, a missing table, an out-of-range code or zero-point or a
 * non-finite scale, and QX_E_SIZE when cap < *packed_size (nothing written).
 * QX_Q4X descriptors are packed by qx_pack_q4x (QX_E_ARG here).
 */
int qx_pack_layout(const qx_desc* d, const uint8_t* codes, const uint16_t* scales,
                   const uint16_t* zeros, const uint16_t* codebook, void* packed, size_t cap,
                   size_t* packed_size);

/*
 * qx_pack_q4x -- write the packed blob of one Q4X matrix (host).
 * Passage: Section 3.2, Q4X item (per group of 64 a 2-byte scale, a 2-bit
 * codebook index and 64 4-bit centroid indices; 64 centroids per matrix in 4
 * groups of 16), and the Figure 3a/3b captions.
 *   d          descriptor with kind QX_Q4X, bits 4, group 64.
 *   codes      uint8 [n][k] row-major, each < 16.
 *   scales     fp16 [n][k/64]; any values (W' is their IEEE product).
 *   selectors  uint8 [n][k/64], each < 4.
 *   codebook   fp16 [4][16]: sub-codebook t, entry e at [t][e]; any values.
 *   packed, cap, packed_size as for qx_pack_layout.
 * All pointers are host pointers. Pure and synchronous; returns QX_E_ARG for a
 * descriptor of another kind, a missing input or an out-of-range code or
 * selector, and QX_E_SIZE when cap < *packed_size (nothing written).
 */
int qx_pack_q4x(const qx_desc* d, const uint8_t* codes, const uint16_t* scales,
                const uint8_t* selectors, const uint16_t* codebook, void* packed, size_t cap,
                size_t* packed_size);

/*
 * qx_dequant -- expand a packed blob into fp16 weights or raw codes (device).
 * Passage: the custom dequantization kernels of Section 2.4.
 *   packed   device blob written by qx_pack_layout (copied to the GPU).
 *   out_kind QX_OUT_F16: out = fp16 W' [n][k], uniform W' = fp16_RNE(s*(q-z))
 *            (the exact product, rounded once), codebook W' = C[q], Q4X
 *            W' = fp16_RNE(s*CB[t][q]).
 *            QX_OUT_CODES: out = uint8 codes [n][k].
 *   out      device buffer of n*k*2 (F16) or n*k (CODES) bytes.
 * Results are bit-exact with the definitions above.
 */
int qx_dequant(const qx_desc* d, const void* packed, int out_kind, void* out, hipStream_t stream);

/*
 * qx_gemv -- y = W' x for one activation vector (device).
 * Passage: decoding, the memory-bound case of Section 2.4, with fp16
 * activations (the A16 of Table 1).
 *   packed  device blob; x fp16 [k]; y fp16 [n] (written, RNE from an fp32
 *           accumulator). y must not overlap x or packed.
 * Products of fp16 values are exact, sums are fp32 in a fixed order, so the
 * result is deterministic run to run. Uniform groups are multiplied with their
 * exact levels s*(q - z), the zero point taken out once per group, rather than
 * with W' rounded to binary16: the two differ by that rounding (at most 2^-12
 * of each weight). n = 0 is a no-op.
 */
int qx_gemv(const qx_desc* d, const void* packed, const uint16_t* x, uint16_t* y,
            hipStream_t stream);

/*
 * qx_gemv_a8 -- y = W' x with x quantized to 8 bits (device; every kind).
 * Passage: activations are quantized to 8 bits and not below (Section 2.4);
 * the W3A8 configurations of Table 1 and Table 2's runs use 8-bit
 * round-to-nearest per-token activations.
 *   x fp16 [k], finite, quantized on the fly with one symmetric scale:
 *     amax = max|x|, xq = clamp(rint(x * (127/amax)), -127, 127) (fp32; the
 *     scale s_x = amax/127; amax = 0 gives y = 0);
 *   y fp16 [n] = s_x * sum_j s_j * sum_{k in group j} (q - z_j) * xq, the
 *     integer sums exact, scaled in fp32 and rounded to nearest-even;
 *   codebook (QuantX's non-uniform groups, Section 2.2, in its W3A8
 *     configurations): y = s_x * sum_k C_j[q] * xq, fp32 products of the fp16
 *     table entries and the integers xq, sums in fp32;
 *   Q4X (the paper's Q4X with 8-bit activations, Table 2): y = s_x * sum_j s_j *
 *     sum_{k in group j} CB[t_j][q] * xq, fp32 products of the fp16 entries and
 *     the integers xq, sums in fp32.
 * Descriptors with k <= 88*128 only (QX_E_UNSUPPORTED otherwise).
 * Deterministic; n = 0 is a no-op; buffers and alignment as for qx_gemv.
 */
int qx_gemv_a8(const qx_desc* d, const void* packed, const uint16_t* x, uint16_t* y,
               hipStream_t stream);

/*
 * qx_quantize_a8 -- per-token 8-bit activations for qx_gemm_a8 (device).
 * Passage: activations quantized to 8 bits by round-to-nearest, one scale per
 * token (Section 2.4; the W3A8 rows of Table 1, Table 2's runs).
 *   X fp16 [m][k] row-major, finite, 16-byte aligned; k a positive multiple of
 *   128 (at most 1 << 20), 0 <= m <= 65536.
 *   Xq int8 [m][k] (written, 16-byte aligned), sx fp32 [m] (written), per row
 *   exactly as qx_gemv_a8 quantizes its vector: amax = max|x|, xq = nearest
 *   integer to x * fp32(127/amax) (the product exact), sx = fp32(amax/127);
 *   an all-zero row gives xq = 0, sx = 0.
 * The codes of one X can feed every product that reads that X (q, k and v, or
 * gate and up). QX_E_ARG for bad sizes, null or misaligned pointers.
 */
int qx_quantize_a8(int32_t m, int32_t k, const uint16_t* X, int8_t* Xq, float* sx,
                   hipStream_t stream);

/*
 * qx_gemm_a8 -- Y = X W'^T with 8-bit activations (device; every kind).
 * Passage: as qx_gemv_a8, for m activation rows (prefill of a W3A8 model; Table 2
 * runs Q4X prefill with 8-bit activations).
 *   Xq, sx as qx_quantize_a8 wrote them for the same k; Y fp16 [m][n]
 *   (written, 2-byte aligned), rounded to nearest-even:
 *   uniform: sx[r] * sum_j s_j * sum_{k in group j} (q - z_j) * xq[r][k], the
 *     group sums exact (int8 matrix-core products, int32 accumulation), scaled
 *     in fp32;
 *   codebook: sx[r] * sum_k C_j[q] * xq[r][k] on the fp16 matrix cores (the
 *     table entries and the codes xq as exact fp16 values, fp32 accumulation),
 *     scaled in fp32;
 *   Q4X: sx[r] * sum_j s_j * sum_{k in group j} CB[t_j][q] * xq[r][k], each
 *     group's sum from the fp16 matrix cores scaled by s_j in fp32 (the exact
 *     s * CB, as qx_gemv_a8; one row gives the same bits as qx_gemv_a8 on
 *     the row the codes were quantized from when that row is one-hot).
 * m = 0 or n = 0 is a no-op; m must be <= 65536.
 */
int qx_gemm_a8(const qx_desc* d, const void* packed, int32_t m, const int8_t* Xq, const float* sx,
               uint16_t* Y, hipStream_t stream);

/*
 * qx_gemm -- Y = X W'^T for m activation rows (device; prefill and batched decode).
 * Passage: as qx_gemv, batched over m rows.
 *   X fp16 [m][k] row-major; Y fp16 [m][n] row-major (written; 2-byte
 *   alignment suffices for Y). fp16 products, fp32 accumulate, RNE to fp16:
 *   on the matrix cores with W' decoded exactly into their operands (for a few
 *   rows, m <= 64 by shape and format, each lane decoding its own chunks as in
 *   the GEMV), or, for m <= 4 where that measured faster, GEMV-style with every
 *   code decoded once for all rows. m = 0 or n = 0 is a no-op; m must be
 *   <= 65536. All formats, Q4X included. Deterministic.
 */
int qx_gemm(const qx_desc* d, const void* packed, int32_t m, const uint16_t* X, uint16_t* Y,
            hipStream_t stream);

/* Static string for a status code ("unknown status" for values not listed). */
const char* qx_status_str(int status);

#ifdef __cplusplus
}
#endif

#endif /* QX_H_ */
