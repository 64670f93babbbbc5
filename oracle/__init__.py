"""Plain CPU oracle for the group-wise quantized dequantize-and-multiply path.

TEST INFRASTRUCTURE. Only the tests, the smoke check and the CPU-baseline leg
of the benchmark may import this package. The product path never calls it and
shares no code with it: the oracle has its own packer and unpacker of the
packed layout, its own dequantization and its own fp64 products.

What it computes (the method: weights are quantized group-wise to b bits with
group size g, either uniformly with a per-group scale and zero-point or with a
per-group codebook, Section 2.2 and Figure 2a; inference dequantizes them and
multiplies by 16-bit activations, Section 2.4 and the WbA16Gg notation of
Table 1):

  W'[n,k] = fp16_RNE( s[n,j] * (q[n,k] - z[n,j]) )   uniform, j = k // g
  W'[n,k] = C[n,j][ q[n,k] ]                          codebook
  y[n]    = sum_k W'[n,k] * x[k]                      in fp64
  Y[m,n]  = sum_k X[m,k] * W'[n,k]                    in fp64

The paper's own 4-bit format, Q4X (Section 3.2: a per-matrix codebook of 4 x
16 centroids, per group of 64 a scale and a 2-bit sub-codebook selector), has
its layout and dequantization in ``q4x``:

  W'[n,k] = fp16_RNE( s[n,j] * CB[sel[n,j]][q[n,k]] ),  j = k // 64

8-bit activations (Section 2.4; the W3A8 rows of Table 1): ``a8`` quantizes x
per vector to int8 (symmetric, round to nearest) and multiplies uniform codes
in exact integer arithmetic.

Modules: ``layout`` (pack/unpack of the packed layout), ``dequant``,
``matmul`` (fp64 products and the error metric), ``formats`` (sizes and
bits-per-weight), ``q4x``, ``a8``.
"""
from .layout import chunk_bit_positions, pack, unpack  # noqa: F401
from .dequant import dequant, dequant_packed  # noqa: F401
from .matmul import gemv, gemm, normwise_rel_err  # noqa: F401
from .formats import packed_size, bits_per_weight  # noqa: F401
from . import q4x  # noqa: F401
from . import a8  # noqa: F401
