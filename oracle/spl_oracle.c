/*
 * CPU oracle for bitmask-compressed sparse linear layers.
 *
 * TEST INFRASTRUCTURE ONLY.  Plain, slow and meant to be checked by eye
 * against the paper: only the test suite, the package smoke check and the
 * benchmark's CPU-baseline leg load this library.  The GPU library never
 * links, loads or calls it, and the two share no source, header, table or
 * helper.  Floating point is evaluated in IEEE binary64 unless a step of the
 * method fixes another precision (the int8 epilogue below).
 *
 * What is computed (paper, arXiv 2405.03594):
 *
 *   Bitmask expansion (section 2.4.1 and its worked example; section 2.4.2
 *   extends it to GPU submatrices): the kept entries of a weight matrix are
 *   stored densely, in order, and a bitmask with one bit per matrix position
 *   records which positions are kept.  The compression is lossless, so the
 *   sparse linear layer reaches exactly the plain product
 *
 *        Y[m][n] = sum_k X[m][k] * (W (.) Mask)[n][k]          (W is [N][K])
 *
 *   and the oracle for the linear layers is that definition written out.
 *   The packer and unpacker are the one place where the output is the
 *   method's own encoding; they follow the description step by step.
 *
 * Canonical encoding (the reading taken where the paper leaves it open):
 *   - bitmask: uint32 words, ceil(K/32) per row; bit j (LSB first) of word w
 *     of row n is set iff position (n, 32*w + j) is kept; bits past K are 0;
 *   - values: kept entries, row by row, ascending column order, raw bit
 *     copies (2-byte fp16/bf16 or 1-byte int8 payloads);
 *   - row_offsets[n]: index in values of row n's first kept entry;
 *     row_offsets[N] = number of kept entries.
 *   A position is kept iff mask[n][k] != 0; with no mask, iff the payload is
 *   non-zero (for fp16/bf16 the sign bit is ignored, so -0.0 is not kept).
 *
 * Sparse-quantized linear (section 3.4): int8 weights and int8 activations,
 * exact integer accumulation, then a dequantisation evaluated in binary32 in
 * this order, with no fused multiply-add:
 *        y = to_fp16_rne( (float(acc) * sx[m]) * sw[n] )
 * Build with -ffp-contract=off so no product is fused.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORC_F16 = 1, ORC_BF16 = 2, ORC_I8 = 3 };

/* ---------------------------------------------------------------- numbers */

/* IEEE 754 binary16 -> binary64, from the format definition
 * (1 sign, 5 exponent bits with bias 15, 10 fraction bits). */
double orc_f16_to_f64(uint16_t h) {
  int sign = (h >> 15) & 1;
  int e = (h >> 10) & 0x1f;
  int f = h & 0x3ff;
  double v;
  if (e == 0) {
    v = ldexp((double)f, -24);                 /* subnormal: f * 2^-24 */
  } else if (e == 31) {
    v = (f == 0) ? INFINITY : NAN;
  } else {
    v = ldexp((double)(1024 + f), e - 25);     /* (1 + f/1024) * 2^(e-15) */
  }
  return sign ? -v : v;
}

/* bfloat16 -> binary64 (1 sign, 8 exponent bits with bias 127, 7 fraction
 * bits: the upper half of a binary32). */
double orc_bf16_to_f64(uint16_t b) {
  int sign = (b >> 15) & 1;
  int e = (b >> 7) & 0xff;
  int f = b & 0x7f;
  double v;
  if (e == 0) {
    v = ldexp((double)f, -133);                /* f * 2^-126 / 128 */
  } else if (e == 255) {
    v = (f == 0) ? INFINITY : NAN;
  } else {
    v = ldexp((double)(128 + f), e - 134);     /* (1 + f/128) * 2^(e-127) */
  }
  return sign ? -v : v;
}

/* binary32 -> binary16, round to nearest, ties to even.  Every finite
 * binary16 value is an integer multiple of its spacing q (2^-24 below 2^-14,
 * else 2^(e-10) for |x| in [2^e, 2^(e+1))); x/q is exact in binary64 and
 * rint() rounds it ties-to-even in the default rounding mode. */
uint16_t orc_f32_to_f16(float xf) {
  double x = (double)xf;
  uint16_t sign = signbit(x) ? 0x8000 : 0;
  if (isnan(x)) return (uint16_t)(sign | 0x7e00);
  double a = fabs(x);
  if (isinf(a)) return (uint16_t)(sign | 0x7c00);
  if (a == 0.0) return sign;
  int e;
  frexp(a, &e);                 /* a = m * 2^e, m in [0.5, 1) -> a in [2^(e-1), 2^e) */
  int p = e - 1;                /* a in [2^p, 2^(p+1)) */
  double q = (p < -14) ? ldexp(1.0, -24) : ldexp(1.0, p - 10);
  double r = rint(a / q) * q;   /* nearest representable magnitude (unbounded exponent) */
  if (r >= 65536.0) return (uint16_t)(sign | 0x7c00);   /* beyond the largest finite value */
  if (r < ldexp(1.0, -14)) {
    /* subnormal (or zero): fraction = r / 2^-24 */
    return (uint16_t)(sign | (uint16_t)(r / ldexp(1.0, -24)));
  }
  int er;
  frexp(r, &er);
  int pe = er - 1;              /* r in [2^pe, 2^(pe+1)) */
  uint16_t frac = (uint16_t)(r / ldexp(1.0, pe - 10) - 1024.0);
  return (uint16_t)(sign | (uint16_t)((pe + 15) << 10) | frac);
}

static double elem_to_f64(const void* base, int64_t i, int32_t dtype) {
  if (dtype == ORC_F16) return orc_f16_to_f64(((const uint16_t*)base)[i]);
  if (dtype == ORC_BF16) return orc_bf16_to_f64(((const uint16_t*)base)[i]);
  return (double)((const int8_t*)base)[i];
}

static int elem_bytes(int32_t dtype) { return dtype == ORC_I8 ? 1 : 2; }

static int is_kept(const void* W, int32_t dtype, const uint8_t* mask, int64_t idx) {
  if (mask) return mask[idx] != 0;
  if (dtype == ORC_I8) return ((const int8_t*)W)[idx] != 0;
  return (((const uint16_t*)W)[idx] & 0x7fff) != 0;
}

/* ---------------------------------------------------------------- packer */

int64_t orc_words_per_row(int64_t K) { return (K + 31) / 32; }

/* Number of kept entries. */
int64_t orc_pack_nnz(const void* W, int32_t dtype, const uint8_t* mask, int64_t N, int64_t K) {
  int64_t c = 0;
  for (int64_t i = 0; i < N * K; ++i) c += is_kept(W, dtype, mask, i);
  return c;
}

/* Bitmask expansion encoder: walk each row in column order; for a kept
 * position set its bit and append its payload to values. */
void orc_pack(const void* W, int32_t dtype, const uint8_t* mask, int64_t N, int64_t K,
              uint32_t* bitmask, void* values, int32_t* row_offsets) {
  int64_t words = orc_words_per_row(K);
  int eb = elem_bytes(dtype);
  memset(bitmask, 0, (size_t)(N * words) * sizeof(uint32_t));
  int64_t c = 0;
  for (int64_t n = 0; n < N; ++n) {
    row_offsets[n] = (int32_t)c;
    for (int64_t k = 0; k < K; ++k) {
      int64_t idx = n * K + k;
      if (is_kept(W, dtype, mask, idx)) {
        bitmask[n * words + k / 32] |= (uint32_t)1u << (k % 32);
        memcpy((char*)values + c * eb, (const char*)W + idx * eb, (size_t)eb);
        ++c;
      }
    }
  }
  row_offsets[N] = (int32_t)c;
}

/* Decoder: every set bit takes the next stored payload of its row; every
 * other position becomes +0. */
void orc_unpack(const uint32_t* bitmask, const void* values, const int32_t* row_offsets, int32_t dtype,
                int64_t N, int64_t K, void* W_out) {
  int64_t words = orc_words_per_row(K);
  int eb = elem_bytes(dtype);
  memset(W_out, 0, (size_t)(N * K * eb));
  for (int64_t n = 0; n < N; ++n) {
    int64_t c = row_offsets[n];
    for (int64_t k = 0; k < K; ++k) {
      if ((bitmask[n * words + k / 32] >> (k % 32)) & 1u) {
        memcpy((char*)W_out + (n * K + k) * eb, (const char*)values + c * eb, (size_t)eb);
        ++c;
      }
    }
  }
}

/* ---------------------------------------------------------- tiled layout */
/*
 * GPU layout (section 2.4.2: the compressed matrix is cut into submatrices
 * sized for the register file, each stored as its own bitmask plus its dense
 * kept values).  Submatrices are TR x TC = 16 x 32 tiles: tile (b, s) covers
 * rows 16b..16b+15 and columns 32s..32s+31.  Tiles are ordered by b, then s.
 *   bitmask_t[(b*S + s)*16 + r]: bit j set iff (16b + r, 32s + j) is kept
 *                                (0 for rows >= N and columns >= K);
 *   values_t: each tile's kept payloads, column group by column group, inside
 *             a group row by row, inside a row ascending column.  A column
 *             group is the 16 bytes of dense payload one matrix-core lane
 *             holds: G = 16 / element bytes columns (8 for fp16/bf16, 16 for
 *             int8), groups g = 0 .. 32/G - 1 covering columns G g .. G g + G - 1;
 *   tile_offsets[b*S + s]: index in values_t of the tile's first payload;
 *   tile_offsets[B*S] = nnz.   (B = ceil(N/16) row blocks, S = ceil(K/32).)
 */
static int64_t tile_group_cols(int32_t dtype) { return 16 / elem_bytes(dtype); }
int64_t orc_tile_blocks(int64_t N) { return (N + 15) / 16; }
int64_t orc_tile_ksteps(int64_t K) { return (K + 31) / 32; }

void orc_pack_tiled(const void* W, int32_t dtype, const uint8_t* mask, int64_t N, int64_t K,
                    uint32_t* bitmask_t, void* values_t, int32_t* tile_offsets) {
  int64_t B = orc_tile_blocks(N), S = orc_tile_ksteps(K);
  int eb = elem_bytes(dtype);
  int64_t G = tile_group_cols(dtype);
  int64_t c = 0;
  for (int64_t b = 0; b < B; ++b) {
    for (int64_t s = 0; s < S; ++s) {
      int64_t t = b * S + s;
      tile_offsets[t] = (int32_t)c;
      for (int64_t r = 0; r < 16; ++r) bitmask_t[t * 16 + r] = 0;
      for (int64_t g = 0; g < 32 / G; ++g) {
        for (int64_t r = 0; r < 16; ++r) {
          int64_t n = 16 * b + r;
          for (int64_t j = G * g; j < G * g + G; ++j) {
            int64_t k = 32 * s + j;
            if (n < N && k < K && is_kept(W, dtype, mask, n * K + k)) {
              bitmask_t[t * 16 + r] |= (uint32_t)1u << j;
              memcpy((char*)values_t + c * eb, (const char*)W + (n * K + k) * eb, (size_t)eb);
              ++c;
            }
          }
        }
      }
    }
  }
  tile_offsets[B * S] = (int32_t)c;
}

void orc_unpack_tiled(const uint32_t* bitmask_t, const void* values_t, const int32_t* tile_offsets, int32_t dtype,
                      int64_t N, int64_t K, void* W_out) {
  int64_t B = orc_tile_blocks(N), S = orc_tile_ksteps(K);
  int eb = elem_bytes(dtype);
  int64_t G = tile_group_cols(dtype);
  memset(W_out, 0, (size_t)(N * K * eb));
  for (int64_t b = 0; b < B; ++b) {
    for (int64_t s = 0; s < S; ++s) {
      int64_t t = b * S + s;
      int64_t c = tile_offsets[t];
      for (int64_t g = 0; g < 32 / G; ++g) {
        for (int64_t r = 0; r < 16; ++r) {
          for (int64_t j = G * g; j < G * g + G; ++j) {
            if ((bitmask_t[t * 16 + r] >> j) & 1u) {
              int64_t n = 16 * b + r, k = 32 * s + j;
              memcpy((char*)W_out + (n * K + k) * eb, (const char*)values_t + c * eb, (size_t)eb);
              ++c;
            }
          }
        }
      }
    }
  }
}

/* Decode one row of the packed matrix into binary64 (zeros where not kept). */
static void expand_row_f64(const uint32_t* bitmask, const void* values, const int32_t* row_offsets,
                           int32_t dtype, int64_t K, int64_t n, double* out) {
  int64_t words = orc_words_per_row(K);
  int64_t c = row_offsets[n];
  for (int64_t k = 0; k < K; ++k) {
    if ((bitmask[n * words + k / 32] >> (k % 32)) & 1u) {
      out[k] = elem_to_f64(values, c, dtype);
      ++c;
    } else {
      out[k] = 0.0;
    }
  }
}

static void set_threads(int nthreads) {
#ifdef _OPENMP
  if (nthreads > 0) omp_set_num_threads(nthreads);
#else
  (void)nthreads;
#endif
}

int orc_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* ---------------------------------------------------------- fp linear */

/* Y[m][n] = sum_k X[m][k] * D[n][k], D the decoded packed weight, binary64,
 * k summed in ascending order.  X holds fp16 or bf16 payloads ([M][K]);
 * Y is [M][N]. */
void orc_linear_f64(const uint16_t* X, int64_t M, int64_t K, int32_t dtype,
                    const uint32_t* bitmask, const uint16_t* values, const int32_t* row_offsets,
                    int64_t N, double* Y, int nthreads) {
  set_threads(nthreads);
  double* Xd = (double*)malloc((size_t)(M * K) * sizeof(double));
  for (int64_t i = 0; i < M * K; ++i) Xd[i] = elem_to_f64(X, i, dtype);
#pragma omp parallel
  {
    double* Dn = (double*)malloc((size_t)K * sizeof(double));
#pragma omp for schedule(dynamic, 4)
    for (int64_t n = 0; n < N; ++n) {
      expand_row_f64(bitmask, values, row_offsets, dtype, K, n, Dn);
      for (int64_t m = 0; m < M; ++m) {
        double s = 0.0;
        for (int64_t k = 0; k < K; ++k) s += Xd[m * K + k] * Dn[k];
        Y[m * N + n] = s;
      }
    }
    free(Dn);
  }
  free(Xd);
}

/* The same definition evaluated only at the listed (m, n) output positions. */
void orc_linear_f64_pairs(const uint16_t* X, int64_t M, int64_t K, int32_t dtype,
                          const uint32_t* bitmask, const uint16_t* values, const int32_t* row_offsets,
                          int64_t N, const int64_t* ms, const int64_t* ns, int64_t count, double* out,
                          int nthreads) {
  (void)M; (void)N;
  set_threads(nthreads);
#pragma omp parallel
  {
    double* Dn = (double*)malloc((size_t)K * sizeof(double));
#pragma omp for schedule(dynamic, 16)
    for (int64_t i = 0; i < count; ++i) {
      expand_row_f64(bitmask, values, row_offsets, dtype, K, ns[i], Dn);
      double s = 0.0;
      for (int64_t k = 0; k < K; ++k) s += elem_to_f64(X, ms[i] * K + k, dtype) * Dn[k];
      out[i] = s;
    }
    free(Dn);
  }
}

/* Dense reference: Y[m][n] = sum_k X[m][k] * W[n][k] in binary64, W dense [N][K]. */
void orc_dense_f64(const uint16_t* X, int64_t M, int64_t K, int32_t dtype, const uint16_t* W, int64_t N,
                   double* Y, int nthreads) {
  set_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 4)
  for (int64_t n = 0; n < N; ++n) {
    for (int64_t m = 0; m < M; ++m) {
      double s = 0.0;
      for (int64_t k = 0; k < K; ++k) s += elem_to_f64(X, m * K + k, dtype) * elem_to_f64(W, n * K + k, dtype);
      Y[m * N + n] = s;
    }
  }
}

/* ---------------------------------------------------------- int8 linear */

/* Dequantisation of one accumulator, binary32, no fused multiply-add. */
uint16_t orc_dequant_f16(int32_t acc, float sx, float sw) {
  volatile float a = (float)acc;      /* int32 -> binary32, round to nearest even */
  volatile float t = a * sx;
  volatile float y = t * sw;
  return orc_f32_to_f16(y);
}

/* acc[m][n] = sum over kept k of Xq[m][k] * Wq[n][k] (exact integers);
 * Y[m][n] = dequant(acc, sx[m], sw[n]) as fp16 bits.  Returns 0, or -1 if an
 * accumulator leaves the int32 range (it cannot at the layer shapes). */
int orc_linear_i8(const int8_t* Xq, const float* sx, int64_t M, int64_t K,
                  const uint32_t* bitmask, const int8_t* values, const int32_t* row_offsets,
                  const float* sw, int64_t N, int32_t* acc, uint16_t* Y, int nthreads) {
  int64_t words = orc_words_per_row(K);
  int bad = 0;
  set_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 4) reduction(| : bad)
  for (int64_t n = 0; n < N; ++n) {
    for (int64_t m = 0; m < M; ++m) {
      int64_t s = 0;
      int64_t c = row_offsets[n];
      for (int64_t k = 0; k < K; ++k) {
        if ((bitmask[n * words + k / 32] >> (k % 32)) & 1u) {
          s += (int64_t)Xq[m * K + k] * (int64_t)values[c];
          ++c;
        }
      }
      if (s > INT32_MAX || s < INT32_MIN) bad = 1;
      if (acc) acc[m * N + n] = (int32_t)s;
      if (Y) Y[m * N + n] = orc_dequant_f16((int32_t)s, sx[m], sw[n]);
    }
  }
  return bad ? -1 : 0;
}

/* Dense int8 reference with the same epilogue (W dense [N][K]). */
int orc_dense_i8(const int8_t* Xq, const float* sx, int64_t M, int64_t K, const int8_t* Wq,
                 const float* sw, int64_t N, int32_t* acc, uint16_t* Y, int nthreads) {
  int bad = 0;
  set_threads(nthreads);
#pragma omp parallel for schedule(dynamic, 4) reduction(| : bad)
  for (int64_t n = 0; n < N; ++n) {
    for (int64_t m = 0; m < M; ++m) {
      int64_t s = 0;
      for (int64_t k = 0; k < K; ++k) s += (int64_t)Xq[m * K + k] * (int64_t)Wq[n * K + k];
      if (s > INT32_MAX || s < INT32_MIN) bad = 1;
      if (acc) acc[m * N + n] = (int32_t)s;
      if (Y) Y[m * N + n] = orc_dequant_f16((int32_t)s, sx[m], sw[n]);
    }
  }
  return bad ? -1 : 0;
}

/* Per-token activation quantisation for the sparse-quantized path (section
 * 3.4 quantises activations to int8; the reading taken: symmetric, one scale
 * per row, binary32).  For each row m of X (fp16 or bf16 payload bits):
 *   amax = max over k of |x|,  scale = amax / 127 (1 when amax is 0),
 *   code = clamp(round-half-to-even(x / scale), -127, 127),
 * each division rounded to binary32. */
void orc_quantize_rows_i8(const uint16_t* X, int32_t dtype, int64_t M, int64_t K, int8_t* Xq, float* sx) {
  for (int64_t m = 0; m < M; ++m) {
    float amax = 0.0f;
    for (int64_t k = 0; k < K; ++k) {
      const float a = fabsf((float)elem_to_f64(X, m * K + k, dtype));   /* fp16/bf16 -> binary32 is exact */
      if (a > amax) amax = a;
    }
    volatile float scale = amax / 127.0f;
    if (amax == 0.0f) scale = 1.0f;
    sx[m] = scale;
    for (int64_t k = 0; k < K; ++k) {
      volatile float r = (float)elem_to_f64(X, m * K + k, dtype) / scale;
      float q = nearbyintf(r);                                          /* default mode: to nearest, ties even */
      if (q > 127.0f) q = 127.0f;
      if (q < -127.0f) q = -127.0f;
      Xq[m * K + k] = (int8_t)q;
    }
  }
}

/* Element-wise helpers exposed for the oracle's own checks. */
void orc_f16_to_f64_array(const uint16_t* in, int64_t n, double* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_f16_to_f64(in[i]);
}
void orc_bf16_to_f64_array(const uint16_t* in, int64_t n, double* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_bf16_to_f64(in[i]);
}
void orc_f32_to_f16_array(const float* in, int64_t n, uint16_t* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_f32_to_f16(in[i]);
}
void orc_dequant_f16_array(const int32_t* acc, const float* sx, const float* sw, int64_t n, uint16_t* out) {
  for (int64_t i = 0; i < n; ++i) out[i] = orc_dequant_f16(acc[i], sx[i], sw[i]);
}
