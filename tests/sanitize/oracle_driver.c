/* Sanitizer driver for the CPU oracle (test infrastructure).  Built together
 * with oracle/spl_oracle.c under -fsanitize=address,undefined, it runs every
 * oracle routine on small ragged shapes (one row or column, K not a multiple
 * of 32, nothing kept, everything kept, no mask) so that any out-of-bounds
 * access or undefined operation aborts the run, and it cross-checks the
 * routines against each other:
 *   unpack(pack(W, mask)) == W . mask in both layouts (bit for bit);
 *   the sparse products == the dense products of the unpacked matrix;
 *   the sampled products == the full ones.
 * Prints "ok <cases>" and exits 0, or names the failing case and exits 1. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int64_t orc_words_per_row(int64_t K);
int64_t orc_pack_nnz(const void* W, int32_t dtype, const uint8_t* mask, int64_t N, int64_t K);
void orc_pack(const void* W, int32_t dtype, const uint8_t* mask, int64_t N, int64_t K, uint32_t* bitmask,
              void* values, int32_t* row_offsets);
void orc_unpack(const uint32_t* bitmask, const void* values, const int32_t* row_offsets, int32_t dtype, int64_t N,
                int64_t K, void* W_out);
int64_t orc_tile_blocks(int64_t N);
int64_t orc_tile_ksteps(int64_t K);
void orc_pack_tiled(const void* W, int32_t dtype, const uint8_t* mask, int64_t N, int64_t K, uint32_t* bitmask_t,
                    void* values_t, int32_t* tile_offsets);
void orc_unpack_tiled(const uint32_t* bitmask_t, const void* values_t, const int32_t* tile_offsets, int32_t dtype,
                      int64_t N, int64_t K, void* W_out);
void orc_linear_f64(const uint16_t* X, int64_t M, int64_t K, int32_t dtype, const uint32_t* bitmask,
                    const uint16_t* values, const int32_t* row_offsets, int64_t N, double* Y, int nthreads);
void orc_linear_f64_pairs(const uint16_t* X, int64_t M, int64_t K, int32_t dtype, const uint32_t* bitmask,
                          const uint16_t* values, const int32_t* row_offsets, int64_t N, const int64_t* ms,
                          const int64_t* ns, int64_t count, double* out, int nthreads);
void orc_dense_f64(const uint16_t* X, int64_t M, int64_t K, int32_t dtype, const uint16_t* W, int64_t N, double* Y,
                   int nthreads);
int orc_linear_i8(const int8_t* Xq, const float* sx, int64_t M, int64_t K, const uint32_t* bitmask,
                  const int8_t* values, const int32_t* row_offsets, const float* sw, int64_t N, int32_t* acc,
                  uint16_t* Y, int nthreads);
int orc_dense_i8(const int8_t* Xq, const float* sx, int64_t M, int64_t K, const int8_t* Wq, const float* sw,
                 int64_t N, int32_t* acc, uint16_t* Y, int nthreads);
void orc_quantize_rows_i8(const uint16_t* X, int32_t dtype, int64_t M, int64_t K, int8_t* Xq, float* sx);

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static uint32_t next_u32(void) {       /* xorshift64*: test data only */
  rng_state ^= rng_state >> 12;
  rng_state ^= rng_state << 25;
  rng_state ^= rng_state >> 27;
  return (uint32_t)((rng_state * 0x2545F4914F6CDD1Dull) >> 32);
}

/* A finite fp16/bf16 payload of moderate magnitude (exponent bits kept away
 * from the all-ones pattern). */
static uint16_t finite16(int dtype) {
  const uint32_t r = next_u32();
  if (dtype == 1) return (uint16_t)((r & 0x8000u) | (((r >> 16) % 20u + 5u) << 10) | (r & 0x3FFu));
  return (uint16_t)((r & 0x8000u) | (((r >> 16) % 40u + 100u) << 7) | (r & 0x7Fu));
}

static void* xmalloc(size_t n) {       /* never zero bytes, so every case gets a real block */
  void* p = malloc(n ? n : 1);
  if (!p) abort();
  return p;
}

static int fail(const char* what, int dtype, int64_t N, int64_t K, int mode) {
  fprintf(stderr, "FAIL %s dtype=%d N=%lld K=%lld mode=%d\n", what, dtype, (long long)N, (long long)K, mode);
  return 1;
}

/* mode 0: random mask; 1: nothing kept; 2: everything kept; 3: no mask (W != 0). */
static int run_case(int dtype, int64_t N, int64_t K, int mode) {
  const int eb = dtype == 3 ? 1 : 2;
  const int64_t n = N * K, words = orc_words_per_row(K);
  const int64_t B = orc_tile_blocks(N), S = orc_tile_ksteps(K);
  unsigned char* W = xmalloc((size_t)(n * eb));
  uint8_t* mask = xmalloc((size_t)n);
  for (int64_t i = 0; i < n; ++i) {
    if (eb == 1) {
      ((int8_t*)W)[i] = (int8_t)((int)(next_u32() % 255u) - 127);
    } else {
      ((uint16_t*)W)[i] = (next_u32() % 5u == 0u) ? 0 : finite16(dtype);
    }
    mask[i] = mode == 0 ? (uint8_t)(next_u32() % 10u < 3u) : mode == 2 ? 1 : 0;
  }
  const uint8_t* mk = mode == 3 ? NULL : mask;
  const int64_t nnz = orc_pack_nnz(W, dtype, mk, N, K);
  int bad = 0;

  /* the masked dense matrix, as the definition gives it */
  unsigned char* WM = xmalloc((size_t)(n * eb));
  for (int64_t i = 0; i < n; ++i) {
    int keep;
    if (mk) keep = mk[i] != 0;
    else keep = eb == 1 ? ((int8_t*)W)[i] != 0 : (((uint16_t*)W)[i] & 0x7FFFu) != 0;
    if (eb == 1) ((int8_t*)WM)[i] = keep ? ((int8_t*)W)[i] : 0;
    else ((uint16_t*)WM)[i] = keep ? ((uint16_t*)W)[i] : 0;
  }

  uint32_t* bm = xmalloc((size_t)(N * words) * 4);
  void* vals = xmalloc((size_t)(nnz * eb));
  int32_t* offs = xmalloc((size_t)(N + 1) * 4);
  orc_pack(W, dtype, mk, N, K, bm, vals, offs);
  if (offs[N] != nnz) bad |= fail("row nnz", dtype, N, K, mode);
  unsigned char* back = xmalloc((size_t)(n * eb));
  orc_unpack(bm, vals, offs, dtype, N, K, back);
  if (memcmp(back, WM, (size_t)(n * eb)) != 0) bad |= fail("row round trip", dtype, N, K, mode);

  uint32_t* bmt = xmalloc((size_t)(B * S * 16) * 4);
  void* valt = xmalloc((size_t)(nnz * eb));
  int32_t* offt = xmalloc((size_t)(B * S + 1) * 4);
  orc_pack_tiled(W, dtype, mk, N, K, bmt, valt, offt);
  if (offt[B * S] != nnz) bad |= fail("tile nnz", dtype, N, K, mode);
  memset(back, 0xA5, (size_t)(n * eb));
  orc_unpack_tiled(bmt, valt, offt, dtype, N, K, back);
  if (memcmp(back, WM, (size_t)(n * eb)) != 0) bad |= fail("tile round trip", dtype, N, K, mode);

  const int64_t M = 3;
  if (eb == 2) {
    uint16_t* X = xmalloc((size_t)(M * K) * 2);
    for (int64_t i = 0; i < M * K; ++i) X[i] = finite16(dtype);
    double* Ys = xmalloc((size_t)(M * N) * 8);
    double* Yd = xmalloc((size_t)(M * N) * 8);
    orc_linear_f64(X, M, K, dtype, bm, vals, offs, N, Ys, 1);
    orc_dense_f64(X, M, K, dtype, (const uint16_t*)WM, N, Yd, 1);
    for (int64_t i = 0; i < M * N; ++i)
      if (Ys[i] != Yd[i]) { bad |= fail("sparse vs dense f64", dtype, N, K, mode); break; }
    int64_t ms[4] = {0, M - 1, 1, 0}, ns[4] = {0, N - 1, N / 2, N - 1};
    double pr[4];
    orc_linear_f64_pairs(X, M, K, dtype, bm, vals, offs, N, ms, ns, 4, pr, 1);
    for (int i = 0; i < 4; ++i)
      if (pr[i] != Ys[ms[i] * N + ns[i]]) { bad |= fail("pairs vs full", dtype, N, K, mode); break; }
    int8_t* Xq = xmalloc((size_t)(M * K));
    float* sx = xmalloc((size_t)M * 4);
    orc_quantize_rows_i8(X, dtype, M, K, Xq, sx);
    for (int64_t i = 0; i < M * K; ++i)
      if (Xq[i] < -127 || Xq[i] > 127) { bad |= fail("quantised code range", dtype, N, K, mode); break; }
    free(X), free(Ys), free(Yd), free(Xq), free(sx);
  } else {
    int8_t* Xq = xmalloc((size_t)(M * K));
    float* sx = xmalloc((size_t)M * 4);
    float* sw = xmalloc((size_t)N * 4);
    for (int64_t i = 0; i < M * K; ++i) Xq[i] = (int8_t)((int)(next_u32() % 255u) - 127);
    for (int64_t i = 0; i < M; ++i) sx[i] = 0.01f * (float)(1 + i);
    for (int64_t i = 0; i < N; ++i) sw[i] = 0.002f * (float)(1 + i % 7);
    int32_t* as = xmalloc((size_t)(M * N) * 4);
    int32_t* ad = xmalloc((size_t)(M * N) * 4);
    uint16_t* ys = xmalloc((size_t)(M * N) * 2);
    uint16_t* yd = xmalloc((size_t)(M * N) * 2);
    const int e1 = orc_linear_i8(Xq, sx, M, K, bm, (const int8_t*)vals, offs, sw, N, as, ys, 1);
    const int e2 = orc_dense_i8(Xq, sx, M, K, (const int8_t*)WM, sw, N, ad, yd, 1);
    if (e1 || e2) bad |= fail("int8 accumulator range", dtype, N, K, mode);
    if (memcmp(as, ad, (size_t)(M * N) * 4) != 0 || memcmp(ys, yd, (size_t)(M * N) * 2) != 0)
      bad |= fail("sparse vs dense int8", dtype, N, K, mode);
    free(Xq), free(sx), free(sw), free(as), free(ad), free(ys), free(yd);
  }
  free(W), free(mask), free(WM), free(bm), free(vals), free(offs), free(back), free(bmt), free(valt), free(offt);
  return bad;
}

int main(void) {
  static const int64_t Ns[] = {1, 3, 16, 17, 33};
  static const int64_t Ks[] = {1, 8, 31, 32, 33, 64, 100};
  int bad = 0, cases = 0;
  for (int dtype = 1; dtype <= 3; ++dtype)
    for (size_t a = 0; a < sizeof Ns / sizeof Ns[0]; ++a)
      for (size_t b = 0; b < sizeof Ks / sizeof Ks[0]; ++b)
        for (int mode = 0; mode < 4; ++mode, ++cases) bad |= run_case(dtype, Ns[a], Ks[b], mode);
  if (bad) return 1;
  printf("ok %d\n", cases);
  return 0;
}
