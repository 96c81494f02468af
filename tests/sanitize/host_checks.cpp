// Sanitizer driver for the host side of libspl (test infrastructure).  Built
// with the entry points' translation unit under -fsanitize=address,undefined
// (host code only), it calls every entry point with arguments that the host
// checks must reject before any HIP call, and every size function at its
// limits, so that an overflow in the size arithmetic or an out-of-bounds read
// in the checks aborts the run.  No GPU is needed: nothing here reaches a
// launch.  Prints "ok <checks>" and exits 0, or names the first failed check.
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <limits>

#include "spl.h"

static int checks = 0, failed = 0;

static void expect(bool ok, const char* what, int line) {
  ++checks;
  if (!ok && !failed) fprintf(stderr, "FAIL line %d: %s\n", line, what);
  failed += ok ? 0 : 1;
}
#define EXPECT(c) expect((c), #c, __LINE__)
#define REJECTS(call) expect((call) != SPL_OK, #call, __LINE__)

static const int64_t kBig = std::numeric_limits<int64_t>::max();
static const int64_t kMin = std::numeric_limits<int64_t>::min();

// Fake, suitably aligned addresses: never dereferenced by the host checks.
static void* at(uintptr_t a) { return reinterpret_cast<void*>(a); }

static spl_matrix view(int64_t N, int64_t K, int32_t dtype, int32_t layout, int64_t nnz) {
  spl_matrix m;
  memset(&m, 0, sizeof m);
  m.rows = N, m.cols = K, m.dtype = dtype, m.layout = layout, m.nnz = nnz;
  m.bitmask = static_cast<const uint32_t*>(at(0x10000));
  m.values = at(0x20000);
  m.row_offsets = static_cast<const int32_t*>(at(0x30000));
  m.tile_offsets = static_cast<const int32_t*>(at(0x40000));
  m.values_bytes = spl_values_bytes(dtype == SPL_I4 ? SPL_I4 : dtype, nnz);
  return m;
}

int main() {
  const int64_t dims[] = {kMin, -1, 0, 1, 15, 16, 17, 4096, 11008, (1ll << 31) - 1, 1ll << 31, 1ll << 40, kBig};
  const int32_t dtypes[] = {-1, 0, SPL_F16, SPL_BF16, SPL_I8, SPL_I4, 99};

  // size functions at their limits: no overflow, and no result past the documented form
  for (int32_t d : dtypes)
    for (int64_t n : dims) {
      const int64_t b = spl_values_bytes(d, n);
      EXPECT(b == 0 || (b >= 16 && b % 16 == 0 && b <= 2 * n + 48));
    }
  for (int64_t n : dims) {
    const int64_t b = spl_int4_values_bytes(n);
    EXPECT(b == -1 || b == 0 || (b >= 16 && b <= n / 2 + 48));
  }
  for (int64_t a : dims)
    for (int64_t c : dims) {
      const int64_t t = spl_tile16_count(a, c);
      EXPECT(t >= 0);
      for (int64_t m : dims) {
        const int64_t w = spl_sparse_weight_grad_workspace_bytes(m, a, c);
        EXPECT(w >= -1);
        const int64_t p = spl_transpose_perm_workspace_bytes(a, c, m);
        EXPECT(p >= -1);
      }
    }
  EXPECT(spl_magnitude_mask_workspace_bytes() > 0);
  EXPECT(spl_sparse_linear_expanded_workspace_bytes(nullptr) == -1);
  for (int s = -2; s < 8; ++s) EXPECT(spl_status_string(s) != nullptr);
  EXPECT(spl_version() > 0);

  // matrix views: every field at its limits
  for (int64_t N : dims)
    for (int64_t K : dims)
      for (int32_t d : dtypes)
        for (int32_t layout : {-1, (int)SPL_LAYOUT_ROWS, (int)SPL_LAYOUT_TILE16, 7})
          for (int64_t nnz : {kMin, (int64_t)-1, (int64_t)0, (int64_t)1, ((int64_t)1 << 31) - 1, (int64_t)1 << 31, kBig}) {
            spl_matrix m = view(N, K, d, layout, nnz);
            const spl_status st = spl_check_matrix(&m);
            const bool sane = N >= 1 && K >= 1 && N < (1ll << 31) && K < (1ll << 31) && nnz >= 0 &&
                              nnz < (1ll << 31) && d >= SPL_F16 && d <= SPL_I8 &&
                              (layout == SPL_LAYOUT_ROWS || layout == SPL_LAYOUT_TILE16);
            if (!sane) EXPECT(st != SPL_OK);
            const int64_t wsb = spl_sparse_linear_expanded_workspace_bytes(&m);
            EXPECT((st == SPL_OK) == (wsb >= 0));
            if (st == SPL_OK) EXPECT(wsb >= (d == SPL_I8 ? 1 : 2) * N * K && wsb % 256 == 0);
            m.values_bytes = -1;
            EXPECT(spl_check_matrix(&m) != SPL_OK);
          }
  REJECTS(spl_check_matrix(nullptr));
  REJECTS(spl_validate(nullptr, nullptr));

  spl_matrix bad = view(64, 64, SPL_BF16, SPL_LAYOUT_TILE16, kBig);   // fails spl_check_matrix
  spl_matrix i8bad = view(64, 64, SPL_I8, SPL_LAYOUT_TILE16, -1);
  spl_matrix rows = view(64, 64, SPL_BF16, SPL_LAYOUT_ROWS, 10);
  spl_matrix i4 = view(64, 64, SPL_I4, SPL_LAYOUT_TILE16, 10);
  void* X = at(0x50000);
  void* Y = at(0x60000);
  void* odd = at(0x50002);
  const float* sc = static_cast<const float*>(at(0x70000));
  const int8_t* q = static_cast<const int8_t*>(at(0x80000));

  REJECTS(spl_read_probe(nullptr, 16, static_cast<uint32_t*>(Y), nullptr));
  REJECTS(spl_read_probe(X, kBig, nullptr, nullptr));
  REJECTS(spl_read_probe(X, 15, static_cast<uint32_t*>(Y), nullptr));
  REJECTS(spl_retile16(&bad, static_cast<uint32_t*>(Y), X, static_cast<int32_t*>(Y), nullptr));
  REJECTS(spl_retile16(&rows, nullptr, X, static_cast<int32_t*>(Y), nullptr));
  for (int64_t N : dims)
    for (int64_t K : dims) {
      int64_t nnz = 0;
      REJECTS(spl_pack_count(X, SPL_BF16, nullptr, N, K, 9, static_cast<int32_t*>(Y), &nnz, nullptr));
      REJECTS(spl_pack_sparse(X, SPL_BF16, nullptr, N, K, SPL_LAYOUT_TILE16, static_cast<int32_t*>(Y), nullptr, Y,
                              nullptr));
      REJECTS(spl_magnitude_mask(X, SPL_I8, N, K, 0, static_cast<uint8_t*>(Y), Y, nullptr));
      REJECTS(spl_magnitude_mask_noalloc(X, SPL_BF16, N, K, -1, static_cast<uint8_t*>(Y), nullptr));
      REJECTS(spl_dense_linear(X, 1, nullptr, SPL_BF16, N, K, Y, nullptr));
      REJECTS(spl_dense_linear_int8(q, sc, 1, q, nullptr, N, K, Y, nullptr, nullptr));
      if (N > 0 && K > 0) REJECTS(spl_transpose16(at(0x50001), N, K, Y, nullptr));   // misaligned source
    }
  REJECTS(spl_unpack(&bad, Y, nullptr));
  REJECTS(spl_unpack(&rows, odd, nullptr));
  for (int64_t M : dims) {
    if (M != 0) REJECTS(spl_sparse_linear(odd, M, &rows, Y, nullptr));
    REJECTS(spl_sparse_linear(X, M, &bad, Y, nullptr));
    REJECTS(spl_sparse_linear_ex(X, M, &bad, Y, 77, nullptr));
    REJECTS(spl_sparse_linear_expanded(X, M, &bad, Y, Y, nullptr));
    REJECTS(spl_sparse_linear_expanded(X, M, &rows, Y, nullptr, nullptr));
    REJECTS(spl_sparse_linear_int8_expanded(q, sc, M, &i8bad, sc, Y, nullptr, Y, nullptr));
    REJECTS(spl_sparse_linear_int8_expanded(q, sc, M, &rows, sc, Y, nullptr, nullptr, nullptr));
    REJECTS(spl_sparse_linear_silu_mul(X, M, &bad, &bad, Y, SPL_ALGO_AUTO, nullptr));
    REJECTS(spl_sparse_linear_int8(q, sc, M, &i8bad, sc, Y, nullptr, nullptr));
    REJECTS(spl_sparse_linear_int4(q, sc, M, &rows, sc, Y, nullptr, nullptr));
    REJECTS(spl_quantize_rows_i8(X, 42, M, 64, const_cast<int8_t*>(q), const_cast<float*>(sc), nullptr));
    REJECTS(spl_sparse_weight_grad(X, X, M, &bad, Y, Y, nullptr));
    REJECTS(spl_sparse_input_grad(X, M, &bad, Y, Y, nullptr));
    {
      const spl_weight_grad_task wt[2] = {{X, X, &bad, Y}, {X, X, &rows, Y}};
      REJECTS(spl_sparse_weight_grad_group(wt, 2, M, Y, nullptr));
      REJECTS(spl_sparse_weight_grad_group(wt, 0, M, Y, nullptr));
    }
    if (M != 0) REJECTS(spl_sparse_input_grad(X, M, &rows, Y, Y, nullptr));
    EXPECT(spl_sparse_input_grad_workspace_bytes(M, &bad) == -1);
    REJECTS(spl_dense_linear_ex(X, M, X, SPL_BF16, 64, 64, Y, 77, nullptr));
  }
  REJECTS(spl_pack_int4(&i4, static_cast<uint8_t*>(Y), nullptr, nullptr));
  REJECTS(spl_pack_int4(&bad, static_cast<uint8_t*>(Y), nullptr, nullptr));
  REJECTS(spl_sparse_sgd_update(&bad, X, 0.1f, nullptr));
  REJECTS(spl_gather_tiled(X, &bad, Y, nullptr));
  REJECTS(spl_transpose_perm(&bad, &bad, static_cast<int32_t*>(Y), Y, nullptr));
  REJECTS(spl_permute_values(X, nullptr, 10, Y, nullptr));
  REJECTS(spl_permute_values(X, static_cast<const int32_t*>(Y), kBig, Y, nullptr));

  // grouped launches: counts out of range, null arrays, one bad task among good ones
  spl_sparse_task st[SPL_MAX_GROUP + 1];
  spl_dense_task dt[SPL_MAX_GROUP + 1];
  spl_int8_task it[SPL_MAX_GROUP + 1];
  spl_dense_int8_task dit[SPL_MAX_GROUP + 1];
  spl_matrix ok_view = view(64, 64, SPL_BF16, SPL_LAYOUT_TILE16, 10);
  spl_matrix ok_i8 = view(64, 64, SPL_I8, SPL_LAYOUT_TILE16, 10);
  for (int i = 0; i <= SPL_MAX_GROUP; ++i) {
    st[i] = spl_sparse_task{X, &ok_view, Y};
    dt[i] = spl_dense_task{X, X, 64, 64, Y};
    it[i] = spl_int8_task{q, sc, &ok_i8, sc, Y, nullptr};
    dit[i] = spl_dense_int8_task{q, sc, q, sc, 64, 64, Y, nullptr};
  }
  for (int32_t count : {-1, 0, (int)SPL_MAX_GROUP + 1, 1 << 30}) {
    REJECTS(spl_sparse_linear_group(st, count, 1, SPL_ALGO_AUTO, nullptr));
    REJECTS(spl_dense_linear_group(dt, count, 1, SPL_BF16, SPL_ALGO_AUTO, nullptr));
    REJECTS(spl_sparse_linear_int8_group(it, count, 1, nullptr));
    REJECTS(spl_dense_linear_int8_group(dit, count, 1, nullptr));
  }
  REJECTS(spl_sparse_linear_group(nullptr, 2, 1, SPL_ALGO_AUTO, nullptr));
  REJECTS(spl_dense_linear_group(nullptr, 2, 1, SPL_BF16, SPL_ALGO_AUTO, nullptr));
  REJECTS(spl_sparse_linear_int8_group(nullptr, 2, 1, nullptr));
  REJECTS(spl_dense_linear_int8_group(nullptr, 2, 1, nullptr));
  st[SPL_MAX_GROUP - 1].W = &bad;
  dt[SPL_MAX_GROUP - 1].K = kBig;
  it[SPL_MAX_GROUP - 1].Wq = &i8bad;
  dit[SPL_MAX_GROUP - 1].N = kMin;
  REJECTS(spl_sparse_linear_group(st, SPL_MAX_GROUP, 1, SPL_ALGO_AUTO, nullptr));
  REJECTS(spl_dense_linear_group(dt, SPL_MAX_GROUP, 1, SPL_BF16, SPL_ALGO_AUTO, nullptr));
  REJECTS(spl_sparse_linear_int8_group(it, SPL_MAX_GROUP, 1, nullptr));
  REJECTS(spl_dense_linear_int8_group(dit, SPL_MAX_GROUP, 1, nullptr));

  if (failed) return 1;
  printf("ok %d\n", checks);
  return 0;
}
