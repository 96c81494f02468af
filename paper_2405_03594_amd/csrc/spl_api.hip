// extern "C" entry points of libspl: argument checks on the host, then
// launches on the caller's stream.  No entry point allocates device memory.
#include <stdint.h>

#include <atomic>
#include <mutex>

#include "spl.h"
#include "spl_common.h"

namespace {

constexpr int64_t kMaxDim = (int64_t)1 << 31;        // N, K, M < 2^31
constexpr int64_t kMaxElems = (int64_t)1 << 40;      // N * K, M * K, M * N
constexpr int64_t kDecodeMaxM = 32;
constexpr int64_t kGatedDecodeMaxM = 16;           // the paired decode kernel holds one 16-row batch tile
// The decode kernels address the activations [M][K] with 32-bit byte offsets.
bool decode_fits(int64_t M, int64_t K) { return M <= kDecodeMaxM && 2 * M * K <= ((int64_t)1 << 31); }

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

bool dims_ok(int64_t a, int64_t b) {
  return a >= 1 && b >= 1 && a < kMaxDim && b < kMaxDim && a <= kMaxElems / b;
}

bool fp_dtype(int32_t d) { return d == SPL_F16 || d == SPL_BF16; }
bool any_dtype(int32_t d) { return d == SPL_F16 || d == SPL_BF16 || d == SPL_I8; }

spl_status launched(hipError_t e) {
  if (e == hipSuccess) return SPL_OK;
  return e == hipErrorNotSupported ? SPL_ERR_UNSUPPORTED : SPL_ERR_DEVICE;
}

// Shared checks of an activation/output pair for a [M][K] x [N][K]^T product.
spl_status check_xy(const void* X, int64_t M, int64_t K, int64_t N, const void* Y) {
  if (M < 0) return SPL_ERR_INVALID_ARG;
  if (M == 0) return SPL_OK;
  if (!X || !Y) return SPL_ERR_INVALID_ARG;
  if (!dims_ok(M, K) || !dims_ok(M, N)) return SPL_ERR_INVALID_ARG;
  if (!aligned(X, 16) || !aligned(Y, 16)) return SPL_ERR_INVALID_ARG;
  return SPL_OK;
}

}  // namespace

extern "C" {

int32_t spl_version(void) { return (1 << 16) | 0; }

const char* spl_status_string(int32_t status) {
  switch (status) {
    case SPL_OK: return "ok";
    case SPL_ERR_INVALID_ARG: return "invalid argument";
    case SPL_ERR_UNSUPPORTED: return "unsupported";
    case SPL_ERR_OVERFLOW: return "overflow: nnz >= 2^31";
    case SPL_ERR_DEVICE: return "HIP runtime error";
  }
  return "unknown status";
}

spl_status spl_read_probe(const void* buf, int64_t bytes, uint32_t* sink, hipStream_t stream) {
  if (!buf || !sink || bytes <= 0 || bytes % 16 != 0 || !aligned(buf, 16) || !aligned(sink, 4))
    return SPL_ERR_INVALID_ARG;
  (void)hipGetLastError();
  return launched(spl::launch_read_probe(buf, bytes, sink, spl::device_cus(), stream));
}

int64_t spl_values_bytes(int32_t dtype, int64_t nnz) {
  if (nnz < 0 || nnz >= kMaxDim) return 0;
  int64_t payload = 0;
  if (dtype == SPL_F16 || dtype == SPL_BF16) payload = 2 * nnz;
  else if (dtype == SPL_I8) payload = nnz;
  else if (dtype == SPL_I4) payload = (nnz + 1) / 2;
  else return 0;
  return (payload + 15) / 16 * 16 + 16;
}

spl_status spl_check_matrix(const spl_matrix* Wc) {
  if (!Wc) return SPL_ERR_INVALID_ARG;
  if (!dims_ok(Wc->rows, Wc->cols)) return SPL_ERR_INVALID_ARG;
  if (!any_dtype(Wc->dtype)) return SPL_ERR_INVALID_ARG;
  if (Wc->layout != SPL_LAYOUT_ROWS && Wc->layout != SPL_LAYOUT_TILE16) return SPL_ERR_INVALID_ARG;
  if (Wc->nnz < 0) return SPL_ERR_INVALID_ARG;
  if (Wc->nnz >= kMaxDim) return SPL_ERR_OVERFLOW;
  if (Wc->nnz > Wc->rows * Wc->cols) return SPL_ERR_INVALID_ARG;
  if (!Wc->bitmask) return SPL_ERR_INVALID_ARG;
  if (Wc->layout == SPL_LAYOUT_ROWS && !Wc->row_offsets) return SPL_ERR_INVALID_ARG;
  if (Wc->layout == SPL_LAYOUT_TILE16 && !Wc->tile_offsets) return SPL_ERR_INVALID_ARG;
  if (!Wc->values || Wc->values_bytes < spl_values_bytes(Wc->dtype, Wc->nnz)) return SPL_ERR_INVALID_ARG;
  if (!aligned(Wc->bitmask, 16)) return SPL_ERR_INVALID_ARG;
  if (Wc->row_offsets && !aligned(Wc->row_offsets, 4)) return SPL_ERR_INVALID_ARG;
  if (Wc->tile_offsets && !aligned(Wc->tile_offsets, 4)) return SPL_ERR_INVALID_ARG;
  if (Wc->values && !aligned(Wc->values, 16)) return SPL_ERR_INVALID_ARG;
  return SPL_OK;
}

int64_t spl_tile16_count(int64_t N, int64_t K) {
  if (!dims_ok(N, K)) return 0;
  return ((N + 15) / 16) * ((K + 31) / 32);
}

spl_status spl_retile16(const spl_matrix* rows_in, uint32_t* bitmask_out, void* values_out,
                        int32_t* tile_offsets_out, hipStream_t stream) {
  const spl_status st = spl_check_matrix(rows_in);
  if (st != SPL_OK) return st;
  if (rows_in->layout != SPL_LAYOUT_ROWS) return SPL_ERR_INVALID_ARG;
  if (!bitmask_out || !tile_offsets_out || !aligned(bitmask_out, 16) || !aligned(tile_offsets_out, 4))
    return SPL_ERR_INVALID_ARG;
  if (rows_in->nnz > 0 && (!values_out || !aligned(values_out, 16))) return SPL_ERR_INVALID_ARG;
  if (values_out && values_out == rows_in->values) return SPL_ERR_INVALID_ARG;
  (void)hipGetLastError();
  return launched(spl::launch_retile16(*rows_in, bitmask_out, values_out, tile_offsets_out, stream));
}

spl_status spl_pack_count(const void* W, int32_t dtype, const uint8_t* mask, int64_t N, int64_t K, int32_t layout,
                          int32_t* offsets, int64_t* h_nnz, hipStream_t stream) {
  if (!W || !offsets || !h_nnz) return SPL_ERR_INVALID_ARG;
  if (!any_dtype(dtype) || !dims_ok(N, K)) return SPL_ERR_INVALID_ARG;
  if (layout != SPL_LAYOUT_ROWS && layout != SPL_LAYOUT_TILE16) return SPL_ERR_INVALID_ARG;
  if (!aligned(W, 16) || !aligned(offsets, 4)) return SPL_ERR_INVALID_ARG;
  const int64_t blocks = layout == SPL_LAYOUT_ROWS ? N : spl::tile_blocks(N) * spl::tile_steps(K);
  (void)hipGetLastError();
  const hipError_t e = layout == SPL_LAYOUT_ROWS ? spl::launch_pack_count(W, dtype, mask, N, K, offsets, stream)
                                                 : spl::launch_pack_count_tiled(W, dtype, mask, N, K, offsets, stream);
  if (e != hipSuccess) return SPL_ERR_DEVICE;
  int32_t total = 0;
  if (hipMemcpyAsync(&total, offsets + blocks, sizeof(int32_t), hipMemcpyDeviceToHost, stream) != hipSuccess)
    return SPL_ERR_DEVICE;
  if (hipStreamSynchronize(stream) != hipSuccess) return SPL_ERR_DEVICE;
  if (total < 0) return SPL_ERR_OVERFLOW;
  *h_nnz = total;
  return SPL_OK;
}

spl_status spl_pack_sparse(const void* W, int32_t dtype, const uint8_t* mask, int64_t N, int64_t K, int32_t layout,
                           const int32_t* offsets, uint32_t* bitmask, void* values, hipStream_t stream) {
  if (!W || !offsets || !bitmask || !values) return SPL_ERR_INVALID_ARG;
  if (!any_dtype(dtype) || !dims_ok(N, K)) return SPL_ERR_INVALID_ARG;
  if (layout != SPL_LAYOUT_ROWS && layout != SPL_LAYOUT_TILE16) return SPL_ERR_INVALID_ARG;
  if (!aligned(W, 16) || !aligned(bitmask, 16) || !aligned(offsets, 4) || !aligned(values, 16))
    return SPL_ERR_INVALID_ARG;
  (void)hipGetLastError();
  if (layout == SPL_LAYOUT_TILE16)
    return launched(spl::launch_pack_scatter_tiled(W, dtype, mask, N, K, offsets, bitmask, values, stream));
  return launched(spl::launch_pack_scatter(W, dtype, mask, N, K, offsets, bitmask, values, stream));
}

// The result word of spl_validate: one per device (each device has its own
// copy of a __device__ variable); its address is looked up once per device.
__device__ uint32_t g_validate_err;

static uint32_t* validate_word() {
  static std::atomic<uint32_t*> addr[spl::kMaxDevices];
  const int dev = spl::current_device();
  if (dev < 0) return nullptr;
  uint32_t* p = addr[dev].load(std::memory_order_acquire);
  if (p) return p;
  void* q = nullptr;
  if (hipGetSymbolAddress(&q, HIP_SYMBOL(g_validate_err)) != hipSuccess || !q) return nullptr;
  addr[dev].store(static_cast<uint32_t*>(q), std::memory_order_release);
  return static_cast<uint32_t*>(q);
}

spl_status spl_validate(const spl_matrix* Wc, hipStream_t stream) {
  const spl_status st = spl_check_matrix(Wc);
  if (st != SPL_OK) return st;
  static std::mutex one_at_a_time;                 // the word is shared: one validation in flight per process
  std::lock_guard<std::mutex> hold(one_at_a_time);
  uint32_t* err = validate_word();
  if (!err) return SPL_ERR_DEVICE;
  (void)hipGetLastError();
  if (spl::launch_validate(*Wc, err, stream) != hipSuccess) return SPL_ERR_DEVICE;
  uint32_t bits = 0;
  if (hipMemcpyAsync(&bits, err, sizeof(bits), hipMemcpyDeviceToHost, stream) != hipSuccess) return SPL_ERR_DEVICE;
  if (hipStreamSynchronize(stream) != hipSuccess) return SPL_ERR_DEVICE;
  return bits ? SPL_ERR_INVALID_ARG : SPL_OK;
}

spl_status spl_unpack(const spl_matrix* Wc, void* W_dense, hipStream_t stream) {
  const spl_status st = spl_check_matrix(Wc);
  if (st != SPL_OK) return st;
  if (!W_dense || !aligned(W_dense, 16)) return SPL_ERR_INVALID_ARG;
  (void)hipGetLastError();
  return launched(spl::launch_unpack(*Wc, W_dense, stream));
}

// Checks of one fp16/bf16 sparse task; *algo is resolved from AUTO.
static spl_status check_sparse_task(const void* X, int64_t M, const spl_matrix* Wc, const void* Y, int32_t* algo) {
  const spl_status st = spl_check_matrix(Wc);
  if (st != SPL_OK) return st;
  if (!fp_dtype(Wc->dtype) || Wc->layout != SPL_LAYOUT_TILE16) return SPL_ERR_UNSUPPORTED;
  if (*algo < SPL_ALGO_AUTO || *algo > SPL_ALGO_PREFILL) return SPL_ERR_INVALID_ARG;
  const spl_status xy = check_xy(X, M, Wc->cols, Wc->rows, Y);
  if (xy != SPL_OK) return xy;
  if (Wc->cols % 8 != 0) return SPL_ERR_UNSUPPORTED;
  if (*algo == SPL_ALGO_AUTO) *algo = decode_fits(M, Wc->cols) ? SPL_ALGO_DECODE : SPL_ALGO_PREFILL;
  if (*algo == SPL_ALGO_DECODE && !decode_fits(M, Wc->cols)) return SPL_ERR_UNSUPPORTED;
  return SPL_OK;
}

static spl_status check_dense_task(const spl_dense_task* t, int64_t M, int32_t dtype, int32_t* algo) {
  if (!t->W || !fp_dtype(dtype) || !dims_ok(t->N, t->K) || !aligned(t->W, 16)) return SPL_ERR_INVALID_ARG;
  if (*algo < SPL_ALGO_AUTO || *algo > SPL_ALGO_PREFILL) return SPL_ERR_INVALID_ARG;
  const spl_status xy = check_xy(t->X, M, t->K, t->N, t->Y);
  if (xy != SPL_OK) return xy;
  if (t->K % 8 != 0) return SPL_ERR_UNSUPPORTED;
  if (*algo == SPL_ALGO_AUTO) *algo = decode_fits(M, t->K) ? SPL_ALGO_DECODE : SPL_ALGO_PREFILL;
  if (*algo == SPL_ALGO_DECODE && !decode_fits(M, t->K)) return SPL_ERR_UNSUPPORTED;
  return SPL_OK;
}

spl_status spl_sparse_linear_ex(const void* X, int64_t M, const spl_matrix* Wc, void* Y, int32_t algo,
                                hipStream_t stream) {
  const spl_sparse_task t{X, Wc, Y};
  return spl_sparse_linear_group(&t, 1, M, algo, stream);
}

int64_t spl_sparse_linear_expanded_workspace_bytes(const spl_matrix* Wc) {
  if (spl_check_matrix(Wc) != SPL_OK) return -1;
  const int64_t eb = Wc->dtype == SPL_I8 ? 1 : 2;
  return (eb * Wc->rows * Wc->cols + 255) / 256 * 256;   // rows, cols < 2^31: far from 2^63
}

spl_status spl_sparse_linear_expanded(const void* X, int64_t M, const spl_matrix* Wc, void* Y, void* workspace,
                                      hipStream_t stream) {
  int32_t algo = SPL_ALGO_PREFILL;
  const spl_status st = check_sparse_task(X, M, Wc, Y, &algo);
  if (st != SPL_OK) return st;
  if (!workspace || !aligned(workspace, 16)) return SPL_ERR_INVALID_ARG;
  if (spl::tile_blocks(Wc->rows) >= kMaxDim) return SPL_ERR_OVERFLOW;
  if (M == 0) return SPL_OK;
  (void)hipGetLastError();
  const spl_status e = launched(spl::launch_unpack(*Wc, workspace, stream));   // the decoded [N][K] matrix
  if (e != SPL_OK) return e;
  return launched(spl::launch_dense_prefill(X, M, workspace, Wc->dtype, Wc->rows, Wc->cols, Y, stream));
}

spl_status spl_sparse_linear_group(const spl_sparse_task* tasks, int32_t count, int64_t M, int32_t algo,
                                   hipStream_t stream) {
  if (!tasks || count < 1 || count > SPL_MAX_GROUP || M < 0) return SPL_ERR_INVALID_ARG;
  int64_t blocks = 0;
  int32_t resolved = algo;
  for (int32_t i = 0; i < count; ++i) {
    if (!tasks[i].W) return SPL_ERR_INVALID_ARG;
    int32_t a = algo;
    const spl_status st = check_sparse_task(tasks[i].X, M, tasks[i].W, tasks[i].Y, &a);
    if (st != SPL_OK) return st;
    if (tasks[i].W->dtype != tasks[0].W->dtype) return SPL_ERR_INVALID_ARG;
    resolved = a;                                      // AUTO depends on M only: the same for every task
    blocks += spl::tile_blocks(tasks[i].W->rows);
  }
  if (blocks >= kMaxDim) return SPL_ERR_OVERFLOW;
  if (M == 0) return SPL_OK;
  (void)hipGetLastError();
  if (resolved == SPL_ALGO_DECODE) return launched(spl::launch_sparse_decode(tasks, count, M, stream));
  for (int32_t i = 0; i < count; ++i) {
    const spl_status st = launched(spl::launch_sparse_prefill(tasks[i].X, M, *tasks[i].W, tasks[i].Y, stream));
    if (st != SPL_OK) return st;
  }
  return SPL_OK;
}

spl_status spl_sparse_linear(const void* X, int64_t M, const spl_matrix* Wc, void* Y, hipStream_t stream) {
  return spl_sparse_linear_ex(X, M, Wc, Y, SPL_ALGO_AUTO, stream);
}

spl_status spl_sparse_linear_silu_mul(const void* X, int64_t M, const spl_matrix* Wgate, const spl_matrix* Wup,
                                      void* Y, int32_t algo, hipStream_t stream) {
  if (!Wgate || !Wup || M < 0) return SPL_ERR_INVALID_ARG;
  int32_t ag = algo, au = algo;
  spl_status st = check_sparse_task(X, M, Wgate, Y, &ag);
  if (st != SPL_OK) return st;
  st = check_sparse_task(X, M, Wup, Y, &au);
  if (st != SPL_OK) return st;
  if (Wup->dtype != Wgate->dtype || Wup->rows != Wgate->rows || Wup->cols != Wgate->cols) return SPL_ERR_INVALID_ARG;
  if (algo == SPL_ALGO_AUTO)
    ag = M <= kGatedDecodeMaxM && decode_fits(M, Wgate->cols) ? SPL_ALGO_DECODE : SPL_ALGO_PREFILL;
  if (ag == SPL_ALGO_DECODE && (M > kGatedDecodeMaxM || !decode_fits(M, Wgate->cols))) return SPL_ERR_UNSUPPORTED;
  if (2 * spl::tile_blocks(Wgate->rows) >= kMaxDim) return SPL_ERR_OVERFLOW;
  if (M == 0) return SPL_OK;
  (void)hipGetLastError();
  if (ag == SPL_ALGO_DECODE) return launched(spl::launch_gated_decode(X, M, *Wgate, *Wup, Y, stream));
  return launched(spl::launch_gated_prefill(X, M, *Wgate, *Wup, Y, stream));
}

int64_t spl_magnitude_mask_workspace_bytes(void) { return 4 * spl::magnitude_mask_workspace_words(); }

spl_status spl_magnitude_mask(const void* W, int32_t dtype, int64_t N, int64_t K, int64_t prune, uint8_t* mask,
                              void* workspace, hipStream_t stream) {
  if (!W || !mask || !workspace || !dims_ok(N, K)) return SPL_ERR_INVALID_ARG;
  if (!fp_dtype(dtype)) return SPL_ERR_UNSUPPORTED;
  if (K % 8 != 0 || N * K >= ((int64_t)1 << 31)) return SPL_ERR_UNSUPPORTED;
  if (prune < 0 || prune > N * K) return SPL_ERR_INVALID_ARG;
  if (!aligned(W, 16) || !aligned(mask, 8) || !aligned(workspace, 16)) return SPL_ERR_INVALID_ARG;
  (void)hipGetLastError();
  return launched(spl::launch_magnitude_mask(static_cast<const uint16_t*>(W), N * K, (uint32_t)prune, mask,
                                             static_cast<uint32_t*>(workspace), stream));
}

// Scratch of spl_magnitude_mask_noalloc: the histogram, the threshold pair and
// the per-chunk tie counts of the pruning kernels.  Each device holds its own
// copy until the process ends.  Host code uses the device address from
// hipGetSymbolAddress (kept per device), never the array's name.
constexpr int64_t kNoallocWords = 34818;
static __device__ __align__(256) uint32_t scratch[kNoallocWords];

static uint32_t* noalloc_scratch() {
  static std::atomic<uint32_t*> addr[spl::kMaxDevices];
  const int dev = spl::current_device();
  if (dev < 0) return nullptr;
  uint32_t* p = addr[dev].load(std::memory_order_acquire);
  if (p) return p;
  void* q = nullptr;
  if (hipGetSymbolAddress(&q, HIP_SYMBOL(scratch)) != hipSuccess || !q) return nullptr;
  addr[dev].store(static_cast<uint32_t*>(q), std::memory_order_release);
  return static_cast<uint32_t*>(q);
}

spl_status spl_magnitude_mask_noalloc(const void* W, int32_t dtype, int64_t N, int64_t K, int64_t prune,
                                      uint8_t* mask, hipStream_t stream) {
  if (spl::magnitude_mask_workspace_words() > kNoallocWords) return SPL_ERR_UNSUPPORTED;   // build mismatch
  if (!W || !mask || !dims_ok(N, K)) return SPL_ERR_INVALID_ARG;
  if (!fp_dtype(dtype)) return SPL_ERR_UNSUPPORTED;
  if (K % 8 != 0 || N * K >= ((int64_t)1 << 31)) return SPL_ERR_UNSUPPORTED;
  if (prune < 0 || prune > N * K) return SPL_ERR_INVALID_ARG;
  if (!aligned(W, 16) || !aligned(mask, 8)) return SPL_ERR_INVALID_ARG;
  uint32_t* ws = noalloc_scratch();
  if (!ws) return SPL_ERR_DEVICE;
  (void)hipGetLastError();
  return launched(spl::launch_magnitude_mask(static_cast<const uint16_t*>(W), N * K, (uint32_t)prune, mask, ws,
                                             stream));
}

spl_status spl_transpose16(const void* src, int64_t R, int64_t C, void* dst, hipStream_t stream) {
  if (R == 0 || C == 0) return (R < 0 || C < 0) ? SPL_ERR_INVALID_ARG : SPL_OK;
  if (!src || !dst || !dims_ok(R, C) || !aligned(src, 2) || !aligned(dst, 2)) return SPL_ERR_INVALID_ARG;
  if ((R + 63) / 64 > 65535) return SPL_ERR_UNSUPPORTED;
  (void)hipGetLastError();
  return launched(spl::launch_transpose16(src, R, C, dst, stream));
}

// A tile-layout fp16/bf16 pattern whose values can be read or written.
static spl_status check_tiled_fp(const spl_matrix* P) {
  const spl_status st = spl_check_matrix(P);
  if (st != SPL_OK) return st;
  if (!fp_dtype(P->dtype) || P->layout != SPL_LAYOUT_TILE16) return SPL_ERR_UNSUPPORTED;
  if (P->nnz > 0 && !P->values) return SPL_ERR_INVALID_ARG;
  return SPL_OK;
}

spl_status spl_gather_tiled(const void* W_dense, const spl_matrix* pattern, void* values_out, hipStream_t stream) {
  const spl_status st = check_tiled_fp(pattern);
  if (st != SPL_OK) return st;
  if (!W_dense || !values_out || !aligned(W_dense, 16) || !aligned(values_out, 2)) return SPL_ERR_INVALID_ARG;
  if (pattern->cols % 8 != 0) return SPL_ERR_UNSUPPORTED;
  if (pattern->nnz == 0) return SPL_OK;
  (void)hipGetLastError();
  return launched(spl::launch_gather_tiled(W_dense, *pattern, values_out, stream));
}

int64_t spl_sparse_weight_grad_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  if (M < 0 || !dims_ok(N, K)) return -1;
  if (M > 0 && (!dims_ok(M, N) || !dims_ok(M, K))) return -1;   // the sizes below stay far from 2^63
  return spl::weight_grad_workspace_bytes(M, N, K);
}

spl_status spl_sparse_weight_grad(const void* dY, const void* X, int64_t M, const spl_matrix* Wc, void* grad_values,
                                  void* workspace, hipStream_t stream) {
  const spl_status st = check_tiled_fp(Wc);
  if (st != SPL_OK) return st;
  if (M < 0 || !grad_values || !aligned(grad_values, 2)) return SPL_ERR_INVALID_ARG;
  if (M == 0) return SPL_ERR_UNSUPPORTED;            // a sum over no tokens: the caller zeroes the gradient
  if (!dY || !X || !workspace || !dims_ok(M, Wc->rows) || !dims_ok(M, Wc->cols)) return SPL_ERR_INVALID_ARG;
  if (!aligned(dY, 2) || !aligned(X, 2) || !aligned(workspace, 256)) return SPL_ERR_INVALID_ARG;
  if (M % 8 != 0 || Wc->cols % 8 != 0 || (M + 63) / 64 > 65535) return SPL_ERR_UNSUPPORTED;
  if (Wc->nnz == 0) return SPL_OK;                   // no kept entry: no gradient to write
  (void)hipGetLastError();
  return launched(spl::launch_weight_grad(dY, X, M, *Wc, grad_values, workspace, stream));
}

spl_status spl_sparse_weight_grad_group(const spl_weight_grad_task* tasks, int32_t count, int64_t M,
                                        void* workspace, hipStream_t stream) {
  if (!tasks || count < 1 || count > SPL_MAX_GROUP) return SPL_ERR_INVALID_ARG;
  for (int32_t i = 0; i < count; ++i) {
    const spl_weight_grad_task& t = tasks[i];
    const spl_status st = check_tiled_fp(t.W);
    if (st != SPL_OK) return st;
    if (t.W->dtype != tasks[0].W->dtype) return SPL_ERR_INVALID_ARG;
    if (M < 0 || !t.grad_values || !aligned(t.grad_values, 2)) return SPL_ERR_INVALID_ARG;
    if (M == 0) return SPL_ERR_UNSUPPORTED;
    if (!t.dY || !t.X || !workspace || !dims_ok(M, t.W->rows) || !dims_ok(M, t.W->cols)) return SPL_ERR_INVALID_ARG;
    if (!aligned(t.dY, 2) || !aligned(t.X, 2) || !aligned(workspace, 256)) return SPL_ERR_INVALID_ARG;
    if (M % 8 != 0 || t.W->cols % 8 != 0 || (M + 63) / 64 > 65535) return SPL_ERR_UNSUPPORTED;
  }
  (void)hipGetLastError();
  return launched(spl::launch_weight_grad_group(tasks, count, M, workspace, stream));
}

int64_t spl_sparse_input_grad_workspace_bytes(int64_t M, const spl_matrix* Wc) {
  if (check_tiled_fp(Wc) != SPL_OK || M < 0) return -1;
  if (M > 0 && (!dims_ok(M, Wc->rows) || !dims_ok(M, Wc->cols))) return -1;
  return spl::input_grad_workspace_bytes(M, *Wc);
}

spl_status spl_sparse_input_grad(const void* dY, int64_t M, const spl_matrix* Wc, void* dX, void* workspace,
                                 hipStream_t stream) {
  const spl_status st = check_tiled_fp(Wc);
  if (st != SPL_OK) return st;
  const spl_status xy = check_xy(dY, M, Wc->rows, Wc->cols, dX);   // dY [M][N], dX [M][K]
  if (xy != SPL_OK || M == 0) return xy;
  if (!spl::sparse_input_grad_applies(M, *Wc)) {
    if (Wc->rows % 8 != 0) return SPL_ERR_UNSUPPORTED;             // the dense product's 16-byte rows of dY
    if (!workspace || !aligned(workspace, 256)) return SPL_ERR_INVALID_ARG;
  }
  (void)hipGetLastError();
  return launched(spl::launch_input_grad(dY, M, *Wc, dX, workspace, stream));
}

spl_status spl_sparse_sgd_update(const spl_matrix* Wc, const void* grad_values, float lr, hipStream_t stream) {
  const spl_status st = check_tiled_fp(Wc);
  if (st != SPL_OK) return st;
  if (Wc->nnz > 0 && (!grad_values || !aligned(grad_values, 2))) return SPL_ERR_INVALID_ARG;
  (void)hipGetLastError();
  return launched(spl::launch_sgd(*Wc, grad_values, lr, stream));
}

int64_t spl_transpose_perm_workspace_bytes(int64_t N, int64_t K, int64_t nnz) {
  if (!dims_ok(N, K) || nnz < 0 || nnz > N * K) return -1;
  return spl::transpose_perm_workspace_bytes(N, K, nnz);
}

spl_status spl_transpose_perm(const spl_matrix* W, const spl_matrix* Wt, int32_t* perm, void* workspace,
                              hipStream_t stream) {
  spl_status st = check_tiled_fp(W);
  if (st != SPL_OK) return st;
  st = check_tiled_fp(Wt);
  if (st != SPL_OK) return st;
  if (Wt->rows != W->cols || Wt->cols != W->rows || Wt->nnz != W->nnz || Wt->dtype != W->dtype)
    return SPL_ERR_INVALID_ARG;
  if (W->cols % 8 != 0 || W->rows % 8 != 0 || (W->rows + 63) / 64 > 65535 || (W->cols + 63) / 64 > 65535)
    return SPL_ERR_UNSUPPORTED;
  if (W->nnz == 0) return SPL_OK;
  if (!perm || !workspace || !aligned(perm, 4) || !aligned(workspace, 256)) return SPL_ERR_INVALID_ARG;
  (void)hipGetLastError();
  return launched(spl::launch_transpose_perm(*W, *Wt, perm, workspace, stream));
}

spl_status spl_permute_values(const void* src, const int32_t* perm, int64_t nnz, void* dst, hipStream_t stream) {
  if (nnz < 0) return SPL_ERR_INVALID_ARG;
  if (nnz >= kMaxDim) return SPL_ERR_OVERFLOW;         // value counts are below 2^31, as nnz everywhere
  if (nnz == 0) return SPL_OK;
  if (!src || !perm || !dst || !aligned(src, 2) || !aligned(perm, 4) || !aligned(dst, 2)) return SPL_ERR_INVALID_ARG;
  (void)hipGetLastError();
  return launched(spl::launch_permute_values(src, perm, nnz, dst, stream));
}

int64_t spl_int4_values_bytes(int64_t nnz) { return nnz < 0 ? -1 : spl::int4_values_bytes(nnz); }

spl_status spl_pack_int4(const spl_matrix* W8, uint8_t* values4, int32_t* bad_codes, hipStream_t stream) {
  const spl_status st = spl_check_matrix(W8);
  if (st != SPL_OK) return st;
  if (W8->dtype != SPL_I8 || W8->layout != SPL_LAYOUT_TILE16) return SPL_ERR_UNSUPPORTED;
  if (!values4 || !aligned(values4, 16)) return SPL_ERR_INVALID_ARG;
  if (bad_codes && !aligned(bad_codes, 4)) return SPL_ERR_INVALID_ARG;
  (void)hipGetLastError();
  return launched(spl::launch_pack_nibbles(static_cast<const int8_t*>(W8->values), W8->nnz, values4, bad_codes,
                                           stream));
}

// A SPL_I4 view: the checks of spl_check_matrix with the 4-bit dtype and the tile layout.
static spl_status check_i4_view(const spl_matrix* W) {
  if (!W) return SPL_ERR_INVALID_ARG;
  if (W->dtype != SPL_I4 || W->layout != SPL_LAYOUT_TILE16) return SPL_ERR_UNSUPPORTED;
  if (W->values_bytes < spl_values_bytes(SPL_I4, W->nnz)) return SPL_ERR_INVALID_ARG;
  spl_matrix v = *W;
  v.dtype = SPL_I8;                                   // the same scalar and pointer rules
  v.values_bytes = spl_values_bytes(SPL_I8, W->nnz);  // (the 4-bit capacity is checked above)
  return spl_check_matrix(&v);
}

spl_status spl_sparse_linear_int4(const int8_t* Xq, const float* x_scales, int64_t M, const spl_matrix* W4,
                                  const float* w_scales, void* Y, int32_t* acc_out, hipStream_t stream) {
  const spl_status st = check_i4_view(W4);
  if (st != SPL_OK) return st;
  if (M < 0) return SPL_ERR_INVALID_ARG;
  if (M > 16) return SPL_ERR_UNSUPPORTED;
  const spl_status xy = check_xy(Xq, M, W4->cols, W4->rows, Y);
  if (xy != SPL_OK || M == 0) return xy;
  if (!x_scales || !w_scales || !aligned(x_scales, 4) || !aligned(w_scales, 4)) return SPL_ERR_INVALID_ARG;
  if (acc_out && !aligned(acc_out, 16)) return SPL_ERR_INVALID_ARG;
  if (W4->cols % 16 != 0) return SPL_ERR_UNSUPPORTED;
  (void)hipGetLastError();
  return launched(spl::launch_sparse_int4(Xq, x_scales, M, *W4, w_scales, Y, acc_out, stream));
}

// Arguments of one sparse-quantized task (those of spl_sparse_linear_int8).
static spl_status check_int8_task(const spl_int8_task* t, int64_t M) {
  const spl_status st = spl_check_matrix(t->Wq);
  if (st != SPL_OK) return st;
  if (t->Wq->dtype != SPL_I8 || t->Wq->layout != SPL_LAYOUT_TILE16) return SPL_ERR_UNSUPPORTED;
  const spl_status xy = check_xy(t->Xq, M, t->Wq->cols, t->Wq->rows, t->Y);
  if (xy != SPL_OK || M == 0) return xy;                 // M == 0: nothing is read or written
  if (!t->x_scales || !t->w_scales || !aligned(t->x_scales, 4) || !aligned(t->w_scales, 4)) return SPL_ERR_INVALID_ARG;
  if (t->acc_out && !aligned(t->acc_out, 16)) return SPL_ERR_INVALID_ARG;
  if (t->Wq->cols % 16 != 0) return SPL_ERR_UNSUPPORTED;
  return SPL_OK;
}

spl_status spl_sparse_linear_int8(const int8_t* Xq, const float* x_scales, int64_t M, const spl_matrix* Wqc,
                                  const float* w_scales, void* Y, int32_t* acc_out, hipStream_t stream) {
  const spl_int8_task t{Xq, x_scales, Wqc, w_scales, Y, acc_out};
  return spl_sparse_linear_int8_group(&t, 1, M, stream);
}

spl_status spl_sparse_linear_int8_expanded(const int8_t* Xq, const float* x_scales, int64_t M, const spl_matrix* Wqc,
                                           const float* w_scales, void* Y, int32_t* acc_out, void* workspace,
                                           hipStream_t stream) {
  const spl_int8_task t{Xq, x_scales, Wqc, w_scales, Y, acc_out};
  if (!Wqc) return SPL_ERR_INVALID_ARG;
  const spl_status st = check_int8_task(&t, M);
  if (st != SPL_OK) return st;
  if (!workspace || !aligned(workspace, 16)) return SPL_ERR_INVALID_ARG;
  if (spl::tile_blocks(Wqc->rows) >= kMaxDim || M >= kMaxDim) return SPL_ERR_OVERFLOW;
  if (M == 0) return SPL_OK;
  (void)hipGetLastError();
  const spl_status e = launched(spl::launch_unpack(*Wqc, workspace, stream));   // the decoded [N][K] codes
  if (e != SPL_OK) return e;
  const spl_dense_int8_task d{Xq, x_scales, static_cast<const int8_t*>(workspace), w_scales, Wqc->rows, Wqc->cols,
                              Y, acc_out};
  return launched(spl::launch_dense_prefill_i8(d, M, stream));
}

spl_status spl_sparse_linear_int8_group(const spl_int8_task* tasks, int32_t count, int64_t M, hipStream_t stream) {
  if (!tasks || count < 1 || count > SPL_MAX_GROUP || M < 0) return SPL_ERR_INVALID_ARG;
  int64_t blocks = 0;
  for (int32_t i = 0; i < count; ++i) {
    const spl_status st = check_int8_task(&tasks[i], M);
    if (st != SPL_OK) return st;
    blocks += spl::tile_blocks(tasks[i].Wq->rows);
  }
  if (blocks >= kMaxDim || M >= kMaxDim) return SPL_ERR_OVERFLOW;
  if (M == 0) return SPL_OK;
  (void)hipGetLastError();
  return launched(spl::launch_sparse_int8(tasks, count, M, stream));
}

spl_status spl_dense_linear_ex(const void* X, int64_t M, const void* W, int32_t dtype, int64_t N, int64_t K,
                               void* Y, int32_t algo, hipStream_t stream) {
  const spl_dense_task t{X, W, N, K, Y};
  return spl_dense_linear_group(&t, 1, M, dtype, algo, stream);
}

spl_status spl_dense_linear_group(const spl_dense_task* tasks, int32_t count, int64_t M, int32_t dtype,
                                  int32_t algo, hipStream_t stream) {
  if (!tasks || count < 1 || count > SPL_MAX_GROUP || M < 0) return SPL_ERR_INVALID_ARG;
  int64_t blocks = 0;
  int32_t resolved = algo;
  for (int32_t i = 0; i < count; ++i) {
    int32_t a = algo;
    const spl_status st = check_dense_task(&tasks[i], M, dtype, &a);
    if (st != SPL_OK) return st;
    resolved = a;
    blocks += spl::tile_blocks(tasks[i].N);
  }
  if (blocks >= kMaxDim) return SPL_ERR_OVERFLOW;
  if (M == 0) return SPL_OK;
  (void)hipGetLastError();
  if (resolved == SPL_ALGO_DECODE) return launched(spl::launch_dense_decode(tasks, count, M, dtype, stream));
  for (int32_t i = 0; i < count; ++i) {
    const spl_status st = launched(spl::launch_dense_prefill(tasks[i].X, M, tasks[i].W, dtype, tasks[i].N,
                                                             tasks[i].K, tasks[i].Y, stream));
    if (st != SPL_OK) return st;
  }
  return SPL_OK;
}

spl_status spl_dense_linear(const void* X, int64_t M, const void* W, int32_t dtype, int64_t N, int64_t K,
                            void* Y, hipStream_t stream) {
  return spl_dense_linear_ex(X, M, W, dtype, N, K, Y, SPL_ALGO_AUTO, stream);
}

// Arguments of one dense int8 task (those of spl_dense_linear_int8).
static spl_status check_dense_int8_task(const spl_dense_int8_task* t, int64_t M) {
  if (!t->Wq || !dims_ok(t->N, t->K) || !aligned(t->Wq, 16)) return SPL_ERR_INVALID_ARG;
  const spl_status xy = check_xy(t->Xq, M, t->K, t->N, t->Y);
  if (xy != SPL_OK || M == 0) return xy;                 // M == 0: nothing is read or written
  if (!t->x_scales || !t->w_scales || !aligned(t->x_scales, 4) || !aligned(t->w_scales, 4)) return SPL_ERR_INVALID_ARG;
  if (t->acc_out && !aligned(t->acc_out, 16)) return SPL_ERR_INVALID_ARG;
  if (t->K % 16 != 0) return SPL_ERR_UNSUPPORTED;
  return SPL_OK;
}

spl_status spl_dense_linear_int8(const int8_t* Xq, const float* x_scales, int64_t M, const int8_t* Wq,
                                 const float* w_scales, int64_t N, int64_t K, void* Y, int32_t* acc_out,
                                 hipStream_t stream) {
  const spl_dense_int8_task t{Xq, x_scales, Wq, w_scales, N, K, Y, acc_out};
  return spl_dense_linear_int8_group(&t, 1, M, stream);
}

spl_status spl_dense_linear_int8_group(const spl_dense_int8_task* tasks, int32_t count, int64_t M,
                                       hipStream_t stream) {
  if (!tasks || count < 1 || count > SPL_MAX_GROUP || M < 0) return SPL_ERR_INVALID_ARG;
  int64_t blocks = 0;
  for (int32_t i = 0; i < count; ++i) {
    const spl_status st = check_dense_int8_task(&tasks[i], M);
    if (st != SPL_OK) return st;
    blocks += (tasks[i].N + 15) / 16;
  }
  if (blocks >= kMaxDim || M >= kMaxDim) return SPL_ERR_OVERFLOW;
  if (M == 0) return SPL_OK;
  (void)hipGetLastError();
  return launched(spl::launch_dense_int8(tasks, count, M, stream));
}

spl_status spl_quantize_rows_i8(const void* X, int32_t dtype, int64_t M, int64_t K, int8_t* Xq, float* x_scales,
                                hipStream_t stream) {
  if (M < 0) return SPL_ERR_INVALID_ARG;
  if (!fp_dtype(dtype)) return SPL_ERR_UNSUPPORTED;
  if (M == 0) return SPL_OK;
  if (!X || !Xq || !x_scales || !dims_ok(M, K)) return SPL_ERR_INVALID_ARG;
  if (K % 8 != 0) return SPL_ERR_UNSUPPORTED;
  if (!aligned(X, 16) || !aligned(Xq, 16) || !aligned(x_scales, 4)) return SPL_ERR_INVALID_ARG;
  (void)hipGetLastError();
  return launched(spl::launch_quantize_rows_i8(X, dtype, M, K, Xq, x_scales, stream));
}

}  // extern "C"
