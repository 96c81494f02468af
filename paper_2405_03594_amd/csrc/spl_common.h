// Internal helpers shared by the gfx950 kernels of libspl (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "spl.h"

namespace spl {

constexpr int kWave = 64;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));

// Storage tags: a 16-bit float payload and how to widen / narrow it.
struct Bf16 {
  static constexpr int32_t code = SPL_BF16;
  static __device__ __forceinline__ float to_f32(uint32_t bits16) { return __uint_as_float(bits16 << 16); }
  // binary32 -> bfloat16, round to nearest even; NaN stays NaN.
  static __device__ __forceinline__ uint16_t from_f32(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
  }
};

struct F16 {
  static constexpr int32_t code = SPL_F16;
  static __device__ __forceinline__ float to_f32(uint32_t bits16) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)bits16);
  }
  // binary32 -> binary16, round to nearest even.  The empty asm keeps the
  // compiler from folding a preceding multiply or add into the conversion
  // (v_fma_mixlo_f16 rounds the exact result once, straight to binary16).
  static __device__ __forceinline__ uint16_t from_f32(float f) {
    asm("" : "+v"(f));
    return __builtin_bit_cast(uint16_t, (_Float16)f);   // v_cvt_f16_f32
  }
};

__device__ __forceinline__ uint32_t lane_id() { return __lane_id(); }

// Number of set bits of a 64-bit wave mask below this lane.
__device__ __forceinline__ uint32_t mbcnt64(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Order this wave's LDS writes before its later LDS reads of other lanes' data.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Inclusive prefix sum across each group of 16 lanes (DPP row shifts; lanes
// shifted in from outside the row contribute 0).
__device__ __forceinline__ uint32_t row16_inclusive_scan(uint32_t x) {
  x += __builtin_amdgcn_update_dpp(0u, x, 0x111, 0xf, 0xf, false);   // row_shr:1
  x += __builtin_amdgcn_update_dpp(0u, x, 0x112, 0xf, 0xf, false);   // row_shr:2
  x += __builtin_amdgcn_update_dpp(0u, x, 0x114, 0xf, 0xf, false);   // row_shr:4
  x += __builtin_amdgcn_update_dpp(0u, x, 0x118, 0xf, 0xf, false);   // row_shr:8
  return x;
}

// Inclusive prefix sum across each half (32 lanes) of the wave: the 16-lane
// scans, then lane 15's total added to lanes 16-31 and lane 47's to 48-63
// (DPP row_bcast:15 into rows 1 and 3).
__device__ __forceinline__ uint32_t half_inclusive_scan(uint32_t x) {
  x = row16_inclusive_scan(x);
  x += __builtin_amdgcn_update_dpp(0u, x, 0x142, 0xa, 0xf, false);   // row_bcast:15, rows 1 and 3
  return x;
}

// Inclusive prefix sum across the whole wave (64 lanes): the half scans, then
// lane 31's total added to lanes 32-63 (DPP row_bcast:31 into rows 2 and 3).
__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t x) {
  x = half_inclusive_scan(x);
  x += __builtin_amdgcn_update_dpp(0u, x, 0x143, 0xc, 0xf, false);   // row_bcast:31, rows 2 and 3
  return x;
}

// Task of this workgroup in a grouped launch whose task i owns workgroups
// [first[i], first[i + 1]) along x (wave-uniform).
__device__ __forceinline__ int find_task(const int32_t* first, int count) {
  int ti = 0;
  for (int i = 1; i < count; ++i) ti = (int)blockIdx.x >= first[i] ? i : ti;
  return ti;
}

// v_perm_b32 selectors that expand one 4-column nibble of the bitmask.  The
// nibble's stored values sit, in order, in the 8 source bytes {hi:lo}; a
// kept column takes the bytes of its rank among the nibble's set bits, a
// dropped one selector 0x0C (a zero byte).
//   selector16: the 16-bit elements (2h, 2h + 1) of the nibble (two bytes each).
//   selector8: the four 1-byte elements, values starting at byte p (p + rank <= 7).
__host__ __device__ __forceinline__ uint32_t nibble_rank(uint32_t nib, int j) {
  return (uint32_t)__builtin_popcount(nib & ((1u << j) - 1u));
}
__host__ __device__ __forceinline__ uint32_t nibble_selector16(uint32_t nib, int h) {
  uint32_t sel = 0;
  for (int e = 0; e < 2; ++e) {
    const int j = 2 * h + e;
    const uint32_t r = nibble_rank(nib, j);
    const uint32_t s16 = ((nib >> j) & 1u) ? (2u * r) | ((2u * r + 1u) << 8) : 0x0C0Cu;
    sel |= s16 << (16 * e);
  }
  return sel;
}
__host__ __device__ __forceinline__ uint32_t nibble_selector8(uint32_t nib, uint32_t p = 0) {
  uint32_t sel = 0;
  for (int j = 0; j < 4; ++j) sel |= (((nib >> j) & 1u) ? p + nibble_rank(nib, j) : 0x0Cu) << (8 * j);
  return sel;
}

typedef __attribute__((address_space(3))) unsigned char lds_t;

// 32-bit LDS offset of a pointer into shared memory, and loads at such offsets.
__device__ __forceinline__ uint32_t lds_off(const void* p) {
  return (uint32_t)(uintptr_t)(const lds_t*)p;     // address-space cast: generic -> LDS offset
}
__device__ __forceinline__ u32x4 lds_load16(uint32_t addr) {
  return *reinterpret_cast<const __attribute__((address_space(3))) u32x4*>((uintptr_t)addr);
}
__device__ __forceinline__ uint32_t lds_load4(uint32_t addr) {
  return *reinterpret_cast<const __attribute__((address_space(3))) uint32_t*>((uintptr_t)addr);
}
__device__ __forceinline__ u32x2 lds_load8(uint32_t addr) {
  return *reinterpret_cast<const __attribute__((address_space(3))) u32x2*>((uintptr_t)addr);
}

__host__ __device__ __forceinline__ int64_t words_per_row(int64_t K) { return (K + 31) / 32; }
// Tile layout geometry: 16-row blocks and 32-column steps.
__host__ __device__ __forceinline__ int64_t tile_blocks(int64_t N) { return (N + 15) / 16; }
__host__ __device__ __forceinline__ int64_t tile_steps(int64_t K) { return (K + 31) / 32; }

// Host-side facts and settings kept per device: a process may drive several
// GPUs, so nothing learned with one device current is reused on another.
constexpr int kMaxDevices = 64;

// The current device, or -1 when it cannot be read or lies past kMaxDevices.
inline int current_device() {
  int d = -1;
  return hipGetDevice(&d) == hipSuccess && d >= 0 && d < kMaxDevices ? d : -1;
}

// Compute units of the current device (256 when the query fails).
inline int device_cus() {
  static std::atomic<int> cache[kMaxDevices];
  const int d = current_device();
  if (d < 0) return 256;
  int n = cache[d].load(std::memory_order_relaxed);
  if (n > 0) return n;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, d) != hipSuccess || n <= 0) n = 256;
  cache[d].store(n, std::memory_order_relaxed);
  return n;
}

// Raises a kernel's dynamic LDS limit on the current device, once per device;
// `done` belongs to one kernel (a static at its launch site).
struct PerDeviceFlag {
  std::atomic<int> set[kMaxDevices];
};
template <class F>
hipError_t allow_lds_once(PerDeviceFlag& done, F* kernel, size_t bytes) {
  const int d = current_device();
  if (d >= 0 && done.set[d].load(std::memory_order_acquire)) return hipSuccess;
  const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
  if (e == hipSuccess && d >= 0) done.set[d].store(1, std::memory_order_release);
  return e;
}

}  // namespace spl

// Launchers implemented in the kernel translation units (host side).
namespace spl {
hipError_t launch_pack_count(const void* W, int32_t dtype, const uint8_t* mask, int64_t N, int64_t K,
                             int32_t* row_offsets, hipStream_t s);
hipError_t launch_pack_scatter(const void* W, int32_t dtype, const uint8_t* mask, int64_t N, int64_t K,
                               const int32_t* row_offsets, uint32_t* bitmask, void* values, hipStream_t s);
hipError_t launch_unpack(const spl_matrix& Wc, void* W_dense, hipStream_t s);
// Pack straight into the tile layout: per-tile counts -> exclusive tile offsets, then bitmask + values.
hipError_t launch_pack_count_tiled(const void* W, int32_t dtype, const uint8_t* mask, int64_t N, int64_t K,
                                   int32_t* tile_offsets, hipStream_t s);
hipError_t launch_pack_scatter_tiled(const void* W, int32_t dtype, const uint8_t* mask, int64_t N, int64_t K,
                                     const int32_t* tile_offsets, uint32_t* bitmask, void* values, hipStream_t s);
// Format check of a view: error bits (1 offsets vs popcounts, 2 first/last offset, 4 pad bits) OR-ed into *err.
hipError_t launch_validate(const spl_matrix& Wc, uint32_t* err, hipStream_t s);
hipError_t launch_retile16(const spl_matrix& rows_in, uint32_t* bitmask_t, void* values_t, int32_t* tile_offsets,
                           hipStream_t s);
// Y[0..count16) = +0 (16-bit elements).
hipError_t launch_zero_fill(void* Y, int64_t count16, hipStream_t s);

// Decode kernels over a group of 1..SPL_MAX_GROUP validated tasks (one launch).
hipError_t launch_sparse_decode(const spl_sparse_task* tasks, int count, int64_t M, hipStream_t s);
hipError_t launch_dense_decode(const spl_dense_task* tasks, int count, int64_t M, int32_t dtype, hipStream_t s);
hipError_t launch_sparse_prefill(const void* X, int64_t M, const spl_matrix& Wc, void* Y, hipStream_t s);
hipError_t launch_dense_prefill(const void* X, int64_t M, const void* W, int32_t dtype, int64_t N, int64_t K,
                                void* Y, hipStream_t s);
// The same product written only at the kept positions of the tile pattern P
// (P.rows == M, P.cols == N), in P's value order (fp16/bf16).
hipError_t launch_dense_prefill_gather(const void* X, int64_t M, const void* W, int32_t dtype, int64_t N, int64_t K,
                                       const spl_matrix& P, void* values, hipStream_t s);
// The same from contraction-major factors, Y = Xc^T Wc (Xc [K][M], Wc [K][N]),
// where dense_prefill_tr_applies (M % 256, N % 128 and K % 64 all zero, a
// launch of at least one 128 x 256 block per CU, 16-byte aligned factors).
bool dense_prefill_tr_applies(int64_t M, int64_t N, int64_t K, const void* Xc, const void* Wc);
// The input gradient dX [M][K] = dY [M][N] (W.Mask) from W's packed tiles
// where sparse_input_grad_applies (M % 256, N % 64 and K % 128 all zero, a
// launch of at least one 128 x 256 block per CU; W in the tile layout, 16-bit).
bool sparse_input_grad_applies(int64_t M, const spl_matrix& W);
hipError_t launch_sparse_input_grad(const void* dY, int64_t M, const spl_matrix& W, void* dX, hipStream_t s);
// A group of such products (one dtype; each where dense_prefill_tr_applies)
// in as few launches as possible.
struct TrTask {
  const void* Xc;
  const void* Wc;
  int64_t M, N, K;
  const spl_matrix* P;
  void* values;
};
hipError_t launch_dense_prefill_gather_tr(const TrTask* tasks, int count, int32_t dtype, hipStream_t s);
// Sparse-quantized kernels over a group of 1..SPL_MAX_GROUP validated tasks (one launch).
hipError_t launch_sparse_int8(const spl_int8_task* tasks, int count, int64_t M, hipStream_t s);
hipError_t launch_dense_int8(const spl_dense_int8_task* tasks, int count, int64_t M, hipStream_t s);
hipError_t launch_sparse_prefill_i8(const spl_int8_task& t, int64_t M, hipStream_t s);
hipError_t launch_dense_prefill_i8(const spl_dense_int8_task& t, int64_t M, hipStream_t s);
// Gated half of a Llama MLP, Y = silu(X Wg^T) * (X Wu^T): M <= 16 (decode) or any M (prefill).
hipError_t launch_gated_decode(const void* X, int64_t M, const spl_matrix& Wg, const spl_matrix& Wu, void* Y,
                               hipStream_t s);
hipError_t launch_gated_prefill(const void* X, int64_t M, const spl_matrix& Wg, const spl_matrix& Wu, void* Y,
                                hipStream_t s);
// Magnitude pruning mask of n = N K fp16/bf16 entries (n % 8 == 0, n < 2^31)
// with a workspace of magnitude_mask_workspace_words() 32-bit words.
int64_t magnitude_mask_workspace_words();
hipError_t launch_magnitude_mask(const uint16_t* W, int64_t n, uint32_t prune, uint8_t* mask, uint32_t* ws,
                                 hipStream_t s);
// Training with the mask held fixed: transposes, gather into a tile pattern,
// the weight gradient (workspace of weight_grad_workspace_bytes) and SGD.
hipError_t launch_transpose16(const void* src, int64_t R, int64_t C, void* dst, hipStream_t s);
hipError_t launch_gather_tiled(const void* dense, const spl_matrix& P, void* values, hipStream_t s);
int64_t weight_grad_workspace_bytes(int64_t M, int64_t N, int64_t K);
hipError_t launch_weight_grad(const void* dY, const void* X, int64_t M, const spl_matrix& Wc, void* grad_values,
                              void* ws, hipStream_t s);
hipError_t launch_weight_grad_group(const spl_weight_grad_task* tasks, int count, int64_t M, void* ws,
                                    hipStream_t s);
hipError_t launch_sgd(const spl_matrix& Wc, const void* grad_values, float lr, hipStream_t s);
int64_t input_grad_workspace_bytes(int64_t M, const spl_matrix& W);
hipError_t launch_input_grad(const void* dY, int64_t M, const spl_matrix& W, void* dX, void* ws, hipStream_t s);
int64_t transpose_perm_workspace_bytes(int64_t N, int64_t K, int64_t nnz);
hipError_t launch_transpose_perm(const spl_matrix& W, const spl_matrix& Wt, int32_t* perm, void* ws, hipStream_t s);
hipError_t launch_permute_values(const void* src, const int32_t* perm, int64_t nnz, void* dst, hipStream_t s);
// 4-bit payloads: nibble packing of int8 tile values and the decode kernel (M <= 16).
int64_t int4_values_bytes(int64_t nnz);
// bad (optional): set to the number of codes outside [-8, 7] (their low 4 bits are stored).
hipError_t launch_pack_nibbles(const int8_t* v8, int64_t nnz, uint8_t* v4, int32_t* bad, hipStream_t s);
hipError_t launch_sparse_int4(const int8_t* Xq, const float* sx, int64_t M, const spl_matrix& W4, const float* sw,
                              void* Y, int32_t* acc_out, hipStream_t s);
// Streaming-read probe over `bytes` (a multiple of 16) of a 16-byte aligned buffer.
hipError_t launch_read_probe(const void* buf, int64_t bytes, uint32_t* sink, int cus, hipStream_t s);
hipError_t launch_quantize_rows_i8(const void* X, int32_t dtype, int64_t M, int64_t K, int8_t* Xq, float* sx,
                                   hipStream_t s);
}  // namespace spl
