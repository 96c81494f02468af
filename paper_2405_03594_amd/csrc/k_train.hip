// Sparse training step with the mask held fixed (paper Algorithm 1): the
// gradient of Y = X (W.Mask)^T with respect to the kept weights, and the SGD
// update of the stored values.
//
// Weight gradient G = Mask . (dY^T X): both operands are [M][*] row-major and
// the reduction runs over M.  Where the shapes allow, the contraction-major
// core of the prefill kernels reads dY and X as stored (LDS transpose reads);
// otherwise they are first transposed into [N][M] and [K][M] (the workspace)
// and a dense prefill kernel multiplies those.  Either way the product's
// epilogue writes only the kept entries, rounded once to the payload type,
// straight into the tile layout's value order: no dense [N][K] gradient is
// formed.  The input gradient dX = dY (W.Mask) is read from W's own packed
// tiles where the shapes allow, else from a decoded, transposed copy.
//
// k_gather_tiled (spl_gather_tiled) is the stand-alone form of that order:
// lane (fr, fg) of a tile's wave owns row fr, columns 8 fg .. 8 fg + 7, and
// its values start at the exclusive wave scan of the lanes' kept counts.
#include "spl_common.h"

namespace spl {
namespace {

constexpr int kTT = 64;                 // transpose tile edge

// dst[c][r] = src[r][c] for a 16-bit [R][C] matrix: 64 x 64 tiles through LDS
// (a padded row so that the column reads hit distinct banks).
__global__ void __launch_bounds__(256) k_transpose16(const uint16_t* __restrict__ src, int64_t R, int64_t C,
                                                     uint16_t* __restrict__ dst) {
  __shared__ uint16_t tile[kTT][kTT + 2];
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int64_t c0 = (int64_t)blockIdx.x * kTT, r0 = (int64_t)blockIdx.y * kTT;
#pragma unroll 4
  for (int i = ty; i < kTT; i += 4) {
    const int64_t r = r0 + i, c = c0 + tx;
    tile[i][tx] = (r < R && c < C) ? src[r * C + c] : (uint16_t)0;
  }
  __syncthreads();
#pragma unroll 4
  for (int i = ty; i < kTT; i += 4) {
    const int64_t c = c0 + i, r = r0 + tx;
    if (c < C && r < R) dst[c * R + r] = tile[tx][i];
  }
}

// The same transpose for R % 8 == 0 and C % 8 == 0 (16-byte aligned rows):
// each thread moves one 8 x 8 block with eight 16-byte loads (rows r..r+7,
// columns c..c+7), a register transpose (v_perm_b32 picks the 16-bit halves)
// and eight 16-byte stores (rows c..c+7 of dst, columns r..r+7).  Lane
// 8 y + x of a wave takes block (8 y, 8 x) of its 64 x 64 tile: per load the
// eight lanes of one y read one 128-byte segment of a src row, and per store
// the eight lanes of one x write one 128-byte segment of a dst row.  Four
// waves per workgroup take four tiles along the columns.
constexpr int kT8Tile = 64;
__global__ void __launch_bounds__(256) k_transpose16_b8(const uint16_t* __restrict__ src, int64_t R, int64_t C,
                                                        uint16_t* __restrict__ dst) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t r = (int64_t)blockIdx.y * kT8Tile + 8 * (lane >> 3);                 // block's first row
  const int64_t c = ((int64_t)blockIdx.x * 4 + wave) * kT8Tile + 8 * (lane & 7);   // and first column
  if (r >= R || c >= C) return;                      // whole blocks: R % 8 == C % 8 == 0
  u32x4 v[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = *reinterpret_cast<const u32x4*>(src + (r + i) * C + c);
  // o[j] = column j of the block: its dword d holds rows 2d (low half) and 2d + 1 (high half)
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t sel = (j & 1) ? 0x07060302u : 0x05040100u;
    u32x4 o;
    o.x = __builtin_amdgcn_perm(v[1][j >> 1], v[0][j >> 1], sel);
    o.y = __builtin_amdgcn_perm(v[3][j >> 1], v[2][j >> 1], sel);
    o.z = __builtin_amdgcn_perm(v[5][j >> 1], v[4][j >> 1], sel);
    o.w = __builtin_amdgcn_perm(v[7][j >> 1], v[6][j >> 1], sel);
    *reinterpret_cast<u32x4*>(dst + (c + j) * R + r) = o;
  }
}

// Kept entries of a dense [N][K] matrix (K % 8 == 0) in the order of a tile
// pattern: one wave per tile, 4 tiles per workgroup.
__global__ void __launch_bounds__(256) k_gather_tiled(const uint16_t* __restrict__ dense,
                                                      const uint32_t* __restrict__ bm_tiles,
                                                      const int32_t* __restrict__ toff, int64_t N, int64_t K,
                                                      int64_t tiles, uint16_t* __restrict__ values) {
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= tiles) return;                            // whole waves leave together
  const int lane = threadIdx.x & 63, fr = lane & 15, fg = lane >> 4;
  const int64_t S = tile_steps(K);
  const int64_t n = (t / S) * 16 + fr;
  const int64_t k0 = (t % S) * 32 + 8 * fg;
  const uint32_t byte = (bm_tiles[t * 16 + fr] >> (8 * fg)) & 0xffu;   // pad rows and columns: zero bits
  const uint32_t cnt = __popc(byte);
  uint32_t off = (uint32_t)toff[t] + wave_inclusive_scan(cnt) - cnt;
  if (byte == 0u) return;                            // (after the scan: every lane took part)
  const u32x4 v = *reinterpret_cast<const u32x4*>(dense + n * K + k0);   // byte != 0: n < N, k0 + 8 <= K
#pragma unroll
  for (int j = 0; j < 8; ++j)
    if ((byte >> j) & 1u) values[off++] = (uint16_t)((v[j >> 1] >> (16 * (j & 1))) & 0xffffu);
}

// The value position of every kept entry of a tile pattern, written into a
// dense [N][K] image as two 16-bit planes (low and high halves); entries off
// the pattern are not written.  The same lane schedule as k_gather_tiled.
__global__ void __launch_bounds__(256) k_scatter_positions(const uint32_t* __restrict__ bm_tiles,
                                                           const int32_t* __restrict__ toff, int64_t K, int64_t tiles,
                                                           uint16_t* __restrict__ lo, uint16_t* __restrict__ hi) {
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= tiles) return;
  const int lane = threadIdx.x & 63, fr = lane & 15, fg = lane >> 4;
  const int64_t S = tile_steps(K);
  const int64_t n = (t / S) * 16 + fr;
  const int64_t k0 = (t % S) * 32 + 8 * fg;
  const uint32_t byte = (bm_tiles[t * 16 + fr] >> (8 * fg)) & 0xffu;
  const uint32_t cnt = __popc(byte);
  uint32_t off = (uint32_t)toff[t] + wave_inclusive_scan(cnt) - cnt;
  if (byte == 0u) return;
#pragma unroll
  for (int j = 0; j < 8; ++j)
    if ((byte >> j) & 1u) {
      lo[n * K + k0 + j] = (uint16_t)(off & 0xffffu);
      hi[n * K + k0 + j] = (uint16_t)(off >> 16);
      ++off;
    }
}

__global__ void __launch_bounds__(256) k_join_halves(const uint16_t* __restrict__ lo, const uint16_t* __restrict__ hi,
                                                     int64_t nnz, int32_t* __restrict__ perm) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < nnz; i += (int64_t)gridDim.x * 256)
    perm[i] = (int32_t)((uint32_t)lo[i] | ((uint32_t)hi[i] << 16));
}

// dst[i] = src[perm[i]] (16-bit payloads, src of nnz entries); a position
// outside [0, nnz) (a permutation of another pattern) reads nothing and gives 0.
__global__ void __launch_bounds__(256) k_permute_values(const uint16_t* __restrict__ src,
                                                        const int32_t* __restrict__ perm, int64_t nnz,
                                                        uint16_t* __restrict__ dst) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < nnz; i += (int64_t)gridDim.x * 256) {
    const int32_t p = perm[i];
    dst[i] = (p >= 0 && (int64_t)p < nnz) ? src[p] : (uint16_t)0;
  }
}

// values[i] = RNE(values[i] - lr * grad[i]), each operation rounded to binary32.
template <class T>
__global__ void __launch_bounds__(256) k_sgd(uint16_t* __restrict__ values, const uint16_t* __restrict__ grad,
                                             int64_t nnz, float lr) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < nnz; i += (int64_t)gridDim.x * 256) {
    const float w = T::to_f32(values[i]), g = T::to_f32(grad[i]);
    values[i] = T::from_f32(__fsub_rn(w, __fmul_rn(lr, g)));
  }
}

constexpr int64_t align256(int64_t b) { return (b + 255) / 256 * 256; }

}  // namespace

hipError_t launch_transpose16(const void* src, int64_t R, int64_t C, void* dst, hipStream_t s) {
  if (R % 8 == 0 && C % 8 == 0 && reinterpret_cast<uintptr_t>(src) % 16 == 0 &&
      reinterpret_cast<uintptr_t>(dst) % 16 == 0) {
    const dim3 grid((unsigned)((C + 4 * kT8Tile - 1) / (4 * kT8Tile)), (unsigned)((R + kT8Tile - 1) / kT8Tile));
    hipLaunchKernelGGL(k_transpose16_b8, grid, dim3(256), 0, s, static_cast<const uint16_t*>(src), R, C,
                       static_cast<uint16_t*>(dst));
    return hipGetLastError();
  }
  const dim3 grid((unsigned)((C + kTT - 1) / kTT), (unsigned)((R + kTT - 1) / kTT));
  hipLaunchKernelGGL(k_transpose16, grid, dim3(256), 0, s, static_cast<const uint16_t*>(src), R, C,
                     static_cast<uint16_t*>(dst));
  return hipGetLastError();
}

hipError_t launch_gather_tiled(const void* dense, const spl_matrix& P, void* values, hipStream_t s) {
  const int64_t tiles = tile_blocks(P.rows) * tile_steps(P.cols);
  hipLaunchKernelGGL(k_gather_tiled, dim3((unsigned)((tiles + 3) / 4)), dim3(256), 0, s,
                     static_cast<const uint16_t*>(dense), P.bitmask, P.tile_offsets, P.rows, P.cols, tiles,
                     static_cast<uint16_t*>(values));
  return hipGetLastError();
}

int64_t weight_grad_workspace_bytes(int64_t M, int64_t N, int64_t K) {
  return align256(2 * N * M) + align256(2 * K * M);
}

hipError_t launch_weight_grad(const void* dY, const void* X, int64_t M, const spl_matrix& Wc, void* grad_values,
                              void* ws, hipStream_t s) {
  const int64_t N = Wc.rows, K = Wc.cols;
  // dY [M][N] and X [M][K] are the contraction-major factors of dY^T X
  if (dense_prefill_tr_applies(N, K, M, dY, X)) {
    const TrTask t{dY, X, N, K, M, &Wc, grad_values};
    return launch_dense_prefill_gather_tr(&t, 1, Wc.dtype, s);
  }
  unsigned char* base = static_cast<unsigned char*>(ws);
  void* dYt = base;                                  // [N][M]
  void* Xt = base + align256(2 * N * M);             // [K][M]
  hipError_t e = launch_transpose16(dY, M, N, dYt, s);
  if (e == hipSuccess) e = launch_transpose16(X, M, K, Xt, s);
  // the kept entries of dYt Xt^T ([N][K], Wc's pattern) in Wc's value order
  if (e == hipSuccess) e = launch_dense_prefill_gather(dYt, N, Xt, Wc.dtype, K, M, Wc, grad_values, s);
  return e;
}

// The input gradient dX [M][K] = dY [M][N] (W.Mask): straight from W's packed
// tiles where the direct kernel applies (no workspace); otherwise W is decoded
// and transposed into the workspace ([N][K], then [K][N]) and multiplied by
// the dense prefill kernels.
int64_t input_grad_workspace_bytes(int64_t M, const spl_matrix& W) {
  return sparse_input_grad_applies(M, W) ? 0 : 2 * align256(2 * W.rows * W.cols);
}

hipError_t launch_input_grad(const void* dY, int64_t M, const spl_matrix& W, void* dX, void* ws, hipStream_t s) {
  if (W.nnz == 0) return launch_zero_fill(dX, M * W.cols, s);
  if (sparse_input_grad_applies(M, W)) return launch_sparse_input_grad(dY, M, W, dX, s);
  const int64_t N = W.rows, K = W.cols;
  unsigned char* base = static_cast<unsigned char*>(ws);
  void* Wd = base;                                   // [N][K]
  void* Wt = base + align256(2 * N * K);             // [K][N]
  hipError_t e = launch_unpack(W, Wd, s);
  if (e == hipSuccess) e = launch_transpose16(Wd, N, K, Wt, s);
  if (e == hipSuccess) e = launch_dense_prefill(dY, M, Wt, W.dtype, K, N, dX, s);   // dY Wt^T
  return e;
}

// Several weight gradients of one batch (one dtype): one grouped launch when
// every task reads its factors as stored, else one call per task (the
// workspace serving them in turn).
hipError_t launch_weight_grad_group(const spl_weight_grad_task* tasks, int count, int64_t M, void* ws,
                                    hipStream_t s) {
  TrTask tr[SPL_MAX_GROUP];
  int n = 0;
  bool direct = true;
  for (int i = 0; i < count; ++i) {
    const spl_matrix& W = *tasks[i].W;
    if (W.nnz == 0) continue;                        // no kept entry: nothing to write
    if (!dense_prefill_tr_applies(W.rows, W.cols, M, tasks[i].dY, tasks[i].X)) direct = false;
    tr[n++] = TrTask{tasks[i].dY, tasks[i].X, W.rows, W.cols, M, &W, tasks[i].grad_values};
  }
  if (n == 0) return hipSuccess;
  if (direct) return launch_dense_prefill_gather_tr(tr, n, tasks[0].W->dtype, s);
  for (int i = 0; i < count; ++i) {
    if (tasks[i].W->nnz == 0) continue;
    const hipError_t e = launch_weight_grad(tasks[i].dY, tasks[i].X, M, *tasks[i].W, tasks[i].grad_values, ws, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

int64_t transpose_perm_workspace_bytes(int64_t N, int64_t K, int64_t nnz) {
  return 4 * align256(2 * N * K) + 2 * align256(2 * nnz);
}

// perm[i] = the position in W's values of the entry that is value i of Wt,
// Wt's pattern being the transpose of W's: position images of W (two 16-bit
// planes), transposed, then gathered at Wt's pattern and joined.
hipError_t launch_transpose_perm(const spl_matrix& W, const spl_matrix& Wt, int32_t* perm, void* ws, hipStream_t s) {
  const int64_t N = W.rows, K = W.cols;
  unsigned char* b = static_cast<unsigned char*>(ws);
  uint16_t* lo = reinterpret_cast<uint16_t*>(b);
  uint16_t* hi = reinterpret_cast<uint16_t*>(b + align256(2 * N * K));
  uint16_t* lot = reinterpret_cast<uint16_t*>(b + 2 * align256(2 * N * K));
  uint16_t* hit = reinterpret_cast<uint16_t*>(b + 3 * align256(2 * N * K));
  uint16_t* plo = reinterpret_cast<uint16_t*>(b + 4 * align256(2 * N * K));
  uint16_t* phi = reinterpret_cast<uint16_t*>(b + 4 * align256(2 * N * K) + align256(2 * Wt.nnz));
  const int64_t tiles = tile_blocks(N) * tile_steps(K);
  hipLaunchKernelGGL(k_scatter_positions, dim3((unsigned)((tiles + 3) / 4)), dim3(256), 0, s, W.bitmask,
                     W.tile_offsets, K, tiles, lo, hi);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess) e = launch_transpose16(lo, N, K, lot, s);
  if (e == hipSuccess) e = launch_transpose16(hi, N, K, hit, s);
  if (e == hipSuccess) e = launch_gather_tiled(lot, Wt, plo, s);
  if (e == hipSuccess) e = launch_gather_tiled(hit, Wt, phi, s);
  if (e != hipSuccess) return e;
  int64_t blocks = (Wt.nnz + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(k_join_halves, dim3((unsigned)blocks), dim3(256), 0, s, plo, phi, Wt.nnz, perm);
  return hipGetLastError();
}

hipError_t launch_permute_values(const void* src, const int32_t* perm, int64_t nnz, void* dst, hipStream_t s) {
  int64_t blocks = (nnz + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(k_permute_values, dim3((unsigned)blocks), dim3(256), 0, s, static_cast<const uint16_t*>(src),
                     perm, nnz, static_cast<uint16_t*>(dst));
  return hipGetLastError();
}

hipError_t launch_sgd(const spl_matrix& Wc, const void* grad_values, float lr, hipStream_t s) {
  if (Wc.nnz == 0) return hipSuccess;
  int64_t blocks = (Wc.nnz + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  uint16_t* v = static_cast<uint16_t*>(const_cast<void*>(Wc.values));   // the view's values, updated in place
  const uint16_t* g = static_cast<const uint16_t*>(grad_values);
  if (Wc.dtype == SPL_BF16)
    hipLaunchKernelGGL(k_sgd<Bf16>, dim3((unsigned)blocks), dim3(256), 0, s, v, g, Wc.nnz, lr);
  else
    hipLaunchKernelGGL(k_sgd<F16>, dim3((unsigned)blocks), dim3(256), 0, s, v, g, Wc.nnz, lr);
  return hipGetLastError();
}

}  // namespace spl
