// Sparse-quantized linear layer (paper section 3.4: int8 weights and int8
// activations) and its dense comparator, for gfx950.
//
// acc[m][n] = sum over kept k of Xq[m][k] * Wq[n][k] is accumulated exactly in
// int32 by v_mfma_i32_16x16x64_i8; the epilogue is
//   Y[m][n] = fp16_rne( (float(acc) * sx[m]) * sw[n] )
// with each product rounded to binary32 (no fused multiply-add).
//
// One MFMA covers 64 columns, i.e. two consecutive 16 x 32 tiles of the
// bitmask layout: lanes 0-31 take tile s, lanes 32-63 tile s + 1; each lane
// expands 16 int8 values of one tile row from two unaligned 8-byte loads and
// a byte-indexed v_perm_b32 selector table (paper section 2.4.1).
//
// Grid: x = 16-row tile block, y = 16*MT-row batch chunk.  A workgroup of
// kI8Waves waves splits the column range in groups of kI8Unroll tile pairs;
// partial int32 sums are combined through LDS (integer addition, so the
// result does not depend on the order).
#include "spl_common.h"

namespace spl {
namespace {

constexpr int kI8Waves = 8;
constexpr int kI8Threads = 64 * kI8Waves;
constexpr int kI8Unroll = 4;   // tile pairs per wave per group

__device__ __forceinline__ uint32_t i8_nibble_selector(uint32_t byte, int e) {
  uint32_t sel = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int bit = 4 * e + j;
    uint32_t s = 0x0Cu;                       // v_perm_b32: selector 12 yields a zero byte
    if ((byte >> bit) & 1u) s = __popc(byte & ((1u << bit) - 1u));
    sel |= s << (8 * j);
  }
  return sel;
}

__device__ __forceinline__ uint32_t i8_row16_inclusive_scan(uint32_t x) {
  x += __builtin_amdgcn_update_dpp(0u, x, 0x111, 0xf, 0xf, false);   // row_shr:1
  x += __builtin_amdgcn_update_dpp(0u, x, 0x112, 0xf, 0xf, false);   // row_shr:2
  x += __builtin_amdgcn_update_dpp(0u, x, 0x114, 0xf, 0xf, false);   // row_shr:4
  x += __builtin_amdgcn_update_dpp(0u, x, 0x118, 0xf, 0xf, false);   // row_shr:8
  return x;
}

__device__ __forceinline__ i32x4 mfma_i8(u32x4 a, u32x4 b, i32x4 c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4, a), __builtin_bit_cast(i32x4, b), c, 0, 0,
                                               0);
}

// Combine the waves' partial sums and run the epilogue.  part: [kI8Waves][MT][4][64] int32 in LDS.
template <int MT>
__device__ __forceinline__ void i8_finish(const i32x4 (&acc)[MT], int32_t* part, int wave, int lane, int64_t n0,
                                          int64_t N, int64_t m0, int64_t M, const float* __restrict__ sx,
                                          const float* __restrict__ sw, uint16_t* __restrict__ Y,
                                          int32_t* __restrict__ acc_out) {
#pragma unroll
  for (int f = 0; f < MT; ++f)
#pragma unroll
    for (int r = 0; r < 4; ++r) part[((wave * MT + f) * 4 + r) * 64 + lane] = acc[f][r];
  __syncthreads();
  // output (f, r, l): n = n0 + 4*(l/16) + r, m = m0 + 16 f + l%16
  for (int o = threadIdx.x; o < MT * 4 * 64; o += kI8Threads) {
    int32_t s = 0;
#pragma unroll
    for (int w = 0; w < kI8Waves; ++w) s += part[w * MT * 256 + o];
    const int f = o / 256, r = (o / 64) & 3, l = o & 63;
    const int64_t n = n0 + 4 * (l >> 4) + r;
    const int64_t m = m0 + 16 * f + (l & 15);
    if (n < N && m < M) {
      if (acc_out) acc_out[m * N + n] = s;
      const float a = static_cast<float>(s);
      const float t = __fmul_rn(a, sx[m]);
      const float y = __fmul_rn(t, sw[n]);
      Y[m * N + n] = F16::from_f32(y);
    }
  }
}

template <int MT>
__global__ void __launch_bounds__(kI8Threads) k_sparse_int8(const int8_t* __restrict__ Xq, const float* __restrict__ sx,
                                                            int64_t M, int64_t K, const uint32_t* __restrict__ bm_tiles,
                                                            const int8_t* __restrict__ values,
                                                            const int32_t* __restrict__ tile_offsets, int64_t N,
                                                            const float* __restrict__ sw, uint16_t* __restrict__ Y,
                                                            int32_t* __restrict__ acc_out, int any_values) {
  __shared__ u32x2 lut[256];
  __shared__ int32_t part[kI8Waves * MT * 256];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int fr = lane & 15, fg = lane >> 4;
  const int half = fg & 1, tsel = fg >> 1;
  const int S = (int)tile_steps(K);
  const int P = (S + 1) / 2;                              // tile pairs
  const int G = (P + kI8Unroll - 1) / kI8Unroll;          // groups of pairs
  const int64_t b = blockIdx.x;
  const int64_t m0 = (int64_t)blockIdx.y * 16 * MT;

  for (int i = threadIdx.x; i < 256; i += kI8Threads)
    lut[i] = u32x2{i8_nibble_selector(i, 0), i8_nibble_selector(i, 1)};
  __syncthreads();

  int64_t xrow[MT];
#pragma unroll
  for (int f = 0; f < MT; ++f) {
    const int64_t m = m0 + 16 * f + fr;
    xrow[f] = (m < M ? m : M - 1) * K;
  }
  const unsigned char* vb = reinterpret_cast<const unsigned char*>(values);
  const int hshift = 16 * half;
  const uint32_t lowmask = half ? 0xffffu : 0u;

  i32x4 acc[MT];
#pragma unroll
  for (int f = 0; f < MT; ++f) acc[f] = i32x4{0, 0, 0, 0};

  for (int g = wave; g < G; g += kI8Waves) {
    uint32_t w[kI8Unroll];
    uint32_t to[kI8Unroll];
    bool live[kI8Unroll];
#pragma unroll
    for (int u = 0; u < kI8Unroll; ++u) {
      const int p = g * kI8Unroll + u;
      const int s = 2 * p + tsel;
      live[u] = p < P && s < S;
      const int sc = s < S ? s : S - 1;
      const int64_t t = b * S + sc;
      w[u] = bm_tiles[t * 16 + fr];
      to[u] = (uint32_t)tile_offsets[t];
      if (!live[u]) w[u] = 0u;
    }
    u32x2 v0[kI8Unroll], v1[kI8Unroll];
    uint32_t b0[kI8Unroll], b1[kI8Unroll];
    u32x4 xb[kI8Unroll][MT];
#pragma unroll
    for (int u = 0; u < kI8Unroll; ++u) {
      const uint32_t pc = __popc(w[u]);
      const uint32_t above = i8_row16_inclusive_scan(pc) - pc;
      const uint32_t bits = (w[u] >> hshift) & 0xffffu;
      b0[u] = bits & 0xffu;
      b1[u] = bits >> 8;
      const uint32_t oa = to[u] + above + __popc(w[u] & lowmask);
      const uint32_t ob = oa + __popc(b0[u]);
      v0[u] = v1[u] = u32x2{0u, 0u};
      if (any_values) {                                   // values may be absent when nnz == 0
        __builtin_memcpy(&v0[u], vb + oa, 8);
        __builtin_memcpy(&v1[u], vb + ob, 8);
      }
      const int p = g * kI8Unroll + u;
      int64_t k = (int64_t)p * 64 + 16 * fg;
      const bool kok = k < K && p < P;
      if (!kok) k = 0;
#pragma unroll
      for (int f = 0; f < MT; ++f) {
        u32x4 x = *reinterpret_cast<const u32x4*>(Xq + xrow[f] + k);
        if (!kok) x = u32x4{0u, 0u, 0u, 0u};
        xb[u][f] = x;
      }
    }
#pragma unroll
    for (int u = 0; u < kI8Unroll; ++u) {
      const u32x2 s0 = lut[b0[u]], s1 = lut[b1[u]];
      u32x4 a;
      a.x = __builtin_amdgcn_perm(v0[u].y, v0[u].x, s0.x);
      a.y = __builtin_amdgcn_perm(v0[u].y, v0[u].x, s0.y);
      a.z = __builtin_amdgcn_perm(v1[u].y, v1[u].x, s1.x);
      a.w = __builtin_amdgcn_perm(v1[u].y, v1[u].x, s1.y);
#pragma unroll
      for (int f = 0; f < MT; ++f) acc[f] = mfma_i8(a, xb[u][f], acc[f]);
    }
  }
  i8_finish<MT>(acc, part, wave, lane, b * 16, N, m0, M, sx, sw, Y, acc_out);
}

template <int MT>
__global__ void __launch_bounds__(kI8Threads) k_dense_int8(const int8_t* __restrict__ Xq, const float* __restrict__ sx,
                                                           int64_t M, int64_t K, const int8_t* __restrict__ Wq,
                                                           int64_t N, const float* __restrict__ sw,
                                                           uint16_t* __restrict__ Y, int32_t* __restrict__ acc_out) {
  __shared__ int32_t part[kI8Waves * MT * 256];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int fr = lane & 15, fg = lane >> 4;
  const int Q = (int)((K + 63) / 64);                     // 64-column steps
  const int G = (Q + kI8Unroll - 1) / kI8Unroll;
  const int64_t n0 = (int64_t)blockIdx.x * 16;
  const int64_t m0 = (int64_t)blockIdx.y * 16 * MT;
  const int64_t wrow = (n0 + fr < N ? n0 + fr : N - 1) * K;
  int64_t xrow[MT];
#pragma unroll
  for (int f = 0; f < MT; ++f) {
    const int64_t m = m0 + 16 * f + fr;
    xrow[f] = (m < M ? m : M - 1) * K;
  }
  i32x4 acc[MT];
#pragma unroll
  for (int f = 0; f < MT; ++f) acc[f] = i32x4{0, 0, 0, 0};
  for (int g = wave; g < G; g += kI8Waves) {
    u32x4 a[kI8Unroll];
    u32x4 xb[kI8Unroll][MT];
#pragma unroll
    for (int u = 0; u < kI8Unroll; ++u) {
      const int q = g * kI8Unroll + u;
      int64_t k = (int64_t)q * 64 + 16 * fg;
      const bool kok = k < K && q < Q;
      if (!kok) k = 0;
      u32x4 v = *reinterpret_cast<const u32x4*>(Wq + wrow + k);
      if (!kok) v = u32x4{0u, 0u, 0u, 0u};
      a[u] = v;
#pragma unroll
      for (int f = 0; f < MT; ++f) {
        u32x4 x = *reinterpret_cast<const u32x4*>(Xq + xrow[f] + k);
        if (!kok) x = u32x4{0u, 0u, 0u, 0u};
        xb[u][f] = x;
      }
    }
#pragma unroll
    for (int u = 0; u < kI8Unroll; ++u)
#pragma unroll
      for (int f = 0; f < MT; ++f) acc[f] = mfma_i8(a[u], xb[u][f], acc[f]);
  }
  i8_finish<MT>(acc, part, wave, lane, n0, N, m0, M, sx, sw, Y, acc_out);
}

int i8_fragments(int64_t M) { return M <= 16 ? 1 : (M <= 32 ? 2 : 4); }

}  // namespace

hipError_t launch_sparse_int8(const int8_t* Xq, const float* sx, int64_t M, const spl_matrix& Wc, const float* sw,
                              void* Y, int32_t* acc_out, hipStream_t s) {
  const int MT = i8_fragments(M);
  const dim3 grid((unsigned)tile_blocks(Wc.rows), (unsigned)((M + 16 * MT - 1) / (16 * MT))), block(kI8Threads);
  const int8_t* vals = static_cast<const int8_t*>(Wc.values);
  const int any = Wc.nnz > 0 ? 1 : 0;
  uint16_t* y = static_cast<uint16_t*>(Y);
  if (MT == 1)
    hipLaunchKernelGGL((k_sparse_int8<1>), grid, block, 0, s, Xq, sx, M, Wc.cols, Wc.bitmask, vals, Wc.tile_offsets,
                       Wc.rows, sw, y, acc_out, any);
  else if (MT == 2)
    hipLaunchKernelGGL((k_sparse_int8<2>), grid, block, 0, s, Xq, sx, M, Wc.cols, Wc.bitmask, vals, Wc.tile_offsets,
                       Wc.rows, sw, y, acc_out, any);
  else
    hipLaunchKernelGGL((k_sparse_int8<4>), grid, block, 0, s, Xq, sx, M, Wc.cols, Wc.bitmask, vals, Wc.tile_offsets,
                       Wc.rows, sw, y, acc_out, any);
  return hipGetLastError();
}

hipError_t launch_dense_int8(const int8_t* Xq, const float* sx, int64_t M, const int8_t* Wq, const float* sw,
                             int64_t N, int64_t K, void* Y, int32_t* acc_out, hipStream_t s) {
  const int MT = i8_fragments(M);
  const dim3 grid((unsigned)((N + 15) / 16), (unsigned)((M + 16 * MT - 1) / (16 * MT))), block(kI8Threads);
  uint16_t* y = static_cast<uint16_t*>(Y);
  if (MT == 1)
    hipLaunchKernelGGL((k_dense_int8<1>), grid, block, 0, s, Xq, sx, M, K, Wq, N, sw, y, acc_out);
  else if (MT == 2)
    hipLaunchKernelGGL((k_dense_int8<2>), grid, block, 0, s, Xq, sx, M, K, Wq, N, sw, y, acc_out);
  else
    hipLaunchKernelGGL((k_dense_int8<4>), grid, block, 0, s, Xq, sx, M, K, Wq, N, sw, y, acc_out);
  return hipGetLastError();
}

}  // namespace spl
