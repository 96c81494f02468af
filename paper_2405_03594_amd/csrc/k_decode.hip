// Decode-shaped kernels (batch M <= 32) for gfx950.
//
// Sparse (paper section 2.4.2): compressed submatrices are moved from HBM
// on-chip and expanded there under the bitmask, then the matrix cores
// multiply them as if they were dense.  Here the submatrix is a 16-row block
// of W by a 256-column chunk; each wave of the workgroup owns every eighth
// chunk of the block:
//   1. the 16 rows' value spans of the chunk are copied HBM -> LDS with 16-byte
//      loads (four lanes per row);
//   2. each lane owns 64 columns of one row (two bitmask words): it zeroes them
//      in an LDS dense tile and walks its set bits with find-first-set, writing
//      the stored values to their columns in order;
//   3. eight v_mfma_f32_16x16x32 steps multiply the tile (A: rows n, 32
//      columns k) with the activations (B: k x batch column m, read straight
//      from global memory; the batch is padded to 16 or 32 with zeros);
//   4. the eight waves' partial 16 x 16 tiles are summed in LDS in a fixed
//      order (deterministic) and rounded once to the output type.
// Dense comparator: the same schedule with the A operand loaded directly from
// the dense W rows.
#include "spl_common.h"

namespace spl {
namespace {

constexpr int kDecWaves = 8;
constexpr int kDecThreads = kDecWaves * kWave;
constexpr int kDecRows = 16;
constexpr int kDecChunk = 256;                       // columns per chunk
constexpr int kDecChunkWords = kDecChunk / 32;       // 8 bitmask words per row
constexpr int kDecTileStride = kDecChunk * 2 + 16;   // bytes per dense tile row (padded)
constexpr int kDecTileBytes = kDecRows * kDecTileStride;
constexpr int kDecStageStride = kDecChunk * 2 + 32;  // bytes per staged row span (alignment slack)
constexpr int kDecStageBytes = kDecRows * kDecStageStride;
constexpr int kDecWaveBytes = kDecTileBytes + kDecStageBytes;
constexpr int kDecMaxChunks = 256;                   // K <= 65536 (offset table fits LDS)

template <class T>
struct Mfma16;
template <>
struct Mfma16<Bf16> {
  static __device__ __forceinline__ f32x4 run(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
  }
};
template <>
struct Mfma16<F16> {
  static __device__ __forceinline__ f32x4 run(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                  0, 0);
  }
};

// Sum the waves' partial accumulators (lane layout of the 16x16 MFMA result:
// lane l, register i holds row 4*(l/16)+i, column l%16) and store Y[m][n].
template <class T, int MT>
__device__ __forceinline__ void reduce_store(unsigned char* smem, const f32x4* acc, int M, int64_t n0, int64_t N,
                                             uint16_t* __restrict__ Y) {
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  __syncthreads();
  float* red = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int t = 0; t < MT; ++t) *reinterpret_cast<f32x4*>(red + ((wave * MT + t) * 64 + lane) * 4) = acc[t];
  __syncthreads();
  for (int e = threadIdx.x; e < 256 * MT; e += kDecThreads) {
    const int t = e >> 8;
    const int li = (e >> 2) & 63;
    const int ri = e & 3;
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) s += red[((w * MT + t) * 64 + li) * 4 + ri];
    const int64_t n = n0 + 4 * (li >> 4) + ri;
    const int m = t * 16 + (li & 15);
    if (m < M && n < N) Y[(int64_t)m * N + n] = T::from_f32(s);
  }
}

template <class T, int MT>
__global__ void __launch_bounds__(kDecThreads) k_sparse_decode(const uint16_t* __restrict__ X, int M, int64_t K,
                                                               const uint32_t* __restrict__ bitmask,
                                                               const uint16_t* __restrict__ values,
                                                               const int32_t* __restrict__ row_offsets, int64_t N,
                                                               uint16_t* __restrict__ Y) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int64_t n0 = (int64_t)blockIdx.x * kDecRows;
  const int64_t words = words_per_row(K);
  const int nchunks = (int)((K + kDecChunk - 1) / kDecChunk);
  unsigned char* tile = smem + wave * kDecWaveBytes;
  unsigned char* stage = tile + kDecTileBytes;
  int32_t* choff = reinterpret_cast<int32_t*>(smem + kDecWaves * kDecWaveBytes);   // [nchunks][16]

  // decompression role: row r of the block, quarter q of the chunk (64 columns)
  const int r = lane >> 2;
  const int q = lane & 3;
  const int64_t n = n0 + r;
  const bool row_ok = n < N;
  const uint32_t* brow = bitmask + (row_ok ? n : 0) * words;

  // kept count of every (chunk, row), then per-row running offsets
  for (int c = wave; c < nchunks; c += kDecWaves) {
    const int64_t w0 = (int64_t)c * kDecChunkWords + 2 * q;
    uint32_t cnt = 0;
    if (row_ok && w0 < words) cnt += __popc(brow[w0]);
    if (row_ok && w0 + 1 < words) cnt += __popc(brow[w0 + 1]);
    cnt += __shfl_xor(cnt, 1);
    cnt += __shfl_xor(cnt, 2);
    if (q == 0) choff[c * kDecRows + r] = (int32_t)cnt;
  }
  __syncthreads();
  if (threadIdx.x < kDecRows) {
    const int rr = threadIdx.x;
    int32_t run = (n0 + rr < N) ? row_offsets[n0 + rr] : 0;
    for (int c = 0; c < nchunks; ++c) {
      const int32_t v = choff[c * kDecRows + rr];
      choff[c * kDecRows + rr] = run;
      run += v;
    }
  }
  __syncthreads();

  f32x4 acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int fr = lane & 15;   // MFMA operand row (A) / batch column (B)
  const int fg = lane >> 4;   // 8-column group inside a 32-column k-step
  const unsigned char* vbytes = reinterpret_cast<const unsigned char*>(values);

  for (int c = wave; c < nchunks; c += kDecWaves) {
    const int64_t w0 = (int64_t)c * kDecChunkWords + 2 * q;
    const uint32_t m0 = (row_ok && w0 < words) ? brow[w0] : 0u;
    const uint32_t m1 = (row_ok && w0 + 1 < words) ? brow[w0 + 1] : 0u;
    const uint32_t cnt = __popc(m0) + __popc(m1);
    uint32_t incl = cnt;
    uint32_t up = __shfl_up(incl, 1, 4);
    if (q >= 1) incl += up;
    up = __shfl_up(incl, 2, 4);
    if (q >= 2) incl += up;
    const uint32_t row_cnt = __shfl(incl, (lane & ~3) + 3);   // kept entries of row r in this chunk

    // 1. copy the row's value span into the staging area, 16-byte pieces
    const int64_t vstart = choff[c * kDecRows + r];
    const int64_t b0 = (vstart * 2) & ~int64_t(15);
    const int64_t b1 = (vstart + (int64_t)row_cnt) * 2;
    const int npieces = row_cnt ? (int)((b1 - b0 + 15) >> 4) : 0;
    unsigned char* srow = stage + r * kDecStageStride;
    for (int p = q; p < npieces; p += 4)
      *reinterpret_cast<u32x4*>(srow + p * 16) = *reinterpret_cast<const u32x4*>(vbytes + b0 + p * 16);

    // 2. zero my 64 columns of the dense tile and expand my stored values into them
    unsigned char* trow = tile + r * kDecTileStride + q * 128;
#pragma unroll
    for (int i = 0; i < 8; ++i) *reinterpret_cast<u32x4*>(trow + i * 16) = u32x4{0u, 0u, 0u, 0u};
    wave_lds_sync();
    const uint16_t* src = reinterpret_cast<const uint16_t*>(srow + (vstart * 2 - b0)) + (incl - cnt);
    uint32_t m = m0;
    while (m) {
      const int b = __builtin_ctz(m);
      m &= m - 1;
      *reinterpret_cast<uint16_t*>(trow + b * 2) = *src++;
    }
    m = m1;
    while (m) {
      const int b = __builtin_ctz(m);
      m &= m - 1;
      *reinterpret_cast<uint16_t*>(trow + 64 + b * 2) = *src++;
    }
    wave_lds_sync();

    // 3. eight MFMA k-steps over the chunk
#pragma unroll
    for (int s = 0; s < kDecChunk / 32; ++s) {
      const u32x4 a = *reinterpret_cast<const u32x4*>(tile + fr * kDecTileStride + s * 64 + fg * 16);
      const int64_t k = (int64_t)c * kDecChunk + s * 32 + fg * 8;
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        const int mm = t * 16 + fr;
        u32x4 bv = {0u, 0u, 0u, 0u};
        if (mm < M && k < K) bv = *reinterpret_cast<const u32x4*>(X + (int64_t)mm * K + k);
        acc[t] = Mfma16<T>::run(a, bv, acc[t]);
      }
    }
    wave_lds_sync();
  }

  reduce_store<T, MT>(smem, acc, M, n0, N, Y);
}

template <class T, int MT>
__global__ void __launch_bounds__(kDecThreads) k_dense_decode(const uint16_t* __restrict__ X, int M, int64_t K,
                                                              const uint16_t* __restrict__ W, int64_t N,
                                                              uint16_t* __restrict__ Y) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int64_t n0 = (int64_t)blockIdx.x * kDecRows;
  const int fr = lane & 15;
  const int fg = lane >> 4;
  const int64_t nrow = n0 + fr;
  const bool rok = nrow < N;
  const uint16_t* wrow = W + (rok ? nrow : 0) * K;
  f32x4 acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int64_t nsteps = (K + 31) / 32;
  constexpr int U = 4;
  for (int64_t s0 = (int64_t)wave * U; s0 < nsteps; s0 += (int64_t)kDecWaves * U) {
    u32x4 a[U];
    u32x4 bv[U][MT];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t k = (s0 + u) * 32 + fg * 8;
      a[u] = u32x4{0u, 0u, 0u, 0u};
      if (rok && k < K) a[u] = *reinterpret_cast<const u32x4*>(wrow + k);
#pragma unroll
      for (int t = 0; t < MT; ++t) {
        const int mm = t * 16 + fr;
        bv[u][t] = u32x4{0u, 0u, 0u, 0u};
        if (mm < M && k < K) bv[u][t] = *reinterpret_cast<const u32x4*>(X + (int64_t)mm * K + k);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int t = 0; t < MT; ++t) acc[t] = Mfma16<T>::run(a[u], bv[u][t], acc[t]);
  }
  reduce_store<T, MT>(smem, acc, M, n0, N, Y);
}

template <class T>
hipError_t sparse_decode_t(const void* X, int64_t M, const spl_matrix& Wc, void* Y, hipStream_t s) {
  const int nchunks = (int)((Wc.cols + kDecChunk - 1) / kDecChunk);
  const size_t lds = (size_t)kDecWaves * kDecWaveBytes + (size_t)nchunks * kDecRows * sizeof(int32_t);
  const dim3 grid((unsigned)((Wc.rows + kDecRows - 1) / kDecRows)), block(kDecThreads);
  const auto* x = static_cast<const uint16_t*>(X);
  const auto* v = static_cast<const uint16_t*>(Wc.values);
  auto* y = static_cast<uint16_t*>(Y);
  if (M <= 16) {
    hipLaunchKernelGGL((k_sparse_decode<T, 1>), grid, block, lds, s, x, (int)M, Wc.cols, Wc.bitmask, v,
                       Wc.row_offsets, Wc.rows, y);
  } else {
    hipLaunchKernelGGL((k_sparse_decode<T, 2>), grid, block, lds, s, x, (int)M, Wc.cols, Wc.bitmask, v,
                       Wc.row_offsets, Wc.rows, y);
  }
  return hipGetLastError();
}

template <class T>
hipError_t dense_decode_t(const void* X, int64_t M, const void* W, int64_t N, int64_t K, void* Y, hipStream_t s) {
  const size_t lds = (size_t)kDecWaves * 2 * 64 * 16;
  const dim3 grid((unsigned)((N + kDecRows - 1) / kDecRows)), block(kDecThreads);
  const auto* x = static_cast<const uint16_t*>(X);
  const auto* w = static_cast<const uint16_t*>(W);
  auto* y = static_cast<uint16_t*>(Y);
  if (M <= 16) {
    hipLaunchKernelGGL((k_dense_decode<T, 1>), grid, block, lds, s, x, (int)M, K, w, N, y);
  } else {
    hipLaunchKernelGGL((k_dense_decode<T, 2>), grid, block, lds, s, x, (int)M, K, w, N, y);
  }
  return hipGetLastError();
}

}  // namespace

int decode_max_k() { return kDecMaxChunks * kDecChunk; }

hipError_t launch_sparse_decode(const void* X, int64_t M, const spl_matrix& Wc, void* Y, hipStream_t s) {
  return Wc.dtype == SPL_BF16 ? sparse_decode_t<Bf16>(X, M, Wc, Y, s) : sparse_decode_t<F16>(X, M, Wc, Y, s);
}

hipError_t launch_dense_decode(const void* X, int64_t M, const void* W, int32_t dtype, int64_t N, int64_t K,
                               void* Y, hipStream_t s) {
  return dtype == SPL_BF16 ? dense_decode_t<Bf16>(X, M, W, N, K, Y, s) : dense_decode_t<F16>(X, M, W, N, K, Y, s);
}

}  // namespace spl
