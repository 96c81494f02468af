// Decode-shaped kernels (batch M <= 32) for gfx950.
//
// Sparse (paper section 2.4.2): compressed submatrices move from HBM into the
// register file, the bitmask guides their expansion there, and the matrix
// cores consume the expanded operand as if it were dense.  On CDNA4:
//
//   * W is stored as 16 x 32 tiles, each with its 16 bitmask words and its
//     dense values (one tile = one MFMA A operand); a workgroup owns a 16-row
//     block, its eight waves split the block's tiles into contiguous ranges
//     and stage their bitmask words in LDS with 16-byte loads;
//   * lane (fr, fg) supplies tile row fr, columns 8fg..8fg+7, exactly its A
//     operand of v_mfma_f32_16x16x32 (8 bf16/fp16 values);
//   * the stored-value offset of those columns is the tile offset + the kept
//     count of the tile rows above (16-lane DPP scan of popcounts) + the
//     popcount of the lower bits of the row's word; a tile's values are one
//     contiguous run, so a wave's loads touch few cache lines;
//     the values of each 4-column nibble are fetched with one unaligned 8-byte
//     load, and a 256-entry selector table expands them with v_perm_b32 into
//     the four operand dwords (zero bytes where the bit is clear);
//   * activations form the B operand (batch padded to 16 or 32; padded
//     columns hold copies of real rows and their outputs are discarded);
//   * loads run one group of eight k-steps ahead of the multiply, and the
//     eight waves' partial 16x16 results are summed in a fixed order
//     (deterministic) and rounded once to the output type.
//
// Dense comparator: the same schedule with the A operand loaded directly from
// the dense rows of W.
#include "spl_common.h"

namespace spl {
namespace {

constexpr int kDecWaves = 8;
constexpr int kDecThreads = kDecWaves * kWave;
constexpr int kDecRows = 16;
constexpr int kGroup = 4;                 // k-steps per pipeline stage
constexpr int kDecodeMaxK = 32 * 1536;    // per-wave bitmask words and tile offsets in LDS: <= ~105 KB

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

// v_perm_b32 selector for the two 16-bit elements (2h, 2h+1) of a 4-column
// nibble whose stored values sit, in order, in the 8 source bytes {hi:lo}:
// a kept element takes the two bytes of its rank, a dropped one 0x0C (zero).
__device__ __forceinline__ uint32_t nibble_selector(uint32_t nib, int h) {
  uint32_t sel = 0;
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    const int j = 2 * h + e;
    uint32_t s16 = 0x0C0Cu;
    if ((nib >> j) & 1u) {
      const uint32_t r = __popc(nib & ((1u << j) - 1u));
      s16 = (2u * r) | ((2u * r + 1u) << 8);
    }
    sel |= s16 << (16 * e);
  }
  return sel;
}

// Entry b expands bitmask byte b (two nibbles) into four operand dwords.
__device__ __forceinline__ void build_selector_table(u32x4* lut) {
  for (int b = threadIdx.x; b < 256; b += blockDim.x) {
    lut[b] = u32x4{nibble_selector(b & 15u, 0), nibble_selector(b & 15u, 1), nibble_selector(b >> 4, 0),
                   nibble_selector(b >> 4, 1)};
  }
}

// 8 bytes at any 2-byte aligned offset (gfx950 serves unaligned global loads).
__device__ __forceinline__ u32x2 load8_at(const unsigned char* __restrict__ base, uint32_t byte_off) {
  u32x2 v;
  __builtin_memcpy(&v, base + byte_off, 8);
  return v;
}

// Sum the waves' partial accumulators (lane layout of the 16x16 MFMA result:
// lane l, register i holds row 4*(l/16)+i, column l%16) and store Y[m][n].
template <class T, int MT>
__device__ __forceinline__ void reduce_store(float* red, const f32x4* acc, int M, int64_t n0, int64_t N,
                                             uint16_t* __restrict__ Y) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  const int lane = threadIdx.x & 63;
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

// B operand of k-step s for every batch tile: X[m][32s + 8fg .. +8].  The
// batch row m is clamped to M-1 (those columns only feed discarded outputs).
// Past K the A operand is zero (bitmask bits past K are zero) and the B
// operand is set to zero too, so no activation value is read out of range.
template <int MT>
__device__ __forceinline__ void load_x(u32x4 (&xb)[MT], const uint16_t* __restrict__ X, int M, int64_t K, int64_t s,
                                       int fr, int fg) {
  int64_t k = s * 32 + fg * 8;
  const bool in = k < K;
  if (!in) k = K - 8;
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    int mm = t * 16 + fr;
    if (mm > M - 1) mm = M - 1;
    xb[t] = *reinterpret_cast<const u32x4*>(X + (int64_t)mm * K + k);
    if (!in) xb[t] = u32x4{0u, 0u, 0u, 0u};
  }
}

// Inclusive prefix sum across each group of 16 lanes (DPP row shifts).
__device__ __forceinline__ uint32_t row16_inclusive_scan(uint32_t x) {
  x += __builtin_amdgcn_update_dpp(0u, x, 0x111, 0xf, 0xf, false);   // row_shr:1
  x += __builtin_amdgcn_update_dpp(0u, x, 0x112, 0xf, 0xf, false);   // row_shr:2
  x += __builtin_amdgcn_update_dpp(0u, x, 0x114, 0xf, 0xf, false);   // row_shr:4
  x += __builtin_amdgcn_update_dpp(0u, x, 0x118, 0xf, 0xf, false);   // row_shr:8
  return x;
}

template <class T, int MT>
__global__ void __launch_bounds__(kDecThreads) k_sparse_decode(const uint16_t* __restrict__ X, int M, int64_t K,
                                                               const uint32_t* __restrict__ bm_tiles,
                                                               const uint16_t* __restrict__ values,
                                                               const int32_t* __restrict__ tile_offsets, int64_t N,
                                                               uint16_t* __restrict__ Y) {
  // per wave: [Lmax + kGroup] tiles of 16 bitmask words, then [Lmax + kGroup] tile offsets
  extern __shared__ __align__(16) uint32_t smem[];
  __shared__ u32x4 lut[256];
  __shared__ float red[kDecWaves * MT * 64 * 4];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  const int lane = threadIdx.x & 63;
  const int64_t blk = blockIdx.x;
  const int64_t n0 = blk * kDecRows;
  const int S = (int)tile_steps(K);                 // 32-column k-steps = tiles per row block
  const int ks0 = (int)((int64_t)S * wave / kDecWaves);
  const int ks1 = (int)((int64_t)S * (wave + 1) / kDecWaves);
  const int L = ks1 - ks0;
  // padded tiles per wave region: the pipeline reads up to 2*kGroup - 1 slots
  // past its last tile, and those read as empty tiles
  const int Lp = (S + kDecWaves - 1) / kDecWaves + 2 * kGroup;
  uint32_t* wl = smem + wave * Lp * 17;              // words [Lp][16]
  int32_t* tl = reinterpret_cast<int32_t*>(wl + Lp * 16);   // tile offsets [Lp]

  build_selector_table(lut);

  // 1. this wave's tiles: bitmask words (64 B per tile, 16-byte loads) and tile
  //    offsets -> LDS; the region past the range reads as empty tiles
  {
    const u32x4* src = reinterpret_cast<const u32x4*>(bm_tiles + (blk * S + ks0) * 16);
    u32x4* dst = reinterpret_cast<u32x4*>(wl);
    const int nq = 4 * Lp;
    for (int q0 = 0; q0 < nq; q0 += 4 * kWave) {
      u32x4 w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int q = q0 + lane + i * kWave;
        w[i] = u32x4{0u, 0u, 0u, 0u};
        if (q < 4 * L) w[i] = src[q];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int q = q0 + lane + i * kWave;
        if (q < nq) dst[q] = w[i];
      }
    }
    const int32_t* toffs = tile_offsets + blk * S + ks0;
    for (int j = lane; j < Lp; j += kWave) tl[j] = toffs[j < L ? j : L];   // past the range: the range end
  }
  __syncthreads();

  // 2. expand and multiply; lane = (tile row fr, column group fg)
  const int fr = lane & 15;
  const int fg = lane >> 4;
  const uint32_t lowmask = (1u << (8 * fg)) - 1u;   // bits of the word below my byte
  const int byte_shift = 8 * fg;
  const unsigned char* vbytes = reinterpret_cast<const unsigned char*>(values);
  const unsigned char* xbytes = reinterpret_cast<const unsigned char*>(X);
  uint32_t xrow[MT];                                 // byte offset of X[m][0] (M*K*2 < 2^32)
#pragma unroll
  for (int t = 0; t < MT; ++t) {
    const int mm = t * 16 + fr < M ? t * 16 + fr : M - 1;
    xrow[t] = (uint32_t)((int64_t)mm * K * 2);
  }
  const uint32_t kmax = (uint32_t)K - 8u;           // last 8-column group inside a row of X
  const bool k_tail = (K & 31) != 0;                 // last k-step partly past K

  f32x4 acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};

  struct Stage {
    u32x2 v0[kGroup], v1[kGroup];
    uint32_t byte[kGroup];
    u32x4 xb[kGroup][MT];
  };
  // loads of the group starting j0 tiles into this wave's range
  auto issue = [&](Stage& st, int j0) {
    uint32_t w[kGroup];
    int32_t to[kGroup];
#pragma unroll
    for (int i = 0; i < kGroup; ++i) {
      const int j = j0 + i < Lp - 1 ? j0 + i : Lp - 1;   // wave-uniform; slots >= L are empty
      w[i] = wl[j * 16 + fr];
      to[i] = tl[j];
    }
#pragma unroll
    for (int i = 0; i < kGroup; ++i) {
      const uint32_t pc = __popc(w[i]);
      const uint32_t above = row16_inclusive_scan(pc) - pc;   // kept entries of the tile rows above mine
      const uint32_t b = (w[i] >> byte_shift) & 0xffu;
      const uint32_t oa = (uint32_t)to[i] + above + __popc(w[i] & lowmask);
      const uint32_t ob = oa + __popc(b & 0xfu);
      st.byte[i] = b;
      st.v0[i] = load8_at(vbytes, oa * 2u);
      st.v1[i] = load8_at(vbytes, ob * 2u);
      int sk = ks0 + j0 + i;                         // past the range: any in-range step (unused)
      if (sk > ks1 - 1) sk = ks1 - 1;
      uint32_t kc = (uint32_t)sk * 32u + 8u * (uint32_t)fg;
      kc = kc < kmax ? kc : kmax;                    // columns past K: zeroed before use
#pragma unroll
      for (int t = 0; t < MT; ++t)
        st.xb[i][t] = *reinterpret_cast<const u32x4*>(xbytes + xrow[t] + kc * 2u);
    }
  };
  auto consume = [&](Stage& st, int j0) {
#pragma unroll
    for (int i = 0; i < kGroup; ++i) {
      const int s = ks0 + j0 + i;
      if (s < ks1) {
        const u32x4 sel = lut[st.byte[i]];
        u32x4 a;
        a.x = __builtin_amdgcn_perm(st.v0[i].y, st.v0[i].x, sel.x);
        a.y = __builtin_amdgcn_perm(st.v0[i].y, st.v0[i].x, sel.y);
        a.z = __builtin_amdgcn_perm(st.v1[i].y, st.v1[i].x, sel.z);
        a.w = __builtin_amdgcn_perm(st.v1[i].y, st.v1[i].x, sel.w);
        if (k_tail && s == S - 1 && 32 * s + 8 * fg >= K) {
#pragma unroll
          for (int t = 0; t < MT; ++t) st.xb[i][t] = u32x4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int t = 0; t < MT; ++t) acc[t] = Mfma16<T>::run(a, st.xb[i][t], acc[t]);
      }
    }
  };
  if (L > 0) {
    Stage sa, sb;
    issue(sa, 0);
    for (int j0 = 0; j0 < L; j0 += 2 * kGroup) {
      issue(sb, j0 + kGroup);
      consume(sa, j0);
      if (j0 + kGroup >= L) break;
      issue(sa, j0 + 2 * kGroup);
      consume(sb, j0 + kGroup);
    }
  }
  reduce_store<T, MT>(red, acc, M, n0, N, Y);
}

template <class T, int MT>
__global__ void __launch_bounds__(kDecThreads) k_dense_decode(const uint16_t* __restrict__ X, int M, int64_t K,
                                                              const uint16_t* __restrict__ W, int64_t N,
                                                              uint16_t* __restrict__ Y) {
  __shared__ float red[kDecWaves * MT * 64 * 4];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  const int lane = threadIdx.x & 63;
  const int64_t n0 = (int64_t)blockIdx.x * kDecRows;
  const int64_t nsteps = (K + 31) / 32;
  const int64_t ks0 = nsteps * wave / kDecWaves;
  const int64_t ks1 = nsteps * (wave + 1) / kDecWaves;
  const int fr = lane & 15;
  const int fg = lane >> 4;
  const int64_t row = n0 + fr < N ? n0 + fr : N - 1;
  const uint16_t* wrow = W + row * K;
  f32x4 acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};

  struct Stage {
    u32x4 a[kGroup];
    u32x4 xb[kGroup][MT];
  };
  auto issue = [&](Stage& st, int64_t s0) {
#pragma unroll
    for (int i = 0; i < kGroup; ++i) {
      int64_t s = s0 + i;
      if (s > ks1 - 1) s = ks1 - 1;
      int64_t k = s * 32 + fg * 8;
      const bool in = k < K;
      if (!in) k = K - 8;
      st.a[i] = *reinterpret_cast<const u32x4*>(wrow + k);
      if (!in) st.a[i] = u32x4{0u, 0u, 0u, 0u};
      load_x<MT>(st.xb[i], X, M, K, s, fr, fg);
    }
  };
  auto consume = [&](const Stage& st, int64_t s0) {
#pragma unroll
    for (int i = 0; i < kGroup; ++i) {
      if (s0 + i < ks1) {
#pragma unroll
        for (int t = 0; t < MT; ++t) acc[t] = Mfma16<T>::run(st.a[i], st.xb[i][t], acc[t]);
      }
    }
  };
  if (ks1 > ks0) {
    Stage sa, sb;
    issue(sa, ks0);
    for (int64_t s0 = ks0; s0 < ks1; s0 += 2 * kGroup) {
      issue(sb, s0 + kGroup);
      consume(sa, s0);
      if (s0 + kGroup >= ks1) break;
      issue(sa, s0 + 2 * kGroup);
      consume(sb, s0 + kGroup);
    }
  }
  reduce_store<T, MT>(red, acc, M, n0, N, Y);
}

// With no stored value the product is exactly +0 everywhere.
__global__ void __launch_bounds__(256) k_zero_out(uint16_t* __restrict__ Y, int64_t count) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count; i += (int64_t)gridDim.x * 256) Y[i] = 0;
}

template <class T>
hipError_t sparse_decode_t(const void* X, int64_t M, const spl_matrix& Wc, void* Y, hipStream_t s) {
  if (Wc.nnz == 0) return launch_zero_fill(Y, M * Wc.rows, s);
  const dim3 grid((unsigned)((Wc.rows + kDecRows - 1) / kDecRows)), block(kDecThreads);
  const int64_t Lp = (tile_steps(Wc.cols) + kDecWaves - 1) / kDecWaves + 2 * kGroup;
  const size_t lds = (size_t)kDecWaves * Lp * 17 * sizeof(uint32_t);
  const auto* x = static_cast<const uint16_t*>(X);
  const auto* v = static_cast<const uint16_t*>(Wc.values);
  auto* y = static_cast<uint16_t*>(Y);
  if (M <= 16) {
    hipLaunchKernelGGL((k_sparse_decode<T, 1>), grid, block, lds, s, x, (int)M, Wc.cols, Wc.bitmask, v,
                       Wc.tile_offsets, Wc.rows, y);
  } else {
    hipLaunchKernelGGL((k_sparse_decode<T, 2>), grid, block, lds, s, x, (int)M, Wc.cols, Wc.bitmask, v,
                       Wc.tile_offsets, Wc.rows, y);
  }
  return hipGetLastError();
}

template <class T>
hipError_t dense_decode_t(const void* X, int64_t M, const void* W, int64_t N, int64_t K, void* Y, hipStream_t s) {
  const dim3 grid((unsigned)((N + kDecRows - 1) / kDecRows)), block(kDecThreads);
  const auto* x = static_cast<const uint16_t*>(X);
  const auto* w = static_cast<const uint16_t*>(W);
  auto* y = static_cast<uint16_t*>(Y);
  if (M <= 16) {
    hipLaunchKernelGGL((k_dense_decode<T, 1>), grid, block, 0, s, x, (int)M, K, w, N, y);
  } else {
    hipLaunchKernelGGL((k_dense_decode<T, 2>), grid, block, 0, s, x, (int)M, K, w, N, y);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_zero_fill(void* Y, int64_t count16, hipStream_t s) {
  int64_t blocks = (count16 + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_zero_out, dim3((unsigned)blocks), dim3(256), 0, s, static_cast<uint16_t*>(Y), count16);
  return hipGetLastError();
}

int decode_max_k() { return kDecodeMaxK; }

hipError_t launch_sparse_decode(const void* X, int64_t M, const spl_matrix& Wc, void* Y, hipStream_t s) {
  return Wc.dtype == SPL_BF16 ? sparse_decode_t<Bf16>(X, M, Wc, Y, s) : sparse_decode_t<F16>(X, M, Wc, Y, s);
}

hipError_t launch_dense_decode(const void* X, int64_t M, const void* W, int32_t dtype, int64_t N, int64_t K,
                               void* Y, hipStream_t s) {
  return dtype == SPL_BF16 ? dense_decode_t<Bf16>(X, M, W, N, K, Y, s) : dense_decode_t<F16>(X, M, W, N, K, Y, s);
}

}  // namespace spl
