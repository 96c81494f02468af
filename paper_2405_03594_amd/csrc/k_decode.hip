// Decode-shaped kernels (batch M <= 32) for gfx950.
//
// Sparse (paper section 2.4.2): compressed submatrices move from HBM into the
// register file, the bitmask guides their expansion there, and the matrix
// cores consume the expanded operand as if it were dense.  On CDNA4:
//
//   * W is stored as 16 x 32 tiles, each with its 16 bitmask words and its
//     dense values (one tile = one MFMA A operand).  A workgroup owns one
//     16-row block; its 16 waves split the block's k-steps (tiles) into
//     contiguous ranges, so a 4096-column matrix gives every wave 8 tiles;
//   * the values of consecutive tiles are contiguous, so a wave fetches a
//     whole chunk of tiles (as many as fit a 4 KB staging buffer, at most 8)
//     with aligned, coalesced 16-byte loads into its LDS buffer; the chunk's
//     bitmask words arrive with one coalesced load per 4 tiles and are
//     regrouped by row in LDS, and tile offsets come through the scalar cache;
//   * lane (fr, fg) supplies tile row fr, columns 8fg..8fg+7, exactly its A
//     operand of v_mfma_f32_16x16x32 (8 bf16/fp16 values).  Their offset in the
//     stored values is the tile offset + the kept count of the tile rows above
//     (a 16-lane DPP scan of popcounts, two k-steps per scan in 16-bit halves)
//     + the popcount of the lower bits of the row's word.  Each 4-column
//     nibble's values are read from LDS as an 8-byte window (aligned dword
//     reads + v_alignbyte_b32) and a 256-entry selector table expands them
//     with v_perm_b32 into the operand dwords (zero bytes where the bit is
//     clear);
//   * activations form the B operand (batch padded to 16 or 32 columns; the
//     padding lanes hold zeros).  When M x K fits 48 KB the workgroup copies
//     X into LDS once; otherwise each k-step's operand is loaded directly;
//   * the waves' partial 16x16 results are summed in a fixed order
//     (deterministic) and rounded once to the output type.
//
// Dense comparator: the same schedule with the A operand loaded directly from
// the dense rows of W (aligned 16-byte loads).
#include <type_traits>

#include "spl_common.h"

namespace spl {
namespace {

constexpr int kDecWaves = 16;
constexpr int kDecThreads = kDecWaves * kWave;
constexpr int kDecRows = 16;
constexpr int kVBuf = 4096;                 // staged value bytes per wave and chunk
constexpr int kVBufAlloc = kVBuf + 16;      // + room for the last 8-byte window's third dword
constexpr int kXLdsMax = 48 * 1024;         // activations staged in LDS when M*K*2 fits

// k-steps per chunk: every load of a chunk is in flight at once, so the
// register budget (<= 128 VGPRs for 4 waves per SIMD) sets it.
template <int MT>
struct DecChunk {
  static constexpr int C = MT == 1 ? 8 : 4;
};

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

// Inclusive prefix sum across each group of 16 lanes (DPP row shifts).
__device__ __forceinline__ uint32_t row16_inclusive_scan(uint32_t x) {
  x += __builtin_amdgcn_update_dpp(0u, x, 0x111, 0xf, 0xf, false);   // row_shr:1
  x += __builtin_amdgcn_update_dpp(0u, x, 0x112, 0xf, 0xf, false);   // row_shr:2
  x += __builtin_amdgcn_update_dpp(0u, x, 0x114, 0xf, 0xf, false);   // row_shr:4
  x += __builtin_amdgcn_update_dpp(0u, x, 0x118, 0xf, 0xf, false);   // row_shr:8
  return x;
}

// This wave's contiguous range of k-steps [*beg, *end) of S.
__device__ __forceinline__ void wave_range(int S, int wave, int* beg, int* end) {
  const int L = (S + kDecWaves - 1) / kDecWaves;
  const int b = wave * L < S ? wave * L : S;
  *beg = b;
  *end = b + L < S ? b + L : S;
}

// Activation operand read directly from X: lane (fr, fg) of batch tile t
// reads X[16t + fr][32s + 8fg .. +8]; rows past M are not read (zeros).
template <int MT>
struct XGlobal {
  const uint16_t* row[MT];
  bool live[MT];
  __device__ __forceinline__ XGlobal(const uint16_t* __restrict__ X, int M, int64_t K, int fr, int fg) {
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      const int m = 16 * t + fr;
      live[t] = m < M;
      row[t] = X + (int64_t)(live[t] ? m : 0) * K + 8 * fg;
    }
  }
  // k-step s; kin: this lane's 8 columns lie inside [0, K)
  __device__ __forceinline__ void load(u32x4 (&xb)[MT], int s, bool kin) const {
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      xb[t] = u32x4{0u, 0u, 0u, 0u};
      if (kin && live[t]) xb[t] = *reinterpret_cast<const u32x4*>(row[t] + 32 * (int64_t)s);
    }
  }
};

// Activations staged in LDS (MT == 1, M*K*2 <= kXLdsMax): rows of K + 8
// elements (the 16-byte pad spreads rows over the LDS banks).
struct XShared {
  const uint16_t* row;
  bool live;
  __device__ __forceinline__ XShared(const uint16_t* xs, int M, int64_t K, int fr, int fg) {
    live = fr < M;
    row = xs + (int64_t)(live ? fr : 0) * (K + 8) + 8 * fg;
  }
  __device__ __forceinline__ void load(u32x4 (&xb)[1], int s, bool kin) const {
    xb[0] = u32x4{0u, 0u, 0u, 0u};
    if (kin && live) xb[0] = *reinterpret_cast<const u32x4*>(row + 32 * s);
  }
};

// Cooperative copy of X [M][K] into LDS rows of K + 8 elements.
__device__ __forceinline__ void stage_x(uint16_t* xs, const uint16_t* __restrict__ X, int M, int64_t K) {
  const int per_row = (int)(K / 8);
  const int total = M * per_row;
  for (int p = threadIdx.x; p < total; p += kDecThreads) {
    const int m = p / per_row, q = p - m * per_row;
    *reinterpret_cast<u32x4*>(xs + (int64_t)m * (K + 8) + 8 * q) =
        *reinterpret_cast<const u32x4*>(X + (int64_t)m * K + 8 * q);
  }
}

// Sum the waves' partial accumulators (lane layout of the 16x16 MFMA result:
// lane l, register i holds row 4*(l/16)+i, column l%16) and store Y[m][n].
// Called by every thread after all waves have finished with `red`'s memory.
template <class T, int MT>
__device__ __forceinline__ void reduce_store(float* red, const f32x4 (&acc)[MT], int M, int64_t n0, int64_t N,
                                             uint16_t* __restrict__ Y) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int t = 0; t < MT; ++t) *reinterpret_cast<f32x4*>(red + ((wave * MT + t) * 64 + lane) * 4) = acc[t];
  __syncthreads();
  for (int e = threadIdx.x; e < 256 * MT; e += kDecThreads) {
    const int t = e >> 8;
    const int li = (e >> 2) & 63;
    const int ri = e & 3;
    const int64_t n = n0 + 4 * (li >> 4) + ri;
    const int m = t * 16 + (li & 15);
    if (m < M && n < N) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < kDecWaves; ++w) s += red[((w * MT + t) * 64 + li) * 4 + ri];
      Y[(int64_t)m * N + n] = T::from_f32(s);
    }
  }
}

// Dynamic LDS: per-wave value staging buffers, then (XL) the staged activations.
__host__ __device__ constexpr size_t dec_vbuf_bytes() { return (size_t)kDecWaves * kVBufAlloc; }

template <class T, int MT, bool XL>
__global__ void __launch_bounds__(kDecThreads) k_sparse_decode(const uint16_t* __restrict__ X, int M, int64_t K,
                                                               const uint32_t* __restrict__ bm_tiles,
                                                               const uint16_t* __restrict__ values,
                                                               const int32_t* __restrict__ tile_offsets, int64_t N,
                                                               uint16_t* __restrict__ Y) {
  constexpr int C = DecChunk<MT>::C;
  extern __shared__ __align__(16) unsigned char dsm[];
  __shared__ u32x4 lut[256];
  __shared__ __align__(16) uint32_t words[kDecWaves][16 * C];   // per wave: [row][tile of the chunk]
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int fr = lane & 15, fg = lane >> 4;
  const int64_t blk = blockIdx.x;
  const int S = (int)tile_steps(K);
  int kbeg, kend;
  wave_range(S, wave, &kbeg, &kend);
  unsigned char* vbuf = dsm + wave * kVBufAlloc;
  const uint32_t* vbuf32 = reinterpret_cast<const uint32_t*>(vbuf);
  uint16_t* xs = reinterpret_cast<uint16_t*>(dsm + dec_vbuf_bytes());

  build_selector_table(lut);
  if constexpr (XL) stage_x(xs, X, M, K);
  __syncthreads();

  const uint32_t* bmb = bm_tiles + blk * S * 16;      // this row block's tiles, 16 words each
  const int32_t* tob = tile_offsets + blk * S;        // + S + 1 entries (the next block's first = this end)
  const unsigned char* vbytes = reinterpret_cast<const unsigned char*>(values);
  using XOp = std::conditional_t<XL, XShared, XGlobal<MT>>;
  const XOp xop = [&]() {
    if constexpr (XL) return XShared(xs, M, K, fr, fg);
    else return XGlobal<MT>(X, M, K, fr, fg);
  }();
  const uint32_t lowmask = (1u << (8 * fg)) - 1u;      // bits of the word below my byte
  uint32_t* wl = words[wave];

  f32x4 acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int c0 = kbeg; c0 < kend;) {
    // tile offsets of the chunk's tiles and of its end (wave-uniform: scalar loads)
    int32_t to[C + 1];
#pragma unroll
    for (int j = 0; j <= C; ++j) to[j] = tob[c0 + j < kend ? c0 + j : kend];
    // chunk length: the most tiles (<= C, inside the range) whose values fit the staging buffer
    const uint32_t a0 = (2u * (uint32_t)to[0]) & ~15u;
    int cn = 1;
#pragma unroll
    for (int j = 2; j <= C; ++j)
      if (c0 + j <= kend && ((2u * (uint32_t)to[j] + 15u) & ~15u) - a0 <= (uint32_t)kVBuf) cn = j;
    const int np = (int)((2u * (uint32_t)to[cn] - a0 + 15u) >> 4);    // 16-byte pieces, <= kVBuf / 16

    // issue: value pieces, bitmask words, activations
    constexpr int kPieceRounds = kVBuf / 16 / kWave;
    u32x4 vp[kPieceRounds];
#pragma unroll
    for (int r = 0; r < kPieceRounds; ++r) {
      vp[r] = u32x4{0u, 0u, 0u, 0u};
      if (lane + kWave * r < np)
        vp[r] = *reinterpret_cast<const u32x4*>(vbytes + a0 + 16u * (uint32_t)(lane + kWave * r));
    }
    uint32_t wv[C / 4];
#pragma unroll
    for (int i = 0; i < C / 4; ++i) {
      wv[i] = 0u;
      if (fg + 4 * i < cn) wv[i] = bmb[(int64_t)(c0 + fg + 4 * i) * 16 + fr];
    }
    u32x4 xb[C][MT];
#pragma unroll
    for (int j = 0; j < C; ++j) xop.load(xb[j], c0 + j, j < cn && 32 * (int64_t)(c0 + j) + 8 * fg < K);

    // stage values and regroup words by row
#pragma unroll
    for (int r = 0; r < kPieceRounds; ++r)
      if (lane + kWave * r < np) *reinterpret_cast<u32x4*>(vbuf + 16 * (lane + kWave * r)) = vp[r];
#pragma unroll
    for (int i = 0; i < C / 4; ++i) wl[fr * C + fg + 4 * i] = wv[i];
    wave_lds_sync();
    uint32_t w[C];
#pragma unroll
    for (int q = 0; q < C / 4; ++q) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(wl + fr * C + 4 * q);
      w[4 * q] = v.x;
      w[4 * q + 1] = v.y;
      w[4 * q + 2] = v.z;
      w[4 * q + 3] = v.w;
    }
    // kept count of the rows above mine, two tiles per scan (16-bit halves, sums <= 512)
    uint32_t above[C];
#pragma unroll
    for (int j = 0; j < C; j += 2) {
      const uint32_t pc = __popc(w[j]) | (__popc(w[j + 1]) << 16);
      const uint32_t ex = row16_inclusive_scan(pc) - pc;
      above[j] = ex & 0xffffu;
      above[j + 1] = ex >> 16;
    }
#pragma unroll
    for (int j = 0; j < C; ++j) {
      if (j < cn) {
        const uint32_t byte = (w[j] >> (8 * fg)) & 0xffu;
        const uint32_t oa = (uint32_t)to[j] + above[j] + __popc(w[j] & lowmask);
        const uint32_t ob = oa + __popc(byte & 0xfu);
        // 8-byte windows at byte positions pa, pb of the staging buffer
        const uint32_t pa = 2u * oa - a0, pb = 2u * ob - a0;
        const uint32_t qa = pa >> 2, qb = pb >> 2, sa = pa & 3u, sb = pb & 3u;
        const uint32_t a_0 = vbuf32[qa], a_1 = vbuf32[qa + 1], a_2 = vbuf32[qa + 2];
        const uint32_t b_0 = vbuf32[qb], b_1 = vbuf32[qb + 1], b_2 = vbuf32[qb + 2];
        const uint32_t vlo = __builtin_amdgcn_alignbyte(a_1, a_0, sa), vhi = __builtin_amdgcn_alignbyte(a_2, a_1, sa);
        const uint32_t ulo = __builtin_amdgcn_alignbyte(b_1, b_0, sb), uhi = __builtin_amdgcn_alignbyte(b_2, b_1, sb);
        const u32x4 sel = lut[byte];
        u32x4 a;
        a.x = __builtin_amdgcn_perm(vhi, vlo, sel.x);
        a.y = __builtin_amdgcn_perm(vhi, vlo, sel.y);
        a.z = __builtin_amdgcn_perm(uhi, ulo, sel.z);
        a.w = __builtin_amdgcn_perm(uhi, ulo, sel.w);
#pragma unroll
        for (int t = 0; t < MT; ++t) acc[t] = Mfma16<T>::run(a, xb[j][t], acc[t]);
      }
    }
    wave_lds_sync();                                   // the next chunk overwrites the buffers
    c0 += cn;
  }
  __syncthreads();                                     // every wave is done with its staging buffer
  reduce_store<T, MT>(reinterpret_cast<float*>(dsm), acc, M, blk * kDecRows, N, Y);
}

template <class T, int MT, bool XL>
__global__ void __launch_bounds__(kDecThreads) k_dense_decode(const uint16_t* __restrict__ X, int M, int64_t K,
                                                              const uint16_t* __restrict__ W, int64_t N,
                                                              uint16_t* __restrict__ Y) {
  constexpr int C = DecChunk<MT>::C;
  extern __shared__ __align__(16) unsigned char dsm[];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int fr = lane & 15, fg = lane >> 4;
  const int64_t blk = blockIdx.x;
  const int S = (int)tile_steps(K);
  int kbeg, kend;
  wave_range(S, wave, &kbeg, &kend);
  uint16_t* xs = reinterpret_cast<uint16_t*>(dsm + dec_vbuf_bytes());
  if constexpr (XL) stage_x(xs, X, M, K);
  __syncthreads();
  const int64_t row = blk * kDecRows + fr < N ? blk * kDecRows + fr : N - 1;   // rows past N feed discarded outputs
  const uint16_t* wrow = W + row * K + 8 * fg;
  using XOp = std::conditional_t<XL, XShared, XGlobal<MT>>;
  const XOp xop = [&]() {
    if constexpr (XL) return XShared(xs, M, K, fr, fg);
    else return XGlobal<MT>(X, M, K, fr, fg);
  }();

  f32x4 acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int c0 = kbeg; c0 < kend; c0 += C) {
    u32x4 a[C];
    u32x4 xb[C][MT];
#pragma unroll
    for (int j = 0; j < C; ++j) {
      const int s = c0 + j;
      const bool kin = s < kend && 32 * (int64_t)s + 8 * fg < K;
      a[j] = u32x4{0u, 0u, 0u, 0u};
      if (kin) a[j] = *reinterpret_cast<const u32x4*>(wrow + 32 * (int64_t)s);
      xop.load(xb[j], s, kin);
    }
#pragma unroll
    for (int j = 0; j < C; ++j)
#pragma unroll
      for (int t = 0; t < MT; ++t) acc[t] = Mfma16<T>::run(a[j], xb[j][t], acc[t]);
  }
  reduce_store<T, MT>(reinterpret_cast<float*>(dsm), acc, M, blk * kDecRows, N, Y);
}

__global__ void __launch_bounds__(256) k_zero_out(uint16_t* __restrict__ Y, int64_t count) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count; i += (int64_t)gridDim.x * 256) Y[i] = 0;
}

bool x_in_lds(int64_t M, int64_t K) { return M <= 16 && M * K * 2 <= kXLdsMax; }

size_t x_lds_bytes(int64_t M, int64_t K) { return (size_t)M * (size_t)(K + 8) * 2; }

// Raise the kernel's dynamic LDS limit once (it is above the 64 KB default).
template <class F>
hipError_t allow_lds(F* kernel, size_t bytes) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                             (int)bytes);
}

template <class T, int MT, bool XL>
hipError_t sparse_decode_launch(const void* X, int64_t M, const spl_matrix& Wc, void* Y, hipStream_t s) {
  auto* kernel = k_sparse_decode<T, MT, XL>;
  const size_t lds = dec_vbuf_bytes() + (XL ? x_lds_bytes(M, Wc.cols) : 0);
  static const hipError_t attr = allow_lds(kernel, dec_vbuf_bytes() + (XL ? x_lds_bytes(16, kXLdsMax / 32) : 0));
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(kernel, dim3((unsigned)tile_blocks(Wc.rows)), dim3(kDecThreads), lds, s,
                     static_cast<const uint16_t*>(X), (int)M, Wc.cols, Wc.bitmask,
                     static_cast<const uint16_t*>(Wc.values), Wc.tile_offsets, Wc.rows, static_cast<uint16_t*>(Y));
  return hipGetLastError();
}

template <class T>
hipError_t sparse_decode_t(const void* X, int64_t M, const spl_matrix& Wc, void* Y, hipStream_t s) {
  if (Wc.nnz == 0) return launch_zero_fill(Y, M * Wc.rows, s);
  if (x_in_lds(M, Wc.cols)) return sparse_decode_launch<T, 1, true>(X, M, Wc, Y, s);
  if (M <= 16) return sparse_decode_launch<T, 1, false>(X, M, Wc, Y, s);
  return sparse_decode_launch<T, 2, false>(X, M, Wc, Y, s);
}

template <class T, int MT, bool XL>
hipError_t dense_decode_launch(const void* X, int64_t M, const void* W, int64_t N, int64_t K, void* Y,
                               hipStream_t s) {
  auto* kernel = k_dense_decode<T, MT, XL>;
  const size_t lds = dec_vbuf_bytes() + (XL ? x_lds_bytes(M, K) : 0);
  static const hipError_t attr = allow_lds(kernel, dec_vbuf_bytes() + (XL ? x_lds_bytes(16, kXLdsMax / 32) : 0));
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(kernel, dim3((unsigned)tile_blocks(N)), dim3(kDecThreads), lds, s,
                     static_cast<const uint16_t*>(X), (int)M, K, static_cast<const uint16_t*>(W), N,
                     static_cast<uint16_t*>(Y));
  return hipGetLastError();
}

template <class T>
hipError_t dense_decode_t(const void* X, int64_t M, const void* W, int64_t N, int64_t K, void* Y, hipStream_t s) {
  if (x_in_lds(M, K)) return dense_decode_launch<T, 1, true>(X, M, W, N, K, Y, s);
  if (M <= 16) return dense_decode_launch<T, 1, false>(X, M, W, N, K, Y, s);
  return dense_decode_launch<T, 2, false>(X, M, W, N, K, Y, s);
}

}  // namespace

hipError_t launch_zero_fill(void* Y, int64_t count16, hipStream_t s) {
  int64_t blocks = (count16 + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_zero_out, dim3((unsigned)blocks), dim3(256), 0, s, static_cast<uint16_t*>(Y), count16);
  return hipGetLastError();
}

// No per-K limit: a wave walks its k-range in chunks.
int decode_max_k() { return 1 << 30; }

hipError_t launch_sparse_decode(const void* X, int64_t M, const spl_matrix& Wc, void* Y, hipStream_t s) {
  return Wc.dtype == SPL_BF16 ? sparse_decode_t<Bf16>(X, M, Wc, Y, s) : sparse_decode_t<F16>(X, M, Wc, Y, s);
}

hipError_t launch_dense_decode(const void* X, int64_t M, const void* W, int32_t dtype, int64_t N, int64_t K,
                               void* Y, hipStream_t s) {
  return dtype == SPL_BF16 ? dense_decode_t<Bf16>(X, M, W, N, K, Y, s) : dense_decode_t<F16>(X, M, W, N, K, Y, s);
}

}  // namespace spl
