// Prefill-shaped kernels (any batch M, sized for M >= 64) for gfx950.
//
// Sparse (paper section 2.4.2): the compressed 16 x 32 submatrices of W are
// expanded in registers into MFMA A operands (bitmask-guided v_perm_b32 of
// the stored values, as in the decode kernel) and multiplied at the dense
// rate against activation tiles staged in LDS.
//
//   * a workgroup (4 waves) owns a 64 (n) x 128 (m) output block; wave
//     (wn, wm) owns 32 x 64: two W tiles (rows) by four 16-column batch
//     fragments, i.e. eight v_mfma_f32_16x16x32 per 32-column k-step;
//   * activations X[m0 .. m0+128)[k-step] go HBM -> registers -> LDS, double
//     buffered two k-steps at a time; each wave reads its B operands with
//     16-byte LDS reads;
//   * W operands for the next k-step pair are fetched (words, tile offsets,
//     nibble windows) while the current pair is multiplied.
// Dense comparator: the same schedule with W operands loaded directly from
// the dense rows.
#include "spl_common.h"

namespace spl {
namespace {

constexpr int kPfThreads = 256;
constexpr int kPfBN = 64;                  // W rows per workgroup
constexpr int kPfBM = 128;                 // batch rows per workgroup
constexpr int kPfStage = 2;                // k-steps (32 columns each) per LDS stage
constexpr int kPfXStride = 64 + 16;        // bytes per staged activation row of one k-step (padded)
constexpr int kPfXStep = kPfBM * kPfXStride;          // bytes per k-step of staged activations
constexpr int kPfXBuf = kPfStage * kPfXStep;          // bytes per stage buffer

template <class T>
struct MfmaP;
template <>
struct MfmaP<Bf16> {
  static __device__ __forceinline__ f32x4 run(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
  }
};
template <>
struct MfmaP<F16> {
  static __device__ __forceinline__ f32x4 run(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                  0, 0);
  }
};

__device__ __forceinline__ uint32_t pf_nibble_selector(uint32_t nib, int h) {
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


// Activation staging: thread t moves X[m0 + t/2][32s + 16(t%2) .. +16] for
// the k-steps of one stage (two 16-byte pieces per k-step).  Rows past M and
// columns past K are zero.
struct XStage {
  u32x4 v[kPfStage][2];
};

__device__ __forceinline__ void x_fetch(XStage& st, const uint16_t* __restrict__ X, int64_t M, int64_t K, int64_t m0,
                                        int s0, int S) {
  const int t = threadIdx.x;
  const int64_t m = m0 + (t >> 1);
  const bool mok = m < M;
  const int64_t mm = mok ? m : M - 1;
#pragma unroll
  for (int j = 0; j < kPfStage; ++j) {
    const int s = s0 + j < S ? s0 + j : S - 1;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      int64_t k = (int64_t)s * 32 + (t & 1) * 16 + h * 8;
      const bool kok = k < K && s0 + j < S;
      if (k > K - 8) k = K - 8;
      u32x4 v = *reinterpret_cast<const u32x4*>(X + mm * K + k);
      if (!(mok && kok)) v = u32x4{0u, 0u, 0u, 0u};
      st.v[j][h] = v;
    }
  }
}

__device__ __forceinline__ void x_store(const XStage& st, unsigned char* buf) {
  const int t = threadIdx.x;
#pragma unroll
  for (int j = 0; j < kPfStage; ++j)
#pragma unroll
    for (int h = 0; h < 2; ++h)
      *reinterpret_cast<u32x4*>(buf + j * kPfXStep + (t >> 1) * kPfXStride + (t & 1) * 32 + h * 16) = st.v[j][h];
}

// W operands of one wave for one stage: two tiles x kPfStage k-steps.
struct WStage {
  u32x2 v0[kPfStage][2], v1[kPfStage][2];
  uint32_t byte[kPfStage][2];
};

template <class T>
__global__ void __launch_bounds__(kPfThreads) k_sparse_prefill(const uint16_t* __restrict__ X, int64_t M, int64_t K,
                                                               const uint32_t* __restrict__ bm_tiles,
                                                               const uint16_t* __restrict__ values,
                                                               const int32_t* __restrict__ tile_offsets, int64_t N,
                                                               uint16_t* __restrict__ Y) {
  __shared__ __align__(16) unsigned char xs[2][kPfXBuf];
  __shared__ u32x4 lut[256];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int wn = wave & 1, wm = wave >> 1;
  const int fr = lane & 15, fg = lane >> 4;
  const int S = (int)tile_steps(K);
  const int64_t B = tile_blocks(N);
  const int64_t m0 = (int64_t)blockIdx.y * kPfBM;
  const int64_t b0 = (int64_t)blockIdx.x * (kPfBN / 16) + 2 * wn;   // first of the wave's two tile rows
  const int64_t bt[2] = {b0 < B ? b0 : B - 1, b0 + 1 < B ? b0 + 1 : B - 1};
  const bool bok[2] = {b0 < B, b0 + 1 < B};

  for (int b = threadIdx.x; b < 256; b += kPfThreads)
    lut[b] = u32x4{pf_nibble_selector(b & 15u, 0), pf_nibble_selector(b & 15u, 1), pf_nibble_selector(b >> 4, 0),
                   pf_nibble_selector(b >> 4, 1)};

  const uint32_t lowmask = (1u << (8 * fg)) - 1u;
  const int byte_shift = 8 * fg;
  const unsigned char* vbytes = reinterpret_cast<const unsigned char*>(values);

  auto w_fetch = [&](WStage& ws, int s0) {
#pragma unroll
    for (int j = 0; j < kPfStage; ++j) {
      const int s = s0 + j < S ? s0 + j : S - 1;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int64_t t = bt[u] * S + s;
        uint32_t w = bm_tiles[t * 16 + fr];
        if (!bok[u] || s0 + j >= S) w = 0u;
        const uint32_t pc = __popc(w);
        const uint32_t above = row16_inclusive_scan(pc) - pc;
        const uint32_t b = (w >> byte_shift) & 0xffu;
        const uint32_t oa = (uint32_t)tile_offsets[t] + above + __popc(w & lowmask);
        const uint32_t ob = oa + __popc(b & 0xfu);
        ws.byte[j][u] = b;
        __builtin_memcpy(&ws.v0[j][u], vbytes + oa * 2u, 8);
        __builtin_memcpy(&ws.v1[j][u], vbytes + ob * 2u, 8);
      }
    }
  };

  f32x4 acc[2][4];
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int f = 0; f < 4; ++f) acc[u][f] = f32x4{0.f, 0.f, 0.f, 0.f};

  XStage xst;
  WStage ws;
  x_fetch(xst, X, M, K, m0, 0, S);
  w_fetch(ws, 0);
  x_store(xst, xs[0]);
  __syncthreads();
  int buf = 0;
  for (int s0 = 0; s0 < S; s0 += kPfStage) {
    const bool more = s0 + kPfStage < S;
    // expand this stage's W operands before the registers are refilled
    u32x4 a[kPfStage][2];
#pragma unroll
    for (int j = 0; j < kPfStage; ++j)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const u32x4 sel = lut[ws.byte[j][u]];
        a[j][u].x = __builtin_amdgcn_perm(ws.v0[j][u].y, ws.v0[j][u].x, sel.x);
        a[j][u].y = __builtin_amdgcn_perm(ws.v0[j][u].y, ws.v0[j][u].x, sel.y);
        a[j][u].z = __builtin_amdgcn_perm(ws.v1[j][u].y, ws.v1[j][u].x, sel.z);
        a[j][u].w = __builtin_amdgcn_perm(ws.v1[j][u].y, ws.v1[j][u].x, sel.w);
      }
    if (more) {
      x_fetch(xst, X, M, K, m0, s0 + kPfStage, S);
      w_fetch(ws, s0 + kPfStage);
    }
    const unsigned char* xb = xs[buf];
#pragma unroll
    for (int j = 0; j < kPfStage; ++j) {
      if (s0 + j < S) {
#pragma unroll
        for (int f = 0; f < 4; ++f) {
          const u32x4 bop = *reinterpret_cast<const u32x4*>(xb + j * kPfXStep + (wm * 64 + f * 16 + fr) * kPfXStride +
                                                            fg * 16);
#pragma unroll
          for (int u = 0; u < 2; ++u) acc[u][f] = MfmaP<T>::run(a[j][u], bop, acc[u][f]);
        }
      }
    }
    if (more) {
      x_store(xst, xs[buf ^ 1]);
      __syncthreads();
      buf ^= 1;
    }
  }

  // D layout: lane l, register i -> row (n) 4*(l/16)+i of the tile, column (m) l%16
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int64_t nb = (b0 + u) * 16 + 4 * fg;
#pragma unroll
    for (int f = 0; f < 4; ++f) {
      const int64_t m = m0 + wm * 64 + f * 16 + fr;
      if (m < M && b0 + u < B) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (nb + i < N) Y[m * N + nb + i] = T::from_f32(acc[u][f][i]);
      }
    }
  }
}

template <class T>
__global__ void __launch_bounds__(kPfThreads) k_dense_prefill(const uint16_t* __restrict__ X, int64_t M, int64_t K,
                                                              const uint16_t* __restrict__ W, int64_t N,
                                                              uint16_t* __restrict__ Y) {
  __shared__ __align__(16) unsigned char xs[2][kPfXBuf];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int wn = wave & 1, wm = wave >> 1;
  const int fr = lane & 15, fg = lane >> 4;
  const int S = (int)tile_steps(K);
  const int64_t m0 = (int64_t)blockIdx.y * kPfBM;
  const int64_t n0 = (int64_t)blockIdx.x * kPfBN + 32 * wn;
  const int64_t rows[2] = {n0 + fr < N ? n0 + fr : N - 1, n0 + 16 + fr < N ? n0 + 16 + fr : N - 1};

  struct WD {
    u32x4 a[kPfStage][2];
  };
  auto w_fetch = [&](WD& wd, int s0) {
#pragma unroll
    for (int j = 0; j < kPfStage; ++j) {
      const int s = s0 + j < S ? s0 + j : S - 1;
      int64_t k = (int64_t)s * 32 + fg * 8;
      const bool kok = k < K && s0 + j < S;
      if (k > K - 8) k = K - 8;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        u32x4 v = *reinterpret_cast<const u32x4*>(W + rows[u] * K + k);
        if (!kok) v = u32x4{0u, 0u, 0u, 0u};
        wd.a[j][u] = v;
      }
    }
  };
  f32x4 acc[2][4];
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int f = 0; f < 4; ++f) acc[u][f] = f32x4{0.f, 0.f, 0.f, 0.f};

  XStage xst;
  WD wd;
  x_fetch(xst, X, M, K, m0, 0, S);
  w_fetch(wd, 0);
  x_store(xst, xs[0]);
  __syncthreads();
  int buf = 0;
  for (int s0 = 0; s0 < S; s0 += kPfStage) {
    const bool more = s0 + kPfStage < S;
    WD cur = wd;
    if (more) {
      x_fetch(xst, X, M, K, m0, s0 + kPfStage, S);
      w_fetch(wd, s0 + kPfStage);
    }
    const unsigned char* xb = xs[buf];
#pragma unroll
    for (int j = 0; j < kPfStage; ++j) {
      if (s0 + j < S) {
#pragma unroll
        for (int f = 0; f < 4; ++f) {
          const u32x4 bop = *reinterpret_cast<const u32x4*>(xb + j * kPfXStep + (wm * 64 + f * 16 + fr) * kPfXStride +
                                                            fg * 16);
#pragma unroll
          for (int u = 0; u < 2; ++u) acc[u][f] = MfmaP<T>::run(cur.a[j][u], bop, acc[u][f]);
        }
      }
    }
    if (more) {
      x_store(xst, xs[buf ^ 1]);
      __syncthreads();
      buf ^= 1;
    }
  }
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int64_t nb = n0 + 16 * u + 4 * fg;
#pragma unroll
    for (int f = 0; f < 4; ++f) {
      const int64_t m = m0 + wm * 64 + f * 16 + fr;
      if (m < M) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (nb + i < N) Y[m * N + nb + i] = T::from_f32(acc[u][f][i]);
      }
    }
  }
}

template <class T>
hipError_t sparse_prefill_t(const void* X, int64_t M, const spl_matrix& Wc, void* Y, hipStream_t s) {
  if (Wc.nnz == 0) return launch_zero_fill(Y, M * Wc.rows, s);
  const dim3 grid((unsigned)((Wc.rows + kPfBN - 1) / kPfBN), (unsigned)((M + kPfBM - 1) / kPfBM)),
      block(kPfThreads);
  hipLaunchKernelGGL((k_sparse_prefill<T>), grid, block, 0, s, static_cast<const uint16_t*>(X), M, Wc.cols,
                     Wc.bitmask, static_cast<const uint16_t*>(Wc.values), Wc.tile_offsets, Wc.rows,
                     static_cast<uint16_t*>(Y));
  return hipGetLastError();
}

template <class T>
hipError_t dense_prefill_t(const void* X, int64_t M, const void* W, int64_t N, int64_t K, void* Y, hipStream_t s) {
  const dim3 grid((unsigned)((N + kPfBN - 1) / kPfBN), (unsigned)((M + kPfBM - 1) / kPfBM)), block(kPfThreads);
  hipLaunchKernelGGL((k_dense_prefill<T>), grid, block, 0, s, static_cast<const uint16_t*>(X), M, K,
                     static_cast<const uint16_t*>(W), N, static_cast<uint16_t*>(Y));
  return hipGetLastError();
}

}  // namespace

hipError_t launch_sparse_prefill(const void* X, int64_t M, const spl_matrix& Wc, void* Y, hipStream_t s) {
  return Wc.dtype == SPL_BF16 ? sparse_prefill_t<Bf16>(X, M, Wc, Y, s) : sparse_prefill_t<F16>(X, M, Wc, Y, s);
}

hipError_t launch_dense_prefill(const void* X, int64_t M, const void* W, int32_t dtype, int64_t N, int64_t K,
                                void* Y, hipStream_t s) {
  return dtype == SPL_BF16 ? dense_prefill_t<Bf16>(X, M, W, N, K, Y, s) : dense_prefill_t<F16>(X, M, W, N, K, Y, s);
}

}  // namespace spl
