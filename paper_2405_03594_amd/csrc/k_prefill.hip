// Prefill-shaped kernels (any batch M, sized for M >= 128) for gfx950.
//
// One GEMM core serves both kernels.  A workgroup of NW waves computes a
// BN (n) x BM (m) block of Y = X W^T: 128 x 256 with 8 waves for large grids,
// 64 x 128 with 4 waves for launches that would leave CUs idle; wave
// (wn, wm) owns BN/2 x 64 of it, BN/32 x 4 v_mfma_f32_16x16x32 fragments per
// 32-column k-step.  When even the small blocks leave at most one workgroup
// per CU, KS = 2 groups of NW waves share a block: group h takes the h-th
// contiguous half of the stages with its own LDS buffers, and group 1 hands its
// partial sums to group 0 through LDS at the end (a fixed order of addition),
// so each SIMD runs two waves instead of one.  K advances 64
// columns per stage through two LDS buffers per operand: rows of 64
// elements (128 bytes), the 16-byte chunk c of row r stored at chunk
// c ^ (r % 8), so that eight consecutive rows' fragment reads (and the
// staging writes of one row) fall in distinct banks.  The next stage's global loads are
// in flight while the current stage is multiplied, and one barrier per stage
// hands the buffers over; within a stage the second k-step's fragment reads
// are interleaved with the first k-step's MFMAs.  Launches whose blocks and
// stages all lie inside the matrix use loads without bounds branches.
//
//   * dense (comparator): W rows are copied into the A buffer exactly like
//     X rows into the B buffer; launches whose 128 x 256 blocks and stages
//     all lie inside the matrices move both operands straight from global
//     memory into three rotating LDS stage buffers instead (see
//     k_dense_prefill_dma);
//   * sparse (paper section 2.4.2): the A buffer is filled by expanding the
//     stage's compressed 16 x 32 tiles (BN/16 row blocks x 2 k-steps, shared
//     out over the waves), each once per workgroup and one stage ahead, before
//     the current stage's MFMAs: bitmask words are fetched three stages ahead
//     and value windows two ahead (the two tiles a wave expands per stage
//     share one offset scan); a lane expands its row's 8 columns with
//     v_perm_b32 under a nibble selector table, as in the decode kernel, and
//     writes them with one 16-byte LDS store.
#include <type_traits>

#include "spl_common.h"

namespace spl {
namespace {

constexpr int kPfBK = 64;                        // k columns per stage: two 32-column tile steps
constexpr int kPfRow = kPfBK * 2;                // bytes per staged row (8 chunks of 16 bytes, swizzled)
// LDS of a BN x BM workgroup: two W (A operand) buffers of BN rows, two X (B operand) buffers of BM rows
constexpr int pf_lds(int BN, int BM) { return 2 * (BN + BM) * kPfRow; }

// int8 payloads (paper section 3.4): int8 weights and activations, exact int32 sums.
struct I8P {};

template <class T>
struct MfmaP;
template <>
struct MfmaP<Bf16> {
  using acc_t = f32x4;
  static __device__ __forceinline__ f32x4 run(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
  }
};
template <>
struct MfmaP<F16> {
  using acc_t = f32x4;
  static __device__ __forceinline__ f32x4 run(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0,
                                                  0, 0);
  }
};
// One 16 x 16 x 64 int8 product: a 128-byte staged row holds the same two
// k-steps (of 64 int8 columns) as it holds for 16-bit payloads (32 columns).
template <>
struct MfmaP<I8P> {
  using acc_t = i32x4;
  static __device__ __forceinline__ i32x4 run(u32x4 a, u32x4 b, i32x4 c) {
    return __builtin_amdgcn_mfma_i32_16x16x64_i8(__builtin_bit_cast(i32x4, a), __builtin_bit_cast(i32x4, b), c, 0, 0,
                                                 0);
  }
};

// Rows [r0, r0 + RR P) x columns [k0, k0 + 64) of a row-major [R][K] matrix,
// moved through registers by a group of 8 RR threads: thread t holds rows
// r0 + t/8 + RR i (i < P), columns k0 + 8 (t % 8) .. +8.  Checked fetches
// read rows past R and columns past K as zeros (K % 8 == 0, so a 16-byte
// piece is wholly inside or outside); unchecked ones are for launches whose
// blocks and stages all lie inside the matrix, and load without branches.
template <int P>
struct Slab {
  u32x4 v[P];
};

template <int RR>
struct SlabSrc {
  const uint16_t* row0;   // this thread's first row at column 8 (t % 8)
  int64_t stride;         // elements between its rows (RR K)
  int rows_left;          // rows of the matrix from its first row on
  int col;                // its column offset 8 (t % 8)

  __device__ __forceinline__ SlabSrc(const uint16_t* __restrict__ A, int64_t R, int64_t K, int64_t r0, int t) {
    const int64_t r = r0 + (t >> 3);
    col = 8 * (t & 7);
    rows_left = r < R ? (int)(R - r) : 0;
    row0 = A + (r < R ? r : 0) * K + col;
    stride = RR * K;
  }
  template <bool kChecked, int P>
  __device__ __forceinline__ void fetch(Slab<P>& sl, int64_t K, int64_t k0) const {
    if constexpr (kChecked) {
      const bool kok = k0 + col < K;
#pragma unroll
      for (int i = 0; i < P; ++i) {
        sl.v[i] = u32x4{0u, 0u, 0u, 0u};
        if (kok && RR * i < rows_left) sl.v[i] = *reinterpret_cast<const u32x4*>(row0 + i * stride + k0);
      }
    } else {
#pragma unroll
      for (int i = 0; i < P; ++i) sl.v[i] = *reinterpret_cast<const u32x4*>(row0 + i * stride + k0);
    }
  }
};

// Byte offset of 16-byte chunk c (0..7) of staged row r.
__device__ __forceinline__ uint32_t pf_chunk(int r, int c) { return (uint32_t)(r * kPfRow + 16 * (c ^ (r & 7))); }

template <int RR, int P>
__device__ __forceinline__ void slab_store(const Slab<P>& sl, uint32_t buf, int t) {
  // rows t/8 + RR i share their row % 8 with row t/8 (RR is a multiple of 8)
  const uint32_t base = buf + pf_chunk(t >> 3, t & 7);
#pragma unroll
  for (int i = 0; i < P; ++i)
    *reinterpret_cast<__attribute__((address_space(3))) u32x4*>((uintptr_t)(base + RR * kPfRow * i)) = sl.v[i];
}

// One stage of MFMA work: wave (wn, wm) multiplies its 16 FN x 64 block over
// the stage's two k-steps from the A (W) and B (X) buffers.  Both k-steps'
// fragments are read up front; the scheduling hints issue the first k-step's
// reads, then put one second-k-step read after each of the first MFMAs, so
// the LDS reads overlap the matrix cores instead of waiting ahead of them.
template <class T, int FN, int FM>
__device__ __forceinline__ void pf_mfma_stage(typename MfmaP<T>::acc_t (&acc)[FN][FM], uint32_t abuf, uint32_t bbuf,
                                              int wn, int wm, int fr, int fg) {
  // fragment rows differ by multiples of 16, so every row a lane reads has row % 8 == fr % 8
  u32x4 a[2][FN], b[2][FM];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    const uint32_t a0 = abuf + pf_chunk(wn * 16 * FN + fr, 4 * ks + fg);
    const uint32_t b0 = bbuf + pf_chunk(wm * 16 * FM + fr, 4 * ks + fg);
#pragma unroll
    for (int i = 0; i < FN; ++i) a[ks][i] = lds_load16(a0 + 16 * kPfRow * i);
#pragma unroll
    for (int j = 0; j < FM; ++j) b[ks][j] = lds_load16(b0 + 16 * kPfRow * j);
  }
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
      for (int j = 0; j < FM; ++j) acc[i][j] = MfmaP<T>::run(a[ks][i], b[ks][j], acc[i][j]);
  // masks: 0x100 LDS read, 0x008 MFMA
  __builtin_amdgcn_sched_group_barrier(0x100, FN + FM, 0);
#pragma unroll
  for (int q = 0; q < FN + FM; ++q) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, 2 * FN * FM - (FN + FM), 0);
}

// D layout: lane l, register r -> row (n) 4 (l / 16) + r, column (m) l % 16.
template <class T, int FN, int FM>
__device__ __forceinline__ void pf_store(const f32x4 (&acc)[FN][FM], uint16_t* __restrict__ Y, int64_t M, int64_t N,
                                         int64_t n0, int64_t m0, int wn, int wm, int fr, int fg) {
#pragma unroll
  for (int j = 0; j < FM; ++j) {
    const int64_t m = m0 + wm * 16 * FM + 16 * j + fr;
    if (m >= M) continue;
#pragma unroll
    for (int i = 0; i < FN; ++i) {
      const int64_t n = n0 + wn * 16 * FN + 16 * i + 4 * fg;
      uint16_t* y = Y + m * N + n;
      if (n + 3 < N && (N & 3) == 0) {
        u32x2 p;
        p.x = (uint32_t)T::from_f32(acc[i][j][0]) | ((uint32_t)T::from_f32(acc[i][j][1]) << 16);
        p.y = (uint32_t)T::from_f32(acc[i][j][2]) | ((uint32_t)T::from_f32(acc[i][j][3]) << 16);
        *reinterpret_cast<u32x2*>(y) = p;
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (n + r < N) y[r] = T::from_f32(acc[i][j][r]);
      }
    }
  }
}

// The int8 epilogue: Y = fp16_rne((float(acc) * sx[m]) * sw[n]), each product
// rounded to binary32 (no fused multiply-add); acc_out (optional) gets the
// exact int32 sums.
template <int FN, int FM>
__device__ __forceinline__ void pf_store_i8(const i32x4 (&acc)[FN][FM], uint16_t* __restrict__ Y,
                                            int32_t* __restrict__ acc_out, const float* __restrict__ sx,
                                            const float* __restrict__ sw, int64_t M, int64_t N, int64_t n0,
                                            int64_t m0, int wn, int wm, int fr, int fg) {
#pragma unroll
  for (int j = 0; j < FM; ++j) {
    const int64_t m = m0 + wm * 16 * FM + 16 * j + fr;
    if (m >= M) continue;
    const float xs = sx[m];
#pragma unroll
    for (int i = 0; i < FN; ++i) {
      const int64_t n = n0 + wn * 16 * FN + 16 * i + 4 * fg;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        if (n + r >= N) continue;
        const int32_t v = acc[i][j][r];
        if (acc_out) acc_out[m * N + n + r] = v;
        const float y = __fmul_rn(__fmul_rn((float)v, xs), sw[n + r]);
        Y[m * N + n + r] = F16::from_f32(y);
      }
    }
  }
}

// The gated epilogue (the gated half of a Llama MLP): the workgroup's virtual
// rows alternate 16-row blocks of the gate and the up matrix, so fragments 2p
// and 2p + 1 of a wave hold the gate and up sums of the same outputs, in the
// same lanes.  Y[m][n] = silu(g) * u, silu(z) = z / (1 + e^-z), from the fp32
// sums; n0 is the workgroup's first real row.
template <class T, int FN, int FM>
__device__ __forceinline__ void pf_store_gated(const f32x4 (&acc)[FN][FM], uint16_t* __restrict__ Y, int64_t M,
                                               int64_t N, int64_t n0, int64_t m0, int wn, int wm, int fr, int fg) {
  static_assert(FN % 2 == 0, "gate and up fragments pair up");
#pragma unroll
  for (int j = 0; j < FM; ++j) {
    const int64_t m = m0 + wm * 16 * FM + 16 * j + fr;
    if (m >= M) continue;
#pragma unroll
    for (int p = 0; p < FN / 2; ++p) {
      const int64_t n = n0 + wn * 8 * FN + 16 * p + 4 * fg;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        if (n + r >= N) continue;
        const float gs = acc[2 * p][j][r], us = acc[2 * p + 1][j][r];
        Y[m * N + n + r] = T::from_f32(gs / (1.0f + expf(-gs)) * us);
      }
    }
  }
}

// Split K: after every wave's last MFMA, k-group 1 hands its partial sums to
// k-group 0 through the (then free) stage buffers; group 0 adds them (a fixed
// order) and is the one that stores.  Returns whether this thread stores.
template <int FN, int FM, int NT, int KS, class A>
__device__ __forceinline__ bool pf_combine(A (&acc)[FN][FM], unsigned char* dsm, int kh, int t) {
  if constexpr (KS == 1) {
    return true;
  } else {
    static_assert(KS == 2, "two k-groups");
    A* part = reinterpret_cast<A*>(dsm);             // [FN * FM][NT]
    __syncthreads();
    if (kh == 1) {
#pragma unroll
      for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j) part[(i * FM + j) * NT + t] = acc[i][j];
    }
    __syncthreads();
    if (kh == 0) {
#pragma unroll
      for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j) acc[i][j] += part[(i * FM + j) * NT + t];
    }
    return kh == 0;
  }
}

// Compressed operands of a wave's TW tiles of one stage: tile i is row block
// (TW/2) wave + i/2 of the workgroup's BN/16, k-step i % 2 of the stage.
template <int TW>
struct TileWords {
  uint32_t w[TW];         // bitmask word of row fr
  int32_t off[TW];        // tile offset (index of the tile's first value)
};
template <int TW>
struct TileWindows {
  uint32_t byte[TW];      // this lane's 8 columns of row fr (16 for int8)
  u32x2 v0[TW], v1[TW];   // 8-byte windows from the first value of each nibble
};

// Arguments of a prefill launch.  Activations and dense weights are read as
// rows of 16-bit units: a row of K int8 values is K/2 units.
struct PfArgs {
  const uint16_t* X;             // [M][K] activations
  const uint16_t* W;             // dense comparator: [N][K] weights
  const uint32_t* bm;            // sparse: tile bitmask words
  const unsigned char* values;   // sparse: payload bytes (followed by 16 readable bytes)
  const int32_t* toff;           // sparse: tile offsets
  const uint32_t* bm2;           // gated: the up matrix (bm, values, toff are the gate)
  const unsigned char* values2;
  const int32_t* toff2;
  int64_t M, N, K;               // K in payload elements
  uint16_t* Y;                   // out [M][N]: the payload type, fp16 for int8
  const float* sx;               // int8: activation scales [M]
  const float* sw;               // int8: weight scales [N]
  int32_t* acc;                  // int8: optional exact sums [M][N]
  const uint32_t* gbm;           // gather: tile pattern of the [M][N] product (bitmask words)
  const int32_t* gtoff;          // gather: its tile offsets
  uint16_t* gval;                // gather: out, the kept entries in the pattern's value order
};

// The gather epilogue (weight gradients): the product Y [M][N] is only wanted
// at the kept positions of a tile pattern of tile_blocks(M) x tile_steps(N)
// tiles, in its value order, so no dense Y is written.  A 16 x 32 tile is
// fragments (j, 2p) and (j, 2p + 1) of a wave: in the D layout lane l holds
// tile row l % 16 and tile columns 16 h + 4 (l / 16) + r (r < 4) of fragment
// 2p + h.  A tile's values are ordered by 8-column group, then row, then
// column (the decode kernels' lane order), so a kept entry's index is the
// tile offset + the kept entries of the column groups left of its own (all
// rows) + those of its group in the rows above + those left of it in its row
// and group.  The per-group counts of the 16 rows are scanned in one 16-lane
// DPP scan (four 8-bit fields; a field sums at most 16 x 8 = 128).  Values
// are rounded once to the payload type.
// A wave's part of the pattern: its row's bitmask word of each of its
// FM x FN/2 tiles (zero past the pattern), and the tiles' offsets, tile i's in
// lane i (vector loads: a scalar load here would be waited for at once),
// loaded apart from the epilogue so that a kernel can issue the loads early.
template <int FN, int FM>
struct GatherMeta {
  uint32_t w[FM][FN / 2];
  uint32_t off;
};

template <int FN, int FM>
__device__ __forceinline__ void pf_gather_meta(GatherMeta<FN, FM>& gm, const PfArgs& g, int64_t n0, int64_t m0, int wn,
                                               int wm, int lane) {
  static_assert(FM * FN / 2 <= 64, "one tile offset per lane");
  const int64_t B = tile_blocks(g.M);
  const int64_t S = tile_steps(g.N);
  const int fr = lane & 15;
  const int64_t b0 = (m0 + wm * 16 * FM) / 16, s0 = (n0 + wn * 16 * FN) / 32;
#pragma unroll
  for (int j = 0; j < FM; ++j) {
#pragma unroll
    for (int p = 0; p < FN / 2; ++p) {
      const bool ok = b0 + j < B && s0 + p < S;                // wave-uniform
      gm.w[j][p] = ok ? g.gbm[((b0 + j) * S + s0 + p) * 16 + fr] : 0u;   // my row's word
    }
  }
  const int jl = lane / (FN / 2), pl = lane % (FN / 2);        // lane i: tile i = (j, p) = (i / (FN/2), i % (FN/2))
  const bool okl = lane < FM * FN / 2 && b0 + jl < B && s0 + pl < S;
  gm.off = okl ? (uint32_t)g.gtoff[(b0 + jl) * S + s0 + pl] : 0u;
}

template <class T, int FN, int FM>
__device__ __forceinline__ void pf_store_gather(const f32x4 (&acc)[FN][FM], const GatherMeta<FN, FM>& gm,
                                                const PfArgs& g, int lane) {
  const int q = lane >> 4;
#pragma unroll
  for (int j = 0; j < FM; ++j) {
#pragma unroll
    for (int p = 0; p < FN / 2; ++p) {
      const uint32_t w = gm.w[j][p];
      const uint32_t c = __popc(w & 0xffu) | (__popc((w >> 8) & 0xffu) << 8) | (__popc((w >> 16) & 0xffu) << 16) |
                         (__popc(w >> 24) << 24);
      const uint32_t incl = row16_inclusive_scan(c);
      const uint32_t tot = (uint32_t)__builtin_amdgcn_readlane((int)incl, 15);   // every 16-lane row: the same tile
      const uint32_t above = incl - c;                         // per group: rows above mine
      const uint32_t base = (uint32_t)__builtin_amdgcn_readlane((int)gm.off, j * (FN / 2) + p);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int col = 16 * h + 4 * q;                        // my first tile column in this fragment
        const int f = col >> 3;                                // its 8-column group
        uint32_t idx = base + __builtin_amdgcn_ubfe(above, 8 * f, 8);
        if (f > 0) idx += tot & 0xffu;
        if (f > 1) idx += (tot >> 8) & 0xffu;
        if (f > 2) idx += (tot >> 16) & 0xffu;
        if (col & 4) idx += __popc(__builtin_amdgcn_ubfe(w, 8 * f, 4));
        const uint32_t nib = __builtin_amdgcn_ubfe(w, col, 4);
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if ((nib >> r) & 1u) g.gval[idx++] = T::from_f32(acc[2 * p + h][j][r]);
      }
    }
  }
}

// The same epilogue through LDS, for a kernel whose LDS is free at its end:
// the wave writes its tiles' kept entries into its own region (FM runs of
// 1024 16-bit slots) in value order - the two tiles (j, 0) and (j, 1) are
// consecutive in the pattern, so their values are one run - then stores each
// run with coalesced 2-byte stores (64 consecutive entries per store) instead
// of one predicated scattered store per entry.  bf16 values are rounded by
// the hardware conversion (round to nearest even, as T::from_f32 for finite
// values).
template <class T, int FN, int FM>
__device__ __forceinline__ void pf_store_gather_lds(const f32x4 (&acc)[FN][FM], const GatherMeta<FN, FM>& gm,
                                                    const PfArgs& g, int lane, uint16_t* __restrict__ run) {
  static_assert(FN == 4, "two tiles per m-fragment: one run of at most 1024 entries");
  const int q = lane >> 4;
  uint32_t len[FM];
#pragma unroll
  for (int j = 0; j < FM; ++j) {
    uint32_t n = 0;                                            // entries of the run so far (wave-uniform)
#pragma unroll
    for (int p = 0; p < FN / 2; ++p) {
      const uint32_t w = gm.w[j][p];
      const uint32_t c = __popc(w & 0xffu) | (__popc((w >> 8) & 0xffu) << 8) | (__popc((w >> 16) & 0xffu) << 16) |
                         (__popc(w >> 24) << 24);
      const uint32_t incl = row16_inclusive_scan(c);
      const uint32_t tot = (uint32_t)__builtin_amdgcn_readlane((int)incl, 15);
      const uint32_t above = incl - c;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int col = 16 * h + 4 * q;
        const int f = col >> 3;
        uint32_t idx = n + __builtin_amdgcn_ubfe(above, 8 * f, 8);   // within the run
        if (f > 0) idx += tot & 0xffu;
        if (f > 1) idx += (tot >> 8) & 0xffu;
        if (f > 2) idx += (tot >> 16) & 0xffu;
        if (col & 4) idx += __popc(__builtin_amdgcn_ubfe(w, 8 * f, 4));
        const uint32_t nib = __builtin_amdgcn_ubfe(w, col, 4);
        uint16_t v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          if constexpr (std::is_same<T, Bf16>::value)
            v[r] = __builtin_bit_cast(uint16_t, (__bf16)acc[2 * p + h][j][r]);
          else
            v[r] = T::from_f32(acc[2 * p + h][j][r]);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if ((nib >> r) & 1u) run[1024 * j + idx++] = v[r];
      }
      n += (tot & 0xffu) + ((tot >> 8) & 0xffu) + ((tot >> 16) & 0xffu) + (tot >> 24);
    }
    len[j] = n;
  }
  // the wave's LDS operations complete in order: its stores above precede these reads
#pragma unroll
  for (int j = 0; j < FM; ++j) {
    const uint32_t base0 = (uint32_t)__builtin_amdgcn_readlane((int)gm.off, j * (FN / 2));
    for (uint32_t i = (uint32_t)lane; i < len[j]; i += 64) g.gval[base0 + i] = run[1024 * j + i];
  }
}

template <class T, int FN, int FM>
__device__ __forceinline__ void pf_store_gather(const f32x4 (&acc)[FN][FM], const PfArgs& g, int64_t n0, int64_t m0,
                                                int wn, int wm, int lane) {
  GatherMeta<FN, FM> gm;
  pf_gather_meta<FN, FM>(gm, g, n0, m0, wn, wm, lane);
  pf_store_gather<T, FN, FM>(acc, gm, g, lane);
}

// kGated: the workgroup's BN virtual rows are BN/32 row blocks of the gate and
// of the up matrix, alternating (wave w expands virtual block w: matrix w % 2,
// real block BN/32 x + w / 2), stored through pf_store_gated.
template <class T, int BN, int BM, int NW, int KS, bool kChecked, bool kGated = false>
__global__ void __launch_bounds__(64 * NW * KS, 8 / (NW * KS)) k_sparse_prefill(const PfArgs g) {
  extern __shared__ __align__(16) unsigned char dsm[];
  constexpr bool kI8 = std::is_same<T, I8P>::value;
  // selector tables: 16 x 8 bytes (16-bit payloads), or 16 nibbles x 5 window starts (int8)
  __shared__ __align__(16) uint32_t lut[80];
  using Acc = typename MfmaP<T>::acc_t;
  constexpr int NT = 64 * NW;                        // threads of one k-group
  const int kh = KS == 1 ? 0 : __builtin_amdgcn_readfirstlane((int)threadIdx.x / NT);
  const int tid = (int)threadIdx.x - kh * NT;        // thread index within the k-group
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = threadIdx.x & 63;
  const int wn = wave & 1, wm = wave >> 1;
  const int fr = lane & 15, fg = lane >> 4;
  const int64_t M = g.M, N = g.N, K = g.K;
  const int64_t Kh = kI8 ? K / 2 : K;                // activation row in 16-bit units
  const int S = (int)tile_steps(K);
  const int nst = (int)((Kh + kPfBK - 1) / kPfBK);   // stages of 128 bytes per row: 2 tiles (4 for int8)
  const int nh = (nst + KS - 1) / KS;                // stages per k-group (uniform: every group's barriers)
  const int sb = kh * nh;                            // this group's first stage
  const int nl = nst - sb < nh ? (nst > sb ? nst - sb : 0) : nh;   // its stages (the last group may hold fewer)
  const int64_t B = tile_blocks(N);
  constexpr int FN = BN / 32;                        // n-fragments per wave
  constexpr int TW = BN / 8 / NW;                    // operand units per wave per stage: tiles (int8: tile pairs)
  constexpr int RR = 8 * NW;                         // rows per staging round
  constexpr int FM = BM / (8 * NW);                  // m-fragments per wave
  static_assert(BM % (8 * NW) == 0 && FM <= 8 && TW % 2 == 0, "wave layout: 2 x NW/2 waves of BN/2 x 16 FM");
  static_assert(KS == 1 || FN * FM * NT * 16 <= KS * pf_lds(BN, BM), "partial sums fit the stage buffers");
  const int64_t n0 = (int64_t)blockIdx.x * BN;
  const int64_t m0 = (int64_t)blockIdx.y * BM;
  static_assert(!kGated || (!kI8 && TW == 2), "gated: 16-bit payloads, one row block per wave");
  const int gm = kGated ? (wave & 1) : 0;            // gated: this wave's matrix (0 gate, 1 up)
  // first row block of this wave's units
  const int64_t wb = kGated ? (int64_t)blockIdx.x * (BN / 32) + (wave >> 1) : n0 / 16 + (TW / 2) * wave;
  unsigned char* gb = dsm + kh * pf_lds(BN, BM);     // this group's stage buffers
  const uint32_t abuf[2] = {lds_off(gb), lds_off(gb + BN * kPfRow)};
  const uint32_t bbuf[2] = {lds_off(gb + 2 * BN * kPfRow), lds_off(gb + (2 * BN + BM) * kPfRow)};
  const uint32_t lut_addr = lds_off(lut);
  const unsigned char* vbytes = gm ? g.values2 : g.values;
  const uint32_t* __restrict__ bm_tiles = gm ? g.bm2 : g.bm;
  const int32_t* __restrict__ tile_offsets = gm ? g.toff2 : g.toff;
  if constexpr (kI8) {
    if (threadIdx.x < 80) lut[threadIdx.x] = nibble_selector8(threadIdx.x / 5, threadIdx.x % 5);
  } else {
    if (threadIdx.x < 16) {
      lut[2 * threadIdx.x] = nibble_selector16(threadIdx.x, 0);
      lut[2 * threadIdx.x + 1] = nibble_selector16(threadIdx.x, 1);
    }
  }

  // Unit i of a stage is row block (TW/2) wave + i/2 of the workgroup's BN/16
  // and k-step 2 st + i % 2: one tile (16-bit payloads), or the pair of tiles
  // 4 st + 2 (i % 2) + {0, 1} (int8: lanes 0-31 the first, 32-63 the second).
  auto fetch_words = [&](TileWords<TW>& tw, int st) {
#pragma unroll
    for (int i = 0; i < TW; ++i) {
      const int64_t b = wb + (i >> 1);
      const int s = kI8 ? 4 * st + 2 * (i & 1) + (fg >> 1) : 2 * st + (i & 1);
      if constexpr (kChecked) {
        const bool ok = b < B && s < S;
        const int64_t t = ok ? b * S + s : 0;
        tw.w[i] = ok ? bm_tiles[t * 16 + fr] : 0u;
        tw.off[i] = tile_offsets[t];
      } else {                                       // N % BN == 0 and whole stages: always inside
        const int64_t t = b * S + s;
        tw.w[i] = bm_tiles[t * 16 + fr];
        tw.off[i] = tile_offsets[t];
      }
    }
  };
  auto fetch_windows = [&](TileWindows<TW>& tv, const TileWords<TW>& tw) {
#pragma unroll
    for (int i = 0; i < TW; i += 2) {
      if constexpr (kI8) {
        // my 16 columns: half fg % 2 of my tile's word.  A tile's values are ordered by 16-column
        // group, then row, i.e. in the order of the tile's 32 lanes, so the values before mine are
        // the exclusive scan over my half of the wave (two units per scan in 16-bit halves)
        const uint32_t h0 = __builtin_amdgcn_ubfe(tw.w[i], 16 * (fg & 1), 16);
        const uint32_t h1 = __builtin_amdgcn_ubfe(tw.w[i + 1], 16 * (fg & 1), 16);
        const uint32_t pc = __popc(h0) | (__popc(h1) << 16);
        const uint32_t ex = half_inclusive_scan(pc) - pc;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const uint32_t hw = h ? h1 : h0;
          const uint32_t oa = (uint32_t)tw.off[i + h] + (h ? ex >> 16 : ex & 0xffffu);
          const uint32_t ob = oa + __popc(hw & 0xffu);   // nibbles 2 and 3 start after nibbles 0 and 1
          tv.byte[i + h] = hw;
          __builtin_memcpy(&tv.v0[i + h], vbytes + oa, 8);
          __builtin_memcpy(&tv.v1[i + h], vbytes + ob, 8);
        }
      } else {
        // values stored before mine: a tile's values are ordered by column group (fg), then row (fr),
        // i.e. in lane order, so this is the exclusive wave scan of the lanes' kept counts; the
        // pair of tiles shares one scan in 16-bit halves (sums <= 512)
        const uint32_t b0 = __builtin_amdgcn_ubfe(tw.w[i], 8 * fg, 8);
        const uint32_t b1 = __builtin_amdgcn_ubfe(tw.w[i + 1], 8 * fg, 8);
        const uint32_t pc = __popc(b0) | (__popc(b1) << 16);
        const uint32_t ex = wave_inclusive_scan(pc) - pc;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const uint32_t byte = h ? b1 : b0;
          const uint32_t oa = (uint32_t)tw.off[i + h] + (h ? ex >> 16 : ex & 0xffffu);
          const uint32_t ob = oa + __popc(byte & 0xfu);
          tv.byte[i + h] = byte;
          __builtin_memcpy(&tv.v0[i + h], vbytes + 2u * oa, 8);
          __builtin_memcpy(&tv.v1[i + h], vbytes + 2u * ob, 8);
        }
      }
    }
  };
  auto expand_store = [&](const TileWindows<TW>& tv, uint32_t buf) {
#pragma unroll
    for (int i = 0; i < TW; ++i) {
      u32x4 a;
      if constexpr (kI8) {
        const uint32_t hw = tv.byte[i];
        const uint32_t n0_ = hw & 15u, n1 = (hw >> 4) & 15u, n2 = (hw >> 8) & 15u, n3 = hw >> 12;
        const uint32_t s0 = lds_load4(lut_addr + 20u * n0_);
        const uint32_t s1 = lds_load4(lut_addr + 20u * n1 + 4u * __popc(n0_));
        const uint32_t s2 = lds_load4(lut_addr + 20u * n2);
        const uint32_t s3 = lds_load4(lut_addr + 20u * n3 + 4u * __popc(n2));
        a.x = __builtin_amdgcn_perm(tv.v0[i].y, tv.v0[i].x, s0);
        a.y = __builtin_amdgcn_perm(tv.v0[i].y, tv.v0[i].x, s1);
        a.z = __builtin_amdgcn_perm(tv.v1[i].y, tv.v1[i].x, s2);
        a.w = __builtin_amdgcn_perm(tv.v1[i].y, tv.v1[i].x, s3);
      } else {
        const u32x2 slo = lds_load8(lut_addr + 8u * (tv.byte[i] & 0xfu));
        const u32x2 shi = lds_load8(lut_addr + 8u * (tv.byte[i] >> 4));
        a.x = __builtin_amdgcn_perm(tv.v0[i].y, tv.v0[i].x, slo.x);
        a.y = __builtin_amdgcn_perm(tv.v0[i].y, tv.v0[i].x, slo.y);
        a.z = __builtin_amdgcn_perm(tv.v1[i].y, tv.v1[i].x, shi.x);
        a.w = __builtin_amdgcn_perm(tv.v1[i].y, tv.v1[i].x, shi.y);
      }
      const uint32_t at = buf + pf_chunk(16 * ((TW / 2) * wave + (i >> 1)) + fr, 4 * (i & 1) + fg);
      *reinterpret_cast<__attribute__((address_space(3))) u32x4*>((uintptr_t)at) = a;
    }
  };

  Acc acc[FN][FM];
#pragma unroll
  for (int i = 0; i < FN; ++i)
#pragma unroll
    for (int j = 0; j < FM; ++j) acc[i][j] = Acc{0, 0, 0, 0};

  // Pipeline: bitmask words three stages ahead, value windows and X slabs two
  // ahead (X in alternating register sets, the loop unrolled by two stages).
  // At the start of stage st, stage st + 1's W tiles are expanded into the
  // other LDS buffers and its X slab stored there (their last readers, stage
  // st - 1's MFMAs, finished before the previous barrier), so that this ALU
  // and LDS work can interleave with the matrix cores; one barrier per stage.
  // Stages are counted within the k-group (global stage sb + st); data steps
  // are guarded by the group's nl stages, barriers by the uniform nh.
  const SlabSrc<RR> xsrc(g.X, M, Kh, m0, tid);
  Slab<BM / RR> x0, x1;
  TileWords<TW> tw;
  TileWindows<TW> tv;
  if (nl > 0) {
    fetch_words(tw, sb);
    xsrc.template fetch<kChecked>(x0, Kh, (int64_t)kPfBK * sb);
    fetch_windows(tv, tw);                             // stage 0
    if (nl > 1) {
      fetch_words(tw, sb + 1);
      xsrc.template fetch<kChecked>(x1, Kh, (int64_t)kPfBK * (sb + 1));
    }
  }
  __syncthreads();                                     // the selector table
  if (nl > 0) {
    expand_store(tv, abuf[0]);
    slab_store<RR>(x0, bbuf[0], tid);
    if (nl > 1) {
      fetch_windows(tv, tw);                           // stage 1
      if (nl > 2) fetch_words(tw, sb + 2);
    }
  }
  __syncthreads();
  // (xl holds stage st + 1; xn receives stage st + 2)
  auto step = [&](int st, Slab<BM / RR>& xn, Slab<BM / RR>& xl) {
    const int cur = st & 1;
    if (st + 1 < nl) {
      expand_store(tv, abuf[cur ^ 1]);                 // stage st + 1
      slab_store<RR>(xl, bbuf[cur ^ 1], tid);
      if (st + 2 < nl) {
        fetch_windows(tv, tw);                         // stage st + 2 (its words were fetched a stage ago)
        if (st + 3 < nl) fetch_words(tw, sb + st + 3);
        xsrc.template fetch<kChecked>(xn, Kh, (int64_t)kPfBK * (sb + st + 2));
      }
    }
    if (st < nl) pf_mfma_stage<T, FN, FM>(acc, abuf[cur], bbuf[cur], wn, wm, fr, fg);
    if (st + 1 < nh) __syncthreads();
  };
  for (int st = 0; st < nh; st += 2) {
    step(st, x0, x1);                                  // stage st + 1 from set 1, stage st + 2 -> set 0
    if (st + 1 < nh) step(st + 1, x1, x0);             // stage st + 2 from set 0, stage st + 3 -> set 1
  }
  if (pf_combine<FN, FM, NT, KS>(acc, dsm, kh, tid)) {
    if constexpr (kI8)
      pf_store_i8<FN, FM>(acc, g.Y, g.acc, g.sx, g.sw, M, N, n0, m0, wn, wm, fr, fg);
    else if constexpr (kGated)
      pf_store_gated<T, FN, FM>(acc, g.Y, M, N, (int64_t)blockIdx.x * (BN / 2), m0, wn, wm, fr, fg);
    else
      pf_store<T, FN, FM>(acc, g.Y, M, N, n0, m0, wn, wm, fr, fg);
  }
}

// kGather: only the kept entries of the product at a tile pattern are written
// (pf_store_gather), for 16-bit payloads.
template <class T, int BN, int BM, int NW, int KS, bool kChecked, bool kGather = false>
__global__ void __launch_bounds__(64 * NW * KS, 8 / (NW * KS)) k_dense_prefill(const PfArgs g) {
  extern __shared__ __align__(16) unsigned char dsm[];
  constexpr bool kI8 = std::is_same<T, I8P>::value;
  using Acc = typename MfmaP<T>::acc_t;
  constexpr int NT = 64 * NW;                         // threads of one k-group
  const int kh = KS == 1 ? 0 : __builtin_amdgcn_readfirstlane((int)threadIdx.x / NT);
  const int tid = (int)threadIdx.x - kh * NT;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = threadIdx.x & 63;
  const int wn = wave & 1, wm = wave >> 1;
  const int fr = lane & 15, fg = lane >> 4;
  const int64_t M = g.M, N = g.N, K = g.K;
  const int64_t Kh = kI8 ? K / 2 : K;
  const int nst = (int)((Kh + kPfBK - 1) / kPfBK);
  const int nh = (nst + KS - 1) / KS;
  const int sb = kh * nh;
  const int nl = nst - sb < nh ? (nst > sb ? nst - sb : 0) : nh;
  constexpr int FN = BN / 32;                         // n-fragments per wave
  constexpr int RR = 8 * NW;                          // rows per staging round
  constexpr int FM = BM / (8 * NW);                   // m-fragments per wave
  static_assert(BM % (8 * NW) == 0 && FM <= 8 && BN % RR == 0, "wave layout: 2 x NW/2 waves of BN/2 x 16 FM");
  static_assert(KS == 1 || FN * FM * NT * 16 <= KS * pf_lds(BN, BM), "partial sums fit the stage buffers");
  const int64_t n0 = (int64_t)blockIdx.x * BN;
  const int64_t m0 = (int64_t)blockIdx.y * BM;
  unsigned char* gb = dsm + kh * pf_lds(BN, BM);
  const uint32_t abuf[2] = {lds_off(gb), lds_off(gb + BN * kPfRow)};
  const uint32_t bbuf[2] = {lds_off(gb + 2 * BN * kPfRow), lds_off(gb + (2 * BN + BM) * kPfRow)};

  Acc acc[FN][FM];
#pragma unroll
  for (int i = 0; i < FN; ++i)
#pragma unroll
    for (int j = 0; j < FM; ++j) acc[i][j] = Acc{0, 0, 0, 0};

  // Global loads run two stages ahead of the multiplication: register sets
  // (x0, w0) and (x1, w1) alternate, the loop unrolled by two stages.  Stage
  // st + 1 is stored to LDS at the start of stage st, so one barrier per stage
  // both publishes it and retires stage st's reads.
  const SlabSrc<RR> xsrc(g.X, M, Kh, m0, tid), wsrc(g.W, N, Kh, n0, tid);
  Slab<BM / RR> x0, x1;
  Slab<BN / RR> w0, w1;
  if (nl > 0) {
    xsrc.template fetch<kChecked>(x0, Kh, (int64_t)kPfBK * sb);
    wsrc.template fetch<kChecked>(w0, Kh, (int64_t)kPfBK * sb);
    if (nl > 1) {
      xsrc.template fetch<kChecked>(x1, Kh, (int64_t)kPfBK * (sb + 1));
      wsrc.template fetch<kChecked>(w1, Kh, (int64_t)kPfBK * (sb + 1));
    }
    slab_store<RR>(w0, abuf[0], tid);
    slab_store<RR>(x0, bbuf[0], tid);
  }
  __syncthreads();
  // stage st is in the LDS buffers st % 2; (xl, wl) hold stage st + 1, which
  // is written to the other buffers before this stage's MFMAs (their last
  // readers, stage st - 1's MFMAs, finished before the previous barrier), and
  // (xn, wn_) receive stage st + 2
  auto step = [&](int st, Slab<BM / RR>& xn, Slab<BN / RR>& wn_, Slab<BM / RR>& xl, Slab<BN / RR>& wl) {
    const int cur = st & 1;
    if (st + 1 < nl) {
      slab_store<RR>(wl, abuf[cur ^ 1], tid);
      slab_store<RR>(xl, bbuf[cur ^ 1], tid);
    }
    if (st + 2 < nl) {
      xsrc.template fetch<kChecked>(xn, Kh, (int64_t)kPfBK * (sb + st + 2));
      wsrc.template fetch<kChecked>(wn_, Kh, (int64_t)kPfBK * (sb + st + 2));
    }
    if (st < nl) pf_mfma_stage<T, FN, FM>(acc, abuf[cur], bbuf[cur], wn, wm, fr, fg);
    if (st + 1 < nh) __syncthreads();
  };
  for (int st = 0; st < nh; st += 2) {
    step(st, x0, w0, x1, w1);                          // stage st + 2 -> set 0, stage st + 1 from set 1
    if (st + 1 < nh) step(st + 1, x1, w1, x0, w0);     // stage st + 3 -> set 1, stage st + 2 from set 0
  }
  static_assert(!kGather || (!kI8 && FN % 2 == 0), "gather: 16-bit payloads, whole tiles per wave");
  if (pf_combine<FN, FM, NT, KS>(acc, dsm, kh, tid)) {
    if constexpr (kI8)
      pf_store_i8<FN, FM>(acc, g.Y, g.acc, g.sx, g.sw, M, N, n0, m0, wn, wm, fr, fg);
    else if constexpr (kGather)
      pf_store_gather<T, FN, FM>(acc, g, n0, m0, wn, wm, lane);
    else
      pf_store<T, FN, FM>(acc, g.Y, M, N, n0, m0, wn, wm, fr, fg);
  }
}

// Direct-to-LDS staging, for launches whose 128 x 256 blocks and 64-column
// stages all lie inside the matrices (16-bit payloads; eight waves of 64 x 64
// as above).  Operand rows go from global memory straight into LDS
// (global_load_lds_dwordx4: lane i of a request fills the 16-byte slot i of a
// 1 KB run, i.e. row i / 8 of an 8-row group at position i % 8, so the lane
// fetches the chunk whose swizzled position that is), which takes no
// registers and no LDS store instructions.  Three stage buffers per staged
// operand: stage st + 2 is requested while stage st is multiplied, and one
// barrier per stage both publishes stage st + 1 (each wave first waits for
// its own requests of it) and retires the buffer that the next request
// overwrites (last read by stage st).
constexpr int kDmaBN = 128, kDmaBM = 256, kDmaStages = 3, kDmaWaves = 8;
constexpr int kDmaStageBytes = (kDmaBN + kDmaBM) * kPfRow;     // 48 KB

__device__ __forceinline__ void lds_dma16(const uint16_t* src, unsigned char* dst) {
  __builtin_amdgcn_global_load_lds((const void __attribute__((address_space(1)))*)src,
                                   (void __attribute__((address_space(3)))*)dst, 16, 0, 0);
}

// Wait until at most kOutstanding of this wave's vector memory requests remain
// (they complete in order) and its LDS operations are done, then a bare
// workgroup barrier: __syncthreads() would wait for every request.  The
// compiler-only fences keep LDS accesses from moving across the barrier.
template <int kOutstanding>
__device__ __forceinline__ void dma_barrier() {
  static_assert(kOutstanding >= 0 && kOutstanding < 16, "vmcnt's low field");
  __builtin_amdgcn_s_waitcnt(0x0070 | kOutstanding);   // vmcnt(n) expcnt(7) lgkmcnt(0)
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// A wave's part of one stage's requests: `groups` 8-row groups of rows
// [8 groups w, 8 groups (w + 1)) of a staged operand, from the lane's first
// row `src` (row lane / 8 of the wave's first group, at its swizzled chunk).
template <int kGroups>
__device__ __forceinline__ void dma_rows(const uint16_t* src, int64_t K, int st, unsigned char* buf, int wave) {
#pragma unroll
  for (int i = 0; i < kGroups; ++i)
    lds_dma16(src + 8 * K * i + kPfBK * st, buf + (8 * kGroups * wave + 8 * i) * kPfRow);
}

// (int8 payloads, I8P: rows of K bytes staged as K/2 16-bit units, exact int32 sums, the int8 epilogue)
template <class T, bool kGather, int NW>
__global__ void __launch_bounds__(64 * NW, 1) k_dense_prefill_dma(const PfArgs g) {
  constexpr bool kI8 = std::is_same<T, I8P>::value;
  static_assert(!(kI8 && kGather), "gather: 16-bit payloads");
  using Acc = typename MfmaP<T>::acc_t;
  constexpr int FN = 4, FM = kDmaBM / (8 * NW);
  constexpr int GA = kDmaBN / 8 / NW, GB = kDmaBM / 8 / NW;      // 8-row groups per wave: W, X
  constexpr int kLoads = GA + GB;                                 // 1 KB requests per wave and stage
  extern __shared__ __align__(16) unsigned char dsm[];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int wn = wave & 1, wm = wave >> 1;
  const int fr = lane & 15, fg = lane >> 4;
  const int64_t M = g.M, N = g.N, K = g.K;
  const int64_t Kh = kI8 ? K / 2 : K;                 // row length in 16-bit units
  const int nst = (int)(Kh / kPfBK);
  const int64_t n0 = (int64_t)blockIdx.x * kDmaBN, m0 = (int64_t)blockIdx.y * kDmaBM;
  // my slot in an 8-row group: row lane / 8, position lane % 8, holding chunk (lane % 8) ^ (lane / 8)
  const int lr = lane >> 3, lc = (lane & 7) ^ lr;
  // wave w requests W rows 8 GA w .. + 8 GA and X rows 8 GB w .. + 8 GB
  const uint16_t* wsrc = g.W + (n0 + 8 * GA * wave + lr) * Kh + 8 * lc;
  const uint16_t* xsrc = g.X + (m0 + 8 * GB * wave + lr) * Kh + 8 * lc;
  auto request = [&](int st, int buf) {
    unsigned char* a = dsm + buf * kDmaStageBytes;
    dma_rows<GA>(wsrc, Kh, st, a, wave);
    dma_rows<GB>(xsrc, Kh, st, a + kDmaBN * kPfRow, wave);
  };

  Acc acc[FN][FM];
#pragma unroll
  for (int i = 0; i < FN; ++i)
#pragma unroll
    for (int j = 0; j < FM; ++j) acc[i][j] = Acc{0, 0, 0, 0};

  request(0, 0);
  if (nst > 1) request(1, 1);
  int cur = 0;
  for (int st = 0; st < nst; ++st) {
    // my requests of stage st are done once at most the next stage's remain
    if (st + 1 < nst) dma_barrier<kLoads>();
    else dma_barrier<0>();
    if (st + 2 < nst) request(st + 2, cur == 0 ? 2 : cur - 1);
    const uint32_t abuf = lds_off(dsm + cur * kDmaStageBytes);
    pf_mfma_stage<T, FN, FM>(acc, abuf, abuf + kDmaBN * kPfRow, wn, wm, fr, fg);
    cur = cur == kDmaStages - 1 ? 0 : cur + 1;
  }
  if constexpr (kI8)
    pf_store_i8<FN, FM>(acc, g.Y, g.acc, g.sx, g.sw, M, N, n0, m0, wn, wm, fr, fg);
  else if constexpr (kGather)
    pf_store_gather<T, FN, FM>(acc, g, n0, m0, wn, wm, lane);
  else
    pf_store<T, FN, FM>(acc, g.Y, M, N, n0, m0, wn, wm, fr, fg);
}

// Contraction-major factors (the weight gradient dY^T X, both factors stored
// with the token as the row): the same 128 x 256 blocks and eight waves, the
// operands again moved straight from global memory into three rotating LDS
// stage buffers, now as kPfBK contraction rows of the block's 128 W columns
// (256-byte rows) and 256 X columns (512-byte rows), so that no transposed
// copy of either factor is written first.  The fragments are read with
// ds_read_b64_tr_b16: within each 16-lane quarter of the wave, lane s reads 8
// bytes at its own address and lane t receives, as its element e, element
// t % 4 of the 8 bytes of lane 4 e + t / 4.  Lane s points at contraction row
// k0 + s / 4, columns c0 + 4 (s % 4) .. + 3, so lane t receives column c0 + t
// at rows k0 .. k0 + 3: the MFMA operand layout (fragment row lane % 16,
// contraction index 8 (lane / 16) + j), in two reads per 16 x 32 fragment.
// Swizzle: the 16-byte chunk c of staged row r sits at chunk c ^ 2 h(r),
// h(r) = r % 4 + 4 ((r / 8) % 2).  A read of half a wave covers rows
// r0 .. r0 + 3 and r0 + 8 .. r0 + 11 (r0 % 16 = 0 or 4), 32 bytes each, and
// h places those 8 pieces in 8 distinct 32-byte bank groups; h is the same
// for rows 4 and 32 apart, so a fragment's four reads share one address
// register and differ in the instruction's offset.
constexpr int kTrRowA = 2 * kDmaBN, kTrRowB = 2 * kDmaBM;      // bytes per staged contraction row: W, X
constexpr int kTrOffB = kPfBK * kTrRowA;                        // X part of a stage buffer

// The same 16-byte direct-to-LDS request as lds_dma16, issued from inline
// assembly: the compiler then does not count it, and so does not wait for
// every outstanding request before each ds_read_b64_tr_b16 (which it cannot
// tell apart from reads of the buffer being filled).  dma_barrier's explicit
// wait is what orders the requests before the reads.  M0 (the request's LDS
// base) is declared clobbered; the kernel that uses this issues no other
// instruction that reads M0.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void lds_dma16_opaque(const uint16_t* src, unsigned char* dst) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(lds_off(dst))
               : "memory", "m0");
}
#pragma clang diagnostic pop

__device__ __forceinline__ u32x2 lds_load_tr8(uint32_t addr) {
  typedef short s16x4 __attribute__((ext_vector_type(4)));
  const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)(uintptr_t)addr);
  return __builtin_bit_cast(u32x2, v);
}

// One stage of MFMA work from contraction-major buffers: ao / bo are the
// lane's byte offsets of its A and B fragments' first read in a stage buffer.
template <class T, int FN, int FM>
__device__ __forceinline__ void pf_mfma_stage_tr(typename MfmaP<T>::acc_t (&acc)[FN][FM], uint32_t buf,
                                                 const uint32_t (&ao)[FN], const uint32_t (&bo)[FM]) {
  u32x4 a[2][FN], b[2][FM];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
    for (int i = 0; i < FN; ++i) {
      const uint32_t p = buf + ao[i] + 32 * kTrRowA * ks;
      const u32x2 lo = lds_load_tr8(p), hi = lds_load_tr8(p + 4 * kTrRowA);
      a[ks][i] = u32x4{lo.x, lo.y, hi.x, hi.y};
    }
#pragma unroll
    for (int j = 0; j < FM; ++j) {
      const uint32_t p = buf + bo[j] + 32 * kTrRowB * ks;
      const u32x2 lo = lds_load_tr8(p), hi = lds_load_tr8(p + 4 * kTrRowB);
      b[ks][j] = u32x4{lo.x, lo.y, hi.x, hi.y};
    }
  }
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
      for (int j = 0; j < FM; ++j) acc[i][j] = MfmaP<T>::run(a[ks][i], b[ks][j], acc[i][j]);
  // masks: 0x100 LDS read, 0x008 MFMA; two reads per fragment
  __builtin_amdgcn_sched_group_barrier(0x100, 2 * (FN + FM), 0);
#pragma unroll
  for (int q = 0; q < FN + FM; ++q) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, 2 * FN * FM - (FN + FM), 0);
}

// A grouped launch of the contraction-major core: task i (its own factors,
// shapes and pattern, one dtype) owns workgroups [first[i], first[i + 1]),
// block b of it at n-block b % (N / 128), m-block b / (N / 128).
constexpr int kTrGroupMax = 4;
struct TrGroupArg {
  PfArgs t[kTrGroupMax];
  int32_t first[kTrGroupMax + 1];
  int32_t count;
};

// Y = Xc^T Wc for Xc [K][M] and Wc [K][N] (g.X, g.W), kept entries only
// (pf_store_gather); M % 256 == 0, N % 128 == 0, K % kPfBK == 0.
template <class T, int NW>
__global__ void __launch_bounds__(64 * NW, 1) k_dense_prefill_dma_tr(const TrGroupArg ga) {
  const int ti = find_task(ga.first, ga.count);
  const PfArgs& g = ga.t[ti];
  static_assert(!std::is_same<T, I8P>::value && NW == 8, "16-bit payloads, eight waves");
  using Acc = typename MfmaP<T>::acc_t;
  constexpr int FN = 4, FM = kDmaBM / (8 * NW);
  constexpr int RA = kPfBK * kTrRowA / 1024 / NW, RB = kPfBK * kTrRowB / 1024 / NW;   // 1 KB runs per wave: 2, 4
  constexpr int kLoads = RA + RB;
  extern __shared__ __align__(16) unsigned char dsm[];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int wn = wave & 1, wm = wave >> 1;
  const int64_t M = g.M, N = g.N, K = g.K;
  const int nst = (int)(K / kPfBK);
  const int64_t b = (int64_t)blockIdx.x - ga.first[ti], tn = N / kDmaBN;
  const int64_t n0 = (b % tn) * kDmaBN, m0 = (b / tn) * kDmaBM;
  // wave w requests rows 8 w .. 8 w + 7 of each operand's stage (bit 3 of the row: w % 2).
  // W run u: rows 8 w + 4 u + lane / 16, the lane's slot lane % 16 of the row;
  // X run u: rows 8 w + 2 u + lane / 32, slot lane % 32 (h depends on u % 2).
  const int hw = (wave & 1) << 2;
  const uint16_t* wsrc = g.W + (int64_t)(8 * wave + (lane >> 4)) * N + n0 + 8 * ((lane & 15) ^ (2 * ((lane >> 4) | hw)));
  const uint16_t* xsrc[2];
#pragma unroll
  for (int p = 0; p < 2; ++p)
    xsrc[p] = g.X + (int64_t)(8 * wave + 2 * p + (lane >> 5)) * M + m0 + 8 * ((lane & 31) ^ (2 * ((2 * p + (lane >> 5)) | hw)));
  auto request = [&](int st, int buf) {
    unsigned char* a = dsm + buf * kDmaStageBytes;
    const int64_t k0 = (int64_t)kPfBK * st;
#pragma unroll
    for (int u = 0; u < RA; ++u) lds_dma16_opaque(wsrc + (k0 + 4 * u) * N, a + (RA * wave + u) * 1024);
#pragma unroll
    for (int u = 0; u < RB; ++u)
      lds_dma16_opaque(xsrc[u & 1] + (k0 + 4 * (u >> 1)) * M, a + kTrOffB + (RB * wave + u) * 1024);
  };
  // my fragments' first reads: row r0 = 8 (lane / 16) + t / 4 (t = lane % 16), columns 16 i + 4 (t % 4) of the wave's
  const int t = lane & 15, r0 = 8 * (lane >> 4) + (t >> 2);
  const int h = (t >> 2) | (((lane >> 4) & 1) << 2);
  uint32_t ao[FN], bo[FM];
#pragma unroll
  for (int i = 0; i < FN; ++i)
    ao[i] = (uint32_t)(r0 * kTrRowA + 16 * ((8 * wn + 2 * i + ((t & 3) >> 1)) ^ (2 * h)) + 8 * (t & 1));
#pragma unroll
  for (int j = 0; j < FM; ++j)
    bo[j] = (uint32_t)(kTrOffB + r0 * kTrRowB + 16 * ((8 * wm + 2 * j + ((t & 3) >> 1)) ^ (2 * h)) + 8 * (t & 1));

  Acc acc[FN][FM];
#pragma unroll
  for (int i = 0; i < FN; ++i)
#pragma unroll
    for (int j = 0; j < FM; ++j) acc[i][j] = Acc{0, 0, 0, 0};

  // the epilogue's pattern loads go first: the stage waits complete them, so the
  // epilogue does not wait for their latency after the last MFMAs
  GatherMeta<FN, FM> gm;
  pf_gather_meta<FN, FM>(gm, g, n0, m0, wn, wm, lane);
  request(0, 0);
  if (nst > 1) request(1, 1);
  int cur = 0;
  for (int st = 0; st < nst; ++st) {
    if (st + 1 < nst) dma_barrier<kLoads>();
    else dma_barrier<0>();
    if (st + 2 < nst) request(st + 2, cur == 0 ? 2 : cur - 1);
    pf_mfma_stage_tr<T, FN, FM>(acc, lds_off(dsm + cur * kDmaStageBytes), ao, bo);
    cur = cur == kDmaStages - 1 ? 0 : cur + 1;
  }
  static_assert(2 * 1024 * FM * NW <= kDmaStages * kDmaStageBytes, "the waves' value runs fit the stage buffers");
  __syncthreads();                                   // every wave is done reading the stage buffers
  pf_store_gather_lds<T, FN, FM>(acc, gm, g, lane, reinterpret_cast<uint16_t*>(dsm) + 1024 * FM * wave);
}

// One stage of MFMA work with the A operand read by LDS transpose reads from
// a contraction-major buffer (ao: the lane's first-read offsets) and the B
// operand from a staged X buffer as in pf_mfma_stage.
template <class T, int FN, int FM>
__device__ __forceinline__ void pf_mfma_stage_trA(typename MfmaP<T>::acc_t (&acc)[FN][FM], uint32_t abuf,
                                                  const uint32_t (&ao)[FN], uint32_t bbuf, int wm, int fr, int fg) {
  u32x4 a[2][FN], b[2][FM];
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
    for (int i = 0; i < FN; ++i) {
      const uint32_t p = abuf + ao[i] + 32 * kTrRowA * ks;
      const u32x2 lo = lds_load_tr8(p), hi = lds_load_tr8(p + 4 * kTrRowA);
      a[ks][i] = u32x4{lo.x, lo.y, hi.x, hi.y};
    }
    const uint32_t b0 = bbuf + pf_chunk(wm * 16 * FM + fr, 4 * ks + fg);
#pragma unroll
    for (int j = 0; j < FM; ++j) b[ks][j] = lds_load16(b0 + 16 * kPfRow * j);
  }
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
      for (int j = 0; j < FM; ++j) acc[i][j] = MfmaP<T>::run(a[ks][i], b[ks][j], acc[i][j]);
  // masks: 0x100 LDS read, 0x008 MFMA
  __builtin_amdgcn_sched_group_barrier(0x100, 2 * FN + FM, 0);
#pragma unroll
  for (int q = 0; q < 2 * FN + FM; ++q) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, 2 * FN * FM - (2 * FN + FM), 0);
}

// The input gradient through a sparse layer (Algorithm 1's backward pass):
// dX [M][K] = dY [M][N] (W.Mask) straight from W's packed tiles, with no
// packed transpose.  The contraction runs over W's rows, so a stage takes 64
// of them (four row blocks) across the workgroup's 128 columns: wave w
// expands the stage's tiles (row block 4 st + w / 2, k-steps 2 (w % 2) + {0, 1}
// of the block's four; a consecutive pair, one scan) exactly as
// k_sparse_prefill does, but stores each lane's 8 columns of row r into a
// contraction-major buffer of 256-byte rows (chunk c of row r at c ^ 2 h(r),
// h(r) = r % 4 + 4 ((r / 8) % 2)), from which the A fragments (fragment row =
// column of W, contraction = row of W) come with LDS transpose reads as in
// k_dense_prefill_dma_tr; dY rows are staged and read as X is.  The same
// pipeline as k_sparse_prefill: words three stages ahead, windows and dY
// slabs two ahead, the next stage expanded before this stage's MFMAs, one
// barrier per stage.  M % 256 == 0, N % 64 == 0, K % 128 == 0 (every tile
// and slab inside the matrices).
template <class T>
__global__ void __launch_bounds__(512, 1) k_sparse_prefill_t(const PfArgs g) {
  static_assert(!std::is_same<T, I8P>::value, "16-bit payloads");
  extern __shared__ __align__(16) unsigned char dsm[];
  __shared__ __align__(16) uint32_t lut[32];
  using Acc = typename MfmaP<T>::acc_t;
  constexpr int NW = 8, BN = 128, BM = 256, FN = 4, FM = 4, TW = 2, RR = 8 * NW;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lane = tid & 63;
  const int wn = wave & 1, wm = wave >> 1;
  const int fr = lane & 15, fg = lane >> 4;
  const int64_t M = g.M, N = g.N, K = g.K;              // dY [M][N], W [N][K], dX [M][K]
  const int64_t S = tile_steps(K);
  const int nst = (int)(N / kPfBK);
  const int64_t k0 = (int64_t)blockIdx.x * BN, m0 = (int64_t)blockIdx.y * BM;
  const int64_t s0 = k0 / 32 + 2 * (wave & 1);          // my tiles' k-steps: s0, s0 + 1
  const int rbw = wave >> 1;                             // my row block within a stage
  const uint32_t abuf[2] = {lds_off(dsm), lds_off(dsm + kPfBK * kTrRowA)};
  const uint32_t bbuf[2] = {lds_off(dsm + 2 * kPfBK * kTrRowA), lds_off(dsm + 2 * kPfBK * kTrRowA + BM * kPfRow)};
  const uint32_t lut_addr = lds_off(lut);
  if (tid < 16) {
    lut[2 * tid] = nibble_selector16(tid, 0);
    lut[2 * tid + 1] = nibble_selector16(tid, 1);
  }
  // where my expanded 8 columns go: row r = 16 rbw + fr of the stage, chunk 4 (2 (w % 2) + i) + fg
  const int er = 16 * rbw + fr;
  const int eh = (er & 3) | (((er >> 3) & 1) << 2);
  uint32_t eo[TW];
#pragma unroll
  for (int i = 0; i < TW; ++i) eo[i] = (uint32_t)(er * kTrRowA + 16 * ((4 * (2 * (wave & 1) + i) + fg) ^ (2 * eh)));
  // my A fragments' first reads (as in k_dense_prefill_dma_tr)
  const int t = lane & 15, r0 = 8 * (lane >> 4) + (t >> 2);
  const int h = (t >> 2) | (((lane >> 4) & 1) << 2);
  uint32_t ao[FN];
#pragma unroll
  for (int i = 0; i < FN; ++i)
    ao[i] = (uint32_t)(r0 * kTrRowA + 16 * ((8 * wn + 2 * i + ((t & 3) >> 1)) ^ (2 * h)) + 8 * (t & 1));

  auto fetch_words = [&](TileWords<TW>& tw, int st) {
#pragma unroll
    for (int i = 0; i < TW; ++i) {
      const int64_t tt = (int64_t)(4 * st + rbw) * S + s0 + i;
      tw.w[i] = g.bm[tt * 16 + fr];
      tw.off[i] = g.toff[tt];
    }
  };
  auto fetch_windows = [&](TileWindows<TW>& tv, const TileWords<TW>& tw) {
    // the pair's values before mine: the exclusive wave scan of the lanes' kept counts (16-bit halves)
    const uint32_t b0 = __builtin_amdgcn_ubfe(tw.w[0], 8 * fg, 8);
    const uint32_t b1 = __builtin_amdgcn_ubfe(tw.w[1], 8 * fg, 8);
    const uint32_t pc = __popc(b0) | (__popc(b1) << 16);
    const uint32_t ex = wave_inclusive_scan(pc) - pc;
#pragma unroll
    for (int i = 0; i < TW; ++i) {
      const uint32_t byte = i ? b1 : b0;
      const uint32_t oa = (uint32_t)tw.off[i] + (i ? ex >> 16 : ex & 0xffffu);
      const uint32_t ob = oa + __popc(byte & 0xfu);
      tv.byte[i] = byte;
      __builtin_memcpy(&tv.v0[i], g.values + 2u * oa, 8);
      __builtin_memcpy(&tv.v1[i], g.values + 2u * ob, 8);
    }
  };
  auto expand_store = [&](const TileWindows<TW>& tv, uint32_t buf) {
#pragma unroll
    for (int i = 0; i < TW; ++i) {
      const u32x2 slo = lds_load8(lut_addr + 8u * (tv.byte[i] & 0xfu));
      const u32x2 shi = lds_load8(lut_addr + 8u * (tv.byte[i] >> 4));
      u32x4 a;
      a.x = __builtin_amdgcn_perm(tv.v0[i].y, tv.v0[i].x, slo.x);
      a.y = __builtin_amdgcn_perm(tv.v0[i].y, tv.v0[i].x, slo.y);
      a.z = __builtin_amdgcn_perm(tv.v1[i].y, tv.v1[i].x, shi.x);
      a.w = __builtin_amdgcn_perm(tv.v1[i].y, tv.v1[i].x, shi.y);
      *reinterpret_cast<__attribute__((address_space(3))) u32x4*>((uintptr_t)(buf + eo[i])) = a;
    }
  };

  Acc acc[FN][FM];
#pragma unroll
  for (int i = 0; i < FN; ++i)
#pragma unroll
    for (int j = 0; j < FM; ++j) acc[i][j] = Acc{0, 0, 0, 0};

  const SlabSrc<RR> xsrc(g.X, M, N, m0, tid);
  Slab<BM / RR> x0, x1;
  TileWords<TW> tw;
  TileWindows<TW> tv;
  if (nst > 0) {
    fetch_words(tw, 0);
    xsrc.template fetch<false>(x0, N, 0);
    fetch_windows(tv, tw);                               // stage 0
    if (nst > 1) {
      fetch_words(tw, 1);
      xsrc.template fetch<false>(x1, N, kPfBK);
    }
  }
  __syncthreads();                                       // the selector table
  if (nst > 0) {
    expand_store(tv, abuf[0]);
    slab_store<RR>(x0, bbuf[0], tid);
    if (nst > 1) {
      fetch_windows(tv, tw);                             // stage 1
      if (nst > 2) fetch_words(tw, 2);
    }
  }
  __syncthreads();
  // (xl holds stage st + 1; xn receives stage st + 2)
  auto step = [&](int st, Slab<BM / RR>& xn, Slab<BM / RR>& xl) {
    const int cur = st & 1;
    if (st + 1 < nst) {
      expand_store(tv, abuf[cur ^ 1]);                   // stage st + 1
      slab_store<RR>(xl, bbuf[cur ^ 1], tid);
      if (st + 2 < nst) {
        fetch_windows(tv, tw);                           // stage st + 2 (its words were fetched a stage ago)
        if (st + 3 < nst) fetch_words(tw, st + 3);
        xsrc.template fetch<false>(xn, N, (int64_t)kPfBK * (st + 2));
      }
    }
    pf_mfma_stage_trA<T, FN, FM>(acc, abuf[cur], ao, bbuf[cur], wm, fr, fg);
    if (st + 1 < nst) __syncthreads();
  };
  for (int st = 0; st < nst; st += 2) {
    step(st, x0, x1);
    if (st + 1 < nst) step(st + 1, x1, x0);
  }
  pf_store<T, FN, FM>(acc, g.Y, M, K, k0, m0, wn, wm, fr, fg);
}

int pf_cus() { return device_cus(); }

// Workgroup tile of a launch: 128 x 256 (8 waves) when that still gives every
// CU a workgroup, else 64 x 128 (4 waves, four times as many workgroups).
bool pf_large_tile(int64_t N, int64_t M) { return ((N + 127) / 128) * ((M + 255) / 256) >= (int64_t)pf_cus(); }

// Small tiles split K over two wave groups when they leave at most one
// workgroup per CU.
bool pf_split_k(int64_t N, int64_t M) { return ((N + 63) / 64) * ((M + 127) / 128) <= (int64_t)pf_cus(); }

// Blocks and stages all inside the matrix: the unchecked (branch-free) loads apply.
constexpr bool pf_inside(int64_t N, int64_t M, int64_t K, int BN, int BM) {
  return N % BN == 0 && M % BM == 0 && K % kPfBK == 0;
}

template <class T, int BN, int BM, int NW, int KS, bool kChecked, bool kGated = false>
hipError_t sparse_prefill_launch(const PfArgs& a, hipStream_t s) {
  auto* kernel = k_sparse_prefill<T, BN, BM, NW, KS, kChecked, kGated>;
  static PerDeviceFlag lds_set;
  constexpr int lds = KS * pf_lds(BN, BM);
  const hipError_t attr = allow_lds_once(lds_set, kernel, lds);
  if (attr != hipSuccess) return attr;
  constexpr int RN = kGated ? BN / 2 : BN;            // real rows per workgroup
  const dim3 grid((unsigned)((a.N + RN - 1) / RN), (unsigned)((a.M + BM - 1) / BM)), block(64 * NW * KS);
  hipLaunchKernelGGL(kernel, grid, block, lds, s, a);
  return hipGetLastError();
}

// Row length of the activations in 16-bit units.
template <class T>
constexpr int64_t pf_units(int64_t K) { return std::is_same<T, I8P>::value ? K / 2 : K; }

template <class T, int BN, int BM, int NW, int KS>
hipError_t sparse_prefill_tile(const PfArgs& a, hipStream_t s) {
  return pf_inside(a.N, a.M, pf_units<T>(a.K), BN, BM) ? sparse_prefill_launch<T, BN, BM, NW, KS, false>(a, s)
                                                       : sparse_prefill_launch<T, BN, BM, NW, KS, true>(a, s);
}

template <class T>
hipError_t sparse_prefill_t(const PfArgs& a, hipStream_t s) {
  if (pf_large_tile(a.N, a.M)) return sparse_prefill_tile<T, 128, 256, 8, 1>(a, s);
  return pf_split_k(a.N, a.M) ? sparse_prefill_tile<T, 64, 128, 4, 2>(a, s)
                              : sparse_prefill_tile<T, 64, 128, 4, 1>(a, s);
}

// Gated: the tiling of a launch of 2N virtual rows; inside when N % (BN / 2) == 0.
template <class T, int BN, int BM, int NW, int KS>
hipError_t gated_prefill_tile(const PfArgs& a, hipStream_t s) {
  return pf_inside(2 * a.N, a.M, a.K, BN, BM) ? sparse_prefill_launch<T, BN, BM, NW, KS, false, true>(a, s)
                                              : sparse_prefill_launch<T, BN, BM, NW, KS, true, true>(a, s);
}

template <class T>
hipError_t gated_prefill_t(const PfArgs& a, hipStream_t s) {
  const int64_t Nv = 2 * a.N;
  if (pf_large_tile(Nv, a.M)) return gated_prefill_tile<T, 128, 256, 8, 1>(a, s);
  return pf_split_k(Nv, a.M) ? gated_prefill_tile<T, 64, 128, 4, 2>(a, s) : gated_prefill_tile<T, 64, 128, 4, 1>(a, s);
}

template <class T, int BN, int BM, int NW, int KS, bool kChecked, bool kGather>
hipError_t dense_prefill_launch(const PfArgs& a, hipStream_t s) {
  auto* kernel = k_dense_prefill<T, BN, BM, NW, KS, kChecked, kGather>;
  static PerDeviceFlag lds_set;
  const hipError_t attr = allow_lds_once(lds_set, kernel, KS * pf_lds(BN, BM));
  if (attr != hipSuccess) return attr;
  const dim3 grid((unsigned)((a.N + BN - 1) / BN), (unsigned)((a.M + BM - 1) / BM)), block(64 * NW * KS);
  hipLaunchKernelGGL(kernel, grid, block, KS * pf_lds(BN, BM), s, a);
  return hipGetLastError();
}

template <class T, int BN, int BM, int NW, int KS, bool kGather>
hipError_t dense_prefill_tile(const PfArgs& a, hipStream_t s) {
  return pf_inside(a.N, a.M, pf_units<T>(a.K), BN, BM)
             ? dense_prefill_launch<T, BN, BM, NW, KS, false, kGather>(a, s)
             : dense_prefill_launch<T, BN, BM, NW, KS, true, kGather>(a, s);
}

template <class T, bool kGather>
hipError_t dense_prefill_dma(const PfArgs& a, hipStream_t s) {
  constexpr int NW = kDmaWaves;
  auto* kernel = k_dense_prefill_dma<T, kGather, NW>;
  static PerDeviceFlag lds_set;
  const hipError_t attr = allow_lds_once(lds_set, kernel, kDmaStages * kDmaStageBytes);
  if (attr != hipSuccess) return attr;
  const dim3 grid((unsigned)(a.N / kDmaBN), (unsigned)(a.M / kDmaBM)), block(64 * NW);
  hipLaunchKernelGGL(kernel, grid, block, kDmaStages * kDmaStageBytes, s, a);
  return hipGetLastError();
}

template <class T>
hipError_t dense_prefill_tr(const PfArgs* a, int count, hipStream_t s) {
  constexpr int NW = kDmaWaves;
  auto* kernel = k_dense_prefill_dma_tr<T, NW>;
  static PerDeviceFlag lds_set;
  const hipError_t attr = allow_lds_once(lds_set, kernel, kDmaStages * kDmaStageBytes);
  if (attr != hipSuccess) return attr;
  for (int c0 = 0; c0 < count; c0 += kTrGroupMax) {          // kTrGroupMax tasks per launch
    TrGroupArg ga{};
    ga.count = count - c0 < kTrGroupMax ? count - c0 : kTrGroupMax;
    ga.first[0] = 0;
    for (int i = 0; i < ga.count; ++i) {
      ga.t[i] = a[c0 + i];
      ga.first[i + 1] = ga.first[i] + (int32_t)((a[c0 + i].N / kDmaBN) * (a[c0 + i].M / kDmaBM));
    }
    hipLaunchKernelGGL(kernel, dim3((unsigned)ga.first[ga.count]), dim3(64 * NW), kDmaStages * kDmaStageBytes, s, ga);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <class T, bool kGather = false>
hipError_t dense_prefill_t(const PfArgs& a, hipStream_t s) {
  if (pf_large_tile(a.N, a.M) && pf_inside(a.N, a.M, pf_units<T>(a.K), kDmaBN, kDmaBM))
    return dense_prefill_dma<T, kGather>(a, s);
  if (pf_large_tile(a.N, a.M)) return dense_prefill_tile<T, 128, 256, 8, 1, kGather>(a, s);
  return pf_split_k(a.N, a.M) ? dense_prefill_tile<T, 64, 128, 4, 2, kGather>(a, s)
                              : dense_prefill_tile<T, 64, 128, 4, 1, kGather>(a, s);
}

}  // namespace

hipError_t launch_sparse_prefill(const void* X, int64_t M, const spl_matrix& Wc, void* Y, hipStream_t s) {
  if (Wc.nnz == 0) return launch_zero_fill(Y, M * Wc.rows, s);
  PfArgs a{};
  a.X = static_cast<const uint16_t*>(X);
  a.bm = Wc.bitmask;
  a.values = static_cast<const unsigned char*>(Wc.values);
  a.toff = Wc.tile_offsets;
  a.M = M, a.N = Wc.rows, a.K = Wc.cols;
  a.Y = static_cast<uint16_t*>(Y);
  return Wc.dtype == SPL_BF16 ? sparse_prefill_t<Bf16>(a, s) : sparse_prefill_t<F16>(a, s);
}

hipError_t launch_dense_prefill(const void* X, int64_t M, const void* W, int32_t dtype, int64_t N, int64_t K,
                                void* Y, hipStream_t s) {
  PfArgs a{};
  a.X = static_cast<const uint16_t*>(X);
  a.W = static_cast<const uint16_t*>(W);
  a.M = M, a.N = N, a.K = K;
  a.Y = static_cast<uint16_t*>(Y);
  return dtype == SPL_BF16 ? dense_prefill_t<Bf16>(a, s) : dense_prefill_t<F16>(a, s);
}

// The kept entries of X W^T at the tile pattern P ([M][N], P.rows == M,
// P.cols == N), in P's value order; no dense product is written.
hipError_t launch_dense_prefill_gather(const void* X, int64_t M, const void* W, int32_t dtype, int64_t N, int64_t K,
                                       const spl_matrix& P, void* values, hipStream_t s) {
  if (P.rows != M || P.cols != N) return hipErrorInvalidValue;
  PfArgs a{};
  a.X = static_cast<const uint16_t*>(X);
  a.W = static_cast<const uint16_t*>(W);
  a.M = M, a.N = N, a.K = K;
  a.gbm = P.bitmask, a.gtoff = P.tile_offsets, a.gval = static_cast<uint16_t*>(values);
  return dtype == SPL_BF16 ? dense_prefill_t<Bf16, true>(a, s) : dense_prefill_t<F16, true>(a, s);
}

// The kept entries of Xc^T Wc (Xc [K][M], Wc [K][N]) at the tile pattern P
// ([M][N]), in P's value order, read from the contraction-major factors
// directly.
bool dense_prefill_tr_applies(int64_t M, int64_t N, int64_t K, const void* Xc, const void* Wc) {
  return pf_large_tile(N, M) && pf_inside(N, M, K, kDmaBN, kDmaBM) &&
         (((uintptr_t)Xc | (uintptr_t)Wc) & 15) == 0;
}

hipError_t launch_dense_prefill_gather_tr(const TrTask* tasks, int count, int32_t dtype, hipStream_t s) {
  PfArgs a[SPL_MAX_GROUP];
  if (count < 1 || count > SPL_MAX_GROUP) return hipErrorInvalidValue;
  for (int i = 0; i < count; ++i) {
    const TrTask& t = tasks[i];
    if (t.P->rows != t.M || t.P->cols != t.N || !dense_prefill_tr_applies(t.M, t.N, t.K, t.Xc, t.Wc))
      return hipErrorInvalidValue;
    a[i] = PfArgs{};
    a[i].X = static_cast<const uint16_t*>(t.Xc);
    a[i].W = static_cast<const uint16_t*>(t.Wc);
    a[i].M = t.M, a[i].N = t.N, a[i].K = t.K;
    a[i].gbm = t.P->bitmask, a[i].gtoff = t.P->tile_offsets, a[i].gval = static_cast<uint16_t*>(t.values);
  }
  return dtype == SPL_BF16 ? dense_prefill_tr<Bf16>(a, count, s) : dense_prefill_tr<F16>(a, count, s);
}

// dX [M][K] = dY [M][N] (W.Mask) from W's packed tiles (W [N][K], tile layout).
bool sparse_input_grad_applies(int64_t M, const spl_matrix& W) {
  return M % 256 == 0 && W.rows % 64 == 0 && W.cols % 128 == 0 && pf_large_tile(W.cols, M);
}

hipError_t launch_sparse_input_grad(const void* dY, int64_t M, const spl_matrix& W, void* dX, hipStream_t s) {
  if (!sparse_input_grad_applies(M, W)) return hipErrorInvalidValue;
  PfArgs a{};
  a.X = static_cast<const uint16_t*>(dY);
  a.bm = W.bitmask;
  a.values = static_cast<const unsigned char*>(W.values);
  a.toff = W.tile_offsets;
  a.M = M, a.N = W.rows, a.K = W.cols;
  a.Y = static_cast<uint16_t*>(dX);
  auto* kernel = W.dtype == SPL_BF16 ? k_sparse_prefill_t<Bf16> : k_sparse_prefill_t<F16>;
  static PerDeviceFlag lds_set[2];
  const int lds = pf_lds(128, 256);
  const hipError_t attr = allow_lds_once(lds_set[W.dtype == SPL_BF16 ? 0 : 1], kernel, lds);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(kernel, dim3((unsigned)(W.cols / 128), (unsigned)(M / 256)), dim3(512), lds, s, a);
  return hipGetLastError();
}

// Gated half of a Llama MLP: Y = silu(X Wg^T) * (X Wu^T) (same dtype and shape).
hipError_t launch_gated_prefill(const void* X, int64_t M, const spl_matrix& Wg, const spl_matrix& Wu, void* Y,
                                hipStream_t s) {
  if (Wg.nnz == 0 || Wu.nnz == 0) return launch_zero_fill(Y, M * Wg.rows, s);   // silu(0) u = silu(g) 0 = 0
  PfArgs a{};
  a.X = static_cast<const uint16_t*>(X);
  a.bm = Wg.bitmask, a.values = static_cast<const unsigned char*>(Wg.values), a.toff = Wg.tile_offsets;
  a.bm2 = Wu.bitmask, a.values2 = static_cast<const unsigned char*>(Wu.values), a.toff2 = Wu.tile_offsets;
  a.M = M, a.N = Wg.rows, a.K = Wg.cols;
  a.Y = static_cast<uint16_t*>(Y);
  return Wg.dtype == SPL_BF16 ? gated_prefill_t<Bf16>(a, s) : gated_prefill_t<F16>(a, s);
}

// int8 (K % 16 == 0: activation rows are whole 16-byte pieces).
hipError_t launch_sparse_prefill_i8(const spl_int8_task& t, int64_t M, hipStream_t s) {
  const spl_matrix& W = *t.Wq;
  if (W.nnz == 0) {
    if (t.acc_out) {
      const hipError_t e = launch_zero_fill(t.acc_out, 2 * M * W.rows, s);
      if (e != hipSuccess) return e;
    }
    return launch_zero_fill(t.Y, M * W.rows, s);     // (float(0) * sx) * sw = +0
  }
  PfArgs a{};
  a.X = reinterpret_cast<const uint16_t*>(t.Xq);
  a.bm = W.bitmask;
  a.values = static_cast<const unsigned char*>(W.values);
  a.toff = W.tile_offsets;
  a.M = M, a.N = W.rows, a.K = W.cols;
  a.Y = static_cast<uint16_t*>(t.Y);
  a.sx = t.x_scales, a.sw = t.w_scales, a.acc = t.acc_out;
  return sparse_prefill_t<I8P>(a, s);
}

hipError_t launch_dense_prefill_i8(const spl_dense_int8_task& t, int64_t M, hipStream_t s) {
  PfArgs a{};
  a.X = reinterpret_cast<const uint16_t*>(t.Xq);
  a.W = reinterpret_cast<const uint16_t*>(t.Wq);
  a.M = M, a.N = t.N, a.K = t.K;
  a.Y = static_cast<uint16_t*>(t.Y);
  a.sx = t.x_scales, a.sw = t.w_scales, a.acc = t.acc_out;
  return dense_prefill_t<I8P>(a, s);
}

}  // namespace spl
