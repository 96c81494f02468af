// Decode-shaped kernels (batch M <= 32) for gfx950.
//
// Sparse (paper section 2.4.2): compressed submatrices move from HBM into the
// register file, the bitmask guides their expansion there, and the matrix
// cores consume the expanded operand as if it were dense.  On CDNA4:
//
//   * W is stored as 16 x 32 tiles, each with its 16 bitmask words and its
//     dense values (one tile = one MFMA A operand).  A workgroup owns one
//     16-row block of one matrix of the group; its waves (8, or 16 when the
//     grid has fewer than two row blocks per CU) split the block's k-steps
//     (tiles) into contiguous ranges;
//   * the values of consecutive tiles are contiguous, so a wave fetches a
//     chunk of tiles (as many as fit a 3 KB buffer, at most 8) with aligned,
//     coalesced 16-byte loads and stages them in LDS; the chunk's bitmask
//     words arrive with one coalesced load per 4 tiles and are regrouped by
//     row in LDS; the tile offsets of a wave's whole range come with one load
//     (one lane per tile) and size every chunk with a ballot;
//   * each wave is software-pipelined: the next chunk's values and words are
//     in flight while the current chunk is multiplied;
//   * lane (fr, fg) supplies tile row fr, columns 8fg..8fg+7, exactly its A
//     operand of v_mfma_f32_16x16x32 (8 bf16/fp16 values).  A tile's values
//     are stored by column group, then row, i.e. in lane order, so their
//     offset is the tile offset + the kept count of the lanes before (a wave
//     DPP scan of popcounts, two tiles per scan in 16-bit halves), and the
//     lanes of a half-wave read one contiguous run of LDS.  Each 4-column
//     nibble's values are read from LDS as an 8-byte window (aligned dword
//     reads + v_alignbyte_b32) and a 16-entry selector table expands them
//     with v_perm_b32 into the operand dwords (zero bytes where the bit is
//     clear);
//   * activations form the B operand (batch padded to 16 or 32 columns; the
//     padding lanes hold zeros).  The workgroup copies its X into LDS once
//     (and the kernel is held to 64 VGPRs, eight waves per SIMD, so that LDS
//     rather than registers bounds the workgroups per CU) when the copy is
//     small enough to leave several workgroups per CU: a single row (up to
//     32 KB; the dense comparator: any batch up to 32 KB), or a small batch
//     in a large grid (up to 32 KB); otherwise each chunk's operands are
//     loaded directly, which fetches only the live rows;
//   * the waves' partial 16x16 results are summed in a fixed order
//     (deterministic) and rounded once to the output type.
//
// One launch covers a group of independent matrices (for example q, k and v):
// the workgroups of all of them form one grid, so the launch and its ramp-up
// and tail are paid once.
//
// Dense comparator: the same decomposition and pipelining with the A operand
// loaded directly from the dense rows of W (aligned 16-byte loads).
#include <type_traits>

#include "spl_common.h"

namespace spl {
namespace {

// Waves per workgroup (W) is a template parameter: 8 for large grids, 16
// (a finer split of each row block's k-steps) when a launch has fewer than
// two row blocks per CU.
constexpr int kDecRows = 16;
constexpr int kChunk = 8;                   // sparse: at most this many tiles per chunk (4 when M > 16)
constexpr int kDenseChunk = 4;              // dense: tiles per chunk
constexpr int kVBuf = 3072;                 // staged value bytes per wave and chunk
constexpr int kVBufAlloc = kVBuf + 16;      // + room for the last 8-byte window's third dword
constexpr int kPieceRounds = kVBuf / 16 / kWave;
static_assert(kPieceRounds * kWave * 16 == kVBuf, "every round of 16-byte pieces is staged unconditionally");
constexpr int kOffsetLanes = kWave - 1;      // tiles whose offsets one load covers (lane i: tile base + i)
// Activations are staged in LDS when every task's M * 32S * 2 bytes fit this
// budget (32 KB): a sparse workgroup then needs at most ~61 KB of LDS (3 KB
// value buffer per wave), so at least two share a CU's 160 KB.
constexpr int kXLdsMax = 32 * 1024;
constexpr int kXLdsMaxSparse = 32 * 1024;

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

// Entry n expands a 4-column nibble n into two operand dwords.  16 entries of
// 8 bytes cover 32 LDS banks once, so lookups never conflict.
__device__ __forceinline__ void build_nibble_table(u32x2* lut) {
  if (threadIdx.x < 16) lut[threadIdx.x] = u32x2{nibble_selector16(threadIdx.x, 0), nibble_selector16(threadIdx.x, 1)};
}

// This wave's contiguous range of k-steps [*beg, *end) of S (W waves).
template <int W>
__device__ __forceinline__ void wave_range(int S, int wave, int* beg, int* end) {
  const int L = (S + W - 1) / W;
  const int b = wave * L < S ? wave * L : S;
  *beg = b;
  *end = b + L < S ? b + L : S;
}

// Activation operand read directly from X with raw buffer loads: lane
// (fr, fg) of batch tile t reads X[16t + fr][32s + 8fg .. +8].  The base and
// the byte size of X sit in the buffer descriptor (SGPRs), each lane keeps one
// 32-bit byte offset per batch tile (k-step 0) and the k-step goes in the
// scalar offset, so a load costs no vector ALU work.  A lane whose row is past
// M, or whose columns are past K, passes an offset beyond the buffer and the
// hardware returns zeros.  Needs 2 M K <= kXBufMax (the launcher checks).
constexpr uint32_t kXOob = 0x80000000u;              // an offset past any accepted X
constexpr int64_t kXBufMax = (int64_t)kXOob;
template <int MT>
struct XGlobal {
  __amdgpu_buffer_rsrc_t rsrc;
  uint32_t off[MT];
  __device__ __forceinline__ XGlobal(const uint16_t* __restrict__ X, int M, int64_t K, int fr, int fg) {
    rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(X), (short)0, (int)(2 * (int64_t)M * K),
                                             0x00020000);
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      const int m = 16 * t + fr;
      off[t] = m < M ? 2u * ((uint32_t)m * (uint32_t)K + 8u * (uint32_t)fg) : kXOob;
    }
  }
  // k-step s; ragged (wave-uniform): s is the last k-step and K % 32 != 0, so
  // some lanes' columns may lie past K
  __device__ __forceinline__ void load(u32x4 (&xb)[MT], int s, bool ragged, int fg, int64_t K) const {
#pragma unroll
    for (int t = 0; t < MT; ++t) {
      uint32_t o = off[t];
      if (ragged && (uint32_t)(32 * s + 8 * fg) >= (uint32_t)K) o = kXOob;
      xb[t] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, o, 64 * s, 0));
    }
  }
};

// Activations staged in LDS (MT == 1): rows of xs_stride(K) = 32*S + 8
// elements, zero past K (so a ragged last tile reads zeros), the 16-byte pad
// spreading rows over the LDS banks.  Lanes of padding batch rows (m >= M)
// read a 64-byte zero area and do not advance with k; their reads are
// masked off where the operand is kept in a register (one row at M = 1, so
// the activation reads move 64 bytes per tile instead of 1 KB).
__host__ __device__ __forceinline__ int64_t xs_stride(int64_t K) { return 32 * tile_steps(K) + 8; }

struct XShared {
  uint32_t addr;     // LDS byte address of k-step 0 of this lane's operand
  uint32_t step;     // bytes per k-step: 64, or 0 for padding rows
  __device__ __forceinline__ XShared(const uint16_t* xs, const u32x4* zero, int M, int64_t K, int fr, int fg) {
    const bool live = fr < M;
    const uint16_t* p = xs + (int64_t)fr * xs_stride(K) + 8 * fg;
    addr = live ? lds_off(p) : lds_off(zero + fg);
    step = live ? 64u : 0u;
  }
};

// Cooperative copy of X [M][K] into LDS rows of xs_stride(K) elements with
// zeros from K to 32*S, split so that the loads can be issued early.  Piece p
// (16 bytes) of the copy is row m = p / per_row, piece q = p % per_row of that
// row; each thread divides once and steps (m, q) by the thread count between
// rounds.  Staged copies hold at most kXLdsMax bytes, so every product here
// is below 2^24 (24-bit multiplies).
template <int W>
struct XStager {
  static constexpr int kThreads = W * kWave;
  static constexpr int kXRounds = kXLdsMax / 16 / kThreads;   // staged pieces per thread (bounds M * 4S)
  // pieces held in registers between load() and store(); store() copies any
  // further rounds itself, in batches of kXHold
  static constexpr int kXHold = kXRounds < 4 ? kXRounds : 4;
  u32x4 r[kXHold];
  int per_row, total, kp, m0, q0, dm, dq;
  __device__ __forceinline__ void start(int M, int64_t K) {
    per_row = (int)(4 * tile_steps(K));          // 16-byte pieces per staged row (up to 32*S)
    kp = (int)(K / 8);                           // pieces that hold activations
    total = M * per_row;
    dm = kThreads / per_row;                     // wave-uniform
    dq = kThreads - dm * per_row;
    const int p = threadIdx.x;                   // < kThreads <= 1024: a float estimate corrected by one step
    int m = (int)((float)p * (1.0f / (float)per_row));
    if ((int)__umul24(m, per_row) > p) --m;
    if ((int)__umul24(m + 1, per_row) <= p) ++m;
    m0 = m;
    q0 = p - (int)__umul24(m, per_row);
  }
  __device__ __forceinline__ void next(int& m, int& q) const {
    m += dm;
    q += dq;
    if (q >= per_row) q -= per_row, ++m;
  }
  // rounds [i0, i0 + kXHold) into r, (m, q) the coordinates of round i0
  __device__ __forceinline__ void load_batch(const uint16_t* __restrict__ X, int64_t K, int i0, int m, int q) {
#pragma unroll
    for (int i = 0; i < kXHold; ++i) {
      const int p = threadIdx.x + (i0 + i) * kThreads;
      r[i] = u32x4{0u, 0u, 0u, 0u};
      if (p < total && q < kp)   // 32-bit byte offsets from the uniform base (SGPR-based loads)
        r[i] = *reinterpret_cast<const u32x4*>(reinterpret_cast<const unsigned char*>(X) +
                                               2u * (__umul24(m, (uint32_t)K) + 8u * (uint32_t)q));
      next(m, q);
    }
  }
  __device__ __forceinline__ void store_batch(uint16_t* xs, uint32_t stride, int i0, int& m, int& q) const {
#pragma unroll
    for (int i = 0; i < kXHold; ++i) {
      const int p = threadIdx.x + (i0 + i) * kThreads;
      if (p < total) *reinterpret_cast<u32x4*>(xs + __umul24(m, stride) + 8 * q) = r[i];
      next(m, q);
    }
  }
  __device__ __forceinline__ void load(const uint16_t* __restrict__ X, int M, int64_t K) {
    start(M, K);
    load_batch(X, K, 0, m0, q0);
  }
  __device__ __forceinline__ void store(uint16_t* xs, const uint16_t* __restrict__ X, int64_t K) {
    const uint32_t stride = (uint32_t)xs_stride(K);
    int m = m0, q = q0;
    store_batch(xs, stride, 0, m, q);
    for (int i0 = kXHold; i0 < kXRounds && threadIdx.x + i0 * kThreads - (threadIdx.x & 63) < total; i0 += kXHold) {
      load_batch(X, K, i0, m, q);
      int ms = m, qs = q;
      store_batch(xs, stride, i0, ms, qs);
      m = ms, q = qs;
    }
  }
};

// Sum the waves' partial accumulators (lane layout of the 16x16 MFMA result:
// lane l, register i holds row 4*(l/16)+i, column l%16) and store Y[m][n].
// Called by every thread after all waves have finished with `red`'s memory.
template <class T, int MT, int W>
__device__ __forceinline__ void reduce_store(float* red, const f32x4 (&acc)[MT], int M, int64_t n0, int64_t N,
                                             uint16_t* __restrict__ Y) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int t = 0; t < MT; ++t) *reinterpret_cast<f32x4*>(red + ((wave * MT + t) * 64 + lane) * 4) = acc[t];
  __syncthreads();
  for (int e = threadIdx.x; e < 256 * MT; e += W * kWave) {
    const int t = e >> 8;
    const int li = (e >> 2) & 63;
    const int ri = e & 3;
    const int64_t n = n0 + 4 * (li >> 4) + ri;
    const int m = t * 16 + (li & 15);
    if (m < M && n < N) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < W; ++w) s += red[((w * MT + t) * 64 + li) * 4 + ri];
      Y[(int64_t)m * N + n] = T::from_f32(s);
    }
  }
}

// As reduce_store for a gate and an up accumulator of the same row block:
// Y[m][n] = silu(g) * u with g and u the fp32 sums of the waves (fixed order).
template <class T, int W>
__device__ __forceinline__ void reduce_store_gated(float* red, const f32x4& ag, const f32x4& au, int M, int64_t n0,
                                                   int64_t N, uint16_t* __restrict__ Y) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  *reinterpret_cast<f32x4*>(red + ((wave * 2 + 0) * 64 + lane) * 4) = ag;
  *reinterpret_cast<f32x4*>(red + ((wave * 2 + 1) * 64 + lane) * 4) = au;
  __syncthreads();
  for (int e = threadIdx.x; e < 256; e += W * kWave) {
    const int li = (e >> 2) & 63;
    const int ri = e & 3;
    const int64_t n = n0 + 4 * (li >> 4) + ri;
    const int m = li & 15;
    if (m < M && n < N) {
      float sg = 0.f, su = 0.f;
#pragma unroll
      for (int w = 0; w < W; ++w) {
        sg += red[((w * 2 + 0) * 64 + li) * 4 + ri];
        su += red[((w * 2 + 1) * 64 + li) * 4 + ri];
      }
      Y[(int64_t)m * N + n] = T::from_f32(sg / (1.0f + expf(-sg)) * su);
    }
  }
}

// ------------------------------------------------------------------ groups

struct SparseTaskArg {
  const uint16_t* X;
  uint16_t* Y;
  const uint32_t* bm;
  const uint16_t* values;
  const int32_t* toff;
  int64_t N, K;
};
struct SparseGroupArg {
  SparseTaskArg t[SPL_MAX_GROUP];
  int32_t first[SPL_MAX_GROUP + 1];   // first workgroup of each task; first[count] = grid size
  int32_t count;
  int32_t M;
};
struct DenseTaskArg {
  const uint16_t* X;
  uint16_t* Y;
  const uint16_t* W;
  int64_t N, K;
};
struct DenseGroupArg {
  DenseTaskArg t[SPL_MAX_GROUP];
  int32_t first[SPL_MAX_GROUP + 1];
  int32_t count;
  int32_t M;
};


// Dynamic LDS of the sparse kernel: per-wave value staging buffers (later the
// reduction buffer), then (XL) the staged activations.
template <int W>
constexpr size_t sparse_vbuf_bytes() { return (size_t)W * kVBufAlloc; }

// A chunk: `cn` tiles from c0 whose values occupy the 16-byte pieces
// [a0, a0 + 16 np) of the value bytes.
struct Chunk {
  int cn;
  uint32_t a0;
  int np;
};

template <class T, int MT, bool XL, int W>
__global__ void __launch_bounds__(W * kWave, XL ? 8 : 4) k_sparse_decode(const SparseGroupArg g) {
  constexpr int C = MT == 1 ? kChunk : kChunk / 2;
  extern __shared__ __align__(16) unsigned char dsm[];
  __shared__ u32x2 lut[16];
  __shared__ u32x4 xzero[4];
  // per wave: [row][tile of the chunk]; the row stride C + 2 (even, for the 8-byte pair reads) puts
  // the 16 rows in distinct banks
  constexpr int WS = C + 2;
  __shared__ __align__(16) uint32_t words[W][16 * WS];
  const int ti = find_task(g.first, g.count);
  const SparseTaskArg tk = g.t[ti];
  const int M = g.M;
  const int64_t K = tk.K;
  const int64_t blk = (int64_t)blockIdx.x - g.first[ti];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int fr = lane & 15, fg = lane >> 4;
  const int S = (int)tile_steps(K);
  int kbeg, kend;
  wave_range<W>(S, wave, &kbeg, &kend);
  unsigned char* vbuf = dsm + wave * kVBufAlloc;
  uint16_t* xs = reinterpret_cast<uint16_t*>(dsm + sparse_vbuf_bytes<W>());
  const uint32_t* bmb = tk.bm + blk * S * 16;         // this row block's tiles, 16 words each
  const int32_t* tob = tk.toff + blk * S;             // S + 1 entries (the next block's first = this end)
  const unsigned char* vbytes = reinterpret_cast<const unsigned char*>(tk.values);
  uint32_t* wl = words[wave];

  // Offsets of the wave's tiles: lane i holds the offset of tile ob + i
  // (clamped to the range end), for tiles ob .. ob + kOffsetLanes; one load
  // covers every chunk of a range of up to kOffsetLanes tiles.
  int ob = kbeg;
  auto load_offsets = [&](int base) {
    const int t = base + lane < kend ? base + lane : kend;
    return *reinterpret_cast<const int32_t*>(reinterpret_cast<const unsigned char*>(tob) + 4u * (uint32_t)t);
  };
  // The most tiles (<= C, inside the range) from c0 whose values fit the
  // staging buffer: tile j fits iff its end offset <= (a0 + kVBuf) / 2, and
  // the offsets do not decrease, so the count of fitting lanes is the length.
  auto shape = [&](int32_t o, int c0) {
    Chunk ch;
    const int r = c0 - ob;                                  // lane of tile c0 (r + C <= kOffsetLanes)
    ch.a0 = (2u * (uint32_t)__builtin_amdgcn_readlane(o, r)) & ~15u;
    const uint32_t lim = (ch.a0 + kVBuf) >> 1;
    const int jmax = kend - c0 < C ? kend - c0 : C;
    const bool fit = lane >= r + 1 && lane <= r + jmax && (uint32_t)o <= lim;
    ch.cn = __builtin_popcountll(__ballot(fit));            // >= 1: one tile is at most 1 KB
    const uint32_t end = (uint32_t)__builtin_amdgcn_readlane(o, r + ch.cn);
    ch.np = (int)((2u * end - ch.a0 + 15u) >> 4);           // <= kVBuf / 16
    return ch;
  };
  u32x4 vp[kPieceRounds];
  uint32_t wv[C / 4];
  // Unconditional loads: a piece past the chunk's np reloads piece 0 of the
  // chunk, a tile past the range reloads the range's last tile; what they
  // bring is staged but never read (the expansion selects only kept values of
  // the chunk's tiles).  32-bit byte offsets from wave-uniform bases (values
  // < 2^32 bytes: nnz < 2^31 of 2 bytes; bitmask < 2^32 bytes per matrix).
  auto issue = [&](const Chunk& ch, int c0) {
#pragma unroll
    for (int r = 0; r < kPieceRounds; ++r) {
      const uint32_t piece = (uint32_t)(lane + kWave * r);
      const uint32_t off = ch.a0 + (piece < (uint32_t)ch.np ? 16u * piece : 0u);
      vp[r] = *reinterpret_cast<const u32x4*>(vbytes + off);
    }
#pragma unroll
    for (int i = 0; i < C / 4; ++i) {
      const int t = c0 + fg + 4 * i < kend ? c0 + fg + 4 * i : kend - 1;
      const uint32_t wb = 4u * ((uint32_t)t * 16u + (uint32_t)fr);
      wv[i] = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const unsigned char*>(bmb) + wb);
    }
  };

  // prologue: the range's offsets, then the first chunk and the activations in flight (offsets first:
  // loads complete in issue order, and the chunk's addresses wait on them), then the shared tables
  int32_t orng = 0;
  Chunk ch{0, 0u, 0};
  // direct path: a chunk's activations are loaded with its values (every
  // tile of the chunk unconditionally: a k-step past the chunk reads in-range
  // X or, past the buffer, zeros, and is not used), so that their latency
  // overlaps the previous chunk's products
  u32x4 xn[XL ? 1 : C][MT];
  auto load_x_chunk = [&](int c) {
    if constexpr (!XL) {
      const XGlobal<MT> xg(tk.X, M, K, fr, fg);
#pragma unroll
      for (int j = 0; j < C; ++j) xg.load(xn[j], c + j, c + j == S - 1 && (K & 31) != 0, fg, K);
    }
  };
  if (kbeg < kend) {
    orng = load_offsets(ob);
    ch = shape(orng, kbeg);
    issue(ch, kbeg);
    load_x_chunk(kbeg);
  }
  XStager<W> xst;
  if constexpr (XL) xst.load(tk.X, M, K);
  build_nibble_table(lut);
  if (threadIdx.x < 4) xzero[threadIdx.x] = u32x4{0u, 0u, 0u, 0u};
  if constexpr (XL) xst.store(xs, tk.X, K);
  __syncthreads();

  using XOp = std::conditional_t<XL, XShared, XGlobal<MT>>;
  const XOp xop = [&]() {
    if constexpr (XL) return XShared(xs, xzero, M, K, fr, fg);
    else return XGlobal<MT>(tk.X, M, K, fr, fg);
  }();

  const uint32_t lut_addr = lds_off(lut);
  const uint32_t vbuf_addr = lds_off(vbuf);
  u32x4 xlive = u32x4{0u, 0u, 0u, 0u};

  f32x4 acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int c0 = kbeg; c0 < kend;) {
    // 1. stage the current chunk: values into the buffer, words regrouped by row
#pragma unroll
    for (int r = 0; r < kPieceRounds; ++r) *reinterpret_cast<u32x4*>(vbuf + 16 * (lane + kWave * r)) = vp[r];
#pragma unroll
    for (int i = 0; i < C / 4; ++i) wl[fr * WS + fg + 4 * i] = wv[i];
    wave_lds_sync();
    const Chunk cur = ch;
    int32_t tc[C];                                     // the chunk's tile offsets (wave-uniform)
#pragma unroll
    for (int j = 0; j < C; ++j) tc[j] = __builtin_amdgcn_readlane(orng, c0 - ob + j);

    // 2. the current chunk's activations (direct path), then the next chunk's loads and activations
    u32x4 xb[XL ? 1 : C][MT];
    if constexpr (!XL) {
#pragma unroll
      for (int j = 0; j < C; ++j)
#pragma unroll
        for (int t = 0; t < MT; ++t) xb[j][t] = xn[j][t];
    }
    const int c1 = c0 + cur.cn;
    if (c1 < kend) {
      if (c1 - ob + C > kOffsetLanes) {                // past the loaded offsets (ranges over 63 - C tiles)
        ob = c1;
        orng = load_offsets(ob);
      }
      ch = shape(orng, c1);
      issue(ch, c1);
      load_x_chunk(c1);
    }

    // 3. expand and multiply the current chunk, two tiles at a time
    const uint32_t vrel = vbuf_addr - cur.a0;          // LDS address of value byte 0 (a multiple of 4 apart)
    uint32_t xaddr = 0;
    if constexpr (XL) xaddr = xop.addr + xop.step * (uint32_t)c0;
    // values stored before mine in each tile: a tile's values are ordered by
    // column group (my fg), then row (my fr), so this is the exclusive wave scan
    // of the lanes' kept counts, two tiles per scan in 16-bit halves (sums <=
    // 512).  The chunk's scans are independent and run together, so their DPP
    // steps interleave (tiles past the chunk scan staged words no one reads).
    u32x2 wps[C / 2];
    uint32_t exs[C / 2];
#pragma unroll
    for (int q = 0; q < C / 2; ++q) wps[q] = *reinterpret_cast<const u32x2*>(wl + fr * WS + 2 * q);
#pragma unroll
    for (int q = 0; q < C / 2; ++q) {
      const uint32_t pc = __popc(__builtin_amdgcn_ubfe(wps[q].x, 8 * fg, 8)) |
                          (__popc(__builtin_amdgcn_ubfe(wps[q].y, 8 * fg, 8)) << 16);
      exs[q] = wave_inclusive_scan(pc) - pc;
    }
#pragma unroll
    for (int jp = 0; jp < C; jp += 2) {
      if (jp < cur.cn) {
        const u32x2 wp = wps[jp / 2];
        const uint32_t ex = exs[jp / 2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int j = jp + h;
          if (j < cur.cn) {
            const uint32_t wj = h ? wp.y : wp.x;
            const uint32_t before = h ? ex >> 16 : ex & 0xffffu;
            const uint32_t nlo = __builtin_amdgcn_ubfe(wj, 8 * fg, 4);      // my two nibbles
            const uint32_t nhi = __builtin_amdgcn_ubfe(wj, 8 * fg + 4, 4);
            const uint32_t tile0 = (uint32_t)tc[j];
            const uint32_t oa = before + tile0;                             // first value of each nibble
            const uint32_t ob = oa + __popc(nlo);
            // LDS byte addresses of the two 8-byte windows; their low 2 bits are the realignment
            const uint32_t pa = 2u * oa + vrel, pb = 2u * ob + vrel;
            const uint32_t da = pa & ~3u, db = pb & ~3u;
            const uint32_t a_0 = lds_load4(da), a_1 = lds_load4(da + 4), a_2 = lds_load4(da + 8);
            const uint32_t b_0 = lds_load4(db), b_1 = lds_load4(db + 4), b_2 = lds_load4(db + 8);
            const uint32_t vlo = __builtin_amdgcn_alignbyte(a_1, a_0, pa);
            const uint32_t vhi = __builtin_amdgcn_alignbyte(a_2, a_1, pa);
            const uint32_t ulo = __builtin_amdgcn_alignbyte(b_1, b_0, pb);
            const uint32_t uhi = __builtin_amdgcn_alignbyte(b_2, b_1, pb);
            const u32x2 slo = lds_load8(lut_addr + 8u * nlo), shi = lds_load8(lut_addr + 8u * nhi);
            u32x4 a;
            a.x = __builtin_amdgcn_perm(vhi, vlo, slo.x);
            a.y = __builtin_amdgcn_perm(vhi, vlo, slo.y);
            a.z = __builtin_amdgcn_perm(uhi, ulo, shi.x);
            a.w = __builtin_amdgcn_perm(uhi, ulo, shi.y);
            if constexpr (XL) {
              if (xop.step) xlive = lds_load16(xaddr);   // padding rows keep their zero operand
              acc[0] = Mfma16<T>::run(a, xlive, acc[0]);
              xaddr += xop.step;
            } else {
#pragma unroll
              for (int t = 0; t < MT; ++t) acc[t] = Mfma16<T>::run(a, xb[j][t], acc[t]);
            }
          }
        }
      }
    }
    wave_lds_sync();                                   // the next chunk overwrites the buffers
    c0 = c1;
  }
  __syncthreads();                                     // every wave is done with its staging buffer
  reduce_store<T, MT, W>(reinterpret_cast<float*>(dsm), acc, M, blk * kDecRows, tk.N, tk.Y);
}

// Two row blocks per workgroup, for batches whose activations are loaded
// directly (MT batch tiles of 16 rows): every wave walks the same k-range of
// both blocks, so each activation load feeds two MFMAs per batch tile (halving
// the activation loads, which bound this case).  Each block keeps its own offsets window, half of the
// staging buffer, regrouped words and accumulator; a chunk is as many tiles as
// fit both halves.  The second block of a pair past the last row block aliases
// the first with zero words and is not stored.  Otherwise the same steps as
// k_sparse_decode.
constexpr int kHalfVBuf = kVBuf / 2;                 // staged value bytes per block and chunk
constexpr int kHalfVBufAlloc = kHalfVBuf + 16;       // + room for an 8-byte window at the last value
constexpr int kHalfPieceRounds = (kHalfVBuf / 16 + kWave - 1) / kWave;

template <int W>
constexpr size_t sparse2_vbuf_bytes() { return (size_t)W * 2 * kHalfVBufAlloc; }

struct Chunk2 {
  int cn;
  uint32_t a0[2];
  int np[2];
};

// kGated: the gated half of a Llama MLP.  Task 0 is the gate and task 1 the up
// projection (same X, N, K); workgroup j pairs row block j of both and stores
// silu(gate) * up (silu(z) = z / (1 + e^-z), from the fp32 sums) into task 0's Y.
// XL (one activation row): the row is staged in LDS after the value buffers,
// as in k_sparse_decode, and both blocks' MFMAs read it from there.
template <class T, int W, bool kGated, bool XL = false, int MT = 1>
__global__ void __launch_bounds__(W * kWave, 4) k_sparse_decode2(const SparseGroupArg g) {
  static_assert(MT == 1 || (!kGated && !XL), "two batch tiles: plain products with direct activations");
  static_assert((size_t)W * MT * 256 * sizeof(float) <= sparse2_vbuf_bytes<W>(), "one block's partial sums fit");
  constexpr int C = MT == 1 ? kChunk : kChunk / 2;
  extern __shared__ __align__(16) unsigned char dsm[];
  __shared__ u32x2 lut[16];
  __shared__ __align__(16) u32x4 xzero[4];
  constexpr int WS = C + 2;                          // word row stride (see k_sparse_decode)
  __shared__ __align__(16) uint32_t words[W][2][16 * WS];
  const int ti = kGated ? 0 : find_task(g.first, g.count);
  const SparseTaskArg tk = g.t[ti];
  const SparseTaskArg tu = g.t[kGated ? 1 : ti];
  const int M = g.M;
  const int64_t K = tk.K;
  const int64_t B = tile_blocks(tk.N);
  const int64_t blk0 = kGated ? (int64_t)blockIdx.x : 2 * ((int64_t)blockIdx.x - g.first[ti]);
  const bool live1 = kGated || blk0 + 1 < B;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int fr = lane & 15, fg = lane >> 4;
  const int S = (int)tile_steps(K);
  int kbeg, kend;
  wave_range<W>(S, wave, &kbeg, &kend);
  unsigned char* vbuf[2] = {dsm + wave * 2 * kHalfVBufAlloc, dsm + wave * 2 * kHalfVBufAlloc + kHalfVBufAlloc};
  const int64_t blkb[2] = {blk0, kGated ? blk0 : (live1 ? blk0 + 1 : blk0)};
  const uint32_t* bmb[2] = {tk.bm + blkb[0] * S * 16, tu.bm + blkb[1] * S * 16};
  const int32_t* tob[2] = {tk.toff + blkb[0] * S, tu.toff + blkb[1] * S};
  const unsigned char* vbs[2] = {reinterpret_cast<const unsigned char*>(tk.values),
                                 reinterpret_cast<const unsigned char*>(tu.values)};

  int ob = kbeg;
  auto load_offsets = [&](int b, int base) {
    const int t = base + lane < kend ? base + lane : kend;
    return tob[b][t];
  };
  auto shape = [&](const int32_t (&o)[2], int c0) {
    Chunk2 ch;
    const int r = c0 - ob;                             // lane of tile c0 (r + C <= kOffsetLanes)
    const int jmax = kend - c0 < C ? kend - c0 : C;
    int cn = C;
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      ch.a0[b] = (2u * (uint32_t)__builtin_amdgcn_readlane(o[b], r)) & ~15u;
      const uint32_t lim = (ch.a0[b] + kHalfVBuf) >> 1;
      const bool fit = lane >= r + 1 && lane <= r + jmax && (uint32_t)o[b] <= lim;
      const int cb = __builtin_popcountll(__ballot(fit));   // >= 1: one tile is at most 1 KB
      cn = cb < cn ? cb : cn;
    }
    ch.cn = cn;
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const uint32_t end = (uint32_t)__builtin_amdgcn_readlane(o[b], r + cn);
      ch.np[b] = (int)((2u * end - ch.a0[b] + 15u) >> 4);  // <= kHalfVBuf / 16
    }
    return ch;
  };
  u32x4 vp[2][kHalfPieceRounds];
  uint32_t wv[2][C / 4];
  auto issue = [&](const Chunk2& ch, int c0) {
#pragma unroll
    for (int b = 0; b < 2; ++b) {
#pragma unroll
      for (int r = 0; r < kHalfPieceRounds; ++r) {
        vp[b][r] = u32x4{0u, 0u, 0u, 0u};
        const uint32_t off = ch.a0[b] + 16u * (uint32_t)(lane + kWave * r);
        if (lane + kWave * r < ch.np[b]) vp[b][r] = *reinterpret_cast<const u32x4*>(vbs[b] + off);
      }
#pragma unroll
      for (int i = 0; i < C / 4; ++i) {
        wv[b][i] = 0u;
        const uint32_t wi = (uint32_t)(c0 + fg + 4 * i) * 16u + (uint32_t)fr;
        if (fg + 4 * i < ch.cn && (b == 0 || live1)) wv[b][i] = bmb[b][wi];
      }
    }
  };

  uint16_t* xs = reinterpret_cast<uint16_t*>(dsm + sparse2_vbuf_bytes<W>());
  int32_t orng[2] = {0, 0};
  Chunk2 ch{0, {0u, 0u}, {0, 0}};
  if (kbeg < kend) {                                 // offsets first (see k_sparse_decode)
    orng[0] = load_offsets(0, ob);
    orng[1] = load_offsets(1, ob);
    ch = shape(orng, kbeg);
    issue(ch, kbeg);
  }
  XStager<W> xst;
  if constexpr (XL) xst.load(tk.X, M, K);
  build_nibble_table(lut);
  if (threadIdx.x < 4) xzero[threadIdx.x] = u32x4{0u, 0u, 0u, 0u};
  if constexpr (XL) xst.store(xs, tk.X, K);
  __syncthreads();

  const XGlobal<MT> xop(tk.X, M, K, fr, fg);
  const XShared xsh(xs, xzero, M, K, fr, fg);        // (XL only)
  const uint32_t lut_addr = lds_off(lut);
  const uint32_t vbuf_addr[2] = {lds_off(vbuf[0]), lds_off(vbuf[1])};
  f32x4 acc[2][MT];
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int t = 0; t < MT; ++t) acc[b][t] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int c0 = kbeg; c0 < kend;) {
    // 1. stage the current chunk of both blocks
#pragma unroll
    for (int b = 0; b < 2; ++b) {
#pragma unroll
      for (int r = 0; r < kHalfPieceRounds; ++r)
        if (lane + kWave * r < ch.np[b]) *reinterpret_cast<u32x4*>(vbuf[b] + 16 * (lane + kWave * r)) = vp[b][r];
#pragma unroll
      for (int i = 0; i < C / 4; ++i) words[wave][b][fr * WS + fg + 4 * i] = wv[b][i];
    }
    wave_lds_sync();
    const Chunk2 cur = ch;
    int32_t tc[2][C];
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int j = 0; j < C; ++j) tc[b][j] = __builtin_amdgcn_readlane(orng[b], c0 - ob + j);

    // 2. the chunk's activations, then the next chunk's loads
    u32x4 xb[C][MT];
    if constexpr (!XL) {
#pragma unroll
      for (int j = 0; j < C; ++j)
        if (j < cur.cn) xop.load(xb[j], c0 + j, c0 + j == S - 1 && (K & 31) != 0, fg, K);
    }
    const int c1 = c0 + cur.cn;
    if (c1 < kend) {
      if (c1 - ob + C > kOffsetLanes) {
        ob = c1;
        orng[0] = load_offsets(0, ob);
        orng[1] = load_offsets(1, ob);
      }
      ch = shape(orng, c1);
      issue(ch, c1);
    }

    // 3. expand both blocks' tiles and multiply each with the shared activation operand
    const uint32_t vrel[2] = {vbuf_addr[0] - cur.a0[0], vbuf_addr[1] - cur.a0[1]};
#pragma unroll
    for (int jp = 0; jp < C; jp += 2) {
      if (jp < cur.cn) {
        u32x2 wp[2];
        uint32_t ex[2];
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          wp[b] = *reinterpret_cast<const u32x2*>(&words[wave][b][fr * WS + jp]);
          const uint32_t pc = __popc(__builtin_amdgcn_ubfe(wp[b].x, 8 * fg, 8)) |
                              (__popc(__builtin_amdgcn_ubfe(wp[b].y, 8 * fg, 8)) << 16);
          ex[b] = wave_inclusive_scan(pc) - pc;
        }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int j = jp + h;
          if (j < cur.cn) {
            if constexpr (XL) {                      // staged row: zeros past K; padding rows stay zero
              xb[j][0] = u32x4{0u, 0u, 0u, 0u};
              if (xsh.step) xb[j][0] = lds_load16(xsh.addr + xsh.step * (uint32_t)(c0 + j));
            }
#pragma unroll
            for (int b = 0; b < 2; ++b) {
              const uint32_t wj = h ? wp[b].y : wp[b].x;
              const uint32_t before = h ? ex[b] >> 16 : ex[b] & 0xffffu;
              const uint32_t nlo = __builtin_amdgcn_ubfe(wj, 8 * fg, 4);
              const uint32_t nhi = __builtin_amdgcn_ubfe(wj, 8 * fg + 4, 4);
              const uint32_t oa = before + (uint32_t)tc[b][j];
              const uint32_t obv = oa + __popc(nlo);
              const uint32_t pa = 2u * oa + vrel[b], pb = 2u * obv + vrel[b];
              const uint32_t da = pa & ~3u, db = pb & ~3u;
              const uint32_t a_0 = lds_load4(da), a_1 = lds_load4(da + 4), a_2 = lds_load4(da + 8);
              const uint32_t b_0 = lds_load4(db), b_1 = lds_load4(db + 4), b_2 = lds_load4(db + 8);
              const uint32_t vlo = __builtin_amdgcn_alignbyte(a_1, a_0, pa);
              const uint32_t vhi = __builtin_amdgcn_alignbyte(a_2, a_1, pa);
              const uint32_t ulo = __builtin_amdgcn_alignbyte(b_1, b_0, pb);
              const uint32_t uhi = __builtin_amdgcn_alignbyte(b_2, b_1, pb);
              const u32x2 slo = lds_load8(lut_addr + 8u * nlo), shi = lds_load8(lut_addr + 8u * nhi);
              u32x4 a;
              a.x = __builtin_amdgcn_perm(vhi, vlo, slo.x);
              a.y = __builtin_amdgcn_perm(vhi, vlo, slo.y);
              a.z = __builtin_amdgcn_perm(uhi, ulo, shi.x);
              a.w = __builtin_amdgcn_perm(uhi, ulo, shi.y);
#pragma unroll
              for (int t = 0; t < MT; ++t) acc[b][t] = Mfma16<T>::run(a, xb[j][t], acc[b][t]);
            }
          }
        }
      }
    }
    wave_lds_sync();
    c0 = c1;
  }
  __syncthreads();                                     // every wave is done with its staging buffers
  float* red = reinterpret_cast<float*>(dsm);
  if constexpr (kGated) {
    reduce_store_gated<T, W>(red, acc[0][0], acc[1][0], M, blk0 * kDecRows, tk.N, tk.Y);
    return;
  }
  reduce_store<T, MT, W>(red, acc[0], M, blk0 * kDecRows, tk.N, tk.Y);
  if (live1) {
    __syncthreads();                                   // the first block's sums are read before red is reused
    reduce_store<T, MT, W>(red, acc[1], M, (blk0 + 1) * kDecRows, tk.N, tk.Y);
  }
}

template <class T, int MT, bool XL, int W>
__global__ void __launch_bounds__(W * kWave, XL ? 8 : 4) k_dense_decode(const DenseGroupArg g) {
  constexpr int C = kDenseChunk;
  extern __shared__ __align__(16) unsigned char dsm[];
  __shared__ u32x4 xzero[4];
  const int ti = find_task(g.first, g.count);
  const DenseTaskArg tk = g.t[ti];
  const int M = g.M;
  const int64_t K = tk.K, N = tk.N;
  const int64_t blk = (int64_t)blockIdx.x - g.first[ti];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int fr = lane & 15, fg = lane >> 4;
  const int S = (int)tile_steps(K);
  int kbeg, kend;
  wave_range<W>(S, wave, &kbeg, &kend);
  uint16_t* xs = reinterpret_cast<uint16_t*>(dsm);
  const int64_t row = blk * kDecRows + fr < N ? blk * kDecRows + fr : N - 1;   // rows past N feed discarded outputs
  const uint16_t* wrow = tk.W + row * K + 8 * fg;
  auto load_a = [&](u32x4 (&dst)[C], int c0) {
#pragma unroll
    for (int j = 0; j < C; ++j) {
      const int s = c0 + j;
      dst[j] = u32x4{0u, 0u, 0u, 0u};
      if (s < kend && 32 * (int64_t)s + 8 * fg < K) dst[j] = *reinterpret_cast<const u32x4*>(wrow + 32 * (int64_t)s);
    }
  };

  XStager<W> xst;
  if constexpr (XL) xst.load(tk.X, M, K);
  u32x4 a[C], an[C];
  if (kbeg < kend) load_a(a, kbeg);
  if (threadIdx.x < 4) xzero[threadIdx.x] = u32x4{0u, 0u, 0u, 0u};
  if constexpr (XL) xst.store(xs, tk.X, K);
  __syncthreads();
  using XOp = std::conditional_t<XL, XShared, XGlobal<MT>>;
  const XOp xop = [&]() {
    if constexpr (XL) return XShared(xs, xzero, M, K, fr, fg);
    else return XGlobal<MT>(tk.X, M, K, fr, fg);
  }();

  f32x4 acc[MT];
#pragma unroll
  for (int t = 0; t < MT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int c0 = kbeg; c0 < kend; c0 += C) {
    if constexpr (XL) {
      if (c0 + C < kend) load_a(an, c0 + C);
      uint32_t xaddr = xop.addr + xop.step * (uint32_t)c0;
#pragma unroll
      for (int j = 0; j < C; ++j) {
        if (c0 + j < kend) acc[0] = Mfma16<T>::run(a[j], lds_load16(xaddr), acc[0]);   // staged columns only
        xaddr += xop.step;
      }
    } else {
      u32x4 xb[C][MT];
#pragma unroll
      for (int j = 0; j < C; ++j) {
        if (c0 + j < kend) {
          xop.load(xb[j], c0 + j, c0 + j == S - 1 && (K & 31) != 0, fg, K);
        } else {                                       // multiplied below: past the range it must be zero
#pragma unroll
          for (int t = 0; t < MT; ++t) xb[j][t] = u32x4{0u, 0u, 0u, 0u};
        }
      }
      if (c0 + C < kend) load_a(an, c0 + C);
#pragma unroll
      for (int j = 0; j < C; ++j)
#pragma unroll
        for (int t = 0; t < MT; ++t) acc[t] = Mfma16<T>::run(a[j], xb[j][t], acc[t]);
    }
#pragma unroll
    for (int j = 0; j < C; ++j) a[j] = an[j];
  }
  __syncthreads();                                     // every wave is done with the staged activations
  reduce_store<T, MT, W>(reinterpret_cast<float*>(dsm), acc, M, blk * kDecRows, N, tk.Y);
}

__global__ void __launch_bounds__(256) k_zero_out(uint16_t* __restrict__ Y, int64_t count) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count; i += (int64_t)gridDim.x * 256) Y[i] = 0;
}

size_t x_lds_bytes(int64_t M, int64_t K) { return (size_t)M * (size_t)xs_stride(K) * 2; }
constexpr size_t kXLdsAlloc = (size_t)kXLdsMax + 16 * 16;   // the most x_lds_bytes(M, K) can be (see variant)
template <int W>
constexpr size_t red_bytes() { return (size_t)W * 2 * 256 * sizeof(float); }

template <class T, int MT, bool XL, int W>
hipError_t sparse_group_launch(const SparseGroupArg& g, int64_t kmax, hipStream_t s) {
  auto* kernel = k_sparse_decode<T, MT, XL, W>;
  static PerDeviceFlag lds_set;
  const hipError_t attr = allow_lds_once(lds_set, kernel, sparse_vbuf_bytes<W>() + (XL ? kXLdsAlloc : 0));   // a bound
  if (attr != hipSuccess) return attr;
  const size_t lds = sparse_vbuf_bytes<W>() + (XL ? x_lds_bytes(g.M, kmax) : 0);
  hipLaunchKernelGGL(kernel, dim3((unsigned)g.first[g.count]), dim3(W * kWave), lds, s, g);
  return hipGetLastError();
}

template <class T, int MT, bool XL, int W>
hipError_t dense_group_launch(const DenseGroupArg& g, int64_t kmax, hipStream_t s) {
  auto* kernel = k_dense_decode<T, MT, XL, W>;
  static PerDeviceFlag lds_set;
  const hipError_t attr = allow_lds_once(lds_set, kernel, red_bytes<W>() > kXLdsAlloc ? red_bytes<W>() : kXLdsAlloc);
  if (attr != hipSuccess) return attr;
  const size_t xb = XL ? x_lds_bytes(g.M, kmax) : 0;
  const size_t lds = xb > red_bytes<W>() ? xb : red_bytes<W>();
  hipLaunchKernelGGL(kernel, dim3((unsigned)g.first[g.count]), dim3(W * kWave), lds, s, g);
  return hipGetLastError();
}

// Kernel variant for a group: activations in LDS when every task's staged
// rows fit (M * 32S * 2 <= budget, so x_lds_bytes <= kXLdsAlloc), each
// piece of them within the staging loads of a thread.
int variant(int64_t M, int64_t kmax, int64_t budget) {
  if (M <= 16 && M * 32 * tile_steps(kmax) * 2 <= budget) return 0;
  return M <= 16 ? 1 : 2;
}

// 16 waves per workgroup when the launch has fewer than two row blocks per CU.
bool small_grid(int64_t blocks) { return blocks < 2 * (int64_t)device_cus(); }
bool large_grid(int64_t blocks) { return blocks >= 4 * (int64_t)device_cus(); }

// Activation path of the sparse kernels.  One row: staged in LDS when it fits
// (32 KB).  Two to 16 rows: staged only where the launch has two or more row
// blocks per CU and the copy fits 32 KB (then at most ~57 KB of LDS per
// workgroup: two still share a CU); otherwise loaded directly, which fetches
// only the live rows.  Two row blocks per workgroup (direct path) pay off
// above four rows.
int sparse_variant(int64_t M, int64_t kmax, int64_t blocks) {
  const int64_t xbytes = M * 32 * tile_steps(kmax) * 2;
  if (M == 1 && xbytes <= kXLdsMaxSparse) return 0;
  if (M > 1 && M <= 16 && xbytes <= kXLdsMaxSparse && !small_grid(blocks)) return 0;
  return M <= 16 ? 1 : 2;
}

template <class T, int W>
hipError_t sparse_group_w(const SparseGroupArg& g, int64_t kmax, hipStream_t s) {
  switch (sparse_variant(g.M, kmax, g.first[g.count])) {
    case 0: return sparse_group_launch<T, 1, true, W>(g, kmax, s);
    case 1: return sparse_group_launch<T, 1, false, W>(g, kmax, s);
    default: return sparse_group_launch<T, 2, false, W>(g, kmax, s);
  }
}

// Two row blocks per workgroup (direct activations, MT batch tiles): the same
// group with each task's workgroups counted in pairs of row blocks.
template <class T, int W, int MT>
hipError_t sparse_pair_launch(const SparseGroupArg& g1, hipStream_t s) {
  SparseGroupArg g = g1;
  for (int i = 0; i < g.count; ++i)
    g.first[i + 1] = g.first[i] + (int32_t)((tile_blocks(g1.t[i].N) + 1) / 2);
  auto* kernel = k_sparse_decode2<T, W, false, false, MT>;
  static PerDeviceFlag lds_set;
  const hipError_t attr = allow_lds_once(lds_set, kernel, sparse2_vbuf_bytes<W>());
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(kernel, dim3((unsigned)g.first[g.count]), dim3(W * kWave), sparse2_vbuf_bytes<W>(), s, g);
  return hipGetLastError();
}

template <class T>
hipError_t sparse_group_t(const SparseGroupArg& g, int64_t kmax, hipStream_t s) {
  const int64_t blocks = g.first[g.count];
  // direct activations of more than 4 rows: pairs of row blocks when the pairs still fill the chip
  const int v = sparse_variant(g.M, kmax, blocks);
  if (v == 1 && g.M > 4 && !small_grid(blocks)) return sparse_pair_launch<T, 8, 1>(g, s);
  if (v == 2 && !small_grid(blocks)) return sparse_pair_launch<T, 8, 2>(g, s);
  if (small_grid(blocks)) return sparse_group_w<T, 16>(g, kmax, s);
  // four or more row blocks per CU: 4-wave workgroups, so that the whole grid is resident at once
  return large_grid(blocks) && g.M <= 16 ? sparse_group_w<T, 4>(g, kmax, s) : sparse_group_w<T, 8>(g, kmax, s);
}

template <class T, int W>
hipError_t dense_group_w(const DenseGroupArg& g, int64_t kmax, hipStream_t s) {
  switch (variant(g.M, kmax, kXLdsMax)) {
    case 0: return dense_group_launch<T, 1, true, W>(g, kmax, s);
    case 1: return dense_group_launch<T, 1, false, W>(g, kmax, s);
    default: return dense_group_launch<T, 2, false, W>(g, kmax, s);
  }
}

template <class T>
hipError_t dense_group_t(const DenseGroupArg& g, int64_t kmax, hipStream_t s) {
  return small_grid(g.first[g.count]) ? dense_group_w<T, 16>(g, kmax, s) : dense_group_w<T, 8>(g, kmax, s);
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
hipError_t launch_sparse_decode(const spl_sparse_task* tasks, int count, int64_t M, hipStream_t s) {
  SparseGroupArg g{};
  int64_t kmax = 0;
  g.first[0] = 0;
  for (int i = 0; i < count; ++i) {
    const spl_matrix& W = *tasks[i].W;
    g.t[i] = SparseTaskArg{static_cast<const uint16_t*>(tasks[i].X), static_cast<uint16_t*>(tasks[i].Y), W.bitmask,
                           static_cast<const uint16_t*>(W.values), W.tile_offsets, W.rows, W.cols};
    g.first[i + 1] = g.first[i] + (int32_t)tile_blocks(W.rows);
    if (W.cols > kmax) kmax = W.cols;
  }
  if (2 * M * kmax > kXBufMax) return hipErrorNotSupported;   // activations addressed with 32-bit offsets
  g.count = count;
  g.M = (int32_t)M;
  return tasks[0].W->dtype == SPL_BF16 ? sparse_group_t<Bf16>(g, kmax, s) : sparse_group_t<F16>(g, kmax, s);
}

// Gated half of a Llama MLP at batches of up to 16 rows: workgroup j pairs
// row block j of the gate and of the up matrix (k_sparse_decode2, kGated).
hipError_t launch_gated_decode(const void* X, int64_t M, const spl_matrix& Wg, const spl_matrix& Wu, void* Y,
                               hipStream_t s) {
  if (Wg.nnz == 0 || Wu.nnz == 0) return launch_zero_fill(Y, M * Wg.rows, s);   // silu(0) u = silu(g) 0 = 0
  if (2 * M * Wg.cols > kXBufMax) return hipErrorNotSupported;   // activations addressed with 32-bit offsets
  constexpr int W = 8;
  static_assert(W * 2 * kWave * 4 * sizeof(float) <= sparse2_vbuf_bytes<W>(), "both blocks' partial sums fit");
  SparseGroupArg g{};
  const int32_t B = (int32_t)tile_blocks(Wg.rows);
  g.t[0] = SparseTaskArg{static_cast<const uint16_t*>(X), static_cast<uint16_t*>(Y), Wg.bitmask,
                         static_cast<const uint16_t*>(Wg.values), Wg.tile_offsets, Wg.rows, Wg.cols};
  g.t[1] = SparseTaskArg{static_cast<const uint16_t*>(X), static_cast<uint16_t*>(Y), Wu.bitmask,
                         static_cast<const uint16_t*>(Wu.values), Wu.tile_offsets, Wu.rows, Wu.cols};
  g.first[0] = 0, g.first[1] = B, g.first[2] = B;
  g.count = 2;
  g.M = (int32_t)M;
  const bool xl = M == 1 && x_lds_bytes(1, Wg.cols) <= (size_t)kXLdsMax;   // one row: staged in LDS
  auto* kernel = Wg.dtype == SPL_BF16 ? (xl ? k_sparse_decode2<Bf16, W, true, true> : k_sparse_decode2<Bf16, W, true>)
                                      : (xl ? k_sparse_decode2<F16, W, true, true> : k_sparse_decode2<F16, W, true>);
  const size_t lds = sparse2_vbuf_bytes<W>() + (xl ? x_lds_bytes(1, Wg.cols) : 0);
  static PerDeviceFlag lds_set[4];                                                 // one per kernel above
  const hipError_t attr = allow_lds_once(lds_set[(Wg.dtype == SPL_BF16 ? 2 : 0) + (xl ? 1 : 0)], kernel,
                                         sparse2_vbuf_bytes<W>() + kXLdsMax);         // an upper bound
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL(kernel, dim3((unsigned)B), dim3(W * kWave), lds, s, g);
  return hipGetLastError();
}

hipError_t launch_dense_decode(const spl_dense_task* tasks, int count, int64_t M, int32_t dtype, hipStream_t s) {
  DenseGroupArg g{};
  int64_t kmax = 0;
  g.first[0] = 0;
  for (int i = 0; i < count; ++i) {
    g.t[i] = DenseTaskArg{static_cast<const uint16_t*>(tasks[i].X), static_cast<uint16_t*>(tasks[i].Y),
                          static_cast<const uint16_t*>(tasks[i].W), tasks[i].N, tasks[i].K};
    g.first[i + 1] = g.first[i] + (int32_t)tile_blocks(tasks[i].N);
    if (tasks[i].K > kmax) kmax = tasks[i].K;
  }
  if (2 * M * kmax > kXBufMax) return hipErrorNotSupported;   // activations addressed with 32-bit offsets
  g.count = count;
  g.M = (int32_t)M;
  return dtype == SPL_BF16 ? dense_group_t<Bf16>(g, kmax, s) : dense_group_t<F16>(g, kmax, s);
}

}  // namespace spl
